"""HIP graph capture of the per-layer compute step (append, then attention) through the
C ABI. The step is captured once (torch's CUDAGraph, which is a hipGraph on this
runtime: the library's launches on the capturing stream become graph nodes) and
replayed several times, with eager work and device synchronisations between replays.
Before each replay the output is set to NaN bit patterns and the suffix slots of the
pool are poisoned, so a replay that did not run its kernels would fail. Every replay
must equal the eager step bit for bit (both kernels are deterministic and neither
records a memset), and the eager step equals the fp64 oracle within the tolerance."""
import numpy as np
import pytest
import torch

from oracle import attention as oattn
from oracle import datamove as odm
from paper_2603_23049_amd import synth
from gpuio import MAX_ABS, MEAN_ABS, GpuLayer, attn_schedule, error_stats, say

pytestmark = pytest.mark.gpu
BS = 16


def _poison_suffix_slots(L):
    """NaN bit patterns (0xFFFF) in every pool slot the append writes."""
    b = L.batch
    kv = L.pool.k.view(b.pool_blocks, b.num_kv_heads, BS, b.head_dim)
    vv = L.pool.v.view(b.pool_blocks, b.num_kv_heads, b.head_dim, BS)
    slots = torch.from_numpy(L.slots_np.astype(np.int64)).cuda()
    blk, off = slots // BS, slots % BS
    kv[blk, :, off, :] = -1
    vv[blk, :, :, off] = -1


@pytest.mark.parametrize("schedule", ["key_halves", "row_halves"])
@pytest.mark.parametrize("name", ["tiny", "l8b_layer"])
def test_graph_replay_of_layer_step_bitwise(name, schedule):
    b = synth.REGISTRY[name]()
    data = synth.make_layer(b)
    rng = np.random.Generator(np.random.PCG64(31))
    shape = (b.pool_blocks, b.num_kv_heads, BS * b.head_dim)
    pk0, pv0 = synth.normal_bf16(rng, shape), synth.normal_bf16(rng, shape)
    say(f"[gpu] graph replay of append + attention: {name}, {schedule}")
    L = GpuLayer(b, data, pk0, pv0)
    L.load("kernel_pull")
    torch.cuda.synchronize()
    with attn_schedule(schedule):
        L.append()
        L.attn()
        torch.cuda.synchronize()
        want_out, want_k, want_v = L.out.clone(), L.pool.k.clone(), L.pool.v.clone()

        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):      # one eager step on the capture stream first
            L.append()
            L.attn()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            L.append()
            L.attn()
        torch.cuda.synchronize()
        for rep in range(3):
            L.out.fill_(-1)
            _poison_suffix_slots(L)
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            assert torch.equal(L.out, want_out), f"replay {rep}: output differs from the eager step"
            assert torch.equal(L.pool.k, want_k) and torch.equal(L.pool.v, want_v), \
                f"replay {rep}: pool differs from the eager step"
            # eager work between replays
            L.attn()
            torch.cuda.synchronize()
            assert torch.equal(L.out, want_out)
        del g

    plan = odm.plan(b.prefix_lens, b.suffix_lens, b.block_tables, b.host_blocks, BS)
    pk, pv = odm.pool_after_layer(pk0, pv0, data.host_k, data.host_v, plan, data.k_new, data.v_new, BS)
    assert np.array_equal(want_k.cpu().numpy().view(np.uint16), pk)
    assert np.array_equal(want_v.cpu().numpy().view(np.uint16), pv)
    rows = None
    if name != "tiny":   # every 37th (token, q head) row of the 8B layer
        flat = np.arange(0, b.T * b.num_q_heads, 37)
        rows = np.stack([flat // b.num_q_heads, flat % b.num_q_heads], 1).astype(np.int32)
    ref = oattn.attention(data.q, pk, pv, b.block_tables, np.asarray(b.prefix_lens, np.int32), plan[3],
                          b.num_kv_heads, BS, rows=rows)
    got = synth.bf16_bits_to_f32(want_out.cpu().numpy().view(np.uint16)).astype(np.float64)
    if rows is not None:
        got = got[rows[:, 0], rows[:, 1]]
    mx, mean = error_stats(got, ref)
    say(f"    oracle: max_abs={mx:.3e} mean_abs={mean:.3e}")
    assert mx <= MAX_ABS and mean <= MEAN_ABS
