"""Seeded random shapes for both attention entry points against the fp64 oracle.

Each case draws a ragged batch (1-10 sequences; prefix and suffix lengths half from
block, tile and row-tile edges, half uniform; G from 1 to 16 query heads per kv head;
head_dim 64 or 128), runs the serial layer (load, append, prefill attention) and
checks every row, then runs the decode entry point on each sequence's last token over
the same pool and checks it against the same oracle rows."""
import numpy as np
import pytest
import torch

from oracle import attention as oattn
from oracle import datamove as odm
from paper_2603_23049_amd import pcr, synth
from gpuio import GpuLayer, MAX_ABS, MEAN_ABS, dev, error_stats, say, u16

pytestmark = pytest.mark.gpu

BS = 16
EDGE_P = [0, 1, 15, 16, 17, 63, 64, 65, 127, 128, 129]
EDGE_S = [1, 2, 31, 32, 33, 127, 128, 129]


def _config(seed):
    rng = np.random.Generator(np.random.PCG64(5000 + seed))
    G = int(rng.choice([1, 2, 3, 4, 5, 6, 7, 8, 12, 16]))
    Hkv = int(rng.choice([h for h in (1, 2, 4, 8) if h * G <= 32]))
    d = int(rng.choice([64, 128]))
    B = int(rng.integers(1, 11))
    pl = [int(rng.choice(EDGE_P)) if rng.random() < 0.5 else int(rng.integers(0, 1501)) for _ in range(B)]
    sl = [int(rng.choice(EDGE_S)) if rng.random() < 0.5 else int(rng.integers(0, 301)) for _ in range(B)]
    k = int(rng.integers(0, B))
    sl[k] = max(sl[k], 1)
    extra = int(rng.integers(0, 9))
    return G, Hkv, d, pl, sl, extra


def _check(got, want, label):
    mx, mean = error_stats(got, want)
    say(f"    {label}: max_abs={mx:.3e} mean_abs={mean:.3e}")
    assert np.all(np.isfinite(got)), label
    assert mx <= MAX_ABS and mean <= MEAN_ABS, f"{label}: max {mx} mean {mean}"


@pytest.mark.parametrize("seed", range(48))
def test_random_shapes_prefill_and_decode(seed):
    G, Hkv, d, pl, sl, extra = _config(seed)
    nblocks = sum(-(-(p + s) // BS) for p, s in zip(pl, sl)) + extra
    b = synth.ragged_batch(f"fuzz{seed}", Hq=Hkv * G, Hkv=Hkv, d=d, prefix_lens=pl, suffix_lens=sl,
                           pool_blocks=nblocks, seed=6000 + seed)
    data = synth.make_layer(b)
    rng = np.random.Generator(np.random.PCG64(7000 + seed))
    shape = (b.pool_blocks, Hkv, BS * d)
    pk0, pv0 = synth.normal_bf16(rng, shape), synth.normal_bf16(rng, shape)
    say(f"[gpu] fuzz seed={seed} G={G} Hkv={Hkv} d={d} B={b.B} T={b.T} prefix={pl} suffix={sl}")

    L = GpuLayer(b, data, pk0, pv0)
    L.run_serial("kernel_pull")
    plan = odm.plan(b.prefix_lens, b.suffix_lens, b.block_tables, b.host_blocks, BS)
    pk, pv = odm.pool_after_layer(pk0, pv0, data.host_k, data.host_v, plan, data.k_new, data.v_new, BS)
    cu = plan[3]
    want = oattn.attention(data.q, pk, pv, b.block_tables, np.asarray(pl, np.int32), cu, Hkv, BS)
    _check(L.out_f64(), want, f"prefill seed={seed}")

    # decode: each sequence's last token over its whole context, through the same pool
    seqs = [i for i in range(b.B) if sl[i] > 0]
    last = np.array([cu[i + 1] - 1 for i in seqs], np.int64)
    ctx = np.array([pl[i] + sl[i] for i in seqs], np.int32)
    bt = np.ascontiguousarray(np.asarray(b.block_tables)[seqs])
    out = torch.zeros((len(seqs), b.num_q_heads, d), dtype=torch.int16, device="cuda")
    say(f"[gpu] fuzz seed={seed} decode B={len(seqs)} ctx={ctx.tolist()}")
    pcr.decode_attn(dev(np.ascontiguousarray(data.q[last])), L.pool, dev(bt), dev(ctx), ctx, b.num_q_heads, out)
    torch.cuda.synchronize()
    got = synth.bf16_bits_to_f32(u16(out)).astype(np.float64)
    _check(got, want[last], f"decode seed={seed}")
