"""Seeded random batches against the oracle: both attention entry points, and the copies.

Each case draws a ragged batch (1-10 sequences; prefix and suffix lengths half from
block, tile and row-tile edges, half uniform; G from 1 to 16 query heads per kv head;
head_dim 64 or 128), runs the serial layer (load, append, prefill attention) and
checks every row, then runs the decode entry point on each sequence's last token over
the same pool and checks it against the same oracle rows. The copy cases draw batches
the same way and check the plans, the pool after load and append, a gather and an
offload bit for bit."""
import numpy as np
import pytest
import torch

from oracle import attention as oattn
from oracle import datamove as odm
from paper_2603_23049_amd import pcr, synth
from gpuio import GpuLayer, MAX_ABS, MEAN_ABS, dev, error_stats, pinned, say, u16

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

    # even seeds under the key-halves attention schedule, odd seeds under row halves
    sched = ("key_halves", "row_halves")[seed % 2]
    say(f"    attention schedule {sched}")
    pcr.prefill_attn_set_schedule(sched)
    try:
        L = GpuLayer(b, data, pk0, pv0)
        L.run_serial("kernel_pull")
    finally:
        pcr.prefill_attn_set_schedule("auto")
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


METHODS = ["kernel_pull", "dma_per_block", "dma_staged"]
MARK = np.uint16(0x5A5A)


@pytest.mark.parametrize("seed", range(24))
def test_random_batches_copies_bitexact(seed):
    """On random batches: the plans equal the oracle's; load (each method in turn) and
    append leave the pool equal to the oracle's bit for bit; a random token range of every
    sequence gathers bit-exactly; the computed chunks offload bit-exactly (each method in
    turn) and leave every unlisted host block untouched."""
    G, Hkv, d, pl, sl, extra = _config(100 + seed)
    nblocks = sum(-(-(p + s) // BS) for p, s in zip(pl, sl)) + extra
    b = synth.ragged_batch(f"copies{seed}", Hq=Hkv * G, Hkv=Hkv, d=d, prefix_lens=pl, suffix_lens=sl,
                           pool_blocks=nblocks, seed=8000 + seed)
    data = synth.make_layer(b)
    rng = np.random.Generator(np.random.PCG64(9000 + seed))
    shape = (b.pool_blocks, Hkv, BS * d)
    pk0, pv0 = synth.normal_bf16(rng, shape), synth.normal_bf16(rng, shape)
    plan_c = pcr.plan(pl, sl, b.block_tables, b.host_blocks, BS)
    plan_o = odm.plan(pl, sl, b.block_tables, b.host_blocks, BS)
    for got_a, want_a in zip(plan_c, plan_o):
        assert np.array_equal(got_a, want_a)
    method, off_method = METHODS[seed % 3], METHODS[(seed // 3) % 3]
    src, dst = plan_c[0], plan_c[1]
    say(f"[gpu] copies seed={seed} Hkv={Hkv} d={d} B={b.B} T={b.T} pairs={len(src)} load={method} "
        f"offload={off_method}")

    L = GpuLayer(b, data, pk0, pv0)
    ws = torch.empty(max(pcr.staged_workspace_bytes(max(len(src), 1), Hkv, d), 256), dtype=torch.uint8,
                     device="cuda")
    pcr.load_kv_layer(L.host, src, L.pool, dst, method=method, workspace=ws)
    L.append()
    torch.cuda.synchronize()
    pk, pv = odm.pool_after_layer(pk0, pv0, data.host_k, data.host_v, plan_o, data.k_new, data.v_new, BS)
    assert np.array_equal(u16(L.pool.k), pk), "K pool"
    assert np.array_equal(u16(L.pool.v), pv), "V pool"

    n_tok = [p + s for p, s in zip(pl, sl)]
    starts = np.array([int(rng.integers(0, n)) if n else 0 for n in n_tok], np.int32)
    lens = np.array([int(rng.integers(0, n - a + 1)) if n else 0 for n, a in zip(n_tok, starts)], np.int32)
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    total = int(cu[-1])
    k_out = torch.zeros((max(total, 1), Hkv, d), dtype=torch.int16, device="cuda")
    v_out = torch.zeros_like(k_out)
    pcr.gather_kv(L.pool, L.bt, dev(starts), dev(cu), total, k_out, v_out)
    torch.cuda.synchronize()
    wk, wv = odm.gather(pk, pv, b.block_tables, starts, lens, d, BS)
    assert np.array_equal(u16(k_out)[:total], wk) and np.array_equal(u16(v_out)[:total], wv), "gather"

    chunk = int(rng.choice([16, 64, 256]))
    osrc, odst = pcr.plan_offload(pl, sl, b.block_tables, BS, chunk, first_dst_block=1)
    wsrc, wdst = odm.plan_offload(pl, sl, b.block_tables, BS, chunk, 1)
    assert np.array_equal(osrc, wsrc) and np.array_equal(odst, wdst), "offload plan"
    if len(osrc) == 0:
        return
    n_host = int(odst.max()) + 2
    hshape = (n_host, Hkv, BS * d)
    host = pcr.HostKV(pinned(np.full(hshape, MARK, np.uint16)), pinned(np.full(hshape, MARK, np.uint16)), Hkv, d)
    ows = torch.empty(pcr.staged_workspace_bytes(len(osrc), Hkv, d), dtype=torch.uint8, device="cuda")
    pcr.offload_kv_layer(L.pool, osrc, host, odst, method=off_method, workspace=ows)
    torch.cuda.synchronize()
    hk, hv = np.full(hshape, MARK, np.uint16), np.full(hshape, MARK, np.uint16)
    odm.offload(pk, pv, hk, hv, osrc, odst)
    assert np.array_equal(u16(host.k), hk), "offloaded K"
    assert np.array_equal(u16(host.v), hv), "offloaded V"
