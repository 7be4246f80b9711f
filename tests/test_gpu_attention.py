"""GPU: prefix-prefill attention through the C ABI against the fp64 oracle.

Tolerance (bf16 inputs, fp32 accumulation, bf16 output): max |err| <= 2e-2 and
mean |err| <= 2e-3 against the fp64 oracle. Beyond the tolerance the HIP path
must be deterministic and bit-invariant to which physical blocks hold the KV.
Each test runs under both workgroup schedules (key halves, row halves).
"""
import functools

import numpy as np
import pytest
import torch

from oracle import attention as oattn
from oracle import datamove as odm
from paper_2603_23049_amd import synth
from gpuio import GpuLayer, MAX_ABS, MEAN_ABS, error_stats, say, u16

pytestmark = pytest.mark.gpu

BS = 16


@pytest.fixture(autouse=True, params=["key_halves", "row_halves"])
def schedule(request):
    """Every test of this module runs under both attention schedules (the default picks
    one per launch from its size; forcing each covers small and odd shapes with both)."""
    from paper_2603_23049_amd import pcr
    pcr.prefill_attn_set_schedule(request.param)
    yield request.param
    pcr.prefill_attn_set_schedule("auto")


def _pools(b, seed=99):
    rng = np.random.Generator(np.random.PCG64(seed))
    shape = (b.pool_blocks, b.num_kv_heads, BS * b.head_dim)
    return synth.normal_bf16(rng, shape), synth.normal_bf16(rng, shape)


def _oracle(b, data, pk0, pv0, rows=None, block_tables=None, host_blocks=None):
    bt = b.block_tables if block_tables is None else block_tables
    hb = b.host_blocks if host_blocks is None else host_blocks
    plan = odm.plan(b.prefix_lens, b.suffix_lens, bt, hb, BS)
    pk, pv = odm.pool_after_layer(pk0, pv0, data.host_k, data.host_v, plan, data.k_new, data.v_new, BS)
    return oattn.attention(data.q, pk, pv, bt, np.asarray(b.prefix_lens, np.int32), plan[3], b.num_kv_heads, BS,
                           rows=rows)


def _run(b, data, pk0, pv0, **kw):
    L = GpuLayer(b, data, pk0, pv0, **kw)
    L.run_serial("kernel_pull")
    return L


def _check(got, want, label):
    mx, mean = error_stats(got, want)
    say(f"    {label}: max_abs={mx:.3e} mean_abs={mean:.3e}")
    assert np.all(np.isfinite(got)), label
    assert mx <= MAX_ABS and mean <= MEAN_ABS, f"{label}: max {mx} mean {mean}"


def test_tiny_config_full():
    b = synth.tiny()
    data = synth.make_layer(b)
    pk0, pv0 = _pools(b)
    say("[gpu] attention tiny")
    L = _run(b, data, pk0, pv0)
    _check(L.out_f64(), _oracle(b, data, pk0, pv0), "tiny")


@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("G", [1, 2, 4, 5, 8, 16])
def test_edge_shapes(d, G):
    """p in {0,1,15,16,17,256}, s in {1,2,63,64} (all combinations in one ragged batch
    per (d, G)), plus a long ragged suffix spanning several row tiles. Row tiles hold
    128 packed (token, head) rows, so G = 5 puts tile edges inside a token's heads."""
    pl, sl = [], []
    for p in [0, 1, 15, 16, 17, 256]:
        for s in [1, 2, 63, 64]:
            pl.append(p)
            sl.append(s)
    pl.append(100)
    sl.append(300)
    Hkv = 2
    nblocks = sum(-(-(p + s) // BS) for p, s in zip(pl, sl)) + 5
    b = synth.ragged_batch("edges", Hq=Hkv * G, Hkv=Hkv, d=d, prefix_lens=pl, suffix_lens=sl,
                           pool_blocks=nblocks, seed=10 + d + G)
    data = synth.make_layer(b)
    pk0, pv0 = _pools(b)
    say(f"[gpu] attention edges d={d} G={G} B={b.B} T={b.T}")
    L = _run(b, data, pk0, pv0)
    _check(L.out_f64(), _oracle(b, data, pk0, pv0), f"edges d={d} G={G}")


@pytest.mark.parametrize("G,Hkv,d", [(24, 2, 128), (32, 2, 64), (64, 1, 128)])
def test_wide_groups(G, Hkv, d):
    """More than 16 query heads per kv head: one-token rows then take prefill tiles
    (the decode workgroups hold at most 16 heads), and a token's heads span several
    32-row wave slices and 128-row tiles."""
    pl, sl = [], []
    for p in [0, 17, 256]:
        for s in [1, 2, 63]:
            pl.append(p)
            sl.append(s)
    pl.append(100)
    sl.append(300)
    nblocks = sum(-(-(p + s) // BS) for p, s in zip(pl, sl)) + 5
    b = synth.ragged_batch("wide", Hq=Hkv * G, Hkv=Hkv, d=d, prefix_lens=pl, suffix_lens=sl,
                           pool_blocks=nblocks, seed=70 + G)
    data = synth.make_layer(b)
    pk0, pv0 = _pools(b)
    say(f"[gpu] attention wide groups G={G} Hkv={Hkv} d={d} B={b.B} T={b.T}")
    L = _run(b, data, pk0, pv0)
    _check(L.out_f64(), _oracle(b, data, pk0, pv0), f"wide G={G} d={d}")


@pytest.mark.parametrize("B", [100, 140])
def test_many_sequences(B):
    """More sequences than one lane of the work-map lookup holds (slots 64.. are read by
    the second half of each lane's loads) and, at B = 140, more than the map holds (133
    with new tokens: two launches, the sequences dealt round robin). Some sequences have
    no new tokens."""
    rng = np.random.Generator(np.random.PCG64(1000 + B))
    pl = [int(rng.integers(0, 80)) for _ in range(B)]
    sl = [int(rng.integers(0, 24)) for _ in range(B)]
    sl[0], sl[-1] = 0, 40
    Hkv = 8
    nblocks = sum(-(-(p + s) // BS) for p, s in zip(pl, sl)) + 7
    b = synth.ragged_batch(f"many{B}", Hq=2 * Hkv, Hkv=Hkv, d=128, prefix_lens=pl, suffix_lens=sl,
                           pool_blocks=nblocks, seed=20 + B)
    data = synth.make_layer(b)
    pk0, pv0 = _pools(b)
    say(f"[gpu] attention many sequences B={b.B} T={b.T}")
    L = _run(b, data, pk0, pv0)
    _check(L.out_f64(), _oracle(b, data, pk0, pv0), f"B={B}")


@pytest.mark.parametrize("n_dec", [120, 280])
def test_mixed_prefill_and_many_decode_rows(n_dec):
    """Prefill requests among many decode rows (one new token each, contexts not a
    multiple of 16): 8 + 120 sequences fill one work map, 8 + 280 take three launches
    (sequences dealt round robin). Every row against the oracle, and the result
    repeated bit for bit."""
    rng = np.random.Generator(np.random.PCG64(3000 + n_dec))
    pl = [int(rng.integers(100, 900)) for _ in range(8)] + [int(rng.integers(1, 700)) for _ in range(n_dec)]
    sl = [int(rng.integers(60, 200)) for _ in range(8)] + [1] * n_dec
    order = rng.permutation(len(pl))
    pl, sl = [pl[i] for i in order], [sl[i] for i in order]
    Hkv = 4
    nblocks = sum(-(-(p + s) // BS) for p, s in zip(pl, sl)) + 3
    b = synth.ragged_batch(f"mixed{n_dec}", Hq=4 * Hkv, Hkv=Hkv, d=128, prefix_lens=pl, suffix_lens=sl,
                           pool_blocks=nblocks, seed=40 + n_dec)
    data = synth.make_layer(b)
    pk0, pv0 = _pools(b)
    say(f"[gpu] attention mixed prefill + {n_dec} decode rows B={b.B} T={b.T}")
    L = _run(b, data, pk0, pv0)
    first = u16(L.out).copy()
    _check(L.out_f64(), _oracle(b, data, pk0, pv0), f"mixed n_dec={n_dec}")
    L.out.zero_()
    L.attn()
    torch.cuda.synchronize()
    assert np.array_equal(u16(L.out), first), "attention is not deterministic"


def test_l8b_layer_full_and_deterministic():
    b = synth.l8b_layer()
    data = synth.make_layer(b)
    pk0, pv0 = _pools(b)
    say("[gpu] attention l8b_layer (full oracle)")
    L = _run(b, data, pk0, pv0)
    first = u16(L.out).copy()
    _check(L.out_f64(), _oracle(b, data, pk0, pv0), "l8b_layer")
    L.out.zero_()
    L.attn()
    torch.cuda.synchronize()
    assert np.array_equal(u16(L.out), first), "attention is not deterministic"


def test_block_permutation_and_sharing_bit_invariance():
    """Same logical KV under a different physical block assignment, and with two
    sequences sharing their common prefix blocks: outputs identical bit for bit."""
    Hkv, G, d = 2, 4, 128
    pl, sl = [512, 512, 96], [70, 33, 50]
    b = synth.ragged_batch("perm", Hq=Hkv * G, Hkv=Hkv, d=d, prefix_lens=pl, suffix_lens=sl, pool_blocks=160,
                           seed=21)
    data = synth.make_layer(b)
    # sequences 0 and 1 hold the same cached prefix (same host blocks)
    hb = b.host_blocks.copy()
    hb[1, :32] = hb[0, :32]
    pk0, pv0 = _pools(b)
    say("[gpu] attention permutation/sharing")
    ref = _run(b, data, pk0, pv0, host_blocks=hb)
    rng = np.random.Generator(np.random.PCG64(5))
    perm = rng.permutation(b.pool_blocks).astype(np.int32)
    bt2 = np.where(b.block_tables >= 0, perm[np.maximum(b.block_tables, 0)], -1).astype(np.int32)
    alt = _run(b, data, pk0, pv0, host_blocks=hb, block_tables=bt2)
    assert np.array_equal(u16(ref.out), u16(alt.out)), "output depends on physical block ids"
    bt3 = bt2.copy()
    bt3[1, :32] = bt3[0, :32]   # shared physical prefix blocks
    shared = _run(b, data, pk0, pv0, host_blocks=hb, block_tables=bt3)
    assert len(shared.dst) == len(alt.dst) - 32
    assert np.array_equal(u16(ref.out), u16(shared.out)), "shared prefix blocks change the output"
    _check(ref.out_f64(), _oracle(b, data, pk0, pv0, host_blocks=hb), "perm")


def test_l70b_shape_sampled_rows():
    """70B-shaped layer (64 q / 8 kv heads, p=15360, s=1024): every head of a spread of
    tokens, including the first and last suffix row of both sequences."""
    b = synth.l70b_pipe80()
    data = synth.make_layer(b)
    pk0, pv0 = _pools(b)
    say("[gpu] attention l70b layer 0 (sampled rows)")
    L = _run(b, data, pk0, pv0)
    toks = sorted(set([0, 1, 511, 1023, 1024, 1025, 1500, 2047] + list(range(37, 2048, 211))))
    rows = np.array([[t, h] for t in toks for h in range(b.num_q_heads)], np.int32)
    want = _oracle(b, data, pk0, pv0, rows=rows)
    got = L.out_f64()[rows[:, 0], rows[:, 1]]
    _check(got, want, "l70b sampled")


def test_l70b_tp8_shard_sampled_rows():
    """One GPU's share of the 70B-shaped layer at tensor parallelism 8 (8 q heads, 1 kv
    head, p = 15360, s = 1024): a kv-head count that is not a multiple of the XCD count
    (the work map's padded order). Every head of a spread of tokens, including the first
    and last suffix row of both sequences."""
    b = synth.uniform_batch("l70b_tp8_shard", B=2, Hq=8, Hkv=1, d=128, p=15360, s=1024, pool_blocks=4096,
                            seed=5)
    data = synth.make_layer(b)
    pk0, pv0 = _pools(b)
    say("[gpu] attention l70b tp8 shard (sampled rows)")
    L = _run(b, data, pk0, pv0)
    toks = sorted(set([0, 1, 511, 1023, 1024, 1025, 2047] + list(range(53, 2048, 173))))
    rows = np.array([[t, h] for t in toks for h in range(b.num_q_heads)], np.int32)
    want = _oracle(b, data, pk0, pv0, rows=rows)
    got = L.out_f64()[rows[:, 0], rows[:, 1]]
    _check(got, want, "tp8 shard sampled")


def test_rag_mix_sampled_rows_and_pool():
    """RAG-mix batch (16 ragged requests, prefixes hit in a warmed prefix tree, shared
    tree chunks loaded once, two sequences with no hit): the pool after load + append is
    the oracle's bit for bit, and sampled rows of every sequence (first, second, middle
    and last suffix rows plus a spread) match the oracle for every head."""
    from paper_2603_23049_amd import prefix_tree
    b = prefix_tree.rag_mix_batch()
    data = synth.make_layer(b)
    pk0, pv0 = _pools(b)
    say(f"[gpu] attention rag_mix (T={b.T}, {b.note})")
    L = _run(b, data, pk0, pv0)
    plan = odm.plan(b.prefix_lens, b.suffix_lens, b.block_tables, b.host_blocks, BS)
    pk, pv = odm.pool_after_layer(pk0, pv0, data.host_k, data.host_v, plan, data.k_new, data.v_new, BS)
    assert np.array_equal(u16(L.pool.k).reshape(pk.shape), pk), "pool K after load + append"
    assert np.array_equal(u16(L.pool.v).reshape(pv.shape), pv), "pool V after load + append"
    cu = b.cu_suffix
    rng = np.random.Generator(np.random.PCG64(404))
    toks = []
    for i, s in enumerate(b.suffix_lens):
        local = {0, 1, s // 2, s - 2, s - 1} | set(rng.integers(0, s, size=4).tolist())
        toks += [int(cu[i]) + t for t in sorted(local) if 0 <= t < s]
    rows = np.array([[t, h] for t in toks for h in range(b.num_q_heads)], np.int32)
    want = oattn.attention(data.q, pk, pv, b.block_tables, np.asarray(b.prefix_lens, np.int32), plan[3],
                           b.num_kv_heads, BS, rows=rows)
    got = L.out_f64()[rows[:, 0], rows[:, 1]]
    _check(got, want, "rag_mix sampled")


@functools.lru_cache(maxsize=2)
def _mixed_full_case(n_dec):
    """RAG-mix request lengths + n_dec decode rows of 4352 keys, with one layer's data
    (drawn once for both schedules)."""
    from paper_2603_23049_amd import prefix_tree
    rag = prefix_tree.rag_mix_batch()
    ctx = 4352
    pl = list(rag.prefix_lens) + [ctx - 1] * n_dec
    sl = list(rag.suffix_lens) + [1] * n_dec
    nblocks = sum(-(-(p + s) // BS) for p, s in zip(pl, sl))
    b = synth.ragged_batch("mixed_full", Hq=rag.num_q_heads, Hkv=rag.num_kv_heads, d=rag.head_dim,
                           prefix_lens=pl, suffix_lens=sl, pool_blocks=nblocks, seed=4352 + n_dec)
    return b, synth.make_layer(b), sl, ctx


@pytest.mark.parametrize("n_dec", [64, 256])
def test_mixed_rag_and_decode_rows_full_size(n_dec):
    """The benchmark's mixed launches: the RAG mix's 16 request lengths plus 64 decode rows
    of 4352 keys (32 q / 8 kv heads, d = 128) in one launch, decode rows spread over the
    prefill tiles; with 256 decode rows, three launches of the sequences dealt round robin.
    Every head of every decode row, and the first, middle and last rows of every request,
    against the oracle."""
    b, data, sl, ctx = _mixed_full_case(n_dec)
    shape = (b.pool_blocks, b.num_kv_heads, BS * b.head_dim)
    zero = np.zeros(shape, np.uint16)
    say(f"[gpu] attention mixed full size: rag mix + {n_dec} decode rows of {ctx} keys (T={b.T})")
    L = _run(b, data, zero, zero)
    cu = b.cu_suffix
    toks = []
    for i, s in enumerate(sl):
        toks += sorted({int(cu[i]) + t for t in (0, s // 2, s - 1)})
    heads = range(b.num_q_heads)
    rows = np.array([[t, h] for t in toks for h in heads], np.int32)
    want = _oracle(b, data, zero, zero, rows=rows)
    got = L.out_f64()[rows[:, 0], rows[:, 1]]
    _check(got, want, "mixed full size")


def test_long_context_128k_sampled_rows():
    """One sequence with a 131072-token cached prefix and 256 new tokens (32 q / 8 kv
    heads, d = 128): 2052 key tiles per row tile, so the online softmax runs over
    131k keys in fp32. Sampled rows of every eighth head against the fp64 oracle."""
    b = synth.ragged_batch("long128k", Hq=32, Hkv=8, d=128, prefix_lens=[131072], suffix_lens=[256],
                           pool_blocks=8256, seed=77)
    data = synth.make_layer(b)
    shape = (b.pool_blocks, b.num_kv_heads, BS * b.head_dim)
    zero = np.zeros(shape, np.uint16)
    say("[gpu] attention 128k-token prefix (sampled rows)")
    L = _run(b, data, zero, zero)
    rows = np.array([[t, h] for t in (0, 1, 127, 128, 254, 255) for h in range(0, 32, 8)], np.int32)
    want = _oracle(b, data, zero, zero, rows=rows)
    got = L.out_f64()[rows[:, 0], rows[:, 1]]
    _check(got, want, "128k prefix")


@pytest.mark.parametrize("scale", [0.0, 8.0, 32.0])
def test_softmax_flat_and_sharp(scale):
    """Queries scaled by 0 (every score equal: the output is the mean of the visible
    values), 8 and 32 (near one-hot rows whose running max rises by more than 2^8
    again and again, so the lazy rescale runs)."""
    pl, sl = [0, 1, 100, 1000, 3000], [64, 300, 33, 129, 256]
    b = synth.ragged_batch("sharp", Hq=16, Hkv=4, d=128, prefix_lens=pl, suffix_lens=sl,
                           pool_blocks=sum(-(-(p + s) // BS) for p, s in zip(pl, sl)) + 4, seed=55)
    data = synth.make_layer(b)
    q = synth.bf16_bits_to_f32(data.q) * np.float32(scale)
    data = synth.LayerData(q=synth.f32_to_bf16_bits(q), k_new=data.k_new, v_new=data.v_new, host_k=data.host_k,
                           host_v=data.host_v)
    pk0, pv0 = _pools(b)
    say(f"[gpu] attention softmax scale x{scale}")
    L = _run(b, data, pk0, pv0)
    _check(L.out_f64(), _oracle(b, data, pk0, pv0), f"q x{scale}")
