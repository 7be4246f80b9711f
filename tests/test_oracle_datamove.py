"""Pins for the oracle's plan, load, append and gather (CPU only).

The bit-copy steps are pinned by round trips and canaries rather than by
restating them: load then gather must give back the host-store content in
logical order, append then gather must give back the new rows, and every pool
block that no step names must keep its bits. The layout helper used to build
expectations (tests/pagedkv.py) restates the block layout with numpy reshapes,
independently of the oracle's element loops.
"""
import numpy as np
import pytest

from oracle import datamove as dm
from paper_2603_23049_amd import synth
from pagedkv import ceil_div, scatter_sequence

BS = 16


def _host_logical(host_k, host_v, host_blocks_row, p, d):
    """Host-store content of one sequence's first p tokens, [p][Hkv][d], via reshapes."""
    nb = ceil_div(p, BS)
    blks = host_blocks_row[:nb]
    Hkv = host_k.shape[1]
    k = host_k[blks].reshape(nb, Hkv, BS, d).transpose(0, 2, 1, 3).reshape(nb * BS, Hkv, d)[:p]
    v = host_v[blks].reshape(nb, Hkv, d, BS).transpose(0, 3, 1, 2).reshape(nb * BS, Hkv, d)[:p]
    return k, v


@pytest.mark.parametrize("prefix_lens,suffix_lens", [
    ([256], [64]), ([0, 32, 17], [5, 16, 31]), ([15, 1, 48], [1, 40, 16])])
def test_load_append_gather_round_trip(prefix_lens, suffix_lens):
    d, Hkv = 64, 2
    b = synth.ragged_batch("t", Hq=4, Hkv=Hkv, d=d, prefix_lens=prefix_lens,
                           suffix_lens=suffix_lens, pool_blocks=64, seed=5)
    layer = synth.make_layer(b)
    rng = np.random.Generator(np.random.PCG64(1))
    pool_k = synth.normal_bf16(rng, (64, Hkv, BS * d))
    pool_v = synth.normal_bf16(rng, (64, Hkv, BS * d))
    canary_k, canary_v = pool_k.copy(), pool_v.copy()
    plan = dm.plan(b.prefix_lens, b.suffix_lens, b.block_tables, b.host_blocks, BS)
    src, dst, slots, cu = plan
    assert list(cu) == [0] + list(np.cumsum(suffix_lens))
    assert len(src) == sum(ceil_div(p, BS) for p in prefix_lens)
    pk, pv = dm.pool_after_layer(pool_k, pool_v, layer.host_k, layer.host_v, plan,
                                 layer.k_new, layer.v_new, BS)
    lens = [p + s for p, s in zip(prefix_lens, suffix_lens)]
    k_all, v_all = dm.gather(pk, pv, b.block_tables, [0] * b.B, lens, d, BS)
    r = 0
    for i, (p, s) in enumerate(zip(prefix_lens, suffix_lens)):
        hk, hv = _host_logical(layer.host_k, layer.host_v, b.host_blocks[i], p, d)
        assert np.array_equal(k_all[r:r + p], hk) and np.array_equal(v_all[r:r + p], hv)
        nk = layer.k_new[cu[i]:cu[i + 1]]
        nv = layer.v_new[cu[i]:cu[i + 1]]
        assert np.array_equal(k_all[r + p:r + p + s], nk)
        assert np.array_equal(v_all[r + p:r + p + s], nv)
        r += p + s
    touched = set(int(x) for x in b.block_tables.ravel() if x >= 0)
    for blk in range(64):
        if blk not in touched:
            assert np.array_equal(pk[blk], canary_k[blk]) and np.array_equal(pv[blk], canary_v[blk])


def test_gather_matches_reshape_placement():
    rng = np.random.Generator(np.random.PCG64(2))
    d, Hkv, n = 128, 8, 70
    k = synth.normal_bf16(rng, (n, Hkv, d))
    v = synth.normal_bf16(rng, (n, Hkv, d))
    bt = rng.permutation(10)[:5].astype(np.int32)[None]
    pk = np.zeros((10, Hkv, BS * d), np.uint16)
    pv = np.zeros((10, Hkv, BS * d), np.uint16)
    scatter_sequence(pk, pv, bt[0], k, v, BS)
    gk, gv = dm.gather(pk, pv, bt, [3], [n - 3], d, BS)
    assert np.array_equal(gk, k[3:]) and np.array_equal(gv, v[3:])


def test_append_into_partial_prefix_block_keeps_cached_slots():
    d, Hkv = 64, 1
    b = synth.ragged_batch("t", Hq=1, Hkv=Hkv, d=d, prefix_lens=[20], suffix_lens=[30],
                           pool_blocks=8, seed=3)
    layer = synth.make_layer(b)
    pool = np.zeros((8, Hkv, BS * d), np.uint16)
    plan = dm.plan(b.prefix_lens, b.suffix_lens, b.block_tables, b.host_blocks, BS)
    src, dst, slots, _ = plan
    assert len(dst) == 2                               # block 1 holds 4 cached + 12 new tokens
    assert all(s // BS != dst[0] for s in slots)
    assert sum(1 for s in slots if s // BS == dst[1]) == 12
    pk, pv = dm.pool_after_layer(pool, pool.copy(), layer.host_k, layer.host_v, plan,
                                 layer.k_new, layer.v_new, BS)
    gk, gv = dm.gather(pk, pv, b.block_tables, [16], [4], d, BS)
    hk, hv = _host_logical(layer.host_k, layer.host_v, b.host_blocks[0], 20, d)
    assert np.array_equal(gk, hk[16:20]) and np.array_equal(gv, hv[16:20])


def test_plan_dedupes_shared_prefix_blocks_and_rejects_conflicts():
    bt = np.array([[5, 6, 7, -1], [5, 6, 9, 10]], np.int32)
    hb = np.array([[0, 1, -1], [0, 1, 2]], np.int32)
    src, dst, slots, cu = dm.plan([32, 48], [10, 5], bt, hb, BS)
    assert list(zip(src, dst)) == [(0, 5), (1, 6), (2, 9)]
    assert list(slots) == [7 * 16 + i for i in range(10)] + [10 * 16 + i for i in range(5)]
    with pytest.raises(dm.PlanError):            # one pool block from two host blocks
        dm.plan([32, 32], [1, 1], np.array([[5, 6, 7], [5, 8, 9]], np.int32),
                np.array([[0, 1], [2, 3]], np.int32), BS)
    with pytest.raises(dm.PlanError):            # a new token inside another sequence's loaded block
        dm.plan([16, 20], [4, 4], np.array([[3, 4], [3, 4]], np.int32),
                np.array([[0, -1], [0, 1]], np.int32), BS)
    with pytest.raises(dm.PlanError):            # two new tokens in one slot
        dm.plan([0, 0], [2, 2], np.array([[3], [3]], np.int32), np.zeros((2, 1), np.int32), BS)


def test_slot_mapping_brute_force_tiny_config():
    b = synth.tiny()
    src, dst, slots, cu = dm.plan(b.prefix_lens, b.suffix_lens, b.block_tables, b.host_blocks, BS)
    bt = b.block_tables[0]
    assert list(dst) == list(bt[:16]) and list(src) == list(range(16))
    # token 256+i sits in logical block 16 + i//16 at offset i%16
    assert list(slots) == [int(bt[16 + i // 16]) * 16 + i % 16 for i in range(64)]


def test_plan_offload_lists_exactly_the_computed_whole_chunks():
    """Brute force over tokens: a pool block is offloaded iff all tokens of its chunk are
    computed tokens of the sequence; order follows the sequences and positions."""
    bs, chunk = 16, 64
    prefix_lens = [0, 64, 70, 128, 0]
    suffix_lens = [200, 64, 130, 10, 63]
    rng = np.random.Generator(np.random.PCG64(11))
    need = [-(-(p + s) // bs) for p, s in zip(prefix_lens, suffix_lens)]
    perm = rng.permutation(sum(need)).astype(np.int32)
    bt = np.full((len(need), max(need)), -1, np.int32)
    off = 0
    for b, n in enumerate(need):
        bt[b, :n] = perm[off:off + n]
        off += n
    src, dst = dm.plan_offload(prefix_lens, suffix_lens, bt, bs, chunk, first_dst_block=5)
    want = []
    for b, (p, s) in enumerate(zip(prefix_lens, suffix_lens)):
        for lb in range(-(-(p + s) // bs)):
            c = (lb * bs) // chunk
            tokens = range(c * chunk, (c + 1) * chunk)
            if all(p <= t < p + s for t in tokens):
                want.append(int(bt[b, lb]))
    assert src.tolist() == want
    assert dst.tolist() == list(range(5, 5 + len(want)))
    # 0+200: chunks 0,1,2 (192 tokens); 64+64: chunk 1; 70+130: chunk 2 (128..191); 128+10: none; 0+63: none
    assert len(want) == (3 + 1 + 1) * (chunk // bs)


def test_offload_then_load_round_trip():
    rng = np.random.Generator(np.random.PCG64(12))
    pool_k = rng.integers(0, 65536, size=(20, 2, 64), dtype=np.uint16)
    pool_v = rng.integers(0, 65536, size=(20, 2, 64), dtype=np.uint16)
    host_k = np.zeros((6, 2, 64), np.uint16)
    host_v = np.zeros((6, 2, 64), np.uint16)
    src = [7, 3, 19, 0, 11, 12]
    dm.offload(pool_k, pool_v, host_k, host_v, src, range(6))
    back_k, back_v = np.zeros_like(pool_k), np.zeros_like(pool_v)
    dm.load(back_k, back_v, host_k, host_v, range(6), src)
    for i, s in enumerate(src):
        assert np.array_equal(back_k[s], pool_k[s]) and np.array_equal(back_v[s], pool_v[s])
        assert np.array_equal(host_k[i], pool_k[s])
    untouched = [b for b in range(20) if b not in src]
    assert not back_k[untouched].any()
