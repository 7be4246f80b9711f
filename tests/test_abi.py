"""The C ABI without a GPU: the library loads, exports every declared symbol,
plans batches exactly as the oracle does, and rejects bad arguments on the
host before anything is enqueued."""
import ctypes
import os
import re

import numpy as np
import pytest

from oracle import datamove as odm
from paper_2603_23049_amd import pcr, synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    text = open(os.path.join(ROOT, "include", "pcr.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(pcr_[a-z_0-9]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    L = pcr.lib()
    declared = _declared_functions()
    assert "pcr_prefix_prefill_attn" in declared and len(declared) >= 8
    for name in declared:
        assert hasattr(L, name), f"{name} declared in pcr.h but not exported"
    assert set(declared) == set(pcr.EXPORTS)
    assert "gfx950" in pcr.version()


@pytest.mark.parametrize("mk", [synth.tiny, synth.l8b_layer, synth.l70b_pipe80])
def test_plan_matches_oracle_on_configs(mk):
    b = mk()
    want = odm.plan(b.prefix_lens, b.suffix_lens, b.block_tables, b.host_blocks, b.block_size)
    got = pcr.plan(b.prefix_lens, b.suffix_lens, b.block_tables, b.host_blocks, b.block_size)
    for w, g in zip(want, got):
        assert np.array_equal(w, g)


def test_plan_matches_oracle_ragged_shared_and_partial():
    rng = np.random.Generator(np.random.PCG64(4))
    for trial in range(50):
        B = int(rng.integers(1, 6))
        pl = rng.integers(0, 80, size=B).tolist()
        sl = rng.integers(0, 40, size=B).tolist()
        b = synth.ragged_batch("r", Hq=2, Hkv=1, d=64, prefix_lens=pl, suffix_lens=sl, pool_blocks=64,
                               seed=int(rng.integers(1 << 30)))
        bt, hb = b.block_tables.copy(), b.host_blocks.copy()
        if B >= 2 and pl[0] >= 32 and pl[1] >= 32 and trial % 2 == 0:
            # two sequences share their first two full prefix blocks (same host and pool blocks)
            bt[1, :2] = bt[0, :2]
            hb[1, :2] = hb[0, :2]
        try:
            want = odm.plan(pl, sl, bt, hb, 16)
        except odm.PlanError:
            with pytest.raises(pcr.PcrError) as ei:
                pcr.plan(pl, sl, bt, hb, 16)
            assert ei.value.status == pcr.PCR_ERR_INVALID_ARG
            continue
        got = pcr.plan(pl, sl, bt, hb, 16)
        for w, g in zip(want, got):
            assert np.array_equal(w, g), (trial, pl, sl)


def test_plan_rejects_what_the_oracle_rejects():
    cases = [
        ([32, 32], [1, 1], [[5, 6, 7], [5, 8, 9]], [[0, 1], [2, 3]]),
        ([16, 20], [4, 4], [[3, 4], [3, 4]], [[0, -1], [0, 1]]),
        ([0, 0], [2, 2], [[3], [3]], [[0], [0]]),
        ([16], [1], [[3, -1]], [[0]]),
    ]
    for pl, sl, bt, hb in cases:
        bt, hb = np.array(bt, np.int32), np.array(hb, np.int32)
        with pytest.raises(odm.PlanError):
            odm.plan(pl, sl, bt, hb, 16)
        with pytest.raises(pcr.PcrError):
            pcr.plan(pl, sl, bt, hb, 16)


def _pool(nb=4, Hkv=1, d=64, bs=16, k=0x10000, v=0x20000):
    return pcr._Pool(k, v, nb, bs, Hkv, d)


def test_argument_validation_before_any_device_work():
    L = pcr.lib()
    P = ctypes.byref
    # unsupported head_dim / block_size
    assert L.pcr_append_kv(P(_pool(d=96)), 16, 16, 16, 4, None) == pcr.PCR_ERR_UNSUPPORTED
    assert L.pcr_append_kv(P(_pool(bs=32)), 16, 16, 16, 4, None) == pcr.PCR_ERR_UNSUPPORTED
    assert "block_size" in pcr.last_error()
    # null pool pointers, misaligned inputs, negative sizes
    assert L.pcr_append_kv(P(_pool(k=0)), 16, 16, 16, 4, None) == pcr.PCR_ERR_INVALID_ARG
    assert L.pcr_append_kv(P(_pool()), 18, 16, 16, 4, None) == pcr.PCR_ERR_INVALID_ARG
    assert L.pcr_append_kv(P(_pool()), 16, 16, 16, -1, None) == pcr.PCR_ERR_INVALID_ARG
    # empty work is a no-op
    assert L.pcr_append_kv(P(_pool()), None, None, None, 0, None) == pcr.PCR_OK
    # attention: Hq not a multiple of Hkv, bad scale, too-short block table
    hpl = np.array([16], np.int32)
    hcu = np.array([0, 8], np.int32)
    args = lambda Hq, scale, mb: (16, P(_pool(Hkv=2)), 16, mb, 16, 16, hpl.ctypes.data, hcu.ctypes.data, 1, Hq,
                                  scale, 16, None)
    assert L.pcr_prefix_prefill_attn(*args(3, 0.125, 4)) == pcr.PCR_ERR_UNSUPPORTED
    assert L.pcr_prefix_prefill_attn(*args(4, 0.0, 4)) == pcr.PCR_ERR_INVALID_ARG
    assert L.pcr_prefix_prefill_attn(*args(4, 0.125, 1)) == pcr.PCR_ERR_INVALID_ARG
    hcu0 = np.array([0, 0], np.int32)
    assert L.pcr_prefix_prefill_attn(16, P(_pool()), 16, 4, 16, 16, hpl.ctypes.data, hcu0.ctypes.data, 1, 1,
                                     0.125, 16, None) == pcr.PCR_OK
    # decode: more than 16 query heads per kv head, a sequence with no key, a too-short
    # block table, bad scale; B = 0 is a no-op (all rejected before the device is asked
    # for its compute-unit count)
    hcl = np.array([40, 1], np.int32)
    dargs = lambda Hq, scale, mb, lens: (16, P(_pool(Hkv=2)), 16, mb, 16, lens.ctypes.data, 2, Hq, scale, 16,
                                         None, 0, None)
    assert L.pcr_decode_attn(*dargs(34, 0.125, 4, hcl)) == pcr.PCR_ERR_UNSUPPORTED
    assert "query heads per kv head" in pcr.last_error()
    assert L.pcr_decode_attn(*dargs(3, 0.125, 4, hcl)) == pcr.PCR_ERR_UNSUPPORTED
    assert L.pcr_decode_attn(*dargs(4, 0.0, 4, hcl)) == pcr.PCR_ERR_INVALID_ARG
    assert L.pcr_decode_attn(*dargs(4, 0.125, 2, hcl)) == pcr.PCR_ERR_INVALID_ARG
    assert "max_blocks" in pcr.last_error()
    assert L.pcr_decode_attn(*dargs(4, 0.125, 4, np.array([40, 0], np.int32))) == pcr.PCR_ERR_INVALID_ARG
    assert "no visible key" in pcr.last_error()
    assert L.pcr_decode_attn(16, P(_pool()), 16, 4, 16, hcl.ctypes.data, 0, 1, 0.125, 16, None, 0, None) == \
        pcr.PCR_OK
    nbytes = ctypes.c_int64(-1)
    assert L.pcr_decode_attn_workspace_size(4, 34, 2, 128, 100, ctypes.byref(nbytes)) == pcr.PCR_ERR_UNSUPPORTED
    assert L.pcr_decode_attn_workspace_size(4, 8, 2, 96, 100, ctypes.byref(nbytes)) == pcr.PCR_ERR_UNSUPPORTED
    assert L.pcr_decode_attn_workspace_size(0, 8, 2, 128, 100, ctypes.byref(nbytes)) == pcr.PCR_OK
    assert nbytes.value == 0
    # load: block ids out of range and repeated destinations are caught on the host
    host = pcr._Host(0x30000, 0x40000, 8, 16, 1, 64)
    src = np.array([0, 9], np.int32)
    dst = np.array([1, 2], np.int32)
    assert L.pcr_load_kv_layer(P(host), src.ctypes.data, P(_pool()), dst.ctypes.data, 2, None) == \
        pcr.PCR_ERR_INVALID_ARG
    src = np.array([0, 1], np.int32)
    dst = np.array([1, 1], np.int32)
    assert L.pcr_load_kv_layer(P(host), src.ctypes.data, P(_pool()), dst.ctypes.data, 2, None) == \
        pcr.PCR_ERR_INVALID_ARG
    assert "twice" in pcr.last_error()
    assert L.pcr_load_kv_layer(P(host), None, P(_pool()), None, 0, None) == pcr.PCR_OK
    host_bad = pcr._Host(0x30000, 0x40000, 8, 16, 2, 64)
    assert L.pcr_load_kv_layer(P(host_bad), src.ctypes.data, P(_pool()), dst.ctypes.data, 2, None) == \
        pcr.PCR_ERR_INVALID_ARG
    assert L.pcr_load_kv_layer_method(P(host), src.ctypes.data, P(_pool()), dst.ctypes.data, 2, 9, None) == \
        pcr.PCR_ERR_INVALID_ARG
    # pipeline: zero layers is a no-op, equal streams are refused
    assert L.pcr_pipeline_run(None, 0, None, 0, None, None, None) == pcr.PCR_OK
    lay = (pcr._LayerIO * 1)()
    bat = pcr._Batch()
    assert L.pcr_pipeline_run(lay, 1, P(bat), 0, 0x5, 0x5, None) == pcr.PCR_ERR_INVALID_ARG
    # the attention arguments of every layer are checked before anything is queued
    # (the stream handles are never used on these paths)
    lay2 = (pcr._LayerIO * 2)()
    for i in range(2):
        lay2[i].pool = _pool(Hkv=2, k=0x10000 + 0x100000 * i, v=0x20000 + 0x100000 * i)
        lay2[i].q = lay2[i].out = 16
    bat2 = pcr._Batch(block_tables=16, max_blocks=4, prefix_lens=16, cu_suffix=16,
                      host_prefix_lens=hpl.ctypes.data, host_cu_suffix=hcu.ctypes.data, B=1, num_q_heads=4,
                      sm_scale=0.0)
    assert L.pcr_pipeline_run(lay2, 2, P(bat2), 0, 0x5, 0x6, None) == pcr.PCR_ERR_INVALID_ARG
    assert "pcr_pipeline_run" in pcr.last_error() and "sm_scale" in pcr.last_error()
    bat2.sm_scale = 0.125
    lay2[1].q = 18                     # misaligned q in the second layer
    assert L.pcr_pipeline_run(lay2, 2, P(bat2), 0, 0x5, 0x6, None) == pcr.PCR_ERR_INVALID_ARG
    assert "aligned" in pcr.last_error()
    lay2[1].q = 16
    # two layers on one pool (or a pool whose K is its V) are refused before anything is queued
    lay2[1].pool = _pool(Hkv=2)
    lay2[0].pool = _pool(Hkv=2)
    assert L.pcr_pipeline_run(lay2, 2, P(bat2), 0, 0x5, 0x6, None) == pcr.PCR_ERR_INVALID_ARG
    assert "own pool" in pcr.last_error()
    lay2[1].pool = _pool(Hkv=2, k=0x50000, v=0x50000)
    lay2[0].pool = _pool(Hkv=2)
    assert L.pcr_pipeline_run(lay2, 2, P(bat2), 0, 0x5, 0x6, None) == pcr.PCR_ERR_INVALID_ARG
    lay2[1].pool = _pool(Hkv=2, k=0x110000, v=0x120000)
    bat2.num_q_heads = 3
    assert L.pcr_pipeline_run_offload(lay2, None, 2, P(bat2), None, None, 0, 0, 0, None, 0, 0x5, 0x6, 0x7,
                                      None) == pcr.PCR_ERR_UNSUPPORTED
    # attention schedule: three values, anything else refused
    assert L.pcr_prefill_attn_set_schedule(3) == pcr.PCR_ERR_INVALID_ARG
    assert L.pcr_prefill_attn_set_schedule(-1) == pcr.PCR_ERR_INVALID_ARG
    for sch in (2, 1, 0):
        assert L.pcr_prefill_attn_set_schedule(sch) == pcr.PCR_OK
    # staged pipeline: streams, workspace and pool shapes are checked before anything is queued
    slot = 2 * 3 * 16 * 2 * 64 * 2        # 3 pairs of (16-token, 2-head, d=64) K and V blocks
    bat2.n_pairs = 3
    assert L.pcr_pipeline_run_staged(None, 0, None, None, 0, None, None, None, None) == pcr.PCR_OK
    assert L.pcr_pipeline_run_staged(lay2, 2, P(bat2), 0x1000, slot, 0x5, 0x5, 0x6, None) == \
        pcr.PCR_ERR_INVALID_ARG and "scatter stream" in pcr.last_error()
    assert L.pcr_pipeline_run_staged(lay2, 2, P(bat2), 0x1000, slot, 0x5, 0x6, 0x6, None) == \
        pcr.PCR_ERR_INVALID_ARG
    assert L.pcr_pipeline_run_staged(lay2, 2, P(bat2), None, slot, 0x5, 0x7, 0x6, None) == \
        pcr.PCR_ERR_INVALID_ARG and "NULL workspace" in pcr.last_error()
    assert L.pcr_pipeline_run_staged(lay2, 2, P(bat2), 0x1008, slot, 0x5, 0x7, 0x6, None) == \
        pcr.PCR_ERR_INVALID_ARG and "aligned" in pcr.last_error()
    assert L.pcr_pipeline_run_staged(lay2, 2, P(bat2), 0x1000, slot - 16, 0x5, 0x7, 0x6, None) == \
        pcr.PCR_ERR_INVALID_ARG and f"needs {slot}" in pcr.last_error()
    lay2[1].pool = _pool(Hkv=1, k=0x110000, v=0x120000)
    assert L.pcr_pipeline_run_staged(lay2, 2, P(bat2), 0x1000, slot, 0x5, 0x7, 0x6, None) == \
        pcr.PCR_ERR_INVALID_ARG and "shape differs" in pcr.last_error()
    lay2[1].pool = _pool(Hkv=2, k=0x110000, v=0x120000)
    # the four-stream form also needs the scatter and offload streams apart
    assert L.pcr_pipeline_run_offload_staged(lay2, None, 2, P(bat2), None, None, 0, 0, None, 0, 0x1000, slot, 0x5,
                                             0x7, 0x6, 0x7, None) == pcr.PCR_ERR_INVALID_ARG
    assert "scatter stream must differ" in pcr.last_error() or "offload stream" in pcr.last_error()
    assert L.pcr_pipeline_run_offload_staged(lay2, None, 2, P(bat2), None, None, 0, 0, None, 0, 0x1000, slot, 0x5,
                                             0x8, 0x6, 0x7, None) == pcr.PCR_ERR_UNSUPPORTED
    # valid workspace: the attention checks come next (three q heads over two kv heads)
    assert L.pcr_pipeline_run_staged(lay2, 2, P(bat2), 0x1000, slot, 0x5, 0x7, 0x6, None) == \
        pcr.PCR_ERR_UNSUPPORTED


@pytest.mark.parametrize("mk", [synth.tiny, synth.l8b_layer, synth.l70b_pipe80])
def test_plan_offload_matches_oracle(mk):
    b = mk()
    for chunk in (16, 64, 256):
        want = odm.plan_offload(b.prefix_lens, b.suffix_lens, b.block_tables, 16, chunk, first_dst_block=3)
        got = pcr.plan_offload(b.prefix_lens, b.suffix_lens, b.block_tables, 16, chunk, first_dst_block=3)
        for w, g in zip(want, got):
            assert np.array_equal(w, g)


def test_plan_offload_on_rag_mix_and_errors():
    from paper_2603_23049_amd import prefix_tree
    b = prefix_tree.rag_mix_batch()
    want = odm.plan_offload(b.prefix_lens, b.suffix_lens, b.block_tables)
    got = pcr.plan_offload(b.prefix_lens, b.suffix_lens, b.block_tables)
    assert all(np.array_equal(w, g) for w, g in zip(want, got)) and len(got[0]) > 0
    with pytest.raises(pcr.PcrError):
        pcr.plan_offload([0], [64], np.array([[0, 1, 2, -1]], np.int32), 16, 64)   # missing pool block
    with pytest.raises(pcr.PcrError):
        pcr.plan_offload([0], [64], np.array([[0, 1, 2, 3]], np.int32), 16, 40)    # chunk not a block multiple
