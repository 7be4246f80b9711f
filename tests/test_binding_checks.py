"""CPU tests of the Python binding's length checks: the library reads device arrays by
the lengths it is given and cannot see the allocations, so the binding refuses a tensor
shorter than what the call would read, before anything reaches the library. Numpy
arrays stand in for the device tensors (no call is made)."""
import numpy as np
import pytest

from paper_2603_23049_amd import pcr

Hkv, d, Hq, BS = 2, 64, 4, 16


def _pool(blocks=8):
    z = np.zeros((blocks, Hkv, BS * d), np.int16)
    return pcr.KVPool(z, z.copy(), Hkv, d)


def _i32(n):
    return np.zeros(n, np.int32)


def test_append_refuses_short_slot_mapping_and_rows():
    pool = _pool()
    T = 5
    kv = np.zeros((T, Hkv, d), np.int16)
    with pytest.raises(ValueError, match="slot_mapping"):
        pcr.append_kv(pool, kv, kv, _i32(T - 1))
    with pytest.raises(ValueError, match="v_new"):
        pcr.append_kv(pool, kv, kv[:T - 1], _i32(T))


def test_attention_refuses_short_q_out_and_tables():
    pool = _pool()
    hpl, hcu = np.array([16, 0], np.int32), np.array([0, 3, 7], np.int32)   # T = 7
    q = np.zeros((7, Hq, d), np.int16)
    bt = np.zeros((2, 4), np.int32)
    args = dict(block_tables=bt, prefix_lens=_i32(2), cu_suffix=_i32(3), host_prefix_lens=hpl,
                host_cu_suffix=hcu, num_q_heads=Hq)
    with pytest.raises(ValueError, match="q holds"):
        pcr.prefix_prefill_attn(q[:6], pool, out=q, **args)
    with pytest.raises(ValueError, match="out holds"):
        pcr.prefix_prefill_attn(q, pool, out=q[:6], **args)
    with pytest.raises(ValueError, match="block_tables"):
        pcr.prefix_prefill_attn(q, pool, out=q, **{**args, "block_tables": bt[:1]})
    with pytest.raises(ValueError, match="cu_suffix"):
        pcr.prefix_prefill_attn(q, pool, out=q, **{**args, "cu_suffix": _i32(2)})


@pytest.mark.parametrize("fn", [pcr.decode_attn, pcr.decode_attn_noalloc])
def test_decode_refuses_short_lengths_and_rows(fn):
    pool = _pool()
    B = 3
    q = np.zeros((B, Hq, d), np.int16)
    bt = np.zeros((B, 4), np.int32)
    hcl = np.array([5, 9, 17], np.int32)
    with pytest.raises(ValueError, match="context_lens"):
        fn(q, pool, bt, _i32(B - 1), hcl, Hq, q)
    with pytest.raises(ValueError, match="out holds"):
        fn(q, pool, bt, _i32(B), hcl, Hq, q[:B - 1])


def test_gather_refuses_short_outputs():
    pool = _pool()
    kv = np.zeros((10, Hkv, d), np.int16)
    with pytest.raises(ValueError, match="k_out"):
        pcr.gather_kv(pool, np.zeros((2, 4), np.int32), _i32(2), _i32(3), 11, kv, kv)


def test_pipeline_refuses_short_layer_tensors_and_batch():
    pool = _pool()
    hcu = np.array([0, 4], np.int32)
    bp = pcr.BatchPlan(_i32(0), _i32(0), _i32(4), np.zeros((1, 4), np.int32), _i32(1), _i32(2),
                       np.array([16], np.int32), hcu, Hq, 0.125)
    host = pcr.HostKV(np.zeros((4, Hkv, BS * d), np.int16), np.zeros((4, Hkv, BS * d), np.int16), Hkv, d)
    q = np.zeros((4, Hq, d), np.int16)
    kv = np.zeros((4, Hkv, d), np.int16)
    good = pcr.Layer(host, pool, q, kv, kv, q)
    pcr._layers_io([good], bp)          # lengths match: accepted
    with pytest.raises(ValueError, match="layer 1 k_new"):
        pcr._layers_io([good, pcr.Layer(host, _pool(), q, kv[:3], kv, q)], bp)
    short = pcr.BatchPlan(_i32(0), _i32(0), _i32(3), np.zeros((1, 4), np.int32), _i32(1), _i32(2),
                          np.array([16], np.int32), hcu, Hq, 0.125)
    with pytest.raises(ValueError, match="slot_mapping"):
        short.c()
