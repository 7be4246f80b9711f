"""GPU: load, append and gather through the C ABI are bit-exact against the oracle."""
import numpy as np
import pytest
import torch

from oracle import datamove as odm
from paper_2603_23049_amd import pcr, synth
from gpuio import GpuLayer, dev, say, u16

pytestmark = pytest.mark.gpu

BS = 16


def _batch(prefix_lens, suffix_lens, d=64, Hkv=2, pool=64, seed=3):
    return synth.ragged_batch("t", Hq=Hkv * 2, Hkv=Hkv, d=d, prefix_lens=prefix_lens, suffix_lens=suffix_lens,
                              pool_blocks=pool, seed=seed)


def _canary_pools(b, seed=99):
    rng = np.random.Generator(np.random.PCG64(seed))
    shape = (b.pool_blocks, b.num_kv_heads, BS * b.head_dim)
    return synth.normal_bf16(rng, shape), synth.normal_bf16(rng, shape)


def _methods():
    ms = ["dma_per_block", "kernel_pull"]
    return ms


CASES = [
    ("tiny", lambda: synth.tiny()),
    ("l8b_layer", lambda: synth.l8b_layer()),
    ("ragged_partial", lambda: _batch([15, 1, 48, 0, 300], [1, 40, 16, 7, 33], d=128, Hkv=8, pool=64)),
    ("ragged_d64", lambda: _batch([17, 256], [63, 64], d=64, Hkv=2, pool=64)),
]


@pytest.mark.parametrize("name,mk", CASES)
@pytest.mark.parametrize("method", ["dma_per_block", "kernel_pull"])
def test_load_then_append_bitexact(name, mk, method):
    b = mk()
    data = synth.make_layer(b)
    pk0, pv0 = _canary_pools(b)
    say(f"[gpu] load+append {name} method={method} B={b.B} T={b.T}")
    L = GpuLayer(b, data, pk0, pv0)
    L.load(method)
    torch.cuda.synchronize()
    plan = odm.plan(b.prefix_lens, b.suffix_lens, b.block_tables, b.host_blocks, BS)
    want_k, want_v = pk0.copy(), pv0.copy()
    odm.load(want_k, want_v, data.host_k, data.host_v, plan[0], plan[1])
    assert np.array_equal(u16(L.pool.k), want_k) and np.array_equal(u16(L.pool.v), want_v)
    L.append()
    torch.cuda.synchronize()
    odm.append(want_k, want_v, data.k_new, data.v_new, plan[2], BS)
    assert np.array_equal(u16(L.pool.k), want_k), "K pool differs after append"
    assert np.array_equal(u16(L.pool.v), want_v), "V pool differs after append"


def test_load_dma_batch_bitexact_or_unsupported():
    """The batched-copy method is bit-exact where the process's HIP runtime has
    hipMemcpyBatchAsync; where it has not (the runtime bundled with this PyTorch), the
    call fails with PCR_ERR_UNSUPPORTED, names the missing call, and queues nothing:
    the pool still holds its canary bytes."""
    b = synth.tiny()
    data = synth.make_layer(b)
    pk0, pv0 = _canary_pools(b)
    say("[gpu] load dma_batch tiny")
    L = GpuLayer(b, data, pk0, pv0)
    want_k, want_v = pk0.copy(), pv0.copy()
    try:
        L.load("dma_batch")
    except pcr.PcrError as e:
        assert e.status == pcr.PCR_ERR_UNSUPPORTED
        assert "hipMemcpyBatchAsync" in str(e)
        torch.cuda.synchronize()
        assert np.array_equal(u16(L.pool.k), want_k) and np.array_equal(u16(L.pool.v), want_v), \
            "a refused batched load changed the pool"
        return
    torch.cuda.synchronize()
    odm.load(want_k, want_v, data.host_k, data.host_v, L.src, L.dst)
    assert np.array_equal(u16(L.pool.k), want_k) and np.array_equal(u16(L.pool.v), want_v)


def test_load_rejects_pageable_host_memory():
    b = synth.tiny()
    data = synth.make_layer(b)
    pk0, pv0 = _canary_pools(b)
    L = GpuLayer(b, data, pk0, pv0)
    pageable = pcr.HostKV(torch.from_numpy(data.host_k.view(np.int16)), torch.from_numpy(data.host_v.view(np.int16)),
                          b.num_kv_heads, b.head_dim)
    with pytest.raises(pcr.PcrError) as ei:
        pcr.load_kv_layer(pageable, L.src, L.pool, L.dst)
    assert ei.value.status == pcr.PCR_ERR_NOT_PINNED


@pytest.mark.parametrize("d", [64, 128])
def test_gather_bitexact(d):
    b = _batch([0, 33, 100], [20, 40, 3], d=d, Hkv=4, pool=64, seed=8)
    data = synth.make_layer(b)
    pk0, pv0 = _canary_pools(b)
    say(f"[gpu] gather d={d}")
    L = GpuLayer(b, data, pk0, pv0)
    starts = np.array([0, 5, 90], np.int32)
    lens = np.array([20, 68, 13], np.int32)
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    total = int(cu[-1])
    k_out = torch.zeros((total, b.num_kv_heads, d), dtype=torch.int16, device="cuda")
    v_out = torch.zeros_like(k_out)
    pcr.gather_kv(L.pool, L.bt, dev(starts), dev(cu), total, k_out, v_out)
    torch.cuda.synchronize()
    wk, wv = odm.gather(pk0, pv0, b.block_tables, starts, lens, d, BS)
    assert np.array_equal(u16(k_out), wk) and np.array_equal(u16(v_out), wv)


@pytest.mark.parametrize("layout", ["block_order", "ragged_300"])
def test_append_sweep_size_bitexact(layout):
    """The append sweep's largest size: 131072 new tokens (8 kv heads, d = 128: 512 MiB
    of K+V read and written), either in block order over a random order of the pool's
    blocks, or as sequences of 300 tokens each starting at a block of its own, so that
    the kernel's tiles start inside the sequences' 8-slot V chunks. The whole pool
    (canaries in every slot the list does not name) equals the oracle's bit for bit."""
    T, Hkv, d = 131072, 8, 128
    rng = np.random.Generator(np.random.PCG64(131 + len(layout)))
    t = np.arange(T, dtype=np.int64)
    if layout == "block_order":
        nb = -(-T // BS)
        blocks = rng.permutation(nb).astype(np.int64)
        slots = blocks[t // BS] * BS + t % BS
    else:
        seq, per_seq = 300, -(-300 // BS)
        nb = -(-T // seq) * per_seq
        blocks = rng.permutation(nb).astype(np.int64)
        pos = t % seq
        slots = blocks[(t // seq) * per_seq + pos // BS] * BS + pos % BS
    slots = slots.astype(np.int32)
    shape = (nb, Hkv, BS * d)
    pk0, pv0 = synth.normal_bf16(rng, shape), synth.normal_bf16(rng, shape)
    k_new, v_new = synth.normal_bf16(rng, (T, Hkv, d)), synth.normal_bf16(rng, (T, Hkv, d))
    say(f"[gpu] append sweep size {layout}: T={T} blocks={nb}")
    pool = pcr.KVPool(dev(pk0), dev(pv0), Hkv, d)
    pcr.append_kv(pool, dev(k_new), dev(v_new), dev(slots))
    torch.cuda.synchronize()
    want_k, want_v = pk0.copy(), pv0.copy()
    odm.append(want_k, want_v, k_new, v_new, slots, BS)
    assert np.array_equal(u16(pool.k), want_k), "K pool differs after append"
    assert np.array_equal(u16(pool.v), want_v), "V pool differs after append"


def test_append_empty_and_load_empty_are_noops():
    b = synth.tiny()
    data = synth.make_layer(b)
    pk0, pv0 = _canary_pools(b)
    L = GpuLayer(b, data, pk0, pv0)
    pcr.append_kv(L.pool, L.k_new[:0], L.v_new[:0], L.slots[:0])
    pcr.load_kv_layer(L.host, L.src[:0], L.pool, L.dst[:0])
    torch.cuda.synchronize()
    assert np.array_equal(u16(L.pool.k), pk0) and np.array_equal(u16(L.pool.v), pv0)
