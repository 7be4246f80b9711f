"""GPU: pool-to-host offload of the computed chunks (Alg. 1 LayerwiseDownload), alone and
as the third stream of the layer pipeline, bit for bit against the oracle.

The host destination is filled with a marker pattern first: listed blocks must hold
exactly the pool blocks after the layer's load + append, every other block must keep
the marker. In the pipeline, each layer's offload must see that layer's finished
append (it runs after the layer's compute), never stale pool bits.
"""
import numpy as np
import pytest
import torch

from paper_2603_23049_amd import pcr, synth
from gpuio import attn_schedule, GpuLayer, pinned, say, u16
from oracle import datamove as odm

pytestmark = pytest.mark.gpu

BS = 16
MARK = np.uint16(0x5A5A)
NAN_BITS = np.uint16(0x7FC1)


def _host_out(b, n_blocks):
    shape = (n_blocks, b.num_kv_heads, BS * b.head_dim)
    return pcr.HostKV(pinned(np.full(shape, MARK, np.uint16)), pinned(np.full(shape, MARK, np.uint16)),
                      b.num_kv_heads, b.head_dim)


def _want(b, data, pk0, pv0, src, dst, n_blocks):
    plan = odm.plan(b.prefix_lens, b.suffix_lens, b.block_tables, b.host_blocks, BS)
    pk, pv = odm.pool_after_layer(pk0, pv0, data.host_k, data.host_v, plan, data.k_new, data.v_new, BS)
    shape = (n_blocks, b.num_kv_heads, BS * b.head_dim)
    hk, hv = np.full(shape, MARK, np.uint16), np.full(shape, MARK, np.uint16)
    odm.offload(pk, pv, hk, hv, src, dst)
    return hk, hv


@pytest.mark.parametrize("method", ["kernel_pull", "dma_per_block", "dma_staged"])
@pytest.mark.parametrize("chunk", [16, 64, 256])
def test_offload_bitexact(method, chunk):
    b = synth.ragged_batch("off", Hq=16, Hkv=4, d=128, prefix_lens=[0, 256, 48, 512], suffix_lens=[300, 256, 500, 40],
                           pool_blocks=160, seed=21)
    data = synth.make_layer(b)
    rng = np.random.Generator(np.random.PCG64(22))
    shape = (b.pool_blocks, b.num_kv_heads, BS * b.head_dim)
    pk0, pv0 = synth.normal_bf16(rng, shape), synth.normal_bf16(rng, shape)
    src, dst = pcr.plan_offload(b.prefix_lens, b.suffix_lens, b.block_tables, BS, chunk, first_dst_block=2)
    assert len(src) > 0
    n_blocks = int(dst.max()) + 3
    say(f"[gpu] offload chunk={chunk} method={method} blocks={len(src)}")
    L = GpuLayer(b, data, pk0, pv0)
    L.run_serial("kernel_pull")
    host = _host_out(b, n_blocks)
    ws = torch.empty(pcr.staged_workspace_bytes(len(src), b.num_kv_heads, b.head_dim), dtype=torch.uint8,
                     device="cuda")
    # reversed host order too: the staged copies then have one run per block
    order = slice(None, None, -1) if chunk == 64 else slice(None)
    pcr.offload_kv_layer(L.pool, src[order], host, dst[order], method=method, workspace=ws)
    torch.cuda.synchronize()
    hk, hv = _want(b, data, pk0, pv0, src, dst, n_blocks)
    assert np.array_equal(u16(host.k), hk)
    assert np.array_equal(u16(host.v), hv)


def test_offload_rejects_pageable_and_bad_ids():
    b = synth.tiny()
    data = synth.make_layer(b)
    shape = (b.pool_blocks, b.num_kv_heads, BS * b.head_dim)
    z = np.zeros(shape, np.uint16)
    L = GpuLayer(b, data, z, z)
    pageable = pcr.HostKV(torch.zeros((4, b.num_kv_heads, BS * b.head_dim), dtype=torch.int16),
                          torch.zeros((4, b.num_kv_heads, BS * b.head_dim), dtype=torch.int16), b.num_kv_heads,
                          b.head_dim)
    with pytest.raises(pcr.PcrError) as e:
        pcr.offload_kv_layer(L.pool, [0], pageable, [0])
    assert e.value.status == pcr.PCR_ERR_NOT_PINNED
    host = _host_out(b, 4)
    with pytest.raises(pcr.PcrError):
        pcr.offload_kv_layer(L.pool, [b.pool_blocks], host, [0])        # src outside the pool
    with pytest.raises(pcr.PcrError):
        pcr.offload_kv_layer(L.pool, [0, 1], host, [2, 2])              # dst named twice
    ws = torch.empty(1024, dtype=torch.uint8, device="cuda")
    with pytest.raises(pcr.PcrError):
        pcr.offload_kv_layer(L.pool, [0, 1], host, [0, 1], method="dma_staged", workspace=ws)   # too small
    with pytest.raises(pcr.PcrError):
        pcr.offload_kv_layer(L.pool, [0], host, [0], method="dma_staged")                       # no workspace
    pcr.offload_kv_layer(L.pool, [], host, [])                          # empty: no-op
    torch.cuda.synchronize()
    assert np.all(u16(host.k) == MARK)


@pytest.mark.parametrize("method", ["kernel_pull", "dma_per_block", "dma_staged"])
def test_pipeline_with_offload_bitwise(method):
    n = 5
    b = synth.uniform_batch("pipe_off", B=2, Hq=32, Hkv=8, d=128, p=1024, s=520, pool_blocks=512, seed=3,
                            num_layers=n, layer_seed_base=3100)
    shape = (b.pool_blocks, b.num_kv_heads, BS * b.head_dim)
    poison = np.full(shape, NAN_BITS, np.uint16)
    layers = [GpuLayer(b, synth.make_layer(b, l), poison, poison) for l in range(n)]
    src, dst = pcr.plan_offload(b.prefix_lens, b.suffix_lens, b.block_tables, BS, 256)
    assert len(src) == 2 * 2 * 16          # chunks 4 and 5 of each sequence
    n_blocks = len(src)
    outs = [_host_out(b, n_blocks) for _ in range(n)]
    say(f"[gpu] pipeline with offload, {n} layers, method={method}")
    load_method = "kernel_pull" if method == "dma_staged" else method
    ws = torch.empty(pcr.staged_workspace_bytes(len(src), b.num_kv_heads, b.head_dim), dtype=torch.uint8,
                     device="cuda")
    serial = []
    for L in layers:
        L.run_serial(load_method)
        serial.append(u16(L.out).copy())
        L.pool.k.copy_(torch.from_numpy(poison.view(np.int16)))
        L.pool.v.copy_(torch.from_numpy(poison.view(np.int16)))
        L.out.zero_()
    torch.cuda.synchronize()
    cs, ks, os_ = torch.cuda.Stream(), torch.cuda.Stream(), torch.cuda.Stream()
    t = pcr.pipeline_run_offload([L.layer_io() for L in layers], outs, layers[0].batch_plan(), src, dst, cs, ks,
                                 os_, method=load_method, offload_method=method, workspace=ws, timing=True)
    torch.cuda.synchronize()
    for l, L in enumerate(layers):
        assert np.array_equal(u16(L.out), serial[l]), f"layer {l}: output differs from serial"
        hk, hv = _want(b, synth.make_layer(b, l), poison, poison, src, dst, n_blocks)
        assert np.array_equal(u16(outs[l].k), hk), f"layer {l}: offloaded K"
        assert np.array_equal(u16(outs[l].v), hv), f"layer {l}: offloaded V"
    assert np.all(t["offload_ms"] > 0) and t["total_ms"] >= t["compute_end_ms"] > 0
    assert np.all(t["offload_end_ms"][1:] >= t["offload_end_ms"][:-1])


@pytest.mark.parametrize("offload_method", ["dma_staged", "kernel_pull"])
def test_pipeline_with_offload_staged_loads_bitwise(offload_method):
    """Four streams: staged loads (transfers, then a scatter on its own stream), compute,
    offload. Pools poisoned with NaN bit patterns, the scatter and offload streams each
    delayed by unrelated device work queued first: outputs equal the serialized ones
    and every offloaded block the oracle's, bit for bit."""
    n = 5
    b = synth.uniform_batch("pipe_off_stg", B=2, Hq=32, Hkv=8, d=128, p=1024, s=520, pool_blocks=512, seed=4,
                            num_layers=n, layer_seed_base=3200)
    shape = (b.pool_blocks, b.num_kv_heads, BS * b.head_dim)
    poison = np.full(shape, NAN_BITS, np.uint16)
    layers = [GpuLayer(b, synth.make_layer(b, l), poison, poison) for l in range(n)]
    src, dst = pcr.plan_offload(b.prefix_lens, b.suffix_lens, b.block_tables, BS, 256)
    n_blocks = len(src)
    outs = [_host_out(b, n_blocks) for _ in range(n)]
    say(f"[gpu] pipeline with staged loads and offload ({offload_method}), {n} layers")
    serial = []
    for L in layers:
        L.run_serial("kernel_pull")
        serial.append(u16(L.out).copy())
        L.pool.k.copy_(torch.from_numpy(poison.view(np.int16)))
        L.pool.v.copy_(torch.from_numpy(poison.view(np.int16)))
        L.out.zero_()
    torch.cuda.synchronize()
    bp = layers[0].batch_plan()
    ows = torch.empty(pcr.staged_workspace_bytes(len(src), b.num_kv_heads, b.head_dim), dtype=torch.uint8,
                      device="cuda")
    lws = torch.empty(2 * pcr.pipeline_staged_slot_bytes(len(bp.src_blocks), b.num_kv_heads, b.head_dim),
                      dtype=torch.uint8, device="cuda")
    cs, ss, ks, os_ = torch.cuda.Stream(), torch.cuda.Stream(), torch.cuda.Stream(), torch.cuda.Stream()
    junk = torch.empty(256 << 20, dtype=torch.uint8, device="cuda")
    for st_ in (ss, os_):
        with torch.cuda.stream(st_):
            junk.fill_(7)
            junk.add_(1)
    t = pcr.pipeline_run_offload_staged([L.layer_io() for L in layers], outs, bp, src, dst, lws, cs, ss, ks, os_,
                                        offload_method=offload_method, offload_workspace=ows, timing=True)
    torch.cuda.synchronize()
    for l, L in enumerate(layers):
        got = u16(L.out)
        assert not np.any((got & 0x7F80) == 0x7F80), f"layer {l}: non-finite output (missing wait)"
        assert np.array_equal(got, serial[l]), f"layer {l}: output differs from serial"
        hk, hv = _want(b, synth.make_layer(b, l), poison, poison, src, dst, n_blocks)
        assert np.array_equal(u16(outs[l].k), hk), f"layer {l}: offloaded K"
        assert np.array_equal(u16(outs[l].v), hv), f"layer {l}: offloaded V"
    assert np.all(t["offload_ms"] > 0) and np.all(t["load_ms"] > 0) and t["total_ms"] >= t["compute_end_ms"] > 0


def test_staged_load_bitexact():
    b = synth.ragged_batch("ld", Hq=16, Hkv=4, d=128, prefix_lens=[512, 48, 0, 300], suffix_lens=[10, 20, 30, 1],
                           pool_blocks=100, seed=23)
    data = synth.make_layer(b)
    rng = np.random.Generator(np.random.PCG64(24))
    shape = (b.pool_blocks, b.num_kv_heads, BS * b.head_dim)
    pk0, pv0 = synth.normal_bf16(rng, shape), synth.normal_bf16(rng, shape)
    L = GpuLayer(b, data, pk0, pv0)
    ws = torch.empty(pcr.staged_workspace_bytes(len(L.src), b.num_kv_heads, b.head_dim), dtype=torch.uint8,
                     device="cuda")
    say(f"[gpu] staged load, {len(L.src)} blocks")
    pcr.load_kv_layer(L.host, L.src, L.pool, L.dst, method="dma_staged", workspace=ws)
    torch.cuda.synchronize()
    pk, pv = pk0.copy(), pv0.copy()
    odm.load(pk, pv, data.host_k, data.host_v, L.src, L.dst)
    assert np.array_equal(u16(L.pool.k), pk) and np.array_equal(u16(L.pool.v), pv)


@pytest.mark.parametrize("method", ["dma_staged", "kernel_pull"])
def test_pipeline_with_offload_full_size(method):
    """The benchmark's three-stream pipeline at full size: 32 layers of 4 sequences x
    (4096 cached + 6144 new tokens), loads by the pull kernel, the computed whole
    256-token chunks offloaded (96 MiB per layer) staged or by the push kernel; four
    distinct layer data sets used round-robin, every layer with its own pool (poisoned
    with NaN bit patterns), output and marker-filled host destination. Every layer's
    offloaded blocks equal the oracle's bit for bit (unlisted blocks keep the marker)
    and every output equals its data set's serialized result."""
    b = synth.l8b_pipe32(6144)
    n, distinct = b.num_layers, 4
    shape = (b.pool_blocks, b.num_kv_heads, BS * b.head_dim)
    poison = np.full(shape, NAN_BITS, np.uint16)
    src, dst = pcr.plan_offload(b.prefix_lens, b.suffix_lens, b.block_tables, BS, 256)
    n_blocks = len(src)
    assert n_blocks * BS * b.num_kv_heads * b.head_dim * 2 * 2 == 96 << 20
    say(f"[gpu] pipeline with offload {b.name}: {n} layers, offload {method}")
    base = [GpuLayer(b, synth.make_layer(b, l), poison, poison) for l in range(distinct)]
    serial = []
    for L in base:
        with attn_schedule("key_halves"):   # the pull-load pipeline's attention schedule
            L.run_serial("kernel_pull")
        serial.append(L.out.clone())
        L.pool.k.fill_(int(NAN_BITS))
        L.pool.v.fill_(int(NAN_BITS))
        L.out.zero_()
    ios = [L.layer_io() for L in base]
    for l in range(distinct, n):
        s_ = base[l % distinct]
        pool = pcr.KVPool(torch.full(shape, int(NAN_BITS), dtype=torch.int16, device="cuda"),
                          torch.full(shape, int(NAN_BITS), dtype=torch.int16, device="cuda"), b.num_kv_heads,
                          b.head_dim)
        ios.append(pcr.Layer(s_.host, pool, s_.q, s_.k_new, s_.v_new, torch.zeros_like(s_.out)))
    outs = [_host_out(b, n_blocks) for _ in range(n)]
    ws = torch.empty(pcr.staged_workspace_bytes(n_blocks, b.num_kv_heads, b.head_dim), dtype=torch.uint8,
                     device="cuda")
    torch.cuda.synchronize()
    cs, ks, os_ = torch.cuda.Stream(), torch.cuda.Stream(), torch.cuda.Stream()
    pcr.pipeline_run_offload(ios, outs, base[0].batch_plan(), src, dst, cs, ks, os_, method="kernel_pull",
                             offload_method=method, workspace=ws)
    torch.cuda.synchronize()
    for k in range(distinct):
        hk, hv = _want(b, synth.make_layer(b, k), poison, poison, src, dst, n_blocks)
        for l in range(k, n, distinct):
            assert torch.equal(ios[l].out, serial[k]), f"layer {l}: output differs from serial"
            assert np.array_equal(u16(outs[l].k), hk), f"layer {l}: offloaded K"
            assert np.array_equal(u16(outs[l].v), hv), f"layer {l}: offloaded V"
