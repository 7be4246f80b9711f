"""GPU: the two-stream layer pipeline gives, per layer, exactly the serialized result.

The pool of every layer is poisoned with NaN bit patterns before the pipeline
runs: if any layer's compute started before its load landed, NaNs (or other
wrong bits) reach its output. A large dummy copy queued ahead of the loads
delays them, which must not change a single bit either.
"""
import numpy as np
import pytest
import torch

from paper_2603_23049_amd import pcr, synth
from gpuio import GpuLayer, MAX_ABS, MEAN_ABS, error_stats, pinned, say, u16
from oracle import attention as oattn
from oracle import datamove as odm

pytestmark = pytest.mark.gpu

BS = 16
NAN_BITS = np.uint16(0x7FC1)


def _layers(b, n):
    shape = (b.pool_blocks, b.num_kv_heads, BS * b.head_dim)
    poison = np.full(shape, NAN_BITS, np.uint16)
    return [GpuLayer(b, synth.make_layer(b, l), poison, poison) for l in range(n)], poison


@pytest.mark.parametrize("method", ["kernel_pull", "dma_per_block"])
def test_pipeline_equals_serial_bitwise(method):
    base = synth.l8b_pipe32()
    n = 6
    b = synth.uniform_batch("pipe", B=2, Hq=32, Hkv=8, d=128, p=1024, s=200, pool_blocks=512, seed=3,
                            num_layers=n, layer_seed_base=3000)
    assert base.num_kv_heads == b.num_kv_heads
    say(f"[gpu] pipeline {n} layers method={method}")
    layers, poison = _layers(b, n)
    serial = []
    for L in layers:
        L.run_serial(method)
        serial.append(u16(L.out).copy())
        L.pool.k.copy_(torch.from_numpy(poison.view(np.int16)))
        L.pool.v.copy_(torch.from_numpy(poison.view(np.int16)))
        L.out.zero_()
    torch.cuda.synchronize()
    copy_s, comp_s = torch.cuda.Stream(), torch.cuda.Stream()
    # delay the copy stream with a large unrelated host-to-device copy
    big_h = pinned(np.ones(64 << 20, np.uint8))
    big_d = torch.empty(64 << 20, dtype=torch.uint8, device="cuda")
    with torch.cuda.stream(copy_s):
        big_d.copy_(big_h, non_blocking=True)
    timing = pcr.pipeline_run([L.layer_io() for L in layers], layers[0].batch_plan(), copy_s, comp_s,
                              method=method, timing=True)
    torch.cuda.synchronize()
    for l, L in enumerate(layers):
        got = u16(L.out)
        assert not np.any((got & 0x7F80) == 0x7F80), f"layer {l}: non-finite output (missing wait)"
        assert np.array_equal(got, serial[l]), f"layer {l}: pipeline differs from serial"
    assert timing["total_ms"] > 0 and np.all(timing["load_ms"] > 0) and np.all(timing["compute_ms"] > 0)
    assert abs(timing["sum_compute_ms"] - float(timing["compute_ms"].sum())) < 1e-3
    # layer 0 against the oracle
    L = layers[0]
    data = synth.make_layer(b, 0)
    plan = odm.plan(b.prefix_lens, b.suffix_lens, b.block_tables, b.host_blocks, BS)
    pk, pv = odm.pool_after_layer(poison, poison, data.host_k, data.host_v, plan, data.k_new, data.v_new, BS)
    rows = np.array([[t, h] for t in range(0, b.T, 23) for h in range(0, 32, 5)], np.int32)
    want = oattn.attention(data.q, pk, pv, b.block_tables, np.asarray(b.prefix_lens, np.int32), plan[3], 8, BS,
                           rows=rows)
    got = synth.bf16_bits_to_f32(serial[0]).astype(np.float64)[rows[:, 0], rows[:, 1]]
    mx, mean = error_stats(got, want)
    assert mx <= MAX_ABS and mean <= MEAN_ABS


def test_pipeline_partial_prefix_block_ordering():
    """p % 16 != 0: the last cached block is loaded whole and then partly
    overwritten by the append; the pipeline must keep that order per layer."""
    n = 4
    b = synth.ragged_batch("partial", Hq=8, Hkv=2, d=64, prefix_lens=[37, 250], suffix_lens=[30, 9],
                           pool_blocks=40, seed=31)
    b.num_layers = n
    layers, poison = _layers(b, n)
    serial = []
    for L in layers:
        L.run_serial("kernel_pull")
        serial.append(u16(L.out).copy())
        L.pool.k.copy_(torch.from_numpy(poison.view(np.int16)))
        L.pool.v.copy_(torch.from_numpy(poison.view(np.int16)))
        L.out.zero_()
    copy_s, comp_s = torch.cuda.Stream(), torch.cuda.Stream()
    say("[gpu] pipeline partial-block ordering")
    pcr.pipeline_run([L.layer_io() for L in layers], layers[0].batch_plan(), copy_s, comp_s, method="kernel_pull")
    torch.cuda.synchronize()
    for l, L in enumerate(layers):
        assert np.array_equal(u16(L.out), serial[l]), f"layer {l}"


@pytest.mark.parametrize("mk", [synth.l8b_pipe32, synth.l70b_pipe80, lambda: synth.l8b_pipe32(6144)],
                         ids=["l8b_pipe32", "l70b_pipe80", "l8b_pipe32_s6144"])
def test_pipeline_full_size(mk):
    """The benchmark's pipelines in their launch configuration: the 32-layer
    Llama-3-8B-shaped one (4 sequences, 4096 cached + 256 new tokens), the 80-layer
    70B-shaped one (2 x 15360 + 1024) and the compute-bound 32-layer one (4 x 4096 +
    6144); method "auto", four distinct layer data sets used round-robin, every layer
    with its own pool and output, all pools poisoned with NaN bit patterns beforehand.
    Every layer's pool after the pipeline is the oracle's bit for bit, every output
    equals its data set's serialized result bit for bit, and sampled rows of the first
    and last layer match the fp64 oracle."""
    b = mk()
    n, distinct = b.num_layers, 4
    shape = (b.pool_blocks, b.num_kv_heads, BS * b.head_dim)
    poison = np.full(shape, NAN_BITS, np.uint16)
    say(f"[gpu] pipeline {b.name}: {n} layers, {distinct} distinct data sets")
    base = [GpuLayer(b, synth.make_layer(b, l), poison, poison) for l in range(distinct)]
    serial = []
    for L in base:
        L.run_serial("auto")
        serial.append(L.out.clone())
        L.pool.k.fill_(int(NAN_BITS))
        L.pool.v.fill_(int(NAN_BITS))
        L.out.zero_()
    ios = [L.layer_io() for L in base]
    for l in range(distinct, n):
        src = base[l % distinct]
        pool = pcr.KVPool(torch.full(shape, int(NAN_BITS), dtype=torch.int16, device="cuda"),
                          torch.full(shape, int(NAN_BITS), dtype=torch.int16, device="cuda"), b.num_kv_heads,
                          b.head_dim)
        ios.append(pcr.Layer(src.host, pool, src.q, src.k_new, src.v_new, torch.zeros_like(src.out)))
    torch.cuda.synchronize()
    copy_s, comp_s = torch.cuda.Stream(), torch.cuda.Stream()
    pcr.pipeline_run(ios, base[0].batch_plan(), copy_s, comp_s, method="auto")
    torch.cuda.synchronize()
    plan = odm.plan(b.prefix_lens, b.suffix_lens, b.block_tables, b.host_blocks, BS)
    for k in range(distinct):
        data = synth.make_layer(b, k)
        pk, pv = odm.pool_after_layer(poison, poison, data.host_k, data.host_v, plan, data.k_new, data.v_new, BS)
        pk_d = torch.from_numpy(pk.view(np.int16)).cuda()
        pv_d = torch.from_numpy(pv.view(np.int16)).cuda()
        for l in range(k, n, distinct):
            io = ios[l]
            assert torch.equal(io.pool.k, pk_d) and torch.equal(io.pool.v, pv_d), f"layer {l}: pool differs"
            assert torch.equal(io.out, serial[k]), f"layer {l}: pipeline output differs from serial"
        if k in (0, (n - 1) % distinct):
            l = k if k == 0 else n - 1
            T = b.T
            toks = sorted(set([0, 1, T // 2, T - 2, T - 1] + list(range(5, T, max(1, T // 24)))))
            rows = np.array([[t, h] for t in toks for h in range(0, b.num_q_heads, 3)], np.int32)
            want = oattn.attention(data.q, pk, pv, b.block_tables, np.asarray(b.prefix_lens, np.int32), plan[3],
                                   b.num_kv_heads, BS, rows=rows)
            got = synth.bf16_bits_to_f32(u16(ios[l].out)).astype(np.float64)[rows[:, 0], rows[:, 1]]
            mx, mean = error_stats(got, want)
            say(f"    layer {l}: max_abs={mx:.3e} mean_abs={mean:.3e}")
            assert mx <= MAX_ABS and mean <= MEAN_ABS
        del pk_d, pv_d
