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
