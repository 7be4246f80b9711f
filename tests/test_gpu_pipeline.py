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
from gpuio import GpuLayer, MAX_ABS, MEAN_ABS, attn_schedule, error_stats, pinned, say, u16
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


@pytest.mark.parametrize("slots", [1, 2, 3, 9])
def test_staged_pipeline_equals_serial_bitwise(slots):
    """Loads as copy-engine transfers into workspace slots and a scatter on a third
    stream: with one slot every transfer waits for the previous scatter, with more the
    transfers run ahead (9 slots for 6 layers: each layer its own). Pools poisoned with
    NaN bit patterns, the copy and the scatter streams each delayed by a large unrelated
    copy queued first: every output must equal the serialized one bit for bit."""
    n = 6
    b = synth.uniform_batch("pipe", B=2, Hq=32, Hkv=8, d=128, p=1024, s=200, pool_blocks=512, seed=3,
                            num_layers=n, layer_seed_base=3000)
    say(f"[gpu] staged pipeline {n} layers, {slots} workspace slots")
    layers, poison = _layers(b, n)
    serial = []
    for L in layers:
        L.run_serial("kernel_pull")
        serial.append(u16(L.out).copy())
        L.pool.k.copy_(torch.from_numpy(poison.view(np.int16)))
        L.pool.v.copy_(torch.from_numpy(poison.view(np.int16)))
        L.out.zero_()
    torch.cuda.synchronize()
    bp = layers[0].batch_plan()
    slot = pcr.pipeline_staged_slot_bytes(len(bp.src_blocks), b.num_kv_heads, b.head_dim)
    ws = torch.empty(slots * slot + 8, dtype=torch.uint8, device="cuda")   # a partial slot beyond is unused
    copy_s, scat_s, comp_s = torch.cuda.Stream(), torch.cuda.Stream(), torch.cuda.Stream()
    big_h = pinned(np.ones(64 << 20, np.uint8))
    big_d = torch.empty(64 << 20, dtype=torch.uint8, device="cuda")
    big_d2 = torch.empty(256 << 20, dtype=torch.uint8, device="cuda")
    with torch.cuda.stream(copy_s):
        big_d.copy_(big_h, non_blocking=True)
    with torch.cuda.stream(scat_s):
        big_d2.fill_(3)
        big_d2.add_(1)
    timing = pcr.pipeline_run_staged([L.layer_io() for L in layers], bp, ws, copy_s, scat_s, comp_s, timing=True)
    torch.cuda.synchronize()
    for l, L in enumerate(layers):
        got = u16(L.out)
        assert not np.any((got & 0x7F80) == 0x7F80), f"layer {l}: non-finite output (missing wait)"
        assert np.array_equal(got, serial[l]), f"layer {l}: staged pipeline differs from serial"
    assert timing["total_ms"] > 0 and np.all(timing["load_ms"] > 0) and np.all(timing["compute_ms"] > 0)


def test_staged_pipeline_twice_on_one_workspace():
    """Two staged pipelines queued back to back on the same workspace and streams, the
    second over other layers: the second call's first transfers wait for the first
    call's scatters (which read the slots), so both give the serialized outputs."""
    n = 4
    b = synth.uniform_batch("pipe2", B=2, Hq=16, Hkv=4, d=128, p=700, s=90, pool_blocks=160, seed=5,
                            num_layers=2 * n, layer_seed_base=5000)
    layers, poison = _layers(b, 2 * n)
    serial = []
    for L in layers:
        L.run_serial("kernel_pull")
        serial.append(u16(L.out).copy())
        L.pool.k.copy_(torch.from_numpy(poison.view(np.int16)))
        L.pool.v.copy_(torch.from_numpy(poison.view(np.int16)))
        L.out.zero_()
    torch.cuda.synchronize()
    bp = layers[0].batch_plan()
    ws = torch.empty(pcr.pipeline_staged_slot_bytes(len(bp.src_blocks), b.num_kv_heads, b.head_dim) * 2,
                     dtype=torch.uint8, device="cuda")
    copy_s, scat_s, comp_s = torch.cuda.Stream(), torch.cuda.Stream(), torch.cuda.Stream()
    say("[gpu] two staged pipelines on one workspace")
    pcr.pipeline_run_staged([L.layer_io() for L in layers[:n]], bp, ws, copy_s, scat_s, comp_s)
    pcr.pipeline_run_staged([L.layer_io() for L in layers[n:]], bp, ws, copy_s, scat_s, comp_s)
    torch.cuda.synchronize()
    for l, L in enumerate(layers):
        assert np.array_equal(u16(L.out), serial[l]), f"layer {l}"


def test_staged_pipeline_without_cached_blocks_and_one_layer():
    """No cached prefix (nothing to load): the staged form needs no workspace and still
    runs every layer's append and attention; and a one-layer staged pipeline."""
    for p_len, n, need_ws in ((0, 3, False), (300, 1, True)):
        b = synth.uniform_batch("pipe_edge", B=2, Hq=8, Hkv=2, d=64, p=p_len, s=77, pool_blocks=64, seed=7,
                                num_layers=n, layer_seed_base=7000)
        layers, poison = _layers(b, n)
        serial = []
        for L in layers:
            L.run_serial("kernel_pull")
            serial.append(u16(L.out).copy())
            L.pool.k.copy_(torch.from_numpy(poison.view(np.int16)))
            L.pool.v.copy_(torch.from_numpy(poison.view(np.int16)))
            L.out.zero_()
        torch.cuda.synchronize()
        bp = layers[0].batch_plan()
        assert (len(bp.src_blocks) > 0) == need_ws
        ws = None
        if need_ws:
            ws = torch.empty(pcr.pipeline_staged_slot_bytes(len(bp.src_blocks), b.num_kv_heads, b.head_dim),
                             dtype=torch.uint8, device="cuda")
        copy_s, scat_s, comp_s = torch.cuda.Stream(), torch.cuda.Stream(), torch.cuda.Stream()
        say(f"[gpu] staged pipeline, prefix {p_len}, {n} layer(s)")
        pcr.pipeline_run_staged([L.layer_io() for L in layers], bp, ws, copy_s, scat_s, comp_s)
        torch.cuda.synchronize()
        for l, L in enumerate(layers):
            assert np.array_equal(u16(L.out), serial[l]), f"prefix {p_len} layer {l}"


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


# The benchmark's pipelines in their launch configuration, with the number of distinct
# generated layer data sets the benchmark uses (every layer has its own pool and output
# either way): all 32 layers of the Llama-3-8B stack distinct; 6 sets round-robin for the
# 80-layer 70B-shaped stack and the compute-bound 32-layer one (the first, middle and
# last layers then all differ).
FULL = {"l8b_pipe32": (synth.l8b_pipe32, 32), "l70b_pipe80": (synth.l70b_pipe80, 6),
        "l8b_pipe32_s6144": (lambda: synth.l8b_pipe32(6144), 6)}
_FULL_RESULTS = {}


def _special_layers(n):
    return (0, n // 2, n - 1)


def _full_pipeline(name):
    """Runs the named pipeline once per test session with method "auto", then again with
    staged loads (every pool poisoned with NaN bit patterns before each run; the
    pull-load pipeline's attention takes key halves, the staged one's the default
    schedule, row halves at the 70B and compute-bound shapes) and checks, for every layer, that its pool is the
    oracle's bit for bit and its output equals its data set's serialized result bit for
    bit. Keeps, for the first, middle and last layers, the staged run's output and the
    oracle's inputs."""
    if name in _FULL_RESULTS:
        return _FULL_RESULTS[name]
    mk, distinct = FULL[name]
    b = mk()
    n = b.num_layers
    sets = synth.pipeline_data_sets(n, distinct)
    n_sets = max(sets) + 1
    shape = (b.pool_blocks, b.num_kv_heads, BS * b.head_dim)
    poison = np.full(shape, NAN_BITS, np.uint16)
    say(f"[gpu] pipeline {b.name}: {n} layers, {n_sets} distinct data sets (generating)")
    datas = synth.make_layers(b, range(n_sets))
    base = [GpuLayer(b, datas[k], poison, poison) for k in range(n_sets)]
    # serial references: under key halves for the pull-load pipeline (which takes them),
    # under the default schedule for the staged one
    serial = {"auto": [], "staged": []}
    for L in base:
        for form, sched in (("auto", "key_halves"), ("staged", "auto")):
            with attn_schedule(sched):
                L.run_serial("auto")
            serial[form].append(L.out.clone())
            L.pool.k.fill_(int(NAN_BITS))
            L.pool.v.fill_(int(NAN_BITS))
            L.out.zero_()
    ios = [L.layer_io() for L in base]
    for l in range(n_sets, n):
        src = base[sets[l]]
        pool = pcr.KVPool(torch.full(shape, int(NAN_BITS), dtype=torch.int16, device="cuda"),
                          torch.full(shape, int(NAN_BITS), dtype=torch.int16, device="cuda"), b.num_kv_heads,
                          b.head_dim)
        ios.append(pcr.Layer(src.host, pool, src.q, src.k_new, src.v_new, torch.zeros_like(src.out)))
    torch.cuda.synchronize()
    plan = odm.plan(b.prefix_lens, b.suffix_lens, b.block_tables, b.host_blocks, BS)
    special = _special_layers(n)
    keep = {}
    oracle_pools = [None] * n_sets
    bp = base[0].batch_plan()
    copy_s, scat_s, comp_s = torch.cuda.Stream(), torch.cuda.Stream(), torch.cuda.Stream()
    ws = torch.empty(2 * pcr.pipeline_staged_slot_bytes(len(bp.src_blocks), b.num_kv_heads, b.head_dim),
                     dtype=torch.uint8, device="cuda")
    for form in ("auto", "staged"):
        say(f"    running the pipeline ({form} loads)")
        if form == "auto":
            pcr.pipeline_run(ios, bp, copy_s, comp_s, method="auto")
        else:
            for io in ios:
                io.pool.k.fill_(int(NAN_BITS))
                io.pool.v.fill_(int(NAN_BITS))
                io.out.zero_()
            torch.cuda.synchronize()
            pcr.pipeline_run_staged(ios, bp, ws, copy_s, scat_s, comp_s)
        torch.cuda.synchronize()
        for k in range(n_sets):
            data = datas[k]
            if oracle_pools[k] is None:
                oracle_pools[k] = odm.pool_after_layer(poison, poison, data.host_k, data.host_v, plan, data.k_new,
                                                       data.v_new, BS)
            pk, pv = oracle_pools[k]
            pk_d = torch.from_numpy(pk.view(np.int16)).cuda()
            pv_d = torch.from_numpy(pv.view(np.int16)).cuda()
            for l in range(n):
                if sets[l] != k:
                    continue
                io = ios[l]
                assert torch.equal(io.pool.k, pk_d) and torch.equal(io.pool.v, pv_d), \
                    f"layer {l}: pool differs ({form})"
                assert torch.equal(io.out, serial[form][k]), f"layer {l}: pipeline output differs from serial ({form})"
                if l in special and form == "staged":
                    keep[l] = {"out": u16(io.out), "q": data.q, "pk": pk, "pv": pv}
            del pk_d, pv_d
        say(f"    every layer's pool equals the oracle's and every output the serial result, bit for bit")
    del ws, oracle_pools
    res = {"batch": b, "plan": plan, "layers": keep}
    del ios, base, serial
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    _FULL_RESULTS[name] = res
    return res


@pytest.mark.parametrize("name", list(FULL))
def test_pipeline_full_size(name):
    """The benchmark's three pipelines at full size, with pull-kernel loads and with
    staged loads (two workspace slots): every layer's pool after the pipeline is the
    oracle's bit for bit, every output equals its data set's serialized result bit for
    bit."""
    res = _full_pipeline(name)
    assert set(res["layers"]) == set(_special_layers(res["batch"].num_layers))


@pytest.mark.parametrize("name,which", [(nm, w) for nm in FULL for w in ("first", "middle", "last")])
def test_pipeline_full_size_every_row(name, which):
    """Every row of every head of the first, middle and last layer of each full-size
    pipeline against the fp64 oracle (suffix rows equal full-prefill rows, Sec. 2.2)."""
    res = _full_pipeline(name)
    b = res["batch"]
    l = dict(zip(("first", "middle", "last"), _special_layers(b.num_layers)))[which]
    rec = res["layers"][l]
    say(f"[gpu] pipeline {b.name} layer {l}: every row against the oracle")
    want = oattn.attention(rec["q"], rec["pk"], rec["pv"], b.block_tables, np.asarray(b.prefix_lens, np.int32),
                           res["plan"][3], b.num_kv_heads, BS)
    got = synth.bf16_bits_to_f32(rec["out"]).astype(np.float64)
    assert got.shape == want.shape == (b.T, b.num_q_heads, b.head_dim)
    mx, mean = error_stats(got, want)
    say(f"    layer {l}: {got.size} outputs, max_abs={mx:.3e} mean_abs={mean:.3e}")
    assert np.all(np.isfinite(got)) and mx <= MAX_ABS and mean <= MEAN_ABS
