#!/usr/bin/env python3
"""Benchmark of the per-layer prefix-reuse prefill step on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload l8b_layer]
                    [--no-pipeline] [--no-cpu-baseline]

Prints ONE JSON line. The timed step is one layer's compute step of the
Llama-3-8B-shaped batch (4 sequences, 32 q / 8 kv heads, head_dim 128, 4096
cached + 256 new tokens each) with every input resident in HBM: the plan is
made once, the cached prefix blocks are loaded once before timing, and each
step runs append (new K/V into the pool) then paged prefix-prefill attention
on one stream. `value` = attention FLOPs (causal-exact) / step time.

Reported beside it:
  roofline      the attention kernel's achieved TFLOP/s (HIP events around each
                launch) against the bf16 MFMA peak;
  load          host-to-pool copy of the layer's 64 MiB of cached blocks, per
                copy method, against a measured contiguous pinned copy;
  append        the scatter's HBM bytes/s;
  pipeline      the 32-layer two-stream pipeline: exposed load per layer,
                the flow-shop least exposure, and their difference;
  cpu_baseline  the fp64 oracle on a bounded sample of the same layer.

The copy, compute and offload streams of a pipeline overlap only if HIP maps them
to different hardware queues. HIP maps a process's streams, in creation order,
onto GPU_MAX_HW_QUEUES hardware queues (4 unless set), so with the several streams
this script creates two of a pipeline's streams can share a queue and run in
series; the script therefore raises the count to 8 (before HIP starts) unless the
environment already sets it.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

os.environ.setdefault("GPU_MAX_HW_QUEUES", "8")

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

MFMA_BF16_PEAK_TFLOPS = 2500.0     # MI355X dense bf16
HBM_PEAK_GBS = 8000.0              # MI355X HBM3E
ATTN_SOURCE = os.path.join(ROOT, "paper_2603_23049_amd", "csrc", "attn.hip")
# Committed counter summaries of the attention's HBM traffic, per workload.
TRAFFIC_PROFILES = {"l70b_pipe80": os.path.join(ROOT, "profiles", "prefill_attn_l70b_pipe80_layer_traffic.md"),
                    "l8b_layer": os.path.join(ROOT, "profiles", "prefill_attn_l8b_layer_traffic.md")}


def source_sha256(path: str) -> str:
    import hashlib
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def measured_traffic(workload_name: str):
    """HBM bytes per attention launch from the committed counter summary of this
    workload, or None when the summary is missing or was taken on a different
    attention source."""
    path = TRAFFIC_PROFILES.get(workload_name)
    if path is None or not os.path.exists(path):
        return None
    fields = {}
    for line in open(path):
        if line.startswith("- ") and ":" in line:
            k, v = line[2:].split(":", 1)
            fields[k.strip()] = v.strip().strip("`")
    if fields.get("attn_source_sha256") != source_sha256(ATTN_SOURCE):
        return None
    try:
        return float(fields["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def copy_calibration(nbytes=256 << 20, reps=5):
    """A plain device copy of known size, for scaling the FETCH_SIZE / WRITE_SIZE counters."""
    import torch
    src = torch.ones(nbytes, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read_per_launch": nbytes, "copy_bytes_written_per_launch": nbytes,
                      "launches": reps}), flush=True)


def attention_flops(prefix_lens, suffix_lens, num_q_heads, head_dim) -> float:
    """Causal-exact multiply-add count x2 of QK^T and PV: 4*d per (query, key) pair."""
    pairs = sum(s * p + s * (s + 1) // 2 for p, s in zip(prefix_lens, suffix_lens))
    return 4.0 * head_dim * num_q_heads * pairs


def load_bytes(prefix_lens, num_kv_heads, head_dim, block_size=16) -> int:
    """K and V bytes of every cached block (whole blocks move)."""
    blocks = sum(-(-p // block_size) for p in prefix_lens)
    return blocks * block_size * num_kv_heads * head_dim * 2 * 2


def append_bytes(T, num_kv_heads, head_dim) -> int:
    """New K and V rows read once and written once."""
    return 2 * T * num_kv_heads * head_dim * 2 * 2


def flow_shop_exposure(load_ms: float, compute_ms: float, n: int) -> float:
    """Least total exposed load of n layers on two in-order queues (loads back to back,
    layer l's compute after its load and after layer l-1's compute):
    makespan = max over l of ((l+1) c + (n-l) p); exposure = makespan - n p."""
    makespan = max((l + 1) * load_ms + (n - l) * compute_ms for l in range(n))
    return makespan - n * compute_ms


def workload(name):
    """Named batch: the generator registry plus the RAG mix built through the prefix tree."""
    from paper_2603_23049_amd import prefix_tree, synth
    if name == "rag_mix":
        return prefix_tree.rag_mix_batch()
    if name == "l8b_pipe32_s6144":
        return synth.l8b_pipe32(suffix=6144)
    return synth.REGISTRY[name]()


def _median(xs):
    return float(np.median(np.asarray(xs, dtype=np.float64)))


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


def _setup_layer(batch, layer=0, method="kernel_pull", data=None):
    import torch
    from paper_2603_23049_amd import pcr, synth
    data = synth.make_layer(batch, layer) if data is None else data
    Hkv, d, bs = batch.num_kv_heads, batch.head_dim, batch.block_size

    def dev(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16) if a.dtype == np.uint16 else a).cuda()

    def pin(a):
        t = torch.empty(a.shape, dtype=torch.int16, pin_memory=True)
        t.copy_(torch.from_numpy(a.view(np.int16)))
        return t

    pool = pcr.KVPool(torch.zeros((batch.pool_blocks, Hkv, bs * d), dtype=torch.int16, device="cuda"),
                      torch.zeros((batch.pool_blocks, Hkv, bs * d), dtype=torch.int16, device="cuda"), Hkv, d)
    host = pcr.HostKV(pin(data.host_k), pin(data.host_v), Hkv, d)
    src, dst, slots, cu = pcr.plan(batch.prefix_lens, batch.suffix_lens, batch.block_tables, batch.host_blocks, bs)
    pl = np.asarray(batch.prefix_lens, np.int32)
    L = pcr.Layer(host, pool, dev(data.q), dev(data.k_new), dev(data.v_new),
                  torch.zeros(data.q.shape, dtype=torch.int16, device="cuda"))
    bp = pcr.BatchPlan(src, dst, dev(slots), dev(batch.block_tables), dev(pl), dev(cu), pl, cu,
                       batch.num_q_heads, 1.0 / math.sqrt(d))
    return L, bp, data


def _setup_pipeline(batch, distinct):
    """n layers with their own pools; host store, Q and new K/V come from `distinct`
    generated data sets, layer l taking set l % distinct (the same bytes are moved and
    computed per layer either way; the GPU tests run the same assignment)."""
    import torch
    from paper_2603_23049_amd import pcr, synth
    sets = synth.pipeline_data_sets(batch.num_layers, distinct)
    datas = synth.make_layers(batch, range(max(sets) + 1))
    base = []
    bp = None
    for k, data in enumerate(datas):
        L, bp_l, _ = _setup_layer(batch, k, data=data)
        base.append(L)
        bp = bp or bp_l
    del datas
    layers = list(base)
    Hkv, d, bs = batch.num_kv_heads, batch.head_dim, batch.block_size
    for l in range(len(base), batch.num_layers):
        src = base[sets[l]]
        pool = pcr.KVPool(torch.zeros((batch.pool_blocks, Hkv, bs * d), dtype=torch.int16, device="cuda"),
                          torch.zeros((batch.pool_blocks, Hkv, bs * d), dtype=torch.int16, device="cuda"), Hkv, d)
        layers.append(pcr.Layer(src.host, pool, src.q, src.k_new, src.v_new, src.out))
    return layers, bp


def _attn(L, bp, stream=None):
    from paper_2603_23049_amd import pcr
    pcr.prefix_prefill_attn(L.q, L.pool, bp.block_tables, bp.prefix_lens, bp.cu_suffix, bp.host_prefix_lens,
                            bp.host_cu_suffix, bp.num_q_heads, L.out, sm_scale=bp.sm_scale, stream=stream)


class ClockSampler:
    """amd-smi clock and power samples. The sampling shell is started before this
    process touches the GPU (a process that has initialised the GPU starts no other
    program) and waits on a pipe until start() tells it to begin."""

    def __init__(self, n=6, period_s=0.25):
        import shutil
        import subprocess
        self.proc = None
        smi = shutil.which("amd-smi")
        if smi is None:
            return
        script = (f"read go || exit 0; for i in $(seq 1 {n}); do echo @sample; "
                  f"timeout 5 {smi} metric -g 0 --clock --power --json 2>/dev/null; sleep {period_s}; done")
        # its own process group, so that close() can end the shell and any amd-smi child
        self.proc = subprocess.Popen(["bash", "-c", script], stdin=subprocess.PIPE, stdout=subprocess.PIPE,
                                     stderr=subprocess.DEVNULL, text=True, start_new_session=True)

    def start(self):
        if self.proc:
            self.proc.stdin.write("go\n")
            self.proc.stdin.flush()

    def running(self):
        return self.proc is not None and self.proc.poll() is None

    def _kill_group(self):
        import signal
        try:
            os.killpg(self.proc.pid, signal.SIGKILL)
        except (ProcessLookupError, PermissionError):
            pass

    def collect(self, timeout=30):
        """[(gfx MHz per XCD, socket power W)] of the samples that parsed."""
        if self.proc is None:
            return []
        try:
            out, _ = self.proc.communicate(timeout=timeout)
        except Exception:
            self._kill_group()
            self.proc.wait()
            return []
        samples = []
        for body in out.split("@sample")[1:]:
            try:
                g = json.loads(body)["gpu_data"][0]
                clk = g["clock"]
                gfx = [clk[k]["clk"]["value"] for k in sorted(clk) if k.startswith("gfx_")]
                samples.append((gfx, g["power"]["socket_power"]["value"]))
            except Exception:
                continue
        return samples

    def close(self):
        """Ends the sampling shell and everything it started (its whole process group),
        and reaps it, so no process outlives the benchmark."""
        if self.proc is None:
            return
        if self.proc.poll() is None:
            try:
                self.proc.stdin.close()
                self.proc.wait(timeout=10)
            except Exception:
                pass
        self._kill_group()       # a hung amd-smi child may outlive the shell
        try:
            self.proc.wait(timeout=10)
        except Exception:
            pass


def measure_clock_hold(batch, sampler, settle_s=0.5, max_s=15.0):
    """The attention kept running back to back while amd-smi samples the clocks and the
    socket power (after settle_s of load). Returns the samples' per-XCD mean clocks, their
    mean, the mean power and the attention time per launch during the sampling."""
    import torch
    from paper_2603_23049_amd import pcr
    if sampler is None or sampler.proc is None:
        return None
    L, bp, _ = _setup_layer(batch)
    pcr.load_kv_layer(L.host, bp.src_blocks, L.pool, bp.dst_blocks, method="kernel_pull")
    torch.cuda.synchronize()
    s = torch.cuda.current_stream()
    t0 = time.perf_counter()
    started = False
    launches, ms = 0, 0.0
    while time.perf_counter() - t0 < max_s:
        a, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(s)
        for _ in range(50):
            _attn(L, bp, s)
        e.record(s)
        e.synchronize()
        if started:
            launches += 50
            ms += a.elapsed_time(e)
            if not sampler.running():
                break
        elif time.perf_counter() - t0 >= settle_s:
            sampler.start()
            started = True
    samples = sampler.collect()
    if not samples or launches == 0:
        return None
    n_x = min(len(g) for g, _ in samples)
    per_xcd = [float(np.mean([g[x] for g, _ in samples])) for x in range(n_x)]
    return {"gfx_mhz_per_xcd": per_xcd, "gfx_mhz_mean": float(np.mean(per_xcd)),
            "gfx_mhz_min": float(min(per_xcd)), "socket_power_w": float(np.mean([p for _, p in samples])),
            "samples": len(samples), "attn_ms_during": ms / launches, "source": "amd-smi metric --clock --power"}


def warm_up(fn, min_ms, min_calls=3):
    """Calls fn until at least min_calls calls and min_ms of wall time have passed. After
    an idle gap the GPU clock starts low and ramps up under sustained load: with 10
    warm-up steps the l8b_layer step measured about 10% slower than after 200-1600
    (72.2-72.8 us per step from 200 on)."""
    import torch
    t0 = time.perf_counter()
    n = 0
    while True:
        fn()
        n += 1
        if n >= min_calls and n % 4 == 0:
            torch.cuda.synchronize()
            if (time.perf_counter() - t0) * 1e3 >= min_ms:
                return n


def measure_step(batch, steps, warmup, min_warm_ms=500.0, graph=True):
    """Timed compute step (append + attention) with prefix KV already in the pool.

    Warm-up: `warmup` steps, then more until at least min_warm_ms of sustained work has
    passed (after an idle gap the GPU clock starts low and ramps up under load), whatever
    `warmup` says. Timed region: `steps` steps between one event pair and the wall clock,
    synchronized on both sides; inside it each attention launch is bracketed by its own
    event pair on the stream it runs on, so the attention's per-launch time comes from
    the same window as the step time. Then the append alone, back to back, for its
    per-launch time (a launch-bound kernel at these sizes), the attention alone back to
    back, and (graph=True) the step replayed from a HIP graph."""
    import torch
    from paper_2603_23049_amd import pcr
    L, bp, _ = _setup_layer(batch)
    pcr.load_kv_layer(L.host, bp.src_blocks, L.pool, bp.dst_blocks, method="kernel_pull")
    torch.cuda.synchronize()
    s = torch.cuda.current_stream()

    def step():
        pcr.append_kv(L.pool, L.k_new, L.v_new, bp.slot_mapping, stream=s)
        _attn(L, bp, s)

    for _ in range(warmup):
        step()
    warm_calls = warm_up(step, min_warm_ms)
    torch.cuda.synchronize()
    ev = lambda: torch.cuda.Event(enable_timing=True)
    a, e = ev(), ev()
    pairs = [(ev(), ev()) for _ in range(steps)]
    t0 = time.perf_counter()
    a.record(s)
    for x, y in pairs:
        pcr.append_kv(L.pool, L.k_new, L.v_new, bp.slot_mapping, stream=s)
        x.record(s)
        _attn(L, bp, s)
        y.record(s)
    e.record(s)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    step_ms = a.elapsed_time(e) / steps
    launches = [x.elapsed_time(y) for x, y in pairs]
    attn_ms = float(np.mean(launches))

    a2, e2 = ev(), ev()
    a2.record(s)
    for _ in range(steps):
        pcr.append_kv(L.pool, L.k_new, L.v_new, bp.slot_mapping, stream=s)
    e2.record(s)
    e2.synchronize()
    append_ms = a2.elapsed_time(e2) / steps
    # the attention alone, back to back under one event pair (no per-launch gaps: for a
    # short launch the per-launch events above add several microseconds each)
    a3, e3 = ev(), ev()
    a3.record(s)
    for _ in range(steps):
        _attn(L, bp, s)
    e3.record(s)
    e3.synchronize()
    graph_ms = _graph_step_ms(L, bp, steps) if graph else None
    return dict(step_ms=float(step_ms), wall_ms_per_step=wall / steps * 1e3, append_ms=append_ms,
                graph_step_ms=graph_ms,
                attn_ms=attn_ms, attn_ms_min=float(min(launches)), attn_ms_max=float(max(launches)),
                attn_ms_median=_median(launches), attn_b2b_ms=a3.elapsed_time(e3) / steps, wall_s=wall,
                warmup_calls=warmup + warm_calls)


def _graph_step_ms(L, bp, steps):
    """The compute step (append + attention) captured once into a HIP graph (torch's
    CUDAGraph: the library's launches on the capturing stream become its nodes) and
    replayed `steps` times back to back under one event pair: the step without the host
    launch gaps between its kernels."""
    import torch
    from paper_2603_23049_amd import pcr

    def step():   # on the current stream (the capturing one inside the graph context)
        pcr.append_kv(L.pool, L.k_new, L.v_new, bp.slot_mapping)
        _attn(L, bp)

    s = torch.cuda.current_stream()
    side = torch.cuda.Stream()
    side.wait_stream(s)
    with torch.cuda.stream(side):    # one eager step on a side stream before capture
        step()
    s.wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    g.replay()
    torch.cuda.synchronize()
    a, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record(s)
    for _ in range(steps):
        g.replay()
    e.record(s)
    e.synchronize()
    ms = a.elapsed_time(e) / steps
    del g
    return float(ms)


def measure_load(batch, reps=10):
    """Host-to-pool copy of one layer's cached blocks, per method; plus a contiguous
    256 MiB pinned host-to-device copy as the link reference."""
    import torch
    from paper_2603_23049_amd import pcr
    L, bp, _ = _setup_layer(batch)
    nbytes = load_bytes(batch.prefix_lens, batch.num_kv_heads, batch.head_dim)
    s = torch.cuda.Stream()
    out = {"bytes_per_layer": nbytes}
    for method in ("kernel_pull", "dma_per_block", "dma_batch"):
        try:
            times = []
            for r in range(reps + 2):
                a, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                a.record(s)
                pcr.load_kv_layer(L.host, bp.src_blocks, L.pool, bp.dst_blocks, method=method, stream=s)
                e.record(s)
                e.synchronize()
                if r >= 2:
                    times.append(a.elapsed_time(e))
            ms = _median(times)
            out[method] = {"ms": ms, "GBps": nbytes / ms / 1e6}
        except Exception as ex:  # a method this runtime lacks
            out[method] = {"error": str(ex)[:200]}
    # staged: copy-engine transfers into a workspace, then the scatter kernel; the
    # transfers alone (the same bytes host to workspace) give the two stages' times
    ws = torch.empty(pcr.staged_workspace_bytes(len(bp.src_blocks), batch.num_kv_heads, batch.head_dim),
                     dtype=torch.uint8, device="cuda")
    half = nbytes // 2
    hk = L.host.k.view(-1).view(torch.uint8)[:half]
    hv = L.host.v.view(-1).view(torch.uint8)[:half]

    def transfers():
        with torch.cuda.stream(s):
            ws[:half].copy_(hk, non_blocking=True)
            ws[half:].copy_(hv, non_blocking=True)

    def staged():
        pcr.load_kv_layer(L.host, bp.src_blocks, L.pool, bp.dst_blocks, method="dma_staged", stream=s, workspace=ws)

    stg = {}
    for key, fn in (("ms", staged), ("transfer_ms", transfers)):
        times = []
        for r in range(reps + 2):
            a, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(s)
            fn()
            e.record(s)
            e.synchronize()
            if r >= 2:
                times.append(a.elapsed_time(e))
        stg[key] = _median(times)
    stg["GBps"] = nbytes / stg["ms"] / 1e6
    stg["scatter_ms"] = max(stg["ms"] - stg["transfer_ms"], 0.0)
    out["dma_staged"] = stg
    del ws
    big = 256 << 20
    h = torch.empty(big, dtype=torch.uint8, pin_memory=True)
    h.fill_(1)
    d = torch.empty(big, dtype=torch.uint8, device="cuda")
    times = []
    for r in range(12):
        a, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        with torch.cuda.stream(s):
            a.record(s)
            d.copy_(h, non_blocking=True)
            e.record(s)
        e.synchronize()
        if r >= 2:
            times.append(a.elapsed_time(e))
    out["contiguous_h2d_GBps"] = big / _median(times) / 1e6
    return out


def _bracketed_ms(run, start_stream, end_stream, reps):
    """Best of `reps` runs of `run()` after one warm-up, each timed by one event pair:
    the start recorded on start_stream before the call, the end on end_stream after it
    (the pipelines' own per-layer events add gaps to the streams they sit on, so the
    totals come from untimed runs)."""
    import torch
    times = []
    for r in range(reps + 1):
        torch.cuda.synchronize()
        a, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(start_stream)
        run()
        e.record(end_stream)
        e.synchronize()
        if r >= 1:
            times.append(a.elapsed_time(e))
    return min(times)


def measure_pipeline(batch, method, load_ms_iso, compute_ms_iso, reps=3, distinct=None, staged_stages=None,
                     layers_bp=None):
    """The n-layer pipeline. Exposure per layer is the pipeline's time per layer beyond
    the layer's isolated compute; its least possible value follows from the isolated
    per-layer load and compute times (two in-order queues; for method "staged", the
    three stages transfer, scatter and compute from `staged_stages` = (transfer ms,
    scatter ms)). The total comes from untimed runs; one timed run gives the per-layer
    breakdown. With `distinct`, only that many layers' host/Q/K/V data are generated and
    reused round-robin (every layer still has its own pool and moves its own bytes).
    Method "staged" runs pcr_pipeline_run_staged with two workspace slots."""
    import torch
    from paper_2603_23049_amd import pcr
    n = batch.num_layers
    layers, bp = layers_bp or _setup_pipeline(batch, distinct or n)
    copy_s, comp_s = torch.cuda.Stream(), torch.cuda.Stream()
    if method == "staged":
        scat_s = torch.cuda.Stream()
        ws = torch.empty(2 * pcr.pipeline_staged_slot_bytes(len(bp.src_blocks), batch.num_kv_heads, batch.head_dim),
                         dtype=torch.uint8, device="cuda")
        run = lambda timing=False: pcr.pipeline_run_staged(layers, bp, ws, copy_s, scat_s, comp_s, timing=timing)
    else:
        run = lambda timing=False: pcr.pipeline_run(layers, bp, copy_s, comp_s, method=method, timing=timing)
    total = _bracketed_ms(lambda: run(), comp_s, comp_s, reps)
    best = run(timing=True)
    e_raw = total / n - compute_ms_iso
    if method == "staged":
        bound = flow_shop3_makespan(staged_stages[0], staged_stages[1], compute_ms_iso, n)
    else:
        bound = flow_shop_exposure(load_ms_iso, compute_ms_iso, n) + n * compute_ms_iso
    e_min = bound / n - compute_ms_iso
    del layers
    torch.cuda.synchronize()
    return {"layers": n, "workload": batch.name, "method": method, "distinct_layer_data": distinct or n,
            "total_ms": total, "total_ms_timed_run": best["total_ms"],
            "sum_compute_ms_in_pipeline": best["sum_compute_ms"],
            "load_ms_per_layer_isolated": load_ms_iso, "compute_ms_per_layer_isolated": compute_ms_iso,
            "load_ms_per_layer_in_pipeline": float(np.median(best["load_ms"])),
            "compute_ms_per_layer_in_pipeline": float(np.median(best["compute_ms"])),
            "exposed_ms_per_layer": e_raw, "exposed_min_ms_per_layer": e_min,
            "exposed_over_min_ms_per_layer": e_raw - e_min,
            "exposed_over_min_frac_of_load": (e_raw - e_min) / load_ms_iso if load_ms_iso > 0 else None,
            "exposed_frac_of_load": e_raw / load_ms_iso if load_ms_iso > 0 else None,
            "bound_makespan_ms": bound,
            "exposed_ideal_ms_per_layer": load_ms_iso / n if compute_ms_iso >= load_ms_iso else None}


def measure_decode(B=64, ctx=4352, Hq=32, Hkv=8, d=128, steps=30, seed=71, name=None, prefill_beside=True):
    """One decode step (one new token per sequence, attending over its context) of a
    Llama-3-8B-shaped batch, attention only, through the split-key decode entry point
    with the workspace its size query asks for; `ctx` is one length for every sequence
    or one per sequence (ragged). The prefill kernel on the same rows (one-token
    suffixes) is timed beside it. Pool, Q and tables drawn on the device (the values do
    not change the work). HBM bytes = every key's K and V once + Q + out."""
    import torch
    from paper_2603_23049_amd import pcr
    bs = 16
    n_h = np.asarray(ctx, np.int32) if np.ndim(ctx) else np.full(B, ctx, np.int32)
    B = int(n_h.shape[0])
    nbs = -(-n_h // bs)
    mb = int(nbs.max())
    g = torch.Generator(device="cuda").manual_seed(seed)
    pool_blocks = int(nbs.sum())
    pk = torch.randn((pool_blocks, Hkv, bs * d), device="cuda", dtype=torch.bfloat16, generator=g).view(torch.int16)
    pv = torch.randn((pool_blocks, Hkv, bs * d), device="cuda", dtype=torch.bfloat16, generator=g).view(torch.int16)
    pool = pcr.KVPool(pk, pv, Hkv, d)
    perm = torch.randperm(pool_blocks, device="cuda", generator=g).to(torch.int32).cpu().numpy()
    bt_h = np.full((B, mb), -1, np.int32)
    off = np.concatenate([[0], np.cumsum(nbs)])
    for b in range(B):
        bt_h[b, :nbs[b]] = perm[off[b]:off[b + 1]]
    bt = torch.from_numpy(bt_h).cuda()
    q = torch.randn((B, Hq, d), device="cuda", dtype=torch.bfloat16, generator=g).view(torch.int16)
    out = torch.empty_like(q)
    n_d = torch.from_numpy(n_h).cuda()
    ws_bytes = pcr.decode_attn_workspace_bytes(B, Hq, Hkv, d, int(n_h.max()))
    ws = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device="cuda")
    pl_h = n_h - 1
    cu_h = np.arange(B + 1, dtype=np.int32)
    pl, cu = torch.from_numpy(pl_h).cuda(), torch.from_numpy(cu_h).cuda()
    s = torch.cuda.current_stream()

    def timed(fn):
        warm_up(fn, 30.0)
        a, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(s)
        for _ in range(steps):
            fn()
        e.record(s)
        e.synchronize()
        return a.elapsed_time(e) / steps

    ms = timed(lambda: pcr.decode_attn(q, pool, bt, n_d, n_h, Hq, out, workspace=ws, stream=s))
    ms_prefill = timed(lambda: pcr.prefix_prefill_attn(q, pool, bt, pl, cu, pl_h, cu_h, Hq, out, stream=s)) \
        if prefill_beside else None
    keys = int(n_h.sum())
    nbytes = keys * Hkv * d * 2 * 2 + 2 * B * Hq * d * 2
    label = name or f"decode B={B} ctx={int(n_h[0]) if np.all(n_h == n_h[0]) else 'ragged'} Hq={Hq} Hkv={Hkv} d={d}"
    rec = {"workload": label, "keys": keys, "max_context": int(n_h.max()), "attn_ms": ms, "hbm_bytes": nbytes,
           "GBps": nbytes / ms / 1e6, "frac_hbm": nbytes / ms / 1e6 / HBM_PEAK_GBS, "tokens_per_s": B / ms * 1e3,
           "workspace_bytes": ws_bytes}
    if ms_prefill is not None:
        rec.update(prefill_kernel_ms=ms_prefill, prefill_kernel_frac_hbm=nbytes / ms_prefill / 1e6 / HBM_PEAK_GBS)
    return rec


def measure_decode_ragged():
    """Decode steps of ragged batches: 64 sequences with contexts drawn uniformly from
    1024-8192 keys (seed 3), and the RAG mix's 16 requests at their full contexts (the
    decode of the requests the prefill step served)."""
    rng = np.random.default_rng(3)
    rag = workload("rag_mix")
    return [measure_decode(ctx=rng.integers(1024, 8193, 64).astype(np.int32), name="decode B=64 ctx 1k-8k ragged",
                           prefill_beside=False),
            measure_decode(ctx=(np.asarray(rag.prefix_lens) + np.asarray(rag.suffix_lens)).astype(np.int32),
                           name="decode RAG mix 16 requests", prefill_beside=False)]


def measure_mixed(n_dec=64, ctx=4352, steps=20, seed=81):
    """A mixed batch through the prefill entry point: the RAG mix's 16 prefill requests
    plus n_dec decode rows (one new token over ctx keys each), against the prefill
    requests alone and the decode rows alone through the same entry point (one launch
    up to 128 sequences, consecutive launches beyond). Pool and Q drawn on the device
    (the values do not change the work)."""
    import torch
    from paper_2603_23049_amd import pcr, synth
    rag = workload("rag_mix")
    Hq, Hkv, d, bs = rag.num_q_heads, rag.num_kv_heads, rag.head_dim, rag.block_size
    cases = {"prefill_only": (list(rag.prefix_lens), list(rag.suffix_lens)),
             "decode_only": ([ctx - 1] * n_dec, [1] * n_dec),
             "mixed": (list(rag.prefix_lens) + [ctx - 1] * n_dec, list(rag.suffix_lens) + [1] * n_dec)}
    s = torch.cuda.current_stream()
    g = torch.Generator(device="cuda").manual_seed(seed)
    rec = {"workload": f"RAG mix {len(rag.prefix_lens)} requests + {n_dec} decode rows of {ctx} keys, "
                       f"Hq={Hq} Hkv={Hkv} d={d}, prefill entry point"}
    for name, (pl_l, sl_l) in cases.items():
        nb = sum(-(-(a + b) // bs) for a, b in zip(pl_l, sl_l))
        b = synth.ragged_batch(name, Hq=Hq, Hkv=Hkv, d=d, prefix_lens=pl_l, suffix_lens=sl_l, pool_blocks=nb,
                               seed=seed)
        pk = torch.randn((nb, Hkv, bs * d), device="cuda", dtype=torch.bfloat16, generator=g).view(torch.int16)
        pv = torch.randn((nb, Hkv, bs * d), device="cuda", dtype=torch.bfloat16, generator=g).view(torch.int16)
        pool = pcr.KVPool(pk, pv, Hkv, d)
        q = torch.randn((b.T, Hq, d), device="cuda", dtype=torch.bfloat16, generator=g).view(torch.int16)
        out = torch.empty_like(q)
        pl_h = np.asarray(pl_l, np.int32)
        cu_h = np.concatenate([[0], np.cumsum(sl_l)]).astype(np.int32)
        bt = torch.from_numpy(np.ascontiguousarray(b.block_tables)).cuda()
        pl, cu = torch.from_numpy(pl_h).cuda(), torch.from_numpy(cu_h).cuda()

        def fn():
            pcr.prefix_prefill_attn(q, pool, bt, pl, cu, pl_h, cu_h, Hq, out, stream=s)

        warm_up(fn, 200.0)
        a, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(s)
        for _ in range(steps):
            fn()
        e.record(s)
        e.synchronize()
        ms = a.elapsed_time(e) / steps
        rec[f"{name}_ms"] = ms
        rec[f"{name}_tflops"] = attention_flops(pl_l, sl_l, Hq, d) / ms / 1e9
        del pk, pv, q, out, pool
        torch.cuda.empty_cache()
    rec["mixed_over_prefill_ms"] = rec["mixed_ms"] - rec["prefill_only_ms"]
    return rec


def measure_prefetch(windows=(0, 4, 6), chunk_mib=4, dram_sweep=(48, 96, 192), request_compute_ms=30.0,
                     n_serve=40):
    """Serving loop through DRAM and SSD tiers with the queue-window prefetch: SSD stall
    per request for each window size and each DRAM capacity (in chunks), on this
    machine's disk (O_DIRECT when the file system allows it), with the number of chunks
    read ahead and then evicted before their request came. Chunks are scaled to
    chunk_mib MiB; compute is a sleep of request_compute_ms per 2500 computed tokens."""
    import shutil
    import tempfile
    from paper_2603_23049_amd import prefetch, synth
    stream = synth.rag_stream(4, n_requests=64 + n_serve)
    base = os.path.join(ROOT, ".pytest_store")
    os.makedirs(base, exist_ok=True)
    d = tempfile.mkdtemp(dir=base)
    out = {"chunk_bytes": chunk_mib << 20, "requests": n_serve, "compute_ms_per_2500_tokens": request_compute_ms,
           "by_dram_chunks": {}}
    try:
        for dram_chunks in dram_sweep:
            row = {}
            for w in windows:
                st = prefetch.serve(stream.requests, store_path=os.path.join(d, f"w{w}.bin"),
                                    chunk_bytes=chunk_mib << 20, dram_chunks=dram_chunks, window=w,
                                    compute_ms_per_token=request_compute_ms / 2500, io_threads=4)
                row[f"window_{w}"] = {"stall_ms_per_request": st.stall_ms / max(st.requests, 1),
                                      "on_demand_reads": st.on_demand_reads, "prefetch_reads": st.prefetch_reads,
                                      "prefetch_hits": st.prefetch_hits, "dram_hits": st.dram_hits,
                                      "prefetch_evicted_before_use": st.prefetch_evicted, "wall_ms": st.wall_ms}
            out["by_dram_chunks"][str(dram_chunks)] = row
        probe = prefetch.page_aligned_buffer(chunk_mib << 20)
        from paper_2603_23049_amd import pcr
        store = pcr.ChunkStore(os.path.join(d, "probe.bin"), chunk_mib << 20, 4)
        bufs = [prefetch.page_aligned_buffer(chunk_mib << 20) for _ in range(16)]
        for i, b in enumerate(bufs):
            store.write_async(i, b)
        store.wait()
        t0 = time.perf_counter()
        for i, b in enumerate(bufs):
            store.read_async(i, b)
        store.wait()
        dt = time.perf_counter() - t0
        out["ssd_read_GBps"] = 16 * (chunk_mib << 20) / dt / 1e9
        sts = store.stats()
        out["direct_io"] = sts["direct_io"]
        out["direct_fallbacks"] = sts["direct_fallbacks"]
        store.close()
        del probe
    finally:
        shutil.rmtree(d, ignore_errors=True)
    return out


def flow_shop3_makespan(load_ms: float, compute_ms: float, offload_ms: float, n: int) -> float:
    """Least makespan of n identical layers through three in-order queues (load, then
    compute, then offload): one layer's three steps plus n-1 times the slowest step."""
    return load_ms + compute_ms + offload_ms + (n - 1) * max(load_ms, compute_ms, offload_ms)


def _host_store(batch, n_blocks):
    import torch
    from paper_2603_23049_amd import pcr
    shape = (max(n_blocks, 1), batch.num_kv_heads, batch.block_size * batch.head_dim)
    return pcr.HostKV(torch.zeros(shape, dtype=torch.int16, pin_memory=True),
                      torch.zeros(shape, dtype=torch.int16, pin_memory=True), batch.num_kv_heads, batch.head_dim)


def measure_offload(batch, reps=6, chunk=256):
    """Pool-to-host copy of one layer's computed whole chunks, per method; plus a
    contiguous 256 MiB device-to-pinned copy as the link reference."""
    import torch
    from paper_2603_23049_amd import pcr
    L, bp, _ = _setup_layer(batch)
    src, dst = pcr.plan_offload(batch.prefix_lens, batch.suffix_lens, batch.block_tables, batch.block_size, chunk)
    host = _host_store(batch, len(dst))
    nbytes = len(src) * batch.block_size * batch.num_kv_heads * batch.head_dim * 2 * 2
    s = torch.cuda.Stream()
    ws = torch.empty(pcr.staged_workspace_bytes(len(src), batch.num_kv_heads, batch.head_dim), dtype=torch.uint8,
                     device="cuda")
    out = {"bytes_per_layer": nbytes, "blocks": int(len(src))}
    for method in ("kernel_pull", "dma_per_block", "dma_staged"):
        times = []
        for r in range(reps + 2):
            a, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(s)
            pcr.offload_kv_layer(L.pool, src, host, dst, method=method, stream=s, workspace=ws)
            e.record(s)
            e.synchronize()
            if r >= 2:
                times.append(a.elapsed_time(e))
        ms = _median(times)
        out["kernel_push" if method == "kernel_pull" else method] = {"ms": ms, "GBps": nbytes / ms / 1e6}
    big = 256 << 20
    h = torch.empty(big, dtype=torch.uint8, pin_memory=True)
    d = torch.ones(big, dtype=torch.uint8, device="cuda")
    times = []
    for r in range(8):
        a, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        with torch.cuda.stream(s):
            a.record(s)
            h.copy_(d, non_blocking=True)
            e.record(s)
        e.synchronize()
        if r >= 2:
            times.append(a.elapsed_time(e))
    out["contiguous_d2h_GBps"] = big / _median(times) / 1e6
    return out, src, dst


def measure_pipeline_offload(batch, method, load_ms_iso, compute_ms_iso, offload_ms_iso, src, dst, reps=2,
                             distinct=4, offload_method="dma_staged", staged_stages=None):
    """The three-stream pipeline (load, compute, offload of the computed chunks), or with
    method "staged" the four-stream one (transfers, scatter, compute, offload).
    Exposure per layer = (pipeline time - n x isolated compute) / n; its least value
    follows from the isolated per-layer times of the steps (staged_stages = (transfer
    ms, scatter ms) for the staged loads)."""
    import torch
    from paper_2603_23049_amd import pcr
    n = batch.num_layers
    layers, bp = _setup_pipeline(batch, distinct)
    outs = [_host_store(batch, len(dst)) for _ in range(min(distinct, n))]
    dsts = [outs[l % len(outs)] for l in range(n)]
    cs, ks, os_ = torch.cuda.Stream(), torch.cuda.Stream(), torch.cuda.Stream()
    ws = torch.empty(pcr.staged_workspace_bytes(len(src), batch.num_kv_heads, batch.head_dim), dtype=torch.uint8,
                     device="cuda")
    if method == "staged":
        ss = torch.cuda.Stream()
        lws = torch.empty(2 * pcr.pipeline_staged_slot_bytes(len(bp.src_blocks), batch.num_kv_heads, batch.head_dim),
                          dtype=torch.uint8, device="cuda")
        run = lambda timing=False: pcr.pipeline_run_offload_staged(layers, dsts, bp, src, dst, lws, cs, ss, ks, os_,
                                                                   offload_method=offload_method,
                                                                   offload_workspace=ws, timing=timing)
    else:
        run = lambda timing=False: pcr.pipeline_run_offload(layers, dsts, bp, src, dst, cs, ks, os_, method=method,
                                                            offload_method=offload_method, workspace=ws,
                                                            timing=timing)
    total = _bracketed_ms(lambda: run(), ks, os_, reps)
    best = run(timing=True)
    e_raw = total / n - compute_ms_iso
    if method == "staged":
        stages = (staged_stages[0], staged_stages[1], compute_ms_iso, offload_ms_iso)
        bound = sum(stages) + (n - 1) * max(stages)
    else:
        bound = flow_shop3_makespan(load_ms_iso, compute_ms_iso, offload_ms_iso, n)
    e_min = bound / n - compute_ms_iso
    del layers, outs, dsts
    torch.cuda.synchronize()
    return {"layers": n, "workload": batch.name, "method": method, "offload_method": offload_method,
            "distinct_layer_data": distinct, "total_ms": total, "total_ms_timed_run": best["total_ms"],
            "compute_end_ms": best["compute_end_ms"],
            "load_ms_per_layer_isolated": load_ms_iso, "compute_ms_per_layer_isolated": compute_ms_iso,
            "offload_ms_per_layer_isolated": offload_ms_iso,
            "offload_ms_per_layer_in_pipeline": float(np.median(best["offload_ms"])),
            "exposed_ms_per_layer": e_raw, "exposed_min_ms_per_layer": e_min,
            "exposed_over_min_ms_per_layer": e_raw - e_min,
            "exposed_frac_of_transfer": e_raw / (load_ms_iso + offload_ms_iso),
            "bound_makespan_ms": bound,
            "synchronous_ms": n * (load_ms_iso + compute_ms_iso + offload_ms_iso)}


def _oracle_layer(batch, layer=0):
    """One layer's oracle inputs: the layer's data, the plan, and the pools after the
    oracle's own load and append."""
    from oracle import datamove as odm
    from paper_2603_23049_amd import synth
    data = synth.make_layer(batch, layer)
    plan = odm.plan(batch.prefix_lens, batch.suffix_lens, batch.block_tables, batch.host_blocks, 16)
    shape = (batch.pool_blocks, batch.num_kv_heads, 16 * batch.head_dim)
    pk, pv = odm.pool_after_layer(np.zeros(shape, np.uint16), np.zeros(shape, np.uint16), data.host_k, data.host_v,
                                  plan, data.k_new, data.v_new)
    return data, plan, pk, pv


def _time_oracle_attention(batch, budget_s=0.0, rows=None, inputs=None):
    """The fp64 oracle on a layer (every row, or the given (token, head) rows), repeated
    until budget_s of wall time has passed (at least once). Returns (passes, seconds,
    FLOPs per pass)."""
    from oracle import attention as oattn
    data, plan, pk, pv = inputs or _oracle_layer(batch)
    pl = np.asarray(batch.prefix_lens, np.int32)
    if rows is None:
        flops = attention_flops(batch.prefix_lens, batch.suffix_lens, batch.num_q_heads, batch.head_dim)
    else:   # 4*d FLOPs per (row, visible key) pair
        cu = plan[3]
        seq = np.searchsorted(cu, rows[:, 0], side="right") - 1
        keys = pl[seq] + (rows[:, 0] - cu[seq]) + 1
        flops = 4.0 * batch.head_dim * float(keys.sum())
    reps, t0 = 0, time.perf_counter()
    while True:
        oattn.attention(data.q, pk, pv, batch.block_tables, pl, plan[3], batch.num_kv_heads, 16, rows=rows)
        reps += 1
        dt = time.perf_counter() - t0
        if dt >= budget_s:
            return reps, dt, flops


def cpu_baseline(batch, budget_s=12.0, inputs=None):
    """The fp64 oracle (as it stands) on one whole layer of the headline workload (every
    row of every head), repeated until about budget_s has passed; TFLOP/s by the layer's
    causal-exact FLOPs."""
    from oracle import attention as oattn
    reps, dt, flops = _time_oracle_attention(batch, budget_s, inputs=inputs)
    return {"value": reps * flops / dt / 1e12, "unit": "TFLOP/s", "cores": oattn.num_threads(), "kind": "oracle",
            "sample": f"one whole layer of {batch.name} (every row of every head), fp64, {reps} pass(es) in "
                      f"{dt:.1f} s", "ms_per_layer": dt / reps * 1e3}


def cpu_baseline_legs(headline=None):
    """The oracle timed on the other configurations (reported beside the headline, never
    a target): tiny, the Llama-3-8B layer and the RAG mix in full; one layer of the
    32-layer stack (the 8B layer's shape) and of the 80-layer stack with the x n
    extrapolation labelled; one thread on a sampled part of the 8B layer; and the host
    memcpy rates of the load, append and gather oracles."""
    from oracle import attention as oattn
    from oracle import datamove as odm
    from paper_2603_23049_amd import synth
    cores = oattn.num_threads()
    legs = {"cores": cores}
    for name in ("tiny", "l8b_layer", "rag_mix"):
        b = workload(name)
        reps, dt, flops = _time_oracle_attention(b, 1.0)
        legs[name] = {"ms": dt / reps * 1e3, "GFLOPs": flops / dt * reps / 1e9, "flops": flops,
                      "what": f"every row of every head, {reps} pass(es)"}
    per = legs["l8b_layer"]["ms"]
    legs["l8b_pipe32"] = {"ms_per_layer": per, "ms_extrapolated_x32": 32 * per,
                          "what": "one layer timed (the l8b_layer shape), x32 extrapolated"}
    if headline is not None:
        legs["l70b_pipe80"] = {"ms_per_layer": headline["ms_per_layer"],
                               "ms_extrapolated_x80": 80 * headline["ms_per_layer"],
                               "what": "one layer timed (the headline cpu_baseline), x80 extrapolated"}
    # one thread: every 8th token's rows of the 8B layer
    b = synth.l8b_layer()
    inputs = _oracle_layer(b)
    rows = np.array([[t, h] for t in range(0, b.T, 8) for h in range(b.num_q_heads)], np.int32)
    oattn.set_num_threads(1)
    try:
        reps, dt, flops = _time_oracle_attention(b, 3.0, rows=rows, inputs=inputs)
    finally:
        oattn.set_num_threads(cores)
    legs["one_thread"] = {"GFLOPs": reps * flops / dt / 1e9, "threads": 1,
                          "what": f"l8b_layer, every 8th new token's rows ({len(rows)} rows), {reps} pass(es)"}
    # host memcpy rates of the bit-copy oracles on the 8B layer
    data, plan, pk, pv = inputs
    src, dst, slots, cu = plan
    zk, zv = np.zeros_like(pk), np.zeros_like(pv)
    t0 = time.perf_counter()
    odm.load(zk, zv, data.host_k, data.host_v, src, dst)
    t_load = time.perf_counter() - t0
    t0 = time.perf_counter()
    odm.append(zk, zv, data.k_new, data.v_new, slots, 16)
    t_app = time.perf_counter() - t0
    starts = np.zeros(b.B, np.int64)
    lens = [512] * b.B                   # the first 512 tokens of each sequence
    t0 = time.perf_counter()
    odm.gather(pk, pv, b.block_tables, starts, lens, b.head_dim, 16)
    t_gat = time.perf_counter() - t0
    lb = load_bytes(b.prefix_lens, b.num_kv_heads, b.head_dim)
    ab = append_bytes(b.T, b.num_kv_heads, b.head_dim)
    gb = 2 * sum(lens) * b.num_kv_heads * b.head_dim * 2 * 2
    legs["memcpy"] = {"load_GBps": lb / t_load / 1e9, "append_GBps": ab / t_app / 1e9,
                      "gather_GBps": gb / t_gat / 1e9,
                      "what": "numpy bit-copy oracles on the l8b_layer layer (load 64 MiB, append 4+4 MiB, "
                              "gather of each sequence's first 512 tokens; bytes read + written)"}
    return legs


def hit_ratio_report(capacities=(64, 128, 200, 300), n_requests=400):
    """RAG-mix stream (seed 4, 400 requests): token hit ratio through a prefix tree of
    limited capacity (in 256-token chunks), with the look-ahead over the next 4 waiting
    requests and with plain leaf LRU; and with no capacity limit."""
    from paper_2603_23049_amd import prefix_tree as pt
    out = {"stream": f"rag_stream(4), {n_requests} requests, first 64 only warm the tree", "window": 4}
    rows = []
    for cap in capacities:
        rows.append({"capacity_chunks": cap,
                     "lookahead": pt.hit_ratio_under_capacity(4, capacity_chunks=cap, lookahead=True,
                                                              n_requests=n_requests),
                     "lru": pt.hit_ratio_under_capacity(4, capacity_chunks=cap, lookahead=False,
                                                        n_requests=n_requests)})
    out["by_capacity"] = rows
    out["unbounded"] = pt.hit_ratio_under_capacity(4, capacity_chunks=None, lookahead=False, n_requests=n_requests)
    return out


def measure_append_sweep(token_counts=(1024, 4096, 16384, 65536, 131072), Hkv=8, d=128, reps=20,
                         ragged_seq=300):
    """The scatter (pcr_append_kv) from 1k to 128k new tokens (8 MiB to 1 GiB of K+V
    moved: every row read once and written once), each size timed back to back after a
    warm-up, for two slot lists: `sizes`, the tokens in block order over a random order
    of the pool's blocks (every 8-slot chunk of V aligned with the workgroups' tiles);
    `ragged`, sequences of `ragged_seq` new tokens laid end to end, each starting at a
    block of its own (random blocks), so that the tiles of the token stream start
    inside the sequences' chunks, as in a ragged batch."""
    import torch
    from paper_2603_23049_amd import pcr
    bs = 16
    s = torch.cuda.current_stream()
    g = torch.Generator(device="cuda").manual_seed(17)

    def timed(T, nb, slots):
        pool = pcr.KVPool(torch.zeros((nb, Hkv, bs * d), dtype=torch.int16, device="cuda"),
                          torch.zeros((nb, Hkv, bs * d), dtype=torch.int16, device="cuda"), Hkv, d)
        k = torch.randint(-32768, 32767, (T, Hkv, d), dtype=torch.int16, device="cuda", generator=g)
        v = torch.randint(-32768, 32767, (T, Hkv, d), dtype=torch.int16, device="cuda", generator=g)
        fn = lambda: pcr.append_kv(pool, k, v, slots, stream=s)
        warm_up(fn, 30.0)
        a, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(s)
        for _ in range(reps):
            fn()
        e.record(s)
        e.synchronize()
        ms = a.elapsed_time(e) / reps
        nbytes = append_bytes(T, Hkv, d)
        del pool, k, v
        return {"T": T, "bytes": nbytes, "ms": ms, "GBps": nbytes / ms / 1e6, "frac_hbm": nbytes / ms / 1e6 / HBM_PEAK_GBS}

    out, ragged = [], []
    for T in token_counts:
        nb = -(-T // bs)
        perm = torch.randperm(nb, device="cuda", generator=g).to(torch.int32)
        slots = (perm.repeat_interleave(bs)[:T] * bs + torch.arange(T, device="cuda", dtype=torch.int32) % bs)
        out.append(timed(T, nb, slots.to(torch.int32).contiguous()))
        per_seq = -(-ragged_seq // bs)
        n_seq = -(-T // ragged_seq)
        nbr = n_seq * per_seq
        blocks = torch.randperm(nbr, device="cuda", generator=g).to(torch.int32)
        idx = torch.arange(T, device="cuda", dtype=torch.int32)
        pos = idx % ragged_seq
        slots_r = blocks[(idx // ragged_seq) * per_seq + pos // bs] * bs + pos % bs
        ragged.append(timed(T, nbr, slots_r.to(torch.int32).contiguous()))
        del perm, slots, blocks, slots_r
    torch.cuda.synchronize()
    # reference: a plain device copy of 256 MiB (read + write, like the append)
    src = torch.ones(256 << 20, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    fn = lambda: dst.copy_(src)
    warm_up(fn, 30.0)
    a, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record(s)
    for _ in range(reps):
        fn()
    e.record(s)
    e.synchronize()
    copy_gbps = 2 * (256 << 20) / (a.elapsed_time(e) / reps) / 1e6
    del src, dst
    return {"sizes": out, "asymptotic_GBps": out[-1]["GBps"], "asymptotic_frac_hbm": out[-1]["frac_hbm"],
            "device_copy_256MiB_GBps": copy_gbps, "asymptotic_frac_of_device_copy": out[-1]["GBps"] / copy_gbps,
            "ragged": ragged, "ragged_seq_tokens": ragged_seq, "ragged_asymptotic_GBps": ragged[-1]["GBps"]}


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=20,
                    help="untimed steps first; the warm-up then continues until at least 500 ms of sustained "
                         "work has passed (the GPU clock needs that long to settle), whatever this says")
    ap.add_argument("--workload", default="l70b_pipe80",
                    help="headline step: one layer (append + attention) of this workload")
    ap.add_argument("--step-only", action="store_true",
                    help="only the headline step (the run the kernel-trace and counter profiles take)")
    ap.add_argument("--no-pipeline", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-load", action="store_true", help="skip the host-to-pool copy measurements")
    ap.add_argument("--no-extra", action="store_true",
                    help="skip the secondary lines (8B layer, RAG mix, decode, SSD tier, offload, append sweep, "
                         "hit ratios) and the 80-layer and compute-bound pipelines")
    ap.add_argument("--pipeline-method", default="auto", choices=("auto", "kernel_pull", "staged", "dma_per_block"),
                    help="the pipelines' load method: pull kernel, staged (copy-engine transfers into a "
                         "workspace, then a scatter kernel on a third stream) or per-block copies; auto "
                         "measures the first two and reports staged for compute-bound pipelines (a layer's "
                         "compute at least its load), the pull kernel for copy-bound ones")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a 256 MiB device copy (reference for the traffic counters)")
    ap.add_argument("--decode-only", action="store_true",
                    help="only run the decode-step measurement and print its JSON")
    ap.add_argument("--append-sweep-only", action="store_true",
                    help="only run the append (scatter) sweep and print its JSON")
    ap.add_argument("--pipeline-only", action="store_true",
                    help="only run one pipeline (--pipeline-workload) with its isolated load and compute times, "
                         "per load method, and print its JSON")
    ap.add_argument("--pipeline-workload", default="l8b_pipe32",
                    choices=("l8b_pipe32", "l8b_pipe32_s6144", "l70b_pipe80"))
    ap.add_argument("--pipeline-reps", type=int, default=3,
                    help="with --pipeline-only: untimed pipeline runs per load method after one warm-up run")
    ap.add_argument("--no-clocks", action="store_true",
                    help="skip the amd-smi clock samples under the attention (never taken under a profiler)")
    args = ap.parse_args(argv)
    if args.step_only:
        args.no_pipeline = args.no_cpu_baseline = args.no_load = args.no_extra = args.no_clocks = True

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU only (the path exchanges nothing between GPUs: each GPU "
              "would run its own share of the batch); run with --gpus 1", file=sys.stderr)
        return 2

    # The oracle's library must be current before the GPU is initialised: building it
    # starts the compiler, which a process that has touched the GPU may not do.
    if not args.no_cpu_baseline and not (args.copy_calibration or args.decode_only or args.pipeline_only
                                         or args.append_sweep_only):
        from oracle import build as obuild
        obuild.ensure_built()
    # Under a profiler the tool library has initialised the GPU before this script runs,
    # so no other program may be started from here: no clock sampling then.
    under_profiler = (any(k.startswith(("ROCPROF", "ROCP_")) for k in os.environ)
                      or "rocprof" in os.environ.get("LD_PRELOAD", ""))
    sampler = (ClockSampler() if not (args.copy_calibration or args.decode_only or args.pipeline_only or args.no_clocks
                                      or args.append_sweep_only or under_profiler) else None)
    try:
        return _main(args, sampler)
    finally:
        if sampler:
            sampler.close()


def _step_record(batch, st):
    flops = attention_flops(batch.prefix_lens, batch.suffix_lens, batch.num_q_heads, batch.head_dim)
    return {"workload": batch.name, "ms_per_step": st["step_ms"], "attn_ms": st["attn_b2b_ms"],
            "attn_ms_in_step_events": st["attn_ms"], "append_ms": st["append_ms"], "flops": flops,
            "step_tflops": flops / (st["step_ms"] * 1e-3) / 1e12,
            "attn_tflops": flops / (st["attn_b2b_ms"] * 1e-3) / 1e12,
            "attn_frac": flops / (st["attn_b2b_ms"] * 1e-3) / 1e12 / MFMA_BF16_PEAK_TFLOPS,
            "attn_timing": "back to back, one event pair over the launches", "warmup_calls": st["warmup_calls"],
            "graph_ms_per_step": st["graph_step_ms"],
            "graph_step_tflops": flops / (st["graph_step_ms"] * 1e-3) / 1e12 if st["graph_step_ms"] else None}


def _main(args, sampler):
    import torch
    from paper_2603_23049_amd import pcr, synth
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    pcr.lib()   # fails loudly if libpcr.so is missing
    if args.copy_calibration:
        copy_calibration()
        return 0
    if args.decode_only:
        print(json.dumps({"decode": measure_decode(), "decode_ragged": measure_decode_ragged(),
                          "mixed": measure_mixed(), "mixed_256": measure_mixed(n_dec=256)}), flush=True)
        return 0
    if args.append_sweep_only:
        print(json.dumps({"append_sweep": measure_append_sweep()}), flush=True)
        return 0
    if args.pipeline_only:
        pb = workload(args.pipeline_workload)
        pst = measure_step(pb, args.steps, args.warmup)
        pcr.prefill_attn_set_schedule("key_halves")   # the pull-load pipeline's attention schedule
        try:
            pst_keys = measure_step(pb, args.steps, args.warmup)
        finally:
            pcr.prefill_attn_set_schedule("auto")
        pld = measure_load(pb)
        dist = pb.num_layers if pb.name == "l8b_pipe32" else 6
        lbp = _setup_pipeline(pb, dist)
        res = {}
        for m in (("kernel_pull", "staged") if args.pipeline_method == "auto" else (args.pipeline_method,)):
            if m == "staged":
                sg = pld["dma_staged"]
                res[m] = measure_pipeline(pb, m, sg["ms"], pst["step_ms"], staged_stages=(sg["transfer_ms"],
                                                                                            sg["scatter_ms"]),
                                          reps=args.pipeline_reps, distinct=dist, layers_bp=lbp)
            else:
                res[m] = measure_pipeline(pb, m, pld[m]["ms"], pst_keys["step_ms"], reps=args.pipeline_reps,
                                          distinct=dist, layers_bp=lbp)
        print(json.dumps({"pipeline": res, "load": pld, "step_ms": pst["step_ms"],
                          "step_ms_key_halves": pst_keys["step_ms"]}), flush=True)
        return 0

    batch = workload(args.workload)
    flops = attention_flops(batch.prefix_lens, batch.suffix_lens, batch.num_q_heads, batch.head_dim)
    _say(f"[bench] step: {args.workload} warmup={args.warmup} (+ at least 500 ms) steps={args.steps}")
    # (no graph replays in the profiled run: its trace's timed window is the attention
    # dispatches before the last 20)
    st = measure_step(batch, args.steps, args.warmup, graph=not args.step_only)
    value = flops / (st["step_ms"] * 1e-3) / 1e12
    attn_tflops = flops / (st["attn_ms"] * 1e-3) / 1e12
    app_b = append_bytes(batch.T, batch.num_kv_heads, batch.head_dim)
    _say(f"[bench] step {st['step_ms']:.4f} ms, attention {st['attn_ms']:.4f} ms = {attn_tflops:.1f} TFLOP/s")
    clocks = None
    if sampler is not None:
        _say("[bench] clocks under the attention (amd-smi)")
        clocks = measure_clock_hold(batch, sampler)

    method = "kernel_pull"
    pipeline_methods = ("kernel_pull", "staged") if args.pipeline_method == "auto" else (args.pipeline_method,)
    load = None
    if not args.no_load:
        _say("[bench] load")
        load = measure_load(batch)
    pipelines = {}
    extra = {}
    if not args.no_extra:
        b8 = synth.l8b_layer()
        _say("[bench] secondary step: l8b_layer")
        extra["l8b_layer"] = _step_record(b8, measure_step(b8, args.steps, args.warmup, min_warm_ms=300.0))
    if not args.no_pipeline:
        if load is None:
            load = measure_load(batch)
        todo = [(batch, st, load, synth.pipeline_data_sets(batch.num_layers, 6))]
        if not args.no_extra:
            for pb in (synth.l8b_pipe32(), synth.l8b_pipe32(suffix=6144)):
                todo.append((pb, None, None, None))
        for pb, pst, pld, _ in todo:
            distinct = pb.num_layers if pb.name == "l8b_pipe32" else 6
            _say(f"[bench] pipeline: {pb.name} ({pb.num_layers} layers, {distinct} distinct layer data sets)")
            pst = pst or measure_step(pb, 20, 3, min_warm_ms=200.0)
            # the pipelines with pull loads run their attention with key halves (the
            # default schedule may take row halves for this size): their isolated step
            # is measured that way too
            pcr.prefill_attn_set_schedule("key_halves")
            try:
                pst_keys = measure_step(pb, 20, 3, min_warm_ms=200.0)
            finally:
                pcr.prefill_attn_set_schedule("auto")
            pld = pld or measure_load(pb, reps=4)
            lbp = _setup_pipeline(pb, distinct)
            recs = {}
            for m in pipeline_methods:
                if m == "staged":
                    sg = pld["dma_staged"]
                    step = pst
                    rec = measure_pipeline(pb, "staged", sg["ms"], step["step_ms"], reps=2, distinct=distinct,
                                           staged_stages=(sg["transfer_ms"], sg["scatter_ms"]), layers_bp=lbp)
                    rec["load_GBps"] = sg["GBps"]
                else:
                    step = pst_keys
                    rec = measure_pipeline(pb, m, pld[method]["ms"], step["step_ms"], reps=2, distinct=distinct,
                                           layers_bp=lbp)
                    rec["load_GBps"] = pld[method]["GBps"]
                rec["attn_tflops"] = attention_flops(pb.prefix_lens, pb.suffix_lens, pb.num_q_heads,
                                                     pb.head_dim) / (step["attn_b2b_ms"] * 1e-3) / 1e12
                recs[m] = rec
            del lbp
            torch.cuda.synchronize()
            # the pipeline's figure: the requested load method, or with "auto" the staged loads
            # when a layer's compute is at least its load (compute-bound: the pull kernel's
            # workgroups would slow the attention) and the pull kernel otherwise (copy-bound:
            # the link sets the time, and the pull kernel adds no scatter); both are reported
            if args.pipeline_method == "auto":
                pick = "staged" if pst["step_ms"] >= pld[method]["ms"] else "kernel_pull"
            else:
                pick = args.pipeline_method
            pipelines[pb.name] = dict(recs[pick], methods_measured={m: {k: r[k] for k in (
                "total_ms", "bound_makespan_ms", "exposed_ms_per_layer", "exposed_frac_of_load",
                "exposed_over_min_frac_of_load", "sum_compute_ms_in_pipeline")} for m, r in recs.items()})
            if pb.name == "l8b_pipe32_s6144":
                _say(f"[bench] offload: {pb.name}")
                off, osrc, odst = measure_offload(pb)
                extra["offload"] = off
                for om, key in (("dma_staged", "dma_staged"), ("kernel_pull", "kernel_push")):
                    _say(f"[bench] pipeline with offload ({key}): {pb.name}")
                    pipelines[f"{pb.name}_offload_{key}"] = measure_pipeline_offload(
                        pb, method, pld[method]["ms"], pst_keys["step_ms"], off[key]["ms"], osrc, odst,
                        offload_method=om, distinct=6)
                _say(f"[bench] pipeline with staged loads and offload (dma_staged): {pb.name}")
                sg = pld["dma_staged"]
                pipelines[f"{pb.name}_staged_offload_dma_staged"] = measure_pipeline_offload(
                    pb, "staged", sg["ms"], pst["step_ms"], off["dma_staged"]["ms"], osrc, odst,
                    offload_method="dma_staged", distinct=6, staged_stages=(sg["transfer_ms"], sg["scatter_ms"]))
    if not args.no_extra:
        _say("[bench] SSD tier: queue-window prefetch")
        extra["prefetch"] = measure_prefetch()
        _say("[bench] decode step")
        extra["decode"] = measure_decode()
        extra["decode_ragged"] = measure_decode_ragged()
        _say("[bench] mixed prefill + decode launches")
        extra["mixed"] = measure_mixed()
        extra["mixed_256"] = measure_mixed(n_dec=256)
        rb = workload("rag_mix")
        _say(f"[bench] rag_mix attention (T={rb.T})")
        rst = measure_step(rb, max(10, args.steps // 4), 3, min_warm_ms=200.0)
        rfl = attention_flops(rb.prefix_lens, rb.suffix_lens, rb.num_q_heads, rb.head_dim)
        extra["rag_mix"] = dict(_step_record(rb, rst), T=rb.T, hit_ratio=rb.extra["hit_ratio"],
                                load_bytes=load_bytes(rb.prefix_lens, rb.num_kv_heads, rb.head_dim))
        tb = synth.uniform_batch("l70b_tp8_shard", B=2, Hq=8, Hkv=1, d=128, p=15360, s=1024, pool_blocks=4096,
                                 seed=5)
        _say("[bench] one GPU's share of the 70B-shaped layer at tensor parallelism 8 (Hq 8, Hkv 1)")
        tst = measure_step(tb, max(20, args.steps // 2), 3, min_warm_ms=200.0)
        tld = measure_load(tb, reps=6)
        extra["tp8_shard"] = dict(_step_record(tb, tst), load_ms=tld["kernel_pull"]["ms"],
                                  load_GBps=tld["kernel_pull"]["GBps"], load_bytes=tld["bytes_per_layer"])
        _say("[bench] append sweep")
        extra["append_sweep"] = measure_append_sweep()
        _say("[bench] prefix-tree hit ratio under capacity (host)")
        extra["hit_ratio"] = hit_ratio_report()
    cpu = legs = None
    if not args.no_cpu_baseline:
        _say("[bench] cpu baseline (oracle)")
        cpu = cpu_baseline(batch)
        if not args.no_extra:
            _say("[bench] cpu baseline legs (oracle)")
            legs = cpu_baseline_legs(cpu)

    headline_pipe = pipelines.get(batch.name)
    rec = {
        "metric": "prefix-reuse prefill TFLOP/s + % MFMA peak; exposed KV-load ms/layer",
        "value": value,
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": st["step_ms"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": args.workload, "batch": batch.B, "num_q_heads": batch.num_q_heads,
                   "num_kv_heads": batch.num_kv_heads, "head_dim": batch.head_dim,
                   "prefix_len": batch.prefix_lens[0], "suffix_len": batch.suffix_lens[0],
                   "block_size": batch.block_size, "pool_blocks": batch.pool_blocks, "layers": batch.num_layers,
                   "step": "one layer: append + attention, prefix KV resident in HBM",
                   "warmup_calls": st["warmup_calls"]},
        "mfma_frac": value / MFMA_BF16_PEAK_TFLOPS,
        "roofline": {"bound": "mfma", "kernel": "prefill_attn_kernel", "achieved": attn_tflops,
                     "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s", "frac": attn_tflops / MFMA_BF16_PEAK_TFLOPS,
                     "traffic": measured_traffic(batch.name), "flops_per_launch": flops,
                     "avg_launch_ms": st["attn_ms"], "median_launch_ms": st["attn_ms_median"],
                     "launch_ms_range": [st["attn_ms_min"], st["attn_ms_max"]],
                     "back_to_back_launch_ms": st["attn_b2b_ms"],
                     "timed": "HIP events around each attention launch inside the timed steps",
                     "sampled_clock_mhz": clocks["gfx_mhz_mean"] if clocks else None,
                     "peak_at_sampled_clock": (MFMA_BF16_PEAK_TFLOPS * clocks["gfx_mhz_mean"] / 2400.0
                                               if clocks else None),
                     "frac_at_sampled_clock": (attn_tflops / (MFMA_BF16_PEAK_TFLOPS * clocks["gfx_mhz_mean"] / 2400.0)
                                               if clocks else None)},
        "clocks": clocks,
        "append": {"ms": st["append_ms"], "bytes": app_b, "GBps": app_b / st["append_ms"] / 1e6,
                   "frac_hbm": app_b / st["append_ms"] / 1e6 / HBM_PEAK_GBS},
        "load": load,
        "pipeline": headline_pipe,
        "pipelines": pipelines or None,
        "exposed_kv_load_ms_per_layer": headline_pipe["exposed_ms_per_layer"] if headline_pipe else None,
        "cpu_baseline": cpu,
        "cpu_baseline_legs": legs,
        "wall_s_timed": st["wall_s"],
        "wall_ms_per_step": st["wall_ms_per_step"],
        "graph_ms_per_step": st["graph_step_ms"],
    }
    rec.update({k: extra.get(k) for k in ("l8b_layer", "rag_mix", "tp8_shard", "offload", "decode", "decode_ragged", "mixed", "mixed_256",
                                          "prefetch",
                                          "append_sweep", "hit_ratio")})
    print(json.dumps(rec), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
