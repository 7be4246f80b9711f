// Layer pipeline (Sec. 4.3 layer-wise overlap; Alg. 1 LayerwiseUpload, then
// WaitForUploadEvents before each layer's compute, and LayerwiseDownload).
//
// Every layer has its own pool, so the copy stream runs the loads back to back,
// each followed by an event; the compute stream waits for layer l's event and
// then runs layer l's append and attention. With an offload stream
// (the three-stream form of Sec. 5), that stream waits for layer l's compute and
// then copies the layer's new blocks to the host store. The copy stream first
// waits for everything already queued on the compute (and offload) stream, so a
// load never overwrites a pool that earlier work is still reading.
//
// The staged form splits each load in two: the copy engines move the layer's host
// blocks into a workspace slot (copy stream), and a scatter kernel on a third
// stream moves them from the slot into the pool. The host-link transfer then holds
// no compute unit while the attention runs, and with two or more slots the transfer
// of layer l+1 runs while layer l is scattered; the transfer into a slot waits for
// the scatter that last read it.
#include <algorithm>
#include <vector>

#include "pcr_internal.h"

namespace pcr {
namespace {

// Events are reused across calls on the same thread: a wait enqueued on a stream
// refers to the record that preceded it, so re-recording afterwards is safe.
struct EventPool {
    std::vector<hipEvent_t> ev;
    unsigned flags;
    explicit EventPool(unsigned f) : flags(f) {}
    // Events live until the process ends (destroying them from a thread-exit
    // destructor could run after the HIP runtime has shut down).
    hipError_t ensure(size_t n)
    {
        while (ev.size() < n) {
            hipEvent_t e;
            hipError_t r = hipEventCreateWithFlags(&e, flags);
            if (r != hipSuccess) return r;
            ev.push_back(e);
        }
        return hipSuccess;
    }
};

thread_local EventPool g_sync_events(hipEventDisableTiming);
thread_local EventPool g_timed_events(hipEventDefault);

float elapsed(hipEvent_t a, hipEvent_t b)
{
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, a, b) != hipSuccess) return -1.f;
    return ms;
}

}  // namespace
}  // namespace pcr

using namespace pcr;

namespace {

// The staged loads' workspace and scatter stream (pcr_pipeline_run_staged).
struct StagedLoads {
    char *ws;
    int64_t ws_bytes;
    hipStream_t scatter;
};

pcr_status run_pipeline(const pcr_layer_io *layers, const pcr_host_kv *offload_dst, int32_t n_layers,
                        const pcr_batch *batch, const int32_t *off_src, const int32_t *off_dst, int32_t n_off,
                        pcr_load_method method, pcr_load_method offload_method, void *workspace,
                        int64_t workspace_bytes, void *copy_stream, void *compute_stream, void *offload_stream,
                        bool with_offload, const StagedLoads *staged, float *timing_ms, const char *who)
{
    if (n_layers < 0) return fail(PCR_ERR_INVALID_ARG, "%s: n_layers < 0", who);
    if (n_layers == 0) return PCR_OK;
    if (!layers || !batch) return fail(PCR_ERR_INVALID_ARG, "%s: NULL layers or batch", who);
    if (copy_stream == compute_stream)
        return fail(PCR_ERR_INVALID_ARG, "%s: copy and compute streams must differ", who);
    // staged loads: slots of one layer's K and V blocks each, in the caller's workspace
    int64_t slot_bytes = 0;
    int64_t n_slots = 0;
    if (staged) {
        if (staged->scatter == static_cast<hipStream_t>(copy_stream) ||
            staged->scatter == static_cast<hipStream_t>(compute_stream))
            return fail(PCR_ERR_INVALID_ARG, "%s: the scatter stream must differ from the other two", who);
        if (batch->n_pairs < 0) return fail(PCR_ERR_INVALID_ARG, "%s: n_pairs < 0", who);
        const pcr_kv_pool &p0 = layers[0].pool;
        if (p0.block_size <= 0 || p0.num_kv_heads <= 0 || p0.head_dim <= 0)
            return fail(PCR_ERR_INVALID_ARG, "%s: layer 0's pool has a non-positive shape", who);
        for (int32_t l = 1; l < n_layers; ++l)
            if (layers[l].pool.block_size != p0.block_size || layers[l].pool.num_kv_heads != p0.num_kv_heads ||
                layers[l].pool.head_dim != p0.head_dim)
                return fail(PCR_ERR_INVALID_ARG, "%s: layer %d's pool shape differs from layer 0's", who, l);
        slot_bytes = 2 * (int64_t)batch->n_pairs * kv_block_bytes(p0.block_size, p0.num_kv_heads, p0.head_dim);
        if (slot_bytes > 0) {
            if (!staged->ws) return fail(PCR_ERR_INVALID_ARG, "%s: NULL workspace", who);
            if ((uintptr_t)staged->ws & 15)
                return fail(PCR_ERR_INVALID_ARG, "%s: workspace must be 16-byte aligned", who);
            n_slots = staged->ws_bytes / slot_bytes;
            if (n_slots < 1)
                return fail(PCR_ERR_INVALID_ARG, "%s: workspace of %lld bytes, one layer's load needs %lld", who,
                            (long long)staged->ws_bytes, (long long)slot_bytes);
            n_slots = std::min<int64_t>(n_slots, n_layers);
        }
    }
    if (with_offload) {
        if (offload_stream == compute_stream || offload_stream == copy_stream)
            return fail(PCR_ERR_INVALID_ARG, "%s: the offload stream must differ from the other two", who);
        if (n_off < 0) return fail(PCR_ERR_INVALID_ARG, "%s: n_off < 0", who);
        if (n_off > 0 && (!offload_dst || !off_src || !off_dst))
            return fail(PCR_ERR_INVALID_ARG, "%s: NULL offload argument", who);
        if (staged && staged->scatter == static_cast<hipStream_t>(offload_stream))
            return fail(PCR_ERR_INVALID_ARG, "%s: the scatter and offload streams must differ", who);
    }
    // Every layer needs a pool of its own: nothing orders layer l+1's load (copy stream)
    // after layer l's compute (compute stream), so two layers sharing pool memory would
    // have one layer's load overwrite blocks the other's attention is still reading.
    {
        std::vector<const void *> bufs;
        bufs.reserve(2 * (size_t)n_layers);
        for (int32_t l = 0; l < n_layers; ++l) {   // NULL pools are reported by the checks below
            if (layers[l].pool.k) bufs.push_back(layers[l].pool.k);
            if (layers[l].pool.v) bufs.push_back(layers[l].pool.v);
        }
        std::sort(bufs.begin(), bufs.end());
        if (std::adjacent_find(bufs.begin(), bufs.end()) != bufs.end())
            return fail(PCR_ERR_INVALID_ARG, "%s: two layers (or a layer's K and V) share a pool buffer; every "
                        "layer needs its own pool", who);
    }
    // The attention's arguments, batch-wide and per layer, are checked before anything is
    // queued, so a bad scale, head count or length table leaves the streams untouched.
    for (int32_t l = 0; l < n_layers; ++l) {
        int64_t T = 0;
        pcr_status st = attn_check(layers[l].q, &layers[l].pool, batch->block_tables, batch->max_blocks,
                                   batch->prefix_lens, batch->cu_suffix, batch->host_prefix_lens,
                                   batch->host_cu_suffix, batch->B, batch->num_q_heads, batch->sm_scale,
                                   layers[l].out, who, &T);
        if (st) return st;
    }
    hipStream_t cs = static_cast<hipStream_t>(copy_stream);
    hipStream_t ks = static_cast<hipStream_t>(compute_stream);
    hipStream_t os = static_cast<hipStream_t>(offload_stream);
    const bool timed = timing_ms != nullptr;
    const size_t n = (size_t)n_layers;

    // events: [0] start, [1] offload-stream start, [2] scatter-stream start, then per
    // layer: load start, loaded, compute start, compute end, offload start, offload
    // end, transfers done (timed); loaded, compute end, transfers done (untimed)
    EventPool &pool = timed ? g_timed_events : g_sync_events;
    const size_t per = timed ? 7 : 3;
    hipError_t e = pool.ensure(3 + per * n);
    if (e != hipSuccess) return hip_fail(e, "pcr_pipeline_run: hipEventCreate");
    hipEvent_t ev_start = pool.ev[0], ev_ostart = pool.ev[1], ev_sstart = pool.ev[2];
    auto ev = [&](size_t l, int k) { return pool.ev[3 + per * l + k]; };
    auto ev_loaded = [&](size_t l) { return ev(l, timed ? 1 : 0); };
    auto ev_cend = [&](size_t l) { return ev(l, timed ? 3 : 1); };
    auto ev_dma = [&](size_t l) { return ev(l, timed ? 6 : 2); };
    hipStream_t ss = staged ? staged->scatter : nullptr;

#define PCR_HIP(call, what)                          \
    do {                                             \
        hipError_t r_ = (call);                      \
        if (r_ != hipSuccess) return hip_fail(r_, what); \
    } while (0)

    PCR_HIP(hipEventRecord(ev_start, ks), "pcr_pipeline_run: record start");
    PCR_HIP(hipStreamWaitEvent(cs, ev_start, 0), "pcr_pipeline_run: copy waits for compute");
    if (with_offload) {
        PCR_HIP(hipEventRecord(ev_ostart, os), "pcr_pipeline_run: record offload start");
        PCR_HIP(hipStreamWaitEvent(cs, ev_ostart, 0), "pcr_pipeline_run: copy waits for offload");
    }
    if (staged) {
        // the first transfers wait for earlier scatters (which read the workspace), and
        // the scatters for earlier compute (which reads the pools)
        PCR_HIP(hipEventRecord(ev_sstart, ss), "pcr_pipeline_run: record scatter start");
        PCR_HIP(hipStreamWaitEvent(cs, ev_sstart, 0), "pcr_pipeline_run: copy waits for scatter");
        PCR_HIP(hipStreamWaitEvent(ss, ev_start, 0), "pcr_pipeline_run: scatter waits for compute");
        if (with_offload)   // the scatters write pools that earlier offloads may still read
            PCR_HIP(hipStreamWaitEvent(ss, ev_ostart, 0), "pcr_pipeline_run: scatter waits for offload");
    }
    // One layer at a time: its load, then its compute (and offload). The streams run as
    // far ahead as their events allow either way; queuing a layer's compute right after
    // its load lets the compute stream start once the first load is done, not only after
    // the host has queued every load (about 0.2 ms each with the pull kernel).
    for (size_t l = 0; l < n; ++l) {
        pcr_status st = PCR_OK;
        if (staged) {
            // slot l % n_slots was last read by the scatter of layer l - n_slots
            if (l >= (size_t)n_slots && n_slots > 0)
                PCR_HIP(hipStreamWaitEvent(cs, ev_loaded(l - (size_t)n_slots), 0),
                        "pcr_pipeline_run: transfer waits for its slot");
            if (timed) PCR_HIP(hipEventRecord(ev(l, 0), cs), "pcr_pipeline_run: record load start");
            char *slot = n_slots > 0 ? staged->ws + (int64_t)(l % (size_t)n_slots) * slot_bytes : staged->ws;
            st = load_staged_split(&layers[l].host, batch->src_blocks, &layers[l].pool, batch->dst_blocks,
                                   batch->n_pairs, slot, slot_bytes, cs, ss, ev_dma(l));
            if (st) return st;
            PCR_HIP(hipEventRecord(ev_loaded(l), ss), "pcr_pipeline_run: record loaded");
        } else {
            if (timed) PCR_HIP(hipEventRecord(ev(l, 0), cs), "pcr_pipeline_run: record load start");
            st = pcr_load_kv_layer_method(&layers[l].host, batch->src_blocks, &layers[l].pool, batch->dst_blocks,
                                          batch->n_pairs, method, copy_stream);
            if (st) return st;
            PCR_HIP(hipEventRecord(ev_loaded(l), cs), "pcr_pipeline_run: record loaded");
        }
        PCR_HIP(hipStreamWaitEvent(ks, ev_loaded(l), 0), "pcr_pipeline_run: compute waits for load");
        if (timed) PCR_HIP(hipEventRecord(ev(l, 2), ks), "pcr_pipeline_run: record compute start");
        st = pcr_append_kv(&layers[l].pool, layers[l].k_new, layers[l].v_new, batch->slot_mapping,
                                      batch->T, compute_stream);
        if (st) return st;
        // Beside pull-kernel loads the attention takes key halves: its shorter workgroups
        // let a load's copy workgroups onto a compute unit sooner.
        st = prefix_prefill_attn(layers[l].q, &layers[l].pool, batch->block_tables, batch->max_blocks,
                                 batch->prefix_lens, batch->cu_suffix, batch->host_prefix_lens,
                                 batch->host_cu_suffix, batch->B, batch->num_q_heads, batch->sm_scale,
                                 layers[l].out, compute_stream,
                                 staged ? PCR_ATTN_SCHEDULE_AUTO : PCR_ATTN_SCHEDULE_KEY_HALVES);
        if (st) return st;
        PCR_HIP(hipEventRecord(ev_cend(l), ks), "pcr_pipeline_run: record compute end");
        if (with_offload) {
            PCR_HIP(hipStreamWaitEvent(os, ev_cend(l), 0), "pcr_pipeline_run: offload waits for compute");
            if (timed) PCR_HIP(hipEventRecord(ev(l, 4), os), "pcr_pipeline_run: record offload start");
            st = offload_with(&layers[l].pool, off_src, &offload_dst[l], off_dst, n_off, offload_method, workspace,
                              workspace_bytes, offload_stream);
            if (st) return st;
            if (timed) PCR_HIP(hipEventRecord(ev(l, 5), os), "pcr_pipeline_run: record offload end");
        }
    }
    if (!timed) return PCR_OK;

    hipEvent_t last = with_offload ? ev(n - 1, 5) : ev_cend(n - 1);
    PCR_HIP(hipEventSynchronize(last), "pcr_pipeline_run: synchronize");
    double sum_compute = 0.0;
    const size_t stride = with_offload ? 6 : 4;
    for (size_t l = 0; l < n; ++l) {
        const float comp = elapsed(ev(l, 2), ev_cend(l));
        timing_ms[stride * l + 0] = elapsed(ev(l, 0), ev_loaded(l));
        timing_ms[stride * l + 1] = comp;
        timing_ms[stride * l + 2] = elapsed(l == 0 ? ev_start : ev_cend(l - 1), ev(l, 2));
        timing_ms[stride * l + 3] = elapsed(ev_start, ev_cend(l));
        if (with_offload) {
            timing_ms[stride * l + 4] = elapsed(ev(l, 4), ev(l, 5));
            timing_ms[stride * l + 5] = elapsed(ev_start, ev(l, 5));
        }
        sum_compute += comp;
    }
    timing_ms[stride * n] = elapsed(ev_start, last);
    timing_ms[stride * n + 1] = (float)sum_compute;
    if (with_offload) timing_ms[stride * n + 2] = elapsed(ev_start, ev_cend(n - 1));
#undef PCR_HIP
    return PCR_OK;
}

}  // namespace

extern "C" pcr_status pcr_pipeline_run(const pcr_layer_io *layers, int32_t n_layers, const pcr_batch *batch,
                                       pcr_load_method method, void *copy_stream, void *compute_stream,
                                       float *timing_ms)
{
    return run_pipeline(layers, nullptr, n_layers, batch, nullptr, nullptr, 0, method, PCR_LOAD_AUTO, nullptr, 0,
                        copy_stream, compute_stream, nullptr, false, nullptr, timing_ms, "pcr_pipeline_run");
}

extern "C" pcr_status pcr_pipeline_run_staged(const pcr_layer_io *layers, int32_t n_layers, const pcr_batch *batch,
                                              void *workspace, int64_t workspace_bytes, void *copy_stream,
                                              void *scatter_stream, void *compute_stream, float *timing_ms)
{
    StagedLoads st{static_cast<char *>(workspace), workspace_bytes, static_cast<hipStream_t>(scatter_stream)};
    return run_pipeline(layers, nullptr, n_layers, batch, nullptr, nullptr, 0, PCR_LOAD_DMA_STAGED, PCR_LOAD_AUTO,
                        nullptr, 0, copy_stream, compute_stream, nullptr, false, &st, timing_ms,
                        "pcr_pipeline_run_staged");
}

extern "C" pcr_status pcr_pipeline_run_offload_staged(
    const pcr_layer_io *layers, const pcr_host_kv *offload_dst, int32_t n_layers, const pcr_batch *batch,
    const int32_t *off_src, const int32_t *off_dst, int32_t n_off, pcr_load_method offload_method,
    void *offload_workspace, int64_t offload_workspace_bytes, void *load_workspace, int64_t load_workspace_bytes,
    void *copy_stream, void *scatter_stream, void *compute_stream, void *offload_stream, float *timing_ms)
{
    StagedLoads st{static_cast<char *>(load_workspace), load_workspace_bytes,
                   static_cast<hipStream_t>(scatter_stream)};
    return run_pipeline(layers, offload_dst, n_layers, batch, off_src, off_dst, n_off, PCR_LOAD_DMA_STAGED,
                        offload_method, offload_workspace, offload_workspace_bytes, copy_stream, compute_stream,
                        offload_stream, true, &st, timing_ms, "pcr_pipeline_run_offload_staged");
}

extern "C" pcr_status pcr_pipeline_run_offload(const pcr_layer_io *layers, const pcr_host_kv *offload_dst,
                                               int32_t n_layers, const pcr_batch *batch, const int32_t *off_src,
                                               const int32_t *off_dst, int32_t n_off, pcr_load_method method,
                                               pcr_load_method offload_method, void *workspace,
                                               int64_t workspace_bytes, void *copy_stream, void *compute_stream,
                                               void *offload_stream, float *timing_ms)
{
    return run_pipeline(layers, offload_dst, n_layers, batch, off_src, off_dst, n_off, method, offload_method,
                        workspace, workspace_bytes, copy_stream, compute_stream, offload_stream, true, nullptr,
                        timing_ms, "pcr_pipeline_run_offload");
}
