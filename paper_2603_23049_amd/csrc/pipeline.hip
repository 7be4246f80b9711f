// Two-stream layer pipeline (Sec. 4.3 layer-wise overlap; Alg. 1 LayerwiseUpload
// then WaitForUploadEvents before each layer's compute).
//
// Every layer has its own pool, so all loads are enqueued up front on the copy
// stream, each followed by an event; the compute stream waits for layer l's
// event and then runs layer l's append and attention. The copy stream first
// waits for everything already queued on the compute stream, so a load never
// overwrites a pool that earlier compute is still reading.
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

extern "C" pcr_status pcr_pipeline_run(const pcr_layer_io *layers, int32_t n_layers, const pcr_batch *batch,
                                       pcr_load_method method, void *copy_stream, void *compute_stream,
                                       float *timing_ms)
{
    const char *who = "pcr_pipeline_run";
    if (n_layers < 0) return fail(PCR_ERR_INVALID_ARG, "%s: n_layers < 0", who);
    if (n_layers == 0) return PCR_OK;
    if (!layers || !batch) return fail(PCR_ERR_INVALID_ARG, "%s: NULL layers or batch", who);
    if (copy_stream == compute_stream)
        return fail(PCR_ERR_INVALID_ARG, "%s: copy and compute streams must differ", who);
    hipStream_t cs = static_cast<hipStream_t>(copy_stream);
    hipStream_t ks = static_cast<hipStream_t>(compute_stream);
    const bool timed = timing_ms != nullptr;
    const size_t n = (size_t)n_layers;

    // timed: [0] start, [1+l] load start, [1+n+l] loaded, [1+2n+l] compute start, [1+3n+l] compute end
    EventPool &pool = timed ? g_timed_events : g_sync_events;
    hipError_t e = pool.ensure(timed ? 1 + 4 * n : 1 + n);
    if (e != hipSuccess) return hip_fail(e, "pcr_pipeline_run: hipEventCreate");
    hipEvent_t ev_start = pool.ev[0];
    auto ev_lstart = [&](size_t l) { return pool.ev[1 + l]; };
    auto ev_loaded = [&](size_t l) { return timed ? pool.ev[1 + n + l] : pool.ev[1 + l]; };
    auto ev_cstart = [&](size_t l) { return pool.ev[1 + 2 * n + l]; };
    auto ev_cend = [&](size_t l) { return pool.ev[1 + 3 * n + l]; };

#define PCR_HIP(call, what)                          \
    do {                                             \
        hipError_t r_ = (call);                      \
        if (r_ != hipSuccess) return hip_fail(r_, what); \
    } while (0)

    PCR_HIP(hipEventRecord(ev_start, ks), "pcr_pipeline_run: record start");
    PCR_HIP(hipStreamWaitEvent(cs, ev_start, 0), "pcr_pipeline_run: copy waits for compute");
    for (size_t l = 0; l < n; ++l) {
        if (timed) PCR_HIP(hipEventRecord(ev_lstart(l), cs), "pcr_pipeline_run: record load start");
        pcr_status st = pcr_load_kv_layer_method(&layers[l].host, batch->src_blocks, &layers[l].pool,
                                                 batch->dst_blocks, batch->n_pairs, method, copy_stream);
        if (st) return st;
        PCR_HIP(hipEventRecord(ev_loaded(l), cs), "pcr_pipeline_run: record loaded");
    }
    for (size_t l = 0; l < n; ++l) {
        PCR_HIP(hipStreamWaitEvent(ks, ev_loaded(l), 0), "pcr_pipeline_run: compute waits for load");
        if (timed) PCR_HIP(hipEventRecord(ev_cstart(l), ks), "pcr_pipeline_run: record compute start");
        pcr_status st = pcr_append_kv(&layers[l].pool, layers[l].k_new, layers[l].v_new, batch->slot_mapping,
                                      batch->T, compute_stream);
        if (st) return st;
        st = pcr_prefix_prefill_attn(layers[l].q, &layers[l].pool, batch->block_tables, batch->max_blocks,
                                     batch->prefix_lens, batch->cu_suffix, batch->host_prefix_lens,
                                     batch->host_cu_suffix, batch->B, batch->num_q_heads, batch->sm_scale,
                                     layers[l].out, compute_stream);
        if (st) return st;
        if (timed) PCR_HIP(hipEventRecord(ev_cend(l), ks), "pcr_pipeline_run: record compute end");
    }
    if (!timed) return PCR_OK;

    PCR_HIP(hipEventSynchronize(ev_cend(n - 1)), "pcr_pipeline_run: synchronize");
    double sum_compute = 0.0;
    for (size_t l = 0; l < n; ++l) {
        const float load = elapsed(ev_lstart(l), ev_loaded(l));
        const float comp = elapsed(ev_cstart(l), ev_cend(l));
        const float wait = elapsed(l == 0 ? ev_start : ev_cend(l - 1), ev_cstart(l));
        timing_ms[4 * l + 0] = load;
        timing_ms[4 * l + 1] = comp;
        timing_ms[4 * l + 2] = wait;
        timing_ms[4 * l + 3] = elapsed(ev_start, ev_cend(l));
        sum_compute += comp;
    }
    timing_ms[4 * n] = elapsed(ev_start, ev_cend(n - 1));
    timing_ms[4 * n + 1] = (float)sum_compute;
#undef PCR_HIP
    return PCR_OK;
}
