// Internal declarations shared by the libpcr translation units (not installed).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/pcr.h"

namespace pcr {

constexpr int kBlockSize = 16;   // tokens per pool block (the serving engine's block, Sec. 5)

// Records a formatted message as this thread's last error and returns `st`.
pcr_status fail(pcr_status st, const char *fmt, ...);
// Turns a HIP error into PCR_ERR_HIP with the call site named.
pcr_status hip_fail(hipError_t e, const char *what);

// Up to this many (src, dst) block pairs travel in one pull-kernel launch as
// kernel arguments (so no device copy of the host lists is needed).
constexpr int kPullPairsPerLaunch = 480;

struct PullArgs {
    int32_t n;
    int32_t src[kPullPairsPerLaunch];
    int32_t dst[kPullPairsPerLaunch];
};

// Kernel launchers (kv_move.hip).
hipError_t launch_append_kv(const pcr_kv_pool &pool, const void *k_new, const void *v_new,
                            const int32_t *slot_mapping, int32_t T, hipStream_t s);
hipError_t launch_gather_kv(const pcr_kv_pool &pool, const int32_t *block_tables, int32_t max_blocks,
                            const int32_t *starts, const int32_t *cu_out, int32_t B, int32_t total,
                            void *k_out, void *v_out, hipStream_t s);
hipError_t launch_pull_blocks(const void *host_k, const void *host_v, int64_t host_blocks,
                              void *pool_k, void *pool_v, int32_t pool_blocks, int64_t block_bytes,
                              const PullArgs &args, hipStream_t s);
hipError_t launch_device_blocks(const void *src_k, const void *src_v, int64_t src_blocks, void *dst_k, void *dst_v,
                                int64_t dst_blocks, int64_t block_bytes, const PullArgs &args, hipStream_t s);
hipError_t launch_push_blocks(const void *pool_k, const void *pool_v, int32_t pool_blocks, void *host_k,
                              void *host_v, int64_t host_blocks, int64_t block_bytes, const PullArgs &args,
                              hipStream_t s);

// Attention launcher (attn.hip).
// The lengths travel in the launches' arguments (the work map), taken from the host
// copies, which the caller guarantees equal the device arrays.
hipError_t launch_prefix_prefill_attn(const void *q, const pcr_kv_pool &pool,
                                      const int32_t *block_tables, int32_t max_blocks,
                                      const int32_t *host_prefix_lens, const int32_t *host_cu_suffix,
                                      int32_t B, int32_t num_q_heads, int32_t T, float sm_scale, void *out,
                                      hipStream_t s, int auto_schedule, int n_cu);
// Compute units of the current device (queried once per device).
pcr_status device_cu_count(int32_t *n_cu, const char *who);

// Decode attention (decode.hip). The key range of each (sequence, kv head) is cut
// into chunks of `chunk` keys, at most n_split per sequence. Without the context
// lengths (or when it does not shorten the chunks) the chunk follows from the
// largest context; with them, from the total count of keys (a ragged batch then
// gives its long sequences more chunks than its short ones). lds_merge: every
// sequence has n_split <= 4 chunks and they merge in LDS; otherwise chunks of one
// sequence merge through the workspace. bound_workspace_bytes covers every batch of
// B sequences with contexts up to max_context, under either rule.
struct DecodePlan {
    int32_t n_split;
    int32_t chunk;
    int32_t lds_merge;
    int32_t ws_wg_waves;   // waves per workgroup when chunks merge through the workspace
    int32_t k_streamed;    // every sequence of one length: K loads non-temporal
    int64_t workspace_bytes;
    int64_t bound_workspace_bytes;
};
// ctx: the host context lengths (NULL: plan from max_context alone); the rule by total
// keys is taken only when its workspace fits ws_limit bytes.
DecodePlan decode_plan(int32_t B, int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                       int32_t max_context, int32_t n_cu, const int32_t *ctx = nullptr, int64_t ws_limit = 0);
int decode_max_cols();
hipError_t launch_decode_attn(const void *q, const pcr_kv_pool &pool, const int32_t *block_tables,
                              int32_t max_blocks, const int32_t *context_lens, int32_t B, int32_t num_q_heads,
                              const DecodePlan &plan, float sm_scale, void *out, void *workspace, hipStream_t s);
// Size of the allocation-free decode entry point's per-device scratch (decode.hip),
// and its device address on the current device (taken with hipGetSymbolAddress on the
// first call per device, then reused).
constexpr int64_t kDecodeScratchBytes = PCR_DECODE_NOALLOC_SCRATCH_BYTES;
hipError_t decode_noalloc_scratch(void **ptr);

// The staged host-to-pool load (every check of pcr_load_kv_layer_staged) with its two
// halves on two streams: the copy-engine transfers into the workspace on dma_stream,
// then dma_done is recorded there, scatter_stream waits for it and runs the scatter
// into the pool. The workspace is free again once the scatter has run.
pcr_status load_staged_split(const pcr_host_kv *src, const int32_t *src_blocks, const pcr_kv_pool *dst,
                             const int32_t *dst_blocks, int32_t n, void *workspace, int64_t workspace_bytes,
                             hipStream_t dma_stream, hipStream_t scatter_stream, hipEvent_t dma_done);

// Size in bytes of one pool block of K (or V): block_size * num_kv_heads * head_dim bf16.
inline int64_t kv_block_bytes(int32_t block_size, int32_t num_kv_heads, int32_t head_dim)
{
    return (int64_t)block_size * num_kv_heads * head_dim * 2;
}

// Pool-to-host offload with any method (the staged one takes the workspace); used by
// the pipeline, which chooses the method per call.
pcr_status offload_with(const pcr_kv_pool *src, const int32_t *src_blocks, const pcr_host_kv *dst,
                        const int32_t *dst_blocks, int32_t n, pcr_load_method method, void *workspace,
                        int64_t workspace_bytes, void *stream);

// pcr_prefix_prefill_attn with a schedule preference: when the process-wide schedule
// is PCR_ATTN_SCHEDULE_AUTO, auto_schedule PCR_ATTN_SCHEDULE_KEY_HALVES takes key
// halves whatever the size (PCR_ATTN_SCHEDULE_AUTO: the size rule).
pcr_status prefix_prefill_attn(const void *q, const pcr_kv_pool *pool, const int32_t *block_tables,
                               int32_t max_blocks, const int32_t *prefix_lens, const int32_t *cu_suffix,
                               const int32_t *host_prefix_lens, const int32_t *host_cu_suffix, int32_t B,
                               int32_t num_q_heads, float sm_scale, void *out, void *stream, int auto_schedule);

// Rows of packed (token, head-in-group) queries one attention workgroup handles with
// key halves (the most row tiles any schedule launches per sequence).
int attn_rows_per_workgroup(int head_dim);
// Process-wide attention schedule (PCR_ATTN_SCHEDULE_*), read at each launch.
void attn_set_schedule(int schedule);

// Every argument check of pcr_prefix_prefill_attn, with no launch (errors name `who`);
// on success *T_out is the suffix token count (0: nothing to do).
pcr_status attn_check(const void *q, const pcr_kv_pool *pool, const int32_t *block_tables, int32_t max_blocks,
                      const int32_t *prefix_lens, const int32_t *cu_suffix, const int32_t *host_prefix_lens,
                      const int32_t *host_cu_suffix, int32_t B, int32_t num_q_heads, float sm_scale,
                      const void *out, const char *who, int64_t *T_out);

}  // namespace pcr
