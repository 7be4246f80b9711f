// libpcr host runtime: argument validation, the batch planner, the three
// host-to-pool copy methods, and the two-stream layer pipeline.
#include <dlfcn.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <atomic>
#include <mutex>
#include <unordered_map>
#include <unordered_set>
#include <vector>

#include "pcr_internal.h"

namespace pcr {

static thread_local char g_err[512] = "";

pcr_status fail(pcr_status st, const char *fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return st;
}

pcr_status hip_fail(hipError_t e, const char *what)
{
    return fail(PCR_ERR_HIP, "%s: %s (%d)", what, hipGetErrorString(e), (int)e);
}

namespace {

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

pcr_status check_layout(int32_t block_size, int32_t num_kv_heads, int32_t head_dim, const char *who)
{
    if (block_size <= 0 || num_kv_heads <= 0 || head_dim <= 0)
        return fail(PCR_ERR_INVALID_ARG, "%s: block_size, num_kv_heads and head_dim must be positive", who);
    if (block_size != kBlockSize)
        return fail(PCR_ERR_UNSUPPORTED, "%s: block_size %d unsupported (only %d)", who, block_size, kBlockSize);
    if (head_dim != 64 && head_dim != 128)
        return fail(PCR_ERR_UNSUPPORTED, "%s: head_dim %d unsupported (64 or 128)", who, head_dim);
    return PCR_OK;
}

pcr_status check_pool(const pcr_kv_pool *pool, const char *who)
{
    if (!pool) return fail(PCR_ERR_INVALID_ARG, "%s: pool is NULL", who);
    if (!pool->k || !pool->v) return fail(PCR_ERR_INVALID_ARG, "%s: pool k/v pointer is NULL", who);
    if (pool->num_blocks <= 0) return fail(PCR_ERR_INVALID_ARG, "%s: pool has no blocks", who);
    pcr_status st = check_layout(pool->block_size, pool->num_kv_heads, pool->head_dim, who);
    if (st) return st;
    if (((uintptr_t)pool->k | (uintptr_t)pool->v) & 15)
        return fail(PCR_ERR_INVALID_ARG, "%s: pool k/v must be 16-byte aligned", who);
    return PCR_OK;
}

int64_t block_bytes(int32_t block_size, int32_t Hkv, int32_t d) { return kv_block_bytes(block_size, Hkv, d); }

// A host range is acceptable for the copy methods if HIP knows it as pinned host memory.
pcr_status check_pinned(const void *ptr, int64_t bytes, const char *who, void **device_alias)
{
    const char *bytes_p = static_cast<const char *>(ptr);
    const void *ends[2] = {ptr, bytes_p + (bytes > 0 ? bytes - 1 : 0)};
    for (int k = 0; k < 2; ++k) {
        hipPointerAttribute_t attr;
        memset(&attr, 0, sizeof attr);
        hipError_t e = hipPointerGetAttributes(&attr, ends[k]);
        if (e != hipSuccess) {
            (void)hipGetLastError();
            return fail(PCR_ERR_NOT_PINNED, "%s: host KV store is not pinned memory (%s)", who,
                        hipGetErrorString(e));
        }
        if (attr.type != hipMemoryTypeHost)
            return fail(PCR_ERR_NOT_PINNED, "%s: host KV store is not pinned host memory (type %d)", who,
                        (int)attr.type);
        if (k == 0 && device_alias) {
            *device_alias = attr.devicePointer;
            if (!attr.devicePointer)
                return fail(PCR_ERR_NOT_PINNED, "%s: host KV store has no device mapping", who);
        }
    }
    return PCR_OK;
}

// hipMemcpyBatchAsync exists only in newer HIP runtimes. The library binds to
// whichever runtime the process already uses (e.g. one bundled with a
// framework), so the entry point is looked up at run time in that runtime.
typedef hipError_t (*memcpy_batch_fn)(void **, void **, size_t *, size_t, hipMemcpyAttributes *, size_t *,
                                      size_t, size_t *, hipStream_t);

// The batched copy takes at least one attribute (the first applying from copy 0):
// sources read in stream order, no location hints (plain pinned host and device
// pointers), no flags.
hipMemcpyAttributes stream_ordered_copy()
{
    hipMemcpyAttributes a;
    memset(&a, 0, sizeof a);
    a.srcAccessOrder = hipMemcpySrcAccessOrderStream;
    return a;
}

memcpy_batch_fn memcpy_batch()
{
    static memcpy_batch_fn fn = [] {
        void *h = dlopen("libamdhip64.so.7", RTLD_LAZY | RTLD_NOLOAD);
        memcpy_batch_fn f = h ? reinterpret_cast<memcpy_batch_fn>(dlsym(h, "hipMemcpyBatchAsync")) : nullptr;
        return f;
    }();
    return fn;
}

}  // namespace
}  // namespace pcr

using namespace pcr;

extern "C" {

const char *pcr_last_error(void) { return g_err; }

const char *pcr_version(void) { return "libpcr 0.1 gfx950"; }

pcr_status pcr_plan(int32_t B, const int32_t *prefix_lens, const int32_t *suffix_lens,
                    const int32_t *block_tables, int32_t max_blocks,
                    const int32_t *host_blocks, int32_t max_host_blocks, int32_t block_size,
                    int32_t *src_blocks, int32_t *dst_blocks, int32_t cap_pairs, int32_t *n_pairs,
                    int32_t *slot_mapping, int32_t *cu_suffix)
{
    g_err[0] = 0;
    if (B < 0) return fail(PCR_ERR_INVALID_ARG, "pcr_plan: B < 0");
    if (block_size <= 0) return fail(PCR_ERR_INVALID_ARG, "pcr_plan: block_size must be positive");
    if (!n_pairs || !cu_suffix || (B > 0 && (!prefix_lens || !suffix_lens || !block_tables)))
        return fail(PCR_ERR_INVALID_ARG, "pcr_plan: NULL argument");
    const int64_t bs = block_size;
    int64_t need_pairs = 0, T = 0;
    for (int b = 0; b < B; ++b) {
        if (prefix_lens[b] < 0 || suffix_lens[b] < 0)
            return fail(PCR_ERR_INVALID_ARG, "pcr_plan: sequence %d has a negative length", b);
        const int64_t nb = ceil_div((int64_t)prefix_lens[b] + suffix_lens[b], bs);
        if (nb > max_blocks)
            return fail(PCR_ERR_INVALID_ARG, "pcr_plan: sequence %d needs %lld blocks, table has %d", b,
                        (long long)nb, max_blocks);
        if (ceil_div(prefix_lens[b], bs) > max_host_blocks)
            return fail(PCR_ERR_INVALID_ARG, "pcr_plan: sequence %d needs more host blocks than given", b);
        need_pairs += ceil_div(prefix_lens[b], bs);
        T += suffix_lens[b];
    }
    if (T > INT32_MAX) return fail(PCR_ERR_INVALID_ARG, "pcr_plan: too many new tokens");
    if (need_pairs > 0 && (!host_blocks || !src_blocks || !dst_blocks))
        return fail(PCR_ERR_INVALID_ARG, "pcr_plan: NULL host_blocks or pair arrays");
    if (T > 0 && !slot_mapping) return fail(PCR_ERR_INVALID_ARG, "pcr_plan: NULL slot_mapping");

    // Load list: sequence by sequence, logical block ascending; a repeated pair once.
    std::unordered_map<int32_t, int32_t> src_of_dst;         // pool block -> host block
    std::unordered_map<int32_t, int32_t> loader_of_dst;      // pool block -> loading sequence, -2 if several
    int32_t np = 0;
    for (int b = 0; b < B; ++b) {
        const int64_t npb = ceil_div(prefix_lens[b], bs);
        for (int64_t j = 0; j < npb; ++j) {
            const int32_t s_blk = host_blocks[(int64_t)b * max_host_blocks + j];
            const int32_t d_blk = block_tables[(int64_t)b * max_blocks + j];
            if (s_blk < 0 || d_blk < 0)
                return fail(PCR_ERR_INVALID_ARG, "pcr_plan: sequence %d prefix block %lld has no host or pool block",
                            b, (long long)j);
            auto lo = loader_of_dst.find(d_blk);
            if (lo == loader_of_dst.end()) loader_of_dst[d_blk] = b;
            else if (lo->second != b) lo->second = -2;
            auto it = src_of_dst.find(d_blk);
            if (it != src_of_dst.end()) {
                if (it->second != s_blk)
                    return fail(PCR_ERR_INVALID_ARG, "pcr_plan: pool block %d is loaded from two host blocks", d_blk);
                continue;
            }
            src_of_dst[d_blk] = s_blk;
            if (np >= cap_pairs) return fail(PCR_ERR_INVALID_ARG, "pcr_plan: cap_pairs %d too small", cap_pairs);
            src_blocks[np] = s_blk;
            dst_blocks[np] = d_blk;
            ++np;
        }
    }
    // Slots of the new tokens.
    std::unordered_set<int64_t> used;
    used.reserve((size_t)T * 2 + 1);
    int64_t k = 0;
    cu_suffix[0] = 0;
    for (int b = 0; b < B; ++b) {
        const int64_t p = prefix_lens[b];
        for (int64_t i = 0; i < suffix_lens[b]; ++i) {
            const int64_t t = p + i;
            const int32_t blk = block_tables[(int64_t)b * max_blocks + t / bs];
            if (blk < 0)
                return fail(PCR_ERR_INVALID_ARG, "pcr_plan: sequence %d token %lld has no pool block", b, (long long)t);
            auto lo = loader_of_dst.find(blk);
            if (lo != loader_of_dst.end() && lo->second != b)
                return fail(PCR_ERR_INVALID_ARG,
                            "pcr_plan: sequence %d token %lld lands in a block another sequence loads", b,
                            (long long)t);
            const int64_t slot = (int64_t)blk * bs + t % bs;
            if (slot > INT32_MAX) return fail(PCR_ERR_INVALID_ARG, "pcr_plan: slot overflows int32");
            if (!used.insert(slot).second)
                return fail(PCR_ERR_INVALID_ARG, "pcr_plan: two new tokens share slot %lld", (long long)slot);
            slot_mapping[k++] = (int32_t)slot;
        }
        cu_suffix[b + 1] = cu_suffix[b] + suffix_lens[b];
    }
    *n_pairs = np;
    return PCR_OK;
}

}  // extern "C"

namespace {

// Workspace check of the staged copies: 2 * n blocks (K then V), 16-byte aligned.
pcr_status check_workspace(void *ws, int64_t ws_bytes, int32_t n, int64_t bb, const char *who)
{
    if (!ws) return fail(PCR_ERR_INVALID_ARG, "%s: the staged method needs a workspace", who);
    if ((uintptr_t)ws & 15) return fail(PCR_ERR_INVALID_ARG, "%s: workspace must be 16-byte aligned", who);
    if (ws_bytes < 2 * (int64_t)n * bb)
        return fail(PCR_ERR_INVALID_ARG, "%s: workspace of %lld bytes, %lld needed", who, (long long)ws_bytes,
                    (long long)(2 * (int64_t)n * bb));
    return PCR_OK;
}

// Copy-engine transfers of the runs of consecutive host blocks between the host
// store and workspace slots 0..n-1 (K region then V region of the workspace).
pcr_status staged_dma(char *hk, char *hv, char *ws, const int32_t *host_blocks, int32_t n, int64_t bb,
                      bool to_host, hipStream_t s, const char *who)
{
    char *wk = ws, *wv = ws + (int64_t)n * bb;
    int32_t i = 0;
    while (i < n) {
        int32_t j = i + 1;
        while (j < n && host_blocks[j] == host_blocks[j - 1] + 1) ++j;
        const int64_t bytes = (int64_t)(j - i) * bb, h = (int64_t)host_blocks[i] * bb, w = (int64_t)i * bb;
        const hipMemcpyKind kind = to_host ? hipMemcpyDeviceToHost : hipMemcpyHostToDevice;
        hipError_t e = to_host ? hipMemcpyAsync(hk + h, wk + w, bytes, kind, s) : hipMemcpyAsync(wk + w, hk + h, bytes, kind, s);
        if (e == hipSuccess)
            e = to_host ? hipMemcpyAsync(hv + h, wv + w, bytes, kind, s) : hipMemcpyAsync(wv + w, hv + h, bytes, kind, s);
        if (e != hipSuccess) return hip_fail(e, who);
        i = j;
    }
    return PCR_OK;
}

// Kernel copies between listed pool blocks and workspace slots, in slices.
pcr_status staged_kernel(const pcr_kv_pool *pool, char *ws, const int32_t *pool_blocks, int32_t n, int64_t bb,
                         bool pool_to_ws, hipStream_t s, const char *who)
{
    char *wk = ws, *wv = ws + (int64_t)n * bb;
    for (int32_t off = 0; off < n; off += kPullPairsPerLaunch) {
        PullArgs a;
        a.n = std::min<int32_t>(kPullPairsPerLaunch, n - off);
        for (int32_t k = 0; k < a.n; ++k) {
            a.src[k] = pool_to_ws ? pool_blocks[off + k] : off + k;
            a.dst[k] = pool_to_ws ? off + k : pool_blocks[off + k];
        }
        hipError_t e = pool_to_ws
            ? launch_device_blocks(pool->k, pool->v, pool->num_blocks, wk, wv, n, bb, a, s)
            : launch_device_blocks(wk, wv, n, pool->k, pool->v, pool->num_blocks, bb, a, s);
        if (e != hipSuccess) return hip_fail(e, who);
    }
    return PCR_OK;
}

// scatter_stream / dma_done: for the staged method only, optionally run the scatter on
// a second stream: dma_done is recorded on copy_stream after the transfers, and the
// scatter stream waits for it (the pipeline's staged form).
pcr_status load_impl(const pcr_host_kv *src, const int32_t *src_blocks, const pcr_kv_pool *dst,
                     const int32_t *dst_blocks, int32_t n, pcr_load_method method, void *ws, int64_t ws_bytes,
                     void *copy_stream, hipStream_t scatter_stream = nullptr, hipEvent_t dma_done = nullptr)
{
    g_err[0] = 0;
    const char *who = "pcr_load_kv_layer";
    if (n < 0) return fail(PCR_ERR_INVALID_ARG, "%s: n < 0", who);
    if (!src || !dst) return fail(PCR_ERR_INVALID_ARG, "%s: NULL src or dst", who);
    pcr_status st = check_pool(dst, who);
    if (st) return st;
    if (!src->k || !src->v) return fail(PCR_ERR_INVALID_ARG, "%s: host k/v pointer is NULL", who);
    st = check_layout(src->block_size, src->num_kv_heads, src->head_dim, who);
    if (st) return st;
    if (src->block_size != dst->block_size || src->num_kv_heads != dst->num_kv_heads ||
        src->head_dim != dst->head_dim)
        return fail(PCR_ERR_INVALID_ARG, "%s: host store and pool shapes differ", who);
    if (method < PCR_LOAD_AUTO || method > PCR_LOAD_DMA_STAGED)
        return fail(PCR_ERR_INVALID_ARG, "%s: unknown method %d", who, (int)method);
    if (n == 0) return PCR_OK;
    if (!src_blocks || !dst_blocks) return fail(PCR_ERR_INVALID_ARG, "%s: NULL block list", who);
    if (src->num_blocks <= 0) return fail(PCR_ERR_INVALID_ARG, "%s: host store has no blocks", who);
    {
        std::vector<char> seen((size_t)dst->num_blocks, 0);
        for (int32_t i = 0; i < n; ++i) {
            if (src_blocks[i] < 0 || src_blocks[i] >= src->num_blocks)
                return fail(PCR_ERR_INVALID_ARG, "%s: src block %d (pair %d) outside host store of %lld", who,
                            src_blocks[i], i, (long long)src->num_blocks);
            if (dst_blocks[i] < 0 || dst_blocks[i] >= dst->num_blocks)
                return fail(PCR_ERR_INVALID_ARG, "%s: dst block %d (pair %d) outside pool of %d", who,
                            dst_blocks[i], i, dst->num_blocks);
            if (seen[dst_blocks[i]]++)
                return fail(PCR_ERR_INVALID_ARG, "%s: dst block %d named twice", who, dst_blocks[i]);
        }
    }
    const int64_t bb = block_bytes(dst->block_size, dst->num_kv_heads, dst->head_dim);
    const int64_t host_bytes = src->num_blocks * bb;
    void *dk = nullptr, *dv = nullptr;
    st = check_pinned(src->k, host_bytes, who, &dk);
    if (st) return st;
    st = check_pinned(src->v, host_bytes, who, &dv);
    if (st) return st;

    hipStream_t s = static_cast<hipStream_t>(copy_stream);
    const char *hk = static_cast<const char *>(src->k);
    const char *hv = static_cast<const char *>(src->v);
    char *pk = static_cast<char *>(dst->k);
    char *pv = static_cast<char *>(dst->v);
    if (method == PCR_LOAD_AUTO) method = PCR_LOAD_KERNEL_PULL;

    if (method == PCR_LOAD_DMA_STAGED) {
        st = check_workspace(ws, ws_bytes, n, bb, who);
        if (st) return st;
        st = staged_dma(const_cast<char *>(hk), const_cast<char *>(hv), static_cast<char *>(ws), src_blocks, n, bb,
                        false, s, "pcr_load_kv_layer: hipMemcpyAsync");
        if (st) return st;
        if (dma_done) {
            hipError_t e = hipEventRecord(dma_done, s);
            if (e == hipSuccess) e = hipStreamWaitEvent(scatter_stream, dma_done, 0);
            if (e != hipSuccess) return hip_fail(e, "pcr_load_kv_layer: scatter stream waits for the transfers");
            s = scatter_stream;
        }
        return staged_kernel(dst, static_cast<char *>(ws), dst_blocks, n, bb, false, s,
                             "pcr_load_kv_layer: scatter kernel launch");
    }
    if (method == PCR_LOAD_DMA_PER_BLOCK) {
        for (int32_t i = 0; i < n; ++i) {
            hipError_t e = hipMemcpyAsync(pk + dst_blocks[i] * bb, hk + (int64_t)src_blocks[i] * bb, bb,
                                          hipMemcpyHostToDevice, s);
            if (e == hipSuccess)
                e = hipMemcpyAsync(pv + dst_blocks[i] * bb, hv + (int64_t)src_blocks[i] * bb, bb,
                                   hipMemcpyHostToDevice, s);
            if (e != hipSuccess) return hip_fail(e, "pcr_load_kv_layer: hipMemcpyAsync");
        }
        return PCR_OK;
    }
    if (method == PCR_LOAD_DMA_BATCH) {
        // Merge runs where both source and destination blocks are consecutive.
        std::vector<void *> dsts, srcs;
        std::vector<size_t> sizes;
        dsts.reserve(2 * n);
        srcs.reserve(2 * n);
        sizes.reserve(2 * n);
        for (int kv = 0; kv < 2; ++kv) {
            const char *h = kv ? hv : hk;
            char *p = kv ? pv : pk;
            int32_t i = 0;
            while (i < n) {
                int32_t j = i + 1;
                while (j < n && src_blocks[j] == src_blocks[j - 1] + 1 && dst_blocks[j] == dst_blocks[j - 1] + 1) ++j;
                dsts.push_back(p + (int64_t)dst_blocks[i] * bb);
                srcs.push_back(const_cast<char *>(h) + (int64_t)src_blocks[i] * bb);
                sizes.push_back((size_t)((j - i) * bb));
                i = j;
            }
        }
        memcpy_batch_fn batch = memcpy_batch();
        if (!batch)
            return fail(PCR_ERR_UNSUPPORTED, "%s: this HIP runtime has no hipMemcpyBatchAsync", who);
        size_t fail_idx = 0;
        hipMemcpyAttributes attr = stream_ordered_copy();
        size_t attr_first = 0;   // the one attribute applies from copy 0 on
        hipError_t e = batch(dsts.data(), srcs.data(), sizes.data(), dsts.size(), &attr, &attr_first, 1, &fail_idx, s);
        if (e != hipSuccess) return hip_fail(e, "pcr_load_kv_layer: hipMemcpyBatchAsync");
        return PCR_OK;
    }
    // PCR_LOAD_KERNEL_PULL: block lists travel as kernel arguments, in slices.
    for (int32_t off = 0; off < n; off += kPullPairsPerLaunch) {
        PullArgs a;
        a.n = std::min<int32_t>(kPullPairsPerLaunch, n - off);
        memcpy(a.src, src_blocks + off, sizeof(int32_t) * a.n);
        memcpy(a.dst, dst_blocks + off, sizeof(int32_t) * a.n);
        hipError_t e = launch_pull_blocks(dk, dv, src->num_blocks, dst->k, dst->v, dst->num_blocks, bb, a, s);
        if (e != hipSuccess) return hip_fail(e, "pcr_load_kv_layer: pull kernel launch");
    }
    return PCR_OK;
}

}  // namespace

extern "C" {

pcr_status pcr_plan_offload(int32_t B, const int32_t *prefix_lens, const int32_t *suffix_lens,
                            const int32_t *block_tables, int32_t max_blocks, int32_t block_size,
                            int32_t chunk_tokens, int32_t first_dst_block,
                            int32_t *src_blocks, int32_t *dst_blocks, int32_t cap, int32_t *n_pairs)
{
    g_err[0] = 0;
    const char *who = "pcr_plan_offload";
    if (!n_pairs) return fail(PCR_ERR_INVALID_ARG, "%s: n_pairs is NULL", who);
    *n_pairs = 0;
    if (B < 0 || cap < 0 || first_dst_block < 0) return fail(PCR_ERR_INVALID_ARG, "%s: negative count", who);
    if (B == 0) return PCR_OK;
    if (!prefix_lens || !suffix_lens || !block_tables)
        return fail(PCR_ERR_INVALID_ARG, "%s: NULL input array", who);
    if (block_size <= 0 || chunk_tokens <= 0 || chunk_tokens % block_size)
        return fail(PCR_ERR_INVALID_ARG, "%s: chunk_tokens %d is not a positive multiple of block_size %d", who,
                    chunk_tokens, block_size);
    const int64_t per_chunk = chunk_tokens / block_size;
    int64_t k = 0;
    for (int32_t b = 0; b < B; ++b) {
        const int64_t p = prefix_lens[b], s = suffix_lens[b];
        if (p < 0 || s < 0) return fail(PCR_ERR_INVALID_ARG, "%s: sequence %d has a negative length", who, b);
        const int64_t c0 = ceil_div(p, chunk_tokens), c1 = (p + s) / chunk_tokens;   // whole chunks in [p, p+s)
        for (int64_t c = c0; c < c1; ++c) {
            for (int64_t j = 0; j < per_chunk; ++j) {
                const int64_t lb = c * per_chunk + j;
                const int32_t blk = lb < max_blocks ? block_tables[(int64_t)b * max_blocks + lb] : -1;
                if (blk < 0)
                    return fail(PCR_ERR_INVALID_ARG, "%s: sequence %d logical block %lld has no pool block", who, b,
                                (long long)lb);
                if (k >= cap) return fail(PCR_ERR_INVALID_ARG, "%s: more than cap=%d pairs", who, cap);
                if (first_dst_block + k > INT32_MAX)
                    return fail(PCR_ERR_INVALID_ARG, "%s: host block ids overflow int32", who);
                src_blocks[k] = blk;
                dst_blocks[k] = (int32_t)(first_dst_block + k);
                ++k;
            }
        }
    }
    *n_pairs = (int32_t)k;
    return PCR_OK;
}

}  // extern "C"

namespace {

pcr_status offload_impl(const pcr_kv_pool *src, const int32_t *src_blocks, const pcr_host_kv *dst,
                        const int32_t *dst_blocks, int32_t n, pcr_load_method method, void *ws, int64_t ws_bytes,
                        void *stream)
{
    g_err[0] = 0;
    const char *who = "pcr_offload_kv_layer";
    if (n < 0) return fail(PCR_ERR_INVALID_ARG, "%s: n < 0", who);
    if (!src || !dst) return fail(PCR_ERR_INVALID_ARG, "%s: NULL src or dst", who);
    pcr_status st = check_pool(src, who);
    if (st) return st;
    if (!dst->k || !dst->v) return fail(PCR_ERR_INVALID_ARG, "%s: host k/v pointer is NULL", who);
    st = check_layout(dst->block_size, dst->num_kv_heads, dst->head_dim, who);
    if (st) return st;
    if (src->block_size != dst->block_size || src->num_kv_heads != dst->num_kv_heads ||
        src->head_dim != dst->head_dim)
        return fail(PCR_ERR_INVALID_ARG, "%s: pool and host store shapes differ", who);
    if (method < PCR_LOAD_AUTO || method > PCR_LOAD_DMA_STAGED)
        return fail(PCR_ERR_INVALID_ARG, "%s: unknown method %d", who, (int)method);
    if (n == 0) return PCR_OK;
    if (!src_blocks || !dst_blocks) return fail(PCR_ERR_INVALID_ARG, "%s: NULL block list", who);
    if (dst->num_blocks <= 0) return fail(PCR_ERR_INVALID_ARG, "%s: host store has no blocks", who);
    {
        std::vector<char> seen((size_t)dst->num_blocks, 0);
        for (int32_t i = 0; i < n; ++i) {
            if (src_blocks[i] < 0 || src_blocks[i] >= src->num_blocks)
                return fail(PCR_ERR_INVALID_ARG, "%s: src block %d (pair %d) outside pool of %d", who, src_blocks[i],
                            i, src->num_blocks);
            if (dst_blocks[i] < 0 || dst_blocks[i] >= dst->num_blocks)
                return fail(PCR_ERR_INVALID_ARG, "%s: dst block %d (pair %d) outside host store of %lld", who,
                            dst_blocks[i], i, (long long)dst->num_blocks);
            if (seen[dst_blocks[i]]++)
                return fail(PCR_ERR_INVALID_ARG, "%s: dst block %d named twice", who, dst_blocks[i]);
        }
    }
    const int64_t bb = block_bytes(src->block_size, src->num_kv_heads, src->head_dim);
    const int64_t host_bytes = dst->num_blocks * bb;
    void *dk = nullptr, *dv = nullptr;
    st = check_pinned(dst->k, host_bytes, who, &dk);
    if (st) return st;
    st = check_pinned(dst->v, host_bytes, who, &dv);
    if (st) return st;

    hipStream_t s = static_cast<hipStream_t>(stream);
    char *hk = static_cast<char *>(const_cast<void *>(dst->k));
    char *hv = static_cast<char *>(const_cast<void *>(dst->v));
    const char *pk = static_cast<const char *>(src->k);
    const char *pv = static_cast<const char *>(src->v);
    if (method == PCR_LOAD_AUTO) method = ws ? PCR_LOAD_DMA_STAGED : PCR_LOAD_KERNEL_PULL;
    if (method == PCR_LOAD_DMA_STAGED) {
        st = check_workspace(ws, ws_bytes, n, bb, who);
        if (st) return st;
        st = staged_kernel(src, static_cast<char *>(ws), src_blocks, n, bb, true, s,
                           "pcr_offload_kv_layer: gather kernel launch");
        if (st) return st;
        return staged_dma(hk, hv, static_cast<char *>(ws), dst_blocks, n, bb, true, s,
                          "pcr_offload_kv_layer: hipMemcpyAsync");
    }
    if (method == PCR_LOAD_DMA_PER_BLOCK) {
        for (int32_t i = 0; i < n; ++i) {
            hipError_t e = hipMemcpyAsync(hk + (int64_t)dst_blocks[i] * bb, pk + (int64_t)src_blocks[i] * bb, bb,
                                          hipMemcpyDeviceToHost, s);
            if (e == hipSuccess)
                e = hipMemcpyAsync(hv + (int64_t)dst_blocks[i] * bb, pv + (int64_t)src_blocks[i] * bb, bb,
                                   hipMemcpyDeviceToHost, s);
            if (e != hipSuccess) return hip_fail(e, "pcr_offload_kv_layer: hipMemcpyAsync");
        }
        return PCR_OK;
    }
    if (method == PCR_LOAD_DMA_BATCH) {
        memcpy_batch_fn batch = memcpy_batch();
        if (!batch) return fail(PCR_ERR_UNSUPPORTED, "%s: this HIP runtime has no hipMemcpyBatchAsync", who);
        std::vector<void *> dsts, srcs;
        std::vector<size_t> sizes;
        for (int kv = 0; kv < 2; ++kv) {
            char *h = kv ? hv : hk;
            const char *p = kv ? pv : pk;
            int32_t i = 0;
            while (i < n) {
                int32_t j = i + 1;
                while (j < n && src_blocks[j] == src_blocks[j - 1] + 1 && dst_blocks[j] == dst_blocks[j - 1] + 1) ++j;
                dsts.push_back(h + (int64_t)dst_blocks[i] * bb);
                srcs.push_back(const_cast<char *>(p) + (int64_t)src_blocks[i] * bb);
                sizes.push_back((size_t)((j - i) * bb));
                i = j;
            }
        }
        size_t fail_idx = 0;
        hipMemcpyAttributes attr = stream_ordered_copy();
        size_t attr_first = 0;   // the one attribute applies from copy 0 on
        hipError_t e = batch(dsts.data(), srcs.data(), sizes.data(), dsts.size(), &attr, &attr_first, 1, &fail_idx, s);
        if (e != hipSuccess) return hip_fail(e, "pcr_offload_kv_layer: hipMemcpyBatchAsync");
        return PCR_OK;
    }
    for (int32_t off = 0; off < n; off += kPullPairsPerLaunch) {
        PullArgs a;
        a.n = std::min<int32_t>(kPullPairsPerLaunch, n - off);
        memcpy(a.src, src_blocks + off, sizeof(int32_t) * a.n);
        memcpy(a.dst, dst_blocks + off, sizeof(int32_t) * a.n);
        hipError_t e = launch_push_blocks(src->k, src->v, src->num_blocks, dk, dv, dst->num_blocks, bb, a, s);
        if (e != hipSuccess) return hip_fail(e, "pcr_offload_kv_layer: push kernel launch");
    }
    return PCR_OK;
}

}  // namespace

extern "C" {

pcr_status pcr_load_kv_layer_method(const pcr_host_kv *src, const int32_t *src_blocks, const pcr_kv_pool *dst,
                                    const int32_t *dst_blocks, int32_t n, pcr_load_method method,
                                    void *copy_stream)
{
    if (method == PCR_LOAD_DMA_STAGED)
        return fail(PCR_ERR_INVALID_ARG, "pcr_load_kv_layer: the staged method needs pcr_load_kv_layer_staged");
    return load_impl(src, src_blocks, dst, dst_blocks, n, method, nullptr, 0, copy_stream);
}

pcr_status pcr_load_kv_layer(const pcr_host_kv *src, const int32_t *src_blocks, const pcr_kv_pool *dst,
                             const int32_t *dst_blocks, int32_t n, void *copy_stream)
{
    return load_impl(src, src_blocks, dst, dst_blocks, n, PCR_LOAD_AUTO, nullptr, 0, copy_stream);
}

pcr_status pcr_load_kv_layer_staged(const pcr_host_kv *src, const int32_t *src_blocks, const pcr_kv_pool *dst,
                                    const int32_t *dst_blocks, int32_t n, void *workspace, int64_t workspace_bytes,
                                    void *stream)
{
    return load_impl(src, src_blocks, dst, dst_blocks, n, PCR_LOAD_DMA_STAGED, workspace, workspace_bytes, stream);
}

pcr_status pcr_offload_kv_layer_method(const pcr_kv_pool *src, const int32_t *src_blocks, const pcr_host_kv *dst,
                                       const int32_t *dst_blocks, int32_t n, pcr_load_method method, void *stream)
{
    if (method == PCR_LOAD_DMA_STAGED)
        return fail(PCR_ERR_INVALID_ARG,
                    "pcr_offload_kv_layer: the staged method needs pcr_offload_kv_layer_staged");
    return offload_impl(src, src_blocks, dst, dst_blocks, n, method, nullptr, 0, stream);
}

pcr_status pcr_offload_kv_layer(const pcr_kv_pool *src, const int32_t *src_blocks, const pcr_host_kv *dst,
                                const int32_t *dst_blocks, int32_t n, void *stream)
{
    return offload_impl(src, src_blocks, dst, dst_blocks, n, PCR_LOAD_AUTO, nullptr, 0, stream);
}

pcr_status pcr_offload_kv_layer_staged(const pcr_kv_pool *src, const int32_t *src_blocks, const pcr_host_kv *dst,
                                       const int32_t *dst_blocks, int32_t n, void *workspace, int64_t workspace_bytes,
                                       void *stream)
{
    return offload_impl(src, src_blocks, dst, dst_blocks, n, PCR_LOAD_DMA_STAGED, workspace, workspace_bytes,
                        stream);
}


pcr_status pcr_append_kv(const pcr_kv_pool *pool, const void *k_new, const void *v_new,
                         const int32_t *slot_mapping, int32_t T, void *stream)
{
    g_err[0] = 0;
    const char *who = "pcr_append_kv";
    pcr_status st = check_pool(pool, who);
    if (st) return st;
    if (T < 0) return fail(PCR_ERR_INVALID_ARG, "%s: T < 0", who);
    if (T == 0) return PCR_OK;
    if (!k_new || !v_new || !slot_mapping) return fail(PCR_ERR_INVALID_ARG, "%s: NULL argument", who);
    if (((uintptr_t)k_new | (uintptr_t)v_new) & 15)
        return fail(PCR_ERR_INVALID_ARG, "%s: k_new/v_new must be 16-byte aligned", who);
    hipError_t e = launch_append_kv(*pool, k_new, v_new, slot_mapping, T, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "pcr_append_kv: launch");
    return PCR_OK;
}

}  // extern "C"

namespace pcr {

pcr_status attn_check(const void *q, const pcr_kv_pool *pool, const int32_t *block_tables, int32_t max_blocks,
                      const int32_t *prefix_lens, const int32_t *cu_suffix, const int32_t *host_prefix_lens,
                      const int32_t *host_cu_suffix, int32_t B, int32_t num_q_heads, float sm_scale,
                      const void *out, const char *who, int64_t *T_out)
{
    *T_out = 0;
    pcr_status st = check_pool(pool, who);
    if (st) return st;
    if (B < 0) return fail(PCR_ERR_INVALID_ARG, "%s: B < 0", who);
    if (B == 0) return PCR_OK;
    if (!host_prefix_lens || !host_cu_suffix)
        return fail(PCR_ERR_INVALID_ARG, "%s: NULL host length arrays", who);
    if (num_q_heads <= 0 || num_q_heads % pool->num_kv_heads != 0)
        return fail(PCR_ERR_UNSUPPORTED, "%s: num_q_heads %d is not a positive multiple of num_kv_heads %d", who,
                    num_q_heads, pool->num_kv_heads);
    if (!(sm_scale > 0.f) || !(sm_scale < 1e30f)) return fail(PCR_ERR_INVALID_ARG, "%s: bad sm_scale", who);
    if (host_cu_suffix[0] != 0) return fail(PCR_ERR_INVALID_ARG, "%s: cu_suffix[0] must be 0", who);
    const int G = num_q_heads / pool->num_kv_heads;
    const int rows_per_wg = attn_rows_per_workgroup(pool->head_dim);
    int64_t tiles = 0;   // row tiles of all sequences at the finest schedule, one kv head
    for (int b = 0; b < B; ++b) {
        const int64_t s = (int64_t)host_cu_suffix[b + 1] - host_cu_suffix[b];
        if (s < 0 || host_prefix_lens[b] < 0)
            return fail(PCR_ERR_INVALID_ARG, "%s: sequence %d has a negative length", who, b);
        if (ceil_div((int64_t)host_prefix_lens[b] + s, kBlockSize) > max_blocks)
            return fail(PCR_ERR_INVALID_ARG, "%s: sequence %d needs more blocks than max_blocks %d", who, b,
                        max_blocks);
        tiles += ceil_div(s * G, rows_per_wg);
    }
    const int64_t T = host_cu_suffix[B];
    if (T == 0) return PCR_OK;
    if (T > INT32_MAX / num_q_heads) return fail(PCR_ERR_INVALID_ARG, "%s: T too large", who);
    if (!q || !out || !block_tables || !prefix_lens || !cu_suffix)
        return fail(PCR_ERR_INVALID_ARG, "%s: NULL device argument", who);
    if (((uintptr_t)q | (uintptr_t)out) & 15)
        return fail(PCR_ERR_INVALID_ARG, "%s: q/out must be 16-byte aligned", who);
    // (each launch's grid, at most every tile of every kv head, stays far inside the
    // 2^32 work items of one grid dimension)
    if (tiles * pool->num_kv_heads > (int64_t)1 << 22)
        return fail(PCR_ERR_UNSUPPORTED, "%s: batch too large", who);
    *T_out = T;
    return PCR_OK;
}

}  // namespace pcr

extern "C" {

pcr_status pcr_prefix_prefill_attn(const void *q, const pcr_kv_pool *pool, const int32_t *block_tables,
                                   int32_t max_blocks, const int32_t *prefix_lens, const int32_t *cu_suffix,
                                   const int32_t *host_prefix_lens, const int32_t *host_cu_suffix, int32_t B,
                                   int32_t num_q_heads, float sm_scale, void *out, void *stream)
{
    return pcr::prefix_prefill_attn(q, pool, block_tables, max_blocks, prefix_lens, cu_suffix, host_prefix_lens,
                                    host_cu_suffix, B, num_q_heads, sm_scale, out, stream, PCR_ATTN_SCHEDULE_AUTO);
}

static pcr_status decode_heads_ok(int32_t num_q_heads, int32_t num_kv_heads, const char *who)
{
    if (num_q_heads <= 0 || num_q_heads % num_kv_heads != 0)
        return fail(PCR_ERR_UNSUPPORTED, "%s: num_q_heads %d is not a positive multiple of num_kv_heads %d", who,
                    num_q_heads, num_kv_heads);
    if (num_q_heads / num_kv_heads > decode_max_cols())
        return fail(PCR_ERR_UNSUPPORTED, "%s: more than %d query heads per kv head (use pcr_prefix_prefill_attn "
                    "with one-token suffixes)", who, decode_max_cols());
    return PCR_OK;
}


pcr_status pcr_prefill_attn_set_schedule(int32_t schedule)
{
    g_err[0] = 0;
    if (schedule != PCR_ATTN_SCHEDULE_AUTO && schedule != PCR_ATTN_SCHEDULE_KEY_HALVES &&
        schedule != PCR_ATTN_SCHEDULE_ROW_HALVES)
        return fail(PCR_ERR_INVALID_ARG, "pcr_prefill_attn_set_schedule: unknown schedule %d", (int)schedule);
    attn_set_schedule(schedule);
    return PCR_OK;
}

pcr_status pcr_decode_attn_workspace_size(int32_t B, int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                                          int32_t max_context, int64_t *bytes)
{
    g_err[0] = 0;
    const char *who = "pcr_decode_attn_workspace_size";
    if (!bytes) return fail(PCR_ERR_INVALID_ARG, "%s: bytes is NULL", who);
    *bytes = 0;
    pcr_status st = check_layout(kBlockSize, num_kv_heads, head_dim, who);
    if (st) return st;
    st = decode_heads_ok(num_q_heads, num_kv_heads, who);
    if (st) return st;
    if (B < 0 || max_context < 0) return fail(PCR_ERR_INVALID_ARG, "%s: negative B or max_context", who);
    if (B == 0 || max_context == 0) return PCR_OK;
    int32_t n_cu = 0;
    st = device_cu_count(&n_cu, who);
    if (st) return st;
    *bytes = decode_plan(B, num_q_heads, num_kv_heads, head_dim, max_context, n_cu).bound_workspace_bytes;
    return PCR_OK;
}

}  // extern "C"

// Every host-side check of the decode entry points; on success *plan is the launch plan
// (plan->n_split == 0: nothing to do).
static pcr_status decode_check(const void *q, const pcr_kv_pool *pool, const int32_t *block_tables,
                               int32_t max_blocks, const int32_t *context_lens, const int32_t *host_context_lens,
                               int32_t B, int32_t num_q_heads, float sm_scale, const void *out, int64_t ws_limit,
                               const char *who, DecodePlan *plan)
{
    *plan = DecodePlan{};
    pcr_status st = check_pool(pool, who);
    if (st) return st;
    if (B < 0) return fail(PCR_ERR_INVALID_ARG, "%s: B < 0", who);
    if (B == 0) return PCR_OK;
    if (!host_context_lens) return fail(PCR_ERR_INVALID_ARG, "%s: NULL host length array", who);
    st = decode_heads_ok(num_q_heads, pool->num_kv_heads, who);
    if (st) return st;
    if (!(sm_scale > 0.f) || !(sm_scale < 1e30f)) return fail(PCR_ERR_INVALID_ARG, "%s: bad sm_scale", who);
    if (max_blocks <= 0) return fail(PCR_ERR_INVALID_ARG, "%s: max_blocks must be positive", who);
    if ((int64_t)B * num_q_heads > (int64_t)1 << 30)
        return fail(PCR_ERR_UNSUPPORTED, "%s: batch too large for one launch", who);
    int32_t max_ctx = 0;
    for (int b = 0; b < B; ++b) {
        const int32_t n = host_context_lens[b];
        if (n < 1) return fail(PCR_ERR_INVALID_ARG, "%s: sequence %d has no visible key", who, b);
        if (ceil_div(n, kBlockSize) > max_blocks)
            return fail(PCR_ERR_INVALID_ARG, "%s: sequence %d needs more blocks than max_blocks %d", who, b,
                        max_blocks);
        max_ctx = std::max(max_ctx, n);
    }
    if (!q || !out || !block_tables || !context_lens)
        return fail(PCR_ERR_INVALID_ARG, "%s: NULL device argument", who);
    if (((uintptr_t)q | (uintptr_t)out) & 15)
        return fail(PCR_ERR_INVALID_ARG, "%s: q/out must be 16-byte aligned", who);
    int32_t n_cu = 0;
    st = device_cu_count(&n_cu, who);
    if (st) return st;
    *plan = decode_plan(B, num_q_heads, pool->num_kv_heads, pool->head_dim, max_ctx, n_cu, host_context_lens,
                        ws_limit);
    return PCR_OK;
}

extern "C" {

pcr_status pcr_decode_attn_noalloc(const void *q, const pcr_kv_pool *pool, const int32_t *block_tables,
                                   int32_t max_blocks, const int32_t *context_lens,
                                   const int32_t *host_context_lens, int32_t B, int32_t num_q_heads,
                                   float sm_scale, void *out, void *stream)
{
    g_err[0] = 0;
    const char *who = "pcr_decode_attn_noalloc";
    DecodePlan plan;
    pcr_status st = decode_check(q, pool, block_tables, max_blocks, context_lens, host_context_lens, B, num_q_heads,
                                 sm_scale, out, kDecodeScratchBytes, who, &plan);
    if (st || plan.n_split == 0) return st;
    void *ws = nullptr;
    if (plan.workspace_bytes > 0) {
        if (plan.workspace_bytes > kDecodeScratchBytes)
            return fail(PCR_ERR_UNSUPPORTED, "%s: this batch needs %lld bytes of scratch; the allocation-free entry "
                        "point holds %lld (use pcr_decode_attn with a workspace)", who,
                        (long long)plan.workspace_bytes, (long long)kDecodeScratchBytes);
        hipError_t e = decode_noalloc_scratch(&ws);
        if (e != hipSuccess) return hip_fail(e, "pcr_decode_attn_noalloc: scratch address");
    }
    hipError_t e = launch_decode_attn(q, *pool, block_tables, max_blocks, context_lens, B, num_q_heads, plan,
                                      sm_scale, out, ws, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "pcr_decode_attn_noalloc: launch");
    return PCR_OK;
}

pcr_status pcr_decode_attn(const void *q, const pcr_kv_pool *pool, const int32_t *block_tables, int32_t max_blocks,
                           const int32_t *context_lens, const int32_t *host_context_lens, int32_t B,
                           int32_t num_q_heads, float sm_scale, void *out, void *workspace, int64_t workspace_bytes,
                           void *stream)
{
    g_err[0] = 0;
    const char *who = "pcr_decode_attn";
    DecodePlan plan;
    // The plan by total keys is taken when its workspace fits the one given and the
    // allocation-free entry point's scratch, so that both entry points make the same plan
    // for a batch whenever the workspace holds pcr_decode_attn_workspace_size bytes.
    const int64_t ws_limit = workspace ? std::min<int64_t>(workspace_bytes, kDecodeScratchBytes) : 0;
    pcr_status st = decode_check(q, pool, block_tables, max_blocks, context_lens, host_context_lens, B, num_q_heads,
                                 sm_scale, out, ws_limit, who, &plan);
    if (st || plan.n_split == 0) return st;
    if (plan.workspace_bytes > 0) {
        if (!workspace || workspace_bytes < plan.workspace_bytes)
            return fail(PCR_ERR_INVALID_ARG, "%s: this batch needs a workspace of %lld bytes (%lld given)", who,
                        (long long)plan.workspace_bytes, (long long)(workspace ? workspace_bytes : 0));
        if ((uintptr_t)workspace & 15)
            return fail(PCR_ERR_INVALID_ARG, "%s: workspace must be 16-byte aligned", who);
    }
    hipError_t e = launch_decode_attn(q, *pool, block_tables, max_blocks, context_lens, B, num_q_heads, plan,
                                      sm_scale, out, workspace, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "pcr_decode_attn: launch");
    return PCR_OK;
}

pcr_status pcr_gather_kv(const pcr_kv_pool *pool, const int32_t *block_tables, int32_t max_blocks,
                         const int32_t *starts, const int32_t *cu_out, int32_t B, int32_t total, void *k_out,
                         void *v_out, void *stream)
{
    g_err[0] = 0;
    const char *who = "pcr_gather_kv";
    pcr_status st = check_pool(pool, who);
    if (st) return st;
    if (B < 0 || total < 0) return fail(PCR_ERR_INVALID_ARG, "%s: negative B or total", who);
    if (B == 0 || total == 0) return PCR_OK;
    if (!block_tables || !starts || !cu_out || !k_out || !v_out)
        return fail(PCR_ERR_INVALID_ARG, "%s: NULL argument", who);
    if (max_blocks <= 0) return fail(PCR_ERR_INVALID_ARG, "%s: max_blocks must be positive", who);
    if (((uintptr_t)k_out | (uintptr_t)v_out) & 15)
        return fail(PCR_ERR_INVALID_ARG, "%s: outputs must be 16-byte aligned", who);
    hipError_t e = launch_gather_kv(*pool, block_tables, max_blocks, starts, cu_out, B, total, k_out, v_out,
                                    static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "pcr_gather_kv: launch");
    return PCR_OK;
}

}  // extern "C"

namespace pcr {

namespace {
std::atomic<int32_t> g_cu_count[64];   // per device id, 0 until queried
}  // namespace

pcr_status device_cu_count(int32_t *n_cu, const char *who)
{
    int dev = 0, cu = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, who);
    if (dev >= 0 && dev < 64 && (cu = g_cu_count[dev].load(std::memory_order_relaxed)) > 0) {
        *n_cu = cu;
        return PCR_OK;
    }
    e = hipDeviceGetAttribute(&cu, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return hip_fail(e, who);
    *n_cu = cu > 0 ? cu : 1;
    if (dev >= 0 && dev < 64) g_cu_count[dev].store(*n_cu, std::memory_order_relaxed);
    return PCR_OK;
}

pcr_status prefix_prefill_attn(const void *q, const pcr_kv_pool *pool, const int32_t *block_tables,
                               int32_t max_blocks, const int32_t *prefix_lens, const int32_t *cu_suffix,
                               const int32_t *host_prefix_lens, const int32_t *host_cu_suffix, int32_t B,
                               int32_t num_q_heads, float sm_scale, void *out, void *stream, int auto_schedule)
{
    g_err[0] = 0;
    int64_t T = 0;
    pcr_status st = attn_check(q, pool, block_tables, max_blocks, prefix_lens, cu_suffix, host_prefix_lens,
                               host_cu_suffix, B, num_q_heads, sm_scale, out, "pcr_prefix_prefill_attn", &T);
    if (st || T == 0) return st;
    int32_t n_cu = 0;
    st = device_cu_count(&n_cu, "pcr_prefix_prefill_attn");
    if (st) return st;
    hipError_t e = launch_prefix_prefill_attn(q, *pool, block_tables, max_blocks, host_prefix_lens,
                                              host_cu_suffix, B, num_q_heads, (int32_t)T, sm_scale, out,
                                              static_cast<hipStream_t>(stream), auto_schedule, n_cu);
    if (e != hipSuccess) return hip_fail(e, "pcr_prefix_prefill_attn: launch");
    return PCR_OK;
}

pcr_status load_staged_split(const pcr_host_kv *src, const int32_t *src_blocks, const pcr_kv_pool *dst,
                             const int32_t *dst_blocks, int32_t n, void *workspace, int64_t workspace_bytes,
                             hipStream_t dma_stream, hipStream_t scatter_stream, hipEvent_t dma_done)
{
    return load_impl(src, src_blocks, dst, dst_blocks, n, PCR_LOAD_DMA_STAGED, workspace, workspace_bytes,
                     dma_stream, scatter_stream, dma_done);
}

pcr_status offload_with(const pcr_kv_pool *src, const int32_t *src_blocks, const pcr_host_kv *dst,
                        const int32_t *dst_blocks, int32_t n, pcr_load_method method, void *workspace,
                        int64_t workspace_bytes, void *stream)
{
    return offload_impl(src, src_blocks, dst, dst_blocks, n, method, workspace, workspace_bytes, stream);
}

}  // namespace pcr
