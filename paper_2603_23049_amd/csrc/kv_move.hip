// KV data-movement kernels for gfx950: append (new K/V rows into pool slots),
// gather (pool back to logical order) and the host-pull block copy.
//
// All three are pure bit movement; every access is 16 bytes wide where the
// layout allows, and every block id or slot read from device memory is
// range-checked in the kernel before use, so a bad table entry skips its row
// rather than touching memory outside the pool.
#include "pcr_internal.h"

namespace pcr {
namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned short u16;

constexpr int kTileTokens = 16;
// New tokens per append workgroup: 32 measured as fast as 16 on block-aligned slot lists
// and 31% faster on the RAG mix's (whose tiles start inside chunks); 64 was 3.5% slower
// on aligned lists of 128k tokens.
constexpr int kAppendTile = 32;

// ---------------------------------------------------------------------------
// append: grid (ceil(T/TILE), Hkv), 256 threads. One workgroup writes TILE new
// tokens of one kv head. K rows are copied 16 B at a time. V is written d-major
// inside each block: the tile's V rows go through LDS, and each aligned run of 8
// slots of one dim (a 16-byte chunk of a block's V) that the tile's tokens fill is
// written by one 16-byte store. A chunk the tile fills only in part (a run of
// slots that starts or ends inside it: a sequence boundary, a tile edge, a slot
// list that is not 8-aligned) gets element stores for its filled slots.
// ---------------------------------------------------------------------------
template <int D, int TILE>
__global__ __launch_bounds__(256) void append_kv_kernel(
    u16 *__restrict__ pool_k, u16 *__restrict__ pool_v, int32_t num_blocks, int32_t Hkv,
    const u16 *__restrict__ k_new, const u16 *__restrict__ v_new,
    const int32_t *__restrict__ slot_mapping, int32_t T)
{
    static_assert(TILE <= 64, "one wave ranks the chunk runs");
    constexpr int CPR = D / 8;                 // 16-B chunks per row
    constexpr int NCH = (TILE * CPR + 255) / 256;
    __shared__ u16 vs[TILE][D + 8];            // +8 elements: stagger rows across banks
    __shared__ int32_t slots[TILE];
    __shared__ int32_t runs[TILE];             // (first token << 8) | tokens, one per chunk run
    __shared__ int32_t n_runs;

    const int tile = blockIdx.x, g = blockIdx.y, tid = threadIdx.x;
    const int tok0 = tile * TILE;

    // The K/V rows do not depend on the slot list: their loads go out first, so the two
    // memory round trips (slots, rows) overlap.
    u32x4 kv[NCH], vv[NCH];
#pragma unroll
    for (int i = 0; i < NCH; ++i) {
        const int c = tid + 256 * i, r = c / CPR, cc = c % CPR;
        kv[i] = u32x4{0u, 0u, 0u, 0u};
        vv[i] = u32x4{0u, 0u, 0u, 0u};
        if (c < TILE * CPR && tok0 + r < T) {
            const int64_t src = ((int64_t)(tok0 + r) * Hkv + g) * D + cc * 8;
            kv[i] = *reinterpret_cast<const u32x4 *>(k_new + src);
            vv[i] = *reinterpret_cast<const u32x4 *>(v_new + src);
        }
    }
    if (tid < TILE) {
        const int t = tok0 + tid;
        int32_t sl = -1;
        if (t < T) {
            sl = slot_mapping[t];
            if (sl < 0 || sl / kBlockSize >= num_blocks) sl = -1;
        }
        slots[tid] = sl;
    }
    __syncthreads();

#pragma unroll
    for (int i = 0; i < NCH; ++i) {
        const int c = tid + 256 * i, r = c / CPR, cc = c % CPR;
        if (c < TILE * CPR && tok0 + r < T) {
            *reinterpret_cast<u32x4 *>(&vs[r][cc * 8]) = vv[i];
            const int32_t sl = slots[r];
            if (sl >= 0) {
                const int64_t blk = sl / kBlockSize, o = sl % kBlockSize;
                const int64_t dst = ((blk * Hkv + g) * kBlockSize + o) * D + cc * 8;
                *reinterpret_cast<u32x4 *>(pool_k + dst) = kv[i];
            }
        }
    }
    // Chunk runs (wave 0): a token starts one when its slot is valid and either opens an
    // aligned chunk of 8 slots or does not follow the previous token's slot; the run
    // goes on over the following tokens until the next start or invalid slot (a
    // continuing token's slot is its predecessor's plus one, inside the same chunk).
    if (tid < 64) {
        const int32_t sl = tid < TILE ? slots[tid] : -1;
        const bool valid = sl >= 0;
        const bool start = valid && (tid == 0 || sl % 8 == 0 || slots[tid - 1] != sl - 1);
        const uint64_t starts = __builtin_amdgcn_ballot_w64(start);
        const uint64_t stops = starts | ~__builtin_amdgcn_ballot_w64(valid);   // bits past TILE are stops
        if (start) {
            const uint64_t after = tid == 63 ? 0ull : stops >> (tid + 1);
            const int len = after ? 1 + __builtin_ctzll(after) : 64 - tid;
            const int idx = __builtin_popcountll(starts & ((1ull << tid) - 1ull));
            runs[idx] = (tid << 8) | len;
        }
        if (tid == 0) n_runs = __builtin_popcountll(starts);
    }
    __syncthreads();

    // V: task = (run, dim)
    const int nr = n_runs;
    for (int task = tid; task < nr * D; task += 256) {
        const int k = task / D, x = task % D;
        const int rv = runs[k], r0 = rv >> 8, len = rv & 0xff;
        const int32_t s0 = slots[r0];
        const int64_t blk = s0 / kBlockSize, o = s0 % kBlockSize;
        u16 *dst = pool_v + ((blk * Hkv + g) * D + x) * kBlockSize + o;
        if (len == 8) {   // a whole aligned chunk (a run of 8 starts at a multiple of 8)
            u16 e[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) e[j] = vs[r0 + j][x];
            u32x4 w;
            w.x = e[0] | ((unsigned)e[1] << 16);
            w.y = e[2] | ((unsigned)e[3] << 16);
            w.z = e[4] | ((unsigned)e[5] << 16);
            w.w = e[6] | ((unsigned)e[7] << 16);
            *reinterpret_cast<u32x4 *>(dst) = w;
        } else {
            for (int j = 0; j < len; ++j) dst[j] = vs[r0 + j][x];
        }
    }
}

// ---------------------------------------------------------------------------
// gather: grid (ceil(total/16), Hkv), 256 threads; out rows in logical order.
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(256) void gather_kv_kernel(
    const u16 *__restrict__ pool_k, const u16 *__restrict__ pool_v, int32_t num_blocks, int32_t Hkv,
    const int32_t *__restrict__ block_tables, int32_t max_blocks,
    const int32_t *__restrict__ starts, const int32_t *__restrict__ cu_out, int32_t B,
    int32_t total, u16 *__restrict__ k_out, u16 *__restrict__ v_out)
{
    constexpr int CPR = D / 8;
    const int g = blockIdx.y, tid = threadIdx.x;
    if (tid >= kTileTokens * CPR) return;
    const int r = blockIdx.x * kTileTokens + tid / CPR, c = tid % CPR;
    if (r >= total) return;
    int lo = 0, hi = B - 1;                  // sequence b with cu_out[b] <= r < cu_out[b+1]
    while (lo < hi) {
        const int mid = (lo + hi + 1) / 2;
        if (cu_out[mid] <= r) lo = mid; else hi = mid - 1;
    }
    const int b = lo;
    const int t = starts[b] + (r - cu_out[b]);
    const int64_t dst = ((int64_t)r * Hkv + g) * D + c * 8;
    u32x4 kw = {0u, 0u, 0u, 0u}, vw = {0u, 0u, 0u, 0u};
    const int lb = t / kBlockSize;
    if (t >= 0 && lb < max_blocks) {
        const int64_t blk = block_tables[(int64_t)b * max_blocks + lb];
        const int64_t o = t % kBlockSize;
        if (blk >= 0 && blk < num_blocks) {
            kw = *reinterpret_cast<const u32x4 *>(pool_k + ((blk * Hkv + g) * kBlockSize + o) * D + c * 8);
            const u16 *vb = pool_v + ((blk * Hkv + g) * D + c * 8) * kBlockSize + o;
            u16 e[8];
#pragma unroll
            for (int k = 0; k < 8; ++k) e[k] = vb[k * kBlockSize];
            vw.x = e[0] | ((unsigned)e[1] << 16);
            vw.y = e[2] | ((unsigned)e[3] << 16);
            vw.z = e[4] | ((unsigned)e[5] << 16);
            vw.w = e[6] | ((unsigned)e[7] << 16);
        }
    }
    *reinterpret_cast<u32x4 *>(k_out + dst) = kw;
    *reinterpret_cast<u32x4 *>(v_out + dst) = vw;
}

// ---------------------------------------------------------------------------
// host pull / push: each workgroup copies whole blocks (K or V of one pair)
// between the pinned host store and the pool, 16 B per lane, 8 loads in flight
// per lane before their stores. Grid-stride over the 2*n block copies. Pull
// (host -> pool) reads the host pages with non-temporal loads; push (pool ->
// host) writes them with non-temporal stores, so host data never occupies L2.
// ---------------------------------------------------------------------------
constexpr int kPullUnroll = 8;
// Workgroups of one pull launch: 32 x 256 lanes x 8 x 16 B = 1 MiB in flight, enough
// to saturate a PCIe 5 x16 host link while leaving the other CUs to the compute stream
// (on MI355X, 16 workgroups reach about 85% of the link, 32 and more the full link).
constexpr int kPullWorkgroups = 32;

enum CopyDir { kHostToDevice = 0, kDeviceToHost = 1, kDeviceToDevice = 2 };

template <int kDir>
__global__ __launch_bounds__(256) void copy_blocks_kernel(
    const u32x4 *__restrict__ src_k, const u32x4 *__restrict__ src_v, int64_t src_blocks,
    u32x4 *__restrict__ dst_k, u32x4 *__restrict__ dst_v, int64_t dst_blocks,
    int64_t block_vecs, const PullArgs args)
{
    const int units = 2 * args.n;
    for (int u = blockIdx.x; u < units; u += gridDim.x) {
        const int pair = u >> 1;
        const bool is_v = u & 1;
        const int64_t sb = args.src[pair], db = args.dst[pair];
        if (sb < 0 || sb >= src_blocks || db < 0 || db >= dst_blocks) continue;
        const u32x4 *src = (is_v ? src_v : src_k) + sb * block_vecs;
        u32x4 *dst = (is_v ? dst_v : dst_k) + db * block_vecs;
        for (int64_t base = 0; base < block_vecs; base += 256 * kPullUnroll) {
            u32x4 r[kPullUnroll];
#pragma unroll
            for (int k = 0; k < kPullUnroll; ++k) {
                const int64_t i = base + k * 256 + threadIdx.x;
                if (i < block_vecs) r[k] = kDir == kHostToDevice ? __builtin_nontemporal_load(src + i) : src[i];
            }
#pragma unroll
            for (int k = 0; k < kPullUnroll; ++k) {
                const int64_t i = base + k * 256 + threadIdx.x;
                if (i < block_vecs) {
                    if (kDir == kDeviceToHost) __builtin_nontemporal_store(r[k], dst + i);
                    else dst[i] = r[k];
                }
            }
        }
    }
}

}  // namespace

hipError_t launch_append_kv(const pcr_kv_pool &pool, const void *k_new, const void *v_new,
                            const int32_t *slot_mapping, int32_t T, hipStream_t s)
{
    const dim3 grid((T + kAppendTile - 1) / kAppendTile, pool.num_kv_heads);
    auto *pk = static_cast<u16 *>(pool.k);
    auto *pv = static_cast<u16 *>(pool.v);
    auto *kn = static_cast<const u16 *>(k_new);
    auto *vn = static_cast<const u16 *>(v_new);
    if (pool.head_dim == 128)
        hipLaunchKernelGGL((append_kv_kernel<128, kAppendTile>), grid, dim3(256), 0, s, pk, pv, pool.num_blocks,
                           pool.num_kv_heads, kn, vn, slot_mapping, T);
    else
        hipLaunchKernelGGL((append_kv_kernel<64, kAppendTile>), grid, dim3(256), 0, s, pk, pv, pool.num_blocks,
                           pool.num_kv_heads, kn, vn, slot_mapping, T);
    return hipGetLastError();
}

hipError_t launch_gather_kv(const pcr_kv_pool &pool, const int32_t *block_tables, int32_t max_blocks,
                            const int32_t *starts, const int32_t *cu_out, int32_t B, int32_t total,
                            void *k_out, void *v_out, hipStream_t s)
{
    const dim3 grid((total + kTileTokens - 1) / kTileTokens, pool.num_kv_heads);
    auto *pk = static_cast<const u16 *>(pool.k);
    auto *pv = static_cast<const u16 *>(pool.v);
    if (pool.head_dim == 128)
        hipLaunchKernelGGL(gather_kv_kernel<128>, grid, dim3(256), 0, s, pk, pv, pool.num_blocks,
                           pool.num_kv_heads, block_tables, max_blocks, starts, cu_out, B, total,
                           static_cast<u16 *>(k_out), static_cast<u16 *>(v_out));
    else
        hipLaunchKernelGGL(gather_kv_kernel<64>, grid, dim3(256), 0, s, pk, pv, pool.num_blocks,
                           pool.num_kv_heads, block_tables, max_blocks, starts, cu_out, B, total,
                           static_cast<u16 *>(k_out), static_cast<u16 *>(v_out));
    return hipGetLastError();
}

hipError_t launch_pull_blocks(const void *host_k, const void *host_v, int64_t host_blocks,
                              void *pool_k, void *pool_v, int32_t pool_blocks, int64_t block_bytes,
                              const PullArgs &args, hipStream_t s)
{
    if (args.n <= 0) return hipSuccess;
    const int units = 2 * args.n;
    const int grid = units < kPullWorkgroups ? units : kPullWorkgroups;
    hipLaunchKernelGGL(copy_blocks_kernel<kHostToDevice>, dim3(grid), dim3(256), 0, s,
                       static_cast<const u32x4 *>(host_k), static_cast<const u32x4 *>(host_v),
                       host_blocks, static_cast<u32x4 *>(pool_k), static_cast<u32x4 *>(pool_v),
                       (int64_t)pool_blocks, block_bytes / 16, args);
    return hipGetLastError();
}

hipError_t launch_push_blocks(const void *pool_k, const void *pool_v, int32_t pool_blocks, void *host_k,
                              void *host_v, int64_t host_blocks, int64_t block_bytes, const PullArgs &args,
                              hipStream_t s)
{
    if (args.n <= 0) return hipSuccess;
    const int units = 2 * args.n;
    const int grid = units < kPullWorkgroups ? units : kPullWorkgroups;
    hipLaunchKernelGGL(copy_blocks_kernel<kDeviceToHost>, dim3(grid), dim3(256), 0, s,
                       static_cast<const u32x4 *>(pool_k), static_cast<const u32x4 *>(pool_v),
                       (int64_t)pool_blocks, static_cast<u32x4 *>(host_k), static_cast<u32x4 *>(host_v),
                       host_blocks, block_bytes / 16, args);
    return hipGetLastError();
}

hipError_t launch_device_blocks(const void *src_k, const void *src_v, int64_t src_blocks, void *dst_k, void *dst_v,
                                int64_t dst_blocks, int64_t block_bytes, const PullArgs &args, hipStream_t s)
{
    if (args.n <= 0) return hipSuccess;
    // HBM to HBM: one workgroup per block copy, all CUs if there is work for them
    const int grid = 2 * args.n;
    hipLaunchKernelGGL(copy_blocks_kernel<kDeviceToDevice>, dim3(grid), dim3(256), 0, s,
                       static_cast<const u32x4 *>(src_k), static_cast<const u32x4 *>(src_v), src_blocks,
                       static_cast<u32x4 *>(dst_k), static_cast<u32x4 *>(dst_v), dst_blocks, block_bytes / 16, args);
    return hipGetLastError();
}

}  // namespace pcr
