// Split-key decode attention for gfx950: one query token per sequence (bf16 in,
// fp32 accumulate, bf16 out).
//
// For sequence b with n_b visible keys (its cached context plus the token being
// decoded) and query head h: out = softmax_j(sm_scale <q, k_j>) v_j over
// j = 0 .. n_b - 1, K/V read from the paged pool through the block table. This
// is the suffix row of a sequence with prefix n_b - 1 and a one-token suffix
// (Sec. 2.2); the prefill kernel computes the same rows inside mixed batches,
// but its 128-row tiles would carry only G = Hq/Hkv useful rows here, and a
// decode step is bound by reading K/V from HBM, not by matrix work.
//
// Work decomposition. The key range of each (sequence, kv head) is cut into
// n_split chunks of `chunk` keys (a multiple of 32). Each chunk is the work of
// one wave (decode_wave::chunk, decode_wave.h: the G query heads as MFMA columns,
// K and V straight from HBM into registers, here with three register sets so that
// two steps of loads are in flight while a third is used); the host picks n_split
// so that every SIMD gets about one wave. Every byte is used once: V loads are
// non-temporal, and K loads too when every sequence has one length and the chunks
// give every SIMD a wave (the kernel then streams HBM at full rate, where bypassing
// the caches measured about 10% faster than ordinary loads for both); otherwise K
// loads are ordinary ones (decode_wave.h: K_CACHED).
//
// A chunk that covers its whole sequence writes the output row. Up to four
// chunks of one (sequence, kv head) form one workgroup and are merged through
// LDS (running max and sum in the log2 domain). With more chunks, each wave
// writes its unnormalised O, max and sum to the workspace and
// decode_combine_kernel merges the chunks of each (sequence, head).
#include <algorithm>
#include <mutex>

#include "decode_wave.h"
#include "pcr_internal.h"

// Scratch of the allocation-free decode entry point: the split kernel's partial
// outputs (O, max, sum per chunk and query head) when a batch's chunks merge
// through memory. One copy per device, held until the process ends. In host code
// this name is a stand-in, not a device address: kernels get the address that
// hipGetSymbolAddress returns for the current device (decode_noalloc_scratch).
static __device__ __align__(256) unsigned char scratch[pcr::kDecodeScratchBytes];

namespace pcr {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef unsigned short u16;

constexpr int kWaves = 4;              // tasks (waves) per workgroup
constexpr int kThreads = 64 * kWaves;
constexpr int kStepKeys = decode_wave::kStepKeys;   // keys per step: two pool blocks
constexpr int kMaxCols = decode_wave::kMaxCols;   // query heads per kv head held by one tile
// Waves per CU the split count aims at: one per SIMD, each with three register sets
// of K/V loads (two steps in flight while a third is used), measured faster than
// two waves per SIMD with two sets each.
constexpr int waves_per_cu(int) { return 4; }
constexpr int kMinChunk = 256;         // keys; shorter chunks spend more on set-up than on loads
constexpr float kLog2e = 1.4426950408889634f;

template <int D, bool K_CACHED>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(1))) void decode_split_kernel(
    const u16 *__restrict__ q, const u16 *__restrict__ pool_k, const u16 *__restrict__ pool_v,
    int32_t num_blocks, int32_t Hkv, const int32_t *__restrict__ block_tables, int32_t max_blocks,
    const int32_t *__restrict__ context_lens, int32_t B, int32_t Hq, int32_t n_split, int32_t chunk,
    float scale_log2, int32_t lds_merge, u16 *__restrict__ out, float *__restrict__ ws_o,
    float *__restrict__ ws_ml)
{
    constexpr int MT = D / 16;    // V products (16 dims each)
    const int lane = (int)(threadIdx.x & 63);
    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const int wg_waves = (int)(blockDim.x >> 6);   // n_split when the chunks merge in LDS
    const int64_t task = (int64_t)blockIdx.x * wg_waves + wave;
    if (task >= (int64_t)B * Hkv * n_split) return;   // never for a merging workgroup (exact grid)
    const int sp = (int)(task % n_split);
    const int bg = (int)(task / n_split);
    const int g = bg % Hkv, b = bg / Hkv;
    const int n_keys = context_lens[b];
    const int kbeg = sp * chunk;
    const bool active = kbeg < n_keys;             // wave-uniform
    if (!active && !lds_merge) return;             // a merging wave stays for the barrier
    const int kend = min(n_keys, kbeg + chunk);
    const int last_blk = max(0, min((n_keys - 1) >> 4, max_blocks - 1));   // last block with a visible key
    const int G = Hq / Hkv;
    const int c = lane & 15, q4 = lane >> 4;
    const bool col = c < G;
    const int h = g * G + c;

    f32x4 o[MT];
    float m_run = -INFINITY, l_run = 0.f;
    if (active) {
        const u16 *qrow = q + ((int64_t)b * Hq + (col ? h : g * G)) * D + 8 * q4;
        decode_wave::chunk<D, 3, K_CACHED>(qrow, col, pool_k, pool_v, num_blocks, Hkv, g, block_tables + (int64_t)b * max_blocks,
                                 last_blk, kbeg, kend, scale_log2, o, m_run, l_run);
    } else {
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) o[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
    }

    float l_tot = l_run + __shfl_xor(l_run, 16);
    l_tot += __shfl_xor(l_tot, 32);
    if (lds_merge) {
        // The workgroup holds every chunk of one (sequence, kv head). Waves 1.. leave
        // their O (lane layout), max and sum in LDS; wave 0 merges and writes. A chunk
        // past the sequence's end contributes max -inf, sum 0, O 0; chunk 0 always has
        // keys, so the merged max is finite.
        extern __shared__ f32x4 part_o[];          // [wave][MT][64 lanes]
        f32x2 *part_ml = reinterpret_cast<f32x2 *>(part_o + wg_waves * MT * 64);   // [wave][64 lanes]
        if (wave > 0) {
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) part_o[(wave * MT + mt) * 64 + lane] = o[mt];
            part_ml[wave * 64 + lane] = f32x2{m_run, l_tot};
        }
        __syncthreads();
        if (wave > 0) return;
        float M = m_run;
        for (int w = 1; w < wg_waves; ++w) M = fmaxf(M, part_ml[w * 64 + lane][0]);
        const float a0 = __builtin_amdgcn_exp2f(m_run - M);
        l_tot *= a0;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) o[mt] *= a0;
        for (int w = 1; w < wg_waves; ++w) {
            const f32x2 ml = part_ml[w * 64 + lane];
            const float a = __builtin_amdgcn_exp2f(ml[0] - M);
            l_tot += a * ml[1];
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) o[mt] += a * part_o[(w * MT + mt) * 64 + lane];
        }
    }
    if (!col) return;
    if (lds_merge || (kbeg == 0 && kend == n_keys)) {   // merged, or the only chunk of its sequence
        const float inv = 1.f / l_tot;
        u16 *orow = out + ((int64_t)b * Hq + h) * D + 4 * q4;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            const bf16x4 v = __builtin_convertvector(o[mt] * inv, bf16x4);
            *reinterpret_cast<u32x2 *>(orow + 16 * mt) = __builtin_bit_cast(u32x2, v);
        }
        return;
    }
    const int64_t part = task * G + c;
    float *po = ws_o + part * D + 4 * q4;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) *reinterpret_cast<f32x4 *>(po + 16 * mt) = o[mt];
    if (q4 == 0) *reinterpret_cast<f32x2 *>(ws_ml + 2 * part) = f32x2{m_run, l_tot};
}

// One wave per (sequence, query head) of a sequence cut into more than one chunk:
// out = sum_c 2^(m_c - M) O_c / sum_c 2^(m_c - M) l_c with M = max_c m_c.
template <int D>
__global__ __launch_bounds__(kThreads) void decode_combine_kernel(
    const float *__restrict__ ws_o, const float *__restrict__ ws_ml, const int32_t *__restrict__ context_lens,
    int32_t B, int32_t Hkv, int32_t Hq, int32_t n_split, int32_t chunk, u16 *__restrict__ out)
{
    constexpr int E = D / 64;     // output elements per lane
    const int lane = (int)(threadIdx.x & 63);
    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const int64_t pair = (int64_t)blockIdx.x * kWaves + wave;
    if (pair >= (int64_t)B * Hq) return;
    const int h = (int)(pair % Hq), b = (int)(pair / Hq);
    const int G = Hq / Hkv, g = h / G, c = h % G;
    const int n_keys = context_lens[b];
    const int ns = min((n_keys + chunk - 1) / chunk, n_split);
    if (ns <= 1) return;                            // written by the split kernel
    const int64_t part0 = ((int64_t)b * Hkv + g) * n_split * G + c;
    // Up to 64 chunks per pass: lane j reads chunk k0 + j's max and sum (all loads in
    // flight together), the wave reduces them, and the O rows are read eight chunks at a
    // time with their loads issued before any is used. Across passes the running max,
    // sum and accumulator are rescaled. The accumulator adds the chunks in their order.
    float M = -INFINITY, L = 0.f, acc[E];
#pragma unroll
    for (int e = 0; e < E; ++e) acc[e] = 0.f;
    for (int k0 = 0; k0 < ns; k0 += 64) {
        const int nk = min(64, ns - k0);
        f32x2 ml = f32x2{-INFINITY, 0.f};
        if (lane < nk) ml = *reinterpret_cast<const f32x2 *>(ws_ml + 2 * (part0 + (int64_t)(k0 + lane) * G));
        float mb = ml[0];
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) mb = fmaxf(mb, __shfl_xor(mb, off));
        const float Mn = fmaxf(M, mb);                  // finite: chunk k0 has keys
        const float r = __builtin_amdgcn_exp2f(M - Mn);  // 0 on the first pass
        M = Mn;
        const float w = __builtin_amdgcn_exp2f(ml[0] - M);   // 0 past the last chunk
        float lw = w * ml[1];
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) lw += __shfl_xor(lw, off);
        L = L * r + lw;
#pragma unroll
        for (int e = 0; e < E; ++e) acc[e] *= r;
        for (int j0 = 0; j0 < nk; j0 += 8) {
            float po[8][E];
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const int j = min(j0 + i, nk - 1);       // a chunk past nk is reread, weight 0
                const float *src = ws_o + (part0 + (int64_t)(k0 + j) * G) * D + E * lane;
#pragma unroll
                for (int e = 0; e < E; ++e) po[i][e] = src[e];
            }
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const float wi = __builtin_bit_cast(
                    float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, w), min(j0 + i, 63)));
                const float wv = j0 + i < nk ? wi : 0.f;
#pragma unroll
                for (int e = 0; e < E; ++e) acc[e] += wv * po[i][e];
            }
        }
    }
    const float inv = 1.f / L;
    u16 *orow = out + ((int64_t)b * Hq + h) * D + E * lane;
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const __bf16 v = (__bf16)(acc[e] * inv);
        orow[e] = __builtin_bit_cast(u16, v);
    }
}

}  // namespace

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices];   // device address of `scratch` on each device, once taken
}  // namespace

hipError_t decode_noalloc_scratch(void **ptr)
{
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));   // this device's copy (the device is current)
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        g_scratch_ptr[dev] = p;
    }
    *ptr = g_scratch_ptr[dev];
    return hipSuccess;
}

namespace {
DecodePlan decode_split_plan(int32_t B, int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                             int32_t max_context, int32_t n_cu, const int32_t *ctx, int64_t ws_limit)
{
    DecodePlan p{};
    const int64_t pairs = (int64_t)B * num_kv_heads;
    if (pairs <= 0 || max_context <= 0) return p;
    const int64_t G = num_q_heads / num_kv_heads;
    const int64_t part_bytes = G * (head_dim + 2) * 4;      // one chunk's O, max and sum per query head
    const int64_t waves = (int64_t)n_cu * waves_per_cu(head_dim);
    const int64_t want = (waves + pairs - 1) / pairs;      // chunks per sequence that fill the SIMDs
    const int64_t cap = ((int64_t)max_context + kMinChunk - 1) / kMinChunk;
    auto round_chunk = [](int64_t c) { return (c + kStepKeys - 1) / kStepKeys * kStepKeys; };
    // Rule by the largest context: every sequence gets up to `bound` chunks of equal size.
    const int64_t bound = std::max<int64_t>(1, std::min(want, cap));
    const int64_t chunk = round_chunk(((int64_t)max_context + bound - 1) / bound);
    p.chunk = (int32_t)chunk;
    p.n_split = (int32_t)(((int64_t)max_context + chunk - 1) / chunk);
    p.lds_merge = p.n_split > 1 && p.n_split <= kWaves;
    p.ws_wg_waves = kWaves;
    p.workspace_bytes = p.n_split > kWaves ? pairs * p.n_split * part_bytes : 0;
    // Rule by the total count of keys (ragged batches; only when the sequences alone do
    // not fill the SIMDs): the smallest chunk whose chunks over all sequences still give
    // at most one wave per SIMD, with up to 2 * want chunks for the longest sequence.
    const int64_t s_max = want > 1 ? std::min(cap, 2 * want) : 1;
    const int64_t bound_old = bound > kWaves ? pairs * bound * part_bytes : 0;
    // (a plan by total keys needing more than the allocation-free scratch is never taken)
    p.bound_workspace_bytes =
        std::max(bound_old, s_max > 1 ? std::min<int64_t>(pairs * s_max * part_bytes, kDecodeScratchBytes) : 0);
    if (!ctx || s_max <= 1) return p;
    auto active = [&](int64_t c) {
        int64_t n = 0;
        for (int32_t b = 0; b < B; ++b) n += ((int64_t)ctx[b] + c - 1) / c;
        return n * num_kv_heads;
    };
    int64_t lo = round_chunk(std::max<int64_t>(kMinChunk, ((int64_t)max_context + s_max - 1) / s_max));
    int64_t hi = chunk;
    if (lo >= hi || active(hi) > waves) return p;
    while (lo < hi) {   // smallest chunk (a multiple of kStepKeys) with active(chunk) <= waves
        const int64_t mid = round_chunk((lo + hi) / 2);
        if (mid >= hi) break;
        if (active(mid) <= waves) hi = mid; else lo = mid + kStepKeys;
    }
    const int64_t c2 = hi;
    if (c2 >= chunk) return p;
    const int64_t n2 = ((int64_t)max_context + c2 - 1) / c2;
    bool full = true;   // every sequence has all n2 chunks: they can merge in LDS
    for (int32_t b = 0; b < B && full; ++b) full = ((int64_t)ctx[b] + c2 - 1) / c2 == n2;
    const bool lds = n2 > 1 && n2 <= kWaves && full;
    const int64_t ws = (n2 > 1 && !lds) ? pairs * n2 * part_bytes : 0;
    if (ws > ws_limit) return p;
    p.chunk = (int32_t)c2;
    p.n_split = (int32_t)n2;
    p.lds_merge = lds;
    // One wave per workgroup: chunks past a short sequence's end then end their own
    // workgroup at once and leave the SIMD to another chunk (a wave takes a whole SIMD,
    // so a four-wave workgroup holds a compute unit until its longest chunk is done).
    p.ws_wg_waves = 1;
    p.workspace_bytes = ws;
    return p;
}
}  // namespace

DecodePlan decode_plan(int32_t B, int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                       int32_t max_context, int32_t n_cu, const int32_t *ctx, int64_t ws_limit)
{
    DecodePlan p = decode_split_plan(B, num_q_heads, num_kv_heads, head_dim, max_context, n_cu, ctx, ws_limit);
    // Non-temporal K loads when every sequence has one length and its chunks give every
    // SIMD a wave: then every wave streams one chunk length for the whole kernel and HBM
    // is the bound. Otherwise (ragged or small batches, bound by what each compute unit
    // has in flight) ordinary K loads, which fetch each K line once per step.
    bool same = ctx != nullptr;
    for (int32_t b = 0; b < B && same; ++b) same = ctx[b] == max_context;
    p.k_streamed = same && (int64_t)B * num_kv_heads * p.n_split >= (int64_t)n_cu * waves_per_cu(head_dim);
    return p;
}

int decode_max_cols() { return kMaxCols; }

hipError_t launch_decode_attn(const void *q, const pcr_kv_pool &pool, const int32_t *block_tables,
                              int32_t max_blocks, const int32_t *context_lens, int32_t B, int32_t num_q_heads,
                              const DecodePlan &plan, float sm_scale, void *out, void *workspace, hipStream_t s)
{
    const int Hkv = pool.num_kv_heads, G = num_q_heads / Hkv, D = pool.head_dim;
    const int64_t n_tasks = (int64_t)B * Hkv * plan.n_split;
    // Up to kWaves chunks of a sequence share one workgroup and merge in LDS when every
    // sequence has all n_split of them; otherwise they go through the workspace and
    // decode_combine_kernel (a chunk past its sequence's end then ends its wave at once).
    const int lds_merge = plan.lds_merge;
    const bool through_ws = plan.n_split > 1 && !lds_merge;
    const int wg_waves = through_ws ? plan.ws_wg_waves : plan.n_split;
    const dim3 grid((unsigned)((n_tasks + wg_waves - 1) / wg_waves));
    const size_t lds = lds_merge ? (size_t)wg_waves * 64 * ((D / 16) * 16 + 8) : 0;
    float *ws_o = through_ws ? static_cast<float *>(workspace) : nullptr;
    float *ws_ml = through_ws ? ws_o + n_tasks * G * D : nullptr;
    const float scale_log2 = sm_scale * kLog2e;
    auto *qq = static_cast<const u16 *>(q);
    auto *pk = static_cast<const u16 *>(pool.k);
    auto *pv = static_cast<const u16 *>(pool.v);
    auto *oo = static_cast<u16 *>(out);
    auto split = [&](auto kernel) {
        hipLaunchKernelGGL(kernel, grid, dim3(64 * wg_waves), lds, s, qq, pk, pv, pool.num_blocks, Hkv, block_tables,
                           max_blocks, context_lens, B, num_q_heads, plan.n_split, plan.chunk, scale_log2, lds_merge,
                           oo, ws_o, ws_ml);
    };
    if (D == 128) {
        if (plan.k_streamed) split(decode_split_kernel<128, false>); else split(decode_split_kernel<128, true>);
    } else {
        if (plan.k_streamed) split(decode_split_kernel<64, false>); else split(decode_split_kernel<64, true>);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || !through_ws) return e;
    const dim3 cgrid((unsigned)(((int64_t)B * num_q_heads + kWaves - 1) / kWaves));
    if (D == 128)
        hipLaunchKernelGGL(decode_combine_kernel<128>, cgrid, dim3(kThreads), 0, s, ws_o, ws_ml, context_lens, B,
                           Hkv, num_q_heads, plan.n_split, plan.chunk, oo);
    else
        hipLaunchKernelGGL(decode_combine_kernel<64>, cgrid, dim3(kThreads), 0, s, ws_o, ws_ml, context_lens, B,
                           Hkv, num_q_heads, plan.n_split, plan.chunk, oo);
    return hipGetLastError();
}

}  // namespace pcr
