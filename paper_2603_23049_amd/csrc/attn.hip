// Paged prefix-reuse prefill attention for gfx950 (bf16 in, fp32 accumulate, bf16 out).
//
// For sequence b with p cached and s new tokens, query head h and suffix row i
// (absolute position p+i): out = softmax_j(sm_scale <q, k_j>) v_j over keys
// j = 0 .. p+i, with K/V read from the paged pool through the block table
// (exact prefix reuse, Sec. 2.2; paged blocks, Sec. 5).
//
// Work decomposition. The s*G query rows of one (sequence, kv head) pair, G
// = Hq/Hkv, are packed token-major (row r = token r/G, head-in-group r%G) so
// that all rows of a workgroup share one K/V stream. A workgroup takes 128
// packed rows (4 waves x 32) and walks 64-key tiles (4 pool blocks) from key 0
// to its last row's causal limit.
//
// Per wave and tile, with v_mfma_f32_32x32x16_bf16:
//   S^T[key][q] = K Q^T   A = K rows from LDS, B = this wave's Q (registers)
//   O^T[d][q]  += V^T P^T A = V^T from LDS,  B = P (registers)
// Each lane holds one query column q = lane%32 of both accumulators, so the
// online softmax (running max, rescale, exp2) is in-lane; the two half-waves
// holding the same query exchange only their tile max (one shuffle) and their
// partial sums at the end. K rows are fed to the first product in a permuted
// key order chosen so that the S^T accumulator registers of a lane are, in
// order, the P^T operand registers of the second product: no data moves
// between the two products. V is stored d-major inside each pool block, so a
// V^T operand (8 consecutive keys of one dim) is one 16-byte LDS read.
//
// LDS holds two K/V tiles (double buffer): the next tile's global loads are
// issued before the current tile's math and written to the other buffer after
// it, with one barrier per tile. 16-byte chunks are XOR-swizzled so that the
// 32 lanes reading 32 different key rows (K) or dims (V) hit distinct banks.
#include "pcr_internal.h"

namespace pcr {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef unsigned short u16;

constexpr int kWaves = 4;
constexpr int kRowsPerWave = 32;
constexpr int kRowsPerWG = kWaves * kRowsPerWave;
constexpr int kTileKeys = 64;
constexpr int kTileBlocks = kTileKeys / kBlockSize;
constexpr float kLog2e = 1.4426950408889634f;

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// Key (within a 32-key half tile) whose K row is fed as A-operand row i of the
// first product. With this order, accumulator register r of lane (q, half)
// holds key 16*(r/8) + 8*half + r%8 of the half tile, i.e. registers 8t..8t+7
// are the 8 keys P^T needs in the second product's k-step t.
__device__ __forceinline__ constexpr int key_of_row(int i)
{
    return 16 * (i >> 4) + 8 * ((i >> 2) & 1) + 4 * ((i >> 3) & 1) + (i & 3);
}

template <int D>
__global__ __launch_bounds__(256) void prefill_attn_kernel(
    const u16 *__restrict__ q, const u16 *__restrict__ pool_k, const u16 *__restrict__ pool_v,
    int32_t num_blocks, int32_t Hkv, const int32_t *__restrict__ block_tables, int32_t max_blocks,
    const int32_t *__restrict__ prefix_lens, const int32_t *__restrict__ cu_suffix, int32_t Hq,
    int32_t T, float scale_log2, u16 *__restrict__ out)
{
    constexpr int CPR = D / 8;                 // 16-B chunks per K row
    constexpr int KSTEPS = D / 16;             // k-steps of the first product
    constexpr int MT = D / 32;                 // 32-dim tiles of O^T
    constexpr int CPB = kBlockSize * D / 8;    // 16-B chunks per (block, head) payload
    constexpr int NCH = kTileBlocks * CPB / 256;  // chunks per thread per tile (K; same for V)
    constexpr int64_t kHeadPayload = kBlockSize * D;

    __shared__ __attribute__((aligned(16))) u16 lds_k[2][kTileKeys * D];
    __shared__ __attribute__((aligned(16))) u16 lds_v[2][kTileBlocks * D * kBlockSize];

    const int rt = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int qc = lane & 31, half = lane >> 5;

    const int p = prefix_lens[b];
    const int t0 = cu_suffix[b];
    const int s = cu_suffix[b + 1] - t0;
    const int G = Hq / Hkv;
    const int rows_total = s * G;
    const int row0 = rt * kRowsPerWG;
    if (s <= 0 || row0 >= rows_total) return;   // uniform over the workgroup
    const int total = p + s;

    // This lane's packed query row (rows past the end compute a copy of the last row).
    const int R = row0 + wave * kRowsPerWave + qc;
    const bool row_valid = R < rows_total;
    const int Rc = row_valid ? R : rows_total - 1;
    const int i = Rc / G, hl = Rc - i * G;
    const int h = g * G + hl;
    const int limit = p + i;                         // last key this row attends to
    const int64_t tq = (int64_t)t0 + i;

    const int wg_last = min(rows_total - 1, row0 + kRowsPerWG - 1);
    const int ntiles = (p + wg_last / G) / kTileKeys + 1;
    const int w_first = min(rows_total - 1, row0 + wave * kRowsPerWave);
    const int w_last = min(rows_total - 1, row0 + wave * kRowsPerWave + kRowsPerWave - 1);
    const int w_min_limit = p + w_first / G;
    const int w_max_limit = p + w_last / G;

    // Q^T operand fragments (k-step ks: dims 16ks + 8half .. +7 of this lane's row).
    bf16x8 qf[KSTEPS];
    {
        const bool ok = tq < T;
        const u16 *qrow = q + (ok ? (tq * Hq + h) * D : 0);
#pragma unroll
        for (int ks = 0; ks < KSTEPS; ++ks) {
            u32x4 v = {0u, 0u, 0u, 0u};
            if (ok) v = *reinterpret_cast<const u32x4 *>(qrow + 16 * ks + 8 * half);
            qf[ks] = as_bf16x8(v);
        }
    }

    f32x16 o_acc[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int r = 0; r < 16; ++r) o_acc[mt][r] = 0.f;
    float m_run = -INFINITY;   // running max of scaled scores (log2 domain)
    float l_run = 0.f;         // this lane's part of the running denominator

    const int32_t *bt = block_tables + (int64_t)b * max_blocks;
    u32x4 kreg[NCH], vreg[NCH];

    auto load_tile = [&](int kt) {
#pragma unroll
        for (int u = 0; u < NCH; ++u) {
            const int id = tid + 256 * u;
            const int j = id / CPB, within = id % CPB;
            const int lb = kt * kTileBlocks + j;
            const int key0 = lb * kBlockSize;
            int64_t blk = -1;
            if (key0 < total && lb < max_blocks) {
                blk = bt[lb];
                if (blk >= num_blocks) blk = -1;
            }
            u32x4 kv = {0u, 0u, 0u, 0u}, vv = {0u, 0u, 0u, 0u};
            if (blk >= 0) {
                const int64_t base = (blk * Hkv + g) * kHeadPayload + within * 8;
                kv = *reinterpret_cast<const u32x4 *>(pool_k + base);
                vv = *reinterpret_cast<const u32x4 *>(pool_v + base);
                // V chunk = one dim, keys key0 + 8*(within&1) .. +7; slots past the
                // sequence end are zeroed (their probabilities are 0, their bits
                // may be anything).
                const int nvalid = total - (key0 + 8 * (within & 1));
                if (nvalid < 8) {
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        if (e >= nvalid) vv[e >> 1] &= (e & 1) ? 0x0000FFFFu : 0xFFFF0000u;
                }
            }
            kreg[u] = kv;
            vreg[u] = vv;
        }
    };
    auto store_tile = [&](int buf) {
#pragma unroll
        for (int u = 0; u < NCH; ++u) {
            const int id = tid + 256 * u;
            const int j = id / CPB, within = id % CPB;
            const int key = kBlockSize * j + within / CPR, c = within % CPR;
            const int pc = c ^ (key % CPR);
            *reinterpret_cast<u32x4 *>(&lds_k[buf][key * D + pc * 8]) = kreg[u];
            const int d = within >> 1, ch = within & 1;
            const int pch = ch ^ ((d >> 3) & 1);
            *reinterpret_cast<u32x4 *>(&lds_v[buf][(j * D + d) * kBlockSize + pch * 8]) = vreg[u];
        }
    };

    load_tile(0);
    store_tile(0);
    __syncthreads();

    for (int kt = 0; kt < ntiles; ++kt) {
        const int buf = kt & 1;
        if (kt + 1 < ntiles) load_tile(kt + 1);
        const int kbase = kt * kTileKeys;
        if (kbase <= w_max_limit) {
            // ---- S^T = K Q^T over two 32-key halves ----
            f32x16 st[2];
#pragma unroll
            for (int m = 0; m < 2; ++m) {
#pragma unroll
                for (int r = 0; r < 16; ++r) st[m][r] = 0.f;
                const int krow = 32 * m + key_of_row(qc);
#pragma unroll
                for (int ks = 0; ks < KSTEPS; ++ks) {
                    const int pc = (2 * ks + half) ^ (krow % CPR);
                    const bf16x8 a =
                        as_bf16x8(*reinterpret_cast<const u32x4 *>(&lds_k[buf][krow * D + pc * 8]));
                    st[m] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[ks], st[m], 0, 0, 0);
                }
            }
            // ---- online softmax (log2 domain) ----
            const bool need_mask = kbase + kTileKeys - 1 > w_min_limit;
            float sv[32];
            float mx = -INFINITY;
#pragma unroll
            for (int m = 0; m < 2; ++m)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    float x = st[m][r] * scale_log2;
                    if (need_mask) {
                        const int key = kbase + 32 * m + 16 * (r >> 3) + 8 * half + (r & 7);
                        if (key > limit) x = -INFINITY;
                    }
                    sv[16 * m + r] = x;
                    mx = fmaxf(mx, x);
                }
            mx = fmaxf(mx, __shfl_xor(mx, 32));
            const float m_new = fmaxf(m_run, mx);
            const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
            float psum = 0.f;
#pragma unroll
            for (int e = 0; e < 32; ++e) {
                const float pe = __builtin_amdgcn_exp2f(sv[e] - m_new);
                sv[e] = pe;
                psum += pe;
            }
            l_run = l_run * alpha + psum;
            m_run = m_new;
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                for (int r = 0; r < 16; ++r) o_acc[mt][r] *= alpha;
            // ---- O^T += V^T P^T, k-step t = pool block t of the tile ----
#pragma unroll
            for (int t = 0; t < kTileBlocks; ++t) {
                f32x8 pv;
#pragma unroll
                for (int e = 0; e < 8; ++e) pv[e] = sv[16 * (t >> 1) + 8 * (t & 1) + e];
                const bf16x8 pf = __builtin_convertvector(pv, bf16x8);
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) {
                    const int d = 32 * mt + qc;
                    const int pch = half ^ ((d >> 3) & 1);
                    const bf16x8 a = as_bf16x8(*reinterpret_cast<const u32x4 *>(
                        &lds_v[buf][(t * D + d) * kBlockSize + pch * 8]));
                    o_acc[mt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pf, o_acc[mt], 0, 0, 0);
                }
            }
        }
        if (kt + 1 < ntiles) store_tile(buf ^ 1);
        __syncthreads();
    }

    // ---- normalise and store: lane holds dims 32mt + 8R + 4half + c of its row ----
    const float l_tot = l_run + __shfl_xor(l_run, 32);
    const float inv = 1.f / l_tot;
    if (row_valid && tq < T) {
        u16 *orow = out + (tq * Hq + h) * D;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int R4 = 0; R4 < 4; ++R4) {
                typedef float f32x4 __attribute__((ext_vector_type(4)));
                typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
                f32x4 v;
#pragma unroll
                for (int c = 0; c < 4; ++c) v[c] = o_acc[mt][4 * R4 + c] * inv;
                const bf16x4 bv = __builtin_convertvector(v, bf16x4);
                const int d0 = 32 * mt + 8 * R4 + 4 * half;
                *reinterpret_cast<u32x2 *>(orow + d0) = __builtin_bit_cast(u32x2, bv);
            }
    }
}

}  // namespace

int attn_rows_per_workgroup(int) { return kRowsPerWG; }

hipError_t launch_prefix_prefill_attn(const void *q, const pcr_kv_pool &pool,
                                      const int32_t *block_tables, int32_t max_blocks,
                                      const int32_t *prefix_lens, const int32_t *cu_suffix,
                                      int32_t B, int32_t num_q_heads, int32_t T,
                                      int32_t max_row_tiles, float sm_scale, void *out,
                                      hipStream_t s)
{
    const dim3 grid(max_row_tiles, pool.num_kv_heads, B);
    const float scale_log2 = sm_scale * kLog2e;
    auto *qq = static_cast<const u16 *>(q);
    auto *pk = static_cast<const u16 *>(pool.k);
    auto *pv = static_cast<const u16 *>(pool.v);
    auto *oo = static_cast<u16 *>(out);
    if (pool.head_dim == 128)
        hipLaunchKernelGGL(prefill_attn_kernel<128>, grid, dim3(256), 0, s, qq, pk, pv,
                           pool.num_blocks, pool.num_kv_heads, block_tables, max_blocks, prefix_lens,
                           cu_suffix, num_q_heads, T, scale_log2, oo);
    else
        hipLaunchKernelGGL(prefill_attn_kernel<64>, grid, dim3(256), 0, s, qq, pk, pv,
                           pool.num_blocks, pool.num_kv_heads, block_tables, max_blocks, prefix_lens,
                           cu_suffix, num_q_heads, T, scale_log2, oo);
    return hipGetLastError();
}

}  // namespace pcr
