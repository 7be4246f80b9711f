// Paged prefix-reuse prefill attention for gfx950 (bf16 in, fp32 accumulate, bf16 out).
//
// For sequence b with p cached and s new tokens, query head h and suffix row i
// (absolute position p+i): out = softmax_j(sm_scale <q, k_j>) v_j over keys
// j = 0 .. p+i, with K/V read from the paged pool through the block table
// (exact prefix reuse, Sec. 2.2; paged blocks, Sec. 5).
//
// Work decomposition. The s*G query rows of one (sequence, kv head) pair,
// G = Hq/Hkv, are packed token-major (row r = token r/G, head-in-group r%G)
// so that all rows of a workgroup share one K/V stream. A workgroup of 8 waves
// takes 128 packed rows. Waves 0-3 and 4-7 form two groups that hold the same
// rows (32 per wave) and walk the two halves of the key range, so each SIMD
// runs one wave of each group: one wave's softmax overlaps the other's
// matrix work. The halves are merged through LDS at the end.
//
// Per wave and 64-key tile (4 pool blocks), with v_mfma_f32_32x32x16_bf16:
//   S^T[key][q] = K Q^T   A = K rows from LDS, B = this wave's Q (registers)
//   O^T[d][q]  += V^T P^T A = V^T from LDS,  B = P (registers)
// Each lane holds one query column q = lane%32 of both accumulators, so the
// online softmax is in-lane; the two half-waves holding the same query trade
// only their tile max (one shuffle) and their partial sums at the end. K rows
// are fed to the first product in a permuted key order chosen so that the S^T
// accumulator registers of a lane are, in order, the P^T operand registers of
// the second product. V is stored d-major inside each pool block, so a V^T
// operand (8 consecutive keys of one dim) is one 16-byte LDS read.
//
// Softmax runs in the log2 domain with the scale folded into one FMA. The
// running max is only raised (and O rescaled) when a tile's max exceeds it by
// more than 2^8; otherwise the stale max stays, which keeps probabilities
// below 256 and skips the rescale of 64 accumulators per lane.
//
// Tiles move global -> LDS with global_load_lds_dwordx4 (no staging
// registers), double-buffered with one barrier per tile. LDS chunks are
// XOR-swizzled so that lanes reading 32 different key rows (K) or dims (V)
// hit distinct banks; the swizzle is applied through the source address of
// each lane, since a direct load writes lane l's 16 bytes at base + 16*l.
#include "pcr_internal.h"

namespace pcr {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef unsigned short u16;

constexpr int kGroupWaves = 4;
constexpr int kRowsPerWave = 32;
constexpr int kRowsPerWG = kGroupWaves * kRowsPerWave;   // 128 rows, shared by both groups
constexpr int kThreads = 2 * kGroupWaves * 64;           // 512
constexpr int kTileKeys = 64;
constexpr int kTileBlocks = kTileKeys / kBlockSize;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kRescaleThreshold = 8.0f;                // log2 units
constexpr int kXcds = 8;                                 // MI355X: 8 XCDs, workgroups dealt round-robin

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// Key (within a 32-key half tile) whose K row is fed as A-operand row i of the
// first product. With this order, accumulator register r of lane (q, half)
// holds key 16*(r/8) + 8*half + r%8 of the half tile, i.e. registers 8t..8t+7
// are the 8 keys P^T needs in the second product's k-step t.
__device__ __forceinline__ constexpr int key_of_row(int i)
{
    return 16 * (i >> 4) + 8 * ((i >> 2) & 1) + 4 * ((i >> 3) & 1) + (i & 3);
}

// LDS chunk swizzle of a K tile row (chunks of 16 B; CPR chunks per row).
template <int CPR>
__device__ __forceinline__ constexpr int k_swizzle(int key) { return key % CPR; }

template <int D>
struct TileGeom {
    static constexpr int CPR = D / 8;                          // 16-B chunks per K row
    static constexpr int KBYTES = kTileKeys * D * 2;           // K tile bytes
    static constexpr int VBYTES = kTileKeys * D * 2;           // V tile bytes
    static constexpr int BYTES = KBYTES + VBYTES;
    static constexpr int SLABS = BYTES / 1024;                 // 1 KB per wave-wide direct load
    static constexpr int LOADS = SLABS / kGroupWaves;          // direct loads per thread per tile
    static constexpr int KSLABS = KBYTES / 1024;
};

__device__ __forceinline__ void wait_vmem() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

template <int D>
__global__ __launch_bounds__(kThreads) void prefill_attn_kernel(
    const u16 *__restrict__ q, const u16 *__restrict__ pool_k, const u16 *__restrict__ pool_v,
    int32_t num_blocks, int32_t Hkv, const int32_t *__restrict__ block_tables, int32_t max_blocks,
    const int32_t *__restrict__ prefix_lens, const int32_t *__restrict__ cu_suffix, int32_t Hq,
    int32_t T, int32_t B, int32_t row_tiles, float scale_log2, u16 *__restrict__ out)
{
    using Geo = TileGeom<D>;
    constexpr int CPR = Geo::CPR;
    constexpr int KSTEPS = D / 16;
    constexpr int MT = D / 32;
    constexpr int64_t kHeadPayload = kBlockSize * D;

    // [group][buffer][K tile | V tile]; reused for the merge at the end.
    __shared__ __attribute__((aligned(1024))) char lds[2][2][Geo::BYTES];

    // XCD-aware order: workgroup L runs on XCD L % 8, so consecutive work items
    // (the row tiles of one (sequence, kv head), which read the same K/V) are
    // given to workgroups of one XCD and share its L2.
    const int n_work = row_tiles * Hkv * B;
    const int per_xcd = (int)(gridDim.x / kXcds);
    const int w = (int)(blockIdx.x % kXcds) * per_xcd + (int)(blockIdx.x / kXcds);
    if (w >= n_work) return;
    const int rt = w % row_tiles;
    const int g = (w / row_tiles) % Hkv;
    const int b = w / (row_tiles * Hkv);
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int grp = wave >> 2;              // 0: first half of the keys, 1: second half
    const int wg = wave & 3;                // wave within the group (selects the rows)
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
    const int R = row0 + wg * kRowsPerWave + qc;
    const bool row_valid = R < rows_total;
    const int Rc = row_valid ? R : rows_total - 1;
    const int i = Rc / G, hl = Rc - i * G;
    const int h = g * G + hl;
    const int limit = p + i;                         // last key this row attends to
    const int64_t tq = (int64_t)t0 + i;

    const int wg_last = min(rows_total - 1, row0 + kRowsPerWG - 1);
    const int ntiles = (p + wg_last / G) / kTileKeys + 1;
    const int split = (ntiles + 1) >> 1;             // group 0: [0, split), group 1: [split, ntiles)
    const int niter = split;
    const int tile_begin = grp ? split : 0;
    const int tile_end = grp ? ntiles : split;
    const int w_first = min(rows_total - 1, row0 + wg * kRowsPerWave);
    const int w_last = min(rows_total - 1, row0 + wg * kRowsPerWave + kRowsPerWave - 1);
    const int w_min_limit = p + w_first / G;
    const int w_max_limit = p + w_last / G;
    const int valid_blocks = min((total + kBlockSize - 1) / kBlockSize, max_blocks);

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
    float m_run = -INFINITY;   // reference max of raw scores times scale_log2
    float l_run = 0.f;         // this lane's part of the denominator

    const int32_t *bt = block_tables + (int64_t)b * max_blocks;

    // Block ids of one tile (4 pool blocks), read as scalars; ids past the
    // sequence or outside the pool become block 0 (their keys are masked and
    // their V entries zeroed), so no load ever leaves the pool.
    auto tile_ids = [&](int kt, int32_t (&ids)[kTileBlocks]) {
#pragma unroll
        for (int j = 0; j < kTileBlocks; ++j) {
            const int lb = kt * kTileBlocks + j;
            int32_t blk = 0;
            if (lb < valid_blocks) {
                blk = bt[lb];
                if (blk < 0 || blk >= num_blocks) blk = 0;
            }
            ids[j] = blk;
        }
    };

    // Issue the direct loads of a tile (block ids given) into this group's buffer buf.
    auto issue_tile = [&](const int32_t (&ids)[kTileBlocks], int buf) {
        char *tbase = lds[grp][buf];
#pragma unroll
        for (int u = 0; u < Geo::LOADS; ++u) {
            const int slab = u * kGroupWaves + wg;                 // wave-uniform
            const bool is_k = slab < Geo::KSLABS;                  // wave-uniform
            const int P = slab * 64 + lane;                        // 16-B chunk position in the tile
            const int Pk = is_k ? P : P - Geo::KBYTES / 16;
            const int j = is_k ? (slab * 64) / (CPR * kBlockSize) : ((slab - Geo::KSLABS) * 64) / (2 * D);
            const int64_t head_base = ((int64_t)ids[j] * Hkv + g) * kHeadPayload;
            const u16 *src;
            if (is_k) {
                const int key = Pk / CPR, pc = Pk % CPR;
                const int c = pc ^ k_swizzle<CPR>(key);
                src = pool_k + head_base + (key % kBlockSize) * D + c * 8;
            } else {
                const int within = Pk % (2 * D);
                const int d = within >> 1, pch = within & 1;
                const int ch = pch ^ ((d >> 3) & 1);
                src = pool_v + head_base + d * kBlockSize + ch * 8;
            }
            __builtin_amdgcn_global_load_lds(
                (const void *)src, (__attribute__((address_space(3))) void *)(tbase + slab * 1024), 16, 0, 0);
        }
    };

    // Zero the V entries of keys >= total in a tile's buffer (their slots may hold
    // anything, and a zero probability times a NaN would still poison the sum).
    auto zero_tail = [&](int kt, int buf) {
        u16 *vt = reinterpret_cast<u16 *>(lds[grp][buf] + Geo::KBYTES);
        const int gtid = tid & 255;
        for (int e = gtid; e < kTileBlocks * D; e += 256) {       // one (block, dim) row of 16 keys
            const int j = e / D, d = e % D;
            const int key0 = kt * kTileKeys + j * kBlockSize;
#pragma unroll
            for (int o = 0; o < kBlockSize; ++o)
                if (key0 + o >= total) {
                    const int pch = (o >> 3) ^ ((d >> 3) & 1);
                    vt[(j * D + d) * kBlockSize + pch * 8 + (o & 7)] = 0;
                }
        }
    };

    // One tile's math for this wave. masked: some key of the tile lies past some
    // row's causal limit (only the last tiles of a row range; wave-uniform).
    auto compute_tile = [&](bool masked, int kt, int buf) {
        const int kbase = kt * kTileKeys;
        const char *tk = lds[grp][buf];
        const char *tv = tk + Geo::KBYTES;
        // ---- S^T = K Q^T over two 32-key halves ----
        f32x16 st[2];
#pragma unroll
        for (int m = 0; m < 2; ++m) {
#pragma unroll
            for (int r = 0; r < 16; ++r) st[m][r] = 0.f;
            const int krow = 32 * m + key_of_row(qc);
#pragma unroll
            for (int ks = 0; ks < KSTEPS; ++ks) {
                const int pc = (2 * ks + half) ^ k_swizzle<CPR>(krow);
                const bf16x8 a = as_bf16x8(*reinterpret_cast<const u32x4 *>(tk + (krow * CPR + pc) * 16));
                st[m] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[ks], st[m], 0, 0, 0);
            }
        }
        // ---- online softmax (log2 domain, lazy rescale) ----
        if (masked) {
            // register r of half tile m holds key kbase + 32m + 16(r/8) + 8half + r%8
            const int lim = limit - kbase - 8 * half;
#pragma unroll
            for (int m = 0; m < 2; ++m)
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    st[m][r] = (32 * m + 16 * (r >> 3) + (r & 7)) > lim ? -INFINITY : st[m][r];
        }
        float mx = -INFINITY;
#pragma unroll
        for (int m = 0; m < 2; ++m)
#pragma unroll
            for (int r = 0; r < 16; r += 2) mx = fmaxf(mx, fmaxf(st[m][r], st[m][r + 1]));
        mx = fmaxf(mx, __shfl_xor(mx, 32)) * scale_log2;
        if (__builtin_amdgcn_ballot_w64(mx > m_run + kRescaleThreshold)) {
            const float m_new = fmaxf(m_run, mx);
            const float alpha = (m_new == -INFINITY) ? 1.f : __builtin_amdgcn_exp2f(m_run - m_new);
            m_run = m_new;
            l_run *= alpha;
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                for (int r = 0; r < 16; ++r) o_acc[mt][r] *= alpha;
        }
        // A row with no key yet has m_run = -inf and only masked scores: exp2(-inf) = 0.
        const float neg_m = (m_run == -INFINITY) ? 0.f : -m_run;
        // ---- per pool block t of the tile: P = exp2(s*scale - m) in bf16, row sums from
        // the bf16 values the MFMA uses, then O^T += V^T P^T (k-step t) ----
        const bf16x2_t ones = {(__bf16)1.0f, (__bf16)1.0f};
#pragma unroll
        for (int t = 0; t < kTileBlocks; ++t) {
            f32x8 pv;
#pragma unroll
            for (int e = 0; e < 8; ++e)
                pv[e] = __builtin_amdgcn_exp2f(__builtin_fmaf(st[t >> 1][8 * (t & 1) + e], scale_log2, neg_m));
            const bf16x8 pf = __builtin_convertvector(pv, bf16x8);
#pragma unroll
            for (int e = 0; e < 8; e += 2) {
                const bf16x2_t pair = {pf[e], pf[e + 1]};
                l_run = __builtin_amdgcn_fdot2_f32_bf16(pair, ones, l_run, false);
            }
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                const int d = 32 * mt + qc;
                const int pch = half ^ ((d >> 3) & 1);
                const bf16x8 a =
                    as_bf16x8(*reinterpret_cast<const u32x4 *>(tv + ((t * D + d) * 2 + pch) * 16));
                o_acc[mt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pf, o_acc[mt], 0, 0, 0);
            }
        }
    };

    const int last_tile = ntiles - 1;
    const bool last_needs_zero = (last_tile + 1) * kTileKeys > total;
    const int last_owner = last_tile >= split ? 1 : 0;
    const int last_iter = last_tile - (last_owner ? split : 0);

    int32_t ids[kTileBlocks];
    if (tile_begin < tile_end) {
        tile_ids(tile_begin, ids);
        issue_tile(ids, 0);
        if (tile_begin + 1 < tile_end) tile_ids(tile_begin + 1, ids);
    }

    for (int it = 0; it < niter; ++it) {
        const int buf = it & 1;
        const int kt = tile_begin + it;
        const bool have = kt < tile_end;
        wait_vmem();
        __syncthreads();
        if (last_needs_zero && it == last_iter) {                  // uniform over the workgroup
            if (grp == last_owner) zero_tail(kt, buf);
            __syncthreads();
        }
        if (have && kt + 1 < tile_end) {
            issue_tile(ids, buf ^ 1);                              // ids of tile kt+1
            if (kt + 2 < tile_end) tile_ids(kt + 2, ids);
        }
        if (!have || kt * kTileKeys > w_max_limit) continue;
        compute_tile(kt * kTileKeys + kTileKeys - 1 > w_min_limit, kt, buf);
    }

    // ---- merge the two key halves through LDS, normalise, store ----
    const float l_tot = l_run + __shfl_xor(l_run, 32);
    __syncthreads();
    float *xch = reinterpret_cast<float *>(&lds[0][0][0]);
    constexpr int XW = 4 * MT + 1;                 // float4 slots per lane: O, then (m, l)
    if (grp == 1) {
        f32x4 *x4 = reinterpret_cast<f32x4 *>(xch) + (size_t)wg * XW * 64;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int r4 = 0; r4 < 4; ++r4) {
                f32x4 v;
#pragma unroll
                for (int c = 0; c < 4; ++c) v[c] = o_acc[mt][4 * r4 + c];
                x4[(mt * 4 + r4) * 64 + lane] = v;
            }
        f32x4 ml = {m_run, l_tot, 0.f, 0.f};
        x4[(XW - 1) * 64 + lane] = ml;
    }
    __syncthreads();
    if (grp == 1) return;

    const f32x4 *x4 = reinterpret_cast<const f32x4 *>(xch) + (size_t)wg * XW * 64;
    const f32x4 ml = x4[(XW - 1) * 64 + lane];
    const float m1 = ml[0], l1 = ml[1];
    const float mm = fmaxf(m_run, m1);
    const float a0 = (m_run == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(m_run - mm);
    const float a1 = (m1 == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(m1 - mm);
    const float inv = 1.f / (a0 * l_tot + a1 * l1);
    if (row_valid && tq < T) {
        u16 *orow = out + (tq * Hq + h) * D;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int r4 = 0; r4 < 4; ++r4) {
                const f32x4 o1 = x4[(mt * 4 + r4) * 64 + lane];
                f32x4 v;
#pragma unroll
                for (int c = 0; c < 4; ++c) v[c] = (a0 * o_acc[mt][4 * r4 + c] + a1 * o1[c]) * inv;
                const bf16x4 bv = __builtin_convertvector(v, bf16x4);
                const int d0 = 32 * mt + 8 * r4 + 4 * half;
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
    const int64_t n_work = (int64_t)max_row_tiles * pool.num_kv_heads * B;
    const dim3 grid((unsigned)(((n_work + kXcds - 1) / kXcds) * kXcds));
    const float scale_log2 = sm_scale * kLog2e;
    auto *qq = static_cast<const u16 *>(q);
    auto *pk = static_cast<const u16 *>(pool.k);
    auto *pv = static_cast<const u16 *>(pool.v);
    auto *oo = static_cast<u16 *>(out);
    if (pool.head_dim == 128)
        hipLaunchKernelGGL(prefill_attn_kernel<128>, grid, dim3(kThreads), 0, s, qq, pk, pv,
                           pool.num_blocks, pool.num_kv_heads, block_tables, max_blocks, prefix_lens,
                           cu_suffix, num_q_heads, T, B, max_row_tiles, scale_log2, oo);
    else
        hipLaunchKernelGGL(prefill_attn_kernel<64>, grid, dim3(kThreads), 0, s, qq, pk, pv,
                           pool.num_blocks, pool.num_kv_heads, block_tables, max_blocks, prefix_lens,
                           cu_suffix, num_q_heads, T, B, max_row_tiles, scale_log2, oo);
    return hipGetLastError();
}

}  // namespace pcr
