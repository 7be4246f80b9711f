// Paged prefix-reuse prefill attention for gfx950 (bf16 in, fp32 accumulate, bf16 out).
//
// For sequence b with p cached and s new tokens, query head h and suffix row i
// (absolute position p+i): out = softmax_j(sm_scale <q, k_j>) v_j over keys
// j = 0 .. p+i, with K/V read from the paged pool through the block table
// (exact prefix reuse, Sec. 2.2; paged blocks, Sec. 5).
//
// Work decomposition. The s*G query rows of one (sequence, kv head) pair,
// G = Hq/Hkv, are packed token-major (row r = token r/G, head-in-group r%G)
// so that all rows of a workgroup share one K/V stream. A workgroup has 8 waves in
// two groups (waves 0-3 and 4-7, 32 rows per wave), so each SIMD runs one wave of
// each group: one wave's softmax overlaps the other's matrix work. Two schedules:
//   key halves: the workgroup takes 128 packed rows; both groups hold the same rows
//     and walk the two halves of the key range, merged through LDS at the end;
//   row halves: the workgroup takes 256 packed rows, 128 per group, and both groups
//     walk the whole key range, group 1 one phase behind, through one copy of each
//     tile that group 0 loads; no merge.
// Row halves give each workgroup twice the work for one start-up and no merge; the
// host takes them when the launch still has at least two workgroups per compute
// unit, key halves otherwise (twice the workgroups for small launches).
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
// Softmax runs in the log2 domain. The first product of a tile starts from
// -m_ref, so the raw scores <q, k> come out already shifted, and one fp32
// multiply by c = sm_scale * log2(e) precedes each exp2. (Folding c into Q
// instead would round q*c to bf16: a relative error of 2^-9 on every score,
// which for sharp rows of large |<q, k>| moves the output by far more than the
// bf16 inputs themselves do.) The reference max m_ref is only raised (and O
// rescaled) when a tile's scaled max exceeds it by more than 8, i.e. a factor
// of 2^8; otherwise the stale value stays, which keeps probabilities below 256
// and skips the rescale of 64 accumulators per lane.
//
// Tiles move global -> LDS with global_load_lds_dwordx4 (no staging
// registers), double-buffered with one barrier per tile. LDS chunks are
// XOR-swizzled so that lanes reading 32 different key rows (K) or dims (V)
// hit distinct banks; the swizzle is applied through the source address of
// each lane, since a direct load writes lane l's 16 bytes at base + 16*l.
#include <algorithm>
#include <atomic>
#include <type_traits>
#include <vector>

#include "decode_wave.h"
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
constexpr int kRowsPerWG = kGroupWaves * kRowsPerWave;   // 128 rows (key halves: both groups)
constexpr int kThreads = 2 * kGroupWaves * 64;           // 512
constexpr int kTileKeys = 64;
constexpr int kTileBlocks = kTileKeys / kBlockSize;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kRescaleThreshold = 8.0f;                // log2 units: P <= 2^8
// LDS fragment reads kept in flight ahead of the MFMAs in the matrix cluster. With the
// shared row-halves tiles 3 and 4 measured 0.4-0.8% faster than 5 and 1-2% faster than 6
// or 7 on the 70B and RAG-mix shapes: the reads are bound by the LDS's throughput, not
// its latency.
#ifndef KAHEAD
#define KAHEAD 4
#endif
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
    static constexpr int KLOADS = KBYTES / 1024 / kGroupWaves; // 1 KB direct loads per thread, K tile
    static constexpr int VLOADS = VBYTES / 1024 / kGroupWaves; // same, V tile
};

__device__ __forceinline__ void wait_vmem() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }
// s_waitcnt immediate that waits for LDS, scalar-memory and message counters only
// (lgkmcnt = 0; vmcnt and expcnt at their maxima, so they do not wait).
constexpr int kWaitLgkm0 = 0xC07F;

// Workgroup barrier without a memory fence. The phase schedule orders its memory
// traffic explicitly: every direct load is waited for (vmcnt) by the wave that
// issued it before the barrier that precedes its first reader, and every LDS read
// is consumed before its wave reaches the next barrier. The empty asm statements
// keep the compiler from moving memory operations across the barrier.
__device__ __forceinline__ void phase_barrier()
{
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
}

// One wave-wide direct load global -> LDS: lane l's 16 bytes at src land at
// lds_dst + 16*l (lds_dst wave-uniform). Issued as inline assembly because the
// compiler counts a global-to-LDS load as a pending LDS access of unknown order and
// then drains every outstanding LDS read (lgkmcnt(0)) at the next operand wait,
// which would empty the fragment pipeline after each load. The hardware signals
// completion of these loads on vmcnt only; the kernel waits for them explicitly
// before the barrier that precedes their first reader.
// The source is a wave-uniform base (SGPR pair) plus a 32-bit per-lane byte offset.
// lds_dst is an LDS byte address (M0 form). M0 is a register the compiler reserves:
// it does not honour the clobber, and relies on M0 only for instructions that read
// it, of which this file has none besides these loads (each sets it first).
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void dma16(const char *base, uint32_t lane_off, uint32_t lds_dst)
{
    const unsigned m0 = __builtin_amdgcn_readfirstlane(lds_dst);
    // The base is wave-uniform; reading it through readfirstlane states that to the
    // register allocator (free when it already sits in SGPRs), which otherwise may keep
    // it in VGPRs under SGPR pressure and then cannot meet the "s" constraint.
    // (readfirstlane returns int: each half goes through uint32_t before widening, or a
    // low word with bit 31 set would sign-extend into the high half of the address)
    const uint64_t b64 = reinterpret_cast<uint64_t>(base);
    const uint64_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(b64 >> 32));
    const uint64_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)b64);
    const uint64_t sb = (hi << 32) | lo;
    asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(lane_off),
                 "s"(reinterpret_cast<const char *>(sb)), "s"(m0)
                 : "memory", "m0");
}
#pragma clang diagnostic pop

// Wait until at most N vector-memory operations of this wave are outstanding
// (the N most recent may still be in flight).
template <int N>
__device__ __forceinline__ void wait_vmem_keep()
{
    static_assert(N >= 0 && N < 64, "vmcnt range");
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Order of one launch's work items (row tile of a sequence, kv head), built on the
// host from the sequence lengths and passed by value in the kernel arguments.
// Sequences are taken heaviest first (longest key range), and inside a sequence the
// last row tiles (the most keys) first, so the long items start early and the
// short ones fill the tail. Each slot also carries its sequence's lengths, so a
// workgroup finds everything it needs about its sequence in one parallel read of
// the map (the kernel arguments) instead of a chain of dependent loads.
constexpr int kMaxMapSeqs = 128;
struct AttnWorkMap {
    int32_t n_seq;                      // slots in use (sequences with new tokens)
    int32_t per_head;                   // row tiles of all sequences, one kv head
    int32_t seq[kMaxMapSeqs];           // sequence in each slot
    int32_t tiles_end[kMaxMapSeqs];     // row tiles of the slots up to and including this one
    int32_t prefix[kMaxMapSeqs];        // the slot's cached tokens p
    int32_t first[kMaxMapSeqs];         // the slot's first new token (row of q and out)
    int32_t count[kMaxMapSeqs];         // the slot's new tokens s
};

// A sequence with one new token in a prefill launch (a decode row, Sec. 2.2; prefill
// and decode rows in one pass, Sec. 4.3): its G rows would fill G columns of the
// 128- or 256-row tiles, and the workgroup would spend the matrix time of the whole
// tile on them while its loads sit idle. Its workgroup instead runs the decode
// kernel's wave routine (decode_wave.h): the 8 waves each take one chunk of the keys
// (with two register sets, which the prefill kernel's register budget allows) and
// merge their (O, max, sum) through LDS. The work is then bound by reading K/V, and
// it overlaps the matrix-bound workgroups of the prefill rows on the other compute
// units.
template <int D>
__device__ __forceinline__ void decode_workgroup(const u16 *__restrict__ q, const u16 *__restrict__ pool_k,
                                                 const u16 *__restrict__ pool_v, int32_t num_blocks, int32_t Hkv,
                                                 const int32_t *__restrict__ bt_row, int32_t max_blocks, int g, int G,
                                                 int32_t Hq, int p, int64_t t0, float scale_log2,
                                                 u16 *__restrict__ out, char *lds)
{
    constexpr int MT = D / 16;
    constexpr int kWaves = kThreads / 64;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int n_keys = p + 1;                       // keys 0 .. p: the row's causal range
    const int chunk = ((n_keys + kWaves - 1) / kWaves + decode_wave::kStepKeys - 1) / decode_wave::kStepKeys *
                      decode_wave::kStepKeys;
    const int kbeg = wave * chunk;
    const int kend = min(n_keys, kbeg + chunk);
    const int last_blk = max(0, min((n_keys - 1) >> 4, max_blocks - 1));
    const int c = lane & 15, q4 = lane >> 4;
    const bool col = c < G;
    const int h = g * G + c;
    f32x4 o[MT];
    float m_run = -INFINITY, l_run = 0.f;
    if (kbeg < n_keys) {
        const u16 *qrow = q + (t0 * Hq + (col ? h : g * G)) * D + 8 * q4;
        decode_wave::chunk<D, 2, true>(qrow, col, pool_k, pool_v, num_blocks, Hkv, g, bt_row, last_blk, kbeg, kend,
                                 scale_log2, o, m_run, l_run);
    } else {
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) o[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    float l_tot = l_run + __shfl_xor(l_run, 16);
    l_tot += __shfl_xor(l_tot, 32);
    // Waves 1.. leave O (lane layout), max and sum in LDS; wave 0 merges and writes. A
    // chunk past the end contributes max -inf, sum 0, O 0; chunk 0 always has keys.
    f32x4 *part_o = reinterpret_cast<f32x4 *>(lds);                         // [wave][MT][64 lanes]
    float *part_ml = reinterpret_cast<float *>(part_o + kWaves * MT * 64);   // [wave][64 lanes][2]
    if (wave > 0) {
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) part_o[(wave * MT + mt) * 64 + lane] = o[mt];
        part_ml[2 * (wave * 64 + lane)] = m_run;
        part_ml[2 * (wave * 64 + lane) + 1] = l_tot;
    }
    __syncthreads();
    // (no early return here: a return on a lane condition inside this inlined function
    // made the compiler treat the prefill path's block offsets as divergent)
    if (wave == 0) {
        float M = m_run;
        for (int w = 1; w < kWaves; ++w) M = fmaxf(M, part_ml[2 * (w * 64 + lane)]);
        const float a0 = __builtin_amdgcn_exp2f(m_run - M);
        l_tot *= a0;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) o[mt] *= a0;
        for (int w = 1; w < kWaves; ++w) {
            const float a = __builtin_amdgcn_exp2f(part_ml[2 * (w * 64 + lane)] - M);
            l_tot += a * part_ml[2 * (w * 64 + lane) + 1];
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) o[mt] += a * part_o[(w * MT + mt) * 64 + lane];
        }
        if (col) {
            const float inv = 1.f / l_tot;
            u16 *orow = out + (t0 * Hq + h) * D + 4 * q4;
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                const bf16x4 v = __builtin_convertvector(o[mt] * inv, bf16x4);
                *reinterpret_cast<u32x2 *>(orow + 16 * mt) = __builtin_bit_cast(u32x2, v);
            }
        }
    }
}

template <int D, bool ROWS>
__global__ __launch_bounds__(kThreads) void prefill_attn_kernel(
    const u16 *__restrict__ q, const u16 *__restrict__ pool_k, const u16 *__restrict__ pool_v,
    int32_t num_blocks, int32_t Hkv, const int32_t *__restrict__ block_tables, int32_t max_blocks, int32_t Hq,
    int32_t T, float scale_log2, float rescale_thr, u16 *__restrict__ out, const AttnWorkMap wm)
{
    using Geo = TileGeom<D>;
    constexpr int CPR = Geo::CPR;
    constexpr int KSTEPS = D / 16;
    constexpr int MT = D / 32;
    constexpr int64_t kPayloadBytes = kBlockSize * D * 2;   // one (block, kv head) of K or V
    constexpr int kSlabs = (int)(kPayloadBytes / 1024);       // 1 KB slabs per payload
    static_assert(kGroupWaves % kSlabs == 0, "slab-to-wave mapping");
    constexpr int kKLoads = Geo::KLOADS, kVLoads = Geo::VLOADS;
    constexpr int RPW = ROWS ? 2 * kRowsPerWG : kRowsPerWG;   // packed rows per workgroup

    // Per group: K buffers 0/1 then V buffers 0/1 (double-buffered, tile j in buffer j&1);
    // with row halves both groups use group 0's. The whole array is reused for the merge
    // at the end of key halves.
    __shared__ __attribute__((aligned(1024))) char lds[2][2 * (Geo::KBYTES + Geo::VBYTES)];

    // XCD-aware order: workgroup L runs on XCD L % 8. The row tiles of one (sequence,
    // kv head), which read the same K/V, go to workgroups of one XCD and share its L2.
    // With the work map and Hkv a multiple of 8, XCD x takes kv heads x, x+8, ... of
    // every sequence, so the eight XCDs get equal work.
    const int tid = threadIdx.x, lane = tid & 63;
    int b, g, rt, p, t0, s;
    {
        const int x = (int)(blockIdx.x % kXcds), i = (int)(blockIdx.x / kXcds);
        const int per_xcd = (int)(gridDim.x / kXcds);
        int j;
        if (Hkv % kXcds == 0) {
            const int hh = i / wm.per_head;
            g = x + kXcds * hh;
            j = i - hh * wm.per_head;
        } else {
            const int w = x * per_xcd + i;
            g = w / wm.per_head;
            j = w - g * wm.per_head;
        }
        if (g >= Hkv) return;
        // Slot of row tile j: the number of slots whose tiles end at or before j. Lane l
        // reads slots l and l + 64 (all fields at once); the slot's fields are then taken
        // from the lane that holds them.
        int e[2], fs[2], fp[2], ft[2], fc[2];
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
            const int k = lane + 64 * hf;
            const bool in = k < wm.n_seq;
            e[hf] = in ? wm.tiles_end[k] : INT32_MAX;
            fs[hf] = in ? wm.seq[k] : 0;
            fp[hf] = in ? wm.prefix[k] : 0;
            ft[hf] = in ? wm.first[k] : 0;
            fc[hf] = in ? wm.count[k] : 0;
        }
        const int slot = __builtin_popcountll(__builtin_amdgcn_ballot_w64(e[0] <= j)) +
                         __builtin_popcountll(__builtin_amdgcn_ballot_w64(e[1] <= j));
        const int hf = slot >> 6, sl = slot & 63;
        b = __builtin_amdgcn_readlane(hf ? fs[1] : fs[0], sl);
        p = __builtin_amdgcn_readlane(hf ? fp[1] : fp[0], sl);
        t0 = __builtin_amdgcn_readlane(hf ? ft[1] : ft[0], sl);
        s = __builtin_amdgcn_readlane(hf ? fc[1] : fc[0], sl);
        rt = __builtin_amdgcn_readlane(hf ? e[1] : e[0], sl) - 1 - j;
    }
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int grp = wave >> 2;              // key halves: which half of the keys; row halves: of the rows
    const int wg = wave & 3;                // wave within the group (selects the rows)
    const int qc = lane & 31, half = lane >> 5;

    const int G = Hq / Hkv;
    const int rows_total = s * G;
    const int row0 = rt * RPW;
    if (s <= 0 || row0 >= rows_total || T <= 0) return;   // uniform over the workgroup
    if (s == 1 && G <= decode_wave::kMaxCols) {           // a decode row (uniform too)
        static_assert(kThreads / 64 * (D / 16) * 64 * 16 + kThreads / 64 * 64 * 8 <= (int)sizeof(lds), "merge area");
        if (t0 < T)
            decode_workgroup<D>(q, pool_k, pool_v, num_blocks, Hkv, block_tables + (int64_t)b * max_blocks,
                                max_blocks, g, G, Hq, p, t0, scale_log2, out, &lds[0][0]);
        return;
    }
    const int total = p + s;

    // This lane's packed query row (rows past the end compute a copy of the last row).
    const int wrow0 = row0 + (ROWS ? grp * kRowsPerWG : 0) + wg * kRowsPerWave;   // this wave's first row
    const int R = wrow0 + qc;
    const bool row_valid = R < rows_total;
    const int Rc = row_valid ? R : rows_total - 1;
    const int i = Rc / G, hl = Rc - i * G;
    const int h = g * G + hl;
    const int limit = p + i;                         // last key this row attends to
    const int64_t tq = (int64_t)t0 + i;

    const int wg_last = min(rows_total - 1, row0 + RPW - 1);
    const int ntiles = (p + wg_last / G) / kTileKeys + 1;
    // key halves: group 0 takes tiles [0, split), group 1 [split, ntiles); row halves:
    // both take every tile
    const int split = ROWS ? ntiles : (ntiles + 1) >> 1;
    const int tile_begin = (!ROWS && grp) ? split : 0;
    const int n = (ROWS || !grp ? split : ntiles) - tile_begin;   // this group's tiles
    const int w_first = min(rows_total - 1, wrow0);
    const int w_min_limit = p + w_first / G;
    const int valid_blocks = min((total + kBlockSize - 1) / kBlockSize, max_blocks);

    // Q^T operand fragments (k-step ks: dims 16ks + 8half .. +7 of this lane's row). The
    // loads go out here; the scaling waits until the first K tile has been requested.
    // All eight loads are unconditional, so that they are in flight together (a row past
    // the end reads row 0 of head 0, which exists since T > 0, and is zeroed later).
    const bool q_ok = tq < T;
    u32x4 q_raw[KSTEPS];
    bf16x8 qf[KSTEPS];    // the Q^T operand, set once K(0) has been requested
    {
        const u16 *qrow = q + (q_ok ? (tq * Hq + h) * D : 0);
#pragma unroll
        for (int ks = 0; ks < KSTEPS; ++ks) q_raw[ks] = *reinterpret_cast<const u32x4 *>(qrow + 16 * ks + 8 * half);
    }

    f32x16 o_acc[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int r = 0; r < 16; ++r) o_acc[mt][r] = 0.f;
    // Scores are kept relative to a reference m_ref (raw units of <q,k>): the first
    // product starts from -m_ref, so S^T holds <q,k> - m_ref and P = exp2(c * S^T) with
    // c = scale_log2.
    float m_ref = 0.f;
    // The reference moves when a tile's max (relative to it) exceeds thr: -inf until the
    // first real score of the row, then rescale_thr = 8 / c, so P stays <= 2^8 and O is
    // rescaled rarely.
    float thr = -INFINITY;
    // Row sums of the bf16 P on the matrix pipe (64 fewer VALU instructions per tile in
    // the softmax than adding the rounded values there, for 4 short MFMAs that fill idle
    // matrix-pipe cycles): v_mfma_f32_16x16x32_bf16 with B = a P^T
    // operand of the second product (read in that instruction's layout: column c = lane%16
    // takes the 8-key runs of lanes c, c+16, c+32, c+48, i.e. queries c and c+16, each over
    // both key halves) and a constant A whose row m is 1 on the runs of query c when m is
    // even and of query c+16 when m is odd. Per tile, four such products (one per P^T
    // operand) start from zero; lane l then holds the tile's sum of query l%16 in
    // tsum[0] and of query l%16+16 in tsum[1], i.e. of its own query (l%32) in
    // tsum[(l >> 4) & 1]. The next softmax adds it to the running sum before any
    // rescale, so the running sum stays one fp32 per lane.
    f32x4 tsum = {0.f, 0.f, 0.f, 0.f};   // the last PV'd tile's sums (zero before the first)
    float l_run = 0.f;                     // this lane's query: sum over the earlier tiles
    bf16x8 sum_pat;
    {
        const __bf16 one = (((lane & 15) ^ (lane >> 4)) & 1) ? (__bf16)0.f : (__bf16)1.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) sum_pat[e] = one;
    }
    f32x16 nbias;
#pragma unroll
    for (int r = 0; r < 16; ++r) nbias[r] = 0.f;

    const int32_t *bt = block_tables + (int64_t)b * max_blocks;
    const int lgrp = ROWS ? 0 : grp;        // whose tile buffers this group reads
    auto kbuf = [&](int j) __attribute__((always_inline)) { return &lds[lgrp][(j & 1) * Geo::KBYTES]; };
    auto vbuf = [&](int j) __attribute__((always_inline)) { return &lds[lgrp][2 * Geo::KBYTES + (j & 1) * Geo::VBYTES]; };
    // The same buffers as LDS byte addresses, for the direct loads (no generic-pointer casts).
    const uint32_t lds_addr = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char *)&lds[lgrp][0];
    auto kbuf_off = [&](int j) __attribute__((always_inline)) { return (uint32_t)((j & 1) * Geo::KBYTES); };
    auto vbuf_off = [&](int j) __attribute__((always_inline)) { return (uint32_t)(2 * Geo::KBYTES + (j & 1) * Geo::VBYTES); };

    // Pool block ids of this group's tile j, read raw (as scalars) one phase before
    // use. Logical blocks past the sequence read the last valid entry, so the four loads
    // are independent and nothing consumes their values until the range check at use:
    // every key past the sequence is masked and the V entries past it are cleared in
    // the last tile, so any in-pool block can stand in there; an id outside the pool
    // becomes block 0, so no load ever leaves the pool.
    const char *bt_bytes = reinterpret_cast<const char *>(bt);
    auto tile_ids = [&](int j, int32_t (&ids)[kTileBlocks]) __attribute__((always_inline)) {
#pragma unroll
        for (int jb = 0; jb < kTileBlocks; ++jb) {
            const uint32_t lb = (uint32_t)min((tile_begin + j) * kTileBlocks + jb, valid_blocks - 1);
            ids[jb] = *reinterpret_cast<const int32_t *>(bt_bytes + lb * 4u);   // 32-bit offset form
        }
    };
    // Byte offset of the (pool block, kv head g) payload of a raw block id; an id outside
    // the pool becomes block 0. (blk * Hkv + g fits in 32 bits for any pool that fits in
    // memory: 2^32 payloads would be 8 TB.)
    auto payload_off = [&](int32_t blk) __attribute__((always_inline)) -> int64_t {
        const uint32_t b = (uint32_t)blk < (uint32_t)num_blocks ? (uint32_t)blk : 0u;
        return (int64_t)(b * (uint32_t)Hkv + (uint32_t)g) * kPayloadBytes;
    };
    auto to_offs = [&](const int32_t (&ids)[kTileBlocks], int64_t (&offs)[kTileBlocks]) __attribute__((always_inline)) {
#pragma unroll
        for (int jb = 0; jb < kTileBlocks; ++jb) offs[jb] = payload_off(ids[jb]);
    };
    int32_t ids_raw[kTileBlocks];   // ids of the tile two ahead, read in a vector cluster
    // Direct-load addressing. A tile's K (or V) is 4 pool blocks of one kv head, each a
    // contiguous payload of kSlabs 1 KB slabs; wave wg loads slabs u*4 + wg. Because 4
    // is a multiple of kSlabs, a lane's byte offset inside the payload is the same for
    // every u, so it is computed once here; the LDS swizzle is applied through it.
    const char *pool_k_bytes = reinterpret_cast<const char *>(pool_k);
    const char *pool_v_bytes = reinterpret_cast<const char *>(pool_v);
    uint32_t k_off, v_off;
    {
        const int chunk = (wg % kSlabs) * 64 + lane;          // 16-B chunk within the payload
        const int key = chunk / CPR, pc = chunk % CPR;        // K: row (slot) and chunk of the row
        k_off = (uint32_t)(key * 2 * D + ((pc ^ k_swizzle<CPR>(key)) * 16));
        const int d = chunk >> 1, pch = chunk & 1;            // V: dim and half of its 16 slots
        v_off = (uint32_t)(d * 2 * kBlockSize + ((pch ^ ((d >> 3) & 1)) * 16));
    }

    // Direct loads of this group's tile j (K or V) into its buffer; 1 KB slab per
    // wave-wide load; the LDS swizzle is applied through each lane's source.
    // One direct load (load u of the tile's K or V) of this group's tile j into its buffer:
    // a 1 KB slab per wave-wide load; the LDS swizzle is applied through each lane's source.
    auto load_k = [&](int j, const int64_t (&offs)[kTileBlocks], int u) __attribute__((always_inline)) {
        const int slab = u * kGroupWaves + wg;                             // wave-uniform
        dma16(pool_k_bytes + offs[slab / kSlabs], k_off, lds_addr + kbuf_off(j) + slab * 1024);
    };
    auto load_v = [&](int j, const int64_t (&offs)[kTileBlocks], int u) __attribute__((always_inline)) {
        const int slab = u * kGroupWaves + wg;
        dma16(pool_v_bytes + offs[slab / kSlabs], v_off, lds_addr + vbuf_off(j) + slab * 1024);
    };
    auto issue_k = [&](int j, const int64_t (&offs)[kTileBlocks]) __attribute__((always_inline)) {
#pragma unroll
        for (int u = 0; u < kKLoads; ++u) load_k(j, offs, u);
    };

    // ---- matrix work: O^T += V^T(j) P^T(j), k-step t = pool block t of the tile.
    // In the tile holding the sequence end, V entries of keys >= total are cleared
    // in the operand (their slots may hold anything; 0 * NaN would poison O).
    auto pv = [&](int j, const bf16x8 (&pf)[kTileBlocks], auto clear_tag) __attribute__((always_inline)) {
        constexpr bool CLEAR = decltype(clear_tag)::value;
        const char *tv = vbuf(j);
        const int vlim = total - (tile_begin + j) * kTileKeys;     // valid keys in the tile
#pragma unroll
        for (int t = 0; t < kTileBlocks; ++t) {
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                const int d = 32 * mt + qc;
                const int pch = half ^ ((d >> 3) & 1);
                u32x4 raw = *reinterpret_cast<const u32x4 *>(tv + ((t * D + d) * 2 + pch) * 16);
                if constexpr (CLEAR) {
                    const int nvalid = vlim - 16 * t - 8 * half;   // valid keys among this lane's 8
#pragma unroll
                    for (int wd = 0; wd < 4; ++wd)
                        raw[wd] &= (2 * wd < nvalid ? 0x0000FFFFu : 0u) | (2 * wd + 1 < nvalid ? 0xFFFF0000u : 0u);
                }
                o_acc[mt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(raw), pf[t], o_acc[mt], 0, 0, 0);
            }
            tsum = __builtin_amdgcn_mfma_f32_16x16x32_bf16(sum_pat, pf[t], t == 0 ? f32x4{0.f, 0.f, 0.f, 0.f} : tsum,
                                                           0, 0, 0);
        }
    };

    // ---- matrix cluster: PV(j) (optional) then QK(j+1) (optional) as one stream of
    // (LDS fragment, MFMA) pairs, the fragment reads running kAhead pairs ahead (a single
    // wave gets about one 1 KB LDS read per MFMA time, so reads must stay in flight
    // behind the MFMAs). When QK runs, the cluster also issues the direct loads of
    // V(j+1) and K(j+2), one per few MFMAs, so the texture path never backs up a wave.
    auto matrix_cluster = [&](auto pv_tag, auto qk_tag, int j, const bf16x8 (&pf)[kTileBlocks],
                              f32x16 (&st)[2], int64_t (&idv)[kTileBlocks], int64_t (&idk)[kTileBlocks],
                              auto convert_tag, auto load_tag) __attribute__((always_inline)) {
        constexpr bool DO_PV = decltype(pv_tag)::value, DO_QK = decltype(qk_tag)::value;
        constexpr bool LOADS = decltype(load_tag)::value;

        constexpr int NPV = DO_PV ? kTileBlocks * MT : 0, NQK = DO_QK ? 2 * KSTEPS : 0, NALL = NPV + NQK;
        constexpr int NLD = DO_QK && LOADS ? kVLoads + kKLoads : 0;
        constexpr int NLD1 = NLD > 0 ? NLD : 1;
        constexpr int EVERY = NALL / NLD1 > 0 ? NALL / NLD1 : 1;
        constexpr int kAhead = KAHEAD;
        const char *tv = vbuf(j);
        const char *tk = kbuf(j + 1);
        auto frag = [&](int i) __attribute__((always_inline)) -> u32x4 {
            if (i < NPV) {
                const int t = i / MT, mt = i % MT;
                const int d = 32 * mt + qc;
                const int pch = half ^ ((d >> 3) & 1);
                return *reinterpret_cast<const u32x4 *>(tv + ((t * D + d) * 2 + pch) * 16);
            }
            const int m = (i - NPV) / KSTEPS, ks = (i - NPV) % KSTEPS;
            const int krow = 32 * m + key_of_row(qc);
            const int pc = (2 * ks + half) ^ k_swizzle<CPR>(krow);
            return *reinterpret_cast<const u32x4 *>(tk + (krow * CPR + pc) * 16);
        };
        // The wave in its matrix cluster takes issue priority over the other wave of its
        // SIMD (in its vector cluster): otherwise the older wave of each SIMD always wins
        // arbitration and the younger group is late in every phase.
        __builtin_amdgcn_s_setprio(1);
        u32x4 fr[NALL];
#pragma unroll
        for (int i = 0; i < kAhead && i < NALL; ++i) fr[i] = frag(i);
        __builtin_amdgcn_sched_barrier(0);
        if constexpr (decltype(convert_tag)::value && LOADS) {
            // Block ids read in the preceding vector cluster (and waited for at its end)
            // become payload offsets here, while the first fragment reads are in flight.
#pragma unroll
            for (int jb = 0; jb < kTileBlocks; ++jb) {
                idv[jb] = idk[jb];
                idk[jb] = payload_off(ids_raw[jb]);
            }
            __builtin_amdgcn_sched_barrier(0);
        }
        int ld = 0;
#pragma unroll
        for (int i = 0; i < NALL; ++i) {
            if (i + kAhead < NALL) fr[i + kAhead] = frag(i + kAhead);
            if (i < NPV) {
                const int t = i / MT, mt = i % MT;
                o_acc[mt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(fr[i]), pf[t], o_acc[mt], 0, 0, 0);
                if (mt == MT - 1)
                    tsum = __builtin_amdgcn_mfma_f32_16x16x32_bf16(sum_pat, pf[t],
                                                                   t == 0 ? f32x4{0.f, 0.f, 0.f, 0.f} : tsum, 0, 0, 0);
            } else {
                const int m = (i - NPV) / KSTEPS, ks = (i - NPV) % KSTEPS;
                st[m] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(fr[i]), qf[ks], ks == 0 ? nbias : st[m],
                                                                0, 0, 0);
            }
            if (NLD && i % EVERY == EVERY - 1 && ld < NLD) {
                if (ld < kVLoads) load_v(j + 1, idv, ld);
                else load_k(j + 2, idk, ld - kVLoads);
                ++ld;
            }
        }
        // keep that schedule: (read, MFMA[, load]) groups, then the last MFMAs
#pragma unroll
        for (int i = 0; i < NALL; ++i) {
            if (i + kAhead < NALL) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
            if (i < NPV && i % MT == MT - 1)   // PV MFMA, then the row-sum MFMA
                __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
            else
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        }
        __builtin_amdgcn_sched_barrier(0);
        __builtin_amdgcn_s_setprio(0);
    };

    // ---- vector work: online softmax of S^T(j) into bf16 P(j) (lazy rescale) ----
    auto softmax = [&](int j, f32x16 (&st)[2], bf16x8 (&pf)[kTileBlocks]) __attribute__((always_inline)) {
        l_run += (lane & 16) ? tsum[1] : tsum[0];   // tile j-1 (zero before the first tile)
        const int kbase = (tile_begin + j) * kTileKeys;
        if (kbase + kTileKeys - 1 > w_min_limit) {
            // register r of half tile m holds key kbase + 32m + 16(r/8) + 8half + r%8
            const int lim = limit - kbase - 8 * half;
#pragma unroll
            for (int m = 0; m < 2; ++m)
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    st[m][r] = (32 * m + 16 * (r >> 3) + (r & 7)) > lim ? -INFINITY : st[m][r];
        }
        // NaN-propagating maximum (v_maximum3_f32): unlike fmaxf it needs no
        // canonicalisation of the MFMA results. Written as two chains of
        // max(max(m, a), b), one three-operand instruction per two scores; a pairwise
        // tree would spend a three-operand instruction on every pair.
        float mc[2];
#pragma unroll
        for (int m = 0; m < 2; ++m) {
            mc[m] = __builtin_elementwise_maximum(st[m][0], st[m][1]);
#pragma unroll
            for (int r = 2; r < 16; r += 2)
                mc[m] = __builtin_elementwise_maximum(__builtin_elementwise_maximum(mc[m], st[m][r]), st[m][r + 1]);
        }
        float mx = __builtin_elementwise_maximum(mc[0], mc[1]);
        {   // The other half-wave holds the other 32 keys of the same query: swap halves and
            // take the larger. The two swap results are copied out of the returned vector
            // before the bit casts: a bit cast applied to an element of it directly reads
            // element 0 for both, which drops the half-wave's own keys from its max.
            const unsigned mine = __builtin_bit_cast(unsigned, mx);
            const auto sw = __builtin_amdgcn_permlane32_swap(mine, mine, false, false);
            const unsigned lo = sw[0], hi = sw[1];
            mx = __builtin_elementwise_maximum(__builtin_bit_cast(float, lo), __builtin_bit_cast(float, hi));
        }
        const bool need = mx > thr;
        if (__builtin_amdgcn_ballot_w64(need)) {
            const float delta = need ? mx : 0.f;
            // Before a row's first real score nothing has accumulated, and that first max
            // may lie far below the initial reference (2^-delta would overflow to +inf
            // and turn the zero accumulators into NaN): scale by 0 then.
            const float alpha = thr == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(-delta * scale_log2);
            thr = need ? rescale_thr : thr;
            m_ref += delta;
            l_run *= alpha;
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                for (int r = 0; r < 16; ++r) o_acc[mt][r] *= alpha;
#pragma unroll
            for (int m = 0; m < 2; ++m)
#pragma unroll
                for (int r = 0; r < 16; ++r) st[m][r] -= delta;
#pragma unroll
            for (int r = 0; r < 16; ++r) nbias[r] = -m_ref;
        }
        // P rounded to bf16 is both the second product's operand and what the row sums
        // add (on the matrix pipe, see tsum): the weights then sum to one however P
        // rounds (a one-hot row returns its V row exactly), where a sum of the fp32
        // values would leave up to 2^-8 of relative error on a dominant term.
#pragma unroll
        for (int t = 0; t < kTileBlocks; ++t) {
            f32x8 pv8;
#pragma unroll
            for (int e = 0; e < 8; ++e)
                pv8[e] = __builtin_amdgcn_exp2f(st[t >> 1][8 * (t & 1) + e] * scale_log2);
            pf[t] = __builtin_convertvector(pv8, bf16x8);
        }
    };

    // Ping-pong schedule. Each group runs the cluster sequence
    //   C(-1), M(0), C(0), M(1), C(1), ..., M(n-1), C(n-1)
    // with C(j) = [PV(j), QK(j+1), direct loads of V(j+1) and K(j+2)] (matrix) and
    // M(j) = [softmax(j)] (vector). Group 1 runs one phase behind group 0, so in every
    // phase each SIMD has one wave in a matrix cluster and one in a vector cluster.
    // Every phase ends with a workgroup barrier (both groups pass the same number);
    // the loads issued in C(j) are waited for at the end of M(j+1), one phase before
    // C(j+1) reads them. Rows whose causal limit ends before a tile get P = 0 there.
    // Block offsets travel one phase ahead: at C(j), ids_v holds tile j+1's (for
    // V(j+1)) and ids_k tile j+2's (for K(j+2)).
    // With row halves both groups walk the same tiles, and only group 0 loads them:
    // group 1 reads group 0's buffers one phase later. Two buffers per operand still
    // suffice: group 0's C(j) (phase 2j+2 counted from the first barrier) overwrites the
    // buffers of V(j-1) and K(j), whose last reader is group 1's C(j-1) in phase 2j+1,
    // and the barrier between phases orders the two. The LDS then takes one tile's
    // direct-load writes per two phases instead of two, on a path whose fragment reads
    // already run near its bandwidth.
    const bool loader = !ROWS || grp == 0;
    int64_t ids_v[kTileBlocks], ids_k[kTileBlocks];   // payload byte offsets
    tile_ids(0, ids_raw);
    to_offs(ids_raw, ids_v);
    if (n > 0 && loader) issue_k(0, ids_v);            // K(0) for C(-1)
    tile_ids(1, ids_raw);
    to_offs(ids_raw, ids_k);
    // Q^T operand fragments (k-step ks: dims 16ks + 8half .. +7 of this lane's row),
    // the bf16 input as it is.
#pragma unroll
    for (int ks = 0; ks < KSTEPS; ++ks) qf[ks] = as_bf16x8(q_ok ? q_raw[ks] : u32x4{0u, 0u, 0u, 0u});
    wait_vmem();
    __syncthreads();

    const int n0 = split, n1 = ROWS ? ntiles : ntiles - split;
    const int phases = max(2 * n0 + 1, 2 * n1 + 2);
    int ph = 0;
    auto phase_end = [&]() __attribute__((always_inline)) {
        phase_barrier();
        ++ph;
    };
    // M(j): softmax of tile j; block ids of tile j+2 (read now, range-checked and
    // converted at the start of C(j)) when this group loads; then wait for the loads
    // C(j-1) issued.
    auto vector_cluster = [&](int j, f32x16 (&st)[2], bf16x8 (&pf)[kTileBlocks], auto load_tag) __attribute__((always_inline)) {
        // The scalar loads of the ids go out before the softmax, whose length covers
        // their latency (left to itself the scheduler sinks them next to their use).
        if constexpr (decltype(load_tag)::value) tile_ids(j + 2, ids_raw);
        __builtin_amdgcn_sched_barrier(0);
        softmax(j, st, pf);
        wait_vmem();
        // The id loads landed long ago; an explicit wait here (seen by the compiler) keeps
        // it from placing one among the next matrix cluster's fragment reads.
        __builtin_amdgcn_sched_barrier(0);
        __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
    };

    f32x16 st[2];
    bf16x8 pf[kTileBlocks];
    if (grp == 1) phase_end();
    // The tile loop, instantiated once for a group that loads and once for one that
    // only reads (row halves, group 1), so that no branch splits a matrix cluster.
    auto run_tiles = [&](auto load_tag) __attribute__((always_inline)) {
        constexpr std::true_type T_{};
        constexpr std::false_type F_{};
        // C(-1): QK(0), loads of V(0) and K(1) (K(1) lands in an unused buffer if n == 1)
        matrix_cluster(F_, T_, -1, pf, st, ids_v, ids_k, F_, load_tag);
        phase_end();
        // Four (M, C) pairs per iteration: the scores made in one pair's matrix cluster
        // feed the next pair's softmax in the same registers, and the register copies
        // that the loop-carried scores and the softmax shift cost at the iteration
        // boundary are paid once per four tiles (about 0.7% faster than two pairs).
        // C(j): PV(j), QK(j+1), loads of V(j+1) and K(j+2) (the last K lands unused).
        int j = 0;
        for (; j + 4 < n; j += 4) {
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                vector_cluster(j + u, st, pf, load_tag);
                phase_end();
                matrix_cluster(T_, T_, j + u, pf, st, ids_v, ids_k, T_, load_tag);
                phase_end();
            }
        }
        for (; j + 2 < n; j += 2) {
            vector_cluster(j, st, pf, load_tag);
            phase_end();
            matrix_cluster(T_, T_, j, pf, st, ids_v, ids_k, T_, load_tag);
            phase_end();
            vector_cluster(j + 1, st, pf, load_tag);
            phase_end();
            matrix_cluster(T_, T_, j + 1, pf, st, ids_v, ids_k, T_, load_tag);
            phase_end();
        }
        if (j + 1 < n) {
            vector_cluster(j, st, pf, load_tag);
            phase_end();
            matrix_cluster(T_, T_, j, pf, st, ids_v, ids_k, T_, load_tag);
            phase_end();
        }
        vector_cluster(n - 1, st, pf, load_tag);
        phase_end();
        // The group's last tile may hold the sequence end: clear V past it.
        if ((tile_begin + n) * kTileKeys > total) pv(n - 1, pf, T_);
        else matrix_cluster(T_, F_, n - 1, pf, st, ids_v, ids_k, F_, load_tag);
        phase_end();
    };
    if (n > 0) {
        if (loader) run_tiles(std::true_type{});
        else run_tiles(std::false_type{});
    }
    while (ph < phases) phase_end();

    if constexpr (ROWS) {
        // ---- row halves: every group saw all keys of its rows; normalise, store ----
        const float inv = 1.f / (l_run + ((lane & 16) ? tsum[1] : tsum[0]));
        if (row_valid && tq < T) {
            u16 *orow = out + (tq * Hq + h) * D;
#pragma unroll
            for (int k = 0; k < MT; ++k)
#pragma unroll
                for (int r4 = 0; r4 < 4; ++r4) {
                    f32x4 v;
#pragma unroll
                    for (int c = 0; c < 4; ++c) v[c] = o_acc[k][4 * r4 + c] * inv;
                    const bf16x4 bv = __builtin_convertvector(v, bf16x4);
                    const int d0 = 32 * k + 8 * r4 + 4 * half;
                    *reinterpret_cast<u32x2 *>(orow + d0) = __builtin_bit_cast(u32x2, bv);
                }
        }
        return;
    }

    // ---- key halves: merge the two halves through LDS, normalise, store ----
    // Each group finalises half of the head dims (group 0 the first MT/2 blocks of 32,
    // group 1 the rest): it sends the partner wave holding the same rows the other half
    // of its accumulator and its (m, l), then merges the half it received.
    const float l_tot = l_run + ((lane & 16) ? tsum[1] : tsum[0]);   // plus the group's last tile
    const bool has_ref = thr > -INFINITY;      // this row saw a real score in this key half
    constexpr int MH = MT / 2;
    constexpr int XW = 4 * MH + 1;                 // float4 slots per lane: half of O, then (m, l)
    static_assert(2 * kGroupWaves * XW * 64 * 16 <= (int)sizeof(lds), "merge area");
    const int my0 = grp ? MH : 0, other0 = grp ? 0 : MH;
    __syncthreads();
    f32x4 *xch = reinterpret_cast<f32x4 *>(&lds[0][0]);
    {
        f32x4 *xo = xch + (size_t)(grp * kGroupWaves + wg) * XW * 64;
#pragma unroll
        for (int k = 0; k < MH; ++k)
#pragma unroll
            for (int r4 = 0; r4 < 4; ++r4) {
                f32x4 v;
#pragma unroll
                for (int c = 0; c < 4; ++c) v[c] = o_acc[other0 + k][4 * r4 + c];
                xo[(k * 4 + r4) * 64 + lane] = v;
            }
        xo[(XW - 1) * 64 + lane] = f32x4{has_ref ? m_ref : -INFINITY, l_tot, 0.f, 0.f};
    }
    __syncthreads();

    const f32x4 *xi = xch + (size_t)((1 - grp) * kGroupWaves + wg) * XW * 64;
    const f32x4 ml = xi[(XW - 1) * 64 + lane];
    const float m1 = ml[0], l1 = ml[1];
    const float m0 = has_ref ? m_ref : -INFINITY;
    const float mm = fmaxf(m0, m1);
    const float a0 = (m0 == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f((m0 - mm) * scale_log2);
    const float a1 = (m1 == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f((m1 - mm) * scale_log2);
    const float inv = 1.f / (a0 * l_tot + a1 * l1);
    if (row_valid && tq < T) {
        u16 *orow = out + (tq * Hq + h) * D;
#pragma unroll
        for (int k = 0; k < MH; ++k)
#pragma unroll
            for (int r4 = 0; r4 < 4; ++r4) {
                const f32x4 o1 = xi[(k * 4 + r4) * 64 + lane];
                f32x4 v;
#pragma unroll
                for (int c = 0; c < 4; ++c) v[c] = (a0 * o_acc[my0 + k][4 * r4 + c] + a1 * o1[c]) * inv;
                const bf16x4 bv = __builtin_convertvector(v, bf16x4);
                const int d0 = 32 * (my0 + k) + 8 * r4 + 4 * half;
                *reinterpret_cast<u32x2 *>(orow + d0) = __builtin_bit_cast(u32x2, bv);
            }
    }
}

}  // namespace

int attn_rows_per_workgroup(int) { return kRowsPerWG; }

namespace {
// Schedule override (pcr_prefill_attn_set_schedule): 0 chooses per launch.
std::atomic<int> g_schedule{PCR_ATTN_SCHEDULE_AUTO};

template <int D, bool ROWS>
void launch_attn(dim3 grid, hipStream_t s, const u16 *qq, const u16 *pk, const u16 *pv, const pcr_kv_pool &pool,
                 const int32_t *block_tables, int32_t max_blocks, int32_t num_q_heads, int32_t T, float scale_log2,
                 float rescale_thr, u16 *oo, const AttnWorkMap &wm)
{
    hipLaunchKernelGGL((prefill_attn_kernel<D, ROWS>), grid, dim3(kThreads), 0, s, qq, pk, pv, pool.num_blocks,
                       pool.num_kv_heads, block_tables, max_blocks, num_q_heads, T, scale_log2, rescale_thr, oo,
                       wm);
}

// One launch over the sequences seq[0..n) (each with new tokens, n <= kMaxMapSeqs,
// longest context first): builds the work map, picks the schedule, launches.
hipError_t launch_group(const int32_t *seq, int n, const u16 *qq, const pcr_kv_pool &pool,
                        const int32_t *block_tables, int32_t max_blocks, const int32_t *host_prefix_lens,
                        const int32_t *host_cu_suffix, int32_t num_q_heads, int32_t T, float scale_log2,
                        float rescale_thr, u16 *oo, hipStream_t s, int auto_schedule, int n_cu)
{
    const int Hkv = pool.num_kv_heads, G = num_q_heads / Hkv;
    auto rows_of = [&](int32_t b) { return ((int64_t)host_cu_suffix[b + 1] - host_cu_suffix[b]) * G; };
    int64_t tiles_rows = 0;   // row tiles of 256 rows over the group's sequences, one kv head
    for (int k = 0; k < n; ++k) tiles_rows += (rows_of(seq[k]) + 2 * kRowsPerWG - 1) / (2 * kRowsPerWG);
    // Row halves when the launch keeps at least two workgroups per compute unit
    // with them (each workgroup then pays its start-up and end for twice the work),
    // unless the caller prefers key halves (shorter workgroups free a compute unit
    // sooner for copy kernels that share the device).
    int sched = g_schedule.load(std::memory_order_relaxed);
    if (sched == PCR_ATTN_SCHEDULE_AUTO) sched = auto_schedule;
    const bool rows = sched == PCR_ATTN_SCHEDULE_ROW_HALVES ||
                      (sched == PCR_ATTN_SCHEDULE_AUTO && tiles_rows * Hkv >= 2 * (int64_t)n_cu);
    const int64_t rpw = rows ? 2 * kRowsPerWG : kRowsPerWG;
    auto tiles_of = [&](int32_t b) { return (rows_of(b) + rpw - 1) / rpw; };

    // Slot order: the given order (longest context first), with the decode rows (one
    // new token, one workgroup each, bound by HBM) spread evenly over the prefill
    // tiles (bound by the matrix cores): run back to back they would take every
    // compute unit at once and queue on HBM.
    AttnWorkMap wm;
    {
        const bool dec_rows = G <= decode_wave::kMaxCols;
        int32_t pre[kMaxMapSeqs], dec[kMaxMapSeqs];
        int np = 0, nd = 0;
        int64_t pre_tiles = 0;
        for (int k = 0; k < n; ++k) {
            if (dec_rows && rows_of(seq[k]) == G) {
                dec[nd++] = seq[k];
            } else {
                pre[np++] = seq[k];
                pre_tiles += tiles_of(seq[k]);
            }
        }
        int m = 0, di = 0;
        int64_t done = 0;
        for (int k = 0; k < np; ++k) {
            wm.seq[m++] = pre[k];
            done += tiles_of(pre[k]);
            for (; di < nd && (int64_t)di * pre_tiles < (int64_t)nd * done; ++di) wm.seq[m++] = dec[di];
        }
        for (; di < nd; ++di) wm.seq[m++] = dec[di];
    }
    int32_t cum = 0;
    for (int k = 0; k < n; ++k) {
        const int32_t b = wm.seq[k];
        cum += (int32_t)tiles_of(b);
        wm.tiles_end[k] = cum;
        wm.prefix[k] = host_prefix_lens[b];
        wm.first[k] = host_cu_suffix[b];
        wm.count[k] = host_cu_suffix[b + 1] - host_cu_suffix[b];
    }
    wm.n_seq = n;
    wm.per_head = cum;
    const int64_t n_items = (Hkv % kXcds == 0) ? (int64_t)cum * Hkv : ((int64_t)cum * Hkv + kXcds - 1) / kXcds * kXcds;
    const dim3 grid((unsigned)n_items);
    auto *pk = static_cast<const u16 *>(pool.k);
    auto *pv = static_cast<const u16 *>(pool.v);
    if (pool.head_dim == 128) {
        if (rows)
            launch_attn<128, true>(grid, s, qq, pk, pv, pool, block_tables, max_blocks, num_q_heads, T, scale_log2,
                                   rescale_thr, oo, wm);
        else
            launch_attn<128, false>(grid, s, qq, pk, pv, pool, block_tables, max_blocks, num_q_heads, T, scale_log2,
                                    rescale_thr, oo, wm);
    } else {
        if (rows)
            launch_attn<64, true>(grid, s, qq, pk, pv, pool, block_tables, max_blocks, num_q_heads, T, scale_log2,
                                  rescale_thr, oo, wm);
        else
            launch_attn<64, false>(grid, s, qq, pk, pv, pool, block_tables, max_blocks, num_q_heads, T, scale_log2,
                                   rescale_thr, oo, wm);
    }
    return hipGetLastError();
}
}  // namespace

void attn_set_schedule(int schedule) { g_schedule.store(schedule, std::memory_order_relaxed); }

hipError_t launch_prefix_prefill_attn(const void *q, const pcr_kv_pool &pool,
                                      const int32_t *block_tables, int32_t max_blocks,
                                      const int32_t *host_prefix_lens, const int32_t *host_cu_suffix,
                                      int32_t B, int32_t num_q_heads, int32_t T, float sm_scale, void *out,
                                      hipStream_t s, int auto_schedule, int n_cu)
{
    // The sequences with new tokens, longest context first.
    std::vector<int32_t> seq;
    seq.reserve((size_t)std::max(B, 0));
    for (int32_t b = 0; b < B; ++b)
        if (host_cu_suffix[b + 1] > host_cu_suffix[b]) seq.push_back(b);
    if (seq.empty()) return hipSuccess;
    auto keys = [&](int32_t b) { return (int64_t)host_prefix_lens[b] + host_cu_suffix[b + 1] - host_cu_suffix[b]; };
    std::stable_sort(seq.begin(), seq.end(), [&](int32_t a, int32_t c) { return keys(a) > keys(c); });
    const float scale_log2 = sm_scale * kLog2e;
    const float rescale_thr = kRescaleThreshold / scale_log2;   // in units of <q,k>
    auto *qq = static_cast<const u16 *>(q);
    auto *oo = static_cast<u16 *>(out);
    // More sequences than one work map holds: consecutive launches on the stream, the
    // sequences dealt round robin (sequence k of the sorted list to launch k mod
    // n_launch), so that every launch gets the same mix of long and short ones.
    const int n_act = (int)seq.size();
    const int n_launch = (n_act + kMaxMapSeqs - 1) / kMaxMapSeqs;
    int32_t group[kMaxMapSeqs];
    for (int l = 0; l < n_launch; ++l) {
        int n = 0;
        for (int k = l; k < n_act; k += n_launch) group[n++] = seq[k];
        const hipError_t e = launch_group(group, n, qq, pool, block_tables, max_blocks, host_prefix_lens,
                                          host_cu_suffix, num_q_heads, T, scale_log2, rescale_thr, oo, s,
                                          auto_schedule, n_cu);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace pcr
