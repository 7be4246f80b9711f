// One wave's chunk of a decode row: the keys [kbeg, kend) of one (sequence, kv head),
// for the G query heads of that kv head (the rows of one new token; Sec. 2.2 with a
// one-token suffix). Shared by the decode kernel (decode.hip) and by the decode
// workgroups of the prefill kernel (attn.hip).
//
// The wave holds the G <= 16 query heads as the columns of v_mfma_f32_16x16x32_bf16
// tiles and walks its chunk 32 keys (two pool blocks) at a time:
//   S^T[key][h] = K Q^T     A = 16 key rows x 32 dims of K,  B = Q^T (registers)
//   O^T[d][h]  += V^T P^T   A = 16 dims x 32 keys of V^T,    B = P^T (registers)
// No operand is shared between waves, so K and V go from HBM straight into registers:
// K is key-major and V d-major inside each pool block, so every A operand is one
// 16-byte run. Lane (c, q4) (c = lane % 16, q4 = lane / 16) loads key row
// 8*(c/4) + 4r + c%4 for the r-th K product, so that its eight scores are keys
// 8*q4 .. 8*q4 + 7 of the step, which are exactly its eight P^T operand values in the
// V product: the softmax is in-lane apart from the column max over the four lanes of
// a column. NSETS register sets of one step's K/V rotate (NSETS - 1 steps in flight
// while one is used). Every byte is used once, so V loads are non-temporal; K loads are
// non-temporal too when the caller streams HBM at full rate with every wave (K_CACHED
// false), and ordinary loads otherwise: a key row's 128-byte lines are read in two
// 64-byte halves by two load instructions (dims 32*kk .. for kk = 0, 1 and 2, 3), and
// an ordinary load lets the vector L1 fetch each line once. Measured: a compute unit running one decode workgroup alone moved 37 GB/s
// with non-temporal K loads and 47 GB/s with ordinary ones, while a batch that keeps
// HBM busy with every wave ran 2% slower with ordinary K loads.
//
// Result per lane: the unnormalised O^T columns it holds, the running max (log2
// domain, scaled) and the running sum of the bf16-rounded probabilities over this
// lane's keys (the caller adds the four q4 lanes of a column).
#pragma once

#include "pcr_internal.h"

namespace pcr {
namespace decode_wave {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned short u16;

constexpr int kStepKeys = 32;   // keys per step: two pool blocks
constexpr int kMaxCols = 16;    // query heads per kv head that one wave's tiles hold

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

template <int D>
struct StepRegs {
    u32x4 k[2][D / 32];   // K operands of the two products (row group r, dims 32*kk ..)
    u32x4 v[D / 16];      // V^T operands (dims 16*mt ..)
};

// qrow: this lane's query row (head g*G + c, or any valid row when c >= G) plus 8*q4.
// bt_row: the sequence's block-table row; last_blk: its last block with a visible key.
template <int D, int NSETS, bool K_CACHED>
__device__ __forceinline__ void chunk(const u16 *__restrict__ qrow, bool col, const u16 *__restrict__ pool_k,
                                      const u16 *__restrict__ pool_v, int32_t num_blocks, int32_t Hkv, int g,
                                      const int32_t *__restrict__ bt_row, int last_blk, int kbeg, int kend,
                                      float scale_log2, f32x4 (&o)[D / 16], float &m_run, float &l_run)
{
    static_assert(NSETS == 2 || NSETS == 3, "two or three register sets");
    constexpr int KK = D / 32;    // K products per row group (32 dims each)
    constexpr int MT = D / 16;    // V products (16 dims each)
    const int lane = (int)(threadIdx.x & 63);
    const int c = lane & 15, q4 = lane >> 4;

    // Q^T operands: lane (c, q4) holds dims 32*kk + 8*q4 .. +7 of its head (zero past G).
    u32x4 qf[KK];
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
        const u32x4 raw = *reinterpret_cast<const u32x4 *>(qrow + 32 * kk);
        qf[kk] = col ? raw : u32x4{0u, 0u, 0u, 0u};
    }

    auto block_id = [&](int li) __attribute__((always_inline)) -> int32_t {
        const int32_t id = bt_row[min(li, last_blk)];
        return (uint32_t)id < (uint32_t)num_blocks ? id : 0;   // a bad entry reads block 0, never outside
    };
    const int krow = 8 * ((c >> 2) & 1) + (c & 3);    // slot of row group 0; row group 1 is 4 slots on
    auto load_step = [&](int step, StepRegs<D> &R) __attribute__((always_inline)) {
        const int li = (kbeg + step * kStepKeys) >> 4;
        const int32_t b0 = block_id(li), b1 = block_id(li + 1);
        const int32_t kb = (c >> 3) ? b1 : b0;
        const int32_t vb = (q4 >> 1) ? b1 : b0;
        const u16 *kp = pool_k + ((int64_t)kb * Hkv + g) * (kBlockSize * D) + krow * D + 8 * q4;
        const u16 *vp = pool_v + ((int64_t)vb * Hkv + g) * (kBlockSize * D) + c * kBlockSize + 8 * (q4 & 1);
#pragma unroll
        for (int r = 0; r < 2; ++r)
#pragma unroll
            for (int kk = 0; kk < KK; ++kk)
            {
                const u32x4 *kq = reinterpret_cast<const u32x4 *>(kp + 4 * r * D + 32 * kk);
                if constexpr (K_CACHED)
                    R.k[r][kk] = *kq;
                else
                    R.k[r][kk] = __builtin_nontemporal_load(kq);
            }
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
            R.v[mt] = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(vp + 16 * mt * kBlockSize));
    };

    m_run = -INFINITY;
    l_run = 0.f;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) o[mt] = f32x4{0.f, 0.f, 0.f, 0.f};

    auto process = [&](int step, const StepRegs<D> &R) __attribute__((always_inline)) {
        f32x4 s[2];
#pragma unroll
        for (int r = 0; r < 2; ++r) {
            s[r] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kk = 0; kk < KK; ++kk)
                s[r] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(R.k[r][kk]), as_bf16x8(qf[kk]), s[r],
                                                               0, 0, 0);
        }
        const int k0 = kbeg + step * kStepKeys;
        const bool ragged = k0 + kStepKeys > kend;  // wave-uniform: only a chunk's last step is ragged
        if (ragged) {
#pragma unroll
            for (int r = 0; r < 2; ++r)
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    if (k0 + 8 * q4 + 4 * r + i >= kend) s[r][i] = -INFINITY;
        }
        float mx = fmaxf(fmaxf(fmaxf(s[0][0], s[0][1]), fmaxf(s[0][2], s[0][3])),
                         fmaxf(fmaxf(s[1][0], s[1][1]), fmaxf(s[1][2], s[1][3])));
        mx = fmaxf(mx, __shfl_xor(mx, 16));
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        const float m_new = fmaxf(m_run, mx * scale_log2);   // finite: key k0 is visible
        const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
        m_run = m_new;
        bf16x8 pb;
        float ps = 0.f;
#pragma unroll
        for (int r = 0; r < 2; ++r)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(s[r][i], scale_log2, -m_new));
                pb[4 * r + i] = (__bf16)p;
                ps += (float)pb[4 * r + i];     // the rounded value the product weights V with
            }
        l_run = l_run * alpha + ps;
        if (__builtin_amdgcn_ballot_w64(alpha != 1.f)) {   // the max rose in some column
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) o[mt] *= alpha;
        }
        // In a ragged step the V^T operand entries of keys >= kend are cleared: their P is 0,
        // but the slots past a context's end may hold anything (never written, or another
        // request's data), and 0 * NaN or 0 * Inf would poison every output column. The
        // lane's 8 values are keys k0 + 8*q4 .. +7, the same keys as its P^T operand.
        const int nvalid = kend - (k0 + 8 * q4);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            u32x4 vv = R.v[mt];
            if (ragged) {
#pragma unroll
                for (int wd = 0; wd < 4; ++wd)
                    vv[wd] &= (2 * wd < nvalid ? 0x0000FFFFu : 0u) | (2 * wd + 1 < nvalid ? 0xFFFF0000u : 0u);
            }
            o[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(vv), pb, o[mt], 0, 0, 0);
        }
    };

    // Every load inside the loops is unconditional (a step index past the chunk's end
    // rereads its last step), so the wait before each step leaves the later steps'
    // loads in flight.
    const int n_steps = (kend - kbeg + kStepKeys - 1) / kStepKeys;
    if constexpr (NSETS == 3) {
        StepRegs<D> ra, rb, rc;
        load_step(0, ra);
        load_step(min(1, n_steps - 1), rb);
        int j = 0;
        for (; j + 4 < n_steps; j += 3) {
            load_step(j + 2, rc);
            process(j, ra);
            load_step(j + 3, ra);
            process(j + 1, rb);
            load_step(j + 4, rb);
            process(j + 2, rc);
        }
        const int left = n_steps - j;               // 1 .. 4; ra holds step j, rb step j + 1
        if (left == 1) {
            process(j, ra);
        } else if (left == 2) {
            process(j, ra);
            process(j + 1, rb);
        } else if (left == 3) {
            load_step(j + 2, rc);
            process(j, ra);
            process(j + 1, rb);
            process(j + 2, rc);
        } else {
            load_step(j + 2, rc);
            process(j, ra);
            load_step(j + 3, ra);
            process(j + 1, rb);
            process(j + 2, rc);
            process(j + 3, ra);
        }
    } else {
        StepRegs<D> ra, rb;
        load_step(0, ra);
        int j = 0;
        for (; j + 2 < n_steps; j += 2) {
            load_step(j + 1, rb);
            process(j, ra);
            load_step(j + 2, ra);
            process(j + 1, rb);
        }
        const int left = n_steps - j;               // 1 or 2; ra holds step j
        if (left == 2) {
            load_step(j + 1, rb);
            process(j, ra);
            process(j + 1, rb);
        } else {
            process(j, ra);
        }
    }
}

}  // namespace decode_wave
}  // namespace pcr
