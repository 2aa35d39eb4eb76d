// Flash-style non-causal softmax attention for gfx950 (MI355X), bf16 MFMA.
//
// Computes, per head h and query i (Sec. 3.3 Property of computational
// independence; the attention step of Alg. 1):
//   O[h][i] = sum_j softmax_j(scale * <Q[h][i], K[h][j]>) V[h][j],  j < S.
// The S x S score matrix is never stored: keys are visited in blocks of
// kBC = 64 with a running maximum and running sum per query (online softmax),
// so memory is O(S d) per head.
//
// Work decomposition
//   * one workgroup = WAVES waves (8 for d = 128, 4 for d = 64) = one tile of
//     32 * WAVES queries of one head; each wave owns 32 queries for the whole
//     key loop.  Two waves per SIMD.  With 8 waves the register file holds
//     exactly one workgroup per CU, so a workgroup dispatched while other
//     kernels occupy part of the GPU can never be queued behind two running
//     ones on the same CU, and every staged K/V block feeds 256 queries;
//   * K and V blocks are staged in LDS by all threads, K one block ahead of
//     V.  With d = 128 and bf16 storage (attention_dma_kernel) the blocks go
//     from global memory straight into LDS, three steps ahead of their use,
//     through four LDS buffers per tensor.  Otherwise they pass through
//     registers (global -> registers -> LDS) into double buffers; with bf16
//     storage two register sets alternate, so each block's global loads are
//     issued a whole step before its LDS stores;
//   * scores are computed transposed, S^T = K Q^T, with
//     v_mfma_f32_32x32x16_bf16: keys are the M dimension and queries the N
//     dimension.  In the accumulator layout each lane then holds one query
//     (column) and 16 keys (rows) per 32 x 32 tile, so the row max and row sum
//     of the softmax are in-lane reductions plus one swap between the two
//     32-lane halves of the wave (v_permlane32_swap, registers only);
//   * the same layout is exactly the B operand that O^T += V^T P^T needs, so P
//     never leaves registers.  V is stored transposed in LDS ([d][key]) with the
//     keys of every 16-key group permuted (bits 2 and 3 of the key index
//     swapped) to match the order in which the accumulator rows arrive;
//   * software pipeline: while the VALU computes the exponentials of block j,
//     the MFMA unit already computes the scores of block j + 1 (no dependency
//     between the two), then O^T += V_j^T P_j^T (attention_dma_kernel splits
//     each block's exponentials over both halves of a step).  K operands are read from
//     LDS four MFMAs ahead and V operands two (the first two before the
//     overflow test below); scheduling hints spread the exponentials between the score
//     MFMAs and the next blocks' LDS stores between the PV MFMAs.  The loop is
//     unrolled by two so the score registers alternate roles instead of being
//     copied;
//   * exp2 is the hardware v_exp_f32 on the argument s * c - m * c (one FMA),
//     c = scale * log2(e);
//   * lazy rescaling: the running maximum m is set by block 0 and raised only
//     when a block's exponentials, summed over its 64 keys, exceed 2^8; that
//     block is then recomputed against its own maximum and O and l are
//     rescaled.  So the common path computes no maximum at all, every
//     exponential used is at most 2^8 (bf16 and fp32 hold it exactly in
//     range), and the final O / l is unchanged;
//   * P is rounded to bf16 (nearest-even, v_cvt_pk_bf16_f32) for the PV MFMA.
//     attention_kernel's row sum l adds exactly these rounded values
//     (v_dot2c_f32_bf16 with a (1, 1) pair); attention_dma_kernel's adds the
//     fp32 weights before rounding (v_add_f32, which issues beside the
//     MFMAs).  All accumulation (scores, O, l) is fp32;
//   * the grid is remapped so that the 8 XCDs each take a contiguous range of
//     (head, query tile) pairs, so concurrent workgroups of an XCD stream the
//     same K/V blocks through that XCD's L2.
//
// Tails: loads go through buffer resources bounded by the head's tensor, so
// query and key rows >= S read as zeros; such queries are not stored and such
// keys get score -inf in the last block only.
#include <algorithm>

#include "attention_tiles.h"
#include "copy_tiles.h"
#include "hcms_internal.h"

#ifndef HCMS_ATTN_NT128
#define HCMS_ATTN_NT128 1
#endif

namespace hcms {
namespace {

using namespace tiles;

// S^T[nt][mt] = K[mt] Q[nt]^T for the 64 keys of a block (2 tiles of 32
// keys) and the wave's NT tiles of 32 queries; every K operand read from LDS
// feeds NT MFMAs, and the reads run four operands ahead of their use.
template <int D, int NT>
__device__ inline void qk_mfma(f32x16 (&sacc)[NT][2], const __bf16 *ks,
                               const bf16x8 (&qreg)[NT][D / 16], int li, int g) {
    constexpr int N = 2 * (D / 16);
    constexpr int AHEAD = 4;
    bf16x8 a[N];
#pragma unroll
    for (int i = 0; i < AHEAD; ++i)
        a[i] = *reinterpret_cast<const bf16x8 *>(ks + ((i & 1) * 32 + li) * Lds<D>::KS + ((i >> 1) * 2 + g) * 8);
#pragma unroll
    for (int i = 0; i < N; ++i) {
        if (i + AHEAD < N) {
            const int n = i + AHEAD;
            a[n] = *reinterpret_cast<const bf16x8 *>(ks + ((n & 1) * 32 + li) * Lds<D>::KS + ((n >> 1) * 2 + g) * 8);
        }
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
            sacc[nt][i & 1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                a[i], qreg[nt][i >> 1], i < 2 ? f32x16{} : sacc[nt][i & 1], 0, 0, 0);
    }
}

// O^T[dt][nt] += V^T[dt] P[nt]^T over the 64 keys of a block (4 k-steps of 16
// keys); every V operand read from LDS feeds NT MFMAs.  The first kPvAhead
// operands come in `pre` (read earlier by pv_prefetch), the others are read
// kPvAhead MFMAs ahead of their use.  Two, not more: the kernel stays within
// 248 VGPRs, so two waves per SIMD leave 16 registers per lane for the waves
// of a pack or unpack running beside them.
constexpr int kPvAhead = 2;

// Operand i = (ks, dt) = (i / DT, i % DT): consecutive MFMAs update different
// O^T tiles, so none waits for the result of the one before it; each tile
// still accumulates its four k-steps in order.
template <int D>
__device__ inline const bf16x8 &vt_operand(const __bf16 *vts, int i, int li, int g) {
    constexpr int DT = D / 32;
    return *reinterpret_cast<const bf16x8 *>(vts + ((i % DT) * 32 + li) * Lds<D>::VS + ((i / DT) * 2 + g) * 8);
}

template <int D>
__device__ inline void pv_prefetch(bf16x8 (&pre)[kPvAhead], const __bf16 *vts, int li, int g) {
#pragma unroll
    for (int i = 0; i < kPvAhead; ++i) pre[i] = vt_operand<D>(vts, i, li, g);
}

template <int D, int NT>
__device__ inline void pv_mfma(f32x16 (&oacc)[D / 32][NT], const bf16x8 (&pb)[NT][4],
                               const __bf16 *vts, const bf16x8 (&pre)[kPvAhead], int li, int g) {
    constexpr int N = 4 * (D / 32);
    bf16x8 a[N];
#pragma unroll
    for (int i = 0; i < kPvAhead; ++i) a[i] = pre[i];
#pragma unroll
    for (int i = 0; i < N; ++i) {
        if (i + kPvAhead < N) a[i + kPvAhead] = vt_operand<D>(vts, i + kPvAhead, li, g);
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
            oacc[i % (D / 32)][nt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                a[i], pb[nt][i / (D / 32)], oacc[i % (D / 32)][nt], 0, 0, 0);
    }
}

// Scheduling hints.  First half of a step: block j's exponentials (FMA,
// v_exp_f32, bf16 conversion and row sum) fill the LDS latency of the first K
// operand reads and then run between block j + 1's score MFMAs, about 6 VALU
// instructions per MFMA, so the VALU works while the MFMA unit is busy; the
// first V operands of the PV MFMAs are read before the overflow test.
template <int D, int NT>
__device__ inline void interleave_qk_exp() {
    constexpr int N = 2 * (D / 16);  // K operands per block
    constexpr int AHEAD = 4;         // K operand reads in flight (as in qk_mfma)
    __builtin_amdgcn_sched_group_barrier(0x100, AHEAD, 0);  // DS read
    __builtin_amdgcn_sched_group_barrier(0x002, 12, 0);     // VALU
#pragma unroll
    for (int i = 0; i < N; ++i) {
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
            __builtin_amdgcn_sched_group_barrier(0x002, 5, 0);  // VALU
        }
        if (i + AHEAD < N) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x100, kPvAhead, 0);  // V operand prefetch
}

// Second half: the PV MFMAs with their V operand reads, and between them the
// LDS stores of the next K and V blocks (and the V transpose's byte
// permutes), so those stores are done by the time the step's barrier comes.
template <int D, int NT>
__device__ inline void interleave_pv_stage() {
    constexpr int N = 4 * (D / 32);  // V operands per block
#pragma unroll
    for (int i = 0; i < N; ++i) {
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
        if (i + kPvAhead < N) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);            // DS read
        if (i >= 2) {
            __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);  // DS write
            __builtin_amdgcn_sched_group_barrier(0x002, 2, 0);  // VALU
        }
    }
}

// Both 32-lane halves of the wave hold the same 32 queries (different keys).
// v_permlane32_swap with both operands x returns (x of the lower half,
// x of the upper half) in every lane, so both halves combine the two values in
// the same order and get bit-identical results.
__device__ inline float halves_sum(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(unsigned, x),
                                                    __builtin_bit_cast(unsigned, x), false, false);
    return __builtin_bit_cast(float, static_cast<unsigned>(r[0])) +
           __builtin_bit_cast(float, static_cast<unsigned>(r[1]));
}

__device__ inline float halves_max(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(unsigned, x),
                                                    __builtin_bit_cast(unsigned, x), false, false);
    return fmaxf(__builtin_bit_cast(float, static_cast<unsigned>(r[0])),
                 __builtin_bit_cast(float, static_cast<unsigned>(r[1])));
}

// A block's exponentials are recomputed against its own maximum when their
// sum over the 64 keys exceeds this bound.
constexpr float kRaiseBound = 256.0f;

// Keys at or past `kvalid` inside the block get the score -inf.  Key
// mt * 32 + (r >> 2) * 8 + g * 4 + (r & 3) is compared as its constant part
// against kvalid - 4 g, so no per-lane key indices need registers.
__device__ inline void mask_block(f32x16 (&s)[2], int g, int kvalid) {
    const int kv = kvalid - g * 4;
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int key = mt * 32 + (r >> 2) * 8 + (r & 3);
            if (key >= kv) s[mt][r] = -INFINITY;
        }
}

// Block maximum of this lane's query over all 64 keys (both halves).
__device__ inline float block_max(const f32x16 (&s)[2]) {
    float mx = s[0][0];
#pragma unroll
    for (int r = 1; r < 16; ++r) mx = fmaxf(mx, s[0][r]);
#pragma unroll
    for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[1][r]);
    return halves_max(mx);
}

// P = exp2(c s - mc) rounded to bf16 as the B operands of the PV MFMAs
// (one FMA and one v_exp_f32 per score); returns this lane's sum of exactly
// those rounded values (v_dot2c_f32_bf16 with a (1, 1) pair), so the weights
// that multiply V are normalised exactly.
__device__ inline float exp_block(const f32x16 (&s)[2], float c, float mc, bf16x8 (&pb)[4]) {
    const bf16x2 ones = {static_cast<__bf16>(1.0f), static_cast<__bf16>(1.0f)};
    float sum = 0.f;
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            f32x8 p;
#pragma unroll
            for (int r = 0; r < 8; ++r)
                p[r] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[mt][h * 8 + r], c, -mc));
            const bf16x8 pbf = __builtin_convertvector(p, bf16x8);
            pb[mt * 2 + h] = pbf;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const bf16x2 pair = {pbf[2 * r], pbf[2 * r + 1]};
                sum = __builtin_amdgcn_fdot2_f32_bf16(pair, ones, sum, false);
            }
        }
    }
    return sum;
}

typedef float f32x2 __attribute__((ext_vector_type(2)));

#ifndef HCMS_ATTN_FP32_SUM
#define HCMS_ATTN_FP32_SUM 1
#endif
// The exponentials of one 32-key tile of a block (exp_block's pb[2 mt] and
// pb[2 mt + 1] for tile mt) in p0 and p1; returns sum plus this lane's sum of
// the tile's 16 weights.  That sum adds the fp32 weights before their
// rounding to bf16, in a fixed order with v_add_f32: unlike
// v_dot2c_f32_bf16, which does not issue while the matrix core is busy, an
// add issues beside the MFMAs.  l is then the sum of the unrounded weights
// while V is multiplied by their bf16 roundings, a relative difference below
// 2^-9 that averages out over the keys.
__device__ inline float exp_half(const f32x16 &s, float c, float mc, bf16x8 &p0, bf16x8 &p1,
                                 float sum) {
#if HCMS_ATTN_FP32_SUM
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        bf16x8 pbf;
#pragma unroll
        for (int r = 0; r < 8; r += 2) {
            const float a = __builtin_amdgcn_exp2f(__builtin_fmaf(s[h * 8 + r], c, -mc));
            const float b = __builtin_amdgcn_exp2f(__builtin_fmaf(s[h * 8 + r + 1], c, -mc));
            const bf16x2 ab = __builtin_convertvector((f32x2){a, b}, bf16x2);
            pbf[r] = ab[0];
            pbf[r + 1] = ab[1];
            sum += a + b;
        }
        (h == 0 ? p0 : p1) = pbf;
    }
    return sum;
#else
    const bf16x2 ones = {static_cast<__bf16>(1.0f), static_cast<__bf16>(1.0f)};
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        f32x8 p;
#pragma unroll
        for (int r = 0; r < 8; ++r) p[r] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[h * 8 + r], c, -mc));
        const bf16x8 pbf = __builtin_convertvector(p, bf16x8);
        (h == 0 ? p0 : p1) = pbf;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const bf16x2 pair = {pbf[2 * r], pbf[2 * r + 1]};
            sum = __builtin_amdgcn_fdot2_f32_bf16(pair, ones, sum, false);
        }
    }
    return sum;
#endif
}

template <int D, typename T, int WAVES, int NT, int PER_CU>
__global__ __launch_bounds__(64 * WAVES, PER_CU * WAVES / 4) void attention_kernel(
    const T *__restrict__ q, const T *__restrict__ k, const T *__restrict__ v, T *__restrict__ o,
    float *__restrict__ lse, int S, int n_qtiles, float c) {
    constexpr int KK = D / 16;  // MFMA k-steps over the head dimension
    constexpr int DT = D / 32;  // 32-row tiles of O^T
    __shared__ __attribute__((aligned(16))) __bf16 kbuf[2][Lds<D>::KT];
    __shared__ __attribute__((aligned(16))) __bf16 vbuf[2][Lds<D>::VT];

    // XCD-aware tile order: workgroup b runs on XCD b % 8; give each XCD a
    // contiguous range of (head, query tile) pairs.
    const int nb = gridDim.x, b = blockIdx.x;
    const int xcd = b & 7, per = nb >> 3, rem = nb & 7;
    const int logical = xcd * per + min(xcd, rem) + (b >> 3);
    const int head = logical / n_qtiles;
    const int qtile = logical - head * n_qtiles;

    const int64_t hoff = static_cast<int64_t>(head) * S * D;
    const int64_t hbytes = static_cast<int64_t>(S) * D * sizeof(T);
    const __amdgpu_buffer_rsrc_t qr = head_rsrc(q + hoff, hbytes);
    const __amdgpu_buffer_rsrc_t kr = head_rsrc(k + hoff, hbytes);
    const __amdgpu_buffer_rsrc_t vr = head_rsrc(v + hoff, hbytes);
    T *oh = o + hoff;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int li = lane & 31;   // row / column index inside a 32-wide MFMA tile
    const int g = lane >> 5;    // which half of the wave
    // The wave's queries: tile nt holds q0 + 32 nt + [0, 32); this lane holds
    // query q0 + 32 nt + li of each tile.
    const int q0 = (qtile * WAVES + wave) * (kQW * NT);

    // Q^T as the B operand: lane (g, n) holds query n, head dims 16 kk + 8 g + [0, 8).
    // Rows past S read as zeros and are never stored.
    bf16x8 qreg[NT][KK];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int kk = 0; kk < KK; ++kk)
            qreg[nt][kk] = __builtin_bit_cast(
                bf16x8, load8<T>(qr, static_cast<unsigned>((q0 + nt * kQW + li) * D + kk * 16 + g * 8) *
                                         sizeof(T)));

    f32x16 oacc[DT][NT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) oacc[dt][nt] = f32x16{};
    const int nkb = (S + kBC - 1) / kBC;

    // Prologue: K_0, V_0 and K_1 in LDS, scores of block 0.
    // NSETS register sets carry the next blocks from global memory to LDS.
    // With two (bf16 storage), the loads for the blocks stored in step j are
    // issued in step j - 1, a whole step ahead of their use; with one (fp32
    // storage, whose loads need twice the registers), in step j itself.
    constexpr int NSETS = sizeof(T) == 2 ? 2 : 1;
    Stage<D, T, WAVES> st[NSETS];
    st[0].load(kr, vr, 0, 0, tid);
    st[0].store_k(kbuf[0], tid);
    st[0].store_v(vbuf[0], tid);
    st[1 % NSETS].load(kr, vr, 1, 1, tid);
    st[1 % NSETS].store_k(kbuf[1], tid);
    if (NSETS == 2) st[0].load(kr, vr, 2, 1, tid);
    __syncthreads();
    f32x16 sa[NT][2], sb[NT][2];
    qk_mfma<D, NT>(sa, kbuf[0], qreg, li, g);
    __syncthreads();  // kbuf[0] is overwritten below

    // Block 0 sets the running maximum m used by the exponentials
    // exp2(c s - c m).  m is raised lazily: only when a block's exponentials,
    // summed over its 64 keys, exceed 2^8 is the block recomputed against its
    // own maximum (and O, l rescaled).  Every exponential used is therefore at
    // most 2^8, and the common path needs no maximum at all.  The decision is
    // per query (both halves of the wave combine their sums in the same
    // order); a wave only takes the recompute branch when some query needs it,
    // and a query that does not need it recomputes the same values and
    // multiplies by exactly 1 there.  So the arithmetic of every query depends
    // only on its own row, never on which other queries share the wave, tile,
    // chunk or launch: any head chunking gives bit-identical results.
    float m[NT], mc[NT], lsum[NT];
    bf16x8 pb[NT][4];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
        if (nkb == 1) mask_block(sa[nt], g, S);
        m[nt] = block_max(sa[nt]);
        mc[nt] = m[nt] * c;
        lsum[nt] = exp_block(sa[nt], c, mc[nt], pb[nt]);
    }

    // Recompute branch of a block whose exponentials overflowed the bound.
    auto raise_m = [&](const f32x16(&s)[NT][2], const bool (&up)[NT], float (&bsum)[NT]) {
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
            const float mx = block_max(s[nt]);
            const float m_new = up[nt] ? mx : m[nt];
            const float alpha = up[nt] ? __builtin_amdgcn_exp2f((m[nt] - mx) * c) : 1.0f;
            m[nt] = m_new;
            mc[nt] = m_new * c;
            bsum[nt] = exp_block(s[nt], c, mc[nt], pb[nt]);
            lsum[nt] *= alpha;
#pragma unroll
            for (int dt = 0; dt < DT; ++dt)
#pragma unroll
                for (int r = 0; r < 16; ++r) oacc[dt][nt][r] *= alpha;
        }
    };
    // Exponentials of one block, the per-query overflow test and, when some
    // query needs it, the recompute branch.
    bf16x8 vpre[kPvAhead];
    auto softmax = [&](const f32x16(&s)[NT][2], const __bf16 *vts) {
        float bsum[NT];
        bool up[NT], any_up = false;
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) bsum[nt] = exp_block(s[nt], c, mc[nt], pb[nt]);
        pv_prefetch<D>(vpre, vts, li, g);
        interleave_qk_exp<D, NT>();
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
            up[nt] = halves_sum(bsum[nt]) > kRaiseBound;
            any_up = any_up || up[nt];
        }
        if (__any(any_up)) raise_m(s, up, bsum);
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) lsum[nt] += bsum[nt];
    };

    if (nkb > 1) {
        // Block 0's PV and block 1's scores.
        st[1 % NSETS].load(kr, vr, 1 + NSETS, NSETS, tid);
        qk_mfma<D, NT>(sb, kbuf[1], qreg, li, g);
        pv_prefetch<D>(vpre, vbuf[0], li, g);
        pv_mfma<D, NT>(oacc, pb, vbuf[0], vpre, li, g);
        st[0].store_k(kbuf[0], tid);
        st[0].store_v(vbuf[1], tid);
        __syncthreads();
    }

    // Steady state: block j's exponentials and PV overlap block j + 1's
    // scores.  LDS holds K_{j+1} in kbuf[(j+1)&1] and V_j in vbuf[j&1]; K_{j+2}
    // and V_{j+1} land from registers in the buffers freed by K_j and V_{j-1}.
    // Step j loads K_{j+1+NSETS} and V_{j+NSETS} into set (j + 1) % NSETS and
    // stores from set j % NSETS.
    auto step = [&](int j, f32x16(&scur)[NT][2], f32x16(&snext)[NT][2], Stage<D, T, WAVES> &ld,
                    Stage<D, T, WAVES> &sto) {
        ld.load(kr, vr, j + 1 + NSETS, j + NSETS, tid);
        qk_mfma<D, NT>(snext, kbuf[(j + 1) & 1], qreg, li, g);
        softmax(scur, vbuf[j & 1]);
        pv_mfma<D, NT>(oacc, pb, vbuf[j & 1], vpre, li, g);
        sto.store_k(kbuf[j & 1], tid);
        sto.store_v(vbuf[(j + 1) & 1], tid);
        interleave_pv_stage<D, NT>();
        __syncthreads();
    };
    int j = 1;
    if (nkb > 1) {
        for (; j + 2 < nkb; j += 2) {
            step(j, sb, sa, st[0], st[1 % NSETS]);
            step(j + 1, sa, sb, st[1 % NSETS], st[0]);
        }
        if (j + 1 < nkb) {
            step(j, sb, sa, st[0], st[1 % NSETS]);
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) {
                sb[nt][0] = sa[nt][0];
                sb[nt][1] = sa[nt][1];
            }
            ++j;
        }
        // Last block (j = nkb - 1): mask the keys past S.
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) mask_block(sb[nt], g, S - j * kBC);
        softmax(sb, vbuf[j & 1]);
        pv_mfma<D, NT>(oacc, pb, vbuf[j & 1], vpre, li, g);
    } else {
        pv_prefetch<D>(vpre, vbuf[0], li, g);
        pv_mfma<D, NT>(oacc, pb, vbuf[0], vpre, li, g);
    }

    // ---- O = O^T / l, rounded to the storage type ----
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
        const int qi = q0 + nt * kQW + li;
        const float l = halves_sum(lsum[nt]);
        const float inv = 1.0f / l;
        // log2 of the softmax denominator of c * s: P_ij = exp2(c s_ij - L2_i)
        // (the statistic the backward pass recomputes P from).
        if (lse != nullptr && g == 0 && qi < S)
            lse[static_cast<int64_t>(head) * S + qi] = mc[nt] + __builtin_amdgcn_logf(l);
        if (qi < S) {
            T *orow = oh + static_cast<int64_t>(qi) * D;
#pragma unroll
            for (int dt = 0; dt < DT; ++dt)
#pragma unroll
                for (int rb = 0; rb < 4; ++rb) {
                    const f32x4 x = {oacc[dt][nt][rb * 4 + 0] * inv, oacc[dt][nt][rb * 4 + 1] * inv,
                                     oacc[dt][nt][rb * 4 + 2] * inv, oacc[dt][nt][rb * 4 + 3] * inv};
                    store4(orow + dt * 32 + rb * 8 + g * 4, x);
                }
        }
    }
}

// ---------------------------------------------------------------------------
// d = 128 with bf16 storage: K and V blocks go from global memory straight
// into LDS (buffer_load_dwordx4 ... lds), several blocks ahead of their use,
// without passing through registers.
//
// LDS holds kNB buffers of K blocks and kNB of V blocks, each 64 keys x 256
// bytes row-major.  One DMA instruction of a wave writes 1 KiB of LDS
// contiguously (lane l at byte 16 l), i.e. four key rows; every lane chooses
// which 16-byte chunk of its row it fetches, so the chunks are stored
// XOR-swizzled:
//   K: chunk c of row r at position c ^ (r & 15), so the 16-byte score operand
//      reads of 16 consecutive rows hit 16 different groups of 4 banks;
//   V: chunk c of row r at position c ^ 4 (r & 3), so the transposing reads
//      below (4 rows x 64 bytes per 32 lanes) hit 16 different groups.
// The V^T operand of O^T += V^T P^T (lane (li, g) needs V[key][32 dt + li] for
// the keys 4g + {0..3} and 8 + 4g + {0..3} of a 16-key group, the order in
// which the score accumulator rows arrive) comes from two ds_read_b64_tr_b16.
// Within each group of 16 lanes that instruction hands lane t element t mod 4
// of the 8 bytes read by lanes 4r + t / 4, r = 0..3.  So lane 4r + q of the
// group reads row key_base + r at columns d_base + 4q .. 4q + 3, and lane t
// receives column d_base + t of the four rows.
// The compiler does not see these loads (inline asm; with the intrinsic it
// would wait for all of them before every LDS read).  The key loop issues no
// other vector memory instruction, and the kernel waits for its loads itself
// (s_waitcnt vmcnt) before each step's barrier.  The operand values and the
// MFMA order are those of attention_kernel; the row sum differs (exp_half).
namespace dma {

constexpr int kD = 128;
constexpr int kWaves = 8;
constexpr int kRowB = kD * 2;                          // bytes per key row
constexpr int kTileB = kBC * kRowB;                    // one 64-key block: 16 KiB
constexpr int kNB = 3;                                 // LDS buffers per tensor
constexpr int kPerWave = kTileB / (64 * 16) / kWaves;  // DMA instructions per wave and block
// Steps between a block's load and the step that reads it.
constexpr int kDist = 2;
static_assert(kDist >= 1 && kDist + 1 <= kNB, "more blocks in flight than LDS buffers");
static_assert(kPerWave == 2, "the wait counts below assume two DMA instructions per block");

// Key segments.  Every query visits its keys as kSeg fixed segments of whole
// blocks (one segment when the sequence has fewer than kSegMinBlocks blocks),
// each an online softmax of its own, and the segments' states are merged in a
// fixed order (merge_states).  The boundaries depend only on S, so the
// arithmetic of a query never depends on which workgroups computed which
// segments: a tile may be computed whole by one workgroup or split over
// several, with bit-identical results.
constexpr int kSeg = 3;
constexpr int kSegMinBlocks = 12;
__host__ __device__ inline int n_segments(int nkb) { return nkb >= kSegMinBlocks ? kSeg : 1; }
// First block of segment g (g = n_segments: one past the last block).
__host__ __device__ inline int seg_begin(int nkb, int g) {
    const int n = n_segments(nkb);
    return g <= 0 ? 0 : g >= n ? nkb : (g * nkb + n / 2) / n;
}
// A segment's unnormalised output, rounded to bf16, kept in LDS between
// segments: 64 values per lane, chunk k (values 8k .. 8k + 7) of lane l of
// wave w at byte w * 8 KiB + k * 1 KiB + 16 l.  Partial states of split tiles
// use the same layout in global memory.
constexpr int kStashWaveB = 64 * 64 * 2;
constexpr int kStashB = kWaves * kStashWaveB;           // 64 KiB
constexpr int kLdsB = 2 * kNB * kTileB + kStashB;       // 160 KiB, all of a CU's LDS

// Score operands: S^T[i & 1] += K rows 32 (i & 1) + li, chunk 2 (i >> 1) + g,
// times Q^T; `k_rd[i >> 1]` is the lane's byte offset of its row and chunk.
#ifndef HCMS_ATTN_KAHEAD
#define HCMS_ATTN_KAHEAD 4
#endif
#ifndef HCMS_ATTN_VAHEAD
#define HCMS_ATTN_VAHEAD 2
#endif
constexpr int kKAhead = HCMS_ATTN_KAHEAD;  // score operand reads in flight
constexpr int kVAhead = HCMS_ATTN_VAHEAD;  // V^T operands read ahead of their MFMA

__device__ inline void qk(f32x16 (&sacc)[2], const char *kb, const unsigned (&k_rd)[kD / 16],
                          const bf16x8 (&qreg)[kD / 16]) {
    constexpr int N = 2 * (kD / 16);
    constexpr int AHEAD = kKAhead;
    auto rd = [&](int n) {
        return *reinterpret_cast<const bf16x8 *>(kb + k_rd[n >> 1] + (n & 1) * 32 * kRowB);
    };
    bf16x8 a[N];
#pragma unroll
    for (int i = 0; i < AHEAD; ++i) a[i] = rd(i);
#pragma unroll
    for (int i = 0; i < N; ++i) {
        if (i + AHEAD < N) a[i + AHEAD] = rd(i + AHEAD);
        sacc[i & 1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], qreg[i >> 1],
                                                              i < 2 ? f32x16{} : sacc[i & 1], 0, 0, 0);
    }
}

// V^T operand i = (ks, dt) = (i / 4, i % 4): keys 16 ks + 4g + {0..3} and
// 16 ks + 8 + 4g + {0..3} of column 32 dt + li.
__device__ inline bf16x8 vt(const char *vb, const unsigned (&v_rd)[kD / 32], int i) {
    typedef __attribute__((address_space(3))) bf16x4 LdsV4;
    const char *p = vb + v_rd[i % (kD / 32)] + (i / (kD / 32)) * 16 * kRowB;
    const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((LdsV4 *)(p));
    const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((LdsV4 *)(p + 8 * kRowB));
    return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
}

__device__ inline void pv_prefetch(bf16x8 (&pre)[kVAhead], const char *vb, const unsigned (&v_rd)[kD / 32]) {
#pragma unroll
    for (int i = 0; i < kVAhead; ++i) pre[i] = vt(vb, v_rd, i);
}

// O^T[i % 4] += V^T operand i times P^T[i / 4], in the order of pv_mfma; P^T
// comes as its keys 0-31 (lo) and 32-63 (hi).
__device__ inline void pv(f32x16 (&oacc)[kD / 32], const bf16x8 (&lo)[2], const bf16x8 (&hi)[2],
                          const char *vb, const unsigned (&v_rd)[kD / 32], const bf16x8 (&pre)[kVAhead]) {
    constexpr int DT = kD / 32, N = 4 * DT;
    bf16x8 a[N];
#pragma unroll
    for (int i = 0; i < kVAhead; ++i) a[i] = pre[i];
#pragma unroll
    for (int i = 0; i < N; ++i) {
        if (i + kVAhead < N) a[i + kVAhead] = vt(vb, v_rd, i + kVAhead);
        const int ks = i / DT;
        oacc[i % DT] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], ks < 2 ? lo[ks] : hi[ks - 2],
                                                               oacc[i % DT], 0, 0, 0);
    }
}

// Scheduling hints.  Each phase of a step holds half of the softmax VALU work
// (the exponentials of 32 keys: FMA, v_exp_f32, conversion, row sum), about
// three VALU instructions per MFMA.  The hints pin two of them after each
// score MFMA and each PV MFMA and leave the rest to the scheduler, which
// measured faster than pinning all three.  A V operand takes two LDS reads.
#ifndef HCMS_ATTN_QK_VALU
#define HCMS_ATTN_QK_VALU 2
#endif
#ifndef HCMS_ATTN_PV_VALU
#define HCMS_ATTN_PV_VALU 2
#endif
#ifndef HCMS_ATTN_QK_VALU0
#define HCMS_ATTN_QK_VALU0 4
#endif
constexpr int kQkValu = HCMS_ATTN_QK_VALU;   // VALU instructions after each score MFMA
constexpr int kPvValu = HCMS_ATTN_PV_VALU;   // VALU instructions after each PV MFMA
__device__ inline void interleave_qk() {
    constexpr int N = 2 * (kD / 16), AHEAD = kKAhead;
    __builtin_amdgcn_sched_group_barrier(0x100, AHEAD, 0);  // DS read
    __builtin_amdgcn_sched_group_barrier(0x002, HCMS_ATTN_QK_VALU0, 0);  // VALU
#pragma unroll
    for (int i = 0; i < N; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
        __builtin_amdgcn_sched_group_barrier(0x002, kQkValu, 0);  // VALU
        if (i + AHEAD < N) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x100, 2 * kVAhead, 0);  // V operand prefetch
}

__device__ inline void interleave_pv() {
    constexpr int N = 4 * (kD / 32);
#pragma unroll
    for (int i = 0; i < N; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                        // MFMA
        if (i + kVAhead < N) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);   // DS read
        __builtin_amdgcn_sched_group_barrier(0x002, kPvValu, 0);                  // VALU
    }
}

template <int P>
struct Phase {
    static constexpr int value = P;
};

}  // namespace dma

// Copies that ride in an attention launch.  A launch of W attention
// workgroups on n_cu CUs, one workgroup per CU, ends in a round that leaves
// n_cu * ceil(W / n_cu) - W CUs idle.  The fused schedule appends that many
// workgroups after the attention workgroups; the dispatcher hands them out
// once every attention workgroup has a CU, so they fill the idle CUs of the
// last round, and they move a neighbouring chunk's head rows (the next
// chunk's pack, the previous chunk's unpack) meanwhile.  Rider workgroup r of
// R takes copy blocks 2 r + half, 2 r + half + 2 R, ... over the jobs in
// order, each half of its 512 threads one copy block at a time.
struct RiderJob {
    copy::PackPtrs p;
    int64_t h0;
    unsigned hc, n_tensors, blocks;  // blocks = copy::blocks_x * hc * n_tensors
    int unpack;
};

struct Riders {
    RiderJob job[2];
    int64_t S, H;
    unsigned n_jobs, bx;  // bx = copy::blocks_x(S, 4)
};

// Rows of d = 128 bf16 elements: 256 bytes = 16 units of 16 bytes.
constexpr int kRiderLog2U = 4;
static_assert((dma::kD * 2) >> 4 == 1 << kRiderLog2U, "rider rows are the attention rows");

__device__ inline void run_riders(const Riders &r, unsigned rider, unsigned n_riders) {
    const unsigned half = threadIdx.x >> 8, t = threadIdx.x & 255;
    const unsigned total = r.job[0].blocks + (r.n_jobs > 1 ? r.job[1].blocks : 0u);
    for (unsigned v = 2 * rider + half; v < total; v += 2 * n_riders) {
        const bool second = v >= r.job[0].blocks;
        const RiderJob &jb = second ? r.job[1] : r.job[0];
        const unsigned w = second ? v - r.job[0].blocks : v;
        const unsigned x = w % r.bx, rest = w / r.bx;
        const unsigned j = rest % jb.hc, z = rest / jb.hc;
        if (jb.unpack)
            copy::copy_block<kRiderLog2U, true>(jb.p, r.S, r.H, jb.h0, x, j, z, t);
        else
            copy::copy_block<kRiderLog2U, false>(jb.p, r.S, r.H, jb.h0, x, j, z, t);
    }
}

// Tiles split over several workgroups (the launch's last, partial round of
// tiles; see plan_split).  Workgroup n_whole + u computes segments of tile
// n_whole + u % n_split: with 3 ways segment u / n_split, with 2 ways
// segments 0-1 (u < n_split) or 2.  Each writes its partial state to slot
// u (the normalised output in the stash layout, and (m, l, E) per query)
// and counts itself in on its tile's counter; the last to arrive merges the
// tile's partial states in segment order, writes the output and sets the
// counter back to zero.
struct TailSplit {
    char *part;      // n_split * ways slots of kStashB bytes
    float4 *ml;      // n_split * ways slots of 256 (m, l, E, 0) per query
    int *count;      // n_split counters, zero between launches
    int n_whole;     // tiles computed whole by one workgroup: the first n_whole
    int n_split;     // tiles split: the last n_split
    int ways;        // 2 or 3
};

// The state of a query after some of its key segments: the maximum m of its
// raw scores, the row sum l of exp2(c (s - m)), and the normalised output N
// (this lane's 64 values of it).  Between segments a state is kept in 16 bits
// per value: N scaled by 2^-E, E the binary exponent of the query's largest
// |N| (over both halves of the wave), rounded to fp16 (nearest-even), so a
// stored value keeps 11 significant bits relative to the query's largest.
// quantise applies exactly that rounding in registers; store_state and
// load_state move the rounded values through LDS or global memory unchanged.
__device__ inline int state_exponent(const f32x16 (&n)[4]) {
    float a = 0.f;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
        for (int r = 0; r < 16; ++r) a = fmaxf(a, fabsf(n[dt][r]));
    return __builtin_amdgcn_frexp_expf(halves_max(a));   // max = f 2^E, f in [0.5, 1)
}
__device__ inline void quantise(f32x16 (&n)[4], int E) {
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
        for (int r = 0; r < 16; ++r)
            n[dt][r] = __builtin_ldexpf(static_cast<float>(static_cast<_Float16>(__builtin_ldexpf(n[dt][r], -E))), E);
}
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
// Chunk k (values 8k .. 8k + 7) of lane l at base + k * 1 KiB + 16 l.  The
// pointers come from the stash or the split scratch; the compiler infers LDS
// or global after inlining.
__device__ inline void store_state(char *base, const f32x16 (&n)[4], int E, int lane) {
#pragma unroll
    for (int k = 0; k < 8; ++k) {
        f16x8 h;
#pragma unroll
        for (int i = 0; i < 8; ++i)
            h[i] = static_cast<_Float16>(__builtin_ldexpf(n[k >> 1][(k & 1) * 8 + i], -E));
        *reinterpret_cast<f16x8 *>(base + k * 1024 + 16 * lane) = h;
    }
}
__device__ inline void load_state(f32x16 (&n)[4], const char *base, int E, int lane) {
#pragma unroll
    for (int k = 0; k < 8; ++k) {
        const f16x8 h = *reinterpret_cast<const f16x8 *>(base + k * 1024 + 16 * lane);
#pragma unroll
        for (int i = 0; i < 8; ++i) n[k >> 1][(k & 1) * 8 + i] = __builtin_ldexpf(static_cast<float>(h[i]), E);
    }
}

// The state of one segment from its online softmax: N = O / l, in place.
__device__ inline void segment_state(f32x16 (&o)[4], float l) {
    const float inv = 1.0f / l;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[dt][r] *= inv;
}

// Canonical merge of two states of one query (A of the earlier segments, B
// of the later): the merged maximum and row sum, and the weights of A's and
// B's normalised outputs, N = fma(N_A, wa, N_B * wb) element by element.
__device__ inline void merge_weights(float mA, float lA, float mB, float lB, float c, float &m,
                                     float &l, float &wa, float &wb) {
    m = fmaxf(mA, mB);
    const float a = __builtin_amdgcn_exp2f((mA - m) * c) * lA;
    const float b = __builtin_amdgcn_exp2f((mB - m) * c) * lB;
    l = a + b;
    const float inv = 1.0f / l;
    wa = a * inv;
    wb = b * inv;
}
// Merges a stored state (chunk k of lane l at base + k * 1 KiB + 16 l, scale
// 2^E) into this lane's 64 values n, chunk by chunk: stored_is_a says whether
// the stored state is A (the earlier segments) or B.
__device__ inline void merge_stored(f32x16 (&n)[4], const char *base, int E, int lane, float wa,
                                    float wb, bool stored_is_a) {
#pragma unroll
    for (int k = 0; k < 8; ++k) {
        const f16x8 h = *reinterpret_cast<const f16x8 *>(base + k * 1024 + 16 * lane);
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const float x = __builtin_ldexpf(static_cast<float>(h[i]), E);
            const float y = n[k >> 1][(k & 1) * 8 + i];
            n[k >> 1][(k & 1) * 8 + i] = stored_is_a ? __builtin_fmaf(x, wa, y * wb) : __builtin_fmaf(y, wa, x * wb);
        }
    }
}

template <bool kRiders>
__global__ __launch_bounds__(64 * dma::kWaves, dma::kWaves / 4) void attention_dma_kernel(
    const __bf16 *__restrict__ q, const __bf16 *__restrict__ k, const __bf16 *__restrict__ v,
    __bf16 *__restrict__ o, float *__restrict__ lse, int S, int n_qtiles, float c, TailSplit tail,
    Riders riders) {
    using namespace dma;
    const int n_attn = tail.n_whole + tail.n_split * tail.ways;
    if constexpr (kRiders) {
        if (blockIdx.x >= static_cast<unsigned>(n_attn)) {
            run_riders(riders, blockIdx.x - n_attn, gridDim.x - n_attn);
            return;
        }
    }
    constexpr int D = kD, KK = D / 16, DT = D / 32;
    __shared__ __attribute__((aligned(1024))) char lds[kLdsB];
    const char *const kbase = lds;                  // K buffer b at kbase + b * kTileB
    const char *const vbase = lds + kNB * kTileB;   // V buffer b at vbase + b * kTileB
    char *const stash = lds + 2 * kNB * kTileB;

    // Which tile, and which of its segments.  Whole tiles: XCD-aware order,
    // workgroup b runs on XCD b % 8 and each XCD takes a contiguous range of
    // (head, query tile) pairs, so concurrent workgroups of an XCD stream the
    // same K/V blocks through its L2.
    const int b = blockIdx.x;
    int logical, split_u = -1;
    if (b < tail.n_whole) {
        const int nb = tail.n_whole;
        const int xcd = b & 7, per = nb >> 3, rem = nb & 7;
        logical = xcd * per + min(xcd, rem) + (b >> 3);
    } else {
        split_u = b - tail.n_whole;
        logical = tail.n_whole + split_u % tail.n_split;
    }
    const int head = logical / n_qtiles;
    const int qtile = logical - head * n_qtiles;
    const int nkb = (S + kBC - 1) / kBC;
    const int nseg = n_segments(nkb);
    int g_first = 0, g_last = nseg;
    if (split_u >= 0) {
        const int p = split_u / tail.n_split;
        g_first = tail.ways == 3 ? p : 2 * p;
        g_last = tail.ways == 3 ? p + 1 : (p == 0 ? 2 : 3);
    }

    const int64_t hoff = static_cast<int64_t>(head) * S * D;
    const int64_t hbytes = static_cast<int64_t>(S) * D * 2;
    const __amdgpu_buffer_rsrc_t qr = head_rsrc(q + hoff, hbytes);
    const __amdgpu_buffer_rsrc_t kr = head_rsrc(k + hoff, hbytes);
    const __amdgpu_buffer_rsrc_t vr = head_rsrc(v + hoff, hbytes);
    __bf16 *oh = o + hoff;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int li = lane & 31;
    const int g = lane >> 5;
    const int q0 = (qtile * kWaves + wave) * kQW;

    bf16x8 qreg[KK];
#pragma unroll
    for (int kk = 0; kk < KK; ++kk)
        qreg[kk] = __builtin_bit_cast(
            bf16x8, load8<__bf16>(qr, static_cast<unsigned>((q0 + li) * D + kk * 16 + g * 8) * 2));

    // Lane offsets: DMA sources (row r = 4 (2 wave + i) + lane / 16 of the
    // block, chunk at position lane % 16), score operand reads and transposing
    // V reads (lane t = lane % 16 of group G = lane / 16).
    unsigned k_src[kPerWave], v_src[kPerWave];
#pragma unroll
    for (int i = 0; i < kPerWave; ++i) {
        const unsigned r = 4 * (kPerWave * wave + i) + (lane >> 4), p = lane & 15;
        k_src[i] = r * kRowB + ((p ^ (r & 15)) << 4);
        v_src[i] = r * kRowB + ((p ^ ((r & 3) << 2)) << 4);
    }
    unsigned k_rd[KK];
#pragma unroll
    for (int qq = 0; qq < KK; ++qq) k_rd[qq] = li * kRowB + (((2 * qq + g) ^ (li & 15)) << 4);
    unsigned v_rd[DT];
    {
        const unsigned G = lane >> 4, t = lane & 15;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
            v_rd[dt] = (4 * (G >> 1) + (t >> 2)) * kRowB +
                       ((((dt ^ (t >> 2)) << 2) + 2 * (G & 1) + ((t >> 1) & 1)) << 4) + ((t & 1) << 3);
    }
    // Opaque to the compiler: with the offsets' known bits it turns base +
    // constant into an OR, which the transposing read's immediate offset does
    // not take.
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) asm volatile("" : "+v"(v_rd[dt]));
    const unsigned lds0 = static_cast<unsigned>(reinterpret_cast<uintptr_t>(lds));
    const unsigned wave_dst = lds0 + kPerWave * wave * 1024;

    f32x16 oacc[DT];
    float m = 0.f, mc = 0.f, lsum = 0.f;

    // One segment: blocks blk0 .. blk0 + nb - 1 of the keys, an online softmax
    // starting afresh (its first block sets the running maximum).  Leaves the
    // segment's unnormalised output in oacc, its maximum in m and this lane's
    // share of its row sum in lsum.  Block j of the segment (relative index)
    // sits in LDS buffer j % kNB.
    auto segment = [&](const int blk0, const int nb) {
        auto issue_k = [&](int j) {
            const unsigned dst = wave_dst + (j % kNB) * kTileB;
#pragma unroll
            for (int i = 0; i < kPerWave; ++i) load_lds(dst + i * 1024, kr, k_src[i], (blk0 + j) * kTileB);
        };
        auto issue_v = [&](int j) {
            const unsigned dst = wave_dst + (kNB + j % kNB) * kTileB;
#pragma unroll
            for (int i = 0; i < kPerWave; ++i) load_lds(dst + i * 1024, vr, v_src[i], (blk0 + j) * kTileB);
        };
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) oacc[dt] = f32x16{};
        // Prologue: K_0, V_0, ..., K_{kDist-1}, V_{kDist-1}, K_kDist in
        // flight; step j then issues K_{j+1+kDist} and V_{j+kDist} (blocks
        // past the segment are loaded but never used; past S they read as
        // zeros).
#pragma unroll
        for (int j = 0; j <= kDist; ++j) {
            issue_k(j);
            if (j < kDist) issue_v(j);
        }
        wait_vm<4 * kDist>();  // K_0 landed
        __syncthreads();
        f32x16 sa[2], sb[2];
        qk(sa, kbase, k_rd, qreg);
        wait_vm<4 * kDist - 4>();  // V_0 and K_1 landed
        __syncthreads();           // and every wave is done with K_0's buffer

        // The first block sets the running maximum; the lazy rescaling is that
        // of attention_kernel.  The exponentials of block j are split over two
        // steps: keys 0-31 (tile 0) during the PV of block j - 1, keys 32-63
        // (tile 1) during the scores of block j + 1, followed by the overflow
        // test of block j.  So both phases of a step carry half of the VALU
        // work next to their 16 MFMAs.  lo[j & 1] holds tile 0 of block j's P,
        // hi tile 1; s0 the row sum over tile 0 (continued by tile 1 in
        // exp_block's order).
        float s0 = 0.f;
        bf16x8 lo[2][2], hi[2];
        if (nb == 1) mask_block(sa, g, S - blk0 * kBC);
        m = block_max(sa);
        mc = m * c;
        lsum = exp_half(sa[1], c, mc, hi[0], hi[1], exp_half(sa[0], c, mc, lo[0][0], lo[0][1], 0.f));

        bf16x8 vpre[kVAhead];
        // Tile 1 of block j (scores s, tile 0 already in lo_j with sum s0),
        // the overflow test and, when some query needs it, the recompute
        // branch.
        auto finish = [&](const f32x16(&s)[2], bf16x8(&lo_j)[2], const char *vb) {
            float bsum = exp_half(s[1], c, mc, hi[0], hi[1], s0);
            pv_prefetch(vpre, vb, v_rd);
            interleave_qk();
            const bool up = halves_sum(bsum) > kRaiseBound;
            if (__any(up)) {
                const float mx = block_max(s);
                const float m_new = up ? mx : m;
                const float alpha = up ? __builtin_amdgcn_exp2f((m - mx) * c) : 1.0f;
                m = m_new;
                mc = m_new * c;
                bsum = exp_half(s[1], c, mc, hi[0], hi[1], exp_half(s[0], c, mc, lo_j[0], lo_j[1], 0.f));
                lsum *= alpha;
#pragma unroll
                for (int dt = 0; dt < DT; ++dt)
#pragma unroll
                    for (int r = 0; r < 16; ++r) oacc[dt][r] *= alpha;
            }
            lsum += bsum;
        };
        // PV of block j beside tile 0 of block j + 1 (scores sn, already
        // masked when block j + 1 is the last one of the keys).
        auto pv_next = [&](const bf16x8(&lo_j)[2], const char *vb, f32x16(&sn)[2], bf16x8(&lo_n)[2]) {
            pv(oacc, lo_j, hi, vb, v_rd, vpre);
            s0 = exp_half(sn[0], c, mc, lo_n[0], lo_n[1], 0.f);
            interleave_pv();
        };

        // Step j: K_{j+1} is in buffer (j + 1) % kNB, V_j in buffer j % kNB.
        // The step of the segment's last scores masks them (a no-op unless
        // that block is the last of the keys); the other steps carry no
        // masking code.
        auto step = [&](int j, auto ph, auto first, auto last, f32x16(&scur)[2], f32x16(&snext)[2],
                        bf16x8(&lo_j)[2], bf16x8(&lo_n)[2]) {
            // P: j % 6 (buffers j % kNB and the score registers' alternation
            // j % 2), or -1 when only known at run time.
            constexpr int P = decltype(ph)::value;
            const int kb = P >= 0 ? (P + 1) % kNB : (j + 1) % kNB;
            const int vb = P >= 0 ? P % kNB : j % kNB;
            issue_k(j + 1 + kDist);
            issue_v(j + kDist);
            qk(snext, kbase + kb * kTileB, k_rd, qreg);
            if constexpr (decltype(first)::value) pv_prefetch(vpre, vbase, v_rd);
            else finish(scur, lo_j, vbase + vb * kTileB);
            if constexpr (decltype(last)::value) mask_block(snext, g, S - (blk0 + j + 1) * kBC);
            pv_next(lo_j, vbase + vb * kTileB, snext, lo_n);
            wait_vm<4 * (kDist - 1)>();  // K_{j+2} and V_{j+1} landed
            __syncthreads();
        };
        using Last = std::true_type;
        using NotLast = std::false_type;
        using First = std::true_type;
        using Next = std::false_type;
        if (nb > 1) {
            // Step 0: block 0's PV and block 1's scores.
            if (nb == 2) step(0, Phase<0>{}, First{}, Last{}, sa, sb, lo[0], lo[1]);
            else step(0, Phase<0>{}, First{}, NotLast{}, sa, sb, lo[0], lo[1]);
            int j = 1;
            // Odd steps hold the current block's scores in sb, even ones in sa.
            auto steady = [&](auto ph) {
                if constexpr (decltype(ph)::value % 2 == 1)
                    step(j, ph, Next{}, NotLast{}, sb, sa, lo[1], lo[0]);
                else
                    step(j, ph, Next{}, NotLast{}, sa, sb, lo[0], lo[1]);
                ++j;
            };
            while (j + 7 < nb) {
                steady(Phase<1>{});
                steady(Phase<2>{});
                steady(Phase<3>{});
                steady(Phase<4>{});
                steady(Phase<5>{});
                steady(Phase<0>{});
            }
            if (j + 2 < nb) {
                steady(Phase<1>{});
                if (j + 2 < nb) {
                    steady(Phase<2>{});
                    if (j + 2 < nb) {
                        steady(Phase<3>{});
                        if (j + 2 < nb) {
                            steady(Phase<4>{});
                            if (j + 2 < nb) steady(Phase<5>{});
                        }
                    }
                }
            }
            // Block j's scores and tile 0 are in sa and lo[0] when j is even.
            if (j + 1 < nb) {
                // The step of the last scores (j = nb - 2); it leaves the last
                // block's scores and tile 0 in sa and lo[0].
                if ((j & 1) == 0) {
                    sb[0] = sa[0];
                    sb[1] = sa[1];
                    lo[1][0] = lo[0][0];
                    lo[1][1] = lo[0][1];
                }
                step(j, Phase<-1>{}, Next{}, Last{}, sb, sa, lo[1], lo[0]);
                ++j;
                sb[0] = sa[0];
                sb[1] = sa[1];
                lo[1][0] = lo[0][0];
                lo[1][1] = lo[0][1];
            }
            // Last block of the segment (j = nb - 1) in sb and lo[1].
            finish(sb, lo[1], vbase + (j % kNB) * kTileB);
            pv(oacc, lo[1], hi, vbase + (j % kNB) * kTileB, v_rd, vpre);
        } else {
            pv_prefetch(vpre, vbase, v_rd);
            pv(oacc, lo[0], hi, vbase, v_rd, vpre);
        }
        wait_vm<0>();   // no load into LDS is pending
        __syncthreads();  // every wave is done with the buffers the next segment loads into
    };

    const int qi = q0 + li;
    char *const my_stash = stash + wave * kStashWaveB;
    float m_s = 0.f, l_s = 0.f;       // merged state of the segments so far
    int e_s = 0;
    bool normalised = false;          // oacc holds N (several segments) or O (one)
    for (int gs = g_first; gs < g_last; ++gs) {
        const int b0 = seg_begin(nkb, gs);
        segment(b0, seg_begin(nkb, gs + 1) - b0);
        const float l_g = halves_sum(lsum);
        if (nseg == 1) {  // one segment: its state is the result
            m_s = m;
            l_s = l_g;
            break;
        }
        normalised = true;
        // This segment's state, quantised like every segment state ...
        segment_state(oacc, l_g);
        const int e_g = state_exponent(oacc);
        quantise(oacc, e_g);
        if (gs == g_first) {
            m_s = m;
            l_s = l_g;
            e_s = e_g;
        } else {
            // ... merged into the stored state of the earlier segments.
            float wa, wb;
            merge_weights(m_s, l_s, m, l_g, c, m_s, l_s, wa, wb);
            merge_stored(oacc, my_stash, e_s, lane, wa, wb, true);
            if (gs + 1 < nseg) {   // segments 0-1 merged: quantised as a stored state
                e_s = state_exponent(oacc);
                quantise(oacc, e_s);
            }
        }
        if (gs + 1 < g_last) store_state(my_stash, oacc, e_s, lane);  // read back by this lane only
    }

    if (split_u >= 0) {
        // A share of a split tile: publish this workgroup's partial state, and
        // the last of the tile's workgroups to arrive merges them all.
        const int slot = split_u;
        store_state(tail.part + static_cast<int64_t>(slot) * kStashB + wave * kStashWaveB, oacc, e_s, lane);
        if (g == 0)
            tail.ml[slot * 256 + wave * kQW + li] = make_float4(m_s, l_s, __builtin_bit_cast(float, e_s), 0.f);
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
        // The stash is free now: its first word carries thread 0's arrival
        // count to the other waves.
        volatile int *arrived = reinterpret_cast<volatile int *>(stash);
        __syncthreads();
        const int tt = split_u % tail.n_split;
        if (tid == 0) *arrived = atomicAdd(&tail.count[tt], 1);
        __syncthreads();
        if (*arrived != tail.ways - 1) return;
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
        // The tile's partial states in segment order (slots tt + p n_split),
        // this workgroup's own read back like the others.
        auto slot_of = [&](int p) { return tt + p * tail.n_split; };
        auto part_of = [&](int p) {
            return tail.part + static_cast<int64_t>(slot_of(p)) * kStashB + wave * kStashWaveB;
        };
        float4 st = tail.ml[slot_of(0) * 256 + wave * kQW + li];
        m_s = st.x;
        l_s = st.y;
        load_state(oacc, part_of(0), __builtin_bit_cast(int, st.z), lane);
        for (int p = 1; p < tail.ways; ++p) {
            st = tail.ml[slot_of(p) * 256 + wave * kQW + li];
            float wa, wb;
            merge_weights(m_s, l_s, st.x, st.y, c, m_s, l_s, wa, wb);
            merge_stored(oacc, part_of(p), __builtin_bit_cast(int, st.z), lane, wa, wb, false);
            if (p + 1 < tail.ways) quantise(oacc, state_exponent(oacc));   // segments 0-1 merged
        }
        if (tid == 0) atomicExch(&tail.count[tt], 0);   // ready for the next launch on this scratch
    }

    const float inv = normalised ? 1.0f : 1.0f / l_s;
    if (lse != nullptr && g == 0 && qi < S)
        lse[static_cast<int64_t>(head) * S + qi] = m_s * c + __builtin_amdgcn_logf(l_s);
    if (qi < S) {
        __bf16 *orow = oh + static_cast<int64_t>(qi) * D;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
            for (int rb = 0; rb < 4; ++rb) {
                const f32x4 x = {oacc[dt][rb * 4 + 0] * inv, oacc[dt][rb * 4 + 1] * inv,
                                 oacc[dt][rb * 4 + 2] * inv, oacc[dt][rb * 4 + 3] * inv};
                store4(orow + dt * 32 + rb * 8 + g * 4, x);
            }
    }
}

// Launch shape per head dimension: WAVES waves per workgroup, NT tiles of 32
// queries per wave, 256 queries per workgroup.  d = 128: four waves of 64
// queries, one wave per SIMD (every K and V operand read from LDS feeds two
// MFMAs); d = 64: four waves of 32 queries, two workgroups per CU.
#ifndef HCMS_ATTN_LDS_DMA
#define HCMS_ATTN_LDS_DMA 1
#endif
// d = 128 with bf16 storage runs attention_dma_kernel.
constexpr bool kLdsDma = HCMS_ATTN_LDS_DMA != 0;

template <int D>
struct Shape {
    static constexpr int NT = D == 128 ? HCMS_ATTN_NT128 : 1;
    static constexpr int WAVES = D == 128 && NT == 1 ? 8 : 4;
    static constexpr int BR = kQW * NT * WAVES;       // queries per workgroup
    static constexpr int PER_CU = D == 128 ? 1 : 2;   // workgroups one CU holds
};

// The split of a d = 128 bf16 launch of W tiles on n_cu CUs (one workgroup
// per CU): when its last round holds rem = W mod n_cu tiles and 3 rem (or
// 2 rem) workgroups fit in one round, those tiles are split three (or two)
// ways by key segments, so the last round lasts a third (two thirds) as
// long.  With sp->tail >= 0 the last min(tail, W) tiles are the ones split:
// a launch whose last round is shared with another stream's launch splits
// the tiles that close the pooled rounds.  Needs scratch (none: every tile
// whole, the same results).
TailSplit plan_split(int64_t W, int S, const SplitScratch *sp) {
    TailSplit t{nullptr, nullptr, nullptr, static_cast<int>(W), 0, 1};
    const int nkb = (S + kBC - 1) / kBC;
    if (!sp || !sp->part || sp->n_cu < 2 || dma::n_segments(nkb) != dma::kSeg) return t;
    const int64_t n = sp->n_cu, rem = sp->tail >= 0 ? std::min(sp->tail, W) : W % n;
    if (rem == 0) return t;
    const int ways = 3 * rem <= n ? 3 : 2 * rem <= n ? 2 : 0;
    if (ways == 0 || rem * ways > sp->slots || rem > sp->counters) return t;
    t.part = static_cast<char *>(sp->part);
    t.ml = static_cast<float4 *>(sp->ml);
    t.count = sp->count;
    t.n_whole = static_cast<int>(W - rem);
    t.n_split = static_cast<int>(rem);
    t.ways = ways;
    return t;
}

template <int D, typename T>
hipError_t launch_typed(const void *q, const void *k, const void *v, void *o, float *lse, int S,
                        int n_heads, float c, const SplitScratch *split, hipStream_t stream) {
    using Sh = Shape<D>;
    const int n_qtiles = (S + Sh::BR - 1) / Sh::BR;
    const int64_t blocks = static_cast<int64_t>(n_qtiles) * n_heads;
    if (blocks > 0x7fffffff) return hipErrorInvalidValue;
    if constexpr (D == dma::kD && sizeof(T) == 2 && kLdsDma) {
        static_assert(Sh::NT == 1 && Sh::WAVES == dma::kWaves, "the DMA kernel covers 256 queries in 8 waves");
        const TailSplit t = plan_split(blocks, S, split);
        const int64_t grid = t.n_whole + static_cast<int64_t>(t.n_split) * t.ways;
        if (grid > 0x7fffffff) return hipErrorInvalidValue;
        attention_dma_kernel<false><<<static_cast<unsigned>(grid), 64 * dma::kWaves, 0, stream>>>(
            static_cast<const __bf16 *>(q), static_cast<const __bf16 *>(k), static_cast<const __bf16 *>(v),
            static_cast<__bf16 *>(o), lse, S, n_qtiles, c, t, Riders{});
    } else {
        attention_kernel<D, T, Sh::WAVES, Sh::NT, Sh::PER_CU><<<static_cast<unsigned>(blocks), 64 * Sh::WAVES, 0, stream>>>(
            static_cast<const T *>(q), static_cast<const T *>(k), static_cast<const T *>(v),
            static_cast<T *>(o), lse, S, n_qtiles, c);
    }
    return hipGetLastError();
}

}  // namespace

int attention_queries_per_block(int d) { return d == 128 ? Shape<128>::BR : Shape<64>::BR; }
int attention_blocks_per_cu(int d) { return d == 128 ? Shape<128>::PER_CU : Shape<64>::PER_CU; }

int64_t attention_split_slot_bytes() { return dma::kStashB + 256 * int64_t{sizeof(float4)}; }

int attention_split_ways(int64_t W, int S, int d, int dtype, int n_cu, int64_t tail) {
    if (!(kLdsDma && d == dma::kD && dtype == 0)) return 1;
    SplitScratch sp{};
    sp.part = sp.ml = reinterpret_cast<void *>(uintptr_t{256});   // placeholders: never dereferenced
    sp.n_cu = n_cu;
    sp.slots = sp.counters = n_cu;
    sp.tail = tail;
    const TailSplit t = plan_split(W, S, &sp);
    return t.n_split > 0 ? t.ways : 1;
}

hipError_t launch_attention(const void *q, const void *k, const void *v, void *o, float *lse, int S,
                            int n_heads, int d, float scale_log2e, int dtype,
                            const SplitScratch *split, hipStream_t stream) {
    if (S == 0 || n_heads == 0) return hipSuccess;
    if (d == 128 && dtype == 0)
        return launch_typed<128, __bf16>(q, k, v, o, lse, S, n_heads, scale_log2e, split, stream);
    if (d == 64 && dtype == 0)
        return launch_typed<64, __bf16>(q, k, v, o, lse, S, n_heads, scale_log2e, split, stream);
    if (d == 128 && dtype == 1)
        return launch_typed<128, float>(q, k, v, o, lse, S, n_heads, scale_log2e, split, stream);
    if (d == 64 && dtype == 1)
        return launch_typed<64, float>(q, k, v, o, lse, S, n_heads, scale_log2e, split, stream);
    return hipErrorInvalidValue;
}

hipError_t launch_attention_riding(const void *q, const void *k, const void *v, void *o, float *lse,
                                   int S, int n_heads, int d, float scale_log2e, int dtype,
                                   const RidingCopy *copies, int n_copies, int64_t H, int n_cu,
                                   const SplitScratch *split, bool *riding, hipStream_t stream) {
    *riding = false;
    const bool can = kLdsDma && d == dma::kD && dtype == 0 && S > 0 && n_heads > 0 && copies &&
                     n_copies >= 1 && n_copies <= 2 && n_cu > 0 && copy::strided_span_fits(H);
    if (!can)
        return launch_attention(q, k, v, o, lse, S, n_heads, d, scale_log2e, dtype, split, stream);
    using Sh = Shape<dma::kD>;
    const int64_t n_qtiles = (S + Sh::BR - 1) / Sh::BR;
    const TailSplit t = plan_split(n_qtiles * n_heads, S, split);
    const int64_t n_attn = t.n_whole + static_cast<int64_t>(t.n_split) * t.ways;
    const int64_t idle = (n_cu - n_attn % n_cu) % n_cu;
    Riders r{};
    r.S = S;
    r.H = H;
    r.n_jobs = static_cast<unsigned>(n_copies);
    const int64_t bx = copy::blocks_x(S, kRiderLog2U);
    r.bx = static_cast<unsigned>(bx);
    int64_t total = 0;
    for (int i = 0; i < n_copies; ++i) {
        const RidingCopy &cp = copies[i];
        if (cp.n_tensors < 1 || cp.n_tensors > 3 || cp.hc < 1 || cp.h0 < 0 || cp.h0 + cp.hc > H)
            return hipErrorInvalidValue;
        RiderJob &jb = r.job[i];
        for (int z = 0; z < cp.n_tensors; ++z) {
            jb.p.src[z] = static_cast<const char *>(cp.src[z]);
            jb.p.dst[z] = static_cast<char *>(cp.dst[z]);
        }
        jb.h0 = cp.h0;
        jb.hc = static_cast<unsigned>(cp.hc);
        jb.n_tensors = static_cast<unsigned>(cp.n_tensors);
        jb.unpack = cp.unpack ? 1 : 0;
        const int64_t blocks = bx * cp.hc * cp.n_tensors;
        jb.blocks = static_cast<unsigned>(blocks);
        total += blocks;
    }
    // Too few idle CUs, or more copy blocks than the 32-bit rider loop
    // counts: the caller launches the copies itself.
    if (idle < std::max(1, n_cu / 8) || total >= (int64_t{1} << 31) ||
        n_attn + idle > 0x7fffffff)
        return launch_attention(q, k, v, o, lse, S, n_heads, d, scale_log2e, dtype, split, stream);
    attention_dma_kernel<true><<<static_cast<unsigned>(n_attn + idle), 64 * dma::kWaves, 0, stream>>>(
        static_cast<const __bf16 *>(q), static_cast<const __bf16 *>(k), static_cast<const __bf16 *>(v),
        static_cast<__bf16 *>(o), lse, S, static_cast<int>(n_qtiles), scale_log2e, t, r);
    const hipError_t e = hipGetLastError();
    if (e == hipSuccess) *riding = true;
    return e;
}

}  // namespace hcms
