// Backward of the non-causal softmax attention, for gfx950 (bf16 MFMA).
//
// For one head, with s_ij = <q_i, k_j>, c = scale * log2(e), the forward's
// statistic L_i = log2 sum_j exp2(c s_ij) and the output gradient dO:
//   P_ij  = exp2(c s_ij - L_i)                       (softmax weights)
//   D_i   = <dO_i, O_i>          (= sum_j P_ij dP_ij, since O_i = sum_j P_ij v_j)
//   dP_ij = <dO_i, v_j>
//   dS_ij = P_ij (dP_ij - D_i)                       (gradient of scale * s_ij)
//   dQ_i  = scale sum_j dS_ij k_j
//   dK_j  = scale sum_i dS_ij q_i
//   dV_j  = sum_i P_ij dO_i
// the chain rule through the row softmax of the attention step of Alg. 1
// (Sec. 3.3 Property), used for training (the appendix's correctness and
// training validation).
//
// Two launches per head chunk, no atomics, so the result is deterministic and
// does not depend on the chunking:
//   * attention_dq_kernel, query-parallel (the forward's decomposition): a
//     wave owns 32 queries, keeps Q and dO as MFMA B operands in registers and
//     walks the key blocks, one 32-key half at a time: S^T = K Q^T and
//     dP^T = V dO^T (K and V row-major in LDS), then dS, then
//     dQ^T += K^T dS^T with K^T stored transposed in LDS, keys permuted like
//     V^T in the forward so that dS leaves the accumulator layout directly as
//     the B operand.  Its prologue computes D_i from dO and O and stores it
//     for the second launch.
//   * attention_dkdv_kernel, key-parallel: a wave owns 32 keys, keeps K as B
//     operands in registers (the workgroup's V rows sit in LDS for the whole
//     launch), and walks blocks of 32 queries.  Per block, S = Q K^T and
//     dP = dO V^T put one key per lane (the column) and 16 queries per lane
//     (rows), so P and dS are already B operands of dV^T += dO^T P and
//     dK^T += Q^T dS, with dO^T and Q^T transposed in LDS, queries permuted.
// Both run two waves per SIMD (8 waves per workgroup at d = 128, 4 waves and
// two workgroups per CU at d = 64): the 32-key halves in the first kernel
// and V in LDS in the second keep each wave within 256 registers, so one
// wave's MFMAs overlap the other's exponentials and LDS reads.
//
// At d = 128 with bf16 storage the two launches run DMA forms of these kernels
// (attention_dq_dma_kernel, attention_dkdv_dma_kernel): the streamed tiles (K
// and V, or Q, dO, L and D) go from global memory straight into LDS, three
// blocks ahead through four buffers, instead of through registers, and the
// transposed operands come from the row-major tiles by ds_read_b64_tr_b16.
// A 16-byte chunk c of tile row r sits at chunk position c ^ f(r), with
// f(r) = 4 (r mod 4) + (r / 4 mod 4), which keeps both the 16-byte row reads
// and the transposing reads free of bank conflicts.  The dQ form uses the
// operand values and MFMA order of attention_dq_kernel, so the two give the
// same bits; the dK/dV form adds the per-query statistics through one more
// MFMA each (see there), so its rounding differs from attention_dkdv_kernel's
// in the last bits.  Either way every query's and key's arithmetic depends on
// S, d and the data only, never on the chunking.
//
// With a caller's score-gradient workspace (d = 128, bf16) dQ comes from the
// stored dS instead: D = <dO, O> first (attention_delta_kernel), then the
// key-parallel launch, which also stores every dS tile it computes, then
// dQ^T = scale K^T dS^T over the stored tiles (attention_dq_ds_kernel): the
// scores and dP are computed once, 10 S^2 d FLOP per head instead of 14, for
// 2 S^2 bytes of dS written and read.
//
// Tails: loads go through buffer resources bounded by the head's tensor (rows
// >= S read as zeros); keys or queries past S get P = 0 and are not stored.
#include <algorithm>

#include "attention_tiles.h"
#include "hcms_internal.h"

namespace hcms {
namespace {

using namespace tiles;

// Query-parallel kernel: 8 waves (d = 128) or 4 waves at two workgroups per
// CU (d = 64), two waves per SIMD either way.
template <int D>
struct QTile {
    static constexpr int waves = D == 128 ? 8 : 4;
    static constexpr int threads = 64 * waves;
    static constexpr int per_cu = 8 / waves;
};
constexpr int kQB = 32;  // queries per block of the key-parallel kernel

// Transposed tiles of 32 queries: [D][kQB + 8], the same 16-byte padding as
// the forward's V^T (rows of 80 bytes: 16 consecutive rows hit disjoint banks).
template <int D>
struct QLds {
    static constexpr int RS = D + 8;        // row-major row stride (elements)
    static constexpr int TS = kQB + 8;      // transposed row stride (elements)
    static constexpr int R = kQB * RS;      // row-major tile (elements)
    static constexpr int TT = D * TS;       // transposed tile (elements)
};

__device__ inline unsigned bits(float x) { return __builtin_bit_cast(unsigned, x); }
__device__ inline float swap_halves_sum(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(bits(x), bits(x), false, false);
    return __builtin_bit_cast(float, static_cast<unsigned>(r[0])) +
           __builtin_bit_cast(float, static_cast<unsigned>(r[1]));
}

// XCD-aware order: workgroup b runs on XCD b % 8; each XCD takes a contiguous
// range of (head, tile) pairs.
__device__ inline int xcd_logical(int b, int nb) {
    const int xcd = b & 7, per = nb >> 3, rem = nb & 7;
    return xcd * per + min(xcd, rem) + (b >> 3);
}

// A 32 x 32 product over the head dimension: acc = A B^T with A rows from an
// LDS tile (row-major, stride RS) and B held as the D/16 register operands.
template <int D>
__device__ inline f32x16 rows_times_regs(const __bf16 *a, int rs, const bf16x8 (&b)[D / 16], int li,
                                          int g) {
    f32x16 acc = {};
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk) {
        const bf16x8 x = *reinterpret_cast<const bf16x8 *>(a + li * rs + kk * 16 + g * 8);
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(x, b[kk], acc, 0, 0, 0);
    }
    return acc;
}

// ---------------------------------------------------------------------------
// dQ (and D): query-parallel
// ---------------------------------------------------------------------------
template <int D, typename T>
__global__ __launch_bounds__(QTile<D>::threads, QTile<D>::per_cu) void attention_dq_kernel(
    const T *__restrict__ q, const T *__restrict__ k, const T *__restrict__ v,
    const T *__restrict__ o, const T *__restrict__ dout, const float *__restrict__ lse,
    T *__restrict__ dq, float *__restrict__ delta, int S, int n_qtiles, float c, float scale) {
    constexpr int KK = D / 16, DT = D / 32;
    __shared__ __attribute__((aligned(16))) __bf16 kbuf[2][Lds<D>::KT];   // K, row-major
    __shared__ __attribute__((aligned(16))) __bf16 vbuf[2][Lds<D>::KT];   // V, row-major
    __shared__ __attribute__((aligned(16))) __bf16 ktbuf[2][Lds<D>::VT];  // K^T, keys permuted

    const int logical = xcd_logical(blockIdx.x, gridDim.x);
    const int head = logical / n_qtiles;
    const int qtile = logical - head * n_qtiles;
    const int64_t hoff = static_cast<int64_t>(head) * S * D;
    const int64_t hbytes = static_cast<int64_t>(S) * D * sizeof(T);
    const __amdgpu_buffer_rsrc_t qr = head_rsrc(q + hoff, hbytes);
    const __amdgpu_buffer_rsrc_t kr = head_rsrc(k + hoff, hbytes);
    const __amdgpu_buffer_rsrc_t vr = head_rsrc(v + hoff, hbytes);
    const __amdgpu_buffer_rsrc_t or_ = head_rsrc(o + hoff, hbytes);
    const __amdgpu_buffer_rsrc_t dr = head_rsrc(dout + hoff, hbytes);

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int li = lane & 31, g = lane >> 5;
    const int qi = qtile * (kQW * QTile<D>::waves) + wave * kQW + li;

    bf16x8 qreg[KK], doreg[KK];
    float dpart = 0.f;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
        const unsigned off = static_cast<unsigned>(qi * D + kk * 16 + g * 8) * sizeof(T);
        qreg[kk] = __builtin_bit_cast(bf16x8, load8<T>(qr, off));
        doreg[kk] = __builtin_bit_cast(bf16x8, load8<T>(dr, off));
        const bf16x8 ov = __builtin_bit_cast(bf16x8, load8<T>(or_, off));
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const bf16x2 a = {doreg[kk][2 * e], doreg[kk][2 * e + 1]};
            const bf16x2 b = {ov[2 * e], ov[2 * e + 1]};
            dpart = __builtin_amdgcn_fdot2_f32_bf16(a, b, dpart, false);
        }
    }
    const float Di = swap_halves_sum(dpart);
    const float Li = qi < S ? lse[static_cast<int64_t>(head) * S + qi] : 0.f;
    if (g == 0 && qi < S) delta[static_cast<int64_t>(head) * S + qi] = Di;

    f32x16 dqacc[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) dqacc[dt] = f32x16{};
    const int nkb = (S + kBC - 1) / kBC;

    // Staging: V in the row pattern, K in the key-pair pattern (written both
    // row-major and transposed).
    Stage<D, T, QTile<D>::waves> st;
    st.load(vr, kr, 0, 0, tid);
    st.store_k(vbuf[0], tid);
    st.store_v_rows(kbuf[0], tid);
    st.store_v(ktbuf[0], tid);
    __syncthreads();

    for (int j = 0; j < nkb; ++j) {
        const int b = j & 1;
        if (j + 1 < nkb) st.load(vr, kr, j + 1, j + 1, tid);
        const int kvalid = S - j * kBC;
        // The block's two 32-key halves one after the other: S^T and dP^T of
        // the half, dS, then its two 16-key steps of dQ^T += K^T dS^T.
#pragma unroll
        for (int mt = 0; mt < 2; ++mt) {
            f32x16 sacc = {}, dpacc = {};
#pragma unroll
            for (int kk = 0; kk < KK; ++kk) {
                const int row = (mt * 32 + li) * Lds<D>::KS + kk * 16 + g * 8;
                const bf16x8 ka = *reinterpret_cast<const bf16x8 *>(kbuf[b] + row);
                const bf16x8 va = *reinterpret_cast<const bf16x8 *>(vbuf[b] + row);
                sacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qreg[kk], sacc, 0, 0, 0);
                dpacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, doreg[kk], dpacc, 0, 0, 0);
            }
            bf16x8 dsb[2];
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                f32x8 x;
#pragma unroll
                for (int r = 0; r < 8; ++r) {
                    const int rr = h * 8 + r;
                    const int key = mt * 32 + (rr >> 2) * 8 + g * 4 + (rr & 3);
                    const float p = key < kvalid
                        ? __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[rr], c, -Li)) : 0.f;
                    x[r] = p * (dpacc[rr] - Di);
                }
                dsb[h] = __builtin_convertvector(x, bf16x8);
            }
#pragma unroll
            for (int dt = 0; dt < DT; ++dt)
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    const int ks = mt * 2 + h;
                    const bf16x8 a = *reinterpret_cast<const bf16x8 *>(
                        ktbuf[b] + (dt * 32 + li) * Lds<D>::VS + (ks * 2 + g) * 8);
                    dqacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, dsb[h], dqacc[dt], 0, 0, 0);
                }
        }
        if (j + 1 < nkb) {
            st.store_k(vbuf[b ^ 1], tid);
            st.store_v_rows(kbuf[b ^ 1], tid);
            st.store_v(ktbuf[b ^ 1], tid);
        }
        __syncthreads();
    }

    if (qi < S) {
        T *row = dq + hoff + static_cast<int64_t>(qi) * D;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
            for (int rb = 0; rb < 4; ++rb) {
                const f32x4 x = {dqacc[dt][rb * 4 + 0] * scale, dqacc[dt][rb * 4 + 1] * scale,
                                 dqacc[dt][rb * 4 + 2] * scale, dqacc[dt][rb * 4 + 3] * scale};
                store4(row + dt * 32 + rb * 8 + g * 4, x);
            }
    }
}

// dQ for d = 128 with bf16 storage: K and V blocks go from global memory
// straight into LDS (load_lds), three steps ahead, through four buffers each;
// K^T operands come from the row-major K tile by ds_read_b64_tr_b16 (see
// attention_dma_kernel for the instruction's lane layout).  Both tiles are
// 64 keys x 256 bytes with chunk c of row r at position c ^ swz(r),
// swz(r) = 4 (r mod 4) + (r / 4) mod 4: 16 consecutive rows of one chunk land
// in 16 different groups of 4 banks (the 16-byte row reads of S^T = K Q^T and
// dP^T = V dO^T), and so do 4 rows x 4 chunks (the transposing reads).  The
// operand values and the MFMA order are those of attention_dq_kernel.
namespace bdma {

constexpr int kD = 128;
constexpr int kWaves = 8;
constexpr int kRowB = kD * 2;
constexpr int kTileB = kBC * kRowB;                    // 16 KiB
constexpr int kNB = 4;                                 // LDS buffers per tensor
constexpr int kDist = 3;                               // steps between a block's load and its use
constexpr int kPerWave = kTileB / (64 * 16) / kWaves;  // DMA instructions per wave and block
static_assert(kPerWave == 2 && kDist + 1 <= kNB, "wait counts below assume this");

__device__ inline unsigned swz(unsigned r) { return ((r & 3) << 2) | ((r >> 2) & 3); }

constexpr int kDsTileB = kQW * kQB * 2;  // one stored 32 x 32 tile of dS (bf16)
constexpr int kDsGroupB = 8 * kDsTileB;   // the tiles of 8 query blocks at one key tile

template <int P>
struct Phase {
    static constexpr int value = P;
};
template <bool B>
struct Flag {
    static constexpr bool value = B;
};

// x = hi + mid + lo exactly, each a bf16 (a float's 24-bit significand in
// three 8-bit pieces, each piece's rounding error carried into the next).
__device__ inline void split3(float x, __bf16 &hi, __bf16 &mid, __bf16 &lo) {
    hi = static_cast<__bf16>(x);
    const float r = x - static_cast<float>(hi);
    mid = static_cast<__bf16>(r);
    lo = static_cast<__bf16>(r - static_cast<float>(mid));
}

}  // namespace bdma

__global__ __launch_bounds__(64 * bdma::kWaves, bdma::kWaves / 4) void attention_dq_dma_kernel(
    const __bf16 *__restrict__ q, const __bf16 *__restrict__ k, const __bf16 *__restrict__ v,
    const __bf16 *__restrict__ o, const __bf16 *__restrict__ dout, const float *__restrict__ lse,
    __bf16 *__restrict__ dq, float *__restrict__ delta, int S, int n_qtiles, float c, float scale) {
    using namespace bdma;
    constexpr int D = kD, KK = D / 16, DT = D / 32;
    __shared__ __attribute__((aligned(1024))) char lds[2 * kNB * kTileB];
    const char *const kbase = lds;                 // K buffer b at kbase + b * kTileB
    const char *const vbase = lds + kNB * kTileB;  // V buffer b at vbase + b * kTileB

    const int logical = xcd_logical(blockIdx.x, gridDim.x);
    const int head = logical / n_qtiles;
    const int qtile = logical - head * n_qtiles;
    const int64_t hoff = static_cast<int64_t>(head) * S * D;
    const int64_t hbytes = static_cast<int64_t>(S) * D * 2;
    const __amdgpu_buffer_rsrc_t qr = head_rsrc(q + hoff, hbytes);
    const __amdgpu_buffer_rsrc_t kr = head_rsrc(k + hoff, hbytes);
    const __amdgpu_buffer_rsrc_t vr = head_rsrc(v + hoff, hbytes);
    const __amdgpu_buffer_rsrc_t or_ = head_rsrc(o + hoff, hbytes);
    const __amdgpu_buffer_rsrc_t dr = head_rsrc(dout + hoff, hbytes);

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int li = lane & 31, g = lane >> 5;
    const int qi = qtile * (kQW * kWaves) + wave * kQW + li;

    bf16x8 qreg[KK], doreg[KK];
    float dpart = 0.f;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
        const unsigned off = static_cast<unsigned>(qi * D + kk * 16 + g * 8) * 2;
        qreg[kk] = __builtin_bit_cast(bf16x8, load8<__bf16>(qr, off));
        doreg[kk] = __builtin_bit_cast(bf16x8, load8<__bf16>(dr, off));
        const bf16x8 ov = __builtin_bit_cast(bf16x8, load8<__bf16>(or_, off));
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const bf16x2 a = {doreg[kk][2 * e], doreg[kk][2 * e + 1]};
            const bf16x2 b = {ov[2 * e], ov[2 * e + 1]};
            dpart = __builtin_amdgcn_fdot2_f32_bf16(a, b, dpart, false);
        }
    }
    const float Di = swap_halves_sum(dpart);
    const float Li = qi < S ? lse[static_cast<int64_t>(head) * S + qi] : 0.f;
    if (g == 0 && qi < S) delta[static_cast<int64_t>(head) * S + qi] = Di;
    drain_vm_loads();

    // Lane offsets: DMA sources (row r = 4 (2 wave + i) + lane / 16, chunk at
    // position lane % 16), 16-byte row reads (row li of a 32-key half, chunk
    // 2 kk + g) and transposing K^T reads (lane t = lane % 16 of group
    // G = lane / 16; second read 8 rows on, whose swizzle differs).
    unsigned src[kPerWave];
#pragma unroll
    for (int i = 0; i < kPerWave; ++i) {
        const unsigned r = 4 * (kPerWave * wave + i) + (lane >> 4), p = lane & 15;
        src[i] = r * kRowB + ((p ^ swz(r)) << 4);
    }
    unsigned row_rd[KK];
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) row_rd[kk] = li * kRowB + (((2 * kk + g) ^ swz(li)) << 4);
    unsigned tr_rd[2][DT];
    {
        const unsigned G = lane >> 4, t = lane & 15;
#pragma unroll
        for (int hh = 0; hh < 2; ++hh)
#pragma unroll
            for (int dt = 0; dt < DT; ++dt) {
                const unsigned r = 4 * (G >> 1) + (t >> 2) + 8 * hh;  // key row within a 16-key step
                const unsigned col = dt * 32 + 16 * (G & 1) + 4 * (t & 3);
                tr_rd[hh][dt] = r * kRowB + (((col >> 3) ^ swz(r)) << 4) + ((col & 7) << 1);
            }
    }
#pragma unroll
    for (int hh = 0; hh < 2; ++hh)
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) asm volatile("" : "+v"(tr_rd[hh][dt]));
    const unsigned lds0 = static_cast<unsigned>(reinterpret_cast<uintptr_t>(lds));
    const unsigned wave_dst = lds0 + kPerWave * wave * 1024;
    auto issue = [&](int blk) {
        const unsigned kd = wave_dst + (blk & (kNB - 1)) * kTileB;
#pragma unroll
        for (int i = 0; i < kPerWave; ++i) load_lds(kd + i * 1024, kr, src[i], blk * kTileB);
#pragma unroll
        for (int i = 0; i < kPerWave; ++i) load_lds(kd + kNB * kTileB + i * 1024, vr, src[i], blk * kTileB);
    };

    f32x16 dqacc[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) dqacc[dt] = f32x16{};
    const int nkb = (S + kBC - 1) / kBC;

    // Prologue: blocks 0..kDist-1 in flight; step j issues block j + kDist.
#pragma unroll
    for (int blk = 0; blk < kDist; ++blk) issue(blk);
    wait_vm<4 * (kDist - 1)>();  // block 0 landed
    __syncthreads();

    typedef __attribute__((address_space(3))) bf16x4 LdsV4;
    // Block j in buffer P (P = j % kNB, or -1 when known only at run time);
    // only the last block (M) can hold keys past S.
    auto step = [&](int j, auto ph, auto masked) {
        constexpr int P = decltype(ph)::value;
        constexpr bool M = decltype(masked)::value;
        const int bi = P >= 0 ? P : j % kNB;
        const char *kb = kbase + bi * kTileB;
        const char *vb = vbase + bi * kTileB;
        issue(j + kDist);
        const int kvalid = S - j * kBC;
#pragma unroll
        for (int mt = 0; mt < 2; ++mt) {
            f32x16 sacc = {}, dpacc = {};
            // Row operands read two k-steps ahead of their MFMAs (the fences
            // keep the compiler from moving the reads next to their use).
            bf16x8 ka[3], va[3];
#pragma unroll
            for (int kk = 0; kk < 2; ++kk) {
                ka[kk] = *reinterpret_cast<const bf16x8 *>(kb + row_rd[kk] + mt * 32 * kRowB);
                va[kk] = *reinterpret_cast<const bf16x8 *>(vb + row_rd[kk] + mt * 32 * kRowB);
            }
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int kk = 0; kk < KK; ++kk) {
                if (kk + 2 < KK) {
                    ka[(kk + 2) % 3] = *reinterpret_cast<const bf16x8 *>(kb + row_rd[kk + 2] + mt * 32 * kRowB);
                    va[(kk + 2) % 3] = *reinterpret_cast<const bf16x8 *>(vb + row_rd[kk + 2] + mt * 32 * kRowB);
                }
                sacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[kk % 3], qreg[kk], sacc, 0, 0, 0);
                dpacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va[kk % 3], doreg[kk], dpacc, 0, 0, 0);
                __builtin_amdgcn_sched_barrier(0);
            }
            // The K^T operands of this half's dQ products, read before the
            // softmax so that its arithmetic covers their latency.
            bf16x8 kt[DT][2];
#pragma unroll
            for (int dt = 0; dt < DT; ++dt)
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    const char *p0 = kb + (mt * 2 + h) * 16 * kRowB;
                    const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((LdsV4 *)(p0 + tr_rd[0][dt]));
                    const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((LdsV4 *)(p0 + tr_rd[1][dt]));
                    kt[dt][h] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
                }
            __builtin_amdgcn_sched_barrier(0);
            bf16x8 dsb[2];
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                f32x8 x;
#pragma unroll
                for (int r = 0; r < 8; ++r) {
                    const int rr = h * 8 + r;
                    const int key = mt * 32 + (rr >> 2) * 8 + g * 4 + (rr & 3);
                    const float p = !M || key < kvalid
                        ? __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[rr], c, -Li)) : 0.f;
                    x[r] = p * (dpacc[rr] - Di);
                }
                dsb[h] = __builtin_convertvector(x, bf16x8);
            }
#pragma unroll
            for (int dt = 0; dt < DT; ++dt)
#pragma unroll
                for (int h = 0; h < 2; ++h)
                    dqacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kt[dt][h], dsb[h], dqacc[dt], 0, 0, 0);
        }
        wait_vm<4 * (kDist - 1)>();  // block j + 1 landed
        __syncthreads();
    };
    const int nwhole = nkb - 1;  // every block but the last holds 64 keys below S
    int j = 0;
    for (; j + 4 <= nwhole; j += 4) {
        step(j, Phase<0>{}, Flag<false>{});
        step(j + 1, Phase<1>{}, Flag<false>{});
        step(j + 2, Phase<2>{}, Flag<false>{});
        step(j + 3, Phase<3>{}, Flag<false>{});
    }
    for (; j < nwhole; ++j) step(j, Phase<-1>{}, Flag<false>{});
    step(nwhole, Phase<-1>{}, Flag<true>{});
    wait_vm<0>();  // no load into LDS is pending when the workgroup ends

    if (qi < S) {
        __bf16 *row = dq + hoff + static_cast<int64_t>(qi) * D;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
            for (int rb = 0; rb < 4; ++rb) {
                const f32x4 x = {dqacc[dt][rb * 4 + 0] * scale, dqacc[dt][rb * 4 + 1] * scale,
                                 dqacc[dt][rb * 4 + 2] * scale, dqacc[dt][rb * 4 + 3] * scale};
                store4(row + dt * 32 + rb * 8 + g * 4, x);
            }
    }
}

// ---------------------------------------------------------------------------
// dK, dV: key-parallel
// ---------------------------------------------------------------------------
// Key-parallel kernel: 8 waves (d = 128) or 4 waves at two workgroups per CU
// (d = 64); a wave owns 32 keys.
template <int D>
struct KTile {
    static constexpr int waves = D == 128 ? 8 : 4;
    static constexpr int threads = 64 * waves;
    static constexpr int per_cu = 8 / waves;
    static constexpr int keys = kQW * waves;
};

// Staging of one block of 32 queries: Q (first half of the threads) and dO
// (second half) in query pairs, stored row-major and transposed; L and D as 32
// floats each.
template <int D, typename T>
struct QStage {
    static constexpr int CH = D / 8;
    static constexpr unsigned ROWB = D * sizeof(T), CHB = 8 * sizeof(T);
    static constexpr int TASKS = (kQB / 2) * CH;  // (query pair, chunk) tasks per tensor
    static_assert(2 * TASKS <= KTile<D>::threads, "one task per thread at most");
    u32x4 x[2];
    f32x4 stat;

    __device__ static int pair(int t) { return t & 15; }
    __device__ static int chunk(int t) { return t >> 4; }

    __device__ void load(__amdgpu_buffer_rsrc_t qr, __amdgpu_buffer_rsrc_t dr,
                         __amdgpu_buffer_rsrc_t lr, __amdgpu_buffer_rsrc_t er, int blk, int tid) {
        const unsigned q0 = static_cast<unsigned>(blk) * kQB;
        if (tid < 2 * TASKS) {
            const int t = tid % TASKS;
            const unsigned off = (q0 + 2 * pair(t)) * ROWB + chunk(t) * CHB;
            x[0] = load8<T>(tid < TASKS ? qr : dr, off);
            x[1] = load8<T>(tid < TASKS ? qr : dr, off + ROWB);
        }
        // Threads 0..7 fetch L, 8..15 fetch D, 4 floats each.
        if (tid < 16) {
            const unsigned off = (q0 + (tid & 7) * 4) * 4u;
            stat = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                                 tid < 8 ? lr : er, off, 0, 0));
        }
    }

    __device__ void store(__bf16 *qrow, __bf16 *drow, __bf16 *qt, __bf16 *dt, float *ls, float *ds,
                          int tid) const {
        if (tid < 2 * TASKS) {
            const int t = tid % TASKS, p = pair(t), ch = chunk(t);
            __bf16 *r = (tid < TASKS ? qrow : drow) + 2 * p * QLds<D>::RS + ch * 8;
            *reinterpret_cast<u32x4 *>(r) = x[0];
            *reinterpret_cast<u32x4 *>(r + QLds<D>::RS) = x[1];
            __bf16 *tp = (tid < TASKS ? qt : dt) + ch * 8 * QLds<D>::TS + vt_pos(2 * p);
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const unsigned sel = (e & 1) ? 0x07060302u : 0x05040100u;
                *reinterpret_cast<unsigned *>(tp + e * QLds<D>::TS) =
                    __builtin_amdgcn_perm(x[1][e >> 1], x[0][e >> 1], sel);
            }
        }
        if (tid < 16) *reinterpret_cast<f32x4 *>((tid < 8 ? ls : ds) + (tid & 7) * 4) = stat;
    }
};

// dK, dV for d = 128 with bf16 storage: the blocks of 32 queries (Q, dO, L,
// D) go from global memory straight into LDS, three blocks ahead, through four
// buffers each; Q and dO tiles are 32 x 256 bytes with the swizzle of
// attention_dq_dma_kernel, read as 16-byte rows (S = Q K^T, dP = dO V^T) and
// transposed by ds_read_b64_tr_b16 (dV^T += dO^T P, dK^T += Q^T dS).  Waves
// 0 and 1 also load L and D (4 bytes per lane), so they count one more load
// per block.  L and D enter the scores through one more MFMA each, and the two
// waves of each SIMD take a step's work in different orders (both below).
template <bool kDs>
__global__ __launch_bounds__(64 * bdma::kWaves, bdma::kWaves / 4) void attention_dkdv_dma_kernel(
    const __bf16 *__restrict__ q, const __bf16 *__restrict__ k, const __bf16 *__restrict__ v,
    const __bf16 *__restrict__ dout, const float *__restrict__ lse, const float *__restrict__ delta,
    __bf16 *__restrict__ dk, __bf16 *__restrict__ dv, char *__restrict__ dsg, int S, int n_ktiles,
    float c, float scale) {
    using namespace bdma;
    constexpr int D = kD, KK = D / 16, DT = D / 32, NT = 64 * kWaves, KEYS = kQW * kWaves;
    constexpr int QTB = kQB * kRowB;  // one block of 32 queries: 8 KiB
    constexpr int STB = 64 * 4;       // one statistics load: 64 floats
    static_assert(QTB == 1024 * kWaves, "one DMA instruction per wave and tensor");
    __shared__ __attribute__((aligned(16))) __bf16 vrows[KEYS * QLds<D>::RS];
    __shared__ __attribute__((aligned(1024))) char lds[kNB * (2 * QTB + 2 * STB)];
    const char *const qbase = lds;                  // Q block buffer b at qbase + b * QTB
    const char *const dbase = lds + kNB * QTB;      // dO
    const char *const lbase = lds + 2 * kNB * QTB;  // L (STB bytes per buffer)
    const char *const ebase = lbase + kNB * STB;    // D

    const int logical = xcd_logical(blockIdx.x, gridDim.x);
    const int head = logical / n_ktiles;
    const int ktile = logical - head * n_ktiles;
    const int64_t hoff = static_cast<int64_t>(head) * S * D;
    const int64_t hbytes = static_cast<int64_t>(S) * D * 2;
    const __amdgpu_buffer_rsrc_t qr = head_rsrc(q + hoff, hbytes);
    const __amdgpu_buffer_rsrc_t kr = head_rsrc(k + hoff, hbytes);
    const __amdgpu_buffer_rsrc_t vr = head_rsrc(v + hoff, hbytes);
    const __amdgpu_buffer_rsrc_t dr = head_rsrc(dout + hoff, hbytes);
    const __amdgpu_buffer_rsrc_t lr = head_rsrc(lse + static_cast<int64_t>(head) * S, int64_t{S} * 4);
    const __amdgpu_buffer_rsrc_t er = head_rsrc(delta + static_cast<int64_t>(head) * S, int64_t{S} * 4);

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int li = lane & 31, g = lane >> 5;
    const int key0 = ktile * KEYS;
    const int kj = key0 + wave * kQW + li;

    bf16x8 kreg[KK];
#pragma unroll
    for (int kk = 0; kk < KK; ++kk)
        kreg[kk] = __builtin_bit_cast(
            bf16x8, load8<__bf16>(kr, static_cast<unsigned>(kj * D + kk * 16 + g * 8) * 2));
    constexpr int CH = D / 8;
#pragma unroll
    for (int i = 0; i < KEYS * CH / NT; ++i) {
        const int u = tid + i * NT, row = u / CH, ch = u % CH;
        *reinterpret_cast<u32x4 *>(vrows + row * QLds<D>::RS + ch * 8) =
            load8<__bf16>(vr, static_cast<unsigned>((key0 + row) * D + ch * 8) * 2);
    }
    drain_vm_loads();
    f32x16 dkacc[DT], dvacc[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
        dkacc[dt] = f32x16{};
        dvacc[dt] = f32x16{};
    }
    const int nqb = (S + kQB - 1) / kQB;
    const __bf16 *vmine = vrows + (wave * kQW + li) * QLds<D>::RS + g * 8;

    // Lane offsets: DMA source (row 4 wave + lane / 16, chunk at position
    // lane % 16), 16-byte row reads (query li, chunk 2 kk + g) and the two
    // transposing reads of each 16-query step.
    unsigned src;
    {
        const unsigned r = 4 * wave + (lane >> 4), p = lane & 15;
        src = r * kRowB + ((p ^ swz(r)) << 4);
    }
    unsigned row_rd[KK];
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) row_rd[kk] = li * kRowB + (((2 * kk + g) ^ swz(li)) << 4);
    unsigned tr_rd[2][DT];
    {
        const unsigned G = lane >> 4, t = lane & 15;
#pragma unroll
        for (int hh = 0; hh < 2; ++hh)
#pragma unroll
            for (int dt = 0; dt < DT; ++dt) {
                const unsigned r = 4 * (G >> 1) + (t >> 2) + 8 * hh;
                const unsigned col = dt * 32 + 16 * (G & 1) + 4 * (t & 3);
                tr_rd[hh][dt] = r * kRowB + (((col >> 3) ^ swz(r)) << 4) + ((col & 7) << 1);
            }
    }
#pragma unroll
    for (int hh = 0; hh < 2; ++hh)
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) asm volatile("" : "+v"(tr_rd[hh][dt]));
    const unsigned lds0 = static_cast<unsigned>(reinterpret_cast<uintptr_t>(lds));
    auto issue = [&](int blk) {
        const unsigned b = blk & (kNB - 1);
        load_lds(lds0 + b * QTB + wave * 1024, qr, src, blk * QTB);
        load_lds(lds0 + kNB * QTB + b * QTB + wave * 1024, dr, src, blk * QTB);
        if (wave == 0) load_lds_b32(lds0 + 2 * kNB * QTB + b * STB, lr, lane * 4, blk * kQB * 4);
        if (wave == 1) load_lds_b32(lds0 + 2 * kNB * QTB + kNB * STB + b * STB, er, lane * 4, blk * kQB * 4);
    };
    // All but the latest block's loads of this wave landed.
    auto wait_one_block = [&]() {
        if (wave < 2) wait_vm<3>();
        else wait_vm<2>();
    };

#pragma unroll
    for (int blk = 0; blk < kDist; ++blk) issue(blk);
    wait_one_block();  // blocks 0 and 1 landed (and the V rows were stored)
    __syncthreads();

    // The statistics of a block's queries enter S and dP through one more
    // MFMA each: A holds -L_i / c (or -D_i) of query i = li in three bf16
    // pieces at k = 0..2, B holds ones there and zeros elsewhere, so the
    // product adds the exact fp32 value to all 32 keys' entries of that query
    // (its accumulator row), with no broadcast of per-row values.
    // A fourth term at k = 3 takes keys past S out: A holds -2^100 there and
    // B holds 1 in the column of a key past S (0 for the others, whose sums
    // gain an exact -0), so such a key's score and dP become about -2^100,
    // its P exactly 0 and its dS exactly -0 for every query.  Their dK and dV
    // are never stored; the stored dS (kDs) needs them finite and zero.
    const __bf16 past = kj < S ? static_cast<__bf16>(0.f) : static_cast<__bf16>(1.f);
    const bf16x8 ones = g == 0 ? bf16x8{1, 1, 1, past, 0, 0, 0, 0} : bf16x8{};
    const float inv_c = 1.0f / c;
    auto pieces = [](float x) {
        __bf16 h, m, l;
        split3(x, h, m, l);
        return bf16x8{h, m, l, static_cast<__bf16>(-0x1p100f), 0, 0, 0, 0};
    };
    // Score gradients kept for the dQ product (kDs): the wave's 32 keys are
    // key tile kw = 8 ktile + wave; the 32 x 32 tile of query block i sits at
    // byte ((head nqt + i / 8) nkw + kw) 16 KiB + (i % 8) 2 KiB of dsg
    // (nqt = n_ktiles tiles of 256 queries), lane (li, g)'s dsb[h] at
    // h KiB + 32 li + 16 g in it (see attention_dq_ds_kernel).
    const int nkw = 8 * n_ktiles;
    char *const ds_wave =
        kDs ? dsg + (static_cast<int64_t>(head) * n_ktiles * nkw + ktile * 8 + wave) * kDsGroupB
            : nullptr;
    const int64_t ds_step = static_cast<int64_t>(nkw) * kDsGroupB;   // per 8 query blocks
    const unsigned ds_lane = li * 32 + g * 16;

    // s = Q K^T - L / c and dp = dO V^T - D of the block in buffer bi, rows =
    // queries; the statistic is added last, so dp - D rounds once, as a
    // subtraction would (a query whose dP equals D gets dS = 0 exactly).
    auto scores = [&](int bi, f32x16 &s, f32x16 &dp) {
        const char *qb = qbase + bi * QTB;
        const char *db = dbase + bi * QTB;
        const float *lb = reinterpret_cast<const float *>(lbase + bi * STB);
        const float *eb = reinterpret_cast<const float *>(ebase + bi * STB);
        s = f32x16{};
        dp = f32x16{};
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) {
            const bf16x8 qa = *reinterpret_cast<const bf16x8 *>(qb + row_rd[kk]);
            const bf16x8 da = *reinterpret_cast<const bf16x8 *>(db + row_rd[kk]);
            const bf16x8 vb = *reinterpret_cast<const bf16x8 *>(vmine + kk * 16);
            s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qa, kreg[kk], s, 0, 0, 0);
            dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(da, vb, dp, 0, 0, 0);
        }
        s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(pieces(-lb[li] * inv_c), ones, s, 0, 0, 0);
        dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(pieces(-eb[li]), ones, dp, 0, 0, 0);
    };
    typedef __attribute__((address_space(3))) bf16x4 LdsV4;
    // P and dS of block i from its scores (queries past S get P = 0 when M),
    // then dV^T += dO^T P and dK^T += Q^T dS from buffer bi.
    auto products = [&](int i, int bi, const f32x16 &s, const f32x16 &dp, auto masked) {
        constexpr bool M = decltype(masked)::value;
        const char *qb = qbase + bi * QTB;
        const char *db = dbase + bi * QTB;
        const int qvalid = S - i * kQB;
        bf16x8 pb[2], dsb[2];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            f32x8 p, ds;
#pragma unroll
            for (int r = 0; r < 8; ++r) {
                const int rr = h * 8 + r;
                const int qrow = (rr >> 2) * 8 + g * 4 + (rr & 3);
                p[r] = !M || qrow < qvalid ? __builtin_amdgcn_exp2f(s[rr] * c) : 0.f;
                ds[r] = p[r] * dp[rr];
            }
            pb[h] = __builtin_convertvector(p, bf16x8);
            dsb[h] = __builtin_convertvector(ds, bf16x8);
        }
        if constexpr (kDs) {
            // Through a buffer resource over the 8 tiles of this key tile
            // (scalar base and offset): no 64-bit lane addresses.
            const __amdgpu_buffer_rsrc_t dr = head_rsrc(ds_wave + (i >> 3) * ds_step, kDsGroupB);
            __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, dsb[0]), dr, ds_lane,
                                                   (i & 7) * kDsTileB, 0);
            __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, dsb[1]), dr,
                                                   ds_lane + 1024, (i & 7) * kDsTileB, 0);
        }
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
            for (int qs = 0; qs < 2; ++qs) {
                const char *d0 = db + qs * 16 * kRowB, *q0p = qb + qs * 16 * kRowB;
                const bf16x4 dlo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((LdsV4 *)(d0 + tr_rd[0][dt]));
                const bf16x4 dhi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((LdsV4 *)(d0 + tr_rd[1][dt]));
                const bf16x4 qlo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((LdsV4 *)(q0p + tr_rd[0][dt]));
                const bf16x4 qhi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((LdsV4 *)(q0p + tr_rd[1][dt]));
                const bf16x8 da = __builtin_shufflevector(dlo, dhi, 0, 1, 2, 3, 4, 5, 6, 7);
                const bf16x8 qa = __builtin_shufflevector(qlo, qhi, 0, 1, 2, 3, 4, 5, 6, 7);
                dvacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(da, pb[qs], dvacc[dt], 0, 0, 0);
                dkacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qa, dsb[qs], dkacc[dt], 0, 0, 0);
            }
    };
    // The two waves of a SIMD (w and w + 4) take a step's work in different
    // orders, so that one's MFMAs run while the other computes exponentials:
    // waves 0-3 compute block i's scores, then its softmax and products;
    // waves 4-7 start a step with the softmax and products of block i (scores
    // from the step before) and end it with the scores of block i + 1.  Step
    // i loads block i + 3 into the buffer block i - 1 left and ends when
    // block i + 2 has landed, which the late scores of waves 4-7 need.
    // Each group runs its own loop (the same number of barriers).
    const int nwhole = nqb - 1;  // every block but the last holds 32 queries below S
    auto run = [&](auto late_flag) {
        constexpr bool kLate = decltype(late_flag)::value;
        f32x16 sc, dpc;
        if (kLate) scores(0, sc, dpc);
        auto step = [&](int i, auto ph, auto masked) {
            constexpr int P = decltype(ph)::value;
            constexpr bool M = decltype(masked)::value;
            const int bi = P >= 0 ? P : i % kNB;
            issue(i + kDist);
            if constexpr (!kLate) {
                scores(bi, sc, dpc);
                products(i, bi, sc, dpc, masked);
            } else {
                products(i, bi, sc, dpc, masked);
                if constexpr (!M) scores((bi + 1) & (kNB - 1), sc, dpc);
            }
            wait_one_block();
            __syncthreads();
        };
        int i = 0;
        for (; i + 4 <= nwhole; i += 4) {
            step(i, Phase<0>{}, Flag<false>{});
            step(i + 1, Phase<1>{}, Flag<false>{});
            step(i + 2, Phase<2>{}, Flag<false>{});
            step(i + 3, Phase<3>{}, Flag<false>{});
        }
        for (; i < nwhole; ++i) step(i, Phase<-1>{}, Flag<false>{});
        step(nwhole, Phase<-1>{}, Flag<true>{});
    };
    if (wave < 4) run(Flag<false>{});
    else run(Flag<true>{});
    wait_vm<0>();

    if (kj < S) {
        __bf16 *krow = dk + hoff + static_cast<int64_t>(kj) * D;
        __bf16 *vrow = dv + hoff + static_cast<int64_t>(kj) * D;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
            for (int rb = 0; rb < 4; ++rb) {
                const f32x4 xk = {dkacc[dt][rb * 4 + 0] * scale, dkacc[dt][rb * 4 + 1] * scale,
                                  dkacc[dt][rb * 4 + 2] * scale, dkacc[dt][rb * 4 + 3] * scale};
                const f32x4 xv = {dvacc[dt][rb * 4 + 0], dvacc[dt][rb * 4 + 1], dvacc[dt][rb * 4 + 2],
                                  dvacc[dt][rb * 4 + 3]};
                store4(krow + dt * 32 + rb * 8 + g * 4, xk);
                store4(vrow + dt * 32 + rb * 8 + g * 4, xv);
            }
    }
}

// ---------------------------------------------------------------------------
// dQ from stored score gradients
// ---------------------------------------------------------------------------
// With a score-gradient workspace the key-parallel launch (kDs) also stores
// every dS tile it computes, as rounded to bf16 for its own dK product, and
// dQ becomes one product over that matrix, dQ^T = scale K^T dS^T: 2 S^2 d
// FLOP per head in place of the query-parallel kernel's 6 S^2 d, which
// recomputes the scores and dP.  The product reads the S x S bf16 dS once
// (128 FLOP per byte), so HBM bandwidth bounds it.
//
// Stored layout, per head: the tile of query block i (32 queries) and key
// tile kw (32 keys) at byte ((i / 8) nkw + kw) 16 KiB + (i % 8) 2 KiB,
// nkw = 8 ceil(S / 256), so the 8 query blocks of a workgroup below find the
// tiles of one 64-key step in 32 contiguous KiB.  A tile is two 1 KiB halves
// h, each row-major [32 keys][16 query positions] (32-byte rows); position
// 8 g + r of half h is query (rr / 4) 8 + 4 g + rr % 4 of the block,
// rr = 8 h + r (the key-parallel kernel's accumulator rows).  Keys past S
// hold exact zeros there; query blocks past S are never written.
//
// A workgroup has 8 waves; wave w owns query block 8 qtile + w and builds
// its dQ^T (128 x 32) in four 32 x 32 accumulators.  A step takes 64 keys:
// their K rows (16 KiB, shared, with the swizzle of attention_dq_dma_kernel)
// and each wave's two dS tiles (4 KiB, its own) go straight into LDS, two
// steps ahead through three buffers.  Both operands come out of LDS by
// ds_read_b64_tr_b16 at the same key rows, so each product pairs equal keys:
// A = K^T (head dimension = lane % 32), B = dS^T (query position = lane % 32).
namespace dsq {
constexpr int kWaves = 8;
constexpr int kKB = 64;                                       // keys per step
constexpr int kTiles = kKB / 32;                              // key tiles per step
constexpr int kKTileB = kKB * bdma::kRowB;                    // K rows of a step
constexpr int kDsWaveB = kTiles * bdma::kDsTileB;             // dS of a step, per wave
constexpr int kStageB = kKTileB + kWaves * kDsWaveB;          // 48 KiB
constexpr int kNB = 3;                                        // LDS buffers (32-key steps
                                                              // through 6 measured 1.5 % slower)
constexpr int kDist = kNB - 1;                                // steps a block is loaded ahead
constexpr int kKLoads = kKTileB / 1024 / kWaves;              // K loads per wave and step
constexpr int kDLoads = kDsWaveB / 1024;                      // dS loads per wave and step
static_assert(kKLoads >= 1 && kNB * kStageB <= 160 * 1024, "layout assumed below");
}  // namespace dsq

__global__ __launch_bounds__(64 * dsq::kWaves, dsq::kWaves / 4) void attention_dq_ds_kernel(
    const __bf16 *__restrict__ k, const char *__restrict__ dsg, __bf16 *__restrict__ dq, int S,
    int n_qtiles, int nkw, float scale) {
    using namespace dsq;
    using bdma::kRowB;
    using bdma::kDsTileB;
    using bdma::swz;
    constexpr int D = bdma::kD, DT = D / 32;
    __shared__ __attribute__((aligned(1024))) char lds[kNB * kStageB];

    const int logical = xcd_logical(blockIdx.x, gridDim.x);
    const int head = logical / n_qtiles;
    const int qtile = logical - head * n_qtiles;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int li = lane & 31;
    const int nqb = (S + kQB - 1) / kQB;
    const int qb = qtile * kWaves + wave;  // a block past S reads unwritten tiles, stores nothing
    const int64_t hoff = static_cast<int64_t>(head) * S * D;
    const __amdgpu_buffer_rsrc_t kr = head_rsrc(k + hoff, static_cast<int64_t>(S) * D * 2);
    const __amdgpu_buffer_rsrc_t dr =
        head_rsrc(dsg + (static_cast<int64_t>(head) * n_qtiles + qtile) * nkw * bdma::kDsGroupB,
                  static_cast<int64_t>(nkw) * bdma::kDsGroupB);

    // Lane offsets: K rows as in attention_dq_dma_kernel (row 4 (2 wave + i)
    // + lane / 16, chunk at position lane % 16); the wave's two dS tiles of a
    // step (key tiles 2 j and 2 j + 1 of its query block) copied as stored;
    // transposing reads of 16-key steps (lane t = lane % 16 of group
    // G = lane / 16, rows 4 (G / 2) + t / 4 and 8 more).
    unsigned src_k[kKLoads];
#pragma unroll
    for (int i = 0; i < kKLoads; ++i) {
        const unsigned r = 4 * (kKLoads * wave + i) + (lane >> 4), p = lane & 15;
        src_k[i] = r * kRowB + ((p ^ swz(r)) << 4);
    }
    unsigned tr_k[2][DT], tr_d[2];
    {
        const unsigned G = lane >> 4, t = lane & 15;
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
            const unsigned r = 4 * (G >> 1) + (t >> 2) + 8 * hh;
#pragma unroll
            for (int dt = 0; dt < DT; ++dt) {
                const unsigned col = dt * 32 + 16 * (G & 1) + 4 * (t & 3);
                tr_k[hh][dt] = r * kRowB + (((col >> 3) ^ swz(r)) << 4) + ((col & 7) << 1);
            }
            tr_d[hh] = (G & 1) * 1024 + r * 32 + (t & 3) * 8;
        }
    }
    const unsigned lds0 = static_cast<unsigned>(reinterpret_cast<uintptr_t>(lds));
    auto issue = [&](int j, int buf) {
        const unsigned st = lds0 + buf * kStageB;
#pragma unroll
        for (int i = 0; i < kKLoads; ++i)
            load_lds(st + (kKLoads * wave + i) * 1024, kr, src_k[i], j * kKTileB);
#pragma unroll
        for (int i = 0; i < kDLoads; ++i)
            load_lds(st + kKTileB + wave * kDsWaveB + i * 1024, dr,
                     (i >> 1) * bdma::kDsGroupB + wave * kDsTileB + (i & 1) * 1024 + lane * 16,
                     j * kTiles * bdma::kDsGroupB);
    };

    typedef __attribute__((address_space(3))) bf16x4 LdsV4;
    f32x16 acc[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) acc[dt] = f32x16{};
    auto step = [&](int buf) {
        const char *kb = lds + buf * kStageB;
        const char *db = kb + kKTileB + wave * kDsWaveB;
#pragma unroll
        for (int ks = 0; ks < kKB / 16; ++ks) {
            const char *d0 = db + (ks >> 1) * kDsTileB + (ks & 1) * 16 * 32;
            const bf16x4 blo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((LdsV4 *)(d0 + tr_d[0]));
            const bf16x4 bhi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((LdsV4 *)(d0 + tr_d[1]));
            const bf16x8 b = __builtin_shufflevector(blo, bhi, 0, 1, 2, 3, 4, 5, 6, 7);
            const char *k0 = kb + ks * 16 * kRowB;
#pragma unroll
            for (int dt = 0; dt < DT; ++dt) {
                const bf16x4 alo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((LdsV4 *)(k0 + tr_k[0][dt]));
                const bf16x4 ahi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((LdsV4 *)(k0 + tr_k[1][dt]));
                const bf16x8 a = __builtin_shufflevector(alo, ahi, 0, 1, 2, 3, 4, 5, 6, 7);
                acc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[dt], 0, 0, 0);
            }
        }
    };

    // Step j waits for block j (only the loads of blocks j + 1 .. j + kDist - 1
    // may be pending), then, past the barrier that ends every wave's step
    // j - 1, loads block j + kDist into that step's buffer.  Blocks past the
    // last read zeros (K) or tiles of keys past S (dS), and are not used.
    const int nblk = (S + kKB - 1) / kKB;
#pragma unroll
    for (int j = 0; j < kDist; ++j) issue(j, j);
    int buf = 0;
    for (int j = 0; j < nblk; ++j) {
        wait_vm<(kDist - 1) * (kKLoads + kDLoads)>();
        __syncthreads();
        issue(j + kDist, buf == 0 ? kNB - 1 : buf - 1);
        step(buf);
        buf = buf == kNB - 1 ? 0 : buf + 1;
    }
    wait_vm<0>();  // no load into LDS is pending when the workgroup ends

    // Lane l holds query position n = l % 32 of its block and, per
    // accumulator, head-dimension rows 8 rb + 4 g + 0..3.
    if (qb < nqb) {
        const int hh = li >> 4, r = li & 7, rr = 8 * hh + r;
        const int qi = qb * kQB + (rr >> 2) * 8 + ((li >> 3) & 1) * 4 + (rr & 3);
        const int g = lane >> 5;
        if (qi < S) {
            __bf16 *row = dq + hoff + static_cast<int64_t>(qi) * D;
#pragma unroll
            for (int dt = 0; dt < DT; ++dt)
#pragma unroll
                for (int rb = 0; rb < 4; ++rb) {
                    const f32x4 x = {acc[dt][rb * 4 + 0] * scale, acc[dt][rb * 4 + 1] * scale,
                                     acc[dt][rb * 4 + 2] * scale, acc[dt][rb * 4 + 3] * scale};
                    store4(row + dt * 32 + rb * 8 + g * 4, x);
                }
        }
    }
}

// D_i = <dO_i, O_i> for the path with stored score gradients (elsewhere the
// query-parallel kernel's prologue computes it), with that prologue's
// products in its order, so the key-parallel launch gets the same D either
// way.  A wave covers 32 queries; lane (li, g) sums half of query li's row.
__global__ __launch_bounds__(256) void attention_delta_kernel(const __bf16 *__restrict__ o,
                                                              const __bf16 *__restrict__ dout,
                                                              float *__restrict__ delta, int S,
                                                              int nqb, int n_waves) {
    constexpr int D = bdma::kD, KK = D / 16;
    const int wv = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (wv >= n_waves) return;
    const int head = wv / nqb, qb = wv - head * nqb;
    const int lane = threadIdx.x & 63, li = lane & 31, g = lane >> 5;
    const int qi = qb * kQB + li;
    const int64_t hoff = static_cast<int64_t>(head) * S * D;
    const int64_t hbytes = static_cast<int64_t>(S) * D * 2;
    const __amdgpu_buffer_rsrc_t or_ = head_rsrc(o + hoff, hbytes);
    const __amdgpu_buffer_rsrc_t dr = head_rsrc(dout + hoff, hbytes);
    float dpart = 0.f;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
        const unsigned off = static_cast<unsigned>(qi * D + kk * 16 + g * 8) * 2;
        const bf16x8 dv = __builtin_bit_cast(bf16x8, load8<__bf16>(dr, off));
        const bf16x8 ov = __builtin_bit_cast(bf16x8, load8<__bf16>(or_, off));
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const bf16x2 a = {dv[2 * e], dv[2 * e + 1]};
            const bf16x2 b = {ov[2 * e], ov[2 * e + 1]};
            dpart = __builtin_amdgcn_fdot2_f32_bf16(a, b, dpart, false);
        }
    }
    const float Di = swap_halves_sum(dpart);
    if (g == 0 && qi < S) delta[static_cast<int64_t>(head) * S + qi] = Di;
}

template <int D, typename T>
__global__ __launch_bounds__(KTile<D>::threads, KTile<D>::per_cu) void attention_dkdv_kernel(
    const T *__restrict__ q, const T *__restrict__ k, const T *__restrict__ v,
    const T *__restrict__ dout, const float *__restrict__ lse, const float *__restrict__ delta,
    T *__restrict__ dk, T *__restrict__ dv, int S, int n_ktiles, float c, float scale) {
    constexpr int KK = D / 16, DT = D / 32, NT = KTile<D>::threads;
    __shared__ __attribute__((aligned(16))) __bf16 vrows[KTile<D>::keys * QLds<D>::RS];
    __shared__ __attribute__((aligned(16))) __bf16 qbuf[2][QLds<D>::R];
    __shared__ __attribute__((aligned(16))) __bf16 dbuf[2][QLds<D>::R];
    __shared__ __attribute__((aligned(16))) __bf16 qtbuf[2][QLds<D>::TT];
    __shared__ __attribute__((aligned(16))) __bf16 dtbuf[2][QLds<D>::TT];
    __shared__ __attribute__((aligned(16))) float lbuf[2][kQB];
    __shared__ __attribute__((aligned(16))) float ebuf[2][kQB];

    const int logical = xcd_logical(blockIdx.x, gridDim.x);
    const int head = logical / n_ktiles;
    const int ktile = logical - head * n_ktiles;
    const int64_t hoff = static_cast<int64_t>(head) * S * D;
    const int64_t hbytes = static_cast<int64_t>(S) * D * sizeof(T);
    const __amdgpu_buffer_rsrc_t qr = head_rsrc(q + hoff, hbytes);
    const __amdgpu_buffer_rsrc_t kr = head_rsrc(k + hoff, hbytes);
    const __amdgpu_buffer_rsrc_t vr = head_rsrc(v + hoff, hbytes);
    const __amdgpu_buffer_rsrc_t dr = head_rsrc(dout + hoff, hbytes);
    const __amdgpu_buffer_rsrc_t lr = head_rsrc(lse + static_cast<int64_t>(head) * S, int64_t{S} * 4);
    const __amdgpu_buffer_rsrc_t er = head_rsrc(delta + static_cast<int64_t>(head) * S, int64_t{S} * 4);

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int li = lane & 31, g = lane >> 5;
    const int key0 = ktile * KTile<D>::keys;
    const int kj = key0 + wave * kQW + li;

    // K^T as B operands in registers: lane (g, key li) holds head dims
    // 16 kk + 8 g + [0, 8).  The workgroup's V rows go to LDS once.
    bf16x8 kreg[KK];
#pragma unroll
    for (int kk = 0; kk < KK; ++kk)
        kreg[kk] = __builtin_bit_cast(
            bf16x8, load8<T>(kr, static_cast<unsigned>(kj * D + kk * 16 + g * 8) * sizeof(T)));
    constexpr int CH = D / 8;
#pragma unroll
    for (int i = 0; i < KTile<D>::keys * CH / NT; ++i) {
        const int u = tid + i * NT, row = u / CH, ch = u % CH;
        *reinterpret_cast<u32x4 *>(vrows + row * QLds<D>::RS + ch * 8) =
            load8<T>(vr, static_cast<unsigned>((key0 + row) * D + ch * 8) * sizeof(T));
    }
    f32x16 dkacc[DT], dvacc[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
        dkacc[dt] = f32x16{};
        dvacc[dt] = f32x16{};
    }
    const int nqb = (S + kQB - 1) / kQB;
    const __bf16 *vmine = vrows + (wave * kQW + li) * QLds<D>::RS + g * 8;

    QStage<D, T> st;
    st.load(qr, dr, lr, er, 0, tid);
    st.store(qbuf[0], dbuf[0], qtbuf[0], dtbuf[0], lbuf[0], ebuf[0], tid);
    __syncthreads();

    for (int i = 0; i < nqb; ++i) {
        const int b = i & 1;
        if (i + 1 < nqb) st.load(qr, dr, lr, er, i + 1, tid);
        // S and dP: lane (g, key li), rows = queries 8 (r / 4) + 4 g + r % 4.
        f32x16 s = {}, dp = {};
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) {
            const int off = li * QLds<D>::RS + kk * 16 + g * 8;
            const bf16x8 qa = *reinterpret_cast<const bf16x8 *>(qbuf[b] + off);
            const bf16x8 da = *reinterpret_cast<const bf16x8 *>(dbuf[b] + off);
            const bf16x8 vb = *reinterpret_cast<const bf16x8 *>(vmine + kk * 16);
            s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qa, kreg[kk], s, 0, 0, 0);
            dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(da, vb, dp, 0, 0, 0);
        }
        const int qvalid = S - i * kQB;
        bf16x8 pb[2], dsb[2];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const f32x4 l0 = *reinterpret_cast<const f32x4 *>(&lbuf[b][h * 16 + g * 4]);
            const f32x4 l1 = *reinterpret_cast<const f32x4 *>(&lbuf[b][h * 16 + 8 + g * 4]);
            const f32x4 e0 = *reinterpret_cast<const f32x4 *>(&ebuf[b][h * 16 + g * 4]);
            const f32x4 e1 = *reinterpret_cast<const f32x4 *>(&ebuf[b][h * 16 + 8 + g * 4]);
            f32x8 p, ds;
#pragma unroll
            for (int r = 0; r < 8; ++r) {
                const int rr = h * 8 + r;
                const int qrow = (rr >> 2) * 8 + g * 4 + (rr & 3);
                const float Lr = (r < 4) ? l0[r & 3] : l1[r & 3];
                const float Dr = (r < 4) ? e0[r & 3] : e1[r & 3];
                p[r] = qrow < qvalid ? __builtin_amdgcn_exp2f(__builtin_fmaf(s[rr], c, -Lr)) : 0.f;
                ds[r] = p[r] * (dp[rr] - Dr);
            }
            pb[h] = __builtin_convertvector(p, bf16x8);
            dsb[h] = __builtin_convertvector(ds, bf16x8);
        }
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
            for (int qs = 0; qs < 2; ++qs) {
                const int off = (dt * 32 + li) * QLds<D>::TS + (qs * 2 + g) * 8;
                const bf16x8 da = *reinterpret_cast<const bf16x8 *>(dtbuf[b] + off);
                const bf16x8 qa = *reinterpret_cast<const bf16x8 *>(qtbuf[b] + off);
                dvacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(da, pb[qs], dvacc[dt], 0, 0, 0);
                dkacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qa, dsb[qs], dkacc[dt], 0, 0, 0);
            }
        if (i + 1 < nqb)
            st.store(qbuf[b ^ 1], dbuf[b ^ 1], qtbuf[b ^ 1], dtbuf[b ^ 1], lbuf[b ^ 1], ebuf[b ^ 1], tid);
        __syncthreads();
    }

    if (kj < S) {
        T *krow = dk + hoff + static_cast<int64_t>(kj) * D;
        T *vrow = dv + hoff + static_cast<int64_t>(kj) * D;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
            for (int rb = 0; rb < 4; ++rb) {
                const f32x4 xk = {dkacc[dt][rb * 4 + 0] * scale, dkacc[dt][rb * 4 + 1] * scale,
                                  dkacc[dt][rb * 4 + 2] * scale, dkacc[dt][rb * 4 + 3] * scale};
                const f32x4 xv = {dvacc[dt][rb * 4 + 0], dvacc[dt][rb * 4 + 1], dvacc[dt][rb * 4 + 2],
                                  dvacc[dt][rb * 4 + 3]};
                store4(krow + dt * 32 + rb * 8 + g * 4, xk);
                store4(vrow + dt * 32 + rb * 8 + g * 4, xv);
            }
    }
}

#ifndef HCMS_BWD_DQ_DMA
#define HCMS_BWD_DQ_DMA 1
#endif
// d = 128 with bf16 storage runs attention_dq_dma_kernel.
constexpr bool kDqDma = HCMS_BWD_DQ_DMA != 0;
#ifndef HCMS_BWD_DKDV_DMA
#define HCMS_BWD_DKDV_DMA 1
#endif
// d = 128 with bf16 storage runs attention_dkdv_dma_kernel.
constexpr bool kDkdvDma = HCMS_BWD_DKDV_DMA != 0;

// Bytes of stored score gradients per head (attention_dq_ds_kernel's
// layout): ceil(S / 256) groups of 8 query blocks x 8 ceil(S / 256) key
// tiles x 16 KiB.
int64_t ds_head_bytes(int S) {
    const int64_t n = (static_cast<int64_t>(S) + KTile<bdma::kD>::keys - 1) / KTile<bdma::kD>::keys;
    return n * 8 * n * bdma::kDsGroupB;
}

// The path with stored score gradients, for `group` heads at a time: D for
// every head, then per group the key-parallel launch (dK, dV, and dS into
// ds) and the dQ product over ds.
hipError_t launch_bwd_ds(const __bf16 *q, const __bf16 *k, const __bf16 *v, const __bf16 *o,
                         const __bf16 *dout, const float *lse, __bf16 *dq, __bf16 *dk, __bf16 *dv,
                         float *delta, char *ds, int S, int n_heads, int group, float c, float scale,
                         hipStream_t stream) {
    constexpr int D = bdma::kD;
    const int nqb = (S + kQB - 1) / kQB;
    const int64_t n_waves = static_cast<int64_t>(nqb) * n_heads;
    if ((n_waves + 3) / 4 > 0x7fffffff) return hipErrorInvalidValue;
    attention_delta_kernel<<<static_cast<unsigned>((n_waves + 3) / 4), 256, 0, stream>>>(
        o, dout, delta, S, nqb, static_cast<int>(n_waves));
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int n_tiles = (S + KTile<D>::keys - 1) / KTile<D>::keys;
    const int n_qt = (S + kQW * dsq::kWaves - 1) / (kQW * dsq::kWaves);
    for (int h0 = 0; h0 < n_heads; h0 += group) {
        const int hg = min(group, n_heads - h0);
        const int64_t off = static_cast<int64_t>(h0) * S * D, soff = static_cast<int64_t>(h0) * S;
        attention_dkdv_dma_kernel<true><<<static_cast<unsigned>(static_cast<int64_t>(n_tiles) * hg),
                                          KTile<D>::threads, 0, stream>>>(
            q + off, k + off, v + off, dout + off, lse + soff, delta + soff, dk + off, dv + off, ds, S,
            n_tiles, c, scale);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        attention_dq_ds_kernel<<<static_cast<unsigned>(static_cast<int64_t>(n_qt) * hg),
                                 64 * dsq::kWaves, 0, stream>>>(k + off, ds, dq + off, S, n_qt,
                                                                8 * n_tiles, scale);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    return hipSuccess;
}

template <int D, typename T>
hipError_t launch_bwd_typed(const void *q, const void *k, const void *v, const void *o,
                            const void *dout, const float *lse, void *dq, void *dk, void *dv,
                            float *delta, void *ds, int64_t ds_bytes, int S, int n_heads, float c,
                            float scale, hipStream_t stream) {
    const int n_qt = (S + kQW * QTile<D>::waves - 1) / (kQW * QTile<D>::waves);
    const int64_t qblocks = static_cast<int64_t>(n_qt) * n_heads;
    const int n_tiles = (S + KTile<D>::keys - 1) / KTile<D>::keys;
    const int64_t blocks = static_cast<int64_t>(n_tiles) * n_heads;
    if (blocks > 0x7fffffff || qblocks > 0x7fffffff) return hipErrorInvalidValue;
    if constexpr (D == bdma::kD && sizeof(T) == 2 && kDkdvDma) {
        const int64_t group = ds ? std::min<int64_t>(n_heads, ds_bytes / ds_head_bytes(S)) : 0;
        if (group >= 1)
            return launch_bwd_ds(static_cast<const __bf16 *>(q), static_cast<const __bf16 *>(k),
                                 static_cast<const __bf16 *>(v), static_cast<const __bf16 *>(o),
                                 static_cast<const __bf16 *>(dout), lse, static_cast<__bf16 *>(dq),
                                 static_cast<__bf16 *>(dk), static_cast<__bf16 *>(dv), delta,
                                 static_cast<char *>(ds), S, n_heads, static_cast<int>(group), c,
                                 scale, stream);
    }
    if constexpr (D == bdma::kD && sizeof(T) == 2 && kDqDma) {
        static_assert(QTile<D>::waves == bdma::kWaves, "the DMA kernel covers 256 queries in 8 waves");
        attention_dq_dma_kernel<<<static_cast<unsigned>(qblocks), QTile<D>::threads, 0, stream>>>(
            static_cast<const __bf16 *>(q), static_cast<const __bf16 *>(k), static_cast<const __bf16 *>(v),
            static_cast<const __bf16 *>(o), static_cast<const __bf16 *>(dout), lse,
            static_cast<__bf16 *>(dq), delta, S, n_qt, c, scale);
    } else {
        attention_dq_kernel<D, T><<<static_cast<unsigned>(qblocks), QTile<D>::threads, 0, stream>>>(
            static_cast<const T *>(q), static_cast<const T *>(k), static_cast<const T *>(v),
            static_cast<const T *>(o), static_cast<const T *>(dout), lse, static_cast<T *>(dq), delta, S,
            n_qt, c, scale);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if constexpr (D == bdma::kD && sizeof(T) == 2 && kDkdvDma) {
        static_assert(KTile<D>::waves == bdma::kWaves, "the DMA kernel covers 256 keys in 8 waves");
        attention_dkdv_dma_kernel<false><<<static_cast<unsigned>(blocks), KTile<D>::threads, 0, stream>>>(
            static_cast<const __bf16 *>(q), static_cast<const __bf16 *>(k), static_cast<const __bf16 *>(v),
            static_cast<const __bf16 *>(dout), lse, delta, static_cast<__bf16 *>(dk),
            static_cast<__bf16 *>(dv), nullptr, S, n_tiles, c, scale);
    } else {
        attention_dkdv_kernel<D, T><<<static_cast<unsigned>(blocks), KTile<D>::threads, 0, stream>>>(
            static_cast<const T *>(q), static_cast<const T *>(k), static_cast<const T *>(v),
            static_cast<const T *>(dout), lse, delta, static_cast<T *>(dk), static_cast<T *>(dv), S,
            n_tiles, c, scale);
    }
    return hipGetLastError();
}

}  // namespace

int64_t attention_backward_ds_head_bytes(int S, int d, int dtype) {
    if (S <= 0 || d != bdma::kD || dtype != 0 || !kDkdvDma) return 0;
    return ds_head_bytes(S);
}

hipError_t launch_attention_backward(const void *q, const void *k, const void *v, const void *o,
                                     const void *dout, const float *lse, void *dq, void *dk,
                                     void *dv, float *delta, void *ds, int64_t ds_bytes, int S,
                                     int n_heads, int d, float scale, int dtype,
                                     hipStream_t stream) {
    if (S == 0 || n_heads == 0) return hipSuccess;
    const float c = static_cast<float>(static_cast<double>(scale) * 1.4426950408889634);
    if (d == 128 && dtype == 0)
        return launch_bwd_typed<128, __bf16>(q, k, v, o, dout, lse, dq, dk, dv, delta, ds, ds_bytes, S,
                                             n_heads, c, scale, stream);
    if (d == 64 && dtype == 0)
        return launch_bwd_typed<64, __bf16>(q, k, v, o, dout, lse, dq, dk, dv, delta, ds, ds_bytes, S,
                                            n_heads, c, scale, stream);
    if (d == 128 && dtype == 1)
        return launch_bwd_typed<128, float>(q, k, v, o, dout, lse, dq, dk, dv, delta, ds, ds_bytes, S,
                                            n_heads, c, scale, stream);
    if (d == 64 && dtype == 1)
        return launch_bwd_typed<64, float>(q, k, v, o, dout, lse, dq, dk, dv, delta, ds, ds_bytes, S,
                                           n_heads, c, scale, stream);
    return hipErrorInvalidValue;
}

}  // namespace hcms
