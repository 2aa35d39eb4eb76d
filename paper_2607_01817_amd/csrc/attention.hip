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
//   * K and V blocks are staged in LDS by all threads (global -> registers ->
//     LDS), K one block ahead of V, each double-buffered;
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
//   * software pipeline: while the VALU computes the softmax of block j, the
//     MFMA unit already computes the scores of block j + 1 (no dependency
//     between the two), then O^T += V_j^T P_j^T.  The K operands of the score
//     MFMAs are read from LDS four MFMAs ahead; the loop is unrolled by two so
//     the score registers alternate roles instead of being copied;
//   * lazy rescaling: the running maximum used for the exponentials is only
//     raised when a block's maximum exceeds it by more than 2^8 in the exp2
//     domain.  Exponentials are then at most 2^8, which bf16 and fp32 hold
//     exactly in range; the final O / l is unchanged.  The decision is taken per
//     query (per lane); a wave only skips the multiply when no lane needs it,
//     and a lane that does not need it multiplies by exactly 1.  So the
//     arithmetic of every query depends only on its own row, never on which
//     other queries share the wave, tile, chunk or launch: any head chunking
//     gives bit-identical results;
//   * exp2 is the hardware v_exp_f32 on the argument s * c - m * c (one FMA),
//     c = scale * log2(e);
//   * P is rounded to bf16 (nearest-even, v_cvt_pk_bf16_f32) for the PV MFMA;
//     the row sum l adds exactly these rounded values (v_dot2c_f32_bf16 with a
//     (1, 1) pair), so the weights that multiply V are normalised exactly; all
//     accumulation (scores, O, l) is fp32;
//   * the grid is remapped so that the 8 XCDs each take a contiguous range of
//     (head, query tile) pairs, so concurrent workgroups of an XCD stream the
//     same K/V blocks through that XCD's L2.
//
// Tails: loads go through buffer resources bounded by the head's tensor, so
// query and key rows >= S read as zeros; such queries are not stored and such
// keys get score -inf in the last block only.
#include "attention_tiles.h"
#include "hcms_internal.h"

namespace hcms {
namespace {

using namespace tiles;

// S^T[mt] = K[mt] Q^T for the 64 keys of a block (2 tiles of 32 keys); the
// K operands are read from LDS four MFMAs ahead of their use.
template <int D>
__device__ inline void qk_mfma(f32x16 (&sacc)[2], const __bf16 *ks, const bf16x8 (&qreg)[D / 16],
                               int li, int g) {
    constexpr int N = 2 * (D / 16);
    constexpr int AHEAD = 4;
    bf16x8 a[N];
#pragma unroll
    for (int i = 0; i < AHEAD; ++i)
        a[i] = *reinterpret_cast<const bf16x8 *>(ks + ((i & 1) * 32 + li) * Lds<D>::KS + ((i >> 1) * 2 + g) * 8);
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) sacc[mt] = f32x16{};
#pragma unroll
    for (int i = 0; i < N; ++i) {
        if (i + AHEAD < N) {
            const int n = i + AHEAD;
            a[n] = *reinterpret_cast<const bf16x8 *>(ks + ((n & 1) * 32 + li) * Lds<D>::KS + ((n >> 1) * 2 + g) * 8);
        }
        sacc[i & 1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], qreg[i >> 1], sacc[i & 1], 0, 0, 0);
    }
}

// O^T[dt] += V^T[dt] P^T over the 64 keys of a block (4 k-steps of 16 keys).
template <int D>
__device__ inline void pv_mfma(f32x16 (&oacc)[D / 32], const bf16x8 (&pb)[4], const __bf16 *vts,
                               int li, int g) {
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt) {
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
            const bf16x8 a = *reinterpret_cast<const bf16x8 *>(vts + (dt * 32 + li) * Lds<D>::VS +
                                                                (ks * 2 + g) * 8);
            oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb[ks], oacc[dt], 0, 0, 0);
        }
    }
}

// Online softmax of one block for this lane's query: updates the running
// maximum m_used (lazily) and the row sum, returns the rescale factor of O and
// the bf16 B operands P^T.  With MASK, keys at or past `kvalid` inside the
// block get score -inf.
template <bool MASK>
__device__ inline float softmax_block(f32x16 (&sacc)[2], float &m_used, float &lsum,
                                      bf16x8 (&pb)[4], float c, int g, int kvalid, bool &raise) {
    if (MASK) {
#pragma unroll
        for (int mt = 0; mt < 2; ++mt)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int key = mt * 32 + (r >> 2) * 8 + g * 4 + (r & 3);
                if (key >= kvalid) sacc[mt][r] = -INFINITY;
            }
    }
    float mx = sacc[0][0];
#pragma unroll
    for (int r = 1; r < 16; ++r) mx = fmaxf(mx, sacc[0][r]);
#pragma unroll
    for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sacc[1][r]);
    {
        const auto r = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(unsigned, mx),
                                                        __builtin_bit_cast(unsigned, mx), false, false);
        mx = fmaxf(__builtin_bit_cast(float, static_cast<unsigned>(r[0])),
                   __builtin_bit_cast(float, static_cast<unsigned>(r[1])));
    }
    // First block: m_used = -inf, so the test is true and alpha = 0.
    raise = (mx - m_used) * c > kRescaleThreshold;
    const float alpha = raise ? __builtin_amdgcn_exp2f((m_used - mx) * c) : 1.0f;
    m_used = raise ? mx : m_used;
    lsum *= alpha;
    const float mc = m_used * c;
    const bf16x2 ones = {static_cast<__bf16>(1.0f), static_cast<__bf16>(1.0f)};
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            f32x8 p;
#pragma unroll
            for (int r = 0; r < 8; ++r)
                p[r] = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[mt][h * 8 + r], c, -mc));
            const bf16x8 pbf = __builtin_convertvector(p, bf16x8);
            pb[mt * 2 + h] = pbf;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const bf16x2 pair = {pbf[2 * r], pbf[2 * r + 1]};
                lsum = __builtin_amdgcn_fdot2_f32_bf16(pair, ones, lsum, false);
            }
        }
    }
    return alpha;
}

template <int D, typename T, int WAVES>
__global__ __launch_bounds__(64 * WAVES, 8 / WAVES) void attention_kernel(
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
    const int q0 = qtile * (kQW * WAVES) + wave * kQW;
    const int qi = q0 + li;     // this lane's query

    // Q^T as the B operand: lane (g, n) holds query n, head dims 16 kk + 8 g + [0, 8).
    // Rows past S read as zeros and are never stored.
    bf16x8 qreg[KK];
#pragma unroll
    for (int kk = 0; kk < KK; ++kk)
        qreg[kk] = __builtin_bit_cast(
            bf16x8, load8<T>(qr, static_cast<unsigned>(qi * D + kk * 16 + g * 8) * sizeof(T)));

    f32x16 oacc[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) oacc[dt] = f32x16{};
    float m_used = -INFINITY, lsum = 0.f;
    const int nkb = (S + kBC - 1) / kBC;

    // Prologue: K_0, V_0 and K_1 in LDS, scores of block 0.
    Stage<D, T, WAVES> st;
    st.load(kr, vr, 0, 0, tid);
    st.store_k(kbuf[0], tid);
    st.store_v(vbuf[0], tid);
    st.load(kr, vr, 1, 1, tid);
    st.store_k(kbuf[1], tid);
    __syncthreads();
    f32x16 scur[2];
    qk_mfma<D>(scur, kbuf[0], qreg, li, g);
    __syncthreads();  // kbuf[0] is overwritten in the first iteration

    // Steady state: block j's softmax and PV overlap block j + 1's scores.
    // LDS holds K_{j+1} in kbuf[(j+1)&1] and V_j in vbuf[j&1]; K_{j+2} and
    // V_{j+1} travel through registers and land in the buffers freed by K_j
    // and V_{j-1}.
    auto step = [&](int j, f32x16(&scur)[2], f32x16(&snext)[2]) {
        st.load(kr, vr, j + 2, j + 1, tid);
        qk_mfma<D>(snext, kbuf[(j + 1) & 1], qreg, li, g);
        bf16x8 pb[4];
        bool raise;
        const float alpha = softmax_block<false>(scur, m_used, lsum, pb, c, g, kBC, raise);
        if (__any(raise)) {
#pragma unroll
            for (int dt = 0; dt < DT; ++dt)
#pragma unroll
                for (int r = 0; r < 16; ++r) oacc[dt][r] *= alpha;
        }
        pv_mfma<D>(oacc, pb, vbuf[j & 1], li, g);
        st.store_k(kbuf[j & 1], tid);
        st.store_v(vbuf[(j + 1) & 1], tid);
        __syncthreads();
    };
    f32x16 salt[2];
    int j0 = 0;
    for (; j0 + 2 < nkb; j0 += 2) {
        step(j0, scur, salt);
        step(j0 + 1, salt, scur);
    }
    if (j0 + 1 < nkb) {
        step(j0, scur, salt);
        scur[0] = salt[0];
        scur[1] = salt[1];
    }

    // Last block: mask the keys past S.
    {
        const int j = nkb - 1;
        bf16x8 pb[4];
        bool raise;
        const float alpha = softmax_block<true>(scur, m_used, lsum, pb, c, g, S - j * kBC, raise);
        if (__any(raise)) {
#pragma unroll
            for (int dt = 0; dt < DT; ++dt)
#pragma unroll
                for (int r = 0; r < 16; ++r) oacc[dt][r] *= alpha;
        }
        pv_mfma<D>(oacc, pb, vbuf[j & 1], li, g);
    }

    // ---- O = O^T / l, rounded to the storage type ----
    float l;
    {
        const auto r = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(unsigned, lsum),
                                                        __builtin_bit_cast(unsigned, lsum), false, false);
        l = __builtin_bit_cast(float, static_cast<unsigned>(r[0])) +
            __builtin_bit_cast(float, static_cast<unsigned>(r[1]));
    }
    const float inv = 1.0f / l;
    // log2 of the softmax denominator of c * s: P_ij = exp2(c s_ij - L2_i)
    // (the statistic the backward pass recomputes P from).
    if (lse != nullptr && g == 0 && qi < S)
        lse[static_cast<int64_t>(head) * S + qi] = m_used * c + __builtin_amdgcn_logf(l);
    if (qi < S) {
        T *orow = oh + static_cast<int64_t>(qi) * D;
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

// Waves per workgroup: 8 for d = 128 (one workgroup per CU, two waves per
// SIMD), 4 for d = 64 (two workgroups per CU).
template <int D>
struct Waves {
    static constexpr int value = D == 128 ? 8 : 4;
};

template <int D, typename T>
hipError_t launch_typed(const void *q, const void *k, const void *v, void *o, float *lse, int S,
                        int n_heads, float c, hipStream_t stream) {
    constexpr int WAVES = Waves<D>::value;
    constexpr int BR = kQW * WAVES;
    const int n_qtiles = (S + BR - 1) / BR;
    const int64_t blocks = static_cast<int64_t>(n_qtiles) * n_heads;
    if (blocks > 0x7fffffff) return hipErrorInvalidValue;
    attention_kernel<D, T, WAVES><<<static_cast<unsigned>(blocks), 64 * WAVES, 0, stream>>>(
        static_cast<const T *>(q), static_cast<const T *>(k), static_cast<const T *>(v),
        static_cast<T *>(o), lse, S, n_qtiles, c);
    return hipGetLastError();
}

}  // namespace

int attention_queries_per_block(int d) { return kQW * (d == 128 ? Waves<128>::value : Waves<64>::value); }
int attention_blocks_per_cu(int d) { return 8 / (d == 128 ? Waves<128>::value : Waves<64>::value); }

hipError_t launch_attention(const void *q, const void *k, const void *v, void *o, float *lse, int S,
                            int n_heads, int d, float scale_log2e, int dtype, hipStream_t stream) {
    if (S == 0 || n_heads == 0) return hipSuccess;
    if (d == 128 && dtype == 0)
        return launch_typed<128, __bf16>(q, k, v, o, lse, S, n_heads, scale_log2e, stream);
    if (d == 64 && dtype == 0)
        return launch_typed<64, __bf16>(q, k, v, o, lse, S, n_heads, scale_log2e, stream);
    if (d == 128 && dtype == 1)
        return launch_typed<128, float>(q, k, v, o, lse, S, n_heads, scale_log2e, stream);
    if (d == 64 && dtype == 1)
        return launch_typed<64, float>(q, k, v, o, lse, S, n_heads, scale_log2e, stream);
    return hipErrorInvalidValue;
}

}  // namespace hcms
