// Projection GEMM for gfx950 (MI355X), bf16 MFMA with fp32 accumulation:
//   Y[m][n] = sum_k X[m][k] W[n][k]       X [M][K], W [N][K], Y [M][N]
// i.e. Y = X W^T with the weight stored [out][in].  It is the QKV projection
// before the split along heads and the output projection after the
// concatenation (Alg. 1, the main-stream steps around the chunk loop).
//
// Two epilogues.  The plain one stores Y.  The QKV one splits Y's columns
// n = z H d + h d + e into three [M][H][d] tensors (z = 0, 1, 2: queries, keys,
// values) and rotates the query and key pairs (e, e + 1), e even, by the rotary
// position embedding of token m on its latent grid (RoFormer's rotation; the
// pairs of a head vector form consecutive groups, each turning with one grid
// axis), in fp32 before the rounding to the storage type: the split along
// heads and the position embedding fused into the producing kernel.
//
// Work decomposition
//   * one workgroup = 8 waves = one 256 (m) x 256 (n) tile of Y; wave w owns
//     the 64 rows 64 (w >> 1) + [0, 64) and the 128 columns 128 (w & 1) +
//     [0, 128) of the tile, as 2 x 4 tiles of 32 x 32;
//   * both operands are K-contiguous rows, which is the operand layout of
//     v_mfma_f32_32x32x16_bf16 (8 consecutive k per lane), so neither needs a
//     transpose: the MFMA computes Y^T tiles, D[n][m] = sum_k W[n][k] X[m][k],
//     with W rows as the A operand and X rows as the B operand.  Each lane
//     then holds one row m and, per 32 x 32 tile, 4 runs of 4 consecutive
//     columns n: whole rotation pairs; bf16 output goes through LDS so that
//     it leaves as 16-byte stores covering whole row segments;
//   * k advances in blocks of 64: the 256 x 64 blocks of X and W are staged
//     global -> registers -> LDS (rows padded to 144 bytes, so 16 lanes
//     reading 16 rows hit 16 disjoint groups of 4 banks), double-buffered in
//     LDS, with two register sets so that each block's global loads are
//     issued two k-blocks before its MFMAs; every operand read from LDS feeds
//     2 (W) or 4 (X) MFMAs;
//   * tiles are ordered in groups of 8 row tiles (all column tiles of a group
//     before the next group); the grid holds one persistent workgroup per CU,
//     each round of the grid takes the next G tiles of that order, and the 8
//     XCDs each take a contiguous range of a round, so the 32 workgroups
//     resident on an XCD share 8 X panels and 4 W panels through its L2;
//   * a workgroup's tiles form one stream of k-blocks, so the next tile's
//     first blocks load during the current tile's last ones and its epilogue.
//
// Tails: rows past M or N are read through buffer resources bounded by the
// last row, so they read as zeros; rows past M and columns past N are not
// stored.  K must be a multiple of 64 and N of 8 (checked by the caller).
#include "attention_tiles.h"
#include "hcms_internal.h"

namespace hcms {
namespace {

using namespace tiles;

typedef float f32x2 __attribute__((ext_vector_type(2)));

constexpr int kBM = 256, kBN = 256, kBK = 64;
#ifndef HCMS_LINEAR_WAVES
#define HCMS_LINEAR_WAVES 8
#endif
constexpr int kWaves = HCMS_LINEAR_WAVES;    // 8: 64 x 128 per wave; 4: 128 x 128 per wave
constexpr int kThreads = 64 * kWaves;
constexpr int kWavesN = 2;                   // waves across the 256 columns
constexpr int kWavesM = kWaves / kWavesN;    // waves across the 256 rows
constexpr int kMT = kBM / kWavesM / 32;      // 32-row tiles per wave
constexpr int kNT = kBN / kWavesN / 32;      // 32-column tiles per wave
constexpr int kRow = kBK + 8;            // LDS row stride, elements (144 bytes)
constexpr int kTile = 256 * kRow;        // one staged 256 x 64 block, elements
constexpr int kGroupM = 8;               // row tiles per group of the tile order
constexpr int kPersistK = 1024;          // longest K run by persistent workgroups
constexpr int kPass = 256 * (kBK / 8) / kThreads;  // 16-byte chunks per thread per block
constexpr int kRowsPerPass = kThreads / 8;

// Arguments of the QKV epilogue: destinations, and the rotation (table NULL:
// no rotation).  table holds (cos, sin) pairs; axis a, coordinate c, pair i'
// of the axis's group is entry tab_off[a] + c * pairs[a] + i'.
template <typename T>
struct QkvOut {
    T *dst[3];
    const float *table;
    int H, d;
    RopeAxes ax;
};

// Resource over [base, base + min(bytes, 2^32 - 1)).
__device__ inline __amdgpu_buffer_rsrc_t span_rsrc(const void *base, int64_t bytes) {
    const int64_t n = bytes < 0 ? 0 : (bytes > 0xFFFFFFFFll ? 0xFFFFFFFFll : bytes);
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), 0,
                                             static_cast<int>(static_cast<uint32_t>(n)), 0x00020000);
}

// load8 with the byte offset split into a per-lane part and a scalar part
// (the buffer range check covers both).
template <typename T>
__device__ inline u32x4 load8s(__amdgpu_buffer_rsrc_t r, unsigned voff, unsigned soff);
template <>
__device__ inline u32x4 load8s<__bf16>(__amdgpu_buffer_rsrc_t r, unsigned voff, unsigned soff) {
    return __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0);
}
template <>
__device__ inline u32x4 load8s<float>(__amdgpu_buffer_rsrc_t r, unsigned voff, unsigned soff) {
    const f32x4 a = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
    const f32x4 b = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, voff + 16, soff, 0));
    const f32x8 x = {a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
    return __builtin_bit_cast(u32x4, __builtin_convertvector(x, bf16x8));
}

// Global -> register staging of the 256 x 64 blocks of X and W at column k0.
// Thread tid moves chunk tid % 8 (8 elements) of rows tid / 8 + kRowsPerPass p:
// a per-lane offset fixed for the whole launch (row and chunk, the same for X
// and W) plus the block's column in the scalar offset, so the k-loop computes
// no addresses (temporaries written there made the compiler wait for the
// loads in flight on every step).
template <typename T>
__device__ inline void stage_offsets(unsigned (&voff)[kPass], unsigned row_bytes, int tid) {
#pragma unroll
    for (int p = 0; p < kPass; ++p)
        voff[p] = static_cast<unsigned>(tid / 8 + kRowsPerPass * p) * row_bytes + (tid & 7) * 8 * sizeof(T);
}
template <typename T>
struct Stager {
    u32x4 xr[kPass], wr[kPass];
    __device__ void load(__amdgpu_buffer_rsrc_t xs, __amdgpu_buffer_rsrc_t ws,
                         const unsigned (&voff)[kPass], int k0) {
        const unsigned soff = static_cast<unsigned>(k0) * sizeof(T);
#pragma unroll
        for (int p = 0; p < kPass; ++p) {
            xr[p] = load8s<T>(xs, voff[p], soff);
            wr[p] = load8s<T>(ws, voff[p], soff);
        }
    }
    __device__ void store(__bf16 *xt, __bf16 *wt, int tid) const {
#pragma unroll
        for (int p = 0; p < kPass; ++p) {
            const int e = (tid / 8 + kRowsPerPass * p) * kRow + (tid & 7) * 8;
            *reinterpret_cast<u32x4 *>(xt + e) = xr[p];
            *reinterpret_cast<u32x4 *>(wt + e) = wr[p];
        }
    }
};

// Scheduling hint for one k-block: the operand reads of k-step ks + 1 and,
// when the LDS stores of the next block follow the MFMAs, those stores run
// between the MFMAs of k-step ks.
template <bool kStores>
__device__ inline void interleave_k_block() {
    constexpr int kReads = kNT + kMT;            // operand reads per k-step
    constexpr int kMfma = kNT * kMT;             // MFMAs per k-step
    constexpr int kWrites = 2 * kPass;           // LDS stores per k-block
    constexpr int kSteps = kBK / 16;
    __builtin_amdgcn_sched_group_barrier(0x100, kReads, 0);  // DS read, k-step 0
#pragma unroll
    for (int ks = 0; ks < kSteps; ++ks) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            __builtin_amdgcn_sched_group_barrier(0x008, kMfma / 2, 0);           // MFMA
            if (ks + 1 < kSteps) __builtin_amdgcn_sched_group_barrier(0x100, kReads / 2, 0);
            if constexpr (kStores)
                __builtin_amdgcn_sched_group_barrier(0x200, kWrites / (2 * kSteps), 0);  // DS write
        }
    }
}

template <typename T, bool QKV>
__global__ __launch_bounds__(kThreads, 1) void linear_kernel(const T *__restrict__ x,
                                                             const T *__restrict__ w,
                                                             T *__restrict__ y, int M, int N, int K,
                                                             int tiles_m, int tiles_n, QkvOut<T> qo) {
    __shared__ __attribute__((aligned(16))) __bf16 xt[2][kTile];
    __shared__ __attribute__((aligned(16))) __bf16 wt[2][kTile];

    // Persistent tiles: the grid has at most one workgroup per CU, and round r
    // of workgroup b computes tile r G + slot(b) of the grouped order (G = the
    // grid size).  Workgroup b runs on XCD b % 8, and slot(b) gives each XCD a
    // contiguous range of every round, so the workgroups resident on an XCD
    // share a few X and W panels through its L2.
    const int G = gridDim.x, b = blockIdx.x;
    const int xcd = b & 7, per = G >> 3, rem = G & 7;
    const int slot = xcd * per + min(xcd, rem) + (b >> 3);
    const int n_tiles = tiles_m * tiles_n;
    if (slot >= n_tiles) return;
    const int n_mine = (n_tiles - 1 - slot) / G + 1;
    auto origin = [&](int r, int &m0, int &n0) {
        const int L = r * G + slot;
        const int group = L / (kGroupM * tiles_n);
        const int first_m = group * kGroupM;
        const int gm = min(tiles_m - first_m, kGroupM);
        const int in_group = L - group * kGroupM * tiles_n;
        m0 = (first_m + in_group % gm) * kBM;
        n0 = (in_group / gm) * kBN;
    };

    const unsigned row_bytes = static_cast<unsigned>(K) * sizeof(T);
    auto x_rsrc = [&](int m0) {
        return span_rsrc(x + static_cast<int64_t>(m0) * K, static_cast<int64_t>(M - m0) * row_bytes);
    };
    auto w_rsrc = [&](int n0) {
        return span_rsrc(w + static_cast<int64_t>(n0) * K, static_cast<int64_t>(N - n0) * row_bytes);
    };

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int li = lane & 31, g = lane >> 5;
    const int wm = wave / kWavesN, wn = wave % kWavesN;

    f32x16 acc[kNT][kMT];  // [n tile][m tile]
#pragma unroll
    for (int nt = 0; nt < kNT; ++nt)
#pragma unroll
        for (int mt = 0; mt < kMT; ++mt) acc[nt][mt] = f32x16{};

    // ---- Epilogue: Y of the tile at (m0, n0) from the D^T accumulators,
    // rounded to T.  Lane (li, g) holds token m = ... + li and, per 32 x 32
    // tile, runs of 4 consecutive features n = ... + 8 rb + 4 g.
    // Per grid axis, the table entry of pair 0 of the axis at token m's
    // coordinate (QKV epilogue with a rotation only).
    auto table_rows = [&](int m, int (&tab_row)[kRopeMaxAxes]) {
        int rest = m;
        for (int a = qo.ax.n_axes - 1; a >= 0; --a) {
            const int cc = rest % qo.ax.grid[a];
            rest /= qo.ax.grid[a];
            tab_row[a] = qo.ax.tab_off[a] + cc * qo.ax.pairs[a] - qo.ax.pair_start[a];
        }
    };
    // Features n .. n + 3 (n < N) of a token whose table rows are tab_row,
    // rotated in place when they are query or key features.
    auto rotate = [&](f32x4 &v, int n, const int (&tab_row)[kRopeMaxAxes]) {
        const int hd = qo.H * qo.d;
        const int z = n / hd, e = (n - z * hd) % qo.d;  // e a multiple of 4: pairs e/2, e/2 + 1
        if (z >= 2) return;
#pragma unroll
        for (int q2 = 0; q2 < 2; ++q2) {
            const int p = e / 2 + q2;
            int a = 0;
            while (a + 1 < qo.ax.n_axes && p >= qo.ax.pair_start[a + 1]) ++a;
            const f32x2 cs = *reinterpret_cast<const f32x2 *>(qo.table + 2 * (tab_row[a] + p));
            const float x0 = v[2 * q2], x1 = v[2 * q2 + 1];
            v[2 * q2] = __builtin_fmaf(x0, cs[0], -(x1 * cs[1]));
            v[2 * q2 + 1] = __builtin_fmaf(x0, cs[1], x1 * cs[0]);
        }
    };
    // Where feature n of token m goes: Y, or the split q, k, v (8 consecutive
    // features never straddle two of them: N and H d are multiples of 8).
    auto dest = [&](int m, int n) -> T * {
        if constexpr (QKV) {
            const int hd = qo.H * qo.d;
            const int z = n / hd;
            return qo.dst[z] + static_cast<int64_t>(m) * hd + (n - z * hd);
        } else {
            return y + static_cast<int64_t>(m) * N + n;
        }
    };
    // Direct stores of each lane's runs: fp32 storage (16 bytes a run) and the
    // QKV epilogue, whose K = D reductions make its one tile per workgroup
    // long, so that its stores cost little (staging them, with the rotation,
    // ran 5 % slower).
    auto store_direct = [&](int m0, int n0) {
#pragma unroll
        for (int mt = 0; mt < kMT; ++mt) {
            const int m = m0 + wm * kMT * 32 + mt * 32 + li;
            if (m >= M) continue;
            int tab_row[kRopeMaxAxes] = {};
            if (QKV && qo.table != nullptr) table_rows(m, tab_row);
#pragma unroll
            for (int nt = 0; nt < kNT; ++nt)
#pragma unroll
                for (int rb = 0; rb < 4; ++rb) {
                    const int n = n0 + wn * kNT * 32 + nt * 32 + rb * 8 + g * 4;
                    if (n >= N) continue;
                    f32x4 v = {acc[nt][mt][rb * 4 + 0], acc[nt][mt][rb * 4 + 1],
                               acc[nt][mt][rb * 4 + 2], acc[nt][mt][rb * 4 + 3]};
                    if (QKV && qo.table != nullptr) rotate(v, n, tab_row);
                    store4(dest(m, n), v);
                }
        }
    };
    // Plain epilogue, bf16 storage: runs of 8 bytes, 32 rows apart, coalesce
    // badly (the output projection, K = H d = 640, lost a fifth of its time
    // to them), so each wave
    // transposes its 64 x 128 part through LDS, 32 tokens at a time, in a
    // private 32 x 264-byte region of the buffer the tile's last k-block left
    // free, and stores whole 256-byte row segments, 16 bytes per lane.
    constexpr int kStRow = 128 * 2 + 8;  // bytes per staged row, 8 of them padding
    static_assert(4 * 32 * kStRow <= kTile * 2 && kNT * 32 == 128, "staging fits one buffer");
    auto store_staged = [&](int m0, int n0, char *stage) {
#pragma unroll
        for (int mt = 0; mt < kMT; ++mt) {
#pragma unroll
            for (int nt = 0; nt < kNT; ++nt)
#pragma unroll
                for (int rb = 0; rb < 4; ++rb) {
                    const int c = nt * 32 + rb * 8 + g * 4;
                    const f32x4 v = {acc[nt][mt][rb * 4 + 0], acc[nt][mt][rb * 4 + 1],
                                     acc[nt][mt][rb * 4 + 2], acc[nt][mt][rb * 4 + 3]};
                    *reinterpret_cast<bf16x4 *>(stage + li * kStRow + c * 2) =
                        __builtin_convertvector(v, bf16x4);
                }
            const int c = (lane & 15) * 8;  // the lane's 8 features of a staged row
            const int n = n0 + wn * kNT * 32 + c;
#pragma unroll
            for (int q0 = 0; q0 < 8; q0 += 4) {
                u32x4 o[4];
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    o[q] = *reinterpret_cast<const u32x4 *>(stage + ((q0 + q) * 4 + (lane >> 4)) * kStRow + c * 2);
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int mm = m0 + wm * kMT * 32 + mt * 32 + (q0 + q) * 4 + (lane >> 4);
                    if (mm < M && n < N)
                        *reinterpret_cast<u32x4 *>(y + static_cast<int64_t>(mm) * N + n) = o[q];
                }
            }
        }
    };

    // The k-blocks of the workgroup's tiles form one stream: NSETS register
    // sets carry its blocks from global memory to LDS.  With two (bf16
    // storage), stream block s is loaded into set s & 1 during block s - 2 and
    // stored to LDS buffer s & 1 after block s - 1's MFMAs, so each load has
    // two k-blocks to arrive, also across a tile boundary (the next tile's
    // first blocks load during the current tile's last ones and its
    // epilogue); with one (fp32 storage, whose loads need twice the
    // registers) it is loaded during block s - 1.  The loads of blocks past
    // the stream's end read within the last tile's resources (the next row's
    // data or zeros) and the last store goes to a buffer nobody reads.
    constexpr int NSETS = sizeof(T) == 2 ? 2 : 1;
    const int nkb = K / kBK;
    int ld_r = 0, ld_kb = 0;  // tile round and k-block of the next load
    int lm0, ln0;
    origin(0, lm0, ln0);
    __amdgpu_buffer_rsrc_t lxs = x_rsrc(lm0), lws = w_rsrc(ln0);
    unsigned voff[kPass];
    stage_offsets<T>(voff, row_bytes, tid);
    auto load_next = [&](Stager<T> &st) {
        st.load(lxs, lws, voff, ld_kb * kBK);
        if (++ld_kb == nkb && ld_r + 1 < n_mine) {
            ld_kb = 0;
            ++ld_r;
            origin(ld_r, lm0, ln0);
            lxs = x_rsrc(lm0);
            lws = w_rsrc(ln0);
        }
    };

    Stager<T> st[NSETS];
    load_next(st[0]);
    st[0].store(xt[0], wt[0], tid);
    if (NSETS == 2) load_next(st[1 % NSETS]);
    __syncthreads();
    // With two register sets the next block's LDS stores go first, right
    // after the barrier that ended every wave's reads of that buffer (its
    // loads were issued a step earlier), then the MFMAs; the plain epilogue's
    // k-loop keeps hints for the operand reads, the QKV one (one long tile per
    // workgroup) leaves the order to the compiler, each measured fastest
    // (about 2 % over the stores between the MFMAs).  With one set the block
    // is loaded during this step and stored after the MFMAs.
    constexpr bool kStoreFirst = NSETS == 2;
    auto step = [&](int s, Stager<T> &ld, const Stager<T> &sto) {
        load_next(ld);
        if constexpr (kStoreFirst) sto.store(xt[(s + 1) & 1], wt[(s + 1) & 1], tid);
        const __bf16 *xa = xt[s & 1] + (wm * kMT * 32 + li) * kRow + g * 8;
        const __bf16 *wa = wt[s & 1] + (wn * kNT * 32 + li) * kRow + g * 8;
#pragma unroll
        for (int ks = 0; ks < kBK / 16; ++ks) {
            bf16x8 a[kNT], bx[kMT];
#pragma unroll
            for (int nt = 0; nt < kNT; ++nt)
                a[nt] = *reinterpret_cast<const bf16x8 *>(wa + nt * 32 * kRow + ks * 16);
#pragma unroll
            for (int mt = 0; mt < kMT; ++mt)
                bx[mt] = *reinterpret_cast<const bf16x8 *>(xa + mt * 32 * kRow + ks * 16);
#pragma unroll
            for (int nt = 0; nt < kNT; ++nt)
#pragma unroll
                for (int mt = 0; mt < kMT; ++mt)
                    acc[nt][mt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[nt], bx[mt], acc[nt][mt],
                                                                          0, 0, 0);
        }
        if constexpr (!kStoreFirst) {
            sto.store(xt[(s + 1) & 1], wt[(s + 1) & 1], tid);
            interleave_k_block<true>();
        } else if constexpr (!QKV) {
            interleave_k_block<false>();
        }
        __syncthreads();
    };
    // The k-blocks of one tile run in a loop of two steps without branches
    // (register set and LDS buffer follow the stream index's parity), so the
    // compiler's waits for the staged loads stay two blocks deep; the
    // epilogue sits between tiles.
    int s = 0;
    for (int r = 0; r < n_mine; ++r) {
        int kb = 0;
        if (s & 1) {
            step(s, st[1 % NSETS], st[0]);
            ++s;
            ++kb;
        }
        for (; kb + 1 < nkb; kb += 2, s += 2) {
            step(s, st[0], st[1 % NSETS]);
            step(s + 1, st[1 % NSETS], st[0]);
        }
        if (kb < nkb) {
            step(s, st[0], st[1 % NSETS]);
            ++s;
        }
        int m0, n0;
        origin(r, m0, n0);
        if constexpr (sizeof(T) == 2 && !QKV) {
            // The buffer of the tile's last block (stream block s - 1) is free
            // until the next step stores block s + 1 there, after a barrier.
            char *base = reinterpret_cast<char *>(wave < 4 ? xt[(s - 1) & 1] : wt[(s - 1) & 1]);
            store_staged(m0, n0, base + (wave & 3) * 32 * kStRow);
            __syncthreads();
        } else {
            store_direct(m0, n0);
        }
#pragma unroll
        for (int nt = 0; nt < kNT; ++nt)
#pragma unroll
            for (int mt = 0; mt < kMT; ++mt) acc[nt][mt] = f32x16{};
    }
}

// Rotation table: entry e of axis a (tab_off[a] <= e < tab_off[a] + grid[a] *
// pairs[a]) is (cos, sin) of c * base^(-i' / pairs[a]), c = (e - tab_off[a]) /
// pairs[a], i' = (e - tab_off[a]) % pairs[a]; computed in fp64, rounded to fp32.
__global__ __launch_bounds__(256) void rope_table_kernel(float *table, RopeAxes ax, double base,
                                                         int total) {
    const int e = blockIdx.x * 256 + threadIdx.x;
    if (e >= total) return;
    int a = 0;
    while (a + 1 < ax.n_axes && e >= ax.tab_off[a + 1]) ++a;
    const int rel = e - ax.tab_off[a];
    const int c = rel / ax.pairs[a], ip = rel % ax.pairs[a];
    const double ang = static_cast<double>(c) *
                       pow(base, -static_cast<double>(ip) / static_cast<double>(ax.pairs[a]));
    table[2 * e] = static_cast<float>(cos(ang));
    table[2 * e + 1] = static_cast<float>(sin(ang));
}

template <typename T, bool QKV>
hipError_t launch_typed(const void *x, const void *w, void *y, int M, int N, int K,
                        const QkvOut<T> &qo, hipStream_t stream) {
    const int tiles_m = (M + kBM - 1) / kBM, tiles_n = (N + kBN - 1) / kBN;
    const int64_t tiles = static_cast<int64_t>(tiles_m) * tiles_n;
    if (tiles > 0x7fffffff) return hipErrorInvalidValue;
    int device = 0, n_cu = 0;
    hipError_t e = hipGetDevice(&device);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, device);
    if (e != hipSuccess) return e;
    // Short reductions (K of at most kPersistK) run one persistent workgroup
    // per CU, whose tiles stream without a pipeline refill; longer ones one
    // workgroup per tile.
    const int64_t blocks = K <= kPersistK && tiles > n_cu ? n_cu : tiles;
    if (blocks < 1) return hipErrorInvalidValue;
    linear_kernel<T, QKV><<<static_cast<unsigned>(blocks), kThreads, 0, stream>>>(
        static_cast<const T *>(x), static_cast<const T *>(w), static_cast<T *>(y), M, N, K, tiles_m,
        tiles_n, qo);
    return hipGetLastError();
}

template <typename T>
QkvOut<T> qkv_out(void *q, void *k, void *v, const float *table, const RopeAxes &ax, int H, int d) {
    QkvOut<T> o{};
    o.dst[0] = static_cast<T *>(q);
    o.dst[1] = static_cast<T *>(k);
    o.dst[2] = static_cast<T *>(v);
    o.table = table;
    o.H = H;
    o.d = d;
    o.ax = ax;
    return o;
}

}  // namespace

int linear_k_multiple() { return kBK; }

hipError_t launch_linear(const void *x, const void *w, void *y, int M, int N, int K, int dtype,
                         hipStream_t stream) {
    if (M == 0 || N == 0) return hipSuccess;
    if (dtype == 0) return launch_typed<__bf16, false>(x, w, y, M, N, K, QkvOut<__bf16>{}, stream);
    if (dtype == 1) return launch_typed<float, false>(x, w, y, M, N, K, QkvOut<float>{}, stream);
    return hipErrorInvalidValue;
}

hipError_t launch_qkv_projection(const void *x, const void *w, void *q, void *k, void *v,
                                 const float *table, const RopeAxes &ax, int S, int D, int H, int d,
                                 int dtype, hipStream_t stream) {
    if (S == 0) return hipSuccess;
    const int N = 3 * H * d;
    if (dtype == 0)
        return launch_typed<__bf16, true>(x, w, nullptr, S, N, D,
                                          qkv_out<__bf16>(q, k, v, table, ax, H, d), stream);
    if (dtype == 1)
        return launch_typed<float, true>(x, w, nullptr, S, N, D,
                                         qkv_out<float>(q, k, v, table, ax, H, d), stream);
    return hipErrorInvalidValue;
}

hipError_t launch_rope_table(float *table, const RopeAxes &ax, double base, hipStream_t stream) {
    const int last = ax.n_axes - 1;
    const int total = ax.tab_off[last] + ax.grid[last] * ax.pairs[last];
    if (total == 0) return hipSuccess;
    rope_table_kernel<<<(total + 255) / 256, 256, 0, stream>>>(table, ax, base, total);
    return hipGetLastError();
}

}  // namespace hcms
