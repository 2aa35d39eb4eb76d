// Tile helpers shared by the forward and backward attention kernels (gfx950,
// bf16 MFMA 32x32x16).  See attention.hip for the layouts they serve.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace hcms {
namespace tiles {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

inline constexpr int kQW = 32;              // queries per wave (one 32-wide MFMA tile)
inline constexpr int kBC = 64;              // keys per block

// Buffer resource over one head's [S][D] tensor: loads past its end return 0,
// which is how the query and key tails are read without branches.
__device__ inline __amdgpu_buffer_rsrc_t head_rsrc(const void *base, int64_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), 0,
                                             static_cast<int>(bytes), 0x00020000);
}

// 8 consecutive elements at byte offset `off` as bf16 (fp32 storage is rounded
// to nearest-even), returned as raw 32-bit words.
template <typename T>
__device__ inline u32x4 load8(__amdgpu_buffer_rsrc_t r, unsigned off);

template <>
__device__ inline u32x4 load8<__bf16>(__amdgpu_buffer_rsrc_t r, unsigned off) {
    return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
}

// The two loads are reinterpreted as whole float vectors before the
// conversion: converting lane-wise bit casts of u32 vector elements to bf16
// miscompiles with this toolchain (elements are dropped).
template <>
__device__ inline u32x4 load8<float>(__amdgpu_buffer_rsrc_t r, unsigned off) {
    const f32x4 a = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
    const f32x4 b = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off + 16, 0, 0));
    const f32x8 x = {a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
    return __builtin_bit_cast(u32x4, __builtin_convertvector(x, bf16x8));
}

__device__ inline void store4(__bf16 *p, f32x4 x) {
    *reinterpret_cast<bf16x4 *>(p) = __builtin_convertvector(x, bf16x4);
}
__device__ inline void store4(float *p, f32x4 x) { *reinterpret_cast<f32x4 *>(p) = x; }

// One wave's 1 KiB of a block loaded straight into LDS (gfx950
// buffer_load_dwordx4 ... lds): lane l's 16 bytes at `voff` plus the block
// offset `soff` (the buffer range check covers both; out-of-range lanes write
// zeros) land at LDS byte lds_addr + 16 l.  Inline asm: with the intrinsic the
// compiler waits for every such load before any later LDS read, so the
// kernels count these loads themselves (wait_vm).  M0 is written here and read
// by nothing else in the kernels.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ inline void load_lds(unsigned lds_addr, __amdgpu_buffer_rsrc_t r, unsigned voff, unsigned soff) {
    asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds"
                 :: "s"(lds_addr), "v"(voff), "s"(r), "s"(soff) : "memory", "m0");
}
// The same with 4 bytes per lane (lane l at LDS byte lds_addr + 4 l).
__device__ inline void load_lds_b32(unsigned lds_addr, __amdgpu_buffer_rsrc_t r, unsigned voff, unsigned soff) {
    asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dword %1, %2, %3 offen lds"
                 :: "s"(lds_addr), "v"(voff), "s"(r), "s"(soff) : "memory", "m0");
}
#pragma clang diagnostic pop

// Wait until at most N of this wave's vector memory instructions are pending.
template <int N>
__device__ inline void wait_vm() {
    asm volatile("s_waitcnt vmcnt(%0)" :: "n"(N) : "memory");
}

// Wait for every vector memory load of this wave (s_waitcnt vmcnt(0),
// expcnt and lgkmcnt left open: simm16 0x0F70), issued as the compiler's own
// instruction.  The compiler places waits for register loads by counting the
// loads it can see; it does not see the loads into LDS above.  After a
// prologue that fills registers by plain loads, its first use of those
// registers inside a key loop would otherwise get a vmcnt wait on every
// iteration, which in hardware also waits for the LDS loads in flight.  This
// wait, which the compiler does see, ends those loads before the loop.
__device__ inline void drain_vm_loads() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// Position of key `k` (0..63) inside a transposed V row: bits 2 and 3 swapped.
__device__ inline int vt_pos(int k) { return (k & ~12) | ((k & 4) << 1) | ((k & 8) >> 1); }

// LDS tiles are padded by 16 bytes per row: K is [kBC][D + 8] and V^T is
// [D][kBC + 8] (bf16 elements).  With rows of 272 (K, D = 128) or 144 bytes the
// 16-byte operand reads of 16 consecutive rows land on 16 disjoint groups of 4
// banks, and every LDS address is one per-lane base plus an immediate offset.
template <int D>
struct Lds {
    static constexpr int KS = D + 8;      // K row stride (elements)
    static constexpr int VS = kBC + 8;    // V^T row stride (elements)
    static constexpr int KT = kBC * KS;   // K tile size (elements)
    static constexpr int VT = D * VS;     // V^T tile size (elements)
};

// Global -> register -> LDS staging of one K block and one V block.
template <int D, typename T, int WAVES>
struct Stage {
    static constexpr int kThreads = 64 * WAVES;
    static constexpr int CH = D / 8;                        // 16-byte bf16 chunks per row
    static constexpr unsigned ROWB = D * sizeof(T);          // bytes per stored row
    static constexpr unsigned CHB = 8 * sizeof(T);           // bytes per stored chunk
    static constexpr int KPASS = kBC * CH / kThreads;       // K chunks per thread
    static constexpr int VTASK = (kBC / 2) * CH / kThreads; // V (key pair, chunk) tasks
    static_assert(KPASS >= 1 && VTASK >= 1, "tile too small for the workgroup");

    u32x4 kreg[KPASS];
    u32x4 vreg[VTASK][2];

    // K: thread -> (row, chunk), CH threads cover a row.
    __device__ static int k_row(int p, int tid) { return p * (kThreads / CH) + tid / CH; }
    __device__ static int k_chunk(int tid) { return tid % CH; }
    // V: a wave covers 16 key pairs x 4 chunks; key pair kp = keys 2kp, 2kp + 1.
    __device__ static int v_pair(int task) { return ((task >> 6) & 1) * 16 + (task & 15); }
    __device__ static int v_chunk(int task) { return (task >> 7) * 4 + ((task >> 4) & 3); }

    // Offsets stay below 2^32: a head is at most 2^31 - 1 bytes and blocks past
    // its end are at most three blocks away.
    __device__ void load(__amdgpu_buffer_rsrc_t kr, __amdgpu_buffer_rsrc_t vr, int kblk, int vblk,
                         int tid) {
        const unsigned key0 = static_cast<unsigned>(kblk) * kBC;
#pragma unroll
        for (int p = 0; p < KPASS; ++p)
            kreg[p] = load8<T>(kr, (key0 + k_row(p, tid)) * ROWB + k_chunk(tid) * CHB);
        const unsigned vkey0 = static_cast<unsigned>(vblk) * kBC;
#pragma unroll
        for (int i = 0; i < VTASK; ++i) {
            const int task = tid + i * kThreads;
            const unsigned off = (vkey0 + 2 * v_pair(task)) * ROWB + v_chunk(task) * CHB;
            vreg[i][0] = load8<T>(vr, off);
            vreg[i][1] = load8<T>(vr, off + ROWB);
        }
    }

    __device__ void store_k(__bf16 *ks, int tid) const {
#pragma unroll
        for (int p = 0; p < KPASS; ++p)
            *reinterpret_cast<u32x4 *>(ks + k_row(p, tid) * Lds<D>::KS + k_chunk(tid) * 8) = kreg[p];
    }

    // The key pairs of the V pattern stored row-major ([kBC][D + 8]), for a
    // tensor that is needed in both layouts.
    __device__ void store_v_rows(__bf16 *ks, int tid) const {
#pragma unroll
        for (int i = 0; i < VTASK; ++i) {
            const int task = tid + i * kThreads;
            __bf16 *dst = ks + 2 * v_pair(task) * Lds<D>::KS + v_chunk(task) * 8;
            *reinterpret_cast<u32x4 *>(dst) = vreg[i][0];
            *reinterpret_cast<u32x4 *>(dst + Lds<D>::KS) = vreg[i][1];
        }
    }

    __device__ void store_v(__bf16 *vts, int tid) const {
#pragma unroll
        for (int i = 0; i < VTASK; ++i) {
            const int task = tid + i * kThreads;
            __bf16 *dst = vts + v_chunk(task) * 8 * Lds<D>::VS + vt_pos(2 * v_pair(task));
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                // (V[2kp][e], V[2kp+1][e]) as one 32-bit word of V^T row 8 chunk + e.
                const unsigned sel = (e & 1) ? 0x07060302u : 0x05040100u;
                *reinterpret_cast<unsigned *>(dst + e * Lds<D>::VS) =
                    __builtin_amdgcn_perm(vreg[i][1][e >> 1], vreg[i][0][e >> 1], sel);
            }
        }
    }
};

}  // namespace tiles
}  // namespace hcms
