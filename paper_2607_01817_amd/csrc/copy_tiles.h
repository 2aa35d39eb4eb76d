// Index maps and the per-block body of the head-chunk layout copies (pack and
// unpack, Sec. 3.1 and the split equation of Sec. 3.3), shared by the copy
// kernels and by the attention launch that carries a neighbouring chunk's
// copies as extra workgroups.
//
// A copy block is 256 threads moving kUnitsPerBlock consecutive 16-byte units
// of one head of one tensor on the dense (head-major) side.  Block (x, j, z)
// covers dense units [x * kUnitsPerBlock, (x + 1) * kUnitsPerBlock) of chunk
// head j of tensor z; those are rows t0 .. t0 + kUnitsPerBlock / U - 1 of the
// strided ([S][H][d]) side, which lie within 4096 * H * kUnroll bytes of the
// row of t0.  Addresses are one 32-bit lane offset plus a scalar offset per
// unit, into buffer resources whose range check handles the ragged tail
// (out-of-range loads read zero, out-of-range stores are dropped).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace hcms {
namespace copy {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

inline constexpr int kThreads = 256;                       // threads of one copy block
inline constexpr int kUnroll = 3;                          // 16-byte units per thread
inline constexpr int kUnitsPerBlock = kThreads * kUnroll;  // 16-byte units per block
inline constexpr int kNonTemporal = 2;                     // cache-policy bit of a streaming load

struct PackPtrs {
    const char *src[3];
    char *dst[3];
};

// Resource over [base, base + min(bytes, 2^32 - 1)).
__device__ inline __amdgpu_buffer_rsrc_t span_rsrc(const char *base, int64_t bytes) {
    const int64_t n = bytes < 0 ? 0 : (bytes > 0xFFFFFFFFll ? 0xFFFFFFFFll : bytes);
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<char *>(base), 0,
                                             static_cast<int>(static_cast<uint32_t>(n)),
                                             0x00020000);
}

struct BlockSpans {
    int64_t dense_off, dense_left, strided_off, strided_left;
};

template <int LOG2U>
__device__ inline BlockSpans block_spans(int64_t S, int64_t H, int64_t h0, int64_t x, int64_t j) {
    const int64_t u0 = x * kUnitsPerBlock;
    const int64_t t0 = u0 >> LOG2U;
    BlockSpans b;
    b.dense_off = ((j * S) << (LOG2U + 4)) + (u0 << 4);
    b.dense_left = ((S << LOG2U) - u0) << 4;
    b.strided_off = ((t0 * H + h0 + j) << (LOG2U + 4));
    b.strided_left = ((S * H) << (LOG2U + 4)) - b.strided_off;
    return b;
}

// Byte offset of local unit lu = tid + i * kThreads on the strided side,
// relative to the row of t0: (lu / U) rows of H heads, then the unit in row.
template <int LOG2U>
__device__ inline uint32_t strided_lane_off(uint32_t tid, uint32_t H) {
    return (((tid >> LOG2U) * H) << (LOG2U + 4)) + ((tid & ((1u << LOG2U) - 1)) << 4);
}

// Copy block (x, j, z), thread tid < kThreads.  Pack gathers rows of head
// h0 + j from the strided side into the dense side; unpack scatters back.
template <int LOG2U, bool kUnpack>
__device__ inline void copy_block(const PackPtrs &p, int64_t S, int64_t H, int64_t h0, int64_t x,
                                  int64_t j, int z, uint32_t tid) {
    const BlockSpans b = block_spans<LOG2U>(S, H, h0, x, j);
    const uint32_t so = strided_lane_off<LOG2U>(tid, static_cast<uint32_t>(H));
    const uint32_t step = static_cast<uint32_t>(H) * (kThreads << 4);  // kThreads units down
    u32x4 buf[kUnroll];
    if constexpr (!kUnpack) {
        const __amdgpu_buffer_rsrc_t src = span_rsrc(p.src[z] + b.strided_off, b.strided_left);
        const __amdgpu_buffer_rsrc_t dst = span_rsrc(p.dst[z] + b.dense_off, b.dense_left);
#pragma unroll
        for (int i = 0; i < kUnroll; ++i)
            buf[i] = __builtin_amdgcn_raw_buffer_load_b128(src, so, i * step, kNonTemporal);
#pragma unroll
        for (int i = 0; i < kUnroll; ++i)
            __builtin_amdgcn_raw_buffer_store_b128(buf[i], dst, tid << 4, i * (kThreads << 4), 0);
    } else {
        const __amdgpu_buffer_rsrc_t src = span_rsrc(p.src[z] + b.dense_off, b.dense_left);
        const __amdgpu_buffer_rsrc_t dst = span_rsrc(p.dst[z] + b.strided_off, b.strided_left);
#pragma unroll
        for (int i = 0; i < kUnroll; ++i)
            buf[i] = __builtin_amdgcn_raw_buffer_load_b128(src, tid << 4, i * (kThreads << 4),
                                                           kNonTemporal);
#pragma unroll
        for (int i = 0; i < kUnroll; ++i)
            __builtin_amdgcn_raw_buffer_store_b128(buf[i], dst, so, i * step, 0);
    }
}

// Copy blocks along x of one (head, tensor): ceil(S * U / kUnitsPerBlock).
inline int64_t blocks_x(int64_t S, int log2_units) {
    return ((S << log2_units) + kUnitsPerBlock - 1) / kUnitsPerBlock;
}

// Lane offsets on the strided side are 32-bit: a block spans at most
// kUnitsPerBlock rows of H heads, 16 KiB * H bytes.
inline bool strided_span_fits(int64_t H) {
    return H > 0 && H * (int64_t{kUnitsPerBlock} << 4) < (int64_t{1} << 32);
}

}  // namespace copy
}  // namespace hcms
