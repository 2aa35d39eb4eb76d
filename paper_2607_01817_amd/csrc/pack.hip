// Head-chunk pack / unpack kernels for gfx950.
//
// Pack is the local share of the Ulysses input all-to-all plus the split along
// heads (Sec. 3.1, Sec. 3.3 split equation, Alg. 1 SplitByHeads/AllToAll):
//   dst[j][t][:] = src[t][h0 + j][:]      src [S][H][d], dst [hc][S][d]
// where t = p * (S / P) + s is the global token of shard p, local index s: a
// contiguous [P][S/P][H][d] buffer is byte-for-byte [S][H][d].  Unpack is the
// inverse (output all-to-all + concatenation along heads).
//
// The element of the permutation is a whole d-row (128, 256 or 512 bytes for
// the supported shapes), so both the gather side and the scatter side touch
// complete, aligned 128-byte cache lines.  Consecutive lanes move consecutive
// 16-byte units of the dense side; the strided side is still read or written in
// full rows.  No LDS stage is needed for coalescing.  Each thread issues all of
// its loads before any store to keep several 16-byte requests in flight.  The
// source is read once, so its loads carry the non-temporal hint.
//
// Register budget.  In the pipelined schedules these kernels run while an
// attention workgroup holds its CU; that workgroup leaves 16 VGPRs per SIMD
// lane free (two waves of at most 248).  A copy wave that fits in those 16
// registers is placed beside the attention waves instead of waiting for the CU
// to drain, so the copy never delays an attention workgroup's start.  The
// kernels therefore keep three 16-byte units per lane in flight, address
// memory through buffer resources built per workgroup (64-bit bases in scalar
// registers, one 32-bit lane offset, the per-unit step as a scalar offset),
// and let the hardware range check of the resource replace per-lane tail
// branches: out-of-range loads return zero and out-of-range stores are
// dropped.
#include "hcms_internal.h"

namespace hcms {
namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr unsigned kMaxLdsReserve = 64 * 1024;  // at most 64 KiB per workgroup
constexpr int kUnroll = 3;
constexpr int kUnitsPerBlock = kThreads * kUnroll;  // 16-byte units per workgroup
constexpr int kNonTemporal = 2;                     // cache-policy bit of a streaming load

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

// Workgroup (x, j, z) moves dense units [u0, u0 + kUnitsPerBlock) of chunk
// head j of tensor z; those are rows t0 .. t0 + kUnitsPerBlock / U - 1 of the
// strided side, which lie within 4096 * H * kUnroll bytes of the row of t0.
struct BlockSpans {
    int64_t dense_off, dense_left, strided_off, strided_left;
};

template <int LOG2U>
__device__ inline BlockSpans block_spans(int64_t S, int64_t H, int64_t h0) {
    const int64_t j = blockIdx.y;
    const int64_t u0 = static_cast<int64_t>(blockIdx.x) * kUnitsPerBlock;
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

// grid: x = ceil(S * U / kUnitsPerBlock), y = hc, z = tensor.
template <int LOG2U>
__global__ __launch_bounds__(kThreads) void pack_kernel(PackPtrs p, int64_t S, int64_t H,
                                                        int64_t h0) {
    const BlockSpans b = block_spans<LOG2U>(S, H, h0);
    const __amdgpu_buffer_rsrc_t src =
        span_rsrc(p.src[blockIdx.z] + b.strided_off, b.strided_left);
    const __amdgpu_buffer_rsrc_t dst = span_rsrc(p.dst[blockIdx.z] + b.dense_off, b.dense_left);
    const uint32_t tid = threadIdx.x;
    const uint32_t so = strided_lane_off<LOG2U>(tid, static_cast<uint32_t>(H));
    const uint32_t step = static_cast<uint32_t>(H) * (kThreads << 4);  // kThreads units down
    u32x4 buf[kUnroll];
#pragma unroll
    for (int i = 0; i < kUnroll; ++i)
        buf[i] = __builtin_amdgcn_raw_buffer_load_b128(src, so, i * step, kNonTemporal);
#pragma unroll
    for (int i = 0; i < kUnroll; ++i)
        __builtin_amdgcn_raw_buffer_store_b128(buf[i], dst, tid << 4, i * (kThreads << 4), 0);
}

// grid: x = ceil(S * U / kUnitsPerBlock), y = hc, z = tensor.
template <int LOG2U>
__global__ __launch_bounds__(kThreads) void unpack_kernel(PackPtrs p, int64_t S, int64_t H,
                                                          int64_t h0) {
    const BlockSpans b = block_spans<LOG2U>(S, H, h0);
    const __amdgpu_buffer_rsrc_t src = span_rsrc(p.src[blockIdx.z] + b.dense_off, b.dense_left);
    const __amdgpu_buffer_rsrc_t dst = span_rsrc(p.dst[blockIdx.z] + b.strided_off, b.strided_left);
    const uint32_t tid = threadIdx.x;
    const uint32_t so = strided_lane_off<LOG2U>(tid, static_cast<uint32_t>(H));
    const uint32_t step = static_cast<uint32_t>(H) * (kThreads << 4);
    u32x4 buf[kUnroll];
#pragma unroll
    for (int i = 0; i < kUnroll; ++i)
        buf[i] = __builtin_amdgcn_raw_buffer_load_b128(src, tid << 4, i * (kThreads << 4), kNonTemporal);
#pragma unroll
    for (int i = 0; i < kUnroll; ++i)
        __builtin_amdgcn_raw_buffer_store_b128(buf[i], dst, so, i * step, 0);
}

dim3 grid_for(int64_t S, int64_t hc, int log2_units, int n_tensors) {
    const int64_t units = S << log2_units;
    return dim3(static_cast<unsigned>((units + kUnitsPerBlock - 1) / kUnitsPerBlock),
                static_cast<unsigned>(hc), static_cast<unsigned>(n_tensors));
}

// lds_reserve: bytes of LDS each workgroup holds without using them (see
// launch_pack).
template <int LOG2U>
void pack_dispatch(const PackPtrs &p, int n_tensors, int64_t S, int64_t H, int64_t h0,
                   int64_t hc, unsigned lds_reserve, hipStream_t stream) {
    pack_kernel<LOG2U><<<grid_for(S, hc, LOG2U, n_tensors), kThreads, lds_reserve, stream>>>(p, S, H, h0);
}

template <int LOG2U>
void unpack_dispatch(const PackPtrs &p, int n_tensors, int64_t S, int64_t H, int64_t h0,
                     int64_t hc, unsigned lds_reserve, hipStream_t stream) {
    unpack_kernel<LOG2U><<<grid_for(S, hc, LOG2U, n_tensors), kThreads, lds_reserve, stream>>>(p, S, H, h0);
}

// Lane offsets on the strided side are 32-bit: a workgroup spans at most
// kUnitsPerBlock rows of H heads, 16 KiB * H bytes.
bool strided_span_fits(int64_t H) { return H > 0 && H * (int64_t{kUnitsPerBlock} << 4) < (int64_t{1} << 32); }

}  // namespace

hipError_t launch_pack(const void *const *src, void *const *dst, int n_tensors, int64_t S,
                       int64_t H, int64_t h0, int64_t hc, int log2_units, unsigned lds_reserve,
                       hipStream_t stream) {
    if (S == 0 || hc == 0) return hipSuccess;
    if (lds_reserve > kMaxLdsReserve) return hipErrorInvalidValue;
    if (!strided_span_fits(H) || n_tensors < 1 || n_tensors > 3) return hipErrorInvalidValue;
    PackPtrs p{};
    for (int z = 0; z < n_tensors; ++z) {
        p.src[z] = static_cast<const char *>(src[z]);
        p.dst[z] = static_cast<char *>(dst[z]);
    }
    switch (log2_units) {
        case 0: pack_dispatch<0>(p, n_tensors, S, H, h0, hc, lds_reserve, stream); break;
        case 1: pack_dispatch<1>(p, n_tensors, S, H, h0, hc, lds_reserve, stream); break;
        case 2: pack_dispatch<2>(p, n_tensors, S, H, h0, hc, lds_reserve, stream); break;
        case 3: pack_dispatch<3>(p, n_tensors, S, H, h0, hc, lds_reserve, stream); break;
        case 4: pack_dispatch<4>(p, n_tensors, S, H, h0, hc, lds_reserve, stream); break;
        case 5: pack_dispatch<5>(p, n_tensors, S, H, h0, hc, lds_reserve, stream); break;
        case 6: pack_dispatch<6>(p, n_tensors, S, H, h0, hc, lds_reserve, stream); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_unpack(const void *const *src, void *const *dst, int n_tensors, int64_t S,
                         int64_t H, int64_t h0, int64_t hc, int log2_units, unsigned lds_reserve,
                         hipStream_t stream) {
    if (S == 0 || hc == 0) return hipSuccess;
    if (lds_reserve > kMaxLdsReserve) return hipErrorInvalidValue;
    if (!strided_span_fits(H) || n_tensors < 1 || n_tensors > 3) return hipErrorInvalidValue;
    PackPtrs p{};
    for (int z = 0; z < n_tensors; ++z) {
        p.src[z] = static_cast<const char *>(src[z]);
        p.dst[z] = static_cast<char *>(dst[z]);
    }
    switch (log2_units) {
        case 0: unpack_dispatch<0>(p, n_tensors, S, H, h0, hc, lds_reserve, stream); break;
        case 1: unpack_dispatch<1>(p, n_tensors, S, H, h0, hc, lds_reserve, stream); break;
        case 2: unpack_dispatch<2>(p, n_tensors, S, H, h0, hc, lds_reserve, stream); break;
        case 3: unpack_dispatch<3>(p, n_tensors, S, H, h0, hc, lds_reserve, stream); break;
        case 4: unpack_dispatch<4>(p, n_tensors, S, H, h0, hc, lds_reserve, stream); break;
        case 5: unpack_dispatch<5>(p, n_tensors, S, H, h0, hc, lds_reserve, stream); break;
        case 6: unpack_dispatch<6>(p, n_tensors, S, H, h0, hc, lds_reserve, stream); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace hcms
