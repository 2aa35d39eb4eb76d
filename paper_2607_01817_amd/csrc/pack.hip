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
#include "hcms_internal.h"

namespace hcms {
namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kUnroll = 4;
constexpr int kUnitsPerBlock = kThreads * kUnroll;

struct PackPtrs {
    const u32x4 *src[3];
    u32x4 *dst[3];
};

// grid: x = ceil(S * units_per_row / kUnitsPerBlock), y = hc, z = tensor.
template <int LOG2U>
__global__ __launch_bounds__(kThreads) void pack_kernel(PackPtrs p, int64_t S, int64_t H,
                                                        int64_t h0) {
    const int64_t j = blockIdx.y;
    const u32x4 *__restrict__ src = p.src[blockIdx.z];
    u32x4 *__restrict__ dst = p.dst[blockIdx.z] + ((j * S) << LOG2U);
    const int64_t n = S << LOG2U;
    const int64_t base = static_cast<int64_t>(blockIdx.x) * kUnitsPerBlock + threadIdx.x;
    u32x4 buf[kUnroll];
#pragma unroll
    for (int i = 0; i < kUnroll; ++i) {
        const int64_t u = base + i * kThreads;
        if (u < n) {
            const int64_t t = u >> LOG2U;
            const int64_t w = u & ((1 << LOG2U) - 1);
            buf[i] = __builtin_nontemporal_load(src + ((t * H + h0 + j) << LOG2U) + w);
        }
    }
#pragma unroll
    for (int i = 0; i < kUnroll; ++i) {
        const int64_t u = base + i * kThreads;
        if (u < n) dst[u] = buf[i];
    }
}

// grid: x = ceil(S * units_per_row / kUnitsPerBlock), y = hc.
template <int LOG2U>
__global__ __launch_bounds__(kThreads) void unpack_kernel(const u32x4 *__restrict__ src_all,
                                                          u32x4 *__restrict__ dst, int64_t S,
                                                          int64_t H, int64_t h0) {
    const int64_t j = blockIdx.y;
    const u32x4 *__restrict__ src = src_all + ((j * S) << LOG2U);
    const int64_t n = S << LOG2U;
    const int64_t base = static_cast<int64_t>(blockIdx.x) * kUnitsPerBlock + threadIdx.x;
    u32x4 buf[kUnroll];
#pragma unroll
    for (int i = 0; i < kUnroll; ++i) {
        const int64_t u = base + i * kThreads;
        if (u < n) buf[i] = __builtin_nontemporal_load(src + u);
    }
#pragma unroll
    for (int i = 0; i < kUnroll; ++i) {
        const int64_t u = base + i * kThreads;
        if (u < n) {
            const int64_t t = u >> LOG2U;
            const int64_t w = u & ((1 << LOG2U) - 1);
            dst[((t * H + h0 + j) << LOG2U) + w] = buf[i];
        }
    }
}

dim3 grid_for(int64_t S, int64_t hc, int log2_units, int n_tensors) {
    const int64_t units = S << log2_units;
    return dim3(static_cast<unsigned>((units + kUnitsPerBlock - 1) / kUnitsPerBlock),
                static_cast<unsigned>(hc), static_cast<unsigned>(n_tensors));
}

template <int LOG2U>
void pack_dispatch(const PackPtrs &p, int n_tensors, int64_t S, int64_t H, int64_t h0,
                   int64_t hc, hipStream_t stream) {
    pack_kernel<LOG2U><<<grid_for(S, hc, LOG2U, n_tensors), kThreads, 0, stream>>>(p, S, H, h0);
}

template <int LOG2U>
void unpack_dispatch(const u32x4 *src, u32x4 *dst, int64_t S, int64_t H, int64_t h0,
                     int64_t hc, hipStream_t stream) {
    unpack_kernel<LOG2U><<<grid_for(S, hc, LOG2U, 1), kThreads, 0, stream>>>(src, dst, S, H, h0);
}

}  // namespace

hipError_t launch_pack(const void *const *src, void *const *dst, int n_tensors, int64_t S,
                       int64_t H, int64_t h0, int64_t hc, int log2_units, hipStream_t stream) {
    if (S == 0 || hc == 0) return hipSuccess;
    PackPtrs p{};
    for (int z = 0; z < n_tensors; ++z) {
        p.src[z] = static_cast<const u32x4 *>(src[z]);
        p.dst[z] = static_cast<u32x4 *>(dst[z]);
    }
    switch (log2_units) {
        case 0: pack_dispatch<0>(p, n_tensors, S, H, h0, hc, stream); break;
        case 1: pack_dispatch<1>(p, n_tensors, S, H, h0, hc, stream); break;
        case 2: pack_dispatch<2>(p, n_tensors, S, H, h0, hc, stream); break;
        case 3: pack_dispatch<3>(p, n_tensors, S, H, h0, hc, stream); break;
        case 4: pack_dispatch<4>(p, n_tensors, S, H, h0, hc, stream); break;
        case 5: pack_dispatch<5>(p, n_tensors, S, H, h0, hc, stream); break;
        case 6: pack_dispatch<6>(p, n_tensors, S, H, h0, hc, stream); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_unpack(const void *src, void *dst, int64_t S, int64_t H, int64_t h0,
                         int64_t hc, int log2_units, hipStream_t stream) {
    if (S == 0 || hc == 0) return hipSuccess;
    const u32x4 *s = static_cast<const u32x4 *>(src);
    u32x4 *d = static_cast<u32x4 *>(dst);
    switch (log2_units) {
        case 0: unpack_dispatch<0>(s, d, S, H, h0, hc, stream); break;
        case 1: unpack_dispatch<1>(s, d, S, H, h0, hc, stream); break;
        case 2: unpack_dispatch<2>(s, d, S, H, h0, hc, stream); break;
        case 3: unpack_dispatch<3>(s, d, S, H, h0, hc, stream); break;
        case 4: unpack_dispatch<4>(s, d, S, H, h0, hc, stream); break;
        case 5: unpack_dispatch<5>(s, d, S, H, h0, hc, stream); break;
        case 6: unpack_dispatch<6>(s, d, S, H, h0, hc, stream); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace hcms
