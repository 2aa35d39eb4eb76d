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
#include "copy_tiles.h"
#include "hcms_internal.h"

namespace hcms {
namespace {

using copy::kThreads;
using copy::PackPtrs;

constexpr unsigned kMaxLdsReserve = 64 * 1024;  // at most 64 KiB per workgroup

// grid: x = copy::blocks_x(S, LOG2U), y = hc, z = tensor.
template <int LOG2U>
__global__ __launch_bounds__(kThreads) void pack_kernel(PackPtrs p, int64_t S, int64_t H,
                                                        int64_t h0) {
    copy::copy_block<LOG2U, false>(p, S, H, h0, blockIdx.x, blockIdx.y, blockIdx.z, threadIdx.x);
}

// grid: x = copy::blocks_x(S, LOG2U), y = hc, z = tensor.
template <int LOG2U>
__global__ __launch_bounds__(kThreads) void unpack_kernel(PackPtrs p, int64_t S, int64_t H,
                                                          int64_t h0) {
    copy::copy_block<LOG2U, true>(p, S, H, h0, blockIdx.x, blockIdx.y, blockIdx.z, threadIdx.x);
}

dim3 grid_for(int64_t S, int64_t hc, int log2_units, int n_tensors) {
    return dim3(static_cast<unsigned>(copy::blocks_x(S, log2_units)), static_cast<unsigned>(hc),
                static_cast<unsigned>(n_tensors));
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

bool strided_span_fits(int64_t H) { return copy::strided_span_fits(H); }

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
