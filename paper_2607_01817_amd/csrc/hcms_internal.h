// Internal launchers of the HCMS HIP library (not part of the C ABI).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace hcms {

// Thread-local error detail behind hcms_last_error: fail() records a message
// and returns `status`, ok() clears it and returns HCMS_OK.
int fail(int status, const char *fmt, ...) __attribute__((format(printf, 2, 3)));
int ok();
const char *last_error();

// Copy `n_tensors` (1..3) head chunks at once.  Each tensor z moves
//   dst[z][j][t][:] = src[z][t][h0 + j][:]   (pack)
// for t < S, j < hc, where a row ([:]) is 16 << log2_units bytes.
// lds_reserve (at most 64 KiB): LDS bytes every workgroup holds unused.  The
// kernels need none; a reservation larger than the LDS an attention
// workgroup leaves free on its CU (kCopyBesideAttentionLds) keeps the copy's
// workgroups off CUs that run attention, so a copy issued beside an attention
// launch runs on the CUs its last round leaves idle instead of taking issue
// slots from the attention waves.
hipError_t launch_pack(const void *const *src, void *const *dst, int n_tensors,
                       int64_t S, int64_t H, int64_t h0, int64_t hc, int log2_units,
                       unsigned lds_reserve, hipStream_t stream);

// Each tensor z moves  dst[z][t][h0 + j][:] = src[z][j][t][:]   (unpack)
hipError_t launch_unpack(const void *const *src, void *const *dst, int n_tensors, int64_t S,
                         int64_t H, int64_t h0, int64_t hc, int log2_units, unsigned lds_reserve,
                         hipStream_t stream);

// The d = 128 bf16 attention kernels hold 128 KiB or more of a CU's 160 KiB
// of LDS; a copy workgroup holding 40 KiB therefore never shares a CU with one.
inline constexpr unsigned kCopyBesideAttentionLds = 40 * 1024;

// Attention of `n_heads` consecutive heads, head-major [n_heads][S][d]
// buffers starting at the chunk's first head.  scale_log2e = scale * log2(e).
// dtype: 0 = bf16 storage, 1 = fp32 storage.  d in {64, 128}.
// Tiling of the attention launch: queries per workgroup, and workgroups one
// CU holds at once, for head dimension d (64 or 128).
int attention_queries_per_block(int d);

// The plan HCMS_MODE_AUTO runs for these chunks (hcms_auto_mode's rule; the
// arguments are not validated).
int auto_plan(int S, int d, int dtype, const int *sizes, int C, int n_cu);
int attention_blocks_per_cu(int d);

// Scratch for splitting a launch's last round of tiles over several
// workgroups (d = 128 bf16): `slots` partial states of
// attention_split_slot_bytes() bytes each (part: slots x 64 KiB, ml: slots x
// 4 KiB, 16-byte aligned) and `counters` ints that are zero between launches.  At most one
// launch may use one scratch at a time (launches on one stream are ordered).
struct SplitScratch {
    void *part;
    void *ml;
    int *count;
    int slots, counters;
    int n_cu;
    // Tiles at the end of the launch to split: -1 for the launch's own last
    // round (W mod n_cu); otherwise this many (at most W), for a launch whose
    // last tiles close a round that other launches' workgroups share.
    int64_t tail = -1;
};
int64_t attention_split_slot_bytes();
// Workgroups per split tile (2 or 3) a d = 128 bf16 launch of W tiles splits
// its last `tail` tiles into on n_cu CUs (tail -1: W mod n_cu), or 1 when it
// splits none.
int attention_split_ways(int64_t W, int S, int d, int dtype, int n_cu, int64_t tail = -1);

// lse, if not NULL, receives [n_heads][S] fp32 log2 softmax denominators:
// P_ij = exp2(scale_log2e * <q_i, k_j> - lse_i).  split: NULL, or scratch
// that lets the launch split its last round (same results either way).
hipError_t launch_attention(const void *q, const void *k, const void *v, void *o, float *lse,
                            int S, int n_heads, int d, float scale_log2e, int dtype,
                            const SplitScratch *split, hipStream_t stream);

// A head-chunk copy that can ride in an attention launch: the arguments of
// launch_pack (unpack = false) or launch_unpack (unpack = true) for rows of
// d = 128 bf16 elements.
struct RidingCopy {
    const void *src[3];
    void *dst[3];
    int n_tensors;
    bool unpack;
    int64_t h0, hc;
};
// launch_attention, with up to two copies appended to the same launch as
// extra workgroups after the attention workgroups, as many as the launch's
// last round leaves CUs idle on n_cu CUs (H: heads of the [S][H][d] side).
// Sets *riding when it did so; otherwise (not d = 128 bf16, fewer than
// n_cu / 8 idle CUs, or copies too large) it launches only the attention and
// the caller launches the copies after it.  A rider copy and the attention it
// rides with must not touch the same bytes.
hipError_t launch_attention_riding(const void *q, const void *k, const void *v, void *o, float *lse,
                                   int S, int n_heads, int d, float scale_log2e, int dtype,
                                   const RidingCopy *copies, int n_copies, int64_t H, int n_cu,
                                   const SplitScratch *split, bool *riding, hipStream_t stream);
// Backward of attention for `n_heads` consecutive heads (head-major buffers
// starting at the chunk's first head; lse and delta [n_heads][S] fp32).
// Without a score-gradient workspace (ds NULL, or ds_bytes below one head's
// attention_backward_ds_head_bytes): one query-parallel launch writing
// delta = <dO, O> and dq, then one key-parallel launch writing dk and dv.
// With one (d = 128, bf16): delta first, then per group of
// ds_bytes / head-bytes heads the key-parallel launch (dk, dv, and dS into
// ds) and the dQ product over the stored dS.
hipError_t launch_attention_backward(const void *q, const void *k, const void *v, const void *o,
                                     const void *dout, const float *lse, void *dq, void *dk,
                                     void *dv, float *delta, void *ds, int64_t ds_bytes, int S,
                                     int n_heads, int d, float scale, int dtype,
                                     hipStream_t stream);
// Bytes of score-gradient workspace one head needs (0: the path does not
// apply to this d and dtype).
int64_t attention_backward_ds_head_bytes(int S, int d, int dtype);

// Rotary position embedding on a latent grid of n_axes axes (row-major, the
// last axis fastest): the d/2 pairs of a head vector form consecutive groups
// of pairs[a] pairs, starting at pair_start[a], that turn with coordinate a.
// The rotation table holds grid[a] * pairs[a] (cos, sin) entries per axis,
// axis a's first at entry tab_off[a].
inline constexpr int kRopeMaxAxes = 4;
struct RopeAxes {
    int n_axes;
    int grid[kRopeMaxAxes], pairs[kRopeMaxAxes], pair_start[kRopeMaxAxes], tab_off[kRopeMaxAxes];
};

// Projection GEMM Y[M][N] = X[M][K] W[N][K]^T (bf16 MFMA, fp32 accumulation,
// Y rounded to the storage type); K a multiple of linear_k_multiple(), N of 8.
int linear_k_multiple();
hipError_t launch_linear(const void *x, const void *w, void *y, int M, int N, int K, int dtype,
                         hipStream_t stream);

// QKV projection: X[S][D] times W[3 H d][D]^T, split into q, k, v [S][H][d],
// q and k rotated with `table` (NULL: no rotation).
hipError_t launch_qkv_projection(const void *x, const void *w, void *q, void *k, void *v,
                                 const float *table, const RopeAxes &ax, int S, int D, int H, int d,
                                 int dtype, hipStream_t stream);

// Fills the rotation table of `ax` (fp32 (cos, sin) pairs).
hipError_t launch_rope_table(float *table, const RopeAxes &ax, double base, hipStream_t stream);

}  // namespace hcms
