/*
 * hcms.h -- C ABI of the single-GPU hot path of HCMS (Head-Chunked Multi-Stream
 * pipeline for sequence-parallel attention, arXiv 2607.01817) on AMD MI355X
 * (gfx950).
 *
 * One GPU's share of HCMS under Ulysses sequence parallelism is: a layout
 * permutation of each head chunk from sequence-sharded [P][S/P][H][d] to
 * head-major [H_c][S][d] ("pack", the local share of the input all-to-all),
 * full-sequence non-causal softmax attention on the chunk, and the inverse
 * permutation back ("unpack", the local share of the output all-to-all plus the
 * concatenation along heads), scheduled on a copy stream and a compute stream
 * ordered by events (Sec. 3.4-3.6, Alg. 1).
 *
 * Conventions for every entry point
 *   - Buffers are device memory owned by the caller, contiguous, row-major,
 *     16-byte aligned.  The library allocates no device memory on any call
 *     except hcms_ctx_create (which creates events only).
 *   - `stream` arguments are hipStream_t handles passed as void*.  NULL is the
 *     null stream of the current device.  Streams are borrowed, never destroyed.
 *   - All compute calls are asynchronous and stream-ordered; a kernel fault
 *     surfaces at the caller's next synchronisation.
 *   - Arguments are validated completely before any HIP call: on error nothing
 *     is enqueued and a negative hcms_status is returned.  hcms_last_error()
 *     then gives a thread-local human-readable detail.  No C++ exception
 *     crosses this boundary.
 *   - Input and output buffers of one call must not overlap (checked; returns
 *     HCMS_ERR_ALIAS).
 *   - S = 0 (an empty sequence) is valid and enqueues nothing; the tensor
 *     pointers may then be NULL.
 *   - Supported: d in {64, 128} for attention; for pack/unpack any d whose row
 *     (d * element size) is a power of two from 16 to 1024 bytes; dtype bf16 or
 *     fp32 storage.
 *     Attention computes with bf16 MFMA operands and fp32 accumulation; fp32
 *     storage is rounded to bf16 (nearest-even) when loaded.
 *   - Calls on different streams that write the same buffer race; ordering is
 *     the caller's (or hcms_forward's) business.
 */
#ifndef HCMS_H
#define HCMS_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define HCMS_ABI_VERSION 3

#if defined(__GNUC__)
#define HCMS_API __attribute__((visibility("default")))
#else
#define HCMS_API
#endif

typedef enum hcms_dtype {
    HCMS_BF16 = 0, /* 2-byte bfloat16 storage */
    HCMS_FP32 = 1  /* 4-byte IEEE float storage */
} hcms_dtype;

typedef enum hcms_status {
    HCMS_OK = 0,
    HCMS_ERR_NULL = -1,     /* a required pointer is NULL */
    HCMS_ERR_SHAPE = -2,    /* S < 0, H < 1, P < 1, S % P != 0, unsupported d, size overflow */
    HCMS_ERR_CHUNKS = -3,   /* n_chunks < 1 or > H, a size < 1, sizes not summing to H,
                               head range outside [0, H), more chunks than the context holds */
    HCMS_ERR_DTYPE = -4,    /* dtype not one of hcms_dtype */
    HCMS_ERR_ALIGN = -5,    /* a buffer is not 16-byte aligned */
    HCMS_ERR_HIP = -6,      /* a HIP runtime call or kernel launch failed */
    HCMS_ERR_ARG = -7,      /* bad scalar argument: scale not finite and > 0, bad mode,
                               context bound to another device */
    HCMS_ERR_ALIAS = -8,    /* an input buffer overlaps an output buffer */
    HCMS_ERR_CAPACITY = -9  /* output array too small (hcms_plan, timing queries) */
} hcms_status;

/* ABI version of the loaded library (HCMS_ABI_VERSION it was built with). */
HCMS_API int hcms_abi_version(void);

/* Static string naming a status code ("HCMS_OK", "HCMS_ERR_SHAPE", ...). */
HCMS_API const char *hcms_status_string(int status);

/* Thread-local detail of the last error returned on this thread ("" if none).
   Valid until the next hcms_* call on the same thread. */
HCMS_API const char *hcms_last_error(void);

/*
 * Head-chunk sizes for H heads in C chunks, larger chunks first
 * (Sec. 3.3, chunk-size equation: H_c = floor(H/C) + 1 if c < H mod C, else
 * floor(H/C); Sec. 4.1 calls it "more-first-less-later").
 *   sizes_out : host array of C ints, written on success.
 * Returns HCMS_OK, HCMS_ERR_NULL, or HCMS_ERR_CHUNKS unless 1 <= C <= H.
 */
HCMS_API int hcms_default_chunks(int H, int C, int *sizes_out);

/*
 * Pack one head chunk (Sec. 3.3 split along heads + the local share of the
 * input all-to-all of Sec. 3.1, Alg. 1 SplitByHeads / AllToAll):
 *   dst_hm[j][p*(S/P) + s][e] = src_seq[p][s][h_begin + j][e]
 * for p < P, s < S/P, j < h_count, e < d.  A pure byte move.
 *   src_seq : device, [P][S/P][H][d] (identical bytes to [S][H][d])
 *   dst_hm  : device, [h_count][S][d]
 *   dtype   : element size only (the move is bit-exact)
 * Errors: NULL, SHAPE (S % P, row size), CHUNKS (head range), DTYPE,
 * ALIGN, ALIAS, HIP.
 */
HCMS_API int hcms_pack(const void *src_seq, void *dst_hm, int P, int S, int H, int d,
              int h_begin, int h_count, int dtype, void *stream);

/*
 * Inverse of hcms_pack (the local share of the output all-to-all and the
 * concatenation along heads of Alg. 1):
 *   dst_seq[p][s][h_begin + j][e] = src_hm[j][p*(S/P) + s][e]
 * Head slots outside [h_begin, h_begin + h_count) of dst_seq are not touched.
 * Same arguments and errors as hcms_pack.
 */
HCMS_API int hcms_unpack(const void *src_hm, void *dst_seq, int P, int S, int H, int d,
                int h_begin, int h_count, int dtype, void *stream);

/*
 * Head-chunked attention (Sec. 3.3 Property of computational independence;
 * Alg. 1, compute-stream loop): for every head h < H and query i < S
 *   O[h][i] = sum_j softmax_j(scale * <Q[h][i], K[h][j]>) V[h][j]
 * over all S keys (non-causal, no mask).  The heads are processed as
 * n_chunks consecutive ranges of chunk_sizes[c] heads, one kernel launch per
 * chunk, in order, on `stream`.
 *   q, k, v, out : device, head-major [H][S][d]
 *   scale        : finite and > 0 (1/sqrt(d) for the usual attention)
 *   chunk_sizes  : host array of n_chunks positive ints summing to H
 * The result for a head does not depend on how the heads are chunked: any two
 * chunkings give bit-identical outputs.  Runs are deterministic.
 * Errors: NULL, SHAPE (d not 64/128), CHUNKS, DTYPE, ALIGN, ARG, ALIAS, HIP.
 */
HCMS_API int hcms_attention(const void *q, const void *k, const void *v, void *out,
                   int S, int H, int d, float scale,
                   const int *chunk_sizes, int n_chunks, int dtype, void *stream);

/*
 * Training forward: hcms_attention plus, per head h and query i, the log2 of
 * the softmax denominator,
 *   lse[h][i] = log2 sum_j exp2(c <Q[h][i], K[h][j]>),  c = scale * log2(e),
 * the statistic the backward pass recomputes the weights from:
 * P_ij = exp2(c <Q[h][i], K[h][j]> - lse[h][i]).
 *   lse : device, [H][S] fp32, 4-byte aligned, disjoint from q, k, v, out
 * out is bit-identical to hcms_attention's.  Errors: as hcms_attention, plus
 * NULL, ALIGN and ALIAS for lse.
 */
HCMS_API int hcms_attention_lse(const void *q, const void *k, const void *v, void *out, float *lse,
                                int S, int H, int d, float scale, const int *chunk_sizes,
                                int n_chunks, int dtype, void *stream);

/*
 * Backward of head-chunked attention, for training (the forward's gradient
 * through the row softmax; the appendix validates HCMS for training).  With
 * s_ij = <Q[h][i], K[h][j]>, P_ij = exp2(c s_ij - lse[h][i]) (the forward's
 * weights), D_i = <dO[h][i], O[h][i]>:
 *   dV[h][j] = sum_i P_ij dO[h][i]
 *   dQ[h][i] = scale sum_j P_ij (<dO[h][i], V[h][j]> - D_i) K[h][j]
 *   dK[h][j] = scale sum_i P_ij (<dO[h][i], V[h][j]> - D_i) Q[h][i]
 * Per chunk, in order on `stream`, without a score-gradient workspace: one
 * query-parallel launch (D into delta, then dq) and one key-parallel launch
 * (dk, dv); the query-parallel one recomputes the scores and dP, so the two
 * execute 14 S^2 d FLOP per head for the 10 S^2 d of the five products.
 * With a workspace of at least hcms_backward_ds_bytes for one head (d = 128,
 * bf16; ignored otherwise): D into delta, then per group of
 * ds_bytes / (that size) heads the key-parallel launch, which also stores
 * every dS_ij (rounded to bf16, as its dK product uses it) in the workspace,
 * and dq as one product over the stored dS (10 S^2 d FLOP per head, plus
 * 2 S^2 bytes written and read).  dk and dv are the same bits either way; dq
 * differs from the other path's only in its fp32 summation order.  No
 * atomics: deterministic, and the result does not depend on the chunking.
 * Operands are rounded to bf16 for the MFMAs (fp32 storage included),
 * accumulation is fp32, dq, dk, dv are rounded to the storage type.
 *   q, k, v, out : the forward's inputs and output, [H][S][d]
 *   dout         : dL/dO, [H][S][d]
 *   lse          : [H][S] fp32 from hcms_attention_lse on the same q, k, v, scale
 *   dq, dk, dv   : outputs, [H][S][d], disjoint from every input and each other
 *   delta        : [H][S] fp32 workspace (receives D)
 *   ds, ds_bytes : device workspace for the score gradients, 256-byte
 *                  aligned, disjoint from every other buffer; NULL or too
 *                  small for one head: the path without it
 * Errors: as hcms_attention, plus NULL, ALIGN and ALIAS for the added buffers,
 * ARG for ds_bytes < 0.
 */
HCMS_API int hcms_attention_backward(const void *q, const void *k, const void *v, const void *out,
                                     const void *dout, const float *lse, void *dq, void *dk,
                                     void *dv, float *delta, void *ds, int64_t ds_bytes, int S,
                                     int H, int d, float scale, const int *chunk_sizes,
                                     int n_chunks, int dtype, void *stream);

/* Bytes of score-gradient workspace that one head of hcms_attention_backward
   (or of hcms_backward, per region) needs: 8 ceil(S / 256)^2 * 16 KiB, about
   2 S^2 bytes; 0 where the path does not apply (d != 128 or fp32 storage).
   Errors: NULL, SHAPE (S < 0), DTYPE. */
HCMS_API int hcms_backward_ds_bytes(int S, int d, int dtype, int64_t *bytes_out);

/*
 * hcms_attention_backward without the delta workspace, for callers that
 * cannot allocate device memory (code under HIP graph capture, tight serving
 * or training loops, harnesses that forbid hipMalloc).  D = <dO, O> per query
 * goes to a scratch array inside the library instead: one per device,
 * HCMS_NOALLOC_DELTA_MAX floats (16 MiB), allocated with the library's code
 * object and held until the process ends.  The call itself allocates nothing
 * (no hipMalloc, no hipFree); the caller passes every input and output.
 * Arguments, results and errors are those of hcms_attention_backward without
 * a score-gradient workspace (dq, dk, dv bit-identical to it), plus CAPACITY
 * when S * H > HCMS_NOALLOC_DELTA_MAX.
 * The first call on a device looks up that device's copy of the array.
 * Calls on one device share its array: two calls whose launches can overlap
 * on one GPU (different streams without an ordering between them) race and
 * give undefined gradients.  Calls ordered on one stream are safe; every call
 * writes D before it reads it, so nothing needs clearing between calls.
 */
#define HCMS_NOALLOC_DELTA_MAX (4 * 1024 * 1024)
HCMS_API int hcms_attention_backward_noalloc(const void *q, const void *k, const void *v,
                                             const void *out, const void *dout, const float *lse,
                                             void *dq, void *dk, void *dv, int S, int H, int d,
                                             float scale, const int *chunk_sizes, int n_chunks,
                                             int dtype, void *stream);

/* ------------------------------------------------------------------------ */
/* Scheduler                                                                 */
/* ------------------------------------------------------------------------ */

/* Modes of hcms_forward / hcms_plan. */
#define HCMS_MODE_SERIAL 0     /* every op on the main stream, chunk by chunk */
#define HCMS_MODE_PIPELINED 1  /* Alg. 1: copy stream + compute stream + events */
#define HCMS_MODE_INLINE 2     /* one lane, four synchronisations (see hcms_plan) */
#define HCMS_MODE_LANES 3      /* chunks alternate between two streams (see hcms_plan) */
#define HCMS_MODE_AUTO 4       /* the mode hcms_auto_mode picks (fused, inline, lanes or serial;
                                  hcms_backward with stored score gradients: lanes);
                                  hcms_forward, hcms_forward_slots and hcms_backward take it,
                                  hcms_plan does not (no fixed plan) */
#define HCMS_MODE_SLOTS 5      /* Alg. 1's streams, copies interleaved so slots can be reused */
#define HCMS_MODE_FUSED 6      /* one stream; neighbouring copies ride in each attention launch */

/* Op kinds, streams and event ids of a plan (hcms_plan). */
#define HCMS_OP_RECORD 0     /* record event `event` on `stream` */
#define HCMS_OP_WAIT 1       /* make `stream` wait for event `event` */
#define HCMS_OP_PACK 2       /* pack Q, K and V of chunk `chunk` */
#define HCMS_OP_ATTENTION 3  /* attention of chunk `chunk` */
#define HCMS_OP_UNPACK 4     /* unpack O of chunk `chunk` */

#define HCMS_STREAM_MAIN 0
#define HCMS_STREAM_COPY 1
#define HCMS_STREAM_COMPUTE 2
#define HCMS_STREAM_IN_ATTENTION 3  /* runs inside the next ATTENTION op's launch (fused mode) */

typedef struct hcms_op {
    int kind;    /* HCMS_OP_* */
    int stream;  /* HCMS_STREAM_* */
    int chunk;   /* chunk index of PACK / ATTENTION / UNPACK, else -1 */
    int event;   /* event id of RECORD / WAIT, else -1.  With C chunks:
                    0 = E_main, 1 + c = E_c^pack, 1 + C + c = E_c^attn,
                    1 + 2C = E_done */
} hcms_op;

/*
 * Dry run of the scheduler: the exact op sequence hcms_forward issues, in host
 * issue order.  Pipelined mode follows Alg. 1: record E_main on main; the copy
 * stream waits E_main and packs chunk c then records E_c^pack, for every c;
 * the compute stream waits E_main, then for every c waits E_c^pack, runs the
 * attention of c and records E_c^attn; the copy stream then, for every c, waits
 * E_c^attn and unpacks c; finally E_done is recorded on the copy stream and the
 * main stream waits it (the join of Alg. 1 as a stream wait, not a host sync).
 * Serial mode is pack c, attention c, unpack c on the main stream for every c.
 * Inline and lanes modes are schedules for one GPU, where a pack or unpack
 * costs a few hundred times less than a chunk's attention and each event
 * record or wait on the critical path costs about as much as a copy.
 * Inline mode keeps one lane on the main stream with four synchronisations:
 * the main stream packs chunk 0 and records E_0^pack; the copy stream waits
 * it, packs chunks 1..C-1 and records E_{C-1}^pack; the main stream runs
 * every attention, waiting E_{C-1}^pack before attention 1 and recording
 * E_{C-2}^attn before attention C-1; the copy stream waits E_{C-2}^attn,
 * unpacks chunks 0..C-2 and records E_done; the main stream unpacks chunk
 * C-1 and waits E_done.  The compute stream is not used.
 * Lanes mode alternates chunks between the main stream (even c) and the
 * compute stream (odd c), each running pack c, attention c, unpack c in
 * order: the main stream records E_0^pack after chunk 0's pack, the compute
 * stream waits it before its first chunk and records E_done after its last,
 * and the main stream waits E_done after its own last chunk.  Besides the
 * copies, the attention launches of the two lanes overlap, so that the
 * workgroups of one fill the CUs the last round of the other leaves idle.
 * No launch splits its own last round; instead the last launch of each lane
 * (d = 128 bf16) splits its last rem tiles by key segments, rem the
 * workgroups of all chunks summed, mod n_cu: the tiles past the last whole
 * pooled round (same results either way).
 * The copy stream is not used.
 * Slots mode uses Alg. 1's streams and events but interleaves the copy stream
 * with the attentions: the copy stream packs chunks 0 and 1, then, for every
 * c, waits E_c^attn, unpacks c and packs c + 2 (recording E_{c+2}^pack), so
 * that chunk c + 2 can reuse chunk c's workspace slot (the input layout of one
 * chunk and the output layout of another beside a chunk's attention,
 * Sec. 3.5).  The host issues every record before any wait on it.
 * Fused mode is the overlap of Sec. 3.5 (the input layout of chunk c + 1 and
 * the output layout of chunk c - 1 beside the attention of chunk c) with the
 * dependencies of Alg. 1 kept by stream order alone, so it needs no events.
 * It runs on the main stream: it packs chunk 0; then, for every c, the pack
 * of chunk c + 1 (c + 1 < C) and the unpack of chunk c - 1 (c >= 1) are
 * issued on HCMS_STREAM_IN_ATTENTION, which means
 * that they run inside the launch of the ATTENTION op that follows them, as
 * workgroups dispatched after all of that launch's attention workgroups, on
 * the CUs its last round leaves idle; after the last attention the main
 * stream unpacks chunk C-1.  An op on HCMS_STREAM_IN_ATTENTION is ordered
 * after every main-stream op before that attention and before every one
 * after it, and overlaps the attention itself (it touches other heads'
 * buffers).  Where a launch cannot carry them (not d = 128 bf16, or its last
 * round leaves fewer than n_cu / 8 CUs idle) hcms_forward runs them right
 * after that attention on the main stream instead.
 * With one chunk the inline, lanes and fused plans are the serial plan.
 *   ops : host array of `cap` entries, or NULL to query the count.
 * Returns the number of ops (>= 0), HCMS_ERR_CHUNKS (n_chunks < 1),
 * HCMS_ERR_ARG (mode, or HCMS_MODE_AUTO, which has no fixed plan) or
 * HCMS_ERR_CAPACITY (cap too small; nothing written).
 */
HCMS_API int hcms_plan(int n_chunks, int mode, hcms_op *ops, int cap);

/*
 * The plan HCMS_MODE_AUTO runs: attention of chunk c launches
 * W_c = ceil(S / Br) * H_c workgroups, of which n_cu * B run at once (Br and
 * B the attention tiling for head dimension d: 256 queries and one workgroup
 * per CU for d = 128, 128 and two for d = 64).  One lane takes
 * sum_c ceil(W_c / (n_cu * B)) rounds of workgroups; two lanes pool them,
 * ceil(sum_c W_c / (n_cu * B)).  A launch's last round leaves
 * n_cu * B * ceil(W_c / (n_cu * B)) - W_c slots idle.  Returns
 * HCMS_MODE_SERIAL for one chunk; HCMS_MODE_LANES when pooling saves a round;
 * otherwise, for d = 128 with bf16 storage, HCMS_MODE_FUSED when some launch
 * leaves at least n_cu * B / 8 slots idle (where the neighbouring chunks'
 * copies ride) and HCMS_MODE_SERIAL when none does (the fused plan would run
 * the serial plan's launches); for the other kernels HCMS_MODE_INLINE when
 * chunk 0's launch leaves that many slots idle (where packs 1..C-1 run) and
 * HCMS_MODE_SERIAL otherwise.  Errors: HCMS_ERR_SHAPE (S < 0, d),
 * HCMS_ERR_DTYPE, HCMS_ERR_ARG (n_cu < 1), HCMS_ERR_NULL or HCMS_ERR_CHUNKS.
 * Host only.
 */
HCMS_API int hcms_auto_mode(int S, int d, int dtype, const int *chunk_sizes, int n_chunks,
                            int n_cu);

/*
 * Time model of HCMS (Sec. 3.7, Theorem of the optimal chunk count; appendix
 * equations of the HCMS time, the optimal chunk count and the speedup).
 * Host only; times in any one unit.
 *
 * hcms_model_time: T_hcms(C) = t0 + t_comm / C + t_attn + C * beta, the time
 *   of C chunks with fixed overhead t0 (projections), communication t_comm
 *   (here: the layout kernels), attention t_attn and per-chunk overhead beta.
 *   Errors: NULL, CHUNKS (C < 1), ARG (a time negative or not finite).
 * hcms_model_optimal_chunks: returns the integer C in [1, H] that minimises
 *   T_hcms (one of the two integers around C* = sqrt(t_comm / beta); ties go to
 *   fewer chunks; beta = 0 gives H) and writes C* itself to *c_real_out unless
 *   it is NULL.  Errors: SHAPE (H < 1), ARG.
 * hcms_model_speedup: S(C) = 1 / (1 - rho (C - 1) / C + C beta / T_total)
 *   with rho = t_comm / T_total in [0, 1].  Errors: NULL, CHUNKS, ARG (rho out
 *   of range, beta / T_total < 0, or a non-positive model time).
 * hcms_model_fit: least-squares fit of T(C) = a + t_comm / C + beta C to n >= 3
 *   measured (chunk count, time) pairs, giving a = t0 + t_attn.  Errors: NULL,
 *   CHUNKS (a count < 1), ARG (n < 3, a time not finite, or fewer than three
 *   distinct counts).
 */
HCMS_API int hcms_model_time(double t0, double t_comm, double t_attn, double beta, int n_chunks,
                             double *t_out);
HCMS_API int hcms_model_optimal_chunks(double t_comm, double beta, int H, double *c_real_out);
HCMS_API int hcms_model_speedup(double rho, double beta_over_total, int n_chunks, double *s_out);
HCMS_API int hcms_model_fit(const int *chunk_counts, const double *times, int n, double *a_out,
                            double *t_comm_out, double *beta_out);

/*
 * One-GPU extension of the time model (this library's, for the chunk-count
 * study of Sec. 3.7 and the adaptive chunk count the paper leaves as future
 * work, Sec. 6).  On one GPU the attention time depends on the chunking: a
 * launch of W workgroups on n slots (n = n_cu for d = 128, 2 n_cu for
 * d = 64) runs floor(W / n) full rounds and, when n does not divide W, a
 * partial round keeping a fraction f = (W mod n) / n of the slots busy,
 * which lasts t_round (g0 + (1 - g0) f) (the clock rises when part of the
 * chip idles; g0 = 1: a partial round costs a full one).  When the attention
 * kernel splits that round's tiles by key segments (hcms_forward's d = 128
 * bf16 launches: 3 rem <= n three ways, else 2 rem <= n two ways, with S of
 * 12 key blocks or more; in the lanes plan the last launch of each lane
 * splits the rem = sum W mod n tiles past the pooled rounds) the round holds
 * ways rem workgroups and lasts a third (three ways) or two thirds (two ways)
 * as long.  Every launch on the critical path adds `drain` rounds (its last
 * workgroups finish at different times).  Inputs measured on the device:
 * t_round (one full round of attention workgroups), g0 in (0, 1], drain >= 0,
 * t_copy (the layout kernel for one head of one tensor) and beta (one event
 * record or wait on the critical path).
 *
 * hcms_model_plan_time: model time of `mode` (a plan, or HCMS_MODE_AUTO for
 *   the plan hcms_auto_mode picks) on chunk_sizes:
 *     attention: the sum of the launches' rounds plus C drains
 *       (HCMS_MODE_LANES: the chunks' workgroups pooled into one launch's
 *       rounds, its partial round split as above, plus ceil(C / 2) drains),
 *       times t_round;
 *     copies on the critical path, in head-tensors times t_copy (a pack moves
 *       3 per head, an unpack 1): all 4 H in serial mode; otherwise chunk 0's
 *       pack and the last chunk's unpack, plus in fused mode the copies a
 *       launch with fewer than n / 8 idle slots cannot carry;
 *     synchronisations times beta: 0 (serial, fused), 4 (inline, lanes),
 *       2 C + 3 (pipelined, slots: the compute stream's wait and record per
 *       chunk, the fork and the join).
 *   With every launch filling whole rounds and equal chunks, the pipelined
 *   plan's time is the paper's T_hcms(C) with T_comm = 4 H t_copy, per-chunk
 *   overhead 2 beta + drain t_round and T_0 = 3 beta.
 *   Errors: NULL, SHAPE (S < 0, d), DTYPE, CHUNKS, ARG (mode; a time or drain
 *   negative or not finite; n_cu < 1; g0 outside (0, 1]).
 * hcms_choose_chunks: for C = 1 .. min(H, max_chunks), the chunk rule's sizes
 *   (hcms_default_chunks) in the plan HCMS_MODE_AUTO would run; writes the
 *   fastest under the model to sizes_out (room for min(H, max_chunks) ints),
 *   its plan to *mode_out and its model time to *t_out (either may be NULL),
 *   and returns its chunk count.  Ties go to fewer chunks.  Errors: as
 *   hcms_model_plan_time, plus SHAPE (H < 1) and CHUNKS (max_chunks < 1).
 * Host only.
 */
HCMS_API int hcms_model_plan_time(int S, int d, int dtype, const int *chunk_sizes, int n_chunks,
                                  int mode, int n_cu, double t_round, double g0, double drain,
                                  double t_copy, double beta, double *t_out);
HCMS_API int hcms_choose_chunks(int S, int H, int d, int dtype, int n_cu, double t_round,
                                double g0, double drain, double t_copy, double beta,
                                int max_chunks, int *sizes_out, int *mode_out, double *t_out);

typedef struct hcms_ctx hcms_ctx;

/*
 * Create a scheduler context bound to HIP device `device`: it owns the events
 * of up to `max_chunks` chunks (created once, reused by every call; the
 * device-level stream/event caching of Sec. 4.1), so hcms_forward creates
 * nothing.  Errors: NULL, ARG (device out of range), CHUNKS (max_chunks < 1),
 * HIP.
 */
HCMS_API int hcms_ctx_create(int device, int max_chunks, hcms_ctx **out);

/* The plan mode the context's last hcms_forward ran (HCMS_MODE_AUTO resolved;
   -1 before the first call), and the device's compute-unit count. */
HCMS_API int hcms_ctx_last_mode(const hcms_ctx *ctx);
HCMS_API int hcms_ctx_num_cu(const hcms_ctx *ctx);

/* Give hcms_backward a caller-owned score-gradient workspace (see
   hcms_attention_backward): `bytes` bytes at `ws`, 256-byte aligned, used as
   two regions of floor(bytes / 2) (rounded down to 256 bytes), one for the
   backward launches on the main stream and one for those on the compute
   stream, so that lanes mode can run two chunks at once.  A region smaller
   than one head's hcms_backward_ds_bytes leaves the path without it, in every
   mode.  ws NULL or bytes 0 removes it.  The memory must stay valid, and must
   not be touched by the caller, while a backward that uses it is pending.
   Errors: NULL (ctx), ARG (bytes < 0), ALIGN. */
HCMS_API int hcms_ctx_set_ds_workspace(hcms_ctx *ctx, void *ws, int64_t bytes);

/* Destroy a context (its events).  The caller must not destroy it while work
   that waits on its events is still pending.  NULL is accepted. */
HCMS_API int hcms_ctx_destroy(hcms_ctx *ctx);

/*
 * Per-kernel timing (for benchmarks).  hcms_ctx_set_timing(ctx, max_calls)
 * with max_calls > 0 makes the next max_calls hcms_forward calls bracket every
 * pack, attention and unpack launch with timing events on the stream that
 * runs it (events are created here, once; later calls are not timed);
 * max_calls = 0 turns timing off.  Each call resets the record.
 * hcms_ctx_kernel_ms waits for the recorded events and writes the durations in
 * milliseconds, call by call and chunk by chunk, in issue order.  In fused
 * mode a copy that rides in an attention launch reports that launch's time.
 *   kind : HCMS_OP_PACK, HCMS_OP_ATTENTION or HCMS_OP_UNPACK
 * Returns the number of durations written, HCMS_ERR_ARG (timing off / bad
 * kind / max_calls < 0), HCMS_ERR_CAPACITY or HCMS_ERR_HIP.
 */
HCMS_API int hcms_ctx_set_timing(hcms_ctx *ctx, int max_calls);
HCMS_API int hcms_ctx_kernel_ms(hcms_ctx *ctx, int kind, float *ms_out, int cap);

/*
 * The single-GPU share of one HCMS forward (Alg. 1 from SplitByHeads to the
 * final Concat): for every chunk c with heads [h0_c, h0_c + H_c),
 *   pack Q, K, V of the chunk into heads [h0_c, h0_c + H_c) of the head-major
 *   workspaces, run attention on them into o_hm, and unpack o_hm's chunk into
 *   the head slots [h0_c, h0_c + H_c) of o_seq,
 * scheduled as hcms_plan(n_chunks, mode) describes (HCMS_MODE_AUTO: the mode
 * hcms_auto_mode picks for the device's CU count).  Returns when everything
 * is enqueued; `main_stream` is ordered after all of it on return (no host
 * synchronisation).  All modes and all chunkings give bit-identical o_seq.
 *   q_seq, k_seq, v_seq, o_seq : device, [P][S/P][H][d]
 *   q_hm, k_hm, v_hm, o_hm     : device workspaces, [H][S][d] each
 *   lse                        : NULL, or [H][S] fp32: the attention's log2
 *                                softmax denominators (hcms_attention_lse), kept
 *                                for hcms_backward
 *   copy_stream, compute_stream: used in pipelined mode; must be distinct from
 *                                each other and from main_stream.  Inline mode
 *                                uses copy_stream only, lanes mode
 *                                compute_stream only (distinct from main);
 *                                fused mode uses neither.
 * Errors: as hcms_pack and hcms_attention, plus ARG (mode, stream reuse,
 * context of another device) and CHUNKS (n_chunks > the context's max_chunks).
 */
HCMS_API int hcms_forward(hcms_ctx *ctx,
                 const void *q_seq, const void *k_seq, const void *v_seq, void *o_seq,
                 void *q_hm, void *k_hm, void *v_hm, void *o_hm, float *lse,
                 int P, int S, int H, int d, float scale,
                 const int *chunk_sizes, int n_chunks, int dtype, int mode,
                 void *main_stream, void *copy_stream, void *compute_stream);

/*
 * hcms_forward with two chunk slots instead of full head-major workspaces
 * (the memory reduction of the chunked pipeline: only the chunks in flight
 * need a head-major copy).  q_slots, k_slots, v_slots, o_slots are device
 * buffers of [2][slot_heads][S][d] each; chunk c uses slot c % 2 (its heads
 * at the slot's start), so slot_heads must be at least every chunk size.
 * Modes: HCMS_MODE_SERIAL, HCMS_MODE_LANES, HCMS_MODE_SLOTS, HCMS_MODE_FUSED and
 * HCMS_MODE_AUTO (the mode hcms_auto_mode picks, serial in place of inline).  Pipelined and inline
 * modes would pack chunk c + 2 into chunk c's slot while its attention may
 * still run, and are rejected with HCMS_ERR_ARG.  No lse output: the backward
 * needs every head's head-major tensors.  o_seq is bit-identical to
 * hcms_forward's for the same inputs, whatever the mode and chunking.
 * Errors: as hcms_forward, plus CHUNKS (slot_heads < 1 or below a chunk size)
 * and ARG (mode).
 */
HCMS_API int hcms_forward_slots(hcms_ctx *ctx, const void *q_seq, const void *k_seq,
                                const void *v_seq, void *o_seq, void *q_slots, void *k_slots,
                                void *v_slots, void *o_slots, int slot_heads, int P, int S, int H,
                                int d, float scale, const int *chunk_sizes, int n_chunks, int dtype,
                                int mode, void *main_stream, void *copy_stream,
                                void *compute_stream);

/*
 * The backward of hcms_forward, for training: the reverse pipeline of the
 * chunked schedule.  Per chunk c, on the same plan as hcms_plan(n_chunks,
 * mode) (PACK, ATTENTION and UNPACK ops):
 *   PACK c      dout_seq's heads of chunk c into do_hm ([P][S/P][H][d] ->
 *               [H_c][S][d], the gradient's all-to-all to head shards);
 *   ATTENTION c hcms_attention_backward of the chunk into dq_hm, dk_hm,
 *               dv_hm (D into delta), with the context's score-gradient
 *               region of the stream it runs on, if any
 *               (hcms_ctx_set_ds_workspace);
 *   UNPACK c    dq_hm, dk_hm, dv_hm of chunk c into the head slots of
 *               dq_seq, dk_seq, dv_seq (the all-to-all back to sequence
 *               shards).
 *   q_hm, k_hm, v_hm, o_hm, lse : as hcms_forward (with lse) left them for the
 *                    same inputs, scale and d (any chunking)
 *   dout_seq         : dL/dO, [P][S/P][H][d]
 *   dq_seq, dk_seq, dv_seq : outputs, [P][S/P][H][d]
 *   do_hm, dq_hm, dk_hm, dv_hm : device workspaces, [H][S][d] each
 *   delta            : device workspace, [H][S] fp32
 * Streams and modes as hcms_forward; in fused mode the copies run right after
 * each chunk's backward launches (these carry none).  HCMS_MODE_AUTO runs lanes
 * when the context's score-gradient workspace applies and there are two chunks
 * or more (one chunk's HBM-bound dQ product then overlaps the next chunk's
 * key-parallel launch), else what hcms_auto_mode picks.  Every mode and
 * chunking gives bit-identical gradients.  Errors: as hcms_forward and
 * hcms_attention_backward.
 */
HCMS_API int hcms_backward(hcms_ctx *ctx, const void *dout_seq, void *dq_seq, void *dk_seq,
                           void *dv_seq, const void *q_hm, const void *k_hm, const void *v_hm,
                           const void *o_hm, const float *lse, void *do_hm, void *dq_hm,
                           void *dk_hm, void *dv_hm, float *delta, int P, int S, int H, int d,
                           float scale, const int *chunk_sizes, int n_chunks, int dtype, int mode,
                           void *main_stream, void *copy_stream, void *compute_stream);

/* ------------------------------------------------------------------------ */
/* Layer neighbours of the chunk loop: projections and rotary embedding      */
/* ------------------------------------------------------------------------ */

/*
 * Projection GEMM (the QKV projection before Alg. 1's split along heads and
 * the output projection after its Concat; Sec. 2 lists them in the Ulysses
 * layer):  y[m][n] = sum_k x[m][k] w[n][k],  i.e. y = x w^T.
 *   x : device, [M][K];  w : device, [N][K] (the weight stored [out][in]);
 *   y : device, [M][N], must not overlap x or w.
 * bf16 MFMA operands (fp32 storage is rounded to bf16 when loaded), fp32
 * accumulation, y rounded to the storage type.  Deterministic.
 * Requires K a positive multiple of 64 and at most 2^20, N a multiple of 8
 * and at most 2^20, M >= 0 (M = 0 or N = 0: nothing is enqueued).
 * Errors: NULL, SHAPE, DTYPE, ALIGN, ALIAS, HIP.
 */
HCMS_API int hcms_linear(const void *x, const void *w, void *y, int M, int N, int K, int dtype,
                         void *stream);

/*
 * Rotary position embedding on a latent grid (RoFormer's rotation, cited by
 * the paper in Sec. 2 for the Ulysses layer).  Token t of a sequence laid on
 * the row-major grid grid[0] x ... x grid[n_axes-1] (last axis fastest, e.g.
 * frames x rows x columns of video latents) has one coordinate c_a per axis.
 * The d/2 pairs (2i, 2i + 1) of a head vector form consecutive groups of
 * axis_pairs[a] pairs; pair i' of group a turns by the angle
 *   c_a * base^(-i' / axis_pairs[a])
 * mapping (x, y) to (x cos - y sin, x sin + y cos).  One axis is RoFormer's
 * one-dimensional position.
 *
 * hcms_rope_table_entries: the number E = sum_a grid[a] * axis_pairs[a] of
 *   (cos, sin) entries of the rotation table; host only.  Errors: NULL, ARG
 *   (n_axes not in 1..4), SHAPE (a size < 1, more than 2^31 - 1 tokens or
 *   2^28 entries).
 * hcms_rope_table: fills `table` (device, E pairs of fp32, 16-byte aligned)
 *   with the (cos, sin) of every axis, coordinate and pair, computed in fp64 and
 *   rounded to fp32.  Errors: as above, plus NULL, ALIGN and ARG (base not
 *   finite and > 1), HIP.
 */
HCMS_API int hcms_rope_table_entries(const int *grid, const int *axis_pairs, int n_axes);
HCMS_API int hcms_rope_table(float *table, const int *grid, const int *axis_pairs, int n_axes,
                             double base, void *stream);

/*
 * QKV projection with the split along heads and the rotary embedding fused:
 *   qkv[t][n] = sum_k x[t][k] w_qkv[n][k],  n = z H d + h d + e,
 *   q_seq[t][h][e] = qkv[t][0 H d + h d + e], k_seq likewise from z = 1,
 *   v_seq from z = 2, and, unless table is NULL, the pairs of q_seq[t][h] and
 *   k_seq[t][h] rotated for token t (hcms_rope_table on the same grid,
 *   axis_pairs, n_axes), in fp32 before the rounding to the storage type.
 *   x : device, [S][D];  w_qkv : device, [3 H d][D];
 *   q_seq, k_seq, v_seq : device, [S][H][d] each (the sequence-sharded
 *   [P][S/P][H][d] layout hcms_forward takes), disjoint from the inputs and
 *   each other.
 * Requires D as K of hcms_linear, d a positive multiple of 8, 3 H d <= 2^20,
 * and with a table: the grid's product = S, the pair counts' sum = d/2.
 * Errors: as hcms_linear and hcms_rope_table_entries, plus ALIAS for table.
 */
HCMS_API int hcms_qkv_projection(const void *x, const void *w_qkv, const float *table,
                                 const int *grid, const int *axis_pairs, int n_axes, void *q_seq,
                                 void *k_seq, void *v_seq, int S, int D, int H, int d, int dtype,
                                 void *stream);

/*
 * One attention layer around the HCMS chunk loop on one GPU: on main_stream
 * hcms_qkv_projection(x, w_qkv, table, ...) into q_seq, k_seq, v_seq; then
 * hcms_forward(ctx, q_seq, k_seq, v_seq, o_seq, q_hm, k_hm, v_hm, o_hm, NULL,
 * ...) in `mode`; then, on main_stream after the join,
 *   y[t][j] = sum_{h, e} o_seq[t][h][e] w_o[j][h d + e]
 * (hcms_linear of the concatenated heads, [S][H d], by w_o [D][H d]).
 *   y : device, [S][D].  Every other argument as in hcms_qkv_projection and
 *   hcms_forward; no output or workspace may overlap an input or y.
 * All modes and chunkings give bit-identical y.  Validation of all three
 * steps completes before anything is enqueued.
 */
HCMS_API int hcms_layer_forward(hcms_ctx *ctx, const void *x, const void *w_qkv, const void *w_o,
                                const float *table, const int *grid, const int *axis_pairs,
                                int n_axes, void *y, void *q_seq, void *k_seq, void *v_seq,
                                void *o_seq, void *q_hm, void *k_hm, void *v_hm, void *o_hm, int P,
                                int S, int D, int H, int d, float scale, const int *chunk_sizes,
                                int n_chunks, int dtype, int mode, void *main_stream,
                                void *copy_stream, void *compute_stream);

#ifdef __cplusplus
}
#endif

#endif /* HCMS_H */
