// C ABI of the HCMS single-GPU hot path: argument validation, the chunk
// scheduler (Alg. 1 as an op list plus an executor on HIP streams/events) and
// the event-caching context.  Declarations and the contract live in hcms.h.
#include "hcms.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <mutex>
#include <new>
#include <vector>

#include "hcms_internal.h"

namespace hcms {

namespace {
thread_local char g_last_error[512] = "";
}  // namespace

int fail(int status, const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    std::vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
    va_end(ap);
    return status;
}

int ok() {
    g_last_error[0] = '\0';
    return HCMS_OK;
}

const char *last_error() { return g_last_error; }

}  // namespace hcms

namespace {

using hcms::fail;
using hcms::ok;

int hip_fail(hipError_t e, const char *what) {
    return fail(HCMS_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

int elem_bytes(int dtype) { return dtype == HCMS_BF16 ? 2 : 4; }

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Byte ranges [a, a + na) and [b, b + nb) overlap.
bool overlaps(const void *a, int64_t na, const void *b, int64_t nb) {
    if (na <= 0 || nb <= 0) return false;
    const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
    return x < y + static_cast<uintptr_t>(nb) && y < x + static_cast<uintptr_t>(na);
}

int check_dtype(int dtype) {
    if (dtype != HCMS_BF16 && dtype != HCMS_FP32)
        return fail(HCMS_ERR_DTYPE, "dtype %d is neither HCMS_BF16 (0) nor HCMS_FP32 (1)", dtype);
    return HCMS_OK;
}

// S >= 0, H >= 1, P >= 1, S % P == 0, and the [S][H][d] tensor fits int64
// bytes and each head's [S][d] fits the 32-bit range of a buffer resource.
int check_dims(int P, int S, int H, int d, int dtype) {
    if (S < 0 || H < 1 || P < 1 || d < 1)
        return fail(HCMS_ERR_SHAPE, "need S >= 0, H >= 1, P >= 1, d >= 1 (S=%d H=%d P=%d d=%d)", S,
                    H, P, d);
    if (S % P != 0)
        return fail(HCMS_ERR_SHAPE, "S=%d is not a multiple of the shard count P=%d", S, P);
    const int64_t head_bytes = static_cast<int64_t>(S) * d * elem_bytes(dtype);
    if (head_bytes > 0x7fffffffLL)
        return fail(HCMS_ERR_SHAPE, "one head is %lld bytes; the limit is 2^31 - 1",
                    static_cast<long long>(head_bytes));
    return HCMS_OK;
}

// Pack / unpack rows are moved as 16-byte units: d * elem must be 16 << k.
int row_log2_units(int d, int dtype, int *log2_units) {
    const int row = d * elem_bytes(dtype);
    for (int k = 0; k <= 6; ++k)
        if (row == (16 << k)) {
            *log2_units = k;
            return HCMS_OK;
        }
    return fail(HCMS_ERR_SHAPE,
                "pack/unpack need d * element size in {16, 32, ..., 1024} bytes (d=%d, %d bytes)", d,
                row);
}

int check_chunks(int H, const int *sizes, int n) {
    if (!sizes) return fail(HCMS_ERR_NULL, "chunk_sizes is NULL");
    if (n < 1 || n > H) return fail(HCMS_ERR_CHUNKS, "n_chunks=%d must be in [1, H=%d]", n, H);
    int64_t sum = 0;
    for (int c = 0; c < n; ++c) {
        if (sizes[c] < 1) return fail(HCMS_ERR_CHUNKS, "chunk %d has %d heads", c, sizes[c]);
        sum += sizes[c];
    }
    if (sum != H)
        return fail(HCMS_ERR_CHUNKS, "chunk sizes sum to %lld, not H=%d", static_cast<long long>(sum), H);
    return HCMS_OK;
}

int check_scale(float scale) {
    if (!std::isfinite(scale) || !(scale > 0.0f))
        return fail(HCMS_ERR_ARG, "scale must be finite and > 0 (got %g)", static_cast<double>(scale));
    return HCMS_OK;
}

int check_pack_args(const void *a, const void *b, int P, int S, int H, int d, int h_begin,
                    int h_count, int dtype, int *log2_units) {
    int st;
    if (S > 0 && (!a || !b)) return fail(HCMS_ERR_NULL, "source or destination is NULL");
    if ((st = check_dtype(dtype)) != HCMS_OK) return st;
    if ((st = check_dims(P, S, H, d, dtype)) != HCMS_OK) return st;
    if ((st = row_log2_units(d, dtype, log2_units)) != HCMS_OK) return st;
    if (h_begin < 0 || h_count < 1 || h_begin > H - h_count)
        return fail(HCMS_ERR_CHUNKS, "head range [%d, %d + %d) is not inside [0, H=%d)", h_begin,
                    h_begin, h_count, H);
    if (!aligned16(a) || !aligned16(b)) return fail(HCMS_ERR_ALIGN, "buffers must be 16-byte aligned");
    const int64_t es = elem_bytes(dtype);
    const int64_t seq_bytes = static_cast<int64_t>(S) * H * d * es;
    const int64_t hm_bytes = static_cast<int64_t>(S) * h_count * d * es;
    if (overlaps(a, seq_bytes, b, hm_bytes) || overlaps(a, hm_bytes, b, seq_bytes))
        return fail(HCMS_ERR_ALIAS, "source and destination overlap");
    return HCMS_OK;
}

// ---------------------------------------------------------------------------
// Plan (Alg. 1 as an op list)
// ---------------------------------------------------------------------------
struct PlanWriter {
    hcms_op *ops;
    int cap;
    int n = 0;
    void put(int kind, int stream, int chunk, int event) {
        if (ops && n < cap) ops[n] = hcms_op{kind, stream, chunk, event};
        ++n;
    }
};

void serial_plan(int C, PlanWriter &w) {
    for (int c = 0; c < C; ++c) {
        w.put(HCMS_OP_PACK, HCMS_STREAM_MAIN, c, -1);
        w.put(HCMS_OP_ATTENTION, HCMS_STREAM_MAIN, c, -1);
        w.put(HCMS_OP_UNPACK, HCMS_STREAM_MAIN, c, -1);
    }
}

// Alg. 1 in its printed issue order.
void alg1_plan(int C, PlanWriter &w) {
    const int e_main = 0, e_done = 1 + 2 * C;
    auto e_pack = [](int c) { return 1 + c; };
    auto e_attn = [C](int c) { return 1 + C + c; };
    // Main stream: fork.
    w.put(HCMS_OP_RECORD, HCMS_STREAM_MAIN, -1, e_main);
    // Copy stream: input layout of every chunk.
    w.put(HCMS_OP_WAIT, HCMS_STREAM_COPY, -1, e_main);
    for (int c = 0; c < C; ++c) {
        w.put(HCMS_OP_PACK, HCMS_STREAM_COPY, c, -1);
        w.put(HCMS_OP_RECORD, HCMS_STREAM_COPY, -1, e_pack(c));
    }
    // Compute stream: attention of chunk c as soon as its inputs are laid out.
    w.put(HCMS_OP_WAIT, HCMS_STREAM_COMPUTE, -1, e_main);
    for (int c = 0; c < C; ++c) {
        w.put(HCMS_OP_WAIT, HCMS_STREAM_COMPUTE, -1, e_pack(c));
        w.put(HCMS_OP_ATTENTION, HCMS_STREAM_COMPUTE, c, -1);
        w.put(HCMS_OP_RECORD, HCMS_STREAM_COMPUTE, -1, e_attn(c));
    }
    // Copy stream: output layout of chunk c once its attention is done.
    for (int c = 0; c < C; ++c) {
        w.put(HCMS_OP_WAIT, HCMS_STREAM_COPY, -1, e_attn(c));
        w.put(HCMS_OP_UNPACK, HCMS_STREAM_COPY, c, -1);
    }
    // Join: the main stream is ordered after the last unpack, which is itself
    // ordered after the last attention.
    w.put(HCMS_OP_RECORD, HCMS_STREAM_COPY, -1, e_done);
    w.put(HCMS_OP_WAIT, HCMS_STREAM_MAIN, -1, e_done);
}

// One lane with the fewest stream synchronisations, for one GPU.  On one GPU
// a pack or unpack costs a few hundred times less than a chunk's attention,
// and every event record or wait on the critical path costs a few
// microseconds, about as much as the copies it hides.  So:
//  - attention runs on the main stream (no fork or join of a third stream);
//  - chunk 0's pack, which nothing can hide, runs in front of its attention,
//    and the last chunk's unpack after its attention, on the same stream;
//  - the copy stream starts after chunk 0's pack and packs chunks 1..C-1 while
//    attention 0 runs; attention 1 waits once for all of them (E_{C-1}^pack;
//    the copy stream runs them in order);
//  - unpacks 0..C-2 wait once for attention C-2 (E_{C-2}^attn) and run while
//    attention C-1 does; the main stream waits E_done after the last unpack.
// Every pack c -> attention c -> unpack c dependency of Alg. 1 holds, with
// four synchronisations on the main stream whatever C is.
void inline_plan(int C, PlanWriter &w) {
    if (C == 1) return serial_plan(C, w);
    const int e_done = 1 + 2 * C;
    auto e_pack = [](int c) { return 1 + c; };
    auto e_attn = [C](int c) { return 1 + C + c; };
    w.put(HCMS_OP_PACK, HCMS_STREAM_MAIN, 0, -1);
    w.put(HCMS_OP_RECORD, HCMS_STREAM_MAIN, -1, e_pack(0));
    w.put(HCMS_OP_WAIT, HCMS_STREAM_COPY, -1, e_pack(0));
    for (int c = 1; c < C; ++c) w.put(HCMS_OP_PACK, HCMS_STREAM_COPY, c, -1);
    w.put(HCMS_OP_RECORD, HCMS_STREAM_COPY, -1, e_pack(C - 1));
    for (int c = 0; c < C; ++c) {
        if (c == C - 1) w.put(HCMS_OP_RECORD, HCMS_STREAM_MAIN, -1, e_attn(C - 2));
        if (c == 1) w.put(HCMS_OP_WAIT, HCMS_STREAM_MAIN, -1, e_pack(C - 1));
        w.put(HCMS_OP_ATTENTION, HCMS_STREAM_MAIN, c, -1);
    }
    w.put(HCMS_OP_WAIT, HCMS_STREAM_COPY, -1, e_attn(C - 2));
    for (int c = 0; c < C - 1; ++c) w.put(HCMS_OP_UNPACK, HCMS_STREAM_COPY, c, -1);
    w.put(HCMS_OP_RECORD, HCMS_STREAM_COPY, -1, e_done);
    w.put(HCMS_OP_UNPACK, HCMS_STREAM_MAIN, C - 1, -1);
    w.put(HCMS_OP_WAIT, HCMS_STREAM_MAIN, -1, e_done);
}

// Two lanes, for one GPU.  Chunks alternate between the main stream (even c)
// and the compute stream (odd c); each lane runs pack c, attention c, unpack c
// in order.  No chunk depends on another (the lemma of no inter-chunk
// dependency), so the lanes only meet at the fork and the join.  One lane's
// copies run beside the other lane's attention, and, which matters more on
// one GPU, a chunk's attention launch leaves CUs idle in its last round of
// workgroups that the other lane's attention fills.  The second lane starts
// after chunk 0's pack (E_0^pack) so that its first pack does not take
// bandwidth from the pack attention 0 waits for; the main stream waits E_done,
// recorded at the end of the second lane.  Four synchronisations in all,
// whatever C is.  One chunk has nothing to overlap: its plan is the serial one.
void lanes_plan(int C, PlanWriter &w) {
    if (C == 1) return serial_plan(C, w);
    const int e_pack0 = 1, e_done = 1 + 2 * C;
    auto chunk = [&](int c) {
        const int s = (c & 1) ? HCMS_STREAM_COMPUTE : HCMS_STREAM_MAIN;
        w.put(HCMS_OP_PACK, s, c, -1);
        if (c == 0) w.put(HCMS_OP_RECORD, s, -1, e_pack0);
        w.put(HCMS_OP_ATTENTION, s, c, -1);
        w.put(HCMS_OP_UNPACK, s, c, -1);
    };
    chunk(0);
    w.put(HCMS_OP_WAIT, HCMS_STREAM_COMPUTE, -1, e_pack0);
    for (int c = 1; c < C; ++c) chunk(c);
    w.put(HCMS_OP_RECORD, HCMS_STREAM_COMPUTE, -1, e_done);
    w.put(HCMS_OP_WAIT, HCMS_STREAM_MAIN, -1, e_done);
}

// The copy stream interleaved with the attentions, for chunk slots that are
// reused: Alg. 1's streams and events, but after attention c the copy stream
// unpacks c and then packs c + 2 (which reuses chunk c's slot; attention c + 2
// therefore also comes after unpack c, which freed the output slot).  This is
// the overlap of Sec. 3.5 -- the input layout of one chunk and the output
// layout of another beside a chunk's attention -- in an order that needs only
// two chunks' worth of head-major workspace.  The host issues every record
// before any wait on it: the compute stream's ops of chunk c come before the
// copy stream's ops that follow attention c.
void slots_plan(int C, PlanWriter &w) {
    const int e_main = 0, e_done = 1 + 2 * C;
    auto e_pack = [](int c) { return 1 + c; };
    auto e_attn = [C](int c) { return 1 + C + c; };
    w.put(HCMS_OP_RECORD, HCMS_STREAM_MAIN, -1, e_main);
    w.put(HCMS_OP_WAIT, HCMS_STREAM_COPY, -1, e_main);
    for (int c = 0; c < C && c < 2; ++c) {
        w.put(HCMS_OP_PACK, HCMS_STREAM_COPY, c, -1);
        w.put(HCMS_OP_RECORD, HCMS_STREAM_COPY, -1, e_pack(c));
    }
    w.put(HCMS_OP_WAIT, HCMS_STREAM_COMPUTE, -1, e_main);
    for (int c = 0; c < C; ++c) {
        w.put(HCMS_OP_WAIT, HCMS_STREAM_COMPUTE, -1, e_pack(c));
        w.put(HCMS_OP_ATTENTION, HCMS_STREAM_COMPUTE, c, -1);
        w.put(HCMS_OP_RECORD, HCMS_STREAM_COMPUTE, -1, e_attn(c));
        w.put(HCMS_OP_WAIT, HCMS_STREAM_COPY, -1, e_attn(c));
        w.put(HCMS_OP_UNPACK, HCMS_STREAM_COPY, c, -1);
        if (c + 2 < C) {
            w.put(HCMS_OP_PACK, HCMS_STREAM_COPY, c + 2, -1);
            w.put(HCMS_OP_RECORD, HCMS_STREAM_COPY, -1, e_pack(c + 2));
        }
    }
    w.put(HCMS_OP_RECORD, HCMS_STREAM_COPY, -1, e_done);
    w.put(HCMS_OP_WAIT, HCMS_STREAM_MAIN, -1, e_done);
}

// One stream and no events, for one GPU.  The pack of chunk c + 1 and the
// unpack of chunk c - 1 ride in the launch of attention c as extra
// workgroups, dispatched after all of its attention workgroups, so they run
// on the CUs the launch's last round leaves idle.  Stream order gives every
// dependency of Alg. 1: pack c + 1 (in launch c) comes before attention c + 1
// (launch c + 1), unpack c - 1 (in launch c) after attention c - 1 (launch
// c - 1); and nothing in one launch touches the bytes of another op of the
// same launch (chunk c's workspace heads, chunk c + 1's, chunk c - 1's output
// rows).  Chunk 0's pack and the last unpack stay on the main stream.  The
// copies a launch cannot carry run right after it (see hcms.h).
void fused_plan(int C, PlanWriter &w) {
    if (C == 1) return serial_plan(C, w);
    w.put(HCMS_OP_PACK, HCMS_STREAM_MAIN, 0, -1);
    for (int c = 0; c < C; ++c) {
        if (c + 1 < C) w.put(HCMS_OP_PACK, HCMS_STREAM_IN_ATTENTION, c + 1, -1);
        if (c >= 1) w.put(HCMS_OP_UNPACK, HCMS_STREAM_IN_ATTENTION, c - 1, -1);
        w.put(HCMS_OP_ATTENTION, HCMS_STREAM_MAIN, c, -1);
    }
    w.put(HCMS_OP_UNPACK, HCMS_STREAM_MAIN, C - 1, -1);
}

// Modes with a fixed plan (hcms_plan); HCMS_MODE_AUTO resolves to one of
// them per call.
bool plan_mode(int mode) {
    return mode == HCMS_MODE_SERIAL || mode == HCMS_MODE_PIPELINED ||
           mode == HCMS_MODE_INLINE || mode == HCMS_MODE_LANES || mode == HCMS_MODE_SLOTS ||
           mode == HCMS_MODE_FUSED;
}

int build_plan(int C, int mode, PlanWriter &w) {
    if (mode == HCMS_MODE_SERIAL) serial_plan(C, w);
    else if (mode == HCMS_MODE_PIPELINED) alg1_plan(C, w);
    else if (mode == HCMS_MODE_INLINE) inline_plan(C, w);
    else if (mode == HCMS_MODE_SLOTS) slots_plan(C, w);
    else if (mode == HCMS_MODE_FUSED) fused_plan(C, w);
    else lanes_plan(C, w);
    return w.n;
}

int plan_size(int C, int mode) {
    if (mode == HCMS_MODE_PIPELINED || mode == HCMS_MODE_SLOTS) return 7 * C + 5;
    if (mode == HCMS_MODE_SERIAL || mode == HCMS_MODE_FUSED || C == 1) return 3 * C;
    return mode == HCMS_MODE_INLINE ? 3 * C + 8 : 3 * C + 4;
}

// Rounds of attention workgroups: a launch of W workgroups on `slots`
// concurrent slots takes ceil(W / slots) rounds; two lanes pool the chunks.
// When pooling saves no round, the launches that can carry the neighbouring
// chunks' copies (d = 128, bf16 storage) run the fused plan, the others the
// inline one.
}  // namespace

// The plan HCMS_MODE_AUTO runs (hcms_auto_mode without validation).
int hcms::auto_plan(int S, int d, int dtype, const int *sizes, int C, int n_cu) {
    if (C == 1) return HCMS_MODE_SERIAL;
    const int64_t br = hcms::attention_queries_per_block(d);
    const int64_t slots = static_cast<int64_t>(n_cu) * hcms::attention_blocks_per_cu(d);
    const int64_t tiles = (S + br - 1) / br;
    int64_t rounds = 0, total = 0;
    bool some_idle = false;       // a launch whose last round leaves enough slots idle
    bool first_idle = false;      // ... for chunk 0's launch in particular
    for (int c = 0; c < C; ++c) {
        const int64_t wc = tiles * sizes[c];
        rounds += (wc + slots - 1) / slots;
        total += wc;
        // The workgroups the launch runs: its last round's tiles may be split.
        const int64_t rem = wc % slots;
        const int64_t run = wc - rem + rem * hcms::attention_split_ways(wc, S, d, dtype, n_cu);
        const int64_t idle = (slots - run % slots) % slots;
        const bool enough = idle >= std::max<int64_t>(1, slots / 8);
        some_idle = some_idle || enough;
        if (c == 0) first_idle = enough;
    }
    // Two lanes pool the chunks' partial rounds: a whole round saved.
    if (rounds > (total + slots - 1) / slots) return HCMS_MODE_LANES;
    // The fused plan moves copies only on CUs a launch's last round leaves
    // idle; with none anywhere it would run the serial plan's launches.
    if (d == 128 && dtype == HCMS_BF16) return some_idle ? HCMS_MODE_FUSED : HCMS_MODE_SERIAL;
    // The inline plan pays four synchronisations to run packs 1..C-1 beside
    // attention 0's last round: only worth it when that round has idle CUs.
    return first_idle ? HCMS_MODE_INLINE : HCMS_MODE_SERIAL;
}

namespace {

int auto_mode(int S, int d, int dtype, const int *sizes, int C, int n_cu) {
    return hcms::auto_plan(S, d, dtype, sizes, C, n_cu);
}

// Saves the current device, switches to `dev`, restores on scope exit.
struct DeviceGuard {
    int prev = -1;
    hipError_t err = hipSuccess;
    explicit DeviceGuard(int dev) {
        err = hipGetDevice(&prev);
        if (err == hipSuccess && prev != dev) err = hipSetDevice(dev);
    }
    ~DeviceGuard() {
        int cur = -1;
        if (prev >= 0 && hipGetDevice(&cur) == hipSuccess && cur != prev) (void)hipSetDevice(prev);
    }
};

}  // namespace

namespace {

float scale_log2e(float scale) {
    return static_cast<float>(static_cast<double>(scale) * 1.4426950408889634);
}

// One attention launch per chunk, in order, on `stream`; lse (optional) is
// [H][S] fp32 and advances with the chunk's first head.
int run_attention(const void *q, const void *k, const void *v, void *out, float *lse, int S, int d,
                  float scale, const int *chunk_sizes, int n_chunks, int dtype, hipStream_t stream) {
    const int64_t head = static_cast<int64_t>(S) * d * elem_bytes(dtype);
    const float c = scale_log2e(scale);
    int h0 = 0;
    for (int i = 0; i < n_chunks; ++i) {
        const int64_t off = head * h0;
        const hipError_t e = hcms::launch_attention(
            static_cast<const char *>(q) + off, static_cast<const char *>(k) + off,
            static_cast<const char *>(v) + off, static_cast<char *>(out) + off,
            lse ? lse + static_cast<int64_t>(h0) * S : nullptr, S, chunk_sizes[i], d, c, dtype,
            nullptr, stream);
        if (e != hipSuccess) return hip_fail(e, "attention launch");
        h0 += chunk_sizes[i];
    }
    return ok();
}

// A [H][S] fp32 statistics buffer: non-NULL unless S = 0, 4-byte aligned, and
// disjoint from the four [H][S][d] tensors.
int check_stats(const float *p, const char *name, int S, int H, const void *a, const void *b,
                const void *c, const void *d_, int d, int dtype) {
    if (S == 0) return HCMS_OK;
    if (!p) return fail(HCMS_ERR_NULL, "%s is NULL", name);
    if ((reinterpret_cast<uintptr_t>(p) & 3u) != 0)
        return fail(HCMS_ERR_ALIGN, "%s must be 4-byte aligned", name);
    const int64_t sb = static_cast<int64_t>(S) * H * 4;
    const int64_t tb = static_cast<int64_t>(S) * H * d * elem_bytes(dtype);
    for (const void *t : {a, b, c, d_})
        if (overlaps(p, sb, t, tb)) return fail(HCMS_ERR_ALIAS, "%s overlaps a tensor", name);
    return HCMS_OK;
}

}  // namespace

struct hcms_ctx {
    int device = 0;
    int max_chunks = 0;
    int n_cu = 0;                        // compute units of the device
    int last_mode = -1;                  // plan mode of the last hcms_forward
    std::vector<hipEvent_t> events;      // 2 * max_chunks + 2 sync events
    std::vector<hcms_op> plan;           // scratch for the op list
    int timing_calls = 0;                // calls to time (0 = off)
    std::vector<hipEvent_t> t_begin;     // [call][kind][chunk] timing events
    std::vector<hipEvent_t> t_end;
    std::vector<int> timed_chunks;       // chunk count of each timed call
    // Scratch that lets an attention launch split its last round of tiles:
    // one region for launches on the main stream, one for the compute stream
    // (launches on one stream are ordered, so each region serves one launch
    // at a time).  No region: every tile whole, with the same results.
    void *split_mem = nullptr;
    hcms::SplitScratch split[2] = {};
    // Caller-owned score-gradient workspace of hcms_backward: two regions of
    // ds_region bytes, one for backward launches on the main stream, one for
    // those on the compute stream (NULL: none).
    char *ds = nullptr;
    int64_t ds_region = 0;
};

namespace {

// Validation shared by hcms_forward and hcms_backward; resolves
// HCMS_MODE_AUTO into *mode and returns the row size's log2 unit count.
int check_schedule(hcms_ctx *ctx, int P, int S, int H, int d, float scale, const int *chunk_sizes,
                   int n_chunks, int dtype, int *mode, int *log2u, void *main_stream,
                   void *copy_stream, void *compute_stream, bool slotted = false,
                   bool prefer_lanes = false) {
    int st;
    const int m = *mode;
    if (!plan_mode(m) && m != HCMS_MODE_AUTO)
        return fail(HCMS_ERR_ARG, "mode %d is not serial (0), pipelined (1), inline (2), lanes (3), "
                    "auto (4), slots (5) or fused (6)", m);
    if (slotted && (m == HCMS_MODE_PIPELINED || m == HCMS_MODE_INLINE))
        return fail(HCMS_ERR_ARG, "mode %d packs chunk c + 2 before chunk c's attention is done; "
                    "with two chunk slots use serial, lanes, slots, fused or auto", m);
    if ((st = check_dtype(dtype)) != HCMS_OK) return st;
    if ((st = check_dims(P, S, H, d, dtype)) != HCMS_OK) return st;
    if ((st = row_log2_units(d, dtype, log2u)) != HCMS_OK) return st;
    if (d != 64 && d != 128) return fail(HCMS_ERR_SHAPE, "attention supports d = 64 or 128 (got %d)", d);
    if ((st = check_chunks(H, chunk_sizes, n_chunks)) != HCMS_OK) return st;
    if (n_chunks > ctx->max_chunks)
        return fail(HCMS_ERR_CHUNKS, "n_chunks=%d exceeds the context's max_chunks=%d", n_chunks,
                    ctx->max_chunks);
    if ((st = check_scale(scale)) != HCMS_OK) return st;
    if ((m == HCMS_MODE_PIPELINED || m == HCMS_MODE_SLOTS) &&
        (copy_stream == compute_stream || copy_stream == main_stream || compute_stream == main_stream))
        return fail(HCMS_ERR_ARG, "pipelined and slots modes need three distinct streams");
    int r = m == HCMS_MODE_AUTO ? auto_mode(S, d, dtype, chunk_sizes, n_chunks, ctx->n_cu) : m;
    // The backward with stored score gradients: one chunk's HBM-bound dQ
    // product overlaps the next chunk's key-parallel launch in lanes.
    if (m == HCMS_MODE_AUTO && prefer_lanes && n_chunks >= 2 && compute_stream != main_stream)
        r = HCMS_MODE_LANES;
    // With two chunk slots the one-lane plan with few synchronisations is not
    // available; auto then runs the serial plan (lanes when it saves a round).
    if (slotted && m == HCMS_MODE_AUTO && r == HCMS_MODE_INLINE) r = HCMS_MODE_SERIAL;
    if (r == HCMS_MODE_INLINE && copy_stream == main_stream)
        return fail(HCMS_ERR_ARG, "inline mode needs a copy stream distinct from the main stream");
    if (r == HCMS_MODE_LANES && compute_stream == main_stream)
        return fail(HCMS_ERR_ARG, "lanes mode needs a compute stream distinct from the main stream");
    int cur_dev = -1;
    const hipError_t e = hipGetDevice(&cur_dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (cur_dev != ctx->device)
        return fail(HCMS_ERR_ARG, "context is bound to device %d, current device is %d", ctx->device,
                    cur_dev);
    *mode = r;
    return HCMS_OK;
}

// A copy op of the fused plan waiting for the attention launch it rides in.
struct RiderOp {
    int kind, chunk, h0, hc;
};

// Issues the plan of `mode` (already resolved): RECORD / WAIT ops on the
// context's events, kernel ops through launch(kind, chunk, h0, h_count, stream),
// each bracketed by timing events while the context records.  Ops on
// HCMS_STREAM_IN_ATTENTION are collected and handed to the next ATTENTION op
// through ride(chunk, h0, h_count, stream, riders, n, &riding); when that
// launch cannot carry them (riding false) they are launched right after it.
// A copy that rides reports the time of the launch it rode in.
template <typename Launch, typename Ride>
int execute_plan(hcms_ctx *ctx, int mode, const int *chunk_sizes, int C, void *main_stream,
                 void *copy_stream, void *compute_stream, Launch &&launch, Ride &&ride) {
    PlanWriter w{ctx->plan.data(), static_cast<int>(ctx->plan.size())};
    const int n_ops = build_plan(C, mode, w);
    ctx->last_mode = mode;
    hipStream_t streams[3] = {static_cast<hipStream_t>(main_stream),
                              static_cast<hipStream_t>(copy_stream),
                              static_cast<hipStream_t>(compute_stream)};
    std::vector<int> offs(C + 1, 0);
    for (int c = 0; c < C; ++c) offs[c + 1] = offs[c] + chunk_sizes[c];
    // Sync event id -> ctx event (ids: 0 E_main, 1..C E_pack, C+1..2C E_attn,
    // 2C+1 E_done; the context keeps max_chunks of each kind).
    auto event_of = [&](int id) -> hipEvent_t {
        if (id == 0) return ctx->events[0];
        if (id <= C) return ctx->events[id];
        if (id <= 2 * C) return ctx->events[1 + ctx->max_chunks + (id - 1 - C)];
        return ctx->events[1 + 2 * ctx->max_chunks];
    };
    const bool timed = static_cast<int>(ctx->timed_chunks.size()) < ctx->timing_calls;
    const size_t call = ctx->timed_chunks.size();
    hipError_t e;
    auto slot_of = [&](int kind, int c) {
        return (call * 3 + (kind - HCMS_OP_PACK)) * ctx->max_chunks + c;
    };
    RiderOp riders[2];
    int n_riders = 0;
    for (int i = 0; i < n_ops; ++i) {
        const hcms_op &op = ctx->plan[i];
        if (op.stream == HCMS_STREAM_IN_ATTENTION) {
            if (n_riders == 2) return fail(HCMS_ERR_ARG, "more than two copies ride in one launch");
            riders[n_riders++] = RiderOp{op.kind, op.chunk, offs[op.chunk], chunk_sizes[op.chunk]};
            continue;
        }
        hipStream_t s = streams[op.stream];
        if (op.kind == HCMS_OP_RECORD) {
            if ((e = hipEventRecord(event_of(op.event), s)) != hipSuccess)
                return hip_fail(e, "hipEventRecord");
            continue;
        }
        if (op.kind == HCMS_OP_WAIT) {
            if ((e = hipStreamWaitEvent(s, event_of(op.event), 0)) != hipSuccess)
                return hip_fail(e, "hipStreamWaitEvent");
            continue;
        }
        const int c = op.chunk;
        const int n_ride = op.kind == HCMS_OP_ATTENTION ? n_riders : 0;
        if (timed) {
            if ((e = hipEventRecord(ctx->t_begin[slot_of(op.kind, c)], s)) != hipSuccess)
                return hip_fail(e, "hipEventRecord");
            for (int r = 0; r < n_ride; ++r)
                if ((e = hipEventRecord(ctx->t_begin[slot_of(riders[r].kind, riders[r].chunk)], s)) !=
                    hipSuccess)
                    return hip_fail(e, "hipEventRecord");
        }
        bool riding = false;
        if (n_ride > 0) e = ride(c, offs[c], chunk_sizes[c], s, riders, n_ride, &riding);
        else e = launch(op.kind, c, offs[c], chunk_sizes[c], s);
        if (e != hipSuccess) return hip_fail(e, "kernel launch");
        if (timed) {
            if ((e = hipEventRecord(ctx->t_end[slot_of(op.kind, c)], s)) != hipSuccess)
                return hip_fail(e, "hipEventRecord");
            for (int r = 0; riding && r < n_ride; ++r)
                if ((e = hipEventRecord(ctx->t_end[slot_of(riders[r].kind, riders[r].chunk)], s)) !=
                    hipSuccess)
                    return hip_fail(e, "hipEventRecord");
        }
        for (int r = 0; !riding && r < n_ride; ++r) {
            const RiderOp &ro = riders[r];
            if (timed && (e = hipEventRecord(ctx->t_begin[slot_of(ro.kind, ro.chunk)], s)) != hipSuccess)
                return hip_fail(e, "hipEventRecord");
            if ((e = launch(ro.kind, ro.chunk, ro.h0, ro.hc, s)) != hipSuccess)
                return hip_fail(e, "kernel launch");
            if (timed && (e = hipEventRecord(ctx->t_end[slot_of(ro.kind, ro.chunk)], s)) != hipSuccess)
                return hip_fail(e, "hipEventRecord");
        }
        if (op.kind == HCMS_OP_ATTENTION) n_riders = 0;
    }
    if (n_riders != 0) return fail(HCMS_ERR_ARG, "a riding copy has no attention launch after it");
    if (timed) ctx->timed_chunks.push_back(C);
    return ok();
}

// Arguments of one hcms_forward call.
struct ForwardArgs {
    hcms_ctx *ctx;
    const void *q_seq, *k_seq, *v_seq;
    void *o_seq, *q_hm, *k_hm, *v_hm, *o_hm;
    float *lse;
    int P, S, H, d;
    float scale;
    const int *chunk_sizes;
    int n_chunks, dtype, mode;
    void *main_stream, *copy_stream, *compute_stream;
    int slot_heads = 0;  // 0: workspaces of H heads; else two slots of slot_heads heads
};

// Everything hcms_forward validates; resolves the mode and the row unit.
int check_forward(const ForwardArgs &f, int *mode, int *log2u) {
    int st;
    if (!f.ctx) return fail(HCMS_ERR_NULL, "ctx is NULL");
    if (f.S > 0 && (!f.q_seq || !f.k_seq || !f.v_seq || !f.o_seq || !f.q_hm || !f.k_hm || !f.v_hm ||
                    !f.o_hm))
        return fail(HCMS_ERR_NULL, "a tensor pointer is NULL");
    if ((st = check_schedule(f.ctx, f.P, f.S, f.H, f.d, f.scale, f.chunk_sizes, f.n_chunks, f.dtype,
                             mode, log2u, f.main_stream, f.copy_stream, f.compute_stream,
                             f.slot_heads > 0)) != HCMS_OK)
        return st;
    if (f.slot_heads > 0)
        for (int c = 0; c < f.n_chunks; ++c)
            if (f.chunk_sizes[c] > f.slot_heads)
                return fail(HCMS_ERR_CHUNKS, "chunk %d has %d heads, a slot holds %d", c,
                            f.chunk_sizes[c], f.slot_heads);
    const void *all[8] = {f.q_seq, f.k_seq, f.v_seq, f.o_seq, f.q_hm, f.k_hm, f.v_hm, f.o_hm};
    for (const void *p : all)
        if (f.S > 0 && !aligned16(p)) return fail(HCMS_ERR_ALIGN, "buffers must be 16-byte aligned");
    const int64_t bytes = static_cast<int64_t>(f.S) * f.H * f.d * elem_bytes(f.dtype);
    const int64_t ws_bytes = f.slot_heads > 0
        ? static_cast<int64_t>(2) * f.slot_heads * f.S * f.d * elem_bytes(f.dtype) : bytes;
    for (int i = 0; i < 8; ++i)
        for (int j = i + 1; j < 8; ++j) {
            // Inputs may alias each other (read-only); everything else must not.
            const bool both_inputs = i < 3 && j < 3;
            if (!both_inputs && overlaps(all[i], i < 4 ? bytes : ws_bytes, all[j],
                                         j < 4 ? bytes : ws_bytes))
                return fail(HCMS_ERR_ALIAS, "tensor %d overlaps tensor %d", i, j);
        }
    if (f.lse) {
        if ((st = check_stats(f.lse, "lse", f.S, f.H, f.q_hm, f.k_hm, f.v_hm, f.o_hm, f.d, f.dtype)) !=
            HCMS_OK)
            return st;
        if ((st = check_stats(f.lse, "lse", f.S, f.H, f.q_seq, f.k_seq, f.v_seq, f.o_seq, f.d,
                              f.dtype)) != HCMS_OK)
            return st;
    }
    return HCMS_OK;
}

// LDS reservation of a chunk's copy.  In the inline schedule the copy
// stream's packs (chunks 1..C-1) run beside attention 0 and its unpacks
// (chunks 0..C-2) beside attention C-1.  They hold kCopyBesideAttentionLds,
// which keeps them off the CUs the attention workgroups occupy: they take the
// CUs those launches' last rounds leave idle (or wait for the launch to end)
// instead of taking issue slots from attention waves.  In the other
// schedules a copy becomes ready when a launch starts (an unpack after the
// previous chunk's attention, a lane's pack), and a reserved copy that takes
// a CU first keeps the launch's workgroup off it, so they reserve nothing.
auto copy_lds_reserve(int mode, int C) {
    return [mode, C](int kind, int c) -> unsigned {
        if (mode != HCMS_MODE_INLINE) return 0;
        if ((kind == HCMS_OP_PACK && c == 0) || (kind == HCMS_OP_UNPACK && c == C - 1)) return 0;
        return hcms::kCopyBesideAttentionLds;
    };
}

// Issues a validated hcms_forward (S > 0) in the resolved mode.
int issue_forward(const ForwardArgs &f, int mode, int log2u) {
    const int64_t head_bytes = static_cast<int64_t>(f.S) * f.d * elem_bytes(f.dtype);
    const float c_log2e = scale_log2e(f.scale);
    // Chunk c's head-major buffers: its heads of the full workspaces, or slot
    // c % 2 of the two-slot ones.
    const int slot_heads = f.slot_heads;
    auto at = [head_bytes, slot_heads](void *p, int c, int h0) {
        const int64_t first = slot_heads > 0 ? static_cast<int64_t>(c & 1) * slot_heads : h0;
        return static_cast<char *>(p) + head_bytes * first;
    };
    const auto beside = copy_lds_reserve(mode, f.n_chunks);
    // The split scratch of the stream an attention launch runs on.  In the
    // lanes plan the two lanes' launches share rounds, so none splits its own
    // last round.  The last launch of each lane (chunks C - 2 and C - 1), whose
    // tiles close the pooled rounds, splits its last rem tiles instead, rem
    // the tiles past the last whole pooled round (the chunks' workgroups
    // summed, mod n_cu): which lane's tiles end the pooled rounds depends on
    // how the two queues' workgroups interleave, so both split.
    const int64_t tiles = (static_cast<int64_t>(f.S) + hcms::attention_queries_per_block(f.d) - 1) /
                          hcms::attention_queries_per_block(f.d);
    int64_t pooled = 0;
    for (int c = 0; c < f.n_chunks; ++c) pooled += tiles * f.chunk_sizes[c];
    hcms::SplitScratch lanes_tail{};
    auto split_for = [&](hipStream_t s, int c) -> const hcms::SplitScratch * {
        const int r = s == static_cast<hipStream_t>(f.main_stream) ? 0
                      : s == static_cast<hipStream_t>(f.compute_stream) ? 1 : -1;
        if (r < 0 || !f.ctx->split[r].part) return nullptr;
        if (mode != HCMS_MODE_LANES) return &f.ctx->split[r];
        if (c < f.n_chunks - 2) return nullptr;
        lanes_tail = f.ctx->split[r];
        lanes_tail.tail = pooled % f.ctx->n_cu;
        return &lanes_tail;
    };
    auto launch = [&](int kind, int c, int h0, int hc, hipStream_t s) -> hipError_t {
        if (kind == HCMS_OP_PACK) {
            const void *src[3] = {f.q_seq, f.k_seq, f.v_seq};
            void *dst[3] = {at(f.q_hm, c, h0), at(f.k_hm, c, h0), at(f.v_hm, c, h0)};
            return hcms::launch_pack(src, dst, 3, f.S, f.H, h0, hc, log2u, beside(kind, c), s);
        }
        if (kind == HCMS_OP_ATTENTION)
            return hcms::launch_attention(at(f.q_hm, c, h0), at(f.k_hm, c, h0), at(f.v_hm, c, h0),
                                          at(f.o_hm, c, h0),
                                          f.lse ? f.lse + static_cast<int64_t>(h0) * f.S : nullptr,
                                          f.S, hc, f.d, c_log2e, f.dtype, split_for(s, c), s);
        const void *src[1] = {at(f.o_hm, c, h0)};
        void *dst[1] = {f.o_seq};
        return hcms::launch_unpack(src, dst, 1, f.S, f.H, h0, hc, log2u, beside(kind, c), s);
    };
    auto ride = [&](int c, int h0, int hc, hipStream_t s, const RiderOp *riders, int n,
                    bool *riding) -> hipError_t {
        hcms::RidingCopy cp[2];
        for (int r = 0; r < n; ++r) {
            const RiderOp &ro = riders[r];
            cp[r] = hcms::RidingCopy{};
            cp[r].h0 = ro.h0;
            cp[r].hc = ro.hc;
            if (ro.kind == HCMS_OP_PACK) {
                cp[r].n_tensors = 3;
                cp[r].unpack = false;
                const void *src[3] = {f.q_seq, f.k_seq, f.v_seq};
                void *dst[3] = {at(f.q_hm, ro.chunk, ro.h0), at(f.k_hm, ro.chunk, ro.h0),
                                at(f.v_hm, ro.chunk, ro.h0)};
                for (int z = 0; z < 3; ++z) {
                    cp[r].src[z] = src[z];
                    cp[r].dst[z] = dst[z];
                }
            } else {
                cp[r].n_tensors = 1;
                cp[r].unpack = true;
                cp[r].src[0] = at(f.o_hm, ro.chunk, ro.h0);
                cp[r].dst[0] = f.o_seq;
            }
        }
        return hcms::launch_attention_riding(
            at(f.q_hm, c, h0), at(f.k_hm, c, h0), at(f.v_hm, c, h0), at(f.o_hm, c, h0),
            f.lse ? f.lse + static_cast<int64_t>(h0) * f.S : nullptr, f.S, hc, f.d, c_log2e,
            f.dtype, cp, n, f.H, f.ctx->n_cu, split_for(s, c), riding, s);
    };
    return execute_plan(f.ctx, mode, f.chunk_sizes, f.n_chunks, f.main_stream, f.copy_stream,
                        f.compute_stream, launch, ride);
}

// ---------------------------------------------------------------------------
// Layer neighbours: projections and rotary position embedding
// ---------------------------------------------------------------------------

// Y[M][N] = X[M][K] W[N][K]^T: shapes, pointers, alignment and, when
// y_is_matrix, that the [M][N] output overlaps neither input (the QKV
// projection writes three [M][N/3] tensors instead and checks them itself).
int check_linear(const void *x, const void *w, const void *y, int M, int N, int K, int dtype,
                 bool y_is_matrix = true) {
    int st;
    if ((st = check_dtype(dtype)) != HCMS_OK) return st;
    if (M < 0 || N < 0) return fail(HCMS_ERR_SHAPE, "need M >= 0 and N >= 0 (M=%d N=%d)", M, N);
    const int kq = hcms::linear_k_multiple();
    if (K < kq || K % kq != 0 || K > (1 << 20))
        return fail(HCMS_ERR_SHAPE, "K=%d must be a positive multiple of %d, at most 2^20", K, kq);
    if (N % 8 != 0 || N > (1 << 20))
        return fail(HCMS_ERR_SHAPE, "N=%d must be a multiple of 8, at most 2^20", N);
    if (M == 0 || N == 0) return HCMS_OK;
    if (!x || !w || !y) return fail(HCMS_ERR_NULL, "x, w or y is NULL");
    if (!aligned16(x) || !aligned16(w) || !aligned16(y))
        return fail(HCMS_ERR_ALIGN, "buffers must be 16-byte aligned");
    const int64_t es = elem_bytes(dtype);
    const int64_t xb = static_cast<int64_t>(M) * K * es, wb = static_cast<int64_t>(N) * K * es;
    const int64_t yb = static_cast<int64_t>(M) * N * es;
    if (y_is_matrix && (overlaps(y, yb, x, xb) || overlaps(y, yb, w, wb)))
        return fail(HCMS_ERR_ALIAS, "the output overlaps an input");
    return HCMS_OK;
}

// Rotation axes from the caller's grid and pair counts: 1..kRopeMaxAxes axes,
// every size >= 1; *tokens = product of the grid, *pairs = sum of the counts,
// *entries = table entries.
int rope_axes(const int *grid, const int *axis_pairs, int n_axes, hcms::RopeAxes *ax,
              int64_t *tokens, int64_t *pairs, int64_t *entries) {
    if (!grid || !axis_pairs) return fail(HCMS_ERR_NULL, "grid or axis_pairs is NULL");
    if (n_axes < 1 || n_axes > hcms::kRopeMaxAxes)
        return fail(HCMS_ERR_ARG, "n_axes=%d must be in [1, %d]", n_axes, hcms::kRopeMaxAxes);
    *ax = hcms::RopeAxes{};
    ax->n_axes = n_axes;
    int64_t prod = 1, np = 0, off = 0;
    for (int a = 0; a < n_axes; ++a) {
        if (grid[a] < 1 || axis_pairs[a] < 1)
            return fail(HCMS_ERR_SHAPE, "axis %d: grid size %d and pair count %d must be >= 1", a,
                        grid[a], axis_pairs[a]);
        ax->grid[a] = grid[a];
        ax->pairs[a] = axis_pairs[a];
        ax->pair_start[a] = static_cast<int>(np);
        ax->tab_off[a] = static_cast<int>(off);
        prod *= grid[a];
        np += axis_pairs[a];
        off += static_cast<int64_t>(grid[a]) * axis_pairs[a];
        if (prod > 0x7fffffffLL || off > (1LL << 28))
            return fail(HCMS_ERR_SHAPE, "grid too large (%lld tokens, %lld table entries)",
                        static_cast<long long>(prod), static_cast<long long>(off));
    }
    *tokens = prod;
    *pairs = np;
    *entries = off;
    return HCMS_OK;
}

// q, k, v [S][H][d] outputs of the QKV projection of x [S][D] by w [3 H d][D],
// rotated by `table` when it is not NULL.
int check_qkv(const void *x, const void *w, const float *table, const int *grid,
              const int *axis_pairs, int n_axes, const void *q, const void *k, const void *v, int S,
              int D, int H, int d, int dtype, hcms::RopeAxes *ax) {
    int st;
    if (S < 0 || H < 1 || d < 8 || d % 8 != 0)
        return fail(HCMS_ERR_SHAPE, "need S >= 0, H >= 1, d a positive multiple of 8 (S=%d H=%d d=%d)",
                    S, H, d);
    if (static_cast<int64_t>(3) * H * d > (1 << 20))
        return fail(HCMS_ERR_SHAPE, "3 H d = %lld exceeds 2^20", 3LL * H * d);
    if ((st = check_linear(x, w, q, S, 3 * H * d, D, dtype, false)) != HCMS_OK) return st;
    *ax = hcms::RopeAxes{};
    if (S == 0) return HCMS_OK;
    if (!k || !v) return fail(HCMS_ERR_NULL, "k or v is NULL");
    if (!aligned16(k) || !aligned16(v)) return fail(HCMS_ERR_ALIGN, "buffers must be 16-byte aligned");
    const int64_t es = elem_bytes(dtype);
    const int64_t tb = static_cast<int64_t>(S) * H * d * es;
    const int64_t xb = static_cast<int64_t>(S) * D * es, wb = 3LL * H * d * D * es;
    const void *outs[3] = {q, k, v};
    for (int i = 0; i < 3; ++i) {
        if (overlaps(outs[i], tb, x, xb) || overlaps(outs[i], tb, w, wb))
            return fail(HCMS_ERR_ALIAS, "output %d overlaps an input", i);
        for (int j = i + 1; j < 3; ++j)
            if (overlaps(outs[i], tb, outs[j], tb))
                return fail(HCMS_ERR_ALIAS, "outputs %d and %d overlap", i, j);
    }
    if (table) {
        int64_t tokens = 0, pairs = 0, entries = 0;
        if ((st = rope_axes(grid, axis_pairs, n_axes, ax, &tokens, &pairs, &entries)) != HCMS_OK)
            return st;
        if (tokens != S)
            return fail(HCMS_ERR_SHAPE, "the grid holds %lld tokens, not S=%d",
                        static_cast<long long>(tokens), S);
        if (pairs * 2 != d)
            return fail(HCMS_ERR_SHAPE, "the axis pair counts sum to %lld, not d/2=%d",
                        static_cast<long long>(pairs), d / 2);
        if (!aligned16(table)) return fail(HCMS_ERR_ALIGN, "table must be 16-byte aligned");
        for (int i = 0; i < 3; ++i)
            if (overlaps(table, entries * 8, outs[i], tb))
                return fail(HCMS_ERR_ALIAS, "table overlaps output %d", i);
    }
    return HCMS_OK;
}

}  // namespace

// The scratch array of hcms_attention_backward_noalloc: D = <dO, O> of every
// query of the call, HCMS_NOALLOC_DELTA_MAX floats (16 MiB) per device, held
// until the process ends.  Host code never uses this name as an address: the
// device address of each GPU's copy comes from hipGetSymbolAddress.
static __device__ __align__(256) float scratch[HCMS_NOALLOC_DELTA_MAX];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
float *g_scratch_ptr[kMaxDevices] = {};

// The current device's address of `scratch`, looked up once per device.
int scratch_for_current_device(float **out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (dev < 0 || dev >= kMaxDevices) return fail(HCMS_ERR_ARG, "device %d out of range", dev);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
        if (!p) return fail(HCMS_ERR_HIP, "hipGetSymbolAddress(scratch) returned NULL");
        g_scratch_ptr[dev] = static_cast<float *>(p);
    }
    *out = g_scratch_ptr[dev];
    return HCMS_OK;
}
}  // namespace

extern "C" {

int hcms_abi_version(void) { return HCMS_ABI_VERSION; }

const char *hcms_status_string(int status) {
    switch (status) {
        case HCMS_OK: return "HCMS_OK";
        case HCMS_ERR_NULL: return "HCMS_ERR_NULL";
        case HCMS_ERR_SHAPE: return "HCMS_ERR_SHAPE";
        case HCMS_ERR_CHUNKS: return "HCMS_ERR_CHUNKS";
        case HCMS_ERR_DTYPE: return "HCMS_ERR_DTYPE";
        case HCMS_ERR_ALIGN: return "HCMS_ERR_ALIGN";
        case HCMS_ERR_HIP: return "HCMS_ERR_HIP";
        case HCMS_ERR_ARG: return "HCMS_ERR_ARG";
        case HCMS_ERR_ALIAS: return "HCMS_ERR_ALIAS";
        case HCMS_ERR_CAPACITY: return "HCMS_ERR_CAPACITY";
        default: return "HCMS_UNKNOWN_STATUS";
    }
}

const char *hcms_last_error(void) { return hcms::last_error(); }

int hcms_default_chunks(int H, int C, int *sizes_out) {
    if (!sizes_out) return fail(HCMS_ERR_NULL, "sizes_out is NULL");
    if (H < 1 || C < 1 || C > H) return fail(HCMS_ERR_CHUNKS, "need 1 <= C <= H (H=%d, C=%d)", H, C);
    const int base = H / C, extra = H % C;
    for (int c = 0; c < C; ++c) sizes_out[c] = base + (c < extra ? 1 : 0);
    return ok();
}

int hcms_pack(const void *src_seq, void *dst_hm, int P, int S, int H, int d, int h_begin,
              int h_count, int dtype, void *stream) {
    int log2u = 0;
    const int st = check_pack_args(src_seq, dst_hm, P, S, H, d, h_begin, h_count, dtype, &log2u);
    if (st != HCMS_OK) return st;
    const void *src[1] = {src_seq};
    void *dst[1] = {dst_hm};
    const hipError_t e = hcms::launch_pack(src, dst, 1, S, H, h_begin, h_count, log2u, 0,
                                           static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "pack launch");
    return ok();
}

int hcms_unpack(const void *src_hm, void *dst_seq, int P, int S, int H, int d, int h_begin,
                int h_count, int dtype, void *stream) {
    int log2u = 0;
    const int st = check_pack_args(src_hm, dst_seq, P, S, H, d, h_begin, h_count, dtype, &log2u);
    if (st != HCMS_OK) return st;
    const void *src[1] = {src_hm};
    void *dst[1] = {dst_seq};
    const hipError_t e = hcms::launch_unpack(src, dst, 1, S, H, h_begin, h_count, log2u, 0,
                                             static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "unpack launch");
    return ok();
}

static int check_attention_args(const void *q, const void *k, const void *v, const void *out, int S,
                                int H, int d, float scale, const int *sizes, int n, int dtype) {
    int st;
    if (S > 0 && (!q || !k || !v || !out)) return fail(HCMS_ERR_NULL, "q, k, v or out is NULL");
    if ((st = check_dtype(dtype)) != HCMS_OK) return st;
    if ((st = check_dims(1, S, H, d, dtype)) != HCMS_OK) return st;
    if (d != 64 && d != 128) return fail(HCMS_ERR_SHAPE, "attention supports d = 64 or 128 (got %d)", d);
    if ((st = check_chunks(H, sizes, n)) != HCMS_OK) return st;
    if ((st = check_scale(scale)) != HCMS_OK) return st;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(out))
        return fail(HCMS_ERR_ALIGN, "buffers must be 16-byte aligned");
    const int64_t bytes = static_cast<int64_t>(S) * H * d * elem_bytes(dtype);
    if (overlaps(q, bytes, out, bytes) || overlaps(k, bytes, out, bytes) || overlaps(v, bytes, out, bytes))
        return fail(HCMS_ERR_ALIAS, "out overlaps q, k or v");
    return HCMS_OK;
}

int hcms_attention(const void *q, const void *k, const void *v, void *out, int S, int H, int d,
                   float scale, const int *chunk_sizes, int n_chunks, int dtype, void *stream) {
    const int st = check_attention_args(q, k, v, out, S, H, d, scale, chunk_sizes, n_chunks, dtype);
    if (st != HCMS_OK) return st;
    return run_attention(q, k, v, out, nullptr, S, d, scale, chunk_sizes, n_chunks, dtype,
                         static_cast<hipStream_t>(stream));
}

int hcms_attention_lse(const void *q, const void *k, const void *v, void *out, float *lse, int S,
                       int H, int d, float scale, const int *chunk_sizes, int n_chunks, int dtype,
                       void *stream) {
    int st = check_attention_args(q, k, v, out, S, H, d, scale, chunk_sizes, n_chunks, dtype);
    if (st != HCMS_OK) return st;
    if ((st = check_stats(lse, "lse", S, H, q, k, v, out, d, dtype)) != HCMS_OK) return st;
    return run_attention(q, k, v, out, lse, S, d, scale, chunk_sizes, n_chunks, dtype,
                         static_cast<hipStream_t>(stream));
}

// Validation shared by the two backward entry points; with_delta false: no
// delta workspace (the library's own scratch array takes its place).
static int check_backward_args(const void *q, const void *k, const void *v, const void *out,
                               const void *dout, const float *lse, void *dq, void *dk, void *dv,
                               bool with_delta, const float *delta, int S, int H, int d,
                               float scale, const int *chunk_sizes, int n_chunks, int dtype) {
    int st = check_attention_args(q, k, v, out, S, H, d, scale, chunk_sizes, n_chunks, dtype);
    if (st != HCMS_OK) return st;
    if (S > 0 && (!dout || !dq || !dk || !dv)) return fail(HCMS_ERR_NULL, "a gradient tensor is NULL");
    for (const void *p : {dout, static_cast<const void *>(dq), static_cast<const void *>(dk),
                          static_cast<const void *>(dv)})
        if (S > 0 && !aligned16(p)) return fail(HCMS_ERR_ALIGN, "buffers must be 16-byte aligned");
    const int64_t bytes = static_cast<int64_t>(S) * H * d * elem_bytes(dtype);
    // Outputs are disjoint from every input and from each other.
    const void *ins[5] = {q, k, v, out, dout};
    void *outs[3] = {dq, dk, dv};
    for (int i = 0; i < 3; ++i) {
        for (const void *x : ins)
            if (overlaps(outs[i], bytes, x, bytes))
                return fail(HCMS_ERR_ALIAS, "gradient %d overlaps an input", i);
        for (int j = i + 1; j < 3; ++j)
            if (overlaps(outs[i], bytes, outs[j], bytes))
                return fail(HCMS_ERR_ALIAS, "gradients %d and %d overlap", i, j);
    }
    if ((st = check_stats(lse, "lse", S, H, dq, dk, dv, dout, d, dtype)) != HCMS_OK) return st;
    if (with_delta) {
        if ((st = check_stats(delta, "delta", S, H, dq, dk, dv, dout, d, dtype)) != HCMS_OK) return st;
        if ((st = check_stats(delta, "delta", S, H, q, k, v, out, d, dtype)) != HCMS_OK) return st;
        if (S > 0 && overlaps(lse, int64_t{S} * H * 4, delta, int64_t{S} * H * 4))
            return fail(HCMS_ERR_ALIAS, "lse and delta overlap");
    }
    return HCMS_OK;
}

// A score-gradient workspace (NULL: none) must be 256-byte aligned and
// disjoint from the `n` tensors of `bytes` bytes each and the two [H][S]
// statistics.
static int check_ds_workspace(const void *ds, int64_t ds_bytes, const void *const *tensors, int n,
                              int64_t bytes, const float *lse, const float *delta, int S, int H) {
    if (ds_bytes < 0) return fail(HCMS_ERR_ARG, "ds_bytes=%lld must be >= 0", static_cast<long long>(ds_bytes));
    if (!ds || ds_bytes == 0 || S == 0) return HCMS_OK;
    if (reinterpret_cast<uintptr_t>(ds) % 256 != 0)
        return fail(HCMS_ERR_ALIGN, "the score-gradient workspace must be 256-byte aligned");
    for (int i = 0; i < n; ++i)
        if (overlaps(ds, ds_bytes, tensors[i], bytes))
            return fail(HCMS_ERR_ALIAS, "the score-gradient workspace overlaps tensor %d", i);
    const int64_t sb = int64_t{S} * H * 4;
    if (overlaps(ds, ds_bytes, lse, sb) || (delta && overlaps(ds, ds_bytes, delta, sb)))
        return fail(HCMS_ERR_ALIAS, "the score-gradient workspace overlaps lse or delta");
    return HCMS_OK;
}

// The chunks' backward launches, in order on `stream`.
static int run_backward(const void *q, const void *k, const void *v, const void *out,
                        const void *dout, const float *lse, void *dq, void *dk, void *dv,
                        float *delta, void *ds, int64_t ds_bytes, int S, int d, float scale,
                        const int *chunk_sizes, int n_chunks, int dtype, hipStream_t stream) {
    const int64_t head = static_cast<int64_t>(S) * d * elem_bytes(dtype);
    int h0 = 0;
    for (int i = 0; i < n_chunks; ++i) {
        const int64_t off = head * h0;
        const int64_t soff = static_cast<int64_t>(h0) * S;
        auto at = [off](const void *p) { return static_cast<const char *>(p) + off; };
        auto atw = [off](void *p) { return static_cast<char *>(p) + off; };
        const hipError_t e = hcms::launch_attention_backward(
            at(q), at(k), at(v), at(out), at(dout), lse + soff, atw(dq), atw(dk), atw(dv),
            delta + soff, ds, ds_bytes, S, chunk_sizes[i], d, scale, dtype, stream);
        if (e != hipSuccess) return hip_fail(e, "attention backward launch");
        h0 += chunk_sizes[i];
    }
    return ok();
}

int hcms_attention_backward(const void *q, const void *k, const void *v, const void *out,
                            const void *dout, const float *lse, void *dq, void *dk, void *dv,
                            float *delta, void *ds, int64_t ds_bytes, int S, int H, int d,
                            float scale, const int *chunk_sizes, int n_chunks, int dtype,
                            void *stream) {
    int st = check_backward_args(q, k, v, out, dout, lse, dq, dk, dv, true, delta, S, H, d, scale,
                                 chunk_sizes, n_chunks, dtype);
    if (st != HCMS_OK) return st;
    const void *all[8] = {q, k, v, out, dout, dq, dk, dv};
    const int64_t bytes = static_cast<int64_t>(S) * H * d * elem_bytes(dtype);
    if ((st = check_ds_workspace(ds, ds_bytes, all, 8, bytes, lse, delta, S, H)) != HCMS_OK) return st;
    if (S == 0) return ok();
    return run_backward(q, k, v, out, dout, lse, dq, dk, dv, delta, ds, ds_bytes, S, d, scale,
                        chunk_sizes, n_chunks, dtype, static_cast<hipStream_t>(stream));
}

int hcms_backward_ds_bytes(int S, int d, int dtype, int64_t *bytes_out) {
    if (!bytes_out) return fail(HCMS_ERR_NULL, "bytes_out is NULL");
    *bytes_out = 0;
    if (S < 0) return fail(HCMS_ERR_SHAPE, "S=%d must be >= 0", S);
    int st;
    if ((st = check_dtype(dtype)) != HCMS_OK) return st;
    *bytes_out = hcms::attention_backward_ds_head_bytes(S, d, dtype);
    return ok();
}

int hcms_attention_backward_noalloc(const void *q, const void *k, const void *v, const void *out,
                                    const void *dout, const float *lse, void *dq, void *dk,
                                    void *dv, int S, int H, int d, float scale,
                                    const int *chunk_sizes, int n_chunks, int dtype,
                                    void *stream) {
    int st = check_backward_args(q, k, v, out, dout, lse, dq, dk, dv, false, nullptr, S, H, d,
                                 scale, chunk_sizes, n_chunks, dtype);
    if (st != HCMS_OK) return st;
    if (static_cast<int64_t>(S) * H > HCMS_NOALLOC_DELTA_MAX)
        return fail(HCMS_ERR_CAPACITY, "S * H = %lld exceeds the scratch limit of %d queries",
                    static_cast<long long>(S) * H, HCMS_NOALLOC_DELTA_MAX);
    if (S == 0) return ok();
    float *delta = nullptr;
    if ((st = scratch_for_current_device(&delta)) != HCMS_OK) return st;
    return run_backward(q, k, v, out, dout, lse, dq, dk, dv, delta, nullptr, 0, S, d, scale,
                        chunk_sizes, n_chunks, dtype, static_cast<hipStream_t>(stream));
}

int hcms_plan(int n_chunks, int mode, hcms_op *ops, int cap) {
    if (n_chunks < 1) return fail(HCMS_ERR_CHUNKS, "n_chunks=%d must be >= 1", n_chunks);
    if (!plan_mode(mode))
        return fail(HCMS_ERR_ARG, "mode %d has no fixed plan (serial 0, pipelined 1, inline 2, "
                    "lanes 3, slots 5, fused 6)", mode);
    const int need = plan_size(n_chunks, mode);
    if (ops == nullptr) {
        ok();
        return need;
    }
    if (cap < need) return fail(HCMS_ERR_CAPACITY, "plan needs %d ops, capacity is %d", need, cap);
    PlanWriter w{ops, cap};
    const int n = build_plan(n_chunks, mode, w);
    ok();
    return n;
}

int hcms_auto_mode(int S, int d, int dtype, const int *chunk_sizes, int n_chunks, int n_cu) {
    if (S < 0) return fail(HCMS_ERR_SHAPE, "S=%d must be >= 0", S);
    const int st_dtype = check_dtype(dtype);
    if (st_dtype != HCMS_OK) return st_dtype;
    if (d != 64 && d != 128) return fail(HCMS_ERR_SHAPE, "attention supports d = 64 or 128 (got %d)", d);
    if (n_cu < 1) return fail(HCMS_ERR_ARG, "n_cu=%d must be >= 1", n_cu);
    if (!chunk_sizes) return fail(HCMS_ERR_NULL, "chunk_sizes is NULL");
    if (n_chunks < 1) return fail(HCMS_ERR_CHUNKS, "n_chunks=%d must be >= 1", n_chunks);
    int H = 0;
    for (int c = 0; c < n_chunks; ++c) {
        if (chunk_sizes[c] < 1) return fail(HCMS_ERR_CHUNKS, "chunk %d is empty", c);
        H += chunk_sizes[c];
    }
    int st = check_chunks(H, chunk_sizes, n_chunks);
    if (st != HCMS_OK) return st;
    ok();
    return auto_mode(S, d, dtype, chunk_sizes, n_chunks, n_cu);
}

int hcms_ctx_last_mode(const hcms_ctx *ctx) {
    if (!ctx) return fail(HCMS_ERR_NULL, "ctx is NULL");
    ok();
    return ctx->last_mode;
}

int hcms_ctx_set_ds_workspace(hcms_ctx *ctx, void *ws, int64_t bytes) {
    if (!ctx) return fail(HCMS_ERR_NULL, "ctx is NULL");
    if (bytes < 0) return fail(HCMS_ERR_ARG, "bytes=%lld must be >= 0", static_cast<long long>(bytes));
    if (ws && reinterpret_cast<uintptr_t>(ws) % 256 != 0)
        return fail(HCMS_ERR_ALIGN, "the score-gradient workspace must be 256-byte aligned");
    ctx->ds = ws && bytes > 0 ? static_cast<char *>(ws) : nullptr;
    ctx->ds_region = ctx->ds ? bytes / 2 / 256 * 256 : 0;
    return ok();
}

int hcms_ctx_num_cu(const hcms_ctx *ctx) {
    if (!ctx) return fail(HCMS_ERR_NULL, "ctx is NULL");
    ok();
    return ctx->n_cu;
}

int hcms_ctx_create(int device, int max_chunks, hcms_ctx **out) {
    if (!out) return fail(HCMS_ERR_NULL, "out is NULL");
    *out = nullptr;
    if (max_chunks < 1) return fail(HCMS_ERR_CHUNKS, "max_chunks=%d must be >= 1", max_chunks);
    int n_dev = 0;
    hipError_t e = hipGetDeviceCount(&n_dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDeviceCount");
    if (device < 0 || device >= n_dev)
        return fail(HCMS_ERR_ARG, "device %d out of range [0, %d)", device, n_dev);
    DeviceGuard guard(device);
    if (guard.err != hipSuccess) return hip_fail(guard.err, "hipSetDevice");
    hcms_ctx *ctx = new (std::nothrow) hcms_ctx;
    if (!ctx) return fail(HCMS_ERR_ARG, "out of host memory");
    ctx->device = device;
    ctx->max_chunks = max_chunks;
    e = hipDeviceGetAttribute(&ctx->n_cu, hipDeviceAttributeMultiprocessorCount, device);
    if (e != hipSuccess || ctx->n_cu < 1) {
        delete ctx;
        return hip_fail(e != hipSuccess ? e : hipErrorInvalidValue, "hipDeviceGetAttribute");
    }
    ctx->plan.resize(plan_size(max_chunks, HCMS_MODE_PIPELINED));
    const int n_sync = 2 * max_chunks + 2;
    for (int i = 0; i < n_sync; ++i) {
        hipEvent_t ev;
        e = hipEventCreateWithFlags(&ev, hipEventDisableTiming);
        if (e != hipSuccess) {
            hcms_ctx_destroy(ctx);
            return hip_fail(e, "hipEventCreateWithFlags");
        }
        ctx->events.push_back(ev);
    }
    // Split scratch, two regions of n_cu slots and n_cu counters each.  If it
    // cannot be had, launches keep every tile whole (same results).
    {
        const int64_t slot = hcms::attention_split_slot_bytes();
        const int64_t n = ctx->n_cu;
        const int64_t region = n * slot + n * 4;
        void *mem = nullptr;
        if (hipMalloc(&mem, 2 * region) == hipSuccess && mem) {
            if (hipMemset(mem, 0, 2 * region) == hipSuccess) {
                ctx->split_mem = mem;
                for (int r = 0; r < 2; ++r) {
                    char *base = static_cast<char *>(mem) + r * region;
                    hcms::SplitScratch &sp = ctx->split[r];
                    sp.part = base;
                    sp.ml = base + n * (slot - 256 * 16);
                    sp.count = reinterpret_cast<int *>(base + n * slot);
                    sp.slots = static_cast<int>(n);
                    sp.counters = static_cast<int>(n);
                    sp.n_cu = ctx->n_cu;
                }
            } else {
                (void)hipFree(mem);
            }
        }
        (void)hipGetLastError();
    }
    *out = ctx;
    return ok();
}

int hcms_ctx_destroy(hcms_ctx *ctx) {
    if (!ctx) return ok();
    DeviceGuard guard(ctx->device);
    for (hipEvent_t ev : ctx->events) (void)hipEventDestroy(ev);
    for (hipEvent_t ev : ctx->t_begin) (void)hipEventDestroy(ev);
    for (hipEvent_t ev : ctx->t_end) (void)hipEventDestroy(ev);
    if (ctx->split_mem) (void)hipFree(ctx->split_mem);
    delete ctx;
    return ok();
}

int hcms_ctx_set_timing(hcms_ctx *ctx, int max_calls) {
    if (!ctx) return fail(HCMS_ERR_NULL, "ctx is NULL");
    if (max_calls < 0) return fail(HCMS_ERR_ARG, "max_calls=%d must be >= 0", max_calls);
    const size_t need = static_cast<size_t>(max_calls) * 3 * ctx->max_chunks;
    if (need > ctx->t_begin.size()) {
        DeviceGuard guard(ctx->device);
        if (guard.err != hipSuccess) return hip_fail(guard.err, "hipSetDevice");
        while (ctx->t_begin.size() < need) {
            hipEvent_t a, b;
            hipError_t e = hipEventCreate(&a);
            if (e != hipSuccess) return hip_fail(e, "hipEventCreate");
            e = hipEventCreate(&b);
            if (e != hipSuccess) {
                (void)hipEventDestroy(a);
                return hip_fail(e, "hipEventCreate");
            }
            ctx->t_begin.push_back(a);
            ctx->t_end.push_back(b);
        }
    }
    ctx->timing_calls = max_calls;
    ctx->timed_chunks.clear();
    return ok();
}

int hcms_ctx_kernel_ms(hcms_ctx *ctx, int kind, float *ms_out, int cap) {
    if (!ctx || !ms_out) return fail(HCMS_ERR_NULL, "ctx or ms_out is NULL");
    if (ctx->timing_calls == 0) return fail(HCMS_ERR_ARG, "timing is off");
    if (kind != HCMS_OP_PACK && kind != HCMS_OP_ATTENTION && kind != HCMS_OP_UNPACK)
        return fail(HCMS_ERR_ARG, "kind %d is not PACK, ATTENTION or UNPACK", kind);
    int total = 0;
    for (int n : ctx->timed_chunks) total += n;
    if (cap < total) return fail(HCMS_ERR_CAPACITY, "need %d entries, capacity is %d", total, cap);
    DeviceGuard guard(ctx->device);
    if (guard.err != hipSuccess) return hip_fail(guard.err, "hipSetDevice");
    int w = 0;
    for (size_t call = 0; call < ctx->timed_chunks.size(); ++call) {
        for (int c = 0; c < ctx->timed_chunks[call]; ++c) {
            const size_t slot = (call * 3 + (kind - HCMS_OP_PACK)) * ctx->max_chunks + c;
            hipError_t e = hipEventSynchronize(ctx->t_end[slot]);
            if (e != hipSuccess) return hip_fail(e, "hipEventSynchronize");
            e = hipEventElapsedTime(&ms_out[w++], ctx->t_begin[slot], ctx->t_end[slot]);
            if (e != hipSuccess) return hip_fail(e, "hipEventElapsedTime");
        }
    }
    ok();
    return total;
}

int hcms_forward(hcms_ctx *ctx, const void *q_seq, const void *k_seq, const void *v_seq, void *o_seq,
                 void *q_hm, void *k_hm, void *v_hm, void *o_hm, float *lse, int P, int S, int H,
                 int d, float scale, const int *chunk_sizes, int n_chunks, int dtype, int mode,
                 void *main_stream, void *copy_stream, void *compute_stream) {
    const ForwardArgs f{ctx, q_seq, k_seq, v_seq, o_seq, q_hm, k_hm, v_hm, o_hm, lse, P, S, H, d,
                        scale, chunk_sizes, n_chunks, dtype, mode, main_stream, copy_stream,
                        compute_stream};
    int st, log2u = 0, resolved = mode;
    if ((st = check_forward(f, &resolved, &log2u)) != HCMS_OK) return st;
    if (S == 0) return ok();
    return issue_forward(f, resolved, log2u);
}

int hcms_forward_slots(hcms_ctx *ctx, const void *q_seq, const void *k_seq, const void *v_seq,
                       void *o_seq, void *q_slots, void *k_slots, void *v_slots, void *o_slots,
                       int slot_heads, int P, int S, int H, int d, float scale,
                       const int *chunk_sizes, int n_chunks, int dtype, int mode,
                       void *main_stream, void *copy_stream, void *compute_stream) {
    if (slot_heads < 1) return fail(HCMS_ERR_CHUNKS, "slot_heads=%d must be >= 1", slot_heads);
    ForwardArgs f{ctx, q_seq, k_seq, v_seq, o_seq, q_slots, k_slots, v_slots, o_slots, nullptr, P,
                  S, H, d, scale, chunk_sizes, n_chunks, dtype, mode, main_stream, copy_stream,
                  compute_stream};
    f.slot_heads = slot_heads;
    int st, log2u = 0, resolved = mode;
    if ((st = check_forward(f, &resolved, &log2u)) != HCMS_OK) return st;
    if (S == 0) return ok();
    return issue_forward(f, resolved, log2u);
}

int hcms_linear(const void *x, const void *w, void *y, int M, int N, int K, int dtype,
                void *stream) {
    int st;
    if ((st = check_linear(x, w, y, M, N, K, dtype)) != HCMS_OK) return st;
    if (M == 0 || N == 0) return ok();
    const hipError_t e = hcms::launch_linear(x, w, y, M, N, K, dtype, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "linear launch");
    return ok();
}

int hcms_rope_table_entries(const int *grid, const int *axis_pairs, int n_axes) {
    hcms::RopeAxes ax;
    int64_t tokens = 0, pairs = 0, entries = 0;
    const int st = rope_axes(grid, axis_pairs, n_axes, &ax, &tokens, &pairs, &entries);
    if (st != HCMS_OK) return st;
    ok();
    return static_cast<int>(entries);
}

int hcms_rope_table(float *table, const int *grid, const int *axis_pairs, int n_axes, double base,
                    void *stream) {
    hcms::RopeAxes ax;
    int64_t tokens = 0, pairs = 0, entries = 0;
    int st;
    if ((st = rope_axes(grid, axis_pairs, n_axes, &ax, &tokens, &pairs, &entries)) != HCMS_OK) return st;
    if (!table) return fail(HCMS_ERR_NULL, "table is NULL");
    if (!aligned16(table)) return fail(HCMS_ERR_ALIGN, "table must be 16-byte aligned");
    if (!std::isfinite(base) || !(base > 1.0))
        return fail(HCMS_ERR_ARG, "base must be finite and > 1 (got %g)", base);
    const hipError_t e = hcms::launch_rope_table(table, ax, base, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "rope table launch");
    return ok();
}

int hcms_qkv_projection(const void *x, const void *w_qkv, const float *table, const int *grid,
                        const int *axis_pairs, int n_axes, void *q_seq, void *k_seq, void *v_seq,
                        int S, int D, int H, int d, int dtype, void *stream) {
    hcms::RopeAxes ax;
    int st;
    if ((st = check_qkv(x, w_qkv, table, grid, axis_pairs, n_axes, q_seq, k_seq, v_seq, S, D, H, d,
                        dtype, &ax)) != HCMS_OK)
        return st;
    if (S == 0) return ok();
    const hipError_t e = hcms::launch_qkv_projection(x, w_qkv, q_seq, k_seq, v_seq, table, ax, S, D,
                                                     H, d, dtype, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "qkv projection launch");
    return ok();
}

int hcms_layer_forward(hcms_ctx *ctx, const void *x, const void *w_qkv, const void *w_o,
                       const float *table, const int *grid, const int *axis_pairs, int n_axes,
                       void *y, void *q_seq, void *k_seq, void *v_seq, void *o_seq, void *q_hm,
                       void *k_hm, void *v_hm, void *o_hm, int P, int S, int D, int H, int d,
                       float scale, const int *chunk_sizes, int n_chunks, int dtype, int mode,
                       void *main_stream, void *copy_stream, void *compute_stream) {
    int st;
    hcms::RopeAxes ax;
    if ((st = check_qkv(x, w_qkv, table, grid, axis_pairs, n_axes, q_seq, k_seq, v_seq, S, D, H, d,
                        dtype, &ax)) != HCMS_OK)
        return st;
    const ForwardArgs f{ctx, q_seq, k_seq, v_seq, o_seq, q_hm, k_hm, v_hm, o_hm, nullptr, P, S, H,
                        d, scale, chunk_sizes, n_chunks, dtype, mode, main_stream, copy_stream,
                        compute_stream};
    int log2u = 0, resolved = mode;
    if ((st = check_forward(f, &resolved, &log2u)) != HCMS_OK) return st;
    if ((st = check_linear(o_seq, w_o, y, S, D, H * d, dtype)) != HCMS_OK) return st;
    if (S > 0) {
        // No output or workspace of the layer may overlap an input or y.
        const int64_t es = elem_bytes(dtype);
        const int64_t xb = static_cast<int64_t>(S) * D * es, tb = static_cast<int64_t>(S) * H * d * es;
        const int64_t wqb = 3LL * H * d * D * es, wob = static_cast<int64_t>(D) * H * d * es;
        const void *in[3] = {x, w_qkv, w_o};
        const int64_t inb[3] = {xb, wqb, wob};
        const void *t[9] = {q_seq, k_seq, v_seq, o_seq, q_hm, k_hm, v_hm, o_hm, y};
        for (int i = 0; i < 9; ++i) {
            const int64_t ti = i == 8 ? xb : tb;
            for (int j = 0; j < 3; ++j)
                if (overlaps(t[i], ti, in[j], inb[j]))
                    return fail(HCMS_ERR_ALIAS, "layer buffer %d overlaps input %d", i, j);
            if (i < 8 && overlaps(t[i], tb, y, xb))
                return fail(HCMS_ERR_ALIAS, "layer buffer %d overlaps y", i);
        }
    }
    if (S == 0) return ok();
    const hipStream_t ms = static_cast<hipStream_t>(main_stream);
    hipError_t e = hcms::launch_qkv_projection(x, w_qkv, q_seq, k_seq, v_seq, table, ax, S, D, H, d,
                                               dtype, ms);
    if (e != hipSuccess) return hip_fail(e, "qkv projection launch");
    if ((st = issue_forward(f, resolved, log2u)) != HCMS_OK) return st;
    // o_seq [S][H][d] is the concatenation of the heads, [S][H d].
    e = hcms::launch_linear(o_seq, w_o, y, S, D, H * d, dtype, ms);
    if (e != hipSuccess) return hip_fail(e, "output projection launch");
    return ok();
}

int hcms_backward(hcms_ctx *ctx, const void *dout_seq, void *dq_seq, void *dk_seq, void *dv_seq,
                  const void *q_hm, const void *k_hm, const void *v_hm, const void *o_hm,
                  const float *lse, void *do_hm, void *dq_hm, void *dk_hm, void *dv_hm,
                  float *delta, int P, int S, int H, int d, float scale, const int *chunk_sizes,
                  int n_chunks, int dtype, int mode, void *main_stream, void *copy_stream,
                  void *compute_stream) {
    int st;
    if (!ctx) return fail(HCMS_ERR_NULL, "ctx is NULL");
    const void *all[13] = {q_hm, k_hm, v_hm, o_hm, dout_seq, dq_seq, dk_seq, dv_seq,
                           do_hm, dq_hm, dk_hm, dv_hm, nullptr};
    if (S > 0)
        for (int i = 0; i < 12; ++i)
            if (!all[i]) return fail(HCMS_ERR_NULL, "a tensor pointer is NULL");
    int log2u = 0;
    const int64_t ds_head = hcms::attention_backward_ds_head_bytes(S, d, dtype);
    const bool ds_path = ctx->ds != nullptr && ds_head > 0 && ctx->ds_region >= ds_head;
    if ((st = check_schedule(ctx, P, S, H, d, scale, chunk_sizes, n_chunks, dtype, &mode, &log2u,
                             main_stream, copy_stream, compute_stream, false, ds_path)) != HCMS_OK)
        return st;
    for (int i = 0; i < 12; ++i)
        if (S > 0 && !aligned16(all[i])) return fail(HCMS_ERR_ALIGN, "buffers must be 16-byte aligned");
    // The first five are read only and may alias each other; the seven
    // written tensors must not overlap anything.
    const int64_t bytes = static_cast<int64_t>(S) * H * d * elem_bytes(dtype);
    for (int i = 0; i < 12; ++i)
        for (int j = i + 1; j < 12; ++j)
            if (j >= 5 && overlaps(all[i], bytes, all[j], bytes))
                return fail(HCMS_ERR_ALIAS, "tensor %d overlaps tensor %d", i, j);
    for (int i = 0; i < 12; i += 4) {
        const void *const *g = all + i;
        if ((st = check_stats(lse, "lse", S, H, g[0], g[1], g[2], g[3], d, dtype)) != HCMS_OK) return st;
        if ((st = check_stats(delta, "delta", S, H, g[0], g[1], g[2], g[3], d, dtype)) != HCMS_OK)
            return st;
    }
    if (S > 0 && overlaps(lse, int64_t{S} * H * 4, delta, int64_t{S} * H * 4))
        return fail(HCMS_ERR_ALIAS, "lse and delta overlap");
    if ((st = check_ds_workspace(ctx->ds, 2 * ctx->ds_region, all, 12, bytes, lse, delta, S, H)) !=
        HCMS_OK)
        return st;
    if (S == 0) return ok();

    const int64_t head_bytes = static_cast<int64_t>(S) * d * elem_bytes(dtype);
    auto at = [head_bytes](const void *p, int h0) {
        return const_cast<char *>(static_cast<const char *>(p)) + head_bytes * h0;
    };
    const auto beside = copy_lds_reserve(mode, n_chunks);
    auto launch = [&](int kind, int c, int h0, int hc, hipStream_t s) -> hipError_t {
        if (kind == HCMS_OP_PACK) {
            const void *src[1] = {dout_seq};
            void *dst[1] = {at(do_hm, h0)};
            return hcms::launch_pack(src, dst, 1, S, H, h0, hc, log2u, beside(kind, c), s);
        }
        if (kind == HCMS_OP_ATTENTION) {
            const int64_t so = static_cast<int64_t>(h0) * S;
            // Launches on one stream are ordered, so each stream's region
            // serves one chunk at a time.
            char *ds = ctx->ds ? ctx->ds + (s == static_cast<hipStream_t>(main_stream) ? 0 : ctx->ds_region)
                              : nullptr;
            return hcms::launch_attention_backward(at(q_hm, h0), at(k_hm, h0), at(v_hm, h0),
                                                   at(o_hm, h0), at(do_hm, h0), lse + so,
                                                   at(dq_hm, h0), at(dk_hm, h0), at(dv_hm, h0),
                                                   delta + so, ds, ctx->ds_region, S, hc, d,
                                                   scale, dtype, s);
        }
        const void *src[3] = {at(dq_hm, h0), at(dk_hm, h0), at(dv_hm, h0)};
        void *dst[3] = {dq_seq, dk_seq, dv_seq};
        return hcms::launch_unpack(src, dst, 3, S, H, h0, hc, log2u, beside(kind, c), s);
    };
    // The backward launches carry no copies: the fused plan's copies run
    // right after each chunk's backward launches.
    auto ride = [&](int c, int h0, int hc, hipStream_t s, const RiderOp *, int,
                    bool *riding) -> hipError_t {
        *riding = false;
        return launch(HCMS_OP_ATTENTION, c, h0, hc, s);
    };
    return execute_plan(ctx, mode, chunk_sizes, n_chunks, main_stream, copy_stream, compute_stream,
                        launch, ride);
}

}  // extern "C"
