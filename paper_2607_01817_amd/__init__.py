"""HCMS single-GPU hot path on AMD MI355X (gfx950).

A thin ctypes binding over ``libhcms.so`` (the C ABI in ``include/hcms.h``).
Every step runs in the library's HIP kernels.  This module only checks tensors
(device, dtype, shape, contiguity), passes their device pointers and HIP
stream handles, and turns status codes into exceptions.  PyTorch provides
device memory and streams.

Names follow the paper (arXiv 2607.01817): ``pack``/``unpack`` are one GPU's
share of the input/output all-to-all of a head chunk, ``attention`` runs the
chunks' attention, and :class:`Context` is the dual-stream chunk scheduler
of Alg. 1 with its cached events.
"""
from __future__ import annotations

import ctypes
import os

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libhcms.so")

BF16, FP32 = 0, 1
MODE_SERIAL, MODE_PIPELINED, MODE_INLINE, MODE_LANES, MODE_AUTO, MODE_SLOTS, MODE_FUSED = (
    0, 1, 2, 3, 4, 5, 6)
OP_RECORD, OP_WAIT, OP_PACK, OP_ATTENTION, OP_UNPACK = 0, 1, 2, 3, 4
STREAM_MAIN, STREAM_COPY, STREAM_COMPUTE, STREAM_IN_ATTENTION = 0, 1, 2, 3
NOALLOC_DELTA_MAX = 4 * 1024 * 1024   # S * H limit of attention_backward_noalloc

_DTYPES = {torch.bfloat16: BF16, torch.float32: FP32}
_lib = None


class HcmsError(RuntimeError):
    """A negative status from the C ABI, with the library's detail string."""

    def __init__(self, status: int, name: str, detail: str):
        super().__init__(f"{name} ({status}): {detail}")
        self.status = status
        self.name = name
        self.detail = detail


class Op(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int), ("stream", ctypes.c_int),
                ("chunk", ctypes.c_int), ("event", ctypes.c_int)]


def load():
    """Load ``libhcms.so`` (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                           "`python -m paper_2607_01817_amd.build` (no CPU fallback exists)")
    lib = ctypes.CDLL(LIB_PATH)
    i, vp, f, d = ctypes.c_int, ctypes.c_void_p, ctypes.c_float, ctypes.c_double
    i64 = ctypes.c_int64
    ip = ctypes.POINTER(ctypes.c_int)
    dp = ctypes.POINTER(ctypes.c_double)
    sig = {
        "hcms_abi_version": ([], i),
        "hcms_status_string": ([i], ctypes.c_char_p),
        "hcms_last_error": ([], ctypes.c_char_p),
        "hcms_default_chunks": ([i, i, ip], i),
        "hcms_pack": ([vp, vp, i, i, i, i, i, i, i, vp], i),
        "hcms_unpack": ([vp, vp, i, i, i, i, i, i, i, vp], i),
        "hcms_attention": ([vp, vp, vp, vp, i, i, i, f, ip, i, i, vp], i),
        "hcms_attention_lse": ([vp, vp, vp, vp, vp, i, i, i, f, ip, i, i, vp], i),
        "hcms_attention_backward": ([vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, i64, i, i, i, f,
                                     ip, i, i, vp], i),
        "hcms_backward_ds_bytes": ([i, i, i, ctypes.POINTER(i64)], i),
        "hcms_ctx_set_ds_workspace": ([vp, vp, i64], i),
        "hcms_attention_backward_noalloc": ([vp, vp, vp, vp, vp, vp, vp, vp, vp, i, i, i, f, ip,
                                             i, i, vp], i),
        "hcms_plan": ([i, i, ctypes.POINTER(Op), i], i),
        "hcms_auto_mode": ([i, i, i, ip, i, i], i),
        "hcms_ctx_last_mode": ([vp], i),
        "hcms_model_time": ([d, d, d, d, i, dp], i),
        "hcms_model_optimal_chunks": ([d, d, i, dp], i),
        "hcms_model_speedup": ([d, d, i, dp], i),
        "hcms_model_fit": ([ip, dp, i, dp, dp, dp], i),
        "hcms_model_plan_time": ([i, i, i, ip, i, i, i, d, d, d, d, d, dp], i),
        "hcms_choose_chunks": ([i, i, i, i, i, d, d, d, d, d, i, ip, ip, dp], i),
        "hcms_ctx_num_cu": ([vp], i),
        "hcms_ctx_create": ([i, i, ctypes.POINTER(vp)], i),
        "hcms_ctx_destroy": ([vp], i),
        "hcms_ctx_set_timing": ([vp, i], i),
        "hcms_ctx_kernel_ms": ([vp, i, ctypes.POINTER(ctypes.c_float), i], i),
        "hcms_forward": ([vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, i, i, i, i, f, ip, i, i, i,
                          vp, vp, vp], i),
        "hcms_backward": ([vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, i, i, i, i,
                           f, ip, i, i, i, vp, vp, vp], i),
        "hcms_forward_slots": ([vp, vp, vp, vp, vp, vp, vp, vp, vp, i, i, i, i, i, f, ip, i, i, i,
                                vp, vp, vp], i),
        "hcms_linear": ([vp, vp, vp, i, i, i, i, vp], i),
        "hcms_rope_table_entries": ([ip, ip, i], i),
        "hcms_rope_table": ([vp, ip, ip, i, d, vp], i),
        "hcms_qkv_projection": ([vp, vp, vp, ip, ip, i, vp, vp, vp, i, i, i, i, i, vp], i),
        "hcms_layer_forward": ([vp, vp, vp, vp, vp, ip, ip, i, vp, vp, vp, vp, vp, vp, vp, vp, vp,
                                i, i, i, i, i, f, ip, i, i, i, vp, vp, vp], i),
    }
    for name, (args, res) in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    _lib = lib
    return lib


def _check(status: int) -> int:
    if status < 0:
        lib = load()
        raise HcmsError(status, lib.hcms_status_string(status).decode(),
                        lib.hcms_last_error().decode())
    return status


def _ints(xs):
    xs = [int(x) for x in xs]
    return (ctypes.c_int * max(1, len(xs)))(*xs), len(xs)


def _dtype(t: torch.Tensor) -> int:
    if t.dtype not in _DTYPES:
        raise TypeError(f"unsupported dtype {t.dtype}; use bfloat16 or float32")
    return _DTYPES[t.dtype]


def _dev(t: torch.Tensor, name: str):
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _expect(t: torch.Tensor, shape, dtype, name: str):
    """Shape and dtype of a tensor the C ABI only sees as a pointer (the
    callers check every size first and the devices after, so that a wrong
    size never reaches a launch)."""
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a tensor")
    if tuple(t.shape) != tuple(shape) or t.dtype != dtype:
        raise ValueError(f"{name} must be {list(shape)} of {dtype} "
                         f"(got {list(t.shape)} of {t.dtype})")


def _devs(named):
    for t, n in named:
        _dev(t, n)


def _table_rows(grid, axis_pairs) -> int:
    g, na = _ints(grid)
    p, npairs = _ints(axis_pairs)
    if na != npairs:
        raise ValueError("one pair count per grid axis")
    return _check(load().hcms_rope_table_entries(g, p, na))


def _stream(s) -> ctypes.c_void_p:
    if s is None:
        s = torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def abi_version() -> int:
    return load().hcms_abi_version()


def default_chunks(H: int, C: int) -> list[int]:
    """Chunk sizes of the paper's rule (more first, less later)."""
    buf = (ctypes.c_int * max(1, C))()
    _check(load().hcms_default_chunks(H, C, buf))
    return list(buf[:C])


def plan(n_chunks: int, mode: int = MODE_PIPELINED) -> list[tuple[int, int, int, int]]:
    """The op list hcms_forward issues: (kind, stream, chunk, event) tuples."""
    lib = load()
    n = _check(lib.hcms_plan(n_chunks, mode, None, 0))
    ops = (Op * n)()
    _check(lib.hcms_plan(n_chunks, mode, ops, n))
    return [(o.kind, o.stream, o.chunk, o.event) for o in ops]


def auto_mode(S: int, d: int, chunk_sizes, n_cu: int, dtype: int = BF16) -> int:
    """The plan mode MODE_AUTO runs for these chunks on n_cu compute units."""
    sizes, n = _ints(chunk_sizes)
    return _check(load().hcms_auto_mode(S, d, dtype, sizes, n, n_cu))


def model_time(t0: float, t_comm: float, t_attn: float, beta: float, n_chunks: int) -> float:
    """T_hcms(C) of the paper's time model."""
    out = ctypes.c_double()
    _check(load().hcms_model_time(t0, t_comm, t_attn, beta, n_chunks, ctypes.byref(out)))
    return out.value


def model_optimal_chunks(t_comm: float, beta: float, H: int) -> tuple[int, float]:
    """(best integer chunk count in [1, H], C* = sqrt(t_comm / beta))."""
    c_real = ctypes.c_double()
    best = _check(load().hcms_model_optimal_chunks(t_comm, beta, H, ctypes.byref(c_real)))
    return best, c_real.value


def model_speedup(rho: float, beta_over_total: float, n_chunks: int) -> float:
    out = ctypes.c_double()
    _check(load().hcms_model_speedup(rho, beta_over_total, n_chunks, ctypes.byref(out)))
    return out.value


def model_fit(chunk_counts, times) -> tuple[float, float, float]:
    """(a = t0 + t_attn, t_comm, beta) fitted to measured (C, time) pairs."""
    cs, n = _ints(chunk_counts)
    ts = (ctypes.c_double * max(1, len(times)))(*[float(t) for t in times])
    a, tc, b = ctypes.c_double(), ctypes.c_double(), ctypes.c_double()
    _check(load().hcms_model_fit(cs, ts, n, ctypes.byref(a), ctypes.byref(tc), ctypes.byref(b)))
    return a.value, tc.value, b.value


def model_plan_time(S: int, d: int, chunk_sizes, mode: int, n_cu: int, t_round: float,
                    g0: float, t_copy: float, beta: float, dtype: int = BF16,
                    drain: float = 0.0) -> float:
    """One-GPU model time of a plan (see hcms.h, hcms_model_plan_time)."""
    sizes, n = _ints(chunk_sizes)
    out = ctypes.c_double()
    _check(load().hcms_model_plan_time(S, d, dtype, sizes, n, mode, n_cu, t_round, g0, drain,
                                       t_copy, beta, ctypes.byref(out)))
    return out.value


def choose_chunks(S: int, H: int, d: int, n_cu: int, t_round: float, g0: float, t_copy: float,
                  beta: float, max_chunks: int | None = None, dtype: int = BF16,
                  drain: float = 0.0):
    """(sizes, plan, model time) of the chunk count the one-GPU model predicts
    fastest under the plan MODE_AUTO runs (hcms_choose_chunks)."""
    top = H if max_chunks is None else max_chunks
    buf = (ctypes.c_int * max(1, min(H, top)))()
    mode = ctypes.c_int()
    t = ctypes.c_double()
    n = _check(load().hcms_choose_chunks(S, H, d, dtype, n_cu, t_round, g0, drain, t_copy, beta,
                                         top, buf, ctypes.byref(mode), ctypes.byref(t)))
    return list(buf[:n]), mode.value, t.value


def pack(src_seq: torch.Tensor, P: int, h_begin: int, h_count: int,
         out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """[S][H][d] (= [P][S/P][H][d]) -> [h_count][S][d] chunk of heads."""
    _dev(src_seq, "src_seq")
    S, H, d = src_seq.shape
    if out is None:
        out = torch.empty((h_count, S, d), dtype=src_seq.dtype, device=src_seq.device)
    _dev(out, "out")
    if out.shape != (h_count, S, d) or out.dtype != src_seq.dtype:
        raise ValueError("out must be [h_count][S][d] of the source dtype")
    _check(load().hcms_pack(src_seq.data_ptr(), out.data_ptr(), P, S, H, d, h_begin, h_count,
                            _dtype(src_seq), _stream(stream)))
    return out


def unpack(src_hm: torch.Tensor, dst_seq: torch.Tensor, P: int, h_begin: int,
           stream=None) -> torch.Tensor:
    """Write the [h_count][S][d] chunk into head slots of dst_seq [S][H][d]."""
    _dev(src_hm, "src_hm")
    _dev(dst_seq, "dst_seq")
    hc, S, d = src_hm.shape
    if dst_seq.dim() != 3 or dst_seq.shape[0] != S or dst_seq.shape[2] != d \
            or dst_seq.dtype != src_hm.dtype:
        raise ValueError("dst_seq must be [S][H][d] of the chunk's dtype")
    H = dst_seq.shape[1]
    _check(load().hcms_unpack(src_hm.data_ptr(), dst_seq.data_ptr(), P, S, H, d, h_begin, hc,
                              _dtype(src_hm), _stream(stream)))
    return dst_seq


def attention(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, scale: float,
              chunk_sizes=None, out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """Non-causal softmax attention on head-major [H][S][d] tensors, run as
    one kernel launch per head chunk (default: one chunk of all heads)."""
    for t, n in ((q, "q"), (k, "k"), (v, "v")):
        _dev(t, n)
    if not (q.shape == k.shape == v.shape) or q.dim() != 3:
        raise ValueError("q, k, v must all be [H][S][d]")
    if not (q.dtype == k.dtype == v.dtype):
        raise ValueError("q, k, v must share a dtype")
    H, S, d = q.shape
    if out is None:
        out = torch.empty_like(q)
    _dev(out, "out")
    if out.shape != q.shape or out.dtype != q.dtype:
        raise ValueError("out must match q")
    sizes, n = _ints([H] if chunk_sizes is None else chunk_sizes)
    _check(load().hcms_attention(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(),
                                 S, H, d, float(scale), sizes, n, _dtype(q), _stream(stream)))
    return out



def _same_hm(ts, names, like):
    _dev(like, "q")
    if like.dim() != 3:
        raise ValueError("q must be [H][S][d]")
    for t, n in zip(ts, names):
        _dev(t, n)
        if t.shape != like.shape or t.dtype != like.dtype:
            raise ValueError(f"{n} must match q ([H][S][d], same dtype)")


def _stats(t, name, H, S, device):
    if t is None:
        return torch.empty((H, S), dtype=torch.float32, device=device)
    _dev(t, name)
    if t.dtype != torch.float32 or t.shape != (H, S):
        raise ValueError(f"{name} must be float32 [H][S]")
    return t


def attention_lse(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, scale: float,
                  chunk_sizes=None, out: torch.Tensor | None = None,
                  lse: torch.Tensor | None = None, stream=None):
    """Training forward: ``(out, lse)`` with ``lse[h][i]`` the log2 softmax
    denominator of ``scale * log2(e) * <q_i, k_j>`` (see hcms.h)."""
    _same_hm((k, v), ("k", "v"), q)
    H, S, d = q.shape
    if out is None:
        out = torch.empty_like(q)
    _same_hm((out,), ("out",), q)
    lse = _stats(lse, "lse", H, S, q.device)
    sizes, n = _ints(chunk_sizes if chunk_sizes is not None else [H])
    _check(load().hcms_attention_lse(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(),
                                     lse.data_ptr(), S, H, d, float(scale), sizes, n, _dtype(q),
                                     _stream(stream)))
    return out, lse


def backward_ds_bytes(S: int, d: int, dtype: torch.dtype = torch.bfloat16) -> int:
    """Bytes of score-gradient workspace one head of the backward needs (0
    where that path does not apply: d != 128 or float32 storage)."""
    out = ctypes.c_int64()
    _check(load().hcms_backward_ds_bytes(S, d, _DTYPES[dtype], ctypes.byref(out)))
    return out.value


def _ds_arg(ds):
    if ds is None:
        return None, 0
    if not ds.is_cuda or not ds.is_contiguous():
        raise ValueError("ds must be a contiguous device tensor")
    return ds.data_ptr(), ds.numel() * ds.element_size()


def attention_backward(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, out: torch.Tensor,
                       dout: torch.Tensor, lse: torch.Tensor, scale: float, chunk_sizes=None,
                       dq=None, dk=None, dv=None, delta=None, ds=None, stream=None):
    """``(dq, dk, dv)`` of head-major attention for output gradient ``dout``;
    ``lse`` comes from :func:`attention_lse` on the same inputs.  ``ds``, a
    device tensor of at least :func:`backward_ds_bytes` per head, turns on
    the path that stores the score gradients and computes dq from them."""
    _same_hm((k, v, out, dout), ("k", "v", "out", "dout"), q)
    H, S, d = q.shape
    dq = torch.empty_like(q) if dq is None else dq
    dk = torch.empty_like(q) if dk is None else dk
    dv = torch.empty_like(q) if dv is None else dv
    _same_hm((dq, dk, dv), ("dq", "dk", "dv"), q)
    lse = _stats(lse, "lse", H, S, q.device)
    delta = _stats(delta, "delta", H, S, q.device)
    sizes, n = _ints(chunk_sizes if chunk_sizes is not None else [H])
    ds_ptr, ds_bytes = _ds_arg(ds)
    _check(load().hcms_attention_backward(
        q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(), dout.data_ptr(), lse.data_ptr(),
        dq.data_ptr(), dk.data_ptr(), dv.data_ptr(), delta.data_ptr(), ds_ptr, ds_bytes, S, H, d,
        float(scale), sizes, n, _dtype(q), _stream(stream)))
    return dq, dk, dv


def attention_backward_noalloc(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor,
                               out: torch.Tensor, dout: torch.Tensor, lse: torch.Tensor,
                               scale: float, chunk_sizes, dq: torch.Tensor, dk: torch.Tensor,
                               dv: torch.Tensor, stream=None):
    """:func:`attention_backward` into caller-given ``dq``, ``dk``, ``dv``
    with the library's own scratch array in place of the delta workspace:
    the call allocates nothing (for code that must not allocate, such as a
    captured graph).  S * H is limited to ``NOALLOC_DELTA_MAX``."""
    _same_hm((k, v, out, dout, dq, dk, dv), ("k", "v", "out", "dout", "dq", "dk", "dv"), q)
    H, S, d = q.shape
    lse = _stats(lse, "lse", H, S, q.device)
    sizes, n = _ints(chunk_sizes)
    _check(load().hcms_attention_backward_noalloc(
        q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(), dout.data_ptr(), lse.data_ptr(),
        dq.data_ptr(), dk.data_ptr(), dv.data_ptr(), S, H, d, float(scale), sizes, n, _dtype(q),
        _stream(stream)))
    return dq, dk, dv

def linear(x: torch.Tensor, w: torch.Tensor, out: torch.Tensor | None = None,
           stream=None) -> torch.Tensor:
    """Projection GEMM: x [M][K] times w [N][K] (weight stored [out][in]),
    out [M][N] = x w^T, in the library's MFMA kernel."""
    _dev(x, "x")
    _dev(w, "w")
    if x.dim() != 2 or w.dim() != 2 or x.shape[1] != w.shape[1] or x.dtype != w.dtype:
        raise ValueError("x must be [M][K] and w [N][K] of one dtype")
    M, K = x.shape
    N = w.shape[0]
    if out is None:
        out = torch.empty((M, N), dtype=x.dtype, device=x.device)
    _dev(out, "out")
    if out.shape != (M, N) or out.dtype != x.dtype:
        raise ValueError("out must be [M][N] of the input dtype")
    _check(load().hcms_linear(x.data_ptr(), w.data_ptr(), out.data_ptr(), M, N, K, _dtype(x),
                              _stream(stream)))
    return out


def rope_table(grid, axis_pairs, base: float = 10000.0, device="cuda",
               stream=None) -> torch.Tensor:
    """The rotation table of the latent grid ``grid`` whose head vectors'
    pairs split into consecutive groups of ``axis_pairs`` (one per axis):
    float32 [E][2] (cos, sin), filled on the GPU."""
    g, na = _ints(grid)
    p, npairs = _ints(axis_pairs)
    if na != npairs:
        raise ValueError("one pair count per grid axis")
    lib = load()
    n = _check(lib.hcms_rope_table_entries(g, p, na))
    table = torch.empty((max(1, n), 2), dtype=torch.float32, device=device)
    _check(lib.hcms_rope_table(table.data_ptr(), g, p, na, float(base), _stream(stream)))
    return table[:n]


def qkv_projection(x: torch.Tensor, w_qkv: torch.Tensor, H: int, d: int,
                   table: torch.Tensor | None = None, grid=None, axis_pairs=None,
                   out=None, stream=None):
    """x [S][D] times w_qkv [3 H d][D]: (q, k, v) [S][H][d] each, the query
    and key pairs rotated by ``table`` (from :func:`rope_table` on the same
    grid and axis_pairs) when it is given."""
    if x.dim() != 2:
        raise ValueError("x must be [S][D]")
    S, D = x.shape
    _expect(x, (S, D), x.dtype, "x")
    _expect(w_qkv, (3 * H * d, D), x.dtype, "w_qkv")
    if out is None:
        out = tuple(torch.empty((S, H, d), dtype=x.dtype, device=x.device) for _ in range(3))
    if len(out) != 3:
        raise ValueError("out must be three [S][H][d] tensors")
    for t, n in zip(out, ("q_seq", "k_seq", "v_seq")):
        _expect(t, (S, H, d), x.dtype, n)
    g = p = None
    na = 0
    tp = None
    if table is not None:
        _expect(table, (_table_rows(grid, axis_pairs), 2), torch.float32, "table")
        _dev(table, "table")
        g, na = _ints(grid)
        p, _ = _ints(axis_pairs)
        tp = table.data_ptr()
    _devs(((x, "x"), (w_qkv, "w_qkv"), *zip(out, ("q_seq", "k_seq", "v_seq"))))
    _check(load().hcms_qkv_projection(x.data_ptr(), w_qkv.data_ptr(), tp, g, p, na,
                                      out[0].data_ptr(), out[1].data_ptr(), out[2].data_ptr(),
                                      S, D, H, d, _dtype(x), _stream(stream)))
    return out


class Context:
    """The chunk scheduler (Alg. 1 and its one-GPU schedules) on one device.

    Owns the library context (cached events), a copy stream and a compute
    stream (default priority), and head-major workspaces that are reallocated
    only when the problem shape grows.
    """

    def __init__(self, device: int = 0, max_chunks: int = 64):
        lib = load()
        self.device = device
        self.max_chunks = max_chunks
        h = ctypes.c_void_p()
        with torch.cuda.device(device):
            _check(lib.hcms_ctx_create(device, max_chunks, ctypes.byref(h)))
            self.copy_stream = torch.cuda.Stream(device=device)
            self.compute_stream = torch.cuda.Stream(device=device)
        self._h = h
        self._ws = None
        self._ws_key = None
        self._bws = None
        self._bws_key = None
        self._ds = None

    @property
    def num_cu(self) -> int:
        return _check(load().hcms_ctx_num_cu(self._h))

    def set_ds_workspace(self, ds):
        """Give :meth:`backward` a score-gradient workspace (a contiguous
        device tensor, used as two equal regions, one per stream; see
        :func:`backward_ds_bytes`), or remove it (None).  The context keeps a
        reference to the tensor."""
        ptr, nbytes = _ds_arg(ds)
        _check(load().hcms_ctx_set_ds_workspace(self._h, ptr, nbytes))
        self._ds = ds

    @property
    def last_mode(self) -> int:
        """Plan mode of the last forward (MODE_AUTO resolved), -1 before any."""
        return load().hcms_ctx_last_mode(self._h)

    def close(self):
        if self._h:
            torch.cuda.synchronize(self.device)
            load().hcms_ctx_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            if self._h and _lib is not None:
                _lib.hcms_ctx_destroy(self._h)
        except Exception:
            pass

    def workspaces(self, S: int, H: int, d: int, dtype: torch.dtype):
        key = (S, H, d, dtype)
        if self._ws_key != key:
            self._ws = [torch.empty((H, S, d), dtype=dtype, device=f"cuda:{self.device}")
                        for _ in range(4)]
            self._ws_key = key
        return self._ws

    def set_timing(self, max_calls: int):
        """Time every kernel of the next ``max_calls`` forward calls (0: off)."""
        _check(load().hcms_ctx_set_timing(self._h, int(max_calls)))
        self._timing_calls = int(max_calls)

    def kernel_ms(self, kind: int) -> list[float]:
        """Durations (ms) of the timed calls' kernels of one kind, call by call
        and chunk by chunk (waits for them)."""
        cap = max(1, getattr(self, "_timing_calls", 0)) * self.max_chunks
        buf = (ctypes.c_float * cap)()
        n = _check(load().hcms_ctx_kernel_ms(self._h, kind, buf, cap))
        return list(buf[:n])

    def forward(self, q_seq: torch.Tensor, k_seq: torch.Tensor, v_seq: torch.Tensor, P: int,
                scale: float, chunk_sizes, mode: int = MODE_AUTO,
                out: torch.Tensor | None = None, workspaces=None,
                main_stream=None, lse: torch.Tensor | None = None) -> torch.Tensor:
        """One GPU's share of an HCMS forward: [S][H][d] in, [S][H][d] out.

        The result is ordered on ``main_stream`` (default: the current stream)
        when this returns; nothing blocks the host.  With ``lse`` (float32
        [H][S]) the attention also writes its log2 softmax denominators, and
        the workspaces keep the head-major Q, K, V, O: :meth:`backward` needs
        both.
        """
        for t, n in ((q_seq, "q_seq"), (k_seq, "k_seq"), (v_seq, "v_seq")):
            _dev(t, n)
        if not (q_seq.shape == k_seq.shape == v_seq.shape) or q_seq.dim() != 3:
            raise ValueError("q_seq, k_seq, v_seq must all be [S][H][d]")
        if not (q_seq.dtype == k_seq.dtype == v_seq.dtype):
            raise ValueError("q_seq, k_seq, v_seq must share a dtype")
        S, H, d = q_seq.shape
        if out is None:
            out = torch.empty_like(q_seq)
        _dev(out, "out")
        if out.shape != q_seq.shape or out.dtype != q_seq.dtype:
            raise ValueError("out must match q_seq")
        ws = workspaces if workspaces is not None else self.workspaces(S, H, d, q_seq.dtype)
        for t in ws:
            _dev(t, "workspace")
            if t.numel() != q_seq.numel() or t.dtype != q_seq.dtype:
                raise ValueError("each workspace must hold [H][S][d] of the input dtype")
        sizes, n = _ints(chunk_sizes)
        main = _stream(main_stream)
        lse_p = None
        if lse is not None:
            lse_p = _stats(lse, "lse", H, S, q_seq.device).data_ptr()
        _check(load().hcms_forward(
            self._h, q_seq.data_ptr(), k_seq.data_ptr(), v_seq.data_ptr(), out.data_ptr(),
            ws[0].data_ptr(), ws[1].data_ptr(), ws[2].data_ptr(), ws[3].data_ptr(), lse_p,
            P, S, H, d, float(scale), sizes, n, _dtype(q_seq), int(mode), main,
            ctypes.c_void_p(self.copy_stream.cuda_stream),
            ctypes.c_void_p(self.compute_stream.cuda_stream)))
        return out

    def slot_workspaces(self, S: int, slot_heads: int, d: int, dtype: torch.dtype):
        """Four two-slot head-major workspaces, [2][slot_heads][S][d] each."""
        key = (S, slot_heads, d, dtype)
        if getattr(self, "_sws_key", None) != key:
            self._sws = [torch.empty((2, slot_heads, S, d), dtype=dtype,
                                     device=f"cuda:{self.device}") for _ in range(4)]
            self._sws_key = key
        return self._sws

    def forward_slots(self, q_seq: torch.Tensor, k_seq: torch.Tensor, v_seq: torch.Tensor, P: int,
                      scale: float, chunk_sizes, mode: int = MODE_AUTO,
                      out: torch.Tensor | None = None, slots=None, main_stream=None) -> torch.Tensor:
        """:meth:`forward` with two chunk slots (``slots``: four
        [2][slot_heads][S][d] buffers, slot_heads >= every chunk) instead of
        full head-major workspaces; modes serial, lanes, slots, fused or auto."""
        if q_seq.dim() != 3:
            raise ValueError("q_seq must be [S][H][d]")
        for t, n in ((q_seq, "q_seq"), (k_seq, "k_seq"), (v_seq, "v_seq")):
            _expect(t, q_seq.shape, q_seq.dtype, n)
        S, H, d = q_seq.shape
        if out is None:
            out = torch.empty_like(q_seq)
        _expect(out, q_seq.shape, q_seq.dtype, "out")
        if slots is None:
            slots = self.slot_workspaces(S, max(int(c) for c in chunk_sizes), d, q_seq.dtype)
        if len(slots) != 4 or slots[0].dim() != 4:
            raise ValueError("slots must be four [2][slot_heads][S][d] tensors")
        slot_heads = slots[0].shape[1]
        for t in slots:
            _expect(t, (2, slot_heads, S, d), q_seq.dtype, "slot workspace")
        _devs(((q_seq, "q_seq"), (k_seq, "k_seq"), (v_seq, "v_seq"), (out, "out"),
               *((t, "slot workspace") for t in slots)))
        sizes, n = _ints(chunk_sizes)
        _check(load().hcms_forward_slots(
            self._h, q_seq.data_ptr(), k_seq.data_ptr(), v_seq.data_ptr(), out.data_ptr(),
            *[t.data_ptr() for t in slots], slot_heads, P, S, H, d, float(scale), sizes, n,
            _dtype(q_seq), int(mode), _stream(main_stream),
            ctypes.c_void_p(self.copy_stream.cuda_stream),
            ctypes.c_void_p(self.compute_stream.cuda_stream)))
        return out

    def layer_forward(self, x: torch.Tensor, w_qkv: torch.Tensor, w_o: torch.Tensor, P: int,
                      H: int, d: int, scale: float, chunk_sizes, table=None, grid=None,
                      axis_pairs=None, mode: int = MODE_AUTO, out=None, buffers=None,
                      main_stream=None) -> torch.Tensor:
        """One attention layer around the chunk loop: x [S][D] -> y [S][D]
        (QKV projection with the rotation, :meth:`forward`, output projection).
        ``buffers`` (q_seq, k_seq, v_seq, o_seq, each [S][H][d]) are kept
        between calls with the same shape."""
        if x.dim() != 2:
            raise ValueError("x must be [S][D]")
        S, D = x.shape
        _expect(x, (S, D), x.dtype, "x")
        _expect(w_qkv, (3 * H * d, D), x.dtype, "w_qkv")
        _expect(w_o, (D, H * d), x.dtype, "w_o")
        if out is not None:
            _expect(out, (S, D), x.dtype, "out")
        if buffers is not None:
            if len(buffers) != 4:
                raise ValueError("buffers must be q_seq, k_seq, v_seq, o_seq")
            for b, n in zip(buffers, ("q_seq", "k_seq", "v_seq", "o_seq")):
                _expect(b, (S, H, d), x.dtype, n)
        g = p = None
        na = 0
        tp = None
        if table is not None:
            _expect(table, (_table_rows(grid, axis_pairs), 2), torch.float32, "table")
            _dev(table, "table")
            g, na = _ints(grid)
            p, _ = _ints(axis_pairs)
            tp = table.data_ptr()
        _devs(((x, "x"), (w_qkv, "w_qkv"), (w_o, "w_o")))
        if out is not None:
            _dev(out, "out")
        for b in buffers or ():
            _dev(b, "buffer")
        if out is None:
            out = torch.empty((S, D), dtype=x.dtype, device=x.device)
        if buffers is None:
            key = (S, H, d, x.dtype)
            if getattr(self, "_lbuf_key", None) != key:
                self._lbuf = [torch.empty((S, H, d), dtype=x.dtype, device=x.device)
                              for _ in range(4)]
                self._lbuf_key = key
            buffers = self._lbuf
        ws = self.workspaces(S, H, d, x.dtype)
        sizes, n = _ints(chunk_sizes)
        _check(load().hcms_layer_forward(
            self._h, x.data_ptr(), w_qkv.data_ptr(), w_o.data_ptr(), tp, g, p, na,
            out.data_ptr(), *[b.data_ptr() for b in buffers], *[t.data_ptr() for t in ws],
            P, S, D, H, d, float(scale), sizes, n, _dtype(x), int(mode), _stream(main_stream),
            ctypes.c_void_p(self.copy_stream.cuda_stream),
            ctypes.c_void_p(self.compute_stream.cuda_stream)))
        return out

    def backward_workspaces(self, S: int, H: int, d: int, dtype: torch.dtype):
        """Head-major dO, dQ, dK, dV workspaces and the [H][S] float32 delta."""
        key = (S, H, d, dtype)
        if self._bws_key != key:
            dev = f"cuda:{self.device}"
            self._bws = [torch.empty((H, S, d), dtype=dtype, device=dev) for _ in range(4)]
            self._bws.append(torch.empty((H, S), dtype=torch.float32, device=dev))
            self._bws_key = key
        return self._bws

    def backward(self, dout_seq: torch.Tensor, P: int, scale: float, chunk_sizes, workspaces,
                 lse: torch.Tensor, mode: int = MODE_AUTO, dq=None, dk=None, dv=None,
                 backward_workspaces=None, main_stream=None):
        """Gradients (dq, dk, dv), each [S][H][d], of the forward whose head-major
        workspaces and ``lse`` are given, for the output gradient ``dout_seq``."""
        _dev(dout_seq, "dout_seq")
        if dout_seq.dim() != 3:
            raise ValueError("dout_seq must be [S][H][d]")
        S, H, d = dout_seq.shape
        outs = [torch.empty_like(dout_seq) if t is None else t for t in (dq, dk, dv)]
        for t, nm in zip(outs, ("dq", "dk", "dv")):
            _dev(t, nm)
            if t.shape != dout_seq.shape or t.dtype != dout_seq.dtype:
                raise ValueError(f"{nm} must match dout_seq")
        fw = list(workspaces)
        bw = backward_workspaces if backward_workspaces is not None else \
            self.backward_workspaces(S, H, d, dout_seq.dtype)
        for t in fw + list(bw[:4]):
            _dev(t, "workspace")
            if t.numel() != dout_seq.numel() or t.dtype != dout_seq.dtype:
                raise ValueError("each workspace must hold [H][S][d] of the gradient's dtype")
        lse = _stats(lse, "lse", H, S, dout_seq.device)
        delta = _stats(bw[4], "delta", H, S, dout_seq.device)
        sizes, n = _ints(chunk_sizes)
        _check(load().hcms_backward(
            self._h, dout_seq.data_ptr(), outs[0].data_ptr(), outs[1].data_ptr(), outs[2].data_ptr(),
            fw[0].data_ptr(), fw[1].data_ptr(), fw[2].data_ptr(), fw[3].data_ptr(), lse.data_ptr(),
            bw[0].data_ptr(), bw[1].data_ptr(), bw[2].data_ptr(), bw[3].data_ptr(), delta.data_ptr(),
            P, S, H, d, float(scale), sizes, n, _dtype(dout_seq), int(mode), _stream(main_stream),
            ctypes.c_void_p(self.copy_stream.cuda_stream),
            ctypes.c_void_p(self.compute_stream.cuda_stream)))
        return tuple(outs)


class HcmsAttention(torch.autograd.Function):
    """Autograd over :meth:`Context.forward` and :meth:`Context.backward`:
    ``HcmsAttention.apply(q_seq, k_seq, v_seq, ctx, P, scale, chunk_sizes,
    mode)`` returns the [S][H][d] output, and its backward runs the reverse
    pipeline.  The forward allocates its own head-major workspaces (kept for
    the backward) so that later calls on the same context do not overwrite
    them."""

    @staticmethod
    def forward(fctx, q_seq, k_seq, v_seq, ctx, P, scale, chunk_sizes, mode=MODE_AUTO):
        S, H, d = q_seq.shape
        ws = [torch.empty((H, S, d), dtype=q_seq.dtype, device=q_seq.device) for _ in range(4)]
        lse = torch.empty((H, S), dtype=torch.float32, device=q_seq.device)
        out = ctx.forward(q_seq.contiguous(), k_seq.contiguous(), v_seq.contiguous(), P, scale,
                          chunk_sizes, mode=mode, workspaces=ws, lse=lse)
        fctx.hcms = (ctx, P, scale, tuple(chunk_sizes), mode, ws, lse)
        return out

    @staticmethod
    def backward(fctx, dout):
        ctx, P, scale, sizes, mode, ws, lse = fctx.hcms
        dq, dk, dv = ctx.backward(dout.contiguous(), P, scale, sizes, ws, lse, mode=mode)
        return dq, dk, dv, None, None, None, None, None
