"""Oracle for the single-GPU share of HCMS (arXiv 2607.01817).

TEST INFRASTRUCTURE ONLY.  The test suite, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` are the only callers.  The product path
(``paper_2607_01817_amd``) never imports this package, and this package never
imports the product path: the two share no code, only the seeded inputs that
``paper_2607_01817_amd.inputs`` draws.

Contents, each a plain statement of what the paper defines:

* :func:`default_chunks`  the head-chunk size rule of Sec. 3.3 (chunk-size
  equation): ``H_c = floor(H/C) + [c < H mod C]``, larger chunks first
  ("more-first-less-later", Sec. 4.1, implementation details).
* :func:`attention`        per-head softmax attention, fp64, two-pass, in C
  (``hcms_oracle.c``), Sec. 3.3 Property of computational independence.
* :func:`pack` / :func:`unpack`  the chunk split along heads plus the local
  share of the input/output all-to-all (Sec. 3.1, Sec. 3.3 split equation,
  Alg. 1 SplitByHeads / Concat), as explicit index loops in C.
* :func:`forward`          unpack o attention o pack over every chunk.
* :func:`lse_head`         log2 of each query row's softmax denominator, the
  statistic a training forward keeps for its backward pass.
* :func:`attention_backward_head`  the gradient of one head's attention with
  respect to Q, K and V for a given output gradient, by the chain rule through
  the row softmax, in C (``hcms_oracle.c``).

Modules beside this one: ``oracle.time_model`` (the appendix's time model) and
``oracle.layer`` (QKV projection, rotary position embedding and output
projection around the hot path, Alg. 1's main-stream steps).

Every function here is pinned by tests in ``tests/test_oracle.py`` against
values the paper prints (the uneven-partition table), closed forms, invariants
and a library routine (PyTorch's CPU scaled-dot-product attention in fp64).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "hcms_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None


def build(verbose: bool = False) -> str:
    """Compile ``hcms_oracle.c`` into ``liboracle.so`` with gcc and OpenMP."""
    cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11",
           "-o", _LIB_PATH + ".tmp", _SRC, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(_LIB_PATH + ".tmp", _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        build()
    lib = ctypes.CDLL(_LIB_PATH)
    i64, vp, dp = ctypes.c_int64, ctypes.c_void_p, ctypes.c_double
    lib.oracle_attention_rows.argtypes = [vp, vp, vp, i64, i64, dp, vp, i64, vp]
    lib.oracle_attention_rows.restype = ctypes.c_int
    for fn in (lib.oracle_pack, lib.oracle_unpack):
        fn.argtypes = [vp, vp, i64, i64, i64, i64, i64, i64, i64]
        fn.restype = ctypes.c_int
    lib.oracle_attention_backward.argtypes = [vp, vp, vp, vp, i64, i64, dp, vp, i64, vp, i64,
                                              vp, vp, vp]
    lib.oracle_attention_backward.restype = ctypes.c_int
    lib.oracle_num_threads.argtypes = []
    lib.oracle_num_threads.restype = ctypes.c_int
    _lib = lib
    return lib


def num_threads() -> int:
    """Threads the C attention oracle uses (OpenMP default team size)."""
    return int(_load().oracle_num_threads())


# ---------------------------------------------------------------------------
# Sec. 3.3, chunk-size equation
# ---------------------------------------------------------------------------
def default_chunks(H: int, C: int) -> list[int]:
    """Chunk sizes for ``H`` heads in ``C`` chunks, larger chunks first.

    ``H_c = floor(H / C) + 1 if c < H mod C else floor(H / C)`` for c < C.
    """
    if H < 1 or C < 1 or C > H:
        raise ValueError(f"need 1 <= C <= H, got H={H}, C={C}")
    return [H // C + (1 if c < H % C else 0) for c in range(C)]


def chunk_offsets(sizes) -> list[int]:
    """First head of each chunk: h0_c = sum of the sizes before c."""
    out, acc = [], 0
    for n in sizes:
        out.append(acc)
        acc += int(n)
    return out


# ---------------------------------------------------------------------------
# Attention (fp64, two-pass softmax)
# ---------------------------------------------------------------------------
def attention_head(q: np.ndarray, k: np.ndarray, v: np.ndarray, scale: float,
                   rows=None) -> np.ndarray:
    """Softmax attention of one head.

    ``q`` is ``[Sq][d]``, ``k`` and ``v`` are ``[S][d]`` (any real dtype;
    widened to fp64 exactly).  ``rows`` selects query indices (default: all).
    Returns ``[len(rows)][d]`` fp64.
    """
    q = np.ascontiguousarray(q, dtype=np.float64)
    k = np.ascontiguousarray(k, dtype=np.float64)
    v = np.ascontiguousarray(v, dtype=np.float64)
    if q.ndim != 2 or k.ndim != 2 or v.shape != k.shape or q.shape[1] != k.shape[1]:
        raise ValueError("q must be [Sq][d] and k, v [S][d]")
    S, d = k.shape
    if rows is None:
        rows = np.arange(q.shape[0], dtype=np.int64)
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    if rows.size and (rows.min() < 0 or rows.max() >= q.shape[0]):
        raise ValueError("row index out of range")
    out = np.empty((rows.size, d), dtype=np.float64)
    if rows.size == 0:
        return out
    rc = _load().oracle_attention_rows(
        q.ctypes.data, k.ctypes.data, v.ctypes.data, S, d, float(scale),
        rows.ctypes.data, rows.size, out.ctypes.data)
    if rc != 0:
        raise MemoryError("oracle scratch allocation failed")
    return out


def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, scale: float,
              rows=None) -> np.ndarray:
    """Head-major attention: ``q``, ``k``, ``v`` are ``[H][S][d]``.

    ``rows`` is ``None`` (all queries of every head) or a sequence of per-head
    index arrays.  Returns ``[H][S][d]`` or a list of ``[n_h][d]`` arrays.
    """
    H = q.shape[0]
    if rows is None:
        return np.stack([attention_head(q[h], k[h], v[h], scale) for h in range(H)])
    return [attention_head(q[h], k[h], v[h], scale, rows[h]) for h in range(H)]


def lse_head(q: np.ndarray, k: np.ndarray, scale: float, rows=None) -> np.ndarray:
    """log2 of the softmax denominator of each listed query row:
    ``log2 sum_j exp(scale * <q_i, k_j>)`` (= ``log2 sum_j exp2(c <q_i, k_j>)``
    with ``c = scale * log2(e)``), fp64, with the row maximum taken out before
    the exponentials."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    rows = np.arange(q.shape[0]) if rows is None else np.asarray(rows, dtype=np.int64)
    s = scale * (q[rows] @ k.T)
    m = s.max(axis=1)
    return (m + np.log(np.exp(s - m[:, None]).sum(axis=1))) / np.log(2.0)


def attention_backward_head(q: np.ndarray, k: np.ndarray, v: np.ndarray, g: np.ndarray,
                            scale: float, q_rows=None, k_rows=None):
    """Gradients of one head's attention for output gradient ``g``.

    ``q``, ``k``, ``v``, ``g`` are ``[S][d]``.  Returns ``(dq, dk, dv)``:
    ``dq`` for the query indices ``q_rows`` (default all), ``dk`` and ``dv``
    for the key indices ``k_rows`` (default all), each ``[n][d]`` fp64.
    """
    q, k, v, g = (np.ascontiguousarray(x, dtype=np.float64) for x in (q, k, v, g))
    if not (q.shape == k.shape == v.shape == g.shape) or q.ndim != 2:
        raise ValueError("q, k, v, g must all be [S][d]")
    S, d = q.shape
    qr = np.arange(S, dtype=np.int64) if q_rows is None else np.ascontiguousarray(q_rows, np.int64)
    kr = np.arange(S, dtype=np.int64) if k_rows is None else np.ascontiguousarray(k_rows, np.int64)
    for r in (qr, kr):
        if r.size and (r.min() < 0 or r.max() >= S):
            raise ValueError("row index out of range")
    if np.unique(qr).size != qr.size:
        raise ValueError("q_rows must be distinct")
    dq = np.zeros((qr.size, d))
    dk = np.zeros((kr.size, d))
    dv = np.zeros((kr.size, d))
    rc = _load().oracle_attention_backward(
        q.ctypes.data, k.ctypes.data, v.ctypes.data, g.ctypes.data, S, d, float(scale),
        qr.ctypes.data, qr.size, kr.ctypes.data, kr.size,
        dq.ctypes.data, dk.ctypes.data, dv.ctypes.data)
    if rc != 0:
        raise MemoryError("oracle scratch allocation failed")
    return dq, dk, dv


# ---------------------------------------------------------------------------
# Pack / unpack (byte moves by the index formula)
# ---------------------------------------------------------------------------
def pack(src: np.ndarray, P: int, h0: int, Hc: int) -> np.ndarray:
    """``src`` is ``[S][H][d]`` (equivalently ``[P][S/P][H][d]``); returns the
    chunk ``[Hc][S][d]`` with ``dst[j][p*S/P+s] = src[p][s][h0+j]``."""
    src = np.ascontiguousarray(src)
    S, H, d = src.shape
    dst = np.empty((Hc, S, d), dtype=src.dtype)
    rc = _load().oracle_pack(src.ctypes.data, dst.ctypes.data, P, S, H, d, h0, Hc,
                             src.dtype.itemsize)
    if rc != 0:
        raise ValueError("shape not covered by the pack formula")
    return dst


def unpack(src: np.ndarray, dst: np.ndarray, P: int, h0: int) -> np.ndarray:
    """Write chunk ``src`` (``[Hc][S][d]``) into the head slots ``[h0, h0+Hc)``
    of a copy of ``dst`` (``[S][H][d]``); other heads are left as they were."""
    src = np.ascontiguousarray(src)
    out = np.array(dst, copy=True, order="C")
    Hc, S, d = src.shape
    H = out.shape[1]
    if out.shape != (S, H, d) or out.dtype != src.dtype:
        raise ValueError("dst must be [S][H][d] of the same dtype")
    rc = _load().oracle_unpack(src.ctypes.data, out.ctypes.data, P, S, H, d, h0, Hc,
                               src.dtype.itemsize)
    if rc != 0:
        raise ValueError("shape not covered by the unpack formula")
    return out


def forward(q_seq: np.ndarray, k_seq: np.ndarray, v_seq: np.ndarray, P: int,
            scale: float, chunk_sizes) -> np.ndarray:
    """End-to-end single-GPU share: for each chunk, pack Q/K/V, attend, unpack.

    Inputs are ``[S][H][d]``; the output is ``[S][H][d]`` fp64.
    """
    S, H, d = q_seq.shape
    out = np.zeros((S, H, d), dtype=np.float64)
    for h0, hc in zip(chunk_offsets(chunk_sizes), chunk_sizes):
        qc = pack(q_seq, P, h0, hc)
        kc = pack(k_seq, P, h0, hc)
        vc = pack(v_seq, P, h0, hc)
        oc = attention(qc, kc, vc, scale)
        out = unpack(oc, out, P, h0)
    return out
