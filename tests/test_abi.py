"""The C ABI on the CPU: symbols, validation, the partition rule and the plan.

No test here launches a kernel.  Every call either fails validation (which
the library finishes before any HIP call) or has S = 0 (which enqueues
nothing), so fake device addresses are never dereferenced.
"""
import ctypes
import json
import os
import re

import pytest

import paper_2607_01817_amd as hcms

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "hcms.h")

OK, ENULL, ESHAPE, ECHUNKS, EDTYPE, EALIGN, EHIP, EARG, EALIAS, ECAP = 0, -1, -2, -3, -4, -5, -6, -7, -8, -9

# Fake, 16-byte aligned, far-apart device addresses (never dereferenced).
A, B, C_, D_ = 0x10000000, 0x20000000, 0x30000000, 0x40000000


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(hcms.LIB_PATH):
        from paper_2607_01817_amd import build
        build.build()
    return hcms.load()


def declared_symbols():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"HCMS_API\s+(?:const\s+)?\w+\s*\*?\s*(hcms_\w+)\s*\(", text)))


def test_exports_every_declared_symbol(lib):
    syms = declared_symbols()
    assert len(syms) >= 13
    for s in syms:
        assert hasattr(lib, s), f"{s} declared in hcms.h but not exported"


def test_abi_version_and_status_strings(lib):
    assert hcms.abi_version() == 1
    names = {OK: "HCMS_OK", ENULL: "HCMS_ERR_NULL", ESHAPE: "HCMS_ERR_SHAPE",
             ECHUNKS: "HCMS_ERR_CHUNKS", EDTYPE: "HCMS_ERR_DTYPE", EALIGN: "HCMS_ERR_ALIGN",
             EHIP: "HCMS_ERR_HIP", EARG: "HCMS_ERR_ARG", EALIAS: "HCMS_ERR_ALIAS",
             ECAP: "HCMS_ERR_CAPACITY"}
    for code, name in names.items():
        assert lib.hcms_status_string(code).decode() == name


def test_default_chunks_matches_printed_table(lib):
    with open(os.path.join(ROOT, "tests", "golden", "uneven_chunking.json")) as f:
        for c in json.load(f)["cases"]:
            assert hcms.default_chunks(c["H"], c["C"]) == c["sizes"]
    for H in range(1, 41):
        for C in range(1, H + 1):
            s = hcms.default_chunks(H, C)
            assert sum(s) == H and len(s) == C and s == sorted(s, reverse=True)
    with pytest.raises(hcms.HcmsError) as e:
        hcms.default_chunks(3, 4)
    assert e.value.status == ECHUNKS
    assert lib.hcms_default_chunks(4, 2, None) == ENULL


# ---------------------------------------------------------------------------
# Plan: Alg. 1 as an op list, checked by a happens-before analysis
# ---------------------------------------------------------------------------
def happens_before(ops):
    """Transitive happens-before over op indices from stream order and
    record -> wait edges (a wait sees the latest record issued before it)."""
    n = len(ops)
    edges = [set() for _ in range(n)]
    last_on_stream = {}
    last_record = {}
    for i, (kind, stream, chunk, event) in enumerate(ops):
        if stream in last_on_stream:
            edges[last_on_stream[stream]].add(i)
        last_on_stream[stream] = i
        if kind == hcms.OP_RECORD:
            last_record[event] = i
        elif kind == hcms.OP_WAIT:
            assert event in last_record, f"op {i} waits on event {event} never recorded before it"
            edges[last_record[event]].add(i)
    reach = [set() for _ in range(n)]
    for i in reversed(range(n)):
        for j in edges[i]:
            reach[i].add(j)
            reach[i] |= reach[j]
    return reach


def kernel_ops(ops, kind):
    return {op[2]: i for i, op in enumerate(ops) if op[0] == kind}


@pytest.mark.parametrize("C", [1, 2, 3, 5, 10])
def test_pipelined_plan_orders_every_dependency(lib, C):
    ops = hcms.plan(C, hcms.MODE_PIPELINED)
    assert len(ops) == 7 * C + 5
    reach = happens_before(ops)
    pk, at, up = (kernel_ops(ops, k) for k in (hcms.OP_PACK, hcms.OP_ATTENTION, hcms.OP_UNPACK))
    assert sorted(pk) == sorted(at) == sorted(up) == list(range(C))
    for c in range(C):
        assert ops[pk[c]][1] == hcms.STREAM_COPY
        assert ops[at[c]][1] == hcms.STREAM_COMPUTE
        assert ops[up[c]][1] == hcms.STREAM_COPY
        assert at[c] in reach[pk[c]], "attention must wait for its pack"
        assert up[c] in reach[at[c]], "unpack must wait for its attention"
    # The fork: every kernel is after E_main's record on the main stream.
    assert ops[0] == (hcms.OP_RECORD, hcms.STREAM_MAIN, -1, 0)
    for i, op in enumerate(ops):
        if op[0] in (hcms.OP_PACK, hcms.OP_ATTENTION, hcms.OP_UNPACK):
            assert i in reach[0]
    # The join: the main stream's last op is after every kernel.
    last_main = max(i for i, op in enumerate(ops) if op[1] == hcms.STREAM_MAIN)
    for i, op in enumerate(ops):
        if op[0] in (hcms.OP_PACK, hcms.OP_ATTENTION, hcms.OP_UNPACK):
            assert last_main in reach[i]
    # Overlap is allowed: pack c+1 is not ordered after attention c (Lemma of
    # no inter-chunk dependency), and attention c+1 not after unpack c.
    for c in range(C - 1):
        assert pk[c + 1] not in reach[at[c]]
        assert at[c + 1] not in reach[up[c]]
    # Alg. 1 issue order on the copy stream: all packs before any unpack.
    assert max(pk.values()) < min(up.values())


@pytest.mark.parametrize("C", [1, 4])
def test_serial_plan(lib, C):
    ops = hcms.plan(C, hcms.MODE_SERIAL)
    assert len(ops) == 3 * C
    kinds = [op[0] for op in ops]
    assert kinds == [hcms.OP_PACK, hcms.OP_ATTENTION, hcms.OP_UNPACK] * C
    assert all(op[1] == hcms.STREAM_MAIN for op in ops)
    assert [op[2] for op in ops] == [c for c in range(C) for _ in range(3)]


def test_plan_errors(lib):
    assert lib.hcms_plan(0, 1, None, 0) == ECHUNKS
    assert lib.hcms_plan(2, 7, None, 0) == EARG
    ops = (hcms.Op * 3)()
    assert lib.hcms_plan(2, 1, ops, 3) == ECAP
    assert lib.hcms_plan(2, 1, None, 0) == 19


# ---------------------------------------------------------------------------
# Validation before any HIP call
# ---------------------------------------------------------------------------
def _err(lib):
    return lib.hcms_last_error().decode()


@pytest.mark.parametrize("fn", ["hcms_pack", "hcms_unpack"])
def test_pack_validation(lib, fn):
    f = getattr(lib, fn)
    # (src, dst, P, S, H, d, h_begin, h_count, dtype) -> status
    good = [A, B, 4, 512, 4, 64, 0, 2, 1]
    cases = [
        ([None, B] + good[2:], ENULL),
        ([A, None] + good[2:], ENULL),
        ([A, B, 3, 512, 4, 64, 0, 2, 1], ESHAPE),      # S % P != 0
        ([A, B, 0, 512, 4, 64, 0, 2, 1], ESHAPE),      # P < 1
        ([A, B, 4, -4, 4, 64, 0, 2, 1], ESHAPE),       # S < 0
        ([A, B, 4, 512, 0, 64, 0, 2, 1], ESHAPE),      # H < 1
        ([A, B, 4, 512, 4, 6, 0, 2, 1], ESHAPE),       # 24-byte rows
        ([A, B, 4, 512, 4, 48, 0, 2, 0], ESHAPE),      # 96-byte rows
        ([A, B, 4, 512, 4, 64, 3, 2, 1], ECHUNKS),     # range past H
        ([A, B, 4, 512, 4, 64, -1, 2, 1], ECHUNKS),
        ([A, B, 4, 512, 4, 64, 0, 0, 1], ECHUNKS),     # empty chunk
        ([A, B, 4, 512, 4, 64, 0, 2, 2], EDTYPE),
        ([A + 8, B, 4, 512, 4, 64, 0, 2, 1], EALIGN),
        ([A, B + 4, 4, 512, 4, 64, 0, 2, 1], EALIGN),
        ([A, A + 4096, 4, 512, 4, 64, 0, 2, 1], EALIAS),
        ([A, A, 4, 512, 4, 64, 0, 2, 1], EALIAS),
        ([A, B, 4, 2 ** 24, 4, 64, 0, 2, 1], ESHAPE),  # one head > 2 GiB
    ]
    for args, want in cases:
        got = f(*args, None)
        assert got == want, (fn, args, got, _err(lib))
        assert _err(lib)
    # An empty sequence is valid and enqueues nothing (buffers may be NULL).
    assert f(A, B, 4, 0, 4, 64, 0, 2, 1, None) == OK
    assert _err(lib) == ""
    assert f(None, None, 4, 0, 4, 64, 0, 2, 1, None) == OK


def test_attention_validation(lib):
    f = lib.hcms_attention

    def call(q=A, k=B, v=C_, o=D_, S=512, H=4, d=64, scale=0.125, sizes=(2, 2), dtype=1):
        arr = (ctypes.c_int * max(1, len(sizes)))(*sizes) if sizes is not None else None
        return f(q, k, v, o, S, H, d, scale, arr, len(sizes or ()), dtype, None)

    assert call(q=None) == ENULL
    assert call(o=None) == ENULL
    assert call(sizes=None) == ENULL
    assert call(d=96) == ESHAPE
    assert call(d=32) == ESHAPE
    assert call(S=-1) == ESHAPE
    assert call(H=0, sizes=(1,)) == ESHAPE
    assert call(sizes=(2, 1)) == ECHUNKS          # sum != H
    assert call(sizes=(4, 0)) == ECHUNKS          # empty chunk
    assert call(sizes=(1, 1, 1, 1, 0)) == ECHUNKS  # more chunks than heads
    assert call(sizes=(3, -1, 2)) == ECHUNKS
    assert call(dtype=5) == EDTYPE
    assert call(scale=0.0) == EARG
    assert call(scale=-1.0) == EARG
    assert call(scale=float("nan")) == EARG
    assert call(scale=float("inf")) == EARG
    assert call(v=C_ + 2) == EALIGN
    assert call(o=A) == EALIAS
    assert call(o=B + 4096) == EALIAS
    assert call(S=0) == OK  # empty sequence: nothing enqueued
    assert call(S=0, q=None, k=None, v=None, o=None) == OK


def test_forward_and_ctx_validation(lib):
    h = ctypes.c_void_p()
    assert lib.hcms_ctx_create(0, 4, None) == ENULL
    assert lib.hcms_ctx_create(0, 0, ctypes.byref(h)) == ECHUNKS
    assert lib.hcms_ctx_destroy(None) == OK
    sizes = (ctypes.c_int * 2)(2, 2)
    assert lib.hcms_forward(None, A, B, C_, D_, A + 2**24, B + 2**24, C_ + 2**24, D_ + 2**24,
                            4, 512, 4, 64, 0.125, sizes, 2, 1, 1, None, None, None) == ENULL
    assert lib.hcms_ctx_set_timing(None, 1) == ENULL
    buf = (ctypes.c_float * 4)()
    assert lib.hcms_ctx_kernel_ms(None, hcms.OP_ATTENTION, buf, 4) == ENULL


def test_binding_rejects_cpu_tensors(lib):
    import torch
    x = torch.zeros(8, 2, 64)
    with pytest.raises(ValueError):
        hcms.pack(x, 2, 0, 1)
    with pytest.raises(ValueError):
        hcms.attention(x.permute(1, 0, 2), x.permute(1, 0, 2), x.permute(1, 0, 2), 0.1)
