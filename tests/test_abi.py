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
    assert hcms.abi_version() == 3
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
    record -> wait edges (a wait sees the latest record issued before it).
    An op on STREAM_IN_ATTENTION runs inside the launch of the next ATTENTION
    op on the main stream: after the main-stream op before that launch and
    before the main-stream op after it, unordered against the launch's
    attention."""
    n = len(ops)
    edges = [set() for _ in range(n)]
    last_on_stream = {}
    last_record = {}
    main = [i for i, op in enumerate(ops) if op[1] == hcms.STREAM_MAIN]
    for i, (kind, stream, chunk, event) in enumerate(ops):
        if stream == hcms.STREAM_IN_ATTENTION:
            host = next(j for j in main if j > i)
            assert ops[host][0] == hcms.OP_ATTENTION, f"op {i} rides in no attention launch"
            before = [j for j in main if j < host]
            after = [j for j in main if j > host]
            if before:
                edges[before[-1]].add(i)
            if after:
                edges[i].add(after[0])
            continue
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


def check_pipelined_dependencies(ops, C, attention_stream):
    """The dependencies of Alg. 1 hold in a plan, whatever streams run what:
    pack c -> attention c -> unpack c, every kernel ordered after the main
    stream's position at the call and before its position at the return,
    and nothing else forced between neighbouring chunks (lemma of no
    inter-chunk dependency)."""
    reach = happens_before(ops)
    pk, at, up = (kernel_ops(ops, k) for k in (hcms.OP_PACK, hcms.OP_ATTENTION, hcms.OP_UNPACK))
    assert sorted(pk) == sorted(at) == sorted(up) == list(range(C))
    for c in range(C):
        assert attention_stream is None or ops[at[c]][1] == attention_stream
        assert at[c] in reach[pk[c]], "attention must wait for its pack"
        assert up[c] in reach[at[c]], "unpack must wait for its attention"
    kernels = [i for i, op in enumerate(ops)
               if op[0] in (hcms.OP_PACK, hcms.OP_ATTENTION, hcms.OP_UNPACK)]
    main = [i for i, op in enumerate(ops) if op[1] == hcms.STREAM_MAIN]
    first_main, last_main = main[0], main[-1]
    for i in kernels:   # fork: after the main stream's first op (or it)
        assert i == first_main or i in reach[first_main]
    for i in kernels:   # join: the main stream's last op is after every kernel
        assert i == last_main or last_main in reach[i]
    for c in range(C - 1):
        assert pk[c + 1] not in reach[at[c]]
        assert at[c + 1] not in reach[up[c]]
    # Every wait names an event recorded before it in issue order (checked by
    # happens_before) and every event is recorded at most once per call.
    recorded = [op[3] for op in ops if op[0] == hcms.OP_RECORD]
    assert len(recorded) == len(set(recorded))
    return pk, at, up


@pytest.mark.parametrize("C", [1, 2, 3, 5, 10])
def test_pipelined_plan_orders_every_dependency(lib, C):
    ops = hcms.plan(C, hcms.MODE_PIPELINED)
    assert len(ops) == 7 * C + 5
    assert ops[0] == (hcms.OP_RECORD, hcms.STREAM_MAIN, -1, 0)
    pk, at, up = check_pipelined_dependencies(ops, C, hcms.STREAM_COMPUTE)
    for c in range(C):
        assert ops[pk[c]][1] == hcms.STREAM_COPY
        assert ops[up[c]][1] == hcms.STREAM_COPY
    # Alg. 1 issue order on the copy stream: all packs before any unpack.
    assert max(pk.values()) < min(up.values())


@pytest.mark.parametrize("C", [2, 3, 5, 10])
def test_inline_plan_orders_every_dependency(lib, C):
    ops = hcms.plan(C, hcms.MODE_INLINE)
    assert len(ops) == 3 * C + 8
    pk, at, up = check_pipelined_dependencies(ops, C, hcms.STREAM_MAIN)
    assert ops[pk[0]][1] == hcms.STREAM_MAIN and ops[up[C - 1]][1] == hcms.STREAM_MAIN
    for c in range(1, C):
        assert ops[pk[c]][1] == hcms.STREAM_COPY
        assert ops[up[c - 1]][1] == hcms.STREAM_COPY
    assert all(op[1] != hcms.STREAM_COMPUTE for op in ops)
    reach = happens_before(ops)
    # Packs 1..C-1 start after chunk 0's and overlap attention 0; unpacks
    # 0..C-2 overlap the last attention.
    for c in range(1, C):
        assert pk[c] in reach[pk[0]] and pk[c] not in reach[at[0]]
        assert up[c - 1] not in reach[at[C - 1]] and at[C - 1] not in reach[up[c - 1]]
    # Four synchronisations on the main stream, whatever C is.
    syncs = [op for op in ops if op[1] == hcms.STREAM_MAIN and op[0] in (hcms.OP_RECORD, hcms.OP_WAIT)]
    assert len(syncs) == 4


@pytest.mark.parametrize("C", [2, 3, 5, 10])
def test_lanes_plan_orders_every_dependency(lib, C):
    ops = hcms.plan(C, hcms.MODE_LANES)
    assert len(ops) == 3 * C + 4
    pk, at, up = check_pipelined_dependencies(ops, C, None)
    for c in range(C):
        lane = hcms.STREAM_COMPUTE if c % 2 else hcms.STREAM_MAIN
        assert ops[pk[c]][1] == ops[at[c]][1] == ops[up[c]][1] == lane
    assert all(op[1] != hcms.STREAM_COPY for op in ops)
    reach = happens_before(ops)
    # Chunks of different lanes are unordered: their kernels may overlap.
    for c in range(C):
        for c2 in range(c + 1, C):
            if (c2 - c) % 2 and c > 0:
                for a in (pk[c], at[c], up[c]):
                    for b in (pk[c2], at[c2], up[c2]):
                        assert b not in reach[a] and a not in reach[b], (c, c2)
    # The second lane starts after chunk 0's pack only.
    assert pk[1] in reach[pk[0]] and pk[1] not in reach[at[0]]
    # Four synchronisations, whatever C is.
    assert sum(op[0] in (hcms.OP_RECORD, hcms.OP_WAIT) for op in ops) == 4


@pytest.mark.parametrize("C", [2, 3, 5, 10])
def test_fused_plan_orders_every_dependency(lib, C):
    ops = hcms.plan(C, hcms.MODE_FUSED)
    assert len(ops) == 3 * C
    pk, at, up = check_pipelined_dependencies(ops, C, hcms.STREAM_MAIN)
    # One stream, no events.
    assert all(op[0] not in (hcms.OP_RECORD, hcms.OP_WAIT) for op in ops)
    assert {op[1] for op in ops} == {hcms.STREAM_MAIN, hcms.STREAM_IN_ATTENTION}
    assert ops[pk[0]][1] == hcms.STREAM_MAIN and ops[up[C - 1]][1] == hcms.STREAM_MAIN
    reach = happens_before(ops)
    for c in range(C):
        # Pack c + 1 and unpack c - 1 ride in attention c's launch: they
        # overlap it and nothing else.
        riders = [pk[c + 1]] if c + 1 < C else []
        riders += [up[c - 1]] if c >= 1 else []
        assert len(riders) == (c + 1 < C) + (c >= 1)
        for r in riders:
            assert ops[r][1] == hcms.STREAM_IN_ATTENTION
            assert at[c] not in reach[r] and r not in reach[at[c]]
            assert min(i for i in at.values() if i > r) == at[c]
    # The two chunk slots can be reused.
    check_slot_reuse(ops, C)


def test_one_gpu_plans_with_one_chunk_are_serial(lib):
    assert hcms.plan(1, hcms.MODE_LANES) == hcms.plan(1, hcms.MODE_SERIAL)
    assert hcms.plan(1, hcms.MODE_INLINE) == hcms.plan(1, hcms.MODE_SERIAL)
    assert hcms.plan(1, hcms.MODE_FUSED) == hcms.plan(1, hcms.MODE_SERIAL)


# Rounds of attention workgroups, worked by hand for 256 CUs.  d = 128: 256
# queries per workgroup, one per CU; d = 64: 128 queries, two per CU.
# Where pooling saves no round, d = 128 bf16 runs the fused plan if some
# launch's last round leaves at least 1/8 of the slots idle, the serial one
# if none does; the other kernels run the inline plan if chunk 0's launch
# leaves that many idle, the serial one otherwise.  (want bf16, want fp32)
@pytest.mark.parametrize("S,d,sizes,want", [
    (56160, 128, (2, 2, 1), ("fused", "inline")),   # 220 tiles: 2+2+1 = ceil(1100/256); idle 72, 72, 36
    (56160, 128, (1, 1, 1, 1, 1), ("fused", "inline")),  # 5 x 1 = 5; idle 36 each
    (32760, 128, (5, 5), ("lanes",) * 2),           # 128 tiles: 3+3 = 6 > ceil(1280/256) = 5
    (32760, 128, (4, 3, 3), ("lanes",) * 2),        # 2+2+2 = 6 > 5
    (32760, 128, (2,) * 5, ("serial",) * 2),        # 256 workgroups each: no idle CU anywhere
    (100000, 128, (10, 10, 10, 10), ("lanes",) * 2),  # 391 tiles: 4 x 16 = 64 > ceil(15640/256) = 62
    (100000, 128, (14, 13, 13), ("fused", "inline")),  # 22+20+20 = 62; chunk 0 idles 158
    (65536, 128, (2, 2), ("serial",) * 2),          # 256 tiles: 512 workgroups, no idle CU
    (4096, 128, (3, 3, 2), ("lanes",) * 2),         # 16 tiles: 1+1+1 = 3 > ceil(128/256) = 1
    (4096, 64, (3, 3, 2), ("lanes",) * 2),          # 32 tiles, 512 slots: 3 > 1
    (32768, 64, (4, 4), ("serial",) * 2),           # 256 tiles, 512 slots: 2+2 = 4, no idle slot
    (32768, 64, (3, 5), ("lanes",) * 2),            # 2+3 = 5 > ceil(2048/512) = 4
    (8192, 64, (9, 16), ("inline",) * 2),           # 64 tiles: 576 + 1024 = 2+2 = ceil(1600/512); chunk 0 idles 448
    (8192, 64, (16, 9), ("serial",) * 2),           # chunk 0 fills two rounds exactly
    (56160, 128, (5,), ("serial",) * 2),            # one chunk
    (0, 128, (2, 2), ("serial",) * 2),              # nothing to launch
])
def test_auto_mode_by_rounds(lib, S, d, sizes, want):
    modes = {"serial": hcms.MODE_SERIAL, "inline": hcms.MODE_INLINE, "lanes": hcms.MODE_LANES,
             "fused": hcms.MODE_FUSED}
    assert hcms.auto_mode(S, d, sizes, 256) == modes[want[0]]
    # fp32 storage takes the register-staged kernel, whose launches carry no
    # copies: the inline plan in their place.
    assert hcms.auto_mode(S, d, sizes, 256, dtype=hcms.FP32) == modes[want[1]]


def test_auto_mode_validation(lib):
    sizes = (ctypes.c_int * 2)(2, 2)
    assert lib.hcms_auto_mode(-1, 128, 0, sizes, 2, 256) == ESHAPE
    assert lib.hcms_auto_mode(100, 96, 0, sizes, 2, 256) == ESHAPE
    assert lib.hcms_auto_mode(100, 128, 2, sizes, 2, 256) == EDTYPE
    assert lib.hcms_auto_mode(100, 128, 0, sizes, 2, 0) == EARG
    assert lib.hcms_auto_mode(100, 128, 0, None, 2, 256) == ENULL
    assert lib.hcms_auto_mode(100, 128, 0, sizes, 0, 256) == ECHUNKS
    bad = (ctypes.c_int * 2)(2, 0)
    assert lib.hcms_auto_mode(100, 128, 0, bad, 2, 256) == ECHUNKS
    assert lib.hcms_ctx_last_mode(None) == ENULL
    assert lib.hcms_ctx_num_cu(None) == ENULL


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
    assert lib.hcms_plan(2, hcms.MODE_AUTO, None, 0) == EARG   # no fixed plan
    assert lib.hcms_plan(2, 8, None, 0) == EARG
    assert lib.hcms_plan(2, hcms.MODE_FUSED, None, 0) == 6
    assert lib.hcms_plan(2, hcms.MODE_SLOTS, None, 0) == 19
    assert lib.hcms_plan(2, hcms.MODE_INLINE, None, 0) == 14
    assert lib.hcms_plan(2, hcms.MODE_LANES, None, 0) == 10
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
    assert lib.hcms_forward(None, A, B, C_, D_, A + 2**24, B + 2**24, C_ + 2**24, D_ + 2**24, None,
                            4, 512, 4, 64, 0.125, sizes, 2, 1, 1, None, None, None) == ENULL
    assert lib.hcms_backward(None, A, B, C_, D_, A, B, C_, D_, None, A, B, C_, D_, None,
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


def test_binding_checks_sizes_before_any_launch(lib):
    """The C ABI sees raw pointers, so the binding checks every tensor's
    shape and dtype before its device: an undersized or mistyped output,
    buffer or weight raises ValueError naming it, on the CPU, before the
    library is called (the methods run on a stand-in context object that has
    no library handle, so reaching the call would raise something else)."""
    import torch
    bf = torch.bfloat16
    S, H, d, D, P = 24, 2, 64, 128, 2
    grid, pairs = (2, 3, 4), (12, 10, 10)
    n_table = hcms.load().hcms_rope_table_entries(_ints(grid), _ints(pairs), 3)
    x = torch.zeros(S, D, dtype=bf)
    w_qkv = torch.zeros(3 * H * d, D, dtype=bf)
    w_o = torch.zeros(D, H * d, dtype=bf)
    table = torch.zeros(n_table, 2)
    seq = [torch.zeros(S, H, d, dtype=bf) for _ in range(4)]

    def layer(**kw):
        a = dict(x=x, w_qkv=w_qkv, w_o=w_o, P=P, H=H, d=d, scale=0.125, chunk_sizes=(1, 1),
                 table=table, grid=grid, axis_pairs=pairs, out=torch.zeros(S, D, dtype=bf),
                 buffers=seq)
        a.update(kw)
        return hcms.Context.layer_forward(object(), **a)

    for kw, name in ((dict(w_qkv=w_qkv[:-1]), "w_qkv"), (dict(w_o=w_o[:, :-8]), "w_o"),
                     (dict(w_o=w_o.float()), "w_o"), (dict(out=torch.zeros(S - 1, D, dtype=bf)), "out"),
                     (dict(buffers=seq[:3] + [torch.zeros(S, H, d - 8, dtype=bf)]), "o_seq"),
                     (dict(buffers=[seq[0].float()] + seq[1:]), "q_seq"),
                     (dict(table=table[:-1]), "table"), (dict(table=table.double()), "table")):
        with pytest.raises(ValueError, match=name):
            layer(**kw)
    with pytest.raises(ValueError, match="GPU tensor"):   # every size right: the device check
        layer()

    def qkv(**kw):
        a = dict(x=x, w_qkv=w_qkv, H=H, d=d, table=table, grid=grid, axis_pairs=pairs,
                 out=tuple(seq[:3]))
        a.update(kw)
        return hcms.qkv_projection(**a)

    for kw, name in ((dict(w_qkv=torch.zeros(3 * H * d, D - 64, dtype=bf)), "w_qkv"),
                     (dict(out=(seq[0], seq[1], seq[2][:-1])), "v_seq"),
                     (dict(table=table[1:]), "table")):
        with pytest.raises(ValueError, match=name):
            qkv(**kw)

    slots = [torch.zeros(2, 1, S, d, dtype=bf) for _ in range(4)]

    def fslots(**kw):
        a = dict(q_seq=seq[0], k_seq=seq[1], v_seq=seq[2], P=P, scale=0.125, chunk_sizes=(1, 1),
                 out=seq[3], slots=slots)
        a.update(kw)
        return hcms.Context.forward_slots(object(), **a)

    for kw, name in ((dict(out=torch.zeros(S, H, d - 8, dtype=bf)), "out"),
                     (dict(out=seq[3].float()), "out"), (dict(v_seq=seq[2].float()), "v_seq"),
                     (dict(slots=slots[:3] + [torch.zeros(2, 1, S - 2, d, dtype=bf)]), "slot")):
        with pytest.raises(ValueError, match=name):
            fslots(**kw)


def test_training_forward_and_backward_validation(lib):
    sizes = (ctypes.c_int * 2)(2, 2)
    E, F, G_, H_ = 0x50000000, 0x60000000, 0x70000000, 0x80000000
    L, Dl = 0x90000000, 0x98000000   # [H][S] fp32 statistics, far from the tensors

    def fwd(lse=L, q=A, S=512):
        return lib.hcms_attention_lse(q, B, C_, D_, lse, S, 4, 64, 0.125, sizes, 2, 1, None)

    assert fwd(lse=None) == ENULL
    assert fwd(lse=L + 2) == EALIGN
    assert fwd(lse=A + 64) == EALIAS
    assert fwd(S=0, lse=None, q=None) == OK

    def bwd(dout=E, dq=F, dk=G_, dv=H_, lse=L, delta=Dl, S=512, d=64, ds=None, ds_bytes=0):
        return lib.hcms_attention_backward(A, B, C_, D_, dout, lse, dq, dk, dv, delta, ds,
                                           ds_bytes, S, 4, d, 0.125, sizes, 2, 1, None)

    assert bwd(dout=None) == ENULL
    assert bwd(dq=None) == ENULL
    assert bwd(lse=None) == ENULL
    assert bwd(delta=None) == ENULL
    assert bwd(dk=G_ + 8) == EALIGN
    assert bwd(delta=Dl + 1) == EALIGN
    assert bwd(dq=A) == EALIAS          # a gradient over an input
    assert bwd(dk=F + 64) == EALIAS     # two gradients overlap
    assert bwd(delta=L) == EALIAS       # statistics overlap each other
    assert bwd(delta=F + 16) == EALIAS  # workspace over a gradient
    assert bwd(d=96) == ESHAPE
    assert bwd(S=0, dout=None, dq=None, dk=None, dv=None, lse=None, delta=None) == OK
    # The score-gradient workspace: size, alignment, overlaps.
    W = 0xA0000000
    assert bwd(ds=W, ds_bytes=-1) == EARG
    assert bwd(ds=W + 16, ds_bytes=1 << 20) == EALIGN
    assert bwd(ds=F - 256, ds_bytes=1 << 20) == EALIAS   # over a gradient
    assert bwd(ds=A, ds_bytes=1 << 20) == EALIAS         # over an input
    assert bwd(ds=L - 256, ds_bytes=1 << 20) == EALIAS   # over lse
    assert bwd(ds=Dl, ds_bytes=1 << 20) == EALIAS        # over delta
    assert bwd(S=0, dout=None, dq=None, dk=None, dv=None, lse=None, delta=None, ds=W + 16,
               ds_bytes=1) == OK


def test_backward_ds_bytes(lib):
    """Workspace per head of the path that stores the score gradients:
    ceil(S / 256) groups of 8 query blocks x 8 ceil(S / 256) key tiles x
    16 KiB at d = 128 with bf16 storage, none elsewhere."""
    out = ctypes.c_int64()
    for S, want in ((56160, 220 * 1760 * 16384), (1, 8 * 16384), (0, 0),
                    (257, 2 * 16 * 16384), (32760, 128 * 1024 * 16384)):
        assert lib.hcms_backward_ds_bytes(S, 128, 0, ctypes.byref(out)) == OK
        assert out.value == want, (S, out.value, want)
    assert hcms.backward_ds_bytes(56160, 128) == 220 * 1760 * 16384
    for d, dt in ((64, 0), (128, 1), (64, 1)):
        assert lib.hcms_backward_ds_bytes(4096, d, dt, ctypes.byref(out)) == OK and out.value == 0
    assert lib.hcms_backward_ds_bytes(-1, 128, 0, ctypes.byref(out)) == ESHAPE
    assert lib.hcms_backward_ds_bytes(64, 128, 7, ctypes.byref(out)) == EDTYPE
    assert lib.hcms_backward_ds_bytes(64, 128, 0, None) == ENULL
    assert lib.hcms_ctx_set_ds_workspace(None, None, 0) == ENULL


def test_noalloc_backward_validation(lib):
    """The entry point without a delta workspace validates like
    hcms_attention_backward and rejects S * H past its scratch array."""
    sizes = (ctypes.c_int * 2)(2, 2)
    E, F, G_, H_ = 0x50000000, 0x60000000, 0x70000000, 0x80000000
    L = 0x90000000

    def bwd(dout=E, dq=F, dk=G_, dv=H_, lse=L, S=512, H=4, d=64, sz=sizes, n=2):
        return lib.hcms_attention_backward_noalloc(A, B, C_, D_, dout, lse, dq, dk, dv, S, H, d,
                                                   0.125, sz, n, 1, None)

    assert bwd(dout=None) == ENULL
    assert bwd(lse=None) == ENULL
    assert bwd(dk=G_ + 8) == EALIGN
    assert bwd(dq=A) == EALIAS
    assert bwd(lse=F + 16) == EALIAS
    assert bwd(d=96) == ESHAPE
    assert bwd(S=0, dout=None, dq=None, dk=None, dv=None, lse=None) == OK
    # S * H one past the limit, on fake far-apart [H][S][64] bf16 tensors.
    limit = hcms.NOALLOC_DELTA_MAX
    S = limit // 2 + 8
    span = 2 * S * 64 * 2
    p = [(1 << 40) + i * span for i in range(9)]
    one = (ctypes.c_int * 2)(1, 1)
    st = lib.hcms_attention_backward_noalloc(*p, S, 2, 64, 0.125, one, 2, 0, None)
    assert st == ECAP, hcms.load().hcms_last_error()
    assert b"scratch" in lib.hcms_last_error()


# ---------------------------------------------------------------------------
# Layer neighbours: projection GEMM, rotation table, QKV projection, layer
# ---------------------------------------------------------------------------
def _ints(xs):
    return (ctypes.c_int * max(1, len(xs)))(*xs)


def test_linear_validation(lib):
    f = lib.hcms_linear

    def call(x=A, w=B, y=C_, M=300, N=264, K=128, dtype=0):
        return f(x, w, y, M, N, K, dtype, None)

    assert call(dtype=3) == EDTYPE
    assert call(K=0) == ESHAPE
    assert call(K=100) == ESHAPE            # not a multiple of 64
    assert call(K=2**21) == ESHAPE
    assert call(N=12) == ESHAPE             # not a multiple of 8
    assert call(M=-1) == ESHAPE
    assert call(x=None) == ENULL
    assert call(y=None) == ENULL
    assert call(w=B + 8) == EALIGN
    assert call(y=A) == EALIAS
    assert call(y=B + 1024) == EALIAS
    assert call(M=0) == OK                  # nothing enqueued
    assert call(M=0, x=None, y=None) == OK
    assert call(N=0, w=None, y=None) == OK


def test_rope_table_validation(lib):
    assert lib.hcms_rope_table_entries(_ints((36, 30, 52)), _ints((22, 21, 21)), 3) == \
        36 * 22 + 30 * 21 + 52 * 21
    assert lib.hcms_rope_table_entries(_ints((512,)), _ints((32,)), 1) == 512 * 32
    assert lib.hcms_rope_table_entries(None, _ints((1,)), 1) == ENULL
    assert lib.hcms_rope_table_entries(_ints((4,)), _ints((1,)), 0) == EARG
    assert lib.hcms_rope_table_entries(_ints((1,) * 5), _ints((1,) * 5), 5) == EARG
    assert lib.hcms_rope_table_entries(_ints((4, 0)), _ints((1, 1)), 2) == ESHAPE
    assert lib.hcms_rope_table_entries(_ints((4, 4)), _ints((1, 0)), 2) == ESHAPE
    assert lib.hcms_rope_table_entries(_ints((2**16, 2**16)), _ints((1, 1)), 2) == ESHAPE
    g, p = _ints((4, 6)), _ints((8, 8))
    assert lib.hcms_rope_table(None, g, p, 2, 1e4, None) == ENULL
    assert lib.hcms_rope_table(A + 4, g, p, 2, 1e4, None) == EALIGN
    assert lib.hcms_rope_table(A, g, p, 2, 1.0, None) == EARG
    assert lib.hcms_rope_table(A, g, p, 2, float("inf"), None) == EARG


def test_qkv_projection_validation(lib):
    f = lib.hcms_qkv_projection
    big = 2**26

    def call(x=A, w=B, table=C_, grid=(4, 6, 10), pairs=(12, 10, 10), q=D_, k=D_ + big,
             v=D_ + 2 * big, S=240, D=256, H=4, d=64, dtype=0):
        return f(x, w, table, _ints(grid), _ints(pairs), len(grid), q, k, v, S, D, H, d, dtype, None)

    assert call(d=12) == ESHAPE                 # not a multiple of 8
    assert call(H=0) == ESHAPE
    assert call(D=100) == ESHAPE                # K of the GEMM
    assert call(grid=(4, 6, 11)) == ESHAPE      # 264 tokens, not 240
    assert call(pairs=(12, 10, 9)) == ESHAPE    # 31 pairs, not 32
    assert call(k=None) == ENULL
    assert call(v=D_ + 2 * big + 4) == EALIGN
    assert call(table=C_ + 8) == EALIGN
    assert call(k=D_ + 1024) == EALIAS          # outputs overlap
    assert call(q=A) == EALIAS                  # output overlaps x
    assert call(table=D_ + 4096) == EALIAS      # table overlaps q
    # x right after q's [S][H][d] bytes overlaps nothing: the check goes on to
    # the table's alignment (q is not a [S][3 H d] matrix).
    assert call(x=D_ + 240 * 4 * 64 * 2, table=C_ + 8) == EALIGN
    assert call(S=0, x=None, q=None, k=None, v=None) == OK
    # Without a table, grid and pairs are not looked at.
    assert f(A, B, None, None, None, 0, D_, D_ + big, D_ + 2 * big, 0, 256, 4, 64, 0, None) == OK


def test_layer_forward_validation(lib):
    big = 2**26
    sizes = _ints((2, 2))

    def call(ctx=None, x=A, wq=B, wo=B + big, table=C_, y=C_ + big, S=240, D=256, H=4, d=64,
             grid=(4, 6, 10), pairs=(12, 10, 10)):
        t = [D_ + i * big for i in range(8)]
        return lib.hcms_layer_forward(ctx, x, wq, wo, table, _ints(grid), _ints(pairs), len(grid),
                                      y, *t, 4, S, D, H, d, 0.125, sizes, 2, 0, 1, None, None, None)

    assert call() == ENULL                      # no context
    assert call(grid=(4, 6, 11)) == ESHAPE      # checked before the context
    assert call(D=100) == ESHAPE


# ---------------------------------------------------------------------------
# Two chunk slots: the slots plan and hcms_forward_slots
# ---------------------------------------------------------------------------
def check_slot_reuse(ops, C):
    """Chunk c + 2 reuses chunk c's slot: its pack must come after attention c
    (which reads the Q, K, V slot) and its attention after unpack c (which
    reads the O slot)."""
    reach = happens_before(ops)
    pk, at, up = (kernel_ops(ops, k) for k in (hcms.OP_PACK, hcms.OP_ATTENTION, hcms.OP_UNPACK))
    for c in range(C - 2):
        assert pk[c + 2] in reach[at[c]], f"pack {c + 2} may overwrite slot {c % 2} under attention {c}"
        assert at[c + 2] in reach[up[c]], f"attention {c + 2} may overwrite O slot {c % 2} under unpack {c}"


@pytest.mark.parametrize("C", [1, 2, 3, 5, 10])
def test_slots_plan_orders_every_dependency_and_slot_reuse(lib, C):
    ops = hcms.plan(C, hcms.MODE_SLOTS)
    assert len(ops) == 7 * C + 5
    pk, at, up = check_pipelined_dependencies(ops, C, hcms.STREAM_COMPUTE)
    for c in range(C):
        assert ops[pk[c]][1] == ops[up[c]][1] == hcms.STREAM_COPY
    check_slot_reuse(ops, C)
    reach = happens_before(ops)
    # The copy stream still overlaps: pack c + 1 and unpack c - 1 are not
    # ordered against attention c.
    for c in range(1, C - 1):
        assert at[c] not in reach[pk[c + 1]] and pk[c + 1] not in reach[at[c]]
        assert at[c] not in reach[up[c - 1]] and up[c - 1] not in reach[at[c]]


@pytest.mark.parametrize("mode", ["serial", "lanes"])
@pytest.mark.parametrize("C", [2, 3, 5, 10])
def test_serial_and_lanes_plans_allow_slot_reuse(lib, mode, C):
    check_slot_reuse(hcms.plan(C, getattr(hcms, "MODE_" + mode.upper())), C)


@pytest.mark.parametrize("mode", ["pipelined", "inline"])
def test_pipelined_and_inline_plans_do_not_allow_slot_reuse(lib, mode):
    with pytest.raises(AssertionError):
        check_slot_reuse(hcms.plan(5, getattr(hcms, "MODE_" + mode.upper())), 5)


def test_forward_slots_validation(lib):
    sizes = (ctypes.c_int * 3)(3, 3, 2)

    def call(slot_heads=3, mode=hcms.MODE_SLOTS):
        return lib.hcms_forward_slots(None, A, B, C_, D_, A + 2**24, B + 2**24, C_ + 2**24,
                                      D_ + 2**24, slot_heads, 8, 4096, 8, 128, 0.088, sizes, 3, 0,
                                      mode, None, None, None)

    assert call(slot_heads=0) == ECHUNKS
    assert call() == ENULL          # no context (checked after slot_heads)
