"""The backward path that stores the score gradients (a caller's workspace of
hcms_backward_ds_bytes per head): dK and dV from the key-parallel launch,
which also writes every dS_ij as bf16, and dQ as one product over the stored
dS.  Through the C ABI, against the oracle (MI355X only).

Bars, as for the path without the workspace (tests/test_gpu_backward.py):
  * gradients: max-abs error <= 2e-2 * max|reference| per head and tensor;
  * dK and dV bit-identical to the path without the workspace (same kernel
    arithmetic; only the stores are added);
  * dQ within 5e-3 * max|dQ| of that path's (same bf16 operands up to the
    rounding of P and dP - D, which the two launches form in different
    orders; fp32 sums in different orders);
  * every chunking, every group size (workspace for 1, 2 or all heads) and
    repeated runs bit-identical.
"""
import numpy as np
import pytest
import torch

from paper_2607_01817_amd import inputs
from tests.gpu_util import bits, log

pytestmark = pytest.mark.gpu

GRAD_TOL = 2e-2
DQ_PATHS_TOL = 5e-3


def _data(S, H, d, dtype, seed, sigma=1.0):
    g = torch.Generator().manual_seed(seed)
    q, k, v = (torch.randn(H, S, d, generator=g) * sigma for _ in range(3))
    do = torch.randn(H, S, d, generator=g)
    return [x.to(dtype) for x in (q, k, v, do)]


def _check_grad(got, want, what):
    err = float(np.abs(got - want).max()) if want.size else 0.0
    ref = float(np.abs(want).max()) if want.size else 0.0
    assert err <= GRAD_TOL * ref + 1e-30, f"{what}: max-abs {err:.3e} > {GRAD_TOL} * {ref:.3e}"
    return err / ref if ref else 0.0


def _ws(hcms, S, heads, extra=0):
    n = hcms.backward_ds_bytes(S, 128) * heads + extra
    return torch.empty(n, dtype=torch.uint8, device="cuda")


def _both(hcms, q, k, v, do, scale, chunks=None, heads=None):
    """Gradients without and with a workspace for `heads` heads (all by
    default)."""
    H, S, _ = q.shape
    qd, kd, vd, dod = (x.cuda() for x in (q, k, v, do))
    out, lse = hcms.attention_lse(qd, kd, vd, scale, chunks)
    plain = [t.clone() for t in hcms.attention_backward(qd, kd, vd, out, dod, lse, scale, chunks)]
    ds = _ws(hcms, S, heads or H)
    got = hcms.attention_backward(qd, kd, vd, out, dod, lse, scale, chunks, ds=ds)
    torch.cuda.synchronize()
    return plain, [t.clone() for t in got]


def _compare_paths(plain, got, what):
    assert torch.equal(bits(got[1]), bits(plain[1])), (what, "dk")
    assert torch.equal(bits(got[2]), bits(plain[2])), (what, "dv")
    a, b = got[0].double(), plain[0].double()
    ref = float(b.abs().max())
    err = float((a - b).abs().max())
    assert err <= DQ_PATHS_TOL * ref + 1e-6, f"{what}: dq paths differ by {err:.3e} (max {ref:.3e})"


@pytest.mark.parametrize("S,H,sigma", [
    (1, 1, 1.0), (2, 1, 1.0), (33, 2, 1.0), (200, 2, 1.0), (1000, 1, 0.5), (1000, 1, 2.0),
    (4097, 2, 1.0), (5000, 1, 1.0)])
def test_ds_backward_matches_oracle(hcms, oracle_mod, S, H, sigma):
    """Ragged sequence lengths around the 32-query and 32-key tiles and the
    64-key steps of the dQ product, three value scales (d = 128, bf16)."""
    log(f"[backward ds] S={S} H={H} sigma={sigma}")
    q, k, v, do = _data(S, H, 128, torch.bfloat16, S * 11 + 5, sigma)
    scale = 128 ** -0.5
    plain, (dq, dk, dv) = _both(hcms, q, k, v, do, scale)
    _compare_paths(plain, (dq, dk, dv), f"S={S}")
    if S == 1:
        # One key: P = 1 and dS = dP - D = 0 in exact arithmetic, so the
        # oracle's dQ and dK are exactly 0 and no relative bar applies; the
        # kernels' dP (an MFMA sum) and D (a dot-product sum) may differ in
        # their last bit, which leaves dS, dQ and dK at rounding level.
        assert float(dq.abs().max()) <= 1e-4 and float(dk.abs().max()) <= 1e-4
        return
    worst = 0.0
    for h in range(H):
        Q, K, V, G = (x[h].double().numpy() for x in (q, k, v, do))
        rq, rk, rv = oracle_mod.attention_backward_head(Q, K, V, G, scale)
        for name, got, want in (("dq", dq, rq), ("dk", dk, rk), ("dv", dv, rv)):
            worst = max(worst, _check_grad(got[h].double().cpu().numpy(), want, f"{name} head {h}"))
    log(f"    worst normalised error {worst:.2e}")


@pytest.mark.parametrize("n", range(1, 10))
@pytest.mark.parametrize("ragged", [False, True])
def test_ds_every_block_count(hcms, oracle_mod, n, ragged):
    """Every count of 64-key steps of the dQ product from 1 to 9 (three
    buffers: a remainder of 0 to 2 past whole rounds of them), exact
    (S = 64 n) and ragged (S = 64 n - 41: odd 32-key tile counts, so the last
    step reads a tile of keys past S)."""
    S = 64 * n - 41 if ragged else 64 * n
    log(f"[backward ds blocks] S={S}")
    q, k, v, do = _data(S, 2, 128, torch.bfloat16, 2000 + S, 1.5)
    scale = 128 ** -0.5
    plain, got = _both(hcms, q, k, v, do, scale)
    _compare_paths(plain, got, f"S={S}")
    for h in range(2):
        Q, K, V, G = (x[h].double().numpy() for x in (q, k, v, do))
        rq, rk, rv = oracle_mod.attention_backward_head(Q, K, V, G, scale)
        for name, g, want in zip(("dq", "dk", "dv"), got, (rq, rk, rv)):
            _check_grad(g[h].double().cpu().numpy(), want, f"{name} head {h}")


def test_ds_keys_past_s_with_extreme_statistics(hcms, oracle_mod):
    """Queries whose scores are all far below zero (lse about -2900 in
    log2 units): P of the padding keys past S would overflow if they were
    not taken out, and the dQ product would multiply inf by the zero K rows.
    S = 200 (a partial last 32-key tile)."""
    S = 200
    q, k, v, do = _data(S, 1, 128, torch.bfloat16, 77)
    q = (q.abs() * 6.0).to(torch.bfloat16)
    k = (-k.abs() * 6.0).to(torch.bfloat16)
    scale = 128 ** -0.5
    plain, (dq, dk, dv) = _both(hcms, q, k, v, do, scale)
    for t in (dq, dk, dv):
        assert torch.isfinite(t.float()).all()
    Q, K, V, G = (x[0].double().numpy() for x in (q, k, v, do))
    rq, rk, rv = oracle_mod.attention_backward_head(Q, K, V, G, scale)
    for name, got, want in (("dq", dq, rq), ("dk", dk, rk), ("dv", dv, rv)):
        _check_grad(got[0].double().cpu().numpy(), want, name)


@pytest.mark.parametrize("name", ["small", "wan_p4"])
def test_ds_chunk_and_group_invariance(hcms, name):
    """Every chunking and every group size (workspace for 1, 2 or all heads)
    give the same bits; a workspace below one head runs the path without it."""
    w = inputs.WORKLOADS[name]
    log(f"[backward ds chunks] {name}")
    q, k, v = (x.permute(1, 0, 2).contiguous().cuda() for x in inputs.make_qkv(w))
    do = inputs.make_dout(w).permute(1, 0, 2).contiguous().cuda()
    out, lse = hcms.attention_lse(q, k, v, w.scale)
    plain = [t.clone() for t in hcms.attention_backward(q, k, v, out, do, lse, w.scale)]
    ref = [t.clone() for t in hcms.attention_backward(q, k, v, out, do, lse, w.scale,
                                                      ds=_ws(hcms, w.S, w.H))]
    _compare_paths(plain, ref, name)
    for heads in (1, 2, w.H):
        ds = _ws(hcms, w.S, heads, extra=4096)
        for sizes in w.chunkings:
            got = hcms.attention_backward(q, k, v, out, do, lse, w.scale, sizes, ds=ds)
            for a, b, nm in zip(got, ref, ("dq", "dk", "dv")):
                assert torch.equal(bits(a), bits(b)), (name, heads, sizes, nm)
    small = torch.empty(hcms.backward_ds_bytes(w.S, 128) - 256, dtype=torch.uint8, device="cuda")
    got = hcms.attention_backward(q, k, v, out, do, lse, w.scale, w.chunkings[-1], ds=small)
    for a, b, nm in zip(got, plain, ("dq", "dk", "dv")):
        assert torch.equal(bits(a), bits(b)), (name, "below one head", nm)


@pytest.mark.parametrize("name", ["small", "wan_p4"])
def test_ds_pipeline_bitwise_across_modes_and_chunkings(hcms, name):
    """hcms_backward with the context's workspace (two regions of one head
    each) equals the direct backward with a one-head workspace, bitwise, in
    every mode and chunking."""
    w = inputs.WORKLOADS[name]
    qs, ks, vs = (x.cuda() for x in inputs.make_qkv(w))
    dos = inputs.make_dout(w).cuda()
    log(f"[backward ds pipeline] {name}")
    hm = [x.permute(1, 0, 2).contiguous() for x in (qs, ks, vs, dos)]
    out, lse = hcms.attention_lse(hm[0], hm[1], hm[2], w.scale)
    ref = [t.permute(1, 0, 2).contiguous()
           for t in hcms.attention_backward(hm[0], hm[1], hm[2], out, hm[3], lse, w.scale,
                                            ds=_ws(hcms, w.S, 1))]
    ctx = hcms.Context(max_chunks=16)
    ctx.set_ds_workspace(_ws(hcms, w.S, 2))
    for sizes in w.chunkings:
        for mode in (hcms.MODE_SERIAL, hcms.MODE_PIPELINED, hcms.MODE_INLINE, hcms.MODE_LANES,
                     hcms.MODE_FUSED, hcms.MODE_AUTO):
            ws = [torch.empty_like(hm[0]) for _ in range(4)]
            lse2 = torch.empty_like(lse)
            ctx.forward(qs, ks, vs, w.P, w.scale, sizes, mode=mode, workspaces=ws, lse=lse2)
            got = ctx.backward(dos, w.P, w.scale, sizes, ws, lse2, mode=mode)
            for a, b, nm in zip(got, ref, ("dq", "dk", "dv")):
                assert torch.equal(bits(a), bits(b)), (name, sizes, mode, nm)
            if mode == hcms.MODE_AUTO and len(sizes) >= 2:
                # With the workspace, auto overlaps chunks in two lanes.
                assert ctx.last_mode == hcms.MODE_LANES, (name, sizes, ctx.last_mode)
    ctx.set_ds_workspace(None)
    ctx.close()
