"""Parity of the attention backward (and the training forward's statistic)
with the oracle, through the C ABI (MI355X only).

Bars:
  * gradients: max-abs error <= 2e-2 * max|reference| per head and tensor.
    Operands are rounded to bf16 for the MFMAs (2^-9 relative each) and P and
    dS to bf16 before their products, with fp32 accumulation; measured errors
    are 2.5e-3 to 7.5e-3 of max|reference| (fp32 storage highest, since its
    inputs are rounded while the oracle reads them exactly), so the bar leaves
    a margin of about 3.  An absolute bar cannot be used: gradients scale with
    the data (max|dQ| is 13 at sigma = 2).
  * lse: |error| <= 1e-3 * |reference| (measured at most 3e-4).
  * every chunking and repeated runs bit-identical.
"""
import numpy as np
import pytest
import torch

from paper_2607_01817_amd import inputs
from tests.gpu_util import bits, log

pytestmark = pytest.mark.gpu

GRAD_TOL = 2e-2
LSE_TOL = 1e-3


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


def _run(hcms, q, k, v, do, scale, chunks=None):
    qd, kd, vd, dod = (x.cuda() for x in (q, k, v, do))
    out, lse = hcms.attention_lse(qd, kd, vd, scale, chunks)
    dq, dk, dv = hcms.attention_backward(qd, kd, vd, out, dod, lse, scale, chunks)
    torch.cuda.synchronize()
    return out, lse, dq, dk, dv


@pytest.mark.parametrize("S,H,d,dtype,sigma", [
    (1, 1, 128, torch.bfloat16, 1.0), (2, 1, 64, torch.bfloat16, 1.0),
    (33, 2, 128, torch.bfloat16, 1.0), (127, 1, 64, torch.bfloat16, 1.0),
    (129, 2, 128, torch.float32, 1.0), (200, 2, 128, torch.bfloat16, 1.0),
    (300, 1, 64, torch.float32, 1.0), (1000, 1, 128, torch.bfloat16, 0.5),
    (1000, 1, 128, torch.bfloat16, 2.0), (4097, 1, 128, torch.bfloat16, 1.0)])
def test_backward_matches_oracle(hcms, oracle_mod, S, H, d, dtype, sigma):
    """Ragged sequence lengths around the 32-query and 64-key blocks and the
    128-row tiles, both head dims, both storage types, three value scales."""
    log(f"[backward] S={S} H={H} d={d} {dtype} sigma={sigma}")
    q, k, v, do = _data(S, H, d, dtype, S * 7 + d, sigma)
    scale = d ** -0.5
    out, lse, dq, dk, dv = _run(hcms, q, k, v, do, scale)
    worst = 0.0
    for h in range(H):
        Q, K, V, G = (x[h].double().numpy() for x in (q, k, v, do))
        lw = oracle_mod.lse_head(Q, K, scale)
        gl = lse[h].double().cpu().numpy()
        assert np.all(np.abs(gl - lw) <= LSE_TOL * np.abs(lw) + 1e-6), (h, np.abs(gl - lw).max())
        rq, rk, rv = oracle_mod.attention_backward_head(Q, K, V, G, scale)
        for name, got, want in (("dq", dq, rq), ("dk", dk, rk), ("dv", dv, rv)):
            worst = max(worst, _check_grad(got[h].double().cpu().numpy(), want, f"{name} head {h}"))
    log(f"    worst normalised error {worst:.2e}")
    if S == 1:   # one key: P = 1, dS = 0
        assert torch.count_nonzero(dq) == 0 and torch.count_nonzero(dk) == 0
        assert torch.equal(dv.cpu(), do)


@pytest.mark.parametrize("n", range(1, 10))
@pytest.mark.parametrize("ragged", [False, True])
def test_backward_every_block_count(hcms, oracle_mod, n, ragged):
    """d = 128 bf16: every count of 64-key blocks from 1 to 9 (the dQ kernel's
    key loop, four blocks per pass plus a remainder of 0 to 3) and of 32-query
    blocks from 1 to 18 (the dK/dV kernel's query loop), ragged (S = 64 n - 41:
    n key blocks, 2 n - 1 query blocks, both tails partial) and exact (S = 64 n)."""
    S = 64 * n - 41 if ragged else 64 * n
    log(f"[backward blocks] S={S} (key blocks {n}, query blocks {(S + 31) // 32})")
    q, k, v, do = _data(S, 2, 128, torch.bfloat16, 1000 + S, 1.5)
    scale = 128 ** -0.5
    out, lse, dq, dk, dv = _run(hcms, q, k, v, do, scale)
    for h in range(2):
        Q, K, V, G = (x[h].double().numpy() for x in (q, k, v, do))
        rq, rk, rv = oracle_mod.attention_backward_head(Q, K, V, G, scale)
        for name, got, want in (("dq", dq, rq), ("dk", dk, rk), ("dv", dv, rv)):
            _check_grad(got[h].double().cpu().numpy(), want, f"{name} head {h}")


def test_training_forward_output_equals_inference_forward(hcms):
    q, k, v, _ = _data(3000, 3, 128, torch.bfloat16, 11)
    qd, kd, vd = (x.cuda() for x in (q, k, v))
    out_lse, _ = hcms.attention_lse(qd, kd, vd, 0.09, [2, 1])
    out = hcms.attention(qd, kd, vd, 0.09, [2, 1])
    assert torch.equal(bits(out_lse), bits(out))


@pytest.mark.parametrize("name", ["small", "wan_p4"])
def test_backward_bitwise_chunk_invariance_and_determinism(hcms, name):
    w = inputs.WORKLOADS[name]
    log(f"[backward chunks] {name}")
    q, k, v = (x.permute(1, 0, 2).contiguous().cuda() for x in inputs.make_qkv(w))
    do = inputs.make_dout(w).permute(1, 0, 2).contiguous().cuda()
    out, lse = hcms.attention_lse(q, k, v, w.scale)
    ref = [t.clone() for t in hcms.attention_backward(q, k, v, out, do, lse, w.scale)]
    for sizes in w.chunkings:
        got = hcms.attention_backward(q, k, v, out, do, lse, w.scale, sizes)
        for a, b in zip(got, ref):
            assert torch.equal(bits(a), bits(b)), (name, sizes)
    again = hcms.attention_backward(q, k, v, out, do, lse, w.scale, w.chunkings[-1])
    for a, b in zip(again, ref):
        assert torch.equal(bits(a), bits(b)), (name, "repeat")


def test_backward_wan_p8_sampled_and_gradient_sums(hcms, oracle_mod):
    """The Wan-P8 shape (S = 56160, 5 heads, chunks 2 + 2 + 1), on both paths
    (without a score-gradient workspace, and with one of two heads as the bench
    runs it): head 0 against the oracle on 64 sampled queries (dQ) and 64
    sampled keys (dK, dV); every head against the identities sum_j dK_j = 0
    and sum_j dV_j = sum_i dO_i; dK and dV the same bits on both paths."""
    w = inputs.WORKLOADS["wan_p8"]
    log("[backward wan_p8] GPU")
    qs, ks, vs = inputs.make_qkv(w)
    dos = inputs.make_dout(w)
    q, k, v, do = (x.permute(1, 0, 2).contiguous() for x in (qs, ks, vs, dos))
    qd, kd, vd, dod = (x.cuda() for x in (q, k, v, do))
    out, lse = hcms.attention_lse(qd, kd, vd, w.scale, (2, 2, 1))
    plain = [t.cpu() for t in hcms.attention_backward(qd, kd, vd, out, dod, lse, w.scale, (2, 2, 1))]
    ws = torch.empty(2 * hcms.backward_ds_bytes(w.S, w.d), dtype=torch.uint8, device="cuda")
    stored = [t.cpu() for t in hcms.attention_backward(qd, kd, vd, out, dod, lse, w.scale,
                                                       (2, 2, 1), ds=ws)]
    del ws
    torch.cuda.synchronize()
    assert torch.equal(bits(stored[1]), bits(plain[1])) and torch.equal(bits(stored[2]), bits(plain[2]))
    rng = np.random.default_rng(w.seed + 3000)
    qr = np.sort(rng.choice(w.S, 64, replace=False))
    kr = np.sort(rng.choice(w.S, 64, replace=False))
    log("[backward wan_p8] oracle, head 0 (one pass over all queries)")
    Q, K, V, G = (x[0].double().numpy() for x in (q, k, v, do))
    rq, rk, rv = oracle_mod.attention_backward_head(Q, K, V, G, w.scale, qr, kr)
    for dq, dk, dv in (plain, stored):
        _check_grad(dq[0].double().numpy()[qr], rq, "dq head 0")
        _check_grad(dk[0].double().numpy()[kr], rk, "dk head 0")
        _check_grad(dv[0].double().numpy()[kr], rv, "dv head 0")
    lw = oracle_mod.lse_head(Q, K, w.scale, qr)
    assert np.all(np.abs(lse[0].double().cpu().numpy()[qr] - lw) <= LSE_TOL * np.abs(lw))
    dq, dk, dv = plain
    for h in range(w.H):
        sk = dk[h].double().sum(dim=0)
        sv = dv[h].double().sum(dim=0)
        sg = do[h].double().sum(dim=0)
        # The sums cancel over 56160 rows; bound them by the rows' magnitudes.
        assert float(sk.abs().max()) <= GRAD_TOL * float(dk[h].double().abs().sum(dim=0).max())
        assert float((sv - sg).abs().max()) <= GRAD_TOL * float(sg.abs().max() + 1)


# ---------------------------------------------------------------------------
# The reverse pipeline (hcms_backward) and autograd
# ---------------------------------------------------------------------------
def _seq_case(name):
    w = inputs.WORKLOADS[name]
    qs, ks, vs = (x.cuda() for x in inputs.make_qkv(w))
    dos = inputs.make_dout(w).cuda()
    return w, qs, ks, vs, dos


@pytest.mark.parametrize("name", ["tiny", "small", "wan_p4"])
def test_backward_pipeline_bitwise_across_modes_and_chunkings(hcms, name):
    """hcms_backward (pack dO, backward, unpack dQ/dK/dV on the forward's plan)
    equals the direct backward on torch-transposed inputs, bitwise, for every
    mode and chunking."""
    w, qs, ks, vs, dos = _seq_case(name)
    log(f"[backward pipeline] {name}")
    hm = [x.permute(1, 0, 2).contiguous() for x in (qs, ks, vs, dos)]
    out, lse = hcms.attention_lse(hm[0], hm[1], hm[2], w.scale)
    ref = [t.permute(1, 0, 2).contiguous()
           for t in hcms.attention_backward(hm[0], hm[1], hm[2], out, hm[3], lse, w.scale)]
    ctx = hcms.Context(max_chunks=16)
    for sizes in w.chunkings:
        for mode in (hcms.MODE_SERIAL, hcms.MODE_PIPELINED, hcms.MODE_INLINE, hcms.MODE_LANES,
                     hcms.MODE_FUSED, hcms.MODE_AUTO):
            ws = [torch.empty_like(hm[0]) for _ in range(4)]
            lse2 = torch.empty_like(lse)
            o2 = ctx.forward(qs, ks, vs, w.P, w.scale, sizes, mode=mode, workspaces=ws, lse=lse2)
            got = ctx.backward(dos, w.P, w.scale, sizes, ws, lse2, mode=mode)
            assert torch.equal(bits(lse2), bits(lse)), (name, sizes, mode, "lse")
            assert torch.equal(bits(o2), bits(out.permute(1, 0, 2))), (name, sizes, mode, "out")
            for a, b, nm in zip(got, ref, ("dq", "dk", "dv")):
                assert torch.equal(bits(a), bits(b)), (name, sizes, mode, nm)
    ctx.close()


def test_autograd_matches_oracle(hcms, oracle_mod):
    """loss = <dO, attention(Q, K, V)> through HcmsAttention: loss.backward()
    gives the oracle's gradients (Tiny, fp32 storage, chunks 2 + 2)."""
    w, qs, ks, vs, dos = _seq_case("tiny")
    q, k, v = (x.clone().requires_grad_(True) for x in (qs, ks, vs))
    ctx = hcms.Context()
    out = hcms.HcmsAttention.apply(q, k, v, ctx, w.P, w.scale, (2, 2), hcms.MODE_LANES)
    (out * dos).sum().backward()
    for h in range(w.H):
        Q, K, V, G = (x[:, h].double().cpu().numpy() for x in (qs, ks, vs, dos))
        rq, rk, rv = oracle_mod.attention_backward_head(Q, K, V, G, w.scale)
        for name, got, want in (("dq", q.grad, rq), ("dk", k.grad, rk), ("dv", v.grad, rv)):
            _check_grad(got[:, h].double().cpu().numpy(), want, f"autograd {name} head {h}")
    ctx.close()


def _delay(stream, cycles=40_000_000):
    with torch.cuda.stream(stream):
        torch.cuda._sleep(cycles)


@pytest.mark.parametrize("mode", ["pipelined", "inline", "lanes", "fused", "auto"])
@pytest.mark.parametrize("late", ["copy", "compute", "main"])
def test_backward_pipeline_respects_events_under_delay(hcms, late, mode):
    """Poison the backward workspaces and outputs, delay one stream with a
    bounded spin kernel, read the gradients on the main stream right after the
    call returns: a missing wait would expose poison or stale values."""
    w, qs, ks, vs, dos = _seq_case("small")
    m = getattr(hcms, "MODE_" + mode.upper())
    sizes = (3, 3, 2)
    ctx = hcms.Context(max_chunks=8)
    ws = [torch.empty((w.H, w.S, w.d), dtype=qs.dtype, device="cuda") for _ in range(4)]
    lse = torch.empty((w.H, w.S), dtype=torch.float32, device="cuda")
    ctx.forward(qs, ks, vs, w.P, w.scale, sizes, mode=hcms.MODE_SERIAL, workspaces=ws, lse=lse)
    ref = [t.clone() for t in ctx.backward(dos, w.P, w.scale, sizes, ws, lse, mode=hcms.MODE_SERIAL)]
    torch.cuda.synchronize()
    bws = ctx.backward_workspaces(w.S, w.H, w.d, qs.dtype)
    outs = [torch.empty_like(qs) for _ in range(3)]
    for t in (*bws[:4], *outs):
        t.view(torch.int16).fill_(0x7FC1)
    bws[4].fill_(float("nan"))
    d_in = dos
    if late == "main":
        d_in = torch.empty_like(dos)
        d_in.view(torch.int16).fill_(0x7FC1)
        torch.cuda.synchronize()
        _delay(torch.cuda.current_stream())
        d_in.copy_(dos)
    else:
        torch.cuda.synchronize()
        _delay(ctx.copy_stream if late == "copy" else ctx.compute_stream)
    ctx.backward(d_in, w.P, w.scale, sizes, ws, lse, mode=m, dq=outs[0], dk=outs[1], dv=outs[2])
    seen = [t.clone() for t in outs]   # on the main stream, no host sync in between
    torch.cuda.synchronize()
    for a, b, nm in zip(seen, ref, ("dq", "dk", "dv")):
        assert torch.equal(bits(a), bits(b)), (late, mode, nm)
    ctx.close()
