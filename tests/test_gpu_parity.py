"""Parity of the HIP path with the oracle, through the C ABI (MI355X only).

Bars: pack/unpack bit-exact; attention within max-abs 2e-2 of the fp64 oracle
(bf16 operands, fp32 accumulation), also normalised by max|O|, and on
"planted peak" inputs where |O| is of the order of |V|; every chunking, serial
and pipelined scheduling and repeated runs bit-identical.
"""
import numpy as np
import pytest
import torch

from paper_2607_01817_amd import inputs
from tests.gpu_util import (bits, check_attention_rows, head_major_np, log,
                            workload_inputs)

pytestmark = pytest.mark.gpu

ALL = ["tiny", "small", "wan_p4", "wan_p8", "stress"]
FULL_ORACLE = {"tiny", "small"}          # every query row; the rest are sampled
SENTINEL16 = 0x7FC1                     # a bf16 NaN bit pattern
SENTINEL32 = 0x7FC00001


def _cuda_hm(x: torch.Tensor) -> torch.Tensor:
    """[S][H][d] host tensor -> head-major [H][S][d] on cuda:0 (torch copy)."""
    return x.permute(1, 0, 2).contiguous().cuda()


def _fill_bits(t: torch.Tensor, pattern16=SENTINEL16, pattern32=SENTINEL32):
    if t.element_size() == 2:
        t.view(torch.int16).fill_(pattern16 - (1 << 16) if pattern16 >= 1 << 15 else pattern16)
    else:
        t.view(torch.int32).fill_(pattern32)


# ---------------------------------------------------------------------------
# Pack / unpack
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("name", ALL)
def test_pack_unpack_bit_exact(hcms, oracle_mod, name):
    w = inputs.WORKLOADS[name]
    log(f"[pack/unpack] {name} S={w.S} H={w.H} d={w.d} {w.dtype} P={w.P}")
    q, _, _ = workload_inputs(name)
    qb = bits(q).numpy()
    qd = q.cuda()
    rng = np.random.default_rng(w.seed)
    t_rows = np.sort(rng.choice(w.S, size=min(w.S, 512), replace=False))
    for sizes in w.chunkings:
        out = torch.empty_like(qd)
        _fill_bits(out)
        for h0, hc in zip(oracle_mod.chunk_offsets(sizes), sizes):
            chunk = hcms.pack(qd, w.P, h0, hc)
            torch.cuda.synchronize()
            got = bits(chunk.cpu()).numpy()
            if w.S * w.H * w.d <= 64 * 2**20:
                want = oracle_mod.pack(qb, w.P, h0, hc)
                assert np.array_equal(got, want), (name, sizes, h0)
            else:   # the oracle computes sampled token rows one by one
                want = oracle_mod.pack(qb[t_rows], 1, h0, hc)
                assert np.array_equal(got[:, t_rows], want), (name, sizes, h0)
            hcms.unpack(chunk, out, w.P, h0)
            del chunk
        torch.cuda.synchronize()
        assert torch.equal(bits(out.cpu()), bits(q)), (name, sizes, "roundtrip")
        del out


@pytest.mark.parametrize("d,dtype", [(8, torch.bfloat16), (16, torch.bfloat16),
                                     (16, torch.float32), (64, torch.bfloat16),
                                     (128, torch.float32), (256, torch.float32)])
def test_pack_unpack_every_row_size(hcms, oracle_mod, d, dtype):
    """Rows of 16 .. 1024 bytes (every unit count the kernels specialise on),
    an odd head count, a middle chunk and a token count that leaves a ragged
    last workgroup for every row size."""
    S, H, P, h0, hc = 8 * 131, 7, 8, 2, 3
    log(f"[pack/unpack rows] d={d} {dtype} S={S} H={H} chunk {h0}+{hc}")
    g = torch.Generator().manual_seed(d)
    x = torch.randn(S, H, d, generator=g).to(dtype)
    xb = bits(x).numpy()
    chunk = hcms.pack(x.cuda(), P, h0, hc)
    torch.cuda.synchronize()
    assert np.array_equal(bits(chunk.cpu()).numpy(), oracle_mod.pack(xb, P, h0, hc))
    dst = torch.empty(S, H, d, dtype=dtype, device="cuda")
    _fill_bits(dst)
    before = bits(dst.cpu()).numpy()
    hcms.unpack(chunk, dst, P, h0)
    torch.cuda.synchronize()
    want = oracle_mod.unpack(bits(chunk.cpu()).numpy(), before, P, h0)
    assert np.array_equal(bits(dst.cpu()).numpy(), want)


def test_unpack_leaves_other_heads(hcms):
    S, H, d, P = 1024, 6, 128, 8
    g = torch.Generator().manual_seed(11)
    src = torch.randn(2, S, d, generator=g).to(torch.bfloat16).cuda()
    dst = torch.empty(S, H, d, dtype=torch.bfloat16, device="cuda")
    _fill_bits(dst)
    before = bits(dst.cpu()).clone()
    hcms.unpack(src, dst, P, 3)
    torch.cuda.synchronize()
    after = bits(dst.cpu())
    keep = [0, 1, 2, 5]
    assert torch.equal(after[:, keep], before[:, keep])
    assert torch.equal(after[:, 3:5], bits(src.cpu()).permute(1, 0, 2))


# ---------------------------------------------------------------------------
# Attention vs the oracle
# ---------------------------------------------------------------------------
def _attention_parity(hcms, oracle_mod, name, planted, rows_per_head=None):
    w = inputs.WORKLOADS[name]
    q, k, v = workload_inputs(name, planted)
    sizes = w.chunkings[-1]
    log(f"[attention] {name} planted={planted} chunks={sizes}")
    out = hcms.attention(_cuda_hm(q), _cuda_hm(k), _cuda_hm(v), w.scale, sizes)
    torch.cuda.synchronize()
    out_h = out.float().cpu()
    del out
    rows = inputs.sample_rows(w, 0 if name in FULL_ORACLE else rows_per_head)
    worst = (0.0, 0.0)
    for h in range(w.H):
        want = oracle_mod.attention_head(head_major_np(q, h), head_major_np(k, h),
                                         head_major_np(v, h), w.scale, rows[h])
        got = out_h[h][torch.from_numpy(rows[h])].double().numpy()
        e = check_attention_rows(got, want, f"{name} head {h} planted={planted}")
        worst = max(worst, e)
    log(f"    max-abs {worst[0]:.3e}, normalised {worst[1]:.3e}")


@pytest.mark.parametrize("name", ALL)
def test_attention_matches_oracle(hcms, oracle_mod, name):
    _attention_parity(hcms, oracle_mod, name, planted=False)


@pytest.mark.parametrize("name", ALL)
def test_attention_matches_oracle_planted_peak(hcms, oracle_mod, name):
    rows = 32 if name == "stress" else None
    _attention_parity(hcms, oracle_mod, name, planted=True, rows_per_head=rows)


@pytest.mark.parametrize("S,H,d,dtype", [
    (1, 1, 128, torch.bfloat16), (2, 1, 64, torch.bfloat16), (17, 3, 64, torch.bfloat16),
    (127, 2, 128, torch.bfloat16), (129, 1, 128, torch.float32), (1000, 2, 128, torch.bfloat16),
    (300, 2, 64, torch.float32), (4097, 1, 128, torch.bfloat16)])
def test_attention_ragged_shapes(hcms, oracle_mod, S, H, d, dtype):
    """Query and key tails of every size modulo the 128-query tile and the
    64-key block, both head dims, both storage types."""
    log(f"[ragged] S={S} H={H} d={d} {dtype}")
    g = torch.Generator().manual_seed(S * 31 + H * 7 + d)
    q, k, v = (torch.randn(H, S, d, generator=g).to(dtype) for _ in range(3))
    scale = d ** -0.5
    out = hcms.attention(q.cuda(), k.cuda(), v.cuda(), scale).double().cpu().numpy()
    for h in range(H):
        want = oracle_mod.attention_head(q[h].double().numpy(), k[h].double().numpy(),
                                         v[h].double().numpy(), scale)
        check_attention_rows(out[h], want, f"S={S} h={h}")
    if S == 1:   # one key: O = V exactly
        assert torch.equal(torch.from_numpy(out).to(dtype), v)


@pytest.mark.parametrize("nkb", range(1, 14))
@pytest.mark.parametrize("tail", [0, 7])
def test_attention_every_key_block_count(hcms, oracle_mod, nkb, tail):
    """d = 128, bf16: the key loop is unrolled by four after its first step,
    with up to three more steps, a peeled step for the last scores (which
    masks the last block) and the last block, so each count of 64-key blocks
    from 1 to 13 takes a different path.  Odd counts use logits of std 16,
    which take the recompute branch in those last steps as well."""
    S, H, d = 64 * nkb - tail, 2, 128
    if S < 1:
        pytest.skip("no keys")
    sigma = 4.0 if nkb % 2 else 0.5
    log(f"[key blocks] nkb={nkb} S={S} sigma={sigma}")
    g = torch.Generator().manual_seed(1000 + S)
    q, k, v = (torch.randn(H, S, d, generator=g) * s for s in (sigma, sigma, 1.0))
    q, k, v = (x.to(torch.bfloat16) for x in (q, k, v))
    scale = d ** -0.5
    out = hcms.attention(q.cuda(), k.cuda(), v.cuda(), scale).double().cpu().numpy()
    for h in range(H):
        want = oracle_mod.attention_head(q[h].double().numpy(), k[h].double().numpy(),
                                         v[h].double().numpy(), scale)
        check_attention_rows(out[h], want, f"nkb={nkb} S={S} h={h}")


def test_attention_large_logits_and_rescaling(hcms, oracle_mod):
    """Q, K ~ N(0, 4^2): logits with std 16 keep raising the running maximum,
    exercising the lazy rescale path; also all-equal keys (uniform weights)."""
    S, H, d = 3000, 2, 128
    g = torch.Generator().manual_seed(5)
    q = (torch.randn(H, S, d, generator=g) * 4).to(torch.bfloat16)
    k = (torch.randn(H, S, d, generator=g) * 4).to(torch.bfloat16)
    v = torch.randn(H, S, d, generator=g).to(torch.bfloat16)
    k[1] = k[1, :1].expand(S, d)
    scale = d ** -0.5
    out = hcms.attention(q.cuda(), k.cuda(), v.cuda(), scale).double().cpu().numpy()
    for h in range(H):
        want = oracle_mod.attention_head(q[h].double().numpy(), k[h].double().numpy(),
                                         v[h].double().numpy(), scale)
        check_attention_rows(out[h], want, f"large logits h={h}")


def test_empty_sequence_is_a_no_op(hcms):
    z = torch.empty(4, 0, 64, dtype=torch.bfloat16, device="cuda")
    assert hcms.attention(z, z.clone(), z.clone(), 0.125).numel() == 0
    ctx = hcms.Context(max_chunks=4)
    zs = torch.empty(0, 4, 64, dtype=torch.bfloat16, device="cuda")
    assert ctx.forward(zs, zs.clone(), zs.clone(), 4, 0.125, [2, 2]).numel() == 0
    torch.cuda.synchronize()
    ctx.close()


# ---------------------------------------------------------------------------
# Invariance: chunkings, scheduling modes, repeated runs
# ---------------------------------------------------------------------------
def _chunkings(w):
    ch = list(w.chunkings)
    if w.H <= 10:
        ch.append(tuple([1] * w.H))
    return ch


@pytest.mark.parametrize("name", ALL)
def test_attention_bitwise_chunk_invariance(hcms, name):
    w = inputs.WORKLOADS[name]
    log(f"[chunk invariance] {name}")
    q, k, v = workload_inputs(name)
    qh, kh, vh = _cuda_hm(q), _cuda_hm(k), _cuda_hm(v)
    ref = hcms.attention(qh, kh, vh, w.scale, [w.H])
    for sizes in _chunkings(w):
        out = hcms.attention(qh, kh, vh, w.scale, sizes)
        assert torch.equal(bits(out), bits(ref)), (name, sizes)


FORWARD_MODES = ("serial", "pipelined", "inline", "lanes", "slots", "fused", "auto")


def _forward_modes_case(hcms, oracle_mod, name, rows_per_head):
    """hcms_forward (pack, attention, unpack on two streams) equals attention
    on the torch-transposed inputs, bitwise, for every chunking and mode, and
    matches the oracle on sampled rows of the [S][H][d] output."""
    w = inputs.WORKLOADS[name]
    log(f"[forward] {name}")
    q, k, v = workload_inputs(name)
    qd, kd, vd = q.cuda(), k.cuda(), v.cuda()
    ref = hcms.attention(_cuda_hm(q), _cuda_hm(k), _cuda_hm(v), w.scale).permute(1, 0, 2).contiguous()
    ctx = hcms.Context(max_chunks=16)
    out = torch.empty_like(qd)
    for sizes in _chunkings(w):
        for mode in FORWARD_MODES:
            log(f"    chunks={sizes} mode={mode}")
            _fill_bits(out)
            ctx.forward(qd, kd, vd, w.P, w.scale, sizes, mode=getattr(hcms, "MODE_" + mode.upper()),
                        out=out)
            assert torch.equal(bits(out), bits(ref)), (name, sizes, mode)
    del ref
    out = ctx.forward(qd, kd, vd, w.P, w.scale, w.chunkings[-1]).float().cpu()
    ctx.close()
    del qd, kd, vd
    rows = inputs.sample_rows(w, rows_per_head)
    worst = (0.0, 0.0)
    for h in range(w.H):
        want = oracle_mod.attention_head(head_major_np(q, h), head_major_np(k, h),
                                         head_major_np(v, h), w.scale, rows[h])
        got = out[torch.from_numpy(rows[h]), h].double().numpy()
        worst = max(worst, check_attention_rows(got, want, f"forward {name} head {h}"))
    log(f"    oracle rows: max-abs {worst[0]:.3e}, normalised {worst[1]:.3e}")


@pytest.mark.parametrize("name", ["tiny", "small", "wan_p4", "wan_p8"])
def test_forward_bitwise_across_modes_and_chunkings(hcms, oracle_mod, name):
    _forward_modes_case(hcms, oracle_mod, name, 64)


def test_forward_stress_bitwise_across_modes_and_chunkings(hcms, oracle_mod):
    """All 40 heads of S = 100000 on one GPU, chunkings {40}, {10 x 4} and
    {14, 13, 13}: auto runs the fused plan on {14, 13, 13} (each launch
    carrying copies of 13-14 heads over a 40-head strided layout) and lanes on
    {10 x 4}.  Oracle on 32 sampled rows per head."""
    _forward_modes_case(hcms, oracle_mod, "stress", 32)


@pytest.mark.parametrize("S,H,P,sizes_list", [
    (1000, 6, 8, [(3, 2, 1), (1,) * 6, (2, 4)]),      # ragged: 4 query tiles, 16 key blocks
    (4096, 8, 8, [(1,) * 8, (7, 1)]),                 # 16 tiles per head: many idle CUs
    (56160, 5, 8, [(2, 2, 1), (1,) * 5, (4, 1)]),     # Wan-P8: 440 / 220 / 880 workgroups
    (64000, 2, 8, [(1, 1)]),                          # 250 workgroups: 6 idle CUs, too few to
                                                      # carry the copies; they run after it
    (100000, 40, 8, [(14, 13, 13), (10,) * 4]),       # Stress: copies of 13-14 of 40 heads
])
def test_fused_forward_bitwise_equals_serial(hcms, S, H, P, sizes_list):
    """The fused plan (the next chunk's pack and the previous chunk's unpack
    riding in each attention launch) gives the serial plan's bits, with the
    workspaces and the output poisoned first, so a copy in the wrong launch
    would leave poison."""
    g = torch.Generator().manual_seed(S + H)
    q, k, v = (torch.randn(S, H, 128, generator=g).to(torch.bfloat16).cuda() for _ in range(3))
    scale = 128 ** -0.5
    ctx = hcms.Context(max_chunks=8)
    ref = ctx.forward(q, k, v, P, scale, (H,), mode=hcms.MODE_SERIAL).clone()
    for sizes in sizes_list:
        log(f"[fused] S={S} H={H} chunks={sizes}")
        ws = ctx.workspaces(S, H, 128, q.dtype)
        out = torch.empty_like(q)
        for t in (*ws, out):
            _fill_bits(t)
        torch.cuda.synchronize()
        ctx.forward(q, k, v, P, scale, sizes, mode=hcms.MODE_FUSED, out=out, workspaces=ws)
        seen = out.clone()
        torch.cuda.synchronize()
        assert ctx.last_mode == hcms.MODE_FUSED
        assert torch.equal(bits(seen), bits(ref)), sizes
    ctx.close()


@pytest.mark.parametrize("name,sizes", [("wan_p8", (2, 2, 1)), ("wan_p4", (5, 5)),
                                        ("small", (3, 3, 2)), ("small", (8,))])
def test_auto_mode_runs_the_predicted_plan(hcms, name, sizes):
    w = inputs.WORKLOADS[name]
    q, k, v = (x.cuda() for x in workload_inputs(name))
    ctx = hcms.Context()
    assert ctx.num_cu == torch.cuda.get_device_properties(0).multi_processor_count
    assert ctx.last_mode == -1
    ctx.forward(q, k, v, w.P, w.scale, sizes, mode=hcms.MODE_AUTO)
    assert ctx.last_mode == hcms.auto_mode(w.S, w.d, sizes, ctx.num_cu)
    ctx.forward(q, k, v, w.P, w.scale, sizes, mode=hcms.MODE_PIPELINED)
    assert ctx.last_mode == hcms.MODE_PIPELINED
    torch.cuda.synchronize()
    ctx.close()


@pytest.mark.parametrize("name,sizes", [("wan_p8", (2, 2, 1)), ("wan_p8", (5,)), ("small", (8,)),
                                        ("small", (3, 3, 2))])
def test_forward_is_deterministic(hcms, name, sizes):
    """Repeated forwards give the same bits.  Wan-P8 {5} splits its last round
    of 76 tiles three ways and Small {8} its 128 tiles two ways, so each call
    also checks that the split tiles' arrival counters are back at zero.  The
    lanes plan splits the 76 tiles past the pooled rounds of Wan-P8 {2,2,1}
    in its last chunk's launch."""
    w = inputs.WORKLOADS[name]
    q, k, v = (x.cuda() for x in workload_inputs(name))
    ref = hcms.attention(_cuda_hm(q), _cuda_hm(k), _cuda_hm(v), w.scale).permute(1, 0, 2)
    ctx = hcms.Context()
    for mode in (hcms.MODE_SERIAL, hcms.MODE_FUSED, hcms.MODE_LANES):
        for _ in range(3):
            got = ctx.forward(q, k, v, w.P, w.scale, sizes, mode=mode)
            assert torch.equal(bits(got), bits(ref)), (name, sizes, mode)
    ctx.close()


# ---------------------------------------------------------------------------
# Event ordering of the pipelined schedule, forced from the host
# ---------------------------------------------------------------------------
def _delay(stream, cycles=40_000_000):
    with torch.cuda.stream(stream):
        torch.cuda._sleep(cycles)


@pytest.mark.parametrize("mode", ["pipelined", "inline", "lanes", "fused"])
@pytest.mark.parametrize("late", ["copy", "compute", "main"])
def test_pipelined_respects_events_under_delay(hcms, late, mode):
    """Poison the workspaces and the output, delay one stream with a bounded
    spin kernel, and read the output on the main stream right after the call
    returns.  A missing wait (fork, E_c^pack, E_c^attn or the join) would let
    a kernel read poison or the caller read a stale output."""
    w = inputs.WORKLOADS["small"]
    q, k, v = (x.cuda() for x in workload_inputs("small"))
    ctx = hcms.Context(max_chunks=8)
    sizes = (3, 3, 2)
    ref = ctx.forward(q, k, v, w.P, w.scale, sizes, mode=hcms.MODE_SERIAL).clone()
    torch.cuda.synchronize()
    ws = ctx.workspaces(w.S, w.H, w.d, q.dtype)
    out = torch.empty_like(q)
    for t in (*ws, out):
        _fill_bits(t)
    q_in = q
    if late == "main":
        # The inputs are written on the main stream after a delay: the copy
        # stream must wait for E_main before packing them.
        q_in = torch.empty_like(q)
        _fill_bits(q_in)
        torch.cuda.synchronize()
        _delay(torch.cuda.current_stream())
        q_in.copy_(q)
    else:
        torch.cuda.synchronize()
        _delay(ctx.copy_stream if late == "copy" else ctx.compute_stream)
    m = {"pipelined": hcms.MODE_PIPELINED, "inline": hcms.MODE_INLINE, "lanes": hcms.MODE_LANES,
         "fused": hcms.MODE_FUSED}[mode]
    ctx.forward(q_in, k, v, w.P, w.scale, sizes, mode=m, out=out)
    seen = out.clone()            # on the main stream, no host sync in between
    torch.cuda.synchronize()
    assert torch.equal(bits(seen), bits(ref)), (late, mode)
    ctx.close()


def test_timing_api_reports_every_chunk(hcms):
    w = inputs.WORKLOADS["small"]
    q, k, v = (x.cuda() for x in workload_inputs("small"))
    ctx = hcms.Context(max_chunks=8)
    for mode in (hcms.MODE_AUTO, hcms.MODE_FUSED):
        ctx.set_timing(2)
        for _ in range(3):   # the third call is past the record and not timed
            ctx.forward(q, k, v, w.P, w.scale, (3, 3, 2), mode=mode)
        for kind in (hcms.OP_PACK, hcms.OP_ATTENTION, hcms.OP_UNPACK):
            ms = ctx.kernel_ms(kind)
            assert len(ms) == 6 and all(0 < x < 1000 for x in ms), (mode, kind, ms)
    ctx.close()
