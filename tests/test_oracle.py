"""Pins for the oracle (CPU only).

The oracle is only trusted once it agrees with something other than itself:
values the paper prints, closed forms, invariants, a library routine, and an
analytic worked example.  Each test says which plausible mistake it catches.
"""
import json
import math
import os

import numpy as np
import pytest
import torch

from paper_2607_01817_amd import inputs

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------------------
# Chunk-size rule (Sec. 3.3 equation; Sec. 4.3 uneven partition table)
# ---------------------------------------------------------------------------
def test_default_chunks_matches_printed_table(oracle_mod):
    with open(os.path.join(GOLDEN, "uneven_chunking.json")) as f:
        cases = json.load(f)["cases"]
    for c in cases:
        sizes = oracle_mod.default_chunks(c["H"], c["C"])
        assert sizes == c["sizes"], c
        a = np.array(sizes, dtype=float)
        assert round((a.max() - a.min()) / a.mean() * 100) == c["imbalance_pct"]


def test_default_chunks_properties(oracle_mod):
    for H in range(1, 65):
        for C in range(1, H + 1):
            s = oracle_mod.default_chunks(H, C)
            assert len(s) == C and sum(s) == H
            assert max(s) - min(s) <= 1
            assert s == sorted(s, reverse=True)      # more first, less later
    with pytest.raises(ValueError):
        oracle_mod.default_chunks(4, 5)
    with pytest.raises(ValueError):
        oracle_mod.default_chunks(4, 0)


def test_workload_chunkings_follow_rule(oracle_mod):
    """Every uneven chunking the workloads use is the rule's output."""
    for w in inputs.WORKLOADS.values():
        for ch in w.chunkings:
            assert sum(ch) == w.H
            assert list(ch) == oracle_mod.default_chunks(w.H, len(ch))


# ---------------------------------------------------------------------------
# Pack / unpack
# ---------------------------------------------------------------------------
def _rand_u16(shape, seed):
    return np.random.default_rng(seed).integers(0, 1 << 16, size=shape, dtype=np.uint16)


@pytest.mark.parametrize("P,S,H,d,dtype", [(4, 128, 4, 64, np.float32),
                                           (8, 64, 5, 128, np.uint16),
                                           (3, 24, 7, 8, np.uint16),
                                           (1, 5, 3, 4, np.float32)])
def test_pack_is_numpy_head_slice_transpose(oracle_mod, P, S, H, d, dtype):
    """Library routine: pack of chunk [h0, h0+Hc) equals reshape + slice +
    transpose in numpy.  Catches a swapped index or a wrong shard order."""
    rng = np.random.default_rng(S * H + d)
    src = rng.standard_normal((S, H, d)).astype(np.float32).view(np.uint32) \
        if dtype == np.float32 else _rand_u16((S, H, d), S + H)
    sizes = oracle_mod.default_chunks(H, min(3, H))
    for h0, hc in zip(oracle_mod.chunk_offsets(sizes), sizes):
        got = oracle_mod.pack(src, P, h0, hc)
        want = src.reshape(P, S // P, H, d).reshape(S, H, d)[:, h0:h0 + hc, :].transpose(1, 0, 2)
        assert got.shape == (hc, S, d)
        assert np.array_equal(got, want)


def test_pack_unpack_roundtrip_and_sentinels(oracle_mod):
    S, H, d, P = 96, 6, 16, 4
    src = _rand_u16((S, H, d), 7)
    sentinel = np.full((S, H, d), 0xA5A5, dtype=np.uint16)
    out = sentinel
    sizes = [3, 2, 1]
    seen = np.zeros(H, dtype=int)
    for h0, hc in zip(oracle_mod.chunk_offsets(sizes), sizes):
        chunk = oracle_mod.pack(src, P, h0, hc)
        before = out.copy()
        out = oracle_mod.unpack(chunk, out, P, h0)
        # heads outside the chunk are untouched
        mask = np.ones(H, bool)
        mask[h0:h0 + hc] = False
        assert np.array_equal(out[:, mask], before[:, mask])
        seen[h0:h0 + hc] += 1
    assert np.all(seen == 1)                   # chunks cover every head once
    assert np.array_equal(out, src)            # unpack o pack = identity


def test_pack_rejects_bad_shapes(oracle_mod):
    src = _rand_u16((10, 2, 4), 1)
    with pytest.raises(ValueError):
        oracle_mod.pack(src, 3, 0, 1)          # S % P != 0
    with pytest.raises(ValueError):
        oracle_mod.pack(src, 2, 1, 2)          # head range overflows H


# ---------------------------------------------------------------------------
# Attention: closed forms, worked example, invariants, library routine
# ---------------------------------------------------------------------------
def test_two_key_worked_example(oracle_mod):
    """d = 2, scale = 1/2, q = (1, 0), k0 = 0, k1 = (2 ln 3, 0): the logits are
    0 and ln 3, so the weights are 1/4 and 3/4 and O = (V0 + 3 V1) / 4.
    Catches a missing or inverted scale, a wrong exponent base and a missing
    normalisation."""
    q = np.array([[1.0, 0.0], [0.0, 0.0]])
    k = np.array([[0.0, 0.0], [2.0 * math.log(3.0), 0.0]])
    v = np.array([[4.0, -8.0], [8.0, 12.0]])
    o = oracle_mod.attention_head(q, k, v, 0.5)
    np.testing.assert_allclose(o[0], (v[0] + 3 * v[1]) / 4, rtol=0, atol=1e-14)
    # second query is orthogonal to both keys: uniform weights
    np.testing.assert_allclose(o[1], (v[0] + v[1]) / 2, rtol=0, atol=1e-14)


def test_constant_values(oracle_mod):
    """V rows all equal c  =>  O = c for every query (weights sum to one)."""
    rng = np.random.default_rng(1)
    S, d = 37, 8
    q, k = rng.standard_normal((S, d)) * 3, rng.standard_normal((S, d)) * 3
    c = rng.standard_normal(d)
    v = np.tile(c, (S, 1))
    o = oracle_mod.attention_head(q, k, v, 0.7)
    np.testing.assert_allclose(o, np.tile(c, (S, 1)), rtol=0, atol=1e-13)


def test_equal_keys_and_zero_scale_give_mean(oracle_mod):
    """All K rows equal, or scale = 0  =>  O = mean of V rows."""
    rng = np.random.default_rng(2)
    S, d = 29, 5
    q, v = rng.standard_normal((S, d)), rng.standard_normal((S, d))
    k = np.tile(rng.standard_normal(d), (S, 1))
    mean = v.mean(axis=0)
    np.testing.assert_allclose(oracle_mod.attention_head(q, k, v, 1.3),
                               np.tile(mean, (S, 1)), atol=1e-13)
    k2 = rng.standard_normal((S, d))
    np.testing.assert_allclose(oracle_mod.attention_head(q, k2, v, 0.0),
                               np.tile(mean, (S, 1)), atol=1e-13)


def test_single_token(oracle_mod):
    """S = 1  =>  O = V."""
    q, k, v = np.array([[1.0, 2.0]]), np.array([[3.0, -1.0]]), np.array([[0.25, -7.0]])
    np.testing.assert_array_equal(oracle_mod.attention_head(q, k, v, 0.9), v)


def test_large_logits_do_not_overflow(oracle_mod):
    """Logits near 1e3 overflow exp() unless the maximum is subtracted."""
    q = np.array([[30.0, 0.0]])
    k = np.array([[33.0, 0.0], [33.0 - 2.0 * math.log(2.0) / 30.0, 0.0]])
    v = np.array([[1.0, 0.0], [0.0, 1.0]])
    o = oracle_mod.attention_head(q, k, v, 1.0)
    # logits 990 and 990 - 2 ln 2: weights 4/5 and 1/5
    np.testing.assert_allclose(o[0], [0.8, 0.2], atol=1e-12)


def test_planted_peak_selects_its_value_row(oracle_mod):
    """Q_i = 4 K_pi(i) with unit-norm-ish keys: the softmax weight concentrates
    on pi(i), so O_i = V_pi(i) up to the bound (1 - w) * max|V_j - V_pi|.
    Catches a wrong key/value index or a transposed operand."""
    rng = np.random.default_rng(3)
    S, d = 300, 32
    k = rng.standard_normal((S, d))
    v = rng.standard_normal((S, d))
    perm = rng.permutation(S)
    q = 4.0 * k[perm]
    scale = 1.0 / math.sqrt(d)
    o = oracle_mod.attention_head(q, k, v, scale)
    logits = scale * (q @ k.T)                          # library matmul
    for i in range(S):
        gap = np.exp(logits[i] - logits[i, perm[i]])
        gap[perm[i]] = 0.0
        bound = gap.sum() * np.abs(v - v[perm[i]]).max() + 1e-12
        assert np.abs(o[i] - v[perm[i]]).max() <= bound


def test_convex_hull(oracle_mod):
    rng = np.random.default_rng(4)
    S, d = 64, 16
    q, k, v = (rng.standard_normal((S, d)) * 2 for _ in range(3))
    o = oracle_mod.attention_head(q, k, v, 0.4)
    assert np.all(o <= v.max(axis=0) + 1e-12)
    assert np.all(o >= v.min(axis=0) - 1e-12)


def test_permutation_equivariance(oracle_mod):
    """Permuting (K, V) rows jointly leaves O unchanged; permuting Q rows
    permutes O.  Catches pairing K row j with a different V row."""
    rng = np.random.default_rng(5)
    S, d = 50, 8
    q, k, v = (rng.standard_normal((S, d)) for _ in range(3))
    o = oracle_mod.attention_head(q, k, v, 0.35)
    pk = rng.permutation(S)
    np.testing.assert_allclose(oracle_mod.attention_head(q, k[pk], v[pk], 0.35), o,
                               atol=1e-13)
    pq = rng.permutation(S)
    np.testing.assert_allclose(oracle_mod.attention_head(q[pq], k, v, 0.35), o[pq],
                               atol=1e-15)


def test_head_independence(oracle_mod):
    """Sec. 3.3 Property: perturbing head h' leaves every other head bitwise
    unchanged."""
    rng = np.random.default_rng(6)
    H, S, d = 3, 40, 8
    q, k, v = (rng.standard_normal((H, S, d)) for _ in range(3))
    o = oracle_mod.attention(q, k, v, 0.5)
    q2, k2, v2 = q.copy(), k.copy(), v.copy()
    q2[1] += 1.0
    k2[1] *= -2.0
    v2[1] += 3.0
    o2 = oracle_mod.attention(q2, k2, v2, 0.5)
    assert np.array_equal(o[0], o2[0]) and np.array_equal(o[2], o2[2])
    assert not np.array_equal(o[1], o2[1])


def test_row_subset_matches_full(oracle_mod):
    rng = np.random.default_rng(7)
    S, d = 70, 8
    q, k, v = (rng.standard_normal((S, d)) for _ in range(3))
    full = oracle_mod.attention_head(q, k, v, 0.3)
    rows = np.array([0, 5, 69, 33])
    np.testing.assert_array_equal(oracle_mod.attention_head(q, k, v, 0.3, rows), full[rows])


@pytest.mark.parametrize("name", ["tiny"])
def test_matches_torch_sdpa_fp64(oracle_mod, name):
    """Library routine: PyTorch's CPU scaled_dot_product_attention in fp64, on
    the seeded workload inputs (exact stored values widened to fp64)."""
    w = inputs.WORKLOADS[name]
    q, k, v = inputs.make_qkv(w)
    qh, kh, vh = (x.to(torch.float64).permute(1, 0, 2).contiguous() for x in (q, k, v))
    ref = torch.nn.functional.scaled_dot_product_attention(
        qh[None], kh[None], vh[None], scale=w.scale)[0].numpy()
    got = oracle_mod.attention(qh.numpy(), kh.numpy(), vh.numpy(), w.scale)
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12)


def test_matches_torch_sdpa_fp64_small_head(oracle_mod):
    """Same library check on two heads of the 4096-token bf16 workload,
    sampled rows (the full 4096 x 4096 reference stays cheap)."""
    w = inputs.WORKLOADS["small"]
    q, k, v = inputs.make_qkv(w)
    rows = np.array([0, 1, 777, 2048, 4095])
    for h in (0, 5):
        qh, kh, vh = (x[:, h].to(torch.float64) for x in (q, k, v))
        ref = torch.nn.functional.scaled_dot_product_attention(
            qh[rows][None], kh[None], vh[None], scale=w.scale)[0].numpy()
        got = oracle_mod.attention_head(qh.numpy(), kh.numpy(), vh.numpy(), w.scale, rows)
        np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12)


def test_mpmath_brute_force_tiny(oracle_mod):
    """Extra check in 50-digit arithmetic on a tiny head (not a pin by itself:
    it restates the definition; the pins are the tests above)."""
    mpmath = pytest.importorskip("mpmath")
    mpmath.mp.dps = 50
    rng = np.random.default_rng(8)
    S, d, scale = 9, 4, 0.61
    q, k, v = (rng.standard_normal((S, d)) * 2 for _ in range(3))
    o = oracle_mod.attention_head(q, k, v, scale)
    for i in range(S):
        s = [mpmath.mpf(scale) * mpmath.fsum(mpmath.mpf(q[i, t]) * mpmath.mpf(k[j, t])
                                              for t in range(d)) for j in range(S)]
        w = [mpmath.e ** x for x in s]
        tot = mpmath.fsum(w)
        for t in range(d):
            ref = mpmath.fsum(w[j] * mpmath.mpf(v[j, t]) for j in range(S)) / tot
            assert abs(float(ref) - o[i, t]) <= 1e-13


def test_forward_is_per_token_per_head_attention(oracle_mod):
    """End to end (pack, attention, unpack over uneven chunks) equals attention
    of each head on the [S][H][d] view: the concatenation along heads of
    Alg. 1 loses nothing and mixes no heads."""
    rng = np.random.default_rng(9)
    S, H, d, P = 48, 5, 8, 4
    q, k, v = (rng.standard_normal((S, H, d)) for _ in range(3))
    got = oracle_mod.forward(q, k, v, P, 0.4, [2, 2, 1])
    for h in range(H):
        ref = torch.nn.functional.scaled_dot_product_attention(
            torch.from_numpy(q[:, h])[None], torch.from_numpy(k[:, h])[None],
            torch.from_numpy(v[:, h])[None], scale=0.4)[0].numpy()
        np.testing.assert_allclose(got[:, h], ref, atol=1e-12)
