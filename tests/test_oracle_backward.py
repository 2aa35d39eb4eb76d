"""Pins of the backward oracle (CPU only): a library routine, finite
differences and closed forms of the softmax-attention gradient."""
import numpy as np
import pytest
import torch



def _rand(S, d, seed, n=4, scale=1.0):
    rng = np.random.default_rng(seed)
    return [rng.standard_normal((S, d)) * scale for _ in range(n)]


def test_matches_float64_autograd(oracle_mod):
    """PyTorch's CPU autograd of softmax(scale Q K^T) V in float64."""
    for S, d, scale, seed in ((37, 16, 0.25, 1), (64, 8, 1.3, 2), (5, 32, 0.1, 3)):
        q, k, v, g = _rand(S, d, seed)
        Q, K, V = (torch.tensor(x, requires_grad=True) for x in (q, k, v))
        O = torch.softmax(scale * Q @ K.T, dim=-1) @ V
        O.backward(torch.tensor(g))
        dq, dk, dv = oracle_mod.attention_backward_head(q, k, v, g, scale)
        np.testing.assert_allclose(dq, Q.grad.numpy(), rtol=0, atol=1e-12)
        np.testing.assert_allclose(dk, K.grad.numpy(), rtol=0, atol=1e-12)
        np.testing.assert_allclose(dv, V.grad.numpy(), rtol=0, atol=1e-12)


def test_matches_central_differences_of_the_forward_oracle(oracle_mod):
    """dL/dx for L = <g, O>, with O from the forward oracle."""
    S, d, scale = 6, 4, 0.7
    q, k, v, g = _rand(S, d, 4)
    loss = lambda q, k, v: float(np.sum(g * oracle_mod.attention_head(q, k, v, scale)))  # noqa: E731
    dq, dk, dv = oracle_mod.attention_backward_head(q, k, v, g, scale)
    h = 1e-6
    for name, x, grad in (("q", q, dq), ("k", k, dk), ("v", v, dv)):
        for i in range(S):
            for t in range(d):
                xp, xm = x.copy(), x.copy()
                xp[i, t] += h
                xm[i, t] -= h
                args = {"q": q, "k": k, "v": v}
                fp = loss(**{**args, name: xp})
                fm = loss(**{**args, name: xm})
                assert (fp - fm) / (2 * h) == pytest.approx(grad[i, t], abs=1e-7), (name, i, t)


def test_gradient_sums(oracle_mod):
    """Rows of P sum to 1: sum_j dk_j = 0 and sum_j dv_j = sum_i g_i."""
    q, k, v, g = _rand(300, 24, 5, scale=2.0)
    dq, dk, dv = oracle_mod.attention_backward_head(q, k, v, g, 0.3)
    np.testing.assert_allclose(dk.sum(axis=0), 0.0, atol=1e-10)
    np.testing.assert_allclose(dv.sum(axis=0), g.sum(axis=0), atol=1e-10)


def test_equal_keys_and_zero_scale(oracle_mod):
    S, d = 50, 8
    q, k, v, g = _rand(S, d, 6)
    k_eq = np.repeat(k[:1], S, axis=0)
    dq, dk, dv = oracle_mod.attention_backward_head(q, k_eq, v, g, 0.9)
    np.testing.assert_allclose(dq, 0.0, atol=1e-12)             # uniform weights, sum_j ds_ij = 0
    np.testing.assert_allclose(dv, np.repeat(g.mean(axis=0, keepdims=True), S, axis=0), atol=1e-12)
    dq, dk, dv = oracle_mod.attention_backward_head(q, k, v, g, 0.0)
    assert np.all(dq == 0) and np.all(dk == 0)
    np.testing.assert_allclose(dv, np.repeat(g.mean(axis=0, keepdims=True), S, axis=0), atol=1e-12)


def test_single_key(oracle_mod):
    q, k, v, g = _rand(1, 16, 7)
    dq, dk, dv = oracle_mod.attention_backward_head(q, k, v, g, 0.5)
    assert np.all(dq == 0) and np.all(dk == 0)
    np.testing.assert_array_equal(dv, g)


def test_row_subsets_equal_full_rows(oracle_mod):
    q, k, v, g = _rand(90, 12, 8)
    full = oracle_mod.attention_backward_head(q, k, v, g, 0.4)
    qr, kr = np.array([0, 17, 89]), np.array([3, 44, 45, 88])
    sub = oracle_mod.attention_backward_head(q, k, v, g, 0.4, q_rows=qr, k_rows=kr)
    np.testing.assert_array_equal(sub[0], full[0][qr])
    np.testing.assert_array_equal(sub[1], full[1][kr])
    np.testing.assert_array_equal(sub[2], full[2][kr])
    only_q = oracle_mod.attention_backward_head(q, k, v, g, 0.4, q_rows=qr, k_rows=[])
    np.testing.assert_array_equal(only_q[0], full[0][qr])


def test_lse_matches_torch_logsumexp_and_closed_forms(oracle_mod):
    q, k, _, _ = _rand(40, 16, 9, scale=3.0)
    want = torch.logsumexp(0.3 * torch.tensor(q) @ torch.tensor(k).T, dim=1).numpy() / np.log(2.0)
    np.testing.assert_allclose(oracle_mod.lse_head(q, k, 0.3), want, rtol=0, atol=1e-12)
    k_eq = np.repeat(k[:1], 40, axis=0)    # equal keys: scale s + log(S)
    np.testing.assert_allclose(oracle_mod.lse_head(q, k_eq, 0.3),
                               (0.3 * q @ k[0] + np.log(40)) / np.log(2.0), atol=1e-12)
    np.testing.assert_allclose(oracle_mod.lse_head(q[:1], k[:1], 0.3), 0.3 * q[0] @ k[0] / np.log(2.0),
                               atol=1e-12)
