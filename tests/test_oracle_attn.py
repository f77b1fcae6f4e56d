"""Pins for the fp64 attention oracle (CPU only).

Each test checks the oracle against something other than itself: central
finite differences of the forward, torch's own fp64 attention and autograd,
closed forms, invariants of the softmax gradient and of causal masking, and
special cases that reduce to a textbook result.  A dropped term, a sign, a
transposed operand or a wrong mask index in the oracle fails at least one.
"""
import numpy as np
import pytest
import torch

import oracle


def rnd(rng, *shape, scale=1.0):
    return rng.standard_normal(shape) * scale


def loss_fn(q, k, v, do, causal):
    o, _ = oracle.attn_fwd(q, k, v, causal)
    return float(np.sum(do * o))


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("n,d", [(1, 1), (2, 2), (3, 4), (5, 2), (8, 4), (8, 1)])
def test_finite_differences(n, d, causal):
    """dQ, dK, dV are the gradient of sum(dO o O): central differences, h=1e-5."""
    rng = np.random.default_rng(100 * n + d + (7 if causal else 0))
    q, k, v, do = (rnd(rng, n, d) for _ in range(4))
    dq, dk, dv, _, _ = oracle.attn_bwd(q, k, v, do, causal)
    h = 1e-5
    for name, x, g in (("q", q, dq), ("k", k, dk), ("v", v, dv)):
        num = np.zeros_like(x)
        for idx in np.ndindex(*x.shape):
            xp, xm = x.copy(), x.copy()
            xp[idx] += h
            xm[idx] -= h
            args_p = {"q": q, "k": k, "v": v}
            args_m = dict(args_p)
            args_p[name], args_m[name] = xp, xm
            num[idx] = (loss_fn(args_p["q"], args_p["k"], args_p["v"], do, causal)
                        - loss_fn(args_m["q"], args_m["k"], args_m["v"], do, causal)) / (2 * h)
        ref = max(np.max(np.abs(num)), 1e-3)
        assert np.max(np.abs(num - g)) / ref < 1e-7, name


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("n,d", [(37, 16), (64, 8), (5, 32)])
def test_matches_torch_fp64_sdpa_and_autograd(n, d, causal):
    """Forward and gradients agree with torch's fp64 attention + autograd."""
    g = torch.Generator().manual_seed(n * d)
    q, k, v, do = (torch.randn(2, 3, n, d, generator=g, dtype=torch.float64) for _ in range(4))
    qq, kk, vv = (t.clone().requires_grad_(True) for t in (q, k, v))
    o_t = torch.nn.functional.scaled_dot_product_attention(qq, kk, vv, is_causal=causal)
    o_t.backward(do)
    o, lse = oracle.attn_fwd(q, k, v, causal)
    dq, dk, dv, lse2, D = oracle.attn_bwd(q, k, v, do, causal)
    np.testing.assert_allclose(o, o_t.detach().numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dq, qq.grad.numpy(), rtol=1e-10, atol=1e-11)
    np.testing.assert_allclose(dk, kk.grad.numpy(), rtol=1e-10, atol=1e-11)
    np.testing.assert_allclose(dv, vv.grad.numpy(), rtol=1e-10, atol=1e-11)
    # L is the natural-log logsumexp of the scaled, masked scores
    s = (q @ k.transpose(-1, -2)).numpy() / np.sqrt(d)
    if causal:
        s = np.where(np.tril(np.ones((n, n), bool)), s, -np.inf)
    ref_lse = torch.logsumexp(torch.from_numpy(s), dim=-1).numpy()
    np.testing.assert_allclose(lse, ref_lse, rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(lse2, ref_lse, rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("causal", [False, True])
def test_forward_closed_forms(causal):
    """K = 0: uniform attention, L_i = log(#visible), O_i = mean of visible V rows.
    V = 1: O = 1.  Causal row 0 sees only key 0: O_0 = V_0, L_0 = S_00."""
    rng = np.random.default_rng(3)
    n, d = 23, 6
    q, v = rnd(rng, n, d), rnd(rng, n, d)
    o, lse = oracle.attn_fwd(q, np.zeros((n, d)), v, causal)
    cnt = np.arange(1, n + 1) if causal else np.full(n, n)
    np.testing.assert_allclose(lse, np.log(cnt), rtol=0, atol=1e-14)
    mean = np.cumsum(v, 0) / cnt[:, None] if causal else np.broadcast_to(v.mean(0), (n, d))
    np.testing.assert_allclose(o, mean, rtol=1e-13, atol=1e-14)
    k = rnd(rng, n, d)
    o1, _ = oracle.attn_fwd(q, k, np.ones((n, d)), causal)
    np.testing.assert_allclose(o1, 1.0, rtol=0, atol=1e-14)
    if causal:
        o, lse = oracle.attn_fwd(q, k, v, True)
        np.testing.assert_allclose(o[0], v[0], rtol=0, atol=1e-15)
        assert abs(lse[0] - q[0] @ k[0] / np.sqrt(d)) < 1e-14


def test_backward_special_cases():
    """N = 1: P = [1], so dV = dO and dQ = dK = 0.  V = 0: dP = 0 and O = 0, so
    dS = 0 and dQ = dK = 0 while dV = P^T dO."""
    rng = np.random.default_rng(4)
    q, k, v, do = (rnd(rng, 1, 5) for _ in range(4))
    for causal in (False, True):
        dq, dk, dv, _, _ = oracle.attn_bwd(q, k, v, do, causal)
        np.testing.assert_array_equal(dv, do)
        assert np.max(np.abs(dq)) < 1e-15 and np.max(np.abs(dk)) < 1e-15
    n, d = 9, 4
    q, k, do = rnd(rng, n, d), rnd(rng, n, d), rnd(rng, n, d)
    for causal in (False, True):
        dq, dk, dv, _, _ = oracle.attn_bwd(q, k, np.zeros((n, d)), do, causal)
        assert np.max(np.abs(dq)) == 0 and np.max(np.abs(dk)) == 0
        P = oracle.probs(q, k, causal)
        np.testing.assert_allclose(dv, P.T @ do, rtol=1e-13, atol=1e-14)


@pytest.mark.parametrize("causal", [False, True])
def test_softmax_gradient_invariants(causal):
    """Rows of dS sum to zero, hence sum_j dK_j = 0 and dQ is unchanged by
    adding one vector to every key; sum_j dV_j = sum_i dO_i (rows of P sum to 1);
    and D = rowsum(dO o O) equals rowsum(P o dP) with dP = dO V^T."""
    rng = np.random.default_rng(5)
    n, d = 31, 8
    q, k, v, do = (rnd(rng, n, d) for _ in range(4))
    dq, dk, dv, _, D = oracle.attn_bwd(q, k, v, do, causal)
    scale = np.max(np.abs(dk))
    assert np.max(np.abs(dk.sum(0))) < 1e-12 * n * scale
    np.testing.assert_allclose(dv.sum(0), do.sum(0), rtol=1e-12, atol=1e-12)
    c = rnd(rng, 1, d) * 3
    dq2, _, _, _, _ = oracle.attn_bwd(q, k + c, v, do, causal)
    np.testing.assert_allclose(dq2, dq, rtol=1e-9, atol=1e-11)
    P = oracle.probs(q, k, causal)
    np.testing.assert_allclose(P.sum(1), 1.0, rtol=0, atol=1e-14)
    dP = do @ v.T
    np.testing.assert_allclose(D, (P * dP).sum(1), rtol=1e-12, atol=1e-12)


def test_causal_zero_gradient_invariants():
    """Causal mask: dQ_0 = 0; keys/values after row i do not touch dQ rows <= i;
    queries/output-grads before row j do not touch dK_j, dV_j; the last key is
    seen only by the last query, so dV_{N-1} = P_{N-1,N-1} dO_{N-1}."""
    rng = np.random.default_rng(6)
    n, d, i, j = 17, 5, 7, 9
    q, k, v, do = (rnd(rng, n, d) for _ in range(4))
    dq, dk, dv, _, _ = oracle.attn_bwd(q, k, v, do, True)
    assert np.max(np.abs(dq[0])) < 1e-15
    k2, v2 = k.copy(), v.copy()
    k2[i + 1:] += rnd(rng, n - i - 1, d)
    v2[i + 1:] += rnd(rng, n - i - 1, d)
    dq2, _, _, _, _ = oracle.attn_bwd(q, k2, v2, do, True)
    np.testing.assert_array_equal(dq2[: i + 1], dq[: i + 1])
    q3, do3 = q.copy(), do.copy()
    q3[:j] += rnd(rng, j, d)
    do3[:j] += rnd(rng, j, d)
    _, dk3, dv3, _, _ = oracle.attn_bwd(q3, k, v, do3, True)
    np.testing.assert_array_equal(dk3[j:], dk[j:])
    np.testing.assert_array_equal(dv3[j:], dv[j:])
    P = oracle.probs(q, k, True)
    np.testing.assert_allclose(dv[n - 1], P[n - 1, n - 1] * do[n - 1], rtol=1e-13, atol=1e-15)


@pytest.mark.parametrize("causal", [False, True])
def test_sampled_rows_match_full(causal):
    """Row/column sampling returns the entries of the full computation: dQ rows
    exactly; dK, dV rows to rounding (their L and D then come from the
    all-rows helper, whose sums run in another order)."""
    rng = np.random.default_rng(7)
    q, k, v, do = (rnd(rng, 2, 40, 8) for _ in range(4))
    full = oracle.attn_bwd(q, k, v, do, causal)
    rows, cols = [0, 13, 39], [1, 38]
    part = oracle.attn_bwd(q, k, v, do, causal, dq_rows=rows, kv_rows=cols)
    np.testing.assert_array_equal(part[0][:, rows], full[0][:, rows])
    np.testing.assert_allclose(part[1][:, cols], full[1][:, cols], rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(part[2][:, cols], full[2][:, cols], rtol=1e-12, atol=1e-14)
    assert np.isnan(part[0][:, 1]).all() and np.isnan(part[1][:, 0]).all()
    o, lse = oracle.attn_fwd(q, k, v, causal)
    o2, lse2 = oracle.attn_fwd(q, k, v, causal, rows=rows)
    np.testing.assert_array_equal(o2[:, rows], o[:, rows])
    np.testing.assert_array_equal(lse2[:, rows], lse[:, rows])
    np.testing.assert_array_equal(lse, full[3])


def test_explicit_scale():
    """A non-default softmax scale multiplies S, dQ and dK (not dV): checked
    against torch's attention called with the same explicit scale."""
    g = torch.Generator().manual_seed(11)
    q, k, v, do = (torch.randn(1, 1, 12, 4, generator=g, dtype=torch.float64) for _ in range(4))
    qq, kk, vv = (t.clone().requires_grad_(True) for t in (q, k, v))
    o_t = torch.nn.functional.scaled_dot_product_attention(qq, kk, vv, scale=0.37)
    o_t.backward(do)
    dq, dk, dv, _, _ = oracle.attn_bwd(q, k, v, do, False, scale=0.37)
    np.testing.assert_allclose(dq, qq.grad.numpy(), rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(dk, kk.grad.numpy(), rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(dv, vv.grad.numpy(), rtol=1e-11, atol=1e-12)


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("n,d", [(1, 4), (37, 16), (130, 8)])
def test_lse_and_d_against_torch_and_closed_forms(n, d, causal):
    """The all-rows L and D helper (used for sampled dK/dV rows of long heads):
    L equals torch's logsumexp of the explicitly masked scaled scores, D equals
    rowsum(dO o O) with torch's fp64 attention output; K = 0 gives L_i =
    log(#visible keys) and D_i = dO_i . mean(visible V rows); causal row 0
    gives L_0 = S_00 and D_0 = dO_0 . V_0; the row-block size changes nothing."""
    rng = np.random.default_rng(n + d)
    q, k, v, do = (rnd(rng, n, d) for _ in range(4))
    lse, dvec = oracle.lse_and_d(q, k, v, do, causal)
    s = (q @ k.T) / np.sqrt(d)
    if causal:
        s = np.where(np.tril(np.ones((n, n), bool)), s, -np.inf)
    np.testing.assert_allclose(lse, torch.logsumexp(torch.from_numpy(s), dim=-1).numpy(), rtol=1e-13, atol=1e-13)
    t = [torch.from_numpy(x)[None, None] for x in (q, k, v)]
    o_t = torch.nn.functional.scaled_dot_product_attention(*t, is_causal=causal)[0, 0].numpy()
    np.testing.assert_allclose(dvec, np.sum(do * o_t, axis=1), rtol=1e-11, atol=1e-12)
    l2, d2 = oracle.lse_and_d(q, k, v, do, causal, block=7)
    np.testing.assert_allclose(l2, lse, rtol=1e-14, atol=1e-14)
    np.testing.assert_allclose(d2, dvec, rtol=1e-13, atol=1e-14)
    lz, dz = oracle.lse_and_d(q, np.zeros((n, d)), v, do, causal)
    cnt = np.arange(1, n + 1) if causal else np.full(n, n)
    np.testing.assert_allclose(lz, np.log(cnt), rtol=1e-14, atol=1e-14)
    mean_v = np.cumsum(v, axis=0) / cnt[:, None] if causal else np.broadcast_to(v.mean(axis=0), v.shape)
    np.testing.assert_allclose(dz, np.sum(do * mean_v, axis=1), rtol=1e-12, atol=1e-13)
    if causal:
        assert abs(lse[0] - s[0, 0]) < 1e-13
        assert abs(dvec[0] - do[0] @ v[0]) < 1e-12


@pytest.mark.parametrize("causal", [False, True])
def test_sampled_dkdv_rows_equal_full_pass(causal):
    """dK, dV rows computed with only some dQ rows requested (L and D from the
    all-rows helper) equal those of the full row-by-row pass."""
    rng = np.random.default_rng(11)
    n, d = 150, 16
    q, k, v, do = (rnd(rng, n, d) for _ in range(4))
    rows = [0, 1, 63, 64, 100, 149]
    full = oracle.attn_bwd(q, k, v, do, causal, kv_rows=rows)
    samp = oracle.attn_bwd(q, k, v, do, causal, dq_rows=[5, 149], kv_rows=rows)
    for a, b in ((full[1], samp[1]), (full[2], samp[2])):
        np.testing.assert_allclose(b[rows], a[rows], rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(samp[0][[5, 149]], full[0][[5, 149]], rtol=1e-13, atol=1e-14)
    assert np.isnan(samp[0][6]).all()
