"""The derived error terms (tests/bounds.py) pinned on the CPU: the bf16
spacing against torch's rounding, and the attention backward's sensitivity
to a rounded output gradient against the oracle's own linear response (the
backward is linear in dO for fixed q, k, v, so a unit change of one dO
element gives one column of the exact Jacobian), and the terms of the
backward's bf16 P and dS against sampled roundings."""
import numpy as np
import torch

import bounds
import oracle as O


def test_ulp_bf16_is_the_rounding_step():
    x = np.concatenate([np.linspace(-5, 5, 2001), [1.0, 2.0 ** -126, 3.0e5]])
    u = bounds.ulp_bf16(x)
    xb = torch.tensor(x, dtype=torch.float64).to(torch.float32).to(torch.bfloat16)
    err = np.abs(xb.to(torch.float64).numpy() - x)
    assert np.all(err <= 0.5 * u * (1 + 1e-12))
    assert bounds.ulp_bf16(1.0) == 2.0 ** -7 and bounds.ulp_bf16(1.999) == 2.0 ** -7


def test_attention_dout_sensitivity_matches_the_oracles_jacobian():
    rng = np.random.default_rng(3)
    S, d = 7, 4
    q, k, v, do = (rng.standard_normal((S, d)) for _ in range(4))
    sig2 = rng.uniform(0.01, 1.0, (S, d))
    r = bounds.attention_dout_sensitivity(q, k, v, sig2)
    base = O.attention_bwd(q, k, v, do)
    J = np.zeros((3, S, d, S, d))
    for t in range(S):
        for e in range(d):
            dd = do.copy()
            dd[t, e] += 1.0
            for i, out in enumerate(O.attention_bwd(q, k, v, dd)):
                J[i, :, :, t, e] = out - base[i]
    for i, key in enumerate(("dq", "dk", "dv")):
        var = np.einsum("abte,te->ab", J[i] ** 2, sig2)
        np.testing.assert_allclose(r[key], var, rtol=1e-9, atol=1e-14)
        col = np.einsum("bte,te->b", J[i].sum(0) ** 2, sig2)
        np.testing.assert_allclose(r["sum_" + key], col, rtol=1e-9, atol=1e-12)
    # the column sums' identities: sum_u dV_u = sum_t dO_t, sum_u dK_u = 0
    np.testing.assert_allclose(r["sum_dv"], sig2.sum(0), rtol=1e-12)
    assert np.all(r["sum_dk"] == 0)


def test_attention_qkv_sensitivity_matches_a_numerical_jacobian():
    """First-order variance of the attention output under independent errors
    of q, k, v, against central differences of the oracle's forward."""
    rng = np.random.default_rng(4)
    S, d = 6, 4
    q, k, v = (rng.standard_normal((S, d)) for _ in range(3))
    var = [rng.uniform(0.01, 1.0, (S, d)) for _ in range(3)]
    got = bounds.attention_qkv_sensitivity(q, k, v, *var)
    want = np.zeros((S, d))
    eps = 1e-6
    for which in range(3):
        for t in range(S):
            for e in range(d):
                args = [q.copy(), k.copy(), v.copy()]
                args[which][t, e] += eps
                up, _ = O.attention_fwd(*args)
                args[which][t, e] -= 2 * eps
                dn, _ = O.attention_fwd(*args)
                col = (up - dn) / (2 * eps)
                want += col ** 2 * var[which][t, e]
    np.testing.assert_allclose(got, want, rtol=1e-6, atol=1e-12)


def test_propagated_sums_cover_real_roundings():
    """left/right/colsum: the variance they propagate is the exact variance of
    a product of V's uniform rounding errors (a Monte Carlo of real bf16
    roundings of random V stays inside six standard deviations, and its
    sample variance matches the model), and for at most 12 terms six standard
    deviations bound even the worst case, where every error is ulp/2 with the
    sign of its weight."""
    rng = np.random.default_rng(5)
    T, K, N = 64, 48, 16
    w = rng.standard_normal((K, N))
    x = rng.standard_normal((K, T))
    errs_l, errs_r, errs_c = [], [], []
    for _ in range(200):
        v = rng.standard_normal((T, K)) * rng.uniform(0.1, 10.0)
        vb = torch.tensor(v).to(torch.float32).to(torch.bfloat16).to(torch.float64).numpy()
        d = vb - v
        var = bounds.rounding_var(v)
        for got, bnd, acc in ((d @ w, bounds.left(var, w), errs_l),
                              (x @ d, bounds.right(x.T, var), errs_r),
                              (d.sum(0), bounds.colsum(var), errs_c)):
            assert np.all(np.abs(got) <= bnd)
            acc.append((got / (bnd / bounds.SIGMAS)) ** 2)
    for acc in (errs_l, errs_r, errs_c):
        ratio = float(np.mean(np.concatenate([a.ravel() for a in acc])))
        assert 0.8 < ratio < 1.2, ratio           # the model's variance is the real one
    for n in range(1, 13):
        worst = n * 0.5                            # n errors of ulp/2 (ulp = 1), all aligned
        assert bounds.SIGMAS * np.sqrt(n / 12.0) >= worst - 1e-12


def test_attention_prob_bounds_match_sampled_roundings():
    """The terms of attention_prob_bounds against sampled roundings: P from
    torch's float64 softmax, dS = P (dO V^T - rowsum(dO o)), errors drawn
    uniform on +-ulp/2 at every nonzero P and dS and pushed through the
    products dV = P^T dO, dK = dS^T Q / sqrt(d), dQ = dS K / sqrt(d); the
    sampled standard deviations times SIGMAS give the bounds."""
    rng = np.random.default_rng(5)
    S, d, n = 6, 4, 20000
    q, k, v, do = (rng.standard_normal((S, d)) for _ in range(4))
    bq, bk, bv = bounds.attention_prob_bounds(q, k, v, do)
    s = torch.tensor(q @ k.T / np.sqrt(d))
    s = s.masked_fill(torch.triu(torch.ones(S, S, dtype=torch.bool), 1), float("-inf"))
    P = torch.softmax(s, dim=1).numpy()
    dS = P * (do @ v.T - (do * (P @ v)).sum(1)[:, None])
    ep = rng.uniform(-0.5, 0.5, (n, S, S)) * (bounds.ulp_bf16(P) * (P != 0))
    es = rng.uniform(-0.5, 0.5, (n, S, S)) * (bounds.ulp_bf16(dS) * (dS != 0))
    sampled = (np.einsum("ntu,te->nue", ep, do),
               np.einsum("ntu,te->nue", es, q) / np.sqrt(d),
               np.einsum("ntu,ue->nte", es, k) / np.sqrt(d))
    for err, b, nm in zip(sampled, (bv, bk, bq), ("dv", "dk", "dq")):
        assert b.shape == (S, d), nm
        np.testing.assert_allclose(bounds.SIGMAS * err.std(0), b, rtol=0.05, err_msg=nm)
