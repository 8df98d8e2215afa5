"""Pins of the oracle's speculative accept/resample rule against facts fixed by the
published method (Leviathan et al. 2023; Chen et al. 2023), which the verify step
applies at temperature 1 (paper Sec. 4.1 control table; Sec. 5.3, 5.4): hand-worked
cases, accepted length <= k, p == q accepts every draft, one-hot p is
deterministic, k = 0 is plain inverse-CDF sampling, the emitted-token law equals
the target law (chi-square over 1e6 seeded trials on a 16-token vocabulary, and a
deterministic quadrature of the law), and the closed-form acceptance rate."""
import json
import os

import numpy as np
import pytest
from scipy import stats

from oracle import sampler

HERE = os.path.dirname(os.path.abspath(__file__))


def _softmax_rows(l):
    l = np.asarray(l, np.float64)
    e = np.exp(l - l.max(axis=-1, keepdims=True))
    return e / e.sum(axis=-1, keepdims=True)


def test_hand_worked_cases():
    cases = json.load(open(os.path.join(HERE, "golden", "sampler_hand_cases.json")))["cases"]
    for c in cases:
        q = None if c["q"] is None else np.array(c["q"], np.float32)
        r = sampler.spec_accept(np.array(c["logits"], np.float32), np.array(c["drafts"]),
                                np.array(c["u"], np.float32), q)
        assert r["tokens"].tolist() == c["tokens"], c["name"]
        assert r["n_accepted"].tolist() == c["n_accepted"], c["name"]
        want = np.array([[np.nan if v is None else v for v in row] for row in c["logprobs"]])
        np.testing.assert_allclose(r["logprobs"], want, atol=1e-6, equal_nan=True, err_msg=c["name"])


def test_accepted_length_bounded_and_padding():
    rng = np.random.default_rng(1)
    B, k, V = 300, 5, 40
    l = rng.normal(size=(B, k + 1, V)).astype(np.float32)
    q = _softmax_rows(rng.normal(size=(B, k, V))).astype(np.float32)
    d = rng.integers(0, V, (B, k))
    u = rng.random((B, k + 1)).astype(np.float32)
    r = sampler.spec_accept(l, d, u, q)
    n = r["n_accepted"]
    assert ((n >= 0) & (n <= k)).all()
    for b in range(B):
        assert (r["tokens"][b, : n[b]] == d[b, : n[b]]).all()       # accepted drafts kept
        assert 0 <= r["tokens"][b, n[b]] < V                         # one emitted token
        assert (r["tokens"][b, n[b] + 1:] == -1).all()
        assert np.isnan(r["logprobs"][b, n[b] + 1:]).all()
        assert np.isfinite(r["logprobs"][b, : n[b] + 1]).all()


def test_p_equals_q_accepts_everything():
    rng = np.random.default_rng(2)
    B, k, V = 500, 4, 64
    l = (rng.normal(size=(B, k + 1, V)) * 2).astype(np.float32)
    q = _softmax_rows(l[:, :k]).astype(np.float32)        # q = p, rounded once to float32
    d = np.array([[rng.choice(V, p=q[b, i] / q[b, i].sum()) for i in range(k)] for b in range(B)])
    u = np.nextafter(np.float32(1), np.float32(0)) * np.ones((B, k + 1), np.float32)  # worst case u
    u[:, :] = np.maximum(u, rng.random((B, k + 1)).astype(np.float32))
    r = sampler.spec_accept(l, d, u, q)
    assert (r["n_accepted"] == k).all()


def test_one_hot_target_is_deterministic():
    rng = np.random.default_rng(3)
    B, k, V = 200, 3, 16
    a = rng.integers(0, V, (B, k + 1))
    l = np.full((B, k + 1, V), -np.inf, np.float32)
    for b in range(B):
        for j in range(k + 1):
            l[b, j, a[b, j]] = rng.normal()
    q = _softmax_rows(rng.normal(size=(B, k, V))).astype(np.float32)
    d = rng.integers(0, V, (B, k))
    d[::2] = a[::2, :k]                                 # half the drafts are the argmax
    u = rng.random((B, k + 1)).astype(np.float32)
    r = sampler.spec_accept(l, d, u, q)
    for b in range(B):
        n = r["n_accepted"][b]
        want_n = 0
        while want_n < k and d[b, want_n] == a[b, want_n]:
            want_n += 1
        assert n == want_n
        assert (r["tokens"][b, : n + 1] == a[b, : n + 1]).all()
        np.testing.assert_allclose(r["logprobs"][b, : n + 1], 0.0, atol=0)


def test_k_zero_is_inverse_cdf_sampling():
    rng = np.random.default_rng(4)
    B, V = 2000, 50
    l = rng.normal(size=(B, 1, V)).astype(np.float32)
    u = rng.random((B, 1)).astype(np.float32)
    r = sampler.spec_accept(l, np.zeros((B, 0), np.int64), u, None)
    assert (r["n_accepted"] == 0).all()
    p = _softmax_rows(l[:, 0])
    c = np.cumsum(p, axis=1)
    direct = np.array([np.searchsorted(c[b], np.float64(u[b, 0]), side="right") for b in range(B)])
    # continuous inverse CDF agrees except within 1e-9 of a boundary (grid quantisation)
    dist = np.min(np.abs(c - u.astype(np.float64)), axis=1)
    ok = dist > 1e-9
    assert ok.mean() > 0.99
    assert (r["tokens"][ok, 0] == direct[ok]).all()


def _chi2_setup(V=16, k=3, seed=5):
    rng = np.random.default_rng(seed)
    lp = rng.normal(size=(k + 1, V)) * 1.5
    lq = lp[:k] + rng.normal(size=(k, V)) * 1.0
    p = _softmax_rows(lp)
    q = _softmax_rows(lq).astype(np.float32)
    return lp.astype(np.float32), p, q


def test_emitted_law_equals_target_chi_square_1e6():
    """1e6 seeded trials, V = 16: drafts x_i ~ q_i; at every position the emitted token
    (accepted draft or replacement) must follow p_{i-1} given the position is reached."""
    V, k, N = 16, 3, 1_000_000
    lp, p, q = _chi2_setup(V, k)
    rng = np.random.Generator(np.random.Philox(12345))
    drafts = np.stack([rng.choice(V, size=N, p=q[i].astype(np.float64) / q[i].astype(np.float64).sum())
                       for i in range(k)], axis=1)
    u = rng.random((N, k + 1), dtype=np.float32)
    logits = np.broadcast_to(lp, (N, k + 1, V))
    qq = np.broadcast_to(q, (N, k, V))
    r = sampler.spec_accept(logits, drafts, u, qq)
    tok, n = r["tokens"], r["n_accepted"]
    for pos in range(k + 1):
        reached = n >= pos                # a token is emitted at `pos` iff n >= pos
        counts = np.bincount(tok[reached, pos], minlength=V)
        exp = p[pos] * reached.sum()
        keep = exp > 5
        chi2 = (((counts - exp) ** 2 / exp)[keep]).sum()
        pval = stats.chi2.sf(chi2, keep.sum() - 1)
        assert pval > 1e-3, (pos, chi2, pval)
    # acceptance rate vs the closed form E[n] = sum_i prod_{j<=i} alpha_j
    alphas = [sampler.acceptance_prob(p[i], q[i].astype(np.float64)) for i in range(k)]
    en = sampler.expected_accepted(alphas)
    sd = n.std() / np.sqrt(N)
    assert abs(n.mean() - en) < 5 * sd, (n.mean(), en)


def test_first_token_law_by_quadrature():
    """Deterministic: integrate the rule over a grid of both uniforms for every draft
    (k = 1, V = 4) and weight by q; the law of the first emitted token must be p0
    up to the grid's resolution."""
    V, G = 4, 400
    lp = np.array([[0.3, -1.0, 1.2, 0.0], [0.0, 0.5, -0.5, 0.1]], np.float32)
    p0 = _softmax_rows(lp[0])
    q = np.array([[0.4, 0.3, 0.1, 0.2]], np.float32)
    grid = ((np.arange(G) + 0.5) / G).astype(np.float32)
    u0, u1 = np.meshgrid(grid, grid, indexing="ij")
    U = np.stack([u0.ravel(), u1.ravel()], axis=1)
    law = np.zeros(V)
    for x in range(V):
        N = U.shape[0]
        r = sampler.spec_accept(np.broadcast_to(lp, (N, 2, V)), np.full((N, 1), x), U,
                                np.broadcast_to(q, (N, 1, V)))
        law += q[0, x] * np.bincount(r["tokens"][:, 0], minlength=V) / N
    np.testing.assert_allclose(law, p0, atol=3.0 / G)


def test_residual_mass_zero_falls_back_to_p():
    """p = [1/2, 1/2]; q = [1/2, 1/2 + 2^-24] (a caller's q may sum past 1 by rounding).
    Draft 1 with u = 1 - 2^-24 >= p/q is rejected, max(0, p - q) is zero everywhere, and
    the final token is drawn from p with the same uniform."""
    l = np.zeros((2, 2, 2), np.float32)
    q = np.array([[[0.5, 0.5 + 2.0 ** -24]]] * 2, np.float32)
    u = np.array([[1 - 2.0 ** -24, 0.3], [1 - 2.0 ** -24, 0.7]], np.float32)
    r = sampler.spec_accept(l, np.array([[1], [1]]), u, q)
    assert r["n_accepted"].tolist() == [0, 0]
    assert r["tokens"][:, 0].tolist() == [0, 1]
    j, tot, _ = sampler.fixed_point_draw(np.zeros((1, 4)), np.array([0.3], np.float32))
    assert tot[0] == 0 and j[0] == -1


def test_fixed_point_target_arithmetic():
    # the 128-bit target split agrees with Python's exact integers
    rng = np.random.default_rng(6)
    r = rng.random((50, 33))
    r /= r.sum(axis=1, keepdims=True)           # a distribution (mass <= 1)
    u = rng.random(50).astype(np.float32)
    j, tot, _ = sampler.fixed_point_draw(r, u)
    for i in range(50):
        R = [int(x) for x in np.floor(r[i] * 2.0 ** 62)]
        T = sum(R)
        assert T == int(tot[i])
        target = (T * int(np.floor(np.float64(u[i]) * 2 ** 32))) >> 32
        c = 0
        for idx, x in enumerate(R):
            c += x
            if c > target:
                break
        assert idx == j[i]
