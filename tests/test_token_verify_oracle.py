"""Pins of the token verification oracle (CPU only).

The oracle restates modified rejection sampling (paper Sec. 1 and Sec. 6; the
published scheme of Leviathan et al. 2023 / Chen et al. 2023).  It is pinned
here by what the mathematics fixes, not by itself:
  * the guarantee the paper relies on: the first emitted token of a round is
    distributed exactly as the target's p_1 (grid quadrature over every draft
    token and a grid of uniforms), and every later emitted token as its p_i;
  * the law of the accepted count: P(n >= i) = prod_{j <= i} alpha_j with
    alpha_j = sum_x min(p_j(x), q_j(x))  (chi-square on seeded trials);
  * hand-computed inverse-CDF thresholds and exact ties of the accept test;
  * special cases: p == q accepts everything, p(x) = 0 always rejects, a
    one-hot residual is drawn regardless of the uniform, the Z = 0 fallback,
    out-of-range draft tokens, rows without probability mass.
A final test plants plausible mistakes into copies of the oracle and checks
that every one of them fails some pin.
"""
from __future__ import annotations

import os
import types

import numpy as np
import pytest
from scipy import stats

from oracle import token_verify as TV

ORACLE_SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle",
                          "token_verify.py")


# ---------------------------------------------------------------------------
# pin checks, written against any module with the oracle's interface
# ---------------------------------------------------------------------------
def _dist(rng, V, conc=1.0):
    x = rng.gamma(conc, size=V)
    return (x / x.sum()).astype(np.float32)


def check_inverse_cdf_hand_values(M):
    # weights 0, 3/8, 0, 5/8 (exact binary fractions): tokens 1 and 3 only
    p = np.array([0.0, 0.375, 0.0, 0.625], np.float32)
    W = M.weights(p)
    assert W.tolist() == [0, 3 * 2 ** 37, 0, 5 * 2 ** 37]
    assert M.inverse_cdf(W, 0.0) == 1
    assert M.inverse_cdf(W, 0.375 - 2.0 ** -24) == 1
    assert M.inverse_cdf(W, 0.375) == 3               # T lands exactly on C(1): next token
    assert M.inverse_cdf(W, 1.0 - 2.0 ** -24) == 3
    assert M.inverse_cdf(W, 1.0) == 3                 # clamped uniform
    assert M.inverse_cdf(W, float("inf")) == 3
    assert M.inverse_cdf(W, float("nan")) == 1        # NaN uniform counts as 0
    assert M.inverse_cdf(np.zeros(4, np.int64), 0.5) == -1
    # correction weights: positive part of p - q, 0.75 - 0.25 = 0.5 exactly
    Wc = M.weights(np.array([0.75, 0.25, 0.0], np.float32), np.array([0.25, 0.5, 0.25], np.float32))
    assert Wc.tolist() == [2 ** 39, 0, 0]
    # values outside [0, 1] are clamped; NaN weighs nothing
    assert M.weights(np.array([2.0, -0.5, np.nan, 0.5], np.float32)).tolist() == [2 ** 40, 0, 0, 2 ** 39]


def check_accept_exact_ties(M):
    # u * q == p exactly: not accepted (strict); one ulp more p: accepted
    assert not M.accept(0.5, 0.5, 0.25)
    assert M.accept(0.5, 0.5, np.nextafter(np.float32(0.25), np.float32(1)))
    # the fp32 quotient p / q would round: 1/3 vs 0.1 / 0.3
    u, q, p = np.float32(1 / 3), np.float32(0.3), np.float32(0.1)
    exact = float(u) * float(q) < float(p)
    assert M.accept(u, q, p) == exact
    assert not M.accept(float("nan"), 0.5, 0.5)


def check_first_token_quadrature(M, V=4, G=64):
    """sum_x q(x) * P_{r,u}(first emitted token = y | x) == p(y) (k = 1)."""
    rng = np.random.default_rng(7)
    p1 = _dist(rng, V)
    q1 = _dist(rng, V)
    p2 = _dist(rng, V)
    grid = (np.arange(G, dtype=np.float64) + 0.5) / G
    xs, rs, us = np.meshgrid(np.arange(V), grid, grid, indexing="ij")
    Bn = xs.size
    P = np.broadcast_to(np.stack([p1, p2])[None], (Bn, 2, V)).copy()
    Q = np.broadcast_to(q1[None, None], (Bn, 1, V)).copy()
    n, tok = M.verify_tokens(P, Q, xs.reshape(Bn, 1), rs.reshape(Bn, 1).astype(np.float32),
                             us.reshape(Bn).astype(np.float32))
    wq = q1.astype(np.float64)[xs.reshape(Bn)] / (G * G)
    freq = np.array([wq[tok[:, 0] == y].sum() for y in range(V)])
    assert np.all(tok[:, 0] >= 0)
    np.testing.assert_allclose(freq, p1.astype(np.float64), atol=3.0 / G)


def _trials(M, k, V, N, seed):
    rng = np.random.default_rng(seed)
    p = np.stack([_dist(rng, V, 0.7) for _ in range(k + 1)])
    q = np.stack([_dist(rng, V, 0.7) for _ in range(k)])
    q64 = q.astype(np.float64)
    draft = np.stack([rng.choice(V, size=N, p=q64[i] / q64[i].sum()) for i in range(k)], axis=1)
    ua = rng.random((N, k), dtype=np.float32)
    us = rng.random(N, dtype=np.float32)
    P = np.broadcast_to(p[None], (N, k + 1, V)).copy()
    Q = np.broadcast_to(q[None], (N, k, V)).copy()
    n, tok = M.verify_tokens(P, Q, draft, ua, us)
    return p.astype(np.float64), q.astype(np.float64), n, tok


def check_accept_count_law(M, k=3, V=6, N=30000):
    p, q, n, _ = _trials(M, k, V, N, seed=11)
    alpha = np.minimum(p[:k], q).sum(axis=1)
    surv = np.concatenate([[1.0], np.cumprod(alpha)])          # P(n >= i), i = 0..k
    law = surv[:k + 1] - np.concatenate([surv[1:k + 1], [0.0]])
    obs = np.bincount(n, minlength=k + 1)
    res = stats.chisquare(obs, law * N)
    assert res.pvalue > 1e-4, (obs, law * N)


def check_emitted_token_laws(M, k=3, V=6, N=30000):
    """The token emitted at position i (given the round reaches it) ~ p_i."""
    p, q, n, tok = _trials(M, k, V, N, seed=23)
    for i in range(k + 1):
        reach = n >= i
        obs = np.bincount(tok[reach, i], minlength=V)
        assert obs.sum() == reach.sum() and (tok[reach, i] >= 0).all()
        res = stats.chisquare(obs, p[i] / p[i].sum() * obs.sum())
        assert res.pvalue > 1e-4, (i, obs, p[i] * obs.sum())


def check_special_cases(M):
    rng = np.random.default_rng(3)
    V, k, B = 16, 4, 64
    p = np.stack([np.stack([_dist(rng, V) for _ in range(k + 1)]) for _ in range(B)])
    draft = rng.integers(0, V, size=(B, k))
    ua = rng.random((B, k), dtype=np.float32)
    us = rng.random(B, dtype=np.float32)
    # identical distributions: everything accepted, the bonus comes from p_{k+1}
    n, tok = M.verify_tokens(p, p[:, :k].copy(), draft, ua, us)
    assert (n == k).all() and (tok[:, :k] == draft).all()
    for b in range(B):
        assert tok[b, k] == M.inverse_cdf(M.weights(p[b, k]), us[b])
    # zero target probability of draft token 2: rejected there whenever reached
    p0 = p.copy()
    p0[np.arange(B), 2, draft[:, 2]] = 0.0
    n, tok = M.verify_tokens(p0, p[:, :k].copy(), draft, ua, us)
    assert (n == 2).all()
    assert (tok[:, 3:] == -1).all()
    # one-hot target at token 5 on the rejected row: correction is 5 for any uniform
    q = np.stack([np.stack([_dist(rng, V) for _ in range(k)]) for _ in range(B)])
    q[:, 0, 5] = 0.0
    q[:, 0] /= q[:, 0].sum(axis=1, keepdims=True)
    p1 = p.copy()
    p1[:, 0] = 0.0
    p1[:, 0, 5] = 1.0
    d1 = draft.copy()
    d1[:, 0] = (5 + 1 + np.arange(B)) % V
    d1[d1[:, 0] == 5, 0] = 6
    for uu in (0.0, 0.5, 1.0 - 2.0 ** -24):
        n, tok = M.verify_tokens(p1, q, d1, ua, np.full(B, uu, np.float32))
        assert (n == 0).all() and (tok[:, 0] == 5).all() and (tok[:, 1:] == -1).all()
    # out-of-range draft tokens are rejected
    d2 = draft.copy()
    d2[:, 1] = np.where(np.arange(B) % 2 == 0, -1, V)
    n, _ = M.verify_tokens(p, p[:, :k].copy(), d2, ua, us)
    assert (n == 1).all()
    # rejected although p == q (uniform of 1.0): residual is empty, p is sampled
    ua1 = ua.copy()
    ua1[:, 0] = 1.0
    n, tok = M.verify_tokens(p, p[:, :k].copy(), draft, ua1, us)
    assert (n == 0).all()
    for b in range(B):
        assert tok[b, 0] == M.inverse_cdf(M.weights(p[b, 0]), us[b]) >= 0
    # no probability mass anywhere: token -1
    n, tok = M.verify_tokens(np.zeros((2, 1, V), np.float32), np.zeros((2, 0, V), np.float32),
                             np.zeros((2, 0), np.int64), np.zeros((2, 0), np.float32),
                             np.full(2, 0.5, np.float32))
    assert (n == 0).all() and (tok[:, 0] == -1).all()
    # a token of zero weight is never drawn, at either end of the uniform range
    w = np.array([0.0, 0.5, 0.0, 0.0, 0.5, 0.0], np.float32)
    for uu in (0.0, 2.0 ** -24, 0.5 - 2.0 ** -24, 0.5, 1.0 - 2.0 ** -24):
        assert M.inverse_cdf(M.weights(w), uu) in (1, 4)


CHECKS = [check_inverse_cdf_hand_values, check_accept_exact_ties, check_first_token_quadrature,
          check_accept_count_law, check_emitted_token_laws, check_special_cases]


# ---------------------------------------------------------------------------
@pytest.mark.parametrize("check", CHECKS, ids=[c.__name__ for c in CHECKS])
def test_oracle_pin(check):
    check(TV)


def test_threshold_is_exact_for_large_sums():
    # Z close to 2^60 (V = 2^20 weights of 1.0): T = floor(U * Z / 2^24) exactly
    Z = (2 ** 20) * (2 ** 40)
    U = 2 ** 24 - 1
    assert TV.threshold(U / 2 ** 24, Z) == (U * Z) // 2 ** 24
    assert TV.threshold(0.25, 12345678901234) == 12345678901234 // 4


# ---------------------------------------------------------------------------
# planted mistakes: each must fail at least one pin
# ---------------------------------------------------------------------------
MUTANTS = {
    "ratio_inverted": ("float(np.float32(u)) * float(np.float32(q_x)) < float(np.float32(p_x))",
                       "float(np.float32(u)) * float(np.float32(p_x)) < float(np.float32(q_x))"),
    "non_strict_accept": ("float(np.float32(q_x)) < float(np.float32(p_x))",
                          "float(np.float32(q_x)) <= float(np.float32(p_x))"),
    "residual_abs": ("w = np.where(w > 0, w, np.float32(0.0))", "w = np.abs(w)"),
    "residual_from_p": ("tok = inverse_cdf(weights(p[b, n], q[b, n]), u_sample[b])",
                        "tok = inverse_cdf(weights(p[b, n]), u_sample[b])"),
    "residual_from_next_row": ("tok = inverse_cdf(weights(p[b, n], q[b, n]), u_sample[b])",
                               "tok = inverse_cdf(weights(p[b, n + 1], q[b, n]), u_sample[b])"),
    "bonus_from_last_draft_row": ("tok = inverse_cdf(weights(p[b, k]), u_sample[b])",
                                  "tok = inverse_cdf(weights(p[b, k - 1]), u_sample[b])"),
    "searchsorted_left": ('side="right"', 'side="left"'),
    "same_accept_uniform": ("accept(u_accept[b, n], q[b, n, x], p[b, n, x])",
                            "accept(u_accept[b, 0], q[b, n, x], p[b, n, x])"),
    "rejected_token_counted": ("            if not accept(u_accept[b, n], q[b, n, x], p[b, n, x]):\n"
                               "                break\n",
                               "            if not accept(u_accept[b, n], q[b, n, x], p[b, n, x]):\n"
                               "                n += 1\n                break\n"),
    "shifted_prefix": ("out[b, :n] = draft[b, :n]", "out[b, :n] = np.roll(draft[b], 1)[:n]"),
    "uniform_not_clamped": ("    elif uf >= 1.0:", "    elif uf > 1.0:"),
    "weight_not_clamped_at_one": ("w = np.minimum(w, np.float32(1.0))", "w = w"),
    "no_zero_sum_fallback": ("            if tok < 0:\n                tok = inverse_cdf(weights(p[b, n]), u_sample[b])\n",
                             ""),
}


def _mutant(name, old, new):
    src = open(ORACLE_SRC).read()
    assert src.count(old) >= 1, f"mutation {name} does not apply"
    mod = types.ModuleType(f"tv_mutant_{name}")
    exec(compile(src.replace(old, new), f"<mutant {name}>", "exec"), mod.__dict__)
    return mod


def _fails_some_pin(M):
    for check in CHECKS:
        try:
            check(M)
        except Exception:  # AssertionError or a crash both count as caught
            return True
    return False


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(name):
    old, new = MUTANTS[name]
    assert _fails_some_pin(_mutant(name, old, new)), f"mutant {name} passed every pin"
