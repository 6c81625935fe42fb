"""Pins of the block verification oracle (CPU only).

The oracle restates block verification (the alternative to token verification
the paper names in Sec. 6).  It is pinned by what defines a valid verification
scheme and by what makes block verification the better one, both checked by
exact enumeration over every draft block and every emitted sequence of small
random models whose distributions depend on the whole prefix:
  * losslessness: the emitted tokens of a round, continued with samples of the
    target, have exactly the target's sequence distribution;
  * E[emitted tokens] is at least token verification's (computed here from its
    own definition, not from the oracle under test);
and further by the sampled form agreeing with the exact distribution
(chi-square over seeded rounds), special cases, hand-computed decisions at
their boundaries, and planted mistakes that the enumeration must catch."""
import itertools
import math
import types

import numpy as np
import pytest

from oracle import block_verify as BV
from oracle import token_verify as TV


def _models(V, k, seed):
    """Target (Mb) and draft (Ms) distributions for every prefix up to k+1 tokens."""
    rng = np.random.default_rng(seed)
    Mb, Ms = {}, {}
    for L in range(k + 2):
        for pre in itertools.product(range(V), repeat=L):
            a = rng.gamma(0.6, size=V)
            c = rng.gamma(0.6, size=V)
            Mb[pre] = a / a.sum()
            Ms[pre] = c / c.sum()
    return Mb, Ms


def _rows(Mb, Ms, X):
    k = len(X)
    P = np.stack([Mb[tuple(X[:i])] for i in range(k + 1)])
    Q = np.stack([Ms[tuple(X[:i])] for i in range(k)]) if k else np.zeros((0, P.shape[1]))
    return P, Q


def _token_distribution(P, Q, X):
    """Token verification's exact output distribution, from its definition."""
    k, dist, acc = len(X), {}, 1.0
    for i in range(k):
        a = min(1.0, P[i, X[i]] / Q[i, X[i]])
        r = np.maximum(P[i] - Q[i], 0.0)
        if r.sum() > 0:
            for y in range(P.shape[1]):
                key = tuple(X[:i]) + (y,)
                dist[key] = dist.get(key, 0.0) + acc * (1 - a) * r[y] / r.sum()
        acc *= a
    for y in range(P.shape[1]):
        key = tuple(X) + (y,)
        dist[key] = dist.get(key, 0.0) + acc * P[k, y]
    return dist


def _round_distribution(Mb, Ms, V, k, dist_fn):
    """Emitted-sequence distribution of one round, the draft block drawn from Ms."""
    total = {}
    for X in itertools.product(range(V), repeat=k):
        px = math.prod(Ms[X[:i]][X[i]] for i in range(k))
        P, Q = _rows(Mb, Ms, X)
        for seq, pr in dist_fn(P, Q, X).items():
            total[seq] = total.get(seq, 0.0) + px * pr
    return total


def _lossless_error(Mb, V, k, total):
    """max over z in V^{k+1} of |P(round then target continuation = z) - Mb(z)|."""
    worst = 0.0
    for z in itertools.product(range(V), repeat=k + 1):
        lhs = 0.0
        for j in range(1, k + 2):
            pr = total.get(z[:j], 0.0)
            for i in range(j, k + 1):
                pr *= Mb[z[:i]][z[i]]
            lhs += pr
        rhs = math.prod(Mb[z[:i]][z[i]] for i in range(k + 1))
        worst = max(worst, abs(lhs - rhs))
    return worst


@pytest.mark.parametrize("V,k,seed", [(2, 1, 0), (3, 2, 1), (3, 3, 2), (4, 2, 3), (2, 4, 4)])
def test_lossless_and_at_least_token_verification(V, k, seed):
    Mb, Ms = _models(V, k, seed)
    block = _round_distribution(Mb, Ms, V, k, BV.output_distribution)
    token = _round_distribution(Mb, Ms, V, k, _token_distribution)
    assert sum(block.values()) == pytest.approx(1.0, abs=1e-12)
    assert _lossless_error(Mb, V, k, block) < 1e-12
    assert _lossless_error(Mb, V, k, token) < 1e-12   # the comparison scheme is itself valid
    e_block = sum(len(s) * p for s, p in block.items())
    e_token = sum(len(s) * p for s, p in token.items())
    assert e_block >= e_token - 1e-12
    if k >= 2:
        assert e_block > e_token + 1e-6   # strictly better on these random models


def _fixed_case():
    rng = np.random.default_rng(7)
    V, k = 5, 3
    P = rng.gamma(0.8, size=(k + 1, V)).astype(np.float32)
    P /= P.sum(-1, keepdims=True)
    Q = rng.gamma(0.8, size=(k, V)).astype(np.float32)
    Q /= Q.sum(-1, keepdims=True)
    X = np.array([int(np.argmax(Q[i])) for i in range(k)])  # likely draft tokens
    return P.astype(np.float32), Q.astype(np.float32), X


def test_sampled_form_follows_the_exact_distribution():
    P, Q, X = _fixed_case()
    k, V = len(X), P.shape[1]
    exact = BV.output_distribution(P.astype(np.float64), Q.astype(np.float64), X)
    N = 40000
    rng = np.random.default_rng(11)
    ua = rng.random((N, k), dtype=np.float32)
    us = rng.random(N, dtype=np.float32)
    n, toks = BV.verify_block(np.broadcast_to(P, (N, k + 1, V)), np.broadcast_to(Q, (N, k, V)),
                              np.broadcast_to(X, (N, k)), ua, us)
    counts = {}
    for b in range(N):
        key = tuple(int(t) for t in toks[b, : n[b] + 1])
        counts[key] = counts.get(key, 0) + 1
    assert set(counts) <= set(exact)
    chi2, dof = 0.0, -1
    for key, pr in exact.items():
        e = N * pr
        if e < 5:
            continue
        chi2 += (counts.get(key, 0) - e) ** 2 / e
        dof += 1
    # chi-square with dof degrees of freedom: mean dof, sd sqrt(2 dof); 6 sd is far out
    assert chi2 < dof + 6 * math.sqrt(2 * dof)


def test_identical_models_accept_every_draft_token():
    P, Q, X = _fixed_case()
    k, V = len(X), P.shape[1]
    Pq = P.copy()
    Pq[:k] = Q
    rng = np.random.default_rng(3)
    n, toks = BV.verify_block(np.broadcast_to(Pq, (200, k + 1, V)), np.broadcast_to(Q, (200, k, V)),
                              np.broadcast_to(X, (200, k)), rng.random((200, k), dtype=np.float32),
                              rng.random(200, dtype=np.float32))
    assert (n == k).all()
    assert (toks[:, :k] == X).all()


def test_zero_target_probability_bounds_the_accepted_prefix():
    P, Q, X = _fixed_case()
    k, V = len(X), P.shape[1]
    P = P.copy()
    P[1, X[1]] = 0.0  # the second draft token is impossible under the target
    pw = BV.prefix_weights(P, Q, X)
    assert pw[2] == 0.0 and pw[3] == 0.0
    rng = np.random.default_rng(5)
    n, _ = BV.verify_block(np.broadcast_to(P, (500, k + 1, V)), np.broadcast_to(Q, (500, k, V)),
                           np.broadcast_to(X, (500, k)), rng.random((500, k), dtype=np.float32),
                           rng.random(500, dtype=np.float32))
    assert n.max() <= 1


def test_out_of_range_draft_tokens_are_never_accepted():
    P, Q, X = _fixed_case()
    k, V = len(X), P.shape[1]
    for bad in (-1, V):
        Xb = X.copy()
        Xb[0] = bad
        assert BV.prefix_weights(P, Q, Xb)[1:] == [0.0] * k
        n, toks = BV.verify_block(P[None], Q[None], Xb[None], np.zeros((1, k), np.float32),
                                  np.full(1, 0.3, np.float32))
        assert n[0] == 0 and 0 <= toks[0, 0] < V


def test_no_draft_tokens_is_token_verification():
    rng = np.random.default_rng(9)
    V, B = 50, 64
    P = rng.random((B, 1, V), dtype=np.float32)
    P /= P.sum(-1, keepdims=True)
    us = rng.random(B, dtype=np.float32)
    a = BV.verify_block(P, np.zeros((B, 0, V), np.float32), np.zeros((B, 0), np.int32),
                        np.zeros((B, 0), np.float32), us)
    b = TV.verify_tokens(P, np.zeros((B, 0, V), np.float32), np.zeros((B, 0), np.int32),
                         np.zeros((B, 0), np.float32), us)
    assert (a[0] == b[0]).all() and (a[1] == b[1]).all()


def test_stop_decisions_at_their_boundaries():
    """k = 1: h_1 = p_1 = P_0(x) / Q_0(x) exactly; with p_1 = 1/2 a uniform just
    below 1/2 stops at 1, 1/2 itself does not (strict test)."""
    V = 4
    Q = np.array([[0.5, 0.25, 0.125, 0.125]], np.float32)
    P = np.array([[0.25, 0.25, 0.25, 0.25], [0.0, 1.0, 0.0, 0.0]], np.float32)
    X = np.array([0])
    assert BV.prefix_weights(P, Q, X) == [1.0, 0.5]
    below = np.float32(np.nextafter(np.float32(0.5), np.float32(0.0)))
    n, toks = BV.verify_block(P[None], Q[None], X[None], np.array([[below]], np.float32), np.array([0.9], np.float32))
    assert n[0] == 1 and toks[0, 1] == 1         # accepted; bonus from P_1 = one-hot at 1
    n, toks = BV.verify_block(P[None], Q[None], X[None], np.array([[0.5]], np.float32), np.array([0.0], np.float32))
    assert n[0] == 0
    # residual of row 0 with p_0 = 1: max(P - Q, 0) = (0, 0, 0.125, 0.125): u = 0 takes token 2
    assert toks[0, 0] == 2


def test_residual_weights_hand_computed():
    P = np.array([0.5, 0.25, 0.25], np.float32)
    Q = np.array([0.125, 0.5, 0.375], np.float32)
    W = BV.row_weights(0.5, P, Q)   # 0.5 * P - Q = (0.125, -0.375, -0.25)
    assert W.tolist() == [2 ** 37, 0, 0]
    assert BV.row_weights(1.0, P).tolist() == [2 ** 39, 2 ** 38, 2 ** 38]
    # S / (S + (1 - p) 2^40) with S = 2^37, p = 1/2: 2^37 / (2^37 + 2^39) = 1/5
    assert BV.stop_probability(2 ** 37, 0.5) == pytest.approx(0.2, rel=1e-15)
    assert BV.stop_probability(0, 1.0) == 1.0   # 0/0 convention


# planted mistakes: each must break losslessness on one of the small models
MUTANTS = {
    "forward_walk": ("for i in range(k, -1, -1):", "for i in range(0, k + 1):"),
    "previous_weight_in_residual": ("r = np.maximum(p[i] * P[i] - Q[i], 0.0)",
                                    "r = np.maximum(p[max(i - 1, 0)] * P[i] - Q[i], 0.0)"),
    "no_cap_at_one": ("p.append(min(p[-1] * P[i - 1, x] / Q[i - 1, x], 1.0))",
                      "p.append(p[-1] * P[i - 1, x] / Q[i - 1, x])"),
    "top_always_stops": ("h.append(p[k])", "h.append(1.0)"),
    "residual_reversed": ("r = np.maximum(p[i] * P[i] - Q[i], 0.0)", "r = np.maximum(Q[i] - p[i] * P[i], 0.0)"),
    "stop_without_one_minus_p": ("den = s + 1.0 - p[i]", "den = s + 1.0"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistakes_are_caught(name):
    import inspect
    old, new = MUTANTS[name]
    src = inspect.getsource(BV.output_distribution)
    assert old in src
    mod = types.ModuleType("bv_mutant")
    mod.np = np
    exec(src.replace(old, new), mod.__dict__)
    caught = False
    for V, k, seed in [(3, 2, 1), (3, 3, 2), (2, 4, 4)]:
        Mb, Ms = _models(V, k, seed)
        try:
            total = _round_distribution(Mb, Ms, V, k, mod.output_distribution)
            err = _lossless_error(Mb, V, k, total)
        except (ZeroDivisionError, FloatingPointError, ValueError):
            err = math.inf
        if not err < 1e-9:
            caught = True
            break
    assert caught
