"""Block verification oracle (test infrastructure only).

Only the test suite, the package smoke check and the benchmark's CPU-baseline
leg use this module; the HIP library never does.  The paper verifies draft
tokens one at a time (token verification, paper Sec. 6) and notes that its
results should hold with block verification too (Sec. 6, citing Sun et al.
2024).  Block verification decides on the draft block as a whole; restated
from the published algorithm:

  p_0 = 1,   p_i = min(p_{i-1} * P_{i-1}(x_i) / Q_{i-1}(x_i), 1)      i = 1..k
  residual   r_i(x) = max(p_i * P_i(x) - Q_i(x), 0),  s_i = sum_x r_i(x)   i < k
  h_i = s_i / (s_i + 1 - p_i)  for i < k,   h_k = p_k
  going down from i = k, stop at the first i with eta_i ~ Bernoulli(h_i) = 1
  (h_0 = 1, so the walk always stops): tau = that i
  emit x_1..x_tau, then one token drawn from r_tau / s_tau (tau < k) or from
  P_k (tau = k)

P_i is the target's distribution of the token after x_1..x_i (row i of the
verify pass), Q_i the draft's for x_{i+1}.  The emitted tokens follow the
target's distribution exactly, and in expectation at least as many are
accepted as with token verification; `output_distribution` states the
algorithm in exact fp64 arithmetic so the tests can check both by enumeration.

Precision readings of the sampled form (`verify_block`); the HIP path takes
every decision in the same way, so results agree bit for bit:
  * p_i in fp64: with t = p_{i-1} * P(x) (fp64), p_i = 1 when t >= Q(x), else
    t / Q(x); p_i = 0 when p_{i-1} = 0, the token is outside [0, V), P(x) is
    not > 0 or Q(x) is not >= 0 (NaN included), and then every later p_j is 0;
  * residual weights: w(x) = p32 * P(x) - Q(x) with p32 = p_i rounded to fp32
    and both operations rounded in fp32 (no fused multiply-add), turned into
    the integer weights of token verification, floor(clamp(w, 0, 1) * 2^40);
    the row k weights are those of P_k (p32 = 1, no Q);
  * s_i = the exact integer sum of row i's weights, h_i decided in fp64 as
    S / (S + (1 - p_i) * 2^40) with S = s_i converted with one rounding
    (h_i = 1 when the denominator is 0), h_k = p_k; eta_i = 1 when u_i < h_i,
    u_i = u_accept[i - 1] (fp32), NaN compares false;
  * the emitted token: token verification's inverse CDF over the weights of
    row tau with the uniform u_sample; a residual row of total weight 0 draws
    from P_tau instead; a row of P of total weight 0 yields -1.
"""
from __future__ import annotations

import numpy as np

from oracle import token_verify as TV

TWO40 = float(2 ** TV.SHIFT)


def prefix_weights(p, q, draft) -> list:
    """p_0 .. p_k of one sequence (fp64), with the validity rules above.
    p [k+1, V], q [k, V] fp32; draft [k] ints."""
    k = len(draft)
    V = p.shape[-1]
    out = [1.0]
    for i in range(1, k + 1):
        prev = out[-1]
        x = int(draft[i - 1])
        if prev > 0.0 and 0 <= x < V:
            P = float(np.float32(p[i - 1, x]))
            Q = float(np.float32(q[i - 1, x]))
            if P > 0.0 and Q >= 0.0:
                t = prev * P
                out.append(1.0 if t >= Q else t / Q)
                continue
        out.append(0.0)
    return out


def row_weights(p_i: float, P_row, Q_row=None) -> np.ndarray:
    """Integer sampling weights of a residual row (Q given) or of P (Q None)."""
    P = np.asarray(P_row, dtype=np.float32)
    if Q_row is None:
        return TV.weights(P)
    scaled = np.multiply(np.float32(p_i), P, dtype=np.float32)   # one fp32 rounding per entry
    return TV.weights(scaled, np.asarray(Q_row, dtype=np.float32))


def to_f64(S: int) -> float:
    """An integer below 2^63 rounded once to fp64 (round to nearest even)."""
    return float(S)


def stop_probability(S: int, p_i: float) -> float:
    """h_i for a residual row: S / (S + (1 - p_i) 2^40) in fp64; 1 if that is 0/0."""
    Sd = to_f64(S)
    den = Sd + (1.0 - p_i) * TWO40
    if not den > 0.0:
        return 1.0
    return Sd / den


def verify_block(p, q, draft, u_accept, u_sample):
    """Block verification of a batch; same arguments and results as
    token_verify.verify_tokens: (n_accepted [B] int32, tokens [B, k+1] int32)."""
    p = np.asarray(p, dtype=np.float32)
    B, kp1, V = p.shape
    k = kp1 - 1
    q = np.asarray(q, dtype=np.float32).reshape(B, k, V)
    draft = np.asarray(draft).reshape(B, k)
    u_accept = np.asarray(u_accept, dtype=np.float32).reshape(B, k)
    u_sample = np.asarray(u_sample, dtype=np.float32).reshape(B)
    n_acc = np.zeros(B, dtype=np.int32)
    out = np.full((B, k + 1), -1, dtype=np.int32)
    for b in range(B):
        pw = prefix_weights(p[b], q[b], draft[b])
        tau = 0
        for i in range(k, 0, -1):
            if i == k:
                h = pw[k]
            else:
                h = stop_probability(int(row_weights(np.float32(pw[i]), p[b, i], q[b, i]).sum()), pw[i])
            if float(u_accept[b, i - 1]) < h:
                tau = i
                break
        out[b, :tau] = draft[b, :tau]
        if tau < k:
            tok = TV.inverse_cdf(row_weights(np.float32(pw[tau]), p[b, tau], q[b, tau]), u_sample[b])
            if tok < 0:
                tok = TV.inverse_cdf(row_weights(1.0, p[b, tau]), u_sample[b])
        else:
            tok = TV.inverse_cdf(row_weights(1.0, p[b, k]), u_sample[b])
        n_acc[b] = tau
        out[b, tau] = tok
    return n_acc, out


def output_distribution(P, Q, draft) -> dict:
    """Exact distribution of the emitted tokens of one round in fp64, for a
    fixed draft block: {tuple(emitted tokens): probability}.  P [k+1, V] and
    Q [k, V] are probability rows (any float dtype)."""
    P = np.asarray(P, dtype=np.float64)
    Q = np.asarray(Q, dtype=np.float64)
    k = len(draft)
    p = [1.0]
    for i in range(1, k + 1):
        x = int(draft[i - 1])
        p.append(min(p[-1] * P[i - 1, x] / Q[i - 1, x], 1.0))
    h, res = [], []
    for i in range(k):
        r = np.maximum(p[i] * P[i] - Q[i], 0.0)
        s = r.sum()
        den = s + 1.0 - p[i]
        h.append(1.0 if den <= 0.0 else s / den)
        res.append(r / s if s > 0.0 else P[i])
    h.append(p[k])
    res.append(P[k])
    dist, survive = {}, 1.0   # survive: probability that every eta above i was 0
    for i in range(k, -1, -1):
        w = survive * h[i]
        survive *= 1.0 - h[i]
        if w == 0.0:
            continue
        for y in range(P.shape[-1]):
            if res[i][y] > 0.0:
                key = tuple(int(t) for t in draft[:i]) + (y,)
                dist[key] = dist.get(key, 0.0) + w * res[i][y]
    return dist
