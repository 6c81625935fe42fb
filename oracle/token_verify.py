"""Token verification oracle: modified rejection sampling (test infrastructure only).

Only the test suite, the package smoke check and the benchmark's CPU-baseline
leg use this module; the HIP library never does.  It is a plain per-sequence
statement of the token verification step that follows the target's parallel
verify pass (paper Sec. 1: accepted draft tokens are guaranteed to follow the
target's distribution thanks to a modified rejection sampling scheme; Sec. 6:
the experiments use token verification; Table 1's caption: a round emits
between 1 and k+1 tokens, 0..k of them accepted before the first rejection).
The scheme itself is the published one the paper cites (Leviathan et al. 2023,
Chen et al. 2023), restated here:

  for i = 1 .. k:  accept draft token x_i with probability min(1, p_i(x_i) / q_i(x_i));
                   stop at the first rejection;
  n = number accepted;
  if n < k:  emit one token drawn from norm(max(0, p_{n+1} - q_{n+1}))   (correction)
  else:      emit one token drawn from p_{k+1}                          (bonus)

Precision readings (the paper fixes none of them); the HIP path takes every
decision in the same way, so results are comparable bit for bit:
  * accept test: r_i * q_i(x_i) < p_i(x_i), evaluated in fp64, where the
    product of two fp32 numbers is exact; NaN compares false (reject);
  * a draft token outside [0, V) is rejected;
  * sampling: inverse CDF on integer weights W(x) = floor(w(x) * 2^40), with
    w = clamp(p - q, 0, 1) computed in fp32 (correction) or clamp(p, 0, 1)
    (bonus); NaN counts as 0.  With Z = sum W and U = floor(u * 2^24) clamped
    to [0, 2^24 - 1], the threshold is T = floor(U * Z / 2^24) and the token is
    the smallest x with W(0) + ... + W(x) > T.  Integer sums do not depend on
    the order of summation, and a token of zero weight is never drawn;
  * a correction row with Z = 0 (p <= q everywhere at this resolution) draws
    from p of the same row instead; a row whose p has Z = 0 yields token -1.
"""
from __future__ import annotations

import math

import numpy as np

SHIFT = 40      # fraction bits of a fixed-point sampling weight
U_BITS = 24     # fraction bits taken from a sampling uniform


def weights(p_row, q_row=None) -> np.ndarray:
    """Integer sampling weights of one row: floor(clamp(w, 0, 1) * 2^40), with
    w = p - q rounded to fp32 (correction) or w = p (bonus)."""
    p = np.asarray(p_row, dtype=np.float32)
    if q_row is None:
        w = p.copy()
    else:
        w = np.subtract(p, np.asarray(q_row, dtype=np.float32), dtype=np.float32)
    w = np.where(w > 0, w, np.float32(0.0))   # negatives and NaN -> 0
    w = np.minimum(w, np.float32(1.0))
    # w * 2^40 is exact in fp64; floor of a non-negative value is truncation
    return np.floor(w.astype(np.float64) * float(2 ** SHIFT)).astype(np.int64)


def threshold(u, Z: int) -> int:
    """T = floor(U * Z / 2^24), U = floor(u * 2^24) clamped to [0, 2^24 - 1]."""
    uf = float(np.float32(u))
    if not uf > 0.0:          # u <= 0 or NaN
        U = 0
    elif uf >= 1.0:           # 1, larger values and +inf
        U = 2 ** U_BITS - 1
    else:                     # uf * 2^24 is exact; floor(uf * 2^24) <= 2^24 - 1
        U = int(math.floor(uf * float(2 ** U_BITS)))
    return (U * int(Z)) >> U_BITS     # Python integers: exact


def inverse_cdf(W: np.ndarray, u) -> int:
    """Smallest x with W[0] + ... + W[x] > T, or -1 when all weights are 0."""
    Z = int(W.sum())                  # < 2^60 for V <= 2^20: exact in int64
    if Z == 0:
        return -1
    T = threshold(u, Z)
    C = np.cumsum(W)
    return int(np.searchsorted(C, T, side="right"))


def accept(u, q_x, p_x) -> bool:
    """Accept with probability min(1, p/q): u * q < p with an exact fp64 product."""
    return float(np.float32(u)) * float(np.float32(q_x)) < float(np.float32(p_x))


def verify_tokens(p, q, draft, u_accept, u_sample):
    """Token verification of a batch.

    p         [B, k+1, V] target probabilities (fp32): row i scores the token
              that follows the last accepted token and draft tokens 1..i
    q         [B, k, V]   draft probabilities (fp32) of the k draft tokens
    draft     [B, k]      draft tokens x_1 .. x_k
    u_accept  [B, k]      uniforms of the accept tests
    u_sample  [B]         uniform of the emitted (correction or bonus) token
    Returns (n_accepted [B] int32, tokens [B, k+1] int32): tokens[b, :n] are
    the accepted draft tokens, tokens[b, n] the emitted token, the rest -1.
    """
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
        n = 0
        while n < k:
            x = int(draft[b, n])
            if not (0 <= x < V):
                break
            if not accept(u_accept[b, n], q[b, n, x], p[b, n, x]):
                break
            n += 1
        out[b, :n] = draft[b, :n]
        if n < k:
            tok = inverse_cdf(weights(p[b, n], q[b, n]), u_sample[b])
            if tok < 0:
                tok = inverse_cdf(weights(p[b, n]), u_sample[b])
        else:
            tok = inverse_cdf(weights(p[b, k]), u_sample[b])
        n_acc[b] = n
        out[b, n] = tok
    return n_acc, out
