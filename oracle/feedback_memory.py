"""Feedback-memory mixing -- oracle (test infrastructure only).

Only the test suite, the package smoke check and the benchmark's CPU-baseline
leg use this module; the HIP library never does.  Paper Sec. 3.3: the draft
is a Feedback Transformer whose attention reads memory vectors instead of the
layer's own activations, and the memory vector of a token is a convex mix of
that token's activations after every layer (layer 0 is the embedding):

    m_t   = sum_l exp(w_l)   x_t^l / sum_l exp(w_l)          (one set of weights)
    m_t^i = sum_l exp(w_il)  x_t^l / sum_l exp(w_il)         (one set per draft layer i)

with learnable weights w (a row per draft layer in the per-layer form).  This
states the per-layer form directly, in fp64, from the stored inputs: x of
shape [L+1, B, d] (activations of the step's tokens after each layer),
w of shape [n_out, L+1]; the result has shape [n_out, B, d].  The exponent
is taken after subtracting the row's maximum weight, which changes nothing
mathematically and keeps exp finite.
"""
from __future__ import annotations

import math

import numpy as np


def mix_weights(w_row) -> np.ndarray:
    """exp(w_l) / sum_l exp(w_l) for one row of weights, in fp64."""
    w = [float(v) for v in np.asarray(w_row, dtype=np.float64)]
    top = max(w)
    e = [math.exp(v - top) for v in w]
    s = sum(e)
    return np.array([v / s for v in e])


def feedback_memory(x, w) -> np.ndarray:
    """x [L+1, B, d] (any float dtype, read exactly), w [n_out, L+1] -> fp64 [n_out, B, d]."""
    x = np.asarray(x, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    n_out = w.shape[0]
    Lp1, B, d = x.shape
    assert w.shape[1] == Lp1
    out = np.zeros((n_out, B, d))
    for i in range(n_out):
        a = mix_weights(w[i])
        for l in range(Lp1):
            out[i] += a[l] * x[l]
    return out
