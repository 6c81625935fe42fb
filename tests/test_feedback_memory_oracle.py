"""Pins of the feedback-memory oracle (paper Sec. 3.3), CPU only: equal
weights give the plain mean of the layers; a dominant weight selects that
layer exactly; adding a constant to a row of weights changes nothing; the
result is a convex combination (inside the per-element range of the layers);
brute force with explicit sums of exp(w) on tiny inputs; and the mixing
weights of a row are torch's softmax of that row (an independent routine)."""
import math

import numpy as np
import pytest
import torch

from oracle import feedback_memory as FM


def _x(rng, Lp1=3, B=4, d=16):
    return rng.normal(0, 2, size=(Lp1, B, d))


def test_equal_weights_give_the_mean():
    rng = np.random.default_rng(0)
    x = _x(rng)
    m = FM.feedback_memory(x, np.zeros((2, 3)))
    np.testing.assert_allclose(m[0], x.mean(axis=0), rtol=0, atol=1e-15)
    np.testing.assert_allclose(m[1], x.mean(axis=0), rtol=0, atol=1e-15)


def test_dominant_weight_selects_its_layer():
    rng = np.random.default_rng(1)
    x = _x(rng, Lp1=4)
    w = np.array([[-800.0, 0.0, -800.0, -800.0], [3.0, -900.0, -900.0, -900.0]])
    m = FM.feedback_memory(x, w)
    assert np.array_equal(m[0], x[1]) and np.array_equal(m[1], x[0])


def test_shift_invariance_and_convexity():
    rng = np.random.default_rng(2)
    x = _x(rng, Lp1=5)
    w = rng.normal(0, 3, size=(3, 5))
    a = FM.feedback_memory(x, w)
    b = FM.feedback_memory(x, w + np.array([[7.0], [-50.0], [123.0]]))
    np.testing.assert_allclose(a, b, rtol=0, atol=1e-12)
    lo, hi = x.min(axis=0), x.max(axis=0)
    assert np.all(a >= lo - 1e-12) and np.all(a <= hi + 1e-12)


def test_brute_force_and_torch_softmax():
    rng = np.random.default_rng(3)
    x = _x(rng, Lp1=3, B=2, d=5)
    w = rng.normal(0, 1, size=(2, 3))
    m = FM.feedback_memory(x, w)
    for i in range(2):
        den = sum(math.exp(w[i, l]) for l in range(3))
        for b in range(2):
            for e in range(5):
                num = sum(math.exp(w[i, l]) * x[l, b, e] for l in range(3))
                assert abs(m[i, b, e] - num / den) <= 1e-14
        sm = torch.softmax(torch.tensor(w[i], dtype=torch.float64), dim=0).numpy()
        np.testing.assert_allclose(FM.mix_weights(w[i]), sm, rtol=1e-15, atol=1e-16)


def test_large_weights_stay_finite():
    rng = np.random.default_rng(4)
    x = _x(rng)
    a = FM.feedback_memory(x, np.array([[1000.0, 999.0, 998.0]]))
    b = FM.feedback_memory(x, np.array([[2.0, 1.0, 0.0]]))
    assert np.all(np.isfinite(a))
    np.testing.assert_allclose(a, b, rtol=0, atol=1e-13)


# planted mistakes: each must fail one of the pins above
import os  # noqa: E402
import types  # noqa: E402

SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle",
                   "feedback_memory.py")
MUTANTS = {
    "unnormalised": ("return np.array([v / s for v in e])", "return np.array([v for v in e])"),
    "raw_weights": ("e = [math.exp(v - top) for v in w]", "e = [v - top for v in w]"),
    "no_max_shift": ("e = [math.exp(v - top) for v in w]", "e = [math.exp(v) for v in w]"),
    "first_layer_only": ("out[i] += a[l] * x[l]", "out[i] += a[l] * x[0]"),
    "wrong_row": ("a = mix_weights(w[i])", "a = mix_weights(w[0])"),
}
CHECKS = [test_equal_weights_give_the_mean, test_dominant_weight_selects_its_layer,
          test_shift_invariance_and_convexity, test_brute_force_and_torch_softmax,
          test_large_weights_stay_finite]


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(name, monkeypatch):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert old in src
    mod = types.ModuleType("fm_mutant")
    exec(compile(src.replace(old, new), f"<mutant {name}>", "exec"), mod.__dict__)
    monkeypatch.setattr(FM, "feedback_memory", mod.feedback_memory)
    monkeypatch.setattr(FM, "mix_weights", mod.mix_weights)
    caught = False
    for check in CHECKS:
        try:
            check()
        except Exception:
            caught = True
            break
    assert caught, name
