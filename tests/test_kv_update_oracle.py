"""Pins of the KV cache update oracle (CPU only).

The oracle states the cache writes around a round: the target's append of
the verified tokens (paper Sec. 2), the draft's sink/ring write with a spill
of the evicted row, and the rollback of rejected draft steps (Sec. 3.1's
constant-size StreamingLLM cache).  Pinned here by:
  * its rounding functions against torch's own bf16 / float8_e4m3fn
    conversions (an independent implementation), every bf16 and e4m3fn code
    mapping to itself, and hand-computed ties, saturation, subnormals, NaN;
  * kv_append: the logical rows read back through the block table are the
    torch-rounded new values, and every other stored byte is untouched;
  * draft_append against the caller-side tensor copy of the workload module
    (workloads.write_step_token) on unrounded storage;
  * the round-trip law: k draft writes then a rollback to n accepted leave
    exactly the bytes of n + 1 draft writes (for every n, full and filling
    rings, wrap-around, sinks, no window);
and by planted mistakes, each of which must fail one of these checks.
"""
from __future__ import annotations

import math
import os
import types

import numpy as np
import pytest
import torch

from oracle import kv_update as KU
from paper_2504_06419_amd import workloads as W

ORACLE_SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle",
                          "kv_update.py")


def _torch_e4m3(x: np.ndarray) -> np.ndarray:
    t = torch.from_numpy(np.asarray(x, np.float32)).clamp(-448.0, 448.0)
    return t.to(torch.float8_e4m3fn).view(torch.uint8).numpy()


def _torch_bf16(x: np.ndarray) -> np.ndarray:
    return torch.from_numpy(np.asarray(x, np.float32)).to(torch.bfloat16).view(torch.int16).numpy() \
        .astype(np.uint16)


# ---------------------------------------------------------------------------
def check_e4m3(M):
    rng = np.random.default_rng(1)
    x = np.concatenate([rng.normal(0, 60, 5000), rng.normal(0, 0.01, 2000),
                        rng.uniform(-448, 448, 2000)]).astype(np.float32)
    mine = np.array([M.round_e4m3fn(float(v)) for v in x], np.uint8)
    assert np.array_equal(mine, _torch_e4m3(x))
    for code in range(256):
        v = M.e4m3fn_value(code)
        if math.isnan(v):
            assert M.round_e4m3fn(v) == 0x7F
        else:
            assert M.round_e4m3fn(v) == code, code
    hand = [(1.0625, 0x38), (1.1875, 0x3A), (448.0, 0x7E), (449.0, 0x7E), (470.0, 0x7E),
            (1e30, 0x7E), (math.inf, 0x7E), (-math.inf, 0xFE), (-1e30, 0xFE), (2.0 ** -9, 0x01),
            (2.0 ** -10, 0x00), (3 * 2.0 ** -10, 0x02), (-(2.0 ** -11), 0x80), (-0.0, 0x80),
            (0.0, 0x00), (240.0, 0x77), (248.0, 0x78)]
    for v, code in hand:
        assert M.round_e4m3fn(v) == code, (v, hex(M.round_e4m3fn(v)), hex(code))
    assert M.round_e4m3fn(math.nan) == 0x7F


def check_bf16(M):
    rng = np.random.default_rng(2)
    x = np.concatenate([rng.normal(0, 3, 5000), rng.normal(0, 1e-39, 500),
                        np.array([3.3895e38, 3.3896e38, 3.39e38, 3.4e38, -3.4e38, 1e-45, -0.0,
                                  1.00390625, 1.01171875])]).astype(np.float32)
    mine = np.array([M.round_bf16_bits(v) for v in x], np.uint16)
    assert np.array_equal(mine, _torch_bf16(x))
    for bits in range(0, 1 << 16, 7):
        v = np.uint32(bits << 16).view(np.float32)
        got = M.round_bf16_bits(v)
        if np.isnan(v):
            assert got == (bits | 0x40)
        else:
            assert got == bits, hex(bits)
    # ties: 1 + 2^-8 sits between 1 and 1 + 2^-7 -> even (1.0); 1 + 3*2^-8 -> 1 + 2^-6
    assert M.round_bf16_bits(np.float32(1.00390625)) == 0x3F80
    assert M.round_bf16_bits(np.float32(1.01171875)) == 0x3F82


def _paged(seed, dtype, B=5, Hkv=2, D=8, ps=4, T=3):
    rng = np.random.default_rng(seed)
    lens = rng.integers(0, 13, size=B)
    blocks = [(int(n) + T + ps - 1) // ps for n in lens]
    maxb = max(blocks) + 1
    pages = sum(blocks) + 3
    perm = rng.permutation(pages)
    table = np.full((B, maxb), -1, np.int32)
    pos = 0
    for b in range(B):
        table[b, :blocks[b]] = perm[pos:pos + blocks[b]]
        pos += blocks[b]
    npdt = {"f32": np.float32, "bf16": np.uint16, "fp8": np.uint8}[dtype]
    ks = rng.integers(0, 200, size=(pages, Hkv, ps, D)).astype(npdt)
    vs = rng.integers(0, 200, size=(pages, Hkv, ps, D)).astype(npdt)
    kn = rng.normal(0, 3, size=(B, T, Hkv, D)).astype(np.float32)
    vn = rng.normal(0, 3, size=(B, T, Hkv, D)).astype(np.float32)
    sc = (0.5 + rng.random(Hkv)).astype(np.float32)
    return lens, table, ks, vs, kn, vn, sc, ps


def check_kv_append(M):
    for dtype in ("f32", "bf16", "fp8"):
        lens, table, ks, vs, kn, vn, sc, ps = _paged(7, dtype)
        k0, v0 = ks.copy(), vs.copy()
        kw, vw = (sc, sc * 1.5) if dtype == "fp8" else (None, None)
        M.kv_append(ks, vs, kn, vn, lens, dtype, ps, table, kw, vw)
        touched = np.zeros(ks.shape[:1] + ks.shape[2:3], bool)
        B, T, Hkv, D = kn.shape
        for b in range(B):
            for t in range(T):
                j = int(lens[b]) + t
                page, row = int(table[b, j // ps]), j % ps
                touched[page, row] = True
                for h in range(Hkv):
                    for src, dst, s in ((kn, ks, None if kw is None else kw[h]),
                                        (vn, vs, None if vw is None else vw[h])):
                        want = src[b, t, h]
                        if dtype == "bf16":
                            want = _torch_bf16(want)
                        elif dtype == "fp8":
                            want = _torch_e4m3(want / np.float32(s))
                        assert np.array_equal(dst[page, h, row], want), (dtype, b, t, h)
        for a, a0 in ((ks, k0), (vs, v0)):
            assert np.array_equal(a.transpose(0, 2, 1, 3)[~touched], a0.transpose(0, 2, 1, 3)[~touched])
    # positions without storage are skipped: contiguous beyond capacity
    store = np.zeros((2, 1, 4, 2), np.float32)
    M.kv_append(store, store.copy(), np.ones((2, 3, 1, 2), np.float32), np.ones((2, 3, 1, 2), np.float32),
                [2, -5], "f32")
    assert store[0, 0, 2:].sum() == 4 and store[0, 0, :2].sum() == 0 and store[1].sum() == 0


def _draft_state(seed, B, Hkv, D, S, Wn, lo, hi):
    rng = np.random.default_rng(seed)
    base = rng.integers(lo, hi + 1, size=B)
    off = rng.integers(0, max(Wn, 1), size=B)
    sk = rng.normal(size=(B, Hkv, S, D)).astype(np.float32)
    sv = rng.normal(size=(B, Hkv, S, D)).astype(np.float32)
    rk = rng.normal(size=(B, Hkv, Wn, D)).astype(np.float32)
    rv = rng.normal(size=(B, Hkv, Wn, D)).astype(np.float32)
    return rng, base, off, sk, sv, rk, rv


def check_draft_append_matches_tensor_copy(M):
    spec = W.DraftSpec(B=6, Hq=4, Hkv=2, D=8, S=3, W=5, steps=3, ctx_lo=1, ctx_hi=12,
                       kv_dtype="f32", q_dtype="f32")
    inp = W.make_draft_inputs(spec, 11, device="cpu", poison=None)
    sk, sv = inp.sink_k.numpy().copy(), inp.sink_v.numpy().copy()
    rk, rv = inp.ring_k.numpy().copy(), inp.ring_v.numpy().copy()
    for step in range(spec.steps):
        M.draft_append(sk, sv, rk, rv, inp.new_k[step].numpy(), inp.new_v[step].numpy(),
                       inp.seq_lens(step).numpy(), inp.ring_offset.numpy(), spec.S, spec.W, "f32")
        W.write_step_token(inp, step)
        assert np.array_equal(sk, inp.sink_k.numpy()) and np.array_equal(sv, inp.sink_v.numpy())
        assert np.array_equal(rk, inp.ring_k.numpy()) and np.array_equal(rv, inp.ring_v.numpy())


def check_rollback_round_trip(M):
    # (S, W, length range): full rings, filling rings, sinks being written,
    # no window, and windows shorter than the k = 4 steps, where steps of one
    # round share slots (W = 2, 1: two rejected steps share one)
    cases = [(4, 8, 100, 140), (0, 6, 1, 20), (2, 5, 1, 9), (3, 0, 1, 6), (1, 3, 2, 40),
             (1, 2, 3, 30), (0, 1, 1, 10)]
    k = 4
    for ci, (S, Wn, lo, hi) in enumerate(cases):
        B, Hkv, D = 7, 2, 4
        rng, base, off, sk, sv, rk, rv = _draft_state(100 + ci, B, Hkv, D, S, Wn, lo, hi)
        new_k = rng.normal(size=(k, B, Hkv, D)).astype(np.float32)
        new_v = rng.normal(size=(k, B, Hkv, D)).astype(np.float32)
        for n in range(k):
            full = [a.copy() for a in (sk, sv, rk, rv)]
            spk = np.zeros((k, B, Hkv, D), np.float32)
            spv = np.zeros((k, B, Hkv, D), np.float32)
            for s in range(k):
                M.draft_append(*full, new_k[s], new_v[s], base + s + 1, off, S, Wn, "f32",
                               spill_k=spk[s], spill_v=spv[s])
            M.draft_rollback(*full, spk, spv, base, np.full(B, n), k, off, S, Wn)
            part = [a.copy() for a in (sk, sv, rk, rv)]
            for s in range(n + 1):
                M.draft_append(*part, new_k[s], new_v[s], base + s + 1, off, S, Wn, "f32")
            # sinks and ring agree byte for byte, unused rows included
            for a, c in zip(full, part):
                assert np.array_equal(a, c), (ci, n)


CHECKS = [check_e4m3, check_bf16, check_kv_append, check_draft_append_matches_tensor_copy,
          check_rollback_round_trip]


@pytest.mark.parametrize("check", CHECKS, ids=[c.__name__ for c in CHECKS])
def test_oracle_pin(check):
    check(KU)


# ---------------------------------------------------------------------------
MUTANTS = {
    "ties_away_from_zero": ("cands = [c for c in cands if c % 2 == 0] or cands",
                            "cands = [max(cands)]"),
    "no_saturation": ("    if a >= FP8_MAX:\n        return sign | int(codes[-1])\n", ""),
    "scale_multiplied": ("y = (x / np.float32(scale)).astype(np.float32)",
                         "y = (x * np.float32(scale)).astype(np.float32)"),
    "bf16_truncates": ("    if dlo < dhi or (dlo == dhi and lo % 2 == 0):\n        return lo\n",
                       "    if True:\n        return lo\n"),
    "bf16_ties_up": ("dlo == dhi and lo % 2 == 0", "dlo == dhi and lo % 2 == 1"),
    "negative_zero_lost": ("        return sign  # +0 / -0 keep the sign", "        return 0"),
    "append_off_by_one": ("j = int(positions[b]) + t", "j = int(positions[b]) + t + 1"),
    "append_wrong_page_row": ("idx = (page, slice(None), j % page_size)",
                              "idx = (page, slice(None), (j + 1) % page_size)"),
    "slot_sign": ("return (\"ring\", (offset + p - S) % W)", "return (\"ring\", (offset - p + S) % W)"),
    "spill_after_write": ("            if spill_k is not None:\n                spill_k[b, h] = dst_k[b, h, row]\n"
                          "                spill_v[b, h] = dst_v[b, h, row]\n"
                          "            dst_k[b, h, row] = to_storage(k_new[b, h], dtype, ks)\n"
                          "            dst_v[b, h, row] = to_storage(v_new[b, h], dtype, vs)\n",
                          "            dst_k[b, h, row] = to_storage(k_new[b, h], dtype, ks)\n"
                          "            dst_v[b, h, row] = to_storage(v_new[b, h], dtype, vs)\n"
                          "            if spill_k is not None:\n                spill_k[b, h] = dst_k[b, h, row]\n"
                          "                spill_v[b, h] = dst_v[b, h, row]\n"),
    "rollback_keeps_first_rejected": ("for s in range(steps - 1, n, -1):", "for s in range(steps - 1, n + 1, -1):"),
    "rollback_drops_accepted": ("for s in range(steps - 1, n, -1):", "for s in range(steps - 1, n - 1, -1):"),
    "rollback_forward_order": ("for s in range(steps - 1, n, -1):", "for s in range(n + 1, steps):"),
}


def _mutant(name, old, new):
    src = open(ORACLE_SRC).read()
    assert src.count(old) >= 1, f"mutation {name} does not apply"
    mod = types.ModuleType(f"ku_mutant_{name}")
    exec(compile(src.replace(old, new), f"<mutant {name}>", "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(name):
    M = _mutant(name, *MUTANTS[name])
    caught = False
    for check in CHECKS:
        try:
            check(M)
        except Exception:
            caught = True
            break
    assert caught, f"mutant {name} passed every pin"
