"""KV cache updates around a speculation round -- oracle (test infrastructure only).

Only the test suite, the package smoke check and the benchmark's CPU-baseline
leg use this module; the HIP library never does.  It states, with plain
per-row loops over host copies of the stored bytes, what the library's cache
update calls must leave in memory:

  * kv_append: the target appends the K/V of the tokens a round verified
    (paper Sec. 2: the target's forward pass on the k+1 tokens of a round)
    at positions n_b .. n_b + T - 1 of each sequence's cache, rounded to the
    storage dtype;
  * draft_append: one draft step stores its token's K/V at its sink row or
    ring slot of the StreamingLLM cache, whose size stays constant (Sec. 3.1),
    keeping the row it overwrites (for a full ring: the evicted position) in a
    spill slot;
  * draft_rollback: after verification accepted n of the k draft tokens, the
    rows written for rejected positions get their old bytes back, so the
    cache is again exactly the one a round of n + 1 steps would leave.

Rounding to storage (the paper fixes none of it; the readings are):
  * bf16: round to nearest, ties to even, from the fp32 value; NaN stays a
    quiet NaN (its sign kept);
  * fp8 (OCP e4m3fn): the fp32 value is divided by the per-head scale in fp32
    (IEEE division), then rounded to the nearest finite e4m3fn value with
    ties to the even code; magnitudes beyond 448 saturate to +-448, +-inf
    too; NaN becomes 0x7F;
  * f32 storage keeps the fp32 value; bf16 input is widened exactly first.
Both rounding functions below pick the nearest representable value by
searching every candidate, independent of any bit manipulation.
"""
from __future__ import annotations

import math
from functools import lru_cache

import numpy as np

FP8_MAX = 448.0


# ---------------------------------------------------------------------------
# value sets of the storage formats
# ---------------------------------------------------------------------------
def e4m3fn_value(code: int) -> float:
    """OCP e4m3fn: sign bit 7, exponent bits 6..3 (bias 7), mantissa bits 2..0;
    exponent 0 is subnormal (2^-6 * m/8); S.1111.111 is NaN; no infinities."""
    s = -1.0 if code & 0x80 else 1.0
    e = (code >> 3) & 0xF
    m = code & 0x7
    if e == 0xF and m == 0x7:
        return math.nan
    if e == 0:
        return s * 2.0 ** -6 * (m / 8.0)
    return s * 2.0 ** (e - 7) * (1.0 + m / 8.0)


@lru_cache(maxsize=1)
def _e4m3_positive():
    """(values, codes) of the non-negative finite e4m3fn codes, ascending."""
    codes = [c for c in range(0x80) if not math.isnan(e4m3fn_value(c))]
    vals = np.array([e4m3fn_value(c) for c in codes])
    order = np.argsort(vals, kind="stable")
    return vals[order], np.array(codes)[order]


def round_e4m3fn(x: float) -> int:
    """Nearest e4m3fn code of a finite or infinite fp32 value (ties to the even
    code, saturating at 448); NaN -> 0x7F."""
    if math.isnan(x):
        return 0x7F
    sign = 0x80 if math.copysign(1.0, x) < 0 else 0x00
    a = abs(x)
    vals, codes = _e4m3_positive()
    if a >= FP8_MAX:
        return sign | int(codes[-1])
    # nearest by exhaustive comparison of distances; ties -> even code
    d = np.abs(vals - a)
    best = d.min()
    cands = [int(c) for c, dd in zip(codes, d) if dd == best]
    if len(cands) > 1:
        cands = [c for c in cands if c % 2 == 0] or cands
    code = cands[0]
    if code == 0:
        return sign  # +0 / -0 keep the sign
    return sign | code


def _bf16_value(bits: int) -> float:
    """Value of a bf16 bit pattern; the pattern just past the largest finite
    value counts as 2^128, the value an unbounded exponent would give."""
    if bits & 0x7FFF == 0x7F80:
        return math.copysign(2.0 ** 128, -1.0 if bits & 0x8000 else 1.0)
    return float(np.uint32(bits << 16).view(np.float32))


def round_bf16_bits(x) -> int:
    """Nearest bfloat16 bit pattern of an fp32 value (ties to an even last
    bit; past the largest finite value by half an ulp or more: infinity),
    found by comparing the two neighbouring bf16 values.  NaN stays a quiet
    NaN with its sign."""
    u = int(np.float32(x).view(np.uint32))
    if math.isnan(float(x)):
        return ((u >> 16) | 0x40) & 0xFFFF
    if math.isinf(float(x)):
        return u >> 16
    lo = u >> 16                    # truncation: same sign, magnitude not larger
    a = abs(float(x))
    v_lo = abs(_bf16_value(lo))
    if a == v_lo:
        return lo
    hi = lo + 1                     # the next bf16 away from zero
    v_hi = abs(_bf16_value(hi))
    dlo, dhi = a - v_lo, v_hi - a
    if dlo < dhi or (dlo == dhi and lo % 2 == 0):
        return lo
    return hi & 0xFFFF


def to_storage(x: np.ndarray, dtype: str, scale: float = 1.0) -> np.ndarray:
    """Round a row of fp32 values to storage bytes: returns float32 (f32),
    uint16 bf16 bits, or uint8 e4m3fn codes."""
    x = np.asarray(x, dtype=np.float32)
    if dtype == "f32":
        return x.copy()
    if dtype == "bf16":
        return np.array([round_bf16_bits(v) for v in x], dtype=np.uint16)
    if dtype == "fp8":
        # fp32 IEEE division; a quotient beyond the fp32 range becomes +-inf,
        # which (like every magnitude of 448 and above) saturates to +-448 below
        with np.errstate(over="ignore"):
            y = (x / np.float32(scale)).astype(np.float32)
        return np.array([round_e4m3fn(float(v)) for v in y], dtype=np.uint8)
    raise ValueError(dtype)


# ---------------------------------------------------------------------------
# cache updates on host copies of the stored bytes
# ---------------------------------------------------------------------------
def kv_append(k_store, v_store, k_new, v_new, positions, dtype, page_size=0, block_table=None,
              k_scale=None, v_scale=None, capacity=None):
    """Write token t of sequence b (t < T) at cache position j = positions[b] + t.

    k_store / v_store: numpy arrays of the stored elements, contiguous
      [B, Hkv, cap, D] or paged [pages, Hkv, page_size, D], dtype float32 (f32),
      uint16 (bf16 bits) or uint8 (fp8 codes); they are updated in place.
    k_new / v_new: float32 [B, T, Hkv, D] (bf16 inputs widened by the caller).
    A position with no storage (j < 0, j beyond the capacity, or a page id
    outside [0, pages)) is skipped.
    """
    B, T, Hkv, D = k_new.shape
    for b in range(B):
        for t in range(T):
            j = int(positions[b]) + t
            if j < 0:
                continue
            if page_size > 0:
                blk = j // page_size
                if blk >= block_table.shape[1]:
                    continue
                page = int(block_table[b, blk])
                if page < 0 or page >= k_store.shape[0]:
                    continue
                idx = (page, slice(None), j % page_size)
            else:
                cap = k_store.shape[2] if capacity is None else capacity
                if j >= cap:
                    continue
                idx = (b, slice(None), j)
            for h in range(Hkv):
                ks = 1.0 if k_scale is None else float(k_scale[h])
                vs = 1.0 if v_scale is None else float(v_scale[h])
                k_store[idx[0], h, idx[2]] = to_storage(k_new[b, t, h], dtype, ks)
                v_store[idx[0], h, idx[2]] = to_storage(v_new[b, t, h], dtype, vs)


def draft_slot(p: int, S: int, W: int, offset: int):
    """Where logical position p lives: ('sink', p) for 0 <= p < S, ('ring', slot)
    with slot = (offset + p - S) mod W, or None (negative p, or no window)."""
    if p < 0:
        return None
    if p < S:
        return ("sink", p)
    if W <= 0:
        return None
    return ("ring", (offset + p - S) % W)


def draft_append(sink_k, sink_v, ring_k, ring_v, k_new, v_new, seq_lens, ring_offset, S, W, dtype,
                 k_scale=None, v_scale=None, spill_k=None, spill_v=None):
    """Store the token at logical position p = m_b - 1 of every sequence
    (m_b = seq_lens[b] >= 1) in its sink row or ring slot.  If a spill area is
    given, the row about to be overwritten is first copied into spill[b] --
    for a full ring (p >= S + W) that is the evicted position p - W.  Stores:
    sink [B, Hkv, S, D], ring [B, Hkv, W, D], spill [B, Hkv, D], all in
    storage representation."""
    B, Hkv, D = k_new.shape
    for b in range(B):
        p = int(seq_lens[b]) - 1
        if p < 0:
            continue
        where = draft_slot(p, S, W, int(ring_offset[b]) % W if W > 0 else 0)
        if where is None:
            continue
        dst_k, dst_v = (sink_k, sink_v) if where[0] == "sink" else (ring_k, ring_v)
        row = where[1]
        for h in range(Hkv):
            ks = 1.0 if k_scale is None else float(k_scale[h])
            vs = 1.0 if v_scale is None else float(v_scale[h])
            if spill_k is not None:
                spill_k[b, h] = dst_k[b, h, row]
                spill_v[b, h] = dst_v[b, h, row]
            dst_k[b, h, row] = to_storage(k_new[b, h], dtype, ks)
            dst_v[b, h, row] = to_storage(v_new[b, h], dtype, vs)


def draft_rollback(sink_k, sink_v, ring_k, ring_v, spill_k, spill_v, base_lens, n_accepted, steps,
                   ring_offset, S, W):
    """Undo the writes of rejected draft steps.  Step s of the round wrote
    logical position base_lens[b] + s (s = 0 .. steps-1) and kept the row it
    overwrote in spill[s, b].  With n accepted draft tokens, steps s > n wrote
    tokens that were rejected: their rows get the spilled bytes back, latest
    step first (so two steps of one round that share a slot unwind in order).
    Afterwards the storage holds exactly what n + 1 steps would have left.
    spill: [steps, B, Hkv, D]."""
    B = spill_k.shape[1]
    for b in range(B):
        n = int(n_accepted[b])
        for s in range(steps - 1, n, -1):
            p = int(base_lens[b]) + s
            where = draft_slot(p, S, W, int(ring_offset[b]) % W if W > 0 else 0)
            if where is None:
                continue
            dst_k, dst_v = (sink_k, sink_v) if where[0] == "sink" else (ring_k, ring_v)
            dst_k[b, :, where[1]] = spill_k[s, b]
            dst_v[b, :, where[1]] = spill_v[s, b]
