"""The paper's implementation-agnostic performance model, as a calculator that
can also be fed with measured MI355X times.

Paper Sec. 2 (evaluation metric):
  * throughput multiplier = tau / dt, with tau the average number of tokens a
    round generates and the iteration time multiplier
        dt = (k * t_draft + t_verify) / t_target,
    t_draft / t_target the latency of one draft / target forward pass on one
    token and t_verify that of the target on the k+1 tokens of a round;
  * a forward pass costs max(compute FLOPs, (weight bytes + KV bytes) * HOI)
    FLOP-equivalents (computation and memory access fully overlapped), HOI
    being the hardware operational intensity in FLOPs per byte;
  * hence dt = [k * max(C_d, (N_d + KV_d) HOI) + max((k+1) C_t, (N_t + KV_t) HOI)]
               / max(C_t, (N_t + KV_t) HOI).
Paper Sec. 5 (cost analysis): with U units spent on decoding, drafting with a
multiplier m saves U * (1 - 1/m) units; the draft's training cost is
subtracted from that saving.

On MI355X, HOI = peak dense matrix FLOP/s / HBM bytes/s (2.5 PFLOP/s bf16 or
5.0 PFLOP/s fp8 over 8 TB/s).  `attention_round` applies the model to the
attention of one round alone (no weights), from the same per-sequence shapes
the library's kernels run, so that the modeled dt can be set beside the dt
measured from kernel times (`measured_dt`).
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Sequence

HBM_BYTES_PER_S = 8.0e12
PEAK_FLOPS = {"bf16": 2.5e15, "fp8": 5.0e15, "f32": 157.3e12}


def hoi(peak_flops: float, bytes_per_s: float) -> float:
    """Hardware operational intensity, FLOPs per byte (Sec. 2)."""
    return peak_flops / bytes_per_s


def forward_cost(flops: float, mem_bytes: float, hoi_: float) -> float:
    """max(compute, memory * HOI) in FLOP-equivalents (Sec. 2)."""
    return max(flops, mem_bytes * hoi_)


def iteration_time_multiplier(k: int, c_draft: float, mem_draft: float, c_target: float,
                              mem_target: float, hoi_: float) -> float:
    """dt from per-pass FLOPs and bytes: k draft passes on one token plus one
    target pass on k+1 tokens, relative to one target pass on one token.
    mem_* = weight bytes + KV bytes of one pass; c_target is the FLOPs of the
    target on ONE token (verification does k+1 times that)."""
    t_draft = forward_cost(c_draft, mem_draft, hoi_)
    t_verify = forward_cost((k + 1) * c_target, mem_target, hoi_)
    t_target = forward_cost(c_target, mem_target, hoi_)
    return (k * t_draft + t_verify) / t_target


def measured_dt(k: int, t_draft: float, t_verify: float, t_target: float) -> float:
    """dt from measured latencies (Sec. 2's definition)."""
    return (k * t_draft + t_verify) / t_target


def throughput_multiplier(tau: float, dt: float) -> float:
    return tau / dt


def implied_dt(tau: float, multiplier: float) -> float:
    """The iteration time multiplier a printed throughput multiplier implies
    for a measured tau (Sec. 2: multiplier = tau / dt)."""
    return tau / multiplier


def decode_cost_saved(units: float, multiplier: float) -> float:
    """Decoding cost saved out of `units` by a throughput multiplier (Sec. 5)."""
    return units * (1.0 - 1.0 / multiplier)


def net_saving(units: float, multiplier: float, training_cost: float) -> float:
    return decode_cost_saved(units, multiplier) - training_cost


# ---------------------------------------------------------------------------
# attention of one round on the library's shapes
# ---------------------------------------------------------------------------
@dataclass
class AttentionPass:
    flops: float
    kv_bytes: float


def _attn(keys_per_seq: Sequence[int], rows_per_kv_head: int, Hkv: int, D: int, elem: float):
    """FLOPs (QK^T and PV: 4 per row, key and dim) and K+V bytes of one pass."""
    keys = float(sum(keys_per_seq))
    return AttentionPass(flops=4.0 * rows_per_kv_head * D * Hkv * keys,
                         kv_bytes=2.0 * keys * Hkv * D * elem)


def attention_round(context_lens: Sequence[int], k: int, Hq: int, Hkv: int, D: int, S: int, W: int,
                    kv_elem: float):
    """The attention passes of a round for sequences with contexts L_b: the
    k draft steps (step s: min(L_b + s + 1, S + W) keys, g rows per KV head),
    the verification of k+1 tokens (L_b + k + 1 keys, (k+1) g rows) and the
    target's decode of one token (L_b + 1 keys, g rows).
    Returns (list of k draft passes, verify pass, target pass)."""
    g = Hq // Hkv
    drafts = [_attn([min(L + s + 1, S + W) for L in context_lens], g, Hkv, D, kv_elem)
              for s in range(k)]
    verify = _attn([L + k + 1 for L in context_lens], (k + 1) * g, Hkv, D, kv_elem)
    target = _attn([L + 1 for L in context_lens], g, Hkv, D, kv_elem)
    return drafts, verify, target


def attention_dt(context_lens: Sequence[int], k: int, Hq: int, Hkv: int, D: int, S: int, W: int,
                 kv_elem: float, hoi_: float) -> float:
    """Modeled dt of the attention alone (no weights): every pass costs
    max(FLOPs, KV bytes * HOI); the k draft terms are summed step by step."""
    drafts, v, t = attention_round(context_lens, k, Hq, Hkv, D, S, W, kv_elem)
    cd = sum(forward_cost(d.flops, d.kv_bytes, hoi_) for d in drafts)
    cv = forward_cost(v.flops, v.kv_bytes, hoi_)
    ct = forward_cost(t.flops, t.kv_bytes, hoi_)
    return (cd + cv) / ct
