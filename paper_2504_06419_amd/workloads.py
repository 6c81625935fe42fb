"""Seeded synthetic workloads for speculative-round attention.

This module only *prepares inputs*: it draws random numbers, rounds them to the
storage dtype, lays them out in the cache formats the library reads (contiguous,
paged with a block table, sink array plus sliding-window ring) and returns the
per-sequence metadata.  It contains none of the attention arithmetic, so both
the HIP path and the CPU oracle can consume the very same bytes.

Shapes follow the large-batch, long and varied context regime in which the
paper argues that loading the KV cache dominates a speculation round (Sec. 1,
Sec. 3.1): the target verifies k+1 tokens per sequence (Sec. 2) and the draft
reads a StreamingLLM sink + sliding-window cache of constant size (Sec. 3.1,
Sec. 4).  The paper's own contexts come from LongCrawl64, which is not
available; i.i.d. N(0, 1) values with the same shapes stand in for them.

Conventions (shared with the library header and the oracle):
  * verify: sequence b holds n_b = L_b + k + 1 keys (context plus the k+1 new
    tokens, already appended); verify query i in [0, k] sees keys [0, n_b-k+i).
  * draft: m_b is the logical length including the query's own token; logical
    position p < S lives in sink row p, position p >= S in ring slot
    (ring_offset_b + p - S) mod W; visible = [0, min(S, m_b)) U
    [max(S, m_b - W), m_b).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import List, Optional

import torch

MASTER_SEED = 250406419

FP8_MAX = 448.0  # largest finite OCP e4m3fn value

DTYPES = {"f32": torch.float32, "bf16": torch.bfloat16, "fp8": torch.float8_e4m3fn}


# ----------------------------------------------------------------------------
# Workload descriptions
# ----------------------------------------------------------------------------
@dataclass
class VerifySpec:
    B: int
    Hq: int
    Hkv: int
    D: int
    k: int
    ctx_lo: int            # context length L_b range (inclusive); lo == hi is uniform
    ctx_hi: int
    kv_dtype: str = "bf16"
    q_dtype: str = "bf16"
    page_size: int = 0     # 0 = contiguous [B, Hkv, cap, D]
    spare_pages: int = 0   # extra physical pages that no sequence uses (poisoned)
    log_uniform: bool = True


@dataclass
class DraftSpec:
    B: int
    Hq: int
    Hkv: int
    D: int
    S: int                 # sink tokens
    W: int                 # window (ring slots)
    steps: int             # sequential draft steps (k)
    ctx_lo: int            # logical length before the first draft step
    ctx_hi: int
    kv_dtype: str = "bf16"
    q_dtype: str = "bf16"
    log_uniform: bool = True


@dataclass
class TokenSpec:
    """Token verification after the verify pass: per sequence, the target's
    k+1 next-token distributions and the draft's k distributions over a
    vocabulary of V tokens.  Target logits are sigma * N(0,1); draft logits
    add eps * N(0,1) of mismatch (sigma 4, eps 0.55 accept about 4 of 5 draft
    tokens, i.e. about 3.4 tokens per round at k = 4, the average generation
    length the paper reports for SPIRe at L = 512)."""
    B: int
    k: int
    V: int
    sigma: float = 4.0
    eps: float = 0.55


@dataclass
class KvUpdateSpec:
    """Cache writes of one round: k draft steps each store their token in the
    sink/ring cache (keeping the overwritten row in a spill slot), the target
    appends the k+1 verified tokens to its paged cache, and the draft writes
    of rejected steps are rolled back."""
    B: int
    Hkv: int
    D: int
    k: int
    S: int
    W: int
    ctx_lo: int
    ctx_hi: int
    kv_dtype: str = "fp8"
    page_size: int = 16
    accept: float = 0.8     # per-token acceptance of the seeded accepted counts


@dataclass
class FeedbackSpec:
    """Feedback-memory mixing of one draft step: the activations of the B
    tokens after each of `layers` layers (embedding included) are mixed into
    n_out memory vectors, one per draft layer."""
    B: int
    d: int
    layers: int
    n_out: int
    x_dtype: str = "bf16"
    m_dtype: str = "bf16"


def named_workloads():
    """The workloads the library is validated and measured on."""
    return {
        "tiny_f32": dict(
            verify=VerifySpec(B=4, Hq=8, Hkv=2, D=64, k=4, ctx_lo=512, ctx_hi=512,
                              kv_dtype="f32", q_dtype="f32"),
            draft=DraftSpec(B=4, Hq=8, Hkv=2, D=64, S=4, W=128, steps=4,
                            ctx_lo=512, ctx_hi=512, kv_dtype="f32", q_dtype="f32"),
        ),
        "verify_bf16_B64_L8192": dict(
            verify=VerifySpec(B=64, Hq=32, Hkv=8, D=128, k=4, ctx_lo=8192, ctx_hi=8192)),
        "draft_bf16_B64_S4_W2048": dict(
            draft=DraftSpec(B=64, Hq=32, Hkv=8, D=128, S=4, W=2048, steps=4,
                            ctx_lo=32768, ctx_hi=32768)),
        "verify_varlen_paged_bf16_B256": dict(
            verify=VerifySpec(B=256, Hq=32, Hkv=8, D=128, k=4, ctx_lo=512, ctx_hi=65536,
                              page_size=16, spare_pages=64)),
        "round_fp8_B512_k8": dict(
            draft=DraftSpec(B=512, Hq=64, Hkv=8, D=128, S=4, W=4096, steps=8,
                            ctx_lo=2048, ctx_hi=65536, kv_dtype="fp8"),
            verify=VerifySpec(B=512, Hq=64, Hkv=8, D=128, k=8, ctx_lo=2048, ctx_hi=65536,
                              kv_dtype="fp8", page_size=16, spare_pages=64)),
        # the vocabulary of Llama 3 (the model the paper extrapolates to, Sec. 4.3)
        "token_verify_B256_k4_V128256": dict(token=TokenSpec(B=256, k=4, V=128256)),
        "token_verify_B512_k8_V128256": dict(token=TokenSpec(B=512, k=8, V=128256)),
        "kv_update_round_fp8_B512_k8": dict(kvupd=KvUpdateSpec(B=512, Hkv=8, D=128, k=8, S=4, W=4096,
                                                                ctx_lo=2048, ctx_hi=65536)),
        # SPIRe's two-layer draft (embedding + 2 layers mixed into 2 memory
        # vectors) at the width of Llama 3 70B, the model of Sec. 4.3
        "feedback_memory_B512_d8192": dict(fm=FeedbackSpec(B=512, d=8192, layers=3, n_out=2)),
        # one GPU's share of the fp8 round's verification under tensor
        # parallelism over the 8 KV heads: 8 query heads reading 1 KV head
        "verify_tp8shard_fp8_B512_k8": dict(
            verify=VerifySpec(B=512, Hq=8, Hkv=1, D=128, k=8, ctx_lo=2048, ctx_hi=65536,
                              kv_dtype="fp8", page_size=16, spare_pages=64)),
        # block verification (the alternative to token verification, Sec. 6)
        # on inputs drawn like the token verification workloads'
        "block_verify_B256_k4_V128256": dict(block=TokenSpec(B=256, k=4, V=128256)),
        "block_verify_B512_k8_V128256": dict(block=TokenSpec(B=512, k=8, V=128256)),
    }


WORKLOAD_INDEX = {name: i for i, name in enumerate(named_workloads())}


# ----------------------------------------------------------------------------
# Random draws
# ----------------------------------------------------------------------------
def _cpu_gen(seed: int) -> torch.Generator:
    g = torch.Generator(device="cpu")
    g.manual_seed(int(seed))
    return g


def _dev_gen(seed: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    return g


def draw_lengths(gen: torch.Generator, B: int, lo: int, hi: int, log_uniform: bool) -> List[int]:
    """L = floor(exp(U(ln lo, ln hi))) clamped to [lo, hi]; uniform L when lo == hi."""
    if lo == hi:
        return [lo] * B
    u = torch.rand(B, generator=gen, dtype=torch.float64)
    if log_uniform:
        x = torch.exp(math.log(lo) + u * (math.log(hi) - math.log(lo)))
    else:
        x = lo + u * (hi - lo)
    return [int(min(max(math.floor(v), lo), hi)) for v in x.tolist()]


def _randn(shape, gen, device) -> torch.Tensor:
    return torch.randn(*shape, generator=gen, device=device, dtype=torch.float32)


def quantize(x: torch.Tensor, dtype: str, head_dim_axis: int = 1,
             scale: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Round fp32 values to the storage dtype (bf16: RNE; fp8: x / scale[h],
    saturated to +-448, then RNE), `scale` indexed along `head_dim_axis`."""
    if dtype == "f32":
        return x.contiguous()
    if dtype == "bf16":
        return x.to(torch.bfloat16)
    if dtype == "fp8":
        shape = [1] * x.dim()
        shape[head_dim_axis] = -1
        y = (x / scale.to(x.device).view(shape)).clamp_(-FP8_MAX, FP8_MAX)
        return y.to(torch.float8_e4m3fn)
    raise ValueError(dtype)


def draw_fp8_scales(gen: torch.Generator, Hkv: int):
    """Per-KV-head dequantisation scales, one for K and one for V: amax/448
    with amax in [5, 6) so that N(0,1) data almost never saturates and every
    head has a different scale."""
    ks = (5.0 + torch.rand(Hkv, generator=gen, dtype=torch.float64)) / FP8_MAX
    vs = (5.0 + torch.rand(Hkv, generator=gen, dtype=torch.float64)) / FP8_MAX
    return ks.to(torch.float32), vs.to(torch.float32)


def poison_value(dtype: str, kind: str = "nan"):
    """A value written into storage that no visible key may read."""
    if kind == "nan":
        return float("nan")
    return 1.0e4 if dtype != "fp8" else FP8_MAX


# ----------------------------------------------------------------------------
# Verify inputs
# ----------------------------------------------------------------------------
@dataclass
class VerifyInputs:
    spec: VerifySpec
    q: torch.Tensor                      # [B, k+1, Hq, D]
    k_cache: torch.Tensor                # contiguous [B, Hkv, cap, D] or paged [P, Hkv, ps, D]
    v_cache: torch.Tensor
    kv_lens: torch.Tensor                # int32 [B] (n_b)
    context_lens: List[int]              # L_b
    block_table: Optional[torch.Tensor]  # int32 [B, max_blocks] or None
    k_scale: Optional[torch.Tensor]      # fp32 [Hkv] (fp8 only)
    v_scale: Optional[torch.Tensor]
    sm_scale: float
    capacity: int                        # tokens per sequence addressable
    logical_k: Optional[torch.Tensor] = None  # fp32 [B, Hkv, nmax, D] (tiny cases only)
    logical_v: Optional[torch.Tensor] = None

    @property
    def page_size(self) -> int:
        return self.spec.page_size

    def kv_bytes(self) -> int:
        es = self.k_cache.element_size()
        return 2 * int(sum(self.kv_lens.tolist())) * self.spec.Hkv * self.spec.D * es


def make_verify_inputs(spec: VerifySpec, seed: int, device="cpu", keep_logical: bool = False,
                       poison: Optional[str] = "nan", max_blocks_slack: int = 0) -> VerifyInputs:
    """Build one verify batch.  Draw order: lengths, scales, page permutation,
    Q, K, V (then poison of unused storage)."""
    meta = _cpu_gen(seed)
    dgen = _dev_gen(seed + 7919, device)
    B, Hq, Hkv, D, k = spec.B, spec.Hq, spec.Hkv, spec.D, spec.k
    ctx = draw_lengths(meta, B, spec.ctx_lo, spec.ctx_hi, spec.log_uniform)
    n = [L + k + 1 for L in ctx]
    nmax = max(n)
    ps = spec.page_size
    k_scale = v_scale = None

    if spec.kv_dtype == "fp8":
        k_scale, v_scale = draw_fp8_scales(meta, Hkv)

    if ps > 0:
        blocks = [(x + ps - 1) // ps for x in n]
        max_blocks = max(blocks) + max_blocks_slack
        total = sum(blocks)
        phys = total + spec.spare_pages
        perm = torch.randperm(phys, generator=meta).tolist()
        perm_t = torch.tensor(perm, dtype=torch.int32)
        table = torch.full((B, max_blocks), -1, dtype=torch.int32)
        pos = 0
        for b in range(B):
            table[b, : blocks[b]] = perm_t[pos: pos + blocks[b]]
            pos += blocks[b]
        store_shape = (phys, Hkv, ps, D)
        capacity = max_blocks * ps
    else:
        table = None
        capacity = nmax
        store_shape = (B, Hkv, capacity, D)

    q = quantize(_randn((B, k + 1, Hq, D), dgen, device), spec.q_dtype)

    logical_k = logical_v = None
    if keep_logical:
        # draw per-sequence logical K/V first, then scatter into storage
        lk = _randn((B, Hkv, nmax, D), dgen, device)
        lv = _randn((B, Hkv, nmax, D), dgen, device)
        kq = quantize(lk, spec.kv_dtype, 1, k_scale)
        vq = quantize(lv, spec.kv_dtype, 1, v_scale)
        k_cache = torch.zeros(store_shape, dtype=DTYPES[spec.kv_dtype], device=device)
        v_cache = torch.zeros(store_shape, dtype=DTYPES[spec.kv_dtype], device=device)
        _fill_poison(k_cache, spec.kv_dtype, poison)
        _fill_poison(v_cache, spec.kv_dtype, poison)
        for b in range(B):
            if ps > 0:
                for j in range((n[b] + ps - 1) // ps):
                    lo, hi = j * ps, min(n[b], (j + 1) * ps)
                    p = int(table[b, j])
                    k_cache[p, :, : hi - lo] = kq[b, :, lo:hi]
                    v_cache[p, :, : hi - lo] = vq[b, :, lo:hi]
            else:
                k_cache[b, :, : n[b]] = kq[b, :, : n[b]]
                v_cache[b, :, : n[b]] = vq[b, :, : n[b]]
        logical_k, logical_v = kq, vq
    else:
        k_cache = _fill_random(store_shape, spec.kv_dtype, dgen, device, k_scale, head_axis=1)
        v_cache = _fill_random(store_shape, spec.kv_dtype, dgen, device, v_scale, head_axis=1)
        if poison:
            _poison_unused_verify(k_cache, v_cache, n, table, ps, spec.kv_dtype, poison)

    kv_lens = torch.tensor(n, dtype=torch.int32)
    return VerifyInputs(spec=spec, q=q, k_cache=k_cache, v_cache=v_cache, kv_lens=kv_lens.to(device),
                        context_lens=ctx, block_table=None if table is None else table.to(device),
                        k_scale=None if k_scale is None else k_scale.to(device),
                        v_scale=None if v_scale is None else v_scale.to(device),
                        sm_scale=1.0 / math.sqrt(D), capacity=capacity,
                        logical_k=logical_k, logical_v=logical_v)


def _fill_random(shape, dtype, gen, device, scale, head_axis, chunk_rows=1 << 26):
    """N(0,1) storage, generated in chunks along dim 0 to bound fp32 temporaries."""
    out = torch.empty(shape, dtype=DTYPES[dtype], device=device)
    per = max(1, int(chunk_rows // max(1, math.prod(shape[1:]))))
    for s in range(0, shape[0], per):
        e = min(shape[0], s + per)
        x = _randn((e - s,) + tuple(shape[1:]), gen, device)
        out[s:e] = quantize(x, dtype, head_axis, scale)
    return out


def _fill_poison(t: torch.Tensor, dtype: str, kind: Optional[str]):
    if kind is None:
        return
    val = poison_value(dtype, kind)
    if dtype == "fp8":
        t.view(torch.uint8).fill_(0x7F if kind == "nan" else 0x7E)
    else:
        t.fill_(val)


def _fill_poison_rows(t: torch.Tensor, rows: torch.Tensor, dtype: str, kind: Optional[str]):
    """Poison rows `rows` of dim 1 of a [H, rows, D] tensor."""
    if kind is None:
        return
    if dtype == "fp8":
        t.view(torch.uint8)[:, rows] = 0x7F if kind == "nan" else 0x7E
    else:
        t[:, rows] = poison_value(dtype, kind)


def _poison_unused_verify(kc, vc, n, table, ps, dtype, kind):
    """Write the poison value into every storage row no sequence exposes."""
    if ps > 0:
        used = torch.zeros(kc.shape[0], dtype=torch.bool)
        tbl = table.cpu()
        for b, nb in enumerate(n):
            nblk = (nb + ps - 1) // ps
            if nblk == 0:
                continue
            ids = tbl[b, :nblk].long()
            used[ids] = True
            last = int(tbl[b, nblk - 1])
            tail = nb - (nblk - 1) * ps
            if tail < ps:
                _fill_poison(kc[last, :, tail:], dtype, kind)
                _fill_poison(vc[last, :, tail:], dtype, kind)
        spare = (~used).nonzero().flatten().to(kc.device)
        if spare.numel():
            if dtype == "fp8":
                kc.view(torch.uint8)[spare] = 0x7F if kind == "nan" else 0x7E
                vc.view(torch.uint8)[spare] = 0x7F if kind == "nan" else 0x7E
            else:
                kc[spare] = poison_value(dtype, kind)
                vc[spare] = poison_value(dtype, kind)
    else:
        for b, nb in enumerate(n):
            if nb < kc.shape[2]:
                _fill_poison(kc[b, :, nb:], dtype, kind)
                _fill_poison(vc[b, :, nb:], dtype, kind)


# ----------------------------------------------------------------------------
# Draft inputs
# ----------------------------------------------------------------------------
@dataclass
class DraftInputs:
    spec: DraftSpec
    q: torch.Tensor                   # [steps, B, Hq, D]
    sink_k: torch.Tensor              # [B, Hkv, S, D]
    sink_v: torch.Tensor
    ring_k: torch.Tensor              # [B, Hkv, W, D]
    ring_v: torch.Tensor
    new_k: torch.Tensor               # [steps, B, Hkv, D]: K/V of the token each step appends
    new_v: torch.Tensor
    base_lens: List[int]              # logical length before step 0 (L_b)
    ring_offset: torch.Tensor         # int32 [B]
    k_scale: Optional[torch.Tensor]
    v_scale: Optional[torch.Tensor]
    sm_scale: float
    logical_k: Optional[torch.Tensor] = None  # [B, Hkv, L+steps, D] in storage dtype (tiny)
    logical_v: Optional[torch.Tensor] = None

    def seq_lens(self, step: int) -> torch.Tensor:
        """m_b at draft step `step`: the step's own token is the last visible one."""
        return torch.tensor([L + step + 1 for L in self.base_lens], dtype=torch.int32,
                            device=self.q.device)


def ring_slot(offset: int, p: int, S: int, W: int) -> int:
    return (offset + p - S) % W


def make_draft_inputs(spec: DraftSpec, seed: int, device="cpu", keep_logical: bool = False,
                      poison: Optional[str] = "nan") -> DraftInputs:
    """Build a draft cache holding the first L_b logical positions of each
    sequence (sinks + the most recent W positions) and the K/V of the tokens the
    `steps` draft steps append.  Draw order: lengths, ring offsets, scales, Q,
    sink K/V, ring K/V, new-token K/V."""
    meta = _cpu_gen(seed)
    dgen = _dev_gen(seed + 104729, device)
    B, Hq, Hkv, D, S, W = spec.B, spec.Hq, spec.Hkv, spec.D, spec.S, spec.W
    base = draw_lengths(meta, B, spec.ctx_lo, spec.ctx_hi, spec.log_uniform)
    offs = (torch.randint(0, max(W, 1), (B,), generator=meta, dtype=torch.int64)
            if W > 0 else torch.zeros(B, dtype=torch.int64))
    k_scale = v_scale = None
    if spec.kv_dtype == "fp8":
        k_scale, v_scale = draw_fp8_scales(meta, Hkv)
    q = quantize(_randn((spec.steps, B, Hq, D), dgen, device), spec.q_dtype)
    logical_k = logical_v = None
    if keep_logical:
        nmax = max(base) + spec.steps
        lk = quantize(_randn((B, Hkv, nmax, D), dgen, device), spec.kv_dtype, 1, k_scale)
        lv = quantize(_randn((B, Hkv, nmax, D), dgen, device), spec.kv_dtype, 1, v_scale)
        sink_k = torch.zeros((B, Hkv, S, D), dtype=DTYPES[spec.kv_dtype], device=device)
        sink_v = torch.zeros_like(sink_k)
        ring_k = torch.zeros((B, Hkv, W, D), dtype=DTYPES[spec.kv_dtype], device=device)
        ring_v = torch.zeros_like(ring_k)
        for t in (sink_k, sink_v, ring_k, ring_v):
            _fill_poison(t, spec.kv_dtype, poison)
        for b in range(B):
            L = base[b]
            for p in range(min(S, L)):
                sink_k[b, :, p] = lk[b, :, p]
                sink_v[b, :, p] = lv[b, :, p]
            for p in range(max(S, L - W), L):
                s = ring_slot(int(offs[b]), p, S, W)
                ring_k[b, :, s] = lk[b, :, p]
                ring_v[b, :, s] = lv[b, :, p]
        new_k = torch.stack([torch.stack([lk[b, :, base[b] + s] for b in range(B)])
                             for s in range(spec.steps)])
        new_v = torch.stack([torch.stack([lv[b, :, base[b] + s] for b in range(B)])
                             for s in range(spec.steps)])
        logical_k, logical_v = lk, lv
    else:
        sink_k = _fill_random((B, Hkv, S, D), spec.kv_dtype, dgen, device, k_scale, 1)
        sink_v = _fill_random((B, Hkv, S, D), spec.kv_dtype, dgen, device, v_scale, 1)
        ring_k = _fill_random((B, Hkv, W, D), spec.kv_dtype, dgen, device, k_scale, 1)
        ring_v = _fill_random((B, Hkv, W, D), spec.kv_dtype, dgen, device, v_scale, 1)
        new_k = _fill_random((spec.steps, B, Hkv, D), spec.kv_dtype, dgen, device, k_scale, 2)
        new_v = _fill_random((spec.steps, B, Hkv, D), spec.kv_dtype, dgen, device, v_scale, 2)
        if poison:
            for b in range(B):
                L = base[b]
                if L < S:
                    _fill_poison(sink_k[b, :, L:], spec.kv_dtype, poison)
                    _fill_poison(sink_v[b, :, L:], spec.kv_dtype, poison)
                nvalid = max(0, L - S)
                if nvalid < W:  # slots never written so far
                    slots = (torch.arange(nvalid, W) + int(offs[b])) % W
                    slots = slots.to(ring_k.device)
                    _fill_poison_rows(ring_k[b], slots, spec.kv_dtype, poison)
                    _fill_poison_rows(ring_v[b], slots, spec.kv_dtype, poison)
    return DraftInputs(spec=spec, q=q, sink_k=sink_k, sink_v=sink_v, ring_k=ring_k, ring_v=ring_v,
                       new_k=new_k, new_v=new_v, base_lens=base,
                       ring_offset=offs.to(torch.int32).to(device),
                       k_scale=None if k_scale is None else k_scale.to(device),
                       v_scale=None if v_scale is None else v_scale.to(device),
                       sm_scale=1.0 / math.sqrt(D), logical_k=logical_k, logical_v=logical_v)


def append_token_slots(inp: DraftInputs, step: int):
    """Where draft step `step` writes its own token: (is_sink, row) per sequence.
    Logical position p = L_b + step."""
    S, W = inp.spec.S, inp.spec.W
    out = []
    for b, L in enumerate(inp.base_lens):
        p = L + step
        if p < S:
            out.append((True, p))
        elif W > 0:
            out.append((False, ring_slot(int(inp.ring_offset[b]), p, S, W)))
        else:
            out.append((False, None))   # no window: the token is not kept
    return out


def write_step_token(inp: DraftInputs, step: int):
    """Caller-side cache update before draft step `step`: store the step's own
    K/V at its sink row or ring slot (plain tensor copies)."""
    slots = append_token_slots(inp, step)
    dev = inp.ring_k.device
    ring_b = [b for b, (is_sink, row) in enumerate(slots) if not is_sink and row is not None]
    if ring_b:
        bi = torch.tensor(ring_b, dtype=torch.long, device=dev)
        si = torch.tensor([slots[b][1] for b in ring_b], dtype=torch.long, device=dev)
        inp.ring_k[bi, :, si] = inp.new_k[step][bi]
        inp.ring_v[bi, :, si] = inp.new_v[step][bi]
    for b, (is_sink, row) in enumerate(slots):
        if is_sink:
            inp.sink_k[b, :, row] = inp.new_k[step, b]
            inp.sink_v[b, :, row] = inp.new_v[step, b]


# ----------------------------------------------------------------------------
# Token verification inputs
# ----------------------------------------------------------------------------
@dataclass
class TokenInputs:
    spec: TokenSpec
    p: torch.Tensor          # fp32 [B, k+1, V] target probabilities
    q: torch.Tensor          # fp32 [B, k, V]   draft probabilities
    draft: torch.Tensor      # int32 [B, k]     draft tokens, x_i drawn from q_i
    u_accept: torch.Tensor   # fp32 [B, k]      uniforms of the accept tests
    u_sample: torch.Tensor   # fp32 [B]         uniform of the emitted token


def make_token_inputs(spec: TokenSpec, seed: int, device="cpu", chunk_rows: int = 256) -> TokenInputs:
    """Seeded distributions, draft tokens and uniforms.  Draw order: target
    logits, draft-logit noise, draft tokens, accept uniforms, sample uniforms.
    The softmax here only turns synthetic logits into the probability rows the
    verification step consumes."""
    gen = _dev_gen(seed + 15485863, device)
    B, k, V = spec.B, spec.k, spec.V
    p = torch.empty((B, k + 1, V), dtype=torch.float32, device=device)
    q = torch.empty((B, k, V), dtype=torch.float32, device=device)
    draft = torch.empty((B, k), dtype=torch.int32, device=device)
    per = max(1, chunk_rows // (k + 1))
    for s in range(0, B, per):
        e = min(B, s + per)
        zt = spec.sigma * _randn((e - s, k + 1, V), gen, device)
        p[s:e] = torch.softmax(zt, dim=-1)
        if k > 0:
            zd = zt[:, :k] + spec.eps * _randn((e - s, k, V), gen, device)
            q[s:e] = torch.softmax(zd, dim=-1)
            x = torch.multinomial(q[s:e].reshape(-1, V), 1, generator=gen)
            draft[s:e] = x.view(e - s, k).to(torch.int32)
    u_accept = torch.rand((B, k), generator=gen, device=device, dtype=torch.float32)
    u_sample = torch.rand((B,), generator=gen, device=device, dtype=torch.float32)
    return TokenInputs(spec=spec, p=p, q=q, draft=draft, u_accept=u_accept, u_sample=u_sample)


# ----------------------------------------------------------------------------
# Cache update inputs
# ----------------------------------------------------------------------------
@dataclass
class KvUpdateInputs:
    spec: KvUpdateSpec
    base_lens: torch.Tensor     # int32 [B]: L_b, the context before the round
    k_cache: torch.Tensor       # paged [pages, Hkv, ps, D]: only the pages the append touches
    v_cache: torch.Tensor
    block_table: torch.Tensor   # int32 [B, max_blocks] (-1 where no page is mapped)
    new_k: torch.Tensor         # fp32 [B, k+1, Hkv, D]: the verified tokens' K/V
    new_v: torch.Tensor
    sink_k: torch.Tensor        # [B, Hkv, S, D]
    sink_v: torch.Tensor
    ring_k: torch.Tensor        # [B, Hkv, W, D]
    ring_v: torch.Tensor
    ring_offset: torch.Tensor   # int32 [B]
    draft_k: torch.Tensor       # fp32 [k, B, Hkv, D]: the draft steps' K/V
    draft_v: torch.Tensor
    n_accepted: torch.Tensor    # int32 [B]
    k_scale: Optional[torch.Tensor]
    v_scale: Optional[torch.Tensor]


def make_kvupdate_inputs(spec: KvUpdateSpec, seed: int, device="cpu") -> KvUpdateInputs:
    """Seeded state of one round's cache writes.  Draw order: context lengths,
    ring offsets, scales, page permutation, accepted counts, then (on the
    device) stored bytes and the new K/V.  Accepted counts follow
    P(n >= i) = accept^i, truncated at k.  Only the pages holding positions
    L_b .. L_b + k are mapped, so the target storage stays small while the
    positions have the workload's lengths."""
    meta = _cpu_gen(seed)
    dgen = _dev_gen(seed + 32452843, device)
    B, Hkv, D, k, S, Wn, ps = spec.B, spec.Hkv, spec.D, spec.k, spec.S, spec.W, spec.page_size
    base = draw_lengths(meta, B, spec.ctx_lo, spec.ctx_hi, True)
    offs = torch.randint(0, max(Wn, 1), (B,), generator=meta, dtype=torch.int64)
    k_scale = v_scale = None
    if spec.kv_dtype == "fp8":
        k_scale, v_scale = draw_fp8_scales(meta, Hkv)
    max_blocks = (max(base) + k + 1 + ps - 1) // ps + 1
    table = torch.full((B, max_blocks), -1, dtype=torch.int32)
    need = [list(range(L // ps, (L + k) // ps + 1)) for L in base]
    pages = sum(len(x) for x in need)
    perm = torch.randperm(pages, generator=meta)
    pos = 0
    for b in range(B):
        for blk in need[b]:
            table[b, blk] = int(perm[pos])
            pos += 1
    u = torch.rand((B, k), generator=meta, dtype=torch.float64)
    n_acc = torch.zeros(B, dtype=torch.int32)
    for b in range(B):
        n = 0
        while n < k and float(u[b, n]) < spec.accept:
            n += 1
        n_acc[b] = n
    kc = _fill_random((pages, Hkv, ps, D), spec.kv_dtype, dgen, device, k_scale, 1)
    vc = _fill_random((pages, Hkv, ps, D), spec.kv_dtype, dgen, device, v_scale, 1)
    sink_k = _fill_random((B, Hkv, S, D), spec.kv_dtype, dgen, device, k_scale, 1)
    sink_v = _fill_random((B, Hkv, S, D), spec.kv_dtype, dgen, device, v_scale, 1)
    ring_k = _fill_random((B, Hkv, Wn, D), spec.kv_dtype, dgen, device, k_scale, 1)
    ring_v = _fill_random((B, Hkv, Wn, D), spec.kv_dtype, dgen, device, v_scale, 1)
    new_k = _randn((B, k + 1, Hkv, D), dgen, device)
    new_v = _randn((B, k + 1, Hkv, D), dgen, device)
    draft_k = _randn((k, B, Hkv, D), dgen, device)
    draft_v = _randn((k, B, Hkv, D), dgen, device)
    dev = lambda t: None if t is None else t.to(device)
    return KvUpdateInputs(spec=spec, base_lens=torch.tensor(base, dtype=torch.int32, device=device),
                          k_cache=kc, v_cache=vc, block_table=table.to(device), new_k=new_k,
                          new_v=new_v, sink_k=sink_k, sink_v=sink_v, ring_k=ring_k, ring_v=ring_v,
                          ring_offset=offs.to(torch.int32).to(device), draft_k=draft_k,
                          draft_v=draft_v, n_accepted=n_acc.to(device), k_scale=dev(k_scale),
                          v_scale=dev(v_scale))


# ----------------------------------------------------------------------------
# Feedback-memory inputs
# ----------------------------------------------------------------------------
@dataclass
class FeedbackInputs:
    spec: FeedbackSpec
    x: torch.Tensor   # [layers, B, d]
    w: torch.Tensor   # fp32 [n_out, layers]


def make_feedback_inputs(spec: FeedbackSpec, seed: int, device="cpu") -> FeedbackInputs:
    """Activations N(0, 1) per layer, weights N(0, 1).  Draw order: weights, activations."""
    gen = _dev_gen(seed + 49979687, device)
    w = _randn((spec.n_out, spec.layers), gen, device)
    x = quantize(_randn((spec.layers, spec.B, spec.d), gen, device), spec.x_dtype)
    return FeedbackInputs(spec=spec, x=x, w=w)
