#!/usr/bin/env python3
"""Benchmark of speculative-round attention on one MI355X.

A step is one pass of the hot path over one synthetic batch already resident
in HBM:
  * verify workloads: verify partial attention -> combine (a separate plan
    launch first where the LDS-staged or generic kernel serves the call);
  * draft workloads:  the k sequential draft-step attention calls;
  * the fp8 round:    k draft-step calls, then the verify call.
The default workload is the variable-length paged bf16 verify batch (B=256,
contexts log-uniform in [512, 65536], k=4, 32 query / 8 KV heads, head dim
128, 16-token pages in shuffled physical order).

Prints ONE JSON line: value = algorithmic HBM bytes per step / time per step
(GB/s), where the time per step is the median over the K timed steps, each
run between two events on the launch stream after a 512 MiB scratch write
that evicts the caches (so every step streams its K/V from HBM); the same
steps back to back with warm caches are reported beside it.  Also: verified
tokens/s, the roofline of the dominant kernel (its average duration from
events of the caller recorded around each of its launches on the launch
stream), the CPU oracle timed on a bounded sample of the same batch, the HBM
read rate of a plain streaming-read kernel over 4 GiB (the practical ceiling
next to 8 TB/s) and, for the default workload, a `round` object: the fp8
speculation round (8 draft steps then the verification of 9 tokens per
sequence) with its time per round, verified tokens/s per round, the roofline
fractions of its draft and verify kernels and the paper's iteration-time
multiplier dt measured against its model.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_2504_06419_amd import spire  # noqa: E402
from paper_2504_06419_amd import workloads as W  # noqa: E402

METRIC = "KV-attention HBM GB/s (% of peak) + verified tokens/s per round, 1 MI355X"
HBM_PEAK_GBS = 8000.0
DEFAULT_WORKLOAD = "verify_varlen_paged_bf16_B256"
ELEM = {"f32": 4, "bf16": 2, "fp8": 1}


# ---------------------------------------------------------------------------
# algorithmic bytes: visible K+V at storage dtype + Q + fp32 output + lse +
# lengths + page-table entries + scales
# ---------------------------------------------------------------------------
def verify_bytes(inp: W.VerifyInputs) -> int:
    s = inp.spec
    n = inp.kv_lens.tolist()
    kv = 2 * sum(n) * s.Hkv * s.D * ELEM[s.kv_dtype]
    q = s.B * (s.k + 1) * s.Hq * s.D * ELEM[s.q_dtype]
    out = s.B * (s.k + 1) * s.Hq * (s.D + 1) * 4
    meta = 4 * s.B
    if s.page_size:
        meta += 4 * sum((x + s.page_size - 1) // s.page_size for x in n)
    if s.kv_dtype == "fp8":
        meta += 8 * s.Hkv
    return kv + q + out + meta


def draft_step_bytes(inp: W.DraftInputs, step: int) -> int:
    s = inp.spec
    vis = 0
    for L in inp.base_lens:
        m = L + step + 1
        vis += min(m, s.S) + max(0, min(m - s.S, s.W))
    kv = 2 * vis * s.Hkv * s.D * ELEM[s.kv_dtype]
    q = s.B * s.Hq * s.D * ELEM[s.q_dtype]
    out = s.B * s.Hq * (s.D + 1) * 4
    meta = 8 * s.B + (8 * s.Hkv if s.kv_dtype == "fp8" else 0)
    return kv + q + out + meta


def verify_flops(inp: W.VerifyInputs) -> int:
    s = inp.spec
    return 4 * (s.k + 1) * (s.Hq // s.Hkv) * s.D * s.Hkv * sum(inp.kv_lens.tolist())


# ---------------------------------------------------------------------------
def build_workload(name: str, dev):
    wl = W.named_workloads()[name]
    seed = W.MASTER_SEED + W.WORKLOAD_INDEX[name]
    v = W.make_verify_inputs(wl["verify"], seed, device=dev, poison=None) if "verify" in wl else None
    d = W.make_draft_inputs(wl["draft"], seed, device=dev, poison=None) if "draft" in wl else None
    t = W.make_token_inputs(wl["token"], seed, device=dev) if "token" in wl else None
    if "block" in wl:
        t = W.make_token_inputs(wl["block"], seed, device=dev)
    if "kvupd" in wl:
        t = W.make_kvupdate_inputs(wl["kvupd"], seed, device=dev)
    if "fm" in wl:
        t = W.make_feedback_inputs(wl["fm"], seed, device=dev)
    return wl, v, d, t


def token_bytes(t: W.TokenInputs, n_acc) -> int:
    """Algorithmic bytes of one token verification call, given the accepted
    counts: the min(n+1, k) accept tests (p and q at the draft token, the
    token, the uniform), the sampled row of p (and of q for a correction),
    the sample uniform, and the outputs (n and k+1 tokens)."""
    s = t.spec
    total = 0
    for n in n_acc:
        tests = min(n + 1, s.k)
        total += tests * 16 + 4 * s.V * (2 if n < s.k else 1) + 4 + 4 * (s.k + 2)
    return total


def make_token_step(t: W.TokenInputs):
    """Return (step_fn, bytes_per_step, emitted tokens per step, mean tokens per round)."""
    s = t.spec
    ws = spire.workspace(spire.token_verify_workspace_size(s.B, s.k, s.V))
    n_acc = torch.empty((s.B,), dtype=torch.int32, device=t.p.device)
    toks = torch.empty((s.B, s.k + 1), dtype=torch.int32, device=t.p.device)

    rec = spire.LaunchRecorder(4)

    def step():
        spire.token_verify(t.p, t.q, t.draft, t.u_accept, t.u_sample, n_acc, toks, ws)

    def step_recorded():
        spire.token_verify(t.p, t.q, t.draft, t.u_accept, t.u_sample, n_acc, toks, ws, opts=rec.opts())
        return rec.collect()
    step()
    torch.cuda.synchronize()
    n = n_acc.cpu().tolist()
    emitted = sum(x + 1 for x in n)
    return step, step_recorded, token_bytes(t, n), emitted, emitted / s.B


def block_bytes(t: W.TokenInputs) -> int:
    """Algorithmic bytes of one block verification call: every row of p
    (k+1) and of q (k) is read once (every row's residual mass enters the
    accepted count), the k draft tokens with p and q at them, the uniforms,
    and the outputs (n and k+1 tokens)."""
    s = t.spec
    return s.B * (4 * (2 * s.k + 1) * s.V + 16 * s.k + 4 * s.k + 4 + 4 * (s.k + 2))


def make_block_step(t: W.TokenInputs):
    """Return (step_fn, step_recorded_fn, bytes_per_step, emitted tokens per
    step, mean tokens per round) of block verification."""
    s = t.spec
    ws = spire.workspace(spire.block_verify_workspace_size(s.B, s.k, s.V))
    n_acc = torch.empty((s.B,), dtype=torch.int32, device=t.p.device)
    toks = torch.empty((s.B, s.k + 1), dtype=torch.int32, device=t.p.device)
    rec = spire.LaunchRecorder(4)

    def step():
        spire.block_verify(t.p, t.q, t.draft, t.u_accept, t.u_sample, n_acc, toks, ws)

    def step_recorded():
        spire.block_verify(t.p, t.q, t.draft, t.u_accept, t.u_sample, n_acc, toks, ws, opts=rec.opts())
        return rec.collect()
    step()
    torch.cuda.synchronize()
    emitted = int((n_acc + 1).sum().item())
    return step, step_recorded, block_bytes(t), emitted, emitted / s.B


def timed_call(name, fn):
    """Events on the launch stream around one call that launches one kernel:
    returns a recorded variant giving [(name, ms)]."""
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def run():
        st = torch.cuda.current_stream()
        e0.record(st)
        fn()
        e1.record(st)
        torch.cuda.synchronize()
        return [(name, e0.elapsed_time(e1))]
    return run


def make_step(v, d):
    """Return (step_fn, step_recorded_fn, bytes_per_step, tokens_per_step).
    step_recorded runs the same calls with launch events of the caller's
    (spire_launch_opts) and returns [(kernel name, ms)] of every launch."""
    calls, nbytes = [], 0
    tokens = 0
    if d is not None:
        ds = d.spec
        sink = spire.kv_view(d.sink_k, d.sink_v, k_scale=d.k_scale, v_scale=d.v_scale)
        ring = spire.kv_view(d.ring_k, d.ring_v, k_scale=d.k_scale, v_scale=d.v_scale)
        dws = spire.workspace(spire.draft_workspace_size(ds.B, ds.Hq, ds.Hkv, ds.D))
        dout = torch.empty((ds.B, ds.Hq, ds.D), dtype=torch.float32, device=d.q.device)
        dlse = torch.empty((ds.B, ds.Hq), dtype=torch.float32, device=d.q.device)
        qs = [d.q[t].contiguous() for t in range(ds.steps)]
        lens = [d.seq_lens(t) for t in range(ds.steps)]
        for t in range(ds.steps):
            calls.append(lambda opts=None, t=t: spire.draft_sparse_attn(
                qs[t], sink, ring, lens[t], d.ring_offset, ds.S, ds.W, d.sm_scale, ds.Hkv, out=dout,
                lse=dlse, ws=dws, opts=opts))
            nbytes += draft_step_bytes(d, t)
        tokens = ds.B * ds.steps
    if v is not None:
        vs = v.spec
        kv = spire.kv_view(v.k_cache, v.v_cache, v.block_table, v.page_size, v.k_scale, v.v_scale)
        vws = spire.workspace(spire.verify_workspace_size(vs.B, vs.Hq, vs.Hkv, vs.D, vs.k))
        vout = torch.empty((vs.B, vs.k + 1, vs.Hq, vs.D), dtype=torch.float32, device=v.q.device)
        vlse = torch.empty((vs.B, vs.k + 1, vs.Hq), dtype=torch.float32, device=v.q.device)
        calls.append(lambda opts=None: spire.verify_attn(v.q, kv, v.kv_lens, vs.Hkv, vs.k, v.sm_scale,
                                                         out=vout, lse=vlse, ws=vws, opts=opts))
        nbytes += verify_bytes(v)
        tokens = vs.B * (vs.k + 1)
    recs = [spire.LaunchRecorder(8) for _ in calls]

    def step():
        for c in calls:
            c()

    def step_recorded():
        for c, r in zip(calls, recs):
            c(opts=r.opts())
        return [x for r in recs for x in r.collect()]
    return step, step_recorded, nbytes, tokens


def kvupd_launch_bytes(x: W.KvUpdateInputs) -> dict:
    """Algorithmic bytes per launch of each cache-update kernel: the new K/V
    read (fp32), the storage rows written, for a draft write also the row it
    overwrites read and spilled, for a rollback the spilled rows of rejected
    steps read and written back, plus lengths, offsets and page-table entries."""
    s = x.spec
    es = ELEM[s.kv_dtype]
    row_new, row_st = 2 * s.D * 4, 2 * s.D * es
    draft = s.B * s.Hkv * (row_new + 3 * row_st) + 8 * s.B
    append = s.B * (s.k + 1) * (s.Hkv * (row_new + row_st) + 4) + 4 * s.B
    base = x.base_lens.tolist()
    rej = 0
    for b, n in enumerate(x.n_accepted.tolist()):
        for st in range(n + 1, s.k):
            p = base[b] + st
            if p >= 0 and (p < s.S or s.W > 0):
                rej += 1
    rollback = rej * s.Hkv * 2 * row_st + 12 * s.B
    return {"draft_append": draft, "kv_append": append, "draft_rollback": rollback}


def make_kvupd_step(x: W.KvUpdateInputs):
    """One round of cache writes: k draft writes with spills, the target append
    of the k+1 verified tokens, the rollback of rejected draft writes."""
    s = x.spec
    view = spire.kv_view(x.k_cache, x.v_cache, x.block_table, s.page_size, x.k_scale, x.v_scale)
    sink = spire.kv_view(x.sink_k, x.sink_v, k_scale=x.k_scale, v_scale=x.v_scale)
    ring = spire.kv_view(x.ring_k, x.ring_v, k_scale=x.k_scale, v_scale=x.v_scale)
    spk = torch.empty((s.k, s.B, s.Hkv, s.D), dtype=x.ring_k.dtype, device=x.ring_k.device)
    spv = torch.empty_like(spk)
    lens = [(x.base_lens + st + 1).to(torch.int32) for st in range(s.k)]

    calls = [("draft_append", lambda st=st: spire.draft_append(sink, ring, x.draft_k[st], x.draft_v[st], lens[st],
                                                             x.ring_offset, s.S, s.W, spk[st], spv[st]))
             for st in range(s.k)]
    calls.append(("kv_append", lambda: spire.kv_append(view, x.new_k, x.new_v, x.base_lens)))
    calls.append(("draft_rollback", lambda: spire.draft_rollback(sink, ring, spk, spv, x.base_lens, x.n_accepted,
                                                                 x.ring_offset, s.S, s.W)))
    timed = [timed_call(name, fn) for name, fn in calls]

    def step():
        for _, fn in calls:
            fn()

    def step_recorded():
        return [r for t in timed for r in t()]
    per = kvupd_launch_bytes(x)
    nbytes = s.k * per["draft_append"] + per["kv_append"] + per["draft_rollback"]
    return step, step_recorded, nbytes, s.B * (s.k + 1), per, (view, sink, ring, spk, spv, lens)


def make_fm_step(x: W.FeedbackInputs):
    """One feedback-memory mixing call: reads every layer's activations and
    the weights once, writes the n_out memory vectors."""
    s = x.spec
    out = torch.empty((s.n_out, s.B, s.d), dtype=W.DTYPES[s.m_dtype], device=x.x.device)

    def step():
        spire.feedback_memory(x.x, x.w, out=out)
    nbytes = (s.layers * ELEM[s.x_dtype] + s.n_out * ELEM[s.m_dtype]) * s.B * s.d + 4 * x.w.numel()
    return step, timed_call("feedback_memory", step), nbytes, s.B, {"feedback_memory": nbytes}


def cpu_model() -> str:
    """The host CPU's model name (recorded beside the CPU baseline)."""
    try:
        for ln in open("/proc/cpuinfo"):
            if ln.startswith("model name"):
                return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def run_cpu_baseline_fm(x: W.FeedbackInputs, budget_s: float):
    """The feedback-memory oracle (fp64 numpy) on the whole batch, repeated up
    to the time budget."""
    from oracle import feedback_memory as FM
    s = x.spec
    xs, ws = x.x.float().cpu().numpy(), x.w.cpu().numpy()
    nbytes = (s.layers * ELEM[s.x_dtype] + s.n_out * ELEM[s.m_dtype]) * s.B * s.d
    total_t, reps = 0.0, 0
    while total_t < budget_s and reps < 50:
        t0 = time.perf_counter()
        FM.feedback_memory(xs, ws)
        total_t += time.perf_counter() - t0
        reps += 1
    return {"value": reps * nbytes / total_t / 1e9, "unit": "GB/s", "cores": 1, "kind": "oracle",
            "sample": f"the whole batch, {reps} times", "seconds": round(total_t, 3),
            "tokens_per_s": reps * s.B / total_t, "tokens_unit": "draft tokens/s"}


def dominant_bytes(v, d, dominant, token_step_bytes=None):
    if dominant in ("token_weights", "block_weights", "draft_append", "kv_append", "draft_rollback",
                    "feedback_memory"):
        return token_step_bytes[dominant] if isinstance(token_step_bytes, dict) else token_step_bytes
    if dominant == "verify_partial":
        return verify_bytes(v)
    return sum(draft_step_bytes(d, t) for t in range(d.spec.steps)) / d.spec.steps


# ---------------------------------------------------------------------------
def oracle_sample_verify(v, ids):
    from oracle import oracle as O
    s = v.spec
    idx = torch.tensor(ids, dtype=torch.long, device=v.q.device)
    lens = v.kv_lens[idx]
    q = v.q[idx]
    if v.page_size:
        ps = v.page_size
        nblk = [(int(n) + ps - 1) // ps for n in lens.tolist()]
        rows = v.block_table[idx].long()
        pages = torch.cat([rows[i, :nblk[i]] for i in range(len(ids))])
        kc, vc = v.k_cache.index_select(0, pages).cpu(), v.v_cache.index_select(0, pages).cpu()
        table = torch.full((len(ids), max(nblk)), -1, dtype=torch.int32)
        off = 0
        for i, nb in enumerate(nblk):
            table[i, :nb] = torch.arange(off, off + nb, dtype=torch.int32)
            off += nb
    else:
        kc, vc, table, ps = v.k_cache[idx].cpu(), v.v_cache[idx].cpu(), None, 0
    qc, lc = q.cpu(), lens.cpu()
    ks = None if v.k_scale is None else v.k_scale.cpu()
    vs = None if v.v_scale is None else v.v_scale.cpu()
    t0 = time.perf_counter()
    O.verify(qc, kc, vc, lc, s.k, v.sm_scale, ps, table, ks, vs)
    dt = time.perf_counter() - t0
    n = lc.tolist()
    nbytes = (2 * sum(n) * s.Hkv * s.D * ELEM[s.kv_dtype] + len(ids) * (s.k + 1) * s.Hq * s.D *
              (ELEM[s.q_dtype] + 4))
    return dt, nbytes, len(ids) * (s.k + 1)


def oracle_sample_draft(d, ids, step):
    from oracle import oracle as O
    s = d.spec
    idx = torch.tensor(ids, dtype=torch.long, device=d.q.device)
    args = [d.q[step][idx].cpu(), d.sink_k[idx].cpu(), d.sink_v[idx].cpu(), d.ring_k[idx].cpu(),
            d.ring_v[idx].cpu(), d.seq_lens(step)[idx].cpu(), d.ring_offset[idx].cpu()]
    ks = None if d.k_scale is None else d.k_scale.cpu()
    vs = None if d.v_scale is None else d.v_scale.cpu()
    t0 = time.perf_counter()
    O.draft(*args, s.S, s.W, d.sm_scale, ks, vs)
    dt = time.perf_counter() - t0
    vis = sum(min(d.base_lens[b] + step + 1, s.S) + max(0, min(d.base_lens[b] + step + 1 - s.S, s.W))
              for b in ids)
    nbytes = 2 * vis * s.Hkv * s.D * ELEM[s.kv_dtype] + len(ids) * s.Hq * s.D * (ELEM[s.q_dtype] + 4)
    return dt, nbytes, len(ids)


def run_cpu_baseline_block(t: W.TokenInputs, budget_s: float):
    """The block verification oracle (single-threaded Python + numpy) on whole
    sequences of the same batch, a seeded order, until the time budget."""
    from oracle import block_verify as BV
    s = t.spec
    g = torch.Generator().manual_seed(0)
    order = torch.randperm(s.B, generator=g).tolist()
    per_seq = block_bytes(t) / s.B
    total_t, emitted, used, pos = 0.0, 0, 0, 0
    while total_t < budget_s and pos < len(order):
        ids = order[pos:pos + 16]
        pos += len(ids)
        idx = torch.tensor(ids, dtype=torch.long, device=t.p.device)
        args = [x[idx].cpu().numpy() for x in (t.p, t.q, t.draft, t.u_accept, t.u_sample)]
        t0 = time.perf_counter()
        n, _ = BV.verify_block(*args)
        total_t += time.perf_counter() - t0
        emitted += int((n + 1).sum())
        used += len(ids)
    return {"value": per_seq * used / total_t / 1e9, "unit": "GB/s", "cores": 1, "kind": "oracle",
            "sample": f"block verification of {used} of {s.B} sequences (seeded choice)",
            "seconds": round(total_t, 3), "tokens_per_s": emitted / total_t,
            "tokens_unit": "emitted tokens/s"}


def run_cpu_baseline_token(t: W.TokenInputs, budget_s: float):
    """The token verification oracle (single-threaded Python + numpy) on whole
    sequences of the same batch, a seeded order, until the time budget."""
    from oracle import token_verify as TV
    s = t.spec
    g = torch.Generator().manual_seed(0)
    order = torch.randperm(s.B, generator=g).tolist()
    total_t, total_b, emitted, used, pos = 0.0, 0, 0, 0, 0
    while total_t < budget_s and pos < len(order):
        ids = order[pos:pos + 16]
        pos += len(ids)
        idx = torch.tensor(ids, dtype=torch.long, device=t.p.device)
        args = [x[idx].cpu().numpy() for x in (t.p, t.q, t.draft, t.u_accept, t.u_sample)]
        t0 = time.perf_counter()
        n, _ = TV.verify_tokens(*args)
        total_t += time.perf_counter() - t0
        total_b += token_bytes(t, n.tolist())
        emitted += int((n + 1).sum())
        used += len(ids)
    return {"value": total_b / total_t / 1e9, "unit": "GB/s", "cores": 1, "kind": "oracle",
            "sample": f"token verification of {used} of {s.B} sequences (seeded choice)",
            "seconds": round(total_t, 3), "tokens_per_s": emitted / total_t,
            "tokens_unit": "emitted tokens/s"}


def run_cpu_baseline_kvupd(x: W.KvUpdateInputs, budget_s: float):
    """The cache-update oracle (single-threaded Python, per element) on whole
    sequences of the same round, a seeded order, until the time budget."""
    from oracle import kv_update as KU
    s = x.spec
    g = torch.Generator().manual_seed(0)
    order = torch.randperm(s.B, generator=g).tolist()
    per = kvupd_launch_bytes(x)
    per_seq = (s.k * per["draft_append"] + per["kv_append"] + per["draft_rollback"]) / s.B
    es_np = {"f32": np.float32, "bf16": np.uint16, "fp8": np.uint8}[s.kv_dtype]

    def host(t):
        t = t.detach().cpu().contiguous()
        return t.view(torch.uint8).numpy().copy() if s.kv_dtype == "fp8" else (
            t.view(torch.int16).numpy().view(np.uint16).copy() if s.kv_dtype == "bf16" else t.numpy().copy())
    ks = None if x.k_scale is None else x.k_scale.cpu().numpy()
    vs = None if x.v_scale is None else x.v_scale.cpu().numpy()
    total_t, used, pos = 0.0, 0, 0
    while total_t < budget_s and pos < len(order):
        b = order[pos]
        pos += 1
        idx = slice(b, b + 1)
        sk, sv, rk, rv = (host(t[idx]) for t in (x.sink_k, x.sink_v, x.ring_k, x.ring_v))
        pages = [int(p) for p in x.block_table[b].tolist() if p >= 0]
        kc, vc = host(x.k_cache[pages]), host(x.v_cache[pages])
        table = np.full((1, x.block_table.shape[1]), -1, np.int32)
        for i, p in enumerate(x.block_table[b].tolist()):
            if p >= 0:
                table[0, i] = pages.index(p)
        dk, dv = x.draft_k[:, idx].cpu().numpy(), x.draft_v[:, idx].cpu().numpy()
        nk, nv = x.new_k[idx].cpu().numpy(), x.new_v[idx].cpu().numpy()
        base = x.base_lens[idx].cpu().numpy()
        offs = x.ring_offset[idx].cpu().numpy()
        nacc = x.n_accepted[idx].cpu().numpy()
        spk = np.zeros((s.k, 1, s.Hkv, s.D), es_np)
        spv = np.zeros_like(spk)
        t0 = time.perf_counter()
        for st in range(s.k):
            KU.draft_append(sk, sv, rk, rv, dk[st], dv[st], base + st + 1, offs, s.S, s.W, s.kv_dtype,
                            ks, vs, spk[st], spv[st])
        KU.kv_append(kc, vc, nk, nv, base, s.kv_dtype, s.page_size, table, ks, vs)
        KU.draft_rollback(sk, sv, rk, rv, spk, spv, base, nacc, s.k, offs, s.S, s.W)
        total_t += time.perf_counter() - t0
        used += 1
    return {"value": used * per_seq / total_t / 1e9, "unit": "GB/s", "cores": 1, "kind": "oracle",
            "sample": f"one round of cache writes for {used} of {s.B} sequences (seeded choice)",
            "seconds": round(total_t, 3), "tokens_per_s": used * (s.k + 1) / total_t,
            "tokens_unit": "appended target tokens/s"}


def run_cpu_baseline(v, d, budget_s: float):
    from oracle import oracle as O
    cores = O.threads()
    g = torch.Generator().manual_seed(0)
    total_t, total_b, total_tok, used = 0.0, 0, 0, []
    if v is not None:
        order = torch.randperm(v.spec.B, generator=g).tolist()
        chunk = max(1, cores // max(1, v.spec.Hkv) + 1)
        pos = 0
        while total_t < budget_s and pos < len(order):
            ids = order[pos:pos + chunk]
            pos += chunk
            dt, nb, tok = oracle_sample_verify(v, ids)
            total_t += dt; total_b += nb; total_tok += tok; used += ids
        kind = f"verify rows of {len(used)} of {v.spec.B} sequences (seeded choice)"
        unit_tokens = "verified tokens/s"
    else:
        order = torch.randperm(d.spec.B, generator=g).tolist()
        chunk = max(1, cores // max(1, d.spec.Hkv) + 1)
        pos = 0
        while total_t < budget_s and pos < len(order):
            ids = order[pos:pos + chunk]
            pos += chunk
            dt, nb, tok = oracle_sample_draft(d, ids, 0)
            total_t += dt; total_b += nb; total_tok += tok; used += ids
        kind = f"draft step 0 of {len(used)} of {d.spec.B} sequences (seeded choice)"
        unit_tokens = "drafted tokens/s"
    return {"value": total_b / total_t / 1e9, "unit": "GB/s", "cores": cores, "kind": "oracle",
            "sample": kind, "seconds": round(total_t, 3),
            "tokens_per_s": total_tok / total_t, "tokens_unit": unit_tokens}


# ---------------------------------------------------------------------------
KERNEL_SOURCES = ["paper_2504_06419_amd/csrc/attn_mfma.hip",
                  "paper_2504_06419_amd/csrc/attn_staged.hip",
                  "paper_2504_06419_amd/csrc/plan_combine.hip",
                  "paper_2504_06419_amd/csrc/spire_abi.hip",
                  "paper_2504_06419_amd/csrc/token_verify.hip",
                  "paper_2504_06419_amd/csrc/block_verify.hip",
                  "paper_2504_06419_amd/csrc/sampling.h",
                  "paper_2504_06419_amd/csrc/kv_update.hip",
                  "paper_2504_06419_amd/csrc/feedback_memory.hip",
                  "paper_2504_06419_amd/csrc/mfma_common.h",
                  "paper_2504_06419_amd/csrc/spire_internal.h",
                  "paper_2504_06419_amd/build.py"]


def kernel_source_hash() -> str:
    """sha256 over the code of the measured kernels' sources (line comments and
    blank lines left out, so that editing a comment keeps the record valid);
    recorded HBM traffic is reported only while the kernels are the ones the
    counters were taken on."""
    import hashlib
    import re
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        text = open(os.path.join(ROOT, f), encoding="utf-8").read()
        if not f.endswith(".py"):
            text = re.sub(r"//[^\n]*", "", text)
        lines = [ln.rstrip() for ln in text.splitlines()]
        h.update("\n".join(ln for ln in lines if ln).encode())
    return h.hexdigest()


def calibrate_copy(nbytes: int = 4 << 30, reps: int = 3):
    """A plain device-to-device copy of known size (reads and writes `nbytes`):
    the reference dispatch for scaling rocprofv3 FETCH_SIZE / WRITE_SIZE."""
    src = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    src.fill_(1)
    torch.cuda.synchronize()
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"calibration_copy_bytes": nbytes, "reps": reps}), flush=True)


def recorded_traffic(path: str, workload: str, kernel: str):
    """HBM bytes per launch from the counter record, or None if absent/stale."""
    if not os.path.exists(path):
        return None
    try:
        ent = json.load(open(path)).get(workload, {})
    except (ValueError, OSError):
        return None
    if ent.get("kernel") != kernel or ent.get("source_sha256") != kernel_source_hash():
        return None
    return ent.get("bytes_per_launch")


def perf_model_section(v: W.VerifyInputs, d: W.DraftInputs, reps: int) -> dict:
    """The paper's iteration time multiplier dt = (k t_draft + t_verify) / t_target
    for the attention of this round, measured (one draft call averaged over the
    k steps, the verify call, and a target decode: the verify entry point with
    k = 0 over the same caches, L_b + 1 keys) and modeled (each pass costs
    max(FLOPs, KV bytes * HOI), HOI = 2.5 PFLOP/s bf16 matrix peak / 8 TB/s,
    the kernels computing in bf16)."""
    from paper_2504_06419_amd import perf_model as PM
    vs, ds = v.spec, d.spec
    kv = spire.kv_view(v.k_cache, v.v_cache, v.block_table, v.page_size, v.k_scale, v.v_scale)
    sink = spire.kv_view(d.sink_k, d.sink_v, k_scale=d.k_scale, v_scale=d.v_scale)
    ring = spire.kv_view(d.ring_k, d.ring_v, k_scale=d.k_scale, v_scale=d.v_scale)
    q0 = v.q[:, :1].contiguous()
    lens0 = (v.kv_lens - vs.k).to(torch.int32)
    ws_t = spire.workspace(spire.verify_workspace_size(vs.B, vs.Hq, vs.Hkv, vs.D, 0))
    ws_v = spire.workspace(spire.verify_workspace_size(vs.B, vs.Hq, vs.Hkv, vs.D, vs.k))
    ws_d = spire.workspace(spire.draft_workspace_size(ds.B, ds.Hq, ds.Hkv, ds.D))
    qs = [d.q[t].contiguous() for t in range(ds.steps)]
    dl = [d.seq_lens(t) for t in range(ds.steps)]

    def draft_all():
        for t in range(ds.steps):
            spire.draft_sparse_attn(qs[t], sink, ring, dl[t], d.ring_offset, ds.S, ds.W, d.sm_scale,
                                    ds.Hkv, ws=ws_d)

    def timed(fn, n):
        fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(n):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n

    t_draft = timed(draft_all, reps) / ds.steps
    t_verify = timed(lambda: spire.verify_attn(v.q, kv, v.kv_lens, vs.Hkv, vs.k, v.sm_scale, ws=ws_v), reps)
    t_target = timed(lambda: spire.verify_attn(q0, kv, lens0, vs.Hkv, 0, v.sm_scale, ws=ws_t), reps)
    hoi = PM.hoi(PM.PEAK_FLOPS["bf16"], PM.HBM_BYTES_PER_S)
    dt_model = PM.attention_dt(v.context_lens, vs.k, vs.Hq, vs.Hkv, vs.D, ds.S, ds.W,
                               ELEM[vs.kv_dtype], hoi)
    return {"t_draft_ms": round(t_draft, 5), "t_verify_ms": round(t_verify, 5),
            "t_target_ms": round(t_target, 5), "hoi_flop_per_byte": hoi,
            "dt_measured": round(PM.measured_dt(vs.k, t_draft, t_verify, t_target), 4),
            "dt_modeled": round(dt_model, 4),
            "note": "attention only; the paper's dt also counts weights, absent here"}


FLUSH_BYTES = 512 << 20


def timed_steps(step, steps: int, flush: bool) -> list:
    """Time `steps` steps between two events each on the launch stream, after
    a synchronisation on both sides of the region.  With `flush`, before every
    step (outside its events) a 512 MiB scratch buffer is written, which evicts
    the L2s and the 256 MB Infinity Cache, and then a second 512 MiB buffer is
    read with ordinary loads, which replaces the written lines with clean ones:
    every step then reads its K/V from HBM and pays no write-back of the
    flush's own data (measured on the 256-sequence workload: write-only flush
    2.362 ms per step, write + read 2.322 ms, no flush 2.316 ms).  Returns the
    per-step times in ms."""
    st = torch.cuda.current_stream()
    if flush:
        dirty = torch.empty((FLUSH_BYTES,), dtype=torch.uint8, device="cuda")
        clean = torch.ones((FLUSH_BYTES // 4,), dtype=torch.int32, device="cuda")
        total = torch.empty((), dtype=torch.int64, device="cuda")
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    torch.cuda.synchronize()
    for i in range(steps):
        if flush:
            dirty.fill_(i & 0xFF)
            torch.sum(clean, dim=0, out=total)
        ev[i][0].record(st)
        step()
        ev[i][1].record(st)
    torch.cuda.synchronize()
    if flush:
        del dirty, clean, total
    return [a.elapsed_time(b) for a, b in ev]


def summary(times) -> dict:
    q = lambda f: float(np.percentile(times, f))
    return {"iters": len(times), "median_ms": round(q(50), 5), "p10_ms": round(q(10), 5),
            "p90_ms": round(q(90), 5), "mean_ms": round(float(np.mean(times)), 5)}


def per_kernel(step_recorded, reps: int) -> dict:
    """{kernel name: [ms of each launch]} over `reps` recorded steps."""
    out = {}
    for _ in range(reps):
        for name, t in step_recorded():
            out.setdefault(name, []).append(t)
    return out


def round_section(dev, steps: int) -> dict:
    """The fp8 speculation round (B=512, contexts log-uniform in [2048, 65536],
    k=8: 8 draft steps over S=4 sinks + a W=4096 ring, then the verification of
    9 queries per sequence, 64 query / 8 KV heads, fp8 K/V), timed like the
    main workload: per-round times with cold caches, the roofline fraction of
    its draft and verify kernels, and the paper's iteration-time multiplier dt
    measured against its model."""
    name = "round_fp8_B512_k8"
    t0 = time.perf_counter()
    wl, v, d, _ = build_workload(name, dev)
    step, step_recorded, nbytes, tokens = make_step(v, d)
    torch.cuda.synchronize()
    build_s = time.perf_counter() - t0
    for _ in range(2):
        step()
    cold = summary(timed_steps(step, steps, flush=True))
    kern = per_kernel(step_recorded, 2)
    t_round = cold["median_ms"]
    kd = sum(kern["draft_partial"]) / len(kern["draft_partial"])
    kv_ = sum(kern["verify_partial"]) / len(kern["verify_partial"])
    db = sum(draft_step_bytes(d, t) for t in range(d.spec.steps)) / d.spec.steps
    vb = verify_bytes(v)
    pm = perf_model_section(v, d, 3)
    res = {"workload": name, "ms_per_round": t_round, "round_ms_flushed": cold,
           "verified_tokens_per_s": round(tokens / (t_round * 1e-3), 1),
           "gbs": round(nbytes / (t_round * 1e-3) / 1e9, 2), "bytes_per_round": nbytes,
           "draft_partial": {"avg_launch_ms": round(kd, 5), "bytes_per_launch": db,
                             "achieved_gbs": round(db / (kd * 1e-3) / 1e9, 2),
                             "frac": round(db / (kd * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)},
           "verify_partial": {"avg_launch_ms": round(kv_, 5), "bytes_per_launch": vb,
                              "achieved_gbs": round(vb / (kv_ * 1e-3) / 1e9, 2),
                              "frac": round(vb / (kv_ * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)},
           "kernel_ms": {k: round(sum(x) / len(x), 5) for k, x in kern.items()},
           "dt_measured": pm["dt_measured"], "dt_modeled": pm["dt_modeled"], "perf_model": pm,
           "build_s": round(build_s, 1)}
    del v, d, step, step_recorded
    torch.cuda.empty_cache()
    return res


def read_ceiling(nbytes: int = 4 << 30, reps: int = 10) -> dict:
    """HBM read rate of the library's plain streaming-read probe over a 4 GiB
    buffer (HIP events around each launch): the practical ceiling beside the
    8 TB/s specification."""
    buf = torch.empty((nbytes,), dtype=torch.uint8, device="cuda")
    buf.fill_(1)
    sink = torch.empty((spire.HBM_PROBE_SINK_WORDS,), dtype=torch.int32, device="cuda")
    for _ in range(2):
        spire.hbm_read_probe(buf, sink)
    torch.cuda.synchronize()
    probe = timed_call("hbm_read_probe", lambda: spire.hbm_read_probe(buf, sink))
    ms = [t for _ in range(reps) for _, t in probe()]
    del buf
    avg = sum(ms) / len(ms)
    gbs = nbytes / (avg * 1e-3) / 1e9
    return {"gbs": round(gbs, 1), "frac_of_spec": round(gbs / HBM_PEAK_GBS, 4), "bytes": nbytes,
            "reps": reps, "avg_launch_ms": round(avg, 5)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD, choices=list(W.named_workloads()))
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extras", action="store_true",
                    help="skip the read-ceiling probe (profiler runs)")
    ap.add_argument("--no-round", action="store_true",
                    help="skip the fp8 speculation round that the default workload's line also reports")
    ap.add_argument("--traffic-json", default=os.path.join(ROOT, "profiles", "hbm_traffic.json"))
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a 4 GiB device copy (counter calibration) and exit")
    ap.add_argument("--source-hash", action="store_true", help="print the kernel source hash")
    a = ap.parse_args()
    if a.source_hash:
        print(kernel_source_hash())
        return
    if a.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {a.gpus}); this path is not run "
              "sharded over several GPUs.", file=sys.stderr)
        sys.exit(2)
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if a.calibrate_copy:
        calibrate_copy()
        return
    spire.load()
    print(f"[bench] building workload {a.workload}", file=sys.stderr, flush=True)
    wl, v, d, tk = build_workload(a.workload, dev)
    tok_bytes = None
    is_kvupd = isinstance(tk, W.KvUpdateInputs)
    is_fm = isinstance(tk, W.FeedbackInputs)
    is_block = "block" in wl
    if is_fm:
        step, step_recorded, nbytes, tokens, tok_bytes = make_fm_step(tk)
    elif is_kvupd:
        step, step_recorded, nbytes, tokens, tok_bytes, _keep = make_kvupd_step(tk)
    elif tk is not None and is_block:
        step, step_recorded, nbytes, tokens, tau = make_block_step(tk)
        tok_bytes = nbytes
    elif tk is not None:
        step, step_recorded, nbytes, tokens, tau = make_token_step(tk)
        tok_bytes = nbytes
    else:
        step, step_recorded, nbytes, tokens = make_step(v, d)
    torch.cuda.synchronize()

    print(f"[bench] warmup {a.warmup}", file=sys.stderr, flush=True)
    for _ in range(a.warmup):
        step()
    torch.cuda.synchronize()

    # timed region: exactly K steps, each between two events on the launch
    # stream and each after a cache flush; the step time is their median
    print(f"[bench] timing {a.steps} steps (cold caches)", file=sys.stderr, flush=True)
    cold_times = timed_steps(step, a.steps, flush=True)
    cold = summary(cold_times)
    ms = cold["median_ms"]
    # the same steps back to back with warm caches (extra figure)
    warm = summary(timed_steps(step, a.steps, flush=False))

    # per-kernel durations: events of the caller recorded around each launch on
    # its stream (spire_launch_opts), separate pass
    recs = per_kernel(step_recorded, min(a.steps, 10))
    per_kernel_ms = recs
    kavg = {k: sum(x) / len(x) for k, x in recs.items()}
    # the dominant kernel is the attention kernel with the most time per step
    partials = [k for k in ("verify_partial", "draft_partial", "token_weights", "block_weights",
                            "draft_append", "kv_append", "draft_rollback", "feedback_memory") if k in recs]
    dominant = max(partials, key=lambda k: sum(recs[k]))
    dom_ms = kavg[dominant]
    dom_bytes = dominant_bytes(v, d, dominant, tok_bytes)
    achieved = dom_bytes / (dom_ms * 1e-3) / 1e9
    nrec = min(a.steps, 10)

    traffic = recorded_traffic(a.traffic_json, a.workload, dominant)

    ceiling = None
    if not a.no_extras:
        print("[bench] streaming-read ceiling", file=sys.stderr, flush=True)
        ceiling = read_ceiling()

    gbs = nbytes / (ms * 1e-3) / 1e9
    if is_fm:
        spec = tk.spec
        cfg = {"workload": a.workload, "B": spec.B, "d": spec.d, "layers": spec.layers,
               "n_out": spec.n_out, "x_dtype": spec.x_dtype, "m_dtype": spec.m_dtype}
    elif is_kvupd:
        spec = tk.spec
        cfg = {"workload": a.workload, "B": spec.B, "Hkv": spec.Hkv, "D": spec.D, "k": spec.k,
               "S": spec.S, "W": spec.W, "kv_dtype": spec.kv_dtype, "new_dtype": "f32",
               "page_size": spec.page_size, "ctx": [spec.ctx_lo, spec.ctx_hi]}
    elif tk is not None:
        spec = tk.spec
        cfg = {"workload": a.workload, "B": spec.B, "k": spec.k, "V": spec.V,
               "prob_dtype": "f32", "mean_tokens_per_round": round(tau, 4),
               "verification": "block" if is_block else "token"}
    else:
        spec = (v or d).spec
        cfg = {"workload": a.workload, "B": spec.B, "Hq": spec.Hq, "Hkv": spec.Hkv, "D": spec.D,
               "kv_dtype": spec.kv_dtype}
    if v is not None:
        cfg.update({"k": v.spec.k, "ctx": [v.spec.ctx_lo, v.spec.ctx_hi],
                    "page_size": v.spec.page_size, "sum_kv_len": int(sum(v.kv_lens.tolist()))})
    if d is not None:
        cfg.update({"S": d.spec.S, "W": d.spec.W, "draft_steps": d.spec.steps})
    res = {
        "metric": METRIC, "value": round(gbs, 2), "unit": "GB/s", "n_gpus": 1, "steps": a.steps,
        "warmup": a.warmup, "ms_per_step": round(ms, 5), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None,
        "dtype": (spec.x_dtype if is_fm else spec.kv_dtype if is_kvupd else
                  "f32" if tk is not None else spec.kv_dtype),
        "data": "synthetic",
        "config": cfg,
        "frac_of_hbm_peak": round(gbs / HBM_PEAK_GBS, 4),
        "tokens_per_s": round(tokens / (ms * 1e-3), 1),
        "tokens_unit": ("draft tokens/s" if is_fm else "appended target tokens/s" if is_kvupd else
                        "emitted tokens/s" if tk is not None else
                        "verified tokens/s" if v is not None else "drafted tokens/s"),
        "bytes_per_step": nbytes,
        "step_ms_flushed": cold,
        "warm_ms_per_step": warm["mean_ms"], "warm_gbs": round(nbytes / (warm["mean_ms"] * 1e-3) / 1e9, 2),
        "kernel_ms": {k: round(x, 5) for k, x in kavg.items()},
        "kernel_ms_per_step": {k: round(sum(x) / nrec, 5) for k, x in per_kernel_ms.items()},
        "roofline": {"bound": "hbm", "kernel": dominant, "achieved": round(achieved, 2),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": traffic, "bytes_per_launch": dom_bytes,
                     "avg_launch_ms": round(dom_ms, 5)},
    }
    if ceiling is not None:
        res["read_ceiling"] = dict(ceiling, frac_step=round(gbs / ceiling["gbs"], 4),
                                   frac_dominant=round(achieved / ceiling["gbs"], 4))
    if v is not None and d is not None:
        print("[bench] performance-model times (draft call, verify call, target decode)",
              file=sys.stderr, flush=True)
        res["perf_model"] = perf_model_section(v, d, max(3, a.steps // 2))
    if not a.no_cpu_baseline:
        print(f"[bench] cpu baseline (~{a.cpu_seconds}s)", file=sys.stderr, flush=True)
        if is_fm:
            res["cpu_baseline"] = run_cpu_baseline_fm(tk, a.cpu_seconds)
        elif is_kvupd:
            res["cpu_baseline"] = run_cpu_baseline_kvupd(tk, a.cpu_seconds)
        elif tk is not None and is_block:
            res["cpu_baseline"] = run_cpu_baseline_block(tk, a.cpu_seconds)
        elif tk is not None:
            res["cpu_baseline"] = run_cpu_baseline_token(tk, a.cpu_seconds)
        else:
            res["cpu_baseline"] = run_cpu_baseline(v, d, a.cpu_seconds)
        res["cpu_baseline"]["cpu_model"] = cpu_model()
    if a.workload == DEFAULT_WORKLOAD and not a.no_round:
        # the "per round" half of the metric, on the fp8 speculation round
        del v, d, step, step_recorded
        torch.cuda.empty_cache()
        print("[bench] fp8 speculation round (8 draft steps + verification)", file=sys.stderr, flush=True)
        res["round"] = round_section(dev, min(a.steps, 10))
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
