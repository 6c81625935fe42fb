"""Shared helpers of the GPU parity tests: run the HIP path through the C ABI
binding, run the CPU oracle on the same stored bytes (optionally on a subset of
sequences, gathered on the device first), and compare."""
from __future__ import annotations

import math
from typing import Optional, Sequence

import numpy as np
import torch

from oracle import oracle as O
from paper_2504_06419_amd import spire
from paper_2504_06419_amd import workloads as W

TOL = {"f32": 1e-5, "bf16": 5e-3, "fp8": 5e-3}


def banner(msg: str):
    print(f"\n[gpu-test] {msg}", flush=True)


def run_verify(inp: W.VerifyInputs, out_dtype=torch.float32, ws=None, kernel: int = 0):
    kv = spire.kv_view(inp.k_cache, inp.v_cache, inp.block_table, inp.page_size, inp.k_scale,
                       inp.v_scale)
    out, lse = spire.verify_attn(inp.q, kv, inp.kv_lens, inp.spec.Hkv, inp.spec.k, inp.sm_scale,
                                 out_dtype=out_dtype, ws=ws, kernel=kernel)
    torch.cuda.synchronize()
    return out, lse


def draft_views(inp: W.DraftInputs):
    sink = spire.kv_view(inp.sink_k, inp.sink_v, k_scale=inp.k_scale, v_scale=inp.v_scale)
    ring = spire.kv_view(inp.ring_k, inp.ring_v, k_scale=inp.k_scale, v_scale=inp.v_scale)
    return sink, ring


def run_draft(inp: W.DraftInputs, step: int, out_dtype=torch.float32, ws=None, kernel: int = 0):
    sink, ring = draft_views(inp)
    s = inp.spec
    out, lse = spire.draft_sparse_attn(inp.q[step].contiguous(), sink, ring, inp.seq_lens(step),
                                       inp.ring_offset, s.S, s.W, inp.sm_scale, s.Hkv,
                                       out_dtype=out_dtype, ws=ws, kernel=kernel)
    torch.cuda.synchronize()
    return out, lse


def oracle_verify(inp: W.VerifyInputs, seq_ids: Optional[Sequence[int]] = None):
    """fp64 oracle on the stored bytes of the selected sequences (all when None)."""
    if seq_ids is None:
        return O.verify(inp.q, inp.k_cache, inp.v_cache, inp.kv_lens, inp.spec.k, inp.sm_scale,
                        inp.page_size, inp.block_table, inp.k_scale, inp.v_scale)
    ids = torch.tensor(list(seq_ids), dtype=torch.long, device=inp.q.device)
    lens = inp.kv_lens[ids]
    q = inp.q[ids]
    if inp.page_size > 0:
        ps = inp.page_size
        nblk = [(int(n) + ps - 1) // ps for n in lens.tolist()]
        rows = inp.block_table[ids].long()
        pages = torch.cat([rows[i, :nblk[i]] for i in range(len(nblk))])
        kc = inp.k_cache.index_select(0, pages)
        vc = inp.v_cache.index_select(0, pages)
        table = torch.full((len(nblk), max(nblk)), -1, dtype=torch.int32)
        off = 0
        for i, nb in enumerate(nblk):
            table[i, :nb] = torch.arange(off, off + nb, dtype=torch.int32)
            off += nb
        return O.verify(q, kc, vc, lens, inp.spec.k, inp.sm_scale, ps, table, inp.k_scale,
                        inp.v_scale)
    return O.verify(q, inp.k_cache[ids], inp.v_cache[ids], lens, inp.spec.k, inp.sm_scale, 0, None,
                    inp.k_scale, inp.v_scale)


def oracle_draft(inp: W.DraftInputs, step: int, seq_ids: Optional[Sequence[int]] = None):
    s = inp.spec
    if seq_ids is None:
        return O.draft(inp.q[step], inp.sink_k, inp.sink_v, inp.ring_k, inp.ring_v,
                       inp.seq_lens(step), inp.ring_offset, s.S, s.W, inp.sm_scale, inp.k_scale,
                       inp.v_scale)
    ids = torch.tensor(list(seq_ids), dtype=torch.long, device=inp.q.device)
    return O.draft(inp.q[step][ids], inp.sink_k[ids], inp.sink_v[ids], inp.ring_k[ids],
                   inp.ring_v[ids], inp.seq_lens(step)[ids], inp.ring_offset[ids], s.S, s.W,
                   inp.sm_scale, inp.k_scale, inp.v_scale)


def max_err(gpu: torch.Tensor, ref: np.ndarray) -> float:
    g = gpu.detach().double().cpu().numpy()
    assert g.shape == ref.shape, (g.shape, ref.shape)
    fin = np.isfinite(ref)
    assert np.array_equal(np.isfinite(g), fin), "non-finite pattern differs"
    if not fin.any():
        return 0.0
    return float(np.max(np.abs(g[fin] - ref[fin])))


def lse_err(gpu: torch.Tensor, ref: np.ndarray) -> float:
    g = gpu.detach().double().cpu().numpy()
    neg = np.isneginf(ref)
    assert np.array_equal(np.isneginf(g), neg), "empty-row pattern differs"
    if neg.all():
        return 0.0
    return float(np.max(np.abs(g[~neg] - ref[~neg])))


def sample_ids(lens: Sequence[int], count: int, seed: int = 0) -> list:
    """Shortest, longest and a few seeded others."""
    B = len(lens)
    order = sorted(range(B), key=lambda b: lens[b])
    pick = {order[0], order[-1]}
    g = torch.Generator().manual_seed(seed)
    for b in torch.randperm(B, generator=g).tolist():
        if len(pick) >= min(count, B):
            break
        pick.add(b)
    return sorted(pick)


def partition_roles(lens: Sequence[int], cap: int, units: int, tile: int, seg_cost: int,
                    workers: int) -> dict:
    """Sequences whose segments play distinct roles in the stream-K partition
    the attention kernels use (the flattened positions of every (sequence,
    unit) segment -- its tiles, then seg_cost phantom positions -- split into
    `workers` equal ranges): a segment split over three or more workers, the
    first and the last worker's segments, a worker whose range starts inside
    a segment's phantom positions (its segment and the next), and a worker
    covering several whole segments.  Computed on the host from the lengths."""
    n = [min(max(int(x), 0), cap) for x in lens]
    B = len(n)
    span = [max(1, (x + tile - 1) // tile) + seg_cost for x in n]
    prefix = [0]
    for sp in span:
        prefix.append(prefix[-1] + sp)
    T = prefix[B] * units
    worker_of = lambda x: ((x + 1) * workers - 1) // T
    begin = lambda w: w * T // workers
    roles = {"first_worker": 0, "last_worker": B - 1}
    for b in range(B):
        for u in range(units):
            start = prefix[b] * units + u * span[b]
            tiles = span[b] - seg_cost
            wlo, whi = worker_of(start), worker_of(start + tiles - 1)
            if whi - wlo >= 2:
                roles.setdefault("split_over_3_workers", b)
            if wlo == whi and begin(wlo) < start and worker_of(start + span[b]) == wlo:
                roles.setdefault("inside_a_multi_segment_worker", b)
    import bisect
    for w in range(workers):
        x = begin(w)
        if x >= begin(w + 1):
            continue
        b = bisect.bisect_right([p * units for p in prefix], x) - 1
        rel = x - prefix[b] * units
        if rel % span[b] >= span[b] - seg_cost:
            roles.setdefault("worker_starts_in_phantoms", b)
            if b + 1 < B:
                roles.setdefault("after_phantom_start", b + 1)
            break
    return roles


def role_ids(inp: W.VerifyInputs, extra: int = 3, seed: int = 0) -> list:
    """Sample of a full-size verify batch for the oracle: the partition roles of
    the matrix-core kernel the call takes (32-key tiles, one unit per KV head,
    4 workers per compute unit, phantom positions worth 40 KB of K+V per
    segment), the shortest and longest sequences and a few seeded others."""
    s = inp.spec
    es = {"bf16": 2, "fp8": 1, "f32": 4}[s.kv_dtype]
    tile_bytes = 2 * 32 * s.D * es
    seg_cost = (40960 + tile_bytes // 2) // tile_bytes
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    cap = inp.block_table.shape[1] * s.page_size if s.page_size else inp.capacity
    roles = partition_roles(inp.kv_lens.tolist(), cap, s.Hkv, 32, seg_cost, 4 * cus)
    print(f"  partition roles: {roles}", flush=True)
    return sorted(set(roles.values()) | set(sample_ids(inp.kv_lens.tolist(), extra, seed)))
