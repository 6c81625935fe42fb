"""GPU parity: the HIP path (through the C ABI) against the fp64 CPU oracle on
the same seeded inputs.  Tolerances: max abs error <= 1e-5 with fp32 storage,
<= 5e-3 with bf16 / fp8 K/V (fp32 accumulation), on outputs and on the
log-sum-exp.  Small cases compare every element and span several tiles plus a
ragged tail; the full-size workloads compare sampled sequences one by one."""
import math

import numpy as np
import pytest
import torch

from paper_2504_06419_amd import spire
from paper_2504_06419_amd import workloads as W
from tests.gpu_helpers import (TOL, banner, lse_err, max_err, oracle_draft, oracle_verify,
                               role_ids, run_draft, run_verify, sample_ids)

pytestmark = pytest.mark.gpu
DEV = "cuda"
NW = W.named_workloads()


@pytest.fixture(params=[0, 1, 2, 3], ids=["auto", "generic", "mfma_regs", "mfma_lds"])
def variant(request):
    """The kernel family each call asks for (spire_launch_opts.kernel)."""
    return request.param


def _check_verify(inp, tol, seq_ids=None, out_dtype=torch.float32, kernel=0):
    out, lse = run_verify(inp, out_dtype=out_dtype, kernel=kernel)
    ref_o, ref_l = oracle_verify(inp, seq_ids)
    if seq_ids is not None:
        out, lse = out[seq_ids], lse[seq_ids]
    eo, el = max_err(out, ref_o), lse_err(lse, ref_l)
    print(f"  max|out-oracle|={eo:.3e} max|lse-oracle|={el:.3e}", flush=True)
    assert eo <= tol and el <= tol
    return out, lse


def _check_draft(inp, step, tol, seq_ids=None, kernel=0):
    out, lse = run_draft(inp, step, kernel=kernel)
    ref_o, ref_l = oracle_draft(inp, step, seq_ids)
    if seq_ids is not None:
        out, lse = out[seq_ids], lse[seq_ids]
    eo, el = max_err(out, ref_o), lse_err(lse, ref_l)
    print(f"  step {step}: max|out-oracle|={eo:.3e} max|lse-oracle|={el:.3e}", flush=True)
    assert eo <= tol and el <= tol


# ---------------------------------------------------------------------------
# the tiny fp32 workload (every element)
# ---------------------------------------------------------------------------
def test_tiny_f32_verify(variant):
    banner(f"tiny_f32 verify variant={variant}")
    spec = NW["tiny_f32"]["verify"]
    inp = W.make_verify_inputs(spec, W.MASTER_SEED + 0, device=DEV)
    _check_verify(inp, TOL["f32"], kernel=variant)


def test_tiny_f32_draft_steps(variant):
    banner(f"tiny_f32 draft variant={variant}")
    spec = NW["tiny_f32"]["draft"]
    inp = W.make_draft_inputs(spec, W.MASTER_SEED + 0, device=DEV)
    for step in range(spec.steps):
        W.write_step_token(inp, step)
        _check_draft(inp, step, TOL["f32"], kernel=variant)


def test_tiny_f32_draft_on_target_cache_view():
    """Self-speculation: the draft reads the target's own contiguous cache through
    sink rows [0, S) and a ring view of rows [m - W, m)."""
    banner("tiny_f32 draft as a view of the verify cache")
    spec = NW["tiny_f32"]["verify"]
    inp = W.make_verify_inputs(spec, W.MASTER_SEED + 0, device=DEV)
    S, Wn = 4, 128
    m = int(inp.kv_lens[0])
    sink_k, sink_v = inp.k_cache[:, :, :S], inp.v_cache[:, :, :S]
    ring_k, ring_v = inp.k_cache[:, :, m - Wn:m], inp.v_cache[:, :, m - Wn:m]
    offs = torch.full((spec.B,), (S - m) % Wn, dtype=torch.int32, device=DEV)
    q = inp.q[:, -1].contiguous()
    sink = spire.kv_view(sink_k, sink_v, capacity=S)
    ring = spire.kv_view(ring_k, ring_v, capacity=Wn)
    out, lse = spire.draft_sparse_attn(q, sink, ring, inp.kv_lens, offs, S, Wn, inp.sm_scale,
                                       spec.Hkv)
    torch.cuda.synchronize()
    from oracle import oracle as O
    ref, _ = O.draft(q, sink_k, sink_v, ring_k, ring_v, inp.kv_lens, offs, S, Wn, inp.sm_scale)
    assert max_err(out, ref) <= TOL["f32"]


# ---------------------------------------------------------------------------
# small shapes: many tiles, ragged tails, every k, grouped heads, layouts
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("kv_dtype", ["bf16", "fp8"])
@pytest.mark.parametrize("ps", [0, 16, 32])
@pytest.mark.parametrize("k,g", [(0, 1), (1, 4), (4, 4), (7, 8), (8, 8), (3, 2),
                                 (10, 1), (12, 6), (10, 8), (15, 8)])
def test_verify_small_shapes(variant, kv_dtype, ps, k, g):
    """Up to (k+1) * g = 128 rows per KV head (k = 15, 8 query heads per KV
    head): 1-2 row blocks on the register-staged kernel, 3-8 on the LDS-staged
    one (one wave, or two sharing the stage ring)."""
    banner(f"verify small {kv_dtype} ps={ps} k={k} g={g} variant={variant}")
    spec = W.VerifySpec(B=6, Hq=2 * g, Hkv=2, D=128, k=k, ctx_lo=1, ctx_hi=300, kv_dtype=kv_dtype,
                        page_size=ps, spare_pages=3, log_uniform=True)
    inp = W.make_verify_inputs(spec, 1000 + 13 * k + g + ps, device=DEV)
    _check_verify(inp, TOL[kv_dtype], kernel=variant)


@pytest.mark.parametrize("kv_dtype", ["bf16", "fp8"])
@pytest.mark.parametrize("k,g", [(1, 4), (8, 8)])
def test_verify_growing_scores(variant, kv_dtype, k, g):
    """Key magnitudes that grow 20x along the sequence, plus isolated spikes:
    every row's running maximum moves many times inside one worker's range,
    which exercises the rescale path of the online softmax."""
    banner(f"verify growing scores {kv_dtype} k={k} g={g} variant={variant}")
    spec = W.VerifySpec(B=3, Hq=2 * g, Hkv=2, D=128, k=k, ctx_lo=2000, ctx_hi=6000,
                        kv_dtype=kv_dtype)
    inp = W.make_verify_inputs(spec, 4242 + k + g, device=DEV)
    kc = inp.k_cache                                     # [B, Hkv, cap, D]
    cap = kc.shape[2]
    ramp = torch.linspace(0.25, 5.0, cap, device=DEV).view(1, 1, cap, 1)
    kf = kc.float() * ramp
    kf[:, :, 397::811] *= 3.0                           # spikes
    kc.copy_(kf.clamp(-448.0, 448.0).to(kc.dtype))
    _check_verify(inp, TOL[kv_dtype], kernel=variant)


@pytest.mark.parametrize("D", [64, 128])
def test_verify_fp32_and_head_dims(variant, D):
    banner(f"verify f32 D={D} variant={variant}")
    spec = W.VerifySpec(B=3, Hq=8, Hkv=2, D=D, k=4, ctx_lo=30, ctx_hi=200, kv_dtype="f32",
                        q_dtype="f32", page_size=16, spare_pages=2)
    inp = W.make_verify_inputs(spec, 77 + D, device=DEV)
    _check_verify(inp, TOL["f32"], kernel=variant)


def test_verify_bf16_head_dim_64():
    banner("verify bf16 D=64")
    spec = W.VerifySpec(B=4, Hq=8, Hkv=2, D=64, k=2, ctx_lo=10, ctx_hi=150, kv_dtype="bf16")
    inp = W.make_verify_inputs(spec, 5, device=DEV)
    _check_verify(inp, TOL["bf16"])


def test_verify_bf16_output():
    banner("verify bf16 output")
    spec = W.VerifySpec(B=4, Hq=16, Hkv=4, D=128, k=4, ctx_lo=40, ctx_hi=500, page_size=16)
    inp = W.make_verify_inputs(spec, 6, device=DEV)
    _check_verify(inp, TOL["bf16"] + 2 ** -8, out_dtype=torch.bfloat16)


def test_verify_degenerate_lengths():
    """n = k+1 (query 0 sees one key), n < k+1 (empty rows), n = 0."""
    banner("verify degenerate lengths")
    spec = W.VerifySpec(B=5, Hq=8, Hkv=2, D=128, k=4, ctx_lo=0, ctx_hi=0, page_size=16)
    inp = W.make_verify_inputs(spec, 8, device=DEV)
    inp.kv_lens = torch.tensor([5, 3, 0, 1, 5], dtype=torch.int32, device=DEV)
    for v in (0, 1):
        out, lse = run_verify(inp, kernel=v)
        ref_o, ref_l = oracle_verify(inp)
        assert max_err(out, ref_o) <= TOL["bf16"] and lse_err(lse, ref_l) <= TOL["bf16"]


def test_verify_lengths_beyond_capacity_are_clamped():
    banner("verify lengths beyond capacity")
    spec = W.VerifySpec(B=3, Hq=8, Hkv=2, D=128, k=2, ctx_lo=40, ctx_hi=40)
    inp = W.make_verify_inputs(spec, 9, device=DEV)
    cap = inp.capacity
    big = inp.kv_lens.clone()
    big[1] = cap + 1000
    out, lse = spire.verify_attn(inp.q, spire.kv_view(inp.k_cache, inp.v_cache), big, 2, 2,
                                 inp.sm_scale)
    ref, _ = oracle_verify(W.VerifyInputs(**{**inp.__dict__, "kv_lens": torch.clamp(big, max=cap)}))
    assert max_err(out, ref) <= TOL["bf16"]


@pytest.mark.parametrize("which", ["keys", "values"])
def test_fp8_every_byte_pattern(which):
    """Each of the 254 finite e4m3fn patterns through the matrix-core path:
    constant V rows give decode(byte) * v_scale; constant K rows and a unit
    query give lse = ln n + decode(byte) * k_scale * sm_scale."""
    banner(f"fp8 byte patterns ({which})")
    finite = [x for x in range(256) if x not in (0x7F, 0xFF)]
    B = len(finite)
    # 48 keys per sequence: a contiguous capacity the matrix-core kernel takes
    spec = W.VerifySpec(B=B, Hq=2, Hkv=1, D=128, k=0, ctx_lo=47, ctx_hi=47, kv_dtype="fp8")
    inp = W.make_verify_inputs(spec, 10, device=DEV)
    pat = torch.tensor(finite, dtype=torch.uint8, device=DEV).view(B, 1, 1, 1)
    if which == "values":
        inp.v_cache.view(torch.uint8)[:] = pat
        inp.q.zero_()
    else:
        inp.k_cache.view(torch.uint8)[:] = pat
        inp.q.zero_()
        inp.q[..., 0] = 1.0
    out, lse = run_verify(inp)
    ref_o, ref_l = oracle_verify(inp)
    assert max_err(out, ref_o) <= 1e-6 * 448 * 0.02
    assert lse_err(lse, ref_l) <= 1e-5


@pytest.mark.parametrize("kv_dtype", ["bf16", "fp8"])
@pytest.mark.parametrize("S,Wn,lo,hi", [(4, 64, 1, 200), (0, 32, 1, 100), (4, 0, 1, 10),
                                        (1, 128, 100, 400), (8, 48, 1, 12)])
def test_draft_small_shapes(variant, kv_dtype, S, Wn, lo, hi):
    banner(f"draft small {kv_dtype} S={S} W={Wn} ctx=[{lo},{hi}] variant={variant}")
    spec = W.DraftSpec(B=7, Hq=16, Hkv=2, D=128, S=S, W=Wn, steps=3, ctx_lo=lo, ctx_hi=hi,
                       kv_dtype=kv_dtype)
    inp = W.make_draft_inputs(spec, 2000 + S + Wn + lo, device=DEV)
    for step in range(spec.steps):
        W.write_step_token(inp, step)
        _check_draft(inp, step, TOL[kv_dtype], kernel=variant)


@pytest.mark.parametrize("kv_dtype", ["bf16", "fp8"])
@pytest.mark.parametrize("g", [24, 40, 72])
def test_draft_group_sizes(variant, kv_dtype, g):
    """Draft with 17..80 query heads per KV head: two row blocks in the
    register-staged kernel, three to five in the LDS-staged one (ring wrap,
    sinks and filling rings on every path)."""
    banner(f"draft g={g} {kv_dtype} variant={variant}")
    spec = W.DraftSpec(B=5, Hq=2 * g, Hkv=2, D=128, S=4, W=96, steps=2, ctx_lo=1, ctx_hi=400,
                       kv_dtype=kv_dtype)
    inp = W.make_draft_inputs(spec, 3000 + g, device=DEV)
    for step in range(spec.steps):
        W.write_step_token(inp, step)
        _check_draft(inp, step, TOL[kv_dtype], kernel=variant)


# ---------------------------------------------------------------------------
# properties
# ---------------------------------------------------------------------------
def test_deterministic_and_poison_independent():
    banner("determinism and masked-storage independence")
    spec = W.VerifySpec(B=8, Hq=32, Hkv=8, D=128, k=4, ctx_lo=50, ctx_hi=3000, page_size=16,
                        spare_pages=8)
    a = W.make_verify_inputs(spec, 11, device=DEV, poison="nan")
    b = W.make_verify_inputs(spec, 11, device=DEV, poison="big")
    oa1, la1 = run_verify(a)
    oa2, la2 = run_verify(a)
    ob, lb = run_verify(b)
    assert torch.equal(oa1, oa2) and torch.equal(la1, la2)
    assert torch.isfinite(oa1).all()
    assert torch.equal(oa1, ob) and torch.equal(la1, lb)


def test_paged_equals_contiguous_on_gpu():
    banner("paged vs contiguous")
    mk = lambda ps: W.make_verify_inputs(
        W.VerifySpec(B=5, Hq=16, Hkv=4, D=128, k=3, ctx_lo=20, ctx_hi=900, page_size=ps), 12,
        device=DEV, keep_logical=True)
    a, b = mk(0), mk(16)
    oa, la = run_verify(a, kernel=1)   # same arithmetic on both layouts: bitwise equal
    ob, lb = run_verify(b, kernel=1)
    assert torch.equal(oa, ob) and torch.equal(la, lb)
    oc, lc = run_verify(b)             # matrix-core path on the paged layout
    assert (oa - oc).abs().max().item() <= TOL["bf16"]


# ---------------------------------------------------------------------------
# full-size workloads (sampled sequences against the oracle)
# ---------------------------------------------------------------------------
def _finite_everywhere(inp):
    out, lse = run_verify(inp)
    assert torch.isfinite(out).all().item() and torch.isfinite(lse).all().item()


def test_verify_bf16_B64_L8192():
    banner("verify_bf16_B64_L8192")
    spec = NW["verify_bf16_B64_L8192"]["verify"]
    inp = W.make_verify_inputs(spec, W.MASTER_SEED + 1, device=DEV)
    _check_verify(inp, TOL["bf16"], seq_ids=sorted({17} | set(role_ids(inp, seed=1))))
    _finite_everywhere(inp)


def test_draft_bf16_B64_S4_W2048():
    banner("draft_bf16_B64_S4_W2048")
    spec = NW["draft_bf16_B64_S4_W2048"]["draft"]
    inp = W.make_draft_inputs(spec, W.MASTER_SEED + 2, device=DEV)
    for step in range(spec.steps):
        W.write_step_token(inp, step)
        _check_draft(inp, step, TOL["bf16"], seq_ids=[0, 31, 63] if step % 2 else [5, 40])


def test_verify_varlen_paged_bf16_B256():
    banner("verify_varlen_paged_bf16_B256")
    spec = NW["verify_varlen_paged_bf16_B256"]["verify"]
    inp = W.make_verify_inputs(spec, W.MASTER_SEED + 3, device=DEV)
    _check_verify(inp, TOL["bf16"], seq_ids=role_ids(inp, seed=3))
    _finite_everywhere(inp)


def test_round_fp8_B512_k8():
    banner("round_fp8_B512_k8: 8 draft steps then verify")
    wl = NW["round_fp8_B512_k8"]
    d = W.make_draft_inputs(wl["draft"], W.MASTER_SEED + 4, device=DEV)
    for step in range(wl["draft"].steps):
        W.write_step_token(d, step)
        _check_draft(d, step, TOL["fp8"], seq_ids=sample_ids(d.base_lens, 3, seed=step))
        out, lse = run_draft(d, step)
        assert torch.isfinite(out).all().item() and torch.isfinite(lse).all().item()
    del d
    torch.cuda.empty_cache()
    inp = W.make_verify_inputs(wl["verify"], W.MASTER_SEED + 4, device=DEV)
    _check_verify(inp, TOL["fp8"], seq_ids=role_ids(inp, seed=4))
    _finite_everywhere(inp)


def test_verify_tp8shard_fp8_B512_k8():
    banner("verify_tp8shard_fp8_B512_k8: one tensor-parallel shard of the fp8 verify")
    name = "verify_tp8shard_fp8_B512_k8"
    inp = W.make_verify_inputs(NW[name]["verify"], W.MASTER_SEED + W.WORKLOAD_INDEX[name], device=DEV)
    _check_verify(inp, TOL["fp8"], seq_ids=role_ids(inp, seed=9))
    _finite_everywhere(inp)


# (kv dtype, k, query heads per KV head, phantom positions per segment):
# bf16 20 rows and fp8 8 rows run the register-staged kernel, which computes
# the partition itself; fp8 72 rows runs the LDS-staged kernel after the plan
# kernel.  Phantom positions: the tiles holding 40 KB of K+V (32 keys x 128
# dims x 2 tensors: 16 KB per bf16 tile, 8 KB per fp8 tile).
@pytest.mark.parametrize("kv_dtype,k,g,seg_cost", [("bf16", 4, 4, 3), ("fp8", 0, 8, 5), ("fp8", 8, 8, 5)])
def test_plan_partition_invariants(kv_dtype, k, g, seg_cost):
    """The partition read back from the workspace (layout of spire_abi.hip):
    clamped key counts, prefix sums of tile + phantom positions, worker start
    points."""
    banner(f"plan partition: {kv_dtype} k={k} g={g}")
    Hkv = 8
    spec = W.VerifySpec(B=37, Hq=g * Hkv, Hkv=Hkv, D=128, k=k, ctx_lo=1, ctx_hi=5000, page_size=16,
                        kv_dtype=kv_dtype)
    inp = W.make_verify_inputs(spec, 14, device=DEV)
    cap = inp.block_table.shape[1] * 16
    lens = inp.kv_lens.clone()
    lens[3] = 0
    lens[5] = cap + 100
    inp.kv_lens = lens
    ws = spire.workspace(spire.verify_workspace_size(37, g * Hkv, Hkv, 128, k))
    ws.fill_(0xAB)
    run_verify(inp, ws=ws)
    raw = ws.cpu()
    al = lambda x: (x + 255) // 256 * 256
    B, tile, units = 37, 32, Hkv
    nkeys = raw[0:4 * B].view(torch.int32)
    o1 = al(4 * B)
    prefix = raw[o1:o1 + 4 * (B + 1)].view(torch.int32)
    o2 = o1 + al(4 * (B + 1))
    workers = torch.cuda.get_device_properties(0).multi_processor_count * 4
    wstart = raw[o2:o2 + 8 * workers].view(torch.int32).view(-1, 2)
    assert nkeys.tolist() == torch.clamp(lens.cpu(), 0, cap).tolist()
    tiles = [max(1, (n + tile - 1) // tile) + seg_cost for n in nkeys.tolist()]
    assert prefix.tolist() == [sum(tiles[:b]) for b in range(B + 1)]
    T = prefix[B].item() * units
    covered = 0
    for w in range(workers):
        b0, b1 = w * T // workers, (w + 1) * T // workers
        if b0 >= b1:
            assert wstart[w, 0].item() == -1
            continue
        seg, t = wstart[w].tolist()
        b, u = divmod(seg, units)
        assert prefix[b].item() * units + u * tiles[b] + t == b0
        covered += b1 - b0
    assert covered == T


# ---------------------------------------------------------------------------
# fp8 draft views with scales of their own; launch records
# ---------------------------------------------------------------------------
def test_draft_fp8_sink_and_ring_with_their_own_scales(variant):
    """The header lets the sink and ring fp8 views carry different per-head
    scales; each key is dequantised with its own view's scales."""
    banner(f"draft fp8 with separate sink / ring scales variant={variant}")
    spec = W.DraftSpec(B=6, Hq=16, Hkv=2, D=128, S=4, W=96, steps=2, ctx_lo=1, ctx_hi=400,
                       kv_dtype="fp8")
    inp = W.make_draft_inputs(spec, 3100, device=DEV)
    sk = (inp.k_scale * torch.tensor([3.0, 0.25], device=DEV)).contiguous()
    sv = (inp.v_scale * torch.tensor([0.5, 4.0], device=DEV)).contiguous()
    sink = spire.kv_view(inp.sink_k, inp.sink_v, k_scale=sk, v_scale=sv)
    ring = spire.kv_view(inp.ring_k, inp.ring_v, k_scale=inp.k_scale, v_scale=inp.v_scale)
    from oracle import oracle as O
    for step in range(spec.steps):
        W.write_step_token(inp, step)
        out, lse = spire.draft_sparse_attn(inp.q[step].contiguous(), sink, ring, inp.seq_lens(step),
                                           inp.ring_offset, spec.S, spec.W, inp.sm_scale, spec.Hkv,
                                           kernel=variant)
        torch.cuda.synchronize()
        ref_o, ref_l = O.draft(inp.q[step], inp.sink_k, inp.sink_v, inp.ring_k, inp.ring_v,
                               inp.seq_lens(step), inp.ring_offset, spec.S, spec.W, inp.sm_scale,
                               inp.k_scale, inp.v_scale, sink_k_scale=sk, sink_v_scale=sv)
        same, _ = O.draft(inp.q[step], inp.sink_k, inp.sink_v, inp.ring_k, inp.ring_v,
                          inp.seq_lens(step), inp.ring_offset, spec.S, spec.W, inp.sm_scale,
                          inp.k_scale, inp.v_scale)
        assert np.max(np.abs(ref_o - same)) > 1e-2          # the scales matter
        eo, el = max_err(out, ref_o), lse_err(lse, ref_l)
        print(f"  step {step}: max|out-oracle|={eo:.3e} max|lse-oracle|={el:.3e}", flush=True)
        assert eo <= TOL["fp8"] and el <= TOL["fp8"]


@pytest.mark.parametrize("kv_dtype,k,g,kernel,expect", [
    ("bf16", 4, 4, 0, ["verify_partial", "combine", "tail_check"]),            # register-staged
    ("fp8", 8, 8, 0, ["plan", "verify_partial", "combine", "tail_check"]),     # LDS-staged
    ("bf16", 4, 4, 1, ["plan", "verify_partial", "combine"]),                  # generic
])
def test_launch_records(kv_dtype, k, g, kernel, expect):
    """spire_launch_opts: the caller's events bracket each launch of the call, in
    order, with its kernel id; the results equal those of the plain call."""
    banner(f"launch records {kv_dtype} k={k} g={g} kernel={kernel}")
    spec = W.VerifySpec(B=5, Hq=2 * g, Hkv=2, D=128, k=k, ctx_lo=100, ctx_hi=3000, kv_dtype=kv_dtype,
                        page_size=16)
    inp = W.make_verify_inputs(spec, 15, device=DEV)
    rec = spire.LaunchRecorder(8)
    kv = spire.kv_view(inp.k_cache, inp.v_cache, inp.block_table, 16, inp.k_scale, inp.v_scale)
    out, lse = spire.verify_attn(inp.q, kv, inp.kv_lens, spec.Hkv, k, inp.sm_scale, opts=rec.opts(kernel))
    recs = rec.collect()
    assert [name for name, _ in recs] == expect
    assert all(ms >= 0.0 for _, ms in recs)
    ref_o, ref_l = run_verify(inp, kernel=kernel)
    assert torch.equal(out, ref_o) and torch.equal(lse, ref_l)
    small = spire.LaunchRecorder(1)                     # launches beyond max_launches are not recorded
    spire.verify_attn(inp.q, kv, inp.kv_lens, spec.Hkv, k, inp.sm_scale, opts=small.opts(kernel))
    assert [name for name, _ in small.collect()] == expect[:1] and small._n.value == len(expect)
