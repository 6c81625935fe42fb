"""Non-finite values inside the visible keys propagate as the attention
definition has them: a NaN key or value, or a key whose score is +inf, makes
every row that sees it NaN (output and lse); a score of -inf weighs zero.  The
GPU must give the oracle's pattern of NaN rows exactly and match it elsewhere.
(Non-finite values outside the visible set have no effect at all: that is the
poisoned-storage test.)"""
import numpy as np
import pytest
import torch

from paper_2504_06419_amd import spire
from paper_2504_06419_amd import workloads as W
from tests.gpu_helpers import TOL, banner, draft_views, oracle_draft, oracle_verify, run_verify

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _compare(out, lse, ref_o, ref_l, tol):
    g, gl = out.double().cpu().numpy(), lse.double().cpu().numpy()
    assert np.array_equal(np.isnan(g), np.isnan(ref_o)), "NaN pattern of the outputs differs"
    assert np.array_equal(np.isnan(gl), np.isnan(ref_l)), "NaN pattern of the lse differs"
    fin = np.isfinite(ref_o)
    assert np.array_equal(np.isfinite(g), fin)
    err = float(np.max(np.abs(g[fin] - ref_o[fin]))) if fin.any() else 0.0
    lf = np.isfinite(ref_l)
    lerr = float(np.max(np.abs(gl[lf] - ref_l[lf]))) if lf.any() else 0.0
    print(f"  NaN rows {int(np.isnan(ref_l).sum())}, max|out-oracle| {err:.2e}, max|lse-oracle| {lerr:.2e}",
          flush=True)
    assert err <= tol and lerr <= tol


# (k, Hq): 12 rows per KV head (register-staged kernel), 72 rows (LDS-staged)
@pytest.mark.parametrize("kv_dtype", ["bf16", "fp8"])
@pytest.mark.parametrize("variant", [0, 1], ids=["matrix_core", "generic"])
@pytest.mark.parametrize("k,Hq", [(2, 8), (8, 16)])
def test_verify_nonfinite_visible_keys(kv_dtype, variant, k, Hq):
    banner(f"verify with NaN / inf inside the visible keys: kv={kv_dtype} variant={variant} k={k} Hq={Hq}")
    spec = W.VerifySpec(B=3, Hq=Hq, Hkv=2, D=128, k=k, ctx_lo=300, ctx_hi=300, kv_dtype=kv_dtype)
    inp = W.make_verify_inputs(spec, 77, device=DEV)
    if kv_dtype == "fp8":
        kb, vb = inp.k_cache.view(torch.uint8), inp.v_cache.view(torch.uint8)
        kb[1, 0, 5, 7] = 0x7F                       # e4m3fn NaN in a visible key
        vb[2, 1, 10, 3] = 0xFF                      # and in a visible value
    else:
        inp.k_cache[1, 0, 5, 7] = float("nan")
        inp.v_cache[2, 1, 10, 3] = float("nan")
        inp.k_cache[0, 1, 20, 0] = float("inf")     # +inf or -inf scores, by the query's sign
    spire.set_kernel_variant(variant)
    try:
        out, lse = run_verify(inp)
    finally:
        spire.set_kernel_variant(0)
    ref_o, ref_l = oracle_verify(inp)
    assert np.isnan(ref_l).any()
    _compare(out, lse, ref_o, ref_l, TOL[kv_dtype])


def test_draft_nonfinite_visible_slot():
    banner("draft step with a NaN in a visible ring slot and a sink row")
    spec = W.DraftSpec(B=4, Hq=8, Hkv=2, D=128, S=4, W=64, steps=1, ctx_lo=100, ctx_hi=100)
    inp = W.make_draft_inputs(spec, 78, device=DEV)
    W.write_step_token(inp, 0)
    inp.ring_k[1, 0, 9, 4] = float("nan")   # the ring is full: every slot is visible
    inp.sink_v[3, 1, 2, 0] = float("nan")
    sink, ring = draft_views(inp)
    out, lse = spire.draft_sparse_attn(inp.q[0].contiguous(), sink, ring, inp.seq_lens(0), inp.ring_offset,
                                       spec.S, spec.W, inp.sm_scale, spec.Hkv)
    torch.cuda.synchronize()
    ref_o, ref_l = oracle_draft(inp, 0)
    assert np.isnan(ref_l).any()
    _compare(out, lse, ref_o, ref_l, TOL["bf16"])
