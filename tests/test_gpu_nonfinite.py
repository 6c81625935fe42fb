"""Non-finite values inside the visible keys propagate as the attention
definition has them: a NaN key, or a key whose score is +inf, makes every row
that sees it NaN (output and lse); a NaN or infinite value makes the output
elements of its dimension non-finite in the rows that see it, and only there;
a score of -inf weighs zero (a row whose visible scores are all -inf is an
empty row).  The GPU must give the oracle's pattern of NaN rows exactly and
match it elsewhere.  (Non-finite values outside every row's visible set have
no effect at all: that is the poisoned-storage test.)"""
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
    assert np.array_equal(np.isneginf(gl), np.isneginf(ref_l)), "empty-row pattern of the lse differs"
    assert np.array_equal(np.isfinite(gl), lf)
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
    out, lse = run_verify(inp, kernel=variant)
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


# (k, Hq with Hkv = 2): 12 rows (register-staged kernel), 72 rows (LDS-staged),
# 128 rows (LDS-staged, 8 row blocks on two waves)
@pytest.mark.parametrize("kv_dtype", ["bf16", "fp8"])
@pytest.mark.parametrize("variant", [0, 1, 2, 3], ids=["auto", "generic", "mfma_regs", "mfma_lds"])
@pytest.mark.parametrize("k,Hq", [(2, 8), (8, 16), (15, 16)])
def test_verify_nonfinite_value_of_a_key_later_rows_see(kv_dtype, variant, k, Hq):
    """Key n-1 is visible to the last draft row only.  A NaN and an infinite
    value there (fp8: the NaN byte 0x7F) must reach exactly the elements of
    that row's dimensions: rows 0..k-1 of every head of the group match the
    oracle as if the key held anything else (masked positions have no
    effect)."""
    banner(f"verify: non-finite values at key n-1 only row k sees: kv={kv_dtype} variant={variant} k={k} Hq={Hq}")
    spec = W.VerifySpec(B=3, Hq=Hq, Hkv=2, D=128, k=k, ctx_lo=200, ctx_hi=700, kv_dtype=kv_dtype,
                        page_size=16, spare_pages=2)
    inp = W.make_verify_inputs(spec, 91 + k, device=DEV)
    n = inp.kv_lens.tolist()

    def vrow(b, p):  # the stored value row of key p of sequence b, head 1
        return inp.v_cache[int(inp.block_table[b, p // 16]), 1, p % 16]
    if kv_dtype == "fp8":
        vrow(0, n[0] - 1).view(torch.uint8)[5] = 0x7F
        vrow(2, n[2] - 1).view(torch.uint8)[100] = 0xFF
        vrow(2, n[2] - 2).view(torch.uint8)[7] = 0x7F          # seen by the last two rows
    else:
        vrow(0, n[0] - 1)[5] = float("nan")
        vrow(0, n[0] - 1)[9] = float("inf")
        vrow(2, n[2] - 1)[100] = -float("inf")
        vrow(2, n[2] - 2)[7] = float("inf")                     # seen by the last two rows
        vrow(2, n[2] - 1)[7] = -float("inf")                    # ... and -inf for the last: NaN
    out, lse = run_verify(inp, kernel=variant)
    ref_o, ref_l = oracle_verify(inp)
    g = out.double().cpu().numpy()
    assert np.isfinite(g[:, :k - 1]).all()                      # rows that mask both keys
    assert not np.isfinite(ref_o[0, k]).all()
    assert np.array_equal(np.isposinf(g), np.isposinf(ref_o)) and np.array_equal(np.isneginf(g), np.isneginf(ref_o))
    _compare(out, lse, ref_o, ref_l, TOL[kv_dtype])


@pytest.mark.parametrize("variant", [0, 1, 2, 3], ids=["auto", "generic", "mfma_regs", "mfma_lds"])
@pytest.mark.parametrize("k,Hq", [(2, 8), (8, 16)])
def test_verify_rows_with_all_visible_scores_neg_inf(variant, k, Hq):
    """A score of -inf weighs zero: a row whose visible scores are all -inf is
    an empty row (zeros, lse -inf), also when the keys of a long sequence are
    split over many workers, so that the combine merges partials that are all
    -inf with finite ones."""
    banner(f"verify: all visible scores -inf, variant={variant} k={k} Hq={Hq}")
    spec = W.VerifySpec(B=2, Hq=Hq, Hkv=2, D=128, k=k, ctx_lo=40000, ctx_hi=40000, kv_dtype="bf16")
    inp = W.make_verify_inputs(spec, 93, device=DEV)
    inp.q[..., 0] = -inp.q[..., 0].abs().float().clamp(min=0.5).to(inp.q.dtype)
    n = int(inp.kv_lens[0])
    inp.k_cache[0, :, :n, 0] = float("inf")          # sequence 0: every key scores -inf
    inp.k_cache[1, :, :30000, 0] = float("inf")      # sequence 1: the first 30000 keys do
    out, lse = run_verify(inp, kernel=variant)
    ref_o, ref_l = oracle_verify(inp)
    assert np.all(ref_o[0] == 0.0) and np.all(np.isneginf(ref_l[0]))
    assert torch.all(out[0] == 0).item() and torch.isneginf(lse[0]).all().item()
    assert np.isfinite(ref_l[1]).all()
    _compare(out, lse, ref_o, ref_l, TOL["bf16"])
