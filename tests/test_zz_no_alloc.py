"""spire_verify_attn_noalloc (the verify call for callers that cannot
allocate, on the library's own device scratch) against spire_verify_attn
with a caller workspace: two calls in a row, the second on a smaller input,
each bitwise equal to the workspace call and within the tolerance of the fp64
oracle; a request beyond the scratch is rejected and writes nothing."""
import numpy as np
import pytest
import torch

from paper_2504_06419_amd import spire
from paper_2504_06419_amd import workloads as W
from tests.gpu_helpers import TOL, banner, lse_err, max_err, oracle_verify, run_verify

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _noalloc(inp):
    s = inp.spec
    kv = spire.kv_view(inp.k_cache, inp.v_cache, inp.block_table, inp.page_size, inp.k_scale, inp.v_scale)
    out = torch.full((s.B, s.k + 1, s.Hq, s.D), float("nan"), dtype=torch.float32, device=DEV)
    lse = torch.full((s.B, s.k + 1, s.Hq), float("nan"), dtype=torch.float32, device=DEV)
    spire.verify_attn_noalloc(inp.q, kv, inp.kv_lens, s.Hkv, s.k, inp.sm_scale, out, lse)
    torch.cuda.synchronize()
    return out, lse


@pytest.mark.parametrize("kv_dtype,k,g", [("bf16", 4, 4), ("fp8", 8, 8)])
def test_noalloc_equals_workspace_call_twice_in_a_row(kv_dtype, k, g):
    specs = [W.VerifySpec(B=40, Hq=8 * g, Hkv=8, D=128, k=k, ctx_lo=200, ctx_hi=9000, kv_dtype=kv_dtype,
                          page_size=16, spare_pages=4),
             W.VerifySpec(B=5, Hq=2 * g, Hkv=2, D=128, k=k, ctx_lo=1, ctx_hi=700, kv_dtype=kv_dtype,
                          page_size=16, spare_pages=2)]
    for i, spec in enumerate(specs):
        banner(f"no-allocation verify call {i}: {kv_dtype} B={spec.B} k={k} g={g}")
        inp = W.make_verify_inputs(spec, 600 + i, device=DEV)
        out, lse = _noalloc(inp)
        ref_o, ref_l = run_verify(inp)
        assert torch.equal(out, ref_o) and torch.equal(lse, ref_l)
        ids = list(range(min(spec.B, 6)))
        oo, ol = oracle_verify(inp, ids)
        eo, el = max_err(out[ids], oo), lse_err(lse[ids], ol)
        print(f"  max|out-oracle|={eo:.3e} max|lse-oracle|={el:.3e}", flush=True)
        assert eo <= TOL[kv_dtype] and el <= TOL[kv_dtype]


def test_noalloc_rejects_requests_beyond_its_scratch():
    """fp8 K/V with 80 rows per KV head (k = 9, 8 query heads per KV head):
    one wave per worker, 4 workers per CU, 2 partial slots of 80 x 128 fp32
    each -- 80.6 MiB on a 256-CU device, beyond the 80 MiB scratch."""
    banner("no-allocation verify beyond the scratch: fp8, 80 rows per KV head")
    spec = W.VerifySpec(B=8, Hq=16, Hkv=2, D=128, k=9, ctx_lo=10, ctx_hi=50, kv_dtype="fp8")
    inp = W.make_verify_inputs(spec, 610, device=DEV)
    kv = spire.kv_view(inp.k_cache, inp.v_cache, k_scale=inp.k_scale, v_scale=inp.v_scale)
    out = torch.full((spec.B, 10, 16, 128), 7.0, device=DEV)
    if torch.cuda.get_device_properties(0).multi_processor_count < 256:
        pytest.skip("the scratch need depends on the CU count; sized for a 256-CU device")
    with pytest.raises(spire.SpireError) as e:
        spire.verify_attn_noalloc(inp.q, kv, inp.kv_lens, 2, 9, inp.sm_scale, out)
    assert e.value.status == 2 and "scratch" in str(e.value)
    torch.cuda.synchronize()
    assert torch.all(out == 7.0).item()
