"""GPU parity on seeded random medium-size configurations: batch, heads, group
size, k, context ranges, page size, storage type and kernel family are drawn
per case, so that workers cover several whole segments plus pieces at both
ends, segments end on ragged tiles, and every kernel family (generic,
register-staged, LDS-staged) meets many partition shapes.  The HIP path runs
through the C ABI on the whole batch; the fp64 oracle checks a sample of the
sequences (always including the longest and the shortest)."""
import random

import pytest

from paper_2504_06419_amd import spire
from paper_2504_06419_amd import workloads as W
from tests.gpu_helpers import (TOL, banner, lse_err, max_err, oracle_draft, oracle_verify,
                               run_draft, run_verify)

pytestmark = pytest.mark.gpu
DEV = "cuda"
CASES = 24


def _sample(lens, rng, n=5):
    order = sorted(range(len(lens)), key=lambda i: lens[i])
    ids = {order[0], order[-1]}
    while len(ids) < min(n, len(lens)):
        ids.add(rng.randrange(len(lens)))
    return sorted(ids)


def _verify_case(seed):
    rng = random.Random(seed)
    kv_dtype = rng.choice(["bf16", "bf16", "fp8", "fp8", "f32"])
    D = 128 if kv_dtype != "f32" else rng.choice([64, 128])
    k = rng.randrange(0, 16)
    g = rng.choice([1, 2, 3, 4, 6, 8])
    while (k + 1) * g > 128:
        g //= 2
    Hkv = rng.choice([1, 2, 4, 8])
    B = rng.randrange(1, 49)
    lo = rng.randrange(1, 2000)
    hi = lo + rng.randrange(0, 6000)
    ps = rng.choice([0, 16, 32, 64])
    variant = rng.choice([0, 0, 1, 2, 3])
    if seed % 6 == 5:  # the 72 rows of k = 8, g = 8 in fp8 (the one-wave LDS-staged kernel)
        kv_dtype, D, k, g, variant = "fp8", 128, 8, 8, rng.choice([0, 3])
    spec = W.VerifySpec(B=B, Hq=g * Hkv, Hkv=Hkv, D=D, k=k, ctx_lo=lo, ctx_hi=hi,
                        kv_dtype=kv_dtype, q_dtype="f32" if kv_dtype == "f32" else "bf16",
                        page_size=ps, spare_pages=2 if ps else 0, log_uniform=rng.random() < 0.5)
    return spec, variant


def _draft_case(seed):
    rng = random.Random(10_000 + seed)
    kv_dtype = rng.choice(["bf16", "fp8", "f32"])
    D = 128 if kv_dtype != "f32" else rng.choice([64, 128])
    g = rng.choice([1, 2, 4, 8, 16])
    Hkv = rng.choice([1, 2, 4, 8])
    S = rng.choice([0, 1, 4, 7])
    Wn = rng.choice([32, 100, 512, 1024, 3000])
    lo = rng.randrange(1, 2 * Wn)
    hi = lo + rng.randrange(0, 3 * Wn)
    variant = rng.choice([0, 0, 1, 2, 3])
    spec = W.DraftSpec(B=rng.randrange(1, 41), Hq=g * Hkv, Hkv=Hkv, D=D, S=S, W=Wn, steps=2,
                       ctx_lo=lo, ctx_hi=hi, kv_dtype=kv_dtype,
                       q_dtype="f32" if kv_dtype == "f32" else "bf16",
                       log_uniform=rng.random() < 0.5)
    return spec, variant


@pytest.mark.parametrize("seed", range(CASES))
def test_random_verify(seed):
    spec, variant = _verify_case(seed)
    banner(f"random verify seed={seed} variant={variant} {spec}")
    inp = W.make_verify_inputs(spec, 5000 + seed, device=DEV)
    out, lse = run_verify(inp, kernel=variant)
    ids = _sample(inp.kv_lens.tolist(), random.Random(seed))
    ref_o, ref_l = oracle_verify(inp, ids)
    eo, el = max_err(out[ids], ref_o), lse_err(lse[ids], ref_l)
    print(f"  sequences {ids}: max|out-oracle|={eo:.3e} max|lse-oracle|={el:.3e}", flush=True)
    tol = TOL[spec.kv_dtype]
    assert eo <= tol and el <= tol


@pytest.mark.parametrize("seed", range(CASES))
def test_random_draft(seed):
    spec, variant = _draft_case(seed)
    banner(f"random draft seed={seed} variant={variant} {spec}")
    inp = W.make_draft_inputs(spec, 7000 + seed, device=DEV)
    for step in range(spec.steps):
        W.write_step_token(inp, step)
        out, lse = run_draft(inp, step, kernel=variant)
        ids = _sample(inp.seq_lens(step).tolist(), random.Random(seed + step))
        ref_o, ref_l = oracle_draft(inp, step, ids)
        eo, el = max_err(out[ids], ref_o), lse_err(lse[ids], ref_l)
        print(f"  step {step} sequences {ids}: max|out-oracle|={eo:.3e} "
              f"max|lse-oracle|={el:.3e}", flush=True)
        tol = TOL[spec.kv_dtype]
        assert eo <= tol and el <= tol
