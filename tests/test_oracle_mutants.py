"""The oracle's pins must be strong enough to catch plausible mistakes.

Each case copies the oracle source, plants one mistake (a dropped term, a wrong
sign or index, a swapped operand), builds it into a temporary library on the
CPU and checks that the brute-force / closed-form pins reject it.  The real
oracle passes the same battery.
"""
import math
import os
import subprocess

import numpy as np
import pytest
import torch

from oracle import brute
from oracle import oracle as O
from paper_2504_06419_amd import workloads as W

MUTANTS = {
    "causal_off_by_one": ("int64_t visible = n - k + i;", "int64_t visible = n - k + i + 1;"),
    "causal_reversed": ("int64_t visible = n - k + i;", "int64_t visible = n - i;"),
    "gqa_interleaved_heads": ("const int h = hk * g + hg;", "const int h = hg * Hkv + hk;"),
    "softmax_scale_dropped": ("scores[t] = sm_scale * dot;", "scores[t] = dot;"),
    "window_off_by_one": ("int64_t win_begin = m - W > S ? m - W : S;",
                          "int64_t win_begin = m - W + 1 > S ? m - W + 1 : S;"),
    "sink_not_clamped": ("int64_t sink_end = m < S ? m : S;", "int64_t sink_end = S;"),
    "fp8_scales_swapped": ("(double)kv->k_scale[h]", "(double)kv->v_scale[h]"),
    "ring_slot_sign": ("ring_offset[b] + p - S", "ring_offset[b] - p + S"),
    "lse_max_dropped": ("*lse = M + log(L);", "*lse = log(L);"),
    "e4m3_subnormal_exponent": ("mag = ldexp((double)m / 8.0, -6);",
                                "mag = ldexp((double)m / 8.0, -7);"),
    "e4m3_bias": ("mag = ldexp(1.0 + (double)m / 8.0, e - 7);",
                  "mag = ldexp(1.0 + (double)m / 8.0, e - 8);"),
    "bf16_shift": ("(uint32_t)bits << 16", "(uint32_t)bits << 15"),
    "page_row_transposed": ("tok = j % kv->page_size;", "tok = (kv->page_size - 1) - j % kv->page_size;"),
    "normaliser_dropped": ("for (d = 0; d < D; ++d) out[d] /= L;", "for (d = 0; d < D; ++d) out[d] /= 1.0;"),
    "value_head_wrong": ("double vs = (kv->dtype == OR_FP8) ? (double)kv->v_scale[h] : 1.0;",
                         "double vs = (kv->dtype == OR_FP8) ? (double)kv->v_scale[0] : 1.0;"),
    "neg_inf_row_not_empty": ("if (M == -INFINITY && !nan_score) {", "if (0) {"),
    "nan_score_not_noted": ("if (isnan(scores[t])) nan_score = 1;", "if (0) nan_score = 1;"),
}


def _nonfinite_case_ok(lib_path):
    """Rows whose visible scores are all -inf (empty rows), partly -inf, and
    -inf mixed with a NaN score (NaN rows), against the brute force."""
    spec = W.VerifySpec(B=3, Hq=4, Hkv=2, D=8, k=2, ctx_lo=10, ctx_hi=10, kv_dtype="f32",
                        q_dtype="f32", page_size=0, log_uniform=False)
    inp = W.make_verify_inputs(spec, 29, keep_logical=True)
    inp.q[..., 0] = -inp.q[..., 0].abs() - 0.5
    n = int(inp.kv_lens[0])
    for t in (inp.k_cache, inp.logical_k):
        t[0, :, :n, 0] = float("inf")
        t[1, :, :n - 2, 0] = float("inf")
        t[2, :, :n, 0] = float("inf")
        t[2, 0, 3, 1] = float("nan")
    o, l = O.verify(inp.q, inp.k_cache, inp.v_cache, inp.kv_lens, 2, inp.sm_scale, lib_path=lib_path)
    with np.errstate(invalid="ignore"):
        bo, bl = brute.verify(inp.q, inp.logical_k, inp.logical_v, inp.kv_lens.tolist(), 2,
                              inp.sm_scale)
    if not (np.array_equal(np.isnan(o), np.isnan(bo)) and np.array_equal(np.isnan(l), np.isnan(bl))
            and np.array_equal(np.isneginf(l), np.isneginf(bl))):
        return False
    fin, lfin = np.isfinite(bo), np.isfinite(bl)
    return bool(np.max(np.abs(o[fin] - bo[fin])) <= 1e-12 and np.max(np.abs(l[lfin] - bl[lfin])) <= 1e-12)


def _battery(lib_path):
    """Return True when the library agrees with every pin in the battery."""
    if not _nonfinite_case_ok(lib_path):
        return False
    for dtype in ("bf16", "fp8"):
        for ps in (0, 4):
            spec = W.VerifySpec(B=3, Hq=4, Hkv=2, D=8, k=3, ctx_lo=1, ctx_hi=30, kv_dtype=dtype,
                                q_dtype="bf16", page_size=ps, spare_pages=2, log_uniform=False)
            inp = W.make_verify_inputs(spec, 17, keep_logical=True)
            o, l = O.verify(inp.q, inp.k_cache, inp.v_cache, inp.kv_lens, 3, inp.sm_scale, ps,
                            inp.block_table, inp.k_scale, inp.v_scale, lib_path=lib_path)
            bo, bl = brute.verify(inp.q, inp.logical_k, inp.logical_v, inp.kv_lens.tolist(), 3,
                                  inp.sm_scale, inp.k_scale, inp.v_scale)
            if not (np.max(np.abs(o - bo)) <= 1e-12 and np.max(np.abs(l - bl)) <= 1e-12):
                return False
        # (2, 5, 1, 6): rings still filling up; (4, 3, 1, 5): fewer positions than sinks
        for S, Wn, lo, hi in ((2, 5, 1, 20), (2, 5, 1, 6), (4, 3, 1, 5)):
            dspec = W.DraftSpec(B=4, Hq=4, Hkv=2, D=8, S=S, W=Wn, steps=3, ctx_lo=lo, ctx_hi=hi,
                                kv_dtype=dtype, q_dtype="bf16", log_uniform=False)
            d = W.make_draft_inputs(dspec, 23, keep_logical=True)
            for step in range(3):
                W.write_step_token(d, step)
                m = d.seq_lens(step)
                o, l = O.draft(d.q[step], d.sink_k, d.sink_v, d.ring_k, d.ring_v, m,
                               d.ring_offset, S, Wn, d.sm_scale, d.k_scale, d.v_scale,
                               lib_path=lib_path)
                bo, bl = brute.draft(d.q[step], d.logical_k, d.logical_v, m.tolist(), S, Wn,
                                     d.sm_scale, d.k_scale, d.v_scale)
                if not (np.max(np.abs(o - bo)) <= 1e-12 and np.max(np.abs(l - bl)) <= 1e-12):
                    return False
    # decoders against torch on every pattern
    for t in (torch.arange(256, dtype=torch.int32).to(torch.uint8).view(torch.float8_e4m3fn),
              torch.arange(0, 1 << 16, 97, dtype=torch.int32).to(torch.int16).view(torch.bfloat16)):
        h = t.view(torch.uint8) if t.dtype == torch.float8_e4m3fn else t
        L = O.lib(lib_path)
        dt = O.DT[O._dtype_name(t)]
        ours = np.array([L.spire_oracle_decode(dt, h.data_ptr(), i) for i in range(t.numel())])
        ref = t.to(torch.float64).numpy()
        if not np.all((np.isnan(ours) & np.isnan(ref)) | (ours == ref)):
            return False
    return True


def _build_variant(tmp_path, name, old, new):
    src = open(O.SRC).read()
    assert old in src, f"mutation anchor for {name} not found"
    path = tmp_path / f"{name}.c"
    path.write_text(src.replace(old, new))
    so = tmp_path / f"lib_{name}.so"
    subprocess.check_call(["gcc", "-O2", "-fopenmp", "-std=c99", "-shared", "-fPIC", str(path),
                           "-o", str(so), "-lm"])
    return str(so)


def test_real_oracle_passes_battery():
    assert _battery(None)


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(tmp_path, name):
    old, new = MUTANTS[name]
    assert not _battery(_build_variant(tmp_path, name, old, new))
