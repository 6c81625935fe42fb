"""Pins of the fp64 CPU oracle against things other than itself (no GPU).

The paper prints no attention values, so the oracle is pinned by:
  * a pure-Python brute force over logical positions with an explicit mask;
  * torch's float64 scaled_dot_product_attention with a boolean mask;
  * closed forms (zero query, one or two visible keys, constant values);
  * invariants of the problem (Sec. 2 verify of k+1 tokens, Sec. 3.1 / Sec. 4
    sink + window mask): draft with S+W >= m equals dense, verify query i equals
    a single-query decode over n-k+i keys, masked storage has no effect, paged
    equals contiguous, page order and ring rotation do not matter, grouped heads
    equal repeated heads, and the log-sum-exp split identity;
  * exhaustive dtype decoders checked against torch's conversions and the
    OCP e4m3fn reference values in tests/golden/.
"""
import math
import os

import numpy as np
import pytest
import torch

from oracle import brute
from oracle import oracle as O
from paper_2504_06419_amd import workloads as W

TOL = 1e-12


def vin(B=3, Hq=4, Hkv=2, D=8, k=2, lo=1, hi=30, dtype="bf16", ps=0, spare=2, seed=11,
        poison="nan", log_uniform=False):
    qd = "f32" if dtype == "f32" else "bf16"
    spec = W.VerifySpec(B=B, Hq=Hq, Hkv=Hkv, D=D, k=k, ctx_lo=lo, ctx_hi=hi, kv_dtype=dtype,
                        q_dtype=qd, page_size=ps, spare_pages=spare, log_uniform=log_uniform)
    return W.make_verify_inputs(spec, seed, keep_logical=True, poison=poison)


def oracle_verify(inp, **kw):
    return O.verify(inp.q, inp.k_cache, inp.v_cache, inp.kv_lens, inp.spec.k, inp.sm_scale,
                    inp.spec.page_size, inp.block_table, inp.k_scale, inp.v_scale, **kw)


def din(B=4, Hq=4, Hkv=2, D=8, S=2, Wn=5, steps=3, lo=1, hi=20, dtype="bf16", seed=5,
        poison="nan"):
    qd = "f32" if dtype == "f32" else "bf16"
    spec = W.DraftSpec(B=B, Hq=Hq, Hkv=Hkv, D=D, S=S, W=Wn, steps=steps, ctx_lo=lo, ctx_hi=hi,
                       kv_dtype=dtype, q_dtype=qd, log_uniform=False)
    return W.make_draft_inputs(spec, seed, keep_logical=True, poison=poison)


def oracle_draft(inp, step, **kw):
    s = inp.spec
    return O.draft(inp.q[step], inp.sink_k, inp.sink_v, inp.ring_k, inp.ring_v, inp.seq_lens(step),
                   inp.ring_offset, s.S, s.W, inp.sm_scale, inp.k_scale, inp.v_scale, **kw)


# ---------------------------------------------------------------------------
# decoders
# ---------------------------------------------------------------------------
def test_bf16_decoder_exhaustive():
    bits = torch.arange(0, 1 << 16, dtype=torch.int32).to(torch.int16)
    t = bits.view(torch.bfloat16)
    ours = O.decode(t)
    ref = t.to(torch.float64).numpy()
    both_nan = np.isnan(ours) & np.isnan(ref)
    assert np.all(both_nan | (ours == ref))


def test_e4m3fn_decoder_exhaustive_vs_torch():
    t = torch.arange(0, 256, dtype=torch.int32).to(torch.uint8).view(torch.float8_e4m3fn)
    ours = O.decode(t)
    ref = t.to(torch.float64).numpy()
    both_nan = np.isnan(ours) & np.isnan(ref)
    assert np.all(both_nan | (ours == ref))
    assert np.isnan(ours).sum() == 2  # 0x7F and 0xFF only: e4m3fn has no infinities


def test_e4m3fn_decoder_golden_values():
    """Reference points of the OCP 8-bit floating point specification (e4m3)."""
    path = os.path.join(os.path.dirname(__file__), "golden", "e4m3fn_ocp_values.txt")
    rows = [ln.split() for ln in open(path) if ln.strip() and not ln.startswith("#")]
    bits = torch.tensor([int(r[0], 16) for r in rows], dtype=torch.int32).to(torch.uint8)
    ours = O.decode(bits.view(torch.float8_e4m3fn))
    for (hx, val), got in zip(rows, ours):
        want = float(val)
        if math.isnan(want):
            assert math.isnan(got), hx
        else:
            assert got == want and math.copysign(1, got) == math.copysign(1, want), hx


# ---------------------------------------------------------------------------
# brute force and library cross-checks
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("dtype", ["f32", "bf16", "fp8"])
@pytest.mark.parametrize("g", [1, 2, 4])
@pytest.mark.parametrize("k", [0, 1, 2, 3, 4])
@pytest.mark.parametrize("ps", [0, 4])
def test_verify_matches_brute_force(dtype, g, k, ps):
    inp = vin(Hq=2 * g, Hkv=2, k=k, dtype=dtype, ps=ps, seed=100 + 7 * k + g)
    o, l = oracle_verify(inp)
    bo, bl = brute.verify(inp.q, inp.logical_k, inp.logical_v, inp.kv_lens.tolist(), k,
                          inp.sm_scale, inp.k_scale, inp.v_scale)
    assert np.max(np.abs(o - bo)) <= TOL
    assert np.max(np.abs(l - bl)) <= TOL


@pytest.mark.parametrize("S,Wn", [(2, 5), (0, 5), (4, 0), (3, 1), (1, 64), (0, 1)])
@pytest.mark.parametrize("dtype", ["f32", "bf16", "fp8"])
@pytest.mark.parametrize("hi", [6, 20])
def test_draft_matches_brute_force(S, Wn, dtype, hi):
    inp = din(S=S, Wn=Wn, dtype=dtype, seed=31 + S + Wn, hi=hi)
    for step in range(inp.spec.steps):
        W.write_step_token(inp, step)
        m = inp.seq_lens(step).tolist()
        o, l = oracle_draft(inp, step)
        bo, bl = brute.draft(inp.q[step], inp.logical_k, inp.logical_v, m, S, Wn, inp.sm_scale,
                             inp.k_scale, inp.v_scale)
        assert np.max(np.abs(o - bo)) <= TOL
        assert np.max(np.abs(l - bl)) <= TOL


def test_verify_matches_torch_sdpa_float64():
    inp = vin(B=3, Hq=8, Hkv=2, D=16, k=4, lo=3, hi=40, dtype="f32", ps=4, seed=3)
    o, _ = oracle_verify(inp)
    g = 4
    for b in range(3):
        n = int(inp.kv_lens[b])
        Kb = inp.logical_k[b, :, :n].double().repeat_interleave(g, dim=0)   # [Hq, n, D]
        Vb = inp.logical_v[b, :, :n].double().repeat_interleave(g, dim=0)
        Qb = inp.q[b].double().transpose(0, 1)                                # [Hq, k+1, D]
        i = torch.arange(5).view(-1, 1)
        j = torch.arange(n).view(1, -1)
        mask = j < (n - 4 + i)
        ref = torch.nn.functional.scaled_dot_product_attention(
            Qb, Kb, Vb, attn_mask=mask, scale=inp.sm_scale)                   # [Hq, k+1, D]
        assert np.max(np.abs(o[b] - ref.transpose(0, 1).numpy())) <= TOL


# ---------------------------------------------------------------------------
# closed forms
# ---------------------------------------------------------------------------
def test_zero_query_is_mean_of_visible_values():
    inp = vin(k=3, dtype="f32", ps=4, seed=9)
    inp.q.zero_()
    o, l = oracle_verify(inp)
    for b in range(inp.spec.B):
        n = int(inp.kv_lens[b])
        for i in range(4):
            c = n - 3 + i
            mean = inp.logical_v[b, :, :c].double().mean(dim=1).numpy()       # [Hkv, D]
            for h in range(inp.spec.Hq):
                assert np.max(np.abs(o[b, i, h] - mean[h // 2])) <= TOL
                assert abs(l[b, i, h] - math.log(c)) <= TOL


def test_one_and_two_visible_keys():
    """n = k+1: query 0 sees exactly key 0, query 1 sees keys 0 and 1."""
    inp = vin(k=3, lo=0, hi=0, dtype="f32", seed=4)
    assert all(int(x) == 4 for x in inp.kv_lens)
    o, l = oracle_verify(inp)
    for b in range(inp.spec.B):
        for h in range(inp.spec.Hq):
            hk = h // 2
            q0 = inp.q[b, 0, h].double().numpy()
            k0 = inp.logical_k[b, hk, 0].double().numpy()
            v0 = inp.logical_v[b, hk, 0].double().numpy()
            assert np.max(np.abs(o[b, 0, h] - v0)) == 0.0
            assert abs(l[b, 0, h] - inp.sm_scale * float(q0 @ k0)) <= TOL
            q1 = inp.q[b, 1, h].double().numpy()
            k1 = inp.logical_k[b, hk, 1].double().numpy()
            v1 = inp.logical_v[b, hk, 1].double().numpy()
            dlt = inp.sm_scale * float(q1 @ k1 - q1 @ k0)
            want = (v0 + math.exp(dlt) * v1) / (1.0 + math.exp(dlt))
            assert np.max(np.abs(o[b, 1, h] - want)) <= TOL


@pytest.mark.parametrize("dtype", ["f32", "bf16", "fp8"])
def test_constant_values_give_constant_output(dtype):
    inp = vin(dtype=dtype, ps=4, seed=21, poison="big")
    c = 0.75 if dtype != "fp8" else 96.0   # exactly representable in every dtype
    used = inp.v_cache.float().abs() < 400 if dtype == "fp8" else inp.v_cache.float().abs() < 1e3
    vc = inp.v_cache.float()
    vc[used] = c
    inp.v_cache = vc.to(inp.v_cache.dtype)
    o, _ = oracle_verify(inp)
    scale = inp.v_scale.double().numpy() if dtype == "fp8" else np.ones(inp.spec.Hkv)
    for h in range(inp.spec.Hq):
        assert np.max(np.abs(o[:, :, h] - c * scale[h // 2])) <= 1e-13 * c


# ---------------------------------------------------------------------------
# invariants
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("ps", [0, 4])
def test_verify_query_i_equals_single_query_decode(ps):
    k = 4
    inp = vin(k=k, lo=2, hi=33, ps=ps, dtype="bf16", seed=77)
    o, l = oracle_verify(inp)
    for i in range(k + 1):
        lens = inp.kv_lens - k + i
        oi, li = O.verify(inp.q[:, i:i + 1].contiguous(), inp.k_cache, inp.v_cache, lens, 0,
                          inp.sm_scale, ps, inp.block_table)
        assert np.max(np.abs(o[:, i] - oi[:, 0])) <= TOL
        assert np.max(np.abs(l[:, i] - li[:, 0])) <= TOL


@pytest.mark.parametrize("dtype", ["bf16", "fp8"])
def test_masked_storage_has_no_effect(dtype):
    a = vin(k=3, ps=4, dtype=dtype, seed=13, poison="nan", spare=4)
    b = vin(k=3, ps=4, dtype=dtype, seed=13, poison="big", spare=4)
    oa, la = oracle_verify(a)
    ob, lb = oracle_verify(b)
    assert np.all(np.isfinite(oa))
    assert np.array_equal(oa, ob) and np.array_equal(la, lb)
    da = din(S=2, Wn=6, lo=1, hi=12, dtype=dtype, seed=3, poison="nan")
    db = din(S=2, Wn=6, lo=1, hi=12, dtype=dtype, seed=3, poison="big")
    for step in range(3):
        W.write_step_token(da, step)
        W.write_step_token(db, step)
        x, _ = oracle_draft(da, step)
        y, _ = oracle_draft(db, step)
        assert np.all(np.isfinite(x)) and np.array_equal(x, y)


def test_paged_equals_contiguous():
    a = vin(k=2, ps=0, dtype="bf16", seed=41, lo=1, hi=50)
    b = vin(k=2, ps=4, dtype="bf16", seed=41, lo=1, hi=50)
    assert torch.equal(a.logical_k, b.logical_k)
    oa, la = oracle_verify(a)
    ob, lb = oracle_verify(b)
    assert np.array_equal(oa, ob) and np.array_equal(la, lb)


def test_page_permutation_invariance():
    a = vin(k=2, ps=4, dtype="fp8", seed=43, lo=5, hi=60, spare=5)
    oa, _ = oracle_verify(a)
    P = a.k_cache.shape[0]
    perm = torch.randperm(P, generator=torch.Generator().manual_seed(1))
    inv = torch.empty_like(perm)
    inv[perm] = torch.arange(P)
    a.k_cache = a.k_cache[perm].contiguous()      # new page q holds old page perm[q]
    a.v_cache = a.v_cache[perm].contiguous()
    bt = a.block_table.clone().long()
    ok = bt >= 0
    bt[ok] = inv[bt[ok]]
    a.block_table = bt.to(torch.int32)
    ob, _ = oracle_verify(a)
    assert np.array_equal(oa, ob)


def test_ring_rotation_invariance():
    Wn = 7
    base = din(S=2, Wn=Wn, lo=3, hi=25, dtype="bf16", seed=8)
    W.write_step_token(base, 0)
    ref, _ = oracle_draft(base, 0)
    for r in range(1, Wn):
        rot_k = torch.roll(base.ring_k, shifts=r, dims=2)
        rot_v = torch.roll(base.ring_v, shifts=r, dims=2)
        offs = (base.ring_offset + r) % Wn
        o, _ = O.draft(base.q[0], base.sink_k, base.sink_v, rot_k, rot_v, base.seq_lens(0), offs,
                       2, Wn, base.sm_scale)
        assert np.array_equal(o, ref)


def test_gqa_equals_mha_with_repeated_heads():
    inp = vin(Hq=8, Hkv=2, k=2, ps=0, dtype="bf16", seed=55)
    o, _ = oracle_verify(inp)
    kr = inp.k_cache.repeat_interleave(4, dim=1)
    vr = inp.v_cache.repeat_interleave(4, dim=1)
    om, _ = O.verify(inp.q, kr, vr, inp.kv_lens, 2, inp.sm_scale)
    assert np.array_equal(o, om)


def test_log_sum_exp_split_identity():
    """Attention over A u B equals the lse-weighted merge of attention over A and
    over B -- the identity a split-KV partition relies on."""
    inp = vin(B=2, k=0, lo=20, hi=40, ps=0, dtype="f32", seed=66)
    o, l = oracle_verify(inp)
    for b in range(2):
        n = int(inp.kv_lens[b])
        c = n // 3
        q = inp.q[b:b + 1]
        oa, la = O.verify(q, inp.k_cache[b:b + 1], inp.v_cache[b:b + 1], [c], 0, inp.sm_scale)
        ob, lb = O.verify(q, inp.k_cache[b:b + 1, :, c:], inp.v_cache[b:b + 1, :, c:], [n - c], 0,
                          inp.sm_scale)
        M = np.maximum(la, lb)
        wa, wb = np.exp(la - M), np.exp(lb - M)
        merged = (oa * wa[..., None] + ob * wb[..., None]) / (wa + wb)[..., None]
        assert np.max(np.abs(merged[0] - o[b])) <= TOL
        assert np.max(np.abs(M + np.log(wa + wb) - l[b])) <= TOL


@pytest.mark.parametrize("m_extra", [0, 3, 17])
def test_draft_with_window_covering_context_equals_dense(m_extra):
    """S + W >= m: the StreamingLLM mask keeps every position."""
    S, Wn = 3, 40
    inp = din(S=S, Wn=Wn, lo=1, hi=Wn + S - 4, seed=12 + m_extra, steps=4)
    for step in range(4):
        W.write_step_token(inp, step)
        m = inp.seq_lens(step)
        assert int(m.max()) <= S + Wn
        o, l = oracle_draft(inp, step)
        nmax = inp.logical_k.shape[2]
        q1 = inp.q[step][:, None].contiguous()             # [B, 1, Hq, D]
        od, ld = O.verify(q1, inp.logical_k, inp.logical_v, m, 0, inp.sm_scale)
        assert np.max(np.abs(o - od[:, 0])) <= TOL and np.max(np.abs(l - ld[:, 0])) <= TOL
        assert nmax >= int(m.max())


def test_magicdec_view_of_target_cache_equals_masked_dense():
    """Self-speculation (Sec. 4, MagicDec): the draft reads the target's own
    contiguous cache through a sink + window mask.  The ring is a view of cache
    rows [m-W, m) with ring_offset = (S - m) mod W, the sinks are rows [0, S)."""
    S, Wn = 2, 6
    inp = vin(B=3, Hq=4, Hkv=2, D=8, k=0, lo=15, hi=15, dtype="bf16", ps=0, seed=91)
    m = int(inp.kv_lens[0])
    q = inp.q[:, 0].contiguous()
    sink_k, sink_v = inp.k_cache[:, :, :S], inp.v_cache[:, :, :S]
    ring_k, ring_v = inp.k_cache[:, :, m - Wn:m], inp.v_cache[:, :, m - Wn:m]
    offs = torch.full((3,), (S - m) % Wn, dtype=torch.int32)
    o, _ = O.draft(q, sink_k, sink_v, ring_k, ring_v, inp.kv_lens, offs, S, Wn, inp.sm_scale)
    bo, _ = brute.draft(q, inp.logical_k, inp.logical_v, inp.kv_lens.tolist(), S, Wn, inp.sm_scale)
    assert np.max(np.abs(o - bo)) <= TOL


def test_empty_visible_set_outputs_zero():
    inp = vin(k=2, lo=0, hi=0, dtype="f32", seed=2)
    lens = torch.zeros_like(inp.kv_lens)
    o, l = O.verify(inp.q, inp.k_cache, inp.v_cache, lens, 2, inp.sm_scale)
    assert np.all(o == 0.0) and np.all(np.isneginf(l))


@pytest.mark.parametrize("ps", [0, 4])
def test_nonfinite_visible_keys_match_brute_force(ps):
    """A NaN key or value, or a key scoring +inf, inside the visible range
    makes the rows that see it NaN (output and lse) in the C oracle exactly as
    in the Python brute force; a -inf score weighs zero."""
    inp = vin(B=3, Hq=4, Hkv=2, D=8, k=2, lo=10, hi=10, dtype="f32", ps=ps, seed=21)
    # logical position 4 of sequence 1 (visible to every query) and position 6
    # of sequence 2; the stored copy is located through the same layout
    def put(tensor_s, tensor_l, b, h, p, d, val):
        tensor_l[b, h, p, d] = val
        if ps:
            page = int(inp.block_table[b, p // ps])
            tensor_s[page, h, p % ps, d] = val
        else:
            tensor_s[b, h, p, d] = val
    put(inp.k_cache, inp.logical_k, 1, 0, 4, 3, float("nan"))
    put(inp.v_cache, inp.logical_v, 2, 1, 6, 5, float("nan"))
    put(inp.k_cache, inp.logical_k, 0, 1, 2, 0, float("inf"))
    o, l = oracle_verify(inp)
    with np.errstate(invalid="ignore"):  # inf - inf on purpose
        bo, bl = brute.verify(inp.q, inp.logical_k, inp.logical_v, inp.kv_lens.tolist(), inp.spec.k,
                              inp.sm_scale)
    assert np.isnan(l).any() and np.isfinite(l).any()
    assert np.array_equal(np.isnan(o), np.isnan(bo)) and np.array_equal(np.isnan(l), np.isnan(bl))
    fin, lfin = np.isfinite(bo), np.isfinite(bl)
    assert np.array_equal(np.isfinite(o), fin) and np.array_equal(np.isfinite(l), lfin)
    assert np.max(np.abs(o[fin] - bo[fin])) <= TOL
    assert np.max(np.abs(l[lfin] - bl[lfin])) <= TOL


@pytest.mark.parametrize("ps", [0, 4])
def test_rows_with_all_visible_scores_neg_inf_are_empty_rows(ps):
    """A score of -inf weighs zero, like a masked key, so a row whose visible
    scores are all -inf is an empty row (zeros, lse -inf); one finite visible
    key among -inf scores gives that key's value row and score exactly; -inf
    scores mixed with a NaN score make the row NaN wherever the NaN sits.  The
    C oracle against the brute force and against these closed forms."""
    inp = vin(B=3, Hq=4, Hkv=2, D=8, k=2, lo=10, hi=10, dtype="f32", ps=ps, seed=23)
    n = int(inp.kv_lens[0])          # every sequence holds n = 13 keys; k = 2
    k = inp.spec.k
    # every query has a negative first component, so K[.., 0] = +inf scores -inf
    inp.q[..., 0] = -inp.q[..., 0].abs() - 0.5

    def put(tensor_s, tensor_l, b, h, p, d, val):
        tensor_l[b, h, p, d] = val
        if ps:
            page = int(inp.block_table[b, p // ps])
            tensor_s[page, h, p % ps, d] = val
        else:
            tensor_s[b, h, p, d] = val
    inf, nan = float("inf"), float("nan")
    for h in range(2):                # sequence 0: every key of both heads scores -inf
        for p in range(n):
            put(inp.k_cache, inp.logical_k, 0, h, p, 0, inf)
    for h in range(2):                # sequence 1: the keys query 0 sees score -inf
        for p in range(n - k):
            put(inp.k_cache, inp.logical_k, 1, h, p, 0, inf)
    for p in range(n):                # sequence 2, head 0: -inf everywhere but a NaN key
        put(inp.k_cache, inp.logical_k, 2, 0, p, 0, inf)
    put(inp.k_cache, inp.logical_k, 2, 0, 0, 1, nan)        # first position ...
    for p in range(n):                # ... head 1: the NaN key is the last one query 0 sees
        put(inp.k_cache, inp.logical_k, 2, 1, p, 0, inf)
    put(inp.k_cache, inp.logical_k, 2, 1, n - k - 1, 1, nan)
    o, l = oracle_verify(inp)
    with np.errstate(invalid="ignore"):
        bo, bl = brute.verify(inp.q, inp.logical_k, inp.logical_v, inp.kv_lens.tolist(), k,
                              inp.sm_scale)
    # sequence 0: empty rows
    assert np.all(o[0] == 0.0) and np.all(np.isneginf(l[0]))
    # sequence 1: query 0 empty; query 1 sees exactly one finite key (position n-k)
    assert np.all(o[1, 0] == 0.0) and np.all(np.isneginf(l[1, 0]))
    V = inp.logical_v.double().numpy()
    K = inp.logical_k.double().numpy()
    Q = inp.q.double().numpy()
    for h in range(4):
        hk = h // 2
        assert np.array_equal(o[1, 1, h], V[1, hk, n - k])
        s = inp.sm_scale * float(np.dot(Q[1, 1, h], K[1, hk, n - k]))
        assert abs(l[1, 1, h] - s) <= TOL
    # sequence 2: the NaN key is visible to every row of both heads
    assert np.all(np.isnan(o[2])) and np.all(np.isnan(l[2]))
    # the brute force agrees element by element, pattern and value
    assert np.array_equal(np.isnan(o), np.isnan(bo)) and np.array_equal(np.isnan(l), np.isnan(bl))
    assert np.array_equal(np.isneginf(l), np.isneginf(bl))
    fin, lfin = np.isfinite(bo), np.isfinite(bl)
    assert np.array_equal(np.isfinite(o), fin) and np.array_equal(np.isfinite(l), lfin)
    assert np.max(np.abs(o[fin] - bo[fin])) <= TOL
    assert np.max(np.abs(l[lfin] - bl[lfin])) <= TOL


def test_draft_row_with_all_visible_scores_neg_inf_is_empty():
    """The same reading through the draft's sink + window mask."""
    inp = din(B=2, Hq=4, Hkv=2, D=8, S=2, Wn=5, steps=1, lo=12, hi=12, dtype="f32", seed=24)
    W.write_step_token(inp, 0)
    inp.q[0][..., 0] = -inp.q[0][..., 0].abs() - 0.5
    inp.sink_k[0, :, :, 0] = float("inf")       # sequence 0: sinks and every ring slot
    inp.ring_k[0, :, :, 0] = float("inf")
    inp.logical_k[0, :, :, 0] = float("inf")
    o, l = oracle_draft(inp, 0)
    bo, bl = brute.draft(inp.q[0], inp.logical_k, inp.logical_v, inp.seq_lens(0).tolist(),
                         inp.spec.S, inp.spec.W, inp.sm_scale)
    assert np.all(o[0] == 0.0) and np.all(np.isneginf(l[0]))
    assert np.all(np.isfinite(o[1])) and np.all(np.isfinite(l[1]))
    assert np.array_equal(np.isneginf(l), np.isneginf(bl))
    assert np.max(np.abs(o - bo)) <= TOL
    assert np.max(np.abs(l[1] - bl[1])) <= TOL
