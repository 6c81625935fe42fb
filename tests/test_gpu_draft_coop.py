"""GPU parity of draft steps run with whole segments per workgroup: when the
(sequence, KV head) segments number half or a quarter of the device's waves,
each segment gets 2 or 4 waves of one workgroup that split its tiles and merge
their rows in LDS, with no partition and no combine launch.  Every element is
compared with the CPU oracle, and with the stream-K path (kernel choice 2) on
the same inputs: filling rings, lengths below the sink count, empty and
negative lengths, no window, non-finite keys and values."""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2504_06419_amd import spire
from paper_2504_06419_amd import workloads as W
from tests.gpu_helpers import TOL, banner, draft_views, max_err

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _waves() -> int:
    return torch.cuda.get_device_properties(0).multi_processor_count * 4


def _inputs(G, kv_dtype, g, S, Wn, lo, hi, seed, Hkv=8):
    segs = _waves() // G
    assert segs % Hkv == 0
    spec = W.DraftSpec(B=segs // Hkv, Hq=g * Hkv, Hkv=Hkv, D=128, S=S, W=Wn, steps=1, ctx_lo=lo,
                       ctx_hi=hi, kv_dtype=kv_dtype)
    inp = W.make_draft_inputs(spec, seed, device=DEV)
    W.write_step_token(inp, 0)
    return inp


def _lse_err(gpu: torch.Tensor, ref: np.ndarray) -> float:
    """Largest difference of finite entries; NaN and -inf patterns must agree."""
    g = gpu.detach().double().cpu().numpy()
    assert np.array_equal(np.isnan(g), np.isnan(ref)), "NaN-row pattern differs"
    assert np.array_equal(np.isneginf(g), np.isneginf(ref)), "empty-row pattern differs"
    fin = np.isfinite(ref)
    assert np.array_equal(np.isfinite(g), fin)
    return float(np.max(np.abs(g[fin] - ref[fin]))) if fin.any() else 0.0


def _run(inp, lens, kernel, rec=None):
    sink, ring = draft_views(inp)
    s = inp.spec
    out, lse = spire.draft_sparse_attn(inp.q[0].contiguous(), sink, ring, lens, inp.ring_offset, s.S,
                                       s.W, inp.sm_scale, s.Hkv, kernel=kernel,
                                       opts=rec.opts(kernel) if rec is not None else None)
    torch.cuda.synchronize()
    return out, lse


def _oracle(inp, lens):
    s = inp.spec
    return O.draft(inp.q[0], inp.sink_k, inp.sink_v, inp.ring_k, inp.ring_v, lens, inp.ring_offset,
                   s.S, s.W, inp.sm_scale, inp.k_scale, inp.v_scale)


def _check(inp, lens, tol):
    rec = spire.LaunchRecorder(4)
    out, lse = _run(inp, lens, 0, rec)
    names = [nm for nm, _ in rec.collect()]
    assert names == ["draft_partial"], names          # whole segments: no plan, no combine
    ref_o, ref_l = _oracle(inp, lens)
    eo, el = max_err(out, ref_o), _lse_err(lse, ref_l)
    so, sl = _run(inp, lens, 2)                        # the stream-K partition on the same inputs
    es, esl = max_err(out, so.double().cpu().numpy()), _lse_err(lse, sl.double().cpu().numpy())
    print(f"  B={inp.spec.B} max|out-oracle|={eo:.3e} max|lse-oracle|={el:.3e} "
          f"max|out-streamK|={es:.3e} max|lse-streamK|={esl:.3e}", flush=True)
    assert eo <= tol and el <= tol
    # both paths are within tol of the oracle, so within 2 tol of each other
    assert es <= 2 * tol and esl <= 2 * tol
    return out, lse


@pytest.mark.parametrize("G", [2, 4])
@pytest.mark.parametrize("kv_dtype", ["bf16", "fp8"])
@pytest.mark.parametrize("g", [4, 24])
@pytest.mark.parametrize("S,Wn,lo,hi", [(4, 96, 1, 400), (4, 640, 300, 2000), (0, 64, 1, 90),
                                        (8, 0, 1, 12)])
def test_draft_whole_segments(G, kv_dtype, g, S, Wn, lo, hi):
    banner(f"draft whole segments G={G} {kv_dtype} g={g} S={S} W={Wn} ctx=[{lo},{hi}]")
    inp = _inputs(G, kv_dtype, g, S, Wn, lo, hi, 4100 + 7 * G + g + S + Wn)
    _check(inp, inp.seq_lens(0), TOL[kv_dtype])


@pytest.mark.parametrize("G", [2, 4])
def test_draft_whole_segments_degenerate_lengths(G):
    banner(f"draft whole segments G={G}: lengths 0, negative, below S, S, S+1, beyond S+W")
    inp = _inputs(G, "bf16", 4, 4, 96, 1, 400, 4200 + G)
    lens = inp.seq_lens(0).clone()
    lens[0], lens[1], lens[2], lens[3], lens[4], lens[5] = 0, -7, 3, 4, 5, 10 ** 6
    _check(inp, lens, TOL["bf16"])


@pytest.mark.parametrize("G", [2, 4])
def test_draft_whole_segments_nonfinite(G):
    """A NaN value or key in one wave's share makes its rows NaN after the
    merge; keys scoring -inf everywhere leave an empty row (zeros, lse -inf)."""
    banner(f"draft whole segments G={G}: NaN / inf keys and values")
    inp = _inputs(G, "bf16", 4, 4, 96, 200, 400, 4300 + G)
    inp.ring_v[0, 0, 5] = float("nan")        # one value of one wave's share
    inp.ring_k[1, 2, 90] = float("nan")       # a key late in the ring (the last wave's share)
    inp.sink_v[2, 1, 0] = float("inf")        # a sink value: the last wave's share
    lens = inp.seq_lens(0).clone()
    lens[3] = 4                                 # sinks only: one tile in the last wave
    q = inp.q[0]
    q[3, :4] = -1.0                             # KV head 0 of sequence 3: every score -inf
    inp.sink_k[3, 0] = float("inf")
    out, lse = _check(inp, lens, TOL["bf16"])
    assert torch.isnan(out[0, :4]).all() and torch.isnan(out[1, 8:12]).all()
    assert (out[3, :4] == 0).all() and torch.isneginf(lse[3, :4]).all()


def test_draft_bf16_B64_S4_W2048_takes_whole_segments():
    """The bf16 draft workload (64 sequences x 8 KV heads = 512 segments) runs
    with two waves per segment on a 256-CU device; every sampled row matches."""
    if _waves() != 1024:
        pytest.skip("segment / wave ratio is specific to a 256-CU device")
    banner("draft_bf16_B64_S4_W2048 with whole segments per workgroup")
    spec = W.named_workloads()["draft_bf16_B64_S4_W2048"]["draft"]
    inp = W.make_draft_inputs(spec, W.MASTER_SEED + 2, device=DEV)
    ids = [0, 17, 40, 63]
    W.write_step_token(inp, 0)
    lens = inp.seq_lens(0)
    rec = spire.LaunchRecorder(4)
    out, lse = _run(inp, lens, 0, rec)
    assert [nm for nm, _ in rec.collect()] == ["draft_partial"]
    s = inp.spec
    idx = torch.tensor(ids, device=DEV)
    ref_o, ref_l = O.draft(inp.q[0][idx], inp.sink_k[idx], inp.sink_v[idx], inp.ring_k[idx],
                           inp.ring_v[idx], lens[idx], inp.ring_offset[idx], s.S, s.W, inp.sm_scale,
                           inp.k_scale, inp.v_scale)
    eo, el = max_err(out[ids], ref_o), _lse_err(lse[ids], ref_l)
    print(f"  max|out-oracle|={eo:.3e} max|lse-oracle|={el:.3e}", flush=True)
    assert eo <= TOL["bf16"] and el <= TOL["bf16"]
    assert torch.isfinite(out).all()
