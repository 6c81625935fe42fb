"""GPU parity of feedback-memory mixing (paper Sec. 3.3) against the fp64
oracle on the same seeded inputs: every element, fp32 and bf16 activations,
fp32 and bf16 memory vectors, element counts that are and are not multiples
of 4, unaligned views, one to eight draft layers over two to 64 mixed layers,
extreme weights.  The kernel computes in fp32: fp32 output is compared at
max abs error <= 1e-5 * max(1, |m|); bf16 output within one bf16 rounding
(2^-8 relative) of the oracle."""
import numpy as np
import pytest
import torch

from oracle import feedback_memory as FM
from paper_2504_06419_amd import spire
from tests.gpu_helpers import banner

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _check(x, w, out_dtype):
    m = spire.feedback_memory(x, w, out_dtype=out_dtype)
    torch.cuda.synchronize()
    ref = FM.feedback_memory(x.float().cpu().numpy(), w.cpu().numpy())
    got = m.double().cpu().numpy()
    if out_dtype == torch.float32:
        bound = 1e-5 * np.maximum(1.0, np.abs(ref))
    else:
        bound = 2.0 ** -8 * np.abs(ref) + 1e-6
    err = np.abs(got - ref)
    print(f"  max err {float(err.max()):.3e}, worst err/bound {float((err / bound).max()):.3f}", flush=True)
    assert np.all(err <= bound)


@pytest.mark.parametrize("xdt", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("mdt", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("n_out,layers,B,d", [(2, 3, 8, 512), (1, 2, 3, 7), (8, 64, 5, 130),
                                              (4, 9, 17, 4096), (2, 3, 512, 8192)])
def test_feedback_memory_matches_oracle(xdt, mdt, n_out, layers, B, d):
    banner(f"feedback memory x={xdt} m={mdt} n_out={n_out} layers={layers} B={B} d={d}")
    g = torch.Generator(device=DEV).manual_seed(n_out * 1000 + layers * 10 + B + d)
    x = (torch.randn((layers, B, d), generator=g, device=DEV) * 2).to(xdt)
    w = torch.randn((n_out, layers), generator=g, device=DEV) * 3
    _check(x, w, mdt)


def test_feedback_memory_unaligned_views_and_extreme_weights():
    banner("feedback memory: views offset by one element; weights far apart")
    g = torch.Generator(device=DEV).manual_seed(9)
    layers, B, d = 4, 6, 256
    buf = torch.randn(layers * B * d + 1, generator=g, device=DEV)
    x = buf[1:].view(layers, B, d)
    w = torch.tensor([[500.0, -500.0, 0.0, 10.0], [-1e4, -1e4, -1e4, 0.0]], device=DEV)
    _check(x, w, torch.float32)
    out = torch.empty(2 * B * d + 1, device=DEV)[1:].view(2, B, d)
    m = spire.feedback_memory(x, w, out=out)
    torch.cuda.synchronize()
    assert torch.equal(m[1], x[3])             # a dominant weight selects its layer exactly
