"""GPU parity of token verification (modified rejection sampling): the HIP path
through the C ABI against the CPU oracle on the same seeded inputs.  Every
decision of the step is exact (fp64 accept test, integer inverse CDF), so the
accepted counts and emitted tokens must match the oracle bit for bit, for
every sequence: small ragged vocabularies (one 2048-entry piece, several
pieces with a ragged tail, sizes that are not a multiple of 4), both full-size workloads
(128256-token vocabulary) and the degenerate cases of the method."""
import numpy as np
import pytest
import torch

from oracle import token_verify as TV
from paper_2504_06419_amd import spire
from paper_2504_06419_amd import workloads as W
from tests.gpu_helpers import banner

pytestmark = pytest.mark.gpu
DEV = "cuda"
NW = W.named_workloads()


def _run(p, q, draft, ua, us):
    k = p.shape[1] - 1
    n, tok = spire.token_verify(p, q if k > 0 else None, draft if k > 0 else None,
                                ua if k > 0 else None, us)
    torch.cuda.synchronize()
    return n.cpu().numpy(), tok.cpu().numpy()


def _oracle(p, q, draft, ua, us):
    return TV.verify_tokens(p.cpu().numpy(), q.cpu().numpy(), draft.cpu().numpy(),
                            ua.cpu().numpy(), us.cpu().numpy())


def _compare(inp_or_tuple):
    if isinstance(inp_or_tuple, W.TokenInputs):
        t = inp_or_tuple
        args = (t.p, t.q, t.draft, t.u_accept, t.u_sample)
    else:
        args = inp_or_tuple
    n, tok = _run(*args)
    rn, rtok = _oracle(*args)
    bad = np.nonzero((n != rn) | (tok != rtok).any(axis=1))[0]
    print(f"  sequences={len(n)} mean tokens/round={float((n + 1).mean()):.3f} "
          f"mismatches={len(bad)}", flush=True)
    assert len(bad) == 0, (bad[:8], n[bad[:8]], rn[bad[:8]], tok[bad[:4]], rtok[bad[:4]])
    return n, tok


@pytest.mark.parametrize("V", [1, 7, 1000, 2048, 2049, 8193, 20000, 40964])
@pytest.mark.parametrize("k", [0, 1, 4, 8])
def test_token_verify_small(k, V):
    banner(f"token verify B=64 k={k} V={V}")
    spec = W.TokenSpec(B=64, k=k, V=V, sigma=3.0, eps=0.7)
    _compare(W.make_token_inputs(spec, W.MASTER_SEED + 100 + k * 7 + V, device=DEV))


@pytest.mark.parametrize("name", ["token_verify_B256_k4_V128256", "token_verify_B512_k8_V128256"])
def test_token_verify_full_workloads(name):
    banner(f"token verify workload {name} (every sequence)")
    spec = NW[name]["token"]
    inp = W.make_token_inputs(spec, W.MASTER_SEED + W.WORKLOAD_INDEX[name], device=DEV)
    n, _ = _compare(inp)
    assert 0 < n.mean() < spec.k   # both corrections and bonus tokens occur


def _base(B=48, k=4, V=5000, seed=5):
    spec = W.TokenSpec(B=B, k=k, V=V, sigma=3.0, eps=0.7)
    t = W.make_token_inputs(spec, W.MASTER_SEED + seed, device=DEV)
    return t.p.clone(), t.q.clone(), t.draft.clone(), t.u_accept.clone(), t.u_sample.clone()


def test_token_verify_all_accepted_and_empty_corrections():
    banner("token verify: p == q (all accepted; rejection by u = 1 leaves an empty correction)")
    p, q, d, ua, us = _base()
    q = p[:, :4].contiguous()
    _compare((p, q, d, ua, us))
    ua1 = ua.clone()
    ua1[::2, 1] = 1.0            # p == q but u = 1: rejected, p - q = 0 everywhere
    n, _ = _compare((p, q, d, ua1, us))
    assert (n[::2] == 1).all()


def test_token_verify_degenerate_values():
    banner("token verify: NaN / negative / >1 probabilities, bad tokens, extreme uniforms, zero rows")
    p, q, d, ua, us = _base(B=64)
    p[0, :, 3::11] = float("nan")
    q[1, :, 5::13] = float("nan")
    p[2, :, :100] = -0.25
    p[3, :, 7] = 3.0
    d[4, 0] = -5
    d[5, 2] = 5000               # == V: out of range
    ua[6, :] = float("nan")
    us[7] = 0.0
    us[8] = 1.0
    us[9] = float("nan")
    us[10] = float("inf")
    us[11] = 1.0 - 2.0 ** -24
    us[12] = -3.0
    p[13] = 0.0                  # no mass anywhere: token -1
    q[13] = 0.0
    p[14, 0] = 0.0               # one-hot correction row at the last entry
    p[14, 0, -1] = 1.0
    q[14, 0, -1] = 0.0
    d[14, 0] = 0
    _compare((p, q, d, ua, us))


def test_token_verify_mass_in_last_chunk_and_unaligned_rows():
    banner("token verify: mass only in the ragged last piece; rows not 16-byte aligned")
    p, q, d, ua, us = _base(B=32, V=20000)
    p[:, :, :18432] = 0.0        # only the last, partial 2048-entry piece carries weight
    _compare((p, q, d, ua, us))
    # views offset by one float: V % 4 == 0 but the rows are not 16-byte aligned
    B, kp1, V = p.shape
    pb = torch.empty(B * kp1 * V + 1, dtype=torch.float32, device=DEV)
    qb = torch.empty(B * (kp1 - 1) * V + 1, dtype=torch.float32, device=DEV)
    pu = pb[1:].view(B, kp1, V)
    qu = qb[1:].view(B, kp1 - 1, V)
    pu.copy_(p)
    qu.copy_(q)
    _compare((pu, qu, d, ua, us))


def test_token_verify_is_deterministic():
    banner("token verify: repeated calls give identical results")
    p, q, d, ua, us = _base(B=128, V=128256)
    a = _run(p, q, d, ua, us)
    b = _run(p, q, d, ua, us)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
