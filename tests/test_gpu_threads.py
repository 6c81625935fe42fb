"""Reentrancy of the C ABI: the library keeps no per-call state, so two host
threads, each with its own stream, workspace and outputs, may call it at the
same time; every result must equal, bit for bit, the one of a serial call."""
import threading

import pytest
import torch

from paper_2504_06419_amd import spire
from paper_2504_06419_amd import workloads as W
from tests.gpu_helpers import banner, draft_views

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _verify_call(inp, kernel):
    s = inp.spec
    kv = spire.kv_view(inp.k_cache, inp.v_cache, inp.block_table, inp.page_size, inp.k_scale, inp.v_scale)
    ws = spire.workspace(spire.verify_workspace_size(s.B, s.Hq, s.Hkv, s.D, s.k))
    out = torch.empty((s.B, s.k + 1, s.Hq, s.D), dtype=torch.float32, device=DEV)
    lse = torch.empty((s.B, s.k + 1, s.Hq), dtype=torch.float32, device=DEV)

    def call():
        spire.verify_attn(inp.q, kv, inp.kv_lens, s.Hkv, s.k, inp.sm_scale, out=out, lse=lse, ws=ws,
                          kernel=kernel)
        return out, lse
    return call


def _draft_call(inp):
    s = inp.spec
    sink, ring = draft_views(inp)
    ws = spire.workspace(spire.draft_workspace_size(s.B, s.Hq, s.Hkv, s.D))
    out = torch.empty((s.B, s.Hq, s.D), dtype=torch.float32, device=DEV)
    lse = torch.empty((s.B, s.Hq), dtype=torch.float32, device=DEV)
    q, lens = inp.q[0].contiguous(), inp.seq_lens(0)

    def call():
        spire.draft_sparse_attn(q, sink, ring, lens, inp.ring_offset, s.S, s.W, inp.sm_scale, s.Hkv, out=out,
                                lse=lse, ws=ws)
        return out, lse
    return call


def test_two_threads_on_two_streams_equal_serial_calls():
    banner("two host threads, two streams, own workspaces vs serial calls")
    v1 = W.make_verify_inputs(W.VerifySpec(B=24, Hq=32, Hkv=8, D=128, k=4, ctx_lo=100, ctx_hi=6000,
                                           page_size=16, spare_pages=4), 31, device=DEV)
    v2 = W.make_verify_inputs(W.VerifySpec(B=16, Hq=64, Hkv=8, D=128, k=8, ctx_lo=200, ctx_hi=5000,
                                           kv_dtype="fp8", page_size=16), 32, device=DEV)
    d = W.make_draft_inputs(W.DraftSpec(B=20, Hq=32, Hkv=8, D=128, S=4, W=512, steps=1, ctx_lo=100,
                                        ctx_hi=3000), 33, device=DEV)
    W.write_step_token(d, 0)
    # thread 0: bf16 verify (register-staged) and the draft step; thread 1: fp8
    # 72-row verify (LDS-staged) and the generic kernel on the bf16 batch
    jobs = [[_verify_call(v1, 0), _draft_call(d)], [_verify_call(v2, 0), _verify_call(v1, 1)]]
    serial = []
    for calls in jobs:
        res = []
        for c in calls:
            o, l = c()
            torch.cuda.synchronize()
            res.append((o.clone(), l.clone()))
        serial.append(res)

    results = [None, None]
    errors = []

    def worker(t):
        try:
            torch.cuda.set_device(0)
            st = torch.cuda.Stream()
            got = []
            with torch.cuda.stream(st):
                for _ in range(4):
                    for c in jobs[t]:
                        c()
                st.synchronize()
                for c in jobs[t]:
                    o, l = c()
                    st.synchronize()
                    got.append((o.clone(), l.clone()))
            results[t] = got
        except Exception as e:  # reported by the main thread
            errors.append(e)

    threads = [threading.Thread(target=worker, args=(t,)) for t in range(2)]
    for th in threads:
        th.start()
    for th in threads:
        th.join(timeout=120)
    assert not errors, errors
    for t in range(2):
        assert results[t] is not None
        for (o, l), (so, sl) in zip(results[t], serial[t]):
            assert torch.equal(o, so) and torch.equal(l, sl)
