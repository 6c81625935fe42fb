"""A whole speculation round captured in one HIP graph (torch.cuda.CUDAGraph):
the draft steps' sparse attention, the target append of the verified tokens,
the verify attention and the token verification.  The library's calls
allocate nothing, set no memory with memset and never synchronise, so they
can be captured; the graph is replayed several times, with unrelated eager
work and synchronisations in between, and every replay must reproduce the
eager results bit for bit (the kernels are deterministic)."""
import pytest
import torch

from paper_2504_06419_amd import spire
from paper_2504_06419_amd import workloads as W
from tests.gpu_helpers import banner

pytestmark = pytest.mark.gpu
DEV = "cuda"


def test_round_captured_in_a_graph_replays_exactly():
    banner("hip graph: draft steps + kv append + verify + token verification")
    k = 3
    vspec = W.VerifySpec(B=8, Hq=16, Hkv=4, D=128, k=k, ctx_lo=200, ctx_hi=3000, page_size=16,
                         spare_pages=4)
    v = W.make_verify_inputs(vspec, W.MASTER_SEED + 501, device=DEV, poison=None, max_blocks_slack=1)
    dspec = W.DraftSpec(B=8, Hq=16, Hkv=4, D=128, S=4, W=256, steps=k, ctx_lo=200, ctx_hi=3000)
    d = W.make_draft_inputs(dspec, W.MASTER_SEED + 502, device=DEV, poison=None)
    tspec = W.TokenSpec(B=8, k=k, V=20000)
    t = W.make_token_inputs(tspec, W.MASTER_SEED + 503, device=DEV)

    # descriptors hold raw pointers: every tensor they name stays alive here
    kv = spire.kv_view(v.k_cache, v.v_cache, v.block_table, v.page_size)
    sink = spire.kv_view(d.sink_k, d.sink_v)
    ring = spire.kv_view(d.ring_k, d.ring_v)
    gen = torch.Generator(device=DEV).manual_seed(5)
    new_k = torch.randn((vspec.B, k + 1, vspec.Hkv, vspec.D), generator=gen, device=DEV)
    new_v = torch.randn((vspec.B, k + 1, vspec.Hkv, vspec.D), generator=gen, device=DEV)
    pos = (v.kv_lens - (k + 1)).to(torch.int32)   # the round's tokens go where they belong
    qs = [d.q[s].contiguous() for s in range(k)]
    lens = [d.seq_lens(s) for s in range(k)]

    dws = spire.workspace(spire.draft_workspace_size(dspec.B, dspec.Hq, dspec.Hkv, dspec.D))
    vws = spire.workspace(spire.verify_workspace_size(vspec.B, vspec.Hq, vspec.Hkv, vspec.D, k))
    tws = spire.workspace(spire.token_verify_workspace_size(tspec.B, k, tspec.V))
    douts = [torch.empty((dspec.B, dspec.Hq, dspec.D), device=DEV) for _ in range(k)]
    dlses = [torch.empty((dspec.B, dspec.Hq), device=DEV) for _ in range(k)]
    vout = torch.empty((vspec.B, k + 1, vspec.Hq, vspec.D), device=DEV)
    vlse = torch.empty((vspec.B, k + 1, vspec.Hq), device=DEV)
    n_acc = torch.empty((tspec.B,), dtype=torch.int32, device=DEV)
    toks = torch.empty((tspec.B, k + 1), dtype=torch.int32, device=DEV)

    def round_():
        for s in range(k):
            spire.draft_sparse_attn(qs[s], sink, ring, lens[s], d.ring_offset, dspec.S, dspec.W,
                                    d.sm_scale, dspec.Hkv, out=douts[s], lse=dlses[s], ws=dws)
        spire.kv_append(kv, new_k, new_v, pos)
        spire.verify_attn(v.q, kv, v.kv_lens, vspec.Hkv, k, v.sm_scale, out=vout, lse=vlse, ws=vws)
        spire.token_verify(t.p, t.q, t.draft, t.u_accept, t.u_sample, n_acc, toks, tws)

    outputs = lambda: [x.clone() for x in douts + dlses + [vout, vlse, n_acc, toks]]
    round_()
    torch.cuda.synchronize()
    ref = outputs()

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        round_()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        round_()
    torch.cuda.synchronize()

    scratch = torch.zeros(1 << 20, device=DEV)
    for rep in range(4):
        for x in douts + dlses + [vout, vlse]:
            x.fill_(float("nan"))          # the replay must rewrite every output
        n_acc.fill_(-7)
        toks.fill_(-7)
        scratch.add_(1.0)                   # unrelated eager work between replays
        g.replay()
        torch.cuda.synchronize()
        got = outputs()
        same = all(torch.equal(a, b) if a.dtype == torch.int32 else
                   torch.equal(a.view(torch.int32), b.view(torch.int32)) for a, b in zip(got, ref))
        print(f"  replay {rep}: bitwise equal to eager = {same}", flush=True)
        assert same


def test_whole_segment_drafts_and_block_verification_in_a_graph():
    """The draft kernel that gives every segment whole to one workgroup (used
    when the segments number half the device's waves) and block verification,
    captured together: no plan, combine or memset in either, and every replay
    equals the eager run bit for bit."""
    banner("hip graph: whole-segment draft steps + block verification")
    waves = torch.cuda.get_device_properties(0).multi_processor_count * 4
    Hkv, steps = 8, 2
    dspec = W.DraftSpec(B=waves // 2 // Hkv, Hq=4 * Hkv, Hkv=Hkv, D=128, S=4, W=256, steps=steps,
                        ctx_lo=100, ctx_hi=2000)
    d = W.make_draft_inputs(dspec, W.MASTER_SEED + 511, device=DEV, poison=None)
    tspec = W.TokenSpec(B=64, k=4, V=30000)
    t = W.make_token_inputs(tspec, W.MASTER_SEED + 512, device=DEV)
    sink = spire.kv_view(d.sink_k, d.sink_v)
    ring = spire.kv_view(d.ring_k, d.ring_v)
    qs = [d.q[s].contiguous() for s in range(steps)]
    lens = [d.seq_lens(s) for s in range(steps)]
    dws = spire.workspace(spire.draft_workspace_size(dspec.B, dspec.Hq, dspec.Hkv, dspec.D))
    bws = spire.workspace(spire.block_verify_workspace_size(tspec.B, tspec.k, tspec.V))
    douts = [torch.empty((dspec.B, dspec.Hq, dspec.D), device=DEV) for _ in range(steps)]
    dlses = [torch.empty((dspec.B, dspec.Hq), device=DEV) for _ in range(steps)]
    n_acc = torch.empty((tspec.B,), dtype=torch.int32, device=DEV)
    toks = torch.empty((tspec.B, tspec.k + 1), dtype=torch.int32, device=DEV)
    rec = spire.LaunchRecorder(4)
    spire.draft_sparse_attn(qs[0], sink, ring, lens[0], d.ring_offset, dspec.S, dspec.W, d.sm_scale,
                            dspec.Hkv, out=douts[0], lse=dlses[0], ws=dws, opts=rec.opts())
    assert [nm for nm, _ in rec.collect()] == ["draft_partial"]

    def round_():
        for s in range(steps):
            spire.draft_sparse_attn(qs[s], sink, ring, lens[s], d.ring_offset, dspec.S, dspec.W,
                                    d.sm_scale, dspec.Hkv, out=douts[s], lse=dlses[s], ws=dws)
        spire.block_verify(t.p, t.q, t.draft, t.u_accept, t.u_sample, n_acc, toks, bws)

    outputs = lambda: [x.clone() for x in douts + dlses + [n_acc, toks]]
    round_()
    torch.cuda.synchronize()
    ref = outputs()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        round_()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        round_()
    torch.cuda.synchronize()
    scratch = torch.zeros(1 << 20, device=DEV)
    for rep in range(4):
        for x in douts + dlses:
            x.fill_(float("nan"))
        n_acc.fill_(-7)
        toks.fill_(-7)
        scratch.add_(1.0)
        g.replay()
        torch.cuda.synchronize()
        got = outputs()
        same = all(torch.equal(a, b) if a.dtype == torch.int32 else
                   torch.equal(a.view(torch.int32), b.view(torch.int32)) for a, b in zip(got, ref))
        print(f"  replay {rep}: bitwise equal to eager = {same}", flush=True)
        assert same
