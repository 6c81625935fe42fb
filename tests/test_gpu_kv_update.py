"""GPU parity of the KV cache updates: the HIP path (through the C ABI) against
the CPU oracle on the same seeded inputs.  These are byte work, so storage
must match bit for bit: every stored element after spire_kv_append (paged and
contiguous; f32, bf16 and fp8 storage; fp32 and bf16 inputs; NaN, infinities,
saturating and tie values; positions without storage), after sequences of
spire_draft_append calls with spills, and after spire_draft_rollback.  The
full-size fp8 round workload is checked on sampled sequences plus the
property that no byte outside the appended rows changes, and the appended
cache is read back through spire_verify_attn against the attention oracle."""
import numpy as np
import pytest
import torch

from oracle import kv_update as KU
from paper_2504_06419_amd import spire
from paper_2504_06419_amd import workloads as W
from tests.gpu_helpers import TOL, banner, max_err, oracle_verify, run_verify, sample_ids

pytestmark = pytest.mark.gpu
DEV = "cuda"
NPDT = {"f32": np.float32, "bf16": np.uint16, "fp8": np.uint8}


def host_bytes(t: torch.Tensor, dtype: str) -> np.ndarray:
    """Stored elements as numpy (f32 values, bf16 bits, fp8 codes)."""
    t = t.detach().cpu().contiguous()
    if dtype == "f32":
        return t.numpy().copy()
    if dtype == "bf16":
        return t.view(torch.int16).numpy().view(np.uint16).copy()
    return t.view(torch.uint8).numpy().copy()


def special_values(gen, shape):
    """N(0, 3) with NaN, infinities, huge values, fp8 ties and tiny values mixed in."""
    x = torch.randn(shape, generator=gen) * 3
    flat = x.view(-1)
    n = flat.numel()
    idx = torch.randperm(n, generator=gen)[: max(1, n // 8)]
    specials = torch.tensor([float("nan"), float("inf"), -float("inf"), 1e30, -1e30, 500.0, 448.0,
                             1.0625, 1.1875, 2.0 ** -10, 3 * 2.0 ** -10, -0.0, 3.3896e38, 1e-40,
                             1.00390625, 0.0])
    flat[idx] = specials[torch.arange(idx.numel()) % specials.numel()]
    return x


def _paged_cache(gen, dtype, B, Hkv, D, ps, lens, T, spare=3):
    blocks = [(int(n) + T + ps - 1) // ps for n in lens]
    maxb = max(blocks) + 1
    pages = sum(blocks) + spare
    perm = torch.randperm(pages, generator=gen)
    table = torch.full((B, maxb), -1, dtype=torch.int32)
    pos = 0
    for b in range(B):
        table[b, :blocks[b]] = perm[pos:pos + blocks[b]].to(torch.int32)
        pos += blocks[b]
    # one sequence gets no page for its last new token: those writes are skipped
    table[0, blocks[0] - 1] = -1
    dt = W.DTYPES[dtype]
    if dtype == "fp8":
        k = torch.randint(0, 256, (pages, Hkv, ps, D), generator=gen, dtype=torch.uint8).view(dt)
        v = torch.randint(0, 256, (pages, Hkv, ps, D), generator=gen, dtype=torch.uint8).view(dt)
    else:
        k = torch.randn((pages, Hkv, ps, D), generator=gen).to(dt)
        v = torch.randn((pages, Hkv, ps, D), generator=gen).to(dt)
    return k.to(DEV), v.to(DEV), table


def _on_device(x, offset):
    """x on the GPU, `offset` elements past an aligned allocation (offset 1
    misaligns the rows for the 4-element vector path)."""
    if offset == 0:
        return x.to(DEV).contiguous()
    buf = torch.empty((x.numel() + offset,), dtype=x.dtype, device=DEV)
    out = buf[offset:].view(x.shape)
    out.copy_(x.to(DEV))
    return out


@pytest.mark.parametrize("dtype", ["f32", "bf16", "fp8"])
@pytest.mark.parametrize("src", ["f32", "bf16"])
@pytest.mark.parametrize("paged", [True, False])
def test_kv_append_matches_oracle(dtype, src, paged):
    _kv_append_case(dtype, src, paged)


# the element-by-element path: head dims that are not a multiple of 4, and
# inputs that do not start on a 4-element boundary
@pytest.mark.parametrize("dtype", ["f32", "bf16", "fp8"])
@pytest.mark.parametrize("paged", [True, False])
@pytest.mark.parametrize("D,offset", [(30, 0), (128, 1)])
def test_kv_append_scalar_path_matches_oracle(dtype, paged, D, offset):
    _kv_append_case(dtype, "f32", paged, D=D, offset=offset)


def _kv_append_case(dtype, src, paged, D=128, offset=0):
    banner(f"kv append storage={dtype} input={src} paged={paged} D={D} input offset={offset}")
    gen = torch.Generator().manual_seed(300 + 7 * len(dtype) + len(src) + int(paged) + D + offset)
    B, Hkv, T, ps = 6, 2, 5, 16
    lens = torch.randint(0, 40, (B,), generator=gen)
    lens[1] = -3          # negative start: the first positions are skipped
    kn = special_values(gen, (B, T, Hkv, D))
    vn = special_values(gen, (B, T, Hkv, D))
    if src == "bf16":
        kn, vn = kn.to(torch.bfloat16), vn.to(torch.bfloat16)
    ks = vs = None
    if dtype == "fp8":
        ks = (0.5 + torch.rand(Hkv, generator=gen)).to(torch.float32)
        vs = (0.5 + torch.rand(Hkv, generator=gen)).to(torch.float32)
    # the descriptor holds raw device pointers: keep those tensors alive
    ks_d = None if ks is None else ks.to(DEV)
    vs_d = None if vs is None else vs.to(DEV)
    if paged:
        kc, vc, table = _paged_cache(gen, dtype, B, Hkv, D, ps, lens.clamp_min(0).tolist(), T)
        table_d = table.to(DEV)
        view = spire.kv_view(kc, vc, table_d, ps, ks_d, vs_d)
    else:
        cap = 36        # some appended positions fall beyond the capacity
        dt = W.DTYPES[dtype]
        if dtype == "fp8":
            kc = torch.randint(0, 256, (B, Hkv, cap, D), generator=gen, dtype=torch.uint8).view(dt).to(DEV)
            vc = torch.randint(0, 256, (B, Hkv, cap, D), generator=gen, dtype=torch.uint8).view(dt).to(DEV)
        else:
            kc = torch.randn((B, Hkv, cap, D), generator=gen).to(dt).to(DEV)
            vc = torch.randn((B, Hkv, cap, D), generator=gen).to(dt).to(DEV)
        table = None
        view = spire.kv_view(kc, vc, k_scale=ks_d, v_scale=vs_d)
    hk, hv = host_bytes(kc, dtype), host_bytes(vc, dtype)
    spire.kv_append(view, _on_device(kn, offset), _on_device(vn, offset), lens.to(torch.int32).to(DEV))
    torch.cuda.synchronize()
    KU.kv_append(hk, hv, kn.float().numpy(), vn.float().numpy(), lens.numpy(), dtype,
                 ps if paged else 0, None if table is None else table.numpy(),
                 None if ks is None else ks.numpy(), None if vs is None else vs.numpy())
    gk, gv = host_bytes(kc, dtype), host_bytes(vc, dtype)
    # f32 storage: compare bit patterns so that NaN payloads count too
    if dtype == "f32":
        gk, gv, hk, hv = (a.view(np.uint32) for a in (gk, gv, hk, hv))
    bad = int((gk != hk).sum() + (gv != hv).sum())
    print(f"  mismatching elements: {bad}", flush=True)
    assert bad == 0


def _draft_cache(gen, dtype, B, Hkv, D, S, Wn):
    dt = W.DTYPES[dtype]
    if dtype == "fp8":
        mk = lambda n: torch.randint(0, 256, (B, Hkv, n, D), generator=gen, dtype=torch.uint8).view(dt)
    else:
        mk = lambda n: torch.randn((B, Hkv, n, D), generator=gen).to(dt)
    return [mk(S).to(DEV), mk(S).to(DEV), mk(Wn).to(DEV), mk(Wn).to(DEV)]


@pytest.mark.parametrize("dtype", ["bf16", "fp8", "f32"])
@pytest.mark.parametrize("S,Wn,lo,hi", [(4, 64, 100, 200), (4, 64, 1, 40), (0, 16, 1, 30),
                                        (2, 2, 1, 20), (3, 0, 1, 6)])
def test_draft_append_and_rollback_match_oracle(dtype, S, Wn, lo, hi):
    _draft_case(dtype, S, Wn, lo, hi)


# the element-by-element path (head dim not a multiple of 4; misaligned inputs)
@pytest.mark.parametrize("dtype", ["bf16", "fp8", "f32"])
@pytest.mark.parametrize("D,offset", [(30, 0), (64, 1)])
def test_draft_append_and_rollback_scalar_path_match_oracle(dtype, D, offset):
    _draft_case(dtype, 4, 16, 1, 40, D=D, offset=offset)


def _draft_case(dtype, S, Wn, lo, hi, D=64, offset=0):
    banner(f"draft append + rollback storage={dtype} S={S} W={Wn} lengths [{lo}, {hi}] D={D} "
           f"input offset={offset}")
    gen = torch.Generator().manual_seed(900 + S * 31 + Wn + lo + D + offset)
    B, Hkv, k = 9, 2, 4
    base = torch.randint(lo, hi + 1, (B,), generator=gen, dtype=torch.int32)
    offs = torch.randint(0, max(Wn, 1), (B,), generator=gen, dtype=torch.int32)
    offs[0] = -7 if Wn > 0 else 0            # reduced modulo W on the device
    store = _draft_cache(gen, dtype, B, Hkv, D, S, Wn)
    host = [host_bytes(t, dtype) for t in store]
    ks = vs = None
    if dtype == "fp8":
        ks = (0.5 + torch.rand(Hkv, generator=gen)).to(DEV)
        vs = (0.5 + torch.rand(Hkv, generator=gen)).to(DEV)
    sink = spire.kv_view(store[0], store[1], k_scale=ks, v_scale=vs)
    ring = spire.kv_view(store[2], store[3], k_scale=ks, v_scale=vs)
    spk = torch.zeros((k, B, Hkv, D), dtype=W.DTYPES[dtype], device=DEV)
    spv = torch.zeros_like(spk)
    hspk = np.zeros((k, B, Hkv, D), NPDT[dtype])
    hspv = np.zeros_like(hspk)
    news = [(special_values(gen, (B, Hkv, D)), special_values(gen, (B, Hkv, D))) for _ in range(k)]
    offs_np = offs.numpy() % max(Wn, 1)
    for s in range(k):
        kn, vn = news[s]
        lens = (base + s + 1).to(DEV)
        spire.draft_append(sink, ring, _on_device(kn, offset), _on_device(vn, offset), lens, offs.to(DEV),
                           S, Wn, spk[s], spv[s])
        KU.draft_append(*host, kn.numpy(), vn.numpy(), (base + s + 1).numpy(), offs_np, S, Wn, dtype,
                        None if ks is None else ks.cpu().numpy(), None if vs is None else vs.cpu().numpy(),
                        hspk[s], hspv[s])
    torch.cuda.synchronize()
    view = (lambda a: a.view(np.uint32)) if dtype == "f32" else (lambda a: a)
    for g, h in zip(store + [spk, spv], host + [hspk, hspv]):
        assert np.array_equal(view(host_bytes(g, dtype)), view(h))
    n_acc = torch.randint(0, k + 1, (B,), generator=gen, dtype=torch.int32)
    spire.draft_rollback(sink, ring, spk, spv, base.to(DEV), n_acc.to(DEV), offs.to(DEV), S, Wn)
    KU.draft_rollback(*host, hspk, hspv, base.numpy(), n_acc.numpy(), k, offs_np, S, Wn)
    torch.cuda.synchronize()
    for g, h in zip(store, host):
        assert np.array_equal(view(host_bytes(g, dtype)), view(h))
    print(f"  accepted {n_acc.tolist()}: storage bit-exact after {k} writes and the rollback", flush=True)


def test_round_fp8_append_full_size():
    """The k+1 = 9 verified tokens of the fp8 round workload (B=512, 8 KV heads,
    16-token pages) appended after each sequence's context: sampled rows
    against the oracle, every other byte unchanged, and the grown cache read
    back through the verify attention."""
    banner("kv append: round_fp8_B512_k8 full size")
    name = "round_fp8_B512_k8"
    spec = W.named_workloads()[name]["verify"]
    inp = W.make_verify_inputs(spec, W.MASTER_SEED + W.WORKLOAD_INDEX[name], device=DEV, poison=None,
                               max_blocks_slack=1)
    B, Hkv, D, T = spec.B, spec.Hkv, spec.D, spec.k + 1
    gen = torch.Generator(device=DEV).manual_seed(77)
    kn = torch.randn((B, T, Hkv, D), generator=gen, device=DEV, dtype=torch.float32) * 5
    vn = torch.randn((B, T, Hkv, D), generator=gen, device=DEV, dtype=torch.float32) * 5
    # grow each sequence by T: give every sequence the pages it needs (fresh pages at the end)
    ps = inp.page_size
    lens = inp.kv_lens.cpu()
    table = inp.block_table.cpu().clone()
    pages = inp.k_cache.shape[0]
    need = []
    for b in range(B):
        have = (int(lens[b]) + ps - 1) // ps
        want = (int(lens[b]) + T + ps - 1) // ps
        for blk in range(have, want):
            table[b, blk] = pages + len(need)
            need.append((b, blk))
    extra = len(need)
    kc = torch.cat([inp.k_cache, torch.zeros((extra,) + tuple(inp.k_cache.shape[1:]), dtype=inp.k_cache.dtype,
                                             device=DEV)])
    vc = torch.cat([inp.v_cache, torch.zeros_like(kc[:extra])])
    k0, v0 = kc.view(torch.uint8).clone(), vc.view(torch.uint8).clone()
    table = table.to(DEV)
    view = spire.kv_view(kc, vc, table, ps, inp.k_scale, inp.v_scale)
    spire.kv_append(view, kn, vn, inp.kv_lens)
    torch.cuda.synchronize()
    # every byte outside the appended rows is unchanged: put the old bytes back
    # into the appended rows of a copy, which must then equal the old storage
    pos = inp.kv_lens.long()[:, None] + torch.arange(T, device=DEV)[None]
    pgf = table.long().gather(1, pos // ps).reshape(-1)
    rwf = (pos % ps).reshape(-1)
    for cur, old in ((kc, k0), (vc, v0)):
        c = cur.view(torch.uint8).clone()
        c[pgf, :, rwf] = old[pgf, :, rwf]
        assert torch.equal(c, old)
        del c
    # sampled sequences: the written rows are the oracle's codes
    ids = sample_ids(lens.tolist(), 6)
    ksc, vsc = inp.k_scale.cpu().numpy(), inp.v_scale.cpu().numpy()
    for b in ids:
        for t in range(T):
            j = int(lens[b]) + t
            page, row = int(table[b, j // ps]), j % ps
            for h in range(Hkv):
                got_k = kc[page, h, row].view(torch.uint8).cpu().numpy()
                got_v = vc[page, h, row].view(torch.uint8).cpu().numpy()
                assert np.array_equal(got_k, KU.to_storage(kn[b, t, h].cpu().numpy(), "fp8", ksc[h]))
                assert np.array_equal(got_v, KU.to_storage(vn[b, t, h].cpu().numpy(), "fp8", vsc[h]))
    # the grown cache through the verify attention (k = 8 rows over n + 9 keys)
    inp.k_cache, inp.v_cache, inp.block_table = kc, vc, table
    inp.kv_lens = (inp.kv_lens + T).to(torch.int32)
    out, lse = run_verify(inp)
    ref_o, _ = oracle_verify(inp, ids)
    err = max_err(out[ids], ref_o)
    print(f"  sampled {ids}: appended rows bit-exact; verify over the grown cache max err {err:.2e}",
          flush=True)
    assert err <= TOL["fp8"]
