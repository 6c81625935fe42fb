"""C ABI checks that need no GPU: the library loads, exports every function
include/spire.h declares, and rejects invalid arguments on the host before
enqueueing anything (no device pointer is dereferenced on these paths)."""
import ctypes as C
import os
import re
import subprocess

import pytest

from paper_2504_06419_amd import spire

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "spire.h")

OK, INVALID, UNSUPPORTED, WORKSPACE, HIPERR = 0, 1, 2, 3, 4
FAKE = 0x10000  # a 256-byte-aligned non-null address; never dereferenced here


def header_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(spire_[a-z_]+)\s*\(", src)))


def test_header_declares_the_binding_symbols():
    assert header_functions() == sorted(spire.SYMBOLS)


def test_library_exports_every_declared_symbol():
    L = spire.load()
    for name in header_functions():
        assert hasattr(L, name), name
    out = subprocess.run(["nm", "-D", "--defined-only", spire.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\sT\s(spire_\w+)", out))
    assert set(header_functions()) <= exported


def test_version_and_status_strings():
    L = spire.load()
    assert L.spire_version() == 1
    for code, name in spire.STATUS.items():
        assert L.spire_status_string(code).decode() == name
    assert L.spire_status_string(99).decode() == "SPIRE_ERR_UNKNOWN"


def kv(dtype=spire.BF16, page_size=0, capacity=64, table=None, scales=False, reserved=0):
    d = spire.KV()
    d.k, d.v = FAKE, FAKE
    d.block_table = table
    d.k_scale = FAKE if scales else None
    d.v_scale = FAKE if scales else None
    d.s_blk, d.s_head, d.s_tok = 8 * capacity * 128, capacity * 128, 128
    d.dtype, d.page_size = dtype, page_size
    d.max_blocks = 4 if table else 0
    d.num_blocks = 16 if table else 0
    d.capacity = capacity
    d.reserved = reserved
    return d


def verify(**kw):
    a = dict(q=FAKE, q_dtype=spire.BF16, kv=kv(), lens=FAKE, B=2, Hq=32, Hkv=8, D=128, k=4,
             out=FAKE, out_dtype=spire.F32, lse=None, ws=FAKE, ws_bytes=1 << 30)
    a.update(kw)
    L = spire.load()
    kvp = None if a["kv"] is None else C.byref(a["kv"])
    return L.spire_verify_attn(a["q"], a["q_dtype"], kvp, a["lens"], a["B"], a["Hq"], a["Hkv"],
                               a["D"], a["k"], a.get("sm_scale", 0.1), a["out"], a["out_dtype"],
                               a["lse"], a["ws"], a["ws_bytes"], None)


def draft(**kw):
    a = dict(q=FAKE, q_dtype=spire.BF16, sink=kv(capacity=4), ring=kv(capacity=64), lens=FAKE,
             offs=FAKE, B=2, Hq=32, Hkv=8, D=128, S=4, W=64, out=FAKE, ws=FAKE)
    a.update(kw)
    L = spire.load()
    return L.spire_draft_sparse_attn(a["q"], a["q_dtype"], C.byref(a["sink"]), C.byref(a["ring"]),
                                     a["lens"], a["offs"], a["B"], a["Hq"], a["Hkv"], a["D"],
                                     a["S"], a["W"], a.get("sm_scale", 0.1), a["out"], spire.F32,
                                     None, a["ws"],
                                     1 << 30, None)


@pytest.mark.parametrize("kw,status", [
    (dict(B=-1), INVALID),
    (dict(Hq=30), INVALID),
    (dict(Hkv=0), INVALID),
    (dict(D=96), UNSUPPORTED),
    (dict(k=16), UNSUPPORTED),
    (dict(k=-1), UNSUPPORTED),
    (dict(Hq=128, Hkv=1, k=1), UNSUPPORTED),        # (k+1) * g = 256 rows
    (dict(q_dtype=spire.FP8), UNSUPPORTED),
    (dict(out_dtype=spire.FP8), UNSUPPORTED),
    (dict(q=None), INVALID),
    (dict(out=None), INVALID),
    (dict(ws=None), WORKSPACE),
    (dict(ws=FAKE + 16), WORKSPACE),                  # not 256-byte aligned
    (dict(q=FAKE + 2), INVALID),                      # not 16-byte aligned
    (dict(kv=None), INVALID),
    (dict(kv=kv(dtype=7)), INVALID),
    (dict(kv=kv(reserved=1)), INVALID),
    (dict(kv=kv(dtype=spire.FP8)), INVALID),          # fp8 without scales
    (dict(kv=kv(page_size=16)), INVALID),             # paged without a block table
    (dict(kv=kv(capacity=0)), INVALID),
    (dict(lens=None), INVALID),
    (dict(B=9000), UNSUPPORTED),
    (dict(sm_scale=0.0), INVALID),                   # kernels need a positive scale
    (dict(sm_scale=-0.1), INVALID),
    (dict(sm_scale=float("nan")), INVALID),
    (dict(sm_scale=float("inf")), INVALID),
])
def test_verify_rejects_invalid_arguments(kw, status):
    assert verify(**kw) == status
    assert spire.load().spire_last_error().decode() != ""


def test_verify_empty_batch_is_a_no_op():
    assert verify(B=0, q=None, out=None, ws=None, lens=None) == OK


@pytest.mark.parametrize("kw,status", [
    (dict(S=0, W=0), INVALID),
    (dict(S=-1), INVALID),
    (dict(S=8), INVALID),                            # sink capacity 4 < S
    (dict(W=128), INVALID),                          # ring capacity 64 < W
    (dict(sink=kv(dtype=spire.F32, capacity=4)), INVALID),   # dtypes differ
    (dict(ring=kv(page_size=16, table=FAKE)), UNSUPPORTED),  # paged ring
    (dict(lens=None), INVALID),
    (dict(offs=None), INVALID),
    (dict(D=80), UNSUPPORTED),
    (dict(sm_scale=-1.0), INVALID),
])
def test_draft_rejects_invalid_arguments(kw, status):
    assert draft(**kw) == status


def test_invalid_sizes_give_zero_workspace():
    L = spire.load()
    assert L.spire_verify_workspace_size(4, 30, 8, 128, 4) == 0
    assert L.spire_draft_workspace_size(4, 32, 0, 128) == 0


def _opts(kernel=0, max_launches=0, events=None, reserved=0):
    o = spire.LaunchOpts()
    o.kernel, o.max_launches, o.events, o.reserved = kernel, max_launches, events, reserved
    n = C.c_int32(-7)
    o.n_launches = C.addressof(n)
    return o, n


@pytest.mark.parametrize("kw", [dict(kernel=4), dict(kernel=-1), dict(max_launches=-1),
                                dict(max_launches=2), dict(reserved=1)])
def test_invalid_launch_options_are_rejected(kw):
    """Per-call options are checked before anything is enqueued (events NULL
    with max_launches > 0, unknown kernel family, reserved field); the launch
    count reads 0."""
    L = spire.load()
    for call in ("verify", "draft", "token"):
        o, n = _opts(**kw)
        if call == "verify":
            rc = L.spire_verify_attn_ex(FAKE, spire.BF16, C.byref(kv()), FAKE, 2, 32, 8, 128, 4, 0.1, FAKE,
                                        spire.F32, None, FAKE, 1 << 30, None, C.byref(o))
        elif call == "draft":
            rc = L.spire_draft_sparse_attn_ex(FAKE, spire.BF16, C.byref(kv(capacity=4)), C.byref(kv()), FAKE,
                                              FAKE, 2, 32, 8, 128, 4, 64, 0.1, FAKE, spire.F32, None, FAKE,
                                              1 << 30, None, C.byref(o))
        else:
            rc = L.spire_token_verify_ex(FAKE, FAKE, FAKE, FAKE, FAKE, 2, 4, 1000, FAKE, FAKE, FAKE, 1 << 20,
                                         None, C.byref(o))
        assert rc == INVALID, (call, kw)
        assert n.value == 0
        assert "opts" in L.spire_last_error().decode()


def test_library_has_no_mutable_globals_besides_the_device_cache():
    """The boundary is stateless: apart from the per-device compute-unit cache
    (and its mutex), the thread-local error message and the device scratch of
    the no-allocation entry point with its per-device address, the library's
    host code keeps no writable data symbols."""
    out = subprocess.run(["nm", "-C", "--defined-only", spire.LIB_PATH], capture_output=True, text=True,
                         check=True).stdout
    # the no-allocation entry point's device scratch (a host stand-in here) and
    # its per-device address, set once
    allowed = ("g_cus", "g_dev_mu", "g_err", "scratch", "g_scratch")
    writable = []
    for ln in out.splitlines():
        parts = ln.split(None, 2)
        if len(parts) != 3 or parts[1] not in ("B", "b", "D", "d"):
            continue
        name = parts[2]
        if "(" in name.replace("(anonymous namespace)", ""):
            continue  # host-side handles of the kernels, not state
        if name.startswith(("spire", "(anonymous namespace)")):
            writable.append(name)
    assert any("g_cus" in w for w in writable)  # the scan sees the library's own data
    bad = [w for w in writable if not any(a in w for a in allowed)]
    assert not bad, bad


def token(**kw):
    a = dict(p=FAKE, q=FAKE, draft=FAKE, ua=FAKE, us=FAKE, B=2, k=4, V=1000, n=FAKE, out=FAKE,
             ws=FAKE, ws_bytes=1 << 20)
    a.update(kw)
    return spire.load().spire_token_verify(a["p"], a["q"], a["draft"], a["ua"], a["us"], a["B"],
                                           a["k"], a["V"], a["n"], a["out"], a["ws"], a["ws_bytes"],
                                           None)


@pytest.mark.parametrize("kw,status", [
    (dict(B=-1), UNSUPPORTED),
    (dict(B=70000), UNSUPPORTED),
    (dict(k=-1), UNSUPPORTED),
    (dict(k=33), UNSUPPORTED),
    (dict(V=0), UNSUPPORTED),
    (dict(V=(1 << 20) + 1), UNSUPPORTED),
    (dict(p=None), INVALID),
    (dict(us=None), INVALID),
    (dict(n=None), INVALID),
    (dict(out=None), INVALID),
    (dict(q=None), INVALID),                  # k > 0 needs the draft side
    (dict(draft=None), INVALID),
    (dict(ua=None), INVALID),
    (dict(p=FAKE + 2), INVALID),              # not 4-byte aligned
    (dict(ws=None), WORKSPACE),
    (dict(ws=FAKE + 16), WORKSPACE),
    (dict(ws_bytes=8), WORKSPACE),
])
def test_token_verify_rejects_invalid_arguments(kw, status):
    assert token(**kw) == status
    assert spire.load().spire_last_error().decode() != ""


def test_token_verify_sizes_and_empty_batch():
    L = spire.load()
    # one 8-byte sum per 2048-entry piece and sequence plus one 4-byte count per
    # sequence, each part rounded up to 256 bytes
    assert L.spire_token_verify_workspace_size(256, 4, 128256) == 256 * 63 * 8 + 1280
    assert L.spire_token_verify_workspace_size(3, 0, 1) == 512
    assert L.spire_token_verify_workspace_size(2, 33, 10) == 0
    assert L.spire_token_verify_workspace_size(2, 4, 0) == 0
    assert token(B=0, p=None, q=None, draft=None, ua=None, us=None, n=None, out=None, ws=None) == OK
    # k = 0: the draft side may be absent
    assert token(k=0, q=None, draft=None, ua=None, ws_bytes=0) == WORKSPACE


def _append(**kw):
    a = dict(kv=kv(), k=FAKE, v=FAKE, dt=spire.F32, pos=FAKE, B=2, Hkv=8, D=128, T=5)
    a.update(kw)
    return spire.load().spire_kv_append(C.byref(a["kv"]), a["k"], a["v"], a["dt"], a["pos"], a["B"],
                                        a["Hkv"], a["D"], a["T"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(B=-1), INVALID),
    (dict(T=-1), INVALID),
    (dict(Hkv=0), INVALID),
    (dict(k=None), INVALID),
    (dict(pos=None), INVALID),
    (dict(dt=spire.FP8), UNSUPPORTED),               # new K/V must be f32 or bf16
    (dict(D=0), UNSUPPORTED),
    (dict(D=2000), UNSUPPORTED),
    (dict(k=FAKE + 2), INVALID),                      # f32 input not 4-byte aligned
    (dict(kv=kv(dtype=spire.FP8)), INVALID),          # fp8 storage without scales
    (dict(kv=kv(page_size=16)), INVALID),             # paged without a block table
    (dict(kv=kv(reserved=1)), INVALID),
])
def test_kv_append_rejects_invalid_arguments(kw, status):
    assert _append(**kw) == status
    assert spire.load().spire_last_error().decode() != ""


def test_kv_append_empty_is_a_no_op():
    assert _append(B=0, k=None, v=None, pos=None) == OK
    assert _append(T=0, k=None, v=None, pos=None) == OK


def _dappend(**kw):
    a = dict(sink=kv(capacity=4), ring=kv(capacity=64), k=FAKE, v=FAKE, dt=spire.BF16, lens=FAKE,
             offs=FAKE, B=2, Hkv=8, D=128, S=4, W=64, sk=None, sv=None)
    a.update(kw)
    return spire.load().spire_draft_append(C.byref(a["sink"]), C.byref(a["ring"]), a["k"], a["v"],
                                           a["dt"], a["lens"], a["offs"], a["B"], a["Hkv"], a["D"],
                                           a["S"], a["W"], a["sk"], a["sv"], None)


def _rollback(**kw):
    a = dict(sink=kv(capacity=4), ring=kv(capacity=64), sk=FAKE, sv=FAKE, base=FAKE, n=FAKE, steps=4,
             offs=FAKE, B=2, Hkv=8, D=128, S=4, W=64)
    a.update(kw)
    return spire.load().spire_draft_rollback(C.byref(a["sink"]), C.byref(a["ring"]), a["sk"], a["sv"],
                                             a["base"], a["n"], a["steps"], a["offs"], a["B"],
                                             a["Hkv"], a["D"], a["S"], a["W"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(S=0, W=0), INVALID),
    (dict(S=8), INVALID),                             # sink capacity 4 < S
    (dict(W=128), INVALID),                           # ring capacity 64 < W
    (dict(sink=kv(dtype=spire.F32, capacity=4)), INVALID),
    (dict(ring=kv(page_size=16, table=FAKE)), UNSUPPORTED),
    (dict(lens=None), INVALID),
    (dict(offs=None), INVALID),
    (dict(k=None), INVALID),
    (dict(sk=FAKE), INVALID),                         # spill_k without spill_v
    (dict(dt=7), UNSUPPORTED),
])
def test_draft_append_rejects_invalid_arguments(kw, status):
    assert _dappend(**kw) == status


@pytest.mark.parametrize("kw,status", [
    (dict(steps=-1), INVALID),
    (dict(sk=None), INVALID),
    (dict(base=None), INVALID),
    (dict(n=None), INVALID),
    (dict(D=0), UNSUPPORTED),
    (dict(S=-1), INVALID),
])
def test_draft_rollback_rejects_invalid_arguments(kw, status):
    assert _rollback(**kw) == status


def test_draft_updates_empty_are_no_ops():
    assert _dappend(B=0, k=None, v=None, lens=None, offs=None) == OK
    assert _rollback(steps=0, sk=None, sv=None, base=None, n=None, offs=None) == OK


def _fm(**kw):
    a = dict(x=FAKE, xdt=spire.BF16, w=FAKE, n=2, layers=3, B=4, d=128, m=FAKE, mdt=spire.BF16)
    a.update(kw)
    return spire.load().spire_feedback_memory(a["x"], a["xdt"], a["w"], a["n"], a["layers"], a["B"],
                                              a["d"], a["m"], a["mdt"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(n=0), UNSUPPORTED),
    (dict(n=9), UNSUPPORTED),
    (dict(layers=0), UNSUPPORTED),
    (dict(layers=65), UNSUPPORTED),
    (dict(B=-1), INVALID),
    (dict(xdt=spire.FP8), UNSUPPORTED),
    (dict(mdt=spire.FP8), UNSUPPORTED),
    (dict(x=None), INVALID),
    (dict(w=None), INVALID),
    (dict(m=None), INVALID),
    (dict(x=FAKE + 1), INVALID),
    (dict(w=FAKE + 2), INVALID),
])
def test_feedback_memory_rejects_invalid_arguments(kw, status):
    assert _fm(**kw) == status


def test_feedback_memory_empty_is_a_no_op():
    assert _fm(B=0, x=None, w=None, m=None) == OK
    assert _fm(d=0, x=None, w=None, m=None) == OK


def _probe(buf=FAKE, nbytes=1 << 20, sink=FAKE, words=spire.HBM_PROBE_SINK_WORDS):
    return spire.load().spire_hbm_read_probe(buf, nbytes, sink, words, None)


@pytest.mark.parametrize("kw", [
    dict(sink=None),
    dict(buf=None),
    dict(buf=FAKE + 8),
    dict(nbytes=(1 << 20) + 4),
    dict(sink=FAKE + 2),
    dict(words=spire.HBM_PROBE_SINK_WORDS - 1),
])
def test_hbm_read_probe_rejects_invalid_arguments(kw):
    assert _probe(**kw) == INVALID
