"""Thin Python binding of libspire.so (argument marshalling only).

Each function takes torch tensors that already live on the current HIP device,
fills the C descriptors of include/spire.h with their device pointers and
strides, and calls the entry point of the same name on torch's current stream.
All arithmetic happens in the library's HIP kernels; there is no fallback: if
the library is missing or a call fails, an exception is raised.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Optional

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libspire.so")

F32, BF16, FP8 = 0, 1, 2
_DT = {torch.float32: F32, torch.bfloat16: BF16, torch.float8_e4m3fn: FP8}
STATUS = {0: "SPIRE_OK", 1: "SPIRE_ERR_INVALID_ARG", 2: "SPIRE_ERR_UNSUPPORTED",
          3: "SPIRE_ERR_WORKSPACE", 4: "SPIRE_ERR_HIP"}

# exported symbols, in the order include/spire.h declares them
SYMBOLS = ["spire_verify_workspace_size", "spire_verify_attn", "spire_verify_attn_noalloc",
           "spire_draft_workspace_size",
           "spire_draft_sparse_attn", "spire_token_verify_workspace_size", "spire_token_verify",
           "spire_block_verify_workspace_size", "spire_block_verify",
           "spire_kv_append", "spire_draft_append", "spire_draft_rollback", "spire_feedback_memory",
           "spire_hbm_read_probe", "spire_status_string", "spire_last_error", "spire_version",
           "spire_verify_attn_ex", "spire_draft_sparse_attn_ex", "spire_token_verify_ex",
           "spire_block_verify_ex"]

# kernel ids of the launches recorded through spire_launch_opts
KERNEL_IDS = {0: "plan", 1: "verify_partial", 2: "draft_partial", 3: "combine",
              4: "token_weights", 5: "token_select", 11: "tail_check", 12: "block_weights",
              13: "block_select"}
# kernel families (spire_launch_opts.kernel)
KERNEL_AUTO, KERNEL_GENERIC, KERNEL_REGS, KERNEL_LDS = 0, 1, 2, 3
HBM_PROBE_SINK_WORDS = 2048


class SpireError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS.get(status, status)}: {msg}")
        self.status = status


class KV(C.Structure):
    """struct spire_kv"""
    _fields_ = [("k", C.c_void_p), ("v", C.c_void_p), ("block_table", C.c_void_p),
                ("k_scale", C.c_void_p), ("v_scale", C.c_void_p),
                ("s_blk", C.c_int64), ("s_head", C.c_int64), ("s_tok", C.c_int64),
                ("dtype", C.c_int32), ("page_size", C.c_int32), ("max_blocks", C.c_int32),
                ("num_blocks", C.c_int32), ("capacity", C.c_int32), ("reserved", C.c_int32)]


class LaunchOpts(C.Structure):
    """struct spire_launch_opts"""
    _fields_ = [("kernel", C.c_int32), ("max_launches", C.c_int32), ("events", C.c_void_p),
                ("kernel_ids", C.c_void_p), ("n_launches", C.c_void_p), ("reserved", C.c_int32)]


_lib = None


def load(path: Optional[str] = None):
    """Load the HIP library (raises if it has not been built)."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or LIB_PATH
    if not os.path.exists(p):
        raise RuntimeError(f"{p} is missing: build it with `python -m paper_2504_06419_amd.build`")
    L = C.CDLL(p)
    vp, i32, sz = C.c_void_p, C.c_int32, C.c_size_t
    L.spire_verify_workspace_size.restype = sz
    L.spire_verify_workspace_size.argtypes = [i32] * 5
    L.spire_verify_attn.restype = C.c_int
    L.spire_verify_attn.argtypes = [vp, i32, C.POINTER(KV), vp, i32, i32, i32, i32, i32, C.c_float,
                                    vp, i32, vp, vp, sz, vp]
    L.spire_verify_attn_noalloc.restype = C.c_int
    L.spire_verify_attn_noalloc.argtypes = [vp, i32, C.POINTER(KV), vp, i32, i32, i32, i32, i32, C.c_float,
                                            vp, i32, vp, vp]
    L.spire_draft_workspace_size.restype = sz
    L.spire_draft_workspace_size.argtypes = [i32] * 4
    L.spire_draft_sparse_attn.restype = C.c_int
    L.spire_draft_sparse_attn.argtypes = [vp, i32, C.POINTER(KV), C.POINTER(KV), vp, vp, i32, i32,
                                          i32, i32, i32, i32, C.c_float, vp, i32, vp, vp, sz, vp]
    L.spire_token_verify_workspace_size.restype = sz
    L.spire_token_verify_workspace_size.argtypes = [i32] * 3
    L.spire_token_verify.restype = C.c_int
    L.spire_token_verify.argtypes = [vp, vp, vp, vp, vp, i32, i32, i32, vp, vp, vp, sz, vp]
    L.spire_kv_append.restype = C.c_int
    L.spire_kv_append.argtypes = [C.POINTER(KV), vp, vp, i32, vp, i32, i32, i32, i32, vp]
    L.spire_draft_append.restype = C.c_int
    L.spire_draft_append.argtypes = [C.POINTER(KV), C.POINTER(KV), vp, vp, i32, vp, vp, i32, i32, i32,
                                     i32, i32, vp, vp, vp]
    L.spire_draft_rollback.restype = C.c_int
    L.spire_draft_rollback.argtypes = [C.POINTER(KV), C.POINTER(KV), vp, vp, vp, vp, i32, vp, i32, i32,
                                       i32, i32, i32, vp]
    L.spire_feedback_memory.restype = C.c_int
    L.spire_feedback_memory.argtypes = [vp, i32, vp, i32, i32, i32, i32, vp, i32, vp]
    L.spire_status_string.restype = C.c_char_p
    L.spire_status_string.argtypes = [C.c_int]
    L.spire_last_error.restype = C.c_char_p
    L.spire_last_error.argtypes = []
    L.spire_version.restype = i32
    L.spire_verify_attn_ex.restype = C.c_int
    L.spire_verify_attn_ex.argtypes = L.spire_verify_attn.argtypes + [C.POINTER(LaunchOpts)]
    L.spire_draft_sparse_attn_ex.restype = C.c_int
    L.spire_draft_sparse_attn_ex.argtypes = L.spire_draft_sparse_attn.argtypes + [C.POINTER(LaunchOpts)]
    L.spire_token_verify_ex.restype = C.c_int
    L.spire_token_verify_ex.argtypes = L.spire_token_verify.argtypes + [C.POINTER(LaunchOpts)]
    L.spire_block_verify_workspace_size.restype = sz
    L.spire_block_verify_workspace_size.argtypes = [i32] * 3
    L.spire_block_verify.restype = C.c_int
    L.spire_block_verify.argtypes = L.spire_token_verify.argtypes
    L.spire_block_verify_ex.restype = C.c_int
    L.spire_block_verify_ex.argtypes = L.spire_token_verify.argtypes + [C.POINTER(LaunchOpts)]
    L.spire_hbm_read_probe.restype = C.c_int
    L.spire_hbm_read_probe.argtypes = [vp, sz, vp, sz, vp]
    if path is None:
        _lib = L
    return L


def _check(rc: int):
    if rc != 0:
        raise SpireError(rc, load().spire_last_error().decode())


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else t.data_ptr()


def _stream():
    return torch.cuda.current_stream().cuda_stream


def kv_view(k: torch.Tensor, v: torch.Tensor, block_table: Optional[torch.Tensor] = None,
            page_size: int = 0, k_scale: Optional[torch.Tensor] = None,
            v_scale: Optional[torch.Tensor] = None, capacity: Optional[int] = None) -> KV:
    """Describe 4-d storage [blk, h, tok, d] (d contiguous) as a spire_kv.
    Paged when `block_table` is given (blk = physical page), else contiguous
    (blk = sequence, capacity = size of dim 2 unless given)."""
    assert k.shape == v.shape and k.stride() == v.stride() and k.dtype == v.dtype
    assert k.stride(3) == 1, "head dim must be contiguous"
    kv = KV()
    kv.k, kv.v = k.data_ptr(), v.data_ptr()
    kv.s_blk, kv.s_head, kv.s_tok = k.stride(0), k.stride(1), k.stride(2)
    kv.dtype = _DT[k.dtype]
    kv.k_scale, kv.v_scale = _ptr(k_scale), _ptr(v_scale)
    if block_table is not None:
        assert block_table.dtype == torch.int32 and block_table.is_contiguous()
        kv.block_table = block_table.data_ptr()
        kv.page_size = page_size or k.shape[2]
        kv.max_blocks = block_table.shape[1]
        kv.num_blocks = k.shape[0]
        kv.capacity = 0
    else:
        kv.block_table = None
        kv.page_size = 0
        kv.capacity = k.shape[2] if capacity is None else capacity
    kv.reserved = 0
    return kv


def verify_workspace_size(B, Hq, Hkv, D, k) -> int:
    return int(load().spire_verify_workspace_size(B, Hq, Hkv, D, k))


def draft_workspace_size(B, Hq, Hkv, D) -> int:
    return int(load().spire_draft_workspace_size(B, Hq, Hkv, D))


def workspace(nbytes: int, device=None) -> torch.Tensor:
    """A caller-owned workspace buffer (256-byte aligned by the caching allocator)."""
    return torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device or "cuda")


class LaunchRecorder:
    """Caller-owned HIP events the library records around each kernel one call
    launches (spire_launch_opts): pass `rec.opts(kernel)` as `opts`, then
    `rec.collect()` gives [(kernel name, ms)] of that call's launches."""

    def __init__(self, max_launches: int = 8):
        self.max = max_launches
        self.events = [torch.cuda.Event(enable_timing=True) for _ in range(2 * max_launches)]
        for e in self.events:       # torch creates the underlying HIP event on first record
            e.record()
        torch.cuda.synchronize()
        self._handles = (C.c_void_p * (2 * max_launches))(*[e.cuda_event for e in self.events])
        self._ids = (C.c_int32 * max_launches)()
        self._n = C.c_int32(0)

    def opts(self, kernel: int = 0) -> LaunchOpts:
        o = LaunchOpts()
        o.kernel, o.max_launches = kernel, self.max
        o.events = C.cast(self._handles, C.c_void_p)
        o.kernel_ids, o.n_launches = C.addressof(self._ids), C.addressof(self._n)
        o.reserved = 0
        return o

    def collect(self):
        """[(kernel name, ms)] of the recorded launches of the last call (synchronises)."""
        torch.cuda.synchronize()
        n = min(self._n.value, self.max)
        return [(KERNEL_IDS.get(self._ids[i], str(self._ids[i])),
                 self.events[2 * i].elapsed_time(self.events[2 * i + 1])) for i in range(n)]


def _opts(kernel: int, opts: Optional[LaunchOpts]):
    if opts is None and kernel == 0:
        return None
    if opts is None:
        opts = LaunchOpts()
        opts.kernel = kernel
    return C.byref(opts)


def verify_attn(q: torch.Tensor, kv: KV, kv_lens: torch.Tensor, Hkv: int, k: int,
                sm_scale: float, out: Optional[torch.Tensor] = None,
                lse: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None,
                out_dtype=torch.float32, with_lse: bool = True, kernel: int = 0,
                opts: Optional[LaunchOpts] = None):
    """spire_verify_attn (spire_verify_attn_ex with a kernel choice or launch
    events).  q [B, k+1, Hq, D]; returns (out, lse)."""
    B, nq, Hq, D = q.shape
    assert nq == k + 1 and q.is_contiguous()
    if out is None:
        out = torch.empty((B, nq, Hq, D), dtype=out_dtype, device=q.device)
    if lse is None and with_lse:
        lse = torch.empty((B, nq, Hq), dtype=torch.float32, device=q.device)
    if ws is None:
        ws = workspace(verify_workspace_size(B, Hq, Hkv, D, k), q.device)
    lens = kv_lens if kv_lens.dtype == torch.int32 else kv_lens.to(torch.int32)
    _check(load().spire_verify_attn_ex(q.data_ptr(), _DT[q.dtype], C.byref(kv), lens.data_ptr(), B, Hq,
                                       Hkv, D, k, float(sm_scale), out.data_ptr(), _DT[out.dtype],
                                       _ptr(lse), ws.data_ptr(), ws.numel(), _stream(), _opts(kernel, opts)))
    return out, lse


def verify_attn_noalloc(q: torch.Tensor, kv: KV, kv_lens: torch.Tensor, Hkv: int, k: int,
                        sm_scale: float, out: torch.Tensor, lse: Optional[torch.Tensor] = None):
    """spire_verify_attn_noalloc: the verify call with the library's own
    scratch instead of a workspace; the caller passes the outputs
    (out [B, k+1, Hq, D] f32 or bf16, lse [B, k+1, Hq] f32 or None)."""
    B, nq, Hq, D = q.shape
    assert nq == k + 1 and q.is_contiguous() and out.is_contiguous()
    lens = kv_lens if kv_lens.dtype == torch.int32 else kv_lens.to(torch.int32)
    _check(load().spire_verify_attn_noalloc(q.data_ptr(), _DT[q.dtype], C.byref(kv), lens.data_ptr(), B, Hq,
                                            Hkv, D, k, float(sm_scale), out.data_ptr(), _DT[out.dtype],
                                            _ptr(lse), _stream()))
    return out, lse


def draft_sparse_attn(q: torch.Tensor, sink: KV, ring: KV, seq_lens: torch.Tensor,
                      ring_offset: torch.Tensor, S: int, W: int, sm_scale: float, Hkv: int,
                      out: Optional[torch.Tensor] = None, lse: Optional[torch.Tensor] = None,
                      ws: Optional[torch.Tensor] = None, out_dtype=torch.float32,
                      with_lse: bool = True, kernel: int = 0, opts: Optional[LaunchOpts] = None):
    """spire_draft_sparse_attn (the _ex form with a kernel choice or launch
    events).  q [B, Hq, D]; returns (out, lse)."""
    B, Hq, D = q.shape
    assert q.is_contiguous()
    if out is None:
        out = torch.empty((B, Hq, D), dtype=out_dtype, device=q.device)
    if lse is None and with_lse:
        lse = torch.empty((B, Hq), dtype=torch.float32, device=q.device)
    if ws is None:
        ws = workspace(draft_workspace_size(B, Hq, Hkv, D), q.device)
    _check(load().spire_draft_sparse_attn_ex(q.data_ptr(), _DT[q.dtype], C.byref(sink), C.byref(ring),
                                             seq_lens.data_ptr(), ring_offset.data_ptr(), B, Hq, Hkv,
                                             D, S, W, float(sm_scale), out.data_ptr(), _DT[out.dtype],
                                             _ptr(lse), ws.data_ptr(), ws.numel(), _stream(),
                                             _opts(kernel, opts)))
    return out, lse


def token_verify_workspace_size(B, k, V) -> int:
    return int(load().spire_token_verify_workspace_size(B, k, V))


def token_verify(p: torch.Tensor, q: Optional[torch.Tensor], draft: Optional[torch.Tensor],
                 u_accept: Optional[torch.Tensor], u_sample: torch.Tensor,
                 n_accepted: Optional[torch.Tensor] = None, tokens: Optional[torch.Tensor] = None,
                 ws: Optional[torch.Tensor] = None, opts: Optional[LaunchOpts] = None):
    """spire_token_verify.  p [B, k+1, V] fp32, q [B, k, V] fp32, draft [B, k]
    int32, u_accept [B, k] fp32, u_sample [B] fp32; returns (n_accepted [B],
    tokens [B, k+1]) as int32 tensors."""
    B, kp1, V = p.shape
    k = kp1 - 1
    assert p.dtype == torch.float32 and p.is_contiguous() and u_sample.is_contiguous()
    if k > 0:
        assert q.shape == (B, k, V) and q.dtype == torch.float32 and q.is_contiguous()
        assert draft.shape == (B, k) and draft.dtype == torch.int32 and draft.is_contiguous()
        assert u_accept.shape == (B, k) and u_accept.dtype == torch.float32 and u_accept.is_contiguous()
    if n_accepted is None:
        n_accepted = torch.empty((B,), dtype=torch.int32, device=p.device)
    if tokens is None:
        tokens = torch.empty((B, kp1), dtype=torch.int32, device=p.device)
    if ws is None:
        ws = workspace(token_verify_workspace_size(B, k, V), p.device)
    _check(load().spire_token_verify_ex(p.data_ptr(), _ptr(q) if k > 0 else None,
                                        _ptr(draft) if k > 0 else None,
                                        _ptr(u_accept) if k > 0 else None, u_sample.data_ptr(), B, k,
                                        V, n_accepted.data_ptr(), tokens.data_ptr(), ws.data_ptr(),
                                        ws.numel(), _stream(), _opts(0, opts)))
    return n_accepted, tokens


def block_verify_workspace_size(B, k, V) -> int:
    return int(load().spire_block_verify_workspace_size(B, k, V))


def block_verify(p: torch.Tensor, q: Optional[torch.Tensor], draft: Optional[torch.Tensor],
                 u_accept: Optional[torch.Tensor], u_sample: torch.Tensor,
                 n_accepted: Optional[torch.Tensor] = None, tokens: Optional[torch.Tensor] = None,
                 ws: Optional[torch.Tensor] = None, opts: Optional[LaunchOpts] = None):
    """spire_block_verify: arguments and results as token_verify."""
    B, kp1, V = p.shape
    k = kp1 - 1
    assert p.dtype == torch.float32 and p.is_contiguous() and u_sample.is_contiguous()
    if k > 0:
        assert q.shape == (B, k, V) and q.dtype == torch.float32 and q.is_contiguous()
        assert draft.shape == (B, k) and draft.dtype == torch.int32 and draft.is_contiguous()
        assert u_accept.shape == (B, k) and u_accept.dtype == torch.float32 and u_accept.is_contiguous()
    if n_accepted is None:
        n_accepted = torch.empty((B,), dtype=torch.int32, device=p.device)
    if tokens is None:
        tokens = torch.empty((B, kp1), dtype=torch.int32, device=p.device)
    if ws is None:
        ws = workspace(block_verify_workspace_size(B, k, V), p.device)
    _check(load().spire_block_verify_ex(p.data_ptr(), _ptr(q) if k > 0 else None,
                                        _ptr(draft) if k > 0 else None,
                                        _ptr(u_accept) if k > 0 else None, u_sample.data_ptr(), B, k,
                                        V, n_accepted.data_ptr(), tokens.data_ptr(), ws.data_ptr(),
                                        ws.numel(), _stream(), _opts(0, opts)))
    return n_accepted, tokens


def kv_append(kv: KV, k_new: torch.Tensor, v_new: torch.Tensor, positions: torch.Tensor):
    """spire_kv_append.  k_new / v_new [B, T, Hkv, D] (fp32 or bf16), positions [B] int32."""
    B, T, Hkv, D = k_new.shape
    assert v_new.shape == k_new.shape and v_new.dtype == k_new.dtype
    assert k_new.is_contiguous() and v_new.is_contiguous() and positions.dtype == torch.int32
    _check(load().spire_kv_append(C.byref(kv), k_new.data_ptr(), v_new.data_ptr(), _DT[k_new.dtype],
                                  positions.data_ptr(), B, Hkv, D, T, _stream()))


def draft_append(sink: KV, ring: KV, k_new: torch.Tensor, v_new: torch.Tensor,
                 seq_lens: torch.Tensor, ring_offset: torch.Tensor, S: int, W: int,
                 spill_k: Optional[torch.Tensor] = None, spill_v: Optional[torch.Tensor] = None):
    """spire_draft_append.  k_new / v_new [B, Hkv, D]; spill [B, Hkv, D] in the storage dtype."""
    B, Hkv, D = k_new.shape
    assert v_new.shape == k_new.shape and k_new.is_contiguous() and v_new.is_contiguous()
    for t in (spill_k, spill_v):
        assert t is None or (t.is_contiguous() and t.numel() == B * Hkv * D)
    _check(load().spire_draft_append(C.byref(sink), C.byref(ring), k_new.data_ptr(), v_new.data_ptr(),
                                     _DT[k_new.dtype], seq_lens.data_ptr(), ring_offset.data_ptr(), B,
                                     Hkv, D, S, W, _ptr(spill_k), _ptr(spill_v), _stream()))


def draft_rollback(sink: KV, ring: KV, spill_k: torch.Tensor, spill_v: torch.Tensor,
                   base_lens: torch.Tensor, n_accepted: torch.Tensor, ring_offset: torch.Tensor,
                   S: int, W: int):
    """spire_draft_rollback.  spill [steps, B, Hkv, D] in the storage dtype."""
    steps, B, Hkv, D = spill_k.shape
    assert spill_v.shape == spill_k.shape and spill_k.is_contiguous() and spill_v.is_contiguous()
    _check(load().spire_draft_rollback(C.byref(sink), C.byref(ring), spill_k.data_ptr(),
                                       spill_v.data_ptr(), base_lens.data_ptr(), n_accepted.data_ptr(),
                                       steps, ring_offset.data_ptr(), B, Hkv, D, S, W, _stream()))


def feedback_memory(x: torch.Tensor, w: torch.Tensor, out: Optional[torch.Tensor] = None,
                    out_dtype=torch.float32) -> torch.Tensor:
    """spire_feedback_memory.  x [layers, B, d] (fp32 or bf16), w [n_out, layers] fp32;
    returns m [n_out, B, d]."""
    layers, B, d = x.shape
    n_out = w.shape[0]
    assert x.is_contiguous() and w.is_contiguous() and w.dtype == torch.float32 and w.shape[1] == layers
    if out is None:
        out = torch.empty((n_out, B, d), dtype=out_dtype, device=x.device)
    assert out.is_contiguous() and out.shape == (n_out, B, d)
    _check(load().spire_feedback_memory(x.data_ptr(), _DT[x.dtype], w.data_ptr(), n_out, layers, B, d,
                                        out.data_ptr(), _DT[out.dtype], _stream()))
    return out


def hbm_read_probe(buf: torch.Tensor, sink: Optional[torch.Tensor] = None) -> torch.Tensor:
    """spire_hbm_read_probe: stream `buf` (contiguous, 16-byte aligned, a
    multiple of 16 bytes) once; returns the int32 sink of XOR folds."""
    assert buf.is_contiguous() and buf.is_cuda
    if sink is None:
        sink = torch.empty((HBM_PROBE_SINK_WORDS,), dtype=torch.int32, device=buf.device)
    assert sink.dtype == torch.int32 and sink.is_cuda
    _check(load().spire_hbm_read_probe(buf.data_ptr(), buf.numel() * buf.element_size(),
                                       sink.data_ptr(), sink.numel(), _stream()))
    return sink
