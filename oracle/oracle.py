"""ctypes front end of the fp64 CPU oracle (test infrastructure only).

Only the test suite, the package smoke check and the benchmark's CPU-baseline
leg import this module.  It loads `libspire_oracle.so` (built from
`spire_oracle.c` by `build()`), hands it host copies of exactly the bytes the
GPU path reads, and returns fp64 numpy arrays.  Nothing here is shared with the
HIP library.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
from typing import Optional, Sequence

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(_HERE, "spire_oracle.c")
LIB = os.path.join(_HERE, "libspire_oracle.so")

DT = {"f32": 0, "bf16": 1, "fp8": 2}
_TORCH_DT = {torch.float32: "f32", torch.bfloat16: "bf16", torch.float8_e4m3fn: "fp8"}


def build(verbose: bool = False) -> str:
    """Compile the oracle with the host C compiler (gcc, OpenMP)."""
    cmd = ["gcc", "-O2", "-fopenmp", "-std=c99", "-Wall", "-shared", "-fPIC", SRC, "-o", LIB, "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.check_call(cmd)
    return LIB


class _KV(C.Structure):
    _fields_ = [("k", C.c_void_p), ("v", C.c_void_p), ("dtype", C.c_int32),
                ("s_blk", C.c_int64), ("s_head", C.c_int64), ("s_tok", C.c_int64),
                ("page_size", C.c_int32), ("block_table", C.c_void_p), ("max_blocks", C.c_int32),
                ("k_scale", C.c_void_p), ("v_scale", C.c_void_p)]


_libs = {}


def lib(path: Optional[str] = None):
    """Load (building first if stale) the oracle library; `path` loads another
    build of the same source, e.g. a deliberately mutated copy in a test."""
    if path is None:
        path = LIB
        if not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
            build()
    if path not in _libs:
        L = C.CDLL(path)
        L.spire_oracle_verify.restype = C.c_int
        L.spire_oracle_verify.argtypes = [C.c_void_p, C.c_int, C.POINTER(_KV), C.c_void_p,
                                          C.c_void_p, C.c_int, C.c_int, C.c_int, C.c_int, C.c_int,
                                          C.c_double, C.c_void_p, C.c_void_p]
        L.spire_oracle_draft.restype = C.c_int
        L.spire_oracle_draft.argtypes = [C.c_void_p, C.c_int, C.POINTER(_KV), C.POINTER(_KV),
                                         C.c_void_p, C.c_void_p, C.c_void_p, C.c_int, C.c_int,
                                         C.c_int, C.c_int, C.c_int, C.c_int, C.c_double,
                                         C.c_void_p, C.c_void_p]
        L.spire_oracle_decode.restype = C.c_double
        L.spire_oracle_decode.argtypes = [C.c_int, C.c_void_p, C.c_int64]
        L.spire_oracle_threads.restype = C.c_int
        _libs[path] = L
    return _libs[path]


def threads() -> int:
    return lib().spire_oracle_threads()


def _host(t: Optional[torch.Tensor]):
    """Host copy holding the same bytes (fp8 kept as raw bytes)."""
    if t is None:
        return None
    t = t.detach()
    if t.dtype == torch.float8_e4m3fn:
        t = t.view(torch.uint8)
    return t.cpu().contiguous()


def _dtype_name(t: torch.Tensor) -> str:
    return _TORCH_DT[t.dtype]


def _ptr(t):
    return None if t is None else t.data_ptr()


def _kv_struct(k, v, page_size, block_table, k_scale, v_scale, dtype_name, keep):
    """Describe a 4-d storage [blk, h, tok, d] (d contiguous) to the oracle."""
    kh, vh = _host(k), _host(v)
    assert kh.stride() == vh.stride() and kh.stride(3) == 1
    bt = _host(block_table.to(torch.int32)) if block_table is not None else None
    ks = _host(k_scale.float()) if k_scale is not None else None
    vs = _host(v_scale.float()) if v_scale is not None else None
    keep.extend([kh, vh, bt, ks, vs])
    s = kh.stride()
    return _KV(kh.data_ptr(), vh.data_ptr(), DT[dtype_name], s[0], s[1], s[2], page_size,
               _ptr(bt), 0 if bt is None else bt.shape[1], _ptr(ks), _ptr(vs))


def verify(q: torch.Tensor, k_cache: torch.Tensor, v_cache: torch.Tensor, kv_lens,
           k: int, sm_scale: float, page_size: int = 0, block_table=None,
           k_scale=None, v_scale=None, seq_ids: Optional[Sequence[int]] = None,
           lib_path: Optional[str] = None):
    """fp64 verify attention.  q [B, k+1, Hq, D]; returns (out [nsel, k+1, Hq, D],
    lse [nsel, k+1, Hq]) as numpy float64."""
    keep = []
    B, nq, Hq, D = q.shape
    assert nq == k + 1
    Hkv = k_cache.shape[1]
    kv = _kv_struct(k_cache, v_cache, page_size, block_table, k_scale, v_scale,
                    _dtype_name(k_cache), keep)
    qh = _host(q)
    lens = _host(torch.as_tensor(kv_lens).to(torch.int32))
    ids = None if seq_ids is None else torch.tensor(list(seq_ids), dtype=torch.int32)
    nsel = B if ids is None else len(ids)
    out = np.zeros((nsel, nq, Hq, D), dtype=np.float64)
    lse = np.zeros((nsel, nq, Hq), dtype=np.float64)
    rc = lib(lib_path).spire_oracle_verify(qh.data_ptr(), DT[_dtype_name(q)], C.byref(kv), lens.data_ptr(),
                                   _ptr(ids), nsel, Hq, Hkv, D, k, float(sm_scale),
                                   out.ctypes.data, lse.ctypes.data)
    if rc != 0:
        raise RuntimeError(f"oracle verify failed: {rc}")
    return out, lse


def draft(q: torch.Tensor, sink_k, sink_v, ring_k, ring_v, seq_lens, ring_offset, S: int, W: int,
          sm_scale: float, k_scale=None, v_scale=None, seq_ids: Optional[Sequence[int]] = None,
          lib_path: Optional[str] = None, sink_k_scale=None, sink_v_scale=None):
    """fp64 draft sparse attention for one step.  q [B, Hq, D]; sink [B, Hkv, S, D];
    ring [B, Hkv, W, D]; fp8 scales per view (the sink's default to the ring's).
    Returns (out [nsel, Hq, D], lse [nsel, Hq])."""
    keep = []
    B, Hq, D = q.shape
    Hkv = ring_k.shape[1] if W > 0 else sink_k.shape[1]
    dt = _dtype_name(ring_k if W > 0 else sink_k)
    sink = _kv_struct(sink_k, sink_v, 0, None, k_scale if sink_k_scale is None else sink_k_scale,
                      v_scale if sink_v_scale is None else sink_v_scale, dt, keep)
    ring = _kv_struct(ring_k, ring_v, 0, None, k_scale, v_scale, dt, keep)
    qh = _host(q)
    lens = _host(torch.as_tensor(seq_lens).to(torch.int32))
    offs = _host(torch.as_tensor(ring_offset).to(torch.int32))
    ids = None if seq_ids is None else torch.tensor(list(seq_ids), dtype=torch.int32)
    nsel = B if ids is None else len(ids)
    out = np.zeros((nsel, Hq, D), dtype=np.float64)
    lse = np.zeros((nsel, Hq), dtype=np.float64)
    rc = lib(lib_path).spire_oracle_draft(qh.data_ptr(), DT[_dtype_name(q)], C.byref(sink), C.byref(ring),
                                  lens.data_ptr(), offs.data_ptr(), _ptr(ids), nsel, Hq, Hkv, D,
                                  S, W, float(sm_scale), out.ctypes.data, lse.ctypes.data)
    if rc != 0:
        raise RuntimeError(f"oracle draft failed: {rc}")
    return out, lse


def decode(t: torch.Tensor) -> np.ndarray:
    """Decode every element of a storage tensor with the oracle's own decoders."""
    h = _host(t).flatten()
    dt = DT[_dtype_name(t)]
    L = lib()
    return np.array([L.spire_oracle_decode(dt, h.data_ptr(), i) for i in range(h.numel())],
                    dtype=np.float64)
