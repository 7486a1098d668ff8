"""fp64 CPU oracle for scaled dot-product attention -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The GPU library never imports, links or
calls it, and it shares no code with the GPU library.

The arithmetic lives in ``oracle_attn.c`` (plain C, fp64, built with
``-ffp-contract=off`` and no fast-math); its header states what is computed,
with the paper's equations and steps, and every reading taken where the paper
is silent.  This module only compiles it and marshals numpy arrays.

Every function here is pinned by ``tests/test_oracle.py`` against the paper's
worked example (Tables 1 and 2 and the appendix trace), a library routine on
tiny shapes, closed forms and invariants.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle_attn.c")
_LIB_PATH = os.path.join(_HERE, "liboracle_attn.so")
_lib = None

F32, BF16 = 0, 1


def build(force: bool = True) -> str:
    """Compile ``liboracle_attn.so`` next to its source with gcc."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + f".tmp{os.getpid()}"
        cmd = ["gcc", "-O2", "-fopenmp", "-ffp-contract=off", "-fno-fast-math", "-fPIC",
               "-shared", "-std=c11", "-Wall", _SRC, "-o", tmp, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build(force=False)
        lib = ctypes.CDLL(_LIB_PATH)
        i64, vp, f32, ci = ctypes.c_int64, ctypes.c_void_p, ctypes.c_float, ctypes.c_int
        dims = [i64] * 6
        lib.oracle_attn_fwd.argtypes = [vp, vp, vp, ci] + dims + [f32, ci, vp, vp, ci]
        lib.oracle_attn_rows.argtypes = [vp, vp, vp, ci] + dims + [f32, ci, vp, i64, vp, vp, ci]
        lib.oracle_attn_weights.argtypes = [vp, vp, vp, ci] + dims + [f32, ci, vp, vp, vp, vp]
        lib.oracle_attn_bwd.argtypes = [vp, vp, vp, vp, ci] + dims + [f32, ci, vp, vp, vp, ci]
        for f in (lib.oracle_attn_fwd, lib.oracle_attn_rows, lib.oracle_attn_weights,
                  lib.oracle_attn_bwd):
            f.restype = ci
        lib.oracle_max_threads.argtypes = []
        lib.oracle_max_threads.restype = ci
        _lib = lib
    return _lib


def _prep(q, k, v):
    q, k, v = (np.ascontiguousarray(a) for a in (q, k, v))
    if not (q.dtype == k.dtype == v.dtype):
        raise TypeError("Q, K and V must share one storage type")
    if q.dtype == np.float32:
        dt = F32
    elif q.dtype == np.uint16:
        dt = BF16
    else:
        raise TypeError("inputs are float32 arrays or bf16 bit patterns (uint16)")
    if q.ndim != 4 or k.ndim != 4 or v.ndim != 4:
        raise ValueError("Q, K, V are [B, H, N, d]")
    B, H, Nq, dk = q.shape
    Nk = k.shape[2]
    dv = v.shape[3]
    if k.shape != (B, H, Nk, dk) or v.shape != (B, H, Nk, dv):
        raise ValueError(f"shape mismatch: {q.shape} {k.shape} {v.shape}")
    return q, k, v, dt, (B, H, Nq, Nk, dk, dv)


def _scale(scale, dk):
    return float(np.float32(1.0 / np.sqrt(dk))) if scale is None else float(np.float32(scale))


def attention(q, k, v, scale=None, causal=False, nthreads=0, with_lse=False):
    """O [B,H,Nq,dv] in fp64 (and LSE [B,H,Nq] when ``with_lse``)."""
    q, k, v, dt, (B, H, Nq, Nk, dk, dv) = _prep(q, k, v)
    o = np.empty((B, H, Nq, dv), dtype=np.float64)
    lse = np.empty((B, H, Nq), dtype=np.float64) if with_lse else None
    rc = _load().oracle_attn_fwd(q.ctypes.data, k.ctypes.data, v.ctypes.data, dt, B, H, Nq, Nk,
                                 dk, dv, _scale(scale, dk), int(bool(causal)), o.ctypes.data,
                                 lse.ctypes.data if with_lse else None, int(nthreads))
    if rc != 0:
        raise ValueError(f"oracle_attn_fwd rejected the problem (code {rc})")
    return (o, lse) if with_lse else o


def attention_rows(q, k, v, rows, scale=None, causal=False, nthreads=0, with_lse=False):
    """Only the flat rows ``rows`` ((b*H + h)*Nq + i): O [n, dv] (and LSE [n])."""
    q, k, v, dt, (B, H, Nq, Nk, dk, dv) = _prep(q, k, v)
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    n = rows.size
    o = np.empty((n, dv), dtype=np.float64)
    lse = np.empty(n, dtype=np.float64) if with_lse else None
    rc = _load().oracle_attn_rows(q.ctypes.data, k.ctypes.data, v.ctypes.data, dt, B, H, Nq, Nk,
                                  dk, dv, _scale(scale, dk), int(bool(causal)), rows.ctypes.data, n,
                                  o.ctypes.data, lse.ctypes.data if with_lse else None,
                                  int(nthreads))
    if rc != 0:
        raise ValueError(f"oracle_attn_rows rejected the problem (code {rc})")
    return (o, lse) if with_lse else o


def attention_weights(q, k, v, scale=None, causal=False):
    """Tiny shapes: (S, P, O, LSE) with S and P [B,H,Nq,Nk], all fp64."""
    q, k, v, dt, (B, H, Nq, Nk, dk, dv) = _prep(q, k, v)
    s = np.empty((B, H, Nq, Nk), dtype=np.float64)
    p = np.empty((B, H, Nq, Nk), dtype=np.float64)
    o = np.empty((B, H, Nq, dv), dtype=np.float64)
    lse = np.empty((B, H, Nq), dtype=np.float64)
    rc = _load().oracle_attn_weights(q.ctypes.data, k.ctypes.data, v.ctypes.data, dt, B, H, Nq,
                                     Nk, dk, dv, _scale(scale, dk), int(bool(causal)),
                                     s.ctypes.data, p.ctypes.data, o.ctypes.data, lse.ctypes.data)
    if rc != 0:
        raise ValueError(f"oracle_attn_weights rejected the problem (code {rc})")
    return s, p, o, lse


def attention_bwd(q, k, v, do, scale=None, causal=False, nthreads=0):
    """Gradients (dQ, dK, dV), fp64, of a loss whose gradient through O is ``do``
    ([B,H,Nq,dv], same storage type as q, k, v)."""
    q, k, v, dt, (B, H, Nq, Nk, dk, dv) = _prep(q, k, v)
    do = np.ascontiguousarray(do)
    if do.dtype != q.dtype or do.shape != (B, H, Nq, dv):
        raise ValueError("dO must have the storage type of Q and shape [B, H, Nq, dv]")
    dq = np.empty((B, H, Nq, dk), dtype=np.float64)
    dk_ = np.empty((B, H, Nk, dk), dtype=np.float64)
    dv_ = np.empty((B, H, Nk, dv), dtype=np.float64)
    rc = _load().oracle_attn_bwd(q.ctypes.data, k.ctypes.data, v.ctypes.data, do.ctypes.data, dt,
                                 B, H, Nq, Nk, dk, dv, _scale(scale, dk), int(bool(causal)),
                                 dq.ctypes.data, dk_.ctypes.data, dv_.ctypes.data, int(nthreads))
    if rc != 0:
        raise ValueError(f"oracle_attn_bwd rejected the problem (code {rc})")
    return dq, dk_, dv_


def max_threads() -> int:
    return int(_load().oracle_max_threads())
