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
        lib.oracle_attn_bwd_rows.argtypes = ([vp, vp, vp, vp, ci] + dims +
                                             [f32, ci, i64, vp, i64, vp, i64, vp, vp, vp, ci])
        for f in (lib.oracle_attn_fwd, lib.oracle_attn_rows, lib.oracle_attn_weights,
                  lib.oracle_attn_bwd, lib.oracle_attn_bwd_rows):
            f.restype = ci
        lib.oracle_proj.argtypes = [vp, vp, ci, i64, i64, i64, i64, i64, vp, ci]
        lib.oracle_proj.restype = ci
        lib.oracle_bf16_round.argtypes = [vp, i64, vp]
        lib.oracle_bf16_round.restype = None
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


def attention_bwd_rows(q, k, v, do, bh, qrows, krows, scale=None, causal=False, nthreads=0):
    """The gradients of ``attention_bwd`` at sampled outputs of head slice ``bh`` (b*H + h):
    dQ [len(qrows), dk] at query rows ``qrows`` and dK, dV [len(krows), .] at key rows
    ``krows`` (indices within the slice), fp64."""
    q, k, v, dt, (B, H, Nq, Nk, dk, dv) = _prep(q, k, v)
    do = np.ascontiguousarray(do)
    if do.dtype != q.dtype or do.shape != (B, H, Nq, dv):
        raise ValueError("dO must have the storage type of Q and shape [B, H, Nq, dv]")
    qrows = np.ascontiguousarray(qrows, dtype=np.int64)
    krows = np.ascontiguousarray(krows, dtype=np.int64)
    dq = np.empty((qrows.size, dk), dtype=np.float64)
    dk_ = np.empty((krows.size, dk), dtype=np.float64)
    dv_ = np.empty((krows.size, dv), dtype=np.float64)
    rc = _load().oracle_attn_bwd_rows(q.ctypes.data, k.ctypes.data, v.ctypes.data, do.ctypes.data,
                                      dt, B, H, Nq, Nk, dk, dv, _scale(scale, dk),
                                      int(bool(causal)), int(bh), qrows.ctypes.data, qrows.size,
                                      krows.ctypes.data, krows.size, dq.ctypes.data,
                                      dk_.ctypes.data, dv_.ctypes.data, int(nthreads))
    if rc != 0:
        raise ValueError(f"oracle_attn_bwd_rows rejected the problem (code {rc})")
    return dq, dk_, dv_


def projection(x, wt, H, d, nthreads=0):
    """Exact fp64 projection in head-split form: x [B, N, Dm] and wt [H*d, Dm]
    (fp32 or bf16 bit patterns) -> [B, H, N, d] with P[b,h,n,e] = sum_k x[b,n,k] wt[h*d+e, k]."""
    x, wt = np.ascontiguousarray(x), np.ascontiguousarray(wt)
    if x.dtype != wt.dtype or x.dtype not in (np.float32, np.uint16):
        raise TypeError("x and wt share one storage type: float32 or bf16 bit patterns")
    B, N, Dm = x.shape
    if wt.shape != (H * d, Dm):
        raise ValueError(f"wt must be [H*d, Dm] = {(H * d, Dm)}, got {wt.shape}")
    p = np.empty((B, H, N, d), dtype=np.float64)
    dt = F32 if x.dtype == np.float32 else BF16
    rc = _load().oracle_proj(x.ctypes.data, wt.ctypes.data, dt, B, N, Dm, H, d, p.ctypes.data,
                             int(nthreads))
    if rc != 0:
        raise ValueError("oracle_proj rejected the problem")
    return p


def round_bf16(v):
    """fp64 -> bf16 bit patterns (uint16), round to nearest even, directly from fp64."""
    v = np.ascontiguousarray(v, dtype=np.float64)
    out = np.empty(v.shape, dtype=np.uint16)
    _load().oracle_bf16_round(v.ctypes.data, v.size, out.ctypes.data)
    return out


def attention_proj(x, wq, wk, wv, H, d, scale=None, causal=False, nthreads=0, with_lse=False):
    """Self-attention of a sequence through its input projections: Q, K, V = the exact
    projections of x by wq, wk, wv (each [H*d, Dm]) rounded to bf16 -- the storage the
    projected tensors have between the two steps -- then the attention oracle on them.
    Returns (O, Q, K, V) with Q, K, V as bf16 bit patterns [B, H, N, d] (and LSE)."""
    q, k, v = (round_bf16(projection(x, w, H, d, nthreads)) for w in (wq, wk, wv))
    r = attention(q, k, v, scale=scale, causal=causal, nthreads=nthreads, with_lse=with_lse)
    if with_lse:
        return r[0], q, k, v, r[1]
    return r, q, k, v


def max_threads() -> int:
    return int(_load().oracle_max_threads())
