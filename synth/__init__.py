"""Seeded synthetic inputs for the attention workloads.

Random numbers and storage conversion only: nothing in this package computes
any part of attention.  The oracle tests, the GPU parity tests, ``smoke()`` and
``bench.py`` all draw Q, K and V from here, so both sides of every comparison
see the same bytes.  The generator itself is C (``synth.c``, documented there)
because numpy is far too slow for the 16K-token workloads.

Arrays come back as numpy: ``float32`` for fp32 storage and ``uint16`` bit
patterns for bf16 storage (``to_torch`` reinterprets those as ``bfloat16``).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "synth.c")
_LIB_PATH = os.path.join(_HERE, "libsynth.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile ``libsynth.so`` next to its source with gcc."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + f".tmp{os.getpid()}"
        cmd = ["gcc", "-O2", "-fopenmp", "-ffp-contract=off", "-fPIC", "-shared",
               "-std=c11", _SRC, "-o", tmp, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build(force=False)
        lib = ctypes.CDLL(_LIB_PATH)
        i64, u64, dbl, vp = ctypes.c_int64, ctypes.c_uint64, ctypes.c_double, ctypes.c_void_p
        lib.synth_splitmix64.argtypes = [u64, u64]
        lib.synth_splitmix64.restype = u64
        for name in ("synth_normal_f64", "synth_normal_f32", "synth_normal_bf16"):
            getattr(lib, name).argtypes = [u64, i64, dbl, vp]
            getattr(lib, name).restype = None
        lib.synth_f32_to_bf16.argtypes = [vp, i64, vp]
        lib.synth_f32_to_bf16.restype = None
        _lib = lib
    return _lib


def splitmix64(seed: int, k: int) -> int:
    """Output ``k`` (0-based) of the SplitMix64 stream started at ``seed``."""
    return int(_load().synth_splitmix64(seed & (2**64 - 1), k))


def normal(seed: int, shape, sigma: float = 1.0, dtype: str = "bf16") -> np.ndarray:
    """N(0, sigma^2) samples; ``dtype`` is ``"f64"``, ``"f32"`` or ``"bf16"`` (uint16 bits)."""
    n = int(np.prod(shape)) if len(shape) else 1
    lib = _load()
    if dtype == "f64":
        out = np.empty(n, dtype=np.float64)
        lib.synth_normal_f64(seed, n, float(sigma), out.ctypes.data)
    elif dtype == "f32":
        out = np.empty(n, dtype=np.float32)
        lib.synth_normal_f32(seed, n, float(sigma), out.ctypes.data)
    elif dtype == "bf16":
        out = np.empty(n, dtype=np.uint16)
        lib.synth_normal_bf16(seed, n, float(sigma), out.ctypes.data)
    else:
        raise ValueError(f"unknown dtype {dtype!r}")
    return out.reshape(shape)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16 (nearest even); returns the uint16 bit patterns."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty(x.shape, dtype=np.uint16)
    _load().synth_f32_to_bf16(x.ctypes.data, x.size, out.ctypes.data)
    return out


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to fp32 (for building test inputs)."""
    return (np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


@dataclass(frozen=True)
class Workload:
    """One attention problem: shapes, storage type, input distribution, mask."""
    name: str
    B: int
    H: int
    Nq: int
    Nk: int
    dk: int
    dv: int
    dtype: str          # "f32" or "bf16": storage of Q, K and V
    causal: bool
    sigma_qk: float = 1.0
    sigma_v: float = 1.0
    seed: int = 1000

    @property
    def scale(self) -> float:
        return float(np.float32(1.0 / np.sqrt(self.dk)))

    def seeds(self):
        """Per-tensor seeds for Q, K, V."""
        return self.seed * 3 + 0, self.seed * 3 + 1, self.seed * 3 + 2


# The five workloads this library is measured and checked on.
WORKLOADS = {
    w.name: w for w in [
        Workload("single_head_f32_n128_d64", 1, 1, 128, 128, 64, 64, "f32", False, seed=1000),
        Workload("mha_b4h8_n1024_d64_bf16", 4, 8, 1024, 1024, 64, 64, "bf16", False, seed=1001),
        Workload("causal_b2h16_n4096_d128_bf16", 2, 16, 4096, 4096, 128, 128, "bf16", True, seed=1002),
        Workload("causal_long_b1h32_n16384_d128_bf16_qk_sigma3", 1, 32, 16384, 16384, 128, 128,
                 "bf16", True, sigma_qk=3.0, seed=1003),
        Workload("decode_b64h32_nk8192_d128_bf16", 64, 32, 1, 8192, 128, 128, "bf16", False, seed=1004),
    ]
}


def make_inputs(w: Workload):
    """Q [B,H,Nq,dk], K [B,H,Nk,dk], V [B,H,Nk,dv] for workload ``w``."""
    sq, sk, sv = w.seeds()
    q = normal(sq, (w.B, w.H, w.Nq, w.dk), w.sigma_qk, w.dtype)
    k = normal(sk, (w.B, w.H, w.Nk, w.dk), w.sigma_qk, w.dtype)
    v = normal(sv, (w.B, w.H, w.Nk, w.dv), w.sigma_v, w.dtype)
    return q, k, v


def to_torch(a: np.ndarray, device=None):
    """numpy array (float32, float64 or bf16 bits as uint16) -> torch tensor."""
    import torch
    if a.dtype == np.uint16:
        t = torch.from_numpy(a.view(np.int16)).view(torch.bfloat16)
    else:
        t = torch.from_numpy(a)
    return t if device is None else t.to(device)
