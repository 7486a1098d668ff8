"""Helpers for the GPU tests: run the HIP path through the C ABI on seeded
inputs, run the oracle on the same host bytes, compare."""
import sys

import numpy as np

import oracle
import synth

# Max-abs tolerances relative to std(V) (= the generator's sigma_v), per input storage type.
TOL = {"f32": 1e-5, "bf16": 2e-2}


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def gen(B, H, Nq, Nk, d, dtype, seed, sigma_qk=1.0, sigma_v=1.0):
    q = synth.normal(seed * 3 + 0, (B, H, Nq, d), sigma_qk, dtype)
    k = synth.normal(seed * 3 + 1, (B, H, Nk, d), sigma_qk, dtype)
    v = synth.normal(seed * 3 + 2, (B, H, Nk, d), sigma_v, dtype)
    return q, k, v


def run_gpu(q, k, v, causal=False, scale=None, out_dtype=None, num_splits=0, return_lse=False):
    """O (float64 numpy) from the HIP library; inputs are numpy (f32 or bf16 bits)."""
    import torch
    import paper_2606_07713_amd as moa
    tq, tk, tv = (synth.to_torch(a, "cuda") for a in (q, k, v))
    odt = None if out_dtype is None else {"f32": torch.float32, "bf16": torch.bfloat16}[out_dtype]
    r = moa.attn_fwd(tq, tk, tv, scale=scale, causal=causal, out_dtype=odt,
                     num_splits=num_splits, return_lse=return_lse)
    torch.cuda.synchronize()
    if return_lse:
        o, lse = r
        return o.float().cpu().double().numpy(), lse.cpu().double().numpy()
    return r.float().cpu().double().numpy()


def oracle_full(q, k, v, causal=False, scale=None, with_lse=False):
    return oracle.attention(q, k, v, scale=scale, causal=causal, with_lse=with_lse)


def sample_rows(B, H, Nq, n, seed=0, tile=128):
    """Flat rows (b*H + h)*Nq + i: tile edges of the first/last heads plus random rows."""
    rng = np.random.default_rng(seed)
    total = B * H * Nq
    n = min(n, total)
    edges = {min(i, Nq - 1) for i in (0, 1, Nq - 1, tile - 1, tile, Nq // 2)}
    rows = set()
    for bh in {0, B * H - 1, (B * H) // 2}:
        for i in edges:
            rows.add(bh * Nq + i)
    while len(rows) < n:
        rows.add(int(rng.integers(0, total)))
    return np.array(sorted(rows), dtype=np.int64)


def max_err(a, b):
    return float(np.max(np.abs(np.asarray(a, np.float64) - np.asarray(b, np.float64))))
