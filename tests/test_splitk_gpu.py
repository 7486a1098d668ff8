"""Split-K prefill (keys split across workgroups, partial states merged by the
combine pass) against the fp64 oracle, element by element.

The library splits bf16 prefill automatically when the grid is too small to
fill the GPU and the key range is long; explicit ``num_splits`` forces any
split count, including shares that are empty for some (or all) rows of a
causal query tile.  Tolerances as everywhere: 2e-2 (bf16 inputs), 1e-5 (fp32).
"""
import zlib

import numpy as np
import pytest

import paper_2606_07713_amd as moa
from gpu_util import TOL, gen, max_err, oracle_full, run_gpu, say

pytestmark = pytest.mark.gpu


def _seed(*parts):
    return zlib.crc32(repr(parts).encode()) % 100003


def _lse_tol(ref_lse):
    # bf16 weights (relative error <= 2^-8) plus fp32 rounding.
    return 4e-3 + 1e-5 * np.abs(ref_lse).max()


AUTO_SHAPES = [
    # B, H, Nq, Nk, d: small grids with long key ranges -> automatic split
    (1, 2, 100, 5000, 64),
    (1, 1, 300, 3000, 128),
    (2, 2, 64, 4100, 128),
]


@pytest.mark.parametrize("shape", AUTO_SHAPES, ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("causal", [False, True], ids=["full", "causal"])
def test_automatic_split_matches_oracle(shape, causal):
    B, H, Nq, Nk, d = shape
    splits = moa.moa_attn_num_splits(B, H, Nq, Nk, d, d, 0)
    assert splits > 1, "shape meant to exercise the split path"
    say(f"split-K auto {shape} causal={causal} splits={splits}")
    q, k, v = gen(B, H, Nq, Nk, d, "bf16", seed=_seed("auto", shape, causal))
    o, lse = run_gpu(q, k, v, causal=causal, out_dtype="f32", return_lse=True)
    ref, ref_lse = oracle_full(q, k, v, causal=causal, with_lse=True)
    err = max_err(o, ref)
    say(f"  max err {err:.3e}")
    assert err <= TOL["bf16"]
    assert max_err(lse, ref_lse) <= _lse_tol(ref_lse)


FORCED = [
    # B, H, Nq, Nk, d, splits
    (1, 2, 130, 700, 128, 7),     # causal: the last share of the first tile is empty
    (2, 1, 33, 1000, 64, 3),
    (1, 1, 200, 200, 64, 16),     # more splits than key tiles: most shares empty
    (1, 3, 257, 513, 128, 2),
]


@pytest.mark.parametrize("case", FORCED, ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("causal", [False, True], ids=["full", "causal"])
@pytest.mark.parametrize("out_dtype", ["bf16", "f32"])
def test_forced_splits_match_oracle(case, causal, out_dtype):
    B, H, Nq, Nk, d, splits = case
    say(f"split-K forced {case} causal={causal} out={out_dtype}")
    q, k, v = gen(B, H, Nq, Nk, d, "bf16", seed=_seed("forced", case, causal))
    o, lse = run_gpu(q, k, v, causal=causal, out_dtype=out_dtype, num_splits=splits,
                     return_lse=True)
    ref, ref_lse = oracle_full(q, k, v, causal=causal, with_lse=True)
    err = max_err(o, ref)
    say(f"  max err {err:.3e}")
    assert err <= TOL["bf16"]
    assert max_err(lse, ref_lse) <= _lse_tol(ref_lse)


def test_split_counts_agree():
    # Every split count computes the same attention (within the bf16 tolerance of
    # the oracle), and one split is the single-pass kernel.
    B, H, Nq, Nk, d = 1, 2, 150, 2500, 128
    q, k, v = gen(B, H, Nq, Nk, d, "bf16", seed=_seed("agree"))
    ref = oracle_full(q, k, v, causal=True)
    for s in (1, 2, 5, 40):
        o = run_gpu(q, k, v, causal=True, out_dtype="f32", num_splits=s)
        err = max_err(o, ref)
        say(f"  splits={s}: max err {err:.3e}")
        assert err <= TOL["bf16"]


def test_split_on_strided_layout():
    # [B, N, H, d] inputs and output (views, no copies) through the split path.
    import torch
    import synth
    B, H, Nq, Nk, d = 1, 4, 96, 3000, 64
    q, k, v = gen(B, H, Nq, Nk, d, "bf16", seed=_seed("strided"))
    tq, tk, tv = (synth.to_torch(a, "cuda").transpose(1, 2).contiguous().transpose(1, 2)
                  for a in (q, k, v))
    out = torch.empty((B, Nq, H, d), dtype=torch.float32, device="cuda").transpose(1, 2)
    assert moa.moa_attn_num_splits(B, H, Nq, Nk, d, d, 0) > 1
    moa.attn_fwd(tq, tk, tv, out=out, out_dtype=torch.float32)
    torch.cuda.synchronize()
    err = max_err(out.cpu().double().numpy(), oracle_full(q, k, v))
    say(f"  max err {err:.3e}")
    assert err <= TOL["bf16"]


def test_fp32_prefill_ignores_split_request():
    B, H, Nq, Nk, d = 1, 1, 70, 300, 64
    q, k, v = gen(B, H, Nq, Nk, d, "f32", seed=_seed("f32"))
    o = run_gpu(q, k, v, causal=True, num_splits=4)
    assert max_err(o, oracle_full(q, k, v, causal=True)) <= TOL["f32"]
