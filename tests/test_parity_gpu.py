"""Parity of the HIP path with the fp64 oracle on the same seeded inputs.

Tolerances (max-abs, relative to std(V) = 1): 1e-5 for fp32 inputs, 2e-2 for
bf16 inputs.  Small and ragged shapes are compared element by element; the
full-size workloads run in the launch configuration the benchmark times and
are checked on sampled rows the oracle computes one by one.
"""
import zlib

import numpy as np
import pytest

import synth
from gpu_util import TOL, gen, max_err, oracle_full, run_gpu, sample_rows, say
import oracle

pytestmark = pytest.mark.gpu


def _seed(*parts):
    return zlib.crc32(repr(parts).encode()) % 100003


# ---------------------------------------------------------------- small shapes

PREFILL_SHAPES = [
    # B, H, Nq, Nk, d
    (1, 1, 2, 2, 64),
    (1, 2, 17, 17, 64),
    (2, 2, 63, 65, 128),
    (1, 3, 129, 127, 64),      # Nq > Nk (non-causal only)
    (1, 2, 128, 128, 128),
    (2, 1, 200, 1000, 128),    # Nq < Nk: causal is bottom-right aligned
    (1, 1, 1000, 1000, 64),
    (1, 2, 300, 300, 128),
]


@pytest.mark.parametrize("shape", PREFILL_SHAPES, ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("causal", [False, True], ids=["full", "causal"])
@pytest.mark.parametrize("dtype,out_dtype", [("bf16", "bf16"), ("bf16", "f32"), ("f32", "f32")])
def test_prefill_matches_oracle(shape, causal, dtype, out_dtype):
    B, H, Nq, Nk, d = shape
    if causal and Nq > Nk:
        pytest.skip("causal requires Nq <= Nk")
    say(f"prefill {shape} causal={causal} {dtype}->{out_dtype}")
    q, k, v = gen(B, H, Nq, Nk, d, dtype, seed=_seed(shape, causal, dtype))
    o, lse = run_gpu(q, k, v, causal=causal, out_dtype=out_dtype, return_lse=True)
    ref, ref_lse = oracle_full(q, k, v, causal=causal, with_lse=True)
    err = max_err(o, ref)
    say(f"  max err {err:.3e}")
    assert err <= TOL[dtype]
    assert max_err(lse, ref_lse) <= _lse_tol(dtype, ref_lse)


def _lse_tol(dtype, ref_lse):
    # fp32 path: fp32 rounding of the logits.  bf16 path: the denominator is the
    # sum of the bf16-rounded weights that also multiply V (relative error at
    # most 2^-8), so LSE is within ln(1 + 2^-8) < 4e-3 plus fp32 rounding.
    if dtype == "f32":
        return 1e-5 * max(1.0, np.abs(ref_lse).max())
    return 4e-3 + 1e-5 * np.abs(ref_lse).max()


# Grids of >= 1024 work items of 256 queries take the ping-pong layout, grids
# of at least one item per compute unit (256 on MI355X) the per-wave pipelined
# kernel, and the smaller prefill shapes above the key-split layout.  These
# cover the two larger layouts with ragged query and key tails, on sampled
# rows.
PINGPONG_SHAPES = [
    # B, H, Nq, Nk, d
    (4, 64, 1000, 1000, 64),
    (2, 128, 1000, 1100, 128),
    (1, 256, 1024, 1024, 128),
]


@pytest.mark.parametrize("shape", PINGPONG_SHAPES, ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("causal", [False, True], ids=["full", "causal"])
def test_prefill_pingpong_layout_sampled(shape, causal):
    B, H, Nq, Nk, d = shape
    say(f"prefill ping-pong {shape} causal={causal}")
    q, k, v = gen(B, H, Nq, Nk, d, "bf16", seed=_seed("pp", shape, causal))
    o = run_gpu(q, k, v, causal=causal, out_dtype="f32")
    rows = sample_rows(B, H, Nq, 256, seed=3, tile=256)
    ref = oracle.attention_rows(q, k, v, rows, causal=causal)
    err = max_err(o.reshape(-1, d)[rows], ref)
    say(f"  max err {err:.3e}")
    assert err <= TOL["bf16"]


PIPE_SHAPES = [
    # B, H, Nq, Nk, d   (256 <= B*H*ceil(Nq/256) < 1024)
    (2, 64, 1000, 1000, 64),
    (1, 128, 600, 700, 128),
    (4, 16, 1024, 1024, 128),
    (1, 96, 2000, 2000, 128),
]


@pytest.mark.parametrize("shape", PIPE_SHAPES, ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("causal", [False, True], ids=["full", "causal"])
def test_prefill_pipe_layout_sampled(shape, causal):
    B, H, Nq, Nk, d = shape
    say(f"prefill pipelined {shape} causal={causal}")
    q, k, v = gen(B, H, Nq, Nk, d, "bf16", seed=_seed("pipe", shape, causal))
    o, lse = run_gpu(q, k, v, causal=causal, out_dtype="f32", return_lse=True)
    rows = sample_rows(B, H, Nq, 256, seed=5, tile=256)
    ref, ref_lse = oracle.attention_rows(q, k, v, rows, causal=causal, with_lse=True)
    err = max_err(o.reshape(-1, d)[rows], ref)
    lse_err = float(np.abs(lse.reshape(-1)[rows] - ref_lse).max())
    say(f"  max err {err:.3e}  lse err {lse_err:.3e}")
    assert err <= TOL["bf16"]
    assert lse_err <= _lse_tol("bf16", ref_lse)


@pytest.mark.parametrize("causal", [False, True], ids=["full", "causal"])
def test_prefill_pipe_layout_bf16_out(causal):
    B, H, Nq, Nk, d = (1, 128, 600, 700, 128)
    q, k, v = gen(B, H, Nq, Nk, d, "bf16", seed=_seed("pipe-bf16", causal))
    o = run_gpu(q, k, v, causal=causal, out_dtype="bf16")
    rows = sample_rows(B, H, Nq, 256, seed=6, tile=256)
    ref = oracle.attention_rows(q, k, v, rows, causal=causal)
    err = max_err(o.reshape(-1, d)[rows], ref)
    say(f"prefill pipelined bf16 out causal={causal}: max err {err:.3e}")
    assert err <= TOL["bf16"]


DECODE_CASES = [
    # B, H, Nk, d, splits
    (1, 1, 1, 64, 0),
    (2, 3, 7, 128, 0),
    (2, 2, 100, 64, 3),
    (3, 2, 1000, 128, 0),
    (3, 2, 1000, 128, 16),
    (1, 4, 8192, 128, 0),
    (2, 2, 4097, 64, 5),
]


@pytest.mark.parametrize("case", DECODE_CASES, ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("dtype,out_dtype", [("bf16", "bf16"), ("bf16", "f32"), ("f32", "f32")])
@pytest.mark.parametrize("causal", [False, True], ids=["full", "causal"])
def test_decode_matches_oracle(case, dtype, out_dtype, causal):
    B, H, Nk, d, splits = case
    say(f"decode {case} {dtype}->{out_dtype} causal={causal}")
    q, k, v = gen(B, H, 1, Nk, d, dtype, seed=_seed(case, dtype))
    o, lse = run_gpu(q, k, v, causal=causal, out_dtype=out_dtype, num_splits=splits, return_lse=True)
    ref, ref_lse = oracle_full(q, k, v, causal=causal, with_lse=True)
    err = max_err(o, ref)
    say(f"  max err {err:.3e}")
    assert err <= TOL[dtype]
    assert max_err(lse, ref_lse) <= _lse_tol(dtype, ref_lse)


@pytest.mark.parametrize("scale", [0.0, -0.125, 0.3])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("nq", [1, 77])
def test_unusual_scales(scale, dtype, nq):
    say(f"scale {scale} {dtype} nq={nq}")
    q, k, v = gen(2, 2, nq, 150, 64, dtype, seed=17)
    o = run_gpu(q, k, v, causal=True, scale=scale, out_dtype="f32")
    ref = oracle_full(q, k, v, causal=True, scale=scale)
    assert max_err(o, ref) <= TOL[dtype]


# Key-split (4 items), per-wave pipelined (512 items) and ping-pong (1024 items)
# layouts; the two larger ones are checked on sampled rows.
EXTREME_SHAPES = [
    # B, H, Nq, Nk, d
    (2, 2, 77, 700, 128),
    (1, 2, 300, 300, 64),
    (2, 64, 1000, 1000, 64),
    (4, 64, 1000, 1000, 64),
]


@pytest.mark.parametrize("scale", [4.0, 16.0])
@pytest.mark.parametrize("shape", EXTREME_SHAPES, ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("causal", [False, True], ids=["full", "causal"])
def test_extreme_logit_spread(scale, shape, causal):
    # Logits with a standard deviation of 45 to 260 log2 units per row: the
    # running reference is raised again and again (each raise set well above
    # the tile max that caused it), most weights underflow, and the result is
    # close to a one-hot pick of each row's top keys.  bf16 inputs: the path
    # whose softmax keeps the lazily raised reference.
    B, H, Nq, Nk, d = shape
    say(f"extreme logits scale={scale} {shape} causal={causal}")
    q, k, v = gen(B, H, Nq, Nk, d, "bf16", seed=4242 + Nq + H)
    o, lse = run_gpu(q, k, v, causal=causal, scale=scale, out_dtype="f32", return_lse=True)
    assert np.all(np.isfinite(o)) and np.all(np.isfinite(lse))
    if B * H * Nq <= 1024:
        ref, ref_lse = oracle_full(q, k, v, causal=causal, scale=scale, with_lse=True)
    else:
        rows = sample_rows(B, H, Nq, 256, seed=11, tile=256)
        ref, ref_lse = oracle.attention_rows(q, k, v, rows, scale=scale, causal=causal,
                                             with_lse=True)
        o, lse = o.reshape(-1, d)[rows], lse.reshape(-1)[rows]
    err = max_err(o, ref)
    say(f"  max err {err:.3e}")
    assert err <= TOL["bf16"]
    assert max_err(lse, ref_lse) <= _lse_tol("bf16", ref_lse)


# -------------------------------------------------------- full-size workloads

def _check_workload(name, n_rows, out_dtype):
    w = synth.WORKLOADS[name]
    say(f"workload {name} -> {out_dtype}: generating inputs")
    q, k, v = synth.make_inputs(w)
    say("  running GPU")
    o = run_gpu(q, k, v, causal=w.causal, scale=w.scale, out_dtype=out_dtype)
    assert np.all(np.isfinite(o))
    if n_rows is None:
        say("  oracle (all rows)")
        ref = oracle.attention(q, k, v, scale=w.scale, causal=w.causal)
        err = max_err(o, ref)
    else:
        rows = sample_rows(w.B, w.H, w.Nq, n_rows)
        say(f"  oracle ({rows.size} sampled rows)")
        ref = oracle.attention_rows(q, k, v, rows, scale=w.scale, causal=w.causal)
        err = max_err(o.reshape(-1, w.dv)[rows], ref)
    say(f"  max err {err:.3e}")
    assert err <= TOL[w.dtype] * w.sigma_v


def test_workload_single_head_f32():
    _check_workload("single_head_f32_n128_d64", None, "f32")


@pytest.mark.parametrize("out_dtype", ["bf16", "f32"])
def test_workload_mha_d64(out_dtype):
    _check_workload("mha_b4h8_n1024_d64_bf16", None, out_dtype)


@pytest.mark.parametrize("out_dtype", ["bf16", "f32"])
def test_workload_causal_4k(out_dtype):
    _check_workload("causal_b2h16_n4096_d128_bf16", 384, out_dtype)


@pytest.mark.parametrize("out_dtype", ["bf16", "f32"])
def test_workload_causal_16k_wide_logits(out_dtype):
    _check_workload("causal_long_b1h32_n16384_d128_bf16_qk_sigma3", 192, out_dtype)


@pytest.mark.parametrize("out_dtype", ["bf16", "f32"])
def test_workload_decode(out_dtype):
    _check_workload("decode_b64h32_nk8192_d128_bf16", 512, out_dtype)
