"""Parity of the HIP path with the fp64 oracle on the same seeded inputs.

Tolerances (max-abs, relative to std(V) = 1): 1e-5 for fp32 inputs, 2e-2 for
bf16 inputs.  Small and ragged shapes and the five full-size workloads are
compared element by element (the workloads in the launch configuration the
benchmark times); large layout-coverage shapes are checked on sampled rows the
oracle computes one by one.
"""
import os
import time
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
    (1, 2, 17, 64, 64),        # one full key tile: the single-tile ping-pong launch
    (1, 2, 64, 64, 128),
    (2, 9, 250, 600, 64),      # fp32: long keys on more workgroups than compute units
    (1, 4, 1000, 1000, 64),    # fp32: long keys on at most one workgroup per compute unit
    (1, 6, 300, 300, 64),      # fp32: 8 lanes per row (grid of a quarter to a half of the GPU)
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


# Grids of at least one 256-query item per compute unit (256 on MI355X) take
# the ping-pong layout, and the smaller prefill shapes above the key-split
# layout.  These cover the ping-pong layout with ragged query and key tails,
# on sampled rows.
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


MID_SHAPES = [
    # B, H, Nq, Nk, d: from one 256-query item per compute unit up to a few per unit, where the
    # layout choice weighs the ping-pong layout against the key split (uneven rounds of
    # equal-cost items without the mask); ragged query and key counts
    (2, 64, 1000, 1000, 64),
    (1, 128, 600, 700, 128),
    (4, 16, 1024, 1024, 128),
    (1, 96, 2000, 2000, 128),
    (1, 80, 1024, 1024, 128),
    (1, 80, 1000, 1030, 64),
]


@pytest.mark.parametrize("shape", MID_SHAPES, ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("causal", [False, True], ids=["full", "causal"])
def test_prefill_mid_grids_sampled(shape, causal):
    B, H, Nq, Nk, d = shape
    say(f"prefill mid-size grid {shape} causal={causal}")
    q, k, v = gen(B, H, Nq, Nk, d, "bf16", seed=_seed("mid", shape, causal))
    o, lse = run_gpu(q, k, v, causal=causal, out_dtype="f32", return_lse=True)
    rows = sample_rows(B, H, Nq, 256, seed=5, tile=256)
    ref, ref_lse = oracle.attention_rows(q, k, v, rows, causal=causal, with_lse=True)
    err = max_err(o.reshape(-1, d)[rows], ref)
    lse_err = float(np.abs(lse.reshape(-1)[rows] - ref_lse).max())
    say(f"  max err {err:.3e}  lse err {lse_err:.3e}")
    assert err <= TOL["bf16"]
    assert lse_err <= _lse_tol("bf16", ref_lse)


@pytest.mark.parametrize("causal", [False, True], ids=["full", "causal"])
def test_prefill_mid_grid_bf16_out(causal):
    B, H, Nq, Nk, d = (1, 80, 1000, 1030, 64)
    q, k, v = gen(B, H, Nq, Nk, d, "bf16", seed=_seed("mid-bf16", causal))
    o = run_gpu(q, k, v, causal=causal, out_dtype="bf16")
    rows = sample_rows(B, H, Nq, 256, seed=6, tile=256)
    ref = oracle.attention_rows(q, k, v, rows, causal=causal)
    err = max_err(o.reshape(-1, d)[rows], ref)
    say(f"prefill mid-size grid bf16 out causal={causal}: max err {err:.3e}")
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


@pytest.mark.parametrize("shape", [(1, 2, 300, 300, 64), (1, 128, 600, 700, 128),
                                   (4, 64, 1000, 1000, 64)], ids=["keysplit", "pingpong_mid", "pingpong"])
@pytest.mark.parametrize("causal", [False, True], ids=["full", "causal"])
def test_negative_scale_layouts(shape, causal):
    # A negative scale flips the sign of Q inside the kernels (after Q is
    # loaded); every bf16 prefill layout, sampled rows of the larger two.
    B, H, Nq, Nk, d = shape
    q, k, v = gen(B, H, Nq, Nk, d, "bf16", seed=_seed("neg", shape, causal))
    o = run_gpu(q, k, v, causal=causal, scale=-0.3, out_dtype="f32")
    rows = sample_rows(B, H, Nq, 256, seed=13, tile=256)
    ref = oracle.attention_rows(q, k, v, rows, scale=-0.3, causal=causal)
    err = max_err(o.reshape(-1, d)[rows], ref)
    say(f"negative scale {shape} causal={causal}: max err {err:.3e}")
    assert err <= TOL["bf16"]


# Key-split (4 items) and ping-pong (512 and 1024 items) layouts; the two
# larger grids are checked on sampled rows.
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
#
# Every output element of every workload is compared with the oracle, in the
# launch configuration bench.py times (the library's own choice of layout and
# splits).  The oracle of a workload is computed once per session and serves
# both output storage types; the long causal workload takes about 40 s of host
# time on 16 threads.

_REF_CACHE = {}


def _workload_ref(name):
    if name not in _REF_CACHE:
        _REF_CACHE.clear()          # one workload's arrays at a time
        w = synth.WORKLOADS[name]
        say(f"workload {name}: generating inputs")
        q, k, v = synth.make_inputs(w)
        threads = len(os.sched_getaffinity(0))
        say(f"  oracle, all {w.B * w.H * w.Nq} rows, {threads} threads")
        # One batch entry and a few heads per oracle call, so progress is visible.
        ref = np.empty((w.B, w.H, w.Nq, w.dv))
        ref_lse = np.empty((w.B, w.H, w.Nq))
        hs = max(1, min(w.H, (1 << 22) // max(1, w.Nq * w.Nk // (2 if w.causal else 1) // 64)))
        t0 = time.perf_counter()
        for b in range(w.B):
            for h0 in range(0, w.H, hs):
                h1 = min(w.H, h0 + hs)
                sl = (slice(b, b + 1), slice(h0, h1))
                o, l = oracle.attention(*(np.ascontiguousarray(a[sl]) for a in (q, k, v)),
                                        scale=w.scale, causal=w.causal, with_lse=True,
                                        nthreads=threads)
                ref[sl], ref_lse[sl] = o, l
                if w.Nq * w.Nk >= 1 << 24:
                    say(f"    batch {b} heads {h0}..{h1 - 1}: {time.perf_counter() - t0:.1f} s")
        _REF_CACHE[name] = (w, (q, k, v), ref, ref_lse)
    return _REF_CACHE[name]


def _check_workload(name, out_dtype):
    w, (q, k, v), ref, ref_lse = _workload_ref(name)
    say(f"workload {name} -> {out_dtype}: running GPU")
    o, lse = run_gpu(q, k, v, causal=w.causal, scale=w.scale, out_dtype=out_dtype,
                     return_lse=True)
    assert np.all(np.isfinite(o))
    err = max_err(o, ref)
    lse_err = max_err(lse, ref_lse)
    say(f"  max |O - oracle| over all {o.size} outputs: {err:.3e}; max |LSE - oracle| {lse_err:.3e}")
    assert err <= TOL[w.dtype] * w.sigma_v
    assert lse_err <= _lse_tol(w.dtype, ref_lse)


def test_workload_single_head_f32():
    _check_workload("single_head_f32_n128_d64", "f32")


@pytest.mark.parametrize("out_dtype", ["bf16", "f32"])
def test_workload_mha_d64(out_dtype):
    _check_workload("mha_b4h8_n1024_d64_bf16", out_dtype)


@pytest.mark.parametrize("out_dtype", ["bf16", "f32"])
def test_workload_causal_4k(out_dtype):
    _check_workload("causal_b2h16_n4096_d128_bf16", out_dtype)


@pytest.mark.parametrize("out_dtype", ["bf16", "f32"])
def test_workload_causal_16k_wide_logits(out_dtype):
    _check_workload("causal_long_b1h32_n16384_d128_bf16_qk_sigma3", out_dtype)


@pytest.mark.parametrize("out_dtype", ["bf16", "f32"])
def test_workload_decode(out_dtype):
    _check_workload("decode_b64h32_nk8192_d128_bf16", out_dtype)


# ------------------------------------------------ brute force on tiny shapes

TINY_N = (1, 2, 3, 5, 8, 17)


@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("causal", [False, True], ids=["full", "causal"])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_tiny_shape_grid(d, causal, dtype):
    # Every Nq, Nk in {1, 2, 3, 5, 8, 17} (causal: Nq <= Nk), two heads of two
    # batches, every element against the oracle; O in the input type and in
    # fp32.  Nq = 1 is the decode path, the rest prefill.
    worst = 0.0
    bad = []
    for nq in TINY_N:
        for nk in TINY_N:
            if causal and nq > nk:
                continue
            q, k, v = gen(2, 2, nq, nk, d, dtype, seed=_seed("tiny", nq, nk, d, causal, dtype))
            ref, ref_lse = oracle_full(q, k, v, causal=causal, with_lse=True)
            for od in sorted({dtype, "f32"}):
                o, lse = run_gpu(q, k, v, causal=causal, out_dtype=od, return_lse=True)
                err = max_err(o, ref)
                worst = max(worst, err)
                if not (err <= TOL[dtype] and max_err(lse, ref_lse) <= _lse_tol(dtype, ref_lse)):
                    bad.append((nq, nk, od, err, max_err(lse, ref_lse)))
    say(f"tiny grid d={d} causal={causal} {dtype}: worst err {worst:.3e}")
    assert not bad, bad


# ------------------------------------- the paper's worked example on the GPU

def test_worked_example_through_the_library(golden_dir):
    # Sec. "Numerical Verification": n = 3, dk = dv = 4, scores divided by
    # sqrt(4).  The head is zero-padded to d = 64 (zero columns add nothing to
    # the inner products and give zero output columns), the scale stays 1/2.
    import json
    import os
    with open(os.path.join(golden_dir, "worked_example_n3_d4.json")) as f:
        g = json.load(f)
    d = 64

    def pad(a):
        out = np.zeros((1, 1, 3, d), dtype=np.float32)
        out[0, 0, :, :4] = np.asarray(a, dtype=np.float32)
        return out
    q, k, v = pad(g["Q"]), pad(g["K"]), pad(g["V"])
    ref = oracle_full(q, k, v, scale=g["scale"])
    for dtype, tol_oracle in (("f32", 1e-5), ("bf16", 2e-2)):
        qq, kk, vv = (a if dtype == "f32" else synth.f32_to_bf16_bits(a) for a in (q, k, v))
        refd = ref if dtype == "f32" else oracle_full(qq, kk, vv, scale=g["scale"])
        o = run_gpu(qq, kk, vv, scale=g["scale"], out_dtype="f32")
        assert np.all(o[..., 4:] == 0.0)
        err = max_err(o, refd)
        table = max_err(o[0, 0, :, :4], np.asarray(g["O_table2"]))
        say(f"worked example {dtype}: |O - oracle| {err:.3e}, |O - Table 2| {table:.3e}")
        assert err <= tol_oracle
        if dtype == "f32":
            assert table <= 2e-4


# ------------------------------------------ joint K/V row permutation (non-causal)

@pytest.mark.parametrize("shape", [(1, 2, 1, 3000, 128), (2, 2, 300, 517, 64),
                                   (1, 4, 1000, 1000, 128)],
                         ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_joint_kv_row_permutation(shape, dtype):
    # Without a mask the softmax is a sum over keys: permuting the rows of K and
    # V together leaves O unchanged (up to the summation order).
    B, H, Nq, Nk, d = shape
    q, k, v = gen(B, H, Nq, Nk, d, dtype, seed=_seed("perm", shape, dtype))
    perm = np.random.default_rng(7).permutation(Nk)
    kp, vp = np.ascontiguousarray(k[:, :, perm]), np.ascontiguousarray(v[:, :, perm])
    o = run_gpu(q, k, v, out_dtype="f32")
    op = run_gpu(q, kp, vp, out_dtype="f32")
    ref = oracle_full(q, k, v)
    e1, e2, e12 = max_err(o, ref), max_err(op, ref), max_err(o, op)
    say(f"permutation {shape} {dtype}: {e1:.3e} {e2:.3e} {e12:.3e}")
    assert e1 <= TOL[dtype] and e2 <= TOL[dtype] and e12 <= TOL[dtype]
