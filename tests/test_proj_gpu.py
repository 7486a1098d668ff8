"""Projected forward (moa_attn_fwd_proj: Q, K, V = X W_Q, X W_K, X W_V on the
matrix cores, then the attention) against the fp64 oracle.

The projected tensors are checked element by element against the oracle's
exact projection rounded to bf16 (nearest even).  The kernel accumulates the
Dm products in fp32 before the same rounding, so an element may differ by the
fp32 accumulation error, at most Dm * 2^-24 * sum_k |x_k w_k| (which matters
where the sum cancels), plus one bf16 unit where that moves the sum across a
rounding boundary; the test allows 2^-7 |value| + Dm * 2^-23 * sum_k |x_k w_k|,
and checks that almost every element is bit-identical.
O is checked against the oracle's attention of its own rounded Q, K, V with the
bf16 tolerance of the attention itself (2e-2 relative to std(V) = 1: the weights
are drawn with variance 1/Dm, so the projections have unit variance).
"""
import zlib

import numpy as np
import pytest

import oracle
import synth
from gpu_util import TOL, max_err, say

pytestmark = pytest.mark.gpu


def _seed(*parts):
    return zlib.crc32(repr(parts).encode()) % 100003


def _inputs(B, N, Dm, H, d, seed):
    x = synth.normal(seed, (B, N, Dm), 1.0, "bf16")
    ws = tuple(synth.normal(seed + 1 + i, (H * d, Dm), float(1.0 / np.sqrt(Dm)), "bf16")
               for i in range(3))
    return x, ws


def _run(x, ws, H, causal, out_dtype="f32"):
    import torch
    import paper_2606_07713_amd as moa
    tx, tq, tk, tv = (synth.to_torch(a, "cuda") for a in (x, *ws))
    odt = {"f32": torch.float32, "bf16": torch.bfloat16}[out_dtype]
    o, lse, qkv = moa.attn_fwd_proj(tx, tq, tk, tv, H, causal=causal, out_dtype=odt,
                                    return_lse=True, return_qkv=True)
    torch.cuda.synchronize()
    qkv = tuple(t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16) for t in qkv)
    return o.float().cpu().double().numpy(), lse.cpu().double().numpy(), qkv


def _bf16_value(bits):
    return synth.bf16_bits_to_f32(bits).astype(np.float64)


def _check_projection(got, want, x, w, H, d):
    g, v = _bf16_value(got), _bf16_value(want)
    Dm = x.shape[2]
    absum = oracle.projection(x & np.uint16(0x7fff), w & np.uint16(0x7fff), H, d)
    bound = np.abs(v) * 2.0 ** -7 + Dm * 2.0 ** -23 * absum
    assert np.all(np.abs(g - v) <= bound), float(np.max(np.abs(g - v) - bound))
    return float(np.mean(got != want))


SHAPES = [
    # B, N, Dm, H, d
    (1, 128, 128, 2, 64),
    (2, 100, 64, 1, 64),       # ragged tokens; 3*H*d = 192: a partial feature tile
    (3, 77, 320, 3, 128),      # batches straddle token tiles
    (1, 300, 256, 4, 64),
    # H*d a multiple of 256: the one-projection-per-tile kernel
    (3, 77, 320, 2, 128),      # three feature tiles, batches straddle a ragged token tile
    (2, 300, 192, 4, 128),     # two feature tiles per projection, odd k-step count
]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("causal", [False, True], ids=["full", "causal"])
def test_projected_forward_matches_oracle(shape, causal):
    B, N, Dm, H, d = shape
    say(f"proj {shape} causal={causal}")
    x, ws = _inputs(B, N, Dm, H, d, _seed(shape, causal))
    o, lse, qkv = _run(x, ws, H, causal)
    ref_o, rq, rk, rv, ref_lse = oracle.attention_proj(x, *ws, H, d, causal=causal, with_lse=True)
    for got, want, w in zip(qkv, (rq, rk, rv), ws):
        frac = _check_projection(got, want, x, w, H, d)
        say(f"  projection: {frac:.2e} of elements differ from the rounded exact value")
        assert frac < 0.01
    err = max_err(o, ref_o)
    say(f"  max err {err:.3e}")
    assert err <= TOL["bf16"]
    assert max_err(lse, ref_lse) <= 4e-3 + 1e-5 * np.abs(ref_lse).max()


def test_projected_forward_bf16_output_and_decode_shape():
    # One token per sequence: the attention step is decode-shaped (split-K + combine).
    B, N, Dm, H, d = 4, 1, 128, 2, 128
    x, ws = _inputs(B, N, Dm, H, d, _seed("decode"))
    o, _, qkv = _run(x, ws, H, False, out_dtype="bf16")
    ref_o, rq, _, rv = oracle.attention_proj(x, *ws, H, d)
    _check_projection(qkv[0], rq, x, ws[0], H, d)
    # a single key: O is exactly that key's V row (rounded to bf16 on output)
    assert np.array_equal(o, _bf16_value(rv))
    assert max_err(o, ref_o) <= TOL["bf16"]


def test_projected_forward_long_sequence_splits_keys():
    import paper_2606_07713_amd as moa
    B, N, Dm, H, d = 1, 4096, 128, 2, 128
    assert moa.moa_attn_num_splits(B, H, N, N, d, d, 0) > 1
    x, ws = _inputs(B, N, Dm, H, d, _seed("long"))
    o, _, qkv = _run(x, ws, H, True)
    ref_o, rq, rk, rv = oracle.attention_proj(x, *ws, H, d, causal=True)
    for got, want, w in zip(qkv, (rq, rk, rv), ws):
        assert _check_projection(got, want, x, w, H, d) < 0.01
    err = max_err(o, ref_o)
    say(f"  max err {err:.3e}")
    assert err <= TOL["bf16"]


def test_projected_forward_full_size_sampled():
    """A model-sized call (B1 N4096 Dm4096 H32 d128, causal: 412 GFLOP of projections, the
    first shape of the projection measurements): every projected element of one head at
    sampled tokens, and sampled rows of that head's O and LSE, against the oracle (exact
    projections of the head, rounded to bf16, then its attention)."""
    import torch
    import paper_2606_07713_amd as moa
    B, N, Dm, H, d = 1, 4096, 4096, 32, 128
    x, ws = _inputs(B, N, Dm, H, d, _seed("full"))
    say("proj full size: GPU")
    tx, tq, tk, tv = (synth.to_torch(a, "cuda") for a in (x, *ws))
    o, lse, qkv = moa.attn_fwd_proj(tx, tq, tk, tv, H, causal=True, out_dtype=torch.float32,
                                    return_lse=True, return_qkv=True)
    torch.cuda.synchronize()
    h = 19
    toks = np.array([0, 1, 255, 256, 257, 1023, 2048, 3000, 4094, 4095])
    hs = slice(h * d, (h + 1) * d)
    say(f" head {h}: oracle projections of the head")
    exact = [oracle.projection(x, w[hs], 1, d) for w in ws]          # [1, 1, N, d] each
    for t, want, w in zip(qkv, exact, ws):
        got = t[0, h].contiguous().view(torch.int16).cpu().numpy().view(np.uint16)[toks]
        frac = _check_projection(got[None, None], oracle.round_bf16(want[:, :, toks]),
                                 x[:, toks], w[hs], 1, d)
        assert frac < 0.01
    rq, rk, rv = (oracle.round_bf16(a) for a in exact)
    say(" oracle attention rows")
    ref_o, ref_lse = oracle.attention_rows(rq, rk, rv, toks, causal=True, with_lse=True)
    got_o = o[0, h].cpu().double().numpy()[toks]
    got_lse = lse[0, h].cpu().double().numpy()[toks]
    err = max_err(got_o, ref_o)
    say(f"  max err {err:.3e}")
    assert err <= TOL["bf16"]
    assert max_err(got_lse, ref_lse) <= 4e-3 + 1e-5 * np.abs(ref_lse).max()
