"""Backward pass on the GPU (moa_attn_bwd through attn_bwd) against the fp64
oracle's gradients (the chain rule through the softmax Jacobian of the
paper's Stage 5), element by element.

Tolerance, derived from the arithmetic.  With exact inputs (bf16 values, the
oracle's O and LSE), the kernels' only rounding of consequence is P and dS to
bf16 (relative 2^-9 each, round to nearest even) before the gradient
contractions; fp32 accumulation and the hardware exp2 add far less.  So with
A_ij = sum_e |dO_ie| |v_je| (>= |dP_ij|) and Dabs_i = sum_j P_ij A_ij
(>= |D_i|), every element obeys
    |err dV_je| <= 2^-9 * sum_i P_ij |dO_ie|
    |err dQ_ie| <= 2^-8 * scale * sum_j P_ij (A_ij + Dabs_i) |k_je|
    |err dK_je| <= 2^-8 * scale * sum_i P_ij (A_ij + Dabs_i) |q_ie|
and the test allows 2^-7 times those sums.  Fed with this library's own
forward instead (bf16 weights: LSE within ln(1 + 2^-8), O's weights within
2^-8, O itself rounded to bf16 when stored so), the terms add to at most
3.5 * 2^-8 and the test allows 2^-6.  bf16 gradients add their own rounding,
2^-9 of the value (allowed: 2^-8).
"""
import zlib

import numpy as np
import pytest

import oracle
import synth
from gpu_util import gen, say

pytestmark = pytest.mark.gpu

TOL_ISOLATED = 2.0 ** -7
TOL_END_TO_END = 2.0 ** -6
TOL_BF16_STORE = 2.0 ** -8


def _seed(*parts):
    return zlib.crc32(repr(parts).encode()) % 100003


def _inputs(B, H, Nq, Nk, d, seed, sigma_qk=1.0):
    q, k, v = gen(B, H, Nq, Nk, d, "bf16", seed, sigma_qk=sigma_qk)
    do = synth.normal(500009 + seed, (B, H, Nq, d), 1.0, "bf16")
    return q, k, v, do


def _f64(a):
    return synth.bf16_bits_to_f32(a).astype(np.float64) if a.dtype == np.uint16 else a.astype(np.float64)


def _bounds(q, k, v, do, scale, causal):
    """Per-element error scales (bQ, bK, bV) of the tolerance above, fp64, from the oracle's P."""
    _, p, _, _ = oracle.attention_weights(q, k, v, scale=scale, causal=causal)
    qa, ka, va, ga = (np.abs(_f64(a)) for a in (q, k, v, do))
    a = ga @ np.swapaxes(va, 2, 3)                       # [B,H,Nq,Nk]: sum_e |dO_ie||v_je|
    dabs = np.sum(p * a, axis=3, keepdims=True)          # [B,H,Nq,1]
    w = p * (a + dabs)
    s = abs(float(np.float32(scale)))
    bq = s * (w @ ka)
    bk = s * (np.swapaxes(w, 2, 3) @ qa)
    bv = np.swapaxes(p, 2, 3) @ ga
    return bq, bk, bv


def _gpu_bwd(q, k, v, do, o, lse, scale, causal, o_dtype="f32", grad_dtype="f32", repeat=1):
    import torch
    import paper_2606_07713_amd as moa
    tq, tk, tv, tg = (synth.to_torch(a, "cuda") for a in (q, k, v, do))
    todt = {"f32": torch.float32, "bf16": torch.bfloat16}[o_dtype]
    if isinstance(o, np.ndarray):
        to = torch.from_numpy(o.astype(np.float32)).to("cuda").to(todt)
        tl = torch.from_numpy(lse.astype(np.float32)).to("cuda")
    else:
        to, tl = o, lse
    gdt = {"f32": torch.float32, "bf16": torch.bfloat16}[grad_dtype]
    outs = []
    for _ in range(repeat):
        g = moa.attn_bwd(tq, tk, tv, to, tl, tg, scale=scale, causal=causal, grad_dtype=gdt)
        torch.cuda.synchronize()
        outs.append(tuple(x.float().cpu().double().numpy() for x in g))
    return outs if repeat > 1 else outs[0]


def _check(got, ref, bounds, tol, names=("dQ", "dK", "dV"), bf16_store=False):
    for g, r, b, n in zip(got, ref, bounds, names):
        assert not np.isnan(g).any(), f"{n} has NaN"
        # (a zero bound, as for dQ and dK at scale 0, demands an exact zero)
        allow = (tol * b + 1e-6 * float(b.max()) + (TOL_BF16_STORE * np.abs(r) if bf16_store else 0.0)
                 + np.finfo(np.float64).tiny)
        err = np.abs(g - r)
        worst = float(np.max(err / allow))
        say(f"  {n}: max abs err {err.max():.3e}  max |ref| {np.abs(r).max():.3e}  err/allowed {worst:.3f}")
        assert worst <= 1.0, n


# (B, H, Nq, Nk, d): tile edges of both kernels (256-query and 128-key items,
# 64-row stages, 32-row steps) and ragged tails.
SHAPES = [
    (1, 2, 300, 300, 64),
    (1, 2, 1000, 1000, 128),
    (2, 1, 200, 700, 128),       # Nq < Nk: bottom-right causal offset
    (1, 3, 31, 33, 64),
    (2, 4, 1, 777, 128),         # one query per head
    (1, 1, 64, 2048, 64),
]


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("shape", SHAPES)
def test_bwd_matches_oracle(shape, causal):
    B, H, Nq, Nk, d = shape
    say(f"bwd isolated {shape} causal={causal}")
    q, k, v, do = _inputs(B, H, Nq, Nk, d, _seed("iso", shape, causal))
    scale = 1.0 / np.sqrt(d)
    o, lse = oracle.attention(q, k, v, scale=scale, causal=causal, with_lse=True)
    got = _gpu_bwd(q, k, v, do, o, lse, scale, causal)
    ref = oracle.attention_bwd(q, k, v, do, scale=scale, causal=causal)
    _check(got, ref, _bounds(q, k, v, do, scale, causal), TOL_ISOLATED)


@pytest.mark.parametrize("o_dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape,causal", [((1, 2, 1000, 1000, 128), True), ((2, 2, 300, 500, 64), False)])
def test_bwd_end_to_end_from_library_forward(shape, causal, o_dtype):
    """O and LSE from this library's forward, as a training step would use them."""
    import torch
    import paper_2606_07713_amd as moa
    B, H, Nq, Nk, d = shape
    say(f"bwd end-to-end {shape} causal={causal} O {o_dtype}")
    q, k, v, do = _inputs(B, H, Nq, Nk, d, _seed("e2e", shape, causal, o_dtype))
    tq, tk, tv = (synth.to_torch(a, "cuda") for a in (q, k, v))
    odt = {"f32": torch.float32, "bf16": torch.bfloat16}[o_dtype]
    o, lse = moa.attn_fwd(tq, tk, tv, causal=causal, out_dtype=odt, return_lse=True)
    scale = 1.0 / np.sqrt(d)
    got = _gpu_bwd(q, k, v, do, o, lse, scale, causal, o_dtype=o_dtype)
    ref = oracle.attention_bwd(q, k, v, do, scale=scale, causal=causal)
    _check(got, ref, _bounds(q, k, v, do, scale, causal), TOL_END_TO_END)


def test_bwd_bf16_gradients():
    B, H, Nq, Nk, d = 1, 2, 700, 700, 128
    q, k, v, do = _inputs(B, H, Nq, Nk, d, _seed("bf16grad"))
    scale = 1.0 / np.sqrt(d)
    o, lse = oracle.attention(q, k, v, scale=scale, causal=True, with_lse=True)
    got = _gpu_bwd(q, k, v, do, o, lse, scale, True, grad_dtype="bf16")
    ref = oracle.attention_bwd(q, k, v, do, scale=scale, causal=True)
    _check(got, ref, _bounds(q, k, v, do, scale, True), TOL_ISOLATED, bf16_store=True)


@pytest.mark.parametrize("scale", [-0.2, 0.0, 0.5])
def test_bwd_scales(scale):
    """Negative and zero scales (weights uniform at 0), and sharper softmax with sigma 3 inputs."""
    B, H, Nq, Nk, d = 1, 2, 260, 300, 64
    q, k, v, do = _inputs(B, H, Nq, Nk, d, _seed("scale", scale), sigma_qk=3.0 if scale > 0 else 1.0)
    o, lse = oracle.attention(q, k, v, scale=scale, causal=True, with_lse=True)
    got = _gpu_bwd(q, k, v, do, o, lse, scale, True)
    ref = oracle.attention_bwd(q, k, v, do, scale=scale, causal=True)
    _check(got, ref, _bounds(q, k, v, do, scale, True), TOL_ISOLATED)


def test_bwd_many_items_selected_heads():
    """More work items than resident workgroups (each walks several); heads checked on a sample."""
    B, H, Nq, Nk, d = 2, 48, 1024, 1024, 64
    q, k, v, do = _inputs(B, H, Nq, Nk, d, _seed("many"))
    scale = 1.0 / np.sqrt(d)
    o, lse = oracle.attention(q, k, v, scale=scale, causal=True, with_lse=True)
    got = _gpu_bwd(q, k, v, do, o, lse, scale, True)
    for b, h in ((0, 0), (1, 47), (0, 23), (1, 5)):
        sl = (slice(b, b + 1), slice(h, h + 1))
        qs, ks, vs, gs = (a[sl] for a in (q, k, v, do))
        say(f" head ({b}, {h})")
        ref = oracle.attention_bwd(qs, ks, vs, gs, scale=scale, causal=True)
        _check(tuple(g[sl] for g in got), ref, _bounds(qs, ks, vs, gs, scale, True), TOL_ISOLATED)


def test_bwd_deterministic():
    B, H, Nq, Nk, d = 1, 4, 600, 600, 128
    q, k, v, do = _inputs(B, H, Nq, Nk, d, _seed("det"))
    o, lse = oracle.attention(q, k, v, causal=True, with_lse=True)
    a, b = _gpu_bwd(q, k, v, do, o, lse, 1.0 / np.sqrt(d), True, repeat=2)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)


def test_bwd_without_queries_zeroes_key_gradients():
    import torch
    import paper_2606_07713_amd as moa
    B, H, Nk, d = 1, 2, 100, 64
    k = torch.randn(B, H, Nk, d, device="cuda").to(torch.bfloat16)
    v = torch.randn(B, H, Nk, d, device="cuda").to(torch.bfloat16)
    # Zero-row slices of real buffers: valid (non-NULL) pointers, no elements.
    q = torch.zeros(B, H, 1, d, device="cuda", dtype=torch.bfloat16)[:, :, :0]
    g = torch.zeros(B, H, 1, d, device="cuda", dtype=torch.bfloat16)[:, :, :0]
    o = torch.zeros(B, H, 1, d, device="cuda", dtype=torch.float32)[:, :, :0]
    lse = torch.zeros(B, H, 1, device="cuda", dtype=torch.float32)[:, :, :0]
    dq, dk, dv = moa.attn_bwd(q, k, v, o, lse, g, causal=False)
    torch.cuda.synchronize()
    assert dq.numel() == 0
    assert torch.count_nonzero(dk).item() == 0 and torch.count_nonzero(dv).item() == 0


def _bounds_rows(q, k, v, do, bh, qrows, krows, scale, causal, chunk=1024):
    """The tolerance scales of _bounds at sampled rows of head slice bh, in query chunks
    (no Nq x Nk matrix is held)."""
    B, H, Nq, d = q.shape
    Nk = k.shape[2]
    b, h = divmod(bh, H)
    Q, K, V, G = (_f64(a[b, h]) for a in (q, k, v, do))
    Ka, Va, Ga, Qa = np.abs(K), np.abs(V), np.abs(G), np.abs(Q)
    s = abs(float(np.float32(scale)))
    off = Nk - Nq
    bq = np.zeros((len(qrows), d))
    bk = np.zeros((len(krows), d))
    bv = np.zeros((len(krows), d))
    qpos = {int(i): n for n, i in enumerate(qrows)}
    for i0 in range(0, Nq, chunk):
        i1 = min(Nq, i0 + chunk)
        S = float(np.float32(scale)) * (Q[i0:i1] @ K.T)
        if causal:
            S[np.arange(Nk)[None, :] > (np.arange(i0, i1)[:, None] + off)] = -np.inf
        P = np.exp(S - S.max(axis=1, keepdims=True))
        P /= P.sum(axis=1, keepdims=True)
        dabs = np.sum((P @ Va) * Ga[i0:i1], axis=1)                 # sum_j P_ij A_ij
        Pk = P[:, krows]
        Ak = Ga[i0:i1] @ Va[krows].T
        bk += s * ((Pk * (Ak + dabs[:, None])).T @ Qa[i0:i1])
        bv += Pk.T @ Ga[i0:i1]
        for i in range(i0, i1):
            if i in qpos:
                a_row = Ga[i] @ Va.T
                bq[qpos[i]] = s * ((P[i - i0] * (a_row + dabs[i - i0])) @ Ka)
    return bq, bk, bv


def test_bwd_full_size_sampled():
    """The 16K causal workload at full size (B1 H32 d128, logits of sigma 3), as bench.py runs
    it: O and LSE from this library's forward, fp32 gradients; sampled rows of two heads
    (tile edges of both gradient kernels, the first and last rows) against the oracle."""
    import torch
    import paper_2606_07713_amd as moa
    w = synth.WORKLOADS["causal_long_b1h32_n16384_d128_bf16_qk_sigma3"]
    q, k, v = synth.make_inputs(w)
    do = synth.normal(7919, (w.B, w.H, w.Nq, w.dv), 1.0, "bf16")
    say("bwd full size: GPU forward and backward")
    tq, tk, tv, tg = (synth.to_torch(a, "cuda") for a in (q, k, v, do))
    o, lse = moa.attn_fwd(tq, tk, tv, scale=w.scale, causal=True, out_dtype=torch.float32,
                          return_lse=True)
    dq, dk, dv = moa.attn_bwd(tq, tk, tv, o, lse, tg, scale=w.scale, causal=True,
                              grad_dtype=torch.float32)
    torch.cuda.synchronize()
    qrows = np.array([0, 1, 31, 32, 255, 256, 4095, 8191, 8192, 12345, 16383])
    krows = np.array([0, 1, 127, 128, 129, 4096, 8000, 16255, 16256, 16383])
    for bh in (0, w.H - 1):
        b, h = divmod(bh, w.H)
        say(f" head {bh}: oracle on {qrows.size} query and {krows.size} key rows")
        ref = oracle.attention_bwd_rows(q, k, v, do, bh, qrows, krows, scale=w.scale, causal=True)
        got = (dq[b, h][torch.from_numpy(qrows).cuda()].double().cpu().numpy(),
               dk[b, h][torch.from_numpy(krows).cuda()].double().cpu().numpy(),
               dv[b, h][torch.from_numpy(krows).cuda()].double().cpu().numpy())
        bounds = _bounds_rows(q, k, v, do, bh, qrows, krows, w.scale, True)
        _check(got, ref, bounds, TOL_END_TO_END)
