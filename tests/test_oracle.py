"""Pins for the fp64 oracle (CPU only).

Each test checks the oracle against something other than itself: the paper's
printed worked example, a library routine (torch's fp64 scaled dot-product
attention on the CPU), closed forms, or invariants of the definition.  Between
them a dropped scale, a wrong sign, a transposed operand, a missing max
subtraction, a wrong mask orientation or alignment, or a wrong bf16 widening
fails at least one test.
"""
import json
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
import synth

torch.set_num_threads(2)


def _load(golden_dir, name):
    with open(os.path.join(golden_dir, name)) as f:
        return json.load(f)


def _as4(a):
    return np.asarray(a, dtype=np.float32)[None, None]


def _worked_example(golden_dir):
    g = _load(golden_dir, "worked_example_n3_d4.json")
    return g, _as4(g["Q"]), _as4(g["K"]), _as4(g["V"])


# ---------------------------------------------------------------- paper pins

def test_worked_example_tables(golden_dir):
    g, q, k, v = _worked_example(golden_dir)
    s, p, o, lse = oracle.attention_weights(q, k, v, scale=g["scale"])
    # Table 1: attention weights; Table 2: output (both printed to 4 d.p.)
    assert np.max(np.abs(p[0, 0] - np.array(g["P_table1"]))) < 2e-4
    assert np.max(np.abs(o[0, 0] - np.array(g["O_table2"]))) < 2e-4
    # Table 1's row sums are 1 (1.0001 is display rounding per its footnote)
    assert np.max(np.abs(p[0, 0].sum(-1) - 1.0)) < 1e-14
    assert np.max(np.abs(p[0, 0].sum(-1) - np.array(g["P_row_sums_table1"]))) <= 1.5e-4
    # the full-problem entry point gives the same O
    o2 = oracle.attention(q, k, v, scale=g["scale"])
    assert np.array_equal(o, o2)


def test_worked_example_row0_trace(golden_dir):
    g, q, k, v = _worked_example(golden_dir)
    t = _load(golden_dir, "worked_example_row0_trace.json")
    s, p, o, lse = oracle.attention_weights(q, k, v, scale=g["scale"])
    x = s[0, 0, 0]
    m = x.max()
    Z = np.exp(lse[0, 0, 0] - m)          # denominator recovered from the oracle's LSE
    exp_z = p[0, 0, 0] * Z                # numerator recovered from the oracle's weights
    assert np.max(np.abs(x / g["scale"] - np.array(t["s_unscaled"]))) < 3e-4
    assert np.max(np.abs(x - np.array(t["x_scaled"]))) < 2e-4
    assert abs(m - t["m"]) < 2e-4
    assert np.max(np.abs((x - m) - np.array(t["z"]))) < 2e-4
    assert np.max(np.abs(exp_z - np.array(t["exp_z"]))) < 2e-4
    assert abs(Z - t["Z"]) < 2e-4
    assert np.max(np.abs(p[0, 0, 0] - np.array(t["w"]))) < 2e-4
    assert np.max(np.abs(o[0, 0, 0] - np.array(t["output_row0"]))) < 2e-4


# ------------------------------------------------------------ library routine

def _torch_sdpa(q, k, v, scale, causal):
    def t(a):
        if a.dtype == np.uint16:
            return synth.to_torch(a).to(torch.float64)
        return torch.from_numpy(a).to(torch.float64)
    tq, tk, tv = t(q), t(k), t(v)
    Nq, Nk = q.shape[2], k.shape[2]
    mask = None
    if causal:
        # key k visible to query i iff k <= i + (Nk - Nq)
        i = torch.arange(Nq)[:, None]
        j = torch.arange(Nk)[None, :]
        mask = j <= i + (Nk - Nq)
    return F.scaled_dot_product_attention(tq, tk, tv, attn_mask=mask, scale=scale).numpy()


SHAPES = [
    # B, H, Nq, Nk, dk, dv
    (1, 1, 1, 1, 4, 4),
    (1, 2, 3, 5, 4, 6),
    (2, 3, 17, 17, 64, 64),
    (1, 2, 5, 31, 8, 3),
    (2, 1, 33, 64, 64, 128),
    (1, 1, 64, 64, 128, 128),
]


@pytest.mark.parametrize("shape", SHAPES)
@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_matches_torch_sdpa_fp64(shape, causal, dtype):
    B, H, Nq, Nk, dk, dv = shape
    if causal and Nq > Nk:
        pytest.skip("causal needs Nq <= Nk")
    seed = 31 * sum(shape) + (7 if causal else 0) + (1 if dtype == "bf16" else 0)
    q = synth.normal(seed, (B, H, Nq, dk), 1.0, dtype)
    k = synth.normal(seed + 1, (B, H, Nk, dk), 1.0, dtype)
    v = synth.normal(seed + 2, (B, H, Nk, dv), 1.0, dtype)
    scale = float(np.float32(1.0 / np.sqrt(dk)))
    o = oracle.attention(q, k, v, scale=scale, causal=causal)
    ref = _torch_sdpa(q, k, v, scale, causal)
    assert np.max(np.abs(o - ref)) < 1e-12


def test_torch_causal_convention_when_square():
    # With Nq == Nk the oracle's mask equals torch's own is_causal (key j <= query i).
    q = synth.normal(1, (1, 2, 9, 16), 1.0, "f32")
    k = synth.normal(2, (1, 2, 9, 16), 1.0, "f32")
    v = synth.normal(3, (1, 2, 9, 16), 1.0, "f32")
    ref = F.scaled_dot_product_attention(*(torch.from_numpy(a).double() for a in (q, k, v)),
                                         is_causal=True, scale=0.25).numpy()
    assert np.max(np.abs(oracle.attention(q, k, v, scale=0.25, causal=True) - ref)) < 1e-12


def test_weights_and_lse_match_library():
    q = synth.normal(40, (1, 2, 7, 16), 1.0, "f32")
    k = synth.normal(41, (1, 2, 11, 16), 1.0, "f32")
    v = synth.normal(42, (1, 2, 11, 5), 1.0, "f32")
    s, p, o, lse = oracle.attention_weights(q, k, v, scale=0.25)
    tq, tk = torch.from_numpy(q).double(), torch.from_numpy(k).double()
    scores = (tq @ tk.transpose(-1, -2)) * 0.25
    assert np.max(np.abs(s - scores.numpy())) < 1e-13
    assert np.max(np.abs(p - torch.softmax(scores, -1).numpy())) < 1e-14
    assert np.max(np.abs(lse - torch.logsumexp(scores, -1).numpy())) < 1e-13


def test_large_logits_stay_finite():
    # Logits of order 1e3: exp without the row-max subtraction of Step I overflows.
    q = synth.normal(50, (1, 1, 32, 64), 30.0, "f32")
    k = synth.normal(51, (1, 1, 48, 64), 30.0, "f32")
    v = synth.normal(52, (1, 1, 48, 64), 1.0, "f32")
    o, lse = oracle.attention(q, k, v, scale=0.125, with_lse=True)
    assert np.all(np.isfinite(o)) and np.all(np.isfinite(lse))
    ref = _torch_sdpa(q, k, v, 0.125, False)
    assert np.max(np.abs(o - ref)) < 1e-10


# ------------------------------------------------------ closed forms, invariants

@pytest.mark.parametrize("Nq,Nk,causal", [(16, 16, False), (16, 16, True), (5, 12, True), (9, 4, False)])
def test_zero_query_gives_mean_of_visible_values(Nq, Nk, causal):
    q = np.zeros((1, 2, Nq, 64), dtype=np.float32)
    k = synth.normal(60, (1, 2, Nk, 64), 1.0, "f32")
    v = synth.normal(61, (1, 2, Nk, 32), 1.0, "f32").astype(np.float64).astype(np.float32)
    o = oracle.attention(q, k, v, causal=causal)
    vd = v.astype(np.float64)
    for i in range(Nq):
        last = min(Nk, i + (Nk - Nq) + 1) if causal else Nk
        want = vd[:, :, :last, :].mean(axis=2)
        assert np.max(np.abs(o[:, :, i, :] - want)) < 1e-13


def test_zero_scale_gives_column_mean():
    q = synth.normal(62, (1, 1, 8, 64), 1.0, "f32")
    k = synth.normal(63, (1, 1, 10, 64), 1.0, "f32")
    v = synth.normal(64, (1, 1, 10, 64), 1.0, "f32")
    o = oracle.attention(q, k, v, scale=0.0)
    assert np.max(np.abs(o[0, 0] - v[0, 0].astype(np.float64).mean(0))) < 1e-13


def test_single_key_and_causal_first_row():
    q = synth.normal(70, (2, 2, 6, 64), 1.0, "bf16")
    k = synth.normal(71, (2, 2, 1, 64), 1.0, "bf16")
    v = synth.normal(72, (2, 2, 1, 64), 1.0, "bf16")
    o = oracle.attention(q, k, v)
    assert np.array_equal(o, np.broadcast_to(synth.bf16_bits_to_f32(v).astype(np.float64), o.shape))
    k2 = synth.normal(73, (2, 2, 6, 64), 1.0, "bf16")
    v2 = synth.normal(74, (2, 2, 6, 64), 1.0, "bf16")
    o2 = oracle.attention(q, k2, v2, causal=True)
    assert np.array_equal(o2[:, :, 0, :], synth.bf16_bits_to_f32(v2)[:, :, 0, :].astype(np.float64))


@pytest.mark.parametrize("d", [64, 128])
def test_one_hot_dominant_key(d):
    Nq, Nk, kstar = 12, 40, 17
    q = np.zeros((1, 1, Nq, d), dtype=np.float32)
    q[..., 0] = 32.0
    k = synth.normal(80, (1, 1, Nk, d), 1.0, "f32")
    k[..., 0] = 0.0
    k[0, 0, kstar, 0] = 32.0
    v = synth.normal(81, (1, 1, Nk, d), 1.0, "f32")
    o = oracle.attention(q, k, v)
    want = np.broadcast_to(v[0, 0, kstar].astype(np.float64), (Nq, d))
    assert np.max(np.abs(o[0, 0] - want)) < 1e-12


@pytest.mark.parametrize("causal", [False, True])
def test_row_shift_invariance(causal):
    # Augmented last dimension: K[..., -1] = 1, so Q[i, -1] = c adds scale*c to
    # every logit of row i; the softmax must not change.
    B, H, N, d = 1, 2, 24, 64
    q = synth.normal(90, (B, H, N, d), 1.0, "f32")
    k = synth.normal(91, (B, H, N, d), 1.0, "f32")
    v = synth.normal(92, (B, H, N, d), 1.0, "f32")
    k[..., -1] = 1.0
    q[..., -1] = 0.0
    oa = oracle.attention(q, k, v, causal=causal)
    qb = q.copy()
    qb[..., -1] = (2.0 ** (np.arange(N) % 11)).astype(np.float32)[None, None, :]
    ob = oracle.attention(qb, k, v, causal=causal)
    assert np.max(np.abs(oa - ob)) < 1e-12


def test_joint_key_value_permutation_invariance():
    q = synth.normal(100, (1, 2, 20, 64), 1.0, "f32")
    k = synth.normal(101, (1, 2, 33, 64), 1.0, "f32")
    v = synth.normal(102, (1, 2, 33, 64), 1.0, "f32")
    perm = np.random.default_rng(0).permutation(33)
    o = oracle.attention(q, k, v)
    op = oracle.attention(q, k[:, :, perm], v[:, :, perm])
    assert np.max(np.abs(o - op)) < 1e-13


def test_constant_values_give_constant_output():
    q = synth.normal(110, (1, 1, 16, 64), 2.0, "f32")
    k = synth.normal(111, (1, 1, 16, 64), 2.0, "f32")
    v = np.full((1, 1, 16, 64), 0.75, dtype=np.float32)
    for causal in (False, True):
        o = oracle.attention(q, k, v, causal=causal)
        assert np.max(np.abs(o - 0.75)) < 1e-14


def test_rows_entry_point_and_threads_agree():
    q = synth.normal(120, (2, 3, 40, 64), 1.0, "bf16")
    k = synth.normal(121, (2, 3, 40, 64), 1.0, "bf16")
    v = synth.normal(122, (2, 3, 40, 64), 1.0, "bf16")
    o1, l1 = oracle.attention(q, k, v, causal=True, nthreads=1, with_lse=True)
    o4, l4 = oracle.attention(q, k, v, causal=True, nthreads=4, with_lse=True)
    assert np.array_equal(o1, o4) and np.array_equal(l1, l4)
    rows = np.array([0, 5, 39, 40, 119, 239])
    orows, lrows = oracle.attention_rows(q, k, v, rows, causal=True, with_lse=True)
    assert np.array_equal(orows, o1.reshape(-1, 64)[rows])
    assert np.array_equal(lrows, l1.reshape(-1)[rows])


def test_rejects_bad_problems():
    q = np.zeros((1, 1, 4, 8), np.float32)
    k = np.zeros((1, 1, 3, 8), np.float32)
    with pytest.raises(ValueError):
        oracle.attention(q, k, k, causal=True)              # causal with Nq > Nk
    with pytest.raises(ValueError):
        oracle.attention(q, np.zeros((1, 1, 0, 8), np.float32), np.zeros((1, 1, 0, 8), np.float32))
    with pytest.raises(ValueError):
        oracle.attention_rows(q, k, k, [12])               # row out of range


# ---- backward pass (gradients through the softmax Jacobian) ----

def _torch_grads(q, k, v, do, scale, causal):
    """Reference gradients by torch autograd in fp64 on the CPU (explicit softmax)."""
    def t(a):
        if a.dtype == np.uint16:
            return synth.to_torch(a).to(torch.float64)
        return torch.from_numpy(a).to(torch.float64)
    tq, tk, tv, tdo = (t(a).requires_grad_(i < 3) for i, a in enumerate((q, k, v, do)))
    s = scale * (tq @ tk.transpose(-1, -2))
    if causal:
        Nq, Nk = q.shape[2], k.shape[2]
        i = torch.arange(Nq)[:, None]
        j = torch.arange(Nk)[None, :]
        s = s.masked_fill(j > i + (Nk - Nq), float("-inf"))
    o = torch.softmax(s, dim=-1) @ tv
    o.backward(tdo)
    return tq.grad.numpy(), tk.grad.numpy(), tv.grad.numpy()


@pytest.mark.parametrize("shape", [(1, 1, 5, 5, 8, 8), (2, 3, 7, 11, 16, 16), (1, 2, 9, 13, 64, 64)],
                         ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("causal", [False, True], ids=["full", "causal"])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_backward_matches_torch_autograd_fp64(shape, causal, dtype):
    B, H, Nq, Nk, dk, dv = shape
    q = synth.normal(901, (B, H, Nq, dk), 1.0, dtype)
    k = synth.normal(902, (B, H, Nk, dk), 1.0, dtype)
    v = synth.normal(903, (B, H, Nk, dv), 1.0, dtype)
    do = synth.normal(904, (B, H, Nq, dv), 1.0, dtype)
    scale = float(np.float32(1 / np.sqrt(dk)))
    dq, dk_, dv_ = oracle.attention_bwd(q, k, v, do, scale=scale, causal=causal)
    rq, rk, rv = _torch_grads(q, k, v, do, scale, causal)
    for a, b in ((dq, rq), (dk_, rk), (dv_, rv)):
        assert np.max(np.abs(a - b)) < 1e-12


def test_backward_central_differences():
    # L = sum(O * dO).  Inputs are multiples of 2^-8 so that x +- 2^-10 is exact in
    # fp32; the central difference then has truncation error O(eps^2).
    rng = np.random.default_rng(5)
    B, H, Nq, Nk, d = 1, 2, 3, 4, 4
    q, k, v, do = (np.round(rng.standard_normal(sh) * 256) / 256
                   for sh in ((B, H, Nq, d), (B, H, Nk, d), (B, H, Nk, d), (B, H, Nq, d)))
    q, k, v, do = (a.astype(np.float32) for a in (q, k, v, do))
    scale, eps = 0.5, 2.0 ** -10
    for causal in (False, True):
        grads = oracle.attention_bwd(q, k, v, do, scale=scale, causal=causal)

        def loss(qq, kk, vv):
            return float(np.sum(oracle.attention(qq, kk, vv, scale=scale, causal=causal) * do))
        for which, g in enumerate(grads):
            base = (q, k, v)[which]
            for idx in np.ndindex(base.shape):
                plus, minus = base.copy(), base.copy()
                plus[idx] += eps
                minus[idx] -= eps
                args_p = [q, k, v]
                args_m = [q, k, v]
                args_p[which], args_m[which] = plus, minus
                fd = (loss(*args_p) - loss(*args_m)) / (2 * eps)
                assert abs(fd - g[idx]) < 2e-6, (causal, which, idx, fd, g[idx])


@pytest.mark.parametrize("causal", [False, True])
def test_backward_key_gradients_sum_to_zero(causal):
    # Each row of dS sums to zero (the softmax Jacobian annihilates constants), so
    # sum_k dK[k] = scale * sum_i q_i * sum_k dS[i][k] = 0.
    B, H, Nq, Nk, d = 2, 2, 6, 9, 16
    q, k, v, do = (synth.normal(910 + i, sh, 1.0, "f32") for i, sh in
                   enumerate(((B, H, Nq, d), (B, H, Nk, d), (B, H, Nk, d), (B, H, Nq, d))))
    _, dk_, _ = oracle.attention_bwd(q, k, v, do, causal=causal)
    assert np.max(np.abs(dk_.sum(axis=2))) < 1e-12


def test_backward_constant_values():
    # Constant V rows: O is that row whatever Q and K are, so dQ = dK = 0, and
    # dV[k] = sum_i P[i][k] dO[i] with P from the forward oracle.
    B, H, Nq, Nk, d = 1, 2, 5, 7, 8
    q = synth.normal(920, (B, H, Nq, d), 1.0, "f32")
    k = synth.normal(921, (B, H, Nk, d), 1.0, "f32")
    v = np.broadcast_to(synth.normal(922, (B, H, 1, d), 1.0, "f32"), (B, H, Nk, d)).copy()
    do = synth.normal(923, (B, H, Nq, d), 1.0, "f32")
    dq, dk_, dv_ = oracle.attention_bwd(q, k, v, do, causal=True)
    assert np.max(np.abs(dq)) < 1e-13 and np.max(np.abs(dk_)) < 1e-13
    _, p, _, _ = oracle.attention_weights(q, k, v, causal=True)
    ref = np.einsum("bhik,bhic->bhkc", p, do.astype(np.float64))
    assert np.max(np.abs(dv_ - ref)) < 1e-13


def test_backward_rejects_bad_problems():
    q = synth.normal(930, (1, 1, 4, 8), 1.0, "f32")
    with pytest.raises(ValueError):
        oracle.attention_bwd(q, q, q, q[:, :, :3], causal=False)      # dO shape
    with pytest.raises(ValueError):
        oracle.attention_bwd(q, q[:, :, :3], q[:, :, :3], q, causal=True)   # causal Nq > Nk


@pytest.mark.parametrize("shape", [(1, 2, 9, 13, 16, 16), (2, 1, 40, 40, 32, 8), (1, 1, 3, 70, 64, 64)],
                         ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("causal", [False, True], ids=["full", "causal"])
def test_backward_rows_match_torch_autograd_fp64(shape, causal):
    """The sampled-rows backward (used at sequence lengths the full pass cannot reach) gives
    torch autograd's fp64 gradients at its rows, for every head slice, edge rows included."""
    B, H, Nq, Nk, dk, dv = shape
    q = synth.normal(941, (B, H, Nq, dk), 1.0, "bf16")
    k = synth.normal(942, (B, H, Nk, dk), 1.0, "bf16")
    v = synth.normal(943, (B, H, Nk, dv), 1.0, "bf16")
    do = synth.normal(944, (B, H, Nq, dv), 1.0, "bf16")
    scale = float(np.float32(1 / np.sqrt(dk)))
    rq, rk, rv = _torch_grads(q, k, v, do, scale, causal)
    qrows = np.array(sorted({0, Nq // 2, Nq - 1}))
    krows = np.array(sorted({0, 1, Nk // 3, Nk - 1}))
    for bh in range(B * H):
        b, h = divmod(bh, H)
        dq, dk_, dv_ = oracle.attention_bwd_rows(q, k, v, do, bh, qrows, krows, scale=scale,
                                                 causal=causal)
        assert np.max(np.abs(dq - rq[b, h, qrows])) < 1e-12
        assert np.max(np.abs(dk_ - rk[b, h, krows])) < 1e-12
        assert np.max(np.abs(dv_ - rv[b, h, krows])) < 1e-12


def test_backward_rows_rejects_bad_rows():
    q = synth.normal(950, (1, 2, 4, 8), 1.0, "f32")
    with pytest.raises(ValueError):
        oracle.attention_bwd_rows(q, q, q, q, 2, [0], [0])            # head slice past B*H
    with pytest.raises(ValueError):
        oracle.attention_bwd_rows(q, q, q, q, 0, [4], [0])            # query row past Nq
    with pytest.raises(ValueError):
        oracle.attention_bwd_rows(q, q, q, q, 0, [0], [-1])           # key row below 0


# ---------------------------------------------------------------- input projections

@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", [(1, 3, 8, 2, 4), (2, 5, 16, 3, 8), (1, 7, 64, 2, 64)],
                         ids=lambda s: "x".join(map(str, s)))
def test_projection_matches_library_matmul(shape, dtype):
    # The oracle's plain loops against numpy's matmul (a different implementation).
    B, N, Dm, H, d = shape
    x = synth.normal(920, (B, N, Dm), 1.0, dtype)
    wt = synth.normal(921, (H * d, Dm), 0.5, dtype)
    p = oracle.projection(x, wt, H, d)
    xf = synth.bf16_bits_to_f32(x).astype(np.float64) if dtype == "bf16" else x.astype(np.float64)
    wf = synth.bf16_bits_to_f32(wt).astype(np.float64) if dtype == "bf16" else wt.astype(np.float64)
    ref = (xf @ wf.T).reshape(B, N, H, d).transpose(0, 2, 1, 3)
    assert np.max(np.abs(p - ref)) <= 1e-12 * max(1.0, np.abs(ref).max())


def test_projection_identity_weights_select_features():
    # Wt = I (Dm = H*d): the head-split projection is X itself, regrouped by head.
    B, N, H, d = 2, 3, 2, 4
    x = synth.normal(922, (B, N, H * d), 1.0, "f32")
    p = oracle.projection(x, np.eye(H * d, dtype=np.float32), H, d)
    assert np.array_equal(p, x.astype(np.float64).reshape(B, N, H, d).transpose(0, 2, 1, 3))


def _bf16_value(bits):
    return synth.bf16_bits_to_f32(np.asarray(bits, dtype=np.uint16)).astype(np.float64)


def test_bf16_rounding_is_nearest_even_from_fp64():
    # Brute force: the result is the nearer of the two bf16 values bracketing v, and
    # on an exact tie the one with an even last significand bit.
    rng = np.random.default_rng(7)
    v = np.concatenate([rng.standard_normal(4000) * 10.0 ** rng.integers(-6, 6, 4000),
                        [0.0, -0.0, 1.0, -2.5, 3.0e30]])
    # exact ties and near-ties: midpoints between neighbouring bf16 values, nudged
    base = _bf16_value(rng.integers(0x3c00, 0x4400, 200))
    mid = base * (1.0 + 2.0 ** -8)
    v = np.concatenate([v, mid, np.nextafter(mid, np.inf), np.nextafter(mid, -np.inf)])
    got = oracle.round_bf16(v)
    f32 = v.astype(np.float32)
    bits32 = f32.view(np.uint32)
    lo_bits = (bits32 >> 16).astype(np.uint16)
    for i, x in enumerate(v):
        if x == 0.0:
            assert _bf16_value(got[i]) == 0.0
            continue
        cands = [int(lo_bits[i]) + o for o in (-1, 0, 1, 2)]
        vals = _bf16_value(cands)
        dist = np.abs(vals - x)
        best = dist.min()
        winners = [c for c, dd in zip(cands, dist) if dd == best]
        want = winners[0] if len(winners) == 1 else [c for c in winners if c % 2 == 0][0]
        assert int(got[i]) == want, (x, got[i], want)


def test_bf16_rounding_agrees_with_torch_on_fp32_values():
    # For values that are already fp32 there is no double rounding, so torch's
    # fp32 -> bf16 conversion is an independent reference.
    import torch
    x = synth.normal(923, (5000,), 3.0, "f32")
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(oracle.round_bf16(x.astype(np.float64)), ref)


def test_attention_proj_composes_projection_rounding_and_attention():
    B, N, Dm, H, d = 1, 6, 32, 2, 16
    x = synth.normal(924, (B, N, Dm), 1.0, "bf16")
    wq, wk, wv = (synth.normal(925 + i, (H * d, Dm), 0.2, "bf16") for i in range(3))
    o, q, k, v = oracle.attention_proj(x, wq, wk, wv, H, d, causal=True)
    assert np.array_equal(q, oracle.round_bf16(oracle.projection(x, wq, H, d)))
    assert np.array_equal(o, oracle.attention(q, k, v, causal=True))
    # A sequence of identical tokens gives identical V rows: every output row is that row.
    x_same = np.repeat(x[:, :1, :], N, axis=1)
    o2, _, _, v2 = oracle.attention_proj(x_same, wq, wk, wv, H, d, causal=True)
    assert np.max(np.abs(o2 - _bf16_value(v2[:, :, :1, :]))) < 1e-12
