"""Properties of the HIP path that hold at any size (closed forms, invariants,
determinism, buffer hygiene), checked through the C ABI on the GPU."""
import numpy as np
import pytest

import synth
from gpu_util import TOL, gen, max_err, oracle_full, run_gpu, say

pytestmark = pytest.mark.gpu

PATHS = [("bf16", 300, 128), ("bf16", 1, 128), ("f32", 130, 64), ("f32", 1, 64), ("bf16", 200, 64)]
PATH_IDS = ["bf16-prefill", "bf16-decode", "f32-prefill", "f32-decode", "bf16-prefill-d64"]


def _torch():
    import torch
    return torch


@pytest.mark.parametrize("dtype,Nq,d", PATHS, ids=PATH_IDS)
@pytest.mark.parametrize("causal", [False, True])
def test_constant_values(dtype, Nq, d, causal):
    Nk = 333
    q, k, _ = gen(2, 2, Nq, Nk, d, dtype, seed=5, sigma_qk=2.0)
    val = np.float32(0.625)
    v = np.full((2, 2, Nk, d), val, np.float32)
    if dtype == "bf16":
        v = synth.f32_to_bf16_bits(v)
    o = run_gpu(q, k, v, causal=causal, out_dtype="f32")
    assert max_err(o, 0.625) <= (1e-6 if dtype == "f32" else 4e-3)


@pytest.mark.parametrize("dtype,Nq,d", PATHS, ids=PATH_IDS)
@pytest.mark.parametrize("causal", [False, True])
def test_zero_query_is_mean_of_visible_values(dtype, Nq, d, causal):
    Nk = 517
    _, k, v = gen(1, 3, Nq, Nk, d, dtype, seed=6)
    q = np.zeros((1, 3, Nq, d), np.float32 if dtype == "f32" else np.uint16)
    o = run_gpu(q, k, v, causal=causal, out_dtype="f32")
    vf = (synth.bf16_bits_to_f32(v) if dtype == "bf16" else v).astype(np.float64)
    off = Nk - Nq
    for i in sorted({0, Nq // 2, Nq - 1}):
        last = min(Nk, i + off + 1) if causal else Nk
        want = vf[:, :, :last, :].mean(axis=2)
        assert max_err(o[:, :, i, :], want) <= TOL[dtype]


@pytest.mark.parametrize("dtype,Nq,d", PATHS, ids=PATH_IDS)
def test_one_hot_dominant_key(dtype, Nq, d):
    Nk, kstar = 700, 411
    qf = np.zeros((1, 2, Nq, d), np.float32)
    qf[..., 0] = 32.0
    _, kf, vf = gen(1, 2, Nq, Nk, d, "f32", seed=7)
    kf[..., 0] = 0.0
    kf[:, :, kstar, 0] = 32.0
    if dtype == "bf16":
        q, k, v = (synth.f32_to_bf16_bits(a) for a in (qf, kf, vf))
        vv = synth.bf16_bits_to_f32(v)
    else:
        q, k, v, vv = qf, kf, vf, vf
    o = run_gpu(q, k, v, out_dtype="f32")
    want = np.broadcast_to(vv[:, :, kstar:kstar + 1, :], o.shape)
    # every other weight is below e^-90: O is V[k*] up to fp32 rounding of the logits
    assert max_err(o, want) <= 1e-4 * max(1.0, np.abs(vv).max())


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("d", [64, 128])
def test_single_key_and_causal_first_row(dtype, d):
    q, k, v = gen(2, 2, 70, 1, d, dtype, seed=8)
    o = run_gpu(q, k, v, out_dtype="f32")
    vv = (synth.bf16_bits_to_f32(v) if dtype == "bf16" else v).astype(np.float64)
    assert max_err(o, np.broadcast_to(vv, o.shape)) <= 1e-6
    q, k, v = gen(2, 2, 190, 190, d, dtype, seed=9)
    o = run_gpu(q, k, v, causal=True, out_dtype="f32")
    vv = (synth.bf16_bits_to_f32(v) if dtype == "bf16" else v).astype(np.float64)
    assert max_err(o[:, :, 0, :], vv[:, :, 0, :]) <= 1e-6


@pytest.mark.parametrize("dtype,Nq,d", PATHS, ids=PATH_IDS)
@pytest.mark.parametrize("causal", [False, True])
def test_row_shift_invariance(dtype, Nq, d, causal):
    # K[..., -1] = 1, so Q[i, -1] = 2^k_i shifts every logit of row i by
    # scale * 2^k_i (exact in bf16); the softmax, hence O, must not change.
    Nk = max(260, Nq + 20)
    qf, kf, vf = gen(1, 2, Nq, Nk, d, "f32", seed=10)
    kf[..., -1] = 1.0
    qf[..., -1] = 0.0
    qb = qf.copy()
    kmax = 10 if dtype == "bf16" else 6
    qb[..., -1] = (2.0 ** (np.arange(Nq) % (kmax + 1))).astype(np.float32)[None, None, :]
    conv = synth.f32_to_bf16_bits if dtype == "bf16" else (lambda a: a)
    oa = run_gpu(conv(qf), conv(kf), conv(vf), causal=causal, out_dtype="f32")
    ob = run_gpu(conv(qb), conv(kf), conv(vf), causal=causal, out_dtype="f32")
    ref = oracle_full(conv(qf), conv(kf), conv(vf), causal=causal)
    assert max_err(oa, ref) <= TOL[dtype]
    assert max_err(ob, ref) <= TOL[dtype]


def test_decode_splits_agree():
    q, k, v = gen(4, 4, 1, 5000, 128, "bf16", seed=11)
    ref = oracle_full(q, k, v)
    outs = [run_gpu(q, k, v, out_dtype="f32", num_splits=s) for s in (1, 2, 4, 8, 16, 100)]
    for o in outs:
        assert max_err(o, ref) <= TOL["bf16"]
        assert max_err(o, outs[0]) <= 1e-5


@pytest.mark.parametrize("dtype,Nq,d", PATHS, ids=PATH_IDS)
def test_bitwise_deterministic(dtype, Nq, d):
    q, k, v = gen(2, 3, Nq, 999, d, dtype, seed=12)
    a = run_gpu(q, k, v, causal=True)
    b = run_gpu(q, k, v, causal=True)
    assert np.array_equal(a, b)


@pytest.mark.parametrize("dtype,Nq,d", PATHS, ids=PATH_IDS)
def test_output_fully_written_and_guard_bands_untouched(dtype, Nq, d):
    torch = _torch()
    import paper_2606_07713_amd as moa
    B, H, Nk = 2, 2, 321
    q, k, v = gen(B, H, Nq, Nk, d, dtype, seed=13)
    tq, tk, tv = (synth.to_torch(a, "cuda") for a in (q, k, v))
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    n = B * H * Nq * d
    pad = 64  # elements on each side (keeps 16-byte alignment)
    big = torch.full((n + 2 * pad,), float("nan"), dtype=tdt, device="cuda")
    big[:pad] = 7.0
    big[pad + n:] = -7.0
    lse_big = torch.full((B * H * Nq + 2 * pad,), 3.0, dtype=torch.float32, device="cuda")
    lse_big[pad:pad + B * H * Nq] = float("nan")
    ws_bytes = moa.moa_attn_workspace_bytes(B, H, Nq, Nk, d, d, 0)
    ws = torch.empty(max(ws_bytes, 256), dtype=torch.uint8, device="cuda")
    code = moa.MOA_F32 if dtype == "f32" else moa.MOA_BF16
    st = moa.moa_attn_fwd(tq.data_ptr(), tk.data_ptr(), tv.data_ptr(),
                          big.data_ptr() + pad * big.element_size(),
                          lse_big.data_ptr() + pad * 4, B, H, Nq, Nk, d, d, 1.0 / np.sqrt(d), 1,
                          code, code, ws.data_ptr(), ws.numel(), 0,
                          torch.cuda.current_stream().cuda_stream)
    assert st == moa.MOA_OK
    torch.cuda.synchronize()
    out = big[pad:pad + n].float()
    assert torch.isfinite(out).all()
    assert (big[:pad].float() == 7.0).all() and (big[pad + n:].float() == -7.0).all()
    assert torch.isfinite(lse_big[pad:pad + B * H * Nq]).all()
    assert (lse_big[:pad] == 3.0).all() and (lse_big[pad + B * H * Nq:] == 3.0).all()
    ref = oracle_full(q, k, v, causal=True)
    assert max_err(out.cpu().double().numpy().reshape(ref.shape), ref) <= TOL[dtype]


def test_runs_on_a_side_stream():
    torch = _torch()
    import paper_2606_07713_amd as moa
    q, k, v = gen(2, 2, 257, 257, 128, "bf16", seed=14)
    tq, tk, tv = (synth.to_torch(a, "cuda") for a in (q, k, v))
    base = moa.attn_fwd(tq, tk, tv, causal=True)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        o = moa.attn_fwd(tq, tk, tv, causal=True, stream=s)
    s.synchronize()
    torch.cuda.synchronize()
    assert torch.equal(o, base)


def test_rejected_calls_raise():
    torch = _torch()
    import paper_2606_07713_amd as moa
    x = torch.zeros((1, 1, 8, 96), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(moa.MoaAttnError) as e:
        moa.attn_fwd(x, x, x)
    assert e.value.status == moa.MOA_ERR_UNSUPPORTED
    y = torch.zeros((1, 1, 9, 64), dtype=torch.bfloat16, device="cuda")
    z = torch.zeros((1, 1, 8, 64), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(moa.MoaAttnError) as e:
        moa.attn_fwd(y, z, z, causal=True)
    assert e.value.status == moa.MOA_ERR_INVALID_ARG
