"""Strided layouts on the GPU (moa_attn_fwd_strided through attn_fwd): the same
seeded inputs stored as [B, N, H, d] views, packed QKV buffers, padded rows and
K/V shared by every head, against the oracle on the contiguous arrays.  Every
kernel family is covered: the two bf16 prefill layouts (ping-pong on a large
and on a mid-size grid, key split on a small one), fp32 prefill and decode.  The layouts are the
storage functions of the footnote to eq. gamma with per-dimension strides.

Layouts with a strided head dimension -- column-major heads ([B][H][d][N]),
rows that are not 16-byte aligned -- go through moa_attn_fwd_onf's
element-gather kernel; they are checked the same way."""
import zlib

import numpy as np
import pytest

import synth
import oracle
from gpu_util import TOL, gen, max_err, sample_rows, say

pytestmark = pytest.mark.gpu


def _seed(*parts):
    return zlib.crc32(repr(parts).encode()) % 100003


def _views(q, k, v, layout):
    """Device views [B, H, N, d] of the host arrays in the requested storage."""
    import torch
    tq, tk, tv = (synth.to_torch(a, "cuda") for a in (q, k, v))
    if layout == "contiguous":
        return tq, tk, tv
    if layout == "bshd":
        return tuple(t.transpose(1, 2).contiguous().transpose(1, 2) for t in (tq, tk, tv))
    if layout == "padded":
        out = []
        for t in (tq, tk, tv):
            d = t.shape[3]
            pad = torch.full(t.shape[:3] + (d + 8,), float("nan"), dtype=t.dtype, device=t.device)
            pad[..., :d] = t
            out.append(pad[..., :d])
        return tuple(out)
    if layout == "packed":
        B, H, N, d = tq.shape
        buf = torch.empty((B, N, 3, H, d), dtype=tq.dtype, device=tq.device)
        for i, t in enumerate((tq, tk, tv)):
            buf[:, :, i] = t.transpose(1, 2)
        return tuple(buf[:, :, i].transpose(1, 2) for i in range(3))
    if layout == "shared_kv":
        # k, v were generated with one head; every head reads it (head stride 0).
        H = tq.shape[1]
        return tq, tk.expand(-1, H, -1, -1), tv.expand(-1, H, -1, -1)
    if layout == "colmajor":
        # every head stored [d][N]: row stride 1, element stride N
        return tuple(t.transpose(2, 3).contiguous().transpose(2, 3) for t in (tq, tk, tv))
    if layout == "colmajor_k":
        return tq, tk.transpose(2, 3).contiguous().transpose(2, 3), tv
    if layout == "unaligned":
        # rows of d elements one element apart from the next row's start + 1: not 16-byte aligned
        out = []
        for t in (tq, tk, tv):
            B, H, N, d = t.shape
            buf = torch.full((B, H, N * (d + 1) + 1), float("nan"), dtype=t.dtype, device=t.device)
            view = buf[..., 1:].as_strided((B, H, N, d), (H * (N * (d + 1) + 1), N * (d + 1) + 1, d + 1, 1),
                                           buf.storage_offset() + 1)
            view.copy_(t)
            out.append(view)
        return tuple(out)
    raise ValueError(layout)


def _run(q, k, v, layout, out_layout="contiguous", causal=False, out_dtype=None, return_lse=False):
    import torch
    import paper_2606_07713_amd as moa
    tq, tk, tv = _views(q, k, v, layout)
    if layout == "packed":
        assert tk.untyped_storage().data_ptr() == tq.untyped_storage().data_ptr()
    odt = {None: tq.dtype, "f32": torch.float32, "bf16": torch.bfloat16}[out_dtype]
    B, H, Nq, dv = tq.shape[0], tq.shape[1], tq.shape[2], tv.shape[3]
    if out_layout == "bshd":
        out = torch.full((B, Nq, H, dv), float("nan"), dtype=odt, device=tq.device).transpose(1, 2)
    elif out_layout == "colmajor":
        out = torch.full((B, H, dv, Nq), float("nan"), dtype=odt, device=tq.device).transpose(2, 3)
    else:
        out = None
    r = moa.attn_fwd(tq, tk, tv, causal=causal, out_dtype=odt, out=out, return_lse=return_lse)
    torch.cuda.synchronize()
    o, lse = r if return_lse else (r, None)
    if out is not None:
        assert o.data_ptr() == out.data_ptr()
    o = o.float().cpu().double().numpy()
    return (o, lse.cpu().double().numpy()) if return_lse else o


def _inputs(B, H, Nq, Nk, d, dtype, layout, seed):
    if layout == "shared_kv":
        q, _, _ = gen(B, H, Nq, Nk, d, dtype, seed)
        _, k1, v1 = gen(B, 1, Nq, Nk, d, dtype, seed + 1)
        k = np.ascontiguousarray(np.broadcast_to(k1, (B, H, Nk, d)))
        v = np.ascontiguousarray(np.broadcast_to(v1, (B, H, Nk, d)))
        return q, k1, v1, k, v
    q, k, v = gen(B, H, Nq, Nk, d, dtype, seed)
    return q, k, v, k, v


# (B, H, Nq, Nk, d, dtype): kernel family each exercises
SHAPES = {
    "pingpong": (2, 128, 1000, 1000, 64, "bf16"),    # 1024 items of 256 queries
    "pingpong_mid": (1, 128, 600, 600, 128, "bf16"), # 384 items: 1.5 per compute unit
    "keysplit": (2, 4, 300, 300, 128, "bf16"),       # 16 items
    "f32": (2, 3, 100, 100, 64, "f32"),              # fp32 workgroup shapes by grid size:
    "f32_mid": (1, 6, 300, 300, 64, "f32"),          #   16 lanes per row above, 8 here,
    "f32_wide": (1, 4, 1000, 1000, 128, "f32"),      #   4 lanes in 16 key streams,
    "f32_large": (2, 9, 250, 600, 64, "f32"),        #   4 lanes in 8 key streams
    "decode": (4, 8, 1, 3000, 128, "bf16"),
}


@pytest.mark.parametrize("family", list(SHAPES))
@pytest.mark.parametrize("layout", ["bshd", "padded", "packed", "shared_kv"])
def test_strided_inputs_match_oracle(family, layout):
    B, H, Nq, Nk, d, dtype = SHAPES[family]
    if layout == "packed" and Nq != Nk:
        pytest.skip("packed QKV needs Nq == Nk")
    causal = family == "keysplit"
    say(f"layout {layout} family {family} {SHAPES[family]} causal={causal}")
    q, k_dev, v_dev, k, v = _inputs(B, H, Nq, Nk, d, dtype, layout, _seed(family, layout))
    out_dtype = "f32" if dtype == "bf16" else None
    o, lse = _run(q, k_dev, v_dev, layout, causal=causal, out_dtype=out_dtype, return_lse=True)
    rows = sample_rows(B, H, Nq, 192, seed=11, tile=256 if dtype == "bf16" else 64)
    ref, ref_lse = oracle.attention_rows(q, k, v, rows, causal=causal, with_lse=True)
    err = max_err(o.reshape(-1, d)[rows], ref)
    lse_err = float(np.abs(lse.reshape(-1)[rows] - ref_lse).max())
    say(f"  max err {err:.3e}  lse err {lse_err:.3e}")
    assert err <= TOL[dtype]
    lse_tol = (1e-5 * max(1.0, np.abs(ref_lse).max()) if dtype == "f32" or family == "decode"
               else 4e-3 + 1e-5 * np.abs(ref_lse).max())
    assert lse_err <= lse_tol


@pytest.mark.parametrize("family", list(SHAPES))
def test_strided_output_bshd(family):
    """O written into a [B, N, H, d] buffer; every element is written (NaN-filled first)."""
    B, H, Nq, Nk, d, dtype = SHAPES[family]
    causal = family not in ("decode", "pingpong_mid")
    q, k, v = gen(B, H, Nq, Nk, d, dtype, _seed("out", family))
    o = _run(q, k, v, "bshd", out_layout="bshd", causal=causal)
    assert not np.isnan(o).any()
    rows = sample_rows(B, H, Nq, 128, seed=12, tile=256 if dtype == "bf16" else 64)
    ref = oracle.attention_rows(q, k, v, rows, causal=causal)
    err = max_err(o.reshape(-1, d)[rows], ref)
    say(f"output bshd {family}: max err {err:.3e}")
    assert err <= TOL[dtype]


@pytest.mark.parametrize("family", list(SHAPES))
@pytest.mark.parametrize("layout", ["colmajor", "colmajor_k", "unaligned"])
def test_gathered_inputs_match_oracle(family, layout):
    """Strided head dimensions and unaligned rows (moa_attn_fwd_onf's gather kernel)."""
    B, H, Nq, Nk, d, dtype = SHAPES[family]
    causal = family in ("pingpong_mid", "keysplit", "decode")
    say(f"gathered layout {layout} family {family} {SHAPES[family]} causal={causal}")
    q, k, v = gen(B, H, Nq, Nk, d, dtype, _seed("gather", family, layout))
    for out_dtype in dict.fromkeys((dtype, "f32")):
        o, lse = _run(q, k, v, layout, causal=causal, out_dtype=out_dtype, return_lse=True)
        rows = sample_rows(B, H, Nq, 192, seed=17, tile=64)
        ref, ref_lse = oracle.attention_rows(q, k, v, rows, causal=causal, with_lse=True)
        err = max_err(o.reshape(-1, d)[rows], ref)
        lse_err = float(np.abs(lse.reshape(-1)[rows] - ref_lse).max())
        say(f"  out {out_dtype}: max err {err:.3e}  lse err {lse_err:.3e}")
        # fp32 arithmetic throughout: fp32 rounding of O (bf16 output: its own rounding)
        assert err <= (TOL[dtype] if out_dtype == "bf16" else 1e-5)
        assert lse_err <= 1e-5 * max(1.0, np.abs(ref_lse).max())


@pytest.mark.parametrize("family", list(SHAPES))
def test_gathered_output_colmajor(family):
    """O written column-major ([B][H][d][N]): every element written (NaN-filled first), from
    contiguous and from column-major inputs."""
    B, H, Nq, Nk, d, dtype = SHAPES[family]
    causal = family != "decode"
    q, k, v = gen(B, H, Nq, Nk, d, dtype, _seed("out-cm", family))
    rows = sample_rows(B, H, Nq, 128, seed=18, tile=64)
    ref = oracle.attention_rows(q, k, v, rows, causal=causal)
    for layout in ("contiguous", "colmajor"):
        o = _run(q, k, v, layout, out_layout="colmajor", causal=causal)
        assert not np.isnan(o).any()
        err = max_err(o.reshape(-1, d)[rows], ref)
        say(f"output colmajor {family} from {layout}: max err {err:.3e}")
        assert err <= TOL[dtype]


def test_strided_equals_contiguous_bitwise():
    """The same values in two storages give bit-identical outputs (no layout-dependent math)."""
    B, H, Nq, Nk, d, dtype = SHAPES["pingpong_mid"]
    q, k, v = gen(B, H, Nq, Nk, d, dtype, _seed("bits"))
    a = _run(q, k, v, "contiguous", causal=False)
    b = _run(q, k, v, "bshd", causal=False)
    assert np.array_equal(a, b)
