"""The C-ABI library on the CPU: it loads, exports what its header declares,
and rejects invalid calls before touching the GPU (no compute calls here)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "moa_attn.h")

moa = pytest.importorskip("paper_2606_07713_amd", reason="HIP library not built")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(moa_attn_\w+)\s*\(", text)))


def test_header_declares_the_entry_points():
    names = _declared_functions()
    assert names == ["moa_attn_bwd", "moa_attn_bwd_workspace_bytes", "moa_attn_fwd",
                     "moa_attn_fwd_noalloc", "moa_attn_fwd_onf", "moa_attn_fwd_proj",
                     "moa_attn_fwd_strided",
                     "moa_attn_last_hip_error",
                     "moa_attn_num_splits", "moa_attn_proj_workspace_bytes",
                     "moa_attn_status_string", "moa_attn_workspace_bytes"]


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(moa.LIB_PATH)
    for name in _declared_functions():
        assert hasattr(lib, name), name
        assert hasattr(moa, name), f"python binding lacks {name}"


def test_header_is_plain_c():
    # The header must compile as C with no HIP include path.
    import subprocess
    import tempfile
    src = '#include "moa_attn.h"\nint main(void){return MOA_OK;}\n'
    with tempfile.TemporaryDirectory() as d:
        c = os.path.join(d, "t.c")
        open(c, "w").write(src)
        r = subprocess.run(["gcc", "-std=c99", "-Wall", "-Werror", "-I", os.path.dirname(HEADER),
                            c, "-o", os.path.join(d, "t")], capture_output=True, text=True)
        assert r.returncode == 0, r.stderr


def test_status_strings():
    assert moa.moa_attn_status_string(moa.MOA_OK) == "ok"
    for s in (1, 2, 3, 4, 5):
        assert moa.moa_attn_status_string(s) not in ("ok", "unknown status")
    assert moa.moa_attn_status_string(99) == "unknown status"
    assert moa.moa_attn_last_hip_error() == "hipSuccess"


def test_workspace_and_splits():
    # prefill grids that fill the GPU run in one pass, without workspace
    assert moa.moa_attn_workspace_bytes(2, 16, 4096, 4096, 128, 128, 0) == 0
    assert moa.moa_attn_num_splits(2, 16, 4096, 4096, 128, 128, 0) == 1
    assert moa.moa_attn_num_splits(1, 32, 16384, 16384, 128, 128, 0) == 1
    assert moa.moa_attn_num_splits(4, 8, 1024, 1024, 64, 64, 0) == 1      # short keys
    # small prefill grids with long key ranges split the keys across workgroups:
    # splits * (128-query tiles) approaches 256, with >= 1024 keys per split
    assert moa.moa_attn_num_splits(1, 32, 128, 32768, 128, 128, 0) == 8
    assert moa.moa_attn_num_splits(1, 2, 8192, 8192, 128, 128, 0) == 2
    assert moa.moa_attn_num_splits(1, 1, 64, 4096, 64, 64, 0) == 4         # capped by Nk / 1024
    ws = moa.moa_attn_workspace_bytes(1, 32, 128, 32768, 128, 128, 0)
    assert ws == 32 * 128 * 8 * 130 * 4
    # explicit prefill splits: 1 = one pass, more = that many
    assert moa.moa_attn_num_splits(1, 32, 128, 32768, 128, 128, 1) == 1
    assert moa.moa_attn_workspace_bytes(1, 32, 128, 32768, 128, 128, 1) == 0
    assert moa.moa_attn_workspace_bytes(1, 1, 100, 300, 64, 64, 3) == -(-100 * 3 * 66 * 4 // 256) * 256
    # decode: partials of bh*splits rows of (d + 2) floats, rounded up to 256 B;
    # one split writes O directly and needs none
    assert moa.moa_attn_num_splits(4, 32, 1, 32768, 128, 128, 0) == 2
    assert moa.moa_attn_workspace_bytes(4, 32, 1, 32768, 128, 128, 0) == -(-4 * 32 * 2 * 130 * 4 // 256) * 256
    assert moa.moa_attn_workspace_bytes(64, 32, 1, 8192, 128, 128, 0) == 0
    assert moa.moa_attn_workspace_bytes(64, 32, 1, 8192, 128, 128, 1) == 0
    assert moa.moa_attn_num_splits(64, 32, 1, 8192, 128, 128, 5) == 5
    assert moa.moa_attn_workspace_bytes(64, 32, 1, 8192, 128, 128, 5) >= 64 * 32 * 5 * 130 * 4
    # short key ranges are not split below the minimum chunk
    assert moa.moa_attn_num_splits(1, 1, 1, 100, 64, 64, 0) == 1
    # decode aims at one workgroup per compute unit (256): B*H*splits >= 256
    assert moa.moa_attn_num_splits(64, 32, 1, 8192, 128, 128, 0) == 1
    assert moa.moa_attn_num_splits(4, 32, 1, 32768, 128, 128, 0) == 2
    assert moa.moa_attn_num_splits(8, 8, 1, 65536, 128, 128, 0) == 4
    assert moa.moa_attn_num_splits(1, 32, 1, 131072, 128, 128, 0) == 8
    assert moa.moa_attn_num_splits(1, 1, 1, 1024, 128, 128, 0) == 4       # capped by Nk / 256
    assert moa.moa_attn_workspace_bytes(1, 1, 1, 8192, 96, 96, 0) == 0   # unsupported head


# Fake, 16-byte-aligned, non-overlapping "device" addresses: validation must
# reject every call below before it dereferences or launches anything.
A, BUF, C, D, W = 1 << 40, 2 << 40, 3 << 40, 4 << 40, 5 << 40


def _call(**kw):
    args = dict(Q=A, K=BUF, V=C, O=D, LSE=None, B=1, H=1, Nq=8, Nk=8, dk=64, dv=64, scale=0.125,
                causal=0, in_dtype=moa.MOA_BF16, out_dtype=moa.MOA_BF16, workspace=None,
                workspace_bytes=0, num_splits=0, stream=None)
    args.update(kw)
    return moa.moa_attn_fwd(**args)


@pytest.mark.parametrize("kw,status", [
    (dict(Q=None), 1), (dict(K=None), 1), (dict(V=None), 1), (dict(O=None), 1),
    (dict(B=-1), 1), (dict(H=-1), 1), (dict(Nq=-1), 1), (dict(Nk=0), 1), (dict(dk=0), 1),
    (dict(scale=float("nan")), 1), (dict(scale=float("inf")), 1),
    (dict(causal=1, Nq=9, Nk=8), 1), (dict(causal=2), 1),
    (dict(in_dtype=7), 1), (dict(out_dtype=7), 1),
    (dict(in_dtype=0, out_dtype=1), 1),                # fp32 in, bf16 out is not offered
    (dict(Q=A + 2), 1), (dict(O=D + 8), 1), (dict(LSE=D + 4), 1),
    (dict(O=A + 64), 1),                               # O overlaps Q
    (dict(num_splits=-1), 1), (dict(num_splits=257), 1),
    (dict(dk=96, dv=96), 2), (dict(dk=64, dv=128), 2), (dict(dk=256, dv=256), 2),
    (dict(Nq=1, num_splits=2), 3),                     # a split decode needs a workspace
    (dict(Nq=1, num_splits=2, workspace=W, workspace_bytes=16), 3),
    (dict(Nq=1, num_splits=2, workspace=A, workspace_bytes=1 << 20), 1),   # workspace overlaps Q
    (dict(num_splits=2), 3),                           # explicit prefill splits need a workspace
    (dict(num_splits=2, workspace=W, workspace_bytes=256), 3),
    (dict(num_splits=2, workspace=D, workspace_bytes=1 << 20), 1),   # workspace overlaps O
])
def test_validation_rejects_before_any_gpu_work(kw, status):
    assert _call(**kw) == status


def _call_strided(**kw):
    args = dict(Q=A, K=BUF, V=C, O=D, LSE=None, B=2, H=4, Nq=8, Nk=8, dk=64, dv=64,
                q_strides=None, k_strides=None, v_strides=None, o_strides=None, scale=0.125,
                causal=0, in_dtype=moa.MOA_BF16, out_dtype=moa.MOA_BF16, workspace=None,
                workspace_bytes=0, num_splits=0, stream=None)
    args.update(kw)
    return moa.moa_attn_fwd_strided(**args)


# [B, N, H, d] storage of a [B, H, N, d] view: (batch, head, row) strides.
BSHD = (8 * 4 * 64, 64, 4 * 64)


@pytest.mark.parametrize("kw,status", [
    (dict(q_strides=(-1, 64, 64)), 1),                 # negative stride
    (dict(k_strides=(4096, 512, 32)), 1),              # rows of K overlap (row stride < d)
    (dict(o_strides=(512, 0, 64)), 1),                 # O heads write the same rows
    (dict(o_strides=(64, 512, 64)), 1),                # O batches collide with rows
    (dict(q_strides=(4096, 512, 68)), 2),              # rows not 16-byte aligned (bf16)
    (dict(v_strides=(4096, 512, 1 << 28)), 2),         # in-head offsets beyond 2^31 bytes
    (dict(in_dtype=0, out_dtype=0, q_strides=(4096, 512, 66)), 2),   # fp32 rows misaligned
    (dict(O=A + 4096, q_strides=BSHD), 1),             # O inside Q's strided extent
    (dict(Q=None), 1), (dict(dk=96, dv=96), 2),        # the usual checks still apply
])
def test_strided_validation_rejects_before_any_gpu_work(kw, status):
    assert _call_strided(**kw) == status


def test_strided_accepts_common_layouts_without_gpu_work():
    # Empty batches are no-ops after validation: valid layouts return OK
    # without touching the (fake) addresses.
    for layout in (None, BSHD):
        assert _call_strided(B=0, q_strides=layout, k_strides=layout, v_strides=layout,
                             o_strides=layout) == moa.MOA_OK
    # K/V shared by all heads (head stride 0) and a padded row stride are valid.
    assert _call_strided(Nq=0, k_strides=(8 * 64, 0, 64), v_strides=(8 * 64, 0, 64),
                         q_strides=(4 * 8 * 72, 8 * 72, 72)) == moa.MOA_OK
    # A NULL stride array means the contiguous layout of moa_attn_fwd.
    assert _call_strided(B=0) == _call(B=0) == moa.MOA_OK


G, DQ, DK, DV, L = 6 << 40, 7 << 40, 8 << 40, 9 << 40, 10 << 40


def _call_bwd(**kw):
    args = dict(Q=A, K=BUF, V=C, O=D, dO=G, LSE=L, dQ=DQ, dK=DK, dV=DV, B=2, H=4, Nq=8, Nk=8,
                dk=64, dv=64, scale=0.125, causal=0, in_dtype=moa.MOA_BF16, o_dtype=moa.MOA_F32,
                grad_dtype=moa.MOA_F32, workspace=W, workspace_bytes=1 << 20, stream=None)
    args.update(kw)
    return moa.moa_attn_bwd(**args)


def test_bwd_workspace_bytes():
    # one fp32 row sum per query row, rounded up to 256 bytes
    assert moa.moa_attn_bwd_workspace_bytes(2, 16, 4096, 4096, 128, 128) == 2 * 16 * 4096 * 4
    assert moa.moa_attn_bwd_workspace_bytes(1, 1, 3, 8, 64, 64) == 256
    assert moa.moa_attn_bwd_workspace_bytes(1, 1, 0, 8, 64, 64) == 0
    assert moa.moa_attn_bwd_workspace_bytes(1, 1, 8, 8, 96, 96) == 0      # unsupported head
    assert moa.moa_attn_bwd_workspace_bytes(1, 1, 8, 0, 64, 64) == 0      # invalid Nk


@pytest.mark.parametrize("kw,status", [
    (dict(Q=None), 1), (dict(dO=None), 1), (dict(LSE=None), 1), (dict(O=None), 1),
    (dict(dQ=None), 1), (dict(dK=None), 1), (dict(dV=None), 1),
    (dict(B=-1), 1), (dict(Nk=0), 1), (dict(scale=float("nan")), 1),
    (dict(causal=1, Nq=9, Nk=8), 1), (dict(causal=3), 1),
    (dict(o_dtype=5), 1), (dict(grad_dtype=5), 1), (dict(in_dtype=5), 1),
    (dict(dO=G + 8), 1), (dict(dK=DK + 4), 1), (dict(workspace=W + 8), 1),
    (dict(dQ=A + 64), 1),                              # dQ overlaps Q
    (dict(dV=DK + 64), 1),                             # dV overlaps dK
    (dict(workspace=L), 1),                            # workspace overlaps LSE
    (dict(dK=D), 1),                                   # dK overlaps O
    (dict(in_dtype=0), 2),                             # fp32 inputs: not offered
    (dict(dk=96, dv=96), 2), (dict(dk=64, dv=128), 2),
    (dict(workspace=None), 3), (dict(workspace_bytes=16), 3),
])
def test_bwd_validation_rejects_before_any_gpu_work(kw, status):
    assert _call_bwd(**kw) == status


def test_bwd_empty_batch_is_a_no_op():
    assert _call_bwd(B=0) == moa.MOA_OK
    assert _call_bwd(H=0, workspace=None, workspace_bytes=0) == moa.MOA_OK
    # tensors without elements may be NULL
    assert _call_bwd(B=0, **{n: None for n in ("Q", "K", "V", "O", "dO", "LSE", "dQ", "dK",
                                                 "dV", "workspace")}) == moa.MOA_OK
    # with Nq == 0 the query-side tensors may be NULL, but dK and dV are still written
    assert _call_bwd(Nq=0, Q=None, O=None, dO=None, LSE=None, dQ=None, dK=None) == 1


def test_empty_problems_are_no_ops():
    # Nothing to compute: returns OK without launching (no GPU needed).
    assert _call(B=0) == moa.MOA_OK
    assert _call(H=0) == moa.MOA_OK
    assert _call(Nq=0) == moa.MOA_OK
    # fp32 prefill ignores a split request (it never splits), so an empty one is still OK
    assert _call(B=0, in_dtype=moa.MOA_F32, out_dtype=moa.MOA_F32, num_splits=4) == moa.MOA_OK


def test_one_hip_runtime_per_process():
    # The binding must leave exactly one HIP runtime mapped (torch's, when torch
    # is present), whatever was imported first.
    import subprocess
    import sys
    code = ("import paper_2606_07713_amd, torch\n"
            "paths = {l.split()[-1] for l in open('/proc/self/maps') if 'libamdhip64' in l}\n"
            "print(len(paths))\n")
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, cwd=ROOT)
    assert r.returncode == 0, r.stderr
    assert r.stdout.strip().splitlines()[-1] == "1"


X_, WQ, WK, WV = 11 << 40, 12 << 40, 13 << 40, 14 << 40


def _call_proj(**kw):
    args = dict(X=X_, Wq=WQ, Wk=WK, Wv=WV, O=D, LSE=None, B=2, N=16, Dm=128, H=2, d=64,
                scale=0.125, causal=0, out_dtype=moa.MOA_BF16, workspace=W,
                workspace_bytes=1 << 30, stream=None)
    args.update(kw)
    return moa.moa_attn_fwd_proj(**args)


def test_proj_workspace_bytes():
    # Q, K, V in bf16, each rounded up to 256 bytes, then the attention's own workspace
    qkv = 2 * 2 * 16 * 64 * 2
    assert moa.moa_attn_proj_workspace_bytes(2, 16, 128, 2, 64) == 3 * qkv
    # one token per sequence: the attention is decode-shaped and needs its partials
    one = moa.moa_attn_proj_workspace_bytes(4, 1, 128, 2, 128)
    assert one == 3 * 2048 + moa.moa_attn_workspace_bytes(4, 2, 1, 1, 128, 128, 0)
    # a small grid with a long sequence: split-K partials are included
    long_ = moa.moa_attn_proj_workspace_bytes(1, 8192, 512, 2, 128)
    assert long_ == 3 * 2 * 8192 * 128 * 2 + moa.moa_attn_workspace_bytes(1, 2, 8192, 8192, 128, 128, 0)
    assert moa.moa_attn_proj_workspace_bytes(1, 16, 100, 2, 64) == 0      # Dm not a multiple of 64
    assert moa.moa_attn_proj_workspace_bytes(1, 16, 128, 2, 96) == 0      # unsupported head


@pytest.mark.parametrize("kw,status", [
    (dict(X=None), 1), (dict(Wk=None), 1), (dict(O=None), 1),
    (dict(B=-1), 1), (dict(Dm=0), 1), (dict(scale=float("inf")), 1), (dict(causal=2), 1),
    (dict(out_dtype=3), 1), (dict(X=X_ + 8), 1), (dict(LSE=L + 4), 1),
    (dict(O=X_ + 64), 1),                              # O overlaps X
    (dict(workspace=WV + 256), 1),                     # workspace overlaps Wv
    (dict(LSE=W + 1024), 1),                           # LSE inside the workspace
    (dict(d=96), 2), (dict(Dm=96), 2),
    (dict(workspace=None), 3), (dict(workspace_bytes=1024), 3),
])
def test_proj_validation_rejects_before_any_gpu_work(kw, status):
    assert _call_proj(**kw) == status


def test_proj_empty_problems_are_no_ops():
    assert _call_proj(B=0) == moa.MOA_OK
    assert _call_proj(N=0, X=None, O=None, workspace=None) == moa.MOA_OK


def _call_noalloc(**kw):
    # Fake, far-apart, 16-byte-aligned device addresses: every call here is rejected (or
    # is empty) before anything touches them.
    base = 1 << 40
    args = dict(Q=base, K=2 * base, V=3 * base, O=4 * base, LSE=None, B=64, H=32, Nq=1,
                Nk=8192, dk=128, dv=128, scale=0.125, causal=0, in_dtype=moa.MOA_BF16,
                out_dtype=moa.MOA_BF16, num_splits=0, stream=None)
    args.update(kw)
    return moa.moa_attn_fwd_noalloc(**args)


def test_noalloc_validation():
    assert moa.MOA_NOALLOC_SCRATCH_BYTES == 32 << 20
    hdr = open(HEADER).read()
    assert "#define MOA_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)" in hdr
    # empty problems are valid no-ops; invalid arguments are rejected as by moa_attn_fwd
    assert _call_noalloc(B=0) == moa.MOA_OK
    assert _call_noalloc(Nq=0) == moa.MOA_OK
    assert _call_noalloc(Q=None) == moa.MOA_ERR_INVALID_ARG
    assert _call_noalloc(Q=(1 << 40) + 8) == moa.MOA_ERR_INVALID_ARG
    assert _call_noalloc(dk=96, dv=96) == moa.MOA_ERR_UNSUPPORTED
    assert _call_noalloc(causal=1, Nq=9000, Nk=8192) == moa.MOA_ERR_INVALID_ARG
    # decode whose partial states exceed the fixed array: 65536 heads x 2 splits x 130 floats
    need = moa.moa_attn_workspace_bytes(256, 256, 1, 512, 128, 128, 2)
    assert need > moa.MOA_NOALLOC_SCRATCH_BYTES
    assert _call_noalloc(B=256, H=256, Nk=512, num_splits=2) == moa.MOA_ERR_SCRATCH
    # explicit prefill splits beyond the array are rejected too
    need = moa.moa_attn_workspace_bytes(1, 32, 2048, 65536, 128, 128, 8)
    assert need > moa.MOA_NOALLOC_SCRATCH_BYTES
    assert _call_noalloc(H=32, B=1, Nq=2048, Nk=65536, num_splits=8) == moa.MOA_ERR_SCRATCH
    assert "MOA_NOALLOC_SCRATCH_BYTES" in moa.moa_attn_status_string(moa.MOA_ERR_SCRATCH)


def _call_onf(**kw):
    # Fake, far-apart device addresses: every call here is rejected (or empty) before
    # anything touches them.
    base = 1 << 40
    args = dict(Q=base, K=2 * base, V=3 * base, O=4 * base, LSE=None, B=2, H=4, Nq=100, Nk=300,
                dk=64, dv=64, q_strides=None, k_strides=None, v_strides=None, o_strides=None,
                scale=0.125, causal=0, in_dtype=moa.MOA_BF16, out_dtype=moa.MOA_BF16,
                workspace=None, workspace_bytes=0, num_splits=0, stream=None)
    args.update(kw)
    return moa.moa_attn_fwd_onf(**args)


def test_onf_validation():
    colmajor = lambda H, N, d: (H * d * N, d * N, 1, N)       # [B][H][d][N] storage
    # empty problems are valid no-ops on either path
    assert _call_onf(B=0) == moa.MOA_OK
    assert _call_onf(B=0, k_strides=colmajor(4, 300, 64)) == moa.MOA_OK
    assert _call_onf(Nq=0, q_strides=colmajor(4, 0, 64)) == moa.MOA_OK
    # the usual argument checks come first
    assert _call_onf(Q=None) == moa.MOA_ERR_INVALID_ARG
    assert _call_onf(dk=96, dv=96) == moa.MOA_ERR_UNSUPPORTED
    assert _call_onf(causal=1, Nq=400) == moa.MOA_ERR_INVALID_ARG
    assert _call_onf(in_dtype=7) == moa.MOA_ERR_INVALID_ARG
    # negative strides are invalid on every dimension
    for i in range(4):
        st = list(colmajor(4, 300, 64))
        st[i] = -1
        assert _call_onf(B=0 if i == 0 else 2, k_strides=tuple(st)) == moa.MOA_ERR_INVALID_ARG
    # gather path: element alignment of each pointer
    assert _call_onf(K=(2 << 40) + 1, k_strides=colmajor(4, 300, 64)) == moa.MOA_ERR_INVALID_ARG
    assert _call_onf(O=(4 << 40) + 2, out_dtype=moa.MOA_F32,
                     k_strides=colmajor(4, 300, 64)) == moa.MOA_ERR_INVALID_ARG
    # gather path: O must not write an element twice (element stride 0, overlapping rows)
    assert _call_onf(o_strides=(4 * 100 * 64, 100 * 64, 64, 0)) == moa.MOA_ERR_INVALID_ARG
    assert _call_onf(o_strides=(4 * 100 * 64, 100 * 64, 1, 1)) == moa.MOA_ERR_INVALID_ARG
    # gather path: O must not overlap an input (column-major O laid over Q's extent)
    assert _call_onf(O=(1 << 40) + 64, o_strides=colmajor(4, 100, 64),
                     k_strides=colmajor(4, 300, 64)) == moa.MOA_ERR_INVALID_ARG
    # LSE must not overlap O either
    assert _call_onf(LSE=(4 << 40) + 256, k_strides=colmajor(4, 300, 64)) == moa.MOA_ERR_INVALID_ARG
