"""Fused scaled dot-product attention for AMD Instinct MI355X (gfx950).

A thin binding over ``libmoa_attn.so``, whose C ABI is ``include/moa_attn.h``.
The Python names mirror the C entry points (``moa_attn_fwd``,
``moa_attn_fwd_strided``, ``moa_attn_bwd``, ``moa_attn_workspace_bytes``,
``moa_attn_bwd_workspace_bytes``, ``moa_attn_num_splits``, ``moa_attn_fwd_proj``,
``moa_attn_proj_workspace_bytes``,
``moa_attn_status_string``) and only marshal arguments; every step of the
computation runs in the library's HIP kernels.  ``attn_fwd`` is a convenience
wrapper for torch tensors (torch supplies device memory and the stream).

There is no fallback: if the HIP library has not been built, importing this
package raises ``ImportError``.
"""
from __future__ import annotations

import ctypes
import math
import os

__all__ = [
    "MOA_OK", "MOA_ERR_INVALID_ARG", "MOA_ERR_UNSUPPORTED", "MOA_ERR_WORKSPACE", "MOA_ERR_HIP",
    "MOA_F32", "MOA_BF16", "MoaAttnError", "moa_attn_fwd", "moa_attn_workspace_bytes",
    "moa_attn_num_splits", "moa_attn_status_string", "moa_attn_last_hip_error", "attn_fwd",
    "moa_attn_fwd_strided", "moa_attn_bwd", "moa_attn_bwd_workspace_bytes", "attn_bwd", "LIB_PATH",
    "lib", "moa_attn_fwd_proj", "moa_attn_proj_workspace_bytes", "attn_fwd_proj",
    "moa_attn_fwd_noalloc", "MOA_ERR_SCRATCH", "MOA_NOALLOC_SCRATCH_BYTES", "moa_attn_fwd_onf",
]

MOA_OK, MOA_ERR_INVALID_ARG, MOA_ERR_UNSUPPORTED, MOA_ERR_WORKSPACE, MOA_ERR_HIP = 0, 1, 2, 3, 4
MOA_ERR_SCRATCH = 5
MOA_NOALLOC_SCRATCH_BYTES = 32 << 20
MOA_F32, MOA_BF16 = 0, 1

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libmoa_attn.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(
        f"{LIB_PATH} is missing: the HIP attention library has not been built "
        "(run `python paper_2606_07713_amd/build.py` or __graft_entry__.build()).")

# torch ships its own HIP runtime under the same soname as ROCm's.  Whichever
# is loaded first serves the whole process, so load torch's before the library
# resolves its HIP dependency: two runtimes in one process cannot share a GPU
# (kernels enqueued through the second one fail with hipErrorNoDevice).
try:
    import torch as _torch  # noqa: F401
except ImportError:  # plain C-ABI use without torch: ROCm's runtime is used
    _torch = None

lib = ctypes.CDLL(LIB_PATH)

_i64, _vp, _f32, _ci, _sz = ctypes.c_int64, ctypes.c_void_p, ctypes.c_float, ctypes.c_int, ctypes.c_size_t
lib.moa_attn_fwd.argtypes = [_vp, _vp, _vp, _vp, _vp, _i64, _i64, _i64, _i64, _i64, _i64, _f32,
                             _ci, _ci, _ci, _vp, _sz, _ci, _vp]
lib.moa_attn_fwd.restype = _ci
lib.moa_attn_fwd_strided.argtypes = [_vp, _vp, _vp, _vp, _vp, _i64, _i64, _i64, _i64, _i64, _i64,
                                     _vp, _vp, _vp, _vp, _f32, _ci, _ci, _ci, _vp, _sz, _ci, _vp]
lib.moa_attn_fwd_strided.restype = _ci
lib.moa_attn_fwd_onf.argtypes = [_vp, _vp, _vp, _vp, _vp, _i64, _i64, _i64, _i64, _i64, _i64,
                                 _vp, _vp, _vp, _vp, _f32, _ci, _ci, _ci, _vp, _sz, _ci, _vp]
lib.moa_attn_fwd_onf.restype = _ci
lib.moa_attn_fwd_noalloc.argtypes = [_vp, _vp, _vp, _vp, _vp, _i64, _i64, _i64, _i64, _i64, _i64,
                                     _f32, _ci, _ci, _ci, _ci, _vp]
lib.moa_attn_fwd_noalloc.restype = _ci
lib.moa_attn_workspace_bytes.argtypes = [_i64] * 6 + [_ci]
lib.moa_attn_workspace_bytes.restype = _sz
lib.moa_attn_num_splits.argtypes = [_i64] * 6 + [_ci]
lib.moa_attn_num_splits.restype = _ci
lib.moa_attn_bwd_workspace_bytes.argtypes = [_i64] * 6
lib.moa_attn_bwd_workspace_bytes.restype = _sz
lib.moa_attn_bwd.argtypes = [_vp] * 9 + [_i64] * 6 + [_f32, _ci, _ci, _ci, _ci, _vp, _sz, _vp]
lib.moa_attn_bwd.restype = _ci
lib.moa_attn_proj_workspace_bytes.argtypes = [_i64] * 5
lib.moa_attn_proj_workspace_bytes.restype = _sz
lib.moa_attn_fwd_proj.argtypes = [_vp] * 6 + [_i64] * 5 + [_f32, _ci, _ci, _vp, _sz, _vp]
lib.moa_attn_fwd_proj.restype = _ci
lib.moa_attn_status_string.argtypes = [_ci]
lib.moa_attn_status_string.restype = ctypes.c_char_p
lib.moa_attn_last_hip_error.argtypes = []
lib.moa_attn_last_hip_error.restype = ctypes.c_char_p


class MoaAttnError(RuntimeError):
    def __init__(self, status: int):
        self.status = status
        msg = f"moa_attn call failed: {moa_attn_status_string(status)} (status {status})"
        if status == MOA_ERR_HIP:
            msg += f": {moa_attn_last_hip_error()}"
        super().__init__(msg)


def moa_attn_status_string(status: int) -> str:
    return lib.moa_attn_status_string(int(status)).decode()


def moa_attn_last_hip_error() -> str:
    return lib.moa_attn_last_hip_error().decode()


def moa_attn_workspace_bytes(B, H, Nq, Nk, dk, dv, num_splits=0) -> int:
    return int(lib.moa_attn_workspace_bytes(B, H, Nq, Nk, dk, dv, num_splits))


def moa_attn_num_splits(B, H, Nq, Nk, dk, dv, num_splits=0) -> int:
    return int(lib.moa_attn_num_splits(B, H, Nq, Nk, dk, dv, num_splits))


def moa_attn_fwd(Q, K, V, O, LSE, B, H, Nq, Nk, dk, dv, scale, causal, in_dtype, out_dtype,
                 workspace, workspace_bytes, num_splits, stream) -> int:
    """Raw C call: pointers are ints (device addresses) or None; returns the status."""
    return int(lib.moa_attn_fwd(Q, K, V, O, LSE, B, H, Nq, Nk, dk, dv, float(scale), int(causal),
                                in_dtype, out_dtype, workspace, workspace_bytes, num_splits,
                                stream))


def _stride_array(strides):
    if strides is None:
        return None
    if len(strides) != 3:
        raise ValueError("a stride array has three entries: batch, head, row")
    return (ctypes.c_int64 * 3)(*[int(x) for x in strides])


def moa_attn_fwd_strided(Q, K, V, O, LSE, B, H, Nq, Nk, dk, dv, q_strides, k_strides, v_strides,
                         o_strides, scale, causal, in_dtype, out_dtype, workspace,
                         workspace_bytes, num_splits, stream) -> int:
    """Raw C call with per-tensor (batch, head, row) element strides (3-sequences, or None for
    the contiguous default); returns the status."""
    arrs = [_stride_array(x) for x in (q_strides, k_strides, v_strides, o_strides)]
    ptrs = [ctypes.cast(a, ctypes.c_void_p) if a is not None else None for a in arrs]
    return int(lib.moa_attn_fwd_strided(Q, K, V, O, LSE, B, H, Nq, Nk, dk, dv, *ptrs,
                                        float(scale), int(causal), in_dtype, out_dtype, workspace,
                                        workspace_bytes, num_splits, stream))


def _stride_array4(strides):
    if strides is None:
        return None
    if len(strides) != 4:
        raise ValueError("a stride array of moa_attn_fwd_onf has four entries: batch, head, row, "
                         "element")
    return (ctypes.c_int64 * 4)(*[int(x) for x in strides])


def moa_attn_fwd_onf(Q, K, V, O, LSE, B, H, Nq, Nk, dk, dv, q_strides, k_strides, v_strides,
                     o_strides, scale, causal, in_dtype, out_dtype, workspace, workspace_bytes,
                     num_splits, stream) -> int:
    """Raw C call with per-tensor (batch, head, row, element) strides (4-sequences, or None
    for the contiguous default); returns the status."""
    arrs = [_stride_array4(x) for x in (q_strides, k_strides, v_strides, o_strides)]
    ptrs = [ctypes.cast(a, ctypes.c_void_p) if a is not None else None for a in arrs]
    return int(lib.moa_attn_fwd_onf(Q, K, V, O, LSE, B, H, Nq, Nk, dk, dv, *ptrs, float(scale),
                                    int(causal), in_dtype, out_dtype, workspace, workspace_bytes,
                                    num_splits, stream))


def moa_attn_fwd_noalloc(Q, K, V, O, LSE, B, H, Nq, Nk, dk, dv, scale, causal, in_dtype,
                         out_dtype, num_splits, stream) -> int:
    """Raw C call of the forward that allocates nothing (key-split partial states go to the
    library's fixed per-GPU scratch array); pointers are ints or None; returns the status."""
    return int(lib.moa_attn_fwd_noalloc(Q, K, V, O, LSE, B, H, Nq, Nk, dk, dv, float(scale),
                                        int(causal), in_dtype, out_dtype, num_splits, stream))


def moa_attn_bwd_workspace_bytes(B, H, Nq, Nk, dk, dv) -> int:
    return int(lib.moa_attn_bwd_workspace_bytes(B, H, Nq, Nk, dk, dv))


def moa_attn_bwd(Q, K, V, O, dO, LSE, dQ, dK, dV, B, H, Nq, Nk, dk, dv, scale, causal, in_dtype,
                 o_dtype, grad_dtype, workspace, workspace_bytes, stream) -> int:
    """Raw C call of the backward pass: pointers are ints (device addresses) or None; returns
    the status."""
    return int(lib.moa_attn_bwd(Q, K, V, O, dO, LSE, dQ, dK, dV, B, H, Nq, Nk, dk, dv,
                                float(scale), int(causal), in_dtype, o_dtype, grad_dtype,
                                workspace, workspace_bytes, stream))


def _dtype_code(t):
    import torch
    if t == torch.float32:
        return MOA_F32
    if t == torch.bfloat16:
        return MOA_BF16
    raise TypeError(f"unsupported dtype {t}; use torch.float32 or torch.bfloat16")


def attn_fwd(q, k, v, scale=None, causal=False, out_dtype=None, return_lse=False,
             num_splits=0, out=None, workspace=None, stream=None):
    """Fused attention on torch device tensors shaped [B, H, N, d] (same dtype).

    The tensors may be any strided views (e.g. a [B, N, H, d] tensor viewed with
    ``.transpose(1, 2)``, slices of a packed QKV buffer, or column-major heads viewed with
    ``.transpose(2, 3)``); their strides go to ``moa_attn_fwd_onf`` and nothing is copied.  ``out`` may be
    such a view too.  Returns O [B, H, Nq, dv] (and LSE [B, H, Nq] fp32 when
    ``return_lse``).  ``scale`` defaults to 1/sqrt(dk).  Raises ``MoaAttnError`` on a
    rejected call.
    """
    import torch
    if q.dim() != 4 or k.dim() != 4 or v.dim() != 4:
        raise ValueError("q, k, v must be [B, H, N, d]")
    for t in (q, k, v):
        if not t.is_cuda:
            raise ValueError("q, k, v must be device tensors")
    if not (q.dtype == k.dtype == v.dtype):
        raise TypeError("q, k, v must share one dtype")
    B, H, Nq, dk = q.shape
    Nk, dv = k.shape[2], v.shape[3]
    if tuple(k.shape) != (B, H, Nk, dk) or tuple(v.shape) != (B, H, Nk, dv):
        raise ValueError(f"shape mismatch {tuple(q.shape)} {tuple(k.shape)} {tuple(v.shape)}")
    in_code = _dtype_code(q.dtype)
    odt = q.dtype if out_dtype is None else out_dtype
    out_code = _dtype_code(odt)
    if scale is None:
        scale = 1.0 / math.sqrt(dk)
    if out is None:
        out = torch.empty((B, H, Nq, dv), dtype=odt, device=q.device)
    elif tuple(out.shape) != (B, H, Nq, dv) or out.dtype != odt or out.device != q.device:
        raise ValueError("out must be a [B, H, Nq, dv] tensor of the output dtype")
    lse = torch.empty((B, H, Nq), dtype=torch.float32, device=q.device) if return_lse else None
    ws_bytes = moa_attn_workspace_bytes(B, H, Nq, Nk, dk, dv, num_splits)
    if in_code == MOA_F32 and Nq != 1:
        ws_bytes = 0          # fp32 prefill never splits its keys
    if ws_bytes and workspace is None:
        workspace = torch.empty(ws_bytes, dtype=torch.uint8, device=q.device)
    if stream is None:
        stream = torch.cuda.current_stream(q.device)
    ws_ptr = workspace.data_ptr() if workspace is not None else None
    ws_n = workspace.numel() * workspace.element_size() if workspace is not None else 0
    # Contiguous tensors take moa_attn_fwd directly; any other layout goes to
    # moa_attn_fwd_onf, which runs the layouts the matrix-core kernels read
    # exactly as moa_attn_fwd_strided does and the others through its gather
    # kernel.
    if q.is_contiguous() and k.is_contiguous() and v.is_contiguous() and out.is_contiguous():
        st = int(lib.moa_attn_fwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(),
                                  lse.data_ptr() if lse is not None else None, B, H, Nq, Nk, dk,
                                  dv, float(scale), int(causal), in_code, out_code, ws_ptr, ws_n,
                                  num_splits, stream.cuda_stream))
    else:
        st = moa_attn_fwd_onf(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(),
                              lse.data_ptr() if lse is not None else None, B, H, Nq, Nk, dk, dv,
                              q.stride(), k.stride(), v.stride(), out.stride(), scale,
                              causal, in_code, out_code, ws_ptr, ws_n, num_splits,
                              stream.cuda_stream)
    if st != MOA_OK:
        raise MoaAttnError(st)
    return (out, lse) if return_lse else out


def attn_bwd(q, k, v, o, lse, do, scale=None, causal=False, grad_dtype=None, workspace=None,
             stream=None):
    """Gradients (dq, dk, dv) of ``attn_fwd`` on contiguous torch device tensors.

    q, k, v, do: bf16 [B, H, N, d]; o: the forward's output (bf16 or fp32, fp32 gives a
    more accurate row sum D); lse: the forward's fp32 [B, H, Nq] LSE (``return_lse=True``).
    ``scale`` and ``causal`` must be the forward's.  ``grad_dtype`` (default fp32) is the
    storage type of the returned gradients.  Raises ``MoaAttnError`` on a rejected call.
    """
    import torch
    ts = (q, k, v, o, lse, do)
    for t in ts:
        if not t.is_cuda or not t.is_contiguous():
            raise ValueError("attn_bwd takes contiguous device tensors")
    B, H, Nq, dk = q.shape
    Nk, dv = k.shape[2], v.shape[3]
    if (tuple(k.shape) != (B, H, Nk, dk) or tuple(v.shape) != (B, H, Nk, dv)
            or tuple(o.shape) != (B, H, Nq, dv) or tuple(do.shape) != (B, H, Nq, dv)
            or tuple(lse.shape) != (B, H, Nq) or lse.dtype != torch.float32):
        raise ValueError("shape mismatch between q, k, v, o, lse and do")
    if not (q.dtype == k.dtype == v.dtype == do.dtype):
        raise TypeError("q, k, v and do must share one dtype")
    gdt = torch.float32 if grad_dtype is None else grad_dtype
    if scale is None:
        scale = 1.0 / math.sqrt(dk)
    dq = torch.empty_like(q, dtype=gdt)
    dkk = torch.empty_like(k, dtype=gdt)
    dvv = torch.empty_like(v, dtype=gdt)
    ws_bytes = moa_attn_bwd_workspace_bytes(B, H, Nq, Nk, dk, dv)
    if ws_bytes and workspace is None:
        workspace = torch.empty(ws_bytes, dtype=torch.uint8, device=q.device)
    if stream is None:
        stream = torch.cuda.current_stream(q.device)
    st = moa_attn_bwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), do.data_ptr(),
                      lse.data_ptr(), dq.data_ptr(), dkk.data_ptr(), dvv.data_ptr(),
                      B, H, Nq, Nk, dk, dv, scale, causal, _dtype_code(q.dtype),
                      _dtype_code(o.dtype), _dtype_code(gdt),
                      workspace.data_ptr() if workspace is not None else None,
                      workspace.numel() * workspace.element_size() if workspace is not None else 0,
                      stream.cuda_stream)
    if st != MOA_OK:
        raise MoaAttnError(st)
    return dq, dkk, dvv


def moa_attn_proj_workspace_bytes(B, N, Dm, H, d) -> int:
    return int(lib.moa_attn_proj_workspace_bytes(B, N, Dm, H, d))


def moa_attn_fwd_proj(X, Wq, Wk, Wv, O, LSE, B, N, Dm, H, d, scale, causal, out_dtype, workspace,
                      workspace_bytes, stream) -> int:
    """Raw C call of the projected forward: pointers are ints (device addresses) or None;
    returns the status."""
    return int(lib.moa_attn_fwd_proj(X, Wq, Wk, Wv, O, LSE, B, N, Dm, H, d, float(scale),
                                     int(causal), out_dtype, workspace, workspace_bytes, stream))


def attn_fwd_proj(x, wq, wk, wv, heads, scale=None, causal=False, out_dtype=None,
                  return_lse=False, return_qkv=False, workspace=None, stream=None):
    """Self-attention of x [B, N, Dm] (bf16) through the input projections wq, wk, wv
    ([H*d, Dm] bf16 each: the weights transposed, as a dense layer stores them) for
    ``heads`` heads.  Returns O [B, H, N, d] (default dtype bf16), then LSE [B, H, N] when
    ``return_lse``, then the projected (Q, K, V) [B, H, N, d] bf16 when ``return_qkv``.
    ``scale`` defaults to 1/sqrt(d).  Raises ``MoaAttnError`` on a rejected call."""
    import torch
    for t in (x, wq, wk, wv):
        if not t.is_cuda or not t.is_contiguous() or t.dtype != torch.bfloat16:
            raise ValueError("x, wq, wk, wv must be contiguous bf16 device tensors")
    B, N, Dm = x.shape
    F = wq.shape[0]
    if F % heads or tuple(wq.shape) != (F, Dm) or wk.shape != wq.shape or wv.shape != wq.shape:
        raise ValueError("wq, wk, wv must all be [heads*d, Dm]")
    d = F // heads
    odt = torch.bfloat16 if out_dtype is None else out_dtype
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    out = torch.empty((B, heads, N, d), dtype=odt, device=x.device)
    lse = torch.empty((B, heads, N), dtype=torch.float32, device=x.device) if return_lse else None
    need = moa_attn_proj_workspace_bytes(B, N, Dm, heads, d)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=x.device)
    if stream is None:
        stream = torch.cuda.current_stream(x.device)
    st = moa_attn_fwd_proj(x.data_ptr(), wq.data_ptr(), wk.data_ptr(), wv.data_ptr(),
                           out.data_ptr(), lse.data_ptr() if lse is not None else None,
                           B, N, Dm, heads, d, scale, causal, _dtype_code(odt),
                           workspace.data_ptr(), workspace.numel() * workspace.element_size(),
                           stream.cuda_stream)
    if st != MOA_OK:
        raise MoaAttnError(st)
    res = [out]
    if return_lse:
        res.append(lse)
    if return_qkv:
        sz = -(-(B * heads * N * d * 2) // 256) * 256
        raw = workspace.view(torch.uint8)
        res.append(tuple(raw[i * sz: i * sz + B * heads * N * d * 2].view(torch.bfloat16)
                         .view(B, heads, N, d) for i in range(3)))
    return res[0] if len(res) == 1 else tuple(res)
