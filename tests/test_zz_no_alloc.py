"""moa_attn_fwd_noalloc through the C ABI: the forward whose key-split partial
states go to the library's fixed per-GPU scratch array instead of a caller
workspace.  Its output must equal moa_attn_fwd's (same kernels) bit for bit,
and the oracle's within the usual tolerances, on consecutive calls that share
the array, the second one smaller than the first."""
import numpy as np
import pytest

import synth
from gpu_util import TOL, gen, max_err, oracle_full, say

pytestmark = pytest.mark.gpu


def _noalloc(q, k, v, causal, out_dtype, num_splits, with_lse=True):
    import torch
    import paper_2606_07713_amd as moa
    B, H, Nq, dk = q.shape
    Nk, dv = k.shape[2], v.shape[3]
    out = torch.empty((B, H, Nq, dv), dtype=out_dtype, device=q.device)
    lse = torch.empty((B, H, Nq), dtype=torch.float32, device=q.device) if with_lse else None
    code = {torch.float32: moa.MOA_F32, torch.bfloat16: moa.MOA_BF16}
    st = moa.moa_attn_fwd_noalloc(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(),
                                  lse.data_ptr() if lse is not None else None, B, H, Nq, Nk, dk,
                                  dv, 1.0 / np.sqrt(dk), int(causal), code[q.dtype],
                                  code[out_dtype], num_splits,
                                  torch.cuda.current_stream().cuda_stream)
    assert st == moa.MOA_OK, moa.moa_attn_status_string(st)
    return out, lse


# (B, H, Nq, Nk, d, dtype, causal, num_splits): each pair runs a large call, then a smaller
# one of the same kind on the same array.
PAIRS = [
    [(4, 16, 1, 8192, 128, "bf16", False, 0), (3, 5, 1, 1000, 64, "bf16", True, 0)],
    [(2, 16, 1, 4096, 128, "f32", False, 0), (1, 3, 1, 700, 128, "f32", False, 0)],
    [(1, 8, 300, 9000, 128, "bf16", True, 0), (1, 2, 100, 2500, 64, "bf16", False, 3)],
    [(2, 4, 129, 4096, 64, "bf16", False, 6), (1, 1, 40, 1500, 128, "bf16", True, 2)],
]


@pytest.mark.parametrize("pair", PAIRS, ids=lambda p: "_".join("x".join(map(str, c[:5])) for c in p))
def test_noalloc_matches_workspace_entry_point(pair):
    import torch
    import paper_2606_07713_amd as moa
    for i, (B, H, Nq, Nk, d, dtype, causal, splits) in enumerate(pair):
        say(f"noalloc call {i}: B{B} H{H} Nq{Nq} Nk{Nk} d{d} {dtype} causal={causal} "
            f"splits={splits}")
        q, k, v = gen(B, H, Nq, Nk, d, dtype, seed=31 * i + B + H + Nq)
        tq, tk, tv = (synth.to_torch(a, "cuda") for a in (q, k, v))
        need = moa.moa_attn_workspace_bytes(B, H, Nq, Nk, d, d, splits)
        assert 0 < need <= moa.MOA_NOALLOC_SCRATCH_BYTES
        for odt in dict.fromkeys(({"bf16": torch.bfloat16, "f32": torch.float32}[dtype],
                                  torch.float32)):
            o_ref, lse_ref = moa.attn_fwd(tq, tk, tv, causal=causal, out_dtype=odt,
                                          num_splits=splits, return_lse=True)
            o, lse = _noalloc(tq, tk, tv, causal, odt, splits)
            torch.cuda.synchronize()
            assert torch.equal(o, o_ref), "O differs"
            assert torch.equal(lse, lse_ref), "LSE differs"
            err = max_err(o.float().cpu().double().numpy(), oracle_full(q, k, v, causal=causal))
            say(f"  out {odt}: bit-identical to moa_attn_fwd; max err vs oracle {err:.3e}")
            assert err <= TOL[dtype]


def test_noalloc_without_splits():
    # A prefill call that does not split its keys uses no scratch.
    import torch
    import paper_2606_07713_amd as moa
    q, k, v = gen(2, 2, 200, 300, 128, "bf16", seed=5)
    tq, tk, tv = (synth.to_torch(a, "cuda") for a in (q, k, v))
    o, _ = _noalloc(tq, tk, tv, True, torch.float32, 0)
    o_ref = moa.attn_fwd(tq, tk, tv, causal=True, out_dtype=torch.float32)
    torch.cuda.synchronize()
    assert torch.equal(o, o_ref)
