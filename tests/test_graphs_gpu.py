"""Forward calls captured in a HIP graph and replayed.

The library only launches kernels -- it allocates nothing, records no memset or
copy and never synchronises -- so a call on a capturing stream records its
launches and a replay repeats them.  Each case runs the C entry point eagerly
once, captures the same call (same buffers) with torch's graph capture, and
replays it several times; between replays the program does eager work of its
own (the same entry point on other inputs, into the same workspace or scratch
array) and synchronises.  Every replay must reproduce the eager O and LSE bit
for bit.
"""
import numpy as np
import pytest

import synth
from gpu_util import gen, say

pytestmark = pytest.mark.gpu

CASES = [
    # B, H, Nq, Nk, d, dtype, causal, entry point
    (2, 16, 1024, 1024, 128, "bf16", True, "fwd"),      # ping-pong layout
    (1, 4, 300, 700, 64, "bf16", False, "fwd"),         # key-split layout
    (1, 8, 128, 8192, 128, "bf16", False, "fwd"),       # split-K + combine, caller's workspace
    (64, 8, 1, 2048, 64, "bf16", False, "fwd"),         # decode, one split, no workspace
    (8, 4, 1, 4096, 128, "bf16", False, "fwd"),         # decode, split + combine
    (2, 3, 100, 100, 64, "f32", True, "fwd"),           # fp32 prefill
    (1, 8, 128, 8192, 128, "bf16", False, "noalloc"),   # split-K through the fixed scratch array
    (8, 4, 1, 4096, 128, "bf16", False, "noalloc"),     # decode split through the scratch array
]


def _buffers(B, H, Nq, Nk, d, dtype, seed):
    import torch
    q, k, v = gen(B, H, Nq, Nk, d, dtype, seed=seed)
    tq, tk, tv = (synth.to_torch(a, "cuda") for a in (q, k, v))
    odt = torch.float32 if dtype == "f32" else torch.bfloat16
    out = torch.full((B, H, Nq, d), float("nan"), dtype=odt, device="cuda")
    lse = torch.full((B, H, Nq), float("nan"), dtype=torch.float32, device="cuda")
    return tq, tk, tv, out, lse


def _caller(moa, bufs, B, H, Nq, Nk, d, dtype, causal, entry, ws):
    """The C call on whatever stream is current when it runs (the capture stream inside
    torch.cuda.graph)."""
    import torch
    tq, tk, tv, out, lse = bufs
    code = moa.MOA_F32 if dtype == "f32" else moa.MOA_BF16
    scale = 1.0 / np.sqrt(d)

    def call():
        stream = torch.cuda.current_stream().cuda_stream
        if entry == "noalloc":
            return moa.moa_attn_fwd_noalloc(tq.data_ptr(), tk.data_ptr(), tv.data_ptr(),
                                            out.data_ptr(), lse.data_ptr(), B, H, Nq, Nk, d, d,
                                            scale, int(causal), code, code, 0, stream)
        return moa.moa_attn_fwd(tq.data_ptr(), tk.data_ptr(), tv.data_ptr(), out.data_ptr(),
                                lse.data_ptr(), B, H, Nq, Nk, d, d, scale, int(causal), code, code,
                                ws.data_ptr() if ws is not None else None,
                                ws.numel() if ws is not None else 0, 0, stream)
    return call


@pytest.mark.parametrize("case", CASES, ids=lambda c: "x".join(map(str, c[:5])) + f"_{c[5]}_{c[7]}")
def test_captured_call_replays_bit_identical(case):
    import torch
    import paper_2606_07713_amd as moa
    B, H, Nq, Nk, d, dtype, causal, entry = case
    say(f"graph capture {case}")
    need = moa.moa_attn_workspace_bytes(B, H, Nq, Nk, d, d, 0)
    if dtype == "f32" and Nq > 1:
        need = 0
    ws = torch.empty(need, dtype=torch.uint8, device="cuda") if (need and entry == "fwd") else None
    main = _buffers(B, H, Nq, Nk, d, dtype, seed=7)
    other = _buffers(B, H, Nq, Nk, d, dtype, seed=8)
    call = _caller(moa, main, B, H, Nq, Nk, d, dtype, causal, entry, ws)
    call_other = _caller(moa, other, B, H, Nq, Nk, d, dtype, causal, entry, ws)

    assert call() == moa.MOA_OK
    torch.cuda.synchronize()
    ref_o, ref_lse = main[3].clone(), main[4].clone()
    assert not torch.isnan(ref_o.float()).any()

    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        status = call()
    assert status == moa.MOA_OK
    torch.cuda.synchronize()

    for rep in range(4):
        main[3].fill_(float("nan"))
        main[4].fill_(float("nan"))
        # the program's own work in between: the same entry point on other inputs,
        # through the same workspace or scratch array
        assert call_other() == moa.MOA_OK
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(main[3], ref_o), f"replay {rep}: O differs from the eager call"
        assert torch.equal(main[4], ref_lse), f"replay {rep}: LSE differs from the eager call"
    say(f"  {entry}: 4 replays bit-identical to the eager call")
