"""Benchmark of the fused attention hot path on one MI355X.

One step = one call of the library on one batch of seeded synthetic input,
already resident in device memory.  The default run times

  * prefill (the main line): causal attention B=1, H=32, Nq=Nk=16384,
    dk=dv=128, bf16 Q/K ~ N(0, 3^2), V ~ N(0, 1) -- one launch of the fused
    MFMA tile kernel per step;
  * decode (reported in the same line under "decode"): B=64, H=32, Nq=1,
    Nk=8192, dk=dv=128, bf16 -- split-K kernel + combine kernel per step;

each with HIP events on the stream the kernels run on, and reports achieved
TFLOP/s (prefill, matrix-core bound) and GB/s (decode, HBM bound) against the
MI355X peaks.  The fp64 CPU oracle is timed on a bounded sample of the
prefill workload on the host's cores as a reported baseline.

The backward pass of the prefill workload (dQ, dK, dV from the forward's O and
LSE for a seeded dO) is timed in the same run and reported under "backward",
and every one of the library's five workloads is timed and reported under
"configs" (time, TFLOP/s and GB/s against the roofline that bounds it).

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
                       [--no-cpu-baseline] [--no-decode] [--no-backward] [--no-configs]
                       [--calibrate-copy MIB]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "fused attention TFLOP/s + HBM GB/s vs MI355X roofline, bf16 d=128"
PEAK_BF16_TFLOPS = 2500.0      # dense bf16 matrix-core peak, TFLOP/s
PEAK_HBM_GBS = 8000.0          # HBM3E peak, GB/s
DEFAULT_PREFILL = "causal_long_b1h32_n16384_d128_bf16_qk_sigma3"
DEFAULT_DECODE = "decode_b64h32_nk8192_d128_bf16"


def visible_pairs(w) -> int:
    """(query, key) pairs left visible by the mask: key j <= i + (Nk - Nq) when causal."""
    if not w.causal:
        return w.B * w.H * w.Nq * w.Nk
    off = w.Nk - w.Nq
    per_head = sum(min(w.Nk, i + off + 1) for i in range(w.Nq))
    return w.B * w.H * per_head


def algorithmic_flops(w) -> float:
    """Matrix-product flops over visible pairs: 2*dk for Q.K^T plus 2*dv for P.V."""
    return 2.0 * (w.dk + w.dv) * visible_pairs(w)


def backward_flops(w) -> float:
    """Matrix-product flops of the gradients over visible pairs: the recomputed scores
    (2*dk), dP = dO V^T (2*dv), dV (2*dv), dQ and dK (2*dk each) -- 2.5x the forward's."""
    return 2.0 * (3 * w.dk + 2 * w.dv) * visible_pairs(w)


def compulsory_bytes(w, out_bytes: int) -> int:
    """Q, K and V read once, O written once."""
    es = 4 if w.dtype == "f32" else 2
    return w.B * w.H * ((w.Nq * w.dk + w.Nk * (w.dk + w.dv)) * es + w.Nq * w.dv * out_bytes)


KERNEL_SOURCES = {
    "prefill_bf16": ("prefill_bf16.hip", "prefill_bf16_common.h", "device_common.h", "launch.h"),
    "decode_split": ("decode.hip", "device_common.h", "launch.h"),
}


def kernel_source_hash(kernel: str) -> str:
    """First 16 hex digits of the sha256 of the kernel's source files."""
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[kernel]:
        with open(os.path.join(ROOT, "paper_2606_07713_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(kernel: str, workload: str):
    """HBM bytes per launch from the committed counter passes (profiles/traffic.txt),
    or None when they were taken on a different kernel source or workload."""
    path = os.path.join(ROOT, "profiles", "traffic.txt")
    if not os.path.exists(path):
        return None
    want = kernel_source_hash(kernel)
    with open(path) as fh:
        for line in fh:
            parts = line.split()
            if len(parts) == 4 and not line.startswith("#") and parts[0] == kernel \
                    and parts[1] == workload and parts[2] == want:
                return int(parts[3])
    return None


def config_record(w, ms: float, out_bytes: int, layout: str = "bhnd") -> dict:
    """Time and roofline figures of one workload: algorithmic flops and compulsory bytes per
    call over the measured time, against the bf16 matrix-core and HBM peaks.  The fp32 path
    (vector ALU, far below either roofline at its 4 MFLOP size) reports absolute time only."""
    flops = algorithmic_flops(w)
    nbytes = compulsory_bytes(w, out_bytes)
    tflops = flops / (ms * 1e-3) / 1e12
    gbs = nbytes / (ms * 1e-3) / 1e9
    rec = {"workload": w.name, "ms_per_call": round(ms, 5), "tflops": round(tflops, 2),
           "GBps": round(gbs, 1), "flop_per_call": flops, "compulsory_bytes": nbytes,
           "out": "bf16" if out_bytes == 2 else "f32"}
    if w.dtype != "bf16":
        rec.update(bound="latency", frac=None, traffic=None)
    elif flops / nbytes > PEAK_BF16_TFLOPS * 1e12 / (PEAK_HBM_GBS * 1e9):
        rec.update(bound="mfma", frac=round(tflops / PEAK_BF16_TFLOPS, 4),
                   traffic=measured_traffic("prefill_bf16", w.name) if layout == "bhnd" else None)
    else:
        rec.update(bound="hbm", frac=round(gbs / PEAK_HBM_GBS, 4),
                   traffic=measured_traffic("decode_split", w.name) if layout == "bhnd" else None)
    return rec


def _inputs(w, dev):
    import synth
    q, k, v = synth.make_inputs(w)
    return (q, k, v), tuple(synth.to_torch(a, dev) for a in (q, k, v))


def library_call(moa, tq, tk, tv, out, w, ws, stream):
    """One step: a call of the C entry point with its arguments marshalled once beforehand,
    so that the timed loop measures the library, not the Python wrapper (whose argument
    checks cost tens of microseconds of host time per call, more than the smaller
    workloads take on the GPU).  Contiguous tensors go to moa_attn_fwd, strided views to
    moa_attn_fwd_strided, exactly as attn_fwd would pass them."""
    import ctypes
    code = {"torch.float32": moa.MOA_F32, "torch.bfloat16": moa.MOA_BF16}
    in_code, out_code = code[str(tq.dtype)], code[str(out.dtype)]
    ptrs = (tq.data_ptr(), tk.data_ptr(), tv.data_ptr(), out.data_ptr(), None)
    dims = (w.B, w.H, w.Nq, w.Nk, w.dk, w.dv)
    tail = (ctypes.c_float(w.scale), int(w.causal), in_code, out_code,
            ws.data_ptr() if ws is not None else None,
            ws.numel() if ws is not None else 0, 0, stream.cuda_stream)
    if all(t.is_contiguous() for t in (tq, tk, tv, out)):
        fn, args = moa.lib.moa_attn_fwd, ptrs + dims + tail
    else:
        arrs = [(ctypes.c_int64 * 3)(*t.stride()[:3]) for t in (tq, tk, tv, out)]
        fn, args = moa.lib.moa_attn_fwd_strided, ptrs + dims + tuple(
            ctypes.cast(a, ctypes.c_void_p) for a in arrs) + tail
    keep = (tq, tk, tv, out, ws)

    def call():
        st = fn(*args)
        if st != moa.MOA_OK:
            raise moa.MoaAttnError(st)
        return keep
    return call


def time_calls(fn, steps: int, warmup: int, stream):
    """Average ms per call over `steps` calls, HIP events on `stream`."""
    import torch
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    start.record(stream)
    for _ in range(steps):
        fn()
    end.record(stream)
    torch.cuda.synchronize()
    return start.elapsed_time(end) / steps


def cpu_baseline(w, host_inputs, target_s: float = 12.0):
    """Oracle on a bounded random sample of the workload's query rows."""
    import numpy as np
    import oracle
    q, k, v = host_inputs
    threads = len(os.sched_getaffinity(0))
    rng = np.random.default_rng(0)
    total = w.B * w.H * w.Nq

    def flops_of(rows):
        if not w.causal:
            return 2.0 * (w.dk + w.dv) * w.Nk * rows.size
        i = rows % w.Nq
        return 2.0 * (w.dk + w.dv) * float(np.minimum(w.Nk, i + (w.Nk - w.Nq) + 1).sum())

    probe = rng.integers(0, total, size=min(total, 64 * threads)).astype(np.int64)
    t0 = time.perf_counter()
    oracle.attention_rows(q, k, v, probe, scale=w.scale, causal=w.causal, nthreads=threads)
    dt = time.perf_counter() - t0
    n = int(min(total, max(probe.size, probe.size * target_s / max(dt, 1e-3))))
    rows = rng.integers(0, total, size=n).astype(np.int64)
    t0 = time.perf_counter()
    oracle.attention_rows(q, k, v, rows, scale=w.scale, causal=w.causal, nthreads=threads)
    dt = time.perf_counter() - t0
    return {
        "value": flops_of(rows) / dt / 1e12,
        "unit": "TFLOP/s",
        "cores": threads,
        "kind": "oracle",
        "sample": f"{rows.size} random query rows of {w.name} (of {total}), fp64, "
                  f"{dt:.1f} s on {threads} OpenMP threads",
    }


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=DEFAULT_PREFILL)
    ap.add_argument("--decode-workload", default=DEFAULT_DECODE)
    ap.add_argument("--no-decode", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-backward", action="store_true",
                    help="skip the timing of the backward pass (reported under \"backward\")")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the per-workload records (reported under \"configs\")")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="before timing, run one plain copy kernel of MIB MiB (read MIB, "
                         "write MIB) so profiler byte counters can be scaled against it")
    ap.add_argument("--out-dtype", choices=["bf16", "f32"], default=None,
                    help="output storage (default: the input storage type)")
    ap.add_argument("--layout", choices=["bhnd", "bnhd"], default="bhnd",
                    help="storage of Q, K, V and O: [B][H][N][d] (default) or [B][N][H][d], "
                         "the latter passed as strided views (no copies in the timed region)")
    args = ap.parse_args(argv)

    if args.gpus != 1:
        print(f"bench.py: this library runs on one GPU; --gpus {args.gpus} is not supported "
              "(every (batch, head) slice is independent: larger jobs shard over GPUs "
              "by slice with no communication, which one GPU's figure already measures).",
              file=sys.stderr)
        return 2

    import torch
    import synth
    import paper_2606_07713_amd as moa

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream(dev)

    if args.calibrate_copy:
        n = args.calibrate_copy * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        torch.neg(src, out=dst)          # elementwise: reads n*4 bytes, writes n*4 bytes
        torch.cuda.synchronize()
        del src, dst

    def run_workload(name, steps=None):
        w = synth.WORKLOADS[name]
        host, (tq, tk, tv) = _inputs(w, dev)
        odt = {"bf16": torch.bfloat16, "f32": torch.float32}[args.out_dtype or w.dtype]
        if args.layout == "bnhd":
            tq, tk, tv = (t.transpose(1, 2).contiguous().transpose(1, 2) for t in (tq, tk, tv))
            out = torch.empty((w.B, w.Nq, w.H, w.dv), dtype=odt, device=dev).transpose(1, 2)
        else:
            out = torch.empty((w.B, w.H, w.Nq, w.dv), dtype=odt, device=dev)
        ws_bytes = moa.moa_attn_workspace_bytes(w.B, w.H, w.Nq, w.Nk, w.dk, w.dv, 0)
        ws = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device=dev)
        call = library_call(moa, tq, tk, tv, out, w, ws if ws_bytes else None, stream)
        call()
        torch.cuda.synchronize()
        ms = time_calls(call, steps or args.steps, args.warmup, stream)
        return w, host, ms, out.element_size()

    w, host, ms, ob = run_workload(args.workload)
    flops = algorithmic_flops(w)
    tflops = flops / (ms * 1e-3) / 1e12
    nbytes = compulsory_bytes(w, ob)
    mfma_bound = flops / nbytes > PEAK_BF16_TFLOPS * 1e12 / (PEAK_HBM_GBS * 1e9)
    if mfma_bound:
        roof = {"bound": "mfma", "achieved": round(tflops, 2), "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s", "frac": round(tflops / PEAK_BF16_TFLOPS, 4),
                "traffic": measured_traffic("prefill_bf16", w.name)
                if w.dtype == "bf16" and args.layout == "bhnd" else None}
    else:
        gbs = nbytes / (ms * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(gbs / PEAK_HBM_GBS, 4), "traffic": None}
    line = {
        "metric": METRIC,
        "value": round(tflops, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if w.dtype == "bf16" else "f32",
        "data": "synthetic",
        "config": {"workload": w.name, "B": w.B, "H": w.H, "Nq": w.Nq, "Nk": w.Nk, "dk": w.dk,
                   "dv": w.dv, "causal": w.causal, "in": w.dtype, "layout": args.layout,
                   "out": args.out_dtype or w.dtype, "flop_per_step": flops,
                   "compulsory_bytes_per_step": nbytes,
                   "hbm_GBps_compulsory": round(nbytes / (ms * 1e-3) / 1e9, 1)},
        "roofline": roof,
    }
    print(f"# prefill {w.name}: {ms:.4f} ms/step, {tflops:.1f} TFLOP/s", file=sys.stderr, flush=True)

    if not args.no_decode:
        wd, _, msd, obd = run_workload(args.decode_workload)
        bd = compulsory_bytes(wd, obd)
        gbs = bd / (msd * 1e-3) / 1e9
        line["decode"] = {
            "workload": wd.name, "ms_per_call": round(msd, 4),
            "splits": moa.moa_attn_num_splits(wd.B, wd.H, wd.Nq, wd.Nk, wd.dk, wd.dv, 0),
            "value": round(gbs, 1), "unit": "GB/s",
            "tflops": round(algorithmic_flops(wd) / (msd * 1e-3) / 1e12, 2),
            "roofline": {"bound": "hbm", "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS,
                         "unit": "GB/s", "frac": round(gbs / PEAK_HBM_GBS, 4),
                         "traffic": measured_traffic("decode_split", wd.name)
                         if args.layout == "bhnd" else None},
        }
        print(f"# decode {wd.name}: {msd:.4f} ms/call, {gbs:.1f} GB/s", file=sys.stderr, flush=True)

    if not args.no_backward and w.dtype == "bf16" and args.layout == "bhnd":
        # Gradients of the same workload for a seeded dO, from the forward's O and LSE.
        tq, tk, tv = (synth.to_torch(a, dev) for a in host)
        o, lse = moa.attn_fwd(tq, tk, tv, scale=w.scale, causal=w.causal, return_lse=True)
        do = synth.to_torch(synth.normal(7919, (w.B, w.H, w.Nq, w.dv), 1.0, "bf16"), dev)
        ws_b = moa.moa_attn_bwd_workspace_bytes(w.B, w.H, w.Nq, w.Nk, w.dk, w.dv)
        ws_bwd = torch.empty(max(ws_b, 1), dtype=torch.uint8, device=dev)

        def call_bwd():
            moa.attn_bwd(tq, tk, tv, o, lse, do, scale=w.scale, causal=w.causal,
                         grad_dtype=torch.bfloat16, workspace=ws_bwd if ws_b else None,
                         stream=stream)
        steps_b = max(1, args.steps // 5)
        msb = time_calls(call_bwd, steps_b, min(args.warmup, 2), stream)
        fb = backward_flops(w)
        line["backward"] = {"workload": w.name, "ms_per_call": round(msb, 4), "steps": steps_b,
                            "value": round(fb / (msb * 1e-3) / 1e12, 2), "unit": "TFLOP/s",
                            "flop_per_call": fb, "grad_dtype": "bf16",
                            "frac": round(fb / (msb * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4)}
        print(f"# backward {w.name}: {msb:.4f} ms/call, {fb / (msb * 1e-3) / 1e12:.1f} TFLOP/s",
              file=sys.stderr, flush=True)
        del o, lse, do, ws_bwd

    if not args.no_configs:
        # Every workload of the library, each timed like the main line (one library call per
        # step, HIP events on the launch stream); the main and decode workloads reuse the
        # timings above.
        timed = {w.name: (ms, ob)}
        if "decode" in line:
            timed[wd.name] = (msd, obd)
        recs = []
        for name, wc in synth.WORKLOADS.items():
            if name in timed:
                msc, obc = timed[name]
            else:
                _, _, msc, obc = run_workload(name, max(args.steps, 100))
            recs.append(config_record(wc, msc, obc, args.layout))
            print(f"# config {name}: {msc * 1e3:.2f} us/call", file=sys.stderr, flush=True)
        line["configs"] = recs

    line["cpu_baseline"] = None if args.no_cpu_baseline else cpu_baseline(w, host)
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
