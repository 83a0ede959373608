#!/usr/bin/env python3
"""Throughput of the W4A4 rotated linear layer on one MI355X.

Workload: the Llama-2-70B FFN pair at prefill, batch 8 x sequence 2048
(M = 16384 tokens): up-projection shape K = 8192 -> N = 28672 (online
Hadamard n = 8192) and down-projection shape K = 28672 -> N = 8192
(n = 1024 * 28).  Synthetic inputs (seeded normals with 0.5% outlier
channels x100, weights N(0, 0.02^2)), prepared weights resident in HBM.

One step = both layers, each as the two launches quarot_linear makes:
rotate+quantize the activations (quarot_quant_int4), then the W4A4 GEMM
with fused dequant (quarot_w4a4_gemm).  HIP events on the launch stream
bracket every kernel, so the per-kernel averages over the timed steps give
the roofline figures.  value = 2*M*N*K summed over both layers / step time.

Prints one JSON line.
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

# MI355X published peaks
PEAK_I8_TOPS = 5000.0   # dense int8 MFMA, TOP/s
PEAK_HBM_GBS = 8000.0   # HBM3E, GB/s


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


# HBM-side bytes per k_gemm_w4a4 launch on this workload, averaged over the
# up and down launches: FETCH_SIZE x 2 + WRITE_SIZE x 1 (KiB, scaled by what
# the counters read for a plain 1 GiB copy), from the two rocprofv3 --pmc runs
# summarized in profiles/.  Valid only for the kernel source they were taken
# with; after any change to it the figure is reported as null.
GEMM_TRAFFIC = {"source_sha256_16": "40414b49ac9c251e", "bytes_per_launch": 3.452e9}


def gemm_source_hash() -> str:
    import hashlib
    h = hashlib.sha256()
    for f in ("gemm_w4a4.hip", "common.hpp"):
        with open(os.path.join(ROOT, "paper_2404_00456_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def rotate_bytes(M, K):
    """Algorithmic HBM bytes of rotate+quantize: read fp16 x, write packed
    int4 codes and one fp16 scale per row."""
    return M * K * 2 + M * K // 2 + M * 2


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--cpu-rows", type=int, default=64,
                    help="rows per layer of the oracle's CPU-baseline sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-mib", type=int, default=0,
                    help="after timing, copy a buffer of this many MiB once (a plain copy "
                         "kernel of known size, to scale hardware byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(json.dumps({"error": "this build measures one GPU; multi-GPU runs are not "
                                   "part of it", "n_gpus": args.gpus}))
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2404_00456_amd as q
    import workloads

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    layers = []
    for name in ("llama2_70b_up", "llama2_70b_down"):
        wl = workloads.LINEAR[name]
        log(f"generating {name}: M={wl.M} K={wl.K} N={wl.N}")
        x, w, _ = workloads.linear_inputs(wl)
        xd = torch.from_numpy(x).to(dev)
        wd = torch.from_numpy(w).to(dev)
        wq, sw = q.prepare_weight(wd, rotate=True)  # offline step, untimed
        del wd
        ws = torch.empty(q.quarot_linear_workspace_size(wl.M, wl.K), dtype=torch.uint8,
                         device=dev)
        xq = ws[: wl.M * wl.K // 2].view(wl.M, wl.K // 2)
        off = (wl.M * wl.K // 2 + 255) // 256 * 256
        sx = ws[off: off + 2 * wl.M].view(torch.float16)
        y = torch.empty((wl.M, wl.N), dtype=torch.float16, device=dev)
        layers.append(dict(wl=wl, x=x, w=w, xd=xd, wq=wq, sw=sw, xq=xq, sx=sx, y=y))
    torch.cuda.synchronize()

    stream = torch.cuda.current_stream()

    def step(ev=None):
        for li, L in enumerate(layers):
            if ev is not None:
                ev[2 * li].record(stream)
            q.quarot_quant_int4(L["xd"], rotate=True, clip_ratio=1.0, q=L["xq"], scale=L["sx"])
            if ev is not None:
                ev[2 * li + 1].record(stream)
            q.quarot_w4a4_gemm(L["xq"], L["sx"], L["wq"], L["sw"], y=L["y"])
        if ev is not None:
            ev[4].record(stream)

    log(f"warmup {args.warmup}")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    events = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(args.steps)]
    log(f"timing {args.steps} steps")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(args.steps):
        step(events[s])
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_step = (t1 - t0) * 1e3 / args.steps

    # per-kernel durations from the events (ms)
    rot = [[], []]
    gem = [[], []]
    for ev in events:
        for li in range(2):
            rot[li].append(ev[2 * li].elapsed_time(ev[2 * li + 1]))
            end = ev[2 * li + 2] if li == 0 else ev[4]
            gem[li].append(ev[2 * li + 1].elapsed_time(end))
    ops = [2 * L["wl"].M * L["wl"].N * L["wl"].K for L in layers]
    total_ops = sum(ops)
    value = total_ops / (ms_step * 1e-3) / 1e12
    gemm_ms = [float(np.mean(g)) for g in gem]
    rot_ms = [float(np.mean(r)) for r in rot]
    gemm_tops = sum(ops) / (sum(gemm_ms) * 1e-3) / 1e12
    rbytes = [rotate_bytes(L["wl"].M, L["wl"].K) for L in layers]
    kernels = {}
    for li, L in enumerate(layers):
        nm = L["wl"].name
        kernels[nm] = {
            "rotate_quant_us": round(rot_ms[li] * 1e3, 2),
            "rotate_quant_GBps": round(rbytes[li] / (rot_ms[li] * 1e-3) / 1e9, 1),
            "gemm_us": round(gemm_ms[li] * 1e3, 2),
            "gemm_TOPS": round(ops[li] / (gemm_ms[li] * 1e-3) / 1e12, 1),
            "linear_TOPS": round(ops[li] / ((gemm_ms[li] + rot_ms[li]) * 1e-3) / 1e12, 1),
        }

    if args.copy_mib:
        src = torch.empty(args.copy_mib << 20, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        src.fill_(1)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    cpu = None
    if not args.no_cpu_baseline:
        import oracle as orc
        R = args.cpu_rows
        log(f"cpu baseline: oracle weight prep (untimed), then {R} rows per layer")
        preps = [orc.prepare_weight(L["w"], rotate=True) for L in layers]
        t = time.perf_counter()
        for L, (rwq, rsw) in zip(layers, preps):
            orc.linear(L["x"][:R], rwq, rsw, rotate=True, clip=1.0)
        dt = time.perf_counter() - t
        sample_ops = sum(2 * R * L["wl"].N * L["wl"].K for L in layers)
        cpu = {"value": sample_ops / dt / 1e12, "unit": "TOP/s", "cores": orc.max_threads(),
               "kind": "oracle",
               "sample": f"first {R} of {layers[0]['wl'].M} token rows of each layer "
                         f"(rotate+quantize+GEMM+dequant), {dt:.1f} s"}

    traffic = (GEMM_TRAFFIC["bytes_per_launch"]
               if gemm_source_hash() == GEMM_TRAFFIC["source_sha256_16"] else None)
    out = {
        "metric": "W4A4 rotated-linear TOPS + % int8-MFMA peak; Hadamard/quant GB/s "
                  "(Llama2 shapes)",
        "value": round(value, 2),
        "unit": "TOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int4",
        "data": "synthetic",
        "config": {"workload": "llama2_70b_ffn_prefill: M=16384 tokens (batch 8 x seq 2048); "
                               "up K=8192->N=28672 (H_8192), down K=28672->N=8192 "
                               "(H_1024 x H_28)",
                   "global_batch": 8, "seq_len": 2048, "parallelism": "none"},
        "pct_int8_peak": round(100 * value / PEAK_I8_TOPS, 2),
        "roofline": {"bound": "mfma", "kernel": "k_gemm_w4a4",
                     "achieved": round(gemm_tops, 1), "peak": PEAK_I8_TOPS, "unit": "TOP/s",
                     "frac": round(gemm_tops / PEAK_I8_TOPS, 4), "traffic": traffic},
        "kernels": kernels,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
