#!/usr/bin/env python3
"""Throughput of the W4A4 rotated linear layer on one MI355X.

Workload: the Llama-2-70B FFN pair at prefill, batch 8 x sequence 2048
(M = 16384 tokens): up-projection shape K = 8192 -> N = 28672 (online
Hadamard n = 8192) and down-projection shape K = 28672 -> N = 8192
(n = 1024 * 28).  Synthetic inputs (seeded normals with 0.5% outlier
channels x100, weights N(0, 0.02^2)), prepared weights resident in HBM.

One step = both layers, each as the two launches quarot_linear_e3m2 makes:
rotate+quantize the activations straight into the e3m2 operand layout
(quarot_quant_int4_e3m2), then the W4A4 GEMM on gfx950's fp6 matrix
instruction with fused dequant (quarot_w4a4_gemm_e3m2; weights prepared
and repacked once, untimed).  Its outputs equal the int4-operand path's
(quarot_quant_int4 + quarot_w4a4_gemm) bit for bit; that path is timed
beside it under kernels/<layer>/int4_operands.  HIP events on the launch
stream bracket every kernel, so the per-kernel averages over the timed
steps give the roofline figures.  value = 2*M*N*K summed over both layers
/ step time.

The same run then times the 4-bit KV cache path on its own workload (K and V
fp16 [batch 16, 64 heads, 4096 tokens, head_dim 128], 1 GiB each):
rotate + asymmetric int4 quantization per head row (quarot_kv_quant) and the
dequantization back to fp16 (quarot_kv_dequant), reported as HBM GB/s
against 8 TB/s under "kv" (HBM-bound kernels; each tensor is 4x the 256 MB
last-level cache, so the traffic is HBM traffic).

Prints one JSON line.
"""
from __future__ import annotations

import argparse
import gc
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

# MI355X published peaks
PEAK_I8_TOPS = 5000.0   # dense int8 MFMA, TOP/s
PEAK_FP6_TOPS = 10100.0  # dense fp6 / fp4 MFMA, TFLOP/s (ops on exact integers here)
PEAK_F32_ADDS = 78.6e12  # fp32 vector adds per second (157.3 TFLOP/s counts an FMA as 2)
PEAK_HBM_GBS = 8000.0   # HBM3E, GB/s


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


# HBM-side bytes per launch of each per-token GEMM on this workload,
# averaged over the up and down launches: FETCH_SIZE x 2 + WRITE_SIZE x 1
# (KiB, scaled by what the counters read for a plain 1 GiB copy), from the
# two rocprofv3 --pmc runs summarized in profiles/.  Valid only for the
# kernel machine code they were taken with (its fingerprint); after any
# change to it the figure is reported as null.
GEMM_TRAFFIC = {
    "k_gemm_w4a4": {"isa_sha256_16": "a959ef97d8288dd6", "bytes_per_launch": 3.470e+09},
    "k_gemm_w4a4_e3m2": {"isa_sha256_16": "869819c9cf015403", "bytes_per_launch": 4.838e+09},
}


def gemm_isa_hash(kernel: str) -> str:
    """A per-token GEMM kernel's machine-code fingerprint written by the
    build (empty if absent)."""
    try:
        with open(os.path.join(ROOT, "paper_2404_00456_amd", "gemm_isa.sha")) as f:
            for line in f:
                parts = line.split()
                if len(parts) == 2 and parts[0] == kernel:
                    return parts[1]
    except OSError:
        pass
    return ""


def gemm_traffic(kernel: str):
    t = GEMM_TRAFFIC[kernel]
    return t["bytes_per_launch"] if gemm_isa_hash(kernel) == t["isa_sha256_16"] else None


def rotate_bytes(M, K, code_bits=4):
    """Algorithmic HBM bytes of rotate+quantize: read fp16 x, write the codes
    (4 bits each packed, or 6 in the e3m2 layout) and one fp16 scale per row."""
    return M * K * 2 + M * K * code_bits // 8 + M * 2


def kv_bytes(rows, D, group):
    """Algorithmic HBM bytes of one KV tensor: fp16 values, packed uint4
    codes, fp16 scale and zero per group (read one side, write the other)."""
    return rows * D * 2 + rows * D // 2 + rows * (D // group) * 4


def bench_kv(q, workloads, torch, np, dev, stream, iters):
    wl = workloads.KV["kv4_70b"]
    log(f"generating {wl.name}: K, V [{wl.B}, {wl.H}, {wl.S}, {wl.D}]")
    k, v = workloads.kv_inputs(wl)
    rows = wl.rows
    tens = []
    for t in (k, v):
        xd = torch.from_numpy(t.reshape(rows, wl.D)).to(dev)
        codes = torch.empty((rows, wl.D // 2), dtype=torch.uint8, device=dev)
        sc = torch.empty((rows, wl.D // wl.group), dtype=torch.float16, device=dev)
        ze = torch.empty_like(sc)
        out = torch.empty_like(xd)
        tens.append((xd, codes, sc, ze, out))
    del k, v
    torch.cuda.synchronize()

    def once(ev=None):
        for ti, (xd, codes, sc, ze, out) in enumerate(tens):
            if ev is not None:
                ev[3 * ti].record(stream)
            q.quarot_kv_quant(xd, group=wl.group, rotate=True, clip_ratio=wl.clip, q=codes,
                              scale=sc, zero=ze)
            if ev is not None:
                ev[3 * ti + 1].record(stream)
            q.quarot_kv_dequant(codes, sc, ze, group=wl.group, inverse_rotate=False, out=out)
            if ev is not None:
                ev[3 * ti + 2].record(stream)

    once()
    torch.cuda.synchronize()
    # decode step over the whole quantized cache: one rotated query per
    # (batch, head), seq_len = 4096 tokens
    nq = wl.B * wl.H
    kcache = tuple(x.view(nq, wl.S, -1) for x in tens[0][1:4])
    vcache = tuple(x.view(nq, wl.S, -1) for x in tens[1][1:4])
    g = torch.Generator(device=dev)
    g.manual_seed(0)
    qd = torch.randn((nq, wl.D), generator=g, device=dev).to(torch.float16)
    qd = q.quarot_hadamard(qd)
    att_out = torch.empty_like(qd)
    ws_bytes = q.quarot_kv_attention_workspace_size(nq, wl.S, wl.D)
    att_ws = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device=dev)

    def attend():
        q.quarot_kv_decode_attention(qd, kcache, vcache, wl.S, group=wl.group, out=att_out,
                                     workspace=att_ws)

    attend()
    torch.cuda.synchronize()
    a0, a1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    quiet_host()
    a0.record(stream)
    for _ in range(10 * iters):
        attend()
    a1.record(stream)
    torch.cuda.synchronize()
    att_us = a0.elapsed_time(a1) / (10 * iters) * 1e3
    att_bytes = 2 * (rows * wl.D // 2 + rows * (wl.D // wl.group) * 4)  # K and V caches
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(6)] for _ in range(iters)]
    quiet_host()
    log(f"timing kv x{iters}")
    for it in range(iters):
        once(evs[it])
    torch.cuda.synchronize()
    qt = [ev[3 * ti].elapsed_time(ev[3 * ti + 1]) for ev in evs for ti in range(2)]
    dt = [ev[3 * ti + 1].elapsed_time(ev[3 * ti + 2]) for ev in evs for ti in range(2)]
    nbytes = kv_bytes(rows, wl.D, wl.group)
    q_us, d_us = float(np.mean(qt)) * 1e3, float(np.mean(dt)) * 1e3
    q_gbs, d_gbs = nbytes / (q_us * 1e-6) / 1e9, nbytes / (d_us * 1e-6) / 1e9
    res = {"workload": f"{wl.name}: K and V fp16 [{wl.B}, {wl.H}, {wl.S}, {wl.D}], "
                       f"H_{wl.D} per head row, asymmetric uint4, group {wl.group}, "
                       f"clip {wl.clip}",
           "bytes_per_tensor": nbytes,
           "quant_us": round(q_us, 1), "quant_GBps": round(q_gbs, 1),
           "quant_frac_hbm": round(q_gbs / PEAK_HBM_GBS, 4),
           "dequant_us": round(d_us, 1), "dequant_GBps": round(d_gbs, 1),
           "dequant_frac_hbm": round(d_gbs / PEAK_HBM_GBS, 4),
           "decode_attention": {
               "what": f"one rotated fp16 query per (batch, head) over {wl.S} cached tokens",
               "us": round(att_us, 1), "cache_bytes": att_bytes,
               "GBps": round(att_bytes / (att_us * 1e-6) / 1e9, 1),
               "frac_hbm": round(att_bytes / (att_us * 1e-6) / 1e9 / PEAK_HBM_GBS, 4)}}
    # what a plain device-to-device copy of one K tensor (1 GiB read, 1 GiB
    # written; the runtime's copy kernel through torch) reaches on this
    # chip: the practical rate of a read-and-write stream, beside the
    # published peak the fractions above use
    src, dst = tens[0][0], tens[0][4]
    dst.copy_(src)
    c_us = float(np.median(event_times_us(torch, stream, [lambda: dst.copy_(src)], iters)[0]))
    c_bytes = 2 * src.numel() * src.element_size()
    res["device_copy_reference"] = {
        "what": "1 GiB device-to-device copy (torch copy_, read + write)",
        "us": round(c_us, 1), "GBps": round(c_bytes / (c_us * 1e-6) / 1e9, 1),
        "frac_hbm": round(c_bytes / (c_us * 1e-6) / 1e9 / PEAK_HBM_GBS, 4)}
    for t in tens:
        del t
    tens.clear()
    torch.cuda.empty_cache()
    return res


def event_times_us(torch, stream, fns, iters):
    """Per-launch durations (us) of each function in fns, run in turn
    iters times, from HIP events on the launch stream."""
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(len(fns) + 1)]
          for _ in range(iters)]
    quiet_host()
    for it in range(iters):
        for j, fn in enumerate(fns):
            ev[it][j].record(stream)
            fn()
        ev[it][len(fns)].record(stream)
    torch.cuda.synchronize()
    return [[ev[it][j].elapsed_time(ev[it][j + 1]) * 1e3 for it in range(iters)]
            for j in range(len(fns))]


def rotation_bounds(q, M, K, code_bits):
    """(HBM-bound us, VALU-bound us) of rotate+quantize: algorithmic bytes at
    8 TB/s, and log2(2^k) butterfly adds plus m - 1 m-factor adds per
    element at the fp32 vector add rate."""
    k2, m = q.quarot_hadamard_factor(K)
    return (rotate_bytes(M, K, code_bits) / (PEAK_HBM_GBS * 1e9) * 1e6,
            M * K * (k2 + m - 1) / PEAK_F32_ADDS * 1e6)


def bench_layers_7b(q, workloads, torch, np, dev, stream, iters, keep=None):
    """The Llama-2-7B layer shapes at sequence 2048 (M = 2048): up
    4096 -> 11008 (H_4096) and down 11008 -> 4096 (H_64 x H_172), each as
    the two launches of the e3m2 layer, per-kernel event times; and the
    tiny layer (16 x 128 -> 256) as launch latency of the whole call."""
    res = {}
    for name in ("llama2_7b_up", "llama2_7b_down"):
        wl = workloads.LINEAR[name]
        log(f"generating {name}: M={wl.M} K={wl.K} N={wl.N}")
        x, w, _ = workloads.linear_inputs(wl)
        xd = torch.from_numpy(x).to(dev)
        wd = torch.from_numpy(w).to(dev)
        w6, sw = q.prepare_weight_e3m2(wd, rotate=True)
        del wd
        if keep is not None:
            keep[name] = (x[:256].copy(), w)
        x6 = torch.empty((wl.K // 128, wl.M * 96), dtype=torch.uint8, device=dev)
        sx6 = torch.empty((wl.M,), dtype=torch.float16, device=dev)
        y = torch.empty((wl.M, wl.N), dtype=torch.float16, device=dev)
        rot = lambda: q.quarot_quant_int4_e3m2(xd, rotate=True, q6=x6, scale=sx6)
        gem = lambda: q.quarot_w4a4_gemm_e3m2(x6, sx6, w6, sw, y=y)
        for _ in range(3):
            rot(), gem()
        rt, gt = event_times_us(torch, stream, [rot, gem], iters)
        # cold rotation: rotate across copies of X totalling > 512 MB (twice
        # the last-level cache), so every launch reads its input from HBM
        ncp = max(2, -(-(640 << 20) // (xd.numel() * 2)))
        xs = [xd.clone() for _ in range(ncp)]
        cold = [lambda xc=xc: q.quarot_quant_int4_e3m2(xc, rotate=True, q6=x6, scale=sx6)
                for xc in xs]
        ct = event_times_us(torch, stream, cold, 2)
        del xs
        r_us, g_us = float(np.mean(rt)), float(np.mean(gt))
        c_us = float(np.mean([v for c in ct for v in c]))
        hbm_us, valu_us = rotation_bounds(q, wl.M, wl.K, 6)
        ops = 2 * wl.M * wl.N * wl.K
        k2, m = q.quarot_hadamard_factor(wl.K)
        res[name] = {
            "workload": f"M={wl.M} K={wl.K} -> N={wl.N}, H_{2 ** k2}" + (f" x H_{m}" if m > 1 else ""),
            "rotate_quant_us": round(r_us, 2), "rotate_quant_cold_us": round(c_us, 2),
            "rotate_quant_GBps": round(rotate_bytes(wl.M, wl.K, 6) / (r_us * 1e-6) / 1e9, 1),
            "rotate_quant_frac_hbm": round(hbm_us / r_us, 4),
            "rotate_quant_frac_valu_bound": round(valu_us / r_us, 4),
            "gemm_us": round(g_us, 2),
            "gemm_us_p10_p50_p90": [round(float(np.percentile(gt, p)), 1) for p in (10, 50, 90)],
            "gemm_TOPS": round(ops / (g_us * 1e-6) / 1e12, 1),
            "gemm_frac_fp6_peak": round(ops / (g_us * 1e-6) / 1e12 / PEAK_FP6_TOPS, 4),
            "linear_TOPS": round(ops / ((r_us + g_us) * 1e-6) / 1e12, 1),
            "linear_frac_int8_peak": round(ops / ((r_us + g_us) * 1e-6) / 1e12 / PEAK_I8_TOPS, 4),
        }
        del xd, w6, sw, x6, sx6, y
    # the tiny layer: launch latency of the two-launch call, back to back
    wl = workloads.LINEAR["tiny"]
    x, w, _ = workloads.linear_inputs(wl)
    xd = torch.from_numpy(x).to(dev)
    w6, sw = q.prepare_weight_e3m2(torch.from_numpy(w).to(dev), rotate=True)
    ws = torch.empty(q.quarot_linear_e3m2_workspace_size(wl.M, wl.K), dtype=torch.uint8,
                     device=dev)
    y = torch.empty((wl.M, wl.N), dtype=torch.float16, device=dev)
    call = lambda: q.quarot_linear_e3m2(xd, w6, sw, y=y, workspace=ws)
    us = time_us(torch, stream, call, iters=200)
    t0 = time.perf_counter()
    for _ in range(200):
        call()
    host_us = (time.perf_counter() - t0) / 200 * 1e6
    torch.cuda.synchronize()
    res["tiny"] = {"workload": f"M={wl.M} K={wl.K} -> N={wl.N}, H_128 (two launches)",
                   "us_per_call_gpu": round(us, 2), "us_per_call_host_enqueue": round(host_us, 2)}
    torch.cuda.empty_cache()
    return res


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_oracle_per_config(workloads, np, inputs):
    """The oracle on every workload, with all host threads and with one:
    rotate+quantize (elements/s) and the integer product + dequant (int
    ops/s) on a sample of token rows against all N weight rows (weights
    prepared untimed), the KV quantize + dequantize on a sample of head
    rows; each with the full workload's time extrapolated from the sample
    (labelled as such).  inputs: name -> (token rows x, prepared wq, sw),
    the workload's own draws (the tiny layer is drawn here)."""
    import oracle as orc
    allt = orc.max_threads()
    out = {"cpu_model": cpu_model(), "threads_all": allt, "configs": {}}
    sample = {"tiny": (16, 16), "llama2_7b_up": (64, 8), "llama2_7b_down": (64, 8),
              "llama2_70b_up": (64, 4), "llama2_70b_down": (64, 4)}
    for name, (r_all, r_one) in sample.items():
        wl = workloads.LINEAR[name]
        if name in inputs:
            x, wq, sw = inputs[name]
        elif name == "tiny":
            x, w, _ = workloads.linear_inputs(wl)
            wq, sw = orc.prepare_weight(w, rotate=True)
        else:
            continue
        entry = {}
        for th, R in ((allt, r_all), (1, r_one)):
            orc.set_threads(th)
            t = time.perf_counter()
            xq, sx = orc.quant_int4(x[:R], rotate=True, clip=1.0)
            tq = time.perf_counter() - t
            t = time.perf_counter()
            orc.dequant(orc.gemm_i32(xq, wq), sx, sw)
            tg = time.perf_counter() - t
            entry[f"threads_{th}"] = {
                "sample_rows": R,
                "rotate_quant_elems_per_s": round(R * wl.K / tq, 1),
                "gemm_dequant_ops_per_s": round(2 * R * wl.N * wl.K / tg, 1),
                "extrapolated_full_layer_s": round((tq + tg) * wl.M / R, 2)}
        out["configs"][name] = entry
    wl = workloads.KV["kv4_70b"]
    k, _ = workloads.kv_inputs(wl, B=1, S=256)
    kx = k.reshape(-1, wl.D)
    entry = {}
    for th, R in ((allt, kx.shape[0]), (1, 2048)):
        orc.set_threads(th)
        t = time.perf_counter()
        cq, cs, cz = orc.kv_quant(kx[:R], group=wl.group, rotate=True, clip=wl.clip)
        tq = time.perf_counter() - t
        t = time.perf_counter()
        orc.kv_dequant(cq, cs, cz, group=wl.group, inverse_rotate=False)
        td = time.perf_counter() - t
        entry[f"threads_{th}"] = {
            "sample_rows": R, "quant_elems_per_s": round(R * wl.D / tq, 1),
            "dequant_elems_per_s": round(R * wl.D / td, 1),
            "extrapolated_full_KV_s": round((tq + td) * 2 * wl.rows / R, 2)}
    out["configs"]["kv4_70b"] = entry
    orc.set_threads(allt)
    return out


def quiet_host():
    """Collect Python's cyclic garbage now, outside any timed region.  The
    collector is off for the whole run (main): a collection pass in the
    middle of a timed loop stalls the host for tens of milliseconds, the GPU
    runs dry, and the events count the idle time."""
    gc.collect()


def time_us(torch, stream, fn, iters=10):
    fn()
    torch.cuda.synchronize()
    quiet_host()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(iters):
        fn()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / iters * 1e3


def bench_next(q, torch, dev, stream, layers):
    """The built next rows on 70B shapes, timed in the same run:
    - the down-projection input as silu(gate) * up -> H_1024 x H_28 -> int4
      (fused, and unfused as quarot_swiglu then quarot_quant_int4);
    - the out_proj input (64 heads x 128) through the head-wise Hadamard
      -> int4;
    - the 8-bit GEMM (W8A8) on both FFN shapes, its codes from
      quarot_quant_int8 of the same activations and weights;
    - group-wise W4A4: the group quantizer (rotation to binary32, then
      per-group scales) and the grouped GEMM on the FFN shapes, on int4
      operands and (groups of 128 and 256) on e3m2 operands.
    gate/up/attention-output rows are seeded torch.randn draws on the GPU."""
    M = 16384
    g = torch.Generator(device=dev)
    g.manual_seed(1)
    res = {}
    n = 28672
    gate = torch.randn((M, n), generator=g, device=dev).to(torch.float16)
    up = torch.randn((M, n), generator=g, device=dev).to(torch.float16)
    codes = torch.empty((M, n // 2), dtype=torch.uint8, device=dev)
    sc = torch.empty(M, dtype=torch.float16, device=dev)
    h = torch.empty_like(gate)
    us = time_us(torch, stream, lambda: q.quarot_swiglu_quant_int4(gate, up, q=codes, scale=sc))
    us_un = time_us(torch, stream, lambda: (q.quarot_swiglu(gate, up, h=h),
                                            q.quarot_quant_int4(h, q=codes, scale=sc)))
    nb = M * n * 4 + M * n // 2 + 2 * M
    res["swiglu_quant_int4"] = {
        "workload": f"gate, up fp16 [{M}, {n}] -> RN16(silu(gate) up) -> H_1024 x H_28 -> int4",
        "us": round(us, 1), "GBps": round(nb / (us * 1e-6) / 1e9, 1),
        "frac_hbm": round(nb / (us * 1e-6) / 1e9 / PEAK_HBM_GBS, 4),
        "unfused_us": round(us_un, 1)}
    del gate, up, h, codes
    n = 8192
    z = torch.randn((M, n), generator=g, device=dev).to(torch.float16)
    codes = torch.empty((M, n // 2), dtype=torch.uint8, device=dev)
    us = time_us(torch, stream,
                 lambda: q.quarot_hadamard_heads_quant_int4(z, 64, q=codes, scale=sc))
    nb = M * n * 2 + M * n // 2 + 2 * M
    res["hadamard_heads_quant_int4"] = {
        "workload": f"attention output fp16 [{M}, 64 heads x 128] -> H_64 x I_128 -> int4",
        "us": round(us, 1), "GBps": round(nb / (us * 1e-6) / 1e9, 1),
        "frac_hbm": round(nb / (us * 1e-6) / 1e9 / PEAK_HBM_GBS, 4)}
    del z, codes
    w8 = {}
    for L in layers:
        wl = L["wl"]
        xq, sx = q.quarot_quant_int8(L["xd"], rotate=True, bits=8)
        wd = torch.from_numpy(L["w"]).to(dev)
        wq, sw = q.quarot_quant_int8(wd, rotate=True, bits=8)
        del wd
        y = L["y"]
        us = time_us(torch, stream, lambda: q.quarot_w8a8_gemm(xq, sx, wq, sw, y=y))
        ops = 2 * wl.M * wl.N * wl.K
        w8[wl.name] = {"us": round(us, 1), "TOPS": round(ops / (us * 1e-6) / 1e12, 1),
                       "frac_int8_peak": round(ops / (us * 1e-6) / 1e12 / PEAK_I8_TOPS, 4)}
        del xq, wq
    res["w8a8_gemm"] = w8
    # group-wise W4A4 (G = 128 on both FFN shapes; 64 and 256 on the up
    # shape): rotate to binary32 + group quantizer, and the grouped GEMM
    gw = {}
    for L in layers:
        wl = L["wl"]
        for G in ((64, 128, 256) if wl.name == "llama2_70b_up" else (128,)):
            wd = torch.from_numpy(L["w"]).to(dev)
            wq, sw = q.quarot_quant_int4_grouped(wd, group=G, rotate=True)
            del wd
            xq = torch.empty((wl.M, wl.K // 2), dtype=torch.uint8, device=dev)
            sx = torch.empty((wl.K // G, wl.M), dtype=torch.float16, device=dev)
            ws = torch.empty(q.lib().quarot_quant_int4_grouped_workspace_size(wl.M, wl.K, 1),
                             dtype=torch.uint8, device=dev)
            us_q = time_us(torch, stream, lambda: q.quarot_quant_int4_grouped(
                L["xd"], group=G, rotate=True, q=xq, scale=sx, workspace=ws))
            del ws
            y = L["y"]
            us_g = time_us(torch, stream,
                           lambda: q.quarot_w4a4_gemm_grouped(xq, sx, wq, sw, group=G, y=y))
            ops = 2 * wl.M * wl.N * wl.K
            ent = {"quant_us": round(us_q, 1), "gemm_us": round(us_g, 1),
                   "gemm_TOPS": round(ops / (us_g * 1e-6) / 1e12, 1),
                   "frac_int8_peak": round(ops / (us_g * 1e-6) / 1e12 / PEAK_I8_TOPS, 4)}
            if G >= 128:
                # the same codes as e3m2 operands on the fp6 matrix cores
                # (repacked once, untimed, like the per-token path's weights)
                xq6, wq6 = q.quarot_pack_e3m2(xq), q.quarot_pack_e3m2(wq)
                us_6 = time_us(torch, stream, lambda: q.quarot_w4a4_gemm_grouped_e3m2(
                    xq6, sx, wq6, sw, group=G, y=y))
                ent["e3m2_gemm_us"] = round(us_6, 1)
                ent["e3m2_gemm_TOPS"] = round(ops / (us_6 * 1e-6) / 1e12, 1)
                ent["e3m2_frac_int8_peak"] = round(ops / (us_6 * 1e-6) / 1e12 / PEAK_I8_TOPS, 4)
                del xq6, wq6
            gw[f"{wl.name}_g{G}"] = ent
            del xq, sx, wq, sw
    res["w4a4_grouped"] = gw
    torch.cuda.empty_cache()
    return res


def main():
    gc.disable()  # collections happen only at quiet_host(), between timed regions
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--cpu-rows", type=int, default=384,
                    help="rows per layer of the oracle's CPU-baseline sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-kv", action="store_true", help="skip the KV-cache leg")
    ap.add_argument("--kv-iters", type=int, default=5)
    ap.add_argument("--no-next", action="store_true",
                    help="skip the fused-prologue and 8-bit legs")
    ap.add_argument("--no-7b", action="store_true",
                    help="skip the Llama-2-7B layer shapes and the tiny layer")
    ap.add_argument("--only-7b", action="store_true",
                    help="run only the Llama-2-7B layer shapes and the tiny layer (for "
                         "profiling their kernels); prints their figures alone")
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
    if args.only_7b:
        res = bench_layers_7b(q, workloads, torch, np, dev, torch.cuda.current_stream(),
                              max(args.steps, 10))
        print(json.dumps({"llama2_7b_and_tiny": res}), flush=True)
        return
    layers = []
    for name in ("llama2_70b_up", "llama2_70b_down"):
        wl = workloads.LINEAR[name]
        log(f"generating {name}: M={wl.M} K={wl.K} N={wl.N}")
        x, w, _ = workloads.linear_inputs(wl)
        xd = torch.from_numpy(x).to(dev)
        wd = torch.from_numpy(w).to(dev)
        wq, sw = q.prepare_weight(wd, rotate=True)  # offline step, untimed
        del wd
        w6 = q.quarot_pack_e3m2(wq)  # offline repack, untimed
        ws = torch.empty(q.quarot_linear_workspace_size(wl.M, wl.K), dtype=torch.uint8,
                         device=dev)
        xq = ws[: wl.M * wl.K // 2].view(wl.M, wl.K // 2)
        off = (wl.M * wl.K // 2 + 255) // 256 * 256
        sx = ws[off: off + 2 * wl.M].view(torch.float16)
        x6 = torch.empty((wl.K // 128, wl.M * 96), dtype=torch.uint8, device=dev)
        sx6 = torch.empty((wl.M,), dtype=torch.float16, device=dev)
        y = torch.empty((wl.M, wl.N), dtype=torch.float16, device=dev)
        layers.append(dict(wl=wl, x=x, w=w, xd=xd, wq=wq, sw=sw, w6=w6, xq=xq, sx=sx, x6=x6,
                           sx6=sx6, y=y))
    torch.cuda.synchronize()

    stream = torch.cuda.current_stream()

    def step(ev=None):
        for li, L in enumerate(layers):
            if ev is not None:
                ev[2 * li].record(stream)
            q.quarot_quant_int4_e3m2(L["xd"], rotate=True, clip_ratio=1.0, q6=L["x6"],
                                     scale=L["sx6"])
            if ev is not None:
                ev[2 * li + 1].record(stream)
            q.quarot_w4a4_gemm_e3m2(L["x6"], L["sx6"], L["w6"], L["sw"], y=L["y"])
        if ev is not None:
            ev[4].record(stream)

    def step_int4(ev=None):
        for li, L in enumerate(layers):
            if ev is not None:
                ev[2 * li].record(stream)
            q.quarot_quant_int4(L["xd"], rotate=True, clip_ratio=1.0, q=L["xq"], scale=L["sx"])
            if ev is not None:
                ev[2 * li + 1].record(stream)
            q.quarot_w4a4_gemm(L["xq"], L["sx"], L["wq"], L["sw"], y=L["y"])
        if ev is not None:
            ev[4].record(stream)

    def split(events):
        """per-kernel durations from a step's events (ms)"""
        rot = [[], []]
        gem = [[], []]
        for ev in events:
            for li in range(2):
                rot[li].append(ev[2 * li].elapsed_time(ev[2 * li + 1]))
                end = ev[2 * li + 2] if li == 0 else ev[4]
                gem[li].append(ev[2 * li + 1].elapsed_time(end))
        return rot, gem

    log(f"warmup {args.warmup}")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    events = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(args.steps)]
    quiet_host()
    log(f"timing {args.steps} steps")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(args.steps):
        step(events[s])
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_step = (t1 - t0) * 1e3 / args.steps
    rot, gem = split(events)

    # the int4-operand path on the same inputs, for comparison (same outputs)
    for _ in range(args.warmup):
        step_int4()
    ev4 = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(args.steps)]
    quiet_host()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(args.steps):
        step_int4(ev4[s])
    torch.cuda.synchronize()
    ms_step4 = (time.perf_counter() - t0) * 1e3 / args.steps
    rot4, gem4 = split(ev4)
    ops = [2 * L["wl"].M * L["wl"].N * L["wl"].K for L in layers]
    total_ops = sum(ops)
    value = total_ops / (ms_step * 1e-3) / 1e12
    gemm_ms = [float(np.mean(g)) for g in gem]
    rot_ms = [float(np.mean(r)) for r in rot]
    gemm_tops = sum(ops) / (sum(gemm_ms) * 1e-3) / 1e12
    gemm4_ms = [float(np.mean(g)) for g in gem4]
    rot4_ms = [float(np.mean(r)) for r in rot4]
    gemm4_tops = sum(ops) / (sum(gemm4_ms) * 1e-3) / 1e12
    rbytes = [rotate_bytes(L["wl"].M, L["wl"].K, 6) for L in layers]
    rbytes4 = [rotate_bytes(L["wl"].M, L["wl"].K, 4) for L in layers]
    kernels = {}
    for li, L in enumerate(layers):
        wl = L["wl"]
        nm = wl.name
        k2, m = q.quarot_hadamard_factor(wl.K)
        # VALU floor of the rotation: log2(2^k) butterfly adds and m - 1
        # m-factor adds per element at the fp32 vector add rate
        valu_us = wl.M * wl.K * (k2 + m - 1) / PEAK_F32_ADDS * 1e6
        hbm_us = rbytes[li] / (PEAK_HBM_GBS * 1e9) * 1e6
        pct = lambda a, p_: [round(float(np.percentile(a, p_)) * 1e3, 1) for p_ in p_]
        kernels[nm] = {
            "rotate_quant_us": round(rot_ms[li] * 1e3, 2),
            "rotate_quant_us_p10_p50_p90": pct(rot[li], (10, 50, 90)),
            "rotate_quant_GBps": round(rbytes[li] / (rot_ms[li] * 1e-3) / 1e9, 1),
            "rotate_quant_frac_hbm": round(hbm_us / (rot_ms[li] * 1e3), 4),
            "rotate_quant_frac_valu_bound": round(valu_us / (rot_ms[li] * 1e3), 4),
            "gemm_us": round(gemm_ms[li] * 1e3, 2),
            "gemm_us_p10_p50_p90": pct(gem[li], (10, 50, 90)),
            "gemm_TOPS": round(ops[li] / (gemm_ms[li] * 1e-3) / 1e12, 1),
            "linear_TOPS": round(ops[li] / ((gemm_ms[li] + rot_ms[li]) * 1e-3) / 1e12, 1),
            "int4_operands": {
                "rotate_quant_us": round(rot4_ms[li] * 1e3, 2),
                "rotate_quant_GBps": round(rbytes4[li] / (rot4_ms[li] * 1e-3) / 1e9, 1),
                "gemm_us": round(gemm4_ms[li] * 1e3, 2),
                "gemm_us_p10_p50_p90": pct(gem4[li], (10, 50, 90)),
                "gemm_TOPS": round(ops[li] / (gemm4_ms[li] * 1e-3) / 1e12, 1),
                "linear_TOPS": round(ops[li] / ((gemm4_ms[li] + rot4_ms[li]) * 1e-3) / 1e12, 1),
            },
        }

    # the int8 MFMA peak re-derived from the device (CUs x peak clock x 8192
    # ops per clock per CU) and an MFMA-only probe's attainable rate
    cus, clk_khz = q.quarot_device_peaks()
    probe_out = torch.empty(cus * 512, dtype=torch.int32, device=dev)
    probe_ops = q.quarot_mfma_probe(probe_out, cus, 2000)
    torch.cuda.synchronize()
    quiet_host()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(10):
        q.quarot_mfma_probe(probe_out, cus, 2000)
    e1.record(stream)
    torch.cuda.synchronize()
    probe_tops = probe_ops * 10 / (e0.elapsed_time(e1) * 1e-3) / 1e12
    probe6_ops = q.quarot_mfma_probe_fp6(probe_out, cus, 2000)
    torch.cuda.synchronize()
    quiet_host()
    e0.record(stream)
    for _ in range(10):
        q.quarot_mfma_probe_fp6(probe_out, cus, 2000)
    e1.record(stream)
    torch.cuda.synchronize()
    probe6_tops = probe6_ops * 10 / (e0.elapsed_time(e1) * 1e-3) / 1e12
    del probe_out
    peak_i8 = {"cus": cus, "peak_sclk_mhz": clk_khz / 1000,
               "derived_TOPS": round(cus * clk_khz * 1e3 * 8192 / 1e12, 1),
               "published_TOPS": PEAK_I8_TOPS,
               "mfma_probe_TOPS": round(probe_tops, 1),
               "int4_operand_gemm_frac_of_probe": round(gemm4_tops / probe_tops, 4)}
    # fp6: v_mfma_f32_16x16x128_f8f6f4 does 16 x 16 x 128 multiply-adds in 16
    # cycles per SIMD, 16384 ops per clock per CU
    peak_fp6 = {"derived_TOPS": round(cus * clk_khz * 1e3 * 16384 / 1e12, 1),
                "published_TOPS": PEAK_FP6_TOPS,
                "mfma_probe_TOPS": round(probe6_tops, 1),
                "gemm_frac_of_probe": round(gemm_tops / probe6_tops, 4)}

    # the rotations warm (the same input back to back) and cold (copies of
    # the input totalling > 512 MB, twice the last-level cache, in turn)
    for li, L in enumerate(layers):
        wl = L["wl"]
        rot = lambda xd=L["xd"], L=L: q.quarot_quant_int4_e3m2(xd, rotate=True, q6=L["x6"],
                                                               scale=L["sx6"])
        warm = event_times_us(torch, stream, [rot], 10)[0]
        ncp = max(2, -(-(640 << 20) // (L["xd"].numel() * 2)))
        xs = [L["xd"]] + [L["xd"].clone() for _ in range(ncp - 1)]
        cold = event_times_us(torch, stream,
                              [lambda xc=xc, L=L: q.quarot_quant_int4_e3m2(
                                  xc, rotate=True, q6=L["x6"], scale=L["sx6"]) for xc in xs], 3)
        del xs
        hbm_us, _ = rotation_bounds(q, wl.M, wl.K, 6)
        w_us = float(np.mean(warm))
        c_us = float(np.mean([v for c in cold for v in c]))
        kernels[wl.name]["rotate_quant_warm_us"] = round(w_us, 2)
        kernels[wl.name]["rotate_quant_cold_us"] = round(c_us, 2)
        kernels[wl.name]["rotate_quant_cold_frac_hbm"] = round(hbm_us / c_us, 4)
        # the standalone rotation (fp16 in, fp16 out: 4 bytes per element)
        yh = torch.empty_like(L["xd"])
        had = event_times_us(torch, stream,
                             [lambda xd=L["xd"], yh=yh: q.quarot_hadamard(xd, y=yh)], 10)[0]
        del yh
        h_us = float(np.mean(had))
        h_gbs = wl.M * wl.K * 4 / (h_us * 1e-6) / 1e9
        kernels[wl.name]["hadamard_fp16_us"] = round(h_us, 2)
        kernels[wl.name]["hadamard_fp16_GBps"] = round(h_gbs, 1)
        kernels[wl.name]["hadamard_fp16_frac_hbm"] = round(h_gbs / PEAK_HBM_GBS, 4)
    torch.cuda.empty_cache()

    drawn_7b = {}
    small = None if args.no_7b else bench_layers_7b(q, workloads, torch, np, dev, stream,
                                                      max(args.steps, 10), keep=drawn_7b)
    kv = None if args.no_kv else bench_kv(q, workloads, torch, np, dev, stream, args.kv_iters)
    nxt = None if args.no_next else bench_next(q, torch, dev, stream, layers)

    if args.copy_mib:
        src = torch.empty(args.copy_mib << 20, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        src.fill_(1)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    cpu = None
    cpu_all = None
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
                         f"(rotate+quantize+GEMM+dequant), {dt:.1f} s",
               "cpu_model": cpu_model()}
        log("cpu oracle per workload (all threads and one)")
        inputs = {L["wl"].name: (L["x"][:256], *prep) for L, prep in zip(layers, preps)}
        for name, (x7, w7) in drawn_7b.items():
            inputs[name] = (x7, *orc.prepare_weight(w7, rotate=True))
        cpu_all = cpu_oracle_per_config(workloads, np, inputs)

    traffic = gemm_traffic("k_gemm_w4a4_e3m2")
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
        "dtype": "int4 codes as e3m2 (fp6 MFMA, exact fp32 sums)",
        "data": "synthetic",
        "config": {"workload": "llama2_70b_ffn_prefill: M=16384 tokens (batch 8 x seq 2048); "
                               "up K=8192->N=28672 (H_8192), down K=28672->N=8192 "
                               "(H_1024 x H_28)",
                   "global_batch": 8, "seq_len": 2048, "parallelism": "none"},
        "pct_int8_peak": round(100 * value / PEAK_I8_TOPS, 2),
        "roofline": {"bound": "mfma", "kernel": "k_gemm_w4a4_e3m2",
                     "achieved": round(gemm_tops, 1), "peak": PEAK_FP6_TOPS, "unit": "TOP/s",
                     "frac": round(gemm_tops / PEAK_FP6_TOPS, 4), "traffic": traffic},
        "int4_operand_path": {"ms_per_step": round(ms_step4, 4),
                              "value": round(sum(ops) / (ms_step4 * 1e-3) / 1e12, 2),
                              "gemm_kernel": "k_gemm_w4a4", "gemm_TOPS": round(gemm4_tops, 1),
                              "gemm_frac_int8_peak": round(gemm4_tops / PEAK_I8_TOPS, 4),
                              "traffic": gemm_traffic("k_gemm_w4a4")},
        "kernels": kernels,
        "peak_i8": peak_i8,
        "peak_fp6": peak_fp6,
        "llama2_7b_and_tiny": small,
        "kv": kv,
        "next": nxt,
        "cpu_baseline": cpu,
        "cpu_oracle_per_workload": cpu_all,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
