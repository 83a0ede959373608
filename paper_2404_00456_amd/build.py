"""Build libquarot.so (HIP for gfx950) and, beside it, the measurement
library libquarot_probe.so in-tree with hipcc.

    python -m paper_2404_00456_amd.build
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libquarot.so")
SOURCES = ["capi.cpp", "host_rules.cpp", "rotate_quant.hip", "gemm_w4a4.hip", "gemm_grouped.hip", "kv_attention.hip",
           "scratch.hip"]
# MFMA-only rate probes and the device's peak clock (include/quarot_probe.h)
PROBE_LIB = os.path.join(HERE, "libquarot_probe.so")
PROBE_SOURCES = ["probe.hip"]

# -ffp-contract=off: every written add and multiply stays a rounded op of
# its own (the rotation order and the dequant order are part of the result).
# -packed-fp32-ops: no packed fp32 VALU instructions anywhere.
FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-ffp-contract=off", "-fno-fast-math",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function", "-Wno-unknown-pragmas",
]


def hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    p = os.path.join(rocm, "bin", "hipcc")
    return p if os.path.exists(p) else "hipcc"


ISA_SHA = os.path.join(HERE, "gemm_isa.sha")
GEMM_KERNELS = {
    "k_gemm_w4a4": "_ZN6quarot12_GLOBAL__N_111k_gemm_w4a4ENS_8GemmArgsE",
    "k_gemm_w4a4_e3m2": "_ZN6quarot12_GLOBAL__N_116k_gemm_w4a4_e3m2ENS_8GemmArgsE",
}


def kernel_isa_sha(src: str, symbol: str) -> str:
    """sha256[:16] of one kernel's gfx950 assembly (comments and directives
    dropped): it changes exactly when that kernel's machine code does."""
    cmd = [hipcc(), *[f for f in FLAGS if f not in ("-fPIC", "-shared")], "-I",
           os.path.join(ROOT, "include"), "-S", "--cuda-device-only", src, "-o", "-"]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError("hipcc -S failed for " + src)
    asm = res.stdout
    start = asm.index(symbol + ":")
    body = asm[start:asm.index(".Lfunc_end", start)]
    lines = [ln.split(";")[0].strip() for ln in body.splitlines()]
    text = "\n".join(ln for ln in lines if ln and not ln.startswith("."))
    import hashlib
    return hashlib.sha256(text.encode()).hexdigest()[:16]


def _link(sources, lib: str, verbose: bool) -> None:
    srcs = [os.path.join(CSRC, s) for s in sources]
    tmp = lib + ".tmp"
    cmd = [hipcc(), *FLAGS, "-I", os.path.join(ROOT, "include"), *srcs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    # hipcc's host pass warns about the device-only target feature: harmless
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError("hipcc failed building " + os.path.basename(lib))
    os.replace(tmp, lib)


def build(verbose: bool = False) -> str:
    _link(SOURCES, LIB, verbose)
    _link(PROBE_SOURCES, PROBE_LIB, verbose)
    # fingerprints of the per-token GEMMs' machine code, which the bench's
    # stored hardware byte counts refer to: one "name sha" line per kernel
    lines = []
    for name, sym in GEMM_KERNELS.items():
        lines.append(f"{name} {kernel_isa_sha(os.path.join(CSRC, 'gemm_w4a4.hip'), sym)}\n")
    with open(ISA_SHA, "w") as f:
        f.writelines(lines)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
