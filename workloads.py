"""Seeded synthetic inputs for the W4A4 rotated-linear path.

This module holds the workload shapes and the random draws only: no rotation,
quantization or any other step of the method.  It is the one piece that the
GPU path's tests and bench and the CPU oracle's tests both use.

The shapes follow the paper's Llama-2 layer sizes at sequence length 2048
(App. A.10, 4-bit linear-layer table) and its KV-cache setting (§5 Setup:
head dimension 128).  No dataset or checkpoint is used: activations are
normal or Student-t draws with planted outlier channels (the outlier feature
structure that §1 and §3.2 describe), weights are N(0, 0.02^2).

Recipe, per workload, with ``numpy.random.default_rng(seed)``:
  1. outlier channel indices: ``rng.choice(K, n_out, replace=False)``, sorted;
  2. X: ``standard_normal(dtype=float32)`` (or ``standard_t(3)`` cast to
     float32), outlier columns multiplied in float32, then ``astype(float16)``;
  3. W: ``0.02 * standard_normal(dtype=float32)``, then ``astype(float16)``.
KV: K then V, each ``standard_normal(float32)`` of [B, H, S, D]; one
``rng.choice(D, 2, replace=False)`` per (tensor, head) picks two outlier dims
that every batch entry and token shares, scaled by 20.
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np


@dataclasses.dataclass(frozen=True)
class LinearWorkload:
    name: str
    M: int
    K: int
    N: int
    x_dist: str = "normal"          # "normal" or "student_t3"
    n_outliers: int = 0
    outlier_scale: float = 1.0
    seed: int = 0

    @property
    def gemm_ops(self) -> int:
        return 2 * self.M * self.N * self.K


@dataclasses.dataclass(frozen=True)
class KVWorkload:
    name: str
    B: int
    H: int
    S: int
    D: int = 128
    outlier_dims: int = 2
    outlier_scale: float = 20.0
    group: int = 128
    clip: float = 0.95
    seed: int = 0

    @property
    def rows(self) -> int:
        return self.B * self.H * self.S


LINEAR = {
    # 2 fixed outlier channels x50, online Hadamard n = 128
    "tiny": LinearWorkload("tiny", 16, 128, 256, "normal", 2, 50.0),
    # Llama-2-7B QKV/up-proj shape: 1% outlier channels x50 (round(0.01*4096) = 41)
    "llama2_7b_up": LinearWorkload("llama2_7b_up", 2048, 4096, 11008, "normal", 41, 50.0),
    # Llama-2-7B down-proj shape: heavy-tailed activations, n = 64 * 172
    "llama2_7b_down": LinearWorkload("llama2_7b_down", 2048, 11008, 4096, "student_t3"),
    # Llama-2-70B prefill, batch 8 x seq 2048: 0.5% outlier channels x100
    "llama2_70b_up": LinearWorkload("llama2_70b_up", 16384, 8192, 28672, "normal", 41, 100.0),
    "llama2_70b_down": LinearWorkload("llama2_70b_down", 16384, 28672, 8192, "normal", 143,
                                      100.0),
}

KV = {
    "kv4_70b": KVWorkload("kv4_70b", 16, 64, 4096, 128),
}


def linear_inputs(w: LinearWorkload, M: Optional[int] = None, N: Optional[int] = None,
                  weights: bool = True):
    """Returns (x fp16 [M, K], weight fp16 [N, K] or None, outlier indices).

    A smaller ``M`` is its own seeded workload (W is drawn after X, so it
    changes W).  A smaller ``N`` keeps the first N weight rows of the same
    draw.  ``weights=False`` skips the weight draw (X is unaffected)."""
    M = w.M if M is None else M
    N = w.N if N is None else N
    rng = np.random.default_rng(w.seed)
    idx = np.sort(rng.choice(w.K, w.n_outliers, replace=False)) if w.n_outliers else \
        np.zeros(0, np.int64)
    x = np.empty((M, w.K), np.float16)
    chunk = 4096
    for r0 in range(0, M, chunk):
        r1 = min(M, r0 + chunk)
        if w.x_dist == "normal":
            blk = rng.standard_normal((r1 - r0, w.K), dtype=np.float32)
        elif w.x_dist == "student_t3":
            blk = rng.standard_t(3, size=(r1 - r0, w.K)).astype(np.float32)
        else:
            raise ValueError(w.x_dist)
        if len(idx):
            blk[:, idx] *= np.float32(w.outlier_scale)
        x[r0:r1] = blk.astype(np.float16)
    if not weights:
        return x, None, idx
    wt = np.empty((N, w.K), np.float16)
    for r0 in range(0, N, chunk):
        r1 = min(N, r0 + chunk)
        wt[r0:r1] = (np.float32(0.02) *
                     rng.standard_normal((r1 - r0, w.K), dtype=np.float32)).astype(np.float16)
    return x, wt, idx


def kv_inputs(w: KVWorkload, B: Optional[int] = None, S: Optional[int] = None):
    """Returns (k, v) fp16 [B, H, S, D]; smaller B/S give their own draw."""
    B = w.B if B is None else B
    S = w.S if S is None else S
    rng = np.random.default_rng(w.seed)
    outs = []
    for _ in range(2):
        t = np.empty((B, w.H, S, w.D), np.float16)
        dims = [np.sort(rng.choice(w.D, w.outlier_dims, replace=False)) for _ in range(w.H)]
        for b in range(B):
            blk = rng.standard_normal((w.H, S, w.D), dtype=np.float32)
            for h in range(w.H):
                blk[h][:, dims[h]] *= np.float32(w.outlier_scale)
            t[b] = blk.astype(np.float16)
        outs.append(t)
    return outs[0], outs[1]


def random_rows(seed: int, rows: int, n: int, dist: str = "normal", scale: float = 1.0):
    """Plain seeded fp16 rows for property and edge-case tests."""
    rng = np.random.default_rng(seed)
    if dist == "normal":
        a = rng.standard_normal((rows, n), dtype=np.float32)
    elif dist == "student_t3":
        a = rng.standard_t(3, size=(rows, n)).astype(np.float32)
    elif dist == "uniform":
        a = rng.uniform(-1, 1, size=(rows, n)).astype(np.float32)
    else:
        raise ValueError(dist)
    return (a * np.float32(scale)).astype(np.float16)
