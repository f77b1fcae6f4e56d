"""Seeded synthetic inputs for the attention backward workloads.

This module holds no attention arithmetic: it only draws random numbers.  It
is the one piece shared by the HIP path's callers (tests, bench) and the
oracle's callers, so both sides see bit-identical inputs.

Recipe: a CPU ``torch.Generator`` seeded with ``seed`` draws fp32 values
~ N(0, sigma^2) in the order q, k, v, dO, each of shape [B, H, N, d]; every
tensor is then rounded to bf16 (round-to-nearest-even).  The paper benchmarks
on random bf16 inputs (Experimental Setup); these shapes stand in for its
sweep.
"""
from __future__ import annotations

from dataclasses import dataclass

import torch


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    H: int
    N: int
    d: int
    causal: bool
    sigma: float = 1.0

    def flops(self) -> float:
        """Backward FLOPs by the 5-GEMM convention: 4*B*H*N^2*d*2.5, halved when causal."""
        f = 4.0 * self.B * self.H * self.N * self.N * self.d * 2.5
        return f / 2 if self.causal else f


def _token_sweep(d, H, causal, name):
    return {N: Workload(f"{name}_N{N}", 16384 // N, H, N, d, causal) for N in
            (512, 1024, 2048, 4096, 8192, 16384)}


# The workloads: a single-head smoke case, a short-sequence causal case with
# 64x64 tiles, and the fixed-16k-token sweeps of the Experimental Setup
# (B = 16384/N; 16 heads of 128 with a full mask, 32 heads of 128 causal).
WORKLOADS = {
    "single_head_n256_d64_full": Workload("single_head_n256_d64_full", 1, 1, 256, 64, False),
    "b4_h16_n1024_d64_causal": Workload("b4_h16_n1024_d64_causal", 4, 16, 1024, 64, True),
    "b2_h16_n8192_d128_full": Workload("b2_h16_n8192_d128_full", 2, 16, 8192, 128, False),
}
FULL_SWEEP_D128 = _token_sweep(128, 16, False, "tok16k_h16_d128_full")
CAUSAL_SWEEP_D128 = _token_sweep(128, 32, True, "tok16k_h32_d128_causal")


def make_inputs(B: int, H: int, N: int, d: int, seed: int, sigma: float = 1.0):
    """q, k, v, dO as bf16 CPU tensors [B, H, N, d], drawn in that order."""
    g = torch.Generator(device="cpu")
    g.manual_seed(int(seed))
    out = []
    for _ in range(4):
        x = torch.randn((B, H, N, d), generator=g, dtype=torch.float32) * float(sigma)
        out.append(x.to(torch.bfloat16).contiguous())
    return tuple(out)


def make_workload_inputs(w: Workload, seed: int):
    return make_inputs(w.B, w.H, w.N, w.d, seed, w.sigma)
