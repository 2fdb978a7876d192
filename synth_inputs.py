"""Seeded synthetic inputs for the ATP shard block.

This module is the only thing the oracle and the HIP path have in common:
it draws random tensors and holds none of the method's arithmetic (no
sharding, no GEMM, no reduction).  Every draw is

    torch.Generator('cpu').manual_seed(seed * 100 + tensor_id)
    -> randn (float32) * std -> rounded to bf16 (round-to-nearest-even)

so a tensor is fixed by (seed, tensor_id, shape, std) on any machine.
Integer-valued draws (values in [-3, 3]) are exact in bf16 and keep every
fp32 partial sum exact, which gives bit-exact GPU checks.

Distributions (the paper names no dataset; it trains synthetic GPT layers
with batch 4 x sequence 2048, Sec. 5 and Table 2): activations N(0, 1),
weights N(0, 0.02^2) (N(0, 0.01^2) for the h = 20480 stress shape), biases
zero or N(0, 0.02^2), peer partial sums N(0, sigma_p^2) with
sigma_p = sqrt(K_loc) * sigma_w * sigma_in (the spread of a real partial
GEMM output), upstream gradients N(0, 1).
"""
from __future__ import annotations

import math

import torch

# tensor ids: fixed so every harness draws the same values
TID = dict(x=1, a=2, w_qkv=3, w_out=4, w_fc1=5, w_fc2=6, b_qkv=7, b_out=8, b_fc1=9,
           b_fc2=10, dz=11, dqkv=12, do=13, h=14, pre=15)
PEER_TID_BASE = 1000      # + 100 * linear index + peer position
BWD_PEER_TID_BASE = 2000


def _gen(seed: int, tid: int) -> torch.Generator:
    g = torch.Generator(device="cpu")
    g.manual_seed(int(seed) * 100 + int(tid))
    return g


def randn_bf16(shape, std: float, seed: int, tid: int) -> torch.Tensor:
    """N(0, std^2) rounded to bf16, on the CPU."""
    t = torch.randn(tuple(shape), generator=_gen(seed, tid), dtype=torch.float32)
    if std != 1.0:
        t = t * std
    return t.to(torch.bfloat16)


def randn_f32(shape, std: float, seed: int, tid: int) -> torch.Tensor:
    t = torch.randn(tuple(shape), generator=_gen(seed, tid), dtype=torch.float32)
    if std != 1.0:
        t = t * std
    return t


def randint_bf16(shape, seed: int, tid: int, lo: int = -3, hi: int = 3) -> torch.Tensor:
    """Integers in [lo, hi], exact in bf16."""
    t = torch.randint(lo, hi + 1, tuple(shape), generator=_gen(seed, tid))
    return t.to(torch.bfloat16)


def randint_f32(shape, seed: int, tid: int, lo: int = -64, hi: int = 64) -> torch.Tensor:
    t = torch.randint(lo, hi + 1, tuple(shape), generator=_gen(seed, tid))
    return t.to(torch.float32)


def zeros_bf16(shape) -> torch.Tensor:
    return torch.zeros(tuple(shape), dtype=torch.bfloat16)


def peer_sigma(k_loc: int, sigma_w: float, sigma_in: float) -> float:
    return math.sqrt(k_loc) * sigma_w * sigma_in


def randn_device(shape, std: float, seed: int, tid: int, device, dtype=torch.bfloat16):
    """Large draws made directly on a device (benchmark inputs only; the
    generator is torch's own, no kernel of this project is involved)."""
    g = torch.Generator(device=device)
    g.manual_seed(int(seed) * 100 + int(tid))
    t = torch.randn(tuple(shape), generator=g, dtype=torch.float32, device=device)
    if std != 1.0:
        t.mul_(std)
    return t.to(dtype)


# --------------------------------------------------------------------------
# Workloads (sizes follow the paper's GPT layers: Table 2 hidden sizes,
# batch x sequence 2048, Sec. 5), named by what they are.
# mode: "col" = QKV/fc1 column-first, out/fc2 row-first; "row" = swapped.
# --------------------------------------------------------------------------
WORKLOADS = {
    "tiny_mlp_h512_col_2x2": dict(mode="col", mesh=(2, 2), tokens=256, h=512, chunks=2,
                                  sigma_w=0.02, bwd=False),
    "gpt_h4096_col_2x4": dict(mode="col", mesh=(2, 4), tokens=8192, h=4096, chunks=4,
                              sigma_w=0.02, bwd=False),
    "gpt_h4096_row_4x2": dict(mode="row", mesh=(4, 2), tokens=8192, h=4096, chunks=4,
                              sigma_w=0.02, bwd=True, chunk_sweep=(1, 2, 4, 8)),
    "gpt3_h12288_col_4x2": dict(mode="col", mesh=(4, 2), tokens=2048, h=12288, chunks=4,
                                sigma_w=0.02, bwd=True),
    "wide_h20480_col_8x1": dict(mode="col", mesh=(8, 1), tokens=4096, h=20480, chunks=8,
                                sigma_w=0.01, bwd=True),
    "wide_h20480_col_2x4": dict(mode="col", mesh=(2, 4), tokens=4096, h=20480, chunks=8,
                                sigma_w=0.01, bwd=True),
}
