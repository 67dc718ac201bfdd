"""Seeded synthetic inputs for the attention forward pass.

This module is the only code shared by the oracle side and the HIP side: it
draws the inputs and holds none of the method's arithmetic.  Inputs follow the
paper's workloads (Section 4, Table "mha_sweep" and Table "model_params"):
attention shapes only, no dataset.  Q, K and V are i.i.d. N(0, 1), drawn in
float32 from a seeded CPU ``torch.Generator`` and rounded to bfloat16
(round-to-nearest-even), in BHSD contiguous layout.
"""

from __future__ import annotations

import math

import numpy as np
import torch

# The five workloads: (B, Hq, Hkv, S, d, causal).  Seeds are 1000*index + {0,1,2}
# for Q, K, V.
WORKLOADS = {
    "mha_b1_h4_s256_d64": dict(index=1, B=1, Hq=4, Hkv=4, Sq=256, Skv=256, d=64, causal=False),
    "mha_b1_h32_s8192_d128_causal": dict(index=2, B=1, Hq=32, Hkv=32, Sq=8192, Skv=8192, d=128,
                                         causal=True),
    "gqa_b1_hq64_hkv8_s8192_d128_causal": dict(index=3, B=1, Hq=64, Hkv=8, Sq=8192, Skv=8192,
                                               d=128, causal=True),
    "mha_b8_h64_s4096_d128": dict(index=4, B=8, Hq=64, Hkv=64, Sq=4096, Skv=4096, d=128,
                                  causal=False),
    "mha_b1_h16_s131072_d128_causal": dict(index=5, B=1, Hq=16, Hkv=16, Sq=131072, Skv=131072,
                                           d=128, causal=True),
}


def default_scale(d: int) -> float:
    """The float32 value of 1/sqrt(d) that callers pass as ``scale``."""
    return float(np.float32(1.0 / math.sqrt(d)))


def randn_bf16(shape, seed: int) -> torch.Tensor:
    g = torch.Generator(device="cpu")
    g.manual_seed(int(seed))
    return torch.randn(*shape, generator=g, dtype=torch.float32).to(torch.bfloat16)


def make_qkv(B: int, Hq: int, Hkv: int, Sq: int, Skv: int, d: int, seed_base: int):
    """CPU bf16 tensors q[B,Hq,Sq,d], k[B,Hkv,Skv,d], v[B,Hkv,Skv,d]."""
    q = randn_bf16((B, Hq, Sq, d), seed_base + 0)
    k = randn_bf16((B, Hkv, Skv, d), seed_base + 1)
    v = randn_bf16((B, Hkv, Skv, d), seed_base + 2)
    return q, k, v


def workload_inputs(name: str):
    w = WORKLOADS[name]
    return make_qkv(w["B"], w["Hq"], w["Hkv"], w["Sq"], w["Skv"], w["d"], 1000 * w["index"])


def bf16_bits(t: torch.Tensor) -> np.ndarray:
    """uint16 view of a CPU bf16 tensor's bit patterns (no copy when contiguous)."""
    t = t.detach().contiguous()
    if t.dtype != torch.bfloat16 or t.device.type != "cpu":
        raise TypeError("expected a CPU bfloat16 tensor")
    return t.view(torch.int16).numpy().view(np.uint16)


def bits_to_bf16(a: np.ndarray) -> torch.Tensor:
    """CPU bf16 tensor from uint16 bit patterns."""
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.uint16).view(np.int16)).view(
        torch.bfloat16)


def sample_rows(B: int, Hq: int, Sq: int, block_m: int, n_random: int, seed: int) -> np.ndarray:
    """Fixed plus seeded random query rows per (b, hq): rows [n, 3] of (b, hq, i).

    Fixed rows: 0, 1, block_m-1, block_m, Sq//2, Sq-1 (those below Sq), which
    hit the first and a boundary row block and the ragged last block.
    """
    rng = np.random.default_rng(seed)
    fixed = sorted({i for i in (0, 1, block_m - 1, block_m, Sq // 2, Sq - 1) if 0 <= i < Sq})
    out = []
    for b in range(B):
        for h in range(Hq):
            extra = rng.integers(0, Sq, size=n_random) if n_random > 0 else []
            for i in sorted(set(fixed) | {int(x) for x in extra}):
                out.append((b, h, i))
    return np.asarray(out, dtype=np.int64).reshape(-1, 3)
