"""Precision modes of the oracle.

Pinning: ``round_bf16`` is pinned against torch's float32 -> bfloat16
conversion (round-to-nearest-even) in tests/test_oracle_primitives.py.
"""
from __future__ import annotations

import numpy as np

# Where the bf16 mode rounds an fp32 value to bf16 (values are otherwise fp32):
BF16_STORAGE_POINTS = (
    "RMSNorm output (attention, FFN and final norms)",
    "Q/K/V projection output",
    "q and k after QK-norm and RoPE (K/V cache contents)",
    "attention output (input of the O projection)",
    "residual stream after each residual add (fp32 add of bf16 residual and fp32 GEMM result)",
    "SiLU(gate) * up product (fp32 gate/up accumulators)",
    "fused target feature F = RMSNorm(W_c [..]) (fp32 GEMM + fp32 norm)",
    "relay hidden layer SiLU(W1 u + c1)",
    "drafter input rows x (E_mask + beta * LN(h) + gamma)",
)


def round_bf16(x: np.ndarray) -> np.ndarray:
    """fp32 -> nearest-even bf16 value, returned as float32."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    finite = np.isfinite(x)
    r = ((u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) & np.uint32(0xFFFF0000))
    r = np.where(finite, r, u & np.uint32(0xFFFF0000))
    return r.astype(np.uint32).view(np.float32)


class Mode:
    """Arithmetic type and storage rounding of the oracle."""

    def __init__(self, name: str):
        if name not in ("fp64", "fp32", "bf16"):
            raise ValueError(name)
        self.name = name
        self.dt = np.float64 if name == "fp64" else np.float32

    def st(self, x: np.ndarray) -> np.ndarray:
        """Value as stored between steps."""
        if self.name == "bf16":
            return round_bf16(x)
        return np.asarray(x, dtype=self.dt)

    def __repr__(self):
        return f"Mode({self.name})"
