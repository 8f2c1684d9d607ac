"""bfloat16 storage emulation for the oracle.

The bf16 workloads keep weights and the GEMM operands z and h in bfloat16
(8 exponent bits, 7 stored mantissa bits) and accumulate in float32.  ``q``
rounds a value to the nearest bfloat16 with ties to even, after first
rounding it to float32 (the value the device stores before narrowing).
NaN stays NaN; values beyond the bf16 range round to +-inf.  Pinned against
``torch.Tensor.to(torch.bfloat16)`` in a CPU test.
"""

from __future__ import annotations

import numpy as np


def round_bf16(x) -> np.ndarray:
    """Round to bfloat16 (ties to even) and return the value as float64."""
    with np.errstate(over="ignore", invalid="ignore"):
        f = np.asarray(x, dtype=np.float64).astype(np.float32)
    bits = f.view(np.uint32).astype(np.uint64)
    nan = np.isnan(f)
    lsb = (bits >> np.uint64(16)) & np.uint64(1)
    rounded = (bits + np.uint64(0x7FFF) + lsb) & np.uint64(0xFFFF0000)
    rounded = np.where(nan, bits | np.uint64(0x00400000), rounded)
    out = (rounded & np.uint64(0xFFFFFFFF)).astype(np.uint32).view(np.float32)
    return out.astype(np.float64)


def q(x, dtype: str) -> np.ndarray:
    """Storage rounding of the workload's dtype: identity (float64) for fp32."""
    if dtype == "fp32":
        return np.asarray(x, dtype=np.float64)
    if dtype == "bf16":
        return round_bf16(x)
    raise ValueError(f"unknown dtype {dtype!r}")
