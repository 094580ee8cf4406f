"""Helpers shared by the GPU parity tests (error metrics and tensor transfer).

Tolerances (stated once):
* Outputs z of Eq. (10): per-row normwise relative error
      err = max over (beta, h, i) of ||z_gpu[i] - z_ref[i]||_inf / ||z_ref[i]||_inf
  must be <= 2e-4 when q, k, v are fp32 and <= 2e-2 when they are bf16.
  z entries cross zero, so an elementwise relative error is ill-posed; the
  normwise form measures the error against the row's own scale.  (For bf16
  the inputs are the same bf16 values on both sides; the looser bar covers
  the heavier-tailed intermediates of those workloads.)
* Toeplitz products: per-channel normwise relative error <= 2e-4 (fp32 data).
* Feature map phi (> 0, no cancellation): elementwise relative error <= 2e-4.
"""
from __future__ import annotations

import numpy as np
import torch

TOL = {"f32": 2e-4, "bf16": 2e-2}


def rownorm_err(got: np.ndarray, ref: np.ndarray) -> float:
    """max over leading indices of ||got - ref||_inf / ||ref||_inf along the last axis."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    num = np.max(np.abs(got - ref), axis=-1)
    den = np.max(np.abs(ref), axis=-1)
    return float(np.max(num / den))


def to_gpu(x: np.ndarray, dtype: str = "f32") -> torch.Tensor:
    """fp32 numpy -> CUDA tensor; for 'bf16' the values must already be bf16-exact."""
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).cuda()
    if dtype == "bf16":
        tb = t.to(torch.bfloat16)
        assert torch.equal(tb.float(), t), "values are not bf16-exact"
        return tb
    return t


def inputs_to_gpu(d: dict) -> tuple:
    dt = d["workload"].qkv_dtype
    return (to_gpu(d["q"], dt), to_gpu(d["k"], dt), to_gpu(d["v"], dt), to_gpu(d["b"]), to_gpu(d["W"]))


def sample_rows(B: int, H: int, n: int, count: int, seed: int, extra=()) -> list[tuple[int, int, int]]:
    """Seeded (beta, h, i) rows spread over all heads, always including the sequence ends."""
    rng = np.random.default_rng([12566, seed])
    rows = set(extra)
    for beta, h in [(0, 0), (B - 1, H - 1)]:
        for i in (0, 1, n // 2, n - 2, n - 1):
            if 0 <= i < n:
                rows.add((beta, h, i))
    while len(rows) < count:
        rows.add((int(rng.integers(B)), int(rng.integers(H)), int(rng.integers(n))))
    return sorted(rows)
