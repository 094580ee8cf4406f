"""Seeded synthetic workloads for RPE kernelized attention.

This module only *draws inputs*: queries, keys, values, the random-feature
matrix W and the relative-position bias vector b.  It holds none of the
method's arithmetic (no feature map, no Toeplitz product, no attention), so
both the HIP path and the CPU oracle can consume the very same arrays.

Shapes follow the paper's notation (Section 2 and Section 3.2):
  q, k, v : [B, H, n, d]     projected queries / keys / values
  W       : [H, m, d]        rows w_l of the random feature map, Eq. (5)
  b       : [H, 2n-1]        b[h, s] = b_{t} with t = s - (n-1), the layout
                             (b_{-(n-1)}, ..., b_{n-1}) of Algorithm 1

The five workloads are the paper's synthetic long-sequence benchmark shape
(one head of size 64, Section 3.2 speed study) scaled to several batch /
head / length / feature-count settings, plus a BERT-base-shaped layer
(12 heads of size 64, sequence 512, Appendix A.1).  No dataset is used.
"""
from __future__ import annotations

import dataclasses
import numpy as np

__all__ = ["Workload", "WORKLOADS", "make", "bf16_round", "bf16_bits",
           "gaussian_features", "orthogonal_features"]


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic workload: shapes, dtypes and the value distributions."""

    wid: int
    name: str
    B: int
    H: int
    n: int
    d: int
    m: int
    qkv_dtype: str        # "f32" or "bf16" (q, k, v only; W, b and z stay fp32)
    features: str         # "gaussian" | "orthogonal"
    bias: str             # "normal" | "decay" | "causal"
    bias_sigma: float
    causal: bool

    @property
    def tokens(self) -> int:
        return self.B * self.n


WORKLOADS = {
    1: Workload(1, "tiny-n128", 1, 1, 128, 64, 64, "f32", "gaussian", "normal", 0.5, False),
    2: Workload(2, "bert-base-n512", 16, 12, 512, 64, 64, "f32", "orthogonal", "normal", 0.5, False),
    3: Workload(3, "long-classifier-n2048", 32, 8, 2048, 64, 128, "bf16", "orthogonal", "decay", 0.3, False),
    4: Workload(4, "long-n4096", 8, 12, 4096, 64, 128, "f32", "gaussian", "normal", 1.0, False),
    5: Workload(5, "causal-n16384", 1, 16, 16384, 64, 256, "bf16", "orthogonal", "causal", 0.5, True),
    # Beyond one transform block: the paper's speed test (one head, d = 64,
    # synthetic sequences up to 40k tokens; Sec. 3.2) and the causal shape of
    # workload 5 at four times its length.
    6: Workload(6, "speed-h1-n40000", 1, 1, 40000, 64, 128, "f32", "gaussian", "normal", 0.5, False),
    7: Workload(7, "causal-n65536", 1, 16, 65536, 64, 256, "bf16", "orthogonal", "causal", 0.5, True),
}


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to the nearest bfloat16 (ties to even); return fp32.

    Works on the IEEE-754 bit pattern: keep the top 16 bits after adding the
    round-to-nearest-even increment.  Inputs here are finite.
    """
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32)


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """The uint16 bfloat16 encodings of values that are already bf16-exact."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    if np.any(u & 0xFFFF):
        raise ValueError("values are not bfloat16-representable; call bf16_round first")
    return (u >> 16).astype(np.uint16)


def gaussian_features(rng: np.random.Generator, m: int, d: int) -> np.ndarray:
    """i.i.d. w_l ~ N(0, I_d), as stated under Eq. (5)."""
    return rng.standard_normal((m, d))


def orthogonal_features(rng: np.random.Generator, m: int, d: int) -> np.ndarray:
    """Orthogonal random features (the ORF variant of the ablation, Section 4.5).

    Rows come in blocks of d mutually orthogonal directions, each block the Q
    factor of a Gaussian d x d matrix (sign-fixed so that it is Haar
    distributed), and every row is rescaled to an independent chi_d norm so
    that its length is distributed like that of a Gaussian vector.
    """
    blocks = []
    for _ in range((m + d - 1) // d):
        g = rng.standard_normal((d, d))
        qm, r = np.linalg.qr(g)
        qm = qm * np.sign(np.diag(r))[None, :]
        blocks.append(qm.T)
    w = np.concatenate(blocks, axis=0)[:m]
    norms = np.sqrt(rng.chisquare(d, size=m))
    return w * norms[:, None]


def sphere_features(rng: np.random.Generator, m: int, d: int) -> np.ndarray:
    """Sphere-PRF rows (the appendix comparison of feature maps): i.i.d. uniform on the
    sphere of radius sqrt(d), drawn as normalised Gaussian vectors."""
    g = rng.standard_normal((m, d))
    return g / np.linalg.norm(g, axis=1, keepdims=True) * np.sqrt(d)


_FEATURE_DRAWS = {"gaussian": gaussian_features, "orthogonal": orthogonal_features, "sphere": sphere_features}


def _bias(rng: np.random.Generator, wl: Workload) -> np.ndarray:
    n = wl.n
    t = np.arange(-(n - 1), n, dtype=np.float64)
    eps = rng.standard_normal(2 * n - 1) * wl.bias_sigma
    if wl.bias == "normal":
        return eps
    if wl.bias == "decay":
        return -0.01 * np.abs(t) + eps
    if wl.bias == "causal":
        out = eps.copy()
        out[t > 0] = -np.inf
        return out
    raise ValueError(wl.bias)


def make(wid: int | Workload, seed: int | None = None, *, heads: int | None = None) -> dict:
    """Draw one workload's inputs.

    The generator is ``default_rng([2106, 12566, wid])`` (or ``[.., seed]``
    when a seed is given) and the draw order is q, k, v, then W per head,
    then b per head.  q, k, v ~ N(0, 1) * d^(-1/4); for bf16 workloads they
    are rounded to bfloat16 (the returned fp32 arrays hold the exact bf16
    values).  ``heads`` overrides H (used to build smaller parity cases with
    the same distributions).
    """
    wl = WORKLOADS[wid] if isinstance(wid, int) else wid
    H = wl.H if heads is None else heads
    key = [2106, 12566, wl.wid] if seed is None else [2106, 12566, wl.wid, seed]
    rng = np.random.default_rng(key)
    shape = (wl.B, H, wl.n, wl.d)
    scale = wl.d ** -0.25
    q = (rng.standard_normal(shape) * scale).astype(np.float32)
    k = (rng.standard_normal(shape) * scale).astype(np.float32)
    v = (rng.standard_normal(shape) * scale).astype(np.float32)
    if wl.qkv_dtype == "bf16":
        q, k, v = bf16_round(q), bf16_round(k), bf16_round(v)
    feat = _FEATURE_DRAWS[wl.features]
    W = np.stack([feat(rng, wl.m, wl.d) for _ in range(H)]).astype(np.float32)
    b = np.stack([_bias(rng, wl) for _ in range(H)]).astype(np.float32)
    return {"q": q, "k": k, "v": v, "W": W, "b": b, "workload": wl, "H": H}


def custom(B: int, H: int, n: int, d: int, m: int, *, seed: int = 0,
           qkv_dtype: str = "f32", features: str = "gaussian", bias: str = "normal",
           bias_sigma: float = 0.5, qk_scale: float | None = None) -> dict:
    """Inputs with arbitrary shapes and the same distributions (for edge cases).

    features: how the rows of W are drawn, "gaussian", "orthogonal" or "sphere"."""
    wl = Workload(0, f"custom-{B}x{H}x{n}x{d}x{m}", B, H, n, d, m, qkv_dtype,
                  features, bias, bias_sigma, bias == "causal")
    rng = np.random.default_rng([2106, 12566, 0, seed])
    scale = d ** -0.25 if qk_scale is None else qk_scale
    shape = (B, H, n, d)
    q = (rng.standard_normal(shape) * scale).astype(np.float32)
    k = (rng.standard_normal(shape) * scale).astype(np.float32)
    v = (rng.standard_normal(shape) * d ** -0.25).astype(np.float32)
    if qkv_dtype == "bf16":
        q, k, v = bf16_round(q), bf16_round(k), bf16_round(v)
    feat = _FEATURE_DRAWS[features]
    W = np.stack([feat(rng, m, d) for _ in range(H)]).astype(np.float32)
    b = np.stack([_bias(rng, wl) for _ in range(H)]).astype(np.float32)
    return {"q": q, "k": k, "v": v, "W": W, "b": b, "workload": wl, "H": H}
