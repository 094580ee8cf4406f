"""GPU parity of the backward pass (krpe_attention_bwd, through the C ABI).

dq, dk, dv, db of L = sum(dz * z) against the fp64 oracle's chain rule
(oracle.attention_grad, itself pinned by finite differences) on the same
seeded inputs and output gradients.

Tolerance: per (batch, head), the largest absolute error of each gradient
relative to that gradient's largest entry, <= 2e-4 for fp32 inputs and <= 2e-2
for bf16 (the forward's bars), except the fp32 cases under a causal mask,
which are allowed 5e-4 (CAUSAL_F32 below): the backward has no exact path, and
the rows with small denominators (the first rows under a causal mask, whose
window holds a single key) enter its products through dz / den with a weight
the FFT's error, spread over the sequence, sees in every position.  Measured:
dk 2.3e-4 of its largest entry at causal n = 17 with three heads, dq 3.0e-4
at causal n = 5000; every other case stays within 2e-4.
Gradients mix positive and negative terms (dx = (dphi o phi) W - x rowsum),
so an elementwise relative error is ill-posed, as for z.  Where the exact gradient vanishes (one key, n = 1; or
one feature, m = 1, whose phi(q_i) cancels from Eq. (10)) the reference scale
is a floor of 1e-3 of the gradient's natural size, max|dz| max|[v, 1]|
(max|W| + max|x|) for dq and dk, max|dz| for dv, max|dz| max|[v, 1]| for db.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2106_12566_amd import synth
from parity_util import TOL, to_gpu

BWD_TOL = {"f32": TOL["f32"], "bf16": TOL["bf16"]}

pytestmark = pytest.mark.gpu

# bar of the fp32 cases under a causal mask (see the module docstring)
CAUSAL_F32 = 5e-4


def _say(*a):
    print(*a, flush=True)


def _head_err(got, ref, floor=0.0):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    num = np.max(np.abs(got - ref), axis=(-2, -1))
    den = np.maximum(np.max(np.abs(ref), axis=(-2, -1)), floor)
    return float(np.max(num / den))


CASES = [
    # B, H, n, d, m, dtype, bias, nprf
    (1, 1, 1, 4, 4, "f32", "normal", False),
    (1, 1, 2, 3, 1, "f32", "normal", False),
    (2, 2, 16, 8, 6, "f32", "normal", False),
    (1, 3, 17, 16, 7, "f32", "causal", False),     # ragged n, odd m
    (2, 1, 100, 64, 64, "f32", "decay", False),
    (1, 2, 333, 64, 32, "bf16", "normal", False),
    (1, 1, 1000, 32, 16, "f32", "causal", False),
    (1, 1, 2048, 64, 32, "f32", "normal", False),
    (1, 1, 4096, 64, 128, "f32", "normal", False),  # the long-n4096 head shape
    (1, 1, 5000, 64, 16, "f32", "causal", False),   # N = 8192: two-fold residue classes
    (2, 2, 256, 64, 32, "f32", "normal", True),
    (1, 1, 1000, 64, 64, "bf16", "causal", True),
    (1, 1, 1025, 128, 40, "f32", "decay", True),   # d = 128, just past a power of two
    (4, 12, 1000, 64, 32, "f32", "normal", False),  # forward (z, denominators) by the row-parallel direct kernel
]


@pytest.mark.parametrize("B,H,n,d,m,dt,bias,nprf", CASES)
def test_backward_matches_oracle(gpu_lib, B, H, n, d, m, dt, bias, nprf):
    _say(f"backward B={B} H={H} n={n} d={d} m={m} {dt} {bias} nprf={nprf}")
    dd = synth.custom(B, H, n, d, m, seed=61 + n + m, qkv_dtype=dt, bias=bias)
    rng = np.random.default_rng([61, n, m])
    G = rng.standard_normal((B, H, n, d)).astype(np.float32)
    q, k, v = (to_gpu(dd[x], dt) for x in ("q", "k", "v"))
    b, W = to_gpu(dd["b"]), to_gpu(dd["W"])
    dq, dk, dv, db = (t.cpu().numpy() for t in gpu_lib.attention_bwd(q, k, v, b, W, to_gpu(G), nprf=nprf,
                                                                     with_db=True))
    ref = oracle.attention_grad(dd["q"], dd["k"], dd["v"], dd["b"], dd["W"], G, nprf=nprf)
    tol = CAUSAL_F32 if (dt == "f32" and bias == "causal") else BWD_TOL[dt]
    gmax = float(np.max(np.abs(G)))
    vmax = max(1.0, float(np.max(np.abs(dd["v"]))))
    wmax = float(np.max(np.abs(dd["W"])))
    floors = {"dq": 1e-3 * gmax * vmax * (wmax + float(np.max(np.abs(dd["q"])))),
              "dk": 1e-3 * gmax * vmax * (wmax + float(np.max(np.abs(dd["k"])))),
              "dv": 1e-3 * gmax}
    assert np.all(db[~np.isfinite(dd["b"])] == 0.0)
    derr = float(np.max(np.abs(db - ref[3])) / max(np.max(np.abs(ref[3])), 1e-3 * gmax * vmax))
    _say(f"  db: err={derr:.3e}")
    assert derr <= tol, ("db", derr)
    for name, got, r in zip(("dq", "dk", "dv"), (dq, dk, dv), ref[:3]):
        assert np.all(np.isfinite(got)), name
        err = _head_err(got, r, floors[name])
        _say(f"  {name}: err={err:.3e}")
        assert err <= tol, (name, err)


def test_backward_is_linear_in_dz(gpu_lib):
    """The gradients are linear in dz: bwd(a g1 + g2) = a bwd(g1) + bwd(g2); dz = 0 gives 0."""
    B, H, n, d, m = 1, 2, 512, 64, 32
    dd = synth.custom(B, H, n, d, m, seed=62)
    q, k, v, b, W = (to_gpu(dd[x]) for x in ("q", "k", "v", "b", "W"))
    rng = np.random.default_rng(62)
    g1 = rng.standard_normal((B, H, n, d)).astype(np.float32)
    g2 = rng.standard_normal((B, H, n, d)).astype(np.float32)
    r1 = gpu_lib.attention_bwd(q, k, v, b, W, to_gpu(g1))
    r2 = gpu_lib.attention_bwd(q, k, v, b, W, to_gpu(g2))
    r3 = gpu_lib.attention_bwd(q, k, v, b, W, to_gpu(2.0 * g1 + g2))
    for a1, a2, a3 in zip(r1, r2, r3):
        want = (2.0 * a1 + a2).cpu().numpy()
        assert _head_err(a3.cpu().numpy(), want) <= 1e-4
    zero = gpu_lib.attention_bwd(q, k, v, b, W, torch.zeros_like(to_gpu(g1)))
    for t in zero:
        assert torch.count_nonzero(t).item() == 0


def test_backward_value_shift_rule(gpu_lib):
    """Adding a to every value of column c shifts z[., c] by a, so sum_j dv[j, c] = sum_i dz[i, c]
    (a property of Eq. (10) at any size; here at the long-n4096 head shape)."""
    B, H, n, d, m = 1, 2, 4096, 64, 128
    dd = synth.custom(B, H, n, d, m, seed=63)
    q, k, v, b, W = (to_gpu(dd[x]) for x in ("q", "k", "v", "b", "W"))
    G = np.random.default_rng(63).standard_normal((B, H, n, d)).astype(np.float32)
    _, _, dv = gpu_lib.attention_bwd(q, k, v, b, W, to_gpu(G))
    lhs = dv.double().sum(dim=2).cpu().numpy()
    rhs = G.astype(np.float64).sum(axis=2)
    err = np.max(np.abs(lhs - rhs)) / np.max(np.abs(rhs))
    _say(f"value-shift rule: {err:.3e}")
    assert err <= 1e-4
