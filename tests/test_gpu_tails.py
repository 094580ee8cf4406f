"""GPU parity at ragged sizes with poisoned surroundings.

Sizes whose tails do not fill the kernels' tiles:
* the sequence length is not a multiple of the 32-key blocks of the exact-row
  kernel;
* the feature count is not a multiple of its 64-feature steps, odd included;
* the sequence is shorter than the 128-key chunks;
* d is not a multiple of the 32-column tiles;
* at n = 2000 and 4000 the convolutions load phi a feature ahead;
* d = 128, 100 and 2: value columns in two groups of 64, a partial last
  group, and a count the 4-column loads of the value preparation do not take;
* d = 1 and 65: the gram kernel's last pair tile holds a single pair;
* the same tails on the direct route's row-parallel kernel (enough heads for
  it to be taken).

Every input sits at the start of an allocation whose remainder is NaN, and
the workspace and the output are NaN before the call.  Any value read past
the end of a tensor, or from workspace memory no kernel wrote, would reach z
(NaN times a masked zero is still NaN); every row of z must be finite and
match Eq. (10) evaluated directly by the fp64 oracle.  Tolerances are stated
in tests/parity_util.py.
"""
import numpy as np
import pytest

import oracle
from paper_2106_12566_amd import synth
from parity_util import TOL, rownorm_err, to_gpu

pytestmark = pytest.mark.gpu

PAD_BYTES = 1 << 20


def _say(*a):
    print(*a, flush=True)


def _poisoned(t):
    """A copy of t at the start of a larger allocation whose remainder is NaN."""
    import torch
    pad = PAD_BYTES // t.element_size()
    flat = torch.full((t.numel() + pad,), float("nan"), dtype=t.dtype, device=t.device)
    flat[: t.numel()].copy_(t.reshape(-1))
    return flat[: t.numel()].view(t.shape)


# (B, H, n, d, m, dtype, route, bias)
CASES = [
    (1, 2, 333, 48, 33, "f32", "direct", "normal"),
    (1, 2, 333, 64, 64, "bf16", "direct", "causal"),
    (1, 3, 50, 16, 5, "f32", "direct", "normal"),
    (1, 2, 97, 32, 1, "f32", "fft", "normal"),
    (2, 2, 2000, 64, 33, "f32", "fft", "causal"),
    (1, 2, 4000, 64, 96, "bf16", "fft", "normal"),
    # value columns in two groups of 64 (the ones column's pair on its own),
    # a partial last group, and a column count the quad loads do not take
    (1, 2, 300, 128, 64, "bf16", "fft", "normal"),
    (1, 2, 1000, 100, 64, "f32", "fft", "causal"),
    (1, 2, 513, 2, 8, "f32", "fft", "normal"),
    # one value pair in the last pair tile of the gram kernel: d = 1 (the
    # pair [v, 1] alone) and d = 65 (the 33rd pair [v_64, 1])
    (1, 2, 200, 1, 16, "f32", "fft", "normal"),
    (1, 2, 700, 65, 40, "bf16", "fft", "causal"),
    # the direct route's row-parallel kernel (m <= 128 and at least 1536 waves
    # of 32 rows): a feature count that is not a multiple of 64, value columns
    # in two passes, a last row tile whose last waves start past n, causal
    # key ranges; a partial last key block with bf16 values and d = 2; a
    # sequence one past a multiple of 32 with d = 128
    (4, 16, 900, 100, 33, "f32", "direct", "causal"),
    (2, 24, 1000, 2, 64, "bf16", "direct", "normal"),
    (3, 16, 1025, 128, 128, "f32", "direct", "normal"),
]


@pytest.mark.parametrize("B,H,n,d,m,dt,route,bias", CASES)
def test_ragged_tails_read_nothing_outside(gpu_lib, B, H, n, d, m, dt, route, bias):
    import torch
    _say(f"ragged B={B} H={H} n={n} d={d} m={m} {dt} route={route} bias={bias}")
    dd = synth.custom(B, H, n, d, m, seed=91 + n + m, qkv_dtype=dt, bias=bias)
    q, k, v = (_poisoned(to_gpu(dd[x], dt)) for x in ("q", "k", "v"))
    b, W = _poisoned(to_gpu(dd["b"])), _poisoned(to_gpu(dd["W"]))
    ws = torch.full((gpu_lib.attention_fwd_workspace(B, H, n, d, m, route=route),), 0xFF, dtype=torch.uint8,
                    device="cuda")
    out = torch.full((B, H, n, d), float("nan"), dtype=torch.float32, device="cuda")
    z = gpu_lib.attention_fwd(q, k, v, b, W, out=out, workspace=ws, route=route).cpu().numpy()
    fixed = gpu_lib.attention_fwd_fixed_rows(ws, B, H, n, d, m)
    bad = np.argwhere(~np.isfinite(z))
    assert bad.size == 0, f"non-finite z at {bad[:4].tolist()} ({len(bad)} entries)"
    ref, den = oracle.attention(dd["q"], dd["k"], dd["v"], dd["b"], dd["W"])
    assert np.all(den > 0)
    err = rownorm_err(z, ref)
    _say(f"  every row: max err {err:.3e}; rows evaluated exactly: {fixed}")
    assert err <= TOL[dt], err
