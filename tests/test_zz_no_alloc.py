"""The no-allocation entry point krpe_toeplitz_conv_noalloc (static scratch, no workspace argument).

Checked through the C ABI against krpe_toeplitz_conv on the same inputs (the two share every
kernel, so the outputs must agree bit for bit) and against the fp64 oracle's direct product at
the Toeplitz bar (per-channel normwise error <= 2e-4, tests/parity_util.py), on two calls in a
row whose second is smaller: the scratch keeps the first call's contents, and the second call
must not read them.  (Sizes beyond the scratch are refused on the host: tests/test_abi.py.)
"""
import numpy as np
import pytest
import torch

import oracle
from parity_util import rownorm_err, to_gpu

pytestmark = pytest.mark.gpu

SCRATCH_BYTES = 64 << 20


def _case(B, H, C, n, seed):
    rng = np.random.default_rng([91, seed])
    b = (rng.standard_normal((H, 2 * n - 1)) * 0.7).astype(np.float32)
    a = rng.standard_normal((B, H, C, n)).astype(np.float32)
    return b, a


@pytest.mark.parametrize("first,second", [((2, 3, 5, 1000), (1, 2, 3, 300)),      # ragged n, then smaller
                                          ((1, 4, 8, 4096), (1, 1, 2, 17))])      # multi-pass, then tiny
def test_noalloc_matches_workspace_entry_point(gpu_lib, first, second):
    for shape, seed in ((first, 1), (second, 2)):
        B, H, C, n = shape
        print(f"noalloc toeplitz B={B} H={H} C={C} n={n}", flush=True)
        assert gpu_lib.toeplitz_conv_workspace(B, H, C, n) <= SCRATCH_BYTES
        b, a = _case(B, H, C, n, seed)
        bg, ag = to_gpu(b), to_gpu(a)
        y0 = gpu_lib.toeplitz_conv_noalloc(bg, ag)
        y1 = gpu_lib.toeplitz_conv(bg, ag)
        torch.cuda.synchronize()
        assert torch.equal(y0, y1)
        err = rownorm_err(y0.cpu().numpy(), oracle.toeplitz_product(b, a))
        print(f"  err={err:.3e}", flush=True)
        assert err <= 2e-4, err
