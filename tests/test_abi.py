"""C-ABI checks that need no GPU.

* libkrpe.so loads and exports every function that include/krpe.h declares.
* Argument validation: every error code is produced on the host, before any
  HIP call, from invalid arguments.  The pointers passed are never
  dereferenced: each call below is rejected by validation, which is exactly
  what is being tested, so no kernel is launched and no device is touched.
"""
import ctypes
import os
import re

import pytest

from paper_2106_12566_amd import krpe

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "krpe.h")

OK, NULL, SHAPE, UNSUP, DTYPE, WS, ALIAS, HIP, ALIGN = range(9)


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(krpe.lib_path()):
        from paper_2106_12566_amd import build
        build.build()
    return krpe.load()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(krpe_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for required in ("krpe_feature_map", "krpe_toeplitz_conv", "krpe_attention_fwd",
                     "krpe_toeplitz_conv_workspace", "krpe_attention_fwd_workspace",
                     "krpe_attention_fwd_profiled", "krpe_status_str", "krpe_last_error",
                     "krpe_abi_version", "krpe_feature_map_ex", "krpe_attention_fwd_ex",
                     "krpe_attention_fwd_workspace_ex", "krpe_attention_bwd", "krpe_attention_bwd_workspace",
                     "krpe_attention_fwd_route"):
        assert required in names


def test_library_exports_every_declared_symbol(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_version_and_status_strings(lib):
    assert lib.krpe_abi_version() == 6
    for s in range(9):
        assert lib.krpe_status_str(s)
    assert lib.krpe_status_str(99) == b"unknown status"


# Fake, 16-byte aligned, non-overlapping device addresses: only ever seen by
# the validation code, which rejects every call in this file.
BASE = 1 << 40
Q, K, V, BB, W, Z, WSP = (BASE + i * (1 << 36) for i in range(7))


def attn(lib, q=Q, k=K, v=V, dt=0, b=BB, w=W, z=Z, B=1, H=1, n=8, d=4, m=4, ws=WSP, wsb=None):
    if wsb is None:
        wsb = lib.krpe_attention_fwd_workspace(B, H, n, d, m) if n >= 1 else 0
    return lib.krpe_attention_fwd(q, k, v, dt, b, w, z, B, H, n, d, m, ws, wsb, None)


def test_workspace_queries(lib):
    small = lib.krpe_attention_fwd_workspace(1, 1, 8, 4, 4)
    big = lib.krpe_attention_fwd_workspace(2, 3, 100, 64, 64)
    assert 0 < small < big
    assert lib.krpe_attention_fwd_workspace(1, 1, 0, 4, 4) == 0
    assert lib.krpe_attention_fwd_workspace(1, 1, 65537, 4, 4) == 0
    # beyond one transform block (n > 16384) the FFT route's blocked layout
    # holds phi over the whole sequence and per 16384-position block
    fft_long = lib.krpe_attention_fwd_workspace_ex(1, 2, 40000, 64, 64, 16)
    assert fft_long >= 2 * 2 * 64 * 49152 * 4 * 2
    assert lib.krpe_attention_fwd_workspace_ex(1, 2, 40000, 64, 64, 8) > 0
    assert lib.krpe_attention_fwd_workspace_ex(1, 1, 65536, 64, 64, 0) > 0
    # the backward stays within one block; the plain Toeplitz product goes to 65536 in blocks
    assert lib.krpe_attention_bwd_workspace(1, 1, 16385, 4, 4, 0) == 0
    assert lib.krpe_toeplitz_conv_workspace(1, 1, 1, 16385) > lib.krpe_toeplitz_conv_workspace(1, 1, 1, 16384) > 0
    assert lib.krpe_toeplitz_conv_workspace(1, 1, 1, 65536) > 0 and lib.krpe_toeplitz_conv_workspace(1, 1, 1, 65537) == 0
    assert lib.krpe_attention_fwd_workspace(1, 1, 8, 129, 4) == 0
    assert lib.krpe_toeplitz_conv_workspace(1, 2, 3, 100) > 0
    assert lib.krpe_toeplitz_conv_workspace(1, 2, 3, 0) == 0
    assert lib.krpe_toeplitz_conv_workspace(2, 2, 3, 100) > lib.krpe_toeplitz_conv_workspace(1, 2, 3, 100)
    # workspace covers phi(q), phi(k) in fp32 at least
    assert lib.krpe_attention_fwd_workspace(8, 12, 4096, 64, 128) >= 2 * 8 * 12 * 4096 * 128 * 4
    # ... plus one row of slack after each: the convolution's look-ahead load
    # reads one row past the last head's rows (never used)
    assert lib.krpe_attention_fwd_workspace(8, 12, 4096, 64, 128) >= 2 * (8 * 12 * 128 + 1) * 4096 * 4


def test_attention_validation(lib):
    assert attn(lib, q=None) == NULL
    assert attn(lib, z=None) == NULL
    assert attn(lib, n=0) == SHAPE
    assert attn(lib, B=-1) == SHAPE
    assert attn(lib, n=65537) == UNSUP
    assert attn(lib, d=129) == UNSUP
    assert attn(lib, m=1025) == UNSUP
    assert attn(lib, m=0) == SHAPE
    assert attn(lib, dt=7) == DTYPE
    assert attn(lib, q=Q + 4) == ALIGN
    assert attn(lib, ws=None) == WS
    assert attn(lib, wsb=16) == WS
    assert attn(lib, z=Q) == ALIAS                     # output on top of an input
    assert attn(lib, ws=V + 64) == ALIAS               # workspace overlapping v
    assert b"workspace" in lib.krpe_last_error() or lib.krpe_last_error() != b""
    # empty batch: valid, nothing to do (returns before any HIP call)
    assert attn(lib, B=0, q=None, k=None, v=None, z=None) == OK
    assert lib.krpe_last_error() == b""


def test_option_bits_validation(lib):
    wsb = lib.krpe_attention_fwd_workspace(1, 1, 8, 4, 4)
    ex = lambda flags: lib.krpe_attention_fwd_ex(Q, K, V, 0, BB, W, Z, 1, 1, 8, 4, 4, flags, WSP, wsb, None)
    assert ex(64) == UNSUP                   # unknown option bit
    assert ex(1 | 64) == UNSUP
    assert ex(8 | 16) == UNSUP               # both routes
    assert ex(2 | 4) == UNSUP                # TRF and elu + 1 together
    # elu + 1 needs m == d (here d = 4, m = 3); TRF doubles the features (2m <= 1024)
    assert lib.krpe_attention_fwd_ex(Q, K, V, 0, BB, W, Z, 1, 1, 8, 4, 3, 4, WSP, wsb, None) == SHAPE
    assert lib.krpe_attention_fwd_ex(Q, K, V, 0, BB, W, Z, 1, 1, 8, 4, 600, 2, WSP, wsb, None) == UNSUP
    assert lib.krpe_attention_fwd_ex(Q, K, V, 0, BB, None, Z, 1, 1, 8, 4, 4, 2, WSP, wsb, None) == NULL
    assert lib.krpe_attention_fwd_ex(None, K, V, 0, BB, None, Z, 1, 1, 8, 4, 4, 4, WSP, wsb, None) == NULL
    wse = lambda flags, m=4: lib.krpe_attention_fwd_workspace_ex(2, 3, 100, 4, m, flags)
    assert wse(0) == lib.krpe_attention_fwd_workspace(2, 3, 100, 4, 4)
    assert wse(1) == wse(0)                  # normalisation needs no space
    assert wse(2) > wse(0)                   # 2m trigonometric features
    assert wse(4) == wse(0)                  # elu + 1: M = d = m
    assert wse(4, m=3) == 0 and wse(6) == 0 and wse(64) == 0 and wse(24) == 0
    assert wse(32) == wse(0)                 # the causal hint needs no space
    assert wse(8) == wse(0) and wse(16) == wse(0)   # one workspace serves both routes
    assert wse(2, m=513) == 0
    assert lib.krpe_attention_fwd_ex(None, K, V, 0, BB, W, Z, 1, 1, 8, 4, 4, 1, WSP, wsb, None) == NULL
    assert lib.krpe_attention_fwd_ex(Q, K, V, 0, BB, W, Z, 1, 1, 8, 4, 4, 1, None, wsb, None) == WS
    fm = lambda flags: lib.krpe_feature_map_ex(Q, 0, W, Z, 1, 1, 8, 4, 4, flags, None)
    assert fm(64) == UNSUP
    assert fm(6) == UNSUP
    assert lib.krpe_feature_map_ex(Q, 0, W, Z, 1, 1, 8, 4, 3, 4, None) == SHAPE
    assert lib.krpe_feature_map_ex(Q, 0, None, Z, 1, 1, 8, 4, 4, 2, None) == NULL
    assert lib.krpe_feature_map_ex(None, 0, W, Z, 1, 1, 8, 4, 4, 1, None) == NULL


def test_toeplitz_validation(lib):
    ws = lib.krpe_toeplitz_conv_workspace(1, 2, 3, 10)
    call = lambda b=BB, a=Q, y=Z, B=1, H=2, C=3, n=10, w=WSP, wb=ws: lib.krpe_toeplitz_conv(
        b, a, y, B, H, C, n, w, wb, None)
    assert call(a=None) == NULL
    assert call(n=0) == SHAPE
    assert call(C=-1) == SHAPE
    assert call(n=65537) == UNSUP
    assert call(n=20000) == WS               # a valid length whose workspace is larger
    assert call(wb=8) == WS
    assert call(y=Q) == ALIAS
    assert call(y=Z + 8) == ALIGN
    assert call(C=0, a=None, y=None) == OK


def test_toeplitz_noalloc_refuses_sizes_beyond_the_scratch(lib):
    """The no-allocation entry point refuses, on the host and before any HIP call, sizes whose
    workspace exceeds its static scratch (64 MiB), and validates sizes like krpe_toeplitz_conv."""
    big = (64, 4, 64, 16384)
    assert lib.krpe_toeplitz_conv_workspace(*big) > (64 << 20)
    assert lib.krpe_toeplitz_conv_noalloc(None, None, None, *big, None) == UNSUP
    assert b"static scratch" in lib.krpe_last_error()
    assert lib.krpe_toeplitz_conv_noalloc(None, None, None, 1, 1, -1, 10, None) == SHAPE
    assert lib.krpe_toeplitz_conv_noalloc(None, None, None, 1, 1, 2, 65537, None) == UNSUP
    assert lib.krpe_toeplitz_conv_noalloc(None, None, None, 1, 1, 0, 10, None) == OK


def test_feature_map_validation(lib):
    call = lambda x=Q, dt=0, w=W, phi=Z, B=1, H=1, n=8, d=4, m=4: lib.krpe_feature_map(
        x, dt, w, phi, B, H, n, d, m, None)
    assert call(x=None) == NULL
    assert call(dt=2) == DTYPE
    assert call(d=0) == SHAPE
    assert call(m=2000) == UNSUP
    assert call(phi=Q) == ALIAS
    assert call(H=0, x=None, w=None, phi=None) == OK


def test_binding_refuses_cpu_tensors(lib):
    import torch
    x = torch.zeros(1, 1, 8, 4)
    W = torch.zeros(1, 4, 4)
    with pytest.raises(krpe.KrpeError):
        krpe.feature_map(x, W)
    with pytest.raises(krpe.KrpeError):
        krpe.attention_fwd(x, x, x, torch.zeros(1, 15), W)


def test_backward_validation(lib):
    """Argument checks of the backward entry point (all fail before any GPU call)."""
    wsb = lib.krpe_attention_bwd_workspace(1, 1, 8, 4, 4, 0)
    assert wsb > lib.krpe_attention_fwd_workspace(1, 1, 8, 4, 4)
    assert lib.krpe_attention_bwd_workspace(1, 1, 8, 4, 4, 2) == 0      # TRF has no backward here
    assert lib.krpe_attention_bwd_workspace(1, 1, 8, 4, 4, 1) == wsb
    D1, D2, D3 = Z + 4096, Z + 8192, Z + 12288
    call = lambda flags=0, db=None, dq=D1, dz=Q, w=WSP, wb=wsb, n=8: lib.krpe_attention_bwd(
        Q, K, V, 0, BB, W, dz, dq, D2, D3, db, 1, 1, n, 4, 4, flags, w, wb, None)
    assert call(flags=2) == UNSUP
    assert call(flags=64) == UNSUP
    assert call(flags=8 | 16) == UNSUP
    assert call(db=D1) == ALIAS               # db overlapping dq
    assert call(db=Z + 20000 + 4) == ALIGN
    assert call(dz=None) == NULL
    assert call(n=0) == SHAPE
    assert call(wb=8) == WS
    assert call(dq=Q) == ALIAS
    assert call(dq=D2) == ALIAS
    assert call(dq=D1 + 8) == ALIGN


def test_route_query(lib):
    """Route choice: forced by the option bits, else the cost model (direct for short sequences)."""
    route = lib.krpe_attention_fwd_route
    assert route(8, 12, 4096, 64, 128, 8) == 8 and route(8, 12, 128, 64, 64, 16) == 16
    assert route(8, 12, 128, 64, 64, 0) == 8            # short: direct
    assert route(8, 12, 512, 64, 64, 0) == 8
    assert route(8, 12, 4096, 64, 128, 0) == 8          # the long-n4096 layer: direct at 96 heads
    assert route(1, 2, 16384, 64, 128, 0) == 16
    assert route(1, 16, 16384, 64, 256, 0) == 16
    assert route(1, 1, 1000, 64, 64, 0) == 8            # one head: the FFT route's fixed cost dominates
    # past one transform block the FFT route wins by a wide margin (model: 10.5 against 5.3 ms at
    # one head, n = 65536, m = 64)
    assert route(1, 1, 65536, 64, 64, 0) == 16 and route(1, 16, 65536, 64, 256, 0) == 16
    assert route(1, 1, 65536, 64, 128, 8) == 8          # forced, past one transform block
    assert route(1, 1, 65537, 64, 64, 0) == 0 and route(0, 1, 8, 4, 4, 0) == 0
    assert route(1, 1, 8, 4, 4, 8 | 16) == 0 and route(1, 1, 0, 4, 4, 0) == 0 and route(1, 1, 8, 4, 3, 4) == 0
    # a stated causal mask halves the direct route's pairs: the causal-n16384 layer goes direct,
    # the causal-n65536 one stays on the FFT route; a route bit still wins over the hint
    assert route(1, 16, 16384, 64, 256, 32) == 8 and route(1, 16, 65536, 64, 256, 32) == 16
    assert route(1, 16, 16384, 64, 256, 32 | 16) == 16 and route(8, 12, 4096, 64, 128, 32) == 8
    assert route(1, 2, 16384, 64, 128, 32) == 8
