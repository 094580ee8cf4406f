"""Python binding of libkrpe.so: argument marshalling only.

Every function takes torch tensors that live on a GPU, checks that their shapes
agree with each other, allocates the output (and workspace) with torch, and
calls the C entry point of the same name on the current torch stream.  All
arithmetic happens in the library's HIP kernels; there is no CPU path: calling
any of these without the built library or without a GPU raises.

Names and layouts follow the C header ``include/krpe.h``:
  q, k, v : [B, H, n, d]  float32 or bfloat16      W : [H, m, d] float32
  b       : [H, 2n-1] float32, b[h, s] = b_{s-(n-1)} (Algorithm 1's ordering)
"""
from __future__ import annotations

import ctypes
import os

import torch

__all__ = ["KrpeError", "load", "lib_path", "feature_map", "toeplitz_conv", "toeplitz_conv_noalloc",
           "attention_fwd", "attention_bwd",
           "attention_fwd_route",
           "attention_fwd_workspace", "attention_bwd_workspace", "toeplitz_conv_workspace",
           "attention_fwd_fixed_rows", "DTYPES"]

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libkrpe.so")
_lib = None

DTYPES = {torch.float32: 0, torch.bfloat16: 1}
STAGE_EVENTS = 5
NPRF = 1  # option bit: l2-normalise the rows of q and k (x) before the feature map
FEAT_TRF = 2  # option bit: trigonometric random features (2m signed features)
FEAT_ELU = 4  # option bit: elu(x) + 1 (d features, W not read)
FEATURES = {"prf": 0, "trf": FEAT_TRF, "elu": FEAT_ELU}
ROUTE_DIRECT = 8  # option bit: evaluate Eq. (10) directly (quadratic, MFMA)
ROUTE_FFT = 16  # option bit: the FFT route of Section 3.2
ROUTES = {"auto": 0, "direct": ROUTE_DIRECT, "fft": ROUTE_FFT}
HINT_CAUSAL = 32  # option bit: b is -inf for every t > 0 (read by the route choice only)


class KrpeError(RuntimeError):
    """A non-OK status returned by the library, or a missing library/GPU."""


def lib_path() -> str:
    """The library this binding loads: $KRPE_LIBRARY if set (e.g. a build with host-side
    sanitizers), else libkrpe.so next to this file."""
    return os.environ.get("KRPE_LIBRARY") or _LIB_PATH


def load(path: str | None = None) -> ctypes.CDLL:
    """Load the library (once).  Raises KrpeError if it has not been built."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or lib_path()
    if not os.path.exists(p):
        raise KrpeError(f"{p} is missing: build it with `python -m paper_2106_12566_amd.build`")
    lib = ctypes.CDLL(p)
    vp, i, sz, fp = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t, ctypes.c_void_p
    lib.krpe_abi_version.restype = i
    lib.krpe_abi_version.argtypes = []
    lib.krpe_status_str.restype = ctypes.c_char_p
    lib.krpe_status_str.argtypes = [i]
    lib.krpe_last_error.restype = ctypes.c_char_p
    lib.krpe_last_error.argtypes = []
    lib.krpe_feature_map.restype = i
    lib.krpe_feature_map.argtypes = [vp, i, fp, fp, i, i, i, i, i, vp]
    lib.krpe_feature_map_ex.restype = i
    lib.krpe_feature_map_ex.argtypes = [vp, i, fp, fp, i, i, i, i, i, ctypes.c_uint, vp]
    lib.krpe_toeplitz_conv_workspace.restype = sz
    lib.krpe_toeplitz_conv_workspace.argtypes = [i, i, i, i]
    lib.krpe_toeplitz_conv.restype = i
    lib.krpe_toeplitz_conv.argtypes = [fp, fp, fp, i, i, i, i, vp, sz, vp]
    lib.krpe_toeplitz_conv_noalloc.restype = i
    lib.krpe_toeplitz_conv_noalloc.argtypes = [fp, fp, fp, i, i, i, i, vp]
    lib.krpe_attention_fwd_workspace.restype = sz
    lib.krpe_attention_fwd_workspace.argtypes = [i, i, i, i, i]
    lib.krpe_attention_fwd_workspace_ex.restype = sz
    lib.krpe_attention_fwd_workspace_ex.argtypes = [i, i, i, i, i, ctypes.c_uint]
    lib.krpe_attention_fwd.restype = i
    lib.krpe_attention_fwd.argtypes = [vp, vp, vp, i, fp, fp, fp, i, i, i, i, i, vp, sz, vp]
    lib.krpe_attention_fwd_ex.restype = i
    lib.krpe_attention_fwd_ex.argtypes = [vp, vp, vp, i, fp, fp, fp, i, i, i, i, i, ctypes.c_uint, vp, sz, vp]
    lib.krpe_attention_fwd_profiled.restype = i
    lib.krpe_attention_fwd_profiled.argtypes = [vp, vp, vp, i, fp, fp, fp, i, i, i, i, i, ctypes.c_uint, vp, sz,
                                                vp, ctypes.POINTER(ctypes.c_void_p)]
    lib.krpe_attention_fwd_route.restype = i
    lib.krpe_attention_fwd_route.argtypes = [i, i, i, i, i, ctypes.c_uint]
    lib.krpe_attention_bwd_workspace.restype = sz
    lib.krpe_attention_bwd_workspace.argtypes = [i, i, i, i, i, ctypes.c_uint]
    lib.krpe_attention_bwd.restype = i
    lib.krpe_attention_bwd.argtypes = [vp, vp, vp, i, fp, fp, fp, fp, fp, fp, fp, i, i, i, i, i, ctypes.c_uint, vp,
                                       sz, vp]
    lib.krpe_attention_fwd_stats.restype = i
    lib.krpe_attention_fwd_stats.argtypes = [vp, sz, i, i, i, i, i, ctypes.POINTER(ctypes.c_uint), vp]
    if path is None:
        _lib = lib
    return lib


def _check(status: int, what: str) -> None:
    if status != 0:
        lib = load()
        msg = lib.krpe_status_str(status).decode()
        detail = lib.krpe_last_error().decode()
        raise KrpeError(f"{what}: {msg} ({detail})")


def _gpu(t: torch.Tensor, name: str) -> torch.Tensor:
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if not t.is_cuda:
        raise KrpeError(f"{name} must be on a GPU (libkrpe has no CPU path)")
    return t.contiguous()


def _ptr(t: torch.Tensor | None) -> int | None:
    return None if t is None or t.numel() == 0 else t.data_ptr()


def _stream(device: torch.device) -> int:
    return torch.cuda.current_stream(device).cuda_stream


def _dtype_code(t: torch.Tensor, name: str) -> int:
    if t.dtype not in DTYPES:
        raise KrpeError(f"{name} must be float32 or bfloat16, got {t.dtype}")
    return DTYPES[t.dtype]


def _flags(nprf: bool, features: str, route: str = "auto", causal: bool = False) -> int:
    if features not in FEATURES:
        raise KrpeError(f"features must be one of {sorted(FEATURES)}, got {features!r}")
    if route not in ROUTES:
        raise KrpeError(f"route must be one of {sorted(ROUTES)}, got {route!r}")
    return (NPRF if nprf else 0) | FEATURES[features] | ROUTES[route] | (HINT_CAUSAL if causal else 0)


def _proj(W: torch.Tensor | None, H: int, d: int, features: str) -> tuple[torch.Tensor | None, int]:
    """W (None allowed for elu + 1) and the m the C call takes."""
    if features == "elu":
        return None, d
    if W is None:
        raise KrpeError("W is required for the prf and trf feature maps")
    W = _gpu(W, "W")
    if W.dim() != 3 or W.shape[0] != H or W.shape[2] != d or W.dtype != torch.float32:
        raise KrpeError("W must be float32 [H, m, d]")
    return W, W.shape[1]


def feature_map(x: torch.Tensor, W: torch.Tensor | None, nprf: bool = False, features: str = "prf") -> torch.Tensor:
    """phi of x [B,H,n,d] -> [B,H,n,M] fp32 with the projections W [H,m,d].

    features: "prf" (Eq. (5), M = m), "trf" (sin then cos features, M = 2m),
    "elu" (elu(x) + 1, M = d, W unused).  nprf: phi of x / ||x|| (Algorithm 1)."""
    lib = load()
    x = _gpu(x, "x")
    if x.dim() != 4:
        raise KrpeError("x must be [B,H,n,d]")
    B, H, n, d = x.shape
    flags = _flags(nprf, features)
    W, m = _proj(W, H, d, features)
    M = 2 * m if features == "trf" else m
    phi = torch.empty((B, H, n, M), dtype=torch.float32, device=x.device)
    st = lib.krpe_feature_map_ex(_ptr(x), _dtype_code(x, "x"), _ptr(W), _ptr(phi), B, H, n, d, m, flags,
                                 _stream(x.device))
    _check(st, "krpe_feature_map_ex")
    return phi


def toeplitz_conv_workspace(B: int, H: int, C: int, n: int) -> int:
    return int(load().krpe_toeplitz_conv_workspace(B, H, C, n))


def toeplitz_conv(b: torch.Tensor, a: torch.Tensor) -> torch.Tensor:
    """y[beta,h,c,i] = sum_j exp(b[h, j-i+n-1]) a[beta,h,c,j]; b [H,2n-1], a [B,H,C,n] fp32."""
    lib = load()
    b = _gpu(b, "b")
    a = _gpu(a, "a")
    if a.dim() != 4 or b.dim() != 2:
        raise KrpeError("a must be [B,H,C,n] and b [H,2n-1]")
    B, H, C, n = a.shape
    if b.shape != (H, 2 * n - 1) or b.dtype != torch.float32 or a.dtype != torch.float32:
        raise KrpeError("b must be float32 [H, 2n-1] and a float32 [B,H,C,n]")
    y = torch.empty_like(a)
    wsb = lib.krpe_toeplitz_conv_workspace(B, H, C, n)
    ws = torch.empty(max(int(wsb), 1), dtype=torch.uint8, device=a.device)
    st = lib.krpe_toeplitz_conv(_ptr(b), _ptr(a), _ptr(y), B, H, C, n, ws.data_ptr(), ws.numel(),
                                _stream(a.device))
    _check(st, "krpe_toeplitz_conv")
    return y


def toeplitz_conv_noalloc(b: torch.Tensor, a: torch.Tensor, out: torch.Tensor | None = None) -> torch.Tensor:
    """toeplitz_conv through krpe_toeplitz_conv_noalloc: no workspace, the library's static scratch instead.

    Only the output is allocated here (or passed as ``out``); the call itself allocates nothing.  Calls
    that overlap on one GPU share that scratch and race.
    """
    lib = load()
    b = _gpu(b, "b")
    a = _gpu(a, "a")
    if a.dim() != 4 or b.dim() != 2:
        raise KrpeError("a must be [B,H,C,n] and b [H,2n-1]")
    B, H, C, n = a.shape
    if b.shape != (H, 2 * n - 1) or b.dtype != torch.float32 or a.dtype != torch.float32:
        raise KrpeError("b must be float32 [H, 2n-1] and a float32 [B,H,C,n]")
    if out is None:
        out = torch.empty_like(a)
    elif out.shape != a.shape or out.dtype != torch.float32 or not out.is_contiguous():
        raise KrpeError("out must be a contiguous float32 tensor shaped like a")
    st = lib.krpe_toeplitz_conv_noalloc(_ptr(b), _ptr(a), _ptr(out), B, H, C, n, _stream(a.device))
    _check(st, "krpe_toeplitz_conv_noalloc")
    return out


def attention_fwd_workspace(B: int, H: int, n: int, d: int, m: int, nprf: bool = False,
                            features: str = "prf", route: str = "auto", causal: bool = False) -> int:
    return int(load().krpe_attention_fwd_workspace_ex(B, H, n, d, m, _flags(nprf, features, route, causal)))


def attention_fwd_fixed_rows(workspace: torch.Tensor, B: int, H: int, n: int, d: int, m: int) -> int:
    """Rows of the last attention_fwd call on `workspace` that were evaluated exactly (waits for the stream)."""
    lib = load()
    out = ctypes.c_uint(0)
    st = lib.krpe_attention_fwd_stats(workspace.data_ptr(), workspace.numel(), B, H, n, d, m,
                                      ctypes.byref(out), _stream(workspace.device))
    _check(st, "krpe_attention_fwd_stats")
    return int(out.value)


def attention_fwd(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, b: torch.Tensor, W: torch.Tensor | None,
                  out: torch.Tensor | None = None, workspace: torch.Tensor | None = None,
                  events=None, nprf: bool = False, features: str = "prf", route: str = "auto",
                  causal: bool = False) -> torch.Tensor:
    """Eq. (10): z [B,H,n,d] fp32 from q, k, v [B,H,n,d] (fp32 or bf16), b [H,2n-1], W [H,m,d].

    ``nprf``: normalise the rows of q and k first (Algorithm 1's NPRF attention).
    ``features``: "prf" (Eq. (5)), "trf" (trigonometric, 2m features) or "elu"
    (elu + 1, W unused and may be None).
    ``route``: "fft" (Section 3.2), "direct" (Eq. (10) evaluated directly on
    MFMA, faster for short sequences) or "auto" (by sequence length).
    ``causal``: the caller states that b is -inf for every t > 0; only the
    "auto" route choice reads it (the direct route then costs half the pairs).

    ``out`` and ``workspace`` may be passed to reuse allocations (a uint8 tensor
    of at least attention_fwd_workspace() bytes).  ``events``: optional list of
    5 raw hipEvent_t handles recorded around the stages (see the C header).
    """
    lib = load()
    q, k, v = _gpu(q, "q"), _gpu(k, "k"), _gpu(v, "v")
    b = _gpu(b, "b")
    if q.dim() != 4:
        raise KrpeError("q must be [B,H,n,d]")
    B, H, n, d = q.shape
    if k.shape != q.shape or v.shape != q.shape or k.dtype != q.dtype or v.dtype != q.dtype:
        raise KrpeError("q, k, v must share shape and dtype")
    flags = _flags(nprf, features, route, causal)
    W, m = _proj(W, H, d, features)
    if b.shape != (H, 2 * n - 1) or b.dtype != torch.float32:
        raise KrpeError("b must be float32 [H, 2n-1]")
    if out is None:
        out = torch.empty((B, H, n, d), dtype=torch.float32, device=q.device)
    elif out.shape != (B, H, n, d) or out.dtype != torch.float32 or not out.is_contiguous():
        raise KrpeError("out must be a contiguous float32 [B,H,n,d] tensor")
    wsb = int(lib.krpe_attention_fwd_workspace_ex(B, H, n, d, m, flags))
    if workspace is None:
        workspace = torch.empty(max(wsb, 1), dtype=torch.uint8, device=q.device)
    dt = _dtype_code(q, "q")
    if workspace.numel() < wsb:
        raise KrpeError(f"workspace must hold at least {wsb} bytes")
    args = (_ptr(q), _ptr(k), _ptr(v), dt, _ptr(b), _ptr(W), _ptr(out), B, H, n, d, m, flags,
            workspace.data_ptr(), workspace.numel(), _stream(q.device))
    if events is None:
        st = lib.krpe_attention_fwd_ex(*args)
    else:
        if len(events) != STAGE_EVENTS:
            raise KrpeError(f"events must hold {STAGE_EVENTS} hipEvent_t handles")
        arr = (ctypes.c_void_p * STAGE_EVENTS)(*events)
        st = lib.krpe_attention_fwd_profiled(*args, arr)
    _check(st, "krpe_attention_fwd")
    return out


def attention_fwd_route(B: int, H: int, n: int, d: int, m: int, nprf: bool = False, features: str = "prf",
                        route: str = "auto", causal: bool = False) -> str:
    """The route ("direct" or "fft") attention_fwd takes for these sizes and options."""
    r = int(load().krpe_attention_fwd_route(B, H, n, d, m, _flags(nprf, features, route, causal)))
    if r == 0:
        raise KrpeError("invalid sizes or options")
    return "direct" if r == ROUTE_DIRECT else "fft"


def attention_bwd_workspace(B: int, H: int, n: int, d: int, m: int, nprf: bool = False) -> int:
    return int(load().krpe_attention_bwd_workspace(B, H, n, d, m, NPRF if nprf else 0))



def attention_bwd(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, b: torch.Tensor, W: torch.Tensor,
                  dz: torch.Tensor, workspace: torch.Tensor | None = None, nprf: bool = False,
                  with_db: bool = False, route: str = "auto", causal: bool = False) -> tuple:
    """Gradients (dq, dk, dv) [B,H,n,d] fp32 of sum(dz * z), z = attention_fwd(q, k, v, b, W, nprf=nprf)
    with PRF features and W fixed (the C header states the formulas); with_db adds db [H, 2n-1]."""
    lib = load()
    q, k, v = _gpu(q, "q"), _gpu(k, "k"), _gpu(v, "v")
    b, W, dz = _gpu(b, "b"), _gpu(W, "W"), _gpu(dz, "dz")
    if q.dim() != 4:
        raise KrpeError("q must be [B,H,n,d]")
    B, H, n, d = q.shape
    if k.shape != q.shape or v.shape != q.shape or k.dtype != q.dtype or v.dtype != q.dtype:
        raise KrpeError("q, k, v must share shape and dtype")
    if dz.shape != q.shape or dz.dtype != torch.float32:
        raise KrpeError("dz must be float32 [B,H,n,d]")
    if W.dim() != 3 or W.shape[0] != H or W.shape[2] != d or W.dtype != torch.float32:
        raise KrpeError("W must be float32 [H, m, d]")
    if b.shape != (H, 2 * n - 1) or b.dtype != torch.float32:
        raise KrpeError("b must be float32 [H, 2n-1]")
    m = W.shape[1]
    flags = _flags(nprf, "prf", route, causal)
    wsb = int(lib.krpe_attention_bwd_workspace(B, H, n, d, m, flags))
    if workspace is None:
        workspace = torch.empty(max(wsb, 1), dtype=torch.uint8, device=q.device)
    elif workspace.numel() < wsb:
        raise KrpeError(f"workspace must hold at least {wsb} bytes")
    dq = torch.empty((B, H, n, d), dtype=torch.float32, device=q.device)
    dk = torch.empty_like(dq)
    dv = torch.empty_like(dq)
    db = torch.empty((H, 2 * n - 1), dtype=torch.float32, device=q.device) if with_db else None
    st = lib.krpe_attention_bwd(_ptr(q), _ptr(k), _ptr(v), _dtype_code(q, "q"), _ptr(b), _ptr(W), _ptr(dz), _ptr(dq),
                                _ptr(dk), _ptr(dv), _ptr(db), B, H, n, d, m, flags, workspace.data_ptr(),
                                workspace.numel(), _stream(q.device))
    _check(st, "krpe_attention_bwd")
    return (dq, dk, dv, db) if with_db else (dq, dk, dv)
