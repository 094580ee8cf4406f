"""Plain fp64 CPU oracle for kernelized attention with RPE.

TEST INFRASTRUCTURE ONLY.  This module is imported by the test-suite, by the
smoke check of the build entry point and by the CPU-baseline leg of the
benchmark, and by nothing else: the library's compute path never calls it.

It computes the *definitions* written in the paper, directly and slowly, in
float64 (inputs given in fp32 or bf16 are converted exactly):

* ``prf_features``      -- Eq. (5), the positive random feature map.
* ``trf_features``      -- the trigonometric random feature map of Section 2
                           (sin features, then cos features).
* ``elu_features``      -- elu(x) + 1, the linear transformer's map that
                           Section 2 names.
* ``features``          -- one of the three by name.
* ``toeplitz_matrix``   -- the positional-correlation matrix C = {c_{j-i}},
                           c_t = exp(b_t) (Section 3.2, below Eq. (13)).
* ``toeplitz_product``  -- C @ a by plain matrix multiplication: the
                           "naive" quadratic route that the FFT replaces
                           (Eqs. (12)-(13)); FFT and direct product agree
                           exactly up to rounding, so this is the reference.
* ``toeplitz_rows``     -- the same product for selected output positions
                           only, one row of C at a time, so that sequences
                           too long for an n x n matrix can be checked.
* ``attention``         -- Eq. (10): z_i = phi(q_i) sum_j c_{j-i} phi(k_j)^T v_j
                           / phi(q_i) sum_j c_{j-i} phi(k_j)^T, O(n^2), for
                           any of the three feature maps.
* ``attention_rows``    -- the same formula evaluated for selected rows only,
                           so that outputs of full-size workloads can be
                           checked one by one.
* ``attention_grad``    -- gradients of <G, z> with respect to q, k, v and b
                           (W fixed), by the chain rule through Eq. (10),
                           Eq. (5), c = exp(b) and the row normalisation;
                           the paper states no backward pass, so this is the
                           derivative of its forward definition, pinned by
                           finite differences.
* ``normalize_rows``    -- the first step of Algorithm 1 (NPRF attention,
                           Section 3.3): every query and key divided by its
                           l2 norm; ``attention(..., nprf=True)`` applies it.

Conventions (readings of the paper, stated once here):
* b[h, s] holds b_t for t = s - (n - 1), the ordering of Algorithm 1's
  argument (b_{-(n-1)}, ..., b_{n-1}).
* C_ij = c_{j-i} with i the query position and j the key position, as in
  Eq. (6), Eq. (10) and the matrix printed in Eqs. (12)-(13).
* Causal masking is expressed through b alone: b_t = -inf gives c_t = 0
  exactly (Section 3.2, footnote on teacher forcing).
* phi is applied to q and k as given; any 1/sqrt(d) temperature is the
  caller's (Eq. (10) and the PRF variance lemma of Section 3.3 use the raw
  kernel exp(x y^T)).

Every function here is pinned by ``tests/test_oracle_pins.py`` against
brute force, closed forms, the paper's special cases and invariants.
"""
from __future__ import annotations

import numpy as np

__all__ = ["prf_features", "trf_features", "elu_features", "features", "toeplitz_matrix",
           "toeplitz_product", "toeplitz_rows", "attention", "attention_rows", "attention_grad", "normalize_rows"]


def _f64(x) -> np.ndarray:
    return np.asarray(x, dtype=np.float64)


def prf_features(x, W) -> np.ndarray:
    """Positive random features, Eq. (5).

    phi(x)_l = exp(w_l x^T - ||x||^2 / 2) / sqrt(m),  l = 1..m.

    x : [..., H, n, d] (or [n, d]);  W : [H, m, d] (or [m, d]).
    Returns [..., H, n, m] in float64.
    """
    x = _f64(x)
    W = _f64(W)
    m = W.shape[-2]
    proj = x @ np.swapaxes(W, -1, -2)                 # w_l . x for every row
    half_sq = 0.5 * np.sum(x * x, axis=-1, keepdims=True)
    return np.exp(proj - half_sq) / np.sqrt(m)


def trf_features(x, W) -> np.ndarray:
    """Trigonometric random features (Section 2, the map of Peng et al.).

    phi(x) = exp(||x||^2 / 2) / sqrt(m) [sin(w_1 x^T), ..., sin(w_m x^T),
                                         cos(w_1 x^T), ..., cos(w_m x^T)].

    x : [..., H, n, d] (or [n, d]);  W : [H, m, d] (or [m, d]).
    Returns [..., H, n, 2m] in float64 (signed values).
    """
    x = _f64(x)
    W = _f64(W)
    m = W.shape[-2]
    proj = x @ np.swapaxes(W, -1, -2)
    amp = np.exp(0.5 * np.sum(x * x, axis=-1, keepdims=True)) / np.sqrt(m)
    return np.concatenate([amp * np.sin(proj), amp * np.cos(proj)], axis=-1)


def elu_features(x, W=None) -> np.ndarray:
    """elu(x) + 1 elementwise (the linear transformer's map, Section 2): x + 1 for x > 0, exp(x) otherwise.

    d features; W is not used.  Returns [..., n, d] in float64.
    """
    x = _f64(x)
    return np.where(x > 0, x + 1.0, np.exp(np.minimum(x, 0.0)))


_MAPS = {"prf": prf_features, "trf": trf_features, "elu": elu_features}


def features(x, W, kind: str = "prf") -> np.ndarray:
    """phi(x) for kind in {"prf", "trf", "elu"} (W unused for "elu")."""
    return _MAPS[kind](x, W)


def normalize_rows(x) -> np.ndarray:
    """x_i / ||x_i||_2 for every row (last axis), Algorithm 1's first step; zero rows stay zero."""
    x = _f64(x)
    norm = np.sqrt(np.sum(x * x, axis=-1, keepdims=True))
    return np.divide(x, norm, out=np.zeros_like(x), where=norm > 0)


def toeplitz_matrix(b_h) -> np.ndarray:
    """C_ij = exp(b_{j-i}) for one head; b_h has length 2n-1 (index t + n - 1)."""
    b_h = _f64(b_h)
    n = (b_h.shape[-1] + 1) // 2
    i = np.arange(n)[:, None]
    j = np.arange(n)[None, :]
    return np.exp(b_h[j - i + n - 1])


def toeplitz_product(b, a) -> np.ndarray:
    """y[beta, h, c, i] = sum_j exp(b[h, j - i + n - 1]) a[beta, h, c, j].

    The direct (quadratic) product C a of Eqs. (12)-(13), per head.
    b : [H, 2n-1];  a : [B, H, C, n].  Returns [B, H, C, n] float64.
    """
    b = _f64(b)
    a = _f64(a)
    out = np.empty_like(a)
    for h in range(b.shape[0]):
        C = toeplitz_matrix(b[h])
        out[:, h] = a[:, h] @ C.T
    return out


def toeplitz_rows(b, a, rows) -> np.ndarray:
    """y[beta, h, c, r] = sum_j exp(b[h, j - i_r + n - 1]) a[beta, h, c, j] for i_r = rows[r].

    Row i of C of Eqs. (12)-(13) is c_{j-i} = exp(b_{j-i}) over the keys j,
    i.e. the window b[h, n-1-i : 2n-1-i] (Section 3.2, below Eq. (13)).
    b : [H, 2n-1];  a : [B, H, C, n];  rows : output positions.  Returns
    [B, H, C, len(rows)] float64.
    """
    b = _f64(b)
    a = _f64(a)
    n = a.shape[-1]
    out = np.empty(a.shape[:-1] + (len(rows),))
    for r, i in enumerate(rows):
        c_row = np.exp(b[:, n - 1 - i:2 * n - 1 - i])       # [H, n]: c_{j-i} for j = 0..n-1
        out[..., r] = np.einsum("bhcj,hj->bhc", a, c_row)
    return out


def attention(q, k, v, b, W, *, row_tile: int = 1024, nprf: bool = False, kind: str = "prf"):
    """Kernelized attention with RPE, Eq. (10), evaluated directly.

    For every (batch, head): Phi_q, Phi_k by the feature map `kind` (Eq. (5)
    for "prf"); the n x n weight matrix M_ij = c_{j-i} * phi(q_i) phi(k_j)^T;
    numerator M v, denominator M 1.  Rows are processed in tiles to bound
    memory.

    q, k, v : [B, H, n, d];  b : [H, 2n-1];  W : [H, m, d] (None for "elu").
    nprf: q and k rows normalised first (Algorithm 1).
    Returns (z [B, H, n, d], den [B, H, n]) in float64.
    """
    q, k, v, b = map(_f64, (q, k, v, b))
    W = _f64(W) if W is not None else [None] * q.shape[1]
    fmap = _MAPS[kind]
    if nprf:
        q, k = normalize_rows(q), normalize_rows(k)
    Bn, H, n, d = q.shape
    z = np.empty((Bn, H, n, d))
    den = np.empty((Bn, H, n))
    for h in range(H):
        for beta in range(Bn):
            fq = fmap(q[beta, h], W[h])
            fk = fmap(k[beta, h], W[h])
            for i0 in range(0, n, row_tile):
                i1 = min(n, i0 + row_tile)
                rows = np.arange(i0, i1)[:, None]
                cols = np.arange(n)[None, :]
                c = np.exp(b[h][cols - rows + n - 1])      # c_{j-i}
                mt = c * (fq[i0:i1] @ fk.T)
                num = mt @ v[beta, h]
                dd = mt.sum(axis=1)
                z[beta, h, i0:i1] = num / dd[:, None]
                den[beta, h, i0:i1] = dd
    return z, den


def attention_rows(q, k, v, b, W, rows, *, nprf: bool = False, kind: str = "prf"):
    """Eq. (10) for selected output rows only.

    rows : iterable of (beta, h, i).  Returns (z [R, d], den [R]) float64 in
    the order given.  Cost per row is O(n (m + d)) after one O(n m d)
    feature map per distinct (beta, h).
    """
    b = _f64(b)
    if nprf:
        q, k = normalize_rows(q), normalize_rows(k)
    fmap = _MAPS[kind]
    if W is None:
        W = [None] * q.shape[1]
    rows = [tuple(int(t) for t in r) for r in rows]
    n = q.shape[2]
    d = q.shape[3]
    z = np.empty((len(rows), d))
    den = np.empty(len(rows))
    cache = {}
    for r, (beta, h, i) in enumerate(rows):
        if (beta, h) not in cache:
            cache.clear()
            cache[(beta, h)] = fmap(k[beta, h], W[h])
        fk = cache[(beta, h)]
        fq = fmap(_f64(q[beta, h, i])[None, :], W[h])[0]
        c = np.exp(b[h][np.arange(n) - i + n - 1])
        w = c * (fk @ fq)
        den[r] = w.sum()
        z[r] = (w @ _f64(v[beta, h])) / den[r]
    return z, den


def attention_grad(q, k, v, b, W, G, *, nprf: bool = False):
    """Gradients of L = sum z * G through Eq. (10) with PRF features, W fixed.

    Per (batch, head), with Phi_q, Phi_k from Eq. (5), K = Phi_q Phi_k^T,
    C_ij = c_{j-i} = exp(b_{j-i}), A = C * K (elementwise), z = (A v) / (A 1):
      dN_i = G_i / den_i,  dden_i = -(G_i . z_i) / den_i,
      dA = dN v^T + dden 1^T,
      dv = A^T dN,
      dK = dA * C,   dPhi_q = dK Phi_k,   dPhi_k = dK^T Phi_q,
      dC = dA * K,   dc_t = sum over the diagonal j - i = t of dC,  db_t = dc_t c_t,
      dx = (dPhi * Phi) W - x * rowsum(dPhi * Phi)     (d phi_l / dx = phi_l (w_l - x)),
    and with nprf, x = u / ||u|| gives du = (dx - x (x . dx)) / ||u|| (0 for a zero row).
    db is summed over the batch (b is per head); entries with b_t = -inf get 0.

    q, k, v, G : [B, H, n, d];  b : [H, 2n-1];  W : [H, m, d].
    Returns (dq, dk, dv [B, H, n, d], db [H, 2n-1]) in float64.
    """
    q, k, v, b, W, G = map(_f64, (q, k, v, b, W, G))
    Bn, H, n, d = q.shape
    qs, ks = (normalize_rows(q), normalize_rows(k)) if nprf else (q, k)
    dq = np.zeros_like(q)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)
    db = np.zeros_like(b)
    i = np.arange(n)[:, None]
    j = np.arange(n)[None, :]
    for h in range(H):
        C = np.exp(b[h][j - i + n - 1])
        for beta in range(Bn):
            fq = prf_features(qs[beta, h], W[h])
            fk = prf_features(ks[beta, h], W[h])
            K = fq @ fk.T
            A = C * K
            den = A.sum(axis=1)
            z = (A @ v[beta, h]) / den[:, None]
            dN = G[beta, h] / den[:, None]
            dden = -np.sum(G[beta, h] * z, axis=1) / den
            dA = dN @ v[beta, h].T + dden[:, None]
            dv[beta, h] = A.T @ dN
            dK = dA * C
            dfq = dK @ fk
            dfk = dK.T @ fq
            dC = dA * K
            for t in range(-(n - 1), n):
                db[h, t + n - 1] += np.trace(dC, offset=t)
            for x, dphi, phi, out, raw in ((qs[beta, h], dfq, fq, dq, q[beta, h]),
                                           (ks[beta, h], dfk, fk, dk, k[beta, h])):
                P = dphi * phi
                dx = P @ W[h] - x * P.sum(axis=1, keepdims=True)
                if nprf:
                    nrm = np.sqrt(np.sum(raw * raw, axis=1, keepdims=True))
                    dx = np.divide(dx - x * np.sum(x * dx, axis=1, keepdims=True), nrm,
                                   out=np.zeros_like(dx), where=nrm > 0)
                out[beta, h] = dx
    cfin = np.isfinite(b)
    db = np.where(cfin, db * np.exp(np.where(cfin, b, 0.0)), 0.0)
    return dq, dk, dv, db
