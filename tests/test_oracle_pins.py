"""Pins of the fp64 oracle against things other than itself.

Each ``check_*`` function takes the oracle implementation as an argument so
that ``test_oracle_mutants.py`` can re-run the same checks on deliberately
broken copies of it and show that every planted mistake is caught.

Sources of truth used here (none of them re-types the oracle's formula):
* brute force with scalar Python loops straight from Eq. (5) and Eq. (10);
* the paper's own factorisation route: vec-stacked A_1, A_2, the Toeplitz
  matrix of Eqs. (12)-(13) and the ratio of Eq. (10);
* the closed form Eq. (3) (linear attention) that Eq. (10) reduces to when b
  is constant, and its prefix-sum form under the causal mask;
* the PRF variance lemma of Section 3.3 (unbiasedness and exact variance of the PRF kernel estimate);
* for the other feature maps of Section 2: scalar loops, the product-to-sum
  identity of the trigonometric map, its unbiasedness for the softmax kernel
  (E cos(w u) = exp(-|u|^2/2) for Gaussian w), and the linear-attention route;
* for the gradients (the paper states no backward pass): central finite
  differences of the forward definition, and invariances (constant shift of
  b, constant shift of a value column, scale of normalised queries/keys);
* the softmax-with-RPE limit (Eq. (1) with the bias of Eq. (6)) as m grows;
* textbook special cases of a Toeplitz product (identity, shift, sum,
  cumulative sum) and invariants of Eq. (10).
"""
import math

import numpy as np
import pytest

import oracle as ORACLE
from paper_2106_12566_amd import synth


# --------------------------------------------------------------------------
# helpers (independent of the oracle)
# --------------------------------------------------------------------------

def _rand_case(rng, B, H, n, d, m, sigma_b=0.5, scale=None):
    scale = d ** -0.25 if scale is None else scale
    q = rng.standard_normal((B, H, n, d)) * scale
    k = rng.standard_normal((B, H, n, d)) * scale
    v = rng.standard_normal((B, H, n, d))
    W = rng.standard_normal((H, m, d))
    b = rng.standard_normal((H, 2 * n - 1)) * sigma_b
    return q, k, v, b, W


def _rownorm_err(a, ref):
    a = np.asarray(a, np.float64)
    ref = np.asarray(ref, np.float64)
    num = np.max(np.abs(a - ref), axis=-1)
    den = np.max(np.abs(ref), axis=-1)
    return float(np.max(num / den))


def _brute_phi(x_row, W_h):
    """Eq. (5) for one vector, scalar loops."""
    m = len(W_h)
    sq = sum(t * t for t in x_row)
    out = []
    for l in range(m):
        dot = sum(W_h[l][a] * x_row[a] for a in range(len(x_row)))
        out.append(math.exp(dot - sq / 2.0) / math.sqrt(m))
    return out


def _brute_attention(q, k, v, b, W):
    """Eq. (10) with scalar loops; b[h][t + n - 1] = b_t."""
    Bn, H, n, d = q.shape
    z = np.zeros((Bn, H, n, d))
    for beta in range(Bn):
        for h in range(H):
            Wh = W[h].tolist()
            fq = [_brute_phi(q[beta, h, i].tolist(), Wh) for i in range(n)]
            fk = [_brute_phi(k[beta, h, j].tolist(), Wh) for j in range(n)]
            for i in range(n):
                num = [0.0] * d
                den = 0.0
                for j in range(n):
                    kern = sum(a * c for a, c in zip(fq[i], fk[j]))
                    w = math.exp(b[h][j - i + n - 1]) * kern
                    den += w
                    for c in range(d):
                        num[c] += w * v[beta, h, j, c]
                for c in range(d):
                    z[beta, h, i, c] = num[c] / den
    return z


# --------------------------------------------------------------------------
# checks (parametrised by the implementation under test)
# --------------------------------------------------------------------------

def check_brute_force(impl):
    rng = np.random.default_rng(11)
    for (n, d, m) in [(1, 3, 2), (5, 4, 3), (9, 6, 5), (16, 8, 7)]:
        q, k, v, b, W = _rand_case(rng, 2, 2, n, d, m)
        z, _ = impl.attention(q, k, v, b, W)
        assert _rownorm_err(z, _brute_attention(q, k, v, b, W)) < 1e-12, (n, d, m)


def check_toeplitz_factorisation(impl):
    """Eqs. (11)-(13): with A the n x (m d + m) matrix whose row j is
    [vec(phi(k_j)^T v_j), phi(k_j)] and C = {c_{j-i}}, every entry of
    D-tilde = C A equals its summation form sum_j c_{j-i} A[j, :] (scalar
    loops), and phi(q_i) applied to the two blocks of row i gives the
    numerator and denominator of Eq. (10) (the oracle's z and den)."""
    rng = np.random.default_rng(12)
    n, d, m = 13, 5, 6
    q, k, v, b, W = _rand_case(rng, 1, 1, n, d, m)
    Wh, bh = W[0], b[0]
    phi = lambda x: np.exp(x @ Wh.T - 0.5 * (x * x).sum(-1, keepdims=True)) / np.sqrt(m)
    fq, fk, vv = phi(q[0, 0]), phi(k[0, 0]), v[0, 0]
    A = np.concatenate([np.einsum("jl,jc->jlc", fk, vv).reshape(n, m * d), fk], axis=1)
    C = np.array([[math.exp(bh[(j - i) + n - 1]) for j in range(n)] for i in range(n)])
    Dt = C @ A
    for i in (0, 4, n - 1):
        for l in (0, m - 1):
            for c in (0, d - 1):
                s1 = sum(math.exp(bh[j - i + n - 1]) * fk[j, l] * vv[j, c] for j in range(n))
                assert abs(Dt[i, l * d + c] - s1) <= 1e-13 * abs(s1)
            s2 = sum(math.exp(bh[j - i + n - 1]) * fk[j, l] for j in range(n))
            assert abs(Dt[i, m * d + l] - s2) <= 1e-13 * abs(s2)
    num = np.einsum("il,ilc->ic", fq, Dt[:, : m * d].reshape(n, m, d))
    den_ref = np.einsum("il,il->i", fq, Dt[:, m * d:])
    z, den = impl.attention(q, k, v, b, W)
    assert _rownorm_err(z[0, 0], num / den_ref[:, None]) < 1e-12
    assert np.allclose(den[0, 0], den_ref, rtol=1e-12)


def check_single_position(impl):
    rng = np.random.default_rng(13)
    q, k, v, b, W = _rand_case(rng, 2, 3, 1, 4, 8)
    z, den = impl.attention(q, k, v, b, W)
    assert np.allclose(z, v, rtol=1e-13, atol=0)
    assert np.all(den > 0)


def check_const_bias_is_linear_attention(impl):
    """b == kappa makes c a constant, Eq. (10) becomes Eq. (3) (O(n) route)."""
    rng = np.random.default_rng(14)
    n, d, m = 40, 8, 16
    q, k, v, _, W = _rand_case(rng, 2, 2, n, d, m)
    b = np.full((2, 2 * n - 1), 0.37)
    z, _ = impl.attention(q, k, v, b, W)
    for beta in range(2):
        for h in range(2):
            phi = lambda x: np.exp(x @ W[h].T - 0.5 * (x * x).sum(-1, keepdims=True)) / np.sqrt(m)
            fq, fk = phi(q[beta, h]), phi(k[beta, h])
            S = fk.T @ v[beta, h]                 # sum_j phi(k_j)^T v_j
            s = fk.sum(axis=0)                    # sum_j phi(k_j)^T
            ref = (fq @ S) / (fq @ s)[:, None]
            assert _rownorm_err(z[beta, h], ref) < 1e-12


def check_causal_prefix_sums(impl):
    """b_t = kappa for t <= 0, -inf for t > 0: the teacher-forcing mask.

    Query i then sees keys j <= i only and Eq. (10) becomes running sums of
    phi(k_j)^T v_j and phi(k_j)^T.
    """
    rng = np.random.default_rng(15)
    n, d, m = 33, 6, 10
    q, k, v, _, W = _rand_case(rng, 1, 2, n, d, m)
    t = np.arange(-(n - 1), n)
    b = np.where(t <= 0, -0.8, -np.inf)[None, :].repeat(2, axis=0)
    z, den = impl.attention(q, k, v, b, W)
    for h in range(2):
        phi = lambda x: np.exp(x @ W[h].T - 0.5 * (x * x).sum(-1, keepdims=True)) / np.sqrt(m)
        fq, fk = phi(q[0, h]), phi(k[0, h])
        S = np.cumsum(fk[:, :, None] * v[0, h][:, None, :], axis=0)    # [n, m, d]
        s = np.cumsum(fk, axis=0)
        ref = np.einsum("il,ilc->ic", fq, S) / np.einsum("il,il->i", fq, s)[:, None]
        assert _rownorm_err(z[0, h], ref) < 1e-12
        assert np.allclose(den[0, h], math.exp(-0.8) * np.einsum("il,il->i", fq, s), rtol=1e-12)


def check_only_diagonal(impl):
    """Only b_0 finite: C = c_0 I, so z_i = v_i exactly."""
    rng = np.random.default_rng(16)
    n = 17
    q, k, v, _, W = _rand_case(rng, 1, 1, n, 4, 6)
    b = np.full((1, 2 * n - 1), -np.inf)
    b[0, n - 1] = 1.3
    z, den = impl.attention(q, k, v, b, W)
    assert np.allclose(z, v, rtol=1e-13, atol=1e-15)
    assert np.all(den > 0)


def check_shift_kernel(impl):
    """Only b_{+1} finite: row i sees key i+1 only (last row sees nothing).

    Pins the sign of the offset: under C_ij = c_{j-i}, z_i = v_{i+1}.
    """
    rng = np.random.default_rng(17)
    n = 9
    q, k, v, _, W = _rand_case(rng, 1, 1, n, 3, 4)
    b = np.full((1, 2 * n - 1), -np.inf)
    b[0, n] = 0.0          # t = +1
    with np.errstate(invalid="ignore", divide="ignore"):
        z, den = impl.attention(q, k, v, b, W)
    assert np.allclose(z[0, 0, :-1], v[0, 0, 1:], rtol=1e-13, atol=1e-15)
    assert den[0, 0, -1] == 0.0


def check_invariants(impl):
    rng = np.random.default_rng(18)
    n, d, m = 24, 6, 12
    q, k, v, b, W = _rand_case(rng, 1, 2, n, d, m)
    z, _ = impl.attention(q, k, v, b, W)
    # b + kappa scales c, which cancels between numerator and denominator
    z2, _ = impl.attention(q, k, v, b + 0.9, W)
    assert _rownorm_err(z2, z) < 1e-12
    # v == 1 => z == 1 (rows of the attention weights sum to one)
    z1, _ = impl.attention(q, k, np.ones_like(v), b, W)
    assert np.allclose(z1, 1.0, rtol=1e-13)
    # affine equivariance in v
    A = rng.standard_normal((d, d))
    u = rng.standard_normal(d)
    za, _ = impl.attention(q, k, v @ A + u, b, W)
    assert _rownorm_err(za, z @ A + u) < 1e-11
    # convex hull of the values
    assert np.all(z <= v.max(axis=2, keepdims=True) + 1e-12)
    assert np.all(z >= v.min(axis=2, keepdims=True) - 1e-12)
    # reversal: reverse positions and map b_t -> b_{-t}
    zr, _ = impl.attention(q[:, :, ::-1], k[:, :, ::-1], v[:, :, ::-1], b[:, ::-1], W)
    assert _rownorm_err(zr[:, :, ::-1], z) < 1e-12
    # permuting the random features leaves z unchanged
    zp, _ = impl.attention(q, k, v, b, W[:, rng.permutation(m)])
    assert _rownorm_err(zp, z) < 1e-12


def check_causality(impl):
    rng = np.random.default_rng(19)
    n, d, m = 20, 5, 7
    q, k, v, _, W = _rand_case(rng, 1, 1, n, d, m)
    t = np.arange(-(n - 1), n)
    b = np.where(t <= 0, rng.standard_normal(2 * n - 1) * 0.5, -np.inf)[None]
    z, _ = impl.attention(q, k, v, b, W)
    cut = 11
    k2, v2 = k.copy(), v.copy()
    k2[:, :, cut:] += rng.standard_normal(k2[:, :, cut:].shape)
    v2[:, :, cut:] += rng.standard_normal(v2[:, :, cut:].shape)
    z2, _ = impl.attention(q, k2, v2, b, W)
    assert np.array_equal(z[:, :, :cut], z2[:, :, :cut])
    assert not np.allclose(z[:, :, cut:], z2[:, :, cut:])


def check_prf_variance_lemma(impl):
    """E_W[phi(x) phi(y)^T] = exp(x y^T); Var = (exp(|x+y|^2) - 1) exp(x y^T)^2 / m."""
    rng = np.random.default_rng(20)
    d, m, T = 16, 16, 20000
    x = rng.standard_normal(d)
    y = rng.standard_normal(d)
    x *= 0.7 / np.linalg.norm(x)
    y *= 0.7 / np.linalg.norm(y)
    W = rng.standard_normal((T, m, d))
    fx = impl.prf_features(x[None, None, :], W)[:, 0, :]     # [T, m]
    fy = impl.prf_features(y[None, None, :], W)[:, 0, :]
    est = np.sum(fx * fy, axis=1)
    target = math.exp(float(x @ y))
    se = est.std(ddof=1) / math.sqrt(T)
    assert abs(est.mean() - target) < 4 * se
    var_exact = (math.exp(float((x + y) @ (x + y))) - 1.0) * target ** 2 / m
    assert abs(est.var(ddof=1) / var_exact - 1.0) < 0.05


def check_toeplitz_special_cases(impl):
    rng = np.random.default_rng(21)
    n = 15
    a = rng.standard_normal((2, 1, 3, n))
    t = np.arange(-(n - 1), n)
    # identity: only b_0 finite (= 0)
    b = np.where(t == 0, 0.0, -np.inf)[None]
    assert np.array_equal(impl.toeplitz_product(b, a), a)
    # shift: only b_{-1} finite, y_i = a_{i-1}
    b = np.where(t == -1, 0.0, -np.inf)[None]
    y = impl.toeplitz_product(b, a)
    assert np.array_equal(y[..., 1:], a[..., :-1]) and np.all(y[..., 0] == 0)
    # all ones: y_i = sum_j a_j
    b = np.zeros((1, 2 * n - 1))
    assert np.allclose(impl.toeplitz_product(b, a), a.sum(-1, keepdims=True), rtol=1e-13)
    # causal ones: cumulative sum
    b = np.where(t <= 0, 0.0, -np.inf)[None]
    assert np.allclose(impl.toeplitz_product(b, a), np.cumsum(a, axis=-1), rtol=1e-12, atol=1e-14)
    # brute force on random b
    b = rng.standard_normal((1, 2 * n - 1))
    y = impl.toeplitz_product(b, a)
    ref = np.zeros_like(a)
    for i in range(n):
        for j in range(n):
            ref[..., i] += math.exp(b[0, j - i + n - 1]) * a[..., j]
    assert np.allclose(y, ref, rtol=1e-13, atol=1e-13)


def check_toeplitz_rows(impl):
    """Selected rows of C a: scalar brute force on random b, and the special cases of the
    full product (identity, shift, all ones, causal ones) at the rows asked for."""
    rng = np.random.default_rng(23)
    n = 13
    a = rng.standard_normal((2, 2, 3, n))
    rows = [0, 1, 6, n - 1]
    b = rng.standard_normal((2, 2 * n - 1))
    y = impl.toeplitz_rows(b, a, rows)
    assert y.shape == (2, 2, 3, len(rows))
    for r, i in enumerate(rows):
        ref = np.zeros((2, 2, 3))
        for h in range(2):
            for j in range(n):
                ref[:, h] += math.exp(b[h, j - i + n - 1]) * a[:, h, :, j]
        assert np.allclose(y[..., r], ref, rtol=1e-13, atol=1e-13)
    t = np.arange(-(n - 1), n)
    ident = np.where(t == 0, 0.0, -np.inf)[None].repeat(2, 0)
    assert np.array_equal(impl.toeplitz_rows(ident, a, rows), a[..., rows])
    shift = np.where(t == -1, 0.0, -np.inf)[None].repeat(2, 0)
    ys = impl.toeplitz_rows(shift, a, rows)
    assert np.all(ys[..., 0] == 0) and np.array_equal(ys[..., 1:], a[..., [i - 1 for i in rows[1:]]])
    ones = np.zeros((2, 2 * n - 1))
    assert np.allclose(impl.toeplitz_rows(ones, a, rows), a.sum(-1)[..., None].repeat(len(rows), -1), rtol=1e-13)
    causal = np.where(t <= 0, 0.0, -np.inf)[None].repeat(2, 0)
    assert np.allclose(impl.toeplitz_rows(causal, a, rows), np.cumsum(a, axis=-1)[..., rows], rtol=1e-12,
                       atol=1e-14)


def _brute_normalize(x_row):
    """x / ||x||_2 with scalar arithmetic (Algorithm 1, first step); zero stays zero."""
    nrm = math.sqrt(sum(t * t for t in x_row))
    return [t / nrm for t in x_row] if nrm > 0 else [0.0 for _ in x_row]


def check_nprf_brute_force(impl):
    """NPRF attention (Algorithm 1): normalise q and k rows, then Eq. (10), scalar loops."""
    rng = np.random.default_rng(21)
    for (n, d, m) in [(1, 3, 2), (6, 4, 5), (11, 7, 3)]:
        q, k, v, b, W = _rand_case(rng, 2, 2, n, d, m, scale=1.7)
        q[0, 1, 0] = 0.0                      # a zero row stays zero
        qn = np.array([[[_brute_normalize(q[a, h, i].tolist()) for i in range(n)] for h in range(2)]
                       for a in range(2)])
        kn = np.array([[[_brute_normalize(k[a, h, i].tolist()) for i in range(n)] for h in range(2)]
                       for a in range(2)])
        z, _ = impl.attention(q, k, v, b, W, nprf=True)
        assert _rownorm_err(z, _brute_attention(qn, kn, v, b, W)) < 1e-12, (n, d, m)
        rows = [(1, 0, n - 1), (0, 1, 0)]
        zr, _ = impl.attention_rows(q, k, v, b, W, rows, nprf=True)
        for r, (a, h, i) in enumerate(rows):
            assert np.allclose(zr[r], z[a, h, i], rtol=1e-12, atol=1e-14)


def check_nprf_scale_invariance(impl):
    """Under NPRF, rescaling each query and key by a positive factor changes nothing;
    inputs that are already unit rows give the plain Eq. (10) result."""
    rng = np.random.default_rng(22)
    q, k, v, b, W = _rand_case(rng, 1, 2, 12, 6, 9)
    z0, _ = impl.attention(q, k, v, b, W, nprf=True)
    sq = rng.uniform(0.1, 5.0, size=q.shape[:-1] + (1,))
    sk = rng.uniform(0.1, 5.0, size=k.shape[:-1] + (1,))
    z1, _ = impl.attention(q * sq, k * sk, v, b, W, nprf=True)
    assert _rownorm_err(z1, z0) < 1e-12
    qu = q / np.linalg.norm(q, axis=-1, keepdims=True)
    ku = k / np.linalg.norm(k, axis=-1, keepdims=True)
    z2, _ = impl.attention(qu, ku, v, b, W)
    assert _rownorm_err(z2, z0) < 1e-12
    # and the normalisation does matter for inputs that are not unit rows
    z3, _ = impl.attention(q * sq, k * sk, v, b, W)
    assert _rownorm_err(z3, z0) > 1e-6


def check_rows_match_full(impl):
    d = synth.custom(2, 3, 64, 16, 8, seed=5)
    q, k, v, b, W = d["q"], d["k"], d["v"], d["b"], d["W"]
    z, den = impl.attention(q, k, v, b, W)
    rows = [(1, 2, 0), (0, 1, 63), (0, 0, 1), (1, 0, 32), (0, 2, 62), (1, 1, 5)]
    zr, dr = impl.attention_rows(q, k, v, b, W, rows)
    for r, (beta, h, i) in enumerate(rows):
        assert np.allclose(zr[r], z[beta, h, i], rtol=1e-12, atol=1e-14)
        assert np.isclose(dr[r], den[beta, h, i], rtol=1e-12)


def _brute_trf(x_row, W_h):
    """The trigonometric map of Section 2 for one vector, scalar loops: sin features, then cos."""
    m = len(W_h)
    amp = math.exp(sum(t * t for t in x_row) / 2.0) / math.sqrt(m)
    dots = [sum(W_h[l][a] * x_row[a] for a in range(len(x_row))) for l in range(m)]
    return [amp * math.sin(t) for t in dots] + [amp * math.cos(t) for t in dots]


def _brute_elu(x_row, W_h=None):
    """elu(x) + 1 for one vector, scalar branches."""
    return [t + 1.0 if t > 0 else math.exp(t) for t in x_row]


def _brute_attention_map(q, k, v, b, W, phi):
    """Eq. (10) with scalar loops for any feature map phi(row, W_h)."""
    Bn, H, n, d = q.shape
    z = np.zeros((Bn, H, n, d))
    for beta in range(Bn):
        for h in range(H):
            Wh = None if W is None else W[h].tolist()
            fq = [phi(q[beta, h, i].tolist(), Wh) for i in range(n)]
            fk = [phi(k[beta, h, j].tolist(), Wh) for j in range(n)]
            for i in range(n):
                num = [0.0] * d
                den = 0.0
                for j in range(n):
                    w = math.exp(b[h][j - i + n - 1]) * sum(a * c for a, c in zip(fq[i], fk[j]))
                    den += w
                    for c in range(d):
                        num[c] += w * v[beta, h, j, c]
                for c in range(d):
                    z[beta, h, i, c] = num[c] / den
    return z


def check_trf_brute_force(impl):
    """TRF features and Eq. (10) with them against scalar loops (values near 1, so the
    signed denominator stays away from zero)."""
    rng = np.random.default_rng(31)
    for (n, d, m) in [(1, 3, 2), (5, 4, 3), (9, 6, 5)]:
        q, k, v, b, W = _rand_case(rng, 2, 2, n, d, m, scale=0.15)
        W *= 0.3
        ref_phi = np.array([[[_brute_trf(q[a, h, i].tolist(), W[h].tolist()) for i in range(n)]
                             for h in range(2)] for a in range(2)])
        assert np.max(np.abs(impl.trf_features(q, W) - ref_phi)) < 1e-13
        assert np.max(np.abs(impl.features(q, W, "trf") - ref_phi)) < 1e-13
        z, _ = impl.attention(q, k, v, b, W, kind="trf")
        assert _rownorm_err(z, _brute_attention_map(q, k, v, b, W, _brute_trf)) < 1e-11, (n, d, m)
        rows = [(1, 0, n - 1), (0, 1, 0)]
        zr, _ = impl.attention_rows(q, k, v, b, W, rows, kind="trf")
        for r, (a, h, i) in enumerate(rows):
            assert np.allclose(zr[r], z[a, h, i], rtol=1e-12, atol=1e-14)


def check_trf_kernel_identity(impl):
    """sin a sin b + cos a cos b = cos(a - b): phi(x).phi(y) equals
    exp((|x|^2 + |y|^2)/2) / m * sum_l cos(w_l (x - y)), a form with no sin/cos split."""
    rng = np.random.default_rng(32)
    x = rng.standard_normal((7, 5)) * 0.6
    y = rng.standard_normal((9, 5)) * 0.6
    W = rng.standard_normal((11, 5))
    fx, fy = impl.trf_features(x, W), impl.trf_features(y, W)
    assert fx.shape == (7, 22)
    for i in range(7):
        for j in range(9):
            u = x[i] - y[j]
            ref = math.exp((x[i] @ x[i] + y[j] @ y[j]) / 2.0) / 11.0 * sum(math.cos(W[l] @ u) for l in range(11))
            assert abs(fx[i] @ fy[j] - ref) < 1e-12 * max(1.0, abs(ref))


def check_trf_unbiased(impl):
    """With w ~ N(0, I), E[cos(w u)] = exp(-|u|^2/2), so phi(x).phi(y) estimates exp(x y^T)
    (the softmax kernel); the m-term mean of cosines is within 6/sqrt(m) of its expectation."""
    rng = np.random.default_rng(33)
    d, m = 6, 40000
    x = rng.standard_normal(d) * 0.3
    y = rng.standard_normal(d) * 0.3
    W = rng.standard_normal((m, d))
    est = impl.trf_features(x[None], W)[0] @ impl.trf_features(y[None], W)[0]
    amp = math.exp((x @ x + y @ y) / 2.0)
    assert abs(est / amp - math.exp(-((x - y) @ (x - y)) / 2.0)) < 6.0 / math.sqrt(m)
    assert abs(est / math.exp(x @ y) - 1.0) < 6.0 * amp / math.sqrt(m) / math.exp(x @ y)


def check_elu_brute_force(impl):
    """elu + 1 features and Eq. (10) with them against scalar loops, W not used."""
    rng = np.random.default_rng(34)
    for (n, d) in [(1, 3), (6, 4), (10, 7)]:
        q, k, v, b, _ = _rand_case(rng, 2, 2, n, d, 1, scale=1.0)
        q[0, 0, 0, 0] = 0.0
        ref_phi = np.array([[[_brute_elu(q[a, h, i].tolist()) for i in range(n)] for h in range(2)]
                            for a in range(2)])
        assert np.max(np.abs(impl.elu_features(q) - ref_phi)) < 1e-15
        z, _ = impl.attention(q, k, v, b, None, kind="elu")
        assert _rownorm_err(z, _brute_attention_map(q, k, v, b, None, _brute_elu)) < 1e-12, (n, d)
        rows = [(1, 1, n - 1), (0, 0, 0)]
        zr, _ = impl.attention_rows(q, k, v, b, None, rows, kind="elu")
        for r, (a, h, i) in enumerate(rows):
            assert np.allclose(zr[r], z[a, h, i], rtol=1e-12, atol=1e-14)


def check_feature_maps_linear_route(impl):
    """Constant b: Eq. (10) is linear attention, Eq. (3), whatever the feature map;
    computed through the d x M summary sum_j phi(k_j)^T v_j (the O(n) route)."""
    rng = np.random.default_rng(35)
    n, d, m = 30, 6, 8
    q, k, v, _, W = _rand_case(rng, 1, 2, n, d, m, scale=0.3)
    b = np.full((2, 2 * n - 1), -0.21)
    maps = {"trf": lambda x, Wh: [_brute_trf(r, Wh) for r in x.tolist()],
            "elu": lambda x, Wh: [_brute_elu(r) for r in x.tolist()]}
    for kind, phi in maps.items():
        z, _ = impl.attention(q, k, v, b, W if kind == "trf" else None, kind=kind)
        for h in range(2):
            fq = np.array(phi(q[0, h], W[h].tolist()))
            fk = np.array(phi(k[0, h], W[h].tolist()))
            ref = (fq @ (fk.T @ v[0, h])) / (fq @ fk.sum(axis=0))[:, None]
            assert _rownorm_err(z[0, h], ref) < 1e-11, kind


def _fd_grads(impl, q, k, v, b, W, G, nprf, eps=1e-6):
    """Central differences of L = sum(z * G) in every entry of q, k, v and every finite entry of b."""
    def loss(q_, k_, v_, b_):
        z, _ = impl.attention(q_, k_, v_, b_, W, nprf=nprf)
        return float(np.sum(z * G))
    out = []
    for which in range(4):
        args = [q.copy(), k.copy(), v.copy(), b.copy()]
        base = args[which]
        g = np.zeros_like(base)
        for idx in np.ndindex(base.shape):
            if not np.isfinite(base[idx]):
                continue
            keep = base[idx]
            base[idx] = keep + eps
            lp = loss(*args)
            base[idx] = keep - eps
            lm = loss(*args)
            base[idx] = keep
            g[idx] = (lp - lm) / (2 * eps)
        out.append(g)
    return out


def check_grad_finite_differences(impl):
    """attention_grad against central differences of the forward definition (tiny cases,
    plain and normalised, one with a causal b)."""
    rng = np.random.default_rng(51)
    for (n, d, m, nprf, causal) in [(5, 3, 4, False, False), (4, 2, 3, True, False), (6, 3, 5, False, True)]:
        q, k, v, b, W = _rand_case(rng, 1, 2, n, d, m, scale=0.7)
        if causal:
            b[:, n:] = -np.inf
        G = rng.standard_normal(q.shape)
        got = impl.attention_grad(q, k, v, b, W, G, nprf=nprf)
        ref = _fd_grads(impl, q, k, v, b, W, G, nprf)
        for name, a_, r_ in zip("qkvb", got, ref):
            assert a_.shape == r_.shape, name
            scale = max(np.max(np.abs(r_)), 1e-3)
            assert np.max(np.abs(a_ - r_)) <= 1e-6 * scale, (name, n, nprf, causal, np.max(np.abs(a_ - r_)))
        if causal:
            assert np.all(got[3][:, n:] == 0.0)


def check_grad_invariants(impl):
    """A constant shift of b leaves z unchanged (sum_t db_t = 0); adding a to every value of
    column c shifts z[., c] by a (sum_j dv[j, c] = sum_i G[i, c]); under NPRF, scaling a query
    or key changes nothing (dq_i . q_i = dk_j . k_j = 0)."""
    rng = np.random.default_rng(52)
    q, k, v, b, W = _rand_case(rng, 2, 2, 12, 5, 7)
    G = rng.standard_normal(q.shape)
    dq, dk, dv, db = impl.attention_grad(q, k, v, b, W, G)
    assert np.max(np.abs(db.sum(axis=1))) < 1e-10 * np.max(np.abs(db))
    assert np.allclose(dv.sum(axis=2), G.sum(axis=2), rtol=1e-10, atol=1e-12)
    dq, dk, dv, db = impl.attention_grad(q * 2.0, k * 0.5, v, b, W, G, nprf=True)
    assert np.max(np.abs(np.sum(dq * q, axis=-1))) < 1e-10 * np.max(np.abs(dq)) * np.max(np.abs(q))
    assert np.max(np.abs(np.sum(dk * k, axis=-1))) < 1e-10 * np.max(np.abs(dk)) * np.max(np.abs(k))


ALL_CHECKS = [check_brute_force, check_toeplitz_factorisation, check_single_position,
              check_const_bias_is_linear_attention, check_causal_prefix_sums,
              check_only_diagonal, check_shift_kernel, check_invariants,
              check_causality, check_prf_variance_lemma, check_toeplitz_special_cases, check_toeplitz_rows,
              check_rows_match_full, check_nprf_brute_force, check_nprf_scale_invariance,
              check_trf_brute_force, check_trf_kernel_identity, check_trf_unbiased,
              check_elu_brute_force, check_feature_maps_linear_route,
              check_grad_finite_differences, check_grad_invariants]


@pytest.mark.parametrize("check", ALL_CHECKS, ids=lambda f: f.__name__)
def test_oracle_pin(check):
    check(ORACLE)


# --------------------------------------------------------------------------
# statistical pins
# --------------------------------------------------------------------------

def _softmax_rpe(q, k, v, b):
    """Eq. (1) with the additive bias of Eq. (6), raw kernel exp(q k^T + b_{j-i})."""
    n = q.shape[0]
    i = np.arange(n)[:, None]
    j = np.arange(n)[None, :]
    logits = q @ k.T + b[j - i + n - 1]
    logits -= logits.max(axis=1, keepdims=True)
    p = np.exp(logits)
    p /= p.sum(axis=1, keepdims=True)
    return p @ v


def _sphere(rng, n, d, R):
    x = rng.standard_normal((n, d))
    return R * x / np.linalg.norm(x, axis=1, keepdims=True)


@pytest.mark.parametrize("R", [0.5, 1.0])
def test_softmax_limit(R):
    """As m grows, Eq. (10) with PRF approaches softmax attention with RPE.

    Mirrors the paper's simulation for Theorem 3 (queries and keys on a sphere
    of radius R, Gaussian features).  Monte-Carlo error must fall like
    m^(-1/2) and be small at large m for small R.
    """
    rng = np.random.default_rng(22)
    n, d = 32, 16
    q = _sphere(rng, n, d, R)
    k = _sphere(rng, n, d, R)
    v = rng.standard_normal((n, d))
    b = rng.standard_normal(2 * n - 1) * 0.5
    ref = _softmax_rpe(q, k, v, b)
    ms = [2 ** 8, 2 ** 10, 2 ** 12, 2 ** 14, 2 ** 16]
    errs = []
    for m in ms:
        e = []
        for s in range(16):
            W = np.random.default_rng([22, m, s]).standard_normal((1, m, d))
            z, _ = ORACLE.attention(q[None, None], k[None, None], v[None, None], b[None], W)
            e.append(np.mean(np.linalg.norm(z[0, 0] - ref, axis=1) / np.linalg.norm(ref, axis=1)))
        errs.append(np.mean(e))
    slope = np.polyfit(np.log(ms), np.log(errs), 1)[0]
    assert -0.6 < slope < -0.4, (slope, errs)
    if R == 0.5:
        assert errs[-1] < 0.02, errs


def test_denominator_unbiased():
    """E_W[den_i] = sum_j c_{j-i} exp(q_i k_j^T) (the PRF variance lemma's unbiasedness (Section 3.3), summed)."""
    rng = np.random.default_rng(23)
    n, d, m, T = 12, 8, 64, 400
    q = _sphere(rng, n, d, 0.8)
    k = _sphere(rng, n, d, 0.8)
    v = rng.standard_normal((n, d))
    b = rng.standard_normal(2 * n - 1) * 0.5
    i = np.arange(n)[:, None]
    j = np.arange(n)[None, :]
    exact = (np.exp(b[j - i + n - 1]) * np.exp(q @ k.T)).sum(axis=1)
    dens = []
    for s in range(T):
        W = np.random.default_rng([23, s]).standard_normal((1, m, d))
        _, den = ORACLE.attention(q[None, None], k[None, None], v[None, None], b[None], W)
        dens.append(den[0, 0])
    dens = np.array(dens)
    zscore = (dens.mean(0) - exact) / (dens.std(0, ddof=1) / math.sqrt(T))
    assert np.all(np.abs(zscore) < 4.0), zscore


@pytest.mark.parametrize("wid", [1, 2, 3, 4, 5])
def test_denominator_positive_on_workloads(wid):
    """den_i > 0 for sampled rows of every workload (phi > 0, c >= 0, c_0 > 0)."""
    d = synth.make(wid, heads=min(2, synth.WORKLOADS[wid].H))
    q, k, v, b, W = d["q"], d["k"], d["v"], d["b"], d["W"]
    n = q.shape[2]
    rows = [(q.shape[0] - 1, h, i) for h in range(q.shape[1]) for i in (0, 1, n // 2, n - 1)]
    z, den = ORACLE.attention_rows(q, k, v, b, W, rows)
    assert np.all(den > 0) and np.all(np.isfinite(z))
