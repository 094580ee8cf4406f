"""Plant plausible mistakes in copies of the oracle and show the pins catch them.

Each mutant is the oracle's own source with one textual change (a flipped
offset sign, an off-by-one index, a dropped term, a transposed operand, ...),
executed into a throw-away module on the CPU.  The pins of
``test_oracle_pins.py`` are re-run on it and at least one must fail.
"""
import inspect
import types

import numpy as np
import pytest

import oracle.krpe_oracle as ORACLE_SRC
from test_oracle_pins import ALL_CHECKS

MUTANTS = {
    "offset_sign_flipped": ("c = np.exp(b[h][cols - rows + n - 1])", "c = np.exp(b[h][rows - cols + n - 1])"),
    "offset_off_by_one": ("c = np.exp(b[h][cols - rows + n - 1])", "c = np.exp(b[h][(cols - rows + n) % (2 * n - 1)])"),
    "norm_term_dropped": ("return np.exp(proj - half_sq) / np.sqrt(m)", "return np.exp(proj) / np.sqrt(m)"),
    "norm_term_not_halved": ("half_sq = 0.5 * np.sum(x * x, axis=-1, keepdims=True)", "half_sq = np.sum(x * x, axis=-1, keepdims=True)"),
    "sqrt_m_dropped": ("return np.exp(proj - half_sq) / np.sqrt(m)", "return np.exp(proj - half_sq)"),
    "bias_not_exponentiated": ("c = np.exp(b[h][cols - rows + n - 1])", "c = b[h][cols - rows + n - 1]"),
    "query_key_swapped": ("mt = c * (fq[i0:i1] @ fk.T)", "mt = c * (fk[i0:i1] @ fq.T)"),
    "bias_left_out_of_denominator": ("dd = mt.sum(axis=1)", "dd = (fq[i0:i1] @ fk.T).sum(axis=1)"),
    "values_replaced_by_keys": ("num = mt @ v[beta, h]", "num = mt @ k[beta, h]"),
    "toeplitz_transposed": ("out[:, h] = a[:, h] @ C.T", "out[:, h] = a[:, h] @ C"),
    "toeplitz_matrix_sign": ("return np.exp(b_h[j - i + n - 1])", "return np.exp(b_h[i - j + n - 1])"),
    "toeplitz_rows_window_reversed": ("c_row = np.exp(b[:, n - 1 - i:2 * n - 1 - i])",
                                      "c_row = np.exp(b[:, i:i + n][:, ::-1])"),
    "toeplitz_rows_window_off_by_one": ("c_row = np.exp(b[:, n - 1 - i:2 * n - 1 - i])",
                                        "c_row = np.exp(b[:, n - i:2 * n - i])"),
    "rows_offset_sign": ("c = np.exp(b[h][np.arange(n) - i + n - 1])", "c = np.exp(b[h][i - np.arange(n) + n - 1])"),
    "rows_wrong_head_features": ("cache[(beta, h)] = fmap(k[beta, h], W[h])", "cache[(beta, h)] = fmap(k[beta, h], W[0])"),
    "nprf_keys_not_normalised": ("        q, k = normalize_rows(q), normalize_rows(k)\n    Bn", "        q = normalize_rows(q)\n    Bn"),
    "nprf_squared_norm": ("return np.divide(x, norm, out=np.zeros_like(x), where=norm > 0)", "return np.divide(x, norm * norm, out=np.zeros_like(x), where=norm > 0)"),
    "nprf_ignored": ("    if nprf:\n        q, k = normalize_rows(q), normalize_rows(k)\n    Bn", "    Bn"),
    "trf_norm_sign": ("amp = np.exp(0.5 * np.sum(x * x, axis=-1, keepdims=True)) / np.sqrt(m)",
                      "amp = np.exp(-0.5 * np.sum(x * x, axis=-1, keepdims=True)) / np.sqrt(m)"),
    "trf_cos_twice": ("return np.concatenate([amp * np.sin(proj), amp * np.cos(proj)], axis=-1)",
                      "return np.concatenate([amp * np.cos(proj), amp * np.cos(proj)], axis=-1)"),
    "trf_sqrt_2m": ("amp = np.exp(0.5 * np.sum(x * x, axis=-1, keepdims=True)) / np.sqrt(m)",
                    "amp = np.exp(0.5 * np.sum(x * x, axis=-1, keepdims=True)) / np.sqrt(2 * m)"),
    "elu_plus_one_dropped": ("return np.where(x > 0, x + 1.0, np.exp(np.minimum(x, 0.0)))",
                             "return np.where(x > 0, x, np.exp(np.minimum(x, 0.0)) - 1.0)"),
    "grad_den_term_dropped": ("dA = dN @ v[beta, h].T + dden[:, None]", "dA = dN @ v[beta, h].T"),
    "grad_keys_not_transposed": ("dfk = dK.T @ fq", "dfk = dK @ fq"),
    "grad_db_chain_missing": ("db = np.where(cfin, db * np.exp(np.where(cfin, b, 0.0)), 0.0)",
                              "db = np.where(cfin, db, 0.0)"),
    "grad_diagonal_sign": ("db[h, t + n - 1] += np.trace(dC, offset=t)", "db[h, t + n - 1] += np.trace(dC, offset=-t)"),
    "grad_norm_term_dropped": ("dx = P @ W[h] - x * P.sum(axis=1, keepdims=True)", "dx = P @ W[h]"),
    "grad_nprf_projection_dropped": ("dx = np.divide(dx - x * np.sum(x * dx, axis=1, keepdims=True), nrm,",
                                     "dx = np.divide(dx, nrm,"),
    "elu_branch_flipped": ("return np.where(x > 0, x + 1.0, np.exp(np.minimum(x, 0.0)))",
                           "return np.where(x >= 0, np.exp(np.minimum(x, 0.0)), x + 1.0)"),
}


def _mutant(old, new):
    src = inspect.getsource(ORACLE_SRC)
    assert src.count(old) == 1, f"mutation anchor not found exactly once: {old!r}"
    mod = types.ModuleType("oracle_mutant")
    exec(compile(src.replace(old, new), "<oracle-mutant>", "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name):
    mod = _mutant(*MUTANTS[name])
    caught = []
    with np.errstate(all="ignore"):
        for check in ALL_CHECKS:
            try:
                check(mod)
            except Exception:      # AssertionError or a numerical blow-up
                caught.append(check.__name__)
    assert caught, f"no pin detects mutant {name}"
