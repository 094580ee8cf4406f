"""Input generator properties and the oracle regression fixture (CPU only)."""
import json
import os

import numpy as np
import pytest
import torch

import oracle
from paper_2106_12566_amd import synth

HERE = os.path.dirname(os.path.abspath(__file__))


def test_bf16_round_matches_torch():
    rng = np.random.default_rng(0)
    x = (rng.standard_normal(100000) * np.exp(rng.uniform(-20, 20, 100000))).astype(np.float32)
    # include exact ties to check round-half-to-even
    ties = np.array([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -(1.0 + 2 ** -8)], np.float32)
    x = np.concatenate([x, ties])
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    assert np.array_equal(synth.bf16_round(x), ref)
    bits = synth.bf16_bits(ref)
    assert np.array_equal(torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).float().numpy(), ref)


def test_generator_is_deterministic_and_shaped():
    a = synth.make(2, heads=2)
    b = synth.make(2, heads=2)
    for key in "qkvWb":
        assert np.array_equal(a[key], b[key])
    wl = synth.WORKLOADS[2]
    assert a["q"].shape == (wl.B, 2, wl.n, wl.d)
    assert a["W"].shape == (2, wl.m, wl.d)
    assert a["b"].shape == (2, 2 * wl.n - 1)


def test_orthogonal_features_blocks():
    rng = np.random.default_rng(3)
    W = synth.orthogonal_features(rng, 128, 64)
    for blk in (W[:64], W[64:]):
        u = blk / np.linalg.norm(blk, axis=1, keepdims=True)
        assert np.allclose(u @ u.T, np.eye(64), atol=1e-10)
    # chi_64 norms: mean about sqrt(63.5)
    assert 6.5 < np.linalg.norm(W, axis=1).mean() < 9.5


def test_bias_profiles():
    d5 = synth.make(5, heads=1)
    n = synth.WORKLOADS[5].n
    b = d5["b"][0]
    assert np.all(np.isneginf(b[n:])) and np.all(np.isfinite(b[:n]))
    d3 = synth.make(3, heads=1)
    b3 = d3["b"][0]
    n3 = synth.WORKLOADS[3].n
    assert b3[0] < -15 and b3[-1] < -15 and abs(b3[n3 - 1]) < 2
    assert np.all(synth.bf16_round(d3["q"]) == d3["q"])


def test_golden_regression():
    with open(os.path.join(HERE, "golden", "tiny_n128_rows.json")) as f:
        g = json.load(f)
    d = synth.make(1)
    rows = [(0, 0, i) for i in g["rows"]]
    z, den = oracle.attention_rows(d["q"], d["k"], d["v"], d["b"], d["W"], rows)
    assert np.allclose(z, np.array(g["z"]), rtol=1e-12, atol=1e-15)
    assert np.allclose(den, np.array(g["den"]), rtol=1e-12)
