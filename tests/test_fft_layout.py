"""Host-side checks of the index and constant algebra the FFT header relies on.

The transform itself is checked on the GPU against the oracle; these tests pin
the pieces of fft.hpp that are pure index or constant arithmetic, so that a
change to them fails here before it reaches a GPU:

* the tangent table of the fused twiddle butterflies equals tan(2 pi e / 64),
  and every constant twiddle w = exp(+-2 pi i K / NN) is i^q * c (1 + i t) with
  |t| <= 1 under the header's split of the angle;
* the padded LDS address of every butterfly position is pad(base) plus a
  constant (the affine addressing option), for every pass of every
  transform length and radix the library instantiates;
* the order in which a pass reads its inputs is a permutation.
"""
import cmath
import math
import os
import re

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
FFT_HPP = os.path.join(os.path.dirname(HERE), "paper_2106_12566_amd", "csrc", "fft.hpp")


def header_text():
    return open(FFT_HPP).read()


def tan_table():
    m = re.search(r"constexpr float tan64\(int e\) \{\s*constexpr float t\[9\] = \{([^}]*)\}", header_text())
    assert m, "tan64 table not found in fft.hpp"
    return [float(v.strip().rstrip("f")) for v in m.group(1).split(",")]


def test_tangent_table():
    t = tan_table()
    assert len(t) == 9
    for e, v in enumerate(t):
        assert v == pytest.approx(math.tan(2 * math.pi * e / 64), rel=1e-7, abs=1e-9), e
    assert t[0] == 0.0 and t[8] == 1.0


def split(e):
    """The header's split of exp(+2 pi i e / 64): quarter turns qt and residual er in [-8, 8)."""
    qt = ((e + 8) // 16) % 4
    er = e - 16 * ((e + 8) // 16)
    return qt, er


@pytest.mark.parametrize("nn", [2, 4, 8, 16, 32, 64])
@pytest.mark.parametrize("inv", [False, True])
def test_twiddle_split(nn, inv):
    t = tan_table()
    for K in range(-nn, 2 * nn):
        k = ((K % nn + nn) % nn) * (64 // nn)
        e = k if inv else (64 - k) % 64
        qt, er = split(e)
        assert -8 <= er < 8
        tt = t[er] if er >= 0 else -t[-er]
        c = math.cos(2 * math.pi * er / 64)
        w = (1j ** qt) * c * complex(1.0, tt)
        want = cmath.exp((1 if inv else -1) * 2j * math.pi * K / nn)
        assert abs(w - want) < 1e-6, (nn, K, inv)


def pass_positions(log2n, log2r):
    """(pass, butterfly base, stride, radix) of every butterfly of the transform
    of length 2^log2n at 2^log2r values per thread, as the header's passes run."""
    lr = min(log2n, log2r)
    R, N = 1 << lr, 1 << log2n
    T = N // R
    P = 1 if lr == 0 else (log2n + lr - 1) // lr
    for p in range(P):
        lrp = lr if p + 1 < P else log2n - lr * (P - 1)
        RP = 1 << lrp
        U = R // RP
        L = N >> (lr * p)
        SP = L >> lrp
        for tau in range(T):
            for u in range(U):
                b = tau + T * u
                yield p, (b // SP) * L + b % SP, SP, RP, lr


# LDS layout modes of the header (its PAD parameter): (shift, slots per group)
PAD_MODES = {1: (3, 1), 2: (4, 1), 3: (4, 2), 4: (5, 1)}


@pytest.mark.parametrize("log2r", [3, 4])
def test_affine_padded_addresses(log2r):
    count = 0
    for log2n in range(1, 14):
        for p, base, SP, RP, lr in pass_positions(log2n, log2r):
            sh = lr if lr > 0 else 1

            def pad(a):
                return a + (a >> sh)

            for r in range(RP):
                c = SP * r
                assert pad(base + c) == pad(base) + pad(c), (log2n, log2r, p, base, r)
                count += 1
    assert count > 50000


@pytest.mark.parametrize("log2n,log2r,mode", [(12, 3, 3), (12, 4, 3), (12, 3, 2), (12, 3, 1), (12, 4, 4)])
def test_affine_padded_addresses_of_the_other_layouts(log2n, log2r, mode):
    """Two padding slots per 16 positions (the layout of the 4096-point transforms at 8 and 16
    values per thread) and the other modes: every butterfly's padded addresses are still
    pad(base) + pad(c), and the layout is one-to-one."""
    sh, mult = PAD_MODES[mode]

    def pad(a):
        return a + mult * (a >> sh)

    for p, base, SP, RP, lr in pass_positions(log2n, log2r):
        for r in range(RP):
            c = SP * r
            assert pad(base + c) == pad(base) + pad(c), (log2n, log2r, mode, p, base, r)
    n = 1 << log2n
    assert len({pad(a) for a in range(n)}) == n


def read_order(rp, j):
    a = rp // 4 if rp >= 4 else 1
    return (j // 4) + a * (j % 4) if rp >= 4 else j


@pytest.mark.parametrize("rp", [1, 2, 4, 8, 16, 32, 64])
def test_read_order_is_a_permutation(rp):
    assert sorted(read_order(rp, j) for j in range(rp)) == list(range(rp))
    # the first four reads are the inputs of the first radix-4 sub-DFT
    if rp >= 4:
        assert [read_order(rp, j) for j in range(4)] == [(rp // 4) * i for i in range(4)]


def test_header_forms_match():
    """The header states the same read order and padded-offset formulas as checked above."""
    text = re.sub(r"\s+", " ", header_text())
    assert "return RP >= 4 ? (j / 4) + A * (j % 4) : j;" in text
    assert "constexpr int A = RP >= 4 ? RP / 4 : 1;" in text
    assert "static constexpr int pad(int a) { return a + PM * (a >> PSH); }" in text
    assert "static constexpr int PSH = PAD == 0 ? (LR > 0 ? LR : 1) : (PAD == 1 ? 3 : (PAD == 4 ? 5 : 4));" in text
    assert "static constexpr int PM = PAD == 3 ? 2 : 1;" in text
    assert "constexpr int qt = ((e + 8) / 16) % 4;" in text
    assert "constexpr int er = e - 16 * (((e + 8) / 16));" in text
