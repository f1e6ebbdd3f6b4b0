"""Pins for the rdFFT oracle (CPU only).

Each check ties ``oracle.rdfft`` to something other than itself: hand-worked and
closed-form spectra (Sec. 3.1 Eq. (1)), Theorem 1 (conjugate symmetry; DC and
Nyquist bins real), Parseval, linearity, the shift theorem, the exact
round trip, the paper's own index example for its halfcomplex layout
(Sec. 4.1, Proposition 1 example), and the direct O(n^2) definition against the
library FFT route.  A dropped term, a flipped exponent sign, a swapped DC /
Nyquist slot, a transposed (re, im) pair or a wrong 1/n fails at least one.
"""

import os

import numpy as np
import pytest

from oracle import rdfft as rd

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
METHODS = ["direct", "fft"]
SIZES = [2, 4, 8, 16, 64, 256, 1024]
# even lengths whose half has factors 3 and 5 (the mixed-radix rows)
MIXED = [6, 10, 12, 30, 48, 90, 750]


def _read_golden(name):
    out = {}
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, *vals = line.split()
            out[key] = np.array([float(v) for v in vals])
    return out


@pytest.mark.parametrize("method", METHODS)
@pytest.mark.parametrize("name", ["rdfft_ramp_n8.txt", "rdfft_n4_hand.txt"])
def test_golden_worked_examples(name, method):
    g = _read_golden(name)
    got = rd.rdfft_forward(g["input"], method=method)[0]
    np.testing.assert_allclose(got, g["packed"], rtol=0, atol=1e-12)
    back = rd.rdfft_inverse(g["packed"], method=method)[0]
    np.testing.assert_allclose(back, g["input"], rtol=0, atol=1e-12)


@pytest.mark.parametrize("method", METHODS)
@pytest.mark.parametrize("n", SIZES + MIXED)
def test_closed_forms(n, method):
    m = np.arange(n)
    # unit impulse -> every bin is 1
    e0 = np.zeros(n)
    e0[0] = 1
    want = np.zeros(n)
    want[0] = want[1] = 1
    want[2::2] = 1
    np.testing.assert_allclose(rd.rdfft_forward(e0, method)[0], want, atol=1e-12)
    # constant -> DC only
    want = np.zeros(n)
    want[0] = n
    np.testing.assert_allclose(rd.rdfft_forward(np.ones(n), method)[0], want, atol=1e-9)
    # alternating sign -> Nyquist only, in slot 1
    want = np.zeros(n)
    want[1] = n
    np.testing.assert_allclose(rd.rdfft_forward((-1.0) ** m, method)[0], want, atol=1e-9)
    # ramp: Y_0 = n(n+1)/2, Y_{n/2} = -n/2, Y_k = -n/2 + i (n/2) cot(pi k / n)
    want = np.zeros(n)
    want[0] = n * (n + 1) / 2
    want[1] = -n / 2
    for k in range(1, n // 2):
        want[2 * k] = -n / 2
        want[2 * k + 1] = (n / 2) / np.tan(np.pi * k / n)
    np.testing.assert_allclose(rd.rdfft_forward(m + 1.0, method)[0], want, rtol=1e-12, atol=1e-9 * n)
    for k0 in sorted({1, n // 4, n // 2 - 1} - {0}):
        if not 0 < k0 < n // 2:
            continue
        # cosine at bin k0 -> Re Y_k0 = n/2
        want = np.zeros(n)
        want[2 * k0] = n / 2
        got = rd.rdfft_forward(np.cos(2 * np.pi * k0 * m / n), method)[0]
        np.testing.assert_allclose(got, want, atol=1e-9)
        # sine at bin k0 -> Im Y_k0 = -n/2 (forward exponent is negative)
        want = np.zeros(n)
        want[2 * k0 + 1] = -n / 2
        got = rd.rdfft_forward(np.sin(2 * np.pi * k0 * m / n), method)[0]
        np.testing.assert_allclose(got, want, atol=1e-9)


@pytest.mark.parametrize("method", METHODS)
@pytest.mark.parametrize("n", [4, 8, 64, 512, 6, 30, 90])
def test_inverse_of_unit_slots(n, method):
    """Each packed slot's inverse is a known real sinusoid (Eq. (1) with Y_{n-k} = conj Y_k)."""
    m = np.arange(n)
    eye = np.eye(n)
    x = rd.rdfft_inverse(eye, method)
    np.testing.assert_allclose(x[0], np.full(n, 1.0 / n), atol=1e-14)
    np.testing.assert_allclose(x[1], (-1.0) ** m / n, atol=1e-14)
    for k in range(1, n // 2):
        np.testing.assert_allclose(x[2 * k], 2 * np.cos(2 * np.pi * k * m / n) / n, atol=1e-13)
        np.testing.assert_allclose(x[2 * k + 1], -2 * np.sin(2 * np.pi * k * m / n) / n, atol=1e-13)


@pytest.mark.parametrize("n", SIZES + MIXED)
def test_theorem1_and_parseval(n):
    rng = np.random.default_rng(n)
    x = rng.standard_normal((3, n))
    bins = rd.dft_bins(x, method="direct")
    # Theorem 1: DC and Nyquist bins of a real row are real
    scale = np.abs(x).sum(axis=1)
    assert np.all(np.abs(bins[:, 0].imag) <= 1e-12 * scale)
    assert np.all(np.abs(bins[:, n // 2].imag) <= 1e-12 * scale)
    # conjugate symmetry: bin n-k of the full DFT equals conj of bin k
    full = np.fft.fft(x, axis=1)
    k = np.arange(1, n // 2)
    np.testing.assert_allclose(full[:, n - k], np.conj(full[:, k]), atol=1e-10)
    # Parseval on the packed form
    buf = rd.rdfft_forward(x, method="direct")
    energy = (buf[:, 0] ** 2 + buf[:, 1] ** 2 + 2 * (buf[:, 2:] ** 2).sum(axis=1)) / n
    np.testing.assert_allclose(energy, (x**2).sum(axis=1), rtol=1e-12)


@pytest.mark.parametrize("method", METHODS)
@pytest.mark.parametrize("n", [8, 64, 256])
def test_linearity_and_shift(n, method):
    rng = np.random.default_rng(7 + n)
    a, b = rng.standard_normal((2, n))
    fa, fb = rd.dft_bins(a, method), rd.dft_bins(b, method)
    np.testing.assert_allclose(rd.dft_bins(2.5 * a - 0.75 * b, method), 2.5 * fa - 0.75 * fb, atol=1e-10)
    for s in (1, 3, n // 2 + 1):
        shifted = np.roll(a, s)  # shifted[m] = a[(m - s) mod n]
        k = np.arange(n // 2 + 1)
        want = fa * np.exp(-2j * np.pi * k * s / n)
        np.testing.assert_allclose(rd.dft_bins(shifted, method), want, atol=1e-10)


@pytest.mark.parametrize("layout", ["pairs", "halfcomplex"])
@pytest.mark.parametrize("method", METHODS)
@pytest.mark.parametrize("n", SIZES + MIXED)
def test_round_trip_both_ways(n, method, layout):
    rng = np.random.default_rng(100 + n)
    x = rng.standard_normal((4, n))
    np.testing.assert_allclose(rd.rdfft_inverse(rd.rdfft_forward(x, method, layout), method, layout), x, atol=1e-12)
    buf = rng.standard_normal((4, n))  # any n reals are a valid packed spectrum
    np.testing.assert_allclose(rd.rdfft_forward(rd.rdfft_inverse(buf, method, layout), method, layout), buf, atol=1e-11)


@pytest.mark.parametrize("n", [2, 4, 16, 128, 1024] + MIXED)
def test_direct_definition_pins_library_route(n):
    rng = np.random.default_rng(3 * n)
    x = rng.standard_normal((5, n))
    np.testing.assert_allclose(rd.dft_bins(x, "fft"), rd.dft_bins(x, "direct"), atol=1e-10 * np.sqrt(n))
    buf = rng.standard_normal((5, n))
    np.testing.assert_allclose(rd.rdfft_inverse(buf, "fft"), rd.rdfft_inverse(buf, "direct"), atol=1e-12)


def test_sampled_bins_match_full_direct():
    rng = np.random.default_rng(11)
    x = rng.standard_normal((2, 256))
    ks = np.array([0, 1, 17, 64, 127, 128])
    np.testing.assert_allclose(rd.dft_bins(x, "direct", ks=ks), rd.dft_bins(x, "direct")[:, ks], atol=1e-12)


def test_pairs_slot_order():
    """Slot 0 holds DC and slot 1 Nyquist; bin k sits in (2k, 2k+1) as (re, im)."""
    bins = np.array([[10.0, 1 + 2j, 3 - 4j, 5 + 6j, -7.0]])  # n = 8
    np.testing.assert_array_equal(rd.pack_pairs(bins)[0], [10, -7, 1, 2, 3, -4, 5, 6])
    np.testing.assert_array_equal(rd.unpack_pairs(rd.pack_pairs(bins)), bins)


def test_halfcomplex_matches_paper_index_example():
    """Sec. 4.1, example after Proposition 1: in a 16-point buffer, bins 2 and 6 occupy the
    slot pairs (2, 14) and (6, 10)."""
    n = 16
    for k, partner in ((2, 14), (6, 10)):
        bins = np.zeros((1, n // 2 + 1), dtype=complex)
        bins[0, k] = 3.0 - 5.0j
        buf = rd.pack_halfcomplex(bins)[0]
        assert set(np.flatnonzero(buf)) == {k, partner}
        assert buf[k] == 3.0 and buf[partner] == -5.0


def test_odd_length_rejected():
    with pytest.raises(ValueError):
        rd.rdfft_forward(np.ones(7))
    with pytest.raises(ValueError):
        rd.rdfft_inverse(np.ones(9))
