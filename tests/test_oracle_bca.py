"""Pins for the block-circulant oracle (CPU only).

The dense definition (Sec. 3.3, y = C x with C fixed by its first column) is pinned
by a hand-worked circulant, the identity and circular-shift special cases, the
p = 1 case (a plain matrix product) and explicit convolution sums; the gradients
(Eq. (5)) by the adjoint identity, the exact directional derivative in c and
float64 finite differences; the spectral route (Eqs. (4)-(5)) and the element
samplers by agreement with the pinned dense route.
"""

import os

import numpy as np
import pytest

from oracle import bca
from oracle import rdfft as rd

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _spectra(c):
    q, kb, p = c.shape
    return rd.rdfft_forward(c.reshape(q * kb, p)).reshape(q, kb, p)


def _problem(seed, t, d_in, d_out, p):
    rng = np.random.default_rng(seed)
    q, kb = d_out // p, d_in // p
    return rng.standard_normal((t, d_in)), rng.standard_normal((q, kb, p)), rng.standard_normal((t, d_out))


def test_hand_worked_circulant():
    vals = {}
    with open(os.path.join(GOLDEN, "circulant_p4_hand.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                k, *v = line.split()
                vals[k] = np.array([float(a) for a in v])
    c = vals["c"].reshape(1, 1, 4)
    x = vals["x"].reshape(1, 4)
    np.testing.assert_allclose(bca.forward_dense(x, c)[0], vals["y"], atol=1e-14)
    np.testing.assert_allclose(bca.forward_spectral(x, _spectra(c), 4, 4)[0], vals["y"], atol=1e-13)
    np.testing.assert_array_equal(bca.circulant(vals["c"])[:, 0], vals["c"])  # first column is c


def test_circulant_is_circular_convolution():
    rng = np.random.default_rng(5)
    p = 6
    c, x = rng.standard_normal(p), rng.standard_normal(p)
    want = [sum(c[(m - r) % p] * x[r] for r in range(p)) for m in range(p)]
    np.testing.assert_allclose(bca.circulant(c) @ x, want, atol=1e-14)


@pytest.mark.parametrize("p", [4, 8, 32])
def test_identity_blocks(p):
    d = 3 * p
    rng = np.random.default_rng(p)
    x = rng.standard_normal((5, d))
    c = np.zeros((3, 3, p))
    for i in range(3):
        c[i, i, 0] = 1.0
    np.testing.assert_allclose(bca.forward_dense(x, c), x, atol=1e-14)
    np.testing.assert_allclose(bca.forward_spectral(x, _spectra(c), d, p), x, atol=1e-12)


@pytest.mark.parametrize("s", [1, 3, 7])
def test_first_column_impulse_is_circular_shift(s):
    """c = e_s gives y[m] = x[(m - s) mod p]; a first-row reading would shift the other way."""
    p = 16
    rng = np.random.default_rng(s)
    x = rng.standard_normal((4, p))
    c = np.zeros((1, 1, p))
    c[0, 0, s] = 1.0
    want = np.roll(x, s, axis=1)
    np.testing.assert_allclose(bca.forward_dense(x, c), want, atol=1e-14)
    np.testing.assert_allclose(bca.forward_spectral(x, _spectra(c), p, p), want, atol=1e-12)


def test_block_size_one_is_plain_matmul():
    rng = np.random.default_rng(9)
    x = rng.standard_normal((6, 5))
    c = rng.standard_normal((3, 5, 1))
    np.testing.assert_allclose(bca.forward_dense(x, c), x @ c[:, :, 0].T, atol=1e-13)


def test_block_placement():
    """Block (i, j) maps input segment j to output segment i."""
    p = 4
    x = np.zeros((1, 3 * p))
    x[0, 2 * p] = 1.0  # impulse at the start of input segment 2
    c = np.zeros((2, 3, p))
    c[1, 2] = [1.0, 2.0, 3.0, 4.0]
    y = bca.forward_dense(x, c)[0]
    np.testing.assert_allclose(y[:p], 0)
    np.testing.assert_allclose(y[p:], [1, 2, 3, 4])


@pytest.mark.parametrize("shape", [(7, 8, 8, 4), (5, 12, 8, 4), (3, 64, 128, 16)])
def test_spectral_matches_dense(shape):
    t, d_in, d_out, p = shape
    x, c, g = _problem(sum(shape), t, d_in, d_out, p)
    s = _spectra(c)
    np.testing.assert_allclose(bca.effective_c(s, *c.shape), c, atol=1e-13)
    np.testing.assert_allclose(bca.forward_spectral(x, s, d_out, p), bca.forward_dense(x, c), atol=1e-11)
    dx_d, dc_d = bca.backward_dense(x, c, g)
    dx_s, dc_s = bca.backward_spectral(x, s, g, p)
    np.testing.assert_allclose(dx_s, dx_d, atol=1e-11)
    np.testing.assert_allclose(dc_s, dc_d, atol=1e-10)


@pytest.mark.parametrize("route", ["dense", "spectral"])
def test_adjoint_and_directional_derivative(route):
    t, d_in, d_out, p = 6, 16, 24, 8
    x, c, g = _problem(21, t, d_in, d_out, p)
    rng = np.random.default_rng(22)
    dcdir = rng.standard_normal(c.shape)
    if route == "dense":
        dx, dc = bca.backward_dense(x, c, g)
        fwd = lambda xx, cc: bca.forward_dense(xx, cc)  # noqa: E731
    else:
        dx, dc = bca.backward_spectral(x, _spectra(c), g, p)
        fwd = lambda xx, cc: bca.forward_spectral(xx, _spectra(cc), d_out, p)  # noqa: E731
    # <W x, g> = <x, W^T g>
    np.testing.assert_allclose((fwd(x, c) * g).sum(), (x * dx).sum(), rtol=1e-12)
    # y is linear in c, so <dc, dir> = <g, y(c = dir)> exactly
    np.testing.assert_allclose((dc * dcdir).sum(), (g * fwd(x, dcdir)).sum(), rtol=1e-12)


def test_finite_differences_tiny():
    t, d, p = 3, 8, 4
    x, c, g = _problem(33, t, d, d, p)
    dx, dc = bca.backward_dense(x, c, g)
    loss = lambda xx, cc: float((bca.forward_dense(xx, cc) * g).sum())  # noqa: E731
    h = 1e-6
    num_dc = np.zeros_like(c)
    for idx in np.ndindex(c.shape):
        e = np.zeros_like(c)
        e[idx] = h
        num_dc[idx] = (loss(x, c + e) - loss(x, c - e)) / (2 * h)
    np.testing.assert_allclose(dc, num_dc, atol=1e-7)
    num_dx = np.zeros_like(x)
    for idx in np.ndindex(x.shape):
        e = np.zeros_like(x)
        e[idx] = h
        num_dx[idx] = (loss(x + e, c) - loss(x - e, c)) / (2 * h)
    np.testing.assert_allclose(dx, num_dx, atol=1e-7)


def test_entry_samplers_match_dense():
    t, d_in, d_out, p = 4, 16, 24, 8
    x, c, g = _problem(44, t, d_in, d_out, p)
    y = bca.forward_dense(x, c)
    dx, dc = bca.backward_dense(x, c, g)
    ent = [(0, 0, 0), (3, 2, 7), (2, 1, 5)]
    np.testing.assert_allclose(bca.forward_entries(x, c, ent), [y[a, b * p + m] for a, b, m in ent], atol=1e-12)
    ent = [(1, 1, 2), (0, 0, 7), (3, 1, 0)]
    np.testing.assert_allclose(bca.dx_entries(g, c, ent), [dx[a, b * p + r] for a, b, r in ent], atol=1e-12)
    ent = [(2, 1, 3), (0, 0, 0), (1, 1, 7)]
    np.testing.assert_allclose(bca.dc_entries(x, g, 3, 2, p, ent), [dc[i, j, s] for i, j, s in ent], atol=1e-12)


def test_block_size_must_divide():
    x = np.zeros((2, 12))
    with pytest.raises(ValueError):
        bca.forward_spectral(x, np.zeros((1, 1, 8)), 8, 8)


def test_impulse_spectra_helper_matches_oracle():
    """The closed-form impulse spectra that the GPU layer tests feed the library equal the oracle's
    packed transform of the impulse columns (zero blocks stay zero)."""
    from tests._helpers import impulse_spectra

    for p in (2, 4, 64, 256):
        shifts = np.array([[0, 1, -1], [p - 1, p // 2, 3 % p]])
        got = impulse_spectra(shifts, p)
        for i in range(shifts.shape[0]):
            for j in range(shifts.shape[1]):
                col = np.zeros(p)
                if shifts[i, j] >= 0:
                    col[shifts[i, j]] = 1.0
                np.testing.assert_allclose(got[i, j], rd.rdfft_forward(col[None])[0], atol=1e-12)
