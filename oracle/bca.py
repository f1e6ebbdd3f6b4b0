"""Oracle for the circulant / block-circulant layer (test infrastructure; see ``oracle/__init__``).

Paper: Memory-Efficient Training with In-Place FFT Implementation (arXiv 2511.01385),
Sec. 3.3 "FFT based Model Training via Circulant Matrix".

Definitions
-----------
* A p x p circulant matrix is fixed by its first column c (Sec. 3.3):
  C[m, r] = c[(m - r) mod p].  Then (C x)[m] = sum_r c[(m-r) mod p] x[r],
  the circular convolution c (*) x, which Eq. (4) evaluates as
  IFFT(FFT(c) . FFT(x)).
* Block-circulant weights (Sec. 3.3, last paragraph; block size p): a
  d_out x d_in matrix W made of q x kb circulant blocks, q = d_out/p,
  kb = d_in/p.  Block (i, j) has first column c[i, j, :] and maps input
  segment x[j*p:(j+1)*p] to output segment y[i*p:(i+1)*p].  Parameters are
  stored c[q][kb][p], i outermost.
* The layer acts on token rows: y[t] = W x[t], x of shape (T, d_in).
* Gradients (Eq. (5)), for upstream gradient g = dL/dy of shape (T, d_out):
  dx[t] = W^T g[t], i.e. IFFT(conj(FFT(c)) . FFT(g)) per block;
  dc[i, j, r] = sum_t sum_m g[t, i*p+m] * x[t, j*p + ((m - r) mod p)], the
  circular cross-correlation, i.e. IFFT(conj(FFT(x)) . FFT(g)) per block,
  summed over tokens (c is shared by all tokens).

The layer's parameters enter the library as packed spectra of the first
columns; :func:`effective_c` maps them back to the time-domain c that the
dense definitions use.

Two routes, both float64: ``*_dense`` builds W explicitly (the definition);
``*_spectral`` follows Eqs. (4)-(5) with the oracle's own DFT.  Element-wise
direct sums (``*_entries``) evaluate single outputs for sampled checks of large
layers.
"""

from __future__ import annotations

import numpy as np

from . import rdfft as _rd

__all__ = [
    "circulant",
    "block_circulant",
    "effective_c",
    "forward_dense",
    "backward_dense",
    "forward_spectral",
    "backward_spectral",
    "forward_entries",
    "dx_entries",
    "dc_entries",
]


def _shape(d_in: int, d_out: int, p: int):
    if p < 1 or d_in % p or d_out % p:
        # Table 1 marks block sizes that do not divide the width "N/A"
        raise ValueError(f"block size {p} must divide d_in={d_in} and d_out={d_out}")
    return d_out // p, d_in // p


def circulant(c: np.ndarray) -> np.ndarray:
    """C[m, r] = c[(m - r) mod p]: the circulant matrix whose first column is c."""
    c = np.asarray(c, dtype=np.float64)
    p = c.shape[-1]
    idx = (np.arange(p)[:, None] - np.arange(p)[None, :]) % p
    return c[..., idx]


def block_circulant(c: np.ndarray) -> np.ndarray:
    """W of shape (q*p, kb*p) with block (i, j) = circulant(c[i, j])."""
    c = np.asarray(c, dtype=np.float64)
    q, kb, p = c.shape
    w = np.empty((q * p, kb * p), dtype=np.float64)
    for i in range(q):
        for j in range(kb):
            w[i * p : (i + 1) * p, j * p : (j + 1) * p] = circulant(c[i, j])
    return w


def effective_c(c_spectra: np.ndarray, q: int, kb: int, p: int) -> np.ndarray:
    """Time-domain first columns represented by packed spectra c_spectra[q][kb][p]."""
    s = np.asarray(c_spectra, dtype=np.float64).reshape(q * kb, p)
    return _rd.rdfft_inverse(s).reshape(q, kb, p)


def forward_dense(x: np.ndarray, c: np.ndarray) -> np.ndarray:
    """y[t] = W x[t] (Sec. 3.3, y = C x, block-circulant W)."""
    x = np.asarray(x, dtype=np.float64)
    return x @ block_circulant(c).T


def backward_dense(x: np.ndarray, c: np.ndarray, g: np.ndarray):
    """(dx, dc) for L with dL/dy = g: dx = g W, and dc from dW = g^T x through the tied weights.

    W[i*p+m, j*p+r] = c[i, j, (m-r) mod p], so by the chain rule dc[i, j, s]
    collects dW over the positions where (m - r) mod p == s.
    """
    x = np.asarray(x, dtype=np.float64)
    g = np.asarray(g, dtype=np.float64)
    c = np.asarray(c, dtype=np.float64)
    q, kb, p = c.shape
    dx = g @ block_circulant(c)
    dw = g.T @ x
    dc = np.zeros((q, kb, p), dtype=np.float64)
    m = np.arange(p)
    for i in range(q):
        for j in range(kb):
            blk = dw[i * p : (i + 1) * p, j * p : (j + 1) * p]
            for s in range(p):
                dc[i, j, s] = blk[m, (m - s) % p].sum()
    return dx, dc


def _block_bins(a: np.ndarray, nblk: int, p: int) -> np.ndarray:
    """Spectra of each p-segment of each row: shape (T, nblk, p/2+1)."""
    t = a.shape[0]
    return _rd.dft_bins(a.reshape(t * nblk, p)).reshape(t, nblk, p // 2 + 1)


def forward_spectral(x: np.ndarray, c_spectra: np.ndarray, d_out: int, p: int) -> np.ndarray:
    """Eq. (4) per block: y_i = IFFT( sum_j FFT(c_ij) . FFT(x_j) )."""
    x = np.asarray(x, dtype=np.float64)
    q, kb = _shape(x.shape[1], d_out, p)
    cb = _rd.unpack_pairs(np.asarray(c_spectra, dtype=np.float64).reshape(q * kb, p))
    cb = cb.reshape(q, kb, p // 2 + 1)
    xb = _block_bins(x, kb, p)
    yb = np.einsum("ijk,tjk->tik", cb, xb)
    t = x.shape[0]
    return _rd.idft_from_bins(yb.reshape(t * q, -1), p).reshape(t, q * p)


def backward_spectral(x: np.ndarray, c_spectra: np.ndarray, g: np.ndarray, p: int):
    """Eq. (5) per block: dx_j = IFFT(sum_i conj(C_ij) G_i); dc_ij = IFFT(sum_t conj(X_tj) G_ti)."""
    x = np.asarray(x, dtype=np.float64)
    g = np.asarray(g, dtype=np.float64)
    q, kb = _shape(x.shape[1], g.shape[1], p)
    cb = _rd.unpack_pairs(np.asarray(c_spectra, dtype=np.float64).reshape(q * kb, p))
    cb = cb.reshape(q, kb, p // 2 + 1)
    xb = _block_bins(x, kb, p)
    gb = _block_bins(g, q, p)
    t = x.shape[0]
    dxb = np.einsum("ijk,tik->tjk", np.conj(cb), gb)
    dx = _rd.idft_from_bins(dxb.reshape(t * kb, -1), p).reshape(t, kb * p)
    dcb = np.einsum("tjk,tik->ijk", np.conj(xb), gb)
    dc = _rd.idft_from_bins(dcb.reshape(q * kb, -1), p).reshape(q, kb, p)
    return dx, dc


def forward_entries(x: np.ndarray, c: np.ndarray, entries) -> np.ndarray:
    """y[t, i*p+m] = sum_j sum_r c[i, j, (m-r) mod p] * x[t, j*p+r], for (t, i, m) in ``entries``."""
    x = np.asarray(x, dtype=np.float64)
    c = np.asarray(c, dtype=np.float64)
    q, kb, p = c.shape
    r = np.arange(p)
    out = []
    for t, i, m in entries:
        xs = x[t].reshape(kb, p)
        out.append(float((c[i][:, (m - r) % p] * xs).sum()))
    return np.array(out)


def dx_entries(g: np.ndarray, c: np.ndarray, entries) -> np.ndarray:
    """dx[t, j*p+r] = sum_i sum_m c[i, j, (m-r) mod p] * g[t, i*p+m], for (t, j, r) in ``entries``."""
    g = np.asarray(g, dtype=np.float64)
    c = np.asarray(c, dtype=np.float64)
    q, kb, p = c.shape
    m = np.arange(p)
    out = []
    for t, j, r in entries:
        gs = g[t].reshape(q, p)
        out.append(float((c[:, j][:, (m - r) % p] * gs).sum()))
    return np.array(out)


def dc_entries(x: np.ndarray, g: np.ndarray, q: int, kb: int, p: int, entries) -> np.ndarray:
    """dc[i, j, s] = sum_t sum_m g[t, i*p+m] * x[t, j*p + ((m-s) mod p)], for (i, j, s) in ``entries``."""
    x = np.asarray(x, dtype=np.float64)
    g = np.asarray(g, dtype=np.float64)
    m = np.arange(p)
    out = []
    for i, j, s in entries:
        gi = g[:, i * p : (i + 1) * p]
        xj = x[:, j * p : (j + 1) * p][:, (m - s) % p]
        out.append(float((gi * xj).sum()))
    return np.array(out)
