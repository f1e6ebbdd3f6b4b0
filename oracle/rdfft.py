"""Oracle for the packed real-domain FFT (test infrastructure; see ``oracle/__init__``).

Paper: Memory-Efficient Training with In-Place FFT Implementation (arXiv 2511.01385).

What is computed
----------------
Forward (Sec. 3.1, Eq. (1)): for a real row x of even length n,

    Y_k = sum_{m=0}^{n-1} x_m * exp(-2*pi*i*k*m/n),   k = 0 .. n/2,

i.e. only the non-redundant half of the spectrum (Sec. 3.1, Theorem 1:
Y_{n-k} = conj(Y_k)).  Y_0 and Y_{n/2} are real (Sec. 4.1, "Squeeze N+2 into N"),
so the n/2+1 complex bins fit in n real slots.  The slot layout used by the
library ("pairs"):

    buf[0] = Y_0,  buf[1] = Y_{n/2},  buf[2k] = Re Y_k,  buf[2k+1] = Im Y_k  (1 <= k < n/2).

The paper's own figure-based layout ("halfcomplex", Sec. 4.1 "Memory Layout
Design": Re Y_k at slot k, Im Y_k at slot n-k, Y_0 at 0, Y_{n/2} at n/2) is
provided too, for interoperability tests.

Inverse (Sec. 3.1, Eq. (1), second half; the 1/N normalisation of Sec. 3.2):

    x_m = (1/n) * sum_{k=0}^{n-1} Y_k * exp(+2*pi*i*k*m/n),  with Y_{n-k} = conj(Y_k)

and Im Y_0 = Im Y_{n/2} = 0.  Any n reals are a valid packed spectrum, so the
inverse is the exact inverse map R^n -> R^n of the forward one.

Two evaluation routes, both float64:
* ``method="direct"``: the sums above written out (O(n^2) per row), with the
  exponent index k*m reduced mod n before forming the angle;
* ``method="fft"``: NumPy's real FFT (a library FFT used as one step).
The direct route pins the library route in the oracle's own tests.
"""

from __future__ import annotations

import numpy as np

__all__ = [
    "check_length",
    "dft_bins",
    "idft_from_bins",
    "pack_pairs",
    "unpack_pairs",
    "pack_halfcomplex",
    "unpack_halfcomplex",
    "rdfft_forward",
    "rdfft_inverse",
]


def check_length(n: int) -> None:
    """The packed format needs a Nyquist bin, so n must be even (Theorem 1 with N even)."""
    if n < 2 or n % 2:
        raise ValueError(f"packed real spectrum needs an even length >= 2, got {n}")


def _as_rows(a: np.ndarray) -> np.ndarray:
    a = np.asarray(a, dtype=np.float64)
    if a.ndim == 1:
        a = a[None, :]
    if a.ndim != 2:
        raise ValueError("expected a 1-D row or a 2-D (rows, n) array")
    return a


def _direct_bins(x: np.ndarray, ks: np.ndarray) -> np.ndarray:
    """Y_k = sum_m x_m exp(-2 pi i k m / n) for the bins ``ks`` (Eq. (1), forward)."""
    n = x.shape[1]
    m = np.arange(n, dtype=np.int64)
    out = np.empty((x.shape[0], len(ks)), dtype=np.complex128)
    # a block of bins at a time keeps the (bins x n) phase matrix small
    step = max(1, (1 << 22) // n)
    for s in range(0, len(ks), step):
        kk = ks[s : s + step].astype(np.int64)
        idx = np.outer(kk, m) % n  # exact integer reduction of k*m mod n
        phase = np.exp(-2j * np.pi * idx / n)
        out[:, s : s + step] = x @ phase.T
    return out


def dft_bins(x: np.ndarray, method: str = "fft", ks=None) -> np.ndarray:
    """Non-redundant spectrum Y_0..Y_{n/2} of each real row (Eq. (1), Theorem 1).

    ``ks`` selects a subset of bins (direct method only) for sampled checks of
    very long rows.
    """
    x = _as_rows(x)
    n = x.shape[1]
    check_length(n)
    if method == "direct":
        ks = np.arange(n // 2 + 1) if ks is None else np.asarray(ks)
        return _direct_bins(x, ks)
    if method == "fft":
        if ks is not None:
            raise ValueError("bin subsets are only offered by the direct method")
        return np.fft.rfft(x, axis=1)
    raise ValueError(method)


def idft_from_bins(bins: np.ndarray, n: int, method: str = "fft") -> np.ndarray:
    """Real rows from their non-redundant bins (Eq. (1), inverse, with 1/n).

    The imaginary parts of Y_0 and Y_{n/2} are taken as zero; the other half of
    the spectrum is the conjugate mirror (Theorem 1).
    """
    check_length(n)
    bins = np.asarray(bins, dtype=np.complex128)
    if bins.ndim == 1:
        bins = bins[None, :]
    if bins.shape[1] != n // 2 + 1:
        raise ValueError("need n/2+1 bins")
    b = bins.copy()
    b[:, 0] = b[:, 0].real
    b[:, n // 2] = b[:, n // 2].real
    if method == "fft":
        return np.fft.irfft(b, n=n, axis=1)
    if method == "direct":
        full = np.empty((b.shape[0], n), dtype=np.complex128)
        full[:, : n // 2 + 1] = b
        full[:, n // 2 + 1 :] = np.conj(b[:, 1 : n // 2][:, ::-1])  # Y_{n-k} = conj Y_k
        k = np.arange(n, dtype=np.int64)
        out = np.empty((b.shape[0], n), dtype=np.float64)
        step = max(1, (1 << 22) // n)
        for s in range(0, n, step):
            mm = np.arange(s, min(n, s + step), dtype=np.int64)
            idx = np.outer(mm, k) % n
            phase = np.exp(2j * np.pi * idx / n)
            out[:, s : s + step] = (full @ phase.T).real / n
        return out
    raise ValueError(method)


def pack_pairs(bins: np.ndarray) -> np.ndarray:
    """n/2+1 complex bins -> n reals: [Y_0, Y_{n/2}, Re Y_1, Im Y_1, ..., Re Y_{n/2-1}, Im Y_{n/2-1}]."""
    bins = np.asarray(bins, dtype=np.complex128)
    if bins.ndim == 1:
        bins = bins[None, :]
    h = bins.shape[1] - 1
    n = 2 * h
    out = np.empty((bins.shape[0], n), dtype=np.float64)
    out[:, 0] = bins[:, 0].real
    out[:, 1] = bins[:, h].real
    out[:, 2::2] = bins[:, 1:h].real
    out[:, 3::2] = bins[:, 1:h].imag
    return out


def unpack_pairs(buf: np.ndarray) -> np.ndarray:
    """Inverse of :func:`pack_pairs`; the DC and Nyquist bins come back purely real."""
    buf = _as_rows(buf)
    n = buf.shape[1]
    check_length(n)
    h = n // 2
    bins = np.zeros((buf.shape[0], h + 1), dtype=np.complex128)
    bins[:, 0] = buf[:, 0]
    bins[:, h] = buf[:, 1]
    bins[:, 1:h] = buf[:, 2::2] + 1j * buf[:, 3::2]
    return bins


def pack_halfcomplex(bins: np.ndarray) -> np.ndarray:
    """The paper's layout (Sec. 4.1): Re Y_k at slot k, Im Y_k at slot n-k, Y_0 at 0, Y_{n/2} at n/2."""
    bins = np.asarray(bins, dtype=np.complex128)
    if bins.ndim == 1:
        bins = bins[None, :]
    h = bins.shape[1] - 1
    n = 2 * h
    out = np.empty((bins.shape[0], n), dtype=np.float64)
    out[:, 0] = bins[:, 0].real
    out[:, h] = bins[:, h].real
    k = np.arange(1, h)
    out[:, k] = bins[:, 1:h].real
    out[:, n - k] = bins[:, 1:h].imag
    return out


def unpack_halfcomplex(buf: np.ndarray) -> np.ndarray:
    """Inverse of :func:`pack_halfcomplex`."""
    buf = _as_rows(buf)
    n = buf.shape[1]
    check_length(n)
    h = n // 2
    k = np.arange(1, h)
    bins = np.zeros((buf.shape[0], h + 1), dtype=np.complex128)
    bins[:, 0] = buf[:, 0]
    bins[:, h] = buf[:, h]
    bins[:, 1:h] = buf[:, k] + 1j * buf[:, n - k]
    return bins


def rdfft_forward(x: np.ndarray, method: str = "fft", layout: str = "pairs") -> np.ndarray:
    """Packed spectrum of each real row (what ``rdfft_forward`` leaves in the buffer)."""
    bins = dft_bins(x, method=method)
    if layout == "pairs":
        return pack_pairs(bins)
    if layout == "halfcomplex":
        return pack_halfcomplex(bins)
    raise ValueError(layout)


def rdfft_inverse(buf: np.ndarray, method: str = "fft", layout: str = "pairs") -> np.ndarray:
    """Real rows whose packed spectra are ``buf`` (what ``rdfft_inverse`` leaves in the buffer)."""
    buf = _as_rows(buf)
    if layout == "pairs":
        bins = unpack_pairs(buf)
    elif layout == "halfcomplex":
        bins = unpack_halfcomplex(buf)
    else:
        raise ValueError(layout)
    return idft_from_bins(bins, buf.shape[1], method=method)
