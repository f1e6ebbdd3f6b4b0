"""Seeded synthetic inputs shaped like the paper's workloads.

This module only draws random numbers and rounds them to the storage type.  It
holds none of the transform's arithmetic and imports nothing else from this
package, so the GPU library's tests and the CPU oracle can both consume its
output without sharing any computation.

Storage types: float32 arrays for ``"f32"``; for ``"bf16"`` the raw 16-bit
patterns as ``uint16`` (round-to-nearest-even from the float32 value, the same
rounding a bf16 store performs); for ``"f16"`` IEEE half patterns as ``uint16``
(NumPy's round-to-nearest-even conversion from float64).  :func:`to_f64` widens
each exactly.

Circulant parameters.  The paper's layers hold time-domain first columns
c ~ N(0, sigma^2) and the library consumes their packed spectra.  For white
Gaussian c of length p the DFT bins are independent, with
Y_0, Y_{p/2} ~ N(0, p*sigma^2) and Re Y_k, Im Y_k ~ N(0, p*sigma^2/2) for
0 < k < p/2.  :func:`circulant_spectra` draws the packed slots directly from
that law, so no transform is needed to make an input.
"""

from __future__ import annotations

import numpy as np

__all__ = [
    "generator",
    "round_to",
    "to_f64",
    "normal_rows",
    "circulant_spectra",
    "bca_problem",
    "seed_for",
]

# seed = 13850 + config number (configs are numbered from 1)
_SEED_BASE = 13850


def seed_for(config: int, salt: int = 0) -> int:
    return _SEED_BASE + int(config) + 1000 * int(salt)


def generator(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


def _f32_to_bf16_bits(a32: np.ndarray) -> np.ndarray:
    u = np.ascontiguousarray(a32, dtype=np.float32).view(np.uint32)
    # no wrap-around for finite values and infinities (u <= 0xFF800000)
    out = ((u + np.uint32(0x7FFF) + ((u >> 16) & np.uint32(1))) >> 16).astype(np.uint16)
    nan = (u & np.uint32(0x7FFFFFFF)) > np.uint32(0x7F800000)
    if nan.any():
        out[nan] = ((u[nan] >> 16) | 0x40).astype(np.uint16)  # keep NaNs quiet NaNs
    return out


def round_to(a: np.ndarray, dtype: str) -> np.ndarray:
    """float64 values -> storage array of ``dtype`` ("f32", "bf16" or "f16")."""
    if dtype == "f16":
        return np.asarray(a, dtype=np.float64).astype(np.float16).view(np.uint16)
    a32 = np.asarray(a, dtype=np.float64).astype(np.float32)
    if dtype == "f32":
        return a32
    if dtype == "bf16":
        return _f32_to_bf16_bits(a32)
    raise ValueError(dtype)


def to_f64(stored: np.ndarray, dtype: str) -> np.ndarray:
    """Exact float64 view of a storage array."""
    if dtype == "f32":
        return np.asarray(stored, dtype=np.float32).astype(np.float64)
    if dtype == "bf16":
        bits = np.asarray(stored, dtype=np.uint16).astype(np.uint32) << 16
        return bits.view(np.float32).astype(np.float64)
    if dtype == "f16":
        return np.asarray(stored, dtype=np.uint16).view(np.float16).astype(np.float64)
    raise ValueError(dtype)


def normal_rows(seed: int, rows: int, n: int, dtype: str, sigma: float = 1.0) -> np.ndarray:
    """(rows, n) storage array with entries ~ N(0, sigma^2).

    Drawn in row-major order from one PCG64 stream, a block of rows at a time
    (the stream is consumed in the same order as by a single draw).
    """
    if dtype not in ("f32", "bf16", "f16"):
        raise ValueError(dtype)
    g = generator(seed)
    out = np.empty((rows, n), dtype=np.float32 if dtype == "f32" else np.uint16)
    step = max(1, (1 << 20) // max(n, 1))
    for r0 in range(0, rows, step):
        r1 = min(rows, r0 + step)
        out[r0:r1] = round_to(g.standard_normal((r1 - r0, n)) * sigma, dtype)
    return out


def circulant_spectra(rng: np.random.Generator, q: int, kb: int, p: int, sigma: float, dtype: str):
    """Packed spectra (q, kb, p) of white Gaussian first columns c ~ N(0, sigma^2)."""
    z = rng.standard_normal((q, kb, p))
    scale = np.full(p, sigma * np.sqrt(p / 2.0))
    scale[:2] = sigma * np.sqrt(p)  # DC and Nyquist slots are real bins
    return round_to(z * scale, dtype)


def bca_problem(seed: int, tokens: int, d_in: int, d_out: int, p: int, sigma: float, dtype: str):
    """One block-circulant layer problem: x (T, d_in), c_spectra (q, kb, p), g (T, d_out).

    Drawn in the order x, c, g from one PCG64 stream; activations and upstream
    gradients ~ N(0, 1).
    """
    if d_in % p or d_out % p:
        raise ValueError("p must divide d_in and d_out")
    rng = generator(seed)
    x = round_to(rng.standard_normal((tokens, d_in)), dtype)
    c = circulant_spectra(rng, d_out // p, d_in // p, p, sigma, dtype)
    g = round_to(rng.standard_normal((tokens, d_out)), dtype)
    return x, c, g
