"""Helpers shared by the GPU parity tests: host<->device copies of seeded inputs and
the comparison rule.

Comparison rule (both must hold):
* relative L2 error over the compared outputs, ||gpu - ref||_2 / ||ref||_2, at most
  1e-5 for float32 storage and 2e-2 for bfloat16 storage, the reference being the
  float64 oracle on the same stored inputs;
* element by element, |gpu - ref| <= 2^-8 |ref| (bf16) or 2^-11 |ref| (f16): one
  round-to-nearest-even store, + 2e-5 * rms(ref of that row) (float32 arithmetic).

Outputs that pass through `staged` spectra stored in a 16-bit type on the way (the
layer for blocks beyond 8192 keeps its intermediate spectra in the storage type) widen
the element bound by 4 sqrt(staged) u rms(row), u = 2^-8 (bf16): a rounding of a spectrum
spreads over every element of the row after the inverse transform, with an RMS of about
u / (2 sqrt 3) of the row's, and the largest of many millions of such errors reaches about
six times that.

For f16 storage the rel-L2 bound is 2e-3: one store rounding contributes at most
2^-12 relative RMS (2.4e-4) and the float32 arithmetic ~1e-7, so 2e-3 keeps an 8x
margin while still failing on any mistake larger than the storage resolution.
"""

from __future__ import annotations

import numpy as np
import torch

from paper_2511_01385_amd import inputs

TOL = {"f32": 1e-5, "bf16": 2e-2, "f16": 2e-3}
TORCH_DTYPE = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}
ELEMENT_REL = {"f32": 0.0, "bf16": 2.0**-8, "f16": 2.0**-11}


def to_device(stored: np.ndarray, dtype: str, device="cuda") -> torch.Tensor:
    if dtype == "f32":
        return torch.from_numpy(np.ascontiguousarray(stored, dtype=np.float32)).to(device)
    bits = np.ascontiguousarray(stored, dtype=np.uint16).view(np.int16)
    return torch.from_numpy(bits).view(TORCH_DTYPE[dtype]).to(device)


def to_host_f64(t: torch.Tensor) -> np.ndarray:
    t = t.detach().cpu()
    if t.dtype == torch.float32:
        return t.numpy().astype(np.float64)
    if t.dtype == torch.bfloat16:
        return inputs.to_f64(t.view(torch.int16).numpy().view(np.uint16), "bf16")
    if t.dtype == torch.float16:
        return inputs.to_f64(t.view(torch.int16).numpy().view(np.uint16), "f16")
    raise TypeError(t.dtype)


def rel_l2(got: np.ndarray, ref: np.ndarray) -> float:
    den = np.linalg.norm(ref)
    return float(np.linalg.norm(got - ref) / (den if den > 0 else 1.0))


def assert_close(got: np.ndarray, ref: np.ndarray, dtype: str, what: str = "", staged: int = 0) -> float:
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    err = rel_l2(got, ref)
    assert err <= TOL[dtype], f"{what}: rel-L2 {err:.3e} > {TOL[dtype]:.1e}"
    r2 = ref.reshape(-1, ref.shape[-1]) if ref.ndim > 1 else ref.reshape(1, -1)
    g2 = got.reshape(r2.shape)
    rms = np.sqrt(np.mean(r2**2, axis=1, keepdims=True))
    bound = (2e-5 + 4 * np.sqrt(staged) * ELEMENT_REL[dtype]) * rms + ELEMENT_REL[dtype] * np.abs(r2)
    bad = np.abs(g2 - r2) > bound
    if bad.any():
        i, j = np.argwhere(bad)[0]
        raise AssertionError(
            f"{what}: {int(bad.sum())} elements outside the element bound; first at row {i} col {j}: "
            f"gpu {g2[i, j]!r} ref {r2[i, j]!r} bound {bound[i, j] if np.ndim(bound) else bound!r}"
        )
    return err


def sample_rows(rows: int, count: int, seed: int) -> np.ndarray:
    """A sorted sample of row indices that always includes the first and the last row."""
    rng = np.random.default_rng(seed)
    pick = rng.choice(rows, size=min(count, rows), replace=False)
    return np.unique(np.concatenate([pick, [0, rows - 1]]))


def impulse_spectra(shifts, p):
    """Packed spectra of impulse circulants c_ij = e_{s_ij} (s < 0: a zero block), from the closed
    form Y_k = exp(-2 pi i k s / p): slot 0 holds (1, (-1)^s), slot k (cos, -sin)(2 pi k s / p)."""
    q, kb = shifts.shape
    out = np.zeros((q, kb, p))
    k = np.arange(1, p // 2)
    for i in range(q):
        for j in range(kb):
            s = shifts[i, j]
            if s < 0:
                continue
            out[i, j, 0] = 1.0
            out[i, j, 1] = (-1.0) ** s
            out[i, j, 2::2] = np.cos(2 * np.pi * k * s / p)
            out[i, j, 3::2] = -np.sin(2 * np.pi * k * s / p)
    return out
