"""GPU parity of rdfft_forward_halfcomplex / rdfft_inverse_halfcomplex: the transforms with
the spectrum in the paper's halfcomplex layout (Sec. 4.1, Memory Layout).

Checked against the float64 oracle in that layout, and bit for bit against the pairs
transforms followed (forward) or preceded (inverse) by the in-place layout conversion:
every power-of-two n from 2 to 65536 and the mixed-radix lengths, in the three storage
types, with row counts that span several workgroups and a ragged tail; the full
2^16-row batch of n = 4096 on sampled rows; and guard bands around the rows handed over.
"""

import numpy as np
import pytest
import torch

from oracle import rdfft as ord_
from paper_2511_01385_amd import api, inputs
from tests._helpers import TORCH_DTYPE, assert_close, sample_rows, to_device, to_host_f64

pytestmark = pytest.mark.gpu

ALL_N = [2**k for k in range(1, 17)]
MIXED_N = [6, 30, 360, 3000, 6144, 32000]
DTYPES = ["f32", "bf16", "f16"]


def _rows_for(n):
    if n <= 4096:
        return 300 + 37
    return {8192: 19, 16384: 9, 32768: 5, 65536: 3}.get(n, 23)


def _seed(n, dtype, salt):
    return 91_000 + 17 * n % 9973 + (0 if dtype == "f32" else 5) + 1000 * salt


def _bits(t):
    return t.view(torch.int32 if t.dtype == torch.float32 else torch.int16)


@pytest.fixture(scope="module", autouse=True)
def _init():
    print("halfcomplex gpu tests on", torch.cuda.get_device_name(0), flush=True)
    api.rdfft_init()


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("n", ALL_N + MIXED_N)
def test_forward_halfcomplex(n, dtype):
    rows = _rows_for(n)
    x = inputs.normal_rows(_seed(n, dtype, 0), rows, n, dtype)
    t = to_device(x, dtype)
    api.rdfft_forward_halfcomplex(t)
    u = to_device(x, dtype)
    api.rdfft_pairs_to_halfcomplex(api.rdfft_forward(u))
    torch.cuda.synchronize()
    ref = ord_.rdfft_forward(inputs.to_f64(x, dtype), layout="halfcomplex")
    assert_close(to_host_f64(t), ref, dtype, f"forward halfcomplex n={n} {dtype}")
    assert torch.equal(_bits(t), _bits(u)), f"n={n} {dtype}: differs from forward + conversion"


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("n", ALL_N + MIXED_N)
def test_inverse_halfcomplex(n, dtype):
    rows = _rows_for(n)
    y = inputs.normal_rows(_seed(n, dtype, 1), rows, n, dtype)  # any reals are a halfcomplex spectrum
    t = to_device(y, dtype)
    api.rdfft_inverse_halfcomplex(t)
    u = to_device(y, dtype)
    api.rdfft_inverse(api.rdfft_halfcomplex_to_pairs(u))
    torch.cuda.synchronize()
    ref = ord_.rdfft_inverse(inputs.to_f64(y, dtype), layout="halfcomplex")
    assert_close(to_host_f64(t), ref, dtype, f"inverse halfcomplex n={n} {dtype}")
    assert torch.equal(_bits(t), _bits(u)), f"n={n} {dtype}: differs from conversion + inverse"


@pytest.mark.parametrize("n", [2, 1024, 65536, 3000])
def test_round_trip_f32(n):
    rows = _rows_for(n)
    x = inputs.normal_rows(_seed(n, "f32", 2), rows, n, "f32")
    t = to_device(x, "f32")
    api.rdfft_inverse_halfcomplex(api.rdfft_forward_halfcomplex(t))
    torch.cuda.synchronize()
    err = np.linalg.norm(to_host_f64(t) - x) / np.linalg.norm(x)
    assert err < 2e-6, err


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_full_batch_sampled(dtype):
    """2^16 rows of n = 4096, checked on sampled rows."""
    rows, n = 1 << 16, 4096
    x = inputs.normal_rows(inputs.seed_for(2, salt=n), rows, n, dtype)
    t = to_device(x, dtype)
    api.rdfft_forward_halfcomplex(t)
    torch.cuda.synchronize()
    idx = sample_rows(rows, 64, 11)
    sel = torch.as_tensor(idx, device=t.device)
    got = to_host_f64(t[sel])
    assert_close(got, ord_.rdfft_forward(inputs.to_f64(x[idx], dtype), layout="halfcomplex"), dtype, "full forward")
    y = t.clone()
    api.rdfft_inverse_halfcomplex(t)
    torch.cuda.synchronize()
    ref = ord_.rdfft_inverse(to_host_f64(y[sel]), layout="halfcomplex")
    assert_close(to_host_f64(t[sel]), ref, dtype, "full inverse")


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("n", [2, 64, 4096, 65536, 6144])
def test_guard_bands_untouched(n, dtype):
    """Only the rows handed over are read and written."""
    rows, pad = 3 if n >= 16384 else 17, 4096
    x = inputs.normal_rows(_seed(n, dtype, 3), rows, n, dtype)
    big = torch.full((pad + rows * n + pad,), float("nan"), dtype=TORCH_DTYPE[dtype], device="cuda")
    view = big[pad : pad + rows * n].view(rows, n)
    view.copy_(to_device(x, dtype))
    before = big.clone()
    api.rdfft_forward_halfcomplex(view)
    api.rdfft_inverse_halfcomplex(view)
    torch.cuda.synchronize()
    assert torch.equal(_bits(big[:pad]), _bits(before[:pad]))
    assert torch.equal(_bits(big[pad + rows * n :]), _bits(before[pad + rows * n :]))
    assert np.isfinite(to_host_f64(view)).all()


def test_zero_rows_is_a_no_op():
    t = torch.empty((0, 256), dtype=torch.bfloat16, device="cuda")
    api.rdfft_forward_halfcomplex(t)
    api.rdfft_inverse_halfcomplex(t)
    torch.cuda.synchronize()
