"""GPU parity of rdfft_forward / rdfft_inverse against the float64 oracle.

Inputs come from the seeded generator; the reference is ``oracle.rdfft`` on the same
stored values.  Covers every supported n (2 .. 65536), the three storage types
(float32, bfloat16, float16), row counts that span several workgroups with a ragged
tail, the full batched-transform sizes
(2^16 rows for n = 64..4096; 1024 rows for n = 65536) on sampled rows, guard bands,
run-to-run determinism and the absence of device allocation; and the mixed-radix rows
(n/2 = 2^a 3^b 5^c, not a power of two, up to 16384) in every storage type.
"""

import numpy as np
import pytest
import torch

from oracle import rdfft as ord_
from paper_2511_01385_amd import api, inputs
from tests._helpers import TORCH_DTYPE, assert_close, sample_rows, to_device, to_host_f64

pytestmark = pytest.mark.gpu

ALL_N = [2**k for k in range(1, 17)]
DTYPES = ["f32", "bf16", "f16"]


def _rows_for(n):
    # several workgroups plus a ragged tail, sized so the oracle stays fast
    if n <= 4096:
        return 1000 + 37
    return {8192: 67, 16384: 21, 32768: 9, 65536: 5}[n]


def _seed(n, dtype, salt):
    return 777 + 31 * int(np.log2(n)) + (0 if dtype == "f32" else 7) + 1000 * salt


@pytest.fixture(scope="module", autouse=True)
def _init():
    print("rdfft gpu tests on", torch.cuda.get_device_name(0), flush=True)
    api.rdfft_init()


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("n", ALL_N)
def test_forward_parity(n, dtype):
    rows = _rows_for(n)
    x = inputs.normal_rows(_seed(n, dtype, 0), rows, n, dtype)
    t = to_device(x, dtype)
    api.rdfft_forward(t)
    torch.cuda.synchronize()
    ref = ord_.rdfft_forward(inputs.to_f64(x, dtype))
    assert_close(to_host_f64(t), ref, dtype, f"forward n={n} {dtype}")


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("n", ALL_N)
def test_inverse_parity(n, dtype):
    rows = _rows_for(n)
    y = inputs.normal_rows(_seed(n, dtype, 1), rows, n, dtype)  # any reals are a packed spectrum
    t = to_device(y, dtype)
    api.rdfft_inverse(t)
    torch.cuda.synchronize()
    ref = ord_.rdfft_inverse(inputs.to_f64(y, dtype))
    assert_close(to_host_f64(t), ref, dtype, f"inverse n={n} {dtype}")


@pytest.mark.parametrize("n", [2, 64, 1024, 65536])
def test_round_trip_f32(n):
    rows = _rows_for(n)
    x = inputs.normal_rows(_seed(n, "f32", 2), rows, n, "f32")
    t = to_device(x, "f32")
    api.rdfft_inverse(api.rdfft_forward(t))
    torch.cuda.synchronize()
    back = to_host_f64(t)
    err = np.linalg.norm(back - x) / np.linalg.norm(x)
    assert err < 2e-6, err


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("n", [64, 128, 256, 512, 1024, 2048, 4096])
def test_full_batch_sampled(n, dtype):
    """The batched-transform workload: 2^16 rows per n, checked on sampled rows."""
    rows = 1 << 16
    x = inputs.normal_rows(inputs.seed_for(2, salt=n), rows, n, dtype)
    t = to_device(x, dtype)
    api.rdfft_forward(t)
    torch.cuda.synchronize()
    idx = sample_rows(rows, 96, n)
    got = to_host_f64(t[torch.as_tensor(idx, device=t.device)])
    assert_close(got, ord_.rdfft_forward(inputs.to_f64(x[idx], dtype)), dtype, f"full forward n={n}")
    y = t.clone()
    api.rdfft_inverse(t)
    torch.cuda.synchronize()
    got = to_host_f64(t[torch.as_tensor(idx, device=t.device)])
    ref = ord_.rdfft_inverse(to_host_f64(y[torch.as_tensor(idx, device=t.device)]))
    assert_close(got, ref, dtype, f"full inverse n={n}")


def test_long_rows_full_batch_sampled():
    """Rows beyond one LDS: n = 65536, 1024 rows, float32."""
    rows, n = 1024, 65536
    x = inputs.normal_rows(inputs.seed_for(5, salt=2), rows, n, "f32")
    t = to_device(x, "f32")
    api.rdfft_forward(t)
    torch.cuda.synchronize()
    idx = sample_rows(rows, 24, 5)
    got = to_host_f64(t[torch.as_tensor(idx, device=t.device)])
    assert_close(got, ord_.rdfft_forward(x[idx].astype(np.float64)), "f32", "n=65536 forward")
    # a few bins straight from the definition, independent of the library FFT route
    ks = np.array([0, 1, 12345, 32767, 32768])
    direct = ord_.dft_bins(x[idx[:2]].astype(np.float64), method="direct", ks=ks)
    packed = got[:2]
    for col, k in enumerate(ks):
        if k == 0:
            np.testing.assert_allclose(packed[:, 0], direct[:, col].real, rtol=1e-5, atol=1e-2)
        elif k == n // 2:
            np.testing.assert_allclose(packed[:, 1], direct[:, col].real, rtol=1e-5, atol=1e-2)
        else:
            np.testing.assert_allclose(packed[:, 2 * k] + 1j * packed[:, 2 * k + 1], direct[:, col], rtol=1e-5, atol=1e-2)
    y = t.clone()
    api.rdfft_inverse(t)
    torch.cuda.synchronize()
    got = to_host_f64(t[torch.as_tensor(idx, device=t.device)])
    ref = ord_.rdfft_inverse(to_host_f64(y[torch.as_tensor(idx, device=t.device)]))
    assert_close(got, ref, "f32", "n=65536 inverse")


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("n", [2, 16, 64, 4096, 65536])
def test_guard_bands_untouched(n, dtype):
    """Only the rows handed over are read and written."""
    rows, pad = 3 if n >= 16384 else 17, 4096
    x = inputs.normal_rows(_seed(n, dtype, 3), rows, n, dtype)
    big = torch.full((pad + rows * n + pad,), float("nan"), dtype=TORCH_DTYPE[dtype],
                     device="cuda")
    view = big[pad : pad + rows * n].view(rows, n)
    view.copy_(to_device(x, dtype))
    before = big.clone()
    api.rdfft_forward(view)
    api.rdfft_inverse(view)
    torch.cuda.synchronize()
    assert torch.isnan(big[:pad]).all() and torch.isnan(big[pad + rows * n :]).all()
    assert torch.equal(big[:pad].view(torch.int32 if dtype == "f32" else torch.int16),
                       before[:pad].view(torch.int32 if dtype == "f32" else torch.int16))
    assert np.isfinite(to_host_f64(view)).all()


@pytest.mark.parametrize("dtype", DTYPES)
def test_zero_and_single_row(dtype):
    t = torch.empty((0, 256), dtype=TORCH_DTYPE[dtype], device="cuda")
    api.rdfft_forward(t)
    x = inputs.normal_rows(_seed(256, dtype, 4), 1, 256, dtype)
    t = to_device(x, dtype)
    api.rdfft_forward(t)
    torch.cuda.synchronize()
    assert_close(to_host_f64(t), ord_.rdfft_forward(inputs.to_f64(x, dtype)), dtype, "single row")


@pytest.mark.parametrize("n", [1024, 65536])
def test_f16_overflow_gives_infinity(n):
    """float16 stores round to nearest: a DC bin of n = 65536 ones exceeds 65504 and becomes +inf.

    The DC and Nyquist sums of integers are exact in float32; the other bins of a
    constant row are zero up to the float32 rounding of the twiddle products."""
    t = torch.ones((3, n), dtype=torch.float16, device="cuda")
    api.rdfft_forward(t)
    torch.cuda.synchronize()
    got = t.float().cpu()
    want_dc = float("inf") if n > 65504 else float(n)
    assert (got[:, 0] == want_dc).all() and (got[:, 1] == 0).all()
    assert (got[:, 2:].abs() < 1e-2).all()


# even lengths whose half is 2^a 3^b 5^c but not a power of two: the mixed-radix rows
MIXED_N = [6, 10, 12, 30, 48, 96, 120, 360, 1000, 3000, 6144, 12288, 30000, 32000]


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("n", MIXED_N)
def test_mixed_radix_parity(n, dtype):
    rows = 257 if n <= 3000 else 9
    x = inputs.normal_rows(_seed(n, dtype, 6), rows, n, dtype)
    t = to_device(x, dtype)
    api.rdfft_forward(t)
    torch.cuda.synchronize()
    assert_close(to_host_f64(t), ord_.rdfft_forward(inputs.to_f64(x, dtype)), dtype, f"mixed forward n={n} {dtype}")
    y = inputs.normal_rows(_seed(n, dtype, 7), rows, n, dtype)
    t = to_device(y, dtype)
    api.rdfft_inverse(t)
    torch.cuda.synchronize()
    assert_close(to_host_f64(t), ord_.rdfft_inverse(inputs.to_f64(y, dtype)), dtype, f"mixed inverse n={n} {dtype}")


@pytest.mark.parametrize("n", [30, 3000, 32000])
def test_mixed_radix_guard_bands_and_round_trip(n):
    rows, pad = 5, 1024
    x = inputs.normal_rows(_seed(n, "f32", 8), rows, n, "f32")
    big = torch.full((pad + rows * n + pad,), float("nan"), device="cuda")
    view = big[pad : pad + rows * n].view(rows, n)
    view.copy_(to_device(x, "f32"))
    api.rdfft_forward(view)
    api.rdfft_inverse(view)
    torch.cuda.synchronize()
    assert torch.isnan(big[:pad]).all() and torch.isnan(big[pad + rows * n :]).all()
    back = to_host_f64(view)
    assert np.linalg.norm(back - x) / np.linalg.norm(x) < 2e-6


def _split_rows_check(t, n, dtype, rows_checked, what):
    """Forward then inverse over a buffer whose launches are split; checked rows vs the oracle."""
    idx = torch.as_tensor(rows_checked, device=t.device)
    x = to_host_f64(t[idx])
    api.rdfft_forward(t)
    torch.cuda.synchronize()
    assert_close(to_host_f64(t[idx]), ord_.rdfft_forward(x), dtype, f"{what} forward")
    y = to_host_f64(t[idx])
    api.rdfft_inverse(t)
    torch.cuda.synchronize()
    assert_close(to_host_f64(t[idx]), ord_.rdfft_inverse(y), dtype, f"{what} inverse")


def test_launch_split_beyond_grid_limit_n2():
    """2^31 + 3 rows of n = 2 (8 GiB of bf16): more rows than one launch's grid holds."""
    rows = (1 << 31) + 3
    t = torch.ones((rows, 2), dtype=torch.bfloat16, device="cuda")
    edge = [0, 1, (1 << 31) - 2, (1 << 31) - 1, 1 << 31, (1 << 31) + 1, rows - 1]
    vals = inputs.normal_rows(4321, len(edge), 2, "bf16")
    t[torch.as_tensor(edge, device="cuda")] = to_device(vals, "bf16")
    _split_rows_check(t, 2, "bf16", edge, "split n=2")
    # every other row was (1, 1): forward gives (2, 0), the inverse brings it back exactly
    t[torch.as_tensor(edge, device="cuda")] = 1
    for r0 in range(0, rows, 1 << 28):
        assert bool((t[r0 : r0 + (1 << 28)] == 1).all()), r0
    del t
    torch.cuda.empty_cache()


def test_launch_split_beyond_grid_limit_mixed():
    """Mixed-radix rows: 2^25 + 7 rows of n = 6 exceed one launch of 64-thread workgroups."""
    rows = (1 << 25) + 7
    t = torch.ones((rows, 6), dtype=torch.float32, device="cuda")
    edge = [0, (1 << 25) - 1, 1 << 25, rows - 1]
    t[torch.as_tensor(edge, device="cuda")] = to_device(inputs.normal_rows(4322, len(edge), 6, "f32"), "f32")
    _split_rows_check(t, 6, "f32", edge, "split n=6")
    t[torch.as_tensor(edge, device="cuda")] = 1
    assert float((t - 1).abs().max()) < 1e-6
    del t
    torch.cuda.empty_cache()


@pytest.mark.parametrize("n", [128, 4096, 65536])
def test_bitwise_deterministic(n):
    x = inputs.normal_rows(_seed(n, "f32", 5), _rows_for(n), n, "f32")
    a, b = to_device(x, "f32"), to_device(x, "f32")
    api.rdfft_forward(a)
    api.rdfft_forward(b)
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int32), b.view(torch.int32))


def test_special_inputs_closed_forms():
    """Impulse and constant rows give the closed-form spectra exactly up to rounding."""
    n, rows = 1024, 4
    x = np.zeros((rows, n), dtype=np.float32)
    x[0, 0] = 1.0
    x[1, :] = 1.0
    x[2, :] = (-1.0) ** np.arange(n)
    x[3, :] = np.cos(2 * np.pi * 5 * np.arange(n) / n)
    t = to_device(x, "f32")
    api.rdfft_forward(t)
    torch.cuda.synchronize()
    got = to_host_f64(t)
    want = np.zeros((rows, n))
    want[0, 0] = want[0, 1] = 1.0
    want[0, 2::2] = 1.0
    want[1, 0] = n
    want[2, 1] = n
    want[3, 10] = n / 2
    np.testing.assert_allclose(got, want, atol=2e-3)


def _single_bin_rows(n, last_radix):
    """cos and sin rows of one frequency k0 each, and their packed spectra: Y_k0 = n/2 (cos) or
    -i n/2 (sin), zero elsewhere, for 0 < k0 < n/2.  The frequencies cover the first and last
    bins of every group of N/R pair slots (N = n/2, R the radix of the transform's last pass),
    the middle of each group, the quarter and half points, and bins next to them, so every bin
    position of the last pass, and of its partner N - k, is met."""
    N = n // 2
    s = N // last_radix
    ks = sorted({k for j in range(last_radix) for k in (j * s, j * s + s // 2, j * s + s // 2 + 1, j * s - 1)
                 if 0 < k < N} | {N // 2, N // 2 - 1, 1, N - 1})
    m = np.arange(n)
    rows, spectra = [], []
    for k0 in ks:
        for kind in ("cos", "sin"):
            rows.append(np.cos(2 * np.pi * k0 * m / n) if kind == "cos" else np.sin(2 * np.pi * k0 * m / n))
            w = np.zeros(n)
            if kind == "cos":
                w[2 * k0] = n / 2
            else:
                w[2 * k0 + 1] = -n / 2
            spectra.append(w)
    return np.array(rows), np.array(spectra)


LONG_ROW_LAST_RADIX = [(2048, 8), (4096, 8), (65536, 32)]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("n,last_radix", LONG_ROW_LAST_RADIX)
def test_single_bin_closed_forms_long_rows(n, last_radix, dtype):
    """The forward of single-frequency rows is the closed-form spectrum."""
    rows, spectra = _single_bin_rows(n, last_radix)
    t = to_device(inputs.round_to(rows, dtype), dtype)
    api.rdfft_forward(t)
    torch.cuda.synchronize()
    # f32 rows: the DFT of the rounded inputs is the closed form to ~1e-6 n; bf16 rows carry
    # input rounding (relative 2^-9 per sample) and a bf16 store of the output (n/2 lands within n/512)
    atol = 2e-5 * n if dtype == "f32" else 0.004 * n
    np.testing.assert_allclose(to_host_f64(t), spectra, atol=atol)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("n,last_radix", LONG_ROW_LAST_RADIX)
def test_single_bin_inverse_closed_forms_long_rows(n, last_radix, dtype):
    """The inverse of a single-bin spectrum (exact in either storage type) is the cos or sin row."""
    rows, spectra = _single_bin_rows(n, last_radix)
    t = to_device(inputs.round_to(spectra, dtype), dtype)
    api.rdfft_inverse(t)
    torch.cuda.synchronize()
    # unit-amplitude outputs: f32 arithmetic error ~1e-6; bf16 adds one rounding (2^-9 relative)
    atol = 1e-5 if dtype == "f32" else 4e-3
    np.testing.assert_allclose(to_host_f64(t), rows, atol=atol)


@pytest.mark.parametrize("n", [1024, 3000])
def test_no_device_allocation(n):
    x = to_device(inputs.normal_rows(9, 4096, n, "bf16"), "bf16")
    api.rdfft_forward(x)  # first use on this device: table upload
    torch.cuda.synchronize()
    alloc0 = torch.cuda.memory_allocated()
    free0, _ = torch.cuda.mem_get_info()
    for _ in range(3):
        api.rdfft_forward(x)
        api.rdfft_inverse(x)
    torch.cuda.synchronize()
    free1, _ = torch.cuda.mem_get_info()
    assert torch.cuda.memory_allocated() == alloc0
    assert free1 == free0
