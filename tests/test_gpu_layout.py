"""GPU checks of the in-place layout converters (pairs <-> halfcomplex).

The conversion is a permutation, so the bar is bit-exact: the expected halfcomplex
buffer is the oracle's ``pack_halfcomplex(unpack_pairs(.))`` of the same stored
values, stored back in the storage type (exact, as every value already is one).  Any
n reals are a valid packed spectrum, so the inputs are seeded random values; a chain
test also runs the GPU forward transform and compares its halfcomplex form with the
oracle's halfcomplex spectrum to the transform tolerance.
"""

import numpy as np
import pytest
import torch

from oracle import rdfft as ord_
from paper_2511_01385_amd import api, inputs
from tests._helpers import assert_close, to_device, to_host_f64

pytestmark = pytest.mark.gpu

ALL_N = [2**k for k in range(1, 17)]
DTYPES = ["f32", "bf16", "f16"]


def _rows_for(n):
    if n <= 4096:
        return 300 + 7
    return {8192: 33, 16384: 9, 32768: 5, 65536: 3}[n]


def _bits(t: torch.Tensor) -> np.ndarray:
    t = t.detach().cpu()
    return (t.view(torch.int32) if t.dtype == torch.float32 else t.view(torch.int16)).numpy().copy()


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("n", ALL_N)
def test_pairs_to_halfcomplex_bit_exact(n, dtype):
    rows = _rows_for(n)
    y = inputs.normal_rows(4242 + n, rows, n, dtype)
    t = to_device(y, dtype)
    api.rdfft_pairs_to_halfcomplex(t)
    torch.cuda.synchronize()
    want = inputs.round_to(ord_.pack_halfcomplex(ord_.unpack_pairs(inputs.to_f64(y, dtype))), dtype)
    assert np.array_equal(_bits(t), _bits(to_device(want, dtype)))
    api.rdfft_halfcomplex_to_pairs(t)
    torch.cuda.synchronize()
    assert np.array_equal(_bits(t), _bits(to_device(y, dtype)))


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("n", [6, 30, 96, 1000, 12288, 32000])
def test_mixed_lengths_bit_exact(n, dtype):
    """Rows whose half-length has factors 3 and 5 use the same permutation."""
    rows = 31 if n <= 1000 else 3
    y = inputs.normal_rows(7373 + n, rows, n, dtype)
    t = to_device(y, dtype)
    api.rdfft_pairs_to_halfcomplex(t)
    torch.cuda.synchronize()
    want = inputs.round_to(ord_.pack_halfcomplex(ord_.unpack_pairs(inputs.to_f64(y, dtype))), dtype)
    assert np.array_equal(_bits(t), _bits(to_device(want, dtype)))
    api.rdfft_halfcomplex_to_pairs(t)
    torch.cuda.synchronize()
    assert np.array_equal(_bits(t), _bits(to_device(y, dtype)))


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("n", [16, 1024, 65536])
def test_halfcomplex_to_pairs_bit_exact(n, dtype):
    rows = _rows_for(n)
    h = inputs.normal_rows(5151 + n, rows, n, dtype)  # read as a halfcomplex buffer
    t = to_device(h, dtype)
    api.rdfft_halfcomplex_to_pairs(t)
    torch.cuda.synchronize()
    want = inputs.round_to(ord_.pack_pairs(ord_.unpack_halfcomplex(inputs.to_f64(h, dtype))), dtype)
    assert np.array_equal(_bits(t), _bits(to_device(want, dtype)))


def test_payload_bits_survive():
    # NaN payloads, infinities and signed zeros move unchanged
    n, rows = 64, 5
    raw = np.random.default_rng(7).integers(0, 2**32, size=(rows, n), dtype=np.uint64).astype(np.uint32)
    raw[:, :8] = [0x7FC12345, 0xFF800000, 0x80000000, 0x7F800000, 0xFFC00001, 0x00000001, 0, 0x7FFFFFFF]
    t = torch.from_numpy(raw.view(np.int32)).view(torch.float32).cuda()
    api.rdfft_pairs_to_halfcomplex(t)
    api.rdfft_halfcomplex_to_pairs(t)
    torch.cuda.synchronize()
    assert np.array_equal(_bits(t), raw.view(np.int32))


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("n", [8, 256, 4096, 65536])
def test_forward_then_halfcomplex_matches_oracle(n, dtype):
    rows = _rows_for(n)
    x = inputs.normal_rows(6161 + n, rows, n, dtype)
    t = to_device(x, dtype)
    api.rdfft_forward(t)
    api.rdfft_pairs_to_halfcomplex(t)
    torch.cuda.synchronize()
    ref = ord_.rdfft_forward(inputs.to_f64(x, dtype), layout="halfcomplex")
    assert_close(to_host_f64(t), ref, dtype, f"forward+halfcomplex n={n} {dtype}")


def test_zero_rows_and_errors():
    t = torch.zeros(0, 64, device="cuda")
    api.rdfft_pairs_to_halfcomplex(t)
    with pytest.raises(api.RdfftError):
        api.rdfft_pairs_to_halfcomplex(torch.zeros(3, 14, device="cuda"))  # n/2 = 7: no plan


def test_launch_split_beyond_grid_limit_mixed():
    """2^25 + 7 rows of n = 6: more rows than one launch of 64-thread workgroups holds."""
    rows = (1 << 25) + 7
    r = torch.arange(rows, device="cuda", dtype=torch.int64) % 1000
    t = (r[:, None].float() + torch.arange(6, device="cuda").float()[None, :] / 8).contiguous()
    orig = t.clone()
    api.rdfft_pairs_to_halfcomplex(t)
    torch.cuda.synchronize()
    # pair slot k -> real slots (k, n - k), slot 0 -> (0, n/2): [s0, s2, s4, s1, s5, s3]
    perm = torch.as_tensor([0, 2, 4, 1, 5, 3], device="cuda")
    assert torch.equal(t, orig[:, perm])
    api.rdfft_halfcomplex_to_pairs(t)
    torch.cuda.synchronize()
    assert torch.equal(t, orig)
    del t, orig, r
    torch.cuda.empty_cache()
