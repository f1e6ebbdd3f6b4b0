"""Host-side checks of the Python binding's argument validation (no GPU needed).

The library receives only pointers and sizes, so the binding refuses tensors whose shape,
storage type or device disagree before any library call.
"""

import pytest
import torch

from paper_2511_01385_amd import api


def _t(*shape, dtype=torch.float32):
    return torch.empty(shape, dtype=dtype)


@pytest.mark.parametrize(
    "x,c,y,err",
    [
        (_t(8, 256), _t(4, 4, 64), _t(8, 128), ValueError),  # y width != q*p
        (_t(8, 192), _t(4, 4, 64), _t(8, 256), ValueError),  # x width != kb*p
        (_t(8, 256), _t(16, 64), _t(8, 256), ValueError),  # spectra not (q, kb, p)
        (_t(8, 256), _t(4, 4, 64), _t(7, 256), ValueError),  # token counts differ
        (_t(8, 256), _t(4, 4, 64, dtype=torch.bfloat16), _t(8, 256), TypeError),
        (_t(8, 256), _t(4, 4, 64), _t(8, 256, dtype=torch.bfloat16), TypeError),
        (_t(8, 256), _t(4, 4, 64), _t(8, 256), ValueError),  # host tensors
    ],
)
def test_bca_forward_refuses_mismatched_tensors(x, c, y, err):
    with pytest.raises(err):
        api.bca_forward(x, c, y)


@pytest.mark.parametrize(
    "gy,dx,dc,err",
    [
        (_t(8, 128), _t(8, 256), _t(4, 4, 64), ValueError),  # gy width
        (_t(8, 256), _t(8, 128), _t(4, 4, 64), ValueError),  # dx shape
        (_t(8, 256), _t(8, 256, dtype=torch.bfloat16), _t(4, 4, 64), ValueError),  # dx dtype
        (_t(8, 256), _t(8, 256), _t(4, 4, 32), ValueError),  # dc shape
        (_t(8, 256), _t(8, 256), _t(4, 4, 64, dtype=torch.bfloat16), TypeError),  # dc dtype
    ],
)
def test_bca_backward_refuses_mismatched_tensors(gy, dx, dc, err):
    with pytest.raises(err):
        api.bca_backward(_t(8, 256), _t(4, 4, 64), gy, dx, dc)


def test_transform_refuses_host_tensors_and_other_types():
    with pytest.raises(ValueError):
        api.rdfft_forward(_t(4, 64))
    with pytest.raises((TypeError, ValueError)):
        api.rdfft_forward(torch.empty(4, 64, dtype=torch.float64))
