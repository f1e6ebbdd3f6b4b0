"""Host-side checks of the autograd wrapper's argument validation (no GPU needed)."""

import pytest
import torch

from paper_2511_01385_amd.layer import BlockCirculantLinear


@pytest.mark.parametrize("d_in,d_out,p", [(256, 256, 48), (256, 256, 1), (256, 192, 128), (100, 100, 8),
                                          (131072, 131072, 131072), (4194304, 4194304, 16384)])
def test_rejects_bad_block_sizes(d_in, d_out, p):
    with pytest.raises(ValueError):
        BlockCirculantLinear(d_in, d_out, p, device="cpu")


def test_rejects_unsupported_storage_type():
    with pytest.raises(TypeError):
        BlockCirculantLinear(64, 64, 16, dtype=torch.float64, device="cpu")
    BlockCirculantLinear(64, 64, 16, dtype=torch.float16, device="cpu")  # 16-bit IEEE storage is supported


def test_parameter_shape_and_scale():
    layer = BlockCirculantLinear(512, 256, 64, dtype=torch.float32, device="cpu")
    assert layer.c.shape == (4, 8, 64) and layer.c.dtype == torch.float32
    assert abs(layer.c.std().item() - 512 ** -0.5) < 0.01
