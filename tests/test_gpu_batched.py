"""GPU parity of bca_forward_batched / bca_backward_batched: several independent layers of one
shape in one call (Sec. 5.1.2, adapters on the query and value projections of every layer).

Every layer of a batch must give what the single-layer call gives on it: y and dx bit for bit
(the same per-token arithmetic), dc up to the order of its float32 sums (checked against the
float64 oracle at the float32 bar).  Cases: batches that run side by side in the wave kernels
(including more layers than one launch takes, and shared read-only inputs), batches that fall
back to one layer after another (other shapes, dx over gy, too few tokens to stage the dC
sums), and a zero-layer call.
"""

import numpy as np
import pytest
import torch

from oracle import bca as obca
from paper_2511_01385_amd import api, inputs
from tests._helpers import TORCH_DTYPE, assert_close, to_device, to_host_f64

pytestmark = pytest.mark.gpu


def _bits(t):
    return t.view(torch.int32 if t.dtype == torch.float32 else torch.int16)


def _layers(count, tokens, d, p, dtype, seed, shared_x=False):
    out = []
    for b in range(count):
        x, c, g = inputs.bca_problem(seed + (0 if shared_x else b), tokens, d, d, p, 0.02, dtype)
        if shared_x and b > 0:
            _, c, g = inputs.bca_problem(seed + 1000 + b, tokens, d, d, p, 0.02, dtype)
        out.append((x, c, g))
    return out


def _check_batch(layers, d, p, dtype, alias_dx=False, shared_x=False):
    tdt = TORCH_DTYPE[dtype]
    xs = [to_device(x, dtype) for x, _, _ in layers]
    if shared_x:
        xs = [xs[0]] * len(layers)
    cs = [to_device(c, dtype) for _, c, _ in layers]
    tokens = layers[0][0].shape[0]
    # batched
    ys = [torch.empty((tokens, d), dtype=tdt, device="cuda") for _ in layers]
    api.bca_forward_batched(xs, cs, ys)
    gys = [to_device(g, dtype) for _, _, g in layers]
    dxs = gys if alias_dx else [torch.empty((tokens, d), dtype=tdt, device="cuda") for _ in layers]
    dcs = [torch.full(c.shape, float("nan"), device="cuda") for _, c, _ in layers]
    api.bca_backward_batched(xs, cs, gys, dxs, dcs)
    # one layer at a time
    for b, (x, c, g) in enumerate(layers):
        y1 = torch.empty((tokens, d), dtype=tdt, device="cuda")
        api.bca_forward(xs[b], cs[b], y1)
        g1 = to_device(g, dtype)
        dx1 = g1 if alias_dx else torch.empty((tokens, d), dtype=tdt, device="cuda")
        dc1 = torch.empty(c.shape, device="cuda")
        api.bca_backward(xs[b], cs[b], g1, dx1, dc1)
        torch.cuda.synchronize()
        assert torch.equal(_bits(ys[b]), _bits(y1)), f"layer {b}: y differs from the single-layer call"
        assert torch.equal(_bits(dxs[b]), _bits(dx1)), f"layer {b}: dx differs from the single-layer call"
        xf = inputs.to_f64(layers[0][0] if shared_x else x, dtype)
        cf, gf = inputs.to_f64(c, dtype), inputs.to_f64(g, dtype)
        q = kb = d // p
        _, rdc = obca.backward_spectral(xf, cf, gf, p)
        assert_close(to_host_f64(dcs[b]).reshape(q * kb, p), rdc.reshape(q * kb, p), "f32", f"layer {b} dc")
        np.testing.assert_allclose(to_host_f64(dcs[b]), to_host_f64(dc1), rtol=1e-5,
                                   atol=1e-5 * float(np.abs(rdc).max()))
        if b < 2:  # the layer against the oracle too
            assert_close(to_host_f64(ys[b]), obca.forward_spectral(xf, cf, d, p), dtype, f"layer {b} y")


@pytest.fixture(scope="module", autouse=True)
def _init():
    print("batched layer gpu tests on", torch.cuda.get_device_name(0), flush=True)
    api.rdfft_init()


# (count, tokens, d, p, dtype): side by side in the wave kernels
FUSED = [(24, 256, 768, 256, "bf16"), (40, 64, 256, 128, "bf16"), (5, 256, 1024, 512, "f16"),
         (3, 100, 512, 128, "f32")]  # the last: a forward side by side, a backward too short to stage


@pytest.mark.parametrize("shape", FUSED, ids=[f"n{s[0]}_T{s[1]}_{s[2]}_p{s[3]}_{s[4]}" for s in FUSED])
def test_batches_side_by_side(shape):
    count, tokens, d, p, dtype = shape
    _check_batch(_layers(count, tokens, d, p, dtype, 3300 + count), d, p, dtype)


def test_shared_input():
    """Layers may share a read-only input (the query and value adapters of one layer)."""
    _check_batch(_layers(2, 128, 768, 256, "bf16", 3500, shared_x=True), 768, 256, "bf16", shared_x=True)


# one layer after another: another shape, dx over gy, too few tokens to stage the dC sums
SEQUENTIAL = [(2, 8, 4096, 1024, "bf16", False), (4, 64, 768, 256, "bf16", True), (3, 5, 768, 256, "f32", False)]


@pytest.mark.parametrize("shape", SEQUENTIAL, ids=[f"n{s[0]}_T{s[1]}_{s[2]}_p{s[3]}_{s[4]}_{'aliased' if s[5] else 'apart'}"
                                                   for s in SEQUENTIAL])
def test_batches_one_by_one(shape):
    count, tokens, d, p, dtype, alias = shape
    _check_batch(_layers(count, tokens, d, p, dtype, 3600 + count), d, p, dtype, alias_dx=alias)


def test_zero_layers():
    api.bca_forward_batched([], [], [])
    api.bca_backward_batched([], [], [], [], [])
    torch.cuda.synchronize()


def test_overlapping_outputs_refused():
    """What one layer writes may not overlap another layer's buffers; nothing is enqueued."""
    tokens, d, p = 16, 768, 256
    x = torch.zeros((2, tokens, d), dtype=torch.bfloat16, device="cuda")
    c = torch.zeros((3, 3, p), dtype=torch.bfloat16, device="cuda")
    y = torch.zeros((tokens, d), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(api.RdfftError):
        api.bca_forward_batched([x[0], x[1]], [c, c], [y, y])
    with pytest.raises(api.RdfftError):
        api.bca_forward_batched([x[0], y], [c, c], [y, x[1]])
