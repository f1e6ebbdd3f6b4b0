"""GPU parity of bca_forward / bca_backward against the float64 oracle.

The reference is ``oracle.bca`` on the stored inputs: the spectral route (pinned to the
dense definition by the CPU tests) for whole outputs, and the dense definition's
element sums for sampled entries.  The parameters the layer sees are the stored
packed spectra; the oracle maps them back to time-domain columns itself.
"""

import numpy as np
import pytest
import torch

from oracle import bca as obca
from paper_2511_01385_amd import api, inputs
from tests._helpers import ELEMENT_REL, TORCH_DTYPE, assert_close, impulse_spectra, to_device, to_host_f64

pytestmark = pytest.mark.gpu

# (name, tokens, d_in, d_out, p, sigma, dtype): the paper-shaped layers
CONFIGS = [
    ("cfg1 fp32 d=256 p=64", 128, 256, 256, 64, 0.02, "f32"),
    ("cfg3 bf16 d=768 p=256", 4096, 768, 768, 256, 0.02, "bf16"),
    ("cfg4 bf16 d=4096 p=1024", 4096, 4096, 4096, 1024, 0.01, "bf16"),
    ("cfg5a bf16 d=p=8192", 4096, 8192, 8192, 8192, 0.02, "bf16"),
    # one circulant beyond the fused kernels' blocks: the multi-pass layer
    ("circulant bf16 d=p=65536", 1024, 65536, 65536, 65536, 0.004, "bf16"),
]

# small ragged shapes: odd token counts, rectangular layers, every block size
SMALL = [
    (1, 8, 8, 2, "f32"),
    (5, 8, 4, 4, "f32"),
    (37, 48, 16, 8, "bf16"),
    (19, 64, 192, 16, "f32"),
    (33, 96, 32, 32, "bf16"),
    (7, 128, 384, 64, "f32"),
    (45, 512, 256, 128, "f32"),
    (11, 256, 1024, 256, "bf16"),
    (9, 1024, 512, 512, "f32"),
    (6, 2048, 2048, 1024, "f32"),
    (5, 2048, 2048, 2048, "bf16"),
    (3, 4096, 4096, 4096, "f32"),
    (3, 8192, 8192, 8192, "f32"),
    # square layers (q == kb) across the register-resident kernels' thread splits, and
    # square shapes that fall back to the general kernels (too many slots, or q > 4)
    (13, 32, 32, 16, "bf16"),
    (21, 96, 96, 32, "f32"),
    (17, 512, 512, 128, "bf16"),
    (10, 1536, 1536, 512, "f32"),
    (7, 4096, 4096, 2048, "bf16"),
    (5, 8192, 8192, 4096, "f32"),
    (4, 6144, 6144, 2048, "bf16"),
    (9, 256, 256, 16, "f32"),
    # layers whose dC slots exceed LDS: dC over block ranges, then one dx launch
    (5, 4096, 4096, 128, "bf16"),
    (3, 2048, 4096, 64, "f32"),
    (7, 4096, 2048, 256, "f32"),
    # a token's spectra beyond the forward's two-workgroups-per-CU budget (8 x 8 blocks of 1024)
    (3, 8192, 8192, 1024, "bf16"),
    (2, 8192, 8192, 1024, "f32"),
]


def _problem(seed, tokens, d_in, d_out, p, sigma, dtype):
    x, c, g = inputs.bca_problem(seed, tokens, d_in, d_out, p, sigma, dtype)
    return x, c, g


def _run(x, c, g, dtype, d_out, alias_y=False, alias_dx=False):
    xt, ct, gt = to_device(x, dtype), to_device(c, dtype), to_device(g, dtype)
    tokens, d_in = x.shape
    if alias_y:
        yt = xt.clone()
        api.bca_forward(yt, ct, yt)
    else:
        yt = torch.empty((tokens, d_out), dtype=TORCH_DTYPE[dtype], device="cuda")
        api.bca_forward(xt, ct, yt)
    dct = torch.full(c.shape, float("nan"), dtype=torch.float32, device="cuda")  # must be overwritten
    if alias_dx:
        api.bca_backward(xt, ct, gt, gt, dct)
        dxt = gt
    else:
        dxt = torch.empty((tokens, d_in), dtype=TORCH_DTYPE[dtype], device="cuda")
        api.bca_backward(xt, ct, gt, dxt, dct)
    torch.cuda.synchronize()
    return to_host_f64(yt), to_host_f64(dxt), to_host_f64(dct)


def _dc_bar(dtype, p):
    # blocks beyond 8192 keep a 16-bit layer's intermediate spectra in its storage type, so
    # its dc meets that type's bar; every other dc is float32 arithmetic on exactly widened
    # inputs
    return dtype if dtype != "f32" and p > 8192 else "f32"


# relative bound of sampled entries against the dense definition's sums, per storage type
SAMPLE_RTOL = {"f32": 1e-4, "bf16": 2e-2, "f16": 2e-3}


def _check(x, c, g, dtype, d_out, p, got, what, sampled=0, y_staged=None):
    y, dx, dc = got
    x64, c64, g64 = inputs.to_f64(x, dtype), inputs.to_f64(c, dtype), inputs.to_f64(g, dtype)
    q, kb = c.shape[0], c.shape[1]
    staged = 2 if p > 8192 else 0  # spectra stored on the way (storage type)
    assert_close(y, obca.forward_spectral(x64, c64, d_out, p), dtype, f"{what} y",
                 staged if y_staged is None else y_staged)
    rdx, rdc = obca.backward_spectral(x64, c64, g64, p)
    assert_close(dx, rdx, dtype, f"{what} dx", staged)
    assert_close(dc.reshape(q * kb, p), rdc.reshape(q * kb, p), _dc_bar(dtype, p), f"{what} dc", staged)
    if sampled:
        rng = np.random.default_rng(sampled)
        ceff = obca.effective_c(c64, q, kb, p)
        t_ = rng.integers(0, x.shape[0], 8)
        ent = [(int(a), int(rng.integers(q)), int(rng.integers(p))) for a in t_]
        # staged spectra spread their rounding over whole rows: an absolute term of the
        # element bound's size, in units of the output's RMS
        spread = 4 * np.sqrt(staged) * ELEMENT_REL[dtype]
        ref = obca.forward_entries(x64, ceff, ent)
        np.testing.assert_allclose([y[a, i * p + m] for a, i, m in ent], ref, rtol=SAMPLE_RTOL[dtype],
                                   atol=1e-3 * np.abs(ref).max() + spread * np.sqrt(np.mean(y**2)))
        ent = [(int(a), int(rng.integers(kb)), int(rng.integers(p))) for a in t_]
        ref = obca.dx_entries(g64, ceff, ent)
        np.testing.assert_allclose([dx[a, j * p + r] for a, j, r in ent], ref, rtol=SAMPLE_RTOL[dtype],
                                   atol=1e-3 * np.abs(ref).max() + spread * np.sqrt(np.mean(dx**2)))
        ent = [(int(rng.integers(q)), int(rng.integers(kb)), int(rng.integers(p))) for _ in range(4)]
        ref = obca.dc_entries(x64, g64, q, kb, p, ent)
        tol = SAMPLE_RTOL[_dc_bar(dtype, p)]
        np.testing.assert_allclose([dc[i, j, s] for i, j, s in ent], ref, rtol=tol,
                                   atol=tol * np.abs(ref).max() + spread * np.sqrt(np.mean(dc**2)))


# blocks beyond 8192 (the multi-pass layer): kb <= q, several tokens, both storage types
LONG = [
    (3, 16384, 16384, 16384, "f32"),
    (5, 16384, 16384, 16384, "bf16"),
    (4, 32768, 65536, 32768, "f32"),  # q = 2, kb = 1
    (3, 32768, 32768, 16384, "bf16"),  # q = kb = 2
    (2, 49152, 98304, 16384, "f32"),  # q = 6, kb = 3
    (3, 65536, 65536, 65536, "f32"),
    (2, 65536, 65536, 65536, "bf16"),
    (37, 16384, 32768, 16384, "bf16"),  # q = 2, kb = 1, more tokens than dC chunks
    (6, 32768, 32768, 32768, "bf16"),  # single circulants: the fused row kernel
    (4, 32768, 32768, 32768, "f32"),
]


@pytest.fixture(scope="module", autouse=True)
def _init():
    print("bca gpu tests on", torch.cuda.get_device_name(0), flush=True)
    api.rdfft_init()


@pytest.mark.parametrize("cfg", CONFIGS, ids=[c[0] for c in CONFIGS])
def test_paper_shaped_layers(cfg):
    name, tokens, d_in, d_out, p, sigma, dtype = cfg
    x, c, g = _problem(inputs.seed_for(CONFIGS.index(cfg) + 1), tokens, d_in, d_out, p, sigma, dtype)
    got = _run(x, c, g, dtype, d_out)
    _check(x, c, g, dtype, d_out, p, got, name, sampled=17)


@pytest.mark.parametrize("shape", SMALL, ids=[f"T{s[0]}_{s[1]}x{s[2]}_p{s[3]}_{s[4]}" for s in SMALL])
def test_ragged_shapes(shape):
    tokens, d_in, d_out, p, dtype = shape
    x, c, g = _problem(4242 + tokens, tokens, d_in, d_out, p, 0.05, dtype)
    got = _run(x, c, g, dtype, d_out)
    _check(x, c, g, dtype, d_out, p, got, str(shape))


@pytest.mark.parametrize("shape", LONG, ids=[f"T{s[0]}_{s[1]}x{s[2]}_p{s[3]}_{s[4]}" for s in LONG])
def test_long_blocks(shape):
    tokens, d_in, d_out, p, dtype = shape
    x, c, g = _problem(5151 + tokens, tokens, d_in, d_out, p, 0.004, dtype)
    got = _run(x, c, g, dtype, d_out)
    _check(x, c, g, dtype, d_out, p, got, str(shape), sampled=3)


@pytest.mark.parametrize("d", [16384, 32768])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_long_blocks_in_place_forward(dtype, d):
    """y may be x for long blocks too (a single circulant, and 2 x 2 blocks)."""
    tokens, p = 3, 16384
    x, c, g = _problem(77, tokens, d, d, p, 0.004, dtype)
    got = _run(x, c, g, dtype, d, alias_y=True)
    _check(x, c, g, dtype, d, p, got, "long aliased y")


# blocks beyond 8192 whose input spectra do not fit y's segments (kb > q) or a per-bin
# thread (kb > 8): one accumulating pass per input block; a 16-bit y then holds kb
# rounded partial sums of its spectrum on the way
LONG_ACCUMULATE = [
    (3, 32768, 16384, 16384, "bf16"),  # q = 1, kb = 2
    (2, 49152, 32768, 16384, "f32"),  # q = 2, kb = 3
    (2, 147456, 147456, 16384, "f32"),  # q = kb = 9
    (3, 131072, 65536, 65536, "bf16"),  # q = 1, kb = 2
    (2, 98304, 32768, 32768, "f32"),  # q = 1, kb = 3
]


@pytest.mark.parametrize("shape", LONG_ACCUMULATE, ids=[f"T{s[0]}_{s[1]}x{s[2]}_p{s[3]}_{s[4]}"
                                                        for s in LONG_ACCUMULATE])
def test_long_blocks_accumulating_forward(shape):
    tokens, d_in, d_out, p, dtype = shape
    x, c, g = _problem(6161 + tokens, tokens, d_in, d_out, p, 0.004, dtype)
    got = _run(x, c, g, dtype, d_out)
    _check(x, c, g, dtype, d_out, p, got, str(shape), sampled=5, y_staged=d_in // p + 1)


# the in-place backward for blocks beyond 8192 (dx == gy, Sec. 5.1.1): dC from the input
# transforms as they complete (float32 atomics), dX per bin over G in gy
LONG_ALIASED = [
    (3, 16384, 16384, "f32"),
    (5, 16384, 16384, "bf16"),
    (3, 32768, 16384, "bf16"),  # q = kb = 2
    (2, 131072, 16384, "f32"),  # q = kb = 8
    (4, 32768, 32768, "f32"),
    (2, 65536, 65536, "f32"),
    (2, 65536, 65536, "bf16"),
    (19, 65536, 32768, "bf16"),  # q = kb = 2, more tokens
]


@pytest.mark.parametrize("shape", LONG_ALIASED, ids=[f"T{s[0]}_{s[1]}_p{s[2]}_{s[3]}" for s in LONG_ALIASED])
def test_long_blocks_dx_over_gy(shape):
    tokens, d, p, dtype = shape
    x, c, g = _problem(7171 + tokens, tokens, d, d, p, 0.004, dtype)
    got = _run(x, c, g, dtype, d, alias_dx=True)
    _check(x, c, g, dtype, d, p, got, f"{shape} dx over gy", sampled=7)
    got = _run(x, c, g, dtype, d, alias_y=True, alias_dx=True)
    _check(x, c, g, dtype, d, p, got, f"{shape} y over x, dx over gy")


def test_long_blocks_in_place_beyond_eight_blocks_unsupported():
    """In place, a per-bin product holds at most 8 blocks: q = kb = 9 is refused before any launch."""
    tokens, d, p = 1, 147456, 16384
    x = torch.zeros((tokens, d), device="cuda")
    c = torch.zeros((9, 9, p), device="cuda")
    dc = torch.empty((9, 9, p), device="cuda")
    with pytest.raises(api.RdfftError):
        api.bca_forward(x, c, x)
    g = x.clone()
    with pytest.raises(api.RdfftError):
        api.bca_backward(x, c, g, g, dc)


# square layers with enough tokens for the two-stage dC sum (dx apart from gy); 2048 bf16
# tokens fill exactly the tiles it needs, 4093 leave a partial last tile; with dx == gy the
# same shapes take the atomics
STAGED = [(4096, 4096, 1024, "f32", False), (2048, 4096, 1024, "bf16", False), (4093, 4096, 1024, "bf16", False),
          (4096, 4096, 1024, "bf16", True)]


@pytest.mark.parametrize("shape", STAGED, ids=[f"T{s[0]}_{s[1]}_p{s[2]}_{s[3]}_{'aliased' if s[4] else 'apart'}"
                                               for s in STAGED])
def test_square_layer_dc_sums(shape):
    tokens, d, p, dtype, alias = shape
    x, c, g = _problem(606 + tokens, tokens, d, d, p, 0.01, dtype)
    got = _run(x, c, g, dtype, d, alias_dx=alias)
    _check(x, c, g, dtype, d, p, got, str(shape))


# float16 storage: the 256-, 768- and 4096-wide paper-shaped layers at full size, the
# 8192-wide circulant, and shapes that reach every other kernel family (general kernels,
# split dC, blocks beyond 8192, the fused single-circulant row kernel)
F16 = [
    (128, 256, 256, 64, 0.02, 17),
    (4096, 768, 768, 256, 0.02, 17),
    (4096, 4096, 4096, 1024, 0.01, 17),
    (96, 8192, 8192, 8192, 0.02, 0),
    (37, 512, 256, 128, 0.05, 0),
    (5, 4096, 4096, 128, 0.05, 0),
    (3, 16384, 16384, 16384, 0.004, 3),
    (6, 32768, 32768, 32768, 0.004, 0),
]


@pytest.mark.parametrize("shape", F16, ids=[f"T{s[0]}_{s[1]}x{s[2]}_p{s[3]}" for s in F16])
def test_f16_layers(shape):
    tokens, d_in, d_out, p, sigma, sampled = shape
    x, c, g = _problem(9090 + tokens, tokens, d_in, d_out, p, sigma, "f16")
    got = _run(x, c, g, "f16", d_out)
    _check(x, c, g, "f16", d_out, p, got, f"f16 {shape}", sampled=sampled)


# square layers with blocks of 128 ... 512 (the wave kernels): every block count they take, token
# counts that leave a partial last group, that stage the dC sums (every workgroup's first groups
# whole) or add them with atomics, and dx over gy; shapes past their limits fall back to the
# square kernels (p = 256 with 4 x 4 blocks backward, p = 512 with 3 x 3 blocks)
WAVE = [
    (37, 128, 128, "bf16", False),
    (21, 256, 128, "f32", False),
    (13, 384, 128, "bf16", True),
    (9, 512, 128, "f16", False),
    (4104, 512, 128, "bf16", False),
    (11, 256, 256, "f32", True),
    (4099, 768, 256, "bf16", False),
    (4100, 768, 256, "f16", True),
    (333, 1024, 256, "bf16", False),
    (29, 512, 512, "bf16", False),
    (2048, 1024, 512, "f32", False),
    (2053, 1024, 512, "bf16", True),
    (19, 1536, 512, "bf16", False),
]


@pytest.mark.parametrize("shape", WAVE, ids=[f"T{s[0]}_{s[1]}_p{s[2]}_{s[3]}{'_aliased' if s[4] else ''}" for s in WAVE])
def test_wave_kernel_layers(shape):
    tokens, d, p, dtype, alias = shape
    x, c, g = _problem(3131 + tokens, tokens, d, d, p, 0.05, dtype)
    got = _run(x, c, g, dtype, d, alias_dx=alias)
    _check(x, c, g, dtype, d, p, got, f"wave {shape}")


# square layers whose dC slots exceed LDS, with dx == gy: the dC launches read gy, so they
# must all run before the dx launch overwrites it
SPLIT_ALIASED = [(5, 4096, 128, "bf16"), (3, 4096, 512, "f32"), (4, 4096, 512, "bf16"), (3, 8192, 1024, "bf16")]


@pytest.mark.parametrize("shape", SPLIT_ALIASED, ids=[f"T{s[0]}_{s[1]}_p{s[2]}_{s[3]}" for s in SPLIT_ALIASED])
def test_split_dc_with_dx_over_gy(shape):
    tokens, d, p, dtype = shape
    x, c, g = _problem(808 + tokens, tokens, d, d, p, 0.02, dtype)
    got = _run(x, c, g, dtype, d, alias_dx=True)
    _check(x, c, g, dtype, d, p, got, f"{shape} dx over gy")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_in_place_layer(dtype):
    """y may be x itself, and dx may be gy itself, when d_in == d_out."""
    tokens, d, p = 67, 512, 128
    x, c, g = _problem(99, tokens, d, d, p, 0.05, dtype)
    got = _run(x, c, g, dtype, d, alias_y=True, alias_dx=True)
    _check(x, c, g, dtype, d, p, got, "aliased")


def test_zero_tokens_zeroes_dc():
    d, p = 256, 64
    c = to_device(inputs.circulant_spectra(inputs.generator(5), 4, 4, p, 0.02, "f32"), "f32")
    x = torch.empty((0, d), device="cuda")
    y = torch.empty((0, d), device="cuda")
    api.bca_forward(x, c, y)
    dc = torch.full((4, 4, p), 7.0, device="cuda")
    api.bca_backward(x, c, y, y, dc)
    torch.cuda.synchronize()
    assert torch.count_nonzero(dc) == 0


def test_dc_overwritten_not_accumulated():
    tokens, d, p = 16, 256, 64
    x, c, g = _problem(123, tokens, d, d, p, 0.02, "f32")
    a = _run(x, c, g, "f32", d)[2]
    b = _run(x, c, g, "f32", d)[2]
    np.testing.assert_allclose(a, b, rtol=1e-6, atol=1e-6 * np.abs(a).max())


@pytest.mark.parametrize("tokens,d,p", [(512, 4096, 1024), (4096, 4096, 1024), (64, 16384, 16384), (64, 32768, 16384)],
                         ids=["atomic_dc", "two_stage_dc", "circulant_16384", "long_blocks_2x2"])
def test_no_device_allocation(tokens, d, p):
    x, c, g = _problem(7, tokens, d, d, p, 0.01, "bf16")
    xt, ct, gt = to_device(x, "bf16"), to_device(c, "bf16"), to_device(g, "bf16")
    yt = torch.empty_like(xt)
    dxt = torch.empty_like(xt)
    dct = torch.empty(c.shape, dtype=torch.float32, device="cuda")
    api.bca_forward(xt, ct, yt)
    api.bca_backward(xt, ct, gt, dxt, dct)
    torch.cuda.synchronize()
    alloc0 = torch.cuda.memory_allocated()
    free0, _ = torch.cuda.mem_get_info()
    for _ in range(3):
        api.bca_forward(xt, ct, yt)
        api.bca_backward(xt, ct, gt, dxt, dct)
    torch.cuda.synchronize()
    assert torch.cuda.memory_allocated() == alloc0
    assert torch.cuda.mem_get_info()[0] == free0


@pytest.mark.parametrize("tokens,d,p,dtype", [(37, 256, 64, "f32"), (64, 768, 256, "bf16"), (96, 4096, 1024, "bf16"),
                                              (48, 8192, 8192, "bf16"), (8, 65536, 65536, "f32")],
                         ids=["p64_f32", "p256_bf16", "p1024_bf16", "p8192_bf16", "p65536_f32"])
def test_impulse_circulants_shift(tokens, d, p, dtype):
    """With c_ij an impulse at s_ij the layer is a sum of circular shifts, by the definition of a
    circulant (first column c): y_i = sum_j roll(x_j, s_ij) and dx_j = sum_i roll(g_i, -s_ij).
    The spectra are the impulses' closed-form transforms (no oracle, no library transform), and
    dc is checked against the cross-correlation theorem with NumPy's float64 FFT."""
    q = d // p
    rng = np.random.default_rng(2511 + p)
    shifts = rng.integers(0, p, size=(q, q))
    shifts[rng.random((q, q)) < 0.3] = -1  # some zero blocks
    spectra = impulse_spectra(shifts, p)
    x = rng.standard_normal((tokens, d))
    g = rng.standard_normal((tokens, d))
    xs, gs, cs = (inputs.round_to(a, dtype) for a in (x, g, spectra))
    xt, gt, ct = to_device(xs, dtype), to_device(gs, dtype), to_device(cs, dtype)
    yt = torch.empty((tokens, d), dtype=TORCH_DTYPE[dtype], device="cuda")
    dxt = torch.empty_like(yt)
    dct = torch.empty((q, q, p), dtype=torch.float32, device="cuda")
    api.bca_forward(xt, ct, yt)
    api.bca_backward(xt, ct, gt, dxt, dct)
    torch.cuda.synchronize()
    x64, g64 = inputs.to_f64(xs, dtype).reshape(tokens, q, p), inputs.to_f64(gs, dtype).reshape(tokens, q, p)
    y_ref = np.zeros((tokens, q, p))
    dx_ref = np.zeros((tokens, q, p))
    for i in range(q):
        for j in range(q):
            s = shifts[i, j]
            if s >= 0:
                y_ref[:, i] += np.roll(x64[:, j], s, axis=1)
                dx_ref[:, j] += np.roll(g64[:, i], -s, axis=1)
    # the stored spectra are the impulses' transforms rounded to the storage type, so the effective
    # circulants are impulses up to that rounding: the storage type's relative bar applies
    bar = 1e-5 if dtype == "f32" else 2e-2
    for name, got, ref in (("y", yt, y_ref), ("dx", dxt, dx_ref)):
        got = to_host_f64(got).reshape(ref.shape)
        err = np.linalg.norm(got - ref) / np.linalg.norm(ref)
        assert err <= bar, f"{name}: rel-L2 {err:.3e} > {bar}"
    # dc does not depend on c: dc_ij[r] = sum_t sum_m g_i[m] x_j[m - r], a circular
    # cross-correlation, i.e. sum_t IDFT(DFT(g_i) conj(DFT(x_j))); float32 arithmetic on exactly
    # widened inputs, except that blocks beyond 8192 store their spectra in the storage type
    G, X = np.fft.rfft(g64, axis=2), np.fft.rfft(x64, axis=2)
    dc_ref = np.fft.irfft(np.einsum("tik,tjk->ijk", G, np.conj(X)), n=p, axis=2)
    dc_bar = 2e-2 if (dtype == "bf16" and p > 8192) else 1e-5
    got = dct.cpu().numpy().astype(np.float64)
    err = np.linalg.norm(got - dc_ref) / np.linalg.norm(dc_ref)
    assert err <= dc_bar, f"dc: rel-L2 {err:.3e} > {dc_bar}"
