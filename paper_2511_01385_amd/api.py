"""PyTorch-facing binding of the C ABI (same names as include/rdfft.h).

Torch supplies device memory and the current stream; every call passes raw
pointers and sizes to ``librdfft.so`` and checks the returned status.  No torch
operation touches the data.
"""

from __future__ import annotations

import ctypes

import torch

from . import _lib


class RdfftError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: {_lib.status_string(status)}")
        self.status = status


def _code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return _lib.RDFFT_F32
    if t.dtype == torch.bfloat16:
        return _lib.RDFFT_BF16
    if t.dtype == torch.float16:
        return _lib.RDFFT_F16
    raise TypeError(f"rdfft supports float32, bfloat16 and float16 storage, got {t.dtype}")


def _dev(t: torch.Tensor, name: str) -> int:
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t.data_ptr()


def _stream(t: torch.Tensor) -> int:
    if t.device.index is not None and t.device.index != torch.cuda.current_device():
        # the library works on the current device
        raise ValueError(f"tensor on {t.device}, current device is cuda:{torch.cuda.current_device()}")
    return torch.cuda.current_stream(t.device).cuda_stream


def _check(status: int, what: str) -> None:
    if status != _lib.RDFFT_OK:
        raise RdfftError(status, what)


def rdfft_forward(buf: torch.Tensor) -> torch.Tensor:
    """In place: each row (last dim n) becomes its packed spectrum.  Returns ``buf``."""
    n = buf.shape[-1]
    rows = buf.numel() // n if n else 0
    _check(_lib.load().rdfft_forward(_dev(buf, "buf"), rows, n, _code(buf), _stream(buf)), "rdfft_forward")
    return buf


def rdfft_inverse(buf: torch.Tensor) -> torch.Tensor:
    """In place: each packed spectrum row becomes its real signal.  Returns ``buf``."""
    n = buf.shape[-1]
    rows = buf.numel() // n if n else 0
    _check(_lib.load().rdfft_inverse(_dev(buf, "buf"), rows, n, _code(buf), _stream(buf)), "rdfft_inverse")
    return buf


def rdfft_forward_halfcomplex(buf: torch.Tensor) -> torch.Tensor:
    """In place: each row becomes its packed spectrum in the halfcomplex layout.  Returns ``buf``."""
    n = buf.shape[-1]
    rows = buf.numel() // n if n else 0
    st = _lib.load().rdfft_forward_halfcomplex(_dev(buf, "buf"), rows, n, _code(buf), _stream(buf))
    _check(st, "rdfft_forward_halfcomplex")
    return buf


def rdfft_inverse_halfcomplex(buf: torch.Tensor) -> torch.Tensor:
    """In place: each halfcomplex-layout spectrum row becomes its real signal.  Returns ``buf``."""
    n = buf.shape[-1]
    rows = buf.numel() // n if n else 0
    st = _lib.load().rdfft_inverse_halfcomplex(_dev(buf, "buf"), rows, n, _code(buf), _stream(buf))
    _check(st, "rdfft_inverse_halfcomplex")
    return buf


def rdfft_pairs_to_halfcomplex(buf: torch.Tensor) -> torch.Tensor:
    """In place: each packed spectrum row moves from the pairs to the halfcomplex layout."""
    n = buf.shape[-1]
    rows = buf.numel() // n if n else 0
    st = _lib.load().rdfft_pairs_to_halfcomplex(_dev(buf, "buf"), rows, n, _code(buf), _stream(buf))
    _check(st, "rdfft_pairs_to_halfcomplex")
    return buf


def rdfft_halfcomplex_to_pairs(buf: torch.Tensor) -> torch.Tensor:
    """In place: each packed spectrum row moves from the halfcomplex to the pairs layout."""
    n = buf.shape[-1]
    rows = buf.numel() // n if n else 0
    st = _lib.load().rdfft_halfcomplex_to_pairs(_dev(buf, "buf"), rows, n, _code(buf), _stream(buf))
    _check(st, "rdfft_halfcomplex_to_pairs")
    return buf


def _layer_shapes(x: torch.Tensor, c_spectra: torch.Tensor, out: torch.Tensor, out_name: str):
    """(q, kb, p, tokens) after checking that the tensors agree with each other.

    The library sees only pointers and sizes, so a tensor of the wrong shape, storage type
    or device would make it read or write outside that tensor; those are refused here.
    """
    if c_spectra.dim() != 3:
        raise ValueError(f"c_spectra must have shape (q, kb, p), got {tuple(c_spectra.shape)}")
    q, kb, p = c_spectra.shape
    if x.dim() != 2 or x.shape[1] != kb * p:
        raise ValueError(f"x must have shape (tokens, {kb * p}), got {tuple(x.shape)}")
    tokens = x.shape[0]
    if tuple(out.shape) != (tokens, q * p):
        raise ValueError(f"{out_name} must have shape ({tokens}, {q * p}), got {tuple(out.shape)}")
    for name, t in (("c_spectra", c_spectra), (out_name, out)):
        if t.dtype != x.dtype:
            raise TypeError(f"{name} is {t.dtype}, x is {x.dtype}")
        if t.device != x.device:
            raise ValueError(f"{name} is on {t.device}, x on {x.device}")
    return q, kb, p, tokens


def bca_forward(x: torch.Tensor, c_spectra: torch.Tensor, y: torch.Tensor) -> torch.Tensor:
    """y[t] = W x[t] for the block-circulant W whose packed block spectra are ``c_spectra`` (q, kb, p)."""
    q, kb, p, tokens = _layer_shapes(x, c_spectra, y, "y")
    st = _lib.load().bca_forward(
        _dev(x, "x"), _dev(c_spectra, "c_spectra"), _dev(y, "y"), None,
        kb * p, q * p, p, tokens, _code(x), _stream(x),
    )
    _check(st, "bca_forward")
    return y


def bca_backward(x: torch.Tensor, c_spectra: torch.Tensor, gy: torch.Tensor, dx: torch.Tensor, dc: torch.Tensor):
    """Writes dL/dx into ``dx`` and dL/dc (float32, time domain, shape (q, kb, p)) into ``dc``.

    ``gy`` is left unspecified; ``dx`` may be ``gy`` itself when d_in == d_out (for blocks
    beyond 8192, with at most 8 blocks per row).
    """
    q, kb, p, tokens = _layer_shapes(x, c_spectra, gy, "gy")
    if tuple(dx.shape) != tuple(x.shape) or dx.dtype != x.dtype or dx.device != x.device:
        raise ValueError(f"dx must match x: {tuple(x.shape)} {x.dtype} on {x.device}")
    if tuple(dc.shape) != (q, kb, p) or dc.device != x.device:
        raise ValueError(f"dc must have shape ({q}, {kb}, {p}) on {x.device}, got {tuple(dc.shape)}")
    if dc.dtype != torch.float32:
        raise TypeError("dc is float32")
    grads = _lib.BcaGrads(_dev(dx, "dx"), _dev(dc, "dc"))
    st = _lib.load().bca_backward(
        _dev(x, "x"), _dev(c_spectra, "c_spectra"), _dev(gy, "gy"), ctypes.byref(grads),
        kb * p, q * p, p, tokens, _code(x), _stream(x),
    )
    _check(st, "bca_backward")
    return dx, dc


def _pointer_array(ts, name):
    return (ctypes.c_void_p * len(ts))(*[_dev(t, f"{name}[{i}]") for i, t in enumerate(ts)])


def _batch_shapes(xs, cs, outs, out_name):
    if not (len(xs) == len(cs) == len(outs)):
        raise ValueError("one x, c_spectra and output per layer")
    shapes = {_layer_shapes(x, c, o, out_name) for x, c, o in zip(xs, cs, outs)}
    if len(shapes) != 1 or len({x.dtype for x in xs}) != 1 or len({x.device for x in xs}) != 1:
        raise ValueError("the layers of a batch share one shape, storage type and device")
    return shapes.pop()


def bca_forward_batched(xs, c_spectras, ys):
    """``bca_forward`` for several independent layers of one shape (lists of tensors), in one call."""
    if len(xs) == 0:
        return ys
    q, kb, p, tokens = _batch_shapes(xs, c_spectras, ys, "y")
    st = _lib.load().bca_forward_batched(
        len(xs), _pointer_array(xs, "x"), _pointer_array(c_spectras, "c_spectra"), _pointer_array(ys, "y"),
        kb * p, q * p, p, tokens, _code(xs[0]), _stream(xs[0]),
    )
    _check(st, "bca_forward_batched")
    return ys


def bca_backward_batched(xs, c_spectras, gys, dxs, dcs):
    """``bca_backward`` for several independent layers of one shape (lists of tensors), in one call."""
    if len(xs) == 0:
        return dxs, dcs
    q, kb, p, tokens = _batch_shapes(xs, c_spectras, gys, "gy")
    if not (len(dxs) == len(dcs) == len(xs)):
        raise ValueError("one dx and dc per layer")
    for x, dx, dc in zip(xs, dxs, dcs):
        if tuple(dx.shape) != tuple(x.shape) or dx.dtype != x.dtype or dx.device != x.device:
            raise ValueError(f"dx must match x: {tuple(x.shape)} {x.dtype} on {x.device}")
        if tuple(dc.shape) != (q, kb, p) or dc.device != x.device or dc.dtype != torch.float32:
            raise ValueError(f"dc must be float32 of shape ({q}, {kb}, {p}) on {x.device}")
    grads = (_lib.BcaGrads * len(xs))(*[_lib.BcaGrads(_dev(dx, "dx"), _dev(dc, "dc")) for dx, dc in zip(dxs, dcs)])
    st = _lib.load().bca_backward_batched(
        len(xs), _pointer_array(xs, "x"), _pointer_array(c_spectras, "c_spectra"), _pointer_array(gys, "gy"), grads,
        kb * p, q * p, p, tokens, _code(xs[0]), _stream(xs[0]),
    )
    _check(st, "bca_backward_batched")
    return dxs, dcs


def rdfft_init() -> None:
    _check(_lib.load().rdfft_init(), "rdfft_init")


def rdfft_table_bytes() -> int:
    return int(_lib.load().rdfft_table_bytes())
