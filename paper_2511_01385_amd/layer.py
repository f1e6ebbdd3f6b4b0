"""PyTorch autograd wrapper of the block-circulant layer (Sec. 3.3, Eqs. (4)-(5)).

``BlockCirculantLinear`` holds the time-domain first columns c of its q x kb circulant
blocks as a float32 parameter (the float32 gradients of Sec. 5 train it directly).
Every forward rounds c to the storage type, turns it into packed block spectra with
``rdfft_forward`` and calls ``bca_forward``; the backward calls ``bca_backward``,
whose dc output is the gradient with respect to those (rounded) first columns.
All arithmetic on the data runs in the library's kernels; torch only allocates
buffers, casts the parameter and reshapes.

Memory: the forward keeps x and the packed spectra (q*kb*p storage elements) for the
backward, nothing else.  The backward needs one buffer of the upstream gradient's size,
which the library uses as work space and then fills with dx (allowed when
d_in == d_out, and for blocks longer than 8192 when there are at most 8 of them per
row; otherwise dx gets its own buffer).  With ``clobber_grad=True`` it works
in the upstream gradient tensor itself instead of a copy, as the paper does
("overwriting the grad_output", Sec. 5.1.1); only do that when nothing else reads
that gradient afterwards.
"""

from __future__ import annotations

import math

import torch

from . import api


class _BcaFunction(torch.autograd.Function):
    @staticmethod
    def forward(ctx, x2d: torch.Tensor, c: torch.Tensor, dtype: torch.dtype, clobber_grad: bool):
        q, kb, p = c.shape
        spectra = c.detach().to(dtype).contiguous()
        if spectra.data_ptr() == c.data_ptr():  # float32 layer: do not transform the parameter itself
            spectra = spectra.clone()
        api.rdfft_forward(spectra.view(q * kb, p))
        y = torch.empty((x2d.shape[0], q * p), dtype=dtype, device=x2d.device)
        api.bca_forward(x2d, spectra, y)
        ctx.save_for_backward(x2d, spectra)
        ctx.clobber_grad = clobber_grad
        return y

    @staticmethod
    def backward(ctx, gy: torch.Tensor):
        x2d, spectra = ctx.saved_tensors
        q, kb, p = spectra.shape
        gy = gy.contiguous()
        if gy.dtype != x2d.dtype:
            gy = gy.to(x2d.dtype)
        elif not ctx.clobber_grad:
            gy = gy.clone()  # the library overwrites it
        # dx may share the work buffer when the layer is square (for blocks beyond 8192, when
        # a per-bin product holds its q blocks)
        dx = gy if q == kb and (p <= 8192 or q <= 8) else torch.empty_like(x2d)
        dc = torch.empty((q, kb, p), dtype=torch.float32, device=x2d.device)
        api.bca_backward(x2d, spectra, gy, dx, dc)
        return dx, dc, None, None


class BlockCirculantLinear(torch.nn.Module):
    """y = W x with W (d_out x d_in) made of p x p circulant blocks (first columns c).

    x has shape (..., d_in) and the storage type ``dtype`` (bfloat16, float16 or float32); y has
    shape (..., d_out).  p must be a power of two with 2 <= p <= 65536 dividing d_in and
    d_out; blocks longer than 8192 also need (d_in/p)(d_out/p) <= 65535.  c is initialised N(0, sigma^2) with sigma = d_in^-1/2
    unless given.
    """

    def __init__(self, d_in: int, d_out: int, p: int, dtype: torch.dtype = torch.bfloat16,
                 device: str | torch.device = "cuda", sigma: float | None = None, clobber_grad: bool = False):
        super().__init__()
        if p < 2 or p & (p - 1):
            raise ValueError(f"p must be a power of two >= 2, got {p}")
        if d_in % p or d_out % p:
            raise ValueError(f"p = {p} must divide d_in = {d_in} and d_out = {d_out}")
        if p > 65536:
            raise ValueError(f"p = {p} is beyond the largest supported block, 65536")
        if p > 8192 and (d_in // p) * (d_out // p) > 65535:
            raise ValueError(f"blocks of p = {p} > 8192 need (d_in/p)(d_out/p) <= 65535")
        if dtype not in (torch.bfloat16, torch.float16, torch.float32):
            raise TypeError(f"storage type must be bfloat16, float16 or float32, got {dtype}")
        self.d_in, self.d_out, self.p = d_in, d_out, p
        self.dtype = dtype
        self.clobber_grad = clobber_grad
        sigma = 1.0 / math.sqrt(d_in) if sigma is None else sigma
        c = torch.randn((d_out // p, d_in // p, p), dtype=torch.float32, device=device) * sigma
        self.c = torch.nn.Parameter(c)

    def forward(self, x: torch.Tensor) -> torch.Tensor:
        if x.shape[-1] != self.d_in:
            raise ValueError(f"last dimension {x.shape[-1]} != d_in = {self.d_in}")
        if x.dtype != self.dtype:
            raise TypeError(f"input is {x.dtype}, the layer stores {self.dtype}")
        lead = x.shape[:-1]
        x2d = x.reshape(-1, self.d_in).contiguous()
        y = _BcaFunction.apply(x2d, self.c, self.dtype, self.clobber_grad)
        return y.reshape(*lead, self.d_out)

    def extra_repr(self) -> str:
        return f"d_in={self.d_in}, d_out={self.d_out}, p={self.p}, dtype={self.dtype}"
