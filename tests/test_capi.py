"""C-ABI checks that need no GPU: the library loads, exports every entry point that
include/rdfft.h declares, imports no device allocator, and rejects invalid arguments
on the host before any HIP call (every case below must fail validation, so nothing
is ever launched from here)."""

import ctypes
import os
import re
import subprocess

import pytest

from paper_2511_01385_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "rdfft.h")

EINVAL, EUNSUP, OK = _lib.RDFFT_EINVAL, _lib.RDFFT_EUNSUPPORTED, _lib.RDFFT_OK
F32, BF16 = _lib.RDFFT_F32, _lib.RDFFT_BF16

# fake, never dereferenced addresses (validation rejects every call that uses them)
A = 0x7F0000000000
B = A + (1 << 30)


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(_lib.LIB_PATH):
        from paper_2511_01385_amd.build import build

        build(verbose=False)
    return _lib.load()


def _declared():
    text = open(HEADER).read()
    return re.findall(r"RDFFT_API\s+[\w\s\*]+?\b(\w+)\s*\(", text)


def test_header_declares_the_binding_names():
    assert sorted(_declared()) == sorted(_lib.EXPORTS)


def test_library_exports_every_declared_symbol(lib):
    out = subprocess.run(["nm", "-D", "--defined-only", _lib.LIB_PATH], capture_output=True, text=True, check=True).stdout
    exported = {line.split()[-1] for line in out.splitlines() if " T " in line}
    for name in _declared():
        assert name in exported, name
        assert hasattr(lib, name)
    # nothing else leaks out of the C ABI
    assert {n for n in exported if not n.startswith("_")} == set(_declared())


def test_library_imports_no_device_allocator(lib):
    out = subprocess.run(["nm", "-D", "--undefined-only", _lib.LIB_PATH], capture_output=True, text=True, check=True).stdout
    names = {line.split()[-1].split("@")[0] for line in out.splitlines() if line.strip()}
    bad = {n for n in names if re.match(r"hip(Malloc|MallocAsync|MallocManaged|HostMalloc|ExtMallocWithFlags|MallocPitch|Free|FreeAsync|HostRegister)", n)}
    assert not bad, bad


def test_status_strings(lib):
    for code in (OK, EINVAL, EUNSUP, _lib.RDFFT_ELAUNCH, _lib.RDFFT_EDEVICE):
        assert _lib.status_string(code).startswith("RDFFT_")
    assert 0 < lib.rdfft_table_bytes() < (1 << 21)


@pytest.mark.parametrize(
    "args,want",
    [
        ((0, 4, 64, F32), EINVAL),  # null buffer
        ((A + 8, 4, 64, F32), EINVAL),  # misaligned
        ((A, -1, 64, F32), EINVAL),  # negative rows
        ((A, 4, 63, F32), EINVAL),  # odd length: no Nyquist bin
        ((A, 4, 1, F32), EINVAL),
        ((A, 4, 0, F32), EINVAL),
        ((A, 4, -8, F32), EINVAL),
        ((A, 4, 64, 3), EINVAL),  # unknown dtype
        ((A, 4, 14, F32), EUNSUP),  # even, n/2 has a factor 7
        ((A, 4, 49152, F32), EUNSUP),  # n/2 = 3 * 2^13: mixed radix beyond 16384
        ((A, 4, 2 * 3**10, F32), EUNSUP),
        ((A, 4, 131072, BF16), EUNSUP),  # beyond 65536
        ((A, 4, 131072, _lib.RDFFT_F16), EUNSUP),
        ((A, 4, 22, _lib.RDFFT_F16), EUNSUP),
        ((A, 1 << 62, 65536, F32), EINVAL),  # size overflow
    ],
)
def test_transform_validation(lib, args, want):
    for fn in (lib.rdfft_forward, lib.rdfft_inverse, lib.rdfft_pairs_to_halfcomplex, lib.rdfft_halfcomplex_to_pairs):
        assert fn(args[0], args[1], args[2], args[3], None) == want


def test_zero_rows_is_a_no_op(lib):
    # returns before any HIP call, so a null buffer is fine
    assert lib.rdfft_forward(None, 0, 64, F32, None) == OK
    assert lib.rdfft_inverse(None, 0, 4096, BF16, None) == OK
    assert lib.rdfft_pairs_to_halfcomplex(None, 0, 64, BF16, None) == OK
    assert lib.rdfft_halfcomplex_to_pairs(None, 0, 65536, F32, None) == OK
    assert lib.rdfft_forward(None, 0, 2, _lib.RDFFT_F16, None) == OK
    assert lib.rdfft_inverse(None, 0, 30000, BF16, None) == OK  # mixed radix


def _grads(dx, dc):
    return ctypes.byref(_lib.BcaGrads(dx, dc))


@pytest.mark.parametrize(
    "x,c,y,d_in,d_out,p,tokens,dtype,want",
    [
        (A, B, A + (1 << 29), 256, 256, 96, 8, F32, EINVAL),  # p does not divide d
        (A, B, A + (1 << 29), 256, 192, 128, 8, F32, EINVAL),  # p does not divide d_out
        (A, B, A + (1 << 29), 96, 96, 48, 8, F32, EUNSUP),  # even, not a power of two
        (A, B, A + (1 << 29), 131072, 131072, 131072, 8, F32, EUNSUP),  # p beyond 65536
        (A, B, A, 147456, 147456, 16384, 8, F32, EUNSUP),  # long blocks in place, q = kb > 8
        (A, B, A + (1 << 29), 4194304, 4194304, 16384, 1, F32, EUNSUP),  # long blocks, q * kb > 65535
        (A, B, A + (1 << 29), 256, 256, 7, 8, F32, EINVAL),  # odd p
        (A, B, A + (1 << 29), 256, 256, 64, -1, F32, EINVAL),
        (A, B, A + (1 << 29), 0, 256, 64, 8, F32, EINVAL),
        (A, B, A + (1 << 29), 256, 256, 64, 8, 5, EINVAL),
        (A, B, A + (1 << 29), 96, 96, 48, 8, _lib.RDFFT_F16, EUNSUP),  # f16 layer, p not a power of two
        (0, B, A + (1 << 29), 256, 256, 64, 8, F32, EINVAL),  # null x
        (A, 0, A + (1 << 29), 256, 256, 64, 8, F32, EINVAL),  # null spectra
        (A, B, 0, 256, 256, 64, 8, F32, EINVAL),  # null y
        (A + 4, B, A + (1 << 29), 256, 256, 64, 8, F32, EINVAL),  # misaligned
        (A, B, A + 64, 256, 256, 64, 8, F32, EINVAL),  # y overlaps x without being x
        (A, B, A, 256, 512, 64, 8, F32, EINVAL),  # y == x needs d_in == d_out
        (A, A + 256, A + (1 << 29), 256, 256, 64, 8, F32, EINVAL),  # spectra overlap x
    ],
)
def test_bca_forward_validation(lib, x, c, y, d_in, d_out, p, tokens, dtype, want):
    assert lib.bca_forward(x, c, y, None, d_in, d_out, p, tokens, dtype, None) == want


def test_bca_forward_rejects_grads(lib):
    assert lib.bca_forward(A, B, A + (1 << 29), _grads(A, B), 256, 256, 64, 8, F32, None) == EINVAL


def test_bca_forward_zero_tokens(lib):
    assert lib.bca_forward(None, B, None, None, 256, 256, 64, 0, F32, None) == OK


G = A + (1 << 29)  # gy
DX = A + (2 << 29)
DC = A + (3 << 29)


@pytest.mark.parametrize(
    "x,gy,dx,dc,d_in,d_out,want",
    [
        (A, G, DX, 0, 256, 256, EINVAL),  # null dc
        (A, G, 0, DC, 256, 256, EINVAL),  # null dx
        (A, G, DX, DC + 4, 256, 256, EINVAL),  # misaligned dc
        (A, A + 512, DX, DC, 256, 256, EINVAL),  # gy overlaps x
        (A, G, A, DC, 256, 256, EINVAL),  # dx overlaps x
        (A, G, G, DC, 256, 512, EINVAL),  # dx == gy needs d_in == d_out
        (A, G, G + 64, DC, 256, 256, EINVAL),  # dx overlaps gy without being gy
        (A, G, DX, A + 128, 256, 256, EINVAL),  # dc overlaps x
        (A, G, DX, DX, 256, 256, EINVAL),  # dc overlaps dx
        (A, G, DX, B, 256, 256, EINVAL),  # dc overlaps the spectra
    ],
)
def test_bca_backward_validation(lib, x, gy, dx, dc, d_in, d_out, want):
    assert lib.bca_backward(x, B, gy, _grads(dx, dc), d_in, d_out, 64, 8, F32, None) == want


def test_bca_backward_long_blocks_in_place_at_most_eight_blocks(lib):
    # in place (dx == gy) beyond 8192, a per-bin product holds at most 8 blocks
    assert lib.bca_backward(A, B, G, _grads(G, DC), 147456, 147456, 16384, 8, F32, None) == EUNSUP


def _ptrs(*addrs):
    return (ctypes.c_void_p * len(addrs))(*addrs)


def test_bca_batched_validation(lib):
    """Batched layers: the count, every layer's own checks, and no layer writing where another
    layer reads or writes; these are refused before any device work (valid batches reach the
    device check, which fails without a GPU)."""
    d, p, t = 256, 64, 8
    MB = 1 << 24  # well apart
    xs, cs = _ptrs(A, A + MB), _ptrs(B, B)  # the layers may share their spectra
    assert lib.bca_forward_batched(-1, xs, cs, xs, d, d, p, t, F32, None) == EINVAL
    assert lib.bca_forward_batched(1025, xs, cs, xs, d, d, p, t, F32, None) == EINVAL
    assert lib.bca_forward_batched(0, None, None, None, d, d, p, t, F32, None) == OK
    ys = _ptrs(G, G + 64)  # the two outputs overlap
    assert lib.bca_forward_batched(2, xs, cs, ys, d, d, p, t, F32, None) == EINVAL
    ys = _ptrs(G, A + MB)  # layer 1 writes layer 1's own input (in place) - allowed
    assert lib.bca_forward_batched(2, xs, cs, ys, d, d, p, t, F32, None) == _lib.RDFFT_EDEVICE
    ys = _ptrs(A + MB, G)  # layer 0 writes layer 1's input
    assert lib.bca_forward_batched(2, xs, cs, ys, d, d, p, t, F32, None) == EINVAL
    ys = _ptrs(G, G + MB)
    assert lib.bca_forward_batched(2, _ptrs(A, A), cs, ys, d, d, p, t, F32, None) == _lib.RDFFT_EDEVICE  # shared x
    assert lib.bca_forward_batched(2, xs, cs, _ptrs(G, G + MB + 4), d, d, p, t, F32, None) == EINVAL  # misaligned
    dx0, dc0 = A + (5 << 29), A + (6 << 29)  # apart from x, the spectra and gy
    grads = (_lib.BcaGrads * 2)(_lib.BcaGrads(dx0, dc0), _lib.BcaGrads(dx0 + MB, dc0 + MB))
    gys = _ptrs(G, G + MB)
    assert lib.bca_backward_batched(2, xs, cs, gys, grads, d, d, p, t, F32, None) == _lib.RDFFT_EDEVICE
    grads = (_lib.BcaGrads * 2)(_lib.BcaGrads(dx0, dc0), _lib.BcaGrads(dx0 + MB, dc0))  # one dc for both
    assert lib.bca_backward_batched(2, xs, cs, gys, grads, d, d, p, t, F32, None) == EINVAL
    grads = (_lib.BcaGrads * 2)(_lib.BcaGrads(dx0, dc0), _lib.BcaGrads(A, dc0 + MB))  # dx over layer 0's x
    assert lib.bca_backward_batched(2, xs, cs, gys, grads, d, d, p, t, F32, None) == EINVAL
    grads = (_lib.BcaGrads * 2)(_lib.BcaGrads(G, dc0), _lib.BcaGrads(G + MB, dc0 + MB))  # dx over gy: allowed
    assert lib.bca_backward_batched(2, xs, cs, gys, grads, d, d, p, t, F32, None) == _lib.RDFFT_EDEVICE
    assert lib.bca_backward_batched(2, xs, cs, gys, None, d, d, p, t, F32, None) == EINVAL


def test_bca_backward_needs_grads(lib):
    assert lib.bca_backward(A, B, G, None, 256, 256, 64, 8, F32, None) == EINVAL


def test_header_compiles_as_c_and_links(tmp_path):
    """include/rdfft.h is plain C: a C99 program built with gcc against it links with the library and
    gets the documented answers for calls that never reach a device (empty inputs, validation)."""
    src = tmp_path / "abi.c"
    src.write_text(r'''
#include <stdio.h>
#include <string.h>
#include "rdfft.h"
int main(void) {
  rdfft_dtype_t dt = RDFFT_BF16;
  if (rdfft_forward(NULL, 0, 4096, dt, NULL) != RDFFT_OK) return 1;       /* no rows: a no-op */
  if (rdfft_inverse(NULL, 0, 96, RDFFT_F16, NULL) != RDFFT_OK) return 2;  /* mixed radix, no rows */
  if (rdfft_forward(NULL, 4, 14, RDFFT_F32, NULL) != RDFFT_EUNSUPPORTED) return 3;  /* n/2 = 7 */
  if (rdfft_forward(NULL, 4, 64, (rdfft_dtype_t)7, NULL) != RDFFT_EINVAL) return 4;
  bca_grads_t g = {NULL, NULL};
  if (bca_backward(NULL, NULL, NULL, &g, 256, 256, 64, 8, RDFFT_F32, NULL) != RDFFT_EINVAL) return 5;
  if (bca_forward(NULL, NULL, NULL, NULL, 256, 256, 96, 8, RDFFT_F32, NULL) != RDFFT_EINVAL) return 6;
  if (strncmp(rdfft_status_string(RDFFT_OK), "RDFFT_OK", 8) != 0) return 7;
  if (rdfft_table_bytes() <= 0) return 8;
  printf("ok\n");
  return 0;
}
''')
    exe = tmp_path / "abi"
    libdir = os.path.dirname(_lib.LIB_PATH)
    cmd = ["gcc", "-std=c99", "-Wall", "-Werror", f"-I{os.path.join(ROOT, 'include')}", str(src), "-o", str(exe),
           f"-L{libdir}", "-lrdfft", f"-Wl,-rpath,{libdir}"]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0 and r.stdout.strip() == "ok", (r.returncode, r.stdout, r.stderr)
