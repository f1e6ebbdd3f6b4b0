"""CPU oracle for the in-place real-domain FFT (rdFFT) and the block-circulant layer.

TEST INFRASTRUCTURE ONLY.  Nothing in the product library imports, links or calls
this package; only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline``
leg of ``bench.py`` may use it.  It shares no code, table or constant with the HIP
path: its arithmetic is plain NumPy in float64, written from the paper's
definitions (Memory-Efficient Training with In-Place FFT Implementation,
arXiv 2511.01385):

* ``oracle.rdfft`` -- the DFT / IDFT of Sec. 3.1 Eq. (1) restricted to the
  non-redundant bins 0..n/2 (Sec. 3.1, Theorem 1), and the packers that squeeze
  those n+2 reals into n real slots (Sec. 4.1, "Squeeze N+2 into N").
* ``oracle.bca`` -- the circulant / block-circulant linear layer of Sec. 3.3:
  the plain dense-matrix definition y = C x and its gradients, and the spectral
  form of Eqs. (4)-(5).

Every function is pinned by ``tests/test_oracle_*.py`` against closed forms,
brute-force sums, invariants and finite differences, not against itself.
"""

from . import rdfft, bca  # noqa: F401

__all__ = ["rdfft", "bca"]
