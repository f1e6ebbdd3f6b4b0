"""Peak device memory of one block-circulant layer's forward + backward.

The single-layer harness of the paper's memory study (Sec. 5.1, Table 1): for
synthetic x of shape (B, D), D in {1024, 4096}, B in {1, 16, 256} and block sizes p
from 128 to 4096, it runs ``BlockCirculantLinear`` forward and backward once and
reports the peak of ``torch.cuda.max_memory_allocated`` above what was allocated
before the call (the layer's parameter, x and the upstream gradient already resident).
Only this library's path is measured.

    python -m paper_2511_01385_amd.memory_harness [--dtype bf16|f32] [--json]
"""

from __future__ import annotations

import argparse
import json

import torch

from .layer import BlockCirculantLinear

DIMS = (1024, 4096)
BATCHES = (1, 16, 256)
BLOCKS = (128, 256, 512, 1024, 2048, 4096)


def measure(d: int, batch: int, p: int, dtype: torch.dtype, clobber_grad: bool = False) -> dict:
    dev = torch.device("cuda")
    torch.manual_seed(1385 + d + batch + p)
    layer = BlockCirculantLinear(d, d, p, dtype=dtype, device=dev, clobber_grad=clobber_grad)
    x = torch.randn(batch, d, device=dev).to(dtype).requires_grad_(True)
    g = torch.randn(batch, d, device=dev).to(dtype)
    # warm-up: library load, twiddle upload, kernel code objects
    layer(x).backward(g.clone())
    x.grad = None
    layer.c.grad = None
    torch.cuda.synchronize()
    torch.cuda.reset_peak_memory_stats()
    base = torch.cuda.memory_allocated()
    y = layer(x)
    after_fwd = torch.cuda.memory_allocated() - base
    y.backward(g)
    torch.cuda.synchronize()
    peak = torch.cuda.max_memory_allocated() - base
    s = torch.finfo(dtype).bits // 8
    q = kb = d // p
    return {
        "D": d, "B": batch, "p": p, "dtype": str(dtype).replace("torch.", ""), "clobber_grad": clobber_grad,
        "peak_bytes": int(peak), "after_forward_bytes": int(after_fwd),
        "param_bytes": q * kb * p * 4, "spectra_bytes": q * kb * p * s, "activation_bytes": batch * d * s,
        "dense_weight_bytes": d * d * s,
    }


def main() -> None:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--dtype", choices=("bf16", "f32"), default="bf16")
    ap.add_argument("--json", action="store_true", help="one JSON object per line instead of a table")
    args = ap.parse_args()
    dtype = torch.bfloat16 if args.dtype == "bf16" else torch.float32
    rows = []
    for d in DIMS:
        for batch in BATCHES:
            for p in BLOCKS:
                if p > d:
                    continue
                for clobber in (False, True):
                    rows.append(measure(d, batch, p, dtype, clobber))
                    if args.json:
                        print(json.dumps(rows[-1]), flush=True)
    if not args.json:
        print("| D | B | p | grad buffer | peak extra bytes | after forward | spectra | x | dense W (for scale) |")
        print("|---|---|---|---|---|---|---|---|---|")
        for r in rows:
            print(f"| {r['D']} | {r['B']} | {r['p']} | {'reused' if r['clobber_grad'] else 'copied'} | "
                  f"{r['peak_bytes']} | {r['after_forward_bytes']} | {r['spectra_bytes']} | "
                  f"{r['activation_bytes']} | {r['dense_weight_bytes']} |")


if __name__ == "__main__":
    main()
