"""Matrix-core ceiling of this GPU under its power limit, through nsp_mfma_ceiling.

    python -m paper_2609_22755_amd.ceiling [PRODUCTS_PER_SIMD]

Prints, for one and two waves per SIMD, bf16-normal and zero operands and the
four operand patterns of nsp_mfma_ceiling, the time of one launch, its dense
bf16 rate against the 2516.6 TFLOP/s nominal peak and the shader clock it
implies (products per SIMD x 32 cycles over the time).  bench.py measures
pattern 0 with normal operands beside its timed steps.
"""
from __future__ import annotations

import sys

from paper_2609_22755_amd import nsp

PEAK = 2516.6


def main(argv: list[str]) -> None:
    products = int(argv[1]) if len(argv) > 1 else 1 << 21
    print(f"{'waves/SIMD':>10s} {'data':>6s} {'pattern':>7s} {'ms':>8s} {'TFLOP/s':>9s} {'% peak':>7s} {'clock GHz':>9s}")
    for waves in (1, 2):
        for zero in (False, True):
            for pattern in range(4):
                sec, tf = nsp.nsp_mfma_ceiling(pattern, zero, waves, products)
                print(f"{waves:10d} {'zero' if zero else 'normal':>6s} {pattern:7d} {sec * 1e3:8.2f} {tf:9.1f} "
                      f"{100 * tf / PEAK:6.1f}% {products * 32 / sec / 1e9:9.3f}", flush=True)


if __name__ == "__main__":
    main(sys.argv)
