"""Writes the coefficient tensor of the exact CG tensor product for the GPU
comparator kernel, one file per maximum degree L = 0..6:

    tests/golden/cg/cg_L{L}.npz   M [d, d, d] float64 (oracle.cg_tensor,
                                  index order k, i, j) and path [d, d, d]
                                  int16, the index in oracle.cg_tensor.paths(L)
                                  of the path whose block holds each entry
                                  (-1 outside every block)

Run:  python tests/golden/make_cg.py
"""
from __future__ import annotations

import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

from oracle import cg_tensor, dense_layer  # noqa: E402


def main():
    os.makedirs(os.path.join(HERE, "cg"), exist_ok=True)
    for L in range(7):
        M = np.asarray(cg_tensor.cg_tensor(L))
        P = dense_layer.path_index(L).astype(np.int16)
        np.savez_compressed(os.path.join(HERE, "cg", f"cg_L{L}.npz"), M=M, path=P)
        print(L, int(np.count_nonzero(M)), len(cg_tensor.paths(L)))


if __name__ == "__main__":
    main()
