"""Fits and caches the rank-R CP factors of the CG tensor, once per (L, R).

The paper precomputes a rank-R CP decomposition of the CG coefficient tensor
once per maximum degree, caches it, and treats it as constant (Sec. 4.1
"Model Design").  This script does that with the oracle's ALS and writes

    tests/golden/factors/cp_L{L}_R{R}.npz   A, B, D as float32 [d, R]
    tests/golden/factors/report.json        fit error, settings, diagnostics

Factor names: D is the paper's A (output mode), A is the paper's B (node
features), B is the paper's C (edge harmonics).

ALS settings (the paper leaves them open): seeded N(0,1) start, Tikhonov
ridge 1e-3 x mean Gram diagonal (keeps the rank-one components from growing
into large cancelling pairs, which would cost float32 accuracy), at most 2000
sweeps, stop when the relative error changes by < 1e-12, best of 3 seeds.

Run:  python tests/golden/make_factors.py [L R ...]
"""
from __future__ import annotations

import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

from oracle import cg_tensor, cp, wigner  # noqa: E402

SETS = [(2, 32), (3, 64), (4, 128), (6, 256)]
RIDGE = 1e-3
SEED = 20250701


def fit(L: int, R: int) -> dict:
    M = cg_tensor.cg_tensor(L)
    t0 = time.time()
    D, A, B, err = cp.cp_fit(M, R, seed=SEED + 100 * L, restarts=3, max_sweeps=2000, ridge=RIDGE)
    A32, B32, D32 = (np.asarray(a, np.float32) for a in (A, B, D))
    err32 = float(np.linalg.norm(M - cp.cp_reconstruct(D32.astype(np.float64), A32.astype(np.float64),
                                                       B32.astype(np.float64))) / np.linalg.norm(M))
    rng = np.random.default_rng(L)
    d = (L + 1) ** 2
    x, y = rng.normal(size=(2, 1000, d))
    x /= np.linalg.norm(x, axis=1, keepdims=True)
    y /= np.linalg.norm(y, axis=1, keepdims=True)
    eq = [float(np.mean(cp.equivariance_error(D, A, B, wigner.wigner_d_full(L, wigner.random_rotation(rng)),
                                              x[i:i + 1], y[i:i + 1]))) for i in range(1000)]
    path = os.path.join(HERE, "factors", f"cp_L{L}_R{R}.npz")
    os.makedirs(os.path.dirname(path), exist_ok=True)
    np.savez(path, A=A32, B=B32, D=D32)
    comp = np.linalg.norm(D, axis=0) * np.linalg.norm(A, axis=0) * np.linalg.norm(B, axis=0)
    return dict(L=L, R=R, d=d, rel_frobenius_error=err, rel_frobenius_error_f32=err32,
                mean_equivariance_error_unit_inputs=float(np.mean(eq)),
                approximation_error_mean=float(np.mean(cp.approximation_error(M, D, A, B, x, y))),
                tucker_tail=cp.tucker_tail(M, R), sum_component_norms_over_norm=float(comp.sum() / np.linalg.norm(M)),
                ridge=RIDGE, seed=SEED + 100 * L, restarts=3, max_sweeps=2000, seconds=time.time() - t0)


def main(argv):
    sets = SETS if not argv else [(int(argv[i]), int(argv[i + 1])) for i in range(0, len(argv), 2)]
    rep_path = os.path.join(HERE, "factors", "report.json")
    report = json.load(open(rep_path)) if os.path.exists(rep_path) else {}
    for L, R in sets:
        r = fit(L, R)
        report[f"L{L}_R{R}"] = r
        print(json.dumps(r), flush=True)
        os.makedirs(os.path.dirname(rep_path), exist_ok=True)
        with open(rep_path, "w") as f:
            json.dump(report, f, indent=1, sort_keys=True)


if __name__ == "__main__":
    main(sys.argv[1:])
