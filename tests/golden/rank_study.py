"""Rank study of the CP approximation of the CG tensor (data-free): for each
maximum degree L and a grid of ranks R around the paper's schedule R = 7 L^2
(Sec. 4.1 "Model Design"; the paper's rank figures carry no values), fits M
by the oracle's CP-ALS and records

    rel_frobenius_error      ||M - M_hat||_F / ||M||_F
    approximation_error      mean over unit random x, y of
                             ||M(x (x) y) - M_hat(x (x) y)|| / ||M(x (x) y)||   (Sec. 4.1)
    equivariance_error       mean eps(R, x, y) over random rotations (Sec. 3.4)
    tucker_tail              the singular-value tail bound of Thm. 1

into tests/golden/rank_study.json.  Settings: ALS from one seeded N(0,1)
start, ridge 1e-3 x mean Gram diagonal, at most 500 sweeps; 200 samples per
metric.

Run:  python tests/golden/rank_study.py [L ...]
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

MULTIPLES = (1, 2, 4, 7, 10)
OUT = os.path.join(HERE, "rank_study.json")


def study(L: int) -> list[dict]:
    M = cg_tensor.cg_tensor(L)
    d = (L + 1) ** 2
    rng = np.random.default_rng(100 + L)
    x, y = rng.normal(size=(2, 200, d))
    x /= np.linalg.norm(x, axis=1, keepdims=True)
    y /= np.linalg.norm(y, axis=1, keepdims=True)
    rots = [wigner.wigner_d_full(L, wigner.random_rotation(rng)) for _ in range(200)]
    ranks = sorted({min(k * L * L, d * d) for k in MULTIPLES})
    rows = []
    for R in ranks:
        t0 = time.time()
        D, A, B, err = cp.cp_fit(M, R, seed=7 * L + R, restarts=1, max_sweeps=500, ridge=1e-3)
        eq = float(np.mean([cp.equivariance_error(D, A, B, rots[i], x[i:i + 1], y[i:i + 1])[0]
                            for i in range(200)]))
        rows.append(dict(L=L, d=d, R=R, R_over_L2=R / (L * L), rel_frobenius_error=float(err),
                         approximation_error=float(np.mean(cp.approximation_error(M, D, A, B, x, y))),
                         equivariance_error=eq, tucker_tail=float(cp.tucker_tail(M, R)),
                         seconds=time.time() - t0))
        print(json.dumps(rows[-1]), flush=True)
    return rows


def main(argv):
    Ls = [int(a) for a in argv] or [1, 2, 3, 4, 5, 6]
    res = json.load(open(OUT)) if os.path.exists(OUT) else {}
    for L in Ls:
        res[f"L{L}"] = study(L)
        json.dump(res, open(OUT, "w"), indent=1)


if __name__ == "__main__":
    main(sys.argv[1:])
