"""Shared helpers for the GPU parity tests: cached workloads and factor
fixtures, device upload, and the error metrics used for parity.

Parity metric: the relative Frobenius error ||gpu - oracle|| / ||oracle|| per
output tensor, at most 1e-5 for float32 inputs and 2e-2 for bfloat16 inputs,
and no non-finite values."""
from __future__ import annotations

import functools
import os

import numpy as np
import torch

import workloads

HERE = os.path.dirname(os.path.abspath(__file__))
FACTORS = os.path.join(HERE, "golden", "factors")
TOL_F32 = 1e-5
TOL_BF16 = 2e-2


def load_factors(L: int, R: int):
    z = np.load(os.path.join(FACTORS, f"cp_L{L}_R{R}.npz"))
    return z["A"], z["B"], z["D"]


@functools.lru_cache(maxsize=None)
def workload(name: str) -> dict:
    return workloads.make_workload(name)


def random_factors(L: int, R: int, seed: int):
    rng = np.random.default_rng(seed)
    d = (L + 1) ** 2
    return tuple((rng.standard_normal((d, R)) / np.sqrt(d)).astype(np.float32) for _ in range(3))


def device_inputs(w: dict, A, B, D, dev="cuda"):
    bf16 = w["feat_dtype"] == "bf16"
    t = lambda a, dt=torch.float32: torch.from_numpy(np.ascontiguousarray(a)).to(dev, dt)  # noqa: E731
    if bf16:
        x = torch.from_numpy(w["x_bf16"].view(np.int16)).to(dev).view(torch.bfloat16)
        W = torch.from_numpy(w["W_bf16"].view(np.int16)).to(dev).view(torch.bfloat16)
    else:
        x, W = t(w["x"]), t(w["W"])
    return dict(x=x, edge_vec=t(w["edge_vec"]), edge_index=torch.from_numpy(w["edge_index"]).to(dev),
                A=t(A), B=t(B), D=t(D), W=W, radial_w=t(w["radial_w"]))


def rel_err(gpu, ref) -> float:
    """Relative Frobenius error; with TDN_PARITY_LOG set, each value is also
    appended to that file with the running test's id."""
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    assert np.all(np.isfinite(gpu)), "non-finite values in GPU output"
    nrm = np.linalg.norm(ref)
    err = float(np.linalg.norm(gpu - ref) / (nrm if nrm > 0 else 1.0))
    log = os.environ.get("TDN_PARITY_LOG")
    if log:
        test = os.environ.get("PYTEST_CURRENT_TEST", "?").split(" ")[0]
        with open(log, "a") as f:
            f.write(f"{test}\t{gpu.shape}\t{err:.3e}\n")
    return err


def tol(w: dict) -> float:
    return TOL_BF16 if w["feat_dtype"] == "bf16" else TOL_F32


def sample_nodes(w: dict, k: int, seed: int = 0, by: int = 1) -> np.ndarray:
    """k seeded nodes plus the first, the last and the one of largest degree
    (by=1: in-degree, by=0: out-degree)."""
    N = w["N"]
    rng = np.random.default_rng(seed)
    deg = np.bincount(w["edge_index"][by], minlength=N)
    extra = [0, N - 1, int(np.argmax(deg))]
    return np.unique(np.concatenate([rng.choice(N, size=min(k, N), replace=False), extra]))
