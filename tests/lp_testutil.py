"""Shared helpers for the GPU parity tests: move seeded workload inputs to the
GPU, call the library through its binding, and compare with the oracle."""
from __future__ import annotations

import numpy as np
import torch

import oracle as O
from paper_1812_04352_amd import lp as L
from workloads import CONV, Workload, generate

# Tolerances of the parity bar: normwise relative error against the fp64 oracle
# run on the same dtype-rounded inputs.
TOL = {"f32": 1e-5, "f64": 1e-12}


def rel(a, b) -> float:
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    den = np.linalg.norm(b.ravel())
    return float(np.linalg.norm((a - b).ravel()) / (den if den > 0 else 1.0))


def assert_close(gpu, ref, dtype: str, what: str, scale: float = 1.0) -> None:
    """Normwise relative error <= tol, and every element within tol * max|ref|
    (the element-by-element check; a single flipped ReLU derivative moves an
    element by O(h) and is caught here only if it breaks the normwise bar)."""
    tol = TOL[dtype] * scale
    g = np.asarray(gpu, dtype=np.float64)
    r = np.asarray(ref, dtype=np.float64)
    assert g.shape == r.shape, (what, g.shape, r.shape)
    assert np.all(np.isfinite(g)), f"{what}: non-finite GPU values"
    e = rel(g, r)
    assert e <= tol, f"{what}: normwise relative error {e:.3e} > {tol:.1e}"
    amax = float(np.max(np.abs(r))) if r.size else 0.0
    emax = float(np.max(np.abs(g - r))) if r.size else 0.0
    assert emax <= 10 * tol * max(amax, 1e-300), f"{what}: max element error {emax:.3e} vs max|ref| {amax:.3e}"


def tdt(wl: Workload):
    return torch.float32 if wl.dtype == "f32" else torch.float64


def dev(x, wl: Workload):
    return torch.from_numpy(np.ascontiguousarray(x)).to(device="cuda", dtype=tdt(wl))


def prob(wl: Workload, B: int | None = None) -> L.LpProblem:
    return L.problem(wl.dtype, wl.layer, wl.act, wl.N, wl.B if B is None else B, wl.C, wl.H, wl.W, wl.h)


def sched(wl: Workload, iters: int, relax: str | None = None, levels: int | None = None, warm=False,
          rtol=0.0, stag=0.0, cycle: str | None = None) -> L.LpMgrit:
    return L.mgrit(cf=wl.cf, max_levels=wl.max_levels if levels is None else levels, min_coarse=wl.min_coarse,
                   relax=wl.relax if relax is None else relax, max_iter=iters, warm_start=warm, rtol=rtol,
                   stag=stag, cycle=wl.cycle if cycle is None else cycle)


def state_shape(wl: Workload, rows: int, B: int | None = None):
    Bn = wl.B if B is None else B
    return (rows, Bn, wl.C, wl.H, wl.W) if wl.layer == CONV else (rows, Bn, wl.q)


class Case:
    """Inputs of one workload on both sides: numpy (oracle) and torch (GPU)."""

    def __init__(self, wl: Workload):
        self.wl = wl
        self.d = generate(wl)
        d = self.d
        self.K, self.b = dev(d["K"], wl), dev(d["b"], wl)
        self.W, self.mu = dev(d["W"], wl), dev(d["mu"], wl)
        self.y = dev(d["y"], wl)
        self.onehot = dev(d["onehot"], wl)
        self.L_in = dev(d["L_in"], wl) if d["L_in"] is not None else None
        self.p = prob(wl)
        # u^0 on each side, computed independently
        self.u0_ref = O.open_forward(d["y"], d["L_in"], wl.act, wl.opening)
        self.u0 = torch.empty(state_shape(wl, 1)[1:], device="cuda", dtype=tdt(wl))
        L.lp_open_forward(self.p, L.OPENING[wl.opening], wl.n_features, self.y, self.L_in, self.u0)

    def new_traj(self):
        U = torch.zeros(state_shape(self.wl, self.wl.N + 1), device="cuda", dtype=tdt(self.wl))
        U[0] = self.u0
        return U

    def ref_traj(self):
        U = np.zeros(state_shape(self.wl, self.wl.N + 1))
        U[0] = self.u0_ref
        return U
