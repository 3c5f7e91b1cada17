"""Simultaneous (one-shot) layer-parallel training, Algorithm 2 of the paper
(Section 4), as a host loop over the C ABI: per design update, m1 state MGRIT
iterations and m2 adjoint MGRIT iterations, each warm-started from the previous
update's iterates, the reduced gradient from the inexact state and adjoint, and
a plain gradient step on K, b, L_in, W, mu (the scaled-identity Hessian
approximation with step size lr). Every arithmetic step runs in the HIP library.
"""
from __future__ import annotations

from typing import Dict, List, Optional

import torch

from . import lp as L


class OneShotTrainer:
    """Holds the device state of one training run.

    params: dict of GPU tensors K, b, W, mu and (unless the opening is the
    identity) L_in, updated in place. y, c: inputs and class-probability rows."""

    def __init__(self, prob: L.LpProblem, mg_fwd: L.LpMgrit, mg_adj: L.LpMgrit, params: Dict[str, torch.Tensor],
                 y: torch.Tensor, c: torch.Tensor, n_classes: int, opening: int, n_features: int):
        self.p, self.mgF, self.mgA = prob, mg_fwd, mg_adj
        self.P = params
        self.y, self.c = y, c
        self.nc, self.opening, self.nf = n_classes, opening, n_features
        dt = params["K"].dtype
        shape = (prob.N + 1, prob.B) + ((prob.C, prob.H, prob.W) if prob.layer == L.LP_CONV3X3 else (prob.q,))
        self.U = torch.zeros(shape, device="cuda", dtype=dt)
        self.Lam = torch.zeros_like(self.U)
        need = max(L.lp_workspace_bytes(prob, mg_fwd), L.lp_workspace_bytes(prob, mg_adj))
        self.ws = torch.empty(need, dtype=torch.uint8, device="cuda")
        self.J = torch.zeros(1, device="cuda", dtype=torch.float64)
        self.G = {k: torch.empty_like(v) for k, v in params.items()}
        # sigma' along the forward iterate, kept for the adjoint and the gradient
        self.rec = L.alloc_dsig(prob) if L.lp_dsig_bytes(prob) else None
        self.updates = 0

    def step(self, lr: float) -> None:
        """One design update; the loss of the state iterate used for it goes to self.J."""
        P, G, p = self.P, self.G, self.p
        warm = self.updates > 0
        self.mgF.warm_start = int(warm)
        self.mgA.warm_start = int(warm)
        L.lp_open_forward(p, self.opening, self.nf, self.y, P.get("L_in"), self.U[0])
        L.lp_mgrit_forward(p, self.mgF, P["K"], P["b"], self.U, self.ws, history=False, dsig=self.rec)
        L.lp_loss_terminal(p, self.nc, self.U[-1], P["W"], P["mu"], self.c, self.J, self.Lam[-1], G["W"], G["mu"],
                           self.ws)
        L.lp_mgrit_adjoint(p, self.mgA, P["K"], P["b"], self.U, self.Lam, self.ws, history=False, dsig=self.rec)
        L.lp_gradient(p, P["K"], P["b"], self.U, self.Lam, G["K"], G["b"], self.ws, dsig=self.rec)
        if "L_in" in P:
            L.lp_open_grad(p, self.opening, self.nf, self.y, P["L_in"], self.Lam[0], G["L_in"])
        for k in P:
            L.lp_sgd_update(P[k], G[k], lr)
        self.updates += 1

    def run(self, updates: int, lr: float, losses: Optional[List[float]] = None) -> List[float]:
        out = [] if losses is None else losses
        for _ in range(updates):
            self.step(lr)
            out.append(float(self.J.item()))
        return out
