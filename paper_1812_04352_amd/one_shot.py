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
            # the solves read nothing back: a diverging iterate shows up here
            L.lp_check_finite()
            out.append(float(self.J.item()))
        return out


class SerialTrainer:
    """Layer-serial gradient descent on the same objective, the baseline method
    the one-shot run is compared with (Section 5.3): per update the exact
    forward propagation and backpropagation (the state and adjoint equations of
    Section 2.3 solved by forward and backward substitution), the exact reduced
    gradient, and the same plain gradient step as OneShotTrainer. Same
    arguments as OneShotTrainer without the MGRIT schedules."""

    def __init__(self, prob: L.LpProblem, params: Dict[str, torch.Tensor], y: torch.Tensor, c: torch.Tensor,
                 n_classes: int, opening: int, n_features: int):
        self.p, self.P = prob, params
        self.y, self.c = y, c
        self.nc, self.opening, self.nf = n_classes, opening, n_features
        dt = params["K"].dtype
        shape = (prob.N + 1, prob.B) + ((prob.C, prob.H, prob.W) if prob.layer == L.LP_CONV3X3 else (prob.q,))
        self.U = torch.zeros(shape, device="cuda", dtype=dt)
        self.Lam = torch.zeros_like(self.U)
        self.ws = L.alloc_workspace(prob)
        self.J = torch.zeros(1, device="cuda", dtype=torch.float64)
        self.G = {k: torch.empty_like(v) for k, v in params.items()}
        self.rec = L.alloc_dsig(prob) if L.lp_dsig_bytes(prob) else None

    def step(self, lr: float) -> None:
        P, G, p = self.P, self.G, self.p
        L.lp_open_forward(p, self.opening, self.nf, self.y, P.get("L_in"), self.U[0])
        L.lp_serial_forward(p, P["K"], P["b"], self.U, dsig=self.rec)
        L.lp_loss_terminal(p, self.nc, self.U[-1], P["W"], P["mu"], self.c, self.J, self.Lam[-1], G["W"], G["mu"],
                           self.ws)
        L.lp_serial_adjoint(p, P["K"], P["b"], self.U, self.Lam, dsig=self.rec)
        L.lp_gradient(p, P["K"], P["b"], self.U, self.Lam, G["K"], G["b"], self.ws, dsig=self.rec)
        if "L_in" in P:
            L.lp_open_grad(p, self.opening, self.nf, self.y, P["L_in"], self.Lam[0], G["L_in"])
        for k in P:
            L.lp_sgd_update(P[k], G[k], lr)

    def run(self, updates: int, lr: float, losses: Optional[List[float]] = None) -> List[float]:
        out = [] if losses is None else losses
        for _ in range(updates):
            self.step(lr)
            out.append(float(self.J.item()))
        return out


class LbfgsOneShotTrainer:
    """Algorithm 2 (Section 4) with its Hessian approximated by limited-memory BFGS,
    a backtracking line search and a validation-accuracy stop, as a host loop over
    the C ABI. Per design update: m1 state and m2 adjoint MGRIT iterations
    (warm-started from the previous update; mg_fwd / mg_adj carry m1 / m2 as
    max_iter), the reduced gradient at those iterates, the curvature pair
    (s, y) = (design change, gradient change) kept when s.y > 0 (at most `memory`
    pairs), the direction d = -H g by the two-loop recursion (initial matrix
    gamma I, gamma = s.y / y.y of the newest pair), and trial designs
    theta + alpha d, alpha = alpha_start * shrink^t (alpha_start = alpha0 at the
    first update, 1 afterwards), each judged by the loss of the state after m1
    MGRIT iterations warm-started from the current state: the first with
    J_t <= J + c1 alpha g.d is taken (the last trial if none is). line_search =
    "wolfe" searches instead for a step meeting the strong Wolfe conditions
    (_wolfe_search; the slope at a trial is the reduced gradient after m2 adjoint
    iterations at the trial state, dotted with d). With validation
    data the accuracy of the new design (exact forward propagation) is taken after
    every update and the run stops once it reaches target_acc.

    Vector algebra runs in the library (lp_vec_dot, lp_vec_axpby); only scalars
    (dot products, losses, accuracies) come back to the host, where the two-loop
    coefficients and the line-search test are evaluated."""

    def __init__(self, prob: L.LpProblem, mg_fwd: L.LpMgrit, mg_adj: L.LpMgrit, params: Dict[str, torch.Tensor],
                 y: torch.Tensor, c: torch.Tensor, n_classes: int, opening: int, n_features: int,
                 memory: int = 5, alpha0: float = 1e-2, c1: float = 1e-4, shrink: float = 0.5, max_ls: int = 8,
                 y_val: Optional[torch.Tensor] = None, c_val: Optional[torch.Tensor] = None,
                 target_acc: Optional[float] = None, line_search: str = "armijo", c2: float = 0.9):
        if line_search not in ("armijo", "wolfe"):
            raise ValueError(f"line_search must be 'armijo' or 'wolfe', not {line_search!r}")
        self.line_search, self.c2 = line_search, c2
        self.p, self.mgF, self.mgA = prob, mg_fwd, mg_adj
        self.P = params
        self.names = (["L_in"] if "L_in" in params else []) + ["K", "b", "W", "mu"]
        self.y, self.c = y, c
        self.nc, self.opening, self.nf = n_classes, opening, n_features
        self.memory, self.alpha0, self.c1, self.shrink, self.max_ls = memory, alpha0, c1, shrink, max_ls
        dt = params["K"].dtype
        shape = (prob.N + 1, prob.B) + ((prob.C, prob.H, prob.W) if prob.layer == L.LP_CONV3X3 else (prob.q,))
        self.U = torch.zeros(shape, device="cuda", dtype=dt)
        self.Ut = torch.zeros_like(self.U)
        self.Lam = torch.zeros_like(self.U)
        need = max(L.lp_workspace_bytes(prob, mg_fwd), L.lp_workspace_bytes(prob, mg_adj))
        self.ws = torch.empty(need, dtype=torch.uint8, device="cuda")
        self.J = torch.zeros(1, device="cuda", dtype=torch.float64)
        self.lam_scratch = torch.empty_like(self.U[-1])

        def like():
            return {k: torch.empty_like(params[k]) for k in self.names}

        self.G, self.T, self.D, self.Q = like(), like(), like(), like()
        # the strong Wolfe search's trial gradient and trial adjoint
        self.GT = like() if line_search == "wolfe" else None
        self.LamT = torch.zeros_like(self.U) if line_search == "wolfe" else None
        self.wolfe: List[bool] = []
        self.gW, self.gmu = torch.empty_like(params["W"]), torch.empty_like(params["mu"])
        self.prev = None  # (design copy, gradient copy) of the previous update
        self.pairs: List[tuple] = []
        self.dots = torch.zeros((len(self.names), 1 + L.LP_DOT_PARTIALS), device="cuda", dtype=torch.float64)
        self.rec = L.alloc_dsig(prob) if L.lp_dsig_bytes(prob) else None
        self.val = None
        if y_val is not None:
            pv = L.LpProblem.from_buffer_copy(prob)
            pv.B = y_val.shape[0]
            Uv = torch.zeros((prob.N + 1, y_val.shape[0]) + shape[2:], device="cuda", dtype=dt)
            self.val = (pv, Uv, y_val, c_val, L.alloc_workspace(pv),
                        torch.zeros(1, device="cuda", dtype=torch.float64))
        self.target_acc = target_acc
        self.updates = 0
        self.losses: List[float] = []
        self.alphas: List[float] = []
        self.trials: List[int] = []
        self.accuracies: List[float] = []

    # ---- vectors over the design (dicts of tensors in self.names order)
    def _dot(self, a, b) -> float:
        for i, k in enumerate(self.names):
            L.lp_vec_dot(a[k], b[k], self.dots[i])
        return float(sum(float(v) for v in self.dots[:, 0].cpu().tolist()))

    def _axpby(self, y, x, a: float, b: float) -> None:
        for k in self.names:
            L.lp_vec_axpby(y[k], x[k], a, b)

    def _copy(self, x):
        out = {k: torch.empty_like(x[k]) for k in self.names}
        self._axpby(out, x, 1.0, 0.0)
        return out

    def _state_after(self, design, U, warm: bool, dsig=None) -> None:
        """U <- the state after m1 MGRIT iterations at `design`, starting from U."""
        L.lp_open_forward(self.p, self.opening, self.nf, self.y, design.get("L_in"), U[0])
        self.mgF.warm_start = int(warm)
        L.lp_mgrit_forward(self.p, self.mgF, design["K"], design["b"], U, self.ws, history=False, dsig=dsig)

    def _loss(self, design, U, lamN, dW, dmu) -> float:
        L.lp_loss_terminal(self.p, self.nc, U[-1], design["W"], design["mu"], self.c, self.J, lamN, dW, dmu, self.ws)
        return float(self.J.item())

    def _trial(self, alpha: float) -> float:
        """T <- P + alpha D, Ut <- the state after m1 MGRIT iterations at T from U;
        returns the trial loss (inf if the state solve diverged). Leaves the
        trial's terminal adjoint and head gradients in lam_scratch, gW, gmu."""
        self._axpby(self.T, self.P, 1.0, 0.0)
        self._axpby(self.T, self.D, alpha, 1.0)
        L.lp_vec_axpby(self.Ut, self.U, 1.0, 0.0)
        self._state_after(self.T, self.Ut, True)
        Jt = self._loss(self.T, self.Ut, self.lam_scratch, self.gW, self.gmu)
        try:
            L.lp_check_finite()
        except L.LpError as err:  # the trial design's state solve diverged: reject it
            if err.status != L.LP_ENONFINITE:
                raise
            Jt = float("inf")
        return Jt

    def _trial_slope(self) -> float:
        """phi'(alpha) = g_T . D for the trial just taken: the reduced gradient at the
        trial state after m2 adjoint MGRIT iterations warm-started from this update's
        adjoint iterate."""
        T, GT = self.T, self.GT
        L.lp_vec_axpby(self.LamT, self.Lam, 1.0, 0.0)
        L.lp_vec_axpby(self.LamT[-1], self.lam_scratch, 1.0, 0.0)
        self.mgA.warm_start = 1
        L.lp_mgrit_adjoint(self.p, self.mgA, T["K"], T["b"], self.Ut, self.LamT, self.ws, history=False)
        L.lp_gradient(self.p, T["K"], T["b"], self.Ut, self.LamT, GT["K"], GT["b"], self.ws)
        if "L_in" in T:
            L.lp_open_grad(self.p, self.opening, self.nf, self.y, T["L_in"], self.LamT[0], GT["L_in"])
        L.lp_vec_axpby(GT["W"], self.gW, 1.0, 0.0)
        L.lp_vec_axpby(GT["mu"], self.gmu, 1.0, 0.0)
        return self._dot(GT, self.D)

    def _wolfe_search(self, J: float, gd: float, alpha0: float):
        """Step length meeting the strong Wolfe conditions, phi(a) <= J + c1 a gd and
        |phi'(a)| <= c2 |gd| (Section 4): bracketing with step doubling, then zoom by
        bisection (Nocedal and Wright, Numerical Optimization, Algorithms 3.5, 3.6),
        at most max_ls trial losses. Returns (alpha, trials - 1, last trial's alpha);
        records in self.wolfe whether alpha meets both conditions. Without such a
        step: the lower end of the last bracket (the best step with sufficient
        decrease), else the last trial."""
        c1, c2, cap = self.c1, self.c2, self.max_ls
        n, last = 0, alpha0

        def ok_decrease(a, Ja):
            return Ja <= J + c1 * a * gd

        def curvature(slope):
            return abs(slope) <= c2 * abs(gd)

        def zoom(lo, J_lo, hi):
            nonlocal n, last
            while n < cap:
                a = 0.5 * (lo + hi)
                Ja = self._trial(a)
                n, last = n + 1, a
                if not ok_decrease(a, Ja) or Ja >= J_lo:
                    hi = a
                    continue
                slope = self._trial_slope()
                if curvature(slope):
                    return a, True
                if slope * (hi - lo) >= 0.0:
                    hi = lo
                lo, J_lo = a, Ja
            return lo, False

        a_prev, J_prev, a = 0.0, J, alpha0
        while True:
            Ja = self._trial(a)
            n, last = n + 1, a
            if not ok_decrease(a, Ja) or (a_prev > 0.0 and Ja >= J_prev):
                res, met = zoom(a_prev, J_prev, a)
                break
            slope = self._trial_slope()
            if curvature(slope):
                res, met = a, True
                break
            if slope >= 0.0:
                res, met = zoom(a, Ja, a_prev)
                break
            if n >= cap:
                res, met = a, False
                break
            a_prev, J_prev, a = a, Ja, 2.0 * a
        if res == 0.0:
            res = last
        self.wolfe.append(met)
        return res, n - 1, last

    def step(self) -> bool:
        """One design update; returns False once the validation target is reached."""
        P, G = self.P, self.G
        first = self.updates == 0
        self._state_after(P, self.U, not first, self.rec)
        J = self._loss(P, self.U, self.Lam[-1], G["W"], G["mu"])
        self.mgA.warm_start = int(not first)
        L.lp_mgrit_adjoint(self.p, self.mgA, P["K"], P["b"], self.U, self.Lam, self.ws, history=False, dsig=self.rec)
        L.lp_gradient(self.p, P["K"], P["b"], self.U, self.Lam, G["K"], G["b"], self.ws, dsig=self.rec)
        if "L_in" in P:
            L.lp_open_grad(self.p, self.opening, self.nf, self.y, P["L_in"], self.Lam[0], G["L_in"])
        # the state and adjoint solves read nothing back: a diverging iterate shows up here
        L.lp_check_finite()
        # curvature pair from the previous update
        if self.prev is not None:
            xp, gp = self.prev
            s, yv = self._copy(P), self._copy(G)
            self._axpby(s, xp, -1.0, 1.0)
            self._axpby(yv, gp, -1.0, 1.0)
            sy = self._dot(s, yv)
            if sy > 0.0:
                self.pairs.append((s, yv, sy))
                self.pairs = self.pairs[-self.memory:]
        # two-loop recursion: Q <- H g, then D <- -Q
        self._axpby(self.Q, G, 1.0, 0.0)
        coef = []
        for s, yv, sy in reversed(self.pairs):
            a = self._dot(s, self.Q) / sy
            coef.append(a)
            self._axpby(self.Q, yv, -a, 1.0)
        gamma = self.pairs[-1][2] / self._dot(self.pairs[-1][1], self.pairs[-1][1]) if self.pairs else 1.0
        self._axpby(self.Q, self.Q, gamma, 0.0)
        for (s, yv, sy), a in zip(self.pairs, reversed(coef)):
            beta = self._dot(yv, self.Q) / sy
            self._axpby(self.Q, s, a - beta, 1.0)
        self._axpby(self.D, self.Q, -1.0, 0.0)
        gd = self._dot(G, self.D)
        alpha = self.alpha0 if first else 1.0
        if self.line_search == "wolfe":
            alpha, t, last = self._wolfe_search(J, gd, alpha)
            if alpha != last:  # T and Ut hold the last trial: take the accepted one again
                self._trial(alpha)
        else:
            # backtracking line search on the objective at trial designs
            for t in range(self.max_ls):
                Jt = self._trial(alpha)
                if Jt <= J + self.c1 * alpha * gd or t == self.max_ls - 1:
                    break
                alpha *= self.shrink
        self.prev = (self._copy(P), self._copy(G))
        self._axpby(P, self.T, 1.0, 0.0)
        self.U, self.Ut = self.Ut, self.U
        self.losses.append(J)
        self.alphas.append(alpha)
        self.trials.append(t + 1)
        self.updates += 1
        if self.val is not None:
            pv, Uv, yv_, cv, wsv, acc = self.val
            L.lp_open_forward(pv, self.opening, self.nf, yv_, P.get("L_in"), Uv[0])
            L.lp_serial_forward(pv, P["K"], P["b"], Uv)
            L.lp_accuracy(pv, self.nc, Uv[-1], P["W"], P["mu"], cv, acc, wsv)
            a = float(acc.item())
            self.accuracies.append(a)
            if self.target_acc is not None and a >= self.target_acc:
                return False
        return True

    def run(self, updates: int) -> List[float]:
        for _ in range(updates):
            if not self.step():
                break
        return self.losses
