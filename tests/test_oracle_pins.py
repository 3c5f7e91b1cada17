"""Pins of the CPU oracle against what the paper and mathematics fix (no GPU).

Each test checks the oracle against a source other than itself: closed forms,
torch autograd on the same network, central finite differences, Parareal written
from its textbook definition, and the finite-step exactness and fixed-point
properties of MGRIT (Section 3.1).
"""
import os

import numpy as np
import pytest
import torch

import oracle as O
from workloads import WORKLOADS, generate, random_state

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def rel(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return float(np.linalg.norm((a - b).ravel()) / max(np.linalg.norm(b.ravel()), 1e-300))


def tiny_dense(seed=0, B=7, q=5, N=12, nf=3, nc=4, act="tanh", kscale=0.3):
    r = np.random.default_rng(seed)
    return dict(y=r.standard_normal((B, nf)), L_in=0.5 * r.standard_normal((q, nf)),
                K=kscale * r.standard_normal((N, q, q)), b=0.1 * r.standard_normal((N, q)),
                W=0.5 * r.standard_normal((nc, q)), mu=0.1 * r.standard_normal(nc),
                onehot=np.eye(nc)[r.integers(0, nc, B)], h=0.7 / N * 4, act=act)


def tiny_conv(seed=0, B=2, C=3, H=5, W=6, N=4, nc=3, act="tanh"):
    r = np.random.default_rng(seed)
    return dict(y=r.standard_normal((B, 1, H, W)), L_in=0.4 * r.standard_normal((C, 1, 3, 3)),
                K=0.3 * r.standard_normal((N, C, C, 3, 3)), b=0.1 * r.standard_normal((N, C)),
                W=0.3 * r.standard_normal((nc, C * H * W)), mu=0.1 * r.standard_normal(nc),
                onehot=np.eye(nc)[r.integers(0, nc, B)], h=0.25, act=act)


def full_objective(p, opening):
    u0 = O.open_forward(p["y"], p["L_in"], p["act"], opening)
    U = O.serial_forward(u0, p["K"], p["b"], p["h"], p["act"])
    J, lamN, dW, dmu = O.loss_terminal(U[-1], p["W"], p["mu"], p["onehot"])
    return J, U, lamN, dW, dmu


def full_gradient(p, opening):
    J, U, lamN, dW, dmu = full_objective(p, opening)
    Lam = O.serial_adjoint(U, lamN, p["K"], p["b"], p["h"], p["act"])
    dK, db = O.gradient(U, Lam, p["K"], p["b"], p["h"], p["act"])
    dL = O.open_grad(p["y"], p["L_in"], Lam[0], p["act"], opening)
    return dict(K=dK, b=db, W=dW, mu=dmu, L_in=dL), U, Lam


# ---------------------------------------------------------------- activations

def test_smoothrelu_golden_values():
    tab = np.loadtxt(os.path.join(GOLDEN, "smoothrelu.txt"))
    x, s, ds = tab[:, 0], tab[:, 1], tab[:, 2]
    assert np.allclose(O.act(x, "smoothrelu"), s, rtol=0, atol=1e-15)
    assert np.allclose(O.dact(x, "smoothrelu"), ds, rtol=0, atol=1e-15)


def test_smoothrelu_is_c1():
    # value and slope agree from both sides of the branch points +-0.1
    for x0 in (-0.1, 0.1):
        for e in (1e-7, 1e-9):
            lo, hi = O.act(np.array([x0 - e, x0 + e]), "smoothrelu")
            assert abs(hi - lo) < 3 * e
            dlo, dhi = O.dact(np.array([x0 - e, x0 + e]), "smoothrelu")
            assert abs(dhi - dlo) < 1e-5


@pytest.mark.parametrize("kind", ["tanh", "relu", "smoothrelu", "identity"])
def test_dact_matches_autograd(kind):
    z = np.linspace(-2.0, 2.0, 401) + 1e-3  # stay off the ReLU kink at 0
    t = torch.tensor(z, dtype=torch.float64, requires_grad=True)
    if kind == "tanh":
        y = torch.tanh(t)
    elif kind == "relu":
        y = torch.relu(t)
    elif kind == "identity":
        y = t * 1.0
    else:
        y = torch.where(t.abs() <= 0.1, 2.5 * t * t + 0.5 * t + 0.025, torch.relu(t))
    y.sum().backward()
    assert np.allclose(O.act(z, kind), y.detach().numpy(), rtol=0, atol=1e-15)
    assert np.allclose(O.dact(z, kind), t.grad.numpy(), rtol=0, atol=1e-14)


def test_relu_derivative_at_zero_is_zero():
    assert O.dact(np.array([0.0]), "relu")[0] == 0.0


# ---------------------------------------------------------------- convolution

def test_conv_matches_torch_conv2d():
    r = np.random.default_rng(3)
    v = r.standard_normal((3, 4, 7, 9))
    Kn = r.standard_normal((5, 4, 3, 3))
    ref = torch.nn.functional.conv2d(torch.tensor(v), torch.tensor(Kn), padding=1).numpy()
    assert rel(O.conv3x3(Kn, v), ref) < 1e-14


def test_conv_transpose_and_weight_grad_match_autograd():
    r = np.random.default_rng(4)
    v = r.standard_normal((3, 4, 7, 9))
    Kn = r.standard_normal((4, 4, 3, 3))
    s = r.standard_normal((3, 4, 7, 9))
    tv = torch.tensor(v, requires_grad=True)
    tk = torch.tensor(Kn, requires_grad=True)
    (torch.nn.functional.conv2d(tv, tk, padding=1) * torch.tensor(s)).sum().backward()
    assert rel(O.conv3x3_transpose(Kn, s), tv.grad.numpy()) < 1e-14
    assert rel(O.conv3x3_weight_grad(s, v), tk.grad.numpy()) < 1e-14


# ---------------------------------------------------------------- serial closed forms

@pytest.mark.parametrize("kind", ["tanh", "relu", "smoothrelu"])
def test_serial_forward_zero_weights_closed_form(kind):
    # K = 0: u^{n} = u^0 + n h sigma(b) when b is the same in every layer
    r = np.random.default_rng(1)
    N, B, q, h = 9, 4, 6, 0.3
    u0 = r.standard_normal((B, q))
    b1 = 0.5 * r.standard_normal(q)
    U = O.serial_forward(u0, np.zeros((N, q, q)), np.tile(b1, (N, 1)), h, kind)
    sig = {"tanh": np.tanh(b1), "relu": np.maximum(b1, 0),
           "smoothrelu": np.where(np.abs(b1) <= 0.1, 2.5 * b1 ** 2 + 0.5 * b1 + 0.025, np.maximum(b1, 0))}[kind]
    for n in range(N + 1):
        assert rel(U[n], u0 + n * h * sig[None, :]) < 1e-14


def test_serial_forward_linear_closed_form():
    # identity activation, constant K, b = 0: u^N = (I + h K)^N u^0
    r = np.random.default_rng(2)
    N, B, q, h = 17, 5, 6, 0.1
    u0 = r.standard_normal((B, q))
    K1 = r.standard_normal((q, q))
    U = O.serial_forward(u0, np.tile(K1, (N, 1, 1)), np.zeros((N, q)), h, "identity")
    M = np.linalg.matrix_power(np.eye(q) + h * K1, N)
    assert rel(U[N], u0 @ M.T) < 1e-13


def test_serial_adjoint_linear_closed_form():
    r = np.random.default_rng(5)
    N, B, q, h = 11, 3, 4, 0.2
    u0 = r.standard_normal((B, q))
    K1 = r.standard_normal((q, q))
    K = np.tile(K1, (N, 1, 1))
    U = O.serial_forward(u0, K, np.zeros((N, q)), h, "identity")
    lamN = r.standard_normal((B, q))
    Lam = O.serial_adjoint(U, lamN, K, np.zeros((N, q)), h, "identity")
    M = np.linalg.matrix_power(np.eye(q) + h * K1, N)
    assert rel(Lam[0], lamN @ M) < 1e-13


# ---------------------------------------------------------------- autograd / backprop

@pytest.mark.parametrize("kind", ["tanh", "relu", "smoothrelu"])
def test_adjoint_and_gradient_match_torch_autograd_dense(kind):
    p = tiny_dense(seed=7, act=kind)
    g, U, Lam = full_gradient(p, "dense_act")
    t = {k: torch.tensor(p[k], requires_grad=True) for k in ("L_in", "K", "b", "W", "mu")}

    def sig(z):
        if kind == "tanh":
            return torch.tanh(z)
        if kind == "relu":
            return torch.relu(z)
        return torch.where(z.abs() <= 0.1, 2.5 * z * z + 0.5 * z + 0.025, torch.relu(z))

    u = sig(torch.tensor(p["y"]) @ t["L_in"].T)
    us = [u]
    for n in range(p["K"].shape[0]):
        u = u + p["h"] * sig(u @ t["K"][n].T + t["b"][n])
        u.retain_grad()
        us.append(u)
    us[0].retain_grad()
    z = u @ t["W"].T + t["mu"]
    J = -(torch.tensor(p["onehot"]) * torch.log_softmax(z, dim=1)).sum() / z.shape[0]
    J.backward()
    for k in g:
        assert rel(g[k], t[k].grad.numpy()) < 1e-12, k
    for n in range(len(us)):
        assert rel(Lam[n], us[n].grad.numpy()) < 1e-12, n


def test_adjoint_and_gradient_match_torch_autograd_conv():
    p = tiny_conv(seed=8, act="tanh")
    g, U, Lam = full_gradient(p, "conv_act")
    t = {k: torch.tensor(p[k], requires_grad=True) for k in ("L_in", "K", "b", "W", "mu")}
    u = torch.tanh(torch.nn.functional.conv2d(torch.tensor(p["y"]), t["L_in"], padding=1))
    for n in range(p["K"].shape[0]):
        u = u + p["h"] * torch.tanh(torch.nn.functional.conv2d(u, t["K"][n], t["b"][n], padding=1))
    z = u.reshape(u.shape[0], -1) @ t["W"].T + t["mu"]
    J = -(torch.tensor(p["onehot"]) * torch.log_softmax(z, dim=1)).sum() / z.shape[0]
    J.backward()
    for k in g:
        assert rel(g[k], t[k].grad.numpy()) < 1e-12, k


# ---------------------------------------------------------------- finite differences

def test_gradient_central_finite_differences_dense():
    # config-1-sized tanh net (width 8, 32 layers, 2 input features, 5 classes)
    wl = WORKLOADS[1].with_overrides(B=16)
    d = generate(wl)
    p = dict(y=d["y"].astype(np.float64), L_in=d["L_in"].astype(np.float64),
             K=d["K"].astype(np.float64), b=0.05 * np.random.default_rng(9).standard_normal((wl.N, wl.q)),
             W=d["W"].astype(np.float64), mu=0.1 * np.ones(wl.n_classes),
             onehot=d["onehot"], h=wl.h, act="tanh")
    g, _, _ = full_gradient(p, "dense_act")
    eps = 1e-6
    r = np.random.default_rng(10)

    def J_at(pp):
        return full_objective(pp, "dense_act")[0]

    # random directional derivative over all parameters at once
    dirs = {k: r.standard_normal(p[k].shape) for k in g}
    pp = {**p, **{k: p[k] + eps * dirs[k] for k in g}}
    pm = {**p, **{k: p[k] - eps * dirs[k] for k in g}}
    fd = (J_at(pp) - J_at(pm)) / (2 * eps)
    an = sum(float(np.sum(g[k] * dirs[k])) for k in g)
    assert abs(fd - an) <= 1e-7 * abs(an)
    # single entries of every parameter block
    for k, idx in (("K", (3, 2, 5)), ("K", (31, 7, 0)), ("b", (0, 4)), ("b", (20, 1)),
                   ("W", (2, 6)), ("mu", (4,)), ("L_in", (5, 1))):
        e = np.zeros_like(p[k])
        e[idx] = eps
        fd = (J_at({**p, k: p[k] + e}) - J_at({**p, k: p[k] - e})) / (2 * eps)
        assert abs(fd - g[k][idx]) <= 1e-7 * max(abs(g[k][idx]), 1e-3), (k, idx, fd, g[k][idx])


def test_gradient_central_finite_differences_conv():
    p = tiny_conv(seed=11, act="tanh")
    g, _, _ = full_gradient(p, "conv_act")
    eps = 1e-6
    r = np.random.default_rng(12)
    dirs = {k: r.standard_normal(p[k].shape) for k in g}
    Jp = full_objective({**p, **{k: p[k] + eps * dirs[k] for k in g}}, "conv_act")[0]
    Jm = full_objective({**p, **{k: p[k] - eps * dirs[k] for k in g}}, "conv_act")[0]
    an = sum(float(np.sum(g[k] * dirs[k])) for k in g)
    assert abs((Jp - Jm) / (2 * eps) - an) <= 1e-7 * abs(an)


# ---------------------------------------------------------------- residual norms

def test_residual_norm_of_serial_solution_is_zero():
    p = tiny_dense(seed=13)
    U = O.serial_forward(np.random.default_rng(0).standard_normal((7, 5)), p["K"], p["b"], p["h"], "tanh")
    assert O.residual_norm_state(U, p["K"], p["b"], p["h"], "tanh") == 0.0
    Lam = O.serial_adjoint(U, np.ones((7, 5)), p["K"], p["b"], p["h"], "tanh")
    assert O.residual_norm_adjoint(U, Lam, p["K"], p["b"], p["h"], "tanh") == 0.0


def test_residual_norm_single_perturbation_closed_form():
    # K = 0: a perturbation delta at one interior point gives rho = sqrt(2) ||delta||
    r = np.random.default_rng(14)
    N, B, q, h = 10, 3, 4, 0.3
    K = np.zeros((N, q, q))
    b = np.tile(r.standard_normal(q), (N, 1))
    U = O.serial_forward(r.standard_normal((B, q)), K, b, h, "tanh")
    delta = r.standard_normal((B, q))
    U2 = U.copy()
    U2[4] += delta
    rho = O.residual_norm_state(U2, K, b, h, "tanh")
    assert abs(rho - np.sqrt(2) * np.linalg.norm(delta)) < 1e-13 * rho
    U3 = U.copy()
    U3[N] += delta  # last point enters one residual row only
    assert abs(O.residual_norm_state(U3, K, b, h, "tanh") - np.linalg.norm(delta)) < 1e-12


# ---------------------------------------------------------------- MGRIT

def _mgrit_case(seed=20, N=32, B=6, q=5, act="tanh", kscale=0.4):
    r = np.random.default_rng(seed)
    K = kscale * r.standard_normal((N, q, q))
    b = 0.2 * r.standard_normal((N, q))
    u0 = r.standard_normal((B, q))
    return K, b, u0, 5.0 / N


@pytest.mark.parametrize("c", [2, 4, 8])
@pytest.mark.parametrize("relax,gain", [("F", 1), ("FCF", 2), ("FCFCF", 3)])
def test_two_level_finite_step_exactness_forward(relax, gain, c):
    # two-level F: after m iterations points n <= (m+1)c-1 are exact; FCF: n <= (2m+1)c-1;
    # FCFCF: n <= (3m+1)c-1 (each C-relaxation moves the exact front by one interval,
    # the coarse-grid correction by one more)
    K, b, u0, h = _mgrit_case()
    N = K.shape[0]
    S = O.serial_forward(u0, K, b, h, "tanh")
    U = np.zeros_like(S)
    U[0] = u0
    full = -(-N // (gain * c))
    for m in range(1, full + 1):
        Um, _, _ = O.mgrit_forward(U, K, b, h, "tanh", cf=c, max_levels=2, relax=relax, max_iter=m)
        exact = min((gain * m + 1) * c - 1, N)
        err = np.abs(Um - S).reshape(N + 1, -1).max(axis=1)
        assert err[:exact + 1].max() < 1e-14, (m, exact)
        if exact < N and (c >= 4 or m == 1):
            # not exact beyond the front (at c = 2 later iterations may converge
            # there to rounding before the front arrives)
            assert err[exact + 1:].max() > 1e-8
    assert np.abs(Um - S).max() < 1e-14


@pytest.mark.parametrize("c", [2, 4, 8])
@pytest.mark.parametrize("relax,gain", [("F", 1), ("FCF", 2), ("FCFCF", 3)])
def test_two_level_finite_step_exactness_adjoint(relax, gain, c):
    K, b, u0, h = _mgrit_case(seed=21)
    N = K.shape[0]
    U = O.serial_forward(u0, K, b, h, "tanh")
    lamN = np.random.default_rng(0).standard_normal(u0.shape)
    S = O.serial_adjoint(U, lamN, K, b, h, "tanh")
    L = np.zeros_like(S)
    L[N] = lamN
    full = -(-N // (gain * c))
    for m in range(1, full + 1):
        Lm, _, _ = O.mgrit_adjoint(U, L, K, b, h, "tanh", cf=c, max_levels=2, relax=relax, max_iter=m)
        exact = min((gain * m + 1) * c - 1, N)
        err = np.abs(Lm - S).reshape(N + 1, -1).max(axis=1)[::-1]  # distance from the end
        assert err[:exact + 1].max() < 1e-14, (m, exact)
        if exact < N and (c >= 4 or m == 1):
            assert err[exact + 1:].max() > 1e-8
    assert np.abs(Lm - S).max() < 1e-14


def _parareal(u0, K, b, h, c, iters, kind):
    """Parareal (Gander & Vandewalle 2007), the equivalent of two-level MGRIT with
    F-relaxation: fine propagator F_k = c fine steps from T_k, coarse propagator
    G_k = one step of size c h with the weights of layer k c. Iteration:
        U_{k+1}^{new} = G_k(U_k^{new}) + F_k(U_k^{old}) - G_k(U_k^{old}),
    then the fine points are filled by fine propagation from the new C-points."""
    N = K.shape[0]
    Nc = N // c

    def fine(k, v):
        for j in range(c):
            n = k * c + j
            v = v + h * O.act(v @ K[n].T + b[n], kind)
        return v

    def coarse(k, v):
        n = k * c
        return v + c * h * O.act(v @ K[n].T + b[n], kind)

    Uc = [u0] * (Nc + 1)  # cold start: every C-point is u0
    for _ in range(iters):
        Fold = [fine(k, Uc[k]) for k in range(Nc)]
        new = [u0]
        for k in range(Nc):
            new.append(coarse(k, new[k]) + Fold[k] - coarse(k, Uc[k]))
        Uc = new
    out = np.zeros((N + 1,) + u0.shape)
    for k in range(Nc):
        v = Uc[k]
        out[k * c] = v
        for j in range(1, c):
            n = k * c + j - 1
            v = v + h * O.act(v @ K[n].T + b[n], kind)
            out[k * c + j] = v
    out[N] = Uc[Nc]
    return out


@pytest.mark.parametrize("iters", [1, 2, 3])
def test_two_level_F_equals_parareal(iters):
    K, b, u0, h = _mgrit_case(seed=22, kscale=0.6)
    U = np.zeros((K.shape[0] + 1,) + u0.shape)
    U[0] = u0
    Um, _, _ = O.mgrit_forward(U, K, b, h, "tanh", cf=4, max_levels=2, relax="F", max_iter=iters)
    P = _parareal(u0, K, b, h, 4, iters, "tanh")
    assert rel(Um, P) < 1e-13


@pytest.mark.parametrize("levels,relax", [(2, "F"), (3, "FCF"), (4, "FCF"), (3, "F")])
def test_coarse_propagator_exact_when_layers_are_constant_increments(levels, relax):
    # K = 0 and the same bias in every layer: c fine steps of size h equal one coarse step
    # of size c h on every level, so one V-cycle solves the problem exactly.
    r = np.random.default_rng(23)
    N, B, q, h = 64, 3, 4, 0.05
    K = np.zeros((N, q, q))
    b = np.tile(r.standard_normal(q), (N, 1))
    u0 = r.standard_normal((B, q))
    S = O.serial_forward(u0, K, b, h, "tanh")
    U = np.zeros_like(S)
    U[0] = u0
    Um, hist, _ = O.mgrit_forward(U, K, b, h, "tanh", cf=4, max_levels=levels, relax=relax, max_iter=1)
    assert rel(Um, S) < 1e-14
    lamN = r.standard_normal((B, q))
    Ls = O.serial_adjoint(S, lamN, K, b, h, "tanh")
    L0 = np.zeros_like(S)
    L0[N] = lamN
    Lm, _, _ = O.mgrit_adjoint(S, L0, K, b, h, "tanh", cf=4, max_levels=levels, relax=relax, max_iter=1)
    assert rel(Lm, Ls) < 1e-14


@pytest.mark.parametrize("levels", [2, 3, 4])
@pytest.mark.parametrize("kind", ["tanh", "relu"])
def test_fixed_point_is_serial_solution(levels, kind):
    K, b, u0, h = _mgrit_case(seed=24, N=64, act=kind)
    S = O.serial_forward(u0, K, b, h, kind)
    Um, hist, _ = O.mgrit_forward(S, K, b, h, kind, cf=4, max_levels=levels, relax="FCF",
                                  max_iter=1, warm_start=True)
    assert np.abs(Um - S).max() <= 1e-14 * np.abs(S).max()
    assert hist[0] <= 1e-14 * np.linalg.norm(S)
    lamN = np.random.default_rng(1).standard_normal(u0.shape)
    Ls = O.serial_adjoint(S, lamN, K, b, h, kind)
    Lm, hist, _ = O.mgrit_adjoint(S, Ls, K, b, h, kind, cf=4, max_levels=levels, relax="FCF",
                                  max_iter=1, warm_start=True)
    assert np.abs(Lm - Ls).max() <= 1e-14 * np.abs(Ls).max()


@pytest.mark.parametrize("levels,kind", [(3, "tanh"), (4, "relu"), (5, "smoothrelu")])
def test_multilevel_converges_to_serial(levels, kind):
    K, b, u0, h = _mgrit_case(seed=25, N=256, act=kind, kscale=0.3)
    S = O.serial_forward(u0, K, b, h, kind)
    U = np.zeros_like(S)
    U[0] = u0
    Um, hist, it = O.mgrit_forward(U, K, b, h, kind, cf=4, max_levels=levels, relax="FCF",
                                   max_iter=30, rtol=1e-13)
    assert rel(Um, S) < 1e-11, (it, hist)
    lamN = np.random.default_rng(2).standard_normal(u0.shape)
    Ls = O.serial_adjoint(S, lamN, K, b, h, kind)
    L0 = np.zeros_like(S)
    L0[-1] = lamN
    Lm, hist, it = O.mgrit_adjoint(S, L0, K, b, h, kind, cf=4, max_levels=levels, relax="FCF",
                                   max_iter=30, rtol=1e-13)
    assert rel(Lm, Ls) < 1e-11, (it, hist)


def test_degenerate_hierarchies_exact_in_one_iteration():
    K, b, u0, h = _mgrit_case(seed=26, N=16)
    S = O.serial_forward(u0, K, b, h, "tanh")
    U = np.zeros_like(S)
    U[0] = u0
    # one level: the coarsest-level solve is serial propagation
    Um, _, _ = O.mgrit_forward(U, K, b, h, "tanh", cf=4, max_levels=1, max_iter=1)
    assert np.abs(Um - S).max() == 0.0
    # c = N with two levels: one interval; F-relaxation plus the exact coarse solve
    Um, _, _ = O.mgrit_forward(U, K, b, h, "tanh", cf=16, max_levels=2, relax="F", max_iter=1)
    assert np.abs(Um - S).max() < 1e-14


def test_monotone_residual_on_tiny_config():
    wl = WORKLOADS[1]
    d = generate(wl)
    u0 = O.open_forward(d["y"], d["L_in"], wl.act, wl.opening)
    U = np.zeros((wl.N + 1,) + u0.shape)
    U[0] = u0
    _, hist, _ = O.mgrit_forward(U, d["K"], d["b"], wl.h, wl.act, cf=wl.cf, max_levels=wl.max_levels,
                                 relax=wl.relax, max_iter=8)
    for m in range(len(hist) - 1):
        if hist[m] > 1e-12 * hist[0]:
            assert hist[m + 1] < hist[m], hist
    # two-level FCF with N/c = 8 intervals is exact after 4 iterations
    assert hist[4] <= 1e-13 * hist[0]
    S = O.serial_forward(u0, d["K"], d["b"], wl.h, wl.act)
    lamN = O.loss_terminal(S[-1], d["W"], d["mu"], d["onehot"])[1]
    L0 = np.zeros_like(S)
    L0[-1] = lamN
    _, hist, _ = O.mgrit_adjoint(S, L0, d["K"], d["b"], wl.h, wl.act, cf=wl.cf,
                                 max_levels=wl.max_levels, relax=wl.relax, max_iter=8)
    for m in range(len(hist) - 1):
        if hist[m] > 1e-12 * hist[0]:
            assert hist[m + 1] < hist[m], hist


def test_adjoint_mgrit_is_linear_in_terminal_value():
    K, b, u0, h = _mgrit_case(seed=27, N=64)
    U = O.serial_forward(u0, K, b, h, "tanh")
    lamN = np.random.default_rng(3).standard_normal(u0.shape)
    L0 = np.zeros_like(U)
    L0[-1] = lamN
    L1, _, _ = O.mgrit_adjoint(U, L0, K, b, h, "tanh", cf=4, max_levels=3, max_iter=2)
    L2, _, _ = O.mgrit_adjoint(U, 2.5 * L0, K, b, h, "tanh", cf=4, max_levels=3, max_iter=2)
    assert rel(L2, 2.5 * L1) < 1e-14


def test_converged_mgrit_gradient_equals_serial_gradient():
    # Remark after Section 3.3: converged state and adjoint MGRIT give the reduced gradient
    K, b, u0, h = _mgrit_case(seed=28, N=64)
    S = O.serial_forward(u0, K, b, h, "tanh")
    lamN = np.random.default_rng(4).standard_normal(u0.shape)
    Ls = O.serial_adjoint(S, lamN, K, b, h, "tanh")
    U = np.zeros_like(S)
    U[0] = u0
    Um, _, _ = O.mgrit_forward(U, K, b, h, "tanh", cf=4, max_levels=3, max_iter=20, rtol=1e-14)
    L0 = np.zeros_like(S)
    L0[-1] = lamN
    Lm, _, _ = O.mgrit_adjoint(Um, L0, K, b, h, "tanh", cf=4, max_levels=3, max_iter=20, rtol=1e-14)
    dK, db = O.gradient(S, Ls, K, b, h, "tanh")
    dKm, dbm = O.gradient(Um, Lm, K, b, h, "tanh")
    assert rel(dKm, dK) < 1e-11 and rel(dbm, db) < 1e-11


def test_one_shot_with_many_inner_iterations_is_serial_training():
    # Section 4: for large m1, m2 the simultaneous method recovers layer-serial training
    wl = WORKLOADS[5].with_overrides(N=16, B=24, n_features=6)
    d = generate(wl)
    args = (d["y"], d["onehot"], d["L_in"], d["K"], d["b"], d["W"], d["mu"], wl.h, wl.act, wl.opening)
    ls, ws = O.serial_training(*args, updates=4, lr=0.5)
    lo, wo = O.one_shot(*args, cf=4, max_levels=2, min_coarse=1, relax="FCF", updates=4, lr=0.5,
                        m1=4, m2=4)
    assert np.allclose(lo, ls, rtol=1e-12, atol=0)
    for k in ws:
        assert rel(wo[k], ws[k]) < 1e-12
    # with one inner iteration the trajectory differs but the loss still decreases
    l1, _ = O.one_shot(*args, cf=4, max_levels=2, min_coarse=1, relax="FCF", updates=4, lr=0.5)
    assert l1[0] == pytest.approx(ls[0], rel=1e-2) and l1[-1] < l1[0]


def test_level_sizes_of_workloads():
    expect = {1: [32, 8], 2: [256, 64, 16], 3: [2048, 512, 128, 32, 8], 4: [512, 128, 32, 8],
              5: [1024, 256, 64], 6: [2048, 512, 128, 32, 8], 7: [2048, 512, 128, 32, 8]}
    for cfg, sizes in expect.items():
        wl = WORKLOADS[cfg]
        assert O.level_sizes(wl.N, wl.cf, wl.max_levels, wl.min_coarse) == sizes
    with pytest.raises(ValueError):
        O.level_sizes(18, 4, 3, 1)


def test_workload_generator_is_deterministic_and_rounded():
    wl = WORKLOADS[2].with_overrides(N=8, B=10)
    a, b = generate(wl), generate(wl)
    for k in a:
        if a[k] is not None:
            assert np.array_equal(a[k], b[k])
    assert a["K"].dtype == np.float32 and a["y"].dtype == np.float32
    s = random_state(wl, 3)
    assert s.shape == (1, 10, 32) and s.dtype == np.float32


@pytest.mark.parametrize("levels,relax,cycle", [(2, "F", "V"), (3, "F", "V"), (3, "FCF", "V"), (4, "FCF", "V"),
                                                (3, "F", "F"), (4, "FCFCF", "F"), (4, "FCFCF", "V")])
def test_exact_coarse_propagators_solve_in_one_vcycle(levels, relax, cycle):
    # Affine steps with a nilpotent K (K^2 = 0) and a bias in K's null space: c^l fine
    # steps of size h equal exactly one step of size c^l h, so the coarse grids of every
    # level represent their fine grids exactly and one V-cycle reaches the serial
    # solution (to rounding) from any initial guess. The guess is random (a cold start
    # leaves errors in range(K), which K annihilates, and would hide a wrong h_l).
    r = np.random.default_rng(29)
    N, B, q, h = 128, 3, 4, 0.07
    K1 = np.zeros((q, q))
    K1[0, 1] = 2.0
    K1[2, 3] = -1.5
    assert not np.any(K1 @ K1)
    b1 = np.array([0.3, 0.0, -0.2, 0.0])
    assert not np.any(K1 @ b1)
    K, b = np.tile(K1, (N, 1, 1)), np.tile(b1, (N, 1))
    u0 = r.standard_normal((B, q))
    S = O.serial_forward(u0, K, b, h, "identity")
    U = r.standard_normal(S.shape)
    U[0] = u0
    Um, _, _ = O.mgrit_forward(U, K, b, h, "identity", cf=4, max_levels=levels, relax=relax,
                               max_iter=1, warm_start=True, cycle=cycle)
    assert rel(Um, S) < 1e-13
    lamN = r.standard_normal((B, q))
    Ls = O.serial_adjoint(S, lamN, K, b, h, "identity")
    L0 = r.standard_normal(S.shape)
    L0[N] = lamN
    Lm, _, _ = O.mgrit_adjoint(S, L0, K, b, h, "identity", cf=4, max_levels=levels, relax=relax,
                               max_iter=1, warm_start=True, cycle=cycle)
    assert rel(Lm, Ls) < 1e-13


def _relax_by_hand(U, K, b, h, kind, c, relax):
    """F- (and C-) relaxation on the finest grid, written from eqs. Frelax / Crelax."""
    U = U.copy()
    N = K.shape[0]

    def F():
        for k in range(N // c):
            for n in range(k * c + 1, (k + 1) * c):
                U[n] = O.phi(U[n - 1], K[n - 1], b[n - 1], h, kind)

    F()
    if relax == "FCF":
        newC = {k * c: O.phi(U[k * c - 1], K[k * c - 1], b[k * c - 1], h, kind) for k in range(1, N // c + 1)}
        for n, v in newC.items():
            U[n] = v
        F()
    return U


@pytest.mark.parametrize("levels,relax,kind", [(2, "F", "tanh"), (2, "FCF", "tanh"), (3, "FCF", "relu")])
def test_reported_residual_is_full_grid_residual_of_relaxed_iterate(levels, relax, kind):
    # rho_m (Algorithm 1, step 2) is ||G - A(U)|| of the iterate after the relaxation of
    # iteration m; F-point rows of the residual vanish after F-relaxation.
    K, b, u0, h = _mgrit_case(seed=30, N=64, act=kind)
    U = np.zeros((K.shape[0] + 1,) + u0.shape)
    U[0] = u0
    for k in range(1, 64 // 4 + 1):
        U[4 * k] = u0
    _, hist, _ = O.mgrit_forward(U, K, b, h, kind, cf=4, max_levels=levels, relax=relax, max_iter=3)
    prev = U
    for m in range(3):
        R = _relax_by_hand(prev, K, b, h, kind, 4, relax)
        assert abs(hist[m] - O.residual_norm_state(R, K, b, h, kind)) <= 1e-12 * hist[m]
        prev, _, _ = O.mgrit_forward(U, K, b, h, kind, cf=4, max_levels=levels, relax=relax,
                                     max_iter=m + 1)
    # adjoint: same statement on the reversed system
    S = O.serial_forward(u0, K, b, h, kind)
    lamN = np.random.default_rng(5).standard_normal(u0.shape)
    L0 = np.zeros_like(S)
    L0[-1] = lamN
    _, hist, _ = O.mgrit_adjoint(S, L0, K, b, h, kind, cf=4, max_levels=levels, relax=relax, max_iter=2)
    cold = L0.copy()
    for k in range(64 // 4):
        cold[4 * k] = lamN
    Nn = 64
    Lr = cold.copy()
    for k in range(Nn // 4):
        for n in range((k + 1) * 4 - 1, k * 4, -1):
            Lr[n] = O.phibar(Lr[n + 1], S[n], K[n], b[n], h, kind)
    if relax == "FCF":
        newC = {k * 4: O.phibar(Lr[k * 4 + 1], S[k * 4], K[k * 4], b[k * 4], h, kind) for k in range(Nn // 4)}
        for n, v in newC.items():
            Lr[n] = v
        for k in range(Nn // 4):
            for n in range((k + 1) * 4 - 1, k * 4, -1):
                Lr[n] = O.phibar(Lr[n + 1], S[n], K[n], b[n], h, kind)
    assert abs(hist[0] - O.residual_norm_adjoint(S, Lr, K, b, h, kind)) <= 1e-12 * hist[0]


# ---------------------------------------------------------------- F-cycles

@pytest.mark.parametrize("relax,N", [("F", 32), ("FCF", 64)])
def test_fcycle_with_exactly_solved_level_one_equals_two_level(relax, N):
    # c = 4, three levels: level 1 has N/4 points in N/16 coarse intervals. An
    # F-cycle solves level 1's coarse problem with two two-level cycles (the
    # recursive F-cycle, then the V-cycle), and two-level MGRIT with F-relaxation is
    # exact on 2 intervals after 2 iterations (FCF: on 4 intervals after 2), so the
    # three-level F-cycle must coincide with the two-level V-cycle, iterate by
    # iterate, forward and adjoint. A three-level V-cycle (one level-1 cycle) does not.
    K, b, u0, h = _mgrit_case(seed=31, N=N)
    N = K.shape[0]
    U = np.zeros((N + 1,) + u0.shape)
    U[0] = u0
    for m in (1, 2, 3):
        F3, hF, _ = O.mgrit_forward(U, K, b, h, "tanh", cf=4, max_levels=3, relax=relax, max_iter=m, cycle="F")
        V2, hV, _ = O.mgrit_forward(U, K, b, h, "tanh", cf=4, max_levels=2, relax=relax, max_iter=m)
        V3, _, _ = O.mgrit_forward(U, K, b, h, "tanh", cf=4, max_levels=3, relax=relax, max_iter=m)
        assert rel(F3, V2) < 1e-13 and np.allclose(hF, hV, rtol=1e-12, atol=0), m
        if m == 1:
            assert rel(V3, V2) > 1e-8
    S = O.serial_forward(u0, K, b, h, "tanh")
    lamN = np.random.default_rng(3).standard_normal(u0.shape)
    Lm = np.zeros_like(S)
    Lm[N] = lamN
    for m in (1, 2):
        F3, _, _ = O.mgrit_adjoint(S, Lm, K, b, h, "tanh", cf=4, max_levels=3, relax=relax, max_iter=m, cycle="F")
        V2, _, _ = O.mgrit_adjoint(S, Lm, K, b, h, "tanh", cf=4, max_levels=2, relax=relax, max_iter=m)
        assert rel(F3, V2) < 1e-13, m


def test_fcycle_on_two_levels_is_the_vcycle():
    K, b, u0, h = _mgrit_case(seed=32, N=24)
    U = np.zeros((25,) + u0.shape)
    U[0] = u0
    a, _, _ = O.mgrit_forward(U, K, b, h, "tanh", cf=4, max_levels=2, max_iter=2, cycle="F")
    v, _, _ = O.mgrit_forward(U, K, b, h, "tanh", cf=4, max_levels=2, max_iter=2, cycle="V")
    assert np.array_equal(a, v)


@pytest.mark.parametrize("act", ["tanh", "relu", "smoothrelu"])
@pytest.mark.parametrize("relax,cycle", [("FCFCF", "V"), ("FCF", "F"), ("F", "F")])
def test_cycle_variants_converge_to_the_serial_solution(act, relax, cycle):
    # the serial trajectory is the fixed point of every cycle (FAS), and with five
    # levels the iteration reaches it
    K, b, u0, h = _mgrit_case(seed=33, N=256, B=4, q=6, act=act, kscale=0.3)
    N = K.shape[0]
    S = O.serial_forward(u0, K, b, h, act)
    U = np.zeros_like(S)
    U[0] = u0
    Um, hist, it = O.mgrit_forward(U, K, b, h, act, cf=4, max_levels=5, relax=relax, cycle=cycle, max_iter=40,
                                   rtol=1e-13)
    assert rel(Um, S) < 1e-11, (it, hist[-3:])
    lamN = np.random.default_rng(4).standard_normal(u0.shape)
    Ls = O.serial_adjoint(S, lamN, K, b, h, act)
    L0 = np.zeros_like(S)
    L0[N] = lamN
    Lm, _, it = O.mgrit_adjoint(S, L0, K, b, h, act, cf=4, max_levels=5, relax=relax, cycle=cycle, max_iter=40,
                                rtol=1e-13)
    assert rel(Lm, Ls) < 1e-11, it


def test_fcycle_converges_no_slower_than_the_vcycle():
    # more work on the coarse grids per cycle: after a few cycles the F-cycle's
    # residual is below the V-cycle's on a five-level hierarchy
    K, b, u0, h = _mgrit_case(seed=34, N=1024, B=3, q=5, kscale=0.5)
    U = np.zeros((1025,) + u0.shape)
    U[0] = u0
    _, hV, _ = O.mgrit_forward(U, K, b, h, "tanh", cf=4, max_levels=5, relax="FCF", max_iter=4, cycle="V")
    _, hF, _ = O.mgrit_forward(U, K, b, h, "tanh", cf=4, max_levels=5, relax="FCF", max_iter=4, cycle="F")
    assert hF[0] == hV[0]  # the first residual is taken before any coarse-grid work
    assert hF[-1] < hV[-1]


# ---------------------------------------------------------------- Algorithm 2 with L-BFGS

def _pairs(seed, n, m):
    r = np.random.default_rng(seed)
    A = r.standard_normal((n, n))
    A = A @ A.T + n * np.eye(n)  # SPD: y = A s gives s.y > 0
    pairs = []
    for _ in range(m):
        s = r.standard_normal(n)
        pairs.append(([s[:3], s[3:]], [(A @ s)[:3], (A @ s)[3:]]))
    return pairs, r


def test_lbfgs_two_loop_applies_the_dense_bfgs_updates():
    # textbook BFGS inverse update H <- (I - rho s y^T) H (I - rho y s^T) + rho s s^T,
    # applied to H0 = gamma I (gamma from the newest pair) for the stored pairs in order
    n = 7
    pairs, r = _pairs(40, n, 4)
    flat = [(np.concatenate(s), np.concatenate(y)) for s, y in pairs]
    gamma = flat[-1][0] @ flat[-1][1] / (flat[-1][1] @ flat[-1][1])
    H = gamma * np.eye(n)
    for s, y in flat:
        rho = 1.0 / (s @ y)
        V = np.eye(n) - rho * np.outer(y, s)
        H = V.T @ H @ V + rho * np.outer(s, s)
    g = r.standard_normal(n)
    got = np.concatenate(O.lbfgs_direction([g[:3], g[3:]], pairs))
    assert np.allclose(got, H @ g, rtol=1e-12, atol=1e-12)
    # the newest secant equation H y = s, and no pairs: H = I
    s_new, y_new = pairs[-1]
    assert np.allclose(np.concatenate(O.lbfgs_direction(y_new, pairs)), np.concatenate(s_new), rtol=1e-12)
    assert np.array_equal(np.concatenate(O.lbfgs_direction([g[:3], g[3:]], [])), g)


def test_accuracy_counts_argmax_hits():
    r = np.random.default_rng(41)
    uN, W, mu = r.standard_normal((50, 6)), r.standard_normal((4, 6)), r.standard_normal(4)
    labels = r.integers(0, 4, 50)
    hits = sum(int(np.argmax(W @ uN[k] + mu) == labels[k]) for k in range(50))
    assert O.accuracy(uN, W, mu, labels) == hits / 50


def _lbfgs_case():
    wl = WORKLOADS[5].with_overrides(N=32, B=120, n_features=20)
    d = generate(wl.with_overrides(B=wl.B + 80))
    tr = {k: (v[:wl.B] if k in ("y", "onehot", "labels") else v) for k, v in d.items()}
    va = {k: d[k][wl.B:] for k in ("y", "onehot", "labels")}
    return wl, tr, va


def test_one_shot_lbfgs_converges_on_the_training_set_and_stops_on_validation():
    wl, d, va = _lbfgs_case()
    args = (d["y"], d["onehot"], d["L_in"], d["K"], d["b"], d["W"], d["mu"], wl.h, wl.act, wl.opening)
    kw = dict(cf=4, max_levels=3, min_coarse=1, relax="FCF", m1=2, m2=2, alpha0=0.5)
    r = O.one_shot_lbfgs(*args, updates=12, **kw)
    assert r["losses"][-1] < 0.05 * r["losses"][0]
    assert r["alphas"][0] <= 0.5 and all(0 < a <= 1.0 for a in r["alphas"])
    # a stochastic-gradient run of the same length (Algorithm 2 with a scaled identity)
    # stays far above: the curvature pairs are doing the work
    ls, _ = O.one_shot(*args, cf=4, max_levels=3, min_coarse=1, relax="FCF", updates=12, lr=0.5, m1=2, m2=2)
    assert r["losses"][-1] < 0.5 * ls[-1]
    # the validation stop ends the run at the first update that reaches the target
    full = O.one_shot_lbfgs(*args, updates=12, y_val=va["y"], onehot_val=va["onehot"], **kw)
    target = sorted(full["accuracies"])[len(full["accuracies"]) // 2]
    first = next(i for i, a in enumerate(full["accuracies"]) if a >= target)
    stop = O.one_shot_lbfgs(*args, updates=12, y_val=va["y"], onehot_val=va["onehot"], target_acc=target, **kw)
    assert len(stop["losses"]) == first + 1 and stop["accuracies"] == full["accuracies"][:first + 1]


def test_one_shot_lbfgs_with_exact_inner_solves_takes_exact_gradients():
    # with many inner iterations the MGRIT states are the serial ones, so the first
    # direction is -alpha0 times the exact reduced gradient (serial backpropagation)
    wl, d, _ = _lbfgs_case()
    args = (d["y"], d["onehot"], d["L_in"], d["K"], d["b"], d["W"], d["mu"], wl.h, wl.act, wl.opening)
    r = O.one_shot_lbfgs(*args, updates=1, cf=4, max_levels=3, min_coarse=1, relax="FCF", m1=30, m2=30,
                         alpha0=0.25, max_ls=1)
    _, wo = O.serial_training(*args, updates=1, lr=0.25)
    for k in ("K", "b", "W", "mu", "L_in"):
        assert rel(r["weights"][k], wo[k]) < 1e-10, k


def test_working_precision_changes_only_the_rounding():
    """The benchmark times the oracle in a workload's own dtype. Under
    working_precision(float32) every result is float32 and agrees with the fp64
    default to fp32 rounding; leaving the context restores fp64."""
    from workloads import WORKLOADS, generate
    wl = WORKLOADS[2].with_overrides(N=16, B=64, max_levels=2)
    d = generate(wl)
    u0 = O.open_forward(d["y"], d["L_in"], wl.act, wl.opening)
    U64 = O.serial_forward(u0, d["K"], d["b"], wl.h, wl.act)
    M64, h64, _ = O.mgrit_forward(np.concatenate([u0[None], np.zeros((wl.N,) + u0.shape)]), d["K"], d["b"], wl.h,
                                  wl.act, cf=4, max_levels=2, max_iter=2)
    with O.working_precision(np.float32):
        U32 = O.serial_forward(u0, d["K"], d["b"], wl.h, wl.act)
        lam = O.loss_terminal(U32[-1], d["W"], d["mu"], d["onehot"])[1]
        L32 = O.serial_adjoint(U32, lam, d["K"], d["b"], wl.h, wl.act)
        dK32, _ = O.gradient(U32, L32, d["K"], d["b"], wl.h, wl.act)
        M32, h32, _ = O.mgrit_forward(np.concatenate([u0[None], np.zeros((wl.N,) + u0.shape)]), d["K"], d["b"],
                                      wl.h, wl.act, cf=4, max_levels=2, max_iter=2)
    assert U32.dtype == L32.dtype == dK32.dtype == M32.dtype == np.float32
    assert np.linalg.norm(U32 - U64) <= 1e-5 * np.linalg.norm(U64)
    assert np.linalg.norm(M32 - M64) <= 1e-5 * np.linalg.norm(M64)
    assert abs(h32[-1] - h64[-1]) <= 1e-4 * h64[-1]
    assert O.serial_forward(u0, d["K"], d["b"], wl.h, wl.act).dtype == np.float64


def test_expand_cpoints_reproduces_stored_trajectories():
    """C-point storage keeps u^{kc} only; the F-points follow by forward steps. From
    the C-points of the serial solution this is the serial solution (the state
    equations, Section 2.3), and from those of an MGRIT iterate it is that iterate,
    whose last sweep is an F-relaxation (Algorithm 1, step 5)."""
    from workloads import WORKLOADS, generate
    for wl in (WORKLOADS[1], WORKLOADS[2].with_overrides(N=32, B=20)):
        d = generate(wl)
        u0 = O.open_forward(d["y"], d["L_in"], wl.act, wl.opening)
        S = O.serial_forward(u0, d["K"], d["b"], wl.h, wl.act)
        E = O.expand_cpoints(S[::wl.cf], d["K"], d["b"], wl.h, wl.act, wl.cf)
        assert np.array_equal(E, S)
        U0 = np.concatenate([u0[None], np.zeros((wl.N,) + u0.shape)])
        M, _, _ = O.mgrit_forward(U0, d["K"], d["b"], wl.h, wl.act, cf=wl.cf, max_levels=2, max_iter=1)
        E = O.expand_cpoints(M[::wl.cf], d["K"], d["b"], wl.h, wl.act, wl.cf)
        assert np.max(np.abs(E - M)) <= 1e-15 * np.max(np.abs(M))
        # a non-converged iterate: its F-points are not the serial ones
        assert np.max(np.abs(M - S)) > 1e-8


def _line(f, df):
    return (lambda a: (f(a), a)), df


@pytest.mark.parametrize("c2", [0.9, 0.1])
def test_strong_wolfe_search_on_analytic_lines(c2):
    """The line search the paper names (strong Wolfe conditions, Section 4) on 1-D
    functions whose acceptable steps are known in closed form: a quadratic with its
    minimum beyond the first trial (doubling, then zoom), one with its minimum far
    inside it (zoom by bisection from the overshoot), a smooth multi-modal
    function, and a first step that lowers phi while overshooting; each accepted
    step meets both conditions evaluated here directly."""
    c1 = 1e-4
    cases = [
        (lambda a: (a - 3.0) ** 2, lambda a: 2.0 * (a - 3.0)),
        (lambda a: (a - 0.1) ** 2, lambda a: 2.0 * (a - 0.1)),
        # the first step decreases phi but overshoots with a large positive slope: the
        # weak curvature condition would take it, the strong one (c2 = 0.1) does not
        (lambda a: (a - 0.6) ** 2, lambda a: 2.0 * (a - 0.6)),
        (lambda a: -np.exp(-(a - 1.7) ** 2) - 0.2 * np.sin(4.0 * a),
         lambda a: 2.0 * (a - 1.7) * np.exp(-(a - 1.7) ** 2) - 0.8 * np.cos(4.0 * a)),
    ]
    for f, df in cases:
        J, gd = f(0.0), df(0.0)
        assert gd < 0.0
        phi, dphi = _line(f, df)
        a, n, met = O.strong_wolfe_search(phi, dphi, J, gd, 1.0, c1, c2, 30)
        assert met and 1 <= n <= 30
        assert f(a) <= J + c1 * a * gd
        assert abs(df(a)) <= c2 * abs(gd)
    # the quadratic's acceptable set is |2 (a - 3)| <= 6 c2 (sufficient decrease holds there)
    phi, dphi = _line(*cases[0])
    a, _, _ = O.strong_wolfe_search(phi, dphi, 9.0, -6.0, 1.0, c1, c2, 30)
    assert abs(a - 3.0) <= 3.0 * c2
    if c2 == 0.1:
        assert a == 3.0  # 1, 2, 4 (no decrease from 2), then the bracket's midpoint


def test_strong_wolfe_search_limits():
    """Without an acceptable step within max_ls evaluations: a line that keeps
    descending ends at the last doubled step; a minimum far below every trial
    ends at the last bisected step (nothing met sufficient decrease)."""
    phi, dphi = _line(lambda a: -a, lambda a: -1.0)
    a, n, met = O.strong_wolfe_search(phi, dphi, 0.0, -1.0, 1.0, 1e-4, 0.9, 8)
    assert (a, n, met) == (128.0, 8, False)
    phi, dphi = _line(lambda a: (a - 1e-6) ** 2, lambda a: 2.0 * (a - 1e-6))
    a, n, met = O.strong_wolfe_search(phi, dphi, 1e-12, -2e-6, 1.0, 1e-4, 0.9, 3)
    assert (a, n, met) == (0.25, 3, False)


def test_one_shot_lbfgs_with_strong_wolfe_steps():
    """Algorithm 2 with the strong Wolfe line search on a small Peaks-shaped
    problem: every update finds a step meeting both conditions and the loss falls."""
    wl = WORKLOADS[1].with_overrides(N=16, B=60, max_levels=2)
    d = generate(wl)
    r = O.one_shot_lbfgs(d["y"], d["onehot"], d["L_in"], d["K"], d["b"], d["W"], d["mu"], wl.h, wl.act,
                         wl.opening, cf=wl.cf, max_levels=wl.max_levels, min_coarse=wl.min_coarse, relax=wl.relax,
                         updates=5, alpha0=0.5, line_search="wolfe")
    assert r["wolfe"] == [True] * 5
    assert r["losses"][-1] < r["losses"][0]
    assert all(1 <= t <= 8 for t in r["trials"])
