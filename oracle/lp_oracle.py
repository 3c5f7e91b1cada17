"""CPU oracle for layer-parallel ResNet training (Guenther et al., arXiv:1812.04352).

TEST INFRASTRUCTURE ONLY. This module is the plain, slow, fp64 statement of what
the GPU library computes. Only the test suite, the smoke check and the CPU
baseline leg of the benchmark may import it; the product path never does.
It shares no code with the HIP library.

Conventions (all arrays fp64 NumPy):
  state slice    v [B][q]            (conv: [B][C][H][W])
  trajectory     U [N+1][B][q]       (layer index outermost)
  dense weights  K [N][q][q]         K[n][i][j] maps input feature j to output i
  conv weights   K [N][C][C][3][3]   K[n][co][ci][ty][tx], cross-correlation, zero "same" padding
  bias           b [N][q]            (conv: [N][C], one bias per channel)

Every function names the passage of the paper it follows. Where the paper is
silent the reading taken is stated in the docstring.

Parity status: every function here is pinned by the CPU test suite against an
independent source (closed forms, torch autograd, central finite differences,
finite-step exactness of MGRIT, the MGRIT fixed point). The MGRIT iterate after a
fixed, non-converged number of iterations with ReLU or more than two levels has
no closed form: it is pinned only through the oracle's own structure (the same
code reaches the pinned serial solution as iterations grow, and the two-level F
and FCF cases are exact after the finite step counts proven for Parareal).
"""
from __future__ import annotations

import numpy as np


# Working precision of every function below: fp64 for all parity uses. Only the
# benchmark's CPU timing switches it (working_precision) to time the oracle in a
# workload's own dtype; the arithmetic is the same either way.
_DT = np.float64


class working_precision:
    """Context manager: run the oracle in the given numpy float dtype."""

    def __init__(self, dtype):
        self.dtype = np.dtype(dtype).type

    def __enter__(self):
        global _DT
        self.prev, _DT = _DT, self.dtype
        return self

    def __exit__(self, *exc):
        global _DT
        _DT = self.prev
        return False


def _f64(*arrays):
    """Upcast inputs (typically already rounded to the workload dtype) to fp64
    (to the working precision when the benchmark has changed it)."""
    out = tuple(None if a is None else np.asarray(a, dtype=_DT) for a in arrays)
    return out if len(out) > 1 else out[0]


# ---------------------------------------------------------------------------
# Activations (Section 2.1, single-layer perceptron; Section 5.1 smoothed ReLU)
# ---------------------------------------------------------------------------

def act(z, kind):
    """sigma applied componentwise.

    tanh and ReLU are the examples of Section 2.1. The smoothed ReLU of the Peaks
    test case (Section 5.1) is max(x, 0) for |x| > 0.1 and the quadratic
    2.5 x^2 + 0.5 x + 0.025 for |x| <= 0.1 (the printed mixed number "2 1/2" read
    as 5/2; this is the reading that makes sigma continuously differentiable).
    "identity" is a test-only activation that makes the step affine.
    """
    if kind == "tanh":
        return np.tanh(z)
    if kind == "relu":
        return np.maximum(z, 0.0)
    if kind == "smoothrelu":
        quad = 2.5 * z * z + 0.5 * z + 0.025
        return np.where(np.abs(z) <= 0.1, quad, np.maximum(z, 0.0))
    if kind == "identity":
        return z.copy()
    raise ValueError(kind)


def dact(z, kind):
    """sigma'(z). ReLU takes sigma'(0) = 0 (the paper is silent)."""
    if kind == "tanh":
        t = np.tanh(z)
        return 1.0 - t * t
    if kind == "relu":
        return (z > 0.0).astype(z.dtype)
    if kind == "smoothrelu":
        return np.where(np.abs(z) <= 0.1, 5.0 * z + 0.5, (z > 0.0).astype(z.dtype))
    if kind == "identity":
        return np.ones_like(z)
    raise ValueError(kind)


# ---------------------------------------------------------------------------
# The linear operator K(theta) (Section 2.1): dense matrix or 3x3 convolution
# ---------------------------------------------------------------------------

def conv3x3(Kn, v):
    """z[b,co,y,x] = sum_{ci,dy,dx} Kn[co,ci,dy+1,dx+1] v[b,ci,y+dy,x+dx], zero padded."""
    Bn, C, H, W = v.shape
    vp = np.zeros((Bn, C, H + 2, W + 2), dtype=v.dtype)
    vp[:, :, 1:H + 1, 1:W + 1] = v
    z = np.zeros((Bn, Kn.shape[0], H, W), dtype=v.dtype)
    for ty in range(3):
        for tx in range(3):
            z += np.einsum("oc,bcyx->boyx", Kn[:, :, ty, tx], vp[:, :, ty:ty + H, tx:tx + W])
    return z


def conv3x3_transpose(Kn, s):
    """Adjoint of conv3x3 with respect to its input: scatter every output back to
    the inputs that produced it, then drop the padding."""
    Bn, Co, H, W = s.shape
    gp = np.zeros((Bn, Kn.shape[1], H + 2, W + 2), dtype=s.dtype)
    for ty in range(3):
        for tx in range(3):
            gp[:, :, ty:ty + H, tx:tx + W] += np.einsum("oc,boyx->bcyx", Kn[:, :, ty, tx], s)
    return gp[:, :, 1:H + 1, 1:W + 1]


def conv3x3_weight_grad(s, v):
    """d/dKn of sum(s * conv3x3(Kn, v)): [Co][Ci][3][3]."""
    Bn, C, H, W = v.shape
    vp = np.zeros((Bn, C, H + 2, W + 2), dtype=v.dtype)
    vp[:, :, 1:H + 1, 1:W + 1] = v
    g = np.zeros((s.shape[1], C, 3, 3), dtype=v.dtype)
    for ty in range(3):
        for tx in range(3):
            g[:, :, ty, tx] = np.einsum("boyx,bcyx->oc", s, vp[:, :, ty:ty + H, tx:tx + W])
    return g


def _is_conv(Kn):
    return Kn.ndim == 4


def linop(Kn, v):
    """K(theta^n) v for a batch v."""
    return conv3x3(Kn, v) if _is_conv(Kn) else v @ Kn.T


def linop_T(Kn, s):
    """K(theta^n)^T s for a batch s."""
    return conv3x3_transpose(Kn, s) if _is_conv(Kn) else s @ Kn


def add_bias(z, bn):
    """z + B theta^(2): per-feature bias (dense) or per-channel bias (conv)."""
    return z + (bn[None, :, None, None] if z.ndim == 4 else bn[None, :])


def preact(Kn, bn, v):
    """z = K v + b, the argument of sigma in the single-layer perceptron."""
    return add_bias(linop(Kn, v), bn)


# ---------------------------------------------------------------------------
# Layer step Phi and its adjoint (Section 2.2 forward Euler; Section 3.2)
# ---------------------------------------------------------------------------

def phi(v, Kn, bn, hl, kind):
    """Phi(v, theta^n) = v + h F(v, theta^n), F = sigma(K v + b) (forward Euler ResNet step).
    On a coarse level the same step is taken with h_l = c^l h (re-discretisation, Section 3.1.1)."""
    return v + hl * act(preact(Kn, bn, v), kind)


def phibar(lam, u, Kn, bn, hl, kind):
    """(d_u Phi(u, theta^n))^T lam = lam + h K^T (sigma'(K u + b) * lam) (Section 3.2)."""
    s = dact(preact(Kn, bn, u), kind) * lam
    return lam + hl * linop_T(Kn, s)


# ---------------------------------------------------------------------------
# Plain definitions: layer-serial forward, adjoint (backpropagation), gradient
# ---------------------------------------------------------------------------

def serial_forward(u0, K, b, h, kind):
    """State equations u^{n+1} = Phi(u^n, theta^n), n = 0..N-1 (Section 2.3, item 1),
    solved by forward substitution. Returns U [N+1][...]."""
    u0, K, b = _f64(u0, K, b)
    N = K.shape[0]
    U = np.empty((N + 1,) + u0.shape, dtype=_DT)
    U[0] = u0
    for n in range(N):
        U[n + 1] = phi(U[n], K[n], b[n], h, kind)
    return U


def serial_adjoint(U, lamN, K, b, h, kind):
    """Adjoint equations lam^n = (d_u Phi^n)^T lam^{n+1}, n = N-1..0, from the terminal
    value lam^N (Section 2.3, item 2); this is backpropagation. Returns Lam [N+1][...]."""
    U, lamN, K, b = _f64(U, lamN, K, b)
    N = K.shape[0]
    Lam = np.empty_like(U)
    Lam[N] = lamN
    for n in range(N - 1, -1, -1):
        Lam[n] = phibar(Lam[n + 1], U[n], K[n], b[n], h, kind)
    return Lam


def expand_cpoints(Uc, K, b, h, kind, cf):
    """The trajectory implied by C-point storage (Section 3.2, remark on storing or
    recomputing the primal states the adjoint depends on): row k of Uc is the state
    at the C-point k*cf; each F-point is the forward step from the one before,
    u^{kc+j} = Phi(u^{kc+j-1}, theta^{kc+j-1}), j = 1..cf-1 (the F-relaxation, eq.
    Frelax, on the finest level). Returns U [N+1][...]."""
    Uc, K, b = _f64(Uc, K, b)
    N = K.shape[0]
    U = np.empty((N + 1,) + Uc.shape[1:], dtype=_DT)
    for k in range(N // cf):
        U[k * cf] = Uc[k]
        for j in range(1, cf):
            n = k * cf + j
            U[n] = phi(U[n - 1], K[n - 1], b[n - 1], h, kind)
    U[N] = Uc[N // cf]
    return U


def gradient(U, Lam, K, b, h, kind):
    """Design equations for theta^n (Section 2.3, item 3) with R = 0:
    dJ/dK_n = sum_k (d_K Phi(u_k^n))^T lam_k^{n+1} = h sum_k (sigma'(z_k^n) * lam_k^{n+1}) u_k^n^T,
    dJ/db_n = h sum_k sigma'(z_k^n) * lam_k^{n+1}. The 1/s factor lives in lam^N.
    Returns (dK like K, db like b)."""
    U, Lam, K, b = _f64(U, Lam, K, b)
    N = K.shape[0]
    dK = np.empty(K.shape, dtype=_DT)
    db = np.empty(b.shape, dtype=_DT)
    for n in range(N):
        s = dact(preact(K[n], b[n], U[n]), kind) * Lam[n + 1]
        if _is_conv(K[n]):
            dK[n] = h * conv3x3_weight_grad(s, U[n])
            db[n] = h * s.sum(axis=(0, 2, 3))
        else:
            dK[n] = h * (s.T @ U[n])
            db[n] = h * s.sum(axis=0)
    return dK, db


# ---------------------------------------------------------------------------
# Boundary: opening layer, softmax hypothesis and cross-entropy (Section 2.1)
# ---------------------------------------------------------------------------

def open_forward(y, L_in, kind, opening):
    """u^0 = L_in y. The Peaks network applies the activation after a learned dense
    L_in (Section 5.1); here "dense_act" is that, "conv_act" is a learned 3x3
    convolution 1 -> C channels (no bias) followed by the activation, and
    "identity" is u^0 = y."""
    y, L_in = _f64(y, L_in)
    if opening == "identity":
        return y.copy()
    if opening == "dense_act":
        return act(y @ L_in.T, kind)
    if opening == "conv_act":
        return act(conv3x3(L_in, y), kind)
    raise ValueError(opening)


def open_grad(y, L_in, lam0, kind, opening):
    """dJ/dL_in from the Lagrangian term lam^0^T (L_in y - u^0) composed with the
    activation: sum_k (sigma'(L_in y_k) * lam_k^0) y_k^T."""
    y, L_in, lam0 = _f64(y, L_in, lam0)
    if opening == "dense_act":
        s = dact(y @ L_in.T, kind) * lam0
        return s.T @ y
    if opening == "conv_act":
        s = dact(conv3x3(L_in, y), kind) * lam0
        return conv3x3_weight_grad(s, y)
    raise ValueError(opening)


def _flat(u):
    return u.reshape(u.shape[0], -1)


def loss_terminal(uN, W, mu, onehot):
    """Softmax hypothesis S = exp(z)/(e^T exp(z)), z = W u^N + mu, and the mean
    cross-entropy J = (1/s) sum_k -c_k^T log S_k over the batch (Section 2.1, with the
    batch as the sample set, s -> B). Returns
      J, lam^N = (1/s) (d_u l)^T = (1/s) W^T (S - c)  (Section 2.3, adjoint terminal value),
      dW = (1/s) sum_k (S_k - c_k) u_k^N^T,  dmu = (1/s) sum_k (S_k - c_k)."""
    uN, W, mu, onehot = _f64(uN, W, mu, onehot)
    Bn = uN.shape[0]
    uf = _flat(uN)
    z = uf @ W.T + mu
    zmax = z.max(axis=1, keepdims=True)
    ez = np.exp(z - zmax)
    S = ez / ez.sum(axis=1, keepdims=True)
    logS = (z - zmax) - np.log(ez.sum(axis=1, keepdims=True))
    J = float(-(onehot * logS).sum() / Bn)
    d = (S - onehot) / Bn
    lamN = (d @ W).reshape(uN.shape)
    dW = d.T @ uf
    dmu = d.sum(axis=0)
    return J, lamN, dW, dmu


def accuracy(uN, W, mu, labels):
    uN, W, mu = _f64(uN, W, mu)
    z = _flat(uN) @ W.T + mu
    return float((np.argmax(z, axis=1) == labels).mean())


# ---------------------------------------------------------------------------
# Residual norms (the stopping quantity ||G - A(U)||, Section 3.1.1 and Alg. 1 step 6)
# ---------------------------------------------------------------------------

def residual_norm_state(U, K, b, h, kind):
    """(sum_{n=1..N} ||Phi(u^{n-1}) - u^n||^2)^{1/2} over examples and features.
    Row 0 of A(U) = G is u^0 = L_in y itself and contributes nothing."""
    U, K, b = _f64(U, K, b)
    N = K.shape[0]
    acc = 0.0
    for n in range(1, N + 1):
        r = phi(U[n - 1], K[n - 1], b[n - 1], h, kind) - U[n]
        acc += float(np.sum(r * r))
    return np.sqrt(acc)


def residual_norm_adjoint(U, Lam, K, b, h, kind):
    """(sum_{n=0..N-1} ||(d_u Phi^n)^T lam^{n+1} - lam^n||^2)^{1/2} (the adjoint system, Section 3.2)."""
    U, Lam, K, b = _f64(U, Lam, K, b)
    N = K.shape[0]
    acc = 0.0
    for n in range(N):
        r = phibar(Lam[n + 1], U[n], K[n], b[n], h, kind) - Lam[n]
        acc += float(np.sum(r * r))
    return np.sqrt(acc)


# ---------------------------------------------------------------------------
# MGRIT with FAS (Section 3.1, Algorithm 1, applied recursively as a V-cycle)
# ---------------------------------------------------------------------------

def level_sizes(N, cf, max_levels, min_coarse):
    """Grid hierarchy: level l has N_l = N / c^l steps (Section 3.1.1). Coarsen while
    another level is allowed and the current level has more than min_coarse steps;
    every coarsened level must divide by c."""
    sizes = [N]
    while len(sizes) < max_levels and sizes[-1] > min_coarse:
        if sizes[-1] % cf:
            raise ValueError("N_l not divisible by the coarsening factor")
        sizes.append(sizes[-1] // cf)
    return sizes


class _Hierarchy:
    """Level data for one MGRIT solve. Level l holds u_l [N_l+1][...] and the
    right-hand side g_l of A_l(u_l) = g_l; theta on level l is injected,
    theta_l^i = theta^{i c^l}, and the step size is h_l = c^l h (Section 3.1.1)."""

    def __init__(self, sizes, cf, h):
        self.sizes = sizes
        self.cf = cf
        self.h = h
        self.u = [None] * len(sizes)
        self.g = [None] * len(sizes)

    def stride(self, l):
        return self.cf ** l

    def hl(self, l):
        return self.h * self.cf ** l


def _fwd_step(H, K, b, kind, l, i, v):
    """Phi_l^i(v): the level-l step from point i to i+1 with theta^{i c^l} and h_l."""
    n = i * H.stride(l)
    return phi(v, K[n], b[n], H.hl(l), kind)


def _fwd_F_relax(H, K, b, kind, l):
    """F-relaxation (eq. Frelax): every interval k propagates its C-point u^{kc}
    through its F-points kc+1 .. kc+c-1. u^i = Phi_l(u^{i-1}) + g^i."""
    c, u, g = H.cf, H.u[l], H.g[l]
    for k in range(H.sizes[l] // c):
        for j in range(1, c):
            i = k * c + j
            u[i] = _fwd_step(H, K, b, kind, l, i - 1, u[i - 1]) + g[i]


def _fwd_C_relax(H, K, b, kind, l):
    """C-relaxation (eq. Crelax): every C-point kc, k = 1..N_l/c, takes the step from
    its left neighbour (all from the values before this sweep: block Jacobi)."""
    c, u, g = H.cf, H.u[l], H.g[l]
    Nc = H.sizes[l] // c
    new = [_fwd_step(H, K, b, kind, l, k * c - 1, u[k * c - 1]) + g[k * c] for k in range(1, Nc + 1)]
    for k in range(1, Nc + 1):
        u[k * c] = new[k - 1]


# C-relaxations in one relaxation sweep: F, FCF (the paper's default, Section
# 3.1.1) and FCFCF (one more C- and F-relaxation pair)
C_SWEEPS = {"F": 0, "FCF": 1, "FCFCF": 2}


def _coarse_solves(cycle, l, L):
    """Cycles that solve the coarse problem of level l (Algorithm 1, step 3) on level
    l + 1: a V-cycle is one recursive V-cycle; an F-cycle (the multigrid F-cycle the
    paper mentions for visiting coarse grids more often) is a recursive F-cycle
    followed by a V-cycle, the latter left out when level l + 1 is the coarsest
    (whose solve is exact, so a second one changes nothing)."""
    if cycle == "V":
        return ["V"]
    if cycle == "F":
        return ["F"] if l + 1 == L - 1 else ["F", "V"]
    raise ValueError(f"unknown cycle {cycle!r}")


def _fwd_cycle(H, K, b, kind, relax, l, rho_out, cycle="V"):
    """One FAS cycle on level l (Algorithm 1, with step 3 recursive: V- or F-cycle)."""
    c, L = H.cf, len(H.sizes)
    u, g = H.u[l], H.g[l]
    Nl = H.sizes[l]
    if l == L - 1:
        # Coarsest level: solve A_l(u) = g exactly by forward substitution.
        for i in range(1, Nl + 1):
            u[i] = _fwd_step(H, K, b, kind, l, i - 1, u[i - 1]) + g[i]
        return
    # Step 1: F-, FCF- or FCFCF-relaxation.
    _fwd_F_relax(H, K, b, kind, l)
    for _ in range(C_SWEEPS[relax]):
        _fwd_C_relax(H, K, b, kind, l)
        _fwd_F_relax(H, K, b, kind, l)
    # Step 2: residual at the C-points and restriction by injection.
    Nc = Nl // c
    f = [None] * (Nc + 1)
    acc = 0.0
    for k in range(1, Nc + 1):
        f[k] = _fwd_step(H, K, b, kind, l, k * c - 1, u[k * c - 1]) + g[k * c]
        r = f[k] - u[k * c]
        acc += float(np.sum(r * r))
    if l == 0:
        rho_out.append(np.sqrt(acc))
    uc = np.empty((Nc + 1,) + u.shape[1:], dtype=u.dtype)
    gc = np.empty_like(uc)
    for k in range(Nc + 1):
        uc[k] = u[k * c]
    # Coarse right-hand side A_c(U_c) + R_c. Row 0 is g^0; row k is
    #   [u^{kc} - Phi_{l+1}(U_c^{k-1})] + [g^{kc} - u^{kc} + Phi_l(u^{kc-1})],
    # in which u^{kc} cancels, leaving f_k - Phi_{l+1}(U_c^{k-1}).
    gc[0] = g[0]
    for k in range(1, Nc + 1):
        gc[k] = f[k] - _fwd_step(H, K, b, kind, l + 1, k - 1, uc[k - 1])
    H.u[l + 1], H.g[l + 1] = uc, gc
    # Step 3: solve the coarse residual equation (recursively).
    for cyc in _coarse_solves(cycle, l, L):
        _fwd_cycle(H, K, b, kind, relax, l + 1, rho_out, cyc)
    # Steps 4-5: E = V - U at the C-points, U^{kc} <- U^{kc} + E^k, then F-relaxation.
    V = H.u[l + 1]
    for k in range(1, Nc + 1):
        E = V[k] - u[k * c]
        u[k * c] = u[k * c] + E
    _fwd_F_relax(H, K, b, kind, l)


def mgrit_forward(U, K, b, h, kind, cf=4, max_levels=2, min_coarse=1, relax="FCF",
                  max_iter=1, rtol=0.0, stag=0.0, warm_start=False, cycle="V"):
    """Solve A(U, theta) = G (eq. nonlinear_mgrit) with MGRIT/FAS iterations: V- or
    F-cycles (cycle "V" | "F"), with F-, FCF- or FCFCF-relaxation.

    U [N+1][...] holds u^0 in row 0; with warm_start the other rows are the initial
    guess, else the C-points start as copies of u^0 (a generic initial condition,
    Section 3.1.1; only C-points matter because the first sweep is an F-relaxation).
    After iteration m, rho_m = ||R|| of Algorithm 1 step 2 at level 0. Stop when
    rtol > 0 and rho_m <= rtol * rho_1, or when stag > 0 and rho_m > stag * rho_{m-1},
    or after max_iter iterations.
    Returns (U_out, res_hist list, iterations)."""
    K, b = _f64(K, b)
    N = K.shape[0]
    sizes = level_sizes(N, cf, max_levels, min_coarse)
    H = _Hierarchy(sizes, cf, h)
    u = np.array(U, dtype=_DT, copy=True)
    if not warm_start and len(sizes) > 1:
        for k in range(1, N // cf + 1):
            u[k * cf] = u[0]
    g = np.zeros_like(u)
    g[0] = u[0]
    H.u[0], H.g[0] = u, g
    hist = []
    it = 0
    for m in range(1, max_iter + 1):
        _fwd_cycle(H, K, b, kind, relax, 0, hist, cycle)
        it = m
        if len(sizes) == 1:
            hist.append(0.0)
        if rtol > 0 and hist[-1] <= rtol * hist[0]:
            break
        if stag > 0 and m > 1 and hist[-1] > stag * hist[-2]:
            break
    return H.u[0], hist, it


def _adj_step(H, U, K, b, kind, l, i, lam):
    """Phibar_l^i(lam) = lam + h_l K^T (sigma'(K u^{n} + b) * lam), n = i c^l: the
    level-l adjoint step from point i+1 to i, linearised at the injected fine
    state u^{i c^l} with the injected theta (re-discretisation of d_u Phi^T)."""
    n = i * H.stride(l)
    return phibar(lam, U[n], K[n], b[n], H.hl(l), kind)


def _adj_F_relax(H, U, K, b, kind, l):
    """Adjoint F-relaxation: interval k runs from its C-point (k+1)c down through
    the F-points (k+1)c-1 .. kc+1 (eq. Frelax applied to the reversed system)."""
    c, lam, g = H.cf, H.u[l], H.g[l]
    for k in range(H.sizes[l] // c):
        for j in range(c - 1, 0, -1):
            i = k * c + j
            lam[i] = _adj_step(H, U, K, b, kind, l, i, lam[i + 1]) + g[i]


def _adj_C_relax(H, U, K, b, kind, l):
    """Adjoint C-relaxation: C-point kc, k = 0..N_l/c - 1, from its right neighbour."""
    c, lam, g = H.cf, H.u[l], H.g[l]
    Nc = H.sizes[l] // c
    new = [_adj_step(H, U, K, b, kind, l, k * c, lam[k * c + 1]) + g[k * c] for k in range(Nc)]
    for k in range(Nc):
        lam[k * c] = new[k]


def _adj_cycle(H, U, K, b, kind, relax, l, rho_out, cycle="V"):
    """Algorithm 1 on the adjoint system A_U(Lam) = G_U (eq. adjointMGRIT), whose
    block rows run backwards in the layer index."""
    c, L = H.cf, len(H.sizes)
    lam, g = H.u[l], H.g[l]
    Nl = H.sizes[l]
    if l == L - 1:
        for i in range(Nl - 1, -1, -1):
            lam[i] = _adj_step(H, U, K, b, kind, l, i, lam[i + 1]) + g[i]
        return
    _adj_F_relax(H, U, K, b, kind, l)
    for _ in range(C_SWEEPS[relax]):
        _adj_C_relax(H, U, K, b, kind, l)
        _adj_F_relax(H, U, K, b, kind, l)
    Nc = Nl // c
    f = [None] * (Nc + 1)
    acc = 0.0
    for k in range(Nc):
        f[k] = _adj_step(H, U, K, b, kind, l, k * c, lam[k * c + 1]) + g[k * c]
        r = f[k] - lam[k * c]
        acc += float(np.sum(r * r))
    if l == 0:
        rho_out.append(np.sqrt(acc))
    lc = np.empty((Nc + 1,) + lam.shape[1:], dtype=lam.dtype)
    gc = np.empty_like(lc)
    for k in range(Nc + 1):
        lc[k] = lam[k * c]
    gc[Nc] = g[Nl]
    for k in range(Nc):
        gc[k] = f[k] - _adj_step(H, U, K, b, kind, l + 1, k, lc[k + 1])
    H.u[l + 1], H.g[l + 1] = lc, gc
    for cyc in _coarse_solves(cycle, l, L):
        _adj_cycle(H, U, K, b, kind, relax, l + 1, rho_out, cyc)
    V = H.u[l + 1]
    for k in range(Nc):
        E = V[k] - lam[k * c]
        lam[k * c] = lam[k * c] + E
    _adj_F_relax(H, U, K, b, kind, l)


def mgrit_adjoint(U, Lam, K, b, h, kind, cf=4, max_levels=2, min_coarse=1, relax="FCF",
                  max_iter=1, rtol=0.0, stag=0.0, warm_start=False, cycle="V"):
    """Solve the adjoint system (eq. adjointMGRIT) with MGRIT, the primal trajectory U
    fixed. Lam [N+1][...] holds the terminal value lam^N in row N; with warm_start
    the other rows are the initial guess, else the C-points kc (k < N/c) start as
    copies of lam^N. Stop rule as in mgrit_forward. Returns (Lam_out, res_hist, iterations)."""
    U, K, b = _f64(U, K, b)
    N = K.shape[0]
    sizes = level_sizes(N, cf, max_levels, min_coarse)
    H = _Hierarchy(sizes, cf, h)
    lam = np.array(Lam, dtype=_DT, copy=True)
    if not warm_start and len(sizes) > 1:
        for k in range(N // cf):
            lam[k * cf] = lam[N]
    g = np.zeros_like(lam)
    g[N] = lam[N]
    H.u[0], H.g[0] = lam, g
    hist = []
    it = 0
    for m in range(1, max_iter + 1):
        _adj_cycle(H, U, K, b, kind, relax, 0, hist, cycle)
        it = m
        if len(sizes) == 1:
            hist.append(0.0)
        if rtol > 0 and hist[-1] <= rtol * hist[0]:
            break
        if stag > 0 and m > 1 and hist[-1] > stag * hist[-2]:
            break
    return H.u[0], hist, it


# ---------------------------------------------------------------------------
# Simultaneous (one-shot) training, Algorithm 2 with m1 = m2 = 1 iterations and a
# scaled-identity Hessian approximation (plain gradient step with step size lr)
# ---------------------------------------------------------------------------

def one_shot(y, onehot, L_in, K, b, W, mu, h, kind, opening, cf, max_levels, min_coarse,
             relax, updates, lr, m1=1, m2=1, progress=None):
    """Algorithm 2: per design update, m1 state MGRIT iterations and m2 adjoint MGRIT
    iterations (both warm-started from the previous update's iterates), the reduced
    gradient with the inexact state and adjoint, then theta <- theta - lr * grad for
    K, b, L_in, W, mu. The loss J is evaluated on the state iterate used for the
    gradient. Returns the list of losses (one per update) and the final weights.
    progress (optional) is called as progress(update, J) after each update."""
    L_in, K, b, W, mu = (None if a is None else np.array(a, dtype=np.float64, copy=True)
                         for a in (L_in, K, b, W, mu))
    y, onehot = _f64(y, onehot)
    N = K.shape[0]
    u0 = open_forward(y, L_in, kind, opening)
    U = np.zeros((N + 1,) + u0.shape)
    U[0] = u0
    Lam = np.zeros_like(U)
    losses = []
    for it in range(updates):
        U[0] = open_forward(y, L_in, kind, opening)
        U, _, _ = mgrit_forward(U, K, b, h, kind, cf, max_levels, min_coarse, relax,
                                max_iter=m1, warm_start=(it > 0))
        J, lamN, dW, dmu = loss_terminal(U[N], W, mu, onehot)
        losses.append(J)
        Lam[N] = lamN
        Lam, _, _ = mgrit_adjoint(U, Lam, K, b, h, kind, cf, max_levels, min_coarse, relax,
                                  max_iter=m2, warm_start=(it > 0))
        dK, db = gradient(U, Lam, K, b, h, kind)
        dL = open_grad(y, L_in, Lam[0], kind, opening) if opening != "identity" else None
        K -= lr * dK
        b -= lr * db
        W -= lr * dW
        mu -= lr * dmu
        if dL is not None:
            L_in -= lr * dL
        if progress is not None:
            progress(it, J)
    return losses, dict(L_in=L_in, K=K, b=b, W=W, mu=mu)


def serial_training(y, onehot, L_in, K, b, W, mu, h, kind, opening, updates, lr, progress=None):
    """Layer-serial gradient descent on the same objective (the paper's baseline
    method): exact forward propagation, backpropagation and the same update.
    progress (optional) is called as progress(update, J) after each update."""
    L_in, K, b, W, mu = (None if a is None else np.array(a, dtype=np.float64, copy=True)
                         for a in (L_in, K, b, W, mu))
    y, onehot = _f64(y, onehot)
    N = K.shape[0]
    losses = []
    for it in range(updates):
        u0 = open_forward(y, L_in, kind, opening)
        U = serial_forward(u0, K, b, h, kind)
        J, lamN, dW, dmu = loss_terminal(U[N], W, mu, onehot)
        losses.append(J)
        Lam = serial_adjoint(U, lamN, K, b, h, kind)
        dK, db = gradient(U, Lam, K, b, h, kind)
        dL = open_grad(y, L_in, Lam[0], kind, opening) if opening != "identity" else None
        K -= lr * dK
        b -= lr * db
        W -= lr * dW
        mu -= lr * dmu
        if dL is not None:
            L_in -= lr * dL
        if progress is not None:
            progress(it, J)
    return losses, dict(L_in=L_in, K=K, b=b, W=W, mu=mu)


# ---------------------------------------------------------------------------
# Algorithm 2 in full: m1 state and m2 adjoint MGRIT iterations per design
# update, a limited-memory BFGS approximation of the Hessian, a backtracking line
# search on the objective, and a validation-accuracy stop (Section 4)
# ---------------------------------------------------------------------------

def _vdot(a, b):
    return float(sum(np.sum(x * y) for x, y in zip(a, b)))


def lbfgs_direction(g, pairs):
    """H g by the limited-memory BFGS two-loop recursion over the stored pairs
    (s_i, y_i), oldest first, with the initial matrix gamma I, gamma = s.y / y.y of
    the newest pair (1 without pairs). Vectors are lists of arrays."""
    q = [x.copy() for x in g]
    alphas = []
    for s_i, y_i in reversed(pairs):
        a = _vdot(s_i, q) / _vdot(y_i, s_i)
        alphas.append(a)
        q = [x - a * y for x, y in zip(q, y_i)]
    gamma = _vdot(pairs[-1][0], pairs[-1][1]) / _vdot(pairs[-1][1], pairs[-1][1]) if pairs else 1.0
    r = [gamma * x for x in q]
    for (s_i, y_i), a in zip(pairs, reversed(alphas)):
        beta = _vdot(y_i, r) / _vdot(y_i, s_i)
        r = [x + (a - beta) * s for x, s in zip(r, s_i)]
    return r


def strong_wolfe_search(phi, dphi, J, gd, alpha_start, c1, c2, max_ls):
    """A step length meeting the strong Wolfe conditions (Section 4 names them as
    one choice for the line search) by the textbook method: bracketing with step
    doubling, then zoom by bisection (Nocedal and Wright, Numerical Optimization,
    2nd ed., Algorithms 3.5 and 3.6, bisection as the interpolation).
    phi(a) -> (phi value, context), dphi(context) -> phi'(a); J = phi(0),
    gd = phi'(0) < 0. Conditions: phi(a) <= J + c1 a gd and |phi'(a)| <= c2 |gd|.
    At most max_ls evaluations of phi. Returns (alpha, phi evaluations, met): the
    first step found meeting both; else the lower end of the last bracket (the
    best step meeting sufficient decrease), or, if no step met it, the last one
    tried."""
    evals = [0]
    last = [alpha_start]

    def ev(a):
        evals[0] += 1
        last[0] = a
        return phi(a)

    def decrease(a, Ja):
        return Ja <= J + c1 * a * gd

    def zoom(lo, Jlo, hi):
        while evals[0] < max_ls:
            a = 0.5 * (lo + hi)
            Ja, ctx = ev(a)
            if not decrease(a, Ja) or Ja >= Jlo:
                hi = a
                continue
            da = dphi(ctx)
            if abs(da) <= c2 * abs(gd):
                return a, True
            if da * (hi - lo) >= 0.0:
                hi = lo
            lo, Jlo = a, Ja
        return lo, False

    prev_a, prev_J = 0.0, J
    a = alpha_start
    while True:
        Ja, ctx = ev(a)
        if not decrease(a, Ja) or (prev_a > 0.0 and Ja >= prev_J):
            res, met = zoom(prev_a, prev_J, a)
            break
        da = dphi(ctx)
        if abs(da) <= c2 * abs(gd):
            res, met = a, True
            break
        if da >= 0.0:
            res, met = zoom(a, Ja, prev_a)
            break
        if evals[0] >= max_ls:
            res, met = a, False
            break
        prev_a, prev_J = a, Ja
        a = 2.0 * a
    if res == 0.0:
        res = last[0]
    return res, evals[0], met


def one_shot_lbfgs(y, onehot, L_in, K, b, W, mu, h, kind, opening, cf, max_levels, min_coarse, relax,
                   updates, m1=2, m2=2, memory=5, alpha0=1e-2, c1=1e-4, shrink=0.5, max_ls=8,
                   y_val=None, onehot_val=None, target_acc=None, cycle="V", line_search="armijo", c2=0.9):
    """Algorithm 2 with its Hessian approximated by limited-memory BFGS. Per design
    update: m1 state and m2 adjoint MGRIT iterations, warm-started from the previous
    update's iterates (cold at the first); the reduced gradient g of J at those
    inexact iterates; the pair (s, y) = (design change, gradient change) is kept when
    s.y > 0 (at most `memory` pairs); the direction d = -H g (two-loop recursion);
    a backtracking line search: trial steps alpha = alpha_start * shrink^t, t < max_ls,
    the objective at a trial design being the loss of the state after m1 MGRIT
    iterations warm-started from the current state, accepted at the first trial with
    J_t <= J + c1 alpha g.d (the last trial is taken if none is); alpha_start is alpha0
    at the first update (no curvature yet) and 1 afterwards. The accepted trial's
    state becomes the current one. With validation data, the validation accuracy of
    the new design (its exact forward propagation) is taken after every update and the
    run stops once it reaches target_acc.
    line_search = "wolfe" replaces the backtracking by strong_wolfe_search, with
    phi(a) the trial loss above and phi'(a) = g_a.d, g_a the reduced gradient after
    m2 adjoint MGRIT iterations at the trial state warm-started from this update's
    adjoint iterate (the inexact gradient the one-shot method sees), starting from
    alpha_start; the accepted step's state is the state after m1 iterations at that
    design, as for every trial.
    Design vector order: L_in (unless the opening is the identity), K, b, W, mu.
    Returns dict(losses, alphas, trials, accuracies, weights, and with
    line_search = "wolfe" also wolfe: whether each accepted step met both
    conditions); trials counts the loss evaluations of each update."""
    L_in, K, b, W, mu = (None if a is None else np.array(a, dtype=np.float64, copy=True)
                         for a in (L_in, K, b, W, mu))
    y, onehot = _f64(y, onehot)
    N = K.shape[0]
    has_open = opening != "identity"
    sched = dict(cf=cf, max_levels=max_levels, min_coarse=min_coarse, relax=relax, cycle=cycle)

    def design():
        return ([L_in] if has_open else []) + [K, b, W, mu]

    def unpack(v):
        v = list(v)
        return (v.pop(0) if has_open else None), v[0], v[1], v[2], v[3]

    def state_after(Lt, Kt, bt, Ustart, warm):
        U = Ustart.copy()
        U[0] = open_forward(y, Lt, kind, opening)
        U, _, _ = mgrit_forward(U, Kt, bt, h, kind, max_iter=m1, warm_start=warm, **sched)
        return U

    u0 = open_forward(y, L_in, kind, opening)
    U = np.zeros((N + 1,) + u0.shape)
    Lam = np.zeros_like(U)
    pairs = []
    prev = None  # (design, gradient) of the previous update
    out = dict(losses=[], alphas=[], trials=[], accuracies=[])
    U = state_after(L_in, K, b, U, False)
    for it in range(updates):
        if it > 0:
            U = state_after(L_in, K, b, U, True)
        J, lamN, dW, dmu = loss_terminal(U[N], W, mu, onehot)
        Lam[N] = lamN
        Lam, _, _ = mgrit_adjoint(U, Lam, K, b, h, kind, max_iter=m2, warm_start=(it > 0), **sched)
        dK, db = gradient(U, Lam, K, b, h, kind)
        g = ([open_grad(y, L_in, Lam[0], kind, opening)] if has_open else []) + [dK, db, dW, dmu]
        x = design()
        if prev is not None:
            s_v = [a - c for a, c in zip(x, prev[0])]
            y_v = [a - c for a, c in zip(g, prev[1])]
            if _vdot(s_v, y_v) > 0.0:
                pairs.append((s_v, y_v))
                pairs = pairs[-memory:]
        d = [-v for v in lbfgs_direction(g, pairs)]
        gd = _vdot(g, d)
        alpha = alpha0 if it == 0 else 1.0
        if line_search == "wolfe":
            def phi(a):
                Lt, Kt, bt, Wt, mut = unpack([v + a * w for v, w in zip(x, d)])
                Ut = state_after(Lt, Kt, bt, U, True)
                Jt, lamNt, dWt, dmut = loss_terminal(Ut[N], Wt, mut, onehot)
                return Jt, (Lt, Kt, bt, Ut, lamNt, dWt, dmut)

            def dphi(ctx):
                # the reduced gradient at the trial state: m2 adjoint iterations warm-started
                # from this update's adjoint iterate
                Lt, Kt, bt, Ut, lamNt, dWt, dmut = ctx
                La = Lam.copy()
                La[N] = lamNt
                La, _, _ = mgrit_adjoint(Ut, La, Kt, bt, h, kind, max_iter=m2, warm_start=True, **sched)
                dKt, dbt = gradient(Ut, La, Kt, bt, h, kind)
                ga = ([open_grad(y, Lt, La[0], kind, opening)] if has_open else []) + [dKt, dbt, dWt, dmut]
                return _vdot(ga, d)

            alpha, t, met = strong_wolfe_search(phi, dphi, J, gd, alpha, c1, c2, max_ls)
            t -= 1  # trials below counts t + 1
            out.setdefault("wolfe", []).append(met)
            Lt, Kt, bt, Wt, mut = unpack([a + alpha * v for a, v in zip(x, d)])
            Ut = state_after(Lt, Kt, bt, U, True)
        else:
            for t in range(max_ls):
                Lt, Kt, bt, Wt, mut = unpack([a + alpha * v for a, v in zip(x, d)])
                Ut = state_after(Lt, Kt, bt, U, True)
                Jt = loss_terminal(Ut[N], Wt, mut, onehot)[0]
                if Jt <= J + c1 * alpha * gd or t == max_ls - 1:
                    break
                alpha *= shrink
        prev = (x, g)
        L_in, K, b, W, mu = Lt, Kt, bt, Wt, mut
        U = Ut
        out["losses"].append(J)
        out["alphas"].append(alpha)
        out["trials"].append(t + 1)
        if y_val is not None:
            uv = serial_forward(open_forward(_f64(y_val), L_in, kind, opening), K, b, h, kind)[N]
            acc = accuracy(uv, W, mu, np.argmax(_f64(onehot_val), axis=1))
            out["accuracies"].append(acc)
            if target_acc is not None and acc >= target_acc:
                break
    out["weights"] = dict(L_in=L_in, K=K, b=b, W=W, mu=mu)
    return out
