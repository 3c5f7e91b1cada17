"""Seeded synthetic workloads for the layer-parallel ResNet hot path.

This module only draws random numbers and lays them out. It holds none of the
method's arithmetic (no layer step, no activation, no loss), so both the CPU
oracle and the GPU path can consume its output without sharing any code of the
method. Both sides receive exactly the same values: everything is drawn in fp64
with ``numpy.random.default_rng`` (PCG64) and then rounded to the workload's
dtype; the oracle upcasts the rounded values back to fp64.

Draw order (fixed, so a seed names one input set):
  data generator  (seed 1000 + cfg): class structure, labels, features
  weight generator (seed 2000 + cfg): L_in, K_0 .. K_{N-1}, b, W, mu

The workloads stand in for the paper's test cases (Section 5.1: Peaks,
Indian Pines, MNIST), whose data and level-set function are not available;
shapes, widths, depths, step sizes and activations follow the paper where it
fixes them, the rest follows the workload descriptions below.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional

import numpy as np

# Activation and layer kinds are names shared by both sides as plain strings.
TANH, RELU, SMOOTHRELU, IDENTITY = "tanh", "relu", "smoothrelu", "identity"
DENSE, CONV = "dense", "conv3x3"


@dataclasses.dataclass(frozen=True)
class Workload:
    cfg: int
    name: str
    dtype: str            # "f32" or "f64"
    layer: str            # DENSE or CONV
    act: str              # activation of the residual layers
    N: int                # number of residual layers
    B: int                # batch size
    C: int                # width (dense) or channel count (conv)
    H: int                # 1 for dense
    W: int                # 1 for dense
    T: float              # final time; h = T / N
    n_features: int       # input feature count (conv: pixels of the 1-channel image)
    n_classes: int
    opening: str          # "dense_act", "conv_act" or "identity"
    # MGRIT schedule
    cf: int = 4
    max_levels: int = 2
    min_coarse: int = 1
    relax: str = "FCF"    # "F", "FCF" or "FCFCF"
    cycle: str = "V"      # "V" or "F"
    fwd_iters: int = 2
    adj_iters: int = 2
    rtol: float = 0.0
    stag: float = 0.0     # stop when rho_m > stag * rho_{m-1} (0: off)

    @property
    def h(self) -> float:
        return self.T / self.N

    @property
    def q(self) -> int:
        return self.C * self.H * self.W

    @property
    def np_dtype(self):
        return np.float32 if self.dtype == "f32" else np.float64

    def with_overrides(self, **kw) -> "Workload":
        """Same workload family at another size (for parity tests). ``T`` is
        kept, so h = T/N follows N."""
        return dataclasses.replace(self, **kw)


# Workload table. Sizes, activations and schedules of the synthetic stand-ins.
WORKLOADS = {
    1: Workload(cfg=1, name="tiny dense tanh fp64 (q=8, N=32, B=512)", dtype="f64",
                layer=DENSE, act=TANH, N=32, B=512, C=8, H=1, W=1, T=5.0,
                n_features=2, n_classes=5, opening="dense_act",
                cf=4, max_levels=2, relax="FCF", fwd_iters=5, adj_iters=5),
    2: Workload(cfg=2, name="dense relu fp32 (q=32, N=256, B=4096)", dtype="f32",
                layer=DENSE, act=RELU, N=256, B=4096, C=32, H=1, W=1, T=10.0,
                n_features=220, n_classes=16, opening="dense_act",
                cf=4, max_levels=3, relax="FCF", fwd_iters=2, adj_iters=2),
    3: Workload(cfg=3, name="deep dense tanh fp32 (q=64, N=2048, B=16384)", dtype="f32",
                layer=DENSE, act=TANH, N=2048, B=16384, C=64, H=1, W=1, T=8.0,
                n_features=64, n_classes=10, opening="identity",
                cf=4, max_levels=16, min_coarse=8, relax="FCF",
                fwd_iters=20, adj_iters=20, rtol=1e-8, stag=0.9),
    4: Workload(cfg=4, name="conv3x3 relu fp32 (C=8, 28x28, N=512, B=1024)", dtype="f32",
                layer=CONV, act=RELU, N=512, B=1024, C=8, H=28, W=28, T=5.0,
                n_features=784, n_classes=10, opening="conv_act",
                cf=4, max_levels=4, relax="FCF", fwd_iters=2, adj_iters=2),
    5: Workload(cfg=5, name="one-shot dense tanh fp32 (q=32, N=1024, B=16384)", dtype="f32",
                layer=DENSE, act=TANH, N=1024, B=16384, C=32, H=1, W=1, T=10.0,
                n_features=128, n_classes=10, opening="dense_act",
                cf=4, max_levels=3, relax="FCF", fwd_iters=1, adj_iters=1),
    # The Peaks network of Section 5.1 at its largest depth (width 8, smoothed ReLU,
    # T = 5, N = 2048, batch 5000 as in Section 5.2), solved as there until the
    # relative residual has dropped by five orders of magnitude.
    6: Workload(cfg=6, name="Peaks-shaped dense smoothed ReLU fp64 (q=8, N=2048, B=5000)", dtype="f64",
                layer=DENSE, act=SMOOTHRELU, N=2048, B=5000, C=8, H=1, W=1, T=5.0,
                n_features=2, n_classes=5, opening="dense_act",
                cf=4, max_levels=16, min_coarse=8, relax="FCF", fwd_iters=20, adj_iters=20, rtol=1e-5),
    # The hyperspectral network of Section 5.1 (width 220 = the spectral bands,
    # identity opening, smoothed ReLU, 16 classes, T = 20) at its largest depth,
    # N = 2048, with the batch of Section 5.2 (1000 pixels), solved to a relative
    # residual drop of five orders of magnitude; fp32 so that the layer products
    # run on the matrix cores.
    7: Workload(cfg=7, name="hyperspectral-shaped dense smoothed ReLU fp32 (q=220, N=2048, B=1000)", dtype="f32",
                layer=DENSE, act=SMOOTHRELU, N=2048, B=1000, C=220, H=1, W=1, T=20.0,
                n_features=220, n_classes=16, opening="identity",
                cf=4, max_levels=16, min_coarse=8, relax="FCF", fwd_iters=20, adj_iters=20, rtol=1e-5),
}

ONE_SHOT_UPDATES = 100
ONE_SHOT_LR = 1e-2


def _kaiming(rng, shape, fan_in, scale):
    return rng.standard_normal(shape) * (math.sqrt(2.0 / fan_in) * scale)


def _normal(rng, shape, std):
    return rng.standard_normal(shape) * std


def generate(wl: Workload, data_seed: Optional[int] = None,
             weight_seed: Optional[int] = None) -> dict:
    """Draw the inputs of one workload. Returns a dict of numpy arrays, each
    already rounded to the workload dtype (and stored in that dtype):

      y      [B][n_features]  (conv: [B][1][H][W])
      labels [B]   int64 class index
      onehot [B][n_classes]
      L_in   [q][n_features]  (conv: [C][1][3][3]; identity opening: None)
      K      [N][q][q]        (conv: [N][C][C][3][3]); K[n][i][j] maps input j to output i
      b      [N][q]           (conv: [N][C])
      W      [n_classes][q]
      mu     [n_classes]
    """
    ds = 1000 + wl.cfg if data_seed is None else data_seed
    wsd = 2000 + wl.cfg if weight_seed is None else weight_seed
    rd = np.random.default_rng(ds)
    rw = np.random.default_rng(wsd)
    B, N, q, C = wl.B, wl.N, wl.q, wl.C
    nc = wl.n_classes

    # ---- data ----
    if wl.cfg in (1, 6):
        y = rd.uniform(-3.0, 3.0, size=(B, 2))
        A = rd.standard_normal((nc, 2))
        a = rd.standard_normal(nc)
        labels = np.argmax(y @ A.T + a, axis=1)
    elif wl.cfg in (2, 5):
        sigma = 0.5 if wl.cfg == 2 else 0.7
        means = rd.standard_normal((nc, wl.n_features))
        labels = rd.integers(0, nc, size=B)
        y = means[labels] + sigma * rd.standard_normal((B, wl.n_features))
    elif wl.cfg == 3:
        y = rd.standard_normal((B, wl.n_features))
        labels = rd.integers(0, nc, size=B)
    elif wl.cfg == 7:
        # per class a smooth spectrum (three Gaussian bumps over the bands); each
        # pixel scales its class spectrum by a brightness in [0.8, 1.2] and adds noise
        bands = np.arange(wl.n_features, dtype=np.float64)
        centers = rd.uniform(0.0, wl.n_features, size=(nc, 3, 1))
        widths = rd.uniform(10.0, 40.0, size=(nc, 3, 1))
        amps = rd.uniform(0.3, 1.0, size=(nc, 3, 1))
        means = np.sum(amps * np.exp(-((bands - centers) / widths) ** 2), axis=1)
        labels = rd.integers(0, nc, size=B)
        y = means[labels] * rd.uniform(0.8, 1.2, size=(B, 1)) + 0.05 * rd.standard_normal((B, wl.n_features))
    elif wl.cfg == 4:
        patterns = rd.uniform(0.0, 1.0, size=(nc, 5, 5))
        offsets = np.stack([rd.integers(0, wl.H - 4, size=nc), rd.integers(0, wl.W - 4, size=nc)], axis=1) \
            if (wl.H, wl.W) != (28, 28) else rd.integers(0, 24, size=(nc, 2))
        labels = rd.integers(0, nc, size=B)
        y = rd.uniform(0.0, 1.0, size=(B, 1, wl.H, wl.W))
        for k in range(nc):
            sel = labels == k
            oy, ox = offsets[k]
            y[sel, 0, oy:oy + 5, ox:ox + 5] += patterns[k]
    else:
        raise ValueError(f"unknown workload {wl.cfg}")
    onehot = np.zeros((B, nc))
    onehot[np.arange(B), labels] = 1.0

    # ---- weights ----
    if wl.cfg == 1:
        L_in = _normal(rw, (q, wl.n_features), 0.1)
        K = _normal(rw, (N, q, q), 0.1)
        b = np.zeros((N, q))
        W = _normal(rw, (nc, q), 0.1)
    elif wl.cfg in (2, 5):
        L_in = _kaiming(rw, (q, wl.n_features), wl.n_features, 0.1)
        K = _kaiming(rw, (N, q, q), q, 0.1)
        b = np.zeros((N, q))
        W = _kaiming(rw, (nc, q), q, 0.1)
    elif wl.cfg == 3:
        L_in = None
        K = _normal(rw, (N, q, q), 0.05)
        b = _normal(rw, (N, q), 0.01)
        W = _normal(rw, (nc, q), 0.05)
    elif wl.cfg == 6:
        L_in = _normal(rw, (q, wl.n_features), 0.5)
        K = _normal(rw, (N, q, q), 0.3)
        b = _normal(rw, (N, q), 0.05)
        W = _normal(rw, (nc, q), 0.5)
    elif wl.cfg == 7:
        L_in = None
        K = _normal(rw, (N, q, q), 0.003)
        b = _normal(rw, (N, q), 0.01)
        W = _normal(rw, (nc, q), 0.1)
    elif wl.cfg == 4:
        L_in = _kaiming(rw, (C, 1, 3, 3), 9, 0.1)
        K = _kaiming(rw, (N, C, C, 3, 3), 9 * C, 0.1)
        b = np.zeros((N, C))
        W = _kaiming(rw, (nc, q), q, 0.1)
    mu = np.zeros(nc)

    dt = wl.np_dtype
    out = dict(y=y, labels=labels.astype(np.int64), onehot=onehot, L_in=L_in,
               K=K, b=b, W=W, mu=mu)
    for k, v in list(out.items()):
        if v is not None and k != "labels":
            out[k] = np.ascontiguousarray(v.astype(dt))
    return out


def random_state(wl: Workload, seed: int, scale: float = 1.0, rows: int = 1) -> np.ndarray:
    """A seeded random array of ``rows`` state slices [rows][B][q] (conv:
    [rows][B][C][H][W]) in the workload dtype: used as an initial state, a
    terminal adjoint or a perturbation in tests."""
    r = np.random.default_rng(seed)
    shape = (rows, wl.B, wl.C, wl.H, wl.W) if wl.layer == CONV else (rows, wl.B, wl.q)
    return np.ascontiguousarray((scale * r.standard_normal(shape)).astype(wl.np_dtype))
