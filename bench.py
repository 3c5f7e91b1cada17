"""Benchmark of the layer-parallel ResNet hot path on one MI355X.

One step = one gradient evaluation of the workload with MGRIT: the workload's
number of forward MGRIT iterations (cold start), the loss and adjoint terminal
value, the adjoint MGRIT iterations, and the reduced gradient, all through the
C ABI on the current stream, with every input resident in HBM. The metric is
layer-steps x examples per second per MGRIT forward+adjoint iteration:

    value = N * B * (iterations per step) / (seconds per step)

where "iterations per step" counts forward+adjoint iteration pairs; the
gradient's cost is included in the step time. The dominant kernel (largest
summed time in a traced warm-up step) is timed live with HIP events recorded by
the library on the launch stream over the timed steps, and compared with its
algorithmic bytes or flops (the model below) to give the roofline fraction.

The default run measures the deep dense workload (N = 2048, B = 16384, width 64),
the largest dense configuration, and then the convolutional workload, whose line
goes under "extra" with its own roofline; the CPU oracle baseline is the deep
workload's.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--config 3] [--extra 4 ...] [--no-cpu]
                       [--relax F|FCF|FCFCF] [--cycle V|F] [--cf C] [--no-record]
       python bench.py --updates 100     (one-shot and layer-serial loss curves of the one-shot workload)
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
PEAK_TFLOPS = {"f32": 157.3, "f64": 78.6}  # dense MFMA / fp32 vector (packed), fp64

# dense fp32 widths the library runs on the matrix cores (the others on the vector ALUs)
MATRIX_CORE_WIDTHS = (32, 64, 220)

KIND_NAMES = ["fwd_fc", "fwd_fres", "fwd_corrf", "fwd_coarsest", "adj_fc", "adj_fres", "adj_corrf",
              "adj_coarsest", "gradient", "residual", "serial"]


def level_sizes(N, cf, max_levels, min_coarse):
    sizes = [N]
    while len(sizes) < max_levels and sizes[-1] > min_coarse:
        sizes.append(sizes[-1] // cf)
    return sizes


def level_visits(L: int, cycle: str):
    """Times each level is visited by one cycle from the finest level: a V-cycle
    visits every level once; an F-cycle solves each coarse problem with an F-cycle
    and then a V-cycle (the V-cycle left out above the coarsest level)."""
    v = [0] * L

    def go(l, cyc):
        v[l] += 1
        if l == L - 1:
            return
        go(l + 1, "F" if cyc == "F" else "V")
        if cyc == "F" and l + 2 < L:
            go(l + 1, "V")

    go(0, cycle)
    return v


def record_bytes(wl) -> float:
    """Bytes per value of the sigma' record the step keeps (0: none is kept): ReLU
    one bit per value (one byte at width 220), fp32 otherwise."""
    if wl.dtype != "f32" or wl.act == "identity" or (wl.layer == "dense" and wl.q not in MATRIX_CORE_WIDTHS):
        return 0
    if wl.act == "relu":
        return 1 if wl.layer == "dense" and wl.q == 220 else 0.125
    return 4


def kernel_model(wl, kind: str, fwd_iters: int, adj_iters: int, rec: int = 0, cpt: bool = False):
    """Algorithmic HBM bytes and flops of every launch of one kernel kind in one
    step (summed over MGRIT levels and iterations), and the launch count.

    Per interval and example (q features, e bytes per value, c = cf), on level l
    (G rows exist on coarse levels only):
      fwd FC:    read C-point + c G rows, write 1 staged C-point;      c * 2q^2 flops
      fwd FRES:  read 2 C-points + c G rows, write G' and X' (1/c);    c * 2q^2
      fwd CORRF: read C-point + coarse value + (c-1) G rows, write c;  (c-1) * 2q^2
      adjoint:   the same, plus one primal row per step, 4q^2 flops per step,
                 and one extra transposed product (2q^2) in FRES for the coarse step
      coarsest:  read 1 + N_L G rows (+ N_L primal rows), write N_L rows
      gradient:  per layer read U[n], Lam[n+1] and K_n, write dK, db;  4q^2 per layer
    Each launch also reads the weights of its level once: N_l (q^2 + q) values.
    With a sigma' record of rec bytes per value (rrow per example row), the
    adjoint reads one record row per step instead of a primal row and skips the
    forward product (2q^2 flops per step), the gradient (width 64, width 32 with
    ReLU's bit record, convolution) reads the record instead of K_n and takes no
    forward product, and the final finest CORRF writes c record rows per interval
    and takes one more product.
    With C-point storage (cpt) the finest adjoint sweeps read one primal row (the
    lower C-point) per interval and recompute the interval's states with c forward
    products; the finest forward CORRF only corrects the C-points (read 2, write 1,
    no products); the gradient reads the C-points, writes and reads back the
    recomputed states of every layer ((c-1)/c N forward products), and reads Lam."""
    q, B, c = wl.q, wl.B, wl.cf
    e = 4 if wl.dtype == "f32" else 8
    row = B * q * e
    sizes = level_sizes(wl.N, c, wl.max_levels, wl.min_coarse)
    L = len(sizes)
    fcf = wl.relax != "F"
    nfc = {"F": 0, "FCF": 1, "FCFCF": 2}[wl.relax]  # FC sweeps per relaxation
    visits = level_visits(L, wl.cycle)
    adj = kind.startswith("adj")
    iters = adj_iters if adj else fwd_iters
    # multiply-adds of one layer product K v per example: q^2 dense, 9 C^2 H W conv
    mac = q * q if wl.layer == "dense" else 9 * wl.C * wl.C * wl.H * wl.W
    nweights = (q * q + q) if wl.layer == "dense" else (9 * wl.C * wl.C + wl.C)
    rrow = B * q * rec
    # the adjoint's per-step traffic in primal rows, and its flops per step
    arow = (rrow / row) if rec else 1.0
    fstep = (2 if adj and rec else 4 if adj else 2) * mac
    byts = flops = launches = 0
    if kind == "gradient" and cpt:
        return ((wl.N // c + 3 * wl.N) * row + 3 * wl.N * nweights * e,
                (4.0 + 2.0 * (c - 1) / c) * mac * B * wl.N, 1)
    if kind == "gradient":
        # the dense width-32 kernel recomputes sigma' for smooth activations
        if rec and (wl.layer != "dense" or q >= 64 or wl.act == "relu"):
            # (with the record, the dense kernels stage no weights)
            return 2 * wl.N * row + wl.N * rrow + (wl.N * nweights * e if wl.layer != "dense" else 0), \
                2.0 * mac * B * wl.N, 1
        return 2 * wl.N * row + 2 * wl.N * nweights * e, 4.0 * mac * B * wl.N, 1
    # With FCF the finest level's correction is applied inside the next cycle's FC
    # sweep (one more row read per interval from the second cycle on) and its
    # correction + F-relaxation sweep runs once per solve.
    for m in range(iters):
        for l, Nl in enumerate(sizes):
            wbytes = Nl * nweights * e
            g = 1 if l >= 1 else 0
            nv = visits[l]
            if l == L - 1:
                if kind.endswith("coarsest"):
                    byts += nv * ((1 + g * Nl + Nl + (Nl * arow if adj else 0)) * row + wbytes)
                    flops += nv * Nl * fstep * B
                    launches += nv
                continue
            Nc = Nl // c
            xn = (1.0 / c) if (l + 1 < L - 1) else 0.0
            deferred = l == 0 and fcf
            # primal rows the adjoint reads per interval, and the extra recompute products
            prow = (1.0 if cpt and l == 0 else c * arow) if adj else 0.0
            if kind.endswith("_corrf") and cpt and l == 0 and not adj:
                if not deferred or m == iters - 1:
                    byts += nv * Nc * 3 * row
                    launches += nv
                continue
            if kind.endswith("_fc") and fcf:
                # the first FC sweep reads the pending correction on the finest level
                # from the second cycle on; a second one (FCFCF) reads staged C-points
                first = Nc * (2 + g * c + prow + (1 if deferred and m > 0 else 0)) * row
                again = Nc * (2 + g * c + prow) * row
                byts += nv * (first + (nfc - 1) * again + nfc * wbytes)
                flops += nv * nfc * Nc * c * fstep * B
                launches += nv * nfc
            elif kind.endswith("_fres"):
                byts += nv * (Nc * (3 + xn + g * c + prow) * row + wbytes)
                flops += nv * Nc * (c * fstep + (2 * mac if adj else 0)) * B
                launches += nv
            elif kind.endswith("_corrf") and (not deferred or m == iters - 1):
                byts += nv * (Nc * (2 + c + g * (c - 1) + ((1.0 if cpt and l == 0 else (c - 1) * arow)
                                                           if adj else 0)) * row + wbytes)
                flops += nv * Nc * (c - 1) * fstep * B
                if cpt and adj and l == 0:
                    flops += nv * Nc * 2 * mac * B  # the recompute also needs the interval's first product
                if rec and not adj and l == 0:
                    # the final finest sweep keeps the record of all c layers
                    byts += Nc * c * rrow
                    flops += Nc * 2 * mac * B
                launches += nv
    return byts, flops, launches


# Source files that define each kernel family (besides the shared headers).
_FAMILY_SOURCES = {
    "lp::conv::": ["lp_conv.hip"],
    "lp::mfma::": ["lp_dense_mfma.hip"],
    "lp::dense::": ["lp_dense_impl.h", "lp_dense_f32.hip", "lp_dense_f64.hip"],
    "lp::wide::": ["lp_dense_wide.hip"],
}
_SHARED_SOURCES = ["lp_internal.h", "lp_device.h"]


def source_hash(kernels: str = "") -> str:
    """Hash of the sources of the kernel family named in `kernels` (all sources if
    it names none), so a counter summary goes stale only when its kernels change."""
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_1812_04352_amd", "csrc")
    fams = [f for ns, fs in _FAMILY_SOURCES.items() if ns in kernels for f in fs]
    files = sorted(set(fams + _SHARED_SOURCES)) if fams else sorted(os.listdir(csrc))
    for f in files:
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(f.encode() + fh.read())
    return h.hexdigest()[:16]


def measured_traffic(kernel: str, workload: str):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if it was
    taken on the current kernel sources (else None)."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    try:
        rec = json.load(open(path))
    except (OSError, ValueError):
        return None
    ent = rec.get(workload, {}).get(kernel)
    if not ent or ent.get("source_hash") != source_hash(ent.get("kernel", "")):
        return None
    return ent.get("bytes_per_launch")


def kernel_kind(name: str):
    """Trace kind of a library kernel from its (demangled) name, or None."""
    import re
    if "k_grad<" in name or "k_grad_partial<" in name:
        return "gradient"
    m = re.search(r"lp::(mfma|conv|dense|wide)::k_(fwd|adj)(_sweep|_serial|_iv)?<([^>]*)>", name)
    if not m:
        return None
    fam, d, suffix, targs = m.groups()
    args = [t.strip() for t in targs.split(",")]
    if suffix == "_serial":
        mode = 3
    else:
        mode = int(args[{"mfma": 1, "conv": 0, "dense": 2, "wide": 1}[fam]])
    return f"{d}_" + ["fc", "fres", "corrf", "coarsest"][mode]


def summarize_traffic(workload: str, fetch_dir: str, write_dir: str, copy_fetch_dir: str, copy_write_dir: str):
    """HBM bytes per launch of every traced kernel kind from two rocprofv3 --pmc
    runs of the benchmark (FETCH_SIZE, then WRITE_SIZE, KiB per dispatch), each
    scaled by what the same counter reads for a plain copy of known size (two
    more runs with --copy-calibration). Writes the entries of `workload` into
    profiles/traffic.json with the current kernel source hash and prints the
    table as markdown."""
    import collections
    import csv

    def load(d):
        per = collections.defaultdict(list)
        for r in csv.DictReader(open(os.path.join(d, "run_counter_collection.csv"))):
            per[r["Kernel_Name"]].append(float(r["Counter_Value"]))
        return per

    f, w, cf, cw = load(fetch_dir), load(write_dir), load(copy_fetch_dir), load(copy_write_dir)
    copy = [k for k in cf if "copyBuffer" in k or "copy" in k.lower()]
    if not copy:
        raise SystemExit("no copy kernel in the calibration runs")
    ck = max(copy, key=lambda k: sum(cf[k]))
    true_bytes = float(1 << 30)
    f_scale = true_bytes / (sum(cf[ck]) / len(cf[ck]) * 1024.0)
    w_scale = true_bytes / (sum(cw[ck]) / len(cw[ck]) * 1024.0)
    path = os.path.join(ROOT, "profiles", "traffic.json")
    rec = json.load(open(path)) if os.path.exists(path) else {}
    ent = {}
    print(f"Calibration: a plain copy of 1 GiB (`{ck}`, {len(cf[ck])} launches) reads FETCH_SIZE = "
          f"{sum(cf[ck]) / len(cf[ck]):.0f} KiB and WRITE_SIZE = {sum(cw[ck]) / len(cw[ck]):.0f} KiB per launch, "
          f"so true bytes = FETCH_SIZE x {f_scale:.3f} KiB and WRITE_SIZE x {w_scale:.3f} KiB.\n")
    print("| kind | kernel | launches | FETCH_SIZE KiB/launch | WRITE_SIZE KiB/launch | HBM MB/launch |")
    print("|---|---|---:|---:|---:|---:|")
    by_kind = collections.defaultdict(lambda: [0, 0.0, 0.0, []])
    for k in f:
        kind = kernel_kind(k)
        if kind is None or k not in w:
            continue
        b = by_kind[kind]
        b[0] += len(f[k])
        b[1] += sum(f[k])
        b[2] += sum(w[k])
        b[3].append(k)
    for kind, (n, fs, ws, names) in sorted(by_kind.items(), key=lambda t: -(t[1][1] + t[1][2])):
        fk, wk = fs / n, ws / n
        byts = (fk * f_scale + wk * w_scale) * 1024.0
        kn = " / ".join(names)
        ent[kind] = {"bytes_per_launch": byts, "source_hash": source_hash(kn), "kernel": kn}
        print(f"| {kind} | `{' / '.join(names)}` | {n} | {fk:.0f} | {wk:.0f} | {byts / 1e6:.1f} |")
    rec[workload] = ent
    with open(path, "w") as fh:
        json.dump(rec, fh, indent=1)
        fh.write("\n")


def cpu_sample_size(wl) -> int:
    """Examples the CPU oracle baseline runs on: the full batch of the small dense
    workloads, fixed leading slices of the large ones (examples are independent
    in every solve, so the rate per example carries over)."""
    if wl.layer == "conv3x3":
        return min(wl.B, 8)  # one MGRIT iteration pair over 8 examples takes about 14 s
    if wl.q > 64:
        return min(wl.B, 64)
    if wl.cfg in (1, 2, 5):
        return wl.B
    return min(wl.B, 1024)


def cpu_baseline(wl, budget_s: float = 12.0):
    """The oracle timed on the host cores, in the workload's own dtype, on a
    bounded sample of the batch (cpu_sample_size), two legs, each repeated until
    about budget_s / 2 seconds have passed:
      MGRIT: one forward and one adjoint MGRIT iteration with the GPU's schedule
             (the same metric as the GPU line, which is `value`);
      layer-serial: forward propagation, backpropagation and the gradient (the
             paper's baseline method), as layer-steps x examples per second of
             one forward + backward pass."""
    import numpy as np

    import oracle as O
    from workloads import generate
    try:
        from threadpoolctl import threadpool_info, threadpool_limits
    except ImportError:  # pragma: no cover
        threadpool_info = threadpool_limits = None
    ncores = len(os.sched_getaffinity(0))
    Bs = cpu_sample_size(wl)
    d = generate(wl.with_overrides(B=Bs))
    ctx = threadpool_limits(ncores) if threadpool_limits else None
    dt = np.float32 if wl.dtype == "f32" else np.float64
    try:
        with O.working_precision(dt):
            u0 = O.open_forward(d["y"], d["L_in"], wl.act, wl.opening)
            U = np.zeros((wl.N + 1,) + u0.shape, dtype=dt)
            U[0] = u0
            args = dict(cf=wl.cf, max_levels=wl.max_levels, min_coarse=wl.min_coarse, relax=wl.relax, max_iter=1,
                        cycle=wl.cycle)
            t0 = time.perf_counter()
            reps = 0
            while True:
                Uo, _, _ = O.mgrit_forward(U, d["K"], d["b"], wl.h, wl.act, **args)
                lamN = O.loss_terminal(Uo[-1], d["W"], d["mu"], d["onehot"])[1]
                Lam = np.zeros_like(Uo)
                Lam[-1] = lamN
                O.mgrit_adjoint(Uo, Lam, d["K"], d["b"], wl.h, wl.act, **args)
                reps += 1
                if time.perf_counter() - t0 >= budget_s / 2:
                    break
            t_mg = time.perf_counter() - t0
            t0 = time.perf_counter()
            reps_s = 0
            while True:
                Us = O.serial_forward(u0, d["K"], d["b"], wl.h, wl.act)
                lamN = O.loss_terminal(Us[-1], d["W"], d["mu"], d["onehot"])[1]
                Ls = O.serial_adjoint(Us, lamN, d["K"], d["b"], wl.h, wl.act)
                O.gradient(Us, Ls, d["K"], d["b"], wl.h, wl.act)
                reps_s += 1
                if time.perf_counter() - t0 >= budget_s / 2:
                    break
            t_se = time.perf_counter() - t0
            assert Us.dtype == dt and Ls.dtype == dt
        threads = ncores
        if threadpool_info:
            th = [i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"]
            threads = max(th) if th else 1
    finally:
        if ctx is not None:
            ctx.__exit__(None, None, None)
    levels = len(level_sizes(wl.N, wl.cf, wl.max_levels, wl.min_coarse))
    sample = "full batch" if Bs == wl.B else f"first {Bs} of {wl.B} examples"
    return {"value": wl.N * Bs * reps / t_mg, "unit": "layer-steps*examples/s", "cores": threads, "kind": "oracle",
            "sample": f"{sample}, {reps} x (1 forward + 1 adjoint MGRIT iteration, {wl.relax}, {levels} levels), "
                      f"NumPy in {wl.dtype}, {t_mg:.1f} s",
            "layer_serial": {"value": wl.N * Bs * reps_s / t_se, "unit": "layer-steps*examples/s",
                             "sample": f"{sample}, {reps_s} x (forward propagation + backpropagation + gradient), "
                                       f"NumPy in {wl.dtype}, {t_se:.1f} s"}}


def note(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def measure(wl, steps: int, warmup: int, no_record: bool = False, storage: str = "all"):
    """Time `steps` benchmark steps of one workload on the GPU (after `warmup`
    untimed ones) and return its result line: value, ms per step, the dominant
    kernel's live roofline and the per-kind times of a traced warm-up step.
    storage "cpoints": the primal trajectory keeps the C-points only (no record;
    the adjoint and the gradient recompute the F-point states)."""
    import numpy as np
    import torch

    from paper_1812_04352_amd import lp as L
    from workloads import generate

    torch.cuda.set_device(0)
    torch.cuda.reset_peak_memory_stats()
    dt = torch.float32 if wl.dtype == "f32" else torch.float64
    d = generate(wl)
    cpt = storage == "cpoints"

    def g(x):
        return torch.from_numpy(np.ascontiguousarray(x)).to(device="cuda", dtype=dt)

    K, b, W, mu, y, c = (g(d[k]) for k in ("K", "b", "W", "mu", "y", "onehot"))
    Lin = g(d["L_in"]) if d["L_in"] is not None else None
    p = L.problem(wl.dtype, wl.layer, wl.act, wl.N, wl.B, wl.C, wl.H, wl.W, wl.h)
    U = torch.zeros(((wl.N // wl.cf if cpt else wl.N) + 1, wl.B, wl.q), device="cuda", dtype=dt)
    L.lp_open_forward(p, L.OPENING[wl.opening], wl.n_features, y, Lin, U[0])
    Lam = torch.zeros((wl.N + 1, wl.B, wl.q), device="cuda", dtype=dt)
    J = torch.zeros(1, device="cuda", dtype=torch.float64)
    dW, dmu = torch.empty_like(W), torch.empty_like(mu)
    dK, db = torch.empty_like(K), torch.empty_like(b)

    note(f"cfg{wl.cfg} inputs on the GPU")
    # the forward's final sweep keeps sigma'(z) for the adjoint and the gradient
    rec_e = 0 if (no_record or cpt) else record_bytes(wl)
    rec = L.alloc_dsig(p) if rec_e else None
    # iteration counts: fixed by the workload, or found once with its stop rule
    fwd_iters, adj_iters = wl.fwd_iters, wl.adj_iters
    if wl.rtol > 0 or wl.stag > 0:
        mg = L.mgrit(wl.cf, wl.max_levels, wl.min_coarse, wl.relax, wl.fwd_iters, False, wl.rtol, wl.stag,
                     wl.cycle, storage)
        ws = L.alloc_workspace(p, mg)
        fwd_iters, _ = L.lp_mgrit_forward(p, mg, K, b, U, ws, dsig=rec)
        L.lp_loss_terminal(p, wl.n_classes, U[-1], W, mu, c, J, Lam[-1], dW, dmu, ws)
        adj_iters, _ = L.lp_mgrit_adjoint(p, L.mgrit(wl.cf, wl.max_levels, wl.min_coarse, wl.relax,
                                                     wl.adj_iters, False, wl.rtol, wl.stag, wl.cycle, storage), K, b,
                                          U, Lam, ws, dsig=rec)
        del ws
    mgF = L.mgrit(wl.cf, wl.max_levels, wl.min_coarse, wl.relax, fwd_iters, cycle=wl.cycle, storage=storage)
    mgA = L.mgrit(wl.cf, wl.max_levels, wl.min_coarse, wl.relax, adj_iters, cycle=wl.cycle, storage=storage)
    ws = L.alloc_workspace(p, mgF if fwd_iters >= adj_iters else mgA)
    hist = {}

    def step(history=False):
        # the residual histories are read back (a host round trip) only when asked
        _, hf = L.lp_mgrit_forward(p, mgF, K, b, U, ws, history=history, dsig=rec)
        L.lp_loss_terminal(p, wl.n_classes, U[-1], W, mu, c, J, Lam[-1], dW, dmu, ws)
        _, ha = L.lp_mgrit_adjoint(p, mgA, K, b, U, Lam, ws, history=history, dsig=rec)
        if cpt:
            L.lp_gradient_cpoints(p, wl.cf, K, b, U, Lam, dK, db, ws)
        else:
            L.lp_gradient(p, K, b, U, Lam, dK, db, ws, dsig=rec)
        if history:
            hist["fwd"], hist["adj"] = hf, ha

    note(f"iterations fwd={fwd_iters} adj={adj_iters}; warm-up")
    # warm-up; the second step is traced for every kind to find the dominant kernel
    # (the first one also pays for loading the code objects)
    lib = L.load()
    step(history=True)
    torch.cuda.synchronize()
    lib.lp_trace_enable((1 << 11) - 1)
    step()
    torch.cuda.synchronize()
    per_kind = {}
    for k, name in enumerate(KIND_NAMES):
        n, ms = ctypes_read(lib, k)
        if n:
            per_kind[name] = ms
    dominant = max(per_kind, key=per_kind.get)
    lib.lp_trace_enable(0)
    for _ in range(max(0, warmup - 2)):
        step()
    torch.cuda.synchronize()

    note(f"timed region: {steps} steps, dominant kernel {dominant}")
    # timed region: only the dominant kind is traced
    lib.lp_trace_enable(1 << KIND_NAMES.index(dominant))
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    nl, kms = ctypes_read(lib, KIND_NAMES.index(dominant))
    lib.lp_trace_enable(0)
    # the timed solves read nothing back: a non-finite residual norm shows up here
    L.lp_check_finite()
    ms_step = (t1 - t0) * 1000.0 / steps
    pairs = 0.5 * (fwd_iters + adj_iters)
    value = wl.N * wl.B * pairs / (ms_step / 1000.0)

    peak_gb = torch.cuda.max_memory_allocated() / 1e9
    # roofline of the dominant kernel
    byts, flops, launches = kernel_model(wl, dominant, fwd_iters, adj_iters, rec_e, cpt)
    assert nl == launches * steps, (dominant, nl, launches, steps)
    avg_ms = kms / nl
    intensity = flops / byts
    ridge = PEAK_TFLOPS[wl.dtype] * 1e12 / (HBM_PEAK_GBS * 1e9)
    if intensity < ridge:
        achieved = byts / launches / (avg_ms / 1e3) / 1e9
        roof = {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s"}
    else:
        achieved = flops / launches / (avg_ms / 1e3) / 1e12
        on_mfma = wl.dtype == "f32" and (wl.layer == "conv3x3" or wl.q in MATRIX_CORE_WIDTHS) and \
            os.environ.get("LP_DENSE_PATH") != "valu"
        roof = {"bound": "mfma" if on_mfma else "alu", "achieved": achieved, "peak": PEAK_TFLOPS[wl.dtype],
                "unit": "TFLOP/s"}
    roof["frac"] = achieved / roof["peak"]
    roof["traffic"] = measured_traffic(dominant, f"cfg{wl.cfg}")
    roof["kernel"] = dominant
    roof["launches_per_step"] = launches
    roof["avg_launch_ms"] = avg_ms
    roof["algorithmic_bytes_per_launch"] = byts / launches
    roof["algorithmic_flops_per_launch"] = flops / launches

    # executed layer evaluations: every K v product the solves ran (a step Phi, an
    # adjoint step with the record, the coarse step of an FRES sweep; an adjoint step
    # that recomputes sigma' counts its two products), per second of solve time (the
    # step without the gradient)
    mac = wl.q * wl.q if wl.layer == "dense" else 9 * wl.C * wl.C * wl.H * wl.W
    solve_flops = sum(kernel_model(wl, k, fwd_iters, adj_iters, rec_e, cpt)[1]
                      for k in KIND_NAMES if k != "gradient")
    solve_ms = ms_step - per_kind.get("gradient", 0.0)
    products_per_s = solve_flops / (2.0 * mac) / (solve_ms / 1e3)

    # single-GPU context: the layer-serial forward pass (the baseline method)
    Us = torch.empty_like(Lam)
    Us[0] = U[0]
    L.lp_serial_forward(p, K, b, Us)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(5):
        L.lp_serial_forward(p, K, b, Us)
    torch.cuda.synchronize()
    serial_ms = (time.perf_counter() - t0) * 200.0
    del Us, U, Lam, ws, rec
    torch.cuda.empty_cache()
    return {
        "value": value,
        "ms_per_step": ms_step,
        "config": {"workload": f"cfg{wl.cfg}: {wl.name}", "N": wl.N, "B": wl.B, "width": wl.q,
                   "activation": wl.act, "mgrit": {"cf": wl.cf, "levels": len(level_sizes(
                       wl.N, wl.cf, wl.max_levels, wl.min_coarse)), "relax": wl.relax, "cycle": wl.cycle,
                       "fwd_iters": fwd_iters, "adj_iters": adj_iters},
                   "sigma_record": {0: None, 0.125: "bits", 1: "u8", 4: "f32"}[rec_e],
                   "storage": "C-points only (F-point states recomputed)" if cpt else "every layer",
                   "step": "MGRIT forward iterations + loss + MGRIT adjoint iterations + gradient"},
        "device_memory_gb": peak_gb,
        "roofline": roof,
        "kernel_ms_per_step": {k: v for k, v in sorted(per_kind.items(), key=lambda t: -t[1])},
        "layer_products_per_s": products_per_s,
        "serial_forward_ms": serial_ms,
        "residual_history": {"fwd": hist["fwd"], "adj": hist["adj"]},
    }


def one_shot_report(updates: int):
    """Algorithm 2 on the one-shot workload (lr = 1e-2, one forward and one adjoint
    MGRIT iteration per update) next to layer-serial gradient descent from the
    same seed, both on the GPU: the per-update losses, the time per update, and
    the largest relative deviation from the fp64 oracle's curves stored in
    tests/golden/one_shot_losses.txt (where it holds them)."""
    import numpy as np
    import torch

    from paper_1812_04352_amd import lp as L
    from paper_1812_04352_amd.one_shot import OneShotTrainer, SerialTrainer
    from workloads import ONE_SHOT_LR, WORKLOADS, generate

    wl = WORKLOADS[5]
    torch.cuda.set_device(0)
    d = generate(wl)

    def params():
        return {k: torch.from_numpy(np.ascontiguousarray(d[k])).cuda() for k in ("K", "b", "W", "mu", "L_in")}

    y, c = (torch.from_numpy(np.ascontiguousarray(d[k])).cuda() for k in ("y", "onehot"))
    p = L.problem(wl.dtype, wl.layer, wl.act, wl.N, wl.B, wl.C, wl.H, wl.W, wl.h)

    def mg(it):
        return L.mgrit(wl.cf, wl.max_levels, wl.min_coarse, wl.relax, it, cycle=wl.cycle)

    curves, times = {}, {}
    for name in ("one_shot", "layer_serial"):
        note(f"{name}: {updates} updates")
        tr = OneShotTrainer(p, mg(wl.fwd_iters), mg(wl.adj_iters), params(), y, c, wl.n_classes,
                            L.OPENING[wl.opening], wl.n_features) if name == "one_shot" else \
            SerialTrainer(p, params(), y, c, wl.n_classes, L.OPENING[wl.opening], wl.n_features)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        curves[name] = tr.run(updates, ONE_SHOT_LR)
        times[name] = (time.perf_counter() - t0) * 1000.0 / updates
        del tr
        torch.cuda.empty_cache()
    out = {"workload": f"cfg5: {wl.name}", "updates": updates, "lr": ONE_SHOT_LR,
           "ms_per_update": times, "loss": curves}
    path = os.path.join(ROOT, "tests", "golden", "one_shot_losses.txt")
    if os.path.exists(path):
        ref = np.loadtxt(path)
        dev = {}
        for col, name in ((1, "one_shot"), (2, "layer_serial")):
            r = ref[~np.isnan(ref[:, col]), col][:updates]
            if len(r):
                dev[name] = {"updates_compared": int(len(r)),
                             "max_rel_deviation": float(np.max(np.abs(np.array(curves[name][:len(r)]) - r) / np.abs(r)))}
        out["vs_oracle"] = dev
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=3,
                    help="workload 1..7 (default: the third, the deep dense network, the largest dense one)")
    ap.add_argument("--extra", type=int, nargs="*", default=None,
                    help="workloads measured after the headline one and reported under 'extra' (default: 4, the "
                         "convolutional network, when the headline is the default workload)")
    ap.add_argument("--extra-steps", type=int, default=5)
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-record", action="store_true",
                    help="let the adjoint and the gradient recompute sigma' instead of reading the record")
    ap.add_argument("--storage", choices=["all", "cpoints"], default="all",
                    help="primal trajectory storage: every layer, or the C-points only (dense widths 32/64)")
    ap.add_argument("--cpu-budget", type=float, default=16.0)
    ap.add_argument("--updates", type=int, default=0,
                    help="instead of the benchmark: run this many one-shot and layer-serial training updates of "
                         "the one-shot workload and report both loss curves")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 1 GiB device copy 5 times (to scale HBM byte counters)")
    ap.add_argument("--relax", choices=["F", "FCF", "FCFCF"], help="relaxation (default: the workload's)")
    ap.add_argument("--cycle", choices=["V", "F"], help="MGRIT cycle (default: the workload's V-cycle)")
    ap.add_argument("--cf", type=int, help="coarsening factor (default: the workload's, 4)")
    ap.add_argument("--traffic", nargs=4, metavar=("FETCH_DIR", "WRITE_DIR", "COPY_FETCH_DIR", "COPY_WRITE_DIR"),
                    help="summarise rocprofv3 FETCH_SIZE / WRITE_SIZE runs of --config into profiles/traffic.json "
                         "(no GPU needed)")
    args = ap.parse_args()
    if args.traffic:
        summarize_traffic(f"cfg{args.config}", *args.traffic)
        return
    if args.copy_calibration:
        import torch
        n = 1 << 28  # fp32 values = 1 GiB
        src = torch.ones(n, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_read_per_launch": 4 * n, "copy_bytes_written_per_launch": 4 * n,
                          "launches": 5}), flush=True)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (this build has no multi-GPU path); got --gpus {args.gpus}",
              file=sys.stderr)
        sys.exit(2)
    if args.updates:
        print(json.dumps(one_shot_report(args.updates)), flush=True)
        return

    from workloads import WORKLOADS

    def variant(wl):
        ov = {k: v for k, v in (("relax", args.relax), ("cycle", args.cycle), ("cf", args.cf)) if v}
        return wl.with_overrides(**ov) if ov else wl

    wl = variant(WORKLOADS[args.config])
    extra = args.extra if args.extra is not None else ([4] if args.config == 3 else [])
    res = measure(wl, args.steps, args.warmup, args.no_record, args.storage)
    out = {
        "metric": "layer-steps*examples/s per MGRIT fwd+adjoint iteration",
        "value": res["value"],
        "unit": "layer-steps*examples/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": res["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic",
    }
    out.update({k: v for k, v in res.items() if k not in ("value", "ms_per_step")})
    if extra:
        out["extra"] = {}
        for cfg in extra:
            wx = variant(WORKLOADS[cfg])
            rx = measure(wx, args.extra_steps, min(args.warmup, 3), args.no_record,
                         args.storage if wx.layer == "dense" and wx.q in (32, 64) else "all")
            rx["steps"], rx["dtype"] = args.extra_steps, wx.dtype
            out["extra"][f"cfg{cfg}"] = rx
    if not args.no_cpu:
        note("CPU oracle baseline")
        out["cpu_baseline"] = cpu_baseline(wl, args.cpu_budget)
    print(json.dumps(out), flush=True)


def ctypes_read(lib, kind):
    import ctypes
    n = ctypes.c_int32(0)
    ms = ctypes.c_double(0.0)
    rc = lib.lp_trace_read(kind, -1, ctypes.byref(n), ctypes.byref(ms))
    if rc != 0:
        raise RuntimeError(f"lp_trace_read failed: {rc}")
    return n.value, ms.value


if __name__ == "__main__":
    main()
