"""GPU parity: the HIP library (called through its C ABI) against the fp64 oracle
on the same seeded inputs. Sizes here are ones the oracle finishes in seconds and
still span several workgroup tiles and a ragged batch tail; the full workload
sizes are checked on sampled examples in test_gpu_fullsize.py."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_1812_04352_amd import lp as L
from workloads import WORKLOADS, random_state
from lp_testutil import Case, assert_close, sched, tdt

pytestmark = pytest.mark.gpu

# (name, workload) at parity-test sizes
DENSE = [
    ("tiny_f64", WORKLOADS[1]),
    ("relu32", WORKLOADS[2].with_overrides(N=64, B=300)),
    ("tanh64", WORKLOADS[3].with_overrides(N=128, B=300)),
    ("tanh32", WORKLOADS[5].with_overrides(N=64, B=513, n_features=40)),
    ("srelu16_f64", WORKLOADS[1].with_overrides(C=16, act="smoothrelu", N=48, B=257)),
    ("relu8_f32", WORKLOADS[2].with_overrides(C=8, N=32, B=77, n_features=12, n_classes=5)),
    ("conv_relu12", WORKLOADS[4].with_overrides(N=16, B=5, H=12, W=12, n_features=144, max_levels=3)),
    ("conv_tanh28", WORKLOADS[4].with_overrides(N=16, B=3, act="tanh", max_levels=3)),
    # width 220 (weights streamed through LDS in panels): ragged batch tiles, the
    # padded last feature block, every activation and record kind
    ("srelu220", WORKLOADS[7].with_overrides(N=32, B=100, max_levels=3)),
    ("relu220", WORKLOADS[7].with_overrides(act="relu", N=16, B=70, max_levels=2)),
    ("tanh220", WORKLOADS[7].with_overrides(act="tanh", N=16, B=33, max_levels=2)),
]
IDS = [n for n, _ in DENSE]

_cache = {}


def case(wl):
    key = repr(wl)
    if key not in _cache:
        _cache[key] = Case(wl)
    return _cache[key]


def _lamN(c, U_gpu):
    """Terminal adjoint value on each side from its own network output."""
    wl = c.wl
    J = torch.zeros(1, device="cuda", dtype=torch.float64)
    lamN = torch.empty_like(U_gpu[-1])
    dW = torch.empty_like(c.W)
    dmu = torch.empty_like(c.mu)
    L.lp_loss_terminal(c.p, wl.n_classes, U_gpu[-1], c.W, c.mu, c.onehot, J, lamN, dW, dmu, L.alloc_workspace(c.p))
    return lamN, J, dW, dmu


@pytest.mark.parametrize("name,wl", DENSE, ids=IDS)
def test_open_forward(name, wl):
    c = case(wl)
    assert_close(c.u0.cpu().numpy(), c.u0_ref, wl.dtype, "u0")


@pytest.mark.parametrize("name,wl", DENSE, ids=IDS)
def test_serial_forward_and_adjoint(name, wl):
    c = case(wl)
    U = c.new_traj()
    L.lp_serial_forward(c.p, c.K, c.b, U)
    Uref = O.serial_forward(c.u0_ref, c.d["K"], c.d["b"], wl.h, wl.act)
    assert_close(U.cpu().numpy(), Uref, wl.dtype, "U")
    lamN, J, dW, dmu = _lamN(c, U)
    Jr, lamNr, dWr, dmur = O.loss_terminal(Uref[-1], c.d["W"], c.d["mu"], c.d["onehot"])
    assert abs(J.item() - Jr) <= 10 * {"f32": 1e-6, "f64": 1e-14}[wl.dtype] * abs(Jr)
    assert_close(lamN.cpu().numpy(), lamNr, wl.dtype, "lamN")
    assert_close(dW.cpu().numpy(), dWr, wl.dtype, "dW")
    assert_close(dmu.cpu().numpy(), dmur, wl.dtype, "dmu")
    Lam = torch.zeros_like(U)
    Lam[-1] = lamN
    L.lp_serial_adjoint(c.p, c.K, c.b, U, Lam)
    Lref = O.serial_adjoint(Uref, lamNr, c.d["K"], c.d["b"], wl.h, wl.act)
    assert_close(Lam.cpu().numpy(), Lref, wl.dtype, "Lam")
    # reduced gradient of the layer weights and of the opening layer
    ws = L.alloc_workspace(c.p)
    dK, db = torch.empty_like(c.K), torch.empty_like(c.b)
    L.lp_gradient(c.p, c.K, c.b, U, Lam, dK, db, ws)
    dKr, dbr = O.gradient(Uref, Lref, c.d["K"], c.d["b"], wl.h, wl.act)
    assert_close(dK.cpu().numpy(), dKr, wl.dtype, "dK")
    assert_close(db.cpu().numpy(), dbr, wl.dtype, "db")
    if wl.opening != "identity":
        dL = torch.empty_like(c.L_in)
        L.lp_open_grad(c.p, L.OPENING[wl.opening], wl.n_features, c.y, c.L_in, Lam[0], dL)
        dLr = O.open_grad(c.d["y"], c.d["L_in"], Lref[0], wl.act, wl.opening)
        assert_close(dL.cpu().numpy(), dLr, wl.dtype, "dL_in")


@pytest.mark.parametrize("relax", ["FCF", "F"])
@pytest.mark.parametrize("name,wl", DENSE, ids=IDS)
def test_mgrit_forward_iterates(name, wl, relax):
    c = case(wl)
    iters = max(wl.fwd_iters, 3)
    mg = sched(wl, iters, relax=relax)
    ws = L.alloc_workspace(c.p, mg)
    U = c.new_traj()
    it, hist = L.lp_mgrit_forward(c.p, mg, c.K, c.b, U, ws)
    assert it == iters
    Ur, hr, _ = O.mgrit_forward(c.ref_traj(), c.d["K"], c.d["b"], wl.h, wl.act, cf=wl.cf,
                                max_levels=wl.max_levels, min_coarse=wl.min_coarse, relax=relax, max_iter=iters)
    assert_close(U.cpu().numpy(), Ur, wl.dtype, "U iterate")
    # residual history: relative to rho_1 (late entries sit near the rounding floor in fp32)
    floor = {"f32": 3e-5, "f64": 1e-11}[wl.dtype]
    for m in range(iters):
        assert abs(hist[m] - hr[m]) <= floor * hr[0] + 1e-5 * hr[m], (m, hist, hr)


@pytest.mark.parametrize("relax", ["FCF", "F"])
@pytest.mark.parametrize("name,wl", DENSE, ids=IDS)
def test_mgrit_adjoint_iterates(name, wl, relax):
    c = case(wl)
    U = c.new_traj()
    L.lp_serial_forward(c.p, c.K, c.b, U)
    lamN, _, _, _ = _lamN(c, U)
    Uref = O.serial_forward(c.u0_ref, c.d["K"], c.d["b"], wl.h, wl.act)
    lamNr = O.loss_terminal(Uref[-1], c.d["W"], c.d["mu"], c.d["onehot"])[1]
    iters = max(wl.adj_iters, 3)
    mg = sched(wl, iters, relax=relax)
    ws = L.alloc_workspace(c.p, mg)
    Lam = torch.zeros_like(U)
    Lam[-1] = lamN
    it, hist = L.lp_mgrit_adjoint(c.p, mg, c.K, c.b, U, Lam, ws)
    L0 = np.zeros_like(Uref)
    L0[-1] = lamNr
    Lr, hr, _ = O.mgrit_adjoint(Uref, L0, c.d["K"], c.d["b"], wl.h, wl.act, cf=wl.cf, max_levels=wl.max_levels,
                                min_coarse=wl.min_coarse, relax=relax, max_iter=iters)
    assert_close(Lam.cpu().numpy(), Lr, wl.dtype, "Lam iterate")
    floor = {"f32": 3e-5, "f64": 1e-11}[wl.dtype]
    for m in range(iters):
        assert abs(hist[m] - hr[m]) <= floor * hr[0] + 1e-5 * hr[m], (m, hist, hr)


@pytest.mark.parametrize("name,wl", DENSE, ids=IDS)
def test_residual_norms(name, wl):
    c = case(wl)
    mg = sched(wl, 1)
    ws = L.alloc_workspace(c.p, mg)
    U = c.new_traj()
    L.lp_mgrit_forward(c.p, mg, c.K, c.b, U, ws)
    Ur, _, _ = O.mgrit_forward(c.ref_traj(), c.d["K"], c.d["b"], wl.h, wl.act, cf=wl.cf, max_levels=wl.max_levels,
                               min_coarse=wl.min_coarse, relax=wl.relax, max_iter=1)
    r = L.lp_residual_norm(c.p, L.LP_STATE, c.K, c.b, U, None, ws)
    rr = O.residual_norm_state(Ur, c.d["K"], c.d["b"], wl.h, wl.act)
    assert abs(r - rr) <= {"f32": 1e-4, "f64": 1e-10}[wl.dtype] * rr
    # adjoint: each side linearises at its own forward iterate; the terminal value is a
    # seeded random state given to both
    lamN = random_state(wl, 77)[0]
    Lam = torch.zeros_like(U)
    Lam[-1] = torch.from_numpy(lamN).to(U)
    Lr = np.zeros_like(Ur)
    Lr[-1] = lamN
    L.lp_mgrit_adjoint(c.p, mg, c.K, c.b, U, Lam, ws)
    Lr, _, _ = O.mgrit_adjoint(Ur, Lr, c.d["K"], c.d["b"], wl.h, wl.act, cf=wl.cf,
                               max_levels=wl.max_levels, min_coarse=wl.min_coarse, relax=wl.relax, max_iter=1)
    r = L.lp_residual_norm(c.p, L.LP_ADJOINT, c.K, c.b, U, Lam, ws)
    rr = O.residual_norm_adjoint(Ur, Lr, c.d["K"], c.d["b"], wl.h, wl.act)
    assert abs(r - rr) <= {"f32": 1e-4, "f64": 1e-10}[wl.dtype] * rr


@pytest.mark.parametrize("name,wl", DENSE[:4], ids=IDS[:4])
def test_invariants_on_gpu(name, wl):
    """Properties of MGRIT checked on the GPU alone: the serial solution has zero
    residual and is a fixed point; two-level F-relaxation is exact after N/c
    iterations (Parareal finite-step exactness)."""
    c = case(wl)
    S = c.new_traj()
    L.lp_serial_forward(c.p, c.K, c.b, S)
    need = max(L.lp_workspace_bytes(c.p, sched(wl, wl.N // wl.cf, relax="F", levels=2)),
               L.lp_workspace_bytes(c.p, sched(wl, 1, warm=True)))
    big = torch.empty(need, dtype=torch.uint8, device="cuda")
    nrm = float(S.double().norm())
    assert L.lp_residual_norm(c.p, L.LP_STATE, c.K, c.b, S, None, big) <= {"f32": 1e-6, "f64": 1e-14}[wl.dtype] * nrm
    U = S.clone()
    it, hist = L.lp_mgrit_forward(c.p, sched(wl, 1, warm=True), c.K, c.b, U, big)
    assert float((U - S).abs().max()) <= {"f32": 1e-5, "f64": 1e-13}[wl.dtype] * float(S.abs().max())
    assert hist[0] <= {"f32": 1e-5, "f64": 1e-13}[wl.dtype] * nrm
    U = c.new_traj()
    L.lp_mgrit_forward(c.p, sched(wl, wl.N // wl.cf, relax="F", levels=2), c.K, c.b, U, big)
    assert_close(U.cpu().numpy(), S.cpu().numpy(), wl.dtype, "two-level F after N/c iterations")


def test_stop_rules_and_errors():
    wl = DENSE[2][1]
    c = case(wl)
    mg = sched(wl, 30, rtol=1e-4)
    ws = L.alloc_workspace(c.p, mg)
    U = c.new_traj()
    it, hist = L.lp_mgrit_forward(c.p, mg, c.K, c.b, U, ws)
    assert it < 30 and hist[-1] <= 1e-4 * hist[0] and all(h > 1e-4 * hist[0] for h in hist[:-1])
    # workspace too small -> LP_EWORKSPACE before any work is enqueued
    with pytest.raises(L.LpError) as e:
        L.lp_mgrit_forward(c.p, mg, c.K, c.b, U, ws[:128])
    assert e.value.status == L.LP_EWORKSPACE
    # non-finite input -> LP_ENONFINITE
    U = c.new_traj()
    U[0, 0, 0] = float("nan")
    with pytest.raises(L.LpError) as e:
        L.lp_mgrit_forward(c.p, sched(wl, 2), c.K, c.b, U, ws)
    assert e.value.status == L.LP_ENONFINITE
    # the device flag recorded it as well; the check reports it once and clears it
    with pytest.raises(L.LpError) as e:
        L.lp_check_finite()
    assert e.value.status == L.LP_ENONFINITE
    L.lp_check_finite()


@pytest.mark.parametrize("name,wl", [DENSE[1], DENSE[6], DENSE[8]], ids=[DENSE[1][0], DENSE[6][0], DENSE[8][0]])
def test_nonfinite_without_readback(name, wl):
    """Solves that read nothing back (no stopping rule, no history) still record a
    non-finite residual norm on the device; lp_check_finite reports it, and the
    one-shot trainer, which runs that way, raises instead of training on NaN."""
    from paper_1812_04352_amd.one_shot import OneShotTrainer
    c = case(wl)
    L.lp_check_finite()  # nothing pending
    mg = sched(wl, 2)
    ws = L.alloc_workspace(c.p, mg)
    U = c.new_traj()
    U[0].view(-1)[7] = float("nan")
    assert L.lp_mgrit_forward(c.p, mg, c.K, c.b, U, ws, history=False) == (2, [])
    with pytest.raises(L.LpError) as e:
        L.lp_check_finite()
    assert e.value.status == L.LP_ENONFINITE
    L.lp_check_finite()  # cleared
    # a finite solve sets nothing
    U = c.new_traj()
    L.lp_mgrit_forward(c.p, mg, c.K, c.b, U, ws, history=False)
    L.lp_check_finite()
    # a diverging design in the one-shot trainer
    P = {k: getattr(c, k).clone() for k in ("K", "b", "W", "mu") + (("L_in",) if c.L_in is not None else ())}
    P["K"].view(-1)[3] = float("inf")
    tr = OneShotTrainer(c.p, sched(wl, 1), sched(wl, 1), P, c.y, c.onehot, wl.n_classes, L.OPENING[wl.opening],
                        wl.n_features)
    with pytest.raises(L.LpError) as e:
        tr.run(1, 1e-2)
    assert e.value.status == L.LP_ENONFINITE
    L.lp_check_finite()


@pytest.mark.parametrize("name,wl", [DENSE[1], DENSE[2], DENSE[3], DENSE[6], DENSE[8]],
                         ids=[DENSE[i][0] for i in (1, 2, 3, 6, 8)])
def test_gradient_and_loss_are_bitwise_reproducible(name, wl):
    """lp_gradient (with and without the sigma' record) and lp_loss_terminal give
    bit-identical results when called twice on the same inputs, the second time
    with a workspace pre-filled with NaN bytes (so no result may depend on what the
    workspace held): every batch reduction runs in a fixed order."""
    c = case(wl)
    mg = sched(wl, 2)
    ws = L.alloc_workspace(c.p, mg)
    rec = L.alloc_dsig(c.p) if L.lp_dsig_bytes(c.p) else None
    U = c.new_traj()
    L.lp_mgrit_forward(c.p, mg, c.K, c.b, U, ws, dsig=rec)
    Lam = torch.zeros_like(U)
    outs = []
    for t in range(2):
        if t:
            ws.fill_(0xFF)
        J = torch.zeros(1, device="cuda", dtype=torch.float64)
        lamN, dW, dmu = torch.empty_like(U[-1]), torch.empty_like(c.W), torch.empty_like(c.mu)
        L.lp_loss_terminal(c.p, wl.n_classes, U[-1], c.W, c.mu, c.onehot, J, lamN, dW, dmu, ws)
        if t == 0:
            Lam[-1] = lamN
            L.lp_mgrit_adjoint(c.p, mg, c.K, c.b, U, Lam, ws, dsig=rec)
        g = []
        for r in (rec, None):
            if t:
                ws.fill_(0xFF)
            dK, db = torch.empty_like(c.K), torch.empty_like(c.b)
            L.lp_gradient(c.p, c.K, c.b, U, Lam, dK, db, ws, dsig=r)
            g += [dK, db]
        outs.append([J, lamN, dW, dmu] + g)
    names = ["J", "lamN", "dW", "dmu", "dK (record)", "db (record)", "dK", "db"]
    for n, a, b in zip(names, outs[0], outs[1]):
        assert torch.equal(a, b), n


@pytest.mark.parametrize("name,wl", [DENSE[1], DENSE[2], DENSE[6], DENSE[7]],
                         ids=[DENSE[i][0] for i in (1, 2, 6, 7)])
def test_solves_are_bitwise_reproducible(name, wl):
    """Two forward and two adjoint MGRIT solves from the same cold start give
    bit-identical iterates and residual histories (Algorithm 1; the residual norms
    are reduced in a fixed order), the second time with a workspace pre-filled with
    NaN bytes. The conv cases run grids whose size is not a multiple of eight, the
    uneven branch of the sweeps' workgroup order."""
    c = case(wl)
    mg = sched(wl, 2)
    ws = L.alloc_workspace(c.p, mg)
    rec = L.alloc_dsig(c.p) if L.lp_dsig_bytes(c.p) else None
    outs = []
    for t in range(2):
        if t:
            ws.fill_(0xFF)
        U = c.new_traj()
        _, hf = L.lp_mgrit_forward(c.p, mg, c.K, c.b, U, ws, history=True, dsig=rec)
        J = torch.zeros(1, device="cuda", dtype=torch.float64)
        Lam = torch.zeros_like(U)
        dW, dmu = torch.empty_like(c.W), torch.empty_like(c.mu)
        L.lp_loss_terminal(c.p, wl.n_classes, U[-1], c.W, c.mu, c.onehot, J, Lam[-1], dW, dmu, ws)
        _, ha = L.lp_mgrit_adjoint(c.p, mg, c.K, c.b, U, Lam, ws, history=True, dsig=rec)
        outs.append((U, Lam, list(hf), list(ha)))
    (U0, L0, f0, a0), (U1, L1, f1, a1) = outs
    assert torch.equal(U0, U1), "U"
    assert torch.equal(L0, L1), "Lam"
    assert f0 == f1 and a0 == a1, (f0, f1, a0, a1)
    assert len(f0) == 2 and len(a0) == 2


@pytest.mark.parametrize("name,wl", [DENSE[1], DENSE[2], DENSE[7]], ids=[DENSE[1][0], DENSE[2][0], DENSE[7][0]])
def test_solves_without_history_match(name, wl):
    """With no residual history and no stopping rule the solves return without
    waiting for the stream; the iterates must equal those of the reading call."""
    c = case(wl)
    mg = sched(wl, 3)
    ws = L.alloc_workspace(c.p, mg)
    U1, U2 = c.new_traj(), c.new_traj()
    assert L.lp_mgrit_forward(c.p, mg, c.K, c.b, U1, ws)[0] == 3
    assert L.lp_mgrit_forward(c.p, mg, c.K, c.b, U2, ws, history=False) == (3, [])
    torch.cuda.synchronize()
    assert torch.equal(U1, U2)
    L1 = torch.zeros_like(U1)
    L1[-1] = _lamN(c, U1)[0]
    L2 = L1.clone()
    L.lp_mgrit_adjoint(c.p, mg, c.K, c.b, U1, L1, ws)
    assert L.lp_mgrit_adjoint(c.p, mg, c.K, c.b, U1, L2, ws, history=False) == (3, [])
    torch.cuda.synchronize()
    assert torch.equal(L1, L2)


def test_tracing_counts_launches():
    """The trace records one timed entry per traced launch site: with FCF on L
    levels and m V-cycles the forward solve runs m FC and m FRES sweeps per
    non-coarsest level, m coarsest solves, and (with the finest correction
    deferred) m CORRF sweeps per middle level plus one final finest CORRF."""
    wl = DENSE[1][1]
    c = case(wl)
    m = 3
    mg = sched(wl, m)
    ws = L.alloc_workspace(c.p, mg)
    U = c.new_traj()
    L.lp_trace_enable((1 << 11) - 1)
    try:
        L.lp_mgrit_forward(c.p, mg, c.K, c.b, U, ws, history=False)
        torch.cuda.synchronize()
        levels = len(O.level_sizes(wl.N, wl.cf, wl.max_levels, wl.min_coarse))
        got = {k: L.lp_trace_read(k) for k in range(4)}
    finally:
        L.lp_trace_enable(0)
    assert got[0][0] == m * (levels - 1) and got[1][0] == m * (levels - 1)
    assert got[3][0] == m
    assert got[2][0] == m * (levels - 2) + 1
    assert all(ms > 0.0 for n, ms in got.values() if n)
    for k in range(4, 11):
        assert L.lp_trace_read(k) == (0, 0.0)


def test_empty_batch_is_a_no_op():
    wl = DENSE[1][1]
    p = L.problem(wl.dtype, wl.layer, wl.act, wl.N, 0, wl.C, h=wl.h)
    K = torch.zeros((wl.N, wl.C, wl.C), device="cuda", dtype=tdt(wl))
    b = torch.zeros((wl.N, wl.C), device="cuda", dtype=tdt(wl))
    U = torch.zeros((wl.N + 1, 0, wl.C), device="cuda", dtype=tdt(wl))
    ws = L.alloc_workspace(p, sched(wl, 2))
    assert L.lp_mgrit_forward(p, sched(wl, 2), K, b, U, ws) == (0, [])
    dK, db = torch.ones_like(K), torch.ones_like(b)
    L.lp_gradient(p, K, b, U, U.clone(), dK, db, ws)
    assert float(dK.abs().max()) == 0.0 and float(db.abs().max()) == 0.0


@pytest.mark.parametrize("name,wl", [DENSE[1], DENSE[2]], ids=[DENSE[1][0], DENSE[2][0]])
def test_valu_kernels_match_oracle(name, wl, monkeypatch):
    """The vector-ALU kernels for fp32 widths that normally run on the matrix cores
    (selected with LP_DENSE_PATH=valu) also meet the parity bar."""
    monkeypatch.setenv("LP_DENSE_PATH", "valu")
    c = case(wl)
    mg = sched(wl, 3)
    ws = L.alloc_workspace(c.p, mg)
    U = c.new_traj()
    L.lp_mgrit_forward(c.p, mg, c.K, c.b, U, ws)
    Ur, _, _ = O.mgrit_forward(c.ref_traj(), c.d["K"], c.d["b"], wl.h, wl.act, cf=wl.cf, max_levels=wl.max_levels,
                               min_coarse=wl.min_coarse, relax=wl.relax, max_iter=3)
    assert_close(U.cpu().numpy(), Ur, wl.dtype, "U (VALU)")
    lamN = random_state(wl, 5)[0]
    Lam = torch.zeros_like(U)
    Lam[-1] = torch.from_numpy(lamN).to(U)
    L.lp_mgrit_adjoint(c.p, mg, c.K, c.b, U, Lam, ws)
    L0 = np.zeros_like(Ur)
    L0[-1] = lamN
    Lr, _, _ = O.mgrit_adjoint(Ur, L0, c.d["K"], c.d["b"], wl.h, wl.act, cf=wl.cf, max_levels=wl.max_levels,
                               min_coarse=wl.min_coarse, relax=wl.relax, max_iter=3)
    assert_close(Lam.cpu().numpy(), Lr, wl.dtype, "Lam (VALU)")
    dK, db = torch.empty_like(c.K), torch.empty_like(c.b)
    L.lp_gradient(c.p, c.K, c.b, U, Lam, dK, db, ws)
    dKr, dbr = O.gradient(Ur, Lr, c.d["K"], c.d["b"], wl.h, wl.act)
    assert_close(dK.cpu().numpy(), dKr, wl.dtype, "dK (VALU)")
    assert_close(db.cpu().numpy(), dbr, wl.dtype, "db (VALU)")


def test_one_shot_training_matches_oracle():
    """Algorithm 2 with one forward and one adjoint MGRIT iteration per update and a
    plain gradient step: per-update losses and final weights against the oracle's
    one-shot run (reduced size, larger step so that the weights move)."""
    from paper_1812_04352_amd.one_shot import OneShotTrainer
    wl = WORKLOADS[5].with_overrides(N=64, B=300, n_features=40)
    c = case(wl)
    updates, lr = 12, 0.5
    params = {k: getattr(c, k).clone() for k in ("K", "b", "W", "mu", "L_in")}
    tr = OneShotTrainer(c.p, sched(wl, wl.fwd_iters), sched(wl, wl.adj_iters), params, c.y, c.onehot,
                        wl.n_classes, L.OPENING[wl.opening], wl.n_features)
    losses = tr.run(updates, lr)
    d = c.d
    lo, wo = O.one_shot(d["y"], d["onehot"], d["L_in"], d["K"], d["b"], d["W"], d["mu"], wl.h, wl.act, wl.opening,
                        cf=wl.cf, max_levels=wl.max_levels, min_coarse=wl.min_coarse, relax=wl.relax,
                        updates=updates, lr=lr, m1=wl.fwd_iters, m2=wl.adj_iters)
    for i, (a, b) in enumerate(zip(losses, lo)):
        assert abs(a - b) <= 1e-4 * abs(b), (i, a, b)
    assert losses[-1] < losses[0]
    for k in params:
        assert_close(params[k].cpu().numpy(), wo[k], wl.dtype, f"{k} after {updates} updates", scale=10)


def _deepest(wl, most=4):
    """The most levels (up to `most`) the workload's N allows with its cf."""
    for lv in range(most, 1, -1):
        try:
            O.level_sizes(wl.N, wl.cf, lv, wl.min_coarse)
            return lv
        except ValueError:
            pass
    return 2


@pytest.mark.parametrize("relax,cycle", [("FCFCF", "V"), ("FCF", "F"), ("F", "F"), ("FCFCF", "F")])
@pytest.mark.parametrize("name,wl", DENSE, ids=IDS)
def test_mgrit_cycle_variants(name, wl, relax, cycle):
    """F-cycles and FCFCF relaxation on the deepest hierarchy the size allows:
    forward and adjoint iterates and residual histories against the oracle."""
    c = case(wl)
    levels = _deepest(wl)
    iters = 3
    mg = sched(wl, iters, relax=relax, levels=levels, cycle=cycle)
    ws = L.alloc_workspace(c.p, mg)
    U = c.new_traj()
    it, hist = L.lp_mgrit_forward(c.p, mg, c.K, c.b, U, ws)
    assert it == iters
    Ur, hr, _ = O.mgrit_forward(c.ref_traj(), c.d["K"], c.d["b"], wl.h, wl.act, cf=wl.cf, max_levels=levels,
                                min_coarse=wl.min_coarse, relax=relax, max_iter=iters, cycle=cycle)
    assert_close(U.cpu().numpy(), Ur, wl.dtype, "U iterate")
    floor = {"f32": 3e-5, "f64": 1e-11}[wl.dtype]
    for m in range(iters):
        assert abs(hist[m] - hr[m]) <= floor * hr[0] + 1e-5 * hr[m], (m, hist, hr)
    # adjoint, linearised at the serial trajectory on each side
    L.lp_serial_forward(c.p, c.K, c.b, U)
    lamN, _, _, _ = _lamN(c, U)
    Us = O.serial_forward(c.u0_ref, c.d["K"], c.d["b"], wl.h, wl.act)
    lamNr = O.loss_terminal(Us[-1], c.d["W"], c.d["mu"], c.d["onehot"])[1]
    Lam = torch.zeros_like(U)
    Lam[-1] = lamN
    it, hist = L.lp_mgrit_adjoint(c.p, mg, c.K, c.b, U, Lam, ws)
    Lr0 = np.zeros_like(Us)
    Lr0[-1] = lamNr
    Lr, hr, _ = O.mgrit_adjoint(Us, Lr0, c.d["K"], c.d["b"], wl.h, wl.act, cf=wl.cf, max_levels=levels,
                                min_coarse=wl.min_coarse, relax=relax, max_iter=iters, cycle=cycle)
    assert_close(Lam.cpu().numpy(), Lr, wl.dtype, "Lam iterate")
    for m in range(iters):
        assert abs(hist[m] - hr[m]) <= floor * hr[0] + 1e-5 * hr[m], (m, hist, hr)


@pytest.mark.parametrize("cf", [2, 8])
@pytest.mark.parametrize("name,wl", DENSE, ids=IDS)
def test_mgrit_coarsening_factors(name, wl, cf):
    """Coarsening factors other than 4 (the intervals' kernels take c at run time;
    the interval-resident width-32 kernels are built for c = 4, so other factors
    run the per-step kernels): forward and adjoint iterates and residual
    histories on the deepest hierarchy the size allows, the forward keeping the
    sigma' record where the kernels support one (the adjoint then reads it)."""
    wl = wl.with_overrides(cf=cf)
    c = case(wl)
    levels = _deepest(wl)
    iters = 3
    mg = sched(wl, iters, levels=levels)
    ws = L.alloc_workspace(c.p, mg)
    rec = L.alloc_dsig(c.p) if L.lp_dsig_bytes(c.p) else None
    U = c.new_traj()
    it, hist = L.lp_mgrit_forward(c.p, mg, c.K, c.b, U, ws, dsig=rec)
    assert it == iters
    Ur, hr, _ = O.mgrit_forward(c.ref_traj(), c.d["K"], c.d["b"], wl.h, wl.act, cf=cf, max_levels=levels,
                                min_coarse=wl.min_coarse, relax=wl.relax, max_iter=iters)
    assert_close(U.cpu().numpy(), Ur, wl.dtype, f"U iterate, cf={cf}")
    floor = {"f32": 3e-5, "f64": 1e-11}[wl.dtype]
    for m in range(iters):
        assert abs(hist[m] - hr[m]) <= floor * hr[0] + 1e-5 * hr[m], (m, hist, hr)
    # adjoint linearised at each side's own forward iterate
    lamN, _, _, _ = _lamN(c, U)
    lamNr = O.loss_terminal(Ur[-1], c.d["W"], c.d["mu"], c.d["onehot"])[1]
    Lam = torch.zeros_like(U)
    Lam[-1] = lamN
    it, hist = L.lp_mgrit_adjoint(c.p, mg, c.K, c.b, U, Lam, ws, dsig=rec)
    Lr0 = np.zeros_like(Ur)
    Lr0[-1] = lamNr
    Lr, hr, _ = O.mgrit_adjoint(Ur, Lr0, c.d["K"], c.d["b"], wl.h, wl.act, cf=cf, max_levels=levels,
                                min_coarse=wl.min_coarse, relax=wl.relax, max_iter=iters)
    assert_close(Lam.cpu().numpy(), Lr, wl.dtype, f"Lam iterate, cf={cf}")
    for m in range(iters):
        assert abs(hist[m] - hr[m]) <= floor * hr[0] + 1e-5 * hr[m], (m, hist, hr)


DEGENERATE = [DENSE[0], DENSE[1], DENSE[2], DENSE[3], DENSE[6], DENSE[8]]


@pytest.mark.parametrize("N,cf", [(4, 4), (8, 8), (1, 4)])
@pytest.mark.parametrize("name,wl", DEGENERATE, ids=[n for n, _ in DEGENERATE])
def test_degenerate_hierarchies(name, wl, N, cf):
    """A single coarse interval (N = cf: one workgroup is both the first and the
    last interval, so both boundary branches of every sweep run in it) and a
    single layer (N = 1: one level, the serial solve): forward and adjoint iterates
    against the oracle, with the sigma' record where the kernels keep one."""
    wl = wl.with_overrides(N=N, cf=cf, max_levels=2, min_coarse=1, T=wl.T * N / wl.N)
    c = case(wl)
    iters = 2
    mg = sched(wl, iters)
    ws = L.alloc_workspace(c.p, mg)
    rec = L.alloc_dsig(c.p) if L.lp_dsig_bytes(c.p) else None
    U = c.new_traj()
    L.lp_mgrit_forward(c.p, mg, c.K, c.b, U, ws, dsig=rec)
    Ur, _, _ = O.mgrit_forward(c.ref_traj(), c.d["K"], c.d["b"], wl.h, wl.act, cf=cf, max_levels=2,
                               min_coarse=1, relax=wl.relax, max_iter=iters)
    assert_close(U.cpu().numpy(), Ur, wl.dtype, f"U, N={N}, cf={cf}")
    lamN, _, _, _ = _lamN(c, U)
    lamNr = O.loss_terminal(Ur[-1], c.d["W"], c.d["mu"], c.d["onehot"])[1]
    Lam = torch.zeros_like(U)
    Lam[-1] = lamN
    L.lp_mgrit_adjoint(c.p, mg, c.K, c.b, U, Lam, ws, dsig=rec)
    Lr0 = np.zeros_like(Ur)
    Lr0[-1] = lamNr
    Lr, _, _ = O.mgrit_adjoint(Ur, Lr0, c.d["K"], c.d["b"], wl.h, wl.act, cf=cf, max_levels=2, min_coarse=1,
                               relax=wl.relax, max_iter=iters)
    assert_close(Lam.cpu().numpy(), Lr, wl.dtype, f"Lam, N={N}, cf={cf}")


# fp32 widths on the matrix cores with a non-identity activation: the ones that keep a sigma' record
RECORDED = [DENSE[1], DENSE[2], DENSE[3],
            ("srelu32", WORKLOADS[2].with_overrides(act="smoothrelu", N=32, B=77, max_levels=2)),
            DENSE[6], DENSE[7], DENSE[8], DENSE[9]]


def _conv_record(rec, N, B, C, H, W, relu):
    """The convolution record ([N][B] blocks in the kernels' tile order, see
    lp_dsig_bytes in include/lp.h) rearranged to [N][B][C][H][W]: tile t of 16
    pair-pixels, lane l: pair-pixel P = 16 t + l % 16 (ghost lanes P >= H/2 W are
    skipped), value r of the lane = channel 2 (l // 16) + r // 2, row 2 (P // W) +
    r % 2, column P % W. ReLU: one 32-bit word per lane of each wave w (tiles
    7 w .. 7 w + 6), bit 4 (t - 7 w) + r; smooth activations: four fp32 values per
    tile and lane."""
    npp = H // 2 * W
    T = -(-(-(-npp // 16)) // 7) * 7
    if relu:
        words = rec[: N * B * (T // 7) * 64 * 4].cpu().view(torch.int32).numpy().view(np.uint32)
        words = words.reshape(N, B, T // 7, 64)
        vals = np.zeros((N, B, T, 64, 4), dtype=np.uint8)
        for t in range(T):
            for r in range(4):
                vals[:, :, t, :, r] = (words[:, :, t // 7, :] >> (4 * (t % 7) + r)) & 1
    else:
        vals = rec[: N * B * T * 64 * 16].cpu().view(torch.float32).numpy().reshape(N, B, T, 64, 4)
    out = np.zeros((N, B, C, H, W), dtype=vals.dtype)
    for t in range(T):
        for l in range(64):
            P = 16 * t + l % 16
            if P >= npp:
                continue
            Y, x = divmod(P, W)
            for r in range(4):
                out[:, :, 2 * (l // 16) + r // 2, 2 * Y + r % 2, x] = vals[:, :, t, l, r]
    return out.reshape(N, B, C * H * W)


def _check_record(c, U, rec):
    """The record against sigma'(K_n u_n + b_n) evaluated by the oracle in fp64 at
    the trajectory the GPU returned. ReLU's 0/1 decisions may differ from the fp64
    decision only where the pre-activation is within fp32 rounding of zero."""
    wl = c.wl
    Uh = U.double().cpu().numpy()
    z = np.stack([O.preact(c.d["K"][n], c.d["b"][n], Uh[n]) for n in range(wl.N)])
    want = O.dact(z, wl.act)
    if wl.layer == "conv3x3":
        got = _conv_record(rec, wl.N, wl.B, wl.C, wl.H, wl.W, wl.act == "relu").reshape(z.shape)
        if wl.act == "relu":
            assert set(np.unique(got)) <= {0, 1}
            bad = got != want
            assert np.all(np.abs(z[bad]) <= 1e-5 * np.abs(z).max()), f"{bad.sum()} wrong record bits"
        else:
            np.testing.assert_allclose(got, want, rtol=0, atol=2e-5)
        return
    if wl.act == "relu":
        if wl.q == 220:  # one byte per element
            got = rec[: z.size].cpu().numpy().reshape(z.shape)
        else:  # one bit per element in element order, least significant bit first
            got = np.unpackbits(rec[: z.size // 8].cpu().numpy(), bitorder="little").reshape(z.shape)
        assert set(np.unique(got)) <= {0, 1}
        bad = got != want
        scale = np.abs(z).max()
        assert np.all(np.abs(z[bad]) <= 1e-5 * scale), f"{bad.sum()} wrong record values"
    else:
        got = rec.view(torch.float32)[: z.size].cpu().numpy().reshape(z.shape)
        np.testing.assert_allclose(got, want, rtol=0, atol=2e-5)


@pytest.mark.parametrize("relax", ["FCF", "F"])
@pytest.mark.parametrize("name,wl", RECORDED, ids=[n for n, _ in RECORDED])
def test_sigma_record_in_mgrit(name, wl, relax):
    """An MGRIT forward solve that keeps the sigma' record returns the same
    trajectory, and its record holds sigma' at that trajectory; an adjoint that
    reads the record returns what the recomputing adjoint returns bit for bit,
    and the gradient that reads it meets the parity bar."""
    wl = wl.with_overrides(relax=relax)
    c = case(wl)
    mg = sched(wl, 2)
    ws = L.alloc_workspace(c.p, mg)
    U1, U2 = c.new_traj(), c.new_traj()
    rec = L.alloc_dsig(c.p)
    L.lp_mgrit_forward(c.p, mg, c.K, c.b, U1, ws, history=False)
    L.lp_mgrit_forward(c.p, mg, c.K, c.b, U2, ws, history=False, dsig=rec)
    torch.cuda.synchronize()
    assert torch.equal(U1, U2)
    _check_record(c, U1, rec)
    L1 = torch.zeros_like(U1)
    L1[-1] = _lamN(c, U1)[0]
    L2 = L1.clone()
    L.lp_mgrit_adjoint(c.p, mg, c.K, c.b, U1, L1, ws, history=False)
    L.lp_mgrit_adjoint(c.p, mg, c.K, c.b, U1, L2, ws, history=False, dsig=rec)
    torch.cuda.synchronize()
    assert torch.equal(L1, L2)
    dK1, db1 = torch.empty_like(c.K), torch.empty_like(c.b)
    dK2, db2 = torch.empty_like(c.K), torch.empty_like(c.b)
    L.lp_gradient(c.p, c.K, c.b, U1, L1, dK1, db1, ws)
    L.lp_gradient(c.p, c.K, c.b, U1, L1, dK2, db2, ws, dsig=rec)
    dKr, dbr = O.gradient(U1.double().cpu().numpy(), L1.double().cpu().numpy(), c.d["K"], c.d["b"], wl.h, wl.act)
    assert_close(dK2.cpu().numpy(), dKr, wl.dtype, "dK (record)")
    assert_close(db2.cpu().numpy(), dbr, wl.dtype, "db (record)")
    assert_close(dK2.cpu().numpy(), dK1.double().cpu().numpy(), wl.dtype, "dK record vs recompute")


@pytest.mark.parametrize("name,wl", RECORDED[:2] + RECORDED[4:], ids=[n for n, _ in RECORDED[:2] + RECORDED[4:]])
def test_sigma_record_in_serial_solves(name, wl):
    """The serial forward writes the record for every layer; the serial adjoint
    that reads it matches the recomputing one bit for bit. A one-level MGRIT
    solve (a serial solve on the finest level) writes it too."""
    c = case(wl)
    U = c.new_traj()
    rec = L.alloc_dsig(c.p)
    L.lp_serial_forward(c.p, c.K, c.b, U, dsig=rec)
    torch.cuda.synchronize()
    _check_record(c, U, rec)
    L1 = torch.zeros_like(U)
    L1[-1] = _lamN(c, U)[0]
    L2 = L1.clone()
    L.lp_serial_adjoint(c.p, c.K, c.b, U, L1)
    L.lp_serial_adjoint(c.p, c.K, c.b, U, L2, dsig=rec)
    torch.cuda.synchronize()
    assert torch.equal(L1, L2)
    mg = sched(wl, 1, levels=1)
    ws = L.alloc_workspace(c.p, mg)
    rec2 = torch.full_like(rec, 7)
    U2 = c.new_traj()
    L.lp_mgrit_forward(c.p, mg, c.K, c.b, U2, ws, history=False, dsig=rec2)
    torch.cuda.synchronize()
    assert torch.equal(U, U2) and torch.equal(rec, rec2)


def test_sigma_record_is_ignored_where_unsupported():
    """Kernels that keep no record (fp64, the identity) report a size of 0, leave
    a buffer passed anyway untouched and give the same results."""
    wl = DENSE[0][1]
    c = case(wl)
    mg = sched(wl, 2)
    ws = L.alloc_workspace(c.p, mg)
    assert L.lp_dsig_bytes(c.p) == 0
    rec = torch.full((4096,), 3, dtype=torch.uint8, device="cuda")
    U1, U2 = c.new_traj(), c.new_traj()
    L.lp_mgrit_forward(c.p, mg, c.K, c.b, U1, ws, history=False)
    L.lp_mgrit_forward(c.p, mg, c.K, c.b, U2, ws, history=False, dsig=rec)
    torch.cuda.synchronize()
    assert torch.equal(U1, U2)
    assert int(rec.min()) == 3 and int(rec.max()) == 3
    p = L.problem("f32", "dense", "identity", 8, 5, 32, h=0.1)
    assert L.lp_dsig_bytes(p) == 0
    K = torch.zeros(8, 32, 32, device="cuda")
    U = torch.zeros(9, 5, 32, device="cuda")
    L.lp_serial_forward(p, K, torch.zeros(8, 32, device="cuda"), U, dsig=L.alloc_dsig(p))


LBFGS = [
    ("tanh8_f64", WORKLOADS[1].with_overrides(N=32, B=150, max_levels=3)),
    ("tanh32_f32", WORKLOADS[5].with_overrides(N=32, B=120, n_features=20)),
    ("conv_relu12", WORKLOADS[4].with_overrides(N=16, B=6, H=12, W=12, n_features=144, max_levels=3)),
    ("srelu220", WORKLOADS[7].with_overrides(N=16, B=40, max_levels=2)),
]


def _lbfgs_runs(wl, line_search, c2=0.9):
    """The GPU trainer and the oracle's Algorithm 2 with L-BFGS on the same train /
    validation split, 6 updates of m1 = m2 = 2 iterations."""
    from paper_1812_04352_amd.one_shot import LbfgsOneShotTrainer
    from workloads import generate
    from lp_testutil import dev, prob
    Bv = max(4, wl.B // 2)
    d = generate(wl.with_overrides(B=wl.B + Bv))
    tr = {k: (v[:wl.B] if k in ("y", "onehot", "labels") else v) for k, v in d.items()}
    va = {k: d[k][wl.B:] for k in ("y", "onehot")}
    updates, m1, m2, alpha0 = 6, 2, 2, 0.5
    names = [k for k in ("L_in", "K", "b", "W", "mu") if d[k] is not None]
    params = {k: dev(d[k], wl) for k in names}
    trn = LbfgsOneShotTrainer(prob(wl), sched(wl, m1), sched(wl, m2), params, dev(tr["y"], wl), dev(tr["onehot"], wl),
                              wl.n_classes, L.OPENING[wl.opening], wl.n_features, alpha0=alpha0,
                              y_val=dev(va["y"], wl), c_val=dev(va["onehot"], wl), line_search=line_search, c2=c2)
    trn.run(updates)
    r = O.one_shot_lbfgs(tr["y"], tr["onehot"], d["L_in"], d["K"], d["b"], d["W"], d["mu"], wl.h, wl.act,
                         wl.opening, cf=wl.cf, max_levels=wl.max_levels, min_coarse=wl.min_coarse, relax=wl.relax,
                         updates=updates, m1=m1, m2=m2, alpha0=alpha0, y_val=va["y"], onehot_val=va["onehot"],
                         line_search=line_search, c2=c2)
    return trn, r, names, params, Bv


def _check_lbfgs(wl, trn, r, names, params, Bv):
    assert trn.trials == r["trials"], (trn.trials, r["trials"])
    assert trn.alphas == r["alphas"], (trn.alphas, r["alphas"])
    ltol = {"f32": 1e-4, "f64": 1e-10}[wl.dtype]
    for i, (a, b) in enumerate(zip(trn.losses, r["losses"])):
        assert abs(a - b) <= ltol * abs(b), (i, a, b)
    assert trn.losses[-1] < trn.losses[0]
    # an example on a class boundary may be decided differently in fp32 and fp64
    atol = 0.0 if wl.dtype == "f64" else 1.0 / Bv + 1e-12
    for i, (a, b) in enumerate(zip(trn.accuracies, r["accuracies"])):
        assert abs(a - b) <= atol, (i, a, b)
    for k in names:
        assert_close(params[k].cpu().numpy(), r["weights"][k], wl.dtype, f"{k} after {len(trn.losses)} updates",
                     scale={"f32": 100, "f64": 1000}[wl.dtype])


@pytest.mark.parametrize("name,wl", LBFGS, ids=[n for n, _ in LBFGS])
def test_one_shot_lbfgs_matches_oracle(name, wl):
    """Algorithm 2 with the L-BFGS Hessian approximation, line search and validation
    accuracy: per update the trial count, accepted step, loss and validation accuracy
    against the oracle's run on the same train/validation split, then the final
    weights. The line search's accept/reject test and the curvature-pair test are
    taken on each side in its own arithmetic, so the discrete decisions must agree."""
    _check_lbfgs(wl, *_lbfgs_runs(wl, "armijo"))


# c2 = 0.9 (the usual quasi-Newton value) already doubles and bisects steps here;
# c2 = 0.1 takes longer bracketing and zoom paths (fp64 only, where every discrete
# decision must agree)
WOLFE = [(LBFGS[0][0], LBFGS[0][1], 0.9), (LBFGS[1][0], LBFGS[1][1], 0.9), (LBFGS[0][0], LBFGS[0][1], 0.1)]


@pytest.mark.parametrize("name,wl,c2", WOLFE, ids=[f"{n}-c2={c}" for n, _, c in WOLFE])
def test_one_shot_lbfgs_strong_wolfe_matches_oracle(name, wl, c2):
    """The strong Wolfe line search (Section 4): the slope at each trial is the
    reduced gradient after m2 adjoint iterations at the trial state. Per update the
    loss evaluations, the accepted step and whether it met both conditions, then
    losses, accuracies and weights as above."""
    trn, r, names, params, Bv = _lbfgs_runs(wl, "wolfe", c2)
    assert trn.wolfe == r["wolfe"], (trn.wolfe, r["wolfe"])
    _check_lbfgs(wl, trn, r, names, params, Bv)


def test_one_shot_lbfgs_validation_stop():
    """The run ends at the first update whose validation accuracy reaches the target."""
    from paper_1812_04352_amd.one_shot import LbfgsOneShotTrainer
    from workloads import generate
    from lp_testutil import dev, prob
    wl = LBFGS[0][1]
    Bv = wl.B // 2
    d = generate(wl.with_overrides(B=wl.B + Bv))

    def run(target):
        params = {k: dev(d[k], wl) for k in ("L_in", "K", "b", "W", "mu")}
        t = LbfgsOneShotTrainer(prob(wl), sched(wl, 2), sched(wl, 2), params, dev(d["y"][:wl.B], wl),
                                dev(d["onehot"][:wl.B], wl), wl.n_classes, L.OPENING[wl.opening], wl.n_features,
                                alpha0=0.5, y_val=dev(d["y"][wl.B:], wl), c_val=dev(d["onehot"][wl.B:], wl),
                                target_acc=target)
        t.run(8)
        return t
    full = run(None)
    assert len(full.losses) == 8
    target = sorted(full.accuracies)[len(full.accuracies) // 2]
    first = next(i for i, a in enumerate(full.accuracies) if a >= target)
    stop = run(target)
    assert len(stop.losses) == first + 1 and stop.accuracies == full.accuracies[:first + 1]


@pytest.mark.parametrize("dtype", [torch.float32, torch.float64])
@pytest.mark.parametrize("n", [0, 1, 255, 65537, 1 << 20])
def test_vector_algebra(dtype, n):
    """lp_vec_dot (fp64 sum) and lp_vec_axpby against their definitions, over
    lengths that leave workgroups empty, ragged and strided several times."""
    r = np.random.default_rng(n + 7)
    x = r.standard_normal(n).astype(np.float32 if dtype == torch.float32 else np.float64)
    y = r.standard_normal(n).astype(x.dtype)
    xd, yd = torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda()
    out = torch.full((1 + L.LP_DOT_PARTIALS,), float("nan"), device="cuda", dtype=torch.float64)
    L.lp_vec_dot(xd, yd, out)
    ref = float(np.dot(x.astype(np.float64), y.astype(np.float64)))
    assert abs(out[0].item() - ref) <= 1e-13 * max(1.0, float(np.abs(x.astype(np.float64) @ np.abs(y))))
    L.lp_vec_axpby(yd, xd, 0.75, -1.5)
    x64, y64 = x.astype(np.float64), y.astype(np.float64)
    ref = 0.75 * x64 - 1.5 * y64
    # one rounding to the vector dtype (plus at most one in fp64 before it)
    bound = np.finfo(x.dtype).eps * (np.abs(0.75 * x64) + np.abs(1.5 * y64))
    assert np.all(np.abs(yd.cpu().numpy().astype(np.float64) - ref) <= bound)
    yd.fill_(float("nan"))
    L.lp_vec_axpby(yd, xd, 2.0, 0.0)  # b = 0 never reads y
    assert np.array_equal(yd.cpu().numpy(), (2.0 * x64).astype(x.dtype))


@pytest.mark.parametrize("name,wl", DENSE, ids=IDS)
def test_accuracy(name, wl):
    """Fraction of examples whose largest class score is their labelled class, from
    the exact network output on each side."""
    c = case(wl)
    U = c.new_traj()
    L.lp_serial_forward(c.p, c.K, c.b, U)
    acc = torch.full((1,), float("nan"), device="cuda", dtype=torch.float64)
    L.lp_accuracy(c.p, wl.n_classes, U[-1], c.W, c.mu, c.onehot, acc, L.alloc_workspace(c.p))
    Uref = O.serial_forward(c.u0_ref, c.d["K"], c.d["b"], wl.h, wl.act)
    ref = O.accuracy(Uref[-1], c.d["W"], c.d["mu"], c.d["labels"])
    slack = 0.0 if wl.dtype == "f64" else 2.0 / wl.B  # an example on a class boundary
    assert abs(acc.item() - ref) <= slack + 1e-15, (acc.item(), ref)


@pytest.mark.gpu
@pytest.mark.parametrize("q,nc,B", [(32, 1, 45), (32, 3, 257), (32, 17, 45), (32, 64, 45), (220, 10, 33),
                                    (220, 64, 7), (8, 5, 1), (1152, 10, 37), (1152, 64, 5), (6272, 10, 9)])
def test_loss_head_class_counts(q, nc, B):
    """Softmax head, loss, terminal adjoint and classifier gradient against the
    oracle (Section 2.1 loss, Section 2.3 terminal condition) over class counts
    that set the lanes per example (1 .. 64) and batches that leave the last
    workgroup partly empty; width 220 with 64 classes still stages W in LDS, and
    the widths 1152 and 6272 (convolution states) take the path that does not,
    one wave per example."""
    rng = np.random.default_rng(1000 * q + nc + B)
    uN = rng.standard_normal((B, q)).astype(np.float32)
    W = (0.3 * rng.standard_normal((nc, q))).astype(np.float32)
    mu = (0.1 * rng.standard_normal(nc)).astype(np.float32)
    onehot = np.eye(nc, dtype=np.float32)[rng.integers(0, nc, B)]
    if q % 72 == 0 or q == 6272:  # a convolution state: 8 channels of an H x H image
        hw = int(round((q // 8) ** 0.5))
        p = L.problem("f32", "conv3x3", "relu", N=4, B=B, C=8, H=hw, W=hw, h=0.25)
    else:
        p = L.problem("f32", "dense", "relu", N=4, B=B, C=q, h=0.25)
    g = {k: torch.from_numpy(v).cuda() for k, v in dict(uN=uN, W=W, mu=mu, c=onehot).items()}
    J = torch.zeros(1, device="cuda", dtype=torch.float64)
    lamN, dW, dmu = torch.empty_like(g["uN"]), torch.empty_like(g["W"]), torch.empty_like(g["mu"])
    L.lp_loss_terminal(p, nc, g["uN"], g["W"], g["mu"], g["c"], J, lamN, dW, dmu, L.alloc_workspace(p))
    Jr, lamNr, dWr, dmur = O.loss_terminal(uN, W, mu, onehot)
    assert abs(J.item() - Jr) <= 1e-5 * max(abs(Jr), 1e-30)
    assert_close(lamN.cpu().numpy(), lamNr, "f32", "lamN")
    assert_close(dW.cpu().numpy(), dWr, "f32", "dW")
    assert_close(dmu.cpu().numpy(), dmur, "f32", "dmu")


CPT_CASES = [DENSE[1], DENSE[2], DENSE[3], ("tanh64_l3", WORKLOADS[3].with_overrides(N=64, B=77, max_levels=3))]


@pytest.mark.parametrize("name,wl", CPT_CASES, ids=[n for n, _ in CPT_CASES])
@pytest.mark.parametrize("relax", ["F", "FCF"])
def test_cpoint_storage(name, wl, relax):
    """C-point storage (Section 3.2 remark: states stored or recomputed). The
    forward keeps the C-points only, the adjoint and the gradient recompute the
    F-point states by forward steps from them. The C-points, the adjoint iterate,
    the residual histories and the gradient must equal those of full storage bit
    for bit (the recompute repeats the forward F-relaxation's arithmetic), and the
    adjoint and gradient match the oracle run on the oracle's expansion of its own
    C-points."""
    c = case(wl)
    cf = wl.cf
    mgA = sched(wl, 2, relax=relax)
    mgC = L.mgrit(cf=cf, max_levels=wl.max_levels, min_coarse=wl.min_coarse, relax=relax, max_iter=2,
                  storage="cpoints")
    ws = L.alloc_workspace(c.p, mgC)
    U = c.new_traj()
    _, hA = L.lp_mgrit_forward(c.p, mgA, c.K, c.b, U, ws)
    Uc = torch.zeros((wl.N // cf + 1,) + tuple(U.shape[1:]), device="cuda", dtype=U.dtype)
    Uc[0] = c.u0
    _, hC = L.lp_mgrit_forward(c.p, mgC, c.K, c.b, Uc, ws)
    assert hA == hC
    assert torch.equal(Uc, U[::cf].contiguous())
    lamN = _lamN(c, U)[0]
    LA = torch.zeros_like(U)
    LA[-1] = lamN
    LC = LA.clone()
    _, gA = L.lp_mgrit_adjoint(c.p, mgA, c.K, c.b, U, LA, ws)
    _, gC = L.lp_mgrit_adjoint(c.p, mgC, c.K, c.b, Uc, LC, ws)
    assert gA == gC
    assert torch.equal(LA, LC)
    dKA, dbA = torch.empty_like(c.K), torch.empty_like(c.b)
    L.lp_gradient(c.p, c.K, c.b, U, LA, dKA, dbA, ws)
    dKC, dbC = torch.empty_like(c.K), torch.empty_like(c.b)
    L.lp_gradient_cpoints(c.p, cf, c.K, c.b, Uc, LC, dKC, dbC, ws)
    assert torch.equal(dKA, dKC) and torch.equal(dbA, dbC)
    # oracle: C-points of its own MGRIT iterate, expanded, then the adjoint and gradient
    Ur, _, _ = O.mgrit_forward(c.ref_traj(), c.d["K"], c.d["b"], wl.h, wl.act, cf=cf, max_levels=wl.max_levels,
                               min_coarse=wl.min_coarse, relax=relax, max_iter=2)
    assert_close(Uc.cpu().numpy(), Ur[::cf], wl.dtype, "C-points")
    Ue = O.expand_cpoints(Ur[::cf], c.d["K"], c.d["b"], wl.h, wl.act, cf)
    Lr = np.zeros_like(Ue)
    Lr[-1] = O.loss_terminal(Ue[-1], c.d["W"], c.d["mu"], c.d["onehot"])[1]
    Lr, _, _ = O.mgrit_adjoint(Ue, Lr, c.d["K"], c.d["b"], wl.h, wl.act, cf=cf, max_levels=wl.max_levels,
                               min_coarse=wl.min_coarse, relax=relax, max_iter=2)
    assert_close(LC.cpu().numpy(), Lr, wl.dtype, "Lam from C-points")
    dKr, dbr = O.gradient(Ue, Lr, c.d["K"], c.d["b"], wl.h, wl.act)
    if wl.act != "relu":
        assert_close(dKC.cpu().numpy(), dKr, wl.dtype, "dK from C-points")
        assert_close(dbC.cpu().numpy(), dbr, wl.dtype, "db from C-points")
    # warm start from the stored C-points: one more iteration, same on both sides
    mgA.warm_start = mgC.warm_start = 1
    mgA.max_iter = mgC.max_iter = 1
    L.lp_mgrit_forward(c.p, mgA, c.K, c.b, U, ws)
    L.lp_mgrit_forward(c.p, mgC, c.K, c.b, Uc, ws)
    assert torch.equal(Uc, U[::cf].contiguous())


# More batch tiles than a width-64 sweep's workgroup budget (about 2048 workgroups):
# N = 128 gives 32 finest intervals, so 64 workgroups per interval each walk about
# 11 of the 701 tiles (and request the next tile's rows during the current one's
# steps); on the 8 intervals of level 1, 256 workgroups walk about 3 tiles each.
# The last tile holds 29 examples.
WALK_CASES = [
    ("tanh64_walk", WORKLOADS[3].with_overrides(N=128, B=64 * 700 + 29, max_levels=3)),
    ("relu64_walk", WORKLOADS[3].with_overrides(act="relu", N=128, B=64 * 700 + 29, max_levels=3)),
]


@pytest.mark.parametrize("name,wl", WALK_CASES, ids=[n for n, _ in WALK_CASES])
def test_tile_walking_sweeps(name, wl):
    """Width-64 interval sweeps whose workgroups walk several batch tiles, the
    launch configuration of the deep workload at full size. Sampled examples (the
    first ones, the ragged last tile, both sides of tile boundaries that are a
    walk step apart, seeded others) against the oracle run on those examples
    alone (examples are independent in the solves; the oracle's terminal value
    is rescaled from the sample mean to the batch mean). The adjoint linearised
    through the sigma' record, through recomputed sigma', and from C-point
    storage must agree bit for bit."""
    c = Case(wl)
    B, cf = wl.B, wl.cf
    r = np.random.default_rng(7)
    S = {0, 1, 2, 3, B - 29, B - 2, B - 1, 64 * 64 - 1, 64 * 64, 64 * 128, 64 * 256 - 1, 64 * 256}
    S = np.array(sorted(S | set(r.choice(B, 12, replace=False).tolist())))
    Sg = torch.from_numpy(S).cuda()
    mg = sched(wl, 2)
    mgC = L.mgrit(cf=cf, max_levels=wl.max_levels, min_coarse=wl.min_coarse, relax=wl.relax, max_iter=2,
                  storage="cpoints")
    ws = L.alloc_workspace(c.p, mgC)
    rec = L.alloc_dsig(c.p)
    U = c.new_traj()
    _, hF = L.lp_mgrit_forward(c.p, mg, c.K, c.b, U, ws, dsig=rec)
    Ur = np.zeros((wl.N + 1, len(S), wl.q))
    Ur[0] = c.u0_ref[S]
    Ur, _, _ = O.mgrit_forward(Ur, c.d["K"], c.d["b"], wl.h, wl.act, cf=cf, max_levels=wl.max_levels,
                               min_coarse=wl.min_coarse, relax=wl.relax, max_iter=2)
    assert_close(U.index_select(1, Sg).cpu().numpy(), Ur, wl.dtype, f"{name} U sample")
    Uc = torch.zeros((wl.N // cf + 1, B, wl.q), device="cuda", dtype=U.dtype)
    Uc[0] = c.u0
    _, hC = L.lp_mgrit_forward(c.p, mgC, c.K, c.b, Uc, ws)
    assert hC == hF
    assert torch.equal(Uc, U[::cf].contiguous())

    lamN = _lamN(c, U)[0]
    LR = torch.zeros_like(U)
    LR[-1] = lamN
    LP, LC = LR.clone(), LR.clone()
    _, hR = L.lp_mgrit_adjoint(c.p, mg, c.K, c.b, U, LR, ws, dsig=rec)
    _, hP = L.lp_mgrit_adjoint(c.p, mg, c.K, c.b, U, LP, ws)
    _, hCa = L.lp_mgrit_adjoint(c.p, mgC, c.K, c.b, Uc, LC, ws)
    assert hR == hP == hCa
    assert torch.equal(LR, LP) and torch.equal(LR, LC)
    Lr = np.zeros_like(Ur)
    Lr[-1] = O.loss_terminal(Ur[-1], c.d["W"], c.d["mu"], c.d["onehot"][S])[1] * (len(S) / B)
    Lr, _, _ = O.mgrit_adjoint(Ur, Lr, c.d["K"], c.d["b"], wl.h, wl.act, cf=cf, max_levels=wl.max_levels,
                               min_coarse=wl.min_coarse, relax=wl.relax, max_iter=2)
    assert_close(LR.index_select(1, Sg).cpu().numpy(), Lr, wl.dtype, f"{name} Lam sample")
