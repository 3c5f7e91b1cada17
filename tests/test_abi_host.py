"""The C-ABI library on the CPU host (no GPU): it loads, exports every symbol the
header declares, and its host-side argument checks return the documented
status codes before any device work is enqueued."""
import ctypes
import os
import re

import pytest

from paper_1812_04352_amd import lp as L

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def header_symbols():
    text = open(os.path.join(ROOT, "include", "lp.h")).read()
    return sorted(set(re.findall(r"\b(lp_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    lib = L.load()
    declared = header_symbols()
    assert declared, "no declarations found"
    for name in declared:
        assert hasattr(lib, name), name
    assert sorted(L.EXPORTS) == declared


def test_version_and_status_strings():
    lib = L.load()
    assert lib.lp_abi_version() == L.LP_ABI_VERSION
    for s in range(6):
        assert lib.lp_status_string(s)
    assert lib.lp_status_string(99) == b"unknown status"


def _p(**kw):
    base = dict(dtype="f32", layer="dense", act="tanh", N=64, B=100, C=32, h=0.1)
    base.update(kw)
    return L.problem(**base)


FAKE = ctypes.c_void_p(0x1000)  # never dereferenced: every case fails host validation first


def test_problem_validation_codes():
    lib = L.load()
    null = ctypes.c_void_p(0)
    assert lib.lp_serial_forward(None, FAKE, FAKE, FAKE, None, null) == L.LP_EINVAL
    p = _p()
    p.abi_version = 7
    assert lib.lp_serial_forward(ctypes.byref(p), FAKE, FAKE, FAKE, None, null) == L.LP_EINVAL
    assert b"abi_version" in lib.lp_last_error()
    for bad in (dict(N=0), dict(B=-1), dict(h=0.0), dict(h=float("nan")), dict(C=0)):
        assert lib.lp_serial_forward(ctypes.byref(_p(**bad)), FAKE, FAKE, FAKE, None, null) == L.LP_EINVAL, bad
    p = _p()
    p.act = 9
    assert lib.lp_serial_forward(ctypes.byref(p), FAKE, FAKE, FAKE, None, null) == L.LP_EINVAL
    # a width with no kernel is a valid but unsupported problem
    assert lib.lp_serial_forward(ctypes.byref(_p(C=48)), FAKE, FAKE, FAKE, None, null) == L.LP_EUNSUPPORTED
    # NULL arrays
    assert lib.lp_serial_forward(ctypes.byref(_p()), None, FAKE, FAKE, None, null) == L.LP_EINVAL


def test_mgrit_validation_codes():
    lib = L.load()
    p = _p(N=48)
    hist = (ctypes.c_double * 4)()
    it = ctypes.c_int32(-1)

    def call(mg, ws=FAKE, nbytes=1 << 40):
        return lib.lp_mgrit_forward(ctypes.byref(p), ctypes.byref(mg), FAKE, FAKE, FAKE, None, ws, nbytes, hist,
                                    ctypes.byref(it), None)

    assert call(L.mgrit(cf=1)) == L.LP_EINVAL
    assert call(L.mgrit(max_iter=0)) == L.LP_EINVAL
    assert call(L.mgrit(max_levels=0)) == L.LP_EINVAL
    # 48 -> 12 -> 3 is fine with cf = 4, but 12 is not divisible by 5 and 48 % 5 != 0
    assert call(L.mgrit(cf=5, max_levels=2)) == L.LP_EINVAL
    assert b"divisible" in lib.lp_last_error()
    assert call(L.mgrit(cf=4, max_levels=4)) == L.LP_EINVAL  # 48 -> 12 -> 3 -> (3 % 4 != 0)
    # workspace checks happen before any launch
    mg = L.mgrit(cf=4, max_levels=3)
    need = L.lp_workspace_bytes(p, mg)
    assert call(mg, ws=None) == L.LP_EWORKSPACE
    assert call(mg, ws=ctypes.c_void_p(0x1001)) == L.LP_EWORKSPACE  # misaligned
    assert call(mg, nbytes=need - 1) == L.LP_EWORKSPACE
    # adjoint: U and Lam must not alias
    assert lib.lp_mgrit_adjoint(ctypes.byref(p), ctypes.byref(mg), FAKE, FAKE, FAKE, None, FAKE, FAKE, need, hist,
                                ctypes.byref(it), None) == L.LP_EINVAL


def test_workspace_sizes():
    # config-3 shaped problem: 2048 -> 512 -> 128 -> 32 -> 8 with FCF staging
    p = L.problem("f32", "dense", "tanh", 2048, 16384, 64, h=1 / 256)
    mg = L.mgrit(cf=4, max_levels=16, min_coarse=8, max_iter=20)
    slice_bytes = 16384 * 64 * 4
    coarse = sum(n + 1 for n in (512, 128, 32, 8)) * 2 * slice_bytes
    # relaxed C-points of every non-coarsest level, two buffers on the finest one
    staging = (sum(n + 1 for n in (512, 128, 32, 8)) + 513) * slice_bytes
    got = L.lp_workspace_bytes(p, mg)
    assert coarse + staging <= got <= coarse + staging + (64 << 20)
    # F-relaxation needs no staging
    assert L.lp_workspace_bytes(p, L.mgrit(cf=4, max_levels=16, min_coarse=8, relax="F", max_iter=20)) < got
    with pytest.raises(L.LpError):
        L.lp_workspace_bytes(L.problem("f32", "dense", "tanh", 2048, 16384, 48, h=0.1))


def test_dsig_record_sizes(monkeypatch):
    # one bit per value for ReLU (one byte at width 220), fp32 for smooth activations,
    # none for the identity
    assert L.lp_dsig_bytes(_p(act="relu")) == 64 * 100 * 32 // 8
    assert L.lp_dsig_bytes(_p(act="relu", C=64)) == 64 * 100 * 64 // 8
    assert L.lp_dsig_bytes(_p(act="relu", C=220)) == 64 * 100 * 220
    assert L.lp_dsig_bytes(_p(act="tanh")) == 64 * 100 * 32 * 4
    assert L.lp_dsig_bytes(_p(act="smoothrelu", C=64)) == 64 * 100 * 64 * 4
    assert L.lp_dsig_bytes(_p(act="identity")) == 0
    # kernels that keep no record
    assert L.lp_dsig_bytes(_p(act="smoothrelu", dtype="f64")) == 0
    assert L.lp_dsig_bytes(_p(C=8)) == 0
    # conv: one block per (layer, example) in the kernels' tile order: ReLU, one 32-bit
    # word of decision bits per lane of every wave (7 tiles x 4 values); smooth
    # activations, four fp32 values per lane of every tile. 12 x 12 -> 72 pair-pixels,
    # 5 tiles of 16, one wave of 7 tiles; 28 x 28 -> 392 pair-pixels, 25 tiles, 4 waves
    assert L.lp_dsig_bytes(L.problem("f32", "conv3x3", "relu", 16, 5, 8, H=12, W=12, h=0.1)) == 16 * 5 * 1 * 64 * 4
    assert L.lp_dsig_bytes(L.problem("f32", "conv3x3", "relu", 16, 5, 8, H=28, W=28, h=0.1)) == 16 * 5 * 4 * 64 * 4
    assert L.lp_dsig_bytes(L.problem("f32", "conv3x3", "tanh", 16, 5, 8, H=28, W=28, h=0.1)) == 16 * 5 * 28 * 64 * 16
    assert L.lp_dsig_bytes(L.problem("f64", "conv3x3", "tanh", 16, 5, 8, H=28, W=28, h=0.1)) == 0
    monkeypatch.setenv("LP_DENSE_PATH", "valu")
    assert L.lp_dsig_bytes(_p()) == 0
    monkeypatch.delenv("LP_DENSE_PATH")
    bad = _p()
    bad.abi_version = 1
    assert L.lp_dsig_bytes(bad) == 0


def test_helper_validation_codes():
    lib = L.load()
    p = _p()
    J = ctypes.c_void_p(0x2000)
    big = 1 << 40
    for nc in (0, 65):
        assert lib.lp_loss_terminal(ctypes.byref(p), nc, FAKE, FAKE, FAKE, FAKE, J, FAKE, FAKE, FAKE, FAKE, big,
                                    None) == L.LP_EINVAL
    assert lib.lp_loss_terminal(ctypes.byref(p), 10, FAKE, FAKE, FAKE, FAKE, J, FAKE, FAKE, FAKE, FAKE, 1024,
                                None) == L.LP_EWORKSPACE
    assert lib.lp_loss_terminal(ctypes.byref(p), 10, FAKE, FAKE, FAKE, FAKE, J, FAKE, FAKE, FAKE, None, big,
                                None) == L.LP_EWORKSPACE
    assert lib.lp_open_forward(ctypes.byref(p), 5, 3, FAKE, FAKE, FAKE, None) == L.LP_EINVAL
    assert lib.lp_open_grad(ctypes.byref(p), L.LP_OPEN_IDENTITY, 3, FAKE, FAKE, FAKE, FAKE, None) == L.LP_EINVAL
    assert lib.lp_sgd_update(7, 10, 0.1, FAKE, FAKE, None) == L.LP_EINVAL
    assert lib.lp_residual_norm(ctypes.byref(p), 5, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 30,
                                ctypes.byref(ctypes.c_double()), None) == L.LP_EINVAL


def test_binding_refuses_cpu_tensors():
    import torch
    p = _p(N=4, B=3, C=8)
    K = torch.zeros(4, 8, 8)
    with pytest.raises(ValueError):
        L.lp_serial_forward(p, K, torch.zeros(4, 8), torch.zeros(5, 3, 8))


def test_cycle_and_relaxation_options(monkeypatch):
    """F-cycles and FCFCF are accepted; unknown values are LP_EINVAL; FCFCF needs
    one more staging buffer on every coarse non-coarsest level."""
    lib = L.load()
    p = L.problem("f32", "dense", "relu", 256, 64, 32, h=0.04)
    fcf = L.lp_workspace_bytes(p, L.mgrit(4, 4, 1, "FCF", 2))
    fcfcf = L.lp_workspace_bytes(p, L.mgrit(4, 4, 1, "FCFCF", 2))
    slice_ = 64 * 32 * 4
    # levels 256 -> 64 -> 16 -> 4: the extra buffers sit on levels 1 and 2 (17 and 5 slices)
    assert fcfcf - fcf >= (17 + 5) * slice_
    assert L.lp_workspace_bytes(p, L.mgrit(4, 4, 1, "FCF", 2, cycle="F")) == fcf
    m = L.mgrit(4, 4, 1, "FCF", 2)
    m.cycle = 7
    assert lib.lp_workspace_bytes(ctypes.byref(p), ctypes.byref(m)) == 0
    m = L.mgrit(4, 4, 1, "FCF", 2)
    m.relax = 3
    assert lib.lp_workspace_bytes(ctypes.byref(p), ctypes.byref(m)) == 0


def test_loss_workspace_follows_the_head_path():
    """The loss reserves partials for the path it takes: one row per head
    workgroup when W and u^N fit in LDS (dense width 32), one row per 16 examples
    otherwise (the convolutional head, q = 6272), for every class count <= 64."""
    lib = L.load()

    def up(x):
        return (x + 255) // 256 * 256

    conv = L.problem("f32", "conv3x3", "relu", 512, 1024, 8, H=28, W=28, h=5 / 512)
    q, B = 8 * 28 * 28, 1024
    unstaged64 = up(B * 64 * 8) + up(B * 8) + up((B // 16) * 64 * (q + 1) * 8)
    got = L.lp_workspace_bytes(conv)
    assert unstaged64 <= got <= unstaged64 + (128 << 20)  # the gradient's partials are smaller
    assert got < 300 << 20  # not the staged size (four times as many rows)
    # the loss itself checks the size for its class count
    need10 = up(B * 10 * 8) + up(B * 8) + up((B // 16) * 10 * (q + 1) * 8)
    J = ctypes.c_void_p(0x2000)
    assert lib.lp_loss_terminal(ctypes.byref(conv), 10, FAKE, FAKE, FAKE, FAKE, J, FAKE, FAKE, FAKE, FAKE,
                                need10 - 1, None) == L.LP_EWORKSPACE
    # dense width 32, 16 classes: staged head, 16 examples per workgroup, rows of nc (q+1) + 1
    dense = L.problem("f32", "dense", "relu", 8, 4096, 32, h=0.1)
    need16 = up(4096 * 16 * 8) + up(4096 * 8) + up((4096 // 16) * (16 * 33 + 1) * 8)
    assert lib.lp_loss_terminal(ctypes.byref(dense), 16, FAKE, FAKE, FAKE, FAKE, J, FAKE, FAKE, FAKE, FAKE,
                                need16 - 1, None) == L.LP_EWORKSPACE
    assert L.lp_workspace_bytes(dense) >= need16


def test_residual_norm_noalloc_limits():
    """The allocation-free residual norm checks its arguments and its static
    scratch limit (2^21 partials) on the host, before any device work."""
    lib = L.load()
    out = ctypes.byref(ctypes.c_double())
    # (N + 1) * ceil(B / 32) partials: 4096 * 512 = 2^21 fits, 4097 * 512 does not
    big = L.problem("f32", "dense", "tanh", 4096, 16384, 64, h=1e-3)
    assert lib.lp_residual_norm_noalloc(ctypes.byref(big), L.LP_STATE, FAKE, FAKE, FAKE, None, out,
                                        None) == L.LP_EWORKSPACE
    assert b"static scratch" in lib.lp_last_error()
    conv = L.problem("f32", "conv3x3", "relu", 2048, 1024, 8, H=28, W=28, h=1e-3)  # 2049 * 1024 partials
    assert lib.lp_residual_norm_noalloc(ctypes.byref(conv), L.LP_STATE, FAKE, FAKE, FAKE, None, out,
                                        None) == L.LP_EWORKSPACE
    p = _p()
    assert lib.lp_residual_norm_noalloc(ctypes.byref(p), 5, FAKE, FAKE, FAKE, FAKE, out, None) == L.LP_EINVAL
    assert lib.lp_residual_norm_noalloc(ctypes.byref(p), L.LP_ADJOINT, FAKE, FAKE, FAKE, None, out,
                                        None) == L.LP_EINVAL
    assert lib.lp_residual_norm_noalloc(ctypes.byref(p), L.LP_STATE, FAKE, FAKE, FAKE, None, None,
                                        None) == L.LP_EINVAL


def test_cpoint_storage_validation():
    """C-point storage is accepted for the fp32 matrix-core widths with cf = 4 and
    two or more levels, refused (LP_EUNSUPPORTED) elsewhere; its workspace also
    covers the gradient's recompute block."""
    lib = L.load()
    hist = (ctypes.c_double * 4)()
    it = ctypes.c_int32(0)

    def fwd(p, mg):
        return lib.lp_mgrit_forward(ctypes.byref(p), ctypes.byref(mg), FAKE, FAKE, FAKE, None, None, 0, hist,
                                    ctypes.byref(it), None)

    p = L.problem("f32", "dense", "tanh", 2048, 16384, 64, h=1 / 256)
    mg = L.mgrit(cf=4, max_levels=5, min_coarse=8, max_iter=2, storage="cpoints")
    full = L.lp_workspace_bytes(p, L.mgrit(cf=4, max_levels=5, min_coarse=8, max_iter=2))
    need = L.lp_workspace_bytes(p, mg)
    assert need >= 64 * 4 * 16384 * 64 * 4 and need >= full
    assert fwd(p, mg) == L.LP_EWORKSPACE  # valid schedule: only the (absent) workspace is refused
    assert fwd(p, L.mgrit(cf=2, max_levels=5, max_iter=2, storage="cpoints")) == L.LP_EUNSUPPORTED
    assert fwd(p, L.mgrit(cf=4, max_levels=1, max_iter=2, storage="cpoints")) == L.LP_EINVAL
    for q in (_p(C=8), _p(dtype="f64")):
        assert fwd(q, L.mgrit(cf=4, max_levels=2, max_iter=2, storage="cpoints")) == L.LP_EUNSUPPORTED
    bad = L.mgrit(cf=4, max_levels=2, max_iter=2)
    bad.storage = 2
    assert fwd(p, bad) == L.LP_EINVAL
    out = ctypes.c_void_p(0x3000)
    assert lib.lp_gradient_cpoints(ctypes.byref(p), 2, FAKE, FAKE, FAKE, FAKE, out, out, FAKE, 1 << 40,
                                   None) == L.LP_EUNSUPPORTED
    assert lib.lp_gradient_cpoints(ctypes.byref(p), 4, FAKE, FAKE, FAKE, FAKE, out, out, FAKE, 1024,
                                   None) == L.LP_EWORKSPACE
