"""Host-side logic of the benchmark (no GPU): kernel-kind parsing of demangled
names, the levels a V- or F-cycle visits, the algorithmic byte and flop model's
launch counts and closed forms, the sigma' record sizes, and the per-family
source hashes that mark counter summaries stale."""
import bench
from workloads import WORKLOADS


def test_kernel_kind_parses_every_family():
    kk = bench.kernel_kind
    # dense matrix-core kernels: per-step (mode is the 2nd argument) and interval-resident
    assert kk("void lp::mfma::k_fwd<32, 0, 4, 16, false>(lp::SweepArgs)") == "fwd_fc"
    assert kk("void lp::mfma::k_adj<64, 1, 4, 16, true>(lp::SweepArgs)") == "adj_fres"
    assert kk("void lp::mfma::k_fwd<32, 3, 1, 16, false>(lp::SweepArgs)") == "fwd_coarsest"
    assert kk("void lp::mfma::k_adj_iv<32, 2, 4, true, true, false>(lp::SweepArgs)") == "adj_corrf"
    assert kk("void lp::mfma::k_fwd_iv<64, 1, 4, false, true>(lp::SweepArgs)") == "fwd_fres"
    # vector-ALU kernels: mode is the 3rd argument; the serial kernels are the coarsest kind
    assert kk("void lp::dense::k_adj_sweep<double, 8, 1>(lp::SweepArgs)") == "adj_fres"
    assert kk("void lp::dense::k_fwd_serial<double, 8>(lp::SerialArgs)") == "fwd_coarsest"
    # convolution (mode first) and the width-220 family (mode second)
    assert kk("void lp::conv::k_adj<1, 28, 28, 1, false>(lp::SweepArgs, lp::conv::SGeo)") == "adj_fres"
    assert kk("void lp::conv::k_fwd<3, 28, 28, 0, true>(lp::SweepArgs, lp::conv::SGeo)") == "fwd_coarsest"
    assert kk("void lp::wide::k_adj<220, 0, true>(lp::SweepArgs)") == "adj_fc"
    assert kk("void lp::wide::k_fwd<220, 2, false>(lp::SweepArgs)") == "fwd_corrf"
    # gradients of every family; anything else is not a traced kind
    assert kk("void lp::mfma::k_grad<32, false>(lp::GradArgs)") == "gradient"
    assert kk("void lp::dense::k_grad_partial<double, 8>(lp::GradArgs)") == "gradient"
    assert kk("void lp::wide::k_grad<220, true>(lp::GradArgs)") == "gradient"
    assert kk("lp::(anonymous namespace)::k_norm_reduce(double const*, int, double*)") is None
    assert kk("__amd_rocclr_copyBuffer") is None


def test_level_visits_follow_the_cycle_recursion():
    for L in range(1, 7):
        assert bench.level_visits(L, "V") == [1] * L
    # F-cycle: a coarse problem is solved by an F-cycle then a V-cycle one level
    # down, the V-cycle left out above the coarsest level
    assert bench.level_visits(2, "F") == [1, 1]
    assert bench.level_visits(3, "F") == [1, 2, 2]
    assert bench.level_visits(4, "F") == [1, 2, 3, 3]
    assert bench.level_visits(5, "F") == [1, 2, 3, 4, 4]


def _wl(**kw):
    return WORKLOADS[2].with_overrides(**kw)


def test_kernel_model_launch_counts():
    wl = _wl(N=64, B=32, cf=4, max_levels=2, relax="FCF")  # levels 64, 16
    launches = {k: bench.kernel_model(wl, k, 3, 3)[2] for k in bench.KIND_NAMES[:9]}
    # per iteration one FC and one FRES sweep on the finest level and one coarsest
    # solve; the finest correction sweep runs once per solve (FCF defers it)
    assert launches["fwd_fc"] == launches["adj_fc"] == 3
    assert launches["fwd_fres"] == launches["adj_fres"] == 3
    assert launches["fwd_coarsest"] == launches["adj_coarsest"] == 3
    assert launches["fwd_corrf"] == launches["adj_corrf"] == 1
    assert launches["gradient"] == 1
    # F relaxation: no FC sweeps; FCFCF: two per level visit
    assert bench.kernel_model(_wl(N=64, B=32, max_levels=2, relax="F"), "fwd_fc", 3, 3)[2] == 0
    assert bench.kernel_model(_wl(N=64, B=32, max_levels=2, relax="FCFCF"), "fwd_fc", 3, 3)[2] == 6
    # three levels: the middle level's correction is not deferred
    assert bench.kernel_model(_wl(N=64, B=32, max_levels=3), "fwd_corrf", 3, 3)[2] == 1 + 3


def test_kernel_model_closed_forms():
    wl = _wl(N=64, B=32, cf=4, max_levels=2, relax="F")
    q, B, N, e = wl.q, wl.B, wl.N, 4
    row, nw = B * q * e, q * q + q
    # gradient without a record: U[n], Lam[n+1] and K_n read, dK and db written; 4 q^2 per layer and example
    assert bench.kernel_model(wl, "gradient", 1, 1) == (2 * N * row + 2 * N * nw * e, 4.0 * q * q * B * N, 1)
    # one forward FRES sweep, two levels: per interval 2 C-points read + G' written +
    # X' ... (no next-level trajectory below the coarsest: xn = 0), c steps
    Nc = N // wl.cf
    byts, flops, n = bench.kernel_model(wl, "fwd_fres", 1, 1)
    assert n == 1 and byts == Nc * 3 * row + N * nw * e
    assert flops == Nc * wl.cf * 2 * q * q * B
    # the coarsest forward solve: 1 + N_L G rows read and N_L rows written, N_L steps
    NL = N // wl.cf
    byts, flops, n = bench.kernel_model(wl, "fwd_coarsest", 1, 1)
    assert byts == (1 + NL + NL) * row + NL * nw * e and flops == NL * 2 * q * q * B
    # with a byte record the adjoint reads a quarter row per step instead of a
    # primal row and takes one product instead of two
    a0 = bench.kernel_model(wl, "adj_coarsest", 1, 1, rec=0)
    a1 = bench.kernel_model(wl, "adj_coarsest", 1, 1, rec=1)
    assert a0[0] - a1[0] == NL * (row - B * q)
    assert a0[1] == 2 * a1[1]


def test_record_bytes():
    assert bench.record_bytes(WORKLOADS[1]) == 0          # fp64 keeps no record
    assert bench.record_bytes(WORKLOADS[2]) == 0.125      # ReLU: one bit per value
    assert bench.record_bytes(WORKLOADS[3]) == 4          # tanh: fp32
    assert bench.record_bytes(WORKLOADS[4]) == 0.125      # conv ReLU: one bit per value
    assert bench.record_bytes(WORKLOADS[7]) == 4          # width 220, smoothed ReLU
    assert bench.record_bytes(WORKLOADS[2].with_overrides(C=16)) == 0   # a vector-ALU width
    assert bench.record_bytes(WORKLOADS[2].with_overrides(act="identity")) == 0


def test_source_hashes_are_per_family_and_stable():
    h = bench.source_hash
    fams = [h("lp::conv::k"), h("lp::mfma::k"), h("lp::dense::k"), h("lp::wide::k"), h()]
    assert len(set(fams)) == len(fams)
    assert h("void lp::conv::k_adj<1>") == h("lp::conv::") and h() == h("")


def test_cpu_baseline_legs():
    """The CPU baseline times both oracle legs (MGRIT iteration, layer-serial
    forward + backward + gradient) in the workload's dtype on the full batch of
    the small dense workloads and on a leading slice of the large ones."""
    from workloads import WORKLOADS
    assert bench.cpu_sample_size(WORKLOADS[2]) == WORKLOADS[2].B
    assert bench.cpu_sample_size(WORKLOADS[5]) == WORKLOADS[5].B
    assert bench.cpu_sample_size(WORKLOADS[3]) == 1024
    assert bench.cpu_sample_size(WORKLOADS[4]) == 8
    r = bench.cpu_baseline(WORKLOADS[2].with_overrides(N=16, B=64), budget_s=0.2)
    assert r["value"] > 0 and r["layer_serial"]["value"] > 0 and r["cores"] >= 1
    assert "full batch" in r["sample"] and "f32" in r["sample"]


def test_kernel_model_cpoint_storage():
    """With C-point storage the finest adjoint sweeps read one primal row per
    interval instead of c, and the final finest forward correction moves three rows
    per interval with no products."""
    from workloads import WORKLOADS
    wl = WORKLOADS[3].with_overrides(N=64, B=256, max_levels=2)
    full = bench.kernel_model(wl, "adj_fc", 1, 1)
    cpt = bench.kernel_model(wl, "adj_fc", 1, 1, cpt=True)
    row = wl.B * wl.q * 4
    assert full[2] == cpt[2] and full[1] == cpt[1]
    assert full[0] - cpt[0] == (wl.N // wl.cf) * (wl.cf - 1) * row
    b, f, n = bench.kernel_model(wl, "fwd_corrf", 1, 1, cpt=True)
    assert (b, f, n) == ((wl.N // wl.cf) * 3 * row, 0, 1)
