// Host side of the C ABI (include/lp.h): argument checks, the MGRIT level
// hierarchy carved out of the caller's workspace, and the V-cycle schedule of
// Algorithm 1 (Section 3.1) applied recursively, for the state and the adjoint
// systems. Every step of the computation runs in the HIP kernels; this file
// only validates, lays out memory and enqueues launches on the caller's stream.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/lp.h"
#include "lp_internal.h"

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

int hip_fail(hipError_t e, const char* what) {
  if (e == hipErrorNotSupported) return fail(LP_EUNSUPPORTED, "%s: no kernel for this shape", what);
  return fail(LP_EHIP, "%s: %s", what, hipGetErrorString(e));
}

#define LP_TRY(expr, what)                       \
  do {                                           \
    hipError_t _e = (expr);                      \
    if (_e != hipSuccess) return hip_fail(_e, what); \
  } while (0)

// ---------------------------------------------------------------- tracing
// Event pairs around launches of the enabled kinds; summed on lp_trace_read.
struct TraceRec {
  int kind, level;
  hipEvent_t a, b;
};
std::mutex g_trace_mu;
uint32_t g_trace_mask = 0;
std::vector<TraceRec> g_trace;
std::vector<hipEvent_t> g_event_pool;
size_t g_pool_used = 0;
long g_trace_dropped = 0;
constexpr size_t kTraceMax = 65536;

}  // namespace

lp::LaunchEvents& lp::launch_events() {
  static thread_local LaunchEvents e;
  return e;
}

namespace {

hipEvent_t pool_event() {
  if (g_pool_used == g_event_pool.size()) {
    hipEvent_t e;
    // timing-only events: no system-scope fence (cache writeback) around the traced kernels
    if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess) return nullptr;
    g_event_pool.push_back(e);
  }
  return g_event_pool[g_pool_used++];
}

// When the kind is being traced, hands an event pair to the kernel launches
// inside the scope (they record the first kernel's start and the last one's end
// on their own dispatches) and keeps the record if any kernel was launched.
struct TraceScope {
  long idx = -1;
  TraceScope(int kind, int level, hipStream_t) {
    if (!(g_trace_mask & (1u << kind))) return;
    std::lock_guard<std::mutex> lk(g_trace_mu);
    if (g_trace.size() >= kTraceMax) {
      ++g_trace_dropped;
      return;
    }
    hipEvent_t a = pool_event(), b = pool_event();
    if (!a || !b) return;
    idx = (long)g_trace.size();
    g_trace.push_back(TraceRec{kind, level, a, b});
    lp::launch_events() = lp::LaunchEvents{a, b, 0};
  }
  ~TraceScope() {
    if (idx < 0) return;
    lp::LaunchEvents& e = lp::launch_events();
    if (e.launched == 0) {  // nothing ran: void the record (its events hold no times)
      std::lock_guard<std::mutex> lk(g_trace_mu);
      g_trace[idx].kind = -1;
    }
    e = lp::LaunchEvents{};
  }
};

constexpr size_t kAlign = 256;
size_t up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

size_t esize(const lp_problem* p) { return p->dtype == LP_F64 ? 8 : 4; }
size_t qdim(const lp_problem* p) { return (size_t)p->C * p->H * p->W; }
size_t slice_bytes(const lp_problem* p) { return (size_t)p->B * qdim(p) * esize(p); }

lp::Shape shape_of(const lp_problem* p) {
  lp::Shape s;
  s.dtype = p->dtype;
  s.layer = p->layer;
  s.act = p->act;
  s.C = p->C;
  s.H = p->H;
  s.W = p->W;
  return s;
}

int check_problem(const lp_problem* p) {
  if (!p) return fail(LP_EINVAL, "problem is NULL");
  if (p->abi_version != LP_ABI_VERSION)
    return fail(LP_EINVAL, "abi_version %d != %d", p->abi_version, LP_ABI_VERSION);
  if (p->dtype != LP_F32 && p->dtype != LP_F64) return fail(LP_EINVAL, "bad dtype %d", p->dtype);
  if (p->layer != LP_DENSE && p->layer != LP_CONV3X3) return fail(LP_EINVAL, "bad layer %d", p->layer);
  if (p->act < LP_TANH || p->act > LP_IDENTITY) return fail(LP_EINVAL, "bad activation %d", p->act);
  if (p->N < 1) return fail(LP_EINVAL, "N = %d < 1", p->N);
  if (p->B < 0) return fail(LP_EINVAL, "B = %d < 0", p->B);
  if (p->C < 1 || p->H < 1 || p->W < 1) return fail(LP_EINVAL, "bad C/H/W %d/%d/%d", p->C, p->H, p->W);
  if (p->layer == LP_DENSE && (p->H != 1 || p->W != 1)) return fail(LP_EINVAL, "dense layers need H = W = 1");
  if (!(p->h > 0.0) || !isfinite(p->h)) return fail(LP_EINVAL, "step size h must be finite and > 0");
  if (!lp::shape_supported(shape_of(p)))
    return fail(LP_EUNSUPPORTED, "no kernel for dtype %d layer %d C=%d H=%d W=%d", p->dtype, p->layer, p->C,
                p->H, p->W);
  return LP_OK;
}

int check_mgrit(const lp_problem* p, const lp_mgrit* m, std::vector<int>& sizes) {
  if (!m) return fail(LP_EINVAL, "mgrit options are NULL");
  if (m->cf < 2) return fail(LP_EINVAL, "coarsening factor %d < 2", m->cf);
  if (m->max_levels < 1) return fail(LP_EINVAL, "max_levels %d < 1", m->max_levels);
  if (m->min_coarse < 1) return fail(LP_EINVAL, "min_coarse %d < 1", m->min_coarse);
  if (m->relax != LP_RELAX_F && m->relax != LP_RELAX_FCF && m->relax != LP_RELAX_FCFCF)
    return fail(LP_EINVAL, "bad relax %d", m->relax);
  if (m->cycle != LP_CYCLE_V && m->cycle != LP_CYCLE_F) return fail(LP_EINVAL, "bad cycle %d", m->cycle);
  if (m->storage != LP_STORE_ALL && m->storage != LP_STORE_CPOINTS) return fail(LP_EINVAL, "bad storage %d", m->storage);
  if (m->max_iter < 1) return fail(LP_EINVAL, "max_iter %d < 1", m->max_iter);
  if (!(m->rtol >= 0.0) || !(m->stag >= 0.0)) return fail(LP_EINVAL, "rtol and stag must be >= 0");
  sizes.assign(1, p->N);
  while ((int)sizes.size() < m->max_levels && sizes.back() > m->min_coarse) {
    if (sizes.back() % m->cf)
      return fail(LP_EINVAL, "level %d has N_l = %d, not divisible by cf = %d", (int)sizes.size() - 1,
                  sizes.back(), m->cf);
    sizes.push_back(sizes.back() / m->cf);
  }
  if (m->storage == LP_STORE_CPOINTS) {
    if (!lp::cpoints_supported(shape_of(p)) || m->cf != 4)
      return fail(LP_EUNSUPPORTED, "C-point storage needs an fp32 dense width 32 or 64 and cf = 4");
    if (sizes.size() < 2) return fail(LP_EINVAL, "C-point storage needs at least two levels");
  }
  return LP_OK;
}

// Workspace layout for one MGRIT solve.
struct Layout {
  std::vector<size_t> X, G, S;  // byte offsets per level (X[0], G[0] unused)
  std::vector<size_t> S2;       // FCFCF: second staging buffer of the coarse levels
  size_t S0b = 0;               // second finest-level staging buffer
  size_t partial = 0, rho = 0, total = 0;
  int partial_cap = 0;
};

int partial_capacity(const lp_problem* p) {
  const int tile = lp::min_tile(shape_of(p));
  const long tiles = (p->B + tile - 1) / tile;
  return (int)((long)(p->N + 1) * (tiles > 0 ? tiles : 1));
}

Layout mgrit_layout(const lp_problem* p, const lp_mgrit* m, const std::vector<int>& sizes) {
  Layout L;
  const size_t sl = slice_bytes(p);
  const int nl = (int)sizes.size();
  L.X.assign(nl, 0);
  L.G.assign(nl, 0);
  L.S.assign(nl, 0);
  L.S2.assign(nl, 0);
  size_t off = 0;
  for (int l = 1; l < nl; ++l) {
    L.X[l] = off;
    off = up(off + (size_t)(sizes[l] + 1) * sl);
    L.G[l] = off;
    off = up(off + (size_t)(sizes[l] + 1) * sl);
  }
  if (m->relax != LP_RELAX_F) {
    for (int l = 0; l + 1 < nl; ++l) {
      L.S[l] = off;
      off = up(off + (size_t)(sizes[l + 1] + 1) * sl);
    }
    if (nl > 1) {  // second finest-level staging buffer
      L.S0b = off;
      off = up(off + (size_t)(sizes[1] + 1) * sl);
    }
    if (m->relax == LP_RELAX_FCFCF) {  // the second C-relaxation stages into another buffer
      for (int l = 1; l + 1 < nl; ++l) {
        L.S2[l] = off;
        off = up(off + (size_t)(sizes[l + 1] + 1) * sl);
      }
    }
  }
  L.partial_cap = partial_capacity(p);
  L.partial = off;
  off = up(off + (size_t)L.partial_cap * sizeof(double));
  L.rho = off;
  off = up(off + (size_t)(m->max_iter + 1) * sizeof(double));
  L.total = off;
  return L;
}

size_t grad_bytes(const lp_problem* p) {
  const lp::Shape s = shape_of(p);
  const size_t nch = (size_t)lp::grad_chunks(s, p->B, p->N);
  return up((size_t)p->N * nch * lp::grad_partial_floats(s) * esize(p));
}

// lp_gradient_cpoints: the gradient partials, then the states of one block of at
// most kExpandIntervals coarse intervals recomputed from their C-points.
constexpr long kExpandIntervals = 64;
long expand_block(const lp_problem* p, int cf) { return std::min<long>(p->N / cf, kExpandIntervals); }
size_t grad_cpoints_bytes(const lp_problem* p, int cf) {
  return grad_bytes(p) + up((size_t)expand_block(p, cf) * cf * slice_bytes(p));
}

size_t resid_bytes(const lp_problem* p) {
  return up((size_t)partial_capacity(p) * sizeof(double)) + up(sizeof(double));
}

int check_ws(const void* ws, size_t have, size_t need) {
  if (need == 0) return LP_OK;
  if (!ws) return fail(LP_EWORKSPACE, "workspace is NULL (%zu bytes needed)", need);
  if ((uintptr_t)ws % kAlign) return fail(LP_EWORKSPACE, "workspace is not %zu-byte aligned", kAlign);
  if (have < need) return fail(LP_EWORKSPACE, "workspace has %zu bytes, %zu needed", have, need);
  return LP_OK;
}

// One MGRIT solve (state or adjoint) over the hierarchy.
struct Solver {
  const lp_problem* p;
  const lp_mgrit* m;
  lp::Shape sh;
  int dir;
  const void* K;
  const void* b;
  const void* Uf;  // fine primal trajectory (adjoint)
  void* dsig = nullptr;  // sigma' record (written by the forward's final level-0 F-relaxation, read by the adjoint)
  std::vector<int> sizes;
  bool cpt = false;  // C-point storage: the finest trajectory (forward X[0], adjoint Uf) holds C-points only
  std::vector<void*> X, G, S, S2;
  void* S0[2] = {nullptr, nullptr};  // finest-level staging buffers (FCF, FCFCF), used alternately
  int cur0 = 0;
  bool pending = false;              // finest-level correction not yet written back
  double* partial;
  hipStream_t st;
  int partials_used = 0;

  long stride(int l) const {
    long s = 1;
    for (int i = 0; i < l; ++i) s *= m->cf;
    return s;
  }

  // row step of the adjoint's primal trajectory per level-l point (the C-point
  // trajectory holds fine index n at row n / cf; level l >= 1 points are C-points)
  long ustride(int l) const { return cpt ? stride(l) / m->cf : stride(l); }

  // One cycle on level l (Algorithm 1 with step 3 recursive): cyc is LP_CYCLE_V or
  // LP_CYCLE_F (coarse problem solved by an F-cycle and then a V-cycle, the latter
  // left out above the coarsest level, whose solve is exact).
  int cycle(int l, int cyc) {
    const int L = (int)sizes.size();
    const double hl = p->h * (double)stride(l);
    const int kb = dir == lp::DIR_FWD ? LP_TRACE_FWD_FC : LP_TRACE_ADJ_FC;  // first kind of this direction
    if (l == L - 1) {
      lp::SerialArgs a{p->act, K, b, Uf, p->B, sizes[l], stride(l), hl, X[l], G[l],
                       dir == lp::DIR_ADJ || l == 0 ? dsig : nullptr, ustride(l)};
      TraceScope ts(kb + 3, l, st);
      LP_TRY(lp::launch_serial(sh, dir, a, st), "coarsest-level solve");
      return LP_OK;
    }
    const bool fcf = m->relax != LP_RELAX_F;  // at least one C-relaxation
    lp::SweepArgs a{};
    a.act = p->act;
    a.K = K;
    a.b = b;
    a.Uf = Uf;
    a.B = p->B;
    a.Nl = sizes[l];
    a.c = m->cf;
    a.stride = stride(l);
    a.ustride = ustride(l);
    a.cpt = cpt && l == 0;
    a.hl = hl;
    a.hc = hl * (double)m->cf;
    a.X = X[l];
    a.G = G[l];
    a.dsig = dir == lp::DIR_ADJ ? dsig : nullptr;  // the forward writes it in its final F-relaxation only
    // On the finest level with FCF the coarse-grid correction of a cycle is not
    // written back: the next cycle's FC sweep starts from C + (V - C) (the same
    // correction, applied on the fly), and the F-points, which no later sweep
    // reads, are written once by finish() after the last cycle. The relaxed
    // C-points then alternate between two staging buffers.
    const bool defer = l == 0 && fcf;
    void* Sl = defer ? S0[cur0] : S[l];
    a.S = Sl;
    a.finest = l == 0;
    a.mode = lp::SWEEP_FC;
    if (defer && pending) {
      a.Cs = S0[cur0 ^ 1];
      a.cs_stride = 1;
      a.V = X[1];
    }
    if (fcf) {
      TraceScope ts(kb + 0, l, st);
      LP_TRY(lp::launch_sweep(sh, dir, a, st, nullptr), "FC-relaxation");
    }
    if (m->relax == LP_RELAX_FCFCF) {
      // F- and C-relaxation again, from the staged C-points into the other staging
      // buffer (on the finest level the one the previous cycle used, now free);
      // reading them as C + (C - C) = C reuses the correcting form of the sweep
      void* Sn = defer ? S0[cur0 ^ 1] : S2[l];
      a.Cs = Sl;
      a.cs_stride = 1;
      a.V = Sl;
      a.S = Sn;
      {
        TraceScope ts(kb + 0, l, st);
        LP_TRY(lp::launch_sweep(sh, dir, a, st, nullptr), "FC-relaxation");
      }
      Sl = Sn;
      if (defer) cur0 ^= 1;  // S0[cur0] holds the relaxed C-points again
    }
    a.V = nullptr;
    a.Cs = fcf ? Sl : X[l];
    // C-points of the level trajectory: every cf-th row (row k with C-point storage)
    a.cs_stride = fcf || (a.cpt && dir == lp::DIR_FWD) ? 1 : m->cf;
    a.Xn = X[l + 1];
    a.Gn = G[l + 1];
    a.xn_every = (l + 1 < L - 1) ? m->cf : 0;
    a.partial = l == 0 ? partial : nullptr;
    int np = 0;
    a.mode = lp::SWEEP_FRES;
    {
      TraceScope ts(kb + 1, l, st);
      LP_TRY(lp::launch_sweep(sh, dir, a, st, &np), "F-relaxation and restriction");
    }
    if (l == 0) partials_used = np;
    int rc = cycle(l + 1, cyc);
    if (rc != LP_OK) return rc;
    if (cyc == LP_CYCLE_F && l + 2 < L) {
      rc = cycle(l + 1, LP_CYCLE_V);
      if (rc != LP_OK) return rc;
    }
    if (defer) {
      pending = true;
      cur0 ^= 1;
      return LP_OK;
    }
    a.V = X[l + 1];
    a.mode = lp::SWEEP_CORRF;
    a.partial = nullptr;
    if (dir == lp::DIR_FWD && l == 0) a.dsig = dsig;
    TraceScope ts(kb + 2, l, st);
    LP_TRY(lp::launch_sweep(sh, dir, a, st, nullptr), "correction and F-relaxation");
    return LP_OK;
  }

  // Apply the finest level's pending correction and F-relaxation (Algorithm 1,
  // steps 4-5 of the last cycle), writing every row of the solution.
  int finish() {
    if (!pending) return LP_OK;
    lp::SweepArgs a{};
    a.act = p->act;
    a.mode = lp::SWEEP_CORRF;
    a.K = K;
    a.b = b;
    a.Uf = Uf;
    a.B = p->B;
    a.Nl = sizes[0];
    a.c = m->cf;
    a.stride = 1;
    a.ustride = ustride(0);
    a.cpt = cpt;
    a.hl = p->h;
    a.hc = p->h * (double)m->cf;
    a.X = X[0];
    a.Cs = S0[cur0 ^ 1];
    a.cs_stride = 1;
    a.V = X[1];
    a.finest = 1;
    a.dsig = dsig;
    const int kb = dir == lp::DIR_FWD ? LP_TRACE_FWD_FC : LP_TRACE_ADJ_FC;
    TraceScope ts(kb + 2, 0, st);
    LP_TRY(lp::launch_sweep(sh, dir, a, st, nullptr), "correction and F-relaxation");
    pending = false;
    return LP_OK;
  }
};

int mgrit_solve(const lp_problem* p, const lp_mgrit* m, int dir, const void* K, const void* b,
                const void* U, void* Xuser, void* dsig, void* ws, size_t ws_bytes, double* res_hist,
                int32_t* iters, void* stream) {
  int rc = check_problem(p);
  if (rc) return rc;
  std::vector<int> sizes;
  rc = check_mgrit(p, m, sizes);
  if (rc) return rc;
  if (!K || !b || (p->B && (!Xuser || (dir == lp::DIR_ADJ && !U))))
    return fail(LP_EINVAL, "NULL array argument");
  if (p->B && dir == lp::DIR_ADJ && U == Xuser) return fail(LP_EINVAL, "U and Lam alias");
  if (iters) *iters = 0;
  if (p->B == 0) return LP_OK;
  const Layout lay = mgrit_layout(p, m, sizes);
  rc = check_ws(ws, ws_bytes, lay.total);
  if (rc) return rc;
  hipStream_t st = static_cast<hipStream_t>(stream);
  char* w = static_cast<char*>(ws);
  const int L = (int)sizes.size();
  Solver s;
  s.p = p;
  s.m = m;
  s.sh = shape_of(p);
  s.dir = dir;
  s.K = K;
  s.b = b;
  s.Uf = U;
  s.cpt = m->storage == LP_STORE_CPOINTS;
  s.dsig = lp::dsig_supported(shape_of(p)) && !s.cpt ? dsig : nullptr;
  s.sizes = sizes;
  s.X.assign(L, nullptr);
  s.G.assign(L, nullptr);
  s.S.assign(L, nullptr);
  s.S2.assign(L, nullptr);
  s.X[0] = Xuser;
  for (int l = 1; l < L; ++l) {
    s.X[l] = w + lay.X[l];
    s.G[l] = w + lay.G[l];
  }
  if (m->relax != LP_RELAX_F && L > 1) {
    for (int l = 0; l + 1 < L; ++l) s.S[l] = w + lay.S[l];
    s.S0[0] = s.S[0];
    s.S0[1] = w + lay.S0b;
    if (m->relax == LP_RELAX_FCFCF)
      for (int l = 1; l + 1 < L; ++l) s.S2[l] = w + lay.S2[l];
  }
  s.partial = reinterpret_cast<double*>(w + lay.partial);
  s.st = st;
  double* rho = reinterpret_cast<double*>(w + lay.rho);
  const size_t sl = slice_bytes(p);
  const int c = m->cf;
  const int Nc = p->N / c;

  if (!m->warm_start && L > 1) {
    // cold start: every C-point is a copy of the fixed boundary row
    if (dir == lp::DIR_FWD && s.cpt) LP_TRY(lp::launch_copy_rows(Xuser, sl, 0, 1, 1, Nc, st), "cold start");
    else if (dir == lp::DIR_FWD) LP_TRY(lp::launch_copy_rows(Xuser, sl, 0, c, c, Nc, st), "cold start");
    else LP_TRY(lp::launch_copy_rows(Xuser, sl, p->N, 0, c, Nc, st), "cold start");
  }
  const bool early = m->rtol > 0.0 || m->stag > 0.0;
  std::vector<double> hist;
  int it = 0;
  for (int mi = 0; mi < m->max_iter; ++mi) {
    rc = s.cycle(0, m->cycle);
    if (rc) return rc;
    if (L > 1) LP_TRY(lp::launch_norm_reduce(s.partial, s.partials_used, rho + mi, st), "residual norm");
    else LP_TRY(lp::launch_zero(rho + mi, sizeof(double), st), "residual norm");
    it = mi + 1;
    if (early) {
      double r = 0.0;
      LP_TRY(hipMemcpyAsync(&r, rho + mi, sizeof(double), hipMemcpyDeviceToHost, st), "read residual");
      LP_TRY(hipStreamSynchronize(st), "stream sync");
      hist.push_back(r);
      if (!isfinite(r)) break;
      if (m->rtol > 0.0 && r <= m->rtol * hist[0]) break;
      if (m->stag > 0.0 && mi > 0 && r > m->stag * hist[mi - 1]) break;
    }
  }
  rc = s.finish();
  if (rc) return rc;
  // With neither a stopping rule nor a history to return, nothing is read back:
  // the call returns with the work enqueued; a non-finite norm stays recorded in
  // the device flag that lp_check_finite reads.
  if (!early && res_hist) {
    hist.assign(it, 0.0);
    LP_TRY(hipMemcpyAsync(hist.data(), rho, it * sizeof(double), hipMemcpyDeviceToHost, st), "read residuals");
    LP_TRY(hipStreamSynchronize(st), "stream sync");
  }
  if (res_hist) memcpy(res_hist, hist.data(), it * sizeof(double));
  if (iters) *iters = it;
  for (double r : hist)
    if (!isfinite(r)) return fail(LP_ENONFINITE, "residual norm is not finite");
  return LP_OK;
}

}  // namespace

namespace lp {

bool dense_width_supported(int q) { return q == 8 || q == 16 || q == 32 || q == 64; }

int dense_grad_chunks(int B, int N) {
  // enough workgroups to fill the chip when N is small, at least 64 and at most
  // 2048 examples per chunk: each of a chunk's four waves then sums at most 512
  // examples in fp32 before the chunks are summed in fp64, which keeps the
  // gradient's rounding error near 1e-6 relative at any batch size
  int ch = (2048 + N - 1) / N;
  ch = std::max(ch, (B + 2047) / 2048);
  ch = std::min(ch, (B + 63) / 64);
  return ch < 1 ? 1 : ch;
}

bool shape_supported(const Shape& s) {
  if (s.layer == 0)
    return s.H == 1 && s.W == 1 &&
           ((dense_width_supported(s.C) && !(s.dtype == 1 && s.C > 32)) || (s.dtype == 0 && wide_width_supported(s.C)));
  return conv_supported(s);
}

int min_tile(const Shape& s) { return s.layer == 0 ? 32 : conv_tile(s); }

int grad_chunks(const Shape& s, int B, int N) {
  return s.layer == 0 ? dense_grad_chunks(B, N) : conv_grad_chunks(B, N);
}

int grad_nout(const Shape& s) { return s.layer == 0 ? s.C * s.C + s.C : s.C * s.C * 9 + s.C; }

// Values one gradient workgroup writes as its chunk partial: dense dK and db;
// conv the expanded 16 x 96 weight block plus db (see lp_conv.hip).
int grad_partial_floats(const Shape& s) { return s.layer == 0 ? s.C * s.C + s.C : 16 * 96 + s.C; }

// fp32 dense layers of width 32 or 64 run on the matrix cores unless the
// environment variable LP_DENSE_PATH=valu selects the vector-ALU kernels (kept
// for cross-checking the two implementations against each other).
bool use_mfma(const Shape& s) {
  if (s.layer != 0 || s.dtype != 0 || !mfma_width_supported(s.C)) return false;
  const char* e = getenv("LP_DENSE_PATH");
  return !(e && strcmp(e, "valu") == 0);
}

// C-point storage: the matrix-core kernels of widths 32 and 64 recompute F-point states
bool cpoints_supported(const Shape& s) { return use_mfma(s); }

// fp32 dense layers too wide for the per-thread and whole-layer-in-LDS kernels
bool use_wide(const Shape& s) { return s.layer == 0 && s.dtype == 0 && wide_width_supported(s.C); }

// the sigma' record is written and read by the dense matrix-core kernels and
// the convolution kernels (no record exists for the identity activation)
bool dsig_supported(const Shape& s) {
  return s.act != LP_IDENTITY && (use_mfma(s) || use_wide(s) || (s.layer == 1 && conv_supported(s)));
}

hipError_t launch_sweep(const Shape& s, int dir, const SweepArgs& a, hipStream_t st, int* partials) {
  if (s.layer != 0) return conv_sweep(s, dir, a, st, partials);
  if (use_wide(s)) return wide_sweep(s.C, dir, a, st, partials);
  if (use_mfma(s)) return mfma_sweep(s.C, dir, a, st, partials);
  return s.dtype == 0 ? dense_sweep_f32(s.C, dir, a, st, partials) : dense_sweep_f64(s.C, dir, a, st, partials);
}

hipError_t launch_serial(const Shape& s, int dir, const SerialArgs& a, hipStream_t st) {
  if (s.layer != 0) return conv_serial(s, dir, a, st);
  if (use_wide(s)) return wide_serial(s.C, dir, a, st);
  if (use_mfma(s)) return mfma_serial(s.C, dir, a, st);
  return s.dtype == 0 ? dense_serial_f32(s.C, dir, a, st) : dense_serial_f64(s.C, dir, a, st);
}

hipError_t launch_resid(const Shape& s, int dir, const ResidArgs& a, hipStream_t st, int* partials) {
  if (s.layer != 0) return conv_resid(s, dir, a, st, partials);
  if (use_wide(s)) return wide_resid(s.C, dir, a, st, partials);
  return s.dtype == 0 ? dense_resid_f32(s.C, dir, a, st, partials) : dense_resid_f64(s.C, dir, a, st, partials);
}

hipError_t launch_grad(const Shape& s, const GradArgs& a, hipStream_t st) {
  if (s.layer != 0) return conv_grad(s, a, st);
  if (use_wide(s)) return wide_grad(s.C, a, st);
  if (use_mfma(s)) return mfma_grad(s.C, a, st);
  return s.dtype == 0 ? dense_grad_f32(s.C, a, st) : dense_grad_f64(s.C, a, st);
}

}  // namespace lp

extern "C" {

int32_t lp_abi_version(void) { return LP_ABI_VERSION; }

const char* lp_status_string(int32_t s) {
  switch (s) {
    case LP_OK: return "ok";
    case LP_EINVAL: return "invalid argument";
    case LP_EUNSUPPORTED: return "unsupported";
    case LP_EWORKSPACE: return "workspace too small or misaligned";
    case LP_EHIP: return "HIP runtime error";
    case LP_ENONFINITE: return "non-finite residual";
  }
  return "unknown status";
}

const char* lp_last_error(void) { return g_err.c_str(); }

size_t lp_workspace_bytes(const lp_problem* p, const lp_mgrit* m) {
  if (check_problem(p) != LP_OK) return 0;
  size_t need = std::max({grad_bytes(p), resid_bytes(p), lp::loss_workspace_bytes_max(esize(p), p->B, (int)qdim(p), 64)});
  if (m) {
    std::vector<int> sizes;
    if (check_mgrit(p, m, sizes) != LP_OK) return 0;
    need = std::max(need, mgrit_layout(p, m, sizes).total);
    if (m->storage == LP_STORE_CPOINTS) need = std::max(need, grad_cpoints_bytes(p, m->cf));
  }
  g_err.clear();
  return need;
}

size_t lp_dsig_bytes(const lp_problem* p) {
  if (check_problem(p) != LP_OK) return 0;
  g_err.clear();
  if (!lp::dsig_supported(shape_of(p))) return 0;
  if (p->layer == LP_CONV3X3) return (size_t)p->N * p->B * lp::conv_dsig_block_bytes(shape_of(p));
  const size_t vals = (size_t)p->N * p->B * qdim(p);
  // ReLU: one bit per value at widths 32 and 64, one byte at width 220
  if (p->act == LP_RELU) return qdim(p) == 220 ? vals : vals / 8;
  return vals * esize(p);
}

// The record is only written and read where the kernels support it, so a
// forward and an adjoint call on the same problem always agree.
void* dsig_for(const lp_problem* p, const void* dsig) {
  return lp::dsig_supported(shape_of(p)) ? const_cast<void*>(dsig) : nullptr;
}

int32_t lp_serial_forward(const lp_problem* p, const void* K, const void* b, void* U, void* dsig, void* stream) {
  int rc = check_problem(p);
  if (rc) return rc;
  if (!K || !b || (p->B && !U)) return fail(LP_EINVAL, "NULL array argument");
  if (p->B == 0) return LP_OK;
  lp::SerialArgs a{p->act, K, b, nullptr, p->B, p->N, 1, p->h, U, nullptr, dsig_for(p, dsig), 1};
  TraceScope ts(LP_TRACE_SERIAL, 0, static_cast<hipStream_t>(stream));
  LP_TRY(lp::launch_serial(shape_of(p), lp::DIR_FWD, a, static_cast<hipStream_t>(stream)), "serial forward");
  return LP_OK;
}

int32_t lp_serial_adjoint(const lp_problem* p, const void* K, const void* b, const void* U, const void* dsig,
                          void* Lam, void* stream) {
  int rc = check_problem(p);
  if (rc) return rc;
  if (!K || !b || (p->B && (!U || !Lam))) return fail(LP_EINVAL, "NULL array argument");
  if (p->B && U == Lam) return fail(LP_EINVAL, "U and Lam alias");
  if (p->B == 0) return LP_OK;
  lp::SerialArgs a{p->act, K, b, U, p->B, p->N, 1, p->h, Lam, nullptr, dsig_for(p, dsig), 1};
  TraceScope ts(LP_TRACE_SERIAL, 1, static_cast<hipStream_t>(stream));
  LP_TRY(lp::launch_serial(shape_of(p), lp::DIR_ADJ, a, static_cast<hipStream_t>(stream)), "serial adjoint");
  return LP_OK;
}

int32_t lp_mgrit_forward(const lp_problem* p, const lp_mgrit* m, const void* K, const void* b, void* U,
                         void* dsig, void* ws, size_t ws_bytes, double* res_hist, int32_t* iters, void* stream) {
  return mgrit_solve(p, m, lp::DIR_FWD, K, b, nullptr, U, dsig, ws, ws_bytes, res_hist, iters, stream);
}

int32_t lp_mgrit_adjoint(const lp_problem* p, const lp_mgrit* m, const void* K, const void* b, const void* U,
                         const void* dsig, void* Lam, void* ws, size_t ws_bytes, double* res_hist,
                         int32_t* iters, void* stream) {
  return mgrit_solve(p, m, lp::DIR_ADJ, K, b, U, Lam, const_cast<void*>(dsig), ws, ws_bytes, res_hist, iters,
                     stream);
}

int32_t lp_gradient(const lp_problem* p, const void* K, const void* b, const void* U, const void* dsig,
                    const void* Lam, void* dK, void* db, void* ws, size_t ws_bytes, void* stream) {
  int rc = check_problem(p);
  if (rc) return rc;
  if (!K || !b || !dK || !db || (p->B && (!U || !Lam))) return fail(LP_EINVAL, "NULL array argument");
  const lp::Shape s = shape_of(p);
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (p->B == 0) {
    const size_t nw = (size_t)p->N * (lp::grad_nout(s) - p->C) * esize(p);
    LP_TRY(lp::launch_zero(dK, nw, st), "zero gradient");
    LP_TRY(lp::launch_zero(db, (size_t)p->N * p->C * esize(p), st), "zero gradient");
    return LP_OK;
  }
  rc = check_ws(ws, ws_bytes, grad_bytes(p));
  if (rc) return rc;
  lp::GradArgs a{p->act, K, b, U, Lam, p->B, p->N, p->h, ws, lp::grad_chunks(s, p->B, p->N), dK, db,
                 dsig_for(p, dsig), 0};
  TraceScope ts(LP_TRACE_GRADIENT, 0, st);
  LP_TRY(lp::launch_grad(s, a, st), "gradient");
  return LP_OK;
}

namespace {

int residual_norm_args(const lp_problem* p, int32_t which, const void* K, const void* b, const void* U,
                       const void* Lam, const double* norm) {
  int rc = check_problem(p);
  if (rc) return rc;
  if (which != LP_STATE && which != LP_ADJOINT) return fail(LP_EINVAL, "bad system %d", which);
  if (!K || !b || !norm || (p->B && (!U || (which == LP_ADJOINT && !Lam))))
    return fail(LP_EINVAL, "NULL array argument");
  return LP_OK;
}

// The residual kernels write one partial per workgroup into ws, the fixed-order
// reduction the norm into the slot after them; the result is read back.
int residual_norm_in(const lp_problem* p, int32_t which, const void* K, const void* b, const void* U,
                     const void* Lam, void* ws, double* norm, hipStream_t st) {
  double* partial = static_cast<double*>(ws);
  double* out = reinterpret_cast<double*>(static_cast<char*>(ws) + up((size_t)partial_capacity(p) * sizeof(double)));
  lp::ResidArgs a{p->act, K, b, U, Lam, p->B, p->N, p->h, partial};
  int np = 0;
  {
    TraceScope ts(LP_TRACE_RESIDUAL, which, st);
    LP_TRY(lp::launch_resid(shape_of(p), which == LP_STATE ? lp::DIR_FWD : lp::DIR_ADJ, a, st, &np), "residual");
  }
  LP_TRY(lp::launch_norm_reduce(partial, np, out, st), "residual norm");
  LP_TRY(hipMemcpyAsync(norm, out, sizeof(double), hipMemcpyDeviceToHost, st), "read residual norm");
  LP_TRY(hipStreamSynchronize(st), "stream sync");
  if (!isfinite(*norm)) return fail(LP_ENONFINITE, "residual norm is not finite");
  return LP_OK;
}

}  // namespace

int32_t lp_gradient_cpoints(const lp_problem* p, int32_t cf, const void* K, const void* b, const void* Uc,
                            const void* Lam, void* dK, void* db, void* ws, size_t ws_bytes, void* stream) {
  int rc = check_problem(p);
  if (rc) return rc;
  const lp::Shape s = shape_of(p);
  if (!lp::cpoints_supported(s) || cf != 4)
    return fail(LP_EUNSUPPORTED, "C-point storage needs an fp32 dense width 32 or 64 and cf = 4");
  if (p->N % cf) return fail(LP_EINVAL, "N = %d is not divisible by cf = %d", p->N, cf);
  if (!K || !b || !dK || !db || (p->B && (!Uc || !Lam))) return fail(LP_EINVAL, "NULL array argument");
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (p->B == 0) {
    LP_TRY(lp::launch_zero(dK, (size_t)p->N * p->C * p->C * esize(p), st), "zero gradient");
    LP_TRY(lp::launch_zero(db, (size_t)p->N * p->C * esize(p), st), "zero gradient");
    return LP_OK;
  }
  rc = check_ws(ws, ws_bytes, grad_cpoints_bytes(p, cf));
  if (rc) return rc;
  void* Y = static_cast<char*>(ws) + grad_bytes(p);  // states of one block of intervals
  const long Nc = p->N / cf, blk = expand_block(p, cf);
  lp::GradArgs a{p->act, K, b, Y, Lam, p->B, p->N, p->h, ws, lp::grad_chunks(s, p->B, p->N), dK, db, nullptr, 0};
  TraceScope ts(LP_TRACE_GRADIENT, 0, st);
  for (long k0 = 0; k0 < Nc; k0 += blk) {
    const long nk = std::min(blk, Nc - k0);
    LP_TRY(lp::mfma_expand(p->C, p->act, K, b, Uc, Y, p->B, k0, nk, p->h, st), "gradient: recompute states");
    a.n0 = k0 * cf;
    LP_TRY(lp::mfma_grad_partials(p->C, a, nk * cf, st), "gradient");
  }
  LP_TRY(lp::mfma_grad_finish(p->C, a, st), "gradient");
  return LP_OK;
}

int32_t lp_residual_norm(const lp_problem* p, int32_t which, const void* K, const void* b, const void* U,
                         const void* Lam, void* ws, size_t ws_bytes, double* norm, void* stream) {
  int rc = residual_norm_args(p, which, K, b, U, Lam, norm);
  if (rc) return rc;
  if (p->B == 0) {
    *norm = 0.0;
    return LP_OK;
  }
  rc = check_ws(ws, ws_bytes, resid_bytes(p));
  if (rc) return rc;
  return residual_norm_in(p, which, K, b, U, Lam, ws, norm, static_cast<hipStream_t>(stream));
}

int32_t lp_residual_norm_noalloc(const lp_problem* p, int32_t which, const void* K, const void* b, const void* U,
                                 const void* Lam, double* norm, void* stream) {
  int rc = residual_norm_args(p, which, K, b, U, Lam, norm);
  if (rc) return rc;
  if (p->B == 0) {
    *norm = 0.0;
    return LP_OK;
  }
  const size_t need = resid_bytes(p), have = lp::noalloc_scratch_bytes();
  if (need > have)
    return fail(LP_EWORKSPACE, "the residual of this problem needs %zu bytes of scratch; the library's static "
                "scratch holds %zu (at most %zu residual partials; use lp_residual_norm with a workspace)",
                need, have, (have - kAlign) / sizeof(double));
  void* ws = nullptr;
  LP_TRY(lp::noalloc_scratch(&ws), "static scratch");
  return residual_norm_in(p, which, K, b, U, Lam, ws, norm, static_cast<hipStream_t>(stream));
}

int32_t lp_check_finite(void* stream) {
  uint32_t flag = 0u;
  LP_TRY(lp::read_nonfinite(&flag, true, static_cast<hipStream_t>(stream)), "read non-finite flag");
  if (flag) return fail(LP_ENONFINITE, "a residual norm computed on this device was not finite");
  return LP_OK;
}

int32_t lp_open_forward(const lp_problem* p, int32_t opening, int32_t nf, const void* y, const void* L_in,
                        void* u0, void* stream) {
  int rc = check_problem(p);
  if (rc) return rc;
  if (opening < LP_OPEN_IDENTITY || opening > LP_OPEN_CONV_ACT) return fail(LP_EINVAL, "bad opening %d", opening);
  if ((p->B && (!y || !u0)) || (opening != LP_OPEN_IDENTITY && !L_in)) return fail(LP_EINVAL, "NULL array argument");
  if (opening == LP_OPEN_DENSE_ACT && (p->layer != LP_DENSE || nf < 1))
    return fail(LP_EINVAL, "dense opening needs a dense problem and nf >= 1");
  if (opening == LP_OPEN_CONV_ACT && p->layer != LP_CONV3X3) return fail(LP_EINVAL, "conv opening needs a conv problem");
  if (p->B == 0) return LP_OK;
  LP_TRY(lp::launch_open_forward(shape_of(p), opening, nf, p->B, y, L_in, u0, static_cast<hipStream_t>(stream)),
         "opening layer");
  return LP_OK;
}

int32_t lp_open_grad(const lp_problem* p, int32_t opening, int32_t nf, const void* y, const void* L_in,
                     const void* lam0, void* dL_in, void* stream) {
  int rc = check_problem(p);
  if (rc) return rc;
  if (opening != LP_OPEN_DENSE_ACT && opening != LP_OPEN_CONV_ACT)
    return fail(LP_EINVAL, "opening %d has no weights", opening);
  if (!L_in || !dL_in || (p->B && (!y || !lam0))) return fail(LP_EINVAL, "NULL array argument");
  if (opening == LP_OPEN_DENSE_ACT && (p->layer != LP_DENSE || nf < 1 || nf > 1024))
    return fail(LP_EINVAL, "dense opening needs a dense problem and 1 <= nf <= 1024");
  if (opening == LP_OPEN_CONV_ACT && p->layer != LP_CONV3X3) return fail(LP_EINVAL, "conv opening needs a conv problem");
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (p->B == 0) {
    const size_t n = opening == LP_OPEN_DENSE_ACT ? (size_t)p->C * nf : (size_t)p->C * 9;
    LP_TRY(lp::launch_zero(dL_in, n * esize(p), st), "zero gradient");
    return LP_OK;
  }
  LP_TRY(lp::launch_open_grad(shape_of(p), opening, nf, p->B, y, L_in, lam0, dL_in, st), "opening gradient");
  return LP_OK;
}

int32_t lp_loss_terminal(const lp_problem* p, int32_t nc, const void* uN, const void* W, const void* mu,
                         const void* c, double* J, void* lamN, void* dW, void* dmu, void* ws, size_t ws_bytes,
                         void* stream) {
  int rc = check_problem(p);
  if (rc) return rc;
  if (nc < 1 || nc > 64) return fail(LP_EINVAL, "need 1 <= nc <= 64, nc = %d", nc);
  if (!uN || !W || !mu || !c || !J || !lamN || !dW || !dmu) return fail(LP_EINVAL, "NULL array argument");
  if (p->B == 0) return fail(LP_EINVAL, "the mean loss needs B >= 1");
  rc = check_ws(ws, ws_bytes, lp::loss_workspace_bytes(esize(p), p->B, (int)qdim(p), nc));
  if (rc) return rc;
  LP_TRY(lp::launch_loss(p->dtype, p->B, (int)qdim(p), nc, uN, W, mu, c, J, lamN, dW, dmu, ws,
                         static_cast<hipStream_t>(stream)),
         "loss");
  return LP_OK;
}

int32_t lp_sgd_update(int32_t dtype, size_t n, double lr, const void* g, void* x, void* stream) {
  if (dtype != LP_F32 && dtype != LP_F64) return fail(LP_EINVAL, "bad dtype %d", dtype);
  if (n && (!g || !x)) return fail(LP_EINVAL, "NULL array argument");
  LP_TRY(lp::launch_sgd(dtype, n, lr, g, x, static_cast<hipStream_t>(stream)), "sgd update");
  return LP_OK;
}

int32_t lp_vec_axpby(int32_t dtype, size_t n, double a, const void* x, double b, void* y, void* stream) {
  if (dtype != LP_F32 && dtype != LP_F64) return fail(LP_EINVAL, "bad dtype %d", dtype);
  if (n && (!x || !y)) return fail(LP_EINVAL, "NULL array argument");
  LP_TRY(lp::launch_axpby(dtype, n, a, x, b, y, static_cast<hipStream_t>(stream)), "axpby");
  return LP_OK;
}

int32_t lp_vec_dot(int32_t dtype, size_t n, const void* x, const void* y, double* out, void* stream) {
  static_assert(LP_DOT_PARTIALS == lp::DOT_BLOCKS, "dot partial count");
  if (dtype != LP_F32 && dtype != LP_F64) return fail(LP_EINVAL, "bad dtype %d", dtype);
  if (!out || (n && (!x || !y))) return fail(LP_EINVAL, "NULL array argument");
  LP_TRY(lp::launch_dot(dtype, n, x, y, out, static_cast<hipStream_t>(stream)), "dot");
  return LP_OK;
}

int32_t lp_accuracy(const lp_problem* p, int32_t nc, const void* uN, const void* W, const void* mu, const void* c,
                    double* acc, void* ws, size_t ws_bytes, void* stream) {
  int rc = check_problem(p);
  if (rc) return rc;
  if (nc < 1 || nc > 64) return fail(LP_EINVAL, "need 1 <= nc <= 64, nc = %d", nc);
  if (!uN || !W || !mu || !c || !acc) return fail(LP_EINVAL, "NULL array argument");
  if (p->B == 0) return fail(LP_EINVAL, "the accuracy needs B >= 1");
  rc = check_ws(ws, ws_bytes, lp::loss_workspace_bytes(esize(p), p->B, (int)qdim(p), nc));
  if (rc) return rc;
  LP_TRY(lp::launch_accuracy(p->dtype, p->B, (int)qdim(p), nc, uN, W, mu, c, acc, ws,
                             static_cast<hipStream_t>(stream)),
         "accuracy");
  return LP_OK;
}

int32_t lp_trace_enable(uint32_t kind_mask) {
  std::lock_guard<std::mutex> lk(g_trace_mu);
  // earlier records may still be pending on some stream: wait before reusing their events
  for (const TraceRec& r : g_trace) (void)hipEventSynchronize(r.b);
  g_trace.clear();
  g_pool_used = 0;
  g_trace_dropped = 0;
  g_trace_mask = kind_mask & ((1u << LP_TRACE_KINDS) - 1);
  return LP_OK;
}

int32_t lp_trace_read(int32_t kind, int32_t level, int32_t* launches, double* total_ms) {
  if (kind < 0 || kind >= LP_TRACE_KINDS) return fail(LP_EINVAL, "bad trace kind %d", kind);
  if (!launches || !total_ms) return fail(LP_EINVAL, "NULL output");
  std::lock_guard<std::mutex> lk(g_trace_mu);
  int n = 0;
  double ms = 0.0;
  for (const TraceRec& r : g_trace) {
    if (r.kind != kind || (level >= 0 && r.level != level)) continue;
    LP_TRY(hipEventSynchronize(r.b), "trace event");
    float t = 0.f;
    LP_TRY(hipEventElapsedTime(&t, r.a, r.b), "trace event");
    ms += t;
    ++n;
  }
  *launches = n;
  *total_ms = ms;
  return LP_OK;
}

}  // extern "C"
