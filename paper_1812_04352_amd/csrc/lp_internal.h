// Internal interface between the host scheduler (lp_host.cpp) and the kernel
// launchers. Not part of the public ABI.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace lp {

// Tracing hook. While a traced call runs, the kernels it launches record their
// own start (the first launch) and end (every launch; the last one stands) into
// these events on the dispatch itself, so tracing puts no marker packets into
// the stream between kernels. Thread-local; set and cleared by the host.
struct LaunchEvents {
  hipEvent_t start = nullptr, stop = nullptr;
  int launched = 0;
};
LaunchEvents& launch_events();

template <typename... P, typename... A>
inline void launch(void (*k)(P...), dim3 grid, dim3 block, size_t shmem, hipStream_t st, A... args) {
  LaunchEvents& e = launch_events();
  if (e.stop) {
    hipExtLaunchKernelGGL(k, grid, block, (uint32_t)shmem, st, e.launched ? nullptr : e.start, e.stop, 0u,
                          static_cast<P>(args)...);
    ++e.launched;
  } else {
    k<<<grid, block, shmem, st>>>(static_cast<P>(args)...);
  }
}

enum Dir { DIR_FWD = 0, DIR_ADJ = 1 };

// One interval sweep on MGRIT level l. Interval k covers level points kc..(k+1)c.
enum SweepMode {
  SWEEP_FC = 0,    // F- then C-relaxation from the C-points of X; relaxed C-points -> S
  SWEEP_FRES = 1,  // F-relaxation from the relaxed C-points, residual, FAS restriction
  SWEEP_CORRF = 2  // coarse-grid correction of the C-points, then F-relaxation writing X
};

struct SweepArgs {
  int act;             // activation (uniform)
  int mode;            // SweepMode
  const void* K;       // fine weights [N][q][q] (conv [N][C][C][3][3])
  const void* b;       // fine bias [N][q] (conv [N][C])
  const void* Uf;      // fine primal trajectory [N+1][B][q] (adjoint steps only)
  int B;               // batch
  int Nl;              // steps on this level
  int c;               // coarsening factor
  long stride;         // c^l: level point i uses fine weights (and adjoint state) i*stride
  double hl, hc;       // step on this level and on the next coarser level
  void* X;             // level trajectory: forward U_l, adjoint Lam_l
  const void* G;       // level right-hand side (nullptr: zero rows, the finest level)
  const void* Cs;      // relaxed C-points: C_k at Cs + k * cs_stride slices
  long cs_stride;
  void* S;             // FC: staging of the relaxed C-points, N_l/c + 1 slices
  void* Xn;            // FRES: next level trajectory
  void* Gn;            // FRES: next level right-hand side
  int xn_every;        // FRES: write Xn[k] when k % xn_every == 0 (<= 0: boundary point only)
  const void* V;       // CORRF: next level solution
  double* partial;     // FRES: per-workgroup sum of squared residuals (nullable)
  int finest;          // 1 on level 0: the fixed boundary row (u^0 or lam^N) is never written
  void* dsig;          // sigma' record (nullable; dense [N][B][q], conv per-(layer, example) tile blocks): forward level-0 CORRF writes it
                       // (every layer of its intervals), the adjoint reads it at i*stride
  long ustride;        // adjoint: the primal state of level point i is Uf row i*ustride (stride, or
                       // stride / c when Uf holds the fine C-points only)
  int cpt;             // level 0 with C-point storage: forward, X holds C-point k at row k (F-points are
                       // not stored); adjoint, Uf holds the C-points and each interval recomputes its
                       // F-point states (and sigma') by forward steps from its lower C-point
};

// Serial (coarsest level or layer-serial) solve of X over Nl steps.
struct SerialArgs {
  int act;
  const void* K;
  const void* b;
  const void* Uf;      // adjoint only
  int B;
  int Nl;
  long stride;
  double hl;
  void* X;
  const void* G;       // nullable
  void* dsig;          // sigma' record (nullable): written by a level-0 forward solve, read by the adjoint
  long ustride;        // adjoint: primal state of level point i at Uf row i*ustride
};

struct ResidArgs {
  int act;
  const void* K;
  const void* b;
  const void* U;
  const void* Lam;     // adjoint only
  int B;
  int N;
  double h;
  double* partial;     // one per workgroup
};

struct GradArgs {
  int act;
  const void* K;
  const void* b;
  const void* U;
  const void* Lam;
  int B;
  int N;
  double h;
  void* partial;       // [N][nchunks][nout] in the problem dtype
  int nchunks;
  void* dK;
  void* db;
  const void* dsig;    // sigma' record of U (nullable)
  long n0;             // first layer of this launch: grid x runs over layers n0 .. n0 + gridDim.x - 1,
                       // U row j is layer n0 + j (Lam, K, b, dsig and the partials use absolute indices)
};

struct Shape {
  int dtype;   // 0 f32, 1 f64
  int layer;   // 0 dense, 1 conv
  int act;
  int C, H, W; // dense: C = q
};

// Launchers. Each returns hipSuccess, hipErrorNotSupported for a shape with no
// kernel, or the launch error. *partials (when non-null) receives the number of
// residual partials the launch writes.
hipError_t launch_sweep(const Shape& s, int dir, const SweepArgs& a, hipStream_t st, int* partials);
hipError_t launch_serial(const Shape& s, int dir, const SerialArgs& a, hipStream_t st);
hipError_t launch_resid(const Shape& s, int dir, const ResidArgs& a, hipStream_t st, int* partials);
hipError_t launch_grad(const Shape& s, const GradArgs& a, hipStream_t st);
int grad_chunks(const Shape& s, int B, int N);  // batch chunks of the gradient's first pass
bool dsig_supported(const Shape& s);            // kernels that write and read the sigma' record
bool cpoints_supported(const Shape& s);         // kernels with C-point storage (recomputed F-point states)
int grad_nout(const Shape& s);            // weights + bias entries per layer
int grad_partial_floats(const Shape& s);  // values per (layer, chunk) gradient partial
bool shape_supported(const Shape& s);
int min_tile(const Shape& s);             // fewest examples any sweep/residual workgroup covers

// Dense VALU family (lp_dense_impl.h, instantiated per dtype in lp_dense_f32.hip / lp_dense_f64.hip)
#define LP_DENSE_DECL(SFX)                                                                          \
  hipError_t dense_sweep_##SFX(int q, int dir, const SweepArgs& a, hipStream_t st, int* partials);  \
  hipError_t dense_serial_##SFX(int q, int dir, const SerialArgs& a, hipStream_t st);               \
  hipError_t dense_resid_##SFX(int q, int dir, const ResidArgs& a, hipStream_t st, int* partials);  \
  hipError_t dense_grad_##SFX(int q, const GradArgs& a, hipStream_t st);
LP_DENSE_DECL(f32)
LP_DENSE_DECL(f64)
bool dense_width_supported(int q);

// Dense fp32 matrix-core family (lp_dense_mfma.hip), widths 32 and 64
bool mfma_width_supported(int q);
hipError_t mfma_sweep(int q, int dir, const SweepArgs& a, hipStream_t st, int* partials);
hipError_t mfma_serial(int q, int dir, const SerialArgs& a, hipStream_t st);
hipError_t mfma_grad(int q, const GradArgs& a, hipStream_t st);
int dense_grad_chunks(int B, int N);
// C-point storage (c = 4): forward F-relaxation of intervals k0 .. k0 + nk - 1 from the
// C-points Uc[k] (row k), writing fine layers 4 k0 .. 4 (k0 + nk) - 1 to rows 0 .. 4 nk - 1
// of Y, with the arithmetic of the sweeps (the F-point states a full-storage solve stores)
hipError_t mfma_expand(int q, int act, const void* K, const void* b, const void* Uc, void* Y, int B, long k0,
                       long nk, double h, hipStream_t st);
// the first pass of the gradient only (GradArgs.n0 selects the layers), and its second pass
hipError_t mfma_grad_partials(int q, const GradArgs& a, long nl, hipStream_t st);
hipError_t mfma_grad_finish(int q, const GradArgs& a, hipStream_t st);

// Dense fp32 matrix-core family for wide layers (lp_dense_wide.hip), width 220:
// the layer weights stream through LDS in panels
bool wide_width_supported(int q);
hipError_t wide_sweep(int q, int dir, const SweepArgs& a, hipStream_t st, int* partials);
hipError_t wide_serial(int q, int dir, const SerialArgs& a, hipStream_t st);
hipError_t wide_resid(int q, int dir, const ResidArgs& a, hipStream_t st, int* partials);
hipError_t wide_grad(int q, const GradArgs& a, hipStream_t st);

// Conv family (lp_conv.hip)
hipError_t conv_sweep(const Shape& s, int dir, const SweepArgs& a, hipStream_t st, int* partials);
hipError_t conv_serial(const Shape& s, int dir, const SerialArgs& a, hipStream_t st);
hipError_t conv_resid(const Shape& s, int dir, const ResidArgs& a, hipStream_t st, int* partials);
hipError_t conv_grad(const Shape& s, const GradArgs& a, hipStream_t st);
bool conv_supported(const Shape& s);
int conv_grad_chunks(int B, int N);
int conv_tile(const Shape& s);
size_t conv_dsig_block_bytes(const Shape& s);  // sigma' record bytes per (layer, example)

// Library-owned scratch of the allocation-free entry point (lp_noalloc.hip):
// its size, and its address on the current device (looked up once per device).
size_t noalloc_scratch_bytes();
hipError_t noalloc_scratch(void** ptr);

// Common kernels (lp_common.hip)
hipError_t launch_copy_rows(void* X, size_t slice_bytes, long src_row, long dst_row0,
                            long dst_step, long count, hipStream_t st);
hipError_t launch_norm_reduce(const double* partial, int n, double* out, hipStream_t st);
// Wait for st, then read the device's sticky non-finite-norm flag into *flag
// (host); clear it when set and `clear` is true.
hipError_t read_nonfinite(uint32_t* flag, bool clear, hipStream_t st);
hipError_t launch_zero(void* p, size_t bytes, hipStream_t st);
hipError_t launch_open_forward(const Shape& s, int opening, int nf, int B, const void* y, const void* L,
                               void* u0, hipStream_t st);
hipError_t launch_open_grad(const Shape& s, int opening, int nf, int B, const void* y, const void* L,
                            const void* lam0, void* dL, hipStream_t st);
hipError_t launch_loss(int dtype, int B, int q, int nc, const void* uN, const void* Wc, const void* mu,
                       const void* c, double* J, void* lamN, void* dW, void* dmu, void* ws, hipStream_t st);
size_t loss_workspace_bytes(size_t esz, int B, int q, int nc);         // lp_loss.hip: one class count
size_t loss_workspace_bytes_max(size_t esz, int B, int q, int nc_max);  // every class count <= nc_max
hipError_t launch_sgd(int dtype, size_t n, double lr, const void* g, void* x, hipStream_t st);
constexpr int DOT_BLOCKS = 256;  // partials of lp_vec_dot (out[1 .. DOT_BLOCKS])
hipError_t launch_axpby(int dtype, size_t n, double a, const void* x, double b, void* y, hipStream_t st);
hipError_t launch_dot(int dtype, size_t n, const void* x, const void* y, double* out, hipStream_t st);
hipError_t launch_accuracy(int dtype, int B, int q, int nc, const void* uN, const void* Wc, const void* mu,
                           const void* c, double* acc, void* ws, hipStream_t st);  // lp_loss.hip

}  // namespace lp
