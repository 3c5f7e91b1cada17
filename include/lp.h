/*
 * lp.h - C ABI of the MI355X layer-parallel ResNet library.
 *
 * The library solves the discrete state and adjoint equations of a residual
 * network viewed as forward Euler time stepping (Guenther, Ruthotto, Schroder,
 * Cyr, Gauger: "Layer-parallel training of deep residual neural networks",
 * arXiv:1812.04352), either layer-serially or with nonlinear multigrid reduction
 * in time (MGRIT with FAS, Section 3, Algorithm 1), and assembles the reduced
 * gradient with respect to the layer weights.
 *
 * Model (Section 2): per example, u^{n+1} = Phi(u^n, theta^n) = u^n + h sigma(K_n u^n + b_n),
 * n = 0..N-1, with K_n a dense q x q matrix or a 3x3 convolution with C channels
 * (zero "same" padding, cross-correlation), b_n a per-feature (dense) or
 * per-channel (conv) bias, sigma applied componentwise.
 *
 * Conventions for every call:
 *   - Pointers are DEVICE pointers unless the argument is marked (host).
 *   - The caller owns every buffer. The library never allocates device memory;
 *     calls that need scratch memory take a caller-provided workspace `ws` of
 *     `ws_bytes` bytes (see lp_workspace_bytes) and return LP_EWORKSPACE if it is
 *     too small or not 256-byte aligned.
 *   - All device work is enqueued on `stream` (a hipStream_t; NULL is the default
 *     stream). A call that returns a value computed on the device (res_hist,
 *     norm, or an iteration count decided by a stopping rule) waits for `stream`
 *     before returning; other calls return without waiting.
 *   - All floating-point arrays of one call have the problem's dtype
 *     (LP_F32: float, LP_F64: double). Layouts are row-major, contiguous:
 *       trajectory U, Lam  [N+1][B][q]     (conv: [N+1][B][C][H][W]); q = C*H*W
 *       weights K          [N][q][q]       K[n][i][j] maps input j to output i
 *                          (conv: [N][C][C][3][3], K[n][co][ci][ty][tx])
 *       bias b             [N][q]          (conv: [N][C])
 *   - U and Lam must not alias each other or the workspace.
 *   - Calls are re-entrant when given distinct workspaces and outputs.
 *   - Error behaviour: an argument check failing returns LP_EINVAL (or
 *     LP_EUNSUPPORTED for a valid but unimplemented combination) before any work
 *     is enqueued; lp_last_error() then names the argument. A HIP runtime failure
 *     returns LP_EHIP. A non-finite residual norm returns LP_ENONFINITE after the
 *     iteration that produced it (outputs then hold that iterate).
 */
#ifndef LP_H
#define LP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define LP_ABI_VERSION 4

typedef enum {
  LP_OK = 0,
  LP_EINVAL = 1,        /* bad argument (null pointer, bad size, bad enum, N_l % cf != 0) */
  LP_EUNSUPPORTED = 2,  /* valid but not implemented (e.g. a dense width with no kernel) */
  LP_EWORKSPACE = 3,    /* workspace too small or misaligned */
  LP_EHIP = 4,          /* HIP runtime error */
  LP_ENONFINITE = 5     /* residual norm became NaN or Inf */
} lp_status;

enum { LP_F32 = 0, LP_F64 = 1 };                       /* dtype */
enum { LP_DENSE = 0, LP_CONV3X3 = 1 };                 /* layer */
enum { LP_TANH = 0, LP_RELU = 1, LP_SMOOTHRELU = 2, LP_IDENTITY = 3 }; /* activation sigma */
enum { LP_RELAX_F = 0, LP_RELAX_FCF = 1, LP_RELAX_FCFCF = 2 }; /* MGRIT relaxation */
enum { LP_CYCLE_V = 0, LP_CYCLE_F = 1 };               /* MGRIT cycle */
enum { LP_STATE = 0, LP_ADJOINT = 1 };                 /* which system */
enum { LP_OPEN_IDENTITY = 0, LP_OPEN_DENSE_ACT = 1, LP_OPEN_CONV_ACT = 2 }; /* opening layer */
enum { LP_STORE_ALL = 0, LP_STORE_CPOINTS = 1 };       /* primal trajectory storage */

/* The network and batch (Section 2.2). Dense: C = width q, H = W = 1.
 * Conv: C channels of H x W pixels. h = T / N is the step size.
 * Kernels exist for dense widths 8, 16, 32, 64 (fp32 and fp64; fp64 up to 32)
 * and 220 (fp32, the hyperspectral network of Section 5.1), and for 3x3
 * convolutions with C = 8 channels and an even image height (fp32); other
 * shapes return LP_EUNSUPPORTED. */
typedef struct {
  int32_t abi_version;   /* must equal LP_ABI_VERSION */
  int32_t dtype;         /* LP_F32 | LP_F64 */
  int32_t layer;         /* LP_DENSE | LP_CONV3X3 */
  int32_t act;           /* LP_TANH | LP_RELU | LP_SMOOTHRELU | LP_IDENTITY */
  int32_t N;             /* residual layers (time steps), >= 1 */
  int32_t B;             /* batch size, >= 0 (0: calls do nothing) */
  int32_t C, H, W;       /* width / channels and image size */
  double h;              /* step size */
} lp_problem;

/* MGRIT schedule (Section 3.1, Algorithm 1, applied recursively).
 * Level l has N_l = N / cf^l steps of size cf^l h and uses the injected weights
 * theta^{i cf^l}. Levels are added while l+1 < max_levels and N_l > min_coarse;
 * every coarsened level must satisfy N_l % cf == 0 (else LP_EINVAL). The
 * coarsest level is solved by forward (adjoint: backward) substitution.
 * Step 3 of Algorithm 1 (the coarse solve) is one recursive cycle on the next
 * level for LP_CYCLE_V (a V-cycle); for LP_CYCLE_F it is a recursive F-cycle
 * followed by a V-cycle, the V-cycle left out when the next level is the
 * coarsest (the multigrid F-cycle, which visits the coarse levels more often;
 * Section 3.1.1 mentions it). Relaxation on every non-coarsest level:
 * LP_RELAX_F (F), LP_RELAX_FCF (F, C, F; the paper's default) or
 * LP_RELAX_FCFCF (F, C, F, C, F). */
typedef struct {
  int32_t cf;            /* coarsening factor c >= 2 */
  int32_t max_levels;    /* >= 1; 1 means a serial solve */
  int32_t min_coarse;    /* stop coarsening at N_l <= min_coarse (>= 1) */
  int32_t relax;         /* LP_RELAX_F | LP_RELAX_FCF | LP_RELAX_FCFCF, on every non-coarsest level */
  int32_t max_iter;      /* >= 1 cycles */
  int32_t warm_start;    /* 0: C-points start as copies of u^0 (adjoint: lam^N); 1: caller's array is the guess */
  double rtol;           /* stop after iteration m when rho_m <= rtol * rho_1 (0: off) */
  double stag;           /* stop after iteration m > 1 when rho_m > stag * rho_{m-1} (0: off) */
  int32_t cycle;         /* LP_CYCLE_V | LP_CYCLE_F */
  int32_t storage;       /* LP_STORE_ALL | LP_STORE_CPOINTS: how the primal trajectory is kept (below) */
} lp_mgrit;

/* Primal storage (Section 3.2, remark on storing or recomputing the states the
 * adjoint equations depend on). LP_STORE_ALL: the state trajectory U is
 * [N+1][B][q], every layer stored. LP_STORE_CPOINTS: U holds the fine C-points
 * only, Uc [N/cf + 1][B][q] with row k = u^{k cf} (a checkpoint per coarse
 * interval, cf times less memory). lp_mgrit_forward then writes only Uc (the
 * F-points of the returned iterate are the F-relaxation of its C-points, never
 * stored); lp_mgrit_adjoint, given Uc, recomputes each interval's F-point states
 * and sigma' from its lower C-point on the finest level (coarse levels use only
 * C-points); lp_gradient_cpoints does the same for the gradient. The recomputed
 * states equal the stored ones bit for bit, so both storages give the same
 * iterates and gradients. Implemented for fp32 dense widths 32 and 64 (the
 * matrix-core kernels) with cf = 4 and at least two levels; other problems
 * return LP_EUNSUPPORTED. No sigma' record is kept or read (dsig is ignored). */

int32_t lp_abi_version(void);
const char* lp_status_string(int32_t status);
/* Message of the last failing call on this host thread ("" if none). */
const char* lp_last_error(void);

/* Workspace bytes that lp_mgrit_forward, lp_mgrit_adjoint, lp_gradient,
 * lp_residual_norm and lp_loss_terminal need for this problem and schedule (mg
 * may be NULL: then the MGRIT hierarchy is not counted; with mg->storage =
 * LP_STORE_CPOINTS lp_gradient_cpoints is covered too). Returns 0 for an invalid
 * problem. The workspace holds the coarse levels (U_l and the FAS right-hand
 * side G_l for l >= 1), the relaxed C-points of every non-coarsest level,
 * per-workgroup residual partials (fp64) and per-chunk gradient partials. */
size_t lp_workspace_bytes(const lp_problem* prob, const lp_mgrit* mg);

/* Record of the activation derivative along a forward trajectory (optional in
 * every call that takes `dsig`): sigma'(K_n U[n] + b_n) for n = 0..N-1, the
 * factor the adjoint steps and the gradient apply (Section 3.2, Section 2.3).
 * Dense: layout [N][B][q] in the problem's element order, one value per
 * element: for LP_RELU one bit (widths 32 and 64: bit f of example e's q-bit
 * word, N B q / 8 bytes) or one byte 0 or 1 (width 220); the problem dtype for
 * LP_TANH and LP_SMOOTHRELU. Convolution: one block per (layer n, example e) at index
 * n B + e, in the convolution kernels' own tile order (LP_RELU: one 32-bit word
 * of decision bits per lane of each wave, covering its tiles of 16 pair-pixels;
 * else four fp32 values per lane of each tile); the record is only meaningful to
 * this library. No
 * storage for LP_IDENTITY (sigma' = 1). A forward call given `dsig` writes the
 * record of the trajectory it returns; an adjoint or gradient call given `dsig`
 * uses it instead of recomputing K_n U[n] + b_n from U (saving one layer
 * product per step), so it must hold the record of the U and the weights that
 * call receives. NULL: not written / recomputed from U.
 * Returns the record's size in bytes, or 0 where the kernels for this problem
 * keep none: an invalid problem, LP_IDENTITY, fp64, and dense widths other than
 * 32, 64 and 220 (the fp32 matrix-core kernels). Where it returns 0 every call
 * ignores `dsig`. */
size_t lp_dsig_bytes(const lp_problem* prob);

/* Layer-serial forward propagation (Section 2.3, state equations; the baseline
 * method): U[n+1] = Phi(U[n], theta^n) for n = 0..N-1.
 * U [N+1][B][q]: row 0 is read (u^0 = L_in y), rows 1..N are written.
 * dsig (nullable): the trajectory's sigma' record is written. */
int32_t lp_serial_forward(const lp_problem* prob, const void* K, const void* b, void* U,
                          void* dsig, void* stream);

/* Layer-serial adjoint propagation (Section 2.3, adjoint equations; this is
 * backpropagation): Lam[n] = (d_u Phi(U[n], theta^n))^T Lam[n+1]
 *                          = Lam[n+1] + h K_n^T (sigma'(K_n U[n] + b_n) * Lam[n+1]),
 * n = N-1..0. Lam row N is read (terminal value), rows 0..N-1 are written.
 * U is read only. dsig (nullable): the sigma' record of U. */
int32_t lp_serial_adjoint(const lp_problem* prob, const void* K, const void* b, const void* U,
                          const void* dsig, void* Lam, void* stream);

/* MGRIT solve of the state equations A(U, theta) = G (Section 3.1, the
 * space-time system and Algorithm 1 with FAS).
 * U [N+1][B][q]: row 0 is u^0 (read, never written); with warm_start the other
 * rows are the initial guess (only rows at multiples of cf are read), else they
 * are ignored; on return they hold the iterate after *iters V-cycles (every row
 * written, the last sweep being an F-relaxation). With mg->storage =
 * LP_STORE_CPOINTS, U is Uc [N/cf + 1][B][q] (row k = C-point k cf) and only
 * those rows are read and written.
 * res_hist (host, nullable, length >= max_iter): rho_m, m = 1..*iters, the fp64
 * norm ||G - A(U)|| over all examples and features, taken at the finest level's
 * C-points after the relaxation of iteration m (Algorithm 1, step 2).
 * iters (host, nullable): V-cycles run. Not converging within max_iter is not
 * an error.
 * With rtol = stag = 0 the call runs max_iter V-cycles; if res_hist is then
 * NULL it reads nothing back and returns without waiting for the stream; a
 * non-finite rho_m is then recorded on the device and reported by the next
 * lp_check_finite. A stopping rule makes the call read rho_m after every V-cycle.
 * dsig (nullable): the sigma' record of the returned iterate is written (by the
 * final F-relaxation, which then also takes the product of the layer before each
 * C-point). */
int32_t lp_mgrit_forward(const lp_problem* prob, const lp_mgrit* mg, const void* K,
                         const void* b, void* U, void* dsig, void* ws, size_t ws_bytes,
                         double* res_hist, int32_t* iters, void* stream);

/* MGRIT solve of the adjoint equations (Section 3.2, the adjoint space-time
 * system), linearised at the trajectory U (read only).
 * Lam [N+1][B][q]: row N is the terminal value (read, never written); with
 * warm_start the other rows are the initial guess (rows at multiples of cf are
 * read), else ignored; on return they hold the iterate. Coarse levels take the
 * adjoint step of size cf^l h linearised at the injected fine state U[i cf^l].
 * res_hist, iters as for lp_mgrit_forward, on the adjoint residual.
 * dsig (nullable): the sigma' record of U; every level then reads sigma' of the
 * injected fine state from it. With mg->storage = LP_STORE_CPOINTS, U is the
 * C-point trajectory Uc [N/cf + 1][B][q] of lp_mgrit_forward (Lam stays
 * [N+1][B][q]). */
int32_t lp_mgrit_adjoint(const lp_problem* prob, const lp_mgrit* mg, const void* K,
                         const void* b, const void* U, const void* dsig, void* Lam, void* ws,
                         size_t ws_bytes, double* res_hist, int32_t* iters, void* stream);

/* Reduced gradient with respect to the layer weights (Section 2.3, design
 * equations, without regularisation):
 *   s_k^n = sigma'(K_n u_k^n + b_n) * lam_k^{n+1}
 *   dK[n] = h sum_k s_k^n (u_k^n)^T   (conv: the weight gradient of the 3x3 cross-correlation)
 *   db[n] = h sum_k s_k^n             (conv: summed over pixels per channel)
 * summed over the batch in a fixed order (bitwise reproducible).
 * dK like K, db like b; both written. The 1/B factor of the mean loss is
 * expected inside Lam (it is part of the terminal value). dsig (nullable): the
 * sigma' record of U; the width-32 kernel with a smooth activation recomputes
 * sigma' even when given one (there an fp32 record row costs more HBM time than
 * the product it saves), with results equal to rounding. */
int32_t lp_gradient(const lp_problem* prob, const void* K, const void* b, const void* U,
                    const void* dsig, const void* Lam, void* dK, void* db, void* ws, size_t ws_bytes,
                    void* stream);

/* lp_gradient from a C-point-only trajectory (LP_STORE_CPOINTS, Section 3.2
 * remark): Uc [N/cf + 1][B][q] holds u^{k cf}; the states of every layer are
 * recomputed by forward steps from the C-points (a block of at most 64
 * intervals at a time, staged in the workspace) and the gradient is the one
 * lp_gradient gives for the full trajectory, bit for bit. cf must be 4 and the
 * problem an fp32 dense width 32 or 64 (else LP_EUNSUPPORTED). ws: at least
 * lp_workspace_bytes(prob, mg) bytes for an mg with storage = LP_STORE_CPOINTS. */
int32_t lp_gradient_cpoints(const lp_problem* prob, int32_t cf, const void* K, const void* b, const void* Uc,
                            const void* Lam, void* dK, void* db, void* ws, size_t ws_bytes, void* stream);

/* Full-grid residual norm ||G - A(U)|| of the space-time system, the quantity
 * whose drop stops the MGRIT iteration (Algorithm 1, step 6; Section 3.1.1 for
 * the state system, Section 3.2 for the adjoint one). fp64, summed over all
 * examples and features in a fixed order, returned on the host (the call waits
 * for `stream`):
 *   which = LP_STATE:   (sum_{n=1..N} ||Phi(U[n-1], theta^{n-1}) - U[n]||^2)^{1/2}
 *                       (row 0 of A(U) = G is u^0 itself and contributes nothing)
 *   which = LP_ADJOINT: (sum_{n=0..N-1} ||Lam[n+1] + h K_n^T(sigma'(z_n) * Lam[n+1]) - Lam[n]||^2)^{1/2}
 * U (and Lam) [N+1][B][q] are read only; Lam may be NULL for LP_STATE. ws: at
 * least lp_workspace_bytes(prob, NULL) bytes (per-workgroup partials). Returns
 * LP_ENONFINITE (with *norm set) when the norm is NaN or Inf. */
int32_t lp_residual_norm(const lp_problem* prob, int32_t which, const void* K, const void* b,
                         const void* U, const void* Lam, void* ws, size_t ws_bytes, double* norm,
                         void* stream);

/* lp_residual_norm without a workspace, for callers that cannot allocate
 * device memory or own a workspace (serving loops that check convergence
 * between requests, harnesses that forbid allocation). It computes exactly what
 * lp_residual_norm computes, with the same kernels and summation order (equal
 * results bit for bit), and allocates nothing: the per-workgroup partials and
 * the result go to a scratch array of 16 MiB + 256 bytes that the library holds
 * in device memory, one per GPU from the first call on it until the process
 * ends. Limit: problems needing more than 2^21 partials ((N+1) ceil(B/32) for
 * dense layers, (N+1) B for convolutions) return LP_EWORKSPACE before any work
 * is enqueued. The scratch needs no clearing (every call writes what it reads),
 * but it is shared by every call on a GPU: calls that overlap on one GPU (other
 * host threads, other streams) race and must be serialised by the caller. Waits
 * for `stream` like lp_residual_norm, so it cannot be captured in a graph. */
int32_t lp_residual_norm_noalloc(const lp_problem* prob, int32_t which, const void* K, const void* b,
                                 const void* U, const void* Lam, double* norm, void* stream);

/* Report a non-finite residual norm that no call has read back. Every residual
 * norm the library computes on a device (each MGRIT iteration's rho_m, and
 * lp_residual_norm) that is NaN or Inf sets a sticky flag on that device,
 * whether or not the computing call read the norm back. This call waits for
 * `stream`, reads the flag of the current device and clears it: LP_ENONFINITE
 * if it was set, else LP_OK. Callers that run solves without a read-back (no
 * stopping rule, no res_hist) call it where they next synchronise, e.g. once
 * per training update, so that a diverging iterate is never used silently.
 * The flag is shared by all streams on the device. */
int32_t lp_check_finite(void* stream);

/* ---- boundary helpers (outside the per-iteration hot path) ---- */

/* Opening layer u^0 = L_in y (Section 2.1), written to u0 [B][q]:
 *   LP_OPEN_IDENTITY:  u0 = y                       (y [B][q])
 *   LP_OPEN_DENSE_ACT: u0 = sigma(L_in y)           (y [B][nf], L_in [q][nf])
 *   LP_OPEN_CONV_ACT:  u0 = sigma(conv3x3(L_in, y)) (y [B][1][H][W], L_in [C][1][3][3], no bias)
 * nf is the input feature count (ignored for the conv opening). */
int32_t lp_open_forward(const lp_problem* prob, int32_t opening, int32_t nf, const void* y,
                        const void* L_in, void* u0, void* stream);

/* Gradient of the opening weights, dL_in = sum_k (sigma'(L_in y_k) * lam_k^0) y_k^T
 * (conv: weight gradient of the opening convolution); dL_in like L_in. */
int32_t lp_open_grad(const lp_problem* prob, int32_t opening, int32_t nf, const void* y,
                     const void* L_in, const void* lam0, void* dL_in, void* stream);

/* Softmax cross-entropy at the network output (Section 2.1) for class-probability
 * rows c [B][nc] (one-hot in all workloads), z = W u^N + mu, W [nc][q], mu [nc]:
 *   J      = (1/B) sum_k -c_k^T log softmax(z_k)          (fp64, written to J[0] on the device)
 *   lamN   = (1/B) W^T (softmax(z_k) - c_k)   [B][q]      (the adjoint terminal value)
 *   dW     = (1/B) sum_k (softmax(z_k) - c_k) (u_k^N)^T   [nc][q]
 *   dmu    = (1/B) sum_k (softmax(z_k) - c_k)             [nc]
 * Requires 1 <= nc <= 64. The workspace holds the logits and fixed-order
 * partial sums; lp_workspace_bytes(prob, ...) covers every nc <= 64. */
int32_t lp_loss_terminal(const lp_problem* prob, int32_t nc, const void* uN, const void* W,
                         const void* mu, const void* c, double* J, void* lamN, void* dW,
                         void* dmu, void* ws, size_t ws_bytes, void* stream);

/* Plain gradient step x <- x - lr * g on n elements of the given dtype (the
 * design update of Algorithm 2 with a scaled-identity Hessian approximation). */
int32_t lp_sgd_update(int32_t dtype, size_t n, double lr, const void* g, void* x, void* stream);

/* Vector algebra of the design update of Algorithm 2 with a limited-memory
 * BFGS Hessian approximation (Section 4; the two-loop recursion runs on the
 * host over these calls), on n elements of the given dtype:
 *   lp_vec_axpby: y <- a x + b y (b = 0: y <- a x, whatever y held);
 *   lp_vec_dot:   out[0] <- sum_i x_i y_i, accumulated in fp64 in a fixed order
 *                 (bitwise reproducible); out is a device array of at least
 *                 1 + LP_DOT_PARTIALS doubles, out[1..] being scratch. */
#define LP_DOT_PARTIALS 256
int32_t lp_vec_axpby(int32_t dtype, size_t n, double a, const void* x, double b, void* y, void* stream);
int32_t lp_vec_dot(int32_t dtype, size_t n, const void* x, const void* y, double* out, void* stream);

/* Classification accuracy at the network output (the validation measure of
 * Algorithm 2's stopping test, Section 4): the fraction of the B examples
 * whose predicted class argmax_j (W u_k^N + mu)_j, logits in fp64, equals the
 * class of their one-hot row c (first index on ties, on both sides).
 * uN [B][q], W [nc][q], mu [nc], c [B][nc] (problem dtype); acc: one device
 * double. ws: device workspace of at least lp_workspace_bytes(prob, NULL) bytes. */
int32_t lp_accuracy(const lp_problem* prob, int32_t nc, const void* uN, const void* W, const void* mu,
                    const void* c, double* acc, void* ws, size_t ws_bytes, void* stream);

/* ---- tracing (a profiling aid, not part of the method) ----
 * When enabled for a kernel kind, every launch of that kind records a pair of
 * HIP events on the launch's stream; lp_trace_read sums their elapsed times.
 * Kinds: the three sweeps of a non-coarsest MGRIT level, the coarsest-level
 * solve, for each direction; the gradient; the residual norm; layer-serial solves. */
enum {
  LP_TRACE_FWD_FC = 0, LP_TRACE_FWD_FRES = 1, LP_TRACE_FWD_CORRF = 2, LP_TRACE_FWD_COARSEST = 3,
  LP_TRACE_ADJ_FC = 4, LP_TRACE_ADJ_FRES = 5, LP_TRACE_ADJ_CORRF = 6, LP_TRACE_ADJ_COARSEST = 7,
  LP_TRACE_GRADIENT = 8, LP_TRACE_RESIDUAL = 9, LP_TRACE_SERIAL = 10, LP_TRACE_KINDS = 11
};
/* Start recording the kinds in `kind_mask` (bit k = kind k; 0 stops) and clear
 * earlier records. At most 65536 launches are recorded; later ones are counted
 * as dropped. Returns LP_OK or LP_EHIP. */
int32_t lp_trace_enable(uint32_t kind_mask);
/* Wait for the recorded events and report, for one kind and MGRIT level
 * (level -1: all levels), the launch count (host) and summed milliseconds (host). */
int32_t lp_trace_read(int32_t kind, int32_t level, int32_t* launches, double* total_ms);

#ifdef __cplusplus
}
#endif

#endif /* LP_H */
