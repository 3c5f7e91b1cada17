// Dense residual layers on the vector ALUs: one thread per example, the state
// row held in registers across the steps of an interval, the layer weights
// K_n, b_n staged through LDS (double-buffered: the next layer's weights are
// fetched while the current step computes) and read as broadcasts.
//
// Forward step (Section 2.2, forward Euler):  v <- v + h_l sigma(K_n v + b_n) (+ g)
// Adjoint step (Section 3.2):                 v <- v + h_l K_n^T (sigma'(K_n u^n + b_n) * v) (+ g)
// MGRIT sweeps follow Algorithm 1 (Section 3.1) with the F/C relaxations of
// eqs. Frelax / Crelax and FAS restriction by injection.
//
// The activation is a uniform runtime value; the dtype T and the width Q are
// template parameters (the row lives in registers), and each sweep mode is its
// own kernel symbol so profiles attribute time per mode.
// Included once per dtype by lp_dense_f32.hip / lp_dense_f64.hip.
#pragma once

#include "lp_device.h"
#include "lp_internal.h"

namespace lp {
namespace dense {

constexpr int NT = 256;  // threads (= examples) per workgroup

template <typename T, int Q>
struct WStage {
  static constexpr int n = Q * Q + Q;            // K_n then b_n
  static constexpr int per = (n + NT - 1) / NT;  // elements per thread when staging
};

template <typename T, int Q>
using WReg = T[WStage<T, Q>::per];

template <typename T, int Q>
__device__ __forceinline__ void fetch_w(WReg<T, Q>& r, const T* __restrict__ K, const T* __restrict__ b,
                                        size_t n) {
  const T* Kn = K + n * (size_t)(Q * Q);
  const T* bn = b + n * (size_t)Q;
#pragma unroll
  for (int p = 0; p < WStage<T, Q>::per; ++p) {
    const int idx = threadIdx.x + p * NT;
    if (idx < Q * Q) r[p] = Kn[idx];
    else if (idx < WStage<T, Q>::n) r[p] = bn[idx - Q * Q];
  }
}

template <typename T, int Q>
__device__ __forceinline__ void put_w(T* sh, const WReg<T, Q>& r) {
#pragma unroll
  for (int p = 0; p < WStage<T, Q>::per; ++p) {
    const int idx = threadIdx.x + p * NT;
    if (idx < WStage<T, Q>::n) sh[idx] = r[p];
  }
}

// z_i = sum_j W[i][j] v_j + W[Q*Q + i] (W in LDS, read as broadcasts).
// Between the forward and the transposed product of one adjoint step: the
// transposed product reads the weights from LDS again instead of keeping the
// forward product's q^2 + q values live, which at q = 8 in fp64 lowers the
// adjoint sweep from 196 to 126 registers (two to four waves per SIMD; measured
// 5 % faster on the Peaks-shaped workload).
__device__ __forceinline__ void reload_weights() { asm volatile("" ::: "memory"); }

template <typename T, int Q>
__device__ __forceinline__ void matvec(T (&z)[Q], const T (&v)[Q], const T* __restrict__ W) {
  using V = typename Vec16<T>::type;
  constexpr int nv = Vec16<T>::n;
#pragma unroll
  for (int i = 0; i < Q; ++i) {
    const V* kr = reinterpret_cast<const V*>(W + i * Q);
    T acc = T(0);
#pragma unroll
    for (int jj = 0; jj < Q / nv; ++jj) {
      const V kv = kr[jj];
      if constexpr (nv == 4) {
        acc = fma(kv.x, v[4 * jj + 0], acc);
        acc = fma(kv.y, v[4 * jj + 1], acc);
        acc = fma(kv.z, v[4 * jj + 2], acc);
        acc = fma(kv.w, v[4 * jj + 3], acc);
      } else {
        acc = fma(kv.x, v[2 * jj + 0], acc);
        acc = fma(kv.y, v[2 * jj + 1], acc);
      }
    }
    z[i] = acc + W[Q * Q + i];
  }
}

// w_j = sum_i W[i][j] s_i (K^T s), accumulated over i in order.
template <typename T, int Q>
__device__ __forceinline__ void matvec_t(T (&w)[Q], const T (&s)[Q], const T* __restrict__ W) {
  using V = typename Vec16<T>::type;
  constexpr int nv = Vec16<T>::n;
#pragma unroll
  for (int j = 0; j < Q; ++j) w[j] = T(0);
#pragma unroll
  for (int i = 0; i < Q; ++i) {
    const V* kr = reinterpret_cast<const V*>(W + i * Q);
#pragma unroll
    for (int jj = 0; jj < Q / nv; ++jj) {
      const V kv = kr[jj];
      if constexpr (nv == 4) {
        w[4 * jj + 0] = fma(kv.x, s[i], w[4 * jj + 0]);
        w[4 * jj + 1] = fma(kv.y, s[i], w[4 * jj + 1]);
        w[4 * jj + 2] = fma(kv.z, s[i], w[4 * jj + 2]);
        w[4 * jj + 3] = fma(kv.w, s[i], w[4 * jj + 3]);
      } else {
        w[2 * jj + 0] = fma(kv.x, s[i], w[2 * jj + 0]);
        w[2 * jj + 1] = fma(kv.y, s[i], w[2 * jj + 1]);
      }
    }
  }
}

// sigma (or sigma') over a whole row; `act` is uniform, so one branch per row.
template <typename T, int Q, bool DERIV>
__device__ __forceinline__ void apply_act(T (&z)[Q], int act) {
  if (act == ACT_TANH) {
#pragma unroll
    for (int i = 0; i < Q; ++i) z[i] = DERIV ? dact_f<T, ACT_TANH>(z[i]) : act_f<T, ACT_TANH>(z[i]);
  } else if (act == ACT_RELU) {
#pragma unroll
    for (int i = 0; i < Q; ++i) z[i] = DERIV ? dact_f<T, ACT_RELU>(z[i]) : act_f<T, ACT_RELU>(z[i]);
  } else if (act == ACT_SMOOTHRELU) {
#pragma unroll
    for (int i = 0; i < Q; ++i)
      z[i] = DERIV ? dact_f<T, ACT_SMOOTHRELU>(z[i]) : act_f<T, ACT_SMOOTHRELU>(z[i]);
  } else if (DERIV) {
#pragma unroll
    for (int i = 0; i < Q; ++i) z[i] = T(1);
  }
}

template <typename T, int Q>
__device__ __forceinline__ void add_row(T (&v)[Q], const T* __restrict__ g) {
  T t[Q];
  load_row<T, Q>(t, g);
#pragma unroll
  for (int i = 0; i < Q; ++i) v[i] += t[i];
}

// U^{kc} + E with E = V - U (Algorithm 1, steps 4-5)
template <typename T, int Q>
__device__ __forceinline__ void correct_row(T (&v)[Q], const T* __restrict__ cs, const T* __restrict__ vs) {
  T cv[Q], vv[Q];
  load_row<T, Q>(cv, cs);
  load_row<T, Q>(vv, vs);
#pragma unroll
  for (int i = 0; i < Q; ++i) v[i] = cv[i] + (vv[i] - cv[i]);
}

// ------------------------------------------------------------------ forward sweep
// Interval k covers level points kc .. (k+1)c; step j goes from point kc+j to
// kc+j+1 with the fine weights of index (kc+j)*stride and step size h_l.
//   FC:    start from C-point kc; c steps (c-1 F-points, then the C-point (k+1)c)
//          -> S[k+1]; interval 0 also copies C-point 0 to S[0].
//   FRES:  start from relaxed C_k; c steps give f_{k+1} = Phi(u^{(k+1)c-1}) + g;
//          r = f - C_{k+1}; restriction: G'[k+1] = f - Phi_{l+1}(C_k), X'[k+1] = C_{k+1}.
//   CORRF: correct C_k with the coarse solution, then c-1 F steps written to X;
//          the last interval also corrects C-point N_l.
template <typename T, int Q, int MODE>
__global__ __launch_bounds__(NT) void k_fwd_sweep(SweepArgs a) {
  __shared__ T W[2][WStage<T, Q>::n];
  __shared__ double red[NT];
  constexpr int mode = MODE;  // one kernel symbol per sweep mode
  const int k = blockIdx.x;
  const int Nc = gridDim.x;
  const int e = blockIdx.y * NT + threadIdx.x;
  const bool on = e < a.B;
  const size_t slice = (size_t)a.B * Q;
  const size_t row = (size_t)(on ? e : 0) * Q;
  const T* K = static_cast<const T*>(a.K);
  const T* bb = static_cast<const T*>(a.b);
  T* X = static_cast<T*>(a.X);
  const T* G = static_cast<const T*>(a.G);
  const T* Cs = static_cast<const T*>(a.Cs);
  const T* Vn = static_cast<const T*>(a.V);
  const int c = a.c;
  const int nsteps = mode == SWEEP_CORRF ? c - 1 : c;
  const T hl = (T)a.hl;
  const T hc = (T)a.hc;
  const long kc = (long)k * c;

  WReg<T, Q> wr;
  fetch_w<T, Q>(wr, K, bb, (size_t)kc * a.stride);
  put_w<T, Q>(W[0], wr);
  __syncthreads();

  T v[Q];
  if (on) {
    if (mode == SWEEP_FC) {
      // a pending coarse-grid correction of the previous cycle is applied on the fly
      if (Vn) correct_row<T, Q>(v, Cs + (size_t)k * a.cs_stride * slice + row, Vn + (size_t)k * slice + row);
      else load_row<T, Q>(v, X + kc * slice + row);
      if (k == 0) store_row<T, Q>(static_cast<T*>(a.S) + row, v);
    } else if (mode == SWEEP_FRES) {
      load_row<T, Q>(v, Cs + (size_t)k * a.cs_stride * slice + row);
    } else {
      correct_row<T, Q>(v, Cs + (size_t)k * a.cs_stride * slice + row, Vn + (size_t)k * slice + row);
      if (k > 0) store_row<T, Q>(X + kc * slice + row, v);
    }
  }
  T coarse[Q];
  for (int j = 0; j < nsteps; ++j) {
    if (j + 1 < nsteps) fetch_w<T, Q>(wr, K, bb, (size_t)(kc + j + 1) * a.stride);
    if (on) {
      T s[Q];
      matvec<T, Q>(s, v, W[j & 1]);
      apply_act<T, Q, false>(s, a.act);
      if (mode == SWEEP_FRES && j == 0) {
        // coarse step Phi_{l+1} from the same C-point with the same weights
#pragma unroll
        for (int i = 0; i < Q; ++i) coarse[i] = v[i] + hc * s[i];
      }
#pragma unroll
      for (int i = 0; i < Q; ++i) v[i] = v[i] + hl * s[i];
      if (G) add_row<T, Q>(v, G + (kc + j + 1) * slice + row);
      if (mode == SWEEP_CORRF) store_row<T, Q>(X + (kc + j + 1) * slice + row, v);
    }
    if (j + 1 < nsteps) put_w<T, Q>(W[(j + 1) & 1], wr);
    __syncthreads();
  }

  if (mode == SWEEP_FC) {
    if (on) store_row<T, Q>(static_cast<T*>(a.S) + (size_t)(k + 1) * slice + row, v);
  } else if (mode == SWEEP_FRES) {
    double acc = 0.0;
    if (on) {
      T cn[Q];
      load_row<T, Q>(cn, Cs + (size_t)(k + 1) * a.cs_stride * slice + row);
#pragma unroll
      for (int i = 0; i < Q; ++i) {
        const T r = v[i] - cn[i];
        acc += (double)r * (double)r;
        coarse[i] = v[i] - coarse[i];  // g_{l+1}^{k+1} = f_{k+1} - Phi_{l+1}(C_k)
      }
      store_row<T, Q>(static_cast<T*>(a.Gn) + (size_t)(k + 1) * slice + row, coarse);
      if (a.xn_every > 0 && (k + 1) % a.xn_every == 0)
        store_row<T, Q>(static_cast<T*>(a.Xn) + (size_t)(k + 1) * slice + row, cn);
      if (k == 0) {
        load_row<T, Q>(cn, Cs + row);
        store_row<T, Q>(static_cast<T*>(a.Xn) + row, cn);
      }
    }
    if (a.partial) {
      const double s = block_sum<NT>(acc, red);
      if (threadIdx.x == 0) a.partial[(size_t)blockIdx.x * gridDim.y + blockIdx.y] = s;
    }
  } else {
    if (on && k == Nc - 1) {
      correct_row<T, Q>(v, Cs + (size_t)Nc * a.cs_stride * slice + row, Vn + (size_t)Nc * slice + row);
      store_row<T, Q>(X + (size_t)a.Nl * slice + row, v);
    }
  }
}

// ------------------------------------------------------------------ adjoint sweep
// Interval k runs from its upper C-point (k+1)c down to kc; step j produces
// point i = (k+1)c-1-j from point i+1, linearised at the fine state of index
// i*stride with the weights of that index.
//   FC:    start from C-point (k+1)c; c steps -> S[k]; the last interval copies
//          the terminal C-point to S[Nc].
//   FRES:  start from relaxed C_{k+1}; c steps give f_k; r = f_k - C_k;
//          G'[k] = f_k - Phibar_{l+1}(C_{k+1}), X'[k] = C_k.
//   CORRF: correct C_{k+1}, then c-1 F steps written to X; interval 0 also
//          corrects C-point 0.
template <typename T, int Q, int MODE>
__global__ __launch_bounds__(NT) void k_adj_sweep(SweepArgs a) {
  __shared__ T W[2][WStage<T, Q>::n];
  __shared__ double red[NT];
  constexpr int mode = MODE;  // one kernel symbol per sweep mode
  const int k = blockIdx.x;
  const int Nc = gridDim.x;
  const int e = blockIdx.y * NT + threadIdx.x;
  const bool on = e < a.B;
  const size_t slice = (size_t)a.B * Q;
  const size_t row = (size_t)(on ? e : 0) * Q;
  const T* K = static_cast<const T*>(a.K);
  const T* bb = static_cast<const T*>(a.b);
  const T* Uf = static_cast<const T*>(a.Uf);
  T* X = static_cast<T*>(a.X);
  const T* G = static_cast<const T*>(a.G);
  const T* Cs = static_cast<const T*>(a.Cs);
  const T* Vn = static_cast<const T*>(a.V);
  const int c = a.c;
  const int nsteps = mode == SWEEP_CORRF ? c - 1 : c;
  const T hl = (T)a.hl;
  const T hc = (T)a.hc;
  const long top = (long)(k + 1) * c;

  WReg<T, Q> wr;
  fetch_w<T, Q>(wr, K, bb, (size_t)(top - 1) * a.stride);
  put_w<T, Q>(W[0], wr);
  __syncthreads();

  T v[Q];
  T coarse[Q];  // FRES: holds C_{k+1} until the last step, then the coarse step
  if (on) {
    if (mode == SWEEP_FC) {
      if (Vn)
        correct_row<T, Q>(v, Cs + (size_t)(k + 1) * a.cs_stride * slice + row, Vn + (size_t)(k + 1) * slice + row);
      else load_row<T, Q>(v, X + top * slice + row);
      if (k == Nc - 1) store_row<T, Q>(static_cast<T*>(a.S) + (size_t)Nc * slice + row, v);
    } else if (mode == SWEEP_FRES) {
      load_row<T, Q>(v, Cs + (size_t)(k + 1) * a.cs_stride * slice + row);
#pragma unroll
      for (int i = 0; i < Q; ++i) coarse[i] = v[i];
    } else {
      correct_row<T, Q>(v, Cs + (size_t)(k + 1) * a.cs_stride * slice + row, Vn + (size_t)(k + 1) * slice + row);
      if (k + 1 < Nc) store_row<T, Q>(X + top * slice + row, v);
    }
  }
  for (int j = 0; j < nsteps; ++j) {
    const long i = top - 1 - j;
    if (j + 1 < nsteps) fetch_w<T, Q>(wr, K, bb, (size_t)(i - 1) * a.stride);
    if (on) {
      T d[Q], w[Q];
      {
        T u[Q];
        load_row<T, Q>(u, Uf + (size_t)i * a.stride * slice + row);
        matvec<T, Q>(d, u, W[j & 1]);
        apply_act<T, Q, true>(d, a.act);
      }
      reload_weights();
      if (mode == SWEEP_FRES && j == c - 1) {
        // coarse adjoint step from the upper C-point, linearised at the same fine state
#pragma unroll
        for (int q = 0; q < Q; ++q) w[q] = d[q] * coarse[q];
        T w2[Q];
        matvec_t<T, Q>(w2, w, W[j & 1]);
#pragma unroll
        for (int q = 0; q < Q; ++q) coarse[q] = coarse[q] + hc * w2[q];
      }
#pragma unroll
      for (int q = 0; q < Q; ++q) d[q] *= v[q];
      matvec_t<T, Q>(w, d, W[j & 1]);
#pragma unroll
      for (int q = 0; q < Q; ++q) v[q] = v[q] + hl * w[q];
      if (G) add_row<T, Q>(v, G + (size_t)i * slice + row);
      if (mode == SWEEP_CORRF) store_row<T, Q>(X + (size_t)i * slice + row, v);
    }
    if (j + 1 < nsteps) put_w<T, Q>(W[(j + 1) & 1], wr);
    __syncthreads();
  }

  if (mode == SWEEP_FC) {
    if (on) store_row<T, Q>(static_cast<T*>(a.S) + (size_t)k * slice + row, v);
  } else if (mode == SWEEP_FRES) {
    double acc = 0.0;
    if (on) {
      T ck[Q];
      load_row<T, Q>(ck, Cs + (size_t)k * a.cs_stride * slice + row);
#pragma unroll
      for (int q = 0; q < Q; ++q) {
        const T r = v[q] - ck[q];
        acc += (double)r * (double)r;
        coarse[q] = v[q] - coarse[q];  // g_{l+1}^k = f_k - Phibar_{l+1}(C_{k+1})
      }
      store_row<T, Q>(static_cast<T*>(a.Gn) + (size_t)k * slice + row, coarse);
      if (a.xn_every > 0 && k % a.xn_every == 0)
        store_row<T, Q>(static_cast<T*>(a.Xn) + (size_t)k * slice + row, ck);
      if (k == Nc - 1) {
        load_row<T, Q>(ck, Cs + (size_t)Nc * a.cs_stride * slice + row);
        store_row<T, Q>(static_cast<T*>(a.Xn) + (size_t)Nc * slice + row, ck);
      }
    }
    if (a.partial) {
      const double s = block_sum<NT>(acc, red);
      if (threadIdx.x == 0) a.partial[(size_t)blockIdx.x * gridDim.y + blockIdx.y] = s;
    }
  } else {
    if (on && k == 0) {
      correct_row<T, Q>(v, Cs + row, Vn + row);
      store_row<T, Q>(X + row, v);
    }
  }
}

// ------------------------------------------------------------------ serial solves
// Forward: X[i+1] = Phi(X[i]) + G[i+1], i = 0..Nl-1 (forward substitution).
// Adjoint: X[i] = Phibar_i(X[i+1]) + G[i], i = Nl-1..0 (backward substitution).

template <typename T, int Q>
__global__ __launch_bounds__(NT) void k_fwd_serial(SerialArgs a) {
  __shared__ T W[2][WStage<T, Q>::n];
  const int e = blockIdx.x * NT + threadIdx.x;
  const bool on = e < a.B;
  const size_t slice = (size_t)a.B * Q;
  const size_t row = (size_t)(on ? e : 0) * Q;
  const T* K = static_cast<const T*>(a.K);
  const T* bb = static_cast<const T*>(a.b);
  T* X = static_cast<T*>(a.X);
  const T* G = static_cast<const T*>(a.G);
  const T hl = (T)a.hl;
  WReg<T, Q> wr;
  fetch_w<T, Q>(wr, K, bb, 0);
  put_w<T, Q>(W[0], wr);
  __syncthreads();
  T v[Q];
  if (on) load_row<T, Q>(v, X + row);
  for (int i = 0; i < a.Nl; ++i) {
    if (i + 1 < a.Nl) fetch_w<T, Q>(wr, K, bb, (size_t)(i + 1) * a.stride);
    if (on) {
      T s[Q];
      matvec<T, Q>(s, v, W[i & 1]);
      apply_act<T, Q, false>(s, a.act);
#pragma unroll
      for (int q = 0; q < Q; ++q) v[q] = v[q] + hl * s[q];
      if (G) add_row<T, Q>(v, G + (size_t)(i + 1) * slice + row);
      store_row<T, Q>(X + (size_t)(i + 1) * slice + row, v);
    }
    if (i + 1 < a.Nl) put_w<T, Q>(W[(i + 1) & 1], wr);
    __syncthreads();
  }
}

template <typename T, int Q>
__global__ __launch_bounds__(NT) void k_adj_serial(SerialArgs a) {
  __shared__ T W[2][WStage<T, Q>::n];
  const int e = blockIdx.x * NT + threadIdx.x;
  const bool on = e < a.B;
  const size_t slice = (size_t)a.B * Q;
  const size_t row = (size_t)(on ? e : 0) * Q;
  const T* K = static_cast<const T*>(a.K);
  const T* bb = static_cast<const T*>(a.b);
  const T* Uf = static_cast<const T*>(a.Uf);
  T* X = static_cast<T*>(a.X);
  const T* G = static_cast<const T*>(a.G);
  const T hl = (T)a.hl;
  WReg<T, Q> wr;
  fetch_w<T, Q>(wr, K, bb, (size_t)(a.Nl - 1) * a.stride);
  put_w<T, Q>(W[0], wr);
  __syncthreads();
  T v[Q];
  if (on) load_row<T, Q>(v, X + (size_t)a.Nl * slice + row);
  for (int j = 0; j < a.Nl; ++j) {
    const long i = a.Nl - 1 - j;
    if (j + 1 < a.Nl) fetch_w<T, Q>(wr, K, bb, (size_t)(i - 1) * a.stride);
    if (on) {
      T d[Q], w[Q];
      {
        T u[Q];
        load_row<T, Q>(u, Uf + (size_t)i * a.stride * slice + row);
        matvec<T, Q>(d, u, W[j & 1]);
        apply_act<T, Q, true>(d, a.act);
      }
      reload_weights();
#pragma unroll
      for (int q = 0; q < Q; ++q) d[q] *= v[q];
      matvec_t<T, Q>(w, d, W[j & 1]);
#pragma unroll
      for (int q = 0; q < Q; ++q) v[q] = v[q] + hl * w[q];
      if (G) add_row<T, Q>(v, G + (size_t)i * slice + row);
      store_row<T, Q>(X + (size_t)i * slice + row, v);
    }
    if (j + 1 < a.Nl) put_w<T, Q>(W[(j + 1) & 1], wr);
    __syncthreads();
  }
}

// ------------------------------------------------------------------ residuals
// Workgroup (n, tile): forward r = Phi_n(U[n]) - U[n+1]; adjoint
// r = Phibar_n(Lam[n+1]) - Lam[n]; writes the tile's sum of r^2.

template <typename T, int Q, int DIR>
__global__ __launch_bounds__(NT) void k_resid(ResidArgs a) {
  __shared__ T W[WStage<T, Q>::n];
  __shared__ double red[NT];
  const int e = blockIdx.y * NT + threadIdx.x;
  const bool on = e < a.B;
  const size_t slice = (size_t)a.B * Q;
  const size_t row = (size_t)(on ? e : 0) * Q;
  const T* U = static_cast<const T*>(a.U);
  const T* L = static_cast<const T*>(a.Lam);
  const T h = (T)a.h;
  const int n = blockIdx.x;
  {
    WReg<T, Q> wr;
    fetch_w<T, Q>(wr, static_cast<const T*>(a.K), static_cast<const T*>(a.b), n);
    put_w<T, Q>(W, wr);
  }
  __syncthreads();
  double acc = 0.0;
  if (on) {
    T v[Q], t[Q];
    load_row<T, Q>(v, U + (size_t)n * slice + row);
    matvec<T, Q>(t, v, W);
    if constexpr (DIR == DIR_FWD) {
      apply_act<T, Q, false>(t, a.act);
      T nx[Q];
      load_row<T, Q>(nx, U + (size_t)(n + 1) * slice + row);
#pragma unroll
      for (int q = 0; q < Q; ++q) {
        const T r = (v[q] + h * t[q]) - nx[q];
        acc += (double)r * (double)r;
      }
    } else {
      apply_act<T, Q, true>(t, a.act);
      reload_weights();
      T lam[Q];
      load_row<T, Q>(lam, L + (size_t)(n + 1) * slice + row);
#pragma unroll
      for (int q = 0; q < Q; ++q) t[q] *= lam[q];
      T w[Q];
      matvec_t<T, Q>(w, t, W);
      load_row<T, Q>(v, L + (size_t)n * slice + row);
#pragma unroll
      for (int q = 0; q < Q; ++q) {
        const T r = (lam[q] + h * w[q]) - v[q];
        acc += (double)r * (double)r;
      }
    }
  }
  const double s = block_sum<NT>(acc, red);
  if (threadIdx.x == 0) a.partial[(size_t)blockIdx.x * gridDim.y + blockIdx.y] = s;
}

// ------------------------------------------------------------------ gradient

constexpr int GT = 64;  // examples per LDS tile

template <typename T, int Q>
struct GStage {
  static constexpr int ld = Q + 1;                   // padded tile row
  static constexpr int nout = Q * Q + Q;
  static constexpr int per = (Q * Q + NT - 1) / NT;  // dK entries per thread
};

// First pass: grid (N, nchunks). Workgroup (n, chunk) reduces its chunk of the
// batch for layer n into partial[n][chunk][Q*Q + Q]: s = sigma'(K_n u + b_n) * lam^{n+1}
// per example, then dK[i][j] += s_i u_j and db[i] += s_i over the examples in order.
template <typename T, int Q>
__global__ __launch_bounds__(NT) void k_grad_partial(GradArgs a) {
  __shared__ T W[WStage<T, Q>::n];
  __shared__ T ut[GT * GStage<T, Q>::ld];
  __shared__ T st[GT * GStage<T, Q>::ld];
  constexpr int ld = GStage<T, Q>::ld;
  constexpr int PER = GStage<T, Q>::per;
  constexpr int TPE = NT / GT;                // threads per example in the sigma' phase
  constexpr int QP = (Q + TPE - 1) / TPE;     // rows of K per such thread
  const int n = blockIdx.x;
  const int chunk = blockIdx.y;
  const int per_chunk = (((a.B + a.nchunks - 1) / a.nchunks) + GT - 1) / GT * GT;
  const int e0 = chunk * per_chunk;
  const int e1 = min(a.B, e0 + per_chunk);
  const size_t slice = (size_t)a.B * Q;
  const T* U = static_cast<const T*>(a.U) + (size_t)n * slice;
  const T* L = static_cast<const T*>(a.Lam) + (size_t)(n + 1) * slice;
  {
    WReg<T, Q> wr;
    fetch_w<T, Q>(wr, static_cast<const T*>(a.K), static_cast<const T*>(a.b), n);
    put_w<T, Q>(W, wr);
  }
  T acc[PER];
#pragma unroll
  for (int p = 0; p < PER; ++p) acc[p] = T(0);
  T accb = T(0);
  for (int t0 = e0; t0 < e1; t0 += GT) {
    const int nt = min(GT, e1 - t0);
    __syncthreads();
    for (int idx = threadIdx.x; idx < GT * Q; idx += NT) {
      const int r = idx / Q, q = idx - r * Q;
      T uv = T(0), lv = T(0);
      if (r < nt) {
        uv = U[(size_t)(t0 + r) * Q + q];
        lv = L[(size_t)(t0 + r) * Q + q];
      }
      ut[r * ld + q] = uv;
      st[r * ld + q] = lv;
    }
    __syncthreads();
    {
      const int r = threadIdx.x / TPE;
      const int part = threadIdx.x % TPE;
      T z[QP];
#pragma unroll
      for (int p = 0; p < QP; ++p) {
        const int i = part * QP + p;
        T accz = T(0);
        if (i < Q) {
#pragma unroll 8
          for (int j = 0; j < Q; ++j) accz = fma(W[i * Q + j], ut[r * ld + j], accz);
          accz += W[Q * Q + i];
        }
        z[p] = accz;
      }
      apply_act<T, QP, true>(z, a.act);
#pragma unroll
      for (int p = 0; p < QP; ++p) {
        const int i = part * QP + p;
        if (i < Q) st[r * ld + i] *= z[p];
      }
    }
    __syncthreads();
    for (int r = 0; r < nt; ++r) {
#pragma unroll
      for (int p = 0; p < PER; ++p) {
        const int o = threadIdx.x + p * NT;
        if (o < Q * Q) {
          const int i = o / Q, j = o - i * Q;
          acc[p] = fma(st[r * ld + i], ut[r * ld + j], acc[p]);
        }
      }
      if ((int)threadIdx.x < Q) accb += st[r * ld + threadIdx.x];
    }
  }
  T* out = static_cast<T*>(a.partial) + ((size_t)n * a.nchunks + chunk) * GStage<T, Q>::nout;
#pragma unroll
  for (int p = 0; p < PER; ++p) {
    const int o = threadIdx.x + p * NT;
    if (o < Q * Q) out[o] = acc[p];
  }
  if ((int)threadIdx.x < Q) out[Q * Q + threadIdx.x] = accb;
}

// Second pass: sum the chunk partials in chunk order (in fp64) and scale by h.
template <typename T>
__global__ __launch_bounds__(NT) void k_grad_final(GradArgs a, int nw, int nbias) {
  const int nout = nw + nbias;
  const size_t tot = (size_t)a.N * nout;
  const size_t o = (size_t)blockIdx.x * NT + threadIdx.x;
  if (o >= tot) return;
  const size_t n = o / nout;
  const size_t r = o - n * nout;
  const T* p = static_cast<const T*>(a.partial) + n * a.nchunks * nout + r;
  double s = 0.0;  // chunk partials summed in fp64
  for (int ch = 0; ch < a.nchunks; ++ch) s += (double)p[(size_t)ch * nout];
  const T v = (T)(s * a.h);
  if (r < (size_t)nw) static_cast<T*>(a.dK)[n * nw + r] = v;
  else static_cast<T*>(a.db)[n * nbias + (r - nw)] = v;
}

// ------------------------------------------------------------------ launchers

template <typename T, int Q>
hipError_t sweep(int dir, const SweepArgs& a, hipStream_t st, int* partials) {
  const dim3 grid(a.Nl / a.c, (a.B + NT - 1) / NT);
  if (partials) *partials = (int)(grid.x * grid.y);
  if (dir == DIR_FWD) {
    if (a.mode == SWEEP_FC) launch(k_fwd_sweep<T, Q, SWEEP_FC>, grid, NT, 0, st, a);
    else if (a.mode == SWEEP_FRES) launch(k_fwd_sweep<T, Q, SWEEP_FRES>, grid, NT, 0, st, a);
    else launch(k_fwd_sweep<T, Q, SWEEP_CORRF>, grid, NT, 0, st, a);
  } else {
    if (a.mode == SWEEP_FC) launch(k_adj_sweep<T, Q, SWEEP_FC>, grid, NT, 0, st, a);
    else if (a.mode == SWEEP_FRES) launch(k_adj_sweep<T, Q, SWEEP_FRES>, grid, NT, 0, st, a);
    else launch(k_adj_sweep<T, Q, SWEEP_CORRF>, grid, NT, 0, st, a);
  }
  return hipGetLastError();
}

template <typename T, int Q>
hipError_t serial(int dir, const SerialArgs& a, hipStream_t st) {
  const dim3 grid((a.B + NT - 1) / NT);
  if (dir == DIR_FWD) launch(k_fwd_serial<T, Q>, grid, NT, 0, st, a);
  else launch(k_adj_serial<T, Q>, grid, NT, 0, st, a);
  return hipGetLastError();
}

template <typename T, int Q>
hipError_t resid(int dir, const ResidArgs& a, hipStream_t st, int* partials) {
  const dim3 grid(a.N, (a.B + NT - 1) / NT);
  if (partials) *partials = (int)(grid.x * grid.y);
  if (dir == DIR_FWD) launch(k_resid<T, Q, DIR_FWD>, grid, NT, 0, st, a);
  else launch(k_resid<T, Q, DIR_ADJ>, grid, NT, 0, st, a);
  return hipGetLastError();
}

template <typename T, int Q>
hipError_t grad(const GradArgs& a, hipStream_t st) {
  launch(k_grad_partial<T, Q>, dim3(a.N, a.nchunks), NT, 0, st, a);
  const hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  const size_t tot = (size_t)a.N * (Q * Q + Q);
  launch(k_grad_final<T>, (unsigned)((tot + NT - 1) / NT), NT, 0, st, a, Q * Q, Q);
  return hipGetLastError();
}

}  // namespace dense
}  // namespace lp

// Defines the per-dtype entry points dense_*_SFX over the supported widths.
#define LP_DENSE_DEFINE(T, SFX, WIDE)                                                                        \
  namespace lp {                                                                                       \
  hipError_t dense_sweep_##SFX(int q, int dir, const SweepArgs& a, hipStream_t st, int* partials) {    \
    switch (q) {                                                                                       \
      case 8: return dense::sweep<T, 8>(dir, a, st, partials);                                         \
      case 16: return dense::sweep<T, 16>(dir, a, st, partials);                                       \
      case 32: return dense::sweep<T, 32>(dir, a, st, partials);                                       \
      case 64: if (WIDE) return dense::sweep<T, (WIDE ? 64 : 8)>(dir, a, st, partials); break;                                       \
    }                                                                                                  \
    return hipErrorNotSupported;                                                                       \
  }                                                                                                    \
  hipError_t dense_serial_##SFX(int q, int dir, const SerialArgs& a, hipStream_t st) {                 \
    switch (q) {                                                                                       \
      case 8: return dense::serial<T, 8>(dir, a, st);                                                  \
      case 16: return dense::serial<T, 16>(dir, a, st);                                                \
      case 32: return dense::serial<T, 32>(dir, a, st);                                                \
      case 64: if (WIDE) return dense::serial<T, (WIDE ? 64 : 8)>(dir, a, st); break;                                                \
    }                                                                                                  \
    return hipErrorNotSupported;                                                                       \
  }                                                                                                    \
  hipError_t dense_resid_##SFX(int q, int dir, const ResidArgs& a, hipStream_t st, int* partials) {    \
    switch (q) {                                                                                       \
      case 8: return dense::resid<T, 8>(dir, a, st, partials);                                         \
      case 16: return dense::resid<T, 16>(dir, a, st, partials);                                       \
      case 32: return dense::resid<T, 32>(dir, a, st, partials);                                       \
      case 64: if (WIDE) return dense::resid<T, (WIDE ? 64 : 8)>(dir, a, st, partials); break;                                       \
    }                                                                                                  \
    return hipErrorNotSupported;                                                                       \
  }                                                                                                    \
  hipError_t dense_grad_##SFX(int q, const GradArgs& a, hipStream_t st) {                              \
    switch (q) {                                                                                       \
      case 8: return dense::grad<T, 8>(a, st);                                                         \
      case 16: return dense::grad<T, 16>(a, st);                                                       \
      case 32: return dense::grad<T, 32>(a, st);                                                       \
      case 64: if (WIDE) return dense::grad<T, (WIDE ? 64 : 8)>(a, st); break;                                                       \
    }                                                                                                  \
    return hipErrorNotSupported;                                                                       \
  }                                                                                                    \
  }
