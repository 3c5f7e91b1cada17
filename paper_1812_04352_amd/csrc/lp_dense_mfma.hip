// Dense fp32 residual layers of width 32 or 64 on the matrix cores (gfx950
// v_mfma_f32_16x16x4_f32 for the sweeps and serial solves,
// v_mfma_f32_32x32x2_f32 for the gradient).
//
// One wave owns EX examples (16 or 32) for all steps of an interval. The layer
// product z = K_n v is a (q x q) x (q x EX) contraction: M = output feature,
// N = example, K = input feature. Its accumulator layout (see Lay below) is also
// a valid B-operand layout for the next step once the contraction index is
// permuted the same way in the A operand, so chained steps never move the state
// between lanes. K_n and b_n are staged in LDS (row-major, padded rows,
// double-buffered: the next layer is fetched into registers while the current
// step runs); the bias initialises the accumulators.
//
// Forward step (Section 2.2):  v <- v + h_l sigma(K_n v + b_n) (+ g)
// Adjoint step (Section 3.2):  v <- v + h_l K_n^T (sigma'(K_n u^n + b_n) * v) (+ g);
//   the transposed product reads K_n column-wise from the same LDS copy.
// Sweep modes follow Algorithm 1 exactly as the VALU kernels do (lp_dense_impl.h).
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <type_traits>

#include "lp_device.h"
#include "lp_internal.h"

namespace lp {
namespace mfma {

typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int MODE_SERIAL = 3;  // SweepArgs.mode of a whole-level serial solve (k_ser_fwd, k_ser_adj)

// tanh(x) = sign(x) (1 - t) / (1 + t) with t = exp(-2|x|), on the hardware exp2
// and reciprocal; absolute error a few ulp of 1.
__device__ __forceinline__ float tanh_fast(float x) {
  const float t = __builtin_amdgcn_exp2f(-2.885390081777927f * fabsf(x));  // 2 log2(e) |x|
  return copysignf((1.f - t) * __builtin_amdgcn_rcpf(1.f + t), x);
}

template <int Q, int WAVES>
struct Cfg {
  static constexpr int NT = 64 * WAVES;
  static constexpr int MB = Q / 32;               // 32-feature blocks
  static constexpr int LD = Q + 4;                // padded LDS row (floats)
  static constexpr int WSZ = (Q + 1) * LD;        // K rows, then the bias row
  static constexpr int PK = (Q * Q / 4 + NT - 1) / NT;  // float4s of K_n per thread when staging
  static constexpr bool PART = Q * Q / 4 % NT != 0;      // the last float4 slot is not every thread's
};

typedef float f32x4 __attribute__((ext_vector_type(4)));

// One layer's weights in flight between global memory and LDS.
template <int Q, int WAVES>
struct WRegs {
  f32x4 k[Cfg<Q, WAVES>::PK];
  f32x4 b;  // threads < Q/4 carry four bias entries
};

template <int Q, int WAVES>
__device__ __forceinline__ void w_fetch(WRegs<Q, WAVES>& r, const float* __restrict__ K,
                                        const float* __restrict__ b, size_t n) {
  using C = Cfg<Q, WAVES>;
  const f32x4* Kn = reinterpret_cast<const f32x4*>(K + n * (size_t)(Q * Q));
#pragma unroll
  for (int p = 0; p < C::PK; ++p) {
    const int idx = threadIdx.x + p * C::NT;
    r.k[p] = (!C::PART || idx < Q * Q / 4) ? Kn[idx] : f32x4{};
  }
  r.b = threadIdx.x < Q / 4 ? reinterpret_cast<const f32x4*>(b + n * (size_t)Q)[threadIdx.x] : f32x4{};
}

template <int Q, int WAVES>
__device__ __forceinline__ void w_put(float* sh, const WRegs<Q, WAVES>& r) {
  using C = Cfg<Q, WAVES>;
#pragma unroll
  for (int p = 0; p < C::PK; ++p) {
    const int idx = threadIdx.x + p * C::NT;
    if (C::PART && idx >= Q * Q / 4) continue;
    const int el = idx * 4, row = el / Q, col = el - row * Q;
    *reinterpret_cast<f32x4*>(sh + row * C::LD + col) = r.k[p];
  }
  if (threadIdx.x < Q / 4) *reinterpret_cast<f32x4*>(sh + Q * C::LD + threadIdx.x * 4) = r.b;
}

// ------------------------------------------------------------------ layouts
// Per-lane layout of a wave's examples in the accumulators of the two fp32
// matrix-core shapes (lane l):
//   EX = 32, v_mfma_f32_32x32x2_f32: register r of block mb holds feature
//            32mb + 8(r/4) + 4(l/32) + r%4 of example l%32;
//   EX = 16, v_mfma_f32_16x16x4_f32: register r of block mb holds feature
//            16mb + 4(l/16) + r of example l%16.
// In both, the accumulators are the next product's B operand once the A
// operand's contraction index is permuted the same way (k-slice (mb, r) takes
// the feature that register r of block mb holds in each lane group), so chained
// steps never move state between lanes. A wave of the 16-example shape does half
// the work per step with half the latency and needs about two thirds of the
// registers; the sweeps and the serial solve use it, the gradient the other.
// ReLU's sigma' record: one bit per element in element order ([N][B][q], bit f of
// example e's q-bit word, q = 32 or 64), so an example's decisions are one 32- or
// 64-bit word. off is an element offset inside the example's row; the row starts
// at off - off % Q, a multiple of 32 elements, so the word is aligned.
template <int Q>
struct MaskWord {
  static_assert(Q == 32 || Q == 64, "bit records exist for widths 32 and 64");
  using T = typename std::conditional<Q == 64, unsigned long long, uint32_t>::type;
  __device__ static T load(const uint8_t* rec, size_t off) {
    return *reinterpret_cast<const T*>(rec + (off - off % Q) / 8);
  }
  __device__ static void store(uint8_t* rec, size_t off, T w) { *reinterpret_cast<T*>(rec + (off - off % Q) / 8) = w; }
  // 32-bit half i of the word (bits 32 i .. 32 i + 31), shifted right by s: lanes
  // shift once by their own offset and then read bits at constant positions
  __device__ static uint32_t half(T w, int i, int s) { return (uint32_t)(i ? (uint64_t)w >> 32 : w) >> s; }
  // the word from its halves, after an OR over lanes l, l ^ 16, l ^ 32, l ^ 48 (the
  // lanes of one example)
  __device__ static T combine(uint32_t lo, uint32_t hi) {
    lo |= __shfl_xor(lo, 16, 64);
    lo |= __shfl_xor(lo, 32, 64);
    if constexpr (Q == 64) {
      hi |= __shfl_xor(hi, 16, 64);
      hi |= __shfl_xor(hi, 32, 64);
      return ((T)hi << 32) | lo;
    } else {
      return lo;
    }
  }
};
__device__ __forceinline__ float mask_bit(uint32_t h, int b) { return (h >> b) & 1u ? 1.f : 0.f; }

template <int Q, int EX>
struct Lay;

template <int Q>
struct Lay<Q, 32> {
  using V = f32x16;
  static constexpr int NB = Q / 32, NV = 16;

  // p points at the example's row + 4*(lane/32)
  __device__ static void load(V (&v)[NB], const float* __restrict__ p) {
#pragma unroll
    for (int mb = 0; mb < NB; ++mb)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const f32x4 x = *reinterpret_cast<const f32x4*>(p + 32 * mb + 8 * g);
#pragma unroll
        for (int t = 0; t < 4; ++t) v[mb][4 * g + t] = x[t];
      }
  }

  __device__ static void store(float* __restrict__ p, const V (&v)[NB]) {
#pragma unroll
    for (int mb = 0; mb < NB; ++mb)
#pragma unroll
      for (int g = 0; g < 4; ++g)
        *reinterpret_cast<f32x4*>(p + 32 * mb + 8 * g) =
            f32x4{v[mb][4 * g + 0], v[mb][4 * g + 1], v[mb][4 * g + 2], v[mb][4 * g + 3]};
  }

  // sigma' record of ReLU (bits, MaskWord), off at the lane's element offset
  // e Q + 4 (lane / 32): value (mb, 4 g + t) is feature 32 mb + 8 g + 4 (lane / 32) + t
  __device__ static void load_mask(V (&v)[NB], const uint8_t* __restrict__ rec, size_t off) {
    const auto w = MaskWord<Q>::load(rec, off);
    const int h4 = (int)(off % Q);
#pragma unroll
    for (int mb = 0; mb < NB; ++mb) {
      const uint32_t h = MaskWord<Q>::half(w, mb, h4);
#pragma unroll
      for (int g = 0; g < 4; ++g)
#pragma unroll
        for (int t = 0; t < 4; ++t) v[mb][4 * g + t] = mask_bit(h, 8 * g + t);
    }
  }

  // z = K_n v + b_n (W: staged weights, row-major with row pitch LD, bias row last)
  template <int LD>
  __device__ static void prod(V (&z)[NB], const V (&v)[NB], const float* W, int lane) {
    const int h = lane >> 5, i = lane & 31;
#pragma unroll
    for (int ob = 0; ob < NB; ++ob) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const f32x4 bb = *reinterpret_cast<const f32x4*>(W + Q * LD + 32 * ob + 8 * g + 4 * h);
#pragma unroll
        for (int t = 0; t < 4; ++t) z[ob][4 * g + t] = bb[t];
      }
      const float* rowp = W + (32 * ob + i) * LD + 4 * h;
#pragma unroll
      for (int ib = 0; ib < NB; ++ib)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const f32x4 a4 = *reinterpret_cast<const f32x4*>(rowp + 32 * ib + 8 * g);
#pragma unroll
          for (int t = 0; t < 4; ++t)
            z[ob] = __builtin_amdgcn_mfma_f32_32x32x2f32(a4[t], v[ib][4 * g + t], z[ob], 0, 0, 0);
        }
    }
  }

  // w = K_n^T s (column reads of the staged K_n)
  template <int LD>
  __device__ static void prod_t(V (&w)[NB], const V (&s)[NB], const float* W, int lane) {
    const int h = lane >> 5, i = lane & 31;
#pragma unroll
    for (int ob = 0; ob < NB; ++ob) {
      w[ob] = 0.f;
      const float* colp = W + 32 * ob + i + 4 * h * LD;
#pragma unroll
      for (int ib = 0; ib < NB; ++ib) {
        // the block's 16 column values are read before its products start
        float a[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) a[r] = colp[(32 * ib + 8 * (r >> 2) + (r & 3)) * LD];
#pragma unroll
        for (int r = 0; r < 16; ++r) w[ob] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[r], s[ib][r], w[ob], 0, 0, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 16, 0);  // LDS reads
        __builtin_amdgcn_sched_group_barrier(0x008, 16, 0);  // then the products
      }
    }
  }
};

template <int Q>
struct Lay<Q, 16> {
  using V = f32x4;
  static constexpr int NB = Q / 16, NV = 4;

  // p points at the example's row + 4*(lane/16)
  __device__ static void load(V (&v)[NB], const float* __restrict__ p) {
#pragma unroll
    for (int mb = 0; mb < NB; ++mb) v[mb] = *reinterpret_cast<const f32x4*>(p + 16 * mb);
  }

  __device__ static void store(float* __restrict__ p, const V (&v)[NB]) {
#pragma unroll
    for (int mb = 0; mb < NB; ++mb) *reinterpret_cast<f32x4*>(p + 16 * mb) = v[mb];
  }

  // sigma' record of ReLU (bits, MaskWord), off at the lane's element offset
  // e Q + 4 (lane / 16): value (mb, r) is feature 16 mb + 4 (lane / 16) + r
  __device__ static void load_mask(V (&v)[NB], const uint8_t* __restrict__ rec, size_t off) {
    unpack_mask(v, MaskWord<Q>::load(rec, off), (int)(off % Q));
  }
  // g4 = 4 (lane / 16): value (mb, r) is bit 16 (mb % 2) + r of half mb / 2, shifted by g4
  __device__ static void unpack_mask(V (&v)[NB], typename MaskWord<Q>::T w, int g4) {
#pragma unroll
    for (int i = 0; i < (NB + 1) / 2; ++i) {
      const uint32_t h = MaskWord<Q>::half(w, i, g4);
#pragma unroll
      for (int mb = 2 * i; mb < NB && mb < 2 * i + 2; ++mb)
#pragma unroll
        for (int r = 0; r < 4; ++r) v[mb][r] = mask_bit(h, 16 * (mb % 2) + r);
    }
  }

  // the four lanes of an example hold disjoint bits of its word: they are combined
  // across lanes (every lane of the wave must call this) and one of them stores it
  __device__ static void store_mask(uint8_t* __restrict__ rec, size_t off, const V (&v)[NB], bool on) {
    const int g4 = (int)(off % Q);
    uint32_t h[2] = {0u, 0u};
#pragma unroll
    for (int mb = 0; mb < NB; ++mb)
#pragma unroll
      for (int r = 0; r < 4; ++r) h[mb / 2] |= (v[mb][r] != 0.f ? 1u : 0u) << (16 * (mb % 2) + r);
    const auto w = MaskWord<Q>::combine(h[0] << g4, h[1] << g4);
    if (on && g4 == 0) MaskWord<Q>::store(rec, off, w);
  }

  // z = K_n v + b_n: A operand of slice (ib, r) in lane l is K[16ob + l%16][16ib + 4(l/16) + r].
  // At width 64 (DB) the A operands (and bias) of output block ob + 1 are read
  // from LDS while block ob's products run, so the products do not wait on LDS
  // latency; the extra registers are what DB = false saves.
  template <int LD, bool DB = true>
  __device__ static void prod(V (&z)[NB], const V (&v)[NB], const float* W, int lane) {
    const int g = lane >> 4, i = lane & 15;
    if constexpr (NB < 4 || !DB) {
      // width 32: two blocks, few registers to spare (up to eight waves per SIMD)
#pragma unroll
      for (int ob = 0; ob < NB; ++ob) {
        z[ob] = *reinterpret_cast<const f32x4*>(W + Q * LD + 16 * ob + 4 * g);
        const float* rowp = W + (16 * ob + i) * LD + 4 * g;
#pragma unroll
        for (int ib = 0; ib < NB; ++ib) {
          const f32x4 a4 = *reinterpret_cast<const f32x4*>(rowp + 16 * ib);
#pragma unroll
          for (int r = 0; r < 4; ++r) z[ob] = __builtin_amdgcn_mfma_f32_16x16x4f32(a4[r], v[ib][r], z[ob], 0, 0, 0);
        }
      }
      return;
    }
    f32x4 A[2][NB], bz[2];
    auto rd = [&](int buf, int ob) {
      bz[buf] = *reinterpret_cast<const f32x4*>(W + Q * LD + 16 * ob + 4 * g);
      const float* rowp = W + (16 * ob + i) * LD + 4 * g;
#pragma unroll
      for (int ib = 0; ib < NB; ++ib) A[buf][ib] = *reinterpret_cast<const f32x4*>(rowp + 16 * ib);
    };
    rd(0, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, NB + 1, 0);  // block 0's LDS reads
#pragma unroll
    for (int ob = 0; ob < NB; ++ob) {
      const int cb = ob & 1;
      if (ob + 1 < NB) rd(cb ^ 1, ob + 1);
      z[ob] = bz[cb];
#pragma unroll
      for (int ib = 0; ib < NB; ++ib)
#pragma unroll
        for (int r = 0; r < 4; ++r) z[ob] = __builtin_amdgcn_mfma_f32_16x16x4f32(A[cb][ib][r], v[ib][r], z[ob], 0, 0, 0);
      if (ob + 1 < NB) __builtin_amdgcn_sched_group_barrier(0x100, NB + 1, 0);  // next block's LDS reads
      __builtin_amdgcn_sched_group_barrier(0x008, 4 * NB, 0);                 // then this block's products
    }
  }

  // w = K_n^T s: A operand of slice (ib, r) in lane l is K[16ib + 4(l/16) + r][16ob + l%16]
  // (column reads of the staged K_n), double-buffered across output blocks as in prod.
  template <int LD, bool DB = true>
  __device__ static void prod_t(V (&w)[NB], const V (&s)[NB], const float* W, int lane) {
    const int g = lane >> 4, i = lane & 15;
    if constexpr (NB < 4 || !DB) {
#pragma unroll
      for (int ob = 0; ob < NB; ++ob) {
        w[ob] = 0.f;
        const float* colp = W + 16 * ob + i + 4 * g * LD;
        float a[NB][4];
#pragma unroll
        for (int ib = 0; ib < NB; ++ib)
#pragma unroll
          for (int r = 0; r < 4; ++r) a[ib][r] = colp[(16 * ib + r) * LD];
#pragma unroll
        for (int ib = 0; ib < NB; ++ib)
#pragma unroll
          for (int r = 0; r < 4; ++r) w[ob] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[ib][r], s[ib][r], w[ob], 0, 0, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 4 * NB, 0);  // LDS reads
        __builtin_amdgcn_sched_group_barrier(0x008, 4 * NB, 0);  // then the products
      }
      return;
    }
    float A[2][NB][4];
    auto rd = [&](int buf, int ob) {
      const float* colp = W + 16 * ob + i + 4 * g * LD;
#pragma unroll
      for (int ib = 0; ib < NB; ++ib)
#pragma unroll
        for (int r = 0; r < 4; ++r) A[buf][ib][r] = colp[(16 * ib + r) * LD];
    };
    rd(0, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, 4 * NB, 0);  // block 0's LDS reads
#pragma unroll
    for (int ob = 0; ob < NB; ++ob) {
      const int cb = ob & 1;
      if (ob + 1 < NB) rd(cb ^ 1, ob + 1);
      w[ob] = 0.f;
#pragma unroll
      for (int ib = 0; ib < NB; ++ib)
#pragma unroll
        for (int r = 0; r < 4; ++r) w[ob] = __builtin_amdgcn_mfma_f32_16x16x4f32(A[cb][ib][r], s[ib][r], w[ob], 0, 0, 0);
      if (ob + 1 < NB) __builtin_amdgcn_sched_group_barrier(0x100, 4 * NB, 0);  // next block's LDS reads
      __builtin_amdgcn_sched_group_barrier(0x008, 4 * NB, 0);                 // then this block's products
    }
  }
};

template <typename V, int NB>
__device__ __forceinline__ void add_to(V (&v)[NB], const V (&t)[NB]) {
#pragma unroll
  for (int mb = 0; mb < NB; ++mb) v[mb] += t[mb];
}

// sigma (deriv = false) or sigma' (deriv = true) of every value, one branch on the
// activation for the whole array
template <typename V, int NB, int NV>
__device__ __forceinline__ void apply(V (&z)[NB], int act, bool deriv) {
  switch (act) {
    case ACT_TANH:
#pragma unroll
      for (int mb = 0; mb < NB; ++mb)
#pragma unroll
        for (int r = 0; r < NV; ++r) {
          const float t = tanh_fast(z[mb][r]);
          z[mb][r] = deriv ? 1.f - t * t : t;
        }
      break;
    case ACT_RELU:
#pragma unroll
      for (int mb = 0; mb < NB; ++mb)
#pragma unroll
        for (int r = 0; r < NV; ++r)
          z[mb][r] = deriv ? (z[mb][r] > 0.f ? 1.f : 0.f) : (z[mb][r] > 0.f ? z[mb][r] : 0.f);
      break;
    case ACT_SMOOTHRELU:
#pragma unroll
      for (int mb = 0; mb < NB; ++mb)
#pragma unroll
        for (int r = 0; r < NV; ++r)
          z[mb][r] = deriv ? dact_f<float, ACT_SMOOTHRELU>(z[mb][r]) : act_f<float, ACT_SMOOTHRELU>(z[mb][r]);
      break;
    default:
      if (deriv) {
#pragma unroll
        for (int mb = 0; mb < NB; ++mb) z[mb] = 1.f;
      }
      break;
  }
}

// v = c + (v' - c) (Algorithm 1, the coarse-grid correction of a C-point)
template <typename Lt>
__device__ __forceinline__ void correct(typename Lt::V (&v)[Lt::NB], const float* cs, const float* vs) {
  typename Lt::V cv[Lt::NB], vv[Lt::NB];
  Lt::load(cv, cs);
  Lt::load(vv, vs);
#pragma unroll
  for (int mb = 0; mb < Lt::NB; ++mb) v[mb] = cv[mb] + (vv[mb] - cv[mb]);
}

// Sum of squares of (a - b) over the lane's values, in fp64.
template <typename V, int NB, int NV>
__device__ __forceinline__ double sq_diff(const V (&a)[NB], const V (&b)[NB]) {
  double acc = 0.0;
#pragma unroll
  for (int mb = 0; mb < NB; ++mb)
#pragma unroll
    for (int r = 0; r < NV; ++r) {
      const float d = a[mb][r] - b[mb][r];
      acc += (double)d * (double)d;
    }
  return acc;
}

// The sigma' record at element offset off: bits for ReLU (MaskWord), fp32 otherwise.
template <typename Lt>
__device__ __forceinline__ void load_dsig(typename Lt::V (&d)[Lt::NB], const void* rec, size_t off, int act) {
  if (act == ACT_RELU) Lt::load_mask(d, static_cast<const uint8_t*>(rec), off);
  else Lt::load(d, static_cast<const float*>(rec) + off);
}

// on: whether the lane's example exists; every lane of the wave calls this (the
// ReLU bits of an example are gathered across its lanes)
template <typename Lt>
__device__ __forceinline__ void store_dsig(void* rec, size_t off, int act, const typename Lt::V (&d)[Lt::NB], bool on) {
  if (act == ACT_RELU) Lt::store_mask(static_cast<uint8_t*>(rec), off, d, on);
  else if (on) Lt::store(static_cast<float*>(rec) + off, d);
}

// Fixed-order workgroup sum of one double per lane; result in thread 0.
template <int WAVES>
__device__ __forceinline__ double wg_sum(double v, double* red) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  double s = 0.0;
  if (threadIdx.x == 0)
    for (int w = 0; w < WAVES; ++w) s += red[w];
  return s;
}

// ------------------------------------------------------------------ forward
// Interval k = blockIdx.y, examples of blockIdx.x.
// Consecutive workgroups share an interval, so the round-robin dispatch over the
// 8 XCDs gives each XCD every interval's weights once, in order, and its L2 only
// has to hold the few intervals in flight (with the interval as the fast index,
// an XCD received all tiles of every 8th interval and its weights overflowed L2
// at N = 2048, q = 64).
template <int Q, int MODE, int WAVES, int EX, bool REC>
__global__ __launch_bounds__(64 * WAVES) void k_fwd(SweepArgs a) {
  using C = Cfg<Q, WAVES>;
  using Lt = Lay<Q, EX>;
  using V = typename Lt::V;
  constexpr int NB = Lt::NB, NV = Lt::NV;
  __shared__ float W[2][C::WSZ];
  __shared__ double red[WAVES];
  const int lane = threadIdx.x & 63;
  const int k = blockIdx.y;
  const int Nc = gridDim.y;
  const int e = (blockIdx.x * WAVES + (threadIdx.x >> 6)) * EX + (lane % EX);
  const bool on = e < a.B;
  const size_t slice = (size_t)a.B * Q;
  const size_t row = (size_t)(on ? e : 0) * Q + 4 * (lane / EX);
  const float* K = static_cast<const float*>(a.K);
  const float* bb = static_cast<const float*>(a.b);
  float* X = static_cast<float*>(a.X);
  const float* G = static_cast<const float*>(a.G);
  const float* Cs = static_cast<const float*>(a.Cs);
  const float* Vn = static_cast<const float*>(a.V);
  const int c = a.c;
  const int nsteps = MODE == SWEEP_CORRF ? c - 1 : c;
  const float hl = (float)a.hl, hc = (float)a.hc;
  const long kc = (long)k * c;

  WRegs<Q, WAVES> wr;
  w_fetch<Q, WAVES>(wr, K, bb, (size_t)kc * a.stride);
  w_put<Q, WAVES>(W[0], wr);
  __syncthreads();

  V v[NB];
#pragma unroll
  for (int mb = 0; mb < NB; ++mb) v[mb] = 0.f;
  if (on) {
    if (MODE == SWEEP_FC) {
      // a pending coarse-grid correction of the previous cycle is applied on the fly
      if (MODE == SWEEP_FC && Vn)
        correct<Lt>(v, Cs + (size_t)k * a.cs_stride * slice + row, Vn + (size_t)k * slice + row);
      else Lt::load(v, X + kc * slice + row);
      if (MODE == SWEEP_FC && k == 0) Lt::store(static_cast<float*>(a.S) + row, v);
    } else if (MODE == SWEEP_FRES) {
      Lt::load(v, Cs + (size_t)k * a.cs_stride * slice + row);
    } else {
      correct<Lt>(v, Cs + (size_t)k * a.cs_stride * slice + row, Vn + (size_t)k * slice + row);
      if (k > 0) Lt::store(X + kc * slice + row, v);
    }
  }
  V coarse[NB];
  // the final F-relaxation records sigma'(z) of every layer, and also takes the
  // product of the layer before the next C-point
  constexpr bool rec = REC && MODE == SWEEP_CORRF;
  constexpr int extra = rec ? 1 : 0;
  for (int j = 0; j < nsteps; ++j) {
    // prefetch the next layer (the last step re-fetches its own, or the extra one)
    w_fetch<Q, WAVES>(wr, K, bb, (size_t)(kc + (j + 1 < nsteps ? j + 1 : j + extra)) * a.stride);
    V s[NB];
    Lt::template prod<C::LD>(s, v, W[j & 1], lane);
    if constexpr (rec) {
      V dz[NB];
#pragma unroll
      for (int mb = 0; mb < NB; ++mb) dz[mb] = s[mb];
      apply<V, NB, NV>(dz, a.act, true);
      store_dsig<Lt>(a.dsig, (size_t)(kc + j) * a.stride * slice + row, a.act, dz, on);
    }
    apply<V, NB, NV>(s, a.act, false);
    if (MODE == SWEEP_FRES && j == 0) {
#pragma unroll
      for (int mb = 0; mb < NB; ++mb) coarse[mb] = v[mb] + hc * s[mb];
    }
#pragma unroll
    for (int mb = 0; mb < NB; ++mb) v[mb] = v[mb] + hl * s[mb];
    if (on) {
      if (G) {
        V t[NB];
        Lt::load(t, G + (kc + j + 1) * slice + row);
        add_to<V, NB>(v, t);
      }
      if (MODE == SWEEP_CORRF) Lt::store(X + (kc + j + 1) * slice + row, v);
    }
    w_put<Q, WAVES>(W[(j + 1) & 1], wr);
    __syncthreads();
  }

  if constexpr (extra != 0) {
    // sigma' of the layer before the next C-point, from the last F-point
    V z[NB];
    Lt::template prod<C::LD>(z, v, W[nsteps & 1], lane);
    apply<V, NB, NV>(z, a.act, true);
    store_dsig<Lt>(a.dsig, (size_t)(kc + nsteps) * a.stride * slice + row, a.act, z, on);
  }
  if (MODE == SWEEP_FC) {
    if (on) Lt::store(static_cast<float*>(a.S) + (size_t)(k + 1) * slice + row, v);
  } else if (MODE == SWEEP_FRES) {
    double acc = 0.0;
    if (on) {
      V cn[NB];
      Lt::load(cn, Cs + (size_t)(k + 1) * a.cs_stride * slice + row);
      acc = sq_diff<V, NB, NV>(v, cn);
#pragma unroll
      for (int mb = 0; mb < NB; ++mb) coarse[mb] = v[mb] - coarse[mb];  // g_{l+1}^{k+1}
      Lt::store(static_cast<float*>(a.Gn) + (size_t)(k + 1) * slice + row, coarse);
      if (a.xn_every > 0 && (k + 1) % a.xn_every == 0)
        Lt::store(static_cast<float*>(a.Xn) + (size_t)(k + 1) * slice + row, cn);
      if (k == 0) {
        Lt::load(cn, Cs + row);
        Lt::store(static_cast<float*>(a.Xn) + row, cn);
      }
    }
    if (a.partial) {
      const double s = wg_sum<WAVES>(acc, red);
      if (threadIdx.x == 0) a.partial[(size_t)blockIdx.y * gridDim.x + blockIdx.x] = s;
    }
  } else if (MODE == SWEEP_CORRF) {
    if (on && k == Nc - 1) {
      correct<Lt>(v, Cs + (size_t)Nc * a.cs_stride * slice + row, Vn + (size_t)Nc * slice + row);
      Lt::store(X + (size_t)a.Nl * slice + row, v);
    }
  }
}

// ------------------------------------------------------------------ adjoint
// Interval k runs from its upper C-point (k+1)c down to kc; step j produces level
// point i = (k+1)c-1-j, linearised at the fine state of index i*stride.
template <int Q, int MODE, int WAVES, int EX, bool REC>
__global__ __launch_bounds__(64 * WAVES)
__attribute__((amdgpu_waves_per_eu(Q == 64 && REC ? (MODE == SWEEP_FRES ? 3 : 4) : 1, 8))) void k_adj(SweepArgs a) {
  using C = Cfg<Q, WAVES>;
  using Lt = Lay<Q, EX>;
  using V = typename Lt::V;
  constexpr int NB = Lt::NB, NV = Lt::NV;
  __shared__ float W[2][C::WSZ];
  __shared__ double red[WAVES];
  const int lane = threadIdx.x & 63;
  const int k = blockIdx.y;
  const int Nc = gridDim.y;
  const int e = (blockIdx.x * WAVES + (threadIdx.x >> 6)) * EX + (lane % EX);
  const bool on = e < a.B;
  const size_t slice = (size_t)a.B * Q;
  const size_t row = (size_t)(on ? e : 0) * Q + 4 * (lane / EX);
  const float* K = static_cast<const float*>(a.K);
  const float* bb = static_cast<const float*>(a.b);
  const float* Uf = static_cast<const float*>(a.Uf);
  float* X = static_cast<float*>(a.X);
  const float* G = static_cast<const float*>(a.G);
  const float* Cs = static_cast<const float*>(a.Cs);
  const float* Vn = static_cast<const float*>(a.V);
  const int c = a.c;
  const int nsteps = MODE == SWEEP_CORRF ? c - 1 : c;
  const float hl = (float)a.hl, hc = (float)a.hc;
  const long top = (long)(k + 1) * c;

  WRegs<Q, WAVES> wr;
  w_fetch<Q, WAVES>(wr, K, bb, (size_t)(top - 1) * a.stride);
  w_put<Q, WAVES>(W[0], wr);
  __syncthreads();

  V v[NB], cu[NB];
#pragma unroll
  for (int mb = 0; mb < NB; ++mb) v[mb] = 0.f;
  if (on) {
    if (MODE == SWEEP_FC) {
      if (Vn)
        correct<Lt>(v, Cs + (size_t)(k + 1) * a.cs_stride * slice + row, Vn + (size_t)(k + 1) * slice + row);
      else Lt::load(v, X + top * slice + row);
      if (MODE == SWEEP_FC && k == Nc - 1) Lt::store(static_cast<float*>(a.S) + (size_t)Nc * slice + row, v);
    } else if (MODE == SWEEP_FRES) {
      Lt::load(v, Cs + (size_t)(k + 1) * a.cs_stride * slice + row);
    } else {
      correct<Lt>(v, Cs + (size_t)(k + 1) * a.cs_stride * slice + row, Vn + (size_t)(k + 1) * slice + row);
      if (k + 1 < Nc) Lt::store(X + top * slice + row, v);
    }
  }
  if (MODE == SWEEP_FRES) {
#pragma unroll
    for (int mb = 0; mb < NB; ++mb) cu[mb] = v[mb];
  }
  constexpr bool rec = REC;  // sigma' from the record instead of K u + b
  // at width 64 the record row of the next step is requested one step ahead
  // (the extra registers do not lower the occupancy there)
  constexpr bool PFR = rec && Q == 64;
  V rn[NB];
  if (PFR) load_dsig<Lt>(rn, a.dsig, (size_t)(top - 1) * a.stride * slice + row, a.act);
  for (int j = 0; j < nsteps; ++j) {
    const long i = top - 1 - j;
    w_fetch<Q, WAVES>(wr, K, bb, (size_t)(j + 1 < nsteps ? i - 1 : i) * a.stride);
    V d[NB], w[NB];
    if constexpr (rec) {
      // every lane reads a valid row; columns of lanes past the batch are never stored
      if constexpr (PFR) {
#pragma unroll
        for (int mb = 0; mb < NB; ++mb) d[mb] = rn[mb];
        if (j + 1 < nsteps) load_dsig<Lt>(rn, a.dsig, (size_t)(i - 1) * a.stride * slice + row, a.act);
      } else {
        load_dsig<Lt>(d, a.dsig, (size_t)i * a.stride * slice + row, a.act);
      }
    } else {
      V u[NB];
#pragma unroll
      for (int mb = 0; mb < NB; ++mb) u[mb] = 0.f;
      if (on) Lt::load(u, Uf + (size_t)i * a.ustride * slice + row);
      Lt::template prod<C::LD>(d, u, W[j & 1], lane);
      apply<V, NB, NV>(d, a.act, true);
    }
    if (MODE == SWEEP_FRES && j == nsteps - 1) {
      // coarse adjoint step from the upper C-point, linearised at the same fine state
      V s2[NB];
#pragma unroll
      for (int mb = 0; mb < NB; ++mb) s2[mb] = d[mb] * cu[mb];
      Lt::template prod_t<C::LD>(w, s2, W[j & 1], lane);
#pragma unroll
      for (int mb = 0; mb < NB; ++mb) cu[mb] = cu[mb] + hc * w[mb];
    }
#pragma unroll
    for (int mb = 0; mb < NB; ++mb) d[mb] = d[mb] * v[mb];
    Lt::template prod_t<C::LD>(w, d, W[j & 1], lane);
#pragma unroll
    for (int mb = 0; mb < NB; ++mb) v[mb] = v[mb] + hl * w[mb];
    if (on) {
      if (G) {
        V t[NB];
        Lt::load(t, G + (size_t)i * slice + row);
        add_to<V, NB>(v, t);
      }
      if (MODE == SWEEP_CORRF) Lt::store(X + (size_t)i * slice + row, v);
    }
    w_put<Q, WAVES>(W[(j + 1) & 1], wr);
    __syncthreads();
  }

  if (MODE == SWEEP_FC) {
    if (on) Lt::store(static_cast<float*>(a.S) + (size_t)k * slice + row, v);
  } else if (MODE == SWEEP_FRES) {
    double acc = 0.0;
    if (on) {
      V ck[NB];
      Lt::load(ck, Cs + (size_t)k * a.cs_stride * slice + row);
      acc = sq_diff<V, NB, NV>(v, ck);
#pragma unroll
      for (int mb = 0; mb < NB; ++mb) cu[mb] = v[mb] - cu[mb];  // g_{l+1}^k
      Lt::store(static_cast<float*>(a.Gn) + (size_t)k * slice + row, cu);
      if (a.xn_every > 0 && k % a.xn_every == 0)
        Lt::store(static_cast<float*>(a.Xn) + (size_t)k * slice + row, ck);
      if (k == Nc - 1) {
        Lt::load(ck, Cs + (size_t)Nc * a.cs_stride * slice + row);
        Lt::store(static_cast<float*>(a.Xn) + (size_t)Nc * slice + row, ck);
      }
    }
    if (a.partial) {
      const double s = wg_sum<WAVES>(acc, red);
      if (threadIdx.x == 0) a.partial[(size_t)blockIdx.y * gridDim.x + blockIdx.x] = s;
    }
  } else if (MODE == SWEEP_CORRF) {
    if (on && k == 0) {
      correct<Lt>(v, Cs + row, Vn + row);
      Lt::store(X + row, v);
    }
  }
}

// ------------------------------------------------------------------ interval-resident sweeps
// With c = 4 the sweeps of the width-32 layers are latency-bound when every step
// waits on its own rows behind a barrier. These variants stage the weights of all
// the interval's layers in LDS at once and request every row the interval reads
// (right-hand-side rows, sigma' record or primal rows, the second C-point) before
// the first step, so a workgroup waits on memory about once, and the step loop
// has no barrier. Arithmetic and operand order are those of k_fwd / k_adj, step
// by step. Lanes past the batch read example 0's rows (valid memory) and store
// nothing; in the matrix-core products every example is its own column, so those
// lanes do not touch the others' results.
constexpr int IV_CF = 4;

// Weights and biases of NL consecutive layers in flight between global memory and LDS.
template <int Q, int NL, int WAVES>
struct WAll {
  static constexpr int NT = 64 * WAVES;
  static constexpr int KV = Q * Q / 4;  // float4 slots of one K_n
  static constexpr int BV = Q / 4;      // float4 slots of one b_n
  static constexpr int PK = (NL * KV + NT - 1) / NT;
  static constexpr int PB = (NL * BV + NT - 1) / NT;
  f32x4 k[PK];
  f32x4 b[PB];
};

// Slot j holds fine layer (n0 + dn j) * stride.
template <int Q, int NL, int WAVES>
__device__ __forceinline__ void wall_fetch(WAll<Q, NL, WAVES>& r, const float* __restrict__ K,
                                           const float* __restrict__ b, long n0, long dn, long stride) {
  using A = WAll<Q, NL, WAVES>;
#pragma unroll
  for (int p = 0; p < A::PK; ++p) {
    const int idx = threadIdx.x + p * A::NT;
    if (idx < NL * A::KV) {
      const int j = idx / A::KV, w = idx - j * A::KV;
      r.k[p] = reinterpret_cast<const f32x4*>(K + (size_t)((n0 + dn * j) * stride) * (Q * Q))[w];
    }
  }
#pragma unroll
  for (int p = 0; p < A::PB; ++p) {
    const int idx = threadIdx.x + p * A::NT;
    if (idx < NL * A::BV) {
      const int j = idx / A::BV, w = idx - j * A::BV;
      r.b[p] = reinterpret_cast<const f32x4*>(b + (size_t)((n0 + dn * j) * stride) * Q)[w];
    }
  }
}

template <int Q, int NL, int WAVES>
__device__ __forceinline__ void wall_put(float* sh, const WAll<Q, NL, WAVES>& r) {
  using A = WAll<Q, NL, WAVES>;
  using C = Cfg<Q, WAVES>;
#pragma unroll
  for (int p = 0; p < A::PK; ++p) {
    const int idx = threadIdx.x + p * A::NT;
    if (idx < NL * A::KV) {
      const int j = idx / A::KV, w = idx - j * A::KV;
      const int el = w * 4, row = el / Q, col = el - row * Q;
      *reinterpret_cast<f32x4*>(sh + j * C::WSZ + row * C::LD + col) = r.k[p];
    }
  }
#pragma unroll
  for (int p = 0; p < A::PB; ++p) {
    const int idx = threadIdx.x + p * A::NT;
    if (idx < NL * A::BV) {
      const int j = idx / A::BV, w = idx - j * A::BV;
      *reinterpret_cast<f32x4*>(sh + j * C::WSZ + Q * C::LD + w * 4) = r.b[p];
    }
  }
}

// A sigma' record row as loaded (16-example lanes): the example's word of ReLU's
// decision bits (MaskWord) or the fp32 values of the smooth activations.
template <typename Lt, bool BITS>
struct RecRow;
template <typename Lt>
struct RecRow<Lt, true> {
  static constexpr int Q = 16 * Lt::NB;
  typename MaskWord<Q>::T w;
  __device__ void load(const void* rec, size_t off) { w = MaskWord<Q>::load(static_cast<const uint8_t*>(rec), off); }
  __device__ void get(typename Lt::V (&d)[Lt::NB]) const { Lt::unpack_mask(d, w, 4 * ((threadIdx.x & 63) >> 4)); }
};
template <typename Lt>
struct RecRow<Lt, false> {
  typename Lt::V v[Lt::NB];
  __device__ void load(const void* rec, size_t off) { Lt::load(v, static_cast<const float*>(rec) + off); }
  __device__ void get(typename Lt::V (&d)[Lt::NB]) const {
#pragma unroll
    for (int mb = 0; mb < Lt::NB; ++mb) d[mb] = v[mb];
  }
};

// The interval kernels can walk batch tiles: workgroup (g, k) stages the weights
// of interval k once and runs tiles g, g + gridDim.x, ... of 64 examples (tile
// mode TM = 1), so the weights are read from L2 once per workgroup instead of once
// per tile; with TM = 2 the rows of its next tile are requested before the current
// tile's steps (the index is clamped, so every load is issued unconditionally and
// the waits stay exact) and a tile's loads overlap the previous tile's products.
// TM = 0 is one tile per workgroup.
__device__ __forceinline__ size_t iv_row(int t, int waves, int ex, int B, int Q, bool& on) {
  const int lane = threadIdx.x & 63;
  const int e = (t * waves + (threadIdx.x >> 6)) * ex + (lane % ex);
  on = e < B;
  return (size_t)(on ? e : 0) * Q + 4 * (lane / ex);
}

// Rows of one tile for a forward interval sweep: two state rows (FC: the C-point,
// or the staged C-point and the coarse value of a pending correction; FRES: the
// lower and the upper C-point; CORRF: the C-point and its coarse value) and the
// level's right-hand-side rows.
template <typename Lt, int NS, bool HASG>
struct FwdRows {
  typename Lt::V a[Lt::NB], c[Lt::NB];
  typename Lt::V g[HASG ? NS : 1][Lt::NB];
};

// REC: the final F-relaxation writes the sigma' record (CORRF only).
// HASG: the level has right-hand-side rows (every level but the finest).
template <int Q, int MODE, int WAVES, bool REC, bool HASG, int TM, bool CORR>
__global__ __launch_bounds__(64 * WAVES) void k_fwd_iv(SweepArgs a) {
  constexpr int EX = 16;
  using C = Cfg<Q, WAVES>;
  using Lt = Lay<Q, EX>;
  using V = typename Lt::V;
  constexpr int NB = Lt::NB, NV = Lt::NV;
  constexpr bool rec = REC && MODE == SWEEP_CORRF;
  constexpr int NS = MODE == SWEEP_CORRF ? IV_CF - 1 : IV_CF;
  constexpr int NL = NS + (rec ? 1 : 0);
  using Rows = FwdRows<Lt, NS, HASG>;
  __shared__ float W[NL * C::WSZ];
  __shared__ double red[WAVES];
  const int lane = threadIdx.x & 63;
  const int k = blockIdx.y;
  const int Nc = gridDim.y;
  const int ntiles = (a.B + EX * WAVES - 1) / (EX * WAVES);
  const size_t slice = (size_t)a.B * Q;
  float* X = static_cast<float*>(a.X);
  const float* G = static_cast<const float*>(a.G);
  const float* Cs = static_cast<const float*>(a.Cs);
  const float* Vn = static_cast<const float*>(a.V);
  const float hl = (float)a.hl, hc = (float)a.hc;
  const long kc = (long)k * IV_CF;

  if (MODE == SWEEP_CORRF && !HASG && a.cpt) {
    // C-point storage: the corrected C-points are the whole result (the F-points
    // are not stored; the adjoint and the gradient recompute them from these)
    for (int t = blockIdx.x; t < ntiles; t += gridDim.x) {
      bool on;
      const size_t row = iv_row(t, WAVES, EX, a.B, Q, on);
      if (on) {
        V v[NB];
        if (k > 0) {
          correct<Lt>(v, Cs + (size_t)k * a.cs_stride * slice + row, Vn + (size_t)k * slice + row);
          Lt::store(X + (size_t)k * slice + row, v);
        }
        if (k == Nc - 1) {
          correct<Lt>(v, Cs + (size_t)Nc * a.cs_stride * slice + row, Vn + (size_t)Nc * slice + row);
          Lt::store(X + (size_t)Nc * slice + row, v);
        }
      }
    }
    return;
  }

  // FC with CORR (a.V set) reads its C-points as C + (V - C): a pending coarse-grid
  // correction of the previous cycle applied on the fly, or (the second FC sweep of
  // FCFCF) staged C-points read as C + (C - C); with C-point storage C-point k is
  // row k of the level-0 trajectory
  constexpr bool pair = MODE != SWEEP_FC || CORR;
  auto load_rows = [&](Rows& r, size_t row) {
    if (MODE == SWEEP_FC && !pair) {
      Lt::load(r.a, X + (a.cpt ? (long)k : kc) * slice + row);
#pragma unroll
      for (int mb = 0; mb < NB; ++mb) r.c[mb] = 0.f;  // unused; initialised so the rows stay in registers
    } else {
      Lt::load(r.a, Cs + (size_t)k * a.cs_stride * slice + row);
      if (MODE == SWEEP_FRES) Lt::load(r.c, Cs + (size_t)(k + 1) * a.cs_stride * slice + row);
      else Lt::load(r.c, Vn + (size_t)k * slice + row);
    }
    if constexpr (HASG) {
#pragma unroll
      for (int j = 0; j < NS; ++j) Lt::load(r.g[j], G + (kc + j + 1) * slice + row);
    }
  };

  WAll<Q, NL, WAVES> wr;
  wall_fetch<Q, NL, WAVES>(wr, static_cast<const float*>(a.K), static_cast<const float*>(a.b), kc, 1, a.stride);
  Rows cur;
  {
    bool on0;
    load_rows(cur, iv_row(blockIdx.x, WAVES, EX, a.B, Q, on0));
  }
  wall_put<Q, NL, WAVES>(W, wr);
  __syncthreads();

  double acc = 0.0;
  // the work of one tile t, reading the staged weights through Wt
  auto tile = [&](Rows& cur, int t, const float* Wt) {
    bool on;
    const size_t row = iv_row(t, WAVES, EX, a.B, Q, on);
    V v[NB];
    if (MODE == SWEEP_FC && !pair) {
#pragma unroll
      for (int mb = 0; mb < NB; ++mb) v[mb] = cur.a[mb];
    } else if (MODE == SWEEP_FRES) {
#pragma unroll
      for (int mb = 0; mb < NB; ++mb) v[mb] = cur.a[mb];
    } else {
#pragma unroll
      for (int mb = 0; mb < NB; ++mb) v[mb] = cur.a[mb] + (cur.c[mb] - cur.a[mb]);  // C + (V - C)
    }
    if (on) {
      if (MODE == SWEEP_FC && k == 0) Lt::store(static_cast<float*>(a.S) + row, v);
      if (MODE == SWEEP_CORRF && k > 0) Lt::store(X + kc * slice + row, v);
    }

    V coarse[NB];
#pragma unroll
    for (int j = 0; j < NS; ++j) {
      V s[NB];
      Lt::template prod<C::LD>(s, v, Wt + j * C::WSZ, lane);
      if constexpr (rec) {
        V dz[NB];
#pragma unroll
        for (int mb = 0; mb < NB; ++mb) dz[mb] = s[mb];
        apply<V, NB, NV>(dz, a.act, true);
        store_dsig<Lt>(a.dsig, (size_t)(kc + j) * a.stride * slice + row, a.act, dz, on);
      }
      apply<V, NB, NV>(s, a.act, false);
      if (MODE == SWEEP_FRES && j == 0) {
#pragma unroll
        for (int mb = 0; mb < NB; ++mb) coarse[mb] = v[mb] + hc * s[mb];
      }
#pragma unroll
      for (int mb = 0; mb < NB; ++mb) v[mb] = v[mb] + hl * s[mb];
      if constexpr (HASG) add_to<V, NB>(v, cur.g[j]);
      if (MODE == SWEEP_CORRF && on) Lt::store(X + (kc + j + 1) * slice + row, v);
    }

    if constexpr (rec) {
      // sigma' of the layer before the next C-point, from the last F-point
      V z[NB];
      Lt::template prod<C::LD>(z, v, Wt + NS * C::WSZ, lane);
      apply<V, NB, NV>(z, a.act, true);
      store_dsig<Lt>(a.dsig, (size_t)(kc + NS) * a.stride * slice + row, a.act, z, on);
    }
    if (MODE == SWEEP_FC) {
      if (on) Lt::store(static_cast<float*>(a.S) + (size_t)(k + 1) * slice + row, v);
    } else if (MODE == SWEEP_FRES) {
      if (on) {
        acc += sq_diff<V, NB, NV>(v, cur.c);
#pragma unroll
        for (int mb = 0; mb < NB; ++mb) coarse[mb] = v[mb] - coarse[mb];  // g_{l+1}^{k+1}
        Lt::store(static_cast<float*>(a.Gn) + (size_t)(k + 1) * slice + row, coarse);
        if (a.xn_every > 0 && (k + 1) % a.xn_every == 0)
          Lt::store(static_cast<float*>(a.Xn) + (size_t)(k + 1) * slice + row, cur.c);
        if (k == 0) {
          V c0[NB];
          Lt::load(c0, Cs + row);
          Lt::store(static_cast<float*>(a.Xn) + row, c0);
        }
      }
    } else if (MODE == SWEEP_CORRF) {
      if (on && k == Nc - 1) {
        correct<Lt>(v, Cs + (size_t)Nc * a.cs_stride * slice + row, Vn + (size_t)Nc * slice + row);
        Lt::store(X + (size_t)a.Nl * slice + row, v);
      }
    }
  };
  if constexpr (TM == 0) {
    tile(cur, blockIdx.x, W);
  } else {
    for (int t = blockIdx.x; t < ntiles; t += gridDim.x) {
      // the products read the staged weights from LDS in every tile: an offset
      // the compiler cannot see through keeps it from hoisting those reads out of
      // the loop into registers
      int woff = 0;
      asm volatile("" : "+v"(woff));
      Rows nxt;
      if constexpr (TM == 2) {
        bool on1;
        load_rows(nxt, iv_row(min(t + (int)gridDim.x, ntiles - 1), WAVES, EX, a.B, Q, on1));
      } else if (t != (int)blockIdx.x) {
        bool on1;
        load_rows(cur, iv_row(t, WAVES, EX, a.B, Q, on1));
      }
      tile(cur, t, W + woff);
      if constexpr (TM == 2) cur = nxt;
    }
  }
  if (MODE == SWEEP_FRES && a.partial) {
    const double s = wg_sum<WAVES>(acc, red);
    if (threadIdx.x == 0) a.partial[(size_t)blockIdx.y * gridDim.x + blockIdx.x] = s;
  }
}

// Rows of one tile for an adjoint interval sweep: the two state rows (the upper
// C-point, or the staged C-point and coarse value of a correction; FRES: the upper
// and the lower C-point), what each step is linearised at (record rows, primal
// rows, or the lower primal C-point), and the right-hand-side rows.
template <typename Lt, int NS, bool REC, bool RBITS, bool CPT, bool HASG>
struct AdjRows {
  typename Lt::V a[Lt::NB], c[Lt::NB];
  RecRow<Lt, RBITS> rr[REC ? NS : 1];
  typename Lt::V u[(REC || CPT) ? 1 : NS][Lt::NB];
  typename Lt::V g[HASG ? NS : 1][Lt::NB];
};

// REC: sigma' comes from the record (ReLU: RBITS, one bit per value) instead of
// the layer product at the primal state.
// CPT (finest level, C-point storage): Uf holds the fine C-points only (row k is
// u^{kc}); the interval first recomputes its F-point states and sigma'(z_n) for
// n = kc .. kc + 3 by forward steps from its lower C-point, with the arithmetic of
// the forward F-relaxation (so the results equal those of full storage bit for bit).
// TM: tiles per workgroup (0: one; 1: several; 2: several, each one's rows
// requested during the previous one's steps). CORR: FC reads C + (V - C).
//
// Resident waves per SIMD the compiler must allow for. Width 32, finest level, bit
// record, one tile: eight. Width 64: two, which is what LDS allows (70 KB of weights
// per workgroup, two workgroups per CU); left to itself the compiler gives the
// fp32-record sweeps 260 registers, one wave per SIMD. The recomputing FRES sweeps
// that walk tiles are left free: held to 256 registers they spill.
template <int Q, int MODE, bool REC, bool RBITS, bool HASG, bool CPT, int TM>
constexpr int adj_iv_waves() {
  if (Q == 32) return !HASG && REC && RBITS && TM == 0 ? 8 : 1;
  if (Q == 64) return MODE == SWEEP_FRES && !REC && !CPT && TM != 0 ? 1 : 2;
  return 1;
}

template <int Q, int MODE, int WAVES, bool REC, bool RBITS, bool HASG, bool CPT, int TM, bool CORR>
__global__ __launch_bounds__(64 * WAVES)
__attribute__((amdgpu_waves_per_eu(adj_iv_waves<Q, MODE, REC, RBITS, HASG, CPT, TM>(), 8)))
void k_adj_iv(SweepArgs a) {
  static_assert(!(CPT && (REC || HASG)), "C-point storage is a finest-level mode without a record");
  constexpr int EX = 16;
  using C = Cfg<Q, WAVES>;
  using Lt = Lay<Q, EX>;
  using V = typename Lt::V;
  constexpr int NB = Lt::NB, NV = Lt::NV;
  constexpr int NS = MODE == SWEEP_CORRF ? IV_CF - 1 : IV_CF;
  constexpr int NW = CPT ? IV_CF : NS;  // layers staged: the recompute needs all of the interval's
  // at eight waves per SIMD (width 32, finest level, bit record, no prefetch) the
  // registers go to occupancy, and FRES reads its lower C-point after the steps
  constexpr bool LATE_CK = MODE == SWEEP_FRES && Q == 32 && !HASG && REC && RBITS && TM == 0;
  using Rows = AdjRows<Lt, NS, REC, RBITS, CPT, HASG>;
  __shared__ float W[NW * C::WSZ];
  __shared__ double red[WAVES];
  const int lane = threadIdx.x & 63;
  const int k = blockIdx.y;
  const int Nc = gridDim.y;
  const int ntiles = (a.B + EX * WAVES - 1) / (EX * WAVES);
  const size_t slice = (size_t)a.B * Q;
  const float* Uf = static_cast<const float*>(a.Uf);
  float* X = static_cast<float*>(a.X);
  const float* G = static_cast<const float*>(a.G);
  const float* Cs = static_cast<const float*>(a.Cs);
  const float* Vn = static_cast<const float*>(a.V);
  const float hl = (float)a.hl, hc = (float)a.hc;
  const long top = (long)(k + 1) * IV_CF;

  // step j is linearised at fine index (top - 1 - j) * stride, the primal state of
  // which is row (top - 1 - j) * ustride of Uf
  constexpr bool pair = MODE != SWEEP_FC || CORR;  // FC reading C + (V - C), as in k_fwd_iv
  auto load_rows = [&](Rows& r, size_t row) {
    if (MODE == SWEEP_FC && !pair) {
      Lt::load(r.a, X + top * slice + row);
#pragma unroll
      for (int mb = 0; mb < NB; ++mb) r.c[mb] = 0.f;  // unused; initialised so the rows stay in registers
    } else {
      Lt::load(r.a, Cs + (size_t)(k + 1) * a.cs_stride * slice + row);
      if (MODE == SWEEP_FRES) {
        if (!LATE_CK) Lt::load(r.c, Cs + (size_t)k * a.cs_stride * slice + row);
      } else {
        Lt::load(r.c, Vn + (size_t)(k + 1) * slice + row);
      }
    }
    if constexpr (REC) {
#pragma unroll
      for (int j = 0; j < NS; ++j) r.rr[j].load(a.dsig, (size_t)(top - 1 - j) * a.stride * slice + row);
    } else if constexpr (CPT) {
      Lt::load(r.u[0], Uf + (size_t)k * slice + row);  // u^{kc}
    } else {
#pragma unroll
      for (int j = 0; j < NS; ++j) Lt::load(r.u[j], Uf + (size_t)(top - 1 - j) * a.ustride * slice + row);
    }
    if constexpr (HASG) {
#pragma unroll
      for (int j = 0; j < NS; ++j) Lt::load(r.g[j], G + (size_t)(top - 1 - j) * slice + row);
    }
  };

  WAll<Q, NW, WAVES> wr;  // slot j holds layer top - 1 - j
  wall_fetch<Q, NW, WAVES>(wr, static_cast<const float*>(a.K), static_cast<const float*>(a.b), top - 1, -1,
                           a.stride);
  Rows cur;
  {
    bool on0;
    load_rows(cur, iv_row(blockIdx.x, WAVES, EX, a.B, Q, on0));
  }
  wall_put<Q, NW, WAVES>(W, wr);
  __syncthreads();

  double acc = 0.0;
  // the work of one tile t, reading the staged weights through Wt
  auto tile = [&](Rows& cur, int t, const float* Wt) {
    bool on;
    const size_t row = iv_row(t, WAVES, EX, a.B, Q, on);
    // C-point storage: dz[jf] = sigma'(z_{kc+jf}) along u^{kc+jf+1} = u^{kc+jf} + h sigma(z_{kc+jf})
    V dz[CPT ? IV_CF : 1][NB];
    if constexpr (CPT) {
#pragma unroll
      for (int jf = 0; jf < IV_CF; ++jf) {
        V sz[NB];
        Lt::template prod<C::LD, !HASG>(sz, cur.u[0], Wt + (IV_CF - 1 - jf) * C::WSZ, lane);
#pragma unroll
        for (int mb = 0; mb < NB; ++mb) dz[jf][mb] = sz[mb];
        apply<V, NB, NV>(dz[jf], a.act, true);
        if (jf + 1 < IV_CF) {
          apply<V, NB, NV>(sz, a.act, false);
#pragma unroll
          for (int mb = 0; mb < NB; ++mb) cur.u[0][mb] = cur.u[0][mb] + hl * sz[mb];
        }
      }
    }
    V v[NB], cu[NB];
    if (MODE == SWEEP_FC && !pair) {
#pragma unroll
      for (int mb = 0; mb < NB; ++mb) v[mb] = cur.a[mb];
    } else if (MODE == SWEEP_FRES) {
#pragma unroll
      for (int mb = 0; mb < NB; ++mb) v[mb] = cu[mb] = cur.a[mb];
    } else {
#pragma unroll
      for (int mb = 0; mb < NB; ++mb) v[mb] = cur.a[mb] + (cur.c[mb] - cur.a[mb]);  // C + (V - C)
    }
    if (on) {
      if (MODE == SWEEP_FC && k == Nc - 1) Lt::store(static_cast<float*>(a.S) + (size_t)Nc * slice + row, v);
      if (MODE == SWEEP_CORRF && k + 1 < Nc) Lt::store(X + top * slice + row, v);
    }

#pragma unroll
    for (int j = 0; j < NS; ++j) {
      const float* Wj = Wt + j * C::WSZ;
      V d[NB], w[NB];
      if constexpr (REC) {
        cur.rr[j].get(d);
      } else if constexpr (CPT) {
#pragma unroll
        for (int mb = 0; mb < NB; ++mb) d[mb] = dz[IV_CF - 1 - j][mb];
      } else {
        Lt::template prod<C::LD, !HASG>(d, cur.u[j], Wj, lane);
        apply<V, NB, NV>(d, a.act, true);
      }
      if (MODE == SWEEP_FRES && j == NS - 1) {
        // coarse adjoint step from the upper C-point, linearised at the same fine state
        V s2[NB];
#pragma unroll
        for (int mb = 0; mb < NB; ++mb) s2[mb] = d[mb] * cu[mb];
        Lt::template prod_t<C::LD, !HASG>(w, s2, Wj, lane);
#pragma unroll
        for (int mb = 0; mb < NB; ++mb) cu[mb] = cu[mb] + hc * w[mb];
      }
#pragma unroll
      for (int mb = 0; mb < NB; ++mb) d[mb] = d[mb] * v[mb];
      Lt::template prod_t<C::LD, !HASG>(w, d, Wj, lane);
#pragma unroll
      for (int mb = 0; mb < NB; ++mb) v[mb] = v[mb] + hl * w[mb];
      if constexpr (HASG) add_to<V, NB>(v, cur.g[j]);
      if (MODE == SWEEP_CORRF && on) Lt::store(X + (size_t)(top - 1 - j) * slice + row, v);
    }

    if (MODE == SWEEP_FC) {
      if (on) Lt::store(static_cast<float*>(a.S) + (size_t)k * slice + row, v);
    } else if (MODE == SWEEP_FRES) {
      if (on) {
        if (LATE_CK) Lt::load(cur.c, Cs + (size_t)k * a.cs_stride * slice + row);
        acc += sq_diff<V, NB, NV>(v, cur.c);
#pragma unroll
        for (int mb = 0; mb < NB; ++mb) cu[mb] = v[mb] - cu[mb];  // g_{l+1}^k
        Lt::store(static_cast<float*>(a.Gn) + (size_t)k * slice + row, cu);
        if (a.xn_every > 0 && k % a.xn_every == 0)
          Lt::store(static_cast<float*>(a.Xn) + (size_t)k * slice + row, cur.c);
        if (k == Nc - 1) {
          V cN[NB];
          Lt::load(cN, Cs + (size_t)Nc * a.cs_stride * slice + row);
          Lt::store(static_cast<float*>(a.Xn) + (size_t)Nc * slice + row, cN);
        }
      }
    } else if (MODE == SWEEP_CORRF) {
      if (on && k == 0) {
        correct<Lt>(v, Cs + row, Vn + row);
        Lt::store(X + row, v);
      }
    }
  };
  if constexpr (TM == 0) {
    tile(cur, blockIdx.x, W);
  } else {
    for (int t = blockIdx.x; t < ntiles; t += gridDim.x) {
      // the products read the staged weights from LDS in every tile: an offset
      // the compiler cannot see through keeps it from hoisting those reads out of
      // the loop into registers
      int woff = 0;
      asm volatile("" : "+v"(woff));
      Rows nxt;
      if constexpr (TM == 2) {
        bool on1;
        load_rows(nxt, iv_row(min(t + (int)gridDim.x, ntiles - 1), WAVES, EX, a.B, Q, on1));
      } else if (t != (int)blockIdx.x) {
        bool on1;
        load_rows(cur, iv_row(t, WAVES, EX, a.B, Q, on1));
      }
      tile(cur, t, W + woff);
      if constexpr (TM == 2) cur = nxt;
    }
  }
  if (MODE == SWEEP_FRES && a.partial) {
    const double s = wg_sum<WAVES>(acc, red);
    if (threadIdx.x == 0) a.partial[(size_t)blockIdx.y * gridDim.x + blockIdx.x] = s;
  }
}

// ------------------------------------------------------------------ gradient
// Workgroup (layer n, batch chunk). Each wave takes 32 examples at a time:
// s = sigma'(K_n u + b_n) * lam^{n+1} in accumulator layout (one matrix-core
// product), then s and u go through LDS as [example][feature] tiles so that
// dK[i][j] += sum_e s[e][i] u[e][j] runs as a second product with the examples
// as the contraction index (k-slice t pairs examples 2t and 2t+1). db sums the s
// tile's columns. The four waves' accumulators are combined in a fixed order and
// written as the chunk's partial; a second pass sums the chunks in order and
// scales by h (deterministic).
constexpr int GRAD_WAVES = 4;

// With the record (REC) the layer weights are not needed (no forward product), so
// they are not staged: at width 64 the workgroup then takes 67 KB of LDS, two fit
// on a CU, and the kernel is held to two waves per SIMD (left free it takes about
// 276 registers, one wave, and each chunk's loads are waited on in full).
// Lanes of one wave exchanging data through LDS: a wave's LDS instructions run in
// order, so a compiler fence and a wave barrier are enough between the writes and
// the reads.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

template <int Q, bool REC>
__global__ __launch_bounds__(64 * GRAD_WAVES) __attribute__((amdgpu_waves_per_eu(REC && Q == 64 ? 2 : 1, 8)))
void k_grad(GradArgs a) {
  using C = Cfg<Q, GRAD_WAVES>;
  constexpr int MB = C::MB;
  constexpr int TL = Q + 1;  // tile row (floats)
  __shared__ float W[REC ? 1 : C::WSZ];
  __shared__ float tile[GRAD_WAVES][2][32 * TL];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int h = lane >> 5, li = lane & 31;
  const long n = a.n0 + blockIdx.x;  // layer; its state is row blockIdx.x of U
  const int chunk = blockIdx.y;
  const int per = (((a.B + a.nchunks - 1) / a.nchunks) + 32 * GRAD_WAVES - 1) / (32 * GRAD_WAVES) *
                  (32 * GRAD_WAVES);
  const int e0 = chunk * per, e1 = min(a.B, e0 + per);
  const size_t slice = (size_t)a.B * Q;
  const float* U = static_cast<const float*>(a.U) + (size_t)blockIdx.x * slice;
  const float* L = static_cast<const float*>(a.Lam) + (size_t)(n + 1) * slice;
  if constexpr (!REC) {
    WRegs<Q, GRAD_WAVES> wr;
    w_fetch<Q, GRAD_WAVES>(wr, static_cast<const float*>(a.K), static_cast<const float*>(a.b), n);
    w_put<Q, GRAD_WAVES>(W, wr);
    __syncthreads();
  }
  f32x16 acc[MB][MB];
#pragma unroll
  for (int x = 0; x < MB; ++x)
#pragma unroll
    for (int y = 0; y < MB; ++y)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[x][y][r] = 0.f;
  float dbacc = 0.f;  // lane < Q: column sum of s over this wave's examples
  float* st = tile[wave][0];
  float* ut = tile[wave][1];
  using Lt = Lay<Q, 32>;
  // the rows of the wave's 32 examples from base on (zero past the chunk)
  auto ld_rows = [&](int base, f32x16 (&u)[MB], f32x16 (&s)[MB]) {
    const int e = base + wave * 32 + li;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) u[mb] = s[mb] = 0.f;
    if (e < e1) {
      Lt::load(u, U + (size_t)e * Q + 4 * h);
      Lt::load(s, L + (size_t)e * Q + 4 * h);
    }
  };
  // At width 32 the next examples' rows are requested during the contraction
  // (their registers cost no occupancy there); the tiles are the wave's own, so
  // its lanes meet at wave barriers only.
  constexpr bool PF = Q == 32;
  f32x16 un[PF ? MB : 1], sn[PF ? MB : 1];
  if constexpr (PF) ld_rows(e0, un, sn);
  for (int base = e0; base < e1; base += 32 * GRAD_WAVES) {
    const int e = base + wave * 32 + li;
    const size_t row = (size_t)(e < e1 ? e : 0) * Q + 4 * h;
    f32x16 u[MB], s[MB];
    if constexpr (PF) {
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        u[mb] = un[mb];
        s[mb] = sn[mb];
      }
    } else {
      ld_rows(base, u, s);
    }
    {
      f32x16 z[MB];
      if constexpr (REC) {
        load_dsig<Lt>(z, a.dsig, (size_t)n * slice + row, a.act);
      } else {
        Lt::template prod<C::LD>(z, u, W, lane);
        apply<f32x16, MB, 16>(z, a.act, true);
      }
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) s[mb] = z[mb] * s[mb];
    }
    // accumulator layout -> [example][feature] tiles
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int f = 32 * mb + 8 * (r >> 2) + 4 * h + (r & 3);
        st[li * TL + f] = s[mb][r];
        ut[li * TL + f] = u[mb][r];
      }
    if constexpr (PF) {
      wave_lds_sync();
      if (base + 32 * GRAD_WAVES < e1) ld_rows(base + 32 * GRAD_WAVES, un, sn);
    } else {
      __syncthreads();
    }
#pragma unroll
    for (int t = 0; t < 16; ++t) {
      const int er = (2 * t + h) * TL + li;
#pragma unroll
      for (int x = 0; x < MB; ++x) {
        const float av = st[er + 32 * x];
#pragma unroll
        for (int y = 0; y < MB; ++y)
          acc[x][y] = __builtin_amdgcn_mfma_f32_32x32x2f32(av, ut[er + 32 * y], acc[x][y], 0, 0, 0);
      }
    }
    if (lane < Q)
      for (int t = 0; t < 32; ++t) dbacc += st[t * TL + lane];
    if constexpr (PF) wave_lds_sync();
    else __syncthreads();
  }
  if constexpr (PF) __syncthreads();  // the combine below reuses every wave's tiles
  // combine the waves in order: wave w adds its accumulators into a Q x Q buffer
  float* red = &tile[0][0][0];  // Q*Q + Q floats fit in the tiles
  for (int w = 0; w < GRAD_WAVES; ++w) {
    if (wave == w) {
#pragma unroll
      for (int x = 0; x < MB; ++x)
#pragma unroll
        for (int y = 0; y < MB; ++y)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int i = 32 * x + 8 * (r >> 2) + 4 * h + (r & 3), j = 32 * y + li;
            red[i * Q + j] = (w == 0 ? 0.f : red[i * Q + j]) + acc[x][y][r];
          }
      if (lane < Q) red[Q * Q + lane] = (w == 0 ? 0.f : red[Q * Q + lane]) + dbacc;
    }
    __syncthreads();
  }
  float* out = static_cast<float*>(a.partial) + ((size_t)n * a.nchunks + chunk) * (Q * Q + Q);
  for (int o = threadIdx.x; o < Q * Q + Q; o += 64 * GRAD_WAVES) out[o] = red[o];
}

// Sum the chunk partials in chunk order in fp64 and scale by h.
__global__ __launch_bounds__(256) void k_grad_final(GradArgs a, int nw, int nbias) {
  const int nout = nw + nbias;
  const size_t o = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (o >= (size_t)a.N * nout) return;
  const size_t n = o / nout, r = o - n * nout;
  const float* p = static_cast<const float*>(a.partial) + n * a.nchunks * nout + r;
  double s = 0.0;
  for (int ch = 0; ch < a.nchunks; ++ch) s += (double)p[(size_t)ch * nout];
  const float v = (float)(s * a.h);
  if (r < (size_t)nw) static_cast<float*>(a.dK)[n * nw + r] = v;
  else static_cast<float*>(a.db)[n * nbias + (r - nw)] = v;
}

// First pass over `nl` layers starting at a.n0 (grid: layers x chunks).
template <int Q>
hipError_t grad_partials(const GradArgs& a, long nl, hipStream_t st) {
  // at width 32 the kernel is HBM-bound: an fp32 record row read per layer costs
  // more than the forward product it replaces, ReLU's bit record (1/32 of a row)
  // does not
  const bool rec = a.dsig && (Q >= 64 || a.act == ACT_RELU);
  if (rec) launch(k_grad<Q, true>, dim3((unsigned)nl, a.nchunks), 64 * GRAD_WAVES, 0, st, a);
  else launch(k_grad<Q, false>, dim3((unsigned)nl, a.nchunks), 64 * GRAD_WAVES, 0, st, a);
  return hipGetLastError();
}

template <int Q>
hipError_t grad_finish(const GradArgs& a, hipStream_t st) {
  const size_t tot = (size_t)a.N * (Q * Q + Q);
  launch(k_grad_final, (unsigned)((tot + 255) / 256), 256, 0, st, a, Q * Q, Q);
  return hipGetLastError();
}

template <int Q>
hipError_t grad(const GradArgs& a, hipStream_t st) {
  hipError_t err = grad_partials<Q>(a, a.N, st);
  if (err != hipSuccess) return err;
  return grad_finish<Q>(a, st);
}

// C-point storage: the F-relaxation of interval k0 + blockIdx.y from its lower
// C-point Uc[k0 + blockIdx.y], written to rows 4 blockIdx.y .. 4 blockIdx.y + 3 of Y
// (the C-point, then its three F-points), with the arithmetic of the forward
// sweeps' F-relaxation on the finest level (k_fwd_iv), so the states are those a
// full-storage solve stores.
template <int Q>
__global__ __launch_bounds__(64 * 4) void k_expand(const float* __restrict__ K, const float* __restrict__ bias,
                                                   const float* __restrict__ Uc, float* __restrict__ Y, int B,
                                                   long k0, float hl, int act) {
  constexpr int WAVES = 4, EX = 16, NL = IV_CF - 1;
  using C = Cfg<Q, WAVES>;
  using Lt = Lay<Q, EX>;
  using V = typename Lt::V;
  constexpr int NB = Lt::NB, NV = Lt::NV;
  __shared__ float W[NL * C::WSZ];
  const int lane = threadIdx.x & 63;
  const long k = k0 + blockIdx.y, kc = k * IV_CF;
  const int e = (blockIdx.x * WAVES + (threadIdx.x >> 6)) * EX + (lane % EX);
  const bool on = e < B;
  const size_t slice = (size_t)B * Q;
  const size_t row = (size_t)(on ? e : 0) * Q + 4 * (lane / EX);
  float* Yk = Y + (size_t)blockIdx.y * IV_CF * slice;
  WAll<Q, NL, WAVES> wr;
  wall_fetch<Q, NL, WAVES>(wr, K, bias, kc, 1, 1);
  V v[NB];
  Lt::load(v, Uc + (size_t)k * slice + row);
  wall_put<Q, NL, WAVES>(W, wr);
  __syncthreads();
  if (on) Lt::store(Yk + row, v);
#pragma unroll
  for (int j = 0; j < NL; ++j) {
    V s[NB];
    Lt::template prod<C::LD>(s, v, W + j * C::WSZ, lane);
    apply<V, NB, NV>(s, act, false);
#pragma unroll
    for (int mb = 0; mb < NB; ++mb) v[mb] = v[mb] + hl * s[mb];
    if (on) Lt::store(Yk + (size_t)(j + 1) * slice + row, v);
  }
}

// ------------------------------------------------------------------ serial solves
// The coarsest level (and the layer-serial baseline) runs one wave per 16
// examples through all N_l steps in order: few waves, so each step's loads sit
// on the critical path unless they were requested earlier. These kernels keep
// SER_D steps of loads in flight in register rings: the layer after next
// (weights and bias) and the right-hand-side, sigma' record or primal rows of
// the step SER_D ahead. A step writes only the next layer into LDS (double
// buffer, one wave: program order suffices, the barriers are nominal). The
// arithmetic of a step is that of the interval kernels. At width 64 a layer's
// weights take 64 registers per lane, so two layers are in flight there.
constexpr int SER_D = 4;

// Forward: U[j+1] = U[j] + h_l sigma(K_j U[j] + b_j) (+ G[j+1]), j = 0 .. N_l - 1;
// with REC the level-0 solve records sigma'(z) of every layer.
template <int Q, bool REC>
__global__ __launch_bounds__(64) void k_ser_fwd(SweepArgs a) {
  using C = Cfg<Q, 1>;
  using Lt = Lay<Q, 16>;
  using V = typename Lt::V;
  constexpr int NB = Lt::NB, NV = Lt::NV, D = Q <= 32 ? SER_D : 2;
  __shared__ float W[2][C::WSZ];
  const int lane = threadIdx.x & 63;
  const int e = blockIdx.x * 16 + (lane & 15);
  const bool on = e < a.B;
  const size_t slice = (size_t)a.B * Q;
  const size_t row = (size_t)(on ? e : 0) * Q + 4 * (lane >> 4);
  const float* K = static_cast<const float*>(a.K);
  const float* bb = static_cast<const float*>(a.b);
  float* X = static_cast<float*>(a.X);
  const float* G = static_cast<const float*>(a.G);
  const int Nl = a.Nl;
  const float hl = (float)a.hl;

  // rings: slot u holds layer j+1's weights and G row j+1 for the step j = u (mod D)
  WRegs<Q, 1> wr[D];
  V gr[D][NB];
  {
    WRegs<Q, 1> w0;
    w_fetch<Q, 1>(w0, K, bb, 0);
    // every prefetch is issued unconditionally (indices clamped to valid rows), so
    // the number of loads in flight is fixed and the waits stay exact
#pragma unroll
    for (int u = 0; u < D; ++u) w_fetch<Q, 1>(wr[u], K, bb, (size_t)min(u + 1, Nl - 1) * a.stride);
    if (G) {
#pragma unroll
      for (int u = 0; u < D; ++u) Lt::load(gr[u], G + (size_t)min(u + 1, Nl) * slice + row);  // valid rows
    }
    w_put<Q, 1>(W[0], w0);
  }
  V v[NB];
#pragma unroll
  for (int mb = 0; mb < NB; ++mb) v[mb] = 0.f;
  if (on) Lt::load(v, X + row);
  __syncthreads();
  for (int j0 = 0; j0 < Nl; j0 += D) {
#pragma unroll
    for (int u = 0; u < D; ++u) {
      const int j = j0 + u;
      if (j >= Nl) break;
      V s[NB];
      Lt::template prod<C::LD>(s, v, W[j & 1], lane);
      if constexpr (REC) {
        V dz[NB];
#pragma unroll
        for (int mb = 0; mb < NB; ++mb) dz[mb] = s[mb];
        apply<V, NB, NV>(dz, a.act, true);
        store_dsig<Lt>(a.dsig, (size_t)j * a.stride * slice + row, a.act, dz, on);
      }
      apply<V, NB, NV>(s, a.act, false);
#pragma unroll
      for (int mb = 0; mb < NB; ++mb) v[mb] = v[mb] + hl * s[mb];
      if (G) {
        add_to<V, NB>(v, gr[u]);
        Lt::load(gr[u], G + (size_t)min(j + 1 + D, Nl) * slice + row);
      }
      if (on) Lt::store(X + (size_t)(j + 1) * slice + row, v);
      // after the last step this writes a layer nobody reads
      w_put<Q, 1>(W[(j + 1) & 1], wr[u]);
      w_fetch<Q, 1>(wr[u], K, bb, (size_t)min(j + 1 + D, Nl - 1) * a.stride);
      __syncthreads();
    }
  }
}

// Adjoint: Lam[i] = Lam[i+1] + h_l K_i^T (sigma'(K_i U_f[i] + b_i) * Lam[i+1]) (+ G[i]),
// i = N_l - 1 .. 0, the primal state (row i * ustride of Uf, or the record at fine
// index i * stride, RK = 1 bytes, 2 fp32).
template <int Q, int RK>
__global__ __launch_bounds__(64) void k_ser_adj(SweepArgs a) {
  using C = Cfg<Q, 1>;
  using Lt = Lay<Q, 16>;
  using V = typename Lt::V;
  constexpr int NB = Lt::NB, NV = Lt::NV, D = Q <= 32 ? SER_D : 2;
  constexpr bool REC = RK != 0;
  __shared__ float W[2][C::WSZ];
  const int lane = threadIdx.x & 63;
  const int e = blockIdx.x * 16 + (lane & 15);
  const bool on = e < a.B;
  const size_t slice = (size_t)a.B * Q;
  const size_t row = (size_t)(on ? e : 0) * Q + 4 * (lane >> 4);
  const float* K = static_cast<const float*>(a.K);
  const float* bb = static_cast<const float*>(a.b);
  const float* Uf = static_cast<const float*>(a.Uf);
  float* X = static_cast<float*>(a.X);
  const float* G = static_cast<const float*>(a.G);
  const int Nl = a.Nl;
  const float hl = (float)a.hl;

  // rings, slot u for the step j = u (mod D), i = Nl - 1 - j: the weights of the
  // next step's layer i - 1, and the step's own record (or primal) and G rows
  WRegs<Q, 1> wr[D];
  RecRow<Lt, RK == 1> rr[REC ? D : 1];
  V ur[REC ? 1 : D][NB], gr[D][NB];
  {
    WRegs<Q, 1> w0;
    w_fetch<Q, 1>(w0, K, bb, (size_t)(Nl - 1) * a.stride);
    // every prefetch is issued unconditionally (indices clamped to valid rows), so
    // the number of loads in flight is fixed and the waits stay exact
#pragma unroll
    for (int u = 0; u < D; ++u) {
      const int i = max(Nl - 1 - u, 0);  // every lane reads a valid row
      w_fetch<Q, 1>(wr[u], K, bb, (size_t)max(i - 1, 0) * a.stride);
      if constexpr (REC) rr[u].load(a.dsig, (size_t)i * a.stride * slice + row);
      else Lt::load(ur[u], Uf + (size_t)i * a.ustride * slice + row);
      if (G) Lt::load(gr[u], G + (size_t)i * slice + row);
    }
    w_put<Q, 1>(W[0], w0);
  }
  V v[NB];
#pragma unroll
  for (int mb = 0; mb < NB; ++mb) v[mb] = 0.f;
  if (on) Lt::load(v, X + (size_t)Nl * slice + row);
  __syncthreads();
  for (int j0 = 0; j0 < Nl; j0 += D) {
#pragma unroll
    for (int u = 0; u < D; ++u) {
      const int j = j0 + u;
      if (j >= Nl) break;
      const int i = Nl - 1 - j;
      const float* Wj = W[j & 1];
      V d[NB], w[NB];
      const int ip = max(i - D, 0);
      if constexpr (REC) {
        rr[u].get(d);
        rr[u].load(a.dsig, (size_t)ip * a.stride * slice + row);
      } else {
        Lt::template prod<C::LD>(d, ur[u], Wj, lane);
        apply<V, NB, NV>(d, a.act, true);
        Lt::load(ur[u], Uf + (size_t)ip * a.ustride * slice + row);
      }
#pragma unroll
      for (int mb = 0; mb < NB; ++mb) d[mb] = d[mb] * v[mb];
      Lt::template prod_t<C::LD>(w, d, Wj, lane);
#pragma unroll
      for (int mb = 0; mb < NB; ++mb) v[mb] = v[mb] + hl * w[mb];
      if (G) {
        add_to<V, NB>(v, gr[u]);
        Lt::load(gr[u], G + (size_t)ip * slice + row);
      }
      if (on) Lt::store(X + (size_t)i * slice + row, v);
      // after the last step this writes a layer nobody reads
      w_put<Q, 1>(W[(j + 1) & 1], wr[u]);
      w_fetch<Q, 1>(wr[u], K, bb, (size_t)max(i - 1 - D, 0) * a.stride);
      __syncthreads();
    }
  }
}

constexpr int SWEEP_WAVES = 4;   // waves per interval workgroup (2 and 8 measured slower or equal)

// The sweeps run on the 16-example shape: measured faster than the 32-example
// one on every workload (q = 32 and 64, level 0 included), with fewer registers
// per wave and twice the waves.
constexpr int SWEEP_EX = 16;

// Interval-resident sweeps (c = 4): the level's right-hand side, the record kind
// and whether a workgroup prefetches its next tile select the instantiation.
template <int Q, bool HASG, int TM>
void sweep_iv(int dir, const SweepArgs& a, dim3 grid, hipStream_t st) {
  constexpr int W4 = SWEEP_WAVES;
  const bool rec = a.dsig != nullptr, bytes = a.act == ACT_RELU, corr = a.V != nullptr;
  if (dir == DIR_FWD) {
    if (a.mode == SWEEP_FC && corr) launch(k_fwd_iv<Q, SWEEP_FC, W4, false, HASG, TM, true>, grid, 64 * W4, 0, st, a);
    else if (a.mode == SWEEP_FC) launch(k_fwd_iv<Q, SWEEP_FC, W4, false, HASG, TM, false>, grid, 64 * W4, 0, st, a);
    else if (a.mode == SWEEP_FRES) launch(k_fwd_iv<Q, SWEEP_FRES, W4, false, HASG, TM, false>, grid, 64 * W4, 0, st, a);
    else if (rec) launch(k_fwd_iv<Q, SWEEP_CORRF, W4, true, HASG, TM, false>, grid, 64 * W4, 0, st, a);
    else launch(k_fwd_iv<Q, SWEEP_CORRF, W4, false, HASG, TM, false>, grid, 64 * W4, 0, st, a);
    return;
  }
#define LP_ADJ_IV(MODE, CORR)                                                                                         \
  do {                                                                                                                \
    if (!HASG && a.cpt) launch(k_adj_iv<Q, MODE, W4, false, false, false, true, TM, CORR>, grid, 64 * W4, 0, st, a);  \
    else if (!rec) launch(k_adj_iv<Q, MODE, W4, false, false, HASG, false, TM, CORR>, grid, 64 * W4, 0, st, a);       \
    else if (bytes) launch(k_adj_iv<Q, MODE, W4, true, true, HASG, false, TM, CORR>, grid, 64 * W4, 0, st, a);        \
    else launch(k_adj_iv<Q, MODE, W4, true, false, HASG, false, TM, CORR>, grid, 64 * W4, 0, st, a);                  \
  } while (0)
  if (a.mode == SWEEP_FC && corr) LP_ADJ_IV(SWEEP_FC, true);
  else if (a.mode == SWEEP_FC) LP_ADJ_IV(SWEEP_FC, false);
  else if (a.mode == SWEEP_FRES) LP_ADJ_IV(SWEEP_FRES, false);
  else LP_ADJ_IV(SWEEP_CORRF, false);
#undef LP_ADJ_IV
}

// LP_DENSE_SWEEP=staged keeps the double-buffered per-step kernels for c = 4 as
// well (for comparing the two designs).
bool iv_enabled() {
  static const bool on = [] {
    const char* e = getenv("LP_DENSE_SWEEP");
    return !(e && strcmp(e, "staged") == 0);
  }();
  return on;
}

// Which width-64 adjoint FRES sweeps run on the interval-resident kernel instead of
// the per-step one: LP_IV_FRES64 = 0 none, 1 the finest level's (the default:
// 51.1 against 55.7 ms per step on the deep workload; on coarse levels its record
// and right-hand-side rows leave one wave per SIMD), 2 every level's.
int iv_fres64() {
  static const int v = [] {
    const char* e = getenv("LP_IV_FRES64");
    return e ? atoi(e) : 1;
  }();
  return v;
}

// LP_IV_CORRF_WALK=1 lets the correction sweeps walk several tiles per workgroup
// as the other sweeps do (for comparison; they write c rows per tile).
bool iv_corrf_walk() {
  static const bool on = [] {
    const char* e = getenv("LP_IV_CORRF_WALK");
    return e && strcmp(e, "1") == 0;
  }();
  return on;
}

// Workgroups per interval of an interval-resident sweep: enough for about
// iv_target() workgroups in all (a few per resident slot), each walking
// ntiles / groups batch tiles; LP_IV_WG overrides the target.
int iv_target(int q) {
  static const int env = [] {
    const char* e = getenv("LP_IV_WG");
    return e ? atoi(e) : 0;
  }();
  if (env > 0) return env;
  return q == 64 ? 2048 : 1 << 30;
}

int iv_groups(int q, int ntiles, long Nc) {
  const long g = (iv_target(q) + Nc - 1) / Nc;
  return (int)std::max<long>(1, std::min<long>(ntiles, g));
}

template <int Q>
hipError_t sweep(int dir, const SweepArgs& a, hipStream_t st, int* partials) {
  constexpr int W4 = SWEEP_WAVES, EX = SWEEP_EX;
  const long Nc = a.Nl / a.c;
  if (Nc > 65535) return hipErrorNotSupported;  // intervals index the grid's y dimension
  const int ntiles = (a.B + EX * W4 - 1) / (EX * W4);
  const dim3 grid(ntiles, (unsigned)Nc);
  // Interval-resident kernels: every sweep at width 32; at width 64 (four layers,
  // 70 KB of LDS per workgroup) every sweep but the coarse levels' adjoint FRES
  // (iv_fres64). C-point storage (a.cpt, finest level) has interval-resident
  // kernels only.
  if constexpr (Q == 32 || Q == 64) {
    if (a.cpt && a.c != IV_CF) return hipErrorNotSupported;
    if (a.c == IV_CF &&
        (a.cpt || (iv_enabled() && (iv_fres64() > (a.G ? 1 : 0) ||
                                     !(Q == 64 && dir == DIR_ADJ && a.mode == SWEEP_FRES))))) {
      const int tg = a.mode == SWEEP_CORRF && !iv_corrf_walk() ? ntiles : iv_groups(Q, ntiles, Nc);
      const dim3 gi(tg, (unsigned)Nc);
      if (partials) *partials = (int)(gi.x * gi.y);
      // the next tile's rows are prefetched on the finest level only: with the
      // right-hand-side rows of a coarse level they would cost half the occupancy
      if (tg == ntiles) {
        if (a.G) sweep_iv<Q, true, 0>(dir, a, gi, st);
        else sweep_iv<Q, false, 0>(dir, a, gi, st);
      } else {
        if (a.G) sweep_iv<Q, true, 1>(dir, a, gi, st);
        else sweep_iv<Q, false, 2>(dir, a, gi, st);
      }
      return hipGetLastError();
    }
  }
  if (partials) *partials = (int)(grid.x * grid.y);
  const bool rec = a.dsig != nullptr;
  if (dir == DIR_FWD) {
    // only the final F-relaxation writes the sigma' record
    if (a.mode == SWEEP_FC) launch(k_fwd<Q, SWEEP_FC, W4, EX, false>, grid, 64 * W4, 0, st, a);
    else if (a.mode == SWEEP_FRES) launch(k_fwd<Q, SWEEP_FRES, W4, EX, false>, grid, 64 * W4, 0, st, a);
    else if (rec) launch(k_fwd<Q, SWEEP_CORRF, W4, EX, true>, grid, 64 * W4, 0, st, a);
    else launch(k_fwd<Q, SWEEP_CORRF, W4, EX, false>, grid, 64 * W4, 0, st, a);
  } else if (rec) {
    if (a.mode == SWEEP_FC) launch(k_adj<Q, SWEEP_FC, W4, EX, true>, grid, 64 * W4, 0, st, a);
    else if (a.mode == SWEEP_FRES) launch(k_adj<Q, SWEEP_FRES, W4, EX, true>, grid, 64 * W4, 0, st, a);
    else launch(k_adj<Q, SWEEP_CORRF, W4, EX, true>, grid, 64 * W4, 0, st, a);
  } else {
    if (a.mode == SWEEP_FC) launch(k_adj<Q, SWEEP_FC, W4, EX, false>, grid, 64 * W4, 0, st, a);
    else if (a.mode == SWEEP_FRES) launch(k_adj<Q, SWEEP_FRES, W4, EX, false>, grid, 64 * W4, 0, st, a);
    else launch(k_adj<Q, SWEEP_CORRF, W4, EX, false>, grid, 64 * W4, 0, st, a);
  }
  return hipGetLastError();
}

template <int Q>
hipError_t serial(int dir, const SerialArgs& s, hipStream_t st) {
  SweepArgs a{};
  a.act = s.act;
  a.mode = MODE_SERIAL;
  a.K = s.K;
  a.b = s.b;
  a.Uf = s.Uf;
  a.B = s.B;
  a.Nl = s.Nl;
  a.c = 1;
  a.stride = s.stride;
  a.hl = s.hl;
  a.X = s.X;
  a.G = s.G;
  a.dsig = s.dsig;
  a.ustride = s.ustride;
  const dim3 grid((s.B + 15) / 16, 1);
  if (dir == DIR_FWD) {
    if (s.dsig) launch(k_ser_fwd<Q, true>, grid, 64, 0, st, a);
    else launch(k_ser_fwd<Q, false>, grid, 64, 0, st, a);
  } else {
    if (!s.dsig) launch(k_ser_adj<Q, 0>, grid, 64, 0, st, a);
    else if (s.act == ACT_RELU) launch(k_ser_adj<Q, 1>, grid, 64, 0, st, a);
    else launch(k_ser_adj<Q, 2>, grid, 64, 0, st, a);
  }
  return hipGetLastError();
}

}  // namespace mfma

bool mfma_width_supported(int q) { return q == 32 || q == 64; }

hipError_t mfma_sweep(int q, int dir, const SweepArgs& a, hipStream_t st, int* partials) {
  if (q == 32) return mfma::sweep<32>(dir, a, st, partials);
  if (q == 64) return mfma::sweep<64>(dir, a, st, partials);
  return hipErrorNotSupported;
}

hipError_t mfma_serial(int q, int dir, const SerialArgs& a, hipStream_t st) {
  if (q == 32) return mfma::serial<32>(dir, a, st);
  if (q == 64) return mfma::serial<64>(dir, a, st);
  return hipErrorNotSupported;
}

hipError_t mfma_grad(int q, const GradArgs& a, hipStream_t st) {
  if (q == 32) return mfma::grad<32>(a, st);
  if (q == 64) return mfma::grad<64>(a, st);
  return hipErrorNotSupported;
}

hipError_t mfma_expand(int q, int act, const void* K, const void* b, const void* Uc, void* Y, int B, long k0,
                       long nk, double h, hipStream_t st) {
  if (nk <= 0 || B <= 0) return hipSuccess;
  if (nk > 65535) return hipErrorNotSupported;
  const dim3 grid((unsigned)((B + 63) / 64), (unsigned)nk);
  const float* Kp = static_cast<const float*>(K);
  const float* bp = static_cast<const float*>(b);
  const float* up = static_cast<const float*>(Uc);
  float* yp = static_cast<float*>(Y);
  if (q == 32) launch(mfma::k_expand<32>, grid, 256, 0, st, Kp, bp, up, yp, B, k0, (float)h, act);
  else if (q == 64) launch(mfma::k_expand<64>, grid, 256, 0, st, Kp, bp, up, yp, B, k0, (float)h, act);
  else return hipErrorNotSupported;
  return hipGetLastError();
}

hipError_t mfma_grad_partials(int q, const GradArgs& a, long nl, hipStream_t st) {
  if (q == 32) return mfma::grad_partials<32>(a, nl, st);
  if (q == 64) return mfma::grad_partials<64>(a, nl, st);
  return hipErrorNotSupported;
}

hipError_t mfma_grad_finish(int q, const GradArgs& a, hipStream_t st) {
  if (q == 32) return mfma::grad_finish<32>(a, st);
  if (q == 64) return mfma::grad_finish<64>(a, st);
  return hipErrorNotSupported;
}

}  // namespace lp
