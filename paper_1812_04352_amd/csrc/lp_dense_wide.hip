// Dense fp32 residual layers of width 220 (the hyperspectral network of
// Section 5.1, whose width is the number of spectral bands) on the matrix cores.
//
// At this width a layer step is a real dense contraction (2 q^2 = 96.8 kflop per
// example against 2 q e = 1.8 kB of state traffic), so the kernels are bound by
// the matrix cores, not by HBM. One layer's weights (q^2 fp32 = 194 kB) no longer
// fit in LDS next to anything else, so every product streams K_n through LDS in
// panels of 32 contraction indices, double-buffered: the next panel is fetched
// into registers while the current one feeds the matrix cores, then written to
// the other buffer behind one barrier.
//
// Layout (v_mfma_f32_16x16x4_f32, 16 examples per wave, 4 waves per workgroup):
// the width is padded to QP = 224 = 14 blocks of 16 features; register r of
// block mb in lane l holds feature 16 mb + 4 (l/16) + r of example l%16. That
// accumulator layout is the B operand of the next product when the A operand
// supplies, for k-slice (ib, r), the contraction index 16 ib + 4 (l/16) + r, so
// chained steps keep the state in the lanes that own it. Padding features
// (220..223) are never loaded or stored; the padded rows and columns of the LDS
// panels are zero and the padded values of every new state are reset to zero
// after the activation (sigma(0) is not zero for the smoothed ReLU).
//
//   forward product  z = K_n v + b_n : panel p holds K_n[:, 32p .. 32p+31] as
//                    [output][32] rows (pitch 36: a 16-byte read per lane, the
//                    16 lanes of a group on disjoint banks);
//   adjoint product  w = K_n^T s     : panel p holds K_n[32p .. 32p+31, :] as
//                    [32][output] rows (pitch 228: four lane groups 16 banks apart).
//
// Sweep modes, the record of sigma' and the FAS bookkeeping follow Algorithm 1
// (Section 3.1) exactly as the other dense kernels do.
#include <stdlib.h>
#include <string.h>

#include "lp_device.h"
#include "lp_internal.h"

namespace lp {
namespace wide {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int MODE_SERIAL = 3;
constexpr int WAVES = 4;
constexpr int NT = 64 * WAVES;
constexpr int EX = 16;  // examples per wave

template <int Q>
struct Geo {
  static_assert(Q % 4 == 0, "rows are read as 16-byte vectors");
  static constexpr int QP = (Q + 31) / 32 * 32;  // padded width
  static constexpr int NB = QP / 16;             // 16-feature blocks (even: QP is a multiple of 32)
  static constexpr int NP = QP / 32;             // panels per layer
  static constexpr int PLF = 32 + 4;             // forward panel pitch (floats)
  static constexpr int PLA = QP + 4;             // adjoint panel pitch (floats)
  static constexpr int PSZ = QP * PLF > 32 * PLA ? QP * PLF : 32 * PLA;
  static constexpr int PV = QP * 32 / 4;         // 16-byte slots of a panel
  static constexpr int PPT = (PV + NT - 1) / NT;
  // block NB-1 is real for lane groups g < TG (the rest is padding)
  static constexpr int TG = (Q - 16 * (NB - 1)) / 4;
};

// ------------------------------------------------------------------ rows
// p points at the example's row + 4 g (g = lane / 16)
template <int Q>
__device__ __forceinline__ void load_row(f32x4 (&v)[Geo<Q>::NB], const float* __restrict__ p, int g) {
  constexpr int NB = Geo<Q>::NB;
#pragma unroll
  for (int mb = 0; mb < NB; ++mb)
    v[mb] = (mb < NB - 1 || g < Geo<Q>::TG) ? *reinterpret_cast<const f32x4*>(p + 16 * mb) : f32x4{};
}

template <int Q>
__device__ __forceinline__ void store_row(float* __restrict__ p, const f32x4 (&v)[Geo<Q>::NB], int g) {
  constexpr int NB = Geo<Q>::NB;
#pragma unroll
  for (int mb = 0; mb < NB; ++mb)
    if (mb < NB - 1 || g < Geo<Q>::TG) *reinterpret_cast<f32x4*>(p + 16 * mb) = v[mb];
}

// The sigma' record at element offset off: one byte (0/1) per value for ReLU,
// fp32 otherwise.
template <int Q>
__device__ __forceinline__ void load_dsig(f32x4 (&d)[Geo<Q>::NB], const void* rec, size_t off, int act, int g) {
  constexpr int NB = Geo<Q>::NB;
  if (act == ACT_RELU) {
    const uint8_t* p = static_cast<const uint8_t*>(rec) + off;
#pragma unroll
    for (int mb = 0; mb < NB; ++mb) {
      const uint32_t w = (mb < NB - 1 || g < Geo<Q>::TG) ? *reinterpret_cast<const uint32_t*>(p + 16 * mb) : 0u;
#pragma unroll
      for (int r = 0; r < 4; ++r) d[mb][r] = (w >> (8 * r)) & 0xffu ? 1.f : 0.f;
    }
  } else {
    load_row<Q>(d, static_cast<const float*>(rec) + off, g);
  }
}

template <int Q>
__device__ __forceinline__ void store_dsig(void* rec, size_t off, int act, const f32x4 (&d)[Geo<Q>::NB], int g) {
  constexpr int NB = Geo<Q>::NB;
  if (act == ACT_RELU) {
    uint8_t* p = static_cast<uint8_t*>(rec) + off;
#pragma unroll
    for (int mb = 0; mb < NB; ++mb) {
      uint32_t w = 0;
#pragma unroll
      for (int r = 0; r < 4; ++r) w |= (d[mb][r] != 0.f ? 1u : 0u) << (8 * r);
      if (mb < NB - 1 || g < Geo<Q>::TG) *reinterpret_cast<uint32_t*>(p + 16 * mb) = w;
    }
  } else {
    store_row<Q>(static_cast<float*>(rec) + off, d, g);
  }
}

// sigma (deriv = false) or sigma' (deriv = true) of every value; padding values
// are reset to zero
template <int Q>
__device__ __forceinline__ void apply(f32x4 (&z)[Geo<Q>::NB], int act, bool deriv, int g) {
  constexpr int NB = Geo<Q>::NB;
  switch (act) {
    case ACT_TANH:
#pragma unroll
      for (int mb = 0; mb < NB; ++mb)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          z[mb][r] = deriv ? dact_f<float, ACT_TANH>(z[mb][r]) : act_f<float, ACT_TANH>(z[mb][r]);
      break;
    case ACT_RELU:
#pragma unroll
      for (int mb = 0; mb < NB; ++mb)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          z[mb][r] = deriv ? (z[mb][r] > 0.f ? 1.f : 0.f) : (z[mb][r] > 0.f ? z[mb][r] : 0.f);
      break;
    case ACT_SMOOTHRELU:
#pragma unroll
      for (int mb = 0; mb < NB; ++mb)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          z[mb][r] = deriv ? dact_f<float, ACT_SMOOTHRELU>(z[mb][r]) : act_f<float, ACT_SMOOTHRELU>(z[mb][r]);
      break;
    default:
      if (deriv) {
#pragma unroll
        for (int mb = 0; mb < NB; ++mb) z[mb] = 1.f;
      }
      break;
  }
  if (g >= Geo<Q>::TG) z[NB - 1] = 0.f;
}

// v = c + (v' - c) (Algorithm 1, the coarse-grid correction of a C-point)
template <int Q>
__device__ __forceinline__ void correct(f32x4 (&v)[Geo<Q>::NB], const float* cs, const float* vs, int g) {
  constexpr int NB = Geo<Q>::NB;
  f32x4 cv[NB], vv[NB];
  load_row<Q>(cv, cs, g);
  load_row<Q>(vv, vs, g);
#pragma unroll
  for (int mb = 0; mb < NB; ++mb) v[mb] = cv[mb] + (vv[mb] - cv[mb]);
}

template <int Q>
__device__ __forceinline__ double sq_diff(const f32x4 (&a)[Geo<Q>::NB], const f32x4 (&b)[Geo<Q>::NB]) {
  double acc = 0.0;
#pragma unroll
  for (int mb = 0; mb < Geo<Q>::NB; ++mb)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float d = a[mb][r] - b[mb][r];
      acc += (double)d * (double)d;
    }
  return acc;
}

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

// ------------------------------------------------------------------ panels
// One panel in flight between global memory and LDS (PPT 16-byte slots per thread).
template <int Q>
struct Pan {
  f32x4 r[Geo<Q>::PPT];
};

// forward panel p of K_n: slot = (output row o, 4 columns c4) of K_n[:, 32p + 4 c4 ..]
template <int Q>
__device__ __forceinline__ void fetch_f(Pan<Q>& pr, const float* __restrict__ Kn, int p) {
  using G = Geo<Q>;
  const float* base = Kn + 32 * p;  // workgroup-uniform; 32-bit per-slot offsets
#pragma unroll
  for (int s = 0; s < G::PPT; ++s) {
    const int idx = threadIdx.x + s * NT;
    const int o = idx >> 3, c4 = idx & 7;
    const bool ok = idx < G::PV && o < Q && 32 * p + 4 * c4 < Q;
    pr.r[s] = ok ? *reinterpret_cast<const f32x4*>(base + (o * Q + 4 * c4)) : f32x4{};
  }
}

template <int Q>
__device__ __forceinline__ void put_f(float* buf, const Pan<Q>& pr) {
  using G = Geo<Q>;
#pragma unroll
  for (int s = 0; s < G::PPT; ++s) {
    const int idx = threadIdx.x + s * NT;
    if (idx < G::PV) *reinterpret_cast<f32x4*>(buf + (idx >> 3) * G::PLF + 4 * (idx & 7)) = pr.r[s];
  }
}

// adjoint panel p of K_n: slot = (row ii, 4 columns o4) of K_n[32p + ii][4 o4 ..];
// slots S0 .. S1-1 of this thread (the adjoint moves a panel in two parts)
template <int Q, int S0, int S1>
__device__ __forceinline__ void fetch_a(f32x4 (&r)[S1 - S0], const float* __restrict__ Kn, int p) {
  using G = Geo<Q>;
  constexpr int RW = G::QP / 4;  // slots per panel row
  // a workgroup-uniform panel base and 32-bit per-slot offsets (few registers)
  const float* base = Kn + (size_t)(32 * p) * Q;
#pragma unroll
  for (int s = S0; s < S1; ++s) {
    const int idx = threadIdx.x + s * NT;
    const int ii = idx / RW, o4 = idx - ii * RW;
    const bool ok = idx < G::PV && 32 * p + ii < Q && 4 * o4 < Q;
    r[s - S0] = ok ? *reinterpret_cast<const f32x4*>(base + (ii * Q + 4 * o4)) : f32x4{};
  }
}

template <int Q, int S0, int S1>
__device__ __forceinline__ void put_a(float* buf, const f32x4 (&r)[S1 - S0]) {
  using G = Geo<Q>;
  constexpr int RW = G::QP / 4;
#pragma unroll
  for (int s = S0; s < S1; ++s) {
    const int idx = threadIdx.x + s * NT;
    const int ii = idx / RW, o4 = idx - ii * RW;
    if (idx < G::PV) *reinterpret_cast<f32x4*>(buf + ii * G::PLA + 4 * o4) = r[s - S0];
  }
}

// Consecutive forward products share the two panel buffers as a chain: a
// product's last panel fetches the next product's first panel (the next layer is
// known), so a step does not start with a panel load the whole workgroup waits
// for. With an odd number of panels the buffer holding a product's first panel
// alternates; `ph` tracks it and `ready` says whether it is already loaded. (The
// transposed product does not chain: the extra state spilled in the adjoint
// kernels and measured slower.)
struct Chain {
  int ph = 0;
  bool ready = false;
};

// z = K_n v + b_n. Every thread of the workgroup calls it (it holds barriers).
// Knext: the next product's weights (same kind), whose first panel this product
// loads during its last one; nullptr ends the chain.
template <int Q>
__device__ __forceinline__ void prod(f32x4 (&z)[Geo<Q>::NB], const f32x4 (&v)[Geo<Q>::NB],
                                     const float* __restrict__ Kn, const float* __restrict__ bn, float* buf,
                                     int lane, Chain& ch, const float* __restrict__ Knext = nullptr) {
  using G = Geo<Q>;
  constexpr int NB = G::NB;
  const int g = lane >> 4, i = lane & 15;
  Pan<Q> pr;
  load_row<Q>(z, bn + 4 * g, g);
  if (!ch.ready) {
    fetch_f<Q>(pr, Kn, 0);
    put_f<Q>(buf + ch.ph * G::PSZ, pr);
    __syncthreads();
  }
#pragma unroll
  for (int p = 0; p < G::NP; ++p) {
    const bool more = p + 1 < G::NP;
    if (more) fetch_f<Q>(pr, Kn, p + 1);
    else if (Knext) fetch_f<Q>(pr, Knext, 0);
    const float* P = buf + ((ch.ph + p) & 1) * G::PSZ + i * G::PLF + 4 * g;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      // output blocks in two halves: half the A registers, still 7 independent chains
#pragma unroll
      for (int o0 = 0; o0 < NB; o0 += NB / 2) {
        f32x4 av[NB / 2];
#pragma unroll
        for (int ob = 0; ob < NB / 2; ++ob)
          av[ob] = *reinterpret_cast<const f32x4*>(P + 16 * (o0 + ob) * G::PLF + 16 * h);
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
          for (int ob = 0; ob < NB / 2; ++ob)
            z[o0 + ob] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[ob][r], v[2 * p + h][r], z[o0 + ob], 0, 0, 0);
      }
    }
    if (more || Knext) put_f<Q>(buf + ((ch.ph + p + 1) & 1) * G::PSZ, pr);
    __syncthreads();
  }
  ch.ph = (ch.ph + G::NP) & 1;
  ch.ready = Knext != nullptr;
}

// w = K_n^T s (same calling rules as prod). The next panel moves in two parts,
// each fetched before half of the current panel's products and written after it,
// so only half a panel is held in registers at a time.
template <int Q>
__device__ __forceinline__ void prod_t(f32x4 (&w)[Geo<Q>::NB], const f32x4 (&s)[Geo<Q>::NB],
                                       const float* __restrict__ Kn, float* buf, int lane) {
  using G = Geo<Q>;
  constexpr int NB = G::NB, H1 = (G::PPT + 1) / 2;
  const int g = lane >> 4, i = lane & 15;
  {
    f32x4 r0[H1], r1[G::PPT - H1];
    fetch_a<Q, 0, H1>(r0, Kn, 0);
    fetch_a<Q, H1, G::PPT>(r1, Kn, 0);
    put_a<Q, 0, H1>(buf, r0);
    put_a<Q, H1, G::PPT>(buf, r1);
  }
#pragma unroll
  for (int ob = 0; ob < NB; ++ob) w[ob] = 0.f;
  __syncthreads();
#pragma unroll
  for (int p = 0; p < G::NP; ++p) {
    const float* P = buf + (p & 1) * G::PSZ + 4 * g * G::PLA + i;
    float* nxt = buf + ((p + 1) & 1) * G::PSZ;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      f32x4 r0[H1], r1[G::PPT - H1];
      if (p + 1 < G::NP) {
        if (h == 0) fetch_a<Q, 0, H1>(r0, Kn, p + 1);
        else fetch_a<Q, H1, G::PPT>(r1, Kn, p + 1);
      }
      // output blocks in two halves, as in the forward product: 28 A values in
      // registers, 7 independent accumulation chains
#pragma unroll
      for (int o0 = 0; o0 < NB; o0 += NB / 2) {
        float av[4][NB / 2];
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
          for (int ob = 0; ob < NB / 2; ++ob) av[r][ob] = P[(16 * h + r) * G::PLA + 16 * (o0 + ob)];
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
          for (int ob = 0; ob < NB / 2; ++ob)
            w[o0 + ob] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[r][ob], s[2 * p + h][r], w[o0 + ob], 0, 0, 0);
      }
      if (p + 1 < G::NP) {
        if (h == 0) put_a<Q, 0, H1>(nxt, r0);
        else put_a<Q, H1, G::PPT>(nxt, r1);
      }
    }
    __syncthreads();
  }
}

// Work item of linear workgroup id L: the dispatcher deals workgroups to the 8
// XCDs in turn, so item (L % 8) * (n / 8) + L / 8 gives each XCD a contiguous run
// of intervals (all batch tiles of one interval on one XCD: its weights are read
// once into that XCD's L2). Falls back to L when n is not a multiple of 8.
__device__ __forceinline__ void xcd_item(int& tile, int& itv) {
  const unsigned gx = gridDim.x, n = gx * gridDim.y;
  const unsigned L = blockIdx.x + gx * blockIdx.y;
  const unsigned W = n % 8 == 0 ? (L % 8) * (n / 8) + L / 8 : L;
  itv = (int)(W / gx);
  tile = (int)(W - (unsigned)itv * gx);
}

// ------------------------------------------------------------------ forward
template <int Q, int MODE, bool REC>
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(2, 2))) void k_fwd(SweepArgs a) {
  using G = Geo<Q>;
  constexpr int NB = G::NB;
  __shared__ __attribute__((aligned(16))) float buf[2 * G::PSZ];
  __shared__ double red[WAVES];
  const int lane = threadIdx.x & 63, g = lane >> 4;
  int tile, k;
  xcd_item(tile, k);
  const int Nc = gridDim.y;
  const int e = (tile * WAVES + (threadIdx.x >> 6)) * EX + (lane & 15);
  const bool on = e < a.B;
  const size_t slice = (size_t)a.B * Q;
  const size_t row = (size_t)(on ? e : 0) * Q + 4 * g;
  const float* K = static_cast<const float*>(a.K);
  const float* bb = static_cast<const float*>(a.b);
  float* X = static_cast<float*>(a.X);
  const float* Gr = static_cast<const float*>(a.G);
  const float* Cs = static_cast<const float*>(a.Cs);
  const float* Vn = static_cast<const float*>(a.V);
  const int c = a.c;
  const int nsteps = MODE == MODE_SERIAL ? a.Nl : (MODE == SWEEP_CORRF ? c - 1 : c);
  const float hl = (float)a.hl, hc = (float)a.hc;
  const long kc = MODE == MODE_SERIAL ? 0 : (long)k * c;

  f32x4 v[NB];
#pragma unroll
  for (int mb = 0; mb < NB; ++mb) v[mb] = 0.f;
  if (on) {
    if (MODE == SWEEP_FC || MODE == MODE_SERIAL) {
      // a pending coarse-grid correction of the previous cycle is applied on the fly
      if (MODE == SWEEP_FC && Vn)
        correct<Q>(v, Cs + (size_t)k * a.cs_stride * slice + row, Vn + (size_t)k * slice + row, g);
      else load_row<Q>(v, X + kc * slice + row, g);
      if (MODE == SWEEP_FC && k == 0) store_row<Q>(static_cast<float*>(a.S) + row, v, g);
    } else if (MODE == SWEEP_FRES) {
      load_row<Q>(v, Cs + (size_t)k * a.cs_stride * slice + row, g);
    } else {
      correct<Q>(v, Cs + (size_t)k * a.cs_stride * slice + row, Vn + (size_t)k * slice + row, g);
      if (k > 0) store_row<Q>(X + kc * slice + row, v, g);
    }
  }
  // the final F-relaxation (and a level-0 serial solve) records sigma'(z) of every
  // layer; CORRF then also takes the product of the layer before the next C-point
  constexpr bool rec = REC && (MODE == SWEEP_CORRF || MODE == MODE_SERIAL);
  // FRES parks the coarse step's value v + h_c sigma(z) of the first layer in its
  // Gn row and finishes g_{l+1}^{k+1} = v - (that value) after the interval, so it
  // holds no extra row of registers across the steps
  float* gn = MODE == SWEEP_FRES ? static_cast<float*>(a.Gn) + (size_t)(k + 1) * slice + row : nullptr;
  Chain ch;
  for (int j = 0; j < nsteps; ++j) {
    const size_t n = (size_t)(kc + j) * a.stride;
    // the next product: the next step's layer, or CORRF's extra record product
    const float* knext = j + 1 < nsteps                      ? K + (size_t)(kc + j + 1) * a.stride * (Q * Q)
                         : (MODE == SWEEP_CORRF && rec) ? K + (size_t)(kc + nsteps) * a.stride * (Q * Q)
                                                        : nullptr;
    f32x4 z[NB];
    prod<Q>(z, v, K + n * (Q * Q), bb + n * Q, buf, lane, ch, knext);
    if constexpr (rec) {
      f32x4 dz[NB];
#pragma unroll
      for (int mb = 0; mb < NB; ++mb) dz[mb] = z[mb];
      apply<Q>(dz, a.act, true, g);
      if (on) store_dsig<Q>(a.dsig, n * slice + row, a.act, dz, g);
    }
    apply<Q>(z, a.act, false, g);
    if (MODE == SWEEP_FRES && j == 0 && on) {
      f32x4 coarse[NB];
#pragma unroll
      for (int mb = 0; mb < NB; ++mb) coarse[mb] = v[mb] + hc * z[mb];
      store_row<Q>(gn, coarse, g);
    }
#pragma unroll
    for (int mb = 0; mb < NB; ++mb) v[mb] = v[mb] + hl * z[mb];
    if (on) {
      if (Gr) {
        f32x4 t[NB];
        load_row<Q>(t, Gr + (kc + j + 1) * slice + row, g);
#pragma unroll
        for (int mb = 0; mb < NB; ++mb) v[mb] += t[mb];
      }
      if (MODE == SWEEP_CORRF || MODE == MODE_SERIAL) store_row<Q>(X + (kc + j + 1) * slice + row, v, g);
    }
  }
  if constexpr (MODE == SWEEP_CORRF && rec) {
    // sigma' of the layer before the next C-point, from the last F-point
    const size_t n = (size_t)(kc + nsteps) * a.stride;
    f32x4 z[NB];
    prod<Q>(z, v, K + n * (Q * Q), bb + n * Q, buf, lane, ch);
    apply<Q>(z, a.act, true, g);
    if (on) store_dsig<Q>(a.dsig, n * slice + row, a.act, z, g);
  }
  if (MODE == SWEEP_FC) {
    if (on) store_row<Q>(static_cast<float*>(a.S) + (size_t)(k + 1) * slice + row, v, g);
  } else if (MODE == SWEEP_FRES) {
    double acc = 0.0;
    if (on) {
      f32x4 cn[NB], coarse[NB];
      load_row<Q>(cn, Cs + (size_t)(k + 1) * a.cs_stride * slice + row, g);
      acc = sq_diff<Q>(v, cn);
      load_row<Q>(coarse, gn, g);
#pragma unroll
      for (int mb = 0; mb < NB; ++mb) coarse[mb] = v[mb] - coarse[mb];  // g_{l+1}^{k+1}
      store_row<Q>(gn, coarse, g);
      if (a.xn_every > 0 && (k + 1) % a.xn_every == 0)
        store_row<Q>(static_cast<float*>(a.Xn) + (size_t)(k + 1) * slice + row, cn, g);
      if (k == 0) {
        load_row<Q>(cn, Cs + row, g);
        store_row<Q>(static_cast<float*>(a.Xn) + row, cn, g);
      }
    }
    if (a.partial) {
      const double s = wg_sum(acc, red);
      if (threadIdx.x == 0) a.partial[(size_t)k * gridDim.x + tile] = s;
    }
  } else if (MODE == SWEEP_CORRF) {
    if (on && k == Nc - 1) {
      correct<Q>(v, Cs + (size_t)Nc * a.cs_stride * slice + row, Vn + (size_t)Nc * slice + row, g);
      store_row<Q>(X + (size_t)a.Nl * slice + row, v, g);
    }
  }
}

// sigma'(K_n u^n + b_n) of the fine state n: from the record, or by the forward
// product (every thread calls it: the product holds barriers)
template <int Q, bool REC>
__device__ __forceinline__ void sigma_prime(f32x4 (&d)[Geo<Q>::NB], const SweepArgs& a, size_t n, size_t slice,
                                            size_t row, bool on, float* buf, int lane) {
  constexpr int NB = Geo<Q>::NB;
  const int g = lane >> 4;
  if constexpr (REC) {
    // every lane reads a valid row; values of lanes past the batch are never stored
    load_dsig<Q>(d, a.dsig, n * slice + row, a.act, g);
  } else {
    f32x4 u[NB];
#pragma unroll
    for (int mb = 0; mb < NB; ++mb) u[mb] = 0.f;
    if (on) load_row<Q>(u, static_cast<const float*>(a.Uf) + n * slice + row, g);
    Chain own;  // loads its own first panel
    prod<Q>(d, u, static_cast<const float*>(a.K) + n * (Q * Q), static_cast<const float*>(a.b) + n * Q, buf, lane,
            own);
    apply<Q>(d, a.act, true, g);
  }
}

// ------------------------------------------------------------------ adjoint
// Interval k runs from its upper C-point (k+1)c down to kc; step j produces level
// point i = (k+1)c-1-j, linearised at the fine state of index i*stride.
template <int Q, int MODE, bool REC>
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(2, 2))) void k_adj(SweepArgs a) {
  using G = Geo<Q>;
  constexpr int NB = G::NB;
  __shared__ __attribute__((aligned(16))) float buf[2 * G::PSZ];
  __shared__ double red[WAVES];
  const int lane = threadIdx.x & 63, g = lane >> 4;
  int tile, k;
  xcd_item(tile, k);
  const int Nc = gridDim.y;
  const int e = (tile * WAVES + (threadIdx.x >> 6)) * EX + (lane & 15);
  const bool on = e < a.B;
  const size_t slice = (size_t)a.B * Q;
  const size_t row = (size_t)(on ? e : 0) * Q + 4 * g;
  const float* K = static_cast<const float*>(a.K);
  float* X = static_cast<float*>(a.X);
  const float* Gr = static_cast<const float*>(a.G);
  const float* Cs = static_cast<const float*>(a.Cs);
  const float* Vn = static_cast<const float*>(a.V);
  const int c = a.c;
  const int nsteps = MODE == MODE_SERIAL ? a.Nl : (MODE == SWEEP_CORRF ? c - 1 : c);
  const float hl = (float)a.hl, hc = (float)a.hc;
  const long top = MODE == MODE_SERIAL ? (long)a.Nl : (long)(k + 1) * c;

  f32x4 v[NB];
#pragma unroll
  for (int mb = 0; mb < NB; ++mb) v[mb] = 0.f;
  if (on) {
    if (MODE == SWEEP_FC || MODE == MODE_SERIAL) {
      if (MODE == SWEEP_FC && Vn)
        correct<Q>(v, Cs + (size_t)(k + 1) * a.cs_stride * slice + row, Vn + (size_t)(k + 1) * slice + row, g);
      else load_row<Q>(v, X + top * slice + row, g);
      if (MODE == SWEEP_FC && k == Nc - 1) store_row<Q>(static_cast<float*>(a.S) + (size_t)Nc * slice + row, v, g);
    } else if (MODE == SWEEP_FRES) {
      load_row<Q>(v, Cs + (size_t)(k + 1) * a.cs_stride * slice + row, g);
    } else {
      correct<Q>(v, Cs + (size_t)(k + 1) * a.cs_stride * slice + row, Vn + (size_t)(k + 1) * slice + row, g);
      if (k + 1 < Nc) store_row<Q>(X + top * slice + row, v, g);
    }
  }
  double acc = 0.0;  // FRES: squared residual of the lower C-point
  for (int j = 0; j < nsteps; ++j) {
    const long i = top - 1 - j;
    const size_t n = (size_t)i * a.stride;
    f32x4 d[NB], w[NB];
    sigma_prime<Q, REC>(d, a, n, slice, row, on, buf, lane);
#pragma unroll
    for (int mb = 0; mb < NB; ++mb) d[mb] = d[mb] * v[mb];
    prod_t<Q>(w, d, K + n * (Q * Q), buf, lane);
#pragma unroll
    for (int mb = 0; mb < NB; ++mb) v[mb] = v[mb] + hl * w[mb];
    if (on) {
      if (Gr) {
        f32x4 t[NB];
        load_row<Q>(t, Gr + (size_t)i * slice + row, g);
#pragma unroll
        for (int mb = 0; mb < NB; ++mb) v[mb] += t[mb];
      }
      if (MODE == SWEEP_CORRF || MODE == MODE_SERIAL) store_row<Q>(X + (size_t)i * slice + row, v, g);
    }
  }
  if constexpr (MODE == SWEEP_FRES) {
    // coarse adjoint step from the upper C-point, linearised at the fine state of
    // the interval's last step (sigma' is taken again: same operands, same
    // result), then the residual and the FAS restriction with v the relaxed
    // lower C-point. The step is evaluated exactly as the coarse level evaluates
    // its own steps (c + h_c K_n^T (sigma' * c), the product accumulated from
    // zero), so the FAS right-hand side matches the coarse operator bit for bit;
    // accumulating the product onto c instead rounds every partial sum at the
    // size of c and leaves the iteration a residual floor two orders higher.
    // The residual of the lower C-point is taken first and v is parked in its Gn
    // row, so the state's registers are free during the coarse product.
    const size_t n = (size_t)(top - nsteps) * a.stride;
    float* gn = static_cast<float*>(a.Gn) + (size_t)k * slice + row;
    const float* cup = Cs + (size_t)(k + 1) * a.cs_stride * slice + row;
    if (on) {
      f32x4 ck[NB];
      load_row<Q>(ck, Cs + (size_t)k * a.cs_stride * slice + row, g);
      acc = sq_diff<Q>(v, ck);
      if (a.xn_every > 0 && k % a.xn_every == 0)
        store_row<Q>(static_cast<float*>(a.Xn) + (size_t)k * slice + row, ck, g);
      if (k == Nc - 1) {
        load_row<Q>(ck, Cs + (size_t)Nc * a.cs_stride * slice + row, g);
        store_row<Q>(static_cast<float*>(a.Xn) + (size_t)Nc * slice + row, ck, g);
      }
      store_row<Q>(gn, v, g);
    }
    f32x4 d[NB], w[NB], t[NB];
    sigma_prime<Q, REC>(d, a, n, slice, row, on, buf, lane);
#pragma unroll
    for (int mb = 0; mb < NB; ++mb) {
      t[mb] = 0.f;
      w[mb] = 0.f;
    }
    if (on) load_row<Q>(t, cup, g);
#pragma unroll
    for (int mb = 0; mb < NB; ++mb) d[mb] = d[mb] * t[mb];
    prod_t<Q>(w, d, K + n * (Q * Q), buf, lane);
    if (on) {
      f32x4 vl[NB];
      load_row<Q>(t, cup, g);
      load_row<Q>(vl, gn, g);
#pragma unroll
      for (int mb = 0; mb < NB; ++mb) t[mb] = vl[mb] - (t[mb] + hc * w[mb]);  // g_{l+1}^k
      store_row<Q>(gn, t, g);
    }
  }

  if (MODE == SWEEP_FC) {
    if (on) store_row<Q>(static_cast<float*>(a.S) + (size_t)k * slice + row, v, g);
  } else if (MODE == SWEEP_FRES) {
    if (a.partial) {
      const double s = wg_sum(acc, red);
      if (threadIdx.x == 0) a.partial[(size_t)k * gridDim.x + tile] = s;
    }
  } else if (MODE == SWEEP_CORRF) {
    if (on && k == 0) {
      correct<Q>(v, Cs + row, Vn + row, g);
      store_row<Q>(X + row, v, g);
    }
  }
}

// ------------------------------------------------------------------ residual
// Workgroup (layer n, batch tile): the state residual Phi_n(u^n) - u^{n+1} or the
// adjoint residual lam^{n+1} + h K_n^T (sigma'(K_n u^n + b_n) * lam^{n+1}) - lam^n,
// squared and summed in fp64.
template <int Q, int DIR>
__global__ __launch_bounds__(NT) void k_resid(ResidArgs a) {
  using G = Geo<Q>;
  constexpr int NB = G::NB;
  __shared__ __attribute__((aligned(16))) float buf[2 * G::PSZ];
  __shared__ double red[WAVES];
  const int lane = threadIdx.x & 63, g = lane >> 4;
  const int n = blockIdx.x;
  const int e = (blockIdx.y * WAVES + (threadIdx.x >> 6)) * EX + (lane & 15);
  const bool on = e < a.B;
  const size_t slice = (size_t)a.B * Q;
  const size_t row = (size_t)(on ? e : 0) * Q + 4 * g;
  const float* U = static_cast<const float*>(a.U);
  const float* L = static_cast<const float*>(a.Lam);
  const float* Kn = static_cast<const float*>(a.K) + (size_t)n * (Q * Q);
  const float* bn = static_cast<const float*>(a.b) + (size_t)n * Q;
  const float h = (float)a.h;
  f32x4 v[NB], z[NB];
#pragma unroll
  for (int mb = 0; mb < NB; ++mb) v[mb] = 0.f;
  if (on) load_row<Q>(v, U + (size_t)n * slice + row, g);
  Chain ch;
  prod<Q>(z, v, Kn, bn, buf, lane, ch);
  double acc = 0.0;
  if constexpr (DIR == DIR_FWD) {
    apply<Q>(z, a.act, false, g);
    if (on) {
      f32x4 nx[NB];
      load_row<Q>(nx, U + (size_t)(n + 1) * slice + row, g);
#pragma unroll
      for (int mb = 0; mb < NB; ++mb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float d = (v[mb][r] + h * z[mb][r]) - nx[mb][r];
          acc += (double)d * (double)d;
        }
    }
  } else {
    apply<Q>(z, a.act, true, g);
    f32x4 lam[NB], w[NB];
#pragma unroll
    for (int mb = 0; mb < NB; ++mb) lam[mb] = 0.f;
    if (on) load_row<Q>(lam, L + (size_t)(n + 1) * slice + row, g);
#pragma unroll
    for (int mb = 0; mb < NB; ++mb) z[mb] = z[mb] * lam[mb];
    prod_t<Q>(w, z, Kn, buf, lane);
    if (on) {
      load_row<Q>(v, L + (size_t)n * slice + row, g);
#pragma unroll
      for (int mb = 0; mb < NB; ++mb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float d = (lam[mb][r] + h * w[mb][r]) - v[mb][r];
          acc += (double)d * (double)d;
        }
    }
  }
  const double s = wg_sum(acc, red);
  if (threadIdx.x == 0) a.partial[(size_t)blockIdx.x * gridDim.y + blockIdx.y] = s;
}

// ------------------------------------------------------------------ gradient
// Workgroup (layer n, batch chunk), 64 examples at a time: each wave forms
// s = sigma'(z) * lam^{n+1} for its 16 examples (sigma' from the record, or from
// the forward product), then s and u pass through LDS as [example][feature]
// tiles, 32 examples at a time, and dK[i][j] += sum_e s[e][i] u[e][j] runs on
// v_mfma_f32_32x32x2_f32 with the examples as the contraction index (k-slice t
// pairs examples 2t and 2t+1). The 7 x 7 output blocks of 32 x 32 are dealt to
// the four waves (block b to wave b % 4), so no cross-wave reduction is needed;
// db sums the s tile's columns. A second pass sums the chunk partials in order
// and scales by h.
template <int Q, bool REC>
__global__ __launch_bounds__(NT) void k_grad(GradArgs a) {
  using G = Geo<Q>;
  constexpr int NB = G::NB, QP = G::QP;
  constexpr int OB = QP / 32;            // 32-row output blocks per side
  constexpr int NOB = OB * OB;
  constexpr int MAXB = (NOB + WAVES - 1) / WAVES;
  constexpr int TL = QP;                 // tile pitch: rows 2t and 2t+1 on disjoint banks (QP = 32 mod 64)
  constexpr int PB = REC ? 1 : 2 * G::PSZ;
  __shared__ __attribute__((aligned(16))) float tiles[2][32 * TL];
  __shared__ __attribute__((aligned(16))) float buf[PB];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane >> 4, hh = lane >> 5, li = lane & 31;
  const int n = blockIdx.x, chunk = blockIdx.y;
  const int per = (((a.B + a.nchunks - 1) / a.nchunks) + 64 - 1) / 64 * 64;
  const int e0 = chunk * per, e1 = min(a.B, e0 + per);
  const size_t slice = (size_t)a.B * Q;
  const float* U = static_cast<const float*>(a.U) + (size_t)n * slice;
  const float* L = static_cast<const float*>(a.Lam) + (size_t)(n + 1) * slice;
  const float* Kn = static_cast<const float*>(a.K) + (size_t)n * (Q * Q);
  const float* bn = static_cast<const float*>(a.b) + (size_t)n * Q;
  f32x16 acc[MAXB];
#pragma unroll
  for (int b = 0; b < MAXB; ++b) acc[b] = 0.f;
  float dbacc = 0.f;  // thread t < Q: column sum of s
  int xo[MAXB], yo[MAXB];  // this wave's output blocks: row and column offsets
#pragma unroll
  for (int b = 0; b < MAXB; ++b) {
    const int ob = wave + WAVES * b;
    xo[b] = 32 * (ob / OB);
    yo[b] = 32 * (ob % OB);
  }
  float* st = tiles[0];
  float* ut = tiles[1];
  for (int base = e0; base < e1; base += 64) {
    const int e = base + wave * EX + (lane & 15);
    const bool on = e < e1;
    const size_t row = (size_t)(on ? e : 0) * Q + 4 * g;
    f32x4 u[NB], s[NB], d[NB];
#pragma unroll
    for (int mb = 0; mb < NB; ++mb) u[mb] = 0.f;
    if (on) load_row<Q>(u, U + row, g);
    if constexpr (REC) {
      load_dsig<Q>(d, a.dsig, (size_t)n * slice + row, a.act, g);
    } else {
      Chain own;  // loads its own first panel
      prod<Q>(d, u, Kn, bn, buf, lane, own);
      apply<Q>(d, a.act, true, g);
    }
    // lam^{n+1} is loaded after the product, which needs the registers
#pragma unroll
    for (int mb = 0; mb < NB; ++mb) s[mb] = 0.f;
    if (on) load_row<Q>(s, L + row, g);
#pragma unroll
    for (int mb = 0; mb < NB; ++mb) s[mb] = d[mb] * s[mb];
    // two halves of 32 examples: waves 0-1, then waves 2-3 fill the tiles
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      if ((wave >> 1) == half) {
        const int er = (wave & 1) * EX + (lane & 15);
#pragma unroll
        for (int mb = 0; mb < NB; ++mb) {
          *reinterpret_cast<f32x4*>(st + er * TL + 16 * mb + 4 * g) = s[mb];
          *reinterpret_cast<f32x4*>(ut + er * TL + 16 * mb + 4 * g) = u[mb];
        }
      }
      __syncthreads();
#pragma unroll 4
      for (int t = 0; t < 16; ++t) {
        const float* sr = st + (2 * t + hh) * TL + li;
        const float* ur = ut + (2 * t + hh) * TL + li;
#pragma unroll
        for (int b = 0; b < MAXB; ++b)
          if (wave + WAVES * b < NOB)
            acc[b] = __builtin_amdgcn_mfma_f32_32x32x2f32(sr[xo[b]], ur[yo[b]], acc[b], 0, 0, 0);
      }
      if (threadIdx.x < Q)
        for (int t = 0; t < 32; ++t) dbacc += st[t * TL + threadIdx.x];
      __syncthreads();
    }
  }
  float* out = static_cast<float*>(a.partial) + ((size_t)n * a.nchunks + chunk) * (Q * Q + Q);
#pragma unroll
  for (int b = 0; b < MAXB; ++b) {
    const int ob = wave + WAVES * b;
    if (ob >= NOB) continue;
    const int j = 32 * (ob % OB) + li;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int i = 32 * (ob / OB) + 8 * (r >> 2) + 4 * hh + (r & 3);
      if (i < Q && j < Q) out[(size_t)i * Q + j] = acc[b][r];
    }
  }
  if (threadIdx.x < Q) out[(size_t)Q * Q + threadIdx.x] = dbacc;
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

// ------------------------------------------------------------------ launchers
template <int Q>
hipError_t sweep(int dir, const SweepArgs& a, hipStream_t st, int* partials) {
  const long Nc = a.Nl / a.c;
  if (Nc > 65535) return hipErrorNotSupported;  // intervals index the grid's y dimension
  const dim3 grid((a.B + EX * WAVES - 1) / (EX * WAVES), (unsigned)Nc);
  if (partials) *partials = (int)(grid.x * grid.y);
  const bool rec = a.dsig != nullptr;
  if (dir == DIR_FWD) {
    // only the final F-relaxation writes the sigma' record
    if (a.mode == SWEEP_FC) launch(k_fwd<Q, SWEEP_FC, false>, grid, NT, 0, st, a);
    else if (a.mode == SWEEP_FRES) launch(k_fwd<Q, SWEEP_FRES, false>, grid, NT, 0, st, a);
    else if (rec) launch(k_fwd<Q, SWEEP_CORRF, true>, grid, NT, 0, st, a);
    else launch(k_fwd<Q, SWEEP_CORRF, false>, grid, NT, 0, st, a);
  } else if (rec) {
    if (a.mode == SWEEP_FC) launch(k_adj<Q, SWEEP_FC, true>, grid, NT, 0, st, a);
    else if (a.mode == SWEEP_FRES) launch(k_adj<Q, SWEEP_FRES, true>, grid, NT, 0, st, a);
    else launch(k_adj<Q, SWEEP_CORRF, true>, grid, NT, 0, st, a);
  } else {
    if (a.mode == SWEEP_FC) launch(k_adj<Q, SWEEP_FC, false>, grid, NT, 0, st, a);
    else if (a.mode == SWEEP_FRES) launch(k_adj<Q, SWEEP_FRES, false>, grid, NT, 0, st, a);
    else launch(k_adj<Q, SWEEP_CORRF, false>, grid, NT, 0, st, a);
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
  const dim3 grid((s.B + EX * WAVES - 1) / (EX * WAVES), 1);
  if (dir == DIR_FWD) {
    if (s.dsig) launch(k_fwd<Q, MODE_SERIAL, true>, grid, NT, 0, st, a);
    else launch(k_fwd<Q, MODE_SERIAL, false>, grid, NT, 0, st, a);
  } else {
    if (s.dsig) launch(k_adj<Q, MODE_SERIAL, true>, grid, NT, 0, st, a);
    else launch(k_adj<Q, MODE_SERIAL, false>, grid, NT, 0, st, a);
  }
  return hipGetLastError();
}

template <int Q>
hipError_t resid(int dir, const ResidArgs& a, hipStream_t st, int* partials) {
  const dim3 grid((unsigned)a.N, (unsigned)((a.B + EX * WAVES - 1) / (EX * WAVES)));
  if (partials) *partials = (int)(grid.x * grid.y);
  if (dir == DIR_FWD) launch(k_resid<Q, DIR_FWD>, grid, NT, 0, st, a);
  else launch(k_resid<Q, DIR_ADJ>, grid, NT, 0, st, a);
  return hipGetLastError();
}

template <int Q>
hipError_t grad(const GradArgs& a, hipStream_t st) {
  if (a.dsig) launch(k_grad<Q, true>, dim3(a.N, a.nchunks), NT, 0, st, a);
  else launch(k_grad<Q, false>, dim3(a.N, a.nchunks), NT, 0, st, a);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  const size_t tot = (size_t)a.N * (Q * Q + Q);
  launch(k_grad_final, (unsigned)((tot + 255) / 256), 256, 0, st, a, Q * Q, Q);
  return hipGetLastError();
}

}  // namespace wide

bool wide_width_supported(int q) { return q == 220; }

hipError_t wide_sweep(int q, int dir, const SweepArgs& a, hipStream_t st, int* partials) {
  if (q == 220) return wide::sweep<220>(dir, a, st, partials);
  return hipErrorNotSupported;
}

hipError_t wide_serial(int q, int dir, const SerialArgs& a, hipStream_t st) {
  if (q == 220) return wide::serial<220>(dir, a, st);
  return hipErrorNotSupported;
}

hipError_t wide_resid(int q, int dir, const ResidArgs& a, hipStream_t st, int* partials) {
  if (q == 220) return wide::resid<220>(dir, a, st, partials);
  return hipErrorNotSupported;
}

hipError_t wide_grad(int q, const GradArgs& a, hipStream_t st) {
  if (q == 220) return wide::grad<220>(a, st);
  return hipErrorNotSupported;
}

}  // namespace lp
