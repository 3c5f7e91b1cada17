// 3x3 convolution layers with C = 8 channels (fp32) on the matrix cores
// (gfx950 v_mfma_f32_16x16x4_f32), as an implicit GEMM.
//
// Layer operator (Section 2.1, K(theta) a convolution): cross-correlation with
// zero "same" padding, z[co][y][x] = sum_{ci,ty,tx} K[co][ci][ty][tx] u[ci][y+ty-1][x+tx-1] + b[co].
//
// One workgroup owns one example for all steps of an interval; the example's
// state lives in LDS in zero-padded [C][H+2][W+2] buffers (ping-pong). The image
// is split into "pair-pixels": pair-pixel P = (Y, x) stands for the two output
// pixels (2Y, x) and (2Y+1, x). A 16 x 16 x 96 product gives the outputs of 16
// pair-pixels for all (co, dy) in {0..7} x {0,1} (the M = 16 rows), contracting
// over a 4-row window: k = (ci, r, tx), r = 0..3 the rows 2Y-1 .. 2Y+2. Row dy of
// the output uses window rows r = dy .. dy+2, so the expanded weight matrix is
// Wbig[k][(co,dy)] = K[co][ci][r - dy][tx] when 0 <= r - dy <= 2 and 0 otherwise
// (72 of every 96 products are useful). k-slice s and lane group g = lane/16 map
// to ci = g + 4 (s / 12), r = (s % 12) / 3, tx = s % 3, so a lane's patch read for
// slice s is a fixed LDS offset from its pair-pixel's base.
//
// The adjoint step applies K^T, a cross-correlation with the kernel flipped and
// its channel axes swapped; the same product runs with that weight gather.
// The weight gradient contracts over pair-pixels instead: dWbig[(co,dy)][k] =
// sum_P s[co][2Y+dy][x] patch[P][k], then dK[co][ci][ty][tx] = sum_dy dWbig[(co,dy)][(ci, ty+dy, tx)].
#include "lp_device.h"
#include "lp_internal.h"

namespace lp {
namespace conv {

typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int CH = 8;                  // channels
constexpr int MAXPD = 32;              // padded image side bound (H, W <= 30)
constexpr int BUF = CH * MAXPD * MAXPD;  // floats per padded state buffer
constexpr int KW = CH * CH * 9;        // weights per layer
constexpr int WV = KW + CH;            // weights + bias staged per layer
constexpr int WAVES = 4;
constexpr int NT = 64 * WAVES;
constexpr int MAXT = 8;                // tiles per wave held in registers (NT16 <= WAVES * MAXT)
constexpr int MODE_SERIAL = 3;

struct Geo {
  int H, W, PW, PHW, HW, q, NPP, NT16;
  __device__ Geo(int h, int w)
      : H(h), W(w), PW(w + 2), PHW((h + 2) * (w + 2)), HW(h * w), q(CH * h * w), NPP(h / 2 * w),
        NT16((h / 2 * w + 15) / 16) {}
};

__device__ __forceinline__ float tanh_fast(float x) {
  const float t = __builtin_amdgcn_exp2f(-2.885390081777927f * fabsf(x));  // exp(-2|x|)
  return copysignf((1.f - t) * __builtin_amdgcn_rcpf(1.f + t), x);
}

__device__ __forceinline__ float act_v(float z, int act) {
  if (act == ACT_TANH) return tanh_fast(z);
  if (act == ACT_RELU) return z > 0.f ? z : 0.f;
  if (act == ACT_SMOOTHRELU) return act_f<float, ACT_SMOOTHRELU>(z);
  return z;
}

__device__ __forceinline__ float dact_v(float z, int act) {
  if (act == ACT_TANH) {
    const float t = tanh_fast(z);
    return 1.f - t * t;
  }
  if (act == ACT_RELU) return z > 0.f ? 1.f : 0.f;
  if (act == ACT_SMOOTHRELU) return dact_f<float, ACT_SMOOTHRELU>(z);
  return 1.f;
}

__device__ __forceinline__ void stage_w(float* sw, const float* __restrict__ K, const float* __restrict__ b,
                                        size_t n) {
  for (int i = threadIdx.x; i < WV; i += NT) sw[i] = i < KW ? K[n * KW + i] : b[n * CH + (i - KW)];
}

__device__ __forceinline__ void zero_buf(float* buf, int n) {
  for (int i = threadIdx.x; i < n; i += NT) buf[i] = 0.f;
}

// global example row [C][H][W] -> padded LDS interior, optionally corrected:
// dst = c + (v - c) when v is given (Algorithm 1, steps 4-5).
__device__ __forceinline__ void row_in(float* buf, const float* __restrict__ c, const float* __restrict__ v,
                                       const Geo& g) {
  for (int i = threadIdx.x; i < g.q; i += NT) {
    const int ch = i / g.HW, rem = i - ch * g.HW, y = rem / g.W, x = rem - y * g.W;
    float val = c[i];
    if (v) val = val + (v[i] - val);
    buf[ch * g.PHW + (y + 1) * g.PW + x + 1] = val;
  }
}

__device__ __forceinline__ void row_out(float* __restrict__ dst, const float* buf, const Geo& g) {
  for (int i = threadIdx.x; i < g.q; i += NT) {
    const int ch = i / g.HW, rem = i - ch * g.HW, y = rem / g.W, x = rem - y * g.W;
    dst[i] = buf[ch * g.PHW + (y + 1) * g.PW + x + 1];
  }
}

__device__ __forceinline__ void row_copy(float* __restrict__ dst, const float* __restrict__ src, int q) {
  for (int i = threadIdx.x; i < q; i += NT) dst[i] = src[i];
}

// Expanded weights of one lane for the 24 k-slices: A-row (co, dy) = (n/2, n%2)
// with n = lane % 16, slice s and group g = lane / 16. TR selects the adjoint's
// transposed, flipped kernel.
template <bool TR>
__device__ __forceinline__ void gather_w(float (&wr)[24], const float* sw, int lane) {
  const int n = lane & 15, g = lane >> 4;
  const int co = n >> 1, dy = n & 1;
#pragma unroll
  for (int s = 0; s < 24; ++s) {
    const int ci = g + 4 * (s / 12), r = (s % 12) / 3, tx = s % 3, ty = r - dy;
    float w = 0.f;
    if (ty >= 0 && ty <= 2) w = TR ? sw[ci * 72 + co * 9 + (2 - ty) * 3 + (2 - tx)] : sw[co * 72 + ci * 9 + ty * 3 + tx];
    wr[s] = w;
  }
}

// Lane's pair-pixel in tile t and its LDS patch base.
struct TileLane {
  int P;      // pair-pixel (clamped into range)
  bool valid;
  int Y, x;
  int base;   // LDS offset of (ci = lane/16, row 2Y, col x) in padded coordinates
};

__device__ __forceinline__ TileLane tile_lane(int t, int lane, const Geo& g) {
  TileLane L;
  const int P = 16 * t + (lane & 15);
  L.valid = P < g.NPP;
  L.P = L.valid ? P : g.NPP - 1;
  L.Y = L.P / g.W;
  L.x = L.P - L.Y * g.W;
  L.base = (lane >> 4) * g.PHW + 2 * L.Y * g.PW + L.x;
  return L;
}

// acc += Wbig^T-slices x patches of the buffer for one tile
__device__ __forceinline__ f32x4 conv_tile(const float (&wr)[24], const float* buf, int base, const Geo& g,
                                           f32x4 acc) {
#pragma unroll
  for (int s = 0; s < 24; ++s) {
    const int off = (s / 12) * 4 * g.PHW + ((s % 12) / 3) * g.PW + (s % 3);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(wr[s], buf[base + off], acc, 0, 0, 0);
  }
  return acc;
}

// Output element of accumulator register r for the lane: channel and row.
__device__ __forceinline__ int out_ch(int lane, int r) { return 2 * (lane >> 4) + (r >> 1); }

__device__ __forceinline__ double wg_sum(double v, double* red) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  double s = 0.0;
  if (threadIdx.x == 0)
    for (int w = 0; w < WAVES; ++w) s += red[w];
  __syncthreads();
  return s;
}

// ------------------------------------------------------------------ forward
template <int MODE>
__global__ __launch_bounds__(NT) void k_fwd(SweepArgs a, int H, int W) {
  __shared__ float buf[2][BUF];
  __shared__ float sw[2][WV];
  __shared__ double red[WAVES];
  const Geo g(H, W);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int k = blockIdx.x, Nc = gridDim.x;
  const int e = blockIdx.y;
  const size_t slice = (size_t)a.B * g.q;
  const size_t eo = (size_t)e * g.q;
  const float* K = static_cast<const float*>(a.K);
  const float* bb = static_cast<const float*>(a.b);
  float* X = static_cast<float*>(a.X);
  const float* G = static_cast<const float*>(a.G);
  const float* Cs = static_cast<const float*>(a.Cs);
  const float* Vn = static_cast<const float*>(a.V);
  const int c = a.c;
  const int nsteps = MODE == MODE_SERIAL ? a.Nl : (MODE == SWEEP_CORRF ? c - 1 : c);
  const float hl = (float)a.hl, hc = (float)a.hc;
  const long kc = MODE == MODE_SERIAL ? 0 : (long)k * c;

  zero_buf(&buf[0][0], 2 * BUF);
  stage_w(sw[0], K, bb, (size_t)kc * a.stride);
  __syncthreads();
  if (MODE == SWEEP_FC || MODE == MODE_SERIAL) {
    // a pending coarse-grid correction of the previous cycle is applied on the fly
    if (MODE == SWEEP_FC && Vn) row_in(buf[0], Cs + (size_t)k * a.cs_stride * slice + eo, Vn + (size_t)k * slice + eo, g);
    else row_in(buf[0], X + kc * slice + eo, nullptr, g);
    if (MODE == SWEEP_FC && k == 0) row_copy(static_cast<float*>(a.S) + eo, X + eo, g.q);
  } else if (MODE == SWEEP_FRES) {
    row_in(buf[0], Cs + (size_t)k * a.cs_stride * slice + eo, nullptr, g);
  } else {
    row_in(buf[0], Cs + (size_t)k * a.cs_stride * slice + eo, Vn + (size_t)k * slice + eo, g);
  }
  __syncthreads();
  if (MODE == SWEEP_CORRF && k > 0) row_out(X + kc * slice + eo, buf[0], g);

  float coarse[MAXT][4];
  for (int j = 0; j < nsteps; ++j) {
    const int cur = j & 1;
    float wr[24];
    gather_w<false>(wr, sw[cur], lane);
    stage_w(sw[cur ^ 1], K, bb, (size_t)(kc + (j + 1 < nsteps ? j + 1 : j)) * a.stride);
    const float* gi = G ? G + (kc + j + 1) * slice + eo : nullptr;
    float* xo = (MODE == SWEEP_CORRF || MODE == MODE_SERIAL) ? X + (kc + j + 1) * slice + eo : nullptr;
#pragma unroll
    for (int tt = 0; tt < MAXT; ++tt) {
      const int t = wave + tt * WAVES;
      if (t >= g.NT16) break;
      const TileLane L = tile_lane(t, lane, g);
      f32x4 acc;
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[r] = sw[cur][KW + out_ch(lane, r)];
      acc = conv_tile(wr, buf[cur], L.base, g, acc);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int co = out_ch(lane, r), y = 2 * L.Y + (r & 1);
        const int pos = co * g.PHW + (y + 1) * g.PW + L.x + 1;
        const int go = co * g.HW + y * g.W + L.x;
        const float old = buf[cur][pos];
        const float sg = act_v(acc[r], a.act);
        if (MODE == SWEEP_FRES && j == 0) coarse[tt][r] = old + hc * sg;
        float nv = old + hl * sg;
        if (L.valid) {
          if (gi) nv += gi[go];
          buf[cur ^ 1][pos] = nv;
          if (xo) xo[go] = nv;
        }
      }
    }
    __syncthreads();
  }
  const float* fin = buf[nsteps & 1];
  if (MODE == SWEEP_FC) {
    row_out(static_cast<float*>(a.S) + (size_t)(k + 1) * slice + eo, fin, g);
  } else if (MODE == SWEEP_FRES) {
    const float* cn = Cs + (size_t)(k + 1) * a.cs_stride * slice + eo;
    float* gn = static_cast<float*>(a.Gn) + (size_t)(k + 1) * slice + eo;
    double acc = 0.0;
#pragma unroll
    for (int tt = 0; tt < MAXT; ++tt) {
      const int t = wave + tt * WAVES;
      if (t >= g.NT16) break;
      const TileLane L = tile_lane(t, lane, g);
      if (!L.valid) continue;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int co = out_ch(lane, r), y = 2 * L.Y + (r & 1);
        const int pos = co * g.PHW + (y + 1) * g.PW + L.x + 1;
        const int go = co * g.HW + y * g.W + L.x;
        const float f = fin[pos];
        const float rr = f - cn[go];
        acc += (double)rr * (double)rr;
        gn[go] = f - coarse[tt][r];  // g_{l+1}^{k+1} = f_{k+1} - Phi_{l+1}(C_k)
      }
    }
    if (a.xn_every > 0 && (k + 1) % a.xn_every == 0)
      row_copy(static_cast<float*>(a.Xn) + (size_t)(k + 1) * slice + eo, cn, g.q);
    if (k == 0) row_copy(static_cast<float*>(a.Xn) + eo, Cs + eo, g.q);
    if (a.partial) {
      const double s = wg_sum(acc, red);
      if (threadIdx.x == 0) a.partial[(size_t)blockIdx.x * gridDim.y + blockIdx.y] = s;
    }
  } else if (MODE == SWEEP_CORRF) {
    if (k == Nc - 1) {
      const float* cs = Cs + (size_t)Nc * a.cs_stride * slice + eo;
      const float* vs = Vn + (size_t)Nc * slice + eo;
      float* xo = X + (size_t)a.Nl * slice + eo;
      for (int i = threadIdx.x; i < g.q; i += NT) xo[i] = cs[i] + (vs[i] - cs[i]);
    }
  }
}

// ------------------------------------------------------------------ adjoint
// Step: u^n -> LDS, d = sigma'(K u + b), s = d * lam -> LDS, lam' = lam + h K^T s (+ g).
template <int MODE>
__global__ __launch_bounds__(NT) void k_adj(SweepArgs a, int H, int W) {
  __shared__ float buf[3][BUF];  // lam (ping-pong) and the primal state / s
  __shared__ float sw[2][WV];
  __shared__ double red[WAVES];
  const Geo g(H, W);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int k = blockIdx.x, Nc = gridDim.x;
  const int e = blockIdx.y;
  const size_t slice = (size_t)a.B * g.q;
  const size_t eo = (size_t)e * g.q;
  const float* K = static_cast<const float*>(a.K);
  const float* bb = static_cast<const float*>(a.b);
  const float* Uf = static_cast<const float*>(a.Uf);
  float* X = static_cast<float*>(a.X);
  const float* G = static_cast<const float*>(a.G);
  const float* Cs = static_cast<const float*>(a.Cs);
  const float* Vn = static_cast<const float*>(a.V);
  const int c = a.c;
  const int nsteps = MODE == MODE_SERIAL ? a.Nl : (MODE == SWEEP_CORRF ? c - 1 : c);
  const float hl = (float)a.hl, hc = (float)a.hc;
  const long top = MODE == MODE_SERIAL ? (long)a.Nl : (long)(k + 1) * c;
  float* bu = buf[2];

  zero_buf(&buf[0][0], 3 * BUF);
  stage_w(sw[0], K, bb, (size_t)(top - 1) * a.stride);
  __syncthreads();
  if (MODE == SWEEP_FC || MODE == MODE_SERIAL) {
    if (MODE == SWEEP_FC && Vn)
      row_in(buf[0], Cs + (size_t)(k + 1) * a.cs_stride * slice + eo, Vn + (size_t)(k + 1) * slice + eo, g);
    else row_in(buf[0], X + top * slice + eo, nullptr, g);
    if (MODE == SWEEP_FC && k == Nc - 1) row_copy(static_cast<float*>(a.S) + (size_t)Nc * slice + eo, X + top * slice + eo, g.q);
  } else if (MODE == SWEEP_FRES) {
    row_in(buf[0], Cs + (size_t)(k + 1) * a.cs_stride * slice + eo, nullptr, g);
  } else {
    row_in(buf[0], Cs + (size_t)(k + 1) * a.cs_stride * slice + eo, Vn + (size_t)(k + 1) * slice + eo, g);
  }
  __syncthreads();
  if (MODE == SWEEP_CORRF && k + 1 < Nc) row_out(X + top * slice + eo, buf[0], g);

  float dd[MAXT][4];
  float cu[MAXT][4];  // FRES: the upper C-point, then the coarse step
  if (MODE == SWEEP_FRES) {
#pragma unroll
    for (int tt = 0; tt < MAXT; ++tt) {
      const int t = wave + tt * WAVES;
      if (t >= g.NT16) break;
      const TileLane L = tile_lane(t, lane, g);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int co = out_ch(lane, r), y = 2 * L.Y + (r & 1);
        cu[tt][r] = buf[0][co * g.PHW + (y + 1) * g.PW + L.x + 1];
      }
    }
  }
  for (int j = 0; j < nsteps; ++j) {
    const int cur = j & 1;
    const long i = top - 1 - j;
    float wf[24], wt[24];
    gather_w<false>(wf, sw[cur], lane);
    gather_w<true>(wt, sw[cur], lane);
    row_in(bu, Uf + (size_t)i * a.stride * slice + eo, nullptr, g);
    __syncthreads();
    // d = sigma'(K u + b)
#pragma unroll
    for (int tt = 0; tt < MAXT; ++tt) {
      const int t = wave + tt * WAVES;
      if (t >= g.NT16) break;
      const TileLane L = tile_lane(t, lane, g);
      f32x4 acc;
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[r] = sw[cur][KW + out_ch(lane, r)];
      acc = conv_tile(wf, bu, L.base, g, acc);
#pragma unroll
      for (int r = 0; r < 4; ++r) dd[tt][r] = dact_v(acc[r], a.act);
    }
    __syncthreads();
    // s = d * lam into the primal buffer (its halo stays zero)
#pragma unroll
    for (int tt = 0; tt < MAXT; ++tt) {
      const int t = wave + tt * WAVES;
      if (t >= g.NT16) break;
      const TileLane L = tile_lane(t, lane, g);
      if (!L.valid) continue;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int co = out_ch(lane, r), y = 2 * L.Y + (r & 1);
        const int pos = co * g.PHW + (y + 1) * g.PW + L.x + 1;
        bu[pos] = dd[tt][r] * buf[cur][pos];
      }
    }
    stage_w(sw[cur ^ 1], K, bb, (size_t)(j + 1 < nsteps ? i - 1 : i) * a.stride);
    __syncthreads();
    const float* gi = G ? G + (size_t)i * slice + eo : nullptr;
    float* xo = (MODE == SWEEP_CORRF || MODE == MODE_SERIAL) ? X + (size_t)i * slice + eo : nullptr;
#pragma unroll
    for (int tt = 0; tt < MAXT; ++tt) {
      const int t = wave + tt * WAVES;
      if (t >= g.NT16) break;
      const TileLane L = tile_lane(t, lane, g);
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
      acc = conv_tile(wt, bu, L.base, g, acc);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int co = out_ch(lane, r), y = 2 * L.Y + (r & 1);
        const int pos = co * g.PHW + (y + 1) * g.PW + L.x + 1;
        const int go = co * g.HW + y * g.W + L.x;
        float nv = buf[cur][pos] + hl * acc[r];
        if (L.valid) {
          if (gi) nv += gi[go];
          buf[cur ^ 1][pos] = nv;
          if (xo) xo[go] = nv;
        }
      }
    }
    if (MODE == SWEEP_FRES && j == nsteps - 1) {
      // coarse adjoint step from the upper C-point, linearised at the same fine state
      __syncthreads();
#pragma unroll
      for (int tt = 0; tt < MAXT; ++tt) {
        const int t = wave + tt * WAVES;
        if (t >= g.NT16) break;
        const TileLane L = tile_lane(t, lane, g);
        if (!L.valid) continue;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int co = out_ch(lane, r), y = 2 * L.Y + (r & 1);
          bu[co * g.PHW + (y + 1) * g.PW + L.x + 1] = dd[tt][r] * cu[tt][r];
        }
      }
      __syncthreads();
#pragma unroll
      for (int tt = 0; tt < MAXT; ++tt) {
        const int t = wave + tt * WAVES;
        if (t >= g.NT16) break;
        const TileLane L = tile_lane(t, lane, g);
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
        acc = conv_tile(wt, bu, L.base, g, acc);
#pragma unroll
        for (int r = 0; r < 4; ++r) cu[tt][r] = cu[tt][r] + hc * acc[r];
      }
    }
    __syncthreads();
  }
  const float* fin = buf[nsteps & 1];
  if (MODE == SWEEP_FC) {
    row_out(static_cast<float*>(a.S) + (size_t)k * slice + eo, fin, g);
  } else if (MODE == SWEEP_FRES) {
    const float* ck = Cs + (size_t)k * a.cs_stride * slice + eo;
    float* gn = static_cast<float*>(a.Gn) + (size_t)k * slice + eo;
    double acc = 0.0;
#pragma unroll
    for (int tt = 0; tt < MAXT; ++tt) {
      const int t = wave + tt * WAVES;
      if (t >= g.NT16) break;
      const TileLane L = tile_lane(t, lane, g);
      if (!L.valid) continue;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int co = out_ch(lane, r), y = 2 * L.Y + (r & 1);
        const int pos = co * g.PHW + (y + 1) * g.PW + L.x + 1;
        const int go = co * g.HW + y * g.W + L.x;
        const float f = fin[pos];
        const float rr = f - ck[go];
        acc += (double)rr * (double)rr;
        gn[go] = f - cu[tt][r];  // g_{l+1}^k = f_k - Phibar_{l+1}(C_{k+1})
      }
    }
    if (a.xn_every > 0 && k % a.xn_every == 0) row_copy(static_cast<float*>(a.Xn) + (size_t)k * slice + eo, ck, g.q);
    if (k == Nc - 1)
      row_copy(static_cast<float*>(a.Xn) + (size_t)Nc * slice + eo, Cs + (size_t)Nc * a.cs_stride * slice + eo, g.q);
    if (a.partial) {
      const double s = wg_sum(acc, red);
      if (threadIdx.x == 0) a.partial[(size_t)blockIdx.x * gridDim.y + blockIdx.y] = s;
    }
  } else if (MODE == SWEEP_CORRF) {
    if (k == 0) {
      float* xo = X + eo;
      for (int i = threadIdx.x; i < g.q; i += NT) xo[i] = Cs[eo + i] + (Vn[eo + i] - Cs[eo + i]);
    }
  }
}

// ------------------------------------------------------------------ residual
// Workgroup (n, example): forward r = Phi_n(U[n]) - U[n+1]; adjoint
// r = Phibar_n(Lam[n+1]) - Lam[n]; writes the example's sum of r^2.
template <int DIR>
__global__ __launch_bounds__(NT) void k_resid(ResidArgs a, int H, int W) {
  __shared__ float buf[2][BUF];
  __shared__ float sw[WV];
  __shared__ double red[WAVES];
  const Geo g(H, W);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n = blockIdx.x, e = blockIdx.y;
  const size_t slice = (size_t)a.B * g.q;
  const size_t eo = (size_t)e * g.q;
  const float* U = static_cast<const float*>(a.U);
  const float* Lm = static_cast<const float*>(a.Lam);
  const float h = (float)a.h;
  zero_buf(&buf[0][0], 2 * BUF);
  stage_w(sw, static_cast<const float*>(a.K), static_cast<const float*>(a.b), n);
  __syncthreads();
  row_in(buf[0], U + (size_t)n * slice + eo, nullptr, g);
  if (DIR == DIR_ADJ) row_in(buf[1], Lm + (size_t)(n + 1) * slice + eo, nullptr, g);
  __syncthreads();
  float wf[24];
  gather_w<false>(wf, sw, lane);
  float dd[MAXT][4];
  double acc2 = 0.0;
#pragma unroll
  for (int tt = 0; tt < MAXT; ++tt) {
    const int t = wave + tt * WAVES;
    if (t >= g.NT16) break;
    const TileLane L = tile_lane(t, lane, g);
    f32x4 acc;
#pragma unroll
    for (int r = 0; r < 4; ++r) acc[r] = sw[KW + out_ch(lane, r)];
    acc = conv_tile(wf, buf[0], L.base, g, acc);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int co = out_ch(lane, r), y = 2 * L.Y + (r & 1);
      const int pos = co * g.PHW + (y + 1) * g.PW + L.x + 1;
      const int go = co * g.HW + y * g.W + L.x;
      if (DIR == DIR_FWD) {
        const float rr = (buf[0][pos] + h * act_v(acc[r], a.act)) - U[(size_t)(n + 1) * slice + eo + go];
        if (L.valid) acc2 += (double)rr * (double)rr;
      } else {
        dd[tt][r] = dact_v(acc[r], a.act) * buf[1][pos];
      }
    }
  }
  if (DIR == DIR_ADJ) {
    __syncthreads();
#pragma unroll
    for (int tt = 0; tt < MAXT; ++tt) {
      const int t = wave + tt * WAVES;
      if (t >= g.NT16) break;
      const TileLane L = tile_lane(t, lane, g);
      if (!L.valid) continue;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int co = out_ch(lane, r), y = 2 * L.Y + (r & 1);
        buf[0][co * g.PHW + (y + 1) * g.PW + L.x + 1] = dd[tt][r];
      }
    }
    __syncthreads();
    float wt[24];
    gather_w<true>(wt, sw, lane);
#pragma unroll
    for (int tt = 0; tt < MAXT; ++tt) {
      const int t = wave + tt * WAVES;
      if (t >= g.NT16) break;
      const TileLane L = tile_lane(t, lane, g);
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
      acc = conv_tile(wt, buf[0], L.base, g, acc);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int co = out_ch(lane, r), y = 2 * L.Y + (r & 1);
        const int pos = co * g.PHW + (y + 1) * g.PW + L.x + 1;
        const int go = co * g.HW + y * g.W + L.x;
        const float rr = (buf[1][pos] + h * acc[r]) - Lm[(size_t)n * slice + eo + go];
        if (L.valid) acc2 += (double)rr * (double)rr;
      }
    }
  }
  const double s = wg_sum(acc2, red);
  if (threadIdx.x == 0) a.partial[(size_t)blockIdx.x * gridDim.y + blockIdx.y] = s;
}

// ------------------------------------------------------------------ gradient
// Workgroup (layer n, batch chunk). Per example: s = sigma'(K u + b) * lam^{n+1}
// (the forward product), written to LDS; then dWbig[(co,dy)][k] += s[co][2Y+dy][x] *
// patch[P][k] with the pair-pixels as contraction index (k-slice = 4 pair-pixels,
// lane group = one of them): A = s (rows (co,dy)), B = patches (96 columns in 6
// blocks of 16). db sums s. Waves split the pair-pixel slices; the workgroup's
// partial is combined in a fixed order.
constexpr int GOUT = 16 * 96 + CH;  // dWbig then db per chunk

__global__ __launch_bounds__(NT) void k_grad(GradArgs a, int H, int W) {
  __shared__ float buf[2][BUF];  // u (padded), s (padded)
  __shared__ float sw[WV];
  __shared__ float red[GOUT];
  const Geo g(H, W);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n = blockIdx.x, chunk = blockIdx.y;
  const int per = (a.B + a.nchunks - 1) / a.nchunks;
  const int e0 = chunk * per, e1 = min(a.B, e0 + per);
  const size_t slice = (size_t)a.B * g.q;
  const float* U = static_cast<const float*>(a.U) + (size_t)n * slice;
  const float* Lm = static_cast<const float*>(a.Lam) + (size_t)(n + 1) * slice;
  zero_buf(&buf[0][0], 2 * BUF);
  stage_w(sw, static_cast<const float*>(a.K), static_cast<const float*>(a.b), n);
  __syncthreads();
  float wf[24];
  gather_w<false>(wf, sw, lane);
  // B-operand offsets: column k = 16 nb + lane%16 -> (ci, r, tx), relative to the
  // pair-pixel's (row 2Y, col x) origin in padded coordinates
  int koff[6];
#pragma unroll
  for (int nb = 0; nb < 6; ++nb) {
    const int kk = 16 * nb + (lane & 15);
    const int ci = kk / 12, r = (kk % 12) / 3, tx = kk % 3;
    koff[nb] = ci * g.PHW + r * g.PW + tx;
  }
  f32x4 acc[6];
#pragma unroll
  for (int nb = 0; nb < 6; ++nb) acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  float dbacc = 0.f;
  const int nsl = (g.NPP + 3) / 4;  // pair-pixel slices of 4
  for (int e = e0; e < e1; ++e) {
    row_in(buf[0], U + (size_t)e * g.q, nullptr, g);
    __syncthreads();
#pragma unroll
    for (int tt = 0; tt < MAXT; ++tt) {
      const int t = wave + tt * WAVES;
      if (t >= g.NT16) break;
      const TileLane L = tile_lane(t, lane, g);
      f32x4 z;
#pragma unroll
      for (int r = 0; r < 4; ++r) z[r] = sw[KW + out_ch(lane, r)];
      z = conv_tile(wf, buf[0], L.base, g, z);
      if (!L.valid) continue;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int co = out_ch(lane, r), y = 2 * L.Y + (r & 1);
        const int go = co * g.HW + y * g.W + L.x;
        const float s = dact_v(z[r], a.act) * Lm[(size_t)e * g.q + go];
        buf[1][co * g.PHW + (y + 1) * g.PW + L.x + 1] = s;
      }
    }
    __syncthreads();
    // contraction over pair-pixels
    for (int sl = wave; sl < nsl; sl += WAVES) {
      const int P = 4 * sl + (lane >> 4);
      const bool ok = P < g.NPP;
      const int Pc = ok ? P : g.NPP - 1;
      const int Y = Pc / g.W, x = Pc - Y * g.W;
      const int nA = lane & 15, co = nA >> 1, dy = nA & 1;
      const float av = ok ? buf[1][co * g.PHW + (2 * Y + dy + 1) * g.PW + x + 1] : 0.f;
      const int pb = 2 * Y * g.PW + x;  // (row 2Y-1+r, col x-1+tx) padded = (2Y+r, x+tx)
#pragma unroll
      for (int nb = 0; nb < 6; ++nb)
        acc[nb] = __builtin_amdgcn_mfma_f32_16x16x4f32(av, buf[0][pb + koff[nb]], acc[nb], 0, 0, 0);
    }
    // db: thread t sums channel t % 8 over pixels t/8, t/8 + 32, ...
    {
      const int ch = threadIdx.x & (CH - 1);
      for (int p = threadIdx.x >> 3; p < g.HW; p += NT / CH) {
        const int y = p / g.W, x = p - y * g.W;
        dbacc += buf[1][ch * g.PHW + (y + 1) * g.PW + x + 1];
      }
    }
    __syncthreads();
  }
  // combine waves in order: D[(co,dy) = 4(lane/16)+r][k = 16 nb + lane%16]
  for (int w = 0; w < WAVES; ++w) {
    if (wave == w) {
#pragma unroll
      for (int nb = 0; nb < 6; ++nb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int o = (4 * (lane >> 4) + r) * 96 + 16 * nb + (lane & 15);
          red[o] = (w == 0 ? 0.f : red[o]) + acc[nb][r];
        }
    }
    __syncthreads();
  }
  // db: per channel, the 32 thread partials in thread order
  __shared__ float dbp[NT];
  dbp[threadIdx.x] = dbacc;
  __syncthreads();
  if (threadIdx.x < CH) {
    float s = 0.f;
    for (int t = threadIdx.x; t < NT; t += CH) s += dbp[t];
    red[16 * 96 + threadIdx.x] = s;
  }
  __syncthreads();
  float* out = static_cast<float*>(a.partial) + ((size_t)n * a.nchunks + chunk) * GOUT;
  for (int o = threadIdx.x; o < GOUT; o += NT) out[o] = red[o];
}

// dK[n][co][ci][ty][tx] = h sum_chunks sum_dy dWbig[(co,dy)][(ci, ty+dy, tx)], db[n][co] = h sum db.
__global__ __launch_bounds__(NT) void k_grad_final(GradArgs a) {
  const size_t o = (size_t)blockIdx.x * NT + threadIdx.x;
  if (o >= (size_t)a.N * (KW + CH)) return;
  const size_t n = o / (KW + CH);
  const int r = (int)(o - n * (KW + CH));
  const float* p = static_cast<const float*>(a.partial) + n * a.nchunks * GOUT;
  float s = 0.f;
  if (r < KW) {
    const int co = r / 72, ci = (r % 72) / 9, ty = (r % 9) / 3, tx = r % 3;
    for (int ch = 0; ch < a.nchunks; ++ch)
      for (int dy = 0; dy < 2; ++dy) {
        const int kk = ci * 12 + (ty + dy) * 3 + tx;
        s += p[(size_t)ch * GOUT + (2 * co + dy) * 96 + kk];
      }
    static_cast<float*>(a.dK)[n * KW + r] = s * (float)a.h;
  } else {
    for (int ch = 0; ch < a.nchunks; ++ch) s += p[(size_t)ch * GOUT + 16 * 96 + (r - KW)];
    static_cast<float*>(a.db)[n * CH + (r - KW)] = s * (float)a.h;
  }
}

}  // namespace conv

bool conv_supported(const Shape& s) {
  return s.layer == 1 && s.dtype == 0 && s.C == conv::CH && s.H % 2 == 0 && s.H >= 2 && s.W >= 4 &&
         s.H + 2 <= conv::MAXPD && s.W + 2 <= conv::MAXPD &&
         (s.H / 2 * s.W + 15) / 16 <= conv::WAVES * conv::MAXT;
}

int conv_tile(const Shape&) { return 1; }

int conv_grad_chunks(int B, int N) {
  const int want = (2048 + N - 1) / N;
  const int ch = want < B ? want : B;
  return ch < 1 ? 1 : ch;
}

hipError_t conv_sweep(const Shape& s, int dir, const SweepArgs& a, hipStream_t st, int* partials) {
  const dim3 grid(a.Nl / a.c, a.B);
  if (partials) *partials = (int)(grid.x * grid.y);
  using namespace conv;
  if (dir == DIR_FWD) {
    if (a.mode == SWEEP_FC) k_fwd<SWEEP_FC><<<grid, NT, 0, st>>>(a, s.H, s.W);
    else if (a.mode == SWEEP_FRES) k_fwd<SWEEP_FRES><<<grid, NT, 0, st>>>(a, s.H, s.W);
    else k_fwd<SWEEP_CORRF><<<grid, NT, 0, st>>>(a, s.H, s.W);
  } else {
    if (a.mode == SWEEP_FC) k_adj<SWEEP_FC><<<grid, NT, 0, st>>>(a, s.H, s.W);
    else if (a.mode == SWEEP_FRES) k_adj<SWEEP_FRES><<<grid, NT, 0, st>>>(a, s.H, s.W);
    else k_adj<SWEEP_CORRF><<<grid, NT, 0, st>>>(a, s.H, s.W);
  }
  return hipGetLastError();
}

hipError_t conv_serial(const Shape& s, int dir, const SerialArgs& sa, hipStream_t st) {
  SweepArgs a{};
  a.act = sa.act;
  a.mode = conv::MODE_SERIAL;
  a.K = sa.K;
  a.b = sa.b;
  a.Uf = sa.Uf;
  a.B = sa.B;
  a.Nl = sa.Nl;
  a.c = 1;
  a.stride = sa.stride;
  a.hl = sa.hl;
  a.X = sa.X;
  a.G = sa.G;
  const dim3 grid(1, sa.B);
  if (dir == DIR_FWD) conv::k_fwd<conv::MODE_SERIAL><<<grid, conv::NT, 0, st>>>(a, s.H, s.W);
  else conv::k_adj<conv::MODE_SERIAL><<<grid, conv::NT, 0, st>>>(a, s.H, s.W);
  return hipGetLastError();
}

hipError_t conv_resid(const Shape& s, int dir, const ResidArgs& a, hipStream_t st, int* partials) {
  const dim3 grid(a.N, a.B);
  if (partials) *partials = (int)(grid.x * grid.y);
  if (dir == DIR_FWD) conv::k_resid<DIR_FWD><<<grid, conv::NT, 0, st>>>(a, s.H, s.W);
  else conv::k_resid<DIR_ADJ><<<grid, conv::NT, 0, st>>>(a, s.H, s.W);
  return hipGetLastError();
}

hipError_t conv_grad(const Shape& s, const GradArgs& a, hipStream_t st) {
  conv::k_grad<<<dim3(a.N, a.nchunks), conv::NT, 0, st>>>(a, s.H, s.W);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  const size_t tot = (size_t)a.N * (conv::KW + conv::CH);
  conv::k_grad_final<<<(unsigned)((tot + conv::NT - 1) / conv::NT), conv::NT, 0, st>>>(a);
  return hipGetLastError();
}

}  // namespace lp
