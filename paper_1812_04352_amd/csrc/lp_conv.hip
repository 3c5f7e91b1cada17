// 3x3 convolution layers with C = 8 channels (fp32) on the matrix cores
// (gfx950 v_mfma_f32_16x16x4_f32), as an implicit GEMM.
//
// Layer operator (Section 2.1, K(theta) a convolution): cross-correlation with
// zero "same" padding, z[co][y][x] = sum_{ci,ty,tx} K[co][ci][ty][tx] u[ci][y+ty-1][x+tx-1] + b[co].
//
// One workgroup owns one example for all steps of an interval (the sweeps below
// describe the register and LDS layout). The image is split into
// "pair-pixels": pair-pixel P = (Y, x) stands for the two output
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
#include <algorithm>

#include "lp_device.h"
#include "lp_internal.h"

namespace lp {
namespace conv {

typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int CH = 8;                  // channels
constexpr int KW = CH * CH * 9;        // weights per layer
constexpr int WV = KW + CH;            // weights + bias staged per layer
constexpr int NT = 256;                // threads of the elementwise kernels
constexpr int MODE_SERIAL = 3;

__device__ __forceinline__ float tanh_fast(float x) {
  const float t = __builtin_amdgcn_exp2f(-2.885390081777927f * fabsf(x));  // exp(-2|x|)
  return copysignf((1.f - t) * __builtin_amdgcn_rcpf(1.f + t), x);
}

__device__ __forceinline__ void stage_w(float* sw, const float* __restrict__ K, const float* __restrict__ b,
                                        size_t n, int nt = NT) {
  for (int i = threadIdx.x; i < WV; i += nt) sw[i] = i < KW ? K[n * KW + i] : b[n * CH + (i - KW)];
}

// A layer's weights and bias on their way to LDS in a sweep: thread t carries
// entries t, t + nt, ... (WPT of them), fetched at the start of a step and
// written after its product, so the load's latency overlaps the matrix-core work.
template <int WPT>
__device__ __forceinline__ void stage_fetch(float (&r)[WPT], const float* __restrict__ K,
                                            const float* __restrict__ b, size_t n, int nt) {
#pragma unroll
  for (int p = 0; p < WPT; ++p) {
    const int i = threadIdx.x + p * nt;
    r[p] = i < KW ? K[n * KW + i] : i < WV ? b[n * CH + (i - KW)] : 0.f;
  }
}

template <int WPT>
__device__ __forceinline__ void stage_put(float* sw, const float (&r)[WPT], int nt) {
#pragma unroll
  for (int p = 0; p < WPT; ++p) {
    const int i = threadIdx.x + p * nt;
    if (i < WV) sw[i] = r[p];
  }
}

__device__ __forceinline__ void zero_buf(float* buf, int n, int nt = NT) {
  for (int i = threadIdx.x; i < n; i += nt) buf[i] = 0.f;
}

__device__ __forceinline__ void row_copy(float* __restrict__ dst, const float* __restrict__ src, int q, int nt = NT) {
  for (int i = threadIdx.x; i < q; i += nt) dst[i] = src[i];
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

// acc += Wbig^T-slices x patches of the buffer for one tile
__device__ __forceinline__ f32x4 conv_tile(const float (&wr)[24], const float* buf, int base, int cs, int pw,
                                           f32x4 acc) {
#pragma unroll
  for (int s = 0; s < 24; ++s) {
    const int off = (s / 12) * 4 * cs + ((s % 12) / 3) * pw + (s % 3);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(wr[s], buf[base + off], acc, 0, 0, 0);
  }
  return acc;
}

// ------------------------------------------------------------------ sweeps
// One workgroup runs one example through one interval (or, serially, through a
// whole level). The state being evolved lives in registers at the lane's own
// output pixels; the one LDS image buffer holds whatever the next product reads
// (the forward state, the adjoint's primal state and then s = d * lam), with a
// zero halo. Wave w owns tiles w*TPW .. w*TPW+TPW-1; a 28 x 28 image (25 tiles)
// runs on 4 waves, one per SIMD, the last one carrying three ghost tiles (lanes
// past the image repeat its last pair-pixel and write nothing), so every wave
// does the same work and no loop over tiles branches. Each product runs for all
// of the wave's tiles before the elementwise work. The adjoint issues the loads
// of the next step's primal state before its second product.

// Sweep geometry, computed on the host.
struct SGeo {
  int H, W;
  int PW;    // padded row length W + 2
  int CS;    // LDS channel stride: >= (H+2)(W+2) and = 16 (mod 64), so the four
             // 16-lane groups of a patch read (channels g, g+1, g+2, g+3) hit
             // disjoint banks
  int HW, q;
  int NPP;   // pair-pixels (H/2) W
  int NT16;  // tiles of 16 pair-pixels
  int NW;    // waves per workgroup: ceil(NT16 / TPW)
};

constexpr int TPW = 7;   // tiles per wave (each costs 4 registers per per-pixel array)
constexpr int MAXW = 8;  // waves per workgroup at most

constexpr __host__ __device__ SGeo make_geo(int H, int W) {
  const int phw = (H + 2) * (W + 2);
  const int npp = H / 2 * W, nt16 = (H / 2 * W + 15) / 16;
  return SGeo{H, W, W + 2, phw + (((16 - phw) % 64) + 64) % 64, H * W, CH * H * W, npp, nt16, (nt16 + TPW - 1) / TPW};
}

// Geometry of a kernel instance: compile-time for the specialised image sizes
// (the patch reads then use immediate LDS offsets), else the launch argument.
template <int GH, int GW>
__device__ __forceinline__ SGeo geo_of(const SGeo& ga) {
  if constexpr (GH == 0) return ga;
  else return make_geo(GH, GW);
}

// The lane's pair-pixel in tile t: patch origin, own output offsets (register 0:
// channel 2*(lane/16), row 2Y, column x) and whether it lies in the image; lanes
// past the last pair-pixel repeat it and never write.
struct Px {
  int base, lds, gl;
  bool ok;
};

__device__ __forceinline__ Px px_of(const SGeo& g, int t, int lane) {
  Px p;
  int P = 16 * t + (lane & 15);
  p.ok = P < g.NPP;
  if (!p.ok) P = g.NPP - 1;
  const int Y = P / g.W, x = P - Y * g.W, grp = lane >> 4;
  p.base = grp * g.CS + 2 * Y * g.PW + x;
  p.lds = 2 * grp * g.CS + (2 * Y + 1) * g.PW + x + 1;
  p.gl = 2 * grp * g.HW + 2 * Y * g.W + x;
  return p;
}

// accumulator register r: channel 2*(lane/16) + r/2, row 2Y + r%2
__device__ __forceinline__ int lds_r(const SGeo& g, const Px& p, int r) { return p.lds + (r >> 1) * g.CS + (r & 1) * g.PW; }
__device__ __forceinline__ int gl_r(const SGeo& g, const Px& p, int r) { return p.gl + (r >> 1) * g.HW + (r & 1) * g.W; }

__device__ __forceinline__ f32x4 ld_px(const float* __restrict__ src, const SGeo& g, const Px& p) {
  f32x4 v;
#pragma unroll
  for (int r = 0; r < 4; ++r) v[r] = src[gl_r(g, p, r)];
  return v;
}

__device__ __forceinline__ void st_px(float* __restrict__ dst, f32x4 v, const SGeo& g, const Px& p) {
#pragma unroll
  for (int r = 0; r < 4; ++r) dst[gl_r(g, p, r)] = v[r];
}

__device__ __forceinline__ void put_px(float* buf, f32x4 v, const SGeo& g, const Px& p) {
#pragma unroll
  for (int r = 0; r < 4; ++r) buf[lds_r(g, p, r)] = v[r];
}

// The interior of the zero-halo LDS image (channel stride CS, padded rows PW) to a
// state row [C][H][W] in global memory: thread i takes values 4i .. 4i+3, which lie
// in one image row when W % 4 == 0 (else one value at a time).
__device__ __forceinline__ void store_img(float* __restrict__ dst, const float* buf, const SGeo& g, int nt) {
  if (g.W % 4 == 0) {
    for (int i = 4 * (int)threadIdx.x; i < g.q; i += 4 * nt) {
      const int c = i / g.HW, r = i - c * g.HW, y = r / g.W, x = r - y * g.W;
      const float* s = buf + c * g.CS + (y + 1) * g.PW + x + 1;
      *reinterpret_cast<f32x4*>(dst + i) = f32x4{s[0], s[1], s[2], s[3]};
    }
  } else {
    for (int i = threadIdx.x; i < g.q; i += nt) {
      const int c = i / g.HW, r = i - c * g.HW, y = r / g.W, x = r - y * g.W;
      dst[i] = buf[c * g.CS + (y + 1) * g.PW + x + 1];
    }
  }
}

// Products of the wave's tiles, z[tt] = init + Wbig^T x patches.
__device__ __forceinline__ void conv_tiles(f32x4 (&z)[TPW], const float (&wr)[24], const float* buf, const SGeo& g,
                                           int t0, int lane, f32x4 init) {
#pragma unroll
  for (int tt = 0; tt < TPW; ++tt) z[tt] = conv_tile(wr, buf, px_of(g, t0 + tt, lane).base, g.CS, g.PW, init);
}

__device__ __forceinline__ f32x4 bias_px(const float* sw, int lane) {
  const int co = 2 * (lane >> 4);
  return f32x4{sw[KW + co], sw[KW + co], sw[KW + co + 1], sw[KW + co + 1]};
}

// sigma (D = false) or sigma' (D = true) of the wave's tiles, one branch on the
// activation for all of them
template <bool D>
__device__ __forceinline__ void act_tiles(f32x4 (&z)[TPW], int act) {
  switch (act) {
    case ACT_TANH:
#pragma unroll
      for (int tt = 0; tt < TPW; ++tt) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float t = tanh_fast(z[tt][r]);
          z[tt][r] = D ? 1.f - t * t : t;
        }
      }
      break;
    case ACT_RELU:
#pragma unroll
      for (int tt = 0; tt < TPW; ++tt) {
#pragma unroll
        for (int r = 0; r < 4; ++r) z[tt][r] = D ? (z[tt][r] > 0.f ? 1.f : 0.f) : (z[tt][r] > 0.f ? z[tt][r] : 0.f);
      }
      break;
    case ACT_SMOOTHRELU:
#pragma unroll
      for (int tt = 0; tt < TPW; ++tt) {
#pragma unroll
        for (int r = 0; r < 4; ++r)
          z[tt][r] = D ? dact_f<float, ACT_SMOOTHRELU>(z[tt][r]) : act_f<float, ACT_SMOOTHRELU>(z[tt][r]);
      }
      break;
    default:
      if (D) {
#pragma unroll
        for (int tt = 0; tt < TPW; ++tt) z[tt] = f32x4{1.f, 1.f, 1.f, 1.f};
      }
      break;
  }
}

// sigma'(z) of one value, the arithmetic of act_tiles<true>
__device__ __forceinline__ float dact_one(float z, int act) {
  switch (act) {
    case ACT_TANH: {
      const float t = tanh_fast(z);
      return 1.f - t * t;
    }
    case ACT_RELU: return z > 0.f ? 1.f : 0.f;
    case ACT_SMOOTHRELU: return dact_f<float, ACT_SMOOTHRELU>(z);
    default: return 1.f;
  }
}

// The sigma' record of one (layer, example) is a block in the kernels' own tile
// order: slot (wave w, tile tt, lane) = (w TPW + tt) 64 + lane holds the lane's
// four values of that tile (its accumulator registers r = 0..3), as one word of
// four 0/1 bytes for ReLU or as four fp32 values otherwise. Every lane of every
// tile, ghost tiles included, writes its slot, so a block is whole once written
// and each lane reads its values with one vector load. Blocks are indexed by
// layer * B + example.
__host__ __device__ constexpr size_t rec_block_bytes(const SGeo& g, bool bits) {
  return (size_t)g.NW * 64 * (bits ? 4 : TPW * 16);
}

// One lane's record of one step, all of its TPW tiles, as loaded (kept packed
// until used): RB, ReLU's TPW x 4 decisions as bits 4 tt + r of one word (one
// word per lane and step); else TPW quadruples of fp32 values.
template <bool RB>
struct RecW;
template <>
struct RecW<true> {
  uint32_t w;
};
template <>
struct RecW<false> {
  f32x4 f[TPW];
};

// slots: RB, lane of wave t0 / TPW; else, lane of tile t0 + tt
__device__ __forceinline__ size_t rec_slot(int t, int lane) { return (size_t)t * 64 + lane; }

// rec_put takes the pre-activations of the lane's four values in each of its tiles
template <bool RB>
__device__ __forceinline__ void rec_put(void* rec, size_t blk, const SGeo& g, int t0, int lane, const f32x4 (&z)[TPW],
                                        int act) {
  uint8_t* base = static_cast<uint8_t*>(rec) + blk * rec_block_bytes(g, RB);
  if constexpr (RB) {
    uint32_t w = 0;
#pragma unroll
    for (int tt = 0; tt < TPW; ++tt)
#pragma unroll
      for (int r = 0; r < 4; ++r) w |= (z[tt][r] > 0.f ? 1u : 0u) << (4 * tt + r);
    reinterpret_cast<uint32_t*>(base)[rec_slot(t0 / TPW, lane)] = w;
  } else {
#pragma unroll
    for (int tt = 0; tt < TPW; ++tt) {
      f32x4 d;
#pragma unroll
      for (int r = 0; r < 4; ++r) d[r] = dact_one(z[tt][r], act);
      reinterpret_cast<f32x4*>(base)[rec_slot(t0 + tt, lane)] = d;
    }
  }
}

template <bool RB>
__device__ __forceinline__ RecW<RB> rec_load(const void* rec, size_t blk, const SGeo& g, int t0, int lane) {
  const uint8_t* base = static_cast<const uint8_t*>(rec) + blk * rec_block_bytes(g, RB);
  RecW<RB> r;
  if constexpr (RB) {
    r.w = reinterpret_cast<const uint32_t*>(base)[rec_slot(t0 / TPW, lane)];
  } else {
#pragma unroll
    for (int tt = 0; tt < TPW; ++tt) r.f[tt] = reinterpret_cast<const f32x4*>(base)[rec_slot(t0 + tt, lane)];
  }
  return r;
}

// sigma' of the lane's four values in its tile tt
template <bool RB>
__device__ __forceinline__ f32x4 rec_val(const RecW<RB>& r, int tt) {
  if constexpr (!RB) {
    return r.f[tt];
  } else {
    f32x4 d;
#pragma unroll
    for (int q = 0; q < 4; ++q) d[q] = (r.w >> (4 * tt + q)) & 1u ? 1.f : 0.f;
    return d;
  }
}

__device__ __forceinline__ double wg_sum_n(double v, double* red, int nw) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  double s = 0.0;
  if (threadIdx.x == 0)
    for (int w = 0; w < nw; ++w) s += red[w];
  return s;
}

// The sweeps' workgroup for (interval, example). Workgroups go to the eight XCDs
// in turn by linear id, and each XCD has its own L2. This mapping hands each XCD
// one contiguous range of the interval-fastest order instead, so the intervals
// of one example, which share their C-points, run on one XCD at about the same
// time, and the eight XCDs work on examples far apart. It is a bijection of the
// grid for any size. (Measured on 28x28 images, 1024 examples, 512 layers: the
// correction sweeps run 8-14 % faster; a mapping that gives each XCD a block of
// intervals for every example cuts the fetched bytes further but runs no faster
// than the plain order.)
struct Blk {
  int k, ex;
};
__device__ __forceinline__ Blk sweep_block() {
  const unsigned nx = gridDim.x, T = nx * gridDim.y;
  const unsigned p = blockIdx.x + blockIdx.y * nx, x = p % 8u;
  const unsigned L = x * (T / 8u) + min(x, T % 8u) + p / 8u;
  return {(int)(L % nx), (int)(L / nx)};
}

// RK: the sigma' record kind (0 none, 1 ReLU bits, 2 fp32 values). HG: the level
// has right-hand-side rows (every level but the finest); a step requests its row
// before the product, so the load overlaps the matrix-core work (three waves per
// SIMD leave room for it).
template <int MODE, int GH, int GW, int RK, bool HG>
__global__ __launch_bounds__(64 * MAXW)
__attribute__((amdgpu_waves_per_eu(HG || MODE == SWEEP_FRES ? 3 : MODE == SWEEP_CORRF || MODE == MODE_SERIAL ? 4 : 1, 8)))
void k_fwd(SweepArgs a, SGeo ga) {
  constexpr bool REC = RK != 0, RB = RK == 1;
  // weight entries per thread while staging (the specialised geometry fixes the thread count)
  constexpr int WPT = GH ? (WV + 64 * make_geo(GH, GW).NW - 1) / (64 * make_geo(GH, GW).NW) : (WV + 63) / 64;
  const SGeo g = geo_of<GH, GW>(ga);
  extern __shared__ float lds[];
  float* buf = lds;               // CH * CS
  float* sw = lds + CH * g.CS;    // two layers
  __shared__ double red[MAXW];
  int lane = threadIdx.x & 63;
  // the wave's first tile; in the correction sweep it is taken as uniform across
  // the wave, so the tile bases derived from it live in scalar registers (measured
  // per mode: 2.8 % faster there, slower or spilling in the others)
  constexpr bool UNIF = MODE == SWEEP_CORRF;
  const int wave = threadIdx.x >> 6;
  const int t0 = (UNIF ? __builtin_amdgcn_readfirstlane(wave) : wave) * TPW, nt = blockDim.x;
  const Blk wb = sweep_block();
  const int k = wb.k, Nc = gridDim.x;
  const size_t slice = (size_t)a.B * g.q, eo = (size_t)wb.ex * g.q;
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

  zero_buf(buf, CH * g.CS, nt);
  stage_w(sw, K, bb, (size_t)kc * a.stride, nt);
  // starting state: C-point k, corrected when a coarse solution is given
  const float* src;
  const float* vsrc = nullptr;
  if (MODE == SWEEP_FC || MODE == MODE_SERIAL) {
    // a pending coarse-grid correction of the previous cycle is applied on the fly
    if (MODE == SWEEP_FC && Vn) {
      src = Cs + (size_t)k * a.cs_stride * slice + eo;
      vsrc = Vn + (size_t)k * slice + eo;
    } else {
      src = X + kc * slice + eo;
    }
  } else {
    src = Cs + (size_t)k * a.cs_stride * slice + eo;
    if (MODE == SWEEP_CORRF) vsrc = Vn + (size_t)k * slice + eo;
  }
  f32x4 v[TPW];
  if constexpr (MODE == SWEEP_CORRF) {
    // every load of the starting state is issued before the first use: a test of
    // vsrc inside the tile loop splits it into one wait per tile (measured 4.8 %
    // faster here; the FC sweep measured slower with it and keeps the tile loop)
#pragma unroll
    for (int tt = 0; tt < TPW; ++tt) v[tt] = ld_px(src, g, px_of(g, t0 + tt, lane));
    if (vsrc) {
      f32x4 cv[TPW];
#pragma unroll
      for (int tt = 0; tt < TPW; ++tt) cv[tt] = ld_px(vsrc, g, px_of(g, t0 + tt, lane));
#pragma unroll
      for (int tt = 0; tt < TPW; ++tt) v[tt] = v[tt] + (cv[tt] - v[tt]);
    }
  } else {
#pragma unroll
    for (int tt = 0; tt < TPW; ++tt) {
      const Px p = px_of(g, t0 + tt, lane);
      v[tt] = ld_px(src, g, p);
      if (vsrc) v[tt] = v[tt] + (ld_px(vsrc, g, p) - v[tt]);
    }
  }
  __syncthreads();  // halo zeroed
#pragma unroll
  for (int tt = 0; tt < TPW; ++tt) {
    const Px p = px_of(g, t0 + tt, lane);
    if (p.ok) {
      put_px(buf, v[tt], g, p);
      if (MODE == SWEEP_CORRF && k > 0) st_px(X + kc * slice + eo, v[tt], g, p);
    }
  }
  if (MODE == SWEEP_FC && k == 0) row_copy(static_cast<float*>(a.S) + eo, X + eo, g.q, nt);
  __syncthreads();

  // the final F-relaxation (and a level-0 serial solve) records sigma'(z) of every
  // layer; CORRF then also takes the product of the layer before the next C-point
  constexpr bool rec = REC && (MODE == SWEEP_CORRF || MODE == MODE_SERIAL);
  constexpr int extra = MODE == SWEEP_CORRF && rec ? 1 : 0;
  // FRES on a coarse level parks the coarse step's value Phi_{l+1}(C_k) in its
  // output row (the next level's right-hand side) instead of holding it in
  // registers through the interval: with the level's right-hand-side rows also in
  // flight, holding it spills, and each reload from scratch would wait for those
  // rows too. The epilogue reads it back together with the upper C-point.
  constexpr bool PARK = MODE == SWEEP_FRES && HG;
  float* const gn = MODE == SWEEP_FRES ? static_cast<float*>(a.Gn) + (size_t)(k + 1) * slice + eo : nullptr;
  f32x4 coarse[PARK ? 1 : TPW];
  for (int j = 0; j < nsteps; ++j) {
    // an empty asm statement makes the lane index opaque to the optimiser, so the
    // tile offsets derived from it are recomputed each step instead of being kept
    // live in registers through the loop (fewer registers, more resident waves)
    asm volatile("" : "+v"(lane));
    const float* swc = sw + (j & 1) * WV;
    // the serial solve stages in one go (measured faster there)
    constexpr bool SPLIT = MODE != MODE_SERIAL;
    const size_t nxt = (size_t)(kc + (j + 1 < nsteps ? j + 1 : j + extra)) * a.stride;
    float wreg[SPLIT ? WPT : 1];
    if constexpr (SPLIT) stage_fetch<WPT>(wreg, K, bb, nxt, nt);
    else stage_w(sw + ((j & 1) ^ 1) * WV, K, bb, nxt, nt);
    f32x4 z[TPW], gv[HG ? TPW : 1];
    if constexpr (HG) {
#pragma unroll
      for (int tt = 0; tt < TPW; ++tt) gv[tt] = ld_px(G + (kc + j + 1) * slice + eo, g, px_of(g, t0 + tt, lane));
    }
    {
      float wr[24];
      gather_w<false>(wr, swc, lane);
      const f32x4 bias = bias_px(swc, lane);
      conv_tiles(z, wr, buf, g, t0, lane, bias);
    }
    if constexpr (rec) {
      const size_t blk = (size_t)(kc + j) * a.stride * a.B + wb.ex;
      rec_put<RB>(a.dsig, blk, g, t0, lane, z, a.act);
    }
    act_tiles<false>(z, a.act);
    // (without HG the kernel keeps the form it was tuned in: a run-time test that
    // is false on the finest level)
    const float* gi = !HG && G ? G + (kc + j + 1) * slice + eo : nullptr;
#pragma unroll
    for (int tt = 0; tt < TPW; ++tt) {
      if (MODE == SWEEP_FRES && j == 0) {
        if constexpr (PARK) {
          const Px p = px_of(g, t0 + tt, lane);
          if (p.ok) st_px(gn, v[tt] + hc * z[tt], g, p);
        } else {
          coarse[tt] = v[tt] + hc * z[tt];
        }
      }
      v[tt] = v[tt] + hl * z[tt];
      if constexpr (HG) v[tt] += gv[tt];
      else if (gi) v[tt] += ld_px(gi, g, px_of(g, t0 + tt, lane));
    }
    __syncthreads();  // every read of the step's input is done
#pragma unroll
    for (int tt = 0; tt < TPW; ++tt) {
      const Px p = px_of(g, t0 + tt, lane);
      if (p.ok) put_px(buf, v[tt], g, p);
    }
    if constexpr (SPLIT) stage_put<WPT>(sw + ((j & 1) ^ 1) * WV, wreg, nt);
    __syncthreads();
    // the new state is written out from the LDS image in row order, four values
    // per thread and store (the next write of the buffer is a step away, behind
    // that step's first barrier)
    if (MODE == SWEEP_CORRF || MODE == MODE_SERIAL) store_img(X + (kc + j + 1) * slice + eo, buf, g, nt);
  }

  if constexpr (extra != 0) {
    // sigma' of the layer before the next C-point, from the last F-point (in the
    // buffer) and that layer's weights (staged by the last step)
    const float* swc = sw + (nsteps & 1) * WV;
    f32x4 z[TPW];
    float wr[24];
    gather_w<false>(wr, swc, lane);
    conv_tiles(z, wr, buf, g, t0, lane, bias_px(swc, lane));
    const size_t blk = (size_t)(kc + nsteps) * a.stride * a.B + wb.ex;
    rec_put<RB>(a.dsig, blk, g, t0, lane, z, a.act);
  }
  if (MODE == SWEEP_FC) {
    float* so = static_cast<float*>(a.S) + (size_t)(k + 1) * slice + eo;
#pragma unroll
    for (int tt = 0; tt < TPW; ++tt) {
      const Px p = px_of(g, t0 + tt, lane);
      if (p.ok) st_px(so, v[tt], g, p);
    }
  } else if (MODE == SWEEP_FRES) {
    const float* cn = Cs + (size_t)(k + 1) * a.cs_stride * slice + eo;
    double acc = 0.0;
    if constexpr (PARK) {
      asm volatile("" ::: "memory");  // read the parked row back from memory
      f32x4 cv[TPW], pk[TPW];
#pragma unroll
      for (int tt = 0; tt < TPW; ++tt) {
        const Px p = px_of(g, t0 + tt, lane);
        cv[tt] = ld_px(cn, g, p);
        pk[tt] = ld_px(gn, g, p);  // this lane's own step-0 stores (ghost lanes: unused)
      }
#pragma unroll
      for (int tt = 0; tt < TPW; ++tt) {
        const Px p = px_of(g, t0 + tt, lane);
        if (p.ok) {
          const f32x4 rr = v[tt] - cv[tt];
#pragma unroll
          for (int r = 0; r < 4; ++r) acc += (double)rr[r] * (double)rr[r];
          st_px(gn, v[tt] - pk[tt], g, p);  // g_{l+1}^{k+1} = f_{k+1} - Phi_{l+1}(C_k)
        }
      }
    } else {
#pragma unroll
      for (int tt = 0; tt < TPW; ++tt) {
        const Px p = px_of(g, t0 + tt, lane);
        if (p.ok) {
          const f32x4 rr = v[tt] - ld_px(cn, g, p);
#pragma unroll
          for (int r = 0; r < 4; ++r) acc += (double)rr[r] * (double)rr[r];
          st_px(gn, v[tt] - coarse[tt], g, p);  // g_{l+1}^{k+1} = f_{k+1} - Phi_{l+1}(C_k)
        }
      }
    }
    if (a.xn_every > 0 && (k + 1) % a.xn_every == 0)
      row_copy(static_cast<float*>(a.Xn) + (size_t)(k + 1) * slice + eo, cn, g.q, nt);
    if (k == 0) row_copy(static_cast<float*>(a.Xn) + eo, Cs + eo, g.q, nt);
    if (a.partial) {
      const double s = wg_sum_n(acc, red, g.NW);
      if (threadIdx.x == 0) a.partial[(size_t)k * gridDim.y + wb.ex] = s;
    }
  } else if (MODE == SWEEP_CORRF) {
    if (k == Nc - 1) {
      const float* cs = Cs + (size_t)Nc * a.cs_stride * slice + eo;
      const float* vs = Vn + (size_t)Nc * slice + eo;
      float* xo = X + (size_t)a.Nl * slice + eo;
      for (int i = threadIdx.x; i < g.q; i += nt) xo[i] = cs[i] + (vs[i] - cs[i]);
    }
  }
}

// Adjoint step at level point i: d = sigma'(K u + b) with u the fine primal state
// of point i (or d read from the sigma' record: REC), s = d * lam,
// lam' = lam + h K^T s (+ g).
template <int MODE, int GH, int GW, int RK, bool HG>
__global__ __launch_bounds__(64 * MAXW)
__attribute__((amdgpu_waves_per_eu(HG ? 3 : RK == 1 ? 4 : RK == 2 ? 3 : 1, 8)))
void k_adj(SweepArgs a, SGeo ga) {
  constexpr bool REC = RK != 0, RB = RK == 1;
  // weight entries per thread while staging (the specialised geometry fixes the thread count)
  constexpr int WPT = GH ? (WV + 64 * make_geo(GH, GW).NW - 1) / (64 * make_geo(GH, GW).NW) : (WV + 63) / 64;
  const SGeo g = geo_of<GH, GW>(ga);
  extern __shared__ float lds[];
  float* buf = lds;               // CH * CS: u, then s
  float* sw = lds + CH * g.CS;    // two layers
  __shared__ double red[MAXW];
  int lane = threadIdx.x & 63;
  // the wave's first tile; in the FRES sweep with a record it is taken as uniform
  // across the wave, so the tile bases derived from it live in scalar registers
  // (this removes the finest FRES kernel's spill; measured per mode, the other
  // sweeps are slower or spill with it)
  constexpr bool UNIF = MODE == SWEEP_FRES && RK != 0;
  const int wave = threadIdx.x >> 6;
  const int t0 = (UNIF ? __builtin_amdgcn_readfirstlane(wave) : wave) * TPW, nt = blockDim.x;
  const Blk wb = sweep_block();
  const int k = wb.k, Nc = gridDim.x;
  const size_t slice = (size_t)a.B * g.q, eo = (size_t)wb.ex * g.q;
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
  const size_t ustep = (size_t)a.stride * slice;

  zero_buf(buf, CH * g.CS, nt);
  stage_w(sw, K, bb, (size_t)(top - 1) * a.stride, nt);
  const float* src;
  const float* vsrc = nullptr;
  if (MODE == SWEEP_FC || MODE == MODE_SERIAL) {
    if (MODE == SWEEP_FC && Vn) {
      src = Cs + (size_t)(k + 1) * a.cs_stride * slice + eo;
      vsrc = Vn + (size_t)(k + 1) * slice + eo;
    } else {
      src = X + top * slice + eo;
    }
  } else {
    src = Cs + (size_t)(k + 1) * a.cs_stride * slice + eo;
    if (MODE == SWEEP_CORRF) vsrc = Vn + (size_t)(k + 1) * slice + eo;
  }
  // every load of the starting values is issued before the first use: a test of
  // vsrc inside the tile loop splits it into one wait per tile (measured: adjoint
  // CORRF 6.6 % faster, FC unchanged)
  f32x4 lam[TPW], un[TPW];
#pragma unroll
  for (int tt = 0; tt < TPW; ++tt) {
    const Px p = px_of(g, t0 + tt, lane);
    lam[tt] = ld_px(src, g, p);
    if (!REC) un[tt] = ld_px(Uf + (size_t)(top - 1) * ustep + eo, g, p);
  }
  if (vsrc) {
    f32x4 cv[TPW];
#pragma unroll
    for (int tt = 0; tt < TPW; ++tt) cv[tt] = ld_px(vsrc, g, px_of(g, t0 + tt, lane));
#pragma unroll
    for (int tt = 0; tt < TPW; ++tt) lam[tt] = lam[tt] + (cv[tt] - lam[tt]);
  }
  __syncthreads();  // halo zeroed
#pragma unroll
  for (int tt = 0; tt < TPW; ++tt) {
    const Px p = px_of(g, t0 + tt, lane);
    if (p.ok) {
      if (!REC) put_px(buf, un[tt], g, p);
      if (MODE == SWEEP_CORRF && k + 1 < Nc) st_px(X + top * slice + eo, lam[tt], g, p);
    }
  }
  if (MODE == SWEEP_FC && k == Nc - 1) row_copy(static_cast<float*>(a.S) + (size_t)Nc * slice + eo, X + top * slice + eo, g.q, nt);
  __syncthreads();

  f32x4 dd[TPW];  // sigma'(z) of the step (after the loop: of the last one)
  // with the record, the words of step j + 1 are requested during step j
  RecW<RB> rn;
  if constexpr (REC) rn = rec_load<RB>(a.dsig, (size_t)(top - 1) * a.stride * a.B + wb.ex, g, t0, lane);
  for (int j = 0; j < nsteps; ++j) {
    // tile offsets recomputed each step (see k_fwd) where that lowers the
    // register count (compiler-measured per variant)
    constexpr bool OPAQUE = REC ? (MODE == SWEEP_FC || MODE == SWEEP_FRES) : MODE != SWEEP_FRES;
    if constexpr (OPAQUE) asm volatile("" : "+v"(lane));
    const long i = top - 1 - j;
    const bool more = j + 1 < nsteps;
    const float* swc = sw + (j & 1) * WV;
    // the correction and serial sweeps stage in one go: their registers are spoken for
    constexpr bool SPLIT = MODE == SWEEP_FC || MODE == SWEEP_FRES;
    float wreg[SPLIT ? WPT : 1];
    if constexpr (SPLIT) stage_fetch<WPT>(wreg, K, bb, (size_t)(more ? i - 1 : i) * a.stride, nt);
    else stage_w(sw + ((j & 1) ^ 1) * WV, K, bb, (size_t)(more ? i - 1 : i) * a.stride, nt);
    // d = sigma'(K u + b)
    if constexpr (REC) {
#pragma unroll
      for (int tt = 0; tt < TPW; ++tt) dd[tt] = rec_val<RB>(rn, tt);
      if (more) rn = rec_load<RB>(a.dsig, (size_t)(i - 1) * a.stride * a.B + wb.ex, g, t0, lane);
    } else {
      float wr[24];
      gather_w<false>(wr, swc, lane);
      const f32x4 bias = bias_px(swc, lane);
      conv_tiles(dd, wr, buf, g, t0, lane, bias);
      act_tiles<true>(dd, a.act);
    }
    float wt[24];
    gather_w<true>(wt, swc, lane);
    // every read of u is done (with the record, the buffer was last read by the
    // previous step's transposed product, which ended with a barrier)
    if (!REC) __syncthreads();
#pragma unroll
    for (int tt = 0; tt < TPW; ++tt) {
      const Px p = px_of(g, t0 + tt, lane);
      if (p.ok) put_px(buf, dd[tt] * lam[tt], g, p);
    }
    __syncthreads();
    // the next step's primal state arrives while the transposed product runs
    if (!REC && more) {
#pragma unroll
      for (int tt = 0; tt < TPW; ++tt) un[tt] = ld_px(Uf + (size_t)(i - 1) * ustep + eo, g, px_of(g, t0 + tt, lane));
    }
    f32x4 w[TPW], gv[HG ? TPW : 1];
    if constexpr (HG) {
#pragma unroll
      for (int tt = 0; tt < TPW; ++tt) gv[tt] = ld_px(G + (size_t)i * slice + eo, g, px_of(g, t0 + tt, lane));
    }
    conv_tiles(w, wt, buf, g, t0, lane, f32x4{0.f, 0.f, 0.f, 0.f});
    const float* gi = !HG && G ? G + (size_t)i * slice + eo : nullptr;
    float* xo = (MODE == SWEEP_CORRF || MODE == MODE_SERIAL) ? X + (size_t)i * slice + eo : nullptr;
#pragma unroll
    for (int tt = 0; tt < TPW; ++tt) {
      const Px p = px_of(g, t0 + tt, lane);
      lam[tt] = lam[tt] + hl * w[tt];
      if constexpr (HG) lam[tt] += gv[tt];
      else if (gi) lam[tt] += ld_px(gi, g, p);
      if (xo && p.ok) st_px(xo, lam[tt], g, p);
    }
    if constexpr (SPLIT) stage_put<WPT>(sw + ((j & 1) ^ 1) * WV, wreg, nt);
    __syncthreads();  // every read of s is done
    if (!REC) {
      if (more) {
#pragma unroll
        for (int tt = 0; tt < TPW; ++tt) {
          const Px p = px_of(g, t0 + tt, lane);
          if (p.ok) put_px(buf, un[tt], g, p);
        }
      }
      __syncthreads();
    }
  }

  if (MODE == SWEEP_FC) {
    float* so = static_cast<float*>(a.S) + (size_t)k * slice + eo;
#pragma unroll
    for (int tt = 0; tt < TPW; ++tt) {
      const Px p = px_of(g, t0 + tt, lane);
      if (p.ok) st_px(so, lam[tt], g, p);
    }
  } else if (MODE == SWEEP_FRES) {
    // coarse adjoint step from the upper C-point, linearised at the fine state of
    // the interval's last step (its weights are in both layer slots); the lower
    // C-point, for the residual, is requested with the upper one (one wait for
    // both) and used before the coarse step's product, so it is not live there
    const float* ck = Cs + (size_t)k * a.cs_stride * slice + eo;
    f32x4 cu[TPW], cl[TPW];
#pragma unroll
    for (int tt = 0; tt < TPW; ++tt) {
      const Px p = px_of(g, t0 + tt, lane);
      cu[tt] = ld_px(src, g, p);
      cl[tt] = ld_px(ck, g, p);
    }
    double acc = 0.0;
#pragma unroll
    for (int tt = 0; tt < TPW; ++tt) {
      const Px p = px_of(g, t0 + tt, lane);
      // with the record, sigma' of the last step comes from its words, still in
      // registers (the loop requests no further step after the last)
      const f32x4 d = REC ? rec_val<RB>(rn, tt) : dd[tt];
      if (p.ok) {
        put_px(buf, d * cu[tt], g, p);
        const f32x4 rr = lam[tt] - cl[tt];
#pragma unroll
        for (int r = 0; r < 4; ++r) acc += (double)rr[r] * (double)rr[r];
      }
    }
    float wt[24];
    gather_w<true>(wt, sw, lane);
    __syncthreads();
    f32x4 w[TPW];
    conv_tiles(w, wt, buf, g, t0, lane, f32x4{0.f, 0.f, 0.f, 0.f});
#pragma unroll
    for (int tt = 0; tt < TPW; ++tt) cu[tt] += hc * w[tt];
    float* gn = static_cast<float*>(a.Gn) + (size_t)k * slice + eo;
#pragma unroll
    for (int tt = 0; tt < TPW; ++tt) {
      const Px p = px_of(g, t0 + tt, lane);
      if (p.ok) st_px(gn, lam[tt] - cu[tt], g, p);  // g_{l+1}^k = f_k - Phibar_{l+1}(C_{k+1})
    }
    if (a.xn_every > 0 && k % a.xn_every == 0) row_copy(static_cast<float*>(a.Xn) + (size_t)k * slice + eo, ck, g.q, nt);
    if (k == Nc - 1)
      row_copy(static_cast<float*>(a.Xn) + (size_t)Nc * slice + eo, Cs + (size_t)Nc * a.cs_stride * slice + eo, g.q, nt);
    if (a.partial) {
      const double s = wg_sum_n(acc, red, g.NW);
      if (threadIdx.x == 0) a.partial[(size_t)k * gridDim.y + wb.ex] = s;
    }
  } else if (MODE == SWEEP_CORRF) {
    if (k == 0) {
      float* xo = X + eo;
      for (int i = threadIdx.x; i < g.q; i += nt) xo[i] = Cs[eo + i] + (Vn[eo + i] - Cs[eo + i]);
    }
  }
}

// ------------------------------------------------------------------ residual
// Workgroup (n, example), with the sweeps' wave and tile layout: forward
// r = Phi_n(U[n]) - U[n+1]; adjoint r = Phibar_n(Lam[n+1]) - Lam[n]; writes the
// example's sum of r^2 (fp64, lanes and waves combined in a fixed order).
template <int DIR>
__global__ __launch_bounds__(64 * MAXW) void k_resid(ResidArgs a, SGeo g) {
  extern __shared__ float lds[];
  float* buf = lds;              // CH * CS: U[n], then (adjoint) s
  float* sw = lds + CH * g.CS;   // the layer's weights
  __shared__ double red[MAXW];
  const int lane = threadIdx.x & 63, t0 = (threadIdx.x >> 6) * TPW, nt = blockDim.x;
  const int n = blockIdx.x;
  const size_t slice = (size_t)a.B * g.q, eo = (size_t)blockIdx.y * g.q;
  const float* U = static_cast<const float*>(a.U);
  const float* Lm = static_cast<const float*>(a.Lam);
  const float h = (float)a.h;
  zero_buf(buf, CH * g.CS, nt);
  stage_w(sw, static_cast<const float*>(a.K), static_cast<const float*>(a.b), n, nt);
  f32x4 un[TPW];
#pragma unroll
  for (int tt = 0; tt < TPW; ++tt) un[tt] = ld_px(U + (size_t)n * slice + eo, g, px_of(g, t0 + tt, lane));
  __syncthreads();  // halo zeroed, weights staged
#pragma unroll
  for (int tt = 0; tt < TPW; ++tt) {
    const Px p = px_of(g, t0 + tt, lane);
    if (p.ok) put_px(buf, un[tt], g, p);
  }
  __syncthreads();
  f32x4 z[TPW];
  {
    float wr[24];
    gather_w<false>(wr, sw, lane);
    conv_tiles(z, wr, buf, g, t0, lane, bias_px(sw, lane));
  }
  double acc = 0.0;
  if (DIR == DIR_FWD) {
    act_tiles<false>(z, a.act);
#pragma unroll
    for (int tt = 0; tt < TPW; ++tt) {
      const Px p = px_of(g, t0 + tt, lane);
      if (!p.ok) continue;
      const f32x4 rr = (un[tt] + h * z[tt]) - ld_px(U + (size_t)(n + 1) * slice + eo, g, p);
#pragma unroll
      for (int r = 0; r < 4; ++r) acc += (double)rr[r] * (double)rr[r];
    }
  } else {
    act_tiles<true>(z, a.act);
    f32x4 lam[TPW];
#pragma unroll
    for (int tt = 0; tt < TPW; ++tt) lam[tt] = ld_px(Lm + (size_t)(n + 1) * slice + eo, g, px_of(g, t0 + tt, lane));
    __syncthreads();  // every read of U[n] is done
#pragma unroll
    for (int tt = 0; tt < TPW; ++tt) {
      const Px p = px_of(g, t0 + tt, lane);
      if (p.ok) put_px(buf, z[tt] * lam[tt], g, p);
    }
    __syncthreads();
    float wt[24];
    gather_w<true>(wt, sw, lane);
    f32x4 w[TPW];
    conv_tiles(w, wt, buf, g, t0, lane, f32x4{0.f, 0.f, 0.f, 0.f});
#pragma unroll
    for (int tt = 0; tt < TPW; ++tt) {
      const Px p = px_of(g, t0 + tt, lane);
      if (!p.ok) continue;
      const f32x4 rr = (lam[tt] + h * w[tt]) - ld_px(Lm + (size_t)n * slice + eo, g, p);
#pragma unroll
      for (int r = 0; r < 4; ++r) acc += (double)rr[r] * (double)rr[r];
    }
  }
  const double s = wg_sum_n(acc, red, g.NW);
  if (threadIdx.x == 0) a.partial[(size_t)blockIdx.x * gridDim.y + blockIdx.y] = s;
}

// ------------------------------------------------------------------ gradient
// Workgroup (layer n, batch chunk), with the sweeps' wave and tile layout. Per
// example: s = sigma'(K u + b) * lam^{n+1} at the lane's own pixels (the
// forward product over the wave's tiles), written to LDS; then
// dWbig[(co,dy)][k] += s[co][2Y+dy][x] * patch[P][k] with the pair-pixels as
// contraction index (k-slice = 4 pair-pixels, lane group = one of them): A = s
// (rows (co,dy)), B = patches of u (96 columns in 6 blocks of 16). db sums s
// from registers. The next example's u (and, with a record, its lambda and
// record word) is loaded during the contraction; with a record its s is written
// to LDS together with its u, so an example takes two barriers instead of three.
// The contraction loop is wave-uniform and reads each slice's operands while the
// previous slice's products run. Waves and lanes are combined in a fixed order.
constexpr int GOUT = 16 * 96 + CH;  // dWbig then db per chunk

template <int GH, int GW, int RK>
__global__ __launch_bounds__(64 * MAXW) void k_grad(GradArgs a, SGeo ga) {
  constexpr bool REC = RK != 0, RB = RK == 1;
  const SGeo g = geo_of<GH, GW>(ga);
  extern __shared__ float lds[];
  float* bu = lds;                   // CH * CS: u
  float* bs = lds + CH * g.CS;       // CH * CS: s
  float* sw = lds + 2 * CH * g.CS;   // the layer's weights
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, t0 = wave * TPW, nt = blockDim.x;
  const int n = blockIdx.x, chunk = blockIdx.y;
  const int per = (a.B + a.nchunks - 1) / a.nchunks;
  const int e0 = chunk * per, e1 = min(a.B, e0 + per);
  const size_t slice = (size_t)a.B * g.q;
  const float* U = static_cast<const float*>(a.U) + (size_t)n * slice;
  const float* Lm = static_cast<const float*>(a.Lam) + (size_t)(n + 1) * slice;

  zero_buf(lds, 2 * CH * g.CS, nt);
  stage_w(sw, static_cast<const float*>(a.K), static_cast<const float*>(a.b), n, nt);
  // B-operand offsets: column k = 16 nb + lane%16 -> (ci, r, tx), relative to the
  // pair-pixel's (row 2Y, col x) origin in padded coordinates
  int koff[6];
#pragma unroll
  for (int nb = 0; nb < 6; ++nb) {
    const int kk = 16 * nb + (lane & 15);
    koff[nb] = (kk / 12) * g.CS + ((kk % 12) / 3) * g.PW + kk % 3;
  }
  f32x4 acc[6];
#pragma unroll
  for (int nb = 0; nb < 6; ++nb) acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  float db0 = 0.f, db1 = 0.f;  // channels 2*(lane/16) and 2*(lane/16)+1
  const int nsl = (g.NPP + 3) / 4;  // pair-pixel slices of 4
  f32x4 un[TPW], lam[TPW];
  RecW<RB> rw;
  if (e0 < e1) {
#pragma unroll
    for (int tt = 0; tt < TPW; ++tt) {
      const Px p = px_of(g, t0 + tt, lane);
      un[tt] = ld_px(U + (size_t)e0 * g.q, g, p);
      if constexpr (REC) lam[tt] = ld_px(Lm + (size_t)e0 * g.q, g, p);
    }
    if constexpr (REC) rw = rec_load<RB>(a.dsig, (size_t)n * a.B + e0, g, t0, lane);
  }
  __syncthreads();  // buffers zeroed, weights staged
  float wf[24];
  gather_w<false>(wf, sw, lane);
  const f32x4 bias = bias_px(sw, lane);
  // s = sigma' * lam at the lane's own pixels into the s image, and into db
  auto put_s = [&](const f32x4 (&z)[TPW]) {
#pragma unroll
    for (int tt = 0; tt < TPW; ++tt) {
      const Px p = px_of(g, t0 + tt, lane);
      if (p.ok) {
        const f32x4 s = z[tt] * lam[tt];
        put_px(bs, s, g, p);
        db0 += s[0] + s[1];
        db1 += s[2] + s[3];
      }
    }
  };
  // matrix-core operands of pair-pixel slice sl: A = s at (co, dy) = lane % 16 of
  // pair-pixel 4 sl + lane / 16, B = its patch entries 16 nb + lane % 16 (zero A
  // past the last pair-pixel, whose address is clamped)
  auto ld_slice = [&](int sl, float& av, float (&bv)[6]) {
    const int P = 4 * sl + (lane >> 4);
    const bool ok = P < g.NPP;
    const int Pc = ok ? P : g.NPP - 1;
    const int Y = Pc / g.W, x = Pc - Y * g.W;
    const int nA = lane & 15, co = nA >> 1, dy = nA & 1;
    av = ok ? bs[co * g.CS + (2 * Y + dy + 1) * g.PW + x + 1] : 0.f;
    const int pb = 2 * Y * g.PW + x;  // (row 2Y-1+r, col x-1+tx) padded = (2Y+r, x+tx)
#pragma unroll
    for (int nb = 0; nb < 6; ++nb) bv[nb] = bu[pb + koff[nb]];
  };
  // with a record, s of an example needs no product, so it is written together
  // with the example's u, before one barrier (two barriers per example, not three)
  auto put_rec_s = [&]() {
    f32x4 z[TPW];
#pragma unroll
    for (int tt = 0; tt < TPW; ++tt) z[tt] = rec_val<RB>(rw, tt);
    put_s(z);
  };
  if (e0 < e1) {
#pragma unroll
    for (int tt = 0; tt < TPW; ++tt) {
      const Px p = px_of(g, t0 + tt, lane);
      if (p.ok) put_px(bu, un[tt], g, p);
    }
    if constexpr (REC) put_rec_s();
  }
  __syncthreads();
  for (int e = e0; e < e1; ++e) {
    const bool more = e + 1 < e1;
    if constexpr (!REC) {
      f32x4 z[TPW];
#pragma unroll
      for (int tt = 0; tt < TPW; ++tt) lam[tt] = ld_px(Lm + (size_t)e * g.q, g, px_of(g, t0 + tt, lane));
      conv_tiles(z, wf, bu, g, t0, lane, bias);
      act_tiles<true>(z, a.act);
      put_s(z);
      __syncthreads();
    }
    // the next example's primal state, adjoint and record arrive while the
    // contraction runs
    if (more) {
#pragma unroll
      for (int tt = 0; tt < TPW; ++tt) {
        const Px p = px_of(g, t0 + tt, lane);
        un[tt] = ld_px(U + (size_t)(e + 1) * g.q, g, p);
        if constexpr (REC) lam[tt] = ld_px(Lm + (size_t)(e + 1) * g.q, g, p);
      }
      if constexpr (REC) rw = rec_load<RB>(a.dsig, (size_t)n * a.B + e + 1, g, t0, lane);
    }
    // contraction over pair-pixels, wave-uniform and pipelined: a slice's operands
    // are read from LDS while the previous slice's products run (a slice past the
    // end reads in bounds and contributes zero)
    {
      const int wv = __builtin_amdgcn_readfirstlane(wave);
      float av, bv[6];
      ld_slice(wv, av, bv);
      for (int sl = wv; sl < nsl; sl += g.NW) {
        float an, bn[6];
        ld_slice(sl + g.NW, an, bn);
#pragma unroll
        for (int nb = 0; nb < 6; ++nb) acc[nb] = __builtin_amdgcn_mfma_f32_16x16x4f32(av, bv[nb], acc[nb], 0, 0, 0);
        av = an;
#pragma unroll
        for (int nb = 0; nb < 6; ++nb) bv[nb] = bn[nb];
      }
    }
    __syncthreads();
    if (more) {
#pragma unroll
      for (int tt = 0; tt < TPW; ++tt) {
        const Px p = px_of(g, t0 + tt, lane);
        if (p.ok) put_px(bu, un[tt], g, p);
      }
      if constexpr (REC) put_rec_s();
    }
    __syncthreads();
  }
  // combine waves in order (the image buffers are free now):
  // D[(co,dy) = 4(lane/16)+r][k = 16 nb + lane%16]
  float* red = lds;               // GOUT
  float* dbp = lds + GOUT;        // two per thread
  for (int w = 0; w < g.NW; ++w) {
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
  dbp[2 * threadIdx.x] = db0;
  dbp[2 * threadIdx.x + 1] = db1;
  __syncthreads();
  // db per channel: its 16 lanes of every wave, in thread order
  if (threadIdx.x < CH) {
    const int ch = threadIdx.x, grp = ch >> 1;
    float s = 0.f;
    for (int w = 0; w < g.NW; ++w)
      for (int l = 0; l < 16; ++l) s += dbp[2 * (64 * w + 16 * grp + l) + (ch & 1)];
    red[16 * 96 + ch] = s;
  }
  __syncthreads();
  float* out = static_cast<float*>(a.partial) + ((size_t)n * a.nchunks + chunk) * GOUT;
  for (int o = threadIdx.x; o < GOUT; o += nt) out[o] = red[o];
}

// dK[n][co][ci][ty][tx] = h sum_chunks sum_dy dWbig[(co,dy)][(ci, ty+dy, tx)], db[n][co] = h sum db.
__global__ __launch_bounds__(NT) void k_grad_final(GradArgs a) {
  const size_t o = (size_t)blockIdx.x * NT + threadIdx.x;
  if (o >= (size_t)a.N * (KW + CH)) return;
  const size_t n = o / (KW + CH);
  const int r = (int)(o - n * (KW + CH));
  const float* p = static_cast<const float*>(a.partial) + n * a.nchunks * GOUT;
  double s = 0.0;  // chunk partials summed in fp64
  if (r < KW) {
    const int co = r / 72, ci = (r % 72) / 9, ty = (r % 9) / 3, tx = r % 3;
    for (int ch = 0; ch < a.nchunks; ++ch)
      for (int dy = 0; dy < 2; ++dy) {
        const int kk = ci * 12 + (ty + dy) * 3 + tx;
        s += (double)p[(size_t)ch * GOUT + (2 * co + dy) * 96 + kk];
      }
    static_cast<float*>(a.dK)[n * KW + r] = (float)(s * a.h);
  } else {
    for (int ch = 0; ch < a.nchunks; ++ch) s += (double)p[(size_t)ch * GOUT + 16 * 96 + (r - KW)];
    static_cast<float*>(a.db)[n * CH + (r - KW)] = (float)(s * a.h);
  }
}

}  // namespace conv

namespace {

conv::SGeo sweep_geo(const Shape& s) { return conv::make_geo(s.H, s.W); }

size_t sweep_lds(const conv::SGeo& g) { return (size_t)(conv::CH * g.CS + 2 * conv::WV) * sizeof(float); }

// Sweep kernels with the geometry as template arguments (0, 0: runtime).
// Only the forward CORRF and serial kernels write the record; every adjoint
// kernel can read it.
template <int GH, int GW, int RK, bool HG>
void sweep_kernels(int dir, int mode, void (*&f)(SweepArgs, conv::SGeo)) {
  using namespace conv;
  if (dir == DIR_FWD) {
    if (mode == SWEEP_FC) f = k_fwd<SWEEP_FC, GH, GW, 0, HG>;
    else if (mode == SWEEP_FRES) f = k_fwd<SWEEP_FRES, GH, GW, 0, HG>;
    else if (mode == SWEEP_CORRF) f = k_fwd<SWEEP_CORRF, GH, GW, RK, HG>;
    else f = k_fwd<MODE_SERIAL, GH, GW, RK, HG>;
  } else {
    if (mode == SWEEP_FC) f = k_adj<SWEEP_FC, GH, GW, RK, HG>;
    else if (mode == SWEEP_FRES) f = k_adj<SWEEP_FRES, GH, GW, RK, HG>;
    else if (mode == SWEEP_CORRF) f = k_adj<SWEEP_CORRF, GH, GW, RK, HG>;
    else f = k_adj<MODE_SERIAL, GH, GW, RK, HG>;
  }
}

hipError_t launch_conv_sweep(const Shape& s, int dir, const SweepArgs& a, dim3 grid, hipStream_t st) {
  const conv::SGeo g = sweep_geo(s);
  void (*f)(SweepArgs, conv::SGeo) = nullptr;
  const int rk = a.dsig == nullptr ? 0 : a.act == ACT_RELU ? 1 : 2;
  const bool hg = a.G != nullptr;
  if (s.H == 28 && s.W == 28) {  // MNIST-sized images
    if (hg) {
      if (rk == 1) sweep_kernels<28, 28, 1, true>(dir, a.mode, f);
      else if (rk == 2) sweep_kernels<28, 28, 2, true>(dir, a.mode, f);
      else sweep_kernels<28, 28, 0, true>(dir, a.mode, f);
    } else {
      if (rk == 1) sweep_kernels<28, 28, 1, false>(dir, a.mode, f);
      else if (rk == 2) sweep_kernels<28, 28, 2, false>(dir, a.mode, f);
      else sweep_kernels<28, 28, 0, false>(dir, a.mode, f);
    }
  } else {
    if (hg) {
      if (rk == 1) sweep_kernels<0, 0, 1, true>(dir, a.mode, f);
      else if (rk == 2) sweep_kernels<0, 0, 2, true>(dir, a.mode, f);
      else sweep_kernels<0, 0, 0, true>(dir, a.mode, f);
    } else {
      if (rk == 1) sweep_kernels<0, 0, 1, false>(dir, a.mode, f);
      else if (rk == 2) sweep_kernels<0, 0, 2, false>(dir, a.mode, f);
      else sweep_kernels<0, 0, 0, false>(dir, a.mode, f);
    }
  }
  launch(f, grid, dim3(64 * g.NW), sweep_lds(g), st, a, g);
  return hipGetLastError();
}

}  // namespace

// fp32, C = 8, even H; at most MAXW waves of TPW tiles, and the gradient's two
// image buffers within 64 KB of LDS (H, W up to 30 x 30)
bool conv_supported(const Shape& s) {
  if (s.layer != 1 || s.dtype != 0 || s.C != conv::CH || s.H < 2 || s.H % 2 || s.W < 1 || s.H > 4096 || s.W > 4096)
    return false;
  const conv::SGeo g = sweep_geo(s);
  return g.NT16 <= conv::MAXW * conv::TPW && (2 * conv::CH * g.CS + conv::WV) * sizeof(float) <= 65536;
}

int conv_tile(const Shape&) { return 1; }

size_t conv_dsig_block_bytes(const Shape& s) { return conv::rec_block_bytes(sweep_geo(s), s.act == ACT_RELU); }

// Enough workgroups to fill the chip when N is small, and at most GRAD_EX
// examples per chunk: a partial sums GRAD_EX x 784 pixels x 4 terms per matrix-core
// accumulator in fp32, and the chunks are summed in fp64, which keeps the
// gradient's rounding error near 1e-6 relative at any batch size.
constexpr int GRAD_EX = 32;
int conv_grad_chunks(int B, int N) {
  int ch = (2048 + N - 1) / N;
  ch = std::max(ch, (B + GRAD_EX - 1) / GRAD_EX);
  ch = std::min(ch, B);
  return ch < 1 ? 1 : ch;
}

hipError_t conv_sweep(const Shape& s, int dir, const SweepArgs& a, hipStream_t st, int* partials) {
  const dim3 grid(a.Nl / a.c, a.B);
  if (partials) *partials = (int)(grid.x * grid.y);
  return launch_conv_sweep(s, dir, a, grid, st);
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
  a.dsig = sa.dsig;
  return launch_conv_sweep(s, dir, a, dim3(1, sa.B), st);
}

hipError_t conv_resid(const Shape& s, int dir, const ResidArgs& a, hipStream_t st, int* partials) {
  const dim3 grid(a.N, a.B);
  if (partials) *partials = (int)(grid.x * grid.y);
  const conv::SGeo g = sweep_geo(s);
  if (dir == DIR_FWD) launch(conv::k_resid<DIR_FWD>, grid, dim3(64 * g.NW), sweep_lds(g), st, a, g);
  else launch(conv::k_resid<DIR_ADJ>, grid, dim3(64 * g.NW), sweep_lds(g), st, a, g);
  return hipGetLastError();
}

hipError_t conv_grad(const Shape& s, const GradArgs& a, hipStream_t st) {
  const conv::SGeo g = sweep_geo(s);
  // image buffers and weights, reused at the end for the partial and the db terms
  const int fl = 2 * conv::CH * g.CS + conv::WV, red = conv::GOUT + 2 * 64 * g.NW;
  const size_t sh = (size_t)(fl > red ? fl : red) * sizeof(float);
  void (*f)(GradArgs, conv::SGeo);
  const int rk = a.dsig == nullptr ? 0 : a.act == ACT_RELU ? 1 : 2;
  if (s.H == 28 && s.W == 28)
    f = rk == 1 ? conv::k_grad<28, 28, 1> : rk == 2 ? conv::k_grad<28, 28, 2> : conv::k_grad<28, 28, 0>;
  else f = rk == 1 ? conv::k_grad<0, 0, 1> : rk == 2 ? conv::k_grad<0, 0, 2> : conv::k_grad<0, 0, 0>;
  launch(f, dim3(a.N, a.nchunks), 64 * g.NW, sh, st, a, g);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  const size_t tot = (size_t)a.N * (conv::KW + conv::CH);
  launch(conv::k_grad_final, (unsigned)((tot + conv::NT - 1) / conv::NT), conv::NT, 0, st, a);
  return hipGetLastError();
}

}  // namespace lp
