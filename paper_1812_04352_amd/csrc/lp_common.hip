// Kernels shared by every layer family: row copies (the MGRIT cold start), the
// fixed-order residual-norm reduction, and the boundary helpers of the network
// (opening layer and its gradient, the plain gradient step). The helpers sit
// outside the per-iteration hot path. The loss helper lives in lp_loss.hip.
#include <math.h>

#include <algorithm>
#include <type_traits>

#include "lp_device.h"
#include "lp_internal.h"

namespace lp {
namespace {

constexpr int NT = 256;

// X[dst_row0 + t*dst_step] = X[src_row] for t = 0..count-1 (16-byte units; the
// source row is not among the destinations). Workgroup row blockIdx.y takes
// destination rows rows * blockIdx.y .. + rows - 1: each thread reads its units
// of the source row once and writes them to those rows.
__global__ __launch_bounds__(NT) void k_copy_rows(uint4* X, size_t units, long src_row,
                                                  long dst_row0, long dst_step, long count, long rows) {
  const long t0 = (long)blockIdx.y * rows, t1 = min(count, t0 + rows);
  for (size_t u = (size_t)blockIdx.x * NT + threadIdx.x; u < units; u += (size_t)gridDim.x * NT) {
    const uint4 v = X[(size_t)src_row * units + u];
    for (long t = t0; t < t1; ++t) X[(size_t)(dst_row0 + t * dst_step) * units + u] = v;
  }
}

// Sticky per-device record of a non-finite residual norm (any MGRIT solve or
// residual-norm call on this device since the flag was last cleared). Set by the
// reduction below with an ordinary global store; read and cleared by
// lp_check_finite.
__device__ uint32_t g_nonfinite = 0u;

// out[0] = sqrt(sum of partial[0..n)), summed in a fixed order: thread t adds
// partial[t], partial[t + NTR], ... in index order (eight loads issued at a time,
// so the serial chain waits once per eight), then the workgroup tree.
constexpr int NTR = 1024;
__global__ __launch_bounds__(NTR) void k_norm_reduce(const double* partial, int n, double* out) {
  __shared__ double sh[NTR];
  double s = 0.0;
  int i = threadIdx.x;
  for (; i + 7 * NTR < n; i += 8 * NTR) {
    double v[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) v[k] = partial[i + k * NTR];
#pragma unroll
    for (int k = 0; k < 8; ++k) s += v[k];
  }
  for (; i < n; i += NTR) s += partial[i];
  s = block_sum<NTR>(s, sh);
  if (threadIdx.x == 0) {
    const double r = sqrt(s);
    out[0] = r;
    if (!isfinite(r)) g_nonfinite = 1u;
  }
}

// dst[i] = src[i] over 16-byte units.
__global__ __launch_bounds__(NT) void k_copy16(uint4* dst, const uint4* src, size_t units) {
  for (size_t i = (size_t)blockIdx.x * NT + threadIdx.x; i < units; i += (size_t)gridDim.x * NT) dst[i] = src[i];
}

__global__ __launch_bounds__(NT) void k_zero(uint32_t* p, size_t n) {
  for (size_t i = (size_t)blockIdx.x * NT + threadIdx.x; i < n; i += (size_t)gridDim.x * NT) p[i] = 0u;
}

unsigned grid_for(size_t work) {
  size_t g = (work + NT - 1) / NT;
  if (g > 65535u * 8u) g = 65535u * 8u;
  return (unsigned)(g ? g : 1);
}

// ---------------------------------------------------------------- opening layer

template <typename T, int ACT>
__global__ __launch_bounds__(NT) void k_open_dense(const T* y, const T* L, T* u0, int B, int q, int nf) {
  const size_t tot = (size_t)B * q;
  for (size_t i = (size_t)blockIdx.x * NT + threadIdx.x; i < tot; i += (size_t)gridDim.x * NT) {
    const size_t e = i / q, r = i - e * q;
    T acc = T(0);
    for (int f = 0; f < nf; ++f) acc = fma(L[r * nf + f], y[e * nf + f], acc);
    u0[i] = act_f<T, ACT>(acc);
  }
}

// u0[e][co][y][x] = sigma(sum_{ty,tx} L[co][0][ty][tx] y[e][0][y+ty-1][x+tx-1]), zero padded.
template <typename T, int ACT>
__global__ __launch_bounds__(NT) void k_open_conv(const T* y, const T* L, T* u0, int B, int C, int H, int W) {
  const size_t tot = (size_t)B * C * H * W;
  for (size_t i = (size_t)blockIdx.x * NT + threadIdx.x; i < tot; i += (size_t)gridDim.x * NT) {
    size_t t = i;
    const int x = (int)(t % W); t /= W;
    const int yy = (int)(t % H); t /= H;
    const int co = (int)(t % C);
    const size_t e = t / C;
    T acc = T(0);
    for (int ty = 0; ty < 3; ++ty) {
      const int sy = yy + ty - 1;
      if (sy < 0 || sy >= H) continue;
      for (int tx = 0; tx < 3; ++tx) {
        const int sx = x + tx - 1;
        if (sx < 0 || sx >= W) continue;
        acc = fma(L[co * 9 + ty * 3 + tx], y[e * H * W + (size_t)sy * W + sx], acc);
      }
    }
    u0[i] = act_f<T, ACT>(acc);
  }
}

// dL[r][f] = sum_e sigma'(z_er) lam0[e][r] y[e][f]; one workgroup per row r,
// examples in order, z recomputed once per (e, r).
template <typename T, int ACT>
__global__ __launch_bounds__(NT) void k_open_grad_dense(const T* y, const T* L, const T* lam0, T* dL,
                                                        int B, int q, int nf) {
  __shared__ T sv[NT];
  const int r = blockIdx.x;
  // each thread owns features f = threadIdx.x + k*NT
  T acc[4] = {T(0), T(0), T(0), T(0)};  // nf <= 4*NT
  for (int e0 = 0; e0 < B; e0 += NT) {
    const int e = e0 + threadIdx.x;
    T s = T(0);
    if (e < B) {
      T z = T(0);
      for (int f = 0; f < nf; ++f) z = fma(L[(size_t)r * nf + f], y[(size_t)e * nf + f], z);
      s = dact_f<T, ACT>(z) * lam0[(size_t)e * q + r];
    }
    sv[threadIdx.x] = s;
    __syncthreads();
    const int ne = min(NT, B - e0);
    for (int k = 0; k < 4; ++k) {
      const int f = threadIdx.x + k * NT;
      if (f < nf)
        for (int t = 0; t < ne; ++t) acc[k] = fma(sv[t], y[(size_t)(e0 + t) * nf + f], acc[k]);
    }
    __syncthreads();
  }
  for (int k = 0; k < 4; ++k) {
    const int f = threadIdx.x + k * NT;
    if (f < nf) dL[(size_t)r * nf + f] = acc[k];
  }
}

// dL[co][0][ty][tx] = sum_e sum_p sigma'(z[e,co,p]) lam0[e,co,p] y[e, p + t]: one
// workgroup per output channel; thread t accumulates over pixels t, t+NT, ... of
// every example for all 9 taps, then a fixed-order tree combines the threads.
template <typename T, int ACT>
__global__ __launch_bounds__(NT) void k_open_grad_conv(const T* y, const T* L, const T* lam0, T* dL,
                                                       int B, int C, int H, int W) {
  __shared__ double sh[NT];
  const int co = blockIdx.x;
  T acc[9];
  for (int t = 0; t < 9; ++t) acc[t] = T(0);
  const int P = H * W;
  for (int e = 0; e < B; ++e) {
    const T* ye = y + (size_t)e * P;
    for (int p = threadIdx.x; p < P; p += NT) {
      const int yy = p / W, x = p - yy * W;
      T win[9];
      T z = T(0);
      for (int ty = 0; ty < 3; ++ty)
        for (int tx = 0; tx < 3; ++tx) {
          const int sy = yy + ty - 1, sx = x + tx - 1;
          T v = (sy >= 0 && sy < H && sx >= 0 && sx < W) ? ye[sy * W + sx] : T(0);
          win[ty * 3 + tx] = v;
          z = fma(L[co * 9 + ty * 3 + tx], v, z);
        }
      const T s = dact_f<T, ACT>(z) * lam0[((size_t)e * C + co) * P + p];
      for (int t = 0; t < 9; ++t) acc[t] = fma(s, win[t], acc[t]);
    }
  }
  for (int t = 0; t < 9; ++t) {
    double v = block_sum<NT>((double)acc[t], sh);
    if (threadIdx.x == 0) dL[co * 9 + t] = (T)v;
  }
}

template <typename T>
__global__ __launch_bounds__(NT) void k_sgd(size_t n, T lr, const T* g, T* x) {
  for (size_t i = (size_t)blockIdx.x * NT + threadIdx.x; i < n; i += (size_t)gridDim.x * NT)
    x[i] = x[i] - lr * g[i];
}

template <typename T, typename F>
hipError_t with_act(int act, F&& f) {
  switch (act) {
    case ACT_TANH: return f(std::integral_constant<int, ACT_TANH>{});
    case ACT_RELU: return f(std::integral_constant<int, ACT_RELU>{});
    case ACT_SMOOTHRELU: return f(std::integral_constant<int, ACT_SMOOTHRELU>{});
    case ACT_IDENTITY: return f(std::integral_constant<int, ACT_IDENTITY>{});
  }
  return hipErrorNotSupported;
}

template <typename T>
hipError_t open_fwd_t(const Shape& s, int opening, int nf, int B, const void* y, const void* L, void* u0,
                      hipStream_t st) {
  const int q = s.C * s.H * s.W;
  if (opening == 0) {
    const size_t bytes = (size_t)B * q * sizeof(T);
    if (bytes % 16 || (uintptr_t)u0 % 16 || (uintptr_t)y % 16)
      return hipMemcpyAsync(u0, y, bytes, hipMemcpyDeviceToDevice, st);
    k_copy16<<<grid_for(bytes / 16), NT, 0, st>>>(static_cast<uint4*>(u0), static_cast<const uint4*>(y), bytes / 16);
    return hipGetLastError();
  }
  return with_act<T>(s.act, [&](auto ac) -> hipError_t {
    constexpr int ACT = decltype(ac)::value;
    if (opening == 1)
      k_open_dense<T, ACT><<<grid_for((size_t)B * q), NT, 0, st>>>((const T*)y, (const T*)L, (T*)u0, B, q, nf);
    else
      k_open_conv<T, ACT><<<grid_for((size_t)B * q), NT, 0, st>>>((const T*)y, (const T*)L, (T*)u0, B, s.C,
                                                                  s.H, s.W);
    return hipGetLastError();
  });
}

template <typename T>
hipError_t open_grad_t(const Shape& s, int opening, int nf, int B, const void* y, const void* L,
                       const void* lam0, void* dL, hipStream_t st) {
  const int q = s.C * s.H * s.W;
  return with_act<T>(s.act, [&](auto ac) -> hipError_t {
    constexpr int ACT = decltype(ac)::value;
    if (opening == 1)
      k_open_grad_dense<T, ACT><<<q, NT, 0, st>>>((const T*)y, (const T*)L, (const T*)lam0, (T*)dL, B, q, nf);
    else
      k_open_grad_conv<T, ACT><<<s.C, NT, 0, st>>>((const T*)y, (const T*)L, (const T*)lam0, (T*)dL, B, s.C,
                                                   s.H, s.W);
    return hipGetLastError();
  });
}

}  // namespace

hipError_t launch_copy_rows(void* X, size_t slice_bytes, long src_row, long dst_row0, long dst_step,
                            long count, hipStream_t st) {
  if (count <= 0 || slice_bytes == 0) return hipSuccess;
  const size_t units = slice_bytes / 16;
  // about 8192 workgroups: the rows are split into groups when one row's
  // workgroups are fewer
  const unsigned gx = grid_for(units);
  const long want = std::max<long>(1, std::min<long>(count, (8192 + gx - 1) / gx));
  const long rows = (count + want - 1) / want, groups = (count + rows - 1) / rows;
  if (groups > 65535) return hipErrorInvalidValue;  // the grid's y dimension
  k_copy_rows<<<dim3(gx, (unsigned)groups), NT, 0, st>>>(static_cast<uint4*>(X), units, src_row, dst_row0,
                                                         dst_step, count, rows);
  return hipGetLastError();
}

hipError_t launch_norm_reduce(const double* partial, int n, double* out, hipStream_t st) {
  k_norm_reduce<<<1, NTR, 0, st>>>(partial, n, out);
  return hipGetLastError();
}

hipError_t read_nonfinite(uint32_t* flag, bool clear, hipStream_t st) {
  hipError_t e = hipMemcpyFromSymbolAsync(flag, HIP_SYMBOL(g_nonfinite), sizeof(uint32_t), 0,
                                          hipMemcpyDeviceToHost, st);
  if (e != hipSuccess) return e;
  e = hipStreamSynchronize(st);
  if (e != hipSuccess || !clear || *flag == 0u) return e;
  const uint32_t zero = 0u;
  e = hipMemcpyToSymbolAsync(HIP_SYMBOL(g_nonfinite), &zero, sizeof(uint32_t), 0, hipMemcpyHostToDevice, st);
  if (e != hipSuccess) return e;
  return hipStreamSynchronize(st);
}

hipError_t launch_zero(void* p, size_t bytes, hipStream_t st) {
  if (bytes == 0) return hipSuccess;
  k_zero<<<grid_for(bytes / 4), NT, 0, st>>>(static_cast<uint32_t*>(p), bytes / 4);
  return hipGetLastError();
}

hipError_t launch_open_forward(const Shape& s, int opening, int nf, int B, const void* y, const void* L,
                               void* u0, hipStream_t st) {
  return s.dtype == 0 ? open_fwd_t<float>(s, opening, nf, B, y, L, u0, st)
                      : open_fwd_t<double>(s, opening, nf, B, y, L, u0, st);
}

hipError_t launch_open_grad(const Shape& s, int opening, int nf, int B, const void* y, const void* L,
                            const void* lam0, void* dL, hipStream_t st) {
  return s.dtype == 0 ? open_grad_t<float>(s, opening, nf, B, y, L, lam0, dL, st)
                      : open_grad_t<double>(s, opening, nf, B, y, L, lam0, dL, st);
}

// y <- a x + b y (b == 0: y <- a x, whatever y held)
template <typename T>
__global__ __launch_bounds__(NT) void k_axpby(size_t n, double a, const T* x, double b, T* y) {
  for (size_t i = (size_t)blockIdx.x * NT + threadIdx.x; i < n; i += (size_t)gridDim.x * NT)
    y[i] = b == 0.0 ? (T)(a * (double)x[i]) : (T)(a * (double)x[i] + b * (double)y[i]);
}

// Dot product in fp64 and in a fixed order: workgroup w sums the elements
// w NT + t (+ k DOT_BLOCKS NT) per thread, then its threads in a fixed tree; the
// second pass adds the DOT_BLOCKS partials in order.
template <typename T>
__global__ __launch_bounds__(NT) void k_dot_part(size_t n, const T* x, const T* y, double* part) {
  __shared__ double sh[NT];
  double s = 0.0;
  for (size_t i = (size_t)blockIdx.x * NT + threadIdx.x; i < n; i += (size_t)DOT_BLOCKS * NT)
    s += (double)x[i] * (double)y[i];
  s = block_sum<NT>(s, sh);
  if (threadIdx.x == 0) part[blockIdx.x] = s;
}

__global__ __launch_bounds__(64) void k_dot_final(const double* part, double* out) {
  if (threadIdx.x != 0) return;
  double s = 0.0;
  for (int w = 0; w < DOT_BLOCKS; ++w) s += part[w];
  out[0] = s;
}

hipError_t launch_axpby(int dtype, size_t n, double a, const void* x, double b, void* y, hipStream_t st) {
  if (n == 0) return hipSuccess;
  if (dtype == 0) k_axpby<float><<<grid_for(n), NT, 0, st>>>(n, a, (const float*)x, b, (float*)y);
  else k_axpby<double><<<grid_for(n), NT, 0, st>>>(n, a, (const double*)x, b, (double*)y);
  return hipGetLastError();
}

hipError_t launch_dot(int dtype, size_t n, const void* x, const void* y, double* out, hipStream_t st) {
  if (dtype == 0) k_dot_part<float><<<DOT_BLOCKS, NT, 0, st>>>(n, (const float*)x, (const float*)y, out + 1);
  else k_dot_part<double><<<DOT_BLOCKS, NT, 0, st>>>(n, (const double*)x, (const double*)y, out + 1);
  k_dot_final<<<1, 64, 0, st>>>(out + 1, out);
  return hipGetLastError();
}

hipError_t launch_sgd(int dtype, size_t n, double lr, const void* g, void* x, hipStream_t st) {
  if (n == 0) return hipSuccess;
  if (dtype == 0) k_sgd<float><<<grid_for(n), NT, 0, st>>>(n, (float)lr, (const float*)g, (float*)x);
  else k_sgd<double><<<grid_for(n), NT, 0, st>>>(n, lr, (const double*)g, (double*)x);
  return hipGetLastError();
}

}  // namespace lp
