// Device helpers shared by the HIP kernels of the layer-parallel ResNet library:
// activations sigma and sigma' (Section 2.1 and the smoothed ReLU of Section 5.1),
// vectorised row access, and fixed-order workgroup reductions.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lp {

enum Act { ACT_TANH = 0, ACT_RELU = 1, ACT_SMOOTHRELU = 2, ACT_IDENTITY = 3 };

// tanh: the device library's accurate tanh. sigma'(z) = 1 - tanh(z)^2.
__device__ __forceinline__ float dev_tanh(float z) { return tanhf(z); }
__device__ __forceinline__ double dev_tanh(double z) { return tanh(z); }

template <typename T, int ACT>
__device__ __forceinline__ T act_f(T z) {
  if constexpr (ACT == ACT_TANH) {
    return dev_tanh(z);
  } else if constexpr (ACT == ACT_RELU) {
    return z > T(0) ? z : T(0);
  } else if constexpr (ACT == ACT_SMOOTHRELU) {
    // max(z,0) for |z| > 0.1; 2.5 z^2 + 0.5 z + 0.025 on |z| <= 0.1 (C^1 at +-0.1)
    T a = z < T(0) ? -z : z;
    if (a <= T(0.1)) return (T(2.5) * z + T(0.5)) * z + T(0.025);
    return z > T(0) ? z : T(0);
  } else {
    return z;
  }
}

template <typename T, int ACT>
__device__ __forceinline__ T dact_f(T z) {
  if constexpr (ACT == ACT_TANH) {
    T t = dev_tanh(z);
    return T(1) - t * t;
  } else if constexpr (ACT == ACT_RELU) {
    return z > T(0) ? T(1) : T(0);  // sigma'(0) = 0
  } else if constexpr (ACT == ACT_SMOOTHRELU) {
    T a = z < T(0) ? -z : z;
    if (a <= T(0.1)) return T(5) * z + T(0.5);
    return z > T(0) ? T(1) : T(0);
  } else {
    return T(1);
  }
}

// Vector type holding 16 bytes of T.
template <typename T> struct Vec16;
template <> struct Vec16<float> { using type = float4; static constexpr int n = 4; };
template <> struct Vec16<double> { using type = double2; static constexpr int n = 2; };

// Load / store Q consecutive elements (Q * sizeof(T) must be a multiple of 16 and
// the address 16-byte aligned: rows of a [.][B][Q] array with Q*sizeof(T) % 16 == 0).
template <typename T, int Q>
__device__ __forceinline__ void load_row(T (&r)[Q], const T* __restrict__ p) {
  using V = typename Vec16<T>::type;
  constexpr int n = Vec16<T>::n;
  static_assert(Q % n == 0, "row width must fill 16-byte vectors");
  const V* pv = reinterpret_cast<const V*>(p);
#pragma unroll
  for (int i = 0; i < Q / n; ++i) {
    V x = pv[i];
    if constexpr (n == 4) {
      r[4 * i + 0] = x.x; r[4 * i + 1] = x.y; r[4 * i + 2] = x.z; r[4 * i + 3] = x.w;
    } else {
      r[2 * i + 0] = x.x; r[2 * i + 1] = x.y;
    }
  }
}

template <typename T, int Q>
__device__ __forceinline__ void store_row(T* __restrict__ p, const T (&r)[Q]) {
  using V = typename Vec16<T>::type;
  constexpr int n = Vec16<T>::n;
  V* pv = reinterpret_cast<V*>(p);
#pragma unroll
  for (int i = 0; i < Q / n; ++i) {
    V x;
    if constexpr (n == 4) {
      x.x = r[4 * i + 0]; x.y = r[4 * i + 1]; x.z = r[4 * i + 2]; x.w = r[4 * i + 3];
    } else {
      x.x = r[2 * i + 0]; x.y = r[2 * i + 1];
    }
    pv[i] = x;
  }
}

// Fixed-order sum of one double per thread over a workgroup of NT threads
// (NT a power of two <= 1024). Every thread must call it. Result valid in thread 0.
template <int NT>
__device__ __forceinline__ double block_sum(double v, double* sh) {
  sh[threadIdx.x] = v;
  __syncthreads();
#pragma unroll
  for (int s = NT / 2; s > 0; s >>= 1) {
    if ((int)threadIdx.x < s) sh[threadIdx.x] += sh[threadIdx.x + s];
    __syncthreads();
  }
  double r = sh[0];
  __syncthreads();
  return r;
}

}  // namespace lp
