// Softmax hypothesis and cross-entropy loss at the network output, and the
// adjoint terminal value (Section 2.1, the softmax and loss equations; the
// terminal condition of the adjoint equations in Section 2.3):
//   z_k = W u_k^N + mu,  S_k = softmax(z_k),  J = (1/B) sum_k -c_k^T log S_k,
//   d_k = (S_k - c_k) / B,  lam_k^N = W^T d_k,  dW = sum_k d_k (u_k^N)^T,  dmu = sum_k d_k.
// A boundary helper outside the per-iteration hot path; all reductions run in a
// fixed order. Workspace: logits/residuals d [B][nc] (fp64), per-example losses
// [B] (fp64), and per-chunk partials of dW and dmu [nchunks][nc][q+1] (fp64).
#include <math.h>

#include "lp_device.h"
#include "lp_internal.h"

namespace lp {
namespace {

constexpr int NT = 256;
constexpr int CHUNK = 32;  // examples per partial of dW, dmu (short chains, many workgroups)

// Head of the network, one segment of S lanes per example (S = the power of two
// >= nc; lane j of the segment owns class j): the logits z_j = mu_j + W_j . u
// (each lane sums the features i = j mod S, the segment adds the partials),
// the softmax and loss_e with segment reductions, d_j = (S_j - c_j)/B, and
// lam^N = W^T d (each lane takes features i = j mod S). All sums run in fp64 and
// in a fixed order.
template <typename T>
__global__ __launch_bounds__(NT) void k_head(const T* uN, const T* Wc, const T* mu, const T* c, double* d,
                                             double* loss, T* lamN, int B, int q, int nc, int S) {
  __shared__ double dsh[NT];
  const int t = threadIdx.x, j = t & (S - 1), seg = t - j;
  const int e = blockIdx.x * (NT / S) + t / S;
  const bool on = e < B;  // uniform over a segment
  const T* u = uN + (size_t)(on ? e : B - 1) * q;
  double zj = -INFINITY;
  for (int jj = 0; jj < nc; ++jj) {
    double p = 0.0;
    for (int i = j; i < q; i += S) p += (double)Wc[(size_t)jj * q + i] * (double)u[i];
    for (int off = S / 2; off > 0; off >>= 1) p += __shfl_xor(p, off, 64);
    if (j == jj) zj = p + (double)mu[jj];
  }
  double m = zj;
  for (int off = S / 2; off > 0; off >>= 1) m = fmax(m, __shfl_xor(m, off, 64));
  const bool cls = j < nc;
  double den = cls ? exp(zj - m) : 0.0;
  for (int off = S / 2; off > 0; off >>= 1) den += __shfl_xor(den, off, 64);
  const double lden = log(den);
  const double cj = cls && on ? (double)c[(size_t)e * nc + j] : 0.0;
  const double logp = cls ? (zj - m) - lden : 0.0;
  double l = cls ? -cj * logp : 0.0;
  for (int off = S / 2; off > 0; off >>= 1) l += __shfl_xor(l, off, 64);
  const double dj = cls ? (exp(logp) - cj) / (double)B : 0.0;
  if (on) {
    if (cls) d[(size_t)e * nc + j] = dj;
    if (j == 0) loss[e] = l;
  }
  dsh[t] = dj;
  __syncthreads();
  if (!on) return;
  for (int i = j; i < q; i += S) {
    double acc = 0.0;
    for (int jj = 0; jj < nc; ++jj) acc += (double)Wc[(size_t)jj * q + i] * dsh[seg + jj];
    lamN[(size_t)e * q + i] = (T)acc;
  }
}

// J = (1/B) sum_e loss_e, summed in a fixed order by one workgroup.
constexpr int NT_MEAN = 1024;
__global__ __launch_bounds__(NT_MEAN) void k_mean(const double* loss, int B, double* J) {
  __shared__ double sh[NT_MEAN];
  double s = 0.0;
  for (int e = threadIdx.x; e < B; e += NT_MEAN) s += loss[e];
  s = block_sum<NT_MEAN>(s, sh);
  if (threadIdx.x == 0) J[0] = s / (double)B;
}

// partial[ch][j][i] = sum_{e in chunk ch} d[e][j] u[e][i]; column q holds sum_e d[e][j].
template <typename T>
__global__ __launch_bounds__(NT) void k_wpart(const T* uN, const double* d, double* part, int B, int q, int nc) {
  const int ch = blockIdx.x;
  const size_t o = (size_t)blockIdx.y * NT + threadIdx.x;
  const size_t nw = (size_t)nc * (q + 1);
  if (o >= nw) return;
  const int j = (int)(o / (q + 1)), i = (int)(o - (size_t)j * (q + 1));
  const int e0 = ch * CHUNK, e1 = min(B, e0 + CHUNK);
  double acc = 0.0;
#pragma unroll 8
  for (int e = e0; e < e1; ++e) acc += d[(size_t)e * nc + j] * (i < q ? (double)uN[(size_t)e * q + i] : 1.0);
  part[(size_t)ch * nw + o] = acc;
}

// Sum of the chunk partials: a workgroup takes FO outputs, thread group g sums
// chunks g, g + NT/FO, ... of one output, and the groups are added in order.
constexpr int FO = 8;
template <typename T>
__global__ __launch_bounds__(NT) void k_wfinal(const double* part, int nch, T* dW, T* dmu, int q, int nc) {
  __shared__ double sh[NT];
  const size_t nw = (size_t)nc * (q + 1);
  const size_t o = (size_t)blockIdx.x * FO + (threadIdx.x % FO);
  double s = 0.0;
  if (o < nw)
    for (int ch = threadIdx.x / FO; ch < nch; ch += NT / FO) s += part[(size_t)ch * nw + o];
  sh[threadIdx.x] = s;
  __syncthreads();
  if (threadIdx.x >= FO || o >= nw) return;
  double t = 0.0;
  for (int g = 0; g < NT / FO; ++g) t += sh[g * FO + threadIdx.x];
  const int j = (int)(o / (q + 1)), i = (int)(o - (size_t)j * (q + 1));
  if (i < q) dW[(size_t)j * q + i] = (T)t;
  else dmu[j] = (T)t;
}

// Classification hit of each example: 1 when argmax_j (W u + mu)_j equals
// argmax_j c_j (the first index on ties, on both), else 0. One segment of S
// lanes per example as in k_head; logits in fp64.
template <typename T>
__global__ __launch_bounds__(NT) void k_hits(const T* uN, const T* Wc, const T* mu, const T* c, double* hit, int B,
                                             int q, int nc, int S) {
  const int t = threadIdx.x, j = t & (S - 1);
  const int e = blockIdx.x * (NT / S) + t / S;
  const bool on = e < B;
  const T* u = uN + (size_t)(on ? e : B - 1) * q;
  double zj = -INFINITY;
  for (int jj = 0; jj < nc; ++jj) {
    double p = 0.0;
    for (int i = j; i < q; i += S) p += (double)Wc[(size_t)jj * q + i] * (double)u[i];
    for (int off = S / 2; off > 0; off >>= 1) p += __shfl_xor(p, off, 64);
    if (j == jj) zj = p + (double)mu[jj];
  }
  const double cj = j < nc && on ? (double)c[(size_t)(on ? e : 0) * nc + j] : -INFINITY;
  // (value, index) arg-max over the segment: larger value wins, the lower index on ties
  double zv = zj, cv = cj;
  int zi = j, ci = j;
  for (int off = S / 2; off > 0; off >>= 1) {
    const double zo = __shfl_xor(zv, off, 64), co = __shfl_xor(cv, off, 64);
    const int zio = __shfl_xor(zi, off, 64), cio = __shfl_xor(ci, off, 64);
    if (zo > zv || (zo == zv && zio < zi)) zv = zo, zi = zio;
    if (co > cv || (co == cv && cio < ci)) cv = co, ci = cio;
  }
  if (on && j == 0) hit[e] = zi == ci ? 1.0 : 0.0;
}

size_t up(size_t x) { return (x + 255) / 256 * 256; }

template <typename T>
hipError_t loss_t(int B, int q, int nc, const void* uN, const void* Wc, const void* mu, const void* c, double* J,
                  void* lamN, void* dW, void* dmu, void* ws, hipStream_t st) {
  char* w = static_cast<char*>(ws);
  double* z = reinterpret_cast<double*>(w);
  double* loss = reinterpret_cast<double*>(w + up((size_t)B * nc * 8));
  double* part = reinterpret_cast<double*>(w + up((size_t)B * nc * 8) + up((size_t)B * 8));
  const int nch = (B + CHUNK - 1) / CHUNK;
  const size_t nw = (size_t)nc * (q + 1);
  int S = 1;
  while (S < nc) S *= 2;
  const int per = NT / S;  // examples per workgroup
  k_head<T><<<(B + per - 1) / per, NT, 0, st>>>((const T*)uN, (const T*)Wc, (const T*)mu, (const T*)c, z, loss,
                                                (T*)lamN, B, q, nc, S);
  k_mean<<<1, NT_MEAN, 0, st>>>(loss, B, J);
  k_wpart<T><<<dim3(nch, (unsigned)((nw + NT - 1) / NT)), NT, 0, st>>>((const T*)uN, z, part, B, q, nc);
  k_wfinal<T><<<(unsigned)((nw + FO - 1) / FO), NT, 0, st>>>(part, nch, (T*)dW, (T*)dmu, q, nc);
  return hipGetLastError();
}

template <typename T>
hipError_t accuracy_t(int B, int q, int nc, const void* uN, const void* Wc, const void* mu, const void* c,
                      double* acc, void* ws, hipStream_t st) {
  double* hit = static_cast<double*>(ws);
  int S = 1;
  while (S < nc) S *= 2;
  const int per = NT / S;
  k_hits<T><<<(B + per - 1) / per, NT, 0, st>>>((const T*)uN, (const T*)Wc, (const T*)mu, (const T*)c, hit, B, q,
                                                nc, S);
  k_mean<<<1, NT_MEAN, 0, st>>>(hit, B, acc);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_accuracy(int dtype, int B, int q, int nc, const void* uN, const void* Wc, const void* mu,
                           const void* c, double* acc, void* ws, hipStream_t st) {
  return dtype == 0 ? accuracy_t<float>(B, q, nc, uN, Wc, mu, c, acc, ws, st)
                    : accuracy_t<double>(B, q, nc, uN, Wc, mu, c, acc, ws, st);
}

size_t loss_workspace_bytes(int B, int q, int nc) {
  const size_t nch = (size_t)(B + CHUNK - 1) / CHUNK;
  return up((size_t)B * nc * 8) + up((size_t)B * 8) + up(nch * nc * (size_t)(q + 1) * 8);
}

hipError_t launch_loss(int dtype, int B, int q, int nc, const void* uN, const void* Wc, const void* mu,
                       const void* c, double* J, void* lamN, void* dW, void* dmu, void* ws, hipStream_t st) {
  return dtype == 0 ? loss_t<float>(B, q, nc, uN, Wc, mu, c, J, lamN, dW, dmu, ws, st)
                    : loss_t<double>(B, q, nc, uN, Wc, mu, c, J, lamN, dW, dmu, ws, st);
}

}  // namespace lp
