// Softmax hypothesis and cross-entropy loss at the network output, and the
// adjoint terminal value (Section 2.1, the softmax and loss equations; the
// terminal condition of the adjoint equations in Section 2.3):
//   z_k = W u_k^N + mu,  S_k = softmax(z_k),  J = (1/B) sum_k -c_k^T log S_k,
//   d_k = (S_k - c_k) / B,  lam_k^N = W^T d_k,  dW = sum_k d_k (u_k^N)^T,  dmu = sum_k d_k.
// A boundary helper outside the per-iteration hot path; all reductions run in a
// fixed order. Workspace: logits/residuals d [B][nc] (fp64), per-example losses
// [B] (fp64), and per-chunk partials of dW and dmu [nchunks][nc][q+1] (fp64; with
// the staged head each row also carries the chunk's loss sum).
#include <math.h>

#include <algorithm>

#include "lp_device.h"
#include "lp_internal.h"

namespace lp {
namespace {

constexpr int NT = 256;
constexpr int CHUNK = 16;  // examples per partial of dW, dmu (one round of loads, many workgroups)

// Head of the network, one segment of S lanes per example (S = the power of two
// >= nc; lane j of the segment owns class j): the logits z_j = mu_j + W_j . u,
// the softmax and loss_e with segment reductions, d_j = (S_j - c_j)/B, and
// lam^N = W^T d (each lane takes features i = j mod S). All sums run in fp64 and
// in a fixed order.
// STAGE: W (rows padded to q+1 against LDS bank conflicts), mu and the
// workgroup's rows of u^N are first copied to LDS with coalesced loads, and each
// lane sums its own class's dot product in feature order, so no step waits on a
// global load or a shuffle per class; the workgroup then also writes its partial
// of dW and dmu, part[blk][j][i] = sum over its examples, in order, of
// d[e][j] u[e][i] (column q: d[e][j]), and after them the sum of its losses
// (partial rows of nc (q+1) + 1). Otherwise (W and u too large for LDS) the
// segment splits each dot product over its lanes and adds the parts with
// shuffles, and k_wpart forms the partials.
template <typename T, bool STAGE>
__global__ __launch_bounds__(NT) void k_head(const T* uN, const T* Wc, const T* mu, const T* c, double* d,
                                             double* loss, T* lamN, double* part, int B, int q, int nc, int S) {
  extern __shared__ double hsh[];  // STAGE: W [nc][q+1], mu [nc], u rows [NT/S][q], as T
  __shared__ double dsh[NT];
  __shared__ double lsh[NT];  // STAGE: loss of each of the workgroup's examples
  const int t = threadIdx.x, j = t & (S - 1), seg = t - j, per = NT / S;
  const int e = blockIdx.x * per + t / S;
  const bool on = e < B;  // uniform over a segment
  const bool cls = j < nc;
  const double cj = cls && on ? (double)c[(size_t)e * nc + j] : 0.0;
  const T* W = Wc;
  int wp = q;  // row pitch of W
  double zj = -INFINITY;
  if constexpr (STAGE) {
    T* sw = reinterpret_cast<T*>(hsh);
    T* sm = sw + (size_t)nc * (q + 1);
    T* su = sm + nc;
    for (int k = t; k < nc * q; k += NT) {
      const int r = k / q;
      sw[k + r] = Wc[k];
    }
    if (t < nc) sm[t] = mu[t];
    const size_t r0 = (size_t)blockIdx.x * per;
    const int rows = min(per, B - (int)r0);
    for (int k = t; k < rows * q; k += NT) su[k] = uN[r0 * q + k];
    __syncthreads();
    W = sw;
    wp = q + 1;
    if (cls) {
      const T* wr = sw + (size_t)j * (q + 1);
      const T* u = su + (size_t)(on ? t / S : 0) * q;
      double p = (double)sm[j];
      int i = 0;
      for (; i + 8 <= q; i += 8) {
        double x[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) x[k] = (double)wr[i + k] * (double)u[i + k];
#pragma unroll
        for (int k = 0; k < 8; ++k) p += x[k];
      }
      for (; i < q; ++i) p += (double)wr[i] * (double)u[i];
      zj = p;
    }
  } else {
    const T* u = uN + (size_t)(on ? e : B - 1) * q;
    for (int jj = 0; jj < nc; ++jj) {
      double p = 0.0;
      for (int i = j; i < q; i += S) p += (double)Wc[(size_t)jj * q + i] * (double)u[i];
      for (int off = S / 2; off > 0; off >>= 1) p += __shfl_xor(p, off, 64);
      if (j == jj) zj = p + (double)mu[jj];
    }
  }
  double m = zj;
  for (int off = S / 2; off > 0; off >>= 1) m = fmax(m, __shfl_xor(m, off, 64));
  double den = cls ? exp(zj - m) : 0.0;
  for (int off = S / 2; off > 0; off >>= 1) den += __shfl_xor(den, off, 64);
  const double lden = log(den);
  const double logp = cls ? (zj - m) - lden : 0.0;
  double l = cls ? -cj * logp : 0.0;
  for (int off = S / 2; off > 0; off >>= 1) l += __shfl_xor(l, off, 64);
  const double dj = cls ? (exp(logp) - cj) / (double)B : 0.0;
  if (on) {
    if (cls) d[(size_t)e * nc + j] = dj;
    if (j == 0) loss[e] = l;
  }
  dsh[t] = dj;
  if (STAGE && j == 0) lsh[t / S] = l;
  __syncthreads();
  if constexpr (STAGE) {
    const T* su = reinterpret_cast<const T*>(hsh) + (size_t)nc * (q + 1) + nc;
    const int rows = min(per, B - blockIdx.x * per);
    const int nw = nc * (q + 1);
    for (int o = t; o <= nw; o += NT) {
      const int jj = o / (q + 1), i = o - jj * (q + 1);
      double acc = 0.0;
      if (o == nw) {
        for (int r = 0; r < rows; ++r) acc += lsh[r];
      } else if (i < q) {
        for (int r = 0; r < rows; ++r) acc += dsh[r * S + jj] * (double)su[r * q + i];
      } else {
        for (int r = 0; r < rows; ++r) acc += dsh[r * S + jj];
      }
      part[(size_t)blockIdx.x * (nw + 1) + o] = acc;
    }
  }
  if (!on) return;
  for (int i = j; i < q; i += S) {
    double acc = 0.0;
    for (int jj = 0; jj < nc; ++jj) acc += (double)W[(size_t)jj * wp + i] * dsh[seg + jj];
    lamN[(size_t)e * q + i] = (T)acc;
  }
}

// LDS bytes k_head<T, true> needs (W with padded rows, mu and NT/S rows of u, as T).
size_t head_lds(size_t esz, int q, int nc, int S) {
  return ((size_t)nc * (q + 1) + nc + (size_t)(NT / S) * q) * esz;
}
constexpr size_t HEAD_LDS_MAX = 64 * 1024;

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
// The chunk's loads are issued together (clamped rows, their products dropped
// past the end), then added in example order.
template <typename T>
__global__ __launch_bounds__(NT) void k_wpart(const T* uN, const double* d, double* part, int B, int q, int nc) {
  const int ch = blockIdx.x;
  const size_t o = (size_t)blockIdx.y * NT + threadIdx.x;
  const size_t nw = (size_t)nc * (q + 1);
  if (o >= nw) return;
  const int j = (int)(o / (q + 1)), i = (int)(o - (size_t)j * (q + 1));
  const int e0 = ch * CHUNK;
  double dv[CHUNK], uv[CHUNK];
#pragma unroll
  for (int k = 0; k < CHUNK; ++k) {
    const int e = min(e0 + k, B - 1);
    dv[k] = d[(size_t)e * nc + j];
    uv[k] = i < q ? (double)uN[(size_t)e * q + i] : 1.0;
  }
  double acc = 0.0;
#pragma unroll
  for (int k = 0; k < CHUNK; ++k) acc += e0 + k < B ? dv[k] * uv[k] : 0.0;
  part[(size_t)ch * nw + o] = acc;
}

// Sum of the chunk partials: a workgroup takes FO outputs, thread group g sums
// chunks g, g + NT/FO, ... of one output (in that order, loads issued eight at a
// time), and the groups are added in order. Partial rows are `ps` doubles apart;
// with J given, output nc (q+1) is the loss sum and J = that sum / B.
constexpr int FO = 8;
template <typename T>
__global__ __launch_bounds__(NT) void k_wfinal(const double* part, int nch, size_t ps, T* dW, T* dmu, double* J,
                                               int B, int q, int nc) {
  __shared__ double sh[NT];
  const size_t nw = (size_t)nc * (q + 1), nout = nw + (J ? 1 : 0);
  const size_t o = (size_t)blockIdx.x * FO + (threadIdx.x % FO);
  double s = 0.0;
  if (o < nout) {
    constexpr int G = NT / FO;
    int ch = threadIdx.x / FO;
    for (; ch + 7 * G < nch; ch += 8 * G) {
      double v[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) v[k] = part[(size_t)(ch + k * G) * ps + o];
#pragma unroll
      for (int k = 0; k < 8; ++k) s += v[k];
    }
    for (; ch < nch; ch += G) s += part[(size_t)ch * ps + o];
  }
  sh[threadIdx.x] = s;
  __syncthreads();
  if (threadIdx.x >= FO || o >= nout) return;
  double t = 0.0;
  for (int g = 0; g < NT / FO; ++g) t += sh[g * FO + threadIdx.x];
  if (o == nw) {
    J[0] = t / (double)B;
    return;
  }
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
  const size_t lds = head_lds(sizeof(T), q, nc, S);
  if (lds <= HEAD_LDS_MAX) {
    const int nblk = (B + per - 1) / per;
    k_head<T, true><<<nblk, NT, lds, st>>>((const T*)uN, (const T*)Wc, (const T*)mu, (const T*)c, z, loss,
                                           (T*)lamN, part, B, q, nc, S);
    k_wfinal<T><<<(unsigned)((nw + 1 + FO - 1) / FO), NT, 0, st>>>(part, nblk, nw + 1, (T*)dW, (T*)dmu, J, B, q,
                                                                   nc);
    return hipGetLastError();
  }
  // W and u^N do not fit in LDS (wide states): a whole wave per example, so its
  // dot products split over 64 lanes and the batch gives NT/64 examples per
  // workgroup (a segment as narrow as the class count would leave most CUs idle)
  const int Sw = nc <= 64 ? 64 : S;
  k_head<T, false><<<(B + NT / Sw - 1) / (NT / Sw), NT, 0, st>>>((const T*)uN, (const T*)Wc, (const T*)mu,
                                                                 (const T*)c, z, loss, (T*)lamN, nullptr, B, q,
                                                                 nc, Sw);
  k_mean<<<1, NT_MEAN, 0, st>>>(loss, B, J);
  k_wpart<T><<<dim3(nch, (unsigned)((nw + NT - 1) / NT)), NT, 0, st>>>((const T*)uN, z, part, B, q, nc);
  k_wfinal<T><<<(unsigned)((nw + FO - 1) / FO), NT, 0, st>>>(part, nch, nw, (T*)dW, (T*)dmu, nullptr, B, q, nc);
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

// Workspace of the loss for one class count: the logits (B nc doubles), the
// per-example losses (B doubles) and the partials of the path loss_t takes: one
// row of nc (q+1) + 1 doubles per head workgroup of NT/S examples when k_head
// stages W and u^N in LDS, else one row of nc (q+1) doubles per CHUNK examples.
size_t loss_workspace_bytes(size_t esz, int B, int q, int nc) {
  int S = 1;
  while (S < nc) S *= 2;
  const size_t nw = (size_t)nc * (q + 1);
  const size_t part = head_lds(esz, q, nc, S) <= HEAD_LDS_MAX ? (size_t)((B + NT / S - 1) / (NT / S)) * (nw + 1)
                                                              : (size_t)((B + CHUNK - 1) / CHUNK) * nw;
  return up((size_t)B * nc * 8) + up((size_t)B * 8) + up(part * 8);
}

// The largest of the above over every class count 1 .. nc_max.
size_t loss_workspace_bytes_max(size_t esz, int B, int q, int nc_max) {
  size_t need = 0;
  for (int nc = 1; nc <= nc_max; ++nc) need = std::max(need, loss_workspace_bytes(esz, B, q, nc));
  return need;
}

hipError_t launch_loss(int dtype, int B, int q, int nc, const void* uN, const void* Wc, const void* mu,
                       const void* c, double* J, void* lamN, void* dW, void* dmu, void* ws, hipStream_t st) {
  return dtype == 0 ? loss_t<float>(B, q, nc, uN, Wc, mu, c, J, lamN, dW, dmu, ws, st)
                    : loss_t<double>(B, q, nc, uN, Wc, mu, c, J, lamN, dW, dmu, ws, st);
}

}  // namespace lp
