// The classifier bias and the softmax cross-entropy loss of ResNet-50's
// training (Section 5.1 of arXiv:1911.07384), averaged over this GPU's batch,
// with its gradient; no loss scaling (Section 4.2: the method trains without
// it), so gradient entries near 1/(N*K) are binary16 subnormals and are kept.
//
// One block per sample row: logits l = rne16(z + b) (an exact float64 sum
// rounded once), a max and a sum of exp(l - max) over the row (float64,
// reduced in a fixed order), the row's loss and its gradient row.  A second
// kernel sums the stored gradient over the batch for the bias (exact in
// float64, one rounding per class).  The work is tiny (N*K = 128,000 for
// ResNet-50 at batch 128); float64 throughout keeps the results within
// float64 rounding of the exact values.

#include "kernels.hpp"

namespace fp16k {
namespace {

constexpr int kLT = 256;

__device__ __forceinline__ double logit(h16 z, h16 b) {
  return (double)to_f32(dbl_to_h16((double)to_f32(z) + (double)to_f32(b)));
}

// Deterministic block reductions over kLT threads: a butterfly within each
// wave, then the four wave results in order.
__device__ __forceinline__ double block_max(double v, double* red) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v = __builtin_fmax(v, __shfl_xor(v, off, 64));
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  const double r = __builtin_fmax(__builtin_fmax(red[0], red[1]), __builtin_fmax(red[2], red[3]));
  __syncthreads();
  return r;
}

__device__ __forceinline__ double block_sum(double v, double* red) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  const double r = ((red[0] + red[1]) + red[2]) + red[3];
  __syncthreads();
  return r;
}

__global__ __launch_bounds__(kLT) void softmax_ce_rows(int K, double inv_n, const h16* z,
                                                       const h16* __restrict__ bias,
                                                       const int32_t* __restrict__ labels,
                                                       float* __restrict__ loss, h16* dz) {
  __shared__ double red[4];
  __shared__ double l_label;
  const int n = blockIdx.x;
  const int t = threadIdx.x;
  const h16* zr = z + (int64_t)n * K;
  const int y = labels[n];
  if (t == 0) l_label = __builtin_nan("");
  __syncthreads();
  // pass 1: row maximum of the logits (NaN logits do not move it)
  double m = -__builtin_inf();
  for (int j = t; j < K; j += kLT) {
    const double l = logit(zr[j], bias[j]);
    if (j == y) l_label = l;
    if (l > m) m = l;
  }
  m = block_max(m, red);
  // pass 2: sum of exp(l - m)
  double s = 0.0;
  for (int j = t; j < K; j += kLT) s += exp(logit(zr[j], bias[j]) - m);
  s = block_sum(s, red);  // its barriers also publish l_label
  if (t == 0) loss[n] = (float)(log(s) + (m - l_label));
  // pass 3: gradient of the batch-mean loss; each thread rewrites only the
  // entries it read, so dz may equal z
  const double inv_s = 1.0 / s;
  for (int j = t; j < K; j += kLT) {
    const double p = exp(logit(zr[j], bias[j]) - m) * inv_s;
    dz[(int64_t)n * K + j] = dbl_to_h16((p - (j == y ? 1.0 : 0.0)) * inv_n);
  }
}

// The bias gradient: the sum over the batch of each class's dz, rounded once.
// |dz| <= 1 (a probability less the label, over N), so every term is a
// multiple of 2^-24 below 1 in magnitude and the float64 sum of up to 2^17
// of them is exact in any order: eight row groups of 32 classes per
// workgroup, each thread's 16 rows of a 128-row block loaded together, then
// the groups in order (one thread per class walking all rows waited on one
// load at a time: 34 us for 128 x 1000).
__global__ __launch_bounds__(256) void bias_grad(int N, int K, const h16* __restrict__ dz,
                                                 h16* __restrict__ dbias) {
  __shared__ double part[8][32];
  const int c = threadIdx.x & 31, r = threadIdx.x >> 5;
  const int j = blockIdx.x * 32 + c;
  double a = 0.0;
  if (j < K) {
    for (int n0 = r; n0 < N; n0 += 128) {
      float v[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        const int n = n0 + 8 * u;
        v[u] = n < N ? to_f32(dz[(int64_t)n * K + j]) : 0.0f;
      }
#pragma unroll
      for (int u = 0; u < 16; ++u) a += (double)v[u];
    }
  }
  part[r][c] = a;
  __syncthreads();
  if (r == 0 && j < K) {
    double t = 0.0;
#pragma unroll
    for (int g = 0; g < 8; ++g) t += part[g][c];
    dbias[j] = dbl_to_h16(t);
  }
}

}  // namespace

hipError_t launch_softmax_ce(int N, int K, const h16* z, const h16* bias, const int32_t* labels,
                             float* loss, h16* dz, h16* dbias, hipStream_t st) {
  hipLaunchKernelGGL(softmax_ce_rows, dim3(N), dim3(kLT), 0, st, K, 1.0 / (double)N, z, bias,
                     labels, loss, dz);
  hipLaunchKernelGGL(bias_grad, dim3(ceil_div(K, 32)), dim3(256), 0, st, N, K, dz, dbias);
  return hipGetLastError();
}

}  // namespace fp16k
