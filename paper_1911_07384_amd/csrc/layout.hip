// Layout conversions used around the native NHWC kernels: NCHW <-> NHWC,
// channel padding to a multiple of eight (16-byte vectors), and the
// per-stride-phase filter transform that turns the data gradient into
// stride-1 forward-style gathers.  All are plain copies (bit-exact).

#include "kernels.hpp"

namespace fp16k {
namespace {

constexpr int kThreads = 256;

inline unsigned grid_for(int64_t n) {
  int64_t b = (n + kThreads - 1) / kThreads;
  if (b < 1) b = 1;
  if (b > (1 << 20)) b = 1 << 20;
  return (unsigned)b;
}

// dst[n][hw][c] = c < C ? src[n][c][hw] : 0, for c < Cp.
__global__ void nchw_to_nhwc_kernel(const h16* __restrict__ src, h16* __restrict__ dst, int N,
                                    int C, int HW, int Cp) {
  const int64_t total = (int64_t)N * HW * Cp;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int c = (int)(i % Cp);
    const int64_t t = i / Cp;
    const int hw = (int)(t % HW);
    const int64_t n = t / HW;
    dst[i] = c < C ? src[(n * C + c) * HW + hw] : (h16)0.0f;
  }
}

// dst[n][c][hw] = src[n][hw][c] for c < C.
__global__ void nhwc_to_nchw_kernel(const h16* __restrict__ src, h16* __restrict__ dst, int N,
                                    int C, int HW, int Cp) {
  const int64_t total = (int64_t)N * C * HW;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int hw = (int)(i % HW);
    const int64_t t = i / HW;
    const int c = (int)(t % C);
    const int64_t n = t / C;
    dst[i] = src[(n * HW + hw) * Cp + c];
  }
}

__global__ void pad_channels_kernel(const h16* __restrict__ src, h16* __restrict__ dst, int64_t P,
                                    int C, int Cp) {
  const int64_t total = P * Cp;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int c = (int)(i % Cp);
    const int64_t p = i / Cp;
    dst[i] = c < C ? src[p * C + c] : (h16)0.0f;
  }
}

// One stride phase of the data-gradient filter:
// dst[c][tr][ts][k] = k < K ? W[k][r0 + sh*(ntr-1-tr)][s0 + sw*(nts-1-ts)][c] : 0.
__global__ void dgrad_filter_kernel(const h16* __restrict__ w, h16* __restrict__ dst, int K, int C,
                                    int R, int S, int Cw, int Kp, int r0, int s0, int ntr, int nts,
                                    int sh, int sw) {
  const int64_t total = (int64_t)C * ntr * nts * Kp;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int k = (int)(i % Kp);
    int64_t t = i / Kp;
    const int ts = (int)(t % nts);
    t /= nts;
    const int tr = (int)(t % ntr);
    const int c = (int)(t / ntr);
    const int r = r0 + sh * (ntr - 1 - tr);
    const int s = s0 + sw * (nts - 1 - ts);
    dst[i] = k < K ? w[(((int64_t)k * R + r) * S + s) * Cw + c] : (h16)0.0f;
  }
}

}  // namespace

hipError_t launch_nchw_to_nhwc(const h16* src, h16* dst, int N, int C, int HW, int Cp,
                               hipStream_t st) {
  hipLaunchKernelGGL(nchw_to_nhwc_kernel, dim3(grid_for((int64_t)N * HW * Cp)), dim3(kThreads), 0,
                     st, src, dst, N, C, HW, Cp);
  return hipGetLastError();
}

hipError_t launch_nhwc_to_nchw(const h16* src, h16* dst, int N, int C, int HW, int Cp,
                               hipStream_t st) {
  hipLaunchKernelGGL(nhwc_to_nchw_kernel, dim3(grid_for((int64_t)N * C * HW)), dim3(kThreads), 0,
                     st, src, dst, N, C, HW, Cp);
  return hipGetLastError();
}

hipError_t launch_pad_channels(const h16* src, h16* dst, int64_t P, int C, int Cp, hipStream_t st) {
  hipLaunchKernelGGL(pad_channels_kernel, dim3(grid_for(P * Cp)), dim3(kThreads), 0, st, src, dst,
                     P, C, Cp);
  return hipGetLastError();
}

hipError_t launch_dgrad_filter(const h16* w, h16* dst, int K, int C, int R, int S, int Cw, int Kp,
                               int sh, int sw, int pad_h, int pad_w, hipStream_t st) {
  // phases in (ph, pw) row-major order, each filter packed after the previous
  int64_t off = 0;
  for (int ph = 0; ph < sh; ++ph) {
    for (int pw = 0; pw < sw; ++pw) {
      const DgradPhase d = dgrad_phase(ph, pw, 1, 1, R, S, sh, sw, pad_h, pad_w);
      const int64_t n = (int64_t)C * d.ntr * d.nts * Kp;
      if (n > 0) {
        hipLaunchKernelGGL(dgrad_filter_kernel, dim3(grid_for(n)), dim3(kThreads), 0, st, w,
                           dst + off, K, C, R, S, Cw, Kp, d.r0, d.s0, d.ntr, d.nts, sh, sw);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
      }
      off += n;
    }
  }
  return hipSuccess;
}

}  // namespace fp16k
