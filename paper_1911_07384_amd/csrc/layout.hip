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

// Cp a multiple of 8: one thread per pixel, 16-byte stores.  Every load is
// unconditional (channel min(c, C - 1), then zero past C), so a thread's
// loads are in flight together.
__global__ void pad_channels_vec(const h16* __restrict__ src, h16* __restrict__ dst, int64_t P,
                                 int C, int Cp) {
  for (int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; p < P;
       p += (int64_t)gridDim.x * blockDim.x) {
    const h16* s = src + p * C;
    for (int c0 = 0; c0 < Cp; c0 += 8) {
      V8 v;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int c = c0 + e;
        const h16 x = s[c < C ? c : C - 1];
        v.h[e] = c < C ? x : (h16)0.0f;
      }
      store16(dst + p * Cp + c0, v);
    }
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

// All stride phases of the data-gradient filter in one launch, as 64 x 64
// (channel x filter) tile transposes through LDS: block (c tile, k tile, tap)
// reads 64 rows of 64 consecutive channels of W (one filter k each, 16-byte
// loads when the channel count allows) and writes 64 rows of 64 consecutive
// k of dst (one channel each, 16-byte stores).
// The tap table maps each source tap (r, s) to its phase filter and its
// position (tr, ts) there.
constexpr int kMaxTaps = 64;
struct DgradTaps {
  int64_t off[kMaxTaps];  // element offset of the tap's phase filter in dst
  int ntr[kMaxTaps], nts[kMaxTaps], tr[kMaxTaps], ts[kMaxTaps], r[kMaxTaps], s[kMaxTaps];
};

// One 64 x 64 (channel x filter) tile of one tap: reads 64 rows of 64
// consecutive channels of W at tap (r, s) and writes them transposed into the
// phase filter at dst + off (ntr x nts taps, tap (tr, ts)).
__device__ __forceinline__ void dgrad_tile(const h16* __restrict__ w, h16* __restrict__ dst,
                                           int K, int C, int R, int S, int Cw, int Kp, int r,
                                           int s, int64_t off, int ntr, int nts, int tr, int ts,
                                           int c0, int k0) {
  __shared__ h16 tile[64][66];  // [channel][k]
  const int t = threadIdx.x;
  if (Cw % 8 == 0) {
    // 16-byte loads, both of a thread's in flight together
    V8 v[2];
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int ci = t + 256 * q, kk = ci >> 3, c = c0 + (ci & 7) * 8;
      const int k = k0 + kk;
      if (k < K && c < C) {
        v[q] = load16(w + (((int64_t)k * R + r) * S + s) * Cw + c);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) v[q].s[e] = 0;
      }
    }
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int ci = t + 256 * q, kk = ci >> 3, cc = (ci & 7) * 8;
#pragma unroll
      for (int e = 0; e < 8; ++e) tile[cc + e][kk] = v[q].h[e];
    }
  } else {
    const int cc = t & 63;
    const int c = c0 + cc;
    h16 v[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int k = k0 + (t >> 6) + 4 * i;
      v[i] = (k < K && c < C) ? w[(((int64_t)k * R + r) * S + s) * Cw + c] : (h16)0.0f;
    }
#pragma unroll
    for (int i = 0; i < 16; ++i) tile[cc][(t >> 6) + 4 * i] = v[i];
  }
  __syncthreads();
  const int cc = t >> 2, kq = (t & 3) * 16;
  const int c = c0 + cc;
  if (c >= C) return;
  h16* row = dst + off + (((int64_t)c * ntr + tr) * nts + ts) * Kp;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int k = k0 + kq + h * 8;
    if (k < Kp) {  // Kp % 8 == 0: the 8 values stay inside the row
      V8 v;
#pragma unroll
      for (int e = 0; e < 8; ++e) v.h[e] = tile[cc][kq + h * 8 + e];
      store16(row + k, v);
    }
  }
}

__global__ __launch_bounds__(256) void dgrad_filter_tiled(const h16* __restrict__ w,
                                                          h16* __restrict__ dst, int K, int C,
                                                          int R, int S, int Cw, int Kp,
                                                          const DgradTaps taps) {
  const int q = blockIdx.z;
  dgrad_tile(w, dst, K, C, R, S, Cw, Kp, taps.r[q], taps.s[q], taps.off[q], taps.ntr[q],
             taps.nts[q], taps.tr[q], taps.ts[q], blockIdx.x * 64, blockIdx.y * 64);
}

// Many filters' rearrangements in one launch: the jobs (one filter each, all
// its taps) are laid end to end over a 1-D grid of 64 x 64 tiles; each block
// finds its job, then its tap by walking the stride phases in (ph, pw)
// row-major order as the per-filter launcher does.
constexpr int kDfBatch = 32;  // jobs per launch (kernel-argument table)
struct DgradFiltBatch {
  int n;
  DgradFiltJob j[kDfBatch];
};

__global__ __launch_bounds__(256) void dgrad_filter_batched(const DgradFiltBatch b) {
  const int bid = blockIdx.x;
  int i = 0;
  while (i + 1 < b.n && b.j[i + 1].blk0 <= bid) ++i;
  const DgradFiltJob& J = b.j[i];
  const int CT = (J.C + 63) / 64, KT = (J.Kp + 63) / 64;
  int local = bid - J.blk0;
  int q = local / (CT * KT);
  local -= q * CT * KT;
  const int ct = local / KT, kt = local - (local / KT) * KT;
  int64_t off = 0;
  for (int ph = 0; ph < J.sh; ++ph) {
    for (int pw = 0; pw < J.sw; ++pw) {
      const DgradPhase d = dgrad_phase(ph, pw, 1, 1, J.R, J.S, J.sh, J.sw, J.pad_h, J.pad_w);
      const int nt = d.ntr * d.nts;
      if (q < nt) {
        const int tr = q / d.nts, ts = q - (q / d.nts) * d.nts;
        dgrad_tile(J.w, J.dst, J.K, J.C, J.R, J.S, J.C, J.Kp, d.r0 + J.sh * (d.ntr - 1 - tr),
                   d.s0 + J.sw * (d.nts - 1 - ts), off, d.ntr, d.nts, tr, ts, ct * 64, kt * 64);
        return;
      }
      q -= nt;
      off += (int64_t)J.C * nt * J.Kp;
    }
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

// 2x2 space-to-depth of a 3-channel NHWC image (H, W even):
// dst[n][a][b][(dh*2 + dw)*3 + c] = src[n][2a + dh][2b + dw][c], channels
// 12..15 zero.  One thread per destination pixel: 12 loads of 2 bytes (all
// in flight), two 16-byte stores.
__global__ void s2d3_kernel(const h16* __restrict__ src, h16* __restrict__ dst, int N, int H,
                            int W) {
  const int H2 = H / 2, W2 = W / 2;
  const int64_t total = (int64_t)N * H2 * W2;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int b = (int)(i % W2);
    const int64_t t = i / W2;
    const int a = (int)(t % H2);
    const int n = (int)(t / H2);
    const h16* s0 = src + (((int64_t)n * H + 2 * a) * W + 2 * b) * 3;
    const h16* s1 = s0 + (int64_t)W * 3;
    V8 lo, hi;
#pragma unroll
    for (int c = 0; c < 6; ++c) lo.h[c] = s0[c];      // (dh 0, dw 0), (0, 1)
    lo.h[6] = s1[0];
    lo.h[7] = s1[1];
    hi.h[0] = s1[2];                                 // (1, 0) last channel
#pragma unroll
    for (int c = 0; c < 3; ++c) hi.h[1 + c] = s1[3 + c];  // (1, 1)
#pragma unroll
    for (int c = 4; c < 8; ++c) hi.h[c] = (h16)0.0f;
    store16(dst + i * 16, lo);
    store16(dst + i * 16 + 8, hi);
  }
}

hipError_t launch_s2d3(const h16* src, h16* dst, int N, int H, int W, hipStream_t st) {
  hipLaunchKernelGGL(s2d3_kernel, dim3(grid_for((int64_t)N * (H / 2) * (W / 2))), dim3(kThreads),
                     0, st, src, dst, N, H, W);
  return hipGetLastError();
}

hipError_t launch_pad_channels(const h16* src, h16* dst, int64_t P, int C, int Cp, hipStream_t st) {
  if (Cp % 8 == 0)
    hipLaunchKernelGGL(pad_channels_vec, dim3(grid_for(P)), dim3(kThreads), 0, st, src, dst, P, C,
                       Cp);
  else
    hipLaunchKernelGGL(pad_channels_kernel, dim3(grid_for(P * Cp)), dim3(kThreads), 0, st, src,
                       dst, P, C, Cp);
  return hipGetLastError();
}

hipError_t launch_dgrad_filters(const DgradFiltJob* jobs, int n, hipStream_t st) {
  DgradFiltBatch b{};
  int blocks = 0;
  auto flush = [&]() -> hipError_t {
    if (b.n == 0) return hipSuccess;
    hipLaunchKernelGGL(dgrad_filter_batched, dim3(blocks), dim3(256), 0, st, b);
    b.n = 0;
    blocks = 0;
    return hipGetLastError();
  };
  for (int i = 0; i < n; ++i) {
    const DgradFiltJob& J = jobs[i];
    if (J.R * J.S > kMaxTaps || J.Kp % 8 != 0) {
      // outside the tiled path: its own launch(es)
      const hipError_t e = launch_dgrad_filter(J.w, J.dst, J.K, J.C, J.R, J.S, J.C, J.Kp, J.sh,
                                               J.sw, J.pad_h, J.pad_w, st);
      if (e != hipSuccess) return e;
      continue;
    }
    int taps = 0;
    for (int ph = 0; ph < J.sh; ++ph)
      for (int pw = 0; pw < J.sw; ++pw) {
        const DgradPhase d = dgrad_phase(ph, pw, 1, 1, J.R, J.S, J.sh, J.sw, J.pad_h, J.pad_w);
        taps += d.ntr * d.nts;
      }
    const int nb = taps * ((J.C + 63) / 64) * ((J.Kp + 63) / 64);
    if (nb == 0) continue;
    if (b.n == kDfBatch) {
      const hipError_t e = flush();
      if (e != hipSuccess) return e;
    }
    b.j[b.n] = J;
    b.j[b.n].blk0 = blocks;
    ++b.n;
    blocks += nb;
  }
  return flush();
}

hipError_t launch_dgrad_filter(const h16* w, h16* dst, int K, int C, int R, int S, int Cw, int Kp,
                               int sh, int sw, int pad_h, int pad_w, hipStream_t st) {
  // phases in (ph, pw) row-major order, each filter packed after the previous
  if (R * S <= kMaxTaps && Kp % 8 == 0) {
    DgradTaps taps;
    int n = 0;
    int64_t off = 0;
    for (int ph = 0; ph < sh; ++ph) {
      for (int pw = 0; pw < sw; ++pw) {
        const DgradPhase d = dgrad_phase(ph, pw, 1, 1, R, S, sh, sw, pad_h, pad_w);
        for (int tr = 0; tr < d.ntr; ++tr) {
          for (int ts = 0; ts < d.nts; ++ts) {
            taps.off[n] = off;
            taps.ntr[n] = d.ntr;
            taps.nts[n] = d.nts;
            taps.tr[n] = tr;
            taps.ts[n] = ts;
            taps.r[n] = d.r0 + sh * (d.ntr - 1 - tr);
            taps.s[n] = d.s0 + sw * (d.nts - 1 - ts);
            ++n;
          }
        }
        off += (int64_t)C * d.ntr * d.nts * Kp;
      }
    }
    if (n == 0) return hipSuccess;
    hipLaunchKernelGGL(dgrad_filter_tiled, dim3((C + 63) / 64, (Kp + 63) / 64, n), dim3(256), 0, st,
                       w, dst, K, C, R, S, Cw, Kp, taps);
    return hipGetLastError();
  }
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
