// Convolutions with every operation in binary16 (the strict reading of "all
// arithmetic in FP16", arXiv:1911.07384 Section 5.2), for measuring what the
// float32 accumulators of the default kernels buy.
//
// Each output is a binary16 accumulator that starts at +0 and takes its
// terms one at a time as binary16 fused multiply-adds (v_pk_fma_f16: one
// rounding of the exact a*b + acc, binary16 subnormals kept), in a declared
// order of the convolution's logical indices:
//   forward         y[n,k,p,q]  taps (r, s) row-major, channels c ascending;
//   data gradient   dx[n,c,h,w] taps (r, s) row-major that reach (h, w) from
//                               a point of the output grid, then k ascending;
//   weight gradient dW[k,c,r,s] output pixels (n, p, q) in order.
// A tap outside the image (or the output grid) is not a term.  Since every
// output's chain is sequential, the parallelism is across outputs only: each
// lane carries four independent chains as the two halves of four packed
// registers (8 outputs), and the operand that all lanes of a wave share is
// staged in LDS (forward, data gradient) or read with wave-uniform loads
// (weight gradient).  NHWC activations, KRSC filters, any C and K.

#include "kernels.hpp"

namespace fp16k {
namespace {

typedef _Float16 h2 __attribute__((ext_vector_type(2)));

constexpr int kChunk = 1024;  // reduction channels staged in LDS per round

__device__ __forceinline__ h2 fma2(h2 a, h2 b, h2 c) { return __builtin_elementwise_fma(a, b, c); }

__device__ __forceinline__ void store8(h16* out, int64_t base, int valid, const h2 (&acc)[4],
                                       bool vec) {
  if (vec && valid == 8) {
    V8 v;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      v.h[2 * j] = acc[j].x;
      v.h[2 * j + 1] = acc[j].y;
    }
    store16(out + base, v);
  } else {
#pragma unroll
    for (int j = 0; j < 8; ++j)
      if (j < valid) out[base + j] = (j & 1) ? acc[j >> 1].y : acc[j >> 1].x;
  }
}

// Forward.  Thread = one output pixel x 8 output channels; the workgroup's
// 256 pixels share the channel block, whose filter slice of the current tap
// (8 x chunk values, pairs (k, k+1) adjacent) sits in LDS.
__global__ __launch_bounds__(256) void chain_fwd_kernel(const h16* __restrict__ x,
                                                        const h16* __restrict__ w,
                                                        h16* __restrict__ y, ConvChainArgs a) {
  __shared__ h2 wl[kChunk][4];
  const int64_t M = (int64_t)a.N * a.P * a.Q;
  const int64_t m = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int kb = blockIdx.y * 8;
  const bool live = m < M;
  const int64_t mm = live ? m : 0;
  const int q = (int)(mm % a.Q);
  const int p = (int)((mm / a.Q) % a.P);
  const int n = (int)(mm / ((int64_t)a.Q * a.P));
  const bool vec = (a.C % 8) == 0;
  h2 acc[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) acc[j] = h2{(h16)0.0f, (h16)0.0f};
  for (int r = 0; r < a.R; ++r) {
    for (int s = 0; s < a.S; ++s) {
      const int hi = p * a.sh - a.ph + r, wi = q * a.sw - a.pw + s;
      const bool valid = live && hi >= 0 && hi < a.H && wi >= 0 && wi < a.W;
      const h16* xp = x + (((int64_t)n * a.H + (valid ? hi : 0)) * a.W + (valid ? wi : 0)) * a.C;
      for (int c0 = 0; c0 < a.C; c0 += kChunk) {
        const int cn = a.C - c0 < kChunk ? a.C - c0 : kChunk;
        __syncthreads();
        for (int i = threadIdx.x; i < 8 * cn; i += 256) {
          const int kk = i / cn, cc = i % cn;  // contiguous along c in global memory
          const int k = kb + kk;
          const h16 v = k < a.K ? w[(((int64_t)k * a.R + r) * a.S + s) * a.C + c0 + cc] : (h16)0.0f;
          reinterpret_cast<h16*>(&wl[cc][0])[kk] = v;
        }
        __syncthreads();
        if (valid) {
          int cc = 0;
          if (vec) {
            for (; cc < cn; cc += 8) {
              const V8 xv = load16(xp + c0 + cc);
#pragma unroll
              for (int e = 0; e < 8; ++e) {
                const h2 xx = h2{xv.h[e], xv.h[e]};
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[j] = fma2(xx, wl[cc + e][j], acc[j]);
              }
            }
          } else {
            for (; cc < cn; ++cc) {
              const h16 xs = xp[c0 + cc];
              const h2 xx = h2{xs, xs};
#pragma unroll
              for (int j = 0; j < 4; ++j) acc[j] = fma2(xx, wl[cc][j], acc[j]);
            }
          }
        }
      }
    }
  }
  if (live) {
    const int valid_k = a.K - kb < 8 ? a.K - kb : 8;
    store8(y, mm * a.K + kb, valid_k, acc, (a.K % 8) == 0);
  }
}

// Data gradient.  Thread = one input pixel x 8 input channels; the filter
// slice W[k][r][s][cb..cb+7] of the current tap for a chunk of k sits in LDS.
__global__ __launch_bounds__(256) void chain_dgrad_kernel(const h16* __restrict__ dy,
                                                          const h16* __restrict__ w,
                                                          h16* __restrict__ dx, ConvChainArgs a) {
  __shared__ h2 wl[kChunk][4];
  const int64_t M = (int64_t)a.N * a.H * a.W;
  const int64_t m = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int cb = blockIdx.y * 8;
  const bool live = m < M;
  const int64_t mm = live ? m : 0;
  const int wx = (int)(mm % a.W);
  const int hx = (int)((mm / a.W) % a.H);
  const int n = (int)(mm / ((int64_t)a.W * a.H));
  const bool vec_k = (a.K % 8) == 0;
  const bool vec_c = (a.C % 8) == 0;
  h2 acc[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) acc[j] = h2{(h16)0.0f, (h16)0.0f};
  for (int r = 0; r < a.R; ++r) {
    for (int s = 0; s < a.S; ++s) {
      const int th = hx + a.ph - r, tw = wx + a.pw - s;
      const int p = th >= 0 ? th / a.sh : -1, q = tw >= 0 ? tw / a.sw : -1;
      const bool valid = live && th >= 0 && tw >= 0 && th % a.sh == 0 && tw % a.sw == 0 &&
                         p < a.P && q < a.Q;
      const h16* dyp = dy + (((int64_t)n * a.P + (valid ? p : 0)) * a.Q + (valid ? q : 0)) * a.K;
      for (int k0 = 0; k0 < a.K; k0 += kChunk) {
        const int kn = a.K - k0 < kChunk ? a.K - k0 : kChunk;
        __syncthreads();
        for (int i = threadIdx.x; i < kn; i += 256) {
          const h16* src = w + (((int64_t)(k0 + i) * a.R + r) * a.S + s) * a.C + cb;
          V8 v;
          if (vec_c) {
            v = load16(src);
          } else {
#pragma unroll
            for (int e = 0; e < 8; ++e) v.h[e] = cb + e < a.C ? src[e] : (h16)0.0f;
          }
#pragma unroll
          for (int j = 0; j < 4; ++j) wl[i][j] = h2{v.h[2 * j], v.h[2 * j + 1]};
        }
        __syncthreads();
        if (valid) {
          int kk = 0;
          if (vec_k) {
            for (; kk < kn; kk += 8) {
              const V8 dv = load16(dyp + k0 + kk);
#pragma unroll
              for (int e = 0; e < 8; ++e) {
                const h2 dd = h2{dv.h[e], dv.h[e]};
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[j] = fma2(dd, wl[kk + e][j], acc[j]);
              }
            }
          } else {
            for (; kk < kn; ++kk) {
              const h16 ds = dyp[k0 + kk];
              const h2 dd = h2{ds, ds};
#pragma unroll
              for (int j = 0; j < 4; ++j) acc[j] = fma2(dd, wl[kk][j], acc[j]);
            }
          }
        }
      }
    }
  }
  if (live) {
    const int valid_c = a.C - cb < 8 ? a.C - cb : 8;
    store8(dx, mm * a.C + cb, valid_c, acc, vec_c);
  }
}

// Weight gradient.  A wave = 64 consecutive output channels k (one per lane)
// for one tap (r, s) and one block of 8 input channels: per output pixel each
// lane loads its dy value and the wave shares one 8-channel input vector.
// Workgroup = 4 waves on 4 consecutive channel blocks.
constexpr int kWgUnroll = 8;

__global__ __launch_bounds__(256) void chain_wgrad_kernel(const h16* __restrict__ x,
                                                          const h16* __restrict__ dy,
                                                          h16* __restrict__ dw, ConvChainArgs a) {
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int k = blockIdx.x * 64 + lane;
  const int tap = blockIdx.y;
  const int r = tap / a.S, s = tap % a.S;
  const int cb = (blockIdx.z * 4 + wave) * 8;
  if (cb >= a.C) return;  // whole wave: no barrier in this kernel
  const bool klive = k < a.K;
  const int kc = klive ? k : 0;
  const bool vec_c = (a.C % 8) == 0 && cb + 8 <= a.C;
  h2 acc[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) acc[j] = h2{(h16)0.0f, (h16)0.0f};
  const int64_t npix = (int64_t)a.N * a.P * a.Q;
  // output pixel t = (n, p, q), advanced incrementally (wave-uniform)
  int n = 0, p = 0, q = 0;
  for (int64_t t0 = 0; t0 < npix; t0 += kWgUnroll) {
    h16 dv[kWgUnroll];
    V8 xv[kWgUnroll];
    bool ok[kWgUnroll];
#pragma unroll
    for (int u = 0; u < kWgUnroll; ++u) {
      const bool live = t0 + u < npix;  // past the end: (n, p, q) stays on the last pixel
      const int hi = p * a.sh - a.ph + r, wi = q * a.sw - a.pw + s;
      ok[u] = live && hi >= 0 && hi < a.H && wi >= 0 && wi < a.W;
      const int64_t t = ((int64_t)n * a.P + p) * a.Q + q;
      dv[u] = dy[t * a.K + kc];
      const h16* xp = x + (((int64_t)n * a.H + (ok[u] ? hi : 0)) * a.W + (ok[u] ? wi : 0)) * a.C + cb;
      if (vec_c) {
        xv[u] = load16(xp);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) xv[u].h[e] = cb + e < a.C ? xp[e] : (h16)0.0f;
      }
      if (t0 + u + 1 < npix) {
        if (++q == a.Q) {
          q = 0;
          if (++p == a.P) {
            p = 0;
            ++n;
          }
        }
      }
    }
#pragma unroll
    for (int u = 0; u < kWgUnroll; ++u) {
      if (ok[u]) {
        const h2 dd = h2{dv[u], dv[u]};
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[j] = fma2(dd, h2{xv[u].h[2 * j], xv[u].h[2 * j + 1]}, acc[j]);
      }
    }
  }
  if (klive) {
    const int valid_c = a.C - cb < 8 ? a.C - cb : 8;
    store8(dw, (((int64_t)k * a.R + r) * a.S + s) * a.C + cb, valid_c, acc, (a.C % 8) == 0);
  }
}

}  // namespace

hipError_t launch_conv_chain(const ConvChainArgs& a, int pass, const h16* in0, const h16* in1,
                             h16* out, hipStream_t st) {
  if (pass == 0) {
    const int64_t M = (int64_t)a.N * a.P * a.Q;
    hipLaunchKernelGGL(chain_fwd_kernel, dim3((unsigned)ceil_div64(M, 256), ceil_div(a.K, 8)),
                       dim3(256), 0, st, in0, in1, out, a);
  } else if (pass == 1) {
    const int64_t M = (int64_t)a.N * a.H * a.W;
    hipLaunchKernelGGL(chain_dgrad_kernel, dim3((unsigned)ceil_div64(M, 256), ceil_div(a.C, 8)),
                       dim3(256), 0, st, in0, in1, out, a);
  } else {
    hipLaunchKernelGGL(chain_wgrad_kernel,
                       dim3(ceil_div(a.K, 64), a.R * a.S, ceil_div(ceil_div(a.C, 8), 4)),
                       dim3(256), 0, st, in0, in1, out, a);
  }
  return hipGetLastError();
}

}  // namespace fp16k
