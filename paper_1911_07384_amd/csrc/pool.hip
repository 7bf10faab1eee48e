// Pooling layers of ResNet-50 (Section 5.1 of arXiv:1911.07384): the 3x3
// stride-2 max pool after the stem and the global average pool before the
// classifier, with their backwards.
//
// Bandwidth-bound.  The NHWC path (C a multiple of 8) gives each thread eight
// channels of one position, so every access is a 16-byte vector (an 8-byte
// vector for the one-byte tap indices); NCHW and other channel counts take
// a per-element path.  Backwards are gathers (each input position collects
// from the windows that contain it), so no two threads write one element and
// no atomics are involved.  Every sum of binary16 terms here is exact in
// float64 (few enough terms; see the shape limits checked by the ABI), so
// the order of the additions does not matter and one rounding follows.

#include "kernels.hpp"

namespace fp16k {
namespace {

constexpr int kPT = 256;

// First tap of a window that lies inside the image (windows are never empty).
__device__ __forceinline__ int first_tap(int o, int st, int pad) {
  const int lo = o * st - pad;
  return lo < 0 ? -lo : 0;
}

__device__ __forceinline__ int64_t act_at(const PoolArgs& a, int n, int c, int h, int w) {
  return a.layout == 0 ? (((int64_t)n * a.H + h) * a.W + w) * a.C + c
                       : (((int64_t)n * a.C + c) * a.H + h) * a.W + w;
}
__device__ __forceinline__ int64_t out_at(const PoolArgs& a, int n, int c, int p, int q) {
  return a.layout == 0 ? (((int64_t)n * a.P + p) * a.Q + q) * a.C + c
                       : (((int64_t)n * a.C + c) * a.P + p) * a.Q + q;
}

// ---- max pooling forward --------------------------------------------------------

__global__ __launch_bounds__(kPT) void maxpool_fwd_vec(const h16* __restrict__ x,
                                                       h16* __restrict__ y,
                                                       uint8_t* __restrict__ idx, PoolArgs a) {
  const int CV = a.C / 8;
  const int64_t total = (int64_t)a.N * a.P * a.Q * CV;
  for (int64_t v = (int64_t)blockIdx.x * kPT + threadIdx.x; v < total;
       v += (int64_t)gridDim.x * kPT) {
    const int j = (int)(v % CV);
    int64_t r = v / CV;
    const int q = (int)(r % a.Q);
    r /= a.Q;
    const int p = (int)(r % a.P);
    const int n = (int)(r / a.P);
    // start from the window's first position inside the image, then scan
    // every position (the start itself is never strictly larger than itself)
    const int r0 = first_tap(p, a.sh, a.ph), s0 = first_tap(q, a.sw, a.pw);
    const h16* xb = x + ((int64_t)n * a.H * a.W) * a.C + j * 8;
    V8 win = load16(xb + ((int64_t)(p * a.sh - a.ph + r0) * a.W + (q * a.sw - a.pw + s0)) * a.C);
    float best[8];
    int tap[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      best[e] = to_f32(win.h[e]);
      tap[e] = r0 * a.S + s0;
    }
    for (int rr = r0; rr < a.R; ++rr) {
      const int h = p * a.sh - a.ph + rr;
      if (h >= a.H) break;
      for (int ss = s0; ss < a.S; ++ss) {
        const int w = q * a.sw - a.pw + ss;
        if (w >= a.W) break;
        const V8 xv = load16(xb + ((int64_t)h * a.W + w) * a.C);
        const int t = rr * a.S + ss;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float f = to_f32(xv.h[e]);
          const bool tk = pool_takes(best[e], f);
          best[e] = tk ? f : best[e];
          win.s[e] = tk ? xv.s[e] : win.s[e];
          tap[e] = tk ? t : tap[e];
        }
      }
    }
    uint32_t lo = 0, hi = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      lo |= (uint32_t)tap[e] << (8 * e);
      hi |= (uint32_t)tap[e + 4] << (8 * e);
    }
    store16(y + v * 8, win);
    *reinterpret_cast<uint2*>(idx + v * 8) = make_uint2(lo, hi);
  }
}

__global__ __launch_bounds__(kPT) void maxpool_fwd_gen(const h16* __restrict__ x,
                                                       h16* __restrict__ y,
                                                       uint8_t* __restrict__ idx, PoolArgs a) {
  const int64_t total = (int64_t)a.N * a.C * a.P * a.Q;
  for (int64_t o = (int64_t)blockIdx.x * kPT + threadIdx.x; o < total;
       o += (int64_t)gridDim.x * kPT) {
    int n, c, p, q;
    int64_t r = o;
    if (a.layout == 0) {
      c = (int)(r % a.C); r /= a.C; q = (int)(r % a.Q); r /= a.Q; p = (int)(r % a.P);
      n = (int)(r / a.P);
    } else {
      q = (int)(r % a.Q); r /= a.Q; p = (int)(r % a.P); r /= a.P; c = (int)(r % a.C);
      n = (int)(r / a.C);
    }
    const int r0 = first_tap(p, a.sh, a.ph), s0 = first_tap(q, a.sw, a.pw);
    h16 win = x[act_at(a, n, c, p * a.sh - a.ph + r0, q * a.sw - a.pw + s0)];
    float best = to_f32(win);
    int tap = r0 * a.S + s0;
    for (int rr = r0; rr < a.R; ++rr) {
      const int h = p * a.sh - a.ph + rr;
      if (h >= a.H) break;
      for (int ss = s0; ss < a.S; ++ss) {
        const int w = q * a.sw - a.pw + ss;
        if (w >= a.W) break;
        const h16 xv = x[act_at(a, n, c, h, w)];
        const float f = to_f32(xv);
        const bool tk = pool_takes(best, f);
        best = tk ? f : best;
        win = tk ? xv : win;
        tap = tk ? rr * a.S + ss : tap;
      }
    }
    y[o] = win;
    idx[o] = (uint8_t)tap;
  }
}

// ---- max pooling backward --------------------------------------------------------
// Output windows containing row h: p*sh - ph <= h <= p*sh - ph + R - 1.
__device__ __forceinline__ void window_range(int h, int pad, int R, int st, int P, int& p0,
                                             int& p1) {
  const int lo = h + pad - R + 1;
  p0 = lo <= 0 ? 0 : (lo + st - 1) / st;
  p1 = (h + pad) / st;
  if (p1 > P - 1) p1 = P - 1;
}

__global__ __launch_bounds__(kPT) void maxpool_bwd_vec(const uint8_t* __restrict__ idx,
                                                       const h16* __restrict__ dy,
                                                       h16* __restrict__ dx, PoolArgs a) {
  const int CV = a.C / 8;
  const int64_t total = (int64_t)a.N * a.H * a.W * CV;
  for (int64_t v = (int64_t)blockIdx.x * kPT + threadIdx.x; v < total;
       v += (int64_t)gridDim.x * kPT) {
    const int j = (int)(v % CV);
    int64_t r = v / CV;
    const int w = (int)(r % a.W);
    r /= a.W;
    const int h = (int)(r % a.H);
    const int n = (int)(r / a.H);
    int p0, p1, q0, q1;
    window_range(h, a.ph, a.R, a.sh, a.P, p0, p1);
    window_range(w, a.pw, a.S, a.sw, a.Q, q0, q1);
    double acc[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] = 0.0;
    for (int p = p0; p <= p1; ++p) {
      for (int q = q0; q <= q1; ++q) {
        const int t = (h - (p * a.sh - a.ph)) * a.S + (w - (q * a.sw - a.pw));
        const int64_t ov = (((int64_t)n * a.P + p) * a.Q + q) * CV + j;
        const uint64_t taps = *reinterpret_cast<const uint64_t*>(idx + ov * 8);
        const V8 g = load16(dy + ov * 8);
#pragma unroll
        for (int e = 0; e < 8; ++e)
          if ((int)((taps >> (8 * e)) & 0xFF) == t) acc[e] += (double)to_f32(g.h[e]);
      }
    }
    V8 o;
#pragma unroll
    for (int e = 0; e < 8; ++e) o.h[e] = dbl_to_h16(acc[e]);
    store16(dx + v * 8, o);
  }
}

// The 3x3 stride-2 pad-1 pool (the ResNet stem's): a thread owns a 2x2 block
// of input positions (rows 2a, 2a+1, columns 2b, 2b+1) and 8 channels.  The
// windows containing them are (p, q) in {a, a+1} x {b, b+1}; each window's
// taps and gradients are loaded once, all four before any is used (a window
// past the last row or column is loaded clamped and contributes nothing).
// Position (2a + i, 2b + j) receives from window (a + u, b + v) when u <= i
// and v <= j, at tap (1 + i - 2u) * 3 + (1 + j - 2v).  At most four binary16
// terms are added in float64, which is exact in any order.
__global__ __launch_bounds__(kPT) void maxpool_bwd_s2(const uint8_t* __restrict__ idx,
                                                      const h16* __restrict__ dy,
                                                      h16* __restrict__ dx, PoolArgs a) {
  const int CV = a.C / 8;
  const int HB = (a.H + 1) / 2, WB = (a.W + 1) / 2;
  const int64_t total = (int64_t)a.N * HB * WB * CV;
  for (int64_t v = (int64_t)blockIdx.x * kPT + threadIdx.x; v < total;
       v += (int64_t)gridDim.x * kPT) {
    const int j = (int)(v % CV);
    int64_t r = v / CV;
    const int b = (int)(r % WB);
    r /= WB;
    const int ab = (int)(r % HB);
    const int n = (int)(r / HB);
    uint64_t taps[2][2];
    V8 g[2][2];
    bool ok[2][2];
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int w = 0; w < 2; ++w) {
        const int p = ab + u, q = b + w;
        ok[u][w] = p < a.P && q < a.Q;
        const int pc = p < a.P ? p : a.P - 1, qc = q < a.Q ? q : a.Q - 1;
        const int64_t ov = (((int64_t)n * a.P + pc) * a.Q + qc) * CV + j;
        taps[u][w] = *reinterpret_cast<const uint64_t*>(idx + ov * 8);
        g[u][w] = load16(dy + ov * 8);
      }
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int h = 2 * ab + i;
#pragma unroll
      for (int jj = 0; jj < 2; ++jj) {
        const int wc = 2 * b + jj;
        double acc[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] = 0.0;
#pragma unroll
        for (int u = 0; u <= i; ++u)
#pragma unroll
          for (int w = 0; w <= jj; ++w) {
            const int t = (1 + i - 2 * u) * 3 + (1 + jj - 2 * w);
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              const bool hit = ok[u][w] && (int)((taps[u][w] >> (8 * e)) & 0xFF) == t;
              acc[e] += hit ? (double)to_f32(g[u][w].h[e]) : 0.0;
            }
          }
        if (h < a.H && wc < a.W) {
          V8 o;
#pragma unroll
          for (int e = 0; e < 8; ++e) o.h[e] = dbl_to_h16(acc[e]);
          store16(dx + ((((int64_t)n * a.H + h) * a.W + wc) * CV + j) * 8, o);
        }
      }
    }
  }
}

__global__ __launch_bounds__(kPT) void maxpool_bwd_gen(const uint8_t* __restrict__ idx,
                                                       const h16* __restrict__ dy,
                                                       h16* __restrict__ dx, PoolArgs a) {
  const int64_t total = (int64_t)a.N * a.C * a.H * a.W;
  for (int64_t i = (int64_t)blockIdx.x * kPT + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * kPT) {
    int n, c, h, w;
    int64_t r = i;
    if (a.layout == 0) {
      c = (int)(r % a.C); r /= a.C; w = (int)(r % a.W); r /= a.W; h = (int)(r % a.H);
      n = (int)(r / a.H);
    } else {
      w = (int)(r % a.W); r /= a.W; h = (int)(r % a.H); r /= a.H; c = (int)(r % a.C);
      n = (int)(r / a.C);
    }
    int p0, p1, q0, q1;
    window_range(h, a.ph, a.R, a.sh, a.P, p0, p1);
    window_range(w, a.pw, a.S, a.sw, a.Q, q0, q1);
    double acc = 0.0;
    for (int p = p0; p <= p1; ++p)
      for (int q = q0; q <= q1; ++q) {
        const int t = (h - (p * a.sh - a.ph)) * a.S + (w - (q * a.sw - a.pw));
        const int64_t o = out_at(a, n, c, p, q);
        if ((int)idx[o] == t) acc += (double)to_f32(dy[o]);
      }
    dx[i] = dbl_to_h16(acc);
  }
}

// ---- global average pooling ---------------------------------------------------------

// The average pools run in 64-thread workgroups.  The forward takes one
// thread per 4 channels of an image (ResNet-50's head: 1,024 waves, one per
// SIMD), its sum over the image pixel by pixel in float64 as one load at a
// time would give it, with 16 pixels' loads in flight.
constexpr int kAvgT = 64;

__global__ __launch_bounds__(kAvgT) void avgpool_fwd_vec(const h16* __restrict__ x,
                                                         h16* __restrict__ y, PoolArgs a) {
  const int CV = a.C / 4;
  const int HW = a.H * a.W;
  const int64_t total = (int64_t)a.N * CV;
  for (int64_t v = (int64_t)blockIdx.x * kAvgT + threadIdx.x; v < total;
       v += (int64_t)gridDim.x * kAvgT) {
    const int j = (int)(v % CV);
    const int n = (int)(v / CV);
    const h16* src = x + (int64_t)n * HW * a.C + j * 4;
    double acc[4] = {0.0, 0.0, 0.0, 0.0};
    for (int i0 = 0; i0 < HW; i0 += 16) {
      uint2 xv[16];
#pragma unroll
      for (int u = 0; u < 16; ++u)
        xv[u] = i0 + u < HW ? *reinterpret_cast<const uint2*>(src + (int64_t)(i0 + u) * a.C)
                            : make_uint2(0u, 0u);
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        if (i0 + u < HW) {
          const h16* h = reinterpret_cast<const h16*>(&xv[u]);
#pragma unroll
          for (int e = 0; e < 4; ++e) acc[e] += (double)to_f32(h[e]);
        }
      }
    }
    h16 o[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) o[e] = dbl_to_h16(acc[e] / (double)HW);
    *reinterpret_cast<uint2*>(y + v * 4) = *reinterpret_cast<const uint2*>(o);
  }
}

__global__ __launch_bounds__(kPT) void avgpool_fwd_gen(const h16* __restrict__ x,
                                                       h16* __restrict__ y, PoolArgs a) {
  const int64_t total = (int64_t)a.N * a.C;
  const int HW = a.H * a.W;
  for (int64_t o = (int64_t)blockIdx.x * kPT + threadIdx.x; o < total;
       o += (int64_t)gridDim.x * kPT) {
    const int c = (int)(o % a.C);
    const int n = (int)(o / a.C);
    double acc = 0.0;
    for (int h = 0; h < a.H; ++h)
      for (int w = 0; w < a.W; ++w) acc += (double)to_f32(x[act_at(a, n, c, h, w)]);
    y[o] = dbl_to_h16(acc / (double)HW);
  }
}

// backward: each thread divides its vector of dy once and stores it to every
// pixel of the image (19 -> 10 us at [128, 7, 7, 2048])
__global__ __launch_bounds__(kAvgT) void avgpool_bwd_vec(const h16* __restrict__ dy,
                                                         h16* __restrict__ dx, PoolArgs a) {
  const int CV = a.C / 8;
  const int HW = a.H * a.W;
  const int64_t total = (int64_t)a.N * CV;
  for (int64_t v = (int64_t)blockIdx.x * kAvgT + threadIdx.x; v < total;
       v += (int64_t)gridDim.x * kAvgT) {
    const int j = (int)(v % CV);
    const int n = (int)(v / CV);
    const V8 g = load16(dy + ((int64_t)n * a.C + j * 8));
    V8 o;
#pragma unroll
    for (int e = 0; e < 8; ++e) o.h[e] = dbl_to_h16((double)to_f32(g.h[e]) / (double)HW);
    h16* dst = dx + (int64_t)n * HW * a.C + j * 8;
    for (int i = 0; i < HW; ++i) store16(dst + (int64_t)i * a.C, o);
  }
}

__global__ __launch_bounds__(kPT) void avgpool_bwd_gen(const h16* __restrict__ dy,
                                                       h16* __restrict__ dx, PoolArgs a) {
  const int64_t total = (int64_t)a.N * a.C * a.H * a.W;
  const int HW = a.H * a.W;
  for (int64_t i = (int64_t)blockIdx.x * kPT + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * kPT) {
    int n, c;
    if (a.layout == 0) {
      c = (int)(i % a.C);
      n = (int)(i / ((int64_t)HW * a.C));
    } else {
      c = (int)((i / HW) % a.C);
      n = (int)(i / ((int64_t)HW * a.C));
    }
    dx[i] = dbl_to_h16((double)to_f32(dy[(int64_t)n * a.C + c]) / (double)HW);
  }
}

unsigned grid_for(int64_t items, int threads = kPT) {
  int64_t b = (items + threads - 1) / threads;
  if (b > 65536) b = 65536;
  if (b < 1) b = 1;
  return (unsigned)b;
}

bool vec_ok(const PoolArgs& a) { return a.layout == 0 && a.C % 8 == 0; }

}  // namespace

hipError_t launch_maxpool_fwd(const PoolArgs& a, const h16* x, h16* y, uint8_t* idx,
                              hipStream_t st) {
  if (vec_ok(a))
    hipLaunchKernelGGL(maxpool_fwd_vec, dim3(grid_for((int64_t)a.N * a.P * a.Q * (a.C / 8))),
                       dim3(kPT), 0, st, x, y, idx, a);
  else
    hipLaunchKernelGGL(maxpool_fwd_gen, dim3(grid_for((int64_t)a.N * a.C * a.P * a.Q)),
                       dim3(kPT), 0, st, x, y, idx, a);
  return hipGetLastError();
}

hipError_t launch_maxpool_bwd(const PoolArgs& a, const uint8_t* idx, const h16* dy, h16* dx,
                              hipStream_t st) {
  if (vec_ok(a) && a.R == 3 && a.S == 3 && a.sh == 2 && a.sw == 2 && a.ph == 1 && a.pw == 1)
    hipLaunchKernelGGL(maxpool_bwd_s2,
                       dim3(grid_for((int64_t)a.N * ((a.H + 1) / 2) * ((a.W + 1) / 2) * (a.C / 8))),
                       dim3(kPT), 0, st, idx, dy, dx, a);
  else if (vec_ok(a))
    hipLaunchKernelGGL(maxpool_bwd_vec, dim3(grid_for((int64_t)a.N * a.H * a.W * (a.C / 8))),
                       dim3(kPT), 0, st, idx, dy, dx, a);
  else
    hipLaunchKernelGGL(maxpool_bwd_gen, dim3(grid_for((int64_t)a.N * a.C * a.H * a.W)),
                       dim3(kPT), 0, st, idx, dy, dx, a);
  return hipGetLastError();
}

hipError_t launch_avgpool_fwd(const PoolArgs& a, const h16* x, h16* y, hipStream_t st) {
  if (vec_ok(a))
    hipLaunchKernelGGL(avgpool_fwd_vec, dim3(grid_for((int64_t)a.N * (a.C / 4), kAvgT)),
                       dim3(kAvgT), 0, st, x, y, a);
  else
    hipLaunchKernelGGL(avgpool_fwd_gen, dim3(grid_for((int64_t)a.N * a.C)), dim3(kPT), 0, st, x,
                       y, a);
  return hipGetLastError();
}

hipError_t launch_avgpool_bwd(const PoolArgs& a, const h16* dy, h16* dx, hipStream_t st) {
  if (vec_ok(a))
    hipLaunchKernelGGL(avgpool_bwd_vec, dim3(grid_for((int64_t)a.N * (a.C / 8), kAvgT)),
                       dim3(kAvgT), 0, st, dy, dx, a);
  else
    hipLaunchKernelGGL(avgpool_bwd_gen, dim3(grid_for((int64_t)a.N * a.C * a.H * a.W)),
                       dim3(kPT), 0, st, dy, dx, a);
  return hipGetLastError();
}

}  // namespace fp16k
