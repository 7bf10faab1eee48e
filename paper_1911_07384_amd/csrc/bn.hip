// Batch normalisation fused with the 0.25 output multiplier, the identity
// shortcut and ReLU (arXiv:1911.07384, Eq. 1-2 of Section 4.1; Section 4.2
// for the multiplier; statistics over the local batch, Section 5.1), and
// its backward.
//
// Forward = reduce (per-channel shifted sums of x and x^2), finalize (mean,
// rstd in float64 -> float32 stats), apply (declared float32 sequence):
//   a = fl(fl(s*gamma)*rstd); b = fl(s*beta); t = fl(x - mean);
//   v = fma(t, a, b); v = fl(v + r); y = rne16(relu(v)).
// Backward = reduce (S1 = sum g, T = sum g*(x - mean)), finalize (S2 =
// rstd*T = sum g*xhat, dgamma, dbeta, apply coefficients), apply (dx,
// dresidual).
//
// BN swap (Section 4.1; Geo::swap = 1): the shortcut joins before gamma,
//   u = s * (gamma * (xhat + r) + beta), applied as
//   sg = fl(s*gamma); w = fma(sg, r, b); v = fma(t, a, w); y = rne16(relu(v)),
// and the backward adds S3 = sum g*r to dgamma and sends gamma*g (rounded
// once) to the shortcut.
//
// Bandwidth-bound.  The NHWC path (C a power-of-two multiple of 8, at most
// 2048) gives each thread a fixed 8-channel chunk, so every access is a
// 16-byte vector and per-channel coefficients are computed once per thread.
// Other shapes and the NCHW layout use a generic per-element path.
// Reductions are float32 within a thread, combined in a fixed order within a
// block and in float64 across blocks: the result does not depend on timing.

#include "kernels.hpp"

namespace fp16k {
namespace {

constexpr int kT = 256;
// from this many channels on the vectorised reduces write block-major
// partials and the finalize takes 64 channels per block (else channel-major
// partials and one block per channel)
constexpr int kBmC = 256;

struct Geo {
  int64_t M;  // elements per channel
  int C, HW, layout;
  int swap;   // 1: the shortcut joins before gamma (BN swap)
};

// memory index of element j (0 <= j < M) of channel c
__device__ __forceinline__ int64_t geo_at(const Geo& g, int c, int64_t j) {
  if (g.layout == 0) return j * g.C + c;
  const int64_t n = j / g.HW;
  return (n * g.C + c) * g.HW + (j - n * g.HW);
}
// channel of memory index i
__device__ __forceinline__ int geo_chan(const Geo& g, int64_t i) {
  return g.layout == 0 ? (int)(i % g.C) : (int)((i / g.HW) % g.C);
}

struct Plan {
  bool vec;
  int CV, RB, G;
  int64_t rpb;  // rows (or elements) per block
};

Plan make_plan(const BnArgs& a) {
  Plan p{};
  const int64_t M = (int64_t)a.N * a.H * a.W;
  const int CV = a.C / 8;
  p.vec = a.layout == 0 && a.C % 8 == 0 && CV >= 1 && CV <= kT && (kT % CV) == 0;
  if (p.vec) {
    p.CV = CV;
    p.RB = kT / CV;
    // about four vectors per thread, at most two blocks per CU: more blocks
    // only add partial sums (on the conv2_x block's last BN backward 965
    // blocks took 27.4 us, 502 took 26.0)
    int64_t G = (M * CV + 4 * kT - 1) / (4 * kT);
    if (G > 512) G = 512;
    if (G < 1) G = 1;
    int64_t rpb = (M + G - 1) / G;
    rpb = (rpb + p.RB - 1) / p.RB * p.RB;
    p.rpb = rpb;
    p.G = (int)((M + rpb - 1) / rpb);
  } else {
    int64_t G = (M + 8 * kT - 1) / (8 * kT);
    if (G > 64) G = 64;
    if (G < 1) G = 1;
    p.rpb = (M + G - 1) / G;
    p.G = (int)((M + p.rpb - 1) / p.rpb);
  }
  return p;
}

// Mask of the ReLU: from the stored output when given, else recomputed bit
// for bit with the forward sequence.  The stored rne16(relu(v)) is positive
// exactly when v > 2^-25 (smaller positive values round to +0, 2^-25 itself
// ties to the even +0; a NaN compares false either way), so the recomputed
// mask is one float32 comparison.
__device__ __forceinline__ bool relu_mask(bool relu, bool has_y, h16 y, float x, const FwdCoef& k,
                                          bool has_r, float r, bool swap) {
  if (!relu) return true;
  if (has_y) return to_f32(y) > 0.0f;
  return fwd_value(x, k, has_r, r, false, swap) > 0x1p-25f;
}

// ---- block reduction of NS x 8 float32 partials per thread -------------------
// Thread t holds sums[v][8] (v < NS) for the 8 channels of chunk j = t % CV.
// Lanes of one wave that hold the same chunk are combined by a butterfly
// over the lane bits at or above log2(CV); the waves' totals (or, for
// CV > 64, the threads' own values) are then summed in a fixed order from
// LDS and written either block-major, out[(block * NS + v) * C + c] (bm:
// each block writes its sums as one contiguous run; from 256 channels on),
// or channel-major, out[(v * C + c) * G + block] (fewer channels: the
// finalize then spreads over one block per channel).  red: [8 * NS][kT].
template <int NS>
__device__ __forceinline__ void block_reduce_vec(float (&sums)[NS][8], float* red, int CV, int RB,
                                                 float* out, bool bm) {
  const int t = threadIdx.x;
  const int lane = t & 63;
  int groups;
  if (CV <= 64) {
    for (int off = CV; off < 64; off <<= 1) {
#pragma unroll
      for (int v = 0; v < NS; ++v)
#pragma unroll
        for (int e = 0; e < 8; ++e) sums[v][e] += __shfl_xor(sums[v][e], off, 64);
    }
    groups = kT / 64;
    if (lane < CV) {
      const int slot = (t >> 6) * CV + lane;
#pragma unroll
      for (int v = 0; v < NS; ++v)
#pragma unroll
        for (int e = 0; e < 8; ++e) red[(v * 8 + e) * kT + slot] = sums[v][e];
    }
  } else {
    groups = RB;
#pragma unroll
    for (int v = 0; v < NS; ++v)
#pragma unroll
      for (int e = 0; e < 8; ++e) red[(v * 8 + e) * kT + t] = sums[v][e];
  }
  __syncthreads();
  const int C = CV * 8;
  for (int idx = t; idx < 8 * NS * CV; idx += kT) {
    const int ve = idx / CV, j = idx - ve * CV;
    float acc = red[ve * kT + j];
    for (int gi = 1; gi < groups; ++gi) acc += red[ve * kT + gi * CV + j];
    const int v = ve >> 3, e = ve & 7;
    if (bm)
      out[((int64_t)blockIdx.x * NS + v) * C + j * 8 + e] = acc;
    else
      out[((int64_t)v * C + j * 8 + e) * gridDim.x + blockIdx.x] = acc;
  }
}

// ---- forward reduce ----------------------------------------------------------
// Sums of (x - K_c) and (x - K_c)^2 with K_c = the channel's first element
// (a shift that keeps the variance free of cancellation).

__global__ __launch_bounds__(kT) void bn_fwd_reduce_vec(const h16* __restrict__ x, Geo g, int CV,
                                                        int RB, int64_t rpb, float* ws) {
  __shared__ float red[16 * kT];
  const int t = threadIdx.x;
  const int j = t % CV;
  const int64_t row0 = (int64_t)blockIdx.x * rpb;
  int64_t row1 = row0 + rpb;
  if (row1 > g.M) row1 = g.M;
  const V8 kv = load16(x + j * 8);
  float sh[8], sums[2][8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    sh[e] = to_f32(kv.h[e]);
    sums[0][e] = 0.0f;
    sums[1][e] = 0.0f;
  }
  // four rows in flight per thread, the sums row by row; the step count is
  // the block's, and a row past the block's last is loaded clamped (in
  // bounds) and adds exact zeros, so no load waits behind a condition
  const int64_t rt = row0 + t / CV;
  const int64_t nsteps = (row1 - row0 + RB - 1) / RB;
  for (int64_t i = 0; i < nsteps; i += 4) {
    V8 v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int64_t row = rt + (i + u) * RB;
      v[u] = load16(x + (row < row1 ? row : row1 - 1) * g.C + j * 8);
    }
    __builtin_amdgcn_sched_barrier(0);  // every load issued before the first use
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const bool ok = rt + (i + u) * RB < row1;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float d = ok ? to_f32(v[u].h[e]) - sh[e] : 0.0f;
        sums[0][e] += d;
        sums[1][e] = __builtin_fmaf(d, d, sums[1][e]);
      }
    }
  }
  block_reduce_vec<2>(sums, red, CV, RB, ws, g.C >= kBmC);
}

// Tree reduction of NS values per thread over the block (fixed order).
// red: [NS][kT].
template <int NS>
__device__ __forceinline__ void block_reduce_1(float (&v)[NS], float* red) {
  const int t = threadIdx.x;
#pragma unroll
  for (int i = 0; i < NS; ++i) red[i * kT + t] = v[i];
  __syncthreads();
  for (int w = kT / 2; w > 0; w >>= 1) {
    if (t < w) {
#pragma unroll
      for (int i = 0; i < NS; ++i) red[i * kT + t] += red[i * kT + t + w];
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < NS; ++i) v[i] = red[i * kT];
}

__global__ __launch_bounds__(kT) void bn_fwd_reduce_gen(const h16* __restrict__ x, Geo g,
                                                        int64_t rpb, float* ws) {
  __shared__ float red[2 * kT];
  const int c = blockIdx.y;
  const int64_t j0 = (int64_t)blockIdx.x * rpb;
  int64_t j1 = j0 + rpb;
  if (j1 > g.M) j1 = g.M;
  const float sh = to_f32(x[geo_at(g, c, 0)]);
  float s1 = 0.0f, s2 = 0.0f;
  for (int64_t j = j0 + threadIdx.x; j < j1; j += kT) {
    const float d = to_f32(x[geo_at(g, c, j)]) - sh;
    s1 += d;
    s2 = __builtin_fmaf(d, d, s2);
  }
  float v[2] = {s1, s2};
  block_reduce_1<2>(v, red);
  if (threadIdx.x == 0) {
    ws[(int64_t)c * gridDim.x + blockIdx.x] = v[0];
    ws[((int64_t)g.C + c) * gridDim.x + blockIdx.x] = v[1];
  }
}

// Sum of the G channel-major partials of channel c in float64: each lane of
// one wave takes every 64th partial, in index order, then a butterfly over
// the wave (a fixed order, so the total does not depend on timing).  The
// partials of a lane are loaded 16 at a time before any is added, so one
// memory round trip covers up to 1,024 partials.
__device__ __forceinline__ void channel_sums(const float* ws1, const float* ws2, int c, int G,
                                             double& S1, double& S2) {
  const int t = threadIdx.x;
  double a = 0.0, b = 0.0;
  const float* p1 = ws1 + (int64_t)c * G;
  const float* p2 = ws2 + (int64_t)c * G;
  constexpr int U = 16;
  for (int j = t; j < G; j += 64 * U) {
    float u1[U], u2[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      // unconditional loads from a clamped index (a load under a lane
      // condition would be waited for before the next one is issued)
      const int i = j + 64 * u < G ? j + 64 * u : G - 1;
      u1[u] = p1[i];
      u2[u] = p2[i];
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const bool ok = j + 64 * u < G;
      a += ok ? (double)u1[u] : 0.0;
      b += ok ? (double)u2[u] : 0.0;
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    a += __shfl_xor(a, off, 64);
    b += __shfl_xor(b, off, 64);
  }
  S1 = a;
  S2 = b;
}

// Sums over the G blocks of the block-major partials part[(b * NS + v) * C + c]
// in float64, for the 64 channels of this block (lane = channel): wave w
// takes the blocks w, w + kFinW, w + 2 kFinW, ... in order (kFinU loads of
// each value in flight, clamped in bounds, so every row read is 256
// contiguous bytes), then the first wave adds the kFinW wave sums in order.
// A fixed order, so the result does not depend on timing.
constexpr int kFinW = 16, kFinU = 8;

template <int NS>
__device__ __forceinline__ void group_sums(const float* part, int C, int G, int c, bool live,
                                           double (&S)[NS]) {
  __shared__ double red[NS][kFinW][64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int cc = live ? c : 0;
  double acc[NS];
#pragma unroll
  for (int v = 0; v < NS; ++v) acc[v] = 0.0;
  for (int b0 = w; b0 < G; b0 += kFinW * kFinU) {
    float u[kFinU][NS];
#pragma unroll
    for (int k = 0; k < kFinU; ++k) {
      const int b = b0 + kFinW * k < G ? b0 + kFinW * k : G - 1;
#pragma unroll
      for (int v = 0; v < NS; ++v) u[k][v] = part[((int64_t)b * NS + v) * C + cc];
    }
#pragma unroll
    for (int k = 0; k < kFinU; ++k) {
      const bool ok = b0 + kFinW * k < G;
#pragma unroll
      for (int v = 0; v < NS; ++v) acc[v] += ok ? (double)u[k][v] : 0.0;
    }
  }
#pragma unroll
  for (int v = 0; v < NS; ++v) red[v][w][lane] = acc[v];
  __syncthreads();
#pragma unroll
  for (int v = 0; v < NS; ++v) {
    double t = 0.0;
    for (int i = 0; i < kFinW; ++i) t += red[v][i][lane];
    S[v] = t;
  }
}

__device__ __forceinline__ void fwd_stats(const h16* x, Geo g, int c, double S1, double S2,
                                          float eps, float* stats) {
  const double sh = (double)to_f32(x[geo_at(g, c, 0)]);
  const double md = S1 / (double)g.M;
  double var = S2 / (double)g.M - md * md;
  if (var < 0.0) var = 0.0;
  stats[c] = (float)(sh + md);
  stats[g.C + c] = (float)(1.0 / __builtin_sqrt(var + (double)eps));
}

// channel-major partials: one 64-thread block per channel
__global__ __launch_bounds__(64) void bn_fwd_finalize(const h16* __restrict__ x, Geo g, int G,
                                                      const float* ws, float eps, float* stats) {
  const int c = blockIdx.x;
  double S1, S2;
  channel_sums(ws, ws + (int64_t)g.C * G, c, G, S1, S2);
  if (threadIdx.x != 0) return;
  fwd_stats(x, g, c, S1, S2, eps, stats);
}

// block-major partials: one block per 64 channels
__global__ __launch_bounds__(64 * kFinW) void bn_fwd_finalize_bm(const h16* __restrict__ x, Geo g,
                                                                 int G, const float* ws, float eps,
                                                                 float* stats) {
  const int c = blockIdx.x * 64 + (threadIdx.x & 63);
  const bool live = c < g.C;
  double S[2];
  group_sums<2>(ws, g.C, G, c, live, S);
  if (threadIdx.x >= 64 || !live) return;
  fwd_stats(x, g, c, S[0], S[1], eps, stats);
}

// Statistics from the records a convolution's epilogue wrote ([nb][3][C]:
// record b covers the 128-row tiles b, b + nb, b + 2nb, ... (one tile each
// where nb is the tile count) and holds per channel c a shift K_b (one of its
// values) and the sums of (y - K_b) and (y - K_b)^2 over its n_b rows).
// About K_0:
//   S1 = sum_b s1_b + n_b d_b,  S2 = sum_b s2_b + 2 d_b s1_b + n_b d_b^2,
// d_b = K_b - K_0, in float64.  Up to kBandOne records: bn_band_finalize, one
// 256-thread block per channel; thread t takes records t, t + 256, ... in
// order (the loads of four of them in flight), then the block's fixed-order
// reduction.  More records, in two kernels:
//  - bn_band_slices: block (channel group of 64, slice s) sums the records
//    [s*kBandRps, (s+1)*kBandRps) of its 64 channels (one lane per channel, so
//    every record row is read with 256-byte coalesced loads; wave w takes every
//    4th record from the w-th, all of them in flight; the waves then in order)
//    and writes the slice sums channel-major, [2][C][nslice] float64;
//  - bn_band_combine: one wave per channel adds its slices (lane t takes every
//    64th in order, then a butterfly) and writes mean and 1/sqrt(var + eps).
// Every sum has a fixed order, so the statistics do not depend on timing.
constexpr int kBandOne = 2048;
constexpr int kBandRps = 32;  // records per slice: 8 per wave

// Rows of record j of nb over M rows: 128 per tile it covers, less the
// last tile's missing rows where that tile is its.
__device__ __forceinline__ int64_t band_rows(int64_t M, int nb, int j) {
  const int64_t nt = (M + 127) / 128;
  if (j >= nt) return 0;
  int64_t r = 128 * ((nt - 1 - j) / nb + 1);
  if (j == (nt - 1) % nb) r -= 128 * nt - M;
  return r;
}

// One record's terms; a record past the last adds exact zeros, so that its
// (clamped, in-bounds) loads stay unconditional and in flight together.
__device__ __forceinline__ void band_term_if(bool ok, int64_t rows, float k, double K0, float s1,
                                             float s2, double& a, double& b) {
  const double n = ok ? (double)rows : 0.0;
  const double d = ok ? (double)k - K0 : 0.0;
  const double t1 = ok ? (double)s1 : 0.0, t2 = ok ? (double)s2 : 0.0;
  a += t1 + n * d;
  b += t2 + 2.0 * d * t1 + n * d * d;
}

__device__ __forceinline__ void band_stats(double a, double b, double K0, Geo g, float eps,
                                           int c, float* stats) {
  const double md = a / (double)g.M;
  double var = b / (double)g.M - md * md;
  if (var < 0.0) var = 0.0;
  stats[c] = (float)(K0 + md);
  stats[g.C + c] = (float)(1.0 / __builtin_sqrt(var + (double)eps));
}

__global__ __launch_bounds__(256) void bn_band_finalize(const float* __restrict__ part, int nb,
                                                        Geo g, float eps, float* stats) {
  __shared__ double red[2][4];
  const int c = blockIdx.x;
  const int t = threadIdx.x;
  const int64_t C3 = (int64_t)3 * g.C;
  const double K0 = (double)part[c];
  double a = 0.0, b = 0.0;
  constexpr int U = 4;
  for (int j0 = t; j0 < nb; j0 += 256 * U) {
    float k[U], s1[U], s2[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int j = j0 + 256 * u;
      const float* rec = part + (int64_t)(j < nb ? j : nb - 1) * C3 + c;
      k[u] = rec[0];
      s1[u] = rec[g.C];
      s2[u] = rec[2 * g.C];
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int j = j0 + 256 * u;
      band_term_if(j < nb, band_rows(g.M, nb, j), k[u], K0, s1[u], s2[u], a, b);
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    a += __shfl_xor(a, off, 64);
    b += __shfl_xor(b, off, 64);
  }
  if ((t & 63) == 0) {
    red[0][t >> 6] = a;
    red[1][t >> 6] = b;
  }
  __syncthreads();
  if (t != 0) return;
  band_stats(((red[0][0] + red[0][1]) + red[0][2]) + red[0][3],
             ((red[1][0] + red[1][1]) + red[1][2]) + red[1][3], K0, g, eps, c, stats);
}

__global__ __launch_bounds__(256) void bn_band_slices(const float* __restrict__ part, int nb,
                                                      Geo g, double* __restrict__ sl, int ns) {
  __shared__ double red[2][4][64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int c = blockIdx.x * 64 + lane;
  const int s = blockIdx.y;
  const int64_t C3 = (int64_t)3 * g.C;
  double a = 0.0, b = 0.0;
  if (c < g.C) {
    const double K0 = (double)part[c];
    constexpr int U = kBandRps / 4;
    float k[U], s1[U], s2[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int j = s * kBandRps + w + 4 * u;
      const float* rec = part + (int64_t)(j < nb ? j : nb - 1) * C3 + c;
      k[u] = rec[0];
      s1[u] = rec[g.C];
      s2[u] = rec[2 * g.C];
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int j = s * kBandRps + w + 4 * u;
      band_term_if(j < nb, band_rows(g.M, nb, j), k[u], K0, s1[u], s2[u], a, b);
    }
  }
  red[0][w][lane] = a;
  red[1][w][lane] = b;
  __syncthreads();
  if (w != 0 || c >= g.C) return;
  const double A = ((red[0][0][lane] + red[0][1][lane]) + red[0][2][lane]) + red[0][3][lane];
  const double B = ((red[1][0][lane] + red[1][1][lane]) + red[1][2][lane]) + red[1][3][lane];
  sl[(int64_t)c * ns + s] = A;
  sl[((int64_t)g.C + c) * ns + s] = B;
}

__global__ __launch_bounds__(64) void bn_band_combine(const float* __restrict__ part,
                                                      const double* __restrict__ sl, int ns,
                                                      Geo g, float eps, float* stats) {
  const int c = blockIdx.x;
  const int t = threadIdx.x;
  const double* pa = sl + (int64_t)c * ns;
  const double* pb = sl + ((int64_t)g.C + c) * ns;
  constexpr int U = 8;
  double a = 0.0, b = 0.0;
  for (int j = t; j < ns; j += 64 * U) {
    double ua[U], ub[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i = j + 64 * u < ns ? j + 64 * u : ns - 1;
      ua[u] = pa[i];
      ub[u] = pb[i];
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const bool ok = j + 64 * u < ns;
      a += ok ? ua[u] : 0.0;
      b += ok ? ub[u] : 0.0;
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    a += __shfl_xor(a, off, 64);
    b += __shfl_xor(b, off, 64);
  }
  if (t != 0) return;
  band_stats(a, b, (double)part[c], g, eps, c, stats);
}

// ---- forward apply -------------------------------------------------------------

// Variants of the vectorised kernels are template bits, so that every load
// of a step is issued without a condition: a load behind a branch (on a lane
// or on a runtime flag) made the compiler wait for all loads in flight before
// the next one.
//   kSwap: BN swap; kRelu: ReLU; kMaskY: the backward takes the ReLU mask from
//   the stored output y; kLoadR: the shortcut r is read; kDres: the backward
//   writes the shortcut gradient; kMaskB: the backward takes the ReLU mask
//   from the bits the forward kept; kKeepF: the forward apply keeps them (one
//   byte per 16-byte vector of y, bit e = [y element e > 0]).
constexpr int kSwap = 1, kRelu = 2, kMaskY = 4, kLoadR = 8, kDres = 16, kMaskB = 32, kKeepF = 64;

// Each block takes runs of kApplyU * kT consecutive 16-byte vectors; a thread
// loads its kApplyU vectors (and residual vectors) before it stores any, so
// several loads per thread are in flight.  The run loop is the block's; a
// vector past the end is loaded clamped (in bounds) and not stored.  y may
// equal x: every element is read and then written by the same thread (a
// clamped load may read an element another lane rewrites; its value is
// discarded).
constexpr int kApplyU = 4;

template <int MODE>
__global__ __launch_bounds__(kT) void bn_fwd_apply_vec(const h16* x, const h16* __restrict__ gamma,
                                                       const h16* __restrict__ beta, const h16* res,
                                                       h16* y, const float* __restrict__ stats,
                                                       Geo g, int CV, float s,
                                                       uint8_t* __restrict__ mout) {
  constexpr bool SWAP = MODE & kSwap, RELU = MODE & kRelu, HAS_R = MODE & kLoadR,
                 KEEP = MODE & kKeepF;
  const int t = threadIdx.x;
  const int j = t % CV;  // run starts and kT are multiples of CV
  FwdCoef k[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) k[e] = fwd_coef(stats, gamma, beta, g.C, j * 8 + e, s);
  const int64_t nvec = g.M * CV;
  constexpr int64_t RUN = (int64_t)kApplyU * kT;
  for (int64_t run = (int64_t)blockIdx.x * RUN; run < nvec; run += (int64_t)gridDim.x * RUN) {
    V8 xv[kApplyU], rv[kApplyU];
#pragma unroll
    for (int u = 0; u < kApplyU; ++u) {
      const int64_t v = run + t + u * kT;
      const int64_t vc = v < nvec ? v : nvec - 1;
      xv[u] = load16(x + vc * 8);
      if (HAS_R) rv[u] = load16(res + vc * 8);
    }
    __builtin_amdgcn_sched_barrier(0);  // every load issued before the first use
#pragma unroll
    for (int u = 0; u < kApplyU; ++u) {
      const int64_t v = run + t + u * kT;
      V8 out;
      uint32_t bits = 0;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        out.h[e] = to_h16(fwd_value(to_f32(xv[u].h[e]), k[e], HAS_R,
                                    HAS_R ? to_f32(rv[u].h[e]) : 0.0f, RELU, SWAP));
        if (KEEP) bits |= (uint32_t)(to_f32(out.h[e]) > 0.0f) << e;
      }
      if (v < nvec) {
        store16(y + v * 8, out);
        if (KEEP) mout[v] = (uint8_t)bits;
      }
    }
  }
}

__global__ __launch_bounds__(kT) void bn_fwd_apply_gen(const h16* x, const h16* __restrict__ gamma,
                                                       const h16* __restrict__ beta, const h16* res,
                                                       h16* y, const float* __restrict__ stats,
                                                       Geo g, float s, int relu) {
  const int64_t total = g.M * g.C;
  for (int64_t i = (int64_t)blockIdx.x * kT + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * kT) {
    const int c = geo_chan(g, i);
    const FwdCoef k = fwd_coef(stats, gamma, beta, g.C, c, s);
    y[i] = to_h16(fwd_value(to_f32(x[i]), k, res != nullptr, res ? to_f32(res[i]) : 0.0f,
                            relu != 0, g.swap != 0));
  }
}

// ---- backward reduce -----------------------------------------------------------

// S1 = sum g, T = sum g*(x - mean); with the BN swap also S3 = sum g*r.
template <int MODE>
__global__ __launch_bounds__(kT) void bn_bwd_reduce_vec(const h16* __restrict__ x,
                                                        const h16* __restrict__ y,
                                                        const h16* __restrict__ dy,
                                                        const h16* __restrict__ gamma,
                                                        const h16* __restrict__ beta,
                                                        const h16* __restrict__ res,
                                                        const float* __restrict__ stats, Geo g,
                                                        int CV, int RB, int64_t rpb, float s,
                                                        float* ws, uint8_t* __restrict__ mbits) {
  constexpr bool SWAP = MODE & kSwap, RELU = MODE & kRelu, MASK_Y = MODE & kMaskY,
                 LOAD_R = MODE & kLoadR, MASK_B = MODE & kMaskB;
  // a mask recomputed from the shortcut is kept, one bit per element and one
  // byte per 16-byte vector (its index in x), so the apply reads that byte
  // instead of the shortcut's 16 bytes; with MASK_B the forward kept it and
  // it is read here (mbits is then the caller's mask, only read)
  constexpr bool KEEP_M = LOAD_R && RELU && !MASK_Y;
  constexpr int NS = SWAP ? 3 : 2;
  __shared__ float red[8 * NS * kT];
  const int t = threadIdx.x;
  const int j = t % CV;
  const int64_t row0 = (int64_t)blockIdx.x * rpb;
  int64_t row1 = row0 + rpb;
  if (row1 > g.M) row1 = g.M;
  FwdCoef k[8];
  float sums[NS][8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    k[e] = fwd_coef(stats, gamma, beta, g.C, j * 8 + e, s);
#pragma unroll
    for (int v = 0; v < NS; ++v) sums[v][e] = 0.0f;
  }
  // one row per step, the next row loaded before this one is summed (two rows
  // in flight); the step count is the block's, and a row past the block's
  // last is loaded clamped (in bounds) and adds exact zeros
  struct Row {
    V8 x, d, y, r;
    uint32_t mb;
  };
  const int64_t rt = row0 + t / CV;
  const int64_t nsteps = (row1 - row0 + RB - 1) / RB;
  auto load_row = [&](Row& b, int64_t i) {
    int64_t row = rt + i * RB;
    if (row >= row1) row = row1 - 1;
    const int64_t off = row * g.C + j * 8;
    b.x = load16(x + off);
    b.d = load16(dy + off);
    if (MASK_Y) b.y = load16(y + off);
    if (LOAD_R) b.r = load16(res + off);
    if (MASK_B) b.mb = mbits[row * CV + j];
  };
  auto sum_row = [&](const Row& b, int64_t i) {
    const bool ok = rt + i * RB < row1;
    uint32_t bits = 0;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float xf = to_f32(b.x.h[e]);
      const float rf = LOAD_R ? to_f32(b.r.h[e]) : 0.0f;
      const bool m = MASK_B ? ((b.mb >> e) & 1u) != 0
                            : relu_mask(RELU, MASK_Y, MASK_Y ? b.y.h[e] : (h16)0.0f, xf, k[e],
                                        LOAD_R, rf, SWAP);
      bits |= (uint32_t)m << e;
      const float gg = ok && m ? s * to_f32(b.d.h[e]) : 0.0f;
      const float xt = ok ? xf - k[e].mean : 0.0f;
      sums[0][e] += gg;
      sums[1][e] = __builtin_fmaf(gg, xt, sums[1][e]);
      if (SWAP) sums[NS - 1][e] = __builtin_fmaf(gg, ok ? rf : 0.0f, sums[NS - 1][e]);
    }
    if (KEEP_M && ok) mbits[(rt + i * RB) * CV + j] = (uint8_t)bits;
  };
  Row ra, rb;
  load_row(ra, 0);
  for (int64_t i = 0; i < nsteps; i += 2) {
    load_row(rb, i + 1);
    __builtin_amdgcn_sched_barrier(0);  // the next row's loads ahead of this row's sums
    sum_row(ra, i);
    load_row(ra, i + 2);
    __builtin_amdgcn_sched_barrier(0);
    sum_row(rb, i + 1);
  }
  block_reduce_vec<NS>(sums, red, CV, RB, ws, g.C >= kBmC);
}

__global__ __launch_bounds__(kT) void bn_bwd_reduce_gen(const h16* __restrict__ x,
                                                        const h16* __restrict__ y,
                                                        const h16* __restrict__ dy,
                                                        const h16* __restrict__ gamma,
                                                        const h16* __restrict__ beta,
                                                        const h16* __restrict__ res,
                                                        const float* __restrict__ stats, Geo g,
                                                        int64_t rpb, float s, int relu, float* ws) {
  __shared__ float red[3 * kT];
  const int c = blockIdx.y;
  const int64_t j0 = (int64_t)blockIdx.x * rpb;
  int64_t j1 = j0 + rpb;
  if (j1 > g.M) j1 = g.M;
  const FwdCoef k = fwd_coef(stats, gamma, beta, g.C, c, s);
  const bool swap = g.swap != 0;
  const bool has_y = y != nullptr, has_r = res != nullptr && !has_y && relu;
  const bool load_r = has_r || swap;
  float v[3] = {0.0f, 0.0f, 0.0f};
  for (int64_t j = j0 + threadIdx.x; j < j1; j += kT) {
    const int64_t i = geo_at(g, c, j);
    const float xf = to_f32(x[i]);
    const float rf = load_r ? to_f32(res[i]) : 0.0f;
    const bool m = relu_mask(relu != 0, has_y, has_y ? y[i] : (h16)0.0f, xf, k, has_r, rf, swap);
    const float gg = m ? s * to_f32(dy[i]) : 0.0f;
    const float xt = xf - k.mean;
    v[0] += gg;
    v[1] = __builtin_fmaf(gg, xt, v[1]);
    v[2] = __builtin_fmaf(gg, rf, v[2]);
  }
  block_reduce_1<3>(v, red);
  if (threadIdx.x == 0) {
    const int64_t G = gridDim.x;
    for (int q = 0; q < (swap ? 3 : 2); ++q) ws[((int64_t)q * g.C + c) * G + blockIdx.x] = v[q];
  }
}

// S2 = rstd*T = sum g*xhat; dbeta = S1, dgamma = S2 (+ S3 with the BN swap),
// one rounding from float64; apply coefficients A = gamma*rstd, B = S1/M and
// D = rstd*S2/M for dx = A * (g - ((x - mean)*D + B)), which is
// A * (g - (xhat*S2/M + S1/M)).  One block per 64 channels (NS = 3 partial
// sums with the BN swap, else 2).
__device__ __forceinline__ void bwd_coef(Geo g, int c, double S1, double T, double S3,
                                         const h16* gamma, const float* stats, h16* dgamma,
                                         h16* dbeta, float* coef) {
  const double rstd = (double)stats[g.C + c];
  const double S2 = rstd * T;
  dbeta[c] = dbl_to_h16(S1);
  dgamma[c] = dbl_to_h16(S2 + S3);
  coef[c] = to_f32(gamma[c]) * stats[g.C + c];
  coef[g.C + c] = (float)(S1 / (double)g.M);
  coef[2 * g.C + c] = (float)(rstd * S2 / (double)g.M);
}

// channel-major partials: one 64-thread block per channel
__global__ __launch_bounds__(64) void bn_bwd_finalize(Geo g, int G, const float* ws,
                                                      const h16* __restrict__ gamma,
                                                      const float* __restrict__ stats, h16* dgamma,
                                                      h16* dbeta, float* coef) {
  const int c = blockIdx.x;
  const int64_t CG = (int64_t)g.C * G;
  double S1, T, S3 = 0.0, unused;
  channel_sums(ws, ws + CG, c, G, S1, T);
  if (g.swap) channel_sums(ws + 2 * CG, ws + 2 * CG, c, G, S3, unused);
  if (threadIdx.x != 0) return;
  bwd_coef(g, c, S1, T, S3, gamma, stats, dgamma, dbeta, coef);
}

// block-major partials (NS = 3 with the BN swap, else 2): one block per 64
// channels
template <int NS>
__global__ __launch_bounds__(64 * kFinW) void bn_bwd_finalize_bm(Geo g, int G, const float* ws,
                                                                 const h16* __restrict__ gamma,
                                                                 const float* __restrict__ stats,
                                                                 h16* dgamma, h16* dbeta,
                                                                 float* coef) {
  const int c = blockIdx.x * 64 + (threadIdx.x & 63);
  const bool live = c < g.C;
  double S[NS];
  group_sums<NS>(ws, g.C, G, c, live, S);
  if (threadIdx.x >= 64 || !live) return;
  bwd_coef(g, c, S[0], S[1], NS == 3 ? S[NS - 1] : 0.0, gamma, stats, dgamma, dbeta, coef);
}

// ---- backward apply ------------------------------------------------------------

template <int MODE>
__global__ __launch_bounds__(kT) void bn_bwd_apply_vec(const h16* x, const h16* y, const h16* dy,
                                                       const h16* __restrict__ gamma,
                                                       const h16* __restrict__ beta, const h16* res,
                                                       const float* __restrict__ stats,
                                                       const float* __restrict__ coef, Geo g,
                                                       int CV, float s,
                                                       const uint8_t* __restrict__ mbits, h16* dx,
                                                       h16* dres) {
  constexpr bool SWAP = MODE & kSwap, RELU = MODE & kRelu, MASK_Y = MODE & kMaskY,
                 DRES = MODE & kDres;
  // the ReLU mask recomputed from x and the shortcut was kept by the reduce,
  // or by the forward (kMaskB): one byte per vector instead of the
  // shortcut's 16
  constexpr bool NEED_R = ((MODE & kLoadR) && RELU && !MASK_Y) || (MODE & kMaskB);
  const int t = threadIdx.x;
  const int j = t % CV;  // run starts and kT are multiples of CV
  FwdCoef k[8];
  float A[8], B[8], D[8], gam[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int c = j * 8 + e;
    k[e] = fwd_coef(stats, gamma, beta, g.C, c, s);
    A[e] = coef[c];
    B[e] = coef[g.C + c];
    D[e] = coef[2 * g.C + c];
    gam[e] = to_f32(gamma[c]);
  }
  const int64_t nvec = g.M * CV;
  constexpr int U = kApplyU / 2;  // vectors per thread and run: 2 to 4 loads each
  constexpr int64_t RUN = (int64_t)U * kT;
  for (int64_t run = (int64_t)blockIdx.x * RUN; run < nvec; run += (int64_t)gridDim.x * RUN) {
    V8 xv[U], dv[U], yv[U];
    uint32_t mb[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t v = run + t + u * kT;
      const int64_t vc = v < nvec ? v : nvec - 1;
      xv[u] = load16(x + vc * 8);
      dv[u] = load16(dy + vc * 8);
      if (MASK_Y) yv[u] = load16(y + vc * 8);
      if (NEED_R) mb[u] = mbits[vc];
    }
    __builtin_amdgcn_sched_barrier(0);  // every load issued before the first use
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t v = run + t + u * kT;
      V8 o, od;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float xf = to_f32(xv[u].h[e]);
        const bool m = NEED_R ? ((mb[u] >> e) & 1u) != 0
                              : relu_mask(RELU, MASK_Y, MASK_Y ? yv[u].h[e] : (h16)0.0f, xf, k[e],
                                          false, 0.0f, SWAP);
        const float gg = m ? s * to_f32(dv[u].h[e]) : 0.0f;
        o.h[e] = to_h16(A[e] * (gg - __builtin_fmaf(xf - k[e].mean, D[e], B[e])));
        if (SWAP)
          od.h[e] = to_h16(gam[e] * gg);
        else
          od.s[e] = m ? dv[u].s[e] : (uint16_t)0;
      }
      if (v < nvec) {
        store16(dx + v * 8, o);
        if (DRES) store16(dres + v * 8, od);
      }
    }
  }
}

__global__ __launch_bounds__(kT) void bn_bwd_apply_gen(const h16* x, const h16* y, const h16* dy,
                                                       const h16* __restrict__ gamma,
                                                       const h16* __restrict__ beta, const h16* res,
                                                       const float* __restrict__ stats,
                                                       const float* __restrict__ coef, Geo g,
                                                       float s, int relu, h16* dx, h16* dres) {
  const int64_t total = g.M * g.C;
  const bool swap = g.swap != 0;
  const bool has_y = y != nullptr, has_r = res != nullptr && !has_y && relu;
  for (int64_t i = (int64_t)blockIdx.x * kT + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * kT) {
    const int c = geo_chan(g, i);
    const FwdCoef k = fwd_coef(stats, gamma, beta, g.C, c, s);
    const float xf = to_f32(x[i]);
    const h16 dyv = dy[i];
    const bool m = relu_mask(relu != 0, has_y, has_y ? y[i] : (h16)0.0f, xf, k, has_r,
                             has_r ? to_f32(res[i]) : 0.0f, swap);
    const float gg = m ? s * to_f32(dyv) : 0.0f;
    dx[i] = to_h16(coef[c] * (gg - __builtin_fmaf(xf - k.mean, coef[2 * g.C + c], coef[g.C + c])));
    if (dres) dres[i] = swap ? to_h16(to_f32(gamma[c]) * gg) : (m ? dyv : (h16)0.0f);
  }
}

// ---- forward apply fused into the max pool that reads it ----------------------
// The apply + ReLU (no shortcut, no swap) evaluated inside the R x S max pool
// over its output: per pooled output vector (8 channels of one position)
// every input of the window is normalised with the apply's float32 sequence
// and rounded to binary16, then pooled with max pooling's comparison (the
// first in-image tap in row-major order starts; a later one replaces it only
// when strictly larger, or as the first NaN), so the pooled values and tap
// indices are bit for bit those of the apply followed by the pool, and the
// normalised tensor is never written.  All R*S loads of a vector are issued
// before the first use (clamped into the image; a tap outside it is no
// candidate).  Grid-stride over output vectors; kT and the stride are
// multiples of C/8, so a thread keeps one channel chunk and its coefficients.
template <int R, int S>
__global__ __launch_bounds__(kT) void bn_apply_maxpool_vec(const h16* __restrict__ x,
                                                           const h16* __restrict__ gamma,
                                                           const h16* __restrict__ beta,
                                                           const float* __restrict__ stats,
                                                           float s, PoolArgs a,
                                                           h16* __restrict__ y,
                                                           uint8_t* __restrict__ idx) {
  const int CV = a.C / 8;
  const int j = threadIdx.x % CV;
  FwdCoef k[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) k[e] = fwd_coef(stats, gamma, beta, a.C, j * 8 + e, s);
  const int64_t total = (int64_t)a.N * a.P * a.Q * CV;
  for (int64_t v = (int64_t)blockIdx.x * kT + threadIdx.x; v < total;
       v += (int64_t)gridDim.x * kT) {
    int64_t r = v / CV;
    const int q = (int)(r % a.Q);
    r /= a.Q;
    const int p = (int)(r % a.P);
    const int n = (int)(r / a.P);
    const int h0 = p * a.sh - a.ph, w0 = q * a.sw - a.pw;
    const h16* xb = x + (int64_t)n * a.H * a.W * a.C + j * 8;
    V8 xv[R][S];
#pragma unroll
    for (int rr = 0; rr < R; ++rr)
#pragma unroll
      for (int ss = 0; ss < S; ++ss) {
        const int h = h0 + rr, w = w0 + ss;
        const int hc = h < 0 ? 0 : (h < a.H ? h : a.H - 1);
        const int wc = w < 0 ? 0 : (w < a.W ? w : a.W - 1);
        xv[rr][ss] = load16(xb + ((int64_t)hc * a.W + wc) * a.C);
      }
    __builtin_amdgcn_sched_barrier(0);  // every load issued before the first use
    float best[8];
    int tap[8];
    V8 win;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      best[e] = 0.0f;
      tap[e] = 0;
      win.s[e] = 0;
    }
    bool started = false;
#pragma unroll
    for (int rr = 0; rr < R; ++rr)
#pragma unroll
      for (int ss = 0; ss < S; ++ss) {
        const int h = h0 + rr, w = w0 + ss;
        const bool in = h >= 0 && h < a.H && w >= 0 && w < a.W;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const h16 z = to_h16(fwd_value(to_f32(xv[rr][ss].h[e]), k[e], false, 0.0f, true, false));
          const float f = to_f32(z);
          const bool tk = in & (!started | pool_takes(best[e], f));
          best[e] = tk ? f : best[e];
          win.h[e] = tk ? z : win.h[e];
          tap[e] = tk ? rr * S + ss : tap[e];
        }
        started = started || in;
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

unsigned apply_grid(int64_t nthreads_wanted, int CV) {
  int64_t b = (nthreads_wanted + kT - 1) / kT;
  if (b > 16384) b = 16384;
  if (b < 1) b = 1;
  (void)CV;  // kT is a multiple of CV, so any grid keeps each thread on one chunk
  return (unsigned)b;
}

// Template variant of the vectorised kernels for these arguments.
int fwd_mode(const BnArgs& a, const h16* res, bool keep) {
  return (a.swap ? kSwap : 0) | (a.relu ? kRelu : 0) | (res ? kLoadR : 0) | (keep ? kKeepF : 0);
}
int bwd_mode(const BnArgs& a, const h16* y, const h16* res, const h16* dres, bool bits) {
  if (bits) return kRelu | kMaskB | (dres ? kDres : 0);  // no swap: checked by the caller
  const bool relu = a.relu != 0, mask_y = relu && y != nullptr;
  const bool load_r = a.swap || (relu && !mask_y && res != nullptr);
  return (a.swap ? kSwap : 0) | (relu ? kRelu : 0) | (mask_y ? kMaskY : 0) |
         (load_r ? kLoadR : 0) | (dres ? kDres : 0);
}

// The valid variants (the BN swap always reads the shortcut).
#define FP16K_BN_FWD_MODES(X) X(0) X(2) X(8) X(10) X(9) X(11) X(66) X(74)
#define FP16K_BN_BWD_MODES(X) X(0) X(6) X(2) X(10) X(9) X(15) X(11) X(34)
#define FP16K_BN_BWD_APPLY_MODES(X) \
  FP16K_BN_BWD_MODES(X) X(16) X(22) X(18) X(26) X(25) X(31) X(27) X(50)

hipError_t launch_fwd_apply_vec(int mode, const Plan& p, const Geo& g, const h16* x,
                                const h16* gamma, const h16* beta, const h16* res, h16* y,
                                const float* stats, float s, uint8_t* mout, hipStream_t st) {
  const dim3 grid(apply_grid(g.M * p.CV / kApplyU, p.CV));
  switch (mode) {
#define FP16K_CASE(m)                                                                          \
  case m:                                                                                      \
    hipLaunchKernelGGL(bn_fwd_apply_vec<m>, grid, dim3(kT), 0, st, x, gamma, beta, res, y,     \
                       stats, g, p.CV, s, mout);                                                \
    break;
    FP16K_BN_FWD_MODES(FP16K_CASE)
#undef FP16K_CASE
    default:
      return hipErrorInvalidValue;
  }
  return hipSuccess;
}

Geo make_geo(const BnArgs& a) {
  Geo g;
  g.M = (int64_t)a.N * a.H * a.W;
  g.C = a.C;
  g.HW = a.H * a.W;
  g.layout = a.layout;
  g.swap = a.swap;
  return g;
}

size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

// Workspace: the partial sums, block-major [G][NS][C] from kBmC channels on,
// else channel-major [NS][C][G] (float32, NS <= 3), then the backward's apply
// coefficients [3][C].
size_t partial_bytes(const Plan& p, int C) { return align256((size_t)3 * p.G * C * sizeof(float)); }

}  // namespace

// the backward's coefficients, after the partials
size_t coef_bytes(int C) { return align256((size_t)3 * C * sizeof(float)); }

// the backward's kept ReLU mask, after the coefficients: one byte per 16-byte
// vector of x
size_t mask_bytes(const Plan& p, const BnArgs& a) {
  return p.vec && a.relu ? align256((size_t)((int64_t)a.N * a.H * a.W * p.CV)) : 0;
}

size_t bn_ws_bytes(const BnArgs& a) {
  const Plan p = make_plan(a);
  return partial_bytes(p, a.C) + coef_bytes(a.C) + mask_bytes(p, a);
}

// Bytes of a kept ReLU mask (one byte per 8 channels of each pixel), or 0
// where the vectorised kernels do not run or there is no ReLU.
size_t bn_keep_mask_bytes(const BnArgs& a) {
  const Plan p = make_plan(a);
  return p.vec && a.relu ? (size_t)((int64_t)a.N * a.H * a.W * p.CV) : 0;
}

// The batch statistics of x into stats (the partial sums in ws).
static void bn_fwd_stats(const BnArgs& a, const Plan& p, const Geo& g, const h16* x, float* stats,
                         void* ws, hipStream_t st) {
  float* part = reinterpret_cast<float*>(ws);
  if (p.vec)
    hipLaunchKernelGGL(bn_fwd_reduce_vec, dim3(p.G), dim3(kT), 0, st, x, g, p.CV, p.RB, p.rpb,
                       part);
  else
    hipLaunchKernelGGL(bn_fwd_reduce_gen, dim3(p.G, a.C), dim3(kT), 0, st, x, g, p.rpb, part);
  if (p.vec && a.C >= kBmC)
    hipLaunchKernelGGL(bn_fwd_finalize_bm, dim3((a.C + 63) / 64), dim3(64 * kFinW), 0, st, x, g,
                       p.G, part, a.eps, stats);
  else
    hipLaunchKernelGGL(bn_fwd_finalize, dim3(a.C), dim3(64), 0, st, x, g, p.G, part, a.eps, stats);
}

hipError_t launch_bn_fwd(const BnArgs& a, const h16* x, const h16* gamma, const h16* beta,
                         const h16* res, h16* y, float* stats, int use_stats, void* ws,
                         uint8_t* mout, hipStream_t st) {
  const Plan p = make_plan(a);
  const Geo g = make_geo(a);
  if (!use_stats) bn_fwd_stats(a, p, g, x, stats, ws, st);
  if (p.vec) {
    const hipError_t e =
        launch_fwd_apply_vec(fwd_mode(a, res, mout != nullptr), p, g, x, gamma, beta, res, y, stats,
                             a.post_scale, mout, st);
    if (e != hipSuccess) return e;
  } else {
    hipLaunchKernelGGL(bn_fwd_apply_gen, dim3(apply_grid(g.M * a.C / 4, 1)), dim3(kT), 0, st, x,
                       gamma, beta, res, y, stats, g, a.post_scale, a.relu);
  }
  return hipGetLastError();
}

bool bn_maxpool_ok(const BnArgs& a, const PoolArgs& pa) {
  return make_plan(a).vec && a.relu && !a.swap && pa.layout == 0 && pa.N == a.N &&
         pa.C == a.C && pa.H == a.H && pa.W == a.W && pa.R == 3 && pa.S == 3;
}

hipError_t launch_bn_fwd_maxpool(const BnArgs& a, const PoolArgs& pa, const h16* x,
                                 const h16* gamma, const h16* beta, float* stats, int use_stats,
                                 void* ws, h16* y, uint8_t* idx, hipStream_t st) {
  const Plan p = make_plan(a);
  const Geo g = make_geo(a);
  if (!use_stats) bn_fwd_stats(a, p, g, x, stats, ws, st);
  const int64_t total = (int64_t)pa.N * pa.P * pa.Q * (pa.C / 8);
  hipLaunchKernelGGL((bn_apply_maxpool_vec<3, 3>), dim3(apply_grid(total, p.CV)), dim3(kT), 0, st,
                     x, gamma, beta, stats, a.post_scale, pa, y, idx);
  return hipGetLastError();
}

size_t bn_band_ws_bytes(int C, int nb) {
  const int64_t ns = ((int64_t)nb + kBandRps - 1) / kBandRps;
  return align256((size_t)2 * C * ns * sizeof(double));
}

hipError_t launch_bn_band_stats(const BnArgs& a, const float* part, int nb, void* band_ws,
                                float* stats, hipStream_t st) {
  const Geo g = make_geo(a);
  if (nb <= kBandOne) {
    hipLaunchKernelGGL(bn_band_finalize, dim3(a.C), dim3(256), 0, st, part, nb, g, a.eps, stats);
  } else {
    const int ns = (nb + kBandRps - 1) / kBandRps;
    double* sl = reinterpret_cast<double*>(band_ws);
    hipLaunchKernelGGL(bn_band_slices, dim3((a.C + 63) / 64, ns), dim3(256), 0, st, part, nb, g,
                       sl, ns);
    hipLaunchKernelGGL(bn_band_combine, dim3(a.C), dim3(64), 0, st, part, sl, ns, g, a.eps,
                       stats);
  }
  return hipGetLastError();
}

hipError_t launch_bn_fwd_bands(const BnArgs& a, const float* part, int nb, void* band_ws,
                               const h16* x, const h16* gamma, const h16* beta, const h16* res,
                               h16* y, float* stats, uint8_t* mout, hipStream_t st) {
  const Plan p = make_plan(a);
  const Geo g = make_geo(a);
  const hipError_t es = launch_bn_band_stats(a, part, nb, band_ws, stats, st);
  if (es != hipSuccess) return es;
  if (p.vec) {
    const hipError_t e =
        launch_fwd_apply_vec(fwd_mode(a, res, mout != nullptr), p, g, x, gamma, beta, res, y, stats,
                             a.post_scale, mout, st);
    if (e != hipSuccess) return e;
  } else {
    hipLaunchKernelGGL(bn_fwd_apply_gen, dim3(apply_grid(g.M * a.C / 4, 1)), dim3(kT), 0, st, x,
                       gamma, beta, res, y, stats, g, a.post_scale, a.relu);
  }
  return hipGetLastError();
}

hipError_t launch_bn_bwd(const BnArgs& a, const h16* x, const h16* y, const h16* dy,
                         const h16* gamma, const h16* beta, const h16* res, const float* stats,
                         h16* dx, h16* dgamma, h16* dbeta, h16* dres, void* ws,
                         const uint8_t* mask, hipStream_t st) {
  const Plan p = make_plan(a);
  const Geo g = make_geo(a);
  float* part = reinterpret_cast<float*>(ws);
  float* coef = reinterpret_cast<float*>(reinterpret_cast<char*>(ws) + partial_bytes(p, a.C));
  // the forward's kept mask (only read), else the workspace's, which the
  // reduce fills when it recomputes the mask from the shortcut
  uint8_t* mbits = mask ? const_cast<uint8_t*>(mask)
                        : reinterpret_cast<uint8_t*>(ws) + partial_bytes(p, a.C) + coef_bytes(a.C);
  if (mask && (!p.vec || a.swap || !a.relu)) return hipErrorInvalidValue;
  const int mode = bwd_mode(a, y, res, dres, mask != nullptr);
  if (p.vec) {
    switch (mode & ~kDres) {
#define FP16K_CASE(m)                                                                          \
  case m:                                                                                      \
    hipLaunchKernelGGL(bn_bwd_reduce_vec<m>, dim3(p.G), dim3(kT), 0, st, x, y, dy, gamma, beta, \
                       res, stats, g, p.CV, p.RB, p.rpb, a.post_scale, part, mbits);             \
    break;
      FP16K_BN_BWD_MODES(FP16K_CASE)
#undef FP16K_CASE
      default:
        return hipErrorInvalidValue;
    }
  } else {
    hipLaunchKernelGGL(bn_bwd_reduce_gen, dim3(p.G, a.C), dim3(kT), 0, st, x, y, dy, gamma, beta,
                       res, stats, g, p.rpb, a.post_scale, a.relu, part);
  }
  if (!(p.vec && a.C >= kBmC))
    hipLaunchKernelGGL(bn_bwd_finalize, dim3(a.C), dim3(64), 0, st, g, p.G, part, gamma, stats,
                       dgamma, dbeta, coef);
  else if (a.swap)
    hipLaunchKernelGGL(bn_bwd_finalize_bm<3>, dim3((a.C + 63) / 64), dim3(64 * kFinW), 0, st, g,
                       p.G, part, gamma, stats, dgamma, dbeta, coef);
  else
    hipLaunchKernelGGL(bn_bwd_finalize_bm<2>, dim3((a.C + 63) / 64), dim3(64 * kFinW), 0, st, g,
                       p.G, part, gamma, stats, dgamma, dbeta, coef);
  if (p.vec) {
    const dim3 grid(apply_grid(g.M * p.CV / (kApplyU / 2), p.CV));
    switch (mode) {
#define FP16K_CASE(m)                                                                          \
  case m:                                                                                      \
    hipLaunchKernelGGL(bn_bwd_apply_vec<m>, grid, dim3(kT), 0, st, x, y, dy, gamma, beta, res, \
                       stats, coef, g, p.CV, a.post_scale, mbits, dx, dres);                    \
    break;
      FP16K_BN_BWD_APPLY_MODES(FP16K_CASE)
#undef FP16K_CASE
      default:
        return hipErrorInvalidValue;
    }
  } else {
    hipLaunchKernelGGL(bn_bwd_apply_gen, dim3(apply_grid(g.M * a.C / 4, 1)), dim3(kT), 0, st, x,
                       y, dy, gamma, beta, res, stats, coef, g, a.post_scale, a.relu, dx, dres);
  }
  return hipGetLastError();
}

}  // namespace fp16k
