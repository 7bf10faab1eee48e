// Weight gradient of the convolution on the gfx950 FP16 matrix cores.
//
// GEMM view: dW[k][col] = sum_pix dy[pix][k] * X[pix][col],
//   pix = (image, p, q) over the output grid (the reduction, length N*P*Q),
//   col = (r, s, c) with c fastest (the KRSC filter row),
//   X[pix][(r,s,c)] = x[image][p*sh - ph + r][q*sw - pw + s][c] (zero outside).
// Both operands are channel-contiguous in memory but the reduction runs over
// pixels, so each thread loads an 8-pixel x 8-channel block (eight 16-byte
// loads), transposes it in registers with byte permutes, and writes eight
// 16-byte channel rows into LDS.  MFMA operands are then 16-byte LDS reads.
//
// The pixel range is split across workgroups (split-K).  Each split writes
// its float32 partial tile to the workspace; a second kernel adds the splits
// in a fixed order and rounds once to binary16, so the result is
// deterministic.

#include "kernels.hpp"

namespace fp16k {
namespace {

constexpr int BKP = 64;         // pixels per k-step
constexpr int LDP = BKP + 8;    // LDS row pitch (halves)

template <int BM, int BN, int WM, int WN>
__global__ __launch_bounds__(256) void wgrad_kernel(const WgradArgs a) {
  constexpr int WTM = BM / WM, WTN = BN / WN;
  constexpr int TM = WTM / 32, TN = WTN / 32;
  constexpr int NA = (BKP / 8) * (BM / 8);  // 8x8 blocks of the dy tile
  constexpr int NB = (BKP / 8) * (BN / 8);  // 8x8 blocks of the x tile
  static_assert(NA + NB <= 256, "one block per thread at most");
  static_assert(NA % 64 == 0, "wave-uniform A/B split");
  static_assert(WM * WN == 4 && TM >= 1 && TN >= 1, "tile shape");

  __shared__ __attribute__((aligned(16))) h16 As[2][BM * LDP];
  __shared__ __attribute__((aligned(16))) h16 Bs[2][BN * LDP];

  const int Nw = a.R * a.S * a.C;
  const int tiles_n = (Nw + BN - 1) / BN;
  const int tile = blockIdx.x;
  const int m0 = (tile / tiles_n) * BM;
  const int n0 = (tile % tiles_n) * BN;
  const int split = blockIdx.y;
  const int64_t npix = (int64_t)a.N * a.P * a.Q;
  const int64_t pbeg = (int64_t)split * a.pix_per_split;
  int64_t pend = pbeg + a.pix_per_split;
  if (pend > npix) pend = npix;

  const int tid = threadIdx.x;
  const bool is_a = tid < NA;
  const bool is_b = !is_a && tid < NA + NB;
  // block coordinates: pixel group pi (8 pixels), channel group ci (8 channels)
  const int bidx = is_a ? tid : tid - NA;
  const int pi = bidx % (BKP / 8);
  const int ci = bidx / (BKP / 8);

  // x column chunk of a B-thread: tap (r, s) and channel offset c
  int br = 0, bs = 0, bc = 0;
  bool bcol_ok = false;
  if (is_b) {
    const int col = n0 + ci * 8;
    bcol_ok = col < Nw;
    const int tap = bcol_ok ? col / a.C : 0;
    bc = col - tap * a.C;
    br = tap / a.S;
    bs = tap - br * a.S;
  }
  const bool acol_ok = is_a && (m0 + ci * 8) < a.K;

  V8 blk[8];
  auto load_tile = [&](int64_t p0) {
    const int64_t pix0 = p0 + pi * 8;
    if (is_a) {
#pragma unroll
      for (int v = 0; v < 8; ++v) {
        const int64_t pix = pix0 + v;
        blk[v] = (acol_ok && pix < pend) ? load16(a.dy + pix * a.K + m0 + ci * 8) : zero8();
      }
    } else if (is_b) {
      // decompose the first pixel, then step (q, p, image) incrementally
      int64_t t = pix0;
      int q = (int)(t % a.Q);
      t /= a.Q;
      int p = (int)(t % a.P);
      int img = (int)(t / a.P);
#pragma unroll
      for (int v = 0; v < 8; ++v) {
        const int ih = p * a.sh - a.ph + br;
        const int iw = q * a.sw - a.pw + bs;
        const bool ok = bcol_ok && (pix0 + v) < pend && (unsigned)ih < (unsigned)a.H &&
                        (unsigned)iw < (unsigned)a.W;
        blk[v] = ok ? load16(a.x + ((int64_t)(img * a.H + ih) * a.W + iw) * a.C + bc) : zero8();
        if (++q == a.Q) {
          q = 0;
          if (++p == a.P) {
            p = 0;
            ++img;
          }
        }
      }
    }
  };
  auto store_tile = [&](int buf) {
    if (!is_a && !is_b) return;
    V8 tr[8];
    transpose8x8(blk, tr);
    h16* base = is_a ? &As[buf][0] : &Bs[buf][0];
#pragma unroll
    for (int j = 0; j < 8; ++j) store16(base + (ci * 8 + j) * LDP + pi * 8, tr[j]);
  };

  const int wave = tid >> 6, lane = tid & 63;
  const int wm = wave / WN, wn = wave % WN;
  const int lrow = lane & 31, lk = (lane >> 5) * 8;

  floatx16 acc[TM][TN];
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int tn = 0; tn < TN; ++tn)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[tm][tn][e] = 0.0f;

  const int KT = pend > pbeg ? (int)((pend - pbeg + BKP - 1) / BKP) : 0;
  if (KT > 0) {
    load_tile(pbeg);
    store_tile(0);
  }
  __syncthreads();
  for (int kt = 0; kt < KT; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < KT) load_tile(pbeg + (int64_t)(kt + 1) * BKP);
#pragma unroll
    for (int ks = 0; ks < BKP / 16; ++ks) {
      half8 af[TM], bf[TN];
#pragma unroll
      for (int tm = 0; tm < TM; ++tm)
        af[tm] = *reinterpret_cast<const half8*>(
            &As[buf][(wm * WTM + tm * 32 + lrow) * LDP + ks * 16 + lk]);
#pragma unroll
      for (int tn = 0; tn < TN; ++tn)
        bf[tn] = *reinterpret_cast<const half8*>(
            &Bs[buf][(wn * WTN + tn * 32 + lrow) * LDP + ks * 16 + lk]);
#pragma unroll
      for (int tm = 0; tm < TM; ++tm)
#pragma unroll
        for (int tn = 0; tn < TN; ++tn) acc[tm][tn] = mfma32x32x16(af[tm], bf[tn], acc[tm][tn]);
    }
    if (kt + 1 < KT) store_tile(buf ^ 1);
    __syncthreads();
  }

  // float32 partial tile of this split
  float* out = a.partial + (int64_t)split * a.K * Nw;
#pragma unroll
  for (int tm = 0; tm < TM; ++tm) {
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int m = m0 + wm * WTM + tm * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
      if (m >= a.K) continue;
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) {
        const int n = n0 + wn * WTN + tn * 32 + lrow;
        if (n < Nw) out[(int64_t)m * Nw + n] = acc[tm][tn][e];
      }
    }
  }
}

// dw = rne16(sum over splits), written KRSC or KCRS with the real C.  A block
// of 256 threads owns 64 consecutive outputs; its four waves each add every
// fourth split (in order), and the four subtotals are added in a fixed order,
// so the result is deterministic.
__global__ __launch_bounds__(256) void wgrad_reduce_kernel(const float* __restrict__ partial,
                                                           int splits, int K, int Kp, int R, int S,
                                                           int C, int Cp, int layout,
                                                           h16* __restrict__ dw) {
  __shared__ float red[4][64];
  const int64_t Nw = (int64_t)R * S * Cp;
  const int64_t total = (int64_t)K * R * S * C;
  const int lane = threadIdx.x & 63, grp = threadIdx.x >> 6;
  const int64_t i = (int64_t)blockIdx.x * 64 + lane;  // enumerates KRSC with the real C
  int64_t src = 0;
  int k = 0, r = 0, s = 0, c = 0;
  if (i < total) {
    c = (int)(i % C);
    int64_t t = i / C;
    s = (int)(t % S);
    t /= S;
    r = (int)(t % R);
    k = (int)(t / R);
    src = (int64_t)k * Nw + ((int64_t)r * S + s) * Cp + c;
  }
  // splits grp, grp+4, grp+8, ... added in that order; eight loads are
  // issued before their adds so the loop is not a chain of load latencies
  float sum = 0.0f;
  if (i < total) {
    const int64_t stride = (int64_t)Kp * Nw;
    const float* p = partial + src;
    int sp = grp;
    for (; sp + 28 < splits; sp += 32) {
      float v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = p[(int64_t)(sp + 4 * u) * stride];
#pragma unroll
      for (int u = 0; u < 8; ++u) sum += v[u];
    }
    for (; sp < splits; sp += 4) sum += p[(int64_t)sp * stride];
  }
  red[grp][lane] = sum;
  __syncthreads();
  if (grp == 0 && i < total) {
    const float v = ((red[0][lane] + red[1][lane]) + red[2][lane]) + red[3][lane];
    const int64_t dst = layout == 0 ? i : (((int64_t)k * C + c) * R + r) * S + s;
    dw[dst] = to_h16(v);
  }
}

// Tile configuration shared by the plan and the launch.
struct WCfg {
  int BM, BN;
};
// Larger tiles re-read less: a wider N tile reuses the dy tile over more
// filter columns (three 3x3 taps at once for 64 output channels), a taller M
// tile reuses the x tile over more output channels.  Each configuration has
// at most one 8x8 load block per thread (BM + BN <= 256).
inline WCfg wgrad_cfg(int K, int Nw) {
  if (K >= 128 && Nw >= 128) return {128, 128};
  if (K >= 128) return {128, 64};
  if (Nw >= 192 && Nw % 192 == 0) return {64, 192};
  if (Nw >= 128) return {64, 128};
  return {64, 64};
}

}  // namespace

void wgrad_plan(int K, int Cp, int R, int S, int64_t npix, int* splits, int* pix_per_split) {
  const int Nw = R * S * Cp;
  const WCfg cfg = wgrad_cfg(K, Nw);
  const int64_t tiles = (int64_t)ceil_div(K, cfg.BM) * ceil_div(Nw, cfg.BN);
  int64_t want = (512 + tiles - 1) / tiles;           // about two workgroups per CU
  const int64_t max_splits = (npix + 2 * BKP - 1) / (2 * BKP);  // at least two k-steps each
  if (want > max_splits) want = max_splits;
  if (want < 1) want = 1;
  int64_t pps = (npix + want - 1) / want;
  pps = (pps + BKP - 1) / BKP * BKP;
  if (pps < BKP) pps = BKP;
  *pix_per_split = (int)pps;
  *splits = (int)((npix + pps - 1) / pps);
  if (*splits < 1) *splits = 1;
}

hipError_t launch_wgrad_partial(const WgradArgs& a, hipStream_t st) {
  const int Nw = a.R * a.S * a.C;
  const WCfg cfg = wgrad_cfg(a.K, Nw);
  const int tiles = ceil_div(a.K, cfg.BM) * ceil_div(Nw, cfg.BN);
  dim3 grid(tiles, a.splits);
  if (cfg.BM == 128 && cfg.BN == 128)
    hipLaunchKernelGGL((wgrad_kernel<128, 128, 2, 2>), grid, dim3(256), 0, st, a);
  else if (cfg.BM == 128)
    hipLaunchKernelGGL((wgrad_kernel<128, 64, 2, 2>), grid, dim3(256), 0, st, a);
  else if (cfg.BN == 192)
    hipLaunchKernelGGL((wgrad_kernel<64, 192, 2, 2>), grid, dim3(256), 0, st, a);
  else if (cfg.BN == 128)
    hipLaunchKernelGGL((wgrad_kernel<64, 128, 2, 2>), grid, dim3(256), 0, st, a);
  else
    hipLaunchKernelGGL((wgrad_kernel<64, 64, 2, 2>), grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_wgrad_reduce(const float* partial, int splits, int K, int Kp, int R, int S, int C,
                               int Cp, int layout, h16* dw, hipStream_t st) {
  const int64_t total = (int64_t)K * R * S * C;
  const int64_t blocks = (total + 63) / 64;
  hipLaunchKernelGGL(wgrad_reduce_kernel, dim3((unsigned)blocks), dim3(256), 0, st, partial, splits,
                     K, Kp, R, S, C, Cp, layout, dw);
  return hipGetLastError();
}

}  // namespace fp16k
