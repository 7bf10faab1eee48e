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

#include <type_traits>

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
        for (int tn = 0; tn < TN; ++tn) {
          acc[tm][tn] = mfma32x32x16(af[tm], bf[tn], acc[tm][tn]);
        }
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

// ---- DMA-staged variant: no register transposes ------------------------------
// For K a multiple of 64 and C a multiple of 8 (when C is not a multiple of
// 64 -- the padded 3-channel stem -- each lane's 8-channel chunk carries its
// own filter tap).  Each stage covers 64 pixels:
// the dy rows (BM channels) and the x patch rows (BN filter columns, 64 per
// tap and channel block) are DMA'd pixel-major straight into LDS, in 8 KB
// sub-tiles of 64 pixel rows x 128 bytes (16-byte chunks XOR-swizzled by
// pixel row).  The MFMA operands, which need 8 consecutive pixels per lane,
// come from the transposing LDS read of gfx950 (ds_read_b64_tr_b16: within
// each 16-lane group, lane b*4+a receives element a of the 8-byte rows that
// lanes b, b+4, b+8 and b+12 address), two reads per operand.  S stages in a
// ring, operand reads one k sub-step ahead, as in the implicit-GEMM kernel.
// The k order (pixels) and the split plan are those of wgrad_kernel, so the
// partial sums are the same.

typedef short short4v __attribute__((ext_vector_type(4)));

// One 16-byte-per-lane DMA from a buffer resource into LDS (1 KB per wave).
__device__ __forceinline__ void wdma16(__amdgpu_buffer_rsrc_t rs, char* lds_dst, uint32_t voff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (__attribute__((address_space(3))) void*)lds_dst, 16,
                                           voff, 0, 0, 0);
}

__device__ __forceinline__ void wbarrier() { __asm__ volatile("s_barrier" ::: "memory"); }

// The transposing read, issued from inline assembly at an LDS byte address
// plus a constant offset.  Through the compiler's builtin, every such read
// waits for all LDS DMAs in flight (the compiler cannot tell the buffers
// apart), so the stage just issued had to land before the next stage could be
// read; from assembly the ring keeps its stages in flight (5-15 % faster on
// the ResNet-50 shapes, bit-identical partials).  The compiler then neither
// orders the read after the DMAs nor waits for its result: the loop orders
// the DMAs by its own vmcnt wait and barrier, and each result by lds_ready()
// before the MFMAs that use it.  Nothing may read the destination registers
// before that wait (not even a register copy); a host-side test checks the
// built code for it.
template <int OFF>
__device__ __forceinline__ short4v ldtr_asm(uint32_t addr) {
  short4v r;
  __asm__ volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(r) : "v"(addr), "i"(OFF));
  return r;
}
// Waits until at most N LDS reads of this wave are in flight; the fragment is
// tied to the wait so that no use of it is scheduled before.
template <int N>
__device__ __forceinline__ void lds_ready(half8& v) {
  __asm__ volatile("s_waitcnt lgkmcnt(%1)" : "+v"(v) : "i"(N));
}
__device__ __forceinline__ void lds_tie(half8& v) { __asm__ volatile("" : "+v"(v)); }

template <int BM, int BN, int WM, int WN, int S>
struct WCfg7 {
  static constexpr int SA = BM / 64, SB = BN / 64;  // 64-channel sub-tiles
  static constexpr int NI = (SA + SB) * 8;          // DMA instructions per stage
  static constexpr int IW = NI / 4;                 // per wave
  static constexpr int STAGE = (SA + SB) * 8192;    // bytes
  static constexpr int WTM = BM / WM, WTN = BN / WN;
  static constexpr int TM = WTM / 32, TN = WTN / 32;
};

template <int BM, int BN, int WM, int WN, int S, bool CGEN = false>
__global__ __launch_bounds__(256) void wgrad7_kernel(const WgradArgs a) {
  using K = WCfg7<BM, BN, WM, WN, S>;
  constexpr int SA = K::SA, SB = K::SB, IW = K::IW, TM = K::TM, TN = K::TN, WTM = K::WTM,
                WTN = K::WTN;
  static_assert(WM * WN == 4 && TM >= 1 && TN >= 1 && S >= 2, "tile shape");
  static_assert(IW * (S - 1) < 64, "vmcnt range");
  __shared__ __attribute__((aligned(1024))) char lds[S * K::STAGE];

  const int Nw = a.R * a.S * a.C;
  const int tiles_n = (Nw + BN - 1) / BN;
  // Workgroups are dealt to the 8 XCDs round-robin in launch order.  Each
  // XCD gets a contiguous run of the split-major order instead, so the tiles
  // that share a pixel range (and so its dy and x rows) share one L2: the
  // layers with 28x28 and larger grids at batch 128 went 1.1-1.9x faster.
  int tile, split;
  {
    const int total = gridDim.x * gridDim.y;
    const int L = blockIdx.y * gridDim.x + blockIdx.x;
    const int q = total >> 3, r = total & 7, xcd = L & 7;
    const int Lg = xcd * q + (xcd < r ? xcd : r) + (L >> 3);
    tile = Lg % gridDim.x;
    split = Lg / gridDim.x;
  }
  const int m0 = (tile / tiles_n) * BM;
  const int n0 = (tile % tiles_n) * BN;
  const int64_t npix = (int64_t)a.N * a.P * a.Q;
  const int64_t pbeg = (int64_t)split * a.pix_per_split;
  int64_t pend = pbeg + a.pix_per_split;
  if (pend > npix) pend = npix;
  const int KT = pend > pbeg ? (int)((pend - pbeg + 63) / 64) : 0;

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  constexpr uint32_t OOB = 0x80000000u;
  const int dy_bytes = (int)(npix * a.K * 2);
  const int x_bytes = (int)((int64_t)a.N * a.H * a.W * a.C * 2);

  // DMA roles: instruction i of this wave fills sub-tile i/2, pixel rows
  // rb*8 .. rb*8+7 with rb = 4*(i%2) + wave; a lane covers pixel row
  // rb*8 + lane/8 and physical chunk lane%8, holding logical chunk
  // (lane%8) ^ swz(row), swz(row) = 2*(row%4).  A transposing read takes
  // 32 bytes (chunks 2i, 2i+1) from each of 4 consecutive rows per 16-lane
  // group; with this swizzle the 4 rows' pairs land on distinct chunk
  // positions, and the two groups served together (the other channel
  // half) on the rest, so the reads are bank-conflict free.
  int prow[2], img[2], pp[2], qq[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    prow[h] = (4 * h + wave) * 8 + (lane >> 3);
    const int64_t pix = pbeg + prow[h];
    const int64_t PQ = (int64_t)a.P * a.Q;
    img[h] = (int)(pix / PQ);
    const int rem = (int)(pix - (int64_t)img[h] * PQ);
    pp[h] = rem / a.Q;
    qq[h] = rem - pp[h] * a.Q;
  }
  const int dq = 64 % a.Q, dp = (64 / a.Q) % a.P, dimg = 64 / (a.P * a.Q);
  int lc[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) lc[h] = (lane & 7) ^ ((prow[h] & 3) << 1);
  // CGEN (C a multiple of 8 but not of 64): a 64-column block of the x patch
  // spans several filter taps, so each lane's 8-channel chunk has a tap of its
  // own; precomputed here (tap row, tap column, channel offset; -1 past Nw)
  int gr[2][CGEN ? SB : 1], gt[2][CGEN ? SB : 1], gc[2][CGEN ? SB : 1];
  if (CGEN) {
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int b = 0; b < SB; ++b) {
        const int col = n0 + b * 64 + lc[h] * 8;
        const int tap = col / a.C;
        gc[h][b] = col < Nw ? col - tap * a.C : -1;
        gr[h][b] = tap / a.S;
        gt[h][b] = tap - gr[h][b] * a.S;
      }
  }

  int64_t pstage = pbeg;  // first pixel of the next stage to issue
  auto issue = [&](char* buf) {
    const __amdgpu_buffer_rsrc_t rs_dy = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<h16*>(a.dy), (short)0, dy_bytes, 0x00020000);
    const __amdgpu_buffer_rsrc_t rs_x = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<h16*>(a.x), (short)0, x_bytes, 0x00020000);
#pragma unroll
    for (int i = 0; i < IW; ++i) {
      const int h = i & 1;
      const int sub = i >> 1;
      const int rb = 4 * h + wave;
      char* dst = buf + sub * 8192 + rb * 1024;
      const int64_t pix = pstage + prow[h];
      const bool pv = pix < pend;
      if (sub < SA) {
        const int m = m0 + sub * 64;
        const uint32_t off = (uint32_t)((pix * a.K + m + lc[h] * 8) * 2);
        wdma16(rs_dy, dst, (pv && m < a.K) ? off : OOB);
      } else if (CGEN) {
        const int b = sub - SA;
        const int ih = pp[h] * a.sh - a.ph + gr[h][b], iw = qq[h] * a.sw - a.pw + gt[h][b];
        const bool v = pv && gc[h][b] >= 0 && (unsigned)ih < (unsigned)a.H &&
                       (unsigned)iw < (unsigned)a.W;
        const uint32_t off =
            (uint32_t)(((((int64_t)img[h] * a.H + ih) * a.W + iw) * a.C + gc[h][b]) * 2);
        wdma16(rs_x, dst, v ? off : OOB);
      } else {
        const int cb = n0 + (sub - SA) * 64;
        const int tap = cb / a.C;
        const int c0 = cb - tap * a.C;
        const int r = tap / a.S, t = tap - r * a.S;
        const int ih = pp[h] * a.sh - a.ph + r, iw = qq[h] * a.sw - a.pw + t;
        const bool v = pv && cb < Nw && (unsigned)ih < (unsigned)a.H && (unsigned)iw < (unsigned)a.W;
        const uint32_t off =
            (uint32_t)(((((int64_t)img[h] * a.H + ih) * a.W + iw) * a.C + c0 + lc[h] * 8) * 2);
        wdma16(rs_x, dst, v ? off : OOB);
      }
    }
    // advance the two pixel rows by 64
    pstage += 64;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      qq[h] += dq;
      const int c1 = qq[h] >= a.Q;
      qq[h] -= c1 ? a.Q : 0;
      pp[h] += dp + c1;
      const int c2 = pp[h] >= a.P;
      pp[h] -= c2 ? a.P : 0;
      img[h] += dimg + c2;
    }
  };

  const int wm = wave / WN, wn = wave % WN;
  const int g = lane >> 4, j = lane & 15;
  // transposing-read address pieces of this lane: pixel row within a k16
  // sub-step, and channel quad within a 32-row operand
  const int kr_l = 8 * (g >> 1) + (j >> 2);
  const int ch_l = 16 * (g & 1) + 4 * (j & 3);
  floatx16 acc[TM][TN];
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int tn = 0; tn < TN; ++tn)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[tm][tn][e] = 0.0f;

  half8 af[2][TM], bf[2][TN];
  auto mma = [&](const half8 (&fa)[TM], const half8 (&fb)[TN]) {
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) acc[tm][tn] = mfma32x32x16(fa[tm], fb[tn], acc[tm][tn]);
  };

  if (KT > 0) {
    // lane part of each operand's read address (the swizzle depends on the
    // pixel row mod 4, which k sub-steps of 16 rows and the +4 row of the
    // second read leave unchanged): sub-step ks of a stage is at +2048*ks,
    // the second read at +512
    const uint32_t lds0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)lds;
    uint32_t oa[TM], ob[TN];
    auto lane_part = [&](int c) {
      const int ch = (c & 63) + ch_l;
      return (uint32_t)((c >> 6) * 8192 + kr_l * 128 + (((ch >> 3) ^ ((kr_l & 3) << 1)) << 4) +
                        ((ch >> 2) & 1) * 8);
    };
#pragma unroll
    for (int tm = 0; tm < TM; ++tm) oa[tm] = lds0 + lane_part(wm * WTM + tm * 32);
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) ob[tn] = lds0 + SA * 8192 + lane_part(wn * WTN + tn * 32);
    constexpr int NR = 2 * (TM + TN);  // reads per sub-step
    static_assert(NR <= 15, "lgkmcnt range");
    auto afetch = [&](auto ks, uint32_t sbase, half8(&fa)[TM], half8(&fb)[TN]) {
      constexpr int KS = decltype(ks)::value;
#pragma unroll
      for (int tm = 0; tm < TM; ++tm) {
        const short4v v0 = ldtr_asm<KS * 2048>(oa[tm] + sbase);
        const short4v v1 = ldtr_asm<KS * 2048 + 512>(oa[tm] + sbase);
        fa[tm] = __builtin_bit_cast(half8, __builtin_shufflevector(v0, v1, 0, 1, 2, 3, 4, 5, 6, 7));
      }
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) {
        const short4v v0 = ldtr_asm<KS * 2048>(ob[tn] + sbase);
        const short4v v1 = ldtr_asm<KS * 2048 + 512>(ob[tn] + sbase);
        fb[tn] = __builtin_bit_cast(half8, __builtin_shufflevector(v0, v1, 0, 1, 2, 3, 4, 5, 6, 7));
      }
    };
    // the fragments of one sub-step are complete once at most NR reads (those
    // of the next sub-step, issued after them) are in flight
    auto ready = [&](half8(&fa)[TM], half8(&fb)[TN]) {
      lds_ready<NR>(fa[0]);
#pragma unroll
      for (int tm = 1; tm < TM; ++tm) lds_tie(fa[tm]);
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) lds_tie(fb[tn]);
    };
#pragma unroll
    for (int s = 0; s < S; ++s) issue(lds + s * K::STAGE);
    constexpr int ALLOW0 = IW * (S - 1);
    constexpr int WAIT0 = (0x0 << 8) | (0x7 << 4) | (ALLOW0 & 0xF) | ((ALLOW0 >> 4) << 14);
    constexpr int ALLOW = IW * (S - 2);
    constexpr int WAIT = (0x0 << 8) | (0x7 << 4) | (ALLOW & 0xF) | ((ALLOW >> 4) << 14);
    __builtin_amdgcn_s_waitcnt(WAIT0);
    wbarrier();
    afetch(std::integral_constant<int, 0>(), 0u, af[0], bf[0]);
    int rd = 0;
    for (int kt = 0; kt < KT; ++kt) {
      const uint32_t cur = (uint32_t)(rd * K::STAGE);
      afetch(std::integral_constant<int, 1>(), cur, af[1], bf[1]);
      ready(af[0], bf[0]);
      mma(af[0], bf[0]);
      afetch(std::integral_constant<int, 2>(), cur, af[0], bf[0]);
      ready(af[1], bf[1]);
      mma(af[1], bf[1]);
      afetch(std::integral_constant<int, 3>(), cur, af[1], bf[1]);
      ready(af[0], bf[0]);
      mma(af[0], bf[0]);
      // every read of this stage is complete (lgkmcnt 0) and stage kt+1 has
      // landed (vmcnt) in every wave before the buffer is refilled
      __builtin_amdgcn_s_waitcnt(WAIT);
      wbarrier();
      issue(lds + rd * K::STAGE);
      rd = rd + 1 == S ? 0 : rd + 1;
      afetch(std::integral_constant<int, 0>(), (uint32_t)(rd * K::STAGE), af[0], bf[0]);
      ready(af[1], bf[1]);
      mma(af[1], bf[1]);
    }
    __builtin_amdgcn_s_waitcnt(0);
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
        const int n = n0 + wn * WTN + tn * 32 + (lane & 31);
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

// Few splits, KRSC output with unpadded channels (the partial rows are then
// the output rows): each thread adds four consecutive outputs over all splits
// in split order (16-byte loads, four splits in flight), and rounds once.
__global__ __launch_bounds__(256) void wgrad_reduce_vec_kernel(const float* __restrict__ partial,
                                                               int splits, int64_t total,
                                                               int64_t stride, h16* __restrict__ dw) {
  const int64_t i = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 4;
  if (i >= total) return;
  const floatx4* p = reinterpret_cast<const floatx4*>(partial + i);
  const int64_t st4 = stride / 4;
  floatx4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
  int sp = 0;
  for (; sp + 4 <= splits; sp += 4) {
    const floatx4 v0 = p[(sp + 0) * st4], v1 = p[(sp + 1) * st4];
    const floatx4 v2 = p[(sp + 2) * st4], v3 = p[(sp + 3) * st4];
    acc += v0;
    acc += v1;
    acc += v2;
    acc += v3;
  }
  for (; sp < splits; ++sp) acc += p[sp * st4];
  union {
    h16 h[4];
    uint2 u;
  } o;
#pragma unroll
  for (int e = 0; e < 4; ++e) o.h[e] = to_h16(acc[e]);
  *reinterpret_cast<uint2*>(dw + i) = o.u;
}

// Tile configuration shared by the plan and the launch.
struct WCfg {
  int BM, BN;
  int S = 2;  // stages of the DMA ring (DMA-staged kernel)
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
// The DMA-staged kernel (channel counts multiples of 64) and its tiles.
inline bool wgrad_dma(int K, int C) { return K % 64 == 0 && C % 8 == 0; }
// (measured on the ResNet-50 shapes at batch 128: 128 x 128 tiles pay once
// the pixel count is large enough to split them over the CUs, 128 x 64 below;
// a third ring stage pays only for the single 64-column tile; 64 x 192 tiles
// cover a 3x3 64-channel filter's 576 columns exactly, where 64 x 256 tiles
// left a quarter of the third tile empty: conv2_x 60.4 -> 53.5 us)
inline WCfg wgrad7_cfg(int K, int Nw, int64_t npix) {
  if (K >= 128 && Nw >= 128 && npix >= 65536) return {128, 128};
  if (K >= 128 && Nw <= 64) return {128, 64, 3};
  if (K >= 128) return {128, 64};
  if (Nw % 192 == 0) return {64, 192};
  if (Nw >= 256) return {64, 256};
  if (Nw >= 128) return {64, 128};
  return {64, 64};
}
inline WCfg wgrad_choice(int K, int C, int Nw, int64_t npix) {
  return wgrad_dma(K, C) ? wgrad7_cfg(K, Nw, npix) : wgrad_cfg(K, Nw);
}

template <bool CGEN>
void launch_wgrad7(const WCfg& cfg, dim3 grid, hipStream_t st, const WgradArgs& a) {
  if (cfg.BM == 128 && cfg.BN == 128)
    hipLaunchKernelGGL((wgrad7_kernel<128, 128, 2, 2, 2, CGEN>), grid, dim3(256), 0, st, a);
  else if (cfg.BM == 128 && cfg.S == 3)
    hipLaunchKernelGGL((wgrad7_kernel<128, 64, 2, 2, 3, CGEN>), grid, dim3(256), 0, st, a);
  else if (cfg.BM == 128)
    hipLaunchKernelGGL((wgrad7_kernel<128, 64, 2, 2, 2, CGEN>), grid, dim3(256), 0, st, a);
  else if (cfg.BN == 256)
    hipLaunchKernelGGL((wgrad7_kernel<64, 256, 1, 4, 2, CGEN>), grid, dim3(256), 0, st, a);
  else if (cfg.BN == 192)
    hipLaunchKernelGGL((wgrad7_kernel<64, 192, 2, 2, 2, CGEN>), grid, dim3(256), 0, st, a);
  else if (cfg.BN == 128)
    hipLaunchKernelGGL((wgrad7_kernel<64, 128, 2, 2, 2, CGEN>), grid, dim3(256), 0, st, a);
  else
    hipLaunchKernelGGL((wgrad7_kernel<64, 64, 2, 2, 2, CGEN>), grid, dim3(256), 0, st, a);
}

}  // namespace

void wgrad_plan(int K, int Cp, int R, int S, int64_t npix, int target, int* splits,
                int* pix_per_split) {
  const int Nw = R * S * Cp;
  const WCfg cfg = wgrad_choice(K, Cp, Nw, npix);
  const int64_t tiles = (int64_t)ceil_div(K, cfg.BM) * ceil_div(Nw, cfg.BN);
  int64_t want = (target + tiles - 1) / tiles;  // about `target` workgroups
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
  const int64_t npix = (int64_t)a.N * a.P * a.Q;
  const WCfg cfg = wgrad_choice(a.K, a.C, Nw, npix);
  const int tiles = ceil_div(a.K, cfg.BM) * ceil_div(Nw, cfg.BN);
  dim3 grid(tiles, a.splits);
  if (wgrad_dma(a.K, a.C)) {
    // channel counts that are multiples of 8 only (the 3-channel stem, padded)
    // take per-lane filter taps
    if (a.C % 64 != 0)
      launch_wgrad7<true>(cfg, grid, st, a);
    else
      launch_wgrad7<false>(cfg, grid, st, a);
    return hipGetLastError();
  }
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

// Split-K partial sums folded in place: block (b, g) adds, for the 64
// float4 columns [64b, 64b + 64) of the split rows (row4 float4 each), the
// splits [g*kFoldGs, (g+1)*kFoldGs) of group g and writes the sum over the
// group's first split.  Wave w takes the group's splits w, w + 4, ... in
// order (all of its loads in flight; a split past the last is loaded
// clamped, in bounds, and not added), then the four wave sums are added in
// order.  Only this block reads or writes these elements of these splits.
constexpr int kFoldGs = 16;

__global__ __launch_bounds__(256) void wgrad_fold_kernel(float* part, int splits, int64_t row4) {
  __shared__ float4 red[3][64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t col = (int64_t)blockIdx.x * 64 + lane;
  const bool live = col < row4;
  const int64_t cc = live ? col : 0;
  const int g0 = blockIdx.y * kFoldGs;
  float4* p = reinterpret_cast<float4*>(part);
  constexpr int U = kFoldGs / 4;
  float4 v[U];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int sp = g0 + w + 4 * u;
    v[u] = p[(int64_t)(sp < splits ? sp : splits - 1) * row4 + cc];
  }
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
  for (int u = 0; u < U; ++u) {
    if (g0 + w + 4 * u < splits) {
      acc.x += v[u].x;
      acc.y += v[u].y;
      acc.z += v[u].z;
      acc.w += v[u].w;
    }
  }
  if (w > 0) red[w - 1][lane] = acc;
  __syncthreads();
  if (w != 0 || !live) return;
#pragma unroll
  for (int i = 0; i < 3; ++i) {
    acc.x += red[i][lane].x;
    acc.y += red[i][lane].y;
    acc.z += red[i][lane].z;
    acc.w += red[i][lane].w;
  }
  p[(int64_t)g0 * row4 + col] = acc;
}

// The stem's weight gradient computed as a 4x4 stride-1 convolution over the
// 2x2 space-to-depth image (16 channels, (dh*2 + dw)*3 + c): original tap
// (r, s, c) is s2d tap ((r+1)/2, (s+1)/2) at channel (((r+1)%2)*2 + (s+1)%2)*3
// + c.  dw[k][r][s][c] (KRSC, 7x7x3) = rne16(sum over the groups, in order, of
// the folded partial[g * kFoldGs][k][(r'*4 + s')*16 + ch]).
__global__ __launch_bounds__(256) void wgrad_reduce_s2d3_kernel(const float* __restrict__ partial,
                                                                 int groups, int64_t stride,
                                                                 int K, h16* __restrict__ dw) {
  const int i = blockIdx.x * 256 + threadIdx.x;  // enumerates k, r, s, c
  if (i >= K * 147) return;
  const int c = i % 3, rs = (i / 3) % 49, k = i / 147;
  const int r = rs / 7, s = rs % 7;
  const int rp = (r + 1) >> 1, sp = (s + 1) >> 1;
  const int ch = (((r + 1) & 1) * 2 + ((s + 1) & 1)) * 3 + c;
  const float* p = partial + (int64_t)k * 256 + (rp * 4 + sp) * 16 + ch;
  constexpr int U = 8;
  float acc = 0.0f;
  for (int g0 = 0; g0 < groups; g0 += U) {
    float v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = p[(int64_t)(g0 + u < groups ? g0 + u : groups - 1) * stride];
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (g0 + u < groups) acc += v[u];
  }
  dw[i] = to_h16(acc);
}

hipError_t launch_wgrad_reduce_s2d3(float* partial, int splits, int K, h16* dw, hipStream_t st) {
  const int64_t row4 = (int64_t)K * 256 / 4;
  const int groups = (splits + kFoldGs - 1) / kFoldGs;
  hipLaunchKernelGGL(wgrad_fold_kernel, dim3((unsigned)((row4 + 63) / 64), groups), dim3(256), 0,
                     st, partial, splits, row4);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(wgrad_reduce_s2d3_kernel, dim3((K * 147 + 255) / 256), dim3(256), 0, st,
                     partial, groups, (int64_t)kFoldGs * K * 256, K, dw);
  return hipGetLastError();
}

hipError_t launch_wgrad_reduce(const float* partial, int splits, int K, int Kp, int R, int S, int C,
                               int Cp, int layout, h16* dw, hipStream_t st) {
  const int64_t total = (int64_t)K * R * S * C;
  if (layout == 0 && C == Cp && splits <= 32) {
    const int64_t threads = total / 4;  // C % 8 == 0 here
    hipLaunchKernelGGL(wgrad_reduce_vec_kernel, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0,
                       st, partial, splits, total, (int64_t)Kp * R * S * Cp, dw);
    return hipGetLastError();
  }
  const int64_t blocks = (total + 63) / 64;
  hipLaunchKernelGGL(wgrad_reduce_kernel, dim3((unsigned)blocks), dim3(256), 0, st, partial, splits,
                     K, Kp, R, S, C, Cp, layout, dw);
  return hipGetLastError();
}

}  // namespace fp16k
