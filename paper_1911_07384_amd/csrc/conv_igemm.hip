// Implicit-GEMM convolution on the gfx950 FP16 matrix cores (forward pass,
// and the data gradient expressed as stride-1 gathers per stride phase).
//
// GEMM view (NHWC activations, filter rows contiguous over taps x channels):
//   C[m][n] = sum_k A[m][k] * B[n][k]
//   m = (image, i, j) over the phase's output grid, n = output channel,
//   k = (r, s, c) with c fastest,
//   A[m][k] = act[image][i*stride_h - pad_h + r][j*stride_w - pad_w + s][c]
//             (zero outside the source image),
//   B[n][k] = filt[n][k].
// Both operands are contiguous along k in runs of Ci channels, so 16-byte
// (8 x binary16) vector loads feed the MFMA operand layout directly.
//
// Tiling: a 256-thread workgroup (4 wave64s) owns a BM x BN output tile and
// walks k in steps of 64, staging A and B tiles through LDS (double
// buffered, one barrier per step; the next step's global loads are in
// flight while the current one is multiplied).  Each wave owns a
// (BM/WM) x (BN/WN) sub-tile computed with v_mfma_f32_32x32x16_f16 into
// float32 accumulators.
//
// Epilogue: each wave stages one 32-row band of its float32 tile in LDS and
// writes it back row by row with 16-byte stores (eight channels per lane,
// whole output rows per instruction).  Every value is rounded once to
// binary16 (RNE), optionally after adding a binary16 addend in float32.

#include "kernels.hpp"

namespace fp16k {
namespace {

constexpr int BK = 64;        // k-step (halves)
constexpr int LDK = BK + 8;   // LDS row pitch in halves (16-byte pad)

template <int BM, int BN, int WM, int WN>
struct Cfg {
  static constexpr int WTM = BM / WM, WTN = BN / WN;
  static constexpr int TM = WTM / 32, TN = WTN / 32;
  static constexpr int A_IT = BM * (BK / 8) / 256;
  static constexpr int B_IT = BN * (BK / 8) / 256;
  static constexpr int SP = WTN + 4;  // staging row pitch (floats)
  static constexpr int MAIN_BYTES = 2 * (BM + BN) * LDK * 2;
  static constexpr int STAGE_BYTES = 4 * 32 * SP * 4;
  static constexpr int LDS_BYTES = MAIN_BYTES > STAGE_BYTES ? MAIN_BYTES : STAGE_BYTES;
};

template <int BM, int BN, int WM, int WN>
__global__ __launch_bounds__(256) void igemm_kernel(const IgemmArgs a) {
  using K = Cfg<BM, BN, WM, WN>;
  constexpr int WTM = K::WTM, WTN = K::WTN, TM = K::TM, TN = K::TN;
  constexpr int A_IT = K::A_IT, B_IT = K::B_IT;
  static_assert(WM * WN == 4, "four waves");
  static_assert(TM >= 1 && TN >= 1 && A_IT >= 1 && B_IT >= 1, "tile shape");

  __shared__ __attribute__((aligned(16))) char smem[K::LDS_BYTES];
  h16* As = reinterpret_cast<h16*>(smem);   // [2][BM][LDK]
  h16* Bs = As + 2 * BM * LDK;             // [2][BN][LDK]

  const IgemmPhase ph = a.ph[blockIdx.z];
  const int HoWo = ph.Ho * ph.Wo;
  const int M = a.N * HoWo;
  const int m0 = blockIdx.x * BM;
  if (m0 >= M) return;  // this phase has fewer rows than the grid covers
  const int n0 = blockIdx.y * BN;
  const int Ci = a.Ci;
  const int Kg = ph.Rt * ph.St * Ci;
  const int tid = threadIdx.x;
  const int kc = tid & 7;      // 8-element chunk of the 64-wide k-step
  const int rbase = tid >> 3;  // 0..31

  // Gather state of the A rows this thread loads.
  int64_t a_base[A_IT];
  int a_ih0[A_IT], a_iw0[A_IT];
#pragma unroll
  for (int it = 0; it < A_IT; ++it) {
    const int m = m0 + rbase + it * 32;
    if (m < M) {
      const int img = m / HoWo;
      const int rem = m - img * HoWo;
      const int i = rem / ph.Wo;
      const int j = rem - i * ph.Wo;
      a_base[it] = (int64_t)img * a.Hi * a.Wi * Ci;
      a_ih0[it] = i * a.stride_h - ph.pad_h;
      a_iw0[it] = j * a.stride_w - ph.pad_w;
    } else {
      a_base[it] = 0;
      a_ih0[it] = -(1 << 28);  // every tap falls outside the image
      a_iw0[it] = 0;
    }
  }

  V8 ra[A_IT], rb[B_IT];
  auto load_tile = [&](int k0) {
    const int kk = k0 + kc * 8;
    const bool kval = kk < Kg;
    const int tap = kval ? kk / Ci : 0;
    const int c = kk - tap * Ci;
    const int r = tap / ph.St;
    const int s = tap - r * ph.St;
#pragma unroll
    for (int it = 0; it < A_IT; ++it) {
      const int ih = a_ih0[it] + r;
      const int iw = a_iw0[it] + s;
      const bool v = kval && (unsigned)ih < (unsigned)a.Hi && (unsigned)iw < (unsigned)a.Wi;
      ra[it] = v ? load16(a.act + a_base[it] + (int64_t)(ih * a.Wi + iw) * Ci + c) : zero8();
    }
#pragma unroll
    for (int it = 0; it < B_IT; ++it) {
      const int n = n0 + rbase + it * 32;
      rb[it] = (kval && n < a.Co) ? load16(ph.filt + (int64_t)n * ph.ldb + kk) : zero8();
    }
  };
  auto store_tile = [&](int buf) {
    h16* as = As + buf * BM * LDK;
    h16* bs = Bs + buf * BN * LDK;
#pragma unroll
    for (int it = 0; it < A_IT; ++it) store16(&as[(rbase + it * 32) * LDK + kc * 8], ra[it]);
#pragma unroll
    for (int it = 0; it < B_IT; ++it) store16(&bs[(rbase + it * 32) * LDK + kc * 8], rb[it]);
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

  const int KT = (Kg + BK - 1) / BK;
  if (KT > 0) {
    load_tile(0);
    store_tile(0);
  }
  __syncthreads();
  for (int kt = 0; kt < KT; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < KT) load_tile((kt + 1) * BK);
    const h16* as = As + buf * BM * LDK;
    const h16* bs = Bs + buf * BN * LDK;
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      half8 af[TM], bf[TN];
#pragma unroll
      for (int tm = 0; tm < TM; ++tm)
        af[tm] = *reinterpret_cast<const half8*>(&as[(wm * WTM + tm * 32 + lrow) * LDK + ks * 16 + lk]);
#pragma unroll
      for (int tn = 0; tn < TN; ++tn)
        bf[tn] = *reinterpret_cast<const half8*>(&bs[(wn * WTN + tn * 32 + lrow) * LDK + ks * 16 + lk]);
#pragma unroll
      for (int tm = 0; tm < TM; ++tm)
#pragma unroll
        for (int tn = 0; tn < TN; ++tn) acc[tm][tn] = mfma32x32x16(af[tm], bf[tn], acc[tm][tn]);
    }
    if (kt + 1 < KT) store_tile(buf ^ 1);
    __syncthreads();
  }

  // ---- epilogue -------------------------------------------------------------
  // Accumulator element e of lane l is row 8*(e/4) + 4*(l/32) + e%4, column
  // l%32 of its 32x32 block.  Stage one 32 x WTN band per wave in LDS, then
  // each lane writes eight consecutive channels of one row.
  float* stg = reinterpret_cast<float*>(smem) + wave * 32 * K::SP;
  constexpr int CPR = WTN / 8;         // 16-byte chunks per band row
  constexpr int RPP = 64 / CPR;        // rows per pass
  const int cc = lane % CPR;
  const int rr = lane / CPR;
  const int n = n0 + wn * WTN + cc * 8;
  const bool vec_ok = (a.ldo % 8) == 0 && n + 8 <= a.Co;
#pragma unroll
  for (int tm = 0; tm < TM; ++tm) {
#pragma unroll
    for (int tn = 0; tn < TN; ++tn)
#pragma unroll
      for (int e = 0; e < 16; ++e)
        stg[(8 * (e >> 2) + 4 * (lane >> 5) + (e & 3)) * K::SP + tn * 32 + lrow] = acc[tm][tn][e];
    __syncthreads();
#pragma unroll
    for (int pass = 0; pass < 32 / RPP; ++pass) {
      const int r = pass * RPP + rr;
      const int m = m0 + wm * WTM + tm * 32 + r;
      if (m < M && n < a.Co) {
        const int img = m / HoWo;
        const int rem = m - img * HoWo;
        const int i = rem / ph.Wo;
        const int j = rem - i * ph.Wo;
        const int oh = i * a.os_h + ph.oph;
        const int ow = j * a.os_w + ph.opw;
        const int64_t off = ((int64_t)(img * a.OH + oh) * a.OW + ow) * a.ldo + n;
        const float* src = stg + r * K::SP + cc * 8;
        float v[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = src[e];
        if (vec_ok) {
          if (a.addend) {
            const V8 ad = load16(a.addend + off);
#pragma unroll
            for (int e = 0; e < 8; ++e) v[e] += to_f32(ad.h[e]);
          }
          V8 o;
#pragma unroll
          for (int e = 0; e < 8; ++e) o.h[e] = to_h16(v[e]);
          store16(a.out + off, o);
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            if (n + e < a.Co) {
              float x = v[e];
              if (a.addend) x += to_f32(a.addend[off + e]);
              a.out[off + e] = to_h16(x);
            }
          }
        }
      }
    }
    __syncthreads();
  }
}

template <int BM, int BN, int WM, int WN>
hipError_t launch_cfg(const IgemmArgs& a, hipStream_t st) {
  int maxM = 0;
  for (int p = 0; p < a.nphase; ++p) {
    const int m = a.N * a.ph[p].Ho * a.ph[p].Wo;
    if (m > maxM) maxM = m;
  }
  if (maxM == 0 || a.nphase == 0) return hipSuccess;
  dim3 grid(ceil_div(maxM, BM), ceil_div(a.Co, BN), a.nphase);
  hipLaunchKernelGGL((igemm_kernel<BM, BN, WM, WN>), grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_igemm(const IgemmArgs& a, hipStream_t st) {
  if (a.Co <= 64) return launch_cfg<128, 64, 4, 1>(a, st);
  return launch_cfg<128, 128, 2, 2>(a, st);
}

}  // namespace fp16k
