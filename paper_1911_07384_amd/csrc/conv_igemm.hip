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
// walks k in steps of 32, staging A and B tiles through LDS (double
// buffered, one barrier per step).  Each wave owns a (BM/WM) x (BN/WN)
// sub-tile computed with v_mfma_f32_32x32x16_f16 (float32 accumulators).
// The epilogue rounds each float32 sum once to binary16 (RNE), optionally
// after adding a binary16 addend in float32.

#include "kernels.hpp"

namespace fp16k {
namespace {

constexpr int BK = 32;        // k-step (halves)
constexpr int LDK = BK + 8;   // LDS row pitch in halves (16-byte pad)

template <int BM, int BN, int WM, int WN>
__global__ __launch_bounds__(256) void igemm_kernel(const IgemmArgs a) {
  constexpr int WTM = BM / WM, WTN = BN / WN;
  constexpr int TM = WTM / 32, TN = WTN / 32;
  constexpr int A_IT = BM * (BK / 8) / 256;
  constexpr int B_IT = BN * (BK / 8) / 256;
  static_assert(WM * WN == 4, "four waves");
  static_assert(TM >= 1 && TN >= 1 && A_IT >= 1 && B_IT >= 1, "tile shape");

  __shared__ __attribute__((aligned(16))) h16 As[2][BM * LDK];
  __shared__ __attribute__((aligned(16))) h16 Bs[2][BN * LDK];

  const IgemmPhase ph = a.ph[blockIdx.z];
  const int HoWo = ph.Ho * ph.Wo;
  const int M = a.N * HoWo;
  const int m0 = blockIdx.x * BM;
  if (m0 >= M) return;  // this phase has fewer rows than the grid covers
  const int n0 = blockIdx.y * BN;
  const int Ci = a.Ci;
  const int Kg = ph.Rt * ph.St * Ci;
  const int tid = threadIdx.x;
  const int kc = tid & 3;     // 8-element chunk of the 32-wide k-step
  const int rbase = tid >> 2; // 0..63

  // Gather state of the A rows this thread loads.
  int64_t a_base[A_IT];
  int a_ih0[A_IT], a_iw0[A_IT];
#pragma unroll
  for (int it = 0; it < A_IT; ++it) {
    const int m = m0 + rbase + it * 64;
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
      const int n = n0 + rbase + it * 64;
      rb[it] = (kval && n < a.Co) ? load16(ph.filt + (int64_t)n * ph.ldb + kk) : zero8();
    }
  };
  auto store_tile = [&](int buf) {
#pragma unroll
    for (int it = 0; it < A_IT; ++it)
      store16(&As[buf][(rbase + it * 64) * LDK + kc * 8], ra[it]);
#pragma unroll
    for (int it = 0; it < B_IT; ++it)
      store16(&Bs[buf][(rbase + it * 64) * LDK + kc * 8], rb[it]);
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
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      half8 af[TM], bf[TN];
#pragma unroll
      for (int tm = 0; tm < TM; ++tm)
        af[tm] = *reinterpret_cast<const half8*>(
            &As[buf][(wm * WTM + tm * 32 + lrow) * LDK + ks * 16 + lk]);
#pragma unroll
      for (int tn = 0; tn < TN; ++tn)
        bf[tn] = *reinterpret_cast<const half8*>(
            &Bs[buf][(wn * WTN + tn * 32 + lrow) * LDK + ks * 16 + lk]);
#pragma unroll
      for (int tm = 0; tm < TM; ++tm)
#pragma unroll
        for (int tn = 0; tn < TN; ++tn) acc[tm][tn] = mfma32x32x16(af[tm], bf[tn], acc[tm][tn]);
    }
    if (kt + 1 < KT) store_tile(buf ^ 1);
    __syncthreads();
  }

  // Epilogue: accumulator element e of lane l is row 8*(e/4) + 4*(l/32) + e%4,
  // column l%32 of the 32x32 block.  One RNE rounding to binary16 per output.
#pragma unroll
  for (int tm = 0; tm < TM; ++tm) {
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int m = m0 + wm * WTM + tm * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
      if (m >= M) continue;
      const int img = m / HoWo;
      const int rem = m - img * HoWo;
      const int i = rem / ph.Wo;
      const int j = rem - i * ph.Wo;
      const int oh = i * a.os_h + ph.oph;
      const int ow = j * a.os_w + ph.opw;
      const int64_t obase = ((int64_t)(img * a.OH + oh) * a.OW + ow) * a.ldo;
      h16* orow = a.out + obase;
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) {
        const int n = n0 + wn * WTN + tn * 32 + lrow;
        if (n < a.Co) {
          float v = acc[tm][tn][e];
          if (a.addend) v += to_f32(a.addend[obase + n]);
          orow[n] = to_h16(v);
        }
      }
    }
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
  if (a.Co <= 64) return launch_cfg<128, 64, 2, 2>(a, st);
  return launch_cfg<128, 128, 2, 2>(a, st);
}

}  // namespace fp16k
