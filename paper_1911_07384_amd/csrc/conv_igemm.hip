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
// (8 x binary16) vector loads feed the MFMA operand layout directly.  All
// loads are buffer loads against a range-checked resource: a tap outside the
// image (or a row past the end) gets an out-of-range offset and reads zeros,
// with no branch.
//
// Three kernels, all v_mfma_f32_32x32x16_f16 with float32 accumulators and
// the same k order (so they give identical bits):
//   igemm_kernel  -- 4 waves in a 2x2 or 4x1 grid; A and B tiles staged in
//                    LDS through registers, k-step 64, double buffered.
//   igemm4_kernel -- 4 waves split M only, so no A element is shared: each
//                    lane loads its own MFMA operand rows from global memory
//                    into registers three k-steps ahead, and only the filter
//                    tile goes through LDS, by DMA (buffer_load ... lds) into
//                    four stage buffers with XOR-swizzled rows.  Needs
//                    Ci % 32 == 0.  Less LDS traffic per MFMA; wins on short
//                    reductions and small M.
//   igemm7_kernel -- both operands DMA'd straight from global memory into a
//                    ring of LDS stages, k-step 64 so that each operand row
//                    of a stage is one whole 128-byte line, per-row tap masks
//                    precomputed so a DMA costs a few ALU operations, and the
//                    MFMA operands read one k sub-step ahead.  Needs
//                    Ci % 64 == 0; wins on the long reductions (every 3x3
//                    layer).
//   pw_kernel     -- 1x1 filters with 64 or 128 input channels (or 256
//                    without an addend) and a dense output of 128+ channels
//                    (bound by the output's bytes): the filter tile stays in
//                    LDS, each workgroup walks over 128-row tiles, and the
//                    MFMA operands are swapped so that the accumulators hold
//                    the transposed tile; lane-pair swaps (v_permlane32_swap)
//                    then give each lane 8 consecutive channels of one output
//                    pixel, staged through LDS into whole-line stores.  Its
//                    epilogue can take the following BN's statistics, or
//                    (a second pass) apply that BN to the recomputed output.
//
// Epilogue (the first three): each wave stages a 32-row band of its float32
// tile in LDS and writes whole output rows with 16-byte stores.  Every value is rounded
// once to binary16 (RNE), optionally after adding a binary16 addend in
// float32.  igemm4_kernel and igemm7_kernel can also take the statistics of a
// BN that follows the convolution, without a second pass over the output:
// per 128-row tile and channel, shifted sums of the rounded values
// (IgemmArgs::stat).

#include "kernels.hpp"


namespace fp16k {
namespace {

// The addend of the 8 outputs at element offset off (a multiple of 8) under
// the ReLU mask byte mb of those 8 (bit e for element off + e): an element
// whose bit is clear adds +0.
__device__ __forceinline__ V8 masked8(V8 v, uint32_t mb) {
#pragma unroll
  for (int e = 0; e < 8; ++e) v.s[e] = ((mb >> e) & 1u) ? v.s[e] : (uint16_t)0;
  return v;
}
__device__ __forceinline__ V8 addend8(const IgemmArgs& a, int64_t off) {
  const V8 v = load16(a.addend + off);
  return a.amask ? masked8(v, a.amask[off >> 3]) : v;
}
// Element offset in the addend of output pixel (img, oh, ow), or -1 where a
// strided addend (IgemmArgs::astride) has no element (the pixel adds +0).
__device__ __forceinline__ int64_t addend_row(const IgemmArgs& a, int img, int oh, int ow) {
  if (a.astride <= 1) return ((int64_t)(img * a.OH + oh) * a.OW + ow) * a.ldo;
  if (oh % a.astride != 0 || ow % a.astride != 0) return -1;
  const int AH = (a.OH + a.astride - 1) / a.astride, AW = (a.OW + a.astride - 1) / a.astride;
  return ((int64_t)(img * AH + oh / a.astride) * AW + ow / a.astride) * a.ldo;
}
// one element of the addend, under the mask
__device__ __forceinline__ float addend1(const IgemmArgs& a, int64_t i) {
  const float v = to_f32(a.addend[i]);
  return (a.amask && !((a.amask[i >> 3] >> (i & 7)) & 1u)) ? 0.0f : v;
}

// keep a value materialised in a VGPR (blocks branchy code motion around it)
__device__ __forceinline__ uint32_t pin_v(uint32_t x) {
  __asm__("" : "+v"(x));
  return x;
}
// workgroup barrier without the implied memory fence; callers wait first
__device__ __forceinline__ void bare_barrier() { __asm__ volatile("s_barrier" ::: "memory"); }
// Tile of this workgroup, for grids of (M-tiles, N-tiles, phases).
// Workgroups are dealt to the 8 XCDs round-robin in launch order (M fastest).
// With gn > 0 each XCD takes a contiguous run of tiles instead, in an order
// that walks groups of gn N-tiles (N fastest, then M), so that its run is a
// compact block of M-tiles x N-tiles whose activation rows are read once into
// that XCD's L2 and shared by its N-tiles.
__device__ __forceinline__ void xcd_tile(int gn, int& z, int& mt, int& nt) {
  if (gn <= 0) {
    z = blockIdx.z;
    mt = blockIdx.x;
    nt = blockIdx.y;
    return;
  }
  const int MT = gridDim.x, NT = gridDim.y, NZ = gridDim.z;
  const int total = MT * NT * NZ;
  const int L = (blockIdx.z * NT + blockIdx.y) * MT + blockIdx.x;
  const int q = total >> 3, r = total & 7, xcd = L & 7;
  const int t = xcd * q + (xcd < r ? xcd : r) + (L >> 3);
  const int u = t / NZ;
  z = t - u * NZ;
  const int g = u / (gn * MT);
  const int w = u - g * gn * MT;
  const int gw = NT - g * gn < gn ? NT - g * gn : gn;
  nt = g * gn + w % gw;
  mt = w / gw;
}

template <int BM, int BN, int WM, int WN, int BK>
struct Cfg {
  static constexpr int LDK = BK + 8;
  static constexpr int KC = BK / 8;           // 16-byte chunks per tile row
  static constexpr int RSTEP = 256 / KC;      // rows covered per load pass
  static constexpr int WTM = BM / WM, WTN = BN / WN;
  static constexpr int TM = WTM / 32, TN = WTN / 32;
  static constexpr int A_IT = BM / RSTEP;
  static constexpr int B_IT = BN / RSTEP;
  static constexpr int SP = WTN + 4;
  static constexpr int MAIN_BYTES = 2 * (BM + BN) * LDK * 2;
  static constexpr int STAGE_BYTES = 4 * 32 * SP * 4;
  static constexpr int LDS_BYTES = MAIN_BYTES > STAGE_BYTES ? MAIN_BYTES : STAGE_BYTES;
};

template <int BM, int BN, int WM, int WN, int BK>
__global__ __launch_bounds__(256) void igemm_kernel(const IgemmArgs a) {
  using K = Cfg<BM, BN, WM, WN, BK>;
  constexpr int LDK = K::LDK, KC = K::KC, RSTEP = K::RSTEP;
  constexpr int WTM = K::WTM, WTN = K::WTN, TM = K::TM, TN = K::TN;
  constexpr int A_IT = K::A_IT, B_IT = K::B_IT;
  static_assert(WM * WN == 4, "four waves");
  static_assert(TM >= 1 && TN >= 1 && A_IT >= 1 && B_IT >= 1, "tile shape");

  __shared__ __attribute__((aligned(16))) char smem[K::LDS_BYTES];
  h16* As = reinterpret_cast<h16*>(smem);
  h16* Bs = As + 2 * BM * LDK;

  int tz, tm_, tn_;
  xcd_tile(a.gn, tz, tm_, tn_);
  const IgemmPhase ph = a.ph[tz];
  const int HoWo = ph.Ho * ph.Wo;
  const int M = a.N * HoWo;
  const int m0 = tm_ * BM;
  if (m0 >= M) return;
  const int n0 = tn_ * BN;
  const int Ci = a.Ci;
  const int Kg = ph.Rt * ph.St * Ci;
  const int tid = threadIdx.x;
  const int kc = tid % KC;
  const int rbase = tid / KC;

  int64_t a_base[A_IT];
  int a_ih0[A_IT], a_iw0[A_IT];
#pragma unroll
  for (int it = 0; it < A_IT; ++it) {
    const int m = m0 + rbase + it * RSTEP;
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
      a_ih0[it] = -(1 << 28);
      a_iw0[it] = 0;
    }
  }

  // range-checked buffer loads: an offset past the end reads zeros, no branch
  const uint32_t act_bytes = (uint32_t)((int64_t)a.N * a.Hi * a.Wi * Ci * 2);
  const __amdgpu_buffer_rsrc_t rs_a = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<h16*>(a.act), (short)0, (int)act_bytes, 0x00020000);
  const uint32_t filt_bytes = (uint32_t)((int64_t)a.Co * ph.ldb * 2);
  const __amdgpu_buffer_rsrc_t rs_b = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<h16*>(ph.filt), (short)0, (int)filt_bytes, 0x00020000);
  constexpr uint32_t OOB = 0x80000000u;
  uint32_t a_off[A_IT];
#pragma unroll
  for (int it = 0; it < A_IT; ++it) a_off[it] = (uint32_t)(a_base[it] * 2);
  auto load_tile = [&](int k0, V8 (&ra)[A_IT], V8 (&rb)[B_IT]) {
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
      const uint32_t off = v ? a_off[it] + (uint32_t)((ih * a.Wi + iw) * Ci + c) * 2u : OOB;
      ra[it].u = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs_a, off, 0, 0));
    }
#pragma unroll
    for (int it = 0; it < B_IT; ++it) {
      const int n = n0 + rbase + it * RSTEP;
      const uint32_t off = (kval && n < a.Co) ? (uint32_t)(n * ph.ldb + kk) * 2u : OOB;
      rb[it].u = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs_b, off, 0, 0));
    }
  };
  auto store_tile = [&](int buf, const V8 (&ra)[A_IT], const V8 (&rb)[B_IT]) {
    h16* as = As + buf * BM * LDK;
    h16* bs = Bs + buf * BN * LDK;
#pragma unroll
    for (int it = 0; it < A_IT; ++it) store16(&as[(rbase + it * RSTEP) * LDK + kc * 8], ra[it]);
#pragma unroll
    for (int it = 0; it < B_IT; ++it) store16(&bs[(rbase + it * RSTEP) * LDK + kc * 8], rb[it]);
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

  auto compute = [&](int buf) {
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
        for (int tn = 0; tn < TN; ++tn) {
          acc[tm][tn] = mfma32x32x16(af[tm], bf[tn], acc[tm][tn]);
        }
    }
  };

  const int KT = (Kg + BK - 1) / BK;
  V8 ra0[A_IT], rb0[B_IT];
  if (KT > 0) {
    load_tile(0, ra0, rb0);
    store_tile(0, ra0, rb0);
  }
  __syncthreads();
  for (int kt = 0; kt < KT; ++kt) {
    if (kt + 1 < KT) load_tile((kt + 1) * BK, ra0, rb0);
    compute(kt & 1);
    if (kt + 1 < KT) store_tile((kt + 1) & 1, ra0, rb0);
    __syncthreads();
  }

  float* stg = reinterpret_cast<float*>(smem) + wave * 32 * K::SP;
  constexpr int CPR = WTN / 8;
  constexpr int RPP = 64 / CPR;
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
            const int64_t ar = addend_row(a, img, oh, ow);
            const V8 ad = ar >= 0 ? addend8(a, ar + n) : zero8();
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
              if (a.addend) {
                const int64_t ar = addend_row(a, img, oh, ow);
                x += ar >= 0 ? addend1(a, ar + n + e) : 0.0f;
              }
              a.out[off + e] = to_h16(x);
            }
          }
        }
      }
    }
    __syncthreads();
  }
}



// ---- A from global into VGPRs, B (filter) through LDS by DMA ---------------
// Four waves split M only, so no A element is shared between waves: each
// lane loads its own MFMA operand rows (16 bytes = 8 channels) straight into
// registers, three k-steps ahead.  The filter tile, shared by all waves, is
// DMA'd into one of four LDS stage buffers (k-step 32, XOR-swizzled 64-byte
// rows).  Wave tile = 32*TM x 32*TN; workgroup tile = 128*TM x 32*TN.
template <int TM, int TN>
struct Cfg4 {
  static constexpr int BM = 4 * 32 * TM, BN = 32 * TN;
  static constexpr int B_INS = BN / 64;                 // DMA instructions per wave per stage
  static constexpr int SP = 64 + 4;                     // epilogue staging pitch (64-column chunks)
  static constexpr int BUF = (BN * 64 > 32 * SP * 4) ? BN * 64 : 32 * SP * 4;
};

template <int TM, int TN>
__global__ __launch_bounds__(256) void igemm4_kernel(const IgemmArgs a) {
  using K = Cfg4<TM, TN>;
  constexpr int BM = K::BM, BN = K::BN, B_INS = K::B_INS;
  static_assert(B_INS >= 1 && TN % 2 == 0, "tile shape");
  __shared__ __attribute__((aligned(1024))) char lds0[K::BUF];
  __shared__ __attribute__((aligned(1024))) char lds1[K::BUF];
  __shared__ __attribute__((aligned(1024))) char lds2[K::BUF];
  __shared__ __attribute__((aligned(1024))) char lds3[K::BUF];

  int tz, tm_, tn_;
  xcd_tile(a.gn, tz, tm_, tn_);
  const IgemmPhase ph = a.ph[tz];
  const int HoWo = ph.Ho * ph.Wo;
  const int M = a.N * HoWo;
  const int m0 = tm_ * BM;
  if (m0 >= M) return;
  const int n0 = tn_ * BN;
  const int Ci = a.Ci;
  const int Kg = ph.Rt * ph.St * Ci;
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const int lrow = lane & 31, lhi = lane >> 5;
  const int act_bytes = (int)((int64_t)a.N * a.Hi * a.Wi * Ci * 2);
  const int filt_bytes = (int)((int64_t)a.Co * ph.ldb * 2);
  constexpr uint32_t OOB = 0x80000000u;

  // A rows of this lane: wave*32*TM + tm*32 + lrow
  uint32_t a_off[TM];
  int a_ih0[TM], a_iw0[TM];
#pragma unroll
  for (int tm = 0; tm < TM; ++tm) {
    const int m = m0 + wave * 32 * TM + tm * 32 + lrow;
    if (m < M) {
      const int img = m / HoWo;
      const int rem = m - img * HoWo;
      const int i = rem / ph.Wo;
      const int j = rem - i * ph.Wo;
      a_off[tm] = (uint32_t)((int64_t)img * a.Hi * a.Wi * Ci * 2) + (uint32_t)lhi * 16u;
      a_ih0[tm] = i * a.stride_h - ph.pad_h;
      a_iw0[tm] = j * a.stride_w - ph.pad_w;
    } else {
      a_off[tm] = 0;
      a_ih0[tm] = -(1 << 28);
      a_iw0[tm] = 0;
    }
  }
  // B (filter) DMA: lane covers row (wave*B_INS + q)*16 + lane/4, slot lane%4
  const int chunk = (lane & 3) ^ ((lane >> 4) & 3);
  uint32_t b_off[B_INS];
#pragma unroll
  for (int q = 0; q < B_INS; ++q) {
    const int n = n0 + (wave * B_INS + q) * 16 + (lane >> 2);
    b_off[q] = n < a.Co ? (uint32_t)n * (uint32_t)ph.ldb * 2u + (uint32_t)chunk * 16u : OOB;
  }

  // k-step state (uniform; Ci % 32 == 0 so a step stays inside one tap)
  int k0 = 0, cb = 0, tr = 0, ts = 0;
  half8 A0[TM][2], A1[TM][2], A2[TM][2], A3[TM][2];

  auto issue = [&](char* bbuf, half8 (&Ar)[TM][2]) {
    const __amdgpu_buffer_rsrc_t rs_a = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<h16*>(a.act), (short)0, act_bytes, 0x00020000);
    const __amdgpu_buffer_rsrc_t rs_b = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<h16*>(ph.filt), (short)0, filt_bytes, 0x00020000);
    const bool kval = k0 < Kg;
#pragma unroll
    for (int q = 0; q < B_INS; ++q) {
      const uint32_t addr = pin_v(b_off[q] + (uint32_t)k0 * 2u);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          rs_b, (__attribute__((address_space(3))) void*)(bbuf + (wave * B_INS + q) * 1024), 16,
          kval ? addr : OOB, 0, 0, 0);
    }
#pragma unroll
    for (int tm = 0; tm < TM; ++tm) {
      const int ih = a_ih0[tm] + tr, iw = a_iw0[tm] + ts;
      const bool v = kval && (unsigned)ih < (unsigned)a.Hi && (unsigned)iw < (unsigned)a.Wi;
      const uint32_t addr = pin_v(a_off[tm] + (uint32_t)((ih * a.Wi + iw) * Ci + cb) * 2u);
      const uint32_t o = v ? addr : OOB;
#pragma unroll
      for (int ks = 0; ks < 2; ++ks)
        Ar[tm][ks] = __builtin_bit_cast(half8, __builtin_amdgcn_raw_buffer_load_b128(rs_a, o + ks * 32, 0, 0));
    }
    k0 += 32;
    cb += 32;
    if (cb == Ci) {
      cb = 0;
      if (++ts == ph.St) {
        ts = 0;
        ++tr;
      }
    }
  };

  floatx16 acc[TM][TN];
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int tn = 0; tn < TN; ++tn)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[tm][tn][e] = 0.0f;

  const int swz = (lrow >> 2) & 3;
  auto compute = [&](const char* bbuf, const half8 (&Ar)[TM][2]) {
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const int pos = ((ks * 2 + lhi) ^ swz) * 16;
      half8 bf[TN];
#pragma unroll
      for (int tn = 0; tn < TN; ++tn)
        bf[tn] = *reinterpret_cast<const half8*>(bbuf + (tn * 32 + lrow) * 64 + pos);
#pragma unroll
      for (int tm = 0; tm < TM; ++tm)
#pragma unroll
        for (int tn = 0; tn < TN; ++tn) acc[tm][tn] = mfma32x32x16(Ar[tm][ks], bf[tn], acc[tm][tn]);
    }
  };

  const int KT = (Kg + 31) / 32;
  issue(lds0, A0);
  issue(lds1, A1);
  issue(lds2, A2);
  constexpr int LPS = B_INS + 2 * TM;   // vector memory instructions per wave per stage
  constexpr int ALLOW = 2 * LPS;        // stages kt+1 and kt+2 stay in flight
  constexpr int WAIT = (0x0 << 8) | (0x7 << 4) | (ALLOW & 0xF) | ((ALLOW >> 4) << 14);
  // one loop exit (guarded steps, no breaks): the accumulators stay in one
  // register set instead of one copy per exit
  for (int kt = 0; kt < KT; kt += 4) {
    __builtin_amdgcn_s_waitcnt(WAIT);
    bare_barrier();
    issue(lds3, A3);
    compute(lds0, A0);
    if (kt + 1 < KT) {
      __builtin_amdgcn_s_waitcnt(WAIT);
      bare_barrier();
      issue(lds0, A0);
      compute(lds1, A1);
    }
    if (kt + 2 < KT) {
      __builtin_amdgcn_s_waitcnt(WAIT);
      bare_barrier();
      issue(lds1, A1);
      compute(lds2, A2);
    }
    if (kt + 3 < KT) {
      __builtin_amdgcn_s_waitcnt(WAIT);
      bare_barrier();
      issue(lds2, A2);
      compute(lds3, A3);
    }
  }
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();

  // epilogue: per wave, 32-row band x 64-column chunk staged in LDS buffer
  // `wave`, written back with 16-byte stores
  float* stg = reinterpret_cast<float*>(wave == 0 ? lds0 : wave == 1 ? lds1 : wave == 2 ? lds2 : lds3);
  const int cc = lane & 7;
  const int rr = lane >> 3;
  // BN statistics: per wave band (32 rows) and channel, the band's first
  // value K and sums of (y - K), (y - K)^2 over its rounded values; the four
  // bands of a 128-row tile are then combined (wave order) into one record
  __shared__ float bst[4][3][64];
  __shared__ int bcnt[4];
#pragma unroll
  for (int tm = 0; tm < TM; ++tm) {
#pragma unroll
    for (int nc = 0; nc < TN / 2; ++nc) {
#pragma unroll
      for (int t2 = 0; t2 < 2; ++t2)
#pragma unroll
        for (int e = 0; e < 16; ++e)
          stg[(8 * (e >> 2) + 4 * lhi + (e & 3)) * K::SP + t2 * 32 + lrow] = acc[tm][nc * 2 + t2][e];
      __syncthreads();
      const int n = n0 + nc * 64 + cc * 8;
      const bool vec_ok = (a.ldo % 8) == 0 && n + 8 <= a.Co;
      const int band_m0 = m0 + wave * 32 * TM + tm * 32;
      // statistics only for one 32-row band per wave (TM = 1): the four
      // waves' bands then form one 128-row tile
      const bool stats = TM == 1 && a.stat != nullptr;
      float K[8], s1[8], s2[8];
      if (stats) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          K[e] = to_f32(to_h16(stg[cc * 8 + e]));  // the band's first row, as stored
          s1[e] = 0.0f;
          s2[e] = 0.0f;
        }
      }
#pragma unroll
      for (int pass = 0; pass < 4; ++pass) {
        const int r = pass * 8 + rr;
        const int m = m0 + wave * 32 * TM + tm * 32 + r;
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
              const int64_t ar = addend_row(a, img, oh, ow);
            const V8 ad = ar >= 0 ? addend8(a, ar + n) : zero8();
#pragma unroll
              for (int e = 0; e < 8; ++e) v[e] += to_f32(ad.h[e]);
            }
            V8 o;
#pragma unroll
            for (int e = 0; e < 8; ++e) o.h[e] = to_h16(v[e]);
            store16(a.out + off, o);
            if (stats) {
#pragma unroll
              for (int e = 0; e < 8; ++e) {
                const float d = to_f32(o.h[e]) - K[e];
                s1[e] += d;
                s2[e] = __builtin_fmaf(d, d, s2[e]);
              }
            }
          } else {
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              if (n + e < a.Co) {
                float x = v[e];
                if (a.addend) {
                  const int64_t ar = addend_row(a, img, oh, ow);
                  x += ar >= 0 ? addend1(a, ar + n + e) : 0.0f;
                }
                a.out[off + e] = to_h16(x);
              }
            }
          }
        }
      }
      if (stats) {
        // lanes with the same 8 channels (lane bits 3-5) combine; lanes 0-7
        // hold the band's sums
#pragma unroll
        for (int sh = 8; sh < 64; sh <<= 1) {
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            s1[e] += __shfl_xor(s1[e], sh, 64);
            s2[e] += __shfl_xor(s2[e], sh, 64);
          }
        }
        if (lane < 8) {
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            bst[wave][0][cc * 8 + e] = K[e];
            bst[wave][1][cc * 8 + e] = s1[e];
            bst[wave][2][cc * 8 + e] = s2[e];
          }
        }
        if (lane == 0) {
          const int rows = M - band_m0;
          bcnt[wave] = rows <= 0 ? 0 : (rows < 32 ? rows : 32);
        }
      }
      if (stats) __syncthreads();
      if (stats && wave == 0 && bcnt[0] > 0 && n0 + nc * 64 + lane < a.Co) {
        // one record per 128-row tile: the bands re-based on the first
        // band's K (differences of two samples: no cancellation), wave order
        const int c = lane;
        const float K0 = bst[0][0][c];
        float S1 = 0.0f, S2 = 0.0f;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          const float nw = (float)bcnt[w];
          if (bcnt[w] == 0) break;
          const float d = bst[w][0][c] - K0;
          const float t1 = bst[w][1][c];
          S1 += __builtin_fmaf(nw, d, t1);
          S2 += __builtin_fmaf(nw * d, d, __builtin_fmaf(2.0f * d, t1, bst[w][2][c]));
        }
        const int tile = m0 / 128;
        float* rec = a.stat + (int64_t)tile * 3 * a.Co + n0 + nc * 64 + c;
        rec[0] = K0;
        rec[a.Co] = S1;
        rec[2 * a.Co] = S2;
      }
      __syncthreads();
    }
  }
}

// ---- pointwise (1x1) convolutions bound by the output's bytes ------------------
// For a 1x1 filter over CI = 64 or 128 input channels with 128+ output
// channels, writing y costs 2-4x more bytes than reading x.  Here:
//  - the BN x CI filter tile is loaded into LDS once (16-byte chunks XOR-
//    swizzled by row, so fragment reads are conflict free) and each workgroup
//    walks over 128-row tiles of the output, grid-stride; every lane loads its
//    own pixel row's operand fragments one tile ahead;
//  - the MFMA runs with the operands swapped, D = W x X^T, so a lane's
//    accumulators hold one output pixel (lane % 32) and channels
//    8*(e/4) + 4*(lane/32) + e%4 of each 32-channel tile.  Swapping the upper
//    lane half of channel group 2g with the lower lane half of group 2g+1
//    (v_permlane32_swap, four register pairs per group pair) leaves each lane
//    with 8 consecutive channels twice;
//  - those rounded 16-byte chunks go through a small per-wave LDS buffer
//    (SW 32-channel tiles at a time, chunks XOR-swizzled by pixel) and come
//    back so that 4*SW consecutive lanes hold one pixel's 64*SW consecutive
//    bytes: each store instruction then writes whole 128-byte (SW = 2) or
//    64-byte lines.  Written straight from the swapped layout, every store
//    instruction split into 32 separate 32-byte writes, and the store path
//    (not HBM) bounded these layers.  With an addend the float32 sums take
//    that path instead (the addend joins before the one rounding), and the
//    addend (and its ReLU mask, one byte per 16-byte chunk) is read in the
//    same whole-line layout;
//  - BN statistics are taken from the rounded values each lane reads back
//    for its stores (8 channels of a few pixels per store group): per
//    channel, (y - K) and its square are added into the lane's float32 sums,
//    kept in registers over every tile the wave walks, about a shift K per
//    channel (the value in the wave's first row, kept in LDS); after the last
//    tile the lanes holding the same channels are added up, and the four
//    waves are combined once into one record covering the tiles blockIdx.x,
//    blockIdx.x + gridDim.x, ... (no barrier per tile).  A lane holds
//    BN / 8 channels over 64 input channels and BN / 4 over 128 or 256: at
//    most 32 (64 would leave one wave per SIMD).
// Each output element is the same k-ordered sum of exact products in both
// MFMA forms, so the values equal the other kernels' bit for bit.
template <int CI, int BN, bool STATS, bool ADD, bool APPLY = false>
struct CfgPw {
  static constexpr int KS = CI / 16;          // k sub-steps of 16 channels
  static constexpr int TN = BN / 32;          // 32-channel tiles
  static constexpr int SW = CI == 64 ? 2 : 1; // 32-channel tiles per store group
  static constexpr int BBYTES = BN * CI * 2;  // resident filter tile
  // [wave][pixel][SW*64 bytes] of rounded values, or [wave][pixel][SW*128
  // bytes] of float32 sums where the addend joins before the rounding
  static constexpr int STG = 4 * 32 * SW * (ADD ? 128 : 64);
  static constexpr int BST = STATS ? 4 * 3 * BN * 4 : 0;  // [wave][K, s1, s2][BN]
  static constexpr int SHARED = STG > BST ? STG : BST;
  // (+ 4 wave row counts and the waves' shifts, [wave][BN] binary16)
  static constexpr int XTRA = STATS ? 16 + 4 * BN * 2 : 0;
  // (+ the BN apply's coefficients: [BN] x {mean, a, b, sg})
  static constexpr int LDS = BBYTES + SHARED + XTRA + (APPLY ? BN * 16 : 0);
};

__device__ __forceinline__ void lane_half_swap(float& x, float& y) {
  const auto r = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(unsigned, x),
                                                  __builtin_bit_cast(unsigned, y), false, false);
  x = __builtin_bit_cast(float, (unsigned)r[0]);
  y = __builtin_bit_cast(float, (unsigned)r[1]);
}

// LDS written by this wave's lanes visible to all of them (LDS operations of
// one wave complete in order; this keeps the compiler from moving them)
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

template <int CI, int BN, bool STATS, bool ADD, bool MASK, bool APPLY = false, bool RES = false>
__global__ __launch_bounds__(256) void pw_kernel(const IgemmArgs a, int ntiles) {
  using K = CfgPw<CI, BN, STATS, ADD, APPLY>;
  constexpr int KS = K::KS, TN = K::TN, SW = K::SW;
  constexpr int SLOTS = 4 * SW;       // 16-byte chunks per staged pixel row
  constexpr int PPI = 64 / SLOTS;     // pixels per store instruction
  static_assert(CI == 64 || CI == 128 || CI == 256, "input channels");
  static_assert(!(STATS && ADD), "statistics are taken without an addend");
  static_assert(ADD || !MASK, "a mask is over the addend");
  static_assert(!APPLY || (!STATS && !ADD), "the BN apply follows the statistics pass");
  static_assert(APPLY || !RES, "the shortcut joins in the BN apply");
  // the early loads in the store layout: the addend, or the apply's shortcut
  constexpr bool EARLY = ADD || RES;
  static_assert(TN % SW == 0, "store groups");
  constexpr int NG = TN / SW;         // store groups
  static_assert(!STATS || NG * 8 <= 32, "statistics: at most 32 channels per lane");
  __shared__ __attribute__((aligned(1024))) char lds[K::LDS];
  char* bt = lds;
  char* shared = lds + K::BBYTES;
  float* bst = reinterpret_cast<float*>(shared);
  int* bcnt = reinterpret_cast<int*>(lds + K::BBYTES + K::SHARED);

  const IgemmPhase ph = a.ph[0];
  const int HoWo = ph.Ho * ph.Wo;
  const int M = a.N * HoWo;
  const int n0 = blockIdx.y * BN;
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const int lrow = lane & 31, lhi = lane >> 5;
  char* stg = shared + wave * 32 * SLOTS * (ADD ? 32 : 16);
  // the wave's shifts: channel n0 + i at kst[i]
  h16* kst = reinterpret_cast<h16*>(lds + K::BBYTES + K::SHARED + 16) + wave * BN;
  // the BN apply's coefficients of channel n0 + i at cof[i]
  float4* cof = reinterpret_cast<float4*>(lds + K::BBYTES + K::SHARED + K::XTRA);
  const h16* early = ADD ? a.addend : a.bn_res;
  if (APPLY) {
    for (int i = tid; i < BN; i += 256) {
      float4 q = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
      if (n0 + i < a.Co) {
        const FwdCoef k = fwd_coef(a.bn_stats, a.bn_gamma, a.bn_beta, a.Co, n0 + i, a.bn_scale);
        q = make_float4(k.mean, k.a, k.b, k.sg);
      }
      cof[i] = q;
    }
  }
  constexpr uint32_t OOB = 0x80000000u;
  const int act_bytes = (int)((int64_t)a.N * a.Hi * a.Wi * CI * 2);
  const __amdgpu_buffer_rsrc_t rs_a = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<h16*>(a.act), (short)0, act_bytes, 0x00020000);

  // filter tile: row n (channel n0 + n), chunk c stored at chunk c ^ (n % 8)
  for (int i = tid; i < BN * (CI / 8); i += 256) {
    const int n = i / (CI / 8), c = i - n * (CI / 8);
    V8 v;
    if (n0 + n < a.Co) {
      v = load16(ph.filt + (int64_t)(n0 + n) * ph.ldb + c * 8);
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) v.s[e] = 0;
    }
    *reinterpret_cast<V8*>(bt + (n * (CI / 8) + (c ^ (n & 7))) * 16) = v;
  }

  // this lane's source pixel row in a tile (out of range: reads zeros)
  auto row_off = [&](int tile) -> uint32_t {
    const int m = tile * 128 + wave * 32 + lrow;
    if (tile >= ntiles || m >= M) return OOB;
    const int img = m / HoWo;
    const int rem = m - img * HoWo;
    const int i = rem / ph.Wo;
    const int j = rem - i * ph.Wo;
    const int pix = (img * a.Hi + i * a.stride_h) * a.Wi + j * a.stride_w;
    return (uint32_t)pix * (uint32_t)(CI * 2) + (uint32_t)lhi * 16u;
  };
  auto load_a = [&](half8 (&A)[KS], uint32_t o) {
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      A[ks] = __builtin_bit_cast(half8, __builtin_amdgcn_raw_buffer_load_b128(
                                            rs_a, o == OOB ? OOB : o + ks * 32, 0, 0));
  };
  half8 Acur[KS], Anext[KS];
  // the lane's running sums of (y - K) and (y - K)^2 for channel e of its
  // chunk in store group g, over the pixels it stored; nrows: the wave's rows
  float s1[STATS ? NG : 1][8], s2[STATS ? NG : 1][8];
#pragma unroll
  for (int g = 0; g < (STATS ? NG : 1); ++g)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      s1[g][e] = 0.0f;
      s2[g][e] = 0.0f;
    }
  int nrows = 0;
  h16 one = (h16)1.0f;
  asm("" : "+v"(one));  // kept opaque, so that y * one is not folded into y
  int tile = blockIdx.x;
  load_a(Acur, row_off(tile));
  __syncthreads();
  const int swz = lrow & 7;
  for (; tile < ntiles; tile += gridDim.x) {
    const int band_m0 = tile * 128 + wave * 32;
    // the tile's addend, loaded before the MFMAs in the store layout (lane:
    // chunk lane % SLOTS of pixel lane / SLOTS + PPI*i; clamped into range)
    // (and with MASK the addend's ReLU mask bytes, applied where it is added)
    // (a strided addend: the row of each of the lane's pixels, or +0)
    V8 adv[EARLY ? TN / SW : 1][EARLY ? 32 / PPI : 1];
    uint32_t amb[MASK ? TN / SW : 1][MASK ? 32 / PPI : 1];
    bool aok[EARLY ? 32 / PPI : 1];
    if (EARLY) {
      int64_t arow[32 / PPI];
#pragma unroll
      for (int i = 0; i < 32 / PPI; ++i) {
        const int m = band_m0 + lane / SLOTS + i * PPI;
        const int mc = m < M ? m : M - 1;
        arow[i] = (int64_t)mc * a.ldo;
        aok[i] = true;
        if (ADD && a.astride > 1) {
          const int img = mc / HoWo;
          const int rem = mc - img * HoWo;
          const int oh = rem / ph.Wo;
          const int64_t r = addend_row(a, img, oh, rem - oh * ph.Wo);
          aok[i] = r >= 0;
          arow[i] = r >= 0 ? r : 0;
        }
      }
#pragma unroll
      for (int g = 0; g < TN / SW; ++g)
#pragma unroll
        for (int i = 0; i < 32 / PPI; ++i) {
          const int n = n0 + g * SW * 32 + (lane % SLOTS) * 8;
          const int64_t off = arow[i] + (n < a.Co ? n : 0);
          adv[g][i] = load16(early + off);
          if (MASK) amb[g][i] = a.amask[off >> 3];
        }
    }
    load_a(Anext, row_off(tile + gridDim.x));
    const bool first = tile == (int)blockIdx.x;
    if (STATS) {
      const int rows = M - band_m0;
      nrows += rows <= 0 ? 0 : (rows < 32 ? rows : 32);
    }
#pragma unroll
    for (int g = 0; g < TN / SW; ++g) {
#pragma unroll
      for (int tl = 0; tl < SW; ++tl) {
        const int tn = g * SW + tl;
        floatx16 at;
#pragma unroll
        for (int e = 0; e < 16; ++e) at[e] = 0.0f;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const int pos = ((ks * 2 + lhi) ^ swz) * 16;
          const half8 bf = *reinterpret_cast<const half8*>(bt + (tn * 32 + lrow) * (CI * 2) + pos);
          at = mfma32x32x16(bf, Acur[ks], at);
        }
        float v[16];
#pragma unroll
        for (int e = 0; e < 16; ++e) v[e] = at[e];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          lane_half_swap(v[q], v[4 + q]);
          lane_half_swap(v[8 + q], v[12 + q]);
        }
        // v[8h .. 8h+7] = channels tn*32 + 16h + 8*lhi + 0..7 of pixel mp:
        // chunk tl*4 + 2h + lhi of this store group's row of pixel lrow
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int k = tl * 4 + 2 * h + lhi;
          if (ADD) {
            // float32: two 16-byte halves per chunk, swizzled over 2*SLOTS slots
#pragma unroll
            for (int j = 0; j < 2; ++j) {
              const int slot = (2 * k + j) ^ (lrow & (2 * SLOTS - 1));
              float4 f;
              f.x = v[h * 8 + 4 * j];
              f.y = v[h * 8 + 4 * j + 1];
              f.z = v[h * 8 + 4 * j + 2];
              f.w = v[h * 8 + 4 * j + 3];
              *reinterpret_cast<float4*>(stg + (lrow * 2 * SLOTS + slot) * 16) = f;
            }
          } else {
            V8 o;
#pragma unroll
            for (int e = 0; e < 8; ++e) o.h[e] = to_h16(v[h * 8 + e]);
            const int slot = k ^ (lrow & (SLOTS - 1));
            *reinterpret_cast<V8*>(stg + (lrow * SLOTS + slot) * 16) = o;
          }
        }
      }
      wave_lds_sync();
      // lane: chunk lane % SLOTS of pixel lane / SLOTS (+ PPI per instruction)
      const int c = lane % SLOTS;
      const int n = n0 + g * SW * 32 + c * 8;
      V8 kv;
      float4 cf[APPLY ? 8 : 1];
      if (APPLY) {
#pragma unroll
        for (int e = 0; e < 8; ++e) cf[e] = cof[g * SW * 32 + c * 8 + e];
      }
      if (STATS) {
        if (first) {
          // the shifts: the values of the wave's first row (staged pixel 0)
          if (lane < SLOTS)
            *reinterpret_cast<V8*>(kst + g * SW * 32 + lane * 8) =
                *reinterpret_cast<const V8*>(stg + lane * 16);
          wave_lds_sync();
        }
        kv = *reinterpret_cast<const V8*>(kst + g * SW * 32 + c * 8);
      }
#pragma unroll
      for (int i = 0; i < 32 / PPI; ++i) {
        const int q = lane / SLOTS + i * PPI;
        V8 o;
        if (ADD) {
          float w[8];
#pragma unroll
          for (int j = 0; j < 2; ++j) {
            const float4 f = *reinterpret_cast<const float4*>(
                stg + (q * 2 * SLOTS + ((2 * c + j) ^ (q & (2 * SLOTS - 1)))) * 16);
            w[4 * j] = f.x;
            w[4 * j + 1] = f.y;
            w[4 * j + 2] = f.z;
            w[4 * j + 3] = f.w;
          }
          V8 ad = MASK ? masked8(adv[g][i], amb[g][i]) : adv[g][i];
          if (!aok[i]) ad = zero8();
#pragma unroll
          for (int e = 0; e < 8; ++e) o.h[e] = to_h16(w[e] + to_f32(ad.h[e]));
        } else {
          o = *reinterpret_cast<const V8*>(stg + (q * SLOTS + (c ^ (q & (SLOTS - 1)))) * 16);
        }
        const int m = band_m0 + q;
        uint32_t zbits = 0;
        if (APPLY) {
          // z from the rounded y with the BN apply's float32 sequence (the
          // shortcut and ReLU per the flags), and its ReLU mask bits
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float4 q4 = cf[e];
            const FwdCoef k{q4.x, q4.y, q4.z, q4.w};
            o.h[e] = to_h16(fwd_value(to_f32(o.h[e]), k, RES, RES ? to_f32(adv[g][i].h[e]) : 0.0f,
                                      a.bn_relu != 0, a.bn_swap != 0));
            zbits |= (uint32_t)(to_f32(o.h[e]) > 0.0f) << e;
          }
        }
        if (m < M && n < a.Co) {
          store16(a.out + (int64_t)m * a.ldo + n, o);
          if (APPLY && a.bn_mask) a.bn_mask[((int64_t)m * a.ldo + n) >> 3] = (uint8_t)zbits;
        }
        if (STATS && m < M) {
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            // y * 1 - K, exact operands and one rounding: the same value as
            // the difference of the two widened values, in one mixed-precision
            // FMA that reads y's binary16 half directly
            const float d = __builtin_fmaf(to_f32(o.h[e]), to_f32(one), -to_f32(kv.h[e]));
            s1[g][e] += d;
            s2[g][e] = __builtin_fmaf(d, d, s2[g][e]);
          }
        }
      }
      wave_lds_sync();
    }
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) Acur[ks] = Anext[ks];
  }
  if (STATS) {
    // lanes l, l + SLOTS, l + 2*SLOTS, ... hold the same channels: add them
    // up (fixed order), then lane l < SLOTS writes its chunks' band sums
#pragma unroll
    for (int off = SLOTS; off < 64; off *= 2)
#pragma unroll
      for (int g = 0; g < NG; ++g)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          s1[g][e] += __shfl_xor(s1[g][e], off, 64);
          s2[g][e] += __shfl_xor(s2[g][e], off, 64);
        }
    __syncthreads();  // every wave is done with its staging buffer
    if (lane < SLOTS) {
#pragma unroll
      for (int g = 0; g < NG; ++g) {
        const V8 kv = *reinterpret_cast<const V8*>(kst + g * SW * 32 + lane * 8);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int ch = g * SW * 32 + lane * 8 + e;
          bst[(wave * 3 + 0) * BN + ch] = to_f32(kv.h[e]);
          bst[(wave * 3 + 1) * BN + ch] = s1[g][e];
          bst[(wave * 3 + 2) * BN + ch] = s2[g][e];
        }
      }
    }
    if (lane == 0) bcnt[wave] = nrows;
    __syncthreads();
    // the workgroup's record: the waves re-based on wave 0's shift, in wave
    // order (wave 0 always has rows: the first tile starts inside M)
    for (int c = tid; c < BN; c += 256) {
      if (n0 + c < a.Co) {
        const float K0 = bst[c];
        float S1 = 0.0f, S2 = 0.0f;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          const float nw = (float)bcnt[w];
          if (bcnt[w] == 0) break;
          const float d = bst[(w * 3) * BN + c] - K0;
          const float t1 = bst[(w * 3 + 1) * BN + c];
          S1 += __builtin_fmaf(nw, d, t1);
          S2 += __builtin_fmaf(nw * d, d,
                               __builtin_fmaf(2.0f * d, t1, bst[(w * 3 + 2) * BN + c]));
        }
        float* rec = a.stat + (int64_t)blockIdx.x * 3 * a.Co + n0 + c;
        rec[0] = K0;
        rec[a.Co] = S1;
        rec[2 * a.Co] = S2;
      }
    }
  }
}

// ---- 3x3 stride-1 convolutions over 64 channels ---------------------------------
// A 3x3 layer with 64 input and 64 output channels (ResNet-50's conv2_x, and
// its data gradient) has a reduction of only 576, and the implicit-GEMM
// kernels above fetch every input pixel once per tap from L2 (9x) for a
// 64-wide output: they keep the matrix cores 14-17% busy.  Here:
//  - the whole 64 x 576 filter (72 KB) stays in LDS (16-byte chunks XOR-
//    swizzled by row/2 within each tap) and each workgroup (one per CU, eight
//    waves) walks over tiles of 256 consecutive output pixels of one image;
//  - a tile's input rows with their one-pixel halo (zeros outside the image)
//    are staged in LDS once, pixel-major, 128 bytes per pixel with chunks
//    XOR-swizzled by pixel/2; the nine taps read shifted windows of it.
//    (The 16 lanes an LDS cycle serves read 16 consecutive pixels or filter
//    rows: 128-byte rows fall into two 128-byte bank halves by parity, and
//    the swizzle by row/2 spreads each half's 8 rows over its 8 chunks.  A
//    swizzle by the row itself left 2-way conflicts on every read);
//  - the next tile's rows are loaded into registers while the current tile
//    is computed, and written to LDS after it;
//  - each wave computes 32 pixels x 64 channels with the operands swapped
//    (D = W x X^T), reading the fragments of step i+2 while the MFMAs of step
//    i run, and writes from registers after lane-half swaps, as pw_kernel
//    does.
// Same k order (tap, then channel) and the same exact products as the other
// kernels, so the values are bit-identical.
constexpr int kC3Tile = 256;                      // output pixels per tile
constexpr int kC3Thr = 512;                       // threads per workgroup
constexpr int kC3Filt = 64 * 576 * 2;             // resident filter, bytes
constexpr int kC3HaloPix = 684;                   // staged input pixels (W <= 112)
constexpr int kC3Pref = (kC3HaloPix * 8 + kC3Thr - 1) / kC3Thr;  // chunks per thread

struct C3Geo {
  int img, p0, oh0, rows;  // tile: image, first pixel, first output row, staged input rows
};
__device__ __forceinline__ C3Geo c3_geo(int tile, int tpi, int H, int W) {
  C3Geo g;
  g.img = tile / tpi;
  g.p0 = (tile - g.img * tpi) * kC3Tile;
  const int HW = H * W;
  const int last = g.p0 + kC3Tile - 1 < HW ? g.p0 + kC3Tile - 1 : HW - 1;
  g.oh0 = g.p0 / W;
  g.rows = last / W - g.oh0 + 3;
  return g;
}

__global__ __launch_bounds__(kC3Thr) void c3_kernel(const IgemmArgs a, int tpi, int ntiles) {
  __shared__ __attribute__((aligned(1024))) char lds[kC3Filt + kC3HaloPix * 128];
  char* filt = lds;
  char* halo = lds + kC3Filt;
  const IgemmPhase ph = a.ph[0];
  const int H = a.Hi, W = a.Wi, HW = H * W, W2 = W + 2;
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const int lrow = lane & 31, lhi = lane >> 5;
  constexpr uint32_t OOB = 0x80000000u;
  const int act_bytes = (int)((int64_t)a.N * HW * 64 * 2);
  const __amdgpu_buffer_rsrc_t rs_a = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<h16*>(a.act), (short)0, act_bytes, 0x00020000);

  // filter: row n, chunk c (of 72: tap*8 + channel chunk) at
  // (c & ~7) | ((c ^ (n >> 1)) & 7)
  for (int i = tid; i < 64 * 72; i += kC3Thr) {
    const int n = i / 72, c = i - n * 72;
    const V8 v = load16(ph.filt + (int64_t)n * ph.ldb + c * 8);
    *reinterpret_cast<V8*>(filt + (n * 72 + ((c & ~7) | ((c ^ (n >> 1)) & 7))) * 16) = v;
  }

  // a tile's staged input: pixel q = row*(W+2) + col of input rows oh0-1 ..,
  // columns -1 .. W; chunk j of it at (q*8 + (j ^ ((q >> 1) & 7)))*16
  V8 pf[kC3Pref];
  auto prefetch = [&](int tile) {
    const C3Geo g = c3_geo(tile < ntiles ? tile : 0, tpi, H, W);
    const int total = g.rows * W2 * 8;
#pragma unroll
    for (int i = 0; i < kC3Pref; ++i) {
      const int q = tid + kC3Thr * i;
      const int pix = q >> 3, j = q & 7;
      const int hr = pix / W2, hc = pix - hr * W2;
      const int ir = g.oh0 - 1 + hr, ic = hc - 1;
      const bool v = tile < ntiles && q < total && (unsigned)ir < (unsigned)H &&
                     (unsigned)ic < (unsigned)W;
      const uint32_t off = (uint32_t)((((g.img * H + ir) * W + ic) * 64 + j * 8) * 2);
      pf[i].u = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs_a, v ? off : OOB, 0, 0));
    }
  };
  auto stage = [&](int tile) {
    const C3Geo g = c3_geo(tile, tpi, H, W);
    const int total = g.rows * W2 * 8;
#pragma unroll
    for (int i = 0; i < kC3Pref; ++i) {
      const int q = tid + kC3Thr * i;
      if (q < total) {
        const int pix = q >> 3, j = q & 7;
        *reinterpret_cast<V8*>(halo + (pix * 8 + (j ^ ((pix >> 1) & 7))) * 16) = pf[i];
      }
    }
  };

  int tile = blockIdx.x;
  prefetch(tile);
  stage(tile);
  __syncthreads();
  for (; tile < ntiles; tile += gridDim.x) {
    const C3Geo g = c3_geo(tile, tpi, H, W);
    prefetch(tile + gridDim.x);
    // this lane's pixel, clamped into the image for the addresses (a pixel
    // past the end is not stored)
    const int m = g.p0 + wave * 32 + lrow;
    int hp0;
    {
      const int mc = m < HW ? m : HW - 1;
      const int oh = mc / W, ow = mc - oh * W;
      hp0 = (oh - g.oh0) * W2 + ow;
    }
    floatx16 acc[2];
#pragma unroll
    for (int tn = 0; tn < 2; ++tn)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[tn][e] = 0.0f;
    // step i = tap*4 + ks: the pixel fragment and the two filter fragments
    half8 xa[3], fb[3][2];
    auto fetch = [&](int i, int buf) {
      const int tap = i >> 2, ks = i & 3;
      const int j = ks * 2 + lhi;
      const int hp = hp0 + (tap / 3) * W2 + tap % 3;
      xa[buf] = *reinterpret_cast<const half8*>(halo + (hp * 8 + (j ^ ((hp >> 1) & 7))) * 16);
#pragma unroll
      for (int tn = 0; tn < 2; ++tn) {
        const int n = tn * 32 + lrow;
        fb[buf][tn] =
            *reinterpret_cast<const half8*>(filt + (n * 72 + tap * 8 + ((j ^ (n >> 1)) & 7)) * 16);
      }
    };
    fetch(0, 0);
    fetch(1, 1);
#pragma unroll
    for (int i = 0; i < 36; ++i) {
      if (i + 2 < 36) fetch(i + 2, (i + 2) % 3);
#pragma unroll
      for (int tn = 0; tn < 2; ++tn) acc[tn] = mfma32x32x16(fb[i % 3][tn], xa[i % 3], acc[tn]);
    }
    __syncthreads();  // every wave is done with this tile's staged rows
    // lane: pixel m, channels 16h + 8*(lane/32) + 0..7 of each 32-channel tile
#pragma unroll
    for (int tn = 0; tn < 2; ++tn) {
      float v[16];
#pragma unroll
      for (int e = 0; e < 16; ++e) v[e] = acc[tn][e];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        lane_half_swap(v[q], v[4 + q]);
        lane_half_swap(v[8 + q], v[12 + q]);
      }
      if (m < HW) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          V8 o;
#pragma unroll
          for (int e = 0; e < 8; ++e) o.h[e] = to_h16(v[h * 8 + e]);
          store16(a.out + ((int64_t)g.img * HW + m) * a.ldo + tn * 32 + h * 16 + lhi * 8, o);
        }
      }
    }
    if (tile + gridDim.x < ntiles) stage(tile + gridDim.x);
    __syncthreads();
  }
}

// Whether the 3x3 kernel takes this problem; tiles per image if so.
int c3_tiles_per_image(const IgemmArgs& a) {
  const IgemmPhase& p = a.ph[0];
  if (a.stat || a.addend || a.nphase != 1 || p.Rt != 3 || p.St != 3 ||
      a.stride_h != 1 || a.stride_w != 1 || p.pad_h != 1 || p.pad_w != 1 || a.Ci != 64 ||
      a.Co != 64 || p.ldb != 576 || p.Ho != a.Hi || p.Wo != a.Wi || a.OH != p.Ho ||
      a.OW != p.Wo || a.os_h != 1 || a.os_w != 1 || p.oph != 0 || p.opw != 0 || a.ldo != 64)
    return 0;
  const int W = a.Wi;
  if (W < 1 || a.Hi < 1) return 0;
  const int rows = 1 + (W + kC3Tile - 2) / W + 2;  // most input rows a tile stages
  if ((int64_t)rows * (W + 2) > kC3HaloPix) return 0;
  if ((int64_t)a.N * a.Hi * a.Wi * 64 * 2 >= ((int64_t)1 << 31)) return 0;
  return (a.Hi * a.Wi + kC3Tile - 1) / kC3Tile;
}

// ---- k-step 64, whole 128-byte operand rows, fragment reads one sub-step ahead
// As igemm6, with a k-step of 64 channels: every operand row of a stage is one
// whole 128-byte line (8 lanes x 16 bytes per row, 8 rows per 1 KB DMA
// instruction), and each wave does 4 x TM x TN MFMAs per barrier.  The
// fragments of k sub-step ks+1 are read from LDS while the MFMAs of sub-step
// ks run; the first sub-step of the next stage is read right after the
// barrier that publishes it, before the last MFMAs of the current stage.
// S stages: the stage refilled at the end of step kt is needed at the end of
// step kt+S-1.  Needs Ci % 64 == 0, at most 32 filter taps per phase, and
// operands below 1 GiB (the out-of-range offsets used for padding).
// One 16-byte-per-lane DMA from a buffer resource into LDS (1 KB per wave).
// (Called through this function: the builtin written directly in the
// igemm7 lambda made the host pass drop that kernel's launch stubs.)
__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t rs, char* lds_dst, uint32_t voff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (__attribute__((address_space(3))) void*)lds_dst, 16,
                                           voff, 0, 0, 0);
}
template <int TM, int TN, int WM, int WN, int S>
struct Cfg7 {
  static constexpr int BM = 32 * TM * WM, BN = 32 * TN * WN;
  static constexpr int IA = BM / 32, IB = BN / 32;  // DMA instructions per wave per stage
  static constexpr int Q = IA + IB;
  static constexpr int STAGE = (BM + BN) * 128;     // bytes
  static constexpr int SP = 32 * TN + 4;            // epilogue staging pitch (floats)
  static constexpr int EPI = 4 * 32 * SP * 4;
  // BN statistics of the epilogue: [WN][4 bands][3][32*TN] floats + 4 row
  // counts, after the staging area
  static constexpr int STAT = WN * 4 * 3 * 32 * TN * 4 + 16;
  static constexpr int LDS = S * STAGE > EPI + STAT ? S * STAGE : EPI + STAT;
};

// TRANS (without statistics): the MFMA operands are swapped so that the
// accumulators hold the transposed tile, and the epilogue writes straight from
// registers after lane-half swaps, as pw_kernel does (no LDS staging).
template <int TM, int TN, int WM, int WN, int S, bool STATS, bool TRANS = !STATS>
__global__ __launch_bounds__(256) void igemm7_kernel(const IgemmArgs a) {
  using K = Cfg7<TM, TN, WM, WN, S>;
  static_assert(!(STATS && TRANS), "statistics are taken from the staged tile");
  constexpr int BM = K::BM, BN = K::BN, IA = K::IA, IB = K::IB;
  static_assert(WM * WN == 4 && IA >= 1 && IB >= 1 && S >= 2, "tile shape");
  static_assert(K::Q * (S - 1) < 64, "vmcnt range");
  __shared__ __attribute__((aligned(1024))) char lds[K::LDS];

  int tz, tm_, tn_;
  xcd_tile(a.gn, tz, tm_, tn_);
  const IgemmPhase ph = a.ph[tz];
  const int HoWo = ph.Ho * ph.Wo;
  const int M = a.N * HoWo;
  const int m0 = tm_ * BM;
  if (m0 >= M) return;
  const int n0 = tn_ * BN;
  const int Ci = a.Ci;
  const int Kg = ph.Rt * ph.St * Ci;
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const int act_bytes = (int)((int64_t)a.N * a.Hi * a.Wi * Ci * 2);
  const int filt_bytes = (int)((int64_t)a.Co * ph.ldb * 2);
  constexpr uint32_t OOB = 0x80000000u;

  // DMA lane roles: row (wave*I + q)*8 + lane/8 of the tile, physical chunk
  // lane%8 holding logical chunk (lane%8) ^ ((row/2)%8).  Per A row: the byte
  // offset of its tap-(0,0) pixel (wrapping below zero in the padding) and a
  // bit mask of the taps that fall inside the image, so that a k-step costs
  // one add, one mask test and one select per DMA.
  uint32_t a_pix[IA], a_vm[IA];
  uint32_t b_off[IB];
#pragma unroll
  for (int q = 0; q < IA; ++q) {
    const int row = (wave * IA + q) * 8 + (lane >> 3);
    const int lc = (lane & 7) ^ ((row >> 1) & 7);
    const int m = m0 + row;
    a_pix[q] = 0;
    a_vm[q] = 0;
    if (m < M) {
      const int img = m / HoWo;
      const int rem = m - img * HoWo;
      const int i = rem / ph.Wo;
      const int j = rem - i * ph.Wo;
      const int ih0 = i * a.stride_h - ph.pad_h;
      const int iw0 = j * a.stride_w - ph.pad_w;
      a_pix[q] = (uint32_t)((int64_t)img * a.Hi * a.Wi * Ci * 2) +
                 (uint32_t)(((int64_t)ih0 * a.Wi + iw0) * Ci * 2) + (uint32_t)lc * 16u;
      for (int r = 0; r < ph.Rt; ++r)
        for (int t = 0; t < ph.St; ++t)
          if ((unsigned)(ih0 + r) < (unsigned)a.Hi && (unsigned)(iw0 + t) < (unsigned)a.Wi)
            a_vm[q] |= 1u << (r * ph.St + t);
    }
  }
#pragma unroll
  for (int q = 0; q < IB; ++q) {
    const int row = (wave * IB + q) * 8 + (lane >> 3);
    const int lc = (lane & 7) ^ ((row >> 1) & 7);
    const int n = n0 + row;
    b_off[q] = n < a.Co ? (uint32_t)n * (uint32_t)ph.ldb * 2u + (uint32_t)lc * 16u : 0x40000000u;
  }

  // k-step state (uniform): channel base, tap, byte offset of the tap's pixel
  int k0 = 0, cb = 0, tap = 0, ts = 0;
  uint32_t tap_off = 0;
  const uint32_t row_bytes = (uint32_t)a.Wi * (uint32_t)Ci * 2u;
  auto issue = [&](char* buf) {
    const __amdgpu_buffer_rsrc_t rs_a = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<h16*>(a.act), (short)0, act_bytes, 0x00020000);
    const __amdgpu_buffer_rsrc_t rs_b = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<h16*>(ph.filt), (short)0, filt_bytes, 0x00020000);
    const bool kval = k0 < Kg;
    const uint32_t bit = kval ? 1u << tap : 0u;
    const uint32_t aoff = tap_off + (uint32_t)cb * 2u;
#pragma unroll
    for (int q = 0; q < IA; ++q) {
      const uint32_t addr = pin_v(a_pix[q] + aoff);
      dma16(rs_a, buf + (wave * IA + q) * 1024, (a_vm[q] & bit) ? addr : OOB);
    }
    const uint32_t boff = kval ? (uint32_t)k0 * 2u : 0x40000000u;
#pragma unroll
    for (int q = 0; q < IB; ++q) {
      dma16(rs_b, buf + BM * 128 + (wave * IB + q) * 1024, b_off[q] + boff);
    }
    k0 += 64;
    cb += 64;
    if (cb == Ci) {
      cb = 0;
      ++tap;
      if (++ts == ph.St) {
        ts = 0;
        tap_off += row_bytes - (uint32_t)(ph.St - 1) * (uint32_t)Ci * 2u;
      } else {
        tap_off += (uint32_t)Ci * 2u;
      }
    }
  };

  const int wm = wave / WN, wn = wave % WN;
  const int lrow = lane & 31, lhi = lane >> 5;
  const int swz = (lrow >> 1) & 7;
  floatx16 acc[TM][TN];
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int tn = 0; tn < TN; ++tn)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[tm][tn][e] = 0.0f;

  half8 af[2][TM], bf[2][TN];
  auto fetch = [&](const char* buf, int ks, half8 (&fa)[TM], half8 (&fb)[TN]) {
    const int pos = ((ks * 2 + lhi) ^ swz) * 16;
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
      fa[tm] = *reinterpret_cast<const half8*>(buf + (wm * 32 * TM + tm * 32 + lrow) * 128 + pos);
#pragma unroll
    for (int tn = 0; tn < TN; ++tn)
      fb[tn] = *reinterpret_cast<const half8*>(buf + BM * 128 + (wn * 32 * TN + tn * 32 + lrow) * 128 + pos);
  };
  auto mma = [&](const half8 (&fa)[TM], const half8 (&fb)[TN]) {
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
      for (int tn = 0; tn < TN; ++tn)
        acc[tm][tn] = TRANS ? mfma32x32x16(fb[tn], fa[tm], acc[tm][tn])
                            : mfma32x32x16(fa[tm], fb[tn], acc[tm][tn]);
  };

  const int KT = (Kg + 63) / 64;
#pragma unroll
  for (int s = 0; s < S; ++s) issue(lds + s * K::STAGE);
  constexpr int ALLOW0 = K::Q * (S - 1);  // prologue: stages 1 .. S-1 stay in flight
  constexpr int WAIT0 = (0x0 << 8) | (0x7 << 4) | (ALLOW0 & 0xF) | ((ALLOW0 >> 4) << 14);
  constexpr int ALLOW = K::Q * (S - 2);   // steady state: stages kt+2 .. kt+S-1
  constexpr int WAIT = (0x0 << 8) | (0x7 << 4) | (ALLOW & 0xF) | ((ALLOW >> 4) << 14);
  __builtin_amdgcn_s_waitcnt(WAIT0);
  bare_barrier();
  fetch(lds, 0, af[0], bf[0]);
  int rd = 0;
  for (int kt = 0; kt < KT; ++kt) {
    const char* cur = lds + rd * K::STAGE;
    fetch(cur, 1, af[1], bf[1]);
    mma(af[0], bf[0]);
    fetch(cur, 2, af[0], bf[0]);
    mma(af[1], bf[1]);
    fetch(cur, 3, af[1], bf[1]);
    mma(af[0], bf[0]);
    // publish stage kt+1, refill this stage's buffer with stage kt+S, and
    // read the next stage's first sub-step before the last MFMAs of this one
    __builtin_amdgcn_s_waitcnt(WAIT);
    bare_barrier();
    issue(lds + rd * K::STAGE);
    rd = rd + 1 == S ? 0 : rd + 1;
    fetch(lds + rd * K::STAGE, 0, af[0], bf[0]);
    mma(af[1], bf[1]);
  }
  __builtin_amdgcn_s_waitcnt(0);
  if (TRANS) {
    // lane: output pixel m (lane % 32 of each 32-row tile) and, after the
    // swaps, channels 16h + 8*(lane/32) + 0..7 of each 32-channel tile
    V8 adv[TM][TN][2];
    uint32_t amb[TM][TN][2];
#pragma unroll
    for (int tm = 0; tm < TM; ++tm) {
      const int m = m0 + wm * 32 * TM + tm * 32 + lrow;
      int64_t base = 0, abase = -1;  // abase: the addend's row, -1 for +0
      if (m < M) {
        const int img = m / HoWo;
        const int rem = m - img * HoWo;
        const int i = rem / ph.Wo;
        const int j = rem - i * ph.Wo;
        const int oh = i * a.os_h + ph.oph, ow = j * a.os_w + ph.opw;
        base = ((int64_t)(img * a.OH + oh) * a.OW + ow) * a.ldo;
        if (a.addend) abase = addend_row(a, img, oh, ow);
      }
      if (a.addend && (a.ldo % 8) == 0) {
        // the addend first, so its loads overlap the swaps and conversions
#pragma unroll
        for (int tn = 0; tn < TN; ++tn)
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const int n = n0 + wn * 32 * TN + tn * 32 + h * 16 + lhi * 8;
            if (abase >= 0 && n + 8 <= a.Co) adv[tm][tn][h] = load16(a.addend + abase + n);
          }
        if (a.amask) {
#pragma unroll
          for (int tn = 0; tn < TN; ++tn)
#pragma unroll
            for (int h = 0; h < 2; ++h) {
              const int n = n0 + wn * 32 * TN + tn * 32 + h * 16 + lhi * 8;
              if (abase >= 0 && n + 8 <= a.Co) amb[tm][tn][h] = a.amask[(abase + n) >> 3];
            }
        }
      }
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) {
        float v[16];
#pragma unroll
        for (int e = 0; e < 16; ++e) v[e] = acc[tm][tn][e];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          lane_half_swap(v[q], v[4 + q]);
          lane_half_swap(v[8 + q], v[12 + q]);
        }
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int n = n0 + wn * 32 * TN + tn * 32 + h * 16 + lhi * 8;
          if (m >= M || n >= a.Co) continue;
          const int64_t off = base + n;
          if ((a.ldo % 8) == 0 && n + 8 <= a.Co) {
            float w[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) w[e] = v[h * 8 + e];
            if (a.addend) {
              V8 ad = a.amask ? masked8(adv[tm][tn][h], amb[tm][tn][h]) : adv[tm][tn][h];
              if (abase < 0) ad = zero8();
#pragma unroll
              for (int e = 0; e < 8; ++e) w[e] += to_f32(ad.h[e]);
            }
            V8 o;
#pragma unroll
            for (int e = 0; e < 8; ++e) o.h[e] = to_h16(w[e]);
            store16(a.out + off, o);
          } else {
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              if (n + e < a.Co) {
                float x = v[h * 8 + e];
                if (a.addend) {
                  x += abase >= 0 ? addend1(a, abase + n + e) : 0.0f;
                }
                a.out[off + e] = to_h16(x);
              }
            }
          }
        }
      }
    }
    return;
  }
  __syncthreads();

  float* stg = reinterpret_cast<float*>(lds) + wave * 32 * K::SP;
  constexpr int CPR = 32 * TN / 8;  // lanes per row
  constexpr int RPP = 64 / CPR;     // rows per pass
  const int cc = lane % CPR;
  const int rr = lane / CPR;
  const int n = n0 + wn * 32 * TN + cc * 8;
  const bool vec_ok = (a.ldo % 8) == 0 && n + 8 <= a.Co;
  // BN statistics of the rounded output (BM == 128: one record per tile):
  // per 32-row band and channel the band's first value K and the sums of
  // (y - K), (y - K)^2, taken column by column from the staged band (one lane
  // per column, rows in order); the four bands are combined in row order below
  // (kept inside the one LDS array: a second __shared__ object makes the
  // compiler wait for every LDS DMA in flight before each LDS read)
  constexpr int NB = 4, CW = 32 * TN;
  constexpr int RH = 32 * CW / 64;  // rows per lane
  static_assert(!STATS || BM == 128, "statistics records cover 128 rows");
  float (*bst)[NB][3][CW] = reinterpret_cast<float (*)[NB][3][CW]>(lds + K::EPI);
  int* bcnt = reinterpret_cast<int*>(lds + K::EPI + K::STAT - 16);
#pragma unroll
  for (int tm = 0; tm < TM; ++tm) {
#pragma unroll
    for (int tn = 0; tn < TN; ++tn)
#pragma unroll
      for (int e = 0; e < 16; ++e)
        stg[(8 * (e >> 2) + 4 * lhi + (e & 3)) * K::SP + tn * 32 + lrow] = acc[tm][tn][e];
    __syncthreads();
    const int band = wm * TM + tm;
    const int band_m0 = m0 + band * 32;
#pragma unroll
    for (int pass = 0; pass < 32 / RPP; ++pass) {
      const int r = pass * RPP + rr;
      const int m = band_m0 + r;
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
            const int64_t ar = addend_row(a, img, oh, ow);
            const V8 ad = ar >= 0 ? addend8(a, ar + n) : zero8();
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
              if (a.addend) {
                const int64_t ar = addend_row(a, img, oh, ow);
                x += ar >= 0 ? addend1(a, ar + n + e) : 0.0f;
              }
              a.out[off + e] = to_h16(x);
            }
          }
        }
      }
    }
    if (STATS) {
      const int rows = M - band_m0 <= 0 ? 0 : (M - band_m0 < 32 ? M - band_m0 : 32);
      const int c = lane % CW, h = lane / CW;
      const float Kc = to_f32(to_h16(stg[c]));  // the band's first row, as stored
      float s1 = 0.0f, s2 = 0.0f;
#pragma unroll
      for (int q = 0; q < RH; ++q) {
        const int r = h * RH + q;
        if (r < rows) {
          const float d = to_f32(to_h16(stg[r * K::SP + c])) - Kc;
          s1 += d;
          s2 = __builtin_fmaf(d, d, s2);
        }
      }
      if (CW < 64) {  // two lanes per column: rows 0-15 and 16-31
        s1 += __shfl_xor(s1, 32, 64);
        s2 += __shfl_xor(s2, 32, 64);
      }
      if (lane < CW) {
        bst[wn][band][0][c] = Kc;
        bst[wn][band][1][c] = s1;
        bst[wn][band][2][c] = s2;
      }
      if (lane == 0 && wn == 0) bcnt[band] = rows;
    }
    __syncthreads();
  }
  if (STATS && tid < WN * CW && bcnt[0] > 0) {
    // one record per 128-row tile: the bands re-based on the first band's K
    // (differences of two samples: no cancellation), in row order
    const int h = tid / CW, c = tid % CW;
    const int col = n0 + h * CW + c;
    if (col < a.Co) {
      const float K0 = bst[h][0][0][c];
      float S1 = 0.0f, S2 = 0.0f;
#pragma unroll
      for (int w = 0; w < NB; ++w) {
        if (bcnt[w] == 0) break;
        const float nw = (float)bcnt[w];
        const float d = bst[h][w][0][c] - K0;
        const float t1 = bst[h][w][1][c];
        S1 += __builtin_fmaf(nw, d, t1);
        S2 += __builtin_fmaf(nw * d, d, __builtin_fmaf(2.0f * d, t1, bst[h][w][2][c]));
      }
      float* rec = a.stat + (int64_t)(m0 / 128) * 3 * a.Co + col;
      rec[0] = K0;
      rec[a.Co] = S1;
      rec[2 * a.Co] = S2;
    }
  }
}

// The XCD tile order (xcd_tile) of a launch: measured on the ResNet-50
// convolutions at batch 128, it pays for the 1x1 filters with several N-tiles
// in one phase (1.01-1.13x: the N-tiles of an XCD share its activation rows
// in L2; all N-tiles per group did best), and costs elsewhere -- up to 0.92x on
// single-N-tile streams (eight distant address ranges instead of one front)
// and 0.5-0.85x on the strided data gradients -- so those keep the launch
// order.
int xcd_group(const IgemmArgs& a, int NT) {
  if (NT < 2 || a.nphase != 1 || a.ph[0].Rt * a.ph[0].St != 1) return 0;
  return NT;
}

template <int TM, int TN, int WM, int WN, int S>
hipError_t launch_cfg7(const IgemmArgs& a0, hipStream_t st) {
  using K = Cfg7<TM, TN, WM, WN, S>;
  int maxM = 0;
  for (int p = 0; p < a0.nphase; ++p) {
    const int m = a0.N * a0.ph[p].Ho * a0.ph[p].Wo;
    if (m > maxM) maxM = m;
  }
  if (maxM == 0 || a0.nphase == 0) return hipSuccess;
  dim3 grid(ceil_div(maxM, K::BM), ceil_div(a0.Co, K::BN), a0.nphase);
  IgemmArgs a = a0;
  a.gn = xcd_group(a, grid.y);
  if (a.stat)
    hipLaunchKernelGGL((igemm7_kernel<TM, TN, WM, WN, S, true>), grid, dim3(256), 0, st, a);
  else
    hipLaunchKernelGGL((igemm7_kernel<TM, TN, WM, WN, S, false>), grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

template <int TM, int TN>
hipError_t launch_cfg4(const IgemmArgs& a0, hipStream_t st) {
  using K = Cfg4<TM, TN>;
  int maxM = 0;
  for (int p = 0; p < a0.nphase; ++p) {
    const int m = a0.N * a0.ph[p].Ho * a0.ph[p].Wo;
    if (m > maxM) maxM = m;
  }
  if (maxM == 0 || a0.nphase == 0) return hipSuccess;
  dim3 grid(ceil_div(maxM, K::BM), ceil_div(a0.Co, K::BN), a0.nphase);
  IgemmArgs a = a0;
  a.gn = xcd_group(a, grid.y);
  hipLaunchKernelGGL((igemm4_kernel<TM, TN>), grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_c3(const IgemmArgs& a, int tpi, hipStream_t st) {
  const int ntiles = a.N * tpi;
  if (ntiles == 0) return hipSuccess;
  hipLaunchKernelGGL(c3_kernel, dim3(ntiles < 256 ? ntiles : 256), dim3(kC3Thr), 0, st, a, tpi,
                     ntiles);
  return hipGetLastError();
}

// workgroups along the rows of the pointwise kernel (nblk channel tiles),
// which walk the 128-row tiles, the filter tile's load into LDS paid once per
// workgroup.  Measured at batch 128: over 64 input channels 512 groups (the
// conv2_x conv3 + bn3 56 us, 64-66 at 256 or 1024); over 128 with statistics
// 128 groups on 4 channel tiles (51 us, 54-58 at 64 or 96, 64 at 192, 74 at
// 512), without them about six tiles per group (the conv3_x block inputs'
// data gradients with the masked addend: 784 tiles, 128 groups on 2 channel
// tiles 64-67 us against 75 at 512; the conv3_x block's own, 3,136 tiles on
// one channel tile: 85 us at 512 groups, 91 at 256, 145 at 128); over 256
// about 256 workgroups in all, one per CU (the conv4_x conv3 +
// bn3 on 8 channel tiles 75-78 us with 32 groups, 92-95 with 64, 117-123 with
// 128; the strided conv3_x shortcut on 4 tiles 114 us with 64 groups, 131
// with 128, 160 with 32)
static int pw_row_groups(int ntiles, int ci, bool stats, int nblk) {
  int cap = ci == 256 ? (nblk > 1 ? (256 + nblk - 1) / nblk : 256)
                      : ci == 128 && stats ? 128 : 512;
  // over 128 channels without statistics: about six tiles per workgroup, the
  // workgroups in all a whole multiple of the 256 CUs (each walks its tiles
  // to the end: 262 of them left six CUs with a second, 90 us against 66)
  if (ci == 128 && !stats) {
    const int want = (ntiles + 5) / 6 < cap ? (ntiles + 5) / 6 : cap;
    const int total = want * nblk;
    cap = total >= 256 ? (total / 256) * 256 / nblk : want;
    if (cap < 1) cap = 1;
  }
  return ntiles < cap ? ntiles : cap;
}

// channel tile of the pointwise kernel for this problem:
//  - 64 input channels: 256, or 128 for the statistics variant on small grids
//    (the conv2_x block's conv3 + bn3 at batch 32: 58.3 -> 56.5 us); at batch
//    128, and without statistics, 256-channel tiles are faster;
//  - 128: 256, and 128 with statistics (32 channels per lane and two waves
//    per SIMD; 256-channel tiles with 64 per lane ran at one wave per SIMD,
//    59-61 us against 51);
//  - 256: 128 (a 64 KB filter tile).
static int pw_tile_n(const IgemmArgs& a) {
  if (a.Ci == 64) {
    const bool narrow = a.stat && (int64_t)a.N * a.OH * a.OW <= 131072;
    return a.Co >= 256 && !narrow ? 256 : 128;
  }
  if (a.Ci == 128) return a.stat ? 128 : 256;
  return 128;
}

template <int CI, int BN>
hipError_t launch_pw(const IgemmArgs& a, hipStream_t st) {
  const int M = a.N * a.ph[0].Ho * a.ph[0].Wo;
  if (M == 0) return hipSuccess;
  const int ntiles = ceil_div(M, 128);
  dim3 grid(pw_row_groups(ntiles, CI, a.stat != nullptr, ceil_div(a.Co, BN)), ceil_div(a.Co, BN));
  if (a.bn_stats) {
    if (a.bn_res)
      hipLaunchKernelGGL((pw_kernel<CI, BN, false, false, false, true, true>), grid, dim3(256), 0,
                         st, a, ntiles);
    else
      hipLaunchKernelGGL((pw_kernel<CI, BN, false, false, false, true, false>), grid, dim3(256), 0,
                         st, a, ntiles);
  } else if (a.stat) {
    if constexpr (BN / (CI == 64 ? 8 : 4) <= 32)  // the lane's channels: see pw_kernel
      hipLaunchKernelGGL((pw_kernel<CI, BN, true, false, false>), grid, dim3(256), 0, st, a,
                         ntiles);
    else
      return hipErrorInvalidValue;
  } else if (a.addend) {
    if constexpr (CI < 256) {  // (igemm_kind takes no addend over 256 channels)
      if (a.amask)
        hipLaunchKernelGGL((pw_kernel<CI, BN, false, true, true>), grid, dim3(256), 0, st, a, ntiles);
      else
        hipLaunchKernelGGL((pw_kernel<CI, BN, false, true, false>), grid, dim3(256), 0, st, a,
                           ntiles);
    } else {
      return hipErrorInvalidValue;
    }
  } else
    hipLaunchKernelGGL((pw_kernel<CI, BN, false, false, false>), grid, dim3(256), 0, st, a, ntiles);
  return hipGetLastError();
}

template <int BM, int BN, int WM, int WN, int BK>
hipError_t launch_cfg(const IgemmArgs& a0, hipStream_t st) {
  int maxM = 0;
  for (int p = 0; p < a0.nphase; ++p) {
    const int m = a0.N * a0.ph[p].Ho * a0.ph[p].Wo;
    if (m > maxM) maxM = m;
  }
  if (maxM == 0 || a0.nphase == 0) return hipSuccess;
  dim3 grid(ceil_div(maxM, BM), ceil_div(a0.Co, BN), a0.nphase);
  IgemmArgs a = a0;
  a.gn = xcd_group(a, grid.y);
  hipLaunchKernelGGL((igemm_kernel<BM, BN, WM, WN, BK>), grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

// ---- the ResNet stem: 7x7 stride-2 convolution of 3-channel images -------------
// The stem (Section 5.1's ResNet-50: 3 -> 64 channels, 7x7, stride 2, pad 3)
// has a reduction of only 147, and padding its channels to 8 for the
// implicit-GEMM kernels wastes 62 % of the matrix-core work on zeros and a
// copy of the image.  Here:
//  - the k order is (filter row r, window pixel s' = 0..7, channel c' = 0..3)
//    with s' = 7 and c' = 3 zero in the filter: 7 x 32 = 224 (14 k-steps of
//    16); the whole 64 x 224 filter stays in registers as MFMA B fragments;
//  - a workgroup (one wave per 128 output pixels of an 8-row tile, Q/16
//    waves) walks over tiles of 8 output rows of one image; the tile's 21
//    input rows are staged in LDS once with 4 channels (8 bytes) per pixel
//    and 3 zero pixels of padding on the left, so the 8-pixel window of
//    output column q starts at pixel 2q of the staged row and each lane's
//    two window pixels are one aligned 16-byte read;
//  - the next tile's rows are loaded into registers (12 bytes = 2 pixels
//    per load) while the current tile is computed, and written to LDS after;
//  - each wave computes its 128 pixels as 4 blocks of 32 x 64 with the
//    operands swapped (D = W X^T: a lane holds one pixel) and stores from
//    registers after lane-half swaps, 16 bytes at a time, as pw_kernel does;
//  - the BN statistics are not taken here: computing the plain product
//    alongside for them (one channel of 16 pixels per lane) made the fused
//    call 22 us slower at batch 128 than this kernel plus the BN's own
//    statistics pass.
constexpr int kStemTR = 8;                      // output rows per tile
constexpr int kStemIR = 2 * kStemTR + 5;        // staged input rows
constexpr int kStemMaxQ = 128;                  // output columns (16 .. 128)
constexpr int kStemLds = kStemIR * (2 * kStemMaxQ + 6) * 8;
constexpr int kStemPairs = 6;                   // staged pixel pairs per thread

__global__ __launch_bounds__(512) void stem_kernel(const IgemmArgs a, int ntiles) {
  __shared__ __attribute__((aligned(16))) char lds[kStemLds];
  const int Q = a.OW, P = a.OH, H = a.Hi, W = a.Wi;
  const int RS = (2 * Q + 6) * 8;  // staged row, bytes
  const int nthr = Q * 4;          // Q / 16 waves
  const int tpi = (P + kStemTR - 1) / kStemTR;
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const int lrow = lane & 31, lhi = lane >> 5;
  constexpr uint32_t OOB = 0x80000000u;
  const int x_bytes = (int)((int64_t)a.N * H * W * 6);
  const __amdgpu_buffer_rsrc_t rs_x = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<h16*>(a.act), (short)0, x_bytes, 0x00020000);

  // the padding pixels (left 3, right past the image) stay zero throughout
  for (int i = tid; i < kStemIR * RS / 16; i += nthr) {
    V8 z;
#pragma unroll
    for (int e = 0; e < 8; ++e) z.s[e] = 0;
    *reinterpret_cast<V8*>(lds + i * 16) = z;
  }

  // filter fragments: lane holds channel nb*32 + lane%32 and, for k-step ks,
  // filter row ks/2, window pixels 4*(ks%2) + 2*lhi + {0, 1}, channels 0..3
  half8 bfr[2][14];
  {
    const h16* f = a.ph[0].filt;
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
      for (int ks = 0; ks < 14; ++ks) {
        V8 v;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int sp = 4 * (ks & 1) + 2 * lhi + (e >> 2), c = e & 3;
          const bool ok = sp < 7 && c < 3;
          const h16 w = f[(int64_t)(nb * 32 + lrow) * 147 + ((ks >> 1) * 7 + (ok ? sp : 0)) * 3 +
                          (ok ? c : 0)];
          v.h[e] = ok ? w : (h16)0.0f;
        }
        bfr[nb][ks] = v.h;
      }
  }

  // staging: pixel pair j = tid + i*nthr (i < kStemPairs) of the tile's
  // 21 rows x Q pairs (W = 2Q): row j / Q, input columns 2(j % Q) + {0, 1}
  uint32_t pf[kStemPairs][3];
  auto prefetch = [&](int tile) {
    const int n = tile / tpi, ih0 = 2 * (tile - n * tpi) * kStemTR - 3;
#pragma unroll
    for (int i = 0; i < kStemPairs; ++i) {
      const int j = tid + i * nthr;
      const int row = j / Q, k = j - row * Q;
      const int ih = ih0 + row;
      const bool ok = tile < ntiles && row < kStemIR && (unsigned)ih < (unsigned)H;
      const uint32_t off = ok ? (uint32_t)((((int64_t)n * H + ih) * W + 2 * k) * 6) : OOB;
      const auto v = __builtin_amdgcn_raw_buffer_load_b96(rs_x, off, 0, 0);
      pf[i][0] = v[0];
      pf[i][1] = v[1];
      pf[i][2] = v[2];
    }
  };
  auto stage = [&]() {
#pragma unroll
    for (int i = 0; i < kStemPairs; ++i) {
      const int j = tid + i * nthr;
      const int row = j / Q, k = j - row * Q;
      if (row < kStemIR) {
        // (c0 c1)(c2 c0')(c1' c2') -> (c0 c1)(c2 0) and (c0' c1')(c2' 0)
        uint2 p0, p1;
        p0.x = pf[i][0];
        p0.y = pf[i][1] & 0xFFFFu;
        p1.x = (pf[i][1] >> 16) | (pf[i][2] << 16);
        p1.y = pf[i][2] >> 16;
        char* dst = lds + row * RS + (2 * k + 3) * 8;
        *reinterpret_cast<uint2*>(dst) = p0;
        *reinterpret_cast<uint2*>(dst + 8) = p1;
      }
    }
  };

  int tile = blockIdx.x;
  prefetch(tile);
  __syncthreads();
  stage();
  __syncthreads();
  for (; tile < ntiles; tile += gridDim.x) {
    prefetch(tile + gridDim.x);
    const int n = tile / tpi, oh0 = (tile - n * tpi) * kStemTR;
    const int64_t M0 = ((int64_t)n * P + oh0) * Q;  // first output pixel of the tile
#pragma unroll 1
    for (int blk = 0; blk < 4; ++blk) {
      const int mb = wave * 128 + blk * 32;  // first pixel of the block in the tile
      const int m = mb + lrow;
      const int ohl = m / Q, ow = m - ohl * Q;
      const char* base = lds + 2 * ohl * RS + 16 * (ow + lhi);
      // D = W X^T: a lane holds one pixel
      floatx16 at[2];
#pragma unroll
      for (int nb = 0; nb < 2; ++nb)
#pragma unroll
        for (int e = 0; e < 16; ++e) at[nb][e] = 0.0f;
      half8 xa[3];
      xa[0] = *reinterpret_cast<const half8*>(base);
      xa[1] = *reinterpret_cast<const half8*>(base + 32);
#pragma unroll
      for (int ks = 0; ks < 14; ++ks) {
        if (ks + 2 < 14)
          xa[(ks + 2) % 3] =
              *reinterpret_cast<const half8*>(base + ((ks + 2) >> 1) * RS + 32 * ((ks + 2) & 1));
#pragma unroll
        for (int nb = 0; nb < 2; ++nb) {
          at[nb] = mfma32x32x16(bfr[nb][ks], xa[ks % 3], at[nb]);
        }
      }
      // stores: after the lane-half swaps v[8h .. 8h+7] are channels
      // nb*32 + 16h + 8*lhi + 0..7 of pixel mb + lane%32
      const bool in_img = oh0 + ohl < P;
#pragma unroll
      for (int nb = 0; nb < 2; ++nb) {
        float v[16];
#pragma unroll
        for (int e = 0; e < 16; ++e) v[e] = at[nb][e];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          lane_half_swap(v[q], v[4 + q]);
          lane_half_swap(v[8 + q], v[12 + q]);
        }
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          V8 o;
#pragma unroll
          for (int e = 0; e < 8; ++e) o.h[e] = to_h16(v[h * 8 + e]);
          if (in_img) store16(a.out + (M0 + m) * 64 + nb * 32 + h * 16 + lhi * 8, o);
        }
      }
    }
    __syncthreads();
    stage();
    __syncthreads();
  }
}

}  // namespace

namespace {

enum class IgemmKind { kLds, kDirect, kDma, kPointwise, k3x3 };

// Kernel choice per problem (measured on MI355X over the ResNet-50 shapes at
// batch 32 and 128): the pointwise kernel for 1x1 filters over 64 or 128
// channels with 128+ output channels; the DMA-staged kernel for reductions of
// 512 and more (every 3x3 layer, the 1x1 layers with 512+ input channels);
// below that the register-direct kernel for short reductions or small M,
// else the LDS-staged one.  All four give identical bits.
IgemmKind igemm_kind(const IgemmArgs& a) {
  if (c3_tiles_per_image(a) > 0) return IgemmKind::k3x3;
  {
    // a 1x1 filter over 64 or 128 channels (or 256 without an addend) with a
    // dense output of 128+ channels: the pointwise kernel.  (Over 256 channels
    // its workgroups, one per CU walking a fixed share of the tiles, ran the
    // conv4_x block inputs' data gradients 48 us against 58 alone, but 82-89
    // against 66 in the training step, beside the weight gradients on the
    // second stream: the register-direct kernel's one-tile workgroups share
    // the CUs better.)
    const IgemmPhase& p = a.ph[0];
    const int64_t act = (int64_t)a.N * a.Hi * a.Wi * a.Ci * 2;
    const bool ci_ok = a.Ci == 64 || a.Ci == 128 || (a.Ci == 256 && !a.addend);
    if (a.nphase == 1 && p.Rt == 1 && p.St == 1 && p.pad_h == 0 && p.pad_w == 0 &&
        p.oph == 0 && p.opw == 0 && a.os_h == 1 && a.os_w == 1 && a.OH == p.Ho &&
        a.OW == p.Wo && ci_ok && p.ldb == a.Ci && a.Co >= 128 &&
        a.Co % 8 == 0 && a.ldo % 8 == 0 && act < ((int64_t)1 << 31))
      return IgemmKind::kPointwise;
  }
  int maxM = 0, maxK = 0, maxT = 0;
  int64_t maxF = 0;
  for (int p = 0; p < a.nphase; ++p) {
    const int m = a.N * a.ph[p].Ho * a.ph[p].Wo;
    const int t = a.ph[p].Rt * a.ph[p].St;
    const int64_t f = (int64_t)a.Co * a.ph[p].ldb * 2;
    if (m > maxM) maxM = m;
    if (t * a.Ci > maxK) maxK = t * a.Ci;
    if (t > maxT) maxT = t;
    if (f > maxF) maxF = f;
  }
  const int64_t act = (int64_t)a.N * a.Hi * a.Wi * a.Ci * 2;
  // (a 512-long 1x1 reduction is faster on it too, except in a strided data
  // gradient, whose empty phases favour the register-direct kernel)
  const int kmin = a.nphase > 1 ? 576 : 512;
  if (a.Ci % 64 == 0 && maxK >= kmin && maxT <= 32 && act < ((int64_t)1 << 31) &&
      maxF <= ((int64_t)1 << 30))
    return IgemmKind::kDma;
  if (a.Ci % 32 == 0 && (maxK <= 512 || maxM <= 8192)) return IgemmKind::kDirect;
  return IgemmKind::kLds;
}

}  // namespace

bool igemm_stats_pay(const IgemmArgs& a) {
  // Measured on every ResNet-50 conv -> BN shape at batch 128 (fused call vs
  // convolution + the BN's own statistics pass): the 3x3 64-channel kernel
  // without statistics beats the DMA-staged kernel with them by more than the
  // statistics pass costs (97.7 vs 78.6 us), and so does the DMA-staged
  // kernel's statistics-free form from 100,352 output rows on (the 28x28
  // layers, 2-5 us); below that, and on the other kernels, fusing pays.
  if (!igemm_takes_stats(a)) return false;
  IgemmArgs b = a;
  b.stat = nullptr;
  if (igemm_kind(b) == IgemmKind::k3x3) return false;
  b.stat = reinterpret_cast<float*>(1);
  return !(igemm_kind(b) == IgemmKind::kDma && (int64_t)a.N * a.OH * a.OW >= 100352);
}

bool igemm_takes_apply(const IgemmArgs& a) {
  // the pointwise kernel over 64 input channels: a second pass that
  // recomputes y from x (a quarter of y's bytes) and writes z in place of the
  // BN apply's read of y
  IgemmArgs b = a;
  b.stat = nullptr;
  return !a.addend && !a.amask && a.Ci == 64 && igemm_kind(b) == IgemmKind::kPointwise;
}

int igemm_stat_records(const IgemmArgs& a) {
  const int ntiles = ceil_div(a.N * a.ph[0].Ho * a.ph[0].Wo, 128);
  return igemm_kind(a) == IgemmKind::kPointwise
             ? pw_row_groups(ntiles, a.Ci, true, ceil_div(a.Co, pw_tile_n(a)))
             : ntiles;
}

bool igemm_takes_stats(const IgemmArgs& a) {
  // the kernel that would run with statistics requested (the 3x3 kernel
  // leaves them to the DMA-staged one)
  IgemmArgs b = a;
  b.stat = reinterpret_cast<float*>(1);
  return igemm_kind(b) != IgemmKind::kLds;
}

// ---- dense GEMM with a split reduction ------------------------------------------
// A 1x1 filter over 1x1 images is the plain GEMM out[m][n] = sum_k act[m][k]
// filt[n][k] (m an image).  With few rows (a classifier's batch) its tiles are
// too few for the CUs and each walks the whole reduction, so the reduction is
// split: workgroup (M tile of 32, N tile of 128, split z) has four waves, one
// 32 x 32 block each, which load both operands' MFMA fragments for k in
// [z*kc, (z+1)*kc) straight from global memory (16 bytes per lane, all of
// them in flight together) and store the float32 block to part[z].  A second kernel
// adds the splits in order (then the addend) and rounds once.
constexpr int kDenseKc = 256;  // reduction elements per split

int dense_gemm_splits(int64_t M, int K, int Co) {
  const int64_t tiles = ((M + 31) / 32) * ((Co + 127) / 128);
  if (M > 512 || K < 2 * kDenseKc || tiles >= 128) return 0;
  return (K + kDenseKc - 1) / kDenseKc;
}

__global__ __launch_bounds__(256) void dense_splitk_kernel(const IgemmArgs a) {
  const int M = a.N, K = a.Ci;
  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int lrow = lane & 31, lhi = lane >> 5;
  const int m = blockIdx.x * 32 + lrow;
  const int n = blockIdx.y * 128 + wave * 32 + lrow;
  const int k0 = blockIdx.z * kDenseKc;
  const int k1 = k0 + kDenseKc < K ? k0 + kDenseKc : K;
  // range-checked buffer loads: a row past M or Co, or k past k1, reads
  // zeros (K % 8 == 0: a lane's 8 elements are all inside or all past k1)
  constexpr uint32_t OOB = 0x80000000u;
  const __amdgpu_buffer_rsrc_t rs_a = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<h16*>(a.act), (short)0, (int)((int64_t)M * K * 2), 0x00020000);
  const __amdgpu_buffer_rsrc_t rs_b = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<h16*>(a.ph[0].filt), (short)0, (int)((int64_t)a.Co * a.ph[0].ldb * 2), 0x00020000);
  const uint32_t a_row = m < M ? (uint32_t)m * (uint32_t)K * 2u : OOB;
  const uint32_t b_row = n < a.Co ? (uint32_t)n * (uint32_t)a.ph[0].ldb * 2u : OOB;
  // all of the split's operand fragments in flight at once, then its MFMAs
  constexpr int KSTEPS = kDenseKc / 16;
  half8 af[KSTEPS], bf[KSTEPS];
#pragma unroll
  for (int u = 0; u < KSTEPS; ++u) {
    const int kk = k0 + 16 * u + 8 * lhi;
    const uint32_t ko = (uint32_t)kk * 2u;
    const bool ok = kk < k1;
    af[u] = __builtin_bit_cast(half8, __builtin_amdgcn_raw_buffer_load_b128(
                                          rs_a, ok && a_row != OOB ? a_row + ko : OOB, 0, 0));
    bf[u] = __builtin_bit_cast(half8, __builtin_amdgcn_raw_buffer_load_b128(
                                          rs_b, ok && b_row != OOB ? b_row + ko : OOB, 0, 0));
  }
  floatx16 acc;
#pragma unroll
  for (int e = 0; e < 16; ++e) acc[e] = 0.0f;
#pragma unroll
  for (int u = 0; u < KSTEPS; ++u) acc = mfma32x32x16(af[u], bf[u], acc);
  // lane: column n; rows 8*(e/4) + 4*lhi + e%4 of the M tile
  if (n >= a.Co) return;
  float* dst = a.part + (int64_t)blockIdx.z * M * a.Co + n;
#pragma unroll
  for (int e = 0; e < 16; ++e) {
    const int mr = blockIdx.x * 32 + 8 * (e >> 2) + 4 * lhi + (e & 3);
    if (mr < M) dst[(int64_t)mr * a.Co] = acc[e];
  }
}

__global__ __launch_bounds__(256) void dense_splitk_reduce(const IgemmArgs a) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t total = (int64_t)a.N * a.Co;
  if (i >= total) return;
  float v = 0.0f;
  for (int z = 0; z < a.splits; ++z) v += a.part[z * total + i];
  const int64_t m = i / a.Co, n = i - m * a.Co;
  const int64_t off = m * a.ldo + n;
  if (a.addend) v += to_f32(a.addend[off]);
  a.out[off] = to_h16(v);
}

// whether launch_igemm runs this problem as a dense GEMM with a split
// reduction (the caller provided part for a.splits splits)
static bool dense_split_ok(const IgemmArgs& a) {
  const IgemmPhase& p = a.ph[0];
  return a.part && a.splits > 1 && !a.stat && !a.bn_stats && !a.amask && a.astride <= 1 &&
         a.nphase == 1 &&
         a.Hi == 1 && a.Wi == 1 && p.Rt == 1 && p.St == 1 && p.pad_h == 0 && p.pad_w == 0 &&
         p.Ho == 1 && p.Wo == 1 && a.OH == 1 && a.OW == 1 && p.oph == 0 && p.opw == 0 &&
         a.Ci % 8 == 0 && p.ldb % 8 == 0 && a.splits == dense_gemm_splits(a.N, a.Ci, a.Co);
}

hipError_t launch_igemm(const IgemmArgs& a, hipStream_t st) {
  if (a.bn_stats && (a.stat || !igemm_takes_apply(a))) return hipErrorInvalidValue;
  if (dense_split_ok(a)) {
    const dim3 grid(ceil_div(a.N, 32), ceil_div(a.Co, 128), a.splits);
    hipLaunchKernelGGL(dense_splitk_kernel, grid, dim3(256), 0, st, a);
    const int64_t total = (int64_t)a.N * a.Co;
    hipLaunchKernelGGL(dense_splitk_reduce, dim3((unsigned)((total + 255) / 256)), dim3(256), 0,
                       st, a);
    return hipGetLastError();
  }
  switch (igemm_kind(a)) {
    case IgemmKind::kDma: {
      // two stages (two workgroups per CU) unless the grid fits the 256 CUs
      // once, where a third stage of prefetch costs no occupancy
      int maxM = 0;
      for (int p = 0; p < a.nphase; ++p) maxM = max(maxM, a.N * a.ph[p].Ho * a.ph[p].Wo);
      const bool narrow = a.Co <= 64;
      const int64_t wgs = (int64_t)ceil_div(maxM, 128) * ceil_div(a.Co, narrow ? 64 : 128) * a.nphase;
      if (narrow) return wgs <= 256 ? launch_cfg7<2, 1, 2, 2, 3>(a, st) : launch_cfg7<2, 1, 2, 2, 2>(a, st);
      return wgs <= 256 ? launch_cfg7<2, 2, 2, 2, 3>(a, st) : launch_cfg7<2, 2, 2, 2, 2>(a, st);
    }
    case IgemmKind::kDirect:
      return a.Co <= 64 ? launch_cfg4<1, 2>(a, st) : launch_cfg4<1, 4>(a, st);
    case IgemmKind::k3x3:
      return launch_c3(a, c3_tiles_per_image(a), st);
    case IgemmKind::kPointwise: {
      const bool wide = pw_tile_n(a) == 256;
      if (a.Ci == 64) return wide ? launch_pw<64, 256>(a, st) : launch_pw<64, 128>(a, st);
      if (a.Ci == 128) return wide ? launch_pw<128, 256>(a, st) : launch_pw<128, 128>(a, st);
      return launch_pw<256, 128>(a, st);
    }
    default:
      return a.Co <= 64 ? launch_cfg<128, 64, 4, 1, 64>(a, st) : launch_cfg<128, 128, 2, 2, 64>(a, st);
  }
}

// The stem kernel's problem: 3 input channels (unpadded NHWC, W a multiple
// of 8), 7x7 filter (KRSC, 147 per output channel), stride 2, pad 3, 64 dense
// output channels, 16 .. 128 output columns in steps of 16, no statistics.
bool stem_conv_ok(const IgemmArgs& a) {
  const IgemmPhase& p = a.ph[0];
  const bool shape = a.Ci == 3 && a.nphase == 1 && p.Rt == 7 && p.St == 7 && p.ldb == 147 &&
                     p.pad_h == 3 && p.pad_w == 3 && a.stride_h == 2 && a.stride_w == 2 &&
                     p.oph == 0 && p.opw == 0 && a.os_h == 1 && a.os_w == 1 && a.Co == 64 &&
                     a.ldo == 64 && !a.addend && a.Wi % 8 == 0 &&
                     a.Wi == 2 * a.OW && a.OH == p.Ho && a.OW == p.Wo &&
                     a.OW % 16 == 0 && a.OW >= 16 && a.OW <= kStemMaxQ &&
                     (int64_t)a.N * a.Hi * a.Wi * 6 < ((int64_t)1 << 31);
  return shape && !a.stat;
}

hipError_t launch_stem(const IgemmArgs& a, hipStream_t st) {
  const int tpi = ceil_div(a.OH, kStemTR);
  const int ntiles = a.N * tpi;
  const int grid = ntiles < 256 ? ntiles : 256;
  const dim3 block(a.OW * 4);
  hipLaunchKernelGGL(stem_kernel, dim3(grid), block, 0, st, a, ntiles);
  return hipGetLastError();
}

}  // namespace fp16k
