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
// Two kernels, both v_mfma_f32_32x32x16_f16 with float32 accumulators and
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
//
// Epilogue (both): each wave stages a 32-row band of its float32 tile in LDS
// and writes whole output rows with 16-byte stores.  Every value is rounded
// once to binary16 (RNE), optionally after adding a binary16 addend in
// float32.  igemm4_kernel can also take the statistics of a BN that follows
// the convolution, without a second pass over the output: per 128-row tile
// and channel, shifted sums of the rounded values (IgemmArgs::stat).

#include "kernels.hpp"

namespace fp16k {
namespace {

// keep a value materialised in a VGPR (blocks branchy code motion around it)
__device__ __forceinline__ uint32_t pin_v(uint32_t x) {
  __asm__("" : "+v"(x));
  return x;
}
// workgroup barrier without the implied memory fence; callers wait first
__device__ __forceinline__ void bare_barrier() { __asm__ volatile("s_barrier" ::: "memory"); }
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

  const IgemmPhase ph = a.ph[blockIdx.z];
  const int HoWo = ph.Ho * ph.Wo;
  const int M = a.N * HoWo;
  const int m0 = blockIdx.x * BM;
  if (m0 >= M) return;
  const int n0 = blockIdx.y * BN;
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
        for (int tn = 0; tn < TN; ++tn) acc[tm][tn] = mfma32x32x16(af[tm], bf[tn], acc[tm][tn]);
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

  const IgemmPhase ph = a.ph[blockIdx.z];
  const int HoWo = ph.Ho * ph.Wo;
  const int M = a.N * HoWo;
  const int m0 = blockIdx.x * BM;
  if (m0 >= M) return;
  const int n0 = blockIdx.y * BN;
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
              const V8 ad = load16(a.addend + off);
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
                if (a.addend) x += to_f32(a.addend[off + e]);
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

template <int TM, int TN>
hipError_t launch_cfg4(const IgemmArgs& a, hipStream_t st) {
  using K = Cfg4<TM, TN>;
  int maxM = 0;
  for (int p = 0; p < a.nphase; ++p) {
    const int m = a.N * a.ph[p].Ho * a.ph[p].Wo;
    if (m > maxM) maxM = m;
  }
  if (maxM == 0 || a.nphase == 0) return hipSuccess;
  dim3 grid(ceil_div(maxM, K::BM), ceil_div(a.Co, K::BN), a.nphase);
  hipLaunchKernelGGL((igemm4_kernel<TM, TN>), grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

template <int BM, int BN, int WM, int WN, int BK>
hipError_t launch_cfg(const IgemmArgs& a, hipStream_t st) {
  int maxM = 0;
  for (int p = 0; p < a.nphase; ++p) {
    const int m = a.N * a.ph[p].Ho * a.ph[p].Wo;
    if (m > maxM) maxM = m;
  }
  if (maxM == 0 || a.nphase == 0) return hipSuccess;
  dim3 grid(ceil_div(maxM, BM), ceil_div(a.Co, BN), a.nphase);
  hipLaunchKernelGGL((igemm_kernel<BM, BN, WM, WN, BK>), grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace

bool igemm_direct(const IgemmArgs& a) {
  int maxM = 0, maxK = 0;
  for (int p = 0; p < a.nphase; ++p) {
    const int m = a.N * a.ph[p].Ho * a.ph[p].Wo;
    const int k = a.ph[p].Rt * a.ph[p].St * a.Ci;
    if (m > maxM) maxM = m;
    if (k > maxK) maxK = k;
  }
  return (a.Ci % 32 == 0) && (maxK <= 512 || maxM <= 8192);
}

// Kernel choice per problem (measured on MI355X over the ResNet-50 shapes):
// the register-direct kernel is faster for short reductions and small M; the
// LDS-staged one for long reductions over large M.  Results are identical.
hipError_t launch_igemm(const IgemmArgs& a, hipStream_t st) {
  int maxM = 0, maxK = 0;
  for (int p = 0; p < a.nphase; ++p) {
    const int m = a.N * a.ph[p].Ho * a.ph[p].Wo;
    const int k = a.ph[p].Rt * a.ph[p].St * a.Ci;
    if (m > maxM) maxM = m;
    if (k > maxK) maxK = k;
  }
  const bool direct = igemm_direct(a);
  if (a.Co <= 64) return direct ? launch_cfg4<1, 2>(a, st) : launch_cfg<128, 64, 4, 1, 64>(a, st);
  return direct ? launch_cfg4<1, 4>(a, st) : launch_cfg<128, 128, 2, 2, 64>(a, st);
}

}  // namespace fp16k
