// Shared device-side types and helpers for the fp16train HIP kernels (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

typedef _Float16 h16;
typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef _Float16 half4 __attribute__((ext_vector_type(4)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// 16-byte vector of eight binary16 values, viewable as halves or dwords.
union V8 {
  u32x4 u;
  half8 h;
  uint32_t d[4];
  uint16_t s[8];
};

__device__ __forceinline__ V8 load16(const void* p) {
  V8 v;
  v.u = *reinterpret_cast<const u32x4*>(p);
  return v;
}

__device__ __forceinline__ void store16(void* p, const V8& v) {
  *reinterpret_cast<u32x4*>(p) = v.u;
}

__device__ __forceinline__ V8 zero8() {
  V8 v;
  v.u = u32x4{0u, 0u, 0u, 0u};
  return v;
}

// float32 -> binary16, round to nearest even (v_cvt_f16_f32 in the default
// rounding mode; binary16 subnormals are produced, not flushed).  The empty
// asm pins the float32 value in a register: without it the compiler may fold
// a preceding fma into v_fma_mix*_f16, which rounds the exact result once to
// binary16 instead of first to float32 -- a different result in rare cases,
// and not the declared sequence.
__device__ __forceinline__ h16 to_h16(float v) {
  __asm__("" : "+v"(v));
  return (h16)v;
}
__device__ __forceinline__ float to_f32(h16 v) { return (float)v; }

// float64 -> binary16 with a single rounding (nearest even).  The double is
// first narrowed to float32 with round-to-odd (truncate, then force the last
// bit to 1 if anything was lost); float32 carries more than 2*11+1 bits, so
// the following RNE to binary16 equals a direct rounding of the double
// (Boldo and Melquiond, "When double rounding is odd", 2005).
__device__ __forceinline__ h16 dbl_to_h16(double d) {
  float f = (float)d;
  if (!__builtin_isnan(d) && (double)f != d && __builtin_fabs(d) < 3.0e38) {
    uint32_t b = __builtin_bit_cast(uint32_t, f);
    if (__builtin_fabs((double)f) > __builtin_fabs(d)) b -= 1u;  // one ulp toward zero
    f = __builtin_bit_cast(float, b | 1u);
  }
  return (h16)f;
}

// Max pooling's comparison: a later element replaces the running maximum
// only if it is strictly larger, or if it is the first NaN (NaN propagates;
// ties keep the earliest position).
__device__ __forceinline__ bool pool_takes(float best, float v) {
  // (non-short-circuit: compare-and-select, no branch per element)
  return ((int)!__builtin_isnan(best) & ((int)__builtin_isnan(v) | (int)(v > best))) != 0;
}

// ReLU keeping NaN and mapping -0 and negatives to +0.
__device__ __forceinline__ float relu_keep_nan(float v) {
  return (v > 0.0f || __builtin_isnan(v)) ? v : 0.0f;
}

// Per-channel forward coefficients of the BN apply's declared float32 sequence
// (Section 4.1: normalise, scale by gamma and the post scale, add beta, then
// the shortcut and the ReLU); shared by the BN kernels and the convolution
// epilogue that applies the BN, so both give the same bits.
struct FwdCoef {
  float mean, a, b, sg;
};
__device__ __forceinline__ FwdCoef fwd_coef(const float* stats, const h16* gamma, const h16* beta,
                                            int C, int c, float s) {
  FwdCoef k;
  k.mean = stats[c];
  const float rstd = stats[C + c];
  const float sg = s * to_f32(gamma[c]);
  k.a = sg * rstd;
  k.b = s * to_f32(beta[c]);
  k.sg = sg;
  return k;
}

__device__ __forceinline__ float fwd_value(float x, const FwdCoef& k, bool has_r, float r,
                                           bool relu, bool swap) {
  const float t = x - k.mean;
  float v;
  if (swap) {
    v = __builtin_fmaf(t, k.a, __builtin_fmaf(k.sg, r, k.b));
  } else {
    v = __builtin_fmaf(t, k.a, k.b);
    if (has_r) v = v + r;
  }
  if (relu) v = relu_keep_nan(v);
  return v;
}

// Transpose an 8x8 block of binary16 values held as eight 16-byte rows:
// out[j].s[i] = in[i].s[j].  Built from byte permutes (v_perm_b32).
__device__ __forceinline__ void transpose8x8(const V8 (&in)[8], V8 (&out)[8]) {
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const uint32_t sel = (j & 1) ? 0x07060302u : 0x05040100u;
#pragma unroll
    for (int i = 0; i < 8; i += 2) {
      // low half <- in[i].s[j], high half <- in[i+1].s[j]
      out[j].d[i >> 1] = __builtin_amdgcn_perm(in[i + 1].d[j >> 1], in[i].d[j >> 1], sel);
    }
  }
}

__device__ __forceinline__ floatx16 mfma32x32x16(const half8& a, const half8& b, const floatx16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
}

inline int ceil_div(int a, int b) { return (a + b - 1) / b; }
inline int64_t ceil_div64(int64_t a, int64_t b) { return (a + b - 1) / b; }
