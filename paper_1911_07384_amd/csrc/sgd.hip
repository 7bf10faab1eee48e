// Momentum SGD on FP16 weights and FP16 momentum, no master copy
// (arXiv:1911.07384, Section 5.1 recipe and Section 5.2).
//
// Per element, in float32 exactly as written (explicit fma, no contraction):
//   d  = fma(wd, w, g)
//   m' = rne16(fma(mu, m, d))
//   w' = rne16(fma(-lr, m', w))
// Bandwidth-bound: 10 bytes per element (read w, g, m; write w, m).  Each
// thread moves 16-byte vectors; the grid strides over the arrays.
// launch_sgd_f16 runs the same update with every operation in binary16.

#include "kernels.hpp"

namespace fp16k {
namespace {

__device__ __forceinline__ void sgd_one(h16& w, h16 g, h16& m, float lr, float mu, float wd) {
  const float wf = to_f32(w);
  const float d = __builtin_fmaf(wd, wf, to_f32(g));
  const h16 m1 = to_h16(__builtin_fmaf(mu, to_f32(m), d));
  const h16 w1 = to_h16(__builtin_fmaf(-lr, to_f32(m1), wf));
  m = m1;
  w = w1;
}

// Strict binary16 arithmetic: three binary16 fused multiply-adds (one
// rounding each, v_fma_f16) with binary16 scalars.
__device__ __forceinline__ void sgd_one_f16(h16& w, h16 g, h16& m, h16 nlr, h16 mu, h16 wd) {
  const h16 d = __builtin_fmaf16(wd, w, g);
  const h16 m1 = __builtin_fmaf16(mu, m, d);
  const h16 w1 = __builtin_fmaf16(nlr, m1, w);
  m = m1;
  w = w1;
}

struct SgdF32 {
  float lr, mu, wd;
  __device__ void operator()(h16& w, h16 g, h16& m) const { sgd_one(w, g, m, lr, mu, wd); }
};
struct SgdF16 {
  h16 nlr, mu, wd;
  __device__ void operator()(h16& w, h16 g, h16& m) const { sgd_one_f16(w, g, m, nlr, mu, wd); }
};

template <class Op>
__global__ __launch_bounds__(256) void sgd_kernel(h16* __restrict__ w, const h16* __restrict__ g,
                                                  h16* __restrict__ m, size_t n, Op op) {
  const size_t nvec = n / 8;
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  for (; i < nvec; i += stride) {
    V8 wv = load16(w + i * 8);
    const V8 gv = load16(g + i * 8);
    V8 mv = load16(m + i * 8);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      h16 we = wv.h[e], me = mv.h[e];
      op(we, gv.h[e], me);
      wv.h[e] = we;
      mv.h[e] = me;
    }
    store16(m + i * 8, mv);
    store16(w + i * 8, wv);
  }
  // tail (n not a multiple of 8): the first threads of the grid take it
  const size_t t = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const size_t j = nvec * 8 + t;
  if (j < n) {
    h16 wv = w[j], mv = m[j];
    op(wv, g[j], mv);
    m[j] = mv;
    w[j] = wv;
  }
}

}  // namespace

namespace {
template <class Op>
hipError_t launch_sgd_op(h16* w, const h16* g, h16* m, size_t n, Op op, hipStream_t st) {
  if (n == 0) return hipSuccess;
  const size_t nvec = n / 8;
  size_t blocks = (nvec + 255) / 256;
  if (blocks < 1) blocks = 1;
  // one vector per thread up to a grid of 64k blocks, grid-stride beyond
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(sgd_kernel<Op>, dim3((unsigned)blocks), dim3(256), 0, st, w, g, m, n, op);
  return hipGetLastError();
}
}  // namespace

hipError_t launch_sgd(h16* w, const h16* g, h16* m, size_t n, float lr, float momentum,
                      float weight_decay, hipStream_t st) {
  return launch_sgd_op(w, g, m, n, SgdF32{lr, momentum, weight_decay}, st);
}

hipError_t launch_sgd_f16(h16* w, const h16* g, h16* m, size_t n, float lr, float momentum,
                          float weight_decay, hipStream_t st) {
  // binary16 roundings (nearest even) of the float32 scalars
  return launch_sgd_op(w, g, m, n, SgdF16{(h16)(-lr), (h16)momentum, (h16)weight_decay}, st);
}

}  // namespace fp16k
