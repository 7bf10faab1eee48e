// Oracle for the all-FP16 training hot path -- TEST INFRASTRUCTURE ONLY.
//
// This library is the plain, slow CPU definition that the HIP kernels are
// checked against.  Only the tests, the smoke check and the CPU-baseline leg
// of the benchmark may load it; the product path never does.  It shares no
// code, header, table or helper with the HIP library.
//
// What it computes follows arXiv:1911.07384 ("Distributed low-precision
// Training Without Mixed Precision"):
//   * every tensor crossing a kernel boundary is stored in IEEE binary16
//     (Section 5.2: activations, weights and gradients all stored in FP16,
//     no high-precision master copy);
//   * rounding to binary16 is IEEE round-to-nearest, ties to even, with
//     gradual underflow and overflow to infinity (Section 3 names IEEE 754;
//     Section 4.2 leaves the rounding method open, reading: IEEE default);
//   * convolutions are ResNet-50's (Section 5.1), written here as plain
//     cross-correlation sums in float64 (exact products of binary16 values);
//   * batch normalisation follows Eq. (1)-(2) of Section 4.1 per channel over
//     (N, H, W), with the 0.25 output multiplier of Section 4.2 and the ReLU
//     that follows each BN (Section 1);
//   * the optimiser is momentum SGD with FP16 weights and FP16 momentum
//     (Section 5.1 recipe, Section 5.2 no master copy);
//   * the rest of ResNet-50 (Section 5.1): 3x3 stride-2 max pooling after the
//     stem, global average pooling, the fully connected classifier with bias,
//     and the softmax cross-entropy loss averaged over the local batch.
//
// Readings where the paper is silent are listed with each function.
//
// Build: g++ -O2 -fopenmp -ffp-contract=off -fno-fast-math -shared -fPIC.
// Contraction is off so that the declared float32 sequences below are
// evaluated exactly as written.

#include <cmath>
#include <cstdint>
#include <cstdlib>
#include <cstring>
#include <vector>

#ifdef _OPENMP
#include <omp.h>
#endif

namespace {

// ---------------------------------------------------------------------------
// binary16 codec (Section 3: IEEE 754 interchange format; 1 sign bit,
// 5 exponent bits with bias 15, 10 fraction bits).
// ---------------------------------------------------------------------------

double half_to_double(uint16_t h) {
  const int sign = (h >> 15) & 1;
  const int exp = (h >> 10) & 0x1F;
  const int frac = h & 0x3FF;
  double mag;
  if (exp == 0) {
    mag = std::ldexp((double)frac, -24);            // zero or subnormal
  } else if (exp == 31) {
    if (frac != 0) return std::nan("");
    mag = INFINITY;
  } else {
    mag = std::ldexp((double)(1024 + frac), exp - 25);  // (1.f) * 2^(exp-15)
  }
  return sign ? -mag : mag;
}

// Round a real (given exactly as a double) to the nearest binary16 value,
// ties to even, subnormals kept (gradual underflow), overflow to +-inf.
uint16_t round_half(double v) {
  if (std::isnan(v)) return 0x7E00;
  const uint16_t sign = std::signbit(v) ? 0x8000 : 0;
  const double a = std::fabs(v);
  if (std::isinf(a)) return sign | 0x7C00;
  if (a < std::ldexp(1.0, -14)) {
    // Subnormal range: the value in units of 2^-24 (exact scaling), rounded
    // to an integer with ties to even.  A result of 1024 is the smallest
    // normal number, whose encoding is exactly 0x0400.
    const double units = std::nearbyint(a * std::ldexp(1.0, 24));
    return sign | (uint16_t)units;
  }
  int e2 = 0;
  std::frexp(a, &e2);          // a = f * 2^e2 with f in [0.5, 1)
  int e = e2 - 1;              // a in [2^e, 2^(e+1))
  double sig = std::nearbyint(a * std::ldexp(1.0, 10 - e));  // in [1024, 2048]
  if (sig == 2048.0) {         // rounding carried into the next binade
    sig = 1024.0;
    e += 1;
  }
  if (e > 15) return sign | 0x7C00;
  return sign | (uint16_t)(((e + 15) << 10) | ((int)sig - 1024));
}

inline float half_to_float(uint16_t h) { return (float)half_to_double(h); }

std::vector<double> decode(const uint16_t* h, int64_t n) {
  std::vector<double> out((size_t)n);
  for (int64_t i = 0; i < n; ++i) out[(size_t)i] = half_to_double(h[i]);
  return out;
}

// ---------------------------------------------------------------------------
// Convolution geometry.  shp = {N, C, H, W, K, R, S, stride_h, stride_w,
// pad_h, pad_w, layout}; layout 0: activations NHWC, filter KRSC;
// layout 1: activations NCHW, filter KCRS.  Output size follows the usual
// zero-padded cross-correlation: P = floor((H + 2 pad_h - R) / stride_h) + 1.
// ---------------------------------------------------------------------------

struct Conv {
  int64_t N, C, H, W, K, R, S, sh, sw, ph, pw, P, Q;
  int layout;
  explicit Conv(const int32_t* s) {
    N = s[0]; C = s[1]; H = s[2]; W = s[3]; K = s[4]; R = s[5]; S = s[6];
    sh = s[7]; sw = s[8]; ph = s[9]; pw = s[10]; layout = s[11];
    P = (H + 2 * ph - R) / sh + 1;
    Q = (W + 2 * pw - S) / sw + 1;
  }
  // activation of C channels on an H x W grid
  int64_t xi(int64_t n, int64_t c, int64_t h, int64_t w) const {
    return layout == 0 ? ((n * H + h) * W + w) * C + c : ((n * C + c) * H + h) * W + w;
  }
  // activation of K channels on the P x Q output grid
  int64_t yi(int64_t n, int64_t k, int64_t p, int64_t q) const {
    return layout == 0 ? ((n * P + p) * Q + q) * K + k : ((n * K + k) * P + p) * Q + q;
  }
  int64_t wi(int64_t k, int64_t c, int64_t r, int64_t s) const {
    return layout == 0 ? ((k * R + r) * S + s) * C + c : ((k * C + c) * R + r) * S + s;
  }
  void y_coords(int64_t idx, int64_t* n, int64_t* k, int64_t* p, int64_t* q) const {
    if (layout == 0) {
      *k = idx % K; idx /= K; *q = idx % Q; idx /= Q; *p = idx % P; *n = idx / P;
    } else {
      *q = idx % Q; idx /= Q; *p = idx % P; idx /= P; *k = idx % K; *n = idx / K;
    }
  }
  void x_coords(int64_t idx, int64_t* n, int64_t* c, int64_t* h, int64_t* w) const {
    if (layout == 0) {
      *c = idx % C; idx /= C; *w = idx % W; idx /= W; *h = idx % H; *n = idx / H;
    } else {
      *w = idx % W; idx /= W; *h = idx % H; idx /= H; *c = idx % C; *n = idx / C;
    }
  }
  void w_coords(int64_t idx, int64_t* k, int64_t* c, int64_t* r, int64_t* s) const {
    if (layout == 0) {
      *c = idx % C; idx /= C; *s = idx % S; idx /= S; *r = idx % R; *k = idx / R;
    } else {
      *s = idx % S; idx /= S; *r = idx % R; idx /= R; *c = idx % C; *k = idx / C;
    }
  }
  int64_t x_size() const { return N * C * H * W; }
  int64_t y_size() const { return N * K * P * Q; }
  int64_t w_size() const { return K * C * R * S; }
};

// Forward: y[n,k,p,q] = sum_{c,r,s} x[n,c,p*sh-ph+r, q*sw-pw+s] * W[k,c,r,s],
// taps outside the image contribute zero (zero padding).
double conv_fwd_elem(const Conv& d, const double* x, const double* w,
                     int64_t n, int64_t k, int64_t p, int64_t q) {
  double acc = 0.0;
  for (int64_t r = 0; r < d.R; ++r) {
    const int64_t h = p * d.sh - d.ph + r;
    if (h < 0 || h >= d.H) continue;
    for (int64_t s = 0; s < d.S; ++s) {
      const int64_t ww = q * d.sw - d.pw + s;
      if (ww < 0 || ww >= d.W) continue;
      for (int64_t c = 0; c < d.C; ++c) acc += x[d.xi(n, c, h, ww)] * w[d.wi(k, c, r, s)];
    }
  }
  return acc;
}

// Data gradient: the adjoint of the forward map with respect to x,
// dx[n,c,h,w] = sum over (k, r, s) such that h + ph - r = p*sh and
// w + pw - s = q*sw for some output position (p, q) inside the P x Q grid,
// of dy[n,k,p,q] * W[k,c,r,s].
double conv_dgrad_elem(const Conv& d, const double* dy, const double* w,
                       int64_t n, int64_t c, int64_t h, int64_t ww) {
  double acc = 0.0;
  for (int64_t r = 0; r < d.R; ++r) {
    const int64_t th = h + d.ph - r;
    if (th < 0 || th % d.sh != 0) continue;
    const int64_t p = th / d.sh;
    if (p >= d.P) continue;
    for (int64_t s = 0; s < d.S; ++s) {
      const int64_t tw = ww + d.pw - s;
      if (tw < 0 || tw % d.sw != 0) continue;
      const int64_t q = tw / d.sw;
      if (q >= d.Q) continue;
      for (int64_t k = 0; k < d.K; ++k) acc += dy[d.yi(n, k, p, q)] * w[d.wi(k, c, r, s)];
    }
  }
  return acc;
}

// Weight gradient: the adjoint of the forward map with respect to W,
// dW[k,c,r,s] = sum_{n,p,q} dy[n,k,p,q] * x[n,c,p*sh-ph+r, q*sw-pw+s].
double conv_wgrad_elem(const Conv& d, const double* x, const double* dy,
                       int64_t k, int64_t c, int64_t r, int64_t s) {
  double acc = 0.0;
  for (int64_t n = 0; n < d.N; ++n)
    for (int64_t p = 0; p < d.P; ++p) {
      const int64_t h = p * d.sh - d.ph + r;
      if (h < 0 || h >= d.H) continue;
      for (int64_t q = 0; q < d.Q; ++q) {
        const int64_t ww = q * d.sw - d.pw + s;
        if (ww < 0 || ww >= d.W) continue;
        acc += dy[d.yi(n, k, p, q)] * x[d.xi(n, c, h, ww)];
      }
    }
  return acc;
}

// ---------------------------------------------------------------------------
// Batch normalisation geometry: shp = {N, C, H, W, layout}.
// ---------------------------------------------------------------------------

struct BN {
  int64_t N, C, H, W;
  int layout;
  explicit BN(const int32_t* s) {
    N = s[0]; C = s[1]; H = s[2]; W = s[3]; layout = s[4];
  }
  int64_t M() const { return N * H * W; }
  // index of the j-th element (j in [0, M)) of channel c
  int64_t at(int64_t c, int64_t j) const {
    const int64_t hw = H * W;
    const int64_t n = j / hw, rem = j % hw;
    return layout == 0 ? (n * hw + rem) * C + c : (n * C + c) * hw + rem;
  }
};

// ReLU as used in the oracle: keeps NaN, maps -0 and negatives to +0.
inline double relu_d(double v) { return (v > 0.0 || std::isnan(v)) ? v : 0.0; }
inline float relu_f(float v) { return (v > 0.0f || std::isnan(v)) ? v : 0.0f; }

}  // namespace

extern "C" {

// ---- codec entry points ---------------------------------------------------

double oracle_h2d(uint16_t h) { return half_to_double(h); }
uint16_t oracle_rne16(double v) { return round_half(v); }

void oracle_h2d_array(const uint16_t* h, double* out, int64_t n) {
  for (int64_t i = 0; i < n; ++i) out[i] = half_to_double(h[i]);
}

void oracle_rne16_array(const double* v, uint16_t* out, int64_t n) {
  for (int64_t i = 0; i < n; ++i) out[i] = round_half(v[i]);
}

// float32 input: promoted exactly to double, so this is one rounding from
// the float32 value.
void oracle_rne16_f32_array(const float* v, uint16_t* out, int64_t n) {
  for (int64_t i = 0; i < n; ++i) out[i] = round_half((double)v[i]);
}

int oracle_num_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

// Threads for the following calls (timing on one core); n < 1 is ignored.
void oracle_set_num_threads(int n) {
#ifdef _OPENMP
  if (n >= 1) omp_set_num_threads(n);
#else
  (void)n;
#endif
}

// ---- convolution ----------------------------------------------------------
// Each pass returns the float64 sum before rounding (y64, may be NULL) and
// its binary16 rounding (y16, may be NULL): one rounding at the store.

void oracle_conv_out_dims(const int32_t* shp, int32_t* p, int32_t* q) {
  Conv d(shp);
  *p = (int32_t)d.P;
  *q = (int32_t)d.Q;
}

void oracle_conv_fwd(const int32_t* shp, const uint16_t* x16, const uint16_t* w16,
                     double* y64, uint16_t* y16) {
  Conv d(shp);
  std::vector<double> x = decode(x16, d.x_size()), w = decode(w16, d.w_size());
  const int64_t total = d.y_size();
#pragma omp parallel for schedule(dynamic, 64)
  for (int64_t i = 0; i < total; ++i) {
    int64_t n, k, p, q;
    d.y_coords(i, &n, &k, &p, &q);
    const double v = conv_fwd_elem(d, x.data(), w.data(), n, k, p, q);
    if (y64) y64[i] = v;
    if (y16) y16[i] = round_half(v);
  }
}

void oracle_conv_dgrad(const int32_t* shp, const uint16_t* dy16, const uint16_t* w16,
                       double* dx64, uint16_t* dx16) {
  Conv d(shp);
  std::vector<double> dy = decode(dy16, d.y_size()), w = decode(w16, d.w_size());
  const int64_t total = d.x_size();
#pragma omp parallel for schedule(dynamic, 64)
  for (int64_t i = 0; i < total; ++i) {
    int64_t n, c, h, ww;
    d.x_coords(i, &n, &c, &h, &ww);
    const double v = conv_dgrad_elem(d, dy.data(), w.data(), n, c, h, ww);
    if (dx64) dx64[i] = v;
    if (dx16) dx16[i] = round_half(v);
  }
}

// Data gradient plus an addend with one rounding: the input gradient of a
// residual block, where the identity shortcut's gradient (the addend) joins
// the branch gradient (Section 4.1's residual connection).
//   dx16 = round_half(dgrad(dy, W) + addend).
void oracle_conv_dgrad_add(const int32_t* shp, const uint16_t* dy16, const uint16_t* w16,
                           const uint16_t* add16, double* dx64, uint16_t* dx16) {
  Conv d(shp);
  std::vector<double> dy = decode(dy16, d.y_size()), w = decode(w16, d.w_size());
  const int64_t total = d.x_size();
#pragma omp parallel for schedule(dynamic, 64)
  for (int64_t i = 0; i < total; ++i) {
    int64_t n, c, h, ww;
    d.x_coords(i, &n, &c, &h, &ww);
    const double v = conv_dgrad_elem(d, dy.data(), w.data(), n, c, h, ww) + half_to_double(add16[i]);
    if (dx64) dx64[i] = v;
    if (dx16) dx16[i] = round_half(v);
  }
}

void oracle_conv_wgrad(const int32_t* shp, const uint16_t* x16, const uint16_t* dy16,
                       double* dw64, uint16_t* dw16) {
  Conv d(shp);
  std::vector<double> x = decode(x16, d.x_size()), dy = decode(dy16, d.y_size());
  const int64_t total = d.w_size();
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t i = 0; i < total; ++i) {
    int64_t k, c, r, s;
    d.w_coords(i, &k, &c, &r, &s);
    const double v = conv_wgrad_elem(d, x.data(), dy.data(), k, c, r, s);
    if (dw64) dw64[i] = v;
    if (dw16) dw16[i] = round_half(v);
  }
}

// Sampled variants: the same element definitions at a list of flat output
// indices (in the output's own layout), for workloads too large to evaluate
// whole.  out64[j] is the float64 sum at idx[j].

void oracle_conv_fwd_at(const int32_t* shp, const uint16_t* x16, const uint16_t* w16,
                        const int64_t* idx, int64_t count, double* out64) {
  Conv d(shp);
  std::vector<double> x = decode(x16, d.x_size()), w = decode(w16, d.w_size());
#pragma omp parallel for schedule(dynamic, 16)
  for (int64_t j = 0; j < count; ++j) {
    int64_t n, k, p, q;
    d.y_coords(idx[j], &n, &k, &p, &q);
    out64[j] = conv_fwd_elem(d, x.data(), w.data(), n, k, p, q);
  }
}

void oracle_conv_dgrad_at(const int32_t* shp, const uint16_t* dy16, const uint16_t* w16,
                          const int64_t* idx, int64_t count, double* out64) {
  Conv d(shp);
  std::vector<double> dy = decode(dy16, d.y_size()), w = decode(w16, d.w_size());
#pragma omp parallel for schedule(dynamic, 16)
  for (int64_t j = 0; j < count; ++j) {
    int64_t n, c, h, ww;
    d.x_coords(idx[j], &n, &c, &h, &ww);
    out64[j] = conv_dgrad_elem(d, dy.data(), w.data(), n, c, h, ww);
  }
}

void oracle_conv_wgrad_at(const int32_t* shp, const uint16_t* x16, const uint16_t* dy16,
                          const int64_t* idx, int64_t count, double* out64) {
  Conv d(shp);
  std::vector<double> x = decode(x16, d.x_size()), dy = decode(dy16, d.y_size());
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t j = 0; j < count; ++j) {
    int64_t k, c, r, s;
    d.w_coords(idx[j], &k, &c, &r, &s);
    out64[j] = conv_wgrad_elem(d, x.data(), dy.data(), k, c, r, s);
  }
}

// ---- batch normalisation --------------------------------------------------
// Forward, Eq. (1)-(2) of Section 4.1, per channel c over the M = N*H*W
// elements of the local batch (Section 5.1: no synchronous BN):
//   mu = (1/M) sum x;  var = (1/M) sum (x - mu)^2  (biased, two passes);
//   xhat = (x - mu) / sqrt(var + eps);  z = gamma * xhat + beta;
//   u = s * z + r;  y = relu(u).
// s is the output multiplier of Section 4.2 (0.25 inside residual blocks,
// 1 for the stem BN); r is the identity shortcut (block-last BN only, may
// be NULL); relu may be switched off.  eps is held as the float32 value the
// caller passes.  y64 (may be NULL) is u or relu(u) before rounding.
//
// swap = 1 is the BN swap of Section 4.1: the shortcut joins before gamma,
//   u = s * (gamma * (xhat + r) + beta)
// (reading: the positions of the residual addition and of gamma exchange;
// the multiplier stays on the BN output).  It needs r.

void oracle_bn_fwd(const int32_t* shp, const uint16_t* x16, const uint16_t* gamma16,
                   const uint16_t* beta16, const uint16_t* res16, float eps, float post_scale,
                   int relu, double* mean_out, double* var_out, double* y64, uint16_t* y16,
                   int swap) {
  BN d(shp);
  const int64_t M = d.M();
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t c = 0; c < d.C; ++c) {
    double sum = 0.0;
    for (int64_t j = 0; j < M; ++j) sum += half_to_double(x16[d.at(c, j)]);
    const double mu = sum / (double)M;
    double ss = 0.0;
    for (int64_t j = 0; j < M; ++j) {
      const double t = half_to_double(x16[d.at(c, j)]) - mu;
      ss += t * t;
    }
    const double var = ss / (double)M;
    const double rstd = 1.0 / std::sqrt(var + (double)eps);
    const double g = half_to_double(gamma16[c]), b = half_to_double(beta16[c]);
    for (int64_t j = 0; j < M; ++j) {
      const int64_t i = d.at(c, j);
      const double xhat = (half_to_double(x16[i]) - mu) * rstd;
      double u;
      if (swap)
        u = (double)post_scale * (g * (xhat + half_to_double(res16[i])) + b);
      else {
        u = (double)post_scale * (g * xhat + b);
        if (res16) u += half_to_double(res16[i]);
      }
      if (relu) u = relu_d(u);
      if (y64) y64[i] = u;
      if (y16) y16[i] = round_half(u);
    }
    if (mean_out) mean_out[c] = mu;
    if (var_out) var_out[c] = var;
  }
}

// Forward apply with given float32 statistics (mean, rstd), as used when the
// statistics are supplied by the caller.  Declared float32 sequence (the
// reading this library fixes; every step is one IEEE float32 operation):
//   a = fl(fl(s * gamma) * rstd);  b = fl(s * beta);  t = fl(x - mean);
//   v = fma(t, a, b);  v = fl(v + r);  y = round_half(relu(v)).
// With swap (u = s*gamma*(xhat + r) + s*beta) the shortcut enters the
// offset instead:  sg = fl(s * gamma);  a = fl(sg * rstd);  b = fl(s * beta);
//   t = fl(x - mean);  w = fma(sg, r, b);  v = fma(t, a, w);  y = round_half(relu(v)).
// The result is the unique binary16 pattern of that sequence.

void oracle_bn_apply_f32(const int32_t* shp, const uint16_t* x16, const uint16_t* gamma16,
                         const uint16_t* beta16, const uint16_t* res16, const float* mean,
                         const float* rstd, float post_scale, int relu, uint16_t* y16,
                         int swap) {
  BN d(shp);
  const int64_t M = d.M();
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t c = 0; c < d.C; ++c) {
    const float sg = post_scale * half_to_float(gamma16[c]);
    const float a = sg * rstd[c];
    const float b = post_scale * half_to_float(beta16[c]);
    for (int64_t j = 0; j < M; ++j) {
      const int64_t i = d.at(c, j);
      const float t = half_to_float(x16[i]) - mean[c];
      float v;
      if (swap) {
        v = std::fmaf(t, a, std::fmaf(sg, half_to_float(res16[i]), b));
      } else {
        v = std::fmaf(t, a, b);
        if (res16) v = v + half_to_float(res16[i]);
      }
      if (relu) v = relu_f(v);
      y16[i] = round_half((double)v);
    }
  }
}

// Backward of the forward above in float64, statistics recomputed from x:
//   mask = [y > 0] from the given forward output y (all ones when relu is off);
//   g = s * dy where mask is 1, +0 where it is 0 (the gradient reaching
//       z = gamma * xhat + beta; the ReLU's derivative is zero there, and
//       the zero is +0 like the ReLU's own output);
//   S1 = sum g;  S2 = sum g * xhat;  dbeta = S1;  dgamma = S2;
//   dx = gamma * rstd * (g - S1 / M - xhat * S2 / M);
//   dr = dy where mask is 1, +0 elsewhere (gradient to the identity shortcut,
//        if requested; ReLU passes the gradient only where its output is positive).
// With swap (u = s * (gamma * (xhat + r) + beta)): g as above;
//   dbeta = S1;  dgamma = S2 + S3 with S3 = sum g * r;  dx as above (xhat is
//   the only path from x);  dr = gamma * g (the shortcut now passes gamma).
// Each output is rounded once to binary16.  The 64-bit outputs may be NULL.

void oracle_bn_bwd(const int32_t* shp, const uint16_t* x16, const uint16_t* y16,
                   const uint16_t* dy16, const uint16_t* gamma16, float eps, float post_scale,
                   int relu, uint16_t* dx16, uint16_t* dgamma16, uint16_t* dbeta16,
                   uint16_t* dres16, double* dx64, double* dgamma64, double* dbeta64, int swap,
                   const uint16_t* res16) {
  BN d(shp);
  const int64_t M = d.M();
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t c = 0; c < d.C; ++c) {
    double sum = 0.0;
    for (int64_t j = 0; j < M; ++j) sum += half_to_double(x16[d.at(c, j)]);
    const double mu = sum / (double)M;
    double ss = 0.0;
    for (int64_t j = 0; j < M; ++j) {
      const double t = half_to_double(x16[d.at(c, j)]) - mu;
      ss += t * t;
    }
    const double rstd = 1.0 / std::sqrt(ss / (double)M + (double)eps);
    double S1 = 0.0, S2 = 0.0, S3 = 0.0;
    for (int64_t j = 0; j < M; ++j) {
      const int64_t i = d.at(c, j);
      const double mask = (!relu || half_to_double(y16[i]) > 0.0) ? 1.0 : 0.0;
      const double g = mask > 0.0 ? (double)post_scale * half_to_double(dy16[i]) : 0.0;
      const double xhat = (half_to_double(x16[i]) - mu) * rstd;
      S1 += g;
      S2 += g * xhat;
      if (swap) S3 += g * half_to_double(res16[i]);
    }
    const double gam = half_to_double(gamma16[c]);
    for (int64_t j = 0; j < M; ++j) {
      const int64_t i = d.at(c, j);
      const double mask = (!relu || half_to_double(y16[i]) > 0.0) ? 1.0 : 0.0;
      const double g = mask > 0.0 ? (double)post_scale * half_to_double(dy16[i]) : 0.0;
      const double xhat = (half_to_double(x16[i]) - mu) * rstd;
      const double v = gam * rstd * (g - S1 / (double)M - xhat * S2 / (double)M);
      if (dx64) dx64[i] = v;
      if (dx16) dx16[i] = round_half(v);
      if (dres16) {
        if (swap)
          dres16[i] = round_half(gam * g);
        else
          dres16[i] = mask > 0.0 ? dy16[i] : (uint16_t)0x0000;
      }
    }
    if (dgamma64) dgamma64[c] = S2 + S3;
    if (dbeta64) dbeta64[c] = S1;
    if (dgamma16) dgamma16[c] = round_half(S2 + S3);
    if (dbeta16) dbeta16[c] = round_half(S1);
  }
}

// ---- momentum SGD ---------------------------------------------------------
// PyTorch-style momentum SGD (the recipe of Section 5.1: dampening 0, no
// Nesterov) with FP16 weights and FP16 momentum and no master copy
// (Section 5.2):  d = g + wd * w;  m <- mu * m + d;  w <- w - lr * m.
// Declared float32 sequence (two storage points, m and w):
//   d = fma(wd, w, g);  m' = round_half(fma(mu, m, d));
//   w' = round_half(fma(-lr, m', w)).
// With a zero-initialised momentum buffer the first step gives m' = d
// rounded, the same value PyTorch stores on its first step.

void oracle_sgd_f32(uint16_t* w16, const uint16_t* g16, uint16_t* m16, int64_t n, float lr,
                    float momentum, float weight_decay) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) {
    const float w = half_to_float(w16[i]);
    const float g = half_to_float(g16[i]);
    const float m = half_to_float(m16[i]);
    const float dd = std::fmaf(weight_decay, w, g);
    const uint16_t m1 = round_half((double)std::fmaf(momentum, m, dd));
    const uint16_t w1 = round_half((double)std::fmaf(-lr, half_to_float(m1), w));
    m16[i] = m1;
    w16[i] = w1;
  }
}

// The same update with every intermediate in float64 and rounding only at
// the two storage points; used to report what the float32 sequence changes.
void oracle_sgd_f64(uint16_t* w16, const uint16_t* g16, uint16_t* m16, int64_t n, double lr,
                    double momentum, double weight_decay) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) {
    const double w = half_to_double(w16[i]);
    const double g = half_to_double(g16[i]);
    const double m = half_to_double(m16[i]);
    const uint16_t m1 = round_half(momentum * m + (g + weight_decay * w));
    const uint16_t w1 = round_half(w - lr * half_to_double(m1));
    m16[i] = m1;
    w16[i] = w1;
  }
}

}  // extern "C"

namespace {

// ---- pooling ----------------------------------------------------------------
// Geometry shp = {N, C, H, W, R, S, stride_h, stride_w, pad_h, pad_w, layout}
// (layout 0: NHWC, 1: NCHW); output P = floor((H + 2 pad_h - R) / stride_h) + 1.
//
// Max pooling (the 3x3 stride-2 pool after ResNet-50's stem): positions in the
// padding are not candidates.  The window is scanned in (r, s) order; a
// later element replaces the running maximum only if it is strictly larger,
// and the first NaN met is kept (NaN propagates; reading: ties and NaN go to
// the earliest position, so the backward has one well-defined target).
// idx (may be NULL) receives the winning tap r * S + s of each output.

struct Pool {
  int64_t N, C, H, W, R, S, sh, sw, ph, pw, P, Q;
  int layout;
  explicit Pool(const int32_t* s) {
    N = s[0]; C = s[1]; H = s[2]; W = s[3]; R = s[4]; S = s[5];
    sh = s[6]; sw = s[7]; ph = s[8]; pw = s[9]; layout = s[10];
    P = (H + 2 * ph - R) / sh + 1;
    Q = (W + 2 * pw - S) / sw + 1;
  }
  int64_t xi(int64_t n, int64_t c, int64_t h, int64_t w) const {
    return layout == 0 ? ((n * H + h) * W + w) * C + c : ((n * C + c) * H + h) * W + w;
  }
  int64_t yi(int64_t n, int64_t c, int64_t p, int64_t q) const {
    return layout == 0 ? ((n * P + p) * Q + q) * C + c : ((n * C + c) * P + p) * Q + q;
  }
  // winning tap of output (n, c, p, q), or -1 if the window has no position
  // inside the image
  int64_t argmax(const uint16_t* x16, int64_t n, int64_t c, int64_t p, int64_t q) const {
    int64_t best = -1;
    double bv = 0.0;
    for (int64_t r = 0; r < R; ++r) {
      const int64_t h = p * sh - ph + r;
      if (h < 0 || h >= H) continue;
      for (int64_t s = 0; s < S; ++s) {
        const int64_t w = q * sw - pw + s;
        if (w < 0 || w >= W) continue;
        const double v = half_to_double(x16[xi(n, c, h, w)]);
        if (best < 0 || (!std::isnan(bv) && (std::isnan(v) || v > bv))) {
          best = r * S + s;
          bv = v;
        }
      }
    }
    return best;
  }
};

}  // namespace

extern "C" {

void oracle_pool_out_dims(const int32_t* shp, int32_t* p, int32_t* q) {
  Pool d(shp);
  *p = (int32_t)d.P;
  *q = (int32_t)d.Q;
}

// y = the winning element itself (no rounding: it is already binary16).
void oracle_maxpool_fwd(const int32_t* shp, const uint16_t* x16, uint16_t* y16, uint8_t* idx) {
  Pool d(shp);
#pragma omp parallel for collapse(2) schedule(static)
  for (int64_t n = 0; n < d.N; ++n)
    for (int64_t c = 0; c < d.C; ++c)
      for (int64_t p = 0; p < d.P; ++p)
        for (int64_t q = 0; q < d.Q; ++q) {
          const int64_t t = d.argmax(x16, n, c, p, q);
          const int64_t o = d.yi(n, c, p, q);
          // a window with no position inside the image has no input; its
          // output is +0 (the ABI rejects such geometries)
          y16[o] = t < 0 ? (uint16_t)0 : x16[d.xi(n, c, p * d.sh - d.ph + t / d.S,
                                                   q * d.sw - d.pw + t % d.S)];
          if (idx) idx[o] = (uint8_t)(t < 0 ? 255 : t);
        }
}

// dx[n,c,h,w] = sum of dy over the outputs whose winning position is (h, w),
// summed in float64 (exact: at most R*S binary16 terms here) and rounded
// once; +0 where no output selects the position.
void oracle_maxpool_bwd(const int32_t* shp, const uint16_t* x16, const uint16_t* dy16,
                        uint16_t* dx16) {
  Pool d(shp);
  const int64_t nx = d.N * d.C * d.H * d.W;
  std::vector<double> acc((size_t)nx, 0.0);
#pragma omp parallel for collapse(2) schedule(static)
  for (int64_t n = 0; n < d.N; ++n)
    for (int64_t c = 0; c < d.C; ++c)
      for (int64_t p = 0; p < d.P; ++p)
        for (int64_t q = 0; q < d.Q; ++q) {
          const int64_t t = d.argmax(x16, n, c, p, q);
          if (t < 0) continue;
          const int64_t h = p * d.sh - d.ph + t / d.S, w = q * d.sw - d.pw + t % d.S;
          acc[(size_t)d.xi(n, c, h, w)] += half_to_double(dy16[d.yi(n, c, p, q)]);
        }
  for (int64_t i = 0; i < nx; ++i) dx16[i] = round_half(acc[(size_t)i]);
}

// Global average pooling (ResNet-50's pool before the classifier), shp as for
// pooling with R = H, S = W: y[n,c] = (sum over the H x W grid of x) / (H W),
// with the sum exact in float64, one float64 division, one rounding.
// y is [N, C] (the NHWC and NCHW orders coincide for a 1 x 1 grid).
void oracle_avgpool_fwd(const int32_t* shp, const uint16_t* x16, double* y64, uint16_t* y16) {
  Pool d(shp);
#pragma omp parallel for collapse(2) schedule(static)
  for (int64_t n = 0; n < d.N; ++n)
    for (int64_t c = 0; c < d.C; ++c) {
      double sum = 0.0;
      for (int64_t h = 0; h < d.H; ++h)
        for (int64_t w = 0; w < d.W; ++w) sum += half_to_double(x16[d.xi(n, c, h, w)]);
      const double v = sum / (double)(d.H * d.W);
      if (y64) y64[n * d.C + c] = v;
      if (y16) y16[n * d.C + c] = round_half(v);
    }
}

// Its adjoint: every position of the grid receives dy[n,c] / (H W), rounded once.
void oracle_avgpool_bwd(const int32_t* shp, const uint16_t* dy16, uint16_t* dx16) {
  Pool d(shp);
#pragma omp parallel for collapse(2) schedule(static)
  for (int64_t n = 0; n < d.N; ++n)
    for (int64_t c = 0; c < d.C; ++c) {
      const uint16_t v = round_half(half_to_double(dy16[n * d.C + c]) / (double)(d.H * d.W));
      for (int64_t h = 0; h < d.H; ++h)
        for (int64_t w = 0; w < d.W; ++w) dx16[d.xi(n, c, h, w)] = v;
    }
}

// ---- classifier bias and softmax cross-entropy -------------------------------
// z[N, K]: the classifier's matrix product (a 1x1 convolution, stored in
// binary16); b[K]: its bias; labels[N] in [0, K).
//   l = round_half(z + b)                     (the logits, a binary16 tensor)
//   loss_n = log(sum_j exp(l_nj - m)) + (m - l_n,label), m = max_j l_nj (float64)
//   mean loss = (1/N) sum_n loss_n            (average over the local batch)
//   dl_nj = (softmax(l_n)_j - [j == label]) / N, rounded once   (= dz)
//   db_j = sum_n dl_nj over the stored dl, exact in float64, rounded once.
// loss_rows (may be NULL) receives loss_n; loss_mean (may be NULL) the mean.
void oracle_softmax_ce(int64_t N, int64_t K, const uint16_t* z16, const uint16_t* b16,
                       const int32_t* labels, double* loss_rows, double* loss_mean,
                       uint16_t* dz16, uint16_t* db16) {
  std::vector<double> rows((size_t)N);
#pragma omp parallel for schedule(static)
  for (int64_t n = 0; n < N; ++n) {
    std::vector<double> l((size_t)K);
    double m = -INFINITY;
    for (int64_t j = 0; j < K; ++j) {
      l[(size_t)j] = half_to_double(round_half(half_to_double(z16[n * K + j]) +
                                               half_to_double(b16[j])));
      if (l[(size_t)j] > m) m = l[(size_t)j];
    }
    double s = 0.0;
    for (int64_t j = 0; j < K; ++j) s += std::exp(l[(size_t)j] - m);
    const int64_t y = labels[n];
    rows[(size_t)n] = std::log(s) + (m - l[(size_t)y]);  // the difference is exact
    for (int64_t j = 0; j < K; ++j) {
      const double pj = std::exp(l[(size_t)j] - m) / s;
      dz16[n * K + j] = round_half((pj - (j == y ? 1.0 : 0.0)) / (double)N);
    }
  }
  double tot = 0.0;
  for (int64_t n = 0; n < N; ++n) {
    if (loss_rows) loss_rows[n] = rows[(size_t)n];
    tot += rows[(size_t)n];
  }
  if (loss_mean) *loss_mean = tot / (double)N;
  if (db16)
    for (int64_t j = 0; j < K; ++j) {
      double a = 0.0;
      for (int64_t n = 0; n < N; ++n) a += half_to_double(dz16[n * K + j]);
      db16[j] = round_half(a);
    }
}

}  // extern "C"

// ===========================================================================
// Strict binary16 arithmetic (the literal reading of Section 5.2: all
// arithmetic in FP16, not only storage).  Used to measure what the float32
// accumulators of the default path buy; not the product's default.
// ===========================================================================

namespace {

// binary16 round-to-nearest-even of the exact value s + err, where s is a
// double and err the exact error of the double addition that produced s
// (TwoSum).  |err| is far below half a binary16 ulp, so it only decides the
// result when s lies exactly halfway between two binary16 values.
uint16_t round_half_exact(double s, double err) {
  const uint16_t r = round_half(s);
  if (err == 0.0 || std::isnan(s) || std::isinf(s)) return r;
  const bool neg = std::signbit(s);
  const double a = std::fabs(s);
  const double e = neg ? -err : err;
  const uint16_t ra = (uint16_t)(r & 0x7FFF);
  const double v = half_to_double(ra);
  if (v == a) return r;
  double lo, hi;
  uint16_t lob, hib;
  if (v < a) {
    lob = ra; lo = v;
    hib = (uint16_t)(ra + 1);
    hi = ra == 0x7BFF ? 65536.0 : half_to_double(hib);  // past the largest finite: the overflow midpoint
  } else {
    hib = ra; hi = std::isinf(v) ? 65536.0 : v;
    lob = (uint16_t)(ra - 1); lo = half_to_double(lob);
  }
  if (a - lo != hi - a) return r;  // not a midpoint: the double already decides
  const uint16_t pick = e > 0 ? hib : lob;
  return (uint16_t)(pick | (neg ? 0x8000 : 0));
}

// One binary16 fused multiply-add: round(a * b + c) with a single rounding.
// The product of two binary16 values is exact in double; the sum's exact
// error comes from TwoSum (Knuth).
uint16_t fma_half(uint16_t a16, uint16_t b16, uint16_t c16) {
  const double a = half_to_double(a16), b = half_to_double(b16), c = half_to_double(c16);
  const double p = a * b;
  const double s = p + c;
  if (std::isnan(s) || std::isinf(s) || std::isinf(p)) return round_half(s);
  const double bb = s - p;
  const double err = (p - (s - bb)) + (c - bb);
  return round_half_exact(s, err);
}

}  // namespace

extern "C" {

uint16_t oracle_fma16(uint16_t a, uint16_t b, uint16_t c) { return fma_half(a, b, c); }

void oracle_fma16_array(const uint16_t* a, const uint16_t* b, const uint16_t* c, uint16_t* out,
                        int64_t n) {
  for (int64_t i = 0; i < n; ++i) out[i] = fma_half(a[i], b[i], c[i]);
}

// SGD with every operation in binary16: the scalars are the binary16
// roundings of the float32 weight decay, momentum and -lr, and
//   d = fma16(wd, w, g);  m' = fma16(mu, m, d);  w' = fma16(-lr, m', w).
void oracle_sgd_f16(uint16_t* w16, const uint16_t* g16, uint16_t* m16, int64_t n, float lr,
                    float momentum, float weight_decay) {
  const uint16_t lam = round_half((double)weight_decay), mu = round_half((double)momentum),
                 nlr = round_half(-(double)lr);
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) {
    const uint16_t d = fma_half(lam, w16[i], g16[i]);
    const uint16_t m1 = fma_half(mu, m16[i], d);
    const uint16_t w1 = fma_half(nlr, m1, w16[i]);
    m16[i] = m1;
    w16[i] = w1;
  }
}

// Convolutions with every operation in binary16 (Section 5.2 read
// literally: all arithmetic in FP16).  Each output is a binary16
// accumulator that starts at +0 and takes its terms one at a time, each as
// one binary16 fused multiply-add, acc = round(a * b + acc) (one rounding of
// the exact value).  The reduction order is declared per pass below, in the
// logical indices of the convolution's definition; a tap whose position lies
// outside the input image (forward, weight gradient) or outside the output
// grid (data gradient) is not a term.  Any layout.

}  // extern "C"

namespace {

// y[n,k,p,q]: taps (r, s) in row-major order, channels c ascending within a tap.
uint16_t fwd_chain(const Conv& d, const uint16_t* x16, const uint16_t* w16, int64_t i) {
  int64_t n, k, p, q;
  d.y_coords(i, &n, &k, &p, &q);
  uint16_t acc = 0x0000;
  for (int64_t r = 0; r < d.R; ++r)
    for (int64_t s = 0; s < d.S; ++s) {
      const int64_t h = p * d.sh - d.ph + r, ww = q * d.sw - d.pw + s;
      if (h < 0 || h >= d.H || ww < 0 || ww >= d.W) continue;
      for (int64_t c = 0; c < d.C; ++c)
        acc = fma_half(x16[d.xi(n, c, h, ww)], w16[d.wi(k, c, r, s)], acc);
    }
  return acc;
}

// dx[n,c,h,w]: the taps (r, s) in row-major order whose output position
// p = (h + pad_h - r) / stride_h, q = (w + pad_w - s) / stride_w is a whole
// grid point inside P x Q, and within a tap the output channels k ascending.
uint16_t dgrad_chain(const Conv& d, const uint16_t* dy16, const uint16_t* w16, int64_t i) {
  int64_t n, c, h, ww;
  d.x_coords(i, &n, &c, &h, &ww);
  uint16_t acc = 0x0000;
  for (int64_t r = 0; r < d.R; ++r)
    for (int64_t s = 0; s < d.S; ++s) {
      const int64_t ph = h + d.ph - r, pw = ww + d.pw - s;
      if (ph < 0 || pw < 0 || ph % d.sh != 0 || pw % d.sw != 0) continue;
      const int64_t p = ph / d.sh, q = pw / d.sw;
      if (p >= d.P || q >= d.Q) continue;
      for (int64_t k = 0; k < d.K; ++k)
        acc = fma_half(dy16[d.yi(n, k, p, q)], w16[d.wi(k, c, r, s)], acc);
    }
  return acc;
}

// dW[k,c,r,s]: the output pixels (n, p, q) in order (n slowest, q fastest).
uint16_t wgrad_chain(const Conv& d, const uint16_t* x16, const uint16_t* dy16, int64_t i) {
  int64_t k, c, r, s;
  d.w_coords(i, &k, &c, &r, &s);
  uint16_t acc = 0x0000;
  for (int64_t n = 0; n < d.N; ++n)
    for (int64_t p = 0; p < d.P; ++p)
      for (int64_t q = 0; q < d.Q; ++q) {
        const int64_t h = p * d.sh - d.ph + r, ww = q * d.sw - d.pw + s;
        if (h < 0 || h >= d.H || ww < 0 || ww >= d.W) continue;
        acc = fma_half(dy16[d.yi(n, k, p, q)], x16[d.xi(n, c, h, ww)], acc);
      }
  return acc;
}

}  // namespace

extern "C" {

void oracle_conv_fwd_f16acc(const int32_t* shp, const uint16_t* x16, const uint16_t* w16,
                            uint16_t* y16) {
  const Conv d(shp);
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < d.y_size(); ++i) y16[i] = fwd_chain(d, x16, w16, i);
}

void oracle_conv_dgrad_f16acc(const int32_t* shp, const uint16_t* dy16, const uint16_t* w16,
                              uint16_t* dx16) {
  const Conv d(shp);
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < d.x_size(); ++i) dx16[i] = dgrad_chain(d, dy16, w16, i);
}

void oracle_conv_wgrad_f16acc(const int32_t* shp, const uint16_t* x16, const uint16_t* dy16,
                              uint16_t* dw16) {
  const Conv d(shp);
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < d.w_size(); ++i) dw16[i] = wgrad_chain(d, x16, dy16, i);
}

// The same chains at chosen flat output indices only (out[j] for idx[j]).
void oracle_conv_fwd_f16acc_at(const int32_t* shp, const uint16_t* x16, const uint16_t* w16,
                               const int64_t* idx, int64_t n, uint16_t* out) {
  const Conv d(shp);
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t j = 0; j < n; ++j) out[j] = fwd_chain(d, x16, w16, idx[j]);
}

void oracle_conv_dgrad_f16acc_at(const int32_t* shp, const uint16_t* dy16, const uint16_t* w16,
                                 const int64_t* idx, int64_t n, uint16_t* out) {
  const Conv d(shp);
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t j = 0; j < n; ++j) out[j] = dgrad_chain(d, dy16, w16, idx[j]);
}

void oracle_conv_wgrad_f16acc_at(const int32_t* shp, const uint16_t* x16, const uint16_t* dy16,
                                 const int64_t* idx, int64_t n, uint16_t* out) {
  const Conv d(shp);
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t j = 0; j < n; ++j) out[j] = wgrad_chain(d, x16, dy16, idx[j]);
}

}  // extern "C"
