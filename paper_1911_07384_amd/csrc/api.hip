// C ABI of fp16train: argument validation, workspace planning and dispatch
// to the HIP kernels.  Nothing here allocates device memory; every call is
// enqueued on the caller's stream.

#include "../../include/fp16train.h"
#include "kernels.hpp"

#include <stdint.h>

#include <vector>

using namespace fp16k;

namespace {

constexpr int64_t kMaxElems = (int64_t)1 << 30;  // buffer-load offsets are 32-bit byte offsets

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

bool overlap(const void* a, size_t na, const void* b, size_t nb) {
  if (!a || !b || na == 0 || nb == 0) return false;
  const uintptr_t pa = (uintptr_t)a, pb = (uintptr_t)b;
  return pa < pb + nb && pb < pa + na;
}

int round8(int v) { return (v + 7) / 8 * 8; }
size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

struct ConvDims {
  int N, C, H, W, K, R, S, sh, sw, ph, pw, P, Q, layout, Cp, Kp, accum;
  int64_t x_elems, y_elems, w_elems;
};

fp16_status check_conv(const fp16_conv_desc* d, ConvDims* o) {
  if (!d) return FP16_ERR_NULL;
  if (d->layout != FP16_NHWC && d->layout != FP16_NCHW) return FP16_ERR_LAYOUT;
  if (d->n < 1 || d->c < 1 || d->h < 1 || d->w < 1 || d->k < 1 || d->r < 1 || d->s < 1 ||
      d->stride_h < 1 || d->stride_w < 1 || d->pad_h < 0 || d->pad_w < 0)
    return FP16_ERR_SHAPE;
  if (d->r > 64 || d->s > 64 || d->stride_h > 64 || d->stride_w > 64 || d->pad_h > 64 ||
      d->pad_w > 64 || d->c > 65535 || d->k > 65535 || d->h > 65535 || d->w > 65535)
    return FP16_ERR_SHAPE;
  if (d->h + 2 * d->pad_h < d->r || d->w + 2 * d->pad_w < d->s) return FP16_ERR_SHAPE;
  if (d->accum != 0 && d->accum != 1) return FP16_ERR_UNSUPPORTED;
  if (d->accum == 1 && d->layout != FP16_NHWC) return FP16_ERR_UNSUPPORTED;
  o->accum = d->accum;
  o->N = d->n; o->C = d->c; o->H = d->h; o->W = d->w; o->K = d->k; o->R = d->r; o->S = d->s;
  o->sh = d->stride_h; o->sw = d->stride_w; o->ph = d->pad_h; o->pw = d->pad_w;
  o->layout = d->layout;
  o->P = (o->H + 2 * o->ph - o->R) / o->sh + 1;
  o->Q = (o->W + 2 * o->pw - o->S) / o->sw + 1;
  o->Cp = round8(o->C);
  o->Kp = round8(o->K);
  o->x_elems = (int64_t)o->N * o->C * o->H * o->W;
  o->y_elems = (int64_t)o->N * o->K * o->P * o->Q;
  o->w_elems = (int64_t)o->K * o->C * o->R * o->S;
  const int64_t xp = (int64_t)o->N * o->Cp * o->H * o->W;
  const int64_t yp = (int64_t)o->N * o->Kp * o->P * o->Q;
  const int64_t wp = (int64_t)o->Kp * o->Cp * o->R * o->S;
  if (xp >= kMaxElems || yp >= kMaxElems || wp >= kMaxElems) return FP16_ERR_SHAPE;
  return FP16_OK;
}

// The ResNet stem's weight gradient (3 channels, 7x7, stride 2, pad 3, even
// image sides) runs as a 4x4 stride-1 convolution over the 2x2 space-to-depth
// image: 16 channels instead of 3 padded to 8, and one 256-column filter tile
// instead of two for 392 columns (half the matrix-core work).
bool stem_s2d(const ConvDims& d) {
  return d.layout == FP16_NHWC && d.C == 3 && d.R == 7 && d.S == 7 && d.sh == 2 && d.sw == 2 &&
         d.ph == 3 && d.pw == 3 && d.H % 2 == 0 && d.W % 2 == 0 && d.P == d.H / 2 &&
         d.Q == d.W / 2 && !d.accum && d.K % 64 == 0 && d.Kp == d.K;
}

// Workspace regions of one convolution pass (byte offsets, 256-aligned).
struct ConvWs {
  size_t x = 0, w = 0, y = 0, wf = 0, part = 0, total = 0;
  bool need_x = false, need_w = false, need_y = false;
  int splits = 0, pps = 0;
};

// (wg: the weight gradient's workgroup target, 0 for kWgradWorkgroups)
ConvWs conv_ws(const ConvDims& d, int pass, int wg = 0) {
  const int target = wg > 0 ? wg : kWgradWorkgroups;
  ConvWs L;
  if (d.accum) return L;  // the binary16 chains read and write the caller's tensors only
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off += align256(bytes);
    return at;
  };
  const bool nchw = d.layout == FP16_NCHW;
  // a 1x1 filter over 1x1 images (a classifier) is a dense GEMM; with few
  // rows its reduction is split (float32 partials)
  const bool dense = !nchw && d.H == 1 && d.W == 1 && d.R == 1 && d.S == 1 && d.ph == 0 &&
                     d.pw == 0 && d.P == 1 && d.Q == 1;
  if (pass == FP16_PASS_FWD && dense && d.Cp == d.C) {
    L.splits = dense_gemm_splits(d.N, d.Cp, d.K);
    if (L.splits > 1) L.part = take((size_t)L.splits * d.N * d.K * 4);
  } else if (pass == FP16_PASS_DGRAD && dense && d.Kp == d.K) {
    L.splits = dense_gemm_splits(d.N, d.Kp, d.C);
    if (L.splits > 1) L.part = take((size_t)L.splits * d.N * d.C * 4);
  }
  if (pass == FP16_PASS_FWD) {
    if (nchw || d.Cp != d.C) {
      L.need_x = L.need_w = true;
      L.x = take((size_t)d.N * d.H * d.W * d.Cp * 2);
      L.w = take((size_t)d.K * d.R * d.S * d.Cp * 2);
    }
    if (nchw) {
      L.need_y = true;
      L.y = take((size_t)d.N * d.P * d.Q * d.K * 2);
    }
  } else if (pass == FP16_PASS_DGRAD) {
    if (nchw || d.Kp != d.K) {  // dy as NHWC with Kp channels
      L.need_y = true;
      L.y = take((size_t)d.N * d.P * d.Q * d.Kp * 2);
    }
    if (nchw) {  // filter KCRS -> KRSC, and dx staged as NHWC
      L.need_w = true;
      L.w = take((size_t)d.K * d.R * d.S * d.C * 2);
      L.need_x = true;
      L.x = take((size_t)d.N * d.H * d.W * d.C * 2);
    }
    L.wf = take((size_t)d.C * d.R * d.S * d.Kp * 2);
  } else if (stem_s2d(d)) {
    L.need_x = true;
    L.x = take((size_t)d.N * d.P * d.Q * 16 * 2);
    wgrad_plan(d.Kp, 16, 4, 4, (int64_t)d.N * d.P * d.Q, target, &L.splits, &L.pps);
    L.part = take((size_t)L.splits * d.Kp * 256 * 4);
  } else {
    if (nchw || d.Cp != d.C) {
      L.need_x = true;
      L.x = take((size_t)d.N * d.H * d.W * d.Cp * 2);
    }
    if (nchw || d.Kp != d.K) {
      L.need_y = true;
      L.y = take((size_t)d.N * d.P * d.Q * d.Kp * 2);
    }
    wgrad_plan(d.Kp, d.Cp, d.R, d.S, (int64_t)d.N * d.P * d.Q, target, &L.splits, &L.pps);
    L.part = take((size_t)L.splits * d.Kp * d.R * d.S * d.Cp * 4);
  }
  L.total = off;
  return L;
}

// Arguments of the stem kernel: the unpadded NHWC input and KRSC filter.
IgemmArgs stem_args(const ConvDims& d, const h16* x, const h16* w, h16* y) {
  IgemmArgs a{};
  a.act = x; a.N = d.N; a.Hi = d.H; a.Wi = d.W; a.Ci = d.C;
  a.stride_h = d.sh; a.stride_w = d.sw;
  a.Co = d.K; a.out = y; a.OH = d.P; a.OW = d.Q; a.ldo = d.K; a.os_h = 1; a.os_w = 1;
  a.nphase = 1;
  a.ph[0] = IgemmPhase{w, d.R * d.S * d.C, d.R, d.S, d.ph, d.pw, d.P, d.Q, 0, 0};
  return a;
}

ConvChainArgs chain_args(const ConvDims& d) {
  return ConvChainArgs{d.N, d.C, d.H, d.W, d.K, d.R, d.S, d.sh, d.sw, d.ph, d.pw, d.P, d.Q};
}

fp16_status hip_status(hipError_t e) { return e == hipSuccess ? FP16_OK : FP16_ERR_HIP; }

#define TRY(expr)                                  \
  do {                                             \
    const hipError_t e_ = (expr);                  \
    if (e_ != hipSuccess) return FP16_ERR_HIP;     \
  } while (0)

fp16_status check_ws(const ConvWs& L, const void* ws, size_t ws_bytes) {
  if (L.total == 0) return FP16_OK;
  if (!ws || ws_bytes < L.total) return FP16_ERR_WORKSPACE;
  if (!aligned16(ws)) return FP16_ERR_MISALIGNED;
  return FP16_OK;
}

h16* wsp(void* ws, size_t off) { return reinterpret_cast<h16*>(static_cast<char*>(ws) + off); }

}  // namespace

extern "C" {

const char* fp16_status_string(fp16_status s) {
  switch (s) {
    case FP16_OK: return "ok";
    case FP16_ERR_NULL: return "null pointer";
    case FP16_ERR_SHAPE: return "invalid shape";
    case FP16_ERR_LAYOUT: return "invalid layout";
    case FP16_ERR_MISALIGNED: return "pointer not 16-byte aligned";
    case FP16_ERR_ALIASING: return "output overlaps an input";
    case FP16_ERR_WORKSPACE: return "workspace missing or too small";
    case FP16_ERR_UNSUPPORTED: return "unsupported";
    case FP16_ERR_HIP: return "HIP runtime error";
  }
  return "unknown status";
}

const char* fp16_version(void) { return "fp16train 0.1"; }

fp16_status fp16_conv_out_dims(const fp16_conv_desc* desc, int32_t* p, int32_t* q) {
  ConvDims d;
  const fp16_status s = check_conv(desc, &d);
  if (s != FP16_OK) return s;
  if (!p || !q) return FP16_ERR_NULL;
  *p = d.P;
  *q = d.Q;
  return FP16_OK;
}

size_t fp16_conv_workspace_bytes(const fp16_conv_desc* desc, int32_t pass) {
  ConvDims d;
  if (check_conv(desc, &d) != FP16_OK) return 0;
  if (pass < FP16_PASS_FWD || pass > FP16_PASS_WGRAD) return 0;
  return conv_ws(d, pass).total;
}

fp16_status fp16_conv_fwd(const fp16_conv_desc* desc, const fp16_t* x, const fp16_t* w, fp16_t* y,
                          void* ws, size_t ws_bytes, fp16_stream_t stream) {
  ConvDims d;
  fp16_status s = check_conv(desc, &d);
  if (s != FP16_OK) return s;
  if (!x || !w || !y) return FP16_ERR_NULL;
  if (!aligned16(x) || !aligned16(w) || !aligned16(y)) return FP16_ERR_MISALIGNED;
  const ConvWs L = conv_ws(d, FP16_PASS_FWD);
  if ((s = check_ws(L, ws, ws_bytes)) != FP16_OK) return s;
  const size_t yb = (size_t)d.y_elems * 2;
  if (overlap(y, yb, x, (size_t)d.x_elems * 2) || overlap(y, yb, w, (size_t)d.w_elems * 2) ||
      overlap(y, yb, ws, L.total))
    return FP16_ERR_ALIASING;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const h16* xe = reinterpret_cast<const h16*>(x);
  const h16* we = reinterpret_cast<const h16*>(w);
  h16* ye = reinterpret_cast<h16*>(y);
  if (d.accum) return hip_status(launch_conv_chain(chain_args(d), 0, xe, we, ye, st));
  if (d.layout == FP16_NHWC) {
    // the ResNet stem reads the unpadded image on its own kernel
    const IgemmArgs sa = stem_args(d, xe, we, ye);
    if (stem_conv_ok(sa)) return hip_status(launch_stem(sa, st));
  }
  if (d.layout == FP16_NCHW) {
    TRY(launch_nchw_to_nhwc(xe, wsp(ws, L.x), d.N, d.C, d.H * d.W, d.Cp, st));
    TRY(launch_nchw_to_nhwc(we, wsp(ws, L.w), d.K, d.C, d.R * d.S, d.Cp, st));
    xe = wsp(ws, L.x);
    we = wsp(ws, L.w);
    ye = wsp(ws, L.y);
  } else if (d.Cp != d.C) {
    TRY(launch_pad_channels(xe, wsp(ws, L.x), (int64_t)d.N * d.H * d.W, d.C, d.Cp, st));
    TRY(launch_pad_channels(we, wsp(ws, L.w), (int64_t)d.K * d.R * d.S, d.C, d.Cp, st));
    xe = wsp(ws, L.x);
    we = wsp(ws, L.w);
  }
  IgemmArgs a{};
  a.act = xe; a.N = d.N; a.Hi = d.H; a.Wi = d.W; a.Ci = d.Cp;
  a.stride_h = d.sh; a.stride_w = d.sw;
  a.Co = d.K; a.out = ye; a.OH = d.P; a.OW = d.Q; a.ldo = d.K; a.os_h = 1; a.os_w = 1;
  a.nphase = 1;
  a.ph[0] = IgemmPhase{we, d.R * d.S * d.Cp, d.R, d.S, d.ph, d.pw, d.P, d.Q, 0, 0};
  if (L.splits > 1) {  // a dense GEMM with its reduction split
    a.part = reinterpret_cast<float*>(static_cast<char*>(ws) + L.part);
    a.splits = L.splits;
  }
  TRY(launch_igemm(a, st));
  if (d.layout == FP16_NCHW) TRY(launch_nhwc_to_nchw(ye, reinterpret_cast<h16*>(y), d.N, d.K,
                                                     d.P * d.Q, d.K, st));
  return FP16_OK;
}

}  // extern "C"

// Bytes of the rearranged data-gradient filter (every stride phase's taps
// together cover the R x S taps once).
static size_t dgrad_filter_bytes(const ConvDims& d) { return (size_t)d.C * d.R * d.S * d.Kp * 2; }

// Data gradient; with wf_given the filter is already rearranged (w is then
// the rearranged filter, fp16_conv_dgrad_filter_bytes long, NHWC only); with
// amask the addend is taken under that ReLU mask (NHWC, C % 8 == 0); with
// astride > 1 the addend holds every astride-th row and column only (NHWC).
static fp16_status conv_dgrad_impl(const fp16_conv_desc* desc, const fp16_t* dy, const fp16_t* w,
                                   const fp16_t* addend, fp16_t* dx, void* ws, size_t ws_bytes,
                                   fp16_stream_t stream, bool wf_given = false,
                                   const uint8_t* amask = nullptr, int astride = 1) {
  ConvDims d;
  fp16_status s = check_conv(desc, &d);
  if (s != FP16_OK) return s;
  if (!dy || !w || !dx) return FP16_ERR_NULL;
  if (astride < 1 || astride > 16) return FP16_ERR_SHAPE;
  if (wf_given && d.layout != FP16_NHWC) return FP16_ERR_UNSUPPORTED;
  if ((amask || astride > 1) && !addend) return FP16_ERR_NULL;
  if ((amask || astride > 1) && (d.layout != FP16_NHWC || d.accum)) return FP16_ERR_UNSUPPORTED;
  if (amask && d.C % 8 != 0) return FP16_ERR_UNSUPPORTED;
  // the binary16 chains: the plain data gradient from the filter only
  if (d.accum && (wf_given || addend)) return FP16_ERR_UNSUPPORTED;
  if (!aligned16(dy) || !aligned16(w) || !aligned16(dx) || (addend && !aligned16(addend)))
    return FP16_ERR_MISALIGNED;
  const ConvWs L = conv_ws(d, FP16_PASS_DGRAD);
  if ((s = check_ws(L, ws, ws_bytes)) != FP16_OK) return s;
  const size_t xb = (size_t)d.x_elems * 2;
  const size_t wb = wf_given ? dgrad_filter_bytes(d) : (size_t)d.w_elems * 2;
  // the addend's bytes: dx's, or those of the subsampled grid
  const size_t ab = astride > 1 ? (size_t)d.N * ((d.H + astride - 1) / astride) *
                                      ((d.W + astride - 1) / astride) * d.C * 2
                                : xb;
  if (astride > 1 && addend == dx) return FP16_ERR_ALIASING;
  if (overlap(dx, xb, dy, (size_t)d.y_elems * 2) || overlap(dx, xb, w, wb) ||
      overlap(dx, xb, ws, L.total) || (addend && addend != dx && overlap(dx, xb, addend, ab)) ||
      (addend && overlap(addend, ab, ws, L.total)) ||
      (amask && (overlap(amask, ab / 16, dx, xb) || overlap(amask, ab / 16, ws, L.total))))
    return FP16_ERR_ALIASING;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const h16* dye = reinterpret_cast<const h16*>(dy);
  const h16* wk = reinterpret_cast<const h16*>(w);
  h16* dxe = reinterpret_cast<h16*>(dx);
  if (d.accum) return hip_status(launch_conv_chain(chain_args(d), 1, dye, wk, dxe, st));
  if (d.layout == FP16_NCHW) {
    TRY(launch_nchw_to_nhwc(dye, wsp(ws, L.y), d.N, d.K, d.P * d.Q, d.Kp, st));
    TRY(launch_nchw_to_nhwc(wk, wsp(ws, L.w), d.K, d.C, d.R * d.S, d.C, st));
    dye = wsp(ws, L.y);
    wk = wsp(ws, L.w);
    dxe = wsp(ws, L.x);
    if (addend) {  // stage the addend as NHWC in the dx buffer and accumulate in place
      TRY(launch_nchw_to_nhwc(reinterpret_cast<const h16*>(addend), dxe, d.N, d.C, d.H * d.W, d.C,
                              st));
    }
  } else if (d.Kp != d.K) {
    TRY(launch_pad_channels(dye, wsp(ws, L.y), (int64_t)d.N * d.P * d.Q, d.K, d.Kp, st));
    dye = wsp(ws, L.y);
  }
  const h16* wf = wk;
  if (!wf_given) {
    h16* wt = wsp(ws, L.wf);
    TRY(launch_dgrad_filter(wk, wt, d.K, d.C, d.R, d.S, d.C, d.Kp, d.sh, d.sw, d.ph, d.pw, st));
    wf = wt;
  }
  IgemmArgs a{};
  a.act = dye; a.N = d.N; a.Hi = d.P; a.Wi = d.Q; a.Ci = d.Kp;
  a.stride_h = 1; a.stride_w = 1;
  a.Co = d.C; a.out = dxe; a.OH = d.H; a.OW = d.W; a.ldo = d.C; a.os_h = d.sh; a.os_w = d.sw;
  a.addend = addend ? (d.layout == FP16_NCHW ? dxe : reinterpret_cast<const h16*>(addend)) : nullptr;
  a.amask = amask;
  a.astride = astride;
  if (L.splits > 1 && !amask && astride == 1) {  // a dense GEMM with its reduction split
    a.part = reinterpret_cast<float*>(static_cast<char*>(ws) + L.part);
    a.splits = L.splits;
  }
  a.nphase = 0;
  int64_t off = 0;
  for (int ph = 0; ph < d.sh; ++ph) {
    for (int pw = 0; pw < d.sw; ++pw) {
      const DgradPhase g = dgrad_phase(ph, pw, d.H, d.W, d.R, d.S, d.sh, d.sw, d.ph, d.pw);
      if (g.Hph > 0 && g.Wph > 0) {
        a.ph[a.nphase++] = IgemmPhase{wf + off, g.ntr * g.nts * d.Kp, g.ntr, g.nts, g.pad_h,
                                      g.pad_w, g.Hph, g.Wph, ph, pw};
        if (a.nphase == 4) {
          TRY(launch_igemm(a, st));
          a.nphase = 0;
        }
      }
      off += (int64_t)d.C * g.ntr * g.nts * d.Kp;
    }
  }
  if (a.nphase > 0) TRY(launch_igemm(a, st));
  if (d.layout == FP16_NCHW)
    TRY(launch_nhwc_to_nchw(dxe, reinterpret_cast<h16*>(dx), d.N, d.C, d.H * d.W, d.C, st));
  return FP16_OK;
}

extern "C" {

fp16_status fp16_conv_dgrad(const fp16_conv_desc* desc, const fp16_t* dy, const fp16_t* w,
                            fp16_t* dx, void* ws, size_t ws_bytes, fp16_stream_t stream) {
  return conv_dgrad_impl(desc, dy, w, nullptr, dx, ws, ws_bytes, stream);
}

fp16_status fp16_conv_dgrad_add(const fp16_conv_desc* desc, const fp16_t* dy, const fp16_t* w,
                                const fp16_t* addend, fp16_t* dx, void* ws, size_t ws_bytes,
                                fp16_stream_t stream) {
  if (!addend) return FP16_ERR_NULL;
  return conv_dgrad_impl(desc, dy, w, addend, dx, ws, ws_bytes, stream);
}

size_t fp16_conv_dgrad_filter_bytes(const fp16_conv_desc* desc) {
  ConvDims d;
  if (check_conv(desc, &d) != FP16_OK || d.layout != FP16_NHWC) return 0;
  return dgrad_filter_bytes(d);
}

fp16_status fp16_conv_dgrad_filter(const fp16_conv_desc* desc, const fp16_t* w, fp16_t* wf,
                                   fp16_stream_t stream) {
  ConvDims d;
  fp16_status s = check_conv(desc, &d);
  if (s != FP16_OK) return s;
  if (d.layout != FP16_NHWC) return FP16_ERR_UNSUPPORTED;
  if (!w || !wf) return FP16_ERR_NULL;
  if (!aligned16(w) || !aligned16(wf)) return FP16_ERR_MISALIGNED;
  if (overlap(wf, dgrad_filter_bytes(d), w, (size_t)d.w_elems * 2)) return FP16_ERR_ALIASING;
  return hip_status(launch_dgrad_filter(reinterpret_cast<const h16*>(w), reinterpret_cast<h16*>(wf),
                                        d.K, d.C, d.R, d.S, d.C, d.Kp, d.sh, d.sw, d.ph, d.pw,
                                        static_cast<hipStream_t>(stream)));
}

fp16_status fp16_conv_dgrad_filters(int32_t count, const fp16_conv_desc* descs,
                                    const fp16_t* const* w, fp16_t* const* wf,
                                    fp16_stream_t stream) {
  if (count == 0) return FP16_OK;
  if (count < 0 || count > FP16_DGRAD_FILTERS_MAX) return FP16_ERR_SHAPE;
  if (!descs || !w || !wf) return FP16_ERR_NULL;
  std::vector<DgradFiltJob> jobs((size_t)count);
  std::vector<size_t> wb((size_t)count), fb((size_t)count);
  for (int i = 0; i < count; ++i) {
    ConvDims d;
    const fp16_status s = check_conv(&descs[i], &d);
    if (s != FP16_OK) return s;
    if (d.layout != FP16_NHWC) return FP16_ERR_UNSUPPORTED;
    if (!w[i] || !wf[i]) return FP16_ERR_NULL;
    if (!aligned16(w[i]) || !aligned16(wf[i])) return FP16_ERR_MISALIGNED;
    wb[i] = (size_t)d.w_elems * 2;
    fb[i] = dgrad_filter_bytes(d);
    DgradFiltJob& J = jobs[(size_t)i];
    J.w = reinterpret_cast<const h16*>(w[i]);
    J.dst = reinterpret_cast<h16*>(wf[i]);
    J.K = d.K;
    J.C = d.C;
    J.R = d.R;
    J.S = d.S;
    J.Kp = d.Kp;
    J.sh = d.sh;
    J.sw = d.sw;
    J.pad_h = d.ph;
    J.pad_w = d.pw;
    J.blk0 = 0;
  }
  // every output apart from every filter and every other output
  for (int i = 0; i < count; ++i)
    for (int j = 0; j < count; ++j) {
      if (overlap(wf[i], fb[i], w[j], wb[j])) return FP16_ERR_ALIASING;
      if (j != i && overlap(wf[i], fb[i], wf[j], fb[j])) return FP16_ERR_ALIASING;
    }
  return hip_status(launch_dgrad_filters(jobs.data(), count, static_cast<hipStream_t>(stream)));
}

fp16_status fp16_conv_dgrad_wf(const fp16_conv_desc* desc, const fp16_t* dy, const fp16_t* wf,
                               const fp16_t* addend, fp16_t* dx, void* ws, size_t ws_bytes,
                               fp16_stream_t stream) {
  return conv_dgrad_impl(desc, dy, wf, addend, dx, ws, ws_bytes, stream, true);
}

fp16_status fp16_conv_dgrad_wf_m(const fp16_conv_desc* desc, const fp16_t* dy, const fp16_t* wf,
                                 const fp16_t* addend, const uint8_t* addend_mask, fp16_t* dx,
                                 void* ws, size_t ws_bytes, fp16_stream_t stream) {
  if (!addend || !addend_mask) return FP16_ERR_NULL;
  return conv_dgrad_impl(desc, dy, wf, addend, dx, ws, ws_bytes, stream, true, addend_mask);
}

fp16_status fp16_conv_dgrad_wf_ex(const fp16_conv_desc* desc, const fp16_t* dy, const fp16_t* wf,
                                  const fp16_t* addend, const uint8_t* addend_mask,
                                  int32_t addend_stride, fp16_t* dx, void* ws, size_t ws_bytes,
                                  fp16_stream_t stream) {
  return conv_dgrad_impl(desc, dy, wf, addend, dx, ws, ws_bytes, stream, true, addend_mask,
                         addend_stride);
}

}  // extern "C"

extern "C" {

fp16_status fp16_conv_wgrad_ex(const fp16_conv_desc* desc, const fp16_t* x, const fp16_t* dy,
                               fp16_t* dw, void* ws, size_t ws_bytes, int32_t workgroups,
                               fp16_stream_t stream) {
  ConvDims d;
  fp16_status s = check_conv(desc, &d);
  if (s != FP16_OK) return s;
  if (workgroups < 0 || workgroups > kWgradWorkgroups) return FP16_ERR_SHAPE;
  if (!x || !dy || !dw) return FP16_ERR_NULL;
  if (!aligned16(x) || !aligned16(dy) || !aligned16(dw)) return FP16_ERR_MISALIGNED;
  const ConvWs L = conv_ws(d, FP16_PASS_WGRAD, workgroups);
  if ((s = check_ws(L, ws, ws_bytes)) != FP16_OK) return s;
  const size_t wb = (size_t)d.w_elems * 2;
  if (overlap(dw, wb, x, (size_t)d.x_elems * 2) || overlap(dw, wb, dy, (size_t)d.y_elems * 2) ||
      overlap(dw, wb, ws, L.total))
    return FP16_ERR_ALIASING;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const h16* xe = reinterpret_cast<const h16*>(x);
  const h16* dye = reinterpret_cast<const h16*>(dy);
  if (d.accum)
    return hip_status(launch_conv_chain(chain_args(d), 2, xe, dye, reinterpret_cast<h16*>(dw), st));
  if (stem_s2d(d)) {
    // 4x4 stride-1 convolution over the space-to-depth image, pad 2 before
    // and 1 after: s2d pixel p + r' - 2 holds original rows 2(p + r') - 4 + dh
    h16* xs = wsp(ws, L.x);
    TRY(launch_s2d3(xe, xs, d.N, d.H, d.W, st));
    float* part = reinterpret_cast<float*>(static_cast<char*>(ws) + L.part);
    WgradArgs a{};
    a.x = xs; a.dy = dye;
    a.N = d.N; a.H = d.P; a.W = d.Q; a.C = 16; a.K = d.Kp; a.R = 4; a.S = 4;
    a.sh = 1; a.sw = 1; a.ph = 2; a.pw = 2; a.P = d.P; a.Q = d.Q;
    a.partial = part; a.splits = L.splits; a.pix_per_split = L.pps;
    TRY(launch_wgrad_partial(a, st));
    return hip_status(launch_wgrad_reduce_s2d3(part, L.splits, d.K, reinterpret_cast<h16*>(dw), st));
  }
  if (d.layout == FP16_NCHW) {
    TRY(launch_nchw_to_nhwc(xe, wsp(ws, L.x), d.N, d.C, d.H * d.W, d.Cp, st));
    TRY(launch_nchw_to_nhwc(dye, wsp(ws, L.y), d.N, d.K, d.P * d.Q, d.Kp, st));
    xe = wsp(ws, L.x);
    dye = wsp(ws, L.y);
  } else {
    if (d.Cp != d.C) {
      TRY(launch_pad_channels(xe, wsp(ws, L.x), (int64_t)d.N * d.H * d.W, d.C, d.Cp, st));
      xe = wsp(ws, L.x);
    }
    if (d.Kp != d.K) {
      TRY(launch_pad_channels(dye, wsp(ws, L.y), (int64_t)d.N * d.P * d.Q, d.K, d.Kp, st));
      dye = wsp(ws, L.y);
    }
  }
  float* part = reinterpret_cast<float*>(static_cast<char*>(ws) + L.part);
  WgradArgs a{};
  a.x = xe; a.dy = dye;
  a.N = d.N; a.H = d.H; a.W = d.W; a.C = d.Cp; a.K = d.Kp; a.R = d.R; a.S = d.S;
  a.sh = d.sh; a.sw = d.sw; a.ph = d.ph; a.pw = d.pw; a.P = d.P; a.Q = d.Q;
  a.partial = part; a.splits = L.splits; a.pix_per_split = L.pps;
  TRY(launch_wgrad_partial(a, st));
  TRY(launch_wgrad_reduce(part, L.splits, d.K, d.Kp, d.R, d.S, d.C, d.Cp, d.layout,
                          reinterpret_cast<h16*>(dw), st));
  return FP16_OK;
}

fp16_status fp16_conv_wgrad(const fp16_conv_desc* desc, const fp16_t* x, const fp16_t* dy,
                            fp16_t* dw, void* ws, size_t ws_bytes, fp16_stream_t stream) {
  return fp16_conv_wgrad_ex(desc, x, dy, dw, ws, ws_bytes, 0, stream);
}

// ---- batch normalisation ----------------------------------------------------

static fp16_status check_bn(const fp16_bn_desc* d, BnArgs* a) {
  if (!d) return FP16_ERR_NULL;
  if (d->layout != FP16_NHWC && d->layout != FP16_NCHW) return FP16_ERR_LAYOUT;
  if (d->n < 1 || d->c < 1 || d->h < 1 || d->w < 1 || d->c > 65535) return FP16_ERR_SHAPE;
  if ((int64_t)d->n * d->c * d->h * d->w >= kMaxElems) return FP16_ERR_SHAPE;
  if (!(d->eps >= 0.0f) || !(d->post_scale == d->post_scale)) return FP16_ERR_SHAPE;
  if (d->use_stats != 0 && d->use_stats != 1) return FP16_ERR_SHAPE;
  if (d->swap != 0 && d->swap != 1) return FP16_ERR_SHAPE;
  a->N = d->n; a->C = d->c; a->H = d->h; a->W = d->w; a->layout = d->layout;
  a->eps = d->eps; a->post_scale = d->post_scale; a->relu = d->relu ? 1 : 0;
  a->swap = d->swap;
  return FP16_OK;
}

size_t fp16_bn_workspace_bytes(const fp16_bn_desc* desc) {
  BnArgs a;
  if (check_bn(desc, &a) != FP16_OK) return 0;
  return bn_ws_bytes(a);
}

// The ReLU mask a forward keeps: one byte per 8 channels of each pixel.
static fp16_status check_mask(const BnArgs& a, const void* mask, size_t* bytes) {
  if (!mask) return FP16_ERR_NULL;
  if (!aligned16(mask)) return FP16_ERR_MISALIGNED;
  if (a.swap) return FP16_ERR_UNSUPPORTED;
  *bytes = bn_keep_mask_bytes(a);
  return *bytes ? FP16_OK : FP16_ERR_UNSUPPORTED;
}

static fp16_status bn_fwd_impl(const fp16_bn_desc* desc, const fp16_t* x, const fp16_t* gamma,
                               const fp16_t* beta, const fp16_t* residual, fp16_t* y, float* stats,
                               uint8_t* mask, bool want_mask, void* ws, size_t ws_bytes,
                               fp16_stream_t stream) {
  BnArgs a;
  fp16_status s = check_bn(desc, &a);
  if (s != FP16_OK) return s;
  if (!x || !gamma || !beta || !y || !stats) return FP16_ERR_NULL;
  size_t mb = 0;
  if (want_mask && (s = check_mask(a, mask, &mb)) != FP16_OK) return s;
  if (a.swap && !residual) return FP16_ERR_NULL;
  if (!aligned16(x) || !aligned16(y) || (residual && !aligned16(residual)) || !aligned16(stats))
    return FP16_ERR_MISALIGNED;
  const size_t need = bn_ws_bytes(a);
  if (!ws || ws_bytes < need) return FP16_ERR_WORKSPACE;
  if (!aligned16(ws)) return FP16_ERR_MISALIGNED;
  const size_t eb = (size_t)a.N * a.C * a.H * a.W * 2;
  const size_t cb = (size_t)a.C * 2;
  if ((y != x && overlap(y, eb, x, eb)) || (residual && y != residual && overlap(y, eb, residual, eb)) ||
      overlap(y, eb, gamma, cb) || overlap(y, eb, beta, cb) || overlap(y, eb, stats, (size_t)a.C * 8) ||
      overlap(y, eb, ws, need) || overlap(stats, (size_t)a.C * 8, ws, need))
    return FP16_ERR_ALIASING;
  // the workspace is written while the inputs are still being read
  if (overlap(ws, need, x, eb) || overlap(ws, need, residual, eb) || overlap(ws, need, gamma, cb) ||
      overlap(ws, need, beta, cb))
    return FP16_ERR_ALIASING;
  if (mb && (overlap(mask, mb, x, eb) || overlap(mask, mb, y, eb) ||
             overlap(mask, mb, residual, eb) || overlap(mask, mb, gamma, cb) ||
             overlap(mask, mb, beta, cb) || overlap(mask, mb, stats, (size_t)a.C * 8) ||
             overlap(mask, mb, ws, need)))
    return FP16_ERR_ALIASING;
  return hip_status(launch_bn_fwd(a, reinterpret_cast<const h16*>(x),
                                  reinterpret_cast<const h16*>(gamma),
                                  reinterpret_cast<const h16*>(beta),
                                  reinterpret_cast<const h16*>(residual), reinterpret_cast<h16*>(y),
                                  stats, desc->use_stats, ws, mb ? mask : nullptr,
                                  static_cast<hipStream_t>(stream)));
}

fp16_status fp16_bn_relu(const fp16_bn_desc* desc, const fp16_t* x, const fp16_t* gamma,
                         const fp16_t* beta, const fp16_t* residual, fp16_t* y, float* stats,
                         void* ws, size_t ws_bytes, fp16_stream_t stream) {
  return bn_fwd_impl(desc, x, gamma, beta, residual, y, stats, nullptr, false, ws, ws_bytes,
                     stream);
}

size_t fp16_bn_mask_bytes(const fp16_bn_desc* desc) {
  BnArgs a;
  if (check_bn(desc, &a) != FP16_OK || a.swap) return 0;
  return bn_keep_mask_bytes(a);
}

fp16_status fp16_bn_relu_m(const fp16_bn_desc* desc, const fp16_t* x, const fp16_t* gamma,
                           const fp16_t* beta, const fp16_t* residual, fp16_t* y, float* stats,
                           uint8_t* mask, void* ws, size_t ws_bytes, fp16_stream_t stream) {
  return bn_fwd_impl(desc, x, gamma, beta, residual, y, stats, mask, true, ws, ws_bytes, stream);
}

static fp16_status bn_bwd_impl(const fp16_bn_desc* desc, const fp16_t* x, const fp16_t* y,
                               const fp16_t* dy, const fp16_t* gamma, const fp16_t* beta,
                               const fp16_t* residual, const float* stats, const uint8_t* mask,
                               bool with_mask, fp16_t* dx, fp16_t* dgamma, fp16_t* dbeta,
                               fp16_t* dresidual, void* ws, size_t ws_bytes,
                               fp16_stream_t stream) {
  BnArgs a;
  fp16_status s = check_bn(desc, &a);
  if (s != FP16_OK) return s;
  if (!x || !dy || !gamma || !beta || !stats || !dx || !dgamma || !dbeta) return FP16_ERR_NULL;
  size_t mb = 0;
  if (with_mask) {
    if ((s = check_mask(a, mask, &mb)) != FP16_OK) return s;
    if (!a.relu) return FP16_ERR_UNSUPPORTED;
  }
  if (a.swap && !residual) return FP16_ERR_NULL;
  if (!aligned16(x) || (y && !aligned16(y)) || !aligned16(dy) || !aligned16(dx) ||
      (residual && !aligned16(residual)) || (dresidual && !aligned16(dresidual)) ||
      !aligned16(stats))
    return FP16_ERR_MISALIGNED;
  const size_t need = bn_ws_bytes(a);
  if (!ws || ws_bytes < need) return FP16_ERR_WORKSPACE;
  if (!aligned16(ws)) return FP16_ERR_MISALIGNED;
  const size_t eb = (size_t)a.N * a.C * a.H * a.W * 2;
  const size_t cb = (size_t)a.C * 2;
  const void* ins[4] = {x, y, residual, gamma};
  const size_t insz[4] = {eb, eb, eb, cb};
  for (int i = 0; i < 4; ++i) {
    if (overlap(dx, eb, ins[i], insz[i])) return FP16_ERR_ALIASING;
    if (dresidual && overlap(dresidual, eb, ins[i], insz[i])) return FP16_ERR_ALIASING;
  }
  if ((dx != dy && overlap(dx, eb, dy, eb)) || (dresidual && overlap(dresidual, eb, dy, eb)) ||
      (dresidual && overlap(dresidual, eb, dx, eb)) || overlap(dx, eb, ws, need) ||
      overlap(dgamma, cb, dbeta, cb) || overlap(dgamma, cb, ws, need) ||
      overlap(dbeta, cb, ws, need) || overlap(dgamma, cb, dx, eb) || overlap(dbeta, cb, dx, eb))
    return FP16_ERR_ALIASING;
  // the workspace (partial sums, the kept ReLU mask) is written while the
  // inputs are still being read
  if (overlap(ws, need, x, eb) || overlap(ws, need, y, eb) || overlap(ws, need, dy, eb) ||
      overlap(ws, need, residual, eb) || overlap(ws, need, gamma, cb) ||
      overlap(ws, need, beta, cb) || overlap(ws, need, stats, (size_t)a.C * 8))
    return FP16_ERR_ALIASING;
  if (mb && (overlap(mask, mb, dx, eb) || overlap(mask, mb, ws, need) ||
             (dresidual && overlap(mask, mb, dresidual, eb)) || overlap(mask, mb, dgamma, cb) ||
             overlap(mask, mb, dbeta, cb)))
    return FP16_ERR_ALIASING;
  return hip_status(launch_bn_bwd(
      a, reinterpret_cast<const h16*>(x), reinterpret_cast<const h16*>(y),
      reinterpret_cast<const h16*>(dy), reinterpret_cast<const h16*>(gamma),
      reinterpret_cast<const h16*>(beta), reinterpret_cast<const h16*>(residual), stats,
      reinterpret_cast<h16*>(dx), reinterpret_cast<h16*>(dgamma), reinterpret_cast<h16*>(dbeta),
      reinterpret_cast<h16*>(dresidual), ws, mb ? mask : nullptr,
      static_cast<hipStream_t>(stream)));
}

fp16_status fp16_bn_relu_bwd(const fp16_bn_desc* desc, const fp16_t* x, const fp16_t* y,
                             const fp16_t* dy, const fp16_t* gamma, const fp16_t* beta,
                             const fp16_t* residual, const float* stats, fp16_t* dx,
                             fp16_t* dgamma, fp16_t* dbeta, fp16_t* dresidual, void* ws,
                             size_t ws_bytes, fp16_stream_t stream) {
  return bn_bwd_impl(desc, x, y, dy, gamma, beta, residual, stats, nullptr, false, dx, dgamma,
                     dbeta, dresidual, ws, ws_bytes, stream);
}

fp16_status fp16_bn_relu_bwd_m(const fp16_bn_desc* desc, const fp16_t* x, const uint8_t* mask,
                               const fp16_t* dy, const fp16_t* gamma, const fp16_t* beta,
                               const float* stats, fp16_t* dx, fp16_t* dgamma, fp16_t* dbeta,
                               fp16_t* dresidual, void* ws, size_t ws_bytes,
                               fp16_stream_t stream) {
  return bn_bwd_impl(desc, x, nullptr, dy, gamma, beta, nullptr, stats, mask, true, dx, dgamma,
                     dbeta, dresidual, ws, ws_bytes, stream);
}

// ---- SGD ------------------------------------------------------------------------

fp16_status fp16_sgd_step(fp16_t* w, const fp16_t* g, fp16_t* m, size_t n, float lr,
                          float momentum, float weight_decay, fp16_stream_t stream) {
  if (n == 0) return FP16_OK;
  if (!w || !g || !m) return FP16_ERR_NULL;
  if (!aligned16(w) || !aligned16(g) || !aligned16(m)) return FP16_ERR_MISALIGNED;
  if (n >= ((size_t)1 << 40)) return FP16_ERR_SHAPE;
  const size_t b = n * 2;
  if (overlap(w, b, g, b) || overlap(m, b, g, b) || overlap(w, b, m, b)) return FP16_ERR_ALIASING;
  return hip_status(launch_sgd(reinterpret_cast<h16*>(w), reinterpret_cast<const h16*>(g),
                               reinterpret_cast<h16*>(m), n, lr, momentum, weight_decay,
                               static_cast<hipStream_t>(stream)));
}

fp16_status fp16_sgd_step_f16(fp16_t* w, const fp16_t* g, fp16_t* m, size_t n, float lr,
                              float momentum, float weight_decay, fp16_stream_t stream) {
  if (n == 0) return FP16_OK;
  if (!w || !g || !m) return FP16_ERR_NULL;
  if (!aligned16(w) || !aligned16(g) || !aligned16(m)) return FP16_ERR_MISALIGNED;
  if (n >= ((size_t)1 << 40)) return FP16_ERR_SHAPE;
  const size_t b = n * 2;
  if (overlap(w, b, g, b) || overlap(m, b, g, b) || overlap(w, b, m, b)) return FP16_ERR_ALIASING;
  return hip_status(launch_sgd_f16(reinterpret_cast<h16*>(w), reinterpret_cast<const h16*>(g),
                                   reinterpret_cast<h16*>(m), n, lr, momentum, weight_decay,
                                   static_cast<hipStream_t>(stream)));
}

// ---- pooling --------------------------------------------------------------------

static fp16_status check_pool(const fp16_pool_desc* d, PoolArgs* a) {
  if (!d) return FP16_ERR_NULL;
  if (d->layout != FP16_NHWC && d->layout != FP16_NCHW) return FP16_ERR_LAYOUT;
  if (d->n < 1 || d->c < 1 || d->h < 1 || d->w < 1 || d->r < 1 || d->s < 1 || d->r > 15 ||
      d->s > 15 || d->stride_h < 1 || d->stride_w < 1 || d->stride_h > 16 || d->stride_w > 16 ||
      d->pad_h < 0 || d->pad_w < 0 || d->pad_h >= d->r || d->pad_w >= d->s ||
      d->c > 65535 || d->h > 65535 || d->w > 65535)
    return FP16_ERR_SHAPE;
  if (d->h + 2 * d->pad_h < d->r || d->w + 2 * d->pad_w < d->s) return FP16_ERR_SHAPE;
  if ((int64_t)d->n * d->c * d->h * d->w >= kMaxElems) return FP16_ERR_SHAPE;
  a->N = d->n; a->C = d->c; a->H = d->h; a->W = d->w; a->R = d->r; a->S = d->s;
  a->sh = d->stride_h; a->sw = d->stride_w; a->ph = d->pad_h; a->pw = d->pad_w;
  a->layout = d->layout;
  a->P = (a->H + 2 * a->ph - a->R) / a->sh + 1;
  a->Q = (a->W + 2 * a->pw - a->S) / a->sw + 1;
  return FP16_OK;
}

fp16_status fp16_pool_out_dims(const fp16_pool_desc* desc, int32_t* p, int32_t* q) {
  PoolArgs a;
  const fp16_status s = check_pool(desc, &a);
  if (s != FP16_OK) return s;
  if (!p || !q) return FP16_ERR_NULL;
  *p = a.P;
  *q = a.Q;
  return FP16_OK;
}

fp16_status fp16_maxpool_fwd(const fp16_pool_desc* desc, const fp16_t* x, fp16_t* y,
                             uint8_t* idx, fp16_stream_t stream) {
  PoolArgs a;
  const fp16_status s = check_pool(desc, &a);
  if (s != FP16_OK) return s;
  if (!x || !y || !idx) return FP16_ERR_NULL;
  if (!aligned16(x) || !aligned16(y) || !aligned16(idx)) return FP16_ERR_MISALIGNED;
  const size_t xb = (size_t)a.N * a.C * a.H * a.W * 2;
  const size_t yn = (size_t)a.N * a.C * a.P * a.Q;
  if (overlap(y, yn * 2, x, xb) || overlap(idx, yn, x, xb) || overlap(y, yn * 2, idx, yn))
    return FP16_ERR_ALIASING;
  return hip_status(launch_maxpool_fwd(a, reinterpret_cast<const h16*>(x),
                                       reinterpret_cast<h16*>(y), idx,
                                       static_cast<hipStream_t>(stream)));
}

fp16_status fp16_maxpool_bwd(const fp16_pool_desc* desc, const uint8_t* idx, const fp16_t* dy,
                             fp16_t* dx, fp16_stream_t stream) {
  PoolArgs a;
  const fp16_status s = check_pool(desc, &a);
  if (s != FP16_OK) return s;
  if (!idx || !dy || !dx) return FP16_ERR_NULL;
  if (!aligned16(idx) || !aligned16(dy) || !aligned16(dx)) return FP16_ERR_MISALIGNED;
  const size_t xb = (size_t)a.N * a.C * a.H * a.W * 2;
  const size_t yn = (size_t)a.N * a.C * a.P * a.Q;
  if (overlap(dx, xb, dy, yn * 2) || overlap(dx, xb, idx, yn)) return FP16_ERR_ALIASING;
  return hip_status(launch_maxpool_bwd(a, idx, reinterpret_cast<const h16*>(dy),
                                       reinterpret_cast<h16*>(dx),
                                       static_cast<hipStream_t>(stream)));
}

fp16_status fp16_bn_relu_maxpool(const fp16_bn_desc* bn, const fp16_pool_desc* pool,
                                 const fp16_t* x, const fp16_t* gamma, const fp16_t* beta,
                                 float* stats, fp16_t* y, uint8_t* idx, void* ws, size_t ws_bytes,
                                 fp16_stream_t stream) {
  BnArgs b;
  PoolArgs pa;
  fp16_status s = check_bn(bn, &b);
  if (s != FP16_OK) return s;
  if ((s = check_pool(pool, &pa)) != FP16_OK) return s;
  if (!x || !gamma || !beta || !stats || !y || !idx) return FP16_ERR_NULL;
  if (pa.N != b.N || pa.C != b.C || pa.H != b.H || pa.W != b.W || pa.layout != b.layout)
    return FP16_ERR_SHAPE;
  if (!bn_maxpool_ok(b, pa)) return FP16_ERR_UNSUPPORTED;
  if (!aligned16(x) || !aligned16(y) || !aligned16(idx) || !aligned16(stats))
    return FP16_ERR_MISALIGNED;
  const size_t need = bn_ws_bytes(b);
  if (!ws || ws_bytes < need) return FP16_ERR_WORKSPACE;
  if (!aligned16(ws)) return FP16_ERR_MISALIGNED;
  const size_t eb = (size_t)b.N * b.C * b.H * b.W * 2, cb = (size_t)b.C * 2,
               sb = (size_t)b.C * 8;
  const size_t yn = (size_t)pa.N * pa.C * pa.P * pa.Q;
  const void* ins[4] = {x, gamma, beta, stats};
  const size_t insz[4] = {eb, cb, cb, sb};
  for (int i = 0; i < 4; ++i)
    if (overlap(y, yn * 2, ins[i], insz[i]) || overlap(idx, yn, ins[i], insz[i]) ||
        (i < 3 && overlap(ws, need, ins[i], insz[i])))
      return FP16_ERR_ALIASING;
  if (overlap(y, yn * 2, idx, yn) || overlap(y, yn * 2, ws, need) || overlap(idx, yn, ws, need) ||
      overlap(stats, sb, ws, need))
    return FP16_ERR_ALIASING;
  return hip_status(launch_bn_fwd_maxpool(
      b, pa, reinterpret_cast<const h16*>(x), reinterpret_cast<const h16*>(gamma),
      reinterpret_cast<const h16*>(beta), stats, bn->use_stats, ws, reinterpret_cast<h16*>(y),
      idx, static_cast<hipStream_t>(stream)));
}

// The global window only.  With r, s <= 15 the window holds at most 225
// binary16 terms, so every float64 sum of them is exact (|sum| < 2^24 in
// units of 2^-24 fits in 53 bits).
static fp16_status check_global_pool(const fp16_pool_desc* desc, PoolArgs* a) {
  const fp16_status s = check_pool(desc, a);
  if (s != FP16_OK) return s;
  if (a->R != a->H || a->S != a->W || a->ph != 0 || a->pw != 0) return FP16_ERR_UNSUPPORTED;
  return FP16_OK;
}

fp16_status fp16_avgpool_fwd(const fp16_pool_desc* desc, const fp16_t* x, fp16_t* y,
                             fp16_stream_t stream) {
  PoolArgs a;
  const fp16_status s = check_global_pool(desc, &a);
  if (s != FP16_OK) return s;
  if (!x || !y) return FP16_ERR_NULL;
  if (!aligned16(x) || !aligned16(y)) return FP16_ERR_MISALIGNED;
  if (overlap(y, (size_t)a.N * a.C * 2, x, (size_t)a.N * a.C * a.H * a.W * 2))
    return FP16_ERR_ALIASING;
  return hip_status(launch_avgpool_fwd(a, reinterpret_cast<const h16*>(x),
                                       reinterpret_cast<h16*>(y),
                                       static_cast<hipStream_t>(stream)));
}

fp16_status fp16_avgpool_bwd(const fp16_pool_desc* desc, const fp16_t* dy, fp16_t* dx,
                             fp16_stream_t stream) {
  PoolArgs a;
  const fp16_status s = check_global_pool(desc, &a);
  if (s != FP16_OK) return s;
  if (!dy || !dx) return FP16_ERR_NULL;
  if (!aligned16(dy) || !aligned16(dx)) return FP16_ERR_MISALIGNED;
  if (overlap(dx, (size_t)a.N * a.C * a.H * a.W * 2, dy, (size_t)a.N * a.C * 2))
    return FP16_ERR_ALIASING;
  return hip_status(launch_avgpool_bwd(a, reinterpret_cast<const h16*>(dy),
                                       reinterpret_cast<h16*>(dx),
                                       static_cast<hipStream_t>(stream)));
}

// ---- classifier bias and softmax cross-entropy ------------------------------------

fp16_status fp16_softmax_ce(int32_t n, int32_t k, const fp16_t* z, const fp16_t* bias,
                            const int32_t* labels, float* loss, fp16_t* dz, fp16_t* dbias,
                            fp16_stream_t stream) {
  // n <= 2^24 keeps the float64 batch sum of the bias gradient exact
  if (n < 1 || k < 1 || k > 65535 || n > (1 << 24)) return FP16_ERR_SHAPE;
  if ((int64_t)n * k >= kMaxElems) return FP16_ERR_SHAPE;
  if (!z || !bias || !labels || !loss || !dz || !dbias) return FP16_ERR_NULL;
  if (!aligned16(z) || !aligned16(bias) || !aligned16(labels) || !aligned16(loss) ||
      !aligned16(dz) || !aligned16(dbias))
    return FP16_ERR_MISALIGNED;
  const size_t zb = (size_t)n * k * 2, kb = (size_t)k * 2, nb = (size_t)n * 4;
  if ((dz != z && overlap(dz, zb, z, zb)) || overlap(dz, zb, bias, kb) ||
      overlap(dz, zb, labels, nb) || overlap(dz, zb, loss, nb) || overlap(dz, zb, dbias, kb) ||
      overlap(dbias, kb, z, zb) || overlap(dbias, kb, bias, kb) || overlap(dbias, kb, labels, nb) ||
      overlap(dbias, kb, loss, nb) || overlap(loss, nb, z, zb) || overlap(loss, nb, bias, kb) ||
      overlap(loss, nb, labels, nb))
    return FP16_ERR_ALIASING;
  return hip_status(launch_softmax_ce(n, k, reinterpret_cast<const h16*>(z),
                                      reinterpret_cast<const h16*>(bias), labels, loss,
                                      reinterpret_cast<h16*>(dz), reinterpret_cast<h16*>(dbias),
                                      static_cast<hipStream_t>(stream)));
}

// ---- convolution fused with the statistics of the BN that follows ---------------

static fp16_status check_conv_bn(const fp16_conv_desc* cd, const fp16_bn_desc* bd, ConvDims* d,
                                 BnArgs* b) {
  fp16_status s = check_conv(cd, d);
  if (s != FP16_OK) return s;
  if ((s = check_bn(bd, b)) != FP16_OK) return s;
  if (d->layout != FP16_NHWC || b->layout != FP16_NHWC || d->K % 8 != 0 || d->accum)
    return FP16_ERR_UNSUPPORTED;
  if (b->N != d->N || b->C != d->K || b->H != d->P || b->W != d->Q || bd->use_stats != 0)
    return FP16_ERR_SHAPE;
  return FP16_OK;
}

// Tile records ([nb][3][K] float32, 128 rows each) and the statistics'
// per-slice sums after the convolution's own workspace; when the kernel picked
// for the convolution does not take the statistics, the BN's own workspace
// takes that place instead.
static size_t conv_bn_band_off(const ConvDims& d) { return conv_ws(d, FP16_PASS_FWD).total; }
static int conv_bn_nb(const ConvDims& d) { return (int)(((int64_t)d.N * d.P * d.Q + 127) / 128); }

size_t fp16_conv_bn_workspace_bytes(const fp16_conv_desc* conv, const fp16_bn_desc* bn) {
  ConvDims d;
  BnArgs b;
  if (check_conv_bn(conv, bn, &d, &b) != FP16_OK) return 0;
  const size_t rec = align256((size_t)3 * d.K * conv_bn_nb(d) * sizeof(float)) +
                     bn_band_ws_bytes(d.K, conv_bn_nb(d));
  const size_t bnw = bn_ws_bytes(b);
  return conv_bn_band_off(d) + (rec > bnw ? rec : bnw);
}

static fp16_status conv_bn_impl(const fp16_conv_desc* conv, const fp16_bn_desc* bn,
                                const fp16_t* x, const fp16_t* w, const fp16_t* gamma,
                                const fp16_t* beta, const fp16_t* residual, fp16_t* y, fp16_t* z,
                                float* stats, uint8_t* mask, bool want_mask, void* ws,
                                size_t ws_bytes, fp16_stream_t stream) {
  ConvDims d;
  BnArgs b;
  fp16_status s = check_conv_bn(conv, bn, &d, &b);
  if (s != FP16_OK) return s;
  if (!x || !w || !gamma || !beta || !y || !z || !stats) return FP16_ERR_NULL;
  size_t mb = 0;
  if (want_mask && (s = check_mask(b, mask, &mb)) != FP16_OK) return s;
  if (b.swap && !residual) return FP16_ERR_NULL;
  if (!aligned16(x) || !aligned16(w) || !aligned16(y) || !aligned16(z) || !aligned16(stats) ||
      (residual && !aligned16(residual)))
    return FP16_ERR_MISALIGNED;
  const size_t need = fp16_conv_bn_workspace_bytes(conv, bn);
  if (!ws || ws_bytes < need) return FP16_ERR_WORKSPACE;
  if (!aligned16(ws)) return FP16_ERR_MISALIGNED;
  const size_t yb = (size_t)d.y_elems * 2, xb = (size_t)d.x_elems * 2,
               wb = (size_t)d.w_elems * 2, cb = (size_t)d.K * 2, sb = (size_t)d.K * 8;
  if (overlap(y, yb, x, xb) || overlap(y, yb, w, wb) || overlap(y, yb, ws, need) ||
      overlap(y, yb, gamma, cb) || overlap(y, yb, beta, cb) || overlap(y, yb, stats, sb) ||
      (z != y && overlap(z, yb, y, yb)) || overlap(z, yb, x, xb) || overlap(z, yb, w, wb) ||
      overlap(z, yb, ws, need) || overlap(z, yb, gamma, cb) || overlap(z, yb, beta, cb) ||
      overlap(z, yb, stats, sb) || (residual && z != residual && overlap(z, yb, residual, yb)) ||
      (residual && overlap(y, yb, residual, yb)) || overlap(stats, sb, ws, need))
    return FP16_ERR_ALIASING;
  if (overlap(ws, need, x, xb) || overlap(ws, need, w, wb) || overlap(ws, need, gamma, cb) ||
      overlap(ws, need, beta, cb) || overlap(ws, need, residual, yb))
    return FP16_ERR_ALIASING;
  if (mb && (overlap(mask, mb, x, xb) || overlap(mask, mb, w, wb) || overlap(mask, mb, y, yb) ||
             overlap(mask, mb, z, yb) || overlap(mask, mb, residual, yb) ||
             overlap(mask, mb, gamma, cb) || overlap(mask, mb, beta, cb) ||
             overlap(mask, mb, stats, sb) || overlap(mask, mb, ws, need)))
    return FP16_ERR_ALIASING;
  uint8_t* mout = mb ? mask : nullptr;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const ConvWs L = conv_ws(d, FP16_PASS_FWD);
  const h16* xe = reinterpret_cast<const h16*>(x);
  const h16* we = reinterpret_cast<const h16*>(w);
  float* part = reinterpret_cast<float*>(static_cast<char*>(ws) + conv_bn_band_off(d));
  {
    // the ResNet stem: its own kernel on the unpadded image, then the BN with
    // its own statistics pass
    const IgemmArgs sa = stem_args(d, xe, we, reinterpret_cast<h16*>(y));
    if (stem_conv_ok(sa)) {
      TRY(launch_stem(sa, st));
      return hip_status(launch_bn_fwd(b, reinterpret_cast<const h16*>(y),
                                      reinterpret_cast<const h16*>(gamma),
                                      reinterpret_cast<const h16*>(beta),
                                      reinterpret_cast<const h16*>(residual),
                                      reinterpret_cast<h16*>(z), stats, 0, part, mout, st));
    }
  }
  if (d.Cp != d.C) {
    TRY(launch_pad_channels(xe, wsp(ws, L.x), (int64_t)d.N * d.H * d.W, d.C, d.Cp, st));
    TRY(launch_pad_channels(we, wsp(ws, L.w), (int64_t)d.K * d.R * d.S, d.C, d.Cp, st));
    xe = wsp(ws, L.x);
    we = wsp(ws, L.w);
  }
  IgemmArgs a{};
  a.act = xe; a.N = d.N; a.Hi = d.H; a.Wi = d.W; a.Ci = d.Cp;
  a.stride_h = d.sh; a.stride_w = d.sw;
  a.Co = d.K; a.out = reinterpret_cast<h16*>(y); a.OH = d.P; a.OW = d.Q; a.ldo = d.K;
  a.os_h = 1; a.os_w = 1;
  a.nphase = 1;
  a.ph[0] = IgemmPhase{we, d.R * d.S * d.Cp, d.R, d.S, d.ph, d.pw, d.P, d.Q, 0, 0};
  const h16* gp = reinterpret_cast<const h16*>(gamma);
  const h16* bp = reinterpret_cast<const h16*>(beta);
  const h16* rp = reinterpret_cast<const h16*>(residual);
  if (!igemm_stats_pay(a)) {
    // the kernel picked for this shape does not take the statistics, or is
    // faster without them: run the convolution and the BN as separate kernels
    // (same results as the two calls)
    TRY(launch_igemm(a, st));
    return hip_status(launch_bn_fwd(b, reinterpret_cast<const h16*>(y), gp, bp, rp,
                                    reinterpret_cast<h16*>(z), stats, 0, part, mout, st));
  }
  a.stat = part;
  a.stat_nb = igemm_stat_records(a);  // at most conv_bn_nb(d), which sizes the space
  TRY(launch_igemm(a, st));
  void* band_ws = reinterpret_cast<char*>(part) +
                  align256((size_t)3 * d.K * a.stat_nb * sizeof(float));
  IgemmArgs z2 = a;
  z2.stat = nullptr;
  if (b.layout == FP16_NHWC && igemm_takes_apply(z2)) {
    // the statistics, then a second pass of the convolution that recomputes
    // y bit for bit from x and writes z = the BN apply of it (with the
    // shortcut and the kept ReLU mask) instead of reading y back
    TRY(launch_bn_band_stats(b, part, a.stat_nb, band_ws, stats, st));
    z2.out = reinterpret_cast<h16*>(z);
    z2.bn_stats = stats;
    z2.bn_gamma = gp;
    z2.bn_beta = bp;
    z2.bn_res = rp;
    z2.bn_mask = mout;
    z2.bn_scale = b.post_scale;
    z2.bn_relu = b.relu;
    z2.bn_swap = b.swap;
    return hip_status(launch_igemm(z2, st));
  }
  return hip_status(launch_bn_fwd_bands(b, part, a.stat_nb, band_ws,
                                        reinterpret_cast<const h16*>(y),
                                        reinterpret_cast<const h16*>(gamma),
                                        reinterpret_cast<const h16*>(beta),
                                        reinterpret_cast<const h16*>(residual),
                                        reinterpret_cast<h16*>(z), stats, mout, st));
}

fp16_status fp16_conv_bn_relu_fwd(const fp16_conv_desc* conv, const fp16_bn_desc* bn,
                                  const fp16_t* x, const fp16_t* w, const fp16_t* gamma,
                                  const fp16_t* beta, const fp16_t* residual, fp16_t* y,
                                  fp16_t* z, float* stats, void* ws, size_t ws_bytes,
                                  fp16_stream_t stream) {
  return conv_bn_impl(conv, bn, x, w, gamma, beta, residual, y, z, stats, nullptr, false, ws,
                      ws_bytes, stream);
}

fp16_status fp16_conv_bn_relu_fwd_m(const fp16_conv_desc* conv, const fp16_bn_desc* bn,
                                    const fp16_t* x, const fp16_t* w, const fp16_t* gamma,
                                    const fp16_t* beta, const fp16_t* residual, fp16_t* y,
                                    fp16_t* z, float* stats, uint8_t* mask, void* ws,
                                    size_t ws_bytes, fp16_stream_t stream) {
  return conv_bn_impl(conv, bn, x, w, gamma, beta, residual, y, z, stats, mask, true, ws,
                      ws_bytes, stream);
}

}  // extern "C"
