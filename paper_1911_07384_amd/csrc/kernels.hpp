// Internal launch interface between the C ABI (api.hip) and the kernel
// translation units.  Every launcher enqueues on `st` and returns the
// hipError_t of the launch.  Arguments have already been validated.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

#include "common.hpp"

namespace fp16k {

// ---- SGD (sgd.hip) --------------------------------------------------------
hipError_t launch_sgd(h16* w, const h16* g, h16* m, size_t n, float lr, float momentum,
                      float weight_decay, hipStream_t st);
// The same update with every operation a binary16 fma (binary16 scalars).
hipError_t launch_sgd_f16(h16* w, const h16* g, h16* m, size_t n, float lr, float momentum,
                          float weight_decay, hipStream_t st);

// ---- layout helpers (layout.hip) -----------------------------------------
// [N][C][HW] -> [N][HW][Cp] with channels c >= C zero-filled (Cp >= C).
hipError_t launch_nchw_to_nhwc(const h16* src, h16* dst, int N, int C, int HW, int Cp,
                               hipStream_t st);
// [N][HW][Cp] -> [N][C][HW] (channels >= C dropped).
hipError_t launch_nhwc_to_nchw(const h16* src, h16* dst, int N, int C, int HW, int Cp,
                               hipStream_t st);
// Repack channels of an NHWC tensor: [P][C] -> [P][Cp] zero-filled.
hipError_t launch_pad_channels(const h16* src, h16* dst, int64_t P, int C, int Cp, hipStream_t st);

// ---- convolution (conv_igemm.hip, conv_wgrad.hip) -------------------------
// One implicit-GEMM "phase": a stride-1-or-sigma gather of the NHWC source
// over an output grid, against a filter laid out [Co][Rt][St][Ci].
struct IgemmPhase {
  const h16* filt;  // [Co][Rt*St*Ci], row stride ldb
  int ldb;
  int Rt, St;       // taps of this phase
  int pad_h, pad_w; // source row = i*stride_h - pad_h + r
  int Ho, Wo;       // output grid of this phase
  int oph, opw;     // output tensor position = (i*os_h + oph, j*os_w + opw)
};

struct IgemmArgs {
  const h16* act;  // NHWC source [N][Hi][Wi][Ci], Ci % 8 == 0
  int N, Hi, Wi, Ci;
  int stride_h, stride_w;
  int Co;          // output channels (GEMM N)
  h16* out;        // NHWC output [N][OH][OW][ldo], writes channels [0, Co)
  const h16* addend;  // nullable, laid out like out: out = rne16(acc + addend)
  // nullable (needs addend, ldo == Co, Co % 8 == 0): a ReLU mask over the
  // addend, bit (i % 8) of byte i / 8 for element i of the addend's layout;
  // an element whose bit is clear adds +0 instead of the addend
  const uint8_t* amask;
  // 0 or 1: the addend is laid out like out; s > 1: it holds only the output
  // pixels whose row and column are multiples of s, as [N][ceil(OH/s)]
  // [ceil(OW/s)][ldo], and every other pixel adds +0
  int astride;
  int OH, OW, ldo;
  int os_h, os_w;
  int nphase;
  IgemmPhase ph[4];
  // Optional statistics of the rounded output for a following BN (single
  // phase, Co % 8 == 0, no addend, and a kernel that takes them, see
  // igemm_takes_stats): nb = igemm_stat_records records; record j covers the
  // 128-row tiles j, j + nb, j + 2nb, ... of the output rows and holds, per
  // channel c, a shift K (one of its values) and the sums of (y - K) and
  // (y - K)^2 over its rows, at stat[(j * 3 + q) * Co + c], q = 0, 1, 2.
  float* stat;
  int stat_nb;
  // N-tiles per group of the XCD-contiguous workgroup-to-tile order, or 0
  // for the launch order (set by the launcher)
  int gn;
  // Optional split of the reduction for a dense GEMM (a 1x1 filter over 1x1
  // images, no statistics, no masked or strided addend; see
  // dense_gemm_splits): float32 partial sums [splits][N][Co], summed in
  // split order, the addend added, and rounded once by a second kernel.
  float* part;
  int splits;
  // Optional BN apply in the epilogue (the pointwise kernel; see
  // igemm_takes_apply): out receives z, the declared float32 apply of the
  // rounded convolution output y with the statistics bn_stats (mean [Co],
  // 1/sqrt(var + eps) [Co]), bn_gamma, bn_beta, bn_scale, the shortcut bn_res
  // (nullable), the BN swap and the ReLU, instead of y; bn_mask (nullable)
  // keeps z's ReLU mask, one byte per 8 channels (bit e = [z element e > 0]).
  const float* bn_stats;
  const h16* bn_gamma;
  const h16* bn_beta;
  const h16* bn_res;
  uint8_t* bn_mask;
  float bn_scale;
  int bn_relu, bn_swap;
};

// Reduction splits for a dense GEMM of M rows, a K-long reduction and Co
// outputs (the classifier at batch 128: fc forward 128 x 2048 -> 1000, data
// gradient 128 x 1000 -> 2048), or 0 where the GEMM runs whole: on tiles of
// 32 x 128 the unsplit problem has too few workgroups to fill the CUs.
int dense_gemm_splits(int64_t M, int K, int Co);

hipError_t launch_igemm(const IgemmArgs& a, hipStream_t st);
// Whether taking the BN statistics in the convolution's epilogue is faster
// than the convolution without them plus a separate statistics pass (false
// where the kernel takes none).
bool igemm_stats_pay(const IgemmArgs& a);
// The ResNet stem convolution (3 channels, 7x7, stride 2, pad 3, 64 outputs)
// on its own kernel: act is the unpadded 3-channel image (Ci = 3) and the
// filter KRSC with ldb = 147.  stem_conv_ok says whether launch_stem takes the
// problem (with statistics when a.stat is set).
bool stem_conv_ok(const IgemmArgs& a);
hipError_t launch_stem(const IgemmArgs& a, hipStream_t st);
// Whether the kernel launch_igemm picks for this problem can take the BN
// statistics (IgemmArgs::stat) in its epilogue.
bool igemm_takes_stats(const IgemmArgs& a);
// Whether launch_igemm can apply a following BN in the epilogue of this
// problem (IgemmArgs::bn_stats; the problem without stats, addend or mask).
bool igemm_takes_apply(const IgemmArgs& a);
// The number of statistics records the kernel picked for this problem writes
// (one per 128-row tile, or fewer where a workgroup sums several tiles);
// never more than the tiles.
int igemm_stat_records(const IgemmArgs& a);

// Geometry of one stride phase (ph, pw) of the data gradient.  Output rows
// h = ph + sh*i (i < Hph) receive exactly the taps r = r0 + sh*t (t < ntr)
// with r0 = (ph + pad_h) mod sh, reading dy row p = i + (ph + pad_h - r0)/sh - t.
// With the taps stored in reverse order (t' = ntr-1-t) this is a stride-1
// gather p = i - pad_h' + t' with pad_h' = ntr - 1 - (ph + pad_h - r0)/sh.
// Columns likewise.  A phase with ntr or nts = 0 receives no tap (zeros).
struct DgradPhase {
  int r0, s0, ntr, nts, Hph, Wph, pad_h, pad_w;
};
__host__ __device__ inline DgradPhase dgrad_phase(int ph, int pw, int H, int W, int R, int S,
                                                  int sh, int sw, int pad_h, int pad_w) {
  DgradPhase d;
  d.r0 = (ph + pad_h) % sh;
  d.s0 = (pw + pad_w) % sw;
  d.ntr = d.r0 < R ? (R - d.r0 + sh - 1) / sh : 0;
  d.nts = d.s0 < S ? (S - d.s0 + sw - 1) / sw : 0;
  d.Hph = ph < H ? (H - ph + sh - 1) / sh : 0;
  d.Wph = pw < W ? (W - pw + sw - 1) / sw : 0;
  d.pad_h = d.ntr - 1 - (ph + pad_h - d.r0) / sh;
  d.pad_w = d.nts - 1 - (pw + pad_w - d.s0) / sw;
  return d;
}

// Filter transform for the data gradient: W [K][R][S][Cw] (KRSC, row channel
// stride Cw) -> per stride phase (ph, pw) a filter [C][nt_r][nt_s][Kp]
// holding W[k][r0 + sh*(nt_r-1-t_r)][s0 + sw*(nt_s-1-t_s)][c] (zero for k >= K).
hipError_t launch_dgrad_filter(const h16* w, h16* dst, int K, int C, int R, int S, int Cw,
                               int Kp, int sh, int sw, int pad_h, int pad_w, hipStream_t st);
// The same rearrangement for n filters (channel stride Cw = C each), in as
// few launches as the kernel-argument table allows.
struct DgradFiltJob {
  const h16* w;
  h16* dst;
  int K, C, R, S, Kp, sh, sw, pad_h, pad_w;
  int blk0;  // first block of this job in its launch (set by the launcher)
};
hipError_t launch_dgrad_filters(const DgradFiltJob* jobs, int n, hipStream_t st);

struct WgradArgs {
  const h16* x;   // NHWC [N][H][W][C], C % 8 == 0
  const h16* dy;  // NHWC [N][P][Q][K], K % 8 == 0
  int N, H, W, C, K, R, S, sh, sw, ph, pw, P, Q;
  float* partial; // [splits][K][R*S*C]
  int splits;
  int pix_per_split;
};
hipError_t launch_wgrad_partial(const WgradArgs& a, hipStream_t st);
// dw[k][r][s][c] = rne16(sum_split partial[split][k][(r*S+s)*Cp + c]) for k < K, c < C,
// with Kp rows per split, written as KRSC (layout 0) or KCRS (layout 1).
hipError_t launch_wgrad_reduce(const float* partial, int splits, int K, int Kp, int R, int S,
                               int C, int Cp, int layout, h16* dw, hipStream_t st);
// The stem's weight gradient through a 2x2 space-to-depth view (layout.hip,
// conv_wgrad.hip): the 3-channel image as 16 channels at half resolution, and
// the 4x4 x 16 partial sums gathered back into the 7x7x3 filter (the splits
// folded in place in groups first, so partial holds scratch afterwards).
hipError_t launch_s2d3(const h16* src, h16* dst, int N, int H, int W, hipStream_t st);
hipError_t launch_wgrad_reduce_s2d3(float* partial, int splits, int K, h16* dw, hipStream_t st);
// Split-K plan of the weight gradient: about `target` workgroups (tiles x
// splits; kWgradWorkgroups, two per CU, unless the caller asks for fewer),
// each split at least two k-steps of pixels.
constexpr int kWgradWorkgroups = 512;
void wgrad_plan(int K, int Cp, int R, int S, int64_t npix, int target, int* splits,
                int* pix_per_split);

// Convolutions with every operation in binary16 (conv_f16chain.hip): each
// output a chain of binary16 fmas from +0 in the declared order.  NHWC
// activations, KRSC filter, any C and K.  pass 0: in0 = x, in1 = w, out = y;
// pass 1: in0 = dy, in1 = w, out = dx; pass 2: in0 = x, in1 = dy, out = dW.
struct ConvChainArgs {
  int N, C, H, W, K, R, S, sh, sw, ph, pw, P, Q;
};
hipError_t launch_conv_chain(const ConvChainArgs& a, int pass, const h16* in0, const h16* in1,
                             h16* out, hipStream_t st);

// ---- batch normalisation (bn.hip) ----------------------------------------
struct BnArgs {
  int N, C, H, W, layout;
  float eps, post_scale;
  int relu;
  int swap;  // BN swap: the shortcut joins before gamma
};
size_t bn_ws_bytes(const BnArgs& a);
// mout (nullable): keep the ReLU mask of y, one byte per 16-byte vector of y
// (bit e = [element e > 0]); needs the vectorised path and ReLU (the caller
// checks bn_keep_mask_bytes > 0).
hipError_t launch_bn_fwd(const BnArgs& a, const h16* x, const h16* gamma, const h16* beta,
                         const h16* res, h16* y, float* stats, int use_stats, void* ws,
                         uint8_t* mout, hipStream_t st);
size_t bn_keep_mask_bytes(const BnArgs& a);
// Forward from the band records of a convolution epilogue (IgemmArgs::stat):
// statistics, then the apply.  part: [nb][3][C] float32, record j over the
// 128-row tiles j, j + nb, ...;
// band_ws: bn_band_ws_bytes(C, nb) bytes of scratch for the per-slice sums.
size_t bn_band_ws_bytes(int C, int nb);
// The statistics alone from such records (mean [C], 1/sqrt(var + eps) [C]).
hipError_t launch_bn_band_stats(const BnArgs& a, const float* part, int nb, void* band_ws,
                                float* stats, hipStream_t st);
hipError_t launch_bn_fwd_bands(const BnArgs& a, const float* part, int nb, void* band_ws,
                               const h16* x, const h16* gamma, const h16* beta, const h16* res,
                               h16* y, float* stats, uint8_t* mout, hipStream_t st);
// mask (nullable): the ReLU mask the forward kept (no BN swap)
hipError_t launch_bn_bwd(const BnArgs& a, const h16* x, const h16* y, const h16* dy,
                         const h16* gamma, const h16* beta, const h16* res, const float* stats,
                         h16* dx, h16* dgamma, h16* dbeta, h16* dres, void* ws,
                         const uint8_t* mask, hipStream_t st);

// ---- pooling (pool.hip) ----------------------------------------------------
struct PoolArgs {
  int N, C, H, W, R, S, sh, sw, ph, pw, P, Q, layout;
};
hipError_t launch_maxpool_fwd(const PoolArgs& a, const h16* x, h16* y, uint8_t* idx,
                              hipStream_t st);
hipError_t launch_maxpool_bwd(const PoolArgs& a, const uint8_t* idx, const h16* dy, h16* dx,
                              hipStream_t st);
// BN forward (batch statistics unless use_stats, ReLU, no shortcut) whose
// output goes straight into a 3x3 max pool (bn.hip): y and idx as
// launch_maxpool_fwd on the BN output, which is not written.  bn_maxpool_ok
// says whether the pair is taken (NHWC, the BN's vectorised path, 3x3 window
// over the BN's tensor).
bool bn_maxpool_ok(const BnArgs& a, const PoolArgs& pa);
hipError_t launch_bn_fwd_maxpool(const BnArgs& a, const PoolArgs& pa, const h16* x,
                                 const h16* gamma, const h16* beta, float* stats, int use_stats,
                                 void* ws, h16* y, uint8_t* idx, hipStream_t st);
hipError_t launch_avgpool_fwd(const PoolArgs& a, const h16* x, h16* y, hipStream_t st);
hipError_t launch_avgpool_bwd(const PoolArgs& a, const h16* dy, h16* dx, hipStream_t st);

// ---- classifier bias and loss (loss.hip) -------------------------------------
hipError_t launch_softmax_ce(int N, int K, const h16* z, const h16* bias, const int32_t* labels,
                             float* loss, h16* dz, h16* dbias, hipStream_t st);

}  // namespace fp16k
