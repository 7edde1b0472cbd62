// Declarations of the HIP kernels' host launchers (internal to libhs).
#pragma once

#include "common.h"

namespace hs {

enum { MODE_FWD = 0, MODE_DGRAD = 1, MODE_WGRAD = 2 };

// Arguments of one implicit-GEMM launch (see igemm.hip for the three modes).
struct GemmParams {
  const void* a;        // FWD: x;  DGRAD: dy;  WGRAD: dy
  const void* b;        // FWD: W;  DGRAD: W;   WGRAD: x
  void* out;            // FWD/DGRAD: [M][N] activation;  WGRAD: fp32 [M][N] (per split)
  const float* bias;    // FWD: [N] added to the output, or null
  const void* addend;   // DGRAD: [M][N] (activation type) added to the output, or null
  const void* mask;     // [M][N] (activation type): output zeroed where mask <= 0, or null
  int relu;             // FWD: clamp the output at zero
  int out_f32;          // FWD/DGRAD: output stored as fp32 (else activation type)
  int M, N, K;
  int ktiles, kt_per_split, tiles_n;  // filled in by the launcher
  int64_t split_stride; // WGRAD: elements between the outputs of consecutive splits
  ConvGeom g;
  // DGRAD of a stride-2 layer by output parity class (fast kernel only):
  // blockIdx.z = class c = 2 * (h % 2) + (w % 2); M counts the n x Hh x Wh
  // pixels of one class; class c sums over its ntap[c] kernel taps taps[c][..]
  int par;
  int Hh, Wh;
  FastDiv HWh, Wh_;
  int ntap[4];
  int taps[4][4];
};

hipError_t launch_igemm(int mode, bool bf16, const GemmParams& p, bool veca, bool vecb, int bm,
                        int bn, int splits, hipStream_t s);
// fast-path kernel (igemm_fast.hip): tiles 128x128, 128x64, 64x128, 256x64, 64x256
bool igemm_fast_ok(int mode, bool bf16, const GemmParams& p, int bm, int bn);
hipError_t launch_igemm_fast(int mode, bool bf16, const GemmParams& p, int bm, int bn, int splits,
                             hipStream_t s);
// NCHW fp32 [n][c][hw] -> NHWC [n][hw][cp] (activation type), channels c..cp-1 zero
hipError_t launch_nchw_to_nhwc_pad(const float* x, void* y, int n, int c, int cp, int hw, bool bf16,
                                   hipStream_t s);
// weights [k][rs][c] fp32 -> [k][rs][cp] activation type, zero padded
hipError_t launch_pad_weights(const float* w, void* wp, int k, int rs, int c, int cp, bool bf16,
                              hipStream_t s);
// weight gradient [k][rs][cp] -> [k][rs][c] (drops the padded channels)
hipError_t launch_unpad_wgrad(const float* gp, float* g, int k, int rs, int c, int cp, hipStream_t s);
hipError_t launch_splitk_reduce(const float* part, int splits, int64_t stride, int64_t count,
                                float* out, hipStream_t s);

// ---- elementwise / reduction kernels (layers.hip) ----
// NCHW fp32 input -> NHWC activation (fp32 or bf16)
hipError_t launch_nchw_to_nhwc(const float* x, void* y, int n, int c, int hw, bool bf16,
                               hipStream_t s);
// flat fp32 [n][d] -> activation type
hipError_t launch_cast_input(const float* x, void* y, int64_t count, bool bf16, hipStream_t s);

// 2x2 / stride 2 max pool, NHWC
hipError_t launch_maxpool_fwd(bool bf16, const void* x, int n, int h, int w, int c, void* y,
                              hipStream_t s);
// dx: gradient of the pool routed to the first maximum of each window,
// multiplied by [x > 0] when relu_mask is set
hipError_t launch_maxpool_bwd(bool bf16, const void* x, const void* dy, int n, int h, int w, int c,
                              int relu_mask, void* dx, hipStream_t s);
// global average pool [n][hw][c] -> [n][c]; backward broadcasts dy / hw,
// masked by [act > 0] if act != null
hipError_t launch_gap_fwd(bool bf16, const void* x, int n, int hw, int c, void* y, hipStream_t s);
hipError_t launch_gap_bwd(bool bf16, const void* dy, const void* act, int n, int hw, int c,
                          void* dx, hipStream_t s);
// softmax cross-entropy over n rows of `classes` logits (fp32): loss (mean,
// may be null), dz = (softmax - onehot)/n as fp32 (dz32, may be null) and as
// activation type (dzt, may be null)
hipError_t launch_softmax_ce(const float* logits, const int32_t* labels, int n, int classes,
                             float* loss, float* dz32, void* dzt, bool bf16, hipStream_t s);
// One-launch per-channel statistics (stats.hip):
//   kind 0: out0 = mean, out1 = 1/sqrt(var + eps) of x
//   kind 1: out0 = sum d, out1 = sum d * (x - mean) * rstd, d = dy * [act > 0]
//   kind 2: out0 = sum d
// Scratch: part1 float [STAT_MAX_BLOCKS][2][C], part2 double [STAT_MAX_GROUPS][2][C],
// counters unsigned [STAT_MAX_GROUPS + 1] (zero before the first launch; left zero).
constexpr int STAT_MAX_BLOCKS = 1024;
constexpr int STAT_MAX_GROUPS = 16;
int stat_blocks(int64_t rows, int C);
hipError_t launch_chan_stats(int kind, bool bf16, const void* x, const void* dy, const void* act,
                             const float* mean, const float* rstd, int64_t rows, int C,
                             float* part1, double* part2, unsigned* counters, float* out0,
                             float* out1, float eps, hipStream_t s);
// vectorised (C % 8 == 0) batch-norm apply / backward and ReLU mask
hipError_t launch_bn_apply8(bool bf16, const void* z, const float* mean, const float* rstd,
                            const float* gamma, const float* beta, const void* res, int relu,
                            int64_t rows, int C, void* y, hipStream_t s);
hipError_t launch_bn_backward8(bool bf16, const void* dy, const void* act, const void* z,
                               const float* mean, const float* rstd, const float* gamma,
                               const float* sum_dy, const float* sum_dyx, int64_t rows, int C,
                               void* dz, hipStream_t s);
hipError_t launch_relu_mask8(bool bf16, const void* dy, const void* act, int64_t count, void* out,
                             hipStream_t s);
// zero a list of [begin, end) element ranges of a float buffer
hipError_t launch_zero_ranges(float* buf, const int64_t* ranges, int count, hipStream_t s);

// ---- optimizer kernels (opt.hip) ----
hipError_t launch_wavg_sgd(const float* const* g, const float* w, int M, float* theta, float* mom,
                           float* gout, int64_t P, float lr, float mu, float wd,
                           uint16_t* theta_bf16, int mode, hipStream_t s);
hipError_t launch_to_bf16(const float* x, uint16_t* y, int64_t P, hipStream_t s);

}  // namespace hs
