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
};

hipError_t launch_igemm(int mode, bool bf16, const GemmParams& p, bool veca, bool vecb, int bm,
                        int bn, int splits, hipStream_t s);
hipError_t launch_splitk_reduce(const float* part, int splits, int64_t stride, int64_t count,
                                float* out, hipStream_t s);

// ---- elementwise / reduction kernels (layers.hip) ----
// NCHW fp32 input -> NHWC activation (fp32 or bf16)
hipError_t launch_nchw_to_nhwc(const float* x, void* y, int n, int c, int hw, bool bf16,
                               hipStream_t s);
// flat fp32 [n][d] -> activation type
hipError_t launch_cast_input(const float* x, void* y, int64_t count, bool bf16, hipStream_t s);

// Per-channel partial sums over rows of an NHWC tensor [rows][C]:
//   kind 0: (sum x, sum x^2)  of x                 (batch-norm statistics)
//   kind 1: (sum dy', sum dy' * xhat)               (batch-norm backward), where
//           dy' = dy * [act > 0] if act != null, xhat = (z - mean) * rstd
//   kind 2: (sum dy, -)                             (bias gradient)
// Partials are double [blocks][2][C]; `blocks` is returned by chan_blocks().
int chan_blocks(int64_t rows, int C);
hipError_t launch_chan_partials(int kind, bool bf16, const void* x, const void* dy,
                                const void* act, const float* mean, const float* rstd, int64_t rows,
                                int C, double* partial, hipStream_t s);
// Batch-norm forward finalise: mean, rstd (fp32) from the kind-0 partials.
hipError_t launch_bn_finalize(const double* partial, int blocks, int C, int64_t count, float eps,
                              float* mean, float* rstd, hipStream_t s);
// Column reduce of kind-1/2 partials: out0[c] = sum, out1[c] = second sum
// (either may be null).
hipError_t launch_chan_reduce(const double* partial, int blocks, int C, float* out0, float* out1,
                              hipStream_t s);
// y = relu?(gamma * (z - mean) * rstd + beta + res)
hipError_t launch_bn_apply(bool bf16, const void* z, const float* mean, const float* rstd,
                           const float* gamma, const float* beta, const void* res, int relu,
                           int64_t rows, int C, void* y, hipStream_t s);
// dz = gamma * rstd * (dy' - (sum_dy + xhat * sum_dyx) / count), dy' as above
hipError_t launch_bn_backward(bool bf16, const void* dy, const void* act, const void* z,
                              const float* mean, const float* rstd, const float* gamma,
                              const float* sum_dy, const float* sum_dyx, int64_t rows, int C,
                              void* dz, hipStream_t s);
// out = dy * [act > 0]
hipError_t launch_relu_mask(bool bf16, const void* dy, const void* act, int64_t count, void* out,
                            hipStream_t s);
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
// zero a list of [begin, end) element ranges of a float buffer
hipError_t launch_zero_ranges(float* buf, const int64_t* ranges, int count, hipStream_t s);

// ---- optimizer kernels (opt.hip) ----
hipError_t launch_wavg_sgd(const float* const* g, const float* w, int M, float* theta, float* mom,
                           float* gout, int64_t P, float lr, float mu, float wd,
                           uint16_t* theta_bf16, int mode, hipStream_t s);
hipError_t launch_to_bf16(const float* x, uint16_t* y, int64_t P, hipStream_t s);

}  // namespace hs
