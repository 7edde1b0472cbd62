// Declarations of the HIP kernels' host launchers (internal to libhs).
#pragma once

#include "common.h"

namespace hs {

enum { MODE_FWD = 0, MODE_DGRAD = 1, MODE_WGRAD = 2 };

// Workers of one grouped launch: the batch is split into consecutive
// segments, worker s owning samples [n0[s], n0[s + 1]).
constexpr int MAX_SEG = 16;
struct Segs {
  int count;
  int n0[MAX_SEG + 1];
};

// Rows of an NHWC tensor by segment, and the blocks of a row-parallel launch
// given to each segment: segment s owns rows [row[s], row[s + 1]) and blocks
// [blk[s], blk[s + 1]).
struct SegRows {
  int count;
  int blk[MAX_SEG + 1];
  int64_t row[MAX_SEG + 1];
};
// rows_per_sample rows per sample; blocks of at least min_rows rows (and at
// most max_blocks blocks in all, at least one per segment)
SegRows seg_rows(const Segs& sg, int64_t rows_per_sample, int64_t min_rows, int max_blocks);

// Arguments of one implicit-GEMM launch (see igemm.hip for the three modes).
struct GemmParams {
  const void* a;        // FWD: x;  DGRAD: dy;  WGRAD: dy
  const void* b;        // FWD: W;  DGRAD: W;   WGRAD: x
  void* out;            // FWD/DGRAD: [M][N] activation;  WGRAD: fp32 [M][N] (per split)
  const float* bias;    // FWD: [N] added to the output, or null
  const void* addend;   // DGRAD: [M][N] (activation type) added to the output, or null
  const void* mask;     // [M][N] (activation type): output zeroed where mask <= 0, or null
  // the same mask as bits, 1 per element: bit e of byte (m N + n) / 8 is
  // [mask[m][n + e] > 0] (N % 8 == 0).  Read instead of mask by the bf16
  // data-gradient epilogues that stage 8 channels per lane; null: none
  const uint8_t* mbits;
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
  // ... and, with a2 set, class 0 (even h, even w) adds one more term: the
  // data gradient of a 1x1 stride-2 convolution of the same input with
  // weights b2 ([K][C]) applied to a2 ([n][Hh][Wh][K], the grid of a): the
  // projection shortcut of a residual block, summed in the same reduction
  const void* a2;
  const void* b2;
  // WGRAD over worker segments: split blockIdx.y belongs to segment s when
  // seg_split[s] <= y < seg_split[s + 1]; segment s reduces over the pixels of
  // its samples seg_n0[s] .. seg_n0[s + 1] - 1, and every split writes its own
  // partial output (out + y * split_stride).  nseg = 0: the whole K range,
  // splits of kt_per_split K tiles.
  int nseg;
  int seg_split[MAX_SEG + 1];
  int seg_n0[MAX_SEG + 1];
  // Batch-norm forward sums of the output, taken in the epilogue (conv64
  // forward and the conv2 / conv2s2f patch-form forwards; null: none), per
  // segment s (samples seg_n0[s] .. seg_n0[s + 1] - 1, nseg segments):
  // stat_part[(slot * 2 + k) * N + n] = sum over a part of the output rows of
  // s of y^(k + 1), y the stored (rounded) output, at the slots of s:
  //   conv64: slot s * blocks + b, block b's rows (zero where b has none);
  //   conv2, conv2s2f: slot t + s, row tile t's rows, and a zero at slot
  //     t + s + 1 when tile t + 1 starts segment s + 1 (conv2_stat_slots,
  //     conv2s2f_stat_slots).
  // Either way segment s's partials are the slots [blk[s], blk[s + 1]).
  // A conv2 data gradient with bz set ([M][N] bf16: the input z of the batch
  // norm whose output gradient this data gradient is) writes instead, at the
  // same conv2 slots, the backward sums of the stored (rounded) output d:
  // k = 0 sum d, k = 1 sum d z (conv2_bsum_ok).
  float* stat_part;
  const void* bz;
};

// K range of weight-gradient split y (default blockIdx.y) over worker segments: the
// pixels [koff, kend) of its segment, and K tiles [kt0, kt1) of bke pixels
// counted from koff.  Table indices are compile-time constants.
__device__ inline void wgrad_split_range(const GemmParams& p, int bke, int& koff, int& kend,
                                         int& kt0, int& kt1, int y) {
  int s = 0;
#pragma unroll
  for (int i = 1; i < MAX_SEG; ++i) s += (i < p.nseg && y >= p.seg_split[i]) ? 1 : 0;
  int sp = 0, a = 0, b = 0;
#pragma unroll
  for (int i = 0; i < MAX_SEG; ++i)
    if (i == s) {
      sp = p.seg_split[i];
      a = p.seg_n0[i];
      b = p.seg_n0[i + 1];
    }
  const int hw = p.g.Ho * p.g.Wo;
  koff = a * hw;
  kend = b * hw;
  kt0 = (y - sp) * p.kt_per_split;
  const int nkt = (kend - koff + bke - 1) / bke;
  kt1 = kt0 + p.kt_per_split < nkt ? kt0 + p.kt_per_split : nkt;
}
__device__ inline void wgrad_split_range(const GemmParams& p, int bke, int& koff, int& kend,
                                         int& kt0, int& kt1) {
  wgrad_split_range(p, bke, koff, kend, kt0, kt1, (int)blockIdx.y);
}

hipError_t launch_igemm(int mode, bool bf16, const GemmParams& p, bool veca, bool vecb, int bm,
                        int bn, int splits, hipStream_t s);
// fast-path kernel (igemm_fast.hip): tiles 128x128, 128x64, 64x128, 256x64, 64x256
bool igemm_fast_ok(int mode, bool bf16, const GemmParams& p, int bm, int bn);
hipError_t launch_igemm_fast(int mode, bool bf16, const GemmParams& p, int bm, int bn, int splits,
                             hipStream_t s);
// bf16 forward / stride-1 data gradient on the 32x32x16 MFMA (conv2.hip):
// 8 waves, 512-row tiles, 16-channel slices with every tap per slice.
// p.b must hold the weights packed by launch_pack_weights for the same mode
// and shape (conv2_packed_elems bf16 elements).
bool conv2_ok(int mode, const GemmParams& p);
int conv2_bn(int N);
int64_t conv2_packed_elems(const GemmParams& p, int mode);
hipError_t launch_pack_weights(const void* W, void* Bp, int mode, const GemmParams& p,
                               hipStream_t s);
hipError_t launch_conv2(int mode, const GemmParams& p, hipStream_t s);
// Whether the conv2 forward can take the batch-norm sums of its output
// (p.stat_part with nseg / seg_n0 set): the patch form, 128-channel column
// tiles, no bias or ReLU, images of a multiple of 16 pixels, nonempty
// segments covering the batch.  conv2_stat_slots fills blk[0 .. nseg] (the
// slot range of each segment) and returns the number of slots.
bool conv2_stats_ok(const GemmParams& p);
int conv2_stat_slots(const GemmParams& p, int* blk);
// Whether the conv2 stride-1 data gradient can take the backward sums of a
// batch norm (p.stat_part, p.bz, nseg / seg_n0 set): the patch form,
// 128-channel column tiles, bf16, images of a multiple of 16 pixels,
// nonempty segments covering the batch; slots as conv2_stat_slots.
bool conv2_bsum_ok(const GemmParams& p);
// Up to PACK_BATCH packings (launch_pack_weights of theta_bf16 + woff into
// Bp + dst, offsets in elements) in one launch, passed by value.
struct PackJob {
  int64_t woff, dst;
  int N, RS, C, transpose;
};
constexpr int PACK_BATCH = 64;
struct PackBatch {
  PackJob job[PACK_BATCH];
  int count;
};
PackJob pack_job(int64_t woff, int64_t dst, int mode, const GemmParams& p);
hipError_t launch_pack_batch(const void* W, void* Bp, const PackBatch& b, hipStream_t s);
// Data gradient of a 3x3 stride-2 pad-1 convolution on the same packed
// weights (conv2.hip, "stride-2 patch form"): p.a = dy [n][Ho][Wo][K], p.out =
// dx [n][2Ho][2Wo][C] bf16 with the mask bits p.mbits (and p.addend) applied;
// with p.a2 / p.b2 (packed 1x1 weights) the shortcut's data gradient is added.
bool conv2s2_ok(const GemmParams& p);
hipError_t launch_conv2s2(const GemmParams& p, hipStream_t s);
// Forward of a 3x3 stride-2 pad-1 convolution in the patch form (conv2.hip):
// p.a = x [n][2Ho][2Wo][C], p.b = weights packed for MODE_FWD, p.out = y
// [n][Ho][Wo][K] bf16, no epilogue operations other than the batch-norm sums
// (p.stat_part with nseg / seg_n0 set; output images of a multiple of 8
// pixels, nonempty segments covering the batch: conv2s2f_stats_ok), whose
// slot ranges conv2s2f_stat_slots gives as conv2_stat_slots does.
bool conv2s2f_ok(const GemmParams& p);
hipError_t launch_conv2s2f(const GemmParams& p, hipStream_t s);
bool conv2s2f_stats_ok(const GemmParams& p);
int conv2s2f_stat_slots(const GemmParams& p, int* blk);
// bf16 forward / data gradient of 64 -> 64 channel 3x3 stride-1 layers on
// 32-wide maps (conv64.hip): packed weights resident in LDS, input patch of 16
// output rows staged once per tile, taps as shifted LDS reads
bool conv64_ok(int mode, const GemmParams& p);
// blocks of a conv64 launch (one per CU, at most one per tile)
int conv64_blocks(const GemmParams& p);
hipError_t launch_conv64(int mode, const GemmParams& p, hipStream_t s);
// bf16 weight gradient of 3x3 pad-1 layers, stride 1 or 2 (wgrad3.hip): the
// input patch of a slice of output pixels staged once in LDS (stride 2: as
// four parity planes), the 9 taps as shifted transposing reads.  kt_per_split counts slices (wgrad3_slices per
// worker segment); the split table (nseg, seg_split, seg_n0) is the caller's;
// out / split_stride as WGRAD.
bool wgrad3_ok(const GemmParams& p);
int wgrad3_slices(const GemmParams& p, int nimg);
hipError_t launch_wgrad3(const GemmParams& p, hipStream_t s);
// NCHW fp32 [n][c][hw] -> NHWC [n][hw][cp] (activation type), channels c..cp-1 zero
// The CIFAR stem in bf16 (stem.hip): 3 -> 64 channels, 3x3, stride 1, pad 1,
// 32x32, from the caller's fp32 NCHW batch x [n][3][32][32] and bf16 weights
// [64][3][3][3]; writes y [n][32][32][64] bf16 and, when x8 is not null, the
// input rounded to bf16 in NHWC with 8 channels (3 real, 5 zero).
bool stem_ok(int cin, int cout, int k, int stride, int pad, int H, int W);
// stat_part (or null): per image b, the batch-norm sums of its stored output,
// stat_part[(b * 2 + k) * 64 + c] = sum over its pixels of y[c]^(k + 1)
hipError_t launch_stem_fwd(const float* x, const void* w_bf16, void* y, void* x8, int n,
                           hipStream_t s, float* stat_part = nullptr);
// The stem's weight gradient in bf16 (stem.hip), split-K per worker segment:
// stem_wgrad_splits fills seg_split (blocks of each segment) from the
// segments' sample counts and returns the split count; launch_stem_wgrad
// writes split y's partial gW [64][27] (fp32) at part + 1728 y, from x (fp32
// NCHW) and dy [n][32][32][64] bf16.  With bn set, dy is the gradient of the
// stem's batch-norm output instead, and the kernel forms the batch-norm
// backward itself as it reads dy (the stem's dz is used nowhere else):
//   d = dy [act > 0] (act may be null), xh = (z - mean_s) rstd_s,
//   dz = gamma rstd_s (d - (sum0_s / rows_s + xh sum1_s / rows_s)), rounded
//   to bf16, with segment s's statistics and its sums of d and d xh
//   (sum0_s, sum1_s), rows_s = 1024 x its samples.
struct StemBnBwd {
  const void* z;                // [n][32][32][64] bf16, the stem convolution's output
  const void* act;              // [n][32][32][64] bf16 or null
  const float* mean;            // segment s at mean + s * mstride
  const float* rstd;
  int mstride;
  const float* gamma;           // [64]
  const float* sum0[MAX_SEG];   // [64] per segment
  const float* sum1[MAX_SEG];
};
int stem_wgrad_splits(const int* n, int nseg, int* seg_split);
hipError_t launch_stem_wgrad(const float* x, const void* dy, float* part, const int* seg_n0,
                             const int* seg_split, int nseg, hipStream_t s,
                             const StemBnBwd* bn = nullptr);
hipError_t launch_nchw_to_nhwc_pad(const float* x, void* y, int n, int c, int cp, int hw, bool bf16,
                                   hipStream_t s);
// weights [k][rs][c] fp32 -> [k][rs][cp] activation type, zero padded
hipError_t launch_pad_weights(const float* w, void* wp, int k, int rs, int c, int cp, bool bf16,
                              hipStream_t s);
// Per-segment split-K reduction: out[s][i] = sum of part[y * stride + i] over
// the splits y of segment s (split0[s] <= y < split0[s + 1]), in split order.
// With cp > c the partial rows are [rows][cp] and the output drops the
// padded columns: out[s][q * c + ch] = sum part[y * stride + q * cp + ch].
hipError_t launch_splitk_reduce_seg(const float* part, int64_t stride, int64_t count,
                                    const int* split0, float* const* out, int nseg, int c, int cp,
                                    hipStream_t s);
// The same reduction weighted over the segments into one output:
// out[i] = w[0] g_0[i], then out[i] = fma(w[s], g_s[i], out[i]) in segment
// order (the arithmetic of the weighted average kernel), where
// g_s[i] is segment s's sum exactly as launch_splitk_reduce_seg forms it (the
// arithmetic of the weighted average of separately stored g_s).
hipError_t launch_splitk_reduce_wsum(const float* part, int64_t stride, int64_t count,
                                     const int* split0, const float* w, float* out, int nseg,
                                     int c, int cp, hipStream_t s);

// ---- attainable MFMA rate (probe.hip): blocks x 512 threads, each wave
// iters x 8 dense 32x32x16 bf16 MFMAs; out[blocks * 512]
hipError_t launch_mfma_loop(int blocks, int iters, float* out, hipStream_t s);
// plain device copy of `bytes` (a multiple of 16; 16-byte aligned pointers)
hipError_t launch_copy(const void* src, void* dst, int64_t bytes, hipStream_t s);

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
// softmax cross-entropy per segment over rows of `classes` logits (fp32):
// loss[s] = mean over the segment's rows (loss may be null), dz = (softmax -
// onehot) / n_s as fp32 (dz32, may be null) and as activation type (dzt, may
// be null)
hipError_t launch_softmax_ce(const float* logits, const int32_t* labels, const Segs& sg,
                             int classes, float* loss, float* dz32, void* dzt, bool bf16,
                             hipStream_t s);
// Per-channel statistics of the rows of every segment (stats.hip), two
// launches (block partials, then a per-segment finish):
//   kind 0: out0[s] = mean, out1[s] = 1/sqrt(var + eps) of x
//   kind 1: out0[s] = sum d, out1[s] = sum d * (x - mean_s) * rstd_s,
//           d = dy * [act > 0], mean_s = mean + s * mstride (rstd likewise)
//   kind 2: out0[s] = sum d
// part: float scratch [STAT_MAX_BLOCKS][2][C].
constexpr int STAT_MAX_BLOCKS = 1024;
// The finish alone, on block partials written elsewhere (GemmParams::
// stat_part): segment s sums partials [s * blocks, (s + 1) * blocks) (with
// seg_blk: [seg_blk[s], seg_blk[s + 1])) of unshifted kind-0 sums over
// rows_per_sample rows per sample.
hipError_t launch_stats_finish_fwd(bool bf16, const float* part, int blocks, const Segs& sg,
                                   int64_t rows_per_sample, int C, float* const* mean,
                                   float* const* rstd, float eps, hipStream_t s,
                                   const int* seg_blk = nullptr);
// Optional weighted sum over the segments of kinds 1 and 2 (the partition-
// weighted gradient): sum0[c] = w[0] out0[0][c] + w[1] out0[1][c] + ... in
// segment order (sum1 likewise from out1), the per-segment outputs still
// written.
struct StatWsum {
  float* sum0;
  float* sum1;
  float w[MAX_SEG];
};
hipError_t launch_chan_stats(int kind, bool bf16, const void* x, const void* dy, const void* act,
                             const float* mean, const float* rstd, int mstride, const Segs& sg,
                             int64_t rows_per_sample, int C, float* part, float* const* out0,
                             float* const* out1, float eps, hipStream_t s,
                             const StatWsum* wsum = nullptr);
// The backward finish alone, on partials of (sum d, sum d z) per segment
// written elsewhere (GemmParams::bz): segment s sums partials [seg_blk[s],
// seg_blk[s + 1]) in double and writes out0[s] = sum d, out1[s] = rstd_s
// (sum d z - mean_s sum d) = sum d (z - mean_s) rstd_s (kind 1's outputs),
// mean_s = mean + s * mstride (rstd likewise); with wsum, also their
// weighted sums as launch_chan_stats.
hipError_t launch_stats_finish_bwd(const float* part, const Segs& sg, int C, const float* mean,
                                   const float* rstd, int mstride, float* const* out0,
                                   float* const* out1, hipStream_t s, const int* seg_blk,
                                   const StatWsum* wsum);
// vectorised (C % 8 == 0) batch-norm apply / backward by segment: segment s
// normalises with mean + s * mstride, rstd + s * mstride; the backward takes
// its sums from sum_dy[s], sum_dyx[s]
// ybits: also [y > 0] of every stored element as bits ([rows][C / 8] bytes,
// the layout of GemmParams::mbits), or null
hipError_t launch_bn_apply8(bool bf16, const void* z, const float* mean, const float* rstd,
                            int mstride, const float* gamma, const float* beta, const void* res,
                            int relu, const Segs& sg, int64_t rows_per_sample, int C, void* y,
                            hipStream_t s, uint8_t* ybits = nullptr);
hipError_t launch_bn_backward8(bool bf16, const void* dy, const void* act, const void* z,
                               const float* mean, const float* rstd, int mstride,
                               const float* gamma, float* const* sum_dy, float* const* sum_dyx,
                               const Segs& sg, int64_t rows_per_sample, int C, void* dz,
                               hipStream_t s);
// zero a list of [begin, end) element ranges of each of nbuf float buffers
hipError_t launch_zero_ranges(float* const* bufs, int nbuf, const int64_t* ranges, int count,
                              hipStream_t s);
// the same with the ranges read from host memory and passed by value in the
// kernel arguments (no device copy of the list)
hipError_t launch_zero_ranges_host(float* const* bufs, int nbuf, const int64_t* ranges, int count,
                                   hipStream_t s);

// ---- optimizer kernels (opt.hip) ----
hipError_t launch_wavg_sgd(const float* const* g, const float* w, int M, float* theta, float* mom,
                           float* gout, int64_t P, float lr, float mu, float wd,
                           uint16_t* theta_bf16, int mode, hipStream_t s);
hipError_t launch_to_bf16(const float* x, uint16_t* y, int64_t P, hipStream_t s);

}  // namespace hs
