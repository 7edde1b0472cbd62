/* Measurement and test entry points of libhs: not part of the step's
 * boundary (include/hs.h), but exported by the same library and declared
 * here so that the benchmark and the tests call them through the C ABI.
 * Same conventions as hs.h (status codes, hs_last_error, device pointers). */
#ifndef HS_TESTING_H
#define HS_TESTING_H

#include "hs.h"

#ifdef __cplusplus
extern "C" {
#endif

/* ------------------------------------------------------------- probing -- */

/* Timing probe of one implicit-GEMM kernel instantiation inside
 * hs_worker_grad (for roofline reports).  While enabled, every launch of the
 * GEMM kernel with the given mode (0 forward, 1 data gradient, 2 weight
 * gradient) and output tile (bm x bn: bm 32, 64, 128, 256 or 512, bn 64, 128
 * or 256; bm = 512 selects the 32x32 MFMA forward / data-gradient kernel,
 * 64 x 64 the 64-channel patch kernels: forward / data gradient in modes 0
 * and 1, 3x3 weight gradient in mode 2; 256 x 256 in mode 1 the stride-2
 * data-gradient patch kernel, in mode 0 the stride-2 forward patch kernel
 * (256 x 128); 32 x 64 the direct bf16 stem, forward in mode 0 and weight
 * gradient in mode 2; 64 x 256 in mode 2 the stride-2 3x3 weight-gradient
 * patch kernel) on this workspace is
 * bracketed by two HIP events on the worker's stream, and its algorithmic
 * FLOPs (2 x pixels x c_out x taps x c_in, i.e. dense 3x3 taps, independent of
 * the stride handling) are added up.  At most `capacity` launches are
 * recorded (events are created here, not on the step path); later launches
 * are not timed.  mode = -1 disables the probe and releases the events. */
hs_status hs_probe_enable(hs_workspace* ws, int32_t mode, int32_t bm, int32_t bn,
                          int32_t capacity);
/* Waits for the recorded events and returns the summed kernel time (ms), the
 * number of timed launches and their summed algorithmic FLOPs, then clears
 * the record (the probe stays enabled). */
hs_status hs_probe_read(hs_workspace* ws, double* total_ms, int64_t* launches, double* flops);

/* The attainable bf16 MFMA rate, for roofline reports: launches `blocks`
 * blocks of 512 threads on `stream` (null: the default stream); each of the
 * 8 waves of a block runs iters x 8 dense 32x32x16 bf16 MFMAs on register
 * operands (2 x 32 x 32 x 16 FLOPs each), with no memory traffic but one
 * float per thread written to out (blocks x 512 floats, device): thread t
 * of a block feeds A elements (t + i) mod 8 and B elements (3 t + i) mod 8,
 * i = 0..7 of its operand registers, and writes the sum of its accumulator
 * elements.  Asynchronous; blocks 1..65536, iters 1..2^20. */
hs_status hs_probe_mfma_loop(int32_t blocks, int32_t iters, float* out, void* stream);

/* The attainable HBM rate, for roofline reports: dst[0, bytes) = src[0,
 * bytes) on `stream` by a plain copy kernel (16 bytes per lane and access).
 * bytes a positive multiple of 16, both pointers device, 16-byte aligned, the
 * ranges disjoint.  Asynchronous. */
hs_status hs_probe_copy(const void* src, void* dst, int64_t bytes, void* stream);

/* ------------------------------------------------------ layer-level access -- */

/* One contraction of a convolution or linear layer, as hs_worker_grad runs it
 * (for layer-level tests and benchmarks).  NHWC activations, OHWI weights
 * [K][R][R][C]; a linear layer is H = W = R = 1, stride 1, pad 0.
 *   mode 0 (forward):      out[n][Ho][Wo][K] = conv(a = x[n][H][W][C], b = W) (+ bias[K])
 *                          (ReLU if relu != 0)
 *   mode 1 (data grad):    out[n][H][W][C]  = gradient w.r.t. x of sum(dy * conv(x, W)),
 *                          a = dy[n][Ho][Wo][K], b = W
 *   mode 2 (weight grad):  out[K][R][R][C]  = gradient w.r.t. W, a = dy, b = x; fp32
 *                          output; split over pixels when scratch (fp32, scratch_floats
 *                          elements) is given, in one pass otherwise
 * For bf16 modes 0 and 1 with a bf16 output, a scratch buffer large enough for
 * a packed copy of the weights (K R R C bf16) selects the kernel the step
 * uses for those layers (32x32 MFMA tiles on packed weights) where the shape
 * allows it: C (mode 0) or K (mode 1) a multiple of 16, the output channel
 * count a multiple of 64, 3x3 or 1x1 filters, stride 1 for mode 1.
 * dtype selects the operand type (HS_FP32: float, HS_BF16: bf16 bits);
 * out_f32 != 0 stores modes 0/1 as fp32 even for bf16 operands.
 * Ho = (H + 2 pad - R) / stride + 1.  stride is 1 or 2.  All pointers device,
 * 16-byte aligned. */
hs_status hs_layer_gemm(int32_t mode, int32_t dtype, int32_t n, int32_t H, int32_t W, int32_t C,
                        int32_t K, int32_t R, int32_t stride, int32_t pad, const void* a,
                        const void* b, void* out, const float* bias, int32_t relu,
                        int32_t out_f32, float* scratch, int64_t scratch_floats, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* HS_TESTING_H */
