/*
 * hs.h -- C ABI of the heterogeneous data-parallel training step on one
 * MI355X (gfx950).
 *
 * The method (arXiv 2110.08941, "Distributed Optimization using Heterogeneous
 * Compute Systems") trains one model with M synchronous workers of different
 * speeds.  Each step:
 *   1. worker m computes g_m, the gradient of its mean loss over its partition
 *      of n_m samples (Section 1, Eq. (1); Section 3)           hs_worker_grad
 *      (all M workers in one pass over the layers:             hs_workers_grad)
 *   2. the gradients are combined with partition-size weights
 *      w_m = n_m / sum n (Section 4.2, Enhanced Dynamic
 *      Partitioning)                                       hs_weighted_average
 *   3. an SGD step with momentum and weight decay (Section 1 update rule,
 *      Section 5 hyper-parameters)                                hs_sgd_step
 *      (2 and 3 fused in one pass over memory:                    hs_wavg_sgd)
 *   4. per-worker times give compute powers CP_m = n_m / X_m (Section 4,
 *      Eq. (2)), and the total batch is repartitioned in proportion to them
 *      (Section 4.1, Algorithm 1)     hs_estimate_cp, hs_repartition,
 *                                     hs_partitioner_*
 * All M workers run on one GPU; their gradient buffers are reduced in HBM.
 *
 * Conventions for every function:
 *   - Return value: HS_OK (0) or a negative hs_status; hs_last_error() gives a
 *     message for the calling thread's last failure.
 *   - Argument errors are detected before any launch and leave every buffer
 *     untouched (HS_ERR_INVALID).  A failed launch returns HS_ERR_HIP.
 *     Device work is asynchronous on `stream` (a hipStream_t, NULL = the
 *     default stream); faults inside kernels surface at the caller's next
 *     synchronisation.
 *   - Device pointers point to device memory owned by the caller, 16-byte
 *     aligned.  The library never frees or reallocates caller memory.
 *   - Model and workspace objects are owned by the library (create/destroy).
 *     All library device memory is allocated in hs_workspace_create; nothing
 *     is allocated on the step path.
 *   - A model is read-only after creation and may be shared by threads.  A
 *     workspace serves one hs_worker_grad at a time: concurrent workers need
 *     one workspace each.  A workspace also owns a second HIP stream (default
 *     priority) on which the ResNet and VGG passes run their weight gradients and
 *     projection shortcuts; a call orders all of its work before its end on
 *     the caller's stream (that stream waits for the second one), so the
 *     caller sees one stream.
 *
 * Flat parameter vector layout (theta, g_m, momentum, theta_bf16):
 *   tensors in forward order; conv weights OHWI [c_out][3][3][c_in] (1x1 for
 *   the ResNet projection); linear weights [out][in]; a layer's bias follows
 *   its weight; batch-norm stores gamma then beta; inside a residual block the
 *   order is conv1, bn1, conv2, bn2 (then conv3, bn3 in a bottleneck),
 *   projection conv, projection bn.  Every
 *   tensor starts at a multiple of 64 elements; the gaps are zero in g_m.
 *   hs_num_params() is the padded length P.
 */
#ifndef HS_H
#define HS_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  HS_OK = 0,
  HS_ERR_INVALID = -1,     /* bad argument; nothing was launched */
  HS_ERR_HIP = -2,         /* a HIP runtime call failed */
  HS_ERR_OOM = -3,         /* device allocation failed */
  HS_ERR_UNSUPPORTED = -4  /* valid request this build does not support */
} hs_status;

typedef enum { HS_MLP = 0, HS_SMALLCNN = 1, HS_RESNET18 = 2, HS_VGG16 = 3,
               HS_RESNET50 = 4 } hs_arch;
typedef enum { HS_FP32 = 0, HS_BF16 = 1 } hs_dtype;
typedef enum { HS_KIND_CONV_W = 0, HS_KIND_LIN_W = 1, HS_KIND_BIAS = 2,
               HS_KIND_BN_GAMMA = 3, HS_KIND_BN_BETA = 4 } hs_tensor_kind;

typedef struct hs_model hs_model;
typedef struct hs_workspace hs_workspace;
typedef struct hs_partitioner hs_partitioner;

/* ---------------------------------------------------------------- models -- */

/* Network description (no device memory).  arch: hs_arch; dtype: HS_FP32
 * (all GEMM operands fp32) or HS_BF16 (GEMM operands bf16 with fp32
 * accumulation; batch-norm statistics, loss, gradients and master weights
 * fp32).  The networks are CIFAR-shaped: MLP 784-256-10; small CNN
 * conv32-conv64-pool-conv128-GAP-FC10; ResNet-18 (3x3 stem, 4 stages of 2
 * basic blocks, widths 64..512); ResNet-50 (3x3 stem, stages of 3-4-6-3
 * bottleneck blocks 1x1 / 3x3 / 1x1 at inner widths 64..512 and output
 * widths 256..2048, stride 2 on the 3x3 of each later stage's first block);
 * VGG-16 (13 conv-BN-ReLU, 5 pools, FC512, FC10).  The paper's experiments
 * use ResNet50 / VGG16 on CIFAR10 (Section 5). */
hs_status hs_model_create(int32_t arch, int32_t dtype, hs_model** out);
hs_status hs_model_destroy(hs_model* model);

int64_t hs_num_params(const hs_model* model);       /* padded P, or -1 if NULL */
int64_t hs_num_true_params(const hs_model* model);  /* without padding */
int32_t hs_num_param_tensors(const hs_model* model);
/* Tensor i of the layout: offset and element count in the flat vector, shape
 * (ndim <= 4, dims[0..ndim-1]), hs_tensor_kind, and a static name string. */
hs_status hs_param_tensor(const hs_model* model, int32_t i, int64_t* offset, int64_t* numel,
                          int32_t* ndim, int64_t dims[4], int32_t* kind, const char** name);
/* Input elements per sample: 784 (MLP) or 3*32*32. */
int64_t hs_input_numel(const hs_model* model);
/* Multiply-accumulates of one forward pass of one sample (dense 3x3 taps). */
int64_t hs_forward_macs(const hs_model* model);

/* Device workspace for one worker of at most max_n samples (activations,
 * batch-norm statistics, split-K partial sums).  Allocated on the current
 * device. */
hs_status hs_workspace_create(const hs_model* model, int32_t max_n, hs_workspace** out);
hs_status hs_workspace_destroy(hs_workspace* ws);
/* Device bytes held by the workspace. */
int64_t hs_workspace_bytes(const hs_workspace* ws);
/* Streams a workspace's calls use (a measurement knob): 2 (the default) runs
 * the weight gradients and projection shortcuts of the ResNet and VGG passes
 * on the workspace's second stream, beside the caller's; 1 runs every launch
 * on the caller's stream, one kernel at a time (per-kernel timings without
 * overlap).  The arithmetic, and so every result, is the same in both.  Takes
 * effect from the next call; not to be changed while a call of this
 * workspace is being issued from another thread. */
hs_status hs_workspace_set_streams(hs_workspace* ws, int32_t streams);

/* ------------------------------------------------------- the step itself -- */

/* Worker gradient (Section 1, Eq. (1); Section 3): g_m <- gradient of
 * f_m = (1/n_m) sum_i CE(net(x_i), y_i) over the worker's n_m samples, with
 * batch-norm statistics taken over this worker's samples only.
 *   theta      device fp32 [P]
 *   theta_bf16 device bf16 [P] (the RNE copy of theta) for HS_BF16 models,
 *              must be NULL for HS_FP32 models
 *   x_m        device fp32, NCHW [n_m][3][32][32] (or [n_m][784] for the MLP)
 *   y_m        device int32 [n_m], labels 0..9
 *   n_m        1 <= n_m <= max_n of the workspace
 *   g_m        device fp32 [P], fully overwritten (padding gaps set to 0)
 *   loss_m     device fp32 scalar receiving f_m, or NULL
 * Labels outside 0..9 give an undefined loss but no out-of-bounds access. */
hs_status hs_worker_grad(const hs_model* model, hs_workspace* ws, const float* theta,
                         const uint16_t* theta_bf16, const float* x_m, const int32_t* y_m,
                         int32_t n_m, float* g_m, float* loss_m, void* stream);

/* Gradients of M workers in one pass (Section 1, Eq. (1); Section 3): the
 * same results as M calls of hs_worker_grad, with every layer launched once
 * over all M partitions.  Worker m owns rows o_m .. o_m + n[m] - 1 of x and y,
 * o_m = n[0] + ... + n[m-1]; its batch-norm statistics, mean loss and
 * gradient are its own.
 *   x, y    device, [sum n] samples laid out as for hs_worker_grad
 *   n       HOST int32 [M], each >= 1, sum n <= max_n of the workspace
 *   M       1 <= M <= 16
 *   g       HOST array of M device fp32 [P] pointers, each fully overwritten
 *   loss    device fp32 [M] receiving f_m, or NULL
 * The workspace serves the whole call (one stream). */
hs_status hs_workers_grad(const hs_model* model, hs_workspace* ws, const float* theta,
                          const uint16_t* theta_bf16, const float* x, const int32_t* y,
                          const int32_t* n, int32_t M, float* const* g, float* loss,
                          void* stream);

/* The partition-weighted gradient of M workers in one pass (Section 4.2 with
 * Section 1, Eq. (1)): g_bar = sum_m w_m g_m, w_m = n[m] / sum n, without
 * storing the g_m.  Each worker's weight-gradient partial sums (split-K over
 * its own samples) and batch-norm / bias sums are reduced per worker exactly
 * as hs_workers_grad reduces them, then combined with w_m (computed in
 * double, applied in fp32, summed in worker order) in the same reduction
 * kernel: g_bar equals, bit for bit, hs_weighted_average of the g_m that
 * hs_workers_grad writes.  One fp32 [P] vector is written instead of M, and
 * the SGD step (hs_sgd_step) reads one instead of M.  Arguments as
 * hs_workers_grad, with g_bar (device fp32 [P], fully overwritten, 16-byte
 * aligned) in place of g; loss[m] is still each worker's mean loss. */
hs_status hs_workers_grad_wavg(const hs_model* model, hs_workspace* ws, const float* theta,
                               const uint16_t* theta_bf16, const float* x, const int32_t* y,
                               const int32_t* n, int32_t M, float* g_bar, float* loss,
                               void* stream);

/* hs_workers_grad without a workspace, for callers that cannot allocate
 * device memory: code under HIP graph capture, allocation-free serving loops,
 * harnesses that forbid hipMalloc.  It calls no hipMalloc, hipFree or other
 * allocating routine; its scratch (activations, batch-norm statistics,
 * split-K partials, packed weights) is a static device buffer of
 * HS_STATIC_SCRATCH_BYTES that every GPU the library runs on holds until the
 * process ends.  Arguments, results and errors as hs_workers_grad, except:
 *   - sum n is limited by that buffer: a call whose layout needs more returns
 *     HS_ERR_INVALID, with the bytes needed in hs_last_error(), before any
 *     launch (hs_workers_grad_static_bytes gives the need: the MLP fits over
 *     5000 samples, the small CNN 62 in fp32 and 124 in bf16, ResNet-18 and
 *     VGG-16 5 in bf16, ResNet-50 bf16 none);
 *   - every launch is on `stream` (no second stream), and the split-K
 *     partial buffer is at its minimum, so the weight-gradient sums may be
 *     split differently from a workspace call (fp32 rounding differences);
 *   - all calls on one GPU share its buffer, which keeps the last call's
 *     contents (each call writes what it reads): calls that overlap on one
 *     GPU -- on different streams, or from different host threads without
 *     ordering -- race and give undefined results; serialize them. */
#define HS_STATIC_SCRATCH_BYTES (128LL << 20)
hs_status hs_workers_grad_static(const hs_model* model, const float* theta,
                                 const uint16_t* theta_bf16, const float* x, const int32_t* y,
                                 const int32_t* n, int32_t M, float* const* g, float* loss,
                                 void* stream);
/* Scratch bytes hs_workers_grad_static needs for total_n samples of the model
 * (host only), or -1 for a NULL model or total_n outside 1..16384. */
int64_t hs_workers_grad_static_bytes(const hs_model* model, int32_t total_n);

/* Partition-weighted gradient (Section 4.2):
 *   g_out[i] = sum_{m<M} w_m g[m][i],  w_m = n[m] / sum_j n[j]  (computed in
 *   double, applied in fp32, summed in worker order).
 * g: HOST array of M device pointers to fp32 [P]; n: HOST int32 [M], n[m] >= 0,
 * sum > 0; 1 <= M <= 16; P >= 0 (P = 0 is a no-op).  g_out may alias none of
 * the g[m]. */
hs_status hs_weighted_average(const float* const* g, const int32_t* n, int32_t M, int64_t P,
                              float* g_out, void* stream);

/* SGD step (Section 1 update; momentum and coupled weight decay of Section 5):
 *   d = g + wd*theta;  mom = mu*mom + d;  theta -= lr*mom
 * mom (fp32 [P]) may be NULL only when mu == 0, then theta -= lr*d.  Momentum
 * starts from zeros (the caller zero-fills it once).  If theta_bf16 is not
 * NULL it receives the round-to-nearest-even bf16 copy of the new theta. */
hs_status hs_sgd_step(float* theta, const float* g, float* mom, int64_t P, float lr, float mu,
                      float wd, uint16_t* theta_bf16, void* stream);

/* hs_weighted_average followed by hs_sgd_step in one pass over memory (the
 * weighted gradient is never stored).  Same arguments and rules as the two. */
hs_status hs_wavg_sgd(const float* const* g, const int32_t* n, int32_t M, float* theta,
                      float* mom, int64_t P, float lr, float mu, float wd,
                      uint16_t* theta_bf16, void* stream);

/* theta_bf16[i] = RNE bf16 of theta[i]. */
hs_status hs_params_to_bf16(const float* theta, uint16_t* theta_bf16, int64_t P, void* stream);

/* --------------------------------------------- compute power, repartition -- */

/* Eq. (2), Section 4: cp_out[m] = n[m] / mean_time[m] (host, double).
 * Requires n[m] >= 1 and mean_time[m] finite and > 0. */
hs_status hs_estimate_cp(const int32_t* n, const double* mean_time, int32_t M, double* cp_out);

/* Algorithm 1, Section 4.1 (host, pure, thread-safe): normalise the compute
 * powers and give worker m a partition of CP_m * N samples.  The fractional
 * sizes are rounded by largest remainder with this exact double arithmetic
 * (no fused operations):  S = sum of throughput (left to right);
 * q_m = (throughput[m] / S) * N;  f_m = floor(q_m);  the N - sum f_m workers
 * with the largest q_m - f_m get one more (ties: lower index); then, while a
 * worker has none, one sample moves from the largest worker (lowest index on
 * ties) to the lowest-index empty worker.  The even split of the first epoch
 * is throughput[m] = 1 for all m.
 * Requires 1 <= M <= N and every throughput finite and > 0. */
hs_status hs_repartition(const double* throughput, int32_t M, int32_t N, int32_t* n_out);

/* Dynamic Partitioning state across steps (Section 4.1).  Created with the
 * even split of Algorithm 1 for epoch 0.  After each step the caller reports
 * n_used[m] (the partition the step ran with: it must equal the current
 * partition, hs_partitioner_partition, else HS_ERR_INVALID and nothing
 * changes), tau[m] (the measured time of worker m's gradient, or n[m] for a
 * model clock) and speed[m] (the simulated relative speed); the worker's batch
 * time is X_m = tau[m] / speed[m].  Every `window` steps the mean X over the
 * window (summed in step order, divided by window) gives CP (Eq. (2)) and the
 * next partition (hs_repartition); *repartitioned is set to 1 on those steps
 * and cp_out (if not NULL) receives the CP vector.  A caller that launches
 * steps ahead of observing them must observe the last step of a window before
 * it reads the partition of the next step.  window = 0 never repartitions.
 * 1 <= M <= 1024, M <= N. */
hs_status hs_partitioner_create(int32_t M, int32_t N, int32_t window, hs_partitioner** out);
hs_status hs_partitioner_destroy(hs_partitioner* p);
hs_status hs_partitioner_partition(const hs_partitioner* p, int32_t* n_out);
hs_status hs_partitioner_set_partition(hs_partitioner* p, const int32_t* n);
hs_status hs_partitioner_observe(hs_partitioner* p, const int32_t* n_used, const double* tau,
                                 const double* speed, int32_t* repartitioned, double* cp_out);

/* Compute-power estimator across windows (Section 4.1: the estimate can use
 * the previous epoch only, which follows changes quickly, or a history of
 * epochs, which is steadier).  c_k is window k's estimate n / mean X
 * (Eq. (2)); the partition of window k + 1 is repartition(CP_k) with
 *   HS_CP_WINDOW  (the default):  CP_k = c_k;
 *   HS_CP_EMA:      CP_k = alpha * c_k + (1 - alpha) * CP_{k-1}, CP_0 = c_0
 *                   (0 < alpha <= 1);
 *   HS_CP_HISTORY:  CP_k = (c_{k-h+1} + ... + c_k) / h, the mean of the last
 *                   h = min(history, k + 1) estimates, summed oldest first
 *                   (1 <= history <= 1024).
 * Double arithmetic in exactly this order, no fused operations.  Setting an
 * estimator clears its history; cp_out of hs_partitioner_observe receives
 * CP_k. */
#define HS_CP_WINDOW 0
#define HS_CP_EMA 1
#define HS_CP_HISTORY 2
hs_status hs_partitioner_set_estimator(hs_partitioner* p, int32_t kind, double alpha,
                                       int32_t history);

/* Message for the calling thread's last non-OK status ("" if none). */
const char* hs_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* HS_H */
