// C ABI of libhs (declared in include/hs.h; the measurement and test entry
// points in include/hs_testing.h): argument checking, object
// lifetime, and the host-side parts of the method (compute-power estimate,
// repartition, the Dynamic Partitioning window).
//
// The repartition arithmetic must not be contracted into fused operations:
// this file is compiled with -ffp-contract=off.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <new>
#include <string>
#include <vector>

#include "../../include/hs.h"
#include "../../include/hs_testing.h"
#include "model.h"

using namespace hs;

struct hs_model {
  Model m;
};

struct hs_workspace {
  const hs_model* model;
  Workspace ws;
  int device;
};

struct hs_partitioner {
  int32_t M, N, window, steps_in_window;
  std::vector<int32_t> n;
  std::vector<double> xsum;
  // compute-power estimator across windows (hs_partitioner_set_estimator)
  int32_t est_kind = HS_CP_WINDOW, est_history = 1;
  double est_alpha = 1.0;
  std::vector<double> cp_prev;                 // EMA: the previous estimate
  std::vector<std::vector<double>> cp_hist;    // HISTORY: the last windows' estimates, oldest first
};

namespace {

thread_local std::string g_err;

hs_status fail(hs_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

hs_status ok() {
  g_err.clear();
  return HS_OK;
}

hs_status hip_fail(hipError_t e, const char* what) {
  return fail(HS_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

void probe_release(Workspace& w) {
  for (hipEvent_t e : w.probe_ev) (void)hipEventDestroy(e);
  w.probe_ev.clear();
  w.probe_flops.clear();
  w.probe_used = 0;
  w.probe_mode = -1;
}

// the workspace's weight-gradient stream and events (tolerates a partial set)
void release_side(Workspace& w) {
  for (int i = 0; i < Workspace::kEvents; ++i) {
    if (w.ev[i]) {
      (void)hipEventDestroy(w.ev[i]);
      w.ev[i] = nullptr;
    }
    if (w.evr[i]) {
      (void)hipEventDestroy(w.evr[i]);
      w.evr[i] = nullptr;
    }
  }
  if (w.side_owned) {
    (void)hipStreamDestroy(w.side_owned);
    w.side_owned = nullptr;
  }
  w.side = nullptr;
}

}  // namespace

extern "C" {

const char* hs_last_error(void) { return g_err.c_str(); }

// ------------------------------------------------------------------ models --
hs_status hs_model_create(int32_t arch, int32_t dtype, hs_model** out) {
  if (!out) return fail(HS_ERR_INVALID, "hs_model_create: out is NULL");
  *out = nullptr;
  if (arch < HS_MLP || arch > HS_RESNET50) return fail(HS_ERR_INVALID, "unknown arch %d", arch);
  if (dtype != HS_FP32 && dtype != HS_BF16) return fail(HS_ERR_INVALID, "unknown dtype %d", dtype);
  hs_model* m = new (std::nothrow) hs_model;
  if (!m) return fail(HS_ERR_OOM, "host allocation failed");
  if (!build_model(arch, dtype, m->m)) {
    delete m;
    return fail(HS_ERR_UNSUPPORTED, "arch %d not supported", arch);
  }
  *out = m;
  return ok();
}

hs_status hs_model_destroy(hs_model* model) {
  delete model;
  return ok();
}

int64_t hs_num_params(const hs_model* model) { return model ? model->m.P : -1; }
int64_t hs_num_true_params(const hs_model* model) { return model ? model->m.P_true : -1; }
int32_t hs_num_param_tensors(const hs_model* model) {
  return model ? (int32_t)model->m.params.size() : -1;
}
int64_t hs_input_numel(const hs_model* model) { return model ? model->m.in_numel : -1; }
int64_t hs_forward_macs(const hs_model* model) { return model ? model->m.fwd_macs : -1; }

hs_status hs_param_tensor(const hs_model* model, int32_t i, int64_t* offset, int64_t* numel,
                          int32_t* ndim, int64_t dims[4], int32_t* kind, const char** name) {
  if (!model) return fail(HS_ERR_INVALID, "hs_param_tensor: model is NULL");
  if (i < 0 || i >= (int32_t)model->m.params.size())
    return fail(HS_ERR_INVALID, "hs_param_tensor: index %d out of range", i);
  const ParamT& p = model->m.params[i];
  if (offset) *offset = p.off;
  if (numel) *numel = p.numel;
  if (ndim) *ndim = (int32_t)p.shape.size();
  if (dims)
    for (int d = 0; d < 4; ++d) dims[d] = d < (int)p.shape.size() ? p.shape[d] : 0;
  if (kind) *kind = p.kind;
  if (name) *name = p.name.c_str();
  return ok();
}

// -------------------------------------------------------------- workspace --
hs_status hs_workspace_create(const hs_model* model, int32_t max_n, hs_workspace** out) {
  if (!out) return fail(HS_ERR_INVALID, "hs_workspace_create: out is NULL");
  *out = nullptr;
  if (!model) return fail(HS_ERR_INVALID, "hs_workspace_create: model is NULL");
  if (max_n < 1 || max_n > 16384)
    return fail(HS_ERR_INVALID, "hs_workspace_create: max_n %d outside 1..16384", max_n);
  hs_workspace* w = new (std::nothrow) hs_workspace;
  if (!w) return fail(HS_ERR_OOM, "host allocation failed");
  w->model = model;
  w->ws.model = &model->m;
  w->ws.max_n = max_n;
  (void)hipGetDevice(&w->device);
  const int64_t bytes = plan_workspace(model->m, max_n, &w->ws);
  hipError_t e = hipMalloc((void**)&w->ws.arena, (size_t)bytes);
  if (e != hipSuccess) {
    delete w;
    return fail(HS_ERR_OOM, "hipMalloc of %lld bytes: %s", (long long)bytes, hipGetErrorString(e));
  }
  w->ws.bytes = bytes;
  plan_workspace(model->m, max_n, &w->ws);
  // the weight-gradient stream (default priority) and its ordering events
  e = hipStreamCreateWithFlags(&w->ws.side_owned, hipStreamNonBlocking);
  w->ws.side = w->ws.side_owned;
  for (int i = 0; e == hipSuccess && i < Workspace::kEvents; ++i) {
    e = hipEventCreateWithFlags(&w->ws.ev[i], hipEventDisableTiming);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&w->ws.evr[i], hipEventDisableTiming);
  }
  if (e != hipSuccess) {
    release_side(w->ws);
    (void)hipFree(w->ws.arena);
    delete w;
    return hip_fail(e, "hs_workspace_create: stream/events");
  }
  const std::vector<int64_t>& gaps = model->m.gaps;
  if (!gaps.empty()) {
    e = hipMemcpy(w->ws.gaps, gaps.data(), gaps.size() * sizeof(int64_t), hipMemcpyHostToDevice);
    if (e != hipSuccess) {
      release_side(w->ws);
      (void)hipFree(w->ws.arena);
      delete w;
      return hip_fail(e, "hs_workspace_create: upload");
    }
  }
  *out = w;
  return ok();
}

hs_status hs_workspace_set_streams(hs_workspace* ws, int32_t streams) {
  if (!ws) return fail(HS_ERR_INVALID, "hs_workspace_set_streams: workspace is NULL");
  if (streams != 1 && streams != 2)
    return fail(HS_ERR_INVALID, "hs_workspace_set_streams: streams must be 1 or 2, not %d", streams);
  // the next call packs on whichever stream it runs; nothing of an earlier
  // call is pending on the second stream once that call's work is ordered
  // on the caller's stream (every call joins it before returning)
  ws->ws.side = streams == 2 ? ws->ws.side_owned : nullptr;
  return ok();
}

hs_status hs_workspace_destroy(hs_workspace* ws) {
  if (!ws) return ok();
  probe_release(ws->ws);
  release_side(ws->ws);
  if (ws->ws.arena) (void)hipFree(ws->ws.arena);
  delete ws;
  return ok();
}

int64_t hs_workspace_bytes(const hs_workspace* ws) { return ws ? ws->ws.bytes : -1; }

// ---------------------------------------------------------------- the step --
hs_status hs_worker_grad(const hs_model* model, hs_workspace* ws, const float* theta,
                         const uint16_t* theta_bf16, const float* x_m, const int32_t* y_m,
                         int32_t n_m, float* g_m, float* loss_m, void* stream) {
  if (!model || !ws) return fail(HS_ERR_INVALID, "hs_worker_grad: model/workspace is NULL");
  if (ws->model != model) return fail(HS_ERR_INVALID, "hs_worker_grad: workspace of another model");
  if (!theta || !x_m || !y_m || !g_m)
    return fail(HS_ERR_INVALID, "hs_worker_grad: theta, x_m, y_m and g_m must not be NULL");
  const bool bf = model->m.dtype == HS_BF16;
  if (bf && !theta_bf16) return fail(HS_ERR_INVALID, "hs_worker_grad: bf16 model needs theta_bf16");
  if (!bf && theta_bf16)
    return fail(HS_ERR_INVALID, "hs_worker_grad: theta_bf16 must be NULL for an fp32 model");
  if (n_m < 1 || n_m > ws->ws.max_n)
    return fail(HS_ERR_INVALID, "hs_worker_grad: n_m %d outside 1..%d", n_m, ws->ws.max_n);
  if (!aligned16(theta) || !aligned16(x_m) || !aligned16(g_m) ||
      (theta_bf16 && !aligned16(theta_bf16)))
    return fail(HS_ERR_INVALID, "hs_worker_grad: device pointers must be 16-byte aligned");
  const int n = n_m;
  float* g = g_m;
  hipError_t e = workers_grad(model->m, ws->ws, theta, theta_bf16, x_m, y_m, &n, 1, &g, loss_m,
                              (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "hs_worker_grad");
  return ok();
}

// argument checks shared by the one-pass calls: fills nn[0..M) and *total
static hs_status check_workers(const char* fn, const hs_model* model, const float* theta,
                               const uint16_t* theta_bf16, const float* x, const int32_t* y,
                               const int32_t* n, int32_t M, float* const* g, int* nn,
                               int64_t* total) {
  if (!model) return fail(HS_ERR_INVALID, "%s: model is NULL", fn);
  if (!theta || !x || !y || !n || !g)
    return fail(HS_ERR_INVALID, "%s: theta, x, y, n and g must not be NULL", fn);
  if (M < 1 || M > MAX_SEG) return fail(HS_ERR_INVALID, "%s: M %d outside 1..%d", fn, M, MAX_SEG);
  const bool bf = model->m.dtype == HS_BF16;
  if (bf && !theta_bf16) return fail(HS_ERR_INVALID, "%s: bf16 model needs theta_bf16", fn);
  if (!bf && theta_bf16)
    return fail(HS_ERR_INVALID, "%s: theta_bf16 must be NULL for an fp32 model", fn);
  *total = 0;
  for (int i = 0; i < M; ++i) {
    if (n[i] < 1) return fail(HS_ERR_INVALID, "%s: n[%d] = %d < 1", fn, i, n[i]);
    if (!g[i]) return fail(HS_ERR_INVALID, "%s: g[%d] is NULL", fn, i);
    if (!aligned16(g[i])) return fail(HS_ERR_INVALID, "%s: g[%d] must be 16-byte aligned", fn, i);
    *total += n[i];
    nn[i] = n[i];
  }
  if (!aligned16(theta) || !aligned16(x) || (theta_bf16 && !aligned16(theta_bf16)))
    return fail(HS_ERR_INVALID, "%s: device pointers must be 16-byte aligned", fn);
  return HS_OK;
}

hs_status hs_workers_grad(const hs_model* model, hs_workspace* ws, const float* theta,
                          const uint16_t* theta_bf16, const float* x, const int32_t* y,
                          const int32_t* n, int32_t M, float* const* g, float* loss,
                          void* stream) {
  if (!model || !ws) return fail(HS_ERR_INVALID, "hs_workers_grad: model/workspace is NULL");
  if (ws->model != model)
    return fail(HS_ERR_INVALID, "hs_workers_grad: workspace of another model");
  int nn[MAX_SEG];
  int64_t total = 0;
  hs_status st = check_workers("hs_workers_grad", model, theta, theta_bf16, x, y, n, M, g, nn,
                               &total);
  if (st != HS_OK) return st;
  if (total > ws->ws.max_n)
    return fail(HS_ERR_INVALID, "hs_workers_grad: sum of n = %lld exceeds the workspace's %d",
                (long long)total, ws->ws.max_n);
  hipError_t e = workers_grad(model->m, ws->ws, theta, theta_bf16, x, y, nn, M, g, loss,
                              (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "hs_workers_grad");
  return ok();
}

hs_status hs_workers_grad_wavg(const hs_model* model, hs_workspace* ws, const float* theta,
                               const uint16_t* theta_bf16, const float* x, const int32_t* y,
                               const int32_t* n, int32_t M, float* g_bar, float* loss,
                               void* stream) {
  if (!model || !ws) return fail(HS_ERR_INVALID, "hs_workers_grad_wavg: model/workspace is NULL");
  if (ws->model != model)
    return fail(HS_ERR_INVALID, "hs_workers_grad_wavg: workspace of another model");
  if (!g_bar || !aligned16(g_bar))
    return fail(HS_ERR_INVALID, "hs_workers_grad_wavg: g_bar must be a 16-byte aligned pointer");
  float* g[MAX_SEG];
  for (int i = 0; i < MAX_SEG; ++i) g[i] = g_bar;   // argument checks only
  int nn[MAX_SEG];
  int64_t total = 0;
  hs_status st = check_workers("hs_workers_grad_wavg", model, theta, theta_bf16, x, y, n, M, g,
                               nn, &total);
  if (st != HS_OK) return st;
  if (total > ws->ws.max_n)
    return fail(HS_ERR_INVALID, "hs_workers_grad_wavg: sum of n = %lld exceeds the workspace's %d",
                (long long)total, ws->ws.max_n);
  // w_m = n_m / sum n, in double, applied in fp32 (as hs_weighted_average)
  float w[MAX_SEG];
  for (int i = 0; i < M; ++i) w[i] = (float)((double)n[i] / (double)total);
  hipError_t e = workers_grad(model->m, ws->ws, theta, theta_bf16, x, y, nn, M, nullptr, loss,
                              (hipStream_t)stream, g_bar, w);
  if (e != hipSuccess) return hip_fail(e, "hs_workers_grad_wavg");
  return ok();
}

// ------------------------------------------ the allocation-free variant --
// The workspace of hs_workers_grad_static is laid out per call in the static
// device buffer of static_scratch.hip: the split-K partial buffer at its
// minimum (one split per worker of the largest weight gradient), one stream,
// the padding ranges of g zeroed from the model's host list by value.
static int64_t static_plan_bytes(const Model& m, int total) {
  Workspace w;
  return plan_workspace(m, total, &w, 0);
}

int64_t hs_workers_grad_static_bytes(const hs_model* model, int32_t total_n) {
  if (!model || total_n < 1 || total_n > 16384) return -1;
  return static_plan_bytes(model->m, total_n);
}

hs_status hs_workers_grad_static(const hs_model* model, const float* theta,
                                 const uint16_t* theta_bf16, const float* x, const int32_t* y,
                                 const int32_t* n, int32_t M, float* const* g, float* loss,
                                 void* stream) {
  int nn[MAX_SEG];
  int64_t total = 0;
  hs_status st = check_workers("hs_workers_grad_static", model, theta, theta_bf16, x, y, n, M, g,
                               nn, &total);
  if (st != HS_OK) return st;
  if (total > 16384)
    return fail(HS_ERR_INVALID, "hs_workers_grad_static: sum of n = %lld exceeds 16384",
                (long long)total);
  const int64_t need = static_plan_bytes(model->m, (int)total);
  if (need > HS_STATIC_SCRATCH_BYTES)
    return fail(HS_ERR_INVALID,
                "hs_workers_grad_static: %lld samples of this model need %lld bytes of scratch, "
                "the static buffer holds %lld (use hs_workers_grad with a workspace)",
                (long long)total, (long long)need, (long long)HS_STATIC_SCRATCH_BYTES);
  void* scratch = nullptr;
  hipError_t e = static_scratch(&scratch);
  if (e != hipSuccess) return hip_fail(e, "hs_workers_grad_static: static scratch address");
  Workspace w;
  w.model = &model->m;
  w.max_n = (int)total;
  w.arena = (char*)scratch;
  w.bytes = plan_workspace(model->m, (int)total, &w, 0);
  w.side = nullptr;
  w.gaps_by_value = true;
  e = workers_grad(model->m, w, theta, theta_bf16, x, y, nn, M, g, loss, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "hs_workers_grad_static");
  return ok();
}

static hs_status check_wavg(const float* const* g, const int32_t* n, int32_t M, int64_t P,
                            float* w) {
  if (!g || !n) return fail(HS_ERR_INVALID, "weighted average: g and n must not be NULL");
  if (M < 1 || M > 16) return fail(HS_ERR_INVALID, "weighted average: M %d outside 1..16", M);
  if (P < 0) return fail(HS_ERR_INVALID, "weighted average: P < 0");
  double total = 0.0;
  for (int m = 0; m < M; ++m) {
    if (n[m] < 0) return fail(HS_ERR_INVALID, "weighted average: n[%d] < 0", m);
    if (!g[m] && P > 0) return fail(HS_ERR_INVALID, "weighted average: g[%d] is NULL", m);
    if (!aligned16(g[m])) return fail(HS_ERR_INVALID, "weighted average: g[%d] not 16-byte aligned", m);
    total += (double)n[m];
  }
  if (!(total > 0.0)) return fail(HS_ERR_INVALID, "weighted average: sum of n must be > 0");
  for (int m = 0; m < M; ++m) w[m] = (float)((double)n[m] / total);
  return HS_OK;
}

hs_status hs_weighted_average(const float* const* g, const int32_t* n, int32_t M, int64_t P,
                              float* g_out, void* stream) {
  float w[16];
  hs_status st = check_wavg(g, n, M, P, w);
  if (st != HS_OK) return st;
  if (P == 0) return ok();
  if (!g_out || !aligned16(g_out))
    return fail(HS_ERR_INVALID, "hs_weighted_average: g_out NULL or not 16-byte aligned");
  for (int m = 0; m < M; ++m)
    if (g[m] == g_out) return fail(HS_ERR_INVALID, "hs_weighted_average: g_out aliases g[%d]", m);
  hipError_t e = launch_wavg_sgd(g, w, M, nullptr, nullptr, g_out, P, 0.f, 0.f, 0.f, nullptr, 0,
                                 (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "hs_weighted_average");
  return ok();
}

static hs_status check_sgd(float* theta, float* mom, int64_t P, float lr, float mu, float wd,
                           uint16_t* tbf) {
  if (P < 0) return fail(HS_ERR_INVALID, "sgd: P < 0");
  if (P > 0 && !theta) return fail(HS_ERR_INVALID, "sgd: theta is NULL");
  if (!mom && mu != 0.f) return fail(HS_ERR_INVALID, "sgd: momentum buffer needed when mu != 0");
  if (!isfinite(lr) || !isfinite(mu) || !isfinite(wd))
    return fail(HS_ERR_INVALID, "sgd: lr, mu, wd must be finite");
  if (!aligned16(theta) || !aligned16(mom) || !aligned16(tbf))
    return fail(HS_ERR_INVALID, "sgd: pointers must be 16-byte aligned");
  return HS_OK;
}

hs_status hs_sgd_step(float* theta, const float* g, float* mom, int64_t P, float lr, float mu,
                      float wd, uint16_t* theta_bf16, void* stream) {
  hs_status st = check_sgd(theta, mom, P, lr, mu, wd, theta_bf16);
  if (st != HS_OK) return st;
  if (P == 0) return ok();
  if (!g || !aligned16(g)) return fail(HS_ERR_INVALID, "hs_sgd_step: g NULL or not aligned");
  const float* gs[1] = {g};
  const float w[1] = {1.f};
  hipError_t e = launch_wavg_sgd(gs, w, 1, theta, mom, nullptr, P, lr, mu, wd, theta_bf16, 1,
                                 (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "hs_sgd_step");
  return ok();
}

hs_status hs_wavg_sgd(const float* const* g, const int32_t* n, int32_t M, float* theta,
                      float* mom, int64_t P, float lr, float mu, float wd, uint16_t* theta_bf16,
                      void* stream) {
  float w[16];
  hs_status st = check_wavg(g, n, M, P, w);
  if (st != HS_OK) return st;
  st = check_sgd(theta, mom, P, lr, mu, wd, theta_bf16);
  if (st != HS_OK) return st;
  if (P == 0) return ok();
  hipError_t e = launch_wavg_sgd(g, w, M, theta, mom, nullptr, P, lr, mu, wd, theta_bf16, 2,
                                 (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "hs_wavg_sgd");
  return ok();
}

hs_status hs_params_to_bf16(const float* theta, uint16_t* theta_bf16, int64_t P, void* stream) {
  if (P < 0) return fail(HS_ERR_INVALID, "hs_params_to_bf16: P < 0");
  if (P == 0) return ok();
  if (!theta || !theta_bf16) return fail(HS_ERR_INVALID, "hs_params_to_bf16: NULL pointer");
  hipError_t e = launch_to_bf16(theta, theta_bf16, P, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "hs_params_to_bf16");
  return ok();
}


hs_status hs_probe_enable(hs_workspace* ws, int32_t mode, int32_t bm, int32_t bn,
                          int32_t capacity) {
  if (!ws) return fail(HS_ERR_INVALID, "hs_probe_enable: workspace is NULL");
  probe_release(ws->ws);
  if (mode < 0) return ok();
  if (mode > 2 || (bm != 32 && bm != 64 && bm != 128 && bm != 256 && bm != 512) ||
      (bn != 64 && bn != 128 && bn != 256) || capacity < 1 || capacity > 1000000)
    return fail(HS_ERR_INVALID, "hs_probe_enable: bad mode/tile/capacity");
  ws->ws.probe_ev.resize(2 * (size_t)capacity + 1, nullptr);
  for (size_t i = 0; i < ws->ws.probe_ev.size(); ++i) {
    // timing only: no system-scope fence (no cache writeback between the
    // launches it brackets, which would add to the measured time)
    hipError_t e = hipEventCreateWithFlags(&ws->ws.probe_ev[i], hipEventDisableSystemFence);
    if (e != hipSuccess) {
      ws->ws.probe_ev.resize(i);
      probe_release(ws->ws);
      return hip_fail(e, "hs_probe_enable");
    }
  }
  ws->ws.probe_flops.assign(capacity, 0.0);
  ws->ws.probe_mode = mode;
  ws->ws.probe_bm = bm;
  ws->ws.probe_bn = bn;
  return ok();
}

hs_status hs_probe_read(hs_workspace* ws, double* total_ms, int64_t* launches, double* flops) {
  if (!ws || !total_ms || !launches || !flops) return fail(HS_ERR_INVALID, "hs_probe_read: NULL");
  Workspace& w = ws->ws;
  double t = 0.0, f = 0.0;
  for (size_t i = 0; i < w.probe_used; ++i) {
    hipError_t e = hipEventSynchronize(w.probe_ev[2 * i + 1]);
    if (e != hipSuccess) return hip_fail(e, "hs_probe_read");
    float ms = 0.f;
    e = hipEventElapsedTime(&ms, w.probe_ev[2 * i], w.probe_ev[2 * i + 1]);
    if (e != hipSuccess) return hip_fail(e, "hs_probe_read");
    t += ms;
    f += w.probe_flops[i];
  }
  *total_ms = t;
  *launches = (int64_t)w.probe_used;
  *flops = f;
  w.probe_used = 0;
  return ok();
}

hs_status hs_probe_mfma_loop(int32_t blocks, int32_t iters, float* out, void* stream) {
  if (blocks < 1 || blocks > 65536 || iters < 1 || iters > (1 << 20))
    return fail(HS_ERR_INVALID, "hs_probe_mfma_loop: blocks %d, iters %d", blocks, iters);
  if (!out) return fail(HS_ERR_INVALID, "hs_probe_mfma_loop: NULL output");
  hipError_t e = launch_mfma_loop(blocks, iters, out, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "hs_probe_mfma_loop");
  return ok();
}

hs_status hs_probe_copy(const void* src, void* dst, int64_t bytes, void* stream) {
  if (!src || !dst) return fail(HS_ERR_INVALID, "hs_probe_copy: NULL pointer");
  if (bytes < 16 || bytes % 16 != 0 || ((uintptr_t)src | (uintptr_t)dst) % 16 != 0)
    return fail(HS_ERR_INVALID, "hs_probe_copy: %lld bytes, pointers must be 16-byte aligned",
                (long long)bytes);
  const uintptr_t s0 = (uintptr_t)src, d0 = (uintptr_t)dst;
  if (s0 < d0 + (uintptr_t)bytes && d0 < s0 + (uintptr_t)bytes)
    return fail(HS_ERR_INVALID, "hs_probe_copy: overlapping ranges");
  hipError_t e = launch_copy(src, dst, bytes, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "hs_probe_copy");
  return ok();
}

hs_status hs_layer_gemm(int32_t mode, int32_t dtype, int32_t n, int32_t H, int32_t W, int32_t C,
                        int32_t K, int32_t R, int32_t stride, int32_t pad, const void* a,
                        const void* b, void* out, const float* bias, int32_t relu,
                        int32_t out_f32, float* scratch, int64_t scratch_floats, void* stream) {
  if (mode < 0 || mode > 2) return fail(HS_ERR_INVALID, "hs_layer_gemm: mode %d", mode);
  if (dtype != HS_FP32 && dtype != HS_BF16) return fail(HS_ERR_INVALID, "hs_layer_gemm: dtype");
  if (n < 1 || H < 1 || W < 1 || C < 1 || K < 1 || R < 1 || pad < 0 || (stride != 1 && stride != 2))
    return fail(HS_ERR_INVALID, "hs_layer_gemm: bad geometry");
  const int Ho = (H + 2 * pad - R) / stride + 1, Wo = (W + 2 * pad - R) / stride + 1;
  if (Ho < 1 || Wo < 1) return fail(HS_ERR_INVALID, "hs_layer_gemm: empty output");
  if ((int64_t)n * H * W * C >= (1ll << 31) || (int64_t)n * Ho * Wo * K >= (1ll << 31))
    return fail(HS_ERR_INVALID, "hs_layer_gemm: tensor too large for 32-bit indexing");
  if (!a || !b || !out) return fail(HS_ERR_INVALID, "hs_layer_gemm: NULL operand");
  if (!aligned16(a) || !aligned16(b) || !aligned16(out) || !aligned16(scratch))
    return fail(HS_ERR_INVALID, "hs_layer_gemm: pointers must be 16-byte aligned");
  if (mode == 1 && dtype == HS_BF16 && out_f32)
    return fail(HS_ERR_INVALID, "hs_layer_gemm: data gradient of bf16 operands is stored as bf16");
  ConvL L{};
  L.cin = C;
  L.cout = K;
  L.k = R;
  L.stride = stride;
  L.pad = pad;
  L.H = H;
  L.W = W;
  L.Ho = Ho;
  L.Wo = Wo;
  L.relu = relu != 0;
  hipError_t e = layer_gemm(mode, dtype == HS_BF16, L, n, a, b, out, bias, out_f32 != 0,
                            scratch, scratch_floats, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "hs_layer_gemm");
  return ok();
}

// ---------------------------------------------- compute power, repartition --
hs_status hs_estimate_cp(const int32_t* n, const double* mean_time, int32_t M, double* cp_out) {
  if (!n || !mean_time || !cp_out || M < 1)
    return fail(HS_ERR_INVALID, "hs_estimate_cp: bad arguments");
  for (int m = 0; m < M; ++m) {
    if (n[m] < 1) return fail(HS_ERR_INVALID, "hs_estimate_cp: n[%d] < 1", m);
    if (!isfinite(mean_time[m]) || !(mean_time[m] > 0.0))
      return fail(HS_ERR_INVALID, "hs_estimate_cp: mean_time[%d] not finite and > 0", m);
  }
  for (int m = 0; m < M; ++m) cp_out[m] = (double)n[m] / mean_time[m];
  return ok();
}

hs_status hs_repartition(const double* throughput, int32_t M, int32_t N, int32_t* n_out) {
  if (!throughput || !n_out) return fail(HS_ERR_INVALID, "hs_repartition: NULL pointer");
  if (M < 1 || N < M) return fail(HS_ERR_INVALID, "hs_repartition: need N >= M >= 1 (M=%d N=%d)", M, N);
  for (int m = 0; m < M; ++m)
    if (!isfinite(throughput[m]) || !(throughput[m] > 0.0))
      return fail(HS_ERR_INVALID, "hs_repartition: throughput[%d] not finite and > 0", m);
  double S = 0.0;
  for (int m = 0; m < M; ++m) S = S + throughput[m];
  std::vector<int64_t> f(M);
  std::vector<double> r(M);
  int64_t fsum = 0;
  for (int m = 0; m < M; ++m) {
    const double c = throughput[m] / S;
    const double q = c * (double)N;
    const double fl = floor(q);
    f[m] = (int64_t)fl;
    r[m] = q - fl;
    fsum += f[m];
  }
  const int64_t left = (int64_t)N - fsum;
  if (left < 0 || left > M) return fail(HS_ERR_INVALID, "hs_repartition: rounding left %lld", (long long)left);
  std::vector<int> order(M);
  for (int m = 0; m < M; ++m) order[m] = m;
  std::stable_sort(order.begin(), order.end(), [&](int a, int b) {
    if (r[a] != r[b]) return r[a] > r[b];
    return a < b;
  });
  for (int64_t i = 0; i < left; ++i) f[order[i]] += 1;
  for (;;) {
    int z = -1;
    for (int m = 0; m < M; ++m)
      if (f[m] == 0) {
        z = m;
        break;
      }
    if (z < 0) break;
    int big = 0;
    for (int m = 1; m < M; ++m)
      if (f[m] > f[big]) big = m;
    f[big] -= 1;
    f[z] += 1;
  }
  for (int m = 0; m < M; ++m) n_out[m] = (int32_t)f[m];
  return ok();
}

hs_status hs_partitioner_create(int32_t M, int32_t N, int32_t window, hs_partitioner** out) {
  if (!out) return fail(HS_ERR_INVALID, "hs_partitioner_create: out is NULL");
  *out = nullptr;
  if (M < 1 || M > 1024 || N < M || window < 0)
    return fail(HS_ERR_INVALID, "hs_partitioner_create: need 1 <= M <= 1024, M <= N, window >= 0");
  hs_partitioner* p = new (std::nothrow) hs_partitioner;
  if (!p) return fail(HS_ERR_OOM, "host allocation failed");
  p->M = M;
  p->N = N;
  p->window = window;
  p->steps_in_window = 0;
  p->n.assign(M, 0);
  p->xsum.assign(M, 0.0);
  std::vector<double> ones(M, 1.0);  // Algorithm 1, epoch 0: CP_m = 1/M
  hs_status st = hs_repartition(ones.data(), M, N, p->n.data());
  if (st != HS_OK) {
    delete p;
    return st;
  }
  *out = p;
  return ok();
}

hs_status hs_partitioner_destroy(hs_partitioner* p) {
  delete p;
  return ok();
}

hs_status hs_partitioner_partition(const hs_partitioner* p, int32_t* n_out) {
  if (!p || !n_out) return fail(HS_ERR_INVALID, "hs_partitioner_partition: NULL pointer");
  memcpy(n_out, p->n.data(), sizeof(int32_t) * p->M);
  return ok();
}

hs_status hs_partitioner_set_partition(hs_partitioner* p, const int32_t* n) {
  if (!p || !n) return fail(HS_ERR_INVALID, "hs_partitioner_set_partition: NULL pointer");
  int64_t s = 0;
  for (int m = 0; m < p->M; ++m) {
    if (n[m] < 1) return fail(HS_ERR_INVALID, "hs_partitioner_set_partition: n[%d] < 1", m);
    s += n[m];
  }
  if (s != p->N) return fail(HS_ERR_INVALID, "hs_partitioner_set_partition: sum != N");
  memcpy(p->n.data(), n, sizeof(int32_t) * p->M);
  return ok();
}

hs_status hs_partitioner_set_estimator(hs_partitioner* p, int32_t kind, double alpha,
                                       int32_t history) {
  if (!p) return fail(HS_ERR_INVALID, "hs_partitioner_set_estimator: NULL pointer");
  if (kind != HS_CP_WINDOW && kind != HS_CP_EMA && kind != HS_CP_HISTORY)
    return fail(HS_ERR_INVALID, "hs_partitioner_set_estimator: unknown kind %d", kind);
  if (kind == HS_CP_EMA && !(alpha > 0.0 && alpha <= 1.0))
    return fail(HS_ERR_INVALID, "hs_partitioner_set_estimator: need 0 < alpha <= 1");
  if (kind == HS_CP_HISTORY && (history < 1 || history > 1024))
    return fail(HS_ERR_INVALID, "hs_partitioner_set_estimator: need 1 <= history <= 1024");
  p->est_kind = kind;
  p->est_alpha = alpha;
  p->est_history = history;
  p->cp_prev.clear();
  p->cp_hist.clear();
  return ok();
}

hs_status hs_partitioner_observe(hs_partitioner* p, const int32_t* n_used, const double* tau,
                                 const double* speed, int32_t* repartitioned, double* cp_out) {
  if (!p || !n_used || !tau || !speed)
    return fail(HS_ERR_INVALID, "hs_partitioner_observe: NULL pointer");
  // the observation must belong to the window being measured: a step run
  // with another partition (one started before the last repartition was
  // observed) would mix two partitions in one compute-power estimate
  for (int m = 0; m < p->M; ++m)
    if (n_used[m] != p->n[m])
      return fail(HS_ERR_INVALID,
                  "hs_partitioner_observe: the step ran with n[%d] = %d, the current partition "
                  "has %d (observe every step of a window before starting the next window)",
                  m, n_used[m], p->n[m]);
  for (int m = 0; m < p->M; ++m) {
    if (!isfinite(tau[m]) || !(tau[m] > 0.0) || !isfinite(speed[m]) || !(speed[m] > 0.0))
      return fail(HS_ERR_INVALID, "hs_partitioner_observe: tau/speed[%d] not finite and > 0", m);
  }
  if (repartitioned) *repartitioned = 0;
  for (int m = 0; m < p->M; ++m) p->xsum[m] = p->xsum[m] + tau[m] / speed[m];
  p->steps_in_window += 1;
  if (p->window == 0 || p->steps_in_window < p->window) return ok();
  std::vector<double> xbar(p->M), cp(p->M);
  for (int m = 0; m < p->M; ++m) xbar[m] = p->xsum[m] / (double)p->window;
  hs_status st = hs_estimate_cp(p->n.data(), xbar.data(), p->M, cp.data());
  if (st != HS_OK) return st;
  // smoothing across windows (Section 4.1: the previous epoch only, or a
  // history of epochs); every operation in this order, no fused ones
  if (p->est_kind == HS_CP_EMA) {
    if (!p->cp_prev.empty())
      for (int m = 0; m < p->M; ++m) cp[m] = p->est_alpha * cp[m] + (1.0 - p->est_alpha) * p->cp_prev[m];
    p->cp_prev = cp;
  } else if (p->est_kind == HS_CP_HISTORY) {
    p->cp_hist.push_back(cp);
    if ((int32_t)p->cp_hist.size() > p->est_history) p->cp_hist.erase(p->cp_hist.begin());
    for (int m = 0; m < p->M; ++m) {
      double sum = 0.0;
      for (const std::vector<double>& h : p->cp_hist) sum = sum + h[m];
      cp[m] = sum / (double)p->cp_hist.size();
    }
  }
  std::vector<int32_t> next(p->M);
  st = hs_repartition(cp.data(), p->M, p->N, next.data());
  if (st != HS_OK) return st;
  p->n = next;
  p->steps_in_window = 0;
  std::fill(p->xsum.begin(), p->xsum.end(), 0.0);
  if (repartitioned) *repartitioned = 1;
  if (cp_out) memcpy(cp_out, cp.data(), sizeof(double) * p->M);
  return ok();
}

}  // extern "C"
