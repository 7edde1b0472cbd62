// Network descriptions and the per-worker forward/backward schedule (host).
#pragma once

#include <string>
#include <unordered_map>
#include <vector>

#include "kernels.h"

namespace hs {

struct ParamT {
  std::string name;
  int kind;                    // hs_tensor_kind
  std::vector<int64_t> shape;
  int64_t off, numel;
};

// A convolution or a linear layer (k = 1 on a 1x1 image).  w/b are offsets
// into the flat parameter vector (b = -1: no bias).
struct ConvL {
  int cin, cout, k, stride, pad, H, W, Ho, Wo;
  int64_t w, b;
  bool relu;                   // bias + ReLU fused into the forward epilogue
};

struct BNL {
  int c;
  int64_t g, b;                // gamma, beta offsets
  int stat;                    // index of this layer's mean/rstd in the workspace
};

// Residual block: basic (c1 3x3, c2 3x3) or bottleneck (c1 1x1, c2 3x3
// carrying the stride, c3 1x1 expansion); cp/bp the projection shortcut.
struct BlockL {
  ConvL c1, c2, c3, cp;
  BNL b1, b2, b3, bp;
  bool proj, bottleneck;
};

struct VggL {
  ConvL c;
  BNL bn;
  bool pool;                   // 2x2 max-pool after the ReLU
};

struct Model {
  int arch, dtype;
  std::vector<ParamT> params;
  int64_t P = 0, P_true = 0;
  std::vector<int64_t> gaps;   // [begin, end) pairs of the padding gaps
  int64_t in_numel = 0, fwd_macs = 0;
  int nbn = 0, max_c = 0;
  int64_t max_act = 0;         // largest activation, elements per sample
  // MLP: fc1, fc2.  Small CNN: c1..c3, fc2.  ResNet-18 / ResNet-50: stem,
  // stem_bn, blocks, fc2.  VGG: vgg, fc1, fc2.
  ConvL fc1{}, fc2{}, c1{}, c2{}, c3{}, stem{};
  BNL stem_bn{};
  std::vector<BlockL> blocks;
  std::vector<VggL> vgg;
};

bool build_model(int arch, int dtype, Model& m);

// Device workspace of one worker.
struct Workspace {
  const Model* model = nullptr;
  int max_n = 0;
  char* arena = nullptr;
  int64_t bytes = 0;
  std::vector<void*> slot;     // forward activations, in plan order
  std::vector<uint8_t*> bits;  // per slot: [slot > 0] as bits (ReLU outputs read as masks), or null
  static constexpr int kGrad = 8;
  void* grad[kGrad] = {};      // gradient scratch buffers (5, or 8 for the ResNet pools)
  int ngrad = 5;
  float* logits = nullptr;
  float* dz32 = nullptr;
  void* dzt = nullptr;
  float* stats = nullptr;      // per batch-norm and worker: mean[max_c], rstd[max_c]
  void* stem_w = nullptr;      // first-layer weights, channel-padded copy
  float* stat_part = nullptr;  // per-channel statistics: block partials
  float* stat_part_side = nullptr;  // the same for statistics on the second stream
  // the batch-norm backward sums taken in data-gradient epilogues, kept until
  // their finish (no other launch writes them in between)
  float* stat_part_bsum = nullptr;
  float* splitk = nullptr;     // split-K partial outputs
  int64_t splitk_floats = 0;
  void* wpack = nullptr;       // bf16 weights packed for the 32x32 MFMA kernel
  int64_t wpack_elems = 0;
  // every layer's packed weights, one region per (layer, mode), filled on the
  // second stream at the start of a call (after the first call has listed
  // the regions): the main stream then launches no packing
  struct Pack {
    int64_t woff, dst;           // weight offset in theta; region offset (elements)
    GemmParams p;                // the contraction's shape
    int mode;
  };
  bf16_t* packed = nullptr;
  int64_t packed_cap = 0, packed_used = 0;
  std::vector<Pack> packs;
  std::unordered_map<int64_t, int> pack_of;   // (woff * 2 + mode) -> packs index
  int pack_ready = -1;         // event slot after this call's packing, -1: not packed
  bool pack_waited = false;
  float* gtmp = nullptr;       // partition-weighted mode: per-worker sums (caller's stream)
  float* gtmp_side = nullptr;  // the same for the second stream
  int64_t gtmp_c = 0;          // channels per slot
  int64_t* gaps = nullptr;     // device copy of the padding ranges
  bool gaps_by_value = false;  // zero the gaps from the model's host list instead
  // second stream for the weight gradients of the backward pass (null: all
  // work on the caller's stream) and events that order the two streams
  hipStream_t side = nullptr;
  hipStream_t side_owned = nullptr;   // the workspace's stream; side is it or null
  static constexpr int kEvents = 64;
  hipEvent_t ev[kEvents] = {};     // fork / join points (either stream)
  int ev_next = 0;
  hipEvent_t evr[kEvents] = {};    // points after second-stream reads (that stream only)
  int evr_next = 0;
  // timing probe of one GEMM instantiation (mode, tile); see hs_probe_enable
  int probe_mode = -1, probe_bm = 0, probe_bn = 0;
  std::vector<hipEvent_t> probe_ev;   // 2 per launch
  std::vector<double> probe_flops;
  size_t probe_used = 0;
};

// Lays out (ws->arena set: binds) a workspace for max_n samples; returns its
// bytes.  The split-K partial buffer holds at least splitk_min_floats floats
// (more splits, shorter weight-gradient launches) and at least one split per
// worker of the largest weight gradient.
constexpr int64_t kSplitkMinFloats = (int64_t)16 << 20;
int64_t plan_workspace(const Model& m, int max_n, Workspace* ws,
                       int64_t splitk_min_floats = kSplitkMinFloats);

// Gradients of M workers in one pass over the layers: worker s owns samples
// [o_s, o_s + n[s]) of x / y (o_s = n[0] + ... + n[s-1]); its gradient goes to
// g[s] and its mean loss to loss[s] (loss may be null).  With gbar (and the
// weights w[0..M)), g is not used: gbar receives sum_s w[s] g_s, each
// parameter's per-worker sums combined in worker order as the weighted
// average of stored g_s does.
hipError_t workers_grad(const Model& m, Workspace& ws, const float* theta,
                        const bf16_t* theta_bf16, const float* x, const int32_t* y, const int* n,
                        int M, float* const* g, float* loss, hipStream_t s,
                        float* gbar = nullptr, const float* w = nullptr);

// Address of this device's static scratch buffer (static_scratch.hip),
// HS_STATIC_SCRATCH_BYTES bytes; looked up once per device.
hipError_t static_scratch(void** ptr);

// One layer contraction (mode 0 forward, 1 data gradient, 2 weight gradient)
// with the schedule hs_worker_grad uses.
hipError_t layer_gemm(int mode, bool bf16, const ConvL& L, int n, const void* a, const void* b,
                      void* out, const float* bias, bool out_f32, float* scratch,
                      int64_t scratch_floats, hipStream_t s);

}  // namespace hs
