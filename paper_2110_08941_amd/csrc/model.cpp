// Network descriptions, workspace plan and the per-worker forward/backward
// launch schedule.
//
// The worker gradient is g_m = grad of the mean softmax cross-entropy over the
// worker's samples (Eq. (1) of the paper with the expectation over the
// worker's partition), batch-norm statistics taken over the worker's own
// samples.  Every contraction runs on the implicit-GEMM MFMA kernel; the
// remaining layers are the bandwidth-bound kernels of layers.hip.
#include "model.h"

#include "../../include/hs.h"

namespace hs {

// Target block counts of the weight-gradient launches (split-K over pixels):
// about this many blocks per launch of the 3x3 patch kernel and of the fast
// kernel, and at most this many splits of the fast kernel's reduction (its
// per-worker reduce sums the splits of an output in sequence).
#ifndef HS_WGRAD3_BLOCKS
#define HS_WGRAD3_BLOCKS 512
#endif
#ifndef HS_WGRAD_FAST_TILES
#define HS_WGRAD_FAST_TILES 1024
#endif
#ifndef HS_WGRAD_FAST_MAX_SPLITS
#define HS_WGRAD_FAST_MAX_SPLITS 256
#endif
constexpr int kWgrad3Blocks = HS_WGRAD3_BLOCKS;
constexpr int kWgradFastMaxSplits = HS_WGRAD_FAST_MAX_SPLITS;
constexpr int kWgradFastTiles = HS_WGRAD_FAST_TILES;

// ----------------------------------------------------------------------------
// model construction
// ----------------------------------------------------------------------------
namespace {

struct Builder {
  Model& m;
  explicit Builder(Model& mm) : m(mm) {}

  int64_t add(const std::string& name, int kind, std::vector<int64_t> shape) {
    int64_t numel = 1;
    for (int64_t d : shape) numel *= d;
    int64_t off = (m.P + 63) / 64 * 64;
    if (off > m.P) {
      m.gaps.push_back(m.P);
      m.gaps.push_back(off);
    }
    m.params.push_back({name, kind, shape, off, numel});
    m.P = off + numel;
    m.P_true += numel;
    return off;
  }

  ConvL conv(const std::string& name, int cin, int cout, int k, int stride, int pad, int H, int W,
             bool bias, bool relu) {
    ConvL c;
    c.cin = cin;
    c.cout = cout;
    c.k = k;
    c.stride = stride;
    c.pad = pad;
    c.H = H;
    c.W = W;
    c.Ho = (H + 2 * pad - k) / stride + 1;
    c.Wo = (W + 2 * pad - k) / stride + 1;
    c.w = add(name + ".weight", HS_KIND_CONV_W, {cout, k, k, cin});
    c.b = bias ? add(name + ".bias", HS_KIND_BIAS, {cout}) : -1;
    c.relu = relu;
    m.fwd_macs += (int64_t)c.Ho * c.Wo * cout * k * k * cin;
    note_act((int64_t)c.Ho * c.Wo * cout);
    note_act((int64_t)H * W * cin);
    return c;
  }

  ConvL linear(const std::string& name, int fin, int fout, bool relu) {
    ConvL c;
    c.cin = fin;
    c.cout = fout;
    c.k = 1;
    c.stride = 1;
    c.pad = 0;
    c.H = c.W = c.Ho = c.Wo = 1;
    c.w = add(name + ".weight", HS_KIND_LIN_W, {fout, fin});
    c.b = add(name + ".bias", HS_KIND_BIAS, {fout});
    c.relu = relu;
    m.fwd_macs += (int64_t)fin * fout;
    note_act(fin);
    note_act(fout);
    return c;
  }

  BNL bn(const std::string& name, int c) {
    BNL b;
    b.c = c;
    b.g = add(name + ".gamma", HS_KIND_BN_GAMMA, {c});
    b.b = add(name + ".beta", HS_KIND_BN_BETA, {c});
    b.stat = m.nbn++;
    if (c > m.max_c) m.max_c = c;
    return b;
  }

  void note_act(int64_t e) {
    if (e > m.max_act) m.max_act = e;
  }
};

}  // namespace

bool build_model(int arch, int dtype, Model& m) {
  m = Model();
  m.arch = arch;
  m.dtype = dtype;
  Builder b(m);
  if (arch == HS_MLP) {
    m.in_numel = 784;
    m.fc1 = b.linear("fc1", 784, 256, true);
    m.fc2 = b.linear("fc2", 256, 10, false);
  } else if (arch == HS_SMALLCNN) {
    m.in_numel = 3 * 32 * 32;
    m.c1 = b.conv("conv1", 3, 32, 3, 1, 1, 32, 32, true, true);
    m.c2 = b.conv("conv2", 32, 64, 3, 1, 1, 32, 32, true, true);
    m.c3 = b.conv("conv3", 64, 128, 3, 1, 1, 16, 16, true, true);
    m.fc2 = b.linear("fc", 128, 10, false);
  } else if (arch == HS_RESNET18) {
    m.in_numel = 3 * 32 * 32;
    m.stem = b.conv("stem", 3, 64, 3, 1, 1, 32, 32, false, false);
    m.stem_bn = b.bn("stem_bn", 64);
    const int widths[4] = {64, 128, 256, 512};
    int cin = 64, H = 32;
    for (int si = 0; si < 4; ++si) {
      for (int bi = 0; bi < 2; ++bi) {
        const int stride = (si > 0 && bi == 0) ? 2 : 1;
        const int w = widths[si];
        std::string nm = "layer" + std::to_string(si + 1) + "." + std::to_string(bi);
        BlockL blk{};
        blk.c1 = b.conv(nm + ".conv1", cin, w, 3, stride, 1, H, H, false, false);
        blk.b1 = b.bn(nm + ".bn1", w);
        const int Ho = blk.c1.Ho;
        blk.c2 = b.conv(nm + ".conv2", w, w, 3, 1, 1, Ho, Ho, false, false);
        blk.b2 = b.bn(nm + ".bn2", w);
        blk.proj = (stride != 1 || cin != w);
        if (blk.proj) {
          blk.cp = b.conv(nm + ".proj", cin, w, 1, stride, 0, H, H, false, false);
          blk.bp = b.bn(nm + ".proj_bn", w);
        }
        m.blocks.push_back(blk);
        cin = w;
        H = Ho;
      }
    }
    m.fc2 = b.linear("fc", 512, 10, false);
  } else if (arch == HS_RESNET50) {
    m.in_numel = 3 * 32 * 32;
    m.stem = b.conv("stem", 3, 64, 3, 1, 1, 32, 32, false, false);
    m.stem_bn = b.bn("stem_bn", 64);
    const int widths[4] = {64, 128, 256, 512}, nblocks[4] = {3, 4, 6, 3};
    int cin = 64, H = 32;
    for (int si = 0; si < 4; ++si) {
      for (int bi = 0; bi < nblocks[si]; ++bi) {
        const int stride = (si > 0 && bi == 0) ? 2 : 1;
        const int mid = widths[si], cout = 4 * widths[si];
        std::string nm = "layer" + std::to_string(si + 1) + "." + std::to_string(bi);
        BlockL blk{};
        blk.bottleneck = true;
        blk.c1 = b.conv(nm + ".conv1", cin, mid, 1, 1, 0, H, H, false, false);
        blk.b1 = b.bn(nm + ".bn1", mid);
        blk.c2 = b.conv(nm + ".conv2", mid, mid, 3, stride, 1, H, H, false, false);
        blk.b2 = b.bn(nm + ".bn2", mid);
        const int Ho = blk.c2.Ho;
        blk.c3 = b.conv(nm + ".conv3", mid, cout, 1, 1, 0, Ho, Ho, false, false);
        blk.b3 = b.bn(nm + ".bn3", cout);
        blk.proj = (stride != 1 || cin != cout);
        if (blk.proj) {
          blk.cp = b.conv(nm + ".proj", cin, cout, 1, stride, 0, H, H, false, false);
          blk.bp = b.bn(nm + ".proj_bn", cout);
        }
        m.blocks.push_back(blk);
        cin = cout;
        H = Ho;
      }
    }
    m.fc2 = b.linear("fc", 2048, 10, false);
  } else if (arch == HS_VGG16) {
    m.in_numel = 3 * 32 * 32;
    const int cfg[18] = {64, 64, -1, 128, 128, -1, 256, 256, 256, -1,
                         512, 512, 512, -1, 512, 512, 512, -1};
    int cin = 3, H = 32, idx = 0;
    for (int i = 0; i < 18; ++i) {
      if (cfg[i] < 0) {
        m.vgg.back().pool = true;
        H /= 2;
        continue;
      }
      ++idx;
      VggL l{};
      l.c = b.conv("conv" + std::to_string(idx), cin, cfg[i], 3, 1, 1, H, H, false, false);
      l.bn = b.bn("bn" + std::to_string(idx), cfg[i]);
      l.pool = false;
      m.vgg.push_back(l);
      cin = cfg[i];
    }
    m.fc1 = b.linear("fc1", 512, 512, true);
    m.fc2 = b.linear("fc2", 512, 10, false);
  } else {
    return false;
  }
  int64_t end = (m.P + 63) / 64 * 64;
  if (end > m.P) {
    m.gaps.push_back(m.P);
    m.gaps.push_back(end);
  }
  m.P = end;
  if (m.max_c < 16) m.max_c = 16;
  return true;
}

// ----------------------------------------------------------------------------
// workspace plan: the same walk sizes the arena (ws->arena == null) and
// binds the slots
// ----------------------------------------------------------------------------
namespace {
struct Bump {
  char* base;
  int64_t off = 0;
  void* take(int64_t bytes) {
    off = (off + 255) / 256 * 256;
    void* p = base ? base + off : nullptr;
    off += bytes;
    return p;
  }
};
}  // namespace

int64_t plan_workspace(const Model& m, int max_n, Workspace* ws, int64_t splitk_min_floats) {
  const int64_t es = m.dtype == HS_BF16 ? 2 : 4;
  Bump a{ws->arena};
  ws->slot.clear();
  ws->bits.clear();
  // bits: the slot is a ReLU output that data gradients read as their mask;
  // it also gets a copy of [value > 0] as bits (one byte per 8 channels)
  auto act = [&](int64_t per_sample, bool bits = false) {
    ws->slot.push_back(a.take(per_sample * max_n * es));
    ws->bits.push_back(bits ? (uint8_t*)a.take(per_sample * max_n / 8) : nullptr);
  };
  if (m.arch == HS_MLP) {
    act(784);    // 0: input in activation type
    act(256);    // 1: hidden (post ReLU)
  } else if (m.arch == HS_SMALLCNN) {
    act(8 * 1024);           // 0: X0 (NHWC, channels padded)
    act(32 * 1024);          // 1: A1
    act(64 * 1024);          // 2: A2
    act(64 * 256);           // 3: P2
    act(128 * 256);          // 4: A3
    act(128);                // 5: F
  } else if (m.arch == HS_RESNET18) {
    act(8 * 1024);           // 0: X0 (channels padded)
    act(64 * 1024);          // 1: Zs
    act(64 * 1024, true);    // 2: As
    for (const BlockL& b : m.blocks) {
      const int64_t e = (int64_t)b.c1.Ho * b.c1.Wo * b.c1.cout;
      act(e);                // Z1
      act(e, true);          // H
      act(e);                // Z2
      act(b.proj ? e : 0);   // ZP
      act(e, true);          // A_out
    }
    act(512);                // F
  } else if (m.arch == HS_RESNET50) {
    act(8 * 1024);           // 0: X0 (channels padded)
    act(64 * 1024);          // 1: Zs
    act(64 * 1024, true);    // 2: As
    for (const BlockL& b : m.blocks) {
      const int64_t ein = (int64_t)b.c1.Ho * b.c1.Wo * b.c1.cout;   // input grid, inner width
      const int64_t emid = (int64_t)b.c2.Ho * b.c2.Wo * b.c2.cout;  // output grid, inner width
      const int64_t eout = (int64_t)b.c3.Ho * b.c3.Wo * b.c3.cout;  // output grid, output width
      act(ein);              // Z1
      act(ein, true);        // H1
      act(emid);             // Z2
      act(emid, true);       // H2
      act(eout);             // Z3
      act(b.proj ? eout : 0);  // ZP
      act(eout, true);       // A_out
    }
    act(2048);               // F
  } else {
    act(8 * 1024);           // 0: X0 (channels padded)
    for (const VggL& l : m.vgg) {
      const int64_t e = (int64_t)l.c.Ho * l.c.Wo * l.c.cout;
      act(e);                // Z
      act(e);                // A
      act(l.pool ? e / 4 : 0);  // P
    }
    act(512);                // Hf (fc1 output)
  }
  // the ResNet and VGG backward passes rotate 8 buffers so that the weight-gradient
  // stream can run a block behind (see GradPool); the others use 5
  ws->ngrad = (m.arch == HS_RESNET18 || m.arch == HS_RESNET50 || m.arch == HS_VGG16)
                  ? Workspace::kGrad : 5;
  for (int i = 0; i < Workspace::kGrad; ++i)
    ws->grad[i] = i < ws->ngrad ? a.take(m.max_act * max_n * es) : nullptr;
  ws->logits = (float*)a.take((int64_t)max_n * 10 * 4);
  ws->dz32 = (float*)a.take((int64_t)max_n * 10 * 4);
  ws->dzt = a.take((int64_t)max_n * 10 * es);
  ws->stats = (float*)a.take((int64_t)(m.nbn > 0 ? m.nbn : 1) * MAX_SEG * 2 * m.max_c * 4);
  const int64_t cmax = m.max_c > 512 ? m.max_c : 512;
  ws->stem_w = a.take((int64_t)64 * 9 * 8 * es);
  ws->stat_part = (float*)a.take((int64_t)STAT_MAX_BLOCKS * 2 * cmax * 4);
  ws->stat_part_side = (float*)a.take((int64_t)STAT_MAX_BLOCKS * 2 * cmax * 4);
  // (the ResNet-18 backward is the one that takes them)
  ws->stat_part_bsum = m.arch == HS_RESNET18 ? (float*)a.take((int64_t)STAT_MAX_BLOCKS * 2 * cmax * 4)
                                             : nullptr;
  // split-K partials: at least one split per worker of the largest weight
  // gradient (first layer counted with its padded channels)
  int64_t max_w = 64 * 9 * 8;
  for (const ParamT& t : m.params)
    if ((t.kind == HS_KIND_CONV_W || t.kind == HS_KIND_LIN_W) && t.numel > max_w) max_w = t.numel;
  const int64_t segs = max_n < MAX_SEG ? max_n : MAX_SEG;
  ws->splitk_floats = splitk_min_floats;
  if (segs * max_w > ws->splitk_floats) ws->splitk_floats = segs * max_w;
  ws->splitk = (float*)a.take(ws->splitk_floats * 4);
  if (m.dtype == HS_BF16) {
    ws->wpack_elems = max_w;
    ws->wpack = a.take(max_w * 2);
    // packed regions: at most two (forward, data gradient) per weight tensor
    int64_t all_w = 0;
    for (const ParamT& t : m.params)
      if (t.kind == HS_KIND_CONV_W || t.kind == HS_KIND_LIN_W) all_w += (t.numel + 63) / 64 * 64;
    ws->packed_cap = 2 * all_w;
    ws->packed = (bf16_t*)a.take(ws->packed_cap * 2);
  }
  // per-worker batch-norm / bias gradient sums of the partition-weighted mode,
  // one set per stream
  ws->gtmp_c = cmax > 512 ? cmax : 512;
  ws->gtmp = (float*)a.take((int64_t)MAX_SEG * 2 * ws->gtmp_c * 4);
  ws->gtmp_side = (float*)a.take((int64_t)MAX_SEG * 2 * ws->gtmp_c * 4);
  ws->gaps = (int64_t*)a.take((int64_t)(m.gaps.size() + 2) * 8);
  return a.off;
}

// ----------------------------------------------------------------------------
// launch helpers
// ----------------------------------------------------------------------------
namespace {

#define HS_TRY(expr)                    \
  do {                                  \
    hipError_t e_ = (expr);             \
    if (e_ != hipSuccess) return e_;    \
  } while (0)

// One pass over the layers for the workers in sg (n = all their samples):
// layer launches cover the whole batch; batch-norm statistics, losses and
// weight gradients are taken per worker, worker s writing g[s].
struct Ctx {
  const Model& m;
  Workspace& ws;
  const float* theta;
  const bf16_t* tbf;
  int n;
  hipStream_t s;
  bool bf;
  int V;  // elements per 16 bytes
  Segs sg;
  float* g[MAX_SEG];
  float* part = nullptr;   // statistics partials of this stream (null: ws.stat_part)
  // partition-weighted mode: every parameter gradient goes to gbar as
  // sum_s w[s] g_s (the per-worker g_s are not stored; per-worker batch-norm
  // and bias sums go to this stream's gtmp slots)
  float* gbar = nullptr;
  float w[MAX_SEG] = {};
  float* sp() const { return part ? part : ws.stat_part; }
  float* gtmp() const { return part ? ws.gtmp_side : ws.gtmp; }
  const void* W(int64_t off) const {
    return bf ? (const void*)(tbf + off) : (const void*)(theta + off);
  }
  // worker s's batch-norm statistics: mean at mean(b) + s * mstride()
  int mstride() const { return 2 * m.max_c; }
  float* mean(const BNL& b, int sg_i = 0) const {
    return ws.stats + ((int64_t)b.stat * MAX_SEG + sg_i) * 2 * m.max_c;
  }
  float* rstd(const BNL& b, int sg_i = 0) const { return mean(b, sg_i) + m.max_c; }
};

Segs one_segment(int n) {
  Segs sg{};
  sg.count = 1;
  sg.n0[0] = 0;
  sg.n0[1] = n;
  return sg;
}

ConvGeom geom(const ConvL& c, int n) {
  ConvGeom g;
  g.n = n;
  g.H = c.H;
  g.W = c.W;
  g.C = c.cin;
  g.Ho = c.Ho;
  g.Wo = c.Wo;
  g.K = c.cout;
  g.R = c.k;
  g.S = c.k;
  g.stride = c.stride;
  g.pad = c.pad;
  g.HWo = make_fastdiv((uint32_t)(c.Ho * c.Wo));
  g.Wo_ = make_fastdiv((uint32_t)c.Wo);
  g.HWi = make_fastdiv((uint32_t)(c.H * c.W));
  g.Wi_ = make_fastdiv((uint32_t)c.W);
  g.Cdiv = make_fastdiv((uint32_t)c.cin);
  g.Kdiv = make_fastdiv((uint32_t)c.cout);
  g.Sdiv = make_fastdiv((uint32_t)c.k);
  return g;
}

GemmParams base_params(const ConvL& c, int n) {
  GemmParams p{};
  p.g = geom(c, n);
  return p;
}

void pick_tiles(int M, int N, int& bm, int& bn) {
  const int cand[4][2] = {{128, 128}, {128, 64}, {64, 128}, {64, 64}};
  for (int i = 0; i < 4; ++i) {
    if (N <= 64 && cand[i][1] == 128) continue;
    if (M <= 64 && cand[i][0] == 128) continue;
    int64_t tiles = (int64_t)ceil_div(M, cand[i][0]) * ceil_div(N, cand[i][1]);
    if (tiles >= 512) {
      bm = cand[i][0];
      bn = cand[i][1];
      return;
    }
  }
  bm = 64;
  bn = 64;
}

// Tile of the fast kernel for an M x N output (0 x 0: none fits).
void pick_fast_tiles(int mode, int M, int N, int& bm, int& bn) {
  if (mode == MODE_WGRAD) {   // M = c_out; split-K supplies the parallelism
    bm = M <= 64 ? 64 : 128;
    bn = 128;
    return;
  }
  const int cand[5][2] = {{256, 64}, {128, 128}, {128, 64}, {64, 128}, {64, 256}};
  int best = -1;
  int64_t best_tiles = 0;
  for (int i = 0; i < 5; ++i) {
    const int cbm = cand[i][0], cbn = cand[i][1];
    if (cbn > 64 && N <= 64) continue;
    if (cbn == 256 && N < 256) continue;
    if (cbm == 256 && N > 64) continue;
    const int64_t tiles = (int64_t)ceil_div(M, cbm) * ceil_div(N, cbn);
    if (tiles >= 768) {
      bm = cbm;
      bn = cbn;
      return;
    }
    if (tiles > best_tiles) {
      best_tiles = tiles;
      best = i;
    }
  }
  bm = cand[best < 0 ? 2 : best][0];
  bn = cand[best < 0 ? 2 : best][1];
}

hipError_t wait_mark(const Ctx& c, int k);

// The packed copy (launch_pack_weights) of weights w -- a tensor of
// theta_bf16 -- for `mode` and the contraction shape `shape`: the tensor's
// listed region (packed on the second stream at the start of every later
// call; waited for here), a new region packed now on the first call, or, with
// scratch_ok, the workspace's one-layer buffer (packed now).  *out is null
// when none of them is available.
hipError_t packed_weights(const Ctx& c, const void* w, int mode, const GemmParams& shape,
                          bool scratch_ok, const void** out) {
  Workspace& ws = c.ws;
  *out = nullptr;
  int64_t woff = c.tbf ? (const bf16_t*)w - c.tbf : -1;
  if (woff >= c.m.P) woff = -1;   // not a tensor of theta
  const int64_t key = woff * 2 + (mode == MODE_DGRAD ? 1 : 0);
  const auto it = ws.packed && woff >= 0 ? ws.pack_of.find(key) : ws.pack_of.end();
  if (it != ws.pack_of.end() && ws.pack_ready >= 0) {
    if (!ws.pack_waited) {
      HS_TRY(wait_mark(c, ws.pack_ready));
      ws.pack_waited = true;
    }
    *out = ws.packed + ws.packs[it->second].dst;
  } else if (it != ws.pack_of.end()) {
    *out = ws.packed + ws.packs[it->second].dst;
    HS_TRY(launch_pack_weights(w, (void*)*out, mode, shape, c.s));
  } else if (ws.packed && woff >= 0 &&
             ws.packed_used + conv2_packed_elems(shape, mode) <= ws.packed_cap) {
    Workspace::Pack e{woff, ws.packed_used, shape, mode};
    ws.packed_used += (conv2_packed_elems(shape, mode) + 63) / 64 * 64;
    ws.pack_of[key] = (int)ws.packs.size();
    ws.packs.push_back(e);
    *out = ws.packed + e.dst;
    HS_TRY(launch_pack_weights(w, (void*)*out, mode, shape, c.s));
  } else if (scratch_ok && conv2_packed_elems(shape, mode) <= ws.wpack_elems) {
    HS_TRY(launch_pack_weights(w, ws.wpack, mode, shape, c.s));
    *out = ws.wpack;
  }
  return hipSuccess;
}

// timing probe (hs_probe_enable): an event before and after a launch of the
// probed (mode, tile) on the launch's stream
bool probe_begin(const Ctx& c, int mode, int bm, int bn) {
  Workspace& ws = c.ws;
  if (!(ws.probe_mode == mode && ws.probe_bm == bm && ws.probe_bn == bn &&
        ws.probe_used * 2 + 1 < ws.probe_ev.size()))
    return false;
  return hipEventRecord(ws.probe_ev[2 * ws.probe_used], c.s) == hipSuccess;
}
hipError_t probe_end(const Ctx& c, double flops) {
  Workspace& ws = c.ws;
  HS_TRY(hipEventRecord(ws.probe_ev[2 * ws.probe_used + 1], c.s));
  ws.probe_flops[ws.probe_used] = flops;
  ws.probe_used += 1;
  return hipSuccess;
}

// Launch one GEMM (fast kernel when the shape allows, generic otherwise);
// brackets it with probe events when it is the probed instantiation.
// With p.stat_part set (a forward), *stats_fused tells whether the kernel
// took the batch-norm sums and stat_blk[0 .. workers] receives their slot
// ranges (GemmParams::stat_part).
hipError_t gemm(const Ctx& c, int mode, const GemmParams& p, bool veca, bool vecb, int bm, int bn,
                int splits, double flops, bool* stats_fused = nullptr, int* stat_blk = nullptr) {
  Workspace& ws = c.ws;
  if (stats_fused) *stats_fused = false;
  int fbm = 0, fbn = 0;
  pick_fast_tiles(mode, p.M, p.N, fbm, fbn);
  const bool fast = p.par || (veca && vecb && igemm_fast_ok(mode, c.bf, p, fbm, fbn));
  if (fast) {
    bm = fbm;
    bn = fbn;
  }
  // bf16 stride-1 forward / data gradient with at least 128 channels per tap
  // on the gathered side: 32x32 MFMA kernel on packed weights (measured faster
  // there; with 64 channels or stride 2 the 128-byte K slices of the kernel
  // above use the cache lines of the gathered operand better)
  const int ctap = mode == MODE_FWD ? p.g.C : p.g.K;
  bool mfma32 = c.bf && mode != MODE_WGRAD && ws.wpack && p.g.stride == 1 && ctap >= 128 &&
                      conv2_ok(mode, p) && conv2_packed_elems(p, mode) <= ws.wpack_elems;
  // bf16 3x3 stride-1 weight gradient: patch kernel (split table in slices)
  const bool wg3 = c.bf && mode == MODE_WGRAD && p.nseg > 0 && wgrad3_ok(p) &&
                   p.split_stride > 0;
  if (wg3) {   // probe label: (64, 64) stride 1, (64, 256) stride 2
    bm = 64;
    bn = p.g.stride == 2 ? 256 : 64;
  }
  // 64 -> 64 channel 3x3 stride-1 on 32-wide maps: LDS patch kernel
  bool w64 = c.bf && mode != MODE_WGRAD && ws.wpack && conv64_ok(mode, p) &&
                   conv2_ok(mode, p) && conv2_packed_elems(p, mode) <= ws.wpack_elems;
  GemmParams q = p;
  // the packed-weight buffer is the main stream's: launches on the second
  // stream (c.part set) take the other kernels
  if (c.part) mfma32 = w64 = false;
  // epilogue statistics (GemmParams::stat_part) per worker: the 64-channel
  // forward kernel and the conv2 patch form (nseg stays 0 for the others,
  // where it means split-K over worker segments), while the partials fit
  // the workspace's buffer
  // (the data gradient's backward sums of a batch norm, GemmParams::bz: the
  // conv2 patch form)
  bool stats = false;
  const bool bsum = mode == MODE_DGRAD && q.bz;
  if ((w64 || mfma32) && (mode == MODE_FWD || bsum) && q.stat_part && stat_blk) {
    q.nseg = c.sg.count;
    for (int i = 0; i <= MAX_SEG; ++i) q.seg_n0[i] = c.sg.n0[i < c.sg.count ? i : c.sg.count];
    int64_t slots = -1;
    if (bsum) {
      if (mfma32 && !w64 && conv2_bsum_ok(q)) slots = conv2_stat_slots(q, stat_blk);
    } else if (w64) {
      const int blocks = conv64_blocks(q);
      for (int i = 0; i <= q.nseg; ++i) stat_blk[i] = i * blocks;
      slots = (int64_t)q.nseg * blocks;
    } else if (conv2_stats_ok(q)) {
      slots = conv2_stat_slots(q, stat_blk);
    }
    stats = slots > 0 && slots * 2 * p.N <= (int64_t)STAT_MAX_BLOCKS * 2 * 512;
  }
  if (!stats) {
    q.stat_part = nullptr;
    q.bz = nullptr;
    q.nseg = p.nseg;
  }
  if (mfma32 || w64) {
    const void* wb = nullptr;
    HS_TRY(packed_weights(c, p.b, mode, p, true, &wb));
    q.b = wb;
    bm = w64 ? 64 : 512;
    bn = w64 ? 64 : conv2_bn(p.N);
  }
  const bool probe = (fast || mfma32 || wg3 || w64) && probe_begin(c, mode, bm, bn);
  if (wg3) HS_TRY(launch_wgrad3(p, c.s));
  else if (w64) HS_TRY(launch_conv64(mode, q, c.s));
  else if (mfma32) HS_TRY(launch_conv2(mode, q, c.s));
  else if (fast) HS_TRY(launch_igemm_fast(mode, c.bf, p, bm, bn, splits, c.s));
  else {
    GemmParams r = p;
    r.mbits = nullptr;   // the generic kernel reads the mask tensor
    HS_TRY(launch_igemm(mode, c.bf, r, veca, vecb, bm, bn, splits, c.s));
  }
  if (probe) HS_TRY(probe_end(c, flops));
  if (stats_fused) *stats_fused = stats;
  return hipSuccess;
}

// algorithmic FLOPs of one contraction of layer L over n samples
double layer_flops(const ConvL& L, int n) {
  return 2.0 * n * L.Ho * L.Wo * (double)L.cout * L.k * L.k * L.cin;
}

// y = conv(x) (+ bias, ReLU); out_f32 forces an fp32 output
// stat_part: request the batch-norm sums of y from the epilogue (see
// GemmParams::stat_part); *stats_fused tells whether the kernel took them,
// stat_blk receives the workers' slot ranges
hipError_t conv_fwd(const Ctx& c, const ConvL& L, const void* x, void* y, bool out_f32,
                    const void* wptr = nullptr, const float* bias = nullptr, double flops = 0.0,
                    float* stat_part = nullptr, bool* stats_fused = nullptr,
                    int* stat_blk = nullptr) {
  GemmParams p = base_params(L, c.n);
  p.stat_part = stat_part;
  p.a = x;
  p.b = wptr ? wptr : c.W(L.w);
  p.out = y;
  p.bias = bias ? bias : (L.b >= 0 ? c.theta + L.b : nullptr);
  p.relu = L.relu ? 1 : 0;
  p.out_f32 = (out_f32 || !c.bf) ? 1 : 0;
  p.M = c.n * L.Ho * L.Wo;
  p.N = L.cout;
  p.K = L.k * L.k * L.cin;
  const bool vec = (L.cin % c.V) == 0;
  if (c.bf && L.stride == 2 && !c.part && c.ws.packed && !wptr && conv2s2f_ok(p)) {
    // bf16 3x3 stride 2: the patch form over whole input images (conv2.hip),
    // with the batch-norm sums per worker when asked and the partials fit
    const void* wb = nullptr;
    HS_TRY(packed_weights(c, p.b, MODE_FWD, p, false, &wb));
    if (wb) {
      GemmParams q = p;
      q.b = wb;
      bool stats = false;
      if (q.stat_part && stat_blk) {
        q.nseg = c.sg.count;
        for (int i = 0; i <= MAX_SEG; ++i) q.seg_n0[i] = c.sg.n0[i < c.sg.count ? i : c.sg.count];
        stats = conv2s2f_stats_ok(q) &&
                (int64_t)conv2s2f_stat_slots(q, stat_blk) * 2 * q.N <= (int64_t)STAT_MAX_BLOCKS * 2 * 512;
      }
      if (!stats) {
        q.stat_part = nullptr;
        q.nseg = p.nseg;
      }
      const bool probe = probe_begin(c, MODE_FWD, 256, 128);
      HS_TRY(launch_conv2s2f(q, c.s));
      if (probe) HS_TRY(probe_end(c, flops > 0 ? flops : layer_flops(L, c.n)));
      if (stats_fused) *stats_fused = stats;
      return hipSuccess;
    }
  }
  int bm, bn;
  pick_tiles(p.M, p.N, bm, bn);
  return gemm(c, MODE_FWD, p, vec, vec, bm, bn, 1, flops > 0 ? flops : layer_flops(L, c.n),
              stats_fused, stat_blk);
}

// dx = dgrad(dy) (+ addend) (* [mask > 0]); a stride-2 layer is computed by
// output parity class when the fast kernel applies (each class sums over
// its own taps only)
// Data gradient of layer L.  With proj set (a 1x1 stride-2 projection of
// the same input, its output gradient dproj), dx also receives the
// projection's data gradient, summed in the same reduction; that needs the
// stride-2 parity path, and when it is not available nothing is launched and
// *fused is false (the caller then runs the two data gradients itself).
// With bsum set, dx is the output gradient d of a batch norm whose input is
// bsum->z: the kernel takes that batch norm's backward sums (sum d, sum d z
// per worker) in its epilogue where it can (the bf16 conv2 patch form),
// *bsum->fused tells whether it did, bsum->blk receives their slot ranges
// (the partials are in the workspace's stat_part_bsum).
struct BsumReq {
  const void* z;
  int blk[MAX_SEG + 1];
  bool fused;
};
hipError_t conv_dgrad(const Ctx& c, const ConvL& L, const void* dy, void* dx, const void* addend,
                      const void* mask, const uint8_t* mbits = nullptr,
                      const ConvL* proj = nullptr, const void* dproj = nullptr,
                      bool* fused = nullptr, BsumReq* bsum = nullptr) {
  if (fused) *fused = false;
  if (bsum) bsum->fused = false;
  GemmParams p = base_params(L, c.n);
  p.a = dy;
  p.b = c.W(L.w);
  p.out = dx;
  p.addend = addend;
  p.mask = mask;
  p.mbits = c.bf && mask ? mbits : nullptr;   // bits of the same mask, where available
  p.out_f32 = c.bf ? 0 : 1;
  p.M = c.n * L.H * L.W;
  p.N = L.cin;
  p.K = L.k * L.k * L.cout;
  const bool veca = (L.cout % c.V) == 0;
  const bool vecb = (L.cin % c.V) == 0;
  const bool can_fuse = proj && dproj && fused && L.k == 3 && L.pad == 1 && proj->k == 1 &&
                        proj->stride == 2 && proj->pad == 0 && proj->cin == L.cin &&
                        proj->cout == L.cout && proj->H == L.H && proj->W == L.W;
  if (c.bf && L.stride == 2 && !c.part && c.ws.packed && (can_fuse || !proj)) {
    // bf16 3x3 stride 2: every parity class from one staged dy patch
    // (conv2.hip, stride-2 patch form), the shortcut's data gradient summed in
    GemmParams q = p;
    if (can_fuse) {
      q.a2 = dproj;
      q.b2 = c.W(proj->w);
    }
    if (conv2s2_ok(q)) {
      GemmParams pshape{};
      if (can_fuse) {
        pshape = base_params(*proj, c.n);
        pshape.N = proj->cin;
      }
      const void *wb = nullptr, *wb2 = nullptr;
      HS_TRY(packed_weights(c, p.b, MODE_DGRAD, p, false, &wb));
      if (wb && can_fuse) HS_TRY(packed_weights(c, q.b2, MODE_DGRAD, pshape, false, &wb2));
      if (wb && (!can_fuse || wb2)) {
        q.b = wb;
        q.b2 = wb2;
        const double flops = layer_flops(L, c.n) + (can_fuse ? layer_flops(*proj, c.n) : 0.0);
        const bool probe = probe_begin(c, MODE_DGRAD, 256, 256);
        HS_TRY(launch_conv2s2(q, c.s));
        if (probe) HS_TRY(probe_end(c, flops));
        if (can_fuse) *fused = true;
        return hipSuccess;
      }
    }
  }
  if (L.stride == 2 && L.H % 2 == 0 && L.W % 2 == 0 && veca && vecb) {
    GemmParams q = p;
    q.par = 1;
    q.Hh = L.H / 2;
    q.Wh = L.W / 2;
    q.HWh = make_fastdiv((uint32_t)(q.Hh * q.Wh));
    q.Wh_ = make_fastdiv((uint32_t)q.Wh);
    q.M = c.n * q.Hh * q.Wh;
    for (int cls = 0; cls < 4; ++cls) {
      const int ph = cls >> 1, pw = cls & 1;
      int nt = 0;
      for (int r = 0; r < L.k; ++r)
        for (int s2 = 0; s2 < L.k; ++s2)
          if (((ph + L.pad - r) & 1) == 0 && ((pw + L.pad - s2) & 1) == 0) q.taps[cls][nt++] = r * L.k + s2;
      q.ntap[cls] = nt;
    }
    double flops = layer_flops(L, c.n);
    const bool fuse = can_fuse;
    if (fuse) {
      q.a2 = dproj;
      q.b2 = c.W(proj->w);
      flops += layer_flops(*proj, c.n);
    }
    int fbm = 0, fbn = 0;
    pick_fast_tiles(MODE_DGRAD, q.M, q.N, fbm, fbn);
    if (igemm_fast_ok(MODE_DGRAD, c.bf, q, fbm, fbn) && (fuse || !proj)) {
      if (fuse) *fused = true;
      return gemm(c, MODE_DGRAD, q, veca, vecb, fbm, fbn, 1, flops);
    }
  }
  if (proj) return hipSuccess;   // fusion requested but not possible
  int bm, bn;
  pick_tiles(p.M, p.N, bm, bn);
  if (bsum && c.bf && !c.part && c.ws.stat_part_bsum) {
    p.bz = bsum->z;
    p.stat_part = c.ws.stat_part_bsum;
  }
  return gemm(c, MODE_DGRAD, p, veca, vecb, bm, bn, 1, layer_flops(L, c.n),
              bsum ? &bsum->fused : nullptr, bsum ? bsum->blk : nullptr);
}

// Whether the weight gradient of a residual block's 1x1 stride-2 projection
// P can be taken in the same launch as that of the block's first 3x3
// stride-2 convolution L (same input): the stride-2 patch kernel, and room in
// the split-K buffer for one split per worker of both partials.
bool wgrad_fuses_proj(const Ctx& c, const ConvL& L, const ConvL& P) {
  if (!c.bf || L.k != 3 || L.stride != 2 || P.k != 1 || P.stride != 2 || P.pad != 0 ||
      P.cin != L.cin || P.cout != L.cout || P.Ho != L.Ho || P.Wo != L.Wo)
    return false;
  GemmParams p = base_params(L, c.n);
  if (!wgrad3_ok(p)) return false;
  const int64_t mn = (int64_t)L.cout * 9 * L.cin + (int64_t)P.cout * P.cin;
  return (int64_t)c.sg.count * mn <= c.ws.splitk_floats;
}

// Weight gradient of every worker: worker s reduces over the pixels of its own
// samples and writes g[s] + L.w.  The reduction is split (split-K) so that
// the launch has about 1024 blocks; the partial sums are added per worker in
// split order.  With cin_true < L.cin the layer's input channels are padded
// and the padded columns of the gradient are dropped.  With proj (see
// wgrad_fuses_proj) the same launch also takes the projection's weight
// gradient from its output gradient dy_proj (same input x).
hipError_t conv_wgrad(const Ctx& c, const ConvL& L, const void* dy, const void* x,
                      int cin_true = 0, double flops = 0.0, const ConvL* proj = nullptr,
                      const void* dy_proj = nullptr) {
  if (flops <= 0) flops = layer_flops(L, c.n);
  if (cin_true <= 0) cin_true = L.cin;
  if (proj && !wgrad_fuses_proj(c, L, *proj)) return hipErrorInvalidValue;
  GemmParams p = base_params(L, c.n);
  p.a = dy;
  p.b = x;
  p.M = L.cout;
  p.N = L.k * L.k * L.cin;
  p.K = c.n * L.Ho * L.Wo;
  const bool veca = (L.cout % c.V) == 0;
  const bool vecb = (L.cin % c.V) == 0;
  const int64_t mn1 = (int64_t)p.M * p.N;
  if (c.bf && cin_true == L.cin && wgrad3_ok(p)) {
    // patch kernel: splits of 64-pixel slices, about 512 blocks in all; a
    // split's output holds the layer's partial and then the projection's
    const int64_t mnp = proj ? (int64_t)proj->cout * proj->cin : 0;
    const int64_t mn = mn1 + mnp;
    if (proj) {
      p.a2 = dy_proj;
      flops += layer_flops(*proj, c.n);
    }
    int ns[MAX_SEG], total = 0;
    for (int i = 0; i < c.sg.count; ++i) {
      ns[i] = wgrad3_slices(p, c.sg.n0[i + 1] - c.sg.n0[i]);
      total += ns[i];
    }
    const int tiles = (L.cout / 64) * (L.cin / 64);
    const int want = tiles >= kWgrad3Blocks ? 1 : kWgrad3Blocks / tiles;
    int per = ceil_div(total, want);
    if (per < 1) per = 1;
    auto count = [&](int q) {
      int t = 0;
      for (int i = 0; i < c.sg.count; ++i) t += ns[i] > 0 ? ceil_div(ns[i], q) : 1;
      return t;
    };
    while ((int64_t)count(per) * mn > c.ws.splitk_floats && per < total) per *= 2;
    if ((int64_t)count(per) * mn > c.ws.splitk_floats) return hipErrorInvalidValue;
    p.nseg = c.sg.count;
    p.kt_per_split = per;
    p.seg_split[0] = 0;
    for (int i = 0; i < c.sg.count; ++i) {
      p.seg_n0[i] = c.sg.n0[i];
      p.seg_split[i + 1] = p.seg_split[i] + (ns[i] > 0 ? ceil_div(ns[i], per) : 1);
    }
    p.seg_n0[c.sg.count] = c.sg.n0[c.sg.count];
    p.out = c.ws.splitk;
    p.split_stride = mn;
    HS_TRY(gemm(c, MODE_WGRAD, p, veca, vecb, 64, 64, p.seg_split[c.sg.count], flops));
    for (int part = 0; part < (proj ? 2 : 1); ++part) {
      const ConvL& T = part ? *proj : L;
      const float* src = c.ws.splitk + (part ? mn1 : 0);
      const int64_t count = part ? mnp : mn1;
      if (c.gbar) {
        HS_TRY(launch_splitk_reduce_wsum(src, mn, count, p.seg_split, c.w, c.gbar + T.w,
                                         c.sg.count, T.cin, T.cin, c.s));
        continue;
      }
      float* outs[MAX_SEG];
      for (int i = 0; i < c.sg.count; ++i) outs[i] = c.g[i] + T.w;
      HS_TRY(launch_splitk_reduce_seg(src, mn, count, p.seg_split, outs, c.sg.count, T.cin, T.cin,
                                      c.s));
    }
    return hipSuccess;
  }
  if (proj) return hipErrorInvalidValue;
  const int64_t mn = mn1;
  const int bm = p.M <= 64 ? 64 : 128, bn = 128;
  const int tiles = ceil_div(p.M, bm) * ceil_div(p.N, bn);
  const int bke = 128 / (c.bf ? 2 : 4);
  const int hw = L.Ho * L.Wo;
  int kt[MAX_SEG], total_kt = 0;
  for (int i = 0; i < c.sg.count; ++i) {
    kt[i] = ceil_div((c.sg.n0[i + 1] - c.sg.n0[i]) * hw, bke);
    total_kt += kt[i];
  }
  int want = ceil_div(kWgradFastTiles, tiles);
  if (want > kWgradFastMaxSplits) want = kWgradFastMaxSplits;
  int per = ceil_div(total_kt, want > 0 ? want : 1);
  if (per < 4) per = 4;
  auto count_splits = [&](int q) {
    int t = 0;
    for (int i = 0; i < c.sg.count; ++i) t += kt[i] > 0 ? ceil_div(kt[i], q) : 1;
    return t;
  };
  while ((int64_t)count_splits(per) * mn > c.ws.splitk_floats && per < total_kt) per *= 2;
  const int splits = count_splits(per);
  const bool direct = c.sg.count == 1 && splits == 1 && cin_true == L.cin;
  // the workspace plan sizes the partial buffer for one split per worker
  if (!direct && (int64_t)splits * mn > c.ws.splitk_floats) return hipErrorInvalidValue;
  p.nseg = c.sg.count;
  p.kt_per_split = per;
  p.seg_split[0] = 0;
  for (int i = 0; i < c.sg.count; ++i) {
    p.seg_n0[i] = c.sg.n0[i];
    p.seg_split[i + 1] = p.seg_split[i] + (kt[i] > 0 ? ceil_div(kt[i], per) : 1);
  }
  p.seg_n0[c.sg.count] = c.sg.n0[c.sg.count];
  if (direct) {
    // one worker (its weight is 1): straight into its gradient
    p.out = (c.gbar ? c.gbar : c.g[0]) + L.w;
    p.split_stride = 0;
    return gemm(c, MODE_WGRAD, p, veca, vecb, bm, bn, splits, flops);
  }
  p.out = c.ws.splitk;
  p.split_stride = mn;
  HS_TRY(gemm(c, MODE_WGRAD, p, veca, vecb, bm, bn, splits, flops));
  const int64_t count = (int64_t)L.cout * L.k * L.k * cin_true;
  if (c.gbar)
    return launch_splitk_reduce_wsum(c.ws.splitk, mn, count, p.seg_split, c.w, c.gbar + L.w,
                                     c.sg.count, cin_true, L.cin, c.s);
  float* outs[MAX_SEG];
  for (int i = 0; i < c.sg.count; ++i) outs[i] = c.g[i] + L.w;
  return launch_splitk_reduce_seg(c.ws.splitk, mn, count, p.seg_split, outs, c.sg.count, cin_true,
                                  L.cin, c.s);
}

// worker s: g[s][bias] = sum over its rows of dy (dy in activation type
// unless f32); rps rows per sample
hipError_t bias_grad(const Ctx& c, int64_t boff, const void* dy, bool f32, int64_t rps, int C) {
  float* out[MAX_SEG];
  StatWsum ws{};
  if (c.gbar) {
    for (int i = 0; i < c.sg.count; ++i) out[i] = c.gtmp() + (int64_t)i * 2 * c.ws.gtmp_c;
    ws.sum0 = c.gbar + boff;
    for (int i = 0; i < c.sg.count; ++i) ws.w[i] = c.w[i];
  } else {
    for (int i = 0; i < c.sg.count; ++i) out[i] = c.g[i] + boff;
  }
  return launch_chan_stats(2, f32 ? false : c.bf, nullptr, dy, nullptr, nullptr, nullptr, 0, c.sg,
                           rps, C, c.sp(), out, nullptr, 0.f, c.s, c.gbar ? &ws : nullptr);
}

// per-worker batch-norm statistics of z (rps rows per sample)
hipError_t bn_stats(const Ctx& c, const BNL& b, const void* z, int64_t rps) {
  float *o0[MAX_SEG], *o1[MAX_SEG];
  for (int i = 0; i < c.sg.count; ++i) {
    o0[i] = c.mean(b, i);
    o1[i] = c.rstd(b, i);
  }
  return launch_chan_stats(0, c.bf, z, nullptr, nullptr, nullptr, nullptr, 0, c.sg, rps, b.c,
                           c.sp(), o0, o1, 1e-5f, c.s);
}

// z = conv(x) and the batch-norm statistics of z: summed in the
// convolution's epilogue where its kernel takes them (the 64-channel 3x3
// layers on 32-wide maps and the stride-1 and stride-2 patch forms:
// partials per block or row tile and worker, then the finish), else by a
// pass over z
hipError_t conv_bn_fwd(const Ctx& c, const ConvL& L, const void* x, void* z, const BNL& b,
                       int64_t rps) {
  bool want = c.bf && !c.part && L.b < 0 && !L.relu && b.c == L.cout && c.sg.count >= 1 &&
              c.sg.n0[0] == 0 && c.sg.n0[c.sg.count] == c.n;
  for (int i = 0; want && i < c.sg.count; ++i) want = c.sg.n0[i + 1] > c.sg.n0[i];
  bool fused = false;
  int blk[MAX_SEG + 1];
  HS_TRY(conv_fwd(c, L, x, z, false, nullptr, nullptr, 0.0, want ? c.sp() : nullptr, &fused,
                  blk));
  if (!fused) return bn_stats(c, b, z, rps);
  float *o0[MAX_SEG], *o1[MAX_SEG];
  for (int i = 0; i < c.sg.count; ++i) {
    o0[i] = c.mean(b, i);
    o1[i] = c.rstd(b, i);
  }
  return launch_stats_finish_fwd(c.bf, c.sp(), 0, c.sg, rps, b.c, o0, o1, 1e-5f, c.s, blk);
}

// y = relu?(batch-norm(z) + res) with every worker's own statistics
hipError_t bn_apply(const Ctx& c, const BNL& b, const void* z, const void* res, int relu,
                    int64_t rps, void* y, uint8_t* ybits = nullptr) {
  return launch_bn_apply8(c.bf, z, c.mean(b), c.rstd(b), c.mstride(), c.theta + b.g,
                          c.theta + b.b, res, relu, c.sg, rps, b.c, y, c.s, ybits);
}

// Where the batch-norm backward's per-worker sums go: the beta and gamma
// gradients of g[s] (or, forming g_bar, this stream's slots, with their
// weighted sums into g_bar)
void bn_sum_targets(const Ctx& c, const BNL& b, float* (&db)[MAX_SEG], float* (&dg)[MAX_SEG],
                    StatWsum& ws) {
  if (c.gbar) {
    // the workers' sums in this stream's slots (the backward below reads
    // them), their weighted sums into gbar
    for (int i = 0; i < c.sg.count; ++i) {
      db[i] = c.gtmp() + (int64_t)i * 2 * c.ws.gtmp_c;
      dg[i] = db[i] + c.ws.gtmp_c;
      ws.w[i] = c.w[i];
    }
    ws.sum0 = c.gbar + b.b;
    ws.sum1 = c.gbar + b.g;
  } else {
    for (int i = 0; i < c.sg.count; ++i) {
      db[i] = c.g[i] + b.b;
      dg[i] = c.g[i] + b.g;
    }
  }
}

// dz = batch-norm backward of dy (masked by [act > 0] if act); writes every
// worker's dbeta, dgamma into its g[s]
hipError_t bn_bwd(const Ctx& c, const BNL& b, const void* dy, const void* act, const void* z,
                  int64_t rps, void* dz) {
  float *db[MAX_SEG], *dg[MAX_SEG];
  StatWsum ws{};
  bn_sum_targets(c, b, db, dg, ws);
  HS_TRY(launch_chan_stats(1, c.bf, z, dy, act, c.mean(b), c.rstd(b), c.mstride(), c.sg, rps, b.c,
                           c.sp(), db, dg, 0.f, c.s, c.gbar ? &ws : nullptr));
  return launch_bn_backward8(c.bf, dy, act, z, c.mean(b), c.rstd(b), c.mstride(), c.theta + b.g,
                             db, dg, c.sg, rps, b.c, dz, c.s);
}

// The batch-norm backward of b where a data gradient's epilogue took its
// sums (BsumReq, fused): the finish into every worker's dbeta, dgamma (as
// bn_bwd), then dz; else bn_bwd itself.
hipError_t bn_bwd_sums(const Ctx& c, const BNL& b, const BsumReq& r, const void* dy,
                       const void* z, int64_t rps, void* dz) {
  if (!r.fused) return bn_bwd(c, b, dy, nullptr, z, rps, dz);
  float *db[MAX_SEG], *dg[MAX_SEG];
  StatWsum ws{};
  bn_sum_targets(c, b, db, dg, ws);
  HS_TRY(launch_stats_finish_bwd(c.ws.stat_part_bsum, c.sg, b.c, c.mean(b), c.rstd(b), c.mstride(), db, dg, c.s,
                                 r.blk, c.gbar ? &ws : nullptr));
  return launch_bn_backward8(c.bf, dy, nullptr, z, c.mean(b), c.rstd(b), c.mstride(), c.theta + b.g,
                             db, dg, c.sg, rps, b.c, dz, c.s);
}

// softmax cross-entropy on the logits, mean per worker; returns the operand
// for the last layer's backward (fp32 or bf16 copy of dz)
hipError_t loss_grad(const Ctx& c, const int32_t* y, float* loss, const void** dzop) {
  HS_TRY(launch_softmax_ce(c.ws.logits, y, c.sg, 10, loss, c.ws.dz32, c.bf ? c.ws.dzt : nullptr,
                           c.bf, c.s));
  *dzop = c.bf ? c.ws.dzt : (const void*)c.ws.dz32;
  return hipSuccess;
}

// The weight gradients of the backward pass run on the workspace's second
// stream, beside the batch-norm and data-gradient chain of the main stream:
// fork() orders the second stream after the work enqueued so far on the
// main one, join() the main stream after the second.  Without a second
// stream (a temporary workspace) both are no-ops and side() is the main
// stream.
hipError_t order(Workspace& w, hipStream_t after, hipStream_t waiter) {
  hipEvent_t e = w.ev[w.ev_next];
  w.ev_next = (w.ev_next + 1) % Workspace::kEvents;
  HS_TRY(hipEventRecord(e, after));
  return hipStreamWaitEvent(waiter, e, 0);
}
hipError_t fork(const Ctx& c) { return c.ws.side ? order(c.ws, c.s, c.ws.side) : hipSuccess; }
hipError_t join(const Ctx& c) { return c.ws.side ? order(c.ws, c.ws.side, c.s) : hipSuccess; }
Ctx side(const Ctx& c) {
  Ctx d = c;
  if (c.ws.side) {
    d.s = c.ws.side;
    d.part = c.ws.stat_part_side;
  }
  return d;
}
// a point of the second stream that the main stream waits for later: the
// ring is recorded on the second stream only, so a reuse before the wait
// makes the wait later than needed, never earlier
int side_mark(const Ctx& c) {
  if (!c.ws.side) return -1;
  const int k = c.ws.evr_next;
  c.ws.evr_next = (c.ws.evr_next + 1) % Workspace::kEvents;
  return hipEventRecord(c.ws.evr[k], c.ws.side) == hipSuccess ? k : -2;
}
hipError_t wait_mark(const Ctx& c, int k) {
  if (k == -2) return hipErrorUnknown;
  return k >= 0 ? hipStreamWaitEvent(c.s, c.ws.evr[k], 0) : hipSuccess;
}

// Gradient buffers of a backward pass whose weight gradients run on the
// second stream: a buffer the second stream reads keeps the event recorded
// after that read, and the main stream waits for it only when it writes the
// buffer again.  Free buffers are handed out least recently released first,
// those without a pending read before the others.
struct GradPool {
  Workspace& w;
  hipStream_t main;
  int n;
  bool live[Workspace::kGrad] = {};
  int pending[Workspace::kGrad];   // event slot of the last second-stream read, or -1
  int64_t stamp[Workspace::kGrad] = {};
  int64_t clock = 0;
  GradPool(Workspace& ws, hipStream_t s) : w(ws), main(s), n(ws.ngrad) {
    for (int i = 0; i < Workspace::kGrad; ++i) pending[i] = -1;
  }
  void* operator[](int i) const { return w.grad[i]; }
  // a free buffer for the main stream to write
  int take(int& out) {
    int best = -1;
    for (int i = 0; i < n; ++i) {
      if (live[i]) continue;
      if (best < 0 || (pending[i] < 0) > (pending[best] < 0) ||
          ((pending[i] < 0) == (pending[best] < 0) && stamp[i] < stamp[best]))
        best = i;
    }
    if (best < 0) return -1;
    if (pending[best] >= 0 && w.side) {
      if (hipStreamWaitEvent(main, w.evr[pending[best]], 0) != hipSuccess) return -1;
    }
    pending[best] = -1;
    live[best] = true;
    out = best;
    return 0;
  }
  void drop(int i) {
    live[i] = false;
    stamp[i] = ++clock;
  }
  // the second stream has been given work that reads buffer i.  The slot's
  // events are recorded on the second stream only, so if the ring reuses it
  // before the wait, the wait covers a later point of that stream: later
  // than needed, never earlier.
  hipError_t read_on_side(int i) {
    if (!w.side) return hipSuccess;
    const int k = w.evr_next;
    w.evr_next = (w.evr_next + 1) % Workspace::kEvents;
    pending[i] = k;
    return hipEventRecord(w.evr[k], w.side);
  }
};

#define HS_TAKE(pool, var)                                 \
  int var = -1;                                            \
  if ((pool).take(var) != 0) return hipErrorInvalidValue;

// ---------------------------------------------------------------- stem ----
// The 3-channel first convolution runs on the fast kernel with its input and
// weights zero-padded to 8 (bf16) or 4 (fp32) channels; its weight gradient
// is computed padded and the padding dropped.
int stem_cpad(const Ctx& c) { return c.bf ? 8 : 4; }

hipError_t stem_fwd(const Ctx& c, const ConvL& L, const float* x, void* X0, void* y) {
  const int cp = stem_cpad(c);
  if (c.bf && stem_ok(L.cin, L.cout, L.k, L.stride, L.pad, L.H, L.W)) {
    // the direct stem kernel (stem.hip); the weight gradient reads x too
    const bool probe = probe_begin(c, MODE_FWD, 32, 64);
    HS_TRY(launch_stem_fwd(x, c.W(L.w), y, nullptr, c.n, c.s));
    if (probe) HS_TRY(probe_end(c, layer_flops(L, c.n)));
    return hipSuccess;
  }
  ConvL st = L;
  st.cin = cp;
  HS_TRY(launch_nchw_to_nhwc_pad(x, X0, c.n, 3, cp, L.H * L.W, c.bf, c.s));
  HS_TRY(launch_pad_weights(c.theta + L.w, c.ws.stem_w, L.cout, L.k * L.k, 3, cp, c.bf, c.s));
  return conv_fwd(c, st, X0, y, false, c.ws.stem_w, nullptr, layer_flops(L, c.n));
}

// The first layer and its batch-norm statistics: the direct bf16 stem takes
// the sums of its stored output per image (one image per block, so one
// worker per block) and the finish adds each worker's images; otherwise the
// statistics pass over z follows.
hipError_t stem_bn_fwd(const Ctx& c, const ConvL& L, const BNL& b, const float* x, void* X0,
                       void* z) {
  bool fuse = c.bf && !c.part && b.c == L.cout && L.cout == 64 &&
              stem_ok(L.cin, L.cout, L.k, L.stride, L.pad, L.H, L.W) &&
              (int64_t)c.n * 2 * 64 <= (int64_t)STAT_MAX_BLOCKS * 2 * 512 && c.sg.count >= 1 &&
              c.sg.n0[0] == 0 && c.sg.n0[c.sg.count] == c.n;
  for (int i = 0; fuse && i < c.sg.count; ++i) fuse = c.sg.n0[i + 1] > c.sg.n0[i];
  if (!fuse) {
    HS_TRY(stem_fwd(c, L, x, X0, z));
    return bn_stats(c, b, z, (int64_t)L.Ho * L.Wo);
  }
  const bool probe = probe_begin(c, MODE_FWD, 32, 64);
  HS_TRY(launch_stem_fwd(x, c.W(L.w), z, nullptr, c.n, c.s, c.sp()));
  if (probe) HS_TRY(probe_end(c, layer_flops(L, c.n)));
  float *o0[MAX_SEG], *o1[MAX_SEG];
  int blk[MAX_SEG + 1];
  for (int i = 0; i < c.sg.count; ++i) {
    o0[i] = c.mean(b, i);
    o1[i] = c.rstd(b, i);
  }
  for (int i = 0; i <= c.sg.count; ++i) blk[i] = c.sg.n0[i];
  return launch_stats_finish_fwd(c.bf, c.sp(), 0, c.sg, (int64_t)L.Ho * L.Wo, b.c, o0, o1, 1e-5f,
                                 c.s, blk);
}

// With bn (the direct kernel only), dz is the batch-norm output's gradient
// and the kernel forms the batch-norm backward as it reads it (StemBnBwd).
hipError_t stem_wgrad(const Ctx& c, const ConvL& L, const void* dz, const void* X0,
                      const float* x, const StemBnBwd* bn = nullptr) {
  if (c.bf && stem_ok(L.cin, L.cout, L.k, L.stride, L.pad, L.H, L.W)) {
    // the direct stem weight gradient (stem.hip): split-K partials per worker
    // from x and dz, then the per-worker reduce
    int nseg_n[MAX_SEG], split[MAX_SEG + 1];
    for (int i = 0; i < c.sg.count; ++i) nseg_n[i] = c.sg.n0[i + 1] - c.sg.n0[i];
    const int splits = stem_wgrad_splits(nseg_n, c.sg.count, split);
    const int64_t mn = (int64_t)L.cout * L.k * L.k * L.cin;
    if ((int64_t)splits * mn > c.ws.splitk_floats) return hipErrorInvalidValue;
    const bool probe = probe_begin(c, MODE_WGRAD, 32, 64);
    HS_TRY(launch_stem_wgrad(x, dz, c.ws.splitk, c.sg.n0, split, c.sg.count, c.s, bn));
    if (probe) HS_TRY(probe_end(c, layer_flops(L, c.n)));
    if (c.gbar)
      return launch_splitk_reduce_wsum(c.ws.splitk, mn, mn, split, c.w, c.gbar + L.w, c.sg.count,
                                       (int)mn, (int)mn, c.s);
    float* outs[MAX_SEG];
    for (int i = 0; i < c.sg.count; ++i) outs[i] = c.g[i] + L.w;
    return launch_splitk_reduce_seg(c.ws.splitk, mn, mn, split, outs, c.sg.count, (int)mn,
                                    (int)mn, c.s);
  }
  if (bn) return hipErrorInvalidValue;
  ConvL st = L;
  st.cin = stem_cpad(c);
  return conv_wgrad(c, st, dz, X0, L.cin, layer_flops(L, c.n));
}

// The first layer's batch-norm backward and weight gradient, last in the
// backward pass: the batch-norm sums on the caller's stream (beside the
// second stream's last weight gradients), the join (the weight gradient
// shares the split-K buffer), then the weight gradient.  The direct bf16 stem
// forms dz = BN backward of dy (dy masked by [act > 0] when act is set) as it
// reads dy and z, since nothing else reads that dz; otherwise dz is written
// to dz_buf first.
hipError_t stem_backward(const Ctx& c, const ConvL& L, const BNL& b, const void* dy,
                         const void* act, const void* z, int64_t rps, void* dz_buf,
                         const void* X0, const float* x) {
  if (c.bf && c.theta && stem_ok(L.cin, L.cout, L.k, L.stride, L.pad, L.H, L.W)) {
    float *db[MAX_SEG], *dg[MAX_SEG];
    StatWsum ws{};
    bn_sum_targets(c, b, db, dg, ws);
    HS_TRY(launch_chan_stats(1, c.bf, z, dy, act, c.mean(b), c.rstd(b), c.mstride(), c.sg, rps,
                             b.c, c.sp(), db, dg, 0.f, c.s, c.gbar ? &ws : nullptr));
    HS_TRY(join(c));
    StemBnBwd bn{};
    bn.z = z;
    bn.act = act;
    bn.mean = c.mean(b);
    bn.rstd = c.rstd(b);
    bn.mstride = c.mstride();
    bn.gamma = c.theta + b.g;
    for (int i = 0; i < c.sg.count; ++i) {
      bn.sum0[i] = db[i];
      bn.sum1[i] = dg[i];
    }
    return stem_wgrad(c, L, dy, X0, x, &bn);
  }
  HS_TRY(bn_bwd(c, b, dy, act, z, rps, dz_buf));
  HS_TRY(join(c));
  return stem_wgrad(c, L, dz_buf, X0, x);
}

// ---------------------------------------------------------------- MLP ----
hipError_t mlp(const Ctx& c, const float* x, const int32_t* y, float* loss) {
  const Model& m = c.m;
  const void* X = x;
  if (c.bf) {
    HS_TRY(launch_cast_input(x, c.ws.slot[0], (int64_t)c.n * 784, true, c.s));
    X = c.ws.slot[0];
  }
  void* Hh = c.ws.slot[1];
  HS_TRY(conv_fwd(c, m.fc1, X, Hh, false));
  HS_TRY(conv_fwd(c, m.fc2, Hh, c.ws.logits, true));
  const void* dz;
  HS_TRY(loss_grad(c, y, loss, &dz));
  HS_TRY(conv_wgrad(c, m.fc2, dz, Hh));
  HS_TRY(bias_grad(c, m.fc2.b, c.ws.dz32, true, 1, 10));
  void* dH = c.ws.grad[0];
  HS_TRY(conv_dgrad(c, m.fc2, dz, dH, nullptr, Hh));
  HS_TRY(bias_grad(c, m.fc1.b, dH, false, 1, 256));
  return conv_wgrad(c, m.fc1, dH, X);
}

// ----------------------------------------------------------- small CNN ----
hipError_t small_cnn(const Ctx& c, const float* x, const int32_t* y, float* loss) {
  const Model& m = c.m;
  void **S = c.ws.slot.data(), **G = c.ws.grad;
  const int n = c.n;
  HS_TRY(stem_fwd(c, m.c1, x, S[0], S[1]));
  HS_TRY(conv_fwd(c, m.c2, S[1], S[2], false));
  HS_TRY(launch_maxpool_fwd(c.bf, S[2], n, 32, 32, 64, S[3], c.s));
  HS_TRY(conv_fwd(c, m.c3, S[3], S[4], false));
  HS_TRY(launch_gap_fwd(c.bf, S[4], n, 256, 128, S[5], c.s));
  HS_TRY(conv_fwd(c, m.fc2, S[5], c.ws.logits, true));
  const void* dz;
  HS_TRY(loss_grad(c, y, loss, &dz));
  HS_TRY(conv_wgrad(c, m.fc2, dz, S[5]));
  HS_TRY(bias_grad(c, m.fc2.b, c.ws.dz32, true, 1, 10));
  HS_TRY(conv_dgrad(c, m.fc2, dz, G[0], nullptr, nullptr));           // dF
  HS_TRY(launch_gap_bwd(c.bf, G[0], S[4], n, 256, 128, G[1], c.s));    // dA3 * [A3 > 0]
  HS_TRY(bias_grad(c, m.c3.b, G[1], false, 256, 128));
  HS_TRY(conv_wgrad(c, m.c3, G[1], S[3]));
  HS_TRY(conv_dgrad(c, m.c3, G[1], G[0], nullptr, nullptr));          // dP2
  HS_TRY(launch_maxpool_bwd(c.bf, S[2], G[0], n, 32, 32, 64, 1, G[2], c.s));  // dA2 * [A2 > 0]
  HS_TRY(bias_grad(c, m.c2.b, G[2], false, 1024, 64));
  HS_TRY(conv_wgrad(c, m.c2, G[2], S[1]));
  HS_TRY(conv_dgrad(c, m.c2, G[2], G[0], nullptr, S[1]));             // dA1 * [A1 > 0]
  HS_TRY(bias_grad(c, m.c1.b, G[0], false, 1024, 32));
  return stem_wgrad(c, m.c1, G[0], S[0], x);
}

// ---------------------------------------------------------- ResNet-18 ----
hipError_t resnet(const Ctx& c, const float* x, const int32_t* y, float* loss) {
  const Model& m = c.m;
  void** S = c.ws.slot.data();
  uint8_t* const* Bt = c.ws.bits.data();   // bits of the ReLU outputs
  void** G = c.ws.grad;
  const int n = c.n;
  const Ctx cs = side(c);   // second stream: projection shortcuts, weight gradients
  HS_TRY(stem_bn_fwd(c, m.stem, m.stem_bn, x, S[0], S[1]));
  HS_TRY(bn_apply(c, m.stem_bn, S[1], nullptr, 1, 1024, S[2], Bt[2]));
  const void* cur = S[2];
  int si = 3;
  for (const BlockL& b : m.blocks) {
    void *Z1 = S[si], *Hh = S[si + 1], *Z2 = S[si + 2], *ZP = S[si + 3], *A = S[si + 4];
    uint8_t *Hb = Bt[si + 1], *Ab = Bt[si + 4];
    si += 5;
    const int64_t rps = (int64_t)b.c1.Ho * b.c1.Wo;
    // the projection shortcut on the second stream, beside conv1 .. bn2
    const void* res = cur;
    int proj_done = -1;
    if (b.proj) {
      HS_TRY(fork(c));
      HS_TRY(conv_fwd(cs, b.cp, cur, ZP, false));
      HS_TRY(bn_stats(cs, b.bp, ZP, rps));
      HS_TRY(bn_apply(cs, b.bp, ZP, nullptr, 0, rps, G[0]));
      proj_done = side_mark(c);
      res = G[0];
    }
    HS_TRY(conv_bn_fwd(c, b.c1, cur, Z1, b.b1, rps));
    HS_TRY(bn_apply(c, b.b1, Z1, nullptr, 1, rps, Hh, Hb));
    HS_TRY(conv_bn_fwd(c, b.c2, Hh, Z2, b.b2, rps));
    HS_TRY(wait_mark(c, proj_done));
    HS_TRY(bn_apply(c, b.b2, Z2, res, 1, rps, A, Ab));
    cur = A;
  }
  void* F = S[si];
  HS_TRY(launch_gap_fwd(c.bf, cur, n, 16, 512, F, c.s));
  HS_TRY(conv_fwd(c, m.fc2, F, c.ws.logits, true));
  // ---- backward
  const void* dz;
  HS_TRY(loss_grad(c, y, loss, &dz));
  HS_TRY(conv_wgrad(c, m.fc2, dz, F));
  HS_TRY(bias_grad(c, m.fc2.b, c.ws.dz32, true, 1, 10));
  HS_TRY(conv_dgrad(c, m.fc2, dz, G[0], nullptr, nullptr));           // dF
  // gradient of the last block's output, masked by its ReLU ([A > 0])
  HS_TRY(launch_gap_bwd(c.bf, G[0], cur, n, 16, 512, G[1], c.s));
  // G[gi]: gradient of the current block's output, already multiplied by the
  // ReLU mask of that output: the data gradient that produces it applies
  // [input of the next block > 0] in its epilogue
  // Weight gradients, and the projection's batch-norm backward, go to the
  // second stream (cs); the buffers it reads are only waited for when the
  // main stream writes them again (GradPool).
  GradPool gp(c.ws, c.s);
  gp.live[1] = true;   // G[1]: gradient of the last block's output
  int gi = 1;
  // the backward sums of the current block's second batch norm, when the
  // data gradient that produced its output gradient took them
  BsumReq carry{};
  for (int bi = (int)m.blocks.size() - 1; bi >= 0; --bi) {
    const BlockL& b = m.blocks[bi];
    const int base = 3 + 5 * bi;
    void *Z1 = S[base], *Hh = S[base + 1], *Z2 = S[base + 2], *ZP = S[base + 3];
    const int in_slot = bi == 0 ? 2 : 3 + 5 * (bi - 1) + 4;      // post-ReLU input
    const void* in = S[in_slot];
    const uint8_t* inb = Bt[in_slot];
    const int64_t rps = (int64_t)b.c1.Ho * b.c1.Wo;
    const int p1 = gi;
    int pz = -1, pz_done = -1;
    // the projection's weight gradient in conv1's launch where the shapes allow
    const bool wfuse = b.proj && wgrad_fuses_proj(cs, b.c1, b.cp);
    if (b.proj) {   // dZP on the second stream, needed only by conv1's data gradient
      if (gp.take(pz) != 0) return hipErrorInvalidValue;
      HS_TRY(fork(c));
      HS_TRY(bn_bwd(cs, b.bp, gp[p1], nullptr, ZP, rps, gp[pz]));          // dZP
      pz_done = side_mark(c);
      if (!wfuse) HS_TRY(conv_wgrad(cs, b.cp, gp[pz], in));
      HS_TRY(gp.read_on_side(pz));
      HS_TRY(gp.read_on_side(p1));
    }
    HS_TAKE(gp, p2);
    HS_TRY(bn_bwd_sums(c, b.b2, carry, gp[p1], Z2, rps, gp[p2]));          // dZ2
    HS_TRY(fork(c));
    HS_TRY(conv_wgrad(cs, b.c2, gp[p2], Hh));
    HS_TRY(gp.read_on_side(p2));
    HS_TAKE(gp, p3);
    BsumReq r1{};
    r1.z = Z1;
    HS_TRY(conv_dgrad(c, b.c2, gp[p2], gp[p3], nullptr, Hh, Bt[base + 1], nullptr, nullptr,
                      nullptr, &r1));                                       // dH * [H > 0]
    gp.drop(p2);
    HS_TAKE(gp, p4);
    HS_TRY(bn_bwd_sums(c, b.b1, r1, gp[p3], Z1, rps, gp[p4]));              // dZ1
    gp.drop(p3);
    HS_TRY(fork(c));
    if (wfuse) {
      HS_TRY(conv_wgrad(cs, b.c1, gp[p4], in, 0, 0.0, &b.cp, gp[pz]));
      HS_TRY(gp.read_on_side(pz));
    } else {
      HS_TRY(conv_wgrad(cs, b.c1, gp[p4], in));
    }
    HS_TRY(gp.read_on_side(p4));
    HS_TAKE(gp, out);
    carry = BsumReq{};
    if (b.proj) {
      HS_TRY(wait_mark(c, pz_done));
      // dIn * [in > 0], the shortcut's data gradient summed in the same pass
      // where the layer shapes allow it, else added from its own output
      bool fused = false;
      HS_TRY(conv_dgrad(c, b.c1, gp[p4], gp[out], nullptr, in, inb, &b.cp, gp[pz], &fused));
      if (!fused) {
        HS_TAKE(gp, sc);
        HS_TRY(conv_dgrad(c, b.cp, gp[pz], gp[sc], nullptr, nullptr));      // shortcut grad
        HS_TRY(conv_dgrad(c, b.c1, gp[p4], gp[out], gp[sc], in, inb));
        gp.drop(sc);
      }
      gp.drop(pz);
    } else {
      // dIn * [in > 0]: the previous block's output gradient, whose second
      // batch norm's sums the epilogue takes (they wait in their own buffer
      // until that block's backward starts)
      carry.z = bi > 0 ? S[3 + 5 * (bi - 1) + 2] : nullptr;
      HS_TRY(conv_dgrad(c, b.c1, gp[p4], gp[out], gp[p1], in, inb, nullptr, nullptr, nullptr,
                        bi > 0 ? &carry : nullptr));
    }
    gp.drop(p4);
    gp.drop(p1);
    gi = out;
  }
  // stem (its ReLU mask is already applied): batch-norm backward and
  // weight gradient; every weight gradient is done when this returns
  HS_TAKE(gp, zs);
  return stem_backward(c, m.stem, m.stem_bn, gp[gi], nullptr, S[1], 1024, gp[zs], S[0], x);
}

// ---------------------------------------------------------- ResNet-50 ----
// Bottleneck blocks: Z1 = conv1(in) (1x1), H1 = relu(bn1(Z1)); Z2 = conv2(H1)
// (3x3, the block's stride), H2 = relu(bn2(Z2)); Z3 = conv3(H2) (1x1),
// out = relu(bn3(Z3) + shortcut), the shortcut being the input or
// bn_p(conv_p(in)) (1x1, the block's stride).
hipError_t resnet_bottleneck(const Ctx& c, const float* x, const int32_t* y, float* loss) {
  const Model& m = c.m;
  void** S = c.ws.slot.data();
  uint8_t* const* Bt = c.ws.bits.data();   // bits of the ReLU outputs
  void** G = c.ws.grad;
  const int n = c.n;
  constexpr int SLOTS = 7;
  const Ctx cs = side(c);   // second stream: projection shortcuts, weight gradients
  HS_TRY(stem_bn_fwd(c, m.stem, m.stem_bn, x, S[0], S[1]));
  HS_TRY(bn_apply(c, m.stem_bn, S[1], nullptr, 1, 1024, S[2], Bt[2]));
  const void* cur = S[2];
  int si = 3;
  for (const BlockL& b : m.blocks) {
    void *Z1 = S[si], *H1 = S[si + 1], *Z2 = S[si + 2], *H2 = S[si + 3], *Z3 = S[si + 4],
         *ZP = S[si + 5], *A = S[si + 6];
    uint8_t *H1b = Bt[si + 1], *H2b = Bt[si + 3], *Ab = Bt[si + 6];
    si += SLOTS;
    const int64_t rin = (int64_t)b.c1.Ho * b.c1.Wo, rout = (int64_t)b.c2.Ho * b.c2.Wo;
    // the projection shortcut on the second stream, beside conv1 .. bn3
    const void* res = cur;
    int proj_done = -1;
    if (b.proj) {
      HS_TRY(fork(c));
      HS_TRY(conv_fwd(cs, b.cp, cur, ZP, false));
      HS_TRY(bn_stats(cs, b.bp, ZP, rout));
      HS_TRY(bn_apply(cs, b.bp, ZP, nullptr, 0, rout, G[0]));
      proj_done = side_mark(c);
      res = G[0];
    }
    HS_TRY(conv_bn_fwd(c, b.c1, cur, Z1, b.b1, rin));
    HS_TRY(bn_apply(c, b.b1, Z1, nullptr, 1, rin, H1, H1b));
    HS_TRY(conv_bn_fwd(c, b.c2, H1, Z2, b.b2, rout));
    HS_TRY(bn_apply(c, b.b2, Z2, nullptr, 1, rout, H2, H2b));
    HS_TRY(conv_bn_fwd(c, b.c3, H2, Z3, b.b3, rout));
    HS_TRY(wait_mark(c, proj_done));
    HS_TRY(bn_apply(c, b.b3, Z3, res, 1, rout, A, Ab));
    cur = A;
  }
  const int cfin = m.blocks.back().c3.cout;
  const int hwfin = m.blocks.back().c3.Ho * m.blocks.back().c3.Wo;
  void* F = S[si];
  HS_TRY(launch_gap_fwd(c.bf, cur, n, hwfin, cfin, F, c.s));
  HS_TRY(conv_fwd(c, m.fc2, F, c.ws.logits, true));
  // ---- backward
  const void* dz;
  HS_TRY(loss_grad(c, y, loss, &dz));
  HS_TRY(conv_wgrad(c, m.fc2, dz, F));
  HS_TRY(bias_grad(c, m.fc2.b, c.ws.dz32, true, 1, 10));
  HS_TRY(conv_dgrad(c, m.fc2, dz, G[0], nullptr, nullptr));           // dF
  HS_TRY(launch_gap_bwd(c.bf, G[0], cur, n, hwfin, cfin, G[1], c.s));  // dA * [A > 0]
  // G[gi]: gradient of the current block's output times its ReLU mask.
  // Weight gradients, and the projection's batch-norm backward, go to the
  // second stream; the buffers it reads are only waited for when the main
  // stream writes them again (GradPool).
  GradPool gp(c.ws, c.s);
  gp.live[1] = true;
  int gi = 1;
  for (int bi = (int)m.blocks.size() - 1; bi >= 0; --bi) {
    const BlockL& b = m.blocks[bi];
    const int base = 3 + SLOTS * bi;
    void *Z1 = S[base], *H1 = S[base + 1], *Z2 = S[base + 2], *H2 = S[base + 3],
         *Z3 = S[base + 4], *ZP = S[base + 5];
    const int in_slot = bi == 0 ? 2 : 3 + SLOTS * (bi - 1) + 6;     // post-ReLU input
    const void* in = S[in_slot];
    const uint8_t* inb = Bt[in_slot];
    const int64_t rin = (int64_t)b.c1.Ho * b.c1.Wo, rout = (int64_t)b.c2.Ho * b.c2.Wo;
    const int p1 = gi;
    int pz = -1, pz_done = -1;
    if (b.proj) {   // dZP on the second stream, needed only by the shortcut's data gradient
      if (gp.take(pz) != 0) return hipErrorInvalidValue;
      HS_TRY(fork(c));
      HS_TRY(bn_bwd(cs, b.bp, gp[p1], nullptr, ZP, rout, gp[pz]));         // dZP
      pz_done = side_mark(c);
      HS_TRY(conv_wgrad(cs, b.cp, gp[pz], in));
      HS_TRY(gp.read_on_side(pz));
      HS_TRY(gp.read_on_side(p1));
    }
    HS_TAKE(gp, p2);
    HS_TRY(bn_bwd(c, b.b3, gp[p1], nullptr, Z3, rout, gp[p2]));             // dZ3
    HS_TRY(fork(c));
    HS_TRY(conv_wgrad(cs, b.c3, gp[p2], H2));
    HS_TRY(gp.read_on_side(p2));
    HS_TAKE(gp, p3);
    HS_TRY(conv_dgrad(c, b.c3, gp[p2], gp[p3], nullptr, H2, Bt[base + 3]));  // dH2 * [H2 > 0]
    gp.drop(p2);
    HS_TAKE(gp, p4);
    HS_TRY(bn_bwd(c, b.b2, gp[p3], nullptr, Z2, rout, gp[p4]));             // dZ2
    gp.drop(p3);
    HS_TRY(fork(c));
    HS_TRY(conv_wgrad(cs, b.c2, gp[p4], H1));
    HS_TRY(gp.read_on_side(p4));
    HS_TAKE(gp, p5);
    HS_TRY(conv_dgrad(c, b.c2, gp[p4], gp[p5], nullptr, H1, Bt[base + 1]));  // dH1 * [H1 > 0]
    gp.drop(p4);
    HS_TAKE(gp, p6);
    HS_TRY(bn_bwd(c, b.b1, gp[p5], nullptr, Z1, rin, gp[p6]));              // dZ1
    gp.drop(p5);
    HS_TRY(fork(c));
    HS_TRY(conv_wgrad(cs, b.c1, gp[p6], in));
    HS_TRY(gp.read_on_side(p6));
    HS_TAKE(gp, out);
    if (b.proj) {
      HS_TRY(wait_mark(c, pz_done));
      HS_TAKE(gp, sc);
      HS_TRY(conv_dgrad(c, b.cp, gp[pz], gp[sc], nullptr, nullptr));        // shortcut grad
      HS_TRY(conv_dgrad(c, b.c1, gp[p6], gp[out], gp[sc], in, inb));        // dIn * [in > 0]
      gp.drop(sc);
      gp.drop(pz);
    } else {
      HS_TRY(conv_dgrad(c, b.c1, gp[p6], gp[out], gp[p1], in, inb));        // dIn * [in > 0]
    }
    gp.drop(p6);
    gp.drop(p1);
    gi = out;
  }
  // the stem's batch-norm backward and weight gradient; every weight
  // gradient is done when this returns
  HS_TAKE(gp, zs);
  return stem_backward(c, m.stem, m.stem_bn, gp[gi], nullptr, S[1], 1024, gp[zs], S[0], x);
}

// -------------------------------------------------------------- VGG-16 ----
hipError_t vgg(const Ctx& c, const float* x, const int32_t* y, float* loss) {
  const Model& m = c.m;
  void** S = c.ws.slot.data();
  void** G = c.ws.grad;
  const int n = c.n;
  const void* cur = S[0];
  const int L = (int)m.vgg.size();
  for (int i = 0; i < L; ++i) {
    const VggL& l = m.vgg[i];
    void *Z = S[1 + 3 * i], *A = S[2 + 3 * i], *P = S[3 + 3 * i];
    const int64_t rps = (int64_t)l.c.Ho * l.c.Wo;
    if (i == 0) {
      HS_TRY(stem_bn_fwd(c, l.c, l.bn, x, S[0], Z));
    } else {
      HS_TRY(conv_bn_fwd(c, l.c, cur, Z, l.bn, rps));
    }
    HS_TRY(bn_apply(c, l.bn, Z, nullptr, 1, rps, A));
    cur = A;
    if (l.pool) {
      HS_TRY(launch_maxpool_fwd(c.bf, A, n, l.c.Ho, l.c.Wo, l.c.cout, P, c.s));
      cur = P;
    }
  }
  const void* F = cur;  // [n][1][1][512]
  void* Hf = S[1 + 3 * L];
  HS_TRY(conv_fwd(c, m.fc1, F, Hf, false));
  HS_TRY(conv_fwd(c, m.fc2, Hf, c.ws.logits, true));
  const void* dz;
  HS_TRY(loss_grad(c, y, loss, &dz));
  HS_TRY(conv_wgrad(c, m.fc2, dz, Hf));
  HS_TRY(bias_grad(c, m.fc2.b, c.ws.dz32, true, 1, 10));
  HS_TRY(conv_dgrad(c, m.fc2, dz, G[0], nullptr, Hf));                // dHf * [Hf > 0]
  HS_TRY(bias_grad(c, m.fc1.b, G[0], false, 1, 512));
  HS_TRY(conv_wgrad(c, m.fc1, G[0], F));
  HS_TRY(conv_dgrad(c, m.fc1, G[0], G[1], nullptr, nullptr));         // dF
  // the conv layers' weight gradients on the second stream (GradPool), the
  // pooling / batch-norm / data-gradient chain on the caller's
  const Ctx cs = side(c);
  GradPool gp(c.ws, c.s);
  gp.live[1] = true;   // G[1]: dF
  int gi = 1;
  for (int i = L - 1; i >= 0; --i) {
    const VggL& l = m.vgg[i];
    void *Z = S[1 + 3 * i], *A = S[2 + 3 * i];
    const void* in = i == 0 ? S[0] : (m.vgg[i - 1].pool ? S[3 + 3 * (i - 1)] : S[2 + 3 * (i - 1)]);
    const int64_t rps = (int64_t)l.c.Ho * l.c.Wo;
    int pa = gi;
    if (l.pool) {
      HS_TAKE(gp, q);
      HS_TRY(launch_maxpool_bwd(c.bf, A, gp[pa], n, l.c.Ho, l.c.Wo, l.c.cout, 0, gp[q], c.s));
      gp.drop(pa);
      pa = q;
    }
    HS_TAKE(gp, dz);
    if (i == 0) {   // the first layer: batch-norm backward and weight gradient
      HS_TRY(stem_backward(c, l.c, l.bn, gp[pa], A, Z, rps, gp[dz], in, x));
      gp.drop(pa);
      break;
    }
    HS_TRY(bn_bwd(c, l.bn, gp[pa], A, Z, rps, gp[dz]));
    gp.drop(pa);
    HS_TRY(fork(c));
    HS_TRY(conv_wgrad(cs, l.c, gp[dz], in));
    HS_TRY(gp.read_on_side(dz));
    HS_TAKE(gp, out);
    HS_TRY(conv_dgrad(c, l.c, gp[dz], gp[out], nullptr, nullptr));
    gp.drop(dz);
    gi = out;
  }
  return hipSuccess;
}

}  // namespace

hipError_t layer_gemm(int mode, bool bf16, const ConvL& L, int n, const void* a, const void* b,
                      void* out, const float* bias, bool out_f32, float* scratch,
                      int64_t scratch_floats, hipStream_t s) {
  Model m;
  m.dtype = bf16 ? HS_BF16 : HS_FP32;
  Workspace ws;
  ws.splitk = scratch;
  ws.splitk_floats = scratch ? scratch_floats : 0;
  if (bf16 && mode != MODE_WGRAD && scratch) {   // scratch holds the packed weights
    ws.wpack = scratch;
    ws.wpack_elems = scratch_floats * 2;
  }
  // weights are addressed at offset 0 of the given operand
  const float* th = bf16 ? nullptr : (const float*)b;
  const bf16_t* tb = bf16 ? (const bf16_t*)b : nullptr;
  ConvL l = L;
  l.w = 0;
  l.b = -1;
  Ctx c{m, ws, th, tb, n, s, bf16, bf16 ? 8 : 4, one_segment(n), {}};
  if (mode == MODE_FWD) return conv_fwd(c, l, a, out, out_f32, b, bias);
  if (mode == MODE_DGRAD) {
    if (out_f32 && bf16) return hipErrorInvalidValue;
    return conv_dgrad(c, l, a, out, nullptr, nullptr);
  }
  c.theta = nullptr;
  c.tbf = nullptr;
  c.g[0] = (float*)out;
  return conv_wgrad(c, l, a, b);
}

hipError_t workers_grad(const Model& m, Workspace& ws, const float* theta,
                        const bf16_t* theta_bf16, const float* x, const int32_t* y, const int* n,
                        int M, float* const* g, float* loss, hipStream_t s, float* gbar,
                        const float* w) {
  if (M < 1 || M > MAX_SEG) return hipErrorInvalidValue;
  if (gbar && !w) return hipErrorInvalidValue;
  Segs sg{};
  sg.count = M;
  sg.n0[0] = 0;
  for (int i = 0; i < M; ++i) sg.n0[i + 1] = sg.n0[i] + n[i];
  Ctx c{m, ws, theta, theta_bf16, sg.n0[M], s, m.dtype == HS_BF16, m.dtype == HS_BF16 ? 8 : 4, sg,
        {}};
  for (int i = 0; i < M; ++i) c.g[i] = gbar ? nullptr : g[i];
  c.gbar = gbar;
  for (int i = 0; i < M; ++i) c.w[i] = gbar ? w[i] : 0.f;
  float* const* zero_bufs = gbar ? &gbar : c.g;
  const int nzero = gbar ? 1 : M;
  if (ws.gaps_by_value)
    HS_TRY(launch_zero_ranges_host(zero_bufs, nzero, m.gaps.data(), (int)(m.gaps.size() / 2), s));
  else
    HS_TRY(launch_zero_ranges(zero_bufs, nzero, ws.gaps, (int)(m.gaps.size() / 2), s));
  // this call's packed weights, on the second stream: every region an
  // earlier call listed, ordered after the work already on the caller's
  // stream (the update of theta_bf16); the first packed launch waits for it
  ws.pack_ready = -1;
  ws.pack_waited = false;
  if (c.bf && ws.side && !ws.packs.empty()) {
    HS_TRY(fork(c));
    PackBatch pb{};
    for (const Workspace::Pack& e : ws.packs) {
      pb.job[pb.count++] = pack_job(e.woff, e.dst, e.mode, e.p);
      if (pb.count == PACK_BATCH) {
        HS_TRY(launch_pack_batch(theta_bf16, ws.packed, pb, ws.side));
        pb.count = 0;
      }
    }
    if (pb.count > 0) HS_TRY(launch_pack_batch(theta_bf16, ws.packed, pb, ws.side));
    ws.pack_ready = side_mark(c);
    if (ws.pack_ready < 0) return hipErrorUnknown;
  }
  hipError_t e;
  if (m.arch == HS_MLP) e = mlp(c, x, y, loss);
  else if (m.arch == HS_SMALLCNN) e = small_cnn(c, x, y, loss);
  else if (m.arch == HS_RESNET18) e = resnet(c, x, y, loss);
  else if (m.arch == HS_RESNET50) e = resnet_bottleneck(c, x, y, loss);
  else e = vgg(c, x, y, loss);
  // the packing is ordered before the caller's stream continues even if no
  // launch used it
  if (e == hipSuccess && ws.pack_ready >= 0 && !ws.pack_waited) e = wait_mark(c, ws.pack_ready);
  ws.pack_ready = -1;
  return e;
}

}  // namespace hs
