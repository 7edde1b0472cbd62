// Implicit-GEMM convolution / linear contractions on MFMA, fast path (gfx950).
//
// Same three contractions as igemm.hip (FWD, DGRAD, WGRAD; see there), for
// the layer shapes where every 16-byte chunk of an operand lies inside one
// kernel tap and every 128-byte K slice of the K-contiguous operands lies
// inside one tap (channel counts that are multiples of the slice, or 1x1
// layers).  Differences from the generic kernel:
//  * the tap (r, s) and channel offset of each K slice are tracked
//    incrementally in scalar registers: no division per chunk;
//  * LDS rows are 128 bytes with an XOR swizzle of the 16-byte chunk slot,
//    slot = chunk ^ ((row ^ row >> 3) & 7), instead of padding: the MFMA
//    fragment reads, the K-contiguous stores and the register-transposed
//    stores are all free of bank conflicts (or nearly so), and the LDS
//    footprint drops to 2 x (BM + BN) x 128 bytes;
//  * the transposing loaders pair lanes across two k-quads so that a group of
//    16 lanes writes 16 distinct half-slots;
//  * the epilogue is specialised at compile time (bias / ReLU / fp32 output
//    for FWD; residual addend / ReLU mask for DGRAD), and bf16 outputs use
//    the hardware round-to-nearest-even conversion.
// Waves are arranged WGM x (4 / WGM) over the BM x BN block tile.
#include "kernels.h"

namespace hs {

namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

enum { EPI_BIAS = 1, EPI_RELU = 2, EPI_F32 = 4, EPI_ADD = 8, EPI_MASK = 16, EPI_MBITS = 32,
       EPI_STAGE = 64 };

__device__ inline int swz(int row) { return (row ^ (row >> 3)) & 7; }
__device__ inline int lds_off(int row, int chunk) { return row * 128 + ((chunk ^ swz(row)) << 4); }

__device__ inline uint32_t pack_bf16x2(float a, float b) {
  f32x2 v = {a, b};
  bf16x2 h = __builtin_convertvector(v, bf16x2);
  uint32_t u;
  __builtin_memcpy(&u, &h, 4);
  return u;
}

template <typename T>
__device__ inline float ldf(const T* p, int64_t i);
template <> __device__ inline float ldf<float>(const float* p, int64_t i) { return p[i]; }
template <> __device__ inline float ldf<bf16_t>(const bf16_t* p, int64_t i) { return bf2f(p[i]); }

// transposed store of a 4 x V unit: in[j] holds V row values of k-row j;
// row rowbase + e receives the 4 k values at k position kpos (multiple of 4)
template <typename T>
__device__ inline void unit_store_swz(char* lds, int rowbase, int kpos, const uint4 in[4]);

template <>
__device__ inline void unit_store_swz<float>(char* lds, int rowbase, int kpos, const uint4 in[4]) {
  const uint32_t* w0 = (const uint32_t*)&in[0];
  const uint32_t* w1 = (const uint32_t*)&in[1];
  const uint32_t* w2 = (const uint32_t*)&in[2];
  const uint32_t* w3 = (const uint32_t*)&in[3];
  const int chunk = kpos >> 2;  // 4 floats per chunk
#pragma unroll
  for (int e = 0; e < 4; ++e)
    *(uint4*)(lds + lds_off(rowbase + e, chunk)) = make_uint4(w0[e], w1[e], w2[e], w3[e]);
}

template <>
__device__ inline void unit_store_swz<bf16_t>(char* lds, int rowbase, int kpos, const uint4 in[4]) {
  const uint32_t* w0 = (const uint32_t*)&in[0];
  const uint32_t* w1 = (const uint32_t*)&in[1];
  const uint32_t* w2 = (const uint32_t*)&in[2];
  const uint32_t* w3 = (const uint32_t*)&in[3];
  const int chunk = kpos >> 3, half = (kpos >> 2) & 1;  // 8 bf16 per chunk
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int d = e >> 1;
    uint32_t lo, hi;
    if (e & 1) {
      lo = __builtin_amdgcn_perm(w1[d], w0[d], 0x07060302u);
      hi = __builtin_amdgcn_perm(w3[d], w2[d], 0x07060302u);
    } else {
      lo = __builtin_amdgcn_perm(w1[d], w0[d], 0x05040100u);
      hi = __builtin_amdgcn_perm(w3[d], w2[d], 0x05040100u);
    }
    *(uint2*)(lds + lds_off(rowbase + e, chunk) + half * 8) = make_uint2(lo, hi);
  }
}

// unit index -> (row vector, k quad); RV row vectors, KQ k quads per slice.
// Lanes 0..7 take consecutive row vectors, lanes 8..15 the same row vectors
// at the other k quad of a pair.
__device__ inline void unit_coords(int u, int RV, int& rv, int& kq) {
  const int rv_lo = u & 7, kq_lo = (u >> 3) & 1, rest = u >> 4;
  const int rvh = RV >> 3;
  rv = (rest % rvh) * 8 + rv_lo;
  kq = (rest / rvh) * 2 + kq_lo;
}

}  // namespace

template <typename T, int MODE, int BM, int BN, int WGM, int EPI>
__global__ __launch_bounds__(256) void igemm_fast_kernel(GemmParams p) {
  constexpr int EB = sizeof(T);
  constexpr int V = 16 / EB;          // elements per 16-byte chunk
  constexpr int BKE = 128 / EB;       // elements per K slice
  constexpr int WGN = 4 / WGM;
  constexpr int WTM = BM / WGM, WTN = BN / WGN;  // wave tile
  constexpr int FM = WTM / 16, FN = WTN / 16;
  constexpr bool A_KC = (MODE != MODE_WGRAD);    // A is K-contiguous
  constexpr bool B_KC = (MODE == MODE_FWD);
  // chunks (K-contiguous) or 4 x 16-byte units (transposed) per thread; a
  // 64-row transposed tile has 128 units, so half of the threads load none
  constexpr int A_UNITS = 2 * BM, B_UNITS = 2 * BN;
  constexpr int A_ITEMS = A_KC ? BM / 32 : (A_UNITS + 255) / 256;
  constexpr int B_ITEMS = B_KC ? BN / 32 : (B_UNITS + 255) / 256;
  constexpr int A_REGS = A_KC ? A_ITEMS : 4 * A_ITEMS;
  constexpr int B_REGS = B_KC ? B_ITEMS : 4 * B_ITEMS;
  constexpr int RVA = BM / V, RVB = BN / V;        // row vectors per tile (transposed loads)

  __shared__ __attribute__((aligned(16))) char smem[2 * (BM + BN) * 128];

  const ConvGeom& g = p.g;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave % WGM, wn = wave / WGM;
  // Weight gradients: the tiles of one split read the same dy rows and
  // input pixels.  Workgroups are handed to the 8 XCDs (each with its own
  // L2) in turn, so the block index is remapped to put the tiles of a split
  // on one XCD, where they share those reads: the first 8 q blocks (q =
  // blocks / 8) are dealt so that XCD k gets logical blocks [k q, (k + 1) q)
  // in order; the rest keep their index.
  int bx = blockIdx.x, split = blockIdx.y;
  if constexpr (MODE == MODE_WGRAD) {
    const int nblk = (int)(gridDim.x * gridDim.y), q8 = nblk / 8;
    int lb = (int)(blockIdx.y * gridDim.x + blockIdx.x);
    if (lb < 8 * q8) lb = (lb % 8) * q8 + lb / 8;
    bx = lb % (int)gridDim.x;
    split = lb / (int)gridDim.x;
  }
  const int tm = bx / p.tiles_n, tn = bx - tm * p.tiles_n;
  const int m0 = tm * BM, n0 = tn * BN;
  const int RS = g.R * g.S;
  const int Ctap = (MODE == MODE_FWD) ? g.C : g.K;   // channels per tap along K (A side)
  // parity class of a stride-2 data gradient (blockIdx.z); its K covers the
  // class's taps only
  const bool par = (MODE == MODE_DGRAD) && p.par;
  const int cls = par ? (int)blockIdx.z : 0, ph = cls >> 1, pw = cls & 1;
  // class 0 with a fused 1x1 stride-2 term: one more "tap" (position ntap[0])
  // whose A is a2 at the class pixel's own grid point and whose B is b2
  const bool extra = par && cls == 0 && p.a2 != nullptr;
  const int ktiles = par ? (p.ntap[cls] + (extra ? 1 : 0)) * (g.K / BKE) : p.ktiles;
  int kt0 = split * p.kt_per_split;
  int kt1 = min(kt0 + p.kt_per_split, ktiles);
  int koff = 0, kend = p.K;   // K range of this split (WGRAD: one worker segment)
  if (MODE == MODE_WGRAD && p.nseg > 0) wgrad_split_range(p, BKE, koff, kend, kt0, kt1, split);
  // the fused term reads the grid point (h / 2, w / 2): the centre tap (1, 1)
  // of the 3x3 filter (the term only exists for 3x3, pad 1, stride 2)
  auto tap_id = [&](int t) { return par ? (t < p.ntap[cls] ? p.taps[cls][t] : 4) : t; };

  // ---- per-thread fixed state of the loaders
  int a_base[A_KC ? A_ITEMS : 1], a_pix[A_KC ? A_ITEMS : 1], a_y[A_KC ? A_ITEMS : 1],
      a_x[A_KC ? A_ITEMS : 1];
  bool a_ok[A_KC ? A_ITEMS : 1];
  if constexpr (A_KC) {
#pragma unroll
    for (int i = 0; i < A_ITEMS; ++i) {
      const int m = m0 + (tid >> 3) + 32 * i;
      a_ok[i] = m < p.M;
      const int mm = a_ok[i] ? m : 0;
      if (MODE == MODE_FWD) {
        const int b = (int)fdiv(mm, g.HWo), rem = mm - b * g.Ho * g.Wo;
        const int ho = (int)fdiv(rem, g.Wo_), wo = rem - ho * g.Wo;
        a_base[i] = b * g.H * g.W * g.C;
        a_y[i] = ho * g.stride - g.pad;
        a_x[i] = wo * g.stride - g.pad;
        a_pix[i] = a_y[i] * g.W + a_x[i];
      } else {
        int b, h, w;
        if (par) {
          b = (int)fdiv(mm, p.HWh);
          const int rem = mm - b * p.Hh * p.Wh;
          const int h2 = (int)fdiv(rem, p.Wh_);
          h = 2 * h2 + ph;
          w = 2 * (rem - h2 * p.Wh) + pw;
        } else {
          b = (int)fdiv(mm, g.HWi);
          const int rem = mm - b * g.H * g.W;
          h = (int)fdiv(rem, g.Wi_);
          w = rem - h * g.W;
        }
        a_base[i] = b * g.Ho * g.Wo * g.K;
        a_y[i] = h + g.pad;
        a_x[i] = w + g.pad;
        a_pix[i] = 0;
      }
    }
  }
  // WGRAD B: the rows (tap, ci) of each unit are fixed for the block
  int bu_r[B_KC ? 1 : B_ITEMS], bu_s[B_KC ? 1 : B_ITEMS], bu_ci[B_KC ? 1 : B_ITEMS];
  bool bu_ok[B_KC ? 1 : B_ITEMS];
  if constexpr (MODE == MODE_WGRAD) {
#pragma unroll
    for (int i = 0; i < B_ITEMS; ++i) {
      int rv, kq;
      unit_coords(tid + 256 * i, RVB, rv, kq);
      const int n = n0 + rv * V;
      bu_ok[i] = n < p.N && tid + 256 * i < B_UNITS;
      const int nn = bu_ok[i] ? n : 0;
      const int tap = (int)fdiv(nn, g.Cdiv);
      bu_ci[i] = nn - tap * g.C;
      bu_r[i] = (int)fdiv(tap, g.Sdiv);
      bu_s[i] = tap - bu_r[i] * g.S;
    }
  }

  // K-slice position (A side of FWD / DGRAD, B side of DGRAD): tap and
  // channel offset, advanced by BKE per slice
  // channel counts below the slice width (FWD only): a slice covers BKE / C
  // taps; chunk c of a thread sits at tap offset (c V) / C, channel (c V) % C
  const bool small_c = (MODE == MODE_FWD) && RS != 1 && Ctap < BKE;
  int f_ctap = 0, f_cci = (tid & 7) * V;
  if (small_c) {
    f_ctap = f_cci / Ctap;
    f_cci -= f_ctap * Ctap;
  }
  int cur_tap = 0, cur_c0 = 0;
  if constexpr (MODE != MODE_WGRAD) {
    const int k = kt0 * BKE;
    if (RS == 1) {
      cur_tap = 0;
      cur_c0 = k;
    } else {
      cur_tap = k / Ctap;
      cur_c0 = k - cur_tap * Ctap;
    }
  }

  auto load_tile = [&](int kt, int tpos, int c0, uint4 (&ra)[A_REGS], uint4 (&rb)[B_REGS]) {
    const int kbase = koff + kt * BKE;
    const int tap = tap_id(tpos);
    int r = (RS == 1) ? 0 : tap / g.S;
    int s = (RS == 1) ? 0 : tap - r * g.S;
    const int cchunk = (tid & 7) * V;
    // ---------------- A
    if constexpr (MODE == MODE_FWD) {
      int ci = c0 + cchunk;
      bool kok = ci < g.C;
      if (small_c) {
        const int tc = tap + f_ctap;
        r = (int)fdiv(tc, g.Sdiv);
        s = tc - r * g.S;
        ci = f_cci;
        kok = kbase + cchunk < p.K;
      }
      const int toff = r * g.W + s;
#pragma unroll
      for (int i = 0; i < A_ITEMS; ++i) {
        const int hi = a_y[i] + r, wi = a_x[i] + s;
        const bool ok = a_ok[i] && kok && (unsigned)hi < (unsigned)g.H && (unsigned)wi < (unsigned)g.W;
        ra[i] = ok ? *(const uint4*)((const T*)p.a + a_base[i] + (a_pix[i] + toff) * g.C + ci)
                   : make_uint4(0, 0, 0, 0);
      }
    } else if constexpr (MODE == MODE_DGRAD) {
      const int co = c0 + cchunk;
      const bool kok = co < g.K;
      const T* asrc = (const T*)(extra && tpos == p.ntap[0] ? p.a2 : p.a);
#pragma unroll
      for (int i = 0; i < A_ITEMS; ++i) {
        int ho = a_y[i] - r, wo = a_x[i] - s;
        bool ok = a_ok[i] && kok;
        if (g.stride != 1) {
          ok = ok && ho >= 0 && wo >= 0 && !(ho & 1) && !(wo & 1);
          ho >>= 1;
          wo >>= 1;
        }
        ok = ok && (unsigned)ho < (unsigned)g.Ho && (unsigned)wo < (unsigned)g.Wo;
        ra[i] = ok ? *(const uint4*)(asrc + a_base[i] + (ho * g.Wo + wo) * g.K + co)
                   : make_uint4(0, 0, 0, 0);
      }
    } else {  // WGRAD A: dy[pixel][co], rows = co
#pragma unroll
      for (int i = 0; i < A_ITEMS; ++i) {
        int rv, kq;
        unit_coords(tid + 256 * i, RVA, rv, kq);
        const int row = m0 + rv * V;
        const bool uok = tid + 256 * i < A_UNITS;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int pix = kbase + kq * 4 + j;
          ra[4 * i + j] = (uok && row < p.M && pix < kend)
                              ? *(const uint4*)((const T*)p.a + (int64_t)pix * g.K + row)
                              : make_uint4(0, 0, 0, 0);
        }
      }
    }
    // ---------------- B
    if constexpr (MODE == MODE_FWD) {  // W[n][k]
      const int k = kbase + cchunk;
#pragma unroll
      for (int i = 0; i < B_ITEMS; ++i) {
        const int n = n0 + (tid >> 3) + 32 * i;
        rb[i] = (n < p.N && k < p.K) ? *(const uint4*)((const T*)p.b + (int64_t)n * p.K + k)
                                     : make_uint4(0, 0, 0, 0);
      }
    } else if constexpr (MODE == MODE_DGRAD) {  // W[co][tap][ci], rows = ci (b2: [co][ci])
      const bool xt = extra && tpos == p.ntap[0];
      const T* bsrc = (const T*)(xt ? p.b2 : p.b);
      const int brs = xt ? 1 : RS, btap = xt ? 0 : tap;
#pragma unroll
      for (int i = 0; i < B_ITEMS; ++i) {
        int rv, kq;
        unit_coords(tid + 256 * i, RVB, rv, kq);
        const int row = n0 + rv * V;
        const bool uok = tid + 256 * i < B_UNITS;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int co = c0 + kq * 4 + j;
          rb[4 * i + j] = (uok && row < p.N && co < g.K)
                              ? *(const uint4*)(bsrc + ((int64_t)co * brs + btap) * g.C + row)
                              : make_uint4(0, 0, 0, 0);
        }
      }
    } else {  // WGRAD B: x[pixel shifted by the unit's tap][ci]
#pragma unroll
      for (int i = 0; i < B_ITEMS; ++i) {
        int rv, kq;
        unit_coords(tid + 256 * i, RVB, rv, kq);
        int pix = kbase + kq * 4;
        int b = (int)fdiv(pix < kend ? pix : 0, g.HWo);
        int rem = pix - b * g.Ho * g.Wo;
        int ho = (int)fdiv(rem, g.Wo_), wo = rem - ho * g.Wo;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int hi = ho * g.stride - g.pad + bu_r[i], wi = wo * g.stride - g.pad + bu_s[i];
          const bool ok = bu_ok[i] && pix + j < kend && (unsigned)hi < (unsigned)g.H &&
                          (unsigned)wi < (unsigned)g.W;
          rb[4 * i + j] = ok ? *(const uint4*)((const T*)p.b +
                                               ((int64_t)(b * g.H + hi) * g.W + wi) * g.C + bu_ci[i])
                             : make_uint4(0, 0, 0, 0);
          if (++wo == g.Wo) {
            wo = 0;
            if (++ho == g.Ho) {
              ho = 0;
              ++b;
            }
          }
        }
      }
    }
  };

  auto store_tile = [&](int buf, const uint4 (&ra)[A_REGS], const uint4 (&rb)[B_REGS]) {
    char* As = smem + buf * (BM + BN) * 128;
    char* Bs = As + BM * 128;
    if constexpr (A_KC) {
#pragma unroll
      for (int i = 0; i < A_ITEMS; ++i)
        *(uint4*)(As + lds_off((tid >> 3) + 32 * i, tid & 7)) = ra[i];
    } else {
#pragma unroll
      for (int i = 0; i < A_ITEMS; ++i) {
        if (tid + 256 * i >= A_UNITS) break;
        int rv, kq;
        unit_coords(tid + 256 * i, RVA, rv, kq);
        unit_store_swz<T>(As, rv * V, kq * 4, &ra[4 * i]);
      }
    }
    if constexpr (B_KC) {
#pragma unroll
      for (int i = 0; i < B_ITEMS; ++i)
        *(uint4*)(Bs + lds_off((tid >> 3) + 32 * i, tid & 7)) = rb[i];
    } else {
#pragma unroll
      for (int i = 0; i < B_ITEMS; ++i) {
        if (tid + 256 * i >= B_UNITS) break;
        int rv, kq;
        unit_coords(tid + 256 * i, RVB, rv, kq);
        unit_store_swz<T>(Bs, rv * V, kq * 4, &rb[4 * i]);
      }
    }
  };

  auto advance = [&](int& tap, int& c0) {
    if constexpr (MODE != MODE_WGRAD) {
      if (small_c) {
        tap += BKE / Ctap;
        return;
      }
      c0 += BKE;
      if (RS != 1 && c0 >= Ctap) {
        c0 = 0;
        ++tap;
      }
    }
  };

  f32x4 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = (f32x4){0.f, 0.f, 0.f, 0.f};

  // fragment rows of this lane
  const int arow0 = wm * WTM + (lane & 15), brow0 = wn * WTN + (lane & 15);
  const int kc = lane >> 4;  // 16-byte chunk within a 64-byte k group

  int tap = cur_tap, c0 = cur_c0;
  uint4 ra[A_REGS], rb[B_REGS];
  if (kt0 < kt1) {
    load_tile(kt0, tap, c0, ra, rb);
    store_tile(0, ra, rb);
    advance(tap, c0);
  }
  __syncthreads();

  for (int kt = kt0; kt < kt1; ++kt) {
    const int buf = (kt - kt0) & 1;
    const bool more = kt + 1 < kt1;
    if (more) load_tile(kt + 1, tap, c0, ra, rb);
    const char* As = smem + buf * (BM + BN) * 128;
    const char* Bs = As + BM * 128;
#pragma unroll
    for (int kg = 0; kg < 2; ++kg) {
      uint4 fa[FM], fb[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i) fa[i] = *(const uint4*)(As + lds_off(arow0 + 16 * i, kg * 4 + kc));
#pragma unroll
      for (int j = 0; j < FN; ++j) fb[j] = *(const uint4*)(Bs + lds_off(brow0 + 16 * j, kg * 4 + kc));
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          if constexpr (EB == 4) {
            const float* a4 = (const float*)&fa[i];
            const float* b4 = (const float*)&fb[j];
#pragma unroll
            for (int q = 0; q < 4; ++q)
              acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(b4[q], a4[q], acc[i][j], 0, 0, 0);
          } else {
            bf16x8 av, bv;
            __builtin_memcpy(&av, &fa[i], 16);
            __builtin_memcpy(&bv, &fb[j], 16);
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bv, av, acc[i][j], 0, 0, 0);
          }
        }
    }
    if (more) {
      store_tile(buf ^ 1, ra, rb);
      advance(tap, c0);
    }
    __syncthreads();
  }

  // ---- data-gradient epilogues that read the addend / mask: each wave
  // stages its WTM x CW fp32 sub-tile (CW = WTN, or WTN / 2 when LDS is
  // short; row stride CW + 4 floats, conflict-free) and handles it row by
  // row, 8 channels per lane, so the loads and stores cover contiguous rows
  // (also the bf16 forward outputs: 16-byte row stores instead of 8-byte
  // pieces of 16 rows)
  constexpr bool STAGE_EPI = (MODE == MODE_DGRAD && EB == 2 && (EPI & (EPI_ADD | EPI_MASK)) != 0) ||
                             (MODE == MODE_FWD && EB == 2 && (EPI & EPI_STAGE) != 0);
  if constexpr (STAGE_EPI) {
    constexpr int SMEM = 2 * (BM + BN) * 128;
    constexpr int CW = 4 * WTM * (WTN + 4) * 4 <= SMEM ? WTN : WTN / 2;
    constexpr int EROW = CW + 4, LPR = CW / 8, RPP = 64 / LPR, NRI = WTM / RPP;
    constexpr bool EADD = (EPI & EPI_ADD) != 0, EMASK = (EPI & EPI_MASK) != 0;
    constexpr bool EBITS = (EPI & EPI_MBITS) != 0;   // the mask as bits: one byte per lane row
    static_assert(4 * WTM * EROW * 4 <= SMEM, "epilogue staging exceeds LDS");
    // The main loop ended with a barrier.  Each wave stages its sub-tile in
    // its own region and reads back only its own rows (one wave's LDS
    // operations run in order), so chunks need no block barrier.  All addend
    // / mask rows of a chunk are loaded before any output row is stored (a
    // store between them would order every load after it); rows or columns
    // outside the output re-read element 0 and are not stored.
    float* E = (float*)smem + wave * WTM * EROW;
#pragma unroll
    for (int c0 = 0; c0 < WTN; c0 += CW) {
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          const int col = 16 * j + (lane >> 4) * 4 - c0;
          if (col >= 0 && col < CW)
            *(float4*)(E + (16 * i + (lane & 15)) * EROW + col) =
                make_float4(acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]);
        }
      __builtin_amdgcn_wave_barrier();
      int64_t offs[NRI];
      bool oks[NRI];
      uint4 addv[EADD ? NRI : 1], maskv[EMASK && !EBITS ? NRI : 1];
      uint32_t maskb[EBITS ? NRI : 1];
#pragma unroll
      for (int k = 0; k < NRI; ++k) {
        const int row = k * RPP + lane / LPR, c8 = 8 * (lane % LPR);
        const int m = m0 + wm * WTM + row;
        const int n = n0 + wn * WTN + c0 + c8;
        oks[k] = m < p.M && n < p.N;
        int64_t orow = m;
        if (par) {
          const int b = (int)fdiv(m, p.HWh), rem = m - b * p.Hh * p.Wh;
          const int h2 = (int)fdiv(rem, p.Wh_), w2 = rem - h2 * p.Wh;
          orow = ((int64_t)b * g.H + 2 * h2 + ph) * g.W + 2 * w2 + pw;
        }
        offs[k] = oks[k] ? orow * p.N + n : 0;
        if constexpr (EADD) addv[k] = *(const uint4*)((const bf16_t*)p.addend + offs[k]);
        if constexpr (EBITS) maskb[k] = p.mbits[offs[k] >> 3];
        else if constexpr (EMASK) maskv[k] = *(const uint4*)((const bf16_t*)p.mask + offs[k]);
      }
#pragma unroll
      for (int k = 0; k < NRI; ++k) {
        const int row = k * RPP + lane / LPR, c8 = 8 * (lane % LPR);
        const float4 lo = *(const float4*)(E + row * EROW + c8);
        const float4 hi = *(const float4*)(E + row * EROW + c8 + 4);
        float v[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
        if constexpr ((EPI & EPI_BIAS) != 0) {
          const int n = n0 + wn * WTN + c0 + c8;
          const float4 b0 = *(const float4*)(p.bias + (oks[k] ? n : 0));
          const float4 b1 = *(const float4*)(p.bias + (oks[k] ? n : 0) + 4);
          v[0] += b0.x; v[1] += b0.y; v[2] += b0.z; v[3] += b0.w;
          v[4] += b1.x; v[5] += b1.y; v[6] += b1.z; v[7] += b1.w;
        }
        if constexpr ((EPI & EPI_RELU) != 0) {
#pragma unroll
          for (int e = 0; e < 8; ++e) v[e] = v[e] > 0.f ? v[e] : 0.f;
        }
        if constexpr (EADD) {
          const uint32_t w[4] = {addv[k].x, addv[k].y, addv[k].z, addv[k].w};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            v[2 * e] += bf2f((bf16_t)(w[e] & 0xffffu));
            v[2 * e + 1] += bf2f((bf16_t)(w[e] >> 16));
          }
        }
        if constexpr (EBITS) {
#pragma unroll
          for (int e = 0; e < 8; ++e)
            if (!((maskb[k] >> e) & 1u)) v[e] = 0.f;
        } else if constexpr (EMASK) {
          const uint32_t w[4] = {maskv[k].x, maskv[k].y, maskv[k].z, maskv[k].w};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            if (!(bf2f((bf16_t)(w[e] & 0xffffu)) > 0.f)) v[2 * e] = 0.f;
            if (!(bf2f((bf16_t)(w[e] >> 16)) > 0.f)) v[2 * e + 1] = 0.f;
          }
        }
        if (oks[k])
          *(uint4*)((bf16_t*)p.out + offs[k]) = make_uint4(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]),
                                                           pack_bf16x2(v[4], v[5]), pack_bf16x2(v[6], v[7]));
      }
      __builtin_amdgcn_wave_barrier();
    }
    return;
  }

  // ---- epilogue: lane holds C[m][n .. n+3] of every 16 x 16 fragment
#pragma unroll
  for (int i = 0; i < FM; ++i) {
    const int m = m0 + wm * WTM + 16 * i + (lane & 15);
    if (m >= p.M) continue;
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int n = n0 + wn * WTN + 16 * j + (lane >> 4) * 4;
      if (n >= p.N) continue;
      float v[4] = {acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]};
      if constexpr (MODE == MODE_WGRAD) {
        float* out = (float*)p.out + (int64_t)split * p.split_stride + (int64_t)m * p.N + n;
        *(float4*)out = make_float4(v[0], v[1], v[2], v[3]);
      } else {
        int64_t row = m;
        if (par) {   // scatter the class pixel back to its place in dx
          const int b = (int)fdiv(m, p.HWh), rem = m - b * p.Hh * p.Wh;
          const int h2 = (int)fdiv(rem, p.Wh_), w2 = rem - h2 * p.Wh;
          row = ((int64_t)b * g.H + 2 * h2 + ph) * g.W + 2 * w2 + pw;
        }
        const int64_t off = row * p.N + n;
        if constexpr ((EPI & EPI_BIAS) != 0) {
          const float4 bb = *(const float4*)(p.bias + n);
          v[0] += bb.x; v[1] += bb.y; v[2] += bb.z; v[3] += bb.w;
        }
        if constexpr ((EPI & EPI_ADD) != 0) {
#pragma unroll
          for (int q = 0; q < 4; ++q) v[q] += ldf<T>((const T*)p.addend, off + q);
        }
        if constexpr ((EPI & EPI_RELU) != 0) {
#pragma unroll
          for (int q = 0; q < 4; ++q) v[q] = v[q] > 0.f ? v[q] : 0.f;
        }
        if constexpr ((EPI & EPI_MASK) != 0) {
#pragma unroll
          for (int q = 0; q < 4; ++q)
            if (!(ldf<T>((const T*)p.mask, off + q) > 0.f)) v[q] = 0.f;
        }
        if constexpr ((EPI & EPI_F32) != 0 || EB == 4) {
          *(float4*)((float*)p.out + off) = make_float4(v[0], v[1], v[2], v[3]);
        } else {
          *(uint2*)((bf16_t*)p.out + off) = make_uint2(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]));
        }
      }
    }
  }
}

// ----------------------------------------------------------------------------
// host-side launch
// ----------------------------------------------------------------------------
// Conditions under which the fast kernel applies (the caller falls back to the
// generic kernel otherwise).
bool igemm_fast_ok(int mode, bool bf16, const GemmParams& p, int bm, int bn) {
  const int EB = bf16 ? 2 : 4, V = 16 / EB, BKE = 128 / EB;
  const ConvGeom& g = p.g;
  const int RS = g.R * g.S;
  if (p.N % 4) return false;                         // vector epilogue
  if (g.stride != 1 && g.stride != 2) return false;
  if (mode == MODE_FWD) {
    if (g.C % V) return false;
    if (RS != 1 && g.C % BKE && BKE % g.C) return false;
  } else if (mode == MODE_DGRAD) {
    if (g.K % V || g.C % V) return false;
    if (RS != 1 && g.K % BKE) return false;
  } else {
    if (g.K % V || g.C % V) return false;
  }
  // transposed tiles need at least 8 row vectors
  if (mode != MODE_FWD && bn / V < 8) return false;
  if (mode == MODE_WGRAD && bm / V < 8) return false;
  return true;
}

template <typename T, int MODE, int BM, int BN, int WGM, int EPI>
static void launch_one(const GemmParams& p, dim3 grid, hipStream_t s) {
  hipLaunchKernelGGL((igemm_fast_kernel<T, MODE, BM, BN, WGM, EPI>), grid, dim3(256), 0, s, p);
}

template <typename T, int MODE, int BM, int BN, int WGM>
static void launch_epi(const GemmParams& p, dim3 grid, hipStream_t s) {
  if constexpr (MODE == MODE_FWD) {
    const bool bias = p.bias != nullptr, relu = p.relu != 0, f32 = p.out_f32 != 0 || sizeof(T) == 4;
    if constexpr (sizeof(T) == 2) {
      if (!f32 && p.N % 8 == 0) {   // bf16 output: staged epilogue, 8 channels per lane row
        if (bias && relu) launch_one<T, MODE, BM, BN, WGM, EPI_STAGE | EPI_BIAS | EPI_RELU>(p, grid, s);
        else if (bias) launch_one<T, MODE, BM, BN, WGM, EPI_STAGE | EPI_BIAS>(p, grid, s);
        else if (relu) launch_one<T, MODE, BM, BN, WGM, EPI_STAGE | EPI_RELU>(p, grid, s);
        else launch_one<T, MODE, BM, BN, WGM, EPI_STAGE>(p, grid, s);
        return;
      }
    }
    if (bias && relu && !f32) launch_one<T, MODE, BM, BN, WGM, EPI_BIAS | EPI_RELU>(p, grid, s);
    else if (bias && relu) launch_one<T, MODE, BM, BN, WGM, EPI_BIAS | EPI_RELU | EPI_F32>(p, grid, s);
    else if (bias && !f32) launch_one<T, MODE, BM, BN, WGM, EPI_BIAS>(p, grid, s);
    else if (bias) launch_one<T, MODE, BM, BN, WGM, EPI_BIAS | EPI_F32>(p, grid, s);
    else if (!f32) launch_one<T, MODE, BM, BN, WGM, 0>(p, grid, s);
    else launch_one<T, MODE, BM, BN, WGM, EPI_F32>(p, grid, s);
  } else if constexpr (MODE == MODE_DGRAD) {
    const bool add = p.addend != nullptr, mask = p.mask != nullptr;
    if constexpr (sizeof(T) == 2) {
      if (p.mbits) {   // bf16 data gradients stage their epilogue: the mask as bits
        if (add) launch_one<T, MODE, BM, BN, WGM, EPI_ADD | EPI_MASK | EPI_MBITS>(p, grid, s);
        else launch_one<T, MODE, BM, BN, WGM, EPI_MASK | EPI_MBITS>(p, grid, s);
        return;
      }
    }
    if (add && mask) launch_one<T, MODE, BM, BN, WGM, EPI_ADD | EPI_MASK>(p, grid, s);
    else if (add) launch_one<T, MODE, BM, BN, WGM, EPI_ADD>(p, grid, s);
    else if (mask) launch_one<T, MODE, BM, BN, WGM, EPI_MASK>(p, grid, s);
    else launch_one<T, MODE, BM, BN, WGM, 0>(p, grid, s);
  } else {
    launch_one<T, MODE, BM, BN, WGM, 0>(p, grid, s);
  }
}

template <typename T, int MODE>
static hipError_t launch_tiles_fast(const GemmParams& p0, int bm, int bn, int splits,
                                    hipStream_t s) {
  GemmParams p = p0;
  constexpr int BKE = 128 / (int)sizeof(T);
  const int tiles_m = ceil_div(p.M, bm);
  p.tiles_n = ceil_div(p.N, bn);
  p.ktiles = ceil_div(p.K, BKE);
  if (p.nseg > 0) splits = p.seg_split[p.nseg];   // kt_per_split set by the caller
  else p.kt_per_split = ceil_div(p.ktiles, splits);
  if (p.par) {   // classes differ in K; one split covers the largest
    int mx = 0;
    for (int c = 0; c < 4; ++c) {
      const int nt = p.ntap[c] + (c == 0 && p.a2 ? 1 : 0);
      mx = nt > mx ? nt : mx;
    }
    p.kt_per_split = mx * (p.g.K / BKE);
  }
  const dim3 grid(tiles_m * p.tiles_n, splits, p.par ? 4 : 1);
  // wave layout: all four waves along M when the N tile is 64 wide
  if (bm == 128 && bn == 128) launch_epi<T, MODE, 128, 128, 2>(p, grid, s);
  else if (bm == 128 && bn == 64) launch_epi<T, MODE, 128, 64, 4>(p, grid, s);
  else if (bm == 64 && bn == 128) launch_epi<T, MODE, 64, 128, 1>(p, grid, s);
  else if (bm == 256 && bn == 64) launch_epi<T, MODE, 256, 64, 4>(p, grid, s);
  else if (bm == 64 && bn == 256) launch_epi<T, MODE, 64, 256, 1>(p, grid, s);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_igemm_fast(int mode, bool bf16, const GemmParams& p, int bm, int bn, int splits,
                             hipStream_t s) {
  if (bf16) {
    if (mode == MODE_FWD) return launch_tiles_fast<bf16_t, MODE_FWD>(p, bm, bn, splits, s);
    if (mode == MODE_DGRAD) return launch_tiles_fast<bf16_t, MODE_DGRAD>(p, bm, bn, splits, s);
    return launch_tiles_fast<bf16_t, MODE_WGRAD>(p, bm, bn, splits, s);
  }
  if (mode == MODE_FWD) return launch_tiles_fast<float, MODE_FWD>(p, bm, bn, splits, s);
  if (mode == MODE_DGRAD) return launch_tiles_fast<float, MODE_DGRAD>(p, bm, bn, splits, s);
  return launch_tiles_fast<float, MODE_WGRAD>(p, bm, bn, splits, s);
}

}  // namespace hs
