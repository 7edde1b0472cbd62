// Forward and stride-1 data-gradient convolutions in bf16 on the 32x32x16
// MFMA, with the gathered operand read straight from global memory.
//
// C[m][n] = sum_k A[m][k] * B[n][k], k = (tap, channel):
//   forward:        m = output pixel, n = output channel, A = input x gathered
//                   at (ho*st - pad + r, wo*st - pad + s), B = W[n][tap][c];
//   data gradient:  m = input pixel, n = input channel, A = dy gathered at
//                   (h + pad - r, w + pad - s), B = W[c][tap][n] (stride 1).
// The reduction runs over slices of 16 channels; within a slice every tap of
// the filter is applied in turn, so the 3x3 taps re-read neighbouring pixels
// of the same 32-byte channel group and those re-reads hit the L1 cache.
//
// Block: 8 waves, 512 x BN output tile; wave w owns rows 64 w .. 64 w + 63 and
// all BN columns.  A fragments never touch LDS: lane l loads the 16 bytes
// (8 channels) of row l % 32 at channel offset 8 (l / 32) that the MFMA
// expects, two taps ahead of their use.  B -- the same for every wave -- is
// staged in LDS once per slice from a packed copy of the weights,
// Bp[slice][tap][kh][N][8] (kh: channel half of the slice), so that both the
// global read and the LDS write of a slice are contiguous and the fragment
// reads (32 consecutive n of one kh plane) are free of bank conflicts.
// One barrier per slice; the next slice's B is fetched into registers while
// the current slice computes.
//
// Patch form (3x3, stride 1, pad 1, whole images per tile: H*W divides 512):
// the gathered loads above cost one L1 tag lookup per row and tap, and that
// address traffic, not the MFMA, bounds the kernel.  In the patch form the
// tile's 512 pixels x 16 channels of a slice are copied once into LDS (two
// planes of 512 x 16 bytes, one per 8-channel half) and every tap reads its A
// fragment there: a tap is a uniform row offset dr * W + ds, and a neighbour
// that lies in the image lies in the tile, so out-of-image taps are a
// per-lane predicate and no zero frame is stored.  Sixteen consecutive lanes
// read sixteen consecutive pixels of one plane: no bank conflicts.  The next
// tap's A and B fragments are read while the current tap's MFMAs run.
#include "kernels.h"

namespace hs {

namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) void* lds_ptr;          // LDS
typedef __attribute__((address_space(1))) const void* gbl_cptr;   // global

enum { EPI_BIAS = 1, EPI_RELU = 2, EPI_ADD = 8, EPI_MASK = 16, EPI_MBITS = 32, EPI_STATS = 64,
       EPI_BSUM = 128 };

constexpr int C2_WAVES = 8;
constexpr int C2_BM = 64 * C2_WAVES;   // rows per block
constexpr int C2_CK = 16;              // channels per slice

__device__ inline uint32_t pack2(float a, float b) {
  f32x2 v = {a, b};
  bf16x2 h = __builtin_convertvector(v, bf16x2);
  uint32_t u;
  __builtin_memcpy(&u, &h, 4);
  return u;
}

__device__ inline float bfl(const bf16_t* p, int64_t i) { return bf2f(p[i]); }

// x plus x of the lane n places over within its row of 16 lanes (DPP row
// rotate)
template <int N>
__device__ inline float add_row_ror(float x) {
  const int y = __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), 0x120 + N, 0xf, 0xf, false);
  return x + __builtin_bit_cast(float, y);
}

// The batch-norm partials of one output tile (TILE rows from row tile_m0 =
// tm * TILE, BN channels from n0) from the sums of its 32 row groups of
// TILE / 32 rows (group gq's two sums at Q[gq / 16] + ((gq % 16) * 2 + k) * BN,
// images are whole groups).  Thread (k, c) < 2 BN adds the groups in order,
// those of other worker segments masked to zero, and writes segment s's
// partial at slot tm + s; where the next tile starts segment s, a zero at
// slot tm + s (slots then increase with (tile, segment) and the slots of
// consecutive segments meet).
template <int BN, int TILE>
__device__ inline void flush_tile_stats(const GemmParams& p, float* const (&Q)[2], int tm, int n0,
                                        int tid) {
  constexpr int G = TILE / 32;
  if (tid >= 2 * BN) return;
  const int k = tid / BN, c = tid % BN;
  const int64_t tile_m0 = (int64_t)tm * TILE;
  const int64_t HW = (int64_t)p.g.Ho * p.g.Wo;
  float v[32];
#pragma unroll
  for (int gq = 0; gq < 32; ++gq) v[gq] = Q[gq >> 4][((gq & 15) * 2 + k) * BN + c];
  // groups of the tile holding output rows
  const int nq = (int)((p.M - tile_m0) / G < 32 ? (p.M - tile_m0) / G : 32);
  for (int sg = 0; sg < p.nseg; ++sg) {
    const int64_t r0 = p.seg_n0[sg] * HW - tile_m0, r1 = p.seg_n0[sg + 1] * HW - tile_m0;
    if (sg > 0 && r0 == TILE) p.stat_part[((int64_t)(tm + sg) * 2 + k) * p.N + n0 + c] = 0.f;
    const int lo = r0 <= 0 ? 0 : (r0 >= (int64_t)G * nq ? nq : (int)(r0 / G));
    const int hi = r1 <= 0 ? 0 : (r1 >= (int64_t)G * nq ? nq : (int)(r1 / G));
    if (lo >= hi) continue;
    float a = 0.f;
#pragma unroll
    for (int gq = 0; gq < 32; ++gq) a += (gq >= lo && gq < hi) ? v[gq] : 0.f;
    p.stat_part[((int64_t)(tm + sg) * 2 + k) * p.N + n0 + c] = a;
  }
}

}  // namespace

// Bp[((s * RS + tap) * 2 + kh) * N + n][e] = B[n][tap][16 s + 8 kh + e]
// forward: B[n][tap][c] = W[n][tap][c]        (W is [N][RS][C])
// data gradient: B[n][tap][c] = W[c][tap][n]  (W is [C][RS][N])
__global__ void pack_weights_kernel(const bf16_t* __restrict__ W, bf16_t* __restrict__ Bp, int N,
                                    int RS, int C, int transpose) {
  const int64_t chunks = (int64_t)(C / C2_CK) * RS * 2 * N;
  for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q < chunks;
       q += (int64_t)gridDim.x * blockDim.x) {
    const int n = (int)(q % N);
    int64_t r = q / N;
    const int kh = (int)(r & 1);
    r >>= 1;
    const int tap = (int)(r % RS);
    const int s = (int)(r / RS);
    const int c0 = s * C2_CK + kh * 8;
    uint4 v;
    if (!transpose) {
      v = *(const uint4*)(W + ((int64_t)n * RS + tap) * C + c0);
    } else {
      uint16_t e[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) e[j] = W[((int64_t)(c0 + j) * RS + tap) * N + n];
      v = make_uint4(e[0] | ((uint32_t)e[1] << 16), e[2] | ((uint32_t)e[3] << 16),
                     e[4] | ((uint32_t)e[5] << 16), e[6] | ((uint32_t)e[7] << 16));
    }
    *(uint4*)(Bp + q * 8) = v;
  }
}

// Several packings in one launch: job blockIdx.y packs theta_bf16 + woff
// into Bp + dst as pack_weights_kernel does.
__global__ void pack_batch_kernel(const bf16_t* __restrict__ W, bf16_t* __restrict__ Bp,
                                  PackBatch b) {
  const PackJob jb = b.job[blockIdx.y];
  const int N = jb.N, RS = jb.RS, C = jb.C;
  const bf16_t* w = W + jb.woff;
  bf16_t* bp = Bp + jb.dst;
  const int64_t chunks = (int64_t)(C / C2_CK) * RS * 2 * N;
  for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q < chunks;
       q += (int64_t)gridDim.x * blockDim.x) {
    const int n = (int)(q % N);
    int64_t r = q / N;
    const int kh = (int)(r & 1);
    r >>= 1;
    const int tap = (int)(r % RS);
    const int s = (int)(r / RS);
    const int c0 = s * C2_CK + kh * 8;
    uint4 v;
    if (!jb.transpose) {
      v = *(const uint4*)(w + ((int64_t)n * RS + tap) * C + c0);
    } else {
      uint16_t e[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) e[j] = w[((int64_t)(c0 + j) * RS + tap) * N + n];
      v = make_uint4(e[0] | ((uint32_t)e[1] << 16), e[2] | ((uint32_t)e[3] << 16),
                     e[4] | ((uint32_t)e[5] << 16), e[6] | ((uint32_t)e[7] << 16));
    }
    *(uint4*)(bp + q * 8) = v;
  }
}

template <int MODE, int BN, int RS, int EPI, bool PATCH>
__global__ __launch_bounds__(512) void conv2_kernel(GemmParams p) {
  constexpr int NB = BN / 32;
  constexpr int SEG = RS * 2 * BN;                 // 16-byte chunks of B per slice
  constexpr int BREG = (SEG + 511) / 512;          // per thread
  // epilogues that read the addend / mask stage each wave's 64 x 32 fp32
  // sub-tile in LDS (row stride 36 floats: conflict-free) and handle it row by
  // row: 4 lanes per row, 8 contiguous channels each
  constexpr bool STAGE_EPI = (EPI & (EPI_ADD | EPI_MASK)) != 0;
  constexpr int EROW = 36;
  constexpr int BS_BYTES = 2 * RS * 2 * BN * 16;
  // patch planes: 512 pixels x 16 bytes, every second plane offset by 128
  // bytes (the two halves of a pixel in different banks); two buffers
  constexpr int PPLANE = C2_BM * 16 + 128;
  constexpr int EPI_BYTES = STAGE_EPI ? C2_WAVES * 64 * EROW * 4 : 0;
  constexpr int SMEM_BYTES = PATCH ? 16 : (BS_BYTES > EPI_BYTES ? BS_BYTES : EPI_BYTES);
  __shared__ __attribute__((aligned(16))) char smem[SMEM_BYTES];
  typedef uint4 BsT[RS][2][BN];
  BsT* Bs = (BsT*)smem;
  float* Ewave = (float*)smem + (threadIdx.x >> 6) * 64 * EROW;   // epilogue staging of this wave
  float* Qst[2] = {nullptr, nullptr};   // statistics: quarter sums of waves 0-3, 4-7

  const ConvGeom& g = p.g;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // row tile tm, column tile tn: with several column tiles, blocks b, b + 8,
  // b + 16, ... (dispatched to the same XCD, whose L2 then serves the rows
  // they share) take the column tiles of one row tile; blocks past the last
  // row tile (grid rounded up to 8) have no work
  int tm, tn;
  if (p.tiles_n > 1) {
    const int b = (int)blockIdx.x;
    tn = (b >> 3) % p.tiles_n;
    tm = (b / (8 * p.tiles_n)) * 8 + (b & 7);
    if ((int64_t)tm * C2_BM >= p.M) return;
  } else {
    tm = (int)blockIdx.x;
    tn = 0;
  }
  const int m0 = tm * C2_BM + wave * 64, n0 = tn * BN;
  const int kh = lane >> 5;
  const int Ctap = MODE == MODE_FWD ? g.C : g.K;   // channels per tap (A side)
  const int Wsrc = MODE == MODE_FWD ? g.W : g.Wo;  // image width of the A tensor
  const int Hsrc = MODE == MODE_FWD ? g.H : g.Ho;
  const int nslices = Ctap / C2_CK;

  f32x16 acc[2][NB];
#pragma unroll
  for (int mb = 0; mb < 2; ++mb)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[mb][nb] = (f32x16){};
  const bf16_t* A = (const bf16_t*)p.a;
  const bf16_t* B = (const bf16_t*)p.b;
  // B chunk i of slice sl (global -> register) and its LDS slot
  auto load_b1 = [&](int sl, int i) -> uint4 {
    const int q = tid + 512 * i;
    uint4 r = make_uint4(0, 0, 0, 0);
    if (q < SEG) {
      const int n = q % BN, rest = q / BN;    // rest = tap * 2 + kh
      r = *(const uint4*)(B + (((int64_t)sl * RS * 2 + rest) * p.N + n0 + n) * 8);
    }
    return r;
  };
  auto store_b1 = [&](int buf, int i, const uint4& r) {
    const int q = tid + 512 * i;
    if (q < SEG) {
      const int n = q % BN, rest = q / BN;
      Bs[buf][rest >> 1][rest & 1][n] = r;
    }
  };


  if constexpr (PATCH) {
    // The two buffers of B and of the patch are distinct LDS arrays and the
    // slice loop is unrolled by two, so that every access names its buffer:
    // the compiler then knows that the copies into one buffer do not alias
    // the fragment reads from the other and waits for them only at the
    // slice's end.  Each B buffer is padded to whole rounds of 512 chunks (no
    // thread's copy is conditional) and is large enough to stage four waves'
    // epilogue tiles.
    constexpr int BBUF = BREG * 512;
    constexpr int BPAD = BBUF * 16 > 4 * 64 * EROW * 4 ? BBUF : 4 * 64 * EROW / 4;
    __shared__ __attribute__((aligned(16))) uint4 sB0[BPAD];
    __shared__ __attribute__((aligned(16))) uint4 sB1[BPAD];
    __shared__ __attribute__((aligned(16))) char sP0[2 * PPLANE];
    __shared__ __attribute__((aligned(16))) char sP1[2 * PPLANE];
    Ewave = (float*)(wave < 4 ? sB0 : sB1) + (wave & 3) * 64 * EROW;
    Qst[0] = (float*)sP0;
    Qst[1] = (float*)sP1;
    static_assert(16 * 2 * BN * 4 <= 2 * PPLANE, "quarter sums fit a patch buffer");

    // Tile rows are whole images: the image-local pixel of tile row q is
    // q % (H * W); bit t of vm[mb] = tap t of that row lies in the image.
    const int tile_m0 = tm * C2_BM;
    const int HW = Hsrc * Wsrc;
    int qa[2];
    uint32_t vm[2];
#pragma unroll
    for (int mb = 0; mb < 2; ++mb) {
      const int q = wave * 64 + 32 * mb + (lane & 31);
      const int pix = q % HW, y = pix / Wsrc, x = pix - (pix / Wsrc) * Wsrc;
      uint32_t bits = 0;
#pragma unroll
      for (int t = 0; t < 9; ++t) {
        const int r = t / 3, c = t % 3;
        const int dr = MODE == MODE_FWD ? r - 1 : 1 - r, dc = MODE == MODE_FWD ? c - 1 : 1 - c;
        if ((unsigned)(y + dr) < (unsigned)Hsrc && (unsigned)(x + dc) < (unsigned)Wsrc) bits |= 1u << t;
      }
      qa[mb] = q;
      vm[mb] = tile_m0 + q < p.M ? bits : 0u;
    }
    // A fragments of tap t from patch buffer P, as read (the read stays in
    // the buffer); out-of-image taps are cleared by mask_a when consumed
    auto read_a = [&](const char* P, int t, uint4 (&ra)[2]) {
      const int r = t / 3, c = t % 3;
      const int dr = MODE == MODE_FWD ? r - 1 : 1 - r, dc = MODE == MODE_FWD ? c - 1 : 1 - c;
      const int toff = dr * Wsrc + dc;
      const char* base = P + kh * PPLANE;
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
        ra[mb] = *(const uint4*)(base + ((qa[mb] + toff) & (C2_BM - 1)) * 16);
    };
    auto mask_a = [&](int t, const uint4& v, int mb) -> uint4 {
      const uint32_t k = 0u - ((vm[mb] >> t) & 1u);
      return make_uint4(v.x & k, v.y & k, v.z & k, v.w & k);
    };
    auto read_b = [&](const uint4* Bb, int t, uint4 (&rb)[NB]) {
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) rb[nb] = Bb[(t * 2 + kh) * BN + nb * 32 + (lane & 31)];
    };
    // Slice sl of B and of the patch into (Bb, P), straight from global memory
    // into LDS (16 bytes per lane, written at the wave's base + 16 * lane; no
    // registers held).  B chunk q = tid + 512 i = (tap * 2 + kh) * BN + n,
    // clamped to the slice's last chunk (the surplus lands in the padding);
    // patch plane h, pixel q = tid; rows past the last image re-read the last
    // row (they only feed output rows that are not stored).
    const int wbase = wave * 64;
    auto dma_slice = [&](int sl, uint4* Bb, char* P) {
#pragma unroll
      for (int i = 0; i < BREG; ++i) {
        int q = tid + 512 * i;
        q = q < SEG ? q : SEG - 1;
        const int n = q % BN, rest = q / BN;
        const bf16_t* src = B + (((int64_t)sl * RS * 2 + rest) * p.N + n0 + n) * 8;
        __builtin_amdgcn_global_load_lds((gbl_cptr)src, (lds_ptr)(Bb + 512 * i + wbase), 16, 0, 0);
      }
      int64_t m = (int64_t)tile_m0 + tid;
      m = m < p.M ? m : p.M - 1;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const bf16_t* src = A + m * Ctap + sl * C2_CK + 8 * h;
        __builtin_amdgcn_global_load_lds((gbl_cptr)src, (lds_ptr)(P + h * PPLANE + wbase * 16), 16, 0, 0);
      }
    };

    uint4 fa[2], fb[NB];
    // one slice from (Bc, Pc) while the next one is copied into (Bn, Pn)
    auto slice = [&](int sl, const uint4* Bc, const char* Pc, uint4* Bn, char* Pn) {
      const bool more = sl + 1 < nslices;
      if (more) dma_slice(sl + 1, Bn, Pn);
      // per tap: mask this tap's A fragments (read during the previous tap),
      // issue the next tap's reads, then the MFMAs; the scheduling barriers
      // keep the reads ahead of the MFMAs that hide their latency
#pragma unroll
      for (int t = 0; t < RS; ++t) {
        const uint4 am[2] = {mask_a(t, fa[0], 0), mask_a(t, fa[1], 1)};
        uint4 na[2], nbv[NB];
        if (t + 1 < RS) {
          read_a(Pc, t + 1, na);
          read_b(Bc, t + 1, nbv);
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int mb = 0; mb < 2; ++mb) {
          bf16x8 av;
          __builtin_memcpy(&av, &am[mb], 16);
#pragma unroll
          for (int nb = 0; nb < NB; ++nb) {
            bf16x8 bv;
            __builtin_memcpy(&bv, &fb[nb], 16);
            acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bv, av, acc[mb][nb], 0, 0, 0);
          }
        }
        __builtin_amdgcn_sched_barrier(0);
        if (t + 1 < RS) {
          fa[0] = na[0];
          fa[1] = na[1];
#pragma unroll
          for (int nb = 0; nb < NB; ++nb) fb[nb] = nbv[nb];
        }
      }
      // this wave's copies have landed; after the barrier every wave's have
      __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");
      __syncthreads();
      if (more) {
        read_a(Pn, 0, fa);
        read_b(Bn, 0, fb);
      }
    };

    static_assert(RS == 9, "patch form: 3x3 filters");
    dma_slice(0, sB0, sP0);
    __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    read_a(sP0, 0, fa);
    read_b(sB0, 0, fb);
    for (int sl = 0; sl < nslices; sl += 2) {
      slice(sl, sB0, sP0, sB1, sP1);
      if (sl + 1 < nslices) slice(sl + 1, sB1, sP1, sB0, sP0);
    }
  } else {
    // rows of this lane: element offset of the pixel origin (may point outside
    // the image; only read when the tap lands inside) and its coordinates
    int apix[2], ay[2], ax[2];
  #pragma unroll
    for (int mb = 0; mb < 2; ++mb) {
      const int m = m0 + 32 * mb + (lane & 31);
      const bool ok = m < p.M;
      const int mm = ok ? m : 0;
      int base;
      if (MODE == MODE_FWD) {
        const int b = (int)fdiv(mm, g.HWo), rem = mm - b * g.Ho * g.Wo;
        const int ho = (int)fdiv(rem, g.Wo_), wo = rem - ho * g.Wo;
        base = b * g.H * g.W * g.C;
        ay[mb] = ho * g.stride - g.pad;
        ax[mb] = wo * g.stride - g.pad;
      } else {
        const int b = (int)fdiv(mm, g.HWi), rem = mm - b * g.H * g.W;
        const int h = (int)fdiv(rem, g.Wi_), w = rem - h * g.W;
        base = b * g.Ho * g.Wo * g.K;
        ay[mb] = h + g.pad;
        ax[mb] = w + g.pad;
      }
      apix[mb] = base + (ay[mb] * Wsrc + ax[mb]) * Ctap + 8 * kh;
      if (!ok) ay[mb] = -(1 << 20);   // every tap out of range
    }

    // A fragment of (slice, tap) for both row blocks: the tap's shift is the
    // same for every lane (dr, ds, element offset)
    auto load_a = [&](int sl, int tap, uint4 (&ra)[2]) {
      const int r = RS == 1 ? 0 : tap / 3, s = RS == 1 ? 0 : tap - 3 * (tap / 3);
      const int dr = MODE == MODE_FWD ? r : -r, ds = MODE == MODE_FWD ? s : -s;
      const int toff = (dr * Wsrc + ds) * Ctap + sl * C2_CK;
  #pragma unroll
      for (int mb = 0; mb < 2; ++mb) {
        const bool ok = (unsigned)(ay[mb] + dr) < (unsigned)Hsrc &&
                        (unsigned)(ax[mb] + ds) < (unsigned)Wsrc;
        ra[mb] = ok ? *(const uint4*)(A + apix[mb] + toff) : make_uint4(0, 0, 0, 0);
      }
    };
    {
      uint4 r0[BREG];
  #pragma unroll
      for (int i = 0; i < BREG; ++i) r0[i] = load_b1(0, i);
  #pragma unroll
      for (int i = 0; i < BREG; ++i) store_b1(0, i, r0[i]);
    }
    // A fragments two steps ahead: cur = step u, nxt = step u + 1
    uint4 cur[2], nxt[2] = {make_uint4(0, 0, 0, 0), make_uint4(0, 0, 0, 0)};
    load_a(0, 0, cur);
    if (RS > 1) load_a(0, 1, nxt);
    else if (nslices > 1) load_a(1, 0, nxt);
    __syncthreads();

    // Next slice's B: with RS >= BREG + 2 taps, chunk i is loaded at tap i and
    // written to the free LDS buffer at tap i + 2 (few registers live);
    // otherwise all chunks are loaded at the first tap and written at the end.
    constexpr bool SPREAD = RS >= BREG + 2;
    for (int sl = 0; sl < nslices; ++sl) {
      const bool more = sl + 1 < nslices;
      const int buf = sl & 1;
      uint4 rb[BREG];
      if (!SPREAD && more) {
  #pragma unroll
        for (int i = 0; i < BREG; ++i) rb[i] = load_b1(sl + 1, i);
      }
  #pragma unroll
      for (int t = 0; t < RS; ++t) {
        if (SPREAD && more) {
          if (t < BREG) rb[t] = load_b1(sl + 1, t);
          if (t >= 2 && t - 2 < BREG) store_b1(buf ^ 1, t - 2, rb[t - 2]);
        }
        const uint4 fa[2] = {cur[0], cur[1]};
        cur[0] = nxt[0];
        cur[1] = nxt[1];
        {   // prefetch step u + 2
          int nt = t + 2, ns = sl;
          while (nt >= RS) {
            nt -= RS;
            ++ns;
          }
          if (ns < nslices) load_a(ns, nt, nxt);
        }
        uint4 fb[NB];
  #pragma unroll
        for (int nb = 0; nb < NB; ++nb) fb[nb] = Bs[buf][t][kh][nb * 32 + (lane & 31)];
  #pragma unroll
        for (int mb = 0; mb < 2; ++mb) {
          bf16x8 av;
          __builtin_memcpy(&av, &fa[mb], 16);
  #pragma unroll
          for (int nb = 0; nb < NB; ++nb) {
            bf16x8 bv;
            __builtin_memcpy(&bv, &fb[nb], 16);
            acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bv, av, acc[mb][nb], 0, 0, 0);
          }
        }
      }
      if (more) {
        if (SPREAD) {
  #pragma unroll
          for (int i = (RS - 2 > 0 ? RS - 2 : 0); i < BREG; ++i) store_b1(buf ^ 1, i, rb[i]);
        } else {
  #pragma unroll
          for (int i = 0; i < BREG; ++i) store_b1(buf ^ 1, i, rb[i]);
        }
      }
      __syncthreads();
    }

  }

  if constexpr ((EPI & EPI_STATS) != 0) {
    // Forward with the batch-norm sums of the stored output per worker
    // segment.  The loop ended with a barrier: B and the patch are no longer
    // read.  Each wave stages its 64 x 32 fp32 chunks in its own region (as
    // below); lane l takes the four consecutive rows 4 (l / 4) + i and the 8
    // channels 8 (l % 4) .. of a chunk, stores them in bf16 and adds the
    // stored values and their squares (bf16 dot products of row pairs,
    // accumulated in fp32).  A row of 16 lanes covers 16
    // consecutive rows (a quarter of the wave's rows, inside one image since
    // images are whole quarters): DPP row rotates by 4 and 8 add its four
    // lanes of each channel group, and lanes 0-3 of the row write the
    // quarter's sums to LDS; flush_tile_stats turns the tile's 32 quarters
    // into one partial per worker segment.
    static_assert(PATCH && MODE == MODE_FWD && EPI == EPI_STATS, "statistics: plain patch forward");
    float* E = Ewave;
    const int c8 = 8 * (lane & 3), r4 = 4 * (lane >> 2);
    float* Qw = Qst[wave >> 2] + ((wave & 3) * 4 + (lane >> 4)) * 2 * BN;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int q = 0; q < 4; ++q)
          *(float4*)(E + (32 * mb + (lane & 31)) * EROW + 8 * q + 4 * kh) =
              make_float4(acc[mb][nb][4 * q], acc[mb][nb][4 * q + 1], acc[mb][nb][4 * q + 2],
                          acc[mb][nb][4 * q + 3]);
      __builtin_amdgcn_wave_barrier();
      float rv[4][8];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = r4 + i, m = m0 + row;
        const float4 lo = *(const float4*)(E + row * EROW + c8);
        const float4 hi = *(const float4*)(E + row * EROW + c8 + 4);
        rv[i][0] = lo.x; rv[i][1] = lo.y; rv[i][2] = lo.z; rv[i][3] = lo.w;
        rv[i][4] = hi.x; rv[i][5] = hi.y; rv[i][6] = hi.z; rv[i][7] = hi.w;
        const uint4 o = make_uint4(pack2(lo.x, lo.y), pack2(lo.z, lo.w), pack2(hi.x, hi.y),
                                   pack2(hi.z, hi.w));
        if (m < p.M) *(uint4*)((bf16_t*)p.out + (int64_t)m * p.N + n0 + nb * 32 + c8) = o;
      }
      __builtin_amdgcn_wave_barrier();
      // per channel: the stored (bf16-rounded) values of rows 0, 1 and 2, 3
      // as pairs; a bf16 dot product adds a pair (with ones) or its squares
      float s0[8], s1[8];
      const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const bf16x2 p01 = __builtin_convertvector((f32x2){rv[0][e], rv[1][e]}, bf16x2);
        const bf16x2 p23 = __builtin_convertvector((f32x2){rv[2][e], rv[3][e]}, bf16x2);
        s0[e] = __builtin_amdgcn_fdot2_f32_bf16(p23, ones, __builtin_amdgcn_fdot2_f32_bf16(p01, ones, 0.f, false), false);
        s1[e] = __builtin_amdgcn_fdot2_f32_bf16(p23, p23, __builtin_amdgcn_fdot2_f32_bf16(p01, p01, 0.f, false), false);
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        s0[e] = add_row_ror<8>(add_row_ror<4>(s0[e]));
        s1[e] = add_row_ror<8>(add_row_ror<4>(s1[e]));
      }
      if ((lane & 12) == 0) {
        float* q0 = Qw + nb * 32 + c8;
        *(float4*)q0 = make_float4(s0[0], s0[1], s0[2], s0[3]);
        *(float4*)(q0 + 4) = make_float4(s0[4], s0[5], s0[6], s0[7]);
        *(float4*)(q0 + BN) = make_float4(s1[0], s1[1], s1[2], s1[3]);
        *(float4*)(q0 + BN + 4) = make_float4(s1[4], s1[5], s1[6], s1[7]);
      }
    }
    __syncthreads();   // every wave's quarter sums are in LDS
    flush_tile_stats<BN, C2_BM>(p, Qst, tm, n0, tid);
    return;
  }

  if constexpr (STAGE_EPI) {
    // The loop ended with a barrier: B is no longer read.  Each wave stages
    // its tile in its own region and reads back only its own rows, so the
    // chunks need no block barrier (one wave's LDS operations run in order).
    // The addend / mask rows of chunk nb + 1 are loaded while chunk nb is
    // written; rows past M re-read row M - 1 and are not stored.
    //
    // With EPI_BSUM (a data gradient whose stored output d is the output
    // gradient of a batch norm with input z, p.bz) the epilogue also takes
    // that batch norm's backward sums, sum d and sum d z per worker, as the
    // forward statistics epilogue takes its sums: lane l handles the four
    // consecutive rows 4 (l / 4) + i, so a row of 16 lanes covers a 16-row
    // quarter inside one image; z is loaded with the addend; per channel the
    // rounded d and z of row pairs go into bf16 dot products; DPP row
    // rotates add the quarter, and flush_tile_stats writes the tile's
    // partials per worker.
    float* E = Ewave;
    constexpr bool EADD = (EPI & EPI_ADD) != 0, EMASK = (EPI & EPI_MASK) != 0;
    constexpr bool EBITS = (EPI & EPI_MBITS) != 0;   // the mask as bits: one byte per lane row
    constexpr bool EBSUM = (EPI & EPI_BSUM) != 0;
    static_assert(!EBSUM || (PATCH && MODE == MODE_DGRAD), "backward sums: patch data gradient");
    auto erow = [&](int i) { return EBSUM ? 4 * (lane >> 2) + i : 16 * i + (lane >> 2); };
    auto epi_off = [&](int nb, int i) -> int64_t {
      const int row = erow(i), c8 = 8 * (lane & 3);
      const int m = m0 + row < p.M ? m0 + row : p.M - 1;
      return (int64_t)m * p.N + n0 + nb * 32 + c8;
    };
    uint4 addv[2][EADD ? 4 : 1], maskv[2][EMASK && !EBITS ? 4 : 1], zv[2][EBSUM ? 4 : 1];
    uint32_t maskb[2][EBITS ? 4 : 1];
    auto load_epi = [&](int nb, int slot) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        if constexpr (EBSUM) zv[slot][i] = *(const uint4*)((const bf16_t*)p.bz + epi_off(nb, i));
        if constexpr (EADD) addv[slot][i] = *(const uint4*)((const bf16_t*)p.addend + epi_off(nb, i));
        if constexpr (EBITS) maskb[slot][i] = p.mbits[epi_off(nb, i) >> 3];
        else if constexpr (EMASK) maskv[slot][i] = *(const uint4*)((const bf16_t*)p.mask + epi_off(nb, i));
      }
    };
    load_epi(0, 0);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      if (nb + 1 < NB) load_epi(nb + 1, (nb + 1) & 1);
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int q = 0; q < 4; ++q)
          *(float4*)(E + (32 * mb + (lane & 31)) * EROW + 8 * q + 4 * kh) =
              make_float4(acc[mb][nb][4 * q], acc[mb][nb][4 * q + 1], acc[mb][nb][4 * q + 2],
                          acc[mb][nb][4 * q + 3]);
      __builtin_amdgcn_wave_barrier();
      uint4 dst[EBSUM ? 4 : 1];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = erow(i), c8 = 8 * (lane & 3);
        const int m = m0 + row;
        const float4 lo = *(const float4*)(E + row * EROW + c8);
        const float4 hi = *(const float4*)(E + row * EROW + c8 + 4);
        float v[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
        if constexpr (EADD) {
          const uint4 u = addv[nb & 1][i];
          const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            v[2 * e] += bf2f((bf16_t)(w[e] & 0xffffu));
            v[2 * e + 1] += bf2f((bf16_t)(w[e] >> 16));
          }
        }
        if constexpr (EBITS) {
          const uint32_t b = maskb[nb & 1][i];
#pragma unroll
          for (int e = 0; e < 8; ++e)
            if (!((b >> e) & 1u)) v[e] = 0.f;
        } else if constexpr (EMASK) {
          const uint4 u = maskv[nb & 1][i];
          const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            if (!(bf2f((bf16_t)(w[e] & 0xffffu)) > 0.f)) v[2 * e] = 0.f;
            if (!(bf2f((bf16_t)(w[e] >> 16)) > 0.f)) v[2 * e + 1] = 0.f;
          }
        }
        const uint4 o = make_uint4(pack2(v[0], v[1]), pack2(v[2], v[3]), pack2(v[4], v[5]), pack2(v[6], v[7]));
        if (m < p.M) *(uint4*)((bf16_t*)p.out + (int64_t)m * p.N + n0 + nb * 32 + c8) = o;
        if constexpr (EBSUM) dst[i] = o;
      }
      __builtin_amdgcn_wave_barrier();
      if constexpr (EBSUM) {
        // per channel pair w (channels 2w, 2w + 1) and row pair (0, 1), (2, 3):
        // the two rows' values of one channel as a bf16 pair (byte selects)
        const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
        float s0[8], s1[8];
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          const uint32_t d0 = ((const uint32_t*)&dst[0])[w], d1 = ((const uint32_t*)&dst[1])[w];
          const uint32_t d2 = ((const uint32_t*)&dst[2])[w], d3 = ((const uint32_t*)&dst[3])[w];
          const uint32_t z0 = ((const uint32_t*)&zv[nb & 1][0])[w], z1 = ((const uint32_t*)&zv[nb & 1][1])[w];
          const uint32_t z2 = ((const uint32_t*)&zv[nb & 1][2])[w], z3 = ((const uint32_t*)&zv[nb & 1][3])[w];
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const uint32_t sel = h ? 0x07060302u : 0x05040100u;   // high or low halves of (b, a)
            bf16x2 pd01, pd23, pz01, pz23;
            const uint32_t ud01 = __builtin_amdgcn_perm(d1, d0, sel), ud23 = __builtin_amdgcn_perm(d3, d2, sel);
            const uint32_t uz01 = __builtin_amdgcn_perm(z1, z0, sel), uz23 = __builtin_amdgcn_perm(z3, z2, sel);
            __builtin_memcpy(&pd01, &ud01, 4);
            __builtin_memcpy(&pd23, &ud23, 4);
            __builtin_memcpy(&pz01, &uz01, 4);
            __builtin_memcpy(&pz23, &uz23, 4);
            const int e = 2 * w + h;
            s0[e] = __builtin_amdgcn_fdot2_f32_bf16(pd23, ones, __builtin_amdgcn_fdot2_f32_bf16(pd01, ones, 0.f, false), false);
            s1[e] = __builtin_amdgcn_fdot2_f32_bf16(pd23, pz23, __builtin_amdgcn_fdot2_f32_bf16(pd01, pz01, 0.f, false), false);
          }
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          s0[e] = add_row_ror<8>(add_row_ror<4>(s0[e]));
          s1[e] = add_row_ror<8>(add_row_ror<4>(s1[e]));
        }
        if ((lane & 12) == 0) {
          float* q0 = Qst[wave >> 2] + ((wave & 3) * 4 + (lane >> 4)) * 2 * BN + nb * 32 + 8 * (lane & 3);
          *(float4*)q0 = make_float4(s0[0], s0[1], s0[2], s0[3]);
          *(float4*)(q0 + 4) = make_float4(s0[4], s0[5], s0[6], s0[7]);
          *(float4*)(q0 + BN) = make_float4(s1[0], s1[1], s1[2], s1[3]);
          *(float4*)(q0 + BN + 4) = make_float4(s1[4], s1[5], s1[6], s1[7]);
        }
      }
    }
    if constexpr (EBSUM) {
      __syncthreads();   // every wave's quarter sums are in LDS
      flush_tile_stats<BN, C2_BM>(p, Qst, tm, n0, tid);
    }
    return;
  }

  // ---- epilogue: lane holds rows m, columns n = 8 q + 4 (l / 32) + 0..3 of
  // every 32 x 32 fragment (q = 0..3)
#pragma unroll
  for (int mb = 0; mb < 2; ++mb) {
    const int m = m0 + 32 * mb + (lane & 31);
    if (m >= p.M) continue;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int n = n0 + nb * 32 + 8 * q + 4 * kh;
        float v[4] = {acc[mb][nb][4 * q], acc[mb][nb][4 * q + 1], acc[mb][nb][4 * q + 2],
                      acc[mb][nb][4 * q + 3]};
        const int64_t off = (int64_t)m * p.N + n;
        if constexpr ((EPI & EPI_BIAS) != 0) {
          const float4 bb = *(const float4*)(p.bias + n);
          v[0] += bb.x; v[1] += bb.y; v[2] += bb.z; v[3] += bb.w;
        }
        if constexpr ((EPI & EPI_ADD) != 0) {
          const uint2 u = *(const uint2*)((const bf16_t*)p.addend + off);
          v[0] += bf2f((bf16_t)(u.x & 0xffffu));
          v[1] += bf2f((bf16_t)(u.x >> 16));
          v[2] += bf2f((bf16_t)(u.y & 0xffffu));
          v[3] += bf2f((bf16_t)(u.y >> 16));
        }
        if constexpr ((EPI & EPI_RELU) != 0) {
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = v[e] > 0.f ? v[e] : 0.f;
        }
        if constexpr ((EPI & EPI_MASK) != 0) {
          const uint2 u = *(const uint2*)((const bf16_t*)p.mask + off);
          if (!(bf2f((bf16_t)(u.x & 0xffffu)) > 0.f)) v[0] = 0.f;
          if (!(bf2f((bf16_t)(u.x >> 16)) > 0.f)) v[1] = 0.f;
          if (!(bf2f((bf16_t)(u.y & 0xffffu)) > 0.f)) v[2] = 0.f;
          if (!(bf2f((bf16_t)(u.y >> 16)) > 0.f)) v[3] = 0.f;
        }
        *(uint2*)((bf16_t*)p.out + off) = make_uint2(pack2(v[0], v[1]), pack2(v[2], v[3]));
      }
    }
  }
}

// ----------------------------------------------------------------------------
// Data gradient of a 3x3, stride-2, pad-1 convolution in the patch form.
//
// With dx[h] = sum over (o, r) with 2 o - 1 + r = h of dy[o] W[r] (per
// dimension), an input pixel of parity a (h = 2 i + a) receives tap r = 1 of
// dy row i when a = 0, and taps r = 2 (dy row i) and r = 0 (dy row i + 1)
// when a = 1.  So the 2 x 2 block of input pixels (2i + a, 2j + b) is a
// function of the dy positions (i, j), (i + 1, j), (i, j + 1), (i + 1, j + 1)
// only: the nine taps of the filter each feed one parity class (a, b), read
// dy at offset (di, dj) in {0, 1}^2 of the class's dy position, and the four
// classes together are one stride-1 contraction over the dy grid whose taps
// go to four accumulators.  A block holds 256 dy positions (whole dy
// images, so a neighbour in the image is in the tile and out-of-image taps
// are a per-lane mask) x 64 input channels; each of its 8 waves owns 32
// positions x 64 channels x 4 classes (eight 32 x 32 accumulators).  The dy
// slice (16 output channels) and the slice's packed weights are copied once
// into LDS (global-to-LDS, double-buffered, as the stride-1 patch kernel) and
// all nine taps read them; the projection shortcut of a residual block (a
// 1 x 1 stride-2 convolution of the same input: class (0, 0) only, dy of the
// shortcut at the same position) runs as further slices with one tap.
// The epilogue stages each (class, 32 channels) tile of a wave in LDS and
// writes rows of 8 channels (16 bytes) to the class's pixels, with the ReLU
// mask bits and the addend of the residual path applied.
// ----------------------------------------------------------------------------
constexpr int S2_POS = 256;   // dy positions per block
constexpr int S2_BN = 64;     // input channels per block
constexpr int S2_CK = 32;     // dy channels per slice (two 16-channel steps)

template <int EPI, bool PROJ>
__global__ __launch_bounds__(512) void conv2s2_kernel(GemmParams p) {
  constexpr int BN = S2_BN, NB = BN / 32, RS = 9;
  constexpr int KK = S2_CK / C2_CK;             // 16-channel steps per slice
  constexpr int NT = RS + (PROJ ? 1 : 0);       // taps per step (the shortcut's last)
  constexpr int SEG = RS * 2 * BN;              // 16-byte B chunks per step (9 taps)
  constexpr int SEG1 = PROJ ? 2 * BN : 0;       // the shortcut's (one tap)
  constexpr int BREG = (KK * (SEG + SEG1) + 511) / 512;
  constexpr int BBUF = BREG * 512;
  constexpr int PPLANE = S2_POS * 16 + 128;
  constexpr int NPL = KK * 2 * (PROJ ? 2 : 1);  // dy planes (8 channels each): main, shortcut
  // dy patch of a slice: [position / 32][piece (8 channels)][position % 32]
  // 16-byte slots, the shortcut's after the main one
  constexpr int AREG = S2_POS * 4 * 16;
  static_assert(KK == 2, "four 8-channel pieces per slice");
  static_assert((PROJ ? 2 : 1) * AREG <= NPL * PPLANE, "dy patches fit their buffers");
  auto aslot = [](int pos, int piece) { return ((pos >> 5) * 4 + piece) * 32 + (pos & 31); };
  constexpr int EROW = 36;
  constexpr bool EADD = (EPI & EPI_ADD) != 0, EBITS = (EPI & EPI_MBITS) != 0;
  static_assert(5 * 32 * EROW * 4 <= BBUF * 16, "epilogue staging of five waves fits a B buffer");
  __shared__ __attribute__((aligned(16))) uint4 sB0[BBUF];
  __shared__ __attribute__((aligned(16))) uint4 sB1[BBUF];
  __shared__ __attribute__((aligned(16))) char sP0[NPL * PPLANE];
  __shared__ __attribute__((aligned(16))) char sP1[NPL * PPLANE];

  const ConvGeom& g = p.g;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // position tile tm, channel tile tn: with several channel tiles, blocks
  // b, b + 8, b + 16, ... (dispatched to the same XCD, whose L2 then serves
  // the dy tile they share) take the channel tiles of one position tile;
  // blocks past the last position tile (grid rounded up to 8) have no work
  int tm, tn;
  if (p.tiles_n > 1) {
    const int b = (int)blockIdx.x;
    tn = (b >> 3) % p.tiles_n;
    tm = (b / (8 * p.tiles_n)) * 8 + (b & 7);
    if ((int64_t)tm * S2_POS >= p.M) return;
  } else {
    tm = (int)blockIdx.x;
    tn = 0;
  }
  const int n0 = tn * BN;
  const int kh = lane >> 5;
  const int Kc = g.K;                           // dy channels (the reduction)
  const int ns = Kc / S2_CK;                    // slices over dy
  const int Ho = g.Ho, Wo = g.Wo, HW = Ho * Wo;
  const int tile_m0 = tm * S2_POS;
  const bf16_t* A = (const bf16_t*)p.a;
  const bf16_t* A2 = (const bf16_t*)p.a2;
  const bf16_t* B = (const bf16_t*)p.b;
  const bf16_t* B2 = (const bf16_t*)p.b2;

  // this lane's dy position (one 32-row block per wave) and its taps' masks:
  // bit t = tap t reads a dy position inside the image; bit 9 = the
  // shortcut's tap (the position itself)
  const int q = wave * 32 + (lane & 31);
  uint32_t vm;
  {
    const int pix = q % HW, i = pix / Wo, j = pix - (pix / Wo) * Wo;
    uint32_t bits = 1u << 9;
#pragma unroll
    for (int t = 0; t < 9; ++t) {
      const int di = t / 3 == 0 ? 1 : 0, dj = t % 3 == 0 ? 1 : 0;
      if (i + di < Ho && j + dj < Wo) bits |= 1u << t;
    }
    vm = tile_m0 + q < p.M ? bits : 0u;
  }

  f32x16 acc[4][NB];
#pragma unroll
  for (int c = 0; c < 4; ++c)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[c][nb] = (f32x16){};

  // The ReLU mask bits of the block's output: its dy positions are whole
  // images, so its dx pixels are the 4 x 256 consecutive pixels from image
  // tile_m0 / HW on; thread t loads the 8 bytes (64 channels of the column
  // tile) of pixels t and t + 512 now, in two coalesced loads, and stores
  // them in LDS for the epilogue after the main loop.
  const int64_t px_total = (int64_t)p.M * 4;
  const int64_t px0 = (int64_t)tile_m0 * 4;
  uint2 mload[2];
#pragma unroll
  for (int r = 0; r < 2; ++r) {
    const int64_t gp = px0 + tid + 512 * r;
    mload[r] = EBITS && gp < px_total
                   ? *(const uint2*)(p.mbits + gp * (p.N / 8) + n0 / 8)
                   : make_uint2(0u, 0u);
  }

  // step u = (16-channel step kk, tap t) of a slice: the dy fragment (8
  // channels of this lane's position, shifted by the tap's dy offset) and the
  // weight fragments of 64 channels
  auto read_tap = [&](const uint4* Bb, const char* P, int u, uint4& ra, uint4 (&rb)[NB]) {
    const int kk = u / NT, t = u - kk * NT;
    if (PROJ && t == RS) {
      ra = *(const uint4*)(P + AREG + aslot(q, 2 * kk + kh) * 16);
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
        rb[nb] = Bb[KK * SEG + (2 * kk + kh) * BN + nb * 32 + (lane & 31)];
    } else {
      const int off = (t / 3 == 0 ? Wo : 0) + (t % 3 == 0 ? 1 : 0);
      ra = *(const uint4*)(P + aslot((q + off) & (S2_POS - 1), 2 * kk + kh) * 16);
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
        rb[nb] = Bb[((kk * RS + t) * 2 + kh) * BN + nb * 32 + (lane & 31)];
    }
  };
  auto masked = [&](uint32_t m, int t, const uint4& v) -> uint4 {
    const uint32_t k = 0u - ((m >> t) & 1u);
    return make_uint4(v.x & k, v.y & k, v.z & k, v.w & k);
  };
  // slice sl of B (and the shortcut's B) and of the dy patches, straight from
  // global memory into LDS; rows past the last image re-read the last row
  // (they feed no stored output).  The packed weights of the slice's KK
  // 16-channel steps are consecutive, so chunk c of the slice is chunk
  // sl * KK * SEG + c of the packed array (likewise for the shortcut).
  const int wbase = wave * 64;
  auto dma_slice = [&](int sl, uint4* Bb, char* P) {
#pragma unroll
    for (int i = 0; i < BREG; ++i) {
      int c = tid + 512 * i;
      const bf16_t* src;
      if (!PROJ || c < KK * SEG) {
        c = c < KK * SEG ? c : KK * SEG - 1;
        const int n = c % BN, rest = c / BN;
        src = B + (((int64_t)sl * KK * RS * 2 + rest) * p.N + n0 + n) * 8;
      } else {
        int c1 = c - KK * SEG;
        c1 = c1 < KK * SEG1 ? c1 : KK * SEG1 - 1;
        const int n = c1 % BN, rest = c1 / BN;
        src = B2 + (((int64_t)sl * KK * 2 + rest) * p.N + n0 + n) * 8;
      }
      __builtin_amdgcn_global_load_lds((gbl_cptr)src, (lds_ptr)(Bb + 512 * i + wbase), 16, 0, 0);
    }
    // wave w copies the 4 pieces of 8 channels of its 32 positions, two
    // pieces per copy: lanes 0-31 one piece, lanes 32-63 the next, so that
    // a position's 64 bytes of the slice are requested together
    int64_t m = (int64_t)tile_m0 + 32 * wave + (lane & 31);
    m = m < p.M ? m : p.M - 1;
#pragma unroll
    for (int inst = 0; inst < 2; ++inst) {
      const int piece = 2 * inst + (lane >> 5);
      const int64_t col = (int64_t)sl * S2_CK + 8 * piece;
      const int dst = aslot(32 * wave, 2 * inst) * 16;
      __builtin_amdgcn_global_load_lds((gbl_cptr)(A + m * Kc + col), (lds_ptr)(P + dst), 16, 0, 0);
      if (PROJ)
        __builtin_amdgcn_global_load_lds((gbl_cptr)(A2 + m * Kc + col), (lds_ptr)(P + AREG + dst),
                                         16, 0, 0);
    }
  };

  uint4 fa, fb[NB];
  // one slice from (Bc, Pc) while the next is copied into (Bn, Pn)
  auto slice = [&](int sl, const uint4* Bc, const char* Pc, uint4* Bn, char* Pn) {
    const bool more = sl + 1 < ns;
    if (more) dma_slice(sl + 1, Bn, Pn);
#pragma unroll
    for (int u = 0; u < KK * NT; ++u) {
      // tap t = (r, s): class (r != 1, s != 1), dy offset (r == 0, s == 0);
      // the shortcut's tap: class (0, 0)
      const int t = u % NT;
      const int cls = t == RS ? 0 : 2 * (t / 3 != 1 ? 1 : 0) + (t % 3 != 1 ? 1 : 0);
      const uint4 am = masked(vm, t, fa);
      uint4 na, nbv[NB];
      if (u + 1 < KK * NT) read_tap(Bc, Pc, u + 1, na, nbv);
      __builtin_amdgcn_sched_barrier(0);
      bf16x8 av;
      __builtin_memcpy(&av, &am, 16);
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        bf16x8 bv;
        __builtin_memcpy(&bv, &fb[nb], 16);
        acc[cls][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bv, av, acc[cls][nb], 0, 0, 0);
      }
      __builtin_amdgcn_sched_barrier(0);
      if (u + 1 < KK * NT) {
        fa = na;
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) fb[nb] = nbv[nb];
      }
    }
    __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (more) read_tap(Bn, Pn, 0, fa, fb);
  };

  dma_slice(0, sB0, sP0);
  __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  read_tap(sB0, sP0, 0, fa, fb);
  for (int sl = 0; sl < ns; sl += 2) {
    slice(sl, sB0, sP0, sB1, sP1);
    if (sl + 1 < ns) slice(sl + 1, sB1, sP1, sB0, sP0);
  }

  // ---- epilogue: per (class, 32 channels), this wave's 32 x 32 tile staged in
  // LDS, then 4 lanes per row write 8 channels each to the class's pixel.
  // The lane's two rows (dy positions) give its pixels' offsets; the mask
  // bytes of all 16 (class, channel half, row) are loaded before the first
  // store, so that their latency is paid once per block.
  float* E = (float*)(wave < 5 ? sB0 : sB1) + (wave < 5 ? wave : wave - 5) * 32 * EROW;
  uint2* mkl = (uint2*)sP0;                     // the block's mask bytes, per dx pixel
  if (EBITS) {
    mkl[tid] = mload[0];
    mkl[tid + 512] = mload[1];
    __syncthreads();
  }
  const int H = g.H, W = g.W;
  const int c8 = 8 * (lane & 3);
  int64_t pbase[2];
  int lpix[2];                                  // dx pixel of class (0, 0), within the block
  bool live[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int q2 = wave * 32 + 16 * i + (lane >> 2);
    const int64_t m = (int64_t)tile_m0 + q2;
    live[i] = m < p.M;
    const int64_t mm = live[i] ? m : 0;
    const int img = (int)(mm / HW), pix = (int)(mm - (int64_t)img * HW);
    const int ii = pix / Wo, jj = pix - (pix / Wo) * Wo;
    pbase[i] = (((int64_t)img * H + 2 * ii) * W + 2 * jj) * p.N + n0 + c8;
    lpix[i] = ((q2 / HW) * H + 2 * ii) * W + 2 * jj;
  }
#pragma unroll
  for (int cls = 0; cls < 4; ++cls) {
    const int a = cls >> 1, b = cls & 1;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
#pragma unroll
      for (int qq = 0; qq < 4; ++qq)
        *(float4*)(E + (lane & 31) * EROW + 8 * qq + 4 * kh) =
            make_float4(acc[cls][nb][4 * qq], acc[cls][nb][4 * qq + 1], acc[cls][nb][4 * qq + 2],
                        acc[cls][nb][4 * qq + 3]);
      __builtin_amdgcn_wave_barrier();
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int row = 16 * i + (lane >> 2);
        const float4 lo = *(const float4*)(E + row * EROW + c8);
        const float4 hi = *(const float4*)(E + row * EROW + c8 + 4);
        if (live[i]) {
          const int64_t off = pbase[i] + ((int64_t)a * W + b) * p.N + nb * 32;
          float v[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
          if constexpr (EADD) {
            const uint4 u = *(const uint4*)((const bf16_t*)p.addend + off);
            const uint32_t w4[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              v[2 * e] += bf2f((bf16_t)(w4[e] & 0xffffu));
              v[2 * e + 1] += bf2f((bf16_t)(w4[e] >> 16));
            }
          }
          if constexpr (EBITS) {
            const uint2 mw = mkl[lpix[i] + a * W + b];
            const uint32_t word = nb == 0 ? mw.x : mw.y;
            const uint32_t bits = (word >> (8 * (lane & 3))) & 0xffu;
#pragma unroll
            for (int e = 0; e < 8; ++e)
              if (!((bits >> e) & 1u)) v[e] = 0.f;
          }
          *(uint4*)((bf16_t*)p.out + off) = make_uint4(pack2(v[0], v[1]), pack2(v[2], v[3]),
                                                       pack2(v[4], v[5]), pack2(v[6], v[7]));
        }
      }
      __builtin_amdgcn_wave_barrier();
    }
  }
}

// ----------------------------------------------------------------------------
// Forward of a 3x3, stride-2, pad-1 convolution in the patch form.
//
// Output position (i, j) reads input pixels (2i + r - 1, 2j + s - 1).  A block
// holds 256 output positions -- whole output images, so their input pixels
// are the 4 x 256 pixels of the same whole input images -- x 128 output
// channels; each of its 8 waves owns 32 positions x 128 channels (four 32 x
// 32 accumulators).  Per 16-channel slice the block copies those 1024 input
// pixels and the slice's packed weights into LDS (global-to-LDS,
// double-buffered); tap (r, s) is a shifted read of the pixel plane.  Only
// r = 0 on output row 0 and s = 0 on output column 0 read outside the image
// (a per-lane mask); the plane offset wraps within the block's pixels there.
// The epilogue stages each 32 x 32 tile in LDS and writes 8-channel rows.
// ----------------------------------------------------------------------------
constexpr int F2_POS = 256;   // output positions per block
constexpr int F2_BN = 128;    // output channels per block

template <bool STATS>
__global__ __launch_bounds__(512) void conv2s2f_kernel(GemmParams p) {
  constexpr int BN = F2_BN, NB = BN / 32, RS = 9;
  constexpr int SEG = RS * 2 * BN;              // 16-byte B chunks per slice
  constexpr int BREG = (SEG + 511) / 512;
  constexpr int BBUF = BREG * 512;
  constexpr int NPIX = 4 * F2_POS;              // input pixels per block
  constexpr int PPLANE = NPIX * 16 + 128;       // one 8-channel half of the slice
  constexpr int EROW = 36;
  static_assert(8 * 32 * EROW * 4 <= BBUF * 16, "epilogue staging fits a B buffer");
  __shared__ __attribute__((aligned(16))) uint4 sB0[BBUF];
  __shared__ __attribute__((aligned(16))) uint4 sB1[BBUF];
  __shared__ __attribute__((aligned(16))) char sP0[2 * PPLANE];
  __shared__ __attribute__((aligned(16))) char sP1[2 * PPLANE];

  const ConvGeom& g = p.g;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int tm, tn;
  if (p.tiles_n > 1) {
    const int b = (int)blockIdx.x;
    tn = (b >> 3) % p.tiles_n;
    tm = (b / (8 * p.tiles_n)) * 8 + (b & 7);
    if ((int64_t)tm * F2_POS >= p.M) return;
  } else {
    tm = (int)blockIdx.x;
    tn = 0;
  }
  const int n0 = tn * BN;
  const int kh = lane >> 5;
  const int C = g.C;
  const int ns = C / C2_CK;
  const int Wo = g.Wo, HWo = g.Ho * Wo, W = g.W, HW = g.H * W;
  const int tile_m0 = tm * F2_POS;
  const int64_t px0 = (int64_t)(tile_m0 / HWo) * HW;   // first input pixel of the block
  const int64_t px_total = (int64_t)g.n * HW;
  const bf16_t* A = (const bf16_t*)p.a;
  const bf16_t* B = (const bf16_t*)p.b;

  // this lane's output position, its pixel base (input pixel (2i - 1, 2j - 1)
  // within the block) and its taps' masks
  const int q = wave * 32 + (lane & 31);
  int pbase;
  uint32_t vm;
  {
    const int pix = q % HWo, i = pix / Wo, j = pix - (pix / Wo) * Wo;
    pbase = (q / HWo) * HW + (2 * i - 1) * W + (2 * j - 1);
    uint32_t bits = 0;
#pragma unroll
    for (int t = 0; t < 9; ++t) {
      const int r = t / 3, s = t % 3;
      if ((i > 0 || r > 0) && (j > 0 || s > 0)) bits |= 1u << t;
    }
    vm = tile_m0 + q < p.M ? bits : 0u;
  }

  f32x16 acc[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) acc[nb] = (f32x16){};

  auto read_tap = [&](const uint4* Bb, const char* P, int t, uint4& ra, uint4 (&rb)[NB]) {
    const int off = (t / 3) * W + (t % 3);
    ra = *(const uint4*)(P + kh * PPLANE + ((pbase + off) & (NPIX - 1)) * 16);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) rb[nb] = Bb[(t * 2 + kh) * BN + nb * 32 + (lane & 31)];
  };
  auto masked = [&](int t, const uint4& v) -> uint4 {
    const uint32_t k = 0u - ((vm >> t) & 1u);
    return make_uint4(v.x & k, v.y & k, v.z & k, v.w & k);
  };
  // slice sl: the packed weights, and the block's input pixels (two 8-channel
  // halves); pixels past the last image re-read the last pixel
  const int wbase = wave * 64;
  auto dma_slice = [&](int sl, uint4* Bb, char* P) {
#pragma unroll
    for (int i = 0; i < BREG; ++i) {
      int c = tid + 512 * i;
      c = c < SEG ? c : SEG - 1;
      const int n = c % BN, rest = c / BN;
      const bf16_t* src = B + (((int64_t)sl * RS * 2 + rest) * p.N + n0 + n) * 8;
      __builtin_amdgcn_global_load_lds((gbl_cptr)src, (lds_ptr)(Bb + 512 * i + wbase), 16, 0, 0);
    }
#pragma unroll
    for (int it = 0; it < 4; ++it) {
      const int c = tid + 512 * it;                // chunk: half c / NPIX, pixel c % NPIX
      const int px = c & (NPIX - 1), h = c / NPIX;
      int64_t gp = px0 + px;
      gp = gp < px_total ? gp : px_total - 1;
      __builtin_amdgcn_global_load_lds((gbl_cptr)(A + gp * C + sl * C2_CK + 8 * h),
                                       (lds_ptr)(P + h * PPLANE +
                                                 ((wbase + 512 * it) & (NPIX - 1)) * 16),
                                       16, 0, 0);
    }
  };

  uint4 fa, fb[NB];
  auto slice = [&](int sl, const uint4* Bc, const char* Pc, uint4* Bn, char* Pn) {
    const bool more = sl + 1 < ns;
    if (more) dma_slice(sl + 1, Bn, Pn);
#pragma unroll
    for (int t = 0; t < RS; ++t) {
      const uint4 am = masked(t, fa);
      uint4 na, nbv[NB];
      if (t + 1 < RS) read_tap(Bc, Pc, t + 1, na, nbv);
      __builtin_amdgcn_sched_barrier(0);
      bf16x8 av;
      __builtin_memcpy(&av, &am, 16);
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        bf16x8 bv;
        __builtin_memcpy(&bv, &fb[nb], 16);
        acc[nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bv, av, acc[nb], 0, 0, 0);
      }
      __builtin_amdgcn_sched_barrier(0);
      if (t + 1 < RS) {
        fa = na;
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) fb[nb] = nbv[nb];
      }
    }
    __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (more) read_tap(Bn, Pn, 0, fa, fb);
  };

  dma_slice(0, sB0, sP0);
  __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  read_tap(sB0, sP0, 0, fa, fb);
  for (int sl = 0; sl < ns; sl += 2) {
    slice(sl, sB0, sP0, sB1, sP1);
    if (sl + 1 < ns) slice(sl + 1, sB1, sP1, sB0, sP0);
  }

  // ---- epilogue: per 32 channels, this wave's 32 x 32 tile staged in LDS
  // (a B buffer, free after the last barrier), then 4 lanes per row write 8
  // channels each
  float* E = (float*)sB0 + wave * 32 * EROW;
  const int c8 = 8 * (lane & 3);
  if constexpr (STATS) {
    // With the batch-norm sums of the stored output per worker segment: lane
    // l takes the two consecutive rows 2 (l / 4) + i, so a row of 16 lanes
    // covers 8 consecutive rows (inside one image: output images are whole
    // 8-row groups); per channel the stored pair's sum and sum of squares
    // (bf16 dot products), DPP row rotates by 4 and 8 over the row's lanes,
    // and lanes 0-3 of each row write the group's sums to a patch buffer
    // (free after the last barrier) for flush_tile_stats.
    static_assert(32 * 2 * BN * 4 <= 2 * PPLANE, "group sums fit a patch buffer");
    float* Qg = (float*)sP0 + (wave * 4 + (lane >> 4)) * 2 * BN;
    const int r2 = 2 * (lane >> 2);
    const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
#pragma unroll
      for (int qq = 0; qq < 4; ++qq)
        *(float4*)(E + (lane & 31) * EROW + 8 * qq + 4 * kh) =
            make_float4(acc[nb][4 * qq], acc[nb][4 * qq + 1], acc[nb][4 * qq + 2], acc[nb][4 * qq + 3]);
      __builtin_amdgcn_wave_barrier();
      float rv[2][8];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int row = r2 + i;
        const int64_t m = (int64_t)tile_m0 + wave * 32 + row;
        const float4 lo = *(const float4*)(E + row * EROW + c8);
        const float4 hi = *(const float4*)(E + row * EROW + c8 + 4);
        rv[i][0] = lo.x; rv[i][1] = lo.y; rv[i][2] = lo.z; rv[i][3] = lo.w;
        rv[i][4] = hi.x; rv[i][5] = hi.y; rv[i][6] = hi.z; rv[i][7] = hi.w;
        if (m < p.M)
          *(uint4*)((bf16_t*)p.out + m * p.N + n0 + nb * 32 + c8) =
              make_uint4(pack2(lo.x, lo.y), pack2(lo.z, lo.w), pack2(hi.x, hi.y), pack2(hi.z, hi.w));
      }
      __builtin_amdgcn_wave_barrier();
      float s0[8], s1[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const bf16x2 p01 = __builtin_convertvector((f32x2){rv[0][e], rv[1][e]}, bf16x2);
        s0[e] = add_row_ror<8>(add_row_ror<4>(__builtin_amdgcn_fdot2_f32_bf16(p01, ones, 0.f, false)));
        s1[e] = add_row_ror<8>(add_row_ror<4>(__builtin_amdgcn_fdot2_f32_bf16(p01, p01, 0.f, false)));
      }
      if ((lane & 12) == 0) {
        float* q0 = Qg + nb * 32 + c8;
        *(float4*)q0 = make_float4(s0[0], s0[1], s0[2], s0[3]);
        *(float4*)(q0 + 4) = make_float4(s0[4], s0[5], s0[6], s0[7]);
        *(float4*)(q0 + BN) = make_float4(s1[0], s1[1], s1[2], s1[3]);
        *(float4*)(q0 + BN + 4) = make_float4(s1[4], s1[5], s1[6], s1[7]);
      }
    }
    __syncthreads();   // every wave's group sums are in LDS
    float* const Q[2] = {(float*)sP0, (float*)sP0 + 16 * 2 * BN};
    flush_tile_stats<BN, F2_POS>(p, Q, tm, n0, tid);
    return;
  }
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
#pragma unroll
    for (int qq = 0; qq < 4; ++qq)
      *(float4*)(E + (lane & 31) * EROW + 8 * qq + 4 * kh) =
          make_float4(acc[nb][4 * qq], acc[nb][4 * qq + 1], acc[nb][4 * qq + 2], acc[nb][4 * qq + 3]);
    __builtin_amdgcn_wave_barrier();
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int row = 16 * i + (lane >> 2);
      const int64_t m = (int64_t)tile_m0 + wave * 32 + row;
      const float4 lo = *(const float4*)(E + row * EROW + c8);
      const float4 hi = *(const float4*)(E + row * EROW + c8 + 4);
      if (m < p.M)
        *(uint4*)((bf16_t*)p.out + m * p.N + n0 + nb * 32 + c8) =
            make_uint4(pack2(lo.x, lo.y), pack2(lo.z, lo.w), pack2(hi.x, hi.y), pack2(hi.z, hi.w));
    }
    __builtin_amdgcn_wave_barrier();
  }
}

// ----------------------------------------------------------------------------
// host side
// ----------------------------------------------------------------------------
int conv2_bn(int N) { return N % 128 == 0 ? 128 : (N % 64 == 0 ? 64 : 0); }

bool conv2_ok(int mode, const GemmParams& p) {
  const ConvGeom& g = p.g;
  const int RS = g.R * g.S;
  if (p.par || p.out_f32) return false;
  if (!(RS == 9 && g.R == 3) && RS != 1) return false;
  if (conv2_bn(p.N) == 0) return false;
  if (mode == MODE_FWD) return g.C % C2_CK == 0 && (g.stride == 1 || g.stride == 2);
  if (mode == MODE_DGRAD) return g.K % C2_CK == 0 && g.stride == 1;
  return false;
}

int64_t conv2_packed_elems(const GemmParams& p, int mode) {
  const int RS = p.g.R * p.g.S;
  const int C = mode == MODE_FWD ? p.g.C : p.g.K;
  return (int64_t)C * RS * p.N;
}

hipError_t launch_pack_weights(const void* W, void* Bp, int mode, const GemmParams& p,
                               hipStream_t s) {
  const ConvGeom& g = p.g;
  const int RS = g.R * g.S;
  const int C = mode == MODE_FWD ? g.C : g.K;
  const int64_t chunks = (int64_t)(C / C2_CK) * RS * 2 * p.N;
  int64_t blocks = (chunks + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(pack_weights_kernel, dim3((unsigned)blocks), dim3(256), 0, s,
                     (const bf16_t*)W, (bf16_t*)Bp, p.N, RS, C, mode == MODE_DGRAD ? 1 : 0);
  return hipGetLastError();
}

PackJob pack_job(int64_t woff, int64_t dst, int mode, const GemmParams& p) {
  PackJob j{};
  j.woff = woff;
  j.dst = dst;
  j.N = p.N;
  j.RS = p.g.R * p.g.S;
  j.C = mode == MODE_FWD ? p.g.C : p.g.K;
  j.transpose = mode == MODE_DGRAD ? 1 : 0;
  return j;
}

hipError_t launch_pack_batch(const void* W, void* Bp, const PackBatch& b, hipStream_t s) {
  if (b.count < 1 || b.count > PACK_BATCH) return hipErrorInvalidValue;
  // blocks per job from the largest job, about 4 chunks per thread (the
  // blocks of smaller jobs past their chunks return at once)
  int64_t most = 0;
  for (int i = 0; i < b.count; ++i) {
    const PackJob& j = b.job[i];
    const int64_t chunks = (int64_t)(j.C / C2_CK) * j.RS * 2 * j.N;
    most = chunks > most ? chunks : most;
  }
  int64_t bx = (most + 1023) / 1024;
  bx = bx < 1 ? 1 : (bx > 1024 ? 1024 : bx);
  hipLaunchKernelGGL(pack_batch_kernel, dim3((unsigned)bx, (unsigned)b.count), dim3(256), 0, s,
                     (const bf16_t*)W, (bf16_t*)Bp, b);
  return hipGetLastError();
}

template <int MODE, int BN, int RS, bool PATCH>
static void launch_epi2(const GemmParams& p, dim3 grid, hipStream_t s) {
  if constexpr (MODE == MODE_FWD) {
    const bool bias = p.bias != nullptr, relu = p.relu != 0;
    if constexpr (PATCH && BN == 128) {
      if (p.stat_part) {   // launch_conv2 checked conv2_stats_ok
        hipLaunchKernelGGL((conv2_kernel<MODE, BN, RS, EPI_STATS, PATCH>), grid, dim3(512), 0, s, p);
        return;
      }
    }
    if (bias && relu) hipLaunchKernelGGL((conv2_kernel<MODE, BN, RS, EPI_BIAS | EPI_RELU, PATCH>), grid, dim3(512), 0, s, p);
    else if (bias) hipLaunchKernelGGL((conv2_kernel<MODE, BN, RS, EPI_BIAS, PATCH>), grid, dim3(512), 0, s, p);
    else if (relu) hipLaunchKernelGGL((conv2_kernel<MODE, BN, RS, EPI_RELU, PATCH>), grid, dim3(512), 0, s, p);
    else hipLaunchKernelGGL((conv2_kernel<MODE, BN, RS, 0, PATCH>), grid, dim3(512), 0, s, p);
  } else {
    const bool add = p.addend != nullptr, mask = p.mask != nullptr || p.mbits != nullptr;
    if constexpr (PATCH && BN == 128) {
      if (p.bz) {   // launch_conv2 checked conv2_bsum_ok
        if (add) hipLaunchKernelGGL((conv2_kernel<MODE, BN, RS, EPI_ADD | EPI_MASK | EPI_MBITS | EPI_BSUM, PATCH>), grid, dim3(512), 0, s, p);
        else hipLaunchKernelGGL((conv2_kernel<MODE, BN, RS, EPI_MASK | EPI_MBITS | EPI_BSUM, PATCH>), grid, dim3(512), 0, s, p);
        return;
      }
    }
    if (add && p.mbits) hipLaunchKernelGGL((conv2_kernel<MODE, BN, RS, EPI_ADD | EPI_MASK | EPI_MBITS, PATCH>), grid, dim3(512), 0, s, p);
    else if (p.mbits) hipLaunchKernelGGL((conv2_kernel<MODE, BN, RS, EPI_MASK | EPI_MBITS, PATCH>), grid, dim3(512), 0, s, p);
    else if (add && mask) hipLaunchKernelGGL((conv2_kernel<MODE, BN, RS, EPI_ADD | EPI_MASK, PATCH>), grid, dim3(512), 0, s, p);
    else if (add) hipLaunchKernelGGL((conv2_kernel<MODE, BN, RS, EPI_ADD, PATCH>), grid, dim3(512), 0, s, p);
    else if (mask) hipLaunchKernelGGL((conv2_kernel<MODE, BN, RS, EPI_MASK, PATCH>), grid, dim3(512), 0, s, p);
    else hipLaunchKernelGGL((conv2_kernel<MODE, BN, RS, 0, PATCH>), grid, dim3(512), 0, s, p);
  }
}

// the patch form: 3x3, stride 1, pad 1, same-size output, whole images per
// 512-row tile
static bool conv2_patch(const GemmParams& p) {
  const ConvGeom& g = p.g;
  const int64_t hw = (int64_t)g.H * g.W;
  return g.R == 3 && g.S == 3 && g.stride == 1 && g.pad == 1 && g.Ho == g.H && g.Wo == g.W &&
         hw >= 1 && C2_BM % hw == 0;
}

template <int MODE>
static hipError_t launch_mode2(const GemmParams& p0, hipStream_t s) {
  GemmParams p = p0;
  const int BN = conv2_bn(p.N);
  const int RS = p.g.R * p.g.S;
  p.tiles_n = p.N / BN;
  const int64_t tiles_m = ceil_div(p.M, C2_BM);
  const dim3 grid((unsigned)(p.tiles_n > 1 ? ceil_div(tiles_m, 8) * 8 * p.tiles_n : tiles_m));
  const bool patch = conv2_patch(p);
  if (BN == 128) {
    if (patch) launch_epi2<MODE, 128, 9, true>(p, grid, s);
    else if (RS == 9) launch_epi2<MODE, 128, 9, false>(p, grid, s);
    else launch_epi2<MODE, 128, 1, false>(p, grid, s);
  } else {
    if (patch) launch_epi2<MODE, 64, 9, true>(p, grid, s);
    else if (RS == 9) launch_epi2<MODE, 64, 9, false>(p, grid, s);
    else launch_epi2<MODE, 64, 1, false>(p, grid, s);
  }
  return hipGetLastError();
}

// the stride-2 data-gradient patch kernel: 3x3, stride 2, pad 1, the input
// exactly twice the dy grid, whole dy images per 256-position tile, channel
// counts in whole slices and column tiles, bf16 output with a mask as bits
// (and optionally an addend); with p.a2 / p.b2 the shortcut's 1 x 1 stride-2
// data gradient is summed into class (0, 0)
bool conv2s2_ok(const GemmParams& p) {
  const ConvGeom& g = p.g;
  const int64_t hw = (int64_t)g.Ho * g.Wo;
  if (p.out_f32 || !p.mbits || p.mask == nullptr) return false;
  if (!(g.R == 3 && g.S == 3 && g.stride == 2 && g.pad == 1)) return false;
  if (g.H != 2 * g.Ho || g.W != 2 * g.Wo || hw < 1 || S2_POS % hw != 0) return false;
  if (g.K % S2_CK != 0 || g.C % S2_BN != 0 || p.N != g.C) return false;
  if ((p.a2 == nullptr) != (p.b2 == nullptr)) return false;
  return true;
}

// p.b (and p.b2) must point to the weights packed for the data gradient
// (launch_pack_weights with MODE_DGRAD: 3x3, and 1x1 for the shortcut)
hipError_t launch_conv2s2(const GemmParams& p0, hipStream_t s) {
  if (!conv2s2_ok(p0)) return hipErrorInvalidValue;
  GemmParams p = p0;
  p.M = p.g.n * p.g.Ho * p.g.Wo;
  p.tiles_n = p.N / S2_BN;
  const int64_t tiles_m = ceil_div(p.M, S2_POS);
  const dim3 grid((unsigned)(p.tiles_n > 1 ? ceil_div(tiles_m, 8) * 8 * p.tiles_n : tiles_m));
  const bool add = p.addend != nullptr, proj = p.a2 != nullptr;
  if (add && proj) hipLaunchKernelGGL((conv2s2_kernel<EPI_ADD | EPI_MBITS, true>), grid, dim3(512), 0, s, p);
  else if (add) hipLaunchKernelGGL((conv2s2_kernel<EPI_ADD | EPI_MBITS, false>), grid, dim3(512), 0, s, p);
  else if (proj) hipLaunchKernelGGL((conv2s2_kernel<EPI_MBITS, true>), grid, dim3(512), 0, s, p);
  else hipLaunchKernelGGL((conv2s2_kernel<EPI_MBITS, false>), grid, dim3(512), 0, s, p);
  return hipGetLastError();
}

// the stride-2 forward patch kernel: 3x3, stride 2, pad 1, the input exactly
// twice the output, whole output images per 256-position tile, input
// channels in whole slices, output channels in 128-wide tiles, a plain bf16
// output (no bias, ReLU or shortcut)
bool conv2s2f_ok(const GemmParams& p) {
  const ConvGeom& g = p.g;
  const int64_t hw = (int64_t)g.Ho * g.Wo;
  if (p.out_f32 || p.bias || p.relu || p.addend || p.mask || p.mbits || p.a2) return false;
  if (!(g.R == 3 && g.S == 3 && g.stride == 2 && g.pad == 1)) return false;
  if (g.H != 2 * g.Ho || g.W != 2 * g.Wo || hw < 1 || F2_POS % hw != 0) return false;
  return g.C % C2_CK == 0 && g.C > 0 && p.N == g.K && g.K % F2_BN == 0;
}

// p.b must point to the weights packed for the forward (launch_pack_weights
// with MODE_FWD and the same p)
hipError_t launch_conv2s2f(const GemmParams& p0, hipStream_t s) {
  if (!conv2s2f_ok(p0)) return hipErrorInvalidValue;
  GemmParams p = p0;
  p.M = p.g.n * p.g.Ho * p.g.Wo;
  p.tiles_n = p.N / F2_BN;
  const int64_t tiles_m = ceil_div(p.M, F2_POS);
  const dim3 grid((unsigned)(p.tiles_n > 1 ? ceil_div(tiles_m, 8) * 8 * p.tiles_n : tiles_m));
  if (p.stat_part) {
    if (!conv2s2f_stats_ok(p)) return hipErrorInvalidValue;
    hipLaunchKernelGGL(conv2s2f_kernel<true>, grid, dim3(512), 0, s, p);
  } else {
    hipLaunchKernelGGL(conv2s2f_kernel<false>, grid, dim3(512), 0, s, p);
  }
  return hipGetLastError();
}

// the statistics map of a forward whose tiles hold whole output images:
// row tile t's partial of segment s at slot t + s
static int stat_slots_by_tile(const GemmParams& p, int64_t tile_rows, int* blk) {
  const int64_t hw = (int64_t)p.g.Ho * p.g.Wo;
  const int tiles_m = (int)ceil_div(p.M, tile_rows);
  for (int s = 0; s < p.nseg; ++s) blk[s] = (int)(p.seg_n0[s] * hw / tile_rows) + s;
  blk[p.nseg] = tiles_m + p.nseg - 1;
  return blk[p.nseg];
}

static bool stat_segments_ok(const GemmParams& p) {
  if (p.nseg < 1 || p.nseg > MAX_SEG || p.seg_n0[0] != 0 || p.seg_n0[p.nseg] != p.g.n) return false;
  for (int i = 0; i < p.nseg; ++i)
    if (p.seg_n0[i + 1] <= p.seg_n0[i]) return false;
  return p.M == (int64_t)p.g.n * p.g.Ho * p.g.Wo;
}

bool conv2s2f_stats_ok(const GemmParams& p) {
  return conv2s2f_ok(p) && ((int64_t)p.g.Ho * p.g.Wo) % (F2_POS / 32) == 0 && stat_segments_ok(p);
}

int conv2s2f_stat_slots(const GemmParams& p, int* blk) { return stat_slots_by_tile(p, F2_POS, blk); }

bool conv2_stats_ok(const GemmParams& p) {
  const ConvGeom& g = p.g;
  if (!conv2_ok(MODE_FWD, p) || !conv2_patch(p) || conv2_bn(p.N) != 128 || p.bias || p.relu)
    return false;
  return (g.H * g.W) % (C2_BM / 32) == 0 && stat_segments_ok(p);
}

int conv2_stat_slots(const GemmParams& p, int* blk) { return stat_slots_by_tile(p, C2_BM, blk); }

bool conv2_bsum_ok(const GemmParams& p) {
  const ConvGeom& g = p.g;
  if (!conv2_ok(MODE_DGRAD, p) || !conv2_patch(p) || conv2_bn(p.N) != 128 || !p.stat_part ||
      !p.bz || !p.mbits || p.out_f32)
    return false;
  return (g.H * g.W) % (C2_BM / 32) == 0 && stat_segments_ok(p);
}

// p.b must point to the packed weights (launch_pack_weights of the same p)
hipError_t launch_conv2(int mode, const GemmParams& p, hipStream_t s) {
  if (!conv2_ok(mode, p)) return hipErrorInvalidValue;
  if (p.bz ? (mode != MODE_DGRAD || !conv2_bsum_ok(p))
           : (p.stat_part && (mode != MODE_FWD || !conv2_stats_ok(p))))
    return hipErrorInvalidValue;
  if (mode == MODE_FWD) return launch_mode2<MODE_FWD>(p, s);
  return launch_mode2<MODE_DGRAD>(p, s);
}

}  // namespace hs
