// Implicit-GEMM convolution / linear kernels on MFMA (gfx950).
//
// One kernel template computes the three contractions of a convolution
// layer (a linear layer is the 1x1 convolution of a 1x1 image):
//
//   FWD    y[p, co]        = sum_{tap, ci} x[p shifted by tap, ci] W[co, tap, ci]
//          GEMM  M = pixels of y, N = c_out, K = taps * c_in
//   DGRAD  dx[p, ci]       = sum_{tap, co} dy[p' : p' * stride + tap = p + pad, co] W[co, tap, ci]
//          GEMM  M = pixels of x, N = c_in,  K = taps * c_out
//   WGRAD  dW[co, tap, ci] = sum_p dy[p, co] x[p shifted by tap, ci]
//          GEMM  M = c_out, N = taps * c_in, K = pixels of y
//
// Tiling: a 256-thread block (4 waves, 2 x 2) owns a BM x BN output tile; each
// wave owns (BM/2) x (BN/2) as 16x16 MFMA tiles.  The K loop moves 128-byte
// K slices (32 fp32 or 64 bf16) of both operands through double-buffered LDS,
// stored K-contiguous ([row][k], 144-byte row pitch) so that every lane reads
// its MFMA fragment with one 16-byte LDS read:
//   fp32: 4 x v_mfma_f32_16x16x4_f32 per 16 k (lane l holds k = 4*(l/16)+q),
//   bf16: 1 x v_mfma_f32_16x16x32_bf16 per 32 k (lane l holds k = 8*(l/16)+q).
// The k order inside a slice is the same for both operands, so the sum is the
// full contraction whatever order the matrix core uses internally.
//
// Operands whose K direction is contiguous in memory (FWD A and B, DGRAD A)
// are copied in 16-byte chunks.  Operands contiguous along the M/N direction
// (DGRAD B = W read across c_in, WGRAD A = dy, WGRAD B = x) are read as 4
// k-rows of 16 bytes and transposed in registers before the LDS store.
//
// The MFMA is issued with the N-side fragment as its first operand, so each
// lane ends up with 4 consecutive output channels of one pixel (16x16 output:
// lane l holds C[m = l%16][n = 4*(l/16) + q]) and stores them as one vector.
#include "kernels.h"

namespace hs {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int PITCH = 144;  // bytes per LDS row: 128 data + 16 pad

template <typename T>
struct ElemBits;
template <> struct ElemBits<float> { typedef uint32_t U; };
template <> struct ElemBits<bf16_t> { typedef uint16_t U; };

// ----------------------------------------------------------------------------
// element-wise (slow path) operand access, used when a 16-byte chunk could
// straddle a tap, a matrix edge or an unaligned address
// ----------------------------------------------------------------------------
template <typename T, int MODE>
__device__ inline typename ElemBits<T>::U elemA(const GemmParams& p, int m, int k, int kend) {
  typedef typename ElemBits<T>::U U;
  const ConvGeom& g = p.g;
  const U* a = (const U*)p.a;
  if (m >= p.M || k >= kend) return 0;
  if (MODE == MODE_FWD) {            // x[b, ho*st-pad+r, wo*st-pad+s, ci]
    int b = m / (g.Ho * g.Wo), rem = m - b * g.Ho * g.Wo;
    int ho = rem / g.Wo, wo = rem - ho * g.Wo;
    int tap = k / g.C, ci = k - tap * g.C;
    int r = tap / g.S, s = tap - r * g.S;
    int hi = ho * g.stride - g.pad + r, wi = wo * g.stride - g.pad + s;
    if (hi < 0 || hi >= g.H || wi < 0 || wi >= g.W) return 0;
    return a[((int64_t)(b * g.H + hi) * g.W + wi) * g.C + ci];
  } else if (MODE == MODE_DGRAD) {   // dy[b, (h+pad-r)/st, (w+pad-s)/st, co]
    int b = m / (g.H * g.W), rem = m - b * g.H * g.W;
    int h = rem / g.W, w = rem - h * g.W;
    int tap = k / g.K, co = k - tap * g.K;
    int r = tap / g.S, s = tap - r * g.S;
    int hn = h + g.pad - r, wn = w + g.pad - s;
    if (hn < 0 || wn < 0 || hn % g.stride || wn % g.stride) return 0;
    int ho = hn / g.stride, wo = wn / g.stride;
    if (ho >= g.Ho || wo >= g.Wo) return 0;
    return a[((int64_t)(b * g.Ho + ho) * g.Wo + wo) * g.K + co];
  } else {                           // dy[p = k, co = m]
    return a[(int64_t)k * g.K + m];
  }
}

template <typename T, int MODE>
__device__ inline typename ElemBits<T>::U elemB(const GemmParams& p, int n, int k, int kend) {
  typedef typename ElemBits<T>::U U;
  const ConvGeom& g = p.g;
  const U* bp = (const U*)p.b;
  if (n >= p.N || k >= kend) return 0;
  if (MODE == MODE_FWD) {            // W[co = n][k]
    return bp[(int64_t)n * p.K + k];
  } else if (MODE == MODE_DGRAD) {   // W[co][tap][ci = n], k = tap * c_out + co
    int tap = k / g.K, co = k - tap * g.K;
    return bp[((int64_t)co * g.R * g.S + tap) * g.C + n];
  } else {                           // x[b, ho*st-pad+r, wo*st-pad+s, ci], n = tap*C+ci, k = p
    int b = k / (g.Ho * g.Wo), rem = k - b * g.Ho * g.Wo;
    int ho = rem / g.Wo, wo = rem - ho * g.Wo;
    int tap = n / g.C, ci = n - tap * g.C;
    int r = tap / g.S, s = tap - r * g.S;
    int hi = ho * g.stride - g.pad + r, wi = wo * g.stride - g.pad + s;
    if (hi < 0 || hi >= g.H || wi < 0 || wi >= g.W) return 0;
    return bp[((int64_t)(b * g.H + hi) * g.W + wi) * g.C + ci];
  }
}

// ----------------------------------------------------------------------------
// fast paths: one 16-byte chunk / one 4 x 16-byte unit
// ----------------------------------------------------------------------------
// Pixel decode of a row of FWD A (output pixel) or DGRAD A (input pixel).
struct RowInfo {
  int base;   // element offset of image b
  int y0, x0; // FWD: ho*st - pad, wo*st - pad;  DGRAD: h + pad, w + pad
  bool ok;
};

template <int MODE>
__device__ inline RowInfo decode_row(const GemmParams& p, int m) {
  const ConvGeom& g = p.g;
  RowInfo ri;
  ri.ok = m < p.M;
  int mm = ri.ok ? m : 0;
  if (MODE == MODE_FWD) {
    int b = (int)fdiv(mm, g.HWo), rem = mm - b * g.Ho * g.Wo;
    int ho = (int)fdiv(rem, g.Wo_), wo = rem - ho * g.Wo;
    ri.base = b * g.H * g.W * g.C;
    ri.y0 = ho * g.stride - g.pad;
    ri.x0 = wo * g.stride - g.pad;
  } else {
    int b = (int)fdiv(mm, g.HWi), rem = mm - b * g.H * g.W;
    int h = (int)fdiv(rem, g.Wi_), w = rem - h * g.W;
    ri.base = b * g.Ho * g.Wo * g.K;
    ri.y0 = h + g.pad;
    ri.x0 = w + g.pad;
  }
  return ri;
}

__device__ inline uint4 zero4() { return make_uint4(0, 0, 0, 0); }

// FWD / DGRAD A chunk: 16 bytes at K offset k of row ri (k multiple of V, and
// the channel count a multiple of V, so the chunk stays inside one tap).
template <typename T, int MODE>
__device__ inline uint4 chunkA(const GemmParams& p, const RowInfo& ri, int k) {
  const ConvGeom& g = p.g;
  if (!ri.ok || k >= p.K) return zero4();
  if (MODE == MODE_FWD) {
    int tap = (int)fdiv(k, g.Cdiv), ci = k - tap * g.C;
    int r = (int)fdiv(tap, g.Sdiv), s = tap - r * g.S;
    int hi = ri.y0 + r, wi = ri.x0 + s;
    if ((unsigned)hi >= (unsigned)g.H || (unsigned)wi >= (unsigned)g.W) return zero4();
    return *(const uint4*)((const T*)p.a + ri.base + (hi * g.W + wi) * g.C + ci);
  } else {
    int tap = (int)fdiv(k, g.Kdiv), co = k - tap * g.K;
    int r = (int)fdiv(tap, g.Sdiv), s = tap - r * g.S;
    int hn = ri.y0 - r, wn = ri.x0 - s;
    int ho, wo;
    if (g.stride == 1) {
      ho = hn;
      wo = wn;
    } else {
      if (hn < 0 || wn < 0 || (hn & 1) || (wn & 1)) return zero4();
      ho = hn >> 1;
      wo = wn >> 1;
    }
    if ((unsigned)ho >= (unsigned)g.Ho || (unsigned)wo >= (unsigned)g.Wo) return zero4();
    return *(const uint4*)((const T*)p.a + ri.base + (ho * g.Wo + wo) * g.K + co);
  }
}

// FWD B chunk: W[n][k .. k+V-1]
template <typename T>
__device__ inline uint4 chunkB_fwd(const GemmParams& p, int n, int k) {
  if (n >= p.N || k >= p.K) return zero4();
  return *(const uint4*)((const T*)p.b + (int64_t)n * p.K + k);
}

// M/N-contiguous unit: rows [row, row+V) at k-rows k..k+3.  out[j] holds the
// V row values of k-row k+j.
template <typename T, int MODE, bool IS_A>
__device__ inline void unit_load(const GemmParams& p, int row, int k, int kend, uint4 out[4]) {
  const ConvGeom& g = p.g;
  if (IS_A) {  // WGRAD A: dy[k][row]
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      int kk = k + j;
      out[j] = (row < p.M && kk < kend) ? *(const uint4*)((const T*)p.a + (int64_t)kk * g.K + row)
                                       : zero4();
    }
  } else if (MODE == MODE_DGRAD) {  // W[co][tap][row], k = tap * c_out + co
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      int kk = k + j;
      if (row < p.N && kk < kend) {
        int tap = (int)fdiv(kk, g.Kdiv), co = kk - tap * g.K;
        out[j] = *(const uint4*)((const T*)p.b + ((int64_t)co * g.R * g.S + tap) * g.C + row);
      } else {
        out[j] = zero4();
      }
    }
  } else {  // WGRAD B: x[pixel k shifted by tap(row)][ci(row)]
    int tap = (int)fdiv(row < p.N ? row : 0, g.Cdiv), ci = row - tap * g.C;
    int r = (int)fdiv(tap, g.Sdiv), s = tap - r * g.S;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      int kk = k + j;
      out[j] = zero4();
      if (row < p.N && kk < kend) {
        int b = (int)fdiv(kk, g.HWo), rem = kk - b * g.Ho * g.Wo;
        int ho = (int)fdiv(rem, g.Wo_), wo = rem - ho * g.Wo;
        int hi = ho * g.stride - g.pad + r, wi = wo * g.stride - g.pad + s;
        if ((unsigned)hi < (unsigned)g.H && (unsigned)wi < (unsigned)g.W)
          out[j] = *(const uint4*)((const T*)p.b + ((int64_t)(b * g.H + hi) * g.W + wi) * g.C + ci);
      }
    }
  }
}

// Store a transposed unit into LDS: row r = rowbase + e gets the 4 k values.
template <typename T>
__device__ inline void unit_store(char* lds, int rowbase, int kbyte, const uint4 in[4]);

template <>
__device__ inline void unit_store<float>(char* lds, int rowbase, int kbyte, const uint4 in[4]) {
  const uint32_t* w0 = (const uint32_t*)&in[0];
  const uint32_t* w1 = (const uint32_t*)&in[1];
  const uint32_t* w2 = (const uint32_t*)&in[2];
  const uint32_t* w3 = (const uint32_t*)&in[3];
#pragma unroll
  for (int e = 0; e < 4; ++e)
    *(uint4*)(lds + (rowbase + e) * PITCH + kbyte) = make_uint4(w0[e], w1[e], w2[e], w3[e]);
}

template <>
__device__ inline void unit_store<bf16_t>(char* lds, int rowbase, int kbyte, const uint4 in[4]) {
  const uint32_t* w0 = (const uint32_t*)&in[0];
  const uint32_t* w1 = (const uint32_t*)&in[1];
  const uint32_t* w2 = (const uint32_t*)&in[2];
  const uint32_t* w3 = (const uint32_t*)&in[3];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    int d = e >> 1;
    uint32_t lo, hi;
    if (e & 1) {
      lo = (w0[d] >> 16) | (w1[d] & 0xffff0000u);
      hi = (w2[d] >> 16) | (w3[d] & 0xffff0000u);
    } else {
      lo = (w0[d] & 0xffffu) | (w1[d] << 16);
      hi = (w2[d] & 0xffffu) | (w3[d] << 16);
    }
    *(uint2*)(lds + (rowbase + e) * PITCH + kbyte) = make_uint2(lo, hi);
  }
}

// ----------------------------------------------------------------------------
// the kernel
// ----------------------------------------------------------------------------
template <typename T, int MODE, int BM, int BN, bool VECA, bool VECB>
__global__ __launch_bounds__(256) void igemm_kernel(GemmParams p) {
  typedef typename ElemBits<T>::U U;
  constexpr int EB = sizeof(T);
  constexpr int V = 16 / EB;        // elements per 16-byte chunk
  constexpr int BKE = 128 / EB;     // elements per K slice
  constexpr int FM = BM / 32, FN = BN / 32;
  constexpr bool A_KCONTIG = (MODE != MODE_WGRAD);
  constexpr bool B_KCONTIG = (MODE == MODE_FWD);
  constexpr int A_ITEMS = A_KCONTIG ? BM / 32 : (2 * BM + 255) / 256;
  constexpr int B_ITEMS = B_KCONTIG ? BN / 32 : (2 * BN + 255) / 256;
  constexpr int A_REGS = A_KCONTIG ? A_ITEMS : 4 * A_ITEMS;
  constexpr int B_REGS = B_KCONTIG ? B_ITEMS : 4 * B_ITEMS;

  __shared__ __attribute__((aligned(16))) char smem[2 * (BM + BN) * PITCH];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int tile = blockIdx.x;
  const int tm = tile / p.tiles_n, tn = tile - tm * p.tiles_n;
  const int m0 = tm * BM, n0 = tn * BN;
  int kt0 = blockIdx.y * p.kt_per_split;
  int kt1 = kt0 + p.kt_per_split;
  if (kt1 > p.ktiles) kt1 = p.ktiles;
  int koff = 0, kend = p.K;   // K range of this split (WGRAD: one worker segment)
  if (MODE == MODE_WGRAD && p.nseg > 0) wgrad_split_range(p, BKE, koff, kend, kt0, kt1);

  // per-thread row decode for K-contiguous A (FWD / DGRAD)
  RowInfo rinfo[A_KCONTIG ? A_ITEMS : 1];
  if (A_KCONTIG && VECA) {
#pragma unroll
    for (int i = 0; i < A_ITEMS; ++i) rinfo[i] = decode_row<MODE>(p, m0 + (tid >> 3) + 32 * i);
  }

  uint4 ra[A_REGS], rb[B_REGS];

  auto load_tile = [&](int kt) {
    const int kbase = koff + kt * BKE;
    // ---- A
    if (A_KCONTIG) {
      const int k = kbase + (tid & 7) * V;
#pragma unroll
      for (int i = 0; i < A_ITEMS; ++i) {
        if (VECA) {
          ra[i] = chunkA<T, MODE>(p, rinfo[i], k);
        } else {
          const int m = m0 + (tid >> 3) + 32 * i;
          U tmp[V];
#pragma unroll
          for (int e = 0; e < V; ++e) tmp[e] = elemA<T, MODE>(p, m, k + e, kend);
          __builtin_memcpy(&ra[i], tmp, 16);
        }
      }
    } else {
#pragma unroll
      for (int i = 0; i < A_ITEMS; ++i) {
        const int u = tid + 256 * i;
        const int rv = u % (BM / V), kq = u / (BM / V);
        const int row = m0 + rv * V, k = kbase + kq * 4;
        if (u < 2 * BM) {
          if (VECA) {
            unit_load<T, MODE, true>(p, row, k, kend, &ra[4 * i]);
          } else {
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              U tmp[V];
#pragma unroll
              for (int e = 0; e < V; ++e) tmp[e] = elemA<T, MODE>(p, row + e, k + j, kend);
              __builtin_memcpy(&ra[4 * i + j], tmp, 16);
            }
          }
        }
      }
    }
    // ---- B
    if (B_KCONTIG) {
      const int k = kbase + (tid & 7) * V;
#pragma unroll
      for (int i = 0; i < B_ITEMS; ++i) {
        const int n = n0 + (tid >> 3) + 32 * i;
        if (VECB) {
          rb[i] = chunkB_fwd<T>(p, n, k);
        } else {
          U tmp[V];
#pragma unroll
          for (int e = 0; e < V; ++e) tmp[e] = elemB<T, MODE>(p, n, k + e, kend);
          __builtin_memcpy(&rb[i], tmp, 16);
        }
      }
    } else {
#pragma unroll
      for (int i = 0; i < B_ITEMS; ++i) {
        const int u = tid + 256 * i;
        const int rv = u % (BN / V), kq = u / (BN / V);
        const int row = n0 + rv * V, k = kbase + kq * 4;
        if (u < 2 * BN) {
          if (VECB) {
            unit_load<T, MODE, false>(p, row, k, kend, &rb[4 * i]);
          } else {
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              U tmp[V];
#pragma unroll
              for (int e = 0; e < V; ++e) tmp[e] = elemB<T, MODE>(p, row + e, k + j, kend);
              __builtin_memcpy(&rb[4 * i + j], tmp, 16);
            }
          }
        }
      }
    }
  };

  auto store_tile = [&](int buf) {
    char* As = smem + buf * (BM + BN) * PITCH;
    char* Bs = As + BM * PITCH;
    if (A_KCONTIG) {
#pragma unroll
      for (int i = 0; i < A_ITEMS; ++i)
        *(uint4*)(As + ((tid >> 3) + 32 * i) * PITCH + (tid & 7) * 16) = ra[i];
    } else {
#pragma unroll
      for (int i = 0; i < A_ITEMS; ++i) {
        const int u = tid + 256 * i;
        if (u < 2 * BM) {
          const int rv = u % (BM / V), kq = u / (BM / V);
          unit_store<T>(As, rv * V, kq * 4 * EB, &ra[4 * i]);
        }
      }
    }
    if (B_KCONTIG) {
#pragma unroll
      for (int i = 0; i < B_ITEMS; ++i)
        *(uint4*)(Bs + ((tid >> 3) + 32 * i) * PITCH + (tid & 7) * 16) = rb[i];
    } else {
#pragma unroll
      for (int i = 0; i < B_ITEMS; ++i) {
        const int u = tid + 256 * i;
        if (u < 2 * BN) {
          const int rv = u % (BN / V), kq = u / (BN / V);
          unit_store<T>(Bs, rv * V, kq * 4 * EB, &rb[4 * i]);
        }
      }
    }
  };

  f32x4 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = (f32x4){0.f, 0.f, 0.f, 0.f};

  if (kt0 < kt1) {
    load_tile(kt0);
    store_tile(0);
  }
  __syncthreads();

  for (int kt = kt0; kt < kt1; ++kt) {
    const int buf = (kt - kt0) & 1;
    const bool more = kt + 1 < kt1;
    if (more) load_tile(kt + 1);
    const char* As = smem + buf * (BM + BN) * PITCH;
    const char* Bs = As + BM * PITCH;
#pragma unroll
    for (int kg = 0; kg < 2; ++kg) {
      uint4 fa[FM], fb[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i)
        fa[i] = *(const uint4*)(As + (wm * (BM / 2) + 16 * i + (lane & 15)) * PITCH + kg * 64 +
                                (lane >> 4) * 16);
#pragma unroll
      for (int j = 0; j < FN; ++j)
        fb[j] = *(const uint4*)(Bs + (wn * (BN / 2) + 16 * j + (lane & 15)) * PITCH + kg * 64 +
                                (lane >> 4) * 16);
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
    if (more) store_tile(buf ^ 1);
    __syncthreads();
  }

  // ---- epilogue: lane holds C[m][n .. n+3]
#pragma unroll
  for (int i = 0; i < FM; ++i) {
    const int m = m0 + wm * (BM / 2) + 16 * i + (lane & 15);
    if (m >= p.M) continue;
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int n = n0 + wn * (BN / 2) + 16 * j + (lane >> 4) * 4;
      if (n >= p.N) continue;
      float v[4] = {acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]};
      if (MODE == MODE_WGRAD) {
        float* out = (float*)p.out + (int64_t)blockIdx.y * p.split_stride + (int64_t)m * p.N + n;
        if (n + 3 < p.N && (p.N & 3) == 0) {
          *(float4*)out = make_float4(v[0], v[1], v[2], v[3]);
        } else {
          for (int q = 0; q < 4 && n + q < p.N; ++q) out[q] = v[q];
        }
        continue;
      }
      const int64_t off = (int64_t)m * p.N + n;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        if (p.bias && n + q < p.N) v[q] += p.bias[n + q];
        if (p.addend && n + q < p.N) v[q] += ld<T>((const T*)p.addend, off + q);
        if (p.relu) v[q] = v[q] > 0.f ? v[q] : 0.f;
        if (p.mask && n + q < p.N && !(ld<T>((const T*)p.mask, off + q) > 0.f)) v[q] = 0.f;
      }
      const bool full = (n + 3 < p.N) && (p.N & 3) == 0;
      if (p.out_f32) {
        float* out = (float*)p.out + off;
        if (full) *(float4*)out = make_float4(v[0], v[1], v[2], v[3]);
        else for (int q = 0; q < 4 && n + q < p.N; ++q) out[q] = v[q];
      } else if (EB == 2) {
        bf16_t* out = (bf16_t*)p.out + off;
        if (full) {
          uint2 pk = make_uint2((uint32_t)f2bf(v[0]) | ((uint32_t)f2bf(v[1]) << 16),
                                (uint32_t)f2bf(v[2]) | ((uint32_t)f2bf(v[3]) << 16));
          *(uint2*)out = pk;
        } else {
          for (int q = 0; q < 4 && n + q < p.N; ++q) out[q] = f2bf(v[q]);
        }
      } else {
        float* out = (float*)p.out + off;
        if (full) *(float4*)out = make_float4(v[0], v[1], v[2], v[3]);
        else for (int q = 0; q < 4 && n + q < p.N; ++q) out[q] = v[q];
      }
    }
  }
}

// Per-segment split-K reduction (see launch_splitk_reduce_seg).  blockIdx.y =
// segment; vectorised by 4 when the output is not unpadded.
struct SegOut {
  float* p[MAX_SEG];
  int split0[MAX_SEG + 1];
};

__global__ __launch_bounds__(256) void splitk_reduce_seg_kernel(const float* __restrict__ part,
                                                                int64_t stride, int64_t count,
                                                                SegOut o, int c, int cp,
                                                                int vec) {
  const int sg = blockIdx.y;
  float* out = o.p[0];
  int y0 = o.split0[0], y1 = o.split0[1];
#pragma unroll
  for (int i = 1; i < MAX_SEG; ++i)
    if (i == sg) {
      out = o.p[i];
      y0 = o.split0[i];
      y1 = o.split0[i + 1];
    }
  if (vec) {   // c == cp, 16-byte aligned, count and stride multiples of 4
    const int64_t groups = count >> 2, st4 = stride >> 2;
    for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q < groups;
         q += (int64_t)gridDim.x * blockDim.x) {
      float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
      const float4* pp = (const float4*)part + q;
      int k = y0;
      for (; k + 4 <= y1; k += 4) {
        const float4 a = pp[(k + 0) * st4], b = pp[(k + 1) * st4], cc = pp[(k + 2) * st4],
                     d = pp[(k + 3) * st4];
        s.x += a.x; s.y += a.y; s.z += a.z; s.w += a.w;
        s.x += b.x; s.y += b.y; s.z += b.z; s.w += b.w;
        s.x += cc.x; s.y += cc.y; s.z += cc.z; s.w += cc.w;
        s.x += d.x; s.y += d.y; s.z += d.z; s.w += d.w;
      }
      for (; k < y1; ++k) {
        const float4 a = pp[k * st4];
        s.x += a.x; s.y += a.y; s.z += a.z; s.w += a.w;
      }
      ((float4*)out)[q] = s;
    }
  } else {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count;
         i += (int64_t)gridDim.x * blockDim.x) {
      const int64_t q = i / c, ch = i - q * c;
      const int64_t src = q * cp + ch;
      float s = 0.f;
      for (int k = y0; k < y1; ++k) s += part[k * stride + src];
      out[i] = s;
    }
  }
}

hipError_t launch_splitk_reduce_seg(const float* part, int64_t stride, int64_t count,
                                    const int* split0, float* const* out, int nseg, int c, int cp,
                                    hipStream_t s) {
  if (nseg < 1 || nseg > MAX_SEG || c < 1 || cp < c) return hipErrorInvalidValue;
  SegOut o{};
  for (int i = 0; i < nseg; ++i) o.p[i] = out[i];
  for (int i = 0; i <= nseg; ++i) o.split0[i] = split0[i];
  for (int i = nseg + 1; i <= MAX_SEG; ++i) o.split0[i] = split0[nseg];
  bool vec = cp == c && count % 4 == 0 && stride % 4 == 0 && ((uintptr_t)part & 15) == 0;
  for (int i = 0; i < nseg; ++i) vec = vec && ((uintptr_t)out[i] & 15) == 0;
  const int64_t work = vec ? count / 4 : count;
  int64_t blocks = (work + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(splitk_reduce_seg_kernel, dim3((unsigned)blocks, nseg), dim3(256), 0, s, part,
                     stride, count, o, c, cp, vec ? 1 : 0);
  return hipGetLastError();
}

// Weighted over the segments into one output (see launch_splitk_reduce_wsum):
// each segment's sum is formed exactly as splitk_reduce_seg_kernel forms it,
// then acc = w0 g0, acc = fma(w_s, g_s, acc) in segment order.
struct SegW {
  int split0[MAX_SEG + 1];
  float w[MAX_SEG];
};

__global__ __launch_bounds__(256) void splitk_reduce_wsum_kernel(const float* __restrict__ part,
                                                                 int64_t stride, int64_t count,
                                                                 SegW o, int nseg,
                                                                 float* __restrict__ out, int c,
                                                                 int cp, int vec) {
  if (vec) {
    const int64_t groups = count >> 2, st4 = stride >> 2;
    for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q < groups;
         q += (int64_t)gridDim.x * blockDim.x) {
      const float4* pp = (const float4*)part + q;
      float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
      for (int sg = 0; sg < MAX_SEG; ++sg) {
        if (sg >= nseg) break;
        float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
        int k = o.split0[sg];
        const int y1 = o.split0[sg + 1];
        for (; k + 4 <= y1; k += 4) {
          const float4 a = pp[(k + 0) * st4], b = pp[(k + 1) * st4], cc = pp[(k + 2) * st4],
                       d = pp[(k + 3) * st4];
          s.x += a.x; s.y += a.y; s.z += a.z; s.w += a.w;
          s.x += b.x; s.y += b.y; s.z += b.z; s.w += b.w;
          s.x += cc.x; s.y += cc.y; s.z += cc.z; s.w += cc.w;
          s.x += d.x; s.y += d.y; s.z += d.z; s.w += d.w;
        }
        for (; k < y1; ++k) {
          const float4 a = pp[k * st4];
          s.x += a.x; s.y += a.y; s.z += a.z; s.w += a.w;
        }
        const float w = o.w[sg];
        if (sg == 0) {
          acc.x = w * s.x; acc.y = w * s.y; acc.z = w * s.z; acc.w = w * s.w;
        } else {
          acc.x = __builtin_fmaf(w, s.x, acc.x);
          acc.y = __builtin_fmaf(w, s.y, acc.y);
          acc.z = __builtin_fmaf(w, s.z, acc.z);
          acc.w = __builtin_fmaf(w, s.w, acc.w);
        }
      }
      ((float4*)out)[q] = acc;
    }
  } else {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count;
         i += (int64_t)gridDim.x * blockDim.x) {
      const int64_t q = i / c, ch = i - q * c;
      const int64_t src = q * cp + ch;
      float acc = 0.f;
#pragma unroll
      for (int sg = 0; sg < MAX_SEG; ++sg) {
        if (sg >= nseg) break;
        float s = 0.f;
        for (int k = o.split0[sg]; k < o.split0[sg + 1]; ++k) s += part[(int64_t)k * stride + src];
        const float w = o.w[sg];
        if (sg == 0) acc = w * s;
        else acc = __builtin_fmaf(w, s, acc);
      }
      out[i] = acc;
    }
  }
}

hipError_t launch_splitk_reduce_wsum(const float* part, int64_t stride, int64_t count,
                                     const int* split0, const float* w, float* out, int nseg,
                                     int c, int cp, hipStream_t s) {
  if (nseg < 1 || nseg > MAX_SEG || c < 1 || cp < c) return hipErrorInvalidValue;
  SegW o{};
  for (int i = 0; i <= nseg; ++i) o.split0[i] = split0[i];
  for (int i = nseg + 1; i <= MAX_SEG; ++i) o.split0[i] = split0[nseg];
  for (int i = 0; i < nseg; ++i) o.w[i] = w[i];
  const bool vec = cp == c && count % 4 == 0 && stride % 4 == 0 &&
                   ((uintptr_t)part & 15) == 0 && ((uintptr_t)out & 15) == 0;
  const int64_t work = vec ? count / 4 : count;
  int64_t blocks = (work + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(splitk_reduce_wsum_kernel, dim3((unsigned)blocks), dim3(256), 0, s, part,
                     stride, count, o, nseg, out, c, cp, vec ? 1 : 0);
  return hipGetLastError();
}

// ----------------------------------------------------------------------------
// host-side launch
// ----------------------------------------------------------------------------
template <typename T, int MODE, int BM, int BN>
static hipError_t launch_tiles(const GemmParams& p0, bool veca, bool vecb, int splits,
                               hipStream_t s) {
  GemmParams p = p0;
  const int tiles_m = ceil_div(p.M, BM);
  p.tiles_n = ceil_div(p.N, BN);
  constexpr int BKE = 128 / (int)sizeof(T);
  p.ktiles = ceil_div(p.K, BKE);
  if (p.nseg > 0) splits = p.seg_split[p.nseg];   // kt_per_split set by the caller
  else p.kt_per_split = ceil_div(p.ktiles, splits);
  dim3 grid(tiles_m * p.tiles_n, splits);
  if (veca && vecb)
    hipLaunchKernelGGL((igemm_kernel<T, MODE, BM, BN, true, true>), grid, dim3(256), 0, s, p);
  else if (veca)
    hipLaunchKernelGGL((igemm_kernel<T, MODE, BM, BN, true, false>), grid, dim3(256), 0, s, p);
  else if (vecb)
    hipLaunchKernelGGL((igemm_kernel<T, MODE, BM, BN, false, true>), grid, dim3(256), 0, s, p);
  else
    hipLaunchKernelGGL((igemm_kernel<T, MODE, BM, BN, false, false>), grid, dim3(256), 0, s, p);
  return hipGetLastError();
}

template <typename T, int MODE>
static hipError_t launch_mode(const GemmParams& p, bool veca, bool vecb, int bm, int bn,
                              int splits, hipStream_t s) {
  if (bm == 128 && bn == 128) return launch_tiles<T, MODE, 128, 128>(p, veca, vecb, splits, s);
  if (bm == 128 && bn == 64) return launch_tiles<T, MODE, 128, 64>(p, veca, vecb, splits, s);
  if (bm == 64 && bn == 128) return launch_tiles<T, MODE, 64, 128>(p, veca, vecb, splits, s);
  return launch_tiles<T, MODE, 64, 64>(p, veca, vecb, splits, s);
}

hipError_t launch_igemm(int mode, bool bf16, const GemmParams& p, bool veca, bool vecb, int bm,
                        int bn, int splits, hipStream_t s) {
  if (bf16) {
    if (mode == MODE_FWD) return launch_mode<bf16_t, MODE_FWD>(p, veca, vecb, bm, bn, splits, s);
    if (mode == MODE_DGRAD) return launch_mode<bf16_t, MODE_DGRAD>(p, veca, vecb, bm, bn, splits, s);
    return launch_mode<bf16_t, MODE_WGRAD>(p, veca, vecb, bm, bn, splits, s);
  }
  if (mode == MODE_FWD) return launch_mode<float, MODE_FWD>(p, veca, vecb, bm, bn, splits, s);
  if (mode == MODE_DGRAD) return launch_mode<float, MODE_DGRAD>(p, veca, vecb, bm, bn, splits, s);
  return launch_mode<float, MODE_WGRAD>(p, veca, vecb, bm, bn, splits, s);
}


}  // namespace hs
