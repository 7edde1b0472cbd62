// Per-channel sums over the rows of an NHWC tensor, per worker segment:
//   kind 0 (batch-norm forward):  mean and 1/sqrt(var + eps) of x
//   kind 1 (batch-norm backward): sum d and sum d * xhat, d = dy * [act > 0],
//                                 xhat = (x - mean) * rstd
//   kind 2 (bias gradient):       sum d
// Two launches.  chan_partial_kernel: every block owns a row range of one
// segment; each thread reads V consecutive channels (16-byte vectors) of a
// strided set of rows, accumulating in fp32; the block adds its row lanes in
// LDS and writes one partial per channel.  chan_finish_kernel: per segment and
// group of 8 channels, 32 lanes per channel add the segment's block partials
// in double, then a fixed-order tree adds the lanes.  Every sum is taken in a
// fixed order: the result does not depend on scheduling.
// Batch-norm forward sums are shifted by the segment's first row, per channel
// (var = E[(x-k)^2] - E[x-k]^2), so that a large mean does not cancel.
#include "kernels.h"

namespace hs {

SegRows seg_rows(const Segs& sg, int64_t rows_per_sample, int64_t min_rows, int max_blocks) {
  SegRows r{};
  r.count = sg.count;
  const int64_t total = (int64_t)(sg.n0[sg.count] - sg.n0[0]) * rows_per_sample;
  int64_t per = min_rows > 0 ? min_rows : 1;
  const int64_t cap = (int64_t)max_blocks - sg.count;   // sum of ceil() <= total/per + count
  if (cap >= 1) {
    const int64_t need = (total + cap - 1) / cap;
    if (need > per) per = need;
  }
  r.blk[0] = 0;
  for (int s = 0; s < sg.count; ++s) {
    r.row[s] = (int64_t)sg.n0[s] * rows_per_sample;
    const int64_t rows = (int64_t)(sg.n0[s + 1] - sg.n0[s]) * rows_per_sample;
    int64_t b = (rows + per - 1) / per;
    if (b < 1) b = 1;
    r.blk[s + 1] = r.blk[s] + (int)b;
  }
  r.row[sg.count] = (int64_t)sg.n0[sg.count] * rows_per_sample;
  for (int s = sg.count + 1; s <= MAX_SEG; ++s) {
    r.blk[s] = r.blk[sg.count];
    r.row[s] = r.row[sg.count];
  }
  return r;
}

namespace {

// Segment of block b and the block's share [r0, r1) of the segment's rows.
// Every table index is a compile-time constant (the tables stay in the
// kernel-argument segment).
__device__ inline void block_rows(const SegRows& sr, int b, int& s, int64_t& r0, int64_t& r1,
                                  int64_t& seg0, int64_t& seg1) {
  s = 0;
#pragma unroll
  for (int i = 1; i < MAX_SEG; ++i) s += (i < sr.count && b >= sr.blk[i]) ? 1 : 0;
  int b0 = 0, b1 = 1;
  seg0 = 0;
  seg1 = 0;
#pragma unroll
  for (int i = 0; i < MAX_SEG; ++i)
    if (i == s) {
      b0 = sr.blk[i];
      b1 = sr.blk[i + 1];
      seg0 = sr.row[i];
      seg1 = sr.row[i + 1];
    }
  const int64_t nb = b1 - b0 > 0 ? b1 - b0 : 1;
  const int64_t per = (seg1 - seg0 + nb - 1) / nb;
  r0 = seg0 + (int64_t)(b - b0) * per;
  if (r0 > seg1) r0 = seg1;
  r1 = r0 + per < seg1 ? r0 + per : seg1;
}

template <typename P>
__device__ inline P pick(const P (&arr)[MAX_SEG], int s) {
  P v = arr[0];
#pragma unroll
  for (int i = 1; i < MAX_SEG; ++i)
    if (i == s) v = arr[i];
  return v;
}

}  // namespace

struct StatArgs {
  const void* x;
  const void* dy;
  const void* act;
  const float* mean;    // kind 1: segment s at mean + s * mstride
  const float* rstd;
  int mstride;
  int C;
  float* part;          // [blocks][2][C]
  SegRows sr;
};

struct FinishArgs {
  const void* x;        // kind 0: the shift rows (null: unshifted sums)
  const float* part;
  int C;
  float eps;
  SegRows sr;
  float* out0[MAX_SEG];
  float* out1[MAX_SEG];
  StatWsum wsum;               // sum0 null: no weighted sum
  const float* mean;           // kind 3: segment s's mean and rstd at + s * mstride
  const float* rstd;
  int mstride;
};

// V consecutive channels of one row kept in their storage format until they
// are used (a bf16 row of 8 channels is 4 registers, not 8).  NT: the load
// bypasses the caches' retention (tensors far larger than the L2 and the
// last-level cache are read once).
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

template <bool NT>
__device__ inline uint4 ld16(const void* p) {
  if (NT) {
    const u32x4_t v = __builtin_nontemporal_load((const u32x4_t*)p);
    return make_uint4(v.x, v.y, v.z, v.w);
  }
  return *(const uint4*)p;
}
template <bool NT>
__device__ inline void st16(void* p, const uint4& u) {
  if (NT) {
    const u32x4_t v = {u.x, u.y, u.z, u.w};
    __builtin_nontemporal_store(v, (u32x4_t*)p);
  } else {
    *(uint4*)p = u;
  }
}
__device__ inline float f_of(uint32_t u) {
  float f;
  __builtin_memcpy(&f, &u, 4);
  return f;
}

template <typename T, int V> struct Raw;
template <> struct Raw<bf16_t, 8> {
  uint4 u;
  template <bool NT> __device__ void load(const bf16_t* p, int64_t i) { u = ld16<NT>(p + i); }
  __device__ float operator[](int j) const {
    const uint32_t w = j < 2 ? u.x : j < 4 ? u.y : j < 6 ? u.z : u.w;
    return f_of((j & 1) ? (w & 0xffff0000u) : (w << 16));
  }
};
template <> struct Raw<float, 8> {
  uint4 a, b;
  template <bool NT> __device__ void load(const float* p, int64_t i) {
    a = ld16<NT>(p + i);
    b = ld16<NT>(p + i + 4);
  }
  __device__ float operator[](int j) const {
    const uint4& h = j < 4 ? a : b;
    const int k = j & 3;
    return f_of(k == 0 ? h.x : k == 1 ? h.y : k == 2 ? h.z : h.w);
  }
};
template <> struct Raw<bf16_t, 1> {
  bf16_t v;
  template <bool NT> __device__ void load(const bf16_t* p, int64_t i) { v = p[i]; }
  __device__ float operator[](int) const { return bf2f(v); }
};
template <> struct Raw<float, 1> {
  float v;
  template <bool NT> __device__ void load(const float* p, int64_t i) { v = p[i]; }
  __device__ float operator[](int) const { return v; }
};

template <typename T, int V>
__device__ inline void load_vec(const T* p, int64_t i, float* v) {
  Raw<T, V> r;
  r.template load<false>(p, i);
#pragma unroll
  for (int j = 0; j < V; ++j) v[j] = r[j];
}

// tensors of at least this many bytes are streamed with nontemporal accesses
constexpr int64_t NT_BYTES = 100ll << 20;

template <typename T, int V, int KIND, bool NT>
__global__ __launch_bounds__(256) void chan_partial_kernel(StatArgs a) {
  __shared__ float red[2][256 * 8];
  const int C = a.C;
  const int TPR = C / V;
  const int RPB = 256 / TPR;
  const int t = threadIdx.x;
  const int cg = t % TPR, rl = t / TPR;
  const int c0 = cg * V;
  int s;
  int64_t r0, r1, seg0, seg1;
  block_rows(a.sr, blockIdx.x, s, r0, r1, seg0, seg1);
  const T* __restrict__ x = (const T*)a.x;
  const T* __restrict__ dy = (const T*)a.dy;
  const T* __restrict__ act = (const T*)a.act;
  float s0[V], s1[V], k[V], mu[V], rs[V];
#pragma unroll
  for (int j = 0; j < V; ++j) s0[j] = s1[j] = 0.f;
  if (rl < RPB) {
    if (KIND == 0) load_vec<T, V>(x, seg0 * C + c0, k);   // shift: segment row 0
    if (KIND == 1) {
#pragma unroll
      for (int j = 0; j < V; ++j) {
        mu[j] = a.mean[(int64_t)s * a.mstride + c0 + j];
        rs[j] = a.rstd[(int64_t)s * a.mstride + c0 + j];
      }
    }
    // four rows per step: up to twelve independent loads in flight; the last
    // step masks the rows past the range
    for (int64_t r = r0 + rl; r < r1; r += 4 * RPB) {
      Raw<T, V> v[4], m[4], z[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int64_t rr = r + u * RPB;
        if (rr < r1) {
          const int64_t i = rr * C + c0;
          if (KIND == 0) {
            v[u].template load<NT>(x, i);
          } else {
            v[u].template load<NT>(dy, i);
            if (act) m[u].template load<NT>(act, i);
            if (KIND == 1) z[u].template load<NT>(x, i);
          }
        }
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        if (r + u * RPB >= r1) continue;
#pragma unroll
        for (int j = 0; j < V; ++j) {
          if (KIND == 0) {
            const float d = v[u][j] - k[j];
            s0[j] += d;
            s1[j] += d * d;
          } else {
            float d = v[u][j];
            if (act && !(m[u][j] > 0.f)) d = 0.f;
            s0[j] += d;
            if (KIND == 1) s1[j] += d * ((z[u][j] - mu[j]) * rs[j]);
          }
        }
      }
    }
  }
  // ---- block: add the row lanes of every channel.  L lanes per channel
  // each add every L-th row lane, then the L lane sums are added in order.
  if (rl < RPB) {
#pragma unroll
    for (int j = 0; j < V; ++j) {
      red[0][rl * C + c0 + j] = s0[j];
      red[1][rl * C + c0 + j] = s1[j];
    }
  }
  __syncthreads();
  const int L = C >= 256 ? 1 : 256 / C;
  float a0 = 0.f, a1 = 0.f;
  int c = t, lane = 0;
  if (L > 1) {
    c = t % C;
    lane = t / C;
  }
  if (lane < L && c < C) {
    for (int q = lane; q < RPB; q += L) {
      a0 += red[0][q * C + c];
      a1 += red[1][q * C + c];
    }
  }
  __syncthreads();
  if (L > 1) {
    if (lane < L) {
      red[0][lane * C + c] = a0;
      red[1][lane * C + c] = a1;
    }
    __syncthreads();
    if (t < C) {
      a0 = a1 = 0.f;
      for (int q = 0; q < L; ++q) {
        a0 += red[0][q * C + t];
        a1 += red[1][q * C + t];
      }
      a.part[((int64_t)blockIdx.x * 2 + 0) * C + t] = a0;
      a.part[((int64_t)blockIdx.x * 2 + 1) * C + t] = a1;
    }
  } else {
    for (int cc = t; cc < C; cc += 256) {
      float b0 = 0.f, b1 = 0.f;
      for (int q = 0; q < RPB; ++q) {
        b0 += red[0][q * C + cc];
        b1 += red[1][q * C + cc];
      }
      a.part[((int64_t)blockIdx.x * 2 + 0) * C + cc] = b0;
      a.part[((int64_t)blockIdx.x * 2 + 1) * C + cc] = b1;
    }
  }
}

// blockIdx.y = segment, blockIdx.x = group of 8 channels; thread = channel
// (t & 7) x lane (t >> 3).  With a weighted sum (a.wsum, kinds 1 to 3) one
// block per channel group takes every segment in turn and also adds the
// segments' results with their weights.  Kind 3 finishes partials of
// (sum d, sum d z) into kind 1's outputs: sum d (z - mean) rstd = rstd
// (sum d z - mean sum d).
template <typename T, int KIND>
__global__ __launch_bounds__(256) void chan_finish_kernel(FinishArgs a) {
  __shared__ double red[2][256];
  const int t = threadIdx.x, lane = t >> 3;
  const int c = blockIdx.x * 8 + (t & 7);
  const int C = a.C;
  const bool wsum = KIND != 0 && a.wsum.sum0 != nullptr;
  const int sfirst = wsum ? 0 : (int)blockIdx.y, slast = wsum ? a.sr.count : (int)blockIdx.y + 1;
  float acc0 = 0.f, acc1 = 0.f;
  for (int s = sfirst; s < slast; ++s) {
    int b0 = 0, b1 = 0;
    int64_t seg0 = 0, seg1 = 0;
    float w = 0.f;
#pragma unroll
    for (int i = 0; i < MAX_SEG; ++i)
      if (i == s) {
        b0 = a.sr.blk[i];
        b1 = a.sr.blk[i + 1];
        seg0 = a.sr.row[i];
        seg1 = a.sr.row[i + 1];
        w = a.wsum.w[i];
      }
    double s0 = 0.0, s1 = 0.0;
    if (c < C) {
      int b = b0 + lane;
      for (; b + 96 < b1; b += 128) {
        float v[8];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          v[2 * u] = a.part[((int64_t)(b + 32 * u) * 2 + 0) * C + c];
          v[2 * u + 1] = a.part[((int64_t)(b + 32 * u) * 2 + 1) * C + c];
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          s0 += (double)v[2 * u];
          s1 += (double)v[2 * u + 1];
        }
      }
      for (; b < b1; b += 32) {
        s0 += (double)a.part[((int64_t)b * 2 + 0) * C + c];
        s1 += (double)a.part[((int64_t)b * 2 + 1) * C + c];
      }
    }
    red[0][t] = s0;
    red[1][t] = s1;
    __syncthreads();
    for (int step = 16; step >= 1; step >>= 1) {
      if (lane < step) {
        red[0][t] += red[0][t + 8 * step];
        red[1][t] += red[1][t + 8 * step];
      }
      __syncthreads();
    }
    if (lane == 0 && c < C) {
      float* o0 = pick(a.out0, s);
      float* o1 = pick(a.out1, s);
      const double t0 = red[0][t];
      double t1 = red[1][t];
      if (KIND == 3)
        t1 = (double)a.rstd[(int64_t)s * a.mstride + c] *
             (t1 - (double)a.mean[(int64_t)s * a.mstride + c] * t0);
      if (KIND == 0) {
        const double cnt = (double)(seg1 - seg0);
        const double m1 = t0 / cnt;
        double var = t1 / cnt - m1 * m1;
        if (var < 0.0) var = 0.0;
        const float shift = a.x ? ld<T>((const T*)a.x, seg0 * C + c) : 0.f;
        o0[c] = (float)((double)shift + m1);
        o1[c] = (float)(1.0 / sqrt(var + (double)a.eps));
      } else {
        const float v0 = (float)t0, v1 = (float)t1;
        if (o0) o0[c] = v0;
        if (KIND != 2 && o1) o1[c] = v1;
        if (wsum) {
          if (s == 0) {
            acc0 = w * v0;
            acc1 = w * v1;
          } else {
            acc0 = __builtin_fmaf(w, v0, acc0);
            acc1 = __builtin_fmaf(w, v1, acc1);
          }
        }
      }
    }
    __syncthreads();   // red is reused by the next segment
  }
  if (wsum && lane == 0 && c < C) {
    a.wsum.sum0[c] = acc0;
    if (KIND != 2 && a.wsum.sum1) a.wsum.sum1[c] = acc1;
  }
}

hipError_t launch_stats_finish_fwd(bool bf16, const float* part, int blocks, const Segs& sg,
                                   int64_t rows_per_sample, int C, float* const* mean,
                                   float* const* rstd, float eps, hipStream_t s,
                                   const int* seg_blk) {
  if (C < 1 || sg.count < 1 || sg.count > MAX_SEG || (!seg_blk && blocks < 1))
    return hipErrorInvalidValue;
  FinishArgs f{};
  f.x = nullptr;
  f.part = part;
  f.C = C;
  f.eps = eps;
  f.sr.count = sg.count;
  for (int i = 0; i <= MAX_SEG; ++i) {
    const int k = i < sg.count ? i : sg.count;
    f.sr.blk[i] = seg_blk ? seg_blk[k] : k * blocks;
    f.sr.row[i] = (int64_t)sg.n0[k] * rows_per_sample;
  }
  for (int i = 0; i < sg.count; ++i) {
    f.out0[i] = mean[i];
    f.out1[i] = rstd[i];
  }
  const dim3 fgrid((C + 7) / 8, sg.count);
  if (bf16) hipLaunchKernelGGL((chan_finish_kernel<bf16_t, 0>), fgrid, dim3(256), 0, s, f);
  else hipLaunchKernelGGL((chan_finish_kernel<float, 0>), fgrid, dim3(256), 0, s, f);
  return hipGetLastError();
}

hipError_t launch_stats_finish_bwd(const float* part, const Segs& sg, int C, const float* mean,
                                   const float* rstd, int mstride, float* const* out0,
                                   float* const* out1, hipStream_t s, const int* seg_blk,
                                   const StatWsum* wsum) {
  if (C < 1 || sg.count < 1 || sg.count > MAX_SEG || !seg_blk || !mean || !rstd)
    return hipErrorInvalidValue;
  FinishArgs f{};
  f.part = part;
  f.C = C;
  f.sr.count = sg.count;
  for (int i = 0; i <= MAX_SEG; ++i) f.sr.blk[i] = seg_blk[i < sg.count ? i : sg.count];
  for (int i = 0; i < sg.count; ++i) {
    f.out0[i] = out0 ? out0[i] : nullptr;
    f.out1[i] = out1 ? out1[i] : nullptr;
  }
  if (wsum) f.wsum = *wsum;
  f.mean = mean;
  f.rstd = rstd;
  f.mstride = mstride;
  const dim3 fgrid((C + 7) / 8, wsum ? 1 : sg.count);
  hipLaunchKernelGGL((chan_finish_kernel<bf16_t, 3>), fgrid, dim3(256), 0, s, f);
  return hipGetLastError();
}

hipError_t launch_chan_stats(int kind, bool bf16, const void* x, const void* dy, const void* act,
                             const float* mean, const float* rstd, int mstride, const Segs& sg,
                             int64_t rows_per_sample, int C, float* part, float* const* out0,
                             float* const* out1, float eps, hipStream_t s, const StatWsum* wsum) {
  if (wsum && kind == 0) return hipErrorInvalidValue;
  if (C < 1 || C > 256 * 8 || (C % 8 != 0 && C > 256)) return hipErrorInvalidValue;
  if (sg.count < 1 || sg.count > MAX_SEG) return hipErrorInvalidValue;
  const bool vec = (C % 8 == 0 && C / 8 <= 256);
  const int V = vec ? 8 : 1;
  const int RPB = 256 / (C / V);
  StatArgs a{x, dy, act, mean, rstd, mstride, C, part,
             seg_rows(sg, rows_per_sample, (int64_t)RPB * 16, STAT_MAX_BLOCKS)};
  FinishArgs f{};
  f.x = x;
  f.part = part;
  f.C = C;
  f.eps = eps;
  f.sr = a.sr;
  for (int i = 0; i < sg.count; ++i) {
    f.out0[i] = out0 ? out0[i] : nullptr;
    f.out1[i] = out1 ? out1[i] : nullptr;
  }
  if (wsum) f.wsum = *wsum;
  const dim3 grid(a.sr.blk[sg.count]), block(256);
  const dim3 fgrid((C + 7) / 8, wsum ? 1 : sg.count);
  const int64_t rows = (int64_t)(sg.n0[sg.count] - sg.n0[0]) * rows_per_sample;
  // the sums over two or three tensors gain from streaming loads only when
  // they are far beyond the last-level cache; the single-tensor forward sums
  // do not
  const bool nt = kind != 0 && rows * C * (bf16 ? 2 : 4) >= 2 * NT_BYTES;
#define HS_STAT(T, VV, K)                                                             \
  do {                                                                                \
    if (nt && VV == 8)                                                                \
      hipLaunchKernelGGL((chan_partial_kernel<T, VV, K, true>), grid, block, 0, s, a); \
    else                                                                              \
      hipLaunchKernelGGL((chan_partial_kernel<T, VV, K, false>), grid, block, 0, s, a); \
    hipLaunchKernelGGL((chan_finish_kernel<T, K>), fgrid, block, 0, s, f);            \
  } while (0)
  if (bf16) {
    if (vec) {
      if (kind == 0) HS_STAT(bf16_t, 8, 0);
      else if (kind == 1) HS_STAT(bf16_t, 8, 1);
      else HS_STAT(bf16_t, 8, 2);
    } else {
      if (kind == 0) HS_STAT(bf16_t, 1, 0);
      else if (kind == 1) HS_STAT(bf16_t, 1, 1);
      else HS_STAT(bf16_t, 1, 2);
    }
  } else {
    if (vec) {
      if (kind == 0) HS_STAT(float, 8, 0);
      else if (kind == 1) HS_STAT(float, 8, 1);
      else HS_STAT(float, 8, 2);
    } else {
      if (kind == 0) HS_STAT(float, 1, 0);
      else if (kind == 1) HS_STAT(float, 1, 1);
      else HS_STAT(float, 1, 2);
    }
  }
#undef HS_STAT
  return hipGetLastError();
}

// ----------------------------------------------------------------------------
// vectorised elementwise batch-norm kernels (8 channels per thread step)
// ----------------------------------------------------------------------------
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// two fp32 -> packed bf16, round to nearest even (hardware conversion)
__device__ inline uint32_t pack_bf16x2(float lo, float hi) {
  const f32x2_t v = {lo, hi};
  const bf16x2_t h = __builtin_convertvector(v, bf16x2_t);
  uint32_t u;
  __builtin_memcpy(&u, &h, 4);
  return u;
}

template <typename T, bool NT>
__device__ inline void store_vec8(T* p, int64_t i, const float* v);
template <>
__device__ inline void store_vec8<bf16_t, false>(bf16_t* p, int64_t i, const float* v) {
  st16<false>(p + i, make_uint4(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]),
                                pack_bf16x2(v[4], v[5]), pack_bf16x2(v[6], v[7])));
}
template <>
__device__ inline void store_vec8<bf16_t, true>(bf16_t* p, int64_t i, const float* v) {
  st16<true>(p + i, make_uint4(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]),
                               pack_bf16x2(v[4], v[5]), pack_bf16x2(v[6], v[7])));
}
template <>
__device__ inline void store_vec8<float, false>(float* p, int64_t i, const float* v) {
  *(float4*)(p + i) = make_float4(v[0], v[1], v[2], v[3]);
  *(float4*)(p + i + 4) = make_float4(v[4], v[5], v[6], v[7]);
}
template <>
__device__ inline void store_vec8<float, true>(float* p, int64_t i, const float* v) {
  const f32x4_t lo = {v[0], v[1], v[2], v[3]}, hi = {v[4], v[5], v[6], v[7]};
  __builtin_nontemporal_store(lo, (f32x4_t*)(p + i));
  __builtin_nontemporal_store(hi, (f32x4_t*)(p + i + 4));
}

// Row-major elementwise work over [rows][C] with C % 8 == 0: every block
// owns a row range of one segment; a thread owns one group of 8 channels (its
// per-channel coefficients stay in registers) and walks rows rl, rl + RPB, ...
// of the block's range, 4 rows per step.
struct RowSplit {
  int TPR, RPB, cg, rl, c0, seg;
  int64_t r0, r1, rows;   // block range; rows of the segment
};

__device__ inline RowSplit row_split(const SegRows& sr, int C) {
  RowSplit w;
  w.TPR = C / 8;
  w.RPB = 256 / w.TPR;
  w.cg = threadIdx.x % w.TPR;
  w.rl = threadIdx.x / w.TPR;
  w.c0 = w.cg * 8;
  int64_t seg0, seg1;
  block_rows(sr, blockIdx.x, w.seg, w.r0, w.r1, seg0, seg1);
  w.rows = seg1 - seg0;
  return w;
}

// about 8 rows per thread, at most 16384 blocks
static inline SegRows row_segs(const Segs& sg, int64_t rows_per_sample, int C) {
  const int RPB = 256 / (C / 8);
  return seg_rows(sg, rows_per_sample, (int64_t)RPB * 8, 16384);
}

struct BnArgs {
  const void* z;
  const void* res;      // apply: added before the ReLU, or null
  const void* dy;       // backward
  const void* act;      // backward: dy masked by [act > 0], or null
  const float* mean;    // segment s at mean + s * mstride
  const float* rstd;
  int mstride;
  const float* gamma;
  const float* beta;
  int relu;
  int C;
  void* out;
  uint8_t* bits;        // apply: [y > 0] as bits, [rows][C / 8] bytes, or null
  SegRows sr;
  float* sum0[MAX_SEG]; // backward: per segment sum d and sum d * xhat
  float* sum1[MAX_SEG];
};

// y = relu?(gamma * (z - mean) * rstd + beta + res)
template <typename T, bool NT>
__global__ __launch_bounds__(256) void bn_apply8_kernel(BnArgs a) {
  const int C = a.C;
  const RowSplit w = row_split(a.sr, C);
  if (w.rl >= w.RPB) return;
  const T* __restrict__ z = (const T*)a.z;
  const T* __restrict__ res = (const T*)a.res;
  T* __restrict__ y = (T*)a.out;
  const float* mean = a.mean + (int64_t)w.seg * a.mstride;
  const float* rstd = a.rstd + (int64_t)w.seg * a.mstride;
  float sa[8], sb[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int c = w.c0 + j;
    sa[j] = a.gamma[c] * rstd[c];
    sb[j] = a.beta[c] - mean[c] * sa[j];
  }
  for (int64_t r = w.r0 + w.rl; r < w.r1; r += 4 * w.RPB) {
    Raw<T, 8> v[4], q[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int64_t rr = r + u * w.RPB;
      if (rr < w.r1) {
        v[u].template load<NT>(z, rr * C + w.c0);
        if (res) q[u].template load<NT>(res, rr * C + w.c0);
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int64_t rr = r + u * w.RPB;
      if (rr >= w.r1) continue;
      float o[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        o[j] = sa[j] * v[u][j] + sb[j];
        if (res) o[j] += q[u][j];
        if (a.relu) o[j] = o[j] > 0.f ? o[j] : 0.f;
      }
      if constexpr (sizeof(T) == 2) {
        // the bits test the stored (rounded) values
        const uint32_t pk[4] = {pack_bf16x2(o[0], o[1]), pack_bf16x2(o[2], o[3]),
                                pack_bf16x2(o[4], o[5]), pack_bf16x2(o[6], o[7])};
        st16<NT>(y + rr * C + w.c0, make_uint4(pk[0], pk[1], pk[2], pk[3]));
        if (a.bits) {
          uint32_t b = 0;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            b |= (bf2f((bf16_t)(pk[e] & 0xffffu)) > 0.f ? 1u : 0u) << (2 * e);
            b |= (bf2f((bf16_t)(pk[e] >> 16)) > 0.f ? 1u : 0u) << (2 * e + 1);
          }
          a.bits[(rr * C + w.c0) >> 3] = (uint8_t)b;
        }
      } else {
        store_vec8<T, NT>(y, rr * C + w.c0, o);
        if (a.bits) {
          uint32_t b = 0;
#pragma unroll
          for (int j = 0; j < 8; ++j) b |= (o[j] > 0.f ? 1u : 0u) << j;
          a.bits[(rr * C + w.c0) >> 3] = (uint8_t)b;
        }
      }
    }
  }
}

hipError_t launch_bn_apply8(bool bf16, const void* z, const float* mean, const float* rstd,
                            int mstride, const float* gamma, const float* beta, const void* res,
                            int relu, const Segs& sg, int64_t rows_per_sample, int C, void* y,
                            hipStream_t s, uint8_t* ybits) {
  if (C % 8 || C / 8 > 256 || sg.count < 1 || sg.count > MAX_SEG) return hipErrorInvalidValue;
  BnArgs a{};
  a.bits = ybits;
  a.z = z;
  a.res = res;
  a.mean = mean;
  a.rstd = rstd;
  a.mstride = mstride;
  a.gamma = gamma;
  a.beta = beta;
  a.relu = relu;
  a.C = C;
  a.out = y;
  a.sr = row_segs(sg, rows_per_sample, C);
  const dim3 grid(a.sr.blk[sg.count]);
  const bool nt = a.sr.row[sg.count] - a.sr.row[0] >= NT_BYTES / (C * (bf16 ? 2 : 4));
  if (bf16) {
    if (nt) hipLaunchKernelGGL((bn_apply8_kernel<bf16_t, true>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((bn_apply8_kernel<bf16_t, false>), grid, dim3(256), 0, s, a);
  } else {
    if (nt) hipLaunchKernelGGL((bn_apply8_kernel<float, true>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((bn_apply8_kernel<float, false>), grid, dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

// dz = gamma * rstd * (d - (sum_d + xhat * sum_dx) / rows), d = dy * [act > 0]
template <typename T, bool NT>
__global__ __launch_bounds__(256) void bn_backward8_kernel(BnArgs a) {
  const int C = a.C;
  const RowSplit w = row_split(a.sr, C);
  if (w.rl >= w.RPB) return;
  const T* __restrict__ dy = (const T*)a.dy;
  const T* __restrict__ act = (const T*)a.act;
  const T* __restrict__ z = (const T*)a.z;
  T* __restrict__ dz = (T*)a.out;
  const float* mean = a.mean + (int64_t)w.seg * a.mstride;
  const float* rstd = a.rstd + (int64_t)w.seg * a.mstride;
  const float* sum_dy = pick(a.sum0, w.seg);
  const float* sum_dyx = pick(a.sum1, w.seg);
  const float inv_rows = 1.0f / (float)w.rows;
  float gr[8], mu[8], rs[8], k1[8], k2[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int c = w.c0 + j;
    rs[j] = rstd[c];
    gr[j] = a.gamma[c] * rs[j];
    mu[j] = mean[c];
    k1[j] = sum_dy[c] * inv_rows;
    k2[j] = sum_dyx[c] * inv_rows;
  }
  for (int64_t r = w.r0 + w.rl; r < w.r1; r += 4 * w.RPB) {
    Raw<T, 8> d[4], zz[4], m[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int64_t rr = r + u * w.RPB;
      if (rr < w.r1) {
        d[u].template load<NT>(dy, rr * C + w.c0);
        zz[u].template load<NT>(z, rr * C + w.c0);
        if (act) m[u].template load<NT>(act, rr * C + w.c0);
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int64_t rr = r + u * w.RPB;
      if (rr >= w.r1) continue;
      float o[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        float g = d[u][j];
        if (act && !(m[u][j] > 0.f)) g = 0.f;
        const float xh = (zz[u][j] - mu[j]) * rs[j];
        o[j] = gr[j] * (g - (k1[j] + xh * k2[j]));
      }
      store_vec8<T, NT>(dz, rr * C + w.c0, o);
    }
  }
}

hipError_t launch_bn_backward8(bool bf16, const void* dy, const void* act, const void* z,
                               const float* mean, const float* rstd, int mstride,
                               const float* gamma, float* const* sum_dy, float* const* sum_dyx,
                               const Segs& sg, int64_t rows_per_sample, int C, void* dz,
                               hipStream_t s) {
  if (C % 8 || C / 8 > 256 || sg.count < 1 || sg.count > MAX_SEG) return hipErrorInvalidValue;
  BnArgs a{};
  a.z = z;
  a.dy = dy;
  a.act = act;
  a.mean = mean;
  a.rstd = rstd;
  a.mstride = mstride;
  a.gamma = gamma;
  a.C = C;
  a.out = dz;
  a.sr = row_segs(sg, rows_per_sample, C);
  for (int i = 0; i < sg.count; ++i) {
    a.sum0[i] = sum_dy[i];
    a.sum1[i] = sum_dyx[i];
  }
  const dim3 grid(a.sr.blk[sg.count]);
  const bool nt = a.sr.row[sg.count] - a.sr.row[0] >= NT_BYTES / (C * (bf16 ? 2 : 4));
  if (bf16) {
    if (nt) hipLaunchKernelGGL((bn_backward8_kernel<bf16_t, true>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((bn_backward8_kernel<bf16_t, false>), grid, dim3(256), 0, s, a);
  } else {
    if (nt) hipLaunchKernelGGL((bn_backward8_kernel<float, true>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((bn_backward8_kernel<float, false>), grid, dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace hs
