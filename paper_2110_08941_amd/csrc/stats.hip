// Per-channel sums over the rows of an NHWC tensor, finished in one launch:
//   kind 0 (batch-norm forward):  mean and 1/sqrt(var + eps) of x
//   kind 1 (batch-norm backward): sum d and sum d * xhat, d = dy * [act > 0],
//                                 xhat = (x - mean) * rstd
//   kind 2 (bias gradient):       sum d
// Each thread reads V consecutive channels (16-byte vectors) over a strided
// set of rows and accumulates in fp32; the block sums its row lanes in LDS and
// writes one partial.  The last block of every group of 64 blocks to finish
// sums that group's partials (double), and the last group to finish sums the
// group partials and writes the result.  Every sum is taken in a fixed
// order, so the result does not depend on which block finishes last.  The
// arrival counters live in the caller's workspace, start at zero and are
// reset by the blocks that consume them.
// Batch-norm forward sums are shifted by the first row's value per channel
// (var = E[(x-k)^2] - E[x-k]^2) so that a large mean does not cancel.
#include "kernels.h"

namespace hs {

constexpr int STAT_GROUP = 64;

struct StatArgs {
  const void* x;
  const void* dy;
  const void* act;
  const float* mean;
  const float* rstd;
  int64_t rows;
  int C;
  float* part1;        // [blocks][2][C]
  double* part2;       // [groups][2][C]
  unsigned* counters;  // [groups + 1]
  float* out0;
  float* out1;
  float eps;
};

template <typename T, int V>
__device__ inline void load_vec(const T* p, int64_t i, float* v);
template <>
__device__ inline void load_vec<bf16_t, 8>(const bf16_t* p, int64_t i, float* v) {
  uint4 u = *(const uint4*)(p + i);
  const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    v[2 * k] = bf2f((bf16_t)(w[k] & 0xffffu));
    v[2 * k + 1] = bf2f((bf16_t)(w[k] >> 16));
  }
}
template <>
__device__ inline void load_vec<float, 8>(const float* p, int64_t i, float* v) {
  float4 a = *(const float4*)(p + i), b = *(const float4*)(p + i + 4);
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
  v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}
template <>
__device__ inline void load_vec<bf16_t, 1>(const bf16_t* p, int64_t i, float* v) { v[0] = bf2f(p[i]); }
template <>
__device__ inline void load_vec<float, 1>(const float* p, int64_t i, float* v) { v[0] = p[i]; }

template <typename T, int V, int KIND>
__global__ __launch_bounds__(256) void chan_stats_kernel(StatArgs a) {
  __shared__ float red[2][256 * 8];
  __shared__ int s_last;
  const int C = a.C;
  const int TPR = C / V;
  const int RPB = 256 / TPR;
  const int t = threadIdx.x;
  const int cg = t % TPR, rl = t / TPR;
  const int c0 = cg * V;
  const int64_t per = (a.rows + gridDim.x - 1) / gridDim.x;
  const int64_t r0 = (int64_t)blockIdx.x * per;
  const int64_t r1 = r0 + per < a.rows ? r0 + per : a.rows;
  float s0[V], s1[V], k[V], mu[V], rs[V];
#pragma unroll
  for (int j = 0; j < V; ++j) s0[j] = s1[j] = 0.f;
  if (rl < RPB) {
    if (KIND == 0) load_vec<T, V>((const T*)a.x, c0, k);          // shift: row 0
    if (KIND == 1) {
#pragma unroll
      for (int j = 0; j < V; ++j) {
        mu[j] = a.mean[c0 + j];
        rs[j] = a.rstd[c0 + j];
      }
    }
    int64_t r = r0 + rl;
    // four rows per iteration: four independent 16-byte loads in flight
    for (; r + 3 * RPB < r1; r += 4 * RPB) {
      float v[4][V];
      if (KIND == 0) {
#pragma unroll
        for (int u = 0; u < 4; ++u) load_vec<T, V>((const T*)a.x, (r + u * RPB) * C + c0, v[u]);
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
          for (int j = 0; j < V; ++j) {
            const float d = v[u][j] - k[j];
            s0[j] += d;
            s1[j] += d * d;
          }
      } else {
        float m[4][V], z[4][V];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int64_t i = (r + u * RPB) * C + c0;
          load_vec<T, V>((const T*)a.dy, i, v[u]);
          if (a.act) load_vec<T, V>((const T*)a.act, i, m[u]);
          if (KIND == 1) load_vec<T, V>((const T*)a.x, i, z[u]);
        }
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
          for (int j = 0; j < V; ++j) {
            float d = v[u][j];
            if (a.act && !(m[u][j] > 0.f)) d = 0.f;
            s0[j] += d;
            if (KIND == 1) s1[j] += d * ((z[u][j] - mu[j]) * rs[j]);
          }
      }
    }
    for (; r < r1; r += RPB) {
      const int64_t i = r * C + c0;
      float v[V];
      if (KIND == 0) {
        load_vec<T, V>((const T*)a.x, i, v);
#pragma unroll
        for (int j = 0; j < V; ++j) {
          const float d = v[j] - k[j];
          s0[j] += d;
          s1[j] += d * d;
        }
      } else {
        load_vec<T, V>((const T*)a.dy, i, v);
        if (a.act) {
          float m[V];
          load_vec<T, V>((const T*)a.act, i, m);
#pragma unroll
          for (int j = 0; j < V; ++j)
            if (!(m[j] > 0.f)) v[j] = 0.f;
        }
        if (KIND == 1) {
          float z[V];
          load_vec<T, V>((const T*)a.x, i, z);
#pragma unroll
          for (int j = 0; j < V; ++j) {
            s0[j] += v[j];
            s1[j] += v[j] * ((z[j] - mu[j]) * rs[j]);
          }
        } else {
#pragma unroll
          for (int j = 0; j < V; ++j) s0[j] += v[j];
        }
      }
    }
  }
  // ---- block: sum the row lanes of every channel, in lane order
  if (rl < RPB) {
#pragma unroll
    for (int j = 0; j < V; ++j) {
      red[0][rl * C + c0 + j] = s0[j];
      red[1][rl * C + c0 + j] = s1[j];
    }
  }
  __syncthreads();
  for (int c = t; c < C; c += 256) {
    float a0 = 0.f, a1 = 0.f;
    for (int q = 0; q < RPB; ++q) {
      a0 += red[0][q * C + c];
      a1 += red[1][q * C + c];
    }
    a.part1[((int64_t)blockIdx.x * 2 + 0) * C + c] = a0;
    a.part1[((int64_t)blockIdx.x * 2 + 1) * C + c] = a1;
  }
  // ---- group: the last block of the group sums the group's partials
  const int nb = gridDim.x;
  const int groups = (nb + STAT_GROUP - 1) / STAT_GROUP;
  const int g = blockIdx.x / STAT_GROUP;
  const int gsize = (g == groups - 1) ? nb - g * STAT_GROUP : STAT_GROUP;
  __threadfence();
  __syncthreads();
  if (t == 0) s_last = (atomicAdd(&a.counters[g], 1u) == (unsigned)(gsize - 1));
  __syncthreads();
  if (!s_last) return;
  __threadfence();
  {
    // L lanes per channel, each summing every L-th block of the group; then
    // the lanes are added in lane order
    __shared__ double dred[2][256];
    const int L = C >= 256 ? 1 : 256 / C;
    for (int cb = 0; cb < C; cb += 256) {
      const int c = cb + (L == 1 ? t : t % C), lane = L == 1 ? 0 : t / C;
      double a0 = 0.0, a1 = 0.0;
      if (c < C && lane < L) {
        const int b0 = g * STAT_GROUP;
#pragma unroll 4
        for (int b = b0 + lane; b < b0 + gsize; b += L) {
          a0 += (double)__builtin_nontemporal_load(&a.part1[((int64_t)b * 2 + 0) * C + c]);
          a1 += (double)__builtin_nontemporal_load(&a.part1[((int64_t)b * 2 + 1) * C + c]);
        }
      }
      dred[0][t] = a0;
      dred[1][t] = a1;
      __syncthreads();
      if (t < 256 / L && cb + t < C) {
        double b0s = 0.0, b1s = 0.0;
        for (int q = 0; q < L; ++q) {
          b0s += dred[0][t + q * C];
          b1s += dred[1][t + q * C];
        }
        a.part2[((int64_t)g * 2 + 0) * C + cb + t] = b0s;
        a.part2[((int64_t)g * 2 + 1) * C + cb + t] = b1s;
      }
      __syncthreads();
    }
  }
  if (t == 0) a.counters[g] = 0u;
  __threadfence();
  __syncthreads();
  if (t == 0) s_last = (atomicAdd(&a.counters[groups], 1u) == (unsigned)(groups - 1));
  __syncthreads();
  if (!s_last) return;
  __threadfence();
  for (int c = t; c < C; c += 256) {
    double a0 = 0.0, a1 = 0.0;
    for (int q = 0; q < groups; ++q) {
      a0 += __builtin_nontemporal_load(&a.part2[((int64_t)q * 2 + 0) * C + c]);
      a1 += __builtin_nontemporal_load(&a.part2[((int64_t)q * 2 + 1) * C + c]);
    }
    if (KIND == 0) {
      const double cnt = (double)a.rows;
      const double m1 = a0 / cnt;
      double var = a1 / cnt - m1 * m1;
      if (var < 0.0) var = 0.0;
      const float shift = ld<T>((const T*)a.x, c);
      a.out0[c] = (float)((double)shift + m1);
      a.out1[c] = (float)(1.0 / sqrt(var + (double)a.eps));
    } else {
      if (a.out0) a.out0[c] = (float)a0;
      if (KIND == 1 && a.out1) a.out1[c] = (float)a1;
    }
  }
  if (t == 0) a.counters[groups] = 0u;
}

int stat_blocks(int64_t rows, int C) {
  const int V = (C % 8 == 0 && C / 8 <= 256) ? 8 : 1;
  const int TPR = C / V;
  const int RPB = 256 / TPR;
  int64_t b = (rows + (int64_t)RPB * 16 - 1) / ((int64_t)RPB * 16);   // >= 16 rows per lane
  if (b > STAT_MAX_BLOCKS) b = STAT_MAX_BLOCKS;
  if (b < 1) b = 1;
  return (int)b;
}

hipError_t launch_chan_stats(int kind, bool bf16, const void* x, const void* dy, const void* act,
                             const float* mean, const float* rstd, int64_t rows, int C,
                             float* part1, double* part2, unsigned* counters, float* out0,
                             float* out1, float eps, hipStream_t s) {
  if (C < 1 || C > 256 * 8 || (C % 8 != 0 && C > 256)) return hipErrorInvalidValue;
  StatArgs a{x, dy, act, mean, rstd, rows, C, part1, part2, counters, out0, out1, eps};
  const bool vec = (C % 8 == 0 && C / 8 <= 256);
  dim3 grid(stat_blocks(rows, C)), block(256);
#define HS_STAT(T, V, K) hipLaunchKernelGGL((chan_stats_kernel<T, V, K>), grid, block, 0, s, a)
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
template <typename T>
__device__ inline void store_vec8(T* p, int64_t i, const float* v);
template <>
__device__ inline void store_vec8<bf16_t>(bf16_t* p, int64_t i, const float* v) {
  uint4 u;
  u.x = (uint32_t)f2bf(v[0]) | ((uint32_t)f2bf(v[1]) << 16);
  u.y = (uint32_t)f2bf(v[2]) | ((uint32_t)f2bf(v[3]) << 16);
  u.z = (uint32_t)f2bf(v[4]) | ((uint32_t)f2bf(v[5]) << 16);
  u.w = (uint32_t)f2bf(v[6]) | ((uint32_t)f2bf(v[7]) << 16);
  *(uint4*)(p + i) = u;
}
template <>
__device__ inline void store_vec8<float>(float* p, int64_t i, const float* v) {
  *(float4*)(p + i) = make_float4(v[0], v[1], v[2], v[3]);
  *(float4*)(p + i + 4) = make_float4(v[4], v[5], v[6], v[7]);
}

static inline int vgrid(int64_t groups) {
  int64_t b = (groups + 255) / 256;
  if (b > 16384) b = 16384;
  if (b < 1) b = 1;
  return (int)b;
}

// Row-major elementwise work over [rows][C] with C % 8 == 0: a thread owns
// one group of 8 channels (its per-channel coefficients stay in registers) and
// walks rows rl, rl + RPB, ... of its block's row range, 4 rows per step.
struct RowSplit {
  int TPR, RPB, cg, rl, c0;
  int64_t r0, r1;
};

__device__ inline RowSplit row_split(int64_t rows, int C) {
  RowSplit w;
  w.TPR = C / 8;
  w.RPB = 256 / w.TPR;
  w.cg = threadIdx.x % w.TPR;
  w.rl = threadIdx.x / w.TPR;
  w.c0 = w.cg * 8;
  const int64_t per = (rows + gridDim.x - 1) / gridDim.x;
  w.r0 = (int64_t)blockIdx.x * per;
  w.r1 = w.r0 + per < rows ? w.r0 + per : rows;
  return w;
}

static inline int row_grid(int64_t rows, int C) {
  const int RPB = 256 / (C / 8);
  int64_t b = (rows + (int64_t)RPB * 8 - 1) / ((int64_t)RPB * 8);   // ~8 rows per thread
  if (b > 16384) b = 16384;
  if (b < 1) b = 1;
  return (int)b;
}

// y = relu?(gamma * (z - mean) * rstd + beta + res)
template <typename T>
__global__ __launch_bounds__(256) void bn_apply8_kernel(const T* __restrict__ z,
                                                        const float* __restrict__ mean,
                                                        const float* __restrict__ rstd,
                                                        const float* __restrict__ gamma,
                                                        const float* __restrict__ beta,
                                                        const T* __restrict__ res, int relu,
                                                        int64_t rows, int C, T* __restrict__ y) {
  const RowSplit w = row_split(rows, C);
  if (w.rl >= w.RPB) return;
  float sa[8], sb[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int c = w.c0 + j;
    sa[j] = gamma[c] * rstd[c];
    sb[j] = beta[c] - mean[c] * sa[j];
  }
  for (int64_t r = w.r0 + w.rl; r < w.r1; r += 4 * w.RPB) {
    float v[4][8], q[4][8];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int64_t rr = r + u * w.RPB;
      if (rr < w.r1) {
        load_vec<T, 8>(z, rr * C + w.c0, v[u]);
        if (res) load_vec<T, 8>(res, rr * C + w.c0, q[u]);
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int64_t rr = r + u * w.RPB;
      if (rr >= w.r1) continue;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        float o = sa[j] * v[u][j] + sb[j];
        if (res) o += q[u][j];
        if (relu) o = o > 0.f ? o : 0.f;
        v[u][j] = o;
      }
      store_vec8<T>(y, rr * C + w.c0, v[u]);
    }
  }
}

hipError_t launch_bn_apply8(bool bf16, const void* z, const float* mean, const float* rstd,
                            const float* gamma, const float* beta, const void* res, int relu,
                            int64_t rows, int C, void* y, hipStream_t s) {
  if (C % 8 || C / 8 > 256) return hipErrorInvalidValue;
  const dim3 grid(row_grid(rows, C));
  if (bf16)
    hipLaunchKernelGGL(bn_apply8_kernel<bf16_t>, grid, dim3(256), 0, s, (const bf16_t*)z, mean,
                       rstd, gamma, beta, (const bf16_t*)res, relu, rows, C, (bf16_t*)y);
  else
    hipLaunchKernelGGL(bn_apply8_kernel<float>, grid, dim3(256), 0, s, (const float*)z, mean,
                       rstd, gamma, beta, (const float*)res, relu, rows, C, (float*)y);
  return hipGetLastError();
}

// dz = gamma * rstd * (d - (sum_d + xhat * sum_dx) / rows), d = dy * [act > 0]
template <typename T>
__global__ __launch_bounds__(256) void bn_backward8_kernel(
    const T* __restrict__ dy, const T* __restrict__ act, const T* __restrict__ z,
    const float* __restrict__ mean, const float* __restrict__ rstd, const float* __restrict__ gamma,
    const float* __restrict__ sum_dy, const float* __restrict__ sum_dyx, int64_t rows, int C,
    float inv_rows, T* __restrict__ dz) {
  const RowSplit w = row_split(rows, C);
  if (w.rl >= w.RPB) return;
  float gr[8], mu[8], rs[8], k1[8], k2[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int c = w.c0 + j;
    rs[j] = rstd[c];
    gr[j] = gamma[c] * rs[j];
    mu[j] = mean[c];
    k1[j] = sum_dy[c] * inv_rows;
    k2[j] = sum_dyx[c] * inv_rows;
  }
  for (int64_t r = w.r0 + w.rl; r < w.r1; r += 4 * w.RPB) {
    float d[4][8], zz[4][8], m[4][8];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int64_t rr = r + u * w.RPB;
      if (rr < w.r1) {
        load_vec<T, 8>(dy, rr * C + w.c0, d[u]);
        load_vec<T, 8>(z, rr * C + w.c0, zz[u]);
        if (act) load_vec<T, 8>(act, rr * C + w.c0, m[u]);
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int64_t rr = r + u * w.RPB;
      if (rr >= w.r1) continue;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        float g = d[u][j];
        if (act && !(m[u][j] > 0.f)) g = 0.f;
        const float xh = (zz[u][j] - mu[j]) * rs[j];
        d[u][j] = gr[j] * (g - (k1[j] + xh * k2[j]));
      }
      store_vec8<T>(dz, rr * C + w.c0, d[u]);
    }
  }
}

hipError_t launch_bn_backward8(bool bf16, const void* dy, const void* act, const void* z,
                               const float* mean, const float* rstd, const float* gamma,
                               const float* sum_dy, const float* sum_dyx, int64_t rows, int C,
                               void* dz, hipStream_t s) {
  if (C % 8 || C / 8 > 256) return hipErrorInvalidValue;
  const float inv = 1.0f / (float)rows;
  const dim3 grid(row_grid(rows, C));
  if (bf16)
    hipLaunchKernelGGL(bn_backward8_kernel<bf16_t>, grid, dim3(256), 0, s, (const bf16_t*)dy,
                       (const bf16_t*)act, (const bf16_t*)z, mean, rstd, gamma, sum_dy, sum_dyx,
                       rows, C, inv, (bf16_t*)dz);
  else
    hipLaunchKernelGGL(bn_backward8_kernel<float>, grid, dim3(256), 0, s, (const float*)dy,
                       (const float*)act, (const float*)z, mean, rstd, gamma, sum_dy, sum_dyx, rows,
                       C, inv, (float*)dz);
  return hipGetLastError();
}

// out = dy * [act > 0]
template <typename T>
__global__ __launch_bounds__(256) void relu_mask8_kernel(const T* __restrict__ dy,
                                                         const T* __restrict__ act, int64_t groups,
                                                         T* __restrict__ out) {
  for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q < groups;
       q += (int64_t)gridDim.x * blockDim.x) {
    float d[8], m[8];
    load_vec<T, 8>(dy, q * 8, d);
    load_vec<T, 8>(act, q * 8, m);
#pragma unroll
    for (int j = 0; j < 8; ++j)
      if (!(m[j] > 0.f)) d[j] = 0.f;
    store_vec8<T>(out, q * 8, d);
  }
}

hipError_t launch_relu_mask8(bool bf16, const void* dy, const void* act, int64_t count, void* out,
                             hipStream_t s) {
  if (count % 8) return hipErrorInvalidValue;
  const int64_t groups = count / 8;
  if (bf16)
    hipLaunchKernelGGL(relu_mask8_kernel<bf16_t>, dim3(vgrid(groups)), dim3(256), 0, s,
                       (const bf16_t*)dy, (const bf16_t*)act, groups, (bf16_t*)out);
  else
    hipLaunchKernelGGL(relu_mask8_kernel<float>, dim3(vgrid(groups)), dim3(256), 0, s,
                       (const float*)dy, (const float*)act, groups, (float*)out);
  return hipGetLastError();
}

}  // namespace hs
