// Bandwidth-bound layer kernels: batch-norm (training statistics), ReLU
// masks, max-pool, global average pool, softmax cross-entropy, layout casts.
// Activations are NHWC, stored as fp32 or bf16 (T); statistics and
// reductions are carried in fp32 / double and are deterministic (fixed
// reduction order, no atomics).
#include "kernels.h"

namespace hs {

static inline int grid_for(int64_t work, int block = 256, int cap = 8192) {
  int64_t b = (work + block - 1) / block;
  if (b < 1) b = 1;
  if (b > cap) b = cap;
  return (int)b;
}

// ----------------------------------------------------------------------------
// layout / casts
// ----------------------------------------------------------------------------
template <typename T>
__global__ void nchw_to_nhwc_kernel(const float* __restrict__ x, T* __restrict__ y, int n, int c,
                                    int hw) {
  const int64_t total = (int64_t)n * c * hw;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    int64_t b = i / ((int64_t)hw * c);
    int64_t r = i - b * hw * c;
    int p = (int)(r / c), ch = (int)(r - (int64_t)p * c);
    st<T>(y, i, x[(b * c + ch) * hw + p]);
  }
}

hipError_t launch_nchw_to_nhwc(const float* x, void* y, int n, int c, int hw, bool bf16,
                               hipStream_t s) {
  int64_t total = (int64_t)n * c * hw;
  if (bf16)
    hipLaunchKernelGGL(nchw_to_nhwc_kernel<bf16_t>, dim3(grid_for(total)), dim3(256), 0, s, x,
                       (bf16_t*)y, n, c, hw);
  else
    hipLaunchKernelGGL(nchw_to_nhwc_kernel<float>, dim3(grid_for(total)), dim3(256), 0, s, x,
                       (float*)y, n, c, hw);
  return hipGetLastError();
}

template <typename T>
__global__ void cast_kernel(const float* __restrict__ x, T* __restrict__ y, int64_t count) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count;
       i += (int64_t)gridDim.x * blockDim.x)
    st<T>(y, i, x[i]);
}

hipError_t launch_cast_input(const float* x, void* y, int64_t count, bool bf16, hipStream_t s) {
  if (bf16)
    hipLaunchKernelGGL(cast_kernel<bf16_t>, dim3(grid_for(count)), dim3(256), 0, s, x,
                       (bf16_t*)y, count);
  else
    hipLaunchKernelGGL(cast_kernel<float>, dim3(grid_for(count)), dim3(256), 0, s, x, (float*)y,
                       count);
  return hipGetLastError();
}

// ----------------------------------------------------------------------------
// per-channel partial sums
// ----------------------------------------------------------------------------
// Thread layout: CT = min(C, 256) channel lanes x RL = 256 / CT row lanes;
// a thread covers channels c, c + CT, ... (at most 2 when C <= 512) and the
// rows rl, rl + RL, ... of its block's row range.
constexpr int CHAN_MAX = 1024;
constexpr int CHAN_PER_THREAD = CHAN_MAX / 256;

int chan_blocks(int64_t rows, int C) {
  int64_t b = (rows + 255) / 256;
  if (b > 1024) b = 1024;
  if (b < 1) b = 1;
  (void)C;
  return (int)b;
}

template <typename T, int KIND>
__global__ __launch_bounds__(256) void chan_partials_kernel(const T* __restrict__ x,
                                                            const T* __restrict__ dy,
                                                            const T* __restrict__ act,
                                                            const float* __restrict__ mean,
                                                            const float* __restrict__ rstd,
                                                            int64_t rows, int C,
                                                            double* __restrict__ partial) {
  __shared__ double red[2][256 * CHAN_PER_THREAD];
  const int CT = C < 256 ? C : 256;
  const int RL = 256 / CT;
  const int t = threadIdx.x;
  const int cl = t % CT, rl = t / CT;
  const int64_t per = (rows + gridDim.x - 1) / gridDim.x;
  const int64_t r0 = (int64_t)blockIdx.x * per;
  int64_t r1 = r0 + per;
  if (r1 > rows) r1 = rows;
  const int nc = (C + CT - 1) / CT;
  double s0[CHAN_PER_THREAD], s1[CHAN_PER_THREAD];
  for (int j = 0; j < CHAN_PER_THREAD; ++j) s0[j] = s1[j] = 0.0;
  if (rl < RL) {
    for (int64_t r = r0 + rl; r < r1; r += RL) {
      for (int j = 0; j < nc; ++j) {
        const int c = cl + j * CT;
        if (c >= C) break;
        const int64_t i = r * C + c;
        if (KIND == 0) {
          double v = (double)ld<T>(x, i);
          s0[j] += v;
          s1[j] += v * v;
        } else if (KIND == 1) {
          float d = ld<T>(dy, i);
          if (act && !(ld<T>(act, i) > 0.f)) d = 0.f;
          float xh = (ld<T>(x, i) - mean[c]) * rstd[c];
          s0[j] += (double)d;
          s1[j] += (double)d * (double)xh;
        } else {
          float d = ld<T>(dy, i);
          if (act && !(ld<T>(act, i) > 0.f)) d = 0.f;
          s0[j] += (double)d;
        }
      }
    }
  }
  for (int j = 0; j < nc; ++j) {
    red[0][t + 256 * j] = s0[j];
    red[1][t + 256 * j] = s1[j];
  }
  __syncthreads();
  // row lane 0 of every channel lane sums the RL lanes in order
  if (rl == 0) {
    for (int j = 0; j < nc; ++j) {
      const int c = cl + j * CT;
      if (c >= C) break;
      double a = 0.0, b = 0.0;
      for (int q = 0; q < RL; ++q) {
        a += red[0][cl + q * CT + 256 * j];
        b += red[1][cl + q * CT + 256 * j];
      }
      partial[((int64_t)blockIdx.x * 2 + 0) * C + c] = a;
      partial[((int64_t)blockIdx.x * 2 + 1) * C + c] = b;
    }
  }
}

hipError_t launch_chan_partials(int kind, bool bf16, const void* x, const void* dy,
                                const void* act, const float* mean, const float* rstd, int64_t rows,
                                int C, double* partial, hipStream_t s) {
  if (C > CHAN_MAX || C < 1) return hipErrorInvalidValue;
  dim3 grid(chan_blocks(rows, C)), block(256);
#define HS_CHAN(T, K)                                                                        \
  hipLaunchKernelGGL((chan_partials_kernel<T, K>), grid, block, 0, s, (const T*)x, (const T*)dy, \
                     (const T*)act, mean, rstd, rows, C, partial)
  if (bf16) {
    if (kind == 0) HS_CHAN(bf16_t, 0);
    else if (kind == 1) HS_CHAN(bf16_t, 1);
    else HS_CHAN(bf16_t, 2);
  } else {
    if (kind == 0) HS_CHAN(float, 0);
    else if (kind == 1) HS_CHAN(float, 1);
    else HS_CHAN(float, 2);
  }
#undef HS_CHAN
  return hipGetLastError();
}

__global__ void bn_finalize_kernel(const double* __restrict__ partial, int blocks, int C,
                                   int64_t count, float eps, float* __restrict__ mean,
                                   float* __restrict__ rstd) {
  int c = blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= C) return;
  double a = 0.0, b = 0.0;
  for (int k = 0; k < blocks; ++k) {
    a += partial[((int64_t)k * 2 + 0) * C + c];
    b += partial[((int64_t)k * 2 + 1) * C + c];
  }
  double mu = a / (double)count;
  double var = b / (double)count - mu * mu;
  if (var < 0.0) var = 0.0;
  mean[c] = (float)mu;
  rstd[c] = (float)(1.0 / sqrt(var + (double)eps));
}

hipError_t launch_bn_finalize(const double* partial, int blocks, int C, int64_t count, float eps,
                              float* mean, float* rstd, hipStream_t s) {
  hipLaunchKernelGGL(bn_finalize_kernel, dim3((C + 255) / 256), dim3(256), 0, s, partial, blocks,
                     C, count, eps, mean, rstd);
  return hipGetLastError();
}

__global__ void chan_reduce_kernel(const double* __restrict__ partial, int blocks, int C,
                                   float* __restrict__ out0, float* __restrict__ out1) {
  int c = blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= C) return;
  double a = 0.0, b = 0.0;
  for (int k = 0; k < blocks; ++k) {
    a += partial[((int64_t)k * 2 + 0) * C + c];
    b += partial[((int64_t)k * 2 + 1) * C + c];
  }
  if (out0) out0[c] = (float)a;
  if (out1) out1[c] = (float)b;
}

hipError_t launch_chan_reduce(const double* partial, int blocks, int C, float* out0, float* out1,
                              hipStream_t s) {
  hipLaunchKernelGGL(chan_reduce_kernel, dim3((C + 255) / 256), dim3(256), 0, s, partial, blocks,
                     C, out0, out1);
  return hipGetLastError();
}

// ----------------------------------------------------------------------------
// batch-norm apply / backward, elementwise (4 channels per thread step)
// ----------------------------------------------------------------------------
template <typename T>
__global__ void bn_apply_kernel(const T* __restrict__ z, const float* __restrict__ mean,
                                const float* __restrict__ rstd, const float* __restrict__ gamma,
                                const float* __restrict__ beta, const T* __restrict__ res, int relu,
                                int64_t rows, int C, T* __restrict__ y) {
  const int64_t total = rows * C;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int c = (int)(i % C);
    float v = gamma[c] * (ld<T>(z, i) - mean[c]) * rstd[c] + beta[c];
    if (res) v += ld<T>(res, i);
    if (relu) v = v > 0.f ? v : 0.f;
    st<T>(y, i, v);
  }
}

hipError_t launch_bn_apply(bool bf16, const void* z, const float* mean, const float* rstd,
                           const float* gamma, const float* beta, const void* res, int relu,
                           int64_t rows, int C, void* y, hipStream_t s) {
  int64_t total = rows * C;
  if (bf16)
    hipLaunchKernelGGL(bn_apply_kernel<bf16_t>, dim3(grid_for(total)), dim3(256), 0, s,
                       (const bf16_t*)z, mean, rstd, gamma, beta, (const bf16_t*)res, relu, rows,
                       C, (bf16_t*)y);
  else
    hipLaunchKernelGGL(bn_apply_kernel<float>, dim3(grid_for(total)), dim3(256), 0, s,
                       (const float*)z, mean, rstd, gamma, beta, (const float*)res, relu, rows, C,
                       (float*)y);
  return hipGetLastError();
}

template <typename T>
__global__ void bn_backward_kernel(const T* __restrict__ dy, const T* __restrict__ act,
                                   const T* __restrict__ z, const float* __restrict__ mean,
                                   const float* __restrict__ rstd, const float* __restrict__ gamma,
                                   const float* __restrict__ sum_dy,
                                   const float* __restrict__ sum_dyx, int64_t rows, int C,
                                   T* __restrict__ dz) {
  const int64_t total = rows * C;
  const float inv = 1.0f / (float)rows;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int c = (int)(i % C);
    float d = ld<T>(dy, i);
    if (act && !(ld<T>(act, i) > 0.f)) d = 0.f;
    const float xh = (ld<T>(z, i) - mean[c]) * rstd[c];
    st<T>(dz, i, gamma[c] * rstd[c] * (d - (sum_dy[c] + xh * sum_dyx[c]) * inv));
  }
}

hipError_t launch_bn_backward(bool bf16, const void* dy, const void* act, const void* z,
                              const float* mean, const float* rstd, const float* gamma,
                              const float* sum_dy, const float* sum_dyx, int64_t rows, int C,
                              void* dz, hipStream_t s) {
  int64_t total = rows * C;
  if (bf16)
    hipLaunchKernelGGL(bn_backward_kernel<bf16_t>, dim3(grid_for(total)), dim3(256), 0, s,
                       (const bf16_t*)dy, (const bf16_t*)act, (const bf16_t*)z, mean, rstd, gamma,
                       sum_dy, sum_dyx, rows, C, (bf16_t*)dz);
  else
    hipLaunchKernelGGL(bn_backward_kernel<float>, dim3(grid_for(total)), dim3(256), 0, s,
                       (const float*)dy, (const float*)act, (const float*)z, mean, rstd, gamma,
                       sum_dy, sum_dyx, rows, C, (float*)dz);
  return hipGetLastError();
}

template <typename T>
__global__ void relu_mask_kernel(const T* __restrict__ dy, const T* __restrict__ act,
                                 int64_t count, T* __restrict__ out) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count;
       i += (int64_t)gridDim.x * blockDim.x)
    st<T>(out, i, ld<T>(act, i) > 0.f ? ld<T>(dy, i) : 0.f);
}

hipError_t launch_relu_mask(bool bf16, const void* dy, const void* act, int64_t count, void* out,
                            hipStream_t s) {
  if (bf16)
    hipLaunchKernelGGL(relu_mask_kernel<bf16_t>, dim3(grid_for(count)), dim3(256), 0, s,
                       (const bf16_t*)dy, (const bf16_t*)act, count, (bf16_t*)out);
  else
    hipLaunchKernelGGL(relu_mask_kernel<float>, dim3(grid_for(count)), dim3(256), 0, s,
                       (const float*)dy, (const float*)act, count, (float*)out);
  return hipGetLastError();
}

// ----------------------------------------------------------------------------
// pooling
// ----------------------------------------------------------------------------
template <typename T>
__global__ void maxpool_fwd_kernel(const T* __restrict__ x, int n, int h, int w, int c,
                                   T* __restrict__ y) {
  const int ho = h / 2, wo = w / 2;
  const int64_t total = (int64_t)n * ho * wo * c;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int ch = (int)(i % c);
    int64_t q = i / c;
    const int ox = (int)(q % wo);
    q /= wo;
    const int oy = (int)(q % ho);
    const int64_t b = q / ho;
    const int64_t base = ((b * h + 2 * oy) * w + 2 * ox) * c + ch;
    float m = ld<T>(x, base);
    float v = ld<T>(x, base + c);
    m = v > m ? v : m;
    v = ld<T>(x, base + (int64_t)w * c);
    m = v > m ? v : m;
    v = ld<T>(x, base + (int64_t)w * c + c);
    m = v > m ? v : m;
    st<T>(y, i, m);
  }
}

hipError_t launch_maxpool_fwd(bool bf16, const void* x, int n, int h, int w, int c, void* y,
                              hipStream_t s) {
  int64_t total = (int64_t)n * (h / 2) * (w / 2) * c;
  if (bf16)
    hipLaunchKernelGGL(maxpool_fwd_kernel<bf16_t>, dim3(grid_for(total)), dim3(256), 0, s,
                       (const bf16_t*)x, n, h, w, c, (bf16_t*)y);
  else
    hipLaunchKernelGGL(maxpool_fwd_kernel<float>, dim3(grid_for(total)), dim3(256), 0, s,
                       (const float*)x, n, h, w, c, (float*)y);
  return hipGetLastError();
}

template <typename T>
__global__ void maxpool_bwd_kernel(const T* __restrict__ x, const T* __restrict__ dy, int n, int h,
                                   int w, int c, int relu_mask, T* __restrict__ dx) {
  const int ho = h / 2, wo = w / 2;
  const int64_t total = (int64_t)n * ho * wo * c;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int ch = (int)(i % c);
    int64_t q = i / c;
    const int ox = (int)(q % wo);
    q /= wo;
    const int oy = (int)(q % ho);
    const int64_t b = q / ho;
    const int64_t base = ((b * h + 2 * oy) * w + 2 * ox) * c + ch;
    const int64_t off[4] = {base, base + c, base + (int64_t)w * c, base + (int64_t)w * c + c};
    float v[4];
    for (int k = 0; k < 4; ++k) v[k] = ld<T>(x, off[k]);
    int arg = 0;
    for (int k = 1; k < 4; ++k)
      if (v[k] > v[arg]) arg = k;  // strict: the first maximum keeps the gradient
    float g = ld<T>(dy, i);
    if (relu_mask && !(v[arg] > 0.f)) g = 0.f;
    for (int k = 0; k < 4; ++k) st<T>(dx, off[k], k == arg ? g : 0.f);
  }
}

hipError_t launch_maxpool_bwd(bool bf16, const void* x, const void* dy, int n, int h, int w, int c,
                              int relu_mask, void* dx, hipStream_t s) {
  int64_t total = (int64_t)n * (h / 2) * (w / 2) * c;
  if (bf16)
    hipLaunchKernelGGL(maxpool_bwd_kernel<bf16_t>, dim3(grid_for(total)), dim3(256), 0, s,
                       (const bf16_t*)x, (const bf16_t*)dy, n, h, w, c, relu_mask, (bf16_t*)dx);
  else
    hipLaunchKernelGGL(maxpool_bwd_kernel<float>, dim3(grid_for(total)), dim3(256), 0, s,
                       (const float*)x, (const float*)dy, n, h, w, c, relu_mask, (float*)dx);
  return hipGetLastError();
}

template <typename T>
__global__ void gap_fwd_kernel(const T* __restrict__ x, int n, int hw, int c, T* __restrict__ y) {
  const int64_t total = (int64_t)n * c;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t b = i / c;
    const int ch = (int)(i - b * c);
    float s = 0.f;
    for (int p = 0; p < hw; ++p) s += ld<T>(x, (b * hw + p) * c + ch);
    st<T>(y, i, s / (float)hw);
  }
}

hipError_t launch_gap_fwd(bool bf16, const void* x, int n, int hw, int c, void* y, hipStream_t s) {
  int64_t total = (int64_t)n * c;
  if (bf16)
    hipLaunchKernelGGL(gap_fwd_kernel<bf16_t>, dim3(grid_for(total)), dim3(256), 0, s,
                       (const bf16_t*)x, n, hw, c, (bf16_t*)y);
  else
    hipLaunchKernelGGL(gap_fwd_kernel<float>, dim3(grid_for(total)), dim3(256), 0, s,
                       (const float*)x, n, hw, c, (float*)y);
  return hipGetLastError();
}

template <typename T>
__global__ void gap_bwd_kernel(const T* __restrict__ dy, const T* __restrict__ act, int n, int hw,
                               int c, T* __restrict__ dx) {
  const int64_t total = (int64_t)n * hw * c;
  const float inv = 1.0f / (float)hw;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int ch = (int)(i % c);
    const int64_t b = i / ((int64_t)hw * c);
    float g = ld<T>(dy, b * c + ch) * inv;
    if (act && !(ld<T>(act, i) > 0.f)) g = 0.f;
    st<T>(dx, i, g);
  }
}

hipError_t launch_gap_bwd(bool bf16, const void* dy, const void* act, int n, int hw, int c,
                          void* dx, hipStream_t s) {
  int64_t total = (int64_t)n * hw * c;
  if (bf16)
    hipLaunchKernelGGL(gap_bwd_kernel<bf16_t>, dim3(grid_for(total)), dim3(256), 0, s,
                       (const bf16_t*)dy, (const bf16_t*)act, n, hw, c, (bf16_t*)dx);
  else
    hipLaunchKernelGGL(gap_bwd_kernel<float>, dim3(grid_for(total)), dim3(256), 0, s,
                       (const float*)dy, (const float*)act, n, hw, c, (float*)dx);
  return hipGetLastError();
}

// ----------------------------------------------------------------------------
// softmax cross-entropy (one block; rows are independent, the loss is summed
// in a fixed tree order)
// ----------------------------------------------------------------------------
constexpr int CE_MAX_CLASSES = 64;

template <typename T>
__global__ __launch_bounds__(256) void softmax_ce_kernel(const float* __restrict__ logits,
                                                         const int32_t* __restrict__ labels, int n,
                                                         int classes, float* __restrict__ loss,
                                                         float* __restrict__ dz32,
                                                         T* __restrict__ dzt) {
  __shared__ double red[256];
  double acc = 0.0;
  const float invn = 1.0f / (float)n;
  for (int r = threadIdx.x; r < n; r += blockDim.x) {
    const float* z = logits + (int64_t)r * classes;
    float zmax = z[0];
    for (int k = 1; k < classes; ++k) zmax = z[k] > zmax ? z[k] : zmax;
    float se = 0.f;
    for (int k = 0; k < classes; ++k) se += expf(z[k] - zmax);
    const float lse = logf(se) + zmax;
    int y = labels[r];
    const bool valid = (y >= 0 && y < classes);
    if (valid) acc += (double)(lse - z[y]);
    for (int k = 0; k < classes; ++k) {
      float p = expf(z[k] - zmax) / se;
      float d = (p - (valid && k == y ? 1.f : 0.f)) * invn;
      if (dz32) dz32[(int64_t)r * classes + k] = d;
      if (dzt) st<T>(dzt, (int64_t)r * classes + k, d);
    }
  }
  red[threadIdx.x] = acc;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0 && loss) *loss = (float)(red[0] / (double)n);
}

hipError_t launch_softmax_ce(const float* logits, const int32_t* labels, int n, int classes,
                             float* loss, float* dz32, void* dzt, bool bf16, hipStream_t s) {
  if (classes > CE_MAX_CLASSES) return hipErrorInvalidValue;
  if (bf16)
    hipLaunchKernelGGL(softmax_ce_kernel<bf16_t>, dim3(1), dim3(256), 0, s, logits, labels, n,
                       classes, loss, dz32, (bf16_t*)dzt);
  else
    hipLaunchKernelGGL(softmax_ce_kernel<float>, dim3(1), dim3(256), 0, s, logits, labels, n,
                       classes, loss, dz32, (float*)dzt);
  return hipGetLastError();
}

// ----------------------------------------------------------------------------
// zero padding gaps of a gradient vector
// ----------------------------------------------------------------------------
__global__ void zero_ranges_kernel(float* __restrict__ buf, const int64_t* __restrict__ ranges,
                                   int count) {
  const int r = blockIdx.x;
  if (r >= count) return;
  const int64_t b = ranges[2 * r], e = ranges[2 * r + 1];
  for (int64_t i = b + threadIdx.x; i < e; i += blockDim.x) buf[i] = 0.f;
}

hipError_t launch_zero_ranges(float* buf, const int64_t* ranges, int count, hipStream_t s) {
  if (count <= 0) return hipSuccess;
  hipLaunchKernelGGL(zero_ranges_kernel, dim3(count), dim3(64), 0, s, buf, ranges, count);
  return hipGetLastError();
}

}  // namespace hs
