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
__global__ void nchw_to_nhwc_pad_kernel(const float* __restrict__ x, T* __restrict__ y, int n, int c,
                                        int cp, int hw) {
  const int64_t total = (int64_t)n * cp * hw;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t b = i / ((int64_t)hw * cp);
    const int64_t r = i - b * hw * cp;
    const int p = (int)(r / cp), ch = (int)(r - (int64_t)p * cp);
    st<T>(y, i, ch < c ? x[(b * c + ch) * hw + p] : 0.f);
  }
}

hipError_t launch_nchw_to_nhwc_pad(const float* x, void* y, int n, int c, int cp, int hw, bool bf16,
                                   hipStream_t s) {
  const int64_t total = (int64_t)n * cp * hw;
  if (bf16)
    hipLaunchKernelGGL(nchw_to_nhwc_pad_kernel<bf16_t>, dim3(grid_for(total)), dim3(256), 0, s, x,
                       (bf16_t*)y, n, c, cp, hw);
  else
    hipLaunchKernelGGL(nchw_to_nhwc_pad_kernel<float>, dim3(grid_for(total)), dim3(256), 0, s, x,
                       (float*)y, n, c, cp, hw);
  return hipGetLastError();
}

template <typename T>
__global__ void pad_weights_kernel(const float* __restrict__ w, T* __restrict__ wp, int k, int rs,
                                   int c, int cp) {
  const int total = k * rs * cp;
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < total; i += gridDim.x * blockDim.x) {
    const int q = i / cp, ch = i - q * cp;
    st<T>(wp, i, ch < c ? w[q * c + ch] : 0.f);
  }
}

hipError_t launch_pad_weights(const float* w, void* wp, int k, int rs, int c, int cp, bool bf16,
                              hipStream_t s) {
  const int total = k * rs * cp;
  if (bf16)
    hipLaunchKernelGGL(pad_weights_kernel<bf16_t>, dim3(grid_for(total)), dim3(256), 0, s, w,
                       (bf16_t*)wp, k, rs, c, cp);
  else
    hipLaunchKernelGGL(pad_weights_kernel<float>, dim3(grid_for(total)), dim3(256), 0, s, w,
                       (float*)wp, k, rs, c, cp);
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
                                                         const int32_t* __restrict__ labels,
                                                         Segs sg, int classes,
                                                         float* __restrict__ loss,
                                                         float* __restrict__ dz32,
                                                         T* __restrict__ dzt) {
  // block = segment: rows [r0, r1), mean over its n rows
  __shared__ double red[256];
  const int seg = blockIdx.x;
  int r0 = 0, r1 = 0;
#pragma unroll
  for (int i = 0; i < MAX_SEG; ++i)
    if (i == seg) {
      r0 = sg.n0[i];
      r1 = sg.n0[i + 1];
    }
  const int n = r1 - r0;
  double acc = 0.0;
  const float invn = 1.0f / (float)n;
  for (int r = r0 + threadIdx.x; r < r1; r += blockDim.x) {
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
  if (threadIdx.x == 0 && loss) loss[seg] = (float)(red[0] / (double)n);
}

hipError_t launch_softmax_ce(const float* logits, const int32_t* labels, const Segs& sg,
                             int classes, float* loss, float* dz32, void* dzt, bool bf16,
                             hipStream_t s) {
  if (classes > CE_MAX_CLASSES || sg.count < 1 || sg.count > MAX_SEG) return hipErrorInvalidValue;
  if (bf16)
    hipLaunchKernelGGL(softmax_ce_kernel<bf16_t>, dim3(sg.count), dim3(256), 0, s, logits, labels,
                       sg, classes, loss, dz32, (bf16_t*)dzt);
  else
    hipLaunchKernelGGL(softmax_ce_kernel<float>, dim3(sg.count), dim3(256), 0, s, logits, labels,
                       sg, classes, loss, dz32, (float*)dzt);
  return hipGetLastError();
}

// ----------------------------------------------------------------------------
// zero the padding gaps of every worker's gradient vector
// ----------------------------------------------------------------------------
struct BufList {
  float* p[MAX_SEG];
};

__global__ void zero_ranges_kernel(BufList bufs, const int64_t* __restrict__ ranges, int count) {
  const int r = blockIdx.x;
  if (r >= count) return;
  float* buf = bufs.p[0];
#pragma unroll
  for (int i = 1; i < MAX_SEG; ++i)
    if (i == (int)blockIdx.y) buf = bufs.p[i];
  const int64_t b = ranges[2 * r], e = ranges[2 * r + 1];
  for (int64_t i = b + threadIdx.x; i < e; i += blockDim.x) buf[i] = 0.f;
}

hipError_t launch_zero_ranges(float* const* bufs, int nbuf, const int64_t* ranges, int count,
                              hipStream_t s) {
  if (count <= 0) return hipSuccess;
  if (nbuf < 1 || nbuf > MAX_SEG) return hipErrorInvalidValue;
  BufList l{};
  for (int i = 0; i < nbuf; ++i) l.p[i] = bufs[i];
  hipLaunchKernelGGL(zero_ranges_kernel, dim3(count, nbuf), dim3(64), 0, s, l, ranges, count);
  return hipGetLastError();
}

// up to kRangesByValue ranges per launch, in the kernel arguments
constexpr int kRangesByValue = 32;
struct RangeList {
  int64_t r[2 * kRangesByValue];
};

__global__ void zero_ranges_byval_kernel(BufList bufs, RangeList rl, int count) {
  const int r = blockIdx.x;
  if (r >= count) return;
  float* buf = bufs.p[0];
#pragma unroll
  for (int i = 1; i < MAX_SEG; ++i)
    if (i == (int)blockIdx.y) buf = bufs.p[i];
  const int64_t b = rl.r[2 * r], e = rl.r[2 * r + 1];
  for (int64_t i = b + threadIdx.x; i < e; i += blockDim.x) buf[i] = 0.f;
}

hipError_t launch_zero_ranges_host(float* const* bufs, int nbuf, const int64_t* ranges, int count,
                                   hipStream_t s) {
  if (count <= 0) return hipSuccess;
  if (nbuf < 1 || nbuf > MAX_SEG) return hipErrorInvalidValue;
  BufList l{};
  for (int i = 0; i < nbuf; ++i) l.p[i] = bufs[i];
  for (int c0 = 0; c0 < count; c0 += kRangesByValue) {
    const int k = count - c0 < kRangesByValue ? count - c0 : kRangesByValue;
    RangeList rl{};
    for (int i = 0; i < 2 * k; ++i) rl.r[i] = ranges[2 * c0 + i];
    hipLaunchKernelGGL(zero_ranges_byval_kernel, dim3(k, nbuf), dim3(64), 0, s, l, rl, k);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace hs
