// Weighted M-way gradient average and SGD update: one streaming pass over
// HBM.  Each thread handles 16-byte groups of 4 parameters; the M gradient
// streams are read once with non-temporal loads (they are not reused), theta
// and the momentum buffer are read and written once.
//
//   mode 0 (average):  gout = sum_m w_m g_m
//   mode 1 (update):   d = g_0 + wd*theta; mom = mu*mom + d; theta -= lr*mom
//   mode 2 (fused):    the update with g_0 replaced by sum_m w_m g_m
// The weighted sum is accumulated in worker order.  Optionally the new theta
// is also written as a round-to-nearest-even bf16 copy.
#include "kernels.h"

namespace hs {

constexpr int MAXW = 16;
typedef float f4 __attribute__((ext_vector_type(4)));

struct WavgArgs {
  const float* g[MAXW];
  float w[MAXW];
};

template <int MODE, bool MOM, bool BF>
__global__ __launch_bounds__(256) void wavg_sgd_kernel(WavgArgs a, int M, float* __restrict__ theta,
                                                       float* __restrict__ mom,
                                                       float* __restrict__ gout, int64_t P,
                                                       float lr, float mu, float wd,
                                                       uint16_t* __restrict__ tbf) {
  const int64_t groups = P >> 2;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < groups; i += stride) {
    f4 gs;
    if (MODE == 1) {
      gs = __builtin_nontemporal_load((const f4*)a.g[0] + i);
    } else {
      // w_0 g_0, then fma(w_m, g_m, sum) in worker order (the arithmetic the
      // weighted reductions of the one-pass gradient repeat exactly)
      gs = a.w[0] * __builtin_nontemporal_load((const f4*)a.g[0] + i);
      for (int m = 1; m < M; ++m) {
        const f4 v = __builtin_nontemporal_load((const f4*)a.g[m] + i);
        gs.x = __builtin_fmaf(a.w[m], v.x, gs.x);
        gs.y = __builtin_fmaf(a.w[m], v.y, gs.y);
        gs.z = __builtin_fmaf(a.w[m], v.z, gs.z);
        gs.w = __builtin_fmaf(a.w[m], v.w, gs.w);
      }
    }
    if (MODE == 0) {
      __builtin_nontemporal_store(gs, (f4*)gout + i);
      continue;
    }
    f4 th = ((const f4*)theta)[i];
    f4 d = gs + wd * th;
    if (MOM) {
      d = mu * ((const f4*)mom)[i] + d;
      ((f4*)mom)[i] = d;
    }
    th = th - lr * d;
    ((f4*)theta)[i] = th;
    if (BF) {
      uint2 pk = make_uint2((uint32_t)f2bf(th.x) | ((uint32_t)f2bf(th.y) << 16),
                            (uint32_t)f2bf(th.z) | ((uint32_t)f2bf(th.w) << 16));
      ((uint2*)tbf)[i] = pk;
    }
  }
  // tail (P not a multiple of 4): the first block handles it element-wise
  if (blockIdx.x == 0) {
    for (int64_t j = (groups << 2) + threadIdx.x; j < P; j += blockDim.x) {
      float gsum;
      if (MODE == 1) {
        gsum = a.g[0][j];
      } else {
        gsum = a.w[0] * a.g[0][j];
        for (int m = 1; m < M; ++m) gsum = __builtin_fmaf(a.w[m], a.g[m][j], gsum);
      }
      if (MODE == 0) {
        gout[j] = gsum;
        continue;
      }
      float t = theta[j];
      float d = gsum + wd * t;
      if (MOM) {
        d = mu * mom[j] + d;
        mom[j] = d;
      }
      t = t - lr * d;
      theta[j] = t;
      if (BF) tbf[j] = f2bf(t);
    }
  }
}

template <int MODE>
static void launch_m(const WavgArgs& a, int M, float* theta, float* mom, float* gout, int64_t P,
                     float lr, float mu, float wd, uint16_t* tbf, hipStream_t s) {
  int64_t groups = P >> 2;
  int blocks = (int)((groups + 255) / 256);
  const int cap = 256 * 8;  // 8 resident blocks per CU is plenty for a stream
  if (blocks > cap) blocks = cap;
  if (blocks < 1) blocks = 1;
  dim3 g(blocks), b(256);
  if (MODE == 0) {
    hipLaunchKernelGGL((wavg_sgd_kernel<0, false, false>), g, b, 0, s, a, M, theta, mom, gout, P,
                       lr, mu, wd, tbf);
    return;
  }
  if (mom && tbf)
    hipLaunchKernelGGL((wavg_sgd_kernel<MODE, true, true>), g, b, 0, s, a, M, theta, mom, gout, P,
                       lr, mu, wd, tbf);
  else if (mom)
    hipLaunchKernelGGL((wavg_sgd_kernel<MODE, true, false>), g, b, 0, s, a, M, theta, mom, gout,
                       P, lr, mu, wd, tbf);
  else if (tbf)
    hipLaunchKernelGGL((wavg_sgd_kernel<MODE, false, true>), g, b, 0, s, a, M, theta, mom, gout,
                       P, lr, mu, wd, tbf);
  else
    hipLaunchKernelGGL((wavg_sgd_kernel<MODE, false, false>), g, b, 0, s, a, M, theta, mom, gout,
                       P, lr, mu, wd, tbf);
}

hipError_t launch_wavg_sgd(const float* const* g, const float* w, int M, float* theta, float* mom,
                           float* gout, int64_t P, float lr, float mu, float wd,
                           uint16_t* theta_bf16, int mode, hipStream_t s) {
  if (M < 1 || M > MAXW) return hipErrorInvalidValue;
  WavgArgs a;
  for (int m = 0; m < MAXW; ++m) {
    a.g[m] = m < M ? g[m] : nullptr;
    a.w[m] = m < M ? w[m] : 0.f;
  }
  if (mode == 0) launch_m<0>(a, M, theta, mom, gout, P, lr, mu, wd, theta_bf16, s);
  else if (mode == 1) launch_m<1>(a, M, theta, mom, gout, P, lr, mu, wd, theta_bf16, s);
  else launch_m<2>(a, M, theta, mom, gout, P, lr, mu, wd, theta_bf16, s);
  return hipGetLastError();
}

__global__ void to_bf16_kernel(const float* __restrict__ x, uint16_t* __restrict__ y, int64_t P) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < P;
       i += (int64_t)gridDim.x * blockDim.x)
    y[i] = f2bf(x[i]);
}

hipError_t launch_to_bf16(const float* x, uint16_t* y, int64_t P, hipStream_t s) {
  int64_t blocks = (P + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(to_bf16_kernel, dim3((int)blocks), dim3(256), 0, s, x, y, P);
  return hipGetLastError();
}

}  // namespace hs
