// Attainable rates, reported beside the published peaks:
//  * MFMA: a loop of dense 32x32x16 bf16 MFMAs on register operands (no
//    memory traffic), eight independent accumulators per wave, so that the
//    matrix pipe is the only limit: the ceiling the GEMM kernels can reach at
//    the clock the GPU sustains under MFMA load;
//  * HBM: a plain copy, 16 bytes per lane and access, eight accesses in
//    flight per lane.
#include "kernels.h"

namespace hs {

namespace {
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
}  // namespace

// Lane t of the block: operand element i of A is (t + i) mod 8, of B
// (3 t + i) mod 8 (small integers, exact in bf16 and in the fp32 sums);
// out[block * 512 + t] = the sum of the lane's accumulator elements.
__global__ __launch_bounds__(512) void mfma_loop_kernel(int iters, float* __restrict__ out) {
  const int t = threadIdx.x;
  bf16x8 a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = (__bf16)(float)((t + i) & 7);
    b[i] = (__bf16)(float)((3 * t + i) & 7);
  }
  f32x16 acc[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) acc[j] = (f32x16){};
  for (int k = 0; k < iters; ++k) {
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[j], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < 8; ++j)
#pragma unroll
    for (int e = 0; e < 16; ++e) s += acc[j][e];
  out[(int64_t)blockIdx.x * 512 + t] = s;
}

// Block b copies the 32 KB chunk [b, b + 1) x 256 lanes x 8 x 16 bytes: all
// eight loads of a lane are issued before its stores, the stores bypass the
// caches (nontemporal: the copy is not read back); the last block takes the
// ragged end one vector per lane and step.
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void copy_kernel(const u32x4* __restrict__ src,
                                                    u32x4* __restrict__ dst, int64_t n) {
  const int64_t base = (int64_t)blockIdx.x * 2048 + threadIdx.x;
  if (base + 7 * 256 < n) {
    u32x4 v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = src[base + u * 256];
#pragma unroll
    for (int u = 0; u < 8; ++u) __builtin_nontemporal_store(v[u], dst + base + u * 256);
  } else {
    for (int64_t i = base; i < n; i += 256) dst[i] = src[i];
  }
}

hipError_t launch_copy(const void* src, void* dst, int64_t bytes, hipStream_t s) {
  if (!src || !dst || bytes < 16 || bytes % 16 != 0) return hipErrorInvalidValue;
  const int64_t n = bytes / 16;
  const int64_t blocks = (n + 2047) / 2048;
  if (blocks > 0x7fffffff) return hipErrorInvalidValue;
  hipLaunchKernelGGL(copy_kernel, dim3((unsigned)blocks), dim3(256), 0, s, (const u32x4*)src,
                     (u32x4*)dst, n);
  return hipGetLastError();
}

hipError_t launch_mfma_loop(int blocks, int iters, float* out, hipStream_t s) {
  if (blocks < 1 || iters < 1 || !out) return hipErrorInvalidValue;
  hipLaunchKernelGGL(mfma_loop_kernel, dim3(blocks), dim3(512), 0, s, iters, out);
  return hipGetLastError();
}

}  // namespace hs
