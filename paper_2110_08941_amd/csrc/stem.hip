// The first convolution of the CIFAR networks in bf16: 3 input channels ->
// 64, 3x3, stride 1, pad 1, on 32x32 images, read straight from the caller's
// fp32 NCHW batch.
//
// One block per image (4 waves).  The image is rounded to bf16 into LDS with
// a one-pixel zero frame (3 x 34 x 34); the reduction over (tap, channel),
// k = (3 r + s) 3 + ci, 27 long, is padded to 32 -- two 16-deep steps of the
// 32x32x16 MFMA -- with zero weights.  Weights are the MFMA's A operand (32
// output channels per fragment, read once per block from the bf16 copy of
// theta, whose layout [co][r][s][ci] is exactly [co][k]); the B operand is
// gathered per lane from the framed image (8 values of k for one output
// pixel).  A wave computes 8 output rows of 32 pixels x 64 channels, one row
// at a time: 4 MFMAs, then the row is staged in LDS and written as whole
// 128-byte pixel rows.  The block also writes the image in the padded NHWC
// layout (8 channels, 5 of them zero) that the weight gradient reads.
#include "kernels.h"

namespace hs {

namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

constexpr int ST_W = 32;                 // image side
constexpr int ST_F = ST_W + 2;           // framed side
constexpr int ST_PLANE = ST_F * ST_F;    // framed plane (bf16 values)
constexpr int ST_CO = 64;                // output channels
constexpr int ST_K = 27;                 // reduction length
constexpr int ST_ROWB = 144;             // staging row: 64 channels + 16 bytes

__device__ inline uint32_t pack2s(float a, float b) {
  f32x2 v = {a, b};
  bf16x2 h = __builtin_convertvector(v, bf16x2);
  uint32_t u;
  __builtin_memcpy(&u, &h, 4);
  return u;
}

__global__ __launch_bounds__(256) void stem_fwd_kernel(const float* __restrict__ x,
                                                       const bf16_t* __restrict__ w,
                                                       bf16_t* __restrict__ y,
                                                       bf16_t* __restrict__ x8) {
  __shared__ __attribute__((aligned(16))) bf16_t img[3 * ST_PLANE + 4];
  __shared__ __attribute__((aligned(16))) char stage[4][32 * ST_ROWB];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, kh = lane >> 5;
  const int64_t b = blockIdx.x;

  // the framed image: zero, then the interior rounded to bf16
  for (int i = tid; i < (3 * ST_PLANE + 4) / 2; i += 256) ((uint32_t*)img)[i] = 0u;
  __syncthreads();
  const float* xb = x + b * 3 * ST_W * ST_W;
  float4 v[3];
#pragma unroll
  for (int it = 0; it < 3; ++it) v[it] = *(const float4*)(xb + 4 * (tid + 256 * it));
#pragma unroll
  for (int it = 0; it < 3; ++it) {
    const int e = 4 * (tid + 256 * it);           // element of the NCHW image
    const int ci = e >> 10, row = (e >> 5) & 31, col = e & 31;
    bf16_t* d = img + ci * ST_PLANE + (row + 1) * ST_F + col + 1;
    d[0] = f2bf(v[it].x);
    d[1] = f2bf(v[it].y);
    d[2] = f2bf(v[it].z);
    d[3] = f2bf(v[it].w);
  }

  // weight fragments: rows co = 32 ct + (lane & 31), k = 16 ks + 8 kh + 0..7
  bf16x8 wa[2][2];
#pragma unroll
  for (int ct = 0; ct < 2; ++ct)
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const bf16_t* wr = w + (32 * ct + (lane & 31)) * ST_K;
      uint16_t t[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int k = 16 * ks + 8 * kh + e;
        t[e] = k < ST_K ? wr[k] : (uint16_t)0;
      }
      __builtin_memcpy(&wa[ct][ks], t, 16);
    }
  // the lane's gather offsets into the framed image for its 16 values of k
  // (relative to the output pixel's frame position); -1: k past the end
  int goff[2][8];
#pragma unroll
  for (int ks = 0; ks < 2; ++ks)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int k = 16 * ks + 8 * kh + e;
      goff[ks][e] = k < ST_K ? (k % 3) * ST_PLANE + (k / 9) * ST_F + (k / 3) % 3 : -1;
    }
  __syncthreads();

  // the padded NHWC copy for the weight gradient: pixel p, 8 channels
  if (x8 != nullptr) {
#pragma unroll
    for (int it = 0; it < 4; ++it) {
      const int p = tid + 256 * it;
      const int o = (1 + (p >> 5)) * ST_F + 1 + (p & 31);
      const uint4 q = make_uint4((uint32_t)img[o] | ((uint32_t)img[ST_PLANE + o] << 16),
                                 (uint32_t)img[2 * ST_PLANE + o], 0u, 0u);
      *(uint4*)(x8 + (b * ST_W * ST_W + p) * 8) = q;
    }
  }

  char* sg = stage[wave];
  for (int rr = 0; rr < 8; ++rr) {
    const int row = 8 * wave + rr;
    const int base = row * ST_F + (lane & 31);   // frame position of (row - 1, col - 1)
    bf16x8 pb[2];
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      uint16_t t[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) t[e] = goff[ks][e] >= 0 ? img[base + goff[ks][e]] : (uint16_t)0;
      __builtin_memcpy(&pb[ks], t, 16);
    }
    f32x16 acc[2];
#pragma unroll
    for (int ct = 0; ct < 2; ++ct) {
      acc[ct] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wa[ct][0], pb[0], (f32x16){}, 0, 0, 0);
      acc[ct] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wa[ct][1], pb[1], acc[ct], 0, 0, 0);
    }
    // lane: pixel (lane & 31), channels 32 ct + 8 qq + 4 kh + 0..3
#pragma unroll
    for (int ct = 0; ct < 2; ++ct)
#pragma unroll
      for (int qq = 0; qq < 4; ++qq)
        *(uint2*)(sg + (lane & 31) * ST_ROWB + (32 * ct + 8 * qq + 4 * kh) * 2) =
            make_uint2(pack2s(acc[ct][4 * qq], acc[ct][4 * qq + 1]),
                       pack2s(acc[ct][4 * qq + 2], acc[ct][4 * qq + 3]));
    __builtin_amdgcn_wave_barrier();
    bf16_t* yo = y + (b * ST_W * ST_W + (int64_t)row * ST_W) * ST_CO;
#pragma unroll
    for (int it = 0; it < 4; ++it) {
      const int c = lane + 64 * it;              // 16-byte chunk: pixel c / 8, channels 8 (c % 8)
      const uint4 q = *(const uint4*)(sg + (c >> 3) * ST_ROWB + (c & 7) * 16);
      *(uint4*)(yo + (c >> 3) * ST_CO + (c & 7) * 8) = q;
    }
    __builtin_amdgcn_wave_barrier();
  }
}

}  // namespace

bool stem_ok(int cin, int cout, int k, int stride, int pad, int H, int W) {
  return cin == 3 && cout == ST_CO && k == 3 && stride == 1 && pad == 1 && H == ST_W && W == ST_W;
}

hipError_t launch_stem_fwd(const float* x, const void* w_bf16, void* y, void* x8, int n,
                           hipStream_t s) {
  if (n < 1) return hipErrorInvalidValue;
  hipLaunchKernelGGL(stem_fwd_kernel, dim3((unsigned)n), dim3(256), 0, s, x,
                     (const bf16_t*)w_bf16, (bf16_t*)y, (bf16_t*)x8);
  return hipGetLastError();
}

}  // namespace hs
