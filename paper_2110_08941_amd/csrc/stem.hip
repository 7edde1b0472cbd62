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
// 128-byte pixel rows.  With x8 set, the block also writes the image in the
// padded NHWC layout (8 channels, 5 of them zero).
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

// With part set, the block also writes its image's batch-norm sums of the
// stored (bf16) output: part[(b * 2 + k) * 64 + c] = sum over the image's
// pixels of y[c]^(k + 1).  Lane c of each wave adds channel c of every row it
// stages (a column of the staged row), the waves' sums are then added in
// order.
__global__ __launch_bounds__(256) void stem_fwd_kernel(const float* __restrict__ x,
                                                       const bf16_t* __restrict__ w,
                                                       bf16_t* __restrict__ y,
                                                       bf16_t* __restrict__ x8,
                                                       float* __restrict__ part) {
  __shared__ __attribute__((aligned(16))) bf16_t img[3 * ST_PLANE + 4];
  __shared__ __attribute__((aligned(16))) char stage[4][32 * ST_ROWB];
  __shared__ float sred[4][2][ST_CO];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, kh = lane >> 5;
  float ssum = 0.f, ssq = 0.f;   // channel `lane`: the wave's rows
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
    if (part) {   // channel `lane` of the row's 32 pixels, as stored
#pragma unroll 8
      for (int px = 0; px < 32; ++px) {
        const float v = __uint_as_float((uint32_t)*(const uint16_t*)(sg + px * ST_ROWB + lane * 2) << 16);
        ssum += v;
        ssq += v * v;
      }
    }
    __builtin_amdgcn_wave_barrier();
  }
  if (part) {
    sred[wave][0][lane] = ssum;
    sred[wave][1][lane] = ssq;
    __syncthreads();
    if (tid < 2 * ST_CO) {
      const int k = tid >> 6, c = tid & (ST_CO - 1);
      part[(b * 2 + k) * ST_CO + c] = ((sred[0][k][c] + sred[1][k][c]) + sred[2][k][c]) + sred[3][k][c];
    }
  }
}

// Weight gradient of the stem: gW[co][k] = sum over the pixels p of a worker's
// images of dy[p][co] x patch[p][k], k = (3 r + s) 3 + ci, in split-K form.
//
// A block takes STW_IMG consecutive images of one worker (split y of the
// launch; segment s owns splits seg_split[s] .. seg_split[s + 1] - 1) and
// writes its partial [64][27] (fp32) at part + y * 1728.  Per image: the fp32
// NCHW image goes to LDS in bf16 as three column-shifted copies
// (img[ci][s][row + 1][c] = x[ci][row][c + s - 1], zero outside), so that the
// 8 consecutive pixels of a tap are one aligned 16-byte read; dy goes to LDS
// a quarter image (8 rows) at a time, transposed to [co][pixel] by the
// copying threads, so that 8 consecutive pixels of a channel are one aligned
// read too; each quarter's inputs are loaded into registers while the
// previous one is computed.  The 32x32x16 MFMA runs with the taps as rows (27 of 32
// used), the output channels as columns (two tiles) and 16 pixels per step;
// the 4 waves take the steps in turn and their accumulators are added in a
// fixed order at the end.
constexpr int STW_IMG = 4;              // images per block
constexpr int STW_ROWP = 32;            // shifted image copy: 32 columns per row
constexpr int STW_COPY = 34 * STW_ROWP; // one shifted copy of one channel
constexpr int STW_QPIX = 256;           // dy pixels per quarter
constexpr int STW_TP = STW_QPIX + 8;    // transposed dy row pitch (bf16)

struct StemWgradArgs {
  const float* x;     // [n][3][32][32]
  const bf16_t* dy;   // [n][32][32][64]
  float* part;        // [splits][64][27]
  int nseg;
  int seg_split[MAX_SEG + 1];
  int seg_n0[MAX_SEG + 1];
  StemBnBwd bn;       // BN > 0: the batch-norm backward formed on the fly
};

// BN: 0 dy is the operand; 1 the operand is the batch-norm backward of dy;
// 2 the same with dy masked by [act > 0]
template <int BN>
__global__ __launch_bounds__(256) void stem_wgrad_kernel(StemWgradArgs a) {
  __shared__ __attribute__((aligned(16))) bf16_t img[9 * STW_COPY];
  // the transposed dy quarter; after the loop, the waves' accumulators
  __shared__ __attribute__((aligned(16))) bf16_t dyt[ST_CO * STW_TP];
  static_assert(3 * 2 * 16 * 64 * 4 <= ST_CO * STW_TP * 2, "accumulators fit the dy buffer");
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, kh = lane >> 5;
  const int y = (int)blockIdx.x;
  int sg = 0;
#pragma unroll
  for (int i = 1; i < MAX_SEG; ++i) sg += (i < a.nseg && y >= a.seg_split[i]) ? 1 : 0;
  int sp = 0, n0 = 0, n1 = 0;
#pragma unroll
  for (int i = 0; i < MAX_SEG; ++i)
    if (i == sg) {
      sp = a.seg_split[i];
      n0 = a.seg_n0[i];
      n1 = a.seg_n0[i + 1];
    }
  const int i0 = n0 + (y - sp) * STW_IMG;
  const int i1 = min(n1, i0 + STW_IMG);
  // batch-norm backward constants of the thread's 8 channels (a thread's
  // dy chunks all hold channels 8 (tid % 8) .. + 7) for this segment
  float bgr[BN ? 8 : 1], bmu[BN ? 8 : 1], brs[BN ? 8 : 1], bk1[BN ? 8 : 1], bk2[BN ? 8 : 1];
  if constexpr (BN > 0) {
    const float* s0 = a.bn.sum0[0];
    const float* s1 = a.bn.sum1[0];
#pragma unroll
    for (int i = 1; i < MAX_SEG; ++i)
      if (i == sg) {
        s0 = a.bn.sum0[i];
        s1 = a.bn.sum1[i];
      }
    const float inv_rows = 1.0f / (float)((n1 - n0) * ST_W * ST_W);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int c = 8 * (tid & 7) + j;
      brs[j] = a.bn.rstd[(int64_t)sg * a.bn.mstride + c];
      bgr[j] = a.bn.gamma[c] * brs[j];
      bmu[j] = a.bn.mean[(int64_t)sg * a.bn.mstride + c];
      bk1[j] = s0[c] * inv_rows;
      bk2[j] = s1[c] * inv_rows;
    }
  }
  const int nq = i1 > i0 ? 4 * (i1 - i0) : 0;   // quarters of this block

  // the lane's tap row k and its offset in the shifted copies (-1: k >= 27)
  const int k = lane & 31;
  const int koff = k < ST_K ? (((k % 3) * 3 + (k / 3) % 3) * 34 + k / 9) * STW_ROWP : -1;
  f32x16 acc[2];
  acc[0] = acc[1] = (f32x16){};

  // quarter q's inputs go to registers one quarter ahead
  float4 xv[3];
  uint4 dv[8], zv[BN ? 8 : 1], mv[BN == 2 ? 8 : 1];
  auto load_x = [&](int im) {
    const float* xb = a.x + (int64_t)im * 3 * ST_W * ST_W;
#pragma unroll
    for (int it = 0; it < 3; ++it) xv[it] = *(const float4*)(xb + 4 * (tid + 256 * it));
  };
  auto load_dy = [&](int im, int qt) {
    const int64_t o = ((int64_t)im * ST_W * ST_W + qt * STW_QPIX) * ST_CO;
#pragma unroll
    for (int it = 0; it < 8; ++it) {
      const int64_t e = o + (int64_t)(tid + 256 * it) * 8;
      dv[it] = *(const uint4*)(a.dy + e);
      if constexpr (BN > 0) zv[it] = *(const uint4*)((const bf16_t*)a.bn.z + e);
      if constexpr (BN == 2) mv[it] = *(const uint4*)((const bf16_t*)a.bn.act + e);
    }
  };
  if (nq > 0) {
    load_x(i0);
    load_dy(i0, 0);
  }
  // the copies' zero borders (never written below)
  for (int i = tid; i < 9 * STW_COPY / 2; i += 256) ((uint32_t*)img)[i] = 0u;

  for (int q = 0; q < nq; ++q) {
    const int qt = q & 3;
    __syncthreads();   // the previous quarter's reads are done
    if (qt == 0) {
      // the image at its three column shifts, rounded to bf16
#pragma unroll
      for (int it = 0; it < 3; ++it) {
        const int e = 4 * (tid + 256 * it);
        const int ci = e >> 10, row = (e >> 5) & 31, col = e & 31;
        const float vv[4] = {xv[it].x, xv[it].y, xv[it].z, xv[it].w};
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
          for (int s2 = 0; s2 < 3; ++s2) {
            const int c = col + u + 1 - s2;
            if (c >= 0 && c < 32) img[((ci * 3 + s2) * 34 + row + 1) * STW_ROWP + c] = f2bf(vv[u]);
          }
      }
    }
    // the dy quarter (rows 8 qt .. 8 qt + 7), transposed into [co][pixel]
#pragma unroll
    for (int it = 0; it < 8; ++it) {
      const int c = tid + 256 * it;               // 16-byte chunk: pixel c / 8, channels 8 (c % 8)
      const int px = c >> 3, co = (c & 7) * 8;
      if constexpr (BN > 0) {   // dz of the 8 channels, as the batch-norm backward forms it
        const uint32_t dw[4] = {dv[it].x, dv[it].y, dv[it].z, dv[it].w};
        const uint32_t zw[4] = {zv[it].x, zv[it].y, zv[it].z, zv[it].w};
        uint32_t mw[4] = {~0u, ~0u, ~0u, ~0u};
        if constexpr (BN == 2) {
          mw[0] = mv[it].x;
          mw[1] = mv[it].y;
          mw[2] = mv[it].z;
          mw[3] = mv[it].w;
        }
        uint32_t ow[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          float o2[2];
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const int j = 2 * e + h;
            float g = __uint_as_float(h ? (dw[e] & 0xffff0000u) : (dw[e] << 16));
            if constexpr (BN == 2) {
              const float m = __uint_as_float(h ? (mw[e] & 0xffff0000u) : (mw[e] << 16));
              if (!(m > 0.f)) g = 0.f;
            }
            const float zf = __uint_as_float(h ? (zw[e] & 0xffff0000u) : (zw[e] << 16));
            const float xh = (zf - bmu[j]) * brs[j];
            o2[h] = bgr[j] * (g - (bk1[j] + xh * bk2[j]));
          }
          ow[e] = (uint32_t)f2bf(o2[0]) | ((uint32_t)f2bf(o2[1]) << 16);
        }
        dv[it] = make_uint4(ow[0], ow[1], ow[2], ow[3]);
      }
      const uint32_t w[4] = {dv[it].x, dv[it].y, dv[it].z, dv[it].w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        dyt[(co + 2 * e) * STW_TP + px] = (bf16_t)(w[e] & 0xffffu);
        dyt[(co + 2 * e + 1) * STW_TP + px] = (bf16_t)(w[e] >> 16);
      }
    }
    if (q + 1 < nq) {
      const int im1 = i0 + ((q + 1) >> 2);
      if (((q + 1) & 3) == 0) load_x(im1);
      load_dy(im1, (q + 1) & 3);
    }
    __syncthreads();
    // steps of 16 pixels: wave w takes steps w, w + 4, w + 8, w + 12
#pragma unroll
    for (int st = 0; st < 4; ++st) {
      const int step = wave + 4 * st;             // pixels 16 step .. + 15 of the quarter
      const int row = qt * 8 + step / 2, col0 = (step & 1) * 16 + 8 * kh;
      uint4 pv = make_uint4(0u, 0u, 0u, 0u);
      if (koff >= 0) pv = *(const uint4*)(img + koff + row * STW_ROWP + col0);
      bf16x8 pa;
      __builtin_memcpy(&pa, &pv, 16);
#pragma unroll
      for (int ct = 0; ct < 2; ++ct) {
        const uint4 dd = *(const uint4*)(dyt + (32 * ct + (lane & 31)) * STW_TP + 16 * step + 8 * kh);
        bf16x8 db8;
        __builtin_memcpy(&db8, &dd, 16);
        acc[ct] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(pa, db8, acc[ct], 0, 0, 0);
      }
    }
  }
  // acc[ct]: lane holds co = 32 ct + (lane & 31), taps k = 8 q + 4 kh + e;
  // waves 1..3 hand theirs to LDS, wave 0 adds them in order and writes
  float (*red)[2][16][64] = (float (*)[2][16][64])dyt;
  __syncthreads();
  if (wave > 0) {
#pragma unroll
    for (int ct = 0; ct < 2; ++ct)
#pragma unroll
      for (int e = 0; e < 16; ++e) red[wave - 1][ct][e][lane] = acc[ct][e];
  }
  __syncthreads();
  if (wave == 0) {
    float* out = a.part + (int64_t)y * (ST_CO * ST_K);
#pragma unroll
    for (int ct = 0; ct < 2; ++ct)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const float v = ((acc[ct][e] + red[0][ct][e][lane]) + red[1][ct][e][lane]) + red[2][ct][e][lane];
        const int kk = 8 * (e >> 2) + 4 * kh + (e & 3);
        if (kk < ST_K) out[(32 * ct + (lane & 31)) * ST_K + kk] = v;
      }
  }
}

}  // namespace

bool stem_ok(int cin, int cout, int k, int stride, int pad, int H, int W) {
  return cin == 3 && cout == ST_CO && k == 3 && stride == 1 && pad == 1 && H == ST_W && W == ST_W;
}

hipError_t launch_stem_fwd(const float* x, const void* w_bf16, void* y, void* x8, int n,
                           hipStream_t s, float* stat_part) {
  if (n < 1) return hipErrorInvalidValue;
  hipLaunchKernelGGL(stem_fwd_kernel, dim3((unsigned)n), dim3(256), 0, s, x,
                     (const bf16_t*)w_bf16, (bf16_t*)y, (bf16_t*)x8, stat_part);
  return hipGetLastError();
}

int stem_wgrad_splits(const int* n, int nseg, int* seg_split) {
  seg_split[0] = 0;
  for (int i = 0; i < nseg; ++i) {
    const int b = n[i] > 0 ? (n[i] + STW_IMG - 1) / STW_IMG : 1;
    seg_split[i + 1] = seg_split[i] + b;
  }
  return seg_split[nseg];
}

hipError_t launch_stem_wgrad(const float* x, const void* dy, float* part, const int* seg_n0,
                             const int* seg_split, int nseg, hipStream_t s, const StemBnBwd* bn) {
  if (nseg < 1 || nseg > MAX_SEG || seg_split[nseg] < 1) return hipErrorInvalidValue;
  if (bn && (!bn->z || !bn->mean || !bn->rstd || !bn->gamma)) return hipErrorInvalidValue;
  if (bn)
    for (int i = 0; i < nseg; ++i)
      if (!bn->sum0[i] || !bn->sum1[i]) return hipErrorInvalidValue;
  StemWgradArgs a{};
  if (bn) a.bn = *bn;
  a.x = x;
  a.dy = (const bf16_t*)dy;
  a.part = part;
  a.nseg = nseg;
  for (int i = 0; i <= nseg; ++i) {
    a.seg_split[i] = seg_split[i];
    a.seg_n0[i] = seg_n0[i];
  }
  for (int i = nseg + 1; i <= MAX_SEG; ++i) {
    a.seg_split[i] = seg_split[nseg];
    a.seg_n0[i] = seg_n0[nseg];
  }
  const dim3 grid((unsigned)seg_split[nseg]);
  if (!bn) hipLaunchKernelGGL(stem_wgrad_kernel<0>, grid, dim3(256), 0, s, a);
  else if (!bn->act) hipLaunchKernelGGL(stem_wgrad_kernel<1>, grid, dim3(256), 0, s, a);
  else hipLaunchKernelGGL(stem_wgrad_kernel<2>, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace hs
