// Weight gradient of a 3x3, stride-1, pad-1 convolution in bf16 on the
// 32x32x16 MFMA:  gW[co][r][s][ci] = sum over pixels p of
//                 dy[p][co] * x[p shifted by (r - 1, s - 1)][ci]   (0 outside).
//
// The reduction runs over slices of PIX output pixels (256 for W >= 16, else
// 128): RG = PIX / W rows of one image, or PIX / (H W) whole images when an
// image is smaller than a slice.  Per slice a block stages in LDS
//   * the dy rows of the PIX pixels, 64 output channels:  PIX x 128 bytes;
//   * the input patch those pixels read, with a one-pixel zero frame:
//     (rows + 2) x (W + 2) slots per image, 64 input channels: slot x 128 B.
// Both keep their natural channel-contiguous rows (plain 16-byte stores).
// MFMA fragments need 8 consecutive pixels per lane; they come from the
// transposing LDS read (ds_read_b64_tr_b16), 4 consecutive rows per read.  A
// tap's shift is a row offset in the patch, and the frame supplies the zero
// padding, so the 9 taps are 9 shifted reads of one patch.  The dy fragment
// of a k step is read once and reused by all 9 taps.
//
// Block: 12 waves, 64 (co) x 64 (ci) x 9 taps; wave (wr, wk, wc) owns filter
// row wr (3 taps), co half wk and ci half wc: 3 accumulators of 32 x 32, so
// three waves per SIMD fit in registers.  LDS rows are 128 bytes with the
// 16-byte chunk slot chunk ^ (4 * bit 1 of the row): 4 consecutive rows x 64
// bytes (what 32 lanes read at once) then fall on distinct banks.  A read's
// first row S is a compile-time constant plus a lane term that is a multiple
// of 4 or a fixed lane value; the swizzled offset of the lane's element
// depends only on S mod 4, so each lane precomputes 4 base offsets and every
// read is base[S mod 4] + a compile-time offset (no address arithmetic in the
// loop).  The reduction is split over slices (split-K, per worker segment):
// split y writes its partial gW at out + y * split_stride.
#include "kernels.h"

namespace hs {

namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef short __attribute__((address_space(3))) * lds_i16p;
typedef i16x4 __attribute__((address_space(3))) * lds_v4p;

constexpr int ROWB = 128;   // bytes per LDS row
__device__ inline int swz_off(int row, int byte) {   // byte offset of (row, byte) in LDS
  return row * ROWB + ((((byte >> 4) ^ (((row >> 1) & 1) << 2)) << 4) | (byte & 15));
}

// Geometry of a slice for image width W (square images)
template <int W>
struct Slice {
  static constexpr int PIX = W >= 16 ? 256 : 128;       // output pixels per slice
  static constexpr int HW = W * W;
  static constexpr bool ROWS = HW >= PIX;              // slice = rows of one image
  static constexpr int RG = ROWS ? PIX / W : W;         // output rows per frame
  static constexpr int NF = ROWS ? 1 : PIX / HW;        // frames (images) per slice
  static constexpr int FW = W + 2, FR = RG + 2;         // frame with its zero border
  static constexpr int FS = FR * FW;                    // slots per frame
  static constexpr int SLOTS = NF * FS;
  static constexpr int SPI = ROWS ? W / RG : 1;         // slices per image (ROWS)
  // pixel p of the slice -> frame, row, column
  __device__ static int frame(int p) { return p / (RG * W); }
  __device__ static int prow(int p) { return (p % (RG * W)) / W; }
  __device__ static int pcol(int p) { return p % W; }
  __device__ static int slot(int p, int r, int s) {
    return frame(p) * FS + (prow(p) + r) * FW + pcol(p) + s;
  }
  // the lane's first fragment pixel is 16 kk + kb + 4 h (kb = 0 or 8): its
  // slot is slot(16 kk + 4 h, r, s) + lane_slot(kb) for every kk, h, r, s
  __device__ static int lane_slot(int kb) {
    if (W >= 16) return kb;                // same output row
    if (W == 8) return (kb / 8) * FW;      // next output row
    return (kb / 4) * FW;                  // W = 4: two rows down in the frame
  }
};

}  // namespace

template <int W>
__global__ __launch_bounds__(768) void wgrad3_kernel(GemmParams p) {
  typedef Slice<W> S;
  constexpr int AROWS = S::PIX;
  // bytes per buffer; the B region has 4 spare rows at its end (the 4-row
  // reads at +8 may pass the last slot by up to 3 rows; those values are
  // never used)
  constexpr int STAGE = (AROWS + S::SLOTS + 4) * ROWB;
  constexpr int ACH = AROWS * 8, BCH = S::SLOTS * 8;   // 16-byte chunks
  constexpr int NT = 768;
  constexpr int AIT = (ACH + NT - 1) / NT, BIT = (BCH + NT - 1) / NT;
  __shared__ __attribute__((aligned(16))) char smem[2 * STAGE];

  const ConvGeom& g = p.g;
  const int C = g.C, K = g.K;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wr = wave >> 2, wk = (wave >> 1) & 1, wc = wave & 1;
  const int tiles_c = C / 64;
  const int k0 = (blockIdx.x / tiles_c) * 64, c0 = (blockIdx.x % tiles_c) * 64;

  // this split's slices: segment sg, slices [j0, j1) of the segment
  int sg = 0;
#pragma unroll
  for (int i = 1; i < MAX_SEG; ++i) sg += (i < p.nseg && (int)blockIdx.y >= p.seg_split[i]) ? 1 : 0;
  int sp = 0, s_n0 = 0, s_n1 = 0;
#pragma unroll
  for (int i = 0; i < MAX_SEG; ++i)
    if (i == sg) {
      sp = p.seg_split[i];
      s_n0 = p.seg_n0[i];
      s_n1 = p.seg_n0[i + 1];
    }
  const int nimg = s_n1 - s_n0;
  const int nsl = S::ROWS ? nimg * S::SPI : (nimg + S::NF - 1) / S::NF;
  // split i of the segment takes slices [i kt_per_split, (i + 1) kt_per_split)
  const int j0 = ((int)blockIdx.y - sp) * p.kt_per_split;
  const int cnt = max(0, min(p.kt_per_split, nsl - j0));   // slices of this split
  const int jst = 1;

  const bf16_t* X = (const bf16_t*)p.b;    // x  [n][H][W][C]
  const bf16_t* DY = (const bf16_t*)p.a;   // dy [n][H][W][K]

  // image and first output row of frame f of slice j (image < 0: empty frame)
  auto frame_origin = [&](int j, int f, int& img, int& y0) {
    if (S::ROWS) {
      img = s_n0 + j / S::SPI;
      y0 = (j % S::SPI) * S::RG;
    } else {
      img = s_n0 + j * S::NF + f;
      y0 = 0;
      if (img >= s_n1) img = -1;
    }
  };

  auto load = [&](int j, uint4 (&ra)[AIT], uint4 (&rb)[BIT]) {
#pragma unroll
    for (int i = 0; i < AIT; ++i) {
      const int q = tid + NT * i;
      if (q < ACH) {
        const int px = q >> 3, ch = q & 7;
        int img, y0;
        frame_origin(j, S::frame(px), img, y0);
        const int y = y0 + S::prow(px), x = S::pcol(px);
        ra[i] = img >= 0 ? *(const uint4*)(DY + ((int64_t)(img * W + y) * W + x) * K + k0 + ch * 8)
                         : make_uint4(0, 0, 0, 0);
      }
    }
#pragma unroll
    for (int i = 0; i < BIT; ++i) {
      const int q = tid + NT * i;
      if (q < BCH) {
        const int sl = q >> 3, ch = q & 7;
        const int f = sl / S::FS, rem = sl - f * S::FS;
        const int fy = rem / S::FW, fx = rem - fy * S::FW;
        int img, y0;
        frame_origin(j, f, img, y0);
        const int y = y0 + fy - 1, x = fx - 1;
        const bool ok = img >= 0 && (unsigned)y < (unsigned)W && (unsigned)x < (unsigned)W;
        rb[i] = ok ? *(const uint4*)(X + ((int64_t)(img * W + y) * W + x) * C + c0 + ch * 8)
                   : make_uint4(0, 0, 0, 0);
      }
    }
  };
  auto store = [&](int buf, const uint4 (&ra)[AIT], const uint4 (&rb)[BIT]) {
    char* As = smem + buf * STAGE;
    char* Bs = As + AROWS * ROWB;
#pragma unroll
    for (int i = 0; i < AIT; ++i) {
      const int q = tid + NT * i;
      if (q < ACH) *(uint4*)(As + swz_off(q >> 3, (q & 7) * 16)) = ra[i];
    }
#pragma unroll
    for (int i = 0; i < BIT; ++i) {
      const int q = tid + NT * i;
      if (q < BCH) *(uint4*)(Bs + swz_off(q >> 3, (q & 7) * 16)) = rb[i];
    }
  };
  // transposing read (ds_read_b64_tr_b16): lane q of a 16-lane group gives
  // the address of row (q >> 2), columns 4 (q & 3) .. + 3 of a 4-row block and
  // receives the 4 rows of column q; `off` is the block's compile-time offset
  auto tr_read = [&](const char* lane_base, int off) -> i16x4 {
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4p)(lds_i16p)(short*)(lane_base + off));
  };
  f32x16 acc[3];
#pragma unroll
  for (int t = 0; t < 3; ++t) acc[t] = (f32x16){};

  // lane roles in the 32x32x16 fragments: column (co for dy, ci for x) =
  // 16 (group & 1) + q within the wave's 32; pixels 8 (lane >> 5) + 0..7
  const int grp = lane >> 4, q = lane & 15;
  const int colA = wk * 32 + 16 * (grp & 1);   // co column base of the group
  const int colB = wc * 32 + 16 * (grp & 1);   // ci column base
  const int kb = 8 * (lane >> 5);              // pixel offset of the lane's half
  // base[ph]: offset of the lane's element for a read whose first row is
  // congruent to ph mod 4 (the row's multiple of 4 is added at the read)
  int baseA[4], baseB[4];
#pragma unroll
  for (int ph = 0; ph < 4; ++ph) {
    baseA[ph] = swz_off(ph + kb + (q >> 2), (colA + 4 * (q & 3)) * 2);
    baseB[ph] = swz_off(ph + S::lane_slot(kb) + (q >> 2), (colB + 4 * (q & 3)) * 2);
  }

  // two register sets: the global loads of slice j + 2 are in flight while
  // slice j computes and slice j + 1 (loaded one slice earlier) is stored
  uint4 ra0[AIT], rb0[BIT], ra1[AIT], rb1[BIT];
  if (cnt > 0) {
    load(j0, ra0, rb0);
    store(0, ra0, rb0);
  }
  if (cnt > 1) load(j0 + jst, ra1, rb1);
  __syncthreads();
  // i-th slice of the split: j0 + i * jst
  auto step = [&](int i, int buf, uint4 (&la)[AIT], uint4 (&lb)[BIT], const uint4 (&sa)[AIT],
                  const uint4 (&sb)[BIT]) {
    if (i + 2 < cnt) load(j0 + (i + 2) * jst, la, lb);
    const char* pa = smem + buf * STAGE;
    const char* pb = pa + AROWS * ROWB;
    // read of the 4-row block whose first row is row0 (compile-time) + lane term
    auto rd = [&](const char* base, const int (&lbase)[4], int row0) {
      return tr_read(base + lbase[row0 & 3], (row0 & ~3) * ROWB);
    };
#pragma unroll
    for (int kk = 0; kk < S::PIX / 16; ++kk) {
      i16x4 a0 = rd(pa, baseA, 16 * kk), a1 = rd(pa, baseA, 16 * kk + 4);
      bf16x8 av;
      __builtin_memcpy(&av, &a0, 8);
      __builtin_memcpy((char*)&av + 8, &a1, 8);
      // the wave's filter row is uniform: the three row variants are
      // compile-time code paths selected once per k step.  The taps s = 0, 1,
      // 2 of a row read the patch rows s .. s + 7 after the lane's first
      // slot; the lane holds all rows of its column, so 4-row blocks at +0,
      // +4, +8 give every tap: s = 1 shifts by one bf16 (byte align), s = 2
      // by one dword (register choice).  With W = 4 the lane's 8 pixels span
      // two image rows: each half does the same with blocks at +0 and +4.
#pragma unroll
      for (int r = 0; r < 3; ++r) {
        if (r != wr) continue;
        uint32_t d[2][6];     // [half][dword] of the loaded rows
        if constexpr (W >= 8) {
          const int r0 = S::slot(16 * kk, r, 0);
          i16x4 v0 = rd(pb, baseB, r0), v1 = rd(pb, baseB, r0 + 4), v2 = rd(pb, baseB, r0 + 8);
          uint32_t w[6];
          __builtin_memcpy(&w[0], &v0, 8);
          __builtin_memcpy(&w[2], &v1, 8);
          __builtin_memcpy(&w[4], &v2, 8);
          // tap s uses rows s .. s + 7 = dwords (shifted by s bf16)
#pragma unroll
          for (int s = 0; s < 3; ++s) {
            uint32_t f[4];
#pragma unroll
            for (int i = 0; i < 4; ++i)
              f[i] = s == 0 ? w[i] : (s == 2 ? w[i + 1] : __builtin_amdgcn_alignbyte(w[i + 1], w[i], 2));
            bf16x8 bv;
            __builtin_memcpy(&bv, f, 16);
            acc[s] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bv, av, acc[s], 0, 0, 0);
          }
          (void)d;
        } else {
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const int r0 = S::slot(16 * kk + 4 * h, r, 0);
            i16x4 v0 = rd(pb, baseB, r0), v1 = rd(pb, baseB, r0 + 4);
            __builtin_memcpy(&d[h][0], &v0, 8);
            __builtin_memcpy(&d[h][2], &v1, 8);
          }
#pragma unroll
          for (int s = 0; s < 3; ++s) {
            uint32_t f[4];
#pragma unroll
            for (int h = 0; h < 2; ++h)
#pragma unroll
              for (int i = 0; i < 2; ++i)
                f[2 * h + i] = s == 0 ? d[h][i]
                                      : (s == 2 ? d[h][i + 1]
                                                : __builtin_amdgcn_alignbyte(d[h][i + 1], d[h][i], 2));
            bf16x8 bv;
            __builtin_memcpy(&bv, f, 16);
            acc[s] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bv, av, acc[s], 0, 0, 0);
          }
        }
      }
    }
    if (i + 1 < cnt) store(buf ^ 1, sa, sb);
    __syncthreads();
  };
  for (int i = 0; i < cnt; i += 2) {
    step(i, 0, ra0, rb0, ra1, rb1);
    if (i + 1 < cnt) step(i + 1, 1, ra1, rb1, ra0, rb0);
  }

  // ---- epilogue: lane holds co = k0 + 32 wk + (lane & 31) and, per group of
  // 4 registers, ci = c0 + 32 wc + 8 (r / 4) + 4 (lane >> 5) + 0..3
  const int co = k0 + wk * 32 + (lane & 31);
  float* out = (float*)p.out + (int64_t)blockIdx.y * p.split_stride;
#pragma unroll
  for (int s = 0; s < 3; ++s)
#pragma unroll
    for (int r4 = 0; r4 < 4; ++r4) {
      const int ci = c0 + wc * 32 + 8 * r4 + 4 * (lane >> 5);
      *(float4*)(out + ((int64_t)co * 9 + 3 * wr + s) * C + ci) =
          make_float4(acc[s][4 * r4], acc[s][4 * r4 + 1], acc[s][4 * r4 + 2], acc[s][4 * r4 + 3]);
    }
}

bool wgrad3_ok(const GemmParams& p) {
  const ConvGeom& g = p.g;
  if (g.R != 3 || g.S != 3 || g.stride != 1 || g.pad != 1) return false;
  if (g.H != g.W || (g.W != 32 && g.W != 16 && g.W != 8 && g.W != 4)) return false;
  return g.C % 64 == 0 && g.K % 64 == 0;
}

// slices of one worker segment of nimg images
int wgrad3_slices(const GemmParams& p, int nimg) {
  const int W = p.g.W, HW = W * W, pix = W >= 16 ? 256 : 128;
  if (HW >= pix) return nimg * (HW / pix);
  return (nimg + pix / HW - 1) / (pix / HW);
}

// p: nseg / seg_split / seg_n0 / kt_per_split (slices per split) set by the
// caller, out = partial buffer with split_stride
hipError_t launch_wgrad3(const GemmParams& p, hipStream_t s) {
  if (!wgrad3_ok(p) || p.nseg < 1) return hipErrorInvalidValue;
  const dim3 grid((unsigned)((p.g.K / 64) * (p.g.C / 64)), (unsigned)p.seg_split[p.nseg]);
  switch (p.g.W) {
    case 32: hipLaunchKernelGGL(wgrad3_kernel<32>, grid, dim3(768), 0, s, p); break;
    case 16: hipLaunchKernelGGL(wgrad3_kernel<16>, grid, dim3(768), 0, s, p); break;
    case 8: hipLaunchKernelGGL(wgrad3_kernel<8>, grid, dim3(768), 0, s, p); break;
    default: hipLaunchKernelGGL(wgrad3_kernel<4>, grid, dim3(768), 0, s, p); break;
  }
  return hipGetLastError();
}

}  // namespace hs
