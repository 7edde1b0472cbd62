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
// Both keep their natural channel-contiguous rows.  They are copied straight
// from global memory into LDS (16 bytes per lane, no registers held); frame
// slots and missing images copy a static zero vector, so no copy is
// conditional, and the two stage buffers are distinct LDS arrays (the slice
// loop is unrolled by two) so that the copies into one buffer are not mistaken
// for writes to the one being read.
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
// depends only on S mod 4, so each lane precomputes 4 base offsets (with its
// wave's filter-row shift folded in) and every read is base[S mod 4] + a
// compile-time offset: no address arithmetic and no branches in the loop.
// The next k step's fragments are read while the current step's MFMAs run.  The reduction is split over slices (split-K, per worker segment):
// split y writes its partial gW at out + y * split_stride.
//
// Stride 2 (wgrad3s2_kernel, output width WO, input width 2 WO): an output
// pixel o reads input rows 2 o - 1, 2 o, 2 o + 1 (and the same columns), so
// consecutive output pixels are two input pixels apart.  The patch is kept
// as four parity planes of the input, plane (a, b) holding the pixels of
// row parity a and column parity b with one zero row on top and one zero
// column on the left: in plane coordinates tap r = 0 is row o of the odd
// plane, r = 1 row o + 1 of the even one, r = 2 row o + 1 of the odd one
// (likewise for columns).  A tap is again a row offset into one plane, and
// the lane's 8 consecutive output pixels are 8 consecutive plane slots:
// taps s = 0 and s = 2 are the odd-column plane at shifts 0 and 1 (three
// reads, one byte-aligned), s = 1 the even-column plane at shift 1 (two
// reads).  A slice is 64 output pixels (four planes of its input take four
// times the slots of a stride-1 patch).  With a2 set (PROJ) the kernel also
// takes the weight gradient of the residual block's 1x1 stride-2 projection
// of the same input: its input pixel (2 o, 2 p) is what tap (1, 1) reads,
// so the four waves of filter row 1 add one more MFMA per k step, with the
// projection's dy (a2, staged as dy) against the tap's operand, into a
// fourth accumulator; that partial follows the 3x3 one in each split's
// output (out + y split_stride + 9 K C, [K][C]).
#include "kernels.h"

namespace hs {

namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef short __attribute__((address_space(3))) * lds_i16p;
typedef i16x4 __attribute__((address_space(3))) * lds_v4p;
typedef __attribute__((address_space(3))) void* lds_ptr;          // LDS
typedef __attribute__((address_space(1))) const void* gbl_cptr;   // global

// source of the zero slots of the patch (frame, missing images)
__device__ __attribute__((aligned(16))) uint4 g_zero16;

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
  constexpr int NT = 768;
  constexpr int AROWS = S::PIX;
  constexpr int ACH = AROWS * 8, BCH = S::SLOTS * 8;   // 16-byte chunks
  constexpr int AIT = (ACH + NT - 1) / NT, BIT = (BCH + NT - 1) / NT;
  static_assert(ACH % 64 == 0, "dy rows: whole waves per copy round");
  // patch rows: the last copying wave writes whole 8-row groups, and the
  // 4-row reads at +8 may pass the last slot by up to 3 rows (values unused)
  constexpr int BR8 = (S::SLOTS + 7) / 8 * 8;
  constexpr int BROWS = BR8 > S::SLOTS + 4 ? BR8 : S::SLOTS + 4;
  __shared__ __attribute__((aligned(16))) char sA0[AROWS * ROWB];
  __shared__ __attribute__((aligned(16))) char sA1[AROWS * ROWB];
  __shared__ __attribute__((aligned(16))) char sB0[BROWS * ROWB];
  __shared__ __attribute__((aligned(16))) char sB1[BROWS * ROWB];

  const ConvGeom& g = p.g;
  const int C = g.C, K = g.K;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wr = wave >> 2, wk = (wave >> 1) & 1, wc = wave & 1;
  // Workgroups are handed to the 8 XCDs (each with its own L2) in turn.  The
  // tiles of one split read the same dy rows and input patch, so the block
  // index is remapped to put all tiles of a split on one XCD, where they run
  // side by side and share those reads through its L2: the first 8 q blocks
  // (q = blocks / 8) are dealt so that XCD k gets logical blocks
  // [k q, (k + 1) q) in order; the rest keep their index.
  const int nblk = (int)(gridDim.x * gridDim.y), q8 = nblk / 8;
  int lb = (int)(blockIdx.y * gridDim.x + blockIdx.x);
  if (lb < 8 * q8) lb = (lb % 8) * q8 + lb / 8;
  const int bx = lb % (int)gridDim.x, by = lb / (int)gridDim.x;
  const int tiles_c = C / 64;
  const int k0 = (bx / tiles_c) * 64, c0 = (bx % tiles_c) * 64;

  // this split's slices: segment sg, slices [j0, j0 + cnt) of the segment
  int sg = 0;
#pragma unroll
  for (int i = 1; i < MAX_SEG; ++i) sg += (i < p.nseg && by >= p.seg_split[i]) ? 1 : 0;
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
  const int j0 = (by - sp) * p.kt_per_split;
  const int cnt = max(0, min(p.kt_per_split, nsl - j0));   // slices of this split

  const bf16_t* X = (const bf16_t*)p.b;    // x  [n][H][W][C]
  const bf16_t* DY = (const bf16_t*)p.a;   // dy [n][H][W][K]
  // the zero vector's address, taken once and kept in registers (a reload
  // inside the loop would be a scalar memory load, whose out-of-order return
  // forces full waits on every LDS read)
  const void* zero16 = &g_zero16;
  __asm__ volatile("" : "+s"(zero16));


  // Copy slice j into (As, Bs).  Copy round i of wave w writes LDS chunks
  // NT i + 64 w + lane (row = chunk / 8, slot in the row = chunk % 8); the
  // swizzle is applied on the global side: that slot holds channel chunk
  // slot ^ (4 * bit 1 of the row).  What a lane copies depends on the slice
  // only through a uniform base (image, first row): the lane parts are
  // computed once here.
  //   dy row:  element offset aoff (pixel in the slice + channel chunk) and,
  //            for whole-image slices, the frame (image) index afr;
  //   patch:   element offset boff relative to the slot (y0 - 1, -1) of the
  //            frame, the row term bfy = fy - 1 for the image-row check, and
  //            the frame index bfr; slots outside the image columns, or past
  //            the last chunk, get bfy = bfr = a value no check passes.
  constexpr int NEVER = 1 << 28;
  int aoff[AIT], afr[AIT], boff[BIT], bfy[BIT], bfr[BIT];
#pragma unroll
  for (int i = 0; i < AIT; ++i) {
    const int d = tid + NT * i, row = d >> 3;
    const int ch = (d & 7) ^ (((row >> 1) & 1) << 2);
    afr[i] = S::frame(row);
    aoff[i] = ((afr[i] * S::HW * (S::ROWS ? 0 : 1)) + S::prow(row) * W + S::pcol(row)) * K + ch * 8;
  }
#pragma unroll
  for (int i = 0; i < BIT; ++i) {
    const int d = tid + NT * i, sl = d >> 3;
    const int ch = (d & 7) ^ (((sl >> 1) & 1) << 2);
    const int f = sl / S::FS, rem = sl - f * S::FS;
    const int fy = rem / S::FW, fx = rem - fy * S::FW;
    const bool colok = d < BCH && (unsigned)(fx - 1) < (unsigned)W;
    boff[i] = ((S::ROWS ? 0 : f * S::HW) + (fy - 1) * W + (fx - 1)) * C + ch * 8;
    bfy[i] = colok ? fy - 1 : NEVER;
    bfr[i] = colok ? f : NEVER;
  }
  auto copy_slice = [&](int j, char* As, char* Bs) {
    // uniform part: first image and first output row of the slice; the
    // number of frames that hold an image
    int img0, y0, nfr;
    if (S::ROWS) {
      img0 = s_n0 + j / S::SPI;
      y0 = (j % S::SPI) * S::RG;
      nfr = 1;
    } else {
      img0 = s_n0 + j * S::NF;
      y0 = 0;
      nfr = s_n1 - img0;
    }
    const bf16_t* dyb = DY + ((int64_t)(img0 * W + y0) * W) * K + k0;
    const bf16_t* xb = X + ((int64_t)(img0 * W + y0) * W) * C + c0;
#pragma unroll
    for (int i = 0; i < AIT; ++i) {
      if (NT * i + 64 * wave >= ACH) continue;              // wave-uniform
      const void* src = afr[i] < nfr || S::ROWS ? (const void*)(dyb + aoff[i]) : zero16;
      __builtin_amdgcn_global_load_lds((gbl_cptr)src, (lds_ptr)(As + (NT * i + 64 * wave) * 16), 16, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < BIT; ++i) {
      if (NT * i + 64 * wave >= BCH) continue;              // wave-uniform
      const bool ok = bfr[i] < nfr && (unsigned)(y0 + bfy[i]) < (unsigned)W;
      const void* src = ok ? (const void*)(xb + boff[i]) : zero16;
      __builtin_amdgcn_global_load_lds((gbl_cptr)src, (lds_ptr)(Bs + (NT * i + 64 * wave) * 16), 16, 0, 0);
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
  // base[ph]: offset of the lane's element for a read whose compile-time
  // first row is congruent to ph mod 4 (its multiple of 4 is added at the
  // read); the patch bases include the wave's filter-row shift wr * FW
  // (adding 4k rows adds 4k * ROWB: the swizzle depends on bit 1 only)
  int baseA[4], baseB[4];
#pragma unroll
  for (int ph = 0; ph < 4; ++ph) {
    baseA[ph] = swz_off(ph + kb + (q >> 2), (colA + 4 * (q & 3)) * 2);
    baseB[ph] = swz_off(ph + wr * S::FW + S::lane_slot(kb) + (q >> 2), (colB + 4 * (q & 3)) * 2);
  }
  auto rd = [&](const char* base, const int (&lbase)[4], int row0) {
    return tr_read(base + lbase[row0 & 3], (row0 & ~3) * ROWB);
  };
  // fragments of k step kk: dy (2 reads) and the patch rows of the wave's
  // filter row (3 reads; W = 4: 2 per image-row half)
  constexpr int NBR = W >= 8 ? 3 : 4;
  auto read_k = [&](const char* pa, const char* pb, int kk, i16x4 (&fa)[2], i16x4 (&fbv)[NBR]) {
    fa[0] = rd(pa, baseA, 16 * kk);
    fa[1] = rd(pa, baseA, 16 * kk + 4);
    if constexpr (W >= 8) {
      const int r0 = S::slot(16 * kk, 0, 0);
      fbv[0] = rd(pb, baseB, r0);
      fbv[1] = rd(pb, baseB, r0 + 4);
      fbv[2] = rd(pb, baseB, r0 + 8);
    } else {
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int r0 = S::slot(16 * kk + 4 * h, 0, 0);
        fbv[2 * h] = rd(pb, baseB, r0);
        fbv[2 * h + 1] = rd(pb, baseB, r0 + 4);
      }
    }
  };
  // MFMA operands of a k step: the dy fragment and the patch fragment of
  // each tap.  The three taps s = 0, 1, 2 of the wave's filter row read the
  // patch rows s .. s + 7 after the lane's first slot; the lane holds all rows
  // of its column, so 4-row blocks at +0, +4, +8 give every tap: s = 1 shifts
  // by one bf16 (byte align), s = 2 by one dword (register choice).  With
  // W = 4 the lane's 8 pixels span two image rows: each half does the same
  // with blocks at +0 and +4.
  auto prep_k = [&](const i16x4 (&fa)[2], const i16x4 (&fbv)[NBR], bf16x8& av, bf16x8 (&bv)[3]) {
    __builtin_memcpy(&av, &fa[0], 8);
    __builtin_memcpy((char*)&av + 8, &fa[1], 8);
    if constexpr (W >= 8) {
      uint32_t w[6];
      __builtin_memcpy(&w[0], &fbv[0], 8);
      __builtin_memcpy(&w[2], &fbv[1], 8);
      __builtin_memcpy(&w[4], &fbv[2], 8);
#pragma unroll
      for (int s = 0; s < 3; ++s) {
        uint32_t f[4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
          f[i] = s == 0 ? w[i] : (s == 2 ? w[i + 1] : __builtin_amdgcn_alignbyte(w[i + 1], w[i], 2));
        __builtin_memcpy(&bv[s], f, 16);
      }
    } else {
      uint32_t d[2][4];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        __builtin_memcpy(&d[h][0], &fbv[2 * h], 8);
        __builtin_memcpy(&d[h][2], &fbv[2 * h + 1], 8);
      }
#pragma unroll
      for (int s = 0; s < 3; ++s) {
        uint32_t f[4];
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
          for (int i = 0; i < 2; ++i)
            f[2 * h + i] = s == 0 ? d[h][i]
                                  : (s == 2 ? d[h][i + 1] : __builtin_amdgcn_alignbyte(d[h][i + 1], d[h][i], 2));
        __builtin_memcpy(&bv[s], f, 16);
      }
    }
  };

  constexpr int KK = S::PIX / 16;
  i16x4 fa[2], fbv[NBR];
  // the i-th slice of the split from (pa, pb) while slice i + 1 is copied into (na, nb)
  auto slice = [&](int i, const char* pa, const char* pb, char* na, char* nb) {
    const bool more = i + 1 < cnt;
    if (more) copy_slice(j0 + i + 1, na, nb);
    // per k step: assemble this step's operands (read during the previous
    // step), issue the next step's reads, then the MFMAs; the scheduling
    // barriers keep that order (a pending global-to-LDS copy makes every LDS
    // wait a full one, so operands are consumed before new reads are issued)
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      bf16x8 av, bv[3];
      prep_k(fa, fbv, av, bv);
      __builtin_amdgcn_sched_barrier(0);
      i16x4 ga[2], gb[NBR];
      if (kk + 1 < KK) read_k(pa, pb, kk + 1, ga, gb);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int s = 0; s < 3; ++s) acc[s] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bv[s], av, acc[s], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
      if (kk + 1 < KK) {
        fa[0] = ga[0];
        fa[1] = ga[1];
#pragma unroll
        for (int u = 0; u < NBR; ++u) fbv[u] = gb[u];
      }
    }
    // this wave's copies have landed; after the barrier every wave's have
    __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (more) read_k(na, nb, 0, fa, fbv);
  };
  if (cnt > 0) {
    copy_slice(j0, sA0, sB0);
    __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    read_k(sA0, sB0, 0, fa, fbv);
  }
  for (int i = 0; i < cnt; i += 2) {
    slice(i, sA0, sB0, sA1, sB1);
    if (i + 1 < cnt) slice(i + 1, sA1, sB1, sA0, sB0);
  }

  // ---- epilogue: lane holds co = k0 + 32 wk + (lane & 31) and, per group of
  // 4 registers, ci = c0 + 32 wc + 8 (r / 4) + 4 (lane >> 5) + 0..3
  const int co = k0 + wk * 32 + (lane & 31);
  float* out = (float*)p.out + (int64_t)by * p.split_stride;
#pragma unroll
  for (int s = 0; s < 3; ++s)
#pragma unroll
    for (int r4 = 0; r4 < 4; ++r4) {
      const int ci = c0 + wc * 32 + 8 * r4 + 4 * (lane >> 5);
      *(float4*)(out + ((int64_t)co * 9 + 3 * wr + s) * C + ci) =
          make_float4(acc[s][4 * r4], acc[s][4 * r4 + 1], acc[s][4 * r4 + 2], acc[s][4 * r4 + 3]);
    }
}

namespace {

// Geometry of a stride-2 slice for output width WO (square images, input
// width 2 WO).  Slot of plane pl = 2 a + b (row parity a, column parity b),
// plane row fy, plane column fx in frame f: f FS + pl PS + fy FW + fx; plane
// row fy of a slice whose first output row is y0 holds input row
// 2 (y0 + fy - 1) + a, plane column fx input column 2 (fx - 1) + b.
template <int WO>
struct Slice2 {
  static constexpr int PIX = 64;                        // output pixels per slice
  static constexpr int WI = 2 * WO;                     // input width
  static constexpr int HWO = WO * WO, HWI = WI * WI;
  static constexpr bool ROWS = HWO >= PIX;              // slice = rows of one image
  static constexpr int RG = ROWS ? PIX / WO : WO;       // output rows per frame
  static constexpr int NF = ROWS ? 1 : PIX / HWO;       // frames (images) per slice
  static constexpr int FW = WO + 1, FR = RG + 1;        // plane with its zero row / column
  static constexpr int PS = FR * FW;                    // slots per plane
  static constexpr int FS = 4 * PS;                     // slots per frame
  static constexpr int SLOTS = NF * FS;
  static constexpr int SPI = ROWS ? WO / RG : 1;        // slices per image (ROWS)
  __device__ static int frame(int p) { return p / (RG * WO); }
  __device__ static int prow(int p) { return (p % (RG * WO)) / WO; }
  __device__ static int pcol(int p) { return p % WO; }
  // slot of output pixel p in plane 0 at plane row / column offset 0: the
  // plane, the filter row's row offset and the tap's column offset are added
  __device__ static int slot(int p) { return frame(p) * FS + prow(p) * FW + pcol(p); }
  // the lane's first fragment pixel is 16 kk + kb + 4 h (kb = 0 or 8)
  __device__ static int lane_slot(int kb) {
    if (WO >= 16) return kb;               // same output row
    if (WO == 8) return (kb / 8) * FW;     // next output row
    return (kb / 4) * FW;                  // WO = 4: two rows down
  }
};

}  // namespace

template <int WO, bool PROJ>
__global__ __launch_bounds__(768) void wgrad3s2_kernel(GemmParams p) {
  typedef Slice2<WO> S;
  constexpr int NT = 768;
  constexpr int AROWS = S::PIX;
  constexpr int ACH = AROWS * 8, BCH = S::SLOTS * 8;   // 16-byte chunks
  constexpr int AIT = (ACH + NT - 1) / NT, BIT = (BCH + NT - 1) / NT;
  static_assert(ACH % 64 == 0, "dy rows: whole waves per copy round");
  // plane rows: the 4-row reads at +8 may pass the last slot by up to 3 rows
  // (values unused)
  constexpr int BR8 = (S::SLOTS + 7) / 8 * 8;
  constexpr int BROWS = BR8 > S::SLOTS + 4 ? BR8 : S::SLOTS + 4;
  __shared__ __attribute__((aligned(16))) char sA0[AROWS * ROWB];
  __shared__ __attribute__((aligned(16))) char sA1[AROWS * ROWB];
  __shared__ __attribute__((aligned(16))) char sB0[BROWS * ROWB];
  __shared__ __attribute__((aligned(16))) char sB1[BROWS * ROWB];
  // the projection's dy rows (PROJ)
  __shared__ __attribute__((aligned(16))) char sC0[PROJ ? AROWS * ROWB : 16];
  __shared__ __attribute__((aligned(16))) char sC1[PROJ ? AROWS * ROWB : 16];

  const ConvGeom& g = p.g;
  const int C = g.C, K = g.K;
  // the wave index as a scalar: the projection's MFMA is then skipped by a
  // scalar branch in the other waves, not issued with an empty exec mask
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wr = wave >> 2, wk = (wave >> 1) & 1, wc = wave & 1;
  const bool sc = PROJ && wr == 1;   // wave-uniform: this wave also takes the projection
  // all tiles of a split on one XCD, as in the stride-1 kernel
  const int nblk = (int)(gridDim.x * gridDim.y), q8 = nblk / 8;
  int lb = (int)(blockIdx.y * gridDim.x + blockIdx.x);
  if (lb < 8 * q8) lb = (lb % 8) * q8 + lb / 8;
  const int bx = lb % (int)gridDim.x, by = lb / (int)gridDim.x;
  const int tiles_c = C / 64;
  const int k0 = (bx / tiles_c) * 64, c0 = (bx % tiles_c) * 64;

  int sg = 0;
#pragma unroll
  for (int i = 1; i < MAX_SEG; ++i) sg += (i < p.nseg && by >= p.seg_split[i]) ? 1 : 0;
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
  const int j0 = (by - sp) * p.kt_per_split;
  const int cnt = max(0, min(p.kt_per_split, nsl - j0));

  const bf16_t* X = (const bf16_t*)p.b;    // x  [n][2 WO][2 WO][C]
  const bf16_t* DY = (const bf16_t*)p.a;   // dy [n][WO][WO][K]
  const bf16_t* DY2 = (const bf16_t*)p.a2; // the projection's dy, same layout (PROJ)
  const void* zero16 = &g_zero16;
  __asm__ volatile("" : "+s"(zero16));

  // Copy slice j into (As, Bs), as the stride-1 kernel: chunk NT i + 64 w +
  // lane of copy round i; the lane parts of the source offsets are computed
  // once.  Plane slots: element offset boff relative to input row 2 y0 of
  // the frame, the relative input row bfy for the image-row check, the
  // frame bfr; zero-column slots and chunks past the last get NEVER.
  constexpr int NEVER = 1 << 28;
  int aoff[AIT], afr[AIT], boff[BIT], bfy[BIT], bfr[BIT];
#pragma unroll
  for (int i = 0; i < AIT; ++i) {
    const int d = tid + NT * i, row = d >> 3;
    const int ch = (d & 7) ^ (((row >> 1) & 1) << 2);
    afr[i] = S::frame(row);
    aoff[i] = ((afr[i] * S::HWO * (S::ROWS ? 0 : 1)) + S::prow(row) * WO + S::pcol(row)) * K + ch * 8;
  }
#pragma unroll
  for (int i = 0; i < BIT; ++i) {
    const int d = tid + NT * i, sl = d >> 3;
    const int ch = (d & 7) ^ (((sl >> 1) & 1) << 2);
    const int f = sl / S::FS, rem = sl - f * S::FS;
    const int pl = rem / S::PS, r2 = rem - pl * S::PS;
    const int fy = r2 / S::FW, fx = r2 - fy * S::FW;
    const int iy = 2 * (fy - 1) + (pl >> 1), ix = 2 * (fx - 1) + (pl & 1);
    const bool colok = d < BCH && (unsigned)ix < (unsigned)S::WI;
    boff[i] = ((S::ROWS ? 0 : f * S::HWI) + iy * S::WI + ix) * C + ch * 8;
    bfy[i] = colok ? iy : NEVER;
    bfr[i] = colok ? f : NEVER;
  }
  auto copy_slice = [&](int j, char* As, char* Bs, char* Cs) {
    int img0, y0, nfr;
    if (S::ROWS) {
      img0 = s_n0 + j / S::SPI;
      y0 = (j % S::SPI) * S::RG;
      nfr = 1;
    } else {
      img0 = s_n0 + j * S::NF;
      y0 = 0;
      nfr = s_n1 - img0;
    }
    const int64_t dyo = ((int64_t)(img0 * WO + y0) * WO) * K + k0;
    const bf16_t* xb = X + ((int64_t)(img0 * S::WI + 2 * y0) * S::WI) * C + c0;
#pragma unroll
    for (int i = 0; i < AIT; ++i) {
      if (NT * i + 64 * wave >= ACH) continue;              // wave-uniform
      const bool live = afr[i] < nfr || S::ROWS;
      const void* src = live ? (const void*)(DY + dyo + aoff[i]) : zero16;
      __builtin_amdgcn_global_load_lds((gbl_cptr)src, (lds_ptr)(As + (NT * i + 64 * wave) * 16), 16, 0, 0);
      if constexpr (PROJ) {
        const void* src2 = live ? (const void*)(DY2 + dyo + aoff[i]) : zero16;
        __builtin_amdgcn_global_load_lds((gbl_cptr)src2, (lds_ptr)(Cs + (NT * i + 64 * wave) * 16), 16, 0, 0);
      }
    }
#pragma unroll
    for (int i = 0; i < BIT; ++i) {
      if (NT * i + 64 * wave >= BCH) continue;              // wave-uniform
      const bool ok = bfr[i] < nfr && (unsigned)(2 * y0 + bfy[i]) < (unsigned)S::WI;
      const void* src = ok ? (const void*)(xb + boff[i]) : zero16;
      __builtin_amdgcn_global_load_lds((gbl_cptr)src, (lds_ptr)(Bs + (NT * i + 64 * wave) * 16), 16, 0, 0);
    }
  };
  auto tr_read = [&](const char* lane_base, int off) -> i16x4 {
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4p)(lds_i16p)(short*)(lane_base + off));
  };
  constexpr int NACC = PROJ ? 4 : 3;
  f32x16 acc[NACC];
#pragma unroll
  for (int t = 0; t < NACC; ++t) acc[t] = (f32x16){};

  const int grp = lane >> 4, q = lane & 15;
  const int colA = wk * 32 + 16 * (grp & 1);
  const int colB = wc * 32 + 16 * (grp & 1);
  const int kb = 8 * (lane >> 5);
  // filter row wr: plane row parity and row offset (r = 0: odd, +0;
  // r = 1: even, +1; r = 2: odd, +1); the odd-column plane at column offset
  // 0 (taps s = 0, 2) and the even-column plane at offset 1 (tap s = 1)
  const int pa = wr == 1 ? 0 : 1, dr = wr == 0 ? 0 : 1;
  const int rowB = dr * S::FW + S::lane_slot(kb) + (q >> 2);
  int baseA[4], baseO[4], baseE[4];
#pragma unroll
  for (int ph = 0; ph < 4; ++ph) {
    baseA[ph] = swz_off(ph + kb + (q >> 2), (colA + 4 * (q & 3)) * 2);
    baseO[ph] = swz_off(ph + (2 * pa + 1) * S::PS + rowB, (colB + 4 * (q & 3)) * 2);
    baseE[ph] = swz_off(ph + 2 * pa * S::PS + 1 + rowB, (colB + 4 * (q & 3)) * 2);
  }
  auto rd = [&](const char* base, const int (&lbase)[4], int row0) {
    return tr_read(base + lbase[row0 & 3], (row0 & ~3) * ROWB);
  };
  // fragments of k step kk: dy (2 reads), the odd-column plane (3 reads; WO
  // = 4: 2 per image-row half) and the even-column plane (2; WO = 4: 1 per
  // half)
  constexpr int NBO = WO >= 8 ? 3 : 4;
  constexpr int NBE = 2;
  // (the projection's dy fragment, fc, is read by the filter-row-1 waves)
  auto read_k = [&](const char* pa_, const char* pb_, const char* pc_, int kk, i16x4 (&fa)[2],
                    i16x4 (&fo)[NBO], i16x4 (&fe)[NBE], i16x4 (&fc)[2]) {
    fa[0] = rd(pa_, baseA, 16 * kk);
    fa[1] = rd(pa_, baseA, 16 * kk + 4);
    if (sc) {
      fc[0] = rd(pc_, baseA, 16 * kk);
      fc[1] = rd(pc_, baseA, 16 * kk + 4);
    }
    if constexpr (WO >= 8) {
      const int r0 = S::slot(16 * kk);
      fo[0] = rd(pb_, baseO, r0);
      fo[1] = rd(pb_, baseO, r0 + 4);
      fo[2] = rd(pb_, baseO, r0 + 8);
      fe[0] = rd(pb_, baseE, r0);
      fe[1] = rd(pb_, baseE, r0 + 4);
    } else {
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int r0 = S::slot(16 * kk + 4 * h);
        fo[2 * h] = rd(pb_, baseO, r0);
        fo[2 * h + 1] = rd(pb_, baseO, r0 + 4);
        fe[h] = rd(pb_, baseE, r0);
      }
    }
  };
  // operands: bv[0] odd plane at shift 0, bv[2] at shift 1 (byte align),
  // bv[1] the even plane as read
  auto prep_k = [&](const i16x4 (&fa)[2], const i16x4 (&fo)[NBO], const i16x4 (&fe)[NBE],
                    bf16x8& av, bf16x8 (&bv)[3]) {
    __builtin_memcpy(&av, &fa[0], 8);
    __builtin_memcpy((char*)&av + 8, &fa[1], 8);
    __builtin_memcpy(&bv[1], &fe[0], 8);
    __builtin_memcpy((char*)&bv[1] + 8, &fe[1], 8);
    if constexpr (WO >= 8) {
      uint32_t w[6];
      __builtin_memcpy(&w[0], &fo[0], 8);
      __builtin_memcpy(&w[2], &fo[1], 8);
      __builtin_memcpy(&w[4], &fo[2], 8);
      uint32_t f0[4], f2[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        f0[i] = w[i];
        f2[i] = __builtin_amdgcn_alignbyte(w[i + 1], w[i], 2);
      }
      __builtin_memcpy(&bv[0], f0, 16);
      __builtin_memcpy(&bv[2], f2, 16);
    } else {
      uint32_t d[2][4];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        __builtin_memcpy(&d[h][0], &fo[2 * h], 8);
        __builtin_memcpy(&d[h][2], &fo[2 * h + 1], 8);
      }
      uint32_t f0[4], f2[4];
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int i = 0; i < 2; ++i) {
          f0[2 * h + i] = d[h][i];
          f2[2 * h + i] = __builtin_amdgcn_alignbyte(d[h][i + 1], d[h][i], 2);
        }
      __builtin_memcpy(&bv[0], f0, 16);
      __builtin_memcpy(&bv[2], f2, 16);
    }
  };

  constexpr int KK = S::PIX / 16;
  i16x4 fa[2], fo[NBO], fe[NBE], fc[2];
  auto slice = [&](int i, const char* pa_, const char* pb_, const char* pc_, char* na, char* nb,
                   char* nc) {
    const bool more = i + 1 < cnt;
    if (more) copy_slice(j0 + i + 1, na, nb, nc);
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      bf16x8 av, bv[3], cv;
      prep_k(fa, fo, fe, av, bv);
      if (sc) {
        __builtin_memcpy(&cv, &fc[0], 8);
        __builtin_memcpy((char*)&cv + 8, &fc[1], 8);
      }
      __builtin_amdgcn_sched_barrier(0);
      i16x4 ga[2], go[NBO], ge[NBE], gc[2];
      if (kk + 1 < KK) read_k(pa_, pb_, pc_, kk + 1, ga, go, ge, gc);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int s = 0; s < 3; ++s) acc[s] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bv[s], av, acc[s], 0, 0, 0);
      if constexpr (PROJ)
        if (sc) acc[NACC - 1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bv[1], cv, acc[NACC - 1], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
      if (kk + 1 < KK) {
        fa[0] = ga[0];
        fa[1] = ga[1];
#pragma unroll
        for (int u = 0; u < NBO; ++u) fo[u] = go[u];
#pragma unroll
        for (int u = 0; u < NBE; ++u) fe[u] = ge[u];
        fc[0] = gc[0];
        fc[1] = gc[1];
      }
    }
    __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (more) read_k(na, nb, nc, 0, fa, fo, fe, fc);
  };
  if (cnt > 0) {
    copy_slice(j0, sA0, sB0, sC0);
    __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    read_k(sA0, sB0, sC0, 0, fa, fo, fe, fc);
  }
  for (int i = 0; i < cnt; i += 2) {
    slice(i, sA0, sB0, sC0, sA1, sB1, sC1);
    if (i + 1 < cnt) slice(i + 1, sA1, sB1, sC1, sA0, sB0, sC0);
  }

  // ---- epilogue as the stride-1 kernel; the projection's partial after
  // the 3x3 one
  const int co = k0 + wk * 32 + (lane & 31);
  float* out = (float*)p.out + (int64_t)by * p.split_stride;
#pragma unroll
  for (int s = 0; s < 3; ++s)
#pragma unroll
    for (int r4 = 0; r4 < 4; ++r4) {
      const int ci = c0 + wc * 32 + 8 * r4 + 4 * (lane >> 5);
      *(float4*)(out + ((int64_t)co * 9 + 3 * wr + s) * C + ci) =
          make_float4(acc[s][4 * r4], acc[s][4 * r4 + 1], acc[s][4 * r4 + 2], acc[s][4 * r4 + 3]);
    }
  if constexpr (PROJ) {
    if (sc) {
      float* out2 = out + (int64_t)9 * K * C;
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        const int ci = c0 + wc * 32 + 8 * r4 + 4 * (lane >> 5);
        *(float4*)(out2 + (int64_t)co * C + ci) =
            make_float4(acc[NACC - 1][4 * r4], acc[NACC - 1][4 * r4 + 1], acc[NACC - 1][4 * r4 + 2],
                        acc[NACC - 1][4 * r4 + 3]);
      }
    }
  }
}

bool wgrad3_ok(const GemmParams& p) {
  const ConvGeom& g = p.g;
  if (g.R != 3 || g.S != 3 || g.pad != 1 || g.C % 64 != 0 || g.K % 64 != 0) return false;
  if (g.stride == 2)   // output 16, 8 or 4 wide, input exactly twice that
    return g.Ho == g.Wo && (g.Wo == 16 || g.Wo == 8 || g.Wo == 4) && g.H == 2 * g.Ho &&
           g.W == 2 * g.Wo;
  if (g.stride != 1) return false;
  return g.H == g.W && (g.W == 32 || g.W == 16 || g.W == 8 || g.W == 4);
}

// slices of one worker segment of nimg images
int wgrad3_slices(const GemmParams& p, int nimg) {
  const int W = p.g.Wo, HW = W * W;
  const int pix = p.g.stride == 2 ? 64 : (W >= 16 ? 256 : 128);
  if (HW >= pix) return nimg * (HW / pix);
  return (nimg + pix / HW - 1) / (pix / HW);
}

// p: nseg / seg_split / seg_n0 / kt_per_split (slices per split) set by the
// caller, out = partial buffer with split_stride
hipError_t launch_wgrad3(const GemmParams& p, hipStream_t s) {
  if (!wgrad3_ok(p) || p.nseg < 1) return hipErrorInvalidValue;
  const dim3 grid((unsigned)((p.g.K / 64) * (p.g.C / 64)), (unsigned)p.seg_split[p.nseg]);
  if (p.g.stride == 2) {
    if (p.a2) {
      switch (p.g.Wo) {
        case 16: hipLaunchKernelGGL((wgrad3s2_kernel<16, true>), grid, dim3(768), 0, s, p); break;
        case 8: hipLaunchKernelGGL((wgrad3s2_kernel<8, true>), grid, dim3(768), 0, s, p); break;
        default: hipLaunchKernelGGL((wgrad3s2_kernel<4, true>), grid, dim3(768), 0, s, p); break;
      }
    } else {
      switch (p.g.Wo) {
        case 16: hipLaunchKernelGGL((wgrad3s2_kernel<16, false>), grid, dim3(768), 0, s, p); break;
        case 8: hipLaunchKernelGGL((wgrad3s2_kernel<8, false>), grid, dim3(768), 0, s, p); break;
        default: hipLaunchKernelGGL((wgrad3s2_kernel<4, false>), grid, dim3(768), 0, s, p); break;
      }
    }
    return hipGetLastError();
  }
  if (p.a2) return hipErrorInvalidValue;   // the projection is taken at stride 2 only
  switch (p.g.W) {
    case 32: hipLaunchKernelGGL(wgrad3_kernel<32>, grid, dim3(768), 0, s, p); break;
    case 16: hipLaunchKernelGGL(wgrad3_kernel<16>, grid, dim3(768), 0, s, p); break;
    case 8: hipLaunchKernelGGL(wgrad3_kernel<8>, grid, dim3(768), 0, s, p); break;
    default: hipLaunchKernelGGL(wgrad3_kernel<4>, grid, dim3(768), 0, s, p); break;
  }
  return hipGetLastError();
}

}  // namespace hs
