// Forward and data gradient of 64 -> 64 channel 3x3, stride-1, pad-1
// convolutions on 32-wide maps in bf16 (the widest layers of the CIFAR
// networks), 32x32x16 MFMA.
//
// A persistent block keeps the whole packed weight tensor in LDS (64 x 576
// bf16, 72 KB, [kq][tap][kh][n][8] as packed for the 32x32 kernel) and walks
// output tiles of 16 image rows x 32 columns (512 pixels).  Per tile it stages
// the input patch those pixels read -- 18 rows x 34 columns with the zero
// border, 64 channels, one 128-byte row per slot -- once, and applies the 9
// taps as shifted reads of it: the operand traffic from L2 drops about 9x
// against gathering every tap from global memory.  The next tile's patch is
// loaded into registers while the current tile computes.
//
// Wave w owns output rows 2w and 2w + 1 of the tile (two 32-pixel MFMA row
// blocks) and all 64 output channels.  Patch slots are XOR-swizzled by 16-byte
// chunk, chunk ^ ((slot >> 1) & 7), so 16 lanes reading 16 consecutive slots
// hit distinct banks.  The data gradient reads dy with the taps mirrored
// (slot offset 2 - r, 2 - s) and the transposed weights.  The epilogue stages
// each wave's 64 x 32 accumulator half-tiles in the patch area and writes
// whole rows.
//
// Block b takes the consecutive tiles [ntiles b / blocks, ntiles (b + 1) /
// blocks).  With stat_part set (forward), the epilogue also sums every stored
// output value and its square per channel, each lane over its own rows; when
// the next tile starts another worker segment (or the block's tiles end) the
// block adds its lanes in a fixed order through the patch area and writes one
// partial per channel for that segment: the batch-norm statistics of the
// output without a second pass over it.
#include "kernels.h"

namespace hs {

namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

enum { EPI_BIAS = 1, EPI_RELU = 2, EPI_ADD = 8, EPI_MASK = 16, EPI_MBITS = 32, EPI_STATS = 64 };

constexpr int P_W = 32;                     // map width
constexpr int P_ROWS = 16;                  // output rows per tile
constexpr int P_FW = P_W + 2, P_FR = P_ROWS + 2;
constexpr int P_SLOTS = P_FW * P_FR;        // 612
constexpr int P_CH = P_SLOTS * 8;           // 16-byte chunks per patch
constexpr int P_IT = (P_CH + 511) / 512;    // per thread
constexpr int W_CH = 4 * 9 * 2 * 64;        // 16-byte chunks of packed weights
constexpr int EROW = 36;                    // epilogue staging row stride (floats)

__device__ inline int pslot_off(int slot, int chunk) {
  return slot * 128 + ((chunk ^ ((slot >> 1) & 7)) << 4);
}

__device__ inline uint32_t pack2(float a, float b) {
  f32x2 v = {a, b};
  bf16x2 h = __builtin_convertvector(v, bf16x2);
  uint32_t u;
  __builtin_memcpy(&u, &h, 4);
  return u;
}

}  // namespace

template <int MODE, int EPI>
__global__ __launch_bounds__(512) void conv64_kernel(GemmParams p, int ntiles) {
  __shared__ __attribute__((aligned(16))) char smem[W_CH * 16 + P_SLOTS * 128];
  uint4* Wl = (uint4*)smem;
  char* Pl = smem + W_CH * 16;
  const ConvGeom& g = p.g;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int kh = lane >> 5, x = lane & 31;
  const int H = g.H;                        // map height (output = input size)
  const int tiles_per_img = H / P_ROWS;
  const bf16_t* A = (const bf16_t*)p.a;     // x (forward) or dy (data gradient), 64 channels

  for (int q = tid; q < W_CH; q += 512) Wl[q] = ((const uint4*)p.b)[q];

  // patch of tile t: slot (ry, cx) holds pixel (y0 - 1 + ry, cx - 1) of image b
  auto load_patch = [&](int t, uint4 (&r)[P_IT]) {
    const int b = t / tiles_per_img, y0 = (t - b * tiles_per_img) * P_ROWS;
#pragma unroll
    for (int i = 0; i < P_IT; ++i) {
      const int q = tid + 512 * i;
      r[i] = make_uint4(0, 0, 0, 0);
      if (q < P_CH) {
        const int slot = q >> 3, ch = q & 7;
        const int ry = slot / P_FW, cx = slot - ry * P_FW;
        const int y = y0 - 1 + ry, xx = cx - 1;
        if ((unsigned)y < (unsigned)H && (unsigned)xx < (unsigned)P_W)
          r[i] = *(const uint4*)(A + (((int64_t)b * H + y) * P_W + xx) * 64 + ch * 8);
      }
    }
  };
  auto store_patch = [&](const uint4 (&r)[P_IT]) {
#pragma unroll
    for (int i = 0; i < P_IT; ++i) {
      const int q = tid + 512 * i;
      if (q < P_CH) *(uint4*)(Pl + pslot_off(q >> 3, q & 7)) = r[i];
    }
  };

  // the block's tiles, and (statistics) the worker segment of a tile
  const int t_first = (int)((int64_t)ntiles * blockIdx.x / gridDim.x);
  const int t_last = (int)((int64_t)ntiles * (blockIdx.x + 1) / gridDim.x);
  constexpr bool ESTATS = (EPI & EPI_STATS) != 0;
  auto seg_of = [&](int tile) {
    const int img = tile / tiles_per_img;
    int sg = 0;
#pragma unroll
    for (int i = 1; i < MAX_SEG; ++i) sg += (i < p.nseg && img >= p.seg_n0[i]) ? 1 : 0;
    return sg;
  };
  // per lane: sums of y and y^2 over its rows, channels 32 nb + 8 (lane & 3) + e
  float st0[2][8], st1[2][8];
#pragma unroll
  for (int nb = 0; nb < 2; ++nb)
#pragma unroll
    for (int e = 0; e < 8; ++e) st0[nb][e] = st1[nb][e] = 0.f;
  // Adds the lanes' sums (called by every thread after a block barrier that
  // follows the last use of the patch area) and writes them as segment sg's
  // partial of this block; leaves the patch area free and the sums zero.
  auto flush = [&](int sg) {
    float* R = (float*)Pl;   // [wave][lane / 4][k][64 channels]
    const int j = lane >> 2, c8 = 8 * (lane & 3);
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
      for (int e = 0; e < 8; e += 4) {
        float* r0 = R + ((wave * 16 + j) * 2 + 0) * 64 + nb * 32 + c8 + e;
        float* r1 = R + ((wave * 16 + j) * 2 + 1) * 64 + nb * 32 + c8 + e;
        *(float4*)r0 = make_float4(st0[nb][e], st0[nb][e + 1], st0[nb][e + 2], st0[nb][e + 3]);
        *(float4*)r1 = make_float4(st1[nb][e], st1[nb][e + 1], st1[nb][e + 2], st1[nb][e + 3]);
        st0[nb][e] = st0[nb][e + 1] = st0[nb][e + 2] = st0[nb][e + 3] = 0.f;
        st1[nb][e] = st1[nb][e + 1] = st1[nb][e + 2] = st1[nb][e + 3] = 0.f;
      }
    __syncthreads();
    // four threads per (k, channel) add 32 of the 128 lane rows each, then
    // the first adds the four in order
    const int kc = tid & 127, part = tid >> 7;
    float ps = 0.f;
#pragma unroll 8
    for (int r = 0; r < 32; ++r) ps += R[((part * 32 + r) * 2 + (kc >> 6)) * 64 + (kc & 63)];
    float* Q = R + 128 * 2 * 64;   // [part][k * 64 + ch], after the lane rows
    Q[part * 128 + kc] = ps;
    __syncthreads();
    if (tid < 128)
      p.stat_part[((int64_t)(sg * (int)gridDim.x + (int)blockIdx.x) * 2 + (tid >> 6)) * 64 +
                  (tid & 63)] = ((Q[tid] + Q[128 + tid]) + Q[256 + tid]) + Q[384 + tid];
    __syncthreads();
  };

  int t = t_first;
  uint4 pre[P_IT];
  if (t < t_last) load_patch(t, pre);
  for (; t < t_last; ++t) {
    store_patch(pre);
    __syncthreads();
    if (t + 1 < t_last) load_patch(t + 1, pre);

    // Epilogue operands (addend, mask) of this tile.  A lane's rows of the
    // epilogue are fixed: row 16 i + lane / 4 of the wave's 64 (mb * 32 +
    // pixel), channels 8 (lane & 3) + 0..7 of each 32-channel half.  The
    // first half's are loaded now, while the taps run; the second half's when
    // the epilogue starts, while the first half is written.
    const int eb = t / tiles_per_img, ey0 = (t - eb * tiles_per_img) * P_ROWS;
    auto epi_off = [&](int nb, int i) -> int64_t {
      const int row = 16 * i + (lane >> 2), c8 = 8 * (lane & 3);
      const int y = ey0 + 2 * wave + (row >> 5), xx = row & 31;
      return (((int64_t)eb * H + y) * P_W + xx) * 64 + nb * 32 + c8;
    };
    constexpr bool EADD = (EPI & EPI_ADD) != 0, EMASK = (EPI & EPI_MASK) != 0;
    constexpr bool EBITS = (EPI & EPI_MBITS) != 0;   // the mask as bits: one byte per lane row
    uint4 add_pre[2][EADD ? 4 : 1], mask_pre[2][EMASK && !EBITS ? 4 : 1];
    uint32_t maskb[2][EBITS ? 4 : 1];
    auto load_epi = [&](int nb) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        if constexpr (EADD) add_pre[nb][i] = *(const uint4*)((const bf16_t*)p.addend + epi_off(nb, i));
        if constexpr (EBITS) maskb[nb][i] = p.mbits[epi_off(nb, i) >> 3];
        else if constexpr (EMASK) mask_pre[nb][i] = *(const uint4*)((const bf16_t*)p.mask + epi_off(nb, i));
      }
    };
    if constexpr (EADD || EMASK) load_epi(0);

    f32x16 acc[2][2];
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
      for (int nb = 0; nb < 2; ++nb) acc[mb][nb] = (f32x16){};
    // taps: forward reads slot (row + r, x + s); data gradient (row + 2 - r, x + 2 - s).
    // The fragments of the next k step (the next tap's first one after the
    // last) are read while the current step's MFMAs run; the scheduling
    // barriers keep the reads ahead of the MFMAs that hide them.  After the
    // last tap the "next" reads repeat tap 8 (in the patch, never used).
    auto read_frag = [&](int tap, int kq, uint4 (&fa)[2], uint4 (&fb)[2]) {
      const int r = tap / 3, s = tap - 3 * (tap / 3);
      const int dr = MODE == MODE_FWD ? r : 2 - r, ds = MODE == MODE_FWD ? s : 2 - s;
      const int slot0 = (2 * wave + dr) * P_FW + x + ds;
#pragma unroll
      for (int mb = 0; mb < 2; ++mb) fa[mb] = *(const uint4*)(Pl + pslot_off(slot0 + mb * P_FW, 2 * kq + kh));
#pragma unroll
      for (int nb = 0; nb < 2; ++nb) fb[nb] = Wl[((kq * 9 + tap) * 2 + kh) * 64 + nb * 32 + x];
    };
    uint4 fa[2], fb[2];
    read_frag(0, 0, fa, fb);
#pragma unroll 1
    for (int tap = 0; tap < 9; ++tap) {
      const int ntap = tap + 1 < 9 ? tap + 1 : 8;
#pragma unroll
      for (int kq = 0; kq < 4; ++kq) {
        uint4 na[2], nbv[2];
        if (kq < 3) read_frag(tap, kq + 1, na, nbv);
        else read_frag(ntap, 0, na, nbv);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int mb = 0; mb < 2; ++mb) {
          bf16x8 av;
          __builtin_memcpy(&av, &fa[mb], 16);
#pragma unroll
          for (int nb = 0; nb < 2; ++nb) {
            bf16x8 bv;
            __builtin_memcpy(&bv, &fb[nb], 16);
            acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bv, av, acc[mb][nb], 0, 0, 0);
          }
        }
        __builtin_amdgcn_sched_barrier(0);
        fa[0] = na[0];
        fa[1] = na[1];
        fb[0] = nbv[0];
        fb[1] = nbv[1];
      }
    }
    __syncthreads();   // patch area free: stage the epilogue there
    if constexpr (EADD || EMASK) load_epi(1);

    // ---- epilogue, one 32-channel half at a time: lane holds pixel x of
    // output row 2 wave + mb and channels 8 q + 4 kh + 0..3 of half nb
    float* E = (float*)Pl + wave * 64 * EROW;
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4)
          *(float4*)(E + (32 * mb + x) * EROW + 8 * q4 + 4 * kh) =
              make_float4(acc[mb][nb][4 * q4], acc[mb][nb][4 * q4 + 1], acc[mb][nb][4 * q4 + 2],
                          acc[mb][nb][4 * q4 + 3]);
      // a wave reads back only its own staging rows (its LDS operations run
      // in order): no block barrier between the halves
      __builtin_amdgcn_wave_barrier();
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = 16 * i + (lane >> 2), c8 = 8 * (lane & 3);   // row: mb * 32 + pixel
        const int64_t off = epi_off(nb, i);
        const float4 lo = *(const float4*)(E + row * EROW + c8);
        const float4 hi = *(const float4*)(E + row * EROW + c8 + 4);
        float v[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
        if constexpr ((EPI & EPI_BIAS) != 0) {
#pragma unroll
          for (int e = 0; e < 8; ++e) v[e] += p.bias[nb * 32 + c8 + e];
        }
        if constexpr ((EPI & EPI_ADD) != 0) {
          const uint4 u = add_pre[nb][i];
          const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            v[2 * e] += bf2f((bf16_t)(w[e] & 0xffffu));
            v[2 * e + 1] += bf2f((bf16_t)(w[e] >> 16));
          }
        }
        if constexpr ((EPI & EPI_RELU) != 0) {
#pragma unroll
          for (int e = 0; e < 8; ++e) v[e] = v[e] > 0.f ? v[e] : 0.f;
        }
        if constexpr (EBITS) {
          const uint32_t b = maskb[nb][i];
#pragma unroll
          for (int e = 0; e < 8; ++e)
            if (!((b >> e) & 1u)) v[e] = 0.f;
        } else if constexpr ((EPI & EPI_MASK) != 0) {
          const uint4 u = mask_pre[nb][i];
          const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            if (!(bf2f((bf16_t)(w[e] & 0xffffu)) > 0.f)) v[2 * e] = 0.f;
            if (!(bf2f((bf16_t)(w[e] >> 16)) > 0.f)) v[2 * e + 1] = 0.f;
          }
        }
        const uint4 o = make_uint4(pack2(v[0], v[1]), pack2(v[2], v[3]), pack2(v[4], v[5]), pack2(v[6], v[7]));
        *(uint4*)((bf16_t*)p.out + off) = o;
        if constexpr (ESTATS) {   // the stored values, widened back from bf16
          const uint32_t w[4] = {o.x, o.y, o.z, o.w};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float lo = __uint_as_float(w[e] << 16), hi = __uint_as_float(w[e] & 0xffff0000u);
            st0[nb][2 * e] += lo;
            st1[nb][2 * e] += lo * lo;
            st0[nb][2 * e + 1] += hi;
            st1[nb][2 * e + 1] += hi * hi;
          }
        }
      }
      __builtin_amdgcn_wave_barrier();
    }
    __syncthreads();   // every wave is done with the patch area: the next tile's patch goes there
    if constexpr (ESTATS) {
      const int sg = seg_of(t);
      if (t + 1 == t_last || seg_of(t + 1) != sg) flush(sg);
    }
  }
  if constexpr (ESTATS) {
    // segments without rows in this block: zero partials
    const int s_lo = t_first < t_last ? seg_of(t_first) : p.nseg;
    const int s_hi = t_first < t_last ? seg_of(t_last - 1) : -1;
    if (tid < 128)
      for (int sg = 0; sg < p.nseg; ++sg)
        if (sg < s_lo || sg > s_hi)
          p.stat_part[((int64_t)(sg * (int)gridDim.x + (int)blockIdx.x) * 2 + (tid >> 6)) * 64 +
                      (tid & 63)] = 0.f;
  }
}

bool conv64_ok(int mode, const GemmParams& p) {
  const ConvGeom& g = p.g;
  if (p.par || p.out_f32 || (mode != MODE_FWD && mode != MODE_DGRAD)) return false;
  return g.R == 3 && g.S == 3 && g.stride == 1 && g.pad == 1 && g.C == 64 && g.K == 64 &&
         g.W == P_W && g.H % P_ROWS == 0 && g.H == g.Ho && g.W == g.Wo;
}

template <int MODE>
static void launch64(const GemmParams& p, int ntiles, dim3 grid, hipStream_t s) {
  if constexpr (MODE == MODE_FWD) {
    const bool bias = p.bias != nullptr, relu = p.relu != 0;
    if (p.stat_part)   // a plain convolution (launch_conv64 rejects bias or ReLU with sums)
      hipLaunchKernelGGL((conv64_kernel<MODE, EPI_STATS>), grid, dim3(512), 0, s, p, ntiles);
    else if (bias && relu) hipLaunchKernelGGL((conv64_kernel<MODE, EPI_BIAS | EPI_RELU>), grid, dim3(512), 0, s, p, ntiles);
    else if (bias) hipLaunchKernelGGL((conv64_kernel<MODE, EPI_BIAS>), grid, dim3(512), 0, s, p, ntiles);
    else if (relu) hipLaunchKernelGGL((conv64_kernel<MODE, EPI_RELU>), grid, dim3(512), 0, s, p, ntiles);
    else hipLaunchKernelGGL((conv64_kernel<MODE, 0>), grid, dim3(512), 0, s, p, ntiles);
  } else {
    const bool add = p.addend != nullptr, mask = p.mask != nullptr || p.mbits != nullptr;
    if (add && p.mbits) hipLaunchKernelGGL((conv64_kernel<MODE, EPI_ADD | EPI_MASK | EPI_MBITS>), grid, dim3(512), 0, s, p, ntiles);
    else if (p.mbits) hipLaunchKernelGGL((conv64_kernel<MODE, EPI_MASK | EPI_MBITS>), grid, dim3(512), 0, s, p, ntiles);
    else if (add && mask) hipLaunchKernelGGL((conv64_kernel<MODE, EPI_ADD | EPI_MASK>), grid, dim3(512), 0, s, p, ntiles);
    else if (add) hipLaunchKernelGGL((conv64_kernel<MODE, EPI_ADD>), grid, dim3(512), 0, s, p, ntiles);
    else if (mask) hipLaunchKernelGGL((conv64_kernel<MODE, EPI_MASK>), grid, dim3(512), 0, s, p, ntiles);
    else hipLaunchKernelGGL((conv64_kernel<MODE, 0>), grid, dim3(512), 0, s, p, ntiles);
  }
}

int conv64_blocks(const GemmParams& p) {
  const int ntiles = p.g.n * (p.g.H / P_ROWS);
  int dev = 0, cus = 256;
  if (hipGetDevice(&dev) == hipSuccess)
    (void)hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  return ntiles < cus ? ntiles : cus;
}

// p.b: packed weights (launch_pack_weights for the same mode); one block per CU
hipError_t launch_conv64(int mode, const GemmParams& p, hipStream_t s) {
  if (!conv64_ok(mode, p)) return hipErrorInvalidValue;
  const int ntiles = p.g.n * (p.g.H / P_ROWS);
  if (p.stat_part) {
    // forward sums of a plain convolution over whole-sample segments
    if (mode != MODE_FWD || p.bias || p.relu || p.nseg < 1 || p.nseg > MAX_SEG ||
        p.seg_n0[0] != 0 || p.seg_n0[p.nseg] != p.g.n)
      return hipErrorInvalidValue;
    for (int i = 0; i < p.nseg; ++i)
      if (p.seg_n0[i + 1] <= p.seg_n0[i]) return hipErrorInvalidValue;
  }
  const dim3 grid((unsigned)conv64_blocks(p));
  if (mode == MODE_FWD) launch64<MODE_FWD>(p, ntiles, grid, s);
  else launch64<MODE_DGRAD>(p, ntiles, grid, s);
  return hipGetLastError();
}

}  // namespace hs
