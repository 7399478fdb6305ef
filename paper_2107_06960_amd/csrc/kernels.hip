// kernels.hip -- gfx950 kernels for one stage of a fused tile group.
//
// A stage is one convolution (3x3 or 1x1, stride 1, zero padding only
// outside the image), with folded batch-norm scale/bias and activation in
// its epilogue and, when the next layer of the group is a 2x2/2 max-pool,
// that pool too; or a lone max-pool.  One launch covers every tile of every
// frame of the stage: the grid enumerates (frame, tile, pixel block, channel
// block), and each tile reads only its own input region (halo included) and
// writes only its own output region.
//
//   conv_mfma_kernel    implicit GEMM on the matrix cores: M = the tile's
//                       output pixels, N = output channels, K = f*f*c_in.
//                       bf16: v_mfma_f32_16x16x32_bf16; fp32:
//                       v_mfma_f32_16x16x4_f32.  Operand tiles are staged
//                       global -> registers -> LDS (double buffered).
//   conv_direct_kernel  vector-ALU direct convolution for layers whose
//                       channel count does not fill a K chunk (the 3-channel
//                       first layer): one thread per output pixel (or per
//                       2x2 pool window), weights through the scalar cache.
//   pool_kernel         a max-pool stage that does not follow a convolution.
#include <hip/hip_runtime.h>

#include "kernel_args.h"

namespace mafat {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

template <int DT> struct Elt;
template <> struct Elt<MAFAT_F32> { using T = float; };
template <> struct Elt<MAFAT_BF16> { using T = uint16_t; };

__device__ __forceinline__ float to_f(float v) { return v; }
__device__ __forceinline__ float to_f(uint16_t h) {
  return __uint_as_float(static_cast<uint32_t>(h) << 16);
}

// float -> bfloat16, round to nearest, ties to even (NaN stays NaN).
__device__ __forceinline__ uint16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7f800000u) == 0x7f800000u)
    return static_cast<uint16_t>((u >> 16) | ((u & 0xffffu) ? 0x40u : 0u));
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}
__device__ __forceinline__ void put(float* p, float v) { *p = v; }
__device__ __forceinline__ void put(uint16_t* p, float v) { *p = f2bf(v); }

__device__ __forceinline__ float activate(float v, int act) {
  return (act == MAFAT_ACT_LEAKY01 && !(v > 0.f)) ? 0.1f * v : v;
}

// Workgroups are dispatched round-robin over the 8 XCDs (workgroup b runs
// on XCD b % 8).  Renumber so that each XCD gets one contiguous range of
// logical blocks: neighbouring pixel blocks of a tile (which share halo rows)
// and the channel blocks of one pixel block (which share the input rows)
// then hit the same L2.
__device__ __forceinline__ int xcd_remap(int bid, int total) {
  constexpr int X = 8;
  const int per = total / X, rem = total % X;
  const int xcd = bid % X, slot = bid / X;
  return (xcd < rem) ? xcd * (per + 1) + slot : rem * (per + 1) + (xcd - rem) * per + slot;
}

struct BlockPos {
  int frame, tile, mb, nb;
};

__device__ __forceinline__ BlockPos decode_block(const StageArgs& a) {
  int bid = xcd_remap(static_cast<int>(blockIdx.x), a.total_blocks);
  const int per_frame = a.mblk_total * a.nblk_n;
  BlockPos p;
  p.frame = bid / per_frame;
  bid -= p.frame * per_frame;
  const int mg = bid / a.nblk_n;
  p.nb = bid - mg * a.nblk_n;
  int t = 0;
  while (t + 1 < a.ntiles && a.mblk_prefix[t + 1] <= mg) ++t;
  p.tile = t;
  p.mb = mg - a.mblk_prefix[t];
  return p;
}

// Output pixel of row m of a tile's GEMM.  Without a fused pool the rows run
// over the computed rectangle in row-major order; with one, every 4
// consecutive rows are one 2x2 pool window (the rectangle has even origin and
// even extent), so the MFMA accumulator rows a lane holds are one window.
template <bool POOL>
__device__ __forceinline__ void row_pixel(const KTile& t, int m, int* oy, int* ox) {
  if (POOL) {
    const int pw = t.cw >> 1;
    const int q = m >> 2, s = m & 3;
    const int qy = q / pw, qx = q - qy * pw;
    *oy = t.cy0 + 2 * qy + (s >> 1);
    *ox = t.cx0 + 2 * qx + (s & 1);
  } else {
    const int yy = m / t.cw;
    *oy = t.cy0 + yy;
    *ox = t.cx0 + (m - yy * t.cw);
  }
}

template <int DT>
__device__ __forceinline__ void mma(f32x4& c, const uint4& a, const uint4& b);

template <>
__device__ __forceinline__ void mma<MAFAT_BF16>(f32x4& c, const uint4& a, const uint4& b) {
  c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                              __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// fp32: the 16-byte fragment of a lane holds 4 consecutive K elements; the
// four 16x16x4 MFMAs each take one of them.  A and B lanes use the same K
// assignment, so the sum runs over all 16 K elements of the chunk.
template <>
__device__ __forceinline__ void mma<MAFAT_F32>(f32x4& c, const uint4& a, const uint4& b) {
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), c, 0, 0, 0);
}

// Implicit-GEMM convolution, block tile BM pixels x BN channels, 4 waves in
// a 2x2 arrangement, K consumed in 64-byte chunks (32 bf16 or 16 fp32
// channels of one filter tap).  Requires c_in % (64 / sizeof(T)) == 0 and
// c_out % 16 == 0 (checked by the host).
template <int DT, int F, int BM, int BN, bool POOL>
__global__ __launch_bounds__(256) void conv_mfma_kernel(const StageArgs a) {
  using T = typename Elt<DT>::T;
  constexpr int P = (F - 1) / 2;
  constexpr int KC = 64 / static_cast<int>(sizeof(T));   // channels per K chunk
  constexpr int EPV = 16 / static_cast<int>(sizeof(T));  // channels per 16 bytes
  constexpr int ALD = BM / 64, BLD = BN / 64;            // staging loads per thread
  constexpr int WM = BM / 2, WN = BN / 2, MT = WM / 16, NT = WN / 16;
  constexpr int LROW = 5;  // uint4 per LDS row: 64 data bytes + 16 pad bytes
  __shared__ uint4 sA[2][BM * LROW];
  __shared__ uint4 sB[2][BN * LROW];

  const BlockPos bp = decode_block(a);
  const KTile tl = a.tiles[bp.tile];
  const int tid = static_cast<int>(threadIdx.x), lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int M = tl.ch * tl.cw;
  const int m0 = bp.mb * BM, n0 = bp.nb * BN;
  const int cin = a.cin, cout = a.cout;
  const T* src = static_cast<const T*>(a.src) + bp.frame * a.src_fstride + tl.src_off;
  T* dst = static_cast<T*>(a.dst) + bp.frame * a.dst_fstride + tl.dst_off;
  const T* wgt = static_cast<const T*>(a.w);
  const int K = F * F * cin;
  const int cblocks = cin / KC;
  const int ksteps = F * F * cblocks;
  const int chunk = tid & 3;

  int a_oy[ALD], a_ox[ALD];
  bool a_ok[ALD];
#pragma unroll
  for (int i = 0; i < ALD; ++i) {
    const int m = m0 + (tid >> 2) + 64 * i;
    a_ok[i] = m < M;
    row_pixel<POOL>(tl, a_ok[i] ? m : 0, &a_oy[i], &a_ox[i]);
  }
  const T* b_ptr[BLD];
  bool b_ok[BLD];
#pragma unroll
  for (int i = 0; i < BLD; ++i) {
    const int co = n0 + (tid >> 2) + 64 * i;
    b_ok[i] = co < cout;
    b_ptr[i] = wgt + static_cast<int64_t>(b_ok[i] ? co : 0) * K + chunk * EPV;
  }

  uint4 ra[ALD], rb[BLD];
  const uint4 zero = make_uint4(0, 0, 0, 0);
  auto gload = [&](int ks) {
    const int tap = ks / cblocks, cb = ks - tap * cblocks;
    const int ky = tap / F, kx = tap - ky * F;
    const int ci0 = cb * KC + chunk * EPV;
#pragma unroll
    for (int i = 0; i < ALD; ++i) {
      const int iy = a_oy[i] + ky - P, ix = a_ox[i] + kx - P;
      const bool ok = a_ok[i] && static_cast<unsigned>(iy) < static_cast<unsigned>(a.in_h) &&
                      static_cast<unsigned>(ix) < static_cast<unsigned>(a.in_w);
      ra[i] = ok ? *reinterpret_cast<const uint4*>(
                       src + ((iy - tl.sy0) * tl.sw + (ix - tl.sx0)) * cin + ci0)
                 : zero;
    }
#pragma unroll
    for (int i = 0; i < BLD; ++i)
      rb[i] = b_ok[i] ? *reinterpret_cast<const uint4*>(b_ptr[i] + tap * cin + cb * KC) : zero;
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < ALD; ++i) sA[buf][((tid >> 2) + 64 * i) * LROW + chunk] = ra[i];
#pragma unroll
    for (int i = 0; i < BLD; ++i) sB[buf][((tid >> 2) + 64 * i) * LROW + chunk] = rb[i];
  };

  f32x4 acc[MT][NT];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < NT; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  gload(0);
  lstore(0);
  __syncthreads();
  for (int ks = 0; ks < ksteps; ++ks) {
    const int cur = ks & 1;
    if (ks + 1 < ksteps) gload(ks + 1);
    uint4 af[MT], bf[NT];
#pragma unroll
    for (int i = 0; i < MT; ++i) af[i] = sA[cur][(wm * WM + i * 16 + (lane & 15)) * LROW + (lane >> 4)];
#pragma unroll
    for (int j = 0; j < NT; ++j) bf[j] = sB[cur][(wn * WN + j * 16 + (lane & 15)) * LROW + (lane >> 4)];
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int j = 0; j < NT; ++j) mma<DT>(acc[i][j], af[i], bf[j]);
    if (ks + 1 < ksteps) lstore(cur ^ 1);
    __syncthreads();
  }

  // Epilogue: lane holds rows 4*(lane/16) .. +3 of each 16x16 accumulator
  // tile, column lane % 16.
  const int rbase = (lane >> 4) * 4;
#pragma unroll
  for (int j = 0; j < NT; ++j) {
    const int co = n0 + wn * WN + j * 16 + (lane & 15);
    if (co >= cout) continue;
    const float s = a.scale[co], b = a.bias[co];
#pragma unroll
    for (int i = 0; i < MT; ++i) {
      const int mrow = m0 + wm * WM + i * 16 + rbase;
      if (mrow >= M) continue;
      float v[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) v[r] = activate(acc[i][j][r] * s + b, a.act);
      if (POOL) {
        const float mx = fmaxf(fmaxf(v[0], v[1]), fmaxf(v[2], v[3]));
        const int pw = tl.cw >> 1;
        const int q = mrow >> 2, qy = q / pw, qx = q - qy * pw;
        const int py = (tl.cy0 >> 1) + qy, px = (tl.cx0 >> 1) + qx;
        put(dst + ((py - tl.dy0) * tl.dw + (px - tl.dx0)) * cout + co, mx);
      } else {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int m = mrow + r;
          if (m < M) {
            int oy, ox;
            row_pixel<false>(tl, m, &oy, &ox);
            put(dst + ((oy - tl.dy0) * tl.dw + (ox - tl.dx0)) * cout + co, v[r]);
          }
        }
      }
    }
  }
}

// Direct convolution on the vector ALUs, one thread per output pixel (or per
// 2x2 pool window), all output channels in chunks of 8.  Weights are read
// with wave-uniform addresses (scalar cache).
template <int DT, int F, bool POOL>
__global__ __launch_bounds__(256) void conv_direct_kernel(const StageArgs a) {
  using T = typename Elt<DT>::T;
  constexpr int P = (F - 1) / 2;
  constexpr int NP = POOL ? 4 : 1;
  constexpr int CO = 8;
  const BlockPos bp = decode_block(a);
  const KTile tl = a.tiles[bp.tile];
  const int units = POOL ? (tl.ch >> 1) * (tl.cw >> 1) : tl.ch * tl.cw;
  const int u = bp.mb * 256 + static_cast<int>(threadIdx.x);
  if (u >= units) return;
  int oy[NP], ox[NP];
#pragma unroll
  for (int p = 0; p < NP; ++p) row_pixel<POOL>(tl, POOL ? 4 * u + p : u, &oy[p], &ox[p]);
  const int cin = a.cin, cout = a.cout, K = F * F * cin;
  const T* src = static_cast<const T*>(a.src) + bp.frame * a.src_fstride + tl.src_off;
  T* dst = static_cast<T*>(a.dst) + bp.frame * a.dst_fstride + tl.dst_off;
  const T* wgt = static_cast<const T*>(a.w);

  for (int co0 = 0; co0 < cout; co0 += CO) {
    const int nco = min(CO, cout - co0);
    float acc[NP][CO];
#pragma unroll
    for (int p = 0; p < NP; ++p)
#pragma unroll
      for (int j = 0; j < CO; ++j) acc[p][j] = 0.f;
#pragma unroll
    for (int ky = 0; ky < F; ++ky)
#pragma unroll
      for (int kx = 0; kx < F; ++kx) {
        const T* px[NP];
        bool ok[NP];
#pragma unroll
        for (int p = 0; p < NP; ++p) {
          const int iy = oy[p] + ky - P, ix = ox[p] + kx - P;
          ok[p] = static_cast<unsigned>(iy) < static_cast<unsigned>(a.in_h) &&
                  static_cast<unsigned>(ix) < static_cast<unsigned>(a.in_w);
          px[p] = ok[p] ? src + ((iy - tl.sy0) * tl.sw + (ix - tl.sx0)) * cin : src;
        }
        const T* wt = wgt + static_cast<int64_t>(co0) * K + (ky * F + kx) * cin;
        for (int ci = 0; ci < cin; ++ci) {
          float xv[NP];
#pragma unroll
          for (int p = 0; p < NP; ++p) xv[p] = ok[p] ? to_f(px[p][ci]) : 0.f;
#pragma unroll
          for (int j = 0; j < CO; ++j)
            if (j < nco) {
              const float wv = to_f(wt[static_cast<int64_t>(j) * K + ci]);
#pragma unroll
              for (int p = 0; p < NP; ++p) acc[p][j] += xv[p] * wv;
            }
        }
      }
#pragma unroll
    for (int j = 0; j < CO; ++j) {
      if (j >= nco) break;
      const int co = co0 + j;
      const float s = a.scale[co], b = a.bias[co];
      float v = activate(acc[0][j] * s + b, a.act);
#pragma unroll
      for (int p = 1; p < NP; ++p) v = fmaxf(v, activate(acc[p][j] * s + b, a.act));
      int yy = oy[0], xx = ox[0];
      if (POOL) { yy >>= 1; xx >>= 1; }
      put(dst + ((yy - tl.dy0) * tl.dw + (xx - tl.dx0)) * cout + co, v);
    }
  }
}

// Lone 2x2/2 max-pool: 64 output pixels per block, 4 threads per pixel
// striding over channels.  The computed rectangle is in pool-output
// coordinates.
template <int DT>
__global__ __launch_bounds__(256) void pool_kernel(const StageArgs a) {
  using T = typename Elt<DT>::T;
  const BlockPos bp = decode_block(a);
  const KTile tl = a.tiles[bp.tile];
  const int u = bp.mb * 64 + (static_cast<int>(threadIdx.x) >> 2);
  if (u >= tl.ch * tl.cw) return;
  const int yy = u / tl.cw;
  const int oy = tl.cy0 + yy, ox = tl.cx0 + (u - yy * tl.cw);
  const int c_in = a.cin;
  const T* src = static_cast<const T*>(a.src) + bp.frame * a.src_fstride + tl.src_off;
  T* dst = static_cast<T*>(a.dst) + bp.frame * a.dst_fstride + tl.dst_off;
  const T* p00 = src + ((2 * oy - tl.sy0) * tl.sw + (2 * ox - tl.sx0)) * c_in;
  const T* p10 = p00 + tl.sw * c_in;
  T* o = dst + ((oy - tl.dy0) * tl.dw + (ox - tl.dx0)) * c_in;
  for (int c = static_cast<int>(threadIdx.x) & 3; c < c_in; c += 4) {
    const float m = fmaxf(fmaxf(to_f(p00[c]), to_f(p00[c + c_in])),
                          fmaxf(to_f(p10[c]), to_f(p10[c + c_in])));
    put(o + c, m);
  }
}

template <int DT, int F, bool POOL>
hipError_t launch_conv(int kind, MfmaShape sh, const StageArgs& args, hipStream_t stream) {
  const dim3 grid(static_cast<unsigned>(args.total_blocks)), block(256);
  if (kind == K_CONV_DIRECT) {
    hipLaunchKernelGGL((conv_direct_kernel<DT, F, POOL>), grid, block, 0, stream, args);
  } else if (sh.bm == 64 && sh.bn == 64) {
    hipLaunchKernelGGL((conv_mfma_kernel<DT, F, 64, 64, POOL>), grid, block, 0, stream, args);
  } else if (sh.bm == 128 && sh.bn == 64) {
    hipLaunchKernelGGL((conv_mfma_kernel<DT, F, 128, 64, POOL>), grid, block, 0, stream, args);
  } else if (sh.bm == 64 && sh.bn == 128) {
    hipLaunchKernelGGL((conv_mfma_kernel<DT, F, 64, 128, POOL>), grid, block, 0, stream, args);
  } else if (sh.bm == 128 && sh.bn == 128) {
    hipLaunchKernelGGL((conv_mfma_kernel<DT, F, 128, 128, POOL>), grid, block, 0, stream, args);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <int DT>
hipError_t launch_dt(int kind, int f, bool pool, MfmaShape sh, const StageArgs& args,
                     hipStream_t stream) {
  if (kind == K_POOL) {
    hipLaunchKernelGGL((pool_kernel<DT>), dim3(static_cast<unsigned>(args.total_blocks)), dim3(256),
                       0, stream, args);
    return hipGetLastError();
  }
  if (f == 3) return pool ? launch_conv<DT, 3, true>(kind, sh, args, stream)
                          : launch_conv<DT, 3, false>(kind, sh, args, stream);
  if (f == 1) return pool ? launch_conv<DT, 1, true>(kind, sh, args, stream)
                          : launch_conv<DT, 1, false>(kind, sh, args, stream);
  return hipErrorInvalidValue;
}

}  // namespace

int block_units(int kind, MfmaShape shape) {
  if (kind == K_CONV_MFMA) return shape.bm;
  if (kind == K_CONV_DIRECT) return 256;
  return 64;
}

hipError_t launch_stage(int kind, int dtype, int f, bool pool, MfmaShape shape,
                        const StageArgs& args, hipStream_t stream) {
  if (args.total_blocks <= 0) return hipSuccess;
  if (dtype == MAFAT_BF16) return launch_dt<MAFAT_BF16>(kind, f, pool, shape, args, stream);
  if (dtype == MAFAT_F32) return launch_dt<MAFAT_F32>(kind, f, pool, shape, args, stream);
  return hipErrorInvalidValue;
}

}  // namespace mafat
