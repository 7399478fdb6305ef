// device_util.h -- device-side helpers shared by the stage kernels:
// element types and bf16 rounding, the workgroup -> (frame, tile, pixel
// block, channel block) decode with the XCD-aware renumbering, the GEMM row
// -> output pixel map, buffer-descriptor loads and the epilogue stores.
#pragma once

#include <hip/hip_runtime.h>

#include "kernel_args.h"

#ifdef MAFAT_TUNING
// Tuning builds only: start (k = 0) and end (k = 1) wall-clock stamps of
// every workgroup (the first 8192) of the last launch of a kernel family.
#define MAFAT_WG_TRACE_DECL(name_) __device__ long long name_[2][8192];
#define MAFAT_WG_MARK(name_, k_)                                            \
  do {                                                                      \
    if (threadIdx.x == 0 && blockIdx.x < 8192) name_[(k_)][blockIdx.x] = wall_clock64(); \
  } while (0)
#else
#define MAFAT_WG_TRACE_DECL(name_)
#define MAFAT_WG_MARK(name_, k_) do {} while (0)
#endif

namespace mafat {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
// Native 16-byte vector (HIP's uint4 is a struct; selects between structs
// compile to stack copies, so the kernels use this type for 16-byte data).
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

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
// logical blocks, which then share that XCD's L2: in pixel-block-major order
// an XCD owns a band of pixels (and streams all the weights), in
// channel-block-major order it owns a slice of the output channels (and
// streams all the input) -- the runtime picks the order with fewer
// compulsory L2 misses.
__device__ __forceinline__ int xcd_remap(int bid, int total) {
  constexpr int X = 8;
  const int per = total / X, rem = total % X;
  const int xcd = bid % X, slot = bid / X;
  return (xcd < rem) ? xcd * (per + 1) + slot : rem * (per + 1) + (xcd - rem) * per + slot;
}

struct BlockPos {
  int frame, tile, mb, nb;
};

// Block -> (frame, tile, pixel block, channel block), and the tile's
// geometry.  The per-tile tables are read with vector loads straight from
// the kernel argument segment, lane k reading entry k, issued before
// anything else so they arrive together with the scalar header fields (a
// dynamic index into the argument block would be a chain of dependent
// scalar loads).  The tile is then found with a ballot over the block
// prefix and its fields are taken with readlane.
//
// `early(nb)` runs once the channel block is known (it needs only the scalar
// header) and before the tile table is used: a kernel issues its first
// weight loads there, so their latency overlaps the table's.
struct NoEarly {
  __device__ void operator()(int) const {}
};
template <typename Early = NoEarly>
__device__ __forceinline__ BlockPos decode_block(const StageArgs& a, KTile* tile, Early early = Early{}) {
  static_assert(kMaxTilesPerLaunch == 64 && sizeof(KTile) == 28, "one tile per lane of a wave");
  const int lane = static_cast<int>(threadIdx.x) & 63;
  // (C-style cast: converts from the constant address space.)
  const StageArgs* ka = (const StageArgs*)__builtin_amdgcn_kernarg_segment_ptr();
  const int pre = ka->mblk_prefix[lane];
  const uint32_t* tw = reinterpret_cast<const uint32_t*>(&ka->tiles[lane]);
  uint32_t w[7];
#pragma unroll
  for (int k = 0; k < 7; ++k) w[k] = tw[k];

  int bid = xcd_remap(static_cast<int>(blockIdx.x), a.total_blocks);
  const int per_frame = a.mblk_total * a.nblk_n;
  BlockPos p;
  p.frame = bid / per_frame;
  const int blk = bid - p.frame * per_frame;
  // channel blocks then pixel blocks (or the other way round)
  int mg;
  if (a.chan_major) {
    p.nb = blk / a.mblk_total;
    mg = blk - p.nb * a.mblk_total;
  } else {
    mg = blk / a.nblk_n;
    p.nb = blk - mg * a.nblk_n;
  }
  early(p.nb);
  // Tiles whose first block is at or before mg, not counting tile 0.
  const int t = __popcll(__builtin_amdgcn_ballot_w64(lane >= 1 && lane < a.ntiles && pre <= mg));
  p.tile = t;
  p.mb = mg - __builtin_amdgcn_readlane(pre, t);
  uint32_t tw_t[7];
#pragma unroll
  for (int k = 0; k < 7; ++k) tw_t[k] = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(w[k]), t));
  __builtin_memcpy(tile, tw_t, sizeof(KTile));
  return p;
}

// Row reuse take-over copies carried by a launch (StageArgs::copy_*): a
// launch that carries copies has a second grid row (blockIdx.y = 1) of
// total_blocks workgroups, whose first copy_blocks copy 16 bytes per thread
// and step and the rest return at once; the first row computes as always,
// its test of blockIdx.y needing no memory access.  The copy table is read
// through the argument segment (a dynamic index into the by-value copy
// would go through private memory).
__device__ __forceinline__ void carried_copies() {
  const StageArgs* ka = (const StageArgs*)__builtin_amdgcn_kernarg_segment_ptr();
  const int cb = static_cast<int>(blockIdx.x);
  if (cb >= ka->copy_blocks) return;
  const int n = ka->ncopy;
  int64_t per_frame = 0;
  for (int k = 0; k < n; ++k) per_frame += ka->copy_bytes[k] >> 4;
  const int64_t total = per_frame * ka->copy_frames;
  const int64_t step = static_cast<int64_t>(ka->copy_blocks) * blockDim.x;
  for (int64_t u = static_cast<int64_t>(cb) * blockDim.x + threadIdx.x; u < total; u += step) {
    const int64_t f = u / per_frame;
    int64_t r = u - f * per_frame;
    int k = 0;
    while (k + 1 < n && r >= (ka->copy_bytes[k] >> 4)) {
      r -= ka->copy_bytes[k] >> 4;
      ++k;
    }
    unsigned char* fb = ka->copy_base + f * ka->copy_fstride;
    const u32x4 v = *reinterpret_cast<const u32x4*>(fb + ka->copy_src[k] + (r << 4));
    *reinterpret_cast<u32x4*>(fb + ka->copy_dst[k] + (r << 4)) = v;
  }
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
__device__ __forceinline__ void mma(f32x4& c, const u32x4& a, const u32x4& b);

template <>
__device__ __forceinline__ void mma<MAFAT_BF16>(f32x4& c, const u32x4& a, const u32x4& b) {
  c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                              __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// fp32: the 16-byte fragment of a lane holds 4 consecutive K elements; the
// four 16x16x4 MFMAs each take one of them.  A and B lanes use the same K
// assignment, so the sum runs over all 16 K elements of the chunk.
template <>
__device__ __forceinline__ void mma<MAFAT_F32>(f32x4& c, const u32x4& a, const u32x4& b) {
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), c, 0, 0, 0);
}

// 16-byte load through a buffer descriptor.  The hardware range check returns
// zero for a byte offset at or past the descriptor's size, which the matrix-core
// kernel uses for its zero padding: an operand that must read as
// zero gets bit 31 set in its offset (sizes stay below 2^31 bytes).
__device__ __forceinline__ u32x4 buf_load16(__amdgpu_buffer_rsrc_t r, unsigned off) {
  return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, static_cast<int>(off), 0, 0));
}
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, unsigned bytes) {
  // Word 3: 32-bit data format (required non-zero for untyped loads).
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, static_cast<int>(bytes), 0x00020000);
}

// Epilogue of the matrix-core kernels.  Two MFMA orientations:
//   - no pool: the weights are the A operand, so accumulator tile acc[j][i]
//     holds output channels (rows) x pixels (columns): lane l has channels
//     4*(l/16) .. +3 of column l % 16, i.e. 4 consecutive channels of one
//     pixel, which leave in one 8-byte (bf16) or 16-byte (fp32) store;
//   - fused 2x2 max-pool: the pixels are the A operand, quad-ordered (see
//     row_pixel), so the 4 accumulator rows a lane holds (rows 4*(l/16) ..
//     +3 of column l % 16) are one pool window of one channel.  The window
//     is reduced in the lane: scale and bias per pixel, the maximum, then
//     the activation -- which is non-decreasing, so applying it after the
//     maximum gives the same value as pooling activated outputs.
// Leaky ReLU(0.1) is max(v, 0.1 v); a linear layer uses slope 1.
__device__ __forceinline__ float act_slope(int act) { return act == MAFAT_ACT_LEAKY01 ? 0.1f : 1.f; }

template <int DT>
__device__ __forceinline__ void store4(float* p, const float (&v)[4]) {
  *reinterpret_cast<f32x4*>(p) = f32x4{v[0], v[1], v[2], v[3]};
}
template <int DT>
__device__ __forceinline__ void store4(uint16_t* p, const float (&v)[4]) {
  typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
  const bf16x4 h = {static_cast<__bf16>(v[0]), static_cast<__bf16>(v[1]), static_cast<__bf16>(v[2]),
                    static_cast<__bf16>(v[3])};  // round to nearest even
  *reinterpret_cast<uint2*>(p) = __builtin_bit_cast(uint2, h);
}
__device__ __forceinline__ void store1(float* p, float v) { *p = v; }
__device__ __forceinline__ void store1(uint16_t* p, float v) {
  *reinterpret_cast<__bf16*>(p) = static_cast<__bf16>(v);
}

}  // namespace
}  // namespace mafat
