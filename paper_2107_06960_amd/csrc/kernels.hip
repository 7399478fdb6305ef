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
//   conv_rgb_kernel     the 3-channel first layer on the vector ALUs
//                       (bf16: packed dot products), patch in registers.
//   pool_kernel         a max-pool stage that does not follow a convolution.
#include <hip/hip_runtime.h>

#include "kernel_args.h"

namespace mafat {
#ifdef MAFAT_TUNING
// Tuning builds only: phase timestamps of a few workgroups.
__device__ long long g_trace[4][64];
#define MAFAT_TRACE(slot_)                                                                     \
  do {                                                                                         \
    if (threadIdx.x == 0 && (blockIdx.x == 0 || blockIdx.x == gridDim.x - 1 ||                 \
                             blockIdx.x == gridDim.x / 2) && (slot_) < 64)                     \
      g_trace[blockIdx.x == 0 ? 0 : (blockIdx.x == gridDim.x - 1 ? 1 : 2)][(slot_)] = wall_clock64(); \
  } while (0)
#else
#define MAFAT_TRACE(slot_) do {} while (0)
#endif
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
__device__ __forceinline__ BlockPos decode_block(const StageArgs& a, KTile* tile) {
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
  MAFAT_TRACE(60 + (bid < 0 ? 1 : 0));
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
  MAFAT_TRACE(61 + (mg < 0 ? 1 : 0));
  // Tiles whose first block is at or before mg, not counting tile 0.
  const int t = __popcll(__builtin_amdgcn_ballot_w64(lane >= 1 && lane < a.ntiles && pre <= mg));
  p.tile = t;
  p.mb = mg - __builtin_amdgcn_readlane(pre, t);
  uint32_t tw_t[7];
#pragma unroll
  for (int k = 0; k < 7; ++k) tw_t[k] = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(w[k]), t));
  __builtin_memcpy(tile, tw_t, sizeof(KTile));
  MAFAT_TRACE(62 + (t < 0 ? 1 : 0));
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

// Epilogue of the matrix-core kernels for a BM x BN block computed by 4
// waves in a 2x2 arrangement: scale, bias, activation, the optional 2x2 max
// (the 4 accumulator rows a lane holds are one pool window), rounding to the
// output type; the block is then transposed through LDS (`smem`, at least
// OROWS * (BN * sizeof(T) + 16) bytes, free for use) and written with
// 16-byte stores along channels.  Lane l holds rows 4*(l/16) .. +3 of each
// 16x16 accumulator tile, column l % 16.
template <int DT, int BM, int BN, bool POOL>
__device__ __forceinline__ void store_block(const f32x4 (&acc)[BM / 32][BN / 32],
                                            unsigned char* smem, const StageArgs& a,
                                            const KTile& tl, int m0, int n0,
                                            typename Elt<DT>::T* dst) {
  using T = typename Elt<DT>::T;
  constexpr int EPV = 16 / static_cast<int>(sizeof(T));
  constexpr int WM = BM / 2, WN = BN / 2, MT = WM / 16, NT = WN / 16;
  constexpr int OROWS = POOL ? BM / 4 : BM;
  constexpr int OSTRIDE = (BN * static_cast<int>(sizeof(T)) + 16) / static_cast<int>(sizeof(T));
  const int tid = static_cast<int>(threadIdx.x), lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int M = tl.ch * tl.cw, cout = a.cout;
  T* sO = reinterpret_cast<T*>(smem);
  const int rq = (lane >> 4) * 4;
#pragma unroll
  for (int j = 0; j < NT; ++j) {
    const int cl = wn * WN + j * 16 + (lane & 15);
    const int co = n0 + cl;
    const float s = co < cout ? a.scale[co] : 0.f, b = co < cout ? a.bias[co] : 0.f;
#pragma unroll
    for (int i = 0; i < MT; ++i) {
      const int ml = wm * WM + i * 16 + rq;
      float v[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) v[r] = activate(acc[i][j][r] * s + b, a.act);
      if (POOL) {
        const float mx = fmaxf(fmaxf(v[0], v[1]), fmaxf(v[2], v[3]));
        put(sO + (ml >> 2) * OSTRIDE + cl, mx);
      } else {
#pragma unroll
        for (int r = 0; r < 4; ++r) put(sO + (ml + r) * OSTRIDE + cl, v[r]);
      }
    }
  }
  __syncthreads();
  constexpr int CPR = BN / EPV;  // 16-byte pieces per output row
  const int pw = tl.cw >> 1;
  for (int c = tid; c < OROWS * CPR; c += 256) {
    const int row = c / CPR, piece = c - row * CPR;
    const int m = m0 + (POOL ? 4 * row : row);
    const int co = n0 + piece * EPV;
    if (m >= M || co >= cout) continue;
    int oy, ox;
    if (POOL) {
      const int qq = m >> 2, qy = qq / pw;
      oy = (tl.cy0 >> 1) + qy;
      ox = (tl.cx0 >> 1) + (qq - qy * pw);
    } else {
      row_pixel<false>(tl, m, &oy, &ox);
    }
    *reinterpret_cast<u32x4*>(dst + ((oy - tl.dy0) * tl.dw + (ox - tl.dx0)) * cout + co) =
        *reinterpret_cast<const u32x4*>(sO + row * OSTRIDE + piece * EPV);
  }
}

// Implicit-GEMM convolution, block tile BM pixels x BN channels, 4 waves in
// a 2x2 arrangement (wave tile BM/2 x BN/2 of 16x16 accumulator tiles).
//
// K runs over (tap, channel) in 64-byte sub-chunks (32 bf16 or 16 fp32
// channels of one filter tap); a pipeline stage holds two sub-chunks
// (128 bytes of every A and B row).  Each thread issues its 16-byte loads for
// stage s+DEPTH while the waves run the MFMAs of stage s from LDS, so DEPTH
// stages are in flight per workgroup; LDS is double buffered with one
// barrier per stage.  Rows are padded to 144 bytes so the 16-lane fragment
// reads of consecutive rows hit distinct banks.
//
// Operands are read through buffer descriptors with 32-bit byte offsets:
// the zero padding of the convolution (taps outside the image), padded
// sub-chunks past the last tap and weight rows past c_out all read as zero
// through the descriptor's range check, so the loop has no masking work.
//
// Epilogue: see store_block.
//
// Requires c_in % (64 / sizeof(T)) == 0, c_out % 16 == 0 and byte offsets
// below 2^31 within a frame's source buffer and the weights (host-checked).
template <int DT, int F, int BM, int BN, bool POOL, int DEPTH>
__global__ __launch_bounds__(256) void conv_mfma_kernel(const StageArgs a) {
  using T = typename Elt<DT>::T;
  constexpr int ESZ = static_cast<int>(sizeof(T));
  constexpr int P = (F - 1) / 2;
  constexpr int KC = 64 / ESZ;   // channels per sub-chunk
  constexpr int EPV = 16 / ESZ;  // channels per 16 bytes
  constexpr int ROWQ = 9;        // u32x4 per LDS row
  constexpr int ALD = BM / 32, BLD = BN / 32;  // loads per thread per stage
  constexpr int WM = BM / 2, WN = BN / 2, MT = WM / 16, NT = WN / 16;
  static_assert(DEPTH >= 3 && DEPTH <= 6, "pipeline depth");
  static_assert(F * F + 2 * DEPTH + 2 < 32, "tap mask width (taps of computed stages)");
  constexpr int NBUF = 2;  // LDS stage buffers
  constexpr int OPND_BYTES = NBUF * (BM + BN) * ROWQ * 16;
  constexpr int OROWS = POOL ? BM / 4 : BM;
  constexpr int OUT_BYTES = OROWS * (BN * ESZ + 16);
  constexpr int SMEM = OPND_BYTES > OUT_BYTES ? OPND_BYTES : OUT_BYTES;
  __shared__ __align__(16) unsigned char smem[SMEM];
  u32x4* sA = reinterpret_cast<u32x4*>(smem);  // [NBUF][BM][ROWQ]
  u32x4* sB = sA + NBUF * BM * ROWQ;           // [NBUF][BN][ROWQ]

  MAFAT_TRACE(0);
  KTile tl;
  const BlockPos bp = decode_block(a, &tl);
  const int tid = static_cast<int>(threadIdx.x), lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  MAFAT_TRACE(4 + (tl.ch > 30000 ? 1 : 0));
  const int M = tl.ch * tl.cw;
  const int m0 = bp.mb * BM, n0 = bp.nb * BN;
  const int cin = a.cin, cout = a.cout, sw = tl.sw;
  const int64_t sbase = bp.frame * a.src_fstride + tl.src_off;
  T* dst = static_cast<T*>(a.dst) + bp.frame * a.dst_fstride + tl.dst_off;
  const int K = F * F * cin;
  const int cblocks = cin / KC;
  const int nsub = F * F * cblocks;    // 64-byte sub-chunks along K
  const int nstage = (nsub + 1) >> 1;  // 128-byte stages
  const __amdgpu_buffer_rsrc_t rsa =
      make_rsrc(static_cast<const T*>(a.src) + sbase, static_cast<unsigned>((a.src_fstride - tl.src_off) * ESZ));
  const __amdgpu_buffer_rsrc_t rsb = make_rsrc(a.w, static_cast<unsigned>(cout * K * ESZ));

  // This thread stages rows r0 + 32 i, 16-byte piece `pc` of sub-chunk `hh`
  // of every stage.  Per A row: the byte offset of its pixel in the source
  // buffer and a mask of the filter taps that read zero (outside the image;
  // bits past the last tap are set, so padded sub-chunks read zero).  Loads
  // that must read zero get bit 31 set in their offset.
  const int r0 = tid >> 3, q = tid & 7, hh = q >> 2, pc = q & 3;
  unsigned a_off[ALD], a_inv[ALD], b_off[BLD];
#pragma unroll
  for (int i = 0; i < ALD; ++i) {
    const int m = m0 + r0 + 32 * i;
    int oy, ox;
    row_pixel<POOL>(tl, m < M ? m : 0, &oy, &ox);
    a_off[i] = static_cast<unsigned>((((oy - tl.sy0) * sw + (ox - tl.sx0)) * cin + pc * EPV) * ESZ);
    unsigned inv = ~0u << (F * F);
#pragma unroll
    for (int t = 0; t < F * F; ++t) {
      const int iy = oy + t / F - P, ix = ox + t % F - P;
      const bool in = static_cast<unsigned>(iy) < static_cast<unsigned>(a.in_h) &&
                      static_cast<unsigned>(ix) < static_cast<unsigned>(a.in_w);
      inv |= in ? 0u : (1u << t);
    }
    a_inv[i] = (m < M) ? inv : ~0u;
  }
#pragma unroll
  for (int i = 0; i < BLD; ++i) {
    const int co = n0 + r0 + 32 * i;
    b_off[i] = co < cout ? static_cast<unsigned>((co * K + pc * EPV) * ESZ) : 0x80000000u;
  }

  u32x4 ra[DEPTH][ALD], rb[DEPTH][BLD];
  // Load cursor (uniform): filter tap and channel block of the first
  // sub-chunk of the next stage to load, advanced by two sub-chunks per load
  // (readfirstlane keeps its arithmetic on the scalar unit).  Padded
  // sub-chunks (tap past the last) re-read the last tap's weights, which
  // meet zero A rows.
  int lc_tap = 0, lc_cb = 0;
#define MAFAT_GLOAD(d_)                                                                        \
  do {                                                                                         \
    const int tap0_ = __builtin_amdgcn_readfirstlane(lc_tap);                                  \
    const int cb0_ = __builtin_amdgcn_readfirstlane(lc_cb);                                    \
    const int w0_ = (cblocks - 2 - cb0_) >> 31; /* -1: the next sub-chunk starts a new tap */  \
    const int tap1_ = tap0_ - w0_, cb1_ = (cb0_ + 1) & ~w0_;                                   \
    const int w1_ = (cblocks - 2 - cb1_) >> 31;                                                \
    const int ky0_ = tap0_ / F, kx0_ = tap0_ - ky0_ * F;                                       \
    const int ky1_ = tap1_ / F, kx1_ = tap1_ - ky1_ * F;                                       \
    const int ao0_ = (((ky0_ - P) * sw + (kx0_ - P)) * cin + cb0_ * KC) * ESZ;                 \
    const int ao1_ = (((ky1_ - P) * sw + (kx1_ - P)) * cin + cb1_ * KC) * ESZ;                 \
    const int bo0_ = (min(tap0_, F * F - 1) * cin + cb0_ * KC) * ESZ;                          \
    const int bo1_ = (min(tap1_, F * F - 1) * cin + cb1_ * KC) * ESZ;                          \
    const int t0c_ = min(tap0_, 31), t1c_ = min(tap1_, 31);                                    \
    const unsigned tap_ = static_cast<unsigned>(hh ? t1c_ : t0c_);                             \
    const unsigned aoff_ = static_cast<unsigned>(hh ? ao1_ : ao0_);                            \
    const unsigned boff_ = static_cast<unsigned>(hh ? bo1_ : bo0_);                            \
    _Pragma("unroll") for (int i = 0; i < ALD; ++i) {                                          \
      const unsigned bad_ = (a_inv[i] >> tap_) & 1u;                                           \
      ra[d_][i] = buf_load16(rsa, (a_off[i] + aoff_) | (bad_ << 31));                         \
    }                                                                                          \
    _Pragma("unroll") for (int i = 0; i < BLD; ++i) rb[d_][i] = buf_load16(rsb, b_off[i] + boff_); \
    lc_tap = tap1_ - w1_;                                                                      \
    lc_cb = (cb1_ + 1) & ~w1_;                                                                 \
  } while (0)
  // Registers (set d_) -> LDS buffer buf_.
#define MAFAT_LSTORE(d_, buf_)                                                                 \
  do {                                                                                         \
    _Pragma("unroll") for (int i = 0; i < ALD; ++i)                                            \
      sA[((buf_) * BM + r0 + 32 * i) * ROWQ + q] = ra[d_][i];                                  \
    _Pragma("unroll") for (int i = 0; i < BLD; ++i)                                            \
      sB[((buf_) * BN + r0 + 32 * i) * ROWQ + q] = rb[d_][i];                                  \
  } while (0)

  f32x4 acc[MT][NT];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < NT; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  // Pipeline, per step st (computing stage st from LDS buffer st % 2):
  //   barrier (stage st is in LDS; every wave is done reading stage st - 1);
  //   read both K-halves' fragments of stage st; issue the global loads of
  //   stage st + DEPTH into the register set stage st came from; MFMAs;
  //   write stage st + 1 (loaded DEPTH - 1 steps ago) to the other buffer.
  // The stage count is padded to a multiple of DEPTH so the loop body has no
  // branches (padded stages read zero A rows).
  const int nst_pad = (nstage + DEPTH - 1) / DEPTH * DEPTH;
  MAFAT_TRACE(5);
  MAFAT_GLOAD(0);
  MAFAT_GLOAD(1);
  MAFAT_GLOAD(2);
  if constexpr (DEPTH >= 4) MAFAT_GLOAD(3);
  if constexpr (DEPTH >= 5) MAFAT_GLOAD(4);
  if constexpr (DEPTH >= 6) MAFAT_GLOAD(5);
  MAFAT_TRACE(6);
  MAFAT_LSTORE(0, 0);
  MAFAT_TRACE(7);
  int rbuf = 0;   // LDS buffer holding stage st
#define MAFAT_STEP(d_, dn_)                                                                      \
  do {                                                                                           \
    __syncthreads();                                                                             \
    u32x4 af[2][MT], bfr[2][NT];                                                                 \
    _Pragma("unroll") for (int h = 0; h < 2; ++h) {                                              \
      _Pragma("unroll") for (int i = 0; i < MT; ++i)                                             \
        af[h][i] = sA[(rbuf * BM + wm * WM + i * 16 + (lane & 15)) * ROWQ + h * 4 + (lane >> 4)]; \
      _Pragma("unroll") for (int j = 0; j < NT; ++j)                                             \
        bfr[h][j] = sB[(rbuf * BN + wn * WN + j * 16 + (lane & 15)) * ROWQ + h * 4 + (lane >> 4)]; \
    }                                                                                            \
    MAFAT_GLOAD(d_);                                                                             \
    _Pragma("unroll") for (int h = 0; h < 2; ++h)                                                \
      _Pragma("unroll") for (int i = 0; i < MT; ++i)                                             \
        _Pragma("unroll") for (int j = 0; j < NT; ++j) mma<DT>(acc[i][j], af[h][i], bfr[h][j]);  \
    rbuf ^= 1;                                                                                   \
    MAFAT_LSTORE(dn_, rbuf);                                                                     \
    MAFAT_TRACE(8 + s0 + (d_));                                                                  \
  } while (0)
  for (int s0 = 0; s0 < nst_pad; s0 += DEPTH) {
    if constexpr (DEPTH == 3) {
      MAFAT_STEP(0, 1); MAFAT_STEP(1, 2); MAFAT_STEP(2, 0);
    } else if constexpr (DEPTH == 4) {
      MAFAT_STEP(0, 1); MAFAT_STEP(1, 2); MAFAT_STEP(2, 3); MAFAT_STEP(3, 0);
    } else if constexpr (DEPTH == 5) {
      MAFAT_STEP(0, 1); MAFAT_STEP(1, 2); MAFAT_STEP(2, 3); MAFAT_STEP(3, 4); MAFAT_STEP(4, 0);
    } else {
      MAFAT_STEP(0, 1); MAFAT_STEP(1, 2); MAFAT_STEP(2, 3); MAFAT_STEP(3, 4); MAFAT_STEP(4, 5);
      MAFAT_STEP(5, 0);
    }
  }
  MAFAT_TRACE(1);
  __syncthreads();
#undef MAFAT_STEP
#undef MAFAT_GLOAD
#undef MAFAT_LSTORE

  MAFAT_TRACE(2);
  store_block<DT, BM, BN, POOL>(acc, smem, a, tl, m0, n0, dst);
  MAFAT_TRACE(3);
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
  KTile tl;
  const BlockPos bp = decode_block(a, &tl);
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

// First layer of an image network: 3 input channels, 3x3 filter.  A K of 27
// does not fill the matrix cores' K chunk, so this runs on the vector ALUs.
// A thread owns one output pixel (or one 2x2 pool window) and one group of 8
// output channels: its (Q+2)x(Q+2)x3 input patch is loaded into registers
// (neighbouring threads of the same pixel hit the same cache lines), the
// weights of its 8 channels are broadcast from LDS, and its result leaves in
// one 16-byte store (the channel groups of a pixel are adjacent threads, so
// the stores of a pixel are contiguous).  bf16 uses the packed dot product
// v_dot2_f32_bf16 on channel pairs (c0,c1) and (c2,0): two multiply-adds per
// instruction with float32 accumulation.
// Requires c_out in {8, 16, 32, 64} (checked by the host).
template <int DT, bool POOL>
__global__ __launch_bounds__(256) 
void conv_rgb_kernel(const StageArgs a) {
  using T = typename Elt<DT>::T;
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  constexpr int Q = POOL ? 2 : 1;   // output pixels per thread along each axis
  constexpr int PR = Q + 2;         // input patch extent
  constexpr int CO = 8;
  constexpr int NJ = (DT == MAFAT_BF16) ? 2 : 3;  // weight words per tap
  __shared__ __align__(16) uint32_t wl[9 * 3 * 64];
  const int cout = a.cout;
  const int cg_n = cout / CO;                     // channel groups per pixel
  const T* wgt = static_cast<const T*>(a.w);
  // LDS weights, [tap][j][co]: bf16 j=0 holds (w_c0, w_c1), j=1 (w_c2, 0);
  // fp32 j is the input channel.
  for (int i = static_cast<int>(threadIdx.x); i < 9 * NJ * cout; i += 256) {
    const int co = i % cout, rest = i / cout, j = rest % NJ, tap = rest / NJ;
    const T* wr = wgt + co * 27 + tap * 3;
    if constexpr (DT == MAFAT_BF16) {
      wl[i] = (j == 0) ? (static_cast<uint32_t>(wr[0]) | (static_cast<uint32_t>(wr[1]) << 16))
                       : static_cast<uint32_t>(wr[2]);
    } else {
      wl[i] = __float_as_uint(to_f(wr[j]));
    }
  }
  __syncthreads();

  KTile tl;
  const BlockPos bp = decode_block(a, &tl);
  const int units = POOL ? (tl.ch >> 1) * (tl.cw >> 1) : tl.ch * tl.cw;
  const int per_block = 256 / cg_n;
  const int u = bp.mb * per_block + static_cast<int>(threadIdx.x) / cg_n;
  const int co0 = (static_cast<int>(threadIdx.x) % cg_n) * CO;
  if (u >= units) return;
  int oy0, ox0;
  if (POOL) {
    const int pw = tl.cw >> 1, qy = u / pw;
    oy0 = tl.cy0 + 2 * qy;
    ox0 = tl.cx0 + 2 * (u - qy * pw);
  } else {
    const int yy = u / tl.cw;
    oy0 = tl.cy0 + yy;
    ox0 = tl.cx0 + (u - yy * tl.cw);
  }
  const T* src = static_cast<const T*>(a.src) + bp.frame * a.src_fstride + tl.src_off;
  T* dst = static_cast<T*>(a.dst) + bp.frame * a.dst_fstride + tl.dst_off;

  // input patch, zero outside the image
  uint32_t pin[PR][PR][NJ];
#pragma unroll
  for (int r = 0; r < PR; ++r)
#pragma unroll
    for (int c = 0; c < PR; ++c) {
      const int iy = oy0 - 1 + r, ix = ox0 - 1 + c;
      const bool ok = static_cast<unsigned>(iy) < static_cast<unsigned>(a.in_h) &&
                      static_cast<unsigned>(ix) < static_cast<unsigned>(a.in_w);
      const T* p = src + (ok ? ((iy - tl.sy0) * tl.sw + (ix - tl.sx0)) * 3 : 0);
      if constexpr (DT == MAFAT_BF16) {
        const uint32_t e0 = p[0], e1 = p[1], e2 = p[2];
        pin[r][c][0] = ok ? (e0 | (e1 << 16)) : 0u;
        pin[r][c][1] = ok ? e2 : 0u;
      } else {
#pragma unroll
        for (int j = 0; j < 3; ++j) {
          const uint32_t e = __float_as_uint(to_f(p[j]));
          pin[r][c][j] = ok ? e : 0u;
        }
      }
    }

  float acc[Q * Q][CO];
#pragma unroll
  for (int q = 0; q < Q * Q; ++q)
#pragma unroll
    for (int c = 0; c < CO; ++c) acc[q][c] = 0.f;
#pragma unroll
  for (int tap = 0; tap < 9; ++tap) {
    const int ky = tap / 3, kx = tap % 3;
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const u32x4 w0 = *reinterpret_cast<const u32x4*>(&wl[(tap * NJ + j) * cout + co0]);
      const u32x4 w1 = *reinterpret_cast<const u32x4*>(&wl[(tap * NJ + j) * cout + co0 + 4]);
      const uint32_t wv[CO] = {w0.x, w0.y, w0.z, w0.w, w1.x, w1.y, w1.z, w1.w};
#pragma unroll
      for (int q = 0; q < Q * Q; ++q) {
        const uint32_t v = pin[q / Q + ky][q % Q + kx][j];
#pragma unroll
        for (int c = 0; c < CO; ++c) {
          if constexpr (DT == MAFAT_BF16)
            acc[q][c] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, v),
                                                        __builtin_bit_cast(bf16x2, wv[c]), acc[q][c], false);
          else
            acc[q][c] = fmaf(__uint_as_float(v), __uint_as_float(wv[c]), acc[q][c]);
        }
      }
    }
  }
  float r[CO];
#pragma unroll
  for (int c = 0; c < CO; ++c) {
    const float s = a.scale[co0 + c], b = a.bias[co0 + c];
    float v = activate(acc[0][c] * s + b, a.act);
#pragma unroll
    for (int q = 1; q < Q * Q; ++q) v = fmaxf(v, activate(acc[q][c] * s + b, a.act));
    r[c] = v;
  }
  int py = oy0, px = ox0;
  if (POOL) { py >>= 1; px >>= 1; }
  T* out = dst + ((py - tl.dy0) * tl.dw + (px - tl.dx0)) * cout + co0;
  if constexpr (DT == MAFAT_BF16) {
    u32x4 o;
    o.x = f2bf(r[0]) | (static_cast<uint32_t>(f2bf(r[1])) << 16);
    o.y = f2bf(r[2]) | (static_cast<uint32_t>(f2bf(r[3])) << 16);
    o.z = f2bf(r[4]) | (static_cast<uint32_t>(f2bf(r[5])) << 16);
    o.w = f2bf(r[6]) | (static_cast<uint32_t>(f2bf(r[7])) << 16);
    *reinterpret_cast<u32x4*>(out) = o;
  } else {
    *reinterpret_cast<u32x4*>(out) = u32x4{__float_as_uint(r[0]), __float_as_uint(r[1]),
                                           __float_as_uint(r[2]), __float_as_uint(r[3])};
    *reinterpret_cast<u32x4*>(out + 4) = u32x4{__float_as_uint(r[4]), __float_as_uint(r[5]),
                                               __float_as_uint(r[6]), __float_as_uint(r[7])};
  }
}

// Lone 2x2/2 max-pool: 64 output pixels per block, 4 threads per pixel
// striding over channels.  The computed rectangle is in pool-output
// coordinates.
template <int DT>
__global__ __launch_bounds__(256) void pool_kernel(const StageArgs a) {
  using T = typename Elt<DT>::T;
  KTile tl;
  const BlockPos bp = decode_block(a, &tl);
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

template <int DT, int F, bool POOL, int DEPTH>
hipError_t launch_mfma(MfmaShape sh, const StageArgs& args, hipStream_t stream) {
  const dim3 grid(static_cast<unsigned>(args.total_blocks)), block(256);
#define MAFAT_SHAPE(bm_, bn_)                                                                  \
  if (sh.bm == (bm_) && sh.bn == (bn_)) {                                                      \
    hipLaunchKernelGGL((conv_mfma_kernel<DT, F, bm_, bn_, POOL, DEPTH>), grid, block, 0, stream, args); \
    return hipGetLastError();                                                                  \
  }
  MAFAT_SHAPE(128, 128) MAFAT_SHAPE(128, 64) MAFAT_SHAPE(64, 128) MAFAT_SHAPE(64, 64)
  MAFAT_SHAPE(64, 32) MAFAT_SHAPE(32, 64) MAFAT_SHAPE(32, 32)
#undef MAFAT_SHAPE
  return hipErrorInvalidValue;
}

template <int DT, int F, bool POOL>
hipError_t launch_conv(int kind, MfmaShape sh, const StageArgs& args, hipStream_t stream) {
  const dim3 grid(static_cast<unsigned>(args.total_blocks)), block(256);
  if (kind == K_CONV_DIRECT) {
    hipLaunchKernelGGL((conv_direct_kernel<DT, F, POOL>), grid, block, 0, stream, args);
    return hipGetLastError();
  }
  if (kind == K_CONV_RGB) {
    if (F != 3) return hipErrorInvalidValue;
    hipLaunchKernelGGL((conv_rgb_kernel<DT, POOL>), grid, block, 0, stream, args);
    return hipGetLastError();
  }
  switch (sh.depth) {
    case 3: return launch_mfma<DT, F, POOL, 3>(sh, args, stream);
    case 4: return launch_mfma<DT, F, POOL, 4>(sh, args, stream);
    case 5: return launch_mfma<DT, F, POOL, 5>(sh, args, stream);
    case 6: return launch_mfma<DT, F, POOL, 6>(sh, args, stream);
    default: return hipErrorInvalidValue;
  }
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

#ifdef MAFAT_TUNING
extern "C" int mafat_debug_trace(long long* host_out) {
  return hipMemcpyFromSymbol(host_out, HIP_SYMBOL(g_trace), sizeof(g_trace)) == hipSuccess ? 0 : -1;
}
#endif

int block_units(int kind, MfmaShape shape) {
  if (kind == K_CONV_MFMA) return shape.bm;
  if (kind == K_CONV_DIRECT || kind == K_CONV_RGB) return 256;
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
