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
//                       (fp32), patch in registers.
//   conv_rgb_mfma_kernel  the 3-channel first layer in bf16 on the matrix
//                       cores, K = 27 zero-padded to 32.
//   pool_kernel         a max-pool stage that does not follow a convolution.
#include <hip/hip_runtime.h>

#include "device_util.h"
#include "kernel_args.h"

namespace mafat {
#ifdef MAFAT_TUNING
// Tuning builds only: phase timestamps of a few workgroups.
__device__ long long g_trace[4][64];
MAFAT_WG_TRACE_DECL(g_wg_rgb)
#define MAFAT_TRACE(slot_)                                                                     \
  do {                                                                                         \
    if (threadIdx.x == 0 && (blockIdx.x == 0 || blockIdx.x == a.total_blocks - 1 ||            \
                             blockIdx.x == a.total_blocks / 2) && (slot_) < 64)                     \
      g_trace[blockIdx.x == 0 ? 0 : (blockIdx.x == a.total_blocks - 1 ? 1 : 2)][(slot_)] = wall_clock64(); \
  } while (0)
#else
#define MAFAT_TRACE(slot_) do {} while (0)
#endif
namespace {


// Scale and bias of a lane's channels of each of its NT channel tiles: 4
// consecutive channels (no pool) or one channel (pool, in element 0).
template <int BN, bool POOL>
__device__ __forceinline__ void load_scale_bias(const StageArgs& a, int n0, f32x4 (&sc)[BN / 32],
                                                f32x4 (&bi)[BN / 32]) {
  constexpr int WN = BN / 2, NT = WN / 16;
  const int lane = static_cast<int>(threadIdx.x) & 63, wn = (static_cast<int>(threadIdx.x) >> 6) & 1;  // any K group
#pragma unroll
  for (int j = 0; j < NT; ++j) {
    if (POOL) {
      const int co = n0 + wn * WN + j * 16 + (lane & 15);
      const int cc = co < a.cout ? co : 0;
      sc[j] = f32x4{a.scale[cc], 0.f, 0.f, 0.f};
      bi[j] = f32x4{a.bias[cc], 0.f, 0.f, 0.f};
    } else {
      const int co = n0 + wn * WN + j * 16 + 4 * (lane >> 4);
      const int cc = co < a.cout ? co : 0;
      sc[j] = *reinterpret_cast<const f32x4*>(a.scale + cc);
      bi[j] = *reinterpret_cast<const f32x4*>(a.bias + cc);
    }
  }
}

// With KG == 2 K groups, group g stores channel tiles [g NT/2, (g+1) NT/2).
template <int DT, int BM, int BN, bool POOL, int KG>
__device__ __forceinline__ void store_direct(const f32x4 (&acc)[BN / 32][BM / 32], const f32x4 (&sc)[BN / 32],
                                             const f32x4 (&bi)[BN / 32], const StageArgs& a,
                                             const KTile& tl, int m0, int n0,
                                             typename Elt<DT>::T* dst) {
  constexpr int WM = BM / 2, WN = BN / 2, MT = WM / 16, NT = WN / 16;
  const int tid = static_cast<int>(threadIdx.x), lane = tid & 63, wave = tid >> 6;
  const int wm = (wave >> 1) & 1, wn = wave & 1, grp = wave >> 2;
  const int M = tl.ch * tl.cw, cout = a.cout;
  const float slope = act_slope(a.act);
#pragma unroll
  for (int i = 0; i < MT; ++i) {
    int oy, ox;
    bool ok;
    if (POOL) {
      // this lane's window: GEMM rows m .. m+3
      const int m = m0 + wm * WM + i * 16 + 4 * (lane >> 4);
      const int pw = tl.cw >> 1, qq = m >> 2, qy = qq / pw;
      oy = (tl.cy0 >> 1) + qy;
      ox = (tl.cx0 >> 1) + (qq - qy * pw);
      ok = m < M;
    } else {
      const int m = m0 + wm * WM + i * 16 + (lane & 15);
      row_pixel<false>(tl, m < M ? m : 0, &oy, &ox);
      ok = m < M;
    }
    typename Elt<DT>::T* drow = dst + ((oy - tl.dy0) * tl.dw + (ox - tl.dx0)) * cout;
#pragma unroll
    for (int j = 0; j < NT; ++j) {
      if (KG == 2 && (j < grp * (NT / 2) || j >= (grp + 1) * (NT / 2))) continue;
      if (POOL) {
        const int co = n0 + wn * WN + j * 16 + (lane & 15);
        float v[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) v[r] = fmaf(acc[j][i][r], sc[j][0], bi[j][0]);
        float m = fmaxf(fmaxf(v[0], v[1]), fmaxf(v[2], v[3]));
        m = fmaxf(m, slope * m);
        if (ok && co < cout) store1(drow + co, m);
      } else {
        const int co = n0 + wn * WN + j * 16 + 4 * (lane >> 4);
        float v[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          v[r] = fmaf(acc[j][i][r], sc[j][r], bi[j][r]);
          v[r] = fmaxf(v[r], slope * v[r]);
        }
        if (ok && co < cout) store4<DT>(drow + co, v);
      }
    }
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
// Epilogue: see store_direct (no LDS).
//
// Requires c_in % (64 / sizeof(T)) == 0, c_out % 16 == 0 and byte offsets
// below 2^31 within a frame's source buffer and the weights (host-checked).
template <int DT, int F, int BM, int BN, bool POOL, int DEPTH, int KG>
__global__ __launch_bounds__(256 * KG) void conv_mfma_kernel(const StageArgs a) {
  if (__builtin_expect(blockIdx.y != 0, 0)) {  // the second grid row: carried band copies (row reuse)
    carried_copies();
    return;
  }
  using T = typename Elt<DT>::T;
  constexpr int ESZ = static_cast<int>(sizeof(T));
  constexpr int P = (F - 1) / 2;
  constexpr int KC = 64 / ESZ;   // channels per sub-chunk
  constexpr int EPV = 16 / ESZ;  // channels per 16 bytes
  constexpr int ROWQ = 9;        // u32x4 per LDS row
  constexpr int RSTEP = 32 * KG;                     // rows staged per pass of the workgroup
  constexpr int ALD = BM / RSTEP, BLD = BN / RSTEP;  // loads per thread per stage
  constexpr int WM = BM / 2, WN = BN / 2, MT = WM / 16, NT = WN / 16;
  constexpr int NH = 2 / KG;  // 64-byte halves of a stage each wave multiplies
  static_assert(KG == 1 || KG == 2, "K groups");
  static_assert(ALD >= 1 && BLD >= 1 && ALD * RSTEP == BM && BLD * RSTEP == BN, "block shape");
  static_assert(KG == 1 || NT % 2 == 0, "two K groups split the channel tiles in the epilogue");
  static_assert(DEPTH >= 3 && DEPTH <= 6, "pipeline depth");
  static_assert(F * F + 2 * DEPTH + 2 < 32, "tap mask width (taps of computed stages)");
  constexpr int NBUF = 2;  // LDS stage buffers
  constexpr int OPND_BYTES = NBUF * (BM + BN) * ROWQ * 16;
  __shared__ __align__(16) unsigned char smem[OPND_BYTES];
  u32x4* sA = reinterpret_cast<u32x4*>(smem);  // [NBUF][BM][ROWQ]
  u32x4* sB = sA + NBUF * BM * ROWQ;           // [NBUF][BN][ROWQ]

  MAFAT_TRACE(0);
  KTile tl;
  const BlockPos bp = decode_block(a, &tl);
  const int tid = static_cast<int>(threadIdx.x), lane = tid & 63, wave = tid >> 6;
  // Waves 4g .. 4g+3 form K group g (2x2 over the block); with two groups,
  // group g multiplies the 64-byte half g of every stage.
  const int grp = wave >> 2, wm = (wave >> 1) & 1, wn = wave & 1;
  const int h0 = (KG == 2) ? grp : 0;
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

  // This thread stages rows r0 + RSTEP i, 16-byte piece `pc` of sub-chunk `hh`
  // of every stage.  Per A row: the byte offset of its pixel in the source
  // buffer and a mask of the filter taps that read zero (outside the image;
  // bits past the last tap are set, so padded sub-chunks read zero).  Loads
  // that must read zero get bit 31 set in their offset.
  const int r0 = tid >> 3, q = tid & 7, hh = q >> 2, pc = q & 3;
  unsigned a_off[ALD], a_inv[ALD], b_off[BLD];
#pragma unroll
  for (int i = 0; i < ALD; ++i) {
    const int m = m0 + r0 + RSTEP * i;
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
    const int co = n0 + r0 + RSTEP * i;
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
      sA[((buf_) * BM + r0 + RSTEP * i) * ROWQ + q] = ra[d_][i];                               \
    _Pragma("unroll") for (int i = 0; i < BLD; ++i)                                            \
      sB[((buf_) * BN + r0 + RSTEP * i) * ROWQ + q] = rb[d_][i];                               \
  } while (0)

  f32x4 acc[NT][MT];  // [channel tile][pixel tile], orientation: see store_direct
#pragma unroll
  for (int j = 0; j < NT; ++j)
#pragma unroll
    for (int i = 0; i < MT; ++i) acc[j][i] = f32x4{0.f, 0.f, 0.f, 0.f};

  // Pipeline, per step st (computing stage st from LDS buffer st % 2):
  //   barrier (stage st is in LDS; every wave is done reading stage st - 1);
  //   read both K-halves' fragments of stage st; issue the global loads of
  //   stage st + DEPTH into the register set stage st came from; MFMAs;
  //   write stage st + 1 (loaded DEPTH - 1 steps ago) to the other buffer.
  // The stage count is padded to a multiple of DEPTH so the unrolled loop
  // body has no branches (padded stages read zero A rows).
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
#define MAFAT_STEP(d_, dn_, load_)                                                               \
  do {                                                                                           \
    __syncthreads();                                                                             \
    u32x4 af[NH][MT], bfr[NH][NT];                                                               \
    _Pragma("unroll") for (int h = 0; h < NH; ++h) {                                             \
      _Pragma("unroll") for (int i = 0; i < MT; ++i)                                             \
        af[h][i] = sA[(rbuf * BM + wm * WM + i * 16 + (lane & 15)) * ROWQ + (h0 + h) * 4 + (lane >> 4)]; \
      _Pragma("unroll") for (int j = 0; j < NT; ++j)                                             \
        bfr[h][j] = sB[(rbuf * BN + wn * WN + j * 16 + (lane & 15)) * ROWQ + (h0 + h) * 4 + (lane >> 4)]; \
    }                                                                                            \
    if (load_) MAFAT_GLOAD(d_);                                                                  \
    _Pragma("unroll") for (int h = 0; h < NH; ++h)                                               \
      _Pragma("unroll") for (int i = 0; i < MT; ++i)                                             \
        _Pragma("unroll") for (int j = 0; j < NT; ++j) {                                         \
          if constexpr (POOL) mma<DT>(acc[j][i], af[h][i], bfr[h][j]);                           \
          else mma<DT>(acc[j][i], bfr[h][j], af[h][i]);                                          \
        }                                                                                        \
    rbuf ^= 1;                                                                                   \
    MAFAT_LSTORE(dn_, rbuf);                                                                     \
    MAFAT_TRACE(8 + s0 + (d_));                                                                  \
  } while (0)
#define MAFAT_STEPS(load_)                                                                       \
  do {                                                                                           \
    if constexpr (DEPTH == 3) {                                                                  \
      MAFAT_STEP(0, 1, load_); MAFAT_STEP(1, 2, load_); MAFAT_STEP(2, 0, load_);                 \
    } else if constexpr (DEPTH == 4) {                                                           \
      MAFAT_STEP(0, 1, load_); MAFAT_STEP(1, 2, load_); MAFAT_STEP(2, 3, load_);                 \
      MAFAT_STEP(3, 0, load_);                                                                   \
    } else if constexpr (DEPTH == 5) {                                                           \
      MAFAT_STEP(0, 1, load_); MAFAT_STEP(1, 2, load_); MAFAT_STEP(2, 3, load_);                 \
      MAFAT_STEP(3, 4, load_); MAFAT_STEP(4, 0, load_);                                          \
    } else {                                                                                     \
      MAFAT_STEP(0, 1, load_); MAFAT_STEP(1, 2, load_); MAFAT_STEP(2, 3, load_);                 \
      MAFAT_STEP(3, 4, load_); MAFAT_STEP(4, 5, load_); MAFAT_STEP(5, 0, load_);                 \
    }                                                                                            \
  } while (0)
  // Steady state: every step loads the stage DEPTH ahead.  The last DEPTH
  // steps load nothing (all their stages are in flight already), so nothing
  // useless sits in the memory queue ahead of the epilogue's scale and bias,
  // which are fetched before those steps.
  int s0 = 0;
  for (; s0 < nst_pad - DEPTH; s0 += DEPTH) MAFAT_STEPS(true);
  f32x4 sc[NT], bi[NT];
  load_scale_bias<BN, POOL>(a, n0, sc, bi);
  MAFAT_STEPS(false);
  MAFAT_TRACE(1);
#undef MAFAT_STEPS
#undef MAFAT_STEP
#undef MAFAT_GLOAD
#undef MAFAT_LSTORE

  MAFAT_TRACE(2);
  if constexpr (KG == 2) {
    // Each group keeps half of the channel tiles: it hands the other half of
    // its partial sums to the partner wave (same 2x2 position) through LDS
    // and adds the partner's partial sums for its own half.
    constexpr int NH2 = NT / 2;
    static_assert(8 * 64 * NH2 * MT * 16 <= OPND_BYTES, "partial sums fit in the operand buffers");
    f32x4* sX = reinterpret_cast<f32x4*>(smem);  // [wave][NT/2][MT][64 lanes]
    __syncthreads();  // every wave is done with the operand buffers
    // (Two copies with constant indices: a wave-dependent index into acc
    // would move it to scratch memory.)
    const int partner = wave ^ 4;
    if (grp == 0) {
#pragma unroll
      for (int j = 0; j < NH2; ++j)
#pragma unroll
        for (int i = 0; i < MT; ++i) sX[((wave * NH2 + j) * MT + i) * 64 + lane] = acc[NH2 + j][i];
    } else {
#pragma unroll
      for (int j = 0; j < NH2; ++j)
#pragma unroll
        for (int i = 0; i < MT; ++i) sX[((wave * NH2 + j) * MT + i) * 64 + lane] = acc[j][i];
    }
    __syncthreads();
    if (grp == 0) {
#pragma unroll
      for (int j = 0; j < NH2; ++j)
#pragma unroll
        for (int i = 0; i < MT; ++i) acc[j][i] += sX[((partner * NH2 + j) * MT + i) * 64 + lane];
    } else {
#pragma unroll
      for (int j = 0; j < NH2; ++j)
#pragma unroll
        for (int i = 0; i < MT; ++i) acc[NH2 + j][i] += sX[((partner * NH2 + j) * MT + i) * 64 + lane];
    }
  }
  store_direct<DT, BM, BN, POOL, KG>(acc, sc, bi, a, tl, m0, n0, dst);
  MAFAT_TRACE(3);
}


// Direct convolution on the vector ALUs, one thread per output pixel (or per
// 2x2 pool window), all output channels in chunks of 8.  Weights are read
// with wave-uniform addresses (scalar cache).  F > 0: an f = F "same"
// convolution (stride 1, padding (F - 1) / 2); F = 0: any filter, stride and
// padding, taken from the stage arguments (a.f, a.s, a.p).
template <int DT, int F, bool POOL>
__global__ __launch_bounds__(256) void conv_direct_kernel(const StageArgs a) {
  if (__builtin_expect(blockIdx.y != 0, 0)) {  // the second grid row: carried band copies (row reuse)
    carried_copies();
    return;
  }
  using T = typename Elt<DT>::T;
  const int f = F > 0 ? F : a.f;
  const int st = F > 0 ? 1 : a.s;
  const int pd = F > 0 ? (F - 1) / 2 : a.p;
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
  const int cin = a.cin, cout = a.cout, K = f * f * cin;
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
    for (int ky = 0; ky < f; ++ky)
      for (int kx = 0; kx < f; ++kx) {
        const T* px[NP];
        bool ok[NP];
#pragma unroll
        for (int p = 0; p < NP; ++p) {
          const int iy = oy[p] * st + ky - pd, ix = ox[p] * st + kx - pd;
          ok[p] = static_cast<unsigned>(iy) < static_cast<unsigned>(a.in_h) &&
                  static_cast<unsigned>(ix) < static_cast<unsigned>(a.in_w);
          px[p] = ok[p] ? src + ((iy - tl.sy0) * tl.sw + (ix - tl.sx0)) * cin : src;
        }
        const T* wt = wgt + static_cast<int64_t>(co0) * K + (ky * f + kx) * cin;
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
  if (__builtin_expect(blockIdx.y != 0, 0)) {  // the second grid row: carried band copies (row reuse)
    carried_copies();
    return;
  }
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

// First layer on the matrix cores (bf16).  Its K = 3x3x3 = 27 runs as three
// v_mfma_f32_16x16x16_bf16, one per filter row ky, each with K = 16 = 4 kx
// slots x 4 channel slots: (kx, c) for kx < 3, c < 3, and zeros (channel
// slot 3, and the whole kx slot 3, have zero weights).  A workgroup computes
// a BR x BC block of conv outputs (all c_out channels) of one tile:
//   1. the (BR+2) x (BC+2) input patch is staged in LDS as 8-byte pixels
//      (c0, c1, c2, 0), so the 4 K values of a lane's operand are one
//      aligned 8-byte LDS read at a per-lane constant offset; a thread
//      fetches whole pixels, each with one aligned 4-byte and one 2-byte
//      buffer load (all of a thread's loads are issued before its first
//      LDS write), zero outside the image and
//      outside the tile's source region (those loads get an offset past
//      the descriptor's range); the weights, scale and bias, the same for
//      every workgroup, are staged with one 16-byte load per thread;
//   2. each wave takes 16-pixel tiles (2 rows x 8 columns, ordered as 4
//      windows of 2x2); lane l loads, for each ky, the pixel (kx = l / 16)
//      of its pixel's (l % 16) filter window (kx slot 3 repeats kx = 2, which
//      meets zero weights);
//   3. epilogue: without a pool the weights are the A operand (a lane ends
//      with 4 consecutive channels of one pixel, one 8-byte store); with a
//      fused 2x2 pool the pixels are (a lane's 4 accumulator rows are one
//      window of one channel: scale and bias, the window maximum, then the
//      activation, which is monotone), and a wave takes whole rows of
//      tiles, whose pooled output is one contiguous run: it is staged in LDS
//      and written with 16-byte stores.
// Requires c_out = 16 * NJ, c_in = 3, f = 3, s = 1, p = 1 (host-checked).
template <bool POOL, int NJ>
__global__ __launch_bounds__(256) void conv_rgb_mfma_kernel(const StageArgs a) {
  if (__builtin_expect(blockIdx.y != 0, 0)) {  // the second grid row: carried band copies (row reuse)
    carried_copies();
    return;
  }
  typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
  typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
  constexpr int BR = kRgbBlockRows, BC = kRgbBlockCols;  // conv outputs per block, even
  constexpr int SR = BR + 2, SC = BC + 2;    // staged input patch (pixels)
  constexpr int RS = SC * 4 + 8;             // bf16 per LDS row (8-byte pixels + pad)
  constexpr int NTILE = BR * BC / 16;        // 16-pixel MFMA tiles
  constexpr int TPR = BC / 8;                // tiles per 2 rows
  constexpr int COUT = 16 * NJ;
  constexpr int W16 = COUT * 27 * 2 / 16;    // 16-byte pieces of the weights
  __shared__ __align__(16) uint16_t sx[SR * RS];
  __shared__ __align__(16) uint16_t swt[COUT * 27];
  __shared__ __align__(16) float ssb[2 * COUT];  // scale, bias
  __shared__ __align__(16) uint16_t spool[POOL ? 4 * 4 * (BC / 8) * COUT : 8];  // per-wave pooled row staging

  MAFAT_WG_MARK(g_wg_rgb, 0);
  MAFAT_TRACE(0);
  const int tid = static_cast<int>(threadIdx.x), lane = tid & 63, wave = tid >> 6;
  // Weights, scale, bias (the same for every block; 16 bytes per thread):
  // fetched before the tile table is decoded, written to LDS after the
  // input patch's loads are issued.
  const u32x4* psrc = (tid < W16)              ? reinterpret_cast<const u32x4*>(a.w) + tid
                      : (tid < W16 + COUT / 4) ? reinterpret_cast<const u32x4*>(a.scale) + (tid - W16)
                      : (tid < W16 + COUT / 2) ? reinterpret_cast<const u32x4*>(a.bias) + (tid - W16 - COUT / 4)
                                               : nullptr;
  u32x4 pv = u32x4{0u, 0u, 0u, 0u};
  if (psrc) pv = *psrc;
  KTile tl;
  const BlockPos bp = decode_block(a, &tl);
  MAFAT_TRACE(4 + (tl.ch > 30000 ? 1 : 0));
  const int nbx = (tl.cw + BC - 1) / BC;
  const int by = bp.mb / nbx, bx = bp.mb - by * nbx;
  const int oy0 = tl.cy0 + by * BR, ox0 = tl.cx0 + bx * BC;
  uint16_t* dst = static_cast<uint16_t*>(a.dst) + bp.frame * a.dst_fstride + tl.dst_off;
  const int kq = lane >> 4;

  // Input patch: rows oy0-1 .. oy0+BR, columns ox0-1 .. ox0+BC, one pixel
  // (3 bf16, 6 bytes) per thread and step: an aligned 4-byte and a 2-byte
  // load (which halves of the pixel they hold depends on its address
  // modulo 4), written to LDS as one 8-byte slot (c0, c1, c2, 0).  Pixels
  // outside the image, or outside this tile's source region (only outputs
  // outside the tile's computed rectangle would read them), read 0.
  const int ylo = max(0, tl.cy0 - 1), yhi = min(a.in_h, tl.cy0 + tl.ch + 1);
  const int xlo = max(0, tl.cx0 - 1), xhi = min(a.in_w, tl.cx0 + tl.cw + 1);
  const int64_t sb = bp.frame * a.src_fstride + tl.src_off;  // elements; the source buffer is 16-byte aligned
  const int bpar = static_cast<int>(sb & 1);
  const __amdgpu_buffer_rsrc_t rs =
      make_rsrc(static_cast<const uint16_t*>(a.src) + sb, static_cast<unsigned>((a.src_fstride - tl.src_off) * 2));
  const int p00 = (oy0 - 1 - tl.sy0) * tl.sw + (ox0 - 1 - tl.sx0);  // patch origin in the source region
  constexpr int NPX = SR * SC;
  constexpr int NPT = (NPX + 255) / 256;  // pixels per thread
  uint32_t la[NPT], lb[NPT];
  bool lodd[NPT];
#pragma unroll
  for (int k = 0; k < NPT; ++k) {
    const int e = tid + 256 * k;
    const int r = e / SC, px = e - r * SC;
    const int iy = oy0 - 1 + r, ix = ox0 - 1 + px;
    const bool ok = e < NPX && static_cast<unsigned>(iy - ylo) < static_cast<unsigned>(yhi - ylo) &&
                    static_cast<unsigned>(ix - xlo) < static_cast<unsigned>(xhi - xlo);
    const int p = p00 + r * tl.sw + px;
    const bool odd = ((bpar + p) & 1) != 0;  // c0 at an address = 2 (mod 4): the dword holds c1, c2
    const unsigned off = static_cast<unsigned>(p * 6);
    const unsigned oa = odd ? off + 2u : off, ob = odd ? off : off + 4u;
    la[k] = __builtin_amdgcn_raw_buffer_load_b32(rs, static_cast<int>(ok ? oa : 0x80000000u), 0, 0);
    lb[k] = __builtin_amdgcn_raw_buffer_load_b16(rs, static_cast<int>(ok ? ob : 0x80000000u), 0, 0);
    lodd[k] = odd;
  }
  if (tid < W16) reinterpret_cast<u32x4*>(swt)[tid] = pv;
  else if (tid < W16 + COUT / 2) reinterpret_cast<u32x4*>(ssb)[tid - W16] = pv;  // scale, then bias
#pragma unroll
  for (int k = 0; k < NPT; ++k) {
    const int e = tid + 256 * k;
    const int r = e / SC, px = e - r * SC;
    const uint32_t b = lb[k] & 0xffffu;
    const u32x2 v = lodd[k] ? u32x2{b | (la[k] << 16), la[k] >> 16} : u32x2{la[k], b};
    if (e < NPX) *reinterpret_cast<u32x2*>(sx + r * RS + px * 4) = v;
  }
  MAFAT_TRACE(6);
  __syncthreads();
  MAFAT_TRACE(7);

  // Weight operand of a lane, per channel tile j and filter row ky: output
  // channel 16 j + (lane & 15), kx slot kq: (w[c0], w[c1], w[c2], 0), zero
  // for kq = 3.  (The same registers serve as A or B operand.)
  u32x2 wf[NJ][3];
#pragma unroll
  for (int j = 0; j < NJ; ++j)
#pragma unroll
    for (int ky = 0; ky < 3; ++ky) {
      const int wr = (16 * j + (lane & 15)) * 27 + ky * 9 + 3 * min(kq, 2);
      const uint32_t w0 = swt[wr], w1 = swt[wr + 1], w2 = swt[wr + 2];
      wf[j][ky] = kq < 3 ? u32x2{w0 | (w1 << 16), w2} : u32x2{0u, 0u};
    }
  float sc[NJ][4], bi[NJ][4];
#pragma unroll
  for (int j = 0; j < NJ; ++j)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int co = POOL ? 16 * j + (lane & 15) : 16 * j + 4 * kq + r;
      sc[j][r] = ssb[co];
      bi[j][r] = ssb[COUT + co];
    }
  const float slope = act_slope(a.act);

  const int p = lane & 15;  // pixel of the MFMA tile whose operand this lane loads
  const int kx = min(kq, 2);
  // MFMAs of 16-pixel tile t: rows 2 (t / TPR) .. +1, columns 8 (t % TPR)
  // .. +7, as 4 windows of 2x2 (pixel p is window p >> 2, position p & 3).
  auto tile_mfma = [&](int t, f32x4 (&acc)[NJ]) {
    const int py = 2 * (t / TPR) + ((p & 3) >> 1);
    const int pxl = 8 * (t % TPR) + 2 * (p >> 2) + (p & 1);
    const u32x2* xp = reinterpret_cast<const u32x2*>(sx + py * RS + (pxl + kx) * 4);
    u32x2 xf[3];
#pragma unroll
    for (int ky = 0; ky < 3; ++ky) xf[ky] = xp[ky * (RS / 4)];
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ky = 0; ky < 3; ++ky) {
        const bf16x4 xa = __builtin_bit_cast(bf16x4, xf[ky]), wa = __builtin_bit_cast(bf16x4, wf[j][ky]);
        acc[j] = POOL ? __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(xa, wa, acc[j], 0, 0, 0)
                      : __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(wa, xa, acc[j], 0, 0, 0);
      }
    }
  };
  if constexpr (POOL) {
    // A wave takes whole tile rows (the TPR tiles of two conv rows, i.e.
    // 4 * TPR pooled pixels of one pooled row, contiguous in the output).
    // A lane's accumulator rows are window kq of its tile, column = its
    // channel: the pooled values go through this wave's LDS staging row,
    // then leave as 16-byte stores (8 channels of one pooled pixel per lane).
    constexpr int PPR = 4 * TPR;   // pooled pixels per tile row
    constexpr int CPL = COUT / 8;  // 16-byte chunks per pooled pixel
    uint16_t* lrow = spool + wave * PPR * COUT;
    for (int tr = wave; tr < BR / 2; tr += 4) {
#pragma unroll
      for (int c = 0; c < TPR; ++c) {
        f32x4 acc[NJ];
        tile_mfma(tr * TPR + c, acc);
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
          float v[4];
#pragma unroll
          for (int r = 0; r < 4; ++r) v[r] = fmaf(acc[j][r], sc[j][0], bi[j][0]);
          float m = fmaxf(fmaxf(v[0], v[1]), fmaxf(v[2], v[3]));
          m = fmaxf(m, slope * m);
          store1(lrow + (c * 4 + kq) * COUT + 16 * j + p, m);
        }
      }
      __builtin_amdgcn_wave_barrier();  // LDS ops of a wave run in order; keep the compiler from moving them
      const int oy = oy0 + 2 * tr;
#pragma unroll
      for (int e = lane; e < PPR * CPL; e += 64) {
        const int q = e / CPL, ck = e - q * CPL;
        const int ox = ox0 + 2 * q;
        const u32x4 v = *reinterpret_cast<const u32x4*>(lrow + q * COUT + ck * 8);
        if ((oy - tl.cy0) < tl.ch && (ox - tl.cx0) < tl.cw)
          *reinterpret_cast<u32x4*>(dst + (((oy >> 1) - tl.dy0) * tl.dw + ((ox >> 1) - tl.dx0)) * COUT + ck * 8) = v;
      }
      __builtin_amdgcn_wave_barrier();
    }
  } else {
    for (int t = wave; t < NTILE; t += 4) {
      f32x4 acc[NJ];
      tile_mfma(t, acc);
      // a lane's accumulator rows are channels 4 kq .. +3 of pixel p
      const int py = 2 * (t / TPR) + ((p & 3) >> 1);
      const int pxl = 8 * (t % TPR) + 2 * (p >> 2) + (p & 1);
      const int oy = oy0 + py, ox = ox0 + pxl;
      const bool ok = (oy - tl.cy0) < tl.ch && (ox - tl.cx0) < tl.cw;
      uint16_t* drow = dst + ((oy - tl.dy0) * tl.dw + (ox - tl.dx0)) * COUT;
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        float v[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          v[r] = fmaf(acc[j][r], sc[j][r], bi[j][r]);
          v[r] = fmaxf(v[r], slope * v[r]);
        }
        if (ok) store4<MAFAT_BF16>(drow + 16 * j + 4 * kq, v);
      }
    }
  }
  MAFAT_WG_MARK(g_wg_rgb, 1);
  MAFAT_TRACE(3);
}


// A max-pool stage (one that does not follow a convolution, or any other
// window than 2x2/2): 64 output pixels per block, 4 threads per pixel
// striding over channels.  Output (y, x) takes the maximum over the in-image
// elements of rows y*s - p .. y*s - p + f - 1 (columns likewise; padding is
// not part of the window).  The computed rectangle is in pool-output
// coordinates.
template <int DT>
__global__ __launch_bounds__(256) void pool_kernel(const StageArgs a) {
  if (__builtin_expect(blockIdx.y != 0, 0)) {  // the second grid row: carried band copies (row reuse)
    carried_copies();
    return;
  }
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
  const int y0 = max(oy * a.s - a.p, 0), y1 = min(oy * a.s - a.p + a.f, a.in_h);
  const int x0 = max(ox * a.s - a.p, 0), x1 = min(ox * a.s - a.p + a.f, a.in_w);
  T* o = dst + ((oy - tl.dy0) * tl.dw + (ox - tl.dx0)) * c_in;
  for (int c = static_cast<int>(threadIdx.x) & 3; c < c_in; c += 4) {
    float m = -INFINITY;
    for (int iy = y0; iy < y1; ++iy)
      for (int ix = x0; ix < x1; ++ix) m = fmaxf(m, to_f(src[((iy - tl.sy0) * tl.sw + (ix - tl.sx0)) * c_in + c]));
    put(o + c, m);
  }
}

template <int DT, int F, bool POOL, int DEPTH>
hipError_t launch_mfma(MfmaShape sh, const StageArgs& args, hipStream_t stream, LaunchEvents ev) {
  const dim3 grid(static_cast<unsigned>(args.total_blocks), args.copy_blocks > 0 ? 2u : 1u);
#define MAFAT_SHAPE(bm_, bn_, kg_)                                                             \
  if (sh.bm == (bm_) && sh.bn == (bn_) && sh.kg == (kg_)) {                                    \
    hipExtLaunchKernelGGL((conv_mfma_kernel<DT, F, bm_, bn_, POOL, DEPTH, kg_>), grid, dim3(256 * (kg_)), 0, \
                          stream, ev.start, ev.stop, 0, args);                                 \
    return hipGetLastError();                                                                  \
  }
  MAFAT_SHAPE(128, 128, 1) MAFAT_SHAPE(128, 64, 1) MAFAT_SHAPE(64, 128, 1) MAFAT_SHAPE(64, 64, 1)
  MAFAT_SHAPE(64, 32, 1) MAFAT_SHAPE(32, 64, 1) MAFAT_SHAPE(32, 32, 1)
  MAFAT_SHAPE(128, 128, 2) MAFAT_SHAPE(128, 64, 2) MAFAT_SHAPE(64, 128, 2) MAFAT_SHAPE(64, 64, 2)
#undef MAFAT_SHAPE
  return hipErrorInvalidValue;
}

template <int DT, int F, bool POOL>
hipError_t launch_conv(int kind, MfmaShape sh, const StageArgs& args, hipStream_t stream, LaunchEvents ev) {
  const dim3 grid(static_cast<unsigned>(args.total_blocks), args.copy_blocks > 0 ? 2u : 1u), block(256);
  if (kind == K_CONV_DIRECT) {
    hipExtLaunchKernelGGL((conv_direct_kernel<DT, F, POOL>), grid, block, 0, stream, ev.start, ev.stop, 0, args);
    return hipGetLastError();
  }
  if (kind == K_CONV_RGB) {
    if (F != 3) return hipErrorInvalidValue;
    hipExtLaunchKernelGGL((conv_rgb_kernel<DT, POOL>), grid, block, 0, stream, ev.start, ev.stop, 0, args);
    return hipGetLastError();
  }
  if (kind == K_CONV_RGB_MFMA) {
    if (F != 3 || DT != MAFAT_BF16) return hipErrorInvalidValue;
    switch (sh.bn) {  // c_out
      case 16: hipExtLaunchKernelGGL((conv_rgb_mfma_kernel<POOL, 1>), grid, block, 0, stream, ev.start, ev.stop, 0, args); break;
      case 32: hipExtLaunchKernelGGL((conv_rgb_mfma_kernel<POOL, 2>), grid, block, 0, stream, ev.start, ev.stop, 0, args); break;
      case 64: hipExtLaunchKernelGGL((conv_rgb_mfma_kernel<POOL, 4>), grid, block, 0, stream, ev.start, ev.stop, 0, args); break;
      default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
  }
  // bf16 matrix-core stages run the LDS-ring kernel (conv_ring.hip); this
  // register-staged kernel serves float32 ("same" 1x1 and 3x3 only).
  if constexpr (DT != MAFAT_F32 || F == 0) return hipErrorInvalidValue;
  else switch (sh.depth) {
    case 3: return launch_mfma<DT, F, POOL, 3>(sh, args, stream, ev);
    case 4: return launch_mfma<DT, F, POOL, 4>(sh, args, stream, ev);
    case 5: return launch_mfma<DT, F, POOL, 5>(sh, args, stream, ev);
    case 6: return launch_mfma<DT, F, POOL, 6>(sh, args, stream, ev);
    default: return hipErrorInvalidValue;
  }
}

template <int DT>
hipError_t launch_dt(int kind, int f, bool pool, MfmaShape sh, const StageArgs& args,
                     hipStream_t stream, LaunchEvents ev) {
  if (kind == K_POOL) {
    hipExtLaunchKernelGGL((pool_kernel<DT>), dim3(static_cast<unsigned>(args.total_blocks), args.copy_blocks > 0 ? 2u : 1u), dim3(256),
                          0, stream, ev.start, ev.stop, 0, args);
    return hipGetLastError();
  }
  if (f == 3) return pool ? launch_conv<DT, 3, true>(kind, sh, args, stream, ev)
                          : launch_conv<DT, 3, false>(kind, sh, args, stream, ev);
  if (f == 1) return pool ? launch_conv<DT, 1, true>(kind, sh, args, stream, ev)
                          : launch_conv<DT, 1, false>(kind, sh, args, stream, ev);
  if (f == 0 && kind == K_CONV_DIRECT)  // any filter, stride and padding (stage arguments)
    return pool ? launch_conv<DT, 0, true>(kind, sh, args, stream, ev)
                : launch_conv<DT, 0, false>(kind, sh, args, stream, ev);
  return hipErrorInvalidValue;
}

}  // namespace

#ifdef MAFAT_TUNING
extern "C" int mafat_debug_wg_rgb(long long* host_out) {
  return hipMemcpyFromSymbol(host_out, HIP_SYMBOL(g_wg_rgb), sizeof(g_wg_rgb)) == hipSuccess ? 0 : -1;
}
extern "C" int mafat_debug_trace(long long* host_out) {
  return hipMemcpyFromSymbol(host_out, HIP_SYMBOL(g_trace), sizeof(g_trace)) == hipSuccess ? 0 : -1;
}
#endif

int block_units(int kind, MfmaShape shape) {
  if (kind == K_CONV_MFMA || kind == K_CONV_RING) return shape.bm;
  if (kind == K_CONV_DIRECT || kind == K_CONV_RGB) return 256;
  return 64;
}

namespace {
// Weight repack for the patch kernel: one 16-byte piece (8 channels) per
// thread, [cout/BN][cin/32][9][BN][32] from KRSC [cout][3][3][cin]; rows
// past c_out are zero.
__global__ __launch_bounds__(256) void pack_weights_kernel(const uint16_t* src, uint16_t* dst, int cout, int cin,
                                                           int bn, int nblk) {
  const int nchunk = cin >> 5;
  const int64_t total = static_cast<int64_t>(nblk) * nchunk * 9 * bn * 4;
  const int64_t e = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (e >= total) return;
  const int q = static_cast<int>(e & 3);                // 8-channel piece of the 32
  int64_t r = e >> 2;
  const int n = static_cast<int>(r % bn); r /= bn;      // row of the channel block
  const int t = static_cast<int>(r % 9); r /= 9;        // tap
  const int c = static_cast<int>(r % nchunk); r /= nchunk;  // 32-channel chunk
  const int b = static_cast<int>(r);                    // channel block
  const int co = b * bn + n;
  u32x4 v = u32x4{0u, 0u, 0u, 0u};
  if (co < cout) v = *reinterpret_cast<const u32x4*>(src + (static_cast<int64_t>(co) * 9 + t) * cin + c * 32 + q * 8);
  *reinterpret_cast<u32x4*>(dst + e * 8) = v;
}

}  // namespace

hipError_t launch_pack_weights(const uint16_t* src, uint16_t* dst, int cout, int cin, int bn, int nblk,
                               hipStream_t stream) {
  const int64_t total = static_cast<int64_t>(nblk) * (cin >> 5) * 9 * bn * 4;
  if (total <= 0) return hipSuccess;
  const dim3 grid(static_cast<unsigned>((total + 255) / 256));
  hipLaunchKernelGGL(pack_weights_kernel, grid, dim3(256), 0, stream, src, dst, cout, cin, bn, nblk);
  return hipGetLastError();
}

namespace {
// Band take-over copies: unit-sized pieces (16 bytes when every offset and
// length allows it, else 2) of all copies one after another; y = frame.
template <typename U>
__global__ __launch_bounds__(256) void band_copy_kernel(unsigned char* scratch, const BandCopyArgs a) {
  unsigned char* frame = scratch + static_cast<int64_t>(blockIdx.y) * a.fstride;
  int64_t total = 0;
  for (int k = 0; k < a.ncopy; ++k) total += a.bytes[k] / static_cast<int64_t>(sizeof(U));
  for (int64_t u = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; u < total;
       u += static_cast<int64_t>(gridDim.x) * 256) {
    int64_t r = u;
    int k = 0;
    while (r >= a.bytes[k] / static_cast<int64_t>(sizeof(U))) {
      r -= a.bytes[k] / static_cast<int64_t>(sizeof(U));
      ++k;
    }
    const U v = *reinterpret_cast<const U*>(frame + a.src[k] + r * static_cast<int64_t>(sizeof(U)));
    *reinterpret_cast<U*>(frame + a.dst[k] + r * static_cast<int64_t>(sizeof(U))) = v;
  }
}
}  // namespace

hipError_t launch_band_copy(void* scratch, const BandCopyArgs& args, int batch, hipStream_t stream) {
  if (args.ncopy <= 0 || batch <= 0) return hipSuccess;
  bool wide = (args.fstride % 16) == 0;
  int64_t total = 0;
  for (int k = 0; k < args.ncopy; ++k) {
    wide = wide && (args.src[k] % 16) == 0 && (args.dst[k] % 16) == 0 && (args.bytes[k] % 16) == 0;
    total += args.bytes[k];
  }
  const int64_t units = total / (wide ? 16 : 2);
  if (units <= 0) return hipSuccess;
  const dim3 grid(static_cast<unsigned>(std::min<int64_t>((units + 255) / 256, 1024)), static_cast<unsigned>(batch));
  if (wide)
    hipLaunchKernelGGL(band_copy_kernel<u32x4>, grid, dim3(256), 0, stream, static_cast<unsigned char*>(scratch), args);
  else
    hipLaunchKernelGGL(band_copy_kernel<uint16_t>, grid, dim3(256), 0, stream, static_cast<unsigned char*>(scratch),
                       args);
  return hipGetLastError();
}

hipError_t launch_stage(int kind, int dtype, int f, bool pool, MfmaShape shape,
                        const StageArgs& args, hipStream_t stream, LaunchEvents ev) {
  if (args.total_blocks <= 0) return hipSuccess;
  if (dtype == MAFAT_BF16) return launch_dt<MAFAT_BF16>(kind, f, pool, shape, args, stream, ev);
  if (dtype == MAFAT_F32) return launch_dt<MAFAT_F32>(kind, f, pool, shape, args, stream, ev);
  return hipErrorInvalidValue;
}

}  // namespace mafat
