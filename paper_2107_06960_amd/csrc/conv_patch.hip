// conv_patch.hip -- bf16 3x3 convolution stage (stride 1, zero padding
// outside the image, folded batch-norm scale/bias, activation, optional
// fused 2x2/2 max-pool) on the matrix cores, with the input patch of a 2-D
// block of output pixels staged in LDS once per channel chunk and shared by
// all nine filter taps.
//
// Why: as an implicit GEMM with im2col rows, every input pixel is fetched
// once per tap (nine times).  Here a workgroup owns a BR x BC block of conv
// outputs of one tile (and BN output channels); for each chunk of 32 input
// channels it loads the (BR+2) x (BC+2) input patch (64 bytes per pixel)
// and the nine 64-byte tap slices of its BN weight rows, and runs the nine
// taps' MFMAs from LDS, the A operand of tap (ky, kx) being the patch
// shifted by (ky, kx).
//
// GEMM view per chunk and tap: M = the block's pixels, window-major (every
// 4 consecutive rows one 2x2 window, which a fused pool reduces in the
// lane), N = BN output channels, K = 32 channels:
// one v_mfma_f32_16x16x32_bf16 per 16x16 accumulator tile.
//
// Data movement: a ring of NS slots in LDS, slot = [patch pixels x 64 B]
// [9 taps x BN rows x 64 B]; chunk c lives in slot c % NS.  Loads are
// buffer_load_dwordx4 ... lds (global -> LDS, 64 lanes = 1 KiB = 16 rows of
// 64 bytes per instruction): lane l writes row (l >> 2) of its 16-row group
// at 16-byte position (l & 3) and fetches the row's 16-byte chunk
// (l & 3) ^ key(row), so that the rows an MFMA fragment read serves per
// LDS cycle hit distinct banks: weight rows use key = (row >> 1) & 3, patch
// pixels the key of patch_key below.  Patch pixels outside the image (the
// zero padding), outside the tile's source region, or past the patch, and
// weight rows past c_out, are fetched at an offset with bit 31 set, past the
// buffer descriptor's range: the range check returns zeros.  Loads run NS-1
// chunks ahead; every chunk costs one explicit vmcnt wait and one barrier.
// With NS = 1 (one slot) a chunk is loaded, awaited and computed in turn:
// the LDS footprint halves, so two workgroups share a CU and hide each
// other's load latency.  The first chunk's weight rows are issued while the
// tile table is still being decoded (they depend only on the channel
// block).  Weights come as KRSC, or packed per channel block and chunk
// ([c_out/BN][c_in/32][9][BN][32]) so that a chunk's rows are one run.
//
// Epilogue: scale, bias, activation and the fused pool in registers, the
// block's outputs staged in LDS as rows of BN channels, then written as
// 16-byte chunks (each output pixel's BN channels contiguous).
//
// Fused variant (template argument N2 = 32 or 64, BN = c_out = 128, no
// pool): the staged block is the A operand of a following 1x1 convolution
// with N2 outputs, run from LDS in the same workgroup, so the 3x3 layer's
// output never goes to memory; with two input chunks the second one's patch and
// first taps load into a second LDS region while the first is computed.
//
// First-layer variant (template argument PRE, one input chunk of 32
// channels, fused pool): the block's input patch is not loaded from memory
// but computed in the workgroup from the group input, by the 3-channel 3x3
// first layer and its 2x2/2 max-pool (the layer pair before this stage):
// the (2 PR + 2) x (2 PC + 2) pixel input patch is staged in LDS as 8-byte
// pixels, every 2x2 window of first-layer outputs is one 16x16x16 MFMA row
// quad (K = 27 as 3 filter rows x 4 column slots x 4 channel slots, as in
// the stand-alone first-layer kernel, so the values are bit-identical to
// it), and the pooled, activated, bf16-rounded values are written straight
// into the patch rows of the slot in the patch layout (zero outside the
// first layer's output, the zero padding of this stage).  The first layer's
// output never goes to memory.
//
// Requires f = 3, c_in % 32 == 0, c_out % 16 == 0, byte offsets below 2^31
// within a frame's source buffer and within the weights (host-checked);
// even block sizes (compile-time); a fused pool needs even tile origins and
// extents.
#include <hip/hip_runtime.h>

#include "device_util.h"
#include "kernel_args.h"

#ifndef MAFAT_PRE_WAVES
#define MAFAT_PRE_WAVES 1
#endif

namespace mafat {
#ifdef MAFAT_TUNING
// Tuning builds only: phase timestamps (wall clock, 100 MHz) of three
// workgroups (the first, the middle and the last of the grid).
__device__ long long g_patch_trace[3][64];
MAFAT_WG_TRACE_DECL(g_wg_patch)
#define MAFAT_PTRACE(slot_)                                                                      \
  do {                                                                                           \
    if (threadIdx.x == 0 && (slot_) < 64 &&                                                      \
        (blockIdx.x == 0 || blockIdx.x == a.total_blocks / 2 || blockIdx.x == a.total_blocks - 1))         \
      g_patch_trace[blockIdx.x == 0 ? 0 : (blockIdx.x == a.total_blocks - 1 ? 2 : 1)][(slot_)] =      \
          wall_clock64();                                                                        \
  } while (0)
#else
#define MAFAT_PTRACE(slot_) do {} while (0)
#endif
namespace {

typedef __attribute__((address_space(3))) void* lds_ptr_t;

template <int N>
__device__ __forceinline__ void pwait_vmcnt() {
  static_assert(N >= 0 && N <= 63, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}
template <int L, int R>
__device__ __forceinline__ void pwait_stage(int rem) {
  if constexpr (R == 0) {
    pwait_vmcnt<0>();
  } else {
    if (rem >= R) {
      pwait_vmcnt<R * L>();
    } else {
      pwait_stage<L, R - 1>(rem);
    }
  }
}
__device__ __forceinline__ void pbarrier() { asm volatile("s_barrier" ::: "memory"); }

// Byte offset of 16-byte chunk q of 64-byte weight row `row` in a slot region.
__device__ __forceinline__ int swz(int row, int q) { return row * 64 + ((q ^ ((row >> 1) & 3)) << 4); }

// GEMM rows of a block are window-major: every 4 consecutive rows are one
// 2x2 window of the block (block sizes are even), windows row by row.  With
// a fused pool a lane's 4 accumulator rows are then one pool window.
template <int BC>
__device__ __forceinline__ void block_pixel(int r, int* py, int* px) {
  constexpr int WC = BC / 2;  // windows per block row
  const int q = r >> 2, s = r & 3, wy = q / WC;
  *py = 2 * wy + (s >> 1);
  *px = 2 * (q - wy * WC) + (s & 1);
}

// Swizzle key of patch pixel (py, px): 16-byte position p of the pixel's
// 64-byte LDS row holds K chunk p ^ key.  A 16-byte LDS read is served 16
// lanes per cycle from 64 banks, the lanes of one cycle being one half of
// the wave with one parity of lane bits 2-4 (calibrated with the hardware's
// bank-conflict counter); an MFMA fragment read (row l & 15, K chunk l >> 4)
// is conflict-free when the 16 (pixel's LDS row index mod 4, chunk ^ key)
// pairs of each such lane set differ.  With window-major GEMM rows, key = py & 3
// bit-reversed makes every tap's fragment reads conflict-free for blocks
// 8 or 16 pixels wide and leaves 0.75-1.3 extra cycles per 4-cycle read for
// 10-, 12- and 18-wide ones (pixel-major rows with the best key of that form:
// 0 for 16-wide blocks, 2.7-3.6 for the others).
__device__ __forceinline__ int patch_key(int py) { return ((py & 1) << 1) | ((py >> 1) & 1); }

// N2 > 0: a 1x1 convolution with N2 outputs of this stage's output (all BN
// = c_out channels in the block) follows in the same workgroup: the block's
// activated bf16 outputs stay in LDS and are the A operand of a second GEMM
// with its weights (a.w2, [N2][BN]), whose result is the stage's output.
template <int BR, int BC, int BM, int BN, int WGM, int WGN, int NS, bool POOL, int N2 = 0, bool PRE = false>
__global__ __launch_bounds__(64 * WGM * WGN) __attribute__((amdgpu_waves_per_eu(PRE ? MAFAT_PRE_WAVES : 1)))
void conv_patch_kernel(const StageArgs a) {
  if (__builtin_expect(blockIdx.y != 0, 0)) {  // the second grid row: carried band copies (row reuse)
    carried_copies();
    return;
  }
  constexpr int NWAVE = WGM * WGN;
  constexpr int WM = BM / WGM, WN = BN / WGN, MT = WM / 16, NT = WN / 16;
  constexpr int PR = BR + 2, PC = BC + 2;
  constexpr int PPX = (PR * PC + 15) / 16 * 16;  // patch rows (pixels), whole 16-row groups
  constexpr int A_BYTES = PPX * 64;
  constexpr int B_ROWS = 9 * BN;
  constexpr int SLOT = A_BYTES + B_ROWS * 64;
  constexpr int NA = PPX / 16, NB = B_ROWS / 16;  // load instructions per chunk
  constexpr int NAW = (NA + NWAVE - 1) / NWAVE, NBW = (NB + NWAVE - 1) / NWAVE;
  constexpr bool SINK = (NAW * NWAVE != NA) || (NBW * NWAVE != NB);
  constexpr int LPS = NAW + NBW;  // loads per thread per chunk
  static_assert(MT >= 1 && NT >= 1 && MT * 16 == WM && NT * 16 == WN, "wave tile");
  static_assert(BR * BC <= BM && BM % (16 * WGM) == 0, "block rows");
  static_assert(BR % 2 == 0 && BC % 2 == 0, "blocks cover whole 2x2 windows (window-major GEMM rows)");
  static_assert(NS >= 1 && NS <= 6 && (NS - 2) * LPS <= 63, "ring depth");
  // Fused variant (N2 > 0): the 1x1 weights in their own LDS region past
  // the ring, then a second region Y for the second chunk's patch and the
  // weights of its first YT taps (instruction k of a chunk's weight part is
  // tap k here), loaded while the first chunk is computed.
  constexpr int W2D = NS * SLOT + (SINK ? 1024 : 0);
  constexpr int YT = 5;
  constexpr int YOFF = W2D + N2 * BN * 2;
  static_assert(N2 == 0 || (NS == 1 && NBW == 9 && NB == 9 * NWAVE), "fused variant: one slot, a tap per instruction");
  // First-layer variant (PRE): one slot and nothing past it.  The weight
  // rows of taps 0-4 load during the tile decode; while the first layer
  // runs, the space of taps 5-8 holds the input patch (IR x IC pixels of 8
  // bytes, rows IRS bytes apart), the first layer's weights (32 x 27 bf16),
  // its scale and bias (32 floats each) and a table of the patch pixels
  // (see below); taps 5-8 load there once the first layer is done, while
  // taps 0-4 are computed.  52 KiB: three workgroups per CU.
  constexpr int IR = 2 * PR + 2, IC = 2 * PC + 2, IRS = IC * 8 + 16;
  constexpr int C0 = 32;                               // first-layer outputs = this stage's c_in
  constexpr int G5 = 5 * BN / 16;                      // weight load instructions of taps 0-4
  constexpr int XOFF = A_BYTES + 5 * BN * 64;          // input patch (where taps 5-8 go later)
  constexpr int W0OFF = XOFF + IR * IRS;               // first-layer weights
  constexpr int SB0OFF = W0OFF + (C0 * 27 * 2 + 15) / 16 * 16;  // scale, bias
  constexpr int QTOFF = SB0OFF + 2 * C0 * 4;           // patch pixel table
  constexpr int PRE_END = QTOFF + PR * PC * 4;
  static_assert(!PRE || (NS == 1 && N2 == 0 && POOL && PRE_END <= SLOT && (5 * BN) % 16 == 0),
                "first-layer variant: one slot, a fused pool, its staging inside the slot");
  constexpr int SMEM = PRE ? SLOT : YOFF + (N2 > 0 ? A_BYTES + YT * BN * 64 : 0);
  __shared__ __align__(1024) unsigned char smem[SMEM];
  static_assert(N2 == 0 || (!POOL && BM == BR * BC && N2 % 16 == 0 && BN % 32 == 0),
                "fused 1x1: no pool, no padding rows");
  // Fused 1x1: its weights ([N2][BN] bf16) go straight to LDS now (rows of
  // BN = 128 channels, 16-byte piece q of row r at slot q ^ (r & 15), so
  // the 16 rows of a fragment read fall in different banks); its scale and
  // bias are fetched into registers.  The second GEMM's waves: WC2 along
  // its channels (CT2 16-channel tiles each) times WP2 along the block's
  // pixels (PG2 16-pixel groups).
  constexpr int WC2 = 2, WP2 = WGM * WGN / WC2;
  constexpr int CT2 = N2 > 0 ? N2 / 16 / WC2 : 1, PG2 = BM / 16 / WP2;
  static_assert(N2 == 0 || (N2 % (16 * WC2) == 0 && (BM / 16) % WP2 == 0 && BN == 128 &&
                            (N2 * BN * 2) % (1024 * WGM * WGN) == 0), "second GEMM");
  float sc2[CT2][4], bi2[CT2][4];
  if constexpr (N2 > 0) {
    const int w0 = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) >> 6);
    const int l0 = static_cast<int>(threadIdx.x) & 63;
    const __amdgpu_buffer_rsrc_t rs2 = make_rsrc(a.w2, static_cast<unsigned>(N2 * BN * 2));
#pragma unroll
    for (int k = 0; k < N2 * BN * 2 / (1024 * WGM * WGN); ++k) {
      const int e = (k * WGM * WGN + w0) * 64 + l0;  // LDS slot of this lane's piece
      const int r = e >> 4, q = (e & 15) ^ (r & 15);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs2, (lds_ptr_t)(smem + W2D + (k * WGM * WGN + w0) * 1024), 16,
                                               (r * 16 + q) * 16, 0, 0, 0);
    }
    const int wc = w0 % WC2;
#pragma unroll
    for (int j = 0; j < CT2; ++j) {
      const int c2 = (wc * CT2 + j) * 16 + 4 * (l0 >> 4);
      const f32x4 s4 = *reinterpret_cast<const f32x4*>(a.scale2 + c2);
      const f32x4 b4 = *reinterpret_cast<const f32x4*>(a.bias2 + c2);
#pragma unroll
      for (int r = 0; r < 4; ++r) { sc2[j][r] = s4[r]; bi2[j][r] = b4[r]; }
    }
  }

  // First-layer variant: its weights, scale and bias (the same for every
  // workgroup, one 16-byte piece per thread) are fetched before the tile
  // table is decoded and written to LDS with the input patch.
  constexpr int W0P = C0 * 27 * 2 / 16;  // 16-byte pieces of the first layer's weights
  static_assert(!PRE || (W0P + C0 / 2 <= 64 * WGM * WGN), "one piece per thread");
  u32x4 pre_v = u32x4{0u, 0u, 0u, 0u};
  if constexpr (PRE) {
    const int t0 = static_cast<int>(threadIdx.x);
    const u32x4* ps = (t0 < W0P)              ? reinterpret_cast<const u32x4*>(a.w0) + t0
                      : (t0 < W0P + C0 / 4)   ? reinterpret_cast<const u32x4*>(a.scale0) + (t0 - W0P)
                      : (t0 < W0P + C0 / 2)   ? reinterpret_cast<const u32x4*>(a.bias0) + (t0 - W0P - C0 / 4)
                                              : nullptr;
    if (ps) pre_v = *ps;
  }

  MAFAT_PTRACE(0);
  MAFAT_WG_MARK(g_wg_patch, 0);
  const int tid = static_cast<int>(threadIdx.x), lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lrow = lane >> 2, lpos = lane & 3;
  const int cin = a.cin, cout = a.cout;
  const int K = 9 * cin;
  // Weights: KRSC, or packed per channel block and chunk ([cout/BN][cin/32]
  // [9][BN][32], rows past c_out zero), where a chunk's BN x 9 rows are one
  // contiguous run (whole lines for the 16-row load instructions).
  const int nchunk = cin >> 5;
  const bool wpk = a.w_packed != 0;
  const __amdgpu_buffer_rsrc_t rsb =
      make_rsrc(a.w, static_cast<unsigned>(wpk ? a.nblk_n * nchunk * 9 * BN * 64 : cout * K * 2));
  const unsigned bstride = wpk ? static_cast<unsigned>(9 * BN * 64) : 64u;  // bytes from one chunk to the next
  // Weight loads: instruction g of a chunk's weight part fills weight rows
  // [16 g, 16 g + 16) of the slot (row = tap * BN + n); g past NB fills the
  // sink.  Chunk c adds 64 c bytes.
  unsigned b_off[NBW];
  auto issue_b = [&](int c, int slot) {
    unsigned char* sl = smem + slot * SLOT;
    const unsigned coff = static_cast<unsigned>(c) * bstride;
#pragma unroll
    for (int k = 0; k < NBW; ++k) {
      const int g = k * NWAVE + wave;
      unsigned char* d = (g < NB) ? sl + A_BYTES + g * 1024 : smem + NS * SLOT;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsb, (lds_ptr_t)d, 16,
                                               static_cast<int>(b_off[k] + coff), 0, 0, 0);
    }
  };
  // The weight rows depend only on the channel block: their first chunk is
  // issued while the tile table is still on its way.
  auto early = [&](int nb) {
    const int n0e = nb * BN;
#pragma unroll
    for (int k = 0; k < NBW; ++k) {
      const int g = k * NWAVE + wave;
      const int row = 16 * g + lrow;           // weight row within the slot
      const int t = row / BN, n = row - t * BN;
      const int co = n0e + n;
      const int chunk = lpos ^ ((row >> 1) & 3);
      if (wpk)
        b_off[k] = (g < NB) ? static_cast<unsigned>(((nb * nchunk) * 9 * BN + row) * 64 + chunk * 16) : 0x80000000u;
      else
        b_off[k] = (g < NB && co < cout) ? static_cast<unsigned>((co * K + t * cin) * 2 + chunk * 16)
                                         : 0x80000000u;
    }
    if constexpr (PRE) {  // taps 0-4 only (their rows: instructions g < G5)
#pragma unroll
      for (int k = 0; k < NBW; ++k) {
        const int g = k * NWAVE + wave;
        if (g < G5)
          __builtin_amdgcn_raw_ptr_buffer_load_lds(rsb, (lds_ptr_t)(smem + A_BYTES + g * 1024), 16,
                                                   static_cast<int>(b_off[k]), 0, 0, 0);
      }
    } else {
      issue_b(0, 0);
    }
  };
  KTile tl;
  const BlockPos bp = decode_block(a, &tl, early);
  MAFAT_PTRACE(1 + (tl.ch < -1 ? 1 : 0));
  const int wm = wave / WGN, wn = wave - wm * WGN;
  const int nbx = (tl.cw + BC - 1) / BC;
  const int bby = bp.mb / nbx, bbx = bp.mb - bby * nbx;
  const int by0 = tl.cy0 + bby * BR, bx0 = tl.cx0 + bbx * BC;  // block origin (conv outputs)
  const int n0 = bp.nb * BN;
  const int sw = tl.sw;
  const int64_t sbase = bp.frame * a.src_fstride + tl.src_off;
  uint16_t* dst = static_cast<uint16_t*>(a.dst) + bp.frame * a.dst_fstride + tl.dst_off;
  const int nstage = cin >> 5;
  const __amdgpu_buffer_rsrc_t rsa = make_rsrc(static_cast<const uint16_t*>(a.src) + sbase,
                                               static_cast<unsigned>((a.src_fstride - tl.src_off) * 2));

  // Scale and bias of this lane's output channels.
  float sc[NT][4], bi[NT][4];
#pragma unroll
  for (int j = 0; j < NT; ++j) {
    if (POOL) {
      const int co = n0 + wn * WN + j * 16 + (lane & 15);
      const int cc = co < cout ? co : 0;
      sc[j][0] = a.scale[cc];
      bi[j][0] = a.bias[cc];
    } else {
      const int co = n0 + wn * WN + j * 16 + 4 * (lane >> 4);
      const int cc = co < cout ? co : 0;
      const f32x4 s4 = *reinterpret_cast<const f32x4*>(a.scale + cc);
      const f32x4 b4 = *reinterpret_cast<const f32x4*>(a.bias + cc);
#pragma unroll
      for (int r = 0; r < 4; ++r) { sc[j][r] = s4[r]; bi[j][r] = b4[r]; }
    }
  }

  // This lane's patch loads (chunk 0; chunk c adds 64 c bytes): instruction
  // g of a chunk's patch part fills patch rows [16 g, 16 g + 16); g past NA
  // fills the sink.
  // Source region of the tile: the conv outputs [cy0, cy0 + ch) read rows
  // [cy0 - 1, cy0 + ch] (columns likewise), clipped to the image.
  const int ry0 = max(tl.cy0 - 1, 0), ry1 = min(tl.cy0 + tl.ch + 1, a.in_h);
  const int rx0 = max(tl.cx0 - 1, 0), rx1 = min(tl.cx0 + tl.cw + 1, a.in_w);
  unsigned a_off[NAW];
#pragma unroll
  for (int k = 0; k < NAW; ++k) {
    const int g = k * NWAVE + wave;
    const int p = 16 * g + lrow;
    const int py = p / PC, px = p - (p / PC) * PC;
    const int iy = by0 - 1 + py, ix = bx0 - 1 + px;
    const bool ok = g < NA && p < PR * PC && iy >= ry0 && iy < ry1 && ix >= rx0 && ix < rx1;
    const int chunk = lpos ^ patch_key(py);
    a_off[k] = ok ? static_cast<unsigned>((((iy - tl.sy0) * sw + (ix - tl.sx0)) * cin) * 2 + chunk * 16)
                  : 0x80000000u;
  }
  auto issue_a = [&](int c, int slot) {
    unsigned char* sl = smem + slot * SLOT;
    const unsigned coff = static_cast<unsigned>(c * 64);
#pragma unroll
    for (int k = 0; k < NAW; ++k) {
      const int g = k * NWAVE + wave;
      unsigned char* d = (g < NA) ? sl + g * 1024 : smem + NS * SLOT;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsa, (lds_ptr_t)d, 16,
                                               static_cast<int>(a_off[k] + coff), 0, 0, 0);
    }
  };
  // A chunk's loads (chunk 0's weight part was issued during the decode).
  auto issue = [&](int c, int slot) {
    issue_a(c, slot);
    if (c > 0) issue_b(c, slot);
  };

  // Fragment reads.  A: lane l supplies GEMM row wm*WM + 16 i + (l & 15),
  // i.e. block pixel (py, px), as patch row (py + ky) * PC + (px + kx) at
  // 16-byte chunk q = l >> 4 (K elements 8q .. 8q+7 of the 32).  B: weight
  // row tap * BN + wn*WN + 16 j + (l & 15), chunk q.
  const int q = lane >> 4;
  // Per fragment: byte offset of the lane's patch pixel (tap (0, 0)) and its
  // K chunk XOR the swizzle key for each tap row.  A padding row (past the
  // block's pixels; its result is discarded) reads the pixel of row r ^ 12,
  // a row served in the same LDS cycle (a broadcast, no conflict), or pixel 0.
  int pb[MT], kq3[MT][3];
#pragma unroll
  for (int i = 0; i < MT; ++i) {
    int r = wm * WM + i * 16 + (lane & 15);
    r = (r < BR * BC) ? r : (((r ^ 12) < BR * BC) ? (r ^ 12) : 0);
    int py, px;
    block_pixel<BC>(r, &py, &px);
    pb[i] = (py * PC + px) * 64;
#pragma unroll
    for (int d = 0; d < 3; ++d) kq3[i][d] = q ^ patch_key(py + d);
  }
  const int rb = wn * WN + (lane & 15);
  const int b_lane = A_BYTES + swz(rb, q);  // (tap * BN + 16 j) rows later: same swizzle

  f32x4 acc[NT][MT];
#pragma unroll
  for (int j = 0; j < NT; ++j)
#pragma unroll
    for (int i = 0; i < MT; ++i) acc[j][i] = f32x4{0.f, 0.f, 0.f, 0.f};

  // Nine taps per chunk, software-pipelined: the fragments of tap t + 1 are
  // read from LDS (into the other register set) before the MFMAs of tap t
  // are issued, and a scheduling barrier keeps the compiler from
  // interleaving them, so each tap's LDS latency hides behind the previous
  // tap's MFMAs.  A chunk's patch is read at spa, its weight rows at spb
  // (the same slot, except in the fused variant's split second chunk).
  auto load_frags = [&](const unsigned char* spa, const unsigned char* spb, int t, u32x4 (&af)[MT],
                        u32x4 (&bfr)[NT]) {
    const int ty = t / 3, tx = t % 3;
#pragma unroll
    for (int i = 0; i < MT; ++i)
      af[i] = *reinterpret_cast<const u32x4*>(spa + pb[i] + (ty * PC + tx) * 64 +
                                              ((kq3[i][ty] & 3) << 4));
#pragma unroll
    for (int j = 0; j < NT; ++j)
      bfr[j] = *reinterpret_cast<const u32x4*>(spb + b_lane + (t * BN + j * 16) * 64);
  };
  auto mfmas = [&](const u32x4 (&af)[MT], const u32x4 (&bfr)[NT]) {
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int j = 0; j < NT; ++j) {
        if constexpr (POOL) mma<MAFAT_BF16>(acc[j][i], af[i], bfr[j]);
        else mma<MAFAT_BF16>(acc[j][i], bfr[j], af[i]);
      }
  };
  // Taps [T0, T1) of one chunk (T0, T1 as std::integral_constant).
  auto taps = [&](const unsigned char* spa, const unsigned char* spb, auto t0c, auto t1c) {
    constexpr int T0 = decltype(t0c)::value, T1 = decltype(t1c)::value;
    u32x4 af0[MT], bf0[NT], af1[MT], bf1[NT];
    load_frags(spa, spb, T0, af0, bf0);
#pragma unroll
    for (int t = T0; t < T1; t += 2) {
      if (t + 1 < T1) load_frags(spa, spb, t + 1, af1, bf1);
      __builtin_amdgcn_sched_barrier(0);
      mfmas(af0, bf0);
      __builtin_amdgcn_sched_barrier(0);
      if (t + 1 < T1) {
        if (t + 2 < T1) load_frags(spa, spb, t + 2, af0, bf0);
        __builtin_amdgcn_sched_barrier(0);
        mfmas(af1, bf1);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  };
  using I0 = std::integral_constant<int, 0>;
  using I9 = std::integral_constant<int, 9>;
  auto compute = [&](int slot) {
    const unsigned char* sp = smem + slot * SLOT;
    taps(sp, sp, I0{}, I9{});
  };

  if constexpr (PRE) {
    // The block's input patch = the pooled first-layer outputs at patch
    // pixels (py, px) <-> first-layer output (by0 - 1 + py, bx0 - 1 + px),
    // i.e. first-layer conv outputs 2 (by0 - 1) + [0, 2 PR) (rows; columns
    // likewise), i.e. group-input pixels starting one row/column earlier.
    const int gy0 = 2 * (by0 - 1) - 1, gx0 = 2 * (bx0 - 1) - 1;  // input patch origin
    // Group-input rows and columns this tile's first-layer outputs read:
    // its pooled region [cy0 - 1, cy0 + ch + 1) of this stage's input
    // (clipped to it), doubled, widened by the 3x3 window, clipped to the
    // image.  Pixels outside read as zero, like the stand-alone kernel's.
    const int ylo = max(0, 2 * ry0 - 1), yhi = min(a.in_h0, 2 * ry1 + 1);
    const int xlo = max(0, 2 * rx0 - 1), xhi = min(a.in_w0, 2 * rx1 + 1);
    const int64_t sb0 = bp.frame * a.src_fstride + tl.src_off;  // elements (3 per pixel)
    const int bpar = static_cast<int>(sb0 & 1);
    const __amdgpu_buffer_rsrc_t rs0 = make_rsrc(static_cast<const uint16_t*>(a.src) + sb0,
                                                 static_cast<unsigned>((a.src_fstride - tl.src_off) * 2));
    constexpr int NPX0 = IR * IC;
    constexpr int NTH = 64 * NWAVE;
    constexpr int NPT0 = (NPX0 + NTH - 1) / NTH;
    uint32_t la[NPT0], lb[NPT0];
    bool lodd[NPT0];
#pragma unroll
    for (int k = 0; k < NPT0; ++k) {  // one pixel (6 bytes): an aligned 4-byte and a 2-byte load
      const int e = tid + NTH * k;
      const int r = e / IC, c = e - r * IC;
      const int iy = gy0 + r, ix = gx0 + c;
      const bool ok = e < NPX0 && iy >= ylo && iy < yhi && ix >= xlo && ix < xhi;
      const int pp = (iy - tl.sy0) * tl.sw + (ix - tl.sx0);
      const bool odd = ((bpar + pp) & 1) != 0;  // c0 at an address = 2 (mod 4): the dword holds c1, c2
      const unsigned off = static_cast<unsigned>(pp * 6);
      la[k] = __builtin_amdgcn_raw_buffer_load_b32(rs0, static_cast<int>(ok ? (odd ? off + 2u : off) : 0x80000000u),
                                                   0, 0);
      lb[k] = __builtin_amdgcn_raw_buffer_load_b16(rs0, static_cast<int>(ok ? (odd ? off : off + 4u) : 0x80000000u),
                                                   0, 0);
      lodd[k] = odd;
    }
    // Patch pixel table, one entry per MFMA row of the first-layer loop
    // (tiles of 4 patch pixels, NIT per wave): entry q = (qy, qx), bits
    // 0-15 the LDS offset of its first-layer window (input patch row 2 qy,
    // column 2 qx), bits 16-31 where its pooled values go: the patch row
    // (64 q) with its swizzle key (window-major rows) in bits 4-5, or,
    // for a pixel outside this stage's input (zero padding) or past the
    // patch, a dummy row (the patch is zeroed first, so padding reads 0).
    constexpr int NQ = PR * PC;            // patch pixels
    constexpr int NG = (NQ + 3) / 4;       // MFMA row tiles (4 patch pixels each)
    constexpr int NIT = (NG + NWAVE - 1) / NWAVE;  // tiles per wave (the last one may run past NG)
    constexpr int NQT = NIT * NWAVE * 4;   // table entries
    constexpr int DUMMY = (QTOFF + NQT * 4 + 63) / 64 * 64;  // a 64-byte dummy patch row
    static_assert(XOFF + 2 * (PR - 1) * IRS + 2 * (PC - 1) * 8 < 65536 && DUMMY + 64 <= SLOT && DUMMY < 65536,
                  "table fields and dummy row");
    static_assert(NQT <= 64 * NWAVE, "one table entry per thread");
    if (tid < NQT) {
      const int qy = tid / PC, qx = tid - (tid / PC) * PC;
      const int gy = by0 - 1 + qy, gx = bx0 - 1 + qx;
      const bool store = tid < NQ && gy >= 0 && gy < a.in_h && gx >= 0 && gx < a.in_w;
      const unsigned row = store ? static_cast<unsigned>(tid * 64 + (patch_key(qy) << 4))
                                 : static_cast<unsigned>(DUMMY);
      const unsigned e = static_cast<unsigned>(XOFF + 2 * min(qy, PR - 1) * IRS + 2 * qx * 8) | (row << 16);
      *reinterpret_cast<unsigned*>(smem + QTOFF + tid * 4) = e;
    }
    // zero the patch (padding pixels keep it)
    for (int k = tid; k < A_BYTES / 16; k += 64 * NWAVE)
      *reinterpret_cast<u32x4*>(smem + k * 16) = u32x4{0u, 0u, 0u, 0u};
    if (tid < W0P)
      *reinterpret_cast<u32x4*>(smem + W0OFF + tid * 16) = pre_v;
    else if (tid < W0P + C0 / 2)  // scale (C0 floats), then bias
      *reinterpret_cast<u32x4*>(smem + SB0OFF + (tid - W0P) * 16) = pre_v;
    typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
#pragma unroll
    for (int k = 0; k < NPT0; ++k) {
      const int e = tid + NTH * k;
      const int r = e / IC, c = e - r * IC;
      const uint32_t b16 = lb[k] & 0xffffu;
      const u32x2 v = lodd[k] ? u32x2{b16 | (la[k] << 16), la[k] >> 16} : u32x2{la[k], b16};
      if (e < NPX0) *reinterpret_cast<u32x2*>(smem + XOFF + r * IRS + c * 8) = v;
    }
    __syncthreads();
    MAFAT_PTRACE(6);

    // First layer on the matrix cores: 16x16x16 MFMAs, A = 16 first-layer
    // outputs (4 pool windows = 4 patch pixels, window-major), B = 16
    // channels, K = (kx slot, channel slot) for one filter row.  Lane l
    // supplies output pixel l & 15 at kx slot l >> 4 (slot 3: zero weights).
    typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
    const int kq = lane >> 4, kx = min(kq, 2), pl = lane & 15;
    const uint16_t* sw0 = reinterpret_cast<const uint16_t*>(smem + W0OFF);
    const float* ssb0 = reinterpret_cast<const float*>(smem + SB0OFF);
    const unsigned* qtab = reinterpret_cast<const unsigned*>(smem + QTOFF);
    u32x2 wf[C0 / 16][3];
    float sc0[C0 / 16], bi0[C0 / 16];
    bool neg = false;
#pragma unroll
    for (int j = 0; j < C0 / 16; ++j) {
#pragma unroll
      for (int ky = 0; ky < 3; ++ky) {
        const int wr = (16 * j + pl) * 27 + ky * 9 + 3 * kx;
        const uint32_t w0 = sw0[wr], w1 = sw0[wr + 1], w2 = sw0[wr + 2];
        wf[j][ky] = kq < 3 ? u32x2{w0 | (w1 << 16), w2} : u32x2{0u, 0u};
      }
      sc0[j] = ssb0[16 * j + pl];
      bi0[j] = ssb0[C0 + 16 * j + pl];
      neg = neg || !(sc0[j] >= 0.f);
    }
    // With a non-negative scale, v -> fma(v, s, b) is non-decreasing, so the
    // window maximum may be taken before the scale (the same value: rounding
    // keeps the order); otherwise (some scale of the wave negative or NaN)
    // every element is scaled first.
    const float slope0 = act_slope(a.act0);
    const int lx = ((pl & 3) >> 1) * IRS + ((pl & 1) + kx) * 8;  // this lane's place in a window
    // this lane's part of a pooled value's store address: chunk (c >> 3) of
    // channel c = 16 j + pl at bits 4-5 (XOR the pixel's key), c & 7 below
    const unsigned sx = static_cast<unsigned>((pl >> 3) << 4), so = static_cast<unsigned>((pl & 7) * 2);
    // A fixed trip count, unrolled and free of branches, so that the
    // compiler can issue the next tiles' table and patch reads while the
    // current tile's MFMAs run; the sign test of the scales is hoisted out.
    auto first_layer = [&](auto negc) {
      constexpr bool NEG = decltype(negc)::value;
#pragma unroll
      for (int it = 0; it < NIT; ++it) {
        const int t = wave + NWAVE * it;
        const unsigned eq = qtab[4 * t + (pl >> 2)];  // operand row: patch pixel 4 t + (pl >> 2), window position pl & 3
        const unsigned eo = qtab[4 * t + kq];         // results: the window of patch pixel 4 t + kq
        const unsigned char* xp = smem + (eq & 0xffffu) + lx;
        u32x2 xf[3];
#pragma unroll
        for (int ky = 0; ky < 3; ++ky) xf[ky] = *reinterpret_cast<const u32x2*>(xp + ky * IRS);
        const unsigned a0 = ((eo >> 16) ^ sx) + so;  // channel tile j = 0; j = 1 is chunk ^ 2
#pragma unroll
        for (int j = 0; j < C0 / 16; ++j) {
          f32x4 acc0 = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int ky = 0; ky < 3; ++ky)
            acc0 = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(bf16x4, xf[ky]),
                                                            __builtin_bit_cast(bf16x4, wf[j][ky]), acc0, 0, 0, 0);
          float m;
          if constexpr (!NEG) {
            m = fmaf(fmaxf(fmaxf(acc0[0], acc0[1]), fmaxf(acc0[2], acc0[3])), sc0[j], bi0[j]);
          } else {
            float v[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) v[r] = fmaf(acc0[r], sc0[j], bi0[j]);
            m = fmaxf(fmaxf(v[0], v[1]), fmaxf(v[2], v[3]));
          }
          m = fmaxf(m, slope0 * m);
          store1(reinterpret_cast<uint16_t*>(smem + (a0 ^ static_cast<unsigned>(32 * j))), m);
        }
      }
    };
    if (__builtin_amdgcn_ballot_w64(neg) != 0)
      first_layer(std::true_type{});
    else
      first_layer(std::false_type{});
    MAFAT_PTRACE(7);
    pbarrier();  // every wave is done with the input patch: taps 5-8 load over it
#pragma unroll
    for (int k = 0; k < NBW; ++k) {
      const int g = k * NWAVE + wave;
      if (g >= G5 && g < NB)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rsb, (lds_ptr_t)(smem + A_BYTES + g * 1024), 16,
                                                 static_cast<int>(b_off[k]), 0, 0, 0);
    }
    MAFAT_PTRACE(8);
    using I5 = std::integral_constant<int, 5>;
    taps(smem, smem, I0{}, I5{});  // taps 0-4 (their rows were in before the first layer started)
    pwait_vmcnt<0>();
    pbarrier();
    MAFAT_PTRACE(9);
    taps(smem, smem, I5{}, I9{});
  } else if constexpr (N2 > 0) {
    if (nstage == 2) {
      // Two chunks, the second one's loads overlapped with compute: its
      // patch and first YT taps go to Y at once, its last taps to the
      // slot once the first chunk is done with it.
      auto issue_b_taps = [&](unsigned char* sl, auto k0c, auto k1c) {
#pragma unroll
        for (int k = decltype(k0c)::value; k < decltype(k1c)::value; ++k)
          __builtin_amdgcn_raw_ptr_buffer_load_lds(rsb, (lds_ptr_t)(sl + A_BYTES + (k * NWAVE + wave) * 1024), 16,
                                                   static_cast<int>(b_off[k] + bstride), 0, 0, 0);
      };
      unsigned char* const Y = smem + YOFF;
      using IY = std::integral_constant<int, YT>;
      issue_a(0, 0);                     // chunk 0's weights are on their way already
      {                                  // chunk 1: patch and taps [0, YT) to Y
        const unsigned coff = 64u;
#pragma unroll
        for (int k = 0; k < NAW; ++k) {
          const int g = k * NWAVE + wave;
          unsigned char* d = (g < NA) ? Y + g * 1024 : smem + NS * SLOT;
          __builtin_amdgcn_raw_ptr_buffer_load_lds(rsa, (lds_ptr_t)d, 16, static_cast<int>(a_off[k] + coff), 0, 0, 0);
        }
        issue_b_taps(Y, I0{}, IY{});
      }
      pwait_vmcnt<NAW + YT>();           // chunk 0 is in
      pbarrier();
      MAFAT_PTRACE(8);
      taps(smem, smem, I0{}, I9{});
      pbarrier();                        // every wave is done with the slot
      issue_b_taps(smem, IY{}, I9{});    // chunk 1, taps [YT, 9), to the slot
      pwait_vmcnt<9 - YT>();             // chunk 1's patch and first taps are in
      pbarrier();
      MAFAT_PTRACE(9);
      taps(Y, Y, I0{}, IY{});
      pwait_vmcnt<0>();
      pbarrier();
      MAFAT_PTRACE(10);
      taps(Y, smem, IY{}, I9{});
    } else {
      for (int s = 0; s < nstage; ++s) {
        if (s > 0) pbarrier();
        issue(s, 0);
        pwait_vmcnt<0>();
        pbarrier();
        compute(0);
      }
    }
  } else if constexpr (NS == 1) {
    // One slot (half the LDS, so two workgroups fit on a CU and hide each
    // other's load latency): load a chunk, wait, compute, repeat.
    for (int s = 0; s < nstage; ++s) {
      if (s > 0) pbarrier();  // every wave is done reading the slot
      issue(s, 0);
      pwait_vmcnt<0>();
      pbarrier();
      MAFAT_PTRACE(8 + s);
      compute(0);
    }
  } else {
#pragma unroll
    for (int p = 0; p < NS - 1; ++p)
      if (p < nstage) issue(p, p);
    int slot = 0;
    for (int s = 0; s < nstage; ++s) {
      pwait_stage<LPS, NS - 2>(nstage - 1 - s);
      pbarrier();
      MAFAT_PTRACE(8 + s);
      if (s + NS - 1 < nstage) issue(s + NS - 1, slot == 0 ? NS - 1 : slot - 1);
      compute(slot);
      slot = (slot == NS - 1) ? 0 : slot + 1;
    }
  }

  MAFAT_PTRACE(4);
  // Epilogue: folded batch-norm, activation (leaky: max(v, 0.1 v)), the
  // fused pool, round to bf16; the block's outputs are staged in LDS (the
  // ring is free by now) as rows of BN channels per output pixel and leave
  // as 16-byte stores, each pixel's BN channels one contiguous run (whole
  // cache lines instead of 8- or 2-byte pieces from every lane).  Only the
  // pixels inside the tile's computed rectangle are stored.
  constexpr int NTHR = 64 * NWAVE;
  constexpr int RSB = BN * 2 + 16;                       // LDS bytes per staged pixel row
  constexpr int NPXO = POOL ? (BR / 2) * (BC / 2) : BR * BC;  // output pixels of the block
  constexpr int CPB = BN / 8;                             // 16-byte chunks per pixel row
  static_assert(NPXO * RSB <= NS * SLOT, "staged block fits in the ring");
  const float slope = act_slope(a.act);
  __syncthreads();  // every wave is done reading the ring
#pragma unroll
  for (int i = 0; i < MT; ++i) {
#pragma unroll
    for (int j = 0; j < NT; ++j) {
      if (POOL) {
        const int r = wm * WM + i * 16 + 4 * (lane >> 4);  // first GEMM row of this lane's window
        float v[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) v[k] = fmaf(acc[j][i][k], sc[j][0], bi[j][0]);
        float mx = fmaxf(fmaxf(v[0], v[1]), fmaxf(v[2], v[3]));
        mx = fmaxf(mx, slope * mx);
        if (r < BR * BC)
          store1(reinterpret_cast<uint16_t*>(smem + (r >> 2) * RSB) + wn * WN + j * 16 + (lane & 15), mx);
      } else {
        const int r = wm * WM + i * 16 + (lane & 15);
        int py, px;
        block_pixel<BC>(r, &py, &px);  // staged at the pixel's row-major index
        float v[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          v[k] = fmaf(acc[j][i][k], sc[j][k], bi[j][k]);
          v[k] = fmaxf(v[k], slope * v[k]);
        }
        if (r < BR * BC)
          store4<MAFAT_BF16>(reinterpret_cast<uint16_t*>(smem + (py * BC + px) * RSB) + wn * WN + j * 16 +
                                 4 * (lane >> 4),
                             v);
      }
    }
  }
  const int vy = tl.cy0 + tl.ch - by0, vx = tl.cx0 + tl.cw - bx0;  // valid extent of this block
  if constexpr (N2 > 0) {
    // Second GEMM, in LDS: out[p][c2] = sum_c act(stage)[p][c] w2[c2][c];
    // the results replace the staged rows once every wave has read them.
    MAFAT_PTRACE(16);
    __syncthreads();  // the staged rows are complete (the weights arrived before the first chunk)
    MAFAT_PTRACE(17);
    const int wp = wave / WC2, wc = wave - (wave / WC2) * WC2;
    f32x4 acc2[PG2][CT2];
#pragma unroll
    for (int i = 0; i < PG2; ++i)
#pragma unroll
      for (int j = 0; j < CT2; ++j) acc2[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int ra = ((wp * PG2) * 16 + (lane & 15)) * RSB + 16 * (lane >> 4);
    const int rb2 = W2D + ((wc * CT2) * 16 + (lane & 15)) * (BN * 2);
#pragma unroll
    for (int k0 = 0; k0 < BN; k0 += 32) {
      u32x4 av[PG2], bv[CT2];
#pragma unroll
      for (int i = 0; i < PG2; ++i) av[i] = *reinterpret_cast<const u32x4*>(smem + ra + i * 16 * RSB + k0 * 2);
#pragma unroll
      for (int j = 0; j < CT2; ++j)
        bv[j] = *reinterpret_cast<const u32x4*>(smem + rb2 + j * 16 * (BN * 2) +
                                                (((k0 >> 3) + (lane >> 4)) ^ (lane & 15)) * 16);
#pragma unroll
      for (int i = 0; i < PG2; ++i)
#pragma unroll
        for (int j = 0; j < CT2; ++j) mma<MAFAT_BF16>(acc2[i][j], bv[j], av[i]);
    }
    MAFAT_PTRACE(18);
    __syncthreads();  // every wave is done reading the staged rows
    // a lane's results: channels 16 j' + 4 (lane >> 4) .. + 3 of pixel
    // 16 i' + (lane & 15) (i', j' the global group and tile)
    const float slope2 = act_slope(a.act2);
#pragma unroll
    for (int i = 0; i < PG2; ++i)
#pragma unroll
      for (int j = 0; j < CT2; ++j) {
        float v[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          v[r] = fmaf(acc2[i][j][r], sc2[j][r], bi2[j][r]);
          v[r] = fmaxf(v[r], slope2 * v[r]);
        }
        store4<MAFAT_BF16>(reinterpret_cast<uint16_t*>(smem + ((wp * PG2 + i) * 16 + (lane & 15)) * RSB) +
                               (wc * CT2 + j) * 16 + 4 * (lane >> 4), v);
      }
    __syncthreads();
    MAFAT_PTRACE(19);
    constexpr int CPB2 = N2 / 8;
    for (int e = tid; e < NPXO * CPB2; e += NTHR) {
      const int p = e / CPB2, k = e - p * CPB2;
      const int py = p / BC, px = p - py * BC;
      if (py < vy && px < vx) {
        const u32x4 v = *reinterpret_cast<const u32x4*>(smem + p * RSB + k * 16);
        *reinterpret_cast<u32x4*>(dst + ((by0 + py - tl.dy0) * tl.dw + (bx0 + px - tl.dx0)) * N2 + k * 8) = v;
      }
    }
    MAFAT_PTRACE(5);
    MAFAT_WG_MARK(g_wg_patch, 1);
    return;
  }
  __syncthreads();
  for (int e = tid; e < NPXO * CPB; e += NTHR) {
    const int p = e / CPB, k = e - p * CPB;
    int oy, ox;
    bool ok;
    if (POOL) {
      constexpr int WC = BC / 2;
      const int wy = p / WC, wx = p - wy * WC;
      ok = 2 * wy < vy && 2 * wx < vx;
      oy = (by0 + 2 * wy) >> 1;
      ox = (bx0 + 2 * wx) >> 1;
    } else {
      const int py = p / BC, px = p - py * BC;
      ok = py < vy && px < vx;
      oy = by0 + py;
      ox = bx0 + px;
    }
    const int c0 = n0 + k * 8;
    if (ok && c0 < cout) {
      const u32x4 v = *reinterpret_cast<const u32x4*>(smem + p * RSB + k * 16);
      *reinterpret_cast<u32x4*>(dst + ((oy - tl.dy0) * tl.dw + (ox - tl.dx0)) * cout + c0) = v;
    }
  }
  MAFAT_PTRACE(5);
  MAFAT_WG_MARK(g_wg_patch, 1);
}

template <bool POOL>
hipError_t launch_patch_p(const MfmaShape& sh, const StageArgs& args, hipStream_t stream, LaunchEvents ev) {
  const dim3 grid(static_cast<unsigned>(args.total_blocks), args.copy_blocks > 0 ? 2u : 1u);
#define MAFAT_PATCH(br_, bc_, bm_, bn_, wgm_, wgn_, ns_)                                               \
  if (sh.br == (br_) && sh.bc == (bc_) && sh.bm == (bm_) && sh.bn == (bn_) && sh.wgm == (wgm_) &&      \
      sh.wgn == (wgn_) && sh.depth == (ns_)) {                                                        \
    if constexpr (!POOL || ((br_) % 2 == 0 && (bc_) % 2 == 0)) {                                      \
      hipExtLaunchKernelGGL((conv_patch_kernel<br_, bc_, bm_, bn_, wgm_, wgn_, ns_, POOL>), grid,      \
                            dim3(64 * (wgm_) * (wgn_)), 0, stream, ev.start, ev.stop, 0, args);       \
      return hipGetLastError();                                                                       \
    }                                                                                                 \
    return hipErrorInvalidValue;                                                                      \
  }
  MAFAT_PATCH_SHAPES
  MAFAT_PATCH_TUNE_SHAPES
#undef MAFAT_PATCH
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_conv_patch_fused(const StageArgs& args, hipStream_t stream, LaunchEvents ev) {
  if (args.total_blocks <= 0) return hipSuccess;
  if (args.cout != 128 || (args.cout2 != 64 && args.cout2 != 32)) return hipErrorInvalidValue;
  const dim3 grid(static_cast<unsigned>(args.total_blocks), args.copy_blocks > 0 ? 2u : 1u);
  if (args.cout2 == 64)
    hipExtLaunchKernelGGL((conv_patch_kernel<8, 16, 128, 128, 4, 2, 1, false, 64>), grid, dim3(512), 0, stream,
                          ev.start, ev.stop, 0, args);
  else
    hipExtLaunchKernelGGL((conv_patch_kernel<8, 16, 128, 128, 4, 2, 1, false, 32>), grid, dim3(512), 0, stream,
                          ev.start, ev.stop, 0, args);
  return hipGetLastError();
}

hipError_t launch_conv_patch_first(const MfmaShape& sh, const StageArgs& args, hipStream_t stream, LaunchEvents ev) {
  if (args.total_blocks <= 0) return hipSuccess;
  if (args.cin != 32 || args.cout != 64 || args.nblk_n != 1) return hipErrorInvalidValue;
#define MAFAT_FIRST(br_, bc_, bm_, wgm_, wgn_)                                                            \
  if (sh.br == (br_) && sh.bc == (bc_) && sh.bm == (bm_) && sh.bn == 64 && sh.wgm == (wgm_) &&            \
      sh.wgn == (wgn_)) {                                                                                 \
    hipExtLaunchKernelGGL((conv_patch_kernel<br_, bc_, bm_, 64, wgm_, wgn_, 1, true, 0, true>),           \
                          dim3(static_cast<unsigned>(args.total_blocks), args.copy_blocks > 0 ? 2u : 1u), dim3(64 * (wgm_) * (wgn_)), 0,  \
                          stream, ev.start, ev.stop, 0, args);                                            \
    return hipGetLastError();                                                                             \
  }
  MAFAT_FIRST_SHAPES
#undef MAFAT_FIRST
  return hipErrorInvalidValue;
}

hipError_t launch_conv_patch(bool pool, const MfmaShape& shape, const StageArgs& args, hipStream_t stream,
                             LaunchEvents ev) {
  if (args.total_blocks <= 0) return hipSuccess;
  return pool ? launch_patch_p<true>(shape, args, stream, ev) : launch_patch_p<false>(shape, args, stream, ev);
}

#ifdef MAFAT_TUNING
extern "C" int mafat_debug_wg_patch(long long* host_out) {
  return hipMemcpyFromSymbol(host_out, HIP_SYMBOL(g_wg_patch), sizeof(g_wg_patch)) == hipSuccess ? 0 : -1;
}
extern "C" int mafat_debug_patch_trace(long long* host_out) {
  return hipMemcpyFromSymbol(host_out, HIP_SYMBOL(g_patch_trace), sizeof(g_patch_trace)) == hipSuccess ? 0 : -1;
}
#endif
}  // namespace mafat
