// conv_ring.hip -- bf16 convolution stage (3x3 or 1x1, stride 1, folded
// batch-norm scale/bias, activation, optional fused 2x2/2 max-pool) as an
// implicit GEMM on the matrix cores, with its operands streamed from global
// memory straight into a ring of LDS stage slots.
//
// GEMM: M = the tile's computed output pixels, N = output channels, K =
// f*f*c_in in (tap, channel) order, the order of the KRSC weight rows.  One
// K stage is 64 bf16 = 128 bytes of every A row (pixel) and B row (output
// channel), made of two 64-byte sub-chunks (32 channels of one filter tap
// each, so c_in = 32 works too).
//
// Data movement (per workgroup, BM pixels x BN channels):
//   - A ring of NS slots in LDS, each holding one K stage of the BM + BN
//     rows (128 bytes per row).  Stage s lives in slot s % NS.
//   - Each thread fetches 16-byte pieces with buffer_load_dwordx4 ... lds:
//     the data goes from L2/HBM directly into LDS (no VGPR staging), 64
//     lanes filling 1 KiB = 8 rows of one slot per instruction.  Lane l
//     writes row (l >> 3), 16-byte position (l & 7) of its 8-row group and
//     fetches the global 16-byte chunk (l & 7) ^ (l >> 3) of that row: an
//     XOR swizzle of the chunk position by the row, so the fragment reads of
//     16 consecutive rows at one K offset spread over all LDS banks.
//   - Zero padding costs nothing: a filter tap outside the image, a pixel
//     past the tile's last row and a weight row past c_out are fetched at
//     an offset with bit 31 set, past the buffer descriptor's range, and
//     the range check returns zeros.
//   - Loads run NS - 1 stages ahead of the MFMAs.  Iteration s waits (an
//     explicit s_waitcnt vmcnt) until this thread's loads of stage s have
//     landed, meets the other waves at a barrier (then stage s is complete
//     in LDS and every wave is done reading slot (s - 1) % NS), issues the
//     loads of stage s + NS - 1 into that freed slot, reads its MFMA
//     fragments of stage s and runs the MFMAs.
// Compute: waves in a WGM x WGN arrangement over the block, each owning a
// (BM/WGM) x (BN/WGN) tile of 16x16 accumulators, v_mfma_f32_16x16x32_bf16.
// With KG = 2 there are two such arrangements (8 waves when WGM x WGN = 4);
// group g multiplies the 64-byte half g of every stage, and the two partial
// sums meet through LDS at the end (each group then stores half of the
// channel tiles).
// Epilogue: without a pool the weights are the MFMA's A operand, so a lane
// holds 4 consecutive channels of one pixel; with a fused pool the pixels
// are, quad-ordered, so a lane's 4 accumulator rows are one 2x2 window,
// reduced in the lane.  The block's outputs are staged in LDS as rows of BN
// channels and leave as 16-byte stores.  The first stage's weight rows are
// issued while the tile table is being decoded.
//
// Requires c_in % 32 == 0, c_out % 16 == 0, byte offsets below 2^31 within
// a frame's source buffer and within the weights (checked by the host).
#include <hip/hip_runtime.h>

#include "device_util.h"
#include "kernel_args.h"

namespace mafat {
#ifdef MAFAT_TUNING
// Tuning builds only: phase timestamps (wall clock, 100 MHz) of three
// workgroups (the first, the middle and the last of the grid).
__device__ long long g_ring_trace[3][64];
MAFAT_WG_TRACE_DECL(g_wg_ring)
#define MAFAT_RTRACE(slot_)                                                                      \
  do {                                                                                           \
    if (threadIdx.x == 0 && (slot_) < 64 &&                                                      \
        (blockIdx.x == 0 || blockIdx.x == a.total_blocks / 2 || blockIdx.x == a.total_blocks - 1))         \
      g_ring_trace[blockIdx.x == 0 ? 0 : (blockIdx.x == a.total_blocks - 1 ? 2 : 1)][(slot_)] =       \
          wall_clock64();                                                                        \
  } while (0)
#else
#define MAFAT_RTRACE(slot_) do {} while (0)
#endif
namespace {

typedef __attribute__((address_space(3))) void* lds_ptr_t;

// Wait until at most N of this thread's vector memory operations are
// outstanding.  (Loads complete in issue order.)
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N <= 63, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Wait until the loads of the oldest outstanding stage have landed, when
// `rem` later stages (L loads each, at most R of them) are in flight.
template <int L, int R>
__device__ __forceinline__ void wait_stage(int rem) {
  if constexpr (R == 0) {
    wait_vmcnt<0>();
  } else {
    if (rem >= R) {
      wait_vmcnt<R * L>();
    } else {
      wait_stage<L, R - 1>(rem);
    }
  }
}

// Workgroup barrier without a memory fence (the fence of __syncthreads
// would wait for every outstanding LDS load); the "memory" clobber keeps
// the compiler from moving LDS reads across it.
__device__ __forceinline__ void wg_barrier() { asm volatile("s_barrier" ::: "memory"); }

template <int F, int BM, int BN, int WGM, int WGN, int KG, int NS, int KORD, bool POOL>
__global__ __launch_bounds__(64 * WGM * WGN * KG) void conv_ring_kernel(const StageArgs a) {
  if (__builtin_expect(blockIdx.y != 0, 0)) {  // the second grid row: carried band copies (row reuse)
    carried_copies();
    return;
  }
  constexpr int NWAVE = WGM * WGN * KG;
  constexpr int P = (F - 1) / 2;
  constexpr int WM = BM / WGM, WN = BN / WGN, MT = WM / 16, NT = WN / 16;
  constexpr int ROWB = 128;                 // bytes of one row per K stage
  constexpr int SLOT = (BM + BN) * ROWB;    // bytes of one ring slot
  constexpr int APW = BM / (8 * NWAVE);     // A load instructions per wave per stage
  constexpr int BPW = BN / (8 * NWAVE);     // B load instructions per wave per stage
  constexpr int LPS = APW + BPW;            // loads per thread per stage
  constexpr int NH = 2 / KG;                // 64-byte halves each wave multiplies per stage
  static_assert(MT >= 1 && NT >= 1 && MT * 16 == WM && NT * 16 == WN, "wave tile");
  static_assert(APW >= 1 && BPW >= 1 && APW * 8 * NWAVE == BM && BPW * 8 * NWAVE == BN, "load split");
  static_assert(NS >= 2 && NS <= 8 && (NS - 2) * LPS <= 63, "ring depth");
  static_assert(KG == 1 || (KG == 2 && NT % 2 == 0), "two K groups split the channel tiles");
  static_assert(F * F < 31, "tap mask (bit 31 marks a padded sub-chunk)");
  __shared__ __align__(1024) unsigned char smem[NS * SLOT];

  MAFAT_RTRACE(0);
  MAFAT_WG_MARK(g_wg_ring, 0);
  const int tid = static_cast<int>(threadIdx.x), lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int cin = a.cin, cout = a.cout;
  const int K = F * F * cin;
  const int cblocks = cin >> 5;            // 32-channel sub-chunks per tap
  const int nsub = F * F * cblocks;
  const int nstage = (nsub + 1) >> 1;
  const __amdgpu_buffer_rsrc_t rsb = make_rsrc(a.w, static_cast<unsigned>(cout * K * 2));
  // This lane's loads: row (lane >> 3) of 8-row group (k * NWAVE + wave) of
  // the A rows (k < APW) and of the B rows (k < BPW); global 16-byte chunk
  // cg of the 128-byte stage row = piece pc of sub-chunk hh.
  const int lrow = lane >> 3;
  const int cg = (lane & 7) ^ lrow;
  const int hh = cg >> 2, pc = cg & 3;

  // Load cursor (wave-uniform) over the 64-byte sub-chunks of K: an outer
  // and an inner index, inner fastest.  KORD 0: outer = filter tap, inner =
  // channel block; KORD 1: outer = channel block, inner = tap, so the f*f
  // taps of one channel block follow each other and their shifted re-reads
  // of the same input pixels hit the L1 cache.  A padded last sub-chunk
  // (past the end of K) reads zero A rows and re-reads valid weights.
  constexpr int TAPS = F * F;
  const int ilim = KORD ? TAPS : cblocks, olim = KORD ? cblocks : TAPS;
  // Offsets of the stage whose first sub-chunk is at cursor (o0, i0), for
  // this lane's half hh: the tap's mask bit (31: an invalid sub-chunk), the
  // A offset (source row width swv) and the B offset; and the next cursor.
  struct SubOff { unsigned tap, aoff, boff; int on, in; };
  auto sub_offsets = [&](int o0, int i0, int swv) {
    const int w0 = (ilim - 2 - i0) >> 31;  // -1: the next sub-chunk starts a new outer index
    const int o1 = o0 - w0, i1 = (i0 + 1) & ~w0;
    const int w1 = (ilim - 2 - i1) >> 31;
    const bool v0 = o0 < olim, v1 = o1 < olim;
    const int tap0 = v0 ? (KORD ? i0 : o0) : 0, cb0 = v0 ? (KORD ? o0 : i0) : 0;
    const int tap1 = v1 ? (KORD ? i1 : o1) : 0, cb1 = v1 ? (KORD ? o1 : i1) : 0;
    const int ky0 = tap0 / F, kx0 = tap0 - ky0 * F;
    const int ky1 = tap1 / F, kx1 = tap1 - ky1 * F;
    const int ao0 = (((ky0 - P) * swv + (kx0 - P)) * cin + cb0 * 32) * 2;
    const int ao1 = (((ky1 - P) * swv + (kx1 - P)) * cin + cb1 * 32) * 2;
    const int bo0 = (tap0 * cin + cb0 * 32) * 2;
    const int bo1 = (tap1 * cin + cb1 * 32) * 2;
    SubOff r;
    r.tap = static_cast<unsigned>(hh ? (v1 ? tap1 : 31) : (v0 ? tap0 : 31));
    r.aoff = static_cast<unsigned>(hh ? ao1 : ao0);
    r.boff = static_cast<unsigned>(hh ? bo1 : bo0);
    r.on = o1 - w1;
    r.in = (i1 + 1) & ~w1;
    return r;
  };
  unsigned b_off[BPW];
  auto issue_b = [&](int slot, unsigned boff) {
    unsigned char* sbase_l = smem + slot * SLOT;
#pragma unroll
    for (int k = 0; k < BPW; ++k)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          rsb, (lds_ptr_t)(sbase_l + (BM + 8 * (k * NWAVE + wave)) * ROWB), 16,
          static_cast<int>(b_off[k] + boff), 0, 0, 0);
  };
  // The weight rows depend only on the channel block: the first stage's are
  // issued while the tile table is still on its way.
  auto early = [&](int nb) {
#pragma unroll
    for (int k = 0; k < BPW; ++k) {
      const int co = nb * BN + 8 * (k * NWAVE + wave) + lrow;
      b_off[k] = co < cout ? static_cast<unsigned>((co * K + pc * 8) * 2) : 0x80000000u;
    }
    issue_b(0, sub_offsets(0, 0, 0).boff);
  };
  KTile tl;
  const BlockPos bp = decode_block(a, &tl, early);
  MAFAT_RTRACE(1 + (tl.ch < -1 ? 1 : 0));
  const int grp = wave / (WGM * WGN), wq = wave - grp * (WGM * WGN);
  const int wm = wq / WGN, wn = wq - wm * WGN;
  const int M = tl.ch * tl.cw;
  const int m0 = bp.mb * BM, n0 = bp.nb * BN;
  const int sw = tl.sw;
  const int64_t sbase = bp.frame * a.src_fstride + tl.src_off;
  uint16_t* dst = static_cast<uint16_t*>(a.dst) + bp.frame * a.dst_fstride + tl.dst_off;
  const __amdgpu_buffer_rsrc_t rsa = make_rsrc(static_cast<const uint16_t*>(a.src) + sbase,
                                               static_cast<unsigned>((a.src_fstride - tl.src_off) * 2));

  // Scale and bias of this lane's output channels (issued first, so their
  // latency overlaps the main loop).
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

  unsigned a_off[APW], a_inv[APW];
#pragma unroll
  for (int k = 0; k < APW; ++k) {
    const int m = m0 + 8 * (k * NWAVE + wave) + lrow;
    int oy, ox;
    row_pixel<POOL>(tl, m < M ? m : 0, &oy, &ox);
    a_off[k] = static_cast<unsigned>((((oy - tl.sy0) * sw + (ox - tl.sx0)) * cin + pc * 8) * 2);
    unsigned inv = ~0u << (F * F);
#pragma unroll
    for (int t = 0; t < F * F; ++t) {
      const int iy = oy + t / F - P, ix = ox + t % F - P;
      const bool in = static_cast<unsigned>(iy) < static_cast<unsigned>(a.in_h) &&
                      static_cast<unsigned>(ix) < static_cast<unsigned>(a.in_w);
      inv |= in ? 0u : (1u << t);
    }
    a_inv[k] = (m < M) ? inv : ~0u;
  }

  // A stage's loads at the cursor (the first stage's weights were issued
  // during the decode).
  int lc_o = 0, lc_i = 0;
  auto issue = [&](int slot, bool skip_b) {
    const int o0 = __builtin_amdgcn_readfirstlane(lc_o);
    const int i0 = __builtin_amdgcn_readfirstlane(lc_i);
    const SubOff so = sub_offsets(o0, i0, sw);
    unsigned char* sbase_l = smem + slot * SLOT;
#pragma unroll
    for (int k = 0; k < APW; ++k) {
      const unsigned bad = (a_inv[k] >> so.tap) & 1u;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          rsa, (lds_ptr_t)(sbase_l + (8 * (k * NWAVE + wave)) * ROWB), 16,
          static_cast<int>((a_off[k] + so.aoff) | (bad << 31)), 0, 0, 0);
    }
    if (!skip_b) issue_b(slot, so.boff);
    lc_o = so.on;
    lc_i = so.in;
  };

  // Fragment reads: lane l supplies rows (l & 15) of a 16-row fragment at K
  // offset 8 (l >> 4) of the 64-byte half h, i.e. global chunk 4h + (l >> 4)
  // of the row, stored at position chunk ^ (row & 7) (row & 7 == l & 7).
  int rd_a[NH], rd_b[NH];
#pragma unroll
  for (int hi = 0; hi < NH; ++hi) {
    const int h = (KG == 2) ? grp : hi;
    const int cpos = (((h * 4) + (lane >> 4)) ^ (lane & 7)) * 16;
    rd_a[hi] = (wm * WM + (lane & 15)) * ROWB + cpos;
    rd_b[hi] = (BM + wn * WN + (lane & 15)) * ROWB + cpos;
  }

  f32x4 acc[NT][MT];  // [channel tile][pixel tile]
#pragma unroll
  for (int j = 0; j < NT; ++j)
#pragma unroll
    for (int i = 0; i < MT; ++i) acc[j][i] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto compute = [&](int slot) {
    const unsigned char* sp = smem + slot * SLOT;
    u32x4 af[NH][MT], bfr[NH][NT];
#pragma unroll
    for (int hi = 0; hi < NH; ++hi) {
#pragma unroll
      for (int i = 0; i < MT; ++i) af[hi][i] = *reinterpret_cast<const u32x4*>(sp + rd_a[hi] + i * 16 * ROWB);
#pragma unroll
      for (int j = 0; j < NT; ++j) bfr[hi][j] = *reinterpret_cast<const u32x4*>(sp + rd_b[hi] + j * 16 * ROWB);
    }
#pragma unroll
    for (int hi = 0; hi < NH; ++hi)
#pragma unroll
      for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int j = 0; j < NT; ++j) {
          if constexpr (POOL) mma<MAFAT_BF16>(acc[j][i], af[hi][i], bfr[hi][j]);
          else mma<MAFAT_BF16>(acc[j][i], bfr[hi][j], af[hi][i]);
        }
  };

  // Prologue: stages 0 .. NS-2 in flight.
#pragma unroll
  for (int p = 0; p < NS - 1; ++p)
    if (p < nstage) issue(p, p == 0);
  int slot = 0;
  for (int s = 0; s < nstage; ++s) {
    wait_stage<LPS, NS - 2>(nstage - 1 - s);
    wg_barrier();
    MAFAT_RTRACE(8 + s);
    if (s + NS - 1 < nstage) issue(slot == 0 ? NS - 1 : slot - 1, false);
    compute(slot);
    slot = (slot == NS - 1) ? 0 : slot + 1;
  }

  MAFAT_RTRACE(4);
  const int M_ = M;
  if constexpr (KG == 2) {
    // Each group keeps half of the channel tiles: it hands the other half
    // of its partial sums to the partner wave (same position in the other
    // group) through LDS and adds the partner's partial sums for its half.
    constexpr int NH2 = NT / 2;
    static_assert(NWAVE * NH2 * MT * 64 * 16 <= NS * SLOT, "partial sums fit in the ring");
    f32x4* sX = reinterpret_cast<f32x4*>(smem);  // [wave][NH2][MT][64 lanes]
    __syncthreads();  // every wave is done with the ring (all loads landed: vmcnt(0) above)
    const int partner = (wave + WGM * WGN) % NWAVE;
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

  // Epilogue: folded batch-norm, activation (leaky: max(v, 0.1 v)), the
  // fused pool, round to bf16; the block's outputs are staged in LDS as rows
  // of BN channels per output pixel and leave as 16-byte stores (each
  // pixel's BN channels one contiguous run); only the tile's own output
  // rectangle is stored.
  constexpr int NTHR = 64 * NWAVE;
  constexpr int RSB = BN * 2 + 16;          // LDS bytes per staged pixel row
  constexpr int NPXO = POOL ? BM / 4 : BM;  // output pixels of the block
  constexpr int CPB = BN / 8;               // 16-byte chunks per pixel row
  static_assert(NPXO * RSB <= NS * SLOT, "staged block fits in the ring");
  const float slope = act_slope(a.act);
  __syncthreads();  // every wave is done with the ring (and the K-group exchange)
#pragma unroll
  for (int i = 0; i < MT; ++i) {
#pragma unroll
    for (int j = 0; j < NT; ++j) {
      if (KG == 2 && (j < grp * (NT / 2) || j >= (grp + 1) * (NT / 2))) continue;
      if (POOL) {
        const int rl = wm * WM + i * 16 + 4 * (lane >> 4);  // first block row of this lane's window
        float v[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) v[r] = fmaf(acc[j][i][r], sc[j][0], bi[j][0]);
        float mx = fmaxf(fmaxf(v[0], v[1]), fmaxf(v[2], v[3]));
        mx = fmaxf(mx, slope * mx);
        store1(reinterpret_cast<uint16_t*>(smem + (rl >> 2) * RSB) + wn * WN + j * 16 + (lane & 15), mx);
      } else {
        const int rl = wm * WM + i * 16 + (lane & 15);
        float v[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          v[r] = fmaf(acc[j][i][r], sc[j][r], bi[j][r]);
          v[r] = fmaxf(v[r], slope * v[r]);
        }
        store4<MAFAT_BF16>(reinterpret_cast<uint16_t*>(smem + rl * RSB) + wn * WN + j * 16 + 4 * (lane >> 4), v);
      }
    }
  }
  __syncthreads();
  for (int e = tid; e < NPXO * CPB; e += NTHR) {
    const int p = e / CPB, k = e - p * CPB;
    const int m = m0 + (POOL ? 4 * p : p);
    const int c0 = n0 + k * 8;
    if (m < M_ && c0 < cout) {
      int oy, ox;
      if (POOL) {
        const int pw = tl.cw >> 1, qq = m >> 2, qy = qq / pw;
        oy = (tl.cy0 >> 1) + qy;
        ox = (tl.cx0 >> 1) + (qq - qy * pw);
      } else {
        row_pixel<false>(tl, m, &oy, &ox);
      }
      const u32x4 v = *reinterpret_cast<const u32x4*>(smem + p * RSB + k * 16);
      *reinterpret_cast<u32x4*>(dst + ((oy - tl.dy0) * tl.dw + (ox - tl.dx0)) * cout + c0) = v;
    }
  }
  MAFAT_RTRACE(5);
  MAFAT_WG_MARK(g_wg_ring, 1);
}

template <int F, bool POOL>
hipError_t launch_ring_fp(const MfmaShape& sh, const StageArgs& args, hipStream_t stream, LaunchEvents ev) {
  const dim3 grid(static_cast<unsigned>(args.total_blocks), args.copy_blocks > 0 ? 2u : 1u);
#define MAFAT_RING(bm_, bn_, wgm_, wgn_, kg_, ns_, ko_)                                             \
  if (sh.bm == (bm_) && sh.bn == (bn_) && sh.wgm == (wgm_) && sh.wgn == (wgn_) && sh.kg == (kg_) && \
      sh.depth == (ns_) && sh.kord == (ko_)) {                                                     \
    hipExtLaunchKernelGGL((conv_ring_kernel<F, bm_, bn_, wgm_, wgn_, kg_, ns_, ko_, POOL>), grid,   \
                          dim3(64 * (wgm_) * (wgn_) * (kg_)), 0, stream, ev.start, ev.stop, 0, args); \
    return hipGetLastError();                                                                      \
  }
  MAFAT_RING_SHAPES
  MAFAT_RING_TUNE_SHAPES
#undef MAFAT_RING
  return hipErrorInvalidValue;
}

}  // namespace

#ifdef MAFAT_TUNING
extern "C" int mafat_debug_wg_ring(long long* host_out) {
  return hipMemcpyFromSymbol(host_out, HIP_SYMBOL(g_wg_ring), sizeof(g_wg_ring)) == hipSuccess ? 0 : -1;
}
extern "C" int mafat_debug_ring_trace(long long* host_out) {
  return hipMemcpyFromSymbol(host_out, HIP_SYMBOL(g_ring_trace), sizeof(g_ring_trace)) == hipSuccess ? 0 : -1;
}
#endif

hipError_t launch_conv_ring(int f, bool pool, const MfmaShape& shape, const StageArgs& args,
                            hipStream_t stream, LaunchEvents ev) {
  if (args.total_blocks <= 0) return hipSuccess;
  if (f == 3) return pool ? launch_ring_fp<3, true>(shape, args, stream, ev) : launch_ring_fp<3, false>(shape, args, stream, ev);
  if (f == 1) return pool ? launch_ring_fp<1, true>(shape, args, stream, ev) : launch_ring_fp<1, false>(shape, args, stream, ev);
  return hipErrorInvalidValue;
}

}  // namespace mafat
