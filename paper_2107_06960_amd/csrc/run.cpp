// run.cpp -- C ABI execution entry points: validate the request, build the
// per-stage argument blocks from the plan and enqueue the stage kernels on
// the caller's stream.  No device allocation, no synchronisation.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <string>
#include <vector>

#include "kernel_args.h"
#include "mafat_internal.h"

#ifdef MAFAT_TUNING
extern "C" int mafat_debug_trace(long long* host_out);
extern "C" int mafat_debug_ring_trace(long long* host_out);
extern "C" int mafat_debug_wg_rgb(long long* host_out);
extern "C" int mafat_debug_wg_patch(long long* host_out);
extern "C" int mafat_debug_wg_ring(long long* host_out);
extern "C" int mafat_debug_patch_trace(long long* host_out);
#endif

namespace mafat {
namespace {

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int fail(int status, const std::string& msg) {
  set_error(msg);
  return status;
}

// The matrix-core kernel needs whole 64-byte K chunks (32 bf16 or 16 fp32
// input channels), output channels in multiples of 16, and its weights
// addressable with 32-bit byte offsets (the source buffer is checked per
// launch).
// The matrix-core and first-layer kernels take "same" convolutions only:
// f = 1 or 3, stride 1, padding (f - 1) / 2.  Every other convolution (and
// channel count) runs on the generic kernel.
bool same_conv(const Stage& S) {
  return S.kind == STAGE_CONV && (S.f == 1 || S.f == 3) && S.s == 1 && S.p == (S.f - 1) / 2;
}

bool mfma_ok(const Stage& S, int dtype) {
  const int kc = (dtype == MAFAT_BF16) ? 32 : 16;
  const int64_t esz = (dtype == MAFAT_BF16) ? 2 : 4;
  return same_conv(S) && S.cin % kc == 0 && S.cout % 16 == 0 &&
         static_cast<int64_t>(S.cout) * S.f * S.f * S.cin * esz < (1ll << 31);
}

// The vector first-layer kernel: 3 input channels, 3x3, 8/16/32/64 outputs.
bool rgb_ok(const Stage& S) {
  return same_conv(S) && S.cin == 3 && S.f == 3 &&
         (S.cout == 8 || S.cout == 16 || S.cout == 32 || S.cout == 64);
}

// Tuning builds only: MAFAT_TUNE="first_layer:bm,bn,depth[,chan_major[,kg[,kind[,kord[,br,bc[,wgm,wgn]]]]]];..."
// forces the configuration of the stage starting at first_layer (kind: 0 the
// register-staged matrix-core kernel, 5 the LDS-ring kernel, 6 the 3x3 patch
// kernel).
StageConfig tune_override(const Stage& S, StageConfig c) {
#ifdef MAFAT_TUNING
  if (const char* env = std::getenv("MAFAT_TUNE")) {
    std::string e(env);
    size_t pos = 0;
    while (pos < e.size()) {
      size_t end = e.find(';', pos);
      if (end == std::string::npos) end = e.size();
      int l, bm, bn, dp, cm = -1, kg = -1, kind = -1, ko = -1, br = -1, bc = -1, wgm = -1, wgn = -1;
      const int got = std::sscanf(e.substr(pos, end - pos).c_str(), "%d:%d,%d,%d,%d,%d,%d,%d,%d,%d,%d,%d", &l,
                                  &bm, &bn, &dp, &cm, &kg, &kind, &ko, &br, &bc, &wgm, &wgn);
      if (got >= 4 && l == S.first) {
        c.bm = bm; c.bn = bn; c.depth = dp;
        if (cm >= 0) c.chan_major = cm;
        if (kg >= 1) c.kg = kg;
        if (kind >= 0) c.kind = kind;
        if (ko >= 0) c.kord = ko;
        if (br > 0 && bc > 0) { c.br = br; c.bc = bc; }
        if (wgm > 0 && wgn > 0) { c.wgm = wgm; c.wgn = wgn; }
      }
      pos = end + 1;
    }
  }
#else
  (void)S;
#endif
  return c;
}

}  // namespace

// Block tile and pipeline depth for the matrix-core kernel, from a small
// time model of one CU: a workgroup costs a fixed ~2 us (first loads,
// epilogue) plus the larger of its MFMA time at the CU's peak (4096
// flop/clock) and its operand traffic at the CU's L2 bandwidth (64
// bytes/clock); workgroups beyond 256 queue on the CUs.  Larger tiles
// re-read fewer operands, smaller ones give more workgroups.
StageConfig choose_config(const Stage& S, int batch, int dtype) {
  StageConfig c{};
  c.bm = 64; c.bn = 64; c.depth = 3; c.kg = 1; c.wgm = 2; c.wgn = 2; c.br = 0; c.bc = 0;
  if (S.kind == STAGE_POOL) { c.kind = K_POOL; return c; }
  if (!mfma_ok(S, dtype)) {
    c.kind = rgb_ok(S) ? K_CONV_RGB : K_CONV_DIRECT;
    // bf16 first layer with 16/32/64 outputs: K = 27 padded to one MFMA K.
    if (c.kind == K_CONV_RGB && dtype == MAFAT_BF16 && (S.cout == 16 || S.cout == 32 || S.cout == 64)) {
      c.kind = K_CONV_RGB_MFMA;
      c.bn = S.cout;
    }
    return tune_override(S, c);
  }
  const int esz = (dtype == MAFAT_BF16) ? 2 : 4;
  const double K = static_cast<double>(S.f) * S.f * S.cin;
  if (dtype == MAFAT_BF16 && S.f == 3) {
    // 3x3 patch kernel (each block's input patch loaded once per 32-channel
    // chunk and shared by the nine taps), 8 waves per workgroup (two per
    // SIMD: LDS reads reach ~220 bytes/clock per CU only with more than one
    // wave per SIMD).  Block shape by a model fitted to a sweep of the
    // YOLOv2 stages at 608x608 (5x5/8/2x2): one workgroup per CU (the ring
    // takes most of the LDS), so a stage takes ceil(workgroups / 256)
    // rounds of ~3 us (decode, first loads, epilogue) plus, per 32-channel
    // chunk, ~0.18 ns per block pixel-channel (edge blocks of a tile compute
    // their full rectangle).  Large blocks waste work on small tiles and
    // leave CUs idle on small stages; small blocks re-load more halo and
    // weights.
    c.kind = K_CONV_PATCH;
    struct PS { int br, bc, bm, bn, wgm, wgn, ns; };
    static const PS kPatch[] = {
#define MAFAT_PATCH(br_, bc_, bm_, bn_, wgm_, wgn_, ns_) {br_, bc_, bm_, bn_, wgm_, wgn_, ns_},
        MAFAT_PATCH_SHAPES
#undef MAFAT_PATCH
    };
    const int chunks = S.cin / 32;
    double best = 1e30;
    for (const PS& r : kPatch) {
      // 128 channels: the fused layer 4-5 pair's shape; 14x18: a first-layer
      // pair's shape (its second stage alone takes it too)
      if ((r.bn > S.cout && r.bn > 32) || r.bn == 128 || r.br == 14) continue;
      // One-slot rings only for single-chunk layers (c_in = 32), where they
      // are measured fastest (several workgroups per CU overlap their loads);
      // among them the model below picks (12x16 blocks on YOLOv2's layer 2
      // at 608x608: 9.8 us against 12 us for 8x16).
      if ((r.ns == 1) != (chunks == 1 && S.cout >= 64)) continue;
      int64_t mb = 0;
      for (const TileGeom& T : S.tiles)
        mb += static_cast<int64_t>((T.ch + r.br - 1) / r.br) * ((T.cw + r.bc - 1) / r.bc);
      const int64_t blocks = mb * ((S.cout + r.bn - 1) / r.bn);
      const double rounds = std::ceil(static_cast<double>(blocks) * batch / 256.0);
      const double t = rounds * (3e-6 + chunks * static_cast<double>(r.bm) * r.bn * 0.18e-9);
      // Within 2 % of the best, fewer blocks win (less halo and weight
      // traffic; e.g. 12x16 over 12x12 blocks, whose GEMM rows are padded
      // from 144 to 192).
      if (t < best * 0.98 || (t < best * 1.02 && blocks < c.blocks)) {
        best = t;
        c.br = r.br; c.bc = r.bc; c.bm = r.bm; c.bn = r.bn; c.wgm = r.wgm; c.wgn = r.wgn; c.depth = r.ns;
        c.blocks = blocks;
      }
    }
  }
  if (dtype == MAFAT_BF16 && (S.f != 3 || c.kind != K_CONV_PATCH || c.br == 0)) {
    // LDS-ring kernel.  Block shapes from a sweep over every YOLOv2 stage
    // at 608x608 (tiling 5x5/8/2x2; blocks 32..128 x 32..128, ring depths
    // 2..8, one or two K groups): the K loop of a workgroup is bound by LDS
    // traffic and by the operand bytes it keeps in flight, so wide layers
    // take large blocks with two K groups (8 waves), narrow ones small
    // blocks with several workgroups per CU, and 1x1 layers with a long K
    // the smallest block.
    c.kind = K_CONV_RING;
    c.depth = 3; c.kg = 1; c.kord = 1;
    if (S.f == 1) {
      c.bm = (S.cin >= 256 && S.cout >= 64) ? 32 : 64;
      c.bn = (S.cout >= 64) ? 64 : 32;
    } else if (S.cout >= 256) {
      c.bm = 128; c.bn = 64; c.kg = 2; c.depth = 4;
    } else if (S.cout >= 128) {
      c.bm = 128; c.bn = 128; c.kg = 2; c.depth = 3;
    } else {
      c.bm = 64; c.bn = (S.cout >= 64) ? 64 : 32;
    }
    int64_t mb = 0;
    for (const TileGeom& T : S.tiles) mb += (static_cast<int64_t>(T.ch) * T.cw + c.bm - 1) / c.bm;
    c.blocks = mb * ((S.cout + c.bn - 1) / c.bn);
  } else if (dtype != MAFAT_BF16) {
    c.kind = K_CONV_MFMA;
    const double clk = 2.4e9, mfma_rate = 4096.0 * clk, l2_rate = 64.0 * clk, t0 = 2e-6;
    static const int kShapes[][2] = {{128, 128}, {128, 64}, {64, 128}, {64, 64}, {64, 32}, {32, 64}};
    double best = 1e30;
    for (const auto& sh : kShapes) {
      const int bm = sh[0], bn = sh[1];
      if (bn > S.cout && bn > 32) continue;
      int64_t mb = 0;
      for (const TileGeom& T : S.tiles) mb += (static_cast<int64_t>(T.ch) * T.cw + bm - 1) / bm;
      const int64_t blocks = mb * ((S.cout + bn - 1) / bn);
      const double wgs = static_cast<double>(blocks) * batch;
      const double flops = 2.0 * bm * bn * K, bytes = (bm + bn) * K * esz;
      const double per_wg = std::max(flops / mfma_rate, bytes / l2_rate);
      const double t = t0 + std::ceil(wgs / 256.0) * per_wg;
      if (t < best * 0.97) {
        best = t;
        c.bm = bm; c.bn = bn; c.blocks = blocks;
      }
    }
    // Two K groups (8 waves) when the grid gives a CU at most two
    // workgroups and the block allows it: the second wave per SIMD hides
    // the latency of the per-stage barrier / LDS / MFMA chain.
    c.kg = (c.bm >= 64 && c.bn >= 64 && c.blocks * batch <= 2 * 256) ? 2 : 1;
    // Pipeline depth: stages of K loaded ahead (3 to 6).  The stage count is
    // padded to a multiple of the depth, so take the deepest one whose
    // padding is at most one stage, or none for short K.
    const int nstage = (S.f * S.f * (S.cin / (64 / esz)) + 1) / 2;  // 128-byte K stages
    c.depth = 3;
    for (int d = 6; d >= 3; --d) {
      const int pad = (nstage + d - 1) / d * d - nstage;
      if (pad == 0 || (pad <= 1 && nstage >= 4 * d)) { c.depth = d; break; }
    }
  }
  // Block order.  Each of the 8 XCDs (own L2) reads, at least once, every
  // operand byte its blocks touch.  Pixel-major: each XCD reads all weights
  // and about 1/8 of the input; channel-major: 1/8 of the weights (when
  // there are at least 8 channel blocks) and all the input.
  {
    const double w_bytes = static_cast<double>(S.cout) * K * esz;
    double a_bytes = 0;
    for (const TileGeom& T : S.tiles)
      a_bytes += static_cast<double>(T.ch + S.f - 1) * (T.cw + S.f - 1) * S.cin * esz;
    a_bytes *= batch;
    const double nb = static_cast<double>((S.cout + c.bn - 1) / c.bn);
    const double pix_major = 8.0 * w_bytes + a_bytes;
    const double chan_major = w_bytes * std::max(1.0, 8.0 / nb) + a_bytes * std::min(8.0, nb);
    c.chan_major = chan_major < pix_major ? 1 : 0;
  }
  return tune_override(S, c);
}

namespace {

// A bf16 3x3 stage with 128 outputs (c_in a multiple of 32, no pool)
// followed by a 1x1 stage 128 -> 64 or 128 -> 32 (no pool) that computes the
// same rectangles (YOLOv2's layers 4 and 5 are the first kind): the pair runs as one kernel, the
// 1x1 GEMM taking the 3x3 block's outputs from LDS (one output pass and
// one kernel boundary less).
bool fused_pair(const mafat_plan& P, const Group& G, int s, int dtype) {
  if (dtype != MAFAT_BF16 || s < 0 || s + 1 >= static_cast<int>(G.stages.size())) return false;
  const Stage& A = G.stages[s];
  const Stage& B = G.stages[s + 1];
  if (A.kind != STAGE_CONV || B.kind != STAGE_CONV) return false;
  if (!same_conv(A) || A.f != 3 || A.pool || A.cin % 32 != 0 || A.cout != 128) return false;
  if (!same_conv(B) || B.f != 1 || B.pool || B.cin != 128 || (B.cout != 64 && B.cout != 32)) return false;
  if (!mfma_ok(A, dtype) || A.tiles.size() != B.tiles.size()) return false;
  for (size_t t = 0; t < A.tiles.size(); ++t) {
    const TileGeom& a = A.tiles[t];
    const TileGeom& b = B.tiles[t];
    if (a.cy0 != b.cy0 || a.cx0 != b.cx0 || a.ch != b.ch || a.cw != b.cw) return false;
  }
  // 32-bit byte offsets within a frame's source buffer
  const auto& din = P.dims[G.l0];
  const int64_t src_frame = (A.src_buf == BUF_GROUP_IO) ? static_cast<int64_t>(din[0]) * din[1] * din[2]
                                                        : G.scratch_frame;
  return src_frame * 2 < (1ll << 31);
}

// The group's first stage is a bf16 3-channel 3x3 convolution (32 outputs)
// with a 2x2/2 pool, and the next stage a 3x3 convolution 32 -> 64 with a
// 2x2/2 pool (YOLOv2's layers 0-3): the pair runs as one kernel, each
// workgroup computing the first layer's pooled outputs over its block's
// input patch in LDS (the first layer's output never goes to memory).
bool fused_first(const mafat_plan& P, const Group& G, int s, int dtype) {
  if (dtype != MAFAT_BF16 || s != 0 || s + 1 >= static_cast<int>(G.stages.size())) return false;
  const Stage& A = G.stages[s];
  const Stage& B = G.stages[s + 1];
  if (A.kind != STAGE_CONV || B.kind != STAGE_CONV || A.src_buf != BUF_GROUP_IO) return false;
  if (!same_conv(A) || A.f != 3 || !A.pool || A.cin != 3 || A.cout != 32) return false;
  if (!same_conv(B) || B.f != 3 || !B.pool || B.cin != 32 || B.cout != 64) return false;
  if (!mfma_ok(B, dtype) || A.tiles.size() != B.tiles.size()) return false;
  // pooled blocks need even tile origins and extents (as for any fused pool)
  for (const TileGeom& T : B.tiles)
    if ((T.cy0 | T.cx0 | T.ch | T.cw) & 1) return false;
  const auto& din = P.dims[G.l0];
  return static_cast<int64_t>(din[0]) * din[1] * din[2] * 2 < (1ll << 31);
}

StageConfig first_pair_config(const Stage& B, int batch) {
  // Blocks of the 3x3 stage's conv outputs, all 64 channels, 4x2 waves, one
  // ring slot: 12x16 (48x32 per wave) or 14x18 (64x32 per wave, 256 GEMM
  // rows for 252 outputs).  Two workgroups fit a CU (LDS), so a launch takes
  // ceil(blocks / 512) rounds; a workgroup costs a fixed ~2.5 us (decode,
  // input and weight latency, epilogue) plus ~0.027 us per GEMM row
  // (per-workgroup timestamps at 608x608, 5x5 tiles, where 14x18 blocks
  // make 500 workgroups, one round, and 12x16 blocks 720, two).
  struct FS { int br, bc, bm; };
  static const FS kShapes[] = {{12, 16, 192}, {14, 18, 256}};
  StageConfig c{};
  c.kind = K_CONV_PATCH;
  c.bn = 64; c.wgm = 4; c.wgn = 2; c.depth = 1; c.kg = 1; c.kord = 1; c.chan_major = 0;
  double best = 1e30;
  for (const FS& f : kShapes) {
    int64_t mb = 0;
    for (const TileGeom& T : B.tiles)
      mb += static_cast<int64_t>((T.ch + f.br - 1) / f.br) * ((T.cw + f.bc - 1) / f.bc);
    const double rounds = std::ceil(static_cast<double>(mb) * batch / 512.0);
    const double t = rounds * (2.5 + 0.027 * f.bm);
    if (t < best) {
      best = t;
      c.br = f.br; c.bc = f.bc; c.bm = f.bm; c.blocks = mb;
    }
  }
  return c;
}

}  // namespace

StageConfig stage_config(const mafat_plan& P, const Group& G, const Stage& S, int batch, int dtype) {
  const int si = static_cast<int>(&S - G.stages.data());
  if (fused_first(P, G, si, dtype)) {
    // its own configuration (the first-layer kernel) when it runs alone;
    // run together with the next stage, the launch takes the pair's shape
    StageConfig c = choose_config(S, P.packed_weights ? 1 : batch, dtype);
    c.fuse = 2;
    return c;
  }
  if (fused_first(P, G, si - 1, dtype)) {
    // run alone (mafat_run_stage) it takes the fused kernel's block shape,
    // so its packed weights serve both
    StageConfig c = first_pair_config(S, P.packed_weights ? 1 : batch);
    c.fuse = -2;
    return c;
  }
  if (fused_pair(P, G, si, dtype)) {
    // 8x16 blocks of all 128 channels, one ring slot (the weights of a
    // 32-channel chunk take 72 KiB): on YOLOv2's layer 4 at 608x608 with
    // 5x5 tiles one workgroup per CU, in one round.
    StageConfig c{};
    c.kind = K_CONV_PATCH;
    c.br = 8; c.bc = 16; c.bm = 128; c.bn = 128; c.wgm = 4; c.wgn = 2; c.depth = 1; c.kg = 1; c.kord = 1;
    int64_t mb = 0;
    for (const TileGeom& T : S.tiles) mb += static_cast<int64_t>((T.ch + 7) / 8) * ((T.cw + 15) / 16);
    c.blocks = mb;
    c.fuse = 1;
    return c;
  }
  // A plan with packed weights fixes the layout for every batch: its
  // stages take the configuration chosen for one frame.
  StageConfig c = choose_config(S, P.packed_weights ? 1 : batch, dtype);
  if (fused_pair(P, G, si - 1, dtype)) c.fuse = -1;
  // The matrix-core kernels address a frame's source buffer with 32-bit
  // byte offsets; the generic kernel covers larger frames.
  const int64_t esz = (dtype == MAFAT_F32) ? 4 : 2;
  const auto& din = P.dims[G.l0];
  const int64_t src_frame = (S.src_buf == BUF_GROUP_IO) ? static_cast<int64_t>(din[0]) * din[1] * din[2]
                                                        : G.scratch_frame;
  if ((c.kind == K_CONV_MFMA || c.kind == K_CONV_RING || c.kind == K_CONV_PATCH) &&
      src_frame * esz >= (1ll << 31))
    c.kind = K_CONV_DIRECT;
  return c;
}

bool packed_layout(const mafat_plan& P, int layer, int dtype, int* bn, int* nblk, int* nchunk) {
  *bn = *nblk = *nchunk = 0;
  if (!P.packed_weights || dtype != MAFAT_BF16) return false;
  for (const Group& G : P.groups)
    for (const Stage& S : G.stages)
      if (S.kind == STAGE_CONV && S.first == layer) {
        const StageConfig c = stage_config(P, G, S, 1, dtype);
        if (c.kind != K_CONV_PATCH) return false;
        *bn = c.bn;
        *nblk = (S.cout + c.bn - 1) / c.bn;
        *nchunk = S.cin / 32;
        return true;
      }
  return false;
}

BandLayout band_layout(const mafat_plan& P, const Group& G, int dtype) {
  BandLayout B;
  const int ns = static_cast<int>(G.stages.size());
  B.base.assign(static_cast<size_t>(ns), {-1, -1});
  B.frame = 0;
  for (int s = 0; s + 1 < ns; ++s) {
    const Stage& S = G.stages[s];
    // A stage run fused with the next one keeps its output on chip (a
    // row-reuse group always runs whole, so its fused pairs always fuse).
    if (stage_config(P, G, S, 1, dtype).fuse > 0) continue;
    const int64_t band = (static_cast<int64_t>(S.band_rows) * S.out_w * S.cout + 127) / 128 * 128;
    B.base[static_cast<size_t>(s)] = {B.frame, B.frame + (S.band_copies - 1) * band};
    B.frame += S.band_copies * band;
  }
  return B;
}

WorkspaceLayout workspace_layout(const mafat_plan& P, const Group& G, int batch, int dtype) {
  const size_t esz = (dtype == MAFAT_F32) ? 4 : 2;
  const int64_t frame = G.reuse ? band_layout(P, G, dtype).frame : G.scratch_frame;
  WorkspaceLayout L{};
  L.scratch = (static_cast<size_t>(batch) * frame * esz + 255) & ~static_cast<size_t>(255);
  L.total = L.scratch;
  return L;
}

namespace {

#ifdef MAFAT_TUNING
// Tuning builds only: per-workgroup spans (MAFAT_WG_DUMP) and the phase
// stamps of three workgroups (MAFAT_TRACE_DUMP) of the launch just
// enqueued, printed to stderr (the stream is synchronised first).
void dump_launch_trace(int kind, const Stage& S, const MfmaShape& shape, const StageArgs& A,
                       hipStream_t stream) {
  if (std::getenv("MAFAT_WG_DUMP") && (kind == K_CONV_RING || kind == K_CONV_PATCH || kind == K_CONV_RGB_MFMA)) {
    static long long wt[2][8192];
    (void)hipStreamSynchronize(stream);
    if (kind == K_CONV_RING) mafat_debug_wg_ring(&wt[0][0]);
    else if (kind == K_CONV_PATCH) mafat_debug_wg_patch(&wt[0][0]);
    else mafat_debug_wg_rgb(&wt[0][0]);
    const int n = std::min(A.total_blocks, 8192);
    std::vector<long long> d(n);
    long long s0 = wt[0][0], s1 = wt[0][0], e0 = wt[1][0], e1 = wt[1][0];
    for (int b = 0; b < n; ++b) {
      s0 = std::min(s0, wt[0][b]); s1 = std::max(s1, wt[0][b]);
      e0 = std::min(e0, wt[1][b]); e1 = std::max(e1, wt[1][b]);
      d[b] = wt[1][b] - wt[0][b];
    }
    std::sort(d.begin(), d.end());
    std::fprintf(stderr, "WGSPAN stage %d-%d kind %d grid %d: span %lld ns, starts %lld, first end %lld, "
                 "dur p10 %lld p50 %lld p90 %lld max %lld ns\n", S.first, S.last, kind, A.total_blocks,
                 (e1 - s0) * 10, (s1 - s0) * 10, (e0 - s0) * 10, d[n / 10] * 10, d[n / 2] * 10,
                 d[(9 * n) / 10] * 10, d.back() * 10);
  }
  if (std::getenv("MAFAT_TRACE_DUMP") && (kind == K_CONV_RING || kind == K_CONV_PATCH)) {
    long long tr[3][64];
    (void)hipStreamSynchronize(stream);
    if (kind == K_CONV_RING) mafat_debug_ring_trace(&tr[0][0]);
    else mafat_debug_patch_trace(&tr[0][0]);
    std::fprintf(stderr, "RTRACE stage %d-%d %dx%d kg%d ns%d grid %d\n", S.first, S.last, shape.bm, shape.bn,
                 shape.kg, shape.depth, A.total_blocks);
    for (int w = 0; w < 3; ++w) {
      std::fprintf(stderr, "  wg%d slots 6-9: %lld %lld %lld %lld\n", w, (tr[w][6] - tr[w][0]) * 10,
                   (tr[w][7] - tr[w][0]) * 10, (tr[w][8] - tr[w][0]) * 10, (tr[w][9] - tr[w][0]) * 10);
      std::fprintf(stderr, "  wg%d decode +%lld staged +%lld loopend +%lld end +%lld iters:", w,
                   (tr[w][1] - tr[w][0]) * 10, (tr[w][6] - tr[w][0]) * 10, (tr[w][4] - tr[w][0]) * 10,
                   (tr[w][5] - tr[w][0]) * 10);
      for (int k = 8; k < 44; ++k) std::fprintf(stderr, " %lld", (tr[w][k] - tr[w][0]) * 10);
      std::fprintf(stderr, "\n");
    }
    std::fprintf(stderr, "  start spread: mid-first %lld last-first %lld ns\n", (tr[1][0] - tr[0][0]) * 10,
                 (tr[2][0] - tr[0][0]) * 10);
  }
  if (std::getenv("MAFAT_TRACE_DUMP") && (kind == K_CONV_MFMA || kind == K_CONV_RGB_MFMA)) {
    long long tr[4][64];
    (void)hipStreamSynchronize(stream);
    mafat_debug_trace(&tr[0][0]);
    std::fprintf(stderr, "TRACE stage %d-%d tile %dx%d depth %d grid %d\n", S.first, S.last,
                 shape.bm, shape.bn, shape.depth, A.total_blocks);
    for (int w = 0; w < 3; ++w) {
      std::fprintf(stderr, "  wg%d decoded +%lld addr +%lld issued +%lld lstored +%lld barrier +%lld loop +%lld end +%lld steps:", w,
                   (tr[w][4] - tr[w][0]) * 10, (tr[w][5] - tr[w][0]) * 10, (tr[w][6] - tr[w][0]) * 10,
                   (tr[w][7] - tr[w][0]) * 10, (tr[w][1] - tr[w][0]) * 10, (tr[w][2] - tr[w][0]) * 10,
                   (tr[w][3] - tr[w][0]) * 10);
      for (int k = 8; k < 20; ++k) std::fprintf(stderr, " %lld", (tr[w][k] - tr[w][0]) * 10);
      std::fprintf(stderr, " | remap +%lld divs +%lld prefix +%lld", (tr[w][60] - tr[w][0]) * 10,
                   (tr[w][61] - tr[w][0]) * 10, (tr[w][62] - tr[w][0]) * 10);
      std::fprintf(stderr, "\n");
    }
    std::fprintf(stderr, "  start spread wg-last minus wg0: %lld ns\n", (tr[1][0] - tr[0][0]) * 10);
  }
}
#endif

// Runs stages [s_begin, s_end) of group g: per tile batch (all tiles
// unless the plan sets fewer), every stage in order, a stage as one launch
// per 64 tiles; a fused pair whose two stages are both in the range as one
// kernel.  events, if given, holds two hipEvent_t per stage, indexed from
// s_begin: events[2k] is recorded when the first kernel of stage
// s_begin + k starts, events[2k + 1] when its last kernel ends (timestamps
// of the dispatches themselves); a fused pair's second stage gets two plain
// records after the pair's kernel.
int run_group_impl(const mafat_plan* plan, int g, int s_begin, int s_end, int batch, int dtype, const void* x, void* y,
                   const void* const* w, const float* const* scale, const float* const* bias,
                   void* ws, size_t ws_bytes, hipStream_t stream, void* const* events) {
  const Group& G = plan->groups[g];
  const size_t esz = (dtype == MAFAT_F32) ? 4 : 2;
  size_t need = 0;
  mafat_workspace_size(plan, batch, dtype, &need);
  if (ws_bytes < need)
    return fail(MAFAT_EWORKSPACE, "workspace " + std::to_string(ws_bytes) + " < " + std::to_string(need) + " bytes");
  if (need > 0 && (!ws || (reinterpret_cast<uintptr_t>(ws) & 255u)))
    return fail(MAFAT_EINVAL, "workspace must be non-NULL and 256-byte aligned");
  if (!x || !y || !aligned16(x) || !aligned16(y))
    return fail(MAFAT_EINVAL, "group " + std::to_string(g) + ": x and y must be non-NULL and 16-byte aligned");
  const auto& din = plan->dims[G.l0];
  const auto& dout = plan->dims[G.l1];
  const int64_t in_frame = static_cast<int64_t>(din[0]) * din[1] * din[2];
  const int64_t out_frame = static_cast<int64_t>(dout[3]) * dout[4] * dout[5];
  BandLayout bands;
  if (G.reuse) bands = band_layout(*plan, G, dtype);
  const int64_t scr_frame = G.reuse ? bands.frame : G.scratch_frame;
  if (in_frame >= (1ll << 31) || out_frame >= (1ll << 31) || scr_frame >= (1ll << 31))
    return fail(MAFAT_EUNSUPPORTED, "a frame's tensor exceeds 2^31 elements");
  {
    const char* xb = static_cast<const char*>(x);
    const char* yb = static_cast<const char*>(y);
    const size_t xs = static_cast<size_t>(in_frame) * batch * esz, ys = static_cast<size_t>(out_frame) * batch * esz;
    if (xb < yb + ys && yb < xb + xs) return fail(MAFAT_EINVAL, "x and y overlap");
  }
  for (int l = G.l0; l <= G.l1; ++l)
    if (plan->layers[l].op == MAFAT_CONV) {
      if (!w || !scale || !bias || !w[l] || !scale[l] || !bias[l])
        return fail(MAFAT_EINVAL, "layer " + std::to_string(l) + ": missing weights, scale or bias");
      if (!aligned16(w[l]) || !aligned16(scale[l]) || !aligned16(bias[l]))
        return fail(MAFAT_EINVAL, "layer " + std::to_string(l) + ": weights, scale or bias not 16-byte aligned");
    }

  // Tile batches (mafat_plan_set_tile_batch): tiles [b0, b0 + K) go through
  // all stages, then the next K tiles; the workspace holds K tiles.
  const int K = G.tile_batch;
  const int64_t bstride = G.partition ? G.scratch_elems : static_cast<int64_t>(K) * G.scratch_elems;
  std::vector<char> started(static_cast<size_t>(s_end - s_begin), 0);  // start event recorded
  // Row reuse: the take-over copy of stage s's band into row i, and which
  // launch carries it: launches are numbered within a row; carrier[s] >= 0:
  // that launch of row i - 1 (the first after the band's reader, which
  // neither reads nor writes it); -1: row i's first launch (it reads the
  // group input and writes another band); -2: a copy launch of its own.
  const int ns_all = static_cast<int>(G.stages.size());
  std::vector<int> launch_of(static_cast<size_t>(ns_all), 0), carrier(static_cast<size_t>(ns_all), -2);
  int nlaunch = 0;
  struct BandCopy { int64_t src, dst, bytes; bool aligned; };
  auto band_copy = [&](int s, int i, BandCopy* c) {
    const Stage& S = G.stages[static_cast<size_t>(s)];
    if (bands.base[static_cast<size_t>(s)][0] < 0) return false;
    const int lo = S.band_lo[static_cast<size_t>(i)], prev_lo = S.band_lo[static_cast<size_t>(i - 1)];
    const int n_rows = S.row_b[static_cast<size_t>(i)] - lo;
    if (n_rows <= 0) return false;
    const int64_t row_elems = static_cast<int64_t>(S.out_w) * S.cout, e = static_cast<int64_t>(esz);
    c->src = (bands.base[static_cast<size_t>(s)][(i - 1) & 1] + (lo - prev_lo) * row_elems) * e;
    c->dst = bands.base[static_cast<size_t>(s)][i & 1] * e;
    c->bytes = n_rows * row_elems * e;
    c->aligned = ((c->src | c->dst | c->bytes | (scr_frame * e)) & 15) == 0;
    return true;
  };
  auto run_copies = [&](const std::vector<BandCopy>& cs) {
    BandCopyArgs C;
    std::memset(&C, 0, sizeof(C));
    C.fstride = scr_frame * static_cast<int64_t>(esz);
    for (size_t k = 0; k < cs.size(); ++k) {
      C.src[C.ncopy] = cs[k].src;
      C.dst[C.ncopy] = cs[k].dst;
      C.bytes[C.ncopy] = cs[k].bytes;
      if (++C.ncopy == kMaxBandCopies || k + 1 == cs.size()) {
        const hipError_t e = launch_band_copy(ws, C, batch, stream);
        if (e != hipSuccess) return fail(MAFAT_EHIP, std::string("band copy failed: ") + hipGetErrorString(e));
        C.ncopy = 0;
      }
    }
    return static_cast<int>(MAFAT_OK);
  };
  if (G.reuse) {
    for (int s = s_begin; s < s_end; ++s) {
      const bool fz = stage_config(*plan, G, G.stages[static_cast<size_t>(s)], batch, dtype).fuse > 0 &&
                      s + 1 < s_end;
      launch_of[static_cast<size_t>(s)] = nlaunch;
      if (fz) launch_of[static_cast<size_t>(++s)] = nlaunch;
      ++nlaunch;
    }
    for (int s = 0; s + 1 < ns_all; ++s) {
      if (bands.base[static_cast<size_t>(s)][0] < 0) continue;
      const int reader = launch_of[static_cast<size_t>(s + 1)];
      carrier[static_cast<size_t>(s)] = (reader + 1 < nlaunch) ? reader + 1
                                        : (launch_of[static_cast<size_t>(s)] != 0 ? -1 : -2);
    }
  }
  for (int b0 = 0; b0 < G.ntiles; b0 += K) {
    const int b1 = std::min(G.ntiles, b0 + K);
    const bool last_batch = b1 >= G.ntiles;
    // Row reuse: batch = tile row `row` (K = the grid's columns).  Each band
    // the row writes into first takes over, from the previous row's band,
    // the rows above its own that the next stage reads (within one buffer
    // the two row ranges do not overlap).  The copies ride in launches that
    // neither read nor write the band (carrier[]); the rest, and any the
    // kernels cannot carry, run as one copy launch before the row.
    const int row = b0 / std::max(K, 1);
    std::vector<BandCopy> first_copies;  // carried by this row's first launch
    if (G.reuse && row > 0) {
      std::vector<BandCopy> own;
      for (int s = 0; s + 1 < ns_all; ++s) {
        BandCopy c;
        if (!band_copy(s, row, &c)) continue;
        if (carrier[static_cast<size_t>(s)] == -1 && c.aligned) first_copies.push_back(c);
        else if (carrier[static_cast<size_t>(s)] < 0 || !c.aligned) own.push_back(c);
      }
      const int rc = run_copies(own);
      if (rc != MAFAT_OK) return rc;
    }
    // A fused pair never writes the buffer it reads: inside a group its
    // input and output would be the same ping-pong scratch buffer (stages
    // s - 1 and s + 1), which other workgroups may still be reading, so the
    // pair writes stage s's buffer instead and the later stages of this
    // batch run with the two scratch buffers swapped.
    bool swapped = false;
    auto eff = [&](int buf) { return (swapped && buf >= 0) ? 1 - buf : buf; };
    int launch = -1;
    for (int s = s_begin; s < s_end; ++s) {
      ++launch;
      const Stage& S = G.stages[s];
      // take-over copies this launch carries: its row's (first launch) and
      // the next row's whose band this launch leaves alone
      std::vector<BandCopy> carry;
      if (G.reuse) {
        if (launch == 0) carry = first_copies;
        if (row + 1 < G.rows)
          for (int sb = 0; sb + 1 < ns_all; ++sb) {
            BandCopy c;
            if (carrier[static_cast<size_t>(sb)] == launch && band_copy(sb, row + 1, &c)) {
              if (c.aligned) carry.push_back(c);
            }
          }
      }
      hipEvent_t ev_start = events ? static_cast<hipEvent_t>(events[2 * (s - s_begin)]) : nullptr;
      hipEvent_t ev_stop = events ? static_cast<hipEvent_t>(events[2 * (s - s_begin) + 1]) : nullptr;
      bool launched = started[static_cast<size_t>(s - s_begin)] != 0;
      const StageConfig scfg = stage_config(*plan, G, S, batch, dtype);
      // Both stages of a fused pair in this call: one kernel for the two
      // (the second stage's interval is recorded empty, after it).  A
      // first-layer pair (fuse 2) computes the second stage's blocks, its
      // first stage inside them, in the pair's own block shape.
      const bool fuse = scfg.fuse > 0 && s + 1 < s_end;
      const bool first = fuse && scfg.fuse == 2;
      const Stage* S2 = fuse ? &G.stages[s + 1] : nullptr;
      const StageConfig cfg = first ? first_pair_config(*S2, batch) : scfg;
      const Stage& SC = first ? *S2 : S;  // the convolution whose GEMM the launch computes
      const int kind = cfg.kind;
      const bool matrix = (kind == K_CONV_MFMA || kind == K_CONV_RING || kind == K_CONV_PATCH);
      const MfmaShape shape{cfg.bm, cfg.bn, cfg.depth, cfg.kg, cfg.wgm, cfg.wgn, cfg.kord, cfg.br, cfg.bc};
      const int bu = (kind == K_CONV_RGB) ? 256 / (S.cout / 8) : block_units(kind, shape);
      StageArgs A;
      std::memset(&A, 0, sizeof(A));
      const Stage& SD = fuse ? *S2 : S;  // the stage whose output this launch writes
      const int src_b = eff(S.src_buf);
      int dst_b = eff(SD.dst_buf);
      if (fuse && dst_b >= 0 && dst_b == src_b) dst_b = eff(S.dst_buf);
      const int64_t src_shift = (S.src_buf >= 0) ? (src_b - S.src_buf) * bstride : 0;
      const int64_t dst_shift = (SD.dst_buf >= 0) ? (dst_b - SD.dst_buf) * bstride : 0;
      A.src = (src_b == BUF_GROUP_IO) ? x : ws;
      A.dst = (dst_b == BUF_GROUP_IO) ? y : ws;
      A.src_fstride = (src_b == BUF_GROUP_IO) ? in_frame : scr_frame;
      A.dst_fstride = (dst_b == BUF_GROUP_IO) ? out_frame : scr_frame;
      if (SC.kind == STAGE_CONV) {
        A.w = w[SC.first];
        A.scale = scale[SC.first];
        A.bias = bias[SC.first];
      }
      if (first) {
        A.w0 = w[S.first];
        A.scale0 = scale[S.first];
        A.bias0 = bias[S.first];
        A.act0 = S.act;
        A.in_h0 = S.in_h; A.in_w0 = S.in_w;
      } else if (fuse) {
        A.w2 = w[S2->first];
        A.scale2 = scale[S2->first];
        A.bias2 = bias[S2->first];
        A.cout2 = S2->cout;
        A.act2 = S2->act;
      }
      A.in_h = SC.in_h; A.in_w = SC.in_w;
      A.f = SC.f; A.s = SC.s; A.p = SC.p;
      A.cin = SC.cin; A.cout = SC.cout;
      A.act = SC.act;
      A.nblk_n = matrix ? (SC.cout + shape.bn - 1) / shape.bn : 1;
      A.chan_major = matrix ? cfg.chan_major : 0;
      A.w_packed = (plan->packed_weights && kind == K_CONV_PATCH) ? 1 : 0;
      for (int t0 = b0; t0 < b1; t0 += kMaxTilesPerLaunch) {
        const int t1 = std::min(b1, t0 + kMaxTilesPerLaunch);
        A.ntiles = t1 - t0;
        int64_t total = 0;
        A.mblk_prefix[0] = 0;
        for (int t = t0; t < t1; ++t) {
          const TileGeom& T = S.tiles[t];
          const TileGeom& TC = SC.tiles[t];  // computed rectangle
          KTile& k = A.tiles[t - t0];
          k.cy0 = static_cast<int16_t>(TC.cy0); k.cx0 = static_cast<int16_t>(TC.cx0);
          k.ch = static_cast<int16_t>(TC.ch);   k.cw = static_cast<int16_t>(TC.cw);
          k.sy0 = static_cast<int16_t>(T.sy0); k.sx0 = static_cast<int16_t>(T.sx0);
          k.sw = static_cast<int16_t>(T.sw);
          const TileGeom& TD = SD.tiles[t];
          k.dy0 = static_cast<int16_t>(TD.dy0); k.dx0 = static_cast<int16_t>(TD.dx0);
          k.dw = static_cast<int16_t>(TD.dw);
          if (G.reuse) {  // this row's bands (the fused pair's output is its second stage's)
            const int sd = static_cast<int>(&SD - G.stages.data());
            const int64_t sb = (s == 0) ? 0 : bands.base[static_cast<size_t>(s - 1)][row & 1];
            const int64_t db = (sd + 1 == static_cast<int>(G.stages.size()))
                                   ? 0 : bands.base[static_cast<size_t>(sd)][row & 1];
            if (sb < 0 || db < 0) return fail(MAFAT_EINVAL, "internal: a stage output kept on chip is read");
            k.src_off = static_cast<int32_t>(sb);
            k.dst_off = static_cast<int32_t>(db);
          } else {
            k.src_off = static_cast<int32_t>(T.src_off + src_shift);
            k.dst_off = static_cast<int32_t>(TD.dst_off + dst_shift);
          }
          int64_t units = static_cast<int64_t>(TC.ch) * TC.cw;
          if ((kind == K_CONV_DIRECT || kind == K_CONV_RGB) && S.pool) units /= 4;
          if (kind == K_CONV_RGB_MFMA)  // 2-D blocks of conv outputs
            total += static_cast<int64_t>((TC.ch + kRgbBlockRows - 1) / kRgbBlockRows) *
                     ((TC.cw + kRgbBlockCols - 1) / kRgbBlockCols);
          else if (kind == K_CONV_PATCH)
            total += static_cast<int64_t>((TC.ch + shape.br - 1) / shape.br) * ((TC.cw + shape.bc - 1) / shape.bc);
          else
            total += (units + bu - 1) / bu;
          A.mblk_prefix[t - t0 + 1] = static_cast<int32_t>(total);
        }
        A.mblk_total = static_cast<int32_t>(total);
        const int64_t blocks = total * A.nblk_n * batch;
        if (blocks >= (1ll << 31)) return fail(MAFAT_EUNSUPPORTED, "grid too large");
        A.total_blocks = static_cast<int32_t>(blocks);
        const bool last_chunk = last_batch && t1 >= b1;
        const LaunchEvents lev{launched ? nullptr : ev_start, last_chunk ? ev_stop : nullptr};
        // carried copies: in the first chunk of the launch, as extra
        // workgroups; those that do not fit (or a launch with nothing to
        // compute) get a copy launch of their own here
        A.copy_blocks = A.ncopy = 0;
        if (t0 == b0 && !carry.empty()) {
          std::vector<BandCopy> rest;
          int64_t units = 0;
          for (const BandCopy& c : carry) {
            if (A.total_blocks > 0 && A.ncopy < kMaxCarriedCopies) {
              A.copy_src[A.ncopy] = c.src;
              A.copy_dst[A.ncopy] = c.dst;
              A.copy_bytes[A.ncopy] = c.bytes;
              ++A.ncopy;
              units += c.bytes / 16;
            } else {
              rest.push_back(c);
            }
          }
          if (A.ncopy > 0) {
            A.copy_base = static_cast<unsigned char*>(ws);
            A.copy_fstride = scr_frame * static_cast<int64_t>(esz);
            A.copy_frames = batch;
            A.copy_blocks = static_cast<int32_t>(
                std::min<int64_t>(std::min<int64_t>((units * batch + 255) / 256, 64), A.total_blocks));
          }
          const int rc = run_copies(rest);
          if (rc != MAFAT_OK) return rc;
        }
        hipError_t e;
        if (A.total_blocks <= 0) {
          e = hipSuccess;
        } else if (kind == K_CONV_RING) {
          e = launch_conv_ring(S.f, S.pool, shape, A, stream, lev);
        } else if (first) {
          e = launch_conv_patch_first(shape, A, stream, lev);
        } else if (fuse) {
          e = launch_conv_patch_fused(A, stream, lev);
        } else if (kind == K_CONV_PATCH) {
          e = launch_conv_patch(S.pool, shape, A, stream, lev);
        } else {
          e = launch_stage(kind, dtype, same_conv(S) ? S.f : 0, S.pool, shape, A, stream, lev);
        }
        if (A.total_blocks > 0) {
          launched = true;
        } else if (last_chunk) {  // nothing launched for the last chunk: close the interval here
          if ((!launched && ev_start && hipEventRecord(ev_start, stream) != hipSuccess) ||
              (ev_stop && hipEventRecord(ev_stop, stream) != hipSuccess))
            return fail(MAFAT_EHIP, "hipEventRecord failed");
        }
        if (e != hipSuccess)
          return fail(MAFAT_EHIP, std::string("stage launch failed: ") + hipGetErrorString(e));
#ifdef MAFAT_TUNING
        dump_launch_trace(kind, S, shape, A, stream);
#endif
      }
      started[static_cast<size_t>(s - s_begin)] = launched ? 1 : 0;
      if (dst_b != eff(SD.dst_buf)) swapped = !swapped;
      if (fuse) {
        ++s;
        if (events) {
          for (int k = 0; k < 2; ++k) {
            hipEvent_t e2 = static_cast<hipEvent_t>(events[2 * (s - s_begin) + k]);
            if (e2 && hipEventRecord(e2, stream) != hipSuccess) return fail(MAFAT_EHIP, "hipEventRecord failed");
          }
        }
      }
    }
  }
  return MAFAT_OK;
}

int check_common(const mafat_plan* plan, int batch, int dtype) {
  if (!plan) return fail(MAFAT_EINVAL, "plan is NULL");
  if (batch < 1) return fail(MAFAT_EINVAL, "batch must be >= 1");
  if (dtype != MAFAT_F32 && dtype != MAFAT_BF16) return fail(MAFAT_EUNSUPPORTED, "dtype must be F32 or BF16");
  return MAFAT_OK;
}

}  // namespace
}  // namespace mafat

using namespace mafat;

namespace mafat {
namespace {
int run_group_checked(const mafat_plan* plan, int group, int batch, int dtype, const void* x, void* y,
                      const void* const* w, const float* const* scale, const float* const* bias, void* workspace,
                      size_t ws_bytes, void* stream, void* const* events) {
  int rc = check_common(plan, batch, dtype);
  if (rc != MAFAT_OK) return rc;
  if (group < 0 || group >= static_cast<int>(plan->groups.size()))
    return fail(MAFAT_EINVAL, "group index out of range");
  return run_group_impl(plan, group, 0, static_cast<int>(plan->groups[group].stages.size()), batch, dtype, x, y,
                        w, scale, bias, workspace, ws_bytes, static_cast<hipStream_t>(stream), events);
}
}  // namespace
}  // namespace mafat

extern "C" int mafat_run_group(const mafat_plan* plan, int32_t group, int32_t batch, int32_t dtype,
                               const void* x, void* y, const void* const* w,
                               const float* const* scale, const float* const* bias,
                               void* workspace, size_t ws_bytes, void* stream) {
  clear_error();
  return run_group_checked(plan, group, batch, dtype, x, y, w, scale, bias, workspace, ws_bytes, stream, nullptr);
}

extern "C" int mafat_run_group_timed(const mafat_plan* plan, int32_t group, int32_t batch, int32_t dtype,
                                     const void* x, void* y, const void* const* w,
                                     const float* const* scale, const float* const* bias,
                                     void* workspace, size_t ws_bytes, void* stream,
                                     void* const* events) {
  clear_error();
  if (!events) return fail(MAFAT_EINVAL, "events is NULL (use mafat_run_group to run without timestamps)");
  return run_group_checked(plan, group, batch, dtype, x, y, w, scale, bias, workspace, ws_bytes, stream, events);
}

extern "C" int mafat_run_stage(const mafat_plan* plan, int32_t group, int32_t stage, int32_t batch,
                               int32_t dtype, const void* x, void* y, const void* const* w,
                               const float* const* scale, const float* const* bias, void* workspace,
                               size_t ws_bytes, void* stream) {
  clear_error();
  int rc = check_common(plan, batch, dtype);
  if (rc != MAFAT_OK) return rc;
  if (group < 0 || group >= static_cast<int>(plan->groups.size()))
    return fail(MAFAT_EINVAL, "group index out of range");
  if (stage < 0 || stage >= static_cast<int>(plan->groups[group].stages.size()))
    return fail(MAFAT_EINVAL, "stage index out of range");
  if (plan->groups[group].tile_batch < plan->groups[group].ntiles || plan->groups[group].reuse)
    return fail(MAFAT_EUNSUPPORTED, "the group runs in tile batches or rows: its stages cannot run one at a time");
  return run_group_impl(plan, group, stage, stage + 1, batch, dtype, x, y, w, scale, bias, workspace, ws_bytes,
                        static_cast<hipStream_t>(stream), nullptr);
}

int mafat::run_network_impl(const mafat_plan* plan, int batch, int dtype, const void* x, void* y,
                            void* const* cut_bufs, const void* const* w, const float* const* scale,
                            const float* const* bias, void* workspace, size_t ws_bytes, void* stream) {
  int rc = check_common(plan, batch, dtype);
  if (rc != MAFAT_OK) return rc;
  const int ng = static_cast<int>(plan->groups.size());
  if (ng > 1 && !cut_bufs) return fail(MAFAT_EINVAL, "cut_bufs is NULL but the plan has several groups");
  for (int g = 0; g < ng; ++g) {
    const void* gin = (g == 0) ? x : cut_bufs[g - 1];
    void* gout = (g == ng - 1) ? y : cut_bufs[g];
    rc = run_group_impl(plan, g, 0, static_cast<int>(plan->groups[g].stages.size()), batch, dtype, gin, gout, w,
                        scale, bias, workspace, ws_bytes,
                        static_cast<hipStream_t>(stream), nullptr);
    if (rc != MAFAT_OK) return rc;
  }
  return MAFAT_OK;
}

extern "C" int mafat_run_network(const mafat_plan* plan, int32_t batch, int32_t dtype,
                                 const void* x, void* y, void* const* cut_bufs,
                                 const void* const* w, const float* const* scale,
                                 const float* const* bias, void* workspace, size_t ws_bytes,
                                 void* stream) {
  clear_error();
  return run_network_impl(plan, batch, dtype, x, y, cut_bufs, w, scale, bias, workspace, ws_bytes, stream);
}

extern "C" int mafat_plan_stage_fused(const mafat_plan* plan, int32_t group, int32_t stage, int32_t batch,
                                      int32_t dtype, int32_t* fused) {
  clear_error();
  if (!plan || !fused || group < 0 || group >= static_cast<int>(plan->groups.size()) || batch < 1) {
    set_error("plan and fused must be non-NULL, the group in range and batch >= 1");
    return MAFAT_EINVAL;
  }
  const Group& G = plan->groups[group];
  if (stage < 0 || stage >= static_cast<int>(G.stages.size())) {
    set_error("stage out of range");
    return MAFAT_EINVAL;
  }
  if (dtype != MAFAT_F32 && dtype != MAFAT_BF16) {
    set_error("dtype must be F32 or BF16");
    return MAFAT_EUNSUPPORTED;
  }
  *fused = (stage + 1 < static_cast<int>(G.stages.size()) &&
            stage_config(*plan, G, G.stages[stage], batch, dtype).fuse > 0) ? 1 : 0;
  return MAFAT_OK;
}

extern "C" int mafat_plan_stage_kernel(const mafat_plan* plan, int32_t group, int32_t stage, int32_t batch,
                                       int32_t dtype, int32_t* kernel) {
  clear_error();
  if (!plan || !kernel || group < 0 || group >= static_cast<int>(plan->groups.size()) || batch < 1) {
    set_error("plan and kernel must be non-NULL, the group in range and batch >= 1");
    return MAFAT_EINVAL;
  }
  const Group& G = plan->groups[group];
  if (stage < 0 || stage >= static_cast<int>(G.stages.size())) {
    set_error("stage out of range");
    return MAFAT_EINVAL;
  }
  if (dtype != MAFAT_F32 && dtype != MAFAT_BF16) {
    set_error("dtype must be F32 or BF16");
    return MAFAT_EUNSUPPORTED;
  }
  // the choice run_group_impl makes (both stages of a fused pair run in
  // the pair's kernel)
  const StageConfig c = stage_config(*plan, G, G.stages[stage], batch, dtype);
  if (c.fuse == 2 || c.fuse == -2) {
    *kernel = MAFAT_KERNEL_PATCH_FIRST;
  } else if (c.fuse == 1 || c.fuse == -1) {
    *kernel = MAFAT_KERNEL_PATCH_1X1;
  } else {
    switch (c.kind) {
      case K_CONV_PATCH: *kernel = MAFAT_KERNEL_PATCH; break;
      case K_CONV_RING: *kernel = MAFAT_KERNEL_RING; break;
      case K_CONV_MFMA: *kernel = MAFAT_KERNEL_MFMA_F32; break;
      case K_CONV_RGB:
      case K_CONV_RGB_MFMA: *kernel = MAFAT_KERNEL_FIRST_LAYER; break;
      case K_POOL: *kernel = MAFAT_KERNEL_POOL; break;
      default: *kernel = MAFAT_KERNEL_GENERIC; break;
    }
  }
  return MAFAT_OK;
}

#ifdef MAFAT_TUNING
// Tuning builds only: the configuration the runtime picks for stage s of
// group g: kind, bm, bn, depth, kg, kord, br, bc.
extern "C" int mafat_debug_config(const mafat_plan* plan, int32_t g, int32_t s, int32_t batch, int32_t dtype,
                                  int32_t* out) {
  const mafat::Stage& S = plan->groups[g].stages[s];
  const mafat::StageConfig c = mafat::choose_config(S, batch, dtype);
  const int32_t v[8] = {c.kind, c.bm, c.bn, c.depth, c.kg, c.kord, c.br, c.bc};
  for (int k = 0; k < 8; ++k) out[k] = v[k];
  return 0;
}
#endif

extern "C" int mafat_packed_weights_size(const mafat_plan* plan, int32_t layer, int32_t dtype, size_t* bytes) {
  clear_error();
  if (!plan || !bytes || layer < 0 || layer >= plan->n) {
    set_error("plan and bytes must be non-NULL and the layer in range");
    return MAFAT_EINVAL;
  }
  if (dtype != MAFAT_F32 && dtype != MAFAT_BF16) {
    set_error("dtype must be F32 or BF16");
    return MAFAT_EUNSUPPORTED;
  }
  int bn, nblk, nchunk;
  *bytes = packed_layout(*plan, layer, dtype, &bn, &nblk, &nchunk)
               ? static_cast<size_t>(nblk) * nchunk * 9 * bn * 32 * 2
               : 0;
  return MAFAT_OK;
}

extern "C" int mafat_pack_weights(const mafat_plan* plan, int32_t layer, int32_t dtype, const void* w_krsc,
                                  void* w_packed, void* stream) {
  size_t bytes = 0;
  int rc = mafat_packed_weights_size(plan, layer, dtype, &bytes);
  if (rc != MAFAT_OK) return rc;
  if (bytes == 0) return fail(MAFAT_EINVAL, "layer " + std::to_string(layer) + " takes KRSC weights (no packing)");
  if (!w_krsc || !w_packed || !aligned16(w_krsc) || !aligned16(w_packed))
    return fail(MAFAT_EINVAL, "weights must be non-NULL and 16-byte aligned");
  int bn, nblk, nchunk;
  packed_layout(*plan, layer, dtype, &bn, &nblk, &nchunk);
  const auto& d = plan->dims[layer];
  const hipError_t e = launch_pack_weights(static_cast<const uint16_t*>(w_krsc), static_cast<uint16_t*>(w_packed),
                                           d[5], d[2], bn, nblk, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(MAFAT_EHIP, std::string("pack launch failed: ") + hipGetErrorString(e));
  return MAFAT_OK;
}
