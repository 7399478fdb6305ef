// mafat_internal.h -- plan structures shared by the planner (plan.cpp), the
// runtime (run.hip) and the kernels (kernels.hip).  Not part of the ABI.
#pragma once

#include <array>
#include <cstdint>
#include <string>
#include <vector>

#include "../../include/mafat.h"

namespace mafat {

// Tiles one kernel launch can describe in its argument block; a stage with
// more tiles is launched in chunks.
constexpr int kMaxTilesPerLaunch = 64;

// Largest tensor extent the 16-bit tile descriptors can address.
constexpr int kMaxExtent = 32767;

// Largest filter and stride of a layer (the generic kernels loop over the
// window at run time).
constexpr int kMaxFilter = 11, kMaxStride = 4;

enum StageKind { STAGE_CONV = 0, STAGE_POOL = 1 };

// Where a stage reads from / writes to.
enum BufKind { BUF_GROUP_IO = -1, BUF_SCRATCH0 = 0, BUF_SCRATCH1 = 1 };

// Geometry of one tile in one stage, all in global coordinates.
struct TileGeom {
  // The rectangle the stage's kernel computes: for a conv stage the conv
  // output rectangle (before any fused pool), for a pool stage the pool
  // output rectangle.
  int cy0, cx0, ch, cw;
  // Source buffer: the element (y, x, c) of the stage input lives at
  // src_off + ((y - sy0) * sw + (x - sx0)) * C + c of one frame's buffer.
  int sy0, sx0, sw;
  // Destination buffer, the same way for the stage output.
  int dy0, dx0, dw;
  int64_t src_off, dst_off;
};

struct Stage {
  int kind;          // StageKind
  int first, last;   // layers [first, last]
  bool pool;         // conv stage with a fused 2x2/2 max-pool
  int in_h, in_w, cin;     // input tensor of the first layer
  int out_h, out_w, cout;  // output tensor of the last layer
  int f, s, p, act;        // filter, stride, padding (conv or pool), activation (conv)
  int src_buf, dst_buf;    // BufKind
  std::vector<TileGeom> tiles;
  // Row reuse (an output that is not the group's): per tile row i, the
  // first row of its output band (band_lo[i]) and the rows it computes,
  // [row_b[i], row_b[i + 1]) of the stage output; band_rows = the largest
  // band, row_b[i + 1] - band_lo[i]; band_copies = 1 when every row's
  // take-over from its predecessor can move within one band buffer (source
  // and destination rows apart), else 2 (rows alternate between two).
  std::vector<int> band_lo, row_b;
  int band_rows = 0, band_copies = 0;
};

struct Group {
  int l0, l1;        // layers [l0, l1]
  int rows, cols, ntiles;
  std::vector<mafat_rect> in_r, out_r;  // [tile * nlayers + (l - l0)]
  std::vector<Stage> stages;
  int64_t scratch_elems;  // per tile per scratch buffer (stage partition: per scratch buffer)
  int nbufs;              // scratch buffers (0, 1 or 2)
  int64_t scratch_frame;  // scratch elements of one frame
  bool partition;         // stage partition: every stage output computed once (full tensors)
  bool reuse = false;     // row reuse: tile rows in order, stage outputs in row bands
  int tile_batch;         // tiles run through the stages together (ntiles unless
                          // mafat_plan_set_tile_batch set fewer); scratch per batch
  int64_t macs_exec, macs_untiled;
};

}  // namespace mafat

struct mafat_plan {
  int n, in_h, in_w, in_c;
  std::vector<mafat_layer> layers;
  std::vector<std::array<int, 6>> dims;  // in_h, in_w, in_c, out_h, out_w, out_c
  std::vector<mafat::Group> groups;
  bool packed_weights = false;  // MAFAT_PLAN_PACKED_WEIGHTS
};

namespace mafat {

// How one stage runs for a given batch and dtype (chosen by the runtime,
// also used to size the workspace).
struct StageConfig {
  int kind;          // KernelKind
  int bm, bn, depth; // matrix-core kernel block tile and pipeline depth
  int kg;            // matrix-core kernel K groups (1 or 2, see MfmaShape)
  int kord;          // LDS-ring kernel K order (see MfmaShape)
  int br, bc;        // patch kernel block (see MfmaShape)
  int wgm, wgn;      // wave arrangement (see MfmaShape)
  int chan_major;    // block order (see StageArgs::chan_major)
  int64_t blocks;    // output blocks per frame (pixel blocks x channel blocks)
  int fuse;          // 1: runs fused with the next (1x1) stage when both are launched
                     //    together; -1: the second stage of such a pair; 0: neither
};
StageConfig choose_config(const Stage& S, int batch, int dtype);

// The configuration a stage runs with in a plan (choose_config with the
// batch the plan's weight layout fixes, and the generic kernel for frames
// too large for 32-bit offsets).
StageConfig stage_config(const mafat_plan& P, const Group& G, const Stage& S, int batch, int dtype);

// Packed weights of a conv layer (run by the bf16 3x3 patch kernel in a
// plan with packed weights): [channel block][32-channel chunk][tap][BN
// rows][32 channels], rows past c_out zero.  Returns false (and bn = 0)
// for a layer whose weights stay KRSC.
bool packed_layout(const mafat_plan& P, int layer, int dtype, int* bn, int* nblk, int* nchunk);

// Workspace layout for one group: the ping-pong scratch buffers of every
// tile of every frame, 256-byte aligned.  Sizes in bytes.
struct WorkspaceLayout {
  size_t scratch, total;
};
WorkspaceLayout workspace_layout(const mafat_plan& P, const Group& G, int batch, int dtype);

// Row reuse: the band buffers of one frame for a dtype.  Tile row i writes
// stage s's output into the band at base[s][i % 2] (elements from the
// frame's scratch start, 256-byte aligned; the two are one buffer when
// band_copies is 1), or there is none (base -1: the group output, or kept
// on chip by a fused kernel).
struct BandLayout {
  std::vector<std::array<int64_t, 2>> base;
  int64_t frame;  // elements of one frame's bands
};
BandLayout band_layout(const mafat_plan& P, const Group& G, int dtype);

// Every group of a plan in order (mafat_run_network without clearing the
// error state), on the given workspace; stream is a hipStream_t.
int run_network_impl(const mafat_plan* plan, int batch, int dtype, const void* x, void* y,
                     void* const* cut_bufs, const void* const* w, const float* const* scale,
                     const float* const* bias, void* workspace, size_t ws_bytes, void* stream);

// Thread-local error detail (mafat_last_error).
void set_error(const std::string& msg);
void clear_error();
}  // namespace mafat
