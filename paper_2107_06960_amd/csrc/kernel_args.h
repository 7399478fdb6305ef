// kernel_args.h -- argument blocks passed by value to the stage kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "mafat_internal.h"

namespace mafat {

// One tile of one stage (see TileGeom); 16-bit coordinates keep the block
// of 64 tiles small enough for the kernel argument segment.
struct KTile {
  int16_t cy0, cx0, ch, cw;  // computed rectangle
  int16_t sy0, sx0, sw;      // source buffer origin and row width (pixels)
  int16_t dy0, dx0, dw;      // destination buffer origin and row width
  int32_t src_off, dst_off;  // element offsets within one frame's buffer
};

struct StageArgs {
  const void* src;
  void* dst;
  const void* w;        // conv: [cout][f][f][cin]
  const float* scale;   // conv: [cout]
  const float* bias;    // conv: [cout]
  int64_t src_fstride;  // elements between frames
  int64_t dst_fstride;
  int32_t in_h, in_w;   // extent of the stage input tensor (zero padding outside)
  int32_t cin, cout;
  int32_t act;
  int32_t ntiles;
  int32_t nblk_n;       // blocks along output channels
  int32_t mblk_total;   // blocks along pixels, summed over tiles
  int32_t total_blocks; // batch * mblk_total * nblk_n
  int32_t chan_major;   // 1: blocks ordered channel-block-major (each XCD gets a slice of
                        //    the weights); 0: pixel-block-major (a slice of the pixels)
  int32_t mblk_prefix[kMaxTilesPerLaunch + 1];
  KTile tiles[kMaxTilesPerLaunch];
};

// Kernel families the runtime picks from.
enum KernelKind { K_CONV_MFMA = 0, K_CONV_DIRECT = 1, K_POOL = 2, K_CONV_RGB = 3, K_CONV_RGB_MFMA = 4 };

// Conv outputs (rows x columns) per workgroup of the matrix-core first-layer
// kernel.
constexpr int kRgbBlockRows = 32, kRgbBlockCols = 32;

// Block shape of the MFMA kernel: output pixels x output channels, the
// depth of its load pipeline (3 to 6 stages of 128 bytes of K in flight) and
// the number of K groups (1: 4 waves; 2: 8 waves, each group of 4 multiplies
// one 64-byte half of every stage).
struct MfmaShape {
  int bm, bn, depth, kg;
};

// Launch one stage chunk.  `units_per_block` is what the kernel covers per
// block along the pixel axis (used to fill mblk_prefix by the caller).
hipError_t launch_stage(int kind, int dtype, int f, bool pool, MfmaShape shape,
                        const StageArgs& args, hipStream_t stream);

// Pixel-axis block size of each kernel family.
int block_units(int kind, MfmaShape shape);

}  // namespace mafat
