// kernel_args.h -- argument blocks passed by value to the stage kernels.
#pragma once

#include <hip/hip_ext.h>
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

// Band take-over copies one stage launch carries (row reuse).
constexpr int kMaxCarriedCopies = 4;

struct StageArgs {
  const void* src;
  void* dst;
  const void* w;        // conv: [cout][f][f][cin]
  const float* scale;   // conv: [cout]
  const float* bias;    // conv: [cout]
  int64_t src_fstride;  // elements between frames
  int64_t dst_fstride;
  int32_t in_h, in_w;   // extent of the stage input tensor (zero padding outside)
  int32_t f, s, p;      // filter, stride, padding of the stage's first layer (generic kernels)
  int32_t cin, cout;
  int32_t act;
  int32_t ntiles;
  int32_t nblk_n;       // blocks along output channels
  int32_t mblk_total;   // blocks along pixels, summed over tiles
  int32_t total_blocks; // batch * mblk_total * nblk_n
  int32_t chan_major;   // 1: blocks ordered channel-block-major (each XCD gets a slice of
                        //    the weights); 0: pixel-block-major (a slice of the pixels)
  int32_t w_packed;     // patch kernel: w is packed [cout/BN][cin/32][9][BN][32] (else KRSC)
  // Fused second layer (a 1x1 convolution of this stage's output, computed
  // in the same workgroup): weights [cout2][cin = cout], its scale and bias.
  const void* w2;
  const float* scale2;
  const float* bias2;
  int32_t cout2, act2;
  // Fused first layer (a 3-channel 3x3 convolution with a 2x2/2 max-pool
  // that produces this stage's input in the same workgroup): its weights
  // [cout0 = cin][3][3][3], scale, bias, activation and its input extent
  // (the group input, read through src / the tile source fields).
  const void* w0;
  const float* scale0;
  const float* bias0;
  int32_t act0, in_h0, in_w0;
  // Row reuse: band take-over copies carried by this launch.  With
  // copy_blocks > 0 the grid has a second row (blockIdx.y = 1) of
  // total_blocks workgroups, of which the first copy_blocks (at most
  // total_blocks) compute nothing: for each of copy_frames frames
  // (copy_fstride bytes apart from copy_base) they move copy_bytes[k] bytes
  // from byte offset copy_src[k] to copy_dst[k].  Offsets and lengths are
  // multiples of 16; no range overlaps another or anything the launch's own
  // workgroups read or write.
  unsigned char* copy_base;
  int64_t copy_fstride;
  int64_t copy_src[kMaxCarriedCopies], copy_dst[kMaxCarriedCopies], copy_bytes[kMaxCarriedCopies];
  int32_t copy_blocks, ncopy, copy_frames;
  int32_t mblk_prefix[kMaxTilesPerLaunch + 1];
  KTile tiles[kMaxTilesPerLaunch];
};

// Kernel families the runtime picks from.
enum KernelKind {
  K_CONV_MFMA = 0,      // matrix cores, operands staged through registers (fp32)
  K_CONV_DIRECT = 1,    // vector ALUs, any shape
  K_POOL = 2,           // lone max-pool
  K_CONV_RGB = 3,       // 3-channel first layer, vector ALUs
  K_CONV_RGB_MFMA = 4,  // 3-channel first layer, matrix cores (bf16)
  K_CONV_RING = 5,      // matrix cores, operands streamed into an LDS ring (bf16)
  K_CONV_PATCH = 6      // 3x3 on the matrix cores, input patch shared by the taps (bf16)
};

// Conv outputs (rows x columns) per workgroup of the matrix-core first-layer
// kernel.
constexpr int kRgbBlockRows = 16, kRgbBlockCols = 32;

// Block shape of the MFMA kernel: output pixels x output channels, the
// depth of its load pipeline (3 to 6 stages of 128 bytes of K in flight) and
// the number of K groups (1: 4 waves; 2: 8 waves, each group of 4 multiplies
// one 64-byte half of every stage).
// For the LDS-ring kernel, depth is the number of ring slots, wgm x wgn
// the wave arrangement of one K group and kord the K order (0: tap-major,
// 1: channel-block-major).
struct MfmaShape {
  int bm, bn, depth, kg;
  int wgm, wgn, kord;
  int br, bc;  // patch kernel: block of br x bc conv outputs (bm >= br * bc GEMM rows)
};

// Instantiated patch kernel shapes: (br, bc, bm, bn, wgm, wgn, ring slots).
#define MAFAT_PATCH_SHAPES                \
  MAFAT_PATCH(16, 16, 256, 64, 8, 1, 2)   \
  MAFAT_PATCH(12, 12, 192, 64, 4, 2, 2)   \
  MAFAT_PATCH(12, 16, 192, 64, 4, 2, 2)   \
  MAFAT_PATCH(16, 12, 192, 64, 4, 2, 2)   \
  MAFAT_PATCH(10, 10, 128, 32, 4, 1, 2)   \
  MAFAT_PATCH(8, 8, 64, 32, 4, 2, 2)      \
  MAFAT_PATCH(8, 16, 128, 64, 8, 1, 1)    \
  MAFAT_PATCH(12, 16, 192, 64, 4, 2, 1)   \
  MAFAT_PATCH(14, 18, 256, 64, 4, 2, 1)   \
  MAFAT_PATCH(8, 16, 128, 128, 4, 2, 1)
#ifdef MAFAT_TUNING
#define MAFAT_PATCH_TUNE_SHAPES           \
  MAFAT_PATCH(10, 10, 128, 32, 4, 1, 3)   \
  MAFAT_PATCH(10, 10, 128, 32, 4, 1, 4)   \
  MAFAT_PATCH(16, 12, 192, 64, 4, 2, 1)   \
  MAFAT_PATCH(16, 16, 256, 64, 8, 1, 1)   \
  MAFAT_PATCH(8, 16, 128, 64, 4, 1, 1)    \
  MAFAT_PATCH(8, 16, 128, 64, 2, 2, 1)
#else
#define MAFAT_PATCH_TUNE_SHAPES
#endif

// Instantiated LDS-ring kernel shapes: (bm, bn, wgm, wgn, kg, ring slots, K order).
#define MAFAT_RING_SHAPES             \
  MAFAT_RING(32, 64, 2, 2, 1, 3, 1)   \
  MAFAT_RING(64, 32, 2, 2, 1, 3, 1)   \
  MAFAT_RING(64, 64, 2, 2, 1, 3, 1)   \
  MAFAT_RING(128, 64, 2, 2, 2, 4, 1)  \
  MAFAT_RING(128, 128, 2, 2, 2, 3, 1)
#ifdef MAFAT_TUNING
#define MAFAT_RING_TUNE_SHAPES        \
  MAFAT_RING(32, 64, 2, 2, 1, 6, 1)   \
  MAFAT_RING(32, 64, 2, 2, 1, 8, 1)   \
  MAFAT_RING(32, 32, 2, 2, 1, 3, 1)   \
  MAFAT_RING(32, 32, 2, 2, 1, 4, 1)   \
  MAFAT_RING(64, 64, 2, 2, 2, 4, 1)
#else
#define MAFAT_RING_TUNE_SHAPES
#endif

// Launch one stage chunk.  `units_per_block` is what the kernel covers per
// block along the pixel axis (used to fill mblk_prefix by the caller).
// Optional kernel timestamps: `start` is recorded when the launched kernel
// starts and `stop` when it ends (hipExtLaunchKernel: timestamps of the
// dispatch itself, no extra packets between kernels); null for none.
struct LaunchEvents {
  hipEvent_t start, stop;
};
hipError_t launch_stage(int kind, int dtype, int f, bool pool, MfmaShape shape,
                        const StageArgs& args, hipStream_t stream, LaunchEvents ev);

// Launch one bf16 LDS-ring convolution stage chunk (conv_ring.hip).
hipError_t launch_conv_ring(int f, bool pool, const MfmaShape& shape, const StageArgs& args,
                            hipStream_t stream, LaunchEvents ev);

// Launch one bf16 3x3 patch-kernel stage chunk (conv_patch.hip).
hipError_t launch_conv_patch(bool pool, const MfmaShape& shape, const StageArgs& args, hipStream_t stream,
                             LaunchEvents ev);

// Launch a bf16 3x3 stage with 128 output channels fused with the 1x1
// stage (64 outputs) that follows it (conv_patch.hip): 8x16 blocks of all
// 128 channels; args.w2 / scale2 / bias2 / cout2 / act2 describe the 1x1
// layer, the destination fields the 1x1 stage's output.
hipError_t launch_conv_patch_fused(const StageArgs& args, hipStream_t stream, LaunchEvents ev);

// Launch a bf16 3-channel first layer with its 2x2/2 pool fused with the
// 3x3 stage (32 -> 64 channels, fused pool) that follows it
// (conv_patch.hip): each workgroup computes the first layer's pooled output
// over its block's input patch into LDS, then the 3x3 stage from there.
// args describe the 3x3 stage (tiles: its computed rectangles and output;
// the source fields: the group input), w0 / scale0 / bias0 / act0 / in_h0 /
// in_w0 the first layer.
hipError_t launch_conv_patch_first(const MfmaShape& shape, const StageArgs& args, hipStream_t stream,
                                   LaunchEvents ev);

// Instantiated block shapes of the first-layer pair: (br, bc, bm, wgm, wgn),
// 64 channels, one ring slot.
#define MAFAT_FIRST_SHAPES           \
  MAFAT_FIRST(12, 16, 192, 4, 2)     \
  MAFAT_FIRST(14, 18, 256, 4, 2)

// Repack one layer's KRSC bf16 weights into the patch kernel's packed layout.
hipError_t launch_pack_weights(const uint16_t* src, uint16_t* dst, int cout, int cin, int bn, int nblk,
                               hipStream_t stream);

// Row reuse: the rows a tile row takes over from its predecessor's bands,
// every band at once.  Copy k moves bytes[k] bytes from byte offset src[k]
// to dst[k] of each frame's scratch (frames fstride bytes apart); no two
// copies' ranges overlap.
constexpr int kMaxBandCopies = 16;
struct BandCopyArgs {
  int64_t src[kMaxBandCopies], dst[kMaxBandCopies], bytes[kMaxBandCopies];
  int64_t fstride;
  int32_t ncopy;
};
hipError_t launch_band_copy(void* scratch, const BandCopyArgs& args, int batch, hipStream_t stream);

// Pixel-axis block size of each kernel family.
int block_units(int kind, MfmaShape shape);

}  // namespace mafat
