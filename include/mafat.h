/*
 * mafat.h -- C ABI of the MI355X (gfx950) fused-tile-partitioning library.
 *
 * Method: MAFAT, memory-aware fusing and tiling (Farley & Gerstlauer,
 * arXiv 2107.06960), built on fused tile partitioning (FTP).  A stack of
 * convolution and max-pool layers is split into layer groups (section 4:
 * one group, or groups separated by cuts; group g covers layers
 * [group_start[g], group_start[g+1])).  Each group has its own output tile
 * grid (section 4; notation N1xM1/c/N2xM2 of section 5.1).  Every tile's
 * input region, halo included, is back-projected through the group's layers
 * (the "Grid"/traversal function of section 4.1); the tile is pushed through
 * every layer of the group without its intermediates being written out as
 * full tensors, and the tile outputs are stitched into the group's output
 * tensor, which the next group re-tiles (section 4).
 *
 * Conventions
 *   - Activations are NHWC, frame-major: element (b, y, x, c) of an
 *     H x W x C tensor is at ((b*H + y)*W + x)*C + c.
 *   - Convolution weights are [c_out][f][f][c_in] (KRSC), in the run dtype.
 *     Per-layer folded batch-norm scale and bias are float32 [c_out].
 *   - Every convolution computes  v = scale[c] * sum(...) + bias[c], then
 *     its activation (linear, or leaky ReLU with slope 0.1); padding is zero
 *     and applies only outside the image, never at a tile border.
 *   - Rectangles are half-open, in the global coordinates of the tensor they
 *     index: {y0, y1, x0, x1} covers rows [y0, y1) and columns [x0, x1).
 *   - dtype MAFAT_F32: float32 activations and weights, float32 accumulate.
 *     dtype MAFAT_BF16: bfloat16 activations and weights, float32 accumulate;
 *     every layer output is rounded to bfloat16 (nearest, ties to even).
 *   - Supported layers: convolution and max-pool with a square filter
 *     1 <= f <= 11, stride 1 <= s <= 4 and padding 0 <= p < f; output extent
 *     floor((in + 2p - f) / s) + 1.  A max-pool takes the maximum over the
 *     in-image elements of its window.  3x3 and 1x1 "same" convolutions
 *     (s = 1, p = (f-1)/2) run on the matrix cores, a 2x2/2 max-pool after
 *     a convolution in its epilogue; other layers on generic vector-ALU
 *     kernels.  Tensor extents must be at most 32767.
 *
 * Ownership and threading
 *   - A plan is created and destroyed by the library, read-only after
 *     creation (except mafat_plan_set_tile_batch, which must not run while
 *     other threads use the plan), and may be shared between threads.
 *   - Every device buffer (input, output, cut tensors, weights, scale, bias,
 *     workspace) is owned by the caller.  The library never allocates or
 *     frees device memory and never synchronises a stream; run functions only
 *     enqueue kernels on the given stream and return.
 *   - Pointer arrays (w, scale, bias, cut_bufs, events) are host arrays of
 *     device pointers / event handles, read during the call only.
 *   - Device tensors (x, y, cut tensors, weights, scale, bias) must be
 *     16-byte aligned (EINVAL otherwise); the workspace 256-byte aligned.
 *
 * Errors
 *   - Every int-returning function returns a mafat_status.  No C++
 *     exception crosses this boundary.  mafat_last_error() gives a
 *     thread-local message about the last failing call.
 *   - Run functions return MAFAT_EHIP if a launch reports an error; faults
 *     that happen while kernels execute surface at the caller's next
 *     synchronisation of the stream.
 */
#ifndef MAFAT_H
#define MAFAT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  MAFAT_OK = 0,
  MAFAT_EINVAL = -1,        /* null pointer, bad index or bad argument value */
  MAFAT_ESHAPE = -2,        /* layer list / input shape / grid inconsistent   */
  MAFAT_EUNSUPPORTED = -3,  /* valid request this library does not implement */
  MAFAT_EWORKSPACE = -4,    /* workspace smaller than mafat_workspace_size    */
  MAFAT_EHIP = -5,          /* the HIP runtime reported an error              */
  MAFAT_ENOMEM = -6         /* host allocation failed                         */
} mafat_status;

typedef enum { MAFAT_CONV = 0, MAFAT_MAXPOOL = 1 } mafat_op;
typedef enum { MAFAT_ACT_LINEAR = 0, MAFAT_ACT_LEAKY01 = 1 } mafat_act;
typedef enum { MAFAT_F32 = 0, MAFAT_BF16 = 1 } mafat_dtype;
typedef enum { MAFAT_MEM_DEVICE = 0, MAFAT_MEM_PAPER = 1, MAFAT_MEM_DEVICE_SEQ = 2 } mafat_mem_model;

/* One layer (section 4.1 describes a layer by width, height, filter size
 * and stride; channels, padding and activation are added).  c_out and act
 * are ignored for max-pool. */
typedef struct {
  int32_t op, c_out, f, s, p, act;
} mafat_layer;

typedef struct {
  int32_t y0, y1, x0, x1;
} mafat_rect;

typedef struct mafat_plan mafat_plan;

/* Builds a plan: shape inference, per-group output tile partition and
 * per-tile, per-layer region back-projection (sections 4 and 4.1).
 *   layers[n_layers]          the stack, applied to an in_h x in_w x in_c input
 *   group_start[n_groups]     first layer of each group; strictly increasing,
 *                             group_start[0] == 0
 *   grid_rows/cols[n_groups]  each group's output tile grid; 1 <= rows <= the
 *                             group output's height (cols: width)
 * Tile (i, j) of an H x W group output covers rows [floor(iH/rows),
 * floor((i+1)H/rows)) and columns likewise; tiles are numbered row-major.
 * On success *out owns the plan (free with mafat_plan_destroy).
 * Errors: EINVAL (null pointer, n < 1), ESHAPE (non-positive extent, group
 * or grid out of range, extent > 32767), EUNSUPPORTED (layer kind outside
 * the supported set). */
int mafat_plan_create(const mafat_layer* layers, int32_t n_layers, int32_t in_h,
                      int32_t in_w, int32_t in_c, const int32_t* group_start,
                      int32_t n_groups, const int32_t* grid_rows,
                      const int32_t* grid_cols, mafat_plan** out);

/* Plan flags (mafat_plan_create_flags). */
enum {
  /* Stage partition: the data-reuse variant of fused tile partitioning
   * (section 3: neighbouring tiles share the overlap they would otherwise
   * both compute), taken to whole stages.  Every stage of a group runs over
   * all tiles before the next one starts; each stage's output is split into
   * the group's grid (floor boundaries, as the group output) and every tile
   * computes only its own part, into a whole-tensor copy of the stage output
   * in the workspace, from which the next stage reads its halo.  Nothing is
   * computed twice, but nothing is fused per tile either: this is the
   * untiled layer-by-layer execution with each layer's work split into the
   * group's tiles.  Results equal the untiled network's (up to accumulation
   * order); executed MACs equal the untiled ones; the workspace holds two
   * whole stage outputs per frame.  mafat_plan_regions and the paper's
   * memory model keep describing the plain (recomputing) partition. */
  MAFAT_PLAN_STAGE_PARTITION = 1,
  /* Packed weights: for every conv layer whose mafat_packed_weights_size is
   * nonzero (bf16 3x3 layers run by the patch kernel), the w[layer] passed
   * to the run functions is that layer's weights repacked by
   * mafat_pack_weights: per block of output channels and 32-channel chunk,
   * the nine taps' rows one contiguous run, so the kernel's weight loads
   * read whole cache lines.  The other layers keep KRSC.  Every batch runs
   * the stage configurations chosen for one frame (the packing follows
   * their output-channel blocks).  A layout of this library, not of the
   * paper. */
  MAFAT_PLAN_PACKED_WEIGHTS = 2,
  /* Row reuse: the data reuse of section 3 (a tile takes the overlap that
   * tiles run before it already computed, instead of computing it again)
   * with the tiles run one grid row after another, each row through all
   * stages of the group before the next (the tiles of a row together).
   * Each stage's output is split into computed parts: the group output
   * along the group's tile boundaries, and every earlier stage output along
   * the back-projected ends of the next stage's parts, so that a tile row
   * computes exactly the rows below its predecessors that its own next
   * stage reads, and nothing twice.  Per stage output the workspace holds
   * a band: the rows a tile row computes plus the rows above them that its
   * next stage reads (taken over from the previous row's band by a copy on
   * the stream), the full width, two such bands per stage output
   * alternating between rows.  Stage outputs that a fused kernel keeps on
   * chip get no band.  Results equal the untiled network's (up to
   * accumulation order); executed MACs equal the untiled ones;
   * mafat_plan_set_tile_batch and mafat_run_stage do not apply
   * (EUNSUPPORTED).  Combines with
   * MAFAT_PLAN_PACKED_WEIGHTS and with given tile boundaries, not with
   * MAFAT_PLAN_STAGE_PARTITION.  mafat_plan_regions and the paper's memory
   * model keep describing the plain (recomputing) partition. */
  MAFAT_PLAN_ROW_REUSE = 4
};

/* mafat_plan_create (sections 4 and 4.1) with flags
 * (MAFAT_PLAN_STAGE_PARTITION or MAFAT_PLAN_ROW_REUSE, and/or
 * MAFAT_PLAN_PACKED_WEIGHTS, or 0).
 * Errors: those of mafat_plan_create, EINVAL for unknown flags and
 * EUNSUPPORTED for MAFAT_PLAN_STAGE_PARTITION with MAFAT_PLAN_ROW_REUSE. */
int mafat_plan_create_flags(const mafat_layer* layers, int32_t n_layers, int32_t in_h,
                            int32_t in_w, int32_t in_c, const int32_t* group_start,
                            int32_t n_groups, const int32_t* grid_rows,
                            const int32_t* grid_cols, int32_t flags, mafat_plan** out);

/* mafat_plan_create_flags with each group's tile boundaries given: variable
 * tiling, which section 6 proposes as future work (end tiles sized unlike
 * the inner ones, so that the tiles' tasks vary less and the largest
 * footprint falls).
 *   row_bounds  concatenated over groups, grid_rows[g] + 1 row boundaries
 *               of group g's output: 0 = b[0] < b[1] < ... < b[rows] = the
 *               output height; tile row i covers rows [b[i], b[i+1])
 *   col_bounds  the same for columns (grid_cols[g] + 1 per group)
 * Either may be NULL: the floor split of mafat_plan_create on that axis for
 * every group.  Host arrays, read during the call only.  Everything else
 * (regions, stages, kernels, workspace, predictor) follows the given tiles.
 * Errors: those of mafat_plan_create_flags; ESHAPE (boundaries not strictly
 * increasing from 0 to the group output extent); EUNSUPPORTED (boundaries
 * with MAFAT_PLAN_STAGE_PARTITION, which splits every stage evenly). */
int mafat_plan_create_bounds(const mafat_layer* layers, int32_t n_layers, int32_t in_h,
                             int32_t in_w, int32_t in_c, const int32_t* group_start,
                             int32_t n_groups, const int32_t* grid_rows,
                             const int32_t* grid_cols, const int32_t* row_bounds,
                             const int32_t* col_bounds, int32_t flags, mafat_plan** out);

/* Balanced tile boundaries for variable tiling (section 6) of the group of
 * layers [first_layer, last_layer] of the stack (shapes inferred from the
 * in_h x in_w x in_c input): `rows` parts of the group output's height into
 * row_bounds[rows + 1], `cols` parts of its width into col_bounds[cols + 1]
 * (either pointer may be NULL to skip that axis).  Along an axis a tile's
 * task extent is the extent of the input region of first_layer that its
 * output interval reads (back-projected through the group, clipped to the
 * tensor, as mafat_plan_regions).  The boundaries minimise the largest task
 * extent, then the sum of the squared task extents, and are the first such
 * list in lexicographic order (exact: bisection on the largest extent, then
 * a dynamic programme).  Pass them to mafat_plan_create_bounds.
 * Errors: EINVAL (null layers, layer range outside the stack), the shape
 * errors of mafat_plan_create, ESHAPE (parts outside 1 .. extent),
 * EUNSUPPORTED (a search too large to run). */
int mafat_balanced_bounds(const mafat_layer* layers, int32_t n_layers, int32_t in_h,
                          int32_t in_w, int32_t in_c, int32_t first_layer,
                          int32_t last_layer, int32_t rows, int32_t cols,
                          int32_t* row_bounds, int32_t* col_bounds);

/* Tile batches (the order of section 4, where the tiles of a group are
 * processed one after another): run at most `tiles` tiles of a group at a
 * time (0: all tiles at once, the default).  mafat_run_group / mafat_run_network then
 * take the group's tiles in row-major batches of `tiles`, each batch through
 * all of the group's stages before the next, and the workspace holds one
 * batch's intermediates instead of every tile's.  With tiles = 1 this is
 * the paper's execution order (tiles one after another, Sec. 4), whose peak
 * memory falls with finer grids; on the GPU a batch must still fill the
 * device to run fast.  Results are bit-identical to the default.  Call
 * before sizing the workspace; mafat_run_stage then fails (EUNSUPPORTED)
 * for groups split into several batches, and the per-stage events of
 * mafat_run_group_timed enclose the stage's first to last launch (other stages'
 * launches in between).  Errors: EINVAL (NULL, tiles < 0), EUNSUPPORTED
 * (a plan with MAFAT_PLAN_STAGE_PARTITION and 0 < tiles < a group's tile
 * count; a plan with MAFAT_PLAN_ROW_REUSE).  Not thread-safe: it rewrites the plan's per-tile workspace
 * offsets, so no other thread may use the plan (run it, size its workspace)
 * during the call; the plan is read-only again afterwards. */
int mafat_plan_set_tile_batch(mafat_plan* plan, int32_t tiles);

/* Weight layout of this library's 3x3 kernels (no counterpart in the paper,
 * whose layers hold their weights as the framework stores them).
 * Bytes of the packed weights of conv layer `layer` in `dtype` (device
 * buffer, 16-byte aligned, caller-owned); 0 when the layer's weights are
 * passed as KRSC (plan without MAFAT_PLAN_PACKED_WEIGHTS, f32, 1x1 or
 * first-layer convolutions, pools).  Errors: EINVAL, EUNSUPPORTED (dtype). */
int mafat_packed_weights_size(const mafat_plan* plan, int32_t layer, int32_t dtype, size_t* bytes);

/* Enqueues on `stream` the repack of conv layer `layer`'s KRSC weights
 * (w_krsc, device, c_out x 3 x 3 x c_in in `dtype`) into w_packed (device,
 * mafat_packed_weights_size bytes); both 16-byte aligned, not overlapping.
 * Done once per set of weights; the packed buffer then serves every run of
 * plans with the same layers, grid and flags.  Errors: EINVAL (no packing
 * for this layer, null or misaligned pointer), EUNSUPPORTED, EHIP. */
int mafat_pack_weights(const mafat_plan* plan, int32_t layer, int32_t dtype, const void* w_krsc,
                       void* w_packed, void* stream);

/* Frees a plan made by mafat_plan_create (NULL is ignored). */
void mafat_plan_destroy(mafat_plan* plan);

/* Shape inference (section 4.1 describes each layer by its width, height,
 * filter and stride; out = floor((in + 2p - f) / s) + 1):
 * dims[6] = in_h, in_w, in_c, out_h, out_w, out_c of layer `layer`.
 * Errors: EINVAL. */
int mafat_plan_layer_shape(const mafat_plan* plan, int32_t layer, int32_t dims[6]);

/* Layer groups and their grids (section 4: a group covers the layers up to
 * a cut and has its own N x M tile grid):
 * group g's first layer, number of layers and number of tiles.
 * Any output pointer may be NULL.  Errors: EINVAL. */
int mafat_plan_group(const mafat_plan* plan, int32_t group, int32_t* first_layer,
                     int32_t* n_layers, int32_t* n_tiles);

/* Number of tiles (grid rows x columns) of group g's output partition
 * (section 4: the group output is split into an N x M grid of tiles).
 * Errors: EINVAL (NULL plan or pointer, group out of range). */
int mafat_plan_num_tiles(const mafat_plan* plan, int32_t group, int32_t* n_tiles);

/* Per-tile regions (section 4.1, the "Grid"/traversal function giving each
 * tile's extent at every layer with its overlap; computed here as the exact
 * receptive-field interval, clipped to the tensor).
 * Region table of group g, [tile][layer - first_layer] (tiles row-major):
 * in_rects = the region of the layer's input the tile reads (halo included,
 * clipped to the tensor); out_rects = the region of the layer's output the
 * tile computes.  Within a tile, in_rects[k] == out_rects[k-1].  The last
 * layer's out_rects partition the group output.  capacity is the number of
 * elements each array can hold (>= n_tiles * n_layers; EINVAL otherwise).
 * Either array may be NULL. */
int mafat_plan_regions(const mafat_plan* plan, int32_t group, mafat_rect* in_rects,
                       mafat_rect* out_rects, int64_t capacity);

/* Work accounting (section 4: overlapping regions are computed by every
 * tile that needs them, so finer grids and deeper groups execute more).
 * Multiply-accumulates of group g per frame: executed (every tile's
 * convolution outputs, halo recompute included, times c_in*f*f) and untiled
 * (the same layers on whole tensors).  Either pointer may be NULL. */
int mafat_plan_macs(const mafat_plan* plan, int32_t group, int64_t* executed,
                    int64_t* untiled);

/* Execution stages of this library (a tile's layers run in order, section
 * 4; a convolution and the max-pool after it run as one stage).
 * Number of kernel stages group g runs and, for stage s, its first and last
 * layer (a convolution directly followed by a 2x2 max-pool in the same group
 * is one stage; every other layer is a stage of its own).  Used for
 * per-stage timing with the events argument of mafat_run_group_timed.
 * Errors: EINVAL. */
int mafat_plan_stages(const mafat_plan* plan, int32_t group, int32_t* n_stages);
int mafat_plan_stage_layers(const mafat_plan* plan, int32_t group, int32_t stage,
                            int32_t* first_layer, int32_t* last_layer);

/* Layer fusion inside a tile (section 3: a tile's sub-convolutions are fused
 * across the layers of its group and run as one unit), taken down to a
 * workgroup's block of pixels.
 * *fused = 1 if mafat_run_group / mafat_run_network run stage `stage` of
 * group g together with stage + 1 in one kernel for this batch and dtype,
 * else 0.  Two pairs qualify (bfloat16): a 3x3 convolution with 128
 * outputs and no pool whose next stage is a 1x1 convolution 128 -> 64 or
 * 128 -> 32 over the same rectangles (YOLOv2's layers 4-5: the 1x1 GEMM
 * runs on the 3x3 outputs held in LDS), and a group's first stage when it is a 3-channel
 * 3x3 convolution with 32 outputs and a 2x2/2 pool followed by a 3x3
 * convolution 32 -> 64 with a 2x2/2 pool (YOLOv2's layers 0-3: each
 * workgroup computes the first layer's pooled output for its own input
 * patch in LDS).  In both the intermediate never goes to memory.
 * mafat_run_stage always runs one stage.  Errors: EINVAL (NULL, index out
 * of range), EUNSUPPORTED (dtype). */
int mafat_plan_stage_fused(const mafat_plan* plan, int32_t group, int32_t stage, int32_t batch,
                           int32_t dtype, int32_t* fused);

/* Kernel families a stage can run on (mafat_plan_stage_kernel). */
typedef enum {
  MAFAT_KERNEL_PATCH = 0,        /* bf16 3x3 on the matrix cores, the input patch shared by the taps */
  MAFAT_KERNEL_PATCH_FIRST = 1,  /* the same with the 3-channel first layer and its pool computed inside */
  MAFAT_KERNEL_PATCH_1X1 = 2,    /* the same with the following 1x1 convolution computed inside */
  MAFAT_KERNEL_RING = 3,         /* bf16 implicit GEMM through an LDS ring (1x1 convolutions) */
  MAFAT_KERNEL_MFMA_F32 = 4,     /* float32 3x3 / 1x1 on the matrix cores */
  MAFAT_KERNEL_FIRST_LAYER = 5,  /* a 3-channel 3x3 first layer run alone */
  MAFAT_KERNEL_GENERIC = 6,      /* vector-ALU convolution: any supported layer and size */
  MAFAT_KERNEL_POOL = 7          /* a max-pool that does not follow a convolution */
} mafat_kernel;

/* The per-tile layer execution of a group (sections 3 and 4) as launched on
 * this GPU, for tests and tools: *kernel = the mafat_kernel family that
 * runs stage `stage` of group g in mafat_run_group / mafat_run_network for
 * this batch and dtype (both stages of a fused pair report the pair's
 * kernel).  Errors: EINVAL (NULL, index out of range, batch < 1),
 * EUNSUPPORTED (dtype). */
int mafat_plan_stage_kernel(const mafat_plan* plan, int32_t group, int32_t stage, int32_t batch,
                            int32_t dtype, int32_t* kernel);

/* Working memory of a group's tiles (section 4: a tile's intermediate
 * results exist only while the tile is processed; section 4.1 sizes them).
 * Bytes of device workspace mafat_run_group / mafat_run_network need for
 * `batch` frames in `dtype` (0 if none).  It holds the tiles' intermediate
 * activations between stages; the largest group decides.  Errors: EINVAL. */
int mafat_workspace_size(const mafat_plan* plan, int32_t batch, int32_t dtype,
                         size_t* bytes);

/* Fused tile execution of one layer group (sections 3 and 4: every tile of
 * the group's grid is pushed through all of the group's layers from its own
 * input region, and the tile outputs are merged into the group output).
 * Runs group g on `batch` frames.
 *   x          device, the group input: batch x H x W x C of the group's first
 *              layer input (the network input for g = 0, else the previous
 *              group's output)
 *   y          device, the group output: batch x H x W x C of its last layer;
 *              every element is written exactly once
 *   w, scale, bias  host arrays indexed by global layer number (n_layers
 *              entries); entries of max-pool layers are ignored
 *   workspace  device, 256-byte aligned, at least mafat_workspace_size bytes
 *   stream     hipStream_t (NULL: the default stream)
 * x and y must not overlap.  Errors: EINVAL, EUNSUPPORTED (dtype, or a
 * frame's group input, output or workspace share holding 2^31 elements or
 * more), EWORKSPACE, EHIP.  Frames of 2^31 bytes or more (but fewer
 * elements) run on the generic kernels. */
int mafat_run_group(const mafat_plan* plan, int32_t group, int32_t batch, int32_t dtype,
                    const void* x, void* y, const void* const* w,
                    const float* const* scale, const float* const* bias,
                    void* workspace, size_t ws_bytes, void* stream);

/* mafat_run_group (sections 3 and 4) with per-stage timestamps, for
 * measurement.  events: 2 * n_stages hipEvent_t (host array): events[2s] is
 * recorded when the first kernel of stage s starts and events[2s+1] when
 * its last kernel ends (timestamps of the kernel dispatches themselves, so
 * timing adds nothing between kernels); entries may be NULL.  For a fused
 * pair (mafat_plan_stage_fused) the first stage's events enclose the pair's
 * kernel; the second stage's two events are recorded after it and time
 * nothing.  Errors: those of mafat_run_group, and EINVAL for a NULL events
 * array. */
int mafat_run_group_timed(const mafat_plan* plan, int32_t group, int32_t batch, int32_t dtype,
                          const void* x, void* y, const void* const* w,
                          const float* const* scale, const float* const* bias,
                          void* workspace, size_t ws_bytes, void* stream,
                          void* const* events);

/* One stage of a group's fused tile execution (sections 3 and 4), for
 * per-stage measurement.
 * Runs only stage `stage` of group g (see mafat_plan_stages): the stage
 * reads the group input x (first stage) or the workspace, and writes the
 * group output y (last stage) or the workspace.  Calling it for stages 0 ..
 * n_stages-1 in order on one stream with the same workspace computes what
 * mafat_run_group computes; one stage alone can be launched repeatedly
 * (e.g. to time its kernel).  It always runs one stage alone (a fused
 * pair's stages as two kernels, see mafat_plan_stage_fused).  Same
 * arguments, conventions and errors as mafat_run_group, plus EINVAL for a
 * stage index out of range and EUNSUPPORTED for a group that runs in
 * several tile batches (mafat_plan_set_tile_batch) and for a plan with
 * MAFAT_PLAN_ROW_REUSE. */
int mafat_run_stage(const mafat_plan* plan, int32_t group, int32_t stage, int32_t batch,
                    int32_t dtype, const void* x, void* y, const void* const* w,
                    const float* const* scale, const float* const* bias, void* workspace,
                    size_t ws_bytes, void* stream);

/* The whole network under a MAFAT configuration (section 4: group 1's tile
 * outputs are merged into the cut tensor, which group 2 re-tiles with its
 * own grid).
 * Runs every group in order on one stream: group 0 reads x, group g writes
 * cut_bufs[g] (n_groups-1 caller-owned tensors, each the shape of its group's
 * output) and group g+1 reads it; the last group writes y.  Same argument
 * conventions and errors as mafat_run_group. */
int mafat_run_network(const mafat_plan* plan, int32_t batch, int32_t dtype,
                      const void* x, void* y, void* const* cut_bufs,
                      const void* const* w, const float* const* scale,
                      const float* const* bias, void* workspace, size_t ws_bytes,
                      void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * mafat_run_network without a workspace argument.  The workspace is a
 * static device array of MAFAT_STATIC_WORKSPACE_MIB MiB that every GPU the
 * library runs on holds until the process ends; the call allocates nothing
 * (no hipMalloc, no allocating library routine).  The caller still owns x,
 * y, the cut tensors and the parameters (same conventions as
 * mafat_run_network).  The stream (NULL: the default stream) must belong to
 * the current device.  All calls on one GPU share its array: calls that
 * overlap in time on one GPU (several streams or threads) race.  Errors:
 * those of mafat_run_network, EWORKSPACE when mafat_workspace_size(plan,
 * batch, dtype) exceeds the array, EINVAL for a stream of another device,
 * EHIP if the array's device address cannot be obtained. */
#define MAFAT_STATIC_WORKSPACE_MIB 32
int mafat_run_network_static(const mafat_plan* plan, int32_t batch, int32_t dtype,
                             const void* x, void* y, void* const* cut_bufs,
                             const void* const* w, const float* const* scale,
                             const float* const* bias, void* stream);

/* Memory prediction for a plan (section 4.1).
 *   model MAFAT_MEM_PAPER: the paper's predictor (Algorithm 1) on this plan's
 *     region tables ("Grid"): the largest, over every tile of every group
 *     and every layer of the group, of
 *       w_out*h_out*c_in*f*f/s (im2col scratch) + w_out*h_out*c_out (output)
 *       + 2 * w_in*h_in*c_in (input),
 *     with the tile's input/output extents at that layer, halo included, in
 *     elements (integer division by s), times the dtype's element size (4 or
 *     2 bytes); batch is ignored.  The paper adds a platform constant (31 MB
 *     on its board); the caller adds its own (see mafat_get_config).
 *   model MAFAT_MEM_DEVICE: the device memory a run of this library needs,
 *     all of it caller-owned: input, output and cut tensors (batch frames),
 *     parameters (weights in dtype, float32 scale and bias) and the
 *     workspace (mafat_workspace_size).  By default every tile of a stage
 *     runs at once on the GPU, so the workspace holds every tile's
 *     intermediates; with a tile batch (mafat_plan_set_tile_batch) it holds
 *     one batch's, with row reuse the stage outputs' row bands.
 *   model MAFAT_MEM_DEVICE_SEQ: the device memory of the same plan run one
 *     tile at a time (tile batch 1, the paper's execution order), whatever
 *     the plan's tile batch; for groups with the stage partition or row
 *     reuse, their workspace as MAFAT_MEM_DEVICE.  With mafat_get_config this is the paper's search
 *     under a device-memory limit.
 * *bytes receives the prediction.  Errors: EINVAL (null plan or pointer,
 * batch < 1, unknown model), EUNSUPPORTED (dtype). */
int mafat_predict_mem(const mafat_plan* plan, int32_t model, int32_t batch, int32_t dtype,
                      int64_t* bytes);

/* Configuration search (section 4.2, Algorithm 2): for each cut in cuts[]
 * (in order; a cut <= 0 or >= n_layers means one group of all layers) and
 * each first-group grid t in grids[] (in order; t x t tiles), the plan
 * {cut, t x t, second_grid x second_grid} is predicted with
 * mafat_predict_mem(model, batch, dtype); the first whose prediction plus
 * bias_bytes is below limit_bytes is returned (*out_fits = 1).  If none
 * fits, the last one tried is returned (*out_fits = 0) -- with the paper's
 * lists (cuts {16, 12, 8}, grids {1..5}, second grid 2) that is its
 * fallback 5x5/8/2x2.  Outputs: *out_cut (n_layers for one group),
 * *out_grid1, *out_grid2 (0 for one group), *out_pred (prediction + bias;
 * may be NULL), *out_fits (may be NULL).  Errors: EINVAL (null pointer,
 * empty list, second_grid < 1) and the errors of mafat_plan_create for a
 * candidate that cannot be planned. */
int mafat_get_config(const mafat_layer* layers, int32_t n_layers, int32_t in_h, int32_t in_w,
                     int32_t in_c, int32_t model, int32_t batch, int32_t dtype, int64_t bias_bytes,
                     int64_t limit_bytes, const int32_t* cuts, int32_t n_cuts, const int32_t* grids,
                     int32_t n_grids, int32_t second_grid, int32_t* out_cut, int32_t* out_grid1,
                     int32_t* out_grid2, int64_t* out_pred, int32_t* out_fits);

/* mafat_get_config with variable tiling (section 6): the same search, with
 * every candidate's groups split at their mafat_balanced_bounds boundaries
 * instead of evenly (square grids, rows and columns balanced alike).  The
 * chosen configuration is planned with mafat_balanced_bounds and
 * mafat_plan_create_bounds.  Same arguments, outputs and errors as
 * mafat_get_config, plus those of mafat_balanced_bounds and ENOMEM. */
int mafat_get_config_balanced(const mafat_layer* layers, int32_t n_layers, int32_t in_h,
                              int32_t in_w, int32_t in_c, int32_t model, int32_t batch,
                              int32_t dtype, int64_t bias_bytes, int64_t limit_bytes,
                              const int32_t* cuts, int32_t n_cuts, const int32_t* grids,
                              int32_t n_grids, int32_t second_grid, int32_t* out_cut,
                              int32_t* out_grid1, int32_t* out_grid2, int64_t* out_pred,
                              int32_t* out_fits);

/* mafat_get_config with every candidate planned with plan_flags (those of
 * mafat_plan_create_flags: MAFAT_PLAN_ROW_REUSE, MAFAT_PLAN_STAGE_PARTITION,
 * MAFAT_PLAN_PACKED_WEIGHTS) and, if balanced is nonzero, with its groups'
 * balanced tile boundaries as mafat_get_config_balanced.  With
 * MAFAT_PLAN_ROW_REUSE and a device model this is the search under a
 * device-memory limit for the data-reuse execution of section 3 (tile rows
 * in order, no halo recompute), whose memory is its row bands.  Same
 * arguments, outputs and errors as mafat_get_config_balanced, plus those of
 * mafat_plan_create_flags for the flags. */
int mafat_get_config_flags(const mafat_layer* layers, int32_t n_layers, int32_t in_h, int32_t in_w,
                           int32_t in_c, int32_t model, int32_t batch, int32_t dtype, int64_t bias_bytes,
                           int64_t limit_bytes, const int32_t* cuts, int32_t n_cuts, const int32_t* grids,
                           int32_t n_grids, int32_t second_grid, int32_t plan_flags, int32_t balanced,
                           int32_t* out_cut, int32_t* out_grid1, int32_t* out_grid2, int64_t* out_pred,
                           int32_t* out_fits);

/* Error reporting of this library (no counterpart in the paper).
 * Static text of a status code. */
const char* mafat_status_string(int status);

/* Error reporting of this library (no counterpart in the paper).
 * Thread-local detail of the last failing call on this thread ("" if none). */
const char* mafat_last_error(void);

#ifdef __cplusplus
}
#endif
#endif
