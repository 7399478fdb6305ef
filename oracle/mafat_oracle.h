/*
 * mafat_oracle.h -- CPU reference ("oracle") for fused tile partitioning (FTP)
 * of a stack of convolution / max-pool layers, as used by MAFAT
 * (Farley & Gerstlauer, "MAFAT: Memory-Aware Fusing and Tiling of Neural
 * Networks for Accelerated Edge Inference", arXiv 2107.06960).
 *
 * TEST INFRASTRUCTURE ONLY.  This library exists to check the GPU library
 * against; nothing in the product path may link, load or call it.  It shares
 * no code, header or table with the GPU library.
 *
 * Everything here is plain, slow and written to be checked by eye:
 *   - tensors are float64 ("double"), NHWC, frame-major;
 *   - convolution weights are [c_out][f][f][c_in];
 *   - one fixed summation order per output element (ky, kx, ci), in double.
 *
 * Rectangles are half-open, in the coordinates of the tensor they index:
 *   rect = {y0, y1, x0, x1}  covers rows [y0, y1) and columns [x0, x1).
 *
 * Return values: 0 on success, negative on error (see ORC_E*).
 */
#ifndef MAFAT_ORACLE_H
#define MAFAT_ORACLE_H

#ifdef __cplusplus
extern "C" {
#endif

enum { ORC_CONV = 0, ORC_MAXPOOL = 1 };
enum { ORC_ACT_LINEAR = 0, ORC_ACT_LEAKY01 = 1 };
enum {
  ORC_OK = 0,
  ORC_EINVAL = -1,     /* bad argument or layer description          */
  ORC_EREGION = -2,    /* a tile read outside the region it was given */
  ORC_ENOMEM = -3,
  ORC_ENOTRECT = -4    /* brute-force receptive field is not a rectangle */
};

/* One layer.  c_out is ignored for max-pool (channels pass through). */
typedef struct {
  int op, c_out, f, s, p, act;
} orc_layer;

/* Shape inference (paper section 4.1: each layer has width, height, filter
 * size and stride; padding and channel counts are added here).
 * dims[6*l + 0..5] = in_h, in_w, in_c, out_h, out_w, out_c of layer l. */
int orc_shapes(const orc_layer* layers, int n, int h, int w, int c, int* dims);

/* Untiled, layer-by-layer forward of layers [l0, l1] for `batch` frames.
 * x is the input of layer l0, y receives the output of layer l1.
 * w/scale/bias are indexed by global layer number (NULL entries for pools).
 * round_bf16 != 0 rounds every layer output to bfloat16 (round to nearest
 * even), emulating a bf16-activation execution. */
int orc_forward_layers(const orc_layer* layers, int n, int h, int w, int c,
                       int l0, int l1, int batch, const double* x,
                       const double* const* wt, const double* const* scale,
                       const double* const* bias, int round_bf16, double* y);

/* Number of ints orc_regions / orc_regions_bruteforce write:
 * sum over groups of tiles(g) * layers(g) * 8. */
int orc_regions_size(int n, const int* group_start, int n_groups,
                     const int* grid_rows, const int* grid_cols);

/* Per-group, per-tile, per-layer regions by interval back-projection
 * (the "Grid"/traversal function of section 4.1).  Layout, concatenated over
 * groups g: [tile t (row-major)][layer l - g0][in y0,y1,x0,x1, out y0,y1,x0,x1].
 * Group g covers layers [group_start[g], group_start[g+1]) (last: to n). */
int orc_regions(const orc_layer* layers, int n, int h, int w, int c,
                const int* group_start, int n_groups, const int* grid_rows,
                const int* grid_cols, int* out);

/* orc_regions with each group's tile boundaries given (variable tiling,
 * proposed in section 6): row_bounds holds, concatenated over groups,
 * grid_rows[g] + 1 increasing row boundaries of group g's output (0 first,
 * the output height last; tile row i covers [b[i], b[i+1])), col_bounds
 * the same for columns.  Either may be NULL for even splits.  ORC_EINVAL
 * for boundaries that are not strictly increasing from 0 to the extent. */
int orc_regions_bounds(const orc_layer* layers, int n, int h, int w, int c,
                       const int* group_start, int n_groups, const int* grid_rows,
                       const int* grid_cols, const int* row_bounds, const int* col_bounds,
                       int* out);

/* The same table, built by enumerating every contributing input element of
 * every output element of each tile (receptive fields), layer by layer.
 * Returns ORC_ENOTRECT if a receptive field is not a full rectangle. */
int orc_regions_bruteforce(const orc_layer* layers, int n, int h, int w, int c,
                           const int* group_start, int n_groups,
                           const int* grid_rows, const int* grid_cols, int* out);

/* orc_regions_bruteforce with given tile boundaries (as orc_regions_bounds). */
int orc_regions_bruteforce_bounds(const orc_layer* layers, int n, int h, int w, int c,
                                  const int* group_start, int n_groups,
                                  const int* grid_rows, const int* grid_cols,
                                  const int* row_bounds, const int* col_bounds, int* out);

/* FTP execution (sections 3-4): every group is split into its own output tile
 * grid, every tile is pushed through all layers of the group using only its
 * own input region, and tile outputs are stitched into the group output,
 * which is the next group's input.  y receives the network output;
 * cut_out[g] (if cut_out and cut_out[g] are non-NULL) receives the output of
 * group g < n_groups-1.  Returns ORC_EREGION if a tile needed an element
 * outside its region. */
int orc_forward_tiled(const orc_layer* layers, int n, int h, int w, int c,
                      int batch, const int* group_start, int n_groups,
                      const int* grid_rows, const int* grid_cols,
                      const double* x, const double* const* wt,
                      const double* const* scale, const double* const* bias,
                      int round_bf16, double* y, double* const* cut_out);

/* orc_forward_tiled with given tile boundaries (as orc_regions_bounds). */
int orc_forward_tiled_bounds(const orc_layer* layers, int n, int h, int w, int c,
                             int batch, const int* group_start, int n_groups,
                             const int* grid_rows, const int* grid_cols,
                             const int* row_bounds, const int* col_bounds,
                             const double* x, const double* const* wt,
                             const double* const* scale, const double* const* bias,
                             int round_bf16, double* y, double* const* cut_out);

/* Row reuse, the data reuse between tiles of section 3 (a tile takes the
 * overlap that tiles run before it already computed instead of computing it
 * again) with every group's tiles run one grid row after another, each row
 * through all layers of the group.  The group output is cut into the tile
 * rows (row_bounds as in orc_regions_bounds, NULL: even split); every earlier
 * layer output of the group is cut where the rows that the next layer's parts
 * read end, so a tile row computes the rows that its next layer reads
 * beyond those of the rows before it, and no row twice.  A tile row keeps
 * each layer's output in a band of full-width rows: its own rows and the
 * rows above them that its next layer reads, taken over from the previous
 * row's band; a read outside the band is ORC_EREGION.  Columns are not cut
 * (the tiles of a row compute the same values together).  y and cut_out as
 * orc_forward_tiled.  band_rows (n values, may be NULL) receives, per layer,
 * the most rows any of its bands holds (0 for a group's last layer).  With x
 * and y both NULL only band_rows is computed. */
int orc_forward_row_reuse(const orc_layer* layers, int n, int h, int w, int c,
                          int batch, const int* group_start, int n_groups,
                          const int* grid_rows, const int* row_bounds,
                          const double* x, const double* const* wt,
                          const double* const* scale, const double* const* bias,
                          int round_bf16, double* y, double* const* cut_out, int* band_rows);

/* Balanced boundaries of `parts` tiles along one axis (0: rows, 1: columns)
 * of the output of layer group [g0, g1] (variable tiling, section 6: end
 * tiles sized differently from inner ones so that task sizes vary less).
 * A tile's task along the axis is the extent of the input region of layer
 * g0 that its output interval reads.  By brute force over every choice of
 * boundaries: the smallest largest task extent, then the smallest sum of
 * squared task extents, then the first boundary list in lexicographic
 * order.  bounds receives parts + 1 values (0 ... extent).  ORC_EINVAL for
 * parts outside 1 .. extent or more than 2e8 choices. */
int orc_balanced_bounds(const orc_layer* layers, int n, int h, int w, int c, int g0, int g1,
                        int axis, int parts, int* bounds);

/* Output of the whole stack [0, n) on one output rectangle of one frame,
 * computed from that rectangle's receptive field only (a one-tile FTP).
 * y holds (oy1-oy0) x (ox1-ox0) x c_out values, NHWC. */
int orc_forward_rect(const orc_layer* layers, int n, int h, int w, int c,
                     const double* x, const double* const* wt,
                     const double* const* scale, const double* const* bias,
                     int round_bf16, int oy0, int oy1, int ox0, int ox1,
                     double* y);

/* bfloat16 round-to-nearest-even of a value (via float32), as a double. */
double orc_round_bf16(double v);

/* Number of threads the layer loops use (default 1): each layer's output
 * rows are split into contiguous bands, every element still computed alone
 * in its fixed summation order, so results do not depend on it.  Errors:
 * ORC_EINVAL for n < 1 (n is capped at 256). */
int orc_set_threads(int n);

#ifdef __cplusplus
}
#endif
#endif
