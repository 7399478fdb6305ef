/*
 * mafat_oracle.c -- plain CPU reference for MAFAT fused tile partitioning.
 *
 * TEST INFRASTRUCTURE ONLY: used by the tests, by the smoke check and by the
 * benchmark's CPU-baseline leg.  The product (the HIP library) never links,
 * loads or calls this file, and this file shares nothing with it.
 *
 * What it follows (arXiv 2107.06960):
 *   - section 3 / section 4: FTP splits a layer stack's output into an even
 *     2-D grid; each tile's sub-convolutions are fused across all layers of
 *     the group and run as one independent unit;
 *   - section 4: MAFAT allows one group or two groups separated by a cut;
 *     the first group's tile outputs are merged into one tensor and re-tiled
 *     by the second group with its own grid;
 *   - section 4.1: the per-layer tile dimensions including the overlap
 *     ("Grid", the traversal function) -- here computed as the exact
 *     receptive-field interval of a tile, clipped to the tensor;
 *   - the per-layer arithmetic (convolution, folded batch-norm scale/bias,
 *     leaky ReLU with slope 0.1, 2x2/2 max-pool) is the plain definition of
 *     the layers of YOLOv2's first 16 layers, the network of section 2/5.
 *
 * Readings where the paper is silent (each also listed in the design notes):
 *   - partition of an extent E into N parts: part i is [floor(iE/N),
 *     floor((i+1)E/N)), unless the caller gives the boundaries (variable
 *     tiling, which section 6 proposes as future work: end tiles of another
 *     size than the inner ones, so that the tiles' tasks vary less);
 *   - balanced boundaries (orc_balanced_bounds): along one axis a tile's
 *     task is the extent of its input region at the group's first layer;
 *     the boundaries minimise the largest task extent, then the sum of the
 *     squared task extents, then come first in lexicographic order;
 *   - padding: convolutions pad only outside the image (never at a tile
 *     border); a tile computes its halo itself (no data reuse);
 *   - every convolution is followed by scale/bias and its activation; a
 *     max-pool takes the maximum of the in-image elements of its window.
 *
 * Arithmetic: float64 everywhere.  The summation order of a convolution
 * output element is fixed (ky, kx, ci ascending), so the tiled and the
 * untiled forward give bit-identical results when the regions are right.
 */
#include "mafat_oracle.h"

#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------ */
/* small helpers                                                        */
/* ------------------------------------------------------------------ */

double orc_round_bf16(double v) {
  float f = (float)v;
  uint32_t u;
  memcpy(&u, &f, 4);
  if ((u & 0x7f800000u) == 0x7f800000u) { /* inf / nan: keep (quiet nan) */
    if (u & 0x007fffffu) u |= 0x00400000u;
    u &= 0xffff0000u;
  } else {
    uint32_t lsb = (u >> 16) & 1u;
    u += 0x7fffu + lsb;
    u &= 0xffff0000u;
  }
  memcpy(&f, &u, 4);
  return (double)f;
}

static int imin(int a, int b) { return a < b ? a : b; }
static int imax(int a, int b) { return a > b ? a : b; }

static int layer_ok(const orc_layer* L) {
  if (L->f < 1 || L->s < 1 || L->p < 0 || L->p >= L->f) return 0;
  if (L->op == ORC_CONV) return L->c_out >= 1 && (L->act == ORC_ACT_LINEAR || L->act == ORC_ACT_LEAKY01);
  return L->op == ORC_MAXPOOL;
}

int orc_shapes(const orc_layer* layers, int n, int h, int w, int c, int* dims) {
  if (!layers || n < 1 || h < 1 || w < 1 || c < 1 || !dims) return ORC_EINVAL;
  for (int l = 0; l < n; ++l) {
    const orc_layer* L = &layers[l];
    if (!layer_ok(L)) return ORC_EINVAL;
    int oh_num = h + 2 * L->p - L->f, ow_num = w + 2 * L->p - L->f;
    if (oh_num < 0 || ow_num < 0) return ORC_EINVAL;
    int oh = oh_num / L->s + 1, ow = ow_num / L->s + 1;
    int oc = (L->op == ORC_CONV) ? L->c_out : c;
    dims[6 * l + 0] = h; dims[6 * l + 1] = w; dims[6 * l + 2] = c;
    dims[6 * l + 3] = oh; dims[6 * l + 4] = ow; dims[6 * l + 5] = oc;
    h = oh; w = ow; c = oc;
  }
  return ORC_OK;
}

/* A read-only window onto a tensor: element (y, x, ch) in global coordinates
 * of the tensor (img_h x img_w x c) is at d[(y-y0)*rs + (x-x0)*c + ch] and is
 * only readable if it lies inside [y0, y0+h) x [x0, x0+w). */
typedef struct {
  const double* d;
  int y0, x0, h, w, c, rs;
  int img_h, img_w;
  int* err;
} view_t;

static double view_at(const view_t* v, int y, int x, int ch) {
  if (y < v->y0 || y >= v->y0 + v->h || x < v->x0 || x >= v->x0 + v->w) {
    *v->err = ORC_EREGION;
    return 0.0;
  }
  return v->d[(size_t)(y - v->y0) * v->rs + (size_t)(x - v->x0) * v->c + ch];
}

/* One output element of a convolution layer, followed by scale, bias and
 * activation:  v = sum_{ky,kx,ci} in[y*S+ky-P][x*S+kx-P][ci] * w[co][ky][kx][ci]
 * over in-image terms only (zero padding), then v = v*scale + bias, then
 * leaky: v > 0 ? v : 0.1 v. */
static double conv_pixel(const view_t* in, const orc_layer* L, const double* wt,
                         double scale, double bias, int y, int x, int co,
                         int round_bf16) {
  const int F = L->f, C = in->c;
  double acc = 0.0;
  for (int ky = 0; ky < F; ++ky) {
    int iy = y * L->s + ky - L->p;
    if (iy < 0 || iy >= in->img_h) continue;
    for (int kx = 0; kx < F; ++kx) {
      int ix = x * L->s + kx - L->p;
      if (ix < 0 || ix >= in->img_w) continue;
      const double* wr = wt + (((size_t)co * F + ky) * F + kx) * C;
      for (int ci = 0; ci < C; ++ci) acc += view_at(in, iy, ix, ci) * wr[ci];
    }
  }
  double v = acc * scale + bias;
  if (L->act == ORC_ACT_LEAKY01 && !(v > 0.0)) v = 0.1 * v;
  return round_bf16 ? orc_round_bf16(v) : v;
}

/* One output element of a max-pool layer: the maximum over the in-image
 * elements of its window, visited in (ky, kx) order. */
static double pool_pixel(const view_t* in, const orc_layer* L, int y, int x,
                         int ch, int round_bf16) {
  double m = -INFINITY;
  int any = 0;
  for (int ky = 0; ky < L->f; ++ky) {
    int iy = y * L->s + ky - L->p;
    if (iy < 0 || iy >= in->img_h) continue;
    for (int kx = 0; kx < L->f; ++kx) {
      int ix = x * L->s + kx - L->p;
      if (ix < 0 || ix >= in->img_w) continue;
      double v = view_at(in, iy, ix, ch);
      if (!any || v > m) m = v;
      any = 1;
    }
  }
  if (!any) *in->err = ORC_EINVAL;
  return round_bf16 ? orc_round_bf16(m) : m;
}

/* Rows [ya, yb) of layer l's output rectangle [oy0,oy1) x [ox0,ox1), into
 * the dense buffer out (rect-local NHWC). */
static void layer_rows(const view_t* in, const orc_layer* L, int out_c,
                       const double* wt, const double* scale, const double* bias,
                       int round_bf16, int oy0, int ya, int yb, int ox0, int ox1,
                       double* out) {
  const int ow = ox1 - ox0;
  for (int y = ya; y < yb; ++y)
    for (int x = ox0; x < ox1; ++x) {
      double* o = out + ((size_t)(y - oy0) * ow + (x - ox0)) * out_c;
      for (int ch = 0; ch < out_c; ++ch)
        o[ch] = (L->op == ORC_CONV)
                    ? conv_pixel(in, L, wt, scale[ch], bias[ch], y, x, ch, round_bf16)
                    : pool_pixel(in, L, y, x, ch, round_bf16);
    }
}

/* Worker threads for layer_rect (orc_set_threads): the output rows of a
 * layer are split into contiguous bands, one per thread.  Every output
 * element is still computed by conv_pixel / pool_pixel alone, in the same
 * summation order, so the result does not depend on the thread count. */
static int g_threads = 1;

int orc_set_threads(int n) {
  if (n < 1) return ORC_EINVAL;
  g_threads = n > 256 ? 256 : n;
  return ORC_OK;
}

typedef struct {
  view_t in;  /* private copy: its err points at this band's flag */
  const orc_layer* L;
  int out_c;
  const double *wt, *scale, *bias;
  int round_bf16, oy0, ya, yb, ox0, ox1;
  double* out;
  int err;
} band_t;

static void* band_run(void* arg) {
  band_t* b = (band_t*)arg;
  layer_rows(&b->in, b->L, b->out_c, b->wt, b->scale, b->bias, b->round_bf16, b->oy0, b->ya, b->yb,
             b->ox0, b->ox1, b->out);
  return NULL;
}

/* Computes layer l on the output rectangle [oy0,oy1) x [ox0,ox1) into the
 * dense buffer out (rect-local NHWC). */
static void layer_rect(const view_t* in, const orc_layer* L, int out_c,
                       const double* wt, const double* scale, const double* bias,
                       int round_bf16, int oy0, int oy1, int ox0, int ox1,
                       double* out) {
  int nt = g_threads < oy1 - oy0 ? g_threads : oy1 - oy0;
  if (nt <= 1) {
    layer_rows(in, L, out_c, wt, scale, bias, round_bf16, oy0, oy0, oy1, ox0, ox1, out);
    return;
  }
  band_t bands[256];
  pthread_t tid[256];
  int started[256];
  for (int k = 0; k < nt; ++k) {
    band_t* b = &bands[k];
    b->in = *in;
    b->err = 0;
    b->in.err = &b->err;
    b->L = L; b->out_c = out_c; b->wt = wt; b->scale = scale; b->bias = bias;
    b->round_bf16 = round_bf16; b->oy0 = oy0; b->ox0 = ox0; b->ox1 = ox1; b->out = out;
    b->ya = oy0 + (int)((int64_t)(oy1 - oy0) * k / nt);
    b->yb = oy0 + (int)((int64_t)(oy1 - oy0) * (k + 1) / nt);
    started[k] = pthread_create(&tid[k], NULL, band_run, b) == 0;
    if (!started[k]) band_run(b); /* no thread: run the band here */
  }
  for (int k = 0; k < nt; ++k) {
    if (started[k]) pthread_join(tid[k], NULL);
    if (bands[k].err) *in->err = bands[k].err;
  }
}

/* ------------------------------------------------------------------ */
/* untiled forward                                                      */
/* ------------------------------------------------------------------ */

int orc_forward_layers(const orc_layer* layers, int n, int h, int w, int c,
                       int l0, int l1, int batch, const double* x,
                       const double* const* wt, const double* const* scale,
                       const double* const* bias, int round_bf16, double* y) {
  if (l0 < 0 || l1 < l0 || l1 >= n || batch < 1 || !x || !y) return ORC_EINVAL;
  int* dims = (int*)malloc(sizeof(int) * 6 * (size_t)n);
  if (!dims) return ORC_ENOMEM;
  int rc = orc_shapes(layers, n, h, w, c, dims);
  if (rc) { free(dims); return rc; }
  for (int l = l0; l <= l1; ++l)
    if (layers[l].op == ORC_CONV && (!wt || !wt[l] || !scale || !scale[l] || !bias || !bias[l])) {
      free(dims); return ORC_EINVAL;
    }
  int err = 0;
  for (int b = 0; b < batch; ++b) {
    const int* d0 = dims + 6 * l0;
    const double* cur = x + (size_t)b * d0[0] * d0[1] * d0[2];
    double* owned = NULL;
    for (int l = l0; l <= l1; ++l) {
      const int* d = dims + 6 * l;
      size_t out_elems = (size_t)d[3] * d[4] * d[5];
      double* nxt = (l == l1) ? y + (size_t)b * out_elems : (double*)malloc(sizeof(double) * out_elems);
      if (!nxt) { free(owned); free(dims); return ORC_ENOMEM; }
      view_t v = {cur, 0, 0, d[0], d[1], d[2], d[1] * d[2], d[0], d[1], &err};
      layer_rect(&v, &layers[l], d[5], wt ? wt[l] : NULL, scale ? scale[l] : NULL,
                 bias ? bias[l] : NULL, round_bf16, 0, d[3], 0, d[4], nxt);
      free(owned);
      owned = (l == l1) ? NULL : nxt;
      cur = nxt;
    }
  }
  free(dims);
  return err;
}

/* ------------------------------------------------------------------ */
/* regions                                                              */
/* ------------------------------------------------------------------ */

static int groups_ok(int n, const int* gs, int ng, const int* rows, const int* cols) {
  if (!gs || !rows || !cols || ng < 1 || gs[0] != 0) return 0;
  for (int g = 0; g < ng; ++g) {
    int end = (g + 1 < ng) ? gs[g + 1] : n;
    if (gs[g] >= end || end > n || rows[g] < 1 || cols[g] < 1) return 0;
  }
  return 1;
}

int orc_regions_size(int n, const int* group_start, int n_groups,
                     const int* grid_rows, const int* grid_cols) {
  if (!groups_ok(n, group_start, n_groups, grid_rows, grid_cols)) return ORC_EINVAL;
  int total = 0;
  for (int g = 0; g < n_groups; ++g) {
    int end = (g + 1 < n_groups) ? group_start[g + 1] : n;
    total += grid_rows[g] * grid_cols[g] * (end - group_start[g]) * 8;
  }
  return total;
}

/* Part i of N of the extent [0, E): [floor(iE/N), floor((i+1)E/N)). */
static void split(int E, int N, int i, int* a, int* b) {
  *a = (int)(((long long)i * E) / N);
  *b = (int)(((long long)(i + 1) * E) / N);
}

/* Part i of N of [0, E): [bounds[i], bounds[i+1]) when the caller gave
 * boundaries, else the even split. */
static void span(int E, int N, int i, const int* bounds, int* a, int* b) {
  if (bounds) { *a = bounds[i]; *b = bounds[i + 1]; }
  else split(E, N, i, a, b);
}

/* Boundaries of N parts of [0, E): 0 = b[0] < b[1] < ... < b[N] = E. */
static int bounds_ok(const int* b, int N, int E) {
  if (b[0] != 0 || b[N] != E) return 0;
  for (int i = 0; i < N; ++i)
    if (b[i + 1] <= b[i]) return 0;
  return 1;
}

/* Checks the per-group boundary lists (concatenated over groups, rows+1 /
 * cols+1 entries per group; NULL = even splits) against the group output
 * extents. */
static int all_bounds_ok(const int* dims, int n, const int* gs, int ng, const int* rows,
                         const int* cols, const int* rb, const int* cb) {
  for (int g = 0; g < ng; ++g) {
    int g1 = ((g + 1 < ng) ? gs[g + 1] : n) - 1;
    const int* dl = dims + 6 * g1;
    if (rb && !bounds_ok(rb, rows[g], dl[3])) return 0;
    if (cb && !bounds_ok(cb, cols[g], dl[4])) return 0;
    if (rb) rb += rows[g] + 1;
    if (cb) cb += cols[g] + 1;
  }
  return 1;
}

/* Input interval of a layer (filter F, stride S, pad P) that the output
 * interval [a, b) reads, clipped to the input extent [0, E). */
static void back_project(int a, int b, int F, int S, int P, int E, int* ia, int* ib) {
  *ia = imax(0, a * S - P);
  *ib = imin(E, (b - 1) * S - P + F);
}

int orc_regions(const orc_layer* layers, int n, int h, int w, int c,
                const int* group_start, int n_groups, const int* grid_rows,
                const int* grid_cols, int* out) {
  return orc_regions_bounds(layers, n, h, w, c, group_start, n_groups, grid_rows, grid_cols,
                            NULL, NULL, out);
}

int orc_regions_bounds(const orc_layer* layers, int n, int h, int w, int c,
                       const int* group_start, int n_groups, const int* grid_rows,
                       const int* grid_cols, const int* row_bounds, const int* col_bounds,
                       int* out) {
  if (!out || !groups_ok(n, group_start, n_groups, grid_rows, grid_cols)) return ORC_EINVAL;
  int* dims = (int*)malloc(sizeof(int) * 6 * (size_t)n);
  if (!dims) return ORC_ENOMEM;
  int rc = orc_shapes(layers, n, h, w, c, dims);
  if (rc) { free(dims); return rc; }
  if (!all_bounds_ok(dims, n, group_start, n_groups, grid_rows, grid_cols, row_bounds, col_bounds)) {
    free(dims);
    return ORC_EINVAL;
  }
  int* o = out;
  const int *rb = row_bounds, *cb = col_bounds;
  for (int g = 0; g < n_groups; ++g) {
    int g0 = group_start[g], g1 = ((g + 1 < n_groups) ? group_start[g + 1] : n) - 1;
    int R = grid_rows[g], Cc = grid_cols[g], nl = g1 - g0 + 1;
    const int* dl = dims + 6 * g1;
    if (R > dl[3] || Cc > dl[4]) { free(dims); return ORC_EINVAL; }
    for (int i = 0; i < R; ++i)
      for (int j = 0; j < Cc; ++j) {
        int oy0, oy1, ox0, ox1;
        span(dl[3], R, i, rb, &oy0, &oy1);
        span(dl[4], Cc, j, cb, &ox0, &ox1);
        for (int l = g1; l >= g0; --l) {
          const orc_layer* L = &layers[l];
          const int* d = dims + 6 * l;
          int iy0, iy1, ix0, ix1;
          back_project(oy0, oy1, L->f, L->s, L->p, d[0], &iy0, &iy1);
          back_project(ox0, ox1, L->f, L->s, L->p, d[1], &ix0, &ix1);
          int* r = o + (size_t)(l - g0) * 8;
          r[0] = iy0; r[1] = iy1; r[2] = ix0; r[3] = ix1;
          r[4] = oy0; r[5] = oy1; r[6] = ox0; r[7] = ox1;
          oy0 = iy0; oy1 = iy1; ox0 = ix0; ox1 = ix1;
        }
        o += nl * 8;
      }
    if (rb) rb += R + 1;
    if (cb) cb += Cc + 1;
  }
  free(dims);
  return ORC_OK;
}

/* Bounding box of a mask, and whether the mask is exactly that box. */
static int mask_rect(const unsigned char* m, int H, int W, int* r) {
  int y0 = H, y1 = -1, x0 = W, x1 = -1;
  for (int y = 0; y < H; ++y)
    for (int x = 0; x < W; ++x)
      if (m[(size_t)y * W + x]) {
        y0 = imin(y0, y); y1 = imax(y1, y); x0 = imin(x0, x); x1 = imax(x1, x);
      }
  if (y1 < 0) return 0;
  for (int y = y0; y <= y1; ++y)
    for (int x = x0; x <= x1; ++x)
      if (!m[(size_t)y * W + x]) return 0;
  r[0] = y0; r[1] = y1 + 1; r[2] = x0; r[3] = x1 + 1;
  return 1;
}

int orc_regions_bruteforce(const orc_layer* layers, int n, int h, int w, int c,
                           const int* group_start, int n_groups,
                           const int* grid_rows, const int* grid_cols, int* out) {
  return orc_regions_bruteforce_bounds(layers, n, h, w, c, group_start, n_groups, grid_rows,
                                       grid_cols, NULL, NULL, out);
}

int orc_regions_bruteforce_bounds(const orc_layer* layers, int n, int h, int w, int c,
                                  const int* group_start, int n_groups,
                                  const int* grid_rows, const int* grid_cols,
                                  const int* row_bounds, const int* col_bounds, int* out) {
  if (!out || !groups_ok(n, group_start, n_groups, grid_rows, grid_cols)) return ORC_EINVAL;
  int* dims = (int*)malloc(sizeof(int) * 6 * (size_t)n);
  if (!dims) return ORC_ENOMEM;
  int rc = orc_shapes(layers, n, h, w, c, dims);
  if (rc) { free(dims); return rc; }
  if (!all_bounds_ok(dims, n, group_start, n_groups, grid_rows, grid_cols, row_bounds, col_bounds)) {
    free(dims);
    return ORC_EINVAL;
  }
  int* o = out;
  const int *rb = row_bounds, *cb = col_bounds;
  for (int g = 0; g < n_groups && rc == 0; ++g) {
    int g0 = group_start[g], g1 = ((g + 1 < n_groups) ? group_start[g + 1] : n) - 1;
    int R = grid_rows[g], Cc = grid_cols[g], nl = g1 - g0 + 1;
    const int* dl = dims + 6 * g1;
    if (R > dl[3] || Cc > dl[4]) { rc = ORC_EINVAL; break; }
    for (int i = 0; i < R && rc == 0; ++i)
      for (int j = 0; j < Cc && rc == 0; ++j) {
        /* the tile's own output elements at the group's last layer */
        int oh = dl[3], ow = dl[4];
        unsigned char* cur = (unsigned char*)calloc((size_t)oh * ow, 1);
        int a, b, p, q;
        span(oh, R, i, rb, &a, &b);
        span(ow, Cc, j, cb, &p, &q);
        for (int y = a; y < b; ++y)
          for (int x = p; x < q; ++x) cur[(size_t)y * ow + x] = 1;
        for (int l = g1; l >= g0 && rc == 0; --l) {
          const orc_layer* L = &layers[l];
          const int* d = dims + 6 * l;
          unsigned char* prev = (unsigned char*)calloc((size_t)d[0] * d[1], 1);
          /* every input element that any marked output element reads */
          for (int y = 0; y < d[3]; ++y)
            for (int x = 0; x < d[4]; ++x) {
              if (!cur[(size_t)y * d[4] + x]) continue;
              for (int ky = 0; ky < L->f; ++ky)
                for (int kx = 0; kx < L->f; ++kx) {
                  int iy = y * L->s + ky - L->p, ix = x * L->s + kx - L->p;
                  if (iy >= 0 && iy < d[0] && ix >= 0 && ix < d[1]) prev[(size_t)iy * d[1] + ix] = 1;
                }
            }
          int* r = o + (size_t)(l - g0) * 8;
          if (!mask_rect(cur, d[3], d[4], r + 4) || !mask_rect(prev, d[0], d[1], r)) rc = ORC_ENOTRECT;
          free(cur);
          cur = prev;
        }
        free(cur);
        o += nl * 8;
      }
    if (rb) rb += R + 1;
    if (cb) cb += Cc + 1;
  }
  free(dims);
  return rc;
}

/* ------------------------------------------------------------------ */
/* tiled (FTP) forward                                                  */
/* ------------------------------------------------------------------ */

/* Pushes one tile of one frame through layers [g0, g1].  regs holds the
 * tile's per-layer {in rect, out rect}.  `src` is the group input tensor of
 * the frame (full, dense); only the tile's first-layer input rect of it may
 * be read.  The tile's output rect at g1 is written into dst (full tensor of
 * the group's last layer). */
static int tile_forward(const orc_layer* layers, const int* dims, int g0, int g1,
                        const int* regs, const double* src, double* dst,
                        const double* const* wt, const double* const* scale,
                        const double* const* bias, int round_bf16) {
  int err = 0;
  const int* d0 = dims + 6 * g0;
  const int* r0 = regs;
  view_t v = {src + ((size_t)r0[0] * d0[1] + r0[2]) * d0[2], r0[0], r0[2],
              r0[1] - r0[0], r0[3] - r0[2], d0[2], d0[1] * d0[2], d0[0], d0[1], &err};
  double* owned = NULL;
  for (int l = g0; l <= g1 && !err; ++l) {
    const int* d = dims + 6 * l;
    const int* r = regs + (size_t)(l - g0) * 8;
    int oh = r[5] - r[4], ow = r[7] - r[6];
    double* buf = (double*)malloc(sizeof(double) * (size_t)oh * ow * d[5]);
    if (!buf) { free(owned); return ORC_ENOMEM; }
    layer_rect(&v, &layers[l], d[5], wt ? wt[l] : NULL, scale ? scale[l] : NULL,
               bias ? bias[l] : NULL, round_bf16, r[4], r[5], r[6], r[7], buf);
    free(owned);
    owned = buf;
    view_t nv = {buf, r[4], r[6], oh, ow, d[5], ow * d[5], d[3], d[4], &err};
    v = nv;
  }
  if (!err) {
    const int* dl = dims + 6 * g1;
    const int* r = regs + (size_t)(g1 - g0) * 8;
    int ow = r[7] - r[6];
    for (int y = r[4]; y < r[5]; ++y)
      memcpy(dst + ((size_t)y * dl[4] + r[6]) * dl[5],
             owned + (size_t)(y - r[4]) * ow * dl[5], sizeof(double) * (size_t)ow * dl[5]);
  }
  free(owned);
  return err;
}

int orc_forward_tiled(const orc_layer* layers, int n, int h, int w, int c,
                      int batch, const int* group_start, int n_groups,
                      const int* grid_rows, const int* grid_cols,
                      const double* x, const double* const* wt,
                      const double* const* scale, const double* const* bias,
                      int round_bf16, double* y, double* const* cut_out) {
  return orc_forward_tiled_bounds(layers, n, h, w, c, batch, group_start, n_groups, grid_rows,
                                  grid_cols, NULL, NULL, x, wt, scale, bias, round_bf16, y, cut_out);
}

int orc_forward_tiled_bounds(const orc_layer* layers, int n, int h, int w, int c,
                             int batch, const int* group_start, int n_groups,
                             const int* grid_rows, const int* grid_cols,
                             const int* row_bounds, const int* col_bounds,
                             const double* x, const double* const* wt,
                             const double* const* scale, const double* const* bias,
                             int round_bf16, double* y, double* const* cut_out) {
  if (batch < 1 || !x || !y) return ORC_EINVAL;
  int nreg = orc_regions_size(n, group_start, n_groups, grid_rows, grid_cols);
  if (nreg < 0) return nreg;
  int* dims = (int*)malloc(sizeof(int) * 6 * (size_t)n);
  int* regs = (int*)malloc(sizeof(int) * (size_t)nreg);
  if (!dims || !regs) { free(dims); free(regs); return ORC_ENOMEM; }
  int rc = orc_shapes(layers, n, h, w, c, dims);
  if (!rc)
    rc = orc_regions_bounds(layers, n, h, w, c, group_start, n_groups, grid_rows, grid_cols,
                            row_bounds, col_bounds, regs);
  for (int l = 0; l < n && !rc; ++l)
    if (layers[l].op == ORC_CONV && (!wt || !wt[l] || !scale || !scale[l] || !bias || !bias[l])) rc = ORC_EINVAL;
  const double* gin = x;
  double* owned = NULL;
  const int* rg = regs;
  for (int g = 0; g < n_groups && !rc; ++g) {
    int g0 = group_start[g], g1 = ((g + 1 < n_groups) ? group_start[g + 1] : n) - 1;
    const int* din = dims + 6 * g0;
    const int* dout = dims + 6 * g1;
    size_t in_elems = (size_t)din[0] * din[1] * din[2];
    size_t out_elems = (size_t)dout[3] * dout[4] * dout[5];
    double* gout;
    if (g == n_groups - 1) gout = y;
    else if (cut_out && cut_out[g]) gout = cut_out[g];
    else gout = NULL;
    double* fresh = NULL;
    if (!gout) {
      fresh = (double*)malloc(sizeof(double) * out_elems * (size_t)batch);
      if (!fresh) { rc = ORC_ENOMEM; break; }
      gout = fresh;
    }
    int ntiles = grid_rows[g] * grid_cols[g], nl = g1 - g0 + 1;
    for (int b = 0; b < batch && !rc; ++b)
      for (int t = 0; t < ntiles && !rc; ++t)
        rc = tile_forward(layers, dims, g0, g1, rg + (size_t)t * nl * 8, gin + (size_t)b * in_elems,
                          gout + (size_t)b * out_elems, wt, scale, bias, round_bf16);
    rg += (size_t)ntiles * nl * 8;
    free(owned);
    owned = fresh;
    gin = gout;
  }
  free(owned);
  free(dims);
  free(regs);
  return rc;
}

/* Row reuse (the data reuse of section 3 -- a tile takes the overlap that
 * tiles run before it computed -- with a group's tiles run one grid row after
 * another).  Row boundaries of every layer output of group [g0, g1]:
 * rb[(l - g0) * (rows + 1) + i].  The group output's are the tile rows'; each
 * earlier layer's output is cut where the rows that the next layer's parts
 * read end, so that a tile row computes the rows its own next layer reads
 * beyond those of earlier tile rows. */
static void reuse_rows(const orc_layer* layers, const int* dims, int g0, int g1, int rows,
                       const int* bounds, int* rb) {
  int* last = rb + (size_t)(g1 - g0) * (rows + 1);
  for (int i = 0; i < rows; ++i) {
    int a, b;
    span(dims[6 * g1 + 3], rows, i, bounds, &a, &b);
    last[i] = a;
  }
  last[rows] = dims[6 * g1 + 3];
  for (int l = g1 - 1; l >= g0; --l) {
    const orc_layer* N = &layers[l + 1];
    const int* nxt = rb + (size_t)(l + 1 - g0) * (rows + 1);
    int* cur = rb + (size_t)(l - g0) * (rows + 1);
    cur[0] = 0;
    for (int i = 1; i <= rows; ++i) {
      int a, b;
      back_project(0, nxt[i], N->f, N->s, N->p, dims[6 * (l + 1)], &a, &b);
      cur[i] = nxt[i] > 0 ? b : 0;
    }
  }
}

/* First row of tile row i's band of layer l's output (l < g1): the first
 * row that the next layer's part of tile row i reads, or the row's own first
 * computed row if that is lower. */
static int reuse_band_lo(const orc_layer* layers, const int* dims, int g0, int l, int rows,
                         const int* rb, int i) {
  const orc_layer* N = &layers[l + 1];
  const int* nxt = rb + (size_t)(l + 1 - g0) * (rows + 1);
  const int* cur = rb + (size_t)(l - g0) * (rows + 1);
  int a, b;
  back_project(nxt[i], nxt[i] + 1, N->f, N->s, N->p, dims[6 * (l + 1)], &a, &b);
  return imin(a, cur[i]);
}

int orc_forward_row_reuse(const orc_layer* layers, int n, int h, int w, int c,
                          int batch, const int* group_start, int n_groups,
                          const int* grid_rows, const int* row_bounds,
                          const double* x, const double* const* wt,
                          const double* const* scale, const double* const* bias,
                          int round_bf16, double* y, double* const* cut_out, int* band_rows) {
  if (batch < 1 || (!x) != (!y) || n < 1 || n_groups < 1 || !group_start || !grid_rows) return ORC_EINVAL;
  int* dims = (int*)malloc(sizeof(int) * 6 * (size_t)n);
  if (!dims) return ORC_ENOMEM;
  int rc = orc_shapes(layers, n, h, w, c, dims);
  if (!rc && group_start[0] != 0) rc = ORC_EINVAL;
  for (int g = 0; g < n_groups && !rc; ++g) {
    int g1 = ((g + 1 < n_groups) ? group_start[g + 1] : n) - 1;
    if (g1 < group_start[g] || g1 >= n || grid_rows[g] < 1 || grid_rows[g] > dims[6 * g1 + 3]) rc = ORC_EINVAL;
  }
  if (!rc && row_bounds) {
    const int* rbp = row_bounds;
    for (int g = 0; g < n_groups && !rc; ++g) {
      int g1 = ((g + 1 < n_groups) ? group_start[g + 1] : n) - 1;
      if (!bounds_ok(rbp, grid_rows[g], dims[6 * g1 + 3])) rc = ORC_EINVAL;
      rbp += grid_rows[g] + 1;
    }
  }
  for (int l = 0; l < n && !rc && x; ++l)
    if (layers[l].op == ORC_CONV && (!wt || !wt[l] || !scale || !scale[l] || !bias || !bias[l])) rc = ORC_EINVAL;
  if (band_rows)
    for (int l = 0; l < n; ++l) band_rows[l] = 0;
  const double* gin = x;
  double* owned = NULL;
  const int* rbp = row_bounds;
  for (int g = 0; g < n_groups && !rc; ++g) {
    const int g0 = group_start[g], g1 = ((g + 1 < n_groups) ? group_start[g + 1] : n) - 1;
    const int rows = grid_rows[g], nl = g1 - g0 + 1;
    int* rb = (int*)malloc(sizeof(int) * (size_t)nl * (rows + 1));
    if (!rb) { rc = ORC_ENOMEM; break; }
    reuse_rows(layers, dims, g0, g1, rows, rbp, rb);
    if (rbp) rbp += rows + 1;
    for (int l = g0; l < g1 && band_rows; ++l)
      for (int i = 0; i < rows; ++i) {
        int hi = rb[(size_t)(l - g0) * (rows + 1) + i + 1];
        int lo = reuse_band_lo(layers, dims, g0, l, rows, rb, i);
        if (hi - lo > band_rows[l]) band_rows[l] = hi - lo;
      }
    if (!x) { free(rb); continue; }  /* geometry only */
    const int* din = dims + 6 * g0;
    const int* dout = dims + 6 * g1;
    size_t in_elems = (size_t)din[0] * din[1] * din[2];
    size_t out_elems = (size_t)dout[3] * dout[4] * dout[5];
    double* gout;
    double* fresh = NULL;
    if (g == n_groups - 1) gout = y;
    else if (cut_out && cut_out[g]) gout = cut_out[g];
    else gout = NULL;
    if (!gout) {
      fresh = (double*)malloc(sizeof(double) * out_elems * (size_t)batch);
      if (!fresh) { free(rb); rc = ORC_ENOMEM; break; }
      gout = fresh;
    }
    double** band = (double**)calloc((size_t)nl, sizeof(double*));
    int* blo = (int*)calloc((size_t)nl, sizeof(int));
    if (!band || !blo) rc = ORC_ENOMEM;
    for (int b = 0; b < batch && !rc; ++b) {
      for (int i = 0; i < rows && !rc; ++i) {
        for (int l = g0; l <= g1 && !rc; ++l) {
          const int* d = dims + 6 * l;
          const int* r = rb + (size_t)(l - g0) * (rows + 1);
          int err = 0;
          /* the input: the group input, or the band of layer l - 1 that
           * tile row i just completed */
          view_t in;
          if (l == g0) {
            view_t v = {gin + (size_t)b * in_elems, 0, 0, d[0], d[1], d[2], d[1] * d[2], d[0], d[1], &err};
            in = v;
          } else {
            const int* rp = rb + (size_t)(l - 1 - g0) * (rows + 1);
            view_t v = {band[l - 1 - g0], blo[l - 1 - g0], 0, rp[i + 1] - blo[l - 1 - g0], d[1], d[2],
                        d[1] * d[2], d[0], d[1], &err};
            in = v;
          }
          const size_t row_elems = (size_t)d[4] * d[5];
          if (l == g1) {  /* straight into the group output */
            layer_rect(&in, &layers[l], d[5], wt ? wt[l] : NULL, scale ? scale[l] : NULL,
                       bias ? bias[l] : NULL, round_bf16, r[i], r[i + 1], 0, d[4],
                       gout + (size_t)b * out_elems + (size_t)r[i] * row_elems);
          } else {  /* a new band: rows taken over from the old one, then its own */
            int lo = reuse_band_lo(layers, dims, g0, l, rows, rb, i);
            size_t nrows = (size_t)(r[i + 1] - lo);
            double* nb = (double*)malloc(sizeof(double) * (nrows ? nrows : 1) * row_elems);
            if (!nb) { rc = ORC_ENOMEM; break; }
            if (r[i] > lo) {
              /* those rows lie in the previous row's band, [blo, r[i]) */
              if (!band[l - g0] || lo < blo[l - g0]) { free(nb); rc = ORC_EREGION; break; }
              memcpy(nb, band[l - g0] + (size_t)(lo - blo[l - g0]) * row_elems,
                     sizeof(double) * (size_t)(r[i] - lo) * row_elems);
            }
            layer_rect(&in, &layers[l], d[5], wt ? wt[l] : NULL, scale ? scale[l] : NULL,
                       bias ? bias[l] : NULL, round_bf16, r[i], r[i + 1], 0, d[4],
                       nb + (size_t)(r[i] - lo) * row_elems);
            free(band[l - g0]);
            band[l - g0] = nb;
            blo[l - g0] = lo;
          }
          if (err) rc = err;
        }
      }
      for (int k = 0; k < nl && band; ++k) { free(band[k]); band[k] = NULL; }
    }
    free(band);
    free(blo);
    free(rb);
    free(owned);
    owned = fresh;
    gin = gout;
  }
  free(owned);
  free(dims);
  return rc;
}

int orc_forward_rect(const orc_layer* layers, int n, int h, int w, int c,
                     const double* x, const double* const* wt,
                     const double* const* scale, const double* const* bias,
                     int round_bf16, int oy0, int oy1, int ox0, int ox1,
                     double* y) {
  if (!x || !y) return ORC_EINVAL;
  int* dims = (int*)malloc(sizeof(int) * 6 * (size_t)n);
  int* regs = (int*)malloc(sizeof(int) * 8 * (size_t)(n > 0 ? n : 1));
  if (!dims || !regs) { free(dims); free(regs); return ORC_ENOMEM; }
  int rc = orc_shapes(layers, n, h, w, c, dims);
  const int* dl = dims + 6 * (n - 1);
  if (!rc && (oy0 < 0 || oy1 > dl[3] || oy0 >= oy1 || ox0 < 0 || ox1 > dl[4] || ox0 >= ox1)) rc = ORC_EINVAL;
  for (int l = 0; l < n && !rc; ++l)
    if (layers[l].op == ORC_CONV && (!wt || !wt[l] || !scale || !scale[l] || !bias || !bias[l])) rc = ORC_EINVAL;
  double* full = NULL;
  if (!rc) {
    /* back-project the requested rectangle through every layer */
    int a = oy0, b = oy1, p = ox0, q = ox1;
    for (int l = n - 1; l >= 0; --l) {
      const orc_layer* L = &layers[l];
      const int* d = dims + 6 * l;
      int iy0, iy1, ix0, ix1;
      back_project(a, b, L->f, L->s, L->p, d[0], &iy0, &iy1);
      back_project(p, q, L->f, L->s, L->p, d[1], &ix0, &ix1);
      int* r = regs + (size_t)l * 8;
      r[0] = iy0; r[1] = iy1; r[2] = ix0; r[3] = ix1;
      r[4] = a; r[5] = b; r[6] = p; r[7] = q;
      a = iy0; b = iy1; p = ix0; q = ix1;
    }
    full = (double*)calloc((size_t)dl[3] * dl[4] * dl[5], sizeof(double));
    if (!full) rc = ORC_ENOMEM;
  }
  if (!rc) rc = tile_forward(layers, dims, 0, n - 1, regs, x, full, wt, scale, bias, round_bf16);
  if (!rc) {
    int ow = ox1 - ox0;
    for (int yy = oy0; yy < oy1; ++yy)
      memcpy(y + (size_t)(yy - oy0) * ow * dl[5], full + ((size_t)yy * dl[4] + ox0) * dl[5],
             sizeof(double) * (size_t)ow * dl[5]);
  }
  free(full);
  free(dims);
  free(regs);
  return rc;
}

/* ------------------------------------------------------------------ */
/* variable tiling: balanced boundaries                                 */
/* ------------------------------------------------------------------ */

/* Extent, at the input of layer g0, of the input region that the output
 * interval [a, b) of layer g1 reads along one axis (axis 0: rows, 1:
 * columns), by back-projecting the interval layer by layer. */
static int task_extent(const orc_layer* layers, const int* dims, int g0, int g1, int axis,
                       int a, int b) {
  for (int l = g1; l >= g0; --l) {
    const orc_layer* L = &layers[l];
    int ia, ib;
    back_project(a, b, L->f, L->s, L->p, dims[6 * l + axis], &ia, &ib);
    a = ia;
    b = ib;
  }
  return b - a;
}

int orc_balanced_bounds(const orc_layer* layers, int n, int h, int w, int c, int g0, int g1,
                        int axis, int parts, int* bounds) {
  if (!bounds || g0 < 0 || g1 < g0 || g1 >= n || (axis != 0 && axis != 1) || parts < 1)
    return ORC_EINVAL;
  int* dims = (int*)malloc(sizeof(int) * 6 * (size_t)n);
  if (!dims) return ORC_ENOMEM;
  int rc = orc_shapes(layers, n, h, w, c, dims);
  const int E = rc ? 0 : dims[6 * g1 + 3 + axis];
  if (!rc && parts > E) rc = ORC_EINVAL;
  /* every choice of the parts-1 inner boundaries out of 1 .. E-1 */
  double combos = 1.0;
  for (int k = 0; k < parts - 1 && !rc; ++k) combos = combos * (double)(E - 1 - k) / (double)(k + 1);
  if (!rc && combos > 2.0e8) rc = ORC_EINVAL;  /* brute force only: small cases */
  int* cur = (int*)malloc(sizeof(int) * (size_t)(parts + 1));
  if (!rc && !cur) rc = ORC_ENOMEM;
  if (!rc) {
    long long best_max = -1, best_sq = 0;
    for (int k = 0; k <= parts; ++k) cur[k] = (k == parts) ? E : k;  /* first in lexicographic order */
    for (;;) {
      long long mx = 0, sq = 0;
      for (int k = 0; k < parts; ++k) {
        long long t = task_extent(layers, dims, g0, g1, axis, cur[k], cur[k + 1]);
        if (t > mx) mx = t;
        sq += t * t;
      }
      /* strictly better only: the first optimum in lexicographic order stays */
      if (best_max < 0 || mx < best_max || (mx == best_max && sq < best_sq)) {
        best_max = mx;
        best_sq = sq;
        memcpy(bounds, cur, sizeof(int) * (size_t)(parts + 1));
      }
      /* next combination: the last inner boundary that can still move */
      int k = parts - 1;
      while (k >= 1 && cur[k] == E - (parts - k)) --k;
      if (k < 1) break;
      ++cur[k];
      for (int j = k + 1; j < parts; ++j) cur[j] = cur[j - 1] + 1;
    }
  }
  free(cur);
  free(dims);
  return rc;
}
