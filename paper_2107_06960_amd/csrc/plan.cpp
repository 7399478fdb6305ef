// plan.cpp -- host-side planning for fused tile partitioning (MAFAT,
// arXiv 2107.06960): shape inference, per-group output tile partition,
// per-tile region back-projection, stage decomposition for the kernels,
// workspace sizing and multiply-accumulate accounting.  Pure integer host
// code; no HIP calls.
#include <algorithm>
#include <climits>
#include <cstdint>
#include <cstring>
#include <new>

#include "mafat_internal.h"

namespace mafat {

static thread_local std::string g_last_error;
void set_error(const std::string& msg) { g_last_error = msg; }
void clear_error() { g_last_error.clear(); }

namespace {

bool layer_supported(const mafat_layer& L, std::string* why) {
  // Any square filter up to kMaxFilter, stride up to kMaxStride, padding
  // below the filter size (zero padding for a convolution; a max-pool takes
  // the maximum over the in-image elements of its window).
  if (L.op != MAFAT_CONV && L.op != MAFAT_MAXPOOL) { *why = "unknown layer op"; return false; }
  if (L.f < 1 || L.f > kMaxFilter) { *why = "filter must be 1.." + std::to_string(kMaxFilter); return false; }
  if (L.s < 1 || L.s > kMaxStride) { *why = "stride must be 1.." + std::to_string(kMaxStride); return false; }
  if (L.p < 0 || L.p >= L.f) { *why = "padding must be 0..f-1"; return false; }
  if (L.op == MAFAT_CONV) {
    if (L.c_out < 1) { *why = "convolution c_out must be positive"; return false; }
    if (L.act != MAFAT_ACT_LINEAR && L.act != MAFAT_ACT_LEAKY01) { *why = "unknown activation"; return false; }
  }
  return true;
}

// A 2x2, stride 2, unpadded max-pool: the one a convolution stage takes
// into its epilogue.
bool pool_2x2(const mafat_layer& L) { return L.op == MAFAT_MAXPOOL && L.f == 2 && L.s == 2 && L.p == 0; }

// Tile i of N over the extent [0, E): [floor(iE/N), floor((i+1)E/N)).
void split(int E, int N, int i, int* a, int* b) {
  *a = static_cast<int>((static_cast<int64_t>(i) * E) / N);
  *b = static_cast<int>((static_cast<int64_t>(i + 1) * E) / N);
}

// The input interval [ia, ib) that outputs [a, b) of a layer with filter F,
// stride S and padding P read, clipped to the input extent [0, E).
void back_project(int a, int b, int F, int S, int P, int E, int* ia, int* ib) {
  *ia = std::max(0, a * S - P);
  *ib = std::min(E, (b - 1) * S - P + F);
}

// Where the input rows (axis 0) or columns (axis 1) that outputs ending at
// b (starting at a) read end (start), through layers [lf, ll] of a stack:
// back_project's two ends, taken apart.
int end_through(const mafat_plan& P, int lf, int ll, int axis, int b) {
  for (int l = ll; l >= lf && b > 0; --l) {
    const mafat_layer& L = P.layers[l];
    b = std::min(P.dims[l][axis], (b - 1) * L.s - L.p + L.f);
  }
  return std::max(b, 0);
}
int start_through(const mafat_plan& P, int lf, int ll, int axis, int a) {
  for (int l = ll; l >= lf; --l) {
    const mafat_layer& L = P.layers[l];
    a = std::max(0, a * L.s - L.p);
  }
  return a;
}

// Boundaries b[0..N] of N parts of [0, E): 0 = b[0] < ... < b[N] = E.
bool bounds_valid(const int32_t* b, int N, int E) {
  if (b[0] != 0 || b[N] != E) return false;
  for (int i = 0; i < N; ++i)
    if (b[i + 1] <= b[i]) return false;
  return true;
}

// rb / cb: the group output's row / column boundaries (rows + 1 / cols + 1
// values), or NULL for the even floor split.
int build_group(mafat_plan& plan, int g0, int g1, int rows, int cols, bool partition, bool reuse,
                const int32_t* rb, const int32_t* cb, Group* out) {
  Group G;
  G.partition = partition;
  G.reuse = reuse;
  G.l0 = g0; G.l1 = g1; G.rows = rows; G.cols = cols; G.ntiles = rows * cols;
  const int nl = g1 - g0 + 1;
  const auto& dl = plan.dims[g1];
  if (rows < 1 || cols < 1 || rows > dl[3] || cols > dl[4]) {
    set_error("grid " + std::to_string(rows) + "x" + std::to_string(cols) +
              " does not fit the group output " + std::to_string(dl[3]) + "x" + std::to_string(dl[4]));
    return MAFAT_ESHAPE;
  }
  if ((rb && !bounds_valid(rb, rows, dl[3])) || (cb && !bounds_valid(cb, cols, dl[4]))) {
    set_error("tile boundaries of a group must rise strictly from 0 to its output extent (" +
              std::to_string(dl[3]) + " rows, " + std::to_string(dl[4]) + " columns)");
    return MAFAT_ESHAPE;
  }
  G.in_r.resize(static_cast<size_t>(G.ntiles) * nl);
  G.out_r.resize(static_cast<size_t>(G.ntiles) * nl);
  for (int i = 0; i < rows; ++i)
    for (int j = 0; j < cols; ++j) {
      const int t = i * cols + j;
      mafat_rect o;
      if (rb) { o.y0 = rb[i]; o.y1 = rb[i + 1]; } else split(dl[3], rows, i, &o.y0, &o.y1);
      if (cb) { o.x0 = cb[j]; o.x1 = cb[j + 1]; } else split(dl[4], cols, j, &o.x0, &o.x1);
      for (int l = g1; l >= g0; --l) {
        const mafat_layer& L = plan.layers[l];
        const auto& d = plan.dims[l];
        mafat_rect in;
        back_project(o.y0, o.y1, L.f, L.s, L.p, d[0], &in.y0, &in.y1);
        back_project(o.x0, o.x1, L.f, L.s, L.p, d[1], &in.x0, &in.x1);
        G.out_r[static_cast<size_t>(t) * nl + (l - g0)] = o;
        G.in_r[static_cast<size_t>(t) * nl + (l - g0)] = in;
        o = in;
      }
    }

  // Multiply-accumulates per frame.
  G.macs_exec = G.macs_untiled = 0;
  for (int l = g0; l <= g1; ++l) {
    const mafat_layer& L = plan.layers[l];
    if (L.op != MAFAT_CONV) continue;
    const auto& d = plan.dims[l];
    const int64_t per_px = static_cast<int64_t>(d[5]) * L.f * L.f * d[2];
    G.macs_untiled += static_cast<int64_t>(d[3]) * d[4] * per_px;
    for (int t = 0; t < G.ntiles; ++t) {
      const mafat_rect& r = G.out_r[static_cast<size_t>(t) * nl + (l - g0)];
      G.macs_exec += static_cast<int64_t>(r.y1 - r.y0) * (r.x1 - r.x0) * per_px;
    }
  }

  // Stages: a convolution directly followed (inside the group) by a 2x2/2
  // max-pool is one stage with the pool fused into its epilogue.
  for (int l = g0; l <= g1;) {
    Stage S{};
    const mafat_layer& L = plan.layers[l];
    S.first = l;
    if (L.op == MAFAT_CONV) {
      S.kind = STAGE_CONV;
      S.pool = (l + 1 <= g1 && pool_2x2(plan.layers[l + 1]));
      S.last = S.pool ? l + 1 : l;
      S.f = L.f; S.s = L.s; S.p = L.p; S.act = L.act;
    } else {
      S.kind = STAGE_POOL;
      S.pool = false;
      S.last = l;
      S.f = L.f; S.s = L.s; S.p = L.p; S.act = MAFAT_ACT_LINEAR;
    }
    const auto& din = plan.dims[S.first];
    const auto& dout = plan.dims[S.last];
    S.in_h = din[0]; S.in_w = din[1]; S.cin = din[2];
    S.out_h = dout[3]; S.out_w = dout[4]; S.cout = dout[5];
    G.stages.push_back(S);
    l = S.last + 1;
  }
  const int ns = static_cast<int>(G.stages.size());
  G.nbufs = std::min(2, ns - 1);
  G.scratch_elems = 0;
  if (reuse) {
    // Row reuse (data reuse between tiles run in order): tile rows one after
    // another.  The group output's parts are the tiles; every earlier stage
    // output is cut at the ends of what the next stage's parts read (the
    // back-projected ends of its boundaries), so tile row i computes, at
    // every stage, the rows below row i - 1's that its own next stage reads
    // and no row twice.  Columns are cut the same way (the tiles of a row
    // run together, so any cut would do).  A stage output that is not the
    // group's lives in a band of full-width rows: [band_lo[i], row_b[i+1])
    // for tile row i, band_lo[i] being the first row its next stage reads
    // (or its own first computed row, if lower); the rows above its own come
    // from row i - 1's band, moved up in the same buffer or, where the rows
    // they leave and the rows they go to would overlap, from the other of
    // two buffers the rows alternate between.
    std::vector<std::vector<int>> rbs(ns), cbs(ns);
    rbs[ns - 1].resize(rows + 1);
    cbs[ns - 1].resize(cols + 1);
    for (int i = 0; i <= rows; ++i) {
      int a, b;
      split(dl[3], rows, std::min(i, rows - 1), &a, &b);
      rbs[ns - 1][i] = rb ? rb[i] : (i < rows ? a : dl[3]);
    }
    for (int j = 0; j <= cols; ++j) {
      int a, b;
      split(dl[4], cols, std::min(j, cols - 1), &a, &b);
      cbs[ns - 1][j] = cb ? cb[j] : (j < cols ? a : dl[4]);
    }
    for (int s = ns - 2; s >= 0; --s) {
      const Stage& N = G.stages[s + 1];
      rbs[s].assign(rows + 1, 0);
      cbs[s].assign(cols + 1, 0);
      for (int i = 1; i <= rows; ++i) rbs[s][i] = end_through(plan, N.first, N.last, 0, rbs[s + 1][i]);
      for (int j = 1; j <= cols; ++j) cbs[s][j] = end_through(plan, N.first, N.last, 1, cbs[s + 1][j]);
      Stage& S = G.stages[s];
      S.row_b = rbs[s];
      S.band_lo.assign(rows, 0);
      S.band_rows = 0;
      S.band_copies = 1;
      for (int i = 0; i < rows; ++i) {
        S.band_lo[i] = std::min(start_through(plan, N.first, N.last, 0, rbs[s + 1][i]), rbs[s][i]);
        S.band_rows = std::max(S.band_rows, rbs[s][i + 1] - S.band_lo[i]);
        // the rows taken over, [band_lo[i], row_b[i]), move from band
        // position band_lo[i] - band_lo[i-1] to position 0
        if (i > 0 && rbs[s][i] - S.band_lo[i] > S.band_lo[i] - S.band_lo[i - 1]) S.band_copies = 2;
      }
    }
    int64_t frame = 0;  // the bands of every stage output (an upper bound of any dtype's)
    for (int s = 0; s < ns; ++s) {
      Stage& S = G.stages[s];
      S.src_buf = (s == 0) ? BUF_GROUP_IO : BUF_SCRATCH0;
      S.dst_buf = (s == ns - 1) ? BUF_GROUP_IO : BUF_SCRATCH0;
      if (s < ns - 1)
        frame += S.band_copies * ((static_cast<int64_t>(S.band_rows) * S.out_w * S.cout + 127) / 128 * 128);
      const int k = S.pool ? 2 : 1;
      for (int i = 0; i < rows; ++i)
        for (int j = 0; j < cols; ++j) {
          TileGeom T{};
          T.cy0 = k * rbs[s][i]; T.ch = k * (rbs[s][i + 1] - rbs[s][i]);
          T.cx0 = k * cbs[s][j]; T.cw = k * (cbs[s][j + 1] - cbs[s][j]);
          T.sy0 = (s == 0) ? 0 : G.stages[s - 1].band_lo[i];
          T.sx0 = 0; T.sw = S.in_w;
          T.dy0 = (s == ns - 1) ? 0 : S.band_lo[i];
          T.dx0 = 0; T.dw = S.out_w;
          T.src_off = T.dst_off = 0;  // band bases: per dtype, at run time
          S.tiles.push_back(T);
        }
    }
    G.nbufs = 0;
    G.scratch_frame = frame;
    G.tile_batch = cols;
    G.macs_exec = 0;
    for (const Stage& S : G.stages)
      if (S.kind == STAGE_CONV)
        for (const TileGeom& T : S.tiles)
          G.macs_exec += static_cast<int64_t>(T.ch) * T.cw * S.cout * S.f * S.f * S.cin;
    *out = std::move(G);
    return MAFAT_OK;
  }
  if (partition) {
    // Tile reuse (the data reuse between adjacent tiles of DeepThings'
    // fused tile partitioning, taken to the whole stage): the stages run one
    // after another over all tiles, so every stage's output is partitioned
    // into the group's grid (the same floor boundaries as the group output)
    // and each tile computes only its own part, into a full tensor of the
    // stage output; the next stage reads its halo from the neighbours'
    // parts.  Nothing is computed twice.  A conv stage with a fused pool
    // computes the conv outputs of its pool windows (twice the partition).
    for (int s = 0; s < ns; ++s) {
      Stage& S = G.stages[s];
      S.src_buf = (s == 0) ? BUF_GROUP_IO : ((s - 1) % 2);
      S.dst_buf = (s == ns - 1) ? BUF_GROUP_IO : (s % 2);
      if (S.dst_buf != BUF_GROUP_IO)
        G.scratch_elems = std::max<int64_t>(G.scratch_elems, static_cast<int64_t>(S.out_h) * S.out_w * S.cout);
      for (int i = 0; i < rows; ++i)
        for (int j = 0; j < cols; ++j) {
          int y0, y1, x0, x1;
          split(S.out_h, rows, i, &y0, &y1);
          split(S.out_w, cols, j, &x0, &x1);
          TileGeom T{};
          const int k = S.pool ? 2 : 1;
          T.cy0 = k * y0; T.ch = k * (y1 - y0);
          T.cx0 = k * x0; T.cw = k * (x1 - x0);
          T.sy0 = 0; T.sx0 = 0; T.sw = S.in_w;
          T.src_off = (S.src_buf == BUF_GROUP_IO) ? 0 : S.src_buf;  // scaled below
          T.dy0 = 0; T.dx0 = 0; T.dw = S.out_w;
          T.dst_off = (S.dst_buf == BUF_GROUP_IO) ? 0 : S.dst_buf;  // scaled below
          S.tiles.push_back(T);
        }
    }
    // Scratch of one frame: [buffer][full stage output], 256-byte aligned.
    G.scratch_elems = (G.scratch_elems + 127) / 128 * 128;
    G.scratch_frame = static_cast<int64_t>(G.nbufs) * G.scratch_elems;
    G.tile_batch = G.ntiles;
    for (Stage& S : G.stages)
      for (TileGeom& T : S.tiles) {
        if (S.src_buf != BUF_GROUP_IO) T.src_off *= G.scratch_elems;
        if (S.dst_buf != BUF_GROUP_IO) T.dst_off *= G.scratch_elems;
      }
    G.macs_exec = 0;  // the conv outputs computed (all of them, less the rows/columns an odd pool drops)
    for (const Stage& S : G.stages)
      if (S.kind == STAGE_CONV)
        for (const TileGeom& T : S.tiles)
          G.macs_exec += static_cast<int64_t>(T.ch) * T.cw * S.cout * S.f * S.f * S.cin;
    *out = std::move(G);
    return MAFAT_OK;
  }
  for (int s = 0; s < ns; ++s) {
    Stage& S = G.stages[s];
    S.src_buf = (s == 0) ? BUF_GROUP_IO : ((s - 1) % 2);
    S.dst_buf = (s == ns - 1) ? BUF_GROUP_IO : (s % 2);
    for (int t = 0; t < G.ntiles; ++t) {
      const mafat_rect& cr = G.out_r[static_cast<size_t>(t) * nl + (S.first - g0)];  // computed rect
      const mafat_rect& sr = G.in_r[static_cast<size_t>(t) * nl + (S.first - g0)];   // read rect
      const mafat_rect& orr = G.out_r[static_cast<size_t>(t) * nl + (S.last - g0)];  // written rect
      TileGeom T{};
      if (S.kind == STAGE_CONV) {
        T.cy0 = cr.y0; T.cx0 = cr.x0; T.ch = cr.y1 - cr.y0; T.cw = cr.x1 - cr.x0;
      } else {
        T.cy0 = orr.y0; T.cx0 = orr.x0; T.ch = orr.y1 - orr.y0; T.cw = orr.x1 - orr.x0;
      }
      if (S.src_buf == BUF_GROUP_IO) {
        T.sy0 = 0; T.sx0 = 0; T.sw = S.in_w; T.src_off = 0;
      } else {
        T.sy0 = sr.y0; T.sx0 = sr.x0; T.sw = sr.x1 - sr.x0;
        T.src_off = (static_cast<int64_t>(S.src_buf) * G.ntiles + t);  // scaled below
      }
      if (S.dst_buf == BUF_GROUP_IO) {
        T.dy0 = 0; T.dx0 = 0; T.dw = S.out_w; T.dst_off = 0;
      } else {
        T.dy0 = orr.y0; T.dx0 = orr.x0; T.dw = orr.x1 - orr.x0;
        T.dst_off = (static_cast<int64_t>(S.dst_buf) * G.ntiles + t);  // scaled below
        G.scratch_elems = std::max<int64_t>(
            G.scratch_elems, static_cast<int64_t>(orr.y1 - orr.y0) * (orr.x1 - orr.x0) * S.cout);
      }
      S.tiles.push_back(T);
    }
  }
  // Scratch buffers of one frame: [buffer][tile][scratch_elems]; every
  // tile's buffer starts on a 256-byte boundary for both dtypes.
  G.scratch_elems = (G.scratch_elems + 127) / 128 * 128;
  G.scratch_frame = static_cast<int64_t>(G.nbufs) * G.ntiles * G.scratch_elems;
  G.tile_batch = G.ntiles;
  for (Stage& S : G.stages)
    for (TileGeom& T : S.tiles) {
      if (S.src_buf != BUF_GROUP_IO) T.src_off *= G.scratch_elems;
      if (S.dst_buf != BUF_GROUP_IO) T.dst_off *= G.scratch_elems;
    }
  *out = std::move(G);
  return MAFAT_OK;
}

// Tile batches of K tiles (fused tile partitioning without the stage partition):
// tile t's intermediates live in slot t mod K of each scratch buffer, so
// the workspace holds K tiles ([buffer][slot][scratch_elems] per frame).
void set_tile_batch(Group& G, int K) {
  G.tile_batch = K;
  G.scratch_frame = static_cast<int64_t>(G.nbufs) * K * G.scratch_elems;
  for (Stage& S : G.stages)
    for (int t = 0; t < G.ntiles; ++t) {
      TileGeom& T = S.tiles[static_cast<size_t>(t)];
      const int64_t slot = t % K;
      if (S.src_buf != BUF_GROUP_IO) T.src_off = (S.src_buf * static_cast<int64_t>(K) + slot) * G.scratch_elems;
      if (S.dst_buf != BUF_GROUP_IO) T.dst_off = (S.dst_buf * static_cast<int64_t>(K) + slot) * G.scratch_elems;
    }
}

}  // namespace
}  // namespace mafat

using namespace mafat;

extern "C" int mafat_plan_create(const mafat_layer* layers, int32_t n_layers, int32_t in_h,
                                 int32_t in_w, int32_t in_c, const int32_t* group_start,
                                 int32_t n_groups, const int32_t* grid_rows,
                                 const int32_t* grid_cols, mafat_plan** out) {
  return mafat_plan_create_flags(layers, n_layers, in_h, in_w, in_c, group_start, n_groups, grid_rows, grid_cols,
                                 0, out);
}

extern "C" int mafat_plan_create_flags(const mafat_layer* layers, int32_t n_layers, int32_t in_h,
                                       int32_t in_w, int32_t in_c, const int32_t* group_start,
                                       int32_t n_groups, const int32_t* grid_rows,
                                       const int32_t* grid_cols, int32_t flags, mafat_plan** out) {
  return mafat_plan_create_bounds(layers, n_layers, in_h, in_w, in_c, group_start, n_groups, grid_rows,
                                  grid_cols, nullptr, nullptr, flags, out);
}

extern "C" int mafat_plan_create_bounds(const mafat_layer* layers, int32_t n_layers, int32_t in_h,
                                        int32_t in_w, int32_t in_c, const int32_t* group_start,
                                        int32_t n_groups, const int32_t* grid_rows,
                                        const int32_t* grid_cols, const int32_t* row_bounds,
                                        const int32_t* col_bounds, int32_t flags, mafat_plan** out) {
  clear_error();
  if (!out) { set_error("out is NULL"); return MAFAT_EINVAL; }
  *out = nullptr;
  if (flags & ~(MAFAT_PLAN_STAGE_PARTITION | MAFAT_PLAN_PACKED_WEIGHTS | MAFAT_PLAN_ROW_REUSE)) {
    set_error("unknown plan flags");
    return MAFAT_EINVAL;
  }
  if ((flags & MAFAT_PLAN_STAGE_PARTITION) && (flags & MAFAT_PLAN_ROW_REUSE)) {
    set_error("the stage partition and row reuse are two different executions: choose one");
    return MAFAT_EUNSUPPORTED;
  }
  if ((flags & MAFAT_PLAN_STAGE_PARTITION) && (row_bounds || col_bounds)) {
    set_error("the stage partition splits every stage evenly: no tile boundaries with it");
    return MAFAT_EUNSUPPORTED;
  }
  if (!layers || !group_start || !grid_rows || !grid_cols || n_layers < 1 || n_groups < 1) {
    set_error("null pointer or empty layer/group list");
    return MAFAT_EINVAL;
  }
  if (in_h < 1 || in_w < 1 || in_c < 1 || in_h > kMaxExtent || in_w > kMaxExtent) {
    set_error("input extent out of range");
    return MAFAT_ESHAPE;
  }
  mafat_plan* plan = new (std::nothrow) mafat_plan();
  if (!plan) return MAFAT_ENOMEM;
  try {
    plan->n = n_layers; plan->in_h = in_h; plan->in_w = in_w; plan->in_c = in_c;
    plan->packed_weights = (flags & MAFAT_PLAN_PACKED_WEIGHTS) != 0;
    plan->layers.assign(layers, layers + n_layers);
    int h = in_h, w = in_w, c = in_c;
    for (int l = 0; l < n_layers; ++l) {
      const mafat_layer& L = layers[l];
      std::string why;
      if (!layer_supported(L, &why)) {
        set_error("layer " + std::to_string(l) + ": " + why);
        delete plan;
        return (L.op == MAFAT_CONV || L.op == MAFAT_MAXPOOL) ? MAFAT_EUNSUPPORTED : MAFAT_EINVAL;
      }
      const int oh_num = h + 2 * L.p - L.f, ow_num = w + 2 * L.p - L.f;
      if (oh_num < 0 || ow_num < 0) {
        set_error("layer " + std::to_string(l) + ": input smaller than the filter");
        delete plan;
        return MAFAT_ESHAPE;
      }
      const int oh = oh_num / L.s + 1, ow = ow_num / L.s + 1;
      const int oc = (L.op == MAFAT_CONV) ? L.c_out : c;
      plan->dims.push_back({h, w, c, oh, ow, oc});
      h = oh; w = ow; c = oc;
    }
    if (group_start[0] != 0) {
      set_error("group_start[0] must be 0");
      delete plan;
      return MAFAT_ESHAPE;
    }
    const int32_t *rb = row_bounds, *cb = col_bounds;
    for (int g = 0; g < n_groups; ++g) {
      const int g0 = group_start[g];
      const int end = (g + 1 < n_groups) ? group_start[g + 1] : n_layers;
      if (g0 < 0 || end <= g0 || end > n_layers) {
        set_error("group starts must be strictly increasing and below n_layers");
        delete plan;
        return MAFAT_ESHAPE;
      }
      Group G;
      const int rc = build_group(*plan, g0, end - 1, grid_rows[g], grid_cols[g],
                                 (flags & MAFAT_PLAN_STAGE_PARTITION) != 0, (flags & MAFAT_PLAN_ROW_REUSE) != 0,
                                 rb, cb, &G);
      if (rc != MAFAT_OK) { delete plan; return rc; }
      if (rb) rb += grid_rows[g] + 1;
      if (cb) cb += grid_cols[g] + 1;
      plan->groups.push_back(std::move(G));
    }
  } catch (const std::bad_alloc&) {
    delete plan;
    set_error("host allocation failed");
    return MAFAT_ENOMEM;
  }
  *out = plan;
  return MAFAT_OK;
}

namespace mafat {
namespace {

// Balanced boundaries of N parts along one axis (0: rows, 1: columns) of
// the output of layers [g0, g1] (variable tiling).  A part's task extent is
// the extent of the input region of layer g0 that its output interval
// reads; the result minimises the largest task extent, then the sum of the
// squared task extents, and is the first such boundary list in
// lexicographic order.
//
// Back-projection maps an interval's start and end independently, so the
// task extent of [a, b) is END[b] - START[a], non-increasing in a and
// non-decreasing in b.  Hence (1) the smallest feasible largest extent T is
// found by bisection, a T being feasible when the greedy left-to-right
// cover (each part as long as T allows) needs at most N parts -- any cover
// with fewer parts refines into exactly N, sub-intervals never costing more;
// (2) boundary k of any cover with extents <= T lies in a window: at most the
// greedy reach of k parts from the left, at least the greedy reach of N - k
// parts from the right; a dynamic programme over the windows minimises the
// sum of squares, and the reconstruction takes the smallest boundary at each
// step.
int balanced_axis(const mafat_plan& P, int g0, int g1, int axis, int N, int32_t* out) {
  const int E = P.dims[g1][3 + axis];
  if (N < 1 || N > E) {
    set_error("parts " + std::to_string(N) + " outside 1.." + std::to_string(E));
    return MAFAT_ESHAPE;
  }
  std::vector<int64_t> st(static_cast<size_t>(E) + 1), en(static_cast<size_t>(E) + 1);
  for (int v = 0; v <= E; ++v) {
    int64_t a = v, b = v;
    for (int l = g1; l >= g0; --l) {
      const mafat_layer& L = P.layers[l];
      const int64_t Ein = P.dims[l][axis];
      a = std::max<int64_t>(0, a * L.s - L.p);
      b = std::min<int64_t>(Ein, (b - 1) * L.s - L.p + L.f);
    }
    st[v] = a;
    en[v] = b;
  }
  auto cost = [&](int a, int b) { return en[b] - st[a]; };
  // Greedy reach from the left after k parts (capped at E) and from the
  // right after j parts, for a bound T; -1 / E + 1 when a part cannot
  // advance.
  auto reach_left = [&](int64_t T, std::vector<int>* r) {
    r->assign(static_cast<size_t>(N) + 1, E);
    int pos = 0, b = 1;
    (*r)[0] = 0;
    for (int k = 1; k <= N; ++k) {
      if (pos >= E) { (*r)[k] = E; continue; }
      if (b <= pos) b = pos + 1;
      if (cost(pos, b) > T) { for (int j = k; j <= N; ++j) (*r)[j] = -1; return; }
      while (b < E && cost(pos, b + 1) <= T) ++b;
      pos = b;
      (*r)[k] = pos;
    }
  };
  auto reach_right = [&](int64_t T, std::vector<int>* q) {
    q->assign(static_cast<size_t>(N) + 1, 0);
    int pos = E, a = E - 1;
    (*q)[0] = E;
    for (int j = 1; j <= N; ++j) {
      if (pos <= 0) { (*q)[j] = 0; continue; }
      if (a >= pos) a = pos - 1;
      if (cost(a, pos) > T) { for (int i = j; i <= N; ++i) (*q)[i] = E + 1; return; }
      while (a > 0 && cost(a - 1, pos) <= T) --a;
      pos = a;
      (*q)[j] = pos;
    }
  };
  std::vector<int> r, q;
  int64_t lo = 1, hi = cost(0, E);
  while (lo < hi) {
    const int64_t mid = lo + (hi - lo) / 2;
    reach_left(mid, &r);
    if (r[N] == E) hi = mid; else lo = mid + 1;
  }
  const int64_t T = lo;
  reach_left(T, &r);
  reach_right(T, &q);
  std::vector<int> wlo(static_cast<size_t>(N) + 1), whi(static_cast<size_t>(N) + 1);
  double work = 0;
  for (int k = 0; k <= N; ++k) {
    wlo[k] = std::max(k, q[N - k]);
    whi[k] = std::min(r[k], E - (N - k));
    if (wlo[k] > whi[k]) {
      set_error("internal: empty boundary window");
      return MAFAT_EINVAL;
    }
    if (k > 0) work += static_cast<double>(whi[k] - wlo[k] + 1) * (whi[k - 1] - wlo[k - 1] + 1);
  }
  if (work > 4.0e9) {
    set_error("balanced boundaries: search too large");
    return MAFAT_EUNSUPPORTED;
  }
  // s[k][b - wlo[k]]: least sum of squares covering [b, E) with N - k parts.
  constexpr int64_t INF = INT64_MAX;
  std::vector<std::vector<int64_t>> sfx(static_cast<size_t>(N) + 1);
  for (int k = N; k >= 0; --k) {
    sfx[k].assign(static_cast<size_t>(whi[k] - wlo[k] + 1), INF);
    for (int b = wlo[k]; b <= whi[k]; ++b) {
      if (k == N) { sfx[k][b - wlo[k]] = (b == E) ? 0 : INF; continue; }
      int64_t best = INF;
      for (int c = std::max(b + 1, wlo[k + 1]); c <= whi[k + 1]; ++c) {
        const int64_t t = cost(b, c);
        if (t > T) break;  // non-decreasing in c
        const int64_t rest = sfx[k + 1][c - wlo[k + 1]];
        if (rest != INF) best = std::min(best, t * t + rest);
      }
      sfx[k][b - wlo[k]] = best;
    }
  }
  if (sfx[0][0] == INF) {
    set_error("internal: no balanced cover");
    return MAFAT_EINVAL;
  }
  out[0] = 0;
  for (int k = 1; k <= N; ++k) {
    const int b = out[k - 1];
    const int64_t need = sfx[k - 1][b - wlo[k - 1]];
    int pick = -1;
    for (int c = std::max(b + 1, wlo[k]); c <= whi[k]; ++c) {
      const int64_t t = cost(b, c);
      if (t > T) break;
      const int64_t rest = sfx[k][c - wlo[k]];
      if (rest != INF && t * t + rest == need) { pick = c; break; }
    }
    if (pick < 0) {
      set_error("internal: balanced reconstruction failed");
      return MAFAT_EINVAL;
    }
    out[k] = pick;
  }
  return MAFAT_OK;
}

}  // namespace
}  // namespace mafat

extern "C" int mafat_balanced_bounds(const mafat_layer* layers, int32_t n_layers, int32_t in_h,
                                     int32_t in_w, int32_t in_c, int32_t first_layer,
                                     int32_t last_layer, int32_t rows, int32_t cols,
                                     int32_t* row_bounds, int32_t* col_bounds) {
  clear_error();
  if (!layers || n_layers < 1 || first_layer < 0 || last_layer < first_layer || last_layer >= n_layers) {
    set_error("null layer list or layer range outside the stack");
    return MAFAT_EINVAL;
  }
  const int32_t start = 0, one = 1;
  mafat_plan* plan = nullptr;
  int rc = mafat_plan_create(layers, n_layers, in_h, in_w, in_c, &start, 1, &one, &one, &plan);
  if (rc != MAFAT_OK) return rc;  // shape inference errors, with their message
  try {
    if (row_bounds) rc = balanced_axis(*plan, first_layer, last_layer, 0, rows, row_bounds);
    if (rc == MAFAT_OK && col_bounds) rc = balanced_axis(*plan, first_layer, last_layer, 1, cols, col_bounds);
  } catch (const std::bad_alloc&) {
    set_error("host allocation failed");
    rc = MAFAT_ENOMEM;
  }
  mafat_plan_destroy(plan);
  return rc;
}

extern "C" void mafat_plan_destroy(mafat_plan* plan) { delete plan; }

extern "C" int mafat_plan_layer_shape(const mafat_plan* plan, int32_t layer, int32_t dims[6]) {
  if (!plan || !dims || layer < 0 || layer >= plan->n) return MAFAT_EINVAL;
  for (int k = 0; k < 6; ++k) dims[k] = plan->dims[layer][k];
  return MAFAT_OK;
}

extern "C" int mafat_plan_group(const mafat_plan* plan, int32_t group, int32_t* first_layer,
                                int32_t* n_layers, int32_t* n_tiles) {
  if (!plan || group < 0 || group >= static_cast<int>(plan->groups.size())) return MAFAT_EINVAL;
  const Group& G = plan->groups[group];
  if (first_layer) *first_layer = G.l0;
  if (n_layers) *n_layers = G.l1 - G.l0 + 1;
  if (n_tiles) *n_tiles = G.ntiles;
  return MAFAT_OK;
}

extern "C" int mafat_plan_num_tiles(const mafat_plan* plan, int32_t group, int32_t* n_tiles) {
  clear_error();
  if (!plan || !n_tiles || group < 0 || group >= static_cast<int>(plan->groups.size())) {
    set_error("plan and n_tiles must be non-NULL and the group in range");
    return MAFAT_EINVAL;
  }
  *n_tiles = plan->groups[group].ntiles;
  return MAFAT_OK;
}

extern "C" int mafat_plan_regions(const mafat_plan* plan, int32_t group, mafat_rect* in_rects,
                                  mafat_rect* out_rects, int64_t capacity) {
  if (!plan || group < 0 || group >= static_cast<int>(plan->groups.size())) return MAFAT_EINVAL;
  const Group& G = plan->groups[group];
  const int64_t need = static_cast<int64_t>(G.in_r.size());
  if (capacity < need) {
    set_error("region capacity " + std::to_string(capacity) + " < " + std::to_string(need));
    return MAFAT_EINVAL;
  }
  if (in_rects) std::memcpy(in_rects, G.in_r.data(), sizeof(mafat_rect) * need);
  if (out_rects) std::memcpy(out_rects, G.out_r.data(), sizeof(mafat_rect) * need);
  return MAFAT_OK;
}

extern "C" int mafat_plan_macs(const mafat_plan* plan, int32_t group, int64_t* executed,
                               int64_t* untiled) {
  if (!plan || group < 0 || group >= static_cast<int>(plan->groups.size())) return MAFAT_EINVAL;
  if (executed) *executed = plan->groups[group].macs_exec;
  if (untiled) *untiled = plan->groups[group].macs_untiled;
  return MAFAT_OK;
}

extern "C" int mafat_plan_stages(const mafat_plan* plan, int32_t group, int32_t* n_stages) {
  if (!plan || !n_stages || group < 0 || group >= static_cast<int>(plan->groups.size()))
    return MAFAT_EINVAL;
  *n_stages = static_cast<int32_t>(plan->groups[group].stages.size());
  return MAFAT_OK;
}

extern "C" int mafat_plan_stage_layers(const mafat_plan* plan, int32_t group, int32_t stage,
                                       int32_t* first_layer, int32_t* last_layer) {
  if (!plan || group < 0 || group >= static_cast<int>(plan->groups.size())) return MAFAT_EINVAL;
  const Group& G = plan->groups[group];
  if (stage < 0 || stage >= static_cast<int>(G.stages.size())) return MAFAT_EINVAL;
  if (first_layer) *first_layer = G.stages[stage].first;
  if (last_layer) *last_layer = G.stages[stage].last;
  return MAFAT_OK;
}

extern "C" int mafat_plan_set_tile_batch(mafat_plan* plan, int32_t tiles) {
  clear_error();
  if (!plan || tiles < 0) {
    set_error("plan must be non-NULL and tiles >= 0");
    return MAFAT_EINVAL;
  }
  for (const Group& G : plan->groups)
    if (G.reuse) {
      set_error("row reuse runs one tile row at a time: no other tile batches");
      return MAFAT_EUNSUPPORTED;
    }
  for (const Group& G : plan->groups)
    if (G.partition && tiles > 0 && tiles < G.ntiles) {
      set_error("the stage partition needs every tile of a stage before the next stage: no tile batches");
      return MAFAT_EUNSUPPORTED;
    }
  for (Group& G : plan->groups)
    if (!G.partition) set_tile_batch(G, (tiles == 0) ? G.ntiles : std::min<int>(tiles, G.ntiles));
  return MAFAT_OK;
}

extern "C" int mafat_workspace_size(const mafat_plan* plan, int32_t batch, int32_t dtype,
                                    size_t* bytes) {
  if (!plan || !bytes || batch < 1) return MAFAT_EINVAL;
  if (dtype != MAFAT_F32 && dtype != MAFAT_BF16) return MAFAT_EUNSUPPORTED;
  size_t best = 0;
  for (const Group& G : plan->groups) best = std::max(best, workspace_layout(*plan, G, batch, dtype).total);
  *bytes = best;
  return MAFAT_OK;
}

extern "C" const char* mafat_status_string(int status) {
  switch (status) {
    case MAFAT_OK: return "ok";
    case MAFAT_EINVAL: return "invalid argument";
    case MAFAT_ESHAPE: return "inconsistent shape, group or grid";
    case MAFAT_EUNSUPPORTED: return "unsupported layer or dtype";
    case MAFAT_EWORKSPACE: return "workspace too small";
    case MAFAT_EHIP: return "HIP runtime error";
    case MAFAT_ENOMEM: return "host allocation failed";
    default: return "unknown status";
  }
}

extern "C" const char* mafat_last_error(void) { return g_last_error.c_str(); }
