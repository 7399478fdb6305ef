// predict.cpp -- memory prediction and configuration search (C ABI).
//
// mafat_predict_mem: two models of a plan's memory.
//   MAFAT_MEM_PAPER  the memory predictor of the paper (section 4.1,
//                    Algorithm 1): for every tile of every group and every
//                    layer of the group, with the tile's input and output
//                    extents at that layer ("Grid", here the plan's region
//                    tables, halo included),
//                      scratch = w_out * h_out * c_in * f^2 / s
//                      input   = w_in * h_in * c_in
//                      output  = w_out * h_out * c_out
//                      mem     = scratch + output + 2 * input
//                    and the prediction is the largest mem (in elements)
//                    times the element size.  The paper adds a platform
//                    constant (31 MB on its board) that the caller supplies.
//   MAFAT_MEM_DEVICE the device memory a run of this library needs: the
//                    caller-owned input, output and cut tensors, the
//                    parameters (weights in the run dtype, float32 scale and
//                    bias) and the workspace.  On the GPU every tile of a
//                    stage runs at once, so the working set is all tiles'
//                    intermediates (the workspace), not the largest tile's;
//                    with a tile batch K, K tiles' intermediates; with row
//                    reuse, the row bands of the stage outputs.
//   MAFAT_MEM_DEVICE_SEQ the same with one tile at a time (tile batch 1;
//                    row reuse as it is).
//
// mafat_get_config: the configuration search of the paper (section 4.2,
// Algorithm 2): cuts are tried in the given order (a cut >= n_layers means
// one group), for each cut the first-group grids t x t in the given order,
// the second group on a fixed grid; the first configuration whose predicted
// memory plus the bias is below the limit is returned, else the last one
// tried.  mafat_get_config_flags plans the candidates with plan flags (row
// reuse: the device models then give its row bands).
#include <algorithm>
#include <cmath>
#include <new>
#include <string>

#include "mafat_internal.h"

using namespace mafat;

namespace {

int64_t paper_group_max(const mafat_plan& P, const Group& G) {
  const int nl = G.l1 - G.l0 + 1;
  int64_t best = 0;
  for (int t = 0; t < G.ntiles; ++t)
    for (int k = 0; k < nl; ++k) {
      const int l = G.l0 + k;
      const mafat_layer& L = P.layers[l];
      const mafat_rect& in = G.in_r[static_cast<size_t>(t) * nl + k];
      const mafat_rect& out = G.out_r[static_cast<size_t>(t) * nl + k];
      const int64_t w_in = in.x1 - in.x0, h_in = in.y1 - in.y0;
      const int64_t w_out = out.x1 - out.x0, h_out = out.y1 - out.y0;
      const int64_t c_in = P.dims[l][2], c_out = P.dims[l][5];
      // scratch = w_out h_out c_in f^2 / s (exact: f^2 / s is 9, 1 or 2 here;
      // rounded down otherwise)
      const int64_t scratch = w_out * h_out * c_in * L.f * L.f / L.s;
      const int64_t input = w_in * h_in * c_in;
      const int64_t output = w_out * h_out * c_out;
      best = std::max(best, scratch + output + 2 * input);
    }
  return best;
}

int64_t device_bytes(const mafat_plan& P, int batch, int dtype, bool one_tile) {
  const int64_t esz = (dtype == MAFAT_F32) ? 4 : 2;
  const auto& d0 = P.dims.front();
  const auto& dn = P.dims.back();
  int64_t total = static_cast<int64_t>(batch) * d0[0] * d0[1] * d0[2] * esz;  // input
  total += static_cast<int64_t>(batch) * dn[3] * dn[4] * dn[5] * esz;         // output
  for (size_t g = 0; g + 1 < P.groups.size(); ++g) {                          // cut tensors
    const auto& d = P.dims[P.groups[g].l1];
    total += static_cast<int64_t>(batch) * d[3] * d[4] * d[5] * esz;
  }
  for (int l = 0; l < P.n; ++l) {  // parameters (packed weights where the plan packs them)
    const mafat_layer& L = P.layers[l];
    if (L.op != MAFAT_CONV) continue;
    const auto& d = P.dims[l];
    int bn, nblk, nchunk;
    const int64_t w = packed_layout(P, l, dtype, &bn, &nblk, &nchunk)
                          ? static_cast<int64_t>(nblk) * nchunk * 9 * bn * 32 * esz
                          : static_cast<int64_t>(d[5]) * L.f * L.f * d[2] * esz;
    total += w + 2 * 4 * static_cast<int64_t>(d[5]);
  }
  size_t ws = 0;
  if (!one_tile) {
    mafat_workspace_size(&P, batch, dtype, &ws);
  } else {  // the workspace of tile batch 1: one tile slot per scratch buffer
    for (const Group& G : P.groups) {
      if (G.reuse) {  // its tile rows run one after another already
        ws = std::max(ws, workspace_layout(P, G, batch, dtype).total);
        continue;
      }
      const int64_t frame = G.partition ? G.scratch_frame : static_cast<int64_t>(G.nbufs) * G.scratch_elems;
      ws = std::max(ws, (static_cast<size_t>(batch) * frame * esz + 255) & ~static_cast<size_t>(255));
    }
  }
  return total + static_cast<int64_t>(ws);
}

int predict(const mafat_plan* plan, int model, int batch, int dtype, int64_t* bytes) {
  if (model == MAFAT_MEM_PAPER) {
    int64_t best = 0;
    for (const Group& G : plan->groups) best = std::max(best, paper_group_max(*plan, G));
    *bytes = best * ((dtype == MAFAT_F32) ? 4 : 2);
    return MAFAT_OK;
  }
  *bytes = device_bytes(*plan, batch, dtype, model == MAFAT_MEM_DEVICE_SEQ);
  return MAFAT_OK;
}

}  // namespace

extern "C" int mafat_predict_mem(const mafat_plan* plan, int32_t model, int32_t batch, int32_t dtype,
                                 int64_t* bytes) {
  clear_error();
  if (!plan || !bytes || batch < 1) {
    set_error("plan and bytes must be non-NULL and batch >= 1");
    return MAFAT_EINVAL;
  }
  if (dtype != MAFAT_F32 && dtype != MAFAT_BF16) {
    set_error("dtype must be F32 or BF16");
    return MAFAT_EUNSUPPORTED;
  }
  if (model != MAFAT_MEM_PAPER && model != MAFAT_MEM_DEVICE && model != MAFAT_MEM_DEVICE_SEQ) {
    set_error("unknown memory model");
    return MAFAT_EINVAL;
  }
  return predict(plan, model, batch, dtype, bytes);
}

namespace {

// Algorithm 2 over the candidates; with `balanced` every candidate's groups
// take their balanced tile boundaries (mafat_balanced_bounds) instead of the
// even split.
int get_config(const mafat_layer* layers, int32_t n_layers, int32_t in_h, int32_t in_w, int32_t in_c,
               int32_t model, int32_t batch, int32_t dtype, int64_t bias_bytes, int64_t limit_bytes,
               const int32_t* cuts, int32_t n_cuts, const int32_t* grids, int32_t n_grids, int32_t second_grid,
               int32_t flags, bool balanced, int32_t* out_cut, int32_t* out_grid1, int32_t* out_grid2,
               int64_t* out_pred, int32_t* out_fits) {
  clear_error();
  if (!layers || !cuts || !grids || n_cuts < 1 || n_grids < 1 || second_grid < 1 || !out_cut || !out_grid1 ||
      !out_grid2) {
    set_error("null pointer, empty cut or grid list, or second grid < 1");
    return MAFAT_EINVAL;
  }
  int last_cut = -1, last_grid = -1;
  int64_t last_pred = 0;
  for (int ci = 0; ci < n_cuts; ++ci) {
    const int cut = cuts[ci];
    const bool split = cut > 0 && cut < n_layers;
    for (int gi = 0; gi < n_grids; ++gi) {
      const int t = grids[gi];
      const int32_t starts[2] = {0, cut};
      const int32_t rows[2] = {t, second_grid};
      mafat_plan* plan = nullptr;
      int rc = MAFAT_OK;
      if (balanced) {
        // boundaries of each group: rows, then columns (square grids)
        std::vector<int32_t> rb, cb;
        const int ng = split ? 2 : 1;
        for (int g = 0; g < ng && rc == MAFAT_OK; ++g) {
          const int g0 = starts[g], g1 = (g + 1 < ng ? starts[g + 1] : n_layers) - 1;
          std::vector<int32_t> r(static_cast<size_t>(rows[g]) + 1), c(static_cast<size_t>(rows[g]) + 1);
          rc = mafat_balanced_bounds(layers, n_layers, in_h, in_w, in_c, g0, g1, rows[g], rows[g], r.data(),
                                     c.data());
          rb.insert(rb.end(), r.begin(), r.end());
          cb.insert(cb.end(), c.begin(), c.end());
        }
        if (rc == MAFAT_OK)
          rc = mafat_plan_create_bounds(layers, n_layers, in_h, in_w, in_c, starts, ng, rows, rows, rb.data(),
                                        cb.data(), flags, &plan);
      } else {
        rc = mafat_plan_create_flags(layers, n_layers, in_h, in_w, in_c, starts, split ? 2 : 1, rows, rows, flags,
                                     &plan);
      }
      if (rc != MAFAT_OK) return rc;  // mafat_last_error() names the problem
      int64_t pred = 0;
      rc = mafat_predict_mem(plan, model, batch, dtype, &pred);
      mafat_plan_destroy(plan);
      if (rc != MAFAT_OK) return rc;
      last_cut = split ? cut : n_layers;
      last_grid = t;
      last_pred = pred;
      if (pred + bias_bytes < limit_bytes) {
        *out_cut = last_cut; *out_grid1 = t; *out_grid2 = split ? second_grid : 0;
        if (out_pred) *out_pred = pred + bias_bytes;
        if (out_fits) *out_fits = 1;
        return MAFAT_OK;
      }
    }
  }
  *out_cut = last_cut; *out_grid1 = last_grid;
  *out_grid2 = (last_cut < n_layers) ? second_grid : 0;
  if (out_pred) *out_pred = last_pred + bias_bytes;
  if (out_fits) *out_fits = 0;
  return MAFAT_OK;
}

}  // namespace

extern "C" int mafat_get_config(const mafat_layer* layers, int32_t n_layers, int32_t in_h, int32_t in_w,
                                int32_t in_c, int32_t model, int32_t batch, int32_t dtype, int64_t bias_bytes,
                                int64_t limit_bytes, const int32_t* cuts, int32_t n_cuts, const int32_t* grids,
                                int32_t n_grids, int32_t second_grid, int32_t* out_cut, int32_t* out_grid1,
                                int32_t* out_grid2, int64_t* out_pred, int32_t* out_fits) {
  return get_config(layers, n_layers, in_h, in_w, in_c, model, batch, dtype, bias_bytes, limit_bytes, cuts, n_cuts,
                    grids, n_grids, second_grid, 0, false, out_cut, out_grid1, out_grid2, out_pred, out_fits);
}

extern "C" int mafat_get_config_balanced(const mafat_layer* layers, int32_t n_layers, int32_t in_h,
                                         int32_t in_w, int32_t in_c, int32_t model, int32_t batch,
                                         int32_t dtype, int64_t bias_bytes, int64_t limit_bytes,
                                         const int32_t* cuts, int32_t n_cuts, const int32_t* grids,
                                         int32_t n_grids, int32_t second_grid, int32_t* out_cut,
                                         int32_t* out_grid1, int32_t* out_grid2, int64_t* out_pred,
                                         int32_t* out_fits) {
  try {
    return get_config(layers, n_layers, in_h, in_w, in_c, model, batch, dtype, bias_bytes, limit_bytes, cuts,
                      n_cuts, grids, n_grids, second_grid, 0, true, out_cut, out_grid1, out_grid2, out_pred,
                      out_fits);
  } catch (const std::bad_alloc&) {
    set_error("host allocation failed");
    return MAFAT_ENOMEM;
  }
}

extern "C" int mafat_get_config_flags(const mafat_layer* layers, int32_t n_layers, int32_t in_h, int32_t in_w,
                                      int32_t in_c, int32_t model, int32_t batch, int32_t dtype,
                                      int64_t bias_bytes, int64_t limit_bytes, const int32_t* cuts,
                                      int32_t n_cuts, const int32_t* grids, int32_t n_grids,
                                      int32_t second_grid, int32_t plan_flags, int32_t balanced,
                                      int32_t* out_cut, int32_t* out_grid1, int32_t* out_grid2,
                                      int64_t* out_pred, int32_t* out_fits) {
  try {
    return get_config(layers, n_layers, in_h, in_w, in_c, model, batch, dtype, bias_bytes, limit_bytes, cuts,
                      n_cuts, grids, n_grids, second_grid, plan_flags, balanced != 0, out_cut, out_grid1, out_grid2,
                      out_pred, out_fits);
  } catch (const std::bad_alloc&) {
    set_error("host allocation failed");
    return MAFAT_ENOMEM;
  }
}
