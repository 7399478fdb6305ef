// run.cpp -- C ABI execution entry points: validate the request, build the
// per-stage argument blocks from the plan and enqueue the stage kernels on
// the caller's stream.  No device allocation, no synchronisation.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>
#include <string>

#include "kernel_args.h"
#include "mafat_internal.h"

namespace mafat {
namespace {

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int fail(int status, const std::string& msg) {
  set_error(msg);
  return status;
}

// The matrix-core kernel needs whole 64-byte K chunks (32 bf16 or 16 fp32
// input channels) and output channels in multiples of 16.
bool mfma_ok(const Stage& S, int dtype) {
  const int kc = (dtype == MAFAT_BF16) ? 32 : 16;
  return S.kind == STAGE_CONV && S.cin % kc == 0 && S.cout % 16 == 0;
}

MfmaShape pick_shape(const Stage& S, int /*dtype*/) {
  (void)S;
  return MfmaShape{64, 64};
}

int run_group_impl(const mafat_plan* plan, int g, int batch, int dtype, const void* x, void* y,
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
  const int64_t scr_frame = static_cast<int64_t>(G.nbufs) * G.ntiles * G.scratch_elems;
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
      if (!aligned16(w[l])) return fail(MAFAT_EINVAL, "layer " + std::to_string(l) + ": weights not 16-byte aligned");
    }

  const int ns = static_cast<int>(G.stages.size());
  for (int s = 0; s < ns; ++s) {
    const Stage& S = G.stages[s];
    if (events && events[s] && hipEventRecord(static_cast<hipEvent_t>(events[s]), stream) != hipSuccess)
      return fail(MAFAT_EHIP, "hipEventRecord failed");
    const int kind = (S.kind == STAGE_POOL) ? K_POOL : (mfma_ok(S, dtype) ? K_CONV_MFMA : K_CONV_DIRECT);
    const MfmaShape shape = pick_shape(S, dtype);
    const int bu = block_units(kind, shape);
    StageArgs A;
    std::memset(&A, 0, sizeof(A));
    A.src = (S.src_buf == BUF_GROUP_IO) ? x : ws;
    A.dst = (S.dst_buf == BUF_GROUP_IO) ? y : ws;
    A.src_fstride = (S.src_buf == BUF_GROUP_IO) ? in_frame : scr_frame;
    A.dst_fstride = (S.dst_buf == BUF_GROUP_IO) ? out_frame : scr_frame;
    if (S.kind == STAGE_CONV) {
      A.w = w[S.first];
      A.scale = scale[S.first];
      A.bias = bias[S.first];
    }
    A.in_h = S.in_h; A.in_w = S.in_w;
    A.cin = S.cin; A.cout = S.cout;
    A.act = S.act;
    A.nblk_n = (kind == K_CONV_MFMA) ? (S.cout + shape.bn - 1) / shape.bn : 1;
    for (int t0 = 0; t0 < G.ntiles; t0 += kMaxTilesPerLaunch) {
      const int t1 = std::min(G.ntiles, t0 + kMaxTilesPerLaunch);
      A.ntiles = t1 - t0;
      int64_t total = 0;
      A.mblk_prefix[0] = 0;
      for (int t = t0; t < t1; ++t) {
        const TileGeom& T = S.tiles[t];
        KTile& k = A.tiles[t - t0];
        k.cy0 = static_cast<int16_t>(T.cy0); k.cx0 = static_cast<int16_t>(T.cx0);
        k.ch = static_cast<int16_t>(T.ch);   k.cw = static_cast<int16_t>(T.cw);
        k.sy0 = static_cast<int16_t>(T.sy0); k.sx0 = static_cast<int16_t>(T.sx0);
        k.sw = static_cast<int16_t>(T.sw);
        k.dy0 = static_cast<int16_t>(T.dy0); k.dx0 = static_cast<int16_t>(T.dx0);
        k.dw = static_cast<int16_t>(T.dw);
        k.src_off = static_cast<int32_t>(T.src_off);
        k.dst_off = static_cast<int32_t>(T.dst_off);
        int64_t units = static_cast<int64_t>(T.ch) * T.cw;
        if (kind == K_CONV_DIRECT && S.pool) units /= 4;
        total += (units + bu - 1) / bu;
        A.mblk_prefix[t - t0 + 1] = static_cast<int32_t>(total);
      }
      A.mblk_total = static_cast<int32_t>(total);
      const int64_t blocks = total * A.nblk_n * batch;
      if (blocks >= (1ll << 31)) return fail(MAFAT_EUNSUPPORTED, "grid too large");
      A.total_blocks = static_cast<int32_t>(blocks);
      const hipError_t e = launch_stage(kind, dtype, S.f, S.pool, shape, A, stream);
      if (e != hipSuccess)
        return fail(MAFAT_EHIP, std::string("stage launch failed: ") + hipGetErrorString(e));
    }
  }
  if (events && events[ns] && hipEventRecord(static_cast<hipEvent_t>(events[ns]), stream) != hipSuccess)
    return fail(MAFAT_EHIP, "hipEventRecord failed");
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

extern "C" int mafat_run_group(const mafat_plan* plan, int32_t group, int32_t batch, int32_t dtype,
                               const void* x, void* y, const void* const* w,
                               const float* const* scale, const float* const* bias,
                               void* workspace, size_t ws_bytes, void* stream,
                               void* const* events) {
  clear_error();
  int rc = check_common(plan, batch, dtype);
  if (rc != MAFAT_OK) return rc;
  if (group < 0 || group >= static_cast<int>(plan->groups.size()))
    return fail(MAFAT_EINVAL, "group index out of range");
  return run_group_impl(plan, group, batch, dtype, x, y, w, scale, bias, workspace, ws_bytes,
                        static_cast<hipStream_t>(stream), events);
}

extern "C" int mafat_run_network(const mafat_plan* plan, int32_t batch, int32_t dtype,
                                 const void* x, void* y, void* const* cut_bufs,
                                 const void* const* w, const float* const* scale,
                                 const float* const* bias, void* workspace, size_t ws_bytes,
                                 void* stream) {
  clear_error();
  int rc = check_common(plan, batch, dtype);
  if (rc != MAFAT_OK) return rc;
  const int ng = static_cast<int>(plan->groups.size());
  if (ng > 1 && !cut_bufs) return fail(MAFAT_EINVAL, "cut_bufs is NULL but the plan has several groups");
  for (int g = 0; g < ng; ++g) {
    const void* gin = (g == 0) ? x : cut_bufs[g - 1];
    void* gout = (g == ng - 1) ? y : cut_bufs[g];
    rc = run_group_impl(plan, g, batch, dtype, gin, gout, w, scale, bias, workspace, ws_bytes,
                        static_cast<hipStream_t>(stream), nullptr);
    if (rc != MAFAT_OK) return rc;
  }
  return MAFAT_OK;
}
