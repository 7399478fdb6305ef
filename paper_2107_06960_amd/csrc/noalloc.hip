// noalloc.hip -- mafat_run_network for callers that cannot allocate device
// memory: the workspace (the tiles' intermediate activations between stages)
// is a file-scope device array of fixed size instead of a caller buffer.
//
// The array is a __device__ symbol: in host code its name stands for a host
// shadow, not a device address, so its device address is looked up once per
// GPU with hipGetSymbolAddress (the current device at the first call on it)
// and only that address is handed to the kernels.  Every GPU holds its own
// copy of the array from the moment the library's code object is loaded on it
// until the process ends.
//
// No stage reads a workspace element before the same run wrote it (each stage
// writes its tiles' outputs before the next stage reads them, on one stream),
// so the array needs no clearing between calls.  Calls that overlap in time on
// one GPU (several streams, several threads) share the array and race.
#include <hip/hip_runtime.h>

#include <mutex>
#include <string>

#include "mafat_internal.h"

namespace mafat {
namespace {

constexpr size_t kStaticWorkspaceBytes = size_t{MAFAT_STATIC_WORKSPACE_MIB} << 20;
constexpr int kMaxDevices = 64;

__device__ __align__(256) unsigned char scratch[kStaticWorkspaceBytes];

std::mutex g_mu;
void* g_scratch_ptr[kMaxDevices] = {};

int fail(int status, const std::string& msg) {
  set_error(msg);
  return status;
}

}  // namespace
}  // namespace mafat

using namespace mafat;

extern "C" int mafat_run_network_static(const mafat_plan* plan, int32_t batch, int32_t dtype, const void* x,
                                        void* y, void* const* cut_bufs, const void* const* w,
                                        const float* const* scale, const float* const* bias, void* stream) {
  clear_error();
  if (!plan) return fail(MAFAT_EINVAL, "plan is NULL");
  size_t need = 0;
  const int rc = mafat_workspace_size(plan, batch, dtype, &need);
  if (rc != MAFAT_OK) return fail(rc, "batch must be >= 1 and dtype F32 or BF16");
  if (need > kStaticWorkspaceBytes)
    return fail(MAFAT_EWORKSPACE, "the plan needs " + std::to_string(need) + " bytes of workspace for batch " +
                                      std::to_string(batch) + "; the static workspace holds " +
                                      std::to_string(kStaticWorkspaceBytes) +
                                      " (use mafat_run_network with a caller buffer)");
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices)
    return fail(MAFAT_EHIP, "no current HIP device (or device index >= 64)");
  if (stream) {
    int sdev = -1;
    if (hipStreamGetDevice(static_cast<hipStream_t>(stream), &sdev) != hipSuccess)
      return fail(MAFAT_EHIP, "hipStreamGetDevice failed");
    if (sdev != dev)
      return fail(MAFAT_EINVAL, "the stream belongs to device " + std::to_string(sdev) + " but device " +
                                    std::to_string(dev) + " is current");
  }
  void* ws = nullptr;
  {
    std::lock_guard<std::mutex> lock(g_mu);
    if (!g_scratch_ptr[dev]) {
      void* p = nullptr;
      const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
      if (e != hipSuccess || !p)
        return fail(MAFAT_EHIP, std::string("hipGetSymbolAddress of the static workspace failed: ") +
                                    hipGetErrorString(e));
      g_scratch_ptr[dev] = p;
    }
    ws = g_scratch_ptr[dev];
  }
  return run_network_impl(plan, batch, dtype, x, y, cut_bufs, w, scale, bias, ws, kStaticWorkspaceBytes, stream);
}
