// tg_ew_forward_noalloc: the EW forward with its workspace in a scratch area
// that the library itself holds in device memory, for callers that cannot
// allocate (code under HIP graph capture, serving loops that must not call
// the allocator). The kernels and their order are those of tg_ew_forward;
// only the origin of the workspace differs.
//
// The scratch area is a file-scope device array. Each GPU the library runs
// on holds its own copy, at its own address, until the process ends; the
// host-side name `scratch` is only a stand-in, so host code uses the device
// address resolved once per device with hipGetSymbolAddress, never the name.
// Nothing in the forward's workspace has to start at zero when the call is
// made: every kernel writes what a later kernel reads, and what must be zero
// when a kernel starts (the grouped GEMMs' tile counters) is
// cleared by the forward's own dispatch kernels, so the host never clears
// the area.
#include <hip/hip_runtime.h>

#include <atomic>
#include <mutex>

#include "tg.h"
#include "tg_launch.h"

static __device__ __align__(256) unsigned char scratch[TG_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch[kMaxDevices];
std::mutex g_scratch_mu;

// Device address of the current device's scratch area, resolved on the
// first call on that device (with the device current) and kept.
tg_status scratch_on_current_device(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess)
    return tg::set_error(TG_ERR_HIP, "tg_ew_forward_noalloc: hipGetDevice: %s",
                         hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices)
    return tg::set_error(TG_ERR_UNSUPPORTED, "tg_ew_forward_noalloc: device %d beyond %d", dev,
                         kMaxDevices);
  void* p = g_scratch[dev].load(std::memory_order_acquire);
  if (!p) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    p = g_scratch[dev].load(std::memory_order_relaxed);
    if (!p) {
      e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
      if (e != hipSuccess || !p)
        return tg::set_error(TG_ERR_HIP, "tg_ew_forward_noalloc: hipGetSymbolAddress: %s",
                             hipGetErrorString(e));
      g_scratch[dev].store(p, std::memory_order_release);
    }
  }
  *out = p;
  return TG_OK;
}

}  // namespace

extern "C" tg_status tg_ew_forward_noalloc(const tg_ew_args* a, void* stream) {
  size_t need = 0;
  tg_status st = tg::ew_check(a, &need);
  if (st != TG_OK) return st;
  if (need > (size_t)TG_NOALLOC_SCRATCH_BYTES)
    return tg::set_error(TG_ERR_WORKSPACE,
                         "tg_ew_forward_noalloc: this batch needs %zu bytes of workspace; the "
                         "library's scratch area holds %zu (use tg_ew_forward with a caller "
                         "workspace, or pass y to keep the per-pair outputs outside it)",
                         need, (size_t)TG_NOALLOC_SCRATCH_BYTES);
  void* ws = nullptr;
  if ((st = scratch_on_current_device(&ws)) != TG_OK) return st;
  return tg::ew_forward(a, ws, (size_t)TG_NOALLOC_SCRATCH_BYTES, stream, nullptr);
}
