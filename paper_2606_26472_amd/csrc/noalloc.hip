// epikv_evict_step_noalloc: the eviction step with its device scratch in a
// file-scope array instead of caller workspace, for callers that cannot
// allocate (code under HIP graph capture, tight serving loops, harnesses
// that forbid allocation).
//
// The array `scratch` below exists once per GPU the library runs on (each
// device holds its own copy of a __device__ variable) and stays allocated
// until the process ends.  In host code its name is only a host-side
// stand-in: the device address comes from hipGetSymbolAddress, looked up
// once per device on the entry point's first call there, with that device
// current, and kept in `g_scratch`.  Only that address is ever handed to a
// kernel.  Every call on one GPU shares the array and it keeps the last
// call's contents; the step's kernels write every scratch word before they
// read it (the selection's histograms are cleared by a fill kernel at the
// start of each call).  Calls that overlap in time on one GPU (two
// streams, two threads) race on it.
#include <mutex>

#include "epikv_internal.h"

#define EPIKV_EXPORT extern "C" __attribute__((visibility("default")))

static_assert(EPIKV_NOALLOC_SCRATCH_BYTES % 256 == 0, "scratch size is whole 256-byte blocks");

static __device__ __align__(256) unsigned char scratch[EPIKV_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;

std::mutex g_mu;
void* g_scratch[kMaxDevices];  // device address of `scratch` per device, once looked up

// Address of this device's scratch array (the device current on the calling
// thread), looked up on the first call for that device.
int scratch_address(int dev, void** out) {
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || p == nullptr) return EPIKV_ELAUNCH;
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return EPIKV_OK;
}

}  // namespace

EPIKV_EXPORT int epikv_evict_step_noalloc(const epikv_cfg* cfg, const epikv_step_io* io,
                                          hipStream_t stream) {
  if (!io) return EPIKV_EINVAL_NULL;
  const int st = epikv_check_cfg(cfg);
  if (st) return st;
  if (io->chunk < 0) return EPIKV_EINVAL_SHAPE;
  const size_t need = epikv_workspace_bytes(cfg, io->chunk);
  if (need == 0 || need > EPIKV_NOALLOC_SCRATCH_BYTES) return EPIKV_EWORKSPACE;
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return EPIKV_ELAUNCH;
  if (dev >= kMaxDevices) return EPIKV_EINVAL_PARAM;
  // The kernels run on the stream's device; its scratch must be the one
  // looked up, which is the current device's.
  if (stream) {
    hipDevice_t sdev = -1;
    if (hipStreamGetDevice(stream, &sdev) != hipSuccess) return EPIKV_ELAUNCH;
    if (sdev != dev) return EPIKV_EINVAL_PARAM;
  }
  void* ptr = nullptr;
  const int sa = scratch_address(dev, &ptr);
  if (sa) return sa;
  epikv_step_io local = *io;
  local.workspace = ptr;
  local.workspace_bytes = EPIKV_NOALLOC_SCRATCH_BYTES;
  return epikv_evict_step(cfg, &local, stream);
}
