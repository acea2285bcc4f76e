// sra_forward_noalloc: the SRA forward with its workspace in a static device array, for callers
// that cannot allocate device memory. Same kernels and results as sra_forward.
#include <hip/hip_runtime.h>

#include <mutex>
#include <string>

#include "sra.h"
#include "sra_internal.h"

namespace {

// The workspace of every sra_forward_noalloc call on a device: the schedule tables (and, for
// plans on the compacted reference stream, the compacted tensors when they fit). One copy per
// device, held until the process ends. In host code `scratch` names a host-side stand-in, not
// device memory: only the address hipGetSymbolAddress returns for the current device is used.
static __device__ __align__(256) unsigned char scratch[SRA_NOALLOC_WORKSPACE_MAX];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of `scratch` on `device` (the current device), looked up once per device.
sra_status scratch_address(int device, void** out) {
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_scratch_ptr[device]) {
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr) {
      const std::string msg = std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e);
      return sra::set_error(SRA_ERR_HIP, msg.c_str());
    }
    g_scratch_ptr[device] = ptr;
  }
  *out = g_scratch_ptr[device];
  return SRA_OK;
}

}  // namespace

extern "C" sra_status sra_forward_noalloc(const sra_problem* p, const void* q_gen, const void* k_gen,
                                          const void* v_gen, const void* q_ref, const void* k_ref,
                                          const void* v_ref, void* o_gen, void* o_ref, float* lse_gen,
                                          float* lse_ref, void* stream) {
  // the size check runs on the host before any device call
  size_t need = 0;
  sra_status st = sra_workspace_size(p, 0, &need);
  if (st != SRA_OK) return st;
  if (need > SRA_NOALLOC_WORKSPACE_MAX) {
    const std::string msg = "forward needs " + std::to_string(need) +
                            " workspace bytes, more than the static scratch maximum of " +
                            std::to_string(size_t(SRA_NOALLOC_WORKSPACE_MAX)) + " (use sra_forward)";
    return sra::set_error(SRA_ERR_WORKSPACE_TOO_SMALL, msg.c_str());
  }
  int device = -1;
  const hipError_t e = hipGetDevice(&device);
  if (e != hipSuccess) {
    const std::string msg = std::string("hipGetDevice: ") + hipGetErrorString(e);
    return sra::set_error(SRA_ERR_HIP, msg.c_str());
  }
  if (device < 0 || device >= kMaxDevices) return sra::set_error(SRA_ERR_UNSUPPORTED, "device index beyond 63");
  if (stream) {  // the scratch address is per device: the stream must be the current device's
    int sdev = -1;
    const hipError_t es = hipStreamGetDevice(static_cast<hipStream_t>(stream), &sdev);
    if (es != hipSuccess) {
      const std::string msg = std::string("hipStreamGetDevice: ") + hipGetErrorString(es);
      return sra::set_error(SRA_ERR_HIP, msg.c_str());
    }
    if (sdev != device) {
      const std::string msg = "stream belongs to device " + std::to_string(sdev) + ", the current device is " +
                              std::to_string(device);
      return sra::set_error(SRA_ERR_INVALID_ARGUMENT, msg.c_str());
    }
  }
  sra::StaticWorkspace sw{nullptr, size_t(SRA_NOALLOC_WORKSPACE_MAX), device};
  st = scratch_address(device, &sw.ptr);
  if (st != SRA_OK) return st;
  return sra::forward_call(p, q_gen, k_gen, v_gen, q_ref, k_ref, v_ref, o_gen, o_ref, lse_gen, lse_ref,
                           nullptr, 0, stream, &sw);
}
