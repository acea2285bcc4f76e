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

// The static workspace of the stream's device: the current device, which the stream must belong
// to (the scratch address is per device).
sra_status static_workspace(void* stream, sra::StaticWorkspace* sw) {
  int device = -1;
  const hipError_t e = hipGetDevice(&device);
  if (e != hipSuccess) {
    const std::string msg = std::string("hipGetDevice: ") + hipGetErrorString(e);
    return sra::set_error(SRA_ERR_HIP, msg.c_str());
  }
  if (device < 0 || device >= kMaxDevices) return sra::set_error(SRA_ERR_UNSUPPORTED, "device index beyond 63");
  if (stream) {
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
  sw->bytes = SRA_NOALLOC_WORKSPACE_MAX;
  sw->device = device;
  return scratch_address(device, &sw->ptr);
}

}  // namespace

extern "C" sra_status sra_forward_noalloc(const sra_problem* p, const void* q_gen, const void* k_gen,
                                          const void* v_gen, const void* q_ref, const void* k_ref,
                                          const void* v_ref, void* o_gen, void* o_ref, float* lse_gen,
                                          float* lse_ref, void* stream) {
  // validation and the size check run on the host before any device call
  return sra::forward_call(p, q_gen, k_gen, v_gen, q_ref, k_ref, v_ref, o_gen, o_ref, lse_gen, lse_ref,
                           nullptr, 0, stream, static_workspace, SRA_NOALLOC_WORKSPACE_MAX);
}
