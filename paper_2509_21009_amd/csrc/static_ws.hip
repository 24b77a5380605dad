// The device array behind rp_generate_static.  In host code `scratch` names
// a host-side stand-in, not device memory: host code only ever uses the
// address hipGetSymbolAddress returns for the current device.
#include "static_ws.hpp"

static __device__ __align__(256) unsigned char scratch[rollpack::kStaticWorkspaceBytes];

namespace rollpack {

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_lock;
void* g_ptr[kMaxDevices] = {};
}  // namespace

std::mutex& static_workspace_lock() { return g_lock; }

hipError_t static_workspace(int device, void** ptr) {
  if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
  if (!g_ptr[device]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_ptr[device] = p;
  }
  *ptr = g_ptr[device];
  return hipSuccess;
}

}  // namespace rollpack
