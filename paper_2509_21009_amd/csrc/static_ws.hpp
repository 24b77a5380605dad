// Library-owned device workspace of rp_generate_static, the entry point for
// callers that cannot allocate: one file-scope device array, which every GPU
// the library runs on holds until the process ends.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <mutex>

namespace rollpack {

// Size of the array: KV pool and scratch workspace of one call together.
constexpr size_t kStaticWorkspaceBytes = size_t{64} << 20;

// Serialises the calls that use the array within this process.
std::mutex& static_workspace_lock();

// Device address of the array on `device`, which must be the current device.
// The address is looked up once per device (hipGetSymbolAddress) and kept;
// the caller holds static_workspace_lock().
hipError_t static_workspace(int device, void** ptr);

}  // namespace rollpack
