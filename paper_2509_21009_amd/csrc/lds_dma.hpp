// Global-to-LDS copies without register staging (gfx950 buffer_load ... lds)
// and explicit vector-memory wait counts, shared by the tiled GEMM and the
// prefill attention.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rollpack {

typedef uint32_t u32x4_raw __attribute__((ext_vector_type(4)));
// Buffer descriptor with the same fields as buffer_rsrc (base, stride 0, size, flags), as the
// four raw dwords an inline-assembly operand needs.
__device__ __forceinline__ u32x4_raw raw_rsrc(const void* p, uint32_t bytes) {
  const uint64_t addr = reinterpret_cast<uint64_t>(p);
  return u32x4_raw{static_cast<uint32_t>(addr), static_cast<uint32_t>(addr >> 32) & 0xffffu, bytes, 0x00020000u};
}
// 16 bytes per lane from byte voff of the buffer into LDS at lds + 16 * lane.  M0 holds the LDS base;
// it is named as clobbered, so the compiler keeps none of its own values there across the load.
__device__ __forceinline__ void dma16(u32x4_raw r, uint32_t lds, int voff) {
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds" : : "s"(lds), "v"(voff), "s"(r) : "memory", "m0");
}
// s_waitcnt vmcnt(N), the other counters at their maxima (gfx9 encoding).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

}  // namespace rollpack
