// Per-class override table of the reference step kernels (greedy.hip,
// beam.hip) in dynamic LDS: the target state of every class overridden in the
// state being scored (int32 per class), then one bit per class marking the
// classes set for that state (cleared per state). At most 135 KB (V = 32767).
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

namespace tbias {

__host__ __device__ inline size_t ref_table_bytes(int32_t V) {
  return 4 * (size_t)V + 4 * (size_t)((V + 31) / 32);
}

__device__ __forceinline__ bool ref_marked(const uint32_t* mark, int32_t c) {
  return (mark[c >> 5] >> (c & 31)) & 1u;
}

// Lets a kernel launch with more than 64 KB of dynamic LDS (the CU holds
// 160 KB). A failure shows in the launch's own error.
template <class F>
inline void allow_dynamic_lds(F* kernel, size_t bytes) {
  if (bytes > 65536)
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(kernel),
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
}

}  // namespace tbias
