// Device helpers shared by the libgist kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace gist {

constexpr int kXcds = 8;  // MI355X: 8 accelerator complex dies, one L2 each

// Workgroups are handed to the XCDs round-robin by linear id.  Remap the
// linear id so that XCD x works on one contiguous range of logical ids:
// neighbouring tiles / rows then share that XCD's L2.  Bijective for any
// grid size (XCD x receives q + (x < r) ids, q = G / 8, r = G % 8).
__device__ __forceinline__ int64_t xcd_remap(int64_t b, int64_t G) {
  const int64_t q = G / kXcds, r = G % kXcds;
  const int64_t x = b % kXcds, i = b / kXcds;
  return x * q + (x < r ? x : r) + i;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
inline bool aligned8(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 7u) == 0; }

}  // namespace gist
