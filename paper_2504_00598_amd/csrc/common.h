// Device helpers shared by the libcfp kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cfp {

constexpr uint32_t kSat = 0xFFFFFFFFu;

// Unsigned add that clamps at 2^32-1 (v_add_u32 with the clamp bit).
__device__ __forceinline__ uint32_t sat_add(uint32_t a, uint32_t b) { return __builtin_elementwise_add_sat(a, b); }

__device__ __forceinline__ uint32_t umin(uint32_t a, uint32_t b) { return a < b ? a : b; }

// Minimum over the 64 lanes of a wave; every lane gets the result.
__device__ __forceinline__ uint32_t wave_min(uint32_t v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v = umin(v, (uint32_t)__shfl_xor((int)v, off, 64));
  return v;
}

template <int KP>
struct Pow2Bits {
  static constexpr int value = KP <= 16 ? 4 : KP <= 32 ? 5 : KP <= 64 ? 6 : KP <= 128 ? 7 : KP <= 256 ? 8 : 9;
};

}  // namespace cfp
