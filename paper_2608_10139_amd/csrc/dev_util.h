// Device-side helpers shared by the HIP kernel files: 16-bit float bit-pattern
// conversions (round to nearest even) for bf16 and fp16 activations.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace aiq {

// activation element types
enum Act : int { ACT_F32 = 0, ACT_BF16 = 1, ACT_F16 = 2 };

__device__ __forceinline__ uint16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}
__device__ __forceinline__ float bf2f(uint16_t b) { return __uint_as_float(static_cast<uint32_t>(b) << 16); }
__device__ __forceinline__ uint16_t f2h(float f) { return __builtin_bit_cast(uint16_t, static_cast<_Float16>(f)); }
__device__ __forceinline__ float h2f(uint16_t h) { return static_cast<float>(__builtin_bit_cast(_Float16, h)); }

// 16-bit activation of type `act` (ACT_BF16 or ACT_F16)
__device__ __forceinline__ uint16_t f2act(float f, int act) { return act == ACT_F16 ? f2h(f) : f2bf(f); }
__device__ __forceinline__ float act2f(uint16_t v, int act) { return act == ACT_F16 ? h2f(v) : bf2f(v); }

}  // namespace aiq
