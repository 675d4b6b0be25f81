// Device-side helpers shared by the okvq HIP kernels (gfx950, wave64).
//
// Floating-point discipline (the codec kernels are bit-exact against a documented fp32 order):
// the library is compiled with -ffp-contract=off, IEEE denormals, and the correctly rounded
// fp32 division and square root of the device library; fp32 -> fp16 conversions round to
// nearest even.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace okvq {

constexpr int kD = 128;      // head dimension
constexpr int kW = 32;       // key window (tokens per min/step group)
constexpr int kWave = 64;    // CDNA wavefront size

// fp32(1/sqrt(128)), the normalization of the Sylvester Hadamard matrix of order 128.
constexpr float kKappa = 0x1.6a09e6p-4f;

__device__ __forceinline__ float h2f(uint32_t bits) {
  return (float)__builtin_bit_cast(_Float16, (uint16_t)bits);
}
__device__ __forceinline__ uint32_t f2h(float x) {  // round to nearest even
  return (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)x);
}
// Correctly rounded with -fhip-fp32-correctly-rounded-divide-sqrt (set by the build).
__device__ __forceinline__ float sqrt_rn(float x) { return __builtin_sqrtf(x); }
__device__ __forceinline__ float div_rn(float a, float b) { return a / b; }

// fp32 norm -> fp16, round to nearest even, saturating at 65504 instead of overflowing.
__device__ __forceinline__ uint32_t norm_to_f16(float n32) { return f2h(fminf(n32, 65504.0f)); }

// Orders LDS traffic between the lanes of one wavefront (each wave owns its LDS region).
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
}

__device__ __forceinline__ int lane_id() { return (int)__lane_id(); }

// Sequence lengths for the stateless codec calls travel as a kernel argument.
constexpr int kMaxLenArgs = 256;
struct LenArgs {
  int32_t lens[kMaxLenArgs];
};

}  // namespace okvq
