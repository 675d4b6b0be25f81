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
constexpr int kResidual = 128;  // fp16 window of the captioning protocol (tokens), a power of two

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

// MXFP4 key window metadata (OCP microscaling format: one E8M0 power-of-two scale per block of 32
// values, FP4 E2M1 elements). Record of one window: bytes 4q..4q+1 hold the minimum's elements of
// channels 4q..4q+3 (4 bits each), bytes 4q+2..4q+3 the step's, byte 128 + 2b the minimum's scale
// byte of channel block b, byte 129 + 2b the step's.
constexpr int kMxRecord = 136;

// Key storage modes (template arguments of the key codec and of decode): fp16 window minimum and
// step, MXFP4 window records, or TurboQuant keys (Gaussian-codebook codes of the Hadamard direction,
// no window metadata; the paper's baseline, Eq. 2 and Eq. 3).
constexpr int kMetaFp16 = 0, kMetaMx = 1, kMetaTq = 2;

// Shared exponent of a block whose largest magnitude is amax: floor(log2(amax)) - 2 (2 is the
// largest E2M1 exponent), clamped to the E8M0 range; -127 for an all-zero block.
__device__ __forceinline__ int mx_exponent(float amax) {
  if (!(amax > 0.0f)) return -127;
  return min(max(ilogbf(amax) - 2, -127), 127);
}
// E2M1 code of t (a block value divided by 2^e, exactly): the nearest of 0, 0.5, 1, 1.5, 2, 3, 4,
// 6 with ties to the even code, saturating at 6; bit 3 is the sign (t < 0).
__device__ __forceinline__ uint32_t e2m1_encode(float t) {
  const float a = fabsf(t);
  const uint32_t c = (uint32_t)(a > 0.25f) + (uint32_t)(a >= 0.75f) + (uint32_t)(a > 1.25f) +
                     (uint32_t)(a >= 1.75f) + (uint32_t)(a > 2.5f) + (uint32_t)(a >= 3.5f) + (uint32_t)(a > 5.0f);
  return c | (t < 0.0f ? 8u : 0u);
}
// Value of E2M1 code c times 2^e (exact in fp32: two significant bits, exponent >= -128).
__device__ __forceinline__ float e2m1_decode(uint32_t c, int e) {
  const uint32_t E = (c >> 1) & 3u, M = c & 1u;
  const float v = ldexpf((float)(E ? 2u + M : M), (E ? (int)E : 1) - 2 + e);
  return (c & 8u) ? -v : v;
}

// Sequence lengths for the stateless codec calls travel as a kernel argument.
constexpr int kMaxLenArgs = 256;
struct LenArgs {
  int32_t lens[kMaxLenArgs];
};

}  // namespace okvq
