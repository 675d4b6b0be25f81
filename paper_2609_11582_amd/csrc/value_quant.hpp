// Value codec (Sec. 2.3 Eq. 6 with the fixed codebook of Eq. 3).
//
// For a token of modality m: y = R_m v (v fp16, R_m fp32), n16 = fp16(||v||) by the same halving
// tree as the keys, and per coordinate code = #{k : y_c > fl(n16 * tau_k)} against the three
// Lloyd-Max thresholds tau of N(0, 1/128) (comparing y with n16 * tau avoids dividing y by the
// norm; a value exactly on a threshold takes the lower code).
//
// Two ways to form y:
//  * exact mode -- acc = 0; acc = fl(acc + fl(R_cj * v_j)) for j = 0..127 (bit-exact order);
//  * MFMA mode  -- v (exact in fp16) times R_m split as fp16 hi + lo, fp32 accumulation on the
//                  matrix cores; differs from the exact order by far less than 2^-16 sum|R_cj v_j|.
//
// Output layout (one 1024-byte block per 32-token window): window token t, channel c live in byte
// 16 * ((c & 15) + 16 * ((t >> 2) & 3)) + 8 * (t >> 4) + (c >> 4), bits 2 (t & 3).
#pragma once

#include "okvq_device.hpp"

namespace okvq {

struct Thresholds {
  float t0, t1, t2;  // fp32 decision thresholds of the N(0, 1/128) codebook, ascending
};

__device__ __forceinline__ uint32_t value_code(float y, float n16f, const Thresholds& th) {
  const float a = n16f * th.t0, b = n16f * th.t1, c = n16f * th.t2;
  return (uint32_t)(y > a) + (uint32_t)(y > b) + (uint32_t)(y > c);
}

__device__ __forceinline__ int value_byte_index(int t, int c) {
  return 16 * ((c & 15) + 16 * ((t >> 2) & 3)) + 8 * (t >> 4) + (c >> 4);
}

}  // namespace okvq
