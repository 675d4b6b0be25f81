// Key directions with a token spread over the 16 lanes of a DPP row: lane j holds channels 8j ..
// 8j + 7. The norm, the butterflies and the scaling run in the key codec's bit-exact order (the
// halving tree, stages h = 1 .. 64, z = w fl(kappa / n16)); the levels and stages that pair a
// channel with one 8 or more apart cross lanes by DPP. Used by the window-parallel append; the
// bit-width ladder's key codec (four lanes per token) uses its DPP exchanges.
#pragma once

#include "key_quant.hpp"

namespace okvq {

// lane l <- lane l ^ m inside the 16-lane rows, all by DPP (no LDS-pipe shuffle): m = 1, 2 by quad
// permutations, m = 8 by a row rotation by 8, m = 4 by rotations by 12 (lanes 0-3, 8-11 take lane
// + 4) and by 4 (lanes 4-7, 12-15 take lane - 4) restricted to those banks
template <int kMask>
__device__ __forceinline__ float xchg(float v) {
  static_assert(kMask == 1 || kMask == 2 || kMask == 4 || kMask == 8, "lane mask within a row");
  const int x = __builtin_bit_cast(int, v);
  if constexpr (kMask == 1) return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, x, 0xB1, 0xf, 0xf, true));
  if constexpr (kMask == 2) return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, x, 0x4E, 0xf, 0xf, true));
  if constexpr (kMask == 8) return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, x, 0x128, 0xf, 0xf, true));
  if constexpr (kMask == 4) {
    const int up = __builtin_amdgcn_update_dpp(0, x, 0x12C, 0xf, 0x5, true);  // row_ror:12 into banks 0, 2
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(up, x, 0x124, 0xf, 0xA, true));  // row_ror:4, banks 1, 3
  }
}

__device__ __forceinline__ uint32_t xchg_u(uint32_t v) {  // lane l ^ 1
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xf, 0xf, true);
}

// fp16 norm of the token held by a 16-lane group (lane j: channels 8j .. 8j + 7) by the halving
// tree t <- t[:n/2] + t[n/2:]: the levels 64, 32, 16, 8 pair lane j with lane j ^ 8, 4, 2, 1 (both
// lanes of a pair form the same sum), the levels 4, 2, 1 stay in the lane. Squares of fp16 values
// are exact. Every lane of the group ends with the norm.
__device__ __forceinline__ uint32_t group_norm(const float (&x)[8]) {
  float t[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const float p = xchg<8>(x[e]);
    t[e] = x[e] * x[e] + p * p;
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) t[e] = t[e] + xchg<4>(t[e]);
#pragma unroll
  for (int e = 0; e < 8; ++e) t[e] = t[e] + xchg<2>(t[e]);
#pragma unroll
  for (int e = 0; e < 8; ++e) t[e] = t[e] + xchg<1>(t[e]);
#pragma unroll
  for (int n = 4; n >= 1; n >>= 1) {
#pragma unroll
    for (int e = 0; e < n; ++e) t[e] = t[e] + t[e + n];
  }
  return norm_to_f16(sqrt_rn(t[0]));
}

// Butterfly stage across lanes j and j ^ m of a group: the lower lane takes a + b, the upper one
// a - b, both as fl(s own + partner) with s = +-1 (an exact product, one rounding).
template <int kMask>
__device__ __forceinline__ void cross_stage(float (&x)[8], int j) {
  const float s = (j & kMask) ? -1.0f : 1.0f;
#pragma unroll
  for (int e = 0; e < 8; ++e) x[e] = __builtin_fmaf(s, x[e], xchg<kMask>(x[e]));
}

// The direction of a token's 8 channels in lane j of its group: the raw fp16 chunk with its int8
// signs applied (the sign bits flipped), the group's fp16 norm (returned), the local butterflies
// h = 1, 2, 4, the cross-lane stages h = 8 .. 64, then z = w fl(kappa / n16) (0 for a zero norm).
__device__ __forceinline__ uint32_t lane_direction(uint4 kraw, uint2 sg, int j, float (&x)[8]) {
  const uint32_t r4[4] = {kraw.x, kraw.y, kraw.z, kraw.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t w = (i < 2) ? sg.x : sg.y;  // int8 signs of channels 8j + 4 (i / 2) .. + 3
    const uint32_t m = (i & 1) ? (((w & 0x00800000u) >> 8) | (w & 0x80000000u))
                               : (((w & 0x00000080u) << 8) | ((w & 0x00008000u) << 16));
    const uint32_t r = r4[i] ^ m;
    x[2 * i] = h2f(r & 0xffffu);
    x[2 * i + 1] = h2f(r >> 16);
  }
  const uint32_t n16 = group_norm(x);
#pragma unroll
  for (int hh = 1; hh < 8; hh <<= 1) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      if ((e & hh) == 0) {
        const float p = x[e], q = x[e + hh];
        x[e] = p + q;
        x[e + hh] = p - q;
      }
    }
  }
  cross_stage<1>(x, j);  // h = 8
  cross_stage<2>(x, j);  // h = 16
  cross_stage<4>(x, j);  // h = 32
  cross_stage<8>(x, j);  // h = 64
  const float cinv = (n16 == 0) ? 0.0f : div_rn(kKappa, h2f(n16));
#pragma unroll
  for (int e = 0; e < 8; ++e) x[e] = x[e] * cinv;
  return n16;
}

}  // namespace okvq
