// Key codec on one wavefront: 64 consecutive tokens (two 32-token windows) of one
// (sequence, KV head). Sec. 2.1 Eq. 2 (norm split, randomized Hadamard) and Sec. 2.3 Eq. 4
// (per-window minimum and range of the rotated direction), 2-bit codes.
//
// Bit-exact operation order (per token row x, fp16):
//   norm   t_c = x_c^2; halving tree t <- t[:n/2] + t[n/2:] to one value; n16 = fp16(sqrt_rn(.))
//   dir    w = butterflies(s * x) for h = 1, 2, ..., 64; z = w * fl(kappa / n16) (z = 0 if n16 = 0)
//   window lo = min z + 0, hi = max z + 0 over the window's valid tokens;
//          step = fl(fl(hi - lo) / 3); m16 = fp16(lo), step16 = fp16(step)
//   code   0 if step16 == 0, else clamp(rint(fl(fl(z - m16) * fl(1 / step16))), 0, 3)
//
// Lane mapping: phase A (lane = token) keeps the 128 channels of a row in registers, so the
// norm tree and all seven butterfly stages run without cross-lane traffic. Phase B transposes
// z through a wave-private LDS tile, 64 channels at a time (lane = channel quad of half a
// window), for the window min / max. Phase C (lane = token) computes and packs the codes.
#pragma once

#include "okvq_device.hpp"

namespace okvq {

constexpr int kKeyPitch = 68;  // LDS row pitch (floats) of the 64-channel transpose tile: 16 lanes hit distinct banks
constexpr int kKeyWaveLds = 64 * kKeyPitch + 2 * kD * 2;  // floats per wave: tile + (m, 1/step) x 2 windows

struct KeyWaveOut {
  uint8_t* codes;  // [cap][32] of this (sequence, head)
  uint16_t* kmin;  // [cap/32][128] fp16 window metadata, or
  uint16_t* kstep; // [cap/32][128]
  uint8_t* kmx;    // [cap/32][136] MXFP4 window records
  uint16_t* knorm; // [cap]
  float tau0, tau1, tau2;  // TurboQuant keys: the codebook's decision thresholds (fp32, ascending)
};

// Lane l <- lane l ^ m for m = 1, 2 (DPP quad permutations) or 4 (LDS-pipe swizzle in xor mode):
// no address registers, unlike a general shuffle.
template <int kMask>
__device__ __forceinline__ float xor_lanes(float v) {
  const int x = __builtin_bit_cast(int, v);
  if constexpr (kMask == 1) return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(x, 0xB1, 0xf, 0xf, false));
  if constexpr (kMask == 2) return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(x, 0x4E, 0xf, 0xf, false));
  static_assert(kMask == 1 || kMask == 2 || kMask == 4, "xor of lane bit 0, 1 or 2");
  return __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(x, (kMask << 10) | 0x1f));
}

// Sign-flip masks for an fp16 pair (channels c, c+1) from the 32 sign words (4 int8 signs each).
__device__ __forceinline__ uint32_t sign_pair_mask(const uint32_t (&sw)[32], int c) {
  const uint32_t w = sw[c >> 2];
  return (c & 2) ? (((w & 0x00800000u) >> 8) | (w & 0x80000000u))
                 : (((w & 0x00000080u) << 8) | ((w & 0x00008000u) << 16));
}

// Phase A, first steps: sign flip and fp16 -> fp32 of the token row held by this lane. raw: the
// row's 128 fp16 channels as 64 dwords (channel 2i in the low half of raw[i]).
__device__ __forceinline__ void key_unpack(const uint32_t (&raw)[64], const uint32_t (&sw)[32], float (&x)[kD]) {
#pragma unroll
  for (int i = 0; i < 64; ++i) {
    const uint32_t r = raw[i] ^ sign_pair_mask(sw, 2 * i);
    x[2 * i] = h2f(r & 0xffffu);
    x[2 * i + 1] = h2f(r >> 16);
  }
}

// fp16 norm of the row: squares, then the halving tree t <- t[:n/2] + t[n/2:] (sign flips do not
// change the squares).
__device__ __forceinline__ uint32_t key_norm(const float (&x)[kD]) {
  float t[64];
#pragma unroll
  for (int c = 0; c < 64; ++c) t[c] = x[c] * x[c] + x[c + 64] * x[c + 64];
#pragma unroll
  for (int n = 32; n >= 1; n >>= 1) {
#pragma unroll
    for (int c = 0; c < n; ++c) t[c] = t[c] + t[c + n];
  }
  return norm_to_f16(sqrt_rn(t[0]));
}

// TurboQuant phase C (Eq. 3 on the key direction): code = #{k : z > tau_k} per channel (a value
// on a threshold takes the lower code), packed in the key byte layout; no window metadata.
__device__ __forceinline__ void key_codes_tq(const float (&x)[kD], uint32_t n16, int tok0, int len, const KeyWaveOut& out) {
  const int lane = lane_id(), tok = tok0 + lane;
  const bool valid = tok < len;
  const int store_slots = min(max(len - tok0 + 31, 0) / 32 * 32, 64);  // slots of valid windows
  if (lane >= store_slots) return;
  uint32_t dw[8];
#pragma unroll
  for (int u = 0; u < 8; ++u) {  // word u: channels 16u .. 16u + 15, even ones low, odd ones high
    uint32_t lo = 0, hi = 0;
#pragma unroll
    for (int jj = 0; jj < 8; ++jj) {
      const float z0 = x[16 * u + 2 * jj], z1 = x[16 * u + 2 * jj + 1];
      const uint32_t c0 = (uint32_t)(z0 > out.tau0) + (uint32_t)(z0 > out.tau1) + (uint32_t)(z0 > out.tau2);
      const uint32_t c1 = (uint32_t)(z1 > out.tau0) + (uint32_t)(z1 > out.tau1) + (uint32_t)(z1 > out.tau2);
      lo |= c0 << (2 * jj);
      hi |= c1 << (2 * jj);
    }
    dw[u] = valid ? (lo | (hi << 16)) : 0u;
  }
  uint4* dst = reinterpret_cast<uint4*>(out.codes + (size_t)tok * 32);
  dst[0] = make_uint4(dw[0], dw[1], dw[2], dw[3]);
  dst[1] = make_uint4(dw[4], dw[5], dw[6], dw[7]);
  out.knorm[tok] = valid ? (uint16_t)n16 : (uint16_t)0;
}

// Phase A, second half, and phases B and C for the 64 tokens [tok0, tok0 + 64) of one wave
// (lane = token). `len` is the sequence length; the slots of every window that holds a valid
// token are written (padded slots get code 0 and norm 0). between_bc() runs after phase B (the
// caller's loads for its next rows go out there, when fewer registers are live). kMeta: kMetaMx
// stores the window minimum and step as MXFP4 records and codes against their dequantized values;
// kMetaTq codes TurboQuant keys (no phase B).
template <int kMeta, typename F>
__device__ __forceinline__ void key_quantize_rows(float (&x)[kD], uint32_t n16, int tok0, int len, KeyWaveOut out,
                                                  float* lds, F&& between_bc) {
  constexpr bool kMx = kMeta == kMetaMx;
  const int lane = lane_id();
  const int tok = tok0 + lane;
  const bool valid = tok < len;
#pragma unroll
  for (int h = 1; h < kD; h <<= 1) {
#pragma unroll
    for (int j = 0; j < kD; ++j) {
      if ((j & h) == 0) {
        const float a = x[j], b = x[j + h];
        x[j] = a + b;
        x[j + h] = a - b;
      }
    }
  }
  // n16 == 0 only for an all-zero row (a nonzero fp16 element has a square >= 2^-48), whose
  // butterflies are all +-0: a zero factor gives z = +-0, which min/max (+0 canonicalization) and
  // the code formula treat exactly like z = 0.
  const float cinv = (n16 == 0) ? 0.0f : div_rn(kKappa, h2f(n16));
#pragma unroll
  for (int c = 0; c < kD; ++c) x[c] = x[c] * cinv;
  if constexpr (kMeta == kMetaTq) {
    between_bc();
    key_codes_tq(x, n16, tok0, len, out);
    return;
  }

  // ---- phase B: window min / max through LDS, 64 channels at a time. Lane l reads channel quad
  // l % 16 of rows 16 ((l / 16) % 2) .. +15 of window l / 32; the two row halves are combined with
  // lane l ^ 16. Rows beyond a partial window's length re-read its last valid row. ----
  float* tile = lds;                          // [64 tokens][kKeyPitch]
  float* stats = lds + 64 * kKeyPitch;        // [2 windows][128 channels] x (m32, inv32)
  const int qd = lane & 15, half = (lane >> 4) & 1, win = lane >> 5;
  const int nvalid = min(max(len - (tok0 + 32 * win), 0), 32);
  const bool full = __all(nvalid == 32);      // both windows complete: constant row offsets
  const int gwin = (tok0 >> 5) + win;
#pragma unroll
  for (int q = 0; q < 2; ++q) {
#pragma unroll
    for (int j = 0; j < 16; ++j)
      *reinterpret_cast<float4*>(&tile[lane * kKeyPitch + 4 * j]) =
          make_float4(x[64 * q + 4 * j], x[64 * q + 4 * j + 1], x[64 * q + 4 * j + 2], x[64 * q + 4 * j + 3]);
    wave_lds_sync();
    float lo[4], hi[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      lo[i] = __builtin_inff();
      hi[i] = -__builtin_inff();
    }
    const float* colp = tile + (32 * win + 16 * half) * kKeyPitch + 4 * qd;
    if (full) {
#pragma unroll
      for (int rr = 0; rr < 16; ++rr) {
        const float4 v = *reinterpret_cast<const float4*>(colp + rr * kKeyPitch);
        lo[0] = __builtin_fminf(lo[0], v.x); hi[0] = __builtin_fmaxf(hi[0], v.x);
        lo[1] = __builtin_fminf(lo[1], v.y); hi[1] = __builtin_fmaxf(hi[1], v.y);
        lo[2] = __builtin_fminf(lo[2], v.z); hi[2] = __builtin_fmaxf(hi[2], v.z);
        lo[3] = __builtin_fminf(lo[3], v.w); hi[3] = __builtin_fmaxf(hi[3], v.w);
      }
    } else {
      const float* rowbase = tile + 32 * win * kKeyPitch + 4 * qd;
      const int last = max(nvalid - 1, 0);
#pragma unroll
      for (int rr = 0; rr < 16; ++rr) {
        const int row = min(16 * half + rr, last);
        const float4 v = *reinterpret_cast<const float4*>(rowbase + row * kKeyPitch);
        lo[0] = __builtin_fminf(lo[0], v.x); hi[0] = __builtin_fmaxf(hi[0], v.x);
        lo[1] = __builtin_fminf(lo[1], v.y); hi[1] = __builtin_fmaxf(hi[1], v.y);
        lo[2] = __builtin_fminf(lo[2], v.z); hi[2] = __builtin_fmaxf(hi[2], v.z);
        lo[3] = __builtin_fminf(lo[3], v.w); hi[3] = __builtin_fmaxf(hi[3], v.w);
      }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      lo[i] = __builtin_fminf(lo[i], __shfl_xor(lo[i], 16));
      hi[i] = __builtin_fmaxf(hi[i], __shfl_xor(hi[i], 16));
    }
    if constexpr (kMx) {
      // MXFP4: a block of 32 channels is held by the 8 lanes l with equal l / 8 (channel quads
      // qd & 7), so the block maxima combine over lane bits 0..2
      // (lo, hi) become (minimum, step), then (dequantized minimum, 1 / dequantized step), in place
      float am = 0.0f, as = 0.0f;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        lo[i] = lo[i] + 0.0f;  // canonical +0
        hi[i] = div_rn((hi[i] + 0.0f) - lo[i], 3.0f);
        am = fmaxf(am, fabsf(lo[i]));
        as = fmaxf(as, hi[i]);
      }
      am = fmaxf(am, xor_lanes<1>(am));
      as = fmaxf(as, xor_lanes<1>(as));
      am = fmaxf(am, xor_lanes<2>(am));
      as = fmaxf(as, xor_lanes<2>(as));
      am = fmaxf(am, xor_lanes<4>(am));
      as = fmaxf(as, xor_lanes<4>(as));
      const int em = mx_exponent(am), es = mx_exponent(as);
      uint32_t word = 0;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const uint32_t cm = e2m1_encode(ldexpf(lo[i], -em)), cs = e2m1_encode(ldexpf(hi[i], -es));
        word |= (cm << (4 * i)) | (cs << (16 + 4 * i));
        const float sv = e2m1_decode(cs, es);
        lo[i] = e2m1_decode(cm, em);
        hi[i] = (sv == 0.0f) ? 0.0f : div_rn(1.0f, sv);
      }
      if (half == 0 && nvalid > 0) {
        // 32-bit record offsets, opaque so that their lane parts are not kept live (as 64-bit
        // values) across the tile loop
        uint32_t off = (uint32_t)gwin * kMxRecord + 4u * (16 * q + qd);
        __asm__ volatile("" : "+v"(off));
        *reinterpret_cast<uint32_t*>(out.kmx + off) = word;
        if ((qd & 7) == 0) {
          uint32_t soff = (uint32_t)gwin * kMxRecord + 128u + 2u * (2 * q + (qd >> 3));
          __asm__ volatile("" : "+v"(soff));
          *reinterpret_cast<uint16_t*>(out.kmx + soff) = (uint16_t)((em + 127) | ((es + 127) << 8));
        }
        float4* sp = reinterpret_cast<float4*>(stats + (win * kD + 64 * q + 4 * qd) * 2);
        sp[0] = make_float4(lo[0], hi[0], lo[1], hi[1]);
        sp[1] = make_float4(lo[2], hi[2], lo[3], hi[3]);
      }
    } else if (half == 0 && nvalid > 0) {
      uint32_t m16[4], s16[4];
      float st[8];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float l0 = lo[i] + 0.0f;  // canonical +0
        const float h0 = hi[i] + 0.0f;
        const float step = div_rn(h0 - l0, 3.0f);
        m16[i] = f2h(l0);
        s16[i] = f2h(step);
        st[2 * i] = h2f(m16[i]);
        st[2 * i + 1] = (s16[i] == 0) ? 0.0f : div_rn(1.0f, h2f(s16[i]));
      }
      int c = 64 * q + 4 * qd;
      __asm__ volatile("" : "+v"(c));  // keeps the lane's channel offset from living across the tile loop
      *reinterpret_cast<uint2*>(out.kmin + gwin * kD + c) = make_uint2(m16[0] | (m16[1] << 16), m16[2] | (m16[3] << 16));
      *reinterpret_cast<uint2*>(out.kstep + gwin * kD + c) = make_uint2(s16[0] | (s16[1] << 16), s16[2] | (s16[3] << 16));
      float4* sp = reinterpret_cast<float4*>(stats + (win * kD + c) * 2);
      sp[0] = make_float4(st[0], st[1], st[2], st[3]);
      sp[1] = make_float4(st[4], st[5], st[6], st[7]);
    }
    wave_lds_sync();
  }

  between_bc();

  // ---- phase C: codes (lane = token). t = fl(fl(z - m16) fl(1 / step16)) is clamped to [0, 3]
  // and rounded to an integer (ties to even) by adding 2^23, which leaves the code in the low bits
  // of the sum's bit pattern; eight such patterns shifted by 2j and OR-ed give the channels' 16
  // code bits in the low half (bits 24 and up only hold the shifted exponent) ----
  const int my_win = lane >> 5;
  const int store_slots = min(max(len - tok0 + 31, 0) / 32 * 32, 64);  // slots of valid windows
  if (lane < store_slots) {
    uint32_t dw[8];
#pragma unroll
    for (int d = 0; d < 8; ++d) dw[d] = 0;
    if (valid) {
      const float4* st = reinterpret_cast<const float4*>(stats + my_win * kD * 2);
      constexpr float kRound = 8388608.0f;  // 2^23
#pragma unroll
      for (int u = 0; u < 8; ++u) {  // word u: channels 16u .. 16u + 15, even ones low, odd ones high
        uint32_t lo = 0, hi = 0;
#pragma unroll
        for (int jj = 0; jj < 8; ++jj) {
          const int c = 16 * u + 2 * jj;
          const float4 s = st[c >> 1];
          const float t0 = (x[c] - s.x) * s.y;
          const float t1 = (x[c + 1] - s.z) * s.w;
          const uint32_t q0 = __builtin_bit_cast(uint32_t, __builtin_amdgcn_fmed3f(t0, 0.0f, 3.0f) + kRound);
          const uint32_t q1 = __builtin_bit_cast(uint32_t, __builtin_amdgcn_fmed3f(t1, 0.0f, 3.0f) + kRound);
          lo |= q0 << (2 * jj);
          hi |= q1 << (2 * jj);
        }
        dw[u] = __builtin_amdgcn_perm(hi, lo, 0x05040100u);  // low halves of lo and hi
      }
    }
    uint4* dst = reinterpret_cast<uint4*>(out.codes + (size_t)tok * 32);
    dst[0] = make_uint4(dw[0], dw[1], dw[2], dw[3]);
    dst[1] = make_uint4(dw[4], dw[5], dw[6], dw[7]);
    out.knorm[tok] = valid ? (uint16_t)n16 : (uint16_t)0;
  }
}

__device__ __forceinline__ void load_sign_words(const int8_t* signs, uint32_t (&sw)[32]) {
  const uint32_t* s = reinterpret_cast<const uint32_t*>(signs);
#pragma unroll
  for (int i = 0; i < 32; ++i) sw[i] = __builtin_amdgcn_readfirstlane(s[i]);
}

__device__ __forceinline__ void load_row_f16(const uint16_t* row, uint32_t (&raw)[64]) {
  const uint4* p = reinterpret_cast<const uint4*>(row);
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const uint4 v = p[i];
    raw[4 * i + 0] = v.x;
    raw[4 * i + 1] = v.y;
    raw[4 * i + 2] = v.z;
    raw[4 * i + 3] = v.w;
  }
}

}  // namespace okvq
