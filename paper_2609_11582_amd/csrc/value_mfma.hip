// Value rotate-and-quantize on the matrix cores (Sec. 2.3, Eq. 6).
//
// y = R_m v for a tile of tokens is a dense [tokens x 128] x [128 x 128] contraction, run as
// v_mfma_f32_16x16x32_f16 with A = v (exact in fp16) and B = R_m^T split into fp16 hi + lo
// (R = hi + lo to about 2^-22 relative), both products accumulated in the same fp32 registers.
//
// Block: 256 threads = 4 waves, 256 tokens of one (sequence, KV head); wave w owns tokens
// [64 w, 64 w + 64) of the tile as four 16-row blocks. R_m is staged in LDS (hi and lo, row
// pitch 136 halves so that the 16 lanes of a quarter-wave read distinct banks) one modality at a
// time, for the modalities present in the tile. For each pair of 16-column output blocks a wave
// reads the B operands once (2 x 4 k-blocks x hi/lo) and runs them against every one of its row
// blocks that holds the modality, so LDS operand traffic is shared by up to four row blocks;
// rows of other modalities in a mixed row block are computed but masked.
//
// Decision: the thresholds are symmetric (-T, 0, T with T = fl(n16 tau_2)), so the code is
// clamp(floor(y fl(1/T)) + 2, 0, 3). Its boundaries sit within 2^-22 T of the exact comparisons,
// far inside the 2^-16 sum_j |R_cj v_j| band that separates MFMA mode from the sequential order;
// zero-norm and other-modality tokens are cleared per byte.
//
// MFMA 16x16x32 f16 lane mapping (wave64): lane l holds A[l % 16][8 (l / 16) + e], e = 0..7,
// B[8 (l / 16) + e][l % 16], and D[4 (l / 16) + i][l % 16], i = 0..3. With rows = tokens and
// columns = output channels, lane l ends with channel 16 nb + l % 16 of four consecutive tokens:
// exactly one byte of the value-code layout, and the lane's eight bytes of a 16-token row block
// are contiguous (offset 16 l + 8 (rb & 1) in the window block).
#include "launch.hpp"
#include "value_quant.hpp"

namespace okvq {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int kRPitch = 136;                  // halves per staged row of R
constexpr int kRStage = kD * kRPitch;         // halves per staged matrix (hi or lo)

__device__ __forceinline__ half8 as_half8(uint4 u) { return __builtin_bit_cast(half8, u); }

// One code byte (four tokens of one channel): code = clamp(floor(y / T) + 2, 0, 3), 2 bits each.
__device__ __forceinline__ uint32_t value_byte(floatx4 y, const float (&it)[4]) {
  uint32_t byte = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int f = __builtin_amdgcn_fmed3f(__builtin_floorf(y[i] * it[i]), -2.0f, 1.0f);
    byte |= (uint32_t)(f + 2) << (2 * i);
  }
  return byte;
}

// R_m as fp16 hi + lo in the staging buffers; thread t converts rows n = t / 16 + 16 it, eight
// consecutive k per step
__device__ __forceinline__ void stage_rotation(const float* __restrict__ rot, int m, _Float16* rhi, _Float16* rlo) {
  const float4* src = reinterpret_cast<const float4*>(rot + (size_t)m * kD * kD);
  float4 f[kD * kD / 8 / 256][2];
#pragma unroll
  for (int it = 0; it < kD * kD / 8 / 256; ++it) {  // every load first
    const int idx = threadIdx.x + 256 * it;
    f[it][0] = src[2 * idx];
    f[it][1] = src[2 * idx + 1];
  }
#pragma unroll
  for (int it = 0; it < kD * kD / 8 / 256; ++it) {
    const int idx = threadIdx.x + 256 * it;
    const int n = idx >> 4, k8 = (idx & 15) * 8;
    const float fv[8] = {f[it][0].x, f[it][0].y, f[it][0].z, f[it][0].w, f[it][1].x, f[it][1].y, f[it][1].z, f[it][1].w};
    half8 hv, lv;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      hv[q] = (_Float16)fv[q];
      lv[q] = (_Float16)(fv[q] - (float)hv[q]);
    }
    *reinterpret_cast<half8*>(rhi + n * kRPitch + k8) = hv;
    *reinterpret_cast<half8*>(rlo + n * kRPitch + k8) = lv;
  }
}

struct ValueTile {  // token geometry of a work-group and wave from (begin, len)
  int begin, len, tile0, wtok0;
};

__device__ __forceinline__ ValueTile value_tile(int begin, int len, int wave) {
  ValueTile t;
  t.begin = begin;
  t.len = len;
  t.tile0 = (begin / kW) * kW + blockIdx.x * 256;  // tiles start at the first open window
  t.wtok0 = t.tile0 + wave * 64;
  return t;
}

// A operands (v rows, fp16, zero outside [begin, len)) and the modality of token wtok0 + lane
__device__ __forceinline__ void load_value_rows(const CodecJob& j, size_t seq, int b, const ValueTile& t, int lane,
                                                uint4 (&a)[4][4], int& mymod) {
  const int r = lane & 15, g = lane >> 4;
#pragma unroll
  for (int rb = 0; rb < 4; ++rb) {
    const int tok = t.wtok0 + 16 * rb + r;
    const bool fresh = tok >= t.begin && tok < t.len;
    const uint4* row = reinterpret_cast<const uint4*>(j.src + (seq * j.n_rows + (size_t)max(tok - t.begin, 0)) * kD);
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) a[rb][kk] = fresh ? row[4 * kk + g] : make_uint4(0, 0, 0, 0);
  }
  const int mytok = t.wtok0 + lane;
  mymod = (mytok >= t.begin && mytok < t.len) ? (int)j.msrc[(size_t)b * j.n_rows + (mytok - t.begin)] : -1;
}

__global__ __launch_bounds__(256, 2) void k_quantize_values_mfma(CodecJob j, const float* __restrict__ rot,
                                                                 Thresholds th, uint8_t* __restrict__ v_codes,
                                                                 uint16_t* __restrict__ v_norm,
                                                                 uint8_t* __restrict__ mod_out) {
  __shared__ __attribute__((aligned(16))) _Float16 rstage[2 * kRStage];  // [2][128][kRPitch]: hi, lo
  __shared__ __attribute__((aligned(16))) float nlds[4][64];              // per wave: token norms (fp16 values)
  __shared__ __attribute__((aligned(16))) int8_t mlds[4][64];             // per wave: token modalities
  __shared__ uint32_t present;

  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform for the compiler
  const int lane = lane_id();
  const int r = lane & 15, g = lane >> 4;
  const int h = blockIdx.y, bz = blockIdx.z, b = j.b0 + bz;
  const size_t seq = (size_t)b * j.H + h;

  // ---- row loads from the planned lengths, then the device lengths decide (append) ----
  ValueTile t = j.begin_dev ? value_tile(j.lens.lens[bz], j.lens.lens[bz] + j.cnts.lens[bz], wave)
                            : value_tile(0, j.lens.lens[bz], wave);
  uint4 a[4][4];  // [row block][k block]
  int mymod;
  load_value_rows(j, seq, b, t, lane, a, mymod);
  int bd = t.begin, ld = t.len;
  if (j.begin_dev) {
    bd = min(max(j.begin_dev[b], 0), j.cap);
    ld = min(bd + min(max(j.count_dev[b], 0), j.n_rows), j.cap);
  }
  _Float16* rhi = rstage;
  _Float16* rlo = rstage + kRStage;
  stage_rotation(rot, 1, rhi, rlo);  // video first, while the rows are in flight
  if (bd != t.begin || ld != t.len) {  // stale host lengths: reload from the device ones
    t = value_tile(bd, ld, wave);
    load_value_rows(j, seq, b, t, lane, a, mymod);
  }
  if (t.len <= t.begin || t.tile0 >= t.len) return;  // whole block idle: no barrier reached
  const int begin = t.begin, len = t.len, wtok0 = t.wtok0;
  const int wend = ((len + kW - 1) / kW) * kW;  // end of the last window

  if (threadIdx.x == 0) present = 0;
  if (mymod >= 0 && mod_out && h == 0) mod_out[(size_t)b * j.cap + wtok0 + lane] = (uint8_t)mymod;
  __syncthreads();
  uint32_t wave_present = 0;
#pragma unroll
  for (int m = 0; m < 3; ++m)
    if (__ballot(mymod == m)) wave_present |= 1u << m;
  if (lane == 0 && wave_present) atomicOr(&present, wave_present);

  // ---- norms by the halving tree; lane (r, g) holds channels 32 kk + 8 g + e of token r ----
#pragma unroll
  for (int rb = 0; rb < 4; ++rb) {
    float x[4][8];
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const half8 hv = as_half8(a[rb][kk]);
#pragma unroll
      for (int e = 0; e < 8; ++e) x[kk][e] = (float)hv[e];
    }
    float s[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      // level 64: c with c + 64 (kk with kk + 2); level 32: c with c + 32 (kk 0 with kk 1)
      const float l0 = x[0][e] * x[0][e] + x[2][e] * x[2][e];
      const float l1 = x[1][e] * x[1][e] + x[3][e] * x[3][e];
      s[e] = l0 + l1;
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) s[e] = s[e] + __shfl_xor(s[e], 32);  // level 16: g with g ^ 2
#pragma unroll
    for (int e = 0; e < 8; ++e)  // level 8: g with g ^ 1 (lane ^ 16, a swizzle within 32 lanes)
      s[e] = s[e] + __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, s[e]), 0x401f));
#pragma unroll
    for (int n = 4; n >= 1; n >>= 1) {
#pragma unroll
      for (int e = 0; e < n; ++e) s[e] = s[e] + s[e + n];
    }
    const int tok = wtok0 + 16 * rb + r;
    const bool fresh = tok >= begin && tok < len;
    const uint32_t n16 = fresh ? norm_to_f16(sqrt_rn(s[0])) : 0u;
    if (g == 0) {
      nlds[wave][16 * rb + r] = h2f(n16);
      if (tok >= begin && tok < wend) v_norm[seq * j.cap + tok] = (uint16_t)n16;
    }
  }
  mlds[wave][lane] = (int8_t)mymod;
  wave_lds_sync();
  // per lane: 1 / T and modalities of the four tokens 16 rb + 4 g + i of its output rows
  float itrow[4][4];
  int mrow[4][4];
#pragma unroll
  for (int rb = 0; rb < 4; ++rb) {
    const float4 n4 = *reinterpret_cast<const float4*>(&nlds[wave][16 * rb + 4 * g]);
    const uint32_t m4 = *reinterpret_cast<const uint32_t*>(&mlds[wave][16 * rb + 4 * g]);
    const float nv[4] = {n4.x, n4.y, n4.z, n4.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int mm = (int)(int8_t)((m4 >> (8 * i)) & 0xffu);
      itrow[rb][i] = (nv[i] > 0.0f) ? __builtin_amdgcn_rcpf(nv[i] * th.t2) : 0.0f;
      mrow[rb][i] = (nv[i] > 0.0f) ? mm : -1;  // zero norm: every code 0
    }
  }
  __syncthreads();
  const uint32_t pres = present;

  uint32_t bytes[4][2];  // [row block][nb / 4]: 8 code bytes per row block
#pragma unroll
  for (int rb = 0; rb < 4; ++rb) bytes[rb][0] = bytes[rb][1] = 0;

  for (int mi = 0; mi < 3; ++mi) {
    const int m = (mi == 0) ? 1 : (mi == 1 ? 0 : 2);  // video (staged above), audio, text
    if (!(pres & (1u << m))) continue;  // block-uniform
    if (mi > 0) {
      __syncthreads();  // previous modality's reads are done
      stage_rotation(rot, m, rhi, rlo);
      __syncthreads();
    }
    if (!(wave_present & (1u << m))) continue;  // wave-uniform
    uint32_t rbm = 0;  // the wave's row blocks holding modality m
#pragma unroll
    for (int rb = 0; rb < 4; ++rb)
      if (__ballot((mymod == m) && ((lane >> 4) == rb))) rbm |= 1u << rb;
    uint32_t keep[4];  // per row block: byte mask of the lane's four tokens of modality m
#pragma unroll
    for (int rb = 0; rb < 4; ++rb) {
      keep[rb] = 0;
#pragma unroll
      for (int i = 0; i < 4; ++i) keep[rb] |= (mrow[rb][i] == m ? 3u : 0u) << (2 * i);
      keep[rb] *= 0x01010101u;
    }
#pragma unroll
    for (int np = 0; np < 4; ++np) {  // output blocks nb = 2 np, 2 np + 1
      half8 bv[2][4][2];                // [nb][kk][hi, lo]
#pragma unroll
      for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int kk = 0; kk < 4; ++kk)
#pragma unroll
          for (int part = 0; part < 2; ++part)
            bv[u][kk][part] = *reinterpret_cast<const half8*>((part ? rlo : rhi) + (16 * (2 * np + u) + r) * kRPitch +
                                                              32 * kk + 8 * g);
      if (rbm == 0xfu) {  // every row block holds modality m: eight independent accumulators
        floatx4 acc[4][2];
#pragma unroll
        for (int rb = 0; rb < 4; ++rb) acc[rb][0] = acc[rb][1] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kk = 0; kk < 4; ++kk)
#pragma unroll
          for (int part = 0; part < 2; ++part)
#pragma unroll
            for (int rb = 0; rb < 4; ++rb)
#pragma unroll
              for (int u = 0; u < 2; ++u)
                acc[rb][u] =
                    __builtin_amdgcn_mfma_f32_16x16x32_f16(as_half8(a[rb][kk]), bv[u][kk][part], acc[rb][u], 0, 0, 0);
#pragma unroll
        for (int rb = 0; rb < 4; ++rb)
#pragma unroll
          for (int u = 0; u < 2; ++u) {
            const int nb = 2 * np + u;
            bytes[rb][nb >> 2] |= (value_byte(acc[rb][u], itrow[rb]) & keep[rb]) << (8 * (nb & 3));
          }
      } else {
#pragma unroll
        for (int rb = 0; rb < 4; ++rb) {
          if (!(rbm & (1u << rb))) continue;  // wave-uniform
          floatx4 acc[2] = {floatx4{0.f, 0.f, 0.f, 0.f}, floatx4{0.f, 0.f, 0.f, 0.f}};
#pragma unroll
          for (int kk = 0; kk < 4; ++kk) {
            const half8 av = as_half8(a[rb][kk]);
#pragma unroll
            for (int part = 0; part < 2; ++part)
#pragma unroll
              for (int u = 0; u < 2; ++u)
                acc[u] = __builtin_amdgcn_mfma_f32_16x16x32_f16(av, bv[u][kk][part], acc[u], 0, 0, 0);
          }
#pragma unroll
          for (int u = 0; u < 2; ++u) {
            const int nb = 2 * np + u;
            bytes[rb][nb >> 2] |= (value_byte(acc[u], itrow[rb]) & keep[rb]) << (8 * (nb & 3));
          }
        }
      }
    }
  }

  // ---- store: one 16-byte chunk per lane per window (row blocks 2w, 2w + 1) ----
#pragma unroll
  for (int w = 0; w < 2; ++w) {
    const int win_tok = wtok0 + 32 * w;
    if (win_tok < len) {
      const int gwin = win_tok / kW;
      uint4* dst = reinterpret_cast<uint4*>(v_codes + (seq * (j.cap / kW) + gwin) * 1024 + 16 * lane);
      uint4 val = make_uint4(bytes[2 * w][0], bytes[2 * w][1], bytes[2 * w + 1][0], bytes[2 * w + 1][1]);
      if (win_tok < begin) {  // the window holds older tokens: keep their code bits
        const int old0 = min(max(begin - (win_tok + 4 * g), 0), 4);       // tokens 4g .. 4g+3
        const int old1 = min(max(begin - (win_tok + 16 + 4 * g), 0), 4);  // tokens 16+4g ..
        const uint32_t k0 = ((1u << (2 * old0)) - 1u) * 0x01010101u;
        const uint32_t k1 = ((1u << (2 * old1)) - 1u) * 0x01010101u;
        const uint4 old = *dst;
        val.x = (old.x & k0) | (val.x & ~k0);
        val.y = (old.y & k0) | (val.y & ~k0);
        val.z = (old.z & k1) | (val.z & ~k1);
        val.w = (old.w & k1) | (val.w & ~k1);
      }
      *dst = val;
    }
  }
}

hipError_t launch_quantize_values_mfma(const CodecJob& j, int nb, int max_tiles_tokens, const float* rot,
                                       const Thresholds& th, uint8_t* v_codes, uint16_t* v_norm,
                                       uint8_t* mod_out, hipStream_t s) {
  dim3 grid((max_tiles_tokens + 255) / 256, j.H, nb);
  hipLaunchKernelGGL(k_quantize_values_mfma, grid, dim3(256), 0, s, j, rot, th, v_codes, v_norm, mod_out);
  return hipGetLastError();
}

}  // namespace okvq
