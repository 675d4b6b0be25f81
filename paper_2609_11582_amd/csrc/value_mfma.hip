// Value rotate-and-quantize on the matrix cores (Sec. 2.3, Eq. 6).
//
// y = R_m v for a tile of tokens is a dense [tokens x 128] x [128 x 128] contraction, run as
// v_mfma_f32_16x16x32_f16 with A = v (exact in fp16) and B = R_m^T split into fp16 hi + lo
// (R = hi + lo to about 2^-22 relative), both products accumulated in the same fp32 registers.
//
// Block: 256 threads = 4 waves, 256 tokens of one (sequence, KV head); wave w owns tokens
// [64 w, 64 w + 64) of the tile as four 16-row blocks. R_m is staged in LDS (hi and lo, row
// pitch 136 halves so that the 16 lanes of a quarter-wave read distinct banks) one modality at a
// time, for the modalities present in the tile; rows of other modalities are computed but masked.
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

__device__ __forceinline__ void job_range_v(const CodecJob& j, int bz, int b, int& begin, int& len) {
  if (j.begin_dev) {
    begin = j.begin_dev[b];
    len = begin + j.count_dev[b];
  } else {
    begin = 0;
    len = j.lens.lens[bz];
  }
}

__global__ __launch_bounds__(256, 2) void k_quantize_values_mfma(CodecJob j, const float* __restrict__ rot,
                                                                 Thresholds th, uint8_t* __restrict__ v_codes,
                                                                 uint16_t* __restrict__ v_norm,
                                                                 uint8_t* __restrict__ mod_out) {
  __shared__ __attribute__((aligned(16))) _Float16 rstage[2 * kRStage];  // [2][128][kRPitch]: hi, lo
  __shared__ uint32_t present;

  const int wave = threadIdx.x >> 6;
  const int lane = lane_id();
  const int r = lane & 15, g = lane >> 4;
  const int h = blockIdx.y, bz = blockIdx.z, b = j.b0 + bz;
  int begin, len;
  job_range_v(j, bz, b, begin, len);
  if (len <= begin) return;
  const int first = (begin / kW) * kW;
  const int tile0 = first + blockIdx.x * 256;
  if (tile0 >= len) return;  // whole block idle: no barrier reached
  const int wtok0 = tile0 + wave * 64;
  const size_t seq = (size_t)b * j.H + h;
  const int wend = ((len + kW - 1) / kW) * kW;  // end of the last window

  if (threadIdx.x == 0) present = 0;
  __syncthreads();

  // ---- A operands (v rows, fp16) and modality of the wave's tokens ----
  uint4 a[4][4];  // [row block][k block]
#pragma unroll
  for (int rb = 0; rb < 4; ++rb) {
    const int t = wtok0 + 16 * rb + r;
    const bool fresh = t >= begin && t < len;
    const uint4* row = reinterpret_cast<const uint4*>(j.src + (seq * j.n_rows + (size_t)max(t - begin, 0)) * kD);
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) a[rb][kk] = fresh ? row[4 * kk + g] : make_uint4(0, 0, 0, 0);
  }
  const int mytok = wtok0 + lane;  // lane = token for the modality ballot
  int mymod = -1;
  if (mytok >= begin && mytok < len) {
    mymod = (int)j.msrc[(size_t)b * j.n_rows + (mytok - begin)];
    if (mod_out && h == 0) mod_out[(size_t)b * j.cap + mytok] = (uint8_t)mymod;
  }
  uint32_t wave_present = 0;
#pragma unroll
  for (int m = 0; m < 3; ++m)
    if (__ballot(mymod == m)) wave_present |= 1u << m;
  if (lane == 0 && wave_present) atomicOr(&present, wave_present);

  // ---- norms by the halving tree; lane (r, g) holds channels 32 kk + 8 g + e of token r ----
  float n16f_tok[4];  // n16 of token 16 rb + r
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
    for (int e = 0; e < 8; ++e) s[e] = s[e] + __shfl_xor(s[e], 16);  // level 8: g with g ^ 1
#pragma unroll
    for (int n = 4; n >= 1; n >>= 1) {
#pragma unroll
      for (int e = 0; e < n; ++e) s[e] = s[e] + s[e + n];
    }
    const int t = wtok0 + 16 * rb + r;
    const bool fresh = t >= begin && t < len;
    const uint32_t n16 = fresh ? norm_to_f16(sqrt_rn(s[0])) : 0u;
    n16f_tok[rb] = h2f(n16);
    if (g == 0 && t >= begin && t < wend) v_norm[seq * j.cap + t] = (uint16_t)n16;
  }
  // per lane: norms and modalities of the four tokens 16 rb + 4 g + i of its output rows
  float nrow[4][4];
  int mrow[4][4];
#pragma unroll
  for (int rb = 0; rb < 4; ++rb) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      nrow[rb][i] = __shfl(n16f_tok[rb], 4 * g + i);
      mrow[rb][i] = __shfl(mymod, 16 * rb + 4 * g + i);
    }
  }
  __syncthreads();
  const uint32_t pres = present;

  uint32_t bytes[4][2];  // [row block][nb / 4]: 8 code bytes per row block
#pragma unroll
  for (int rb = 0; rb < 4; ++rb) bytes[rb][0] = bytes[rb][1] = 0;

  _Float16* rhi = rstage;
  _Float16* rlo = rstage + kRStage;
  for (int m = 0; m < 3; ++m) {
    if (!(pres & (1u << m))) continue;  // block-uniform
    __syncthreads();                    // previous modality's reads are done
    const float4* src = reinterpret_cast<const float4*>(rot + (size_t)m * kD * kD);
    for (int idx = threadIdx.x; idx < kD * kD / 4; idx += 256) {
      const float4 f = src[idx];
      const int n = idx >> 5, k4 = (idx & 31) * 4;
      const float fv[4] = {f.x, f.y, f.z, f.w};
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const _Float16 hi = (_Float16)fv[q];
        rhi[n * kRPitch + k4 + q] = hi;
        rlo[n * kRPitch + k4 + q] = (_Float16)(fv[q] - (float)hi);
      }
    }
    __syncthreads();
    if (!(wave_present & (1u << m))) continue;  // wave-uniform
    // one straight-line MFMA sweep (8 output blocks x 4 k-blocks x hi/lo) per 16-token row block that
    // holds modality m; row blocks without it are skipped by a wave-uniform branch
#pragma unroll
    for (int rb = 0; rb < 4; ++rb) {
      if (!__ballot((mymod == m) && ((lane >> 4) == rb))) continue;
      floatx4 acc[8];
#pragma unroll
      for (int nb = 0; nb < 8; ++nb) acc[nb] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        const half8 av = as_half8(a[rb][kk]);
#pragma unroll
        for (int part = 0; part < 2; ++part) {  // hi then lo: eight independent accumulators in between
          const _Float16* rp = part ? rlo : rhi;
#pragma unroll
          for (int nb = 0; nb < 8; ++nb) {
            const half8 bv = *reinterpret_cast<const half8*>(rp + (16 * nb + r) * kRPitch + 32 * kk + 8 * g);
            acc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(av, bv, acc[nb], 0, 0, 0);
          }
        }
      }
#pragma unroll
      for (int nb = 0; nb < 8; ++nb) {
        uint32_t byte = 0;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const uint32_t code = value_code(acc[nb][i], nrow[rb][i], th);
          byte |= (mrow[rb][i] == m ? code : 0u) << (2 * i);
        }
        bytes[rb][nb >> 2] |= byte << (8 * (nb & 3));
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
