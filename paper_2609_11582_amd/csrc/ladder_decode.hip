// Decode attention over a bit-width-ladder cache (b-bit keys and values, b = 2, 3, 4; the codecs
// are in ladder_codec.hip): Eq. 1 in the rotated spaces of Sec. 2.3, split-K like the 2-bit kernel.
//
// Work-group (split, KV head h, sequence b) = 8 waves; wave w takes the split's 32-token windows
// w, w + 8, ... and keeps its own online softmax for the G <= 8 query heads of the KV head.
//  * scores s_t = n_t (q' . zhat_t), q' = H q sm_scale log2(e). The A operands of the score MFMA
//    come from one contiguous run of each lane's token row (channels 32 g .. 32 g + 31; k-block kb
//    takes channels 32 g + 8 kb .. + 7 in both operands): 2- and 4-bit codes of the method's keys
//    directly, as fp16 subnormals (the field masked per channel pair; the power of two of a
//    channel's bit position is folded into the query operand), 3-bit codes and TurboQuant levels
//    through a small LDS table indexed by a code pair. For the method's keys zhat = m + step code
//    is split as in the 2-bit kernel: the window term q' . m in fp32 (a per-window bias, on the
//    matrix cores against the query's fp16 hi and lo parts) and
//    sum_c q'_c step_c code_c on the matrix cores with B = fp16(q'_c step_c 2^(k0 - shift_c)) --
//    rounding the whole of m + step code to fp16 would cost too much where the keys' window means
//    are large (they drift);
//  * values: each lane dequantizes 64 codes of one token row through a table of codebook levels
//    (a code byte -> four levels for 2-bit values, a code pair -> two otherwise) into the wave's
//    LDS tile (16-byte-chunk XOR swizzle); the PV B operands come back with
//    the transposing LDS read of gfx950 (ds_read_b64_tr_b16), in the token order of the score
//    tile's rows;
//  * per-modality PV (values stay rotated): the A operand's rows 0-7 are the audio-masked p n_v of
//    the 8 heads, rows 8-15 the video-masked ones (taken from lane - 8 by a DPP row rotation); text
//    tokens (the prompt, a few windows) are accumulated in the wave's LDS text tile;
//  * epilogue: the waves' accumulators are combined in LDS, un-rotated on the matrix cores once per
//    present modality against the fp16 table R_m^T, and one normalized record per split goes to the
//    log-sum-exp merge launch shared with the other decode kernels.
#include <hip/hip_ext.h>

#include <algorithm>
#include <cstdlib>

#include "launch.hpp"

namespace okvq {
namespace {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef _Float16 half2v __attribute__((ext_vector_type(2)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef short short4v __attribute__((ext_vector_type(4)));

constexpr int kLw = 8;                   // waves per work-group
constexpr int kLStep = kLw * kW;         // tokens per work-group step
constexpr int kATileL = 3 * kD + 8;      // fp16 row pitch of the un-rotation A tile
constexpr float kLazyL = 8.0f;           // log2 headroom of the lazily updated softmax reference

// Smallest nvb in [nvb0, 16] with every lane's value norm bound `nv` (finite, below 2^16) under
// 2^nvb. Wave-uniform; a short scalar loop.
__device__ __forceinline__ int norm_bound_f(float nv, int nvb0) {
  int nvb = nvb0;
  while (nvb < 16 && __any(nv >= ldexpf(1.0f, nvb))) ++nvb;
  return nvb;
}

__device__ __forceinline__ half8 h8(uint32_t a, uint32_t b, uint32_t c, uint32_t d) {
  return __builtin_bit_cast(half8, make_uint4(a, b, c, d));
}
__device__ __forceinline__ uint32_t pk_h2(float lo, float hi) {
  const half2v v = {(_Float16)lo, (_Float16)hi};
  return __builtin_bit_cast(uint32_t, v);
}
__device__ __forceinline__ float lo_h(uint32_t w) { return (float)__builtin_bit_cast(half2v, w)[0]; }
__device__ __forceinline__ float hi_h(uint32_t w) { return (float)__builtin_bit_cast(half2v, w)[1]; }
__device__ __forceinline__ short4v lds_tr(const uint8_t* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) short4v*)p);
}
__device__ __forceinline__ float dpp_ror8(float v) {  // lane l <- lane (l + 8) mod 16 of its row
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x128, 0xf, 0xf, false));
}
template <int kN>
__device__ __forceinline__ float dpp_ror(float v) {  // a rotation by kN lanes inside each 16-lane row
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x120 + kN, 0xf, 0xf, false));
}
// bits [sh, sh + n) of the 64-bit word hi:lo (sh < 32)
__device__ __forceinline__ uint32_t field64(uint32_t lo, uint32_t hi, int sh) {
  return sh == 0 ? lo : __builtin_amdgcn_alignbit(hi, lo, (uint32_t)sh);
}

// Float offsets of the combine tiles, whose 16-byte slots are XOR-swizzled by the channel so that
// 16 lanes reading or writing one slot of 16 consecutive channels hit distinct banks: a wave's rows
// [channel k][16] (slot s = rows 4 s .. 4 s + 3) and its text rows [channel k][8] (slot s = heads
// 4 s .. 4 s + 3).
__device__ __forceinline__ int row_ofs(int w, int k, int s) { return ((w * kD + k) << 4) + 4 * (s ^ ((k >> 2) & 3)); }
__device__ __forceinline__ int text_ofs(int k, int s) { return (k << 3) + 4 * (s ^ ((k >> 3) & 1)); }

// One window's loads for one lane (issued a window ahead of their use).
template <int kKB, int kVB>
struct LTile {
  uint32_t kw[2][kKB];   // key codes of channels 32 g .. 32 g + 31 of token 16 tb + r (4 kKB bytes)
  uint32_t vc[2 * kVB];  // 64 value codes of row lane / 2, channels 64 (lane % 2) .. + 63
  uint2 nk[2], nv[2];    // norms of tokens 16 tb + 4 g .. + 3
  uint32_t md[2];        // their modality bytes
  uint2 meta;            // 8 bytes of the window's (minimum, step) rows (method keys)
};

template <int kKB, int kVB, bool kTq>
__global__ __launch_bounds__(64 * kLw) void k_ladder_decode(LadderDecodeArgs p) {
  constexpr int kKRow = 16 * kKB, kVRow = 16 * kVB;  // bytes per packed token row
  constexpr uint32_t kKMask = (1u << (2 * kKB)) - 1u, kVMask = (1u << (2 * kVB)) - 1u;
  // 2- and 4-bit codes of the method's keys enter the score MFMA directly as fp16 subnormals (the
  // field masked per channel pair, the power of two folded into the query operand); 3-bit codes and
  // TurboQuant levels through a code-pair table
  constexpr bool kDirect = !kTq && (kKB == 2 || kKB == 4);
  // 2-bit values: a code byte (4 channels) -> four fp16 codebook levels; else a code pair -> two
  constexpr bool kVByte = kVB == 2;
  __shared__ uint32_t klut[kDirect ? 1 : 1 << (2 * kKB)];  // key code pair -> fp16 pair (integers, or TurboQuant levels)
  __shared__ __attribute__((aligned(8))) uint32_t vlut[kVByte ? 512 : 1 << (2 * kVB)];
  __shared__ __attribute__((aligned(16))) float qs[8][kD + 4];
  __shared__ __attribute__((aligned(16))) uint8_t vt[kLw][kW * kD * 2];    // value tiles
  __shared__ __attribute__((aligned(16))) uint16_t mt[kLw][2][kD];         // window (minimum, step)
  __shared__ __attribute__((aligned(16))) _Float16 atile[8][kATileL];
  __shared__ float wst[2][8][kLw];
  __shared__ uint32_t wmask[kLw], nv_all;  // nv_all: the largest value norm (fp32 bits, non-negative)
  __shared__ int wexp[kLw];
  __shared__ __attribute__((aligned(16))) float fac[kLw][8];      // combine factor per wave and head
  __shared__ __attribute__((aligned(16))) float ttx[kLw][kD][8];  // text rows (heads 0-7) per wave, swizzled
  __shared__ float amax_w[4];

  const int split = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, g = lane >> 4, r = lane & 15;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  // the length (a scalar load, read before any divergent branch), then the query rows and signs
  // (waves 0-3), before anything waits
  const int len = min(p.seq_lens[b], p.cap);
  const int hr = 2 * wave + (lane >> 5), c4 = 4 * (lane & 31);
  uint2 qr = make_uint2(0u, 0u);
  uint32_t sg = 0u;
  if (wave < 4 && hr < p.G) {
    qr = *reinterpret_cast<const uint2*>(p.q + ((size_t)b * p.Hq + h * p.G + hr) * kD + c4);
    sg = *reinterpret_cast<const uint32_t*>(p.signs + c4);
  }
  const int t_begin = split * p.tps, t_end = min(t_begin + p.tps, len);
  const size_t seq = (size_t)b * p.H + h;
  float* rec = p.ws + (seq * p.nsplit + split) * kRecFloats;
  if (t_begin >= t_end) {
    write_empty_record(rec, tid);
    return;
  }
  const uint8_t* kbase = p.k_codes + seq * p.cap * kKRow;
  const uint8_t* vbase = p.v_codes + seq * p.cap * kVRow;
  const uint16_t* nkbase = p.k_norm + seq * p.cap;
  const uint16_t* nvbase = p.v_norm + seq * p.cap;
  const uint8_t* mdbase = p.modality + (size_t)b * p.cap;
  const size_t nwcap = p.cap / kW;
  const int ntile = (t_end - t_begin + kW - 1) / kW;
  const int nmine = ntile > wave ? (ntile - wave + kLw - 1) / kLw : 0;
  // The score MFMA's k-block kb takes channels 32 g + 8 kb .. + 7 in lane group g (the A and B
  // operands agree on it, and the contraction covers every channel once), so a lane's four blocks
  // are one contiguous run of 4 kKB bytes of the token row.

  auto issue_tile = [&](int tile, LTile<kKB, kVB>& lt) {
    const int t0 = t_begin + tile * kW;
    const int last = t_end - 1;
#pragma unroll
    for (int tb = 0; tb < 2; ++tb) {
      const uint8_t* row = kbase + (size_t)min(t0 + 16 * tb + r, last) * kKRow + 4 * kKB * g;
      if constexpr (kKB == 2) {
        const uint2 u = *reinterpret_cast<const uint2*>(row);
        lt.kw[tb][0] = u.x;
        lt.kw[tb][1] = u.y;
      } else if constexpr (kKB == 4) {
        const uint4 u = *reinterpret_cast<const uint4*>(row);
        lt.kw[tb][0] = u.x;
        lt.kw[tb][1] = u.y;
        lt.kw[tb][2] = u.z;
        lt.kw[tb][3] = u.w;
      } else {
        const uint32_t* w = reinterpret_cast<const uint32_t*>(row);
#pragma unroll
        for (int i = 0; i < kKB; ++i) lt.kw[tb][i] = w[i];
      }
      // norms and modalities of 4 tokens inside the window (slots past the length are masked later)
      lt.nk[tb] = *reinterpret_cast<const uint2*>(nkbase + t0 + 16 * tb + 4 * g);
      lt.nv[tb] = *reinterpret_cast<const uint2*>(nvbase + t0 + 16 * tb + 4 * g);
      lt.md[tb] = *reinterpret_cast<const uint32_t*>(mdbase + t0 + 16 * tb + 4 * g);
    }
    {
      const uint8_t* vrow = vbase + (size_t)min(t0 + (lane >> 1), last) * kVRow + 8 * kVB * (lane & 1);
      if constexpr (kVB % 2 == 0) {  // 16-byte aligned halves
#pragma unroll
        for (int i = 0; i < kVB / 2; ++i) {
          const uint4 u = reinterpret_cast<const uint4*>(vrow)[i];
          lt.vc[4 * i] = u.x;
          lt.vc[4 * i + 1] = u.y;
          lt.vc[4 * i + 2] = u.z;
          lt.vc[4 * i + 3] = u.w;
        }
      } else {
#pragma unroll
        for (int i = 0; i < kVB; ++i) {
          const uint2 u = reinterpret_cast<const uint2*>(vrow)[i];
          lt.vc[2 * i] = u.x;
          lt.vc[2 * i + 1] = u.y;
        }
      }
    }
    if constexpr (!kTq) {
      const size_t mrow = (seq * nwcap + t0 / kW) * kD;
      const uint16_t* src = (lane < 32 ? p.k_min : p.k_step) + mrow + 4 * (lane & 31);
      lt.meta = *reinterpret_cast<const uint2*>(src);
    }
    __builtin_amdgcn_sched_barrier(0);  // the window's loads go out before the work that follows
  };
  auto issue = [&](int it, LTile<kKB, kVB>& lt) { issue_tile(wave + kLw * it, lt); };
  // The first window is loaded before the tables and the query rotation, and unconditionally (a
  // wave without a window loads the split's last one and never uses it), so that the barrier below
  // waits for the query loads only.
  LTile<kKB, kVB> ta, tn;  // the window being computed, and the next one in flight
  issue_tile(min(wave, ntile - 1), ta);

  // ---- tables, and the rotated query: wave w < 4 rotates heads 2w, 2w + 1 (lane: 4 channels) ----
  // code-pair tables; the codebook levels are picked by selects over constant indices (a dynamic
  // index into the argument arrays would read them through memory, one more round trip)
  auto level = [](const uint16_t (&cb)[16], int c, int n) {
    uint32_t v = (uint32_t)__builtin_amdgcn_readfirstlane((int)cb[0]);
#pragma unroll
    for (int j = 1; j < 16; ++j)
      if (j < n) v = (c == j) ? (uint32_t)__builtin_amdgcn_readfirstlane((int)cb[j]) : v;
    return v;
  };
  if constexpr (!kDirect) {
    for (int i = tid; i < (1 << (2 * kKB)); i += 64 * kLw) {
      const int c0 = i & ((1 << kKB) - 1), c1 = i >> kKB;
      klut[i] = kTq ? level(p.kcb16, c0, 1 << kKB) | (level(p.kcb16, c1, 1 << kKB) << 16) : pk_h2((float)c0, (float)c1);
    }
  }
  if constexpr (kVByte) {
    if (tid < 256) {
      vlut[2 * tid] = level(p.vcb16, tid & 3, 4) | (level(p.vcb16, (tid >> 2) & 3, 4) << 16);
      vlut[2 * tid + 1] = level(p.vcb16, (tid >> 4) & 3, 4) | (level(p.vcb16, tid >> 6, 4) << 16);
    }
  } else {
    for (int i = tid; i < (1 << (2 * kVB)); i += 64 * kLw) {
      const int c0 = i & ((1 << kVB) - 1), c1 = i >> kVB;
      vlut[i] = level(p.vcb16, c0, 1 << kVB) | (level(p.vcb16, c1, 1 << kVB) << 16);
    }
  }
  if (wave < 4) {
    float x[4];
    {  // zero for heads >= G (their loads were skipped)
      const float v[4] = {lo_h(qr.x), hi_h(qr.x), lo_h(qr.y), hi_h(qr.y)};
#pragma unroll
      for (int i = 0; i < 4; ++i) x[i] = ((sg >> (8 * i + 7)) & 1u) ? -v[i] : v[i];
    }
    {  // channel bits 0, 1 inside the lane
      const float a = x[0] + x[1], c = x[0] - x[1], d = x[2] + x[3], e = x[2] - x[3];
      x[0] = a + d;
      x[2] = a - d;
      x[1] = c + e;
      x[3] = c - e;
    }
#pragma unroll
    for (int lb = 1; lb < 32; lb <<= 1) {  // channel bits 2 .. 6 are lane bits 0 .. 4
      const bool hi = (lane & lb) != 0;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float o = __shfl_xor(x[i], lb);
        x[i] = hi ? o - x[i] : x[i] + o;
      }
    }
    float am = 0.0f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      x[i] *= p.qscale;
      am = fmaxf(am, fabsf(x[i]));
    }
#pragma unroll
    for (int lb = 1; lb < 64; lb <<= 1) am = fmaxf(am, __shfl_xor(am, lb));
    if (lane == 0) amax_w[wave] = am;
    if (tid == 0) nv_all = 0u;
    *reinterpret_cast<float4*>(&qs[hr][c4]) = make_float4(x[0], x[1], x[2], x[3]);
  }
  __syncthreads();
  // power-of-two scale 2^k0 of the fp16 query operands: |q'| 2^k0 <= 2^15 (steps are below 1 and
  // codebook levels below 1/4, so the products stay in range too)
  const float amax = fmaxf(fmaxf(amax_w[0], amax_w[1]), fmaxf(amax_w[2], amax_w[3]));
  const int k0 = (amax > 0.0f) ? min(max(14 - ilogbf(amax), -60), 60) : 0;
  // direct key codes: channel c of an 8-channel group sits 2 (c & 3) (2-bit) or 4 (c & 1) (4-bit)
  // bits up in its fp16 half, worth code 2^(shift - 24); the query operand carries 2^-shift
  auto cshift = [](int c) { return kDirect ? (kKB == 2 ? 2 * (c & 3) : 4 * (c & 1)) : 0; };
  const float kinv = ldexpf(1.0f, kDirect ? 24 - k0 : -k0);
  // score B operands: channel 32 g + 8 kb + e, head r (zero rows for heads >= G are already zero)
  uint32_t qop[4][4];
  // bias B operands (method keys): column r < 8 holds fp16(q'[r] 2^k0), column r >= 8 the rounding
  // residual of the same for head r - 8, so that a column pair sums to q' 2^k0 to about 2^-22
  uint32_t qbo[4][4];
#pragma unroll
  for (int kb = 0; kb < 4; ++kb) {
    const float4 a = *reinterpret_cast<const float4*>(&qs[r & 7][32 * g + 8 * kb]);
    const float4 c = *reinterpret_cast<const float4*>(&qs[r & 7][32 * g + 8 * kb + 4]);
    const float qv[8] = {a.x, a.y, a.z, a.w, c.x, c.y, c.z, c.w};
    const bool live = r < 8;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      qop[kb][j] = live ? pk_h2(ldexpf(qv[2 * j], k0 - cshift(2 * j)), ldexpf(qv[2 * j + 1], k0 - cshift(2 * j + 1))) : 0u;
      if constexpr (!kTq) {
        float v[2];
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          const float x = ldexpf(qv[2 * j + u], k0);
          const float hi = (float)(_Float16)x;
          v[u] = live ? hi : x - hi;
        }
        qbo[kb][j] = pk_h2(v[0], v[1]);
      }
    }
  }
  const float bscale = ldexpf(1.0f, -k0);


  floatx4 acc[8];  // rows 0-7 audio heads, 8-15 video heads; channel 16 cb + r
#pragma unroll
  for (int cb = 0; cb < 8; ++cb) acc[cb] = floatx4{0.f, 0.f, 0.f, 0.f};
  float* txw = &ttx[wave][0][0];  // [channel][head]; lanes of g < 2 own heads 4 g .. 4 g + 3
  if (g < 2) {
#pragma unroll
    for (int cb = 0; cb < 8; ++cb)
      *reinterpret_cast<float4*>(txw + text_ofs(16 * cb + r, g)) = make_float4(0.f, 0.f, 0.f, 0.f);
  }
  float m_run = -__builtin_inff(), l_part = 0.0f, nvmax = 0.0f;
  bool started = false;
  // Operand scale 2^E of p n_v (wave-uniform): every value norm seen is below 2^nvb, so with
  // p <= 1 the product p 2^E n_v stays below 2^15 for E = min(15, 15 - nvb); l_part and the
  // accumulators hold 2^E times the unscaled sums (the combine divides it out).
  int nvb = 0, E = 15;
  uint32_t seen = 0;
  uint8_t* vtw = &vt[wave][0];
  const int trow = 4 * g + (r >> 2), tsub = r & 3;
  const int vrw = lane >> 1, vhalf = lane & 1;

  auto compute = [&](int it, const LTile<kKB, kVB>& lt) {
    const int t0 = t_begin + (wave + kLw * it) * kW;
    // ---- key operands ----
    float bias = 0.0f;   // q' . m of this window for head r (method keys), fp32
    uint32_t bq[4][4];   // B operands: fp16(q'_c step_c 2^k0) (method keys), or the query itself
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int j = 0; j < 4; ++j) bq[kb][j] = qop[kb][j];
    if constexpr (!kTq) {
      *reinterpret_cast<uint2*>(&mt[wave][lane >> 5][4 * (lane & 31)]) = lt.meta;
      wave_lds_sync();
      // q' . m on the matrix cores: every A row holds the window's minima, B the query's hi and lo
      // columns; a lane adds its column and the partner column r ^ 8
      floatx4 bacc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        const uint4 mn4 = *reinterpret_cast<const uint4*>(&mt[wave][0][32 * g + 8 * kb]);
        const uint4 st4 = *reinterpret_cast<const uint4*>(&mt[wave][1][32 * g + 8 * kb]);
        bacc = __builtin_amdgcn_mfma_f32_16x16x32_f16(h8(mn4.x, mn4.y, mn4.z, mn4.w),
                                                      h8(qbo[kb][0], qbo[kb][1], qbo[kb][2], qbo[kb][3]), bacc, 0, 0, 0);
        const uint32_t sv[4] = {st4.x, st4.y, st4.z, st4.w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const half2v prod = __builtin_bit_cast(half2v, qop[kb][j]) * __builtin_bit_cast(half2v, sv[j]);
          bq[kb][j] = __builtin_bit_cast(uint32_t, prod);
        }
      }
      bias = (bacc[0] + dpp_ror8(bacc[0])) * bscale;
    }
    floatx4 sc[2] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
#pragma unroll
    for (int tb = 0; tb < 2; ++tb) {
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        uint32_t a[4];
        if constexpr (kDirect && kKB == 2) {  // the 16-bit field in both halves, then shifted by 8
          const uint32_t d = lt.kw[tb][kb >> 1];
          const uint32_t f = __builtin_amdgcn_perm(d, d, (kb & 1) ? 0x03020302u : 0x01000100u), f8 = f >> 8;
          a[0] = f & 0x000c0003u;
          a[1] = f & 0x00c00030u;
          a[2] = f8 & 0x000c0003u;
          a[3] = f8 & 0x00c00030u;
        } else if constexpr (kDirect) {  // 4-bit: byte j of the field holds channels 2j, 2j + 1
          const uint32_t d = lt.kw[tb][kb];
#pragma unroll
          for (int j = 0; j < 4; ++j) a[j] = __builtin_amdgcn_perm(d, d, 0x01010101u * j) & 0x00f0000fu;
        } else {
          // the block's field: bits 8 kKB kb .. + 8 kKB - 1 of the lane's run
          constexpr int kFieldBits = 8 * kKB;
          const int bit = kFieldBits * kb, dw = bit >> 5, sh = bit & 31;
          const uint32_t f = (sh + kFieldBits <= 32) ? (lt.kw[tb][dw] >> sh) : field64(lt.kw[tb][dw], lt.kw[tb][dw + 1], sh);
#pragma unroll
          for (int j = 0; j < 4; ++j) a[j] = klut[(f >> (2 * kKB * j)) & kKMask];
        }
        sc[tb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(h8(a[0], a[1], a[2], a[3]),
                                                        h8(bq[kb][0], bq[kb][1], bq[kb][2], bq[kb][3]), sc[tb],
                                                        0, 0, 0);
      }
    }
    // ---- online softmax; sc[tb][i] = score of token 16 tb + 4 g + i for head r ----
    float x[8], nvf[8];
    uint32_t mdv[2] = {lt.md[0], lt.md[1]};
    float mx = -__builtin_inff();
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int tb = e >> 2, i = e & 3;
      const int t = t0 + 16 * tb + 4 * g + i;
      const bool ok = t < t_end;
      const uint32_t nkw = (i < 2) ? lt.nk[tb].x : lt.nk[tb].y;
      const uint32_t nvw = (i < 2) ? lt.nv[tb].x : lt.nv[tb].y;
      const float nk = (i & 1) ? hi_h(nkw) : lo_h(nkw);
      // computed for every slot and then selected (slots past the length hold whatever the norms'
      // memory holds there): kept out of a branch per slot, which the compiler would otherwise form
      float nvv = (i & 1) ? hi_h(nvw) : lo_h(nvw);
      float xv = nk * __builtin_fmaf(sc[tb][i], kinv, bias);
      __asm__ volatile("" : "+v"(nvv), "+v"(xv));
      nvf[e] = ok ? nvv : 0.0f;
      x[e] = ok ? xv : -__builtin_inff();
      if (!ok) mdv[tb] |= 0x03u << (8 * i);  // modality 3: no token
      mx = fmaxf(mx, x[e]);
    }
    // mx is the lane's maximum; a head's maximum over its four lane groups is needed only where the
    // reference moves (a lane above m_run + kLazyL puts its head above it too)
    auto head_max = [](float v) {
      v = fmaxf(v, __shfl_xor(v, 16));
      return fmaxf(v, __shfl_xor(v, 32));
    };
    float nvl = 0.0f;  // the lane's largest value norm so far, this window's included
#pragma unroll
    for (int e = 0; e < 8; ++e) nvl = fmaxf(nvl, nvf[e]);
    nvmax = fmaxf(nvmax, nvl);
    if (!started) {
      m_run = head_max(mx);
      nvb = min(norm_bound_f(nvmax, 0) + 1, 16);
      E = min(15, 15 - nvb);
      started = true;
    } else if (__any(mx > m_run + kLazyL) || __any(nvmax >= ldexpf(1.0f, nvb))) {
      const float m_new = fmaxf(m_run, head_max(mx));
      const int nb = norm_bound_f(nvmax, nvb);
      const int nvb_new = nb > nvb ? min(nb + 1, 16) : nvb;
      const int E_new = min(15, 15 - nvb_new);
      const float alpha = __builtin_amdgcn_exp2f((m_run - m_new) + (float)(E_new - E));
      l_part *= alpha;
#pragma unroll
      for (int i = 0; i < 4; ++i) {  // accumulator rows 4 g + i are heads (4 g + i) mod 8
        const float ai = __shfl(alpha, (4 * g + i) & 7);
#pragma unroll
        for (int cb = 0; cb < 8; ++cb) acc[cb][i] *= ai;
      }
      if (g < 2) {
#pragma unroll
        for (int cb = 0; cb < 8; ++cb) {
          float4* t4 = reinterpret_cast<float4*>(txw + text_ofs(16 * cb + r, g));
          const float4 v = *t4;
          float ai[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) ai[i] = __shfl(alpha, 4 * g + i);
          *t4 = make_float4(v.x * ai[0], v.y * ai[1], v.z * ai[2], v.w * ai[3]);
        }
      }
      m_run = m_new;
      nvb = nvb_new;
      E = E_new;
    }
    const float mref = m_run + kLazyL - (float)E;  // pe = p 2^E with p = 2^(s - m_run - 8) <= 1
    float pv[8], pp[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float pe = __builtin_amdgcn_exp2f(x[e] - mref);  // 0 for no token
      l_part += pe;
      pv[e] = pe * nvf[e];  // below 2^15: fits fp16
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) pp[e] = dpp_ror8(pv[e]);  // heads r - 8 for the video rows
    uint32_t pres = 0;
#pragma unroll
    for (int e = 0; e < 8; ++e) pres |= 1u << ((mdv[e >> 2] >> (8 * (e & 3))) & 3u);
    const bool has_a = __any(pres & 1u), has_v = __any(pres & 2u), has_t = __any(pres & 4u);
    seen |= (has_a ? 1u : 0u) | (has_v ? 2u : 0u) | (has_t ? 4u : 0u);
    float av[8], tx[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const uint32_t m = (mdv[e >> 2] >> (8 * (e & 3))) & 0xffu;
      av[e] = (r < 8) ? (m == 0u ? pv[e] : 0.0f) : (m == 1u ? pp[e] : 0.0f);
      tx[e] = (r < 8 && m == 2u) ? pv[e] : 0.0f;
    }
    // A operand: row = head slot r, k = 8 g + e <-> token 4 g + e (e < 4), 16 + 4 g + e - 4 (e >= 4)
    const half8 a_av = h8(pk_h2(av[0], av[1]), pk_h2(av[2], av[3]), pk_h2(av[4], av[5]), pk_h2(av[6], av[7]));
    const half8 a_tx = h8(pk_h2(tx[0], tx[1]), pk_h2(tx[2], tx[3]), pk_h2(tx[4], tx[5]), pk_h2(tx[6], tx[7]));

    // ---- value tile: dequantize 64 codes of row lane / 2 into LDS, 8 channels at a time ----
#pragma unroll
    for (int jj = 0; jj < 8; ++jj) {
      uint32_t dq[4];
      if constexpr (kVByte) {  // bytes 2 jj, 2 jj + 1 of the row's 16: channels 8 jj .. 8 jj + 7
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          const int by = 2 * jj + u;
          const uint2 lv = *reinterpret_cast<const uint2*>(&vlut[2 * ((lt.vc[by >> 2] >> (8 * (by & 3))) & 0xffu)]);
          dq[2 * u] = lv.x;
          dq[2 * u + 1] = lv.y;
        }
      } else {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int j = 4 * jj + u;
          const int bit = 2 * kVB * j, d = bit >> 5, sh = bit & 31;
          const uint32_t f = (sh + 2 * kVB <= 32) ? (lt.vc[d] >> sh) : field64(lt.vc[d], lt.vc[d + 1], sh);
          dq[u] = vlut[f & kVMask];
        }
      }
      const int slot = (8 * vhalf + jj) ^ (vrw & 15);
      *reinterpret_cast<uint4*>(vtw + vrw * 256 + 16 * slot) = make_uint4(dq[0], dq[1], dq[2], dq[3]);
    }
    wave_lds_sync();
#pragma unroll
    for (int cb = 0; cb < 8; ++cb) {
      const int slot = ((2 * cb + (tsub >> 1)) ^ trow) * 16 + 8 * (tsub & 1);
      const uint2 l2 = __builtin_bit_cast(uint2, lds_tr(vtw + trow * 256 + slot));
      const uint2 h2 = __builtin_bit_cast(uint2, lds_tr(vtw + (16 + trow) * 256 + slot));
      const half8 vb = h8(l2.x, l2.y, h2.x, h2.y);
      acc[cb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a_av, vb, acc[cb], 0, 0, 0);
      if (has_t) {  // wave-uniform
        const floatx4 t = __builtin_amdgcn_mfma_f32_16x16x32_f16(a_tx, vb, floatx4{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
        if (g < 2) {
          float4* t4 = reinterpret_cast<float4*>(txw + text_ofs(16 * cb + r, g));
          const float4 v = *t4;
          *t4 = make_float4(v.x + t[0], v.y + t[1], v.z + t[2], v.w + t[3]);
        }
      }
    }
    wave_lds_sync();  // transposed reads done before the next window overwrites the tile
  };

  int it = 0;
  for (; it + 2 < nmine; it += 2) {
    issue(it + 1, tn);
    compute(it, ta);
    issue(it + 2, ta);
    compute(it + 1, tn);
  }
  if (it + 1 < nmine) {
    issue(it + 1, tn);
    compute(it, ta);
    compute(it + 1, tn);
  } else if (it < nmine) {
    compute(it, ta);
  }

  // ---- epilogue: the inverse-rotation slice of this wave (output channels 16 wave .. + 15) ----
  uint4 rb[12];
  {
    const uint4* rp = reinterpret_cast<const uint4*>(p.rot16t) + (size_t)(16 * wave + (lane & 15)) * 48 + (lane >> 4);
#pragma unroll
    for (int kk = 0; kk < 12; ++kk) rb[kk] = rp[4 * kk];
  }
  float l_tot = l_part + __shfl_xor(l_part, 16);
  l_tot += __shfl_xor(l_tot, 32);
  // the largest value norm: a maximum over each 16-lane row by DPP rotations, then one LDS atomic per
  // row (non-negative floats order as their bit patterns)
  float nvr = nvmax;
  nvr = fmaxf(nvr, dpp_ror8(nvr));
  nvr = fmaxf(nvr, dpp_ror<4>(nvr));
  nvr = fmaxf(nvr, dpp_ror<2>(nvr));
  nvr = fmaxf(nvr, dpp_ror<1>(nvr));
  if (r == 0) __hip_atomic_fetch_max(&nv_all, __builtin_bit_cast(uint32_t, nvr), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  // [wave][channel][16 rows]: audio 0-7, video 8-15; wave w's rows fill exactly its own value tile,
  // which it no longer reads, so no barrier is needed before the writes
  float* wacc = reinterpret_cast<float*>(&vt[0][0]);
#pragma unroll
  for (int cb = 0; cb < 8; ++cb)
    *reinterpret_cast<float4*>(wacc + row_ofs(wave, 16 * cb + r, g)) =
        make_float4(acc[cb][0], acc[cb][1], acc[cb][2], acc[cb][3]);
  if (lane < 8) {
    wst[0][lane][wave] = started ? m_run : -__builtin_inff();
    wst[1][lane][wave] = ldexpf(l_tot, -E);  // relative to 2^(m_run + kLazyL)
  }
  if (lane == 0) {
    wmask[wave] = seen;
    wexp[wave] = E;
  }
  __syncthreads();
  uint32_t mask = 0;
  const float nmax = __builtin_bit_cast(float, nv_all);
#pragma unroll
  for (int w = 0; w < kLw; ++w) mask |= wmask[w];
  // merged rows divided by L are convex combinations of n_v cb vectors (|cb| < 1/4): the factor
  // 2^e / L with e = 13 - ilogb(n_max) keeps the fp16 A tile below 2^12
  const int e = (nmax > 0.0f) ? 13 - min(max(ilogbf(nmax), -30), 20) : 0;
  if (tid < 8 * kLw) {
    const int hh = tid >> 3, w = tid & 7;
    float M = -__builtin_inff();
#pragma unroll
    for (int u = 0; u < kLw; ++u) M = fmaxf(M, wst[0][hh][u]);
    float L = 0.0f;
#pragma unroll
    for (int u = 0; u < kLw; ++u)
      L += (wst[0][hh][u] == -__builtin_inff()) ? 0.0f : wst[1][hh][u] * __builtin_amdgcn_exp2f(wst[0][hh][u] - M);
    const float scl = (hh < p.G && L > 0.0f) ? ldexpf(1.0f / L, e) : 0.0f;
    // the wave's accumulators carry its operand scale 2^E_w
    fac[w][hh] = (wst[0][hh][w] == -__builtin_inff())
                     ? 0.0f
                     : __builtin_amdgcn_exp2f(wst[0][hh][w] - M - (float)wexp[w]) * scl;
    if (w == 0) {
      rec[hh] = M;
      rec[8 + hh] = L;
    }
  }
  __syncthreads();
  // A tile [head][128 m + k] (fp16): the waves' rows summed with their factors, in wave order;
  // thread = (row quad rq, channel k), rows 4 rq .. 4 rq + 3 = heads 4 (rq & 1) .. + 3 of modality rq / 2
  for (int idx = tid; idx < 6 * kD; idx += 64 * kLw) {
    const int rq = idx >> 7, k = idx & (kD - 1), m = rq >> 1, hq = rq & 1;
    float a[4] = {0.f, 0.f, 0.f, 0.f};
    if (mask & (1u << m)) {
#pragma unroll
      for (int w = 0; w < kLw; ++w) {
        const float4 f = *reinterpret_cast<const float4*>(&fac[w][4 * hq]);
        const float4 v = (m < 2) ? *reinterpret_cast<const float4*>(wacc + row_ofs(w, k, rq))
                                 : *reinterpret_cast<const float4*>(&ttx[w][0][0] + text_ofs(k, hq));
        a[0] = __builtin_fmaf(f.x, v.x, a[0]);
        a[1] = __builtin_fmaf(f.y, v.y, a[1]);
        a[2] = __builtin_fmaf(f.z, v.z, a[2]);
        a[3] = __builtin_fmaf(f.w, v.w, a[3]);
      }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) atile[4 * hq + i][m * kD + k] = (_Float16)a[i];
  }
  __syncthreads();
  floatx4 dacc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int m = 0; m < 3; ++m) {
    if (!(mask & (1u << m))) continue;
#pragma unroll
    for (int k4 = 0; k4 < 4; ++k4) {
      const int kk = 4 * m + k4;
      const half8 a = *reinterpret_cast<const half8*>(&atile[lane & 7][32 * kk + 8 * (lane >> 4)]);
      dacc = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, __builtin_bit_cast(half8, rb[kk]), dacc, 0, 0, 0);
    }
  }
  if (lane < 32) {
    const float scl = ldexpf(1.0f, -e);
#pragma unroll
    for (int i = 0; i < 4; ++i) rec[kRecHeader + (4 * (lane >> 4) + i) * kD + 16 * wave + (lane & 15)] = dacc[i] * scl;
  }
}

template <int kKB, int kVB>
void pick(bool tq, void (*&fn)(LadderDecodeArgs)) {
  fn = tq ? k_ladder_decode<kKB, kVB, true> : k_ladder_decode<kKB, kVB, false>;
}

}  // namespace

LadderPlan plan_ladder(int B, int H, int max_len) {
  const long units = (long)B * H;
  long target_groups = 256;
  if (const char* env = getenv("OKVQ_LADDER_GROUPS")) target_groups = std::max(1L, atol(env));
  long tps = ((long)max_len * units + target_groups - 1) / target_groups;
  tps = std::max(tps, (long)kLStep);
  tps = std::max(tps, ((long)max_len + kMaxSplits - 1) / kMaxSplits);
  tps = (tps + kLStep - 1) / kLStep * kLStep;
  LadderPlan pl;
  pl.tokens_per_split = (int)tps;
  pl.nsplit = max_len > 0 ? (int)((max_len + tps - 1) / tps) : 1;
  return pl;
}

size_t ladder_workspace_bytes(int B, int H, int max_len) {
  const int nsplit_max = std::max(1, std::min((max_len + kLStep - 1) / kLStep, kMaxSplits));
  return (size_t)B * H * nsplit_max * kRecFloats * sizeof(float);
}

hipError_t launch_ladder_decode(const LadderDecodeArgs& a0, int key_bits, int value_bits, bool tq, int B,
                                const LadderPlan& plan, float* out, hipStream_t s, hipEvent_t const* events) {
  LadderDecodeArgs a = a0;
  a.tps = plan.tokens_per_split;
  a.nsplit = plan.nsplit;
  void (*fn)(LadderDecodeArgs) = nullptr;
  const int key = 10 * key_bits + value_bits;
  switch (key) {
    case 22: pick<2, 2>(tq, fn); break;
    case 23: pick<2, 3>(tq, fn); break;
    case 24: pick<2, 4>(tq, fn); break;
    case 32: pick<3, 2>(tq, fn); break;
    case 33: pick<3, 3>(tq, fn); break;
    case 34: pick<3, 4>(tq, fn); break;
    case 42: pick<4, 2>(tq, fn); break;
    case 43: pick<4, 3>(tq, fn); break;
    case 44: pick<4, 4>(tq, fn); break;
    default: return hipErrorInvalidValue;
  }
  const dim3 grid(plan.nsplit, a.H, B), block(64 * kLw);
  if (events)
    hipExtLaunchKernelGGL(fn, grid, block, 0, s, events[0], events[1], 0, a);
  else
    hipLaunchKernelGGL(fn, grid, block, 0, s, a);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  return launch_decode_merge(a.ws, B, a.H, a.Hq, plan.nsplit, out, s, events ? events + 2 : nullptr);
}

}  // namespace okvq
