// Fused decode attention over the packed 2-bit cache (Eq. 1 with the codecs of Eq. 2, 4, 6).
//
// Split-K flash decoding in two launches. k_decode: work-group (split, KV head h, sequence b) =
// 8 waves; wave w takes the split's window pairs (2w + 16k, 2w + 16k + 1) and keeps its own
// online-softmax state. The waves are combined in LDS, the split's per-modality accumulators are
// un-rotated on MFMA (the inverse rotation is linear, so applying it per split and then merging
// equals applying it once per modality after aggregation, Sec. 2.3) and one normalized partial
// output per split is written. k_decode_merge combines the splits by log-sum-exp.
//
// What one wave does per window (all G <= 8 query heads of the KV head from one read):
//  * scores in the rotated key space (Sec. 2.3): s_i = n_i (q'.m_g + sum_c q'_c step_gc code_ic),
//    q' = H q sm_scale log2(e) computed once per work-group. The per-window bias q'.m_g is a
//    VALU dot product; the code term is an MFMA block-diagonal over a window pair: rows = 16
//    tokens, columns 0-7 = heads for window A and columns 8-15 = the same heads for window B
//    (K = 256 = the two windows' 128 channels), so each lane builds the query-times-step operand
//    of one window only, and two 16x16 tiles hold the pair's 64 tokens.
//    Codes enter the MFMA unchanged as fp16 subnormals: (dword & (3 << 2j)) is code * 2^(2j-24),
//    and the matching power of two is folded into the B operand q'_c step_gc 2^(k0 - 2j).
//  * online softmax in base 2 (running max per head, rescale only when it grows);
//  * values stay rotated (Sec. 2.3): two accumulator sets, rows 0-7 audio / 8-15 video heads and
//    rows 0-7 text heads; p n_v is masked per modality. B operands come from a 256-entry LDS
//    table mapping a code byte (one channel, four tokens) to four fp16 codebook values.
#include <hip/hip_ext.h>

#include <algorithm>
#include <cstdlib>

#include "launch.hpp"

namespace okvq {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int kDecWaves = 8;                         // waves per split work-group
constexpr int kRecHeader = 32;                       // m[8], l[8], pad
constexpr int kRecFloats = kRecHeader + 8 * kD;      // + o[8 heads][128], un-rotated, divided by l
constexpr int kATile = 3 * kD + 8;                   // fp16 row pitch of the un-rotation A tile
constexpr int kMinWps = 2 * kDecWaves;              // fewest windows per split (a pair per wave)
constexpr int kMaxSplits = 1024;                     // most splits per (sequence, KV head)
constexpr float kLazy = 8.0f;                        // log2 headroom of the lazily updated softmax max
constexpr float kPvScale = 1.0f / 256.0f;            // 2^-kLazy: keeps p n_v within fp16

struct DecodeArgs {
  const uint8_t* k_codes;
  const uint8_t* v_codes;
  const uint16_t* k_norm;
  const uint16_t* v_norm;
  const uint16_t* k_min;
  const uint16_t* k_step;
  const uint8_t* modality;
  const int32_t* seq_lens;
  const int8_t* signs;
  const uint16_t* q;
  const uint16_t* rot16t;  // [128][3][128] fp16: (c, m, k) -> R_m[k][c]
  float* ws;               // partial records [B][H][nsplit][kRecFloats]
  int H, Hq, G, cap, wps, nsplit;
  float qscale;      // sm_scale * log2(e) / sqrt(128)
  uint32_t cb01;     // fp16 codebook levels 0, 1 (low, high half)
  uint32_t cb23;     // fp16 codebook levels 2, 3
};

__device__ __forceinline__ half8 h8(uint32_t a, uint32_t b, uint32_t c, uint32_t d) {
  return __builtin_bit_cast(half8, make_uint4(a, b, c, d));
}
__device__ __forceinline__ uint32_t pack2(float lo, float hi) {
  return f2h(lo) | (f2h(hi) << 16);
}
// lane l <- lane l ^ 8 within each row of 16 lanes (DPP row rotate by 8)
__device__ __forceinline__ uint32_t swap8(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x128, 0xf, 0xf, false);
}
__device__ __forceinline__ float fswap8(float v) { return __builtin_bit_cast(float, swap8(__builtin_bit_cast(uint32_t, v))); }
// lane l <- lane l ^ 16 and lane l ^ 32 (permutes between rows of 16, no LDS access)
__device__ __forceinline__ float fxor16(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, v), 0x401f));
}
__device__ __forceinline__ float fxor32(float v) { return __shfl_xor(v, 32); }

// Scale exponent of the fp16-subnormal code extraction for pair slot j (0..7) of a dword.
__host__ __device__ constexpr int code_shift(int j) { return j <= 4 ? 2 * j : 2 * j - 10; }
// Channel (0..31 within the lane group's 32) of MFMA k-block kk (0..3), slot e (0..7).
__host__ __device__ constexpr int slot_channel(int kk, int e) {
  return 16 * (kk >> 1) + 8 * (e & 1) + 4 * (kk & 1) + (e >> 1);
}

// A operand (token row half) of k-block kk from the two code dwords of the lane group.
__device__ __forceinline__ half8 key_a_operand(uint32_t d0, uint32_t d1, int kk) {
  const uint32_t d = (kk >> 1) ? d1 : d0;
  if ((kk & 1) == 0) {
    return h8(d & 0x00030003u, d & 0x000c000cu, d & 0x00300030u, d & 0x00c000c0u);
  }
  const uint32_t s = d >> 10;
  return h8(d & 0x03000300u, s & 0x00030003u, s & 0x000c000cu, s & 0x00300030u);
}

// Loads of one window pair (A = wA, B = wA + 1) for one lane. Lanes 0-7 of every row of 16
// score window A, lanes 8-15 window B ("side"); both sides need both windows' key codes (the
// score MFMA is block-diagonal over the pair) and value codes (one PV MFMA per window).
struct PairLoad {
  uint2 ka0, ka1, kb0, kb1;  // key codes of tokens r and 16 + r of windows A, B (bytes 8g .. 8g+7)
  uint4 va, vb;              // value codes of windows A, B (the lane's 16 bytes of each block)
  uint2 nk0, nk1;            // key norms of the side window, tokens 4g .. 4g+3 and 16+4g .. 16+4g+3
  uint2 nv0, nv1;            // value norms of the same tokens
  uint32_t md0, md1;         // modality ids of the same tokens
  uint2 stp, mnp;            // step / min of channels 32g + 4 (col % 8) .. +3 of the side window
};

__device__ __forceinline__ PairLoad load_pair(const DecodeArgs& p, size_t seq, int b, int wA, bool hasB, int lane) {
  const int col = lane & 15, g = lane >> 4, r = lane & 15, side = col >> 3;
  const size_t nwcap = p.cap / kW;
  const uint8_t* kc = p.k_codes + seq * p.cap * 32;
  const uint8_t* vc = p.v_codes + seq * nwcap * 1024 + 16 * lane;
  PairLoad d;
  d.ka0 = *reinterpret_cast<const uint2*>(kc + (size_t)(kW * wA + r) * 32 + 8 * g);
  d.ka1 = *reinterpret_cast<const uint2*>(kc + (size_t)(kW * wA + 16 + r) * 32 + 8 * g);
  d.va = *reinterpret_cast<const uint4*>(vc + (size_t)wA * 1024);
  if (hasB) {
    d.kb0 = *reinterpret_cast<const uint2*>(kc + (size_t)(kW * (wA + 1) + r) * 32 + 8 * g);
    d.kb1 = *reinterpret_cast<const uint2*>(kc + (size_t)(kW * (wA + 1) + 16 + r) * 32 + 8 * g);
    d.vb = *reinterpret_cast<const uint4*>(vc + (size_t)(wA + 1) * 1024);
  } else {
    d.kb0 = d.kb1 = make_uint2(0, 0);
    d.vb = make_uint4(0, 0, 0, 0);
  }
  if (side == 0 || hasB) {
    const int wS = wA + side;
    const size_t t = seq * p.cap + (size_t)kW * wS + 4 * g;
    d.nk0 = *reinterpret_cast<const uint2*>(p.k_norm + t);
    d.nk1 = *reinterpret_cast<const uint2*>(p.k_norm + t + 16);
    d.nv0 = *reinterpret_cast<const uint2*>(p.v_norm + t);
    d.nv1 = *reinterpret_cast<const uint2*>(p.v_norm + t + 16);
    const uint8_t* md = p.modality + (size_t)b * p.cap + kW * wS + 4 * g;
    d.md0 = *reinterpret_cast<const uint32_t*>(md);
    d.md1 = *reinterpret_cast<const uint32_t*>(md + 16);
    const size_t mt = (seq * nwcap + wS) * kD + 32 * g + 4 * (col & 7);
    d.stp = *reinterpret_cast<const uint2*>(p.k_step + mt);
    d.mnp = *reinterpret_cast<const uint2*>(p.k_min + mt);
  } else {
    d.nk0 = d.nk1 = d.nv0 = d.nv1 = d.stp = d.mnp = make_uint2(0, 0);
    d.md0 = d.md1 = 0;
  }
  return d;
}

__device__ __forceinline__ half8 lut_op(const uint2* vlut, uint4 vc, int nb) {
  const uint32_t vw[4] = {vc.x, vc.y, vc.z, vc.w};
  const uint32_t b0 = (vw[nb >> 2] >> (8 * (nb & 3))) & 0xffu;        // tokens 4g .. 4g+3
  const uint32_t b1 = (vw[2 + (nb >> 2)] >> (8 * (nb & 3))) & 0xffu;  // tokens 16+4g .. 16+4g+3
  const uint2 x0 = vlut[b0];
  const uint2 x1 = vlut[b1];
  return h8(x0.x, x0.y, x1.x, x1.y);
}

typedef unsigned short ushort2v __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pkmax_u16(uint32_t a, uint32_t b) {
  return __builtin_bit_cast(uint32_t,
                            __builtin_elementwise_max(__builtin_bit_cast(ushort2v, a), __builtin_bit_cast(ushort2v, b)));
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int lb = 1; lb < 64; lb <<= 1) v = fmaxf(v, __shfl_xor(v, lb));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int lb = 1; lb < 64; lb <<= 1) v += __shfl_xor(v, lb);
  return v;
}

__global__ __launch_bounds__(64 * kDecWaves) void k_decode(DecodeArgs p) {
  __shared__ __attribute__((aligned(16))) uint2 vlut[256];
  __shared__ __attribute__((aligned(16))) float qs[8][kD + 4];                     // rotated queries (padded rows)
  __shared__ float amax_w[kDecWaves];
  __shared__ __attribute__((aligned(16))) uint32_t meta[kDecWaves][2][2][kD / 2];  // [wave][side][step, min]
  __shared__ float wstate[kDecWaves][2][8];                                        // m, l per wave and head
  __shared__ uint32_t wmask[kDecWaves];
  __shared__ uint32_t wnv[kDecWaves];                                              // value-norm maxima
  // per wave: accumulator rows for the combine (rows 0-15 set 1, 16-23 set 2); the merge reuses it
  __shared__ __attribute__((aligned(16))) float wacc[kDecWaves][24][kD + 4];  // padded rows: conflict-free
  __shared__ __attribute__((aligned(16))) _Float16 atile[8][kATile];         // merged rows, fp16
  __shared__ float hst[8];                                                   // per head: scale

  const int split = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, wave = tid >> 6, lane = lane_id();
  const int col = lane & 15, g = lane >> 4, hd = col & 7, side = col >> 3;
  const bool upper = side != 0;
  const size_t seq = (size_t)b * p.H + h;
  float* rec = p.ws + (seq * p.nsplit + split) * kRecFloats;
  const int w_begin = split * p.wps;
  const int w_plan = min(w_begin + p.wps, p.cap / kW);  // windows of this split by the plan
  const int wA0 = w_begin + 2 * wave;                    // this wave's pairs: (wA0 + 16 k, +1)

  // ---- every global load of the prologue goes out before any of them is used: the query rows
  // (waves 0-3), the first pair (speculatively: windows within the plan, the length is checked
  // later), and the sequence length ----
  const int hr = 2 * wave + (lane >> 5), c4 = 4 * (lane & 31);
  uint2 qraw = make_uint2(0, 0);
  uint32_t qsgn = 0;
  if (wave < 4 && hr < p.G) {
    qraw = *reinterpret_cast<const uint2*>(p.q + ((size_t)b * p.Hq + h * p.G + hr) * kD + c4);
    qsgn = *reinterpret_cast<const uint32_t*>(p.signs + c4);
  }
  PairLoad cur;
  if (wA0 < w_plan) cur = load_pair(p, seq, b, wA0, wA0 + 1 < w_plan, lane);
  const int len = min(p.seq_lens[b], p.cap);  // memory-safe if device and host lengths disagree
  const int nwin = (len + kW - 1) / kW;
  const int w_end = min(w_plan, nwin);
  if (w_begin >= w_end) {  // empty split (ragged batch): a header the merge skips
    if (tid < 8) {
      rec[tid] = -__builtin_inff();
      rec[8 + tid] = 0.0f;
    }
    return;
  }

  if (tid < 256) {  // code-byte table: byte -> four fp16 codebook levels (tokens 0..3 of the byte)
    const uint32_t lv[4] = {p.cb01 & 0xffffu, p.cb01 >> 16, p.cb23 & 0xffffu, p.cb23 >> 16};
    vlut[tid] = make_uint2(lv[tid & 3] | (lv[(tid >> 2) & 3] << 16), lv[(tid >> 4) & 3] | (lv[tid >> 6] << 16));
  }
  // ---- query rotation: wave w < 4 rotates heads 2w, 2w+1; lane holds channels c4 .. c4+3 ----
  float x[4] = {0.f, 0.f, 0.f, 0.f};
  if (wave < 4) {
    const uint32_t rr[2] = {qraw.x, qraw.y};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float v = h2f((rr[i >> 1] >> (16 * (i & 1))) & 0xffffu);
      x[i] = ((qsgn >> (8 * i + 7)) & 1u) ? -v : v;
    }
    {  // channel bits 0, 1 in lane
      const float a = x[0] + x[1], c = x[0] - x[1], d = x[2] + x[3], e = x[2] - x[3];
      x[0] = a + d;
      x[2] = a - d;
      x[1] = c + e;
      x[3] = c - e;
    }
#pragma unroll
    for (int lb = 1; lb < 32; lb <<= 1) {  // channel bits 2..6 are lane bits 0..4
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
  }
  __syncthreads();
  const float amax = fmaxf(fmaxf(amax_w[0], amax_w[1]), fmaxf(amax_w[2], amax_w[3]));  // waves 0-3 rotate
  // power-of-two scale k0 keeps |q'_c step_c 2^(k0 - 2j)| <= 2^15 (|step| <= 2/3 + rounding)
  const int k0 = (amax > 0.0f) ? min(max(14 - ilogbf(amax), -60), 60) : 0;
  const float kscale = ldexpf(1.0f, 24 - k0);  // undoes 2^(k0 - 24) on the MFMA result
  if (wave < 4) {  // store q' pre-scaled by 2^(k0 - shift(c)), shift(c) = code_shift(c % 8)
    float o[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) o[i] = ldexpf(x[i], k0 - code_shift((c4 + i) & 7));
    *reinterpret_cast<float4*>(&qs[hr][c4]) = make_float4(o[0], o[1], o[2], o[3]);
  }
  __syncthreads();

  floatx4 acc1[8], acc2[8];
#pragma unroll
  for (int nb = 0; nb < 8; ++nb) {
    acc1[nb] = floatx4{0.f, 0.f, 0.f, 0.f};
    acc2[nb] = floatx4{0.f, 0.f, 0.f, 0.f};
  }
  float m_run = -__builtin_inff(), l_run = 0.0f;
  uint32_t seen = 0;  // modalities seen by this wave
  uint32_t nvm = 0;   // largest value norm seen by this lane (two fp16 halves, non-negative)
  uint32_t* mw = &meta[wave][side][0][0];

  for (int wA = wA0; wA < w_end; wA += 2 * kDecWaves) {
    const bool hasB = wA + 1 < w_end;
    const int wS = wA + side;
    const bool side_ok = !upper || hasB;
    PairLoad nxt = cur;
    {
      const int wn = wA + 2 * kDecWaves;
      if (wn < w_end) nxt = load_pair(p, seq, b, wn, wn + 1 < w_end, lane);  // prefetch
    }

    // ---- side window metadata through wave-private LDS ----
    *reinterpret_cast<uint2*>(&mw[16 * g + 2 * (col & 7)]) = cur.stp;
    *reinterpret_cast<uint2*>(&mw[kD / 2 + 16 * g + 2 * (col & 7)]) = cur.mnp;
    wave_lds_sync();

    // ---- B operand (q' step 2^(k0 - shift)) and the bias q'.m of the side window ----
    uint32_t bq[4][4];
    float bsum[5] = {0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const int dw = 16 * g + 8 * (kk >> 1) + 2 * (kk & 1);  // dword of channel 32g + 16(kk>>1) + 4(kk&1)
      const uint2 s0 = *reinterpret_cast<const uint2*>(&mw[dw]);
      const uint2 s1 = *reinterpret_cast<const uint2*>(&mw[dw + 4]);
      const uint2 m0 = *reinterpret_cast<const uint2*>(&mw[kD / 2 + dw]);
      const uint2 m1 = *reinterpret_cast<const uint2*>(&mw[kD / 2 + dw + 4]);
      const uint32_t sh[2][2] = {{s0.x, s0.y}, {s1.x, s1.y}};
      const uint32_t mh[2][2] = {{m0.x, m0.y}, {m1.x, m1.y}};
      const float4 q0 = *reinterpret_cast<const float4*>(&qs[hd][32 * g + 16 * (kk >> 1) + 4 * (kk & 1)]);
      const float4 q1 = *reinterpret_cast<const float4*>(&qs[hd][32 * g + 16 * (kk >> 1) + 8 + 4 * (kk & 1)]);
      const float qk[2][4] = {{q0.x, q0.y, q0.z, q0.w}, {q1.x, q1.y, q1.z, q1.w}};  // zero rows for heads >= G
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int cls = code_shift(4 * (kk & 1) + i) >> 1;
        float prod[2];
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
          const float stf = h2f((sh[hh][i >> 1] >> (16 * (i & 1))) & 0xffffu);
          const float mnf = h2f((mh[hh][i >> 1] >> (16 * (i & 1))) & 0xffffu);
          prod[hh] = qk[hh][i] * stf;
          bsum[cls] = __builtin_fmaf(qk[hh][i], mnf, bsum[cls]);
        }
        bq[kk][i] = pack2(prod[0], prod[1]);
      }
    }
    float bias = bsum[0] + 4.0f * bsum[1] + 16.0f * bsum[2] + 64.0f * bsum[3] + 256.0f * bsum[4];
    bias += fxor16(bias);
    bias += fxor32(bias);
    bias = ldexpf(bias, -k0);
    wave_lds_sync();  // metadata reads done before the next pair overwrites it

    // ---- scores: two 16-token tiles, each 8 MFMAs block-diagonal over the pair ----
    floatx4 sc0 = {0.f, 0.f, 0.f, 0.f}, sc1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < 8; ++kk) {
      const bool mine = (kk >= 4) == upper;
      const half8 bop = mine ? h8(bq[kk & 3][0], bq[kk & 3][1], bq[kk & 3][2], bq[kk & 3][3]) : h8(0, 0, 0, 0);
      const half8 a0 = (kk < 4) ? key_a_operand(cur.ka0.x, cur.ka0.y, kk & 3) : key_a_operand(cur.kb0.x, cur.kb0.y, kk & 3);
      const half8 a1 = (kk < 4) ? key_a_operand(cur.ka1.x, cur.ka1.y, kk & 3) : key_a_operand(cur.kb1.x, cur.kb1.y, kk & 3);
      sc0 = __builtin_amdgcn_mfma_f32_16x16x32_f16(a0, bop, sc0, 0, 0, 0);
      sc1 = __builtin_amdgcn_mfma_f32_16x16x32_f16(a1, bop, sc1, 0, 0, 0);
    }

    // ---- online softmax (base 2) over the pair's 64 tokens ----
    const uint32_t nkw[4] = {cur.nk0.x, cur.nk0.y, cur.nk1.x, cur.nk1.y};
    const uint32_t nvw[4] = {cur.nv0.x, cur.nv0.y, cur.nv1.x, cur.nv1.y};
    nvm = pkmax_u16(nvm, pkmax_u16(pkmax_u16(nvw[0], nvw[1]), pkmax_u16(nvw[2], nvw[3])));
    float s[8];
    float wmax = -__builtin_inff();
#pragma unroll
    for (int e = 0; e < 8; ++e) {  // e = 4 t + i: token 16 t + 4 g + i of the side window
      const int t = e >> 2, i = e & 3;
      const bool valid = side_ok && (kW * wS + 16 * t + 4 * g + i) < len;
      const float nkf = h2f((nkw[e >> 1] >> (16 * (e & 1))) & 0xffffu);
      const float raw = t ? sc1[i] : sc0[i];
      s[e] = valid ? nkf * __builtin_fmaf(raw, kscale, bias) : -__builtin_inff();
      wmax = fmaxf(wmax, s[e]);
    }
    wmax = fmaxf(wmax, fswap8(wmax));
    wmax = fmaxf(wmax, fxor16(wmax));
    wmax = fmaxf(wmax, fxor32(wmax));
    // lazy rescale: the reference m_run moves only when the max exceeds it by more than 2^8, so
    // p = 2^(s - m_run) <= 2^8; p n_v is stored as fp16 times 2^-8 (undone in the epilogue)
    if (__any(wmax > m_run + kLazy)) {
      const float m_new = fmaxf(m_run, wmax);
      const float alpha = exp2f(m_run - m_new);
      l_run *= alpha;
      float arow[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) arow[i] = __shfl(alpha, (4 * g + i) & 7);
#pragma unroll
      for (int nb = 0; nb < 8; ++nb) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          acc1[nb][i] *= arow[i];
          acc2[nb][i] *= arow[i];
        }
      }
      m_run = m_new;
    }
    float pv[8];
    uint32_t mods = 0;
    const uint32_t mdw[2] = {cur.md0, cur.md1};
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int t = e >> 2, i = e & 3;
      const float pr = exp2f(s[e] - m_run);
      l_run += pr;
      const bool valid = side_ok && (kW * wS + 16 * t + 4 * g + i) < len;
      const float nvf = h2f((nvw[e >> 1] >> (16 * (e & 1))) & 0xffffu);
      pv[e] = valid ? pr * nvf * kPvScale : 0.0f;
      if (valid) mods |= 1u << ((mdw[t] >> (8 * i)) & 3u);
    }
    const bool any_av = __any((mods & 3u) != 0);
    const bool any_t = __any((mods & 4u) != 0);
    seen |= (__any((mods & 1u) != 0) ? 1u : 0u) | (__any((mods & 2u) != 0) ? 2u : 0u) | (any_t ? 4u : 0u);

    // ---- values: one PV MFMA per window and 16-channel block, A = masked p n_v ----
    if (any_av) {  // set 1: rows 0-7 audio heads, rows 8-15 video heads
      uint32_t keep[4], send[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float kv[2], sv[2];
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          const int e = 2 * q + u, t = e >> 2, i = e & 3;
          const uint32_t mi = (mdw[t] >> (8 * i)) & 0xffu;
          const float pa = (mi == 0u) ? pv[e] : 0.0f;
          const float pvid = (mi == 1u) ? pv[e] : 0.0f;
          kv[u] = upper ? pvid : pa;
          sv[u] = upper ? pa : pvid;
        }
        keep[q] = pack2(kv[0], kv[1]);
        send[q] = swap8(pack2(sv[0], sv[1]));
      }
      const half8 opA = upper ? h8(send[0], send[1], send[2], send[3]) : h8(keep[0], keep[1], keep[2], keep[3]);
      const half8 opB = upper ? h8(keep[0], keep[1], keep[2], keep[3]) : h8(send[0], send[1], send[2], send[3]);
#pragma unroll
      for (int nb = 0; nb < 8; ++nb) {
        acc1[nb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(opA, lut_op(vlut, cur.va, nb), acc1[nb], 0, 0, 0);
        acc1[nb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(opB, lut_op(vlut, cur.vb, nb), acc1[nb], 0, 0, 0);
      }
    }
    if (any_t) {  // set 2: rows 0-7 text heads
      uint32_t keep[4], recv[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float kv[2];
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          const int e = 2 * q + u, t = e >> 2, i = e & 3;
          const uint32_t mi = (mdw[t] >> (8 * i)) & 0xffu;
          kv[u] = (mi == 2u) ? pv[e] : 0.0f;
        }
        keep[q] = pack2(kv[0], kv[1]);
        recv[q] = swap8(keep[q]);
      }
      const half8 zero = h8(0, 0, 0, 0);
      const half8 opA = upper ? zero : h8(keep[0], keep[1], keep[2], keep[3]);
      const half8 opB = upper ? zero : h8(recv[0], recv[1], recv[2], recv[3]);
#pragma unroll
      for (int nb = 0; nb < 8; ++nb) {
        acc2[nb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(opA, lut_op(vlut, cur.va, nb), acc2[nb], 0, 0, 0);
        acc2[nb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(opB, lut_op(vlut, cur.vb, nb), acc2[nb], 0, 0, 0);
      }
    }
    cur = nxt;
  }

  // ---- epilogue. This wave's slice of the inverse-rotation table (output channels 16 wave ..
  // 16 wave + 15, all 384 (modality, k) rows) as MFMA B operands, loaded first so that the
  // combine below hides the latency ----
  uint4 rb[12];
  {
    const uint4* rp = reinterpret_cast<const uint4*>(p.rot16t) + (size_t)(16 * wave + (lane & 15)) * 48 + (lane >> 4);
#pragma unroll
    for (int kk = 0; kk < 12; ++kk) rb[kk] = rp[4 * kk];
  }

  // ---- combine the waves of the work-group ----
  l_run += __shfl_xor(l_run, 8);
  l_run += __shfl_xor(l_run, 16);
  l_run += __shfl_xor(l_run, 32);
#pragma unroll
  for (int lb = 1; lb < 64; lb <<= 1) nvm = pkmax_u16(nvm, (uint32_t)__shfl_xor((int)nvm, lb));
  if (lane < 8) {
    wstate[wave][0][lane] = m_run;
    wstate[wave][1][lane] = l_run;
  }
  if (lane == 0) {
    wmask[wave] = seen;
    wnv[wave] = max(nvm & 0xffffu, nvm >> 16);
  }
  __syncthreads();
  uint32_t mask = 0, nmax = 0;
#pragma unroll
  for (int w = 0; w < kDecWaves; ++w) {
    mask |= wmask[w];
    nmax = max(nmax, wnv[w]);
  }
  // Every merged row divided by its softmax sum is a convex combination of n_v cb vectors, so
  // its entries are below n_max * 2^-2.9 (the largest codebook level is 0.1335): the factor
  // 2^e / L with e = 15 - ilogb(n_max) keeps the fp16 A tile below 2^13.
  const float nmf = h2f(nmax);
  const int e = (nmf > 0.0f) ? 15 - min(max(ilogbf(nmf), -30), 20) : 0;
  float frow[4];  // 2^(m_wave - M) for this lane's accumulator rows (head (4g + i) % 8)
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int head = (4 * g + i) & 7;
    float M = -__builtin_inff();
#pragma unroll
    for (int w = 0; w < kDecWaves; ++w) M = fmaxf(M, wstate[w][0][head]);
    const float mwv = wstate[wave][0][head];
    frow[i] = (mwv == -__builtin_inff()) ? 0.0f : exp2f(mwv - M) * (1.0f / kPvScale);
  }
  if (mask & 3u) {
#pragma unroll
    for (int nb = 0; nb < 8; ++nb)
#pragma unroll
      for (int i = 0; i < 4; ++i) wacc[wave][4 * g + i][16 * nb + col] = acc1[nb][i] * frow[i];
  }
  if ((mask & 4u) && g < 2) {
#pragma unroll
    for (int nb = 0; nb < 8; ++nb)
#pragma unroll
      for (int i = 0; i < 4; ++i) wacc[wave][16 + 4 * g + i][16 * nb + col] = acc2[nb][i] * frow[i];
  }
  if (tid < 8) {
    float M = -__builtin_inff();
#pragma unroll
    for (int w = 0; w < kDecWaves; ++w) M = fmaxf(M, wstate[w][0][tid]);
    float L = 0.0f;
#pragma unroll
    for (int w = 0; w < kDecWaves; ++w) {
      const float mwv = wstate[w][0][tid];
      L += (mwv == -__builtin_inff()) ? 0.0f : wstate[w][1][tid] * exp2f(mwv - M);
    }
    hst[tid] = (tid < p.G && L > 0.0f) ? ldexpf(1.0f / L, e) : 0.0f;
    rec[tid] = M;
    rec[8 + tid] = L;
  }
  __syncthreads();
  // acc rows 0-7 audio, 8-15 video (set 1), 16-23 text (set 2), summed over the waves and scaled
  // -> A tile [head][128 m + k] (fp16)
  for (int idx4 = tid; idx4 < 24 * kD / 4; idx4 += 64 * kDecWaves) {
    const int row = idx4 >> 5, c4 = (idx4 & 31) * 4, m = row >> 3, head = row & 7;
    if (!(mask & (1u << m))) continue;
    float4 a = *reinterpret_cast<const float4*>(&wacc[0][row][c4]);
#pragma unroll
    for (int w = 1; w < kDecWaves; ++w) {
      const float4 v = *reinterpret_cast<const float4*>(&wacc[w][row][c4]);
      a.x += v.x;
      a.y += v.y;
      a.z += v.z;
      a.w += v.w;
    }
    const float f = hst[head];
    *reinterpret_cast<uint2*>(&atile[head][m * kD + c4]) = make_uint2(pack2(a.x * f, a.y * f), pack2(a.z * f, a.w * f));
  }
  __syncthreads();
  // ---- inverse rotation on MFMA, once per present modality: wave w computes channels
  // c = 16 w .. 16 w + 15 of o[head][c] = sum_m sum_k A[head][128 m + k] R_m[k][c]. A rows 8-15
  // (lanes whose row is >= 8) only feed output rows that are not stored. ----
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
    const float sc = ldexpf(1.0f, -e);
#pragma unroll
    for (int i = 0; i < 4; ++i) rec[kRecHeader + (4 * (lane >> 4) + i) * kD + 16 * wave + (lane & 15)] = dacc[i] * sc;
  }
}

// ---- merge over splits: o = sum_s 2^(M_s - M) L_s o_s / sum_s 2^(M_s - M) L_s (log-sum-exp) ----
// One work-group of 256 threads per (query head j, sequence b): thread (split group sg, channel
// quad q4) sums the splits s = sg (mod 8). Every load is issued before any is used; empty splits
// carry M = -inf and are skipped (their outputs were never written).
constexpr int kMergeThreads = 256;
constexpr int kMergeUnroll = 8;  // splits per thread held in registers at once

__global__ __launch_bounds__(kMergeThreads) void k_decode_merge(const float* __restrict__ ws, int H, int Hq, int G,
                                                                int nsplit, float* __restrict__ out) {
  __shared__ float red[2][kMergeThreads / 64];
  __shared__ __attribute__((aligned(16))) float4 part[8][32];
  const int j = blockIdx.x, b = blockIdx.y;
  const int h = j / G, hd = j % G;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int q4 = tid & 31, sg = tid >> 5;
  const float* base = ws + ((size_t)b * H + h) * nsplit * kRecFloats;

  float4 o = make_float4(0.f, 0.f, 0.f, 0.f);
  float M = -__builtin_inff(), L = 0.0f;
  // running (M, L, o) over this thread's splits: one pass, all loads of a chunk up front
  for (int s0 = sg; s0 < nsplit; s0 += 8 * kMergeUnroll) {
    float ms[kMergeUnroll], ls[kMergeUnroll];
    float4 v[kMergeUnroll];
#pragma unroll
    for (int u = 0; u < kMergeUnroll; ++u) {
      const int s = s0 + 8 * u;
      const float* rs = base + (size_t)min(s, nsplit - 1) * kRecFloats;
      ms[u] = (s < nsplit) ? rs[hd] : -__builtin_inff();
      ls[u] = rs[8 + hd];
      v[u] = *reinterpret_cast<const float4*>(rs + kRecHeader + hd * kD + 4 * q4);
    }
    float mc = M;
#pragma unroll
    for (int u = 0; u < kMergeUnroll; ++u) mc = fmaxf(mc, ms[u]);
    if (mc == -__builtin_inff()) continue;
    const float a = exp2f(M - mc);  // M = -inf -> 0
    L *= a;
    o.x *= a;
    o.y *= a;
    o.z *= a;
    o.w *= a;
#pragma unroll
    for (int u = 0; u < kMergeUnroll; ++u) {
      if (ms[u] == -__builtin_inff()) continue;
      const float w = exp2f(ms[u] - mc) * ls[u];
      L += w;
      o.x = __builtin_fmaf(w, v[u].x, o.x);
      o.y = __builtin_fmaf(w, v[u].y, o.y);
      o.z = __builtin_fmaf(w, v[u].z, o.z);
      o.w = __builtin_fmaf(w, v[u].w, o.w);
    }
    M = mc;
  }
  // combine the 8 split groups: global max, then rescale
  float mw = wave_max(M);
  if (lane == 0) red[0][wave] = mw;
  __syncthreads();
  float Mt = red[0][0];
#pragma unroll
  for (int w = 1; w < kMergeThreads / 64; ++w) Mt = fmaxf(Mt, red[0][w]);
  const float a = (M == -__builtin_inff()) ? 0.0f : exp2f(M - Mt);
  // L is the same for every channel quad of a split group: count it once per group
  float lw = (q4 == 0) ? L * a : 0.0f;
  lw = wave_sum(lw);
  if (lane == 0) red[1][wave] = lw;
  part[sg][q4] = make_float4(o.x * a, o.y * a, o.z * a, o.w * a);
  __syncthreads();
  if (tid < 32) {
    float Lt = 0.0f;
#pragma unroll
    for (int w = 0; w < kMergeThreads / 64; ++w) Lt += red[1][w];
    float4 t = part[0][tid];
#pragma unroll
    for (int g = 1; g < 8; ++g) {
      const float4 u = part[g][tid];
      t.x += u.x;
      t.y += u.y;
      t.z += u.z;
      t.w += u.w;
    }
    const float inv = (Lt > 0.0f) ? 1.0f / Lt : 0.0f;
    *reinterpret_cast<float4*>(out + ((size_t)b * Hq + j) * kD + 4 * tid) =
        make_float4(t.x * inv, t.y * inv, t.z * inv, t.w * inv);
  }
}

DecodePlan plan_decode(int B, int H, int max_len) {
  const int nwin = (max_len + kW - 1) / kW;
  const long units = (long)B * H;
  long target_groups = 256;  // one work-group per compute unit
  if (const char* env = getenv("OKVQ_DECODE_GROUPS")) target_groups = std::max(1L, atol(env));
  int wps = (int)((nwin * units + target_groups - 1) / target_groups);
  wps = std::max(wps, kMinWps);
  wps = std::max(wps, (nwin + kMaxSplits - 1) / kMaxSplits);
  wps = (wps + 1) / 2 * 2;  // whole window pairs
  DecodePlan p;
  p.wins_per_split = wps;
  p.nsplit = nwin > 0 ? (nwin + wps - 1) / wps : 1;
  return p;
}

static size_t record_bytes(int B, int H, int max_len) {
  const int nwin = (max_len + kW - 1) / kW;
  const int nsplit_max = nwin > 0 ? (nwin + kMinWps - 1) / kMinWps : 1;
  return (size_t)B * H * std::min(nsplit_max, kMaxSplits) * kRecFloats * sizeof(float);
}

size_t decode_workspace_bytes(int B, int H, int /*Hq*/, int max_len) { return record_bytes(B, H, max_len); }

hipError_t launch_decode(const CacheView& c, const uint16_t* q, float sm_scale, float* out, void* ws,
                         const DecodePlan& plan, hipStream_t s, uint32_t cb01, uint32_t cb23, int /*max_len*/,
                         hipEvent_t const* events) {
  const int G = c.Hq / c.H;
  DecodeArgs a;
  a.k_codes = c.k_codes;
  a.v_codes = c.v_codes;
  a.k_norm = c.k_norm;
  a.v_norm = c.v_norm;
  a.k_min = c.k_min;
  a.k_step = c.k_step;
  a.modality = c.modality;
  a.seq_lens = c.seq_lens;
  a.signs = c.signs;
  a.q = q;
  a.rot16t = c.rot16t;
  a.ws = static_cast<float*>(ws);
  a.H = c.H;
  a.Hq = c.Hq;
  a.G = G;
  a.cap = c.cap;
  a.wps = plan.wins_per_split;
  a.nsplit = plan.nsplit;
  a.qscale = sm_scale * 1.4426950408889634f * 0.08838834764831845f;
  a.cb01 = cb01;
  a.cb23 = cb23;
  hipError_t e;
  if (events) {  // events bound to the two dispatches: start and end of each kernel's execution
    hipExtLaunchKernelGGL(k_decode, dim3(plan.nsplit, c.H, c.B), dim3(64 * kDecWaves), 0, s, events[0], events[1], 0,
                          a);
  } else {
    hipLaunchKernelGGL(k_decode, dim3(plan.nsplit, c.H, c.B), dim3(64 * kDecWaves), 0, s, a);
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (events) {
    hipExtLaunchKernelGGL(k_decode_merge, dim3(c.Hq, c.B), dim3(kMergeThreads), 0, s, events[2], events[3], 0,
                          static_cast<const float*>(a.ws), c.H, c.Hq, G, plan.nsplit, out);
  } else {
    hipLaunchKernelGGL(k_decode_merge, dim3(c.Hq, c.B), dim3(kMergeThreads), 0, s, a.ws, c.H, c.Hq, G, plan.nsplit,
                       out);
  }
  return hipGetLastError();
}

// Inverse-rotation table: element (c, m, k) = fp16(R_m[k][c]), one thread per pair of k.
__global__ __launch_bounds__(256) void k_prepare_rotation(const float* __restrict__ rot, uint16_t* __restrict__ rot16t) {
  const int idx = blockIdx.x * 256 + threadIdx.x;
  if (idx >= kD * 3 * kD / 2) return;
  const int c = idx / (3 * kD / 2), r = idx % (3 * kD / 2), m = r / (kD / 2), k = 2 * (r % (kD / 2));
  const float lo = rot[((size_t)m * kD + k) * kD + c], hi = rot[((size_t)m * kD + k + 1) * kD + c];
  reinterpret_cast<uint32_t*>(rot16t)[idx] = f2h(lo) | (f2h(hi) << 16);
}

hipError_t launch_prepare_rotation(const float* rot, uint16_t* rot16t, hipStream_t s) {
  hipLaunchKernelGGL(k_prepare_rotation, dim3(kD * 3 * kD / 2 / 256), dim3(256), 0, s, rot, rot16t);
  return hipGetLastError();
}

}  // namespace okvq
