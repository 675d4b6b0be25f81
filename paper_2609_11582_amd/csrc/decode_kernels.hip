// Fused decode attention over the packed 2-bit cache (Eq. 1 with the codecs of Eq. 2, 4, 6).
//
// Split-K flash decoding. Work-group (split, KV head h, sequence b) = 4 waves; wave w takes the
// split's 32-token windows w, w + 4, ... and keeps its own online-softmax state; the waves are
// combined in LDS and one partial record per work-group is written. A second kernel merges the
// splits (log-sum-exp) and applies the inverse value rotation once per modality.
//
// What one wave does per window (all G <= 8 query heads of the KV head from one read):
//  * scores in the rotated key space (Sec. 2.3): s_i = n_i (q'.m_g + sum_c q'_c step_gc code_ic),
//    q' = H q sm_scale log2(e) computed once per work-group. The per-window bias q'.m_g is a
//    VALU dot product; the code term is one MFMA block-diagonal product: rows = 16 tokens, columns
//    0-7 = heads for tokens 0-15 of the window and columns 8-15 = the same heads for tokens
//    16-31 (K = 256 = two token rows of 128 channels), so a 16x16 tile holds all 32 tokens.
//    Codes enter the MFMA unchanged as fp16 subnormals: (dword & (3 << 2j)) is code * 2^(2j-24),
//    and the matching power of two is folded into the B operand q'_c step_gc 2^(k0 - 2j).
//  * online softmax in base 2 (running max per head, rescale only when it grows);
//  * values stay rotated (Sec. 2.3): two accumulator sets, rows 0-7 audio / 8-15 video heads and
//    rows 0-7 text heads; p n_v is masked per modality. B operands come from a 256-entry LDS
//    table mapping a code byte (one channel, four tokens) to four fp16 codebook values.
#include <algorithm>
#include <cstdlib>

#include "launch.hpp"

namespace okvq {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int kDecWaves = 4;
constexpr int kRecHeader = 32;                       // m[8], l[8], mask, pad
constexpr int kRecFloats = kRecHeader + 3 * 8 * kD;  // + acc[3 modalities][8 heads][128]
constexpr int kMinWps = 4;                           // fewest windows per split
constexpr int kMaxSplits = 1024;                     // most splits per (sequence, KV head)

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
  float* ws;
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

struct WinLoad {
  uint2 kc0, kc1;  // key codes: token r and 16 + r, bytes 8g .. 8g+7
  uint4 vc;        // value codes: the lane's 16 bytes of the window block
  uint2 nk, nv;    // key / value norms of the lane's 4 score rows
  uint32_t md;     // modality ids of those 4 tokens
  uint32_t stp;    // step of channels 32g + 2col, +1 (fp16 pair)
  uint32_t mnp;    // min of the same channels
};

__device__ __forceinline__ WinLoad load_window(const DecodeArgs& p, size_t seq, int b, int w, int lane) {
  const int col = lane & 15, g = lane >> 4, r = lane & 15;
  const int own_tok = 16 * (col >= 8 ? 1 : 0) + 4 * g;
  const int t0 = w * kW;
  const uint8_t* kc = p.k_codes + (seq * p.cap + t0) * 32;
  WinLoad d;
  d.kc0 = *reinterpret_cast<const uint2*>(kc + r * 32 + 8 * g);
  d.kc1 = *reinterpret_cast<const uint2*>(kc + (16 + r) * 32 + 8 * g);
  d.vc = *reinterpret_cast<const uint4*>(p.v_codes + (seq * (p.cap / kW) + w) * 1024 + 16 * lane);
  d.nk = *reinterpret_cast<const uint2*>(p.k_norm + seq * p.cap + t0 + own_tok);
  d.nv = *reinterpret_cast<const uint2*>(p.v_norm + seq * p.cap + t0 + own_tok);
  d.md = *reinterpret_cast<const uint32_t*>(p.modality + (size_t)b * p.cap + t0 + own_tok);
  const size_t meta = (seq * (p.cap / kW) + w) * kD + 32 * g + 2 * col;
  d.stp = *reinterpret_cast<const uint32_t*>(p.k_step + meta);
  d.mnp = *reinterpret_cast<const uint32_t*>(p.k_min + meta);
  return d;
}

__global__ __launch_bounds__(256, 2) void k_decode_split(DecodeArgs p) {
  __shared__ __attribute__((aligned(16))) uint2 vlut[256];
  __shared__ __attribute__((aligned(16))) float qs[kDecWaves][8][kD];          // per wave: rotated queries
  __shared__ __attribute__((aligned(16))) uint32_t meta[kDecWaves][2][kD / 2];  // per wave: step, min
  __shared__ float wstate[kDecWaves][2][8];                                     // m, l per wave and head
  __shared__ uint32_t wmask[kDecWaves];
  __shared__ __attribute__((aligned(16))) float wacc[kDecWaves][24][kD];        // rows 0-15 set 1, 16-23 set 2

  const int split = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, wave = tid >> 6, lane = lane_id();
  const int col = lane & 15, g = lane >> 4, hd = col & 7;
  const bool upper = col >= 8;  // this lane's QK column holds tokens 16..31 of the window
  const int len = min(p.seq_lens[b], p.cap);  // memory-safe if device and host lengths disagree
  const int nwin = (len + kW - 1) / kW;
  const int w_begin = split * p.wps;
  const int w_end = min(w_begin + p.wps, nwin);
  const size_t seq = (size_t)b * p.H + h;
  float* rec = p.ws + (seq * p.nsplit + split) * kRecFloats;
  if (w_begin >= w_end) {  // empty split (ragged batch): mark and leave
    if (tid < 8) {
      rec[tid] = -__builtin_inff();
      rec[8 + tid] = 0.0f;
    }
    if (tid == 0) reinterpret_cast<uint32_t*>(rec)[16] = 0u;
    return;
  }
  // first window's loads go out before the prologue
  const int w0 = w_begin + wave;
  WinLoad cur;
  if (w0 < w_end) cur = load_window(p, seq, b, w0, lane);

  {  // code-byte table: byte -> four fp16 codebook levels (tokens 0..3 of the byte)
    const uint32_t lv[4] = {p.cb01 & 0xffffu, p.cb01 >> 16, p.cb23 & 0xffffu, p.cb23 >> 16};
    vlut[tid] = make_uint2(lv[tid & 3] | (lv[(tid >> 2) & 3] << 16), lv[(tid >> 4) & 3] | (lv[tid >> 6] << 16));
  }

  // ---- per-wave query rotation: lane holds channels 16 (l % 8) + i of head l / 8 ----
  float qv[16];
  {
    const int hr = lane >> 3, cb = 16 * (lane & 7);
    if (hr < p.G) {
      const uint4* src = reinterpret_cast<const uint4*>(p.q + ((size_t)b * p.Hq + h * p.G + hr) * kD + cb);
      const uint4 a = src[0], c = src[1];
      const uint4 sg = *reinterpret_cast<const uint4*>(p.signs + cb);
      const uint32_t qw[8] = {a.x, a.y, a.z, a.w, c.x, c.y, c.z, c.w};
      const uint32_t sw[4] = {sg.x, sg.y, sg.z, sg.w};
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const float x = h2f((qw[i >> 1] >> (16 * (i & 1))) & 0xffffu);
        qv[i] = (sw[i >> 2] >> (8 * (i & 3) + 7)) & 1u ? -x : x;
      }
    } else {
#pragma unroll
      for (int i = 0; i < 16; ++i) qv[i] = 0.0f;
    }
#pragma unroll
    for (int hs = 1; hs < 16; hs <<= 1) {  // butterflies on channel bits 0..3 (in lane)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        if ((i & hs) == 0) {
          const float a = qv[i], c = qv[i + hs];
          qv[i] = a + c;
          qv[i + hs] = a - c;
        }
      }
    }
#pragma unroll
    for (int lb = 1; lb < 8; lb <<= 1) {  // channel bits 4..6 live in lane bits 0..2
      const bool hi = (lane & lb) != 0;
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const float o = __shfl_xor(qv[i], lb);
        qv[i] = hi ? o - qv[i] : qv[i] + o;
      }
    }
  }
  float amax = 0.0f;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    qv[i] *= p.qscale;
    amax = fmaxf(amax, fabsf(qv[i]));
  }
#pragma unroll
  for (int lb = 1; lb < 64; lb <<= 1) amax = fmaxf(amax, __shfl_xor(amax, lb));
  // power-of-two scale k0 keeps |q'_c step_c 2^(k0 - 2j)| <= 2^15 (|step| <= 2/3 + rounding)
  const int k0 = (amax > 0.0f) ? min(max(14 - ilogbf(amax), -60), 60) : 0;
  const float kscale = ldexpf(1.0f, 24 - k0);  // undoes 2^(k0 - 24) on the MFMA result
  {
    float4* dst = reinterpret_cast<float4*>(&qs[wave][lane >> 3][16 * (lane & 7)]);
#pragma unroll
    for (int i = 0; i < 4; ++i) dst[i] = make_float4(qv[4 * i], qv[4 * i + 1], qv[4 * i + 2], qv[4 * i + 3]);
  }
  wave_lds_sync();
  // qk[kk][i][hh] = q'[hd][32 g + slot channel] * 2^(k0 - shift of pair 4 (kk & 1) + i)
  float qk[4][4][2];
#pragma unroll
  for (int kk = 0; kk < 4; ++kk) {
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      const float4 v4 = *reinterpret_cast<const float4*>(&qs[wave][hd][32 * g + 16 * (kk >> 1) + 8 * hh + 4 * (kk & 1)]);
      const float vv[4] = {v4.x, v4.y, v4.z, v4.w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float x = (hd < p.G) ? vv[i] : 0.0f;
        qk[kk][i][hh] = ldexpf(x, k0 - code_shift(4 * (kk & 1) + i));
      }
    }
  }
  __syncthreads();  // code-byte table ready

  floatx4 acc1[8], acc2[8];
#pragma unroll
  for (int nb = 0; nb < 8; ++nb) {
    acc1[nb] = floatx4{0.f, 0.f, 0.f, 0.f};
    acc2[nb] = floatx4{0.f, 0.f, 0.f, 0.f};
  }
  float m_run = -__builtin_inff(), l_run = 0.0f;
  uint32_t seen = 0;  // modalities seen by this wave
  const int own_tok = 16 * (upper ? 1 : 0) + 4 * g;  // first of this lane's 4 score rows

  for (int w = w0; w < w_end; w += kDecWaves) {
    const int t0 = w * kW;
    WinLoad nxt = cur;
    if (w + kDecWaves < w_end) nxt = load_window(p, seq, b, w + kDecWaves, lane);  // prefetch

    // ---- per-window metadata through wave-private LDS ----
    meta[wave][0][16 * g + col] = cur.stp;
    meta[wave][1][16 * g + col] = cur.mnp;
    wave_lds_sync();

    // ---- B operands (q' step 2^(k0 - shift)) and the per-window bias q'.m, by shift class ----
    uint32_t bq[4][4];
    float bsum[5] = {0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const int dw = 16 * g + 8 * (kk >> 1) + 2 * (kk & 1);  // dword of channel 32g + 16(kk>>1) + 4(kk&1)
      const uint2 s0 = *reinterpret_cast<const uint2*>(&meta[wave][0][dw]);
      const uint2 s1 = *reinterpret_cast<const uint2*>(&meta[wave][0][dw + 4]);
      const uint2 m0 = *reinterpret_cast<const uint2*>(&meta[wave][1][dw]);
      const uint2 m1 = *reinterpret_cast<const uint2*>(&meta[wave][1][dw + 4]);
      const uint32_t sh[2][2] = {{s0.x, s0.y}, {s1.x, s1.y}};
      const uint32_t mh[2][2] = {{m0.x, m0.y}, {m1.x, m1.y}};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int cls = code_shift(4 * (kk & 1) + i) >> 1;
        float prod[2];
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
          const float stf = h2f((sh[hh][i >> 1] >> (16 * (i & 1))) & 0xffffu);
          const float mnf = h2f((mh[hh][i >> 1] >> (16 * (i & 1))) & 0xffffu);
          prod[hh] = qk[kk][i][hh] * stf;
          bsum[cls] = __builtin_fmaf(qk[kk][i][hh], mnf, bsum[cls]);
        }
        bq[kk][i] = pack2(prod[0], prod[1]);
      }
    }
    float bias = bsum[0] + 4.0f * bsum[1] + 16.0f * bsum[2] + 64.0f * bsum[3] + 256.0f * bsum[4];
    bias += __shfl_xor(bias, 16);
    bias += __shfl_xor(bias, 32);
    bias = ldexpf(bias, -k0);
    wave_lds_sync();  // metadata reads done before the next window overwrites it

    // ---- scores: 8 MFMAs, block-diagonal over the two token halves ----
    floatx4 sc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < 8; ++kk) {
      const bool mine = (kk >= 4) == upper;
      const half8 bop = mine ? h8(bq[kk & 3][0], bq[kk & 3][1], bq[kk & 3][2], bq[kk & 3][3]) : h8(0, 0, 0, 0);
      const half8 aop =
          (kk < 4) ? key_a_operand(cur.kc0.x, cur.kc0.y, kk & 3) : key_a_operand(cur.kc1.x, cur.kc1.y, kk & 3);
      sc = __builtin_amdgcn_mfma_f32_16x16x32_f16(aop, bop, sc, 0, 0, 0);
    }

    // ---- online softmax (base 2) ----
    const float nkf[4] = {h2f(cur.nk.x & 0xffffu), h2f(cur.nk.x >> 16), h2f(cur.nk.y & 0xffffu), h2f(cur.nk.y >> 16)};
    const float nvf[4] = {h2f(cur.nv.x & 0xffffu), h2f(cur.nv.x >> 16), h2f(cur.nv.y & 0xffffu), h2f(cur.nv.y >> 16)};
    float s[4];
    float wmax = -__builtin_inff();
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const bool valid = (t0 + own_tok + i) < len;
      s[i] = valid ? nkf[i] * __builtin_fmaf(sc[i], kscale, bias) : -__builtin_inff();
      wmax = fmaxf(wmax, s[i]);
    }
    wmax = fmaxf(wmax, __shfl_xor(wmax, 8));
    wmax = fmaxf(wmax, __shfl_xor(wmax, 16));
    wmax = fmaxf(wmax, __shfl_xor(wmax, 32));
    const float m_new = fmaxf(m_run, wmax);
    if (__any(m_new > m_run)) {
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
    float pv[4];
    uint32_t mods = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float pr = exp2f(s[i] - m_run);
      l_run += pr;
      const bool valid = (t0 + own_tok + i) < len;
      pv[i] = valid ? pr * nvf[i] : 0.0f;
      if (valid) mods |= 1u << ((cur.md >> (8 * i)) & 3u);
    }
    const bool any_av = __any((mods & 3u) != 0);
    const bool any_t = __any((mods & 4u) != 0);
    seen |= (__any((mods & 1u) != 0) ? 1u : 0u) | (__any((mods & 2u) != 0) ? 2u : 0u) | (any_t ? 4u : 0u);

    // ---- value B operands from the code-byte table ----
    const uint32_t vw[4] = {cur.vc.x, cur.vc.y, cur.vc.z, cur.vc.w};
    auto vop = [&](int nb) -> half8 {
      const uint32_t b0 = (vw[nb >> 2] >> (8 * (nb & 3))) & 0xffu;        // tokens 4g .. 4g+3
      const uint32_t b1 = (vw[2 + (nb >> 2)] >> (8 * (nb & 3))) & 0xffu;  // tokens 16+4g ..
      const uint2 x0 = vlut[b0];
      const uint2 x1 = vlut[b1];
      return h8(x0.x, x0.y, x1.x, x1.y);
    };

    if (any_av) {
      float keep[4], send[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const uint32_t mi = (cur.md >> (8 * i)) & 0xffu;
        const float pa = (mi == 0u) ? pv[i] : 0.0f;    // audio
        const float pvid = (mi == 1u) ? pv[i] : 0.0f;  // video
        keep[i] = upper ? pvid : pa;
        send[i] = upper ? pa : pvid;
      }
      const uint32_t k01 = pack2(keep[0], keep[1]), k23 = pack2(keep[2], keep[3]);
      const uint32_t r01 = swap8(pack2(send[0], send[1])), r23 = swap8(pack2(send[2], send[3]));
      const half8 aop = upper ? h8(r01, r23, k01, k23) : h8(k01, k23, r01, r23);
#pragma unroll
      for (int nb = 0; nb < 8; ++nb) acc1[nb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(aop, vop(nb), acc1[nb], 0, 0, 0);
    }
    if (any_t) {
      float keep[4], send[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const uint32_t mi = (cur.md >> (8 * i)) & 0xffu;
        const float pt = (mi == 2u) ? pv[i] : 0.0f;
        keep[i] = upper ? 0.0f : pt;
        send[i] = upper ? pt : 0.0f;
      }
      const uint32_t k01 = pack2(keep[0], keep[1]), k23 = pack2(keep[2], keep[3]);
      const uint32_t r01 = swap8(pack2(send[0], send[1])), r23 = swap8(pack2(send[2], send[3]));
      const half8 aop = upper ? h8(0, 0, 0, 0) : h8(k01, k23, r01, r23);
#pragma unroll
      for (int nb = 0; nb < 8; ++nb) acc2[nb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(aop, vop(nb), acc2[nb], 0, 0, 0);
    }
    cur = nxt;
  }

  // ---- combine the waves of the work-group ----
  l_run += __shfl_xor(l_run, 8);
  l_run += __shfl_xor(l_run, 16);
  l_run += __shfl_xor(l_run, 32);
  if (lane < 8) {
    wstate[wave][0][lane] = m_run;
    wstate[wave][1][lane] = l_run;
  }
  if (lane == 0) wmask[wave] = seen;
#pragma unroll
  for (int nb = 0; nb < 8; ++nb) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      wacc[wave][4 * g + i][16 * nb + col] = acc1[nb][i];
      if (g < 2) wacc[wave][16 + 4 * g + i][16 * nb + col] = acc2[nb][i];
    }
  }
  __syncthreads();
  uint32_t mask = 0;
#pragma unroll
  for (int w = 0; w < kDecWaves; ++w) mask |= wmask[w];
  if (tid < 8) {
    float M = -__builtin_inff();
#pragma unroll
    for (int w = 0; w < kDecWaves; ++w) M = fmaxf(M, wstate[w][0][tid]);
    float L = 0.0f;
#pragma unroll
    for (int w = 0; w < kDecWaves; ++w) {
      const float mw = wstate[w][0][tid];
      L += (mw == -__builtin_inff()) ? 0.0f : wstate[w][1][tid] * exp2f(mw - M);
    }
    rec[tid] = M;
    rec[8 + tid] = L;
  }
  if (tid == 0) reinterpret_cast<uint32_t*>(rec)[16] = mask;
  // acc rows: 0-7 audio, 8-15 video (set 1), 16-23 text (set 2) -> record [modality][head][ch]
  for (int idx = tid; idx < 24 * kD; idx += 256) {
    const int row = idx >> 7, ch = idx & 127;
    const int mod = row >> 3, head = row & 7;
    if (!(mask & (1u << mod))) continue;
    float M = -__builtin_inff();
#pragma unroll
    for (int w = 0; w < kDecWaves; ++w) M = fmaxf(M, wstate[w][0][head]);
    float a = 0.0f;
#pragma unroll
    for (int w = 0; w < kDecWaves; ++w) {
      const float mw = wstate[w][0][head];
      if (mw != -__builtin_inff()) a += wacc[w][row][ch] * exp2f(mw - M);
    }
    rec[kRecHeader + idx] = a;
  }
}

// ---- log-sum-exp merge over splits and the inverse value rotation, fused ----
// One block (256 threads) per (query head j, 16-channel slice of the output, sequence b):
//  1. M = max_s m_s, weights w_s = 2^(m_s - M), L = sum_s w_s l_s;
//  2. acc_m = sum_s w_s acc_{s,m} for the three modalities (all 128 rotated channels);
//  3. o_c = sum_m sum_k acc_m[k] R_m[k][c] / L for the slice's 16 channels (Sec. 2.3: once per
//     modality after aggregation, not once per cached value).
__global__ __launch_bounds__(256) void k_decode_merge(const float* __restrict__ ws, const int32_t* __restrict__ seq_lens,
                                                      const float* __restrict__ rot, int H, int Hq, int G, int wps,
                                                      int nsplit, int cap, float* __restrict__ out) {
  __shared__ float wts[kMaxSplits];
  __shared__ uint32_t msk[kMaxSplits];
  __shared__ float red[256];
  __shared__ __attribute__((aligned(16))) float part[8][3][kD];
  __shared__ float acc[3][kD];
  const int j = blockIdx.x, slice = blockIdx.y, b = blockIdx.z;
  const int h = j / G, hd = j % G;
  const int tid = threadIdx.x;
  const int len = min(seq_lens[b], cap);
  const int ns = min((len + kW - 1) / kW + wps - 1, nsplit * wps) / wps;  // non-empty splits
  const float* base = ws + ((size_t)b * H + h) * nsplit * kRecFloats;

  float mloc = -__builtin_inff();
  for (int s = tid; s < ns; s += 256) mloc = fmaxf(mloc, base[(size_t)s * kRecFloats + hd]);
  red[tid] = mloc;
  __syncthreads();
  for (int st = 128; st > 0; st >>= 1) {
    if (tid < st) red[tid] = fmaxf(red[tid], red[tid + st]);
    __syncthreads();
  }
  const float M = red[0];
  __syncthreads();
  float lloc = 0.0f;
  for (int s = tid; s < ns; s += 256) {
    const float* rs = base + (size_t)s * kRecFloats;
    const float ms = rs[hd];
    const float wgt = (ms == -__builtin_inff()) ? 0.0f : exp2f(ms - M);
    wts[s] = wgt;
    msk[s] = reinterpret_cast<const uint32_t*>(rs)[16];
    lloc += wgt * rs[8 + hd];
  }
  red[tid] = lloc;
  __syncthreads();
  for (int st = 128; st > 0; st >>= 1) {
    if (tid < st) red[tid] += red[tid + st];
    __syncthreads();
  }
  const float L = red[0];

  // 2. weighted sum over splits: thread = (channel quad, split group of 8)
  {
    const int qd = tid & 31, grp = tid >> 5;
    float4 a[3] = {make_float4(0.f, 0.f, 0.f, 0.f), make_float4(0.f, 0.f, 0.f, 0.f), make_float4(0.f, 0.f, 0.f, 0.f)};
    for (int s = grp; s < ns; s += 8) {
      const float wgt = wts[s];
      const uint32_t mk = msk[s];
      const float* rs = base + (size_t)s * kRecFloats + kRecHeader;
#pragma unroll
      for (int m = 0; m < 3; ++m) {
        if (mk & (1u << m)) {
          const float4 v = *reinterpret_cast<const float4*>(rs + (m * 8 + hd) * kD + 4 * qd);
          a[m].x += wgt * v.x;
          a[m].y += wgt * v.y;
          a[m].z += wgt * v.z;
          a[m].w += wgt * v.w;
        }
      }
    }
#pragma unroll
    for (int m = 0; m < 3; ++m) *reinterpret_cast<float4*>(&part[grp][m][4 * qd]) = a[m];
  }
  __syncthreads();
  for (int idx = tid; idx < 3 * kD; idx += 256) {
    const int m = idx >> 7, k = idx & 127;
    float sacc = 0.0f;
#pragma unroll
    for (int g8 = 0; g8 < 8; ++g8) sacc += part[g8][m][k];
    acc[m][k] = sacc;
  }
  __syncthreads();

  // 3. un-rotate the slice: thread = (channel of the slice, one of 16 k-slices of 24 (m, k) pairs)
  const int c = 16 * slice + (tid & 15), ks = tid >> 4;
  float o = 0.0f;
#pragma unroll 4
  for (int i = 0; i < 24; ++i) {
    const int idx = ks * 24 + i;
    const int m = idx >> 7, k = idx & 127;
    o = __builtin_fmaf(acc[m][k], rot[((size_t)m * kD + k) * kD + c], o);
  }
  red[tid] = o;
  __syncthreads();
  if (tid < 16) {
    float t = 0.0f;
#pragma unroll
    for (int q = 0; q < 16; ++q) t += red[q * 16 + tid];
    out[((size_t)b * Hq + j) * kD + 16 * slice + tid] = (L > 0.0f) ? t / L : 0.0f;
  }
}

DecodePlan plan_decode(int B, int H, int max_len) {
  const int nwin = (max_len + kW - 1) / kW;
  const long units = (long)B * H;
  long target_groups = 512;  // about two work-groups per compute unit
  if (const char* env = getenv("OKVQ_DECODE_GROUPS")) target_groups = std::max(1L, atol(env));
  int wps = (int)((nwin * units + target_groups - 1) / target_groups);
  wps = std::max(wps, kMinWps);
  wps = std::max(wps, (nwin + kMaxSplits - 1) / kMaxSplits);
  DecodePlan p;
  p.wins_per_split = wps;
  p.nsplit = nwin > 0 ? (nwin + wps - 1) / wps : 1;
  return p;
}

size_t decode_workspace_bytes(int B, int H, int /*Hq*/, int max_len) {
  const int nwin = (max_len + kW - 1) / kW;
  const int wps_min = std::max(kMinWps, (nwin + kMaxSplits - 1) / kMaxSplits);
  const int nsplit_max = nwin > 0 ? (nwin + wps_min - 1) / wps_min : 1;
  return (size_t)B * H * nsplit_max * kRecFloats * sizeof(float);
}

hipError_t launch_decode(const CacheView& c, const uint16_t* q, float sm_scale, float* out, void* ws,
                         const DecodePlan& plan, hipStream_t s, uint32_t cb01, uint32_t cb23, int /*max_len*/) {
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
  hipLaunchKernelGGL(k_decode_split, dim3(plan.nsplit, c.H, c.B), dim3(256), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_decode_merge, dim3(c.Hq, kD / 16, c.B), dim3(256), 0, s, a.ws, c.seq_lens, c.rot, c.H, c.Hq,
                     G, plan.wins_per_split, plan.nsplit, c.cap, out);
  return hipGetLastError();
}

}  // namespace okvq
