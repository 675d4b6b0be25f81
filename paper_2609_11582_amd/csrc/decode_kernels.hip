// Fused decode attention over the packed 2-bit cache (Eq. 1 with the codecs of Eq. 2, 4, 6).
//
// Split-K flash decoding. Work-group (split, KV head h, sequence b) = 4 waves; wave w takes the
// split's 32-token windows w, w + 4, ... and keeps its own online-softmax state; the waves are
// combined in LDS and one partial record per work-group is written. Two small kernels follow:
// a log-sum-exp merge over splits per (query head, modality) and the inverse value rotation.
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
#include "launch.hpp"

namespace okvq {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int kDecWaves = 4;
constexpr int kRecHeader = 32;                       // m[8], l[8], mask, pad
constexpr int kRecFloats = kRecHeader + 3 * 8 * kD;  // + acc[3 modalities][8 heads][128]
constexpr int kMinWps = 4;                           // fewest windows per split

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

__global__ __launch_bounds__(256) void k_decode_split(DecodeArgs p) {
  __shared__ __attribute__((aligned(16))) float qs[8][kD];
  __shared__ __attribute__((aligned(16))) uint2 vlut[256];
  __shared__ __attribute__((aligned(16))) uint32_t meta[kDecWaves][2][kD / 2];  // per wave: step, min (fp16 pairs)
  __shared__ float red[256];
  __shared__ float wstate[kDecWaves][2][8];        // m, l per wave and head
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

  // ---- prologue: rotated queries, code LUT ----
  {
    const int j = tid >> 5, c4 = (tid & 31) * 4;
    float v[4] = {0.f, 0.f, 0.f, 0.f};
    if (j < p.G) {
      const uint2 raw = *reinterpret_cast<const uint2*>(p.q + ((size_t)b * p.Hq + h * p.G + j) * kD + c4);
      const uint32_t sw = *reinterpret_cast<const uint32_t*>(p.signs + c4);
      const uint32_t rr[2] = {raw.x, raw.y};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float x = h2f((rr[i >> 1] >> (16 * (i & 1))) & 0xffffu);
        const int s8 = (int)(int8_t)((sw >> (8 * i)) & 0xffu);
        v[i] = s8 < 0 ? -x : x;
      }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) qs[j][c4 + i] = v[i];
    const uint32_t lo = p.cb01 & 0xffffu, l1 = p.cb01 >> 16, l2 = p.cb23 & 0xffffu, l3 = p.cb23 >> 16;
    const uint32_t lv[4] = {lo, l1, l2, l3};
    vlut[tid] = make_uint2(lv[tid & 3] | (lv[(tid >> 2) & 3] << 16), lv[(tid >> 4) & 3] | (lv[tid >> 6] << 16));
  }
  __syncthreads();
#pragma unroll
  for (int hs = 1; hs < kD; hs <<= 1) {  // Walsh-Hadamard butterflies on the 8 query rows
#pragma unroll
    for (int rep = 0; rep < 2; ++rep) {
      const int pidx = tid + 256 * rep;  // 512 pairs = 8 rows x 64
      const int row = pidx >> 6, pi = pidx & 63;
      const int j0 = (pi / hs) * 2 * hs + (pi % hs);
      const float a = qs[row][j0], c = qs[row][j0 + hs];
      qs[row][j0] = a + c;
      qs[row][j0 + hs] = a - c;
    }
    __syncthreads();
  }
  float amax = 0.0f;
  for (int i = tid; i < 8 * kD; i += 256) {
    const float x = qs[i >> 7][i & 127] * p.qscale;
    qs[i >> 7][i & 127] = x;
    amax = fmaxf(amax, fabsf(x));
  }
  red[tid] = amax;
  __syncthreads();
  for (int s = 128; s > 0; s >>= 1) {
    if (tid < s) red[tid] = fmaxf(red[tid], red[tid + s]);
    __syncthreads();
  }
  amax = red[0];
  // power-of-two scale k0 keeps |q'_c step_c 2^(k0 - 2j)| <= 2^15 (|step| <= 2/3 + rounding)
  const int k0 = (amax > 0.0f) ? min(max(14 - ilogbf(amax), -60), 60) : 0;
  const float kscale = ldexpf(1.0f, 24 - k0);  // undoes 2^(k0 - 24) on the MFMA result

  // per-lane query registers: qk (scaled, for the B operand) and qb (for the bias)
  float qk[32], qb[32];
#pragma unroll
  for (int kk = 0; kk < 4; ++kk) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int ch = 32 * g + slot_channel(kk, e);
      const int j = 4 * (kk & 1) + (e >> 1);
      const float x = (hd < p.G) ? qs[hd][ch] : 0.0f;
      qb[kk * 8 + e] = x;
      qk[kk * 8 + e] = ldexpf(x, k0 - code_shift(j));
    }
  }

  floatx4 acc1[8], acc2[8];
#pragma unroll
  for (int nb = 0; nb < 8; ++nb) {
    acc1[nb] = floatx4{0.f, 0.f, 0.f, 0.f};
    acc2[nb] = floatx4{0.f, 0.f, 0.f, 0.f};
  }
  float m_run = -__builtin_inff(), l_run = 0.0f;
  uint32_t seen = 0;  // modalities seen by this wave

  const uint8_t* kc_base = p.k_codes + seq * p.cap * 32;
  const uint8_t* vc_base = p.v_codes + seq * (p.cap / kW) * 1024;
  const uint16_t* kn_base = p.k_norm + seq * p.cap;
  const uint16_t* vn_base = p.v_norm + seq * p.cap;
  const uint16_t* st_base = p.k_step + seq * (p.cap / kW) * kD;
  const uint16_t* mn_base = p.k_min + seq * (p.cap / kW) * kD;
  const uint8_t* md_base = p.modality + (size_t)b * p.cap;
  const int r = lane & 15;
  const int own_tok = 16 * (upper ? 1 : 0) + 4 * g;  // first of this lane's 4 score rows

  for (int w = w_begin + wave; w < w_end; w += kDecWaves) {
    const int t0 = w * kW;
    // ---- loads ----
    const uint2 kc0 = *reinterpret_cast<const uint2*>(kc_base + (size_t)(t0 + r) * 32 + 8 * g);
    const uint2 kc1 = *reinterpret_cast<const uint2*>(kc_base + (size_t)(t0 + 16 + r) * 32 + 8 * g);
    const uint4 vc = *reinterpret_cast<const uint4*>(vc_base + (size_t)w * 1024 + 16 * lane);
    const uint2 nk = *reinterpret_cast<const uint2*>(kn_base + t0 + own_tok);
    const uint2 nv = *reinterpret_cast<const uint2*>(vn_base + t0 + own_tok);
    const uint32_t md = *reinterpret_cast<const uint32_t*>(md_base + t0 + own_tok);
    const uint32_t stp = *reinterpret_cast<const uint32_t*>(st_base + (size_t)w * kD + 32 * g + 2 * col);
    const uint32_t mnp = *reinterpret_cast<const uint32_t*>(mn_base + (size_t)w * kD + 32 * g + 2 * col);

    // ---- per-window metadata through wave-private LDS ----
    meta[wave][0][16 * g + col] = stp;
    meta[wave][1][16 * g + col] = mnp;
    wave_lds_sync();
    uint32_t sv[16], mv[16];  // fp16 pairs: channels 32 g + 2 i, 2 i + 1
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint4 a = *reinterpret_cast<const uint4*>(&meta[wave][0][16 * g + 4 * i]);
      const uint4 c = *reinterpret_cast<const uint4*>(&meta[wave][1][16 * g + 4 * i]);
      sv[4 * i] = a.x; sv[4 * i + 1] = a.y; sv[4 * i + 2] = a.z; sv[4 * i + 3] = a.w;
      mv[4 * i] = c.x; mv[4 * i + 1] = c.y; mv[4 * i + 2] = c.z; mv[4 * i + 3] = c.w;
    }
    wave_lds_sync();

    // ---- B operands (q' * step * 2^(k0 - shift)) and the per-window bias q'.m ----
    uint32_t bq[4][4];
    float bias = 0.0f;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float prod[2];
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
          const int e = 2 * i + hh;
          const int lc = slot_channel(kk, e);
          const float stf = h2f((sv[lc >> 1] >> (16 * (lc & 1))) & 0xffffu);
          const float mnf = h2f((mv[lc >> 1] >> (16 * (lc & 1))) & 0xffffu);
          prod[hh] = qk[kk * 8 + e] * stf;
          bias = __builtin_fmaf(qb[kk * 8 + e], mnf, bias);
        }
        bq[kk][i] = pack2(prod[0], prod[1]);
      }
    }
    bias += __shfl_xor(bias, 16);
    bias += __shfl_xor(bias, 32);

    // ---- scores: 8 MFMAs, block-diagonal over the two token halves ----
    floatx4 sc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < 8; ++kk) {
      const bool mine = (kk >= 4) == upper;
      const half8 bop = mine ? h8(bq[kk & 3][0], bq[kk & 3][1], bq[kk & 3][2], bq[kk & 3][3]) : h8(0, 0, 0, 0);
      const half8 aop = (kk < 4) ? key_a_operand(kc0.x, kc0.y, kk & 3) : key_a_operand(kc1.x, kc1.y, kk & 3);
      sc = __builtin_amdgcn_mfma_f32_16x16x32_f16(aop, bop, sc, 0, 0, 0);
    }

    // ---- online softmax (base 2) ----
    const float nkf[4] = {h2f(nk.x & 0xffffu), h2f(nk.x >> 16), h2f(nk.y & 0xffffu), h2f(nk.y >> 16)};
    const float nvf[4] = {h2f(nv.x & 0xffffu), h2f(nv.x >> 16), h2f(nv.y & 0xffffu), h2f(nv.y >> 16)};
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
      if (valid) mods |= 1u << ((md >> (8 * i)) & 3u);
    }
    const bool any_av = __any((mods & 3u) != 0);
    const bool any_t = __any((mods & 4u) != 0);
    seen |= (__any((mods & 1u) != 0) ? 1u : 0u) | (__any((mods & 2u) != 0) ? 2u : 0u) | (any_t ? 4u : 0u);

    // ---- value B operands from the code-byte table ----
    const uint32_t vw[4] = {vc.x, vc.y, vc.z, vc.w};
    auto vop = [&](int nb) -> half8 {
      const uint32_t b0 = (vw[nb >> 2] >> (8 * (nb & 3))) & 0xffu;          // tokens 4g .. 4g+3
      const uint32_t b1 = (vw[2 + (nb >> 2)] >> (8 * (nb & 3))) & 0xffu;    // tokens 16+4g ..
      const uint2 x0 = vlut[b0];
      const uint2 x1 = vlut[b1];
      return h8(x0.x, x0.y, x1.x, x1.y);
    };

    if (any_av) {
      float keep[4], send[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const uint32_t mi = (md >> (8 * i)) & 0xffu;
        const float pa = (mi == 0u) ? pv[i] : 0.0f;  // audio
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
        const uint32_t mi = (md >> (8 * i)) & 0xffu;
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
  // header: m, l per head; mask
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

// ---- merge over splits: one block (128 threads = channels) per (b, query head j, modality) ----
__global__ __launch_bounds__(128) void k_decode_merge(const float* __restrict__ ws, const int32_t* __restrict__ seq_lens,
                                                      int H, int Hq, int G, int wps, int nsplit,
                                                      int cap, float* __restrict__ merged) {
  const int j = blockIdx.x, mod = blockIdx.y, b = blockIdx.z;
  const int h = j / G, hd = j % G;
  const int tid = threadIdx.x;
  const int len = min(seq_lens[b], cap);
  const int ns = min((len + kW - 1) / kW + wps - 1, nsplit * wps) / wps;  // non-empty splits
  const float* base = ws + ((size_t)b * H + h) * nsplit * kRecFloats;
  float M = -__builtin_inff();
  for (int s = 0; s < ns; ++s) M = fmaxf(M, base[(size_t)s * kRecFloats + hd]);
  float L = 0.0f, a = 0.0f;
  for (int s = 0; s < ns; ++s) {
    const float* rs = base + (size_t)s * kRecFloats;
    const float ms = rs[hd];
    if (ms == -__builtin_inff()) continue;
    const float f = exp2f(ms - M);
    L += rs[8 + hd] * f;
    const uint32_t mk = reinterpret_cast<const uint32_t*>(rs)[16];
    if (mk & (1u << mod)) a += rs[kRecHeader + (mod * 8 + hd) * kD + tid] * f;
  }
  float* out = merged + (((size_t)b * Hq + j) * 4) * kD;
  out[mod * kD + tid] = (L > 0.0f) ? a / L : 0.0f;
}

// ---- inverse value rotation, once per modality: o = sum_m R_m^T acc_m ----
// One block (128 threads = output channels) per (b, query head j).
__global__ __launch_bounds__(128) void k_decode_unrotate(const float* __restrict__ merged, const float* __restrict__ rot,
                                                         int Hq, float* __restrict__ out) {
  __shared__ float acc[3][kD];
  const int j = blockIdx.x, b = blockIdx.y, c = threadIdx.x;
  const float* src = merged + (((size_t)b * Hq + j) * 4) * kD;
#pragma unroll
  for (int m = 0; m < 3; ++m) acc[m][c] = src[m * kD + c];
  __syncthreads();
  float o = 0.0f;
  for (int m = 0; m < 3; ++m) {
    const float* rm = rot + (size_t)m * kD * kD;
    for (int k = 0; k < kD; ++k) o = __builtin_fmaf(acc[m][k], rm[(size_t)k * kD + c], o);
  }
  out[((size_t)b * Hq + j) * kD + c] = o;
}

DecodePlan plan_decode(int B, int H, int max_len) {
  const int nwin = (max_len + kW - 1) / kW;
  const long units = (long)B * H;
  const long target_groups = 512;  // about two work-groups per compute unit
  int wps = (int)((nwin * units + target_groups - 1) / target_groups);
  wps = wps < kMinWps ? kMinWps : wps;
  DecodePlan p;
  p.wins_per_split = wps;
  p.nsplit = nwin > 0 ? (nwin + wps - 1) / wps : 1;
  return p;
}

size_t decode_workspace_bytes(int B, int H, int Hq, int max_len) {
  const int nwin = (max_len + kW - 1) / kW;
  const int nsplit_max = nwin > 0 ? (nwin + kMinWps - 1) / kMinWps : 1;
  const size_t records = (size_t)B * H * nsplit_max * kRecFloats * sizeof(float);
  const size_t merged = (size_t)B * Hq * 4 * kD * sizeof(float);
  return records + merged;
}

hipError_t launch_decode(const CacheView& c, const uint16_t* q, float sm_scale, float* out, void* ws,
                         const DecodePlan& plan, hipStream_t s, uint32_t cb01, uint32_t cb23, int max_len) {
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
  const int nwin = (max_len + kW - 1) / kW;
  const int nsplit_max = nwin > 0 ? (nwin + kMinWps - 1) / kMinWps : 1;
  float* merged = a.ws + (size_t)c.B * c.H * nsplit_max * kRecFloats;
  hipLaunchKernelGGL(k_decode_merge, dim3(c.Hq, 3, c.B), dim3(128), 0, s, a.ws, c.seq_lens, c.H, c.Hq, G,
                     plan.wins_per_split, plan.nsplit, c.cap, merged);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_decode_unrotate, dim3(c.Hq, c.B), dim3(128), 0, s, merged, c.rot, c.Hq, out);
  return hipGetLastError();
}

}  // namespace okvq
