// Codecs of the bit-width ladder: b-bit keys and values, b = 2, 3, 4 (the K3/V2 row of Tab. 3 and
// the K2V2 / K3V3 / K4V4 columns of Tab. 5), in the token-major bit-stream layout: a token's 128
// codes form a little-endian bit stream, channel c at bits [b c, b c + b) of the token's 16 b bytes.
//
// Keys: the direction in the key codec's bit-exact order (fp16 norm by the halving tree,
// butterflies h = 1 .. 64, z = w fl(kappa / n16)). TurboQuant keys (one work-group of 128 threads
// per 128 tokens, thread = token) take code = #{k : z_c > tau_k} against the 2^b - 1 thresholds of
// the b-bit Gaussian codebook (Eq. 2, Eq. 3), straight from registers. The method's keys (Eq. 4;
// one work-group of 128 threads per 32-token window, four lanes per token) take each window's
// minimum and step (max - min) / (2^b - 1) in fp16 through an LDS tile and the codes
// clamp(rint(fl(fl(z - m16) fl(1 / step16))), 0, 2^b - 1).
//
// Values, exact mode (one work-group of 128 threads, thread = output channel, per 32-token window): the
// exact-mode order of the 2-bit codec -- y_c = sum_j fl(R_cj v_j) left to right in fp32, n16 by the
// halving tree -- and code = #{k : y_c > fl(n16 tau_k)} against the 2^b - 1 thresholds. A thread
// holds its row of R_m in registers for each modality present in the window (R is read once per
// window, not once per token); then a thread per (token, 32 channels) packs b dwords.
#include "key_quant.hpp"
#include "lane_quant.hpp"
#include "launch.hpp"

namespace okvq {
namespace {

constexpr int kTileTokens = 128;

// OR the 32 codes of channels 32 part .. 32 part + 31 (one per byte of `codes`) into the b dwords
// they occupy: bits b (c - 32 part) of the run starting at dword b part.
template <int kBits>
__device__ __forceinline__ void pack32(const uint32_t (&cw)[8], uint32_t (&w)[kBits]) {
#pragma unroll
  for (int i = 0; i < kBits; ++i) w[i] = 0u;
#pragma unroll
  for (int c = 0; c < 32; ++c) {
    const uint32_t v = (cw[c >> 2] >> (8 * (c & 3))) & 0xffu;
    const int bit = kBits * c, d = bit >> 5, sh = bit & 31;
    w[d] |= v << sh;
    if (sh + kBits > 32) w[d + 1] |= v >> (32 - sh);
  }
}

template <int kBits>
__device__ __forceinline__ void store_run(uint8_t* row, int part, const uint32_t (&w)[kBits]) {
  uint32_t* p = reinterpret_cast<uint32_t*>(row) + kBits * part;
#pragma unroll
  for (int i = 0; i < kBits; ++i) p[i] = w[i];
}

template <int kBits>
__global__ __launch_bounds__(kTileTokens) void k_ladder_keys_tq(LadderKeyArgs a) {
  constexpr int kTop = (1 << kBits) - 1;
  constexpr int kRowBytes = 16 * kBits;
  const int h = blockIdx.y, bz = blockIdx.z, b = a.b0 + bz;
  int begin = 0, len = a.lens.lens[bz];
  if (a.begin_dev) {  // append: the device lengths decide, clamped into the buffers
    begin = min(max(a.begin_dev[b], 0), a.cap);
    len = min(begin + min(max(a.count_dev[b], 0), a.n_rows), a.cap);
    if (len <= begin) return;  // uniform
  }
  // TurboQuant keys are per token: only the new tokens are coded
  const int t0 = begin + kTileTokens * blockIdx.x;
  if (t0 >= len) return;  // uniform over the work-group
  const int t = threadIdx.x, tok = t0 + t;
  const bool valid = tok < len;
  const int npad = (len + kW - 1) / kW * kW;  // slots of every window holding a valid token
  const size_t seq = (size_t)b * a.H + h;

  // ---- the direction, in registers (thread = token) ----
  uint32_t sw[32];
  load_sign_words(a.signs, sw);
  uint32_t raw[64];
  if (valid) {
    load_row_f16(a.k + (seq * a.n_rows + (tok - begin)) * kD, raw);
  } else {
#pragma unroll
    for (int i = 0; i < 64; ++i) raw[i] = 0u;
  }
  float x[kD];
  key_unpack(raw, sw, x);
  const uint32_t n16 = key_norm(x);
#pragma unroll
  for (int hh = 1; hh < kD; hh <<= 1) {
#pragma unroll
    for (int j = 0; j < kD; ++j) {
      if ((j & hh) == 0) {
        const float p = x[j], q = x[j + hh];
        x[j] = p + q;
        x[j + hh] = p - q;
      }
    }
  }
  const float cinv = (n16 == 0) ? 0.0f : div_rn(kKappa, h2f(n16));
#pragma unroll
  for (int c = 0; c < kD; ++c) x[c] = x[c] * cinv;
  if (tok < npad) a.k_norm[seq * a.cap + tok] = valid ? (uint16_t)n16 : (uint16_t)0;

  // ---- nearest level of the b-bit codebook, packed straight from registers ----
  if (tok >= npad) return;
  uint8_t* row = a.k_codes + (seq * a.cap + tok) * kRowBytes;
#pragma unroll
  for (int part = 0; part < 4; ++part) {
    uint32_t cw[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) cw[i] = 0u;
#pragma unroll
    for (int c = 0; c < 32; ++c) {
      const float z = x[32 * part + c];
      uint32_t code = 0;
#pragma unroll
      for (int k = 0; k < kTop; ++k) code += (uint32_t)(z > a.tau[k]);
      cw[c >> 2] |= (valid ? code : 0u) << (8 * (c & 3));
    }
    uint32_t w[kBits];
    pack32<kBits>(cw, w);
    store_run<kBits>(row, part, w);
  }
}

// The method's keys, one work-group of 128 threads per 32-token key window: thread (t, q) holds
// channels 32q .. 32q + 31 of window token t, so that a token spans the 4 lanes of a DPP quad. The
// norm tree and the butterflies run in the key codec's bit-exact order: the tree's levels 64 and 32
// pair lane q with q ^ 2 and q ^ 1 (both lanes of a pair form the same exact-order sum), the levels
// 16 .. 1 and the butterfly stages h = 1 .. 16 stay in the lane, and the stages h = 32, 64 cross to
// lane q ^ 1, q ^ 2 as fl(+-own + partner); z = w fl(kappa / n16). The directions go to an LDS tile;
// thread c then takes channel c's window minimum and maximum over the valid tokens (exact in any
// order) and forms the fp16 minimum, step = (max - min) / (2^b - 1) and fl(1 / step16); every thread
// codes its 32 channels, clamp(rint(fl(fl(z - m16) fl(1 / step16))), 0, 2^b - 1), which fill b
// dwords of the token's bit stream (the run at dword b q). TurboQuant keys take the token-per-thread
// kernel above, which needs no window statistics.
constexpr int kQuadThreads = 128;
constexpr int kWinPitch = kD + 4;  // floats per token row of the direction tile

// Butterfly stage across lanes q and q ^ kMask of a quad: the lower lane takes a + b, the upper one
// a - b, both as fl(s own + partner) with s = +-1 (an exact product, one rounding).
template <int kMask, int kN>
__device__ __forceinline__ void quad_stage(float (&x)[kN], int q) {
  const float s = (q & kMask) ? -1.0f : 1.0f;
#pragma unroll
  for (int e = 0; e < kN; ++e) x[e] = __builtin_fmaf(s, x[e], xchg<kMask>(x[e]));
}

template <int kBits>
__global__ __launch_bounds__(kQuadThreads) void k_ladder_keys_quad(LadderKeyArgs a) {
  constexpr int kTop = (1 << kBits) - 1;
  constexpr int kRowBytes = 16 * kBits;
  __shared__ __attribute__((aligned(16))) float zt[kW][kWinPitch];  // the window's directions
  __shared__ __attribute__((aligned(8))) float2 kstat[kD];  // (fp16 minimum, fl(1 / fp16 step)) as fp32
  const int h = blockIdx.y, bz = blockIdx.z, b = a.b0 + bz, wi = blockIdx.x;
  const int tid = threadIdx.x, t = tid >> 2, q = tid & 3;
  int begin = 0, len = a.lens.lens[bz];
  if (a.begin_dev) {  // append: the device lengths decide, clamped into the buffers
    begin = min(max(a.begin_dev[b], 0), a.cap);
    len = min(begin + min(max(a.count_dev[b], 0), a.n_rows), a.cap);
  }
  const int first = (begin / kW) * kW, w0 = first + kW * wi, tok = w0 + t;
  if (len <= begin || w0 >= len) return;  // uniform over the work-group
  const size_t seq = (size_t)b * a.H + h;
  const int npad = (len + kW - 1) / kW * kW;
  const int open = (len / kW) * kW, stok = open + t, last = a.n_rows - 1;
  const bool valid = tok < len;
  const bool staged = a.begin_dev && wi == 0 && begin > first;          // older tokens from the stage
  const bool restage = a.stage && a.begin_dev && wi == 0 && open < len;  // the new open window's rows
  // every load before any use: the signs, the token's 64-byte chunk (or its staged one), the open
  // window's chunk
  const uint4* sp = reinterpret_cast<const uint4*>(a.signs + 32 * q);
  const uint4 sg0 = sp[0], sg1 = sp[1];
  const size_t srow = seq * a.n_rows;
  const uint4 zero = make_uint4(0u, 0u, 0u, 0u);
  const uint4* kp = reinterpret_cast<const uint4*>(a.k + (srow + (size_t)min(max(tok - begin, 0), last)) * kD + 32 * q);
  // the stage (only where it holds older tokens: the stage may be absent otherwise) and the open
  // window's rows (only where the new open window starts after this one)
  const uint4* stp = staged ? reinterpret_cast<const uint4*>(a.stage + (seq * kW + min(t, begin - first - 1)) * kD + 32 * q)
                            : kp;
  const uint4* ssp = (restage && open != first)
                         ? reinterpret_cast<const uint4*>(a.k + (srow + (size_t)min(max(stok - begin, 0), last)) * kD + 32 * q)
                         : kp;
  const bool fresh = valid && tok >= begin, old = staged && tok < begin;
  // kraw: the token's 32 keys (from the stage below begin, zero past the length); sraw: those of
  // token open + t, for the stage
  uint32_t kraw[16], sraw[16];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint4 n = kp[i];
    uint4 o = zero, r = zero;
    if (staged) o = stp[i];
    if (restage && open != first) r = ssp[i];
    const uint4 f = fresh ? n : zero;
    const uint4 k = old ? o : f;
    kraw[4 * i] = k.x;
    kraw[4 * i + 1] = k.y;
    kraw[4 * i + 2] = k.z;
    kraw[4 * i + 3] = k.w;
    sraw[4 * i] = r.x;
    sraw[4 * i + 1] = r.y;
    sraw[4 * i + 2] = r.z;
    sraw[4 * i + 3] = r.w;
  }
  // ---- direction: signs applied (the fp16 sign bits flipped), channel 32q + 8i + e in x[8i + e] ----
  float x[32];
  const uint32_t sw[8] = {sg0.x, sg0.y, sg0.z, sg0.w, sg1.x, sg1.y, sg1.z, sg1.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t r4[4] = {kraw[4 * i], kraw[4 * i + 1], kraw[4 * i + 2], kraw[4 * i + 3]};
#pragma unroll
    for (int d = 0; d < 4; ++d) {
      const uint32_t w = sw[2 * i + (d >> 1)];  // int8 signs of channels 8i + 4 (d / 2) .. + 3
      const uint32_t m = (d & 1) ? (((w & 0x00800000u) >> 8) | (w & 0x80000000u))
                                 : (((w & 0x00000080u) << 8) | ((w & 0x00008000u) << 16));
      const uint32_t rr = r4[d] ^ m;
      x[8 * i + 2 * d] = h2f(rr & 0xffffu);
      x[8 * i + 2 * d + 1] = h2f(rr >> 16);
    }
  }
  // fp16 norm: levels 64 and 32 across the quad, 16 .. 1 in the lane
  float tt[32];
#pragma unroll
  for (int e = 0; e < 32; ++e) {
    const float p = xchg<2>(x[e]);
    tt[e] = x[e] * x[e] + p * p;
  }
#pragma unroll
  for (int e = 0; e < 32; ++e) tt[e] = tt[e] + xchg<1>(tt[e]);
#pragma unroll
  for (int n = 16; n >= 1; n >>= 1) {
#pragma unroll
    for (int e = 0; e < n; ++e) tt[e] = tt[e] + tt[e + n];
  }
  const uint32_t n16 = norm_to_f16(sqrt_rn(tt[0]));
#pragma unroll
  for (int hh = 1; hh < 32; hh <<= 1) {
#pragma unroll
    for (int e = 0; e < 32; ++e) {
      if ((e & hh) == 0) {
        const float p = x[e], r = x[e + hh];
        x[e] = p + r;
        x[e + hh] = p - r;
      }
    }
  }
  quad_stage<1>(x, q);  // h = 32
  quad_stage<2>(x, q);  // h = 64
  const float cinv = (n16 == 0) ? 0.0f : div_rn(kKappa, h2f(n16));
#pragma unroll
  for (int e = 0; e < 32; ++e) x[e] = x[e] * cinv;
  if (q == 0 && tok < npad) a.k_norm[seq * a.cap + tok] = valid ? (uint16_t)n16 : (uint16_t)0;
#pragma unroll
  for (int i = 0; i < 8; ++i)
    *reinterpret_cast<float4*>(&zt[t][32 * q + 4 * i]) = make_float4(x[4 * i], x[4 * i + 1], x[4 * i + 2], x[4 * i + 3]);
  if (restage) __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");  // this thread's stage reads have landed
  __syncthreads();  // the direction tile is complete; every stage read of the work-group has landed
  if (restage && stok >= begin && stok < len) {
    uint4* p = reinterpret_cast<uint4*>(a.stage + (seq * kW + t) * kD + 32 * q);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint32_t* v = (open == first) ? &kraw[4 * i] : &sraw[4 * i];
      p[i] = make_uint4(v[0], v[1], v[2], v[3]);
    }
  }
  {  // thread = channel
    const int c = tid;
    const int nv = min(len - w0, kW);
    float lo4[4], hi4[4];  // four independent chains (the minimum and maximum are exact in any order)
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      lo4[u] = __builtin_inff();
      hi4[u] = -__builtin_inff();
    }
#pragma unroll
    for (int i = 0; i < kW; ++i) {  // all 32 reads in flight at once; slots past the length skipped
      const float v = zt[i][c];
      lo4[i & 3] = (i < nv) ? fminf(lo4[i & 3], v) : lo4[i & 3];
      hi4[i & 3] = (i < nv) ? fmaxf(hi4[i & 3], v) : hi4[i & 3];
    }
    const float lo = fminf(fminf(lo4[0], lo4[1]), fminf(lo4[2], lo4[3])) + 0.0f;  // -0 -> +0
    const float hi = fmaxf(fmaxf(hi4[0], hi4[1]), fmaxf(hi4[2], hi4[3])) + 0.0f;
    const float step = div_rn(hi - lo, (float)kTop);
    const uint32_t m16 = f2h(lo), s16 = f2h(step);
    const size_t mi = (seq * (a.cap / kW) + w0 / kW) * kD + c;
    a.k_min[mi] = (uint16_t)m16;
    a.k_step[mi] = (uint16_t)s16;
    const float sv = h2f(s16);
    kstat[c] = make_float2(h2f(m16), (sv != 0.0f) ? div_rn(1.0f, sv) : 0.0f);
  }
  __syncthreads();  // the window's statistics
  if (tok >= npad) return;
  uint32_t cw[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) cw[i] = 0u;
  if (valid) {
#pragma unroll
    for (int e = 0; e < 32; ++e) {
      const float2 st = kstat[32 * q + e];
      const float tq = (x[e] - st.x) * st.y;
      const uint32_t code = (uint32_t)fminf(fmaxf(__builtin_rintf(tq), 0.0f), (float)kTop);
      cw[e >> 2] |= code << (8 * (e & 3));
    }
  }
  uint32_t w[kBits];
  pack32<kBits>(cw, w);
  store_run<kBits>(a.k_codes + (seq * a.cap + tok) * kRowBytes, q, w);
}

__device__ __forceinline__ float tree_norm_lds(const float* xs) {  // xs: 128 floats (LDS)
  float tt[64];
#pragma unroll
  for (int i = 0; i < 64; ++i) tt[i] = xs[i] * xs[i] + xs[i + 64] * xs[i + 64];
#pragma unroll
  for (int n = 32; n >= 1; n >>= 1) {
#pragma unroll
    for (int i = 0; i < n; ++i) tt[i] = tt[i] + tt[i + n];
  }
  return sqrt_rn(tt[0]);
}

// The value tokens [begin, len) of sequence b: stateless [0, lens), append from the device lengths.
__device__ __forceinline__ void value_span(const LadderValueArgs& a, int bz, int b, int& begin, int& len) {
  begin = 0;
  len = a.lens.lens[bz];
  if (a.begin_dev) {
    begin = min(max(a.begin_dev[b], 0), a.cap);
    len = min(begin + min(max(a.count_dev[b], 0), a.n_rows), a.cap);
  }
}

template <int kBits>
__global__ __launch_bounds__(128) void k_ladder_values(LadderValueArgs a) {
  constexpr int kTop = (1 << kBits) - 1;
  constexpr int kRowBytes = 16 * kBits;
  __shared__ __attribute__((aligned(16))) float xs[kW][kD];
  __shared__ float nrm[kW];
  __shared__ int mods[kW];
  __shared__ __attribute__((aligned(16))) uint8_t ct[kW][kD];
  const int h = blockIdx.y, bz = blockIdx.z, b = a.b0 + bz;
  int begin, len;
  value_span(a, bz, b, begin, len);
  const int t0 = begin + kW * blockIdx.x;
  if (t0 >= len) return;
  const int c = threadIdx.x;
  const size_t seq = (size_t)b * a.H + h;
  for (int t = 0; t < kW; ++t) {
    const int tok = t0 + t;
    xs[t][c] = (tok < len) ? h2f(a.v[(seq * a.n_rows + (tok - begin)) * kD + c]) : 0.0f;
  }
  if (c < kW) {
    const int tok = t0 + c;
    mods[c] = (tok < len) ? (int)a.modality[(size_t)b * a.n_rows + (tok - begin)] : -1;
    if (tok < len && a.mod_out && h == 0) a.mod_out[(size_t)b * a.cap + tok] = (uint8_t)mods[c];
  }
  __syncthreads();
  if (c < kW) {
    const int tok = t0 + c;
    const uint32_t n16 = (tok < len) ? norm_to_f16(tree_norm_lds(xs[c])) : 0u;
    nrm[c] = h2f(n16);
    if (tok < len) a.v_norm[seq * a.cap + tok] = (uint16_t)n16;
  }
  __syncthreads();
  // codes default to 0 (padded or out-of-contract tokens); then, per modality present in the window,
  // this thread's row c of R_m in registers against every token of that modality
  for (int t = 0; t < kW; ++t) ct[t][c] = 0;
  for (int m = 0; m < 3; ++m) {
    bool any = false;
    for (int t = 0; t < kW; ++t) any |= mods[t] == m;
    if (!any) continue;  // uniform over the work-group
    float rr[kD];
    const float4* rp = reinterpret_cast<const float4*>(a.rot + ((size_t)m * kD + c) * kD);
#pragma unroll
    for (int k4 = 0; k4 < kD / 4; ++k4) {
      const float4 f = rp[k4];
      rr[4 * k4] = f.x;
      rr[4 * k4 + 1] = f.y;
      rr[4 * k4 + 2] = f.z;
      rr[4 * k4 + 3] = f.w;
    }
    for (int t = 0; t < kW; ++t) {
      if (mods[t] != m) continue;
      const float4* xr = reinterpret_cast<const float4*>(xs[t]);
      float acc = 0.0f;
#pragma unroll
      for (int k4 = 0; k4 < kD / 4; ++k4) {  // left to right, no contraction: the exact order
        const float4 x4 = xr[k4];
        acc = acc + rr[4 * k4] * x4.x;
        acc = acc + rr[4 * k4 + 1] * x4.y;
        acc = acc + rr[4 * k4 + 2] * x4.z;
        acc = acc + rr[4 * k4 + 3] * x4.w;
      }
      const float nv = nrm[t];
      uint32_t code = 0;
#pragma unroll
      for (int k = 0; k < kTop; ++k) code += (uint32_t)(acc > nv * a.tau[k]);
      ct[t][c] = (uint8_t)code;
    }
  }
  __syncthreads();
  // packing: thread = (token c / 4, channels 32 (c % 4) .. +31)
  const int t = c >> 2, part = c & 3, tok = t0 + t;
  if (tok >= len) return;
  uint32_t cw[8];
  const uint4* src = reinterpret_cast<const uint4*>(&ct[t][32 * part]);
  const uint4 u0 = src[0], u1 = src[1];
  cw[0] = u0.x; cw[1] = u0.y; cw[2] = u0.z; cw[3] = u0.w;
  cw[4] = u1.x; cw[5] = u1.y; cw[6] = u1.z; cw[7] = u1.w;
  uint32_t w[kBits];
  pack32<kBits>(cw, w);
  store_run<kBits>(a.v_codes + (seq * a.cap + tok) * kRowBytes, part, w);
}

// MFMA mode: one work-group of 256 threads (4 waves) per 128 tokens of a (sequence, KV head). The
// value rows (fp16, exact) are staged in LDS as MFMA A operands; wave w computes output channels
// 32 w .. 32 w + 31, per modality, of the 16-token row blocks holding a token of it (ballots of the
// norm step mark them), against its slice of R_m split into
// fp16 hi + lo parts (B operands, converted once per modality and tile), fp32 accumulation. The
// codes then equal the exact order's except where y lies within a small band of a threshold (about
// 2^-22 sum_j |R_cj v_j| of accumulation-order and split error, inside the band the tests allow).
typedef _Float16 half8v __attribute__((ext_vector_type(8)));
typedef float floatx4v __attribute__((ext_vector_type(4)));
constexpr int kVTile = 128;       // tokens per work-group
constexpr int kVPitch = kD + 8;   // fp16 row pitch of the LDS value tile

__device__ __forceinline__ uint32_t hi_lo_pair(float x0, float x1, bool lo) {
  const _Float16 h0 = (_Float16)x0, h1 = (_Float16)x1;
  const _Float16 a = lo ? (_Float16)(x0 - (float)h0) : h0;
  const _Float16 b = lo ? (_Float16)(x1 - (float)h1) : h1;
  return (uint32_t)__builtin_bit_cast(uint16_t, a) | ((uint32_t)__builtin_bit_cast(uint16_t, b) << 16);
}

template <int kBits>
__global__ __launch_bounds__(256) void k_ladder_values_mfma(LadderValueArgs a) {
  constexpr int kTop = (1 << kBits) - 1;
  constexpr int kRowBytes = 16 * kBits;
  __shared__ __attribute__((aligned(16))) uint16_t xs[kVTile][kVPitch];
  __shared__ float nrm[kVTile];
  __shared__ int mods[kVTile];
  __shared__ uint32_t wpres[kVTile / 64];  // bit 8 m + row block: modality m present in those 16 rows
  __shared__ __attribute__((aligned(16))) uint8_t ct[kVTile][kD];
  const int h = blockIdx.y, bz = blockIdx.z, b = a.b0 + bz;
  int begin, len;
  value_span(a, bz, b, begin, len);
  const int t0 = begin + kVTile * blockIdx.x;
  if (t0 >= len) return;  // uniform
  const int tid = threadIdx.x, lane = tid & 63, g = lane >> 4, r = lane & 15;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const size_t seq = (size_t)b * a.H + h;
  // ---- stage the rows (zeros beyond the length), the modalities, the codes' default 0 ----
  for (int idx = tid; idx < kVTile * (kD / 8); idx += 256) {
    const int t = idx >> 4, c8 = idx & 15, tok = t0 + t;
    const uint4 v = (tok < len) ? *reinterpret_cast<const uint4*>(a.v + (seq * a.n_rows + (tok - begin)) * kD + 8 * c8)
                                : make_uint4(0u, 0u, 0u, 0u);
    *reinterpret_cast<uint4*>(&xs[t][8 * c8]) = v;
    *reinterpret_cast<uint2*>(&ct[t][8 * c8]) = make_uint2(0u, 0u);
  }
  if (tid < kVTile) {
    const int tok = t0 + tid;
    mods[tid] = (tok < len) ? (int)a.modality[(size_t)b * a.n_rows + (tok - begin)] : -1;
    if (tok < len && a.mod_out && h == 0) a.mod_out[(size_t)b * a.cap + tok] = (uint8_t)mods[tid];
  }
  __syncthreads();
  if (tid < kVTile) {  // fp16 norm by the halving tree, as the exact mode; the row in 16-byte reads
    const int tok = t0 + tid;
    float x[kD];
#pragma unroll
    for (int c8 = 0; c8 < kD / 8; ++c8) {
      const uint4 v = *reinterpret_cast<const uint4*>(&xs[tid][8 * c8]);
      const uint32_t w4[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        x[8 * c8 + 2 * i] = h2f(w4[i] & 0xffffu);
        x[8 * c8 + 2 * i + 1] = h2f(w4[i] >> 16);
      }
    }
    float tt[64];
#pragma unroll
    for (int i = 0; i < 64; ++i) tt[i] = x[i] * x[i] + x[i + 64] * x[i + 64];
#pragma unroll
    for (int n = 32; n >= 1; n >>= 1) {
#pragma unroll
      for (int i = 0; i < n; ++i) tt[i] = tt[i] + tt[i + n];
    }
    const uint32_t n16 = (tok < len) ? norm_to_f16(sqrt_rn(tt[0])) : 0u;
    nrm[tid] = h2f(n16);
    if (tok < len) a.v_norm[seq * a.cap + tok] = (uint16_t)n16;
    const int mo = mods[tid];  // -1 past the length
    uint32_t pres = 0;
#pragma unroll
    for (int m = 0; m < 3; ++m) {
      const uint64_t bm = __ballot(mo == m);  // this wave's tokens: row blocks 4 wave .. 4 wave + 3
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if ((bm >> (16 * i)) & 0xffffu) pres |= 1u << (8 * m + 4 * wave + i);
    }
    if (lane == 0) wpres[wave] = pres;
  }
  __syncthreads();
  uint32_t present = 0;
#pragma unroll
  for (int w = 0; w < kVTile / 64; ++w) present |= wpres[w];
  for (int m = 0; m < 3; ++m) {
    if (!((present >> (8 * m)) & 0xffu)) continue;  // uniform
    // B operands: channel c = 32 wave + 16 cb + r, k = 32 kb + 8 g .. + 7 of R_m (hi, lo parts)
    uint32_t bh[2][4][4], bl[2][4][4];
#pragma unroll
    for (int cb = 0; cb < 2; ++cb) {
      const float* rrow = a.rot + ((size_t)m * kD + 32 * wave + 16 * cb + r) * kD;
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        const float4 p0 = *reinterpret_cast<const float4*>(rrow + 32 * kb + 8 * g);
        const float4 p1 = *reinterpret_cast<const float4*>(rrow + 32 * kb + 8 * g + 4);
        const float v8[8] = {p0.x, p0.y, p0.z, p0.w, p1.x, p1.y, p1.z, p1.w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          bh[cb][kb][j] = hi_lo_pair(v8[2 * j], v8[2 * j + 1], false);
          bl[cb][kb][j] = hi_lo_pair(v8[2 * j], v8[2 * j + 1], true);
        }
      }
    }
    for (int rb = 0; rb < kVTile / 16; ++rb) {
      if (!((present >> (8 * m + rb)) & 1u)) continue;  // no token of modality m in these rows (uniform)
      floatx4v acc[2] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        const half8v av = *reinterpret_cast<const half8v*>(&xs[16 * rb + r][32 * kb + 8 * g]);
#pragma unroll
        for (int cb = 0; cb < 2; ++cb) {
          acc[cb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(
              av, __builtin_bit_cast(half8v, make_uint4(bh[cb][kb][0], bh[cb][kb][1], bh[cb][kb][2], bh[cb][kb][3])),
              acc[cb], 0, 0, 0);
          acc[cb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(
              av, __builtin_bit_cast(half8v, make_uint4(bl[cb][kb][0], bl[cb][kb][1], bl[cb][kb][2], bl[cb][kb][3])),
              acc[cb], 0, 0, 0);
        }
      }
      // D[token 16 rb + 4 g + i][channel 32 wave + 16 cb + r]
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int t = 16 * rb + 4 * g + i;
        if (mods[t] != m) continue;
        const float nv = nrm[t];
#pragma unroll
        for (int cb = 0; cb < 2; ++cb) {
          uint32_t code = 0;
#pragma unroll
          for (int k = 0; k < kTop; ++k) code += (uint32_t)(acc[cb][i] > nv * a.tau[k]);
          ct[t][32 * wave + 16 * cb + r] = (uint8_t)code;
        }
      }
    }
  }
  __syncthreads();
  // pack: thread = (token, 32 channels), two items each
  for (int it = tid; it < kVTile * 4; it += 256) {
    const int t = it >> 2, part = it & 3, tok = t0 + t;
    if (tok >= len) continue;
    uint32_t cw[8];
    const uint4* src = reinterpret_cast<const uint4*>(&ct[t][32 * part]);
    const uint4 u0 = src[0], u1 = src[1];
    cw[0] = u0.x; cw[1] = u0.y; cw[2] = u0.z; cw[3] = u0.w;
    cw[4] = u1.x; cw[5] = u1.y; cw[6] = u1.z; cw[7] = u1.w;
    uint32_t w[kBits];
    pack32<kBits>(cw, w);
    store_run<kBits>(a.v_codes + (seq * a.cap + tok) * kRowBytes, part, w);
  }
}

template <int kBits>
hipError_t keys_for_bits(const LadderKeyArgs& a, bool tq, int nb, int max_len, hipStream_t s) {
  if (tq) {
    const dim3 grid((max_len + kTileTokens - 1) / kTileTokens, a.H, nb);
    hipLaunchKernelGGL(k_ladder_keys_tq<kBits>, grid, dim3(kTileTokens), 0, s, a);
  } else {
    const dim3 grid((max_len + kW - 1) / kW, a.H, nb);  // one work-group per key window of the span
    hipLaunchKernelGGL(k_ladder_keys_quad<kBits>, grid, dim3(kQuadThreads), 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_ladder_keys(const LadderKeyArgs& a, int bits, bool tq, int nb, int max_len, hipStream_t s) {
  if (nb <= 0 || max_len <= 0) return hipSuccess;
  switch (bits) {
    case 2: return keys_for_bits<2>(a, tq, nb, max_len, s);
    case 3: return keys_for_bits<3>(a, tq, nb, max_len, s);
    case 4: return keys_for_bits<4>(a, tq, nb, max_len, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_ladder_values(const LadderValueArgs& a, int bits, bool exact, int nb, int max_len, hipStream_t s) {
  if (nb <= 0 || max_len <= 0) return hipSuccess;
  if (!exact) {
    const dim3 grid((max_len + kVTile - 1) / kVTile, a.H, nb);
    switch (bits) {
      case 2: hipLaunchKernelGGL(k_ladder_values_mfma<2>, grid, dim3(256), 0, s, a); break;
      case 3: hipLaunchKernelGGL(k_ladder_values_mfma<3>, grid, dim3(256), 0, s, a); break;
      case 4: hipLaunchKernelGGL(k_ladder_values_mfma<4>, grid, dim3(256), 0, s, a); break;
      default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
  }
  const dim3 grid((max_len + kW - 1) / kW, a.H, nb);
  switch (bits) {
    case 2: hipLaunchKernelGGL(k_ladder_values<2>, grid, dim3(128), 0, s, a); break;
    case 3: hipLaunchKernelGGL(k_ladder_values<3>, grid, dim3(128), 0, s, a); break;
    case 4: hipLaunchKernelGGL(k_ladder_values<4>, grid, dim3(128), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace okvq
