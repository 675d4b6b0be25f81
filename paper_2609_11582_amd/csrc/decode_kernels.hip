// Fused decode attention over the packed 2-bit cache (Eq. 1 with the codecs of Eq. 2, 4, 6).
//
// Split-K flash decoding in two launches. k_decode: work-group (split, KV head h, sequence b) =
// 8 waves; wave w takes the split's window pairs (2w + 16k, 2w + 16k + 1) and keeps its own
// online-softmax state. Each wave streams its pairs through three LDS slots filled by direct
// memory-to-LDS loads two pairs ahead of the one it computes. The waves are combined in LDS, the
// split's per-modality accumulators are un-rotated on MFMA (the inverse rotation is linear, so
// applying it per split and then merging equals applying it once per modality after aggregation,
// Sec. 2.3) and one normalized partial output per split is written. k_decode_merge combines the
// splits by log-sum-exp.
//
// What one wave does per window pair (all G <= 8 query heads of the KV head from one read):
//  * scores in the rotated key space (Sec. 2.3): s_i = n_i (q'.m_g + sum_c q'_c step_gc code_ic),
//    q' = H q sm_scale log2(e) computed once per work-group. The bias q'.m_g of both windows is
//    one MFMA chain (minima as A rows, q' split into fp16 hi and lo columns); the code term is
//    an MFMA per window and 16-token tile: rows = tokens, columns 0-7 = heads (the side-0 lanes
//    keep window A's products), 8-15 = the same heads for window B (side-1 lanes), K = the
//    window's 128 channels. Codes enter the MFMA unchanged as fp16 subnormals (a key code word
//    masked with 3 * 0x00010001 << 2j is the channel pair's codes times 2^(2j-24)); the
//    matching power of two is folded into the B operand q'_c step_gc 2^(k0 - 2j), a packed fp16
//    product of a per-lane query register and the lane's window steps.
//  * online softmax in base 2 (running max per head, rescaled only when it grows by 2^8; scores
//    are formed relative to the current reference, so the exponent needs no subtraction). The
//    PV operand p n_v is fp16 with a per-wave power-of-two scale 2^E, E = 15 - (bound exponent
//    of the largest value norm seen), moved lazily like the max: the largest products sit near
//    2^15, so weights down to about 2^-20 of the running max keep full fp16 precision and the
//    rest (down to about 2^-30) are subnormal with an absolute error below 2^-25 of the scaled
//    unit;
//  * values stay rotated (Sec. 2.3): one register accumulator has rows 0-7 = audio heads and
//    8-15 = video heads, a second one rows 0-7 = text heads (the prompt, a few windows). A pair
//    of one modality takes its rows straight from p n_v; a mixed pair masks them per token with
//    a byte-table lookup (v_perm), and the two row halves exchange window halves with one DPP
//    row rotation under a bank mask. B operands come from a 256-entry LDS table mapping a code
//    byte (one channel, four tokens) to four fp16 codebook levels.
#include <hip/hip_ext.h>

#include <algorithm>
#include <cstdlib>

#include "launch.hpp"

namespace okvq {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef _Float16 half2v __attribute__((ext_vector_type(2)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int kDecWaves = 8;                    // waves per split work-group
constexpr int kATile = 3 * kD + 8;              // fp16 row pitch of the un-rotation A tile
constexpr int kAccPitch = 28;                   // combine tile [channel][24 rows + 4]: conflict-free b128
constexpr int kMinWps = 2 * kDecWaves;          // fewest windows per split (a pair per wave)
constexpr float kLazy = 8.0f;                   // log2 headroom of the lazily updated softmax max

struct DecodeArgs {
  const uint8_t* k_codes;
  const uint8_t* v_codes;
  const uint16_t* k_norm;
  const uint16_t* v_norm;
  const uint16_t* k_min;
  const uint16_t* k_step;
  const uint8_t* k_mx;  // MXFP4 window records (k_decode<kMetaMx>) instead of k_min / k_step
  const uint8_t* modality;
  const int32_t* seq_lens;
  const int8_t* signs;
  const uint16_t* q;
  const uint16_t* rot16t;  // [128][3][128] fp16: (c, m, k) -> R_m[k][c]
  float* ws;               // partial records [B][H][nsplit][kRecFloats]
  int H, Hq, G, cap, wps, nsplit;
  int residual;      // tokens at the end of each sequence left to the merge launch (fp16 residual)
  float qscale;      // sm_scale * log2(e) / sqrt(128)
  uint32_t cb01;     // fp16 codebook levels 0, 1 (low, high half)
  uint32_t cb23;     // fp16 codebook levels 2, 3
};

__device__ __forceinline__ half8 h8(uint32_t a, uint32_t b, uint32_t c, uint32_t d) {
  return __builtin_bit_cast(half8, make_uint4(a, b, c, d));
}
__device__ __forceinline__ half8 h8(const uint32_t (&v)[4]) { return h8(v[0], v[1], v[2], v[3]); }
__device__ __forceinline__ uint32_t pack2(float lo, float hi) { return f2h(lo) | (f2h(hi) << 16); }
__device__ __forceinline__ uint32_t pk_mul(uint32_t a, uint32_t b) {  // packed fp16 product
  return __builtin_bit_cast(uint32_t, __builtin_bit_cast(half2v, a) * __builtin_bit_cast(half2v, b));
}
__device__ __forceinline__ float lo_f16(uint32_t w) { return (float)__builtin_bit_cast(half2v, w)[0]; }
__device__ __forceinline__ float hi_f16(uint32_t w) { return (float)__builtin_bit_cast(half2v, w)[1]; }
__device__ __forceinline__ uint32_t pack_f16(float lo, float hi) {
  const half2v v = {(_Float16)lo, (_Float16)hi};
  return __builtin_bit_cast(uint32_t, v);
}
// 2^x on the hardware unit; results below 2^-126 flush to zero (weights that small do not count)
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
// lane l <- lane l ^ 8 within each row of 16 lanes (DPP row rotate by 8)
constexpr int kRowRor8 = 0x128;
__device__ __forceinline__ float fswap8(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), kRowRor8, 0xf, 0xf, false));
}
// lanes of the given banks (4-lane groups of each row; 0x3 = lanes 0-7, 0xc = lanes 8-15) take
// lane ^ 8's src, the others keep old
template <int kBanks>
__device__ __forceinline__ uint32_t take_partner(uint32_t old, uint32_t src) {
  return (uint32_t)__builtin_amdgcn_update_dpp((int)old, (int)src, kRowRor8, 0xf, kBanks, false);
}
// Pairwise combination of lanes l and l ^ 16 (or l ^ 32) with the VALU row swaps of gfx950
// (v_permlane16_swap / v_permlane32_swap): swapping a register with a copy of itself leaves the
// lane's own value in one result and its partner's in the other, so a symmetric op of the two
// results is the pair's value in both lanes, with no LDS-pipe shuffle. The copy is made opaque:
// given the same value twice, the compiler folds the two results into one.
__device__ __forceinline__ uint32_t opaque_copy(uint32_t v) {
  __asm__ volatile("" : "+v"(v));
  return v;
}
__device__ __forceinline__ void swap16(uint32_t v, uint32_t& a, uint32_t& b) {
  const auto r = __builtin_amdgcn_permlane16_swap(v, opaque_copy(v), false, false);
  a = r[0];
  b = r[1];
}
__device__ __forceinline__ void swap32(uint32_t v, uint32_t& a, uint32_t& b) {
  const auto r = __builtin_amdgcn_permlane32_swap(v, opaque_copy(v), false, false);
  a = r[0];
  b = r[1];
}
__device__ __forceinline__ float sum16(float v) {
  uint32_t a, b;
  swap16(__builtin_bit_cast(uint32_t, v), a, b);
  return __builtin_bit_cast(float, a) + __builtin_bit_cast(float, b);
}
__device__ __forceinline__ float sum32(float v) {
  uint32_t a, b;
  swap32(__builtin_bit_cast(uint32_t, v), a, b);
  return __builtin_bit_cast(float, a) + __builtin_bit_cast(float, b);
}
__device__ __forceinline__ float max16(float v) {
  uint32_t a, b;
  swap16(__builtin_bit_cast(uint32_t, v), a, b);
  return fmaxf(__builtin_bit_cast(float, a), __builtin_bit_cast(float, b));
}
__device__ __forceinline__ float max32(float v) {
  uint32_t a, b;
  swap32(__builtin_bit_cast(uint32_t, v), a, b);
  return fmaxf(__builtin_bit_cast(float, a), __builtin_bit_cast(float, b));
}
__device__ __forceinline__ uint32_t pkmax16(uint32_t v);
__device__ __forceinline__ uint32_t pkmax32(uint32_t v);

typedef unsigned short ushort2v __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pkmax_u16(uint32_t a, uint32_t b) {
  return __builtin_bit_cast(uint32_t,
                            __builtin_elementwise_max(__builtin_bit_cast(ushort2v, a), __builtin_bit_cast(ushort2v, b)));
}
__device__ __forceinline__ uint32_t pkmax16(uint32_t v) {
  uint32_t a, b;
  swap16(v, a, b);
  return pkmax_u16(a, b);
}
__device__ __forceinline__ uint32_t pkmax32(uint32_t v) {
  uint32_t a, b;
  swap32(v, a, b);
  return pkmax_u16(a, b);
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

// fp16 bit pattern of 2^nvb (nvb in 0..16; 2^16 maps to +inf, which no stored norm reaches).
__device__ __forceinline__ uint32_t norm_threshold(int nvb) { return (uint32_t)(nvb + 15) << 10; }
// Smallest nvb in [nvb0, 16] with every lane's norms (two fp16 halves of `nv`, non-negative and
// finite) below 2^nvb. Wave-uniform; a short scalar loop.
__device__ __forceinline__ int norm_bound(uint32_t nv, int nvb0) {
  const uint32_t x = max(nv & 0xffffu, nv >> 16);
  int nvb = nvb0;
  while (nvb < 16 && __any(x >= norm_threshold(nvb))) ++nvb;
  return nvb;
}

// Scale exponent of the fp16-subnormal code extraction for channel pair j (0..7) of a key word.
__host__ __device__ constexpr int code_shift(int j) { return j <= 4 ? 2 * j : 2 * j - 10; }

// A operand (one token row, channels 8 kk' .. 8 kk' + 7 of the lane group's 32, kk' = kk & 3)
// from the two code words of the lane group: the channel pairs (2j, 2j + 1) of a word sit in
// its two 16-bit halves at bits 2j; pairs 5-7 are shifted down by 10 to stay subnormal.
__device__ __forceinline__ half8 key_a_operand(uint2 w, int kk) {
  const uint32_t d = (kk & 2) ? w.y : w.x;
  if ((kk & 1) == 0) return h8(d & 0x00030003u, d & 0x000c000cu, d & 0x00300030u, d & 0x00c000c0u);
  const uint32_t s = d >> 10;
  return h8(d & 0x03000300u, s & 0x00030003u, s & 0x000c000cu, s & 0x00300030u);
}

// Modality byte tables for v_perm: byte m of a table is 0xff where the modality m is kept.
// Byte 3 is the modality of an invalid token (never kept).
constexpr uint32_t kTabAudio = 0x000000ffu, kTabVideo = 0x0000ff00u, kTabText = 0x00ff0000u;
constexpr uint32_t kTabBits = 0x00040201u;  // byte m -> 1 << m (presence bits)

// ---- the pair ring: each wave streams its window pairs through three LDS slots, filled by direct
// memory-to-LDS loads two pairs ahead of the one it computes. No register holds a pair in flight,
// so the loads of two pairs per wave stay outstanding while the third is computed. The loads are
// issued from inline assembly: the compiler's wait-count model would otherwise make every read of
// the ring wait for all of them; the kernel counts its own loads instead (every one of them is a
// ring load, issued in a fixed number per pair) and waits with explicit vmcnt values. ----
constexpr int kRingSlots = 3;
constexpr int kSlotBytes = 6144;
// byte offsets in a slot: key codes of window A and B (32 tokens x 32 bytes each), value codes of A
// and B (the window's 1024-byte block), metadata, then norms and modality ids
constexpr int kChKA = 0, kChKB = 1024, kChVA = 2048, kChVB = 3072, kChMeta = 4096, kChSmall = 5120;
// the small chunk: key norms of A (64 bytes) and B, value norms of A and B, modality ids of A (32
// bytes) and B
constexpr int kSmKn = 0, kSmVn = 128, kSmMd = 256;
// fp16 steps (window A then B, 256 bytes each) and minima: where the metadata chunk holds them for
// fp16 metadata, and where decoded MXFP4 records are written (after the records, 272 bytes)
template <int kMeta> constexpr int kStepOff = kMeta == kMetaMx ? kChMeta + 512 : kChMeta;
template <int kMeta> constexpr int kMinOff = kMeta == kMetaMx ? kChSmall + 512 : kChMeta + 512;
// ring loads per pair: four code blocks, the small chunk, and the metadata (one 16-byte load per
// lane for fp16, two 4-byte loads for the 272 bytes of two MXFP4 records, none for TurboQuant keys)
template <int kMeta> constexpr int kPairLoads = kMeta == kMetaFp16 ? 6 : kMeta == kMetaMx ? 7 : 5;

// lane's 16 bytes at g go to LDS lds + 16 lane (lds wave-uniform, passed in m0; an LDS load needs
// one wait state after m0 is written)
__device__ __forceinline__ void dma16(const void* g, uint32_t lds) {
  __asm__ volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(g), "{m0}"(lds) : "memory");
}
// lane's 16 bytes at base + off go to LDS lds + 16 lane (base and lds wave-uniform)
__device__ __forceinline__ void dma16s(const void* base, uint32_t off, uint32_t lds) {
  __asm__ volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(off), "s"(base), "{m0}"(lds) : "memory");
}
// lane's 4 bytes at g go to LDS lds + 4 lane
__device__ __forceinline__ void dma4(const void* g, uint32_t lds) {
  __asm__ volatile("s_nop 0\n\tglobal_load_lds_dword %0, off" ::"v"(g), "{m0}"(lds) : "memory");
}
// waits until at most n ring loads of this wave are outstanding (n a multiple of the per-pair
// count, 0..2 pairs)
template <int kMeta>
__device__ __forceinline__ void ring_wait(int newer_pairs) {
  constexpr int c = kPairLoads<kMeta>;
  if (newer_pairs >= 2) {
    __asm__ volatile("s_waitcnt vmcnt(%0)" ::"n"(2 * c) : "memory");
  } else if (newer_pairs == 1) {
    __asm__ volatile("s_waitcnt vmcnt(%0)" ::"n"(c) : "memory");
  } else {
    __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");
  }
}

struct SeqPtrs {  // uniform per work-group
  const uint8_t* kc;
  const uint8_t* vc;
  const uint16_t* kn;
  const uint16_t* vn;
  const uint16_t* kmin;
  const uint16_t* kstep;
  const uint8_t* kmx;
  const uint8_t* md;
};

// Ring loads of window pair (wA, wB) into the slot at LDS address `slot` (wave-uniform arguments;
// wB = wA when the pair has no second window, whose contents are then never used).
template <int kMeta>
__device__ __forceinline__ void issue_pair(const SeqPtrs& sp, uint32_t wA, uint32_t wB, int lane, uint32_t slot) {
  const uint32_t lo = 16u * lane;
  dma16s(sp.kc + (size_t)wA * 1024u, lo, slot + kChKA);
  dma16s(sp.kc + (size_t)wB * 1024u, lo, slot + kChKB);
  dma16s(sp.vc + (size_t)wA * 1024u, lo, slot + kChVA);
  dma16s(sp.vc + (size_t)wB * 1024u, lo, slot + kChVB);
  if constexpr (kMeta == kMetaFp16) {  // lanes 0-15 steps of A, 16-31 of B, 32-47 minima of A, 48-63 of B
    const uint32_t w = (lane & 16) ? wB : wA;
    const uint16_t* base = (lane & 32) ? sp.kmin : sp.kstep;
    dma16(base + w * kD + 8u * (lane & 15), slot + kChMeta);
  } else if constexpr (kMeta == kMetaMx) {  // 68 record dwords: A's 34, then B's
    const uint32_t d = (uint32_t)lane;
    dma4(sp.kmx + (d < 34u ? wA : wB) * (uint32_t)kMxRecord + 4u * (d < 34u ? d : d - 34u), slot + kChMeta);
    if (lane < 4) dma4(sp.kmx + wB * (uint32_t)kMxRecord + 4u * (30u + lane), slot + kChMeta + 256);
  }
  if (lane < 20) {  // key norms A, B (lanes 0-7), value norms A, B (8-15), modality ids A, B (16-19)
    const uint32_t w = (lane < 16 ? (lane & 4) : (lane & 2)) ? wB : wA;
    const uint8_t* src = lane < 8    ? reinterpret_cast<const uint8_t*>(sp.kn + w * kW) + 16u * (lane & 3)
                         : lane < 16 ? reinterpret_cast<const uint8_t*>(sp.vn + w * kW) + 16u * (lane & 3)
                                     : sp.md + w * kW + 16u * (lane & 1);
    dma16(src, slot + kChSmall);
  }
}

// fp16 minimum / step pairs of 4 channels from their MXFP4 record word and block scale bytes: the
// gfx950 scaled FP4 -> fp16 conversion multiplies by 2^(X - 127) and rounds to nearest even. A
// scale byte of 0 (2^-127) is taken as 2^-126: either way the values are below fp16's range and
// convert to zero.
__device__ __forceinline__ void mx_to_f16(uint32_t word, uint32_t scales, uint2& mnp, uint2& stp) {
  const float sm = __builtin_bit_cast(float, max(scales & 0xffu, 1u) << 23);
  const float ss = __builtin_bit_cast(float, max(scales >> 8, 1u) << 23);
  mnp.x = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(word, sm, 0));
  mnp.y = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(word, sm, 1));
  stp.x = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(word, ss, 2));
  stp.y = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(word, ss, 3));
}

// B operand of the value MFMA for 16-channel block nb: code bytes of tokens 4g..4g+3 and
// 16+4g..16+4g+3 of the lane's channel, each turned into four fp16 codebook levels.
__device__ __forceinline__ half8 lut_op(const uint2* vlut, uint4 vc, int nb) {
  const uint32_t vw[4] = {vc.x, vc.y, vc.z, vc.w};
  const uint32_t b0 = (vw[nb >> 2] >> (8 * (nb & 3))) & 0xffu;
  const uint32_t b1 = (vw[2 + (nb >> 2)] >> (8 * (nb & 3))) & 0xffu;
  const uint2 x0 = vlut[b0];
  const uint2 x1 = vlut[b1];
  return h8(x0.x, x0.y, x1.x, x1.y);
}

// TurboQuant key operand (k-block kk of the pair): the codebook values of channels 32 g + 8 kk'
// .. + 7 (kk' = kk & 3) of the lane's token, from the code-byte table: the word's even channels
// sit in one byte and its odd ones in another, so the operand order is c0, c2, c4, c6, c1, c3, c5,
// c7 (the query operand uses the same order).
__device__ __forceinline__ half8 key_a_lut(const uint2* vlut, uint2 w, int kk) {
  const uint32_t d = (kk & 2) ? w.y : w.x;
  const int hb = 8 * (kk & 1);
  const uint2 e = vlut[(d >> hb) & 0xffu];
  const uint2 o = vlut[(d >> (16 + hb)) & 0xffu];
  return h8(e.x, e.y, o.x, o.y);
}

// kGlobal: every value was rotated by R_0 (the single global rotation): one accumulator set whose
// rows 0-7 sum window A's tokens and rows 8-15 window B's, no modality masks, one un-rotation
template <int kMeta, bool kGlobal>
__global__ __launch_bounds__(64 * kDecWaves) void k_decode(DecodeArgs p) {
  constexpr bool kMx = kMeta == kMetaMx;
  constexpr bool kTq = kMeta == kMetaTq;
  // the pair ring (8 waves x 3 slots x 6 KB); after the pair loop the same memory holds the combine
  // tile (per wave [channel][24 rows + 4]: rows 0-7 audio, 8-15 video, 16-23 text heads) and the
  // fp16 A tile of the un-rotation
  __shared__ __attribute__((aligned(16))) uint4 ring_mem[kDecWaves * kRingSlots * kSlotBytes / 16];
  __shared__ __attribute__((aligned(16))) uint2 vlut[256];
  __shared__ __attribute__((aligned(16))) float qs[8][kD + 4];                     // q' (fp32, padded rows)
  __shared__ float amax_w[kDecWaves];
  __shared__ __attribute__((aligned(16))) float wst[2][8][kDecWaves];              // [m, l][head][wave]
  __shared__ uint32_t wmask[kDecWaves];
  __shared__ uint32_t wnv[kDecWaves];  // value-norm maxima
  __shared__ int wexp[kDecWaves];      // operand scale exponents E
  __shared__ __attribute__((aligned(16))) float fac[8][kDecWaves];    // per head and wave: combine factor
  __shared__ __attribute__((aligned(16))) _Float16 atile[8][kATile];  // merged rows, fp16
  static_assert(sizeof(float) * kD * kAccPitch <= kRingSlots * kSlotBytes, "a wave's combine rows fit in its ring");
  uint8_t* const ring = reinterpret_cast<uint8_t*>(ring_mem);

  const int split = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, lane = lane_id();
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform (scalar) for the compiler
  const int col = lane & 15, g = lane >> 4, hd = col & 7, side = col >> 3, c7 = col & 7;
  const size_t seq = (size_t)b * p.H + h;
  float* rec = p.ws + (seq * p.nsplit + split) * kRecFloats;
  const int w_begin = split * p.wps;
  const int w_plan = min(w_begin + p.wps, p.cap / kW);  // windows of this split by the plan
  const int wA0 = w_begin + 2 * wave;                    // this wave's pairs: (wA0 + 16 k, +1)
  const size_t nwcap = p.cap / kW;
  const SeqPtrs sp{p.k_codes + seq * p.cap * 32,
                   p.v_codes + seq * nwcap * 1024,
                   p.k_norm + seq * p.cap,
                   p.v_norm + seq * p.cap,
                   kMeta == kMetaFp16 ? p.k_min + seq * nwcap * kD : nullptr,
                   kMeta == kMetaFp16 ? p.k_step + seq * nwcap * kD : nullptr,
                   kMx ? p.k_mx + seq * nwcap * kMxRecord : nullptr,
                   p.modality + (size_t)b * p.cap};
  const uint32_t ring_w = (uint32_t)__builtin_amdgcn_readfirstlane(
      (int)(uint32_t)(uintptr_t)(ring + (size_t)wave * kRingSlots * kSlotBytes));  // this wave's slots
  auto slot_lds = [&](int k) { return ring_w + (uint32_t)((k % kRingSlots) * kSlotBytes); };
  auto slot_ptr = [&](int k) { return ring + (size_t)wave * kRingSlots * kSlotBytes + (k % kRingSlots) * kSlotBytes; };
  auto pair_w = [&](int k, int w_lim, uint32_t& wA, uint32_t& wB) {
    wA = (uint32_t)(wA0 + 2 * kDecWaves * k);
    wB = (int)wA + 1 < w_lim ? wA + 1 : wA;
  };

  // ---- prologue: every load goes out before any is used. Waves 0-3 first load their two query
  // rows and the signs into slot 2 of their ring (unused until the loop issues a wave's third
  // pair), then every wave loads its first two pairs of the plan (speculatively: the sequence
  // length, a scalar load, is checked after) ----
  // the length first: a scalar load only while no store or ring load precedes it in the kernel
  const int len_dev = p.seq_lens[b];
  const int hr = 2 * wave + (lane >> 5), c4 = 4 * (lane & 31);
  if (wave < 4) {
    const uint32_t qst = ring_w + 2 * kSlotBytes;
    if (lane < 32 && 2 * wave + (lane >> 4) < p.G)  // 16 lanes x 16 bytes per query row
      dma16(p.q + ((size_t)b * p.Hq + h * p.G + 2 * wave) * kD + 8 * lane, qst);
    if (lane < 8) dma16(p.signs + 16 * lane, qst + 512);
  }
  int issued = 0;  // pairs of this wave issued to the ring
  for (; issued < 2 && wA0 + 2 * kDecWaves * issued < w_plan; ++issued) {
    uint32_t wA, wB;
    pair_w(issued, w_plan, wA, wB);
    issue_pair<kMeta>(sp, wA, wB, lane, slot_lds(issued));
  }
  // memory-safe if device and host lengths disagree; with the fp16 residual the last 128 tokens
  // are the merge launch's
  const int len = max(min(len_dev, p.cap) - p.residual, 0);
  const int nwin = (len + kW - 1) / kW;
  const int w_end = min(w_plan, nwin);
  if (w_begin >= w_end) {  // empty split (ragged batch): a header the merge skips
    __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");  // no ring load may land after the exit
    write_empty_record(rec, tid);
    return;
  }

  if (tid < 256) {  // code-byte table: byte -> four fp16 codebook levels (tokens 0..3 of the byte)
    const uint32_t lv[4] = {p.cb01 & 0xffffu, p.cb01 >> 16, p.cb23 & 0xffffu, p.cb23 >> 16};
    vlut[tid] = make_uint2(lv[tid & 3] | (lv[(tid >> 2) & 3] << 16), lv[(tid >> 4) & 3] | (lv[tid >> 6] << 16));
  }
  // ---- query rotation: wave w < 4 rotates heads 2w, 2w+1; lane holds channels c4 .. c4+3 ----
  if (wave < 4) {
    ring_wait<kMeta>(issued);  // the query and sign loads (issued first) have landed
    const uint8_t* qst = slot_ptr(2);
    uint2 qraw = make_uint2(0, 0);
    if (hr < p.G) qraw = *reinterpret_cast<const uint2*>(qst + 256 * (lane >> 5) + 2 * c4);
    const uint32_t qsgn = *reinterpret_cast<const uint32_t*>(qst + 512 + c4);
    float x[4];
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
    *reinterpret_cast<float4*>(&qs[hr][c4]) = make_float4(x[0], x[1], x[2], x[3]);  // zero rows for heads >= G
  }
  __syncthreads();
  const float amax = fmaxf(fmaxf(amax_w[0], amax_w[1]), fmaxf(amax_w[2], amax_w[3]));
  // power-of-two scale k0 keeps |q'_c step_c 2^(k0 - shift)| <= 2^15: |step| <= 2/3 + rounding for
  // fp16 metadata, and below 1 for MXFP4 (a block's largest step rounds up by at most 3/2)
  const int k0 = (amax > 0.0f) ? min(max(14 - ilogbf(amax), -60), 60) : 0;
  // undoes 2^(k0 - 24) on the MFMA result (TurboQuant keys: 2^k0, the codebook values being exact
  // fp16 operands)
  const float kscale = ldexpf(1.0f, kTq ? -k0 : 24 - k0);
  // Per-lane query operand of the score MFMA, constant over the pairs: for channels
  // 32g + 8 k4 .. +7, fp16(q'[hd][c] 2^(k0 - shift(c))).
  uint32_t qm[4][4];
#pragma unroll
  for (int k4 = 0; k4 < 4; ++k4) {
    const float4 qa = *reinterpret_cast<const float4*>(&qs[hd][32 * g + 8 * k4]);
    const float4 qb = *reinterpret_cast<const float4*>(&qs[hd][32 * g + 8 * k4 + 4]);
    const float qv[8] = {qa.x, qa.y, qa.z, qa.w, qb.x, qb.y, qb.z, qb.w};
    if constexpr (kTq) {  // the key operand's order: c0, c2, c4, c6, c1, c3, c5, c7
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int c0 = (j < 2) ? 4 * j : 4 * (j - 2) + 1;
        qm[k4][j] = pack2(ldexpf(qv[c0], k0), ldexpf(qv[c0 + 2], k0));
      }
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j) {  // channel pair 4 (k4 & 1) + j of the word
        const int sh = k0 - code_shift(4 * (k4 & 1) + j);
        qm[k4][j] = pack2(ldexpf(qv[2 * j], sh), ldexpf(qv[2 * j + 1], sh));
      }
    }
  }
  // B operand of the bias MFMA (Eq. 4 linearity: q'.m_g for the pair's two windows): column col
  // holds fp16(q'[hd] 2^k0) for col < 8 and the rounding residual of the same for col >= 8, so that
  // a column pair sums to q' 2^k0 to about 2^-22 relative; channel 32 g + 8 kk + i at k-block kk
  uint32_t qb[4][4];
  if constexpr (!kTq) {
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const float4 qa = *reinterpret_cast<const float4*>(&qs[hd][32 * g + 8 * kk]);
      const float4 qc = *reinterpret_cast<const float4*>(&qs[hd][32 * g + 8 * kk + 4]);
      const float qv[8] = {qa.x, qa.y, qa.z, qa.w, qc.x, qc.y, qc.z, qc.w};
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        float v[2];
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          const float x = ldexpf(qv[2 * j + u], k0);
          const float hi = (float)(_Float16)x;
          v[u] = side ? x - hi : hi;
        }
        qb[kk][j] = pack2(v[0], v[1]);
      }
    }
  }
  const float bscale = ldexpf(1.0f, -k0);
  // modality tables of this lane: its own row half (set 1: audio for side 0, video for side 1),
  // the partner's, and the text rows (side 0 only)
  const uint32_t tab_own = side ? kTabVideo : kTabAudio;
  const uint32_t tab_oth = side ? kTabAudio : kTabVideo;
  const uint32_t tab_txt0 = side ? 0u : kTabText;

  floatx4 acc1[8], acc2[8];  // set 1: audio rows 0-7, video rows 8-15; set 2: text rows 0-7
#pragma unroll
  for (int nb = 0; nb < 8; ++nb) acc1[nb] = acc2[nb] = floatx4{0.f, 0.f, 0.f, 0.f};
  float m_run = -__builtin_inff(), l_run = 0.0f;
  bool started = false;  // a pair has been processed (wave-uniform)
  uint32_t seen = 0;  // modalities seen by this wave
  uint32_t nvm = 0;   // largest value norm seen by this lane (two fp16 halves, non-negative)
  // Operand scale 2^E of p n_v (wave-uniform): every value norm seen so far is below 2^nvb, so
  // with p <= 1 the fp16 product p 2^E n_v stays below 2^15 for E = min(15, 15 - nvb). The
  // accumulators and l_run hold 2^E times the unscaled sums; the combine divides it out.
  int nvb = 0, E = 15;

  auto process = [&](uint8_t* sl, int wA) {
    const bool hasB = wA + 1 < w_end;
    const bool full = hasB && kW * (wA + 2) <= len;  // every token of both windows is valid
    // ---- the pair's data from the slot ----
    const uint2 ka0 = *reinterpret_cast<const uint2*>(sl + kChKA + 32 * col + 8 * g);
    const uint2 ka1 = *reinterpret_cast<const uint2*>(sl + kChKA + 32 * (16 + col) + 8 * g);
    const uint2 kb0 = *reinterpret_cast<const uint2*>(sl + kChKB + 32 * col + 8 * g);
    const uint2 kb1 = *reinterpret_cast<const uint2*>(sl + kChKB + 32 * (16 + col) + 8 * g);
    const uint4 va = *reinterpret_cast<const uint4*>(sl + kChVA + 16 * lane);
    const uint4 vb = *reinterpret_cast<const uint4*>(sl + kChVB + 16 * lane);
    const uint8_t* sm = sl + kChSmall;
    const uint2 nk0 = *reinterpret_cast<const uint2*>(sm + kSmKn + 64 * side + 8 * g);
    const uint2 nk1 = *reinterpret_cast<const uint2*>(sm + kSmKn + 64 * side + 32 + 8 * g);
    const uint2 nv0 = *reinterpret_cast<const uint2*>(sm + kSmVn + 64 * side + 8 * g);
    const uint2 nv1 = *reinterpret_cast<const uint2*>(sm + kSmVn + 64 * side + 32 + 8 * g);
    uint32_t md[2] = {*reinterpret_cast<const uint32_t*>(sm + kSmMd + 32 * side + 4 * g),
                      *reinterpret_cast<const uint32_t*>(sm + kSmMd + 32 * side + 16 + 4 * g)};
    // metadata of the lane's window (side): channels 32 g .. 32 g + 31
    const uint8_t* stp_s = sl + kStepOff<kMeta> + 256 * side + 64 * g;
    if constexpr (kMx) {  // decode the two records into fp16 steps and minima in the slot
      const uint8_t* rec_s = sl + kChMeta + kMxRecord * side;
      const uint32_t word = *reinterpret_cast<const uint32_t*>(rec_s + 4 * (8 * g + c7));
      const uint32_t scales = *reinterpret_cast<const uint16_t*>(rec_s + 128 + 2 * g);
      uint2 mnp, stp;
      mx_to_f16(word, scales, mnp, stp);
      *reinterpret_cast<uint2*>(sl + kStepOff<kMeta> + 256 * side + 64 * g + 8 * c7) = stp;
      *reinterpret_cast<uint2*>(sl + kMinOff<kMeta> + 256 * side + 64 * g + 8 * c7) = mnp;
      wave_lds_sync();
    }

    float bias = 0.0f;  // TurboQuant keys: no window minimum
    if constexpr (!kTq) {
      // ---- bias q'.m of both windows on the matrix cores: A row r holds the minima of window
      // r & 1 (so every lane group's rows 4g, 4g + 1 are windows A, B), B the query's hi and lo
      // parts; a lane adds its column and the partner column (hi + lo) of its side's row ----
      const uint8_t* min_r = sl + kMinOff<kMeta> + 256 * (col & 1) + 64 * g;
      floatx4 bacc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        const uint4 m = *reinterpret_cast<const uint4*>(min_r + 16 * kk);
        bacc = __builtin_amdgcn_mfma_f32_16x16x32_f16(h8(m.x, m.y, m.z, m.w), h8(qb[kk]), bacc, 0, 0, 0);
      }
      const float bA = bacc[0] + fswap8(bacc[0]), bB = bacc[1] + fswap8(bacc[1]);
      bias = (side ? bB : bA) * bscale;
    }

    // ---- scores: two 16-token tiles per window, 4 MFMAs each over the window's 128 channels. The
    // B operand is the lane's own window's q'_c step_c (its column holds that window's head), so the
    // window-A products are kept by the side-0 lanes and the window-B products by the side-1 lanes ----
    floatx4 sA0 = {0.f, 0.f, 0.f, 0.f}, sA1 = sA0, sB0 = sA0, sB1 = sA0;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const uint32_t* q = qm[kk];
      half8 bop;
      if constexpr (kTq) {
        bop = h8(q[0], q[1], q[2], q[3]);
        sA0 = __builtin_amdgcn_mfma_f32_16x16x32_f16(key_a_lut(vlut, ka0, kk), bop, sA0, 0, 0, 0);
        sA1 = __builtin_amdgcn_mfma_f32_16x16x32_f16(key_a_lut(vlut, ka1, kk), bop, sA1, 0, 0, 0);
        sB0 = __builtin_amdgcn_mfma_f32_16x16x32_f16(key_a_lut(vlut, kb0, kk), bop, sB0, 0, 0, 0);
        sB1 = __builtin_amdgcn_mfma_f32_16x16x32_f16(key_a_lut(vlut, kb1, kk), bop, sB1, 0, 0, 0);
      } else {
        const uint4 sv = *reinterpret_cast<const uint4*>(stp_s + 16 * kk);
        bop = h8(pk_mul(q[0], sv.x), pk_mul(q[1], sv.y), pk_mul(q[2], sv.z), pk_mul(q[3], sv.w));
        sA0 = __builtin_amdgcn_mfma_f32_16x16x32_f16(key_a_operand(ka0, kk), bop, sA0, 0, 0, 0);
        sA1 = __builtin_amdgcn_mfma_f32_16x16x32_f16(key_a_operand(ka1, kk), bop, sA1, 0, 0, 0);
        sB0 = __builtin_amdgcn_mfma_f32_16x16x32_f16(key_a_operand(kb0, kk), bop, sB0, 0, 0, 0);
        sB1 = __builtin_amdgcn_mfma_f32_16x16x32_f16(key_a_operand(kb1, kk), bop, sB1, 0, 0, 0);
      }
    }
    const floatx4 sc0 = side ? sB0 : sA0, sc1 = side ? sB1 : sA1;

    // ---- online softmax (base 2) over the pair's 64 tokens. Scores are formed relative to the
    // current reference mref = m_run + kLazy - E (p 2^E = 2^(s - mref)), so that the exponent needs no
    // subtraction; the first pair of the wave and a moved reference shift them once ----
    const uint32_t nkw[4] = {nk0.x, nk0.y, nk1.x, nk1.y};
    const uint32_t nvw[4] = {nv0.x, nv0.y, nv1.x, nv1.y};
    const float mref0 = started ? m_run + kLazy - (float)E : 0.0f;
    float s[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {  // e = 4 t + i: token 16 t + 4 g + i of the side window
      const float raw = (e >> 2) ? sc1[e & 3] : sc0[e & 3];
      const float nkf = (e & 1) ? hi_f16(nkw[e >> 1]) : lo_f16(nkw[e >> 1]);
      s[e] = __builtin_fmaf(nkf, __builtin_fmaf(raw, kscale, bias), -mref0);
    }
    if (!full) {  // partial pair: tokens beyond the length (or a missing window B) do not count
      const bool side_ok = !side || hasB;
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        int lofs = kW * side + 16 * t + 4 * g;  // opaque: not kept live (or spilled) across the loop
        __asm__ volatile("" : "+v"(lofs));
        const int nvalid = side_ok ? min(max(len - (kW * wA + lofs), 0), 4) : 0;
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (i >= nvalid) s[4 * t + i] = -__builtin_inff();
        md[t] |= (nvalid >= 4) ? 0u : (0x03030303u << (8 * nvalid));  // modality 3: invalid
      }
    }
    float wmax = fmaxf(fmaxf(fmaxf(s[0], s[1]), fmaxf(s[2], s[3])), fmaxf(fmaxf(s[4], s[5]), fmaxf(s[6], s[7])));
    wmax = fmaxf(wmax, fswap8(wmax));
    wmax = max32(max16(wmax));
    // running maximum of the lane's value norms (fp16 bits), including this pair's
    nvm = pkmax_u16(nvm, pkmax_u16(pkmax_u16(nvw[0], nvw[1]), pkmax_u16(nvw[2], nvw[3])));
    // lazy rescale: the reference m_run moves only when the max exceeds it by more than 2^8, so
    // p = 2^(s - m_run - 8) <= 1; the scale exponent E moves down only when a value norm reaches
    // 2^nvb (nvb then gets one binade of headroom above the largest norm seen)
    if (!started) {  // first pair: nothing accumulated yet, the reference and the scale are just set
      m_run = wmax;
      nvb = min(norm_bound(nvm, 0) + 1, 16);
      E = min(15, 15 - nvb);
      started = true;
      const float sh = -(m_run + kLazy - (float)E);
#pragma unroll
      for (int e = 0; e < 8; ++e) s[e] += sh;
    } else if (__any(wmax > (float)E) || __any(max(nvm & 0xffffu, nvm >> 16) >= norm_threshold(nvb))) {
      const float m_new = fmaxf(m_run, wmax + mref0);
      const int nb = norm_bound(nvm, nvb);
      const int nvb_new = nb > nvb ? min(nb + 1, 16) : nvb;
      const int E_new = min(15, 15 - nvb_new);
      const float alpha = fast_exp2((m_run - m_new) + (float)(E_new - E));
      l_run *= alpha;
      float arow[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) arow[i] = __shfl(alpha, (4 * g + i) & 7);
#pragma unroll
      for (int nb = 0; nb < 8; ++nb) {
#pragma unroll
        for (int i = 0; i < 4; ++i) acc1[nb][i] *= arow[i];
      }
      if (seen & 4u) {  // text rows hold something
#pragma unroll
        for (int nb = 0; nb < 8; ++nb) {
#pragma unroll
          for (int i = 0; i < 4; ++i) acc2[nb][i] *= arow[i];
        }
      }
      m_run = m_new;
      nvb = nvb_new;
      E = E_new;
      const float sh = mref0 - (m_run + kLazy - (float)E);
#pragma unroll
      for (int e = 0; e < 8; ++e) s[e] += sh;
    }
    float pr[8];  // p 2^E
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      pr[e] = fast_exp2(s[e]);
      l_run += pr[e];
    }
    uint32_t pv[4];  // p 2^E n_v (fp16 pairs), tokens (4g, 4g+1), (4g+2, 4g+3), (16+4g, ..), (16+4g+2, ..)
#pragma unroll
    for (int q = 0; q < 4; ++q) pv[q] = pk_mul(pack_f16(pr[2 * q], pr[2 * q + 1]), nvw[q]);

    // ---- value operands of set 1 (rows 0-7 audio heads from the side-0 lanes, rows 8-15 video
    // heads from the side-1 lanes). A pair of one modality (audio or video, every token valid:
    // tokens past the length carry id 3) takes its rows straight from p n_v; otherwise the
    // operands are masked per token with v_perm byte tables ----
    uint32_t opA[4], opB[4], sel[4];
    bool has_t = false;
    const bool all_v = !kGlobal && __all(md[0] == 0x01010101u && md[1] == 0x01010101u);
    const bool all_a = !kGlobal && __all((md[0] | md[1]) == 0u);
    if (kGlobal) {  // rows 0-7 take window A's p n_v (side-0 lanes), rows 8-15 window B's (side-1 lanes)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        opA[q] = side ? 0u : pv[q];
        opB[q] = side ? pv[q] : 0u;
      }
      seen |= 1u;
    } else if (all_v) {  // window A's video rows come from the side-0 partner, window B's are the lane's own
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        opA[q] = take_partner<0xc>(0u, pv[q]);
        opB[q] = side ? pv[q] : 0u;
      }
      seen |= 2u;
    } else if (all_a) {  // window A's audio rows are the lane's own, window B's come from the side-1 partner
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        opA[q] = side ? 0u : pv[q];
        opB[q] = take_partner<0x3>(0u, pv[q]);
      }
      seen |= 1u;
    } else {  // modalities present (wave-uniform) and the v_perm selectors of the token pairs
      uint32_t pres = __builtin_amdgcn_perm(kTabBits, kTabBits, md[0]) | __builtin_amdgcn_perm(kTabBits, kTabBits, md[1]);
      pres |= pres >> 16;
      pres |= pres >> 8;
      const bool has_a = __any(pres & 1u), has_v = __any(pres & 2u);
      has_t = __any(pres & 4u);
      seen |= (has_a ? 1u : 0u) | (has_v ? 2u : 0u) | (has_t ? 4u : 0u);  // all wave-uniform
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        sel[q] = __builtin_amdgcn_perm(md[q >> 1], md[q >> 1], (q & 1) ? 0x03030202u : 0x01010000u);
        const uint32_t own = pv[q] & __builtin_amdgcn_perm(tab_own, tab_own, sel[q]);
        const uint32_t oth = pv[q] & __builtin_amdgcn_perm(tab_oth, tab_oth, sel[q]);
        opA[q] = take_partner<0xc>(own, oth);  // window A tokens: video rows from the side-0 partner
        opB[q] = take_partner<0x3>(own, oth);  // window B tokens: audio rows from the side-1 partner
      }
    }
    // ---- values: one PV MFMA per window and 16-channel block, set 1 for every pair (a branch
    // around it would give the accumulators two register homes) ----
#pragma unroll
    for (int nb = 0; nb < 8; ++nb) {
      acc1[nb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(h8(opA), lut_op(vlut, va, nb), acc1[nb], 0, 0, 0);
      acc1[nb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(h8(opB), lut_op(vlut, vb, nb), acc1[nb], 0, 0, 0);
    }
    if (has_t) {  // set 2: rows 0-7 text heads (side-0 lanes), rows 8-15 zero
      uint32_t opA[4], opB[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        opA[q] = pv[q] & __builtin_amdgcn_perm(tab_txt0, tab_txt0, sel[q]);
        const uint32_t txt = pv[q] & __builtin_amdgcn_perm(kTabText, kTabText, sel[q]);
        opB[q] = take_partner<0x3>(0u, txt);
      }
#pragma unroll
      for (int nb = 0; nb < 8; ++nb) {
        acc2[nb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(h8(opA), lut_op(vlut, va, nb), acc2[nb], 0, 0, 0);
        acc2[nb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(h8(opB), lut_op(vlut, vb, nb), acc2[nb], 0, 0, 0);
      }
    }
  };

  // ---- window pairs through the ring: issue pair k + 2 (if it has tokens), wait for pair k ----
  int hi = issued - 1;  // highest pair issued
  for (int k = 0;; ++k) {
    const int wA = wA0 + 2 * kDecWaves * k;
    if (wA >= w_end) break;
    if (wA + 4 * kDecWaves < w_end) {
      uint32_t nA, nB;
      pair_w(k + 2, w_end, nA, nB);
      issue_pair<kMeta>(sp, nA, nB, lane, slot_lds(k + 2));
      hi = k + 2;
    }
    ring_wait<kMeta>(hi - k);
    process(slot_ptr(k), wA);
  }
  __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");  // speculative loads of the plan beyond the length

  // ---- epilogue. Waves 0-3 un-rotate: wave w takes output channels 32 w .. 32 w + 31 (two 16-channel
  // blocks), so the merged rows are read by four waves instead of eight. Its slice of the
  // inverse-rotation table (all 384 (modality, k) rows) is loaded first, as MFMA B operands, so
  // that the combine below hides the latency ----
  constexpr int kRotWaves = 4;
  constexpr int kRotBlocks = kGlobal ? 4 : 12;  // k-blocks of the table read (R_0's only when global)
  uint4 rb[2][12];
  if (wave < kRotWaves) {
#pragma unroll
    for (int cb = 0; cb < 2; ++cb) {
      const uint4* rp =
          reinterpret_cast<const uint4*>(p.rot16t) + (size_t)(32 * wave + 16 * cb + (lane & 15)) * 48 + (lane >> 4);
#pragma unroll
      for (int kk = 0; kk < kRotBlocks; ++kk) rb[cb][kk] = rp[4 * kk];
    }
  }

  // ---- combine the waves of the work-group: every wave writes its raw accumulators and its
  // per-head (m, l); the combining threads derive the factors 2^(m_w - M) themselves ----
  l_run += fswap8(l_run);
  l_run = sum32(sum16(l_run));
  {
    uint32_t t = nvm;
    t = pkmax_u16(t, (uint32_t)__builtin_amdgcn_mov_dpp((int)t, kRowRor8, 0xf, 0xf, false));
    t = pkmax32(pkmax16(t));
    t = pkmax_u16(t, (uint32_t)__builtin_amdgcn_mov_dpp((int)t, 0x124, 0xf, 0xf, false));  // row_ror:4
    t = pkmax_u16(t, (uint32_t)__builtin_amdgcn_mov_dpp((int)t, 0x122, 0xf, 0xf, false));  // row_ror:2
    t = pkmax_u16(t, (uint32_t)__builtin_amdgcn_mov_dpp((int)t, 0x121, 0xf, 0xf, false));  // row_ror:1
    nvm = t;
  }
  if (lane < 8) {
    wst[0][lane][wave] = m_run;
    wst[1][lane][wave] = ldexpf(l_run, -E);  // relative to 2^(m_run + kLazy)
  }
  if (lane == 0) {
    wmask[wave] = seen;
    wnv[wave] = max(nvm & 0xffffu, nvm >> 16);
    wexp[wave] = E;
  }
  // the wave's rows go to its own ring slots, free once its last ring load has landed (no other
  // wave writes there), so no barrier precedes them
  auto wacc = [&](int w) { return reinterpret_cast<float(*)[kAccPitch]>(ring + (size_t)w * kRingSlots * kSlotBytes); };
  {
    float(*mine)[kAccPitch] = wacc(wave);
#pragma unroll
    for (int nb = 0; nb < 8; ++nb)  // rows 4g .. 4g + 3 of set 1 (audio, video heads), channel 16 nb + col
      *reinterpret_cast<float4*>(&mine[16 * nb + col][4 * g]) =
          make_float4(acc1[nb][0], acc1[nb][1], acc1[nb][2], acc1[nb][3]);
    if ((seen & 4u) && g < 2) {  // text rows 16 + 4g .. (set 2 rows 0-7), read only for waves that saw text
#pragma unroll
      for (int nb = 0; nb < 8; ++nb)
        *reinterpret_cast<float4*>(&mine[16 * nb + col][16 + 4 * g]) =
            make_float4(acc2[nb][0], acc2[nb][1], acc2[nb][2], acc2[nb][3]);
    }
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
  // factor table fac[head][wave] = 2^(m_w - M - E_w) 2^e / L (zero for heads >= G and empty waves):
  // one thread per (head, wave)
  if (tid < 8 * kDecWaves) {
    const int hh = tid >> 3, w = tid & 7;
    const float4 m0 = *reinterpret_cast<const float4*>(&wst[0][hh][0]);
    const float4 m1 = *reinterpret_cast<const float4*>(&wst[0][hh][4]);
    const float4 l0 = *reinterpret_cast<const float4*>(&wst[1][hh][0]);
    const float4 l1 = *reinterpret_cast<const float4*>(&wst[1][hh][4]);
    const float mv[8] = {m0.x, m0.y, m0.z, m0.w, m1.x, m1.y, m1.z, m1.w};
    const float lv[8] = {l0.x, l0.y, l0.z, l0.w, l1.x, l1.y, l1.z, l1.w};
    float M = mv[0];
#pragma unroll
    for (int u = 1; u < kDecWaves; ++u) M = fmaxf(M, mv[u]);
    float L = 0.0f;
#pragma unroll
    for (int u = 0; u < kDecWaves; ++u) L += (mv[u] == -__builtin_inff()) ? 0.0f : lv[u] * fast_exp2(mv[u] - M);
    const float sc = (hh < p.G && L > 0.0f) ? ldexpf(1.0f / L, e) : 0.0f;
    // the wave's accumulators carry its operand scale 2^E_w
    fac[hh][w] = (mv[w] == -__builtin_inff()) ? 0.0f : fast_exp2(mv[w] - M - (float)wexp[w]) * sc;
    if (w == 0) {
      rec[hh] = M;
      rec[8 + hh] = L;
    }
  }
  __syncthreads();
  // rows summed over the waves with their factors -> A tile [head][128 m + k] (fp16); thread =
  // (row quad rq, channel k), rows 4 rq .. 4 rq + 3 = heads 4 (rq & 1) .. +3 of modality rq / 2
  // (global rotation: two row quads, each the sum of rows 4 rq .. and 8 + 4 rq .., the two windows' parts)
  for (int idx = tid; idx < (kGlobal ? 2 : 6) * kD; idx += 64 * kDecWaves) {
    const int rq = idx >> 7, k = idx & (kD - 1), m = rq >> 1, h0 = 4 * (rq & 1);
    if (!(mask & (1u << m))) continue;
    float a[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int w4 = 0; w4 < kDecWaves; w4 += 4) {
      float4 f[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) f[i] = *reinterpret_cast<const float4*>(&fac[h0 + i][w4]);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        if (!(wmask[w4 + u] & (1u << m))) continue;  // that wave saw no token of this modality
        float4 v = *reinterpret_cast<const float4*>(&wacc(w4 + u)[k][4 * rq]);
        if constexpr (kGlobal) {
          const float4 v2 = *reinterpret_cast<const float4*>(&wacc(w4 + u)[k][8 + 4 * rq]);
          v = make_float4(v.x + v2.x, v.y + v2.y, v.z + v2.z, v.w + v2.w);
        }
        const float fu[4] = {u == 0 ? f[0].x : u == 1 ? f[0].y : u == 2 ? f[0].z : f[0].w,
                             u == 0 ? f[1].x : u == 1 ? f[1].y : u == 2 ? f[1].z : f[1].w,
                             u == 0 ? f[2].x : u == 1 ? f[2].y : u == 2 ? f[2].z : f[2].w,
                             u == 0 ? f[3].x : u == 1 ? f[3].y : u == 2 ? f[3].z : f[3].w};
        a[0] = __builtin_fmaf(v.x, fu[0], a[0]);
        a[1] = __builtin_fmaf(v.y, fu[1], a[1]);
        a[2] = __builtin_fmaf(v.z, fu[2], a[2]);
        a[3] = __builtin_fmaf(v.w, fu[3], a[3]);
      }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) atile[h0 + i][m * kD + k] = (_Float16)a[i];
  }
  __syncthreads();
  // ---- inverse rotation on MFMA, once per present modality: wave w < 4 computes channels
  // c = 32 w .. 32 w + 31 of o[head][c] = sum_m sum_k A[head][128 m + k] R_m[k][c]. A rows 8-15
  // (lanes whose row is >= 8) only feed output rows that are not stored. ----
  if (wave >= kRotWaves) return;
  floatx4 dacc[2] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
#pragma unroll
  for (int m = 0; m < (kGlobal ? 1 : 3); ++m) {
    if (!(mask & (1u << m))) continue;
#pragma unroll
    for (int k4 = 0; k4 < 4; ++k4) {
      const int kk = 4 * m + k4;
      const half8 a = *reinterpret_cast<const half8*>(&atile[lane & 7][32 * kk + 8 * (lane >> 4)]);
#pragma unroll
      for (int cb = 0; cb < 2; ++cb)
        dacc[cb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, __builtin_bit_cast(half8, rb[cb][kk]), dacc[cb], 0, 0, 0);
    }
  }
  if (lane < 32) {
    const float sc = ldexpf(1.0f, -e);
#pragma unroll
    for (int cb = 0; cb < 2; ++cb) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
        rec[kRecHeader + (4 * (lane >> 4) + i) * kD + 32 * wave + 16 * cb + (lane & 15)] = dacc[cb][i] * sc;
    }
  }
}

// ---- merge over splits: o = sum_s 2^(M_s - M) L_s o_s / sum_s 2^(M_s - M) L_s (log-sum-exp) ----
// One work-group of 256 threads per (query head j, sequence b): thread (split group sg, channel
// quad q4) sums the splits s = sg (mod 8). Every load is issued before any is used; empty splits
// carry M = -inf and are skipped (their outputs are zeros). A record's L is relative to
// 2^(M + kLazy) (the split kernel's lazily updated reference).
constexpr int kMergeThreads = 256;
constexpr int kMergeUnroll = 8;  // splits per thread held in registers at once

// Eight split records of one chunk (splits s0, s0 + 8, ..., s0 + 56) for query head hd and channel
// quad q4, as loaded; the fold treats splits beyond nsplit (read through a clamped index) as empty.
struct SplitChunk {
  float ms[kMergeUnroll], ls[kMergeUnroll];
  float4 v[kMergeUnroll];
  int s0, nsplit;
};

__device__ __forceinline__ void load_split_chunk(const float* base, int nsplit, int hd, int q4, int s0, SplitChunk& c) {
#pragma unroll
  for (int u = 0; u < kMergeUnroll; ++u) {
    const int s = s0 + 8 * u;
    const float* rs = base + (size_t)min(s, nsplit - 1) * kRecFloats;
    // loaded unconditionally (the record index is clamped) and selected in the fold: a conditional
    // load is compiled as a branch, after which the wait before the fold covers every load in flight
    // and the chunk's last loads go out a round trip late; a select here would wait for the load
    // before any later load of the caller goes out
    c.ms[u] = rs[hd];
    c.ls[u] = rs[8 + hd];
    c.v[u] = *reinterpret_cast<const float4*>(rs + kRecHeader + hd * kD + 4 * q4);
  }
  c.s0 = s0;
  c.nsplit = nsplit;
  __builtin_amdgcn_sched_barrier(0);  // the whole chunk's loads go out before the fold
}

// folds a chunk into the running (M, L, o). Branch-free (selects): with a branch here the compiler
// sinks the chunk's weight and output loads below it, a second round trip. Empty splits (M = -inf)
// add nothing: their weight is selected to zero and their outputs are zeros (records past nsplit,
// read through the clamped index, are selected away).
__device__ __forceinline__ void fold_split_chunk(const SplitChunk& c, float& M, float& L, float4& o) {
  float ms[kMergeUnroll];
#pragma unroll
  for (int u = 0; u < kMergeUnroll; ++u) ms[u] = (c.s0 + 8 * u < c.nsplit) ? c.ms[u] : -__builtin_inff();
  float mc = M;
#pragma unroll
  for (int u = 0; u < kMergeUnroll; ++u) mc = fmaxf(mc, ms[u]);
  const bool any = mc != -__builtin_inff();
  const float a = any ? exp2f(M - mc) : 1.0f;  // M = -inf -> 0
  L *= a;
  o.x *= a;
  o.y *= a;
  o.z *= a;
  o.w *= a;
#pragma unroll
  for (int u = 0; u < kMergeUnroll; ++u) {
    const bool live = ms[u] != -__builtin_inff();
    const float w = live ? exp2f(ms[u] - mc) * c.ls[u] : 0.0f;
    L = live ? L + w : L;
    o.x = live ? __builtin_fmaf(w, c.v[u].x, o.x) : o.x;
    o.y = live ? __builtin_fmaf(w, c.v[u].y, o.y) : o.y;
    o.z = live ? __builtin_fmaf(w, c.v[u].z, o.z) : o.z;
    o.w = live ? __builtin_fmaf(w, c.v[u].w, o.w) : o.w;
  }
  M = any ? mc : M;
}

// running (M, L, o) over the splits s = sg (mod 8) of one (sequence, KV head), query head hd
__device__ __forceinline__ void merge_splits(const float* base, int nsplit, int hd, int sg, int q4, float& M,
                                             float& L, float4& o) {
  o = make_float4(0.f, 0.f, 0.f, 0.f);
  M = -__builtin_inff();
  L = 0.0f;
  for (int s0 = sg; s0 < nsplit; s0 += 8 * kMergeUnroll) {
    SplitChunk c;
    load_split_chunk(base, nsplit, hd, q4, s0, c);
    fold_split_chunk(c, M, L, o);
  }
}

// The 8 split groups combined: every group rescaled to the global max Mt; lanes of tid < 32 end
// with the summed outputs of channels 4 tid .. 4 tid + 3 in `t` and the summed L in `Lt`.
__device__ __forceinline__ void combine_groups(float M, float L, float4 o, int tid, float (&red)[2][kMergeThreads / 64],
                                               float4 (&part)[8][32], float& Mt, float& Lt, float4& t) {
  const int lane = tid & 63, wave = tid >> 6, q4 = tid & 31, sg = tid >> 5;
  float mw = wave_max(M);
  if (lane == 0) red[0][wave] = mw;
  __syncthreads();
  Mt = red[0][0];
#pragma unroll
  for (int w = 1; w < kMergeThreads / 64; ++w) Mt = fmaxf(Mt, red[0][w]);
  const float a = (M == -__builtin_inff()) ? 0.0f : exp2f(M - Mt);
  // L is the same for every channel quad of a split group: count it once per group
  float lw = (q4 == 0) ? L * a : 0.0f;
  lw = wave_sum(lw);
  if (lane == 0) red[1][wave] = lw;
  part[sg][q4] = make_float4(o.x * a, o.y * a, o.z * a, o.w * a);
  __syncthreads();
  Lt = 0.0f;
  t = make_float4(0.f, 0.f, 0.f, 0.f);
  if (tid < 32) {
#pragma unroll
    for (int w = 0; w < kMergeThreads / 64; ++w) Lt += red[1][w];
    t = part[0][tid];
#pragma unroll
    for (int g = 1; g < 8; ++g) {
      const float4 u = part[g][tid];
      t.x += u.x;
      t.y += u.y;
      t.z += u.z;
      t.w += u.w;
    }
  }
}

__global__ __launch_bounds__(kMergeThreads) void k_decode_merge(const float* __restrict__ ws, int H, int Hq, int G,
                                                                int nsplit, float* __restrict__ out) {
  __shared__ float red[2][kMergeThreads / 64];
  __shared__ __attribute__((aligned(16))) float4 part[8][32];
  const int j = blockIdx.x, b = blockIdx.y;
  const int h = j / G, hd = j % G;
  const int tid = threadIdx.x;
  float M, L, Mt, Lt;
  float4 o, t;
  merge_splits(ws + ((size_t)b * H + h) * nsplit * kRecFloats, nsplit, hd, tid >> 5, tid & 31, M, L, o);
  combine_groups(M, L, o, tid, red, part, Mt, Lt, t);
  if (tid < 32) {
    const float inv = (Lt > 0.0f) ? 1.0f / Lt : 0.0f;
    *reinterpret_cast<float4*>(out + ((size_t)b * Hq + j) * kD + 4 * tid) =
        make_float4(t.x * inv, t.y * inv, t.z * inv, t.w * inv);
  }
}

// ---- merge with the fp16 residual of the captioning protocol (Sec. 3.1) ----
// The split kernel covered the tokens below L - 128. This work-group also attends query head j
// over the last nt = min(L, 128) tokens [T0, L): key i dequantized from the cache if
// i < Kq = 128 floor(L / 128) (scored against the rotated query, Sec. 2.3), else read in fp16 from
// k_res (scored against the query itself; the rotation is orthogonal); every value in fp16 from
// v_res. Its (max, sum, unnormalized output) joins the splits' log-sum-exp merge. fp32 throughout.
struct TailArgs {
  const int32_t* seq_lens;
  const uint16_t* q;       // [B][Hq][128] fp16
  const int8_t* signs;     // [128]
  const uint8_t* k_codes;
  const uint16_t* k_norm;
  const uint16_t* k_min;   // fp16 window metadata, or
  const uint16_t* k_step;
  const uint8_t* k_mx;     // MXFP4 window records (non-null selects this format)
  const uint16_t* k_res;   // [B][H][128][128] fp16 rings
  const uint16_t* v_res;
  int cap;
  float qscale;            // sm_scale * log2(e): scores in base 2
};

__global__ __launch_bounds__(kMergeThreads) void k_decode_merge_residual(const float* __restrict__ ws, int H, int Hq,
                                                                         int G, int nsplit, float* __restrict__ out,
                                                                         TailArgs ta) {
  __shared__ float red[2][kMergeThreads / 64];
  __shared__ __attribute__((aligned(16))) float4 part[8][32];
  __shared__ __attribute__((aligned(16))) float qp[kD];   // q sm_scale log2(e)
  __shared__ __attribute__((aligned(16))) float qr[kD];   // H q sm_scale log2(e) (rotated query)
  __shared__ float ps[kResidual];                         // tail scores, then weights
  __shared__ __attribute__((aligned(16))) float ot[16][kD];  // tail output partials, 16 token groups
  __shared__ float tred[kMergeThreads / 64];
  __shared__ __attribute__((aligned(16))) float mst[4][2][kD];  // (minimum, step) of the tail's quantized windows
  const int j = blockIdx.x, b = blockIdx.y;
  const int h = j / G, hd = j % G;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int sg = tid >> 5, q4 = tid & 31;
  const size_t seq = (size_t)b * H + h;
  const float* base = ws + seq * nsplit * kRecFloats;

  // ---- every load goes out before any is used: the first chunk of split records, then (once the
  // length is known) the query, the metadata of the tail's quantized windows, the tail's keys
  // (codes and norms, or fp16 rows) and the value rows this thread sums ----
  const int len_dev = ta.seq_lens[b];  // first, a scalar load in flight while the records' loads go out
  SplitChunk ch0;
  if (sg < nsplit) load_split_chunk(base, nsplit, hd, q4, sg, ch0);
  const int L = min(max(len_dev, 0), ta.cap);
  const int T0 = max(L - kResidual, 0), nt = L - T0, Kq = L & ~(kResidual - 1);
  // quantized keys [T0, Kq) lie in windows w0 .. w0 + 3 (Kq - T0 <= 128 and Kq is window aligned)
  const int w0 = T0 / kW, nwq = (Kq > T0) ? (Kq - 1) / kW - w0 + 1 : 0;
  // loaded by every thread (channel tid mod 128) and used after the barrier: a load inside a branch
  // gets its use pulled in behind it, and the wait there holds back every later load
  const uint32_t qx = ta.q[((size_t)b * Hq + j) * kD + (tid & (kD - 1))];
  // and, for the rotation in wave 0, channels 4 l .. 4 l + 3 of lane l (mod 32) with their signs
  const uint2 qrow4 = *reinterpret_cast<const uint2*>(ta.q + ((size_t)b * Hq + j) * kD + 4 * (lane & 31));
  const uint32_t s4 = *reinterpret_cast<const uint32_t*>(ta.signs + 4 * (lane & 31));
  // metadata entries idx = tid, tid + 256 of the (window, channel) table, as loaded (entries past the
  // tail's windows read window w0's, never used): fp16 minimum and step, or the MXFP4 record's
  // nibble bytes and block scales (channel 4q + i in nibble i of bytes 4q, 4q + 1 (minimum), 4q + 2,
  // 4q + 3 (step); scales at 128 + 2 (c / 32), + 1)
  uint32_t mraw[2], sraw[2], mnib[2], snib[2], scl[2];
  {
    // both formats' loads on every path (no branch: a branch between loads makes later ones wait
    // behind earlier ones), from valid addresses: with MXFP4 records the fp16 loads read record bytes,
    // and without them the record loads read the same window's fp16 minima (a record's bytes lie within
    // its window's 256-byte row); the format picks which to decode
    const bool mx = ta.k_mx != nullptr;
    const uint16_t* kmin = mx ? reinterpret_cast<const uint16_t*>(ta.k_mx) : ta.k_min;
    const uint16_t* kstep = mx ? reinterpret_cast<const uint16_t*>(ta.k_mx) : ta.k_step;
    const uint8_t* kmx = mx ? ta.k_mx : reinterpret_cast<const uint8_t*>(ta.k_min);
    const size_t mxstride = mx ? kMxRecord : 2 * kD;
#pragma unroll
    for (int r = 0; r < 2; ++r) {
      const int idx = tid + kMergeThreads * r;
      const int ic = (idx < nwq * kD) ? idx : (idx & (kD - 1));
      const int wi = ic >> 7, c = ic & (kD - 1);
      const size_t w = seq * (ta.cap / kW) + w0 + wi;
      mraw[r] = kmin[mx ? 0 : w * kD + c];
      sraw[r] = kstep[mx ? 0 : w * kD + c];
      const uint8_t* rec = kmx + w * mxstride;
      const int qq = c >> 2, i = c & 3;
      mnib[r] = rec[4 * qq + (i >> 1)];
      snib[r] = rec[4 * qq + 2 + (i >> 1)];
      scl[r] = *reinterpret_cast<const uint16_t*>(rec + 128 + 2 * (c >> 5));  // minimum's scale, step's scale
    }
  }
  // scores: two threads per token tt = tid / 2, channels 64 half .. 64 half + 63
  const int tt = tid >> 1, half = tid & 1, ti = T0 + tt;
  const bool tok = tt < nt, quant = tok && ti < Kq;
  // both forms of the token's key, loaded by every thread (clamped indices, branch-free): a load in
  // a branch makes later loads wait behind it (the two branches share registers)
  const int tc = min(ti, ta.cap - 1);
  const uint4 kq = *reinterpret_cast<const uint4*>(ta.k_codes + (seq * ta.cap + tc) * 32 + 16 * half);
  const uint32_t knrm = ta.k_norm[seq * ta.cap + tc];
  uint4 kr[8];
  {  // the token's ring row, or ring row 0 for a quantized key (one shared line, never used)
    const int rr = quant ? 0 : (ti & (kResidual - 1));
    const uint4* row = reinterpret_cast<const uint4*>(ta.k_res + (seq * kResidual + rr) * kD + 64 * half);
#pragma unroll
    for (int u = 0; u < 8; ++u) kr[u] = row[u];
  }
  // output: thread (channel octet c8, token group tg) sums tokens tg, tg + 16, ..., tg + 112 (16-byte
  // loads: a wave keeps fewer than 64 loads in flight, the most its counter tracks)
  const int c8 = tid & 15, tg = tid >> 4;
  uint4 vv[kResidual / 16];
  {
    const uint4* vr = reinterpret_cast<const uint4*>(ta.v_res + seq * kResidual * kD) + c8;
#pragma unroll
    for (int u = 0; u < kResidual / 16; ++u)  // every ring row (finite); rows past the tail get weight 0
      vv[u] = vr[((T0 + tg + 16 * u) & (kResidual - 1)) * (kD / 8)];
  }
  __builtin_amdgcn_sched_barrier(0);  // every load above goes out before the first use

  // ---- the query, plain and rotated (wave 0: the butterflies in registers), the metadata as fp32 ----
  if (tid < kD) qp[tid] = h2f(qx) * ta.qscale;
  if (wave == 0) {  // Sylvester order, h ascending: channel bits 0, 1 in the lane, bits 2..6 = lane bits 0..4
    const uint32_t qw[2] = {qrow4.x, qrow4.y};
    float x[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float v = h2f((qw[i >> 1] >> (16 * (i & 1))) & 0xffffu);
      x[i] = ((s4 >> (8 * i + 7)) & 1u) ? -v : v;
    }
    {
      const float a = x[0] + x[1], c = x[0] - x[1], d = x[2] + x[3], e = x[2] - x[3];
      x[0] = a + d;
      x[2] = a - d;
      x[1] = c + e;
      x[3] = c - e;
    }
#pragma unroll
    for (int lb = 1; lb < 32; lb <<= 1) {
      const bool hi = (lane & lb) != 0;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float o = __shfl_xor(x[i], lb);
        x[i] = hi ? o - x[i] : x[i] + o;
      }
    }
    const float sc = ta.qscale * 0.08838834764831845f;  // 1 / sqrt(128): H is orthonormal
    if (lane < 32) *reinterpret_cast<float4*>(&qr[4 * lane]) = make_float4(x[0] * sc, x[1] * sc, x[2] * sc, x[3] * sc);
  }
#pragma unroll
  for (int r = 0; r < 2; ++r) {
    const int idx = tid + kMergeThreads * r;
    if (idx < nwq * kD) {
      float mn, st;
      if (ta.k_mx) {
        const int i = idx & 3;
        mn = e2m1_decode((mnib[r] >> (4 * (i & 1))) & 15u, (int)(scl[r] & 0xffu) - 127);
        st = e2m1_decode((snib[r] >> (4 * (i & 1))) & 15u, (int)(scl[r] >> 8) - 127);
      } else {
        mn = h2f(mraw[r]);
        st = h2f(sraw[r]);
      }
      mst[idx >> 7][0][idx & (kD - 1)] = mn;
      mst[idx >> 7][1][idx & (kD - 1)] = st;
    }
  }
  __syncthreads();

  // ---- tail scores ----
  {
    float sc = -__builtin_inff();
    if (tok) {
      float acc = 0.0f;
      if (quant) {  // n16 (q' . (m + step code)) over the window's metadata
        const uint32_t words[4] = {kq.x, kq.y, kq.z, kq.w};
        const float* mrow = mst[ti / kW - w0][0];
        const float* srow = mst[ti / kW - w0][1];
#pragma unroll
        for (int cc = 0; cc < 64; ++cc) {
          const int c = 64 * half + cc;
          const uint32_t code = (words[cc >> 4] >> (16 * (c & 1) + (c & 14))) & 3u;
          acc = __builtin_fmaf(qr[c], __builtin_fmaf(srow[c], (float)code, mrow[c]), acc);
        }
        acc *= h2f(knrm);
      } else {  // fp16 key from the ring
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const uint32_t xs[4] = {kr[u].x, kr[u].y, kr[u].z, kr[u].w};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int c = 64 * half + 8 * u + 2 * e;
            acc = __builtin_fmaf(qp[c], h2f(xs[e] & 0xffffu), acc);
            acc = __builtin_fmaf(qp[c + 1], h2f(xs[e] >> 16), acc);
          }
        }
      }
      acc += __shfl_xor(acc, 1);  // the token's two threads are both active or both not
      sc = acc;
    }
    if (half == 0) ps[tt] = sc;
    float mw = wave_max(sc);
    if (lane == 0) tred[wave] = mw;
  }
  __syncthreads();
  float mtail = tred[0];
#pragma unroll
  for (int w = 1; w < kMergeThreads / 64; ++w) mtail = fmaxf(mtail, tred[w]);
  // weights 2^(s - mtail) (mtail = -inf only for an empty tail, which has no tokens)
  if (tid < nt) ps[tid] = exp2f(ps[tid] - mtail);
  __syncthreads();
  {
    float o[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int u = 0; u < kResidual / 16; ++u) {
      const int t2 = tg + 16 * u;
      const float p = (t2 < nt) ? ps[t2] : 0.0f;
      const uint32_t w4[4] = {vv[u].x, vv[u].y, vv[u].z, vv[u].w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        o[2 * e] = __builtin_fmaf(p, h2f(w4[e] & 0xffffu), o[2 * e]);
        o[2 * e + 1] = __builtin_fmaf(p, h2f(w4[e] >> 16), o[2 * e + 1]);
      }
    }
    *reinterpret_cast<float4*>(&ot[tg][8 * c8]) = make_float4(o[0], o[1], o[2], o[3]);
    *reinterpret_cast<float4*>(&ot[tg][8 * c8 + 4]) = make_float4(o[4], o[5], o[6], o[7]);
  }
  if (wave == 0) {  // sum of the weights
    float lsum = 0.0f;
    for (int t2 = lane; t2 < nt; t2 += 64) lsum += ps[t2];
    lsum = wave_sum(lsum);
    if (lane == 0) tred[0] = lsum;
  }

  // ---- the splits, then everything in the frame of the true maximum ----
  float M = -__builtin_inff(), Ls = 0.0f, Mt, Lt;
  float4 o = make_float4(0.f, 0.f, 0.f, 0.f), t;
  if (sg < nsplit) fold_split_chunk(ch0, M, Ls, o);
  for (int s0 = sg + 8 * kMergeUnroll; s0 < nsplit; s0 += 8 * kMergeUnroll) {
    SplitChunk c;
    load_split_chunk(base, nsplit, hd, q4, s0, c);
    fold_split_chunk(c, M, Ls, o);
  }
  combine_groups(M, Ls, o, tid, red, part, Mt, Lt, t);  // (its barriers also order the tail's LDS writes)
  const float ltail = tred[0];
  if (tid < 32) {
    const float mref = Mt + kLazy;  // the splits' sums are relative to 2^(Mt + kLazy)
    const float mf = fmaxf(mref, mtail);
    const float as = (Mt == -__builtin_inff()) ? 0.0f : exp2f(mref - mf);
    const float at = (nt == 0) ? 0.0f : exp2f(mtail - mf);
    const float ltot = Lt * as + ltail * at;
    const float inv = (ltot > 0.0f) ? 1.0f / ltot : 0.0f;
    float4 tv = *reinterpret_cast<const float4*>(&ot[0][4 * tid]);
#pragma unroll
    for (int g2 = 1; g2 < 16; ++g2) {
      const float4 u = *reinterpret_cast<const float4*>(&ot[g2][4 * tid]);
      tv = make_float4(tv.x + u.x, tv.y + u.y, tv.z + u.z, tv.w + u.w);
    }
    const float r[4] = {(t.x * as + tv.x * at) * inv, (t.y * as + tv.y * at) * inv, (t.z * as + tv.z * at) * inv,
                        (t.w * as + tv.w * at) * inv};
    *reinterpret_cast<float4*>(out + ((size_t)b * Hq + j) * kD + 4 * tid) = make_float4(r[0], r[1], r[2], r[3]);
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
                         hipEvent_t const* events, bool global_rot) {
  const int G = c.Hq / c.H;
  DecodeArgs a;
  a.k_codes = c.k_codes;
  a.v_codes = c.v_codes;
  a.k_norm = c.k_norm;
  a.v_norm = c.v_norm;
  a.k_min = c.k_min;
  a.k_step = c.k_step;
  a.k_mx = c.k_mx;
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
  a.residual = c.residual;
  a.qscale = sm_scale * 1.4426950408889634f * 0.08838834764831845f;
  a.cb01 = cb01;
  a.cb23 = cb23;
  hipError_t e;
  const dim3 grid(plan.nsplit, c.H, c.B), block(64 * kDecWaves);
  auto kern = global_rot ? (c.key_meta == kMetaMx   ? k_decode<kMetaMx, true>
                            : c.key_meta == kMetaTq ? k_decode<kMetaTq, true>
                                                    : k_decode<kMetaFp16, true>)
                         : (c.key_meta == kMetaMx   ? k_decode<kMetaMx, false>
                            : c.key_meta == kMetaTq ? k_decode<kMetaTq, false>
                                                    : k_decode<kMetaFp16, false>);
  if (events)  // events bound to the two dispatches: start and end of each kernel's execution
    hipExtLaunchKernelGGL(kern, grid, block, 0, s, events[0], events[1], 0, a);
  else
    hipLaunchKernelGGL(kern, grid, block, 0, s, a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  const dim3 mgrid(c.Hq, c.B), mblock(kMergeThreads);
  if (c.residual) {
    TailArgs t;
    t.seq_lens = c.seq_lens;
    t.q = q;
    t.signs = c.signs;
    t.k_codes = c.k_codes;
    t.k_norm = c.k_norm;
    t.k_min = c.k_min;
    t.k_step = c.k_step;
    t.k_mx = c.k_mx;
    t.k_res = c.k_res;
    t.v_res = c.v_res;
    t.cap = c.cap;
    t.qscale = sm_scale * 1.4426950408889634f;
    if (events)
      hipExtLaunchKernelGGL(k_decode_merge_residual, mgrid, mblock, 0, s, events[2], events[3], 0,
                            static_cast<const float*>(a.ws), c.H, c.Hq, G, plan.nsplit, out, t);
    else
      hipLaunchKernelGGL(k_decode_merge_residual, mgrid, mblock, 0, s, static_cast<const float*>(a.ws), c.H, c.Hq, G,
                         plan.nsplit, out, t);
  } else if (events) {
    hipExtLaunchKernelGGL(k_decode_merge, mgrid, mblock, 0, s, events[2], events[3], 0,
                          static_cast<const float*>(a.ws), c.H, c.Hq, G, plan.nsplit, out);
  } else {
    hipLaunchKernelGGL(k_decode_merge, mgrid, mblock, 0, s, static_cast<const float*>(a.ws), c.H, c.Hq, G,
                       plan.nsplit, out);
  }
  return hipGetLastError();
}

hipError_t launch_decode_merge(const float* ws, int B, int H, int Hq, int nsplit, float* out, hipStream_t s,
                               hipEvent_t const* events) {
  const dim3 mgrid(Hq, B), mblock(kMergeThreads);
  const int G = Hq / H;
  if (events)
    hipExtLaunchKernelGGL(k_decode_merge, mgrid, mblock, 0, s, events[0], events[1], 0, ws, H, Hq, G, nsplit, out);
  else
    hipLaunchKernelGGL(k_decode_merge, mgrid, mblock, 0, s, ws, H, Hq, G, nsplit, out);
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
