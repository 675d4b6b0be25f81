// Key and value codecs of append and of the stateless MFMA-mode calls, in one persistent launch
// (Sec. 2.1 Eq. 2 and Sec. 2.3 Eq. 4 for keys; Sec. 2.3 Eq. 6 with the codebook of Eq. 3 for
// values).
//
// Work unit: a tile of 256 consecutive tokens of one (sequence, KV head), counted from the
// sequence's first open window. A work-group has one or both of two roles, fixed per wave:
//  * key waves (4): wave k quantizes tokens [64 k, 64 k + 64) of the tile (key_quant.hpp);
//  * value waves (4): phase 1 -- wave v loads the rows of tokens [64 v, 64 v + 64) straight into
//    the work-group's LDS A tile and puts their fp16 norms, decision scales and per-modality
//    token masks into a work-group table; phase 2 -- wave v takes
//    output channels [32 v, 32 v + 32) of all 256 tokens: y = R_m v on the matrix cores with the
//    wave's slice of R_m held in registers as MFMA B operands (fp16 hi + lo, fp32 accumulation),
//    one modality at a time, then the codes.
// Key waves never wait for value waves. The value waves synchronize twice per tile (tables
// written -> read -> free again) through an arrival counter in LDS, not a work-group barrier, so the key waves' VALU work overlaps the
// value waves' loads and MFMAs on the same SIMDs. The grid is persistent: work-group i walks the
// tiles i, i + gridDim.x, ...; a key wave loads its next tile's rows straight into LDS while it
// computes the codes of the current one.
//
// Value decision: the thresholds are symmetric (-T, 0, T with T = fl(n16 tau_2)), so the code is
// clamp(floor(y fl(1/T)) + 2, 0, 3). At 0 it is exact (the product has the sign of y); at +-T it
// can differ from the comparisons only where y lies within about 2^-21 T of the threshold, far
// inside the 2^-16 sum_j |R_cj v_j| band (at least 2^-16 |y|) that separates MFMA mode from the
// sequential order.
//
// MFMA 16x16x32 f16 lane mapping (wave64): lane l holds A[l % 16][8 (l / 16) + e], e = 0..7,
// B[8 (l / 16) + e][l % 16], and D[4 (l / 16) + i][l % 16], i = 0..3. With rows = tokens and
// columns = output channels, lane l ends with channel 16 nb + l % 16 of four consecutive tokens:
// one byte of the value-code layout, at offset 16 l + 8 (rb & 1) + nb of the window block.
#include <hip/hip_ext.h>

#include <algorithm>
#include <cstdlib>

#include "key_quant.hpp"
#include "launch.hpp"

namespace okvq {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ half8 as_half8(uint4 u) { return __builtin_bit_cast(half8, u); }

constexpr int kTile = 256;          // tokens per tile
constexpr int kSpinLimit = 1 << 22;  // polls of the value-wave arrival counter before giving up

struct TileCtx {
  int b, bz, h;
  size_t seq;
  int begin, len;  // the tokens [begin, len) are new (stateless: begin = 0)
  int first;       // first token of the first open window
  int tile0;       // first token of the tile
};

// Tile t of the launch from the host's lengths; t enumerates (x, h, bz), x fastest.
__device__ __forceinline__ TileCtx tile_from_hint(const CodecJob& j, int ntx, int t) {
  TileCtx c;
  const int x = t % ntx, r = t / ntx;
  c.h = r % j.H;
  c.bz = r / j.H;
  c.b = j.b0 + c.bz;
  c.seq = (size_t)c.b * j.H + c.h;
  if (j.begin_dev) {
    c.begin = j.lens.lens[c.bz];
    c.len = c.begin + j.cnts.lens[c.bz];
  } else {
    c.begin = 0;
    c.len = j.lens.lens[c.bz];
  }
  c.first = (c.begin / kW) * kW;
  c.tile0 = c.first + kTile * x;
  return c;
}

// Append: the device lengths decide (clamped, so that values outside the contract stay memory
// safe). Returns true where they differ from the host's copy the tile was planned with.
__device__ __forceinline__ bool tile_check_device(const CodecJob& j, int ntx, int t, TileCtx& c) {
  if (!j.begin_dev) return false;
  const int bd = min(max(j.begin_dev[c.b], 0), j.cap);
  const int ld = min(bd + min(max(j.count_dev[c.b], 0), j.n_rows), j.cap);
  if (bd == c.begin && ld == c.len) return false;
  c.begin = bd;
  c.len = ld;
  c.first = (bd / kW) * kW;
  c.tile0 = c.first + kTile * (t % ntx);
  return true;
}

// ------------------------------------------------------------------------------------------------
// Key role
// ------------------------------------------------------------------------------------------------
// Rows of tokens tok0 + lane into the wave's LDS row buffer (16 blocks of 64 lanes x 16 bytes),
// straight from memory without passing through registers: older rows of the open window from the
// stage, then the new rows. Lanes beyond the length load nothing.
__device__ __forceinline__ void prefetch_key_rows(const CodecJob& j, const TileCtx& c, int tok0, uint4* buf) {
  const int tok = tok0 + lane_id();
  if (tok >= c.len) return;
  const uint4* row = reinterpret_cast<const uint4*>(tok < c.begin ? j.stage + (c.seq * kW + (tok - c.first)) * kD
                                                                   : j.src + (c.seq * j.n_rows + (tok - c.begin)) * kD);
#pragma unroll
  for (int i = 0; i < 16; ++i)
    __builtin_amdgcn_global_load_lds(row + i, (__attribute__((address_space(3))) void*)(buf + 64 * i), 16, 0, 0);
}

// The lane's row from the buffer once every load of the wave has landed; zeros beyond the length.
__device__ __forceinline__ void read_key_rows(const TileCtx& c, int tok0, const uint4* buf, uint32_t (&raw)[64]) {
  __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");
  const int lane = lane_id();
  const bool valid = tok0 + lane < c.len;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const uint4 v = buf[64 * i + lane];
    raw[4 * i + 0] = valid ? v.x : 0u;
    raw[4 * i + 1] = valid ? v.y : 0u;
    raw[4 * i + 2] = valid ? v.z : 0u;
    raw[4 * i + 3] = valid ? v.w : 0u;
  }
}

// The wave holding the old open window rewrites the stage with the raw rows of the new open
// window [open, len). Only this wave reads or writes the stage of (b, h) during the launch.
__device__ __forceinline__ void rewrite_stage(const CodecJob& j, const TileCtx& c, int tok0, const uint32_t (&raw)[64]) {
  const int open = (c.len / kW) * kW;
  if (open >= c.len) return;  // (the stage reads of this tile have landed: raw was read from them)
  const int lane = lane_id(), tok = tok0 + lane;
  int slot = lane & 31;
  __asm__ volatile("" : "+v"(slot));  // keeps the lane's stage-row offset from living across the tile loop
  uint16_t* dst = j.stage + (c.seq * kW + slot) * kD;
  if (open < tok0 + 64) {
    if (tok >= open && tok < c.len) {
      uint4* d4 = reinterpret_cast<uint4*>(dst);
#pragma unroll
      for (int i = 0; i < 16; ++i) d4[i] = make_uint4(raw[4 * i], raw[4 * i + 1], raw[4 * i + 2], raw[4 * i + 3]);
    }
  } else if (lane < 32 && open + slot < c.len) {
    const uint4* s4 = reinterpret_cast<const uint4*>(j.src + (c.seq * j.n_rows + (open + slot - c.begin)) * kD);
    uint4* d4 = reinterpret_cast<uint4*>(dst);
#pragma unroll
    for (int i = 0; i < 16; ++i) d4[i] = s4[i];
  }
}

template <int kMeta>
__device__ __forceinline__ void key_role(const CodecArgs& a, int kw, float* lds) {
  constexpr bool kMx = kMeta == kMetaMx;
  const CodecJob& j = a.j;
  int t = blockIdx.x;  // < ntiles: the grid is never larger
  // The transpose tile of phase B doubles as the row buffer: the next tile's rows are loaded into
  // it after phase B has read it for the last time.
  uint4* pf = reinterpret_cast<uint4*>(lds);
  static_assert(16 * 64 * 16 <= 64 * kKeyPitch * 4, "row buffer fits the transpose tile");
  TileCtx c = tile_from_hint(j, a.ntx, t);
  prefetch_key_rows(j, c, c.tile0 + 64 * kw, pf);
  for (;;) {
    if (tile_check_device(j, a.ntx, t, c)) prefetch_key_rows(j, c, c.tile0 + 64 * kw, pf);
    const int tok0 = c.tile0 + 64 * kw;
    const bool work = c.len > c.begin && tok0 < c.len;  // wave-uniform
    float x[kD];
    uint32_t n16 = 0;
    if (work) {
      uint32_t raw[64];
      read_key_rows(c, tok0, pf, raw);
      uint32_t sw[32];  // sign words, loaded where they are used (scalar registers are scarce)
      load_sign_words(a.signs, sw);
      key_unpack(raw, sw, x);
      if (j.stage && tok0 == c.first) rewrite_stage(j, c, tok0, raw);
      n16 = key_norm(x);
    }
    const int tn = t + gridDim.x;
    TileCtx cn = c;
    auto prefetch = [&]() {  // the next tile's rows, in flight during phase C and the tile change
      if (tn < a.ntiles) {
        cn = tile_from_hint(j, a.ntx, tn);
        prefetch_key_rows(j, cn, cn.tile0 + 64 * kw, pf);
      }
    };
    if (work) {
      const size_t nw = j.cap / kW;
      KeyWaveOut out{a.k_codes + c.seq * j.cap * 32,
                     kMeta == kMetaFp16 ? a.k_min + c.seq * nw * kD : nullptr,
                     kMeta == kMetaFp16 ? a.k_step + c.seq * nw * kD : nullptr,
                     kMx ? a.k_mx + c.seq * nw * kMxRecord : nullptr,
                     a.k_norm + c.seq * j.cap, a.th.t0, a.th.t1, a.th.t2};
      key_quantize_rows<kMeta>(x, n16, tok0, c.len, out, lds, prefetch);
    } else {
      prefetch();
    }
    if (tn >= a.ntiles) break;
    t = tn;
    c = cn;
  }
}

// ------------------------------------------------------------------------------------------------
// Value role
// ------------------------------------------------------------------------------------------------
struct ValueShared {
  uint4 atile[16][4][64];     // the tile's value rows as MFMA A operands: [row block][k-block][lane]
  float itab[kTile];          // fl(1 / T) of each token
  uint8_t ktab[3][64];        // per modality and token quad: 2-bit masks of the quad's coded tokens
  uint32_t rbm[4];            // per phase-1 wave: its row blocks holding each modality (4 bits at 4 m)
  uint32_t count;             // arrivals of the value waves at their synchronization points
};

// The four value waves wait for each other (LDS counter, monotonically increasing). The wait is
// bounded: after `limit` polls the wave goes on with the tables as they are (its codes may then be
// wrong, every address stays in bounds) and the wait reports false, which the caller records in
// the cache's status word.
__device__ __forceinline__ bool value_wave_sync(uint32_t* count, uint32_t target, int limit) {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");  // this wave's table writes are done
  if (lane_id() == 0) __hip_atomic_fetch_add(count, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  bool arrived = false;
  for (int i = 0; i < limit; ++i) {
    const uint32_t seen =
        __builtin_amdgcn_readfirstlane(__hip_atomic_load(count, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP));
    if (seen >= target) {
      arrived = true;
      break;
    }
    __builtin_amdgcn_s_sleep(1);
  }
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
  return arrived;
}

// A value wave that gave up waiting marks the cache's status word (a plain vector store of 1).
__device__ __forceinline__ void report_wait(const CodecArgs& a, bool arrived) {
  if (!arrived && a.status && lane_id() == 0) *reinterpret_cast<volatile int32_t*>(a.status) = 1;
}

// The wave's slice of R_m as B operands: bf[u][kk][part] for output block nb = 2 v + u, k-block kk,
// part 0 = fp16(R) and 1 = fp16(R - fp16(R)). From the prepared fragments when there are any,
// else converted here from the fp32 matrix.
__device__ __forceinline__ void load_rot_slice(const CodecArgs& a, int m, int v, uint4 (&bf)[2][4][2]) {
  const int lane = lane_id();
  if (a.rotfrag) {
    // uniform fragment base plus the lane's 16-byte offset (scalar base, one offset register)
    const char* base = reinterpret_cast<const char*>(a.rotfrag) + (size_t)(m * 8 + 2 * v) * 8 * 1024;
    uint32_t off = 16u * (uint32_t)lane;
    __asm__ volatile("" : "+v"(off));  // computed here, not hoisted as 16 addresses held across the loop
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int kk = 0; kk < 4; ++kk)
#pragma unroll
        for (int part = 0; part < 2; ++part)
          bf[u][kk][part] = *reinterpret_cast<const uint4*>(base + ((u * 4 + kk) * 2 + part) * 1024 + off);
    return;
  }
  const int r = lane & 15, g = lane >> 4;
#pragma unroll
  for (int u = 0; u < 2; ++u)
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const float4* p = reinterpret_cast<const float4*>(a.rot + ((size_t)(m * kD + 16 * (2 * v + u) + r)) * kD + 32 * kk + 8 * g);
      const float4 f0 = p[0], f1 = p[1];
      const float fv[8] = {f0.x, f0.y, f0.z, f0.w, f1.x, f1.y, f1.z, f1.w};
      half8 hv, lv;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        hv[e] = (_Float16)fv[e];
        lv[e] = (_Float16)(fv[e] - (float)hv[e]);
      }
      bf[u][kk][0] = __builtin_bit_cast(uint4, hv);
      bf[u][kk][1] = __builtin_bit_cast(uint4, lv);
    }
}

// floor(x) as an integer in one instruction (v_cvt_flr_i32_f32)
__device__ __forceinline__ int floor_i32(float x) {
  int r;
  __asm__("v_cvt_flr_i32_f32 %0, %1" : "=v"(r) : "v"(x));
  return r;
}

// Two code bytes (output blocks 2v, 2v+1) of the lane's four tokens: code = clamp(floor(y / T) + 2,
// 0, 3) with y / T taken as y fl(1 / T), whose sign is exactly that of y.
__device__ __forceinline__ uint32_t value_bytes(floatx4 y0, floatx4 y1, float4 it) {
  const float iv[4] = {it.x, it.y, it.z, it.w};
  uint32_t s0 = 0, s1 = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int f0 = min(max(floor_i32(y0[i] * iv[i]), -2), 1);
    const int f1 = min(max(floor_i32(y1[i] * iv[i]), -2), 1);
    s0 += (uint32_t)f0 << (2 * i);
    s1 += (uint32_t)f1 << (2 * i);
  }
  return ((s0 + 0xAAu) & 0xFFu) | (((s1 + 0xAAu) & 0xFFu) << 8);  // + 2 per token
}

// The value-code bytes of a finished tile: two bytes per lane and row block, for the windows that
// hold a token below the length.
__device__ __forceinline__ void store_value_codes(const CodecArgs& a, const TileCtx& c, int v, const uint32_t (&vb)[8]) {
  const int lane = lane_id(), g = lane >> 4;
  const int ncw = a.j.cap / kW;
#pragma unroll
  for (int ww = 0; ww < 8; ++ww) {
    const int ws = c.tile0 + 32 * ww;
    if (ws >= c.len) break;
    uint16_t* dst = reinterpret_cast<uint16_t*>(a.v_codes + (c.seq * ncw + ws / kW) * 1024 + 16 * lane + 2 * v);
    uint32_t w0 = vb[ww] & 0xffffu, w1 = vb[ww] >> 16;
    if (ws < c.begin) {  // the window holds older tokens: keep their code bits
      const int old0 = min(max(c.begin - (ws + 4 * g), 0), 4);       // tokens 4g .. 4g+3
      const int old1 = min(max(c.begin - (ws + 16 + 4 * g), 0), 4);  // tokens 16+4g ..
      const uint32_t k0 = ((1u << (2 * old0)) - 1u) * 0x0101u;
      const uint32_t k1 = ((1u << (2 * old1)) - 1u) * 0x0101u;
      w0 = ((uint32_t)dst[0] & k0) | (w0 & ~k0);
      w1 = ((uint32_t)dst[4] & k1) | (w1 & ~k1);
    }
    dst[0] = (uint16_t)w0;
    dst[4] = (uint16_t)w1;
  }
}

__device__ __forceinline__ void value_role(const CodecArgs& a, int v, ValueShared& sh) {
  const CodecJob& j = a.j;
  const int lane = lane_id(), r = lane & 15, g = lane >> 4;
  uint32_t syncs = 0;
  TileCtx pend{};
  uint32_t pvb[8];
  bool has_pend = false;
  for (int t = blockIdx.x; t < a.ntiles; t += gridDim.x) {
    TileCtx c = tile_from_hint(j, a.ntx, t);
    tile_check_device(j, a.ntx, t, c);
    if (c.len <= c.begin || c.tile0 >= c.len) continue;  // uniform over the work-group
    const int wend = ((c.len + kW - 1) / kW) * kW;  // end of the last window

    // ---- phase 1: tokens [64 v, 64 v + 64) of the tile. Their rows go straight to the A tile
    // (lane l of block (rb, kk) holds channels 32 kk + 8 (l / 16) .. + 7 of row 16 rb + l % 16);
    // rows outside [begin, len) are not loaded and read as zero here, their codes are masked ----
    const int wtok0 = c.tile0 + 64 * v;
#pragma unroll
    for (int rb = 0; rb < 4; ++rb) {
      const int tok = wtok0 + 16 * rb + r;
      if (tok >= c.begin && tok < c.len) {
        const uint4* p = reinterpret_cast<const uint4*>(a.vsrc + (c.seq * j.n_rows + (tok - c.begin)) * kD);
#pragma unroll
        for (int kk = 0; kk < 4; ++kk)
          __builtin_amdgcn_global_load_lds(p + 4 * kk + g,
                                           (__attribute__((address_space(3))) void*)&sh.atile[4 * v + rb][kk][0], 16, 0, 0);
      }
    }
    if (has_pend) {  // the previous tile's codes, once this tile's row loads are out
      store_value_codes(a, pend, v, pvb);
      has_pend = false;
    }
    const int mytok = wtok0 + lane;
    const bool myfresh = mytok >= c.begin && mytok < c.len;
    const int mymod = myfresh ? (int)j.msrc[(size_t)c.b * j.n_rows + min(max(mytok - c.begin, 0), j.n_rows - 1)] : 3;
    uint4 bf[2][4][2];
    // the first modality's slice (video; R_0 with the global rotation), in flight during phase 1
    const int m_first = j.global_rot ? 0 : 1;
    if (a.rotfrag) load_rot_slice(a, m_first, v, bf);
    __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");
    uint4 av[4][4];
#pragma unroll
    for (int rb = 0; rb < 4; ++rb) {
      const int tok = wtok0 + 16 * rb + r;
      const bool fresh = tok >= c.begin && tok < c.len;
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) av[rb][kk] = fresh ? sh.atile[4 * v + rb][kk][lane] : make_uint4(0, 0, 0, 0);
    }

    // norms by the halving tree: levels 64 and 32 stay in the lane (k-blocks kk, kk + 2 and
    // 0, 1); level 16 pairs lane groups g, g ^ 2 and level 8 pairs g, g ^ 1, each exchange
    // halving the row blocks a lane keeps, so that lane l ends with token 16 g + r = l
    float p[4][8];
#pragma unroll
    for (int rb = 0; rb < 4; ++rb) {
      const half8 x0 = as_half8(av[rb][0]), x1 = as_half8(av[rb][1]), x2 = as_half8(av[rb][2]),
                  x3 = as_half8(av[rb][3]);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float f0 = (float)x0[e], f1 = (float)x1[e], f2 = (float)x2[e], f3 = (float)x3[e];
        const float l0 = __builtin_fmaf(f0, f0, f2 * f2);  // squares of fp16 values are exact
        const float l1 = __builtin_fmaf(f1, f1, f3 * f3);
        p[rb][e] = l0 + l1;
      }
    }
    const bool upper = g >= 2;
    float q[2][8];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float keep = upper ? p[2 + i][e] : p[i][e];
        const float send = upper ? p[i][e] : p[2 + i][e];
        q[i][e] = keep + __shfl_xor(send, 32);
      }
    const bool odd = (g & 1) != 0;
    float s[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float keep = odd ? q[1][e] : q[0][e];
      const float send = odd ? q[0][e] : q[1][e];
      s[e] = keep + __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, send), 0x401f));
    }
#pragma unroll
    for (int n = 4; n >= 1; n >>= 1) {
#pragma unroll
      for (int e = 0; e < n; ++e) s[e] = s[e] + s[e + n];
    }
    const uint32_t n16 = myfresh ? norm_to_f16(sqrt_rn(s[0])) : 0u;
    // 3: no code; with the global rotation every coded token takes R_0
    const int mt = (n16 != 0 && (uint32_t)mymod <= 2u) ? (j.global_rot ? 0 : mymod) : 3;
    sh.itab[64 * v + lane] = (n16 != 0) ? __builtin_amdgcn_rcpf(h2f(n16) * a.th.t2) : 0.0f;
    if (mytok >= c.begin && mytok < wend) a.v_norm[c.seq * j.cap + mytok] = (uint16_t)n16;
    if (myfresh && a.mod_out && c.h == 0) a.mod_out[(size_t)c.b * j.cap + mytok] = (uint8_t)mymod;
    uint32_t rbw = 0;
#pragma unroll
    for (int m = 0; m < 3; ++m) {
      const uint64_t mb = __ballot(mt == m);
#pragma unroll
      for (int rb = 0; rb < 4; ++rb)
        if ((mb >> (16 * rb)) & 0xffffu) rbw |= 1u << (4 * m + rb);
      if (lane < 16) {  // quad `lane`: tokens 4 lane .. 4 lane + 3 -> bits 2i, 2i + 1
        const uint32_t b4 = (uint32_t)(mb >> (4 * lane)) & 15u;
        const uint32_t spread = (b4 & 1u) | ((b4 & 2u) << 1) | ((b4 & 4u) << 2) | ((b4 & 8u) << 3);
        sh.ktab[m][16 * v + lane] = (uint8_t)(spread * 3u);
      }
    }
    if (lane == 0) sh.rbm[v] = rbw;
    report_wait(a, value_wave_sync(&sh.count, 4 * ++syncs, a.spin_limit));

    // ---- phase 2: output channels [32 v, 32 v + 32) of all 256 tokens ----
    uint32_t rbmask[3];
    {
      const uint4 w4 = *reinterpret_cast<const uint4*>(&sh.rbm[0]);
      const uint32_t ws[4] = {w4.x, w4.y, w4.z, w4.w};
#pragma unroll
      for (int m = 0; m < 3; ++m) {
        rbmask[m] = 0;
#pragma unroll
        for (int u = 0; u < 4; ++u) rbmask[m] |= ((ws[u] >> (4 * m)) & 15u) << (4 * u);
        rbmask[m] = __builtin_amdgcn_readfirstlane(rbmask[m]);
      }
    }
    uint32_t vb[8];  // window ww: bits 0-15 row block 2 ww, bits 16-31 row block 2 ww + 1
#pragma unroll
    for (int ww = 0; ww < 8; ++ww) vb[ww] = 0;
    for (int mi = 0; mi < 3; ++mi) {
      const int m = (mi == 0) ? m_first : (mi == 1 ? 1 - m_first : 2);  // video, audio, text (R_0 first if global)
      const uint32_t rbs = rbmask[m];
      if (rbs == 0) continue;
      if (mi > 0 || !a.rotfrag) load_rot_slice(a, m, v, bf);
      // one window (row blocks 2 ww, 2 ww + 1): 32 MFMAs in four independent chains (two row blocks x
      // two output blocks, each over four k-blocks x hi, lo), then the codes; a row block without
      // the modality has an all-zero keep mask
      auto window = [&](int ww) {
        floatx4 y[2][2];
#pragma unroll
        for (int h = 0; h < 2; ++h) y[h][0] = y[h][1] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
          const half8 x0 = as_half8(sh.atile[2 * ww][kk][lane]);
          const half8 x1 = as_half8(sh.atile[2 * ww + 1][kk][lane]);
#pragma unroll
          for (int part = 0; part < 2; ++part) {
            y[0][0] = __builtin_amdgcn_mfma_f32_16x16x32_f16(x0, as_half8(bf[0][kk][part]), y[0][0], 0, 0, 0);
            y[0][1] = __builtin_amdgcn_mfma_f32_16x16x32_f16(x0, as_half8(bf[1][kk][part]), y[0][1], 0, 0, 0);
            y[1][0] = __builtin_amdgcn_mfma_f32_16x16x32_f16(x1, as_half8(bf[0][kk][part]), y[1][0], 0, 0, 0);
            y[1][1] = __builtin_amdgcn_mfma_f32_16x16x32_f16(x1, as_half8(bf[1][kk][part]), y[1][1], 0, 0, 0);
          }
        }
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int rb = 2 * ww + h;
          const float4 it = *reinterpret_cast<const float4*>(&sh.itab[16 * rb + 4 * g]);
          const uint32_t keep = (uint32_t)sh.ktab[m][4 * rb + g] * 0x0101u;
          vb[ww] |= (value_bytes(y[h][0], y[h][1], it) & keep) << (16 * h);
        }
      };
#pragma unroll
      for (int ww = 0; ww < 8; ++ww)
        if ((rbs >> (2 * ww)) & 3u) window(ww);
    }
    report_wait(a, value_wave_sync(&sh.count, 4 * ++syncs, a.spin_limit));  // tables read: the next tile may refill them

    pend = c;  // stored once the next tile's row loads are out
#pragma unroll
    for (int ww = 0; ww < 8; ++ww) pvb[ww] = vb[ww];
    has_pend = true;
  }
  if (has_pend) store_value_codes(a, pend, v, pvb);
}

// ------------------------------------------------------------------------------------------------
template <bool kKeys, bool kValues, int kMeta>
__global__ __launch_bounds__(256 * (kKeys + kValues), (kKeys && kValues) ? 1 : 2) void k_codec(CodecArgs a) {
  __shared__ __attribute__((aligned(16))) float key_lds[kKeys ? 4 * kKeyWaveLds : 4];
  __shared__ __attribute__((aligned(16))) ValueShared vsh;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform for the compiler
  if (kValues) {
    if (threadIdx.x == 0) vsh.count = 0;
    __syncthreads();  // the only work-group barrier; every wave reaches it
  }
  if (kKeys && wave < 4) {
    key_role<kMeta>(a, wave, key_lds + wave * kKeyWaveLds);
  } else if (kValues) {
    value_role(a, wave - (kKeys ? 4 : 0), vsh);
  }
  if (a.ticket) {
    // Append: the lengths advance once every work-group has read them. Each work-group counts
    // itself after all its waves are done; the last one writes the new lengths and clears the
    // counter for the next launch.
    __shared__ uint32_t last;
    __syncthreads();
    if (threadIdx.x == 0)
      last = (__hip_atomic_fetch_add(a.ticket, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == gridDim.x - 1) ? 1u : 0u;
    __syncthreads();
    if (last) {
      const int nb = a.ntiles / (a.ntx * a.j.H);
      for (int i = threadIdx.x; i < nb; i += blockDim.x) a.seq_lens_out[a.j.b0 + i] += a.j.count_dev[a.j.b0 + i];
      if (threadIdx.x == 0) __hip_atomic_store(a.ticket, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

// Forward rotation fragments: fragment f = ((m 8 + nb) 4 + kk) 2 + part, lane l, element e is
// part(R_m[16 nb + l % 16][32 kk + 8 (l / 16) + e]), part 0 = fp16(R) (RNE), 1 = fp16 of the residual.
__global__ __launch_bounds__(256) void k_prepare_fragments(const float* __restrict__ rot, uint4* __restrict__ frag) {
  const int idx = blockIdx.x * 256 + threadIdx.x;  // (fragment pair, lane)
  if (idx >= kRotFragments / 2 * 64) return;
  const int lane = idx & 63, fp = idx >> 6;  // fp = (m 8 + nb) 4 + kk
  const int kk = fp & 3, nb = (fp >> 2) & 7, m = fp >> 5;
  const float* src = rot + ((size_t)(m * kD + 16 * nb + (lane & 15))) * kD + 32 * kk + 8 * (lane >> 4);
  half8 hv, lv;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const float f = src[e];
    hv[e] = (_Float16)f;
    lv[e] = (_Float16)(f - (float)hv[e]);
  }
  frag[(2 * fp) * 64 + lane] = __builtin_bit_cast(uint4, hv);
  frag[(2 * fp + 1) * 64 + lane] = __builtin_bit_cast(uint4, lv);
}

hipError_t launch_prepare_fragments(const float* rot, uint4* frag, hipStream_t s) {
  hipLaunchKernelGGL(k_prepare_fragments, dim3(kRotFragments / 2 * 64 / 256), dim3(256), 0, s, rot, frag);
  return hipGetLastError();
}

// one launch, bound to the two events when given
template <typename Kernel>
void launch_one(Kernel fn, int grid, int block, hipStream_t s, hipEvent_t const* events, const CodecArgs& a) {
  if (events)
    hipExtLaunchKernelGGL(fn, dim3(grid), dim3(block), 0, s, events[0], events[1], 0, a);
  else
    hipLaunchKernelGGL(fn, dim3(grid), dim3(block), 0, s, a);
}

hipError_t launch_codec(const CodecArgs& args, bool keys, bool values, hipStream_t s, hipEvent_t const* events) {
  if (args.ntiles <= 0 || (!keys && !values)) return hipSuccess;
  CodecArgs a = args;
  a.spin_limit = kSpinLimit;
  // test hook: a smaller bound for the value waves' wait (0 makes every wait give up at once)
  if (const char* env = getenv("OKVQ_CODEC_SPIN_LIMIT")) a.spin_limit = std::max(0, atoi(env));
  int dev = 0, cus = 256;
  if (hipGetDevice(&dev) == hipSuccess) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && n > 0) cus = n;
  }
  // resident work-groups: both roles fill a compute unit (8 waves at up to 256 VGPRs); one role
  // leaves room for two
  const int per_cu = (keys && values) ? 1 : 2;
  const int grid = std::min(a.ntiles, per_cu * cus);
  if (keys && values) {
    if (a.key_meta == kMetaMx)
      launch_one(k_codec<true, true, kMetaMx>, grid, 512, s, events, a);
    else if (a.key_meta == kMetaTq)
      launch_one(k_codec<true, true, kMetaTq>, grid, 512, s, events, a);
    else
      launch_one(k_codec<true, true, kMetaFp16>, grid, 512, s, events, a);
  } else if (keys) {
    if (a.key_meta == kMetaMx)
      launch_one(k_codec<true, false, kMetaMx>, grid, 256, s, events, a);
    else if (a.key_meta == kMetaTq)
      launch_one(k_codec<true, false, kMetaTq>, grid, 256, s, events, a);
    else
      launch_one(k_codec<true, false, kMetaFp16>, grid, 256, s, events, a);
  } else {
    launch_one(k_codec<false, true, kMetaFp16>, grid, 256, s, events, a);
  }
  return hipGetLastError();
}

}  // namespace okvq
