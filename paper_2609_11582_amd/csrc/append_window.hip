// Window-parallel append: the key and value codecs of one append, the fp16 residual rings and the
// length update in a single launch, for appends that touch few key windows per (sequence, KV head)
// -- a generation step, a streamed chunk (Sec. 2.1 Eq. 2 and Sec. 2.3 Eq. 4 for keys; Sec. 2.3
// Eq. 6 with the codebook of Eq. 3 for values; the residual rings of the captioning protocol, Sec.
// 3.1). The results are the bytes of the tile codec (codec_fused.hip): the same operations in the
// same order, spread over more lanes so that the chain from the rows to the codes is short.
//
// Work unit: one 32-token key window of one (sequence, KV head), from the open window
// 32 floor(L / 32) to the new end, and one of its two roles: a key work-group and a value work-group
// of 512 threads each. Thread (t, j) = (tid / 16, tid % 16) holds channels 8j .. 8j + 7 of window
// token t (a wave without a token of its own skips the arithmetic):
//  * key: sign flip, fp16 norm by the halving tree (levels 64 .. 8 across the 16 lanes of the
//    token, 4 .. 1 in the lane), butterflies h = 1, 2, 4 in the lane and h = 8 .. 64 across lanes,
//    z = w fl(kappa / n16); window minimum and maximum per channel by LDS atomics; codes and their
//    packing in the lane, one key-code dword per lane pair;
//  * value: fp16 norm by the same tree; the row goes to an LDS tile of MFMA A operands; wave w then
//    forms output channels 16w .. 16w + 15 of the window's 32 tokens on the matrix cores (R_m as
//    fp16 hi + lo B operands, fp32 accumulation, in the tile codec's order), one modality at a time,
//    and writes their code bytes.
// Older tokens of the open window come from the key stage; their key codes are rewritten with the
// window's new minimum and step, their value codes are kept. The work-group of the first window, the
// only one that reads the stage, rewrites it with the raw rows of the new open window after a
// barrier that follows its reads. The last work-group to finish advances the lengths.
#include <hip/hip_ext.h>

#include "lane_quant.hpp"
#include "launch.hpp"

namespace okvq {
namespace {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 512;
static_assert(kMaxLenArgs <= kThreads, "one thread per sequence of the launch for the length update");

// c ? u : v, component by component (a select of whole vectors becomes one of their addresses)
__device__ __forceinline__ uint4 select4(bool c, uint4 u, uint4 v) {
  return make_uint4(c ? u.x : v.x, c ? u.y : v.y, c ? u.z : v.z, c ? u.w : v.w);
}

// floor(x) as an integer in one instruction (v_cvt_flr_i32_f32)
__device__ __forceinline__ int floor_to_int(float x) {
  int r;
  __asm__("v_cvt_flr_i32_f32 %0, %1" : "=v"(r) : "v"(x));
  return r;
}

// The launch's arguments: the append fields of the codec arguments without the host's copies of
// the lengths (the kernel reads the device lengths), about 200 bytes instead of 2.4 KB.
struct WindowArgs {
  const uint16_t* src;       // key rows [B][H][n_rows][128] fp16
  const uint16_t* vsrc;      // value rows, the same layout
  const uint8_t* msrc;       // [B][n_rows] modality ids
  const int32_t* begin_dev;  // current lengths (device)
  const int32_t* count_dev;  // appended tokens (device)
  uint16_t* stage;           // [B][H][32][128] raw keys of the open window
  const int8_t* signs;
  uint8_t* k_codes;
  uint16_t* k_min;
  uint16_t* k_step;
  uint16_t* k_norm;
  const uint4* rotfrag;      // prepared forward fragments of R_m
  uint8_t* v_codes;
  uint16_t* v_norm;
  uint8_t* mod_out;
  int32_t* seq_lens_out;
  uint32_t* ticket;
  uint16_t* k_res;           // residual rings, or null
  uint16_t* v_res;
  Thresholds th;
  int n_rows, b0, H, cap, global_rot;
};

constexpr int kStatSlots = kD + kD / 8;

struct WindowShared {
  uint4 atile[2][4][64];   // the window's value rows as MFMA A operands: [row block][k-block][lane]
  float kmin[kStatSlots];  // per channel c (slot c + c / 8, spread over the banks): the window
  float kmax[kStatSlots];  // minimum and maximum, taken by LDS atomics
  float2 kstat[kD];        // per channel: (fp16 minimum, fl(1 / fp16 step)) as fp32
  float itab[kW];          // per token: fl(1 / T) of the value decision (0: no code)
  uint32_t tmod[kW];       // per token: the rotation of its value code (3: none)
  uint32_t last;
};

// The row loads of a work-group are not predicated per lane: a lane without a row of its own reads
// the nearest row of its sequence (clamped index, so that lanes spread over distinct rows rather than
// all meeting on one cache line) and drops what it read; no branch separates the loads from each
// other. The stage is read only by the first window's key work-group, and only when it holds older
// tokens.

// Key work-group, thread (t, j), window wi of a sequence whose new tokens are [begin, len): the key
// chunk of window token t (from the stage below begin), and for the first window, if the new open
// window starts after it, the key chunk of token open + t (sraw).
__device__ __forceinline__ void key_inputs(const WindowArgs& a, size_t seq, int begin, int len, int wi, int t, int j,
                                           uint4& kraw, uint4& sraw) {
  const WindowArgs& J = a;
  const int first = (begin / kW) * kW, w0 = first + kW * wi, tok = w0 + t, last = J.n_rows - 1;
  const size_t srow = seq * J.n_rows;
  const uint4 zero = make_uint4(0u, 0u, 0u, 0u);
  const int open = (len / kW) * kW, stok = open + t;
  const bool staged = wi == 0 && begin > first;  // uniform: older tokens of the open window, from the stage
  // every load goes out before the selects (a select right behind its load waits for it and holds
  // back the loads after it)
  const uint4 kn = reinterpret_cast<const uint4*>(J.src + (srow + (size_t)min(max(tok - begin, 0), last)) * kD)[j];
  uint4 ks = zero;
  sraw = zero;
  if (staged) ks = reinterpret_cast<const uint4*>(J.stage + (seq * kW + min(t, begin - first - 1)) * kD)[j];
  if (wi == 0 && open != first && open < len)  // uniform
    sraw = reinterpret_cast<const uint4*>(J.src + (srow + (size_t)min(max(stok - begin, 0), last)) * kD)[j];
  kraw = select4(tok >= begin && tok < len, kn, zero);
  if (staged) kraw = select4(tok < begin, ks, kraw);
}

// Value work-group, thread (t, j): the value chunk of window token t (new tokens only), its
// modality id (3: not a new token), and in lanes 0..31 of every wave the modality id of window token
// `lane` (wmod), for the window's modality set.
__device__ __forceinline__ void value_inputs(const WindowArgs& a, size_t seq, int b, int begin, int len, int wi,
                                             int t, int j, int lane, uint4& vraw, uint32_t& mod, uint32_t& wmod) {
  const WindowArgs& J = a;
  const int first = (begin / kW) * kW, w0 = first + kW * wi, tok = w0 + t, wtok = w0 + (lane & 31);
  const int last = J.n_rows - 1;
  const size_t mrow = (size_t)b * J.n_rows, srow = seq * J.n_rows;
  const bool fresh = tok >= begin && tok < len, wfresh = wtok >= begin && wtok < len;
  const int r = min(max(tok - begin, 0), last);
  const uint4 vn = reinterpret_cast<const uint4*>(a.vsrc + (srow + (size_t)r) * kD)[j];
  const uint32_t tm = J.msrc[mrow + r];
  const uint32_t wm = J.msrc[mrow + min(max(wtok - begin, 0), last)];
  vraw = select4(fresh, vn, make_uint4(0u, 0u, 0u, 0u));
  mod = fresh ? tm : 3u;
  wmod = wfresh ? wm : 3u;
}

// The key work-group of a window: directions, window statistics, codes, norms, the stage and the
// key ring of the residual.
template <int kMeta>
__device__ __forceinline__ void key_window(const WindowArgs& a, WindowShared& sh, size_t seq, int begin, int len,
                                           int wi, int tid) {
  const WindowArgs& J = a;
  const int t = tid >> 4, j = tid & 15;
  const int first = (begin / kW) * kW, w0 = first + kW * wi, tok = w0 + t;
  const bool valid = tok < len, fresh = valid && tok >= begin;
  const uint2 sg = *reinterpret_cast<const uint2*>(a.signs + 8 * j);
  uint4 kraw, sraw;
  key_inputs(a, seq, begin, len, wi, t, j, kraw, sraw);
  const int open = (len / kW) * kW, stok = open + t;
  const bool restage = J.stage && wi == 0 && open < len;
  // ---- direction (thread = token chunk); a wave without a valid token skips the arithmetic ----
  const bool busy = __ballot(valid) != 0;  // wave-uniform
  float x[8];
  uint32_t kn16 = 0;
#pragma unroll
  for (int e = 0; e < 8; ++e) x[e] = 0.0f;
  if (busy) kn16 = lane_direction(kraw, sg, j, x);
  if (a.k_res && fresh && tok >= len - kResidual)  // the residual ring: raw rows of the last 128 tokens
    reinterpret_cast<uint4*>(a.k_res + (seq * kResidual + (tok & (kResidual - 1))) * kD)[j] = kraw;
  // ---- window minimum / maximum per channel: LDS atomics of the valid tokens ----
  if constexpr (kMeta == kMetaFp16) {
    if (valid) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        __hip_atomic_fetch_min(&sh.kmin[9 * j + e], x[e], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        __hip_atomic_fetch_max(&sh.kmax[9 * j + e], x[e], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
      }
    }
  }
  if (restage) __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");  // this thread's stage reads have landed
  __syncthreads();  // B1: window extremes written; every stage read has landed
  if (restage && stok >= begin && stok < len)  // the new open window's raw keys
    reinterpret_cast<uint4*>(J.stage + (seq * kW + t) * kD)[j] = select4(open == first, kraw, sraw);
  const size_t nw = J.cap / kW;
  const int gwin = w0 / kW;
  if constexpr (kMeta == kMetaFp16) {
    if (tid < kD) {
      const float l = sh.kmin[tid + (tid >> 3)] + 0.0f;  // canonical +0
      const float u = sh.kmax[tid + (tid >> 3)] + 0.0f;
      const float step = div_rn(u - l, 3.0f);
      const uint32_t m16 = f2h(l), s16 = f2h(step);
      a.k_min[(seq * nw + gwin) * kD + tid] = (uint16_t)m16;
      a.k_step[(seq * nw + gwin) * kD + tid] = (uint16_t)s16;
      sh.kstat[tid] = make_float2(h2f(m16), (s16 == 0) ? 0.0f : div_rn(1.0f, h2f(s16)));
    }
    __syncthreads();  // B2: window statistics
  }
  // ---- codes: 2 bits per channel; word u of a token holds channels 16u .. 16u + 15, the even ones
  // in its low half; this lane fills bits 8 (j & 1) .. + 7 of both halves of word j / 2 ----
  uint32_t lo16 = 0, hi16 = 0;
  if (valid) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int sh2 = 2 * (4 * (j & 1) + i);
      uint32_t c0, c1;
      if constexpr (kMeta == kMetaFp16) {
        const float4 st = *reinterpret_cast<const float4*>(&sh.kstat[8 * j + 2 * i]);
        constexpr float kRound = 8388608.0f;  // 2^23: rint of the clamped value in the low bits
        const float t0 = (x[2 * i] - st.x) * st.y;
        const float t1 = (x[2 * i + 1] - st.z) * st.w;
        c0 = __builtin_bit_cast(uint32_t, __builtin_amdgcn_fmed3f(t0, 0.0f, 3.0f) + kRound) & 3u;
        c1 = __builtin_bit_cast(uint32_t, __builtin_amdgcn_fmed3f(t1, 0.0f, 3.0f) + kRound) & 3u;
      } else {
        const float z0 = x[2 * i], z1 = x[2 * i + 1];
        c0 = (uint32_t)(z0 > a.th.t0) + (uint32_t)(z0 > a.th.t1) + (uint32_t)(z0 > a.th.t2);
        c1 = (uint32_t)(z1 > a.th.t0) + (uint32_t)(z1 > a.th.t1) + (uint32_t)(z1 > a.th.t2);
      }
      lo16 |= c0 << sh2;
      hi16 |= c1 << sh2;
    }
  }
  uint32_t word = lo16 | (hi16 << 16);
  word |= xchg_u(word);
  if ((j & 1) == 0) reinterpret_cast<uint32_t*>(a.k_codes + (seq * J.cap + tok) * 32)[j >> 1] = word;
  if (j == 0) a.k_norm[seq * J.cap + tok] = valid ? (uint16_t)kn16 : (uint16_t)0;
}

// The value work-group of a window: norms, the A tile, then wave w forms output channels 16w ..
// 16w + 15 of the 32 tokens on the matrix cores, per present modality, and writes their code bytes;
// also the modality map and the value ring of the residual.
__device__ __forceinline__ void value_window(const WindowArgs& a, WindowShared& sh, size_t seq, int b, int h,
                                             int begin, int len, int wi, int tid) {
  const WindowArgs& J = a;
  const int t = tid >> 4, j = tid & 15, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int first = (begin / kW) * kW, w0 = first + kW * wi, tok = w0 + t;
  const bool fresh = tok >= begin && tok < len;
  uint4 vraw;
  uint32_t mymod, wmod;
  value_inputs(a, seq, b, begin, len, wi, t, j, lane, vraw, mymod, wmod);
  // the window's modalities (a superset of those coded) and the B operands of the first of them,
  // loaded first: in flight while the norms, tables and stores below are formed, and across the barrier
  uint32_t mset = 0;
#pragma unroll
  for (int m = 0; m < 3; ++m)
    if (__ballot(wmod == (uint32_t)m)) mset |= 1u << m;
  if (J.global_rot) mset = mset ? 1u : 0u;  // R_0 for every token
  const int m_first = mset ? __builtin_ctz(mset) : 0;
  uint4 bf[4][2];
  {
    const uint4* base = a.rotfrag + (size_t)(m_first * 8 + wave) * 8 * 64 + lane;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk)
#pragma unroll
      for (int part = 0; part < 2; ++part) bf[kk][part] = base[(kk * 2 + part) * 64];
  }
  const bool busy = __ballot(fresh) != 0;  // wave-uniform
  {
    const uint32_t r4[4] = {vraw.x, vraw.y, vraw.z, vraw.w};
    float v[8];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[2 * i] = h2f(r4[i] & 0xffffu);
      v[2 * i + 1] = h2f(r4[i] >> 16);
    }
    const uint32_t vn16 = busy ? group_norm(v) : 0u;  // 0 for the zero rows of older and padded tokens
    sh.atile[t >> 4][j >> 2][16 * (j & 3) + (t & 15)] = vraw;
    if (j == 0) {
      const uint32_t mt = (vn16 != 0 && mymod <= 2u) ? (J.global_rot ? 0u : mymod) : 3u;
      sh.itab[t] = (vn16 != 0) ? __builtin_amdgcn_rcpf(h2f(vn16) * a.th.t2) : 0.0f;
      sh.tmod[t] = mt;
      if (tok >= begin) a.v_norm[seq * J.cap + tok] = (uint16_t)vn16;  // 0 in the padded slots
      if (fresh && a.mod_out && h == 0) a.mod_out[(size_t)b * J.cap + tok] = (uint8_t)mymod;
    }
  }
  if (a.v_res && fresh && tok >= len - kResidual)  // the residual ring: raw rows of the last 128 tokens
    reinterpret_cast<uint4*>(a.v_res + (seq * kResidual + (tok & (kResidual - 1))) * kD)[j] = vraw;
  __syncthreads();  // B1: A tile and token tables written
  const int g = lane >> 4;
  const uint32_t tm = sh.tmod[lane & 31];
  uint32_t vb[2] = {0u, 0u};
#pragma unroll 1
  for (int m = m_first; m < 3; ++m) {
    const uint32_t mb = (uint32_t)__ballot(tm == (uint32_t)m);  // token bits, lanes 0..31
    if (mb == 0) continue;
    if (m != m_first) {
      const uint4* base = a.rotfrag + (size_t)(m * 8 + wave) * 8 * 64 + lane;
#pragma unroll
      for (int kk = 0; kk < 4; ++kk)
#pragma unroll
        for (int part = 0; part < 2; ++part) bf[kk][part] = base[(kk * 2 + part) * 64];
    }
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
      floatx4 y = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        const half8 xa = __builtin_bit_cast(half8, sh.atile[rb][kk][lane]);
#pragma unroll
        for (int part = 0; part < 2; ++part)
          y = __builtin_amdgcn_mfma_f32_16x16x32_f16(xa, __builtin_bit_cast(half8, bf[kk][part]), y, 0, 0, 0);
      }
      const float4 it = *reinterpret_cast<const float4*>(&sh.itab[16 * rb + 4 * g]);
      const float iv[4] = {it.x, it.y, it.z, it.w};
      uint32_t byte = 0;
#pragma unroll
      for (int i = 0; i < 4; ++i) byte |= (uint32_t)(min(max(floor_to_int(y[i] * iv[i]), -2), 1) + 2) << (2 * i);
      const uint32_t b4 = (mb >> (16 * rb + 4 * g)) & 15u;  // the quad's tokens of modality m
      const uint32_t keep = ((b4 & 1u) | ((b4 & 2u) << 1) | ((b4 & 4u) << 2) | ((b4 & 8u) << 3)) * 3u;
      vb[rb] |= byte & keep;
    }
  }
  const size_t nw = J.cap / kW;
  uint8_t* blk = a.v_codes + (seq * nw + w0 / kW) * 1024 + 16 * lane + wave;
#pragma unroll
  for (int rb = 0; rb < 2; ++rb) {
    uint32_t v = vb[rb];
    const int old = min(max(begin - (w0 + 16 * rb + 4 * g), 0), 4);  // older tokens of the quad keep their bits
    if (old > 0) {
      const uint32_t k = (1u << (2 * old)) - 1u;
      v = ((uint32_t)blk[8 * rb] & k) | (v & ~k);
    }
    blk[8 * rb] = (uint8_t)v;
  }
}

// Grid: (2 nwin, H, sequences); x < nwin: the key work-group of window x, else the value work-group
// of window x - nwin.
template <int kMeta>
__global__ __launch_bounds__(kThreads) void k_append_window(WindowArgs a) {
  static_assert(kMeta == kMetaFp16 || kMeta == kMetaTq, "fp16 window metadata or TurboQuant keys");
  __shared__ WindowShared sh;
  const WindowArgs& J = a;
  const int tid = threadIdx.x;
  const int nwin = (int)gridDim.x / 2;
  const bool values = (int)blockIdx.x >= nwin;  // uniform
  const int wi = (int)blockIdx.x - (values ? nwin : 0), h = blockIdx.y, bz = blockIdx.z, b = J.b0 + bz;
  const size_t seq = (size_t)b * J.H + h;
  // the device lengths decide, clamped into the buffers (the host's copy planned the grid)
  const int begin = min(max(J.begin_dev[b], 0), J.cap);
  const int len = min(begin + min(max(J.count_dev[b], 0), J.n_rows), J.cap);
  if (kMeta == kMetaFp16 && !values) {
    if (tid < kStatSlots) {
      sh.kmin[tid] = __builtin_inff();
      sh.kmax[tid] = -__builtin_inff();
    }
    __syncthreads();  // B0 (the waves of a work-group start together)
  }
  const int w0 = (begin / kW) * kW + kW * wi;  // the work-group's window
  if (len > begin && w0 < len) {               // uniform
    if (values)
      value_window(a, sh, seq, b, h, begin, len, wi, tid);
    else
      key_window<kMeta>(a, sh, seq, begin, len, wi, tid);
  }

  // The lengths advance once every work-group has read them: each work-group counts itself after
  // all its threads are done; the last one writes the new lengths and clears the counter.
  __syncthreads();
  if (tid == 0) {
    const uint32_t total = gridDim.x * gridDim.y * gridDim.z;
    sh.last = (__hip_atomic_fetch_add(a.ticket, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == total - 1) ? 1u : 0u;
  }
  __syncthreads();
  if (sh.last) {
    // The counts are read only here: vector reads of the lengths' cache line at the start of every
    // work-group, while the counter's atomics hit that line, made a 4096-work-group launch 4x slower.
    const int nseq = gridDim.z;
    if (tid < nseq) a.seq_lens_out[J.b0 + tid] += J.count_dev[J.b0 + tid];
    if (tid == 0) __hip_atomic_store(a.ticket, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

}  // namespace

hipError_t launch_append_window(const CodecArgs& c, int nwin, int nb, hipStream_t s, hipEvent_t const* events) {
  if (nwin <= 0 || nb <= 0) return hipSuccess;
  WindowArgs a;
  a.src = c.j.src;
  a.vsrc = c.vsrc;
  a.msrc = c.j.msrc;
  a.begin_dev = c.j.begin_dev;
  a.count_dev = c.j.count_dev;
  a.stage = c.j.stage;
  a.signs = c.signs;
  a.k_codes = c.k_codes;
  a.k_min = c.k_min;
  a.k_step = c.k_step;
  a.k_norm = c.k_norm;
  a.rotfrag = c.rotfrag;
  a.v_codes = c.v_codes;
  a.v_norm = c.v_norm;
  a.mod_out = c.mod_out;
  a.seq_lens_out = c.seq_lens_out;
  a.ticket = c.ticket;
  a.k_res = c.k_res;
  a.v_res = c.v_res;
  a.th = c.th;
  a.n_rows = c.j.n_rows;
  a.b0 = c.j.b0;
  a.H = c.j.H;
  a.cap = c.j.cap;
  a.global_rot = c.j.global_rot;
  const int key_meta = c.key_meta;
  const dim3 grid(2 * nwin, a.H, nb);
  if (key_meta != kMetaTq && key_meta != kMetaFp16) return hipErrorInvalidValue;
  void (*fn)(WindowArgs) = key_meta == kMetaTq ? k_append_window<kMetaTq> : k_append_window<kMetaFp16>;
  if (events)
    hipExtLaunchKernelGGL(fn, grid, dim3(kThreads), 0, s, events[0], events[1], 0, a);
  else
    hipLaunchKernelGGL(fn, grid, dim3(kThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace okvq
