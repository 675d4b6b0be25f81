// Dense fp16 decode attention (Eq. 1 over an unquantized fp16 KV cache): the comparison baseline
// for the packed 2-bit cache, on the same split-K shape and the same log-sum-exp merge launch.
//
// Work-group (split, KV head h, sequence b) = 8 waves; wave w takes the split's 32-token tiles
// w, w + 8, w + 16, ... and keeps its own online-softmax state for all G <= 8 query heads of the KV
// head, so one read of K and V serves every head of the group.
//  * Scores on the matrix cores (v_mfma_f32_16x16x32_f16): rows = 16 tokens, columns = the query
//    heads, K = 128 channels in four blocks. The query is read once per work-group as fp16 B
//    operands; key rows go straight from memory into the A operands (16 bytes per lane, 64
//    contiguous bytes per row and instruction).
//  * Value rows arrive in registers (16 bytes per lane, whole 256-byte rows per 16 lanes), are
//    written to the wave's LDS tile under a 16-byte-chunk XOR swizzle, and read back as B operands
//    of the PV product with the transposing LDS read of gfx950 (ds_read_b64_tr_b16: 16 lanes
//    receive a 4 x 4 block of fp16 transposed, lane i taking column i % 4 of the rows addressed by
//    lanes 4e + i / 4). The contraction's token order is chosen to be the score tile's row order,
//    so each lane's own score registers are its A operand.
//  * Two register sets per wave: a tile's loads are in flight while the previous tile is
//    computed. (Loading the values straight into LDS with global_load_lds was tried: mixed with
//    register loads it makes the compiler wait for every outstanding load before each tile.)
//  * Base-2 softmax with a lazily updated reference (moved only when the max grows by 2^8, so
//    the fp16 probabilities stay below 2^8).
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

constexpr int kDnWaves = 8;
constexpr int kDnTile = 32;                     // tokens per wave and step
constexpr int kDnStep = kDnWaves * kDnTile;     // tokens per work-group step
constexpr int kDnTileBytes = kDnTile * kD * 2;  // one wave's value tile: 8 KiB
constexpr float kDnLazy = 8.0f;

struct DenseArgs {
  const uint16_t* k;        // [B][H][cap][128] fp16
  const uint16_t* v;        // [B][H][cap][128] fp16
  const int32_t* seq_lens;  // [B]
  const uint16_t* q;        // [B][Hq][128] fp16
  float* ws;                // split records [B][H][nsplit][kRecFloats]
  int H, Hq, G, cap, tps, nsplit;
  float qscale;             // sm_scale log2(e)
};

__device__ __forceinline__ half8 as_h8(uint4 v) { return __builtin_bit_cast(half8, v); }
__device__ __forceinline__ uint32_t pack_h2(float lo, float hi) {
  const half2v v = {(_Float16)lo, (_Float16)hi};
  return __builtin_bit_cast(uint32_t, v);
}
__device__ __forceinline__ short4v lds_tr(const uint8_t* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) short4v*)p);
}

struct TileRegs {
  uint4 k[2][4];  // A operands: key rows 16 tb + r, channels 32 kb + 8 g .. + 7
  uint4 v[8];     // value rows 4 i + g, 16-byte chunk r ^ (row % 16)
};

__global__ __launch_bounds__(64 * kDnWaves) void k_decode_dense(DenseArgs p) {
  // value tiles [wave][32 rows x 256 B]; after the loop they hold the combine tile
  __shared__ __attribute__((aligned(16))) uint8_t vbuf[kDnWaves][kDnTileBytes];
  __shared__ float wm[kDnWaves][8], wl[kDnWaves][8];
  const int split = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, g = lane >> 4, r = lane & 15;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: the tile loop branches are scalar
  const int len = min(p.seq_lens[b], p.cap);
  const int t_begin = split * p.tps, t_end = min(t_begin + p.tps, len);
  float* rec = p.ws + (((size_t)b * p.H + h) * p.nsplit + split) * kRecFloats;
  if (t_begin >= t_end) {  // an empty split: the merge skips M = -inf
    write_empty_record(rec, tid);
    return;
  }
  const size_t seq = (size_t)b * p.H + h;
  const uint16_t* kbase = p.k + seq * p.cap * kD;
  const uint16_t* vbase = p.v + seq * p.cap * kD;

  // query operands: B[channel 32 kb + 8 g + e][head r], zero for heads >= G
  uint4 qop[4];
  {
    const bool live = r < p.G;
    const uint4* qrow = reinterpret_cast<const uint4*>(p.q + ((size_t)b * p.Hq + h * p.G + (live ? r : 0)) * kD);
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) qop[kb] = live ? qrow[4 * kb + g] : make_uint4(0u, 0u, 0u, 0u);
  }
  const int ntile = (t_end - t_begin + kDnTile - 1) / kDnTile;
  const int nmine = ntile > wave ? (ntile - wave + kDnWaves - 1) / kDnWaves : 0;

  // Loads of this wave's tile `it`. LDS slot (row 4 i + g, chunk r) of the value tile will hold
  // the row's 16-byte chunk r ^ (row % 16). Rows past the split's end read its last token (finite
  // data; their weights are zero).
  auto issue = [&](int it, TileRegs& tr) {
    const int t0 = t_begin + (wave + kDnWaves * it) * kDnTile;
#pragma unroll
    for (int tb = 0; tb < 2; ++tb) {
      const uint4* krow = reinterpret_cast<const uint4*>(kbase + (size_t)min(t0 + 16 * tb + r, t_end - 1) * kD);
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) tr.k[tb][kb] = krow[4 * kb + g];
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int row = 4 * i + g;
      tr.v[i] = reinterpret_cast<const uint4*>(vbase + (size_t)min(t0 + row, t_end - 1) * kD)[r ^ (row & 15)];
    }
    __builtin_amdgcn_sched_barrier(0);  // every load of the tile is issued before the work that follows
  };

  float m_ref = -__builtin_inff();  // head r's softmax reference (base 2)
  float l_part = 0.0f;              // this lane's share of head r's sum, relative to 2^m_ref
  floatx4 acc[8];                   // o[head 4 g + i][channel 16 cb + r], relative to 2^m_ref
#pragma unroll
  for (int cb = 0; cb < 8; ++cb) acc[cb] = floatx4{0.f, 0.f, 0.f, 0.f};
  // transposed-read address of the lane: rows 4 g + r / 4 (+ 16), channels 16 cb + 4 (r % 4)
  const int trow = 4 * g + (r >> 2), tsub = r & 3;

  uint8_t* vt = &vbuf[wave][0];
  auto compute = [&](int it, const TileRegs& tr) {
    const int t0 = t_begin + (wave + kDnWaves * it) * kDnTile;
    // the value tile into LDS (the previous tile's transposed reads precede these writes)
#pragma unroll
    for (int i = 0; i < 8; ++i) *reinterpret_cast<uint4*>(vt + 1024 * i + 16 * lane) = tr.v[i];
    floatx4 s[2] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      s[0] = __builtin_amdgcn_mfma_f32_16x16x32_f16(as_h8(tr.k[0][kb]), as_h8(qop[kb]), s[0], 0, 0, 0);
      s[1] = __builtin_amdgcn_mfma_f32_16x16x32_f16(as_h8(tr.k[1][kb]), as_h8(qop[kb]), s[1], 0, 0, 0);
    }
    // s[tb][i] = score of token 16 tb + 4 g + i for head r
    float x[2][4];
    float mx = -__builtin_inff();
#pragma unroll
    for (int tb = 0; tb < 2; ++tb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int t = t0 + 16 * tb + 4 * g + i;
        x[tb][i] = (t < t_end) ? s[tb][i] * p.qscale : -__builtin_inff();
        mx = fmaxf(mx, x[tb][i]);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 16));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    if (__any(mx > m_ref + kDnLazy)) {  // rare after the first tile: move the references that grew
      const float m_new = (mx > m_ref + kDnLazy) ? mx : m_ref;
      const float alpha = __builtin_amdgcn_exp2f(m_ref - m_new);  // 0 while m_ref = -inf
      l_part *= alpha;
#pragma unroll
      for (int i = 0; i < 4; ++i) {  // accumulator rows are heads 4 g + i: factors from lanes 4 g + i
        const float ai = __shfl(alpha, 4 * g + i);
#pragma unroll
        for (int cb = 0; cb < 8; ++cb) acc[cb][i] *= ai;
      }
      m_ref = m_new;
    }
    float pv[2][4];
#pragma unroll
    for (int tb = 0; tb < 2; ++tb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        pv[tb][i] = __builtin_amdgcn_exp2f(x[tb][i] - m_ref);
        l_part += pv[tb][i];
      }
    // A operand: row = head r, k = 8 g + e <-> token 4 g + e (e < 4), 16 + 4 g + e - 4 (e >= 4)
    const half8 pa = __builtin_bit_cast(half8, make_uint4(pack_h2(pv[0][0], pv[0][1]), pack_h2(pv[0][2], pv[0][3]),
                                                          pack_h2(pv[1][0], pv[1][1]), pack_h2(pv[1][2], pv[1][3])));
    wave_lds_sync();
#pragma unroll
    for (int cb = 0; cb < 8; ++cb) {
      const int slot = ((2 * cb + (tsub >> 1)) ^ trow) * 16 + 8 * (tsub & 1);
      const short4v lo = lds_tr(vt + trow * 256 + slot);
      const short4v hi = lds_tr(vt + (16 + trow) * 256 + slot);
      const uint2 l2 = __builtin_bit_cast(uint2, lo), h2 = __builtin_bit_cast(uint2, hi);
      acc[cb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(pa, __builtin_bit_cast(half8, make_uint4(l2.x, l2.y, h2.x, h2.y)),
                                                       acc[cb], 0, 0, 0);
    }
  };

  // two register sets: tile it + 1's loads are in flight while tile it is computed
  TileRegs ta, tb;
  int it = 0;
  if (nmine > 0) issue(0, ta);
  for (; it + 2 < nmine; it += 2) {
    issue(it + 1, tb);
    compute(it, ta);
    issue(it + 2, ta);
    compute(it + 1, tb);
  }
  if (it + 1 < nmine) {
    issue(it + 1, tb);
    compute(it, ta);
    compute(it + 1, tb);
  } else if (it < nmine) {
    compute(it, ta);
  }

  // ---- combine the 8 waves: per head, M = max of the references, L and o rescaled to it ----
  float l_tot = l_part + __shfl_xor(l_part, 16);
  l_tot += __shfl_xor(l_tot, 32);
  __syncthreads();  // every wave is done with its value tiles: they become the combine tile
  float* cmb = reinterpret_cast<float*>(&vbuf[0][0]);  // [wave][8 heads][128]
  if (g < 2) {
#pragma unroll
    for (int cb = 0; cb < 8; ++cb)
#pragma unroll
      for (int i = 0; i < 4; ++i) cmb[(wave * 8 + 4 * g + i) * kD + 16 * cb + r] = acc[cb][i];
  }
  if (lane < 8) {
    wm[wave][lane] = m_ref;
    wl[wave][lane] = l_tot;
  }
  __syncthreads();
  const int hh = tid >> 6, c2 = 2 * (tid & 63);
  float M = -__builtin_inff();
#pragma unroll
  for (int w = 0; w < kDnWaves; ++w) M = fmaxf(M, wm[w][hh]);
  float L = 0.0f, o0 = 0.0f, o1 = 0.0f;
#pragma unroll
  for (int w = 0; w < kDnWaves; ++w) {
    const float mw = wm[w][hh];
    if (mw == -__builtin_inff()) continue;  // a wave without tiles
    const float f = __builtin_amdgcn_exp2f(mw - M);
    L = __builtin_fmaf(wl[w][hh], f, L);
    const float2 v = *reinterpret_cast<const float2*>(&cmb[(w * 8 + hh) * kD + c2]);
    o0 = __builtin_fmaf(v.x, f, o0);
    o1 = __builtin_fmaf(v.y, f, o1);
  }
  const float inv = (L > 0.0f) ? 1.0f / L : 0.0f;
  *reinterpret_cast<float2*>(&rec[kRecHeader + hh * kD + c2]) = make_float2(o0 * inv, o1 * inv);
  if ((tid & 63) == 0) {
    rec[hh] = M;
    rec[8 + hh] = L;
  }
}

}  // namespace

DensePlan plan_dense(int B, int H, int max_len) {
  const long units = (long)B * H;
  long target_groups = 256;  // one work-group per compute unit (the value tiles take 128 KiB of LDS)
  if (const char* env = getenv("OKVQ_DENSE_GROUPS")) target_groups = std::max(1L, atol(env));
  long tps = ((long)max_len * units + target_groups - 1) / target_groups;
  tps = std::max(tps, (long)kDnStep);
  tps = std::max(tps, ((long)max_len + kMaxSplits - 1) / kMaxSplits);
  tps = (tps + kDnStep - 1) / kDnStep * kDnStep;  // whole work-group steps
  DensePlan p;
  p.tokens_per_split = (int)tps;
  p.nsplit = max_len > 0 ? (int)((max_len + tps - 1) / tps) : 1;
  return p;
}

size_t dense_workspace_bytes(int B, int H, int max_len) {
  const int nsplit_max = std::max(1, std::min((max_len + kDnStep - 1) / kDnStep, kMaxSplits));
  return (size_t)B * H * nsplit_max * kRecFloats * sizeof(float);
}

hipError_t launch_decode_dense(const uint16_t* k, const uint16_t* v, const int32_t* seq_lens, const uint16_t* q, int B,
                               int H, int Hq, int cap, float sm_scale, float* out, void* ws, const DensePlan& plan,
                               hipStream_t s, hipEvent_t const* events) {
  DenseArgs a;
  a.k = k;
  a.v = v;
  a.seq_lens = seq_lens;
  a.q = q;
  a.ws = static_cast<float*>(ws);
  a.H = H;
  a.Hq = Hq;
  a.G = Hq / H;
  a.cap = cap;
  a.tps = plan.tokens_per_split;
  a.nsplit = plan.nsplit;
  a.qscale = sm_scale * 1.4426950408889634f;
  const dim3 grid(plan.nsplit, H, B), block(64 * kDnWaves);
  if (events)
    hipExtLaunchKernelGGL(k_decode_dense, grid, block, 0, s, events[0], events[1], 0, a);
  else
    hipLaunchKernelGGL(k_decode_dense, grid, block, 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_decode_merge(a.ws, B, H, Hq, plan.nsplit, out, s, events ? events + 2 : nullptr);
}

}  // namespace okvq
