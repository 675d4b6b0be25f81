// Modality-aware value-rotation calibration (Sec. 2.3, Eq. 5): the attention weight of every
// calibration token, w_j = sum_i alpha_{i,j}^2 over the causal calibration queries i of every query
// head that reads the KV head, and the weighted second moment per modality,
// C_m = sum_{j in m} w_j v_j^T v_j. The eigendecomposition and R_m = H U_m^T run on the host
// (api.hip).
//
// Scores are dense contractions on the matrix cores: v_mfma_f32_16x16x32_f16 with A = 16 query
// rows x 32 channels and B = 32 channels x 16 keys. Lane l holds A[l % 16][8 (l / 16) + e],
// B[8 (l / 16) + e][l % 16] and D[4 (l / 16) + i][l % 16]: for a row-major fp16 [token][128]
// operand, both A and B fragments of k-block kb are the 16 bytes at channel 32 kb + 8 (l / 16) of
// token l % 16 of the block.
//
//  k_calib_rowstats   (m_i, l_i) of every query row: base-2 running max and sum of 2^(s - m)
//                     over the causal keys (one wave per 16 queries, keys in blocks of 16);
//  k_calib_colweights per query head, the sum over its queries of alpha^2 for every key (per wave
//                     16 keys, every later query tile), alpha = 2^(s - m_i) / l_i;
//  k_calib_groupsum   w_j = the sum over the query heads of the group;
//  k_calib_covariance partial C_m of a 64-token chunk on the matrix cores (A = w v split into fp16
//                     hi + lo parts, B = v), one partial per (chunk, modality);
//  k_calib_reduce     C_m = the sum of the partials, in a fixed order.
#include <algorithm>

#include "launch.hpp"

namespace okvq {

typedef _Float16 c_half8 __attribute__((ext_vector_type(8)));
typedef float c_floatx4 __attribute__((ext_vector_type(4)));

constexpr int kCalThreads = 256;  // 4 waves
constexpr int kCalTile = 64;      // queries (rowstats) or keys (colweights) per work-group
constexpr int kCovChunk = 64;     // tokens per covariance work-group

__device__ __forceinline__ c_half8 as_h8(uint4 u) { return __builtin_bit_cast(c_half8, u); }

// The four k-block fragments of token row `row` (fp16 [128]) for this lane: channels
// 32 kb + 8 (lane / 16) .. + 7. Rows at or beyond `valid` read as zero.
__device__ __forceinline__ void load_frag(const uint16_t* base, int row, int valid, int lane, uint4 (&f)[4]) {
  if (row < valid) {
    const uint4* p = reinterpret_cast<const uint4*>(base + (size_t)row * kD) + (lane >> 4);
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) f[kb] = p[4 * kb];
  } else {
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) f[kb] = make_uint4(0, 0, 0, 0);
  }
}

// max over the 16 lanes of a DPP row (lanes 16 g .. 16 g + 15), in every lane: row rotations by
// 1, 2, 4, 8 on the VALU (no LDS-pipe shuffle)
__device__ __forceinline__ float row16_max(float v) {
  v = fmaxf(v, __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x121, 0xf, 0xf, false)));
  v = fmaxf(v, __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x122, 0xf, 0xf, false)));
  v = fmaxf(v, __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x124, 0xf, 0xf, false)));
  v = fmaxf(v, __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x128, 0xf, 0xf, false)));
  return v;
}
__device__ __forceinline__ float row16_sum(float v) {
  v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x121, 0xf, 0xf, false));
  v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x122, 0xf, 0xf, false));
  v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x124, 0xf, 0xf, false));
  v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x128, 0xf, 0xf, false));
  return v;
}

__device__ __forceinline__ c_floatx4 score_block(const uint4 (&a)[4], const uint4 (&b)[4]) {
  c_floatx4 d = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int kb = 0; kb < 4; ++kb) d = __builtin_amdgcn_mfma_f32_16x16x32_f16(as_h8(a[kb]), as_h8(b[kb]), d, 0, 0, 0);
  return d;
}

// Cooperative tile staging: 64 token rows (fp16 [128]) = 1024 uint4, four per thread of the
// work-group. Rows at or beyond `valid` read as zero.
struct TileRegs {
  uint4 x[4];
};
__device__ __forceinline__ void tile_load(const uint16_t* base, int row0, int valid, int tid, TileRegs& r) {
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int idx = tid + kCalThreads * u, row = row0 + (idx >> 4), part = idx & 15;
    r.x[u] = (row < valid) ? reinterpret_cast<const uint4*>(base + (size_t)row * kD)[part] : make_uint4(0, 0, 0, 0);
  }
}
// LDS tile [64 rows][128 + 8 halves] (the pad spreads the fragment reads over the banks)
constexpr int kTilePitch = kD + 8;
__device__ __forceinline__ void tile_store(_Float16* t, int tid, const TileRegs& r) {
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int idx = tid + kCalThreads * u;
    *reinterpret_cast<uint4*>(t + (idx >> 4) * kTilePitch + 8 * (idx & 15)) = r.x[u];
  }
}
// the four k-block fragments of tile row `row` for this lane
__device__ __forceinline__ void tile_frag(const _Float16* t, int row, int lane, uint4 (&f)[4]) {
#pragma unroll
  for (int kb = 0; kb < 4; ++kb) f[kb] = *reinterpret_cast<const uint4*>(t + row * kTilePitch + 32 * kb + 8 * (lane >> 4));
}

// ---- pass 1: row statistics. Grid (query tiles of 64, Hq, sequences of the launch); wave w holds
// queries 16 w .. 16 w + 15 of the tile in registers and walks the causal key tiles of 64 (staged
// in LDS, the next one loading during the current one's MFMAs). stats[(bz Hq + j) N + i] =
// (m_i, l_i): m in base-2 score units (scores times sm_scale log2 e), l_i = sum_{t <= i} 2^(s_it - m_i).
// The running max is shared by the 16 lanes of a row (reduced once per tile), so every lane keeps
// a partial sum relative to it ----
__global__ __launch_bounds__(kCalThreads) void k_calib_rowstats(const uint16_t* __restrict__ q,
                                                                const uint16_t* __restrict__ k, LenArgs lens, int b0,
                                                                int N, int H, int Hq, float scale2,
                                                                float2* __restrict__ stats) {
  __shared__ __attribute__((aligned(16))) _Float16 kt[2][kCalTile * kTilePitch];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int j = blockIdx.y, bz = blockIdx.z, b = b0 + bz;
  const int G = Hq / H, h = j / G;
  const int L = min(max(lens.lens[bz], 0), N);
  const int q0 = blockIdx.x * kCalTile;
  if (q0 >= L) return;  // (uniform over the work-group)
  const int i0 = q0 + 16 * wave;
  const uint16_t* kbase = k + ((size_t)b * H + h) * N * kD;
  const int col = lane & 15, g = lane >> 4;
  uint4 qa[4];
  load_frag(q + ((size_t)b * Hq + j) * N * kD, i0 + col, L, lane, qa);
  float m[4], l[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    m[i] = -__builtin_inff();
    l[i] = 0.0f;
  }
  const int t_end = min(q0 + kCalTile, L);  // keys of the tiles up to the diagonal one
  TileRegs r;
  tile_load(kbase, 0, t_end, tid, r);
  int buf = 0;
  for (int t0 = 0; t0 < t_end; t0 += kCalTile, buf ^= 1) {
    tile_store(kt[buf], tid, r);
    __syncthreads();  // (also: every wave is done with this buffer's previous tile, two tiles ago)
    if (t0 + kCalTile < t_end) tile_load(kbase, t0 + kCalTile, t_end, tid, r);
    float s[4][4];  // [key block][row]
    // a tile whose keys all precede the wave's first query and the length needs no mask
    const bool open = t0 + kCalTile - 1 <= i0 && t0 + kCalTile <= L;  // (wave-uniform)
#pragma unroll
    for (int kb4 = 0; kb4 < 4; ++kb4) {
      uint4 kf[4];
      tile_frag(kt[buf], 16 * kb4 + col, lane, kf);
      const c_floatx4 d = score_block(qa, kf);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int t = t0 + 16 * kb4 + col, qi = i0 + 4 * g + i;
        s[kb4][i] = (open || (t <= qi && t < L)) ? d[i] * scale2 : -__builtin_inff();
      }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float tm = row16_max(fmaxf(fmaxf(s[0][i], s[1][i]), fmaxf(s[2][i], s[3][i])));
      const float mn = fmaxf(m[i], tm);
      if (mn == -__builtin_inff()) continue;  // nothing visible to this row yet
      l[i] = l[i] * exp2f(m[i] - mn) + (exp2f(s[0][i] - mn) + exp2f(s[1][i] - mn)) +
             (exp2f(s[2][i] - mn) + exp2f(s[3][i] - mn));
      m[i] = mn;
    }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) l[i] = row16_sum(l[i]);
  if (col < 4) {  // lane 16 g + i writes row 4 g + i
    const int i = col, qi = i0 + 4 * g + i;
    const float mv = i == 0 ? m[0] : i == 1 ? m[1] : i == 2 ? m[2] : m[3];
    const float lv = i == 0 ? l[0] : i == 1 ? l[1] : i == 2 ? l[2] : l[3];
    if (qi < L) stats[((size_t)bz * Hq + j) * N + qi] = make_float2(mv, lv);
  }
}

// ---- pass 2: column weights of one query head. Grid (key tiles of 64, Hq, sequences of the
// launch); wave w holds keys 16 w .. 16 w + 15 of the tile in registers and walks the head's query
// tiles from the diagonal on (staged in LDS with their statistics as (2 m, 1 / l^2), so that
// alpha^2 = 2^(2 s - 2 m) / l^2 takes one exp2). wq[(bz Hq + j) N + t]: the head's sum over queries
// (zero beyond L); k_calib_groupsum adds the heads of each group ----
__global__ __launch_bounds__(kCalThreads) void k_calib_colweights(const uint16_t* __restrict__ q,
                                                                  const uint16_t* __restrict__ k, LenArgs lens,
                                                                  int b0, int N, int H, int Hq, float scale2,
                                                                  const float2* __restrict__ stats,
                                                                  float* __restrict__ wq) {
  __shared__ __attribute__((aligned(16))) _Float16 qt[2][kCalTile * kTilePitch];
  __shared__ __attribute__((aligned(16))) float2 st2[2][kCalTile];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int j = blockIdx.y, bz = blockIdx.z, b = b0 + bz;
  const int G = Hq / H, h = j / G;
  const int L = min(max(lens.lens[bz], 0), N);
  const int k0 = blockIdx.x * kCalTile;
  const int t0 = k0 + 16 * wave;  // this wave's 16 keys
  const int col = lane & 15, g = lane >> 4;
  const int t = t0 + col;
  float acc = 0.0f;
  if (k0 < L) {  // (uniform over the work-group)
    uint4 kf[4];
    load_frag(k + ((size_t)b * H + h) * N * kD, t0 + col, L, lane, kf);
    const float scale2x = 2.0f * scale2;
    const int ntile = (L - k0 + kCalTile - 1) / kCalTile;  // query tiles from the diagonal on
    const uint16_t* qb = q + ((size_t)b * Hq + j) * N * kD;
    const float2* sb = stats + ((size_t)bz * Hq + j) * N;
    auto load = [&](int it, TileRegs& r, float2& sv) {
      const int qtile = k0 + kCalTile * it;
      tile_load(qb, qtile, L, tid, r);
      sv = make_float2(0.f, 0.f);
      if (tid < kCalTile && qtile + tid < L) sv = sb[qtile + tid];
    };
    TileRegs r;
    float2 sv;
    load(0, r, sv);
    for (int it = 0, buf = 0; it < ntile; ++it, buf ^= 1) {
      tile_store(qt[buf], tid, r);
      // a query beyond the length gets (2 m, 1 / l^2) = (+inf, 0): its alpha^2 is 2^-inf * 0 = 0
      if (tid < kCalTile)
        st2[buf][tid] = (sv.y > 0.0f) ? make_float2(2.0f * sv.x, 1.0f / (sv.y * sv.y)) : make_float2(__builtin_inff(), 0.0f);
      __syncthreads();
      if (it + 1 < ntile) load(it + 1, r, sv);
      const int qtile = k0 + kCalTile * it;
      const bool diag = it == 0;  // the only query tile that holds queries before the wave's keys
#pragma unroll
      for (int qb4 = 0; qb4 < 4; ++qb4) {
        uint4 qa[4];
        tile_frag(qt[buf], 16 * qb4 + col, lane, qa);
        const c_floatx4 d = score_block(qa, kf);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int ql = 16 * qb4 + 4 * g + i, qi = qtile + ql;
          const float2 sm = st2[buf][ql];
          const float a2 = exp2f(__builtin_fmaf(d[i], scale2x, -sm.x)) * sm.y;
          acc += (!diag || t <= qi) ? a2 : 0.0f;
        }
      }
    }
  }
  acc += __shfl_xor(acc, 16);
  acc += __shfl_xor(acc, 32);
  if (lane < 16 && t0 + lane < N) wq[((size_t)bz * Hq + j) * N + t0 + lane] = (t0 + lane < L) ? acc : 0.0f;
}

// ---- w[(b H + h) N + t] = sum over the group's query heads, in head order. Grid (N / 256, H, nb) ----
__global__ __launch_bounds__(256) void k_calib_groupsum(const float* __restrict__ wq, int b0, int N, int H, int Hq,
                                                        float* __restrict__ w) {
  const int t = blockIdx.x * 256 + threadIdx.x, h = blockIdx.y, bz = blockIdx.z;
  if (t >= N) return;
  const int G = Hq / H;
  float s = 0.0f;
  for (int jj = 0; jj < G; ++jj) s += wq[((size_t)bz * Hq + h * G + jj) * N + t];
  w[((size_t)(b0 + bz) * H + h) * N + t] = s;
}

// ---- weighted covariance partials. Grid (chunks of 64 tokens, H, B): partial[((bz H + h) nchunk +
// chunk) 3 + m][c1][c2] = sum over the chunk's tokens t of modality m of w_t v_t[c1] v_t[c2]. The
// chunk is staged channel-major in LDS: v (fp16) and the hi / lo fp16 parts of w v. Wave w computes
// the 16 x 16 output blocks of rows 2w, 2w + 1 and every column block, modality by modality ----
__global__ __launch_bounds__(kCalThreads) void k_calib_covariance(const uint16_t* __restrict__ v,
                                                                  const uint8_t* __restrict__ modality,
                                                                  const float* __restrict__ w, LenArgs lens, int b0,
                                                                  int N, int H, int nchunk,
                                                                  float* __restrict__ partial) {
  __shared__ __attribute__((aligned(16))) _Float16 vt[kD][kCovChunk + 8];   // v[t][c] at [c][t]
  __shared__ __attribute__((aligned(16))) _Float16 whi[kD][kCovChunk + 8];  // fp16(w v)
  __shared__ __attribute__((aligned(16))) _Float16 wlo[kD][kCovChunk + 8];  // fp16(w v - hi)
  __shared__ uint8_t mods[kCovChunk];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, tid = threadIdx.x;
  const int chunk = blockIdx.x, h = blockIdx.y, bz = blockIdx.z, b = b0 + bz;
  const int L = min(max(lens.lens[bz], 0), N);
  const int tc = chunk * kCovChunk;
  const size_t seq = (size_t)b * H + h;
  // staging: thread (token tt = tid / 4, channel quarter cq = tid % 4): 32 channels of one token
  {
    const int tt = tid >> 2, cq = tid & 3, tok = tc + tt;
    const bool ok = tok < L;
    const float wt = ok ? w[seq * N + tok] : 0.0f;
    const uint4* src = reinterpret_cast<const uint4*>(v + (seq * N + (ok ? tok : 0)) * kD + 32 * cq);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const uint4 x = ok ? src[u] : make_uint4(0, 0, 0, 0);
      const c_half8 hv = as_h8(x);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int c = 32 * cq + 8 * u + e;
        const float f = (float)hv[e] * wt;
        const _Float16 hi = (_Float16)f;
        vt[c][tt] = hv[e];
        whi[c][tt] = hi;
        wlo[c][tt] = (_Float16)(f - (float)hi);
      }
    }
    if (cq == 0) mods[tt] = ok ? modality[(size_t)b * N + tok] : (uint8_t)3;
  }
  __syncthreads();
  const int col = lane & 15, g = lane >> 4;
  float* out = partial + (((size_t)bz * H + h) * nchunk + chunk) * 3 * kD * kD;
  for (int m = 0; m < 3; ++m) {
    c_floatx4 acc[2][8];
#pragma unroll
    for (int r = 0; r < 2; ++r)
#pragma unroll
      for (int cb = 0; cb < 8; ++cb) acc[r][cb] = c_floatx4{0.f, 0.f, 0.f, 0.f};
    for (int ks = 0; ks < kCovChunk; ks += 32) {
      // tokens ks + 8 g .. + 7 of this lane's fragments: keep those of modality m
      bool any = false;
      uint4 mk;  // per-element fp16 masks (0xffff keeps)
      {
        uint32_t mw[4];
#pragma unroll
        for (int p2 = 0; p2 < 4; ++p2) {
          const bool k0 = mods[ks + 8 * g + 2 * p2] == m, k1 = mods[ks + 8 * g + 2 * p2 + 1] == m;
          mw[p2] = (k0 ? 0x0000ffffu : 0u) | (k1 ? 0xffff0000u : 0u);
          any = any || k0 || k1;
        }
        mk = make_uint4(mw[0], mw[1], mw[2], mw[3]);
      }
      if (!__any(any)) continue;  // (wave-uniform)
      uint4 bf[8];
#pragma unroll
      for (int cb = 0; cb < 8; ++cb) bf[cb] = *reinterpret_cast<const uint4*>(&vt[16 * cb + col][ks + 8 * g]);
#pragma unroll
      for (int r = 0; r < 2; ++r) {
        const int c1 = 16 * (2 * wave + r) + col;
        uint4 ah = *reinterpret_cast<const uint4*>(&whi[c1][ks + 8 * g]);
        uint4 al = *reinterpret_cast<const uint4*>(&wlo[c1][ks + 8 * g]);
        ah = make_uint4(ah.x & mk.x, ah.y & mk.y, ah.z & mk.z, ah.w & mk.w);
        al = make_uint4(al.x & mk.x, al.y & mk.y, al.z & mk.z, al.w & mk.w);
#pragma unroll
        for (int cb = 0; cb < 8; ++cb) {
          acc[r][cb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(as_h8(ah), as_h8(bf[cb]), acc[r][cb], 0, 0, 0);
          acc[r][cb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(as_h8(al), as_h8(bf[cb]), acc[r][cb], 0, 0, 0);
        }
      }
    }
    // D[4 g + i][col] of block (row block 2 wave + r, column block cb)
    float* om = out + (size_t)m * kD * kD;
#pragma unroll
    for (int r = 0; r < 2; ++r)
#pragma unroll
      for (int cb = 0; cb < 8; ++cb)
#pragma unroll
        for (int i = 0; i < 4; ++i) om[(16 * (2 * wave + r) + 4 * g + i) * kD + 16 * cb + col] = acc[r][cb][i];
  }
}

// ---- C_m[c1][c2] = the sum of the partials in a fixed order: eight running sums over p = r (mod
// 8) (independent load chains), then added in r order. Grid (kD kD / 256, 3) ----
__global__ __launch_bounds__(256) void k_calib_reduce(const float* __restrict__ partial, int nparts,
                                                      float* __restrict__ cov) {
  const int e = blockIdx.x * 256 + threadIdx.x, m = blockIdx.y;
  float s[8];
#pragma unroll
  for (int r = 0; r < 8; ++r) s[r] = 0.0f;
  for (int p0 = 0; p0 < nparts; p0 += 8) {
    float x[8];
#pragma unroll
    for (int r = 0; r < 8; ++r) x[r] = (p0 + r < nparts) ? partial[((size_t)(p0 + r) * 3 + m) * kD * kD + e] : 0.0f;
#pragma unroll
    for (int r = 0; r < 8; ++r) s[r] += x[r];
  }
  cov[(size_t)m * kD * kD + e] = ((s[0] + s[1]) + (s[2] + s[3])) + ((s[4] + s[5]) + (s[6] + s[7]));
}

size_t calib_workspace_bytes(int B, int H, int Hq, int N) {
  // row statistics (float2) and the per-head column sums (float) of up to 256 sequences
  const size_t stats = (size_t)std::min(B, kMaxLenArgs) * Hq * N * (sizeof(float2) + sizeof(float));
  const size_t nchunk = (N + kCovChunk - 1) / kCovChunk;
  const size_t parts = (size_t)B * H * nchunk * 3 * kD * kD * sizeof(float);
  return std::max(stats, parts);
}

hipError_t launch_calib_weights(const uint16_t* q, const uint16_t* k, const LenArgs& lens, int b0, int nb, int N,
                                int H, int Hq, float sm_scale, float* w, void* ws, hipStream_t s) {
  const float scale2 = sm_scale * 1.4426950408889634f;
  float2* stats = static_cast<float2*>(ws);
  const dim3 gq((N + kCalTile - 1) / kCalTile, Hq, nb);
  hipLaunchKernelGGL(k_calib_rowstats, gq, dim3(kCalThreads), 0, s, q, k, lens, b0, N, H, Hq, scale2, stats);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  float* wq = reinterpret_cast<float*>(stats + (size_t)nb * Hq * N);
  hipLaunchKernelGGL(k_calib_colweights, gq, dim3(kCalThreads), 0, s, q, k, lens, b0, N, H, Hq, scale2,
                     static_cast<const float2*>(stats), wq);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(k_calib_groupsum, dim3((N + 255) / 256, H, nb), dim3(256), 0, s, static_cast<const float*>(wq), b0,
                     N, H, Hq, w);
  return hipGetLastError();
}

hipError_t launch_calib_covariance(const uint16_t* v, const uint8_t* modality, const float* w, const LenArgs& lens,
                                   int b0, int nb, int N, int H, float* partial, int part0, float* cov, bool reduce,
                                   int nparts_total, hipStream_t s) {
  const int nchunk = (N + kCovChunk - 1) / kCovChunk;
  hipLaunchKernelGGL(k_calib_covariance, dim3(nchunk, H, nb), dim3(kCalThreads), 0, s, v, modality, w, lens, b0, N, H,
                     nchunk, partial + (size_t)part0 * 3 * kD * kD);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !reduce) return e;
  hipLaunchKernelGGL(k_calib_reduce, dim3(kD * kD / 256, 3), dim3(256), 0, s, static_cast<const float*>(partial),
                     nparts_total, cov);
  return hipGetLastError();
}

}  // namespace okvq
