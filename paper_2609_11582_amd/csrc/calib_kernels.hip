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
//  k_calib_colweights w_j for every key: per wave 16 keys, every later query block of every query
//                     head of the group, alpha = 2^(s - m_i) / l_i squared and summed;
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

__device__ __forceinline__ c_floatx4 score_block(const uint4 (&a)[4], const uint4 (&b)[4]) {
  c_floatx4 d = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int kb = 0; kb < 4; ++kb) d = __builtin_amdgcn_mfma_f32_16x16x32_f16(as_h8(a[kb]), as_h8(b[kb]), d, 0, 0, 0);
  return d;
}

// ---- pass 1: row statistics. Grid (query tiles, Hq, sequences of the launch). stats[(bz Hq + j) N + i]
// = (m_i, l_i) with
// m in base-2 score units (scores times sm_scale log2 e) and l_i = sum_{t <= i} 2^(s_it - m_i) ----
__global__ __launch_bounds__(kCalThreads) void k_calib_rowstats(const uint16_t* __restrict__ q,
                                                                const uint16_t* __restrict__ k, LenArgs lens, int b0,
                                                                int N, int H, int Hq, float scale2,
                                                                float2* __restrict__ stats) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int j = blockIdx.y, bz = blockIdx.z, b = b0 + bz;
  const int G = Hq / H, h = j / G;
  const int L = min(max(lens.lens[bz], 0), N);
  const int i0 = blockIdx.x * kCalTile + 16 * wave;  // this wave's 16 queries
  if (i0 >= L) return;
  const uint16_t* qb = q + ((size_t)b * Hq + j) * N * kD;
  const uint16_t* kbase = k + ((size_t)b * H + h) * N * kD;
  uint4 qa[4];
  load_frag(qb, i0 + (lane & 15), L, lane, qa);
  const int col = lane & 15, g = lane >> 4;
  float m[4], l[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    m[i] = -__builtin_inff();
    l[i] = 0.0f;
  }
  const int t_end = min(i0 + 16, L);  // causal: keys up to the last query of the block
  uint4 kf[4], kn[4];
  load_frag(kbase, col, t_end, lane, kf);
  for (int t0 = 0; t0 < t_end; t0 += 16) {
    if (t0 + 16 < t_end) load_frag(kbase, t0 + 16 + col, t_end, lane, kn);
    const c_floatx4 d = score_block(qa, kf);
    const int t = t0 + col;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int qi = i0 + 4 * g + i;
      if (t <= qi && t < L) {
        const float s = d[i] * scale2;
        const float mn = fmaxf(m[i], s);
        l[i] = l[i] * exp2f(m[i] - mn) + exp2f(s - mn);  // m = -inf at first: exp2(-inf) = 0
        m[i] = mn;
      }
    }
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) kf[kb] = kn[kb];
  }
  // combine the 16 lanes of each row group (lanes 16 g .. 16 g + 15 hold rows 4 g .. 4 g + 3)
#pragma unroll
  for (int i = 0; i < 4; ++i) {
#pragma unroll
    for (int off = 1; off < 16; off <<= 1) {
      const float mo = __shfl_xor(m[i], off), lo = __shfl_xor(l[i], off);
      const float mn = fmaxf(m[i], mo);
      const float a = (m[i] == -__builtin_inff()) ? 0.0f : l[i] * exp2f(m[i] - mn);
      const float c = (mo == -__builtin_inff()) ? 0.0f : lo * exp2f(mo - mn);
      m[i] = mn;
      l[i] = a + c;
    }
  }
  if (col < 4) {  // lane 16 g + i writes row 4 g + i
    const int i = col, qi = i0 + 4 * g + i;
    const float mv = i == 0 ? m[0] : i == 1 ? m[1] : i == 2 ? m[2] : m[3];
    const float lv = i == 0 ? l[0] : i == 1 ? l[1] : i == 2 ? l[2] : l[3];
    if (qi < L) stats[((size_t)bz * Hq + j) * N + qi] = make_float2(mv, lv);
  }
}

// ---- pass 2: column weights. Grid (key tiles, H, B). w[(b H + h) N + t] for t < L (zero beyond) ----
__global__ __launch_bounds__(kCalThreads) void k_calib_colweights(const uint16_t* __restrict__ q,
                                                                  const uint16_t* __restrict__ k, LenArgs lens,
                                                                  int b0, int N, int H, int Hq, float scale2,
                                                                  const float2* __restrict__ stats,
                                                                  float* __restrict__ w) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int h = blockIdx.y, bz = blockIdx.z, b = b0 + bz;
  const int G = Hq / H;
  const int L = min(max(lens.lens[bz], 0), N);
  const int t0 = blockIdx.x * kCalTile + 16 * wave;  // this wave's 16 keys
  const int col = lane & 15, g = lane >> 4;
  if (t0 >= N) return;
  float acc = 0.0f;
  if (t0 < L) {
    uint4 kf[4];
    load_frag(k + ((size_t)b * H + h) * N * kD, t0 + col, L, lane, kf);
    const int t = t0 + col;
    for (int jj = 0; jj < G; ++jj) {
      const int j = h * G + jj;
      const uint16_t* qb = q + ((size_t)b * Hq + j) * N * kD;
      const float2* st = stats + ((size_t)bz * Hq + j) * N;
      uint4 qa[4], qn[4];
      float2 sr[4], sn[4];
      auto load_block = [&](int i0, uint4 (&f)[4], float2 (&s)[4]) {
        load_frag(qb, i0 + col, L, lane, f);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int qi = i0 + 4 * g + i;
          s[i] = (qi < L) ? st[qi] : make_float2(0.f, 1.f);
        }
      };
      load_block(t0, qa, sr);  // causal: queries from the wave's first key on
      for (int i0 = t0; i0 < L; i0 += 16) {
        if (i0 + 16 < L) load_block(i0 + 16, qn, sn);
        const c_floatx4 d = score_block(qa, kf);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int qi = i0 + 4 * g + i;
          if (t <= qi && qi < L && t < L) {
            const float a = exp2f(d[i] * scale2 - sr[i].x) / sr[i].y;
            acc = __builtin_fmaf(a, a, acc);
          }
        }
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) qa[kb] = qn[kb];
#pragma unroll
        for (int i = 0; i < 4; ++i) sr[i] = sn[i];
      }
    }
  }
  acc += __shfl_xor(acc, 16);
  acc += __shfl_xor(acc, 32);
  if (lane < 16 && t0 + lane < N) w[((size_t)b * H + h) * N + t0 + lane] = (t0 + lane < L) ? acc : 0.0f;
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

// ---- C_m[c1][c2] = sum over the partials in index order. Grid (kD kD / 256, 3) ----
__global__ __launch_bounds__(256) void k_calib_reduce(const float* __restrict__ partial, int nparts,
                                                      float* __restrict__ cov) {
  const int e = blockIdx.x * 256 + threadIdx.x, m = blockIdx.y;
  float s = 0.0f;
  for (int p = 0; p < nparts; ++p) s += partial[((size_t)p * 3 + m) * kD * kD + e];
  cov[(size_t)m * kD * kD + e] = s;
}

size_t calib_workspace_bytes(int B, int H, int Hq, int N) {
  const size_t stats = (size_t)std::min(B, kMaxLenArgs) * Hq * N * sizeof(float2);
  const size_t nchunk = (N + kCovChunk - 1) / kCovChunk;
  const size_t parts = (size_t)B * H * nchunk * 3 * kD * kD * sizeof(float);
  return std::max(stats, parts);
}

hipError_t launch_calib_weights(const uint16_t* q, const uint16_t* k, const LenArgs& lens, int b0, int nb, int N,
                                int H, int Hq, float sm_scale, float* w, void* ws, hipStream_t s) {
  const float scale2 = sm_scale * 1.4426950408889634f;
  float2* stats = static_cast<float2*>(ws);
  const dim3 gq((N + kCalTile - 1) / kCalTile, Hq, nb), gk((N + kCalTile - 1) / kCalTile, H, nb);
  hipLaunchKernelGGL(k_calib_rowstats, gq, dim3(kCalThreads), 0, s, q, k, lens, b0, N, H, Hq, scale2, stats);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_calib_colweights, gk, dim3(kCalThreads), 0, s, q, k, lens, b0, N, H, Hq, scale2,
                     static_cast<const float2*>(stats), w);
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
