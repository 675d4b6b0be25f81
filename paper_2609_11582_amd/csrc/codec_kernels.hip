// Exact-mode value codec and the length update of append.
//
// A "job" names where token rows come from. Stateless calls quantize tokens [0, len) of a
// dense block. Append quantizes the tokens [begin, begin + count) that follow a sequence's
// current length `begin` (device values), token by token (the code bytes shared with older
// tokens are merged, not overwritten). The MFMA-mode values and the keys: codec_fused.hip.
#include "launch.hpp"
#include "value_quant.hpp"

namespace okvq {

__device__ __forceinline__ void job_range(const CodecJob& j, int bz, int b, int& begin, int& len) {
  if (j.begin_dev) {  // clamped: device lengths outside the contract stay memory-safe
    begin = min(max(j.begin_dev[b], 0), j.cap);
    len = min(begin + min(max(j.count_dev[b], 0), j.n_rows), j.cap);
  } else {
    begin = 0;
    len = j.lens.lens[bz];
  }
}

// ------------------------------------------------------------------------------------------------
// Values, exact mode: one block of 128 threads (thread = output channel) per 32-token window.
// y_c = sum_j fl(R_cj * v_j) accumulated left to right in fp32.
// ------------------------------------------------------------------------------------------------
__device__ __forceinline__ float halving_tree_norm(const float* xs) {  // xs: 128 floats (LDS)
  float t[64];
#pragma unroll
  for (int i = 0; i < 64; ++i) t[i] = xs[i] * xs[i] + xs[i + 64] * xs[i + 64];
#pragma unroll
  for (int n = 32; n >= 1; n >>= 1) {
#pragma unroll
    for (int i = 0; i < n; ++i) t[i] = t[i] + t[i + n];
  }
  return sqrt_rn(t[0]);
}

__global__ __launch_bounds__(128) void k_quantize_values_exact(CodecJob j, const float* __restrict__ rot, Thresholds th,
                                                               uint8_t* __restrict__ v_codes,
                                                               uint16_t* __restrict__ v_norm,
                                                               uint8_t* __restrict__ mod_out) {
  __shared__ __attribute__((aligned(16))) float xs[kW][kD];
  __shared__ float nrm[kW];
  __shared__ int mods[kW];
  const int h = blockIdx.y, bz = blockIdx.z, b = j.b0 + bz;
  int begin, len;
  job_range(j, bz, b, begin, len);
  if (len <= begin) return;
  const int t0 = (begin / kW + (int)blockIdx.x) * kW;
  if (t0 >= len) return;
  const int c = threadIdx.x;
  const size_t seq = (size_t)b * j.H + h;
  for (int t = 0; t < kW; ++t) {
    const int tok = t0 + t;
    xs[t][c] = (tok >= begin && tok < len) ? h2f(j.src[(seq * j.n_rows + (tok - begin)) * kD + c]) : 0.0f;
  }
  if (c < kW) {
    const int tok = t0 + c;
    int m = -1;
    if (tok >= begin && tok < len) {
      m = (int)j.msrc[(size_t)b * j.n_rows + (tok - begin)];
      if (mod_out && h == 0) mod_out[(size_t)b * j.cap + tok] = (uint8_t)m;
    }
    mods[c] = m;
  }
  __syncthreads();
  if (c < kW) {
    const int tok = t0 + c;
    const bool fresh = tok >= begin && tok < len;
    const uint32_t n16 = fresh ? norm_to_f16(halving_tree_norm(xs[c])) : 0u;
    nrm[c] = h2f(n16);
    if (tok >= begin) v_norm[seq * j.cap + tok] = (uint16_t)n16;
  }
  __syncthreads();
  uint32_t bytes[8];
#pragma unroll
  for (int gq = 0; gq < 8; ++gq) bytes[gq] = 0;
  for (int t = 0; t < kW; ++t) {
    const int m = mods[t];
    if (m < 0 || m > 2) continue;  // old, padded or out-of-contract token: code 0 here
    const float* r = rot + ((size_t)(j.global_rot ? 0 : m) * kD + c) * kD;
    float acc = 0.0f;
    for (int k = 0; k < kD; ++k) acc = acc + r[k] * xs[t][k];
    bytes[t >> 2] |= value_code(acc, nrm[t], th) << (2 * (t & 3));
  }
  uint8_t* dst = v_codes + (seq * (j.cap / kW) + t0 / kW) * 1024;
#pragma unroll
  for (int gq = 0; gq < 8; ++gq) {
    const int idx = value_byte_index(4 * gq, c);
    const int old_tokens = min(max(begin - (t0 + 4 * gq), 0), 4);  // leading tokens of the byte kept
    if (old_tokens == 4) continue;
    uint32_t v8 = bytes[gq];
    if (old_tokens > 0) {
      const uint32_t keep = (1u << (2 * old_tokens)) - 1u;
      v8 = (dst[idx] & keep) | (v8 & ~keep);
    }
    dst[idx] = (uint8_t)v8;
  }
}

hipError_t launch_quantize_values_exact(const CodecJob& j, int nb, int max_tiles_tokens, const float* rot,
                                        const Thresholds& th, uint8_t* v_codes, uint16_t* v_norm, uint8_t* mod_out,
                                        hipStream_t s) {
  if (max_tiles_tokens <= 0 || nb <= 0) return hipSuccess;
  dim3 grid((max_tiles_tokens + kW - 1) / kW, j.H, nb);
  hipLaunchKernelGGL(k_quantize_values_exact, grid, dim3(128), 0, s, j, rot, th, v_codes, v_norm, mod_out);
  return hipGetLastError();
}

// ------------------------------------------------------------------------------------------------
// fp16 residual of the captioning protocol (Sec. 3.1): the raw key and value rows of the appended
// tokens that are among the last 128 of their sequence go to row token % 128 of the ring buffers.
// One work-group per (sequence, KV head); runs before the codec launch advances the lengths.
// ------------------------------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_residual_store(const uint16_t* __restrict__ k_new,
                                                        const uint16_t* __restrict__ v_new, int n_rows,
                                                        const int32_t* __restrict__ begin_dev,
                                                        const int32_t* __restrict__ count_dev, int H, int cap,
                                                        uint16_t* __restrict__ k_res, uint16_t* __restrict__ v_res) {
  const int seq = blockIdx.x, b = seq / H;
  const int begin = min(max(begin_dev[b], 0), cap);  // clamped like the codec's device lengths
  const int end = min(begin + min(max(count_dev[b], 0), n_rows), cap);
  const int first = max(end - kResidual, begin);
  const int nrow = end - first;  // <= 128: every ring row is written at most once
  const uint4* ks = reinterpret_cast<const uint4*>(k_new + (size_t)seq * n_rows * kD);
  const uint4* vs = reinterpret_cast<const uint4*>(v_new + (size_t)seq * n_rows * kD);
  uint4* kd = reinterpret_cast<uint4*>(k_res + (size_t)seq * kResidual * kD);
  uint4* vd = reinterpret_cast<uint4*>(v_res + (size_t)seq * kResidual * kD);
  for (int idx = threadIdx.x; idx < nrow * 16; idx += 256) {  // 16 uint4 per 128-channel row
    const int tok = first + (idx >> 4), part = idx & 15;
    const size_t src = (size_t)(tok - begin) * 16 + part;
    const int dst = (tok & (kResidual - 1)) * 16 + part;
    kd[dst] = ks[src];
    vd[dst] = vs[src];
  }
}

hipError_t launch_residual_store(const uint16_t* k_new, const uint16_t* v_new, int n_rows, const int32_t* begin_dev,
                                 const int32_t* count_dev, int B, int H, int cap, uint16_t* k_res, uint16_t* v_res,
                                 hipStream_t s) {
  if (n_rows <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_residual_store, dim3(B * H), dim3(256), 0, s, k_new, v_new, n_rows, begin_dev, count_dev, H, cap,
                     k_res, v_res);
  return hipGetLastError();
}

// seq_lens[b] += count[b] after an append (stream-ordered after the codec kernels that read them).
__global__ void k_advance_lengths(int32_t* seq_lens, const int32_t* count, int B) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b < B) seq_lens[b] += count[b];
}

hipError_t launch_advance_lengths(int32_t* seq_lens, const int32_t* count, int B, hipStream_t s) {
  hipLaunchKernelGGL(k_advance_lengths, dim3((B + 255) / 256), dim3(256), 0, s, seq_lens, count, B);
  return hipGetLastError();
}

}  // namespace okvq
