// Key and value codec kernels, shared by the stateless calls and by append.
//
// A "job" names where token rows come from. Stateless calls quantize tokens [0, len) of a
// dense block. Append quantizes the tokens [begin, begin + count) that follow a sequence's
// current length `begin` (device values): keys from the first window that is still open (its
// older raw rows come from the fp16 stage, so the window is re-quantized as a whole), values
// token by token (the code bytes shared with older tokens are merged, not overwritten).
#include "key_quant.hpp"
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
// Keys: grid (tiles of 256 tokens from the first open window, H, batches); 4 waves per block,
// 64 tokens (two windows) per wave.
// ------------------------------------------------------------------------------------------------
// Token rows of one wave: older rows of the open window from the stage, then the new rows;
// zeros beyond the length.
__device__ __forceinline__ void load_key_rows(const CodecJob& j, size_t seq, int begin, int len, int first, int tok0,
                                              uint32_t (&raw)[64]) {
  const int tok = tok0 + lane_id();
  if (tok < begin) {
    load_row_f16(j.stage + (seq * kW + (tok - first)) * kD, raw);
  } else if (tok < len) {
    load_row_f16(j.src + (seq * j.n_rows + (tok - begin)) * kD, raw);
  } else {
#pragma unroll
    for (int i = 0; i < 64; ++i) raw[i] = 0;
  }
}

__global__ __launch_bounds__(256) void k_quantize_keys(CodecJob j, const int8_t* __restrict__ signs,
                                                       uint8_t* __restrict__ k_codes, uint16_t* __restrict__ k_min,
                                                       uint16_t* __restrict__ k_step, uint16_t* __restrict__ k_norm) {
  __shared__ __attribute__((aligned(16))) float lds[4 * kKeyWaveLds];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform for the compiler
  const int h = blockIdx.y, bz = blockIdx.z, b = j.b0 + bz;
  const size_t seq = (size_t)b * j.H + h;
  // rows from the planned lengths (append: the host's copy), then the device lengths decide
  int begin = j.begin_dev ? j.lens.lens[bz] : 0;
  int len = j.begin_dev ? begin + j.cnts.lens[bz] : j.lens.lens[bz];
  int first = (begin / kW) * kW;  // first token of the first open window
  int tok0 = first + (blockIdx.x * 4 + wave) * 64;
  uint32_t raw[64];
  load_key_rows(j, seq, begin, len, first, tok0, raw);
  if (j.begin_dev) {
    const int bd = min(max(j.begin_dev[b], 0), j.cap);
    const int ld = min(bd + min(max(j.count_dev[b], 0), j.n_rows), j.cap);
    if (bd != begin || ld != len) {  // stale host lengths: reload from the device ones
      begin = bd;
      len = ld;
      first = (begin / kW) * kW;
      tok0 = first + (blockIdx.x * 4 + wave) * 64;
      load_key_rows(j, seq, begin, len, first, tok0, raw);
    }
  }
  if (len <= begin || tok0 >= len) return;  // no block-level barrier is used below
  uint32_t sw[32];
  load_sign_words(signs, sw);
  const int tok = tok0 + lane_id();
  if (j.stage && tok0 == first) {
    // The wave holding the old open window rewrites the stage with the raw rows of the new
    // open window [open, len). Only this wave reads or writes the stage of (b, h).
    const int open = (len / kW) * kW;
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");  // the stage reads above have completed
    if (open < len) {
      const int slot = lane_id() & 31;
      const int src_tok = open + slot;
      uint16_t* dst = j.stage + (seq * kW + slot) * kD;
      if (open < tok0 + 64) {
        if (tok >= open && tok < len) {
          uint4* d4 = reinterpret_cast<uint4*>(dst);
#pragma unroll
          for (int i = 0; i < 16; ++i) d4[i] = make_uint4(raw[4 * i], raw[4 * i + 1], raw[4 * i + 2], raw[4 * i + 3]);
        }
      } else if (lane_id() < 32 && src_tok < len) {
        const uint4* s4 = reinterpret_cast<const uint4*>(j.src + (seq * j.n_rows + (src_tok - begin)) * kD);
        uint4* d4 = reinterpret_cast<uint4*>(dst);
#pragma unroll
        for (int i = 0; i < 16; ++i) d4[i] = s4[i];
      }
    }
  }
  KeyWaveOut out{k_codes + seq * j.cap * 32, k_min + seq * (j.cap / kW) * kD, k_step + seq * (j.cap / kW) * kD,
                 k_norm + seq * j.cap};
  key_quantize_wave(raw, tok0, len, sw, out, lds + wave * kKeyWaveLds);
}

hipError_t launch_quantize_keys(const CodecJob& j, int nb, int max_tiles_tokens, const int8_t* signs,
                                uint8_t* k_codes, uint16_t* k_min, uint16_t* k_step, uint16_t* k_norm,
                                hipStream_t s) {
  if (max_tiles_tokens <= 0 || nb <= 0) return hipSuccess;
  dim3 grid((max_tiles_tokens + 255) / 256, j.H, nb);
  hipLaunchKernelGGL(k_quantize_keys, grid, dim3(256), 0, s, j, signs, k_codes, k_min, k_step, k_norm);
  return hipGetLastError();
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
    const float* r = rot + ((size_t)m * kD + c) * kD;
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

hipError_t launch_quantize_values_mfma(const CodecJob& j, int nb, int max_tiles_tokens, const float* rot,
                                       const Thresholds& th, uint8_t* v_codes, uint16_t* v_norm,
                                       uint8_t* mod_out, hipStream_t s);

hipError_t launch_quantize_values(const CodecJob& j, int nb, int max_tiles_tokens, const float* rot,
                                  const Thresholds& th, bool exact, uint8_t* v_codes, uint16_t* v_norm,
                                  uint8_t* mod_out, hipStream_t s) {
  if (max_tiles_tokens <= 0 || nb <= 0) return hipSuccess;
  if (!exact) return launch_quantize_values_mfma(j, nb, max_tiles_tokens, rot, th, v_codes, v_norm, mod_out, s);
  dim3 grid((max_tiles_tokens + kW - 1) / kW, j.H, nb);
  hipLaunchKernelGGL(k_quantize_values_exact, grid, dim3(128), 0, s, j, rot, th, v_codes, v_norm, mod_out);
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
