// Internal launchers shared by the C ABI (api.hip) and the kernel translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "okvq_device.hpp"
#include "value_quant.hpp"

namespace okvq {

// Where the codec kernels read token rows. Stateless calls (begin_dev == nullptr) quantize tokens
// [0, lens[b - b0]) of a dense block. Append quantizes tokens [begin_dev[b], begin_dev[b] +
// count_dev[b]) whose rows are src row (token - begin); older rows of the open key window come
// from the fp16 stage. For append, lens / cnts hold the host's copy of the same lengths: the
// kernels issue their row loads from them and then check the device values (which decide).
struct CodecJob {
  const uint16_t* src;       // [B][H][n_rows][128] fp16
  const uint8_t* msrc;       // [B][n_rows] modality ids (values only)
  int n_rows;
  LenArgs lens;              // lengths (stateless) or current lengths (append) of batches b0 .. b0 + 255
  LenArgs cnts;              // append: appended tokens of the same batches
  const int32_t* begin_dev;  // append: current lengths (device)
  const int32_t* count_dev;  // append: appended tokens (device)
  uint16_t* stage;           // append: [B][H][32][128] raw keys of the open window
  int b0, H, cap;
  int global_rot;            // values: R_0 rotates every token (the single global rotation)
};

// Exact-mode values (OKVQ_VALUE_EXACT): one work-group per 32-token window.
hipError_t launch_quantize_values_exact(const CodecJob& j, int nb, int max_tiles_tokens, const float* rot,
                                        const Thresholds& th, uint8_t* v_codes, uint16_t* v_norm, uint8_t* mod_out,
                                        hipStream_t s);

// Forward rotation of the MFMA-mode values as ready-made MFMA B operands: 3 modalities x 8 output
// blocks x 4 k-blocks x (fp16 hi, fp16 lo) fragments of 64 lanes x 16 bytes.
constexpr int kRotFragments = 3 * 8 * 4 * 2;
constexpr size_t kRotInverseBytes = 128 * 3 * 128 * 2;          // decode's inverse-rotation table
constexpr size_t kRotFragmentBytes = (size_t)kRotFragments * 1024;

// Arguments of the fused codec launch (keys, MFMA-mode values, or both) over tiles of 256 tokens.
struct CodecArgs {
  CodecJob j;
  int ntx;     // tiles per sequence (covering the longest span from a first open window)
  int ntiles;  // ntx * H * sequences in the launch
  // keys
  const int8_t* signs;
  uint8_t* k_codes;
  uint16_t* k_min;   // fp16 window metadata, or
  uint16_t* k_step;
  uint8_t* k_mx;     // MXFP4 window records
  uint16_t* k_norm;
  int key_meta;      // kMetaFp16, kMetaMx or kMetaTq (TurboQuant keys: codes against th, no metadata)
  // values
  const uint16_t* vsrc;  // value rows, laid out like j.src (the key rows)
  const float* rot;      // fp32 R_m (used when rotfrag is null)
  const uint4* rotfrag;  // prepared forward fragments, or null
  Thresholds th;
  uint8_t* v_codes;
  uint16_t* v_norm;
  uint8_t* mod_out;  // append: the cache's modality map (written for KV head 0), else null
  // append: the last work-group to finish adds count_dev[b] to seq_lens[b] for the launch's
  // sequences; `ticket` counts finished work-groups and is returned to zero
  int32_t* seq_lens_out;
  uint32_t* ticket;
  // append: status word set to 1 if a value wave stops waiting for the others (kSpinLimit polls,
  // or the host override below) and goes on with the tables it has; null for the stateless calls
  int32_t* status;
  int spin_limit;  // polls of a value-wave wait before it gives up (set by launch_codec)
  // window path only: the fp16 residual rings (null without them)
  uint16_t* k_res;
  uint16_t* v_res;
};
// events (optional): two events recorded at the start and end of the launch's execution
hipError_t launch_codec(const CodecArgs& a, bool keys, bool values, hipStream_t s, hipEvent_t const* events = nullptr);
// Window-parallel append (MFMA-mode values; fp16 window metadata or TurboQuant keys): one launch
// over nwin key windows per sequence from each open window, with the residual rings and the length
// update (seq_lens_out, ticket as for the tile launch). Writes the tile codec's bytes.
hipError_t launch_append_window(const CodecArgs& a, int nwin, int nb, hipStream_t s, hipEvent_t const* events = nullptr);
hipError_t launch_prepare_fragments(const float* rot, uint4* frag, hipStream_t s);
hipError_t launch_advance_lengths(int32_t* seq_lens, const int32_t* count, int B, hipStream_t s);
// Residual rings: rows of the appended tokens among the last 128 of each sequence (device lengths).
hipError_t launch_residual_store(const uint16_t* k_new, const uint16_t* v_new, int n_rows, const int32_t* begin_dev,
                                 const int32_t* count_dev, int B, int H, int cap, uint16_t* k_res, uint16_t* v_res,
                                 hipStream_t s);

// Value-rotation calibration (Eq. 5): attention weights of up to 256 sequences per launch (the
// workspace holds their row statistics), weighted covariance partials per (sequence, head, 64-token
// chunk) and their reduction.
size_t calib_workspace_bytes(int B, int H, int Hq, int N);
hipError_t launch_calib_weights(const uint16_t* q, const uint16_t* k, const LenArgs& lens, int b0, int nb, int N,
                                int H, int Hq, float sm_scale, float* w, void* ws, hipStream_t s);
hipError_t launch_calib_covariance(const uint16_t* v, const uint8_t* modality, const float* w, const LenArgs& lens,
                                   int b0, int nb, int N, int H, float* partial, int part0, float* cov, bool reduce,
                                   int nparts_total, hipStream_t s);
constexpr int kCalibChunk = 64;  // tokens per covariance partial

struct CacheView {
  int B, H, Hq, cap;
  uint8_t* k_codes;
  uint8_t* v_codes;
  uint16_t* k_norm;
  uint16_t* v_norm;
  uint16_t* k_min;
  uint16_t* k_step;
  uint8_t* k_mx;  // MXFP4 window records, or null for fp16 k_min / k_step
  int key_meta;   // kMetaFp16, kMetaMx or kMetaTq
  uint8_t* modality;
  uint16_t* k_stage;
  int32_t* seq_lens;
  const int8_t* signs;
  const float* rot;
  const uint16_t* rot16t;  // prepared rotation tables: [128][3][128] fp16 inverse, then forward fragments
  int residual;            // 0, or kResidual: the last tokens are read in fp16 from k_res / v_res
  const uint16_t* k_res;   // [B][H][128][128] fp16 rings (token i in row i % 128)
  const uint16_t* v_res;
  int key_bits, value_bits;  // 0: the 2-bit layout above; 2..4: the bit-width ladder layout
};

// Split record of the split-K decode launches (read by the log-sum-exp merge): the running max
// M[8] and sum L[8] of the 8 query-head slots, then o[8][128] divided by L.
constexpr int kRecHeader = 32;
constexpr int kRecFloats = kRecHeader + 8 * kD;
constexpr int kMaxSplits = 1024;  // most splits per (sequence, KV head)

// Record of a split with no tokens (ragged batches): M = -inf, L = 0 and zero outputs, so the
// merge never reads memory this launch did not write. Threads tid < 256 of the work-group call it.
__device__ __forceinline__ void write_empty_record(float* rec, int tid) {
  if (tid < 8) {
    rec[tid] = -__builtin_inff();
    rec[8 + tid] = 0.0f;
  }
  if (tid < 8 * kD / 4) reinterpret_cast<float4*>(rec + kRecHeader)[tid] = make_float4(0.f, 0.f, 0.f, 0.f);
}

struct DecodePlan {
  int wins_per_split;  // 32-token windows per split-K work-group
  int nsplit;          // splits per (sequence, KV head)
};
DecodePlan plan_decode(int B, int H, int max_len);
size_t decode_workspace_bytes(int B, int H, int Hq, int max_len);
hipError_t launch_prepare_rotation(const float* rot, uint16_t* rot16t, hipStream_t s);
// events: nullptr, or four events bound to the launches: split-K start, end; merge start, end
// global_rot: the cache's values were all rotated by R_0 (one accumulator, one un-rotation)
hipError_t launch_decode(const CacheView& c, const uint16_t* q, float sm_scale, float* out, void* ws,
                         const DecodePlan& plan, hipStream_t s, uint32_t cb01, uint32_t cb23, int max_len,
                         hipEvent_t const* events, bool global_rot);

// Log-sum-exp merge of split records [B][H][nsplit][kRecFloats] into out [B][Hq][128]; events:
// nullptr, or two events bound to the launch (start, end).
hipError_t launch_decode_merge(const float* ws, int B, int H, int Hq, int nsplit, float* out, hipStream_t s,
                               hipEvent_t const* events);

// Dense fp16 decode attention (the comparison baseline): split-K over 256-token steps, then the
// same merge. events: nullptr, or four events (split start, end; merge start, end).
struct DensePlan {
  int tokens_per_split;
  int nsplit;
};
DensePlan plan_dense(int B, int H, int max_len);
size_t dense_workspace_bytes(int B, int H, int max_len);
hipError_t launch_decode_dense(const uint16_t* k, const uint16_t* v, const int32_t* seq_lens, const uint16_t* q, int B,
                               int H, int Hq, int cap, float sm_scale, float* out, void* ws, const DensePlan& plan,
                               hipStream_t s, hipEvent_t const* events);

// ---- bit-width ladder: b-bit keys and values (b = 2, 3, 4) in the token-major bit-stream layout ----
// Stateless calls (begin_dev == nullptr): tokens [0, lens[b - b0]) of a dense block. Append:
// tokens [begin_dev[b], begin_dev[b] + count_dev[b]) whose rows are row (token - begin) of the
// block; the device lengths decide (clamped into the buffers) and the host's copy only sizes the
// grid. The method's keys requantize the open window from `first` = 32 floor(begin / 32), its older
// rows taken from the fp16 stage; TurboQuant keys and values are per token and start at begin.
struct LadderKeyArgs {
  const uint16_t* k;  // [B][H][n_rows][128] fp16
  int n_rows, H, cap, b0;
  LenArgs lens;
  const int32_t* begin_dev;  // append: current lengths (device), else null
  const int32_t* count_dev;  // append: appended tokens (device)
  uint16_t* stage;           // append, method keys: [B][H][32][128] raw keys of the open window
  const int8_t* signs;
  uint8_t* k_codes;   // [B][H][cap][16 b]
  uint16_t* k_min;    // [B][H][cap/32][128] fp16 (method keys)
  uint16_t* k_step;
  uint16_t* k_norm;   // [B][H][cap]
  float tau[15];      // TurboQuant keys: the 2^b - 1 thresholds (fp32, ascending)
};
struct LadderValueArgs {
  const uint16_t* v;  // [B][H][n_rows][128] fp16
  const uint8_t* modality;  // [B][n_rows]
  int n_rows, H, cap, b0;
  LenArgs lens;
  const int32_t* begin_dev;  // append: as for the keys
  const int32_t* count_dev;
  uint8_t* mod_out;          // append: the cache's modality map (written by KV head 0), else null
  const float* rot;   // [3][128][128] fp32
  uint8_t* v_codes;   // [B][H][cap][16 b]
  uint16_t* v_norm;
  float tau[15];
};
// max_len: the longest span of tokens from a tile start to the end (stateless: the longest length;
// append: for the method's keys the longest length - first, else the most appended tokens)
hipError_t launch_ladder_keys(const LadderKeyArgs& a, int bits, bool tq, int nb, int max_len, hipStream_t s);
// exact: the sequential fp32 order (bit-exact codes); else the matrix cores (fp16 hi + lo split of R_m)
hipError_t launch_ladder_values(const LadderValueArgs& a, int bits, bool exact, int nb, int max_len, hipStream_t s);

struct LadderDecodeArgs {
  const uint8_t* k_codes;
  const uint8_t* v_codes;
  const uint16_t* k_norm;
  const uint16_t* v_norm;
  const uint16_t* k_min;   // null for TurboQuant keys
  const uint16_t* k_step;
  const uint8_t* modality;
  const int32_t* seq_lens;
  const int8_t* signs;
  const uint16_t* q;
  const uint16_t* rot16t;
  float* ws;
  int H, Hq, G, cap, tps, nsplit;
  float qscale;            // sm_scale log2(e) / sqrt(128) (the butterflies are unnormalized)
  uint16_t kcb16[16];      // fp16 levels of the key codebook (TurboQuant keys)
  uint16_t vcb16[16];      // fp16 levels of the value codebook
};
struct LadderPlan {
  int tokens_per_split;
  int nsplit;
};
LadderPlan plan_ladder(int B, int H, int max_len);
size_t ladder_workspace_bytes(int B, int H, int max_len);
hipError_t launch_ladder_decode(const LadderDecodeArgs& a, int key_bits, int value_bits, bool tq, int B,
                                const LadderPlan& plan, float* out, hipStream_t s, hipEvent_t const* events);

}  // namespace okvq
