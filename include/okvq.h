/*
 * okvq.h -- C ABI of the OmniKVQuant 2-bit KV-cache hot path for AMD Instinct MI355X (gfx950).
 *
 * The method (arXiv 2609.11582, "OmniKVQuant: KV Cache Quantization for Omni-LLMs"):
 *   keys   -- per-token norm split and randomized Hadamard rotation (Sec. 2.1, Eq. 2), then
 *             min / step per group of 32 consecutive tokens and channel (Sec. 2.3, Eq. 4),
 *             2-bit codes;
 *   values -- per-token norm split, rotation by a per-modality orthogonal matrix R_m
 *             (audio / video / text; Sec. 2.3, Eq. 6), 2-bit codes of the fixed Gaussian
 *             codebook (Eq. 3);
 *   decode -- softmax attention of one query per head over the packed cache (Eq. 1), scoring
 *             in the rotated key space after rotating the query once per head, and applying
 *             the inverse value rotation once per modality after aggregation (Sec. 2.3).
 *
 * Conventions shared by every call
 * --------------------------------
 * - head_dim must be 128 and window 32; 1 <= num_q_heads / num_kv_heads <= 8 with
 *   num_q_heads a multiple of num_kv_heads (query head j reads KV head j / G).
 * - Every array argument named "device" is device memory of the current HIP device, caller
 *   owned and 16-byte aligned. fp16 data is passed as uint16_t bit patterns (IEEE binary16).
 * - The library allocates no memory, keeps no state between calls and (except okvq_cache_status)
 *   never synchronizes and never copies between host and device: each call validates its
 *   arguments on the host and then enqueues kernels on `stream` (a hipStream_t; NULL is the
 *   default stream).
 * - Argument errors are detected before anything is enqueued: the call returns a negative
 *   status and writes nothing. A failed kernel launch returns OKVQ_ERR_HIP.
 * - Device data contract: inputs are finite and modality ids are 0, 1 or 2. Violations give
 *   unspecified (but memory-safe) results. The one device-side error channel is the cache's
 *   status word (seq_lens[B + 1], read by okvq_cache_status).
 * - Host "lens" arrays plan the launches; the kernels read lengths on the device where noted.
 *   Callers keep the two equal.
 *
 * Cache layout (per layer; B = batch, H = num_kv_heads, cap = capacity, a multiple of 32)
 * ------------------------------------------------------------------------------------------
 *   k_codes  u8  [B][H][cap][32]      token i, channel c -> byte 32i + 4(c/16) + 2(c%2) + (c/8)%2,
 *                                      bits 2((c/2)%4)..+1 (32-bit word t: channels 16t..16t+15,
 *                                      even ones in the low half, odd ones in the high half)
 *   v_codes  u8  [B][H][cap/32][1024] window token t, channel c -> byte
 *                                      16*((c%16) + 16*((t/4)%4)) + 8*(t/16) + c/16,
 *                                      bits 2(t%4)..+1 (one channel of 4 consecutive tokens)
 *   k_norm   f16 [B][H][cap]          fp16 ||k||
 *   v_norm   f16 [B][H][cap]          fp16 ||v||
 *   k_min    f16 [B][H][cap/32][128]  per (window, channel) minimum of the rotated key direction
 *   k_step   f16 [B][H][cap/32][128]  per (window, channel) step = (max - min) / 3
 *   modality u8  [B][cap]             0 audio, 1 video, 2 text
 *   k_stage  f16 [B][H][32][128]      raw keys of the open (partial) window, used by append
 *   seq_lens i32 [B + 2]              current lengths (device copy), then one word append uses as
 *                                      a work-group counter (zero initially; append leaves it zero),
 *                                      then the status word (zero initially; append sets it to 1 if
 *                                      a wait between the value codec's waves gave up, after which
 *                                      that append's value codes may be wrong; never cleared by
 *                                      the library)
 * Slots of the last window beyond a sequence's length hold code 0 and norm 0.
 * Storage is 84 bytes per token per KV head: 2.625 bits per element, the "FP16 meta." row of
 * the paper's Tab. 3.
 *
 * MXFP4 key metadata (dims.key_meta = OKVQ_KEY_META_MXFP4, the paper's default, Sec. 3.1 and
 * Tab. 3 "Ours (MXFP4 meta.)"): k_min and k_step are replaced by
 *   k_mx     u8  [B][H][cap/32][136]  one record per window. The window's fp32 minimum vector and
 *                                      its fp32 step vector (max - min) / 3 are each stored as
 *                                      MXFP4: 4 blocks of 32 channels, every block one E8M0 scale
 *                                      2^e (byte e + 127, e = floor(log2(max |x|)) - 2, clamped
 *                                      to [-127, 127]; -127 for an all-zero block) and 32 FP4
 *                                      E2M1 elements (nearest value of x / 2^e, ties to even,
 *                                      saturating at 6; the sign is kept). Bytes 4q..4q+1: the
 *                                      minimum's elements of channels 4q..4q+3 (channel 4q + i
 *                                      in bits 4i..4i+3); bytes 4q+2..4q+3: the step's; byte
 *                                      128 + 2b: the minimum's scale of block b (channels
 *                                      32b..32b+31); byte 129 + 2b: the step's scale.
 * Key codes are then computed against the dequantized minimum m and step s (code 0 where s is
 * zero, else clamp(rint(fl(fl(z - m) * fl(1 / s))), 0, 3)). Storage: 72.25 bytes per token per
 * KV head, 2.258 bits per element.
 *
 * TurboQuant keys (dims.key_meta = OKVQ_KEY_META_TURBOQUANT, the paper's baseline, Sec. 2.1 Eq. 2
 * and Eq. 3): the key direction z (as above: fp16 norm, Hadamard butterflies, z = w fl(kappa / n16))
 * takes the nearest entry of the same fixed Gaussian codebook as the values, code = #{k : z_c >
 * tau_k} (a value on a threshold takes the lower code), in the k_codes layout; k_min, k_step and
 * k_mx are not used. Storage: 68 bytes per token per KV head, 2.125 bits per element (Tab. 3
 * "TurboQuant (K2/V2)"; with the single global value rotation R_m = H for every modality it is the
 * whole baseline). Not combined with the fp16 residual.
 *
 * Bit-width ladder (dims.key_bits, dims.value_bits in 2..4; the K3/V2 row of Tab. 3 and the
 * K2V2 / K3V3 / K4V4 columns of Tab. 5): keys of the method take the uniform 2^b-level grid of
 * their window's range (step = (max - min) / (2^b - 1), code = clamp(rint(fl(fl(z - m16)
 * fl(1 / step16))), 0, 2^b - 1)); TurboQuant keys and all values take the 2^b-level Lloyd-Max
 * codebook (code = #{k : x > tau_k}). Layout: a token's 128 codes as a little-endian bit stream,
 * channel c at bits [b c, b c + b) of the token's 16 b bytes:
 *   k_codes  u8 [B][H][cap][16 key_bits]      v_codes  u8 [B][H][cap][16 value_bits]
 *   k_norm, v_norm, k_min, k_step (fp16 metadata; absent for TurboQuant keys) and modality as above;
 *   k_stage as above for the method's keys (none for TurboQuant keys, whose codes are per token);
 *   no k_mx or residual rings. okvq_append fills it (three launches: keys, values, lengths), or
 *   okvq_quantize_keys / okvq_quantize_keys_tq / okvq_quantize_values do (values in either mode;
 *   only slots below a length are written; the modality map is the caller's copy; no stage, so a
 *   cache to be appended to is filled by append from length 0); okvq_decode_attention reads it.
 *   Storage per token and KV head: 16 (key_bits + value_bits) + 4 bytes, + 16 with fp16 metadata
 *   (TurboQuant K3/V2: 84 bytes = 2.625 bits per element).
 *
 * fp16 residual of the captioning protocol (dims.residual = OKVQ_RESIDUAL_TOKENS, Sec. 3.1: keys
 * quantized every 128 tokens in groups of 32, values kept in a 128-token fp16 window before they
 * are quantized). Two more buffers hold the raw rows of the last 128 tokens:
 *   k_res    f16 [B][H][128][128]     key of token i in row i % 128
 *   v_res    f16 [B][H][128][128]     value of token i in row i % 128
 * Append still writes codes for every token (a window's key codes do not depend on when it is
 * quantized, value codes are per token); decode at length L reads key i quantized if
 * i < 128 floor(L / 128), else from k_res, and value i quantized if i < L - 128, else from v_res.
 */
#ifndef OKVQ_H
#define OKVQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t okvq_status;
enum {
  OKVQ_OK = 0,
  OKVQ_ERR_INVALID_ARGUMENT = -1, /* null / misaligned pointer, bad size or length           */
  OKVQ_ERR_UNSUPPORTED = -2,      /* head_dim != 128, window != 32, group size outside 1..8  */
  OKVQ_ERR_CAPACITY = -3,         /* a length (or length + appended tokens) exceeds capacity */
  OKVQ_ERR_WORKSPACE = -4,        /* decode workspace missing or too small                   */
  OKVQ_ERR_HIP = -5               /* a HIP launch failed                                     */
};

enum { OKVQ_MOD_AUDIO = 0, OKVQ_MOD_VIDEO = 1, OKVQ_MOD_TEXT = 2, OKVQ_NUM_MODALITIES = 3 };

/* flags */
enum {
  OKVQ_VALUE_EXACT = 1u << 0,    /* value rotation as a sequential fp32 dot product (bit-exact codes) */
  /* One value rotation for every token: the first table of v_rot (R_0) rotates the values of all
   * modalities, as in TurboQuant's single randomized rotation (Sec. 2.1, Eq. 2 and Eq. 3; the
   * TurboQuant rows of Tab. 3), instead of the per-modality R_m of Eq. 6. Accepted by
   * okvq_quantize_values, okvq_append and the decode calls of the 2-bit layout (the bit-width
   * ladder returns OKVQ_ERR_UNSUPPORTED). The modality map is still stored. A cache appended with
   * the flag must be decoded with it (decode then keeps one accumulator and un-rotates once with
   * R_0); codes and decode equal those of the per-modality path called with v_rot = {R_0, R_0, R_0}. */
  OKVQ_GLOBAL_ROTATION = 1u << 1
};

/* okvq_dims.key_meta: storage of the per-window key minimum and step */
enum {
  OKVQ_KEY_META_FP16 = 0,      /* fp16 k_min, k_step (84 bytes per token per KV head)        */
  OKVQ_KEY_META_MXFP4 = 1,     /* MXFP4 records in k_mx (72.25 bytes per token per KV head) */
  OKVQ_KEY_META_TURBOQUANT = 2 /* TurboQuant keys, the paper's baseline: no window metadata
                                  (68 bytes per token per KV head)                          */
};

/* okvq_dims.residual: 0 (every token read quantized) or the fp16 window of the captioning
 * protocol (Sec. 3.1) */
#define OKVQ_RESIDUAL_TOKENS 128

/* bytes of the prepared rotation tables (okvq_cache.v_rot16, okvq_prepare_rotation) */
#define OKVQ_ROTATION_TABLE_BYTES 294912

/* which_buffer for okvq_buffer_bytes */
enum {
  OKVQ_BUF_K_CODES = 0, OKVQ_BUF_V_CODES, OKVQ_BUF_K_NORM, OKVQ_BUF_V_NORM, OKVQ_BUF_K_MIN,
  OKVQ_BUF_K_STEP, OKVQ_BUF_MODALITY, OKVQ_BUF_K_STAGE, OKVQ_BUF_SEQ_LENS, OKVQ_BUF_K_MX, OKVQ_BUF_K_RES,
  OKVQ_BUF_V_RES, OKVQ_NUM_BUFFERS
};

typedef struct {
  int32_t batch;        /* B                                        */
  int32_t num_kv_heads; /* H                                        */
  int32_t num_q_heads;  /* Hq, a multiple of H, Hq / H <= 8         */
  int32_t head_dim;     /* must be 128                              */
  int32_t window;       /* key group size, must be 32 (Sec. 3.1)    */
  int32_t capacity;     /* token slots per sequence, multiple of 32 */
  int32_t key_meta;     /* OKVQ_KEY_META_*                          */
  int32_t residual;     /* 0 or OKVQ_RESIDUAL_TOKENS (fp16 window)  */
  int32_t key_bits;     /* 0: the 2-bit layout above; 2..4: the bit-width ladder layout below */
  int32_t value_bits;   /* 0, or 2..4 (both 0 or both set)          */
} okvq_dims;

typedef struct {               /* all pointers are device memory, laid out as above; k_min and
                                  k_step are used with fp16 metadata (else may be NULL), k_mx
                                  with MXFP4 metadata (else may be NULL) */
  okvq_dims dims;
  uint8_t* k_codes;
  uint8_t* v_codes;
  uint16_t* k_norm;
  uint16_t* v_norm;
  uint16_t* k_min;
  uint16_t* k_step;
  uint8_t* modality;
  uint16_t* k_stage;
  int32_t* seq_lens;
  const int8_t* key_signs;     /* [128] +1 / -1: H = Had diag(s) / sqrt(128) (Eq. 2)        */
  const float* v_rot;          /* [3][128][128] fp32 row-major R_m, z = R_m u (Eq. 6)       */
  const uint16_t* v_rot16;     /* OKVQ_ROTATION_TABLE_BYTES written by okvq_prepare_rotation
                                  from v_rot: the inverse rotation that decode applies once per
                                  modality (Sec. 2.3), then the forward rotation of append in
                                  the operand layout of its matrix-core kernel              */
  uint8_t* k_mx;               /* [B][H][cap/32][136] MXFP4 key metadata records            */
  uint16_t* k_res;             /* [B][H][128][128] fp16 keys of the last 128 tokens (residual
                                  mode, else may be NULL)                                     */
  uint16_t* v_res;             /* [B][H][128][128] fp16 values of the last 128 tokens        */
} okvq_cache;

/* Library version (major * 10000 + minor * 100 + patch). */
int32_t okvq_version(void);

/* Human-readable name of a status code (static string). */
const char* okvq_status_string(okvq_status status);

/* Bytes of one cache buffer for `dims` (0 for an unknown buffer, invalid dims, or a buffer the
 * metadata format of dims does not use: k_min / k_step unless fp16, k_mx unless MXFP4, k_res / v_res
 * without the residual). */
size_t okvq_buffer_bytes(const okvq_dims* dims, int32_t which_buffer);

/* Fixed Gaussian codebook of Eq. 3 as used by the kernels: the 4 levels and 3 decision
 * thresholds of the Lloyd-Max quantizer of N(0, 1/128), computed by the library on the host.
 * levels: host float[4]; thresholds: host float[3]. */
okvq_status okvq_codebook(float* levels, float* thresholds);

/* The b-bit codebook (b = bits = 2, 3, 4) of the bit-width ladder: the 2^b levels and 2^b - 1
 * thresholds of the Lloyd-Max quantizer of N(0, 1/128). levels: host float[2^b]; thresholds: host
 * float[2^b - 1]. OKVQ_ERR_INVALID_ARGUMENT for another width or a NULL pointer. */
okvq_status okvq_codebook_bits(int32_t bits, float* levels, float* thresholds);

/* Quantize keys (Eq. 2 then Eq. 4) of a dense block into cache-layout buffers.
 *   k          device f16 [B][H][n_tokens][128]; token i of sequence b is valid if i < lens_host[b]
 *   lens_host  host i32 [B], 0 <= lens_host[b] <= min(n_tokens, capacity)
 *   key_signs  device i8 [128]
 *   outputs    device k_codes, k_min, k_step, k_norm in the cache layout of dims->capacity;
 *              windows are aligned to token 0; a partial last window takes its min/step over
 *              its valid tokens; its padded slots get code 0 and norm 0. Nothing beyond the
 *              last window of each sequence is written.
 * Bit-exact contract: norms, min, step and codes equal the documented fp32 operation order.
 * dims->key_meta must be OKVQ_KEY_META_FP16 (else OKVQ_ERR_INVALID_ARGUMENT). */
okvq_status okvq_quantize_keys(const okvq_dims* dims, const uint16_t* k, int32_t n_tokens,
                               const int32_t* lens_host, const int8_t* key_signs, uint8_t* k_codes,
                               uint16_t* k_min, uint16_t* k_step, uint16_t* k_norm, void* stream);

/* okvq_quantize_keys with MXFP4 window metadata (Sec. 3.1: the paper's default storage of the
 * Eq. 4 minimum and scale): the same arguments, with k_mx (device u8 [B][H][cap/32][136], the
 * record layout above) in place of k_min and k_step. dims->key_meta must be
 * OKVQ_KEY_META_MXFP4. Bit-exact contract: norms, records and codes equal the documented fp32
 * operation order followed by the MXFP4 conversion. */
okvq_status okvq_quantize_keys_mx(const okvq_dims* dims, const uint16_t* k, int32_t n_tokens,
                                  const int32_t* lens_host, const int8_t* key_signs, uint8_t* k_codes,
                                  uint8_t* k_mx, uint16_t* k_norm, void* stream);

/* okvq_quantize_keys for TurboQuant keys (Eq. 2, Eq. 3; the layout above): the same arguments
 * without window metadata. dims->key_meta must be OKVQ_KEY_META_TURBOQUANT. Bit-exact contract:
 * norms and codes equal the documented fp32 order followed by the threshold decisions. */
okvq_status okvq_quantize_keys_tq(const okvq_dims* dims, const uint16_t* k, int32_t n_tokens,
                                  const int32_t* lens_host, const int8_t* key_signs, uint8_t* k_codes,
                                  uint16_t* k_norm, void* stream);

/* Quantize values (Eq. 6 with the codebook of Eq. 3) of a dense block into cache-layout buffers.
 *   v          device f16 [B][H][n_tokens][128]
 *   modality   device u8 [B][n_tokens] (0 audio, 1 video, 2 text)
 *   v_rot      device f32 [3][128][128], R_m row-major
 *   flags      OKVQ_VALUE_EXACT: y = R_m v as a sequential fp32 dot product (codes bit-exact with
 *              the documented order); otherwise MFMA with an fp16 hi/lo split of R_m and fp32
 *              accumulation (codes may differ from the exact order only where y lies within a
 *              small band around a decision threshold). Both layouts, both modes.
 *              OKVQ_GLOBAL_ROTATION: R_0 for every token (2-bit layout only).
 *   outputs    device v_codes, v_norm in the cache layout (whole 32-token windows are written;
 *              slots beyond a length get code 0 and norm 0). */
okvq_status okvq_quantize_values(const okvq_dims* dims, const uint16_t* v, const uint8_t* modality,
                                 int32_t n_tokens, const int32_t* lens_host, const float* v_rot,
                                 uint32_t flags, uint8_t* v_codes, uint16_t* v_norm, void* stream);

/* Append n_new[b] tokens to every sequence of a cache (prefill is an append to an empty cache).
 *   lens_host  host i32 [B] current lengths (equal to cache->seq_lens on the device)
 *   k_new,v_new device f16 [B][H][n_max][128]; mod_new device u8 [B][n_max]
 *   n_new_host host i32 [B], n_new_dev the same values in device memory, 0 <= n_new <= n_max
 * The open key window is re-quantized from the staged raw keys plus the new ones, so any
 * chunking of a sequence yields the same cache bytes as one quantization of the whole sequence.
 * cache->seq_lens[b] is advanced by n_new[b] on the device. Fails with OKVQ_ERR_CAPACITY if
 * lens_host[b] + n_new_host[b] > capacity. The MFMA-mode values read the forward rotation from
 * cache->v_rot16 (okvq_prepare_rotation); OKVQ_VALUE_EXACT reads cache->v_rot. The key window
 * metadata is written in the format of cache->dims.key_meta (k_min / k_step, or k_mx). With the
 * residual, the raw key and value rows of the new tokens among the last 128 of each sequence are
 * also written to k_res and v_res (one more launch, before the codec). flags: OKVQ_VALUE_EXACT,
 * OKVQ_GLOBAL_ROTATION (R_0 for every token; the 2-bit layout only). The bit-width ladder layout
 * (Tab. 5 K3V3 / K4V4, Tab. 3 K3/V2) is appended the same way, with its b-bit codecs: the method's
 * keys re-quantize the open window from the stage, TurboQuant keys and values code the new tokens;
 * chunked and one-shot appends give the same bytes there too. */
okvq_status okvq_append(const okvq_cache* cache, const int32_t* lens_host, const uint16_t* k_new,
                        const uint16_t* v_new, const uint8_t* mod_new, const int32_t* n_new_host,
                        const int32_t* n_new_dev, int32_t n_max, uint32_t flags, void* stream);

/* okvq_append that also times its codec: events[0] and events[1] (hipEvent_t handles created by the
 * caller) are recorded at the start and end of the execution of the one launch that codes the keys
 * and values (the window-parallel launch of a small append, or the fused codec launch), so that
 * hipEventElapsedTime of the pair is that kernel's duration without the host's submission. The cache
 * bytes are those of okvq_append. OKVQ_ERR_INVALID_ARGUMENT for a null events array or handle;
 * OKVQ_ERR_UNSUPPORTED where the append takes other launches too or none (the bit-width ladder,
 * OKVQ_VALUE_EXACT, the fp16 residual on the fused-codec path, more than 256 sequences, no new
 * token), before anything is launched. */
okvq_status okvq_append_timed(const okvq_cache* cache, const int32_t* lens_host, const uint16_t* k_new,
                              const uint16_t* v_new, const uint8_t* mod_new, const int32_t* n_new_host,
                              const int32_t* n_new_dev, int32_t n_max, uint32_t flags, void* stream,
                              void* const* events);

/* Status word of a cache (seq_lens[B + 1]): 0, or 1 once an append's value codec stopped waiting for
 * its partner waves after a bounded number of polls and went on with incomplete tables (that
 * append's value codes may be wrong; addresses stay in bounds). The one call of the library that
 * synchronizes: it copies the word to the host after the work already on `stream`.
 *   status  host i32 output
 * OKVQ_ERR_HIP if the copy or the synchronization fails. */
okvq_status okvq_cache_status(const okvq_cache* cache, int32_t* status, void* stream);

/* Rotation tables of a layer, prepared once from v_rot (fp16, round to nearest even):
 *   bytes [0, 98304)       inverse rotation for decode (Sec. 2.3: applied once per modality after
 *                          aggregation): [128][3][128], element (c, m, k) = fp16(R_m[k][c]);
 *   bytes [98304, 294912)  forward rotation for the MFMA-mode values of append (Eq. 6): 192
 *                          blocks of 64 x 8 fp16, block ((m 8 + nb) 4 + kk) 2 + part, row l,
 *                          element e = part(R_m[16 nb + l % 16][32 kk + 8 (l / 16) + e]) with
 *                          part 0 = fp16(R), part 1 = fp16(R - fp16(R)) (fp32 difference).
 *   v_rot    device f32 [3][128][128]
 *   v_rot16  device, OKVQ_ROTATION_TABLE_BYTES bytes: the okvq_cache.v_rot16 of every cache
 *            that uses v_rot */
okvq_status okvq_prepare_rotation(const float* v_rot, uint16_t* v_rot16, void* stream);

/* Device workspace bytes needed by okvq_decode_attention for sequences up to max_seq_len (the
 * partial results of the split-K launch; no initial contents are needed). */
size_t okvq_decode_workspace_bytes(const okvq_dims* dims, int32_t max_seq_len);

/* One decode step: attention of one query per head over the packed cache (Eq. 1): a split-K
 * launch over windows and a log-sum-exp merge launch.
 *   lens_host  host i32 [B] (plans the split-K launch; the kernels read cache->seq_lens)
 *   q          device f16 [B][Hq][128]
 *   sm_scale   softmax scale, normally 1/sqrt(128)
 *   out        device f32 [B][Hq][128]
 *   workspace  device, at least okvq_decode_workspace_bytes(dims, max(lens_host)) bytes
 * Needs cache->v_rot16 (okvq_prepare_rotation); reads the key window metadata in the format of
 * cache->dims.key_meta. With the residual (captioning protocol, Sec. 3.1) the split-K launch covers
 * the tokens below L - 128, and the merge launch also attends the last min(L, 128) tokens -- keys
 * below 128 floor(L / 128) dequantized, the others and all values in fp16 from k_res / v_res --
 * and merges them in. A sequence of length 0 yields zeros. fp32
 * accumulation; the result matches float64 attention over the dequantized cache within 2e-3 of
 * the output norm. flags: 0, or OKVQ_GLOBAL_ROTATION for a cache appended with it (one value
 * accumulator, one un-rotation with R_0; 2-bit layout only). */
okvq_status okvq_decode_attention(const okvq_cache* cache, const int32_t* lens_host, const uint16_t* q,
                                  float sm_scale, uint32_t flags, float* out, void* workspace,
                                  size_t workspace_bytes, void* stream);

/* okvq_decode_attention for callers that cannot allocate (code under HIP graph capture, tight
 * serving loops, harnesses that forbid allocation): the same decode, with the split records in a
 * static device array of OKVQ_NOALLOC_SCRATCH_BYTES on each GPU (held until the process ends)
 * instead of a caller workspace. No hipMalloc, hipFree or other allocation happens in the call;
 * its first call on a GPU looks up that GPU's array address once. Every call on a GPU shares the
 * array: calls that overlap on one GPU (other streams, other threads) race and give wrong results.
 * The array needs no initial contents.
 * OKVQ_ERR_WORKSPACE if this call's split records (sequences x KV heads x splits of its plan,
 * 4224 bytes each; about 256 + B H records by default) exceed the array. */
#define OKVQ_NOALLOC_SCRATCH_BYTES (4u << 20)
okvq_status okvq_decode_attention_noalloc(const okvq_cache* cache, const int32_t* lens_host, const uint16_t* q,
                                          float sm_scale, uint32_t flags, float* out, void* stream);

/* okvq_decode_attention that also times its two launches: events[0] and events[1] are recorded
 * at the start and end of the split-K kernel's execution, events[2] and events[3] at those of
 * the merge kernel (hipEvent_t handles created by the caller; hipEventElapsedTime of a pair is
 * that kernel's duration). */
okvq_status okvq_decode_attention_timed(const okvq_cache* cache, const int32_t* lens_host, const uint16_t* q,
                                        float sm_scale, uint32_t flags, float* out, void* workspace,
                                        size_t workspace_bytes, void* stream, void* const* events);

/* ---- Modality-aware value-rotation calibration (Sec. 2.3, Eq. 5 and Eq. 6) ----------------------
 * Eq. 5 weights every value by how strongly it contributes to the attention output, w_j =
 * sum_i alpha_{i,j}^2, forms C_m = sum_{j of modality m} w_j v_j^T v_j, and takes U_m from the
 * eigendecomposition of C_m; Eq. 6 then rotates values by R_m = H U_m^T. The three calls below
 * produce the okvq_cache.v_rot of a layer from calibration activations: the weights and the
 * covariance on the device, the eigendecomposition and R_m on the host. Readings: alpha is the
 * causal softmax attention of every calibration position i over the tokens j <= i, summed over
 * every query head that reads the KV head; v_j are the raw fp16 values; one C_m per layer (summed
 * over its sequences and KV heads); H is the layer's randomized Hadamard (the key signs). */

/* Device workspace bytes for okvq_calibration_weights and okvq_value_covariance at n_tokens
 * positions per sequence (0 for invalid dims). No initial contents are needed. */
size_t okvq_calibration_workspace_bytes(const okvq_dims* dims, int32_t n_tokens);

/* Attention weights of Eq. 5.
 *   q          device f16 [B][Hq][n_tokens][128]: the calibration query of every position
 *   k          device f16 [B][H][n_tokens][128]
 *   lens_host  host i32 [B], 0 <= lens_host[b] <= n_tokens: positions i < lens_host[b] are queries
 *              and keys
 *   sm_scale   softmax scale, normally 1/sqrt(128)
 *   w          device f32 [B][H][n_tokens] output: w[b][h][t] = sum over the query heads j of KV
 *              head h (GQA, j / G = h) and the positions i in [t, lens) of alpha_{i,t}^2; zero for
 *              t >= lens_host[b]
 * Scores on the matrix cores (fp16 operands, fp32 accumulation), softmax statistics and sums in fp32
 * (two launches: row statistics, then column sums). */
okvq_status okvq_calibration_weights(const okvq_dims* dims, const uint16_t* q, const uint16_t* k, int32_t n_tokens,
                                     const int32_t* lens_host, float sm_scale, float* w, void* workspace,
                                     size_t workspace_bytes, void* stream);

/* Weighted value covariance of Eq. 5.
 *   v          device f16 [B][H][n_tokens][128]; modality device u8 [B][n_tokens] (0..2)
 *   w          device f32 [B][H][n_tokens] (okvq_calibration_weights)
 *   cov        device f32 [3][128][128] output: C_m = sum over sequences, KV heads and tokens
 *              t < lens_host[b] of modality m of w_t v_t v_t^T (overwritten, not accumulated)
 * Products on the matrix cores with w v split into fp16 hi + lo parts (about 2^-22 relative per
 * term), fp32 accumulation; per-chunk partials are summed in a fixed order (deterministic). */
okvq_status okvq_value_covariance(const okvq_dims* dims, const uint16_t* v, const uint8_t* modality, const float* w,
                                  int32_t n_tokens, const int32_t* lens_host, float* cov, void* workspace,
                                  size_t workspace_bytes, void* stream);

/* Rotations from the covariances (Eq. 5 eigendecomposition, Eq. 6), on the host, in double
 * precision (cyclic Jacobi).
 *   cov          host f32 [3][128][128] (its symmetric part is used)
 *   signs        host i8 [128], +1 / -1: H = Had diag(s) / sqrt(128), Had the Sylvester matrix
 *   rot          host f32 [3][128][128] output, R_m = H U_m^T row-major (the okvq_cache.v_rot layout)
 *   eigenvalues  host f64 [3][128] output in descending order, or NULL
 * U_m holds the eigenvectors as columns in descending eigenvalue order, each with its largest
 * component positive (the first one on ties); eigenvectors of equal eigenvalues are not unique. A
 * modality with C_m = 0 (absent from the calibration data) gets U_m = I, i.e. R_m = H. */
okvq_status okvq_rotation_from_covariance(const float* cov, const int8_t* signs, float* rot, double* eigenvalues);

/* ---- Dense fp16 decode attention: the comparison baseline ------------------------------------
 * Eq. 1 over an unquantized fp16 KV cache (no codes, norms, rotations or modality map): the
 * attention that the packed cache replaces, computed the same way (split-K launch, every query head
 * of a KV head served from one read of K and V, scores and PV on the matrix cores with fp16
 * operands and fp32 accumulation, a log-sum-exp merge launch). */

/* Device workspace bytes needed by okvq_decode_attention_dense for sequences up to max_seq_len
 * (0 for invalid dims or a negative length). No initial contents are needed. */
size_t okvq_dense_workspace_bytes(const okvq_dims* dims, int32_t max_seq_len);

/* One dense decode step.
 *   dims       batch, num_kv_heads, num_q_heads (G = Hq / H <= 8), head_dim 128, and capacity =
 *              the token stride of k and v (a multiple of 32); window must be 32, key_meta and
 *              residual are not used
 *   k, v       device f16 [B][H][capacity][128]: rows of token i < seq_lens[b] are read
 *   seq_lens   device i32 [B]: the lengths the kernels use
 *   lens_host  host i32 [B], 0 <= lens_host[b] <= capacity: plans the launch (equal to seq_lens)
 *   q          device f16 [B][Hq][128]; query head j reads KV head j / G
 *   sm_scale   softmax scale, normally 1/sqrt(128)
 *   out        device f32 [B][Hq][128]; a sequence of length 0 yields zeros
 *   workspace  device, at least okvq_dense_workspace_bytes(dims, max(lens_host)) bytes
 *   events     NULL, or four hipEvent_t handles recorded at the start and end of the split-K
 *              kernel's and of the merge kernel's execution
 * Every pointer must be 16-byte aligned; arguments are checked on the host before anything is
 * enqueued. The result matches float64 attention over the same fp16 K and V within 2e-3 of the
 * output norm. */
okvq_status okvq_decode_attention_dense(const okvq_dims* dims, const uint16_t* k, const uint16_t* v,
                                        const int32_t* seq_lens, const int32_t* lens_host, const uint16_t* q,
                                        float sm_scale, float* out, void* workspace, size_t workspace_bytes,
                                        void* stream, void* const* events);

#ifdef __cplusplus
}
#endif

#endif /* OKVQ_H */
