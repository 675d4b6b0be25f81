// C ABI of the okvq library: argument validation, launch planning and the fixed codebook.
// Declarations and contracts: include/okvq.h.
#include <algorithm>
#include <cstdlib>
#include <cmath>
#include <cstring>
#include <mutex>
#include <numeric>
#include <vector>

#include "okvq.h"
#include "launch.hpp"

using namespace okvq;

// Split records of okvq_decode_attention_noalloc: one array per GPU, held until the process ends.
// In host code `scratch` names a host-side stand-in; its device address on each GPU comes from
// hipGetSymbolAddress (scratch_address below) and is the only form passed to kernels.
static __device__ __align__(256) float scratch[OKVQ_NOALLOC_SCRATCH_BYTES / sizeof(float)];

namespace {

constexpr int kMaxDevices = 64;

// Device address of `scratch` on the current device, looked up once per device (with that device
// current) and kept; later calls on the device reuse it.
okvq_status scratch_address(void** out) {
  static std::mutex mu;
  static void* addr[kMaxDevices] = {};
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return OKVQ_ERR_HIP;
  if (dev < 0 || dev >= kMaxDevices) return OKVQ_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return OKVQ_ERR_HIP;
    addr[dev] = p;
  }
  *out = addr[dev];
  return OKVQ_OK;
}

constexpr int32_t kVersion = 600;  // 0.6.0: bit-width ladder (b-bit keys and values)

// ---- fixed Gaussian codebook (Sec. 2.1, Eq. 3): Lloyd-Max quantizer of N(0, 1), 4 levels ----
double phi(double x) { return std::isinf(x) ? 0.0 : std::exp(-0.5 * x * x) / std::sqrt(2.0 * M_PI); }
double cdf(double x) {
  if (std::isinf(x)) return x < 0 ? 0.0 : 1.0;
  return 0.5 * std::erfc(-x / std::sqrt(2.0));
}

struct Codebook {
  int levels;           // 2^b
  float level[16];      // levels of N(0, 1/128), fp32
  float thr[15];        // decision thresholds (midpoints), fp32
  uint16_t level16[16]; // fp16 levels used by the decode kernels
};

Codebook make_codebook(int L) {
  // Lloyd iteration: thresholds are midpoints of neighbouring levels, levels are the centroids
  // of their cells (closed form for a Gaussian density).
  double c[16];
  for (int i = 0; i < L; ++i) c[i] = -(L - 1) / 2.0 + i;
  for (int it = 0; it < 100000; ++it) {
    double e[17];
    e[0] = -INFINITY;
    e[L] = INFINITY;
    for (int i = 0; i + 1 < L; ++i) e[i + 1] = (c[i] + c[i + 1]) / 2;
    double delta = 0.0;
    for (int i = 0; i < L; ++i) {
      const double n = (phi(e[i]) - phi(e[i + 1])) / (cdf(e[i + 1]) - cdf(e[i]));
      delta = std::fmax(delta, std::fabs(n - c[i]));
      c[i] = n;
    }
    if (delta < 1e-15) break;
  }
  double s[16];
  for (int i = 0; i < L; ++i) s[i] = (c[i] - c[L - 1 - i]) / 2;  // exact symmetry of the density
  const double sc = 1.0 / std::sqrt(128.0);
  Codebook cb{};
  cb.levels = L;
  for (int i = 0; i < L; ++i) {
    cb.level[i] = (float)(s[i] * sc);
    cb.level16[i] = __builtin_bit_cast(uint16_t, (_Float16)(s[i] * sc));
  }
  for (int i = 0; i + 1 < L; ++i) cb.thr[i] = (float)(((s[i] + s[i + 1]) / 2) * sc);
  return cb;
}

// the b-bit codebook (b = 2, 3, 4)
const Codebook& codebook(int bits = 2) {
  static const Codebook cb2 = make_codebook(4), cb3 = make_codebook(8), cb4 = make_codebook(16);
  return bits == 3 ? cb3 : bits == 4 ? cb4 : cb2;
}

Thresholds thresholds() {
  const Codebook& cb = codebook();
  return Thresholds{cb.thr[0], cb.thr[1], cb.thr[2]};
}

bool aligned16(const void* p) { return p != nullptr && (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

okvq_status check_dims(const okvq_dims* d) {
  if (!d) return OKVQ_ERR_INVALID_ARGUMENT;
  if (d->head_dim != 128 || d->window != 32) return OKVQ_ERR_UNSUPPORTED;
  if (d->batch < 1 || d->num_kv_heads < 1 || d->num_q_heads < 1) return OKVQ_ERR_INVALID_ARGUMENT;
  if (d->num_q_heads % d->num_kv_heads != 0) return OKVQ_ERR_INVALID_ARGUMENT;
  if (d->num_q_heads / d->num_kv_heads > 8) return OKVQ_ERR_UNSUPPORTED;
  if (d->capacity < 32 || d->capacity % 32 != 0) return OKVQ_ERR_INVALID_ARGUMENT;
  if (d->batch > 65535 || d->num_kv_heads > 65535) return OKVQ_ERR_UNSUPPORTED;
  if (d->key_meta != OKVQ_KEY_META_FP16 && d->key_meta != OKVQ_KEY_META_MXFP4 && d->key_meta != OKVQ_KEY_META_TURBOQUANT)
    return OKVQ_ERR_INVALID_ARGUMENT;
  if (d->residual != 0 && d->residual != OKVQ_RESIDUAL_TOKENS) return OKVQ_ERR_INVALID_ARGUMENT;
  if (d->residual != 0 && d->key_meta == OKVQ_KEY_META_TURBOQUANT) return OKVQ_ERR_UNSUPPORTED;
  // bit-width ladder: both widths 0 (the 2-bit layout) or both in 2..4 (the bit-stream layout)
  if (d->key_bits != 0 || d->value_bits != 0) {
    if (d->key_bits < 2 || d->key_bits > 4 || d->value_bits < 2 || d->value_bits > 4) return OKVQ_ERR_INVALID_ARGUMENT;
    if (d->key_meta == OKVQ_KEY_META_MXFP4 || d->residual != 0) return OKVQ_ERR_UNSUPPORTED;
  }
  return OKVQ_OK;
}

bool is_ladder(const okvq_dims* d) { return d->key_bits != 0; }

bool is_mx(const okvq_dims* d) { return d->key_meta == OKVQ_KEY_META_MXFP4; }
bool is_fp16(const okvq_dims* d) { return d->key_meta == OKVQ_KEY_META_FP16; }
int meta_mode(const okvq_dims* d) {
  return d->key_meta == OKVQ_KEY_META_MXFP4 ? kMetaMx : d->key_meta == OKVQ_KEY_META_TURBOQUANT ? kMetaTq : kMetaFp16;
}

okvq_status check_cache(const okvq_cache* c) {
  if (!c) return OKVQ_ERR_INVALID_ARGUMENT;
  okvq_status st = check_dims(&c->dims);
  if (st != OKVQ_OK) return st;
  const void* ptrs[] = {c->k_codes, c->v_codes, c->k_norm,  c->v_norm, c->modality,
                        c->seq_lens, c->key_signs, c->v_rot, c->v_rot16};
  for (const void* p : ptrs)
    if (!aligned16(p)) return OKVQ_ERR_INVALID_ARGUMENT;
  if ((!is_ladder(&c->dims) || is_fp16(&c->dims)) && !aligned16(c->k_stage)) return OKVQ_ERR_INVALID_ARGUMENT;
  if (is_mx(&c->dims) && !aligned16(c->k_mx)) return OKVQ_ERR_INVALID_ARGUMENT;
  if (is_fp16(&c->dims) && (!aligned16(c->k_min) || !aligned16(c->k_step))) return OKVQ_ERR_INVALID_ARGUMENT;
  if (c->dims.residual && (!aligned16(c->k_res) || !aligned16(c->v_res))) return OKVQ_ERR_INVALID_ARGUMENT;
  return OKVQ_OK;
}

CacheView view(const okvq_cache* c) {
  CacheView v;
  v.B = c->dims.batch;
  v.H = c->dims.num_kv_heads;
  v.Hq = c->dims.num_q_heads;
  v.cap = c->dims.capacity;
  v.k_codes = c->k_codes;
  v.v_codes = c->v_codes;
  v.k_norm = c->k_norm;
  v.v_norm = c->v_norm;
  v.k_min = c->k_min;
  v.k_step = c->k_step;
  v.k_mx = is_mx(&c->dims) ? c->k_mx : nullptr;
  v.key_meta = meta_mode(&c->dims);
  v.modality = c->modality;
  v.k_stage = c->k_stage;
  v.seq_lens = c->seq_lens;
  v.signs = c->key_signs;
  v.rot = c->v_rot;
  v.rot16t = c->v_rot16;
  v.residual = c->dims.residual;
  v.k_res = c->dims.residual ? c->k_res : nullptr;
  v.v_res = c->dims.residual ? c->v_res : nullptr;
  v.key_bits = c->dims.key_bits;
  v.value_bits = c->dims.value_bits;
  return v;
}

okvq_status hip_status(hipError_t e) { return e == hipSuccess ? OKVQ_OK : OKVQ_ERR_HIP; }

// ---- host eigensolver of the calibration (Eq. 5): cyclic Jacobi rotations on a symmetric
// matrix in double precision. Each rotation in the (p, q) plane is chosen to zero a[p][q]; sweeps
// repeat until the off-diagonal mass is negligible. a (n x n, row-major) is destroyed; the columns of
// u are the eigenvectors, d the eigenvalues. ----
void jacobi_eigen(std::vector<double>& a, std::vector<double>& u, std::vector<double>& d, int n) {
  u.assign((size_t)n * n, 0.0);
  for (int i = 0; i < n; ++i) u[(size_t)i * n + i] = 1.0;
  double frob = 0.0;
  for (double x : a) frob += x * x;
  for (int sweep = 0; sweep < 100; ++sweep) {
    double off = 0.0;
    for (int p = 0; p < n; ++p)
      for (int q = p + 1; q < n; ++q) off += a[(size_t)p * n + q] * a[(size_t)p * n + q];
    if (off <= 1e-32 * frob || off == 0.0) break;
    for (int p = 0; p < n - 1; ++p) {
      for (int q = p + 1; q < n; ++q) {
        const double apq = a[(size_t)p * n + q];
        if (apq == 0.0) continue;
        const double app = a[(size_t)p * n + p], aqq = a[(size_t)q * n + q];
        // t = tan(phi) of the rotation that zeroes a[p][q]: the smaller root of t^2 + 2 theta t - 1 = 0
        const double theta = (aqq - app) / (2.0 * apq);
        const double t = (theta >= 0.0 ? 1.0 : -1.0) / (std::fabs(theta) + std::sqrt(theta * theta + 1.0));
        const double c = 1.0 / std::sqrt(t * t + 1.0), s = t * c;
        for (int k = 0; k < n; ++k) {  // columns p, q
          const double akp = a[(size_t)k * n + p], akq = a[(size_t)k * n + q];
          a[(size_t)k * n + p] = c * akp - s * akq;
          a[(size_t)k * n + q] = s * akp + c * akq;
        }
        for (int k = 0; k < n; ++k) {  // rows p, q
          const double apk = a[(size_t)p * n + k], aqk = a[(size_t)q * n + k];
          a[(size_t)p * n + k] = c * apk - s * aqk;
          a[(size_t)q * n + k] = s * apk + c * aqk;
        }
        a[(size_t)p * n + q] = a[(size_t)q * n + p] = 0.0;
        for (int k = 0; k < n; ++k) {
          const double ukp = u[(size_t)k * n + p], ukq = u[(size_t)k * n + q];
          u[(size_t)k * n + p] = c * ukp - s * ukq;
          u[(size_t)k * n + q] = s * ukp + c * ukq;
        }
      }
    }
  }
  d.resize(n);
  for (int i = 0; i < n; ++i) d[i] = a[(size_t)i * n + i];
}

// Tiles of 256 tokens covering `span` tokens from each sequence's first open window.
// Appends take the window-parallel launch when they touch at most 2 key windows of a sequence (a
// generation step), or at most 64 windows and 2048 work-groups in all (a streamed chunk); longer
// spans take the tile launch, whose throughput is higher (32768-token prefill of 4 KV heads:
// 43 us against 103 us).
constexpr int kWindowPathMaxWindows = 64;
constexpr int64_t kWindowPathMaxGroups = 2048;

void plan_tiles(CodecArgs& a, int nb, int span) {
  a.ntx = (span + 255) / 256;
  a.ntiles = a.ntx * a.j.H * nb;
}

}  // namespace

extern "C" {

int32_t okvq_version(void) { return kVersion; }

const char* okvq_status_string(okvq_status s) {
  switch (s) {
    case OKVQ_OK: return "ok";
    case OKVQ_ERR_INVALID_ARGUMENT: return "invalid argument";
    case OKVQ_ERR_UNSUPPORTED: return "unsupported configuration";
    case OKVQ_ERR_CAPACITY: return "capacity exceeded";
    case OKVQ_ERR_WORKSPACE: return "workspace missing or too small";
    case OKVQ_ERR_HIP: return "HIP launch failed";
    default: return "unknown status";
  }
}

size_t okvq_buffer_bytes(const okvq_dims* d, int32_t which) {
  if (check_dims(d) != OKVQ_OK) return 0;
  const size_t B = d->batch, H = d->num_kv_heads, cap = d->capacity, D = d->head_dim, W = d->window;
  if (is_ladder(d)) {  // bit-stream layout: no MXFP4 records or rings; a key stage for the method's keys
    switch (which) {
      case OKVQ_BUF_K_STAGE: return is_fp16(d) ? B * H * W * D * 2 : 0;
      case OKVQ_BUF_K_CODES: return B * H * cap * (D * d->key_bits / 8);
      case OKVQ_BUF_V_CODES: return B * H * cap * (D * d->value_bits / 8);
      case OKVQ_BUF_K_NORM:
      case OKVQ_BUF_V_NORM: return B * H * cap * 2;
      case OKVQ_BUF_K_MIN:
      case OKVQ_BUF_K_STEP: return is_fp16(d) ? B * H * (cap / W) * D * 2 : 0;
      case OKVQ_BUF_MODALITY: return B * cap;
      case OKVQ_BUF_SEQ_LENS: return B * 4 + 8;
      default: return 0;
    }
  }
  switch (which) {
    case OKVQ_BUF_K_CODES: return B * H * cap * (D / 4);
    case OKVQ_BUF_V_CODES: return B * H * cap * (D / 4);
    case OKVQ_BUF_K_NORM: return B * H * cap * 2;
    case OKVQ_BUF_V_NORM: return B * H * cap * 2;
    case OKVQ_BUF_K_MIN: return is_fp16(d) ? B * H * (cap / W) * D * 2 : 0;
    case OKVQ_BUF_K_STEP: return is_fp16(d) ? B * H * (cap / W) * D * 2 : 0;
    case OKVQ_BUF_K_MX: return is_mx(d) ? B * H * (cap / W) * kMxRecord : 0;
    case OKVQ_BUF_MODALITY: return B * cap;
    case OKVQ_BUF_K_STAGE: return B * H * W * D * 2;
    case OKVQ_BUF_SEQ_LENS: return B * 4 + 8;  // the lengths, append's work-group counter, the status word
    case OKVQ_BUF_K_RES:
    case OKVQ_BUF_V_RES: return d->residual ? B * H * OKVQ_RESIDUAL_TOKENS * D * 2 : 0;
    default: return 0;
  }
}

okvq_status okvq_codebook(float* levels, float* thresholds_out) {
  if (!levels || !thresholds_out) return OKVQ_ERR_INVALID_ARGUMENT;
  const Codebook& cb = codebook();
  std::memcpy(levels, cb.level, 4 * sizeof(float));
  std::memcpy(thresholds_out, cb.thr, 3 * sizeof(float));
  return OKVQ_OK;
}

okvq_status okvq_codebook_bits(int32_t bits, float* levels, float* thresholds_out) {
  if (!levels || !thresholds_out || bits < 2 || bits > 4) return OKVQ_ERR_INVALID_ARGUMENT;
  const Codebook& cb = codebook(bits);
  std::memcpy(levels, cb.level, cb.levels * sizeof(float));
  std::memcpy(thresholds_out, cb.thr, (cb.levels - 1) * sizeof(float));
  return OKVQ_OK;
}

static okvq_status quantize_keys_impl(const okvq_dims* dims, const uint16_t* k, int32_t n_tokens,
                                      const int32_t* lens_host, const int8_t* key_signs, uint8_t* k_codes,
                                      uint16_t* k_min, uint16_t* k_step, uint8_t* k_mx, uint16_t* k_norm,
                                      void* stream) {
  for (int b = 0; b < dims->batch; ++b) {
    if (lens_host[b] < 0 || lens_host[b] > n_tokens) return OKVQ_ERR_INVALID_ARGUMENT;
    if (lens_host[b] > dims->capacity) return OKVQ_ERR_CAPACITY;
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (is_ladder(dims)) {
    const Codebook& cb = codebook(dims->key_bits);
    for (int b0 = 0; b0 < dims->batch; b0 += kMaxLenArgs) {
      const int nb = std::min(kMaxLenArgs, dims->batch - b0);
      LadderKeyArgs a{};
      a.k = k;
      a.n_rows = n_tokens;
      a.H = dims->num_kv_heads;
      a.cap = dims->capacity;
      a.b0 = b0;
      int max_len = 0;
      for (int i = 0; i < nb; ++i) {
        a.lens.lens[i] = lens_host[b0 + i];
        max_len = std::max(max_len, lens_host[b0 + i]);
      }
      a.signs = key_signs;
      a.k_codes = k_codes;
      a.k_min = k_min;
      a.k_step = k_step;
      a.k_norm = k_norm;
      for (int i = 0; i + 1 < cb.levels; ++i) a.tau[i] = cb.thr[i];
      okvq_status st = hip_status(launch_ladder_keys(a, dims->key_bits, !is_fp16(dims), nb, max_len, s));
      if (st != OKVQ_OK) return st;
    }
    return OKVQ_OK;
  }
  for (int b0 = 0; b0 < dims->batch; b0 += kMaxLenArgs) {
    const int nb = std::min(kMaxLenArgs, dims->batch - b0);
    CodecArgs a{};
    a.j.src = k;
    a.j.n_rows = n_tokens;
    a.j.b0 = b0;
    a.j.H = dims->num_kv_heads;
    a.j.cap = dims->capacity;
    int max_len = 0;
    for (int i = 0; i < nb; ++i) {
      a.j.lens.lens[i] = lens_host[b0 + i];
      max_len = std::max(max_len, lens_host[b0 + i]);
    }
    plan_tiles(a, nb, max_len);
    a.signs = key_signs;
    a.k_codes = k_codes;
    a.k_min = k_min;
    a.k_step = k_step;
    a.k_mx = k_mx;
    a.k_norm = k_norm;
    a.key_meta = meta_mode(dims);
    a.th = thresholds();
    okvq_status st = hip_status(launch_codec(a, true, false, s));
    if (st != OKVQ_OK) return st;
  }
  return OKVQ_OK;
}

okvq_status okvq_quantize_keys(const okvq_dims* dims, const uint16_t* k, int32_t n_tokens, const int32_t* lens_host,
                               const int8_t* key_signs, uint8_t* k_codes, uint16_t* k_min, uint16_t* k_step,
                               uint16_t* k_norm, void* stream) {
  okvq_status st = check_dims(dims);
  if (st != OKVQ_OK) return st;
  if (n_tokens < 0 || !lens_host || !is_fp16(dims)) return OKVQ_ERR_INVALID_ARGUMENT;
  if (!aligned16(k) || !aligned16(key_signs) || !aligned16(k_codes) || !aligned16(k_min) || !aligned16(k_step) ||
      !aligned16(k_norm))
    return OKVQ_ERR_INVALID_ARGUMENT;
  return quantize_keys_impl(dims, k, n_tokens, lens_host, key_signs, k_codes, k_min, k_step, nullptr, k_norm, stream);
}

okvq_status okvq_quantize_keys_mx(const okvq_dims* dims, const uint16_t* k, int32_t n_tokens,
                                  const int32_t* lens_host, const int8_t* key_signs, uint8_t* k_codes, uint8_t* k_mx,
                                  uint16_t* k_norm, void* stream) {
  okvq_status st = check_dims(dims);
  if (st != OKVQ_OK) return st;
  if (n_tokens < 0 || !lens_host || !is_mx(dims)) return OKVQ_ERR_INVALID_ARGUMENT;
  if (!aligned16(k) || !aligned16(key_signs) || !aligned16(k_codes) || !aligned16(k_mx) || !aligned16(k_norm))
    return OKVQ_ERR_INVALID_ARGUMENT;
  return quantize_keys_impl(dims, k, n_tokens, lens_host, key_signs, k_codes, nullptr, nullptr, k_mx, k_norm, stream);
}

okvq_status okvq_quantize_keys_tq(const okvq_dims* dims, const uint16_t* k, int32_t n_tokens,
                                  const int32_t* lens_host, const int8_t* key_signs, uint8_t* k_codes,
                                  uint16_t* k_norm, void* stream) {
  okvq_status st = check_dims(dims);
  if (st != OKVQ_OK) return st;
  if (n_tokens < 0 || !lens_host || dims->key_meta != OKVQ_KEY_META_TURBOQUANT) return OKVQ_ERR_INVALID_ARGUMENT;
  if (!aligned16(k) || !aligned16(key_signs) || !aligned16(k_codes) || !aligned16(k_norm))
    return OKVQ_ERR_INVALID_ARGUMENT;
  return quantize_keys_impl(dims, k, n_tokens, lens_host, key_signs, k_codes, nullptr, nullptr, nullptr, k_norm, stream);
}

okvq_status okvq_quantize_values(const okvq_dims* dims, const uint16_t* v, const uint8_t* modality, int32_t n_tokens,
                                 const int32_t* lens_host, const float* v_rot, uint32_t flags, uint8_t* v_codes,
                                 uint16_t* v_norm, void* stream) {
  okvq_status st = check_dims(dims);
  if (st != OKVQ_OK) return st;
  if (n_tokens < 0 || !lens_host || (flags & ~(uint32_t)(OKVQ_VALUE_EXACT | OKVQ_GLOBAL_ROTATION)))
    return OKVQ_ERR_INVALID_ARGUMENT;
  if (!aligned16(v) || !aligned16(modality) || !aligned16(v_rot) || !aligned16(v_codes) || !aligned16(v_norm))
    return OKVQ_ERR_INVALID_ARGUMENT;
  const bool global_rot = (flags & OKVQ_GLOBAL_ROTATION) != 0;
  if (global_rot && is_ladder(dims)) return OKVQ_ERR_UNSUPPORTED;
  for (int b = 0; b < dims->batch; ++b) {
    if (lens_host[b] < 0 || lens_host[b] > n_tokens) return OKVQ_ERR_INVALID_ARGUMENT;
    if (lens_host[b] > dims->capacity) return OKVQ_ERR_CAPACITY;
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (is_ladder(dims)) {
    const Codebook& cb = codebook(dims->value_bits);
    for (int b0 = 0; b0 < dims->batch; b0 += kMaxLenArgs) {
      const int nb = std::min(kMaxLenArgs, dims->batch - b0);
      LadderValueArgs a{};
      a.v = v;
      a.modality = modality;
      a.n_rows = n_tokens;
      a.H = dims->num_kv_heads;
      a.cap = dims->capacity;
      a.b0 = b0;
      int max_len = 0;
      for (int i = 0; i < nb; ++i) {
        a.lens.lens[i] = lens_host[b0 + i];
        max_len = std::max(max_len, lens_host[b0 + i]);
      }
      a.rot = v_rot;
      a.v_codes = v_codes;
      a.v_norm = v_norm;
      for (int i = 0; i + 1 < cb.levels; ++i) a.tau[i] = cb.thr[i];
      st = hip_status(launch_ladder_values(a, dims->value_bits, (flags & OKVQ_VALUE_EXACT) != 0, nb, max_len, s));
      if (st != OKVQ_OK) return st;
    }
    return OKVQ_OK;
  }
  const bool exact = (flags & OKVQ_VALUE_EXACT) != 0;
  for (int b0 = 0; b0 < dims->batch; b0 += kMaxLenArgs) {
    const int nb = std::min(kMaxLenArgs, dims->batch - b0);
    CodecArgs a{};
    a.j.src = v;
    a.j.msrc = modality;
    a.j.global_rot = global_rot ? 1 : 0;
    a.j.n_rows = n_tokens;
    a.j.b0 = b0;
    a.j.H = dims->num_kv_heads;
    a.j.cap = dims->capacity;
    int max_len = 0;
    for (int i = 0; i < nb; ++i) {
      a.j.lens.lens[i] = lens_host[b0 + i];
      max_len = std::max(max_len, lens_host[b0 + i]);
    }
    if (exact) {
      st = hip_status(launch_quantize_values_exact(a.j, nb, max_len, v_rot, thresholds(), v_codes, v_norm, nullptr, s));
    } else {
      plan_tiles(a, nb, max_len);
      a.vsrc = v;
      a.rot = v_rot;
      a.th = thresholds();
      a.v_codes = v_codes;
      a.v_norm = v_norm;
      st = hip_status(launch_codec(a, false, true, s));
    }
    if (st != OKVQ_OK) return st;
  }
  return OKVQ_OK;
}

// Append to the bit-width ladder layout: the key codec (the method's keys requantize the open
// window from the stage), the value codec of the new tokens, then the lengths advance.
static okvq_status ladder_append(const okvq_cache* cache, const int32_t* lens_host, const uint16_t* k_new,
                                 const uint16_t* v_new, const uint8_t* mod_new, const int32_t* n_new_host,
                                 const int32_t* n_new_dev, int32_t n_max, bool exact, hipStream_t s) {
  const okvq_dims& d = cache->dims;
  const bool tq = !is_fp16(&d);
  const Codebook& kcb = codebook(d.key_bits);
  const Codebook& vcb = codebook(d.value_bits);
  for (int b0 = 0; b0 < d.batch; b0 += kMaxLenArgs) {
    const int nb = std::min(kMaxLenArgs, d.batch - b0);
    LadderKeyArgs ka{};
    ka.k = k_new;
    ka.n_rows = n_max;
    ka.H = d.num_kv_heads;
    ka.cap = d.capacity;
    ka.b0 = b0;
    ka.begin_dev = cache->seq_lens;
    ka.count_dev = n_new_dev;
    ka.stage = tq ? nullptr : cache->k_stage;
    ka.signs = cache->key_signs;
    ka.k_codes = cache->k_codes;
    ka.k_min = tq ? nullptr : cache->k_min;
    ka.k_step = tq ? nullptr : cache->k_step;
    ka.k_norm = cache->k_norm;
    for (int i = 0; i + 1 < kcb.levels; ++i) ka.tau[i] = kcb.thr[i];
    LadderValueArgs va{};
    va.v = v_new;
    va.modality = mod_new;
    va.n_rows = n_max;
    va.H = d.num_kv_heads;
    va.cap = d.capacity;
    va.b0 = b0;
    va.begin_dev = cache->seq_lens;
    va.count_dev = n_new_dev;
    va.mod_out = cache->modality;
    va.rot = cache->v_rot;
    va.v_codes = cache->v_codes;
    va.v_norm = cache->v_norm;
    for (int i = 0; i + 1 < vcb.levels; ++i) va.tau[i] = vcb.thr[i];
    int key_span = 0, most = 0;
    for (int i = 0; i < nb; ++i) {
      const int L = lens_host[b0 + i], n = n_new_host[b0 + i];
      if (n == 0) continue;
      key_span = std::max(key_span, L + n - (tq ? L : (L / kW) * kW));
      most = std::max(most, n);
    }
    if (most == 0) continue;
    okvq_status st = hip_status(launch_ladder_keys(ka, d.key_bits, tq, nb, key_span, s));
    if (st != OKVQ_OK) return st;
    st = hip_status(launch_ladder_values(va, d.value_bits, exact, nb, most, s));
    if (st != OKVQ_OK) return st;
    st = hip_status(launch_advance_lengths(cache->seq_lens + b0, n_new_dev + b0, nb, s));
    if (st != OKVQ_OK) return st;
  }
  return OKVQ_OK;
}

// events (okvq_append_timed): two events bound to the one launch that codes keys and values
static okvq_status append_impl(const okvq_cache* cache, const int32_t* lens_host, const uint16_t* k_new,
                               const uint16_t* v_new, const uint8_t* mod_new, const int32_t* n_new_host,
                               const int32_t* n_new_dev, int32_t n_max, uint32_t flags, void* stream,
                               void* const* events) {
  okvq_status st = check_cache(cache);
  if (st != OKVQ_OK) return st;
  if (!lens_host || !n_new_host || n_max < 0 || (flags & ~(uint32_t)(OKVQ_VALUE_EXACT | OKVQ_GLOBAL_ROTATION)))
    return OKVQ_ERR_INVALID_ARGUMENT;
  if (is_ladder(&cache->dims) && (flags & OKVQ_GLOBAL_ROTATION)) return OKVQ_ERR_UNSUPPORTED;
  if (!aligned16(k_new) || !aligned16(v_new) || !aligned16(mod_new) || !aligned16(n_new_dev))
    return OKVQ_ERR_INVALID_ARGUMENT;
  const okvq_dims& d = cache->dims;
  int span = 0;  // tokens from the first open window to the new end, largest over sequences
  for (int b = 0; b < d.batch; ++b) {
    const int L = lens_host[b], n = n_new_host[b];
    if (L < 0 || n < 0 || n > n_max) return OKVQ_ERR_INVALID_ARGUMENT;
    if (L > d.capacity || (int64_t)L + n > d.capacity) return OKVQ_ERR_CAPACITY;
    if (n > 0) span = std::max(span, L + n - (L / 32) * 32);
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  const bool exact = (flags & OKVQ_VALUE_EXACT) != 0;
  hipEvent_t ev[2];
  if (events) {  // one codec launch to bind the events to
    if (!events[0] || !events[1]) return OKVQ_ERR_INVALID_ARGUMENT;
    if (is_ladder(&d) || exact || d.batch > kMaxLenArgs || span == 0) return OKVQ_ERR_UNSUPPORTED;
    ev[0] = static_cast<hipEvent_t>(events[0]);
    ev[1] = static_cast<hipEvent_t>(events[1]);
  }
  if (is_ladder(&d)) return span > 0 ? ladder_append(cache, lens_host, k_new, v_new, mod_new, n_new_host, n_new_dev, n_max,
                                                     exact, s)
                                     : OKVQ_OK;
  // Appends that touch few key windows per sequence take the window-parallel launch (codecs,
  // residual rings and lengths in one launch); larger ones the tile launch, which streams longer
  // spans at higher throughput. Both write the same bytes.
  int nwin = 0;  // key windows from the open window to the new end, largest over sequences
  for (int b = 0; b < d.batch; ++b) {
    const int L = lens_host[b], n = n_new_host[b];
    if (n > 0) nwin = std::max(nwin, (L + n + kW - 1) / kW - L / kW);
  }
  const int64_t nwg = (int64_t)nwin * d.num_kv_heads * d.batch;
  bool window_path = !exact && !is_mx(&d) && (nwin <= 2 || (nwin <= kWindowPathMaxWindows && nwg <= kWindowPathMaxGroups));
  if (const char* env = getenv("OKVQ_APPEND_PATH")) {  // "window" / "tile": force a path (tests, timing)
    if (!strcmp(env, "tile")) window_path = false;
    if (!strcmp(env, "window") && !exact && !is_mx(&d)) window_path = true;
  }
  if (events && d.residual && !window_path) return OKVQ_ERR_UNSUPPORTED;  // a second launch
  if (d.residual && span > 0 && !window_path) {  // the fp16 rows, before the codec advances the lengths
    if ((int64_t)d.batch * d.num_kv_heads > INT32_MAX) return OKVQ_ERR_UNSUPPORTED;
    st = hip_status(launch_residual_store(k_new, v_new, n_max, cache->seq_lens, n_new_dev, d.batch, d.num_kv_heads,
                                          d.capacity, cache->k_res, cache->v_res, s));
    if (st != OKVQ_OK) return st;
  }
  for (int b0 = 0; span > 0 && b0 < d.batch; b0 += kMaxLenArgs) {  // launches of up to 256 sequences
    const int nb = std::min(kMaxLenArgs, d.batch - b0);
    CodecArgs a{};
    a.j.src = k_new;
    a.j.msrc = mod_new;
    a.j.global_rot = (flags & OKVQ_GLOBAL_ROTATION) ? 1 : 0;
    a.j.n_rows = n_max;
    a.j.begin_dev = cache->seq_lens;
    a.j.count_dev = n_new_dev;
    a.j.stage = cache->k_stage;
    a.j.b0 = b0;
    a.j.H = d.num_kv_heads;
    a.j.cap = d.capacity;
    int chunk_span = 0;
    for (int i = 0; i < nb; ++i) {
      const int L = lens_host[b0 + i], n = n_new_host[b0 + i];
      a.j.lens.lens[i] = L;
      a.j.cnts.lens[i] = n;
      if (n > 0) chunk_span = std::max(chunk_span, L + n - (L / 32) * 32);
    }
    if (chunk_span == 0) continue;
    plan_tiles(a, nb, chunk_span);
    a.signs = cache->key_signs;
    a.k_codes = cache->k_codes;
    a.k_min = cache->k_min;
    a.k_step = cache->k_step;
    a.k_mx = is_mx(&d) ? cache->k_mx : nullptr;
    a.k_norm = cache->k_norm;
    a.key_meta = meta_mode(&d);
    a.th = thresholds();
    a.v_codes = cache->v_codes;
    a.v_norm = cache->v_norm;
    a.mod_out = cache->modality;
    if (exact) {
      st = hip_status(launch_codec(a, true, false, s));
      if (st != OKVQ_OK) return st;
      CodecJob jv = a.j;
      jv.src = v_new;
      jv.stage = nullptr;
      st = hip_status(launch_quantize_values_exact(jv, nb, chunk_span, cache->v_rot, a.th, cache->v_codes,
                                                   cache->v_norm, cache->modality, s));
      if (st != OKVQ_OK) return st;
      st = hip_status(launch_advance_lengths(cache->seq_lens + b0, n_new_dev + b0, nb, s));
    } else {
      a.vsrc = v_new;
      a.rotfrag = reinterpret_cast<const uint4*>(reinterpret_cast<const char*>(cache->v_rot16) + kRotInverseBytes);
      a.seq_lens_out = cache->seq_lens;
      a.ticket = reinterpret_cast<uint32_t*>(cache->seq_lens + d.batch);
      a.status = cache->seq_lens + d.batch + 1;
      if (window_path) {
        a.k_res = d.residual ? cache->k_res : nullptr;
        a.v_res = d.residual ? cache->v_res : nullptr;
        int chunk_nwin = 0;
        for (int i = 0; i < nb; ++i) {
          const int L = lens_host[b0 + i], n = n_new_host[b0 + i];
          if (n > 0) chunk_nwin = std::max(chunk_nwin, (L + n + kW - 1) / kW - L / kW);
        }
        st = hip_status(launch_append_window(a, chunk_nwin, nb, s, events ? ev : nullptr));
      } else {
        st = hip_status(launch_codec(a, true, true, s, events ? ev : nullptr));
      }
    }
    if (st != OKVQ_OK) return st;
  }
  return OKVQ_OK;
}

okvq_status okvq_append(const okvq_cache* cache, const int32_t* lens_host, const uint16_t* k_new, const uint16_t* v_new,
                        const uint8_t* mod_new, const int32_t* n_new_host, const int32_t* n_new_dev, int32_t n_max,
                        uint32_t flags, void* stream) {
  return append_impl(cache, lens_host, k_new, v_new, mod_new, n_new_host, n_new_dev, n_max, flags, stream, nullptr);
}

okvq_status okvq_append_timed(const okvq_cache* cache, const int32_t* lens_host, const uint16_t* k_new,
                              const uint16_t* v_new, const uint8_t* mod_new, const int32_t* n_new_host,
                              const int32_t* n_new_dev, int32_t n_max, uint32_t flags, void* stream,
                              void* const* events) {
  if (!events) return OKVQ_ERR_INVALID_ARGUMENT;
  return append_impl(cache, lens_host, k_new, v_new, mod_new, n_new_host, n_new_dev, n_max, flags, stream, events);
}

okvq_status okvq_cache_status(const okvq_cache* cache, int32_t* status, void* stream) {
  okvq_status st = check_cache(cache);
  if (st != OKVQ_OK) return st;
  if (!status) return OKVQ_ERR_INVALID_ARGUMENT;
  hipStream_t s = static_cast<hipStream_t>(stream);
  int32_t word = 0;
  if (hipMemcpyAsync(&word, cache->seq_lens + cache->dims.batch + 1, sizeof(word), hipMemcpyDeviceToHost, s) !=
          hipSuccess ||
      hipStreamSynchronize(s) != hipSuccess)
    return OKVQ_ERR_HIP;
  *status = word;
  return OKVQ_OK;
}

okvq_status okvq_prepare_rotation(const float* v_rot, uint16_t* v_rot16, void* stream) {
  if (!aligned16(v_rot) || !aligned16(v_rot16)) return OKVQ_ERR_INVALID_ARGUMENT;
  hipStream_t s = static_cast<hipStream_t>(stream);
  okvq_status st = hip_status(launch_prepare_rotation(v_rot, v_rot16, s));
  if (st != OKVQ_OK) return st;
  return hip_status(launch_prepare_fragments(
      v_rot, reinterpret_cast<uint4*>(reinterpret_cast<char*>(v_rot16) + kRotInverseBytes), s));
}

size_t okvq_decode_workspace_bytes(const okvq_dims* dims, int32_t max_seq_len) {
  if (check_dims(dims) != OKVQ_OK || max_seq_len < 0) return 0;
  if (is_ladder(dims)) return ladder_workspace_bytes(dims->batch, dims->num_kv_heads, max_seq_len);
  return decode_workspace_bytes(dims->batch, dims->num_kv_heads, dims->num_q_heads, max_seq_len);
}

// workspace == nullptr with workspace_bytes == 0 selects the static per-GPU scratch array (the
// allocation-free entry point): the records of this call's plan must fit in it.
static okvq_status decode_impl(const okvq_cache* cache, const int32_t* lens_host, const uint16_t* q, float sm_scale,
                               uint32_t flags, float* out, void* workspace, size_t workspace_bytes, void* stream,
                               void* const* events, bool use_scratch = false) {
  okvq_status st = check_cache(cache);
  if (st != OKVQ_OK) return st;
  if (!lens_host || (flags & ~(uint32_t)OKVQ_GLOBAL_ROTATION) || !std::isfinite(sm_scale))
    return OKVQ_ERR_INVALID_ARGUMENT;
  const bool global_rot = (flags & OKVQ_GLOBAL_ROTATION) != 0;
  if (!aligned16(q) || !aligned16(out)) return OKVQ_ERR_INVALID_ARGUMENT;
  const okvq_dims& d = cache->dims;
  if (global_rot && is_ladder(&d)) return OKVQ_ERR_UNSUPPORTED;
  int max_len = 0;
  for (int b = 0; b < d.batch; ++b) {
    if (lens_host[b] < 0) return OKVQ_ERR_INVALID_ARGUMENT;
    if (lens_host[b] > d.capacity) return OKVQ_ERR_CAPACITY;
    max_len = std::max(max_len, lens_host[b]);
  }
  if (use_scratch) {  // the records of this call's plan, in the static array
    const size_t nsplit = is_ladder(&d) ? plan_ladder(d.batch, d.num_kv_heads, max_len).nsplit
                                        : plan_decode(d.batch, d.num_kv_heads, std::max(max_len - d.residual, 0)).nsplit;
    if ((size_t)d.batch * d.num_kv_heads * nsplit * kRecFloats * sizeof(float) > OKVQ_NOALLOC_SCRATCH_BYTES)
      return OKVQ_ERR_WORKSPACE;
    st = scratch_address(&workspace);
    if (st != OKVQ_OK) return st;
  } else {
    const size_t need = is_ladder(&d) ? ladder_workspace_bytes(d.batch, d.num_kv_heads, max_len)
                                      : decode_workspace_bytes(d.batch, d.num_kv_heads, d.num_q_heads, max_len);
    if (!aligned16(workspace) || workspace_bytes < need) return OKVQ_ERR_WORKSPACE;
  }
  hipEvent_t ev[4];
  if (events) {
    for (int i = 0; i < 4; ++i) {
      if (!events[i]) return OKVQ_ERR_INVALID_ARGUMENT;
      ev[i] = static_cast<hipEvent_t>(events[i]);
    }
  }
  if (is_ladder(&d)) {
    LadderDecodeArgs a{};
    a.k_codes = cache->k_codes;
    a.v_codes = cache->v_codes;
    a.k_norm = cache->k_norm;
    a.v_norm = cache->v_norm;
    a.k_min = is_fp16(&d) ? cache->k_min : nullptr;
    a.k_step = is_fp16(&d) ? cache->k_step : nullptr;
    a.modality = cache->modality;
    a.seq_lens = cache->seq_lens;
    a.signs = cache->key_signs;
    a.q = q;
    a.rot16t = cache->v_rot16;
    a.ws = static_cast<float*>(workspace);
    a.H = d.num_kv_heads;
    a.Hq = d.num_q_heads;
    a.G = d.num_q_heads / d.num_kv_heads;
    a.cap = d.capacity;
    a.qscale = sm_scale * 1.4426950408889634f * 0.08838834764831845f;
    const Codebook& kc = codebook(d.key_bits);
    const Codebook& vc = codebook(d.value_bits);
    for (int i = 0; i < kc.levels; ++i) a.kcb16[i] = kc.level16[i];
    for (int i = 0; i < vc.levels; ++i) a.vcb16[i] = vc.level16[i];
    return hip_status(launch_ladder_decode(a, d.key_bits, d.value_bits, !is_fp16(&d), d.batch,
                                           plan_ladder(d.batch, d.num_kv_heads, max_len), out,
                                           static_cast<hipStream_t>(stream), events ? ev : nullptr));
  }
  // with the fp16 residual the split-K launch covers the tokens below L - 128
  const DecodePlan plan = plan_decode(d.batch, d.num_kv_heads, std::max(max_len - d.residual, 0));
  const Codebook& cb = codebook();
  const uint32_t cb01 = cb.level16[0] | ((uint32_t)cb.level16[1] << 16);
  const uint32_t cb23 = cb.level16[2] | ((uint32_t)cb.level16[3] << 16);
  return hip_status(launch_decode(view(cache), q, sm_scale, out, workspace, plan, static_cast<hipStream_t>(stream),
                                  cb01, cb23, max_len, events ? ev : nullptr, global_rot));
}

okvq_status okvq_decode_attention(const okvq_cache* cache, const int32_t* lens_host, const uint16_t* q, float sm_scale,
                                  uint32_t flags, float* out, void* workspace, size_t workspace_bytes, void* stream) {
  return decode_impl(cache, lens_host, q, sm_scale, flags, out, workspace, workspace_bytes, stream, nullptr);
}

okvq_status okvq_decode_attention_noalloc(const okvq_cache* cache, const int32_t* lens_host, const uint16_t* q,
                                          float sm_scale, uint32_t flags, float* out, void* stream) {
  return decode_impl(cache, lens_host, q, sm_scale, flags, out, nullptr, 0, stream, nullptr, true);
}

okvq_status okvq_decode_attention_timed(const okvq_cache* cache, const int32_t* lens_host, const uint16_t* q,
                                        float sm_scale, uint32_t flags, float* out, void* workspace,
                                        size_t workspace_bytes, void* stream, void* const* events) {
  if (!events) return OKVQ_ERR_INVALID_ARGUMENT;
  return decode_impl(cache, lens_host, q, sm_scale, flags, out, workspace, workspace_bytes, stream, events);
}

size_t okvq_dense_workspace_bytes(const okvq_dims* dims, int32_t max_seq_len) {
  if (check_dims(dims) != OKVQ_OK || max_seq_len < 0) return 0;
  return dense_workspace_bytes(dims->batch, dims->num_kv_heads, max_seq_len);
}

okvq_status okvq_decode_attention_dense(const okvq_dims* dims, const uint16_t* k, const uint16_t* v,
                                        const int32_t* seq_lens, const int32_t* lens_host, const uint16_t* q,
                                        float sm_scale, float* out, void* workspace, size_t workspace_bytes,
                                        void* stream, void* const* events) {
  okvq_status st = check_dims(dims);
  if (st != OKVQ_OK) return st;
  if (!lens_host || !std::isfinite(sm_scale)) return OKVQ_ERR_INVALID_ARGUMENT;
  if (!aligned16(k) || !aligned16(v) || !aligned16(seq_lens) || !aligned16(q) || !aligned16(out))
    return OKVQ_ERR_INVALID_ARGUMENT;
  int max_len = 0;
  for (int b = 0; b < dims->batch; ++b) {
    if (lens_host[b] < 0) return OKVQ_ERR_INVALID_ARGUMENT;
    if (lens_host[b] > dims->capacity) return OKVQ_ERR_CAPACITY;
    max_len = std::max(max_len, lens_host[b]);
  }
  const size_t need = dense_workspace_bytes(dims->batch, dims->num_kv_heads, max_len);
  if (!aligned16(workspace) || workspace_bytes < need) return OKVQ_ERR_WORKSPACE;
  hipEvent_t ev[4];
  if (events) {
    for (int i = 0; i < 4; ++i) {
      if (!events[i]) return OKVQ_ERR_INVALID_ARGUMENT;
      ev[i] = static_cast<hipEvent_t>(events[i]);
    }
  }
  const DensePlan plan = plan_dense(dims->batch, dims->num_kv_heads, max_len);
  return hip_status(launch_decode_dense(k, v, seq_lens, q, dims->batch, dims->num_kv_heads, dims->num_q_heads,
                                        dims->capacity, sm_scale, out, workspace, plan,
                                        static_cast<hipStream_t>(stream), events ? ev : nullptr));
}

size_t okvq_calibration_workspace_bytes(const okvq_dims* dims, int32_t n_tokens) {
  if (check_dims(dims) != OKVQ_OK || n_tokens < 1) return 0;
  return calib_workspace_bytes(dims->batch, dims->num_kv_heads, dims->num_q_heads, n_tokens);
}

okvq_status okvq_calibration_weights(const okvq_dims* dims, const uint16_t* q, const uint16_t* k, int32_t n_tokens,
                                     const int32_t* lens_host, float sm_scale, float* w, void* workspace,
                                     size_t workspace_bytes, void* stream) {
  okvq_status st = check_dims(dims);
  if (st != OKVQ_OK) return st;
  if (n_tokens < 1 || !lens_host || !std::isfinite(sm_scale)) return OKVQ_ERR_INVALID_ARGUMENT;
  if (!aligned16(q) || !aligned16(k) || !aligned16(w)) return OKVQ_ERR_INVALID_ARGUMENT;
  for (int b = 0; b < dims->batch; ++b)
    if (lens_host[b] < 0 || lens_host[b] > n_tokens) return OKVQ_ERR_INVALID_ARGUMENT;
  if (!aligned16(workspace) ||
      workspace_bytes < calib_workspace_bytes(dims->batch, dims->num_kv_heads, dims->num_q_heads, n_tokens))
    return OKVQ_ERR_WORKSPACE;
  hipStream_t s = static_cast<hipStream_t>(stream);
  for (int b0 = 0; b0 < dims->batch; b0 += kMaxLenArgs) {
    const int nb = std::min(kMaxLenArgs, dims->batch - b0);
    LenArgs la{};
    for (int i = 0; i < nb; ++i) la.lens[i] = lens_host[b0 + i];
    st = hip_status(launch_calib_weights(q, k, la, b0, nb, n_tokens, dims->num_kv_heads, dims->num_q_heads, sm_scale,
                                         w, workspace, s));
    if (st != OKVQ_OK) return st;
  }
  return OKVQ_OK;
}

okvq_status okvq_value_covariance(const okvq_dims* dims, const uint16_t* v, const uint8_t* modality, const float* w,
                                  int32_t n_tokens, const int32_t* lens_host, float* cov, void* workspace,
                                  size_t workspace_bytes, void* stream) {
  okvq_status st = check_dims(dims);
  if (st != OKVQ_OK) return st;
  if (n_tokens < 1 || !lens_host) return OKVQ_ERR_INVALID_ARGUMENT;
  if (!aligned16(v) || !aligned16(modality) || !aligned16(w) || !aligned16(cov)) return OKVQ_ERR_INVALID_ARGUMENT;
  for (int b = 0; b < dims->batch; ++b)
    if (lens_host[b] < 0 || lens_host[b] > n_tokens) return OKVQ_ERR_INVALID_ARGUMENT;
  if (!aligned16(workspace) ||
      workspace_bytes < calib_workspace_bytes(dims->batch, dims->num_kv_heads, dims->num_q_heads, n_tokens))
    return OKVQ_ERR_WORKSPACE;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int H = dims->num_kv_heads, nchunk = (n_tokens + kCalibChunk - 1) / kCalibChunk;
  const int nparts = dims->batch * H * nchunk;
  for (int b0 = 0; b0 < dims->batch; b0 += kMaxLenArgs) {
    const int nb = std::min(kMaxLenArgs, dims->batch - b0);
    LenArgs la{};
    for (int i = 0; i < nb; ++i) la.lens[i] = lens_host[b0 + i];
    const bool last = b0 + nb >= dims->batch;
    st = hip_status(launch_calib_covariance(v, modality, w, la, b0, nb, n_tokens, H, static_cast<float*>(workspace),
                                            b0 * H * nchunk, cov, last, nparts, s));
    if (st != OKVQ_OK) return st;
  }
  return OKVQ_OK;
}

okvq_status okvq_rotation_from_covariance(const float* cov, const int8_t* signs, float* rot, double* eigenvalues) {
  if (!cov || !signs || !rot) return OKVQ_ERR_INVALID_ARGUMENT;
  constexpr int n = 128;
  for (int i = 0; i < n; ++i)
    if (signs[i] != 1 && signs[i] != -1) return OKVQ_ERR_INVALID_ARGUMENT;
  for (int i = 0; i < 3 * n * n; ++i)
    if (!std::isfinite(cov[i])) return OKVQ_ERR_INVALID_ARGUMENT;
  const double inv_sqrt_n = 1.0 / std::sqrt((double)n);
  for (int m = 0; m < 3; ++m) {
    std::vector<double> a((size_t)n * n), u, d;
    for (int r = 0; r < n; ++r)  // the symmetric part (the device sums are symmetric up to rounding)
      for (int c = 0; c < n; ++c)
        a[(size_t)r * n + c] = 0.5 * ((double)cov[((size_t)m * n + r) * n + c] + (double)cov[((size_t)m * n + c) * n + r]);
    jacobi_eigen(a, u, d, n);
    std::vector<int> order(n);
    std::iota(order.begin(), order.end(), 0);
    std::stable_sort(order.begin(), order.end(), [&](int x, int y) { return d[x] > d[y]; });
    // U_m: eigenvectors as columns in descending eigenvalue order, each with its largest-magnitude
    // component positive (the first such component on ties)
    std::vector<double> U((size_t)n * n);
    for (int k = 0; k < n; ++k) {
      const int src = order[k];
      int imax = 0;
      for (int i = 1; i < n; ++i)
        if (std::fabs(u[(size_t)i * n + src]) > std::fabs(u[(size_t)imax * n + src])) imax = i;
      const double sg = u[(size_t)imax * n + src] < 0.0 ? -1.0 : 1.0;
      for (int i = 0; i < n; ++i) U[(size_t)i * n + k] = sg * u[(size_t)i * n + src];
      if (eigenvalues) eigenvalues[m * n + k] = d[src];
    }
    // R_m = H U_m^T (Eq. 6), H = Had diag(s) / sqrt(128), Had[a][k] = (-1)^popcount(a & k)
    for (int r = 0; r < n; ++r)
      for (int c = 0; c < n; ++c) {
        double acc = 0.0;
        for (int k = 0; k < n; ++k) {
          const double h = ((__builtin_popcount(r & k) & 1) ? -1.0 : 1.0) * signs[k];
          acc += h * U[(size_t)c * n + k];
        }
        rot[((size_t)m * n + r) * n + c] = (float)(acc * inv_sqrt_n);
      }
  }
  return OKVQ_OK;
}

}  // extern "C"
