// libwd host runtime: the C ABI of include/wd.h.
//
// The host keeps the schedule's counts (they do not depend on which positions
// get decoded, so every launch size is known without reading the device);
// the device keeps the token state and derives the identities of the rows
// (build_rows) from the decoded flags.  Nothing is read back between steps
// unless the caller asks for a step's result.
//
// With adaptive termination (eos_id >= 0) the counts depend on where <eos>
// is decoded, so the host mirrors each sequence's decoded flags (Track),
// reads every step's decisions back and gives each sequence its own phase
// clock, window and live end.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/wd.h"
#include "common.h"
#include "kernels.h"

// ---- scratch of the entry point that allocates nothing (wd_step_noalloc) -------------
// The step's split-K partials, split-KV attention partials and confidence
// partials live here instead of in the caller's workspace.  Each GPU the
// library runs on holds its own copy until the process ends.  Host code must
// not use the array's name (a host-side stand-in, not a device address): it
// uses the address hipGetSymbolAddress gave for the device, kept per device.
constexpr size_t kStaticScratchBytes = WD_STATIC_SCRATCH_BYTES;
static __device__ __align__(256) char scratch[kStaticScratchBytes];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_dev[kMaxDevices] = {};  // device address of `scratch` on each device

}  // namespace

namespace {

thread_local std::string g_err;

wd_status fail(wd_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

#define WD_HIP(call)                                                                   \
  do {                                                                                 \
    hipError_t e_ = (call);                                                            \
    if (e_ != hipSuccess)                                                              \
      return fail(WD_ERR_DEVICE, "%s failed: %s", #call, hipGetErrorString(e_));       \
  } while (0)

#define WD_TRY(call)                   \
  do {                                 \
    wd_status s_ = (call);             \
    if (s_ != WD_OK) return s_;        \
  } while (0)

size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

// Resolves the device address of `scratch` on `device`, which must be the
// current device; once per device.
wd_status init_static_scratch(int device) {
  if (device < 0 || device >= kMaxDevices)
    return fail(WD_ERR_UNSUPPORTED, "device %d beyond the %d the library tracks", device, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_dev[device]) return WD_OK;
  void* p = nullptr;
  const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
  if (e != hipSuccess || !p)
    return fail(WD_ERR_DEVICE, "hipGetSymbolAddress(scratch) failed on device %d: %s", device,
                hipGetErrorString(e));
  g_scratch_dev[device] = p;
  return WD_OK;
}

// -- model shape checks --------------------------------------------------------------
bool cfg_valid(const wd_model_config* c, std::string* why) {
  if (!c) {
    *why = "NULL config";
    return false;
  }
  if (c->n_layers < 1 || c->hidden < 64 || c->n_heads < 1 || c->n_kv_heads < 1 || c->vocab < 2 ||
      c->ffn < 64) {
    *why = "non-positive or too small dimension";
    return false;
  }
  if (c->dtype != WD_DTYPE_F32 && c->dtype != WD_DTYPE_BF16) {
    *why = "dtype must be WD_DTYPE_F32 or WD_DTYPE_BF16";
    return false;
  }
  if (c->head_dim != 64 && c->head_dim != 128) {
    *why = "head_dim must be 64 or 128";
    return false;
  }
  if (c->dtype == WD_DTYPE_BF16 && c->head_dim != 128) {
    *why = "bf16 models need head_dim 128";
    return false;
  }
  if (c->n_heads % c->n_kv_heads) {
    *why = "n_heads must be a multiple of n_kv_heads";
    return false;
  }
  if (c->hidden % 64 || (c->n_heads * c->head_dim) % 64 || c->ffn % 64 || c->vocab % 64) {
    *why = "hidden, n_heads*head_dim, ffn and vocab must be multiples of 64";
    return false;
  }
  if (c->hidden > 16384) {
    *why = "hidden above 16384 is not supported";
    return false;
  }
  if (c->mask_id < 0 || c->mask_id >= c->vocab) {
    *why = "mask_id outside [0, vocab)";
    return false;
  }
  if (c->weight_fp8 != 0 && c->weight_fp8 != 1) {
    *why = "weight_fp8 must be 0 or 1";
    return false;
  }
  if (c->weight_fp8 && c->dtype != WD_DTYPE_BF16) {
    *why = "fp8 weights are a variant of bf16 models";
    return false;
  }
  if (c->qkv_bias != 0 && c->qkv_bias != 1) {
    *why = "qkv_bias must be 0 or 1";
    return false;
  }
  if (!(c->rms_eps > 0.f) || !(c->rope_theta > 1.f)) {
    *why = "rms_eps must be > 0 and rope_theta > 1";
    return false;
  }
  return true;
}

struct TensorSpec {
  long rows, cols;
  std::string name;  // as in the wd_init_model order: emb, layers.<l>.wq, ..., lm_head
};

std::vector<TensorSpec> tensor_specs(const wd_model_config& c) {
  const long H = c.hidden, Q = (long)c.n_heads * c.head_dim, KV = (long)c.n_kv_heads * c.head_dim;
  std::vector<TensorSpec> v;
  v.push_back({c.vocab, H, "emb"});
  for (int l = 0; l < c.n_layers; ++l) {
    const std::string p = "layers." + std::to_string(l) + ".";
    v.push_back({H, 1, p + "attn_norm"});
    v.push_back({Q, H, p + "wq"});
    v.push_back({KV, H, p + "wk"});
    v.push_back({KV, H, p + "wv"});
    if (c.qkv_bias) {
      v.push_back({Q, 1, p + "bq"});
      v.push_back({KV, 1, p + "bk"});
      v.push_back({KV, 1, p + "bv"});
    }
    v.push_back({H, Q, p + "wo"});
    v.push_back({H, 1, p + "ffn_norm"});
    v.push_back({c.ffn, H, p + "wg"});
    v.push_back({c.ffn, H, p + "wu"});
    v.push_back({H, c.ffn, p + "wd"});
  }
  v.push_back({H, 1, "final_norm"});
  v.push_back({c.vocab, H, "lm_head"});
  return v;
}

// -- the schedule's counts (shared by the runtime and wd_plan) ---------------------
struct Counts {
  int E = 0, R = 1, k = 1, na = 1;
  int u = 0;          // undecoded positions per sequence
  int in_window = 0;  // undecoded positions of the current window
  int dp = 0;         // positions decoded in the current phase
  int prev_dp = 0;    // positions decoded in the previous phase
  int phases = 0;     // phases started
  int j = -1;         // steps taken in the current phase (-1: no phase yet)

  bool phase_due() const { return j < 0 || j >= R || in_window == 0; }
  int ctx(int S) const { return u >= E ? S - u + E : S; }
  void start_phase() {
    in_window = std::min(E, u);
    prev_dp = dp;
    dp = 0;
    j = 0;
    ++phases;
  }
  // rows of the refresh step: [0, c), or with the buffer-only variant after
  // the first phase the window plus the previous phase's decoded positions
  int refresh_rows(int c, bool buffer) const { return buffer && phases > 1 ? in_window + prev_dp : c; }
  int n_active() const { return std::min(na, in_window); }
  int n_decode() const { return std::min(k, n_active()); }
  void take_step() {
    const int d = n_decode();
    u -= d;
    in_window -= d;
    dp += d;
    ++j;
  }
};

// Host decode of an e4m3 code (sign, 4-bit exponent with bias 7, 3-bit
// mantissa; exponent 0 holds m * 2^-9) for wd_debug_weight_row.
float e4m3_to_float(uint8_t c) {
  const int e = (c >> 3) & 15, m = c & 7;
  const float mag = e == 0 ? std::ldexp((float)m, -9) : std::ldexp(1.f + m / 8.f, e - 7);
  return (c & 0x80) ? -mag : mag;
}

// Exact host copy of one sequence's schedule under adaptive termination
// (Sec. 4.2): the live end, the decoded flags, the phase's window and its
// retained prefix.
struct Track {
  int n_p = 0, S = 0, end = 0;  // live positions are [0, end)
  int c = 0;                    // retained prefix of the phase
  int j = -1;                   // steps taken in the phase (-1: none yet)
  std::vector<uint8_t> dec, dec0;
  std::vector<int> window;      // W_ex of the phase

  bool done() const {
    for (int p = 0; p < end; ++p)
      if (!dec[p]) return false;
    return true;
  }
  bool live_in_window() const {
    for (int p : window)
      if (p < end && !dec[p]) return true;
    return false;
  }
  bool phase_due(int R) const { return j < 0 || j >= R || !live_in_window(); }
  void slide(int E) {
    window.clear();
    c = end;
    for (int p = 0; p < end; ++p)
      if (!dec[p]) {
        window.push_back(p);
        if ((int)window.size() == E) {
          c = p + 1;
          break;
        }
      }
    dec0 = dec;
    j = 0;
  }
  int ctx() const { return std::min(c, end); }
  int n_active(int na) const {
    int n = 0;
    for (int p : window)
      if (p < end && !dec[p]) ++n;
    return std::min(n, na);
  }
  int n_phase_decoded() const {
    int n = 0;
    for (int p = 0; p < ctx(); ++p) n += dec[p] && !dec0[p];
    return n;
  }
  int live_undecoded() const {
    int n = 0;
    for (int p = 0; p < end; ++p) n += !dec[p];
    return n;
  }
  // a decision of the step: position p now holds token t
  void apply(int p, int t, int eos_id) {
    dec[p] = 1;
    if (t == eos_id && p >= n_p) end = std::min(end, p + 1);
  }
};

}  // namespace

// -- model ---------------------------------------------------------------------------
struct LayerW {
  const void* attn_norm;
  const void* wqkv;
  const void* bqkv;  // NULL without bias
  const void* wo;
  const void* ffn_norm;
  const void* wgu;
  const void* wd;
  // fp8 row scales of the packed matrices (NULL with bf16 / fp32 weights)
  const float *sqkv, *so, *sgu, *sd;
};

struct wd_model {
  wd_model_config cfg;
  hipStream_t stream;
  int device;
  size_t esz;
  int qkv_n;
  const void* emb;
  const void* final_norm;
  const void* lm;
  const float* slm = nullptr;  // fp8 row scales of the LM head
  std::vector<LayerW> layers;
  int live_seqs = 0;
  // kernel timing (wd_profile_enable)
  bool profile = false;
  std::vector<hipEvent_t> ev;    // event pool, two per recorded launch
  size_t n_rec = 0;              // launches recorded since the last read
  std::vector<double> rec_bytes, rec_flops;
  std::vector<int> rec_kind;     // WD_PROF_* class of each recorded launch
};

namespace {

// Byte layout of the packed weight buffer; the same walk sizes and fills it.
struct ModelLayout {
  size_t total = 0;
  size_t emb, final_norm, lm, slm = 0;
  struct L {
    size_t attn_norm, wqkv, bqkv, wo, ffn_norm, wgu, wd;
    size_t sqkv = 0, so = 0, sgu = 0, sd = 0;  // fp8 row scales
  };
  std::vector<L> layers;
};

ModelLayout model_layout(const wd_model_config& c) {
  const size_t e = c.dtype == WD_DTYPE_BF16 ? 2 : 4;
  const size_t H = c.hidden, Q = (size_t)c.n_heads * c.head_dim,
               KV = (size_t)c.n_kv_heads * c.head_dim, F = c.ffn;
  ModelLayout m;
  size_t o = 0;
  auto take = [&](size_t bytes) {
    const size_t at = o;
    o += align256(bytes);
    return at;
  };
  // projection matrices: bf16 fragments (2 bytes per weight), or e4m3 codes
  // (1 byte) plus a float32 scale per output row
  const bool w8 = c.weight_fp8 != 0;
  const size_t ew = w8 ? 1 : e;
  auto scales = [&](size_t rows) { return w8 ? take(rows * 4) : (size_t)0; };
  m.emb = take((size_t)c.vocab * H * e);
  for (int l = 0; l < c.n_layers; ++l) {
    ModelLayout::L L;
    L.attn_norm = take(H * e);
    L.wqkv = take((Q + 2 * KV) * H * ew);
    L.sqkv = scales(Q + 2 * KV);
    L.bqkv = c.qkv_bias ? take((Q + 2 * KV) * e) : 0;
    L.wo = take(H * Q * ew);
    L.so = scales(H);
    L.ffn_norm = take(H * e);
    L.wgu = take(2 * F * H * ew);
    L.sgu = scales(2 * F);
    L.wd = take(H * F * ew);
    L.sd = scales(H);
    m.layers.push_back(L);
  }
  m.final_norm = take(H * e);
  m.lm = take((size_t)c.vocab * H * ew);
  m.slm = scales(c.vocab);
  m.total = o;
  return m;
}

// Copies (fp32) or packs into MFMA fragments (bf16) one [N, K] matrix at dst.
// bf16 weights are packed into MFMA fragments (rows reordered by perm, W2 =
// the up half of kPackGateUp); fp32 weights are copied as they are.
wd_status put_matrix(const wd_model& m, const void* src, long N, long K, char* dst,
                     int perm = wd::kPackPlain, const void* src2 = nullptr,
                     float* scale = nullptr) {
  if (m.cfg.weight_fp8) {
    WD_HIP(wd::pack_fp8((const uint16_t*)src, (int)N, (int)K, dst, scale, m.stream, perm,
                        (const uint16_t*)src2));
  } else if (m.cfg.dtype == WD_DTYPE_BF16) {
    WD_HIP(wd::pack_frags((const uint16_t*)src, (int)N, (int)K, dst, m.stream, perm,
                          (const uint16_t*)src2));
  } else {
    // with src2 (gate then up) each half is N / 2 rows
    const size_t bytes = (size_t)(src2 ? N / 2 : N) * K * 4;
    WD_HIP(hipMemcpyAsync(dst, src, bytes, hipMemcpyDeviceToDevice, m.stream));
    if (src2) WD_HIP(hipMemcpyAsync(dst + bytes, src2, bytes, hipMemcpyDeviceToDevice, m.stream));
  }
  return WD_OK;
}

}  // namespace

extern "C" {

const char* wd_last_error(void) { return g_err.c_str(); }

int32_t wd_weight_count(const wd_model_config* cfg) {
  std::string why;
  if (!cfg_valid(cfg, &why)) return -1;
  return (int32_t)tensor_specs(*cfg).size();
}

wd_status wd_weight_shape(const wd_model_config* cfg, int32_t i, int64_t* rows, int64_t* cols) {
  std::string why;
  if (!cfg_valid(cfg, &why)) return fail(WD_ERR_INVALID_ARG, "invalid config: %s", why.c_str());
  const auto v = tensor_specs(*cfg);
  if (i < 0 || i >= (int32_t)v.size() || !rows || !cols)
    return fail(WD_ERR_INVALID_ARG, "tensor index %d out of range", i);
  *rows = v[i].rows;
  *cols = v[i].cols;
  return WD_OK;
}

size_t wd_model_bytes(const wd_model_config* cfg) {
  std::string why;
  if (!cfg_valid(cfg, &why)) return 0;
  return model_layout(*cfg).total;
}

wd_status wd_init_model(const wd_model_config* cfg, const void* const* weights, int32_t n_weights,
                        void* device_buf, size_t buf_bytes, void* stream, wd_model** out) {
  std::string why;
  if (!out) return fail(WD_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  if (!cfg_valid(cfg, &why)) {
    const bool shape = cfg && why.find("NULL") == std::string::npos &&
                       why.find("non-positive") == std::string::npos;
    return fail(shape ? WD_ERR_UNSUPPORTED : WD_ERR_INVALID_ARG, "invalid config: %s", why.c_str());
  }
  const auto specs = tensor_specs(*cfg);
  if (!weights || n_weights != (int32_t)specs.size())
    return fail(WD_ERR_INVALID_ARG, "expected %zu weight pointers, got %d", specs.size(), n_weights);
  for (size_t i = 0; i < specs.size(); ++i) {
    if (!weights[i]) return fail(WD_ERR_INVALID_ARG, "weight %zu is NULL", i);
    if (((uintptr_t)weights[i]) & 15)
      return fail(WD_ERR_INVALID_ARG, "weight %zu is not 16-byte aligned", i);
  }
  const ModelLayout lay = model_layout(*cfg);
  if (!device_buf) return fail(WD_ERR_INVALID_ARG, "device_buf is NULL");
  if (((uintptr_t)device_buf) & 255) return fail(WD_ERR_INVALID_ARG, "device_buf not 256-byte aligned");
  if (buf_bytes < lay.total)
    return fail(WD_ERR_OUT_OF_MEMORY, "device_buf holds %zu bytes, %zu needed", buf_bytes, lay.total);

  wd_model* m = new (std::nothrow) wd_model();
  if (!m) return fail(WD_ERR_OUT_OF_MEMORY, "host allocation failed");
  m->cfg = *cfg;
  m->stream = (hipStream_t)stream;
  if (hipGetDevice(&m->device) != hipSuccess) {
    delete m;
    return fail(WD_ERR_DEVICE, "hipGetDevice failed");
  }
  if (const wd_status ss = init_static_scratch(m->device); ss != WD_OK) {
    delete m;
    return ss;
  }
  m->esz = cfg->dtype == WD_DTYPE_BF16 ? 2 : 4;
  m->qkv_n = (cfg->n_heads + 2 * cfg->n_kv_heads) * cfg->head_dim;
  char* base = (char*)device_buf;
  const long H = cfg->hidden, Q = (long)cfg->n_heads * cfg->head_dim,
             KV = (long)cfg->n_kv_heads * cfg->head_dim, F = cfg->ffn;
  const size_t e = m->esz;
  const bool w8 = cfg->weight_fp8 != 0;
  const size_t ew = w8 ? 1 : e;  // bytes per packed projection weight
  auto fail_free = [&](wd_status s) {
    delete m;
    return s;
  };
  auto copy = [&](const void* src, size_t bytes, char* dst) -> wd_status {
    WD_HIP(hipMemcpyAsync(dst, src, bytes, hipMemcpyDeviceToDevice, m->stream));
    return WD_OK;
  };
  // packed size of an [N, K] matrix (fragments are exactly N*K elements)
  size_t wi = 0;
  wd_status st;
  if ((st = copy(weights[wi++], (size_t)cfg->vocab * H * e, base + lay.emb)) != WD_OK) return fail_free(st);
  m->emb = base + lay.emb;
  for (int l = 0; l < cfg->n_layers; ++l) {
    const auto& L = lay.layers[l];
    LayerW w{};
    if ((st = copy(weights[wi++], H * e, base + L.attn_norm)) != WD_OK) return fail_free(st);
    const void* wq = weights[wi++];
    const void* wk = weights[wi++];
    const void* wv = weights[wi++];
    const int rp = wd::kPackRopePair;
    float* sq = w8 ? (float*)(base + L.sqkv) : nullptr;
    if ((st = put_matrix(*m, wq, Q, H, base + L.wqkv, rp, nullptr, sq)) != WD_OK) return fail_free(st);
    if ((st = put_matrix(*m, wk, KV, H, base + L.wqkv + Q * H * ew, rp, nullptr, w8 ? sq + Q : nullptr)) !=
        WD_OK)
      return fail_free(st);
    if ((st = put_matrix(*m, wv, KV, H, base + L.wqkv + (Q + KV) * H * ew, rp, nullptr,
                         w8 ? sq + Q + KV : nullptr)) != WD_OK)
      return fail_free(st);
    w.sqkv = sq;
    if (cfg->qkv_bias) {
      if ((st = copy(weights[wi++], Q * e, base + L.bqkv)) != WD_OK) return fail_free(st);
      if ((st = copy(weights[wi++], KV * e, base + L.bqkv + Q * e)) != WD_OK) return fail_free(st);
      if ((st = copy(weights[wi++], KV * e, base + L.bqkv + (Q + KV) * e)) != WD_OK) return fail_free(st);
      w.bqkv = base + L.bqkv;
    }
    w.so = w8 ? (float*)(base + L.so) : nullptr;
    if ((st = put_matrix(*m, weights[wi++], H, Q, base + L.wo, wd::kPackPlain, nullptr,
                         (float*)w.so)) != WD_OK)
      return fail_free(st);
    if ((st = copy(weights[wi++], H * e, base + L.ffn_norm)) != WD_OK) return fail_free(st);
    {
      const void* wg = weights[wi++];
      const void* wu = weights[wi++];
      w.sgu = w8 ? (float*)(base + L.sgu) : nullptr;
      if ((st = put_matrix(*m, wg, 2 * F, H, base + L.wgu, wd::kPackGateUp, wu, (float*)w.sgu)) !=
          WD_OK)
        return fail_free(st);
    }
    w.sd = w8 ? (float*)(base + L.sd) : nullptr;
    if ((st = put_matrix(*m, weights[wi++], H, F, base + L.wd, wd::kPackPlain, nullptr,
                         (float*)w.sd)) != WD_OK)
      return fail_free(st);
    w.attn_norm = base + L.attn_norm;
    w.wqkv = base + L.wqkv;
    w.wo = base + L.wo;
    w.ffn_norm = base + L.ffn_norm;
    w.wgu = base + L.wgu;
    w.wd = base + L.wd;
    m->layers.push_back(w);
  }
  if ((st = copy(weights[wi++], H * e, base + lay.final_norm)) != WD_OK) return fail_free(st);
  m->final_norm = base + lay.final_norm;
  m->slm = w8 ? (float*)(base + lay.slm) : nullptr;
  if ((st = put_matrix(*m, weights[wi++], cfg->vocab, H, base + lay.lm, wd::kPackPlain, nullptr,
                       (float*)m->slm)) != WD_OK)
    return fail_free(st);
  m->lm = base + lay.lm;
  if (hipStreamSynchronize(m->stream) != hipSuccess) {
    delete m;
    return fail(WD_ERR_DEVICE, "weight packing failed");
  }
  *out = m;
  return WD_OK;
}

void wd_free_model(wd_model* m) {
  if (!m) return;
  for (hipEvent_t e : m->ev) (void)hipEventDestroy(e);
  delete m;
}

wd_status wd_debug_weight_row(const wd_model* m, int32_t tensor, int32_t row, float* values,
                              float* scale) {
  if (!m || !values || !scale) return fail(WD_ERR_INVALID_ARG, "NULL argument");
  const wd_model_config& c = m->cfg;
  if (c.dtype != WD_DTYPE_BF16) return fail(WD_ERR_UNSUPPORTED, "fp32 weights are not packed");
  const auto specs = tensor_specs(c);
  if (tensor < 0 || tensor >= (int32_t)specs.size())
    return fail(WD_ERR_INVALID_ARG, "tensor %d out of range", tensor);
  const std::string name = specs[tensor].name;
  const std::string leaf = name.substr(name.rfind('.') + 1);
  const long H = c.hidden, Q = (long)c.n_heads * c.head_dim, KV = (long)c.n_kv_heads * c.head_dim,
             F = c.ffn;
  int layer = -1;
  if (name.compare(0, 7, "layers.") == 0) layer = std::stoi(name.substr(7));
  // the packed matrix holding the tensor, its K, and the packed row of `row`
  const char* base = nullptr;
  const float* sc = nullptr;
  long K = H, rows = 0, prow = 0;
  auto rope_row = [](long r) {  // kPackRopePair: dim d of head h
    const long h = r >> 7, d = r & 127;
    return h * 128 + ((d & 63) >> 3) * 16 + (d >= 64 ? 8 : 0) + (d & 7);
  };
  const bool w8 = c.weight_fp8 != 0;
  const size_t ew = w8 ? 1 : 2;
  if (layer >= 0) {
    const LayerW& w = m->layers[layer];
    if (leaf == "wq" || leaf == "wk" || leaf == "wv") {
      const long off = leaf == "wq" ? 0 : leaf == "wk" ? Q : Q + KV;
      rows = leaf == "wq" ? Q : KV;
      if (row < 0 || row >= rows) return fail(WD_ERR_INVALID_ARG, "row %d out of range", row);
      base = (const char*)w.wqkv + off * H * ew;
      sc = w.sqkv ? w.sqkv + off : nullptr;
      prow = rope_row(row);
    } else if (leaf == "wo") {
      rows = H, K = Q, base = (const char*)w.wo, sc = w.so, prow = row;
    } else if (leaf == "wg" || leaf == "wu") {
      rows = F, base = (const char*)w.wgu, sc = w.sgu;
      prow = (row >> 3) * 16 + (leaf == "wu" ? 8 : 0) + (row & 7);
    } else if (leaf == "wd") {
      rows = H, K = F, base = (const char*)w.wd, sc = w.sd, prow = row;
    }
  } else if (leaf == "lm_head") {
    rows = c.vocab, base = (const char*)m->lm, sc = m->slm, prow = row;
  }
  if (!base) return fail(WD_ERR_INVALID_ARG, "tensor %d (%s) is not a projection matrix", tensor,
                         name.c_str());
  if (row < 0 || row >= rows) return fail(WD_ERR_INVALID_ARG, "row %d out of range", row);
  // one 16-row group is contiguous: K/32 bf16 fragments, or K/64 fp8 fragments, of 1 KB
  const long g = prow >> 4, r = prow & 15, frags = w8 ? K / 64 : K / 32;
  std::vector<uint8_t> buf((size_t)frags * 1024);
  WD_HIP(hipStreamSynchronize(m->stream));
  WD_HIP(hipMemcpy(buf.data(), base + (size_t)g * frags * 1024, buf.size(), hipMemcpyDeviceToHost));
  for (long f = 0; f < frags; ++f)
    for (int q = 0; q < 4; ++q) {
      const uint8_t* lane = buf.data() + (size_t)f * 1024 + (size_t)(q * 16 + r) * 16;
      for (int j = 0; j < 8; ++j) {
        if (w8) {
          values[f * 64 + q * 8 + j] = e4m3_to_float(lane[j]);
          values[f * 64 + 32 + q * 8 + j] = e4m3_to_float(lane[8 + j]);
        } else {
          uint16_t h;
          memcpy(&h, lane + 2 * j, 2);
          const uint32_t u = (uint32_t)h << 16;
          memcpy(&values[f * 32 + q * 8 + j], &u, 4);
        }
      }
    }
  *scale = 1.f;
  if (sc) WD_HIP(hipMemcpy(scale, sc + prow, 4, hipMemcpyDeviceToHost));
  return WD_OK;
}

wd_status wd_profile_enable(wd_model* m, int32_t enable) {
  if (!m) return fail(WD_ERR_INVALID_ARG, "model is NULL");
  m->profile = enable != 0;
  m->n_rec = 0;
  m->rec_bytes.clear();
  m->rec_flops.clear();
  m->rec_kind.clear();
  return WD_OK;
}

wd_status wd_measure_peaks(wd_model* m, double* mfma_bf16_tflops, double* hbm_read_gbs) {
  if (!m || !mfma_bf16_tflops || !hbm_read_gbs) return fail(WD_ERR_INVALID_ARG, "NULL argument");
  if (hipSetDevice(m->device) != hipSuccess) return fail(WD_ERR_DEVICE, "hipSetDevice failed");
  WD_HIP(hipStreamSynchronize(m->stream));
  WD_HIP(wd::measure_peaks(m->stream, mfma_bf16_tflops, hbm_read_gbs));
  return WD_OK;
}

wd_status wd_profile_read(wd_model* m, int32_t kernel, int64_t* launches, double* total_ms,
                          double* alg_bytes, double* alg_flops) {
  if (!m) return fail(WD_ERR_INVALID_ARG, "model is NULL");
  if (kernel < WD_PROF_ALL || kernel > WD_PROF_ATTN)
    return fail(WD_ERR_INVALID_ARG, "unknown kernel class %d", kernel);
  WD_HIP(hipStreamSynchronize(m->stream));
  int64_t n = 0;
  double ms = 0.0, by = 0.0, fl = 0.0;
  for (size_t i = 0; i < m->n_rec; ++i) {
    if (kernel != WD_PROF_ALL && m->rec_kind[i] != kernel) continue;
    float t = 0.f;
    WD_HIP(hipEventElapsedTime(&t, m->ev[2 * i], m->ev[2 * i + 1]));
    ++n;
    ms += t;
    by += m->rec_bytes[i];
    fl += m->rec_flops[i];
  }
  if (launches) *launches = n;
  if (total_ms) *total_ms = ms;
  if (alg_bytes) *alg_bytes = by;
  if (alg_flops) *alg_flops = fl;
  return WD_OK;
}

}  // extern "C"

// -- one generation -----------------------------------------------------------------------
struct wd_seq {
  wd_model* m = nullptr;
  wd_window_config win{};
  int B = 0, G = 0;
  long T = 0;
  int Smax = 0;
  std::vector<int> np, S, off, ctx;
  Counts cnt;
  int t = 0;
  bool refreshed = false;
  int mode = 0;  // 0 = not started, 1 = windowed, 2 = full sequence
  int last_nA = 0;
  // logits of the last step's active rows: written only on request when the
  // LM head reduces its tiles to the confidence inputs itself
  bool keep_logits = false, logits_valid = false;
  // adaptive termination
  int eos_id = -1;
  std::vector<Track> tr;
  // device buffers (carved from the caller's workspace)
  int32_t *x, *seq_len, *row_tok, *row_pos, *row_seq, *row_out, *act_pos, *act_tok, *sel_pos,
      *sel_tok, *err;
  uint8_t *dec, *dec0, *decp;
  float *rope, *h, *C, *logits, *act_conf, *sel_conf, *dbg, *attn_part, *conf_scratch;
  long attn_part_floats = 0;
  void *kc, *vc, *a, *q, *o, *sw, *a_act;
  long M_max = 0, A_max = 0;
  size_t C_floats = 0;
  // pinned host staging for step results
  int32_t* h_buf = nullptr;
};

namespace {

struct SeqLayout {
  size_t total = 0;
  size_t x, seq_len, dec, dec0, decp, kc, vc, rope, h, a, q, o, sw, C, row_tok, row_pos, row_seq, row_out,
      act_pos, act_tok, act_conf, a_act, logits, sel_pos, sel_tok, sel_conf, err, dbg, attn_part,
      conf_scratch;
  long M_max, A_max, attn_part_floats;
  size_t C_floats;
};

int gemm_splits(const wd_model_config& c, int M, int N, int K) {
  if (c.dtype != WD_DTYPE_BF16) return 1;
  return wd::plan_gemm_bf16(M, N, K, c.weight_fp8 != 0).splits;
}

SeqLayout seq_layout(const wd_model& m, const wd_window_config& w, int B, long T, int Smax, int G) {
  const wd_model_config& c = m.cfg;
  const size_t e = m.esz;
  const long H = c.hidden, Q = (long)c.n_heads * c.head_dim, KVd = (long)c.n_kv_heads * c.head_dim,
             F = c.ffn;
  SeqLayout s;
  s.M_max = T;
  s.A_max = std::max<long>((long)B * w.n_active, (long)B * G);
  size_t cf = 0;
  const int shapes[4][2] = {{m.qkv_n, (int)H}, {(int)H, (int)Q}, {(int)(2 * F), (int)H}, {(int)H, (int)F}};
  for (long M = 1; M <= s.M_max; ++M)
    for (auto& sh : shapes) cf = std::max(cf, (size_t)gemm_splits(c, (int)M, sh[0], sh[1]) * M * sh[0]);
  s.C_floats = cf;
  size_t o = 0;
  auto take = [&](size_t bytes) {
    const size_t at = o;
    o += align256(bytes);
    return at;
  };
  s.x = take(T * 4);
  s.seq_len = take(B * 4);
  s.dec = take(T);
  s.dec0 = take(T);
  s.decp = take(T);
  s.kc = take((size_t)c.n_layers * KVd * T * e);
  s.vc = take((size_t)c.n_layers * KVd * T * e);
  s.rope = take((size_t)Smax * c.head_dim * 4);
  s.h = take(s.M_max * H * 4);
  s.a = take(s.M_max * H * e);
  s.q = take(s.M_max * Q * e);
  s.o = take(s.M_max * Q * e);
  s.sw = take(s.M_max * F * e);
  s.C = take(cf * 4);
  s.row_tok = take(s.M_max * 4);
  s.row_pos = take(s.M_max * 4);
  s.row_seq = take(s.M_max * 4);
  s.row_out = take(s.M_max * 4);
  s.act_pos = take(s.A_max * 4);
  s.act_tok = take(s.A_max * 4);
  s.act_conf = take(s.A_max * 4);
  s.a_act = take(s.A_max * H * e);
  s.logits = take((size_t)s.A_max * c.vocab * 4);
  s.sel_pos = take((size_t)B * w.unmask_per_step * 4);
  s.sel_tok = take((size_t)B * w.unmask_per_step * 4);
  s.sel_conf = take((size_t)B * w.unmask_per_step * 4);
  s.err = take(4);
  s.dbg = take((size_t)T * c.head_dim * 4);
  // split-KV partials sized for up to 16 splits of a normal step's rows
  const long rows_normal = std::min<long>(s.M_max, (long)B * (w.n_active + (long)w.unmask_per_step *
                                                                           w.refresh_every));
  s.attn_part_floats = 16L * rows_normal * c.n_heads * (c.head_dim + 2);
  s.attn_part = take(s.attn_part_floats * 4);
  // confidence partials: kConfChunks per row, or one per 64-entry vocabulary
  // tile when the LM head reduces them itself
  s.conf_scratch = take((size_t)3 * s.A_max * std::max<long>(wd::kConfChunks, c.vocab / 64) * 4);
  s.total = o;
  return s;
}

bool win_valid(const wd_window_config* w, std::string* why) {
  if (!w) {
    *why = "NULL window config";
    return false;
  }
  if (w->n_active < 1 || w->n_buffer < 0 || w->refresh_every < 1 || w->unmask_per_step < 1) {
    *why = "need n_active >= 1, n_buffer >= 0, refresh_every >= 1, unmask_per_step >= 1";
    return false;
  }
  if (w->n_active > 64) {
    *why = "n_active above 64 is not supported";
    return false;
  }
  if (w->stop_at_eos != 0 && w->stop_at_eos != 1) {
    *why = "stop_at_eos must be 0 or 1";
    return false;
  }
  if (w->buffer_refresh != 0 && w->buffer_refresh != 1) {
    *why = "buffer_refresh must be 0 or 1";
    return false;
  }
  return true;
}

bool seq_args_valid(const wd_model* m, const wd_window_config* w, int32_t batch,
                    const int32_t* prompt_lens, int32_t gen_len, std::string* why) {
  if (!m) {
    *why = "model is NULL";
    return false;
  }
  if (!win_valid(w, why)) return false;
  if (batch < 1 || batch > WD_MAX_BATCH) {
    *why = "batch must be in [1, 64]";
    return false;
  }
  if (!prompt_lens) {
    *why = "prompt_lens is NULL";
    return false;
  }
  if (gen_len < 1) {
    *why = "gen_len must be >= 1";
    return false;
  }
  long T = 0;
  for (int b = 0; b < batch; ++b) {
    if (prompt_lens[b] < 0) {
      *why = "negative prompt length";
      return false;
    }
    T += prompt_lens[b] + gen_len;
  }
  if (T > (1L << 24)) {
    *why = "too many positions";
    return false;
  }
  if (w->stop_at_eos && (w->eos_id < 0 || w->eos_id >= m->cfg.vocab || w->eos_id == m->cfg.mask_id)) {
    *why = "with stop_at_eos, eos_id must be a token id other than mask_id";
    return false;
  }
  if (m->cfg.dtype == WD_DTYPE_F32) {
    for (int b = 0; b < batch; ++b)
      if (prompt_lens[b] + gen_len > 16384) {
        *why = "fp32 models support sequences of at most 16384 positions";
        return false;
      }
  }
  return true;
}

// ---- the layer stack over a row set ----------------------------------------------------------
struct Rows {
  int M;
  int n_act;  // active rows per sequence (compact index b * n_act + rank)
  WdStepGeom g;
};

// Event pair for one GEMM launch when kernel timing is on (null otherwise);
// the launch records both events from its own dispatch.
wd_status profile_begin(wd_model& m, hipEvent_t* e0, hipEvent_t* e1) {
  *e0 = *e1 = nullptr;
  if (!m.profile) return WD_OK;
  if (m.n_rec >= (1u << 20)) return fail(WD_ERR_OUT_OF_MEMORY, "too many unread timing records");
  while (m.ev.size() < 2 * (m.n_rec + 1)) {
    hipEvent_t e;
    WD_HIP(hipEventCreate(&e));
    m.ev.push_back(e);
  }
  *e0 = m.ev[2 * m.n_rec];
  *e1 = m.ev[2 * m.n_rec + 1];
  return WD_OK;
}

// out_bytes: what the launch writes (fp32 M x N when negative).
wd_status profile_end(wd_model& m, int kind, int M, int N, int K, size_t esz,
                      double out_bytes = -1) {
  if (!m.profile) return WD_OK;
  // weights: esz bytes each, or one byte plus a float32 scale per row with fp8
  const double wbytes = m.cfg.weight_fp8 ? (double)N * K + 4.0 * N : (double)N * K * esz;
  if (out_bytes < 0) out_bytes = (double)M * N * 4;
  m.rec_bytes.push_back(wbytes + (double)M * K * esz + out_bytes);
  m.rec_flops.push_back(2.0 * M * N * K);
  m.rec_kind.push_back(kind);
  m.n_rec++;
  return WD_OK;
}

// One attention unit: K and V of [0, c) per sequence, q rows in, output rows out.
wd_status profile_attention(wd_model& m, const WdStepGeom& g) {
  if (!m.profile) return WD_OK;
  const wd_model_config& c = m.cfg;
  double bytes = 0, flops = 0;
  for (int b = 0; b < g.batch; ++b) {
    if (g.nrows[b] <= 0) continue;
    bytes += 2.0 * g.ctx[b] * c.n_kv_heads * c.head_dim * m.esz;
    bytes += 2.0 * g.nrows[b] * c.n_heads * c.head_dim * m.esz;
    flops += 4.0 * g.nrows[b] * g.ctx[b] * c.n_heads * c.head_dim;
  }
  if (bytes == 0) return WD_OK;  // no rows: nothing was launched, the events stay unused
  m.rec_bytes.push_back(bytes);
  m.rec_flops.push_back(flops);
  m.rec_kind.push_back(WD_PROF_ATTN);
  m.n_rec++;
  return WD_OK;
}

template <typename T>
wd_status gemm_launch(wd_seq* s, const T* X, int ldx, const void* W, const float* wsc, float* C,
                      int M, int N, int K, int max_splits, int* splits, int* kind, hipEvent_t e0,
                      hipEvent_t e1) {
  const wd_model& m = *s->m;
  if (m.cfg.dtype == WD_DTYPE_BF16) {
    const wd::GemmPlan p = wd::plan_gemm_bf16(M, N, K, wsc != nullptr, max_splits);
    if ((size_t)p.splits * M * N > s->C_floats && C == s->C)
      return fail(WD_ERR_DEVICE, "internal: partial buffer too small");
    WD_HIP(wd::gemm_bf16((const uint16_t*)X, ldx, W, C, M, N, K, p, m.stream, e0, e1, wsc));
    *splits = p.splits;
    *kind = p.mf == 8 ? WD_PROF_GEMM_TILED : WD_PROF_GEMM_ROWS;
  } else {
    WD_HIP(wd::gemm_f32((const float*)X, ldx, (const float*)W, C, M, N, K, m.stream, e0, e1));
    *splits = 1;
    *kind = WD_PROF_GEMM_F32;
  }
  return WD_OK;
}

template <typename T>
wd_status gemm(wd_seq* s, const T* X, int ldx, const void* W, const float* wsc, float* C, int M,
               int N, int K, int max_splits, int* splits) {
  wd_model& m = *s->m;
  int kind = WD_PROF_ALL;
  hipEvent_t e0, e1;
  WD_TRY(profile_begin(m, &e0, &e1));
  WD_TRY(gemm_launch<T>(s, X, ldx, W, wsc, C, M, N, K, max_splits, splits, &kind, e0, e1));
  return profile_end(m, kind, M, N, K, m.esz);
}

// The few-row products that carry their own epilogue (bf16, at most 64 rows,
// wide enough for one workgroup per 64 features to fill the GPU).
bool fused_rows(const wd_model& m, int M, int N, int K, int epi) {
  return m.cfg.dtype == WD_DTYPE_BF16 && wd::fused_rows_ok(M, N, K, wd::fused_max_rows(epi));
}

wd_model& m_mut(wd_seq* s) { return *s->m; }

// Which kernels a layer's products take at M rows.  Q/K/V: 0 = the fused
// few-row kernel, 1 = the many-row kernel with the Q/K/V epilogue (no K
// split); both write q and the cache themselves; 2 = split-K partials and
// k_qkv_epilogue.
int qkv_path(const wd_model& m, int M) {
  if (fused_rows(m, M, m.qkv_n, m.cfg.hidden, wd::kEpiQkv)) return 0;
  if (m.cfg.dtype == WD_DTYPE_BF16 && !m.cfg.weight_fp8) {
    const wd::GemmPlan gp = wd::plan_gemm_bf16(M, m.qkv_n, m.cfg.hidden);
    if (gp.dma_mfw && gp.splits == 1) return 1;
  }
  return 2;
}
// gate/up: 0 = the fused few-row kernel with SwiGLU, 1 = the many-row kernel
// with SwiGLU in its epilogue (no K split), 2 = split-K partials and k_swiglu.
int gateup_path(const wd_model& m, int M) {
  const int F = m.cfg.ffn, H = m.cfg.hidden;
  if (fused_rows(m, M, 2 * F, H, wd::kEpiSwiGlu)) return 0;
  if (m.cfg.dtype == WD_DTYPE_BF16 && !m.cfg.weight_fp8) {
    const wd::GemmPlan gp = wd::plan_gemm_bf16(M, 2 * F, H);
    if (gp.dma_mfw && gp.splits == 1) return 1;
  }
  return 2;
}

// Most floats of split-K partials one pass of the layer stack over M rows
// writes (O and down always write them; Q/K/V and gate/up unless fused).
size_t step_partial_floats(const wd_model& m, int M) {
  const wd_model_config& c = m.cfg;
  const int H = c.hidden, Q = c.n_heads * c.head_dim, F = c.ffn;
  auto part = [&](int N, int K) { return (size_t)gemm_splits(c, M, N, K) * M * N; };
  size_t v = std::max(part(H, Q), part(H, F));
  if (qkv_path(m, M) == 2) v = std::max(v, part(m.qkv_n, H));
  if (gateup_path(m, M) == 2) v = std::max(v, part(2 * F, H));
  return v;
}

template <typename T>
wd_status run_layers(wd_seq* s, const Rows& r) {
  const wd_model& m = *s->m;
  const wd_model_config& c = m.cfg;
  hipStream_t st = m.stream;
  const int M = r.M, H = c.hidden, Q = c.n_heads * c.head_dim, F = c.ffn;
  const long KVd = (long)c.n_kv_heads * c.head_dim;
  T* a = (T*)s->a;
  T* q = (T*)s->q;
  T* o = (T*)s->o;
  T* sw = (T*)s->sw;
  WD_HIP(wd::embed_norm<T>(s->x, s->row_tok, (const T*)m.emb, (const T*)m.layers[0].attn_norm,
                           c.rms_eps, s->h, a, M, H, st));
  int S;
  for (int l = 0; l < c.n_layers; ++l) {
    const LayerW& w = m.layers[l];
    T* kc = (T*)s->kc + (size_t)l * KVd * s->T;
    T* vc = (T*)s->vc + (size_t)l * KVd * s->T;
    const int qp = qkv_path(m, M);
    if (qp == 0) {
      hipEvent_t e0, e1;
      WD_TRY(profile_begin(m_mut(s), &e0, &e1));
      WD_HIP(wd::gemm_bf16_qkv_fused((const uint16_t*)a, H, w.wqkv, M, m.qkv_n, H,
                                     (const uint16_t*)w.bqkv, s->rope, s->row_pos, s->row_tok,
                                     c.n_heads, c.n_kv_heads, (uint16_t*)q, (uint16_t*)kc,
                                     (uint16_t*)vc, s->T, st, e0, e1, w.sqkv));
      WD_TRY(profile_end(m_mut(s), WD_PROF_GEMM_ROWS, M, m.qkv_n, H, m.esz,
                         (double)M * m.qkv_n * m.esz));
    } else if (qp == 1) {
      // many rows without a K split: bias, RoPE and the q / K/V stores in the
      // GEMM's epilogue
      const wd::GemmPlan gp = wd::plan_gemm_bf16(M, m.qkv_n, H);
      const wd::QkvOut qo{(const uint16_t*)w.bqkv, s->rope, s->row_pos, s->row_tok,
                          (uint16_t*)q, (uint16_t*)kc, (uint16_t*)vc, s->T, c.n_heads,
                          c.n_kv_heads};
      hipEvent_t e0, e1;
      WD_TRY(profile_begin(m_mut(s), &e0, &e1));
      WD_HIP(wd::gemm_bf16_qkv_tiles((const uint16_t*)a, H, w.wqkv, M, m.qkv_n, H, gp, qo, st, e0,
                                     e1));
      WD_TRY(profile_end(m_mut(s), WD_PROF_GEMM_TILED, M, m.qkv_n, H, m.esz,
                         (double)M * m.qkv_n * m.esz));
    } else {
      WD_TRY(gemm<T>(s, a, H, w.wqkv, w.sqkv, s->C, M, m.qkv_n, H, 1 << 20, &S));
      WD_HIP(wd::qkv_epilogue<T>(s->C, S, M, (const T*)w.bqkv, s->rope, s->row_pos, s->row_tok,
                                 c.n_heads, c.n_kv_heads, c.head_dim, q, kc, vc, s->T, st));
    }
    if (c.dtype == WD_DTYPE_BF16) {
      hipEvent_t e0, e1;
      WD_TRY(profile_begin(m_mut(s), &e0, &e1));
      WD_HIP(wd::attention_bf16((const uint16_t*)q, (const uint16_t*)kc, (const uint16_t*)vc, s->T,
                                (uint16_t*)o, r.g, c.n_heads, c.n_kv_heads, c.head_dim,
                                s->attn_part, s->attn_part_floats, st, e0, e1));
      WD_TRY(profile_attention(m_mut(s), r.g));
    } else {
      WD_HIP(wd::attention_f32((const float*)q, (const float*)kc, (const float*)vc, s->T,
                               (float*)o, s->row_seq, M, r.g, c.n_heads, c.n_kv_heads, c.head_dim,
                               st));
    }
    WD_TRY(gemm<T>(s, o, Q, w.wo, w.so, s->C, M, H, Q, 1 << 20, &S));
    WD_HIP(wd::residual_norm<T>(s->h, s->C, S, M, H, (const T*)w.ffn_norm, c.rms_eps, a, nullptr, st));
    const int gu = gateup_path(m, M);
    if (gu == 0) {
      hipEvent_t e0, e1;
      WD_TRY(profile_begin(m_mut(s), &e0, &e1));
      WD_HIP(wd::gemm_bf16_swiglu_fused((const uint16_t*)a, H, w.wgu, M, F, H, (uint16_t*)sw, st,
                                        e0, e1, w.sgu));
      WD_TRY(profile_end(m_mut(s), WD_PROF_GEMM_ROWS, M, 2 * F, H, m.esz, (double)M * F * m.esz));
    } else if (gu == 1) {
      // many rows without a K split: SwiGLU in the GEMM's epilogue
      const wd::GemmPlan gp = wd::plan_gemm_bf16(M, 2 * F, H);
      hipEvent_t e0, e1;
      WD_TRY(profile_begin(m_mut(s), &e0, &e1));
      WD_HIP(wd::gemm_bf16_swiglu_dma((const uint16_t*)a, H, w.wgu, (uint16_t*)sw, M, F, H, gp, st,
                                      e0, e1));
      WD_TRY(profile_end(m_mut(s), WD_PROF_GEMM_TILED, M, 2 * F, H, m.esz, (double)M * F * m.esz));
    } else {
      WD_TRY(gemm<T>(s, a, H, w.wgu, w.sgu, s->C, M, 2 * F, H, 1 << 20, &S));
      WD_HIP(wd::swiglu<T>(s->C, S, M, F, sw, st));
    }
    WD_TRY(gemm<T>(s, sw, F, w.wd, w.sd, s->C, M, H, F, 1 << 20, &S));
    if (l + 1 < c.n_layers) {
      WD_HIP(wd::residual_norm<T>(s->h, s->C, S, M, H, (const T*)m.layers[l + 1].attn_norm,
                                  c.rms_eps, a, nullptr, st));
    } else {
      WD_HIP(wd::residual_norm<T>(s->h, s->C, S, M, H, (const T*)m.final_norm, c.rms_eps,
                                  (T*)s->a_act, s->row_out, st));
    }
  }
  return WD_OK;
}

// r.g.mode / r.g.nact give each sequence's rows; r.n_act is the compact stride.
wd_status forward(wd_seq* s, const Rows& r) {
  WD_HIP(wd::build_rows(s->dec, s->dec0, s->decp, r.n_act, r.g, s->row_tok, s->row_pos,
                        s->row_seq, s->row_out, s->act_pos, s->err, s->m->stream));
  if (s->m->cfg.dtype == WD_DTYPE_BF16) return run_layers<uint16_t>(s, r);
  return run_layers<float>(s, r);
}

WdStepGeom base_geom(const wd_seq* s) {
  WdStepGeom g;
  memset(&g, 0, sizeof(g));
  g.batch = s->B;
  for (int b = 0; b < s->B; ++b) {
    g.off[b] = s->off[b];
    g.ctx[b] = s->ctx.empty() ? s->S[b] : s->ctx[b];
    g.mode[b] = -1;
    g.end[b] = s->tr.empty() ? s->S[b] : s->tr[b].end;
  }
  return g;
}

// LM head on the compact active rows, confidence, top-k decode.  rows: the
// step's per-sequence modes and active counts (NULL: every sequence has n_act
// active positions), which the decode checks its picks against.
wd_status decide(wd_seq* s, int n_act, const WdStepGeom* rows = nullptr) {
  const wd_model& m = *s->m;
  const wd_model_config& c = m.cfg;
  const int n = s->B * n_act;
  int S;
  if (fused_rows(m, n, c.vocab, c.hidden, wd::kEpiConf)) {
    // the LM head reduces each 64-entry vocabulary tile to the confidence
    // inputs itself; the logits reach memory only when asked for
    const int n_tiles = c.vocab / 64;
    float* pmax = s->conf_scratch;
    int* pidx = (int*)(pmax + (size_t)n * n_tiles);
    float* psum = pmax + 2 * (size_t)n * n_tiles;
    hipEvent_t e0, e1;
    WD_TRY(profile_begin(m_mut(s), &e0, &e1));
    WD_HIP(wd::gemm_bf16_lmhead_conf((const uint16_t*)s->a_act, c.hidden, m.lm, n, c.vocab,
                                     c.hidden, c.mask_id, s->keep_logits ? s->logits : nullptr,
                                     pmax, pidx, psum, m.stream, e0, e1, m.slm));
    WD_TRY(profile_end(m_mut(s), WD_PROF_GEMM_ROWS, n, c.vocab, c.hidden, m.esz,
                       12.0 * n * n_tiles + (s->keep_logits ? 4.0 * n * c.vocab : 0.0)));
    WD_HIP(wd::confidence_tiles(pmax, pidx, psum, n, n_tiles, s->act_tok, s->act_conf, m.stream));
    s->logits_valid = s->keep_logits;
  } else {
    if (c.dtype == WD_DTYPE_BF16)
      WD_TRY(gemm<uint16_t>(s, (const uint16_t*)s->a_act, c.hidden, m.lm, m.slm, s->logits, n,
                            c.vocab, c.hidden, 1, &S));
    else
      WD_TRY(gemm<float>(s, (const float*)s->a_act, c.hidden, m.lm, nullptr, s->logits, n,
                         c.vocab, c.hidden, 1, &S));
    WD_HIP(wd::confidence(s->logits, n, c.vocab, c.mask_id, s->act_tok, s->act_conf,
                          s->conf_scratch, m.stream));
    s->logits_valid = true;
  }
  WdStepGeom g = base_geom(s);
  for (int b = 0; b < s->B; ++b) {
    g.mode[b] = rows ? rows->mode[b] : 0;
    g.nact[b] = rows ? rows->nact[b] : n_act;
  }
  WD_HIP(wd::select_update(s->act_pos, s->act_tok, s->act_conf, n_act, s->win.unmask_per_step, g,
                           s->seq_len, s->x, s->dec, s->sel_pos, s->sel_tok, s->sel_conf, s->err,
                           m.stream));
  s->last_nA = n_act;
  return WD_OK;
}

wd_status do_slide(wd_seq* s) {
  s->cnt.start_phase();
  for (int b = 0; b < s->B; ++b) s->ctx[b] = s->cnt.ctx(s->S[b]);
  s->refreshed = false;
  WdStepGeom g = base_geom(s);
  for (int b = 0; b < s->B; ++b) g.mode[b] = 0;
  WD_HIP(wd::slide(s->dec, s->dec0, s->decp, s->Smax, s->cnt.E, g, s->seq_len, s->err,
                   s->m->stream));
  return WD_OK;
}

wd_status do_refresh(wd_seq* s) {
  Rows r;
  r.g = base_geom(s);
  r.n_act = s->cnt.n_active();
  const bool buffer = s->win.buffer_refresh && s->cnt.phases > 1;
  int row = 0;
  for (int b = 0; b < s->B; ++b) {
    r.g.mode[b] = buffer ? 3 : 0;
    r.g.nact[b] = r.n_act;
    r.g.row0[b] = row;
    r.g.nrows[b] = s->cnt.refresh_rows(s->ctx[b], s->win.buffer_refresh);
    row += r.g.nrows[b];
  }
  r.M = row;
  WD_TRY(forward(s, r));
  s->refreshed = true;
  return WD_OK;
}

wd_status do_normal(wd_seq* s) {
  Rows r;
  r.g = base_geom(s);
  r.n_act = s->cnt.n_active();
  const int nO = r.n_act + s->cnt.dp;
  for (int b = 0; b < s->B; ++b) {
    r.g.mode[b] = 1;
    r.g.nact[b] = r.n_act;
    r.g.row0[b] = b * nO;
    r.g.nrows[b] = nO;
  }
  r.M = s->B * nO;
  return forward(s, r);
}

// One step under adaptive termination, windowed (full = false) or full
// sequence: each unfinished sequence takes its own kind of step, then the
// step's decisions are read back into the host tracks.
wd_status step_tracked(wd_seq* s, wd_step_out* out, bool full) {
  const int B = s->B, E = s->win.n_active + s->win.n_buffer, k = s->win.unmask_per_step;
  Rows r;
  r.g = base_geom(s);
  bool any_slide = false, any_refresh = false;
  int stride = 1, row = 0;
  for (int b = 0; b < B; ++b) {
    Track& t = s->tr[b];
    int mode = -1, na = 0, rows = 0, ctx = 0;
    if (!t.done()) {
      if (full) {
        mode = 2;
        ctx = t.end;
        na = t.live_undecoded();
        rows = ctx;
      } else {
        if (t.phase_due(s->win.refresh_every)) {
          t.slide(E);
          any_slide = true;
          mode = 0;
          rows = t.c;
        } else {
          mode = 1;
        }
        ctx = t.ctx();
        na = t.n_active(s->win.n_active);
        if (mode == 1) rows = na + t.n_phase_decoded();
      }
    }
    any_refresh |= mode == 0 || mode == 2;
    s->ctx[b] = ctx;
    r.g.ctx[b] = ctx;
    r.g.mode[b] = mode;
    r.g.nact[b] = na;
    r.g.row0[b] = row;
    r.g.nrows[b] = rows;
    row += rows;
    stride = std::max(stride, na);
  }
  if (any_slide) {
    WdStepGeom g = r.g;
    for (int b = 0; b < B; ++b) g.ctx[b] = s->tr[b].c;
    WD_HIP(wd::slide(s->dec, s->dec0, s->decp, s->Smax, E, g, s->seq_len, s->err, s->m->stream));
  }
  r.M = row;
  r.n_act = stride;
  WD_TRY(forward(s, r));
  WD_TRY(decide(s, stride, &r.g));
  const int step = s->t;
  s->t++;
  // the decisions, read back every step
  hipStream_t st = s->m->stream;
  WD_HIP(hipMemcpyAsync(s->h_buf, s->sel_pos, B * k * 4, hipMemcpyDeviceToHost, st));
  WD_HIP(hipMemcpyAsync(s->h_buf + B * k, s->sel_tok, B * k * 4, hipMemcpyDeviceToHost, st));
  WD_HIP(hipMemcpyAsync(s->h_buf + 2 * B * k, s->sel_conf, B * k * 4, hipMemcpyDeviceToHost, st));
  WD_HIP(hipMemcpyAsync(s->h_buf + 3 * B * k, s->err, 4, hipMemcpyDeviceToHost, st));
  WD_HIP(hipStreamSynchronize(st));
  if (s->h_buf[3 * B * k] != 0)
    return fail(WD_ERR_DEVICE, "device bookkeeping disagrees with the schedule (code %d)",
                s->h_buf[3 * B * k]);
  int nsel = 0;
  for (int b = 0; b < B; ++b) {
    Track& t = s->tr[b];
    if (r.g.mode[b] < 0) continue;
    // checked against the state before the step (a step may decode an <eos>
    // and, in the same step, a later position), then applied
    int n = 0;
    for (int i = 0; i < k; ++i) {
      const int p = s->h_buf[b * k + i];
      if (p < 0) continue;
      if (p >= t.end || t.dec[p])
        return fail(WD_ERR_DEVICE, "device decoded position %d of sequence %d out of turn", p, b);
      ++n;
    }
    for (int i = 0; i < k; ++i) {
      const int p = s->h_buf[b * k + i];
      if (p >= 0) t.apply(p, s->h_buf[B * k + b * k + i], s->eos_id);
    }
    if (n != std::min(k, r.g.nact[b]))
      return fail(WD_ERR_DEVICE, "sequence %d decoded %d positions, expected %d", b, n,
                  std::min(k, r.g.nact[b]));
    nsel = std::max(nsel, n);
    if (!full) t.j++;
  }
  if (out) {
    out->step = step;
    out->is_refresh = any_refresh ? 1 : 0;
    out->n_rows = row;
    out->n_selected = nsel;
    if (out->positions) memcpy(out->positions, s->h_buf, B * k * 4);
    if (out->tokens) memcpy(out->tokens, s->h_buf + B * k, B * k * 4);
    if (out->conf) memcpy(out->conf, s->h_buf + 2 * B * k, B * k * 4);
  }
  return WD_OK;
}

bool all_done(const wd_seq* s) {
  for (const Track& t : s->tr)
    if (!t.done()) return false;
  return true;
}

wd_status fetch_out(wd_seq* s, wd_step_out* out, int step, int refresh, int rows, int nsel) {
  const int k = s->win.unmask_per_step, B = s->B;
  hipStream_t st = s->m->stream;
  WD_HIP(hipMemcpyAsync(s->h_buf, s->sel_pos, B * k * 4, hipMemcpyDeviceToHost, st));
  WD_HIP(hipMemcpyAsync(s->h_buf + B * k, s->sel_tok, B * k * 4, hipMemcpyDeviceToHost, st));
  WD_HIP(hipMemcpyAsync(s->h_buf + 2 * B * k, s->sel_conf, B * k * 4, hipMemcpyDeviceToHost, st));
  WD_HIP(hipMemcpyAsync(s->h_buf + 3 * B * k, s->err, 4, hipMemcpyDeviceToHost, st));
  WD_HIP(hipStreamSynchronize(st));
  if (s->h_buf[3 * B * k] != 0)
    return fail(WD_ERR_DEVICE, "device bookkeeping disagrees with the schedule (code %d)",
                s->h_buf[3 * B * k]);
  out->step = step;
  out->is_refresh = refresh;
  out->n_rows = rows;
  out->n_selected = nsel;
  if (out->positions) memcpy(out->positions, s->h_buf, B * k * 4);
  if (out->tokens) memcpy(out->tokens, s->h_buf + B * k, B * k * 4);
  if (out->conf) memcpy(out->conf, s->h_buf + 2 * B * k, B * k * 4);
  return WD_OK;
}

}  // namespace

extern "C" {

size_t wd_seq_bytes(const wd_model* m, const wd_window_config* win, int32_t batch,
                    const int32_t* prompt_lens, int32_t gen_len) {
  std::string why;
  if (!seq_args_valid(m, win, batch, prompt_lens, gen_len, &why)) return 0;
  long T = 0;
  int Smax = 0;
  for (int b = 0; b < batch; ++b) {
    T += prompt_lens[b] + gen_len;
    Smax = std::max(Smax, prompt_lens[b] + gen_len);
  }
  return seq_layout(*m, *win, batch, T, Smax, gen_len).total;
}

wd_status wd_prefill_prompt(wd_model* m, const int32_t* prompt_ids, const int32_t* prompt_lens,
                            int32_t batch, int32_t gen_len, const wd_window_config* win,
                            void* workspace, size_t ws_bytes, wd_seq** out) {
  std::string why;
  if (!out) return fail(WD_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  if (!seq_args_valid(m, win, batch, prompt_lens, gen_len, &why))
    return fail(WD_ERR_INVALID_ARG, "%s", why.c_str());
  if (win->stop_at_eos && win->buffer_refresh)
    return fail(WD_ERR_UNSUPPORTED, "adaptive termination with the buffer-only refresh");
  long n_ids = 0;
  for (int b = 0; b < batch; ++b) n_ids += prompt_lens[b];
  if (n_ids > 0 && !prompt_ids) return fail(WD_ERR_INVALID_ARG, "prompt_ids is NULL");
  for (long i = 0; i < n_ids; ++i)
    if (prompt_ids[i] < 0 || prompt_ids[i] >= m->cfg.vocab)
      return fail(WD_ERR_INVALID_ARG, "prompt id %d at %ld outside [0, vocab)", prompt_ids[i], i);
  if (!workspace) return fail(WD_ERR_INVALID_ARG, "workspace is NULL");
  if (((uintptr_t)workspace) & 255) return fail(WD_ERR_INVALID_ARG, "workspace not 256-byte aligned");
  if (hipSetDevice(m->device) != hipSuccess) return fail(WD_ERR_DEVICE, "hipSetDevice failed");

  wd_seq* s = new (std::nothrow) wd_seq();
  if (!s) return fail(WD_ERR_OUT_OF_MEMORY, "host allocation failed");
  s->m = m;
  s->win = *win;
  s->B = batch;
  s->G = gen_len;
  long T = 0;
  for (int b = 0; b < batch; ++b) {
    s->np.push_back(prompt_lens[b]);
    s->S.push_back(prompt_lens[b] + gen_len);
    s->off.push_back((int)T);
    T += prompt_lens[b] + gen_len;
    s->Smax = std::max(s->Smax, prompt_lens[b] + gen_len);
  }
  s->T = T;
  s->ctx.assign(batch, 0);
  const SeqLayout L = seq_layout(*m, *win, batch, T, s->Smax, gen_len);
  if (ws_bytes < L.total) {
    delete s;
    return fail(WD_ERR_OUT_OF_MEMORY, "workspace holds %zu bytes, %zu needed", ws_bytes, L.total);
  }
  char* base = (char*)workspace;
  s->x = (int32_t*)(base + L.x);
  s->seq_len = (int32_t*)(base + L.seq_len);
  s->dec = (uint8_t*)(base + L.dec);
  s->dec0 = (uint8_t*)(base + L.dec0);
  s->decp = (uint8_t*)(base + L.decp);
  s->kc = base + L.kc;
  s->vc = base + L.vc;
  s->rope = (float*)(base + L.rope);
  s->h = (float*)(base + L.h);
  s->a = base + L.a;
  s->q = base + L.q;
  s->o = base + L.o;
  s->sw = base + L.sw;
  s->C = (float*)(base + L.C);
  s->row_tok = (int32_t*)(base + L.row_tok);
  s->row_pos = (int32_t*)(base + L.row_pos);
  s->row_seq = (int32_t*)(base + L.row_seq);
  s->row_out = (int32_t*)(base + L.row_out);
  s->act_pos = (int32_t*)(base + L.act_pos);
  s->act_tok = (int32_t*)(base + L.act_tok);
  s->act_conf = (float*)(base + L.act_conf);
  s->a_act = base + L.a_act;
  s->logits = (float*)(base + L.logits);
  s->sel_pos = (int32_t*)(base + L.sel_pos);
  s->sel_tok = (int32_t*)(base + L.sel_tok);
  s->sel_conf = (float*)(base + L.sel_conf);
  s->err = (int32_t*)(base + L.err);
  s->dbg = (float*)(base + L.dbg);
  s->attn_part = (float*)(base + L.attn_part);
  s->attn_part_floats = L.attn_part_floats;
  s->conf_scratch = (float*)(base + L.conf_scratch);
  s->M_max = L.M_max;
  s->A_max = L.A_max;
  s->C_floats = L.C_floats;

  s->eos_id = win->stop_at_eos ? win->eos_id : -1;
  if (s->eos_id >= 0)
    for (int b = 0; b < batch; ++b) {
      Track t;
      t.n_p = prompt_lens[b];
      t.S = t.end = prompt_lens[b] + gen_len;
      t.dec.assign(t.S, 0);
      std::fill(t.dec.begin(), t.dec.begin() + t.n_p, 1);
      t.dec0 = t.dec;
      s->tr.push_back(std::move(t));
    }
  s->cnt.E = win->n_active + win->n_buffer;
  s->cnt.R = win->refresh_every;
  s->cnt.k = win->unmask_per_step;
  s->cnt.na = win->n_active;
  s->cnt.u = gen_len;
  s->cnt.j = -1;

  // host-side initial state
  std::vector<int32_t> x(T);
  std::vector<uint8_t> dec(T);
  long p = 0, id = 0;
  for (int b = 0; b < batch; ++b) {
    for (int i = 0; i < prompt_lens[b]; ++i) {
      x[p] = prompt_ids[id++];
      dec[p++] = 1;
    }
    for (int i = 0; i < gen_len; ++i) {
      x[p] = m->cfg.mask_id;
      dec[p++] = 0;
    }
  }
  const int half = m->cfg.head_dim / 2;
  std::vector<float> rope((size_t)s->Smax * half * 2);
  for (int pos = 0; pos < s->Smax; ++pos)
    for (int i = 0; i < half; ++i) {
      const double ang = (double)pos * std::pow((double)m->cfg.rope_theta, -2.0 * i / m->cfg.head_dim);
      rope[((size_t)pos * half + i) * 2] = (float)std::cos(ang);
      rope[((size_t)pos * half + i) * 2 + 1] = (float)std::sin(ang);
    }
  const int32_t zero = 0;
  hipStream_t st = m->stream;
  const size_t kv_bytes = (size_t)m->cfg.n_layers * m->cfg.n_kv_heads * m->cfg.head_dim * T * m->esz;
  bool ok = hipHostMalloc((void**)&s->h_buf, (size_t)(3 * batch * win->unmask_per_step + 1) * 4,
                          hipHostMallocDefault) == hipSuccess;
  ok = ok && hipMemcpyAsync(s->x, x.data(), T * 4, hipMemcpyHostToDevice, st) == hipSuccess;
  ok = ok && hipMemcpyAsync(s->dec, dec.data(), T, hipMemcpyHostToDevice, st) == hipSuccess;
  ok = ok && hipMemcpyAsync(s->dec0, dec.data(), T, hipMemcpyHostToDevice, st) == hipSuccess;
  ok = ok && hipMemcpyAsync(s->decp, dec.data(), T, hipMemcpyHostToDevice, st) == hipSuccess;
  ok = ok && hipMemcpyAsync(s->seq_len, s->S.data(), batch * 4, hipMemcpyHostToDevice, st) == hipSuccess;
  ok = ok && hipMemcpyAsync(s->rope, rope.data(), rope.size() * 4, hipMemcpyHostToDevice, st) == hipSuccess;
  ok = ok && hipMemcpyAsync(s->err, &zero, 4, hipMemcpyHostToDevice, st) == hipSuccess;
  // never-written cache rows read as NaN
  ok = ok && hipMemsetAsync(s->kc, 0xff, kv_bytes, st) == hipSuccess;
  ok = ok && hipMemsetAsync(s->vc, 0xff, kv_bytes, st) == hipSuccess;
  ok = ok && hipStreamSynchronize(st) == hipSuccess;
  if (!ok) {
    if (s->h_buf) (void)hipHostFree(s->h_buf);
    delete s;
    return fail(WD_ERR_DEVICE, "initial state upload failed");
  }
  m->live_seqs++;
  *out = s;
  return WD_OK;
}

wd_status wd_slide_window(wd_seq* s) {
  if (!s) return fail(WD_ERR_INVALID_ARG, "seq is NULL");
  if (s->eos_id >= 0)
    return fail(WD_ERR_UNSUPPORTED, "with adaptive termination phases are driven by wd_step");
  if (s->mode == 2) return fail(WD_ERR_STATE, "sequence is driven by wd_full_step");
  if (s->cnt.u == 0) return fail(WD_ERR_STATE, "every position is decoded");
  s->mode = 1;
  return do_slide(s);
}

wd_status wd_refresh_buffer(wd_seq* s) {
  if (!s) return fail(WD_ERR_INVALID_ARG, "seq is NULL");
  if (s->eos_id >= 0)
    return fail(WD_ERR_UNSUPPORTED, "with adaptive termination phases are driven by wd_step");
  if (s->mode == 2) return fail(WD_ERR_STATE, "sequence is driven by wd_full_step");
  if (s->cnt.u == 0) return fail(WD_ERR_STATE, "every position is decoded");
  if (s->cnt.j != 0 || s->refreshed)
    return fail(WD_ERR_STATE, "no phase waiting for its refresh (call wd_slide_window first)");
  s->mode = 1;
  return do_refresh(s);
}

wd_status wd_step(wd_seq* s, wd_step_out* out) {
  if (!s) return fail(WD_ERR_INVALID_ARG, "seq is NULL");
  if (s->mode == 2) return fail(WD_ERR_STATE, "sequence is driven by wd_full_step");
  if (s->eos_id >= 0) {
    if (all_done(s)) return fail(WD_ERR_STATE, "every live position is decoded");
    s->mode = 1;
    return step_tracked(s, out, false);
  }
  if (s->cnt.u == 0) return fail(WD_ERR_STATE, "every position is decoded");
  s->mode = 1;
  if (s->cnt.phase_due()) WD_TRY(do_slide(s));
  const bool refresh = s->cnt.j == 0;
  int rows;
  if (refresh) {
    if (!s->refreshed) WD_TRY(do_refresh(s));
    rows = 0;
    for (int b = 0; b < s->B; ++b) rows += s->cnt.refresh_rows(s->ctx[b], s->win.buffer_refresh);
  } else {
    WD_TRY(do_normal(s));
    rows = s->B * (s->cnt.n_active() + s->cnt.dp);
  }
  const int nA = s->cnt.n_active();
  const int nsel = s->cnt.n_decode();
  WD_TRY(decide(s, nA));
  const int step = s->t;
  s->cnt.take_step();
  s->t++;
  if (out) return fetch_out(s, out, step, refresh ? 1 : 0, rows, nsel);
  return WD_OK;
}

wd_status wd_step_noalloc(wd_seq* s, wd_step_out* out) {
  if (!s) return fail(WD_ERR_INVALID_ARG, "seq is NULL");
  wd_model& m = *s->m;
  const wd_model_config& c = m.cfg;
  if (s->eos_id >= 0)
    return fail(WD_ERR_UNSUPPORTED, "wd_step_noalloc does not take adaptive termination (use wd_step)");
  if (m.profile)
    return fail(WD_ERR_UNSUPPORTED, "kernel timing creates HIP events; disable it for wd_step_noalloc");
  if (s->mode == 2) return fail(WD_ERR_STATE, "sequence is driven by wd_full_step");
  if (s->cnt.u == 0) return fail(WD_ERR_STATE, "every position is decoded");
  void* base = m.device >= 0 && m.device < kMaxDevices ? g_scratch_dev[m.device] : nullptr;
  if (!base) return fail(WD_ERR_DEVICE, "no static scratch address for device %d", m.device);
  // the rows this step runs through the layer stack and the LM head, counted
  // as wd_step will count them (on a copy of the schedule's counts)
  Counts cn = s->cnt;
  const bool due = cn.phase_due();
  if (due) cn.start_phase();
  int rows = 0;
  if (cn.j == 0) {
    for (int b = 0; b < s->B; ++b)
      rows += cn.refresh_rows(due ? cn.ctx(s->S[b]) : s->ctx[b], s->win.buffer_refresh);
  } else {
    rows = s->B * (cn.n_active() + cn.dp);
  }
  const int n_act_rows = s->B * cn.n_active();
  const size_t part_bytes = step_partial_floats(m, rows) * 4;
  const size_t attn_bytes =
      c.dtype == WD_DTYPE_BF16
          ? (size_t)std::min<long>(s->attn_part_floats,
                                   8L * rows * c.n_heads * (c.head_dim + 2)) * 4
          : 0;
  const size_t conf_bytes =
      (size_t)3 * n_act_rows * std::max<long>(wd::kConfChunks, c.vocab / 64) * 4;
  const size_t need = align256(part_bytes) + align256(attn_bytes) + align256(conf_bytes);
  if (need > kStaticScratchBytes)
    return fail(WD_ERR_OUT_OF_MEMORY,
                "step %d runs %d rows and needs %zu bytes of scratch; the static scratch holds %zu "
                "(use wd_step)", s->t, rows, need, kStaticScratchBytes);
  // the same step with its scratch redirected: plans and sizes are unchanged
  // (the capacities the kernels are told stay the workspace's; what they
  // touch fits in the regions above)
  struct Restore {
    wd_seq* s;
    float *part, *attn, *conf;
    ~Restore() {
      s->C = part;
      s->attn_part = attn;
      s->conf_scratch = conf;
    }
  } restore{s, s->C, s->attn_part, s->conf_scratch};
  char* p = (char*)base;
  s->C = (float*)p;
  s->attn_part = (float*)(p + align256(part_bytes));
  s->conf_scratch = (float*)(p + align256(part_bytes) + align256(attn_bytes));
  return wd_step(s, out);
}

wd_status wd_full_step(wd_seq* s, wd_step_out* out) {
  if (!s) return fail(WD_ERR_INVALID_ARG, "seq is NULL");
  if (s->mode == 1) return fail(WD_ERR_STATE, "sequence is driven by the windowed calls");
  if (s->eos_id >= 0) {
    if (all_done(s)) return fail(WD_ERR_STATE, "every live position is decoded");
    s->mode = 2;
    return step_tracked(s, out, true);
  }
  if (s->cnt.u == 0) return fail(WD_ERR_STATE, "every position is decoded");
  s->mode = 2;
  Rows r;
  for (int b = 0; b < s->B; ++b) s->ctx[b] = s->S[b];
  r.g = base_geom(s);
  for (int b = 0; b < s->B; ++b) {
    r.g.mode[b] = 2;
    r.g.nact[b] = s->cnt.u;
    r.g.row0[b] = s->off[b];
    r.g.nrows[b] = s->S[b];
  }
  r.M = (int)s->T;
  r.n_act = s->cnt.u;
  WD_TRY(forward(s, r));
  const int nA = s->cnt.u;
  const int nsel = std::min(s->cnt.k, nA);
  WD_TRY(decide(s, nA));
  const int step = s->t;
  s->cnt.u -= nsel;
  s->t++;
  if (out) return fetch_out(s, out, step, 1, (int)s->T, nsel);
  return WD_OK;
}

wd_status wd_get_state(const wd_seq* s, int32_t* tokens, uint8_t* decoded, int32_t* t) {
  if (!s || !tokens) return fail(WD_ERR_INVALID_ARG, "NULL argument");
  hipStream_t st = s->m->stream;
  WD_HIP(hipStreamSynchronize(st));
  WD_HIP(hipMemcpy(tokens, s->x, s->T * 4, hipMemcpyDeviceToHost));
  if (decoded) WD_HIP(hipMemcpy(decoded, s->dec, s->T, hipMemcpyDeviceToHost));
  if (t) *t = s->t;
  // the device's checks of every step so far against the host's schedule
  int32_t err = 0;
  WD_HIP(hipMemcpy(&err, s->err, 4, hipMemcpyDeviceToHost));
  if (err != 0)
    return fail(WD_ERR_DEVICE, "device bookkeeping disagrees with the schedule (code %d)", err);
  return WD_OK;
}

wd_status wd_seq_ends(const wd_seq* s, int32_t* ends) {
  if (!s || !ends) return fail(WD_ERR_INVALID_ARG, "NULL argument");
  for (int b = 0; b < s->B; ++b) ends[b] = s->tr.empty() ? s->S[b] : s->tr[b].end;
  return WD_OK;
}

wd_status wd_debug_keep_logits(wd_seq* s, int32_t on) {
  if (!s) return fail(WD_ERR_INVALID_ARG, "NULL argument");
  s->keep_logits = on != 0;
  return WD_OK;
}

wd_status wd_debug_logits(const wd_seq* s, float* logits, int32_t* positions, int32_t capacity,
                          int32_t* n_rows) {
  if (!s || !logits || !n_rows) return fail(WD_ERR_INVALID_ARG, "NULL argument");
  if (!s->logits_valid)
    return fail(WD_ERR_STATE, "no logits kept for the last step (wd_debug_keep_logits)");
  const int n = s->B * s->last_nA;
  *n_rows = n;
  if (capacity < n) return fail(WD_ERR_OUT_OF_MEMORY, "capacity %d < %d rows", capacity, n);
  WD_HIP(hipStreamSynchronize(s->m->stream));
  WD_HIP(hipMemcpy(logits, s->logits, (size_t)n * s->m->cfg.vocab * 4, hipMemcpyDeviceToHost));
  if (positions) WD_HIP(hipMemcpy(positions, s->act_pos, (size_t)n * 4, hipMemcpyDeviceToHost));
  return WD_OK;
}

wd_status wd_debug_kv(const wd_seq* s, int32_t layer, int32_t b, float* k, float* v,
                      int32_t capacity, int32_t* ctx_len) {
  if (!s || !k || !v || !ctx_len) return fail(WD_ERR_INVALID_ARG, "NULL argument");
  const wd_model_config& c = s->m->cfg;
  if (layer < 0 || layer >= c.n_layers || b < 0 || b >= s->B)
    return fail(WD_ERR_INVALID_ARG, "layer or sequence out of range");
  const int ctx = s->ctx[b] > 0 ? s->ctx[b] : s->S[b];
  *ctx_len = ctx;
  if (capacity < ctx) return fail(WD_ERR_OUT_OF_MEMORY, "capacity %d < %d positions", capacity, ctx);
  hipStream_t st = s->m->stream;
  const long KVd = (long)c.n_kv_heads * c.head_dim;
  const int d = c.head_dim;
  std::vector<float> tmp((size_t)ctx * d);
  for (int which = 0; which < 2; ++which) {
    const char* base = (const char*)(which ? s->vc : s->kc) + (size_t)layer * KVd * s->T * s->m->esz;
    float* dst = which ? v : k;
    for (int g = 0; g < c.n_kv_heads; ++g) {
      const size_t row0 = ((size_t)g * s->T + s->off[b]) * d;
      if (c.dtype == WD_DTYPE_BF16)
        WD_HIP(wd::widen_rows<uint16_t>((const uint16_t*)base + row0, d, s->dbg, ctx, d, st));
      else
        WD_HIP(wd::widen_rows<float>((const float*)base + row0, d, s->dbg, ctx, d, st));
      WD_HIP(hipStreamSynchronize(st));
      WD_HIP(hipMemcpy(tmp.data(), s->dbg, tmp.size() * 4, hipMemcpyDeviceToHost));
      for (int p = 0; p < ctx; ++p)
        memcpy(dst + ((size_t)p * c.n_kv_heads + g) * d, tmp.data() + (size_t)p * d, d * 4);
    }
  }
  return WD_OK;
}

void wd_free_seq(wd_seq* s) {
  if (!s) return;
  (void)hipStreamSynchronize(s->m->stream);
  if (s->h_buf) (void)hipHostFree(s->h_buf);
  s->m->live_seqs--;
  delete s;
}

int32_t wd_plan(int32_t n_prompt, int32_t gen_len, const wd_window_config* win, int32_t max_steps,
                int32_t* is_refresh, int32_t* ctx_len, int32_t* n_active, int32_t* n_rows,
                int32_t* n_decode) {
  std::string why;
  if (n_prompt < 0 || gen_len < 1 || !win_valid(win, &why)) {
    fail(WD_ERR_INVALID_ARG, "%s", why.empty() ? "bad prompt or generation length" : why.c_str());
    return -1;
  }
  Counts c;
  c.E = win->n_active + win->n_buffer;
  c.R = win->refresh_every;
  c.k = win->unmask_per_step;
  c.na = win->n_active;
  c.u = gen_len;
  const int S = n_prompt + gen_len;
  int t = 0, ctx = 0;
  while (c.u > 0) {
    bool refresh = false;
    if (c.phase_due()) {
      c.start_phase();
      ctx = c.ctx(S);
    }
    refresh = c.j == 0;
    if (t < max_steps) {
      if (is_refresh) is_refresh[t] = refresh ? 1 : 0;
      if (ctx_len) ctx_len[t] = ctx;
      if (n_active) n_active[t] = c.n_active();
      if (n_rows) n_rows[t] = refresh ? c.refresh_rows(ctx, win->buffer_refresh != 0)
                                      : c.n_active() + c.dp;
      if (n_decode) n_decode[t] = c.n_decode();
    }
    c.take_step();
    ++t;
  }
  return t;
}

wd_status wd_debug_gemm_plan(int32_t M, int32_t N, int32_t K, int32_t fp8, int32_t max_splits,
                             int32_t* out) {
  if (!out) return fail(WD_ERR_INVALID_ARG, "NULL argument");
  if (M < 1 || N < 1 || K < 1 || K % 32 || max_splits < 1 || M > (1 << 24) || N > (1 << 24) ||
      K > (1 << 24))
    return fail(WD_ERR_INVALID_ARG, "sizes must be in [1, 2^24], K a multiple of 32");
  const wd::GemmPlan p = wd::plan_gemm_bf16(M, N, K, fp8 != 0, max_splits);
  int kernel, rows, features, waves;
  wd::gemm_plan_tile(p, &kernel, &rows, &features, &waves);
  out[0] = kernel;
  out[1] = rows;
  out[2] = features;
  out[3] = p.splits;
  out[4] = p.ks_per_split;
  out[5] = p.grid;
  out[6] = waves;
  out[7] = (wd::gemm_plan_ok(p, M, N, K, fp8 != 0, false) ? 1 : 0) |
           (wd::gemm_plan_ok(p, M, N, K, fp8 != 0, true) ? 2 : 0);
  return WD_OK;
}

}  // extern "C"
