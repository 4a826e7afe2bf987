// Host runtime behind the C ABI: model and workspace ownership, the launch
// sequence of one dense pass, the denoising step, and the gated block decode loop.
#include <math.h>
#include <stdio.h>
#include <string.h>

#include <mutex>

#include <string>
#include <algorithm>
#include <vector>

#include <new>
#include <stdexcept>

#include "common.hpp"
#include "internal.hpp"

using namespace cora;

namespace {

// last error message of this thread: a fixed buffer, so reporting an error allocates nothing
thread_local char g_err[512];

cora_status fail(cora_status st, const char* msg) noexcept {
  snprintf(g_err, sizeof(g_err), "%s", msg ? msg : "");
  return st;
}

cora_status fail(cora_status st, const std::string& msg) noexcept { return fail(st, msg.c_str()); }

// An exception escaping an entry point becomes a status (the C ABI never throws): host
// allocation failure is CORA_ERR_OOM, anything else CORA_ERR_UNSUPPORTED with its text.
cora_status exception_status() noexcept {
  try {
    throw;
  } catch (const std::bad_alloc&) {
    return fail(CORA_ERR_OOM, "host memory allocation failed");
  } catch (const std::exception& x) {
    return fail(CORA_ERR_UNSUPPORTED, std::string("unexpected C++ exception: ") + x.what());
  } catch (...) {
    return fail(CORA_ERR_UNSUPPORTED, "unexpected C++ exception");
  }
}

// A failed HIP call is reported through the status alone: HIP's per-thread last-error
// slot is cleared, so the caller's next hipGetLastError does not see it again.
cora_status fail_hip(cora_status st, const std::string& msg) {
  (void)hipGetLastError();
  return fail(st, msg);
}

#define HIP_TRY(expr)                                                                   \
  do {                                                                                  \
    hipError_t e_ = (expr);                                                             \
    if (e_ != hipSuccess)                                                               \
      return fail_hip(CORA_ERR_HIP, std::string(#expr) + ": " + hipGetErrorString(e_)); \
  } while (0)

constexpr size_t ALIGN = 256;
inline size_t align_up(size_t x) { return (x + ALIGN - 1) / ALIGN * ALIGN; }
inline int round_up(int x, int m) { return (x + m - 1) / m * m; }

// bump allocator over one device allocation
struct Arena {
  char* base = nullptr;
  size_t used = 0, cap = 0;
  template <class T>
  T* take(size_t n) {
    T* p = reinterpret_cast<T*>(base + used);
    used += align_up(n * sizeof(T));
    return p;
  }
};

}  // namespace

struct cora_model {
  cora_model_cfg cfg{};
  int max_batch = 0, max_seq = 0, max_seq_pad = 0, max_rows = 0;
  int hq = 0, hkv = 0, qkv_n = 0, f_pad = 0;
  void* weight_mem = nullptr;
  void* ws_mem = nullptr;
  size_t weight_bytes = 0, ws_bytes = 0;

  uint16_t *embed = nullptr, *lm_head = nullptr;
  // LM head in the packed layout of the few-row kernel (null when the shape does not fit it)
  uint16_t* lm_head_packed = nullptr;
  float* ones = nullptr;  // all norm weights are 1
  struct Layer {
    uint16_t *wqkv, *wo, *wgu, *wd;
    float* bqkv;
  };
  std::vector<Layer> layers;

  // workspace
  float* h = nullptr;
  uint16_t *a = nullptr, *q = nullptr, *k = nullptr, *vt = nullptr;
  uint16_t *attn = nullptr, *u = nullptr, *logits = nullptr;
  float *rope_cos = nullptr, *rope_sin = nullptr;
  int num_cus = 256;
  float* splitk_ws = nullptr;
  size_t splitk_ws_floats = 0;
  // per-row partial softmax statistics of the fused LM head ([64][lm_head_parts(V)])
  float *lmh_pm = nullptr, *lmh_ps = nullptr;
  int* lmh_pa = nullptr;
  // decode state owned for cora_block_decode
  int32_t *s_tokens = nullptr, *s_prev = nullptr, *s_persist = nullptr, *s_block = nullptr;
  int32_t *s_step = nullptr, *s_top1 = nullptr, *s_done = nullptr, *s_passes = nullptr;
  uint8_t *s_unres = nullptr, *s_decision = nullptr;
  float* s_conf = nullptr;
  int32_t* h_block = nullptr;  // pinned host mirror of block_idx
  // batch-row compaction: a second state buffer set (live rows are gathered into it once
  // some rows finish), row maps (pinned host + device, 3 x max_batch), and the per-block
  // passes of every original row
  DecodeRows s_alt{};
  int32_t* h_map = nullptr;
  int32_t* d_map = nullptr;
  int32_t* s_final_passes = nullptr;
  bool compaction = true;

  // gate/up GEMM timing
  bool timing = false;
  std::vector<hipEvent_t> ev;  // pairs
  size_t ev_used = 0;
  double acc_ms = 0.0;
  int64_t launches = 0;
};

static cora_status validate_cfg(const cora_model_cfg& c) {
  if (c.n_layers < 0 || c.d_model <= 0 || c.n_heads <= 0 || c.n_kv_heads <= 0 ||
      c.ffn_dim <= 0 || c.vocab < 2)
    return fail(CORA_ERR_INVALID_ARG, "model dimensions must be positive (vocab >= 2)");
  if (c.mask_id < 0 || c.mask_id >= c.vocab)
    return fail(CORA_ERR_INVALID_ARG, "mask_id must lie in [0, vocab)");
  if (c.head_dim != 64 && c.head_dim != 128)
    return fail(CORA_ERR_UNSUPPORTED, "head_dim must be 64 or 128");
  if (c.n_heads % c.n_kv_heads != 0)
    return fail(CORA_ERR_UNSUPPORTED, "n_heads must be a multiple of n_kv_heads");
  if (c.d_model % 64 != 0 || (c.n_heads * c.head_dim) % 64 != 0)
    return fail(CORA_ERR_UNSUPPORTED, "d_model and n_heads*head_dim must be multiples of 64");
  if (c.d_model > RESIDUAL_NORM_MAX_D)
    return fail(CORA_ERR_UNSUPPORTED, "d_model must not exceed 8192");
  {
    // the GEMMs address every layer matrix with 32-bit byte offsets
    const int64_t hq = (int64_t)c.n_heads * c.head_dim, hkv = (int64_t)c.n_kv_heads * c.head_dim;
    const int64_t fp = ((int64_t)c.ffn_dim + 63) / 64 * 64, d = c.d_model;
    const int64_t largest = std::max({(hq + 2 * hkv) * d, d * hq, 2 * fp * d, d * fp});
    if (largest * 2 + std::max({d, hq, fp}) * 128 > 0x7fffffffLL)
      return fail(CORA_ERR_UNSUPPORTED, "a layer weight matrix exceeds 2 GB");
  }
  if (!(c.rms_eps > 0.f) || !(c.rope_theta > 0.f) || !isfinite(c.logit_scale) ||
      !(c.init_std >= 0.0))
    return fail(CORA_ERR_INVALID_ARG, "rms_eps, rope_theta must be > 0; logit_scale finite");
  return CORA_OK;
}

static hipStream_t S(void* s) { return reinterpret_cast<hipStream_t>(s); }

// ---------------------------------------------------------------------------------------
extern "C" const char* cora_last_error(void) { return g_err; }

extern "C" cora_status cora_model_destroy(cora_model* m) try {
  if (!m) return CORA_OK;
  for (hipEvent_t e : m->ev) (void)hipEventDestroy(e);
  if (m->h_block) (void)hipHostFree(m->h_block);
  if (m->h_map) (void)hipHostFree(m->h_map);
  if (m->ws_mem) (void)hipFree(m->ws_mem);
  if (m->weight_mem) (void)hipFree(m->weight_mem);
  delete m;
  return CORA_OK;
} catch (...) {
  return exception_status();
}

extern "C" cora_status cora_model_create(const cora_model_cfg* cfg, uint64_t seed,
                                         int32_t max_batch, int32_t max_seq, void* hip_stream,
                                         cora_model** out) try {
  if (!cfg || !out) return fail(CORA_ERR_INVALID_ARG, "null cfg or out");
  if (cora_status st = validate_cfg(*cfg)) return st;
  if (max_batch <= 0 || max_seq <= 0) return fail(CORA_ERR_INVALID_ARG, "max_batch/max_seq <= 0");
  if (max_batch > (1 << 24) || max_seq > (1 << 24))
    return fail(CORA_ERR_UNSUPPORTED, "max_batch x max_seq too large: an activation matrix would exceed 2 GB");
  {
    // the GEMM operand loads address an activation matrix [max_batch * max_seq, width] with
    // 32-bit byte offsets; bound the widest one (fp32 residual, bf16 FFN or head rows)
    const size_t widest = std::max({(size_t)cfg->d_model * 4, (size_t)round_up(cfg->ffn_dim, 64) * 2,
                                    (size_t)cfg->n_heads * cfg->head_dim * 2});
    if ((size_t)max_batch * (size_t)round_up(max_seq, 64) * widest > 0x7fffffffULL)
      return fail(CORA_ERR_UNSUPPORTED,
                  "max_batch x max_seq too large: an activation matrix would exceed 2 GB");
  }
  const hipStream_t s = S(hip_stream);
  cora_model* m = new cora_model();
  // frees the partly built model on every failure path, including an exception
  struct Guard {
    cora_model* m;
    ~Guard() {
      if (m) cora_model_destroy(m);
    }
  } guard{m};
  m->cfg = *cfg;
  m->max_batch = max_batch;
  m->max_seq = max_seq;
  m->max_seq_pad = round_up(max_seq, 64);
  m->max_rows = max_seq < CORA_MAX_BLOCK_LEN ? max_seq : CORA_MAX_BLOCK_LEN;
  const int d = cfg->d_model, V = cfg->vocab, hd = cfg->head_dim;
  m->hq = cfg->n_heads * hd;
  m->hkv = cfg->n_kv_heads * hd;
  m->qkv_n = m->hq + 2 * m->hkv;
  m->f_pad = round_up(cfg->ffn_dim, 64);
  const int64_t L_ = cfg->n_layers;

  // ---- weights
  size_t wb = 2 * align_up((size_t)V * d * 2) + align_up((size_t)d * 4);
  // packed LM-head copy for steps that score at most 64 rows (one extra V x d matrix)
  const bool pack_lm = lm_head_supported(1, V, d, d);
  if (pack_lm) wb += align_up(lm_head_packed_elems(V, d) * 2);
  const size_t per_layer = align_up((size_t)m->qkv_n * d * 2) + align_up((size_t)d * m->hq * 2) +
                           align_up((size_t)2 * m->f_pad * d * 2) +
                           align_up((size_t)d * m->f_pad * 2) +
                           (cfg->qkv_bias ? align_up((size_t)m->qkv_n * 4) : 0);
  wb += per_layer * L_;
  // ---- workspace
  const size_t M = (size_t)max_batch * max_seq;
  const size_t Ms = (size_t)max_batch * m->max_seq_pad;
  const size_t rows = (size_t)max_batch * m->max_rows;
  const size_t BL = M;
  {
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
        cus > 0)
      m->num_cus = cus;
  }
  const size_t skw = gemm_ws_floats_bound(m->num_cus);
  const size_t lmh_parts = (size_t)LM_HEAD_FUSED_MAX_ROWS * lm_head_parts(V);
  size_t wsb = 3 * align_up(lmh_parts * 4) + align_up(skw * 4) + align_up(M * d * 4) + align_up(M * (size_t)(d > m->hq ? d : m->hq) * 2) +
               align_up(Ms * m->hq * 2) + 2 * align_up(Ms * m->hkv * 2) +
               align_up(M * m->hq * 2) + align_up(M * m->f_pad * 2) + align_up(rows * V * 2) +
               2 * align_up((size_t)m->max_seq_pad * (hd / 2) * 4) +
               // decode state
               align_up(BL * 4) * 3 + align_up(BL) + align_up(max_batch * 4) * 3 +
               align_up(BL * 4) * 2 + align_up(rows) + align_up((size_t)max_batch * max_seq * 4) +
               // compaction: second state set, row maps, final passes
               align_up(BL * 4) * 3 + align_up(BL) + align_up(max_batch * 4) * 2 +
               align_up((size_t)max_batch * max_seq * 4) * 2 + align_up(3 * max_batch * 4);
  hipError_t e = hipMalloc(&m->weight_mem, wb);
  if (e != hipSuccess) {
    return fail_hip(e == hipErrorOutOfMemory ? CORA_ERR_OOM : CORA_ERR_HIP,
                std::string("weight allocation: ") + hipGetErrorString(e));
  }
  e = hipMalloc(&m->ws_mem, wsb);
  if (e != hipSuccess) {
    return fail_hip(e == hipErrorOutOfMemory ? CORA_ERR_OOM : CORA_ERR_HIP,
                std::string("workspace allocation: ") + hipGetErrorString(e));
  }
  m->weight_bytes = wb;
  m->ws_bytes = wsb;

  Arena w{(char*)m->weight_mem, 0, wb};
  m->embed = w.take<uint16_t>((size_t)V * d);
  m->lm_head = w.take<uint16_t>((size_t)V * d);
  if (pack_lm) m->lm_head_packed = w.take<uint16_t>(lm_head_packed_elems(V, d));
  m->ones = w.take<float>(d);
  m->layers.resize(L_);
  for (auto& ly : m->layers) {
    ly.wqkv = w.take<uint16_t>((size_t)m->qkv_n * d);
    ly.wo = w.take<uint16_t>((size_t)d * m->hq);
    ly.wgu = w.take<uint16_t>((size_t)2 * m->f_pad * d);
    ly.wd = w.take<uint16_t>((size_t)d * m->f_pad);
    ly.bqkv = cfg->qkv_bias ? w.take<float>(m->qkv_n) : nullptr;
  }
  Arena a{(char*)m->ws_mem, 0, wsb};
  m->lmh_pm = a.take<float>(lmh_parts);
  m->lmh_ps = a.take<float>(lmh_parts);
  m->lmh_pa = a.take<int>(lmh_parts);
  m->splitk_ws = a.take<float>(skw);
  m->splitk_ws_floats = skw;
  m->h = a.take<float>(M * d);
  m->a = a.take<uint16_t>(M * (d > m->hq ? d : m->hq));
  m->q = a.take<uint16_t>(Ms * m->hq);
  m->k = a.take<uint16_t>(Ms * m->hkv);
  m->vt = a.take<uint16_t>(Ms * m->hkv);
  m->attn = a.take<uint16_t>(M * m->hq);
  m->u = a.take<uint16_t>(M * m->f_pad);
  m->logits = a.take<uint16_t>(rows * V);
  m->rope_cos = a.take<float>((size_t)m->max_seq_pad * (hd / 2));
  m->rope_sin = a.take<float>((size_t)m->max_seq_pad * (hd / 2));
  m->s_tokens = a.take<int32_t>(BL);
  m->s_prev = a.take<int32_t>(BL);
  m->s_persist = a.take<int32_t>(BL);
  m->s_unres = a.take<uint8_t>(BL);
  m->s_block = a.take<int32_t>(max_batch);
  m->s_step = a.take<int32_t>(max_batch);
  m->s_done = a.take<int32_t>(max_batch);
  m->s_top1 = a.take<int32_t>(BL);   // [B, gen_len] under the GLOBAL scope
  m->s_conf = a.take<float>(BL);
  m->s_decision = a.take<uint8_t>(rows);
  m->s_passes = a.take<int32_t>((size_t)max_batch * max_seq);
  m->s_alt.tokens = a.take<int32_t>(BL);
  m->s_alt.prev = a.take<int32_t>(BL);
  m->s_alt.persist = a.take<int32_t>(BL);
  m->s_alt.unresolved = a.take<uint8_t>(BL);
  m->s_alt.block_idx = a.take<int32_t>(max_batch);
  m->s_alt.step_idx = a.take<int32_t>(max_batch);
  m->s_alt.passes = a.take<int32_t>((size_t)max_batch * max_seq);
  m->s_final_passes = a.take<int32_t>((size_t)max_batch * max_seq);
  m->d_map = a.take<int32_t>((size_t)3 * max_batch);
  e = hipHostMalloc((void**)&m->h_block, max_batch * sizeof(int32_t), hipHostMallocDefault);
  if (e == hipSuccess)
    e = hipHostMalloc((void**)&m->h_map, 3 * max_batch * sizeof(int32_t), hipHostMallocDefault);
  if (e != hipSuccess) {
    return fail_hip(e == hipErrorOutOfMemory ? CORA_ERR_OOM : CORA_ERR_HIP,
                    std::string("pinned allocation: ") + hipGetErrorString(e));
  }

  // ---- fill weights
  auto st = [&]() -> cora_status {
    HIP_TRY(hipMemsetAsync(m->weight_mem, 0, wb, s));
    const double sd = cfg->init_std;
    HIP_TRY(hipMemsetAsync(m->ws_mem, 0, wsb, s));  // finite zeros in every padding region
    HIP_TRY(launch_init_bf16(m->embed, seed, 1, V, d, d, ROW_IDENTITY, 0, sd, hd, s));
    HIP_TRY(launch_init_bf16(m->lm_head, seed, 2, V, d, d, ROW_IDENTITY, 0, sd, hd, s));
    if (m->lm_head_packed) HIP_TRY(launch_pack_lm_head(m->lm_head, m->lm_head_packed, V, d, s));
    HIP_TRY(launch_fill_f32(m->ones, 1.0f, d, s));
    for (int l = 0; l < (int)L_; ++l) {
      const auto& ly = m->layers[l];
      const uint64_t t0 = 100 + 16 * (uint64_t)l;
      HIP_TRY(launch_init_bf16(ly.wqkv, seed, t0 + 0, m->hq, d, d, ROW_ROPE_PAIR, 0, sd, hd, s, true));
      HIP_TRY(launch_init_bf16(ly.wqkv, seed, t0 + 1, m->hkv, d, d, ROW_ROPE_PAIR, m->hq, sd, hd,
                               s, true));
      HIP_TRY(launch_init_bf16(ly.wqkv, seed, t0 + 2, m->hkv, d, d, ROW_IDENTITY, m->hq + m->hkv,
                               sd, hd, s, true));
      HIP_TRY(launch_init_bf16(ly.wo, seed, t0 + 3, d, m->hq, m->hq, ROW_IDENTITY, 0, sd, hd, s, true));
      HIP_TRY(launch_init_bf16(ly.wgu, seed, t0 + 4, cfg->ffn_dim, d, d, ROW_GATE, 0, sd, hd, s, true));
      HIP_TRY(launch_init_bf16(ly.wgu, seed, t0 + 5, cfg->ffn_dim, d, d, ROW_UP, 0, sd, hd, s, true));
      HIP_TRY(launch_init_bf16(ly.wd, seed, t0 + 6, d, cfg->ffn_dim, m->f_pad, ROW_IDENTITY, 0, sd,
                               hd, s, true));
      if (cfg->qkv_bias) {
        HIP_TRY(launch_init_f32(ly.bqkv, seed, t0 + 7, m->hq, sd, hd, s));
        HIP_TRY(launch_init_f32(ly.bqkv + m->hq, seed, t0 + 8, m->hkv, sd, hd, s));
        HIP_TRY(launch_init_f32(ly.bqkv + m->hq + m->hkv, seed, t0 + 9, m->hkv, sd, 0, s));
      }
    }
    // RoPE tables in fp64, stored fp32: angle = pos * theta^(-2j/hd)
    const int half = hd / 2;
    std::vector<float> cs((size_t)m->max_seq_pad * half), sn(cs.size());
    for (int p = 0; p < m->max_seq_pad; ++p)
      for (int j = 0; j < half; ++j) {
        const double ang = (double)p * pow((double)cfg->rope_theta, -2.0 * j / hd);
        cs[(size_t)p * half + j] = (float)cos(ang);
        sn[(size_t)p * half + j] = (float)sin(ang);
      }
    HIP_TRY(hipMemcpyAsync(m->rope_cos, cs.data(), cs.size() * 4, hipMemcpyHostToDevice, s));
    HIP_TRY(hipMemcpyAsync(m->rope_sin, sn.data(), sn.size() * 4, hipMemcpyHostToDevice, s));
    HIP_TRY(hipStreamSynchronize(s));
    return CORA_OK;
  }();
  if (st != CORA_OK) {
    return st;
  }
  guard.m = nullptr;
  *out = m;
  return CORA_OK;
} catch (...) {
  return exception_status();
}

extern "C" cora_status cora_model_device_bytes(cora_model* m, size_t* wbytes, size_t* wsbytes) try {
  if (!m) return fail(CORA_ERR_INVALID_ARG, "null model");
  if (wbytes) *wbytes = m->weight_bytes;
  if (wsbytes) *wsbytes = m->ws_bytes;
  return CORA_OK;
} catch (...) {
  return exception_status();
}

// ---- timing ------------------------------------------------------------------------------
// Timing events are created without a system-scope fence and handed to the kernel launch,
// which stamps them with the kernel's own start and end.
static cora_status grow_events(cora_model* m, size_t n) {
  while (m->ev.size() < n) {
    hipEvent_t e;
    HIP_TRY(hipEventCreateWithFlags(&e, hipEventDisableSystemFence));
    m->ev.push_back(e);
  }
  return CORA_OK;
}

extern "C" cora_status cora_model_set_compaction(cora_model* m, int32_t enable) try {
  if (!m) return fail(CORA_ERR_INVALID_ARG, "null model");
  m->compaction = enable != 0;
  return CORA_OK;
} catch (...) {
  return exception_status();
}

// Turning timing on or off keeps what has been recorded; read_timing returns and clears it.
extern "C" cora_status cora_model_set_timing(cora_model* m, int32_t enable) try {
  if (!m) return fail(CORA_ERR_INVALID_ARG, "null model");
  m->timing = enable != 0;
  // created up front so the timed passes do not pay for them
  if (m->timing)
    if (cora_status st = grow_events(m, 2 * m->layers.size() * 64)) return st;
  return CORA_OK;
} catch (...) {
  return exception_status();
}

static cora_status drain_events(cora_model* m) {
  for (size_t i = 0; i + 1 < m->ev_used; i += 2) {
    HIP_TRY(hipEventSynchronize(m->ev[i + 1]));
    float ms = 0.f;
    HIP_TRY(hipEventElapsedTime(&ms, m->ev[i], m->ev[i + 1]));
    m->acc_ms += ms;
    m->launches += 1;
  }
  m->ev_used = 0;
  return CORA_OK;
}

extern "C" cora_status cora_model_read_timing(cora_model* m, double* total_ms, int64_t* launches) try {
  if (!m) return fail(CORA_ERR_INVALID_ARG, "null model");
  if (cora_status st = drain_events(m)) return st;
  if (total_ms) *total_ms = m->acc_ms;
  if (launches) *launches = m->launches;
  m->acc_ms = 0.0;
  m->launches = 0;
  return CORA_OK;
} catch (...) {
  return exception_status();
}

// the next free (start, stop) event pair
static cora_status timed_pair(cora_model* m, hipEvent_t* e0, hipEvent_t* e1) {
  if (m->ev_used + 2 > m->ev.size()) {
    if (m->ev.size() >= 8192) {
      if (cora_status st = drain_events(m)) return st;
    } else {
      if (cora_status st = grow_events(m, m->ev.size() + 64)) return st;
    }
  }
  *e0 = m->ev[m->ev_used++];
  *e1 = m->ev[m->ev_used++];
  return CORA_OK;
}

// ---- one dense pass ----------------------------------------------------------------------
// Rows decode independently (R15), and a row's results must not depend on which other rows
// share its pass (batch-row compaction drops finished rows; a row decoded alone must match
// its batched decode).  Every choice that changes an output's summation order (split-K
// count, attention key-range parts, LM-head kernel and its vocab partial layout) is made
// for max_batch rows of the call's per-row length, never for the live row count; only
// choices that leave every sum as it is (GEMM tile shapes) follow the live rows.
static int plan_rows(const cora_model* m, int rows_per_batch_row) {
  return m->max_batch * rows_per_batch_row;
}

static cora_status gemm(cora_model* m, int epi, const GemmArgs& g, hipStream_t s,
                        bool timed = false) {
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (timed)
    if (cora_status st = timed_pair(m, &e0, &e1)) return st;
  HIP_TRY(launch_gemm(epi, g, gemm_plan(g.M, g.N, g.K, m->num_cus), s, e0, e1));
  return CORA_OK;
}

// Split-K GEMM into the partial workspace (plan p with p.splits > 1).
static cora_status gemm_partials(cora_model* m, GemmArgs g, const GemmPlan& p, hipStream_t s) {
  if (p.ws_floats > m->splitk_ws_floats)
    return fail(CORA_ERR_UNSUPPORTED, "shape exceeds the split-K workspace");
  g.C = m->splitk_ws;
  g.ldc = g.N;
  HIP_TRY(launch_gemm(EPI_PART_F32, g, p, s));
  return CORA_OK;
}

// Split plan for the live rows g.M with the split count planned for plan_M rows.
static GemmPlan fixed_split_plan(const cora_model* m, const GemmArgs& g, int plan_M) {
  const int splits = gemm_plan_split(plan_M, g.N, g.K, m->num_cus).splits;
  return gemm_plan_split(g.M, g.N, g.K, m->num_cus, splits);
}

// QKV projection with bias, RoPE and head layout, whole-K or split-K.
static cora_status qkv_gemm(cora_model* m, const GemmArgs& g, int plan_M, hipStream_t s) {
  const GemmPlan p = fixed_split_plan(m, g, plan_M);
  if (p.splits == 1) {
    HIP_TRY(launch_gemm(EPI_QKV_ROPE, g, p, s));
    return CORA_OK;
  }
  if (cora_status st = gemm_partials(m, g, p, s)) return st;
  HIP_TRY(launch_qkv_finish(m->splitk_ws, p.splits, g.M, g.N, g.bias, g.qkv, s));
  return CORA_OK;
}

// Residual update h += A . W^T; when norm_out is given it then receives rmsnorm(h) for the
// next GEMM.  Split-K plans store per-split partials and fold them into h, together with the
// norm, in one row-wise kernel.
static cora_status residual_gemm(cora_model* m, GemmArgs g, uint16_t* norm_out, int plan_M,
                                 hipStream_t s) {
  const auto& c = m->cfg;
  const GemmPlan p = fixed_split_plan(m, g, plan_M);
  float* h = reinterpret_cast<float*>(g.C);
  if (p.splits == 1) {
    HIP_TRY(launch_gemm(EPI_ADD_F32, g, p, s));
    const RowSel all{0, 0, 0, 0, 0, 0, 0, nullptr};
    if (norm_out) HIP_TRY(launch_rmsnorm(h, m->ones, norm_out, g.M, g.N, c.rms_eps, all, s));
    return CORA_OK;
  }
  if (cora_status st = gemm_partials(m, g, p, s)) return st;
  HIP_TRY(launch_residual_norm(h, m->splitk_ws, p.splits, g.M, g.N, m->ones, norm_out,
                               c.rms_eps, s));
  return CORA_OK;
}

static cora_status run_layers(cora_model* m, const int32_t* tokens, int B, int L, hipStream_t s) {
  const auto& c = m->cfg;
  const int d = c.d_model, M = B * L, Ls = round_up(L, 64), Mp = plan_rows(m, L);
  HIP_TRY(launch_embed(tokens, m->embed, m->h, M, d, c.vocab, s));
  const RowSel all{0, L, 0, 0, 0, 0, 0, nullptr};
  HIP_TRY(launch_rmsnorm(m->h, m->ones, m->a, M, d, c.rms_eps, all, s));
  const size_t n_layers = m->layers.size();
  for (size_t l = 0; l < n_layers; ++l) {
    const auto& ly = m->layers[l];
    // m->a holds rmsnorm(h) of this layer's input
    GemmArgs g{m->a, d, ly.wqkv, d, M, m->qkv_n, d, nullptr, 0, ly.bqkv, 1.0f};
    g.w_packed = true;
    g.qkv = QkvOut{m->q, m->k, m->vt, m->rope_cos, m->rope_sin, L, Ls, c.n_heads, c.n_kv_heads,
                   c.head_dim};
    if (cora_status st = qkv_gemm(m, g, Mp, s)) return st;
    HIP_TRY(launch_attention(m->q, m->k, m->vt, m->attn, B, L, Ls, c.n_heads, c.n_kv_heads,
                             c.head_dim, m->max_batch, m->num_cus, s));
    g = GemmArgs{m->attn, m->hq, ly.wo, m->hq, M, d, m->hq, m->h, d, nullptr, 1.0f};
    g.w_packed = true;
    if (cora_status st = residual_gemm(m, g, m->a, Mp, s)) return st;
    g = GemmArgs{m->a, d, ly.wgu, d, M, 2 * m->f_pad, d, m->u, m->f_pad, nullptr, 1.0f};
    g.w_packed = true;
    if (cora_status st = gemm(m, EPI_SWIGLU, g, s, m->timing)) return st;
    g = GemmArgs{m->u, m->f_pad, ly.wd, m->f_pad, M, d, m->f_pad, m->h, d, nullptr, 1.0f};
    g.w_packed = true;
    // the last layer's output is normalised only on the rows the LM head reads
    if (cora_status st = residual_gemm(m, g, l + 1 < n_layers ? m->a : nullptr, Mp, s))
      return st;
  }
  return CORA_OK;
}

// few rows read the packed weights (HBM-bound stream), more rows take the tiled GEMM; the
// choice is made for the planned row count (max_batch x rows per batch row)
static bool lm_head_few_rows(const cora_model* m, int plan_out_rows) {
  return m->lm_head_packed && plan_out_rows <= LM_HEAD_FUSED_MAX_ROWS &&
         lm_head_supported(plan_out_rows, m->cfg.vocab, m->cfg.d_model, m->cfg.d_model);
}

static LmHeadArgs lm_args(const cora_model* m, int n_out_rows) {
  const auto& c = m->cfg;
  LmHeadArgs a{};
  a.A = m->a; a.lda = c.d_model; a.Wp = m->lm_head_packed;
  a.M = n_out_rows; a.N = c.vocab; a.K = c.d_model; a.scale = c.logit_scale;
  a.part_m = m->lmh_pm; a.part_s = m->lmh_ps; a.part_arg = m->lmh_pa;
  a.mask_id = c.mask_id;
  return a;
}

static cora_status lm_head(cora_model* m, const RowSel& sel, int n_out_rows, int plan_out_rows,
                           uint16_t* logits, hipStream_t s) {
  const auto& c = m->cfg;
  HIP_TRY(launch_rmsnorm(m->h, m->ones, m->a, n_out_rows, c.d_model, c.rms_eps, sel, s));
  if (lm_head_few_rows(m, plan_out_rows)) {
    LmHeadArgs a = lm_args(m, n_out_rows);
    a.logits = logits;
    a.ldc = c.vocab;
    HIP_TRY(launch_lm_head(a, false, s));
    return CORA_OK;
  }
  GemmArgs g{m->a, c.d_model, m->lm_head, c.d_model, n_out_rows, c.vocab, c.d_model, logits,
             c.vocab, nullptr, c.logit_scale};
  return gemm(m, EPI_BF16, g, s);
}

// Scores of the selected rows (Eq. 1) into top1/conf[b * out_ld + out_off + r], fused into
// the LM-head pass (no logits written): the packed-weight stream for few rows, the tiled
// GEMM's EPI_TOP1 epilogue for more; logits then the row reduction only where the partials
// do not fit the logits buffer.
static cora_status score_rows(cora_model* m, const RowSel& sel, int B, int n_rows,
                              const VocabGateArgs& vg, hipStream_t s) {
  const auto& c = m->cfg;
  const int M = B * n_rows, Mp = plan_rows(m, n_rows);
  if (lm_head_few_rows(m, Mp)) {
    HIP_TRY(launch_rmsnorm(m->h, m->ones, m->a, M, c.d_model, c.rms_eps, sel, s));
    const LmHeadArgs a = lm_args(m, M);
    HIP_TRY(launch_lm_head(a, true, s));
    HIP_TRY(launch_top1_merge(a, n_rows, vg.out_ld, vg.out_off, vg.top1, vg.conf, s));
    return CORA_OK;
  }
  // more rows: the tiled GEMM folds each wavefront's logit columns into per-row partials
  // (EPI_TOP1), held in the logits buffer, which this path leaves otherwise unused.  The
  // tile config (which sets the columns a partial covers) is the planned row count's.
  const GemmPlan pp = gemm_plan(Mp, c.vocab, c.d_model, m->num_cus);
  const GemmPlan p = gemm_plan_cfg(M, c.vocab, c.d_model, pp.cfg, 1);
  const int np = gemm_top1_parts(p, c.vocab);
  const size_t part_bytes = align_up((size_t)M * np * 4);
  if (3 * align_up((size_t)Mp * np * 4) <= (size_t)m->max_batch * m->max_rows * c.vocab * 2) {
    HIP_TRY(launch_rmsnorm(m->h, m->ones, m->a, M, c.d_model, c.rms_eps, sel, s));
    GemmArgs g{m->a, c.d_model, m->lm_head, c.d_model, M, c.vocab, c.d_model, nullptr, 0,
               nullptr, c.logit_scale};
    char* buf = reinterpret_cast<char*>(m->logits);
    g.part_m = reinterpret_cast<float*>(buf);
    g.part_s = reinterpret_cast<float*>(buf + part_bytes);
    g.part_arg = reinterpret_cast<int*>(buf + 2 * part_bytes);
    g.n_parts = np;
    g.mask_id = c.mask_id;
    HIP_TRY(launch_gemm(EPI_TOP1, g, p, s));
    HIP_TRY(launch_top1_merge_parts(g.part_m, g.part_s, g.part_arg, np, M, n_rows, vg.out_ld,
                                    vg.out_off, vg.top1, vg.conf, s));
    return CORA_OK;
  }
  if (cora_status e = lm_head(m, sel, M, Mp, m->logits, s)) return e;
  VocabGateArgs r = vg;
  r.logits = m->logits;
  r.n_rows = n_rows;
  HIP_TRY(launch_vocab_top1(r, s));
  return CORA_OK;
}

extern "C" cora_status cora_forward_logits(cora_model* m, const int32_t* d_tokens, int32_t B,
                                           int32_t L, int32_t row_begin, int32_t n_rows,
                                           uint16_t* d_logits, void* hip_stream) try {
  if (!m || !d_tokens || !d_logits) return fail(CORA_ERR_INVALID_ARG, "null argument");
  if (B <= 0 || L <= 0 || B > m->max_batch || L > m->max_seq)
    return fail(CORA_ERR_INVALID_ARG, "B/L outside [1, max_batch] x [1, max_seq]");
  if (row_begin < 0 || n_rows < 0 || row_begin + n_rows > L)
    return fail(CORA_ERR_INVALID_ARG, "rows outside the canvas");
  if (n_rows == 0) return CORA_OK;
  const hipStream_t s = S(hip_stream);
  if (cora_status st = run_layers(m, d_tokens, B, L, s)) return st;
  const RowSel sel{1, L, n_rows, row_begin, 0, 0, 0, nullptr};
  return lm_head(m, sel, B * n_rows, plan_rows(m, n_rows), d_logits, s);
} catch (...) {
  return exception_status();
}

// ---- decision rules ----------------------------------------------------------------------
static cora_status check_sched_gate(const cora_sched_cfg* sc, const cora_gate_cfg* gt) {
  if (!sc || !gt) return fail(CORA_ERR_INVALID_ARG, "null sched or gate");
  if (sc->block_len < 1 || sc->block_len > CORA_MAX_BLOCK_LEN)
    return fail(CORA_ERR_UNSUPPORTED, "block_len must lie in [1, 256]");
  if (sc->steps_per_block < 1 || sc->steps_per_block > sc->block_len)
    return fail(CORA_ERR_INVALID_ARG, "steps_per_block must lie in [1, block_len]");
  if (gt->persist_scope != 0 && gt->persist_scope != 1)
    return fail(CORA_ERR_UNSUPPORTED, "persist_scope must be 0 (BLOCK) or 1 (GLOBAL)");
  if (gt->m_req < 0 || isnan(gt->delta_p))
    return fail(CORA_ERR_INVALID_ARG, "m_req must be >= 0 and delta_p a number");
  return CORA_OK;
}

static cora_status check_state(const cora_state* st, const cora_sched_cfg* sc) {
  if (!st) return fail(CORA_ERR_INVALID_ARG, "null state");
  if (!st->tokens || !st->unresolved || !st->prev_top1 || !st->persist || !st->block_idx ||
      !st->step_idx || !st->top1 || !st->conf || !st->decision || !st->done)
    return fail(CORA_ERR_INVALID_ARG, "null state array");
  if (st->B <= 0 || st->prompt_len < 0 || st->gen_len <= 0 || st->gen_len % sc->block_len != 0)
    return fail(CORA_ERR_INVALID_ARG, "B > 0, prompt_len >= 0, gen_len a positive multiple "
                                      "of block_len");
  return CORA_OK;
}

static VocabGateArgs vg_args(const uint16_t* logits, int n_rows, int row_begin, int V,
                             int mask_id, const cora_state* st, int k_transfer,
                             const cora_sched_cfg* sc, const cora_gate_cfg* gt) {
  VocabGateArgs a{};
  a.logits = logits; a.n_rows = n_rows; a.row_begin = row_begin; a.V = V; a.mask_id = mask_id;
  a.tokens = st->tokens; a.unresolved = st->unresolved; a.prev_top1 = st->prev_top1;
  a.persist = st->persist; a.block_idx = st->block_idx; a.step_idx = st->step_idx;
  a.top1 = st->top1; a.conf = st->conf; a.decision = st->decision; a.done = st->done;
  a.passes = st->passes;
  a.B = st->B; a.L = st->prompt_len + st->gen_len; a.prompt_len = st->prompt_len;
  a.block_len = sc->block_len; a.steps_per_block = sc->steps_per_block;
  a.n_blocks = st->gen_len / sc->block_len;
  a.k_transfer = k_transfer;
  a.delta_p = gt->delta_p; a.m_req = gt->m_req; a.gate_enabled = gt->gate_enabled ? 1 : 0;
  a.persist_scope = gt->persist_scope;
  a.out_ld = n_rows;
  a.out_off = 0;
  a.eos_enabled = sc->eos_enabled ? 1 : 0;
  a.eos_id = sc->eos_id;
  return a;
}

static cora_status check_vocab_gate(const uint16_t* d_logits, int32_t n_rows, int32_t row_begin,
                                    int32_t V, int32_t mask_id, const cora_state* st,
                                    const cora_sched_cfg* sc, const cora_gate_cfg* gt) {
  if (cora_status e = check_sched_gate(sc, gt)) return e;
  if (cora_status e = check_state(st, sc)) return e;
  if (!d_logits) return fail(CORA_ERR_INVALID_ARG, "null logits");
  if (V < 2 || mask_id < 0 || mask_id >= V) return fail(CORA_ERR_INVALID_ARG, "bad V/mask_id");
  if (sc->eos_enabled && (sc->eos_id < 0 || sc->eos_id >= V))
    return fail(CORA_ERR_INVALID_ARG, "eos_id must lie in [0, V)");
  const int L = st->prompt_len + st->gen_len;
  if (row_begin >= 0) {
    if (row_begin > st->prompt_len || row_begin + n_rows < L || row_begin + n_rows > L)
      return fail(CORA_ERR_INVALID_ARG, "fixed rows must cover the generation region and stay "
                                        "inside the canvas");
  } else if (n_rows != sc->block_len) {
    return fail(CORA_ERR_INVALID_ARG, "block-following rows need n_rows == block_len");
  } else if (gt->persist_scope == 1) {
    return fail(CORA_ERR_INVALID_ARG, "the GLOBAL persistence scope needs fixed rows covering "
                                      "the generation region");
  }
  if (n_rows <= 0) return fail(CORA_ERR_INVALID_ARG, "n_rows must be positive");
  return CORA_OK;
}

extern "C" cora_status cora_vocab_gate(const uint16_t* d_logits, int32_t n_rows, int32_t row_begin,
                                       int32_t V, int32_t mask_id, cora_state* st,
                                       int32_t k_transfer, const cora_sched_cfg* sc,
                                       const cora_gate_cfg* gt, void* hip_stream) try {
  if (cora_status e = check_vocab_gate(d_logits, n_rows, row_begin, V, mask_id, st, sc, gt))
    return e;
  const VocabGateArgs a = vg_args(d_logits, n_rows, row_begin, V, mask_id, st, k_transfer, sc, gt);
  HIP_TRY(launch_vocab_top1(a, S(hip_stream)));
  HIP_TRY(launch_gate_rules(a, S(hip_stream)));
  return CORA_OK;
} catch (...) {
  return exception_status();
}

// ---- the vocab/gate kernels with a fixed scratch array --------------------------------------
// Partials of the split row reduction live in `scratch`, a file-scope device array (one copy
// per GPU, held until the process ends).  In host code the array's name is only a host-side
// stand-in: its device address is looked up once per device with hipGetSymbolAddress, with
// that device current, and only that address is handed to kernels.  Every call on one GPU
// shares the array and overwrites the partials it reads (nothing must start at zero), so
// calls that overlap on one GPU race.
constexpr int64_t NOALLOC_PARTIALS = CORA_VOCAB_GATE_NOALLOC_MAX_PARTIALS;
constexpr int MAX_DEVICES = 64;
static __device__ __align__(256) unsigned char scratch[NOALLOC_PARTIALS * 12];
static std::mutex g_scratch_mu;
static void* g_scratch_ptr[MAX_DEVICES];
static int g_scratch_cus[MAX_DEVICES];

#define HIP_TRY_NOALLOC(expr)                                                        \
  do {                                                                               \
    hipError_t e_ = (expr);                                                          \
    if (e_ != hipSuccess) {                                                          \
      (void)hipGetLastError();                                                       \
      snprintf(g_err, sizeof(g_err), "%s: %s", #expr, hipGetErrorString(e_));        \
      return CORA_ERR_HIP;                                                           \
    }                                                                                \
  } while (0)

static cora_status scratch_of_current_device(void** ptr, int* num_cus) {
  int dev = 0;
  HIP_TRY_NOALLOC(hipGetDevice(&dev));
  if (dev < 0 || dev >= MAX_DEVICES) return fail(CORA_ERR_UNSUPPORTED, "device index >= 64");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    HIP_TRY_NOALLOC(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (!p) return fail(CORA_ERR_HIP, "hipGetSymbolAddress returned a null scratch address");
    int cus = 0;
    HIP_TRY_NOALLOC(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
    g_scratch_cus[dev] = cus > 0 ? cus : 256;
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  *num_cus = g_scratch_cus[dev];
  return CORA_OK;
}

extern "C" cora_status cora_vocab_gate_noalloc(const uint16_t* d_logits, int32_t n_rows,
                                               int32_t row_begin, int32_t V, int32_t mask_id,
                                               cora_state* st, int32_t k_transfer,
                                               const cora_sched_cfg* sc, const cora_gate_cfg* gt,
                                               void* hip_stream) try {
  if (cora_status e = check_vocab_gate(d_logits, n_rows, row_begin, V, mask_id, st, sc, gt))
    return e;
  const int64_t rows = (int64_t)st->B * n_rows;
  if (rows > NOALLOC_PARTIALS)
    return fail(CORA_ERR_UNSUPPORTED, "B * n_rows exceeds the fixed scratch of "
                                      "cora_vocab_gate_noalloc (262144 rows)");
  void* base = nullptr;
  int cus = 0;
  if (cora_status e = scratch_of_current_device(&base, &cus)) return e;
  const VocabGateArgs a = vg_args(d_logits, n_rows, row_begin, V, mask_id, st, k_transfer, sc, gt);
  VocabSplit sp{};
  sp.parts = vocab_split_parts((int)rows, V, cus, NOALLOC_PARTIALS);
  sp.pm = reinterpret_cast<float*>(base);
  sp.ps = sp.pm + NOALLOC_PARTIALS;
  sp.pa = reinterpret_cast<int*>(sp.ps + NOALLOC_PARTIALS);
  HIP_TRY_NOALLOC(launch_vocab_top1_split(a, sp, S(hip_stream)));
  HIP_TRY_NOALLOC(launch_gate_rules(a, S(hip_stream)));
  return CORA_OK;
} catch (...) {
  return exception_status();
}

static cora_status denoise_step(cora_model* m, cora_state* st, const cora_sched_cfg* sc,
                                const cora_gate_cfg* gt, hipStream_t s) {
  const int B = st->B, L = st->prompt_len + st->gen_len, blk = sc->block_len;
  if (cora_status e = run_layers(m, st->tokens, B, L, s)) return e;
  if (gt->persist_scope == 1) {
    // GLOBAL: score the whole generation region, in chunks of the row workspace, into
    // top1/conf [B, gen_len]; then the rules read every unresolved position's score
    const int G = st->gen_len;
    VocabGateArgs a = vg_args(m->logits, G, st->prompt_len, m->cfg.vocab, m->cfg.mask_id, st,
                              -1, sc, gt);
    for (int r0 = 0; r0 < G; r0 += m->max_rows) {
      const int n = G - r0 < m->max_rows ? G - r0 : m->max_rows;
      const RowSel sel{1, L, n, st->prompt_len + r0, 0, 0, 0, nullptr};
      VocabGateArgs c = a;
      c.out_off = r0;
      if (cora_status e = score_rows(m, sel, B, n, c, s)) return e;
    }
    HIP_TRY(launch_gate_rules(a, s));
    return CORA_OK;
  }
  const RowSel sel{2, L, blk, 0, st->prompt_len, blk, st->gen_len / blk, st->block_idx};
  const VocabGateArgs a = vg_args(m->logits, blk, -1, m->cfg.vocab, m->cfg.mask_id, st, -1, sc,
                                  gt);
  if (cora_status e = score_rows(m, sel, B, blk, a, s)) return e;
  HIP_TRY(launch_gate_rules(a, s));
  return CORA_OK;
}

static cora_status check_step(cora_model* m, const cora_state* st, const cora_sched_cfg* sc,
                              const cora_gate_cfg* gt) {
  if (!m) return fail(CORA_ERR_INVALID_ARG, "null model");
  if (cora_status e = check_sched_gate(sc, gt)) return e;
  if (cora_status e = check_state(st, sc)) return e;
  if (st->B > m->max_batch || st->prompt_len + st->gen_len > m->max_seq)
    return fail(CORA_ERR_INVALID_ARG, "state exceeds the model's max_batch / max_seq");
  if (sc->block_len > m->max_rows)
    return fail(CORA_ERR_INVALID_ARG, "block_len exceeds the model's row workspace");
  if (sc->eos_enabled && (sc->eos_id < 0 || sc->eos_id >= m->cfg.vocab))
    return fail(CORA_ERR_INVALID_ARG, "eos_id must lie in [0, vocab)");
  return CORA_OK;
}

extern "C" cora_status cora_denoise_step(cora_model* m, cora_state* st, const cora_sched_cfg* sc,
                                         const cora_gate_cfg* gt, void* hip_stream) try {
  if (cora_status e = check_step(m, st, sc, gt)) return e;
  return denoise_step(m, st, sc, gt, S(hip_stream));
} catch (...) {
  return exception_status();
}

extern "C" cora_status cora_block_decode(cora_model* m, const int32_t* d_prompt, int32_t B,
                                         int32_t prompt_len, int32_t gen_len,
                                         const cora_sched_cfg* sc, const cora_gate_cfg* gt,
                                         int32_t* d_out_tokens, int32_t* h_passes,
                                         int32_t* h_total_passes, void* hip_stream) try {
  if (!m || !d_out_tokens || !h_passes || (prompt_len > 0 && !d_prompt))
    return fail(CORA_ERR_INVALID_ARG, "null argument");
  const hipStream_t s = S(hip_stream);
  cora_state st{m->s_tokens, m->s_unres, m->s_prev, m->s_persist, m->s_block, m->s_step,
                m->s_top1, m->s_conf, m->s_decision, m->s_done, m->s_passes,
                B, prompt_len, gen_len};
  if (cora_status e = check_step(m, &st, sc, gt)) return e;
  const int n_blocks = gen_len / sc->block_len, L = prompt_len + gen_len;
  HIP_TRY(launch_state_init(d_prompt, B, prompt_len, gen_len, m->cfg.mask_id, st.tokens,
                            st.unresolved, st.prev_top1, st.persist, st.block_idx, st.step_idx,
                            st.passes, n_blocks, s));
  const int64_t max_passes = (int64_t)n_blocks * sc->steps_per_block;
  int64_t total = 0;
  // Rows decode independently (the dense pass attends within a row), so once rows finish
  // their final tokens and passes are written out and the live rows are gathered into the
  // other state buffer set; later passes run on those rows only.  orig[i] is the caller's
  // row of compact row i.
  DecodeRows cur{st.tokens, st.unresolved, st.prev_top1, st.persist, st.block_idx,
                 st.step_idx, st.passes};
  DecodeRows alt = m->s_alt;
  std::vector<int32_t> orig(B);
  for (int b = 0; b < B; ++b) orig[b] = b;
  int Bc = B;
  // final rows of the compact state -> outputs (rows listed in h_map[0, n), originals after)
  auto write_out = [&](const std::vector<int32_t>& rows) -> cora_status {
    const int n = (int)rows.size();
    for (int i = 0; i < n; ++i) {
      m->h_map[i] = rows[i];
      m->h_map[n + i] = orig[rows[i]];
    }
    HIP_TRY(hipMemcpyAsync(m->d_map, m->h_map, 2 * n * sizeof(int32_t), hipMemcpyHostToDevice, s));
    HIP_TRY(launch_scatter_rows(cur.tokens, cur.passes, m->d_map, m->d_map + n, n, L, n_blocks,
                                d_out_tokens, m->s_final_passes, s));
    return CORA_OK;
  };
  for (;;) {
    if (cora_status e = denoise_step(m, &st, sc, gt, s)) return e;
    ++total;
    HIP_TRY(hipMemcpyAsync(m->h_block, st.block_idx, Bc * sizeof(int32_t), hipMemcpyDeviceToHost,
                           s));
    HIP_TRY(hipStreamSynchronize(s));  // also: every earlier use of h_map has completed
    std::vector<int32_t> fin, live;
    for (int b = 0; b < Bc; ++b) (m->h_block[b] >= n_blocks ? fin : live).push_back(b);
    if (live.empty()) break;
    if (total > max_passes)
      return fail(CORA_ERR_STATE, "decode did not terminate within the dense horizon");
    if (!m->compaction || fin.empty()) continue;
    if (cora_status e = write_out(fin)) return e;
    const int nl = (int)live.size();
    for (int i = 0; i < nl; ++i) m->h_map[2 * fin.size() + i] = live[i];
    HIP_TRY(hipMemcpyAsync(m->d_map + 2 * fin.size(), m->h_map + 2 * fin.size(),
                           nl * sizeof(int32_t), hipMemcpyHostToDevice, s));
    HIP_TRY(launch_gather_state(cur, alt, m->d_map + 2 * fin.size(), nl, L, n_blocks, s));
    std::swap(cur, alt);
    std::vector<int32_t> o(nl);
    for (int i = 0; i < nl; ++i) o[i] = orig[live[i]];
    orig.swap(o);
    Bc = nl;
    st.tokens = cur.tokens; st.unresolved = cur.unresolved; st.prev_top1 = cur.prev;
    st.persist = cur.persist; st.block_idx = cur.block_idx; st.step_idx = cur.step_idx;
    st.passes = cur.passes; st.B = Bc;
  }
  std::vector<int32_t> rest(Bc);
  for (int b = 0; b < Bc; ++b) rest[b] = b;
  if (cora_status e = write_out(rest)) return e;
  HIP_TRY(hipMemcpyAsync(h_passes, m->s_final_passes, (size_t)B * n_blocks * sizeof(int32_t),
                         hipMemcpyDeviceToHost, s));
  HIP_TRY(hipStreamSynchronize(s));
  if (h_total_passes) *h_total_passes = (int32_t)total;
  return CORA_OK;
} catch (...) {
  return exception_status();
}

// ---- weight read-back in logical [out, in] layout ---------------------------------------
// Row-major host copy of a layer matrix stored in 64 x 64 blocks (physical rows x ld).
static cora_status read_packed(const uint16_t* d_packed, int64_t rows, int64_t ld,
                               std::vector<uint16_t>& out) {
  std::vector<uint16_t> p((size_t)(rows * ld));
  HIP_TRY(hipMemcpy(p.data(), d_packed, p.size() * 2, hipMemcpyDeviceToHost));
  out.resize(p.size());
  for (int64_t r = 0; r < rows; ++r)
    for (int64_t c = 0; c < ld; ++c)
      out[(size_t)(r * ld + c)] = p[(size_t)(((r >> 6) * (ld >> 6) + (c >> 6)) * 4096 +
                                             (r & 63) * 64 + (c & 63))];
  return CORA_OK;
}

extern "C" cora_status cora_model_copy_tensor(cora_model* m, int32_t tensor_id, void* h_dst,
                                              size_t bytes) try {
  if (!m || !h_dst) return fail(CORA_ERR_INVALID_ARG, "null argument");
  const auto& c = m->cfg;
  const int d = c.d_model;
  auto want = [&](size_t n) -> cora_status {
    return bytes == n * 2 ? CORA_OK
                          : fail(CORA_ERR_INVALID_ARG, "bytes does not match the tensor size");
  };
  if (tensor_id == 1 || tensor_id == 2) {
    if (cora_status e = want((size_t)c.vocab * d)) return e;
    HIP_TRY(hipMemcpy(h_dst, tensor_id == 1 ? m->embed : m->lm_head, bytes, hipMemcpyDeviceToHost));
    return CORA_OK;
  }
  if (tensor_id < 100) return fail(CORA_ERR_INVALID_ARG, "unknown tensor id");
  const int l = (tensor_id - 100) / 16, j = (tensor_id - 100) % 16;
  if (l >= c.n_layers) return fail(CORA_ERR_INVALID_ARG, "layer out of range");
  const auto& ly = m->layers[l];
  uint16_t* out = reinterpret_cast<uint16_t*>(h_dst);
  switch (j) {
    case 0: case 1: case 2: {
      const int rows = j == 0 ? m->hq : m->hkv;
      const int off = j == 0 ? 0 : (j == 1 ? m->hq : m->hq + m->hkv);
      if (cora_status e = want((size_t)rows * d)) return e;
      std::vector<uint16_t> tmp;
      if (cora_status e = read_packed(ly.wqkv, m->qkv_n, d, tmp)) return e;
      const int hd = c.head_dim;
      for (int r = 0; r < rows; ++r) {  // undo the per-head pair interleave of q and k
        const size_t pr = off + (j == 2 ? r : (size_t)(r / hd) * hd + rope_pair_pos(r % hd, hd));
        memcpy(out + (size_t)r * d, tmp.data() + pr * d, (size_t)d * 2);
      }
      return CORA_OK;
    }
    case 3: {
      if (cora_status e = want((size_t)d * m->hq)) return e;
      std::vector<uint16_t> tmp;
      if (cora_status e = read_packed(ly.wo, d, m->hq, tmp)) return e;
      memcpy(out, tmp.data(), bytes);
      return CORA_OK;
    }
    case 4: case 5: {
      const int F = c.ffn_dim;
      if (cora_status e = want((size_t)F * d)) return e;
      std::vector<uint16_t> tmp;
      if (cora_status e = read_packed(ly.wgu, 2 * (int64_t)m->f_pad, d, tmp)) return e;
      for (int r = 0; r < F; ++r) {
        const size_t pr = (size_t)(r >> 5) * 64 + (j == 5 ? 32 : 0) + (r & 31);
        memcpy(out + (size_t)r * d, tmp.data() + pr * d, (size_t)d * 2);
      }
      return CORA_OK;
    }
    case 6: {
      if (cora_status e = want((size_t)d * c.ffn_dim)) return e;
      std::vector<uint16_t> tmp;
      if (cora_status e = read_packed(ly.wd, d, m->f_pad, tmp)) return e;
      for (int r = 0; r < d; ++r)
        memcpy(out + (size_t)r * c.ffn_dim, tmp.data() + (size_t)r * m->f_pad,
               (size_t)c.ffn_dim * 2);
      return CORA_OK;
    }
    case 7: case 8: case 9: {
      if (!c.qkv_bias) return fail(CORA_ERR_INVALID_ARG, "model has no qkv bias");
      const int n = j == 7 ? m->hq : m->hkv;
      const int off = j == 7 ? 0 : (j == 8 ? m->hq : m->hq + m->hkv);
      if (cora_status e = want((size_t)n)) return e;
      std::vector<float> tmp(n);
      HIP_TRY(hipMemcpy(tmp.data(), ly.bqkv + off, (size_t)n * 4, hipMemcpyDeviceToHost));
      const int hd = c.head_dim;
      for (int i = 0; i < n; ++i) {
        const int pi = j == 9 ? i : (i / hd) * hd + rope_pair_pos(i % hd, hd);
        uint32_t u;
        memcpy(&u, &tmp[pi], 4);
        out[i] = (uint16_t)(u >> 16);
      }
      return CORA_OK;
    }
  }
  return fail(CORA_ERR_INVALID_ARG, "unknown tensor id");
} catch (...) {
  return exception_status();
}
