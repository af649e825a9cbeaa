// Host side of the libsevo C ABI: argument validation, split / workspace
// planning, the model handle (RoPE table) and the decode-step composition.
// Every entry point catches everything and reports through sevo_status.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/sevo.h"
#include "kernels.h"

#define SEVO_API extern "C" __attribute__((visibility("default")))

namespace {

thread_local std::string g_err;

sevo_status fail(sevo_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return s;
}

sevo_status hip_fail(hipError_t e, const char* where) {
  return fail(SEVO_ERR_HIP, "%s: %s", where, hipGetErrorString(e));
}

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

inline size_t round_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

bool supported_group(int hq, int hkv) {
  if (hkv <= 0 || hq <= 0 || hq % hkv) return false;
  const int g = hq / hkv;
  return g == 1 || g == 2 || g == 4 || g == 8;
}

// A split spans at most this many logical pages (128 per wave of the split
// kernel, whose page ids are then held one per lane in two registers).
constexpr int kMaxSplitPages = 512;

int min_splits(int max_pages) { return (max_pages + kMaxSplitPages - 1) / kMaxSplitPages; }

// Splits per candidate.  About 512 split workgroups are resident at once (2
// per CU); every split adds a fixed cost (its start-up, partial write and
// combine share), while a count whose n * hkv * S leaves the last round of
// resident workgroups part-empty idles CUs.  So: the fewest splits (at least
// the kMaxSplitPages minimum) that fill one round, raised (up to doubling) to
// the first count that fills whole rounds; at least 32 pages (8 per wave)
// per split where the minimum allows.  Measured on the matrix-core kernel:
// 64 x 8 pairs at 16k-32k -> 4, 16 x 8 pairs at 64k -> 12 (9 and 10 are 7%
// slower), 16 x 8 at 8k-16k -> 4 (28 is 20% slower), 64 x 4 pairs at
// 16k-32k -> 8 (4: 525 against 510 us).
constexpr int kResidentSplitGroups = 512;

int plan_splits(int n, int hkv, int max_pages) {
  const long long pairs = (long long)(n > 0 ? n : 1) * (hkv > 0 ? hkv : 1);
  const int smin = min_splits(max_pages);
  int cap = (max_pages + 31) / 32;
  if (cap < smin) cap = smin;
  long long s = smin;
  if (pairs * s < kResidentSplitGroups) s = (kResidentSplitGroups + pairs - 1) / pairs;
  if (s > cap) return cap;
  for (long long t = s; t <= 2 * s && t <= cap; ++t)
    if ((pairs * t) % kResidentSplitGroups == 0) {
      s = t;
      break;
    }
  // fewer than three rounds of long splits leave a ragged last round (short
  // candidates have empty or partial last splits): twice the splits, while
  // each still spans at least 192 pages
  if (pairs * s < 3 * kResidentSplitGroups && 2 * s <= cap &&
      (max_pages + 2 * s - 1) / (2 * s) >= 192)
    s *= 2;
  return (int)s;
}

// The split count actually used: the requested (or planned) count, raised so
// that no split exceeds kMaxSplitPages, then trimmed so every split is used.
void resolve_splits(int n, int hkv, int max_pages, int requested, int* S, int* chunk) {
  int s = requested > 0 ? requested : plan_splits(n, hkv, max_pages);
  if (s < min_splits(max_pages)) s = min_splits(max_pages);
  if (s > max_pages) s = max_pages;
  const int c = (max_pages + s - 1) / s;
  *chunk = c;
  *S = (max_pages + c - 1) / c;
}

size_t attn_ws(int n, int hq, int d, int S) {
  return round_up((size_t)n * hq * S * 2 * sizeof(float), 256) +
         round_up((size_t)n * hq * S * d * sizeof(float), 256);
}

struct AttnCheck {
  int S, chunk;
};

sevo_status check_attn_shape(int n, int hq, int hkv, int d, int page_size, int max_pages) {
  if (n < 0) return fail(SEVO_ERR_INVALID_ARGUMENT, "n = %d < 0", n);
  if (page_size != SEVO_PAGE_SIZE)
    return fail(SEVO_ERR_UNSUPPORTED, "page_size %d != 16", page_size);
  if (d != 64 && d != 128) return fail(SEVO_ERR_UNSUPPORTED, "head_dim %d not in {64, 128}", d);
  if (!supported_group(hq, hkv))
    return fail(SEVO_ERR_UNSUPPORTED, "n_q_heads %d / n_kv_heads %d: group must be 1, 2, 4 or 8",
                hq, hkv);
  if (max_pages < 1) return fail(SEVO_ERR_INVALID_ARGUMENT, "max_pages %d < 1", max_pages);
  return SEVO_OK;
}

// Kernel timing (see sevo_profile_begin): HIP events recorded on the launch
// stream around the launches of the selected kinds.  Process-wide, guarded by
// a mutex; events come from a pool created by sevo_profile_begin.
struct ProfRecord {
  int kind;
  hipEvent_t b, e;
};
struct Profiler {
  std::mutex mu;
  bool on = false;
  uint32_t mask = 0;
  std::vector<hipEvent_t> pool;
  size_t used = 0;
  std::vector<ProfRecord> recs;
  bool want(int kind) const { return on && ((mask >> kind) & 1u); }
  hipEvent_t take() { return used < pool.size() ? pool[used++] : nullptr; }
} g_prof;

void attach_profiler(sevo::AttnArgs& a) {
  std::lock_guard<std::mutex> lk(g_prof.mu);
  const bool ws = g_prof.want(SEVO_PROF_ATTN_SPLIT), wc = g_prof.want(SEVO_PROF_ATTN_COMBINE);
  if (!ws && !wc) return;
  if (g_prof.used + 3 > g_prof.pool.size()) return;
  a.ev_begin = g_prof.take();
  a.ev_mid = g_prof.take();
  a.ev_end = g_prof.take();
  if (ws) g_prof.recs.push_back({SEVO_PROF_ATTN_SPLIT, a.ev_begin, a.ev_mid});
  if (wc) g_prof.recs.push_back({SEVO_PROF_ATTN_COMBINE, a.ev_mid, a.ev_end});
}

// Brackets one launch (or a few) of the given kind on stream st.
class ProfScope {
 public:
  ProfScope(int kind, hipStream_t st) : kind_(kind), st_(st) {
    std::lock_guard<std::mutex> lk(g_prof.mu);
    if (!g_prof.want(kind) || g_prof.used + 2 > g_prof.pool.size()) return;
    b_ = g_prof.take();
    e_ = g_prof.take();
    (void)hipEventRecord(b_, st_);
  }
  ~ProfScope() {
    if (!b_) return;
    (void)hipEventRecord(e_, st_);
    std::lock_guard<std::mutex> lk(g_prof.mu);
    g_prof.recs.push_back({kind_, b_, e_});
  }
  ProfScope(const ProfScope&) = delete;
  ProfScope& operator=(const ProfScope&) = delete;

 private:
  int kind_;
  hipStream_t st_;
  hipEvent_t b_ = nullptr, e_ = nullptr;
};

}  // namespace

struct sevo_model {
  sevo_model_config cfg;
  const void* embed;
  const void* lm_head;
  const void* final_norm;
  std::vector<const void*> attn_norm, w_qkv, q_norm, k_norm, w_o, ffn_norm, w_gate_up, w_down;
  std::vector<const void*> w_router, w_expert_gate_up, w_expert_down;  // MoE models
  float* rope_cos = nullptr;
  float* rope_sin = nullptr;
  int device = 0;
};

SEVO_API const char* sevo_status_string(sevo_status s) {
  switch (s) {
    case SEVO_OK: return "ok";
    case SEVO_ERR_INVALID_ARGUMENT: return "invalid argument";
    case SEVO_ERR_UNSUPPORTED: return "unsupported";
    case SEVO_ERR_WORKSPACE_TOO_SMALL: return "workspace too small";
    case SEVO_ERR_OUT_OF_MEMORY: return "out of memory";
    case SEVO_ERR_HIP: return "HIP error";
    case SEVO_ERR_BAD_PAGE_TABLE: return "bad page table";
    default: return "unknown status";
  }
}

SEVO_API const char* sevo_last_error(void) { return g_err.c_str(); }

SEVO_API const char* sevo_version(void) { return "sevo 0.1 gfx950"; }

// ------------------------------------------------------------------ model
SEVO_API sevo_status sevo_init_model(const sevo_model_config* cfg, const sevo_weights* w,
                                     sevo_model** out) {
  try {
    if (!cfg || !w || !out) return fail(SEVO_ERR_INVALID_ARGUMENT, "null argument");
    *out = nullptr;
    const sevo_model_config& c = *cfg;
    const bool moe = c.n_experts > 0;
    if (c.n_layers < 1 || c.hidden < 1 || c.vocab < 1 || (!moe && c.ffn < 1) ||
        c.n_experts < 0)
      return fail(SEVO_ERR_INVALID_ARGUMENT, "non-positive model size");
    if (moe && !sevo::moe_supported(c.n_experts, c.n_experts_active, c.expert_ffn, c.hidden))
      return fail(SEVO_ERR_UNSUPPORTED,
                  "MoE: n_experts %d (multiple of 64, <= 256), n_experts_active %d (1..16), "
                  "expert_ffn %d (multiple of 32)", c.n_experts, c.n_experts_active,
                  c.expert_ffn);
    if (c.max_position < 1) return fail(SEVO_ERR_INVALID_ARGUMENT, "max_position < 1");
    if (!(c.rms_eps > 0.f) || !(c.rope_theta > 1.f))
      return fail(SEVO_ERR_INVALID_ARGUMENT, "rms_eps must be > 0 and rope_theta > 1");
    if (c.qk_norm != 0 && c.qk_norm != 1) return fail(SEVO_ERR_INVALID_ARGUMENT, "qk_norm");
    sevo_status st = check_attn_shape(1, c.n_q_heads, c.n_kv_heads, c.head_dim, c.page_size, 1);
    if (st) return st;
    if (c.hidden % 128 || (!moe && c.ffn % 128) || (c.n_q_heads * c.head_dim) % 128 ||
        c.vocab % 64)
      return fail(SEVO_ERR_UNSUPPORTED, "hidden, ffn and n_q_heads*head_dim must be multiples "
                                        "of 128 and vocab of 64");
    if (!w->embed || !w->lm_head || !w->final_norm)
      return fail(SEVO_ERR_INVALID_ARGUMENT, "null embed / lm_head / final_norm");
    const void* const* tabs[] = {w->attn_norm, w->w_qkv, w->w_o, w->ffn_norm,
                                 moe ? w->w_router : w->w_gate_up,
                                 moe ? w->w_expert_gate_up : w->w_down,
                                 moe ? w->w_expert_down : w->w_down};
    for (auto t : tabs)
      if (!t) return fail(SEVO_ERR_INVALID_ARGUMENT, "null per-layer weight table");
    if (c.qk_norm && (!w->q_norm || !w->k_norm))
      return fail(SEVO_ERR_INVALID_ARGUMENT, "qk_norm needs q_norm and k_norm tables");
    const size_t rope_bytes = (size_t)c.max_position * (c.head_dim / 2) * sizeof(float);
    if (rope_bytes > (size_t)16 << 30)
      return fail(SEVO_ERR_OUT_OF_MEMORY, "RoPE table of %zu bytes exceeds 16 GiB", rope_bytes);

    sevo_model* m = new sevo_model();
    m->cfg = c;
    m->embed = w->embed;
    m->lm_head = w->lm_head;
    m->final_norm = w->final_norm;
    for (int l = 0; l < c.n_layers; ++l) {
      m->attn_norm.push_back(w->attn_norm[l]);
      m->w_qkv.push_back(w->w_qkv[l]);
      m->q_norm.push_back(c.qk_norm ? w->q_norm[l] : nullptr);
      m->k_norm.push_back(c.qk_norm ? w->k_norm[l] : nullptr);
      m->w_o.push_back(w->w_o[l]);
      m->ffn_norm.push_back(w->ffn_norm[l]);
      m->w_gate_up.push_back(moe ? nullptr : w->w_gate_up[l]);
      m->w_down.push_back(moe ? nullptr : w->w_down[l]);
      m->w_router.push_back(moe ? w->w_router[l] : nullptr);
      m->w_expert_gate_up.push_back(moe ? w->w_expert_gate_up[l] : nullptr);
      m->w_expert_down.push_back(moe ? w->w_expert_down[l] : nullptr);
      const void* need[] = {m->attn_norm[l], m->w_qkv[l], m->w_o[l], m->ffn_norm[l],
                            moe ? m->w_router[l] : m->w_gate_up[l],
                            moe ? m->w_expert_gate_up[l] : m->w_down[l],
                            moe ? m->w_expert_down[l] : m->w_down[l]};
      for (auto p : need)
        if (!p || !aligned16(p)) {
          delete m;
          return fail(SEVO_ERR_INVALID_ARGUMENT, "layer %d: null or misaligned weight", l);
        }
    }
    // RoPE table: angle p * theta^(-2m/d) in double, cos/sin stored fp32
    const int half = c.head_dim / 2;
    std::vector<float> hc((size_t)c.max_position * half), hs(hc.size());
    for (int mm = 0; mm < half; ++mm) {
      const double inv = std::pow((double)c.rope_theta, -2.0 * mm / c.head_dim);
      for (int p = 0; p < c.max_position; ++p) {
        const double a = (double)p * inv;
        hc[(size_t)p * half + mm] = (float)std::cos(a);
        hs[(size_t)p * half + mm] = (float)std::sin(a);
      }
    }
    hipError_t e = hipGetDevice(&m->device);
    if (e == hipSuccess) e = hipMalloc(&m->rope_cos, rope_bytes);
    if (e == hipSuccess) e = hipMalloc(&m->rope_sin, rope_bytes);
    if (e == hipSuccess) e = hipMemcpy(m->rope_cos, hc.data(), rope_bytes, hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMemcpy(m->rope_sin, hs.data(), rope_bytes, hipMemcpyHostToDevice);
    if (e != hipSuccess) {
      const sevo_status r = e == hipErrorOutOfMemory ? fail(SEVO_ERR_OUT_OF_MEMORY, "RoPE table")
                                                      : hip_fail(e, "sevo_init_model");
      if (m->rope_cos) (void)hipFree(m->rope_cos);
      if (m->rope_sin) (void)hipFree(m->rope_sin);
      delete m;
      return r;
    }
    *out = m;
    return SEVO_OK;
  } catch (...) {
    return fail(SEVO_ERR_OUT_OF_MEMORY, "host allocation failed in sevo_init_model");
  }
}

SEVO_API void sevo_free_model(sevo_model* m) {
  if (!m) return;
  if (m->rope_cos) (void)hipFree(m->rope_cos);
  if (m->rope_sin) (void)hipFree(m->rope_sin);
  delete m;
}

// ------------------------------------------------------------------ attention
SEVO_API int32_t sevo_attn_plan_splits(int32_t n, int32_t n_kv_heads, int32_t max_pages) {
  return plan_splits(n, n_kv_heads, max_pages);
}

SEVO_API size_t sevo_attn_workspace_bytes(int32_t n, int32_t n_q_heads, int32_t n_kv_heads,
                                          int32_t head_dim, int32_t max_pages,
                                          int32_t num_splits) {
  if (n <= 0 || n_q_heads <= 0 || head_dim <= 0 || max_pages <= 0) return 0;
  int S, chunk;
  resolve_splits(n, n_kv_heads, max_pages, num_splits, &S, &chunk);
  return attn_ws(n, n_q_heads, head_dim, S);
}

static sevo_status attn_core(int n, int hq, int hkv, int d, int max_pages, int num_splits,
                             int64_t num_pages, const void* q, const void* kvp,
                             const int32_t* pt, const int32_t* lens, float scale, void* out,
                             void* ws, size_t ws_bytes, hipStream_t st) {
  int S, chunk;
  resolve_splits(n, hkv, max_pages, num_splits, &S, &chunk);
  const size_t need = attn_ws(n, hq, d, S);
  if (ws_bytes < need)
    return fail(SEVO_ERR_WORKSPACE_TOO_SMALL, "attention needs %zu workspace bytes, got %zu",
                need, ws_bytes);
  sevo::AttnArgs a;
  a.n = n; a.hq = hq; a.hkv = hkv; a.d = d; a.max_pages = max_pages; a.num_splits = S;
  a.chunk = chunk; a.num_pages = num_pages;
  a.q = static_cast<const sevo::bf16_t*>(q);
  a.kv_pool = static_cast<const sevo::bf16_t*>(kvp);
  a.page_table = pt; a.seq_lens = lens; a.len_add = 0; a.scale = scale;
  a.out = static_cast<sevo::bf16_t*>(out);
  attach_profiler(a);
  a.part_ml = static_cast<float*>(ws);
  a.part_acc = reinterpret_cast<float*>(static_cast<char*>(ws) +
                                        round_up((size_t)n * hq * S * 2 * sizeof(float), 256));
  hipError_t e = sevo::launch_attn_decode(a, st);
  if (e != hipSuccess) return hip_fail(e, "sevo_attn_decode launch");
  return SEVO_OK;
}

SEVO_API sevo_status sevo_attn_decode(const sevo_attn_args* a, void* stream) {
  if (!a) return fail(SEVO_ERR_INVALID_ARGUMENT, "null args");
  sevo_status st = check_attn_shape(a->n, a->n_q_heads, a->n_kv_heads, a->head_dim,
                                    a->page_size, a->max_pages);
  if (st) return st;
  if (a->num_splits < 0) return fail(SEVO_ERR_INVALID_ARGUMENT, "num_splits < 0");
  if (a->num_pages < 1) return fail(SEVO_ERR_INVALID_ARGUMENT, "num_pages < 1");
  if (!(std::isfinite(a->scale)) || a->scale <= 0.f)
    return fail(SEVO_ERR_INVALID_ARGUMENT, "scale must be finite and > 0");
  if (a->n == 0) return SEVO_OK;
  const void* ptrs[] = {a->q, a->kv_pool, a->page_table, a->seq_lens, a->out,
                        a->workspace};
  for (auto p : ptrs)
    if (!p || !aligned16(p))
      return fail(SEVO_ERR_INVALID_ARGUMENT, "null or non-16-byte-aligned pointer");
  return attn_core(a->n, a->n_q_heads, a->n_kv_heads, a->head_dim, a->max_pages, a->num_splits,
                   a->num_pages, a->q, a->kv_pool, a->page_table, a->seq_lens,
                   a->scale, a->out, a->workspace, a->workspace_bytes,
                   static_cast<hipStream_t>(stream));
}

// ------------------------------------------------------------------ attention, no allocation
// The split partials of sevo_attn_decode_noalloc live in this fixed array:
// each GPU the library runs on holds its own copy until the process ends.  In
// host code the name `scratch` is a host-side stand-in, not a device address:
// host code uses only the address hipGetSymbolAddress returns for the
// current device, taken once per device and kept in g_scratch_ptr.
constexpr size_t kNoAllocScratchBytes = SEVO_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) char scratch[kNoAllocScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];  // device address of `scratch` per device; null = not taken yet

sevo_status scratch_address(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices)
    return fail(SEVO_ERR_UNSUPPORTED, "device %d beyond the %d the scratch table covers", dev,
                kMaxDevices);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (!p || !aligned16(p)) return fail(SEVO_ERR_HIP, "bad scratch address %p", p);
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return SEVO_OK;
}
}  // namespace

SEVO_API sevo_status sevo_attn_decode_noalloc(const sevo_attn_args* a, void* stream) {
  if (!a) return fail(SEVO_ERR_INVALID_ARGUMENT, "null args");
  sevo_status st = check_attn_shape(a->n, a->n_q_heads, a->n_kv_heads, a->head_dim,
                                    a->page_size, a->max_pages);
  if (st) return st;
  if (a->num_splits < 0) return fail(SEVO_ERR_INVALID_ARGUMENT, "num_splits < 0");
  if (a->num_pages < 1) return fail(SEVO_ERR_INVALID_ARGUMENT, "num_pages < 1");
  if (!(std::isfinite(a->scale)) || a->scale <= 0.f)
    return fail(SEVO_ERR_INVALID_ARGUMENT, "scale must be finite and > 0");
  if (a->n == 0) return SEVO_OK;
  const void* ptrs[] = {a->q, a->kv_pool, a->page_table, a->seq_lens, a->out};
  for (auto p : ptrs)
    if (!p || !aligned16(p))
      return fail(SEVO_ERR_INVALID_ARGUMENT, "null or non-16-byte-aligned pointer");
  int S, chunk;
  resolve_splits(a->n, a->n_kv_heads, a->max_pages, a->num_splits, &S, &chunk);
  const size_t need = attn_ws(a->n, a->n_q_heads, a->head_dim, S);
  if (need > kNoAllocScratchBytes)
    return fail(SEVO_ERR_WORKSPACE_TOO_SMALL,
                "attention needs %zu scratch bytes; the fixed scratch holds %zu (use "
                "sevo_attn_decode with a workspace)",
                need, kNoAllocScratchBytes);
  void* ws = nullptr;
  if ((st = scratch_address(&ws))) return st;
  return attn_core(a->n, a->n_q_heads, a->n_kv_heads, a->head_dim, a->max_pages, a->num_splits,
                   a->num_pages, a->q, a->kv_pool, a->page_table, a->seq_lens, a->scale, a->out,
                   ws, kNoAllocScratchBytes, static_cast<hipStream_t>(stream));
}

// ------------------------------------------------------------------ prefill
SEVO_API sevo_status sevo_attn_prefill(const sevo_prefill_attn_args* a, void* stream) {
  if (!a) return fail(SEVO_ERR_INVALID_ARGUMENT, "null args");
  sevo_status st = check_attn_shape(a->n_seqs, a->n_q_heads, a->n_kv_heads, a->head_dim,
                                    a->page_size, a->max_pages);
  if (st) return st;
  if (a->total_tokens < 0 || a->max_seq_len < 0)
    return fail(SEVO_ERR_INVALID_ARGUMENT, "total_tokens / max_seq_len < 0");
  if (a->n_seqs > 0 && (int64_t)a->max_seq_len * a->n_seqs < a->total_tokens)
    return fail(SEVO_ERR_INVALID_ARGUMENT,
                "max_seq_len %d below the mean sequence length (%d tokens in %d sequences)",
                a->max_seq_len, a->total_tokens, a->n_seqs);
  if (a->num_pages < 1) return fail(SEVO_ERR_INVALID_ARGUMENT, "num_pages < 1");
  if (!(std::isfinite(a->scale)) || a->scale <= 0.f)
    return fail(SEVO_ERR_INVALID_ARGUMENT, "scale must be finite and > 0");
  if (a->n_seqs == 0 || a->total_tokens == 0) return SEVO_OK;
  const void* ptrs[] = {a->q, a->kv_pool, a->page_table, a->seq_starts, a->out};
  for (auto p : ptrs)
    if (!p || !aligned16(p))
      return fail(SEVO_ERR_INVALID_ARGUMENT, "null or non-16-byte-aligned pointer");
  sevo::PrefillAttnArgs k;
  k.n_seqs = a->n_seqs; k.hq = a->n_q_heads; k.hkv = a->n_kv_heads; k.d = a->head_dim;
  k.max_pages = a->max_pages; k.max_seq_len = a->max_seq_len; k.num_pages = a->num_pages;
  k.q = static_cast<const sevo::bf16_t*>(a->q);
  k.kv_pool = static_cast<const sevo::bf16_t*>(a->kv_pool);
  k.page_table = a->page_table; k.seq_starts = a->seq_starts; k.start_pos = a->start_pos;
  k.scale = a->scale; k.out = static_cast<sevo::bf16_t*>(a->out); k.out_tiled = 0;
  k.total_tokens = a->total_tokens;
  hipError_t e = sevo::launch_attn_prefill(k, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? SEVO_OK : hip_fail(e, "sevo_attn_prefill");
}

// ------------------------------------------------------------------ sampling
SEVO_API size_t sevo_sample_workspace_bytes(int32_t n, int32_t vocab) {
  if (n <= 0 || vocab <= 0) return 0;
  return round_up(sevo::sample_workspace_bytes(n, vocab), 256);
}

static sevo_status conf_check(int conf_topk, int vocab, const float* out_conf,
                              const float* conf_sum, int top_k, float top_p, float min_p) {
  if (conf_topk < 0 || conf_topk > 32)
    return fail(SEVO_ERR_INVALID_ARGUMENT, "conf_topk %d outside [0, 32]", conf_topk);
  if (conf_topk > vocab)
    return fail(SEVO_ERR_INVALID_ARGUMENT, "conf_topk %d > vocab %d", conf_topk, vocab);
  if (conf_topk > 0 && !out_conf && !conf_sum)
    return fail(SEVO_ERR_INVALID_ARGUMENT, "conf_topk > 0 needs out_conf or conf_sum");
  if (top_k < 0 || top_k > 32 || top_k > vocab)
    return fail(SEVO_ERR_INVALID_ARGUMENT, "top_k %d outside [0, min(32, vocab)]", top_k);
  if (!(top_p > 0.f && top_p <= 1.f))
    return fail(SEVO_ERR_INVALID_ARGUMENT, "top_p must be in (0, 1]");
  if (!(min_p >= 0.f && min_p <= 1.f))
    return fail(SEVO_ERR_INVALID_ARGUMENT, "min_p must be in [0, 1]");
  if (top_k == 0 && (top_p < 1.f || min_p > 0.f))
    return fail(SEVO_ERR_UNSUPPORTED, "top_p / min_p need top_k > 0");
  const int L = top_k > conf_topk ? top_k : conf_topk;
  if (!sevo::sample_conf_supported(vocab, L))
    return fail(SEVO_ERR_UNSUPPORTED, "top-k / confidence lists over a vocabulary of %d", vocab);
  return SEVO_OK;
}

static sevo_status sample_check(const float* logits, int n, int vocab, int64_t ld, float temp) {
  if (n < 0 || vocab < 1 || ld < vocab)
    return fail(SEVO_ERR_INVALID_ARGUMENT, "bad n / vocab / ld (%d, %d, %lld)", n, vocab,
                (long long)ld);
  if (ld % 4) return fail(SEVO_ERR_INVALID_ARGUMENT, "ld must be a multiple of 4");
  if (!std::isfinite(temp) || temp < 0.f)
    return fail(SEVO_ERR_INVALID_ARGUMENT, "temperature must be finite and >= 0");
  if (n > 0 && (!logits || !aligned16(logits)))
    return fail(SEVO_ERR_INVALID_ARGUMENT, "null or misaligned logits");
  return SEVO_OK;
}

SEVO_API sevo_status sevo_logprob_sample(const sevo_sample_args* a, void* stream) {
  if (!a) return fail(SEVO_ERR_INVALID_ARGUMENT, "null args");
  sevo_status st = sample_check(a->logits, a->n, a->vocab, a->ld, a->temperature);
  if (st) return st;
  if (a->n == 0) return SEVO_OK;
  if (!a->cand_uid || !a->positions || !a->out_tokens || !a->out_logprobs || !a->workspace)
    return fail(SEVO_ERR_INVALID_ARGUMENT, "null pointer");
  if (!aligned16(a->workspace)) return fail(SEVO_ERR_INVALID_ARGUMENT, "misaligned workspace");
  st = conf_check(a->conf_topk, a->vocab, a->out_conf, a->conf_sum, a->top_k, a->top_p,
                  a->min_p);
  if (st) return st;
  const size_t need = sevo::sample_workspace_bytes(a->n, a->vocab);
  if (a->workspace_bytes < need)
    return fail(SEVO_ERR_WORKSPACE_TOO_SMALL, "sampler needs %zu workspace bytes, got %zu", need,
                a->workspace_bytes);
  hipError_t e = sevo::launch_logprob_sample(
      a->logits, a->n, a->vocab, a->ld, a->temperature, a->seed, a->cand_uid, a->positions,
      a->out_tokens, a->out_logprobs, static_cast<float*>(a->workspace), a->conf_topk,
      a->out_conf, a->conf_sum, static_cast<hipStream_t>(stream), a->top_k, a->top_p, a->min_p);
  if (e != hipSuccess) return hip_fail(e, "sevo_logprob_sample launch");
  return SEVO_OK;
}

SEVO_API sevo_status sevo_group_confidence(const float* conf_sum, const int32_t* token_counts,
                                           const int32_t* groups, int32_t n_groups,
                                           int32_t group_size, float* out_gc, void* stream) {
  if (n_groups < 0 || group_size < 1)
    return fail(SEVO_ERR_INVALID_ARGUMENT, "bad n_groups / group_size");
  if (n_groups == 0) return SEVO_OK;
  if (!conf_sum || !token_counts || !groups || !out_gc)
    return fail(SEVO_ERR_INVALID_ARGUMENT, "null pointer");
  hipError_t e = sevo::launch_group_confidence(conf_sum, token_counts, groups, n_groups,
                                               group_size, out_gc,
                                               static_cast<hipStream_t>(stream));
  return e == hipSuccess ? SEVO_OK : hip_fail(e, "sevo_group_confidence");
}

// ------------------------------------------------------------------ sub-steps
SEVO_API sevo_status sevo_embed(const void* embed, const int32_t* tokens, int32_t n,
                                int32_t hidden, int32_t vocab, float* x, void* stream) {
  if (n < 0 || hidden < 8 || hidden % 8 || vocab < 1)
    return fail(SEVO_ERR_INVALID_ARGUMENT, "bad n / hidden / vocab");
  if (n == 0) return SEVO_OK;
  if (!embed || !tokens || !x || !aligned16(embed) || !aligned16(x))
    return fail(SEVO_ERR_INVALID_ARGUMENT, "null or misaligned pointer");
  hipError_t e = sevo::launch_embed(static_cast<const sevo::bf16_t*>(embed), tokens, n, hidden,
                                    vocab, x, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? SEVO_OK : hip_fail(e, "sevo_embed");
}

SEVO_API sevo_status sevo_rmsnorm(const float* x, const void* gain, int32_t rows, int32_t cols,
                                  float eps, void* out, void* stream) {
  if (rows < 0 || cols < 4 || cols % 4) return fail(SEVO_ERR_INVALID_ARGUMENT, "bad rows / cols");
  if (!(eps > 0.f)) return fail(SEVO_ERR_INVALID_ARGUMENT, "eps must be > 0");
  if (rows == 0) return SEVO_OK;
  if (!x || !gain || !out || !aligned16(x) || (reinterpret_cast<uintptr_t>(gain) & 7) ||
      (reinterpret_cast<uintptr_t>(out) & 7))
    return fail(SEVO_ERR_INVALID_ARGUMENT, "null or misaligned pointer");
  hipError_t e = sevo::launch_rmsnorm(x, static_cast<const sevo::bf16_t*>(gain), rows, cols, eps,
                                      static_cast<sevo::bf16_t*>(out),
                                      static_cast<hipStream_t>(stream));
  return e == hipSuccess ? SEVO_OK : hip_fail(e, "sevo_rmsnorm");
}

SEVO_API sevo_status sevo_add_rmsnorm(float* x, const float* partials, int32_t n_partials,
                                      const void* gain, int32_t rows, int32_t cols, float eps,
                                      void* out, void* stream) {
  if (rows < 0 || cols < 4 || cols % 4) return fail(SEVO_ERR_INVALID_ARGUMENT, "bad rows / cols");
  if (n_partials < 0 || n_partials > 16)
    return fail(SEVO_ERR_INVALID_ARGUMENT, "n_partials %d outside 0..16", n_partials);
  if (!(eps > 0.f)) return fail(SEVO_ERR_INVALID_ARGUMENT, "eps must be > 0");
  if (rows == 0) return SEVO_OK;
  if (!x || !gain || !out || !aligned16(x) || (n_partials > 0 && (!partials || !aligned16(partials))) ||
      (reinterpret_cast<uintptr_t>(gain) & 7) || (reinterpret_cast<uintptr_t>(out) & 7))
    return fail(SEVO_ERR_INVALID_ARGUMENT, "null or misaligned pointer");
  hipError_t e = sevo::launch_add_rmsnorm(x, n_partials > 0 ? partials : nullptr, n_partials,
                                          static_cast<const sevo::bf16_t*>(gain), rows, cols, eps,
                                          static_cast<sevo::bf16_t*>(out),
                                          static_cast<hipStream_t>(stream));
  return e == hipSuccess ? SEVO_OK : hip_fail(e, "sevo_add_rmsnorm");
}

static sevo_status linear_check(int m, int n_out, int k, int ldx, int mode, int k_splits,
                                int flags) {
  if (m < 0 || n_out < 64 || k < 32) return fail(SEVO_ERR_INVALID_ARGUMENT, "bad m / n_out / k");
  if (k % 32) return fail(SEVO_ERR_UNSUPPORTED, "k %% 32 != 0");
  if (n_out % 64) return fail(SEVO_ERR_UNSUPPORTED, "n_out %% 64 != 0");
  if (mode < 0 || mode > 2) return fail(SEVO_ERR_INVALID_ARGUMENT, "bad mode %d", mode);
  if (flags & ~(SEVO_LINEAR_X_TILED | SEVO_LINEAR_OUT_TILED))
    return fail(SEVO_ERR_INVALID_ARGUMENT, "unknown flags 0x%x", flags);
  if ((flags & SEVO_LINEAR_OUT_TILED) && mode != SEVO_LINEAR_SWIGLU)
    return fail(SEVO_ERR_INVALID_ARGUMENT, "SEVO_LINEAR_OUT_TILED needs SEVO_LINEAR_SWIGLU");
  if (!(flags & SEVO_LINEAR_X_TILED) && (ldx < k || ldx % 8))
    return fail(SEVO_ERR_INVALID_ARGUMENT, "ldx must be >= k and %% 8");
  if (k_splits < 0) return fail(SEVO_ERR_INVALID_ARGUMENT, "k_splits < 0");
  return SEVO_OK;
}

SEVO_API size_t sevo_linear_workspace_bytes(int32_t m, int32_t n_out, int32_t k,
                                            int32_t k_splits) {
  if (m <= 0 || n_out <= 0 || k <= 0) return 0;
  // the STORE / ADD plan; SwiGLU needs no workspace
  return round_up(sevo::linear_workspace_bytes(m, n_out, k, k_splits, SEVO_LINEAR_STORE), 256);
}

SEVO_API sevo_status sevo_linear_plan(int32_t m, int32_t n_out, int32_t k, int32_t k_splits,
                                      int32_t mode, int32_t* plan) {
  if (!plan) return fail(SEVO_ERR_INVALID_ARGUMENT, "null plan");
  if (m < 1 || m >= sevo::kLargeGemmMinM || n_out < 64 || n_out % 64 || k < 32 || k % 32 ||
      k_splits < 0 || mode < SEVO_LINEAR_STORE || mode > SEVO_LINEAR_SWIGLU)
    return fail(SEVO_ERR_INVALID_ARGUMENT, "bad shape m %d n_out %d k %d k_splits %d mode %d", m,
                n_out, k, k_splits, mode);
  const sevo::LinearPlan p = sevo::plan_linear(m, n_out, k, k_splits, mode);
  plan[0] = p.k_splits;
  plan[1] = p.k_chunk;
  plan[2] = p.rb;
  return SEVO_OK;
}

SEVO_API sevo_status sevo_linear(const sevo_linear_args* a, void* stream) {
  if (!a) return fail(SEVO_ERR_INVALID_ARGUMENT, "null args");
  sevo_status st = linear_check(a->m, a->n_out, a->k, a->ldx, a->mode, a->k_splits, a->flags);
  if (st) return st;
  if (a->m == 0) return SEVO_OK;
  if (!a->x || !a->w || !a->out || !aligned16(a->x) || !aligned16(a->w) || !aligned16(a->out))
    return fail(SEVO_ERR_INVALID_ARGUMENT, "null or misaligned pointer");
  if (a->m >= sevo::kLargeGemmMinM && sevo::gemm_large_supported(a->m, a->n_out, a->k)) {
    hipError_t e = sevo::launch_gemm_large(
        a->m, a->n_out, a->k, a->ldx, (a->flags & SEVO_LINEAR_X_TILED) ? 1 : 0, a->mode,
        static_cast<const sevo::bf16_t*>(a->x), static_cast<const sevo::bf16_t*>(a->w), a->out,
        (a->flags & SEVO_LINEAR_OUT_TILED) ? 1 : 0, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? SEVO_OK : hip_fail(e, "sevo_linear (large m)");
  }
  const sevo::LinearPlan plan = sevo::plan_linear(a->m, a->n_out, a->k, a->k_splits, a->mode);
  const size_t need = sevo::linear_workspace_bytes(a->m, a->n_out, a->k, a->k_splits, a->mode);
  if (need > 0) {
    if (!a->workspace || !aligned16(a->workspace) || a->workspace_bytes < need)
      return fail(SEVO_ERR_WORKSPACE_TOO_SMALL, "linear needs %zu workspace bytes, got %zu", need,
                  a->workspace_bytes);
  }
  hipError_t e = sevo::launch_linear(
      a->m, a->n_out, a->k, a->ldx, (a->flags & SEVO_LINEAR_X_TILED) ? 1 : 0, a->mode, plan,
      static_cast<const sevo::bf16_t*>(a->x), static_cast<const sevo::bf16_t*>(a->w), a->out,
      (a->flags & SEVO_LINEAR_OUT_TILED) ? 1 : 0, static_cast<float*>(a->workspace),
      static_cast<hipStream_t>(stream));
  return e == hipSuccess ? SEVO_OK : hip_fail(e, "sevo_linear");
}

SEVO_API sevo_status sevo_pack_weight(const void* src, void* dst, int32_t n_out, int32_t k,
                                      int32_t kind, void* stream) {
  if (n_out < 64 || k < 32) return fail(SEVO_ERR_INVALID_ARGUMENT, "bad n_out / k");
  if (n_out % 64 || k % 32) return fail(SEVO_ERR_UNSUPPORTED, "n_out %% 64 and k %% 32 must be 0");
  if (kind != SEVO_PACK_PLAIN && kind != SEVO_PACK_GATE_UP)
    return fail(SEVO_ERR_INVALID_ARGUMENT, "bad kind %d", kind);
  if (!src || !dst || !aligned16(src) || !aligned16(dst))
    return fail(SEVO_ERR_INVALID_ARGUMENT, "null or misaligned pointer");
  const size_t bytes = (size_t)n_out * k * 2;
  const uintptr_t s0 = reinterpret_cast<uintptr_t>(src), d0 = reinterpret_cast<uintptr_t>(dst);
  if (s0 < d0 + bytes && d0 < s0 + bytes)
    return fail(SEVO_ERR_INVALID_ARGUMENT, "src and dst overlap");
  hipError_t e = sevo::launch_pack_weight(static_cast<const sevo::bf16_t*>(src),
                                          static_cast<sevo::bf16_t*>(dst), n_out, k,
                                          kind == SEVO_PACK_GATE_UP ? 1 : 0,
                                          static_cast<hipStream_t>(stream));
  return e == hipSuccess ? SEVO_OK : hip_fail(e, "sevo_pack_weight");
}

SEVO_API sevo_status sevo_pack_kv(const void* k_pool, const void* v_pool, int64_t num_pages,
                                  int32_t n_kv_heads, int32_t head_dim, void* kv_pool,
                                  void* stream) {
  if (num_pages < 0 || n_kv_heads < 1)
    return fail(SEVO_ERR_INVALID_ARGUMENT, "bad num_pages / n_kv_heads");
  if (head_dim != 64 && head_dim != 128)
    return fail(SEVO_ERR_UNSUPPORTED, "head_dim must be 64 or 128");
  if (num_pages == 0) return SEVO_OK;
  if (!k_pool || !v_pool || !kv_pool || !aligned16(k_pool) || !aligned16(v_pool) ||
      !aligned16(kv_pool))
    return fail(SEVO_ERR_INVALID_ARGUMENT, "null or misaligned pointer");
  const size_t tiles = (size_t)num_pages * n_kv_heads;
  const size_t src_bytes = tiles * SEVO_PAGE_SIZE * head_dim * 2;
  const uintptr_t d0 = reinterpret_cast<uintptr_t>(kv_pool);
  for (const void* p : {k_pool, v_pool}) {
    const uintptr_t s0 = reinterpret_cast<uintptr_t>(p);
    if (s0 < d0 + 2 * src_bytes && d0 < s0 + src_bytes)
      return fail(SEVO_ERR_INVALID_ARGUMENT, "source and destination pools overlap");
  }
  hipError_t e = sevo::launch_pack_kv(static_cast<const sevo::bf16_t*>(k_pool),
                                      static_cast<const sevo::bf16_t*>(v_pool), tiles, head_dim,
                                      static_cast<sevo::bf16_t*>(kv_pool),
                                      static_cast<hipStream_t>(stream));
  return e == hipSuccess ? SEVO_OK : hip_fail(e, "sevo_pack_kv");
}

static void fill_rope_args(const sevo_model* m, int layer, const float* qkv, int qkv_splits,
                           int n, const int32_t* pos, const int32_t* pt, int max_pages,
                           int64_t num_pages, void* q_out, void* kvp,
                           sevo::RopeAppendArgs& r) {
  const sevo_model_config& c = m->cfg;
  r.qkv = qkv; r.qkv_splits = qkv_splits; r.n = n; r.hq = c.n_q_heads; r.hkv = c.n_kv_heads; r.d = c.head_dim;
  r.positions = pos; r.page_table = pt; r.max_pages = max_pages; r.num_pages = num_pages;
  r.rope_cos = m->rope_cos; r.rope_sin = m->rope_sin; r.max_pos = c.max_position;
  r.q_gain = static_cast<const sevo::bf16_t*>(m->q_norm[layer]);
  r.k_gain = static_cast<const sevo::bf16_t*>(m->k_norm[layer]);
  r.qk_norm = c.qk_norm; r.eps = c.rms_eps;
  r.q_out = static_cast<sevo::bf16_t*>(q_out);
  r.kv_pool = static_cast<sevo::bf16_t*>(kvp);
}

SEVO_API sevo_status sevo_qk_norm_rope_append(const sevo_model* m, int32_t layer,
                                              const float* qkv, int32_t n,
                                              const int32_t* positions,
                                              const int32_t* page_table, int32_t max_pages,
                                              int64_t num_pages, void* q_out, void* kv_pool,
                                              void* stream) {
  if (!m) return fail(SEVO_ERR_INVALID_ARGUMENT, "null model");
  if (layer < 0 || layer >= m->cfg.n_layers) return fail(SEVO_ERR_INVALID_ARGUMENT, "bad layer");
  if (n < 0 || max_pages < 1 || num_pages < 1)
    return fail(SEVO_ERR_INVALID_ARGUMENT, "bad n / max_pages / num_pages");
  if (n == 0) return SEVO_OK;
  if (!qkv || !positions || !page_table || !q_out || !kv_pool)
    return fail(SEVO_ERR_INVALID_ARGUMENT, "null pointer");
  sevo::RopeAppendArgs r;
  fill_rope_args(m, layer, qkv, 1, n, positions, page_table, max_pages, num_pages, q_out, kv_pool,
                 r);
  hipError_t e = sevo::launch_qk_norm_rope_append(r, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? SEVO_OK : hip_fail(e, "sevo_qk_norm_rope_append");
}

// ------------------------------------------------------------------ decode step
namespace {

// MoE: (token, slot) entries t * k + slot are int32
constexpr int64_t kMoeMaxEntries = int64_t(1) << 30;

struct StepLayout {
  size_t x, h, part_qkv, q, o, a, logits, part_x, attn, sample, total;
  size_t m_router, m_sel, m_w, m_off, m_assign, m_act;  // MoE buffers
  int S, chunk;
  sevo::LinearPlan p_qkv, p_o, p_gu, p_d, p_lm, p_router;
};

StepLayout step_layout(const sevo_model_config& c, int n, int max_pages, int num_splits) {
  StepLayout L;
  const int qd = c.n_q_heads * c.head_dim;
  const int qkvd = (c.n_q_heads + 2 * c.n_kv_heads) * c.head_dim;
  resolve_splits(n, c.n_kv_heads, max_pages, num_splits, &L.S, &L.chunk);
  L.p_qkv = sevo::plan_linear(n, qkvd, c.hidden, 0, SEVO_LINEAR_STORE);
  L.p_o = sevo::plan_linear(n, c.hidden, qd, 0, SEVO_LINEAR_STORE);
  const bool moe = c.n_experts > 0;
  const int kact = moe ? c.n_experts_active : 0;
  if (!moe) {
    L.p_gu = sevo::plan_linear(n, 2 * c.ffn, c.hidden, 0, SEVO_LINEAR_SWIGLU);
    L.p_d = sevo::plan_linear(n, c.hidden, c.ffn, 0, SEVO_LINEAR_STORE);
  } else {
    L.p_gu = L.p_d = sevo::LinearPlan{1, c.hidden};
    L.p_router = sevo::plan_linear(n, c.n_experts, c.hidden, 0, SEVO_LINEAR_STORE);
  }
  L.p_lm = sevo::plan_linear(n, c.vocab, c.hidden, 1, SEVO_LINEAR_STORE);
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += round_up(bytes, 256);
    return o;
  };
  int sx = L.p_o.k_splits > L.p_d.k_splits ? L.p_o.k_splits : L.p_d.k_splits;
  if (kact > sx) sx = kact;  // MoE: one partial per selected expert slot
  const size_t n16 = round_up((size_t)n, 16);  // tiled activations: 16-row blocks
  L.x = take((size_t)n * c.hidden * 4);
  L.h = take(n16 * c.hidden * 2);
  L.part_qkv = take((size_t)L.p_qkv.k_splits * n * qkvd * 4);
  L.q = take((size_t)n * qd * 2);
  L.o = take(n16 * qd * 2);
  L.a = take(n16 * (moe ? 0 : c.ffn) * 2);
  L.logits = take((size_t)n * c.vocab * 4);
  L.part_x = take((size_t)sx * n * c.hidden * 4);
  L.attn = take(attn_ws(n, c.n_q_heads, c.head_dim, L.S));
  L.sample = take(sevo::sample_workspace_bytes(n, c.vocab));
  L.m_router = L.m_sel = L.m_w = L.m_off = L.m_assign = L.m_act = 0;
  if (moe) {
    L.m_router = take((size_t)L.p_router.k_splits * n * c.n_experts * 4);
    L.m_sel = take((size_t)n * kact * 4);
    L.m_w = take((size_t)n * kact * 4);
    L.m_off = take((size_t)(c.n_experts + 1) * 4);
    L.m_assign = take((size_t)n * kact * 4);
    L.m_act = take((size_t)n * kact * c.expert_ffn * 2);
  }
  L.total = off;
  return L;
}

// The MoE FFN of layer l on the tiled normed input h: router GEMM, top-k,
// expert lists, expert gate/up + down into part [k][n][hidden].
hipError_t run_moe(const sevo_model* m, int l, int n, const sevo::bf16_t* h, char* ws,
                   const StepLayout& L, int32_t* sel, float* wts, float* part, hipStream_t st) {
  const sevo_model_config& c = m->cfg;
  hipError_t e;
  {
    ProfScope ps(SEVO_PROF_MOE_ROUTE, st);
    float* rl = reinterpret_cast<float*>(ws + L.m_router);
    int32_t* off = reinterpret_cast<int32_t*>(ws + L.m_off);
    int32_t* asg = reinterpret_cast<int32_t*>(ws + L.m_assign);
    e = sevo::launch_linear_partials(n, c.n_experts, c.hidden, c.hidden, 1, L.p_router, h,
                                     static_cast<const sevo::bf16_t*>(m->w_router[l]), rl, 0, st);
    if (e == hipSuccess)
      e = sevo::launch_moe_route(rl, L.p_router.k_splits, n, c.n_experts, c.n_experts_active,
                                 sel, wts, st);
    if (e == hipSuccess)
      e = sevo::launch_moe_plan(sel, n * c.n_experts_active, c.n_experts, off, asg, st);
  }
  if (e != hipSuccess) return e;
  ProfScope ps(SEVO_PROF_MOE_EXPERTS, st);
  sevo::MoeExpertArgs ma;
  ma.n = n; ma.hidden = c.hidden; ma.ffn = c.expert_ffn; ma.n_experts = c.n_experts;
  ma.top_k = c.n_experts_active; ma.x = h;
  ma.w_gate_up = static_cast<const sevo::bf16_t*>(m->w_expert_gate_up[l]);
  ma.w_down = static_cast<const sevo::bf16_t*>(m->w_expert_down[l]);
  ma.offsets = reinterpret_cast<const int32_t*>(ws + L.m_off);
  ma.assign = reinterpret_cast<const int32_t*>(ws + L.m_assign);
  ma.weights = wts;
  ma.act = reinterpret_cast<sevo::bf16_t*>(ws + L.m_act);
  ma.part = part;
  return sevo::launch_moe_experts(ma, st);
}

}  // namespace

SEVO_API size_t sevo_step_workspace_bytes(const sevo_model* m, int32_t n, int32_t max_pages,
                                          int32_t num_splits) {
  if (!m || n <= 0 || max_pages <= 0) return 0;
  return step_layout(m->cfg, n, max_pages, num_splits).total;
}

SEVO_API sevo_status sevo_decode_step(sevo_model* m, const sevo_step_args* a, void* stream) {
  if (!m || !a) return fail(SEVO_ERR_INVALID_ARGUMENT, "null model or args");
  const sevo_model_config& c = m->cfg;
  if (a->n < 0 || a->max_pages < 1 || a->num_pages < 1 || a->num_splits < 0)
    return fail(SEVO_ERR_INVALID_ARGUMENT, "bad n / max_pages / num_pages / num_splits");
  if (!std::isfinite(a->temperature) || a->temperature < 0.f)
    return fail(SEVO_ERR_INVALID_ARGUMENT, "temperature must be finite and >= 0");
  if (sevo_status cs = conf_check(a->conf_topk, c.vocab, a->out_conf, a->conf_sum, a->top_k,
                                  a->top_p, a->min_p))
    return cs;
  if (c.n_experts > 0 && (int64_t)a->n * c.n_experts_active > kMoeMaxEntries)
    return fail(SEVO_ERR_INVALID_ARGUMENT, "n %d: more than 2^30 expert entries", a->n);
  if (a->n == 0) return SEVO_OK;
  if (!a->tokens || !a->positions || !a->page_table || !a->kv_pools ||
      !a->cand_uid || !a->out_tokens || !a->out_logprobs || !a->workspace)
    return fail(SEVO_ERR_INVALID_ARGUMENT, "null pointer");
  if (!aligned16(a->workspace)) return fail(SEVO_ERR_INVALID_ARGUMENT, "misaligned workspace");
  if (a->out_logits && !aligned16(a->out_logits))
    return fail(SEVO_ERR_INVALID_ARGUMENT, "misaligned out_logits");
  if (a->out_hidden && !aligned16(a->out_hidden))
    return fail(SEVO_ERR_INVALID_ARGUMENT, "misaligned out_hidden");
  for (int l = 0; l < c.n_layers; ++l)
    if (!a->kv_pools[l] || !aligned16(a->kv_pools[l]))
      return fail(SEVO_ERR_INVALID_ARGUMENT, "layer %d: null or misaligned KV pool", l);
  const int n = a->n;
  const StepLayout L = step_layout(c, n, a->max_pages, a->num_splits);
  if (a->workspace_bytes < L.total)
    return fail(SEVO_ERR_WORKSPACE_TOO_SMALL, "decode step needs %zu workspace bytes, got %zu",
                L.total, a->workspace_bytes);
  hipStream_t st = static_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(a->workspace);
  float* x = reinterpret_cast<float*>(ws + L.x);
  sevo::bf16_t* h = reinterpret_cast<sevo::bf16_t*>(ws + L.h);
  float* part_qkv = reinterpret_cast<float*>(ws + L.part_qkv);
  sevo::bf16_t* q = reinterpret_cast<sevo::bf16_t*>(ws + L.q);
  sevo::bf16_t* o = reinterpret_cast<sevo::bf16_t*>(ws + L.o);
  sevo::bf16_t* act = reinterpret_cast<sevo::bf16_t*>(ws + L.a);
  float* logits = a->out_logits ? a->out_logits : reinterpret_cast<float*>(ws + L.logits);
  float* part_x = reinterpret_cast<float*>(ws + L.part_x);
  char* attn_ws_ptr = ws + L.attn;
  float* smp = reinterpret_cast<float*>(ws + L.sample);

  const int H = c.hidden, F = c.ffn, qd = c.n_q_heads * c.head_dim;
  const int qkvd = (c.n_q_heads + 2 * c.n_kv_heads) * c.head_dim;
  const float scale = 1.0f / std::sqrt((float)c.head_dim);

  // Split-K partials of a projection are summed (in split order) by the
  // kernel that consumes them: QKV by the QK-norm / RoPE / append kernel, the
  // output and down projections by the next residual add + RMSNorm.
  hipError_t e;
  {
    ProfScope ps(SEVO_PROF_EMBED, st);
    e = sevo::launch_embed(static_cast<const sevo::bf16_t*>(m->embed), a->tokens, n, H, c.vocab,
                           x, st);
  }
  if (e != hipSuccess) return hip_fail(e, "embed");
  // x as it enters layer l (after the add that closes layer l - 1), or after
  // the last layer: entry l of out_hidden
  const size_t x_bytes = (size_t)n * H * sizeof(float);
  auto keep_hidden = [&](int l) {
    return a->out_hidden ? hipMemcpyAsync(a->out_hidden + (size_t)l * n * H, x, x_bytes,
                                          hipMemcpyDeviceToDevice, st)
                         : hipSuccess;
  };
  int pending = 0;  // split partials of the last down projection, not yet in x
  for (int l = 0; l < c.n_layers; ++l) {
    {
      ProfScope ps(SEVO_PROF_NORM, st);
      e = sevo::launch_add_rmsnorm(x, pending ? part_x : nullptr, pending,
                                   static_cast<const sevo::bf16_t*>(m->attn_norm[l]), n, H,
                                   c.rms_eps, h, st);
    }
    if (e == hipSuccess) e = keep_hidden(l);
    if (e == hipSuccess) {
      ProfScope ps(SEVO_PROF_QKV, st);
      e = sevo::launch_linear_partials(n, qkvd, H, H, 1, L.p_qkv, h,
                                       static_cast<const sevo::bf16_t*>(m->w_qkv[l]), part_qkv, 0,
                                       st);
    }
    if (e == hipSuccess) {
      ProfScope ps(SEVO_PROF_ROPE_APPEND, st);
      sevo::RopeAppendArgs r;
      fill_rope_args(m, l, part_qkv, L.p_qkv.k_splits, n, a->positions, a->page_table,
                     a->max_pages, a->num_pages, q, a->kv_pools[l], r);
      e = sevo::launch_qk_norm_rope_append(r, st);
    }
    if (e != hipSuccess) return hip_fail(e, "decode step (attention input)");
    // attention over keys 0..p_i: lengths are positions + 1
    sevo::AttnArgs aa;
    aa.n = n; aa.hq = c.n_q_heads; aa.hkv = c.n_kv_heads; aa.d = c.head_dim;
    aa.max_pages = a->max_pages; aa.num_splits = L.S;
    aa.chunk = L.chunk;
    aa.num_pages = a->num_pages;
    aa.q = q;
    aa.kv_pool = static_cast<const sevo::bf16_t*>(a->kv_pools[l]);
    aa.page_table = a->page_table;
    aa.seq_lens = a->positions;
    aa.len_add = 1;
    aa.scale = scale;
    aa.out = o;
    aa.out_tiled = 1;
    aa.part_ml = reinterpret_cast<float*>(attn_ws_ptr);
    aa.part_acc = reinterpret_cast<float*>(
        attn_ws_ptr + round_up((size_t)n * c.n_q_heads * L.S * 2 * sizeof(float), 256));
    attach_profiler(aa);
    e = sevo::launch_attn_decode(aa, st);
    if (e == hipSuccess) {
      ProfScope ps(SEVO_PROF_ATTN_OUT, st);
      e = sevo::launch_linear_partials(n, H, qd, qd, 1, L.p_o, o,
                                       static_cast<const sevo::bf16_t*>(m->w_o[l]), part_x, 0, st);
    }
    if (e == hipSuccess) {
      ProfScope ps(SEVO_PROF_NORM, st);
      e = sevo::launch_add_rmsnorm(x, part_x, L.p_o.k_splits,
                                   static_cast<const sevo::bf16_t*>(m->ffn_norm[l]), n, H,
                                   c.rms_eps, h, st);
    }
    if (c.n_experts > 0) {
      if (e == hipSuccess)
        e = run_moe(m, l, n, h, ws, L, reinterpret_cast<int32_t*>(ws + L.m_sel),
                    reinterpret_cast<float*>(ws + L.m_w), part_x, st);
      pending = c.n_experts_active;
    } else {
      if (e == hipSuccess) {
        ProfScope ps(SEVO_PROF_GATE_UP, st);
        e = sevo::launch_linear(n, 2 * F, H, H, 1, SEVO_LINEAR_SWIGLU, L.p_gu, h,
                                static_cast<const sevo::bf16_t*>(m->w_gate_up[l]), act, 1,
                                nullptr, st);
      }
      if (e == hipSuccess) {
        ProfScope ps(SEVO_PROF_DOWN, st);
        e = sevo::launch_linear_partials(n, H, F, F, 1, L.p_d, act,
                                         static_cast<const sevo::bf16_t*>(m->w_down[l]), part_x,
                                         0, st);
      }
      pending = L.p_d.k_splits;
    }
    if (e != hipSuccess) return hip_fail(e, "decode step (layer)");
  }
  {
    ProfScope ps(SEVO_PROF_NORM, st);
    e = sevo::launch_add_rmsnorm(x, part_x, pending,
                                 static_cast<const sevo::bf16_t*>(m->final_norm), n, H, c.rms_eps,
                                 h, st);
  }
  if (e == hipSuccess) e = keep_hidden(c.n_layers);
  if (e == hipSuccess) {
    ProfScope ps(SEVO_PROF_LM_HEAD, st);
    e = sevo::launch_linear_partials(n, c.vocab, H, H, 1, L.p_lm, h,
                                     static_cast<const sevo::bf16_t*>(m->lm_head), logits, 0, st);
  }
  if (e == hipSuccess) {
    ProfScope ps(SEVO_PROF_SAMPLE, st);
    e = sevo::launch_logprob_sample(logits, n, c.vocab, c.vocab, a->temperature, a->seed,
                                    a->cand_uid, a->positions, a->out_tokens, a->out_logprobs,
                                    smp, a->conf_topk, a->out_conf, a->conf_sum, st, a->top_k,
                                    a->top_p, a->min_p);
  }
  if (e != hipSuccess) return hip_fail(e, "decode step (head / sampler)");
  return SEVO_OK;
}

// ------------------------------------------------------------------ read probe
SEVO_API sevo_status sevo_hbm_read_probe(const void* buf, size_t bytes,
                                         const int32_t* page_order, int32_t grid, void* sink,
                                         void* stream) {
  if (!buf || !sink || !aligned16(buf) || !aligned16(sink))
    return fail(SEVO_ERR_INVALID_ARGUMENT, "null or misaligned buffer");
  if (grid < 1 || grid > (1 << 20)) return fail(SEVO_ERR_INVALID_ARGUMENT, "grid %d", grid);
  if (bytes < 16 || (page_order && bytes < 8192))
    return fail(SEVO_ERR_INVALID_ARGUMENT, "buffer of %zu bytes too small", bytes);
  hipError_t e = sevo::launch_hbm_read_probe(buf, bytes, page_order, grid, sink,
                                             static_cast<hipStream_t>(stream));
  return e == hipSuccess ? SEVO_OK : hip_fail(e, "sevo_hbm_read_probe");
}

// ------------------------------------------------------------------ MoE sub-step
SEVO_API size_t sevo_moe_workspace_bytes(const sevo_model* m, int32_t n) {
  if (!m || n <= 0 || m->cfg.n_experts <= 0) return 0;
  return step_layout(m->cfg, n, 1, 1).total;
}

SEVO_API sevo_status sevo_moe_ffn(const sevo_model* m, int32_t layer, const void* h, int32_t n,
                                  int32_t* out_experts, float* out_weights, float* out_partials,
                                  void* workspace, size_t workspace_bytes, void* stream) {
  if (!m) return fail(SEVO_ERR_INVALID_ARGUMENT, "null model");
  const sevo_model_config& c = m->cfg;
  if (c.n_experts <= 0) return fail(SEVO_ERR_UNSUPPORTED, "dense model: no experts");
  if (layer < 0 || layer >= c.n_layers) return fail(SEVO_ERR_INVALID_ARGUMENT, "bad layer");
  if (n < 0 || (int64_t)n * c.n_experts_active > kMoeMaxEntries)
    return fail(SEVO_ERR_INVALID_ARGUMENT, "n %d outside [0, 2^30 / k]", n);
  if (n == 0) return SEVO_OK;
  if (!h || !out_experts || !out_weights || !out_partials || !workspace || !aligned16(h) ||
      !aligned16(out_partials) || !aligned16(workspace))
    return fail(SEVO_ERR_INVALID_ARGUMENT, "null or misaligned pointer");
  const StepLayout L = step_layout(c, n, 1, 1);
  if (workspace_bytes < L.total)
    return fail(SEVO_ERR_WORKSPACE_TOO_SMALL, "MoE FFN needs %zu workspace bytes, got %zu",
                L.total, workspace_bytes);
  hipError_t e = run_moe(m, layer, n, static_cast<const sevo::bf16_t*>(h),
                         static_cast<char*>(workspace), L, out_experts, out_weights, out_partials,
                         static_cast<hipStream_t>(stream));
  return e == hipSuccess ? SEVO_OK : hip_fail(e, "sevo_moe_ffn");
}

// ------------------------------------------------------------------ confidence engine
namespace {

constexpr int kPrefillLogitRows = 4096;  // scored rows per LM-head chunk

constexpr int kPrefillMoeRows = 65536;  // tokens per MoE FFN chunk (a multiple of 16)

struct PrefillLayout {
  size_t row, pos, x, h, qkv, q, o, a, part, hf, logits, sample, conf, ids, lps, total;
  // MoE FFN, one token chunk at a time: router logits, routing, entry lists,
  // SwiGLU rows, per-slot outputs
  size_t m_router, m_sel, m_w, m_off, m_assign, m_act, m_slots, m_tiles, m_plan;
  int rc;  // rows per LM-head chunk
  int mc;  // tokens per MoE chunk
};

PrefillLayout prefill_layout(const sevo_model_config& c, int T, int R, int moe_chunk = 0) {
  PrefillLayout L;
  const size_t H = c.hidden, F = c.ffn, V = c.vocab;
  const size_t qd = (size_t)c.n_q_heads * c.head_dim;
  const size_t qkvd = (size_t)(c.n_q_heads + 2 * c.n_kv_heads) * c.head_dim;
  L.rc = R < kPrefillLogitRows ? (R > 0 ? R : 1) : kPrefillLogitRows;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += round_up(bytes, 256);
    return o;
  };
  const size_t t = (size_t)T, t16 = round_up(t, 16), rc = (size_t)L.rc, rc16 = round_up(rc, 16);
  L.row = take(t * 4);
  L.pos = take(t * 4);
  L.x = take(t * H * 4);
  L.h = take(t16 * H * 2);
  L.qkv = take(t * qkvd * 4);
  L.q = take(t * qd * 2);
  L.o = take(t16 * qd * 2);
  L.a = take(t16 * F * 2);
  L.part = take(c.n_experts > 0 ? t * H * 4 : 0);  // the MoE FFN's output (dense: added in place)
  L.mc = 0;
  L.m_router = L.m_sel = L.m_w = L.m_off = L.m_assign = L.m_act = L.m_slots = L.m_tiles = 0;
  L.m_plan = 0;
  if (c.n_experts > 0) {
    size_t mc = moe_chunk > 0 && moe_chunk < kPrefillMoeRows ? round_up(moe_chunk, 16)
                                                              : (size_t)kPrefillMoeRows;
    if (mc > t16) mc = t16;
    const size_t kk = c.n_experts_active, E = c.n_experts;
    // the grouped expert GEMMs address a chunk's gathered rows (mc tokens of
    // the normed input, mc k SwiGLU rows of expert_ffn) through one buffer
    // descriptor with 32-bit byte offsets, and mark an unused row by offset
    // 2^31: a chunk's rows must stay below 2^31 bytes
    const size_t row_bytes = 2 * std::max((size_t)H, kk * (size_t)c.expert_ffn);
    const size_t mc_cap = ((((size_t)1 << 31) - 1) / row_bytes) / 16 * 16;
    if (mc > mc_cap) mc = mc_cap;
    L.mc = (int)mc;
    L.m_router = take(mc * E * 4);
    L.m_sel = take(mc * kk * 4);
    L.m_w = take(mc * kk * 4);
    L.m_off = take((E + 1) * 4);
    L.m_assign = take(mc * kk * 4);
    L.m_act = take(mc * kk * c.expert_ffn * 2);
    L.m_slots = take(kk * mc * H * 4);
    L.m_tiles = take((E + 1) * 4);
    L.m_plan = take(sevo::moe_plan_scratch_bytes((int)(mc * kk), (int)E));
  }
  L.hf = take(rc16 * H * 2);
  L.logits = take(rc * V * 4);
  L.sample = take(sevo::sample_workspace_bytes(L.rc, c.vocab));
  L.conf = take((size_t)(R > 0 ? R : 1) * 4);
  L.ids = take(rc * 4);
  L.lps = take(rc * 4);
  L.total = off;
  return L;
}

// One projection of a prefill: the large-M kernel when it applies, else the
// decode kernel in one K split (no workspace).  X in the tiled layout.
hipError_t prefill_gemm(int m, int n_out, int k, int mode, const sevo::bf16_t* x,
                        const void* w, void* out, int out_tiled, hipStream_t st) {
  const sevo::bf16_t* wb = static_cast<const sevo::bf16_t*>(w);
  if (m >= sevo::kLargeGemmMinM && sevo::gemm_large_supported(m, n_out, k))
    return sevo::launch_gemm_large(m, n_out, k, k, 1, mode, x, wb, out, out_tiled, st);
  const sevo::LinearPlan p = sevo::plan_linear(m, n_out, k, 1, mode);
  return sevo::launch_linear(m, n_out, k, k, 1, mode, p, x, wb, out, out_tiled, nullptr, st);
}

// Entries per expert (n k / E on average) from which a prefill chunk's experts
// run as grouped large-M GEMMs (256-entry tiles, each expert's weights read
// once per tile) instead of the decode kernels (16-64-row tiles).
constexpr int kPrefillGroupedMinPerExpert = 32;

// The MoE FFN of prefill rows c0 .. c0 + nc (c0 a multiple of 16) on the tiled
// normed input h: router GEMM, top-k, entry lists, expert gate/up + down into
// per-slot outputs, then part[c0 + i] = their slot-order sum.
hipError_t run_moe_prefill_chunk(const sevo_model* m, int l, int c0, int nc,
                                 const sevo::bf16_t* h, char* ws, const PrefillLayout& L,
                                 float* part, hipStream_t st) {
  const sevo_model_config& c = m->cfg;
  const int H = c.hidden, E = c.n_experts, k = c.n_experts_active;
  const sevo::bf16_t* hc = h + (size_t)(c0 / 16) * (H / 32) * 512;  // 16-row blocks
  float* rl = reinterpret_cast<float*>(ws + L.m_router);
  int32_t* sel = reinterpret_cast<int32_t*>(ws + L.m_sel);
  float* wts = reinterpret_cast<float*>(ws + L.m_w);
  int32_t* off = reinterpret_cast<int32_t*>(ws + L.m_off);
  int32_t* asg = reinterpret_cast<int32_t*>(ws + L.m_assign);
  float* slots = reinterpret_cast<float*>(ws + L.m_slots);
  int32_t* tiles = reinterpret_cast<int32_t*>(ws + L.m_tiles);
  const bool grouped = (long long)nc * k >= (long long)kPrefillGroupedMinPerExpert * E;
  hipError_t e;
  {
    ProfScope ps(SEVO_PROF_MOE_ROUTE, st);
    e = prefill_gemm(nc, E, H, SEVO_LINEAR_STORE, hc, m->w_router[l], rl, 0, st);
    if (e == hipSuccess) e = sevo::launch_moe_route(rl, 1, nc, E, k, sel, wts, st);
    if (e == hipSuccess)
      e = sevo::launch_moe_plan(sel, nc * k, E, off, asg, st, grouped ? tiles : nullptr,
                                reinterpret_cast<int32_t*>(ws + L.m_plan));
  }
  if (e != hipSuccess) return e;
  ProfScope ps(SEVO_PROF_MOE_EXPERTS, st);
  if (grouped) {
    sevo::GroupArgs g;
    g.offsets = off; g.assign = asg; g.tile_off = tiles; g.weights = wts;
    g.E = E; g.k = k; g.n = nc;
    const int max_tiles = (nc * k + sevo::kMoeGroupRows - 1) / sevo::kMoeGroupRows + E;
    sevo::bf16_t* act = reinterpret_cast<sevo::bf16_t*>(ws + L.m_act);
    e = sevo::launch_gemm_grouped(0, nc, 2 * c.expert_ffn, H, hc,
                                  static_cast<const sevo::bf16_t*>(m->w_expert_gate_up[l]), act,
                                  g, max_tiles, st);
    if (e == hipSuccess)
      e = sevo::launch_gemm_grouped(1, nc * k, H, c.expert_ffn, act,
                                    static_cast<const sevo::bf16_t*>(m->w_expert_down[l]), slots,
                                    g, max_tiles, st);
    if (e == hipSuccess)
      e = sevo::launch_moe_sum_slots(slots, k, nc, H, part + (size_t)c0 * H, st);
    return e;
  }
  sevo::MoeExpertArgs ma;
  ma.n = nc; ma.hidden = H; ma.ffn = c.expert_ffn; ma.n_experts = E; ma.top_k = k; ma.x = hc;
  ma.w_gate_up = static_cast<const sevo::bf16_t*>(m->w_expert_gate_up[l]);
  ma.w_down = static_cast<const sevo::bf16_t*>(m->w_expert_down[l]);
  ma.offsets = off;
  ma.assign = asg;
  ma.weights = wts;
  ma.act = reinterpret_cast<sevo::bf16_t*>(ws + L.m_act);
  ma.part = slots;
  e = sevo::launch_moe_experts(ma, st);
  if (e == hipSuccess) e = sevo::launch_moe_sum_slots(slots, k, nc, H, part + (size_t)c0 * H, st);
  return e;
}

}  // namespace

SEVO_API size_t sevo_prefill_workspace_bytes(const sevo_model* m, int32_t total_tokens,
                                             int32_t n_scored) {
  if (!m || total_tokens <= 0 || n_scored < 0) return 0;
  return prefill_layout(m->cfg, total_tokens, n_scored).total;
}

SEVO_API sevo_status sevo_prefill_confidence(sevo_model* m, const sevo_prefill_args* a,
                                             void* stream) {
  if (!m || !a) return fail(SEVO_ERR_INVALID_ARGUMENT, "null model or args");
  const sevo_model_config& c = m->cfg;
  if (a->n_seqs < 1 || a->total_tokens < 0 || a->max_seq_len < 0 || a->max_pages < 1 ||
      a->num_pages < 1)
    return fail(SEVO_ERR_INVALID_ARGUMENT,
                "bad n_seqs / total_tokens / max_seq_len / max_pages / num_pages");
  if ((int64_t)a->max_seq_len * a->n_seqs < a->total_tokens)
    return fail(SEVO_ERR_INVALID_ARGUMENT,
                "max_seq_len %d below the mean sequence length (%d tokens in %d sequences)",
                a->max_seq_len, a->total_tokens, a->n_seqs);
  if (a->conf_topk < 1 || a->conf_topk > 32 || a->conf_topk > c.vocab)
    return fail(SEVO_ERR_INVALID_ARGUMENT, "conf_topk %d outside [1, min(32, vocab)]",
                a->conf_topk);
  if (!sevo::sample_conf_supported(c.vocab, a->conf_topk))
    return fail(SEVO_ERR_UNSUPPORTED, "confidence lists over a vocabulary of %d", c.vocab);
  if (a->moe_chunk < 0) return fail(SEVO_ERR_INVALID_ARGUMENT, "moe_chunk %d < 0", a->moe_chunk);
  if (a->n_scored < 0 || a->n_scored > a->total_tokens)
    return fail(SEVO_ERR_INVALID_ARGUMENT, "n_scored %d outside [0, total_tokens]", a->n_scored);
  if (!a->seq_starts || !a->out_conf || !a->kv_pools || !a->workspace ||
      !aligned16(a->workspace) || !aligned16(a->seq_starts))
    return fail(SEVO_ERR_INVALID_ARGUMENT, "null or misaligned pointer");
  const int T = a->total_tokens, R = a->n_scored;
  hipStream_t st = static_cast<hipStream_t>(stream);
  hipError_t e;
  if (T == 0) {  // every sequence is empty: no scored rows, C = 0
    e = sevo::launch_seq_confidence(nullptr, nullptr, 0, a->seq_starts, a->n_seqs, a->out_conf,
                                    st);
    return e == hipSuccess ? SEVO_OK : hip_fail(e, "prefill confidence");
  }
  if (!a->tokens || !a->page_table || (R > 0 && !a->scored_rows))
    return fail(SEVO_ERR_INVALID_ARGUMENT, "null pointer");
  for (int l = 0; l < c.n_layers; ++l)
    if (!a->kv_pools[l] || !aligned16(a->kv_pools[l]))
      return fail(SEVO_ERR_INVALID_ARGUMENT, "layer %d: null or misaligned KV pool", l);
  const PrefillLayout L = prefill_layout(c, T, R, a->moe_chunk);
  if (a->workspace_bytes < L.total)
    return fail(SEVO_ERR_WORKSPACE_TOO_SMALL, "prefill needs %zu workspace bytes, got %zu",
                L.total, a->workspace_bytes);
  char* ws = static_cast<char*>(a->workspace);
  int32_t* row = reinterpret_cast<int32_t*>(ws + L.row);
  int32_t* pos = reinterpret_cast<int32_t*>(ws + L.pos);
  float* x = reinterpret_cast<float*>(ws + L.x);
  sevo::bf16_t* h = reinterpret_cast<sevo::bf16_t*>(ws + L.h);
  float* qkv = reinterpret_cast<float*>(ws + L.qkv);
  sevo::bf16_t* q = reinterpret_cast<sevo::bf16_t*>(ws + L.q);
  sevo::bf16_t* o = reinterpret_cast<sevo::bf16_t*>(ws + L.o);
  sevo::bf16_t* act = reinterpret_cast<sevo::bf16_t*>(ws + L.a);
  float* part = reinterpret_cast<float*>(ws + L.part);
  sevo::bf16_t* hf = reinterpret_cast<sevo::bf16_t*>(ws + L.hf);
  float* logits = reinterpret_cast<float*>(ws + L.logits);
  float* smp = reinterpret_cast<float*>(ws + L.sample);
  float* row_conf = a->out_row_conf ? a->out_row_conf : reinterpret_cast<float*>(ws + L.conf);
  int32_t* ids = reinterpret_cast<int32_t*>(ws + L.ids);
  float* lps = reinterpret_cast<float*>(ws + L.lps);

  const int H = c.hidden, F = c.ffn, qd = c.n_q_heads * c.head_dim;
  const int qkvd = (c.n_q_heads + 2 * c.n_kv_heads) * c.head_dim;
  const float scale = 1.0f / std::sqrt((float)c.head_dim);

  {
    ProfScope ps(SEVO_PROF_EMBED, st);
    e = sevo::launch_embed(static_cast<const sevo::bf16_t*>(m->embed), a->tokens, T, H, c.vocab,
                           x, st);
  }
  if (e == hipSuccess)
    e = sevo::launch_prefill_index(a->seq_starts, a->start_pos, a->n_seqs, T, row, pos, st);
  if (e != hipSuccess) return hip_fail(e, "prefill (embed)");
  // the output and dense down projections add their product to x in the GEMM
  // epilogue (the same single fp32 add as a separate residual update, without
  // a round trip of the product through memory); a MoE FFN's slot-order sum
  // goes to `part`, which the next residual add + RMSNorm adds to x
  const bool moe = c.n_experts > 0;
  for (int l = 0; l < c.n_layers; ++l) {
    {
      ProfScope ps(SEVO_PROF_NORM, st);
      const bool add_part = l > 0 && moe;
      e = sevo::launch_add_rmsnorm(x, add_part ? part : nullptr, add_part ? 1 : 0,
                                   static_cast<const sevo::bf16_t*>(m->attn_norm[l]), T, H,
                                   c.rms_eps, h, st);
    }
    if (e == hipSuccess) {
      ProfScope ps(SEVO_PROF_QKV, st);
      e = prefill_gemm(T, qkvd, H, SEVO_LINEAR_STORE, h, m->w_qkv[l], qkv, 0, st);
    }
    if (e == hipSuccess) {
      ProfScope ps(SEVO_PROF_ROPE_APPEND, st);
      sevo::RopeAppendArgs r;
      fill_rope_args(m, l, qkv, 1, T, pos, a->page_table, a->max_pages, a->num_pages, q,
                     a->kv_pools[l], r);
      r.row_of_token = row;
      e = sevo::launch_qk_norm_rope_append(r, st);
    }
    if (e == hipSuccess) {
      ProfScope ps(SEVO_PROF_ATTN_PREFILL, st);
      sevo::PrefillAttnArgs pa;
      pa.n_seqs = a->n_seqs; pa.hq = c.n_q_heads; pa.hkv = c.n_kv_heads; pa.d = c.head_dim;
      pa.max_pages = a->max_pages; pa.max_seq_len = a->max_seq_len; pa.num_pages = a->num_pages;
      pa.q = q; pa.kv_pool = static_cast<const sevo::bf16_t*>(a->kv_pools[l]);
      pa.page_table = a->page_table; pa.seq_starts = a->seq_starts; pa.start_pos = a->start_pos;
      pa.scale = scale; pa.out = o; pa.out_tiled = 1; pa.total_tokens = T;
      e = sevo::launch_attn_prefill(pa, st);
    }
    if (e == hipSuccess) {
      ProfScope ps(SEVO_PROF_ATTN_OUT, st);
      e = prefill_gemm(T, H, qd, SEVO_LINEAR_ADD, o, m->w_o[l], x, 0, st);
    }
    if (e == hipSuccess) {
      ProfScope ps(SEVO_PROF_NORM, st);
      e = sevo::launch_add_rmsnorm(x, nullptr, 0, static_cast<const sevo::bf16_t*>(m->ffn_norm[l]),
                                   T, H, c.rms_eps, h, st);
    }
    if (moe) {
      // the mixture of experts, a chunk of tokens at a time: per-slot outputs
      // of the chunk, then their slot-order sum into its rows of `part`
      for (int c0 = 0; c0 < T && e == hipSuccess; c0 += L.mc) {
        const int nc = T - c0 < L.mc ? T - c0 : L.mc;
        e = run_moe_prefill_chunk(m, l, c0, nc, h, ws, L, part, st);
      }
    } else {
      if (e == hipSuccess) {
        ProfScope ps(SEVO_PROF_GATE_UP, st);
        e = prefill_gemm(T, 2 * F, H, SEVO_LINEAR_SWIGLU, h, m->w_gate_up[l], act, 1, st);
      }
      if (e == hipSuccess) {
        ProfScope ps(SEVO_PROF_DOWN, st);
        e = prefill_gemm(T, H, F, SEVO_LINEAR_ADD, act, m->w_down[l], x, 0, st);
      }
    }
    if (e != hipSuccess) return hip_fail(e, "prefill (layer)");
  }
  // scored rows, a chunk at a time: final norm of x (+ the last MoE FFN
  // output), LM head, per-row confidence (greedy pass of the sampler: no noise)
  for (int r0 = 0; r0 < R; r0 += L.rc) {
    const int nr = R - r0 < L.rc ? R - r0 : L.rc;
    {
      ProfScope ps(SEVO_PROF_NORM, st);
      e = sevo::launch_add_rmsnorm(x, moe ? part : nullptr, moe ? 1 : 0,
                                   static_cast<const sevo::bf16_t*>(m->final_norm), nr, H,
                                   c.rms_eps, hf, st, a->scored_rows + r0, T);
    }
    if (e == hipSuccess) {
      ProfScope ps(SEVO_PROF_LM_HEAD, st);
      e = prefill_gemm(nr, c.vocab, H, SEVO_LINEAR_STORE, hf, m->lm_head, logits, 0, st);
    }
    if (e == hipSuccess) {
      ProfScope ps(SEVO_PROF_SAMPLE, st);
      e = sevo::launch_logprob_sample(logits, nr, c.vocab, c.vocab, 0.f, 0, nullptr, nullptr, ids,
                                      lps, smp, a->conf_topk, row_conf + r0, nullptr, st);
    }
    if (e != hipSuccess) return hip_fail(e, "prefill (scored rows)");
  }
  e = sevo::launch_seq_confidence(row_conf, a->scored_rows, R, a->seq_starts, a->n_seqs,
                                  a->out_conf, st);
  return e == hipSuccess ? SEVO_OK : hip_fail(e, "prefill (sequence confidence)");
}

// ------------------------------------------------------------------ utilities
SEVO_API sevo_status sevo_fill_normal_bf16(void* dst, int64_t count, uint64_t key, int64_t offset,
                                           float mul, float add, int32_t use_add, void* stream) {
  if (count < 0 || offset < 0) return fail(SEVO_ERR_INVALID_ARGUMENT, "negative count / offset");
  if (count == 0) return SEVO_OK;
  if (!dst || !aligned16(dst)) return fail(SEVO_ERR_INVALID_ARGUMENT, "null or misaligned dst");
  hipError_t e = sevo::launch_fill_bf16(static_cast<sevo::bf16_t*>(dst), count, key, offset, mul,
                                        add, use_add ? 1 : 0, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? SEVO_OK : hip_fail(e, "sevo_fill_normal_bf16");
}

SEVO_API sevo_status sevo_validate_paging(const int32_t* page_table, const int32_t* lengths,
                                          int32_t n, int32_t max_pages, int64_t num_pages,
                                          void* stream) {
  if (n < 0 || max_pages < 1 || num_pages < 1)
    return fail(SEVO_ERR_INVALID_ARGUMENT, "bad n / max_pages / num_pages");
  if (n == 0) return SEVO_OK;
  if (!page_table || !lengths) return fail(SEVO_ERR_INVALID_ARGUMENT, "null pointer");
  try {
    std::vector<int32_t> pt((size_t)n * max_pages), len(n);
    hipStream_t st = static_cast<hipStream_t>(stream);
    hipError_t e = hipMemcpyAsync(pt.data(), page_table, pt.size() * 4, hipMemcpyDeviceToHost, st);
    if (e == hipSuccess)
      e = hipMemcpyAsync(len.data(), lengths, len.size() * 4, hipMemcpyDeviceToHost, st);
    if (e == hipSuccess) e = hipStreamSynchronize(st);
    if (e != hipSuccess) return hip_fail(e, "sevo_validate_paging copy");
    std::vector<uint8_t> used((size_t)num_pages, 0);
    for (int i = 0; i < n; ++i) {
      if (len[i] < 0 || len[i] > max_pages * SEVO_PAGE_SIZE)
        return fail(SEVO_ERR_BAD_PAGE_TABLE, "candidate %d: length %d outside [0, %d]", i,
                    len[i], max_pages * SEVO_PAGE_SIZE);
      const int np = (len[i] + SEVO_PAGE_SIZE - 1) / SEVO_PAGE_SIZE;
      for (int p = 0; p < np; ++p) {
        const int32_t id = pt[(size_t)i * max_pages + p];
        if (id < 0 || id >= num_pages)
          return fail(SEVO_ERR_BAD_PAGE_TABLE, "candidate %d page %d: id %d outside [0, %lld)", i,
                      p, id, (long long)num_pages);
        if (used[id]) return fail(SEVO_ERR_BAD_PAGE_TABLE, "physical page %d used twice", id);
        used[id] = 1;
      }
    }
    return SEVO_OK;
  } catch (...) {
    return fail(SEVO_ERR_OUT_OF_MEMORY, "host allocation failed in sevo_validate_paging");
  }
}

// ------------------------------------------------------------------ timing
SEVO_API sevo_status sevo_profile_begin(int32_t max_launches, uint32_t kinds) {
  if (max_launches < 1 || max_launches > (1 << 20))
    return fail(SEVO_ERR_INVALID_ARGUMENT, "max_launches must be in [1, 2^20]");
  if (kinds == 0 || (kinds >> SEVO_PROF_NUM_KINDS) != 0)
    return fail(SEVO_ERR_INVALID_ARGUMENT, "bad kinds mask 0x%x", kinds);
  std::lock_guard<std::mutex> lk(g_prof.mu);
  if (g_prof.on) return fail(SEVO_ERR_INVALID_ARGUMENT, "a recording is already open");
  try {
    while (g_prof.pool.size() < (size_t)3 * max_launches) {
      hipEvent_t e;
      // timing-only events: without the system-scope fence, recording one
      // does not write back and invalidate the caches between the kernels it
      // separates (with the fence each recorded event left the GPU idle for
      // about 5.6 us between the two launches)
      hipError_t r = hipEventCreateWithFlags(&e, hipEventDisableSystemFence);
      if (r != hipSuccess) return hip_fail(r, "sevo_profile_begin");
      g_prof.pool.push_back(e);
    }
    g_prof.recs.clear();
    g_prof.recs.reserve((size_t)max_launches * 2);
  } catch (...) {
    return fail(SEVO_ERR_OUT_OF_MEMORY, "sevo_profile_begin");
  }
  g_prof.used = 0;
  g_prof.mask = kinds;
  g_prof.on = true;
  return SEVO_OK;
}

SEVO_API sevo_status sevo_profile_end(float* total_ms, int32_t* launches) {
  std::lock_guard<std::mutex> lk(g_prof.mu);
  g_prof.on = false;
  float ms[SEVO_PROF_NUM_KINDS] = {};
  int32_t cnt[SEVO_PROF_NUM_KINDS] = {};
  for (const ProfRecord& r : g_prof.recs) {
    hipError_t e = hipEventSynchronize(r.e);
    float t = 0.f;
    if (e == hipSuccess) e = hipEventElapsedTime(&t, r.b, r.e);
    if (e != hipSuccess) return hip_fail(e, "sevo_profile_end");
    ms[r.kind] += t;
    ++cnt[r.kind];
  }
  g_prof.recs.clear();
  for (int k = 0; k < SEVO_PROF_NUM_KINDS; ++k) {
    if (total_ms) total_ms[k] = ms[k];
    if (launches) launches[k] = cnt[k];
  }
  return SEVO_OK;
}
