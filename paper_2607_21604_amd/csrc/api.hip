// C ABI of libakvs: argument validation, workspace planning, the step entries and the two
// whole-procedure drivers (reuse prefill, full prefill). Every entry validates all host-
// checkable arguments before it enqueues anything.
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <algorithm>
#include <mutex>
#include <vector>

#include "kernels.h"

using namespace akvs;

namespace {

// ---- errors -------------------------------------------------------------------------------
thread_local char g_err[768] = "";

akvs_status fail(akvs_status s, const char *fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
  return s;
}

#define REQUIRE(cond, status, ...)                 \
  do {                                             \
    if (!(cond)) return fail(status, __VA_ARGS__); \
  } while (0)

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
size_t es_of(int dtype) { return dtype == AKVS_F32 ? 4 : 2; }
size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// ---- kernel timing ------------------------------------------------------------------------
struct ProfRec {
  int cls;
  hipEvent_t a, b;
};
struct Prof {
  std::mutex mu;
  uint32_t mask = 0;
  std::vector<hipEvent_t> pool;
  std::vector<ProfRec> pending;
  int64_t launches[AKVS_K_NCLASSES] = {};
  double ms[AKVS_K_NCLASSES] = {};
};
Prof g_prof;

hipEvent_t prof_event() {
  if (!g_prof.pool.empty()) {
    hipEvent_t e = g_prof.pool.back();
    g_prof.pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

hipEvent_t prof_begin(hipStream_t s, int cls) {
  if (!(g_prof.mask & (1u << cls))) return nullptr;
  std::lock_guard<std::mutex> lk(g_prof.mu);
  hipEvent_t e = prof_event();
  if (e && hipEventRecord(e, s) != hipSuccess) {
    g_prof.pool.push_back(e);
    return nullptr;
  }
  return e;
}

void prof_end(hipStream_t s, int cls, hipEvent_t a) {
  if (!a) return;
  std::lock_guard<std::mutex> lk(g_prof.mu);
  hipEvent_t b = prof_event();
  if (!b || hipEventRecord(b, s) != hipSuccess) {
    g_prof.pool.push_back(a);
    if (b) g_prof.pool.push_back(b);
    return;
  }
  g_prof.pending.push_back({cls, a, b});
}

void prof_drain() {
  for (const ProfRec &r : g_prof.pending) {
    float ms = 0.f;
    if (hipEventSynchronize(r.b) == hipSuccess && hipEventElapsedTime(&ms, r.a, r.b) == hipSuccess) {
      g_prof.launches[r.cls] += 1;
      g_prof.ms[r.cls] += ms;
    }
    g_prof.pool.push_back(r.a);
    g_prof.pool.push_back(r.b);
  }
  g_prof.pending.clear();
}

#define LAUNCH(cls, expr)                                                                  \
  do {                                                                                     \
    hipEvent_t ev_ = prof_begin(stream, cls);                                                   \
    hipError_t er_ = (expr);                                                               \
    if (er_ != hipSuccess) return fail(AKVS_EHIP, "%s: %s", #expr, hipGetErrorString(er_)); \
    prof_end(stream, cls, ev_);                                                            \
  } while (0)

// A projection GEMM and, when it splits K, its fixup pass (timed in the OTHER class so the
// GEMM class times the main kernel alone).
#define GEMM(...)                                                  \
  do {                                                             \
    LAUNCH(AKVS_K_GEMM, launch_gemm(__VA_ARGS__));                 \
    LAUNCH(AKVS_K_OTHER, launch_gemm_fixup(__VA_ARGS__));          \
  } while (0)

// ---- validation -----------------------------------------------------------------------------
akvs_status check_model(const akvs_model_cfg *m) {
  REQUIRE(m, AKVS_EINVAL, "model cfg is NULL");
  REQUIRE(m->dtype == AKVS_F32 || m->dtype == AKVS_BF16, AKVS_EDTYPE,
          "model dtype must be AKVS_F32 or AKVS_BF16 (got %d)", m->dtype);
  REQUIRE(m->n_layers >= 1 && m->d_model >= 8 && m->n_q_heads >= 1 && m->n_kv_heads >= 1 &&
              m->ffn_dim >= 4 && m->vocab >= 1,
          AKVS_EINVAL, "model sizes must be positive");
  REQUIRE(m->head_dim == 64 || m->head_dim == 128, AKVS_EUNSUPPORTED,
          "head_dim %d not supported (64 or 128)", m->head_dim);
  REQUIRE(m->n_q_heads % m->n_kv_heads == 0, AKVS_ESHAPE,
          "n_q_heads %d is not a multiple of n_kv_heads %d", m->n_q_heads, m->n_kv_heads);
  REQUIRE(m->d_model % 8 == 0, AKVS_ESHAPE, "d_model must be a multiple of 8");
  REQUIRE(m->n_kv_heads * m->head_dim <= 2048, AKVS_EUNSUPPORTED,
          "n_kv_heads * head_dim %d above 2048", m->n_kv_heads * m->head_dim);
  if (m->dtype == AKVS_BF16) {
    REQUIRE(m->d_model % 64 == 0 && m->ffn_dim % 64 == 0, AKVS_EUNSUPPORTED,
            "bf16 models need d_model and ffn_dim multiples of 64");
  } else {
    REQUIRE(m->ffn_dim % 4 == 0, AKVS_ESHAPE, "ffn_dim must be a multiple of 4");
  }
  REQUIRE(m->rope_theta > 0.f && m->rms_eps >= 0.f, AKVS_EINVAL, "rope_theta > 0, rms_eps >= 0");
  const long long widest = (long long)(m->n_q_heads + 2 * m->n_kv_heads) * m->head_dim;
  REQUIRE(widest < (1LL << 30) && (long long)m->d_model * m->ffn_dim < (1LL << 40), AKVS_ESHAPE,
          "model too large");
  return AKVS_OK;
}

akvs_status check_layers(const akvs_model_cfg *m, const akvs_layer_w *lw) {
  REQUIRE(lw, AKVS_EINVAL, "layer weights are NULL");
  for (int l = 0; l < m->n_layers; ++l) {
    const void *p[6] = {lw[l].attn_norm, lw[l].w_qkv, lw[l].w_o, lw[l].mlp_norm, lw[l].w_gate_up,
                        lw[l].w_down};
    for (int i = 0; i < 6; ++i) {
      REQUIRE(p[i], AKVS_EINVAL, "layer %d weight %d is NULL", l, i);
      REQUIRE(aligned16(p[i]), AKVS_EINVAL, "layer %d weight %d not 16-byte aligned", l, i);
    }
  }
  return AKVS_OK;
}

struct Meta {
  std::vector<int32_t> m;  // [2][n][4]: key table, value table
  long long t_ctx = 0, sum_b = 0, sum_b_v = 0, row_cap = 0, row_min = 0, t_all = 0;
};

akvs_status check_reuse(const akvs_reuse_cfg *c, int n_layers, Meta *meta) {
  REQUIRE(c, AKVS_EINVAL, "reuse cfg is NULL");
  REQUIRE(c->n_chunks >= 1 && c->chunk_len, AKVS_EINVAL, "need n_chunks >= 1 and chunk_len");
  REQUIRE(c->query_len >= 1, AKVS_EINVAL, "query_len must be >= 1");
  REQUIRE(c->refresh_den >= 1 && c->refresh_num >= 0 && c->refresh_num <= c->refresh_den,
          AKVS_EINVAL, "refresh ratio must satisfy 0 <= num <= den, den >= 1");
  const bool own_v = c->refresh_v_den != 0;
  REQUIRE(!own_v || (c->refresh_v_den >= 1 && c->refresh_v_num >= 0 &&
                     c->refresh_v_num <= c->refresh_v_den),
          AKVS_EINVAL, "value refresh ratio must satisfy 0 <= num <= den, den >= 1 (or den 0)");
  const long long vn = own_v ? c->refresh_v_num : c->refresh_num;
  const long long vd = own_v ? c->refresh_v_den : c->refresh_den;
  const uint32_t known = AKVS_F_NO_CORRECTION | AKVS_F_UNIT_WEIGHTS | AKVS_F_FRESH_IF_RECOMPUTED |
                         AKVS_F_NO_PREFIX_RECOMPUTE | AKVS_F_GIVEN_PROBES |
                         AKVS_F_PRE_ROPE_OFFSETS;
  REQUIRE((c->flags & ~known) == 0, AKVS_EINVAL, "unknown flag bits 0x%x", c->flags & ~known);
  REQUIRE(!(c->flags & AKVS_F_NO_PREFIX_RECOMPUTE) || (c->refresh_num == 0 && vn == 0),
          AKVS_EINVAL, "AKVS_F_NO_PREFIX_RECOMPUTE needs zero refresh ratios");
  if (n_layers > 0)
    REQUIRE(c->check_layer >= 0 && c->check_layer < n_layers, AKVS_EINVAL,
            "check_layer %d outside [0, %d)", c->check_layer, n_layers);
  Meta loc;
  Meta &mt = meta ? *meta : loc;
  const int nc = c->n_chunks;
  mt.m.assign((size_t)nc * 8, 0);
  long long s = 0, off = 0, off_v = 0, cap = 0, lo = 0;
  for (int i = 0; i < nc; ++i) {
    const long long n = c->chunk_len[i];
    REQUIRE(n >= 1, AKVS_EINVAL, "chunk %d has length %lld", i, n);
    const long long b = (c->refresh_num * n + c->refresh_den - 1) / c->refresh_den;
    const long long bv = (vn * n + vd - 1) / vd;
    int32_t *mk = &mt.m[4 * (size_t)i], *mv = &mt.m[4 * ((size_t)nc + i)];
    mk[0] = mv[0] = (int32_t)s;
    mk[1] = mv[1] = (int32_t)n;
    mk[2] = (int32_t)b;
    mk[3] = (int32_t)off;
    mv[2] = (int32_t)bv;
    mv[3] = (int32_t)off_v;
    s += n;
    off += b;
    off_v += bv;
    cap += n < b + bv ? n : b + bv;
    const long long bmax = b > bv ? b : bv;
    lo += n < bmax ? n : bmax;  // the larger probe set alone is min(n, b) distinct rows
    REQUIRE(s + c->query_len < (1LL << 28), AKVS_ESHAPE, "context too long");
  }
  mt.t_ctx = s;
  mt.sum_b = off;
  mt.sum_b_v = off_v;
  mt.row_cap = cap + c->query_len;
  mt.row_min = lo + c->query_len;
  mt.t_all = s + c->query_len;
  return AKVS_OK;
}

akvs_status check_cache(const akvs_cache *c, const akvs_model_cfg *m) {
  REQUIRE(c && c->k && c->v, AKVS_EINVAL, "cache k/v are NULL");
  REQUIRE(aligned16(c->k) && aligned16(c->v), AKVS_EINVAL, "cache not 16-byte aligned");
  if (m->dtype == AKVS_F32) {
    REQUIRE(c->dtype == AKVS_F32, AKVS_EDTYPE, "an fp32 model needs an AKVS_F32 cache");
  } else {
    REQUIRE(c->dtype == AKVS_BF16 || c->dtype == AKVS_U4G64 || c->dtype == AKVS_U2G64 ||
                c->dtype == AKVS_E4M3G64,
            AKVS_EDTYPE, "a bf16 model needs an AKVS_BF16 / U4G64 / U2G64 / E4M3G64 cache");
  }
  if (c->dtype == AKVS_U4G64 || c->dtype == AKVS_U2G64 || c->dtype == AKVS_E4M3G64) {
    REQUIRE(c->k_meta && c->v_meta, AKVS_EINVAL, "quantised cache needs k_meta and v_meta");
    REQUIRE(aligned16(c->k_meta) && aligned16(c->v_meta), AKVS_EINVAL, "meta not aligned");
  }
  return AKVS_OK;
}

// Cache layer view (plain or quantised) of layer l over t_ctx tokens.
CacheLayer cache_layer(const akvs_cache *c, int l, long long t_ctx, int hkv, int hd) {
  CacheLayer v;
  const long long rows = t_ctx * hkv;
  size_t row_bytes;
  if (c->dtype == AKVS_F32) row_bytes = (size_t)hd * 4;
  else if (c->dtype == AKVS_BF16) row_bytes = (size_t)hd * 2;
  else if (c->dtype == AKVS_U4G64) row_bytes = (size_t)hd / 2;
  else if (c->dtype == AKVS_E4M3G64) row_bytes = (size_t)hd;
  else row_bytes = (size_t)hd / 4;
  const size_t lb = (size_t)rows * row_bytes;
  v.k = reinterpret_cast<const char *>(c->k) + (size_t)l * lb;
  v.v = reinterpret_cast<const char *>(c->v) + (size_t)l * lb;
  const size_t mb = (size_t)rows * (hd / 64) * 2;  // halfs per layer
  v.k_meta = c->k_meta ? reinterpret_cast<const _Float16 *>(c->k_meta) + (size_t)l * mb : nullptr;
  v.v_meta = c->v_meta ? reinterpret_cast<const _Float16 *>(c->v_meta) + (size_t)l * mb : nullptr;
  v.dtype = c->dtype;
  return v;
}

// ---- workspace carving ------------------------------------------------------------------------
struct Carver {
  char *base;
  size_t off = 0;
  explicit Carver(void *b) : base(reinterpret_cast<char *>(b)) {}
  template <typename T>
  T *take(size_t count) {
    T *p = base ? reinterpret_cast<T *>(base + off) : nullptr;
    off += align256(count * sizeof(T));
    return p;
  }
};

// Buffers of a decoder pass over `rows` rows (the full layer and the probe layers).
struct LayerBufs {
  void *x, *q, *att, *act;  // model dtype
  float *part_o, *part_ml;  // attention key-split partials (bf16 models)
  long long part_rows;      // splits x rows that part_o / part_ml hold
  float *gpart;             // GEMM K-split partials (bf16 models)
  int32_t *plan;            // attention split plan of full_layer's rows
};

// GEMM partial-tile workspace (floats) of the four projections of one layer over `rows`.
size_t layer_gemm_part(const akvs_model_cfg *m, long long rows) {
  if (m->dtype != AKVS_BF16) return 0;
  const int D = m->d_model, F = m->ffn_dim, hqw = m->n_q_heads * m->head_dim;
  const int qkvw = hqw + 2 * m->n_kv_heads * m->head_dim;
  const int r = (int)rows;
  size_t w = gemm_part_floats(r, qkvw, D, EPI_QKV);
  w = std::max(w, gemm_part_floats(r, D, hqw, EPI_RESID));
  w = std::max(w, gemm_part_floats(r, F, D, EPI_SWIGLU));
  w = std::max(w, gemm_part_floats(r, D, F, EPI_RESID));
  return w;
}

// One attention call of a layer pass: its row count and key count.
struct AttnUse {
  long long rows, n_keys;
};

// rows: the largest row count a layer pass uses; uses: the (rows, keys) of its attention
// calls, which are also the row counts of its projections (sizing the GEMM K-split
// partials and the attention key-split partials of bf16 models).
void carve_layer_bufs(Carver &cv, const akvs_model_cfg *m, long long rows,
                      const std::vector<AttnUse> &uses, LayerBufs &b) {
  const size_t es = es_of(m->dtype);
  b.x = cv.take<char>((size_t)rows * m->d_model * es);
  b.q = cv.take<char>((size_t)rows * m->n_q_heads * m->head_dim * es);
  b.att = cv.take<char>((size_t)rows * m->n_q_heads * m->head_dim * es);
  b.act = cv.take<char>((size_t)rows * m->ffn_dim * es);
  b.part_o = nullptr;
  b.part_ml = nullptr;
  b.part_rows = 0;
  b.gpart = nullptr;
  b.plan = cv.take<int32_t>(kAttnPlanInts);
  size_t g = 0;
  long long worst = 0;
  for (const AttnUse &u : uses) {
    g = std::max(g, layer_gemm_part(m, u.rows));
    if (m->dtype != AKVS_BF16 || u.rows <= 0) continue;
    const long long sp = attn_part_splits((int)u.rows, m->n_q_heads, m->n_kv_heads, m->head_dim,
                                          (int)u.n_keys);
    if (sp > 1 && sp * u.rows > worst) worst = sp * u.rows;
  }
  if (g) b.gpart = cv.take<float>(g);
  if (worst > 0) {
    b.part_o = cv.take<float>((size_t)worst * m->n_q_heads * m->head_dim / 2);  // bf16
    b.part_ml = cv.take<float>((size_t)worst * m->n_q_heads * 2);
    b.part_rows = worst;
  }
}

struct ReuseBufs {
  float *rope;
  int32_t *meta, *tok_delta, *tok_chunk;
  float *h_full;
  LayerBufs lb;
  void *k_chk, *v_chk;
  float *d_k, *d_v, *w_k, *w_v;
  uint8_t *flags;
  int32_t *chunk_rows, *rows, *n_rows, *fresh_row, *probe_k, *probe_v;
  float *h_probe;
  void *k_fresh, *v_fresh;
  float *mu_k, *mu_v;
  float *h_last;  // the query rows' residual stream at the last layer
  void *q_last;   // and their queries
  int32_t *plan_rows, *plan_q;  // attention split plans: recomputed rows, query rows
};

size_t carve_reuse(void *ws, const akvs_model_cfg *m, const akvs_reuse_cfg *c, const Meta &mt,
                   ReuseBufs &b) {
  Carver cv(ws);
  const size_t es = es_of(m->dtype);
  const long long T = mt.t_all, Tc = mt.t_ctx, cap = mt.row_cap;
  const int kvw = m->n_kv_heads * m->head_dim;
  b.rope = cv.take<float>((size_t)T * m->head_dim);
  b.meta = cv.take<int32_t>((size_t)c->n_chunks * 8);
  b.tok_delta = cv.take<int32_t>((size_t)Tc);
  b.tok_chunk = cv.take<int32_t>((size_t)Tc);
  b.h_full = cv.take<float>((size_t)T * m->d_model);
  carve_layer_bufs(cv, m, T, {{T, T}, {cap, T}, {c->query_len, T}}, b.lb);
  b.k_chk = cv.take<char>((size_t)Tc * kvw * es);
  b.v_chk = cv.take<char>((size_t)Tc * kvw * es);
  b.d_k = cv.take<float>((size_t)Tc);
  b.d_v = cv.take<float>((size_t)Tc);
  b.w_k = cv.take<float>((size_t)Tc);
  b.w_v = cv.take<float>((size_t)Tc);
  b.flags = cv.take<uint8_t>((size_t)Tc);
  b.chunk_rows = cv.take<int32_t>((size_t)c->n_chunks);
  b.rows = cv.take<int32_t>((size_t)T);
  b.n_rows = cv.take<int32_t>(1);
  b.fresh_row = cv.take<int32_t>((size_t)T);
  b.probe_k = cv.take<int32_t>((size_t)mt.sum_b + 1);
  b.probe_v = cv.take<int32_t>((size_t)mt.sum_b_v + 1);
  b.h_probe = cv.take<float>((size_t)cap * m->d_model);
  b.k_fresh = cv.take<char>((size_t)cap * kvw * es);
  b.v_fresh = cv.take<char>((size_t)cap * kvw * es);
  b.mu_k = cv.take<float>((size_t)c->n_chunks * kvw);
  b.mu_v = cv.take<float>((size_t)c->n_chunks * kvw);
  b.h_last = cv.take<float>((size_t)c->query_len * m->d_model);
  b.q_last = cv.take<char>((size_t)c->query_len * m->n_q_heads * m->head_dim * es);
  b.plan_rows = cv.take<int32_t>(kAttnPlanInts);
  b.plan_q = cv.take<int32_t>(kAttnPlanInts);
  return cv.off;
}

struct FullBufs {
  float *rope, *h;
  LayerBufs lb;
};

size_t carve_full(void *ws, const akvs_model_cfg *m, long long n, FullBufs &b) {
  Carver cv(ws);
  b.rope = cv.take<float>((size_t)n * m->head_dim);
  b.h = cv.take<float>((size_t)n * m->d_model);
  carve_layer_bufs(cv, m, n, {{n, n}}, b.lb);
  return cv.off;
}

size_t carve_step(void *ws, const akvs_model_cfg *m, long long n, void **x, void **act,
                  float **gpart) {
  Carver cv(ws);
  const size_t es = es_of(m->dtype);
  *x = cv.take<char>((size_t)n * m->d_model * es);
  *act = cv.take<char>((size_t)n * m->ffn_dim * es);
  const size_t g = layer_gemm_part(m, n);
  *gpart = g ? cv.take<float>(g) : nullptr;
  return cv.off;
}

// Small host arrays go to the device as kernel arguments (no pageable copies).
struct IntChunk {
  int n;
  int32_t v[240];
};
__global__ void k_put_ints(IntChunk c, int32_t *dst) {
  for (int i = threadIdx.x; i < c.n; i += blockDim.x) dst[i] = c.v[i];
}
hipError_t put_ints(const int32_t *host, size_t n, int32_t *dst, hipStream_t s) {
  for (size_t o = 0; o < n; o += 240) {
    IntChunk c;
    c.n = (int)((n - o) < 240 ? (n - o) : 240);
    memcpy(c.v, host + o, sizeof(int32_t) * c.n);
    hipLaunchKernelGGL(k_put_ints, dim3(1), dim3(256), 0, s, c, dst + o);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// ---- the layer passes -----------------------------------------------------------------------
Epi qkv_epi(const akvs_model_cfg *m, void *q, void *k, void *v, const int32_t *pos, int pos0,
            int kv_by_pos, const float *rope, int rope_rows, int rope_base) {
  Epi e{};
  e.mode = EPI_QKV;
  e.out_dtype = m->dtype;
  e.q_out = q;
  e.k_out = k;
  e.v_out = v;
  e.n_off = 0;
  e.hq_w = m->n_q_heads * m->head_dim;
  e.kv_w = m->n_kv_heads * m->head_dim;
  e.hd = m->head_dim;
  e.pos = pos;
  e.pos0 = pos0;
  e.kv_by_pos = kv_by_pos;
  e.rope = rope;
  e.rope_rows = rope_rows;
  e.rope_base = rope_base;
  return e;
}

Epi simple_epi(int mode, void *out, int ldo, int dtype) {
  Epi e{};
  e.mode = mode;
  e.out = out;
  e.ldo = ldo;
  e.out_dtype = dtype;
  return e;
}

// Attention output projection + MLP over rows (h updated in place).
akvs_status out_mlp(const akvs_model_cfg *m, const akvs_layer_w &w, float *h, int rows,
                    const int32_t *rows_dev, const void *att, void *x, void *act, float *gpart,
                    hipStream_t stream, int rows_min = 0) {
  const int D = m->d_model, F = m->ffn_dim, hqw = m->n_q_heads * m->head_dim;
  GEMM(att, hqw, w.w_o, hqw, rows, D, hqw, rows_dev, m->dtype,
                                  simple_epi(EPI_RESID, h, D, AKVS_F32), stream, gpart,
                                  rows_min);
  LAUNCH(AKVS_K_NORM, launch_rmsnorm(h, D, rows, rows_dev, nullptr, w.mlp_norm, m->dtype, D,
                                     m->rms_eps, x, m->dtype, D, stream));
  GEMM(x, D, w.w_gate_up, D, rows, F, D, rows_dev, m->dtype,
                                  simple_epi(EPI_SWIGLU, act, F, m->dtype), stream, gpart,
                                  rows_min);
  GEMM(act, F, w.w_down, F, rows, D, F, rows_dev, m->dtype,
                                  simple_epi(EPI_RESID, h, D, AKVS_F32), stream, gpart,
                                  rows_min);
  return AKVS_OK;
}

// Attention split plan of full_layer over n rows (into lb.plan, read by every such layer).
hipError_t plan_full_layers(const akvs_model_cfg *m, int n, const LayerBufs &lb,
                            hipStream_t stream) {
  return launch_attention_plan(nullptr, 0, n, nullptr, n, m->n_q_heads, m->head_dim, m->dtype,
                               lb.part_rows, lb.plan, stream);
}

// One ordinary causal layer over n consecutive rows at positions pos0.. (keys written to
// k_dst / v_dst rows 0..n-1). With planned = true, plan_full_layers(m, n, lb) ran before.
akvs_status full_layer(const akvs_model_cfg *m, const akvs_layer_w &w, float *h, int n, int pos0,
                       const float *rope, const LayerBufs &lb, void *k_dst, void *v_dst,
                       hipStream_t stream, bool planned) {
  const int D = m->d_model;
  const int qkvw = (m->n_q_heads + 2 * m->n_kv_heads) * m->head_dim;
  LAUNCH(AKVS_K_NORM, launch_rmsnorm(h, D, n, nullptr, nullptr, w.attn_norm, m->dtype, D,
                                     m->rms_eps, lb.x, m->dtype, D, stream));
  GEMM(lb.x, D, w.w_qkv, D, n, qkvw, D, nullptr, m->dtype,
                                  qkv_epi(m, lb.q, k_dst, v_dst, nullptr, pos0, 0, rope, n, pos0),
                                  stream, lb.gpart);
  LAUNCH(AKVS_K_ATTENTION, launch_attention(lb.q, nullptr, 0, n, nullptr, k_dst, v_dst, n,
                                            m->n_q_heads, m->n_kv_heads, m->head_dim, m->dtype,
                                            lb.att, lb.part_o, lb.part_ml, lb.part_rows, stream,
                                            nullptr, planned ? lb.plan : nullptr));
  return out_mlp(m, w, h, n, nullptr, lb.att, lb.x, lb.act, lb.gpart, stream);
}

// ---- batched reuse prefill ---------------------------------------------------------------
// Per request: its unit bookkeeping, selection and correction inputs. Shared: the buffers
// of the per-request prefix layers and check layer (used one request after another), and
// the combined row block of all requests' recomputed rows for the layers from the check
// layer on, where request b owns rows row_off[b] .. row_off[b] + n_rows[b].
struct BatchReq {
  int32_t *meta, *tok_delta, *tok_chunk;
  float *h_full;
  float *d_k, *d_v, *w_k, *w_v;
  uint8_t *flags;
  int32_t *chunk_rows, *rows, *fresh_row, *probe_k, *probe_v;
  float *mu_k, *mu_v;
  int32_t *plan_rows, *plan_q;  // attention split plans: recomputed rows, query rows
};

struct BatchBufs {
  float *rope;
  LayerBufs lb_full;  // prefix / check layer of one request at a time
  void *k_chk, *v_chk;
  int32_t *n_rows, *row_off, *pos;  // [B], [B + 1], [sum caps]
  float *h_probe;                   // [sum caps][D]
  void *k_fresh, *v_fresh;          // [sum caps][kvw]
  LayerBufs lb;                     // combined rows (x, q, att, act, partials)
  float *h_last;                    // [sum q][D]
  void *q_last;                     // [sum q][Hq hd]
  std::vector<BatchReq> req;
};

struct BatchPlan {
  std::vector<Meta> mt;
  long long t_max = 0, tc_max = 0, cap_sum = 0, q_sum = 0, min_sum = 0;
};

size_t carve_batch(void *ws, const akvs_model_cfg *m, const akvs_reuse_cfg *cfgs, int B,
                   const BatchPlan &pl, BatchBufs &b) {
  Carver cv(ws);
  const size_t es = es_of(m->dtype);
  const int kvw = m->n_kv_heads * m->head_dim, hqw = m->n_q_heads * m->head_dim;
  const int D = m->d_model;
  b.rope = cv.take<float>((size_t)pl.t_max * m->head_dim);
  {  // each request's prefix layers use the buffers the single-request call would
    std::vector<AttnUse> uses;
    for (int i = 0; i < B; ++i) uses.push_back({pl.mt[i].t_all, pl.mt[i].t_all});
    carve_layer_bufs(cv, m, pl.t_max, uses, b.lb_full);
  }
  b.k_chk = cv.take<char>((size_t)pl.tc_max * kvw * es);
  b.v_chk = cv.take<char>((size_t)pl.tc_max * kvw * es);
  b.n_rows = cv.take<int32_t>((size_t)B);
  b.row_off = cv.take<int32_t>((size_t)B + 1);
  b.pos = cv.take<int32_t>((size_t)pl.cap_sum);
  b.h_probe = cv.take<float>((size_t)pl.cap_sum * D);
  b.k_fresh = cv.take<char>((size_t)pl.cap_sum * kvw * es);
  b.v_fresh = cv.take<char>((size_t)pl.cap_sum * kvw * es);
  // combined row buffers; the attention partials are sized for the largest request call
  b.lb.x = cv.take<char>((size_t)pl.cap_sum * D * es);
  b.lb.q = cv.take<char>((size_t)pl.cap_sum * hqw * es);
  b.lb.att = cv.take<char>((size_t)pl.cap_sum * hqw * es);
  b.lb.act = cv.take<char>((size_t)pl.cap_sum * m->ffn_dim * es);
  b.lb.gpart = nullptr;
  b.lb.part_o = b.lb.part_ml = nullptr;
  b.lb.part_rows = 0;
  b.lb.plan = nullptr;
  {
    const size_t g = std::max(layer_gemm_part(m, pl.cap_sum), layer_gemm_part(m, pl.q_sum));
    if (g) b.lb.gpart = cv.take<float>(g);
  }
  if (m->dtype == AKVS_BF16) {  // attention runs per request: its largest split partials
    long long worst = 0;
    for (int i = 0; i < B; ++i) {
      for (long long r : {pl.mt[i].row_cap, (long long)cfgs[i].query_len}) {
        const long long sp = attn_part_splits((int)r, m->n_q_heads, m->n_kv_heads, m->head_dim,
                                              (int)pl.mt[i].t_all);
        if (sp > 1 && sp * r > worst) worst = sp * r;
      }
    }
    if (worst > 0) {
      b.lb.part_o = cv.take<float>((size_t)worst * hqw / 2);  // bf16 elements
      b.lb.part_ml = cv.take<float>((size_t)worst * m->n_q_heads * 2);
      b.lb.part_rows = worst;
    }
  }
  b.h_last = cv.take<float>((size_t)pl.q_sum * D);
  b.q_last = cv.take<char>((size_t)pl.q_sum * hqw * es);
  b.req.resize(B);
  for (int i = 0; i < B; ++i) {
    const Meta &mt = pl.mt[i];
    BatchReq &r = b.req[i];
    const int nch = cfgs[i].n_chunks;
    r.meta = cv.take<int32_t>((size_t)nch * 8);
    r.tok_delta = cv.take<int32_t>((size_t)mt.t_ctx);
    r.tok_chunk = cv.take<int32_t>((size_t)mt.t_ctx);
    r.h_full = cv.take<float>((size_t)mt.t_all * D);
    r.d_k = cv.take<float>((size_t)mt.t_ctx);
    r.d_v = cv.take<float>((size_t)mt.t_ctx);
    r.w_k = cv.take<float>((size_t)mt.t_ctx);
    r.w_v = cv.take<float>((size_t)mt.t_ctx);
    r.flags = cv.take<uint8_t>((size_t)mt.t_ctx);
    r.chunk_rows = cv.take<int32_t>((size_t)nch);
    r.rows = cv.take<int32_t>((size_t)mt.t_all);
    r.fresh_row = cv.take<int32_t>((size_t)mt.t_all);
    r.probe_k = cv.take<int32_t>((size_t)mt.sum_b + 1);
    r.probe_v = cv.take<int32_t>((size_t)mt.sum_b_v + 1);
    r.mu_k = cv.take<float>((size_t)nch * kvw);
    r.mu_v = cv.take<float>((size_t)nch * kvw);
    r.plan_rows = cv.take<int32_t>(kAttnPlanInts);
    r.plan_q = cv.take<int32_t>(kAttnPlanInts);
  }
  return cv.off;
}

akvs_status batch_plan(const akvs_model_cfg *m, const akvs_reuse_cfg *cfgs, int B,
                       BatchPlan *pl) {
  REQUIRE(B >= 1 && B <= 1024, AKVS_EINVAL, "batch %d outside [1, 1024]", B);
  REQUIRE(cfgs, AKVS_EINVAL, "cfgs is NULL");
  pl->mt.assign(B, Meta());
  for (int i = 0; i < B; ++i) {
    akvs_status st = check_reuse(&cfgs[i], m->n_layers, &pl->mt[i]);
    if (st) return st;
    REQUIRE(cfgs[i].check_layer == cfgs[0].check_layer &&
                (cfgs[i].flags & AKVS_F_NO_PREFIX_RECOMPUTE) ==
                    (cfgs[0].flags & AKVS_F_NO_PREFIX_RECOMPUTE),
            AKVS_EINVAL, "request %d: every request needs the same check layer and prefix mode", i);
    pl->t_max = std::max(pl->t_max, pl->mt[i].t_all);
    pl->tc_max = std::max(pl->tc_max, pl->mt[i].t_ctx);
    pl->cap_sum += pl->mt[i].row_cap;
    pl->q_sum += cfgs[i].query_len;
    pl->min_sum += pl->mt[i].row_min;
  }
  REQUIRE(pl->cap_sum < (1LL << 28), AKVS_ESHAPE, "batch too large");
  return AKVS_OK;
}

}  // namespace

// =============================================================================================
extern "C" {

int32_t akvs_version(void) { return 100; }

const char *akvs_status_string(akvs_status s) {
  switch (s) {
    case AKVS_OK: return "ok";
    case AKVS_EINVAL: return "invalid argument";
    case AKVS_ESHAPE: return "inconsistent shape";
    case AKVS_EDTYPE: return "unsupported dtype for this argument";
    case AKVS_EUNSUPPORTED: return "unsupported configuration";
    case AKVS_ENOSPACE: return "workspace too small";
    case AKVS_EHIP: return "HIP runtime error";
    default: return "unknown status";
  }
}

const char *akvs_last_error(void) { return g_err; }

akvs_status akvs_chunk_meta(const akvs_reuse_cfg *cfg, int32_t *meta_out, int32_t *totals_out) {
  Meta mt;
  akvs_status st = check_reuse(cfg, 0, &mt);
  if (st) return st;
  if (meta_out) memcpy(meta_out, mt.m.data(), mt.m.size() * sizeof(int32_t));
  if (totals_out) {
    totals_out[0] = (int32_t)mt.t_ctx;
    totals_out[1] = (int32_t)mt.sum_b;
    totals_out[2] = (int32_t)mt.row_cap;
    totals_out[3] = (int32_t)mt.t_all;
    totals_out[4] = (int32_t)mt.sum_b_v;
  }
  return AKVS_OK;
}

size_t akvs_workspace_size(const akvs_model_cfg *m, const akvs_reuse_cfg *cfg, int32_t n_tokens) {
  if (check_model(m) != AKVS_OK) return 0;
  if (cfg) {
    Meta mt;
    if (check_reuse(cfg, m->n_layers, &mt) != AKVS_OK) return 0;
    ReuseBufs b;
    return carve_reuse(nullptr, m, cfg, mt, b);
  }
  if (n_tokens < 1) return 0;
  FullBufs b;
  return carve_full(nullptr, m, n_tokens, b);
}

size_t akvs_step_workspace_size(const akvs_model_cfg *m, int32_t n_rows) {
  if (check_model(m) != AKVS_OK || n_rows < 0) return 0;
  void *x, *a;
  float *g;
  return carve_step(nullptr, m, n_rows, &x, &a, &g);
}

akvs_status akvs_profile_enable(int32_t class_mask) {
  std::lock_guard<std::mutex> lk(g_prof.mu);
  g_prof.mask = (uint32_t)class_mask & ((1u << AKVS_K_NCLASSES) - 1u);
  return AKVS_OK;
}

akvs_status akvs_profile_read(int32_t cls, int64_t *launches, double *total_ms) {
  REQUIRE(cls >= 0 && cls < AKVS_K_NCLASSES, AKVS_EINVAL, "kernel class %d", cls);
  std::lock_guard<std::mutex> lk(g_prof.mu);
  prof_drain();
  if (launches) *launches = g_prof.launches[cls];
  if (total_ms) *total_ms = g_prof.ms[cls];
  g_prof.launches[cls] = 0;
  g_prof.ms[cls] = 0.0;
  return AKVS_OK;
}

akvs_status akvs_mfma_busy_loop(int32_t n_blocks, int32_t iters, float *out, hipStream_t stream) {
  REQUIRE(n_blocks >= 0 && iters >= 0, AKVS_EINVAL, "n_blocks and iters must be >= 0");
  REQUIRE(n_blocks == 0 || out, AKVS_EINVAL, "NULL argument");
  REQUIRE(aligned16(out), AKVS_EINVAL, "misaligned argument");
  LAUNCH(AKVS_K_OTHER, launch_mfma_busy_loop(n_blocks, iters, out, stream));
  return AKVS_OK;
}

// ---- step entries ---------------------------------------------------------------------------

akvs_status akvs_rope_table(int32_t n_pos, int32_t head_dim, float rope_theta, float *table,
                            hipStream_t stream) {
  REQUIRE(n_pos >= 0, AKVS_EINVAL, "n_pos must be >= 0");
  REQUIRE(head_dim >= 2 && head_dim % 2 == 0 && head_dim <= 1024, AKVS_EINVAL, "bad head_dim");
  REQUIRE(rope_theta > 0.f, AKVS_EINVAL, "rope_theta must be > 0");
  REQUIRE(table && aligned16(table), AKVS_EINVAL, "table NULL or misaligned");
  LAUNCH(AKVS_K_OTHER, launch_rope_table(0, n_pos, head_dim, (double)rope_theta, table, stream));
  return AKVS_OK;
}

static akvs_status check_kv_geom(int32_t n_tokens, int32_t hkv, int32_t hd) {
  REQUIRE(n_tokens >= 0 && hkv >= 1, AKVS_EINVAL, "n_tokens >= 0, n_kv_heads >= 1");
  REQUIRE(hd == 64 || hd == 128, AKVS_EUNSUPPORTED, "head_dim %d not supported", hd);
  REQUIRE((long long)n_tokens * hkv * hd < (1LL << 40), AKVS_ESHAPE, "too large");
  return AKVS_OK;
}

akvs_status akvs_rerotate_keys(const akvs_cache *src, int32_t n_tokens, int32_t n_kv_heads,
                               int32_t head_dim, const int32_t *pos_delta, const float *rope,
                               int32_t rope_rows, void *k_dst, void *v_dst, int32_t dst_dtype,
                               hipStream_t stream) {
  akvs_status st = check_kv_geom(n_tokens, n_kv_heads, head_dim);
  if (st) return st;
  akvs_model_cfg fake{};
  fake.dtype = dst_dtype;
  REQUIRE(dst_dtype == AKVS_F32 || dst_dtype == AKVS_BF16, AKVS_EDTYPE, "dst dtype");
  st = check_cache(src, &fake);
  if (st) return st;
  REQUIRE(pos_delta && rope && rope_rows >= 1 && k_dst && v_dst, AKVS_EINVAL, "NULL argument");
  REQUIRE(aligned16(rope) && aligned16(k_dst) && aligned16(v_dst), AKVS_EINVAL, "misaligned");
  CacheLayer cl = cache_layer(src, 0, n_tokens, n_kv_heads, head_dim);
  LAUNCH(AKVS_K_CORRECTION,
         launch_correction(cl, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr,
                           nullptr, nullptr, pos_delta, nullptr, 0, n_tokens, n_tokens, n_kv_heads,
                           head_dim, 0u, rope, rope_rows, k_dst, v_dst, dst_dtype, stream));
  return AKVS_OK;
}

akvs_status akvs_check_divergence(const void *k_fresh, const void *v_fresh, int32_t fresh_dtype,
                                  const akvs_cache *cache, int32_t n_tokens, int32_t n_kv_heads,
                                  int32_t head_dim, const int32_t *pos_delta, const float *rope,
                                  int32_t rope_rows, float *d_k, float *d_v, hipStream_t stream) {
  akvs_status st = check_kv_geom(n_tokens, n_kv_heads, head_dim);
  if (st) return st;
  REQUIRE(fresh_dtype == AKVS_F32 || fresh_dtype == AKVS_BF16, AKVS_EDTYPE, "fresh dtype");
  akvs_model_cfg fake{};
  fake.dtype = fresh_dtype;
  st = check_cache(cache, &fake);
  if (st) return st;
  REQUIRE(k_fresh && v_fresh && d_k && d_v, AKVS_EINVAL, "NULL argument");
  REQUIRE(aligned16(k_fresh) && aligned16(v_fresh), AKVS_EINVAL, "misaligned");
  REQUIRE(!pos_delta || (rope && rope_rows >= 1 && aligned16(rope)), AKVS_EINVAL,
          "pos_delta needs a rotary table");
  CacheLayer cl = cache_layer(cache, 0, n_tokens, n_kv_heads, head_dim);
  LAUNCH(AKVS_K_DIVERGENCE,
         launch_divergence(k_fresh, v_fresh, fresh_dtype, cl, n_tokens, n_kv_heads, head_dim,
                           pos_delta, rope, pos_delta ? rope_rows : 1, d_k, d_v, stream));
  return AKVS_OK;
}

akvs_status akvs_select_probes(const float *d_k, const float *d_v, const akvs_reuse_cfg *cfg,
                               const int32_t *chunk_meta, int32_t *probe_k, int32_t *probe_v,
                               float *w_k, float *w_v, uint8_t *flags, int32_t *chunk_rows,
                               int32_t *rows, int32_t *n_rows, int32_t *fresh_row,
                               hipStream_t stream) {
  Meta mt;
  akvs_status st = check_reuse(cfg, 0, &mt);
  if (st) return st;
  REQUIRE(d_k && d_v && chunk_meta && (probe_k || mt.sum_b == 0) &&
              (probe_v || mt.sum_b_v == 0) && w_k && w_v && flags && chunk_rows && rows &&
              n_rows && fresh_row,
          AKVS_EINVAL, "NULL argument");
  REQUIRE(aligned16(chunk_meta), AKVS_EINVAL, "chunk_meta misaligned");
  LAUNCH(AKVS_K_SELECT, launch_select(d_k, d_v, chunk_meta, cfg->n_chunks, (int)mt.t_ctx,
                                      cfg->query_len, cfg->flags, probe_k, probe_v, w_k, w_v, flags,
                                      chunk_rows, rows, n_rows, fresh_row, stream));
  return AKVS_OK;
}

akvs_status akvs_probe_qkv(const float *h, int32_t n_rows, const int32_t *positions,
                           const akvs_model_cfg *m, const akvs_layer_w *lw, const float *rope,
                           int32_t rope_rows, void *q, void *k_fresh, void *v_fresh, void *ws,
                           size_t ws_bytes, hipStream_t stream) {
  akvs_status st = check_model(m);
  if (st) return st;
  REQUIRE(n_rows >= 0, AKVS_EINVAL, "n_rows must be >= 0");
  REQUIRE(lw && lw->attn_norm && lw->w_qkv && aligned16(lw->attn_norm) && aligned16(lw->w_qkv),
          AKVS_EINVAL, "layer weights NULL or misaligned");
  REQUIRE(h && positions && rope && q && k_fresh && v_fresh, AKVS_EINVAL, "NULL argument");
  REQUIRE(aligned16(h) && aligned16(rope) && aligned16(q) && aligned16(k_fresh) &&
              aligned16(v_fresh) && aligned16(ws),
          AKVS_EINVAL, "misaligned argument");
  REQUIRE(rope_rows >= 1, AKVS_EINVAL, "rope_rows must be >= 1");
  void *x, *act;
  float *gpart;
  const size_t need = carve_step(nullptr, m, n_rows, &x, &act, &gpart);
  REQUIRE(ws && ws_bytes >= need, AKVS_ENOSPACE, "workspace %zu < %zu bytes", ws_bytes, need);
  carve_step(ws, m, n_rows, &x, &act, &gpart);
  const int D = m->d_model;
  const int qkvw = (m->n_q_heads + 2 * m->n_kv_heads) * m->head_dim;
  LAUNCH(AKVS_K_NORM, launch_rmsnorm(h, D, n_rows, nullptr, nullptr, lw->attn_norm, m->dtype, D,
                                     m->rms_eps, x, m->dtype, D, stream));
  GEMM(x, D, lw->w_qkv, D, n_rows, qkvw, D, nullptr, m->dtype,
                     qkv_epi(m, q, k_fresh, v_fresh, positions, 0, 0, rope, rope_rows, 0), stream,
                     gpart);
  return AKVS_OK;
}

akvs_status akvs_chunk_offset(const void *k_fresh, const void *v_fresh, const int32_t *fresh_row,
                              const akvs_cache *cache, const akvs_reuse_cfg *cfg,
                              const int32_t *chunk_meta, const int32_t *probe_k,
                              const int32_t *probe_v, const akvs_model_cfg *m, const float *rope,
                              int32_t rope_rows, float *mu_k, float *mu_v, hipStream_t stream) {
  akvs_status st = check_model(m);
  if (st) return st;
  Meta mt;
  if ((st = check_reuse(cfg, 0, &mt))) return st;
  if ((st = check_cache(cache, m))) return st;
  REQUIRE(k_fresh && v_fresh && fresh_row && chunk_meta && (probe_k || mt.sum_b == 0) &&
              (probe_v || mt.sum_b_v == 0) && rope && mu_k && mu_v,
          AKVS_EINVAL, "NULL argument");
  REQUIRE(aligned16(chunk_meta) && aligned16(mu_k) && aligned16(mu_v) && aligned16(rope),
          AKVS_EINVAL, "misaligned argument");
  REQUIRE(rope_rows >= 1, AKVS_EINVAL, "rope_rows must be >= 1");
  CacheLayer cl = cache_layer(cache, 0, mt.t_ctx, m->n_kv_heads, m->head_dim);
  LAUNCH(AKVS_K_OFFSET, launch_chunk_offset(k_fresh, v_fresh, m->dtype, fresh_row, cl, chunk_meta,
                                            cfg->n_chunks, probe_k, probe_v, cfg->flags,
                                            m->n_kv_heads, m->head_dim, rope, rope_rows, mu_k,
                                            mu_v, stream));
  return AKVS_OK;
}

akvs_status akvs_apply_correction(const akvs_cache *cache, const float *mu_k, const float *mu_v,
                                  const float *w_k, const float *w_v, const uint8_t *flags,
                                  const void *k_fresh, const void *v_fresh,
                                  const int32_t *fresh_row, const akvs_reuse_cfg *cfg,
                                  const int32_t *chunk_meta, const akvs_model_cfg *m,
                                  const float *rope, int32_t rope_rows, void *k_corr,
                                  void *v_corr, hipStream_t stream) {
  akvs_status st = check_model(m);
  if (st) return st;
  Meta mt;
  if ((st = check_reuse(cfg, 0, &mt))) return st;
  if ((st = check_cache(cache, m))) return st;
  REQUIRE(mu_k && mu_v && w_k && w_v && flags && k_fresh && v_fresh && fresh_row && chunk_meta &&
              rope && k_corr && v_corr,
          AKVS_EINVAL, "NULL argument");
  REQUIRE(aligned16(mu_k) && aligned16(mu_v) && aligned16(k_fresh) && aligned16(v_fresh) &&
              aligned16(chunk_meta) && aligned16(rope) && aligned16(k_corr) && aligned16(v_corr),
          AKVS_EINVAL, "misaligned argument");
  REQUIRE(rope_rows >= 1, AKVS_EINVAL, "rope_rows must be >= 1");
  CacheLayer cl = cache_layer(cache, 0, mt.t_ctx, m->n_kv_heads, m->head_dim);
  LAUNCH(AKVS_K_CORRECTION,
         launch_correction(cl, mu_k, mu_v, w_k, w_v, flags, k_fresh, v_fresh, fresh_row, nullptr,
                           nullptr, chunk_meta, cfg->n_chunks, (int)mt.t_ctx, (int)mt.t_all,
                           m->n_kv_heads, m->head_dim, cfg->flags, rope, rope_rows, k_corr,
                           v_corr, m->dtype, stream));
  return AKVS_OK;
}

// Key-split partials of one attention call over `rows` rows (bf16 models that split).
static size_t attention_part_floats(const akvs_model_cfg *m, long long rows, long long n_keys,
                                    size_t *ml_floats) {
  *ml_floats = 0;
  if (m->dtype != AKVS_BF16 || rows <= 0) return 0;
  const long long sp =
      attn_part_splits((int)rows, m->n_q_heads, m->n_kv_heads, m->head_dim, (int)n_keys);
  if (sp < 2) return 0;
  *ml_floats = (size_t)(sp * rows) * m->n_q_heads * 2;
  return (size_t)(sp * rows) * m->n_q_heads * m->head_dim / 2;  // bf16 outputs, two per float
}

// The split partials, then the plan of the split (launch_attention_plan).
static size_t attention_ws_bytes(const akvs_model_cfg *m, long long rows, long long n_keys,
                                 size_t *o_floats, size_t *ml_floats) {
  *o_floats = attention_part_floats(m, rows, n_keys, ml_floats);
  if (!*o_floats) return 0;
  return align256(*o_floats * sizeof(float)) + align256(*ml_floats * sizeof(float)) +
         align256(kAttnPlanInts * sizeof(int32_t));
}

size_t akvs_attention_workspace_size(const akvs_model_cfg *m, int32_t n_rows, int32_t n_keys) {
  if (check_model(m) != AKVS_OK || n_rows < 0 || n_keys < 1) return 0;
  size_t o, ml;
  return attention_ws_bytes(m, n_rows, n_keys, &o, &ml);
}

akvs_status akvs_sparse_query_attention(const void *q, const int32_t *positions, int32_t n_rows,
                                        const void *k, const void *v, int32_t n_keys,
                                        const akvs_model_cfg *m, void *out, void *ws,
                                        size_t ws_bytes, hipStream_t stream) {
  akvs_status st = check_model(m);
  if (st) return st;
  REQUIRE(n_rows >= 0 && n_keys >= 1, AKVS_EINVAL, "n_rows >= 0, n_keys >= 1");
  REQUIRE(q && positions && k && v && out, AKVS_EINVAL, "NULL argument");
  REQUIRE(aligned16(q) && aligned16(k) && aligned16(v) && aligned16(out) && aligned16(ws),
          AKVS_EINVAL, "misaligned argument");
  float *part_o = nullptr, *part_ml = nullptr;
  int32_t *plan = nullptr;
  long long part_rows = 0;
  if (ws) {
    size_t o, ml;
    const size_t need = attention_ws_bytes(m, n_rows, n_keys, &o, &ml);
    REQUIRE(ws_bytes >= need, AKVS_ENOSPACE, "workspace %zu bytes, need %zu", ws_bytes, need);
    if (o) {
      Carver cv(ws);
      part_o = cv.take<float>(o);
      part_ml = cv.take<float>(ml);
      plan = cv.take<int32_t>(kAttnPlanInts);
      part_rows = (long long)(ml / ((size_t)m->n_q_heads * 2));
    }
  }
  if (plan)
    LAUNCH(AKVS_K_OTHER, launch_attention_plan(positions, 0, n_rows, nullptr, n_keys,
                                               m->n_q_heads, m->head_dim, m->dtype, part_rows,
                                               plan, stream));
  LAUNCH(AKVS_K_ATTENTION, launch_attention(q, positions, 0, n_rows, nullptr, k, v, n_keys,
                                            m->n_q_heads, m->n_kv_heads, m->head_dim, m->dtype,
                                            out, part_o, part_ml, part_rows, stream, nullptr,
                                            plan));
  return AKVS_OK;
}

akvs_status akvs_probe_out_mlp(float *h, int32_t n_rows, const void *attn_out,
                               const akvs_model_cfg *m, const akvs_layer_w *lw, void *ws,
                               size_t ws_bytes, hipStream_t stream) {
  akvs_status st = check_model(m);
  if (st) return st;
  REQUIRE(n_rows >= 0, AKVS_EINVAL, "n_rows must be >= 0");
  REQUIRE(lw && lw->w_o && lw->mlp_norm && lw->w_gate_up && lw->w_down, AKVS_EINVAL,
          "layer weights NULL");
  REQUIRE(aligned16(lw->w_o) && aligned16(lw->mlp_norm) && aligned16(lw->w_gate_up) &&
              aligned16(lw->w_down),
          AKVS_EINVAL, "layer weights misaligned");
  REQUIRE(h && attn_out && aligned16(h) && aligned16(attn_out) && aligned16(ws), AKVS_EINVAL,
          "NULL or misaligned argument");
  void *x, *act;
  float *gpart;
  const size_t need = carve_step(nullptr, m, n_rows, &x, &act, &gpart);
  REQUIRE(ws && ws_bytes >= need, AKVS_ENOSPACE, "workspace %zu < %zu bytes", ws_bytes, need);
  carve_step(ws, m, n_rows, &x, &act, &gpart);
  return out_mlp(m, *lw, h, n_rows, nullptr, attn_out, x, act, gpart, stream);
}

akvs_status akvs_quantize_cache(const void *x, int32_t x_dtype, int32_t n_rows, int32_t head_dim,
                                int32_t bits, uint8_t *codes, void *meta, hipStream_t stream) {
  REQUIRE(x_dtype == AKVS_F32 || x_dtype == AKVS_BF16, AKVS_EDTYPE, "x dtype");
  REQUIRE(bits == 2 || bits == 4 || bits == 8, AKVS_EINVAL, "bits must be 2, 4 or 8 (E4M3)");
  REQUIRE(n_rows >= 0 && head_dim >= 64 && head_dim % 64 == 0, AKVS_EINVAL,
          "head_dim must be a positive multiple of 64");
  REQUIRE(x && codes && meta, AKVS_EINVAL, "NULL argument");
  LAUNCH(AKVS_K_OTHER, launch_quantize(x, x_dtype, n_rows, head_dim, bits, codes,
                                       reinterpret_cast<_Float16 *>(meta), stream));
  return AKVS_OK;
}

// ---- whole-procedure entries ------------------------------------------------------------------

akvs_status akvs_full_prefill(const int32_t *tokens, int32_t n_tokens, int32_t pos0,
                              const void *embed, const akvs_layer_w *lw, const void *final_norm,
                              const akvs_model_cfg *m, float *h_out, void *k_out, void *v_out,
                              void *ws, size_t ws_bytes, hipStream_t stream) {
  akvs_status st = check_model(m);
  if (st) return st;
  if ((st = check_layers(m, lw))) return st;
  REQUIRE(n_tokens >= 1 && pos0 >= 0 && (long long)pos0 + n_tokens < (1LL << 28), AKVS_EINVAL,
          "need n_tokens >= 1, pos0 >= 0");
  REQUIRE(tokens && embed && final_norm && k_out && v_out, AKVS_EINVAL, "NULL argument");
  REQUIRE(aligned16(embed) && aligned16(final_norm) && aligned16(k_out) && aligned16(v_out) &&
              (!h_out || aligned16(h_out)) && aligned16(ws),
          AKVS_EINVAL, "misaligned argument");
  FullBufs b;
  const size_t need = carve_full(nullptr, m, n_tokens, b);
  REQUIRE(ws && ws_bytes >= need, AKVS_ENOSPACE, "workspace %zu < %zu bytes", ws_bytes, need);
  carve_full(ws, m, n_tokens, b);
  const int D = m->d_model;
  const size_t kvl = (size_t)n_tokens * m->n_kv_heads * m->head_dim * es_of(m->dtype);
  LAUNCH(AKVS_K_OTHER, launch_rope_table(pos0, n_tokens, m->head_dim, (double)m->rope_theta,
                                         b.rope, stream));
  LAUNCH(AKVS_K_OTHER, launch_embed(tokens, n_tokens, embed, m->dtype, m->vocab, D, b.h, stream));
  LAUNCH(AKVS_K_OTHER, plan_full_layers(m, n_tokens, b.lb, stream));
  for (int l = 0; l < m->n_layers; ++l) {
    st = full_layer(m, lw[l], b.h, n_tokens, pos0, b.rope, b.lb,
                    reinterpret_cast<char *>(k_out) + l * kvl,
                    reinterpret_cast<char *>(v_out) + l * kvl, stream, true);
    if (st) return st;
  }
  if (h_out)
    LAUNCH(AKVS_K_NORM, launch_rmsnorm(b.h, D, n_tokens, nullptr, nullptr, final_norm, m->dtype, D,
                                       m->rms_eps, h_out, AKVS_F32, D, stream));
  return AKVS_OK;
}

akvs_status akvs_reuse_prefill(const int32_t *tokens, const void *embed, const akvs_layer_w *lw,
                               const void *final_norm, const akvs_model_cfg *m,
                               const akvs_reuse_cfg *cfg, const akvs_cache *cache,
                               const akvs_reuse_out *out, void *ws, size_t ws_bytes,
                               hipStream_t stream) {
  akvs_status st = check_model(m);
  if (st) return st;
  if ((st = check_layers(m, lw))) return st;
  Meta mt;
  if ((st = check_reuse(cfg, m->n_layers, &mt))) return st;
  if ((st = check_cache(cache, m))) return st;
  REQUIRE(tokens && embed && final_norm && out, AKVS_EINVAL, "NULL argument");
  REQUIRE(out->h_query && out->k_corr && out->v_corr, AKVS_EINVAL,
          "h_query, k_corr and v_corr are required outputs");
  REQUIRE(aligned16(embed) && aligned16(final_norm) && aligned16(out->h_query) &&
              aligned16(out->k_corr) && aligned16(out->v_corr) && aligned16(ws),
          AKVS_EINVAL, "misaligned argument");
  const bool given = (cfg->flags & AKVS_F_GIVEN_PROBES) != 0;
  REQUIRE(!given || (out->probe_k && out->probe_v), AKVS_EINVAL,
          "AKVS_F_GIVEN_PROBES needs out->probe_k and out->probe_v holding the sets");
  ReuseBufs b;
  const size_t need = carve_reuse(nullptr, m, cfg, mt, b);
  REQUIRE(ws && ws_bytes >= need, AKVS_ENOSPACE, "workspace %zu < %zu bytes", ws_bytes, need);
  carve_reuse(ws, m, cfg, mt, b);
  // caller-visible outputs replace their workspace twins
  if (out->probe_k) b.probe_k = out->probe_k;
  if (out->probe_v) b.probe_v = out->probe_v;
  if (out->d_k) b.d_k = out->d_k;
  if (out->d_v) b.d_v = out->d_v;
  if (out->rows) b.rows = out->rows;
  if (out->n_rows) b.n_rows = out->n_rows;

  const int L = m->n_layers, D = m->d_model, hkv = m->n_kv_heads, hd = m->head_dim;
  const int kvw = hkv * hd, hqw = m->n_q_heads * hd;
  const int T = (int)mt.t_all, Tc = (int)mt.t_ctx, cap = (int)mt.row_cap;
  const int nch = cfg->n_chunks;
  const bool no_prefix = (cfg->flags & AKVS_F_NO_PREFIX_RECOMPUTE) != 0;
  const int c = no_prefix ? 0 : cfg->check_layer;
  const size_t es = es_of(m->dtype);
  REQUIRE(out->kv_rows == 0 || out->kv_rows >= T, AKVS_EINVAL,
          "kv_rows %d is below T = %d", out->kv_rows, T);
  const size_t corr_layer = (size_t)(out->kv_rows ? out->kv_rows : T) * kvw * es;
  char *k_corr = reinterpret_cast<char *>(out->k_corr);
  char *v_corr = reinterpret_cast<char *>(out->v_corr);

  LAUNCH(AKVS_K_OTHER, put_ints(mt.m.data(), mt.m.size(), b.meta, stream));
  LAUNCH(AKVS_K_OTHER, launch_rope_table(0, T, hd, (double)m->rope_theta, b.rope, stream));
  LAUNCH(AKVS_K_OTHER, launch_token_setup(b.meta, nch, b.tok_delta, b.tok_chunk, stream));
  LAUNCH(AKVS_K_OTHER, launch_embed(tokens, T, embed, m->dtype, m->vocab, D, b.h_full, stream));

  // layers before the check layer: every token
  if (c > 0) LAUNCH(AKVS_K_OTHER, plan_full_layers(m, T, b.lb, stream));
  for (int l = 0; l < c; ++l) {
    st = full_layer(m, lw[l], b.h_full, T, 0, b.rope, b.lb, k_corr + l * corr_layer,
                    v_corr + l * corr_layer, stream, true);
    if (st) return st;
  }
  // check layer: fresh K/V of every unit token, divergence against the re-rotated cache
  if (!no_prefix) {
    LAUNCH(AKVS_K_NORM, launch_rmsnorm(b.h_full, D, Tc, nullptr, nullptr, lw[c].attn_norm,
                                       m->dtype, D, m->rms_eps, b.lb.x, m->dtype, D, stream));
    Epi e = qkv_epi(m, nullptr, b.k_chk, b.v_chk, nullptr, 0, 0, b.rope, T, 0);
    e.n_off = hqw;
    const char *wkv = reinterpret_cast<const char *>(lw[c].w_qkv) + (size_t)hqw * D * es;
    GEMM(b.lb.x, D, wkv, D, Tc, 2 * kvw, D, nullptr, m->dtype, e,
                                    stream);
    LAUNCH(AKVS_K_DIVERGENCE,
           launch_divergence(b.k_chk, b.v_chk, m->dtype, cache_layer(cache, c, Tc, hkv, hd), Tc,
                             hkv, hd, b.tok_delta, b.rope, T, b.d_k, b.d_v, stream));
  }
  LAUNCH(AKVS_K_SELECT, launch_select(b.d_k, b.d_v, b.meta, nch, Tc, cfg->query_len, cfg->flags,
                                      b.probe_k, b.probe_v, b.w_k, b.w_v, b.flags, b.chunk_rows,
                                      b.rows, b.n_rows, b.fresh_row, stream));
  LAUNCH(AKVS_K_OTHER, launch_gather_rows(b.h_full, T, b.rows, cap, b.n_rows, D, b.h_probe,
                                          stream));
  // one key-split plan per row set, for every layer's attention over it
  LAUNCH(AKVS_K_OTHER, launch_attention_plan(b.rows, 0, cap, b.n_rows, T, m->n_q_heads, hd,
                                             m->dtype, b.lb.part_rows, b.plan_rows, stream));
  LAUNCH(AKVS_K_OTHER, launch_attention_plan(nullptr, Tc, cfg->query_len, nullptr, T,
                                             m->n_q_heads, hd, m->dtype, b.lb.part_rows, b.plan_q,
                                             stream));
  // from the check layer on: recomputed rows only, every unit token corrected
  const int qkvw = hqw + 2 * kvw;
  for (int l = c; l < L; ++l) {
    CacheLayer cl = cache_layer(cache, l, Tc, hkv, hd);
    LAUNCH(AKVS_K_NORM, launch_rmsnorm(b.h_probe, D, cap, b.n_rows, nullptr, lw[l].attn_norm,
                                       m->dtype, D, m->rms_eps, b.lb.x, m->dtype, D, stream));
    GEMM(b.lb.x, D, lw[l].w_qkv, D, cap, qkvw, D, b.n_rows, m->dtype,
                       qkv_epi(m, b.lb.q, b.k_fresh, b.v_fresh, b.rows, 0, 0, b.rope, T, 0),
                       stream, b.lb.gpart, (int)mt.row_min);
    LAUNCH(AKVS_K_OFFSET, launch_chunk_offset(b.k_fresh, b.v_fresh, m->dtype, b.fresh_row, cl,
                                              b.meta, nch, b.probe_k, b.probe_v, cfg->flags, hkv,
                                              hd, b.rope, T, b.mu_k, b.mu_v, stream));
    void *kl = k_corr + l * corr_layer;
    void *vl = v_corr + l * corr_layer;
    LAUNCH(AKVS_K_CORRECTION,
           launch_correction(cl, b.mu_k, b.mu_v, b.w_k, b.w_v, b.flags, b.k_fresh, b.v_fresh,
                             b.fresh_row, b.tok_chunk, b.tok_delta, b.meta, nch, Tc, T, hkv, hd,
                             cfg->flags, b.rope, T, kl, vl, m->dtype, stream));
    if (l + 1 < L) {
      LAUNCH(AKVS_K_ATTENTION, launch_attention(b.lb.q, b.rows, 0, cap, b.n_rows, kl, vl, T,
                                                m->n_q_heads, hkv, hd, m->dtype, b.lb.att,
                                                b.lb.part_o, b.lb.part_ml, b.lb.part_rows,
                                                stream, nullptr, b.plan_rows));
      st = out_mlp(m, lw[l], b.h_probe, cap, b.n_rows, b.lb.att, b.lb.x, b.lb.act, b.lb.gpart,
                   stream, (int)mt.row_min);
      if (st) return st;
      continue;
    }
    // last layer: only the query rows' attention and MLP reach the returned outputs (the
    // recomputed unit rows only had to supply this layer's fresh keys and values)
    const int q = cfg->query_len;
    LAUNCH(AKVS_K_OTHER, launch_copy_tail_rows(b.lb.q, (size_t)hqw * es, q, b.n_rows, b.q_last,
                                               stream));
    LAUNCH(AKVS_K_OTHER, launch_copy_tail_rows(b.h_probe, (size_t)D * 4, q, b.n_rows, b.h_last,
                                               stream));
    LAUNCH(AKVS_K_ATTENTION, launch_attention(b.q_last, nullptr, Tc, q, nullptr, kl, vl, T,
                                              m->n_q_heads, hkv, hd, m->dtype, b.lb.att,
                                              b.lb.part_o, b.lb.part_ml, b.lb.part_rows, stream,
                                              nullptr, b.plan_q));
    st = out_mlp(m, lw[l], b.h_last, q, nullptr, b.lb.att, b.lb.x, b.lb.act, b.lb.gpart, stream);
    if (st) return st;
  }
  LAUNCH(AKVS_K_NORM, launch_rmsnorm(b.h_last, D, cfg->query_len, nullptr, nullptr, final_norm,
                                     m->dtype, D, m->rms_eps, out->h_query, AKVS_F32, D, stream));
  return AKVS_OK;
}

size_t akvs_batch_workspace_size(const akvs_model_cfg *m, const akvs_reuse_cfg *cfgs,
                                 int32_t batch) {
  if (check_model(m) != AKVS_OK) return 0;
  BatchPlan pl;
  if (batch_plan(m, cfgs, batch, &pl) != AKVS_OK) return 0;
  BatchBufs b;
  return carve_batch(nullptr, m, cfgs, batch, pl, b);
}

akvs_status akvs_reuse_prefill_batch(const int32_t *const *tokens, int32_t batch,
                                     const void *embed, const akvs_layer_w *lw,
                                     const void *final_norm, const akvs_model_cfg *m,
                                     const akvs_reuse_cfg *cfgs, const akvs_cache *caches,
                                     const akvs_reuse_out *outs, void *ws, size_t ws_bytes,
                                     hipStream_t stream) {
  akvs_status st = check_model(m);
  if (st) return st;
  if ((st = check_layers(m, lw))) return st;
  BatchPlan pl;
  if ((st = batch_plan(m, cfgs, batch, &pl))) return st;
  REQUIRE(tokens && caches && outs && embed && final_norm, AKVS_EINVAL, "NULL argument");
  REQUIRE(aligned16(embed) && aligned16(final_norm) && aligned16(ws), AKVS_EINVAL,
          "misaligned argument");
  for (int i = 0; i < batch; ++i) {
    if ((st = check_cache(&caches[i], m))) return st;
    const akvs_reuse_out &o = outs[i];
    REQUIRE(tokens[i], AKVS_EINVAL, "request %d: tokens are NULL", i);
    REQUIRE(o.h_query && o.k_corr && o.v_corr, AKVS_EINVAL,
            "request %d: h_query, k_corr and v_corr are required outputs", i);
    REQUIRE(aligned16(o.h_query) && aligned16(o.k_corr) && aligned16(o.v_corr), AKVS_EINVAL,
            "request %d: misaligned output", i);
    REQUIRE(!(cfgs[i].flags & AKVS_F_GIVEN_PROBES) || (o.probe_k && o.probe_v), AKVS_EINVAL,
            "request %d: AKVS_F_GIVEN_PROBES needs out->probe_k and out->probe_v", i);
    REQUIRE(o.kv_rows == 0 || o.kv_rows >= pl.mt[i].t_all, AKVS_EINVAL,
            "request %d: kv_rows below its token count", i);
  }
  BatchBufs b;
  const size_t need = carve_batch(nullptr, m, cfgs, batch, pl, b);
  REQUIRE(ws && ws_bytes >= need, AKVS_ENOSPACE, "workspace %zu < %zu bytes", ws_bytes, need);
  carve_batch(ws, m, cfgs, batch, pl, b);
  for (int i = 0; i < batch; ++i) {  // caller-visible outputs replace their workspace twins
    const akvs_reuse_out &o = outs[i];
    BatchReq &r = b.req[i];
    if (o.probe_k) r.probe_k = o.probe_k;
    if (o.probe_v) r.probe_v = o.probe_v;
    if (o.d_k) r.d_k = o.d_k;
    if (o.d_v) r.d_v = o.d_v;
    if (o.rows) r.rows = o.rows;
  }

  const int L = m->n_layers, D = m->d_model, hkv = m->n_kv_heads, hd = m->head_dim;
  const int kvw = hkv * hd, hqw = m->n_q_heads * hd, qkvw = hqw + 2 * kvw;
  const bool no_prefix = (cfgs[0].flags & AKVS_F_NO_PREFIX_RECOMPUTE) != 0;
  const int c = no_prefix ? 0 : cfgs[0].check_layer;
  const size_t es = es_of(m->dtype);
  const int T_max = (int)pl.t_max, cap_sum = (int)pl.cap_sum, q_sum = (int)pl.q_sum;
  const int32_t *M_dev = b.row_off + batch;  // all requests' recomputed rows

  LAUNCH(AKVS_K_OTHER, launch_rope_table(0, T_max, hd, (double)m->rope_theta, b.rope, stream));
  // per request: bookkeeping, prefix layers, check layer, selection
  for (int i = 0; i < batch; ++i) {
    const Meta &mt = pl.mt[i];
    BatchReq &r = b.req[i];
    const akvs_reuse_cfg &cf = cfgs[i];
    const int T = (int)mt.t_all, Tc = (int)mt.t_ctx, nch = cf.n_chunks;
    const size_t corr_layer = (size_t)(outs[i].kv_rows ? outs[i].kv_rows : T) * kvw * es;
    char *k_corr = reinterpret_cast<char *>(outs[i].k_corr);
    char *v_corr = reinterpret_cast<char *>(outs[i].v_corr);
    LAUNCH(AKVS_K_OTHER, put_ints(mt.m.data(), mt.m.size(), r.meta, stream));
    LAUNCH(AKVS_K_OTHER, launch_token_setup(r.meta, nch, r.tok_delta, r.tok_chunk, stream));
    LAUNCH(AKVS_K_OTHER, launch_embed(tokens[i], T, embed, m->dtype, m->vocab, D, r.h_full, stream));
    for (int l = 0; l < c; ++l) {
      if (l == 0) LAUNCH(AKVS_K_OTHER, plan_full_layers(m, T, b.lb_full, stream));
      st = full_layer(m, lw[l], r.h_full, T, 0, b.rope, b.lb_full, k_corr + l * corr_layer,
                      v_corr + l * corr_layer, stream, true);
      if (st) return st;
    }
    if (!no_prefix) {
      LAUNCH(AKVS_K_NORM, launch_rmsnorm(r.h_full, D, Tc, nullptr, nullptr, lw[c].attn_norm,
                                         m->dtype, D, m->rms_eps, b.lb_full.x, m->dtype, D,
                                         stream));
      Epi e = qkv_epi(m, nullptr, b.k_chk, b.v_chk, nullptr, 0, 0, b.rope, T_max, 0);
      e.n_off = hqw;
      const char *wkv = reinterpret_cast<const char *>(lw[c].w_qkv) + (size_t)hqw * D * es;
      GEMM(b.lb_full.x, D, wkv, D, Tc, 2 * kvw, D, nullptr, m->dtype, e, stream);
      LAUNCH(AKVS_K_DIVERGENCE,
             launch_divergence(b.k_chk, b.v_chk, m->dtype, cache_layer(&caches[i], c, Tc, hkv, hd),
                               Tc, hkv, hd, r.tok_delta, b.rope, T_max, r.d_k, r.d_v, stream));
    }
    LAUNCH(AKVS_K_SELECT, launch_select(r.d_k, r.d_v, r.meta, nch, Tc, cf.query_len, cf.flags,
                                        r.probe_k, r.probe_v, r.w_k, r.w_v, r.flags, r.chunk_rows,
                                        r.rows, b.n_rows + i, r.fresh_row, stream));
  }
  // the combined row block: request i owns rows row_off[i] .. row_off[i] + n_rows[i]
  LAUNCH(AKVS_K_OTHER, launch_batch_layout(b.n_rows, batch, b.row_off, stream));
  for (int i = 0; i < batch; ++i) {
    const Meta &mt = pl.mt[i];
    const int cap = (int)mt.row_cap;
    LAUNCH(AKVS_K_OTHER, launch_gather_rows(b.req[i].h_full, (int)mt.t_all, b.req[i].rows, cap,
                                            b.n_rows + i, D, b.h_probe, stream, b.row_off + i));
    LAUNCH(AKVS_K_OTHER, launch_copy_ints_at(b.req[i].rows, cap, b.n_rows + i, b.pos,
                                             b.row_off + i, stream));
    LAUNCH(AKVS_K_OTHER, launch_attention_plan(b.req[i].rows, 0, cap, b.n_rows + i,
                                               (int)mt.t_all, m->n_q_heads, hd, m->dtype,
                                               b.lb.part_rows, b.req[i].plan_rows, stream));
    LAUNCH(AKVS_K_OTHER, launch_attention_plan(nullptr, (int)mt.t_ctx, cfgs[i].query_len,
                                               nullptr, (int)mt.t_all, m->n_q_heads, hd,
                                               m->dtype, b.lb.part_rows, b.req[i].plan_q,
                                               stream));
  }
  for (int l = c; l < L; ++l) {
    LAUNCH(AKVS_K_NORM, launch_rmsnorm(b.h_probe, D, cap_sum, M_dev, nullptr, lw[l].attn_norm,
                                       m->dtype, D, m->rms_eps, b.lb.x, m->dtype, D, stream));
    GEMM(b.lb.x, D, lw[l].w_qkv, D, cap_sum, qkvw, D, M_dev, m->dtype,
         qkv_epi(m, b.lb.q, b.k_fresh, b.v_fresh, b.pos, 0, 0, b.rope, T_max, 0), stream,
         b.lb.gpart, (int)pl.min_sum);
    const bool last = l + 1 == L;
    int q_off = 0;
    for (int i = 0; i < batch; ++i) {
      const Meta &mt = pl.mt[i];
      BatchReq &r = b.req[i];
      const akvs_reuse_cfg &cf = cfgs[i];
      const int T = (int)mt.t_all, Tc = (int)mt.t_ctx, nch = cf.n_chunks, cap = (int)mt.row_cap;
      const size_t corr_layer = (size_t)(outs[i].kv_rows ? outs[i].kv_rows : T) * kvw * es;
      CacheLayer cl = cache_layer(&caches[i], l, Tc, hkv, hd);
      LAUNCH(AKVS_K_OFFSET,
             launch_chunk_offset(b.k_fresh, b.v_fresh, m->dtype, r.fresh_row, cl, r.meta, nch,
                                 r.probe_k, r.probe_v, cf.flags, hkv, hd, b.rope, T_max, r.mu_k,
                                 r.mu_v, stream, b.row_off + i));
      void *kl = reinterpret_cast<char *>(outs[i].k_corr) + l * corr_layer;
      void *vl = reinterpret_cast<char *>(outs[i].v_corr) + l * corr_layer;
      LAUNCH(AKVS_K_CORRECTION,
             launch_correction(cl, r.mu_k, r.mu_v, r.w_k, r.w_v, r.flags, b.k_fresh, b.v_fresh,
                               r.fresh_row, r.tok_chunk, r.tok_delta, r.meta, nch, Tc, T, hkv, hd,
                               cf.flags, b.rope, T_max, kl, vl, m->dtype, stream, b.row_off + i));
      if (!last) {
        LAUNCH(AKVS_K_ATTENTION,
               launch_attention(b.lb.q, b.pos, 0, cap, b.n_rows + i, kl, vl, T, m->n_q_heads, hkv,
                                hd, m->dtype, b.lb.att, b.lb.part_o, b.lb.part_ml,
                                b.lb.part_rows, stream, b.row_off + i, r.plan_rows));
        continue;
      }
      // last layer: only the query rows (the last q of each request's rows) go on
      const int q = cf.query_len;
      char *ql = reinterpret_cast<char *>(b.q_last) + (size_t)q_off * hqw * es;
      LAUNCH(AKVS_K_OTHER, launch_copy_tail_rows(b.lb.q, (size_t)hqw * es, q, b.n_rows + i, ql,
                                                 stream, b.row_off + i));
      LAUNCH(AKVS_K_OTHER, launch_copy_tail_rows(b.h_probe, (size_t)D * 4, q, b.n_rows + i,
                                                 b.h_last + (size_t)q_off * D, stream,
                                                 b.row_off + i));
      LAUNCH(AKVS_K_ATTENTION,
             launch_attention(ql, nullptr, Tc, q, nullptr, kl, vl, T, m->n_q_heads, hkv, hd,
                              m->dtype, reinterpret_cast<char *>(b.lb.att) + (size_t)q_off * hqw * es,
                              b.lb.part_o, b.lb.part_ml, b.lb.part_rows, stream, nullptr,
                              r.plan_q));
      q_off += q;
    }
    if (!last) {
      st = out_mlp(m, lw[l], b.h_probe, cap_sum, M_dev, b.lb.att, b.lb.x, b.lb.act, b.lb.gpart,
                   stream, (int)pl.min_sum);
    } else {
      st = out_mlp(m, lw[l], b.h_last, q_sum, nullptr, b.lb.att, b.lb.x, b.lb.act, b.lb.gpart,
                   stream);
    }
    if (st) return st;
  }
  int q_off = 0;
  for (int i = 0; i < batch; ++i) {
    LAUNCH(AKVS_K_NORM, launch_rmsnorm(b.h_last + (size_t)q_off * D, D, cfgs[i].query_len, nullptr,
                                       nullptr, final_norm, m->dtype, D, m->rms_eps, outs[i].h_query,
                                       AKVS_F32, D, stream));
    if (outs[i].n_rows) LAUNCH(AKVS_K_OTHER, launch_copy_int(b.n_rows + i, outs[i].n_rows, stream));
    q_off += cfgs[i].query_len;
  }
  return AKVS_OK;
}

// ---- first decode step -----------------------------------------------------------------

struct DecodeBufs {
  float *rope, *h, *hf, *logits, *part_val, *part_o, *part_ml;
  int32_t *part_idx;
  void *x, *q, *att, *act;
  long long part_rows;
  bool one_row_attn;  // partials of the one-row attention kernel, else of the general one
};

// The one-row attention kernel covers bf16 models with hd 64 / 128 and <= 8 query heads per
// KV head; others use the general attention with one row.
static bool decode_one_row_attn(const akvs_model_cfg *m) {
  const int G = m->n_q_heads / m->n_kv_heads;
  return m->dtype == AKVS_BF16 && G >= 1 && G <= 8 && (m->head_dim == 64 || m->head_dim == 128);
}

static size_t carve_decode(void *ws, const akvs_model_cfg *m, long long n_keys, DecodeBufs &b) {
  Carver cv(ws);
  const size_t es = es_of(m->dtype);
  const int D = m->d_model, F = m->ffn_dim, hqw = m->n_q_heads * m->head_dim;
  b.rope = cv.take<float>((size_t)m->head_dim);
  b.h = cv.take<float>((size_t)D);
  b.hf = cv.take<float>((size_t)D);
  b.logits = cv.take<float>((size_t)m->vocab);
  b.part_val = cv.take<float>((size_t)gemv_blocks(m->vocab));
  b.part_idx = cv.take<int32_t>((size_t)gemv_blocks(m->vocab));
  b.x = cv.take<char>((size_t)D * es);
  b.q = cv.take<char>((size_t)hqw * es);
  b.att = cv.take<char>((size_t)hqw * es);
  b.act = cv.take<char>((size_t)F * es);
  b.one_row_attn = decode_one_row_attn(m);
  if (b.one_row_attn) {
    int chunk;
    const size_t nc = (size_t)decode_attn_chunks((int)n_keys, m->n_kv_heads, &chunk);
    b.part_o = cv.take<float>(nc * m->n_q_heads * m->head_dim);
    b.part_ml = cv.take<float>(nc * m->n_q_heads * 2);
    b.part_rows = 0;
    return cv.off;
  }
  size_t ml;
  const size_t o = attention_part_floats(m, 1, n_keys, &ml);
  b.part_o = o ? cv.take<float>(o) : nullptr;
  b.part_ml = o ? cv.take<float>(ml) : nullptr;
  b.part_rows = o ? (long long)(ml / ((size_t)m->n_q_heads * 2)) : 0;
  return cv.off;
}

static GemvEpi gemv_epi(int mode) {
  GemvEpi e{};
  e.mode = mode;
  return e;
}

// Logits and greedy token of one final-normed row (fp32 [D]).
static akvs_status lm_head_row(const akvs_model_cfg *m, const float *hf, const void *w_out,
                               float *logits, float *part_val, int32_t *part_idx,
                               int32_t *token, hipStream_t stream) {
  GemvEpi e = gemv_epi(GV_LOGITS);
  e.out_f32 = logits;
  e.part_val = part_val;
  e.part_idx = part_idx;
  LAUNCH(AKVS_K_GEMV, launch_gemv(hf, AKVS_F32, w_out, m->dtype, m->vocab, m->d_model, e, stream));
  if (token) LAUNCH(AKVS_K_OTHER, launch_pick(part_val, part_idx, gemv_blocks(m->vocab), token, stream));
  return AKVS_OK;
}

size_t akvs_decode_workspace_size(const akvs_model_cfg *m, int32_t n_past) {
  if (check_model(m) != AKVS_OK || n_past < 0) return 0;
  DecodeBufs b;
  return carve_decode(nullptr, m, (long long)n_past + 1, b);
}

akvs_status akvs_lm_head(const float *h, int32_t n_rows, const void *w_out,
                         const akvs_model_cfg *m, float *logits, int32_t *tokens, void *ws,
                         size_t ws_bytes, hipStream_t stream) {
  akvs_status st = check_model(m);
  if (st) return st;
  REQUIRE(n_rows >= 0, AKVS_EINVAL, "n_rows must be >= 0");
  REQUIRE(h && w_out && (logits || tokens), AKVS_EINVAL, "NULL argument");
  REQUIRE(aligned16(h) && aligned16(w_out) && aligned16(ws) && (!logits || aligned16(logits)),
          AKVS_EINVAL, "misaligned argument");
  DecodeBufs b;
  const size_t need = carve_decode(nullptr, m, 1, b);
  REQUIRE(ws && ws_bytes >= need, AKVS_ENOSPACE, "workspace %zu < %zu bytes", ws_bytes, need);
  carve_decode(ws, m, 1, b);
  for (int r = 0; r < n_rows; ++r) {
    float *lg = logits ? logits + (size_t)r * m->vocab : b.logits;
    st = lm_head_row(m, h + (size_t)r * m->d_model, w_out, lg, b.part_val, b.part_idx,
                     tokens ? tokens + r : nullptr, stream);
    if (st) return st;
  }
  return AKVS_OK;
}

}  // extern "C"

// The decode step over a workspace of ws_bytes bytes at ws (a caller's buffer, or the
// library's no-allocation scratch array).
static akvs_status decode_step(const int32_t *token, int32_t n_past, const void *embed,
                               const akvs_layer_w *lw, const void *final_norm, const void *w_out,
                               const akvs_model_cfg *m, void *k_cache, void *v_cache,
                               int32_t cache_rows, float *logits, int32_t *next_token, void *ws,
                               size_t ws_bytes, hipStream_t stream) {
  akvs_status st = check_model(m);
  if (st) return st;
  if ((st = check_layers(m, lw))) return st;
  REQUIRE(n_past >= 0 && cache_rows >= n_past + 1, AKVS_EINVAL,
          "need 0 <= n_past < cache_rows (n_past %d, cache_rows %d)", n_past, cache_rows);
  REQUIRE(token && embed && final_norm && k_cache && v_cache, AKVS_EINVAL, "NULL argument");
  REQUIRE(aligned16(embed) && aligned16(final_norm) && aligned16(k_cache) &&
              aligned16(v_cache) && aligned16(ws) && (!w_out || aligned16(w_out)) &&
              (!logits || aligned16(logits)),
          AKVS_EINVAL, "misaligned argument");
  DecodeBufs b;
  const size_t need = carve_decode(nullptr, m, (long long)n_past + 1, b);
  REQUIRE(ws && ws_bytes >= need, AKVS_ENOSPACE, "workspace %zu < %zu bytes", ws_bytes, need);
  carve_decode(ws, m, (long long)n_past + 1, b);
  const int D = m->d_model, F = m->ffn_dim, hkv = m->n_kv_heads, hd = m->head_dim;
  const int hqw = m->n_q_heads * hd, kvw = hkv * hd, qkvw = hqw + 2 * kvw;
  const size_t es = es_of(m->dtype);
  const size_t layer_bytes = (size_t)cache_rows * kvw * es;
  LAUNCH(AKVS_K_OTHER, launch_rope_table(n_past, 1, hd, (double)m->rope_theta, b.rope, stream));
  LAUNCH(AKVS_K_OTHER, launch_embed(token, 1, embed, m->dtype, m->vocab, D, b.h, stream));
  for (int l = 0; l < m->n_layers; ++l) {
    char *kl = reinterpret_cast<char *>(k_cache) + l * layer_bytes;
    char *vl = reinterpret_cast<char *>(v_cache) + l * layer_bytes;
    // RMSNorm is folded into the matrix-vector kernels that consume it when the row fits LDS
    const bool fold = D <= GEMV_NORM_MAX;
    if (!fold)
      LAUNCH(AKVS_K_NORM, launch_rmsnorm(b.h, D, 1, nullptr, nullptr, lw[l].attn_norm, m->dtype,
                                         D, m->rms_eps, b.x, m->dtype, D, stream));
    GemvEpi e = gemv_epi(GV_QKV);
    e.out_dtype = m->dtype;
    e.q_out = b.q;
    e.k_out = kl + (size_t)n_past * kvw * es;
    e.v_out = vl + (size_t)n_past * kvw * es;
    e.hq_w = hqw;
    e.kv_w = kvw;
    e.hd = hd;
    e.rope = reinterpret_cast<const float2 *>(b.rope);
    if (fold) {
      e.norm = lw[l].attn_norm;
      e.eps = m->rms_eps;
    }
    LAUNCH(AKVS_K_GEMV, launch_gemv(fold ? (const void *)b.h : b.x, fold ? AKVS_F32 : m->dtype,
                                    lw[l].w_qkv, m->dtype, qkvw, D, e, stream));
    if (b.one_row_attn)
      LAUNCH(AKVS_K_ATTENTION, launch_attention_decode(b.q, kl, vl, n_past + 1, m->n_q_heads, hkv,
                                                       hd, b.att, b.part_o, b.part_ml, stream));
    else
      LAUNCH(AKVS_K_ATTENTION, launch_attention(b.q, nullptr, n_past, 1, nullptr, kl, vl,
                                                n_past + 1, m->n_q_heads, hkv, hd, m->dtype,
                                                b.att, b.part_o, b.part_ml, b.part_rows, stream));
    GemvEpi r = gemv_epi(GV_RESID);
    r.out_f32 = b.h;
    LAUNCH(AKVS_K_GEMV, launch_gemv(b.att, m->dtype, lw[l].w_o, m->dtype, D, hqw, r, stream));
    if (!fold)
      LAUNCH(AKVS_K_NORM, launch_rmsnorm(b.h, D, 1, nullptr, nullptr, lw[l].mlp_norm, m->dtype,
                                         D, m->rms_eps, b.x, m->dtype, D, stream));
    GemvEpi g = gemv_epi(GV_SWIGLU);
    g.out = b.act;
    g.out_dtype = m->dtype;
    if (fold) {
      g.norm = lw[l].mlp_norm;
      g.eps = m->rms_eps;
    }
    LAUNCH(AKVS_K_GEMV, launch_gemv(fold ? (const void *)b.h : b.x, fold ? AKVS_F32 : m->dtype,
                                    lw[l].w_gate_up, m->dtype, 2 * F, D, g, stream));
    LAUNCH(AKVS_K_GEMV, launch_gemv(b.act, m->dtype, lw[l].w_down, m->dtype, D, F, r, stream));
  }
  LAUNCH(AKVS_K_NORM, launch_rmsnorm(b.h, D, 1, nullptr, nullptr, final_norm, m->dtype, D,
                                     m->rms_eps, b.hf, AKVS_F32, D, stream));
  return lm_head_row(m, b.hf, w_out ? w_out : embed, logits ? logits : b.logits, b.part_val,
                     b.part_idx, next_token, stream);
}

// ---- the no-allocation decode step --------------------------------------------------------
// A device array of fixed size serves as the decode step's workspace for callers that
// cannot allocate. Every device that runs it holds its own copy of the array (at its own
// address) until the process ends. Host code never uses the array's name as an address:
// the device address comes from hipGetSymbolAddress, looked up once per device with that
// device current, and is what the kernels receive. The decode step's kernels write every
// scratch value before they read it, so nothing needs clearing between calls.
static __device__ __align__(256) unsigned char scratch[AKVS_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
static std::mutex g_scratch_mu;
static void *g_scratch_dev[kMaxDevices];  // device address of `scratch` per device

static akvs_status scratch_address(hipStream_t stream, void **out) {
  int cur = -1;
  hipError_t e = hipGetDevice(&cur);
  if (e != hipSuccess) return fail(AKVS_EHIP, "hipGetDevice: %s", hipGetErrorString(e));
  if (stream) {
    hipDevice_t sd = -1;
    e = hipStreamGetDevice(stream, &sd);
    if (e != hipSuccess) return fail(AKVS_EHIP, "hipStreamGetDevice: %s", hipGetErrorString(e));
    REQUIRE((int)sd == cur, AKVS_EINVAL,
            "the stream belongs to device %d but device %d is current", (int)sd, cur);
  }
  REQUIRE(cur >= 0 && cur < kMaxDevices, AKVS_EUNSUPPORTED, "device index %d above %d", cur,
          kMaxDevices - 1);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_dev[cur]) {
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(AKVS_EHIP, "hipGetSymbolAddress(scratch) on device %d: %s", cur,
                  hipGetErrorString(e));
    g_scratch_dev[cur] = p;
  }
  *out = g_scratch_dev[cur];
  return AKVS_OK;
}

extern "C" {

akvs_status akvs_decode_step(const int32_t *token, int32_t n_past, const void *embed,
                             const akvs_layer_w *lw, const void *final_norm, const void *w_out,
                             const akvs_model_cfg *m, void *k_cache, void *v_cache,
                             int32_t cache_rows, float *logits, int32_t *next_token, void *ws,
                             size_t ws_bytes, hipStream_t stream) {
  return decode_step(token, n_past, embed, lw, final_norm, w_out, m, k_cache, v_cache,
                     cache_rows, logits, next_token, ws, ws_bytes, stream);
}

akvs_status akvs_decode_step_noalloc(const int32_t *token, int32_t n_past, const void *embed,
                                     const akvs_layer_w *lw, const void *final_norm,
                                     const void *w_out, const akvs_model_cfg *m, void *k_cache,
                                     void *v_cache, int32_t cache_rows, float *logits,
                                     int32_t *next_token, hipStream_t stream) {
  akvs_status st = check_model(m);
  if (st) return st;
  REQUIRE(n_past >= 0, AKVS_EINVAL, "n_past must be >= 0");
  const size_t need = akvs_decode_workspace_size(m, n_past);
  REQUIRE(need > 0 && need <= AKVS_NOALLOC_SCRATCH_BYTES, AKVS_ENOSPACE,
          "the decode step needs %zu bytes of scratch with n_past %d; the no-allocation entry "
          "point holds %zu (use akvs_decode_step with a workspace)",
          need, n_past, (size_t)AKVS_NOALLOC_SCRATCH_BYTES);
  void *ws = nullptr;
  if ((st = scratch_address(stream, &ws))) return st;
  return decode_step(token, n_past, embed, lw, final_norm, w_out, m, k_cache, v_cache,
                     cache_rows, logits, next_token, ws, AKVS_NOALLOC_SCRATCH_BYTES, stream);
}

}  // extern "C"
