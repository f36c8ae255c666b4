// Host runtime behind include/rollplex.h: validation, workspace carving and the
// per-layer launch sequence of the prefix pass, the suffix pass and the decode step.
// Every compute entry point validates all host-visible arguments before its first HIP
// call, then only enqueues kernels on the caller's stream (no allocation, no sync).
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <string>
#include <vector>

#include <hip/hip_ext.h>

#include "rp_internal.h"

struct rp_model {
  rp_config cfg;
  const void* embed;
  const void* final_norm;
  const void* lm_head;
  std::vector<rp_layer_weights> layers;
  rp::RopeFreq rope;
};

namespace {

thread_local std::string g_err;

rp_status fail(rp_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return s;
}

bool fault_injected() {
  const char* e = getenv("RP_FAULT_INJECT");
  return e && *e && strcmp(e, "0") != 0;
}

// ---- per-launch event timing (rp_profile_*) ----
struct Profiler {
  bool on = false;
  std::vector<hipEvent_t> ev;        // 2 per bracketed launch
  std::vector<const char*> pending;  // kernel name per bracketed launch
  std::vector<std::string> names;
  std::vector<int64_t> count;
  std::vector<double> ms;
};
Profiler g_prof;

bool prof_begin(hipStream_t s, const char* name, int* slot) {
  *slot = -1;
  if (!g_prof.on) return true;
  const size_t k = g_prof.pending.size();
  if (2 * k + 1 >= g_prof.ev.size()) return true;
  if (hipEventRecord(g_prof.ev[2 * k], s) != hipSuccess) return false;
  g_prof.pending.push_back(name);
  *slot = (int)k;
  return true;
}

bool prof_end(hipStream_t s, int slot) {
  if (slot < 0) return true;
  return hipEventRecord(g_prof.ev[2 * slot + 1], s) == hipSuccess;
}

// Launch `expr` (a launcher returning hipError_t) on stream `s`, timing it when profiling.
#define RP_TRY_LAUNCH_N(name, expr)                                                             \
  do {                                                                                          \
    if (fault_injected()) return fail(RP_ERR_HIP, "injected launch fault (RP_FAULT_INJECT)");   \
    int slot_;                                                                                  \
    if (!prof_begin(s, name, &slot_)) return fail(RP_ERR_HIP, "profiling event record failed"); \
    hipError_t e_ = (expr);                                                                     \
    if (e_ != hipSuccess) return fail(RP_ERR_HIP, "%s failed: %s", name, hipGetErrorString(e_)); \
    if (!prof_end(s, slot_)) return fail(RP_ERR_HIP, "profiling event record failed");          \
  } while (0)

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

size_t elem_size(const rp_config& c) { return c.dtype == RP_F32 ? 4 : 2; }
bool half_dtype(const rp_config& c) { return c.dtype == RP_BF16 || c.dtype == RP_F16; }

// RP_DEBUG (environment, read once): guard bytes after every workspace slice, checked
// after the pass, and range checks of the device-side ids; each checked call then
// synchronises its stream and reports what it found.  Workspace sizes include the guards.
bool debug_mode() {
  static const bool on = [] {
    const char* e = getenv("RP_DEBUG");
    return e && *e && strcmp(e, "0") != 0;
  }();
  return on;
}

// Guard offsets of the last carve into a real workspace (this thread).
thread_local std::vector<uint64_t> g_last_guards;

// Bump allocator over the caller's workspace (sizing pass when base == nullptr).
struct Carver {
  char* base;
  size_t off = 0;
  explicit Carver(void* b) : base((char*)b) {
    if (base) g_last_guards.clear();
  }
  void* take(size_t bytes) {
    off = (off + 255) & ~(size_t)255;
    void* p = base ? base + off : nullptr;
    off += bytes;
    if (debug_mode()) {
      off = (off + 255) & ~(size_t)255;
      if (base) g_last_guards.push_back(off);
      off += rp::kGuardBytes;
    }
    return p;
  }
};

struct LayerWS {
  float* X;   // fp32 residual [M, d]
  void* N;    // normed activations [M, d]
  float* QKV;  // fp32 projections [M, qkv]
  void* Q;     // rotated queries [M, Hq*D]
  void* O;    // attention output [M, Hq*D]
  void* GU;   // [M, 2F]
  void* ACT;  // [M, F]
  float* attn_part = nullptr;  // split-KV attention partials (suffix pass, 16-bit models)
};

// bf16 prefix/suffix layers fuse SwiGLU into the gate/up GEMM and need no [M, 2F] buffer.

void carve_layer(Carver& c, const rp_config& cfg, int64_t M, bool need_x, bool need_gu, LayerWS* w) {
  const size_t es = elem_size(cfg);
  const int64_t d = cfg.d_model, qkv = (int64_t)(cfg.n_q_heads + 2 * cfg.n_kv_heads) * cfg.head_dim;
  w->X = need_x ? (float*)c.take(M * d * 4) : nullptr;
  w->N = c.take(M * d * es);
  w->QKV = (float*)c.take(M * qkv * 4);
  w->Q = c.take(M * (int64_t)cfg.n_q_heads * cfg.head_dim * es);
  w->O = c.take(M * (int64_t)cfg.n_q_heads * cfg.head_dim * es);
  w->GU = need_gu ? c.take(M * 2 * (int64_t)cfg.ffn_dim * es) : nullptr;
  w->ACT = c.take(M * (int64_t)cfg.ffn_dim * es);
}

rp_status check_config(const rp_config* c) {
  if (!c) return fail(RP_ERR_INVALID_ARG, "config is NULL");
  // The caller may store any integer in the enum field; reading it as rp_dtype before
  // it is known to be one of the enumerators is undefined in C++, so read its bytes.
  int dtype_value = 0;
  memcpy(&dtype_value, &c->dtype, sizeof dtype_value);
  if (dtype_value != RP_F32 && dtype_value != RP_BF16 && dtype_value != RP_F16)
    return fail(RP_ERR_INVALID_ARG, "bad dtype %d", dtype_value);
  if (c->weight_layout & ~RP_WEIGHT_LAYOUTS)
    return fail(RP_ERR_INVALID_ARG, "unknown weight_layout bits 0x%x", c->weight_layout);
  if (c->n_layers < 1 || c->d_model < 1 || c->n_q_heads < 1 || c->n_kv_heads < 1 || c->ffn_dim < 1 ||
      c->vocab < 1 || c->max_position < 1)
    return fail(RP_ERR_SHAPE, "config sizes must be positive");
  if (c->n_q_heads % c->n_kv_heads != 0)
    return fail(RP_ERR_SHAPE, "n_q_heads %d not a multiple of n_kv_heads %d", c->n_q_heads, c->n_kv_heads);
  if (c->n_q_heads / c->n_kv_heads > 8)
    return fail(RP_ERR_UNSUPPORTED, "query group size %d > 8", c->n_q_heads / c->n_kv_heads);
  if (c->head_dim != 64 && c->head_dim != 128)
    return fail(RP_ERR_UNSUPPORTED, "head_dim %d (supported: 64, 128)", c->head_dim);
  if (c->d_model % 8 || c->ffn_dim % 8) return fail(RP_ERR_UNSUPPORTED, "d_model and ffn_dim must be multiples of 8");
  if (c->dtype != RP_F32 && (c->d_model % 64 || c->ffn_dim % 64 || (c->n_q_heads * c->head_dim) % 64))
    return fail(RP_ERR_UNSUPPORTED, "16-bit dtypes need d_model, ffn_dim and n_q_heads*head_dim multiples of 64");
  if (!(c->rms_eps > 0.f) || !(c->rope_theta > 0.0)) return fail(RP_ERR_SHAPE, "rms_eps and rope_theta must be > 0");
  const int64_t qkv = (int64_t)(c->n_q_heads + 2 * c->n_kv_heads) * c->head_dim;
  if (qkv > (1 << 30) || (int64_t)c->ffn_dim * 2 > (1 << 30)) return fail(RP_ERR_UNSUPPORTED, "dimension too large");
  return RP_OK;
}

rp_status check_prefix_cu(const rp_model* m, int32_t B, const int32_t* cu, const char* what) {
  if (B < 1 || B > RP_MAX_SEQS) return fail(RP_ERR_SHAPE, "%s: batch %d outside [1, %d]", what, B, RP_MAX_SEQS);
  if (!cu) return fail(RP_ERR_INVALID_ARG, "%s: cu_seqlens is NULL", what);
  if (cu[0] != 0) return fail(RP_ERR_SHAPE, "%s: cu_seqlens[0] = %d, must be 0", what, cu[0]);
  for (int b = 0; b < B; ++b) {
    if (cu[b + 1] <= cu[b])
      return fail(RP_ERR_SHAPE, "%s: sequence %d has length %d (prefixes need >= 1 token)", what, b,
                  cu[b + 1] - cu[b]);
    if (cu[b + 1] - cu[b] > m->cfg.max_position)
      return fail(RP_ERR_SHAPE, "%s: sequence %d length %d exceeds max_position %d", what, b, cu[b + 1] - cu[b],
                  m->cfg.max_position);
  }
  return RP_OK;
}

rp_status check_suffix_cu(const rp_model* m, int32_t B, const int32_t* pcu, const int32_t* scu) {
  rp_status s = check_prefix_cu(m, B, pcu, "prefix_cu");
  if (s != RP_OK) return s;
  if (!scu) return fail(RP_ERR_INVALID_ARG, "suffix_cu is NULL");
  if (scu[0] != 0) return fail(RP_ERR_SHAPE, "suffix_cu[0] = %d, must be 0", scu[0]);
  for (int b = 0; b < B; ++b) {
    const int S = scu[b + 1] - scu[b];
    if (S < 0) return fail(RP_ERR_SHAPE, "suffix sequence %d has negative length %d", b, S);
    const int64_t last = (int64_t)(pcu[b + 1] - pcu[b]) + S;
    if (last > m->cfg.max_position)
      return fail(RP_ERR_SHAPE, "sequence %d: prefix + suffix = %lld exceeds max_position %d", b, (long long)last,
                  m->cfg.max_position);
  }
  return RP_OK;
}

// Shared-prefix suffixes: n_suffix sequences, sequence s scores against prefix
// prefix_of_suffix[s] of the n_prefix prefixes.
rp_status check_grouped_cu(const rp_model* m, int32_t n_prefix, const int32_t* pcu, int32_t n_suffix,
                           const int32_t* grp, const int32_t* scu, const int32_t* rope0 = nullptr) {
  rp_status st = check_prefix_cu(m, n_prefix, pcu, "prefix_cu");
  if (st != RP_OK) return st;
  if (n_suffix < 1 || n_suffix > RP_MAX_SEQS)
    return fail(RP_ERR_SHAPE, "suffix count %d outside [1, %d]", n_suffix, RP_MAX_SEQS);
  if (!grp || !scu) return fail(RP_ERR_INVALID_ARG, "prefix_of_suffix and suffix_cu are required");
  if (scu[0] != 0) return fail(RP_ERR_SHAPE, "suffix_cu[0] must be 0");
  for (int s = 0; s < n_suffix; ++s) {
    if (grp[s] < 0 || grp[s] >= n_prefix)
      return fail(RP_ERR_SHAPE, "prefix_of_suffix[%d] = %d outside [0, %d)", s, grp[s], n_prefix);
    const int64_t S = (int64_t)scu[s + 1] - scu[s];
    if (S < 0) return fail(RP_ERR_SHAPE, "suffix sequence %d has negative length %lld", s, (long long)S);
    const int64_t last = (int64_t)(pcu[grp[s] + 1] - pcu[grp[s]]) + S;
    if (last > m->cfg.max_position)
      return fail(RP_ERR_SHAPE, "suffix %d: prefix + suffix = %lld exceeds max_position %d", s, (long long)last,
                  m->cfg.max_position);
    if (rope0) {
      const int64_t r = (int64_t)rope0[grp[s]];
      if (r < 0 || r + S > m->cfg.max_position)
        return fail(RP_ERR_SHAPE, "suffix %d: rotary positions %lld .. %lld outside [0, max_position %d)", s,
                    (long long)r, (long long)(r + S - 1), m->cfg.max_position);
    }
  }
  return RP_OK;
}

// Sequence table: query rows q_cu[0..B]; the key segment of sequence b is prefix grp[b]
// (b when grp is NULL) of the n_k prefixes k_cu[0..n_k] (none when k_cu is NULL).  The
// first query row after prefix p rotates by position rope0[p] (default: its length).
rp::SeqTable make_table(int32_t B, const int32_t* q_cu, int32_t n_k, const int32_t* k_cu, const int32_t* grp,
                        const int32_t* rope0 = nullptr) {
  rp::SeqTable t;
  memset(&t, 0, sizeof t);
  t.n = B;
  for (int b = 0; b <= B; ++b) t.q_cu[b] = q_cu[b];
  for (int p = 0; p <= n_k && k_cu; ++p) t.k_cu[p] = k_cu[p];
  for (int p = 0; p < n_k && k_cu; ++p) t.rope0[p] = rope0 ? rope0[p] : k_cu[p + 1] - k_cu[p];
  for (int b = 0; b < B; ++b) t.grp[b] = (uint8_t)(grp ? grp[b] : b);
  return t;
}

// split-K factor for small-M GEMMs (decode): up to 64 rows the skinny kernel's (about
// four waves per CU); beyond, >= 2 workgroups of 256x256 tiles per CU.
int decode_splitk(const rp_config& cfg, int32_t M, int32_t N, int32_t K) {
  if (!half_dtype(cfg)) return 1;
  if (M <= 64 && K % 64 == 0) return rp::gemm_skinny_splitk(M, N, K);
  const int tiles = ((M + 255) / 256) * ((N + 255) / 256);
  int s = (512 + tiles - 1) / tiles;
  s = s < 1 ? 1 : s;
  s = s > 16 ? 16 : s;
  const int kb = K / 64;
  return s > kb ? kb : s;
}

// Split-K plan of one decoder layer's GEMMs.
//   prefix: no split (the prefix holds many rows; results are bitwise independent of how
//           sequences are packed);
//   suffix: GEMMs with fewer than 16384 output columns split K into min(8, K/1024) chunks,
//           a factor that depends on the shapes of the weights only, so a row's result
//           does not depend on how many other rows share the launch;
//   decode: split to fill the chip for the batch at hand (decode_splitk).
// Split GEMMs cannot fuse SwiGLU into their epilogue.
enum class Pass { kPrefix, kSuffix, kDecode };
struct LayerPlan {
  int qkv = 1, o = 1, gu = 1, down = 1;
  bool fused = false;
  size_t part_floats = 0;
};
int suffix_splitk(const rp_config& cfg, int32_t N, int32_t K) {
  if (!half_dtype(cfg) || N >= 16384) return 1;
  int s = K / 1024;
  return s < 1 ? 1 : s > 8 ? 8 : s;
}
LayerPlan plan_layer(const rp_config& c, int32_t M, Pass pass) {
  const int d = c.d_model, F = c.ffn_dim, qkv = (c.n_q_heads + 2 * c.n_kv_heads) * c.head_dim;
  const int hq = c.n_q_heads * c.head_dim;
  auto f = [&](int N, int K) {
    return pass == Pass::kPrefix ? 1 : pass == Pass::kSuffix ? suffix_splitk(c, N, K) : decode_splitk(c, M, N, K);
  };
  LayerPlan p;
  p.qkv = f(qkv, d);
  p.o = f(d, hq);
  p.gu = f(2 * F, d);
  p.down = f(d, F);
  p.fused = half_dtype(c) && p.gu == 1;
  const int64_t shapes[4][3] = {{qkv, p.qkv, 0}, {d, p.o, 0}, {2 * F, p.gu, 0}, {d, p.down, 0}};
  for (auto& sh : shapes) {
    const size_t fl = rp::gemm_partial_floats(M, (int32_t)sh[0], (int32_t)sh[1]);
    p.part_floats = fl > p.part_floats ? fl : p.part_floats;
  }
  return p;
}

// Buffers of the last layer's last-row tail (RP_PREFIX_LAST_ROWS_ONLY), B rows each.
struct TailWS {
  float* Qf;    // [B, Hq*D] fp32 query projections of the last rows
  void* Q;      // [B, Hq*D] rotated queries of the last rows
  void* K;      // [B, Hkv*D] their keys and values
  void* V;
  void* O;      // [B, Hq*D] attention output
  void* N;      // [B, d] normed activations
  void* GU;     // [B, 2F] (unfused gate/up)
  void* ACT;    // [B, F]
  float* part;  // split-K partials
  LayerPlan plan;
};

size_t prefix_ws(const rp_model* m, int32_t B, int64_t T, void* base, bool need_x, LayerWS* w, int32_t** vis_idx,
                 TailWS* tail = nullptr, float2** rope_cs = nullptr) {
  Carver c(base);
  int32_t* vi = (int32_t*)c.take(T * 4);
  if (vis_idx) *vis_idx = vi;
  // rotation table of the fused q/k/v epilogue (16-bit models): float2 [T][D/2]
  float2* cs = half_dtype(m->cfg) ? (float2*)c.take(T * (m->cfg.head_dim / 2) * 8) : nullptr;
  if (rope_cs) *rope_cs = cs;
  LayerWS tmp;
  carve_layer(c, m->cfg, T, need_x, !plan_layer(m->cfg, (int32_t)T, Pass::kPrefix).fused, w ? w : &tmp);
  const rp_config& cf = m->cfg;
  const size_t es = elem_size(cf);
  const int64_t hq = (int64_t)cf.n_q_heads * cf.head_dim, kvr = (int64_t)cf.n_kv_heads * cf.head_dim;
  TailWS tt;
  TailWS* t = tail ? tail : &tt;
  t->plan = plan_layer(cf, B, Pass::kDecode);
  const size_t qpart = rp::gemm_partial_floats(B, (int32_t)hq, decode_splitk(cf, B, (int32_t)hq, cf.d_model));
  if (qpart > t->plan.part_floats) t->plan.part_floats = qpart;
  t->Qf = (float*)c.take(B * hq * 4);
  t->Q = c.take(B * hq * es);
  t->K = c.take(B * kvr * es);
  t->V = c.take(B * kvr * es);
  t->O = c.take(B * hq * es);
  t->N = c.take(B * (int64_t)cf.d_model * es);
  t->GU = t->plan.fused ? nullptr : c.take(B * 2 * (int64_t)cf.ffn_dim * es);
  t->ACT = c.take(B * (int64_t)cf.ffn_dim * es);
  t->part = (float*)c.take(t->plan.part_floats * 4);
  return c.off + 256;
}

struct SuffixWS {
  LayerWS L;
  void* Ks;
  void* Vs;
  float* logits;     // [R, V] fp32 (unfused scoring)
  float* lse;        // [R, n_part] float2 and
  float* tgt;        // [R] (fused scoring: RP_SUFFIX_FUSED_LOGPROB)
  float* gemm_part;
  LayerPlan plan;
};

// The fused lm_head needs 16-bit MFMA; an fp32 model always scores unfused.
bool fused_scoring(const rp_model* m, uint32_t flags) {
  return (flags & RP_SUFFIX_FUSED_LOGPROB) && half_dtype(m->cfg);
}

// Split-KV ways of the suffix attention over prefixes 0 .. n_prefix-1 (the most split).
int32_t suffix_attn_splits(const rp_model* m, int32_t n_prefix, const int32_t* pcu) {
  if (!half_dtype(m->cfg)) return 1;
  int32_t S = 1;
  for (int p = 0; p < n_prefix; ++p) S = std::max(S, (int32_t)rp::attn_splits(pcu[p + 1] - pcu[p]));
  return S;
}

size_t suffix_ws(const rp_model* m, int64_t R, uint32_t flags, int32_t splits, void* base, SuffixWS* w) {
  Carver c(base);
  SuffixWS tmp;
  SuffixWS* s = w ? w : &tmp;
  s->plan = plan_layer(m->cfg, (int32_t)R, Pass::kSuffix);
  carve_layer(c, m->cfg, R, true, !s->plan.fused, &s->L);
  const size_t np = rp::attn_partial_floats(R, m->cfg.n_q_heads, m->cfg.head_dim, splits);
  s->L.attn_part = np ? (float*)c.take(np * 4) : nullptr;
  const int64_t kvrow = (int64_t)m->cfg.n_kv_heads * m->cfg.head_dim;
  s->Ks = c.take(R * kvrow * elem_size(m->cfg));
  s->Vs = c.take(R * kvrow * elem_size(m->cfg));
  s->logits = s->lse = s->tgt = nullptr;
  if (fused_scoring(m, flags)) {
    s->lse = (float*)c.take(R * (int64_t)rp::lse_parts(m->cfg.vocab) * 8);
    s->tgt = (float*)c.take(R * 4);
  } else {
    s->logits = (float*)c.take(R * (int64_t)m->cfg.vocab * 4);
  }
  s->gemm_part = (float*)c.take(s->plan.part_floats * 4);
  return c.off + 256;
}

struct PromptWS {
  void* N;        // [n, d] final-norm rows
  int32_t* tid;   // [n] scored token id, -1 for an invalid position
  float* logits;  // [n, V] fp32 (unfused scoring)
  float* lse;     // [n, n_part] float2 and
  float* tgt;     // [n] (fused scoring)
};

size_t prompt_ws(const rp_model* m, int64_t n, uint32_t flags, void* base, PromptWS* w) {
  Carver c(base);
  PromptWS tmp;
  PromptWS* p = w ? w : &tmp;
  p->N = c.take(n * m->cfg.d_model * elem_size(m->cfg));
  p->tid = (int32_t*)c.take(n * 4);
  p->logits = p->lse = p->tgt = nullptr;
  if (fused_scoring(m, flags)) {
    p->lse = (float*)c.take(n * (int64_t)rp::lse_parts(m->cfg.vocab) * 8);
    p->tgt = (float*)c.take(n * 4);
  } else {
    p->logits = (float*)c.take(n * (int64_t)m->cfg.vocab * 4);
  }
  return c.off + 256;
}

struct DecodeWS {
  LayerWS L;
  float* logits;
  float* attn_part;
  float* gemm_part;
  rp::ArgmaxPart* arg_part;  // per-wave row candidates of the fused lm_head + argmax
};

// When the caller wants no logits, the lm_head of a 16-bit model with at most 64 rows
// reduces each row to its argmax in the GEMM (the [B, V] logits are never stored).
bool decode_fused_argmax(const rp_model* m, int32_t B) {
  const rp_config& c = m->cfg;
  return rp::gemm_argmax_supported(c.dtype, B, c.vocab, c.d_model, c.d_model, c.d_model);
}

// own_logits: carve the [B, V] logits too (they go to the workspace when the caller
// passes none and the argmax is not fused).
size_t decode_ws(const rp_model* m, int32_t B, int32_t cap, void* base, DecodeWS* w, bool own_logits = true) {
  Carver c(base);
  DecodeWS tmp;
  DecodeWS* s = w ? w : &tmp;
  const rp_config& cfg = m->cfg;
  carve_layer(c, cfg, B, true, true, &s->L);
  s->logits = own_logits ? (float*)c.take((int64_t)B * cfg.vocab * 4) : nullptr;
  s->arg_part = decode_fused_argmax(m, B)
                    ? (rp::ArgmaxPart*)c.take(rp::gemm_argmax_parts(B, cfg.vocab) * sizeof(rp::ArgmaxPart))
                    : nullptr;
  s->attn_part = (float*)c.take(rp::decode_attn_partial_floats(B, cfg.n_q_heads, cfg.head_dim, cap) * 4);
  const int64_t d = cfg.d_model, F = cfg.ffn_dim, qkv = (int64_t)(cfg.n_q_heads + 2 * cfg.n_kv_heads) * cfg.head_dim;
  const int64_t hq = (int64_t)cfg.n_q_heads * cfg.head_dim;
  // the layer GEMMs write split-K partials (one split included) that the next kernel sums
  size_t need = 0;
  const int64_t shapes[4][2] = {{qkv, d}, {d, hq}, {2 * F, d}, {d, F}};
  for (auto& sh : shapes) {
    const int32_t sk = rp::gemm_effective_splitk(cfg.dtype, (int32_t)sh[1],
                                                 decode_splitk(cfg, B, (int32_t)sh[0], (int32_t)sh[1]));
    const size_t f = (size_t)sk * B * sh[0];
    need = f > need ? f : need;
  }
  const size_t lm = rp::gemm_partial_floats(B, cfg.vocab, decode_splitk(cfg, B, cfg.vocab, (int32_t)d));
  need = lm > need ? lm : need;
  s->gemm_part = (float*)c.take(need * 4);
  return c.off + 256;
}

rp_status check_kv(const rp_model* m, const rp_kv& kv, int64_t rows, const char* what) {
  if (!kv.k || !kv.v) return fail(RP_ERR_INVALID_ARG, "%s: k or v is NULL", what);
  const int64_t per = rows * m->cfg.n_kv_heads * m->cfg.head_dim;
  if (kv.layer_stride < per)
    return fail(RP_ERR_SHAPE, "%s: layer_stride %lld < %lld elements", what, (long long)kv.layer_stride, (long long)per);
  if (!aligned16(kv.k) || !aligned16(kv.v) || (kv.layer_stride % 8))
    return fail(RP_ERR_INVALID_ARG, "%s: KV must be 16-byte aligned (layer_stride multiple of 8)", what);
  return RP_OK;
}

rp_status check_ws(void* ws, size_t have, size_t need) {
  if (have < need) return fail(RP_ERR_WORKSPACE, "workspace %zu bytes < required %zu", have, need);
  if (need && !ws) return fail(RP_ERR_INVALID_ARG, "workspace is NULL");
  if (((uintptr_t)ws & 255u) != 0) return fail(RP_ERR_INVALID_ARG, "workspace must be 256-byte aligned");
  return RP_OK;
}

// Device record of the debug checks: one copy per GPU (file-scope device array; its
// address on the current device comes from hipGetSymbolAddress, taken once per device).
static __device__ int debug_record[4];
std::mutex g_debug_mu;
int* g_debug_addr[64] = {};

rp_status debug_record_addr(int** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(RP_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= 64) return fail(RP_ERR_UNSUPPORTED, "device %d outside [0, 64)", dev);
  std::lock_guard<std::mutex> lock(g_debug_mu);
  if (!g_debug_addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(debug_record));
    if (e != hipSuccess || !p) return fail(RP_ERR_HIP, "hipGetSymbolAddress(debug_record): %s", hipGetErrorString(e));
    g_debug_addr[dev] = (int*)p;
  }
  *out = g_debug_addr[dev];
  return RP_OK;
}

// The checks of one call in debug mode (no-ops otherwise): begin() after the workspace is
// carved fills its guards; check_ids() queues a range check; end() checks the guards,
// synchronises the stream and turns the first recorded problem into the call's status.
struct DebugPass {
  bool on = false;
  hipStream_t s = nullptr;
  uint8_t* ws = nullptr;
  rp::GuardTable gt{};
  int* rec = nullptr;
  struct Check {
    const char* what;
    int lo, hi;
  };
  std::vector<Check> checks;

  rp_status begin(hipStream_t stream, void* workspace) {
    on = debug_mode();
    if (!on) return RP_OK;
    s = stream;
    ws = (uint8_t*)workspace;
    gt.n = 0;
    for (size_t i = 0; i < g_last_guards.size() && gt.n < rp::kMaxGuards; ++i) gt.off[gt.n++] = g_last_guards[i];
    if (!ws) gt.n = 0;
    rp_status st = debug_record_addr(&rec);
    if (st != RP_OK) return st;
    hipError_t e = rp::launch_debug_reset(s, rec);
    if (e == hipSuccess) e = rp::launch_guard_fill(s, ws, gt);
    return e == hipSuccess ? RP_OK : fail(RP_ERR_HIP, "RP_DEBUG set-up: %s", hipGetErrorString(e));
  }
  rp_status check_ids(const int32_t* v, int32_t n, int32_t lo, int32_t hi, const char* what, int code) {
    if (!on) return RP_OK;
    checks.push_back(Check{what, lo, hi});
    const hipError_t e = rp::launch_check_range(s, v, n, lo, hi, code + 16 * (int)(checks.size() - 1), rec);
    return e == hipSuccess ? RP_OK : fail(RP_ERR_HIP, "RP_DEBUG check: %s", hipGetErrorString(e));
  }
  rp_status end(rp_status st) {
    if (!on || st != RP_OK) return st;
    hipError_t e = hipSuccess;
    const char* corrupt = getenv("RP_DEBUG_CORRUPT_GUARD");  // self-test: a forced overflow
    if (corrupt && *corrupt && strcmp(corrupt, "0") != 0) e = rp::launch_guard_corrupt(s, ws, gt);
    if (e == hipSuccess) e = rp::launch_guard_check(s, ws, gt, rec);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    int h[4] = {0, 0, 0, 0};
    if (e == hipSuccess) e = hipMemcpy(h, rec, sizeof h, hipMemcpyDeviceToHost);
    if (e != hipSuccess) return fail(RP_ERR_HIP, "RP_DEBUG check: %s", hipGetErrorString(e));
    if (h[0] == 0) return RP_OK;
    if (h[0] == rp::DBG_GUARD)
      return fail(RP_ERR_HIP, "RP_DEBUG: workspace guard %d (after slice %d) was overwritten", h[1], h[1]);
    const int idx = h[0] / 16, code = h[0] % 16;
    const Check c = idx < (int)checks.size() ? checks[idx] : Check{"value", 0, 0};
    return fail(code == rp::DBG_KV_LEN ? RP_ERR_SHAPE : RP_ERR_INVALID_ARG,
                "RP_DEBUG: %s[%d] = %d outside [%d, %d)", c.what, h[1], h[2], c.lo, c.hi);
  }
};

void* layer_ptr(const rp_model* m, void* base, int64_t stride, int l) {
  return (char*)base + (size_t)l * stride * elem_size(m->cfg);
}

// One decoder layer over M rows; keys/values go to k_out/v_out (rows aligned with
// the query rows); attention reads segment 0 from k0/v0 as described by st.
// Kernel names reported by the per-launch timer, per pass.
struct LayerNames {
  const char *norm1, *qkv, *rope, *attn, *oproj, *norm2, *gate_up, *swiglu, *down;
};
const LayerNames kPrefixNames = {"prefix.rmsnorm", "prefix.gemm_qkv", "prefix.rope_kv", "prefix.attention",
                                 "prefix.gemm_o_proj", "prefix.rmsnorm", "prefix.gemm_gate_up", "prefix.swiglu",
                                 "prefix.gemm_down"};
const LayerNames kSuffixNames = {"suffix.rmsnorm", "suffix.gemm_qkv", "suffix.rope_kv", "suffix.attention",
                                 "suffix.gemm_o_proj", "suffix.rmsnorm", "suffix.gemm_gate_up", "suffix.swiglu",
                                 "suffix.gemm_down"};

// B operands of the row-parallel projections in their stored layout (weight_layout).
rp::BSeg wo_operand(const rp_config& c, const rp_layer_weights& lw) {
  return rp::BSeg{lw.wo, lw.wo, lw.wo, c.d_model, c.d_model, (c.weight_layout & RP_WO_TRANSPOSED) != 0};
}
rp::BSeg w_down_operand(const rp_config& c, const rp_layer_weights& lw) {
  return rp::BSeg{lw.w_down, lw.w_down, lw.w_down, c.d_model, c.d_model, (c.weight_layout & RP_W_DOWN_TRANSPOSED) != 0};
}

rp_status run_layer(const rp_model* m, hipStream_t s, const rp_layer_weights& lw, const rp::SeqTable& st,
                    int32_t M, const LayerWS& w, void* k_out, void* v_out, const void* k0, const void* v0,
                    const LayerPlan& plan, float* gemm_part, const LayerNames& nm,
                    const rp::MRope& mr = rp::MRope{nullptr, 0, 0}, bool norm1_done = false,
                    const void* next_norm = nullptr, bool* next_normed = nullptr,
                    const float2* rope_cs = nullptr) {
  const rp_config& c = m->cfg;
  const rp_dtype dt = c.dtype;
  const int d = c.d_model, Hq = c.n_q_heads, Hkv = c.n_kv_heads, D = c.head_dim, F = c.ffn_dim;
  const int qkv = (Hq + 2 * Hkv) * D, hq = Hq * D;
  // Split-K partials of the q/k/v, o-proj, gate/up and down projections are summed by the
  // kernel that consumes them (RoPE, residual add + RMSNorm, SwiGLU), not by a separate
  // reduction; the
  // down projection's consumer applies the next layer's attention norm (next_norm), which
  // that layer then skips (norm1_done).
  const int s_o = gemm_part ? rp::gemm_effective_splitk(dt, hq, plan.o) : 1;
  const int s_gu = gemm_part ? rp::gemm_effective_splitk(dt, d, plan.gu) : 1;
  const int s_down = gemm_part ? rp::gemm_effective_splitk(dt, F, plan.down) : 1;
  if (next_normed) *next_normed = next_norm != nullptr && s_down > 1;
  if (!norm1_done) RP_TRY_LAUNCH_N(nm.norm1, rp::launch_rmsnorm(s, dt, w.X, lw.attn_norm, c.rms_eps, M, d, w.N));
  rp::BSeg bqkv = {lw.wq, lw.wk, lw.wv, hq, hq + Hkv * D};
  const int s_qkv = gemm_part ? rp::gemm_effective_splitk(dt, d, plan.qkv) : 1;
  if (rope_cs && s_qkv == 1 && half_dtype(c)) {
    // bias, RoPE and the Q/K/V stores in the projection's epilogue (rotation table
    // rope_cs built once per pass for these rows and positions)
    const rp::RopeOut ro = {w.Q, k_out, v_out, lw.bq, lw.bk, lw.bv, rope_cs, hq, Hkv * D, D};
    RP_TRY_LAUNCH_N(nm.qkv, rp::launch_gemm(s, dt, M, qkv, d, w.N, d, bqkv, d, nullptr, qkv, rp::EPI_ROPE, 1, nullptr,
                                            nullptr, &ro));
  } else if (s_qkv > 1 && !mr.pos && (size_t)qkv * sizeof(float) <= 65536) {
    RP_TRY_LAUNCH_N(nm.qkv, rp::launch_gemm(s, dt, M, qkv, d, w.N, d, bqkv, d, nullptr, qkv, rp::EPI_PARTIALS, plan.qkv,
                                            gemm_part));
    RP_TRY_LAUNCH_N(nm.rope, rp::launch_rope_kv_splitk(s, dt, st, gemm_part, s_qkv, M, Hq, Hkv, D, lw.bq, lw.bk, lw.bv,
                                                       m->rope, c.max_position, w.Q, k_out, v_out));
  } else {
    RP_TRY_LAUNCH_N(nm.qkv, rp::launch_gemm(s, dt, M, qkv, d, w.N, d, bqkv, d, w.QKV, qkv, rp::EPI_STORE_F32, plan.qkv,
                                            gemm_part));
    RP_TRY_LAUNCH_N(nm.rope, rp::launch_rope_kv(s, dt, st, w.QKV, M, Hq, Hkv, D, lw.bq, lw.bk, lw.bv, m->rope,
                                                c.max_position, w.Q, k_out, v_out, mr));
  }
  rp::AttnArgs a;
  a.q = w.Q;
  a.q_ld = hq;
  a.k0 = k0;
  a.v0 = v0;
  a.k1 = k_out;
  a.v1 = v_out;
  a.o = w.O;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.D = D;
  a.scale = (float)(1.0 / sqrt((double)D));
  a.part = w.attn_part;
  RP_TRY_LAUNCH_N(nm.attn, rp::launch_attention(s, dt, st, a, M));
  const rp::BSeg bo = wo_operand(c, lw);
  if (s_o > 1) {
    RP_TRY_LAUNCH_N(nm.oproj, rp::launch_gemm(s, dt, M, d, hq, w.O, hq, bo, bo.trans ? d : hq, nullptr, d,
                                              rp::EPI_PARTIALS, plan.o, gemm_part));
    RP_TRY_LAUNCH_N(nm.norm2, rp::launch_splitk_add_rmsnorm(s, dt, gemm_part, s_o, M, d, w.X, lw.mlp_norm, c.rms_eps,
                                                            w.N));
  } else {
    RP_TRY_LAUNCH_N(nm.oproj, rp::launch_gemm(s, dt, M, d, hq, w.O, hq, bo, bo.trans ? d : hq, w.X, d, rp::EPI_ADD_F32,
                                              plan.o, gemm_part));
    RP_TRY_LAUNCH_N(nm.norm2, rp::launch_rmsnorm(s, dt, w.X, lw.mlp_norm, c.rms_eps, M, d, w.N));
  }
  rp::BSeg bgu = {lw.w_gate, lw.w_up, lw.w_up, F, 2 * F};
  if (plan.fused) {
    RP_TRY_LAUNCH_N(nm.gate_up, rp::launch_gemm(s, dt, M, F, d, w.N, d, bgu, d, w.ACT, F, rp::EPI_SWIGLU, 1, nullptr));
  } else if (s_gu > 1) {
    RP_TRY_LAUNCH_N(nm.gate_up, rp::launch_gemm(s, dt, M, 2 * F, d, w.N, d, bgu, d, nullptr, 2 * F, rp::EPI_PARTIALS,
                                                plan.gu, gemm_part));
    RP_TRY_LAUNCH_N(nm.swiglu, rp::launch_splitk_swiglu(s, dt, gemm_part, s_gu, M, F, w.ACT));
  } else {
    RP_TRY_LAUNCH_N(nm.gate_up, rp::launch_gemm(s, dt, M, 2 * F, d, w.N, d, bgu, d, w.GU, 2 * F, rp::EPI_STORE,
                                                plan.gu, gemm_part));
    RP_TRY_LAUNCH_N(nm.swiglu, rp::launch_swiglu(s, dt, w.GU, M, F, w.ACT));
  }
  const rp::BSeg bd = w_down_operand(c, lw);
  if (s_down > 1 && next_norm) {
    RP_TRY_LAUNCH_N(nm.down, rp::launch_gemm(s, dt, M, d, F, w.ACT, F, bd, bd.trans ? d : F, nullptr, d,
                                             rp::EPI_PARTIALS, plan.down, gemm_part));
    RP_TRY_LAUNCH_N(nm.norm1, rp::launch_splitk_add_rmsnorm(s, dt, gemm_part, s_down, M, d, w.X, next_norm,
                                                            c.rms_eps, w.N));
  } else {
    RP_TRY_LAUNCH_N(nm.down, rp::launch_gemm(s, dt, M, d, F, w.ACT, F, bd, bd.trans ? d : F, w.X, d, rp::EPI_ADD_F32,
                                             plan.down, gemm_part));
  }
  return RP_OK;
}

// Last layer of a RP_PREFIX_LAST_ROWS_ONLY prefix pass: the suffix reads every row's K/V
// but only the boundary state, so beyond the K/V projection only each sequence's last row
// is carried on.  Keys and values are projected for every row, the query for the last
// rows only (scattered into the projection buffer, where RoPE rotates it).  The last
// row's query attends to the sequence's other keys (the first key segment, rows cu[b] ..
// cu[b+1]-2) and to its own key; its residual row, gathered into h_last, takes the o-proj
// and the MLP.
rp_status run_last_rows(const rp_model* m, hipStream_t s, const rp_layer_weights& lw, int32_t B, const int32_t* cu,
                        const rp::SeqTable& tab, int32_t T, const LayerWS& w, const TailWS& t, void* kl, void* vl,
                        const rp::MRope& mr, float* h_last) {
  const rp_config& c = m->cfg;
  const rp_dtype dt = c.dtype;
  const int d = c.d_model, Hq = c.n_q_heads, Hkv = c.n_kv_heads, D = c.head_dim, F = c.ffn_dim;
  const int qkv = (Hq + 2 * Hkv) * D, hq = Hq * D;
  const int es = (int)elem_size(c);
  const int kvr = Hkv * D;
  RP_TRY_LAUNCH_N("prefix.rmsnorm", rp::launch_rmsnorm(s, dt, w.X, lw.attn_norm, c.rms_eps, T, d, w.N));
  const rp::BSeg bkv = {lw.wk, lw.wv, lw.wv, kvr, 2 * kvr};
  RP_TRY_LAUNCH_N("prefix.gemm_kv", rp::launch_gemm(s, dt, T, 2 * kvr, d, w.N, d, bkv, d, w.QKV + hq, qkv,
                                                    rp::EPI_STORE_F32, 1, nullptr));
  RP_TRY_LAUNCH_N("prefix.tail_gather_n", rp::launch_copy_last_rows(s, tab, w.N, (int64_t)d * es, t.N, (int64_t)d * es,
                                                                    d * es, false));
  const rp::BSeg bq = {lw.wq, lw.wq, lw.wq, hq, hq};
  RP_TRY_LAUNCH_N("prefix.tail_gemm_q", rp::launch_gemm(s, dt, B, hq, d, t.N, d, bq, d, t.Qf, hq, rp::EPI_STORE_F32,
                                                        decode_splitk(c, B, hq, d), t.part));
  RP_TRY_LAUNCH_N("prefix.tail_scatter_q", rp::launch_copy_last_rows(s, tab, t.Qf, (int64_t)hq * 4, w.QKV,
                                                                     (int64_t)qkv * 4, hq * 4, true));
  RP_TRY_LAUNCH_N("prefix.rope_kv", rp::launch_rope_kv(s, dt, tab, w.QKV, T, Hq, Hkv, D, lw.bq, lw.bk, lw.bv, m->rope,
                                                       c.max_position, w.Q, kl, vl, mr, true));
  RP_TRY_LAUNCH_N("prefix.tail_gather", rp::launch_gather_last(s, tab, w.Q, hq * es, kl, vl, Hkv * D * es, w.X, d, t.Q,
                                                               t.K, t.V, h_last));
  int32_t one[RP_MAX_SEQS + 1];  // one query row per sequence
  for (int b = 0; b <= B; ++b) one[b] = b;
  rp::SeqTable tl = make_table(B, one, B, cu, nullptr);
  tl.k_drop = 1;
  rp::AttnArgs a;
  a.q = t.Q;
  a.q_ld = hq;
  a.k0 = kl;
  a.v0 = vl;
  a.k1 = t.K;
  a.v1 = t.V;
  a.o = t.O;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.D = D;
  a.scale = (float)(1.0 / sqrt((double)D));
  RP_TRY_LAUNCH_N("prefix.tail_attention", rp::launch_attention(s, dt, tl, a, B));
  const rp::BSeg bo = wo_operand(c, lw);
  RP_TRY_LAUNCH_N("prefix.tail_gemm_o_proj", rp::launch_gemm(s, dt, B, d, hq, t.O, hq, bo, bo.trans ? d : hq, h_last, d,
                                                             rp::EPI_ADD_F32, t.plan.o, t.part));
  RP_TRY_LAUNCH_N("prefix.tail_rmsnorm", rp::launch_rmsnorm(s, dt, h_last, lw.mlp_norm, c.rms_eps, B, d, t.N));
  const rp::BSeg bgu = {lw.w_gate, lw.w_up, lw.w_up, F, 2 * F};
  if (t.plan.fused) {
    RP_TRY_LAUNCH_N("prefix.tail_gemm_gate_up", rp::launch_gemm(s, dt, B, F, d, t.N, d, bgu, d, t.ACT, F, rp::EPI_SWIGLU, 1,
                                                                nullptr));
  } else {
    RP_TRY_LAUNCH_N("prefix.tail_gemm_gate_up", rp::launch_gemm(s, dt, B, 2 * F, d, t.N, d, bgu, d, t.GU, 2 * F,
                                                                rp::EPI_STORE, t.plan.gu, t.part));
    RP_TRY_LAUNCH_N("prefix.tail_swiglu", rp::launch_swiglu(s, dt, t.GU, B, F, t.ACT));
  }
  const rp::BSeg bd = w_down_operand(c, lw);
  RP_TRY_LAUNCH_N("prefix.tail_gemm_down", rp::launch_gemm(s, dt, B, d, F, t.ACT, F, bd, bd.trans ? d : F, h_last, d,
                                                           rp::EPI_ADD_F32, t.plan.down, t.part));
  return RP_OK;
}

// Prefix pass over B sequences (1-D positions, or multimodal ones when mr.pos is set).
rp_status prefix_run(const rp_model* m, void* stream, int32_t B, const int32_t* cu, const int32_t* token_ids,
                     const void* visual, int64_t n_visual, const rp::MRope& mr, uint32_t flags, rp_kv kv_out,
                     float* h_last, float* hidden_out, void* ws, size_t ws_bytes) {
  if (!m) return fail(RP_ERR_INVALID_ARG, "model is NULL");
  rp_status st = check_prefix_cu(m, B, cu, "cu_seqlens");
  if (st != RP_OK) return st;
  const int64_t T = cu[B];
  if (!token_ids || !h_last) return fail(RP_ERR_INVALID_ARG, "token_ids and h_last are required");
  if (n_visual < 0) return fail(RP_ERR_SHAPE, "n_visual %lld < 0", (long long)n_visual);
  if (n_visual > 0 && !visual) return fail(RP_ERR_INVALID_ARG, "visual_embeds is NULL with n_visual > 0");
  if (visual && !aligned16(visual)) return fail(RP_ERR_INVALID_ARG, "visual_embeds must be 16-byte aligned");
  if ((hidden_out && !aligned16(hidden_out)) || !aligned16(h_last))
    return fail(RP_ERR_INVALID_ARG, "h_last / hidden_out must be 16-byte aligned");
  if ((st = check_kv(m, kv_out, T, "kv_out")) != RP_OK) return st;
  if (flags & ~RP_PREFIX_FLAGS) return fail(RP_ERR_INVALID_ARG, "unknown prefix flags 0x%x", flags);
  const bool last_rows = (flags & RP_PREFIX_LAST_ROWS_ONLY) != 0;
  if (last_rows && hidden_out)
    return fail(RP_ERR_INVALID_ARG, "RP_PREFIX_LAST_ROWS_ONLY computes no full hidden state (hidden_out must be NULL)");
  if (last_rows && !mr.pos && half_dtype(m->cfg) && m->cfg.head_dim == 64)
    return fail(RP_ERR_UNSUPPORTED,
                "RP_PREFIX_LAST_ROWS_ONLY with 1-D positions is disabled for 16-bit models at head_dim 64 "
                "(a GPU memory fault in a run that included this combination has no known cause)");
  const size_t need = prefix_ws(m, B, T, nullptr, hidden_out == nullptr, nullptr, nullptr);
  if ((st = check_ws(ws, ws_bytes, need)) != RP_OK) return st;

  hipStream_t s = (hipStream_t)stream;
  const rp_config& c = m->cfg;
  const rp_dtype dt = c.dtype;
  LayerWS w;
  TailWS tail;
  int32_t* vis_idx = nullptr;
  float2* rope_cs = nullptr;
  prefix_ws(m, B, T, ws, hidden_out == nullptr, &w, &vis_idx, &tail, &rope_cs);
  if (hidden_out) w.X = hidden_out;
  DebugPass dbg;
  if ((st = dbg.begin(s, ws)) != RP_OK) return st;
  if ((st = dbg.check_ids(token_ids, (int32_t)T, -1, c.vocab, "token_ids", rp::DBG_ID_RANGE)) != RP_OK) return st;
  const rp::SeqTable tab = make_table(B, cu, 0, nullptr, nullptr);
  const LayerPlan plan = plan_layer(c, (int32_t)T, Pass::kPrefix);
  if (rope_cs)
    RP_TRY_LAUNCH_N("prefix.rope_table", rp::launch_rope_table(s, tab, m->rope, c.max_position, mr, (int32_t)T,
                                                               c.head_dim, rope_cs));

  RP_TRY_LAUNCH_N("prefix.visual_index", rp::launch_visual_index(s, token_ids, (int32_t)T, vis_idx));
  // the embedding kernel also applies the first layer's attention norm
  RP_TRY_LAUNCH_N("prefix.embed_norm", rp::launch_embed(s, dt, token_ids, vis_idx, visual, n_visual, m->embed, c.vocab,
                                                        (int32_t)T, c.d_model, w.X, m->layers[0].attn_norm, c.rms_eps,
                                                        w.N));
  for (int l = 0; l < c.n_layers; ++l) {
    void* kl = layer_ptr(m, kv_out.k, kv_out.layer_stride, l);
    void* vl = layer_ptr(m, kv_out.v, kv_out.layer_stride, l);
    if (last_rows && l == c.n_layers - 1)
      return dbg.end(run_last_rows(m, s, m->layers[l], B, cu, tab, (int32_t)T, w, tail, kl, vl, mr, h_last));
    st = run_layer(m, s, m->layers[l], tab, (int32_t)T, w, kl, vl, kl, vl, plan, nullptr, kPrefixNames, mr, l == 0,
                   nullptr, nullptr, rope_cs);
    if (st != RP_OK) return st;
  }
  RP_TRY_LAUNCH_N("prefix.gather_h_last", rp::launch_gather_rows(s, tab, w.X, c.d_model, h_last));
  return dbg.end(RP_OK);
}

// Suffix pass over n_suffix sequences; sequence s reads prefix grp[s] (s when grp is
// NULL) of the n_prefix prefixes: its KV rows pcu[grp[s]].. and boundary state
// h_last[grp[s]].  Lengths were validated by the caller.
rp_status suffix_run(const rp_model* m, void* stream, int32_t n_prefix, const int32_t* pcu, int32_t n_suffix,
                     const int32_t* grp, const int32_t* scu, const int32_t* rope0, uint32_t flags, rp_kv kv,
                     const float* h_last, const int32_t* response_ids, float* logprobs, void* ws, size_t ws_bytes) {
  const int64_t T = pcu[n_prefix], R = scu[n_suffix];
  rp_status st;
  if ((st = check_kv(m, kv, T, "kv")) != RP_OK) return st;
  if (!h_last) return fail(RP_ERR_INVALID_ARG, "h_last is NULL");
  if (!aligned16(h_last)) return fail(RP_ERR_INVALID_ARG, "h_last must be 16-byte aligned");
  if (R > 0 && (!response_ids || !logprobs)) return fail(RP_ERR_INVALID_ARG, "response_ids and logprobs are required");
  const int32_t splits = suffix_attn_splits(m, n_prefix, pcu);
  const size_t need = suffix_ws(m, R, flags, splits, nullptr, nullptr);
  if ((st = check_ws(ws, ws_bytes, need)) != RP_OK) return st;
  if (R == 0) return RP_OK;

  hipStream_t s = (hipStream_t)stream;
  const rp_config& c = m->cfg;
  const rp_dtype dt = c.dtype;
  SuffixWS w;
  suffix_ws(m, R, flags, splits, ws, &w);
  DebugPass dbg;
  if ((st = dbg.begin(s, ws)) != RP_OK) return st;
  if ((st = dbg.check_ids(response_ids, (int32_t)R, 0, c.vocab, "response_ids", rp::DBG_ID_RANGE)) != RP_OK) return st;
  const rp::SeqTable tab = make_table(n_suffix, scu, n_prefix, pcu, grp, rope0);
  RP_TRY_LAUNCH_N("suffix.embed", rp::launch_decode_embed(s, dt, response_ids, m->embed, c.vocab, (int32_t)R, c.d_model, w.L.X));
  bool norm1_done = false;
  for (int l = 0; l < c.n_layers; ++l) {
    const void* kl = layer_ptr(m, kv.k, kv.layer_stride, l);
    const void* vl = layer_ptr(m, kv.v, kv.layer_stride, l);
    const void* next_norm = l + 1 < c.n_layers ? m->layers[l + 1].attn_norm : nullptr;
    bool normed = false;
    st = run_layer(m, s, m->layers[l], tab, (int32_t)R, w.L, w.Ks, w.Vs, kl, vl, w.plan, w.gemm_part, kSuffixNames,
                   rp::MRope{nullptr, 0, 0}, norm1_done, next_norm, &normed);
    if (st != RP_OK) return st;
    norm1_done = normed;
  }
  RP_TRY_LAUNCH_N("suffix.final_norm", rp::launch_final_norm_rows(s, dt, tab, w.L.X, h_last, m->final_norm, c.rms_eps, (int32_t)R,
                                           c.d_model, w.L.N));
  rp::BSeg blm = {m->lm_head, m->lm_head, m->lm_head, c.vocab, c.vocab};
  if (fused_scoring(m, flags)) {
    const rp::LseOut lo = {response_ids, w.lse, w.tgt};
    RP_TRY_LAUNCH_N("suffix.gemm_lm_head_lse", rp::launch_gemm(s, dt, (int32_t)R, c.vocab, c.d_model, w.L.N, c.d_model, blm,
                                                          c.d_model, nullptr, c.vocab, rp::EPI_LSE, 1, nullptr, &lo));
    RP_TRY_LAUNCH_N("suffix.lse_combine", rp::launch_lse_combine(s, w.lse, w.tgt, (int32_t)R, rp::lse_parts(c.vocab), logprobs));
    return dbg.end(RP_OK);
  }
  RP_TRY_LAUNCH_N("suffix.gemm_lm_head", rp::launch_gemm(s, dt, (int32_t)R, c.vocab, c.d_model, w.L.N, c.d_model, blm, c.d_model, w.logits,
                                c.vocab, rp::EPI_STORE_F32, 1, nullptr));
  RP_TRY_LAUNCH_N("suffix.logsoftmax_gather", rp::launch_logsoftmax_gather(s, w.logits, response_ids, (int32_t)R, c.vocab, logprobs));
  return dbg.end(RP_OK);
}

}  // namespace

extern "C" {

const char* rp_last_error(void) { return g_err.c_str(); }

const char* rp_status_string(rp_status s) {
  switch (s) {
    case RP_OK: return "RP_OK";
    case RP_ERR_INVALID_ARG: return "RP_ERR_INVALID_ARG";
    case RP_ERR_SHAPE: return "RP_ERR_SHAPE";
    case RP_ERR_UNSUPPORTED: return "RP_ERR_UNSUPPORTED";
    case RP_ERR_WORKSPACE: return "RP_ERR_WORKSPACE";
    case RP_ERR_HIP: return "RP_ERR_HIP";
  }
  return "RP_UNKNOWN";
}

const char* rp_version(void) { return "rollplex-mi355x 0.1 (gfx950)"; }

rp_status rp_create(const rp_config* cfg, const rp_weights* w, rp_model** out) {
  if (!out) return fail(RP_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  rp_status st = check_config(cfg);
  if (st != RP_OK) return st;
  if (!w || !w->embed || !w->final_norm || !w->lm_head || !w->layers)
    return fail(RP_ERR_INVALID_ARG, "weights: embed, final_norm, lm_head and layers are required");
  for (int l = 0; l < cfg->n_layers; ++l) {
    const rp_layer_weights& lw = w->layers[l];
    const void* req[] = {lw.attn_norm, lw.wq, lw.wk, lw.wv, lw.wo, lw.mlp_norm, lw.w_gate, lw.w_up, lw.w_down};
    for (const void* p : req) {
      if (!p) return fail(RP_ERR_INVALID_ARG, "layer %d: a required weight pointer is NULL", l);
      if (!aligned16(p)) return fail(RP_ERR_INVALID_ARG, "layer %d: weights must be 16-byte aligned", l);
    }
  }
  if (!aligned16(w->embed) || !aligned16(w->lm_head) || !aligned16(w->final_norm))
    return fail(RP_ERR_INVALID_ARG, "embed/lm_head/final_norm must be 16-byte aligned");
  rp_model* m = new rp_model;
  m->cfg = *cfg;
  m->embed = w->embed;
  m->final_norm = w->final_norm;
  m->lm_head = w->lm_head;
  m->layers.assign(w->layers, w->layers + cfg->n_layers);
  memset(&m->rope, 0, sizeof m->rope);
  for (int i = 0; i < cfg->head_dim / 2; ++i)
    m->rope.inv_freq[i] = pow(cfg->rope_theta, -2.0 * (double)i / (double)cfg->head_dim);
  *out = m;
  return RP_OK;
}

void rp_destroy(rp_model* m) { delete m; }

rp_status rp_prefix_workspace_bytes(const rp_model* m, int32_t B, const int32_t* cu, size_t* bytes) {
  if (!m || !bytes) return fail(RP_ERR_INVALID_ARG, "model and bytes are required");
  rp_status s = check_prefix_cu(m, B, cu, "cu_seqlens");
  if (s != RP_OK) return s;
  *bytes = prefix_ws(m, B, cu[B], nullptr, true, nullptr, nullptr);
  return RP_OK;
}

rp_status rp_prefix_forward(const rp_model* m, void* stream, int32_t B, const int32_t* cu, const int32_t* token_ids,
                            const void* visual, int64_t n_visual, rp_kv kv_out, float* h_last, float* hidden_out,
                            void* ws, size_t ws_bytes) {
  return prefix_run(m, stream, B, cu, token_ids, visual, n_visual, rp::MRope{nullptr, 0, 0}, 0u, kv_out, h_last,
                    hidden_out, ws, ws_bytes);
}

rp_status rp_prefix_forward_mrope(const rp_model* m, void* stream, int32_t B, const int32_t* cu,
                                  const int32_t* token_ids, const void* visual, int64_t n_visual,
                                  const int32_t* positions, const int32_t* mrope_section, rp_kv kv_out,
                                  float* h_last, float* hidden_out, void* ws, size_t ws_bytes) {
  if (!m) return fail(RP_ERR_INVALID_ARG, "model is NULL");
  if (!positions || !mrope_section) return fail(RP_ERR_INVALID_ARG, "positions and mrope_section are required");
  return rp_prefix_forward_flags(m, stream, B, cu, token_ids, visual, n_visual, positions, mrope_section, 0u, kv_out,
                                 h_last, hidden_out, ws, ws_bytes);
}

rp_status rp_prefix_forward_flags(const rp_model* m, void* stream, int32_t B, const int32_t* cu,
                                  const int32_t* token_ids, const void* visual, int64_t n_visual,
                                  const int32_t* positions, const int32_t* mrope_section, uint32_t flags,
                                  rp_kv kv_out, float* h_last, float* hidden_out, void* ws, size_t ws_bytes) {
  if (!m) return fail(RP_ERR_INVALID_ARG, "model is NULL");
  if (!positions != !mrope_section)
    return fail(RP_ERR_INVALID_ARG, "positions and mrope_section go together (both NULL: 1-D positions)");
  if (!positions)
    return prefix_run(m, stream, B, cu, token_ids, visual, n_visual, rp::MRope{nullptr, 0, 0}, flags, kv_out, h_last,
                      hidden_out, ws, ws_bytes);
  if (!aligned16(positions)) return fail(RP_ERR_INVALID_ARG, "positions must be 16-byte aligned");
  const int half = m->cfg.head_dim / 2;
  if (mrope_section[0] < 0 || mrope_section[1] < 0 || mrope_section[2] < 0 ||
      mrope_section[0] + mrope_section[1] + mrope_section[2] != half)
    return fail(RP_ERR_SHAPE, "mrope_section (%d, %d, %d) must be non-negative and sum to head_dim / 2 = %d",
                mrope_section[0], mrope_section[1], mrope_section[2], half);
  const rp::MRope mr = {positions, mrope_section[0], mrope_section[0] + mrope_section[1]};
  return prefix_run(m, stream, B, cu, token_ids, visual, n_visual, mr, flags, kv_out, h_last, hidden_out, ws,
                    ws_bytes);
}

rp_status rp_suffix_workspace_bytes(const rp_model* m, int32_t B, const int32_t* pcu, const int32_t* scu,
                                    size_t* bytes) {
  if (!m || !bytes) return fail(RP_ERR_INVALID_ARG, "model and bytes are required");
  rp_status s = check_suffix_cu(m, B, pcu, scu);
  if (s != RP_OK) return s;
  *bytes = suffix_ws(m, scu[B], 0u, suffix_attn_splits(m, B, pcu), nullptr, nullptr);
  return RP_OK;
}

rp_status rp_suffix_logprob(const rp_model* m, void* stream, int32_t B, const int32_t* pcu, const int32_t* scu,
                            rp_kv kv, const float* h_last, const int32_t* response_ids, float* logprobs, void* ws,
                            size_t ws_bytes) {
  if (!m) return fail(RP_ERR_INVALID_ARG, "model is NULL");
  rp_status st = check_suffix_cu(m, B, pcu, scu);
  if (st != RP_OK) return st;
  return suffix_run(m, stream, B, pcu, B, nullptr, scu, nullptr, 0u, kv, h_last, response_ids, logprobs, ws, ws_bytes);
}

rp_status rp_suffix_grouped_workspace_bytes(const rp_model* m, int32_t n_prefix, const int32_t* pcu, int32_t n_suffix,
                                            const int32_t* prefix_of_suffix, const int32_t* scu, uint32_t flags,
                                            size_t* bytes) {
  if (!m || !bytes) return fail(RP_ERR_INVALID_ARG, "model and bytes are required");
  if (flags & ~RP_SUFFIX_FLAGS) return fail(RP_ERR_INVALID_ARG, "unknown suffix flags 0x%x", flags);
  rp_status s = check_grouped_cu(m, n_prefix, pcu, n_suffix, prefix_of_suffix, scu);
  if (s != RP_OK) return s;
  *bytes = suffix_ws(m, scu[n_suffix], flags, suffix_attn_splits(m, n_prefix, pcu), nullptr, nullptr);
  return RP_OK;
}

rp_status rp_suffix_logprob_grouped(const rp_model* m, void* stream, int32_t n_prefix, const int32_t* pcu,
                                    int32_t n_suffix, const int32_t* prefix_of_suffix, const int32_t* scu,
                                    const int32_t* rope_pos0, uint32_t flags, rp_kv kv, const float* h_last,
                                    const int32_t* response_ids, float* logprobs, void* ws, size_t ws_bytes) {
  if (!m) return fail(RP_ERR_INVALID_ARG, "model is NULL");
  if (flags & ~RP_SUFFIX_FLAGS) return fail(RP_ERR_INVALID_ARG, "unknown suffix flags 0x%x", flags);
  rp_status st = check_grouped_cu(m, n_prefix, pcu, n_suffix, prefix_of_suffix, scu, rope_pos0);
  if (st != RP_OK) return st;
  return suffix_run(m, stream, n_prefix, pcu, n_suffix, prefix_of_suffix, scu, rope_pos0, flags, kv, h_last,
                    response_ids, logprobs, ws, ws_bytes);
}

rp_status rp_prompt_logprob_workspace_bytes(const rp_model* m, int32_t n_rows, uint32_t flags, size_t* bytes) {
  if (!m || !bytes) return fail(RP_ERR_INVALID_ARG, "model and bytes are required");
  if (flags & ~RP_SUFFIX_FLAGS) return fail(RP_ERR_INVALID_ARG, "unknown scoring flags 0x%x", flags);
  if (n_rows < 0) return fail(RP_ERR_SHAPE, "n_rows %d < 0", n_rows);
  *bytes = prompt_ws(m, n_rows, flags, nullptr, nullptr);
  return RP_OK;
}

rp_status rp_prompt_logprob(const rp_model* m, void* stream, int32_t B, const int32_t* cu, const int32_t* token_ids,
                            const float* hidden, int32_t n_rows, const int32_t* positions, uint32_t flags,
                            float* logprobs, void* ws, size_t ws_bytes) {
  if (!m) return fail(RP_ERR_INVALID_ARG, "model is NULL");
  if (flags & ~RP_SUFFIX_FLAGS) return fail(RP_ERR_INVALID_ARG, "unknown scoring flags 0x%x", flags);
  rp_status st = check_prefix_cu(m, B, cu, "cu_seqlens");
  if (st != RP_OK) return st;
  if (n_rows < 0) return fail(RP_ERR_SHAPE, "n_rows %d < 0", n_rows);
  if (n_rows > 0 && (!token_ids || !hidden || !positions || !logprobs))
    return fail(RP_ERR_INVALID_ARG, "token_ids, hidden, positions and logprobs are required");
  if (hidden && !aligned16(hidden)) return fail(RP_ERR_INVALID_ARG, "hidden must be 16-byte aligned");
  if ((st = check_ws(ws, ws_bytes, prompt_ws(m, n_rows, flags, nullptr, nullptr))) != RP_OK) return st;
  if (n_rows == 0) return RP_OK;

  hipStream_t s = (hipStream_t)stream;
  const rp_config& c = m->cfg;
  const rp_dtype dt = c.dtype;
  PromptWS w;
  prompt_ws(m, n_rows, flags, ws, &w);
  DebugPass dbg;
  if ((st = dbg.begin(s, ws)) != RP_OK) return st;
  if ((st = dbg.check_ids(token_ids, cu[B], -1, c.vocab, "token_ids", rp::DBG_ID_RANGE)) != RP_OK) return st;
  const rp::SeqTable tab = make_table(B, cu, 0, nullptr, nullptr);
  RP_TRY_LAUNCH_N("prompt.rows", rp::launch_prompt_rows(s, dt, tab, positions, n_rows, token_ids, cu[B], hidden,
                                                        m->final_norm, c.rms_eps, c.d_model, w.N, w.tid));
  rp::BSeg blm = {m->lm_head, m->lm_head, m->lm_head, c.vocab, c.vocab};
  if (fused_scoring(m, flags)) {
    const rp::LseOut lo = {w.tid, w.lse, w.tgt};
    RP_TRY_LAUNCH_N("prompt.gemm_lm_head_lse", rp::launch_gemm(s, dt, n_rows, c.vocab, c.d_model, w.N, c.d_model, blm,
                                                               c.d_model, nullptr, c.vocab, rp::EPI_LSE, 1, nullptr, &lo));
    RP_TRY_LAUNCH_N("prompt.lse_combine",
                    rp::launch_lse_combine(s, w.lse, w.tgt, n_rows, rp::lse_parts(c.vocab), logprobs, w.tid));
    return dbg.end(RP_OK);
  }
  RP_TRY_LAUNCH_N("prompt.gemm_lm_head", rp::launch_gemm(s, dt, n_rows, c.vocab, c.d_model, w.N, c.d_model, blm,
                                                         c.d_model, w.logits, c.vocab, rp::EPI_STORE_F32, 1, nullptr));
  RP_TRY_LAUNCH_N("prompt.logsoftmax_gather",
                  rp::launch_logsoftmax_gather(s, w.logits, w.tid, n_rows, c.vocab, logprobs, true));
  return dbg.end(RP_OK);
}

rp_status rp_decode_workspace_bytes(const rp_model* m, int32_t B, int32_t cap, size_t* bytes) {
  if (!m || !bytes) return fail(RP_ERR_INVALID_ARG, "model and bytes are required");
  if (B < 1 || cap < 1) return fail(RP_ERR_SHAPE, "batch and cap must be >= 1");
  *bytes = decode_ws(m, B, cap, nullptr, nullptr);
  return RP_OK;
}

}  // extern "C"

namespace {

// Host-side checks of a decode step (before any HIP call).
rp_status check_decode(const rp_model* m, int32_t B, const rp_kv& cache, int32_t cap, const int32_t* kv_len,
                       const int32_t* token_ids, const int32_t* next_ids) {
  if (!m) return fail(RP_ERR_INVALID_ARG, "model is NULL");
  if (B < 1 || cap < 1) return fail(RP_ERR_SHAPE, "batch and cap must be >= 1");
  if ((int64_t)B * cap > (int64_t)1 << 31) return fail(RP_ERR_UNSUPPORTED, "batch * cap too large");
  rp_status st = check_kv(m, cache, (int64_t)B * cap, "cache");
  if (st != RP_OK) return st;
  if (!kv_len || !token_ids || !next_ids) return fail(RP_ERR_INVALID_ARG, "kv_len, token_ids and next_ids are required");
  if ((int64_t)(m->cfg.n_q_heads + 2 * m->cfg.n_kv_heads) * m->cfg.head_dim * 4 > 65536)
    return fail(RP_ERR_UNSUPPORTED, "decode step: a q/k/v row must fit 64 KiB of LDS");
  if (m->cfg.dtype == RP_BF16 && m->cfg.head_dim == 64)
    return fail(RP_ERR_UNSUPPORTED,
                "decode step is disabled for bf16 models at head_dim 64 (a GPU memory fault in a run that "
                "included this combination has no known cause)");
  return RP_OK;
}

// The decode step's launches over a validated, large enough workspace (carved with
// own_logits as sized).
rp_status decode_run(const rp_model* m, void* stream, int32_t B, rp_kv cache, int32_t cap, const int32_t* kv_len,
                     const int32_t* token_ids, float* logits, int32_t* next_ids, void* ws, bool own_logits) {
  hipStream_t s = (hipStream_t)stream;
  const rp_config& c = m->cfg;
  const rp_dtype dt = c.dtype;
  DecodeWS w;
  decode_ws(m, B, cap, ws, &w, own_logits);
  float* lg = logits ? logits : w.logits;
  DebugPass dbg;
  rp_status st;
  if ((st = dbg.begin(s, ws)) != RP_OK) return st;
  if ((st = dbg.check_ids(token_ids, B, 0, c.vocab, "token_ids", rp::DBG_ID_RANGE)) != RP_OK) return st;
  if ((st = dbg.check_ids(kv_len, B, 0, std::min(cap, c.max_position), "kv_len", rp::DBG_KV_LEN)) != RP_OK) return st;
  const int d = c.d_model, Hq = c.n_q_heads, Hkv = c.n_kv_heads, D = c.head_dim, F = c.ffn_dim;
  const int qkv = (Hq + 2 * Hkv) * D, hq = Hq * D;
  const float scale = (float)(1.0 / sqrt((double)D));
  // Each layer GEMM writes split-K partials (EPI_PARTIALS) and the kernel that consumes
  // its output sums them: RoPE + cache write, residual add + the next RMSNorm, SwiGLU.
  // The last layer's down projection is followed by the final norm the same way.
  RP_TRY_LAUNCH_N("decode.embed_norm", rp::launch_decode_embed_norm(s, dt, token_ids, m->embed, c.vocab, B, d, w.L.X,
                                                                    m->layers[0].attn_norm, c.rms_eps, w.L.N));
  for (int l = 0; l < c.n_layers; ++l) {
    const rp_layer_weights& lw = m->layers[l];
    void* kl = layer_ptr(m, cache.k, cache.layer_stride, l);
    void* vl = layer_ptr(m, cache.v, cache.layer_stride, l);
    const void* next_norm = l + 1 < c.n_layers ? m->layers[l + 1].attn_norm : m->final_norm;
    rp::BSeg bqkv = {lw.wq, lw.wk, lw.wv, hq, hq + Hkv * D};
    const int s_qkv = decode_splitk(c, B, qkv, d);
    RP_TRY_LAUNCH_N("decode.gemm_qkv", rp::launch_gemm(s, dt, B, qkv, d, w.L.N, d, bqkv, d, nullptr, qkv,
                                                       rp::EPI_PARTIALS, s_qkv, w.gemm_part));
    RP_TRY_LAUNCH_N("decode.rope_kv", rp::launch_decode_rope_kv_splitk(s, dt, w.gemm_part,
                                                                       rp::gemm_effective_splitk(dt, d, s_qkv), B, Hq,
                                                                       Hkv, D, lw.bq, lw.bk, lw.bv, m->rope, kv_len,
                                                                       cap, c.max_position, w.L.Q, kl, vl));
    RP_TRY_LAUNCH_N("decode.attention", rp::launch_decode_attention(s, dt, w.L.Q, hq, kl, vl, kv_len, cap, c.max_position, B, Hq, Hkv,
                                              D, scale, w.attn_part, w.L.O));
    const rp::BSeg bo = wo_operand(c, lw);
    const int s_o = decode_splitk(c, B, d, hq);
    RP_TRY_LAUNCH_N("decode.gemm_o_proj", rp::launch_gemm(s, dt, B, d, hq, w.L.O, hq, bo, bo.trans ? d : hq, nullptr,
                                                          d, rp::EPI_PARTIALS, s_o, w.gemm_part));
    RP_TRY_LAUNCH_N("decode.add_rmsnorm", rp::launch_splitk_add_rmsnorm(s, dt, w.gemm_part,
                                                                        rp::gemm_effective_splitk(dt, hq, s_o), B, d,
                                                                        w.L.X, lw.mlp_norm, c.rms_eps, w.L.N));
    rp::BSeg bgu = {lw.w_gate, lw.w_up, lw.w_up, F, 2 * F};
    const int s_gu = decode_splitk(c, B, 2 * F, d);
    RP_TRY_LAUNCH_N("decode.gemm_gate_up", rp::launch_gemm(s, dt, B, 2 * F, d, w.L.N, d, bgu, d, nullptr, 2 * F,
                                                           rp::EPI_PARTIALS, s_gu, w.gemm_part));
    RP_TRY_LAUNCH_N("decode.swiglu", rp::launch_splitk_swiglu(s, dt, w.gemm_part, rp::gemm_effective_splitk(dt, d, s_gu),
                                                              B, F, w.L.ACT));
    const rp::BSeg bd = w_down_operand(c, lw);
    const int s_down = decode_splitk(c, B, d, F);
    RP_TRY_LAUNCH_N("decode.gemm_down", rp::launch_gemm(s, dt, B, d, F, w.L.ACT, F, bd, bd.trans ? d : F, nullptr, d,
                                                        rp::EPI_PARTIALS, s_down, w.gemm_part));
    RP_TRY_LAUNCH_N("decode.add_rmsnorm", rp::launch_splitk_add_rmsnorm(s, dt, w.gemm_part,
                                                                        rp::gemm_effective_splitk(dt, F, s_down), B, d,
                                                                        w.L.X, next_norm, c.rms_eps, w.L.N));
  }
  rp::BSeg blm = {m->lm_head, m->lm_head, m->lm_head, c.vocab, c.vocab};
  if (!logits && w.arg_part) {
    RP_TRY_LAUNCH_N("decode.gemm_lm_head_argmax", rp::launch_gemm_argmax(s, dt, B, c.vocab, d, w.L.N, d, blm, d,
                                                                         w.arg_part, next_ids));
    return dbg.end(RP_OK);
  }
  RP_TRY_LAUNCH_N("decode.gemm_lm_head", rp::launch_gemm(s, dt, B, c.vocab, d, w.L.N, d, blm, d, lg, c.vocab, rp::EPI_STORE_F32,
                                decode_splitk(c, B, c.vocab, d), w.gemm_part));
  RP_TRY_LAUNCH_N("decode.argmax", rp::launch_argmax(s, lg, B, c.vocab, next_ids));
  return dbg.end(RP_OK);
}

// Library-owned scratch of rp_decode_step_static: one copy on every GPU the library
// runs on, held until the process ends.  In host code the array's name is only a
// stand-in: its device address on the current GPU comes from hipGetSymbolAddress, taken
// once per device and kept in g_scratch_addr.
static __device__ __align__(256) uint8_t scratch[RP_DECODE_STATIC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_addr[kMaxDevices] = {};

rp_status static_scratch(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(RP_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return fail(RP_ERR_UNSUPPORTED, "device %d outside [0, %d)", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(RP_ERR_HIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev, hipGetErrorString(e));
    g_scratch_addr[dev] = p;
  }
  *out = g_scratch_addr[dev];
  return RP_OK;
}

}  // namespace

extern "C" {

rp_status rp_decode_step(const rp_model* m, void* stream, int32_t B, rp_kv cache, int32_t cap, const int32_t* kv_len,
                         const int32_t* token_ids, float* logits, int32_t* next_ids, void* ws, size_t ws_bytes) {
  rp_status st = check_decode(m, B, cache, cap, kv_len, token_ids, next_ids);
  if (st != RP_OK) return st;
  const size_t need = decode_ws(m, B, cap, nullptr, nullptr);
  if ((st = check_ws(ws, ws_bytes, need)) != RP_OK) return st;
  return decode_run(m, stream, B, cache, cap, kv_len, token_ids, logits, next_ids, ws, true);
}

rp_status rp_decode_step_static(const rp_model* m, void* stream, int32_t B, rp_kv cache, int32_t cap,
                                const int32_t* kv_len, const int32_t* token_ids, float* logits, int32_t* next_ids) {
  rp_status st = check_decode(m, B, cache, cap, kv_len, token_ids, next_ids);
  if (st != RP_OK) return st;
  const bool own_logits = logits == nullptr && !decode_fused_argmax(m, B);
  const size_t need = decode_ws(m, B, cap, nullptr, nullptr, own_logits);
  if (need > (size_t)RP_DECODE_STATIC_SCRATCH_BYTES)
    return fail(RP_ERR_WORKSPACE,
                "rp_decode_step_static: batch %d, cap %d needs %zu bytes of scratch%s; the static scratch holds %zu",
                B, cap, need, own_logits ? " (logits included: pass a logits buffer to need less)" : "",
                (size_t)RP_DECODE_STATIC_SCRATCH_BYTES);
  void* ws = nullptr;
  if ((st = static_scratch(&ws)) != RP_OK) return st;
  return decode_run(m, stream, B, cache, cap, kv_len, token_ids, logits, next_ids, ws, own_logits);
}

rp_status rp_profile_enable(int enable, int32_t max_launches) {
  for (hipEvent_t e : g_prof.ev) (void)hipEventDestroy(e);  // teardown of timing events: nothing to report
  g_prof.ev.clear();
  g_prof.pending.clear();
  g_prof.on = false;
  if (!enable) return RP_OK;
  if (max_launches < 1) return fail(RP_ERR_INVALID_ARG, "max_launches must be >= 1");
  g_prof.ev.resize(2 * (size_t)max_launches + 2);
  for (auto& e : g_prof.ev) {
    hipError_t r = hipEventCreate(&e);
    if (r != hipSuccess) {
      g_prof.ev.clear();
      return fail(RP_ERR_HIP, "hipEventCreate: %s", hipGetErrorString(r));
    }
  }
  g_prof.on = true;
  return RP_OK;
}

rp_status rp_profile_collect(void) {
  for (size_t k = 0; k < g_prof.pending.size(); ++k) {
    hipError_t r = hipEventSynchronize(g_prof.ev[2 * k + 1]);
    float ms = 0.f;
    if (r == hipSuccess) r = hipEventElapsedTime(&ms, g_prof.ev[2 * k], g_prof.ev[2 * k + 1]);
    if (r != hipSuccess) {
      g_prof.pending.clear();
      return fail(RP_ERR_HIP, "profiling: %s", hipGetErrorString(r));
    }
    size_t i = 0;
    while (i < g_prof.names.size() && g_prof.names[i] != g_prof.pending[k]) ++i;
    if (i == g_prof.names.size()) {
      g_prof.names.push_back(g_prof.pending[k]);
      g_prof.count.push_back(0);
      g_prof.ms.push_back(0.0);
    }
    g_prof.count[i] += 1;
    g_prof.ms[i] += ms;
  }
  g_prof.pending.clear();
  return RP_OK;
}

int32_t rp_profile_count(void) { return (int32_t)g_prof.names.size(); }

rp_status rp_profile_read(int32_t i, const char** name, int64_t* launches, double* total_ms) {
  if (i < 0 || i >= (int32_t)g_prof.names.size()) return fail(RP_ERR_INVALID_ARG, "profile index %d out of range", i);
  if (name) *name = g_prof.names[i].c_str();
  if (launches) *launches = g_prof.count[i];
  if (total_ms) *total_ms = g_prof.ms[i];
  return RP_OK;
}

void rp_profile_reset(void) {
  g_prof.names.clear();
  g_prof.count.clear();
  g_prof.ms.clear();
  g_prof.pending.clear();
}

rp_status rp_stream_create_cu_masked(int device, const uint32_t* mask, uint32_t n_words, void** out) {
  if (!out || !mask || n_words == 0) return fail(RP_ERR_INVALID_ARG, "mask, n_words and out are required");
  *out = nullptr;
  bool any = false;
  for (uint32_t i = 0; i < n_words; ++i) any |= mask[i] != 0;
  if (!any) return fail(RP_ERR_INVALID_ARG, "CU mask selects no compute unit");
  int prev = 0;
  hipError_t e = hipGetDevice(&prev);
  if (e != hipSuccess) return fail(RP_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  if ((e = hipSetDevice(device)) != hipSuccess) return fail(RP_ERR_HIP, "hipSetDevice(%d): %s", device, hipGetErrorString(e));
  hipStream_t s = nullptr;
  e = hipExtStreamCreateWithCUMask(&s, n_words, mask);
  const hipError_t er = hipSetDevice(prev);
  if (e != hipSuccess) return fail(RP_ERR_HIP, "hipExtStreamCreateWithCUMask: %s", hipGetErrorString(e));
  if (er != hipSuccess) {
    (void)hipStreamDestroy(s);
    return fail(RP_ERR_HIP, "hipSetDevice(%d) after creating the stream: %s", prev, hipGetErrorString(er));
  }
  *out = (void*)s;
  return RP_OK;
}

rp_status rp_stream_destroy(void* stream) {
  if (!stream) return fail(RP_ERR_INVALID_ARG, "stream is NULL");
  hipError_t e = hipStreamDestroy((hipStream_t)stream);
  if (e != hipSuccess) return fail(RP_ERR_HIP, "hipStreamDestroy: %s", hipGetErrorString(e));
  return RP_OK;
}

rp_status rp_calibrate_mfma(void* stream, rp_dtype dtype, int32_t blocks, int32_t iters, float* sink,
                            size_t sink_bytes, double* flops) {
  if (dtype != RP_BF16 && dtype != RP_F16) return fail(RP_ERR_INVALID_ARG, "dtype must be RP_BF16 or RP_F16");
  if (blocks < 1 || iters < 1) return fail(RP_ERR_SHAPE, "blocks and iters must be >= 1");
  if (!sink || !aligned16(sink)) return fail(RP_ERR_INVALID_ARG, "sink must be a 16-byte aligned device buffer");
  if (sink_bytes < (size_t)blocks * 256 * 4)
    return fail(RP_ERR_WORKSPACE, "sink holds %zu bytes, needs %zu", sink_bytes, (size_t)blocks * 256 * 4);
  if (flops) *flops = (double)blocks * 4.0 * (double)iters * 8.0 * 32.0 * 32.0 * 16.0 * 2.0;
  const hipError_t e = rp::launch_mfma_probe((hipStream_t)stream, dtype, blocks, iters, sink);
  if (e != hipSuccess) return fail(RP_ERR_HIP, "mfma probe launch: %s", hipGetErrorString(e));
  return RP_OK;
}

rp_status rp_calibrate_read(void* stream, const void* src, int64_t bytes, int32_t blocks, uint32_t* sink,
                            size_t sink_bytes) {
  if (!src || !sink || !aligned16(src) || !aligned16(sink))
    return fail(RP_ERR_INVALID_ARG, "src and sink must be 16-byte aligned device buffers");
  if (bytes < 16 || (bytes & 15) || blocks < 1) return fail(RP_ERR_SHAPE, "bytes must be a positive multiple of 16");
  if (sink_bytes < (size_t)blocks * 256 * 4)
    return fail(RP_ERR_WORKSPACE, "sink holds %zu bytes, needs %zu", sink_bytes, (size_t)blocks * 256 * 4);
  const hipError_t e = rp::launch_read_probe((hipStream_t)stream, src, bytes, blocks, sink);
  if (e != hipSuccess) return fail(RP_ERR_HIP, "read probe launch: %s", hipGetErrorString(e));
  return RP_OK;
}

int rp_device_cu_count(int device) {
  int n = 0;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, device) != hipSuccess) return -1;
  return n;
}

}  // extern "C"
