// Runtime of the TADM reverse-diffusion step: model weights in HBM, anchor cache,
// block-diffusion context KV, step orchestration on one HIP stream, C ABI.
//
// Every step is a fixed sequence of kernel launches whose sizes are known on the
// host (the unmask count of the linear schedule is a host integer), so a whole
// generation is enqueued without any device-to-host synchronisation.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include <rocprofiler-sdk-roctx/roctx.h>

#include "../../include/tadm.h"
#include "kernels.h"

using namespace tadm;

thread_local tadm::LaunchEvents tadm::next_launch_events;

// ------------------------------------------------------------------ errors ----
static thread_local std::string g_err;

static tadm_status fail(tadm_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

#define HIPCHK(expr)                                                                          \
  do {                                                                                        \
    hipError_t e_ = (expr);                                                                   \
    if (e_ != hipSuccess)                                                                     \
      return fail(e_ == hipErrorOutOfMemory ? TADM_ERR_OOM : TADM_ERR_DEVICE, "%s: %s (%s:%d)", \
                  #expr, hipGetErrorString(e_), __FILE__, __LINE__);                          \
  } while (0)

#define TRY(expr)                      \
  do {                                 \
    tadm_status s_ = (expr);           \
    if (s_ != TADM_OK) return s_;      \
  } while (0)

static size_t align256(size_t x) { return (x + 255) & ~size_t(255); }
static constexpr size_t align_up_const(size_t x) { return (x + 255) & ~size_t(255); }
static int round64(int x) { return (x + 63) / 64 * 64; }

// ----------------------------------------------------------- weight specs ----
namespace {

enum Place { P_COPY, P_ROWS, P_GLU, P_VEC };

struct Spec {
  std::string name;
  long rows, cols;  // cols == 0: vector of `rows` elements
  // destination
  int target;       // index into Model::tensors
  Place place;
  long row_off;
  int glu_half;
  int rope_dh;      // > 0: q/k rows reordered so rotary pairs are adjacent
};

struct Tensor {
  long rows, cols;  // stored shape
  bool f32;         // stored as float32 (norm gains, biases) or model dtype
  size_t off;       // byte offset in the arena
};

struct LayerIdx {
  int attn_norm, wqkv, wo, ffn_norm, wup, wdown;
};

struct Layout {
  std::vector<Spec> specs;
  std::vector<Tensor> tensors;
  int embed, final_norm, w_out;
  int ln_s_w, ln_s_b, ln_a_w, ln_a_b, w1g, b1g, w2, b2, ln_o_w, ln_o_b;  // gated MLP
  int p_wc, p_wh, p_wqkv, p_wo, p_w1, p_w2, p_wg1, p_wg2, p_bg, p_wup;   // paired attention
  std::vector<LayerIdx> layers;
  size_t bytes;
};

int add_tensor(Layout& L, long rows, long cols, bool f32) {
  L.tensors.push_back(Tensor{rows, cols, f32, 0});
  return (int)L.tensors.size() - 1;
}

void add_spec(Layout& L, const std::string& n, long rows, long cols, int target, Place p,
              long row_off = 0, int glu_half = -1, int rope_dh = 0) {
  L.specs.push_back(Spec{n, rows, cols, target, p, row_off, glu_half, rope_dh});
}

Layout make_layout(const tadm_config& c) {
  Layout L{};
  const long d = c.d_model, V = c.vocab, H = c.n_heads, Hk = c.n_kv_heads, dh = c.head_dim,
             F = c.d_ffn;
  L.embed = add_tensor(L, V + 1, d, false);
  L.final_norm = add_tensor(L, d, 1, true);
  L.w_out = add_tensor(L, V, d, false);
  add_spec(L, "embed", V + 1, d, L.embed, P_COPY);
  add_spec(L, "final_norm", d, 0, L.final_norm, P_VEC);
  add_spec(L, "w_out", V, d, L.w_out, P_COPY);
  if (c.fusion_kind == TADM_FUSION_GATED_MLP) {
    L.ln_s_w = add_tensor(L, d, 1, true);
    L.ln_s_b = add_tensor(L, d, 1, true);
    L.ln_a_w = add_tensor(L, d, 1, true);
    L.ln_a_b = add_tensor(L, d, 1, true);
    L.w1g = add_tensor(L, 5 * d, 2 * d, false);  // rows [0,4d) = W1, [4d,5d) = W_g
    L.b1g = add_tensor(L, 5 * d, 1, true);
    L.w2 = add_tensor(L, d, 4 * d, false);
    L.b2 = add_tensor(L, d, 1, true);
    L.ln_o_w = add_tensor(L, d, 1, true);
    L.ln_o_b = add_tensor(L, d, 1, true);
    add_spec(L, "fusion.ln_s_w", d, 0, L.ln_s_w, P_VEC);
    add_spec(L, "fusion.ln_s_b", d, 0, L.ln_s_b, P_VEC);
    add_spec(L, "fusion.ln_a_w", d, 0, L.ln_a_w, P_VEC);
    add_spec(L, "fusion.ln_a_b", d, 0, L.ln_a_b, P_VEC);
    add_spec(L, "fusion.w1", 4 * d, 2 * d, L.w1g, P_ROWS, 0);
    add_spec(L, "fusion.b1", 4 * d, 0, L.b1g, P_VEC, 0);
    add_spec(L, "fusion.wg", d, 2 * d, L.w1g, P_ROWS, 4 * d);
    add_spec(L, "fusion.bg", d, 0, L.b1g, P_VEC, 4 * d);
    add_spec(L, "fusion.w2", d, 4 * d, L.w2, P_COPY);
    add_spec(L, "fusion.b2", d, 0, L.b2, P_VEC);
    add_spec(L, "fusion.ln_o_w", d, 0, L.ln_o_w, P_VEC);
    add_spec(L, "fusion.ln_o_b", d, 0, L.ln_o_b, P_VEC);
  } else {
    const long r = c.fusion_rank;
    L.p_wc = add_tensor(L, r, d, false);
    L.p_wh = add_tensor(L, r, d, false);
    L.p_wqkv = add_tensor(L, 3 * r, 2 * r, false);  // rows W_Q, W_K, W_V
    L.p_wo = add_tensor(L, r, r, false);
    L.p_w1 = add_tensor(L, 2 * r, r, false);
    L.p_w2 = add_tensor(L, r, 2 * r, false);
    L.p_wg1 = add_tensor(L, r, 4 * r, false);
    L.p_wg2 = add_tensor(L, 1, r, true);
    L.p_bg = add_tensor(L, 1, 1, true);
    L.p_wup = add_tensor(L, d, r, false);
    add_spec(L, "fusion.w_c", r, d, L.p_wc, P_COPY);
    add_spec(L, "fusion.w_h", r, d, L.p_wh, P_COPY);
    add_spec(L, "fusion.w_q", r, 2 * r, L.p_wqkv, P_ROWS, 0);
    add_spec(L, "fusion.w_k", r, 2 * r, L.p_wqkv, P_ROWS, r);
    add_spec(L, "fusion.w_v", r, 2 * r, L.p_wqkv, P_ROWS, 2 * r);
    add_spec(L, "fusion.w_o", r, r, L.p_wo, P_COPY);
    add_spec(L, "fusion.w_f1", 2 * r, r, L.p_w1, P_COPY);
    add_spec(L, "fusion.w_f2", r, 2 * r, L.p_w2, P_COPY);
    add_spec(L, "fusion.w_g1", r, 4 * r, L.p_wg1, P_COPY);
    add_spec(L, "fusion.w_g2", 1, r, L.p_wg2, P_COPY);
    add_spec(L, "fusion.b_g", 1, 0, L.p_bg, P_VEC);
    add_spec(L, "fusion.w_up", d, r, L.p_wup, P_COPY);
  }
  const int nl = c.n_shared + c.n_anchor + c.n_denoise;
  const bool glu = c.ffn_kind != TADM_FFN_GELU;
  for (int li = 0; li < nl; ++li) {
    const std::string p = "layer" + std::to_string(li) + ".";
    LayerIdx x;
    x.attn_norm = add_tensor(L, d, 1, true);
    x.wqkv = add_tensor(L, (H + 2 * Hk) * dh, d, false);
    x.wo = add_tensor(L, d, H * dh, false);
    x.ffn_norm = add_tensor(L, d, 1, true);
    x.wup = add_tensor(L, glu ? 2 * F : F, d, false);
    x.wdown = add_tensor(L, d, F, false);
    L.layers.push_back(x);
    add_spec(L, p + "attn_norm", d, 0, x.attn_norm, P_VEC);
    add_spec(L, p + "wq", H * dh, d, x.wqkv, P_ROWS, 0, -1, (int)dh);
    add_spec(L, p + "wk", Hk * dh, d, x.wqkv, P_ROWS, H * dh, -1, (int)dh);
    add_spec(L, p + "wv", Hk * dh, d, x.wqkv, P_ROWS, (H + Hk) * dh);
    add_spec(L, p + "wo", d, H * dh, x.wo, P_COPY);
    add_spec(L, p + "ffn_norm", d, 0, x.ffn_norm, P_VEC);
    if (glu) {
      add_spec(L, p + "w_gate", F, d, x.wup, P_GLU, 0, 0);
      add_spec(L, p + "w_up", F, d, x.wup, P_GLU, 0, 1);
    } else {
      add_spec(L, p + "w_up", F, d, x.wup, P_COPY);
    }
    add_spec(L, p + "w_down", d, F, x.wdown, P_COPY);
  }
  return L;
}

tadm_status finish_layout(Layout& L, size_t esz) {
  size_t off = 0;
  for (auto& t : L.tensors) {
    t.off = off;
    off = align256(off + (size_t)t.rows * (size_t)t.cols * (t.f32 ? 4 : esz));
  }
  L.bytes = off;
  return TADM_OK;
}

bool valid_config(const tadm_config* c, std::string& why) {
  if (!c) { why = "null config"; return false; }
  if (c->dtype != TADM_DTYPE_F32 && c->dtype != TADM_DTYPE_BF16) { why = "dtype"; return false; }
  if (c->vocab < 1 || c->d_model < 4 || c->n_heads < 1 || c->n_kv_heads < 1 || c->head_dim < 2 ||
      c->d_ffn < 16 || c->max_batch < 1 || c->max_seq < 1) { why = "non-positive size"; return false; }
  if (c->n_shared < 0 || c->n_anchor < 0 || c->n_denoise < 0) { why = "layer counts"; return false; }
  if (c->vocab > SAMPLE_MAX_VOCAB) { why = "vocab above the sampler's 262144 entries"; return false; }
  if (c->n_heads % c->n_kv_heads) { why = "n_heads must be a multiple of n_kv_heads"; return false; }
  if (c->head_dim % 4) { why = "head_dim must be a multiple of 4"; return false; }
  if (c->ffn_kind < 0 || c->ffn_kind > 2) { why = "ffn_kind"; return false; }
  if (c->fusion_kind < 0 || c->fusion_kind > 1) { why = "fusion_kind"; return false; }
  if (c->fusion_kind == TADM_FUSION_PAIRED &&
      (c->fusion_rank < 4 || c->paired_heads < 1 || c->fusion_rank % (4 * c->paired_heads) ||
       c->fusion_rank > c->n_kv_heads * c->head_dim || c->fusion_rank > c->n_heads * c->head_dim ||
       2 * c->fusion_rank > c->d_ffn)) {
    why = "paired fusion needs rank a multiple of 4*heads and at most the KV width";
    return false;
  }
  if (c->d_ffn % 16) { why = "d_ffn must be a multiple of 16"; return false; }
  if (c->d_model % 4 || (c->n_heads * c->head_dim) % 4) { why = "widths must be multiples of 4"; return false; }
  if (!(c->rms_eps > 0) || !(c->ln_eps > 0) || !(c->rope_theta > 0)) { why = "eps/theta"; return false; }
  return true;
}

}  // namespace

// ------------------------------------------------------------------ objects ---
struct Workspace {
  int n_tok = 0, n_canvas = 0;  // capacity in tokens / canvas rows
  float *x = nullptr, *c = nullptr, *ht = nullptr, *fus_g = nullptr, *conf = nullptr;
  void *xn = nullptr, *qkv = nullptr, *q = nullptr, *k = nullptr, *vt = nullptr, *ao = nullptr,
       *ffn = nullptr, *fus_h = nullptr;
  float* ffn_pre = nullptr;  // fp32 GLU pre-activations
  // paired-attention fusion
  float *pz = nullptr, *pr = nullptr, *pgate = nullptr;
  void *pzb = nullptr, *pqkv = nullptr, *prb = nullptr, *pmb = nullptr, *pf = nullptr, *pg1 = nullptr;
  int32_t* choice = nullptr;
  int32_t *cidx = nullptr, *row_map = nullptr;  // masked-position list and its inverse
  int* count = nullptr;                         // number of masked positions (device)
  NucleusThr* nthr = nullptr;                   // per-position nucleus thresholds
  // entropy-bound sampler: argmax, exact entropies, 2^40 / A per row, the weights e_v
  // [rows, round64(V)] for the self-conditioning product (lazy) and generation's signal
  int32_t* xhat = nullptr;
  long long* hq = nullptr;
  float* rscale = nullptr;
  void* pw = nullptr;
  size_t pw_cap = 0;
  float* kpart = nullptr;  // K-slice products of split GEMMs (lazy)
  size_t kpart_cap = 0;
  int32_t *zt = nullptr, *zs = nullptr;  // training pair (lazy)
  float* ce = nullptr;
  float* sc = nullptr;
  float* logits = nullptr;
  size_t logits_cap = 0;
  int kv_cap = 0;
  std::vector<void*> allocs;
};

struct ProfRec {
  int stage;
  hipEvent_t a, b;
};

struct OpenStage {
  int stage;
  hipEvent_t a, b;  // b is set for a single-kernel stage: both events ride on its launch
};

struct tadm_model {
  tadm_config cfg;
  DType dt;
  size_t esz;
  int device;
  hipStream_t stream = nullptr;
  Layout lay;
  char* arena = nullptr;
  std::vector<char> loaded;
  float* rope = nullptr;  // rotary table [max_seq][dh/2][cos, sin]
  Workspace ws;
  bool taps = false;
  bool tap_final = false;  // TADM_TAP_FINAL holds every canvas row (full-logits step)
  // objects reused across calls so that a generation allocates nothing after warm-up
  tadm_cache* scratch = nullptr;   // anchor state of context appends (capacity max_batch x max_seq)
  tadm_cache* gcache = nullptr;    // anchor cache of tadm_generate
  tadm_cache* tcache = nullptr;    // anchor cache of tadm_train_loss
  tadm_context* gctx = nullptr;    // context of block-mode tadm_generate
  int32_t* gwin = nullptr;         // active block of block-mode tadm_generate
  void* embT = nullptr;            // embedding rows [0, V) transposed, [d, round64(V)] (lazy)
  bool embT_valid = false;
  int tap_B = 0, tap_L = 0, tap_Lc = 0;
  // per-layer capture (tadm_debug_layers): residual stream entering each layer, after its
  // attention half and leaving it
  float* layer_cap = nullptr;
  size_t layer_cap_bytes = 0;
  // profiling
  int32_t prof_mask = 0;  // bit s: record stage s
  std::vector<ProfRec> recs;
  std::vector<hipEvent_t> pool;
  std::vector<OpenStage> open;  // stages begun and not yet ended

  void* W(int t) const { return arena + lay.tensors[t].off; }
  float* Wf(int t) const { return reinterpret_cast<float*>(arena + lay.tensors[t].off); }
  int n_layers() const { return cfg.n_shared + cfg.n_anchor + cfg.n_denoise; }
};

struct tadm_cache {
  tadm_model* model;
  int B, L;
  float *h = nullptr, *c = nullptr;
  void* a = nullptr;
  // paired attention: token scales, anchor-side projections and phi(Z0, U)
  float *sC = nullptr, *sH = nullptr, *Z0 = nullptr, *U = nullptr, *phi0 = nullptr;
  void* Ub = nullptr;
  int refresh_i = 0;
};

struct tadm_context {
  tadm_model* model;
  int B, cap, len = 0;
  std::vector<void*> k, vt;  // per layer [B, Hkv, cap, dh] / [B, Hkv, dh, cap]
};

// ---------------------------------------------------------------- profiling ---
// Timing-only events: no system-scope fence when they complete (no cache writeback and
// invalidation between the timed kernels); they are read after the stream has drained.
static tadm_status prof_event(tadm_model* m, hipEvent_t* e) {
  if (m->pool.empty()) {
    HIPCHK(hipEventCreateWithFlags(e, hipEventDisableSystemFence));
  } else {
    *e = m->pool.back();
    m->pool.pop_back();
  }
  return TADM_OK;
}

// A single-kernel stage times its first launch with the launch's own timestamps;
// the other stages bracket their launches with recorded events.
static bool single_kernel_stage(int stage) {
  return stage == TADM_STAGE_HEAD || stage == TADM_STAGE_SAMPLE ||
         (stage >= TADM_STAGE_QKV && stage != TADM_STAGE_SELFCOND);  // split product + reduction
}

// Stages nest (a kernel stage inside a layer stage); each end closes the latest begin.
// multi: a single-kernel stage that this time launches more than one kernel (events
// are recorded around its launches instead)
// The method's parts (S, A, Phi, D, head, sampler, selection, context pass) also open a
// roctx range, so that a trace of the host thread (rocprofv3 --marker-trace) shows where
// each part of a step was enqueued; the per-kernel stages do not.
static const char* range_name(int stage) {
  switch (stage) {
    case TADM_STAGE_EMBED: return "tadm S: shared network";
    case TADM_STAGE_ANCHOR: return "tadm A: anchor network";
    case TADM_STAGE_FUSION: return "tadm Phi: fusion";
    case TADM_STAGE_DENOISE: return "tadm D: denoiser";
    case TADM_STAGE_HEAD: return "tadm head";
    case TADM_STAGE_SAMPLE: return "tadm sampler";
    case TADM_STAGE_SELECT: return "tadm unmask";
    case TADM_STAGE_CONTEXT: return "tadm context pass";
    default: return nullptr;
  }
}

static tadm_status prof_begin(tadm_model* m, int stage, bool multi = false) {
  if (const char* r = range_name(stage)) roctxRangePushA(r);
  if (!((m->prof_mask >> stage) & 1)) return TADM_OK;
  OpenStage o{stage, nullptr, nullptr};
  TRY(prof_event(m, &o.a));
  if (single_kernel_stage(stage) && !multi) {
    TRY(prof_event(m, &o.b));
    next_launch_events = LaunchEvents{o.a, o.b};
  } else {
    HIPCHK(hipEventRecord(o.a, m->stream));
  }
  m->open.push_back(o);
  return TADM_OK;
}

static tadm_status prof_end(tadm_model* m, int stage) {
  if (range_name(stage)) roctxRangePop();
  if (!((m->prof_mask >> stage) & 1) || m->open.empty() || m->open.back().stage != stage) return TADM_OK;
  OpenStage o = m->open.back();
  m->open.pop_back();
  if (o.b) {
    if (next_launch_events.start == o.a) {  // nothing was launched: an empty interval
      next_launch_events = LaunchEvents{};
      HIPCHK(hipEventRecord(o.a, m->stream));
      HIPCHK(hipEventRecord(o.b, m->stream));
    }
  } else {
    TRY(prof_event(m, &o.b));
    HIPCHK(hipEventRecord(o.b, m->stream));
  }
  m->recs.push_back(ProfRec{stage, o.a, o.b});
  return TADM_OK;
}

static tadm_status ws_alloc(tadm_model* m, void** p, size_t bytes) {
  HIPCHK(hipMalloc(p, std::max<size_t>(bytes, 256)));
  m->ws.allocs.push_back(*p);
  return TADM_OK;
}

static tadm_status ensure_workspace(tadm_model* m) {
  Workspace& w = m->ws;
  if (w.n_tok) return TADM_OK;
  const tadm_config& c = m->cfg;
  const size_t N = (size_t)c.max_batch * c.max_seq, d = c.d_model, es = m->esz;
  const size_t H = c.n_heads, Hk = c.n_kv_heads, dh = c.head_dim, F = c.d_ffn;
  w.kv_cap = round64(c.max_seq);
  TRY(ws_alloc(m, (void**)&w.x, N * d * 4));
  TRY(ws_alloc(m, (void**)&w.c, N * d * 4));
  TRY(ws_alloc(m, (void**)&w.ht, N * d * 4));
  TRY(ws_alloc(m, &w.xn, N * d * es));
  TRY(ws_alloc(m, &w.qkv, N * (H + 2 * Hk) * dh * es));
  TRY(ws_alloc(m, &w.q, N * H * dh * es));
  TRY(ws_alloc(m, &w.k, (size_t)c.max_batch * Hk * w.kv_cap * dh * es));
  TRY(ws_alloc(m, &w.vt, (size_t)c.max_batch * Hk * w.kv_cap * dh * es));
  TRY(ws_alloc(m, &w.ao, N * H * dh * es));
  TRY(ws_alloc(m, &w.ffn, N * F * es));
  if (m->dt == F32 && c.ffn_kind != TADM_FFN_GELU) TRY(ws_alloc(m, (void**)&w.ffn_pre, N * 2 * F * 4));
  if (c.fusion_kind == TADM_FUSION_GATED_MLP) {
    TRY(ws_alloc(m, &w.fus_h, N * 4 * d * es));
    TRY(ws_alloc(m, (void**)&w.fus_g, N * d * 4));
  } else {
    const size_t r = c.fusion_rank;
    TRY(ws_alloc(m, (void**)&w.pz, N * r * 4));
    TRY(ws_alloc(m, (void**)&w.pr, N * r * 4));
    TRY(ws_alloc(m, (void**)&w.pgate, N * 4));
    TRY(ws_alloc(m, &w.pzb, N * r * es));
    TRY(ws_alloc(m, &w.pqkv, N * 3 * r * es));
    TRY(ws_alloc(m, &w.prb, N * r * es));
    TRY(ws_alloc(m, &w.pmb, N * r * es));
    TRY(ws_alloc(m, &w.pf, N * 4 * r * es));
    TRY(ws_alloc(m, &w.pg1, N * r * es));
  }
  TRY(ws_alloc(m, (void**)&w.choice, N * 4));
  TRY(ws_alloc(m, (void**)&w.cidx, N * 4));
  TRY(ws_alloc(m, (void**)&w.row_map, N * 4));
  TRY(ws_alloc(m, (void**)&w.count, 256));
  TRY(ws_alloc(m, (void**)&w.conf, N * 4));
  TRY(ws_alloc(m, (void**)&w.nthr, N * sizeof(NucleusThr)));
  TRY(ws_alloc(m, (void**)&w.xhat, N * 4));
  TRY(ws_alloc(m, (void**)&w.hq, N * 8));
  TRY(ws_alloc(m, (void**)&w.rscale, N * 4));
  w.n_tok = (int)N;
  w.n_canvas = (int)N;
  return TADM_OK;
}

static tadm_status ensure_logits(tadm_model* m, size_t n) {
  Workspace& w = m->ws;
  if (w.logits_cap >= n) return TADM_OK;
  if (w.logits) HIPCHK(hipFree(w.logits));
  w.logits = nullptr;
  HIPCHK(hipMalloc((void**)&w.logits, n * 4));
  w.logits_cap = n;
  return TADM_OK;
}

// Workspace of K-slice products (grown on demand).
static tadm_status ensure_kpart(tadm_model* m, size_t floats) {
  Workspace& s = m->ws;
  if (s.kpart_cap >= floats) return TADM_OK;
  if (s.kpart) HIPCHK(hipFree(s.kpart));
  s.kpart = nullptr;
  HIPCHK(hipMalloc((void**)&s.kpart, floats * 4));
  s.kpart_cap = floats;
  return TADM_OK;
}

// --------------------------------------------------------------- the layers ---
struct KVTarget {
  void *k, *vt;
  int cap, off;
};

// One pre-norm layer on x [N, d]; prenormed: ws.xn already holds the attention norm of x.
// next_norm: the attention-norm gains of the layer that follows (nullptr if none); when
// the FFN down product's slice sum can write that norm, it does, and *next_prenormed is
// set.
static tadm_status run_layer(tadm_model* m, int li, float* x, int B, int L, int pos0, KVTarget kv,
                             bool prenormed = false, const float* next_norm = nullptr,
                             bool* next_prenormed = nullptr) {
  const tadm_config& c = m->cfg;
  const LayerIdx& w = m->lay.layers[li];
  Workspace& s = m->ws;
  const int N = B * L, d = c.d_model, H = c.n_heads, Hk = c.n_kv_heads, dh = c.head_dim,
            F = c.d_ffn;
  const hipStream_t st = m->stream;
  // capture slots: 3 li (entering layer li), 3 li + 1 (after its attention half) and
  // 3 li + 2 (leaving it), [N, d] float32 each
  const size_t slot = (size_t)N * d;
  const bool capture = m->layer_cap && (3 * (size_t)li + 3) * slot * 4 <= m->layer_cap_bytes;
  if (capture)
    HIPCHK(hipMemcpyAsync(m->layer_cap + 3 * (size_t)li * slot, x, slot * 4, hipMemcpyDeviceToDevice, st));
  if (!prenormed) HIPCHK(rms_norm(m->dt, x, m->Wf(w.attn_norm), c.rms_eps, N, d, N, 0, 0, s.xn, st));
  if (next_prenormed) *next_prenormed = false;
  bool fused_norm = false;
  {
    // q/k/v projection with the rotary embedding and head split in the epilogue
    GemmProblem p{N, (H + 2 * Hk) * dh, d, s.xn, d, d, nullptr, 0, m->W(w.wqkv), d};
    EpiParams e;
    e.L = L;
    e.pos0 = pos0;
    e.H = H;
    e.Hkv = Hk;
    e.dh = dh;
    e.kv_cap = kv.cap;
    e.kv_off = kv.off;
    e.rope = m->rope;
    e.q = s.q;
    e.k = kv.k;
    e.vt = kv.vt;
    TRY(prof_begin(m, TADM_STAGE_QKV));
    HIPCHK(gemm(m->dt, p, EPI_QKV_ROPE, e, st));
    TRY(prof_end(m, TADM_STAGE_QKV));
  }
  TRY(prof_begin(m, TADM_STAGE_ATTN));
  HIPCHK(attention(m->dt, s.q, kv.k, kv.vt, s.ao, B, H, Hk, L, kv.off + L, kv.cap, dh, st));
  TRY(prof_end(m, TADM_STAGE_ATTN));
  {
    GemmProblem p{N, d, H * dh, s.ao, H * dh, H * dh, nullptr, 0, m->W(w.wo), H * dh};
    EpiParams e;
    e.resid = x;
    e.ldr = d;
    const int S = m->dt == BF16 ? gemm_resid_slices(N, d, H * dh) : 1;
    fused_norm = m->dt == BF16 && gemm_resid_norms(N, d, H * dh);
    if (S > 1) {
      TRY(ensure_kpart(m, (size_t)S * N * d));
      e.part = s.kpart;
    }
    if (fused_norm) {  // the slice sum writes the FFN norm of the updated rows
      e.norm_g = m->Wf(w.ffn_norm);
      e.norm_eps = c.rms_eps;
      e.norm_out = s.xn;
    }
    TRY(prof_begin(m, TADM_STAGE_OPROJ, S > 1));
    HIPCHK(gemm(m->dt, p, EPI_RESID, e, st));
    TRY(prof_end(m, TADM_STAGE_OPROJ));
  }
  if (capture)
    HIPCHK(hipMemcpyAsync(m->layer_cap + (3 * (size_t)li + 1) * slot, x, slot * 4, hipMemcpyDeviceToDevice, st));
  if (!fused_norm) HIPCHK(rms_norm(m->dt, x, m->Wf(w.ffn_norm), c.rms_eps, N, d, N, 0, 0, s.xn, st));
  TRY(prof_begin(m, TADM_STAGE_FFN_UP));
  if (c.ffn_kind == TADM_FFN_GELU) {
    GemmProblem p{N, F, d, s.xn, d, d, nullptr, 0, m->W(w.wup), d};
    EpiParams e;
    e.out = s.ffn;
    e.ldo = F;
    HIPCHK(gemm(m->dt, p, EPI_GELU, e, st));
  } else if (m->dt == BF16) {
    GemmProblem p{N, 2 * F, d, s.xn, d, d, nullptr, 0, m->W(w.wup), d};
    EpiParams e;
    e.out = s.ffn;
    e.ldo = F;
    HIPCHK(gemm(m->dt, p, c.ffn_kind == TADM_FFN_SWIGLU ? EPI_GLU_SILU : EPI_GLU_GELU, e, st));
  } else {
    GemmProblem p{N, 2 * F, d, s.xn, d, d, nullptr, 0, m->W(w.wup), d};
    EpiParams e;
    e.out = s.ffn_pre;
    e.ldo = 2 * F;
    HIPCHK(gemm(m->dt, p, EPI_STORE_F32, e, st));
    HIPCHK(glu_f32(s.ffn_pre, N, F, c.ffn_kind == TADM_FFN_SWIGLU, (float*)s.ffn, st));
  }
  TRY(prof_end(m, TADM_STAGE_FFN_UP));
  {
    GemmProblem p{N, d, F, s.ffn, F, F, nullptr, 0, m->W(w.wdown), F};
    EpiParams e;
    e.resid = x;
    e.ldr = d;
    const int S = m->dt == BF16 ? gemm_resid_slices(N, d, F) : 1;
    if (S > 1) {
      TRY(ensure_kpart(m, (size_t)S * N * d));
      e.part = s.kpart;
    }
    if (next_norm && next_prenormed && m->dt == BF16 && gemm_resid_norms(N, d, F)) {
      e.norm_g = next_norm;  // the slice sum writes the next layer's attention norm
      e.norm_eps = c.rms_eps;
      e.norm_out = s.xn;
      *next_prenormed = true;
    }
    TRY(prof_begin(m, TADM_STAGE_FFN_DOWN, S > 1));
    HIPCHK(gemm(m->dt, p, EPI_RESID, e, st));
    TRY(prof_end(m, TADM_STAGE_FFN_DOWN));
  }
  if (capture)
    HIPCHK(hipMemcpyAsync(m->layer_cap + (3 * (size_t)li + 2) * slot, x, slot * 4, hipMemcpyDeviceToDevice, st));
  return TADM_OK;
}

static KVTarget kv_target(tadm_model* m, const tadm_context* ctx, int li) {
  if (ctx) return KVTarget{ctx->k[li], ctx->vt[li], ctx->cap, ctx->len};
  return KVTarget{m->ws.k, m->ws.vt, m->ws.kv_cap, 0};
}

// prenormed: ws.xn already holds the first layer's attention norm of x
static tadm_status run_part(tadm_model* m, int first, int count, float* x, int B, int L, int pos0,
                            const tadm_context* ctx, bool prenormed = false) {
  bool pre = prenormed;
  for (int li = first; li < first + count; ++li) {
    const float* next_norm = li + 1 < first + count ? m->Wf(m->lay.layers[li + 1].attn_norm) : nullptr;
    bool next_pre = false;
    TRY(run_layer(m, li, x, B, L, pos0, kv_target(m, ctx, li), pre, next_norm, &next_pre));
    pre = next_pre;
  }
  return TADM_OK;
}

// c = S(z): embedding gather (plus the self-conditioning signal sc on the columns
// [off, L), if given) then the shared layers (in place on `c`).
static tadm_status shared_net(tadm_model* m, const tadm_context* ctx, const int32_t* z, int B, int L,
                              float* c, const float* sc = nullptr, int off = 0) {
  const int pos0 = ctx ? ctx->len : 0;
  HIPCHK(embed_gather(m->dt, z, B * L, m->W(m->lay.embed), m->cfg.vocab + 1, m->cfg.d_model, c,
                      m->stream));
  if (sc) HIPCHK(add_selfcond(c, sc, B, L, off, m->cfg.d_model, m->stream));
  return run_part(m, 0, m->cfg.n_shared, c, B, L, pos0, ctx);
}

// ---------------------------------------------------- paired-attention fusion
// phi(Z, U) = R + SiLU(R W_1) W_2 with R = Z + MHA(J W_Q, J W_K, J W_V) W_O, J = [Z, U],
// the attention bidirectional over the L positions of each row (App. C.1).  With
// phi0 == nullptr the result goes to cache->phi0 (refresh); otherwise M = phi - phi0 is
// written to ws.pmb in the model type.
static tadm_status paired_mixer(tadm_model* m, int B, int L, const float* Zf, const void* Zb,
                                tadm_cache* cache, bool to_phi0) {
  const tadm_config& cf = m->cfg;
  Workspace& s = m->ws;
  const Layout& Y = m->lay;
  const int N = B * L, r = cf.fusion_rank, nh = cf.paired_heads, dh = r / nh;
  const hipStream_t st = m->stream;
  {
    GemmProblem p{N, 3 * r, 2 * r, Zb, r, r, cache->Ub, r, m->W(Y.p_wqkv), 2 * r};
    EpiParams e;
    e.out = s.pqkv;
    e.ldo = 3 * r;
    HIPCHK(gemm(m->dt, p, EPI_STORE, e, st));
  }
  HIPCHK(rope_split(m->dt, s.pqkv, B, L, nh, nh, dh, 0, nullptr, nullptr, s.q, s.k, s.vt, s.kv_cap, 0, st));
  HIPCHK(attention(m->dt, s.q, s.k, s.vt, s.ao, B, nh, nh, L, L, s.kv_cap, dh, st));
  {
    GemmProblem p{N, r, r, s.ao, r, r, nullptr, 0, m->W(Y.p_wo), r};
    EpiParams e;
    e.out = s.pr;
    e.ldo = r;
    e.aux = Zf;
    e.ld_aux = r;
    e.out_t = s.prb;
    e.ld_out_t = r;
    HIPCHK(gemm(m->dt, p, EPI_ADD_BOTH, e, st));
  }
  {
    GemmProblem p{N, 2 * r, r, s.prb, r, r, nullptr, 0, m->W(Y.p_w1), r};
    EpiParams e;
    e.out = s.ffn;
    e.ldo = 2 * r;
    HIPCHK(gemm(m->dt, p, EPI_SILU, e, st));
  }
  {
    GemmProblem p{N, r, 2 * r, s.ffn, 2 * r, 2 * r, nullptr, 0, m->W(Y.p_w2), 2 * r};
    EpiParams e;
    e.aux = s.pr;
    e.ld_aux = r;
    if (to_phi0) {
      e.out = cache->phi0;
      e.ldo = r;
      HIPCHK(gemm(m->dt, p, EPI_ADD_F32, e, st));
    } else {
      e.aux2 = cache->phi0;
      e.ld_aux2 = r;
      e.out_t = s.pmb;
      e.ld_out_t = r;
      HIPCHK(gemm(m->dt, p, EPI_ADD_SUB, e, st));
    }
  }
  return TADM_OK;
}

// Z = (C / s_C) W_C into ws.pz (float) and ws.pzb (model type).
static tadm_status paired_project(tadm_model* m, int N, const float* C, const float* sC, float* Zf, void* Zb) {
  const tadm_config& cf = m->cfg;
  Workspace& s = m->ws;
  const int d = cf.d_model, r = cf.fusion_rank;
  HIPCHK(scale_rows(m->dt, C, sC, N, d, s.xn, m->stream));
  GemmProblem p{N, r, d, s.xn, d, d, nullptr, 0, m->W(m->lay.p_wc), d};
  EpiParams e;
  e.out = Zf;
  e.ldo = r;
  HIPCHK(gemm(m->dt, p, EPI_STORE_F32, e, m->stream));
  HIPCHK(to_type(m->dt, Zf, (size_t)N * r, Zb, m->stream));
  return TADM_OK;
}

// Refresh: token scales of C0 and H0, Z0, U and phi(Z0, U) into the cache.
static tadm_status paired_prepare(tadm_model* m, int B, int L, tadm_cache* cache) {
  const tadm_config& cf = m->cfg;
  Workspace& s = m->ws;
  const int N = B * L, d = cf.d_model, r = cf.fusion_rank;
  const hipStream_t st = m->stream;
  HIPCHK(row_rms(cache->c, N, d, cf.rms_eps, cache->sC, st));
  HIPCHK(row_rms(cache->h, N, d, cf.rms_eps, cache->sH, st));
  HIPCHK(scale_rows(m->dt, cache->h, cache->sH, N, d, s.xn, st));
  {
    GemmProblem p{N, r, d, s.xn, d, d, nullptr, 0, m->W(m->lay.p_wh), d};
    EpiParams e;
    e.out = cache->U;
    e.ldo = r;
    HIPCHK(gemm(m->dt, p, EPI_STORE_F32, e, st));
  }
  HIPCHK(to_type(m->dt, cache->U, (size_t)N * r, cache->Ub, st));
  TRY(paired_project(m, N, cache->c, cache->sC, cache->Z0, s.pzb));
  return paired_mixer(m, B, L, cache->Z0, s.pzb, cache, true);
}

// Step: H~ = H0 + g * s_H * (M W_up) into ws.x.
static tadm_status paired_fuse(tadm_model* m, int B, int L, const float* c, const tadm_cache* ccache) {
  tadm_cache* cache = const_cast<tadm_cache*>(ccache);  // phi0 is only read here
  const tadm_config& cf = m->cfg;
  Workspace& s = m->ws;
  const Layout& Y = m->lay;
  const int N = B * L, d = cf.d_model, r = cf.fusion_rank;
  const hipStream_t st = m->stream;
  TRY(paired_project(m, N, c, cache->sC, s.pz, s.pzb));
  TRY(paired_mixer(m, B, L, s.pz, s.pzb, cache, false));
  HIPCHK(paired_features(m->dt, cache->U, cache->Z0, s.pz, s.pmb, N, r, s.pf, st));
  {
    GemmProblem p{N, r, 4 * r, s.pf, 4 * r, 4 * r, nullptr, 0, m->W(Y.p_wg1), 4 * r};
    EpiParams e;
    e.out = s.pg1;
    e.ldo = r;
    HIPCHK(gemm(m->dt, p, EPI_SILU, e, st));
  }
  HIPCHK(row_gate(m->dt, s.pg1, m->Wf(Y.p_wg2), m->Wf(Y.p_bg), N, r, s.pgate, st));
  {
    GemmProblem p{N, d, r, s.pmb, r, r, nullptr, 0, m->W(Y.p_wup), r};
    EpiParams e;
    e.out = s.x;
    e.ldo = d;
    e.aux = cache->h;
    e.ld_aux = d;
    e.row1 = s.pgate;
    e.row2 = cache->sH;
    HIPCHK(gemm(m->dt, p, EPI_PAIRED, e, st));
  }
  return TADM_OK;
}

// anchor refresh: h = A(c) into the cache, with the fusion's anchor-side input.
static tadm_status anchor_net(tadm_model* m, const tadm_context* ctx, int B, int L, const float* c,
                              tadm_cache* cache) {
  const tadm_config& cf = m->cfg;
  const size_t n = (size_t)B * L * cf.d_model;
  HIPCHK(copy_f32(c, cache->c, n, m->stream));
  HIPCHK(copy_f32(c, cache->h, n, m->stream));
  TRY(run_part(m, cf.n_shared, cf.n_anchor, cache->h, B, L, ctx ? ctx->len : 0, ctx));
  if (cf.fusion_kind == TADM_FUSION_GATED_MLP)
    HIPCHK(layer_norm(m->dt, cache->h, m->Wf(m->lay.ln_a_w), m->Wf(m->lay.ln_a_b), cf.ln_eps, B * L,
                      cf.d_model, cache->a, nullptr, m->stream));
  else
    TRY(paired_prepare(m, B, L, cache));
  return TADM_OK;
}

// h~ = Phi(c, cache) into ws.x.
// h~ = Phi(c, h') into ws.x.  With the gated MLP fusion and denoiser layers, its closing
// LayerNorm also writes the first denoiser layer's attention norm to ws.xn (*prenormed).
static tadm_status fusion(tadm_model* m, int B, int L, const float* c, const tadm_cache* cache,
                          bool* prenormed) {
  const tadm_config& cf = m->cfg;
  *prenormed = false;
  if (cf.fusion_kind == TADM_FUSION_PAIRED) return paired_fuse(m, B, L, c, cache);
  Workspace& s = m->ws;
  const int N = B * L, d = cf.d_model;
  const Layout& Y = m->lay;
  const hipStream_t st = m->stream;
  HIPCHK(layer_norm(m->dt, c, m->Wf(Y.ln_s_w), m->Wf(Y.ln_s_b), cf.ln_eps, N, d, s.xn, nullptr, st));
  {
    GemmProblem p{N, 5 * d, 2 * d, s.xn, d, d, cache->a, d, m->W(Y.w1g), 2 * d};
    EpiParams e;
    e.out = s.fus_h;
    e.ldo = 4 * d;
    e.bias = m->Wf(Y.b1g);
    e.out2 = s.fus_g;
    e.ldo2 = d;
    e.split = 4 * d;
    TRY(prof_begin(m, TADM_STAGE_FUSION1));
    HIPCHK(gemm(m->dt, p, EPI_FUSION1, e, st));
    TRY(prof_end(m, TADM_STAGE_FUSION1));
  }
  {
    GemmProblem p{N, d, 4 * d, s.fus_h, 4 * d, 4 * d, nullptr, 0, m->W(Y.w2), 4 * d};
    EpiParams e;
    e.resid = s.x;
    e.ldr = d;
    e.bias = m->Wf(Y.b2);
    e.aux = cache->h;
    e.ld_aux = d;
    e.gate = s.fus_g;
    e.ldg = d;
    TRY(prof_begin(m, TADM_STAGE_FUSION2));
    HIPCHK(gemm(m->dt, p, EPI_FUSION2, e, st));
    TRY(prof_end(m, TADM_STAGE_FUSION2));
  }
  if (cf.n_denoise > 0) {
    const float* g0 = m->Wf(Y.layers[cf.n_shared + cf.n_anchor].attn_norm);
    HIPCHK(layer_rms_norm(m->dt, s.x, m->Wf(Y.ln_o_w), m->Wf(Y.ln_o_b), cf.ln_eps, g0, cf.rms_eps, N, d, s.xn, st));
    *prenormed = true;
  } else {
    HIPCHK(layer_norm(m->dt, s.x, m->Wf(Y.ln_o_w), m->Wf(Y.ln_o_b), cf.ln_eps, N, d, nullptr, s.x, st));
  }
  return TADM_OK;
}

// ------------------------------------------------------------- validation -----
static tadm_status check_model(const tadm_model* m) {
  if (!m) return fail(TADM_ERR_INVALID, "null model");
  for (size_t i = 0; i < m->loaded.size(); ++i)
    if (!m->loaded[i]) return fail(TADM_ERR_STATE, "weight %zu (%s) not loaded", i, m->lay.specs[i].name.c_str());
  return TADM_OK;
}

static tadm_status check_window(const tadm_model* m, const tadm_context* ctx, int B, int L) {
  if (B < 1 || B > m->cfg.max_batch) return fail(TADM_ERR_INVALID, "B=%d outside [1, %d]", B, m->cfg.max_batch);
  const int pos0 = ctx ? ctx->len : 0;
  if (L < 1 || pos0 + L > m->cfg.max_seq)
    return fail(TADM_ERR_INVALID, "positions [%d, %d) exceed max_seq %d", pos0, pos0 + L, m->cfg.max_seq);
  if (ctx) {
    if (ctx->model != m) return fail(TADM_ERR_STATE, "context belongs to another model");
    if (ctx->B != B) return fail(TADM_ERR_STATE, "context has B=%d, call has B=%d", ctx->B, B);
    if (ctx->len + L > ctx->cap) return fail(TADM_ERR_INVALID, "context capacity %d too small", ctx->cap);
  }
  if (m->dt == F32 && ctx == nullptr && L > 4096) return fail(TADM_ERR_UNSUPPORTED, "fp32 attention limited to 4096 keys");
  return TADM_OK;
}

static tadm_status check_args(const tadm_step_args* a, int Lc) {
  if (!a) return fail(TADM_ERR_INVALID, "null step args");
  if (a->T < 1 || a->i < 1 || a->i > a->T) return fail(TADM_ERR_INVALID, "step i=%d T=%d", a->i, a->T);
  if (a->n_unmask < 0) return fail(TADM_ERR_INVALID, "negative n_unmask");
  if (!(a->inv_temp > 0) || !std::isfinite(a->inv_temp)) return fail(TADM_ERR_INVALID, "inv_temp must be finite and > 0");
  if (a->mode != TADM_STEP_RANKED && a->mode != TADM_STEP_REMASK && a->mode != TADM_STEP_ENTROPY)
    return fail(TADM_ERR_INVALID, "step mode %d", a->mode);
  if (a->mode == TADM_STEP_ENTROPY) {
    if (!(a->entropy_eta >= 0.f) || !std::isfinite(a->entropy_eta))
      return fail(TADM_ERR_INVALID, "entropy bound must be finite and >= 0");
    if (a->top_p > 0.f && a->top_p < 1.f) return fail(TADM_ERR_UNSUPPORTED, "the entropy-bound sampler has no nucleus");
    if (Lc > ENTROPY_MAX_CANVAS) return fail(TADM_ERR_UNSUPPORTED, "entropy sampler canvas %d > %d", Lc, ENTROPY_MAX_CANVAS);
  }
  if (a->mode == TADM_STEP_REMASK && !(a->p_unmask >= 0.f && a->p_unmask <= 1.f && a->sigma >= 0.f && a->sigma <= 1.f))
    return fail(TADM_ERR_INVALID, "remasking probabilities must lie in [0, 1]");
  if (!(a->top_p >= 0.f && a->top_p <= 1.f)) return fail(TADM_ERR_INVALID, "top_p outside [0, 1]");
  (void)Lc;
  return TADM_OK;
}

// The step's canvas update from the sampled tokens: confidence-ranked unmasking or the
// remasking posterior.
static tadm_status canvas_update(tadm_model* m, const int32_t* canvas, const int32_t* choice, const float* conf,
                                 int B, int L, int off, int pos0, const tadm_step_args* a, int32_t* next) {
  TRY(prof_begin(m, TADM_STAGE_SELECT));
  if (a->mode == TADM_STEP_REMASK)
    HIPCHK(remask_update(canvas, choice, B, L, off, m->cfg.vocab, pos0, a->step_id, a->seed, a->p_unmask, a->sigma,
                         next, m->stream));
  else
    HIPCHK(select_unmask(canvas, choice, conf, B, L, off, m->cfg.vocab, a->n_unmask, a->n_unmask_rows, next,
                         m->stream));
  TRY(prof_end(m, TADM_STAGE_SELECT));
  return TADM_OK;
}

// ------------------------------------------------- allocation-free sampler ---
// Fixed device array of tadm_sample_noalloc: per canvas position the sampled token
// (int32) and confidence (float32), then the nucleus thresholds.  In host code the
// array's name stands for a host-side shadow, not a device address: the device copy
// of each GPU is reached only through the address hipGetSymbolAddress returns with
// that GPU current, kept per device below.
namespace {
constexpr size_t kNoAllocChoice = 0;
constexpr size_t kNoAllocConf = kNoAllocChoice + (size_t)TADM_NOALLOC_MAX_POSITIONS * sizeof(int32_t);
constexpr size_t kNoAllocThr = align_up_const(kNoAllocConf + (size_t)TADM_NOALLOC_MAX_POSITIONS * sizeof(float));
constexpr size_t kNoAllocBytes = kNoAllocThr + (size_t)TADM_NOALLOC_MAX_POSITIONS * sizeof(NucleusThr);
constexpr int kMaxDevices = 64;
}  // namespace

static __device__ __align__(256) char scratch[kNoAllocBytes];
static std::mutex g_scratch_mutex;
static char* g_scratch_dev[kMaxDevices] = {};

// Device address of `scratch` on `device`, looked up once per device with it current.
static tadm_status noalloc_scratch(int device, char** out) {
  if (device < 0 || device >= kMaxDevices) return fail(TADM_ERR_UNSUPPORTED, "device %d", device);
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (!g_scratch_dev[device]) {
    int prev = -1;
    hipError_t e = hipGetDevice(&prev);
    if (e == hipSuccess && prev != device) e = hipSetDevice(device);
    void* ptr = nullptr;
    if (e == hipSuccess) e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (prev >= 0 && prev != device) (void)hipSetDevice(prev);
    if (e != hipSuccess || !ptr)
      return fail(TADM_ERR_DEVICE, "scratch address on device %d: %s", device, hipGetErrorString(e));
    g_scratch_dev[device] = static_cast<char*>(ptr);
  }
  *out = g_scratch_dev[device];
  return TADM_OK;
}

// ============================================================== C ABI =========
extern "C" {

const char* tadm_last_error(void) { return g_err.c_str(); }

int32_t tadm_unmask_count(int32_t M0, int32_t i, int32_t T) {
  if (T < 1 || i < 1 || i > T || M0 < 0) return 0;
  return (int32_t)(((int64_t)M0 * i) / T - ((int64_t)M0 * (i - 1)) / T);
}

int32_t tadm_weight_count(const tadm_config* cfg) {
  std::string why;
  if (!valid_config(cfg, why)) return -1;
  return (int32_t)make_layout(*cfg).specs.size();
}

tadm_status tadm_weight_info(const tadm_config* cfg, int32_t index, int64_t* rows, int64_t* cols) {
  std::string why;
  if (!valid_config(cfg, why)) return fail(TADM_ERR_INVALID, "config: %s", why.c_str());
  Layout L = make_layout(*cfg);
  if (index < 0 || index >= (int32_t)L.specs.size() || !rows || !cols)
    return fail(TADM_ERR_INVALID, "weight index %d", index);
  *rows = L.specs[index].rows;
  *cols = L.specs[index].cols;
  return TADM_OK;
}

tadm_status tadm_model_create(const tadm_config* cfg, tadm_model** out) {
  std::string why;
  if (!out) return fail(TADM_ERR_INVALID, "null output pointer");
  *out = nullptr;
  if (!valid_config(cfg, why)) return fail(TADM_ERR_INVALID, "config: %s", why.c_str());
  if (cfg->dtype == TADM_DTYPE_BF16) {
    const int ks[] = {cfg->d_model, cfg->n_heads * cfg->head_dim, cfg->d_ffn,
                      cfg->fusion_kind == TADM_FUSION_PAIRED ? cfg->fusion_rank : 64};
    for (int k : ks)
      if (k % 64) return fail(TADM_ERR_UNSUPPORTED, "bf16 contractions need K %% 64 == 0 (got %d)", k);
    if (cfg->fusion_kind == TADM_FUSION_PAIRED && cfg->fusion_rank / cfg->paired_heads != 64 &&
        cfg->fusion_rank / cfg->paired_heads != 128)
      return fail(TADM_ERR_UNSUPPORTED, "bf16 paired attention needs heads of width 64 or 128");
    if (cfg->head_dim != 64 && cfg->head_dim != 128)
      return fail(TADM_ERR_UNSUPPORTED, "bf16 attention supports head_dim 64 or 128");
  } else if (cfg->head_dim > 128 || cfg->max_seq > 4096) {
    return fail(TADM_ERR_UNSUPPORTED, "fp32 models support head_dim <= 128 and max_seq <= 4096");
  }
  tadm_model* m = new tadm_model();
  m->cfg = *cfg;
  m->dt = cfg->dtype == TADM_DTYPE_BF16 ? BF16 : F32;
  m->esz = m->dt == BF16 ? 2 : 4;
  m->lay = make_layout(*cfg);
  finish_layout(m->lay, m->esz);
  m->loaded.assign(m->lay.specs.size(), 0);
  hipError_t e = hipGetDevice(&m->device);
  if (e == hipSuccess) e = hipMalloc((void**)&m->arena, m->lay.bytes);
  if (e != hipSuccess) {
    const size_t bytes = m->lay.bytes;
    delete m;
    return fail(e == hipErrorOutOfMemory ? TADM_ERR_OOM : TADM_ERR_DEVICE, "weight arena (%zu bytes): %s",
                bytes, hipGetErrorString(e));
  }
  // rotary table [max_seq, dh/2, (cos, sin)], angles in double precision; the pairs of
  // one position are interleaved so that one 16-byte load fetches two rotary pairs
  const int half = cfg->head_dim / 2;
  std::vector<float> cs((size_t)cfg->max_seq * half * 2);
  for (int p = 0; p < cfg->max_seq; ++p)
    for (int j = 0; j < half; ++j) {
      const double ang = p * std::pow((double)cfg->rope_theta, -2.0 * j / cfg->head_dim);
      cs[((size_t)p * half + j) * 2] = (float)std::cos(ang);
      cs[((size_t)p * half + j) * 2 + 1] = (float)std::sin(ang);
    }
  e = hipMalloc((void**)&m->rope, cs.size() * 4);
  if (e == hipSuccess) e = hipMemcpy(m->rope, cs.data(), cs.size() * 4, hipMemcpyHostToDevice);
  if (e != hipSuccess) {
    tadm_model_destroy(m);
    return fail(TADM_ERR_DEVICE, "rope tables: %s", hipGetErrorString(e));
  }
  *out = m;
  return TADM_OK;
}

tadm_status tadm_model_load_weight(tadm_model* m, int32_t index, const void* src, size_t bytes,
                                   int32_t src_on_device) {
  if (!m || !src) return fail(TADM_ERR_INVALID, "null model or source");
  if (index < 0 || index >= (int32_t)m->lay.specs.size()) return fail(TADM_ERR_INVALID, "weight index %d", index);
  const Spec& sp = m->lay.specs[index];
  const long cols = sp.cols ? sp.cols : 1;
  const size_t want = (size_t)sp.rows * cols * m->esz;
  if (bytes != want)
    return fail(TADM_ERR_INVALID, "weight %d (%s): %zu bytes given, %zu expected", index, sp.name.c_str(), bytes, want);
  const void* dsrc = src;
  void* staging = nullptr;
  if (!src_on_device) {
    HIPCHK(hipMalloc(&staging, bytes));
    hipError_t e = hipMemcpy(staging, src, bytes, hipMemcpyHostToDevice);
    if (e != hipSuccess) {
      (void)hipFree(staging);
      return fail(TADM_ERR_DEVICE, "weight upload: %s", hipGetErrorString(e));
    }
    dsrc = staging;
  }
  const Tensor& t = m->lay.tensors[sp.target];
  hipError_t e = scatter_rows(m->dt, dsrc, sp.rows, (int)cols, m->W(sp.target), t.f32 ? 1 : 0, sp.row_off,
                              sp.place == P_GLU ? sp.glu_half : -1, sp.rope_dh, nullptr);
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (staging) (void)hipFree(staging);
  if (e != hipSuccess) return fail(TADM_ERR_DEVICE, "weight placement: %s", hipGetErrorString(e));
  m->loaded[index] = 1;
  if (sp.target == m->lay.embed) m->embT_valid = false;
  return TADM_OK;
}

tadm_status tadm_model_destroy(tadm_model* m) {
  if (!m) return fail(TADM_ERR_INVALID, "null model");
  (void)hipDeviceSynchronize();
  if (m->scratch) tadm_cache_destroy(m->scratch);
  if (m->gcache) tadm_cache_destroy(m->gcache);
  if (m->tcache) tadm_cache_destroy(m->tcache);
  if (m->ws.zt) (void)hipFree(m->ws.zt);
  if (m->ws.zs) (void)hipFree(m->ws.zs);
  if (m->ws.ce) (void)hipFree(m->ws.ce);
  if (m->gctx) tadm_context_destroy(m->gctx);
  if (m->gwin) (void)hipFree(m->gwin);
  if (m->embT) (void)hipFree(m->embT);
  if (m->ws.pw) (void)hipFree(m->ws.pw);
  if (m->ws.kpart) (void)hipFree(m->ws.kpart);
  if (m->ws.sc) (void)hipFree(m->ws.sc);
  for (void* p : m->ws.allocs) (void)hipFree(p);
  if (m->ws.logits) (void)hipFree(m->ws.logits);
  if (m->arena) (void)hipFree(m->arena);
  if (m->rope) (void)hipFree(m->rope);
  next_launch_events = LaunchEvents{};
  for (auto& o : m->open) {
    (void)hipEventDestroy(o.a);
    if (o.b) (void)hipEventDestroy(o.b);
  }
  for (auto& r : m->recs) {
    (void)hipEventDestroy(r.a);
    (void)hipEventDestroy(r.b);
  }
  for (auto e : m->pool) (void)hipEventDestroy(e);
  delete m;
  return TADM_OK;
}

tadm_status tadm_set_stream(tadm_model* m, void* hip_stream) {
  if (!m) return fail(TADM_ERR_INVALID, "null model");
  m->stream = static_cast<hipStream_t>(hip_stream);
  return TADM_OK;
}

// ------------------------------------------------------------------ cache ---
}  // extern "C"

static tadm_status cache_alloc(tadm_model* m, int B, int L, tadm_cache** out) {
  tadm_cache* c = new tadm_cache();
  c->model = m;
  c->B = B;
  c->L = L;
  const size_t n = (size_t)B * L * m->cfg.d_model;
  hipError_t e = hipMalloc((void**)&c->h, n * 4);
  if (e == hipSuccess) e = hipMalloc((void**)&c->c, n * 4);
  if (e == hipSuccess) e = hipMalloc(&c->a, n * m->esz);
  if (e == hipSuccess && m->cfg.fusion_kind == TADM_FUSION_PAIRED) {
    const size_t rows = (size_t)B * L, r = m->cfg.fusion_rank;
    e = hipMalloc((void**)&c->sC, rows * 4);
    if (e == hipSuccess) e = hipMalloc((void**)&c->sH, rows * 4);
    if (e == hipSuccess) e = hipMalloc((void**)&c->Z0, rows * r * 4);
    if (e == hipSuccess) e = hipMalloc((void**)&c->U, rows * r * 4);
    if (e == hipSuccess) e = hipMalloc((void**)&c->phi0, rows * r * 4);
    if (e == hipSuccess) e = hipMalloc(&c->Ub, rows * r * m->esz);
  }
  if (e != hipSuccess) {
    tadm_cache_destroy(c);
    return fail(e == hipErrorOutOfMemory ? TADM_ERR_OOM : TADM_ERR_DEVICE, "cache: %s", hipGetErrorString(e));
  }
  *out = c;
  return TADM_OK;
}

extern "C" {

tadm_status tadm_cache_create(tadm_model* m, int32_t B, int32_t L, tadm_cache** out) {
  if (!m || !out) return fail(TADM_ERR_INVALID, "null argument");
  *out = nullptr;
  if (B < 1 || B > m->cfg.max_batch || L < 1 || L > m->cfg.max_seq)
    return fail(TADM_ERR_INVALID, "cache shape B=%d L=%d outside the model limits", B, L);
  return cache_alloc(m, B, L, out);
}

tadm_status tadm_cache_destroy(tadm_cache* c) {
  if (!c) return fail(TADM_ERR_INVALID, "null cache");
  (void)hipDeviceSynchronize();
  for (void* p : {(void*)c->h, (void*)c->c, c->a, (void*)c->sC, (void*)c->sH, (void*)c->Z0, (void*)c->U,
                  (void*)c->phi0, c->Ub})
    if (p) (void)hipFree(p);
  delete c;
  return TADM_OK;
}

tadm_status tadm_cache_read(const tadm_cache* c, int32_t field, void* dst_dev, size_t bytes) {
  if (!c || !dst_dev) return fail(TADM_ERR_INVALID, "null argument");
  const size_t n = (size_t)c->B * c->L * c->model->cfg.d_model;
  const void* src;
  size_t sz;
  switch (field) {
    case TADM_CACHE_H: src = c->h; sz = n * 4; break;
    case TADM_CACHE_C: src = c->c; sz = n * 4; break;
    case TADM_CACHE_A: src = c->a; sz = n * c->model->esz; break;
    default: return fail(TADM_ERR_INVALID, "cache field %d", field);
  }
  if (bytes != sz) return fail(TADM_ERR_INVALID, "cache field %d has %zu bytes, %zu requested", field, sz, bytes);
  HIPCHK(hipMemcpyAsync(dst_dev, src, sz, hipMemcpyDeviceToDevice, c->model->stream));
  return TADM_OK;
}

int32_t tadm_cache_refresh_step(const tadm_cache* c) { return c ? c->refresh_i : 0; }

// ---------------------------------------------------------------- context ---
tadm_status tadm_context_create(tadm_model* m, int32_t B, int32_t max_ctx, tadm_context** out) {
  if (!m || !out) return fail(TADM_ERR_INVALID, "null argument");
  *out = nullptr;
  if (B < 1 || B > m->cfg.max_batch || max_ctx < 1 || max_ctx > m->cfg.max_seq)
    return fail(TADM_ERR_INVALID, "context shape B=%d max_ctx=%d outside the model limits", B, max_ctx);
  tadm_context* x = new tadm_context();
  x->model = m;
  x->B = B;
  x->cap = round64(max_ctx);
  const size_t per = (size_t)B * m->cfg.n_kv_heads * x->cap * m->cfg.head_dim * m->esz;
  for (int li = 0; li < m->n_layers(); ++li) {
    void *k = nullptr, *v = nullptr;
    hipError_t e = hipMalloc(&k, per);
    if (e == hipSuccess) e = hipMalloc(&v, per);
    if (e != hipSuccess) {
      if (k) (void)hipFree(k);
      tadm_context_destroy(x);
      return fail(e == hipErrorOutOfMemory ? TADM_ERR_OOM : TADM_ERR_DEVICE, "context: %s", hipGetErrorString(e));
    }
    x->k.push_back(k);
    x->vt.push_back(v);
  }
  *out = x;
  return TADM_OK;
}

int32_t tadm_context_length(const tadm_context* ctx) { return ctx ? ctx->len : 0; }

tadm_status tadm_context_reset(tadm_context* ctx) {
  if (!ctx) return fail(TADM_ERR_INVALID, "null context");
  ctx->len = 0;
  return TADM_OK;
}

tadm_status tadm_context_destroy(tadm_context* ctx) {
  if (!ctx) return fail(TADM_ERR_INVALID, "null context");
  (void)hipDeviceSynchronize();
  for (void* p : ctx->k) (void)hipFree(p);
  for (void* p : ctx->vt) (void)hipFree(p);
  delete ctx;
  return TADM_OK;
}

// Fresh pass over n clean tokens: S, A, Phi(c, fresh h), D; keeps every layer's K, V.
// `scratch` receives the anchor state (capacity at least B x n).
static tadm_status context_append_impl(tadm_model* m, tadm_context* ctx, const int32_t* tok, int B,
                                       int n, tadm_cache* scratch) {
  Workspace& s = m->ws;
  TRY(shared_net(m, ctx, tok, B, n, s.c));
  TRY(anchor_net(m, ctx, B, n, s.c, scratch));
  bool prenormed;
  TRY(fusion(m, B, n, s.c, scratch, &prenormed));
  TRY(run_part(m, m->cfg.n_shared + m->cfg.n_anchor, m->cfg.n_denoise, s.x, B, n, ctx->len, ctx, prenormed));
  ctx->len += n;
  return TADM_OK;
}

static tadm_status ensure_scratch(tadm_model* m) {
  if (!m->scratch) TRY(cache_alloc(m, m->cfg.max_batch, m->cfg.max_seq, &m->scratch));
  return TADM_OK;
}

tadm_status tadm_context_append(tadm_model* m, tadm_context* ctx, const int32_t* tokens_dev, int32_t B,
                                int32_t n) {
  TRY(check_model(m));
  if (!ctx || !tokens_dev) return fail(TADM_ERR_INVALID, "null argument");
  TRY(check_window(m, ctx, B, n));
  TRY(ensure_workspace(m));
  TRY(ensure_scratch(m));
  TRY(prof_begin(m, TADM_STAGE_CONTEXT));
  TRY(context_append_impl(m, ctx, tokens_dev, B, n, m->scratch));
  return prof_end(m, TADM_STAGE_CONTEXT);
}

// ------------------------------------------------------------------ step ----
static tadm_status anchor_impl(tadm_model* m, const tadm_context* ctx, const int32_t* canvas, int B,
                               int L, int i, tadm_cache* cache, const float* sc = nullptr, int off = 0) {
  TRY(prof_begin(m, TADM_STAGE_EMBED));
  TRY(shared_net(m, ctx, canvas, B, L, m->ws.c, sc, off));
  TRY(prof_end(m, TADM_STAGE_EMBED));
  TRY(prof_begin(m, TADM_STAGE_ANCHOR));
  TRY(anchor_net(m, ctx, B, L, m->ws.c, cache));
  TRY(prof_end(m, TADM_STAGE_ANCHOR));
  cache->refresh_i = i;
  return TADM_OK;
}

tadm_status tadm_anchor_forward(tadm_model* m, const tadm_context* ctx, const int32_t* canvas_dev,
                                int32_t B, int32_t L, int32_t i, int32_t T, tadm_cache* cache) {
  TRY(check_model(m));
  if (!canvas_dev || !cache) return fail(TADM_ERR_INVALID, "null argument");
  TRY(check_window(m, ctx, B, L));
  if (T < 1 || i < 1 || i > T) return fail(TADM_ERR_INVALID, "step i=%d T=%d", i, T);
  if (cache->model != m || cache->B != B || cache->L != L)
    return fail(TADM_ERR_STATE, "cache built for another model or shape");
  TRY(ensure_workspace(m));
  return anchor_impl(m, ctx, canvas_dev, B, L, i, cache);
}

tadm_status tadm_anchor_forward_sc(tadm_model* m, const tadm_context* ctx, const int32_t* canvas_dev, int32_t B,
                                   int32_t L, int32_t i, int32_t T, const float* sc_dev, int32_t canvas_off,
                                   tadm_cache* cache) {
  TRY(check_model(m));
  if (!canvas_dev || !cache) return fail(TADM_ERR_INVALID, "null argument");
  TRY(check_window(m, ctx, B, L));
  if (T < 1 || i < 1 || i > T) return fail(TADM_ERR_INVALID, "step i=%d T=%d", i, T);
  if (canvas_off < 0 || canvas_off >= L) return fail(TADM_ERR_INVALID, "canvas_off=%d with L=%d", canvas_off, L);
  if (cache->model != m || cache->B != B || cache->L != L)
    return fail(TADM_ERR_STATE, "cache built for another model or shape");
  TRY(ensure_workspace(m));
  return anchor_impl(m, ctx, canvas_dev, B, L, i, cache, sc_dev, canvas_off);
}

static tadm_status sample_impl(tadm_model* m, const float* logits, const int32_t* row_map,
                               const int32_t* canvas, int B, int L, int off, int pos0,
                               const tadm_step_args* a, int32_t* next, int32_t* choice, float* conf) {
  const int mask = m->cfg.vocab;
  TRY(prof_begin(m, TADM_STAGE_SAMPLE));
  const bool nucleus = a->top_p > 0.f && a->top_p < 1.f;
  if (nucleus)
    HIPCHK(nucleus_thresholds(logits, row_map, canvas, B, L, off, m->cfg.vocab, mask, a->inv_temp, a->top_p,
                              m->ws.nthr, m->stream));
  HIPCHK(sample_tokens(logits, row_map, nucleus ? m->ws.nthr : nullptr, canvas, B, L, off, m->cfg.vocab, mask, pos0,
                       a->step_id, a->seed, a->inv_temp, choice, conf, m->stream));
  TRY(prof_end(m, TADM_STAGE_SAMPLE));
  return canvas_update(m, canvas, choice, conf, B, L, off, pos0, a, next);
}

// Embedding rows [0, V) transposed to [d, round64(V)] (zero padding): the weight operand
// of the self-conditioning product.  Rebuilt after the embedding is reloaded.
static tadm_status ensure_embT(tadm_model* m) {
  if (m->embT_valid) return TADM_OK;
  const int V = m->cfg.vocab, Vp = round64(V), d = m->cfg.d_model;
  if (!m->embT) HIPCHK(hipMalloc(&m->embT, (size_t)d * Vp * m->esz));
  HIPCHK(transpose_rows(m->dt, m->W(m->lay.embed), V, d, m->embT, Vp, m->stream));
  m->embT_valid = true;
  return TADM_OK;
}

// Entropy-bound step (TADM_STEP_ENTROPY) from logits of every canvas row: per-row
// statistics and draws, acceptance and the next canvas, then (sc_out) the
// self-conditioning product s = diag(2^40 / A) e E on the MFMA GEMM.
static tadm_status entropy_impl(tadm_model* m, const float* logits, const int32_t* canvas, int B, int L, int off,
                                int pos0, const tadm_step_args* a, int32_t* next, int32_t* choice, float* conf) {
  Workspace& s = m->ws;
  const int Lc = L - off, V = m->cfg.vocab, Vp = round64(V), d = m->cfg.d_model, rows = B * Lc;
  void* P = nullptr;
  if (a->sc_out) {
    const size_t need = (size_t)rows * Vp * m->esz;
    if (s.pw_cap < need) {
      if (s.pw) HIPCHK(hipFree(s.pw));
      s.pw = nullptr;
      HIPCHK(hipMalloc(&s.pw, need));
      s.pw_cap = need;
    }
    P = s.pw;
    TRY(ensure_embT(m));
  }
  TRY(prof_begin(m, TADM_STAGE_SAMPLE));
  HIPCHK(entropy_stats(logits, B, Lc, V, pos0 + off, a->step_id, a->seed, a->inv_temp, s.xhat, choice, conf, s.hq,
                       s.rscale, m->dt, P, Vp, m->stream));
  TRY(prof_end(m, TADM_STAGE_SAMPLE));
  TRY(prof_begin(m, TADM_STAGE_SELECT));
  const long long etaq = (long long)std::nearbyint((double)a->entropy_eta * 1099511627776.0);
  HIPCHK(entropy_accept(s.hq, s.xhat, choice, canvas, next, B, L, off, pos0 + off, a->step_id, a->seed, V, etaq,
                        a->i == 1 ? 1 : 0, m->stream));
  TRY(prof_end(m, TADM_STAGE_SELECT));
  if (a->sc_out) {
    TRY(prof_begin(m, TADM_STAGE_SELFCOND));
    GemmProblem p{rows, d, Vp, P, Vp, Vp, nullptr, 0, m->embT, Vp};
    EpiParams e;
    e.out = a->sc_out;
    e.ldo = d;
    e.row1 = s.rscale;
    const int S = m->dt == BF16 ? gemm_split_slices(rows, d, Vp) : 1;
    if (S > 1) {
      TRY(ensure_kpart(m, (size_t)S * rows * d));
      e.part = s.kpart;
    }
    HIPCHK(gemm(m->dt, p, EPI_SCALE_F32, e, m->stream));
    TRY(prof_end(m, TADM_STAGE_SELFCOND));
  }
  return TADM_OK;
}

// One reverse step.  With caller logits every canvas row goes through the head;
// otherwise only the masked positions do (carry-over makes the others' logits
// unused), at most max_masked of them (an exact bound the caller guarantees, or B*Lc).
static tadm_status denoise_impl(tadm_model* m, const tadm_context* ctx, const int32_t* canvas, int B,
                                int L, int off, const tadm_cache* cache, const tadm_step_args* a,
                                float* logits, int32_t* next, int max_masked) {
  const tadm_config& cf = m->cfg;
  Workspace& s = m->ws;
  const int pos0 = ctx ? ctx->len : 0, Lc = L - off, d = cf.d_model;
  const bool entropy = a->mode == TADM_STEP_ENTROPY;
  TRY(prof_begin(m, TADM_STAGE_EMBED));
  TRY(shared_net(m, ctx, canvas, B, L, s.c, entropy ? a->sc_in : nullptr, off));
  TRY(prof_end(m, TADM_STAGE_EMBED));
  TRY(prof_begin(m, TADM_STAGE_FUSION));
  bool prenormed;
  TRY(fusion(m, B, L, s.c, cache, &prenormed));
  TRY(prof_end(m, TADM_STAGE_FUSION));
  if (m->taps) HIPCHK(copy_f32(s.x, s.ht, (size_t)B * L * d, m->stream));
  const bool full = logits != nullptr, all_rows = full || entropy;
  const int rows = all_rows ? B * Lc : std::min(max_masked, B * Lc);
  TRY(prof_begin(m, TADM_STAGE_DENOISE));
  TRY(run_part(m, cf.n_shared + cf.n_anchor, cf.n_denoise, s.x, B, L, pos0, ctx, prenormed));
  if (all_rows) {
    HIPCHK(rms_norm(m->dt, s.x, m->Wf(m->lay.final_norm), cf.rms_eps, B * Lc, d, Lc, L, off, s.xn, m->stream));
  } else {
    HIPCHK(compact_masked(canvas, B, L, off, cf.vocab, rows, s.cidx, s.row_map, s.count, m->stream));
    HIPCHK(rms_norm_gather(m->dt, s.x, m->Wf(m->lay.final_norm), cf.rms_eps, s.cidx, s.count, rows, Lc, L,
                           off, d, s.xn, m->stream));
  }
  TRY(prof_end(m, TADM_STAGE_DENOISE));
  m->tap_B = B;
  m->tap_L = L;
  m->tap_Lc = Lc;
  m->tap_final = all_rows;
  // bf16 masked-only head: the sampler runs in the projection's epilogue and only
  // per-(row, 64-entry group) partials reach memory
  // (the nucleus and the entropy-bound sampler need whole rows)
  const bool fused = !all_rows && m->dt == BF16 && !(a->top_p > 0.f && a->top_p < 1.f);
  const int ng = (cf.vocab + 63) / 64;
  if (!full) {
    TRY(ensure_logits(m, fused ? (size_t)B * Lc * ng * (sizeof(SamplePart) / 4) : (size_t)B * Lc * cf.vocab));
    logits = s.logits;
  }
  TRY(prof_begin(m, TADM_STAGE_HEAD));
  {
    GemmProblem p{rows, cf.vocab, d, s.xn, d, d, nullptr, 0, m->W(m->lay.w_out), d};
    if (!all_rows) p.M_dev = s.count;
    EpiParams e;
    if (fused) {
      e.rows_idx = s.cidx;
      e.Lc = Lc;
      e.pos_base = pos0 + off;
      e.n_groups = ng;
      e.step_id = a->step_id;
      e.k0 = (uint32_t)(a->seed & 0xFFFFFFFFu);
      e.k1 = (uint32_t)(a->seed >> 32);
      e.inv_temp = a->inv_temp;
      e.part = s.logits;
      HIPCHK(head_sample(p, e, m->stream));
    } else {
      e.out = logits;
      e.ldo = cf.vocab;
      HIPCHK(gemm(m->dt, p, EPI_STORE_F32, e, m->stream));
    }
  }
  TRY(prof_end(m, TADM_STAGE_HEAD));
  if (entropy) return entropy_impl(m, logits, canvas, B, L, off, pos0, a, next, s.choice, s.conf);
  if (!fused)
    return sample_impl(m, logits, full ? nullptr : s.row_map, canvas, B, L, off, pos0, a, next, s.choice,
                       s.conf);
  TRY(prof_begin(m, TADM_STAGE_SAMPLE));
  HIPCHK(sample_finalize(reinterpret_cast<const SamplePart*>(s.logits), ng, cf.vocab, s.row_map, canvas, B, L, off,
                         cf.vocab, s.choice, s.conf, m->stream));
  TRY(prof_end(m, TADM_STAGE_SAMPLE));
  return canvas_update(m, canvas, s.choice, s.conf, B, L, off, pos0, a, next);
}

tadm_status tadm_denoise_step(tadm_model* m, const tadm_context* ctx, const int32_t* canvas_dev, int32_t B,
                              int32_t L, int32_t canvas_off, const tadm_cache* cache,
                              const tadm_step_args* args, float* logits_dev, int32_t* next_canvas_dev) {
  TRY(check_model(m));
  if (!canvas_dev || !cache || !next_canvas_dev) return fail(TADM_ERR_INVALID, "null argument");
  TRY(check_window(m, ctx, B, L));
  if (canvas_off < 0 || canvas_off >= L) return fail(TADM_ERR_INVALID, "canvas_off=%d with L=%d", canvas_off, L);
  TRY(check_args(args, L - canvas_off));
  if (cache->model != m || cache->B != B || cache->L != L)
    return fail(TADM_ERR_STATE, "cache built for another model or shape");
  if (cache->refresh_i == 0) return fail(TADM_ERR_STATE, "cache was never refreshed");
  if (m->cfg.vocab % 4) return fail(TADM_ERR_UNSUPPORTED, "the vocabulary head needs vocab %% 4 == 0");
  TRY(ensure_workspace(m));
  return denoise_impl(m, ctx, canvas_dev, B, L, canvas_off, cache, args, logits_dev, next_canvas_dev,
                      B * (L - canvas_off));
}

tadm_status tadm_sample(tadm_model* m, const float* logits_dev, const int32_t* canvas_dev, int32_t B, int32_t L,
                        int32_t canvas_off, int32_t pos0, const tadm_step_args* args, int32_t* next_canvas_dev,
                        int32_t* choice_dev, float* conf_dev) {
  if (!m) return fail(TADM_ERR_INVALID, "null model");
  if (!logits_dev || !canvas_dev || !next_canvas_dev) return fail(TADM_ERR_INVALID, "null argument");
  if (B < 1 || B > m->cfg.max_batch || L < 1 || L > m->cfg.max_seq || canvas_off < 0 || canvas_off >= L || pos0 < 0)
    return fail(TADM_ERR_INVALID, "sample shape B=%d L=%d off=%d", B, L, canvas_off);
  TRY(check_args(args, L - canvas_off));
  TRY(ensure_workspace(m));
  if (args->mode == TADM_STEP_ENTROPY)
    return entropy_impl(m, logits_dev, canvas_dev, B, L, canvas_off, pos0, args, next_canvas_dev,
                        choice_dev ? choice_dev : m->ws.choice, conf_dev ? conf_dev : m->ws.conf);
  return sample_impl(m, logits_dev, nullptr, canvas_dev, B, L, canvas_off, pos0, args, next_canvas_dev,
                     choice_dev ? choice_dev : m->ws.choice, conf_dev ? conf_dev : m->ws.conf);
}

tadm_status tadm_sample_noalloc(tadm_model* m, const float* logits_dev, const int32_t* canvas_dev, int32_t B,
                                int32_t L, int32_t canvas_off, int32_t pos0, const tadm_step_args* args,
                                int32_t* next_canvas_dev, int32_t* choice_dev, float* conf_dev) {
  if (!m) return fail(TADM_ERR_INVALID, "null model");
  if (!logits_dev || !canvas_dev || !next_canvas_dev) return fail(TADM_ERR_INVALID, "null argument");
  if (B < 1 || B > m->cfg.max_batch || L < 1 || L > m->cfg.max_seq || canvas_off < 0 || canvas_off >= L || pos0 < 0)
    return fail(TADM_ERR_INVALID, "sample shape B=%d L=%d off=%d", B, L, canvas_off);
  TRY(check_args(args, L - canvas_off));
  if (args->mode == TADM_STEP_ENTROPY) return fail(TADM_ERR_UNSUPPORTED, "entropy mode needs the workspace");
  const long long positions = (long long)B * (L - canvas_off);
  if (positions > TADM_NOALLOC_MAX_POSITIONS)
    return fail(TADM_ERR_INVALID, "%lld canvas positions exceed the %d of the fixed scratch", positions,
                TADM_NOALLOC_MAX_POSITIONS);
  char* base = nullptr;
  TRY(noalloc_scratch(m->device, &base));
  int32_t* choice = choice_dev ? choice_dev : reinterpret_cast<int32_t*>(base + kNoAllocChoice);
  float* conf = conf_dev ? conf_dev : reinterpret_cast<float*>(base + kNoAllocConf);
  NucleusThr* thr = reinterpret_cast<NucleusThr*>(base + kNoAllocThr);
  const int mask = m->cfg.vocab;
  const bool nucleus = args->top_p > 0.f && args->top_p < 1.f;
  if (nucleus)
    HIPCHK(nucleus_thresholds(logits_dev, nullptr, canvas_dev, B, L, canvas_off, m->cfg.vocab, mask, args->inv_temp,
                              args->top_p, thr, m->stream));
  HIPCHK(sample_tokens(logits_dev, nullptr, nucleus ? thr : nullptr, canvas_dev, B, L, canvas_off, m->cfg.vocab, mask,
                       pos0, args->step_id, args->seed, args->inv_temp, choice, conf, m->stream));
  if (args->mode == TADM_STEP_REMASK)
    HIPCHK(remask_update(canvas_dev, choice, B, L, canvas_off, mask, pos0, args->step_id, args->seed, args->p_unmask,
                         args->sigma, next_canvas_dev, m->stream));
  else
    HIPCHK(select_unmask(canvas_dev, choice, conf, B, L, canvas_off, mask, args->n_unmask, args->n_unmask_rows,
                         next_canvas_dev, m->stream));
  return TADM_OK;
}

// --------------------------------------------------------------- generate ---
// Algorithm 1 per block; the model-owned cache, context and window are reused
// across calls, so a warm generation allocates nothing and never synchronises.
void tadm_remask_probs(int32_t i, int32_t T, float eta, float* sigma, float* p_unmask) {
#pragma clang fp contract(off)
  const double a_t = 1.0 - (double)i / T, a_s = 1.0 - (double)(i - 1) / T;
  const double cap = a_t > 0.0 ? (1.0 - a_s) / a_t : INFINITY;
  const double sg = std::min((double)eta, cap);
  if (sigma) *sigma = (float)sg;
  if (p_unmask) *p_unmask = (float)((a_s - (1.0 - sg) * a_t) / (1.0 - a_t));
}

namespace {
// alpha(t) of the ReMDM-Loop schedule: linear 0 -> alpha_on on [t_on, 1], flat on
// [t_off, t_on], linear alpha_on -> 1 on [0, t_off]
double loop_alpha(double t, double t_on, double t_off, double a_on) {
#pragma clang fp contract(off)
  if (t >= t_on) return a_on * (1.0 - t) / (1.0 - t_on);
  if (t >= t_off) return a_on;
  return a_on + (1.0 - a_on) * (t_off - t) / t_off;
}
}  // namespace

void tadm_loop_probs(int32_t i, int32_t T, float eta, double t_on, double t_off, double alpha_on, float* sigma,
                     float* p_unmask) {
#pragma clang fp contract(off)
  const double t = (double)i / T, s = (double)(i - 1) / T;
  const double a_t = loop_alpha(t, t_on, t_off, alpha_on), a_s = loop_alpha(s, t_on, t_off, alpha_on);
  double sg = 0.0;
  if (t <= t_on && s >= t_off) sg = std::min((double)eta, (1.0 - a_s) / a_t);
  if (sigma) *sigma = (float)sg;
  if (p_unmask) *p_unmask = (float)((a_s - (1.0 - sg) * a_t) / (1.0 - a_t));
}

float tadm_entropy_inv_temp(int32_t n, int32_t T, float tau_max, float tau_min) {
#pragma clang fp contract(off)
  const double hi = tau_max, lo = tau_min;
  return (float)(1.0 / (lo + (hi - lo) * n / T));
}

tadm_status tadm_generate(tadm_model* m, const int32_t* prompt_dev, int32_t B, int32_t P, int32_t gen_len,
                          int32_t T, int32_t K, int32_t block_len, uint64_t seed, float temperature,
                          int32_t* tokens_dev) {
  return tadm_generate_sampler(m, prompt_dev, B, P, gen_len, T, K, block_len, seed, temperature, nullptr,
                               tokens_dev);
}

tadm_status tadm_generate_sampler(tadm_model* m, const int32_t* prompt_dev, int32_t B, int32_t P, int32_t gen_len,
                                  int32_t T, int32_t K, int32_t block_len, uint64_t seed, float temperature,
                                  const tadm_sampler* sampler, int32_t* tokens_dev) {
  const bool loop = sampler && sampler->kind == TADM_SAMPLER_LOOP;
  const bool remask = loop || (sampler && sampler->kind == TADM_STEP_REMASK);
  const bool entropy = sampler && sampler->kind == TADM_SAMPLER_ENTROPY;
  if (sampler && sampler->kind != TADM_STEP_RANKED && !remask && !entropy)
    return fail(TADM_ERR_INVALID, "sampler kind %d", sampler->kind);
  if (entropy && !(sampler->eta >= 0.f && std::isfinite(sampler->eta)))
    return fail(TADM_ERR_INVALID, "entropy bound must be finite and >= 0");
  if (entropy && !(sampler->tau_min > 0.f && sampler->tau_min <= sampler->tau_max && std::isfinite(sampler->tau_max)))
    return fail(TADM_ERR_INVALID, "temperatures need 0 < tau_min <= tau_max");
  if (entropy && sampler->top_p > 0.f && sampler->top_p < 1.f)
    return fail(TADM_ERR_UNSUPPORTED, "the entropy-bound sampler has no nucleus");
  if (remask && !(sampler->eta >= 0.f && sampler->eta <= 1.f)) return fail(TADM_ERR_INVALID, "eta outside [0, 1]");
  if (loop && !(0.0 < sampler->t_off && sampler->t_off < sampler->t_on && sampler->t_on < 1.0 &&
                0.0 < sampler->alpha_on && sampler->alpha_on < 1.0))
    return fail(TADM_ERR_INVALID, "loop schedule needs 0 < t_off < t_on < 1 and 0 < alpha_on < 1");
  if (sampler && !(sampler->top_p >= 0.f && sampler->top_p <= 1.f)) return fail(TADM_ERR_INVALID, "top_p outside [0, 1]");
  TRY(check_model(m));
  if (!tokens_dev || (P > 0 && !prompt_dev)) return fail(TADM_ERR_INVALID, "null argument");
  if (B < 1 || B > m->cfg.max_batch) return fail(TADM_ERR_INVALID, "B=%d outside [1, %d]", B, m->cfg.max_batch);
  if (P < 0 || gen_len < 1 || block_len < 1 || gen_len % block_len)
    return fail(TADM_ERR_INVALID, "gen_len=%d must be a positive multiple of block_len=%d", gen_len, block_len);
  if (T < 1 || K < 1) return fail(TADM_ERR_INVALID, "T=%d K=%d", T, K);
  if (!(temperature > 0) || !std::isfinite(temperature)) return fail(TADM_ERR_INVALID, "temperature must be > 0");
  if (P + gen_len > m->cfg.max_seq) return fail(TADM_ERR_INVALID, "P + gen_len exceeds max_seq");
  const bool single = block_len == gen_len;
  if (!single && P < 1) return fail(TADM_ERR_INVALID, "block mode needs a prompt");
  if (m->cfg.vocab % 4) return fail(TADM_ERR_UNSUPPORTED, "the vocabulary head needs vocab %% 4 == 0");
  if (entropy && block_len > ENTROPY_MAX_CANVAS)
    return fail(TADM_ERR_UNSUPPORTED, "entropy sampler canvas %d > %d", block_len, ENTROPY_MAX_CANVAS);
  TRY(ensure_workspace(m));
  if (!m->gcache) TRY(cache_alloc(m, m->cfg.max_batch, m->cfg.max_seq, &m->gcache));
  if (entropy && !m->ws.sc) HIPCHK(hipMalloc((void**)&m->ws.sc, (size_t)m->ws.n_tok * m->cfg.d_model * 4));
  const int L = P + gen_len, mask = m->cfg.vocab;
  tadm_step_args a{};
  a.T = T;
  a.seed = seed;
  a.inv_temp = (float)(1.0 / (double)temperature);
  a.mode = entropy ? TADM_STEP_ENTROPY : remask ? TADM_STEP_REMASK : TADM_STEP_RANKED;
  a.top_p = sampler ? sampler->top_p : 0.f;
  if (entropy) a.entropy_eta = sampler->eta;
  // masked positions entering step i: exactly B floor(M0 i / T) for the ranked sampler;
  // any number up to B M0 under remasking
  auto masked_bound = [&](int M0, int i) { return remask ? B * M0 : (int)(B * (((int64_t)M0 * i) / T)); };
  auto set_step = [&](int M0, int i) {
    a.i = i;
    a.n_unmask = tadm_unmask_count(M0, i, T);
    if (loop)
      tadm_loop_probs(i, T, sampler->eta, sampler->t_on, sampler->t_off, sampler->alpha_on, &a.sigma, &a.p_unmask);
    else if (remask)
      tadm_remask_probs(i, T, sampler->eta, &a.sigma, &a.p_unmask);
    if (entropy) {  // each step reads the previous step's signal and, unless last, writes the next
      a.inv_temp = tadm_entropy_inv_temp(i, T, sampler->tau_max, sampler->tau_min);
      a.sc_in = i == T ? nullptr : m->ws.sc;
      a.sc_out = i > 1 ? m->ws.sc : nullptr;
    }
  };
  HIPCHK(init_canvas(prompt_dev, B, P, gen_len, mask, tokens_dev, m->stream));
  tadm_cache* cache = m->gcache;
  if (single) {
    cache->B = B;
    cache->L = L;
    if (entropy) HIPCHK(init_uniform_tokens(tokens_dev, L, P, B, gen_len, P, 0, seed, m->cfg.vocab, m->stream));
    for (int i = T; i >= 1; --i) {
      set_step(gen_len, i);
      a.step_id = (uint32_t)(T - i);
      if ((T - i) % K == 0) TRY(anchor_impl(m, nullptr, tokens_dev, B, L, i, cache, a.sc_in, P));
      TRY(denoise_impl(m, nullptr, tokens_dev, B, L, P, cache, &a, nullptr, tokens_dev, masked_bound(gen_len, i)));
    }
    return TADM_OK;
  }
  if (!m->gctx) TRY(tadm_context_create(m, m->cfg.max_batch, m->cfg.max_seq, &m->gctx));
  if (!m->gwin) HIPCHK(hipMalloc((void**)&m->gwin, (size_t)m->cfg.max_batch * m->cfg.max_seq * 4));
  TRY(ensure_scratch(m));
  tadm_context* ctx = m->gctx;
  ctx->B = B;  // rows [0, B) of the max_batch-row buffers
  ctx->len = 0;
  cache->B = B;
  cache->L = block_len;
  int32_t* win = m->gwin;
  TRY(prof_begin(m, TADM_STAGE_CONTEXT));
  TRY(context_append_impl(m, ctx, prompt_dev, B, P, m->scratch));
  TRY(prof_end(m, TADM_STAGE_CONTEXT));
  const int nblocks = gen_len / block_len;
  for (int j = 0; j < nblocks; ++j) {
    if (entropy)
      HIPCHK(init_uniform_tokens(win, block_len, 0, B, block_len, P + j * block_len, (uint32_t)j, seed,
                                 m->cfg.vocab, m->stream));
    else
      HIPCHK(fill_i32(win, (size_t)B * block_len, mask, m->stream));
    for (int i = T; i >= 1; --i) {
      set_step(block_len, i);
      a.step_id = (uint32_t)(j * T + (T - i));
      if ((T - i) % K == 0) TRY(anchor_impl(m, ctx, win, B, block_len, i, cache, a.sc_in, 0));
      TRY(denoise_impl(m, ctx, win, B, block_len, 0, cache, &a, nullptr, win, masked_bound(block_len, i)));
    }
    HIPCHK(hipMemcpy2DAsync(tokens_dev + P + j * block_len, (size_t)L * 4, win, (size_t)block_len * 4,
                            (size_t)block_len * 4, B, hipMemcpyDeviceToDevice, m->stream));
    if (j + 1 < nblocks) {
      TRY(prof_begin(m, TADM_STAGE_CONTEXT));
      TRY(context_append_impl(m, ctx, win, B, block_len, m->scratch));
      TRY(prof_end(m, TADM_STAGE_CONTEXT));
    }
  }
  return TADM_OK;
}


// ---------------------------------------------------------------- training ---
namespace {
// Philox4x32-10 on the host (the same rounds as the kernels' and the oracle's)
void philox_host(uint32_t c[4], uint32_t k0, uint32_t k1) {
  for (int r = 0; r < 10; ++r) {
    if (r) {
      k0 += 0x9E3779B9u;
      k1 += 0xBB67AE85u;
    }
    const uint64_t p0 = (uint64_t)0xD2511F53u * c[0], p1 = (uint64_t)0xCD9E8D57u * c[2];
    const uint32_t n0 = (uint32_t)(p1 >> 32) ^ c[1] ^ k0, n2 = (uint32_t)(p0 >> 32) ^ c[3] ^ k1;
    c[0] = n0;
    c[1] = (uint32_t)p1;
    c[2] = n2;
    c[3] = (uint32_t)p0;
  }
}
}  // namespace

void tadm_stale_times(int32_t B, uint64_t seed, uint32_t step, float eps, float* t, float* t_stale, int32_t* K,
                      int32_t* T, int32_t* k) {
#pragma clang fp contract(off)
  static const int Ks[4] = {1, 2, 4, 8}, Ts[6] = {128, 256, 512, 1024, 2048, 4096};
  const uint32_t k0 = (uint32_t)(seed & 0xFFFFFFFFu), k1 = (uint32_t)(seed >> 32);
  double u0 = 0.0;
  const double e = (double)eps;
  for (int b = 0; b < B; ++b) {
    uint32_t c[4] = {0x80000004u, (uint32_t)b, step, 0u};
    philox_host(c, k0, k1);
    if (b == 0) u0 = (double)((float)(2u * (c[0] >> 9) + 1u) * 5.9604644775390625e-08f);  // 2^-24
    const double frac = std::fmod(u0 + (double)b / B, 1.0);
    const float tb = (float)(e + (1.0 - e) * frac);
    const int Kb = Ks[c[1] >> 30];
    const int Tb = Ts[(int)(((uint64_t)c[2] * 6u) >> 32)];
    const int kb = (int)(((uint64_t)c[3] * (uint32_t)Kb) >> 32);
    if (t) t[b] = tb;
    if (t_stale) t_stale[b] = (float)std::min(1.0, (double)tb + (double)kb / (double)Tb);
    if (K) K[b] = Kb;
    if (T) T[b] = Tb;
    if (k) k[b] = kb;
  }
}

tadm_status tadm_train_loss(tadm_model* m, const int32_t* x_dev, int32_t B, int32_t L, const float* t_dev,
                            const float* t_stale_dev, float eps, uint64_t seed, uint32_t step, float* loss_dev,
                            int32_t* n_masked_dev, int32_t* zt_dev, int32_t* zs_dev) {
  TRY(check_model(m));
  if (!x_dev || !t_dev || !t_stale_dev || !loss_dev) return fail(TADM_ERR_INVALID, "null argument");
  if (B < 1 || B > m->cfg.max_batch || L < 1 || L > m->cfg.max_seq)
    return fail(TADM_ERR_INVALID, "B=%d L=%d outside the model's capacity", B, L);
  if (!(eps >= 0.f && eps < 1.f)) return fail(TADM_ERR_INVALID, "eps outside [0, 1)");
  TRY(ensure_workspace(m));
  const tadm_config& cf = m->cfg;
  Workspace& s = m->ws;
  const int N = B * L, d = cf.d_model, V = cf.vocab, mask = cf.vocab;
  if (!s.zt) {
    HIPCHK(hipMalloc((void**)&s.zt, (size_t)s.n_tok * 4));
    HIPCHK(hipMalloc((void**)&s.zs, (size_t)s.n_tok * 4));
    HIPCHK(hipMalloc((void**)&s.ce, (size_t)s.n_tok * 4));
  }
  if (!m->tcache) TRY(cache_alloc(m, cf.max_batch, cf.max_seq, &m->tcache));
  tadm_cache* cache = m->tcache;
  cache->B = B;
  cache->L = L;
  int32_t* zt = zt_dev ? zt_dev : s.zt;
  int32_t* zs = zs_dev ? zs_dev : s.zs;
  HIPCHK(corrupt_pair(x_dev, B, L, t_dev, t_stale_dev, eps, seed, step, mask, zt, zs, m->stream));
  // stale anchor from z_t', current pass on z_t
  TRY(anchor_impl(m, nullptr, zs, B, L, 1, cache));
  TRY(prof_begin(m, TADM_STAGE_EMBED));
  TRY(shared_net(m, nullptr, zt, B, L, s.c));
  TRY(prof_end(m, TADM_STAGE_EMBED));
  TRY(prof_begin(m, TADM_STAGE_FUSION));
  bool prenormed;
  TRY(fusion(m, B, L, s.c, cache, &prenormed));
  TRY(prof_end(m, TADM_STAGE_FUSION));
  TRY(prof_begin(m, TADM_STAGE_DENOISE));
  TRY(run_part(m, cf.n_shared + cf.n_anchor, cf.n_denoise, s.x, B, L, 0, nullptr, prenormed));
  HIPCHK(compact_masked(zt, B, L, 0, mask, B * L, s.cidx, s.row_map, s.count, m->stream));
  HIPCHK(rms_norm_gather(m->dt, s.x, m->Wf(m->lay.final_norm), cf.rms_eps, s.cidx, s.count, N, L, L, 0, d, s.xn,
                         m->stream));
  TRY(prof_end(m, TADM_STAGE_DENOISE));
  TRY(ensure_logits(m, (size_t)N * V));
  TRY(prof_begin(m, TADM_STAGE_HEAD));
  {
    GemmProblem p{N, V, d, s.xn, d, d, nullptr, 0, m->W(m->lay.w_out), d};
    p.M_dev = s.count;
    EpiParams e;
    e.out = s.logits;
    e.ldo = V;
    HIPCHK(gemm(m->dt, p, EPI_STORE_F32, e, m->stream));
  }
  TRY(prof_end(m, TADM_STAGE_HEAD));
  TRY(prof_begin(m, TADM_STAGE_SAMPLE));
  HIPCHK(masked_ce(s.logits, V, N, s.count, s.cidx, x_dev, s.ce, m->stream));
  TRY(prof_end(m, TADM_STAGE_SAMPLE));
  TRY(prof_begin(m, TADM_STAGE_SELECT));
  HIPCHK(weighted_loss(s.ce, s.row_map, B, L, t_dev, loss_dev, n_masked_dev, m->stream));
  TRY(prof_end(m, TADM_STAGE_SELECT));
  return TADM_OK;
}

// ---------------------------------------------------------- observability ---
tadm_status tadm_debug_read(tadm_model* m, int32_t tap, float* dst_dev, size_t bytes) {
  if (!m || !dst_dev) return fail(TADM_ERR_INVALID, "null argument");
  const size_t d = m->cfg.d_model;
  switch (tap) {
    case TADM_TAP_EMBED:
    case TADM_TAP_FUSED: {
      if (tap == TADM_TAP_FUSED && !m->taps) return fail(TADM_ERR_STATE, "enable taps before the step");
      const size_t n = (size_t)m->tap_B * m->tap_L * d;
      if (bytes != n * 4) return fail(TADM_ERR_INVALID, "tap %d has %zu bytes", tap, n * 4);
      HIPCHK(hipMemcpyAsync(dst_dev, tap == TADM_TAP_EMBED ? m->ws.c : m->ws.ht, bytes,
                            hipMemcpyDeviceToDevice, m->stream));
      return TADM_OK;
    }
    case TADM_TAP_FINAL: {
      if (!m->tap_final) return fail(TADM_ERR_STATE, "the last step computed the head for masked rows only");
      const size_t n = (size_t)m->tap_B * m->tap_Lc * d;
      if (bytes != n * 4) return fail(TADM_ERR_INVALID, "tap %d has %zu bytes", tap, n * 4);
      HIPCHK(to_f32(m->dt, m->ws.xn, dst_dev, n, m->stream));
      return TADM_OK;
    }
    case TADM_TAP_CHOICE:
    case TADM_TAP_CONF: {
      const size_t n = (size_t)m->tap_B * m->tap_Lc;
      if (bytes != n * 4) return fail(TADM_ERR_INVALID, "tap %d has %zu bytes", tap, n * 4);
      HIPCHK(hipMemcpyAsync(dst_dev, tap == TADM_TAP_CHOICE ? (const void*)m->ws.choice : (const void*)m->ws.conf,
                            bytes, hipMemcpyDeviceToDevice, m->stream));
      return TADM_OK;
    }
    default:
      return fail(TADM_ERR_INVALID, "tap %d", tap);
  }
}

tadm_status tadm_debug_taps(tadm_model* m, int32_t enable) {
  if (!m) return fail(TADM_ERR_INVALID, "null model");
  m->taps = enable != 0;
  return TADM_OK;
}

tadm_status tadm_debug_layers(tadm_model* m, float* dst_dev, size_t bytes) {
  if (!m) return fail(TADM_ERR_INVALID, "null model");
  if (dst_dev && bytes == 0) return fail(TADM_ERR_INVALID, "empty capture buffer");
  m->layer_cap = dst_dev;
  m->layer_cap_bytes = dst_dev ? bytes : 0;
  return TADM_OK;
}

tadm_status tadm_context_read(const tadm_context* ctx, int32_t layer, void* k_dev, void* vt_dev, size_t bytes) {
  if (!ctx || !k_dev || !vt_dev) return fail(TADM_ERR_INVALID, "null argument");
  const tadm_model* m = ctx->model;
  if (layer < 0 || layer >= m->n_layers()) return fail(TADM_ERR_INVALID, "layer %d", layer);
  const size_t n = (size_t)ctx->B * m->cfg.n_kv_heads * ctx->cap * m->cfg.head_dim * m->esz;
  if (bytes != n) return fail(TADM_ERR_INVALID, "context layer has %zu bytes, got %zu", n, bytes);
  HIPCHK(hipMemcpyAsync(k_dev, ctx->k[layer], n, hipMemcpyDeviceToDevice, m->stream));
  HIPCHK(hipMemcpyAsync(vt_dev, ctx->vt[layer], n, hipMemcpyDeviceToDevice, m->stream));
  return TADM_OK;
}

int32_t tadm_context_capacity(const tadm_context* ctx) { return ctx ? ctx->cap : 0; }

tadm_status tadm_profile_enable(tadm_model* m, int32_t stage_mask) {
  if (!m) return fail(TADM_ERR_INVALID, "null model");
  m->prof_mask = stage_mask;
  return TADM_OK;
}

tadm_status tadm_profile_reset(tadm_model* m) {
  if (!m) return fail(TADM_ERR_INVALID, "null model");
  HIPCHK(hipStreamSynchronize(m->stream));
  for (auto& r : m->recs) {
    m->pool.push_back(r.a);
    m->pool.push_back(r.b);
  }
  m->recs.clear();
  for (auto& o : m->open) {  // left open by a call that failed mid-stage
    m->pool.push_back(o.a);
    if (o.b) m->pool.push_back(o.b);
  }
  m->open.clear();
  next_launch_events = LaunchEvents{};
  return TADM_OK;
}

tadm_status tadm_profile_read(tadm_model* m, int32_t stage, double* total_ms, int64_t* count) {
  if (!m || !total_ms || !count) return fail(TADM_ERR_INVALID, "null argument");
  if (stage < 0 || stage >= TADM_STAGE_COUNT) return fail(TADM_ERR_INVALID, "stage %d", stage);
  HIPCHK(hipStreamSynchronize(m->stream));
  double tot = 0;
  int64_t n = 0;
  for (auto& r : m->recs)
    if (r.stage == stage) {
      float ms = 0;
      HIPCHK(hipEventElapsedTime(&ms, r.a, r.b));
      tot += ms;
      ++n;
    }
  *total_ms = tot;
  *count = n;
  return TADM_OK;
}

}  // extern "C"
