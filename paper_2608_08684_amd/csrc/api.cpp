// C ABI and pass scheduler of the sensitivity profile (Algorithm 1, Section 4.3).
//
// Scheduling: the sequences of a calibration set are processed in batches whose
// rows are concatenated, so every projection GEMM sees M = sum of the batch's
// lengths.  Per batch:
//   ReferencePredict  embed -> L blocks (keeping each block's fp32 input h_l)
//                     -> final RMSNorm -> clean log-sum-exp of the LM head;
//   per (alpha, l)    resume from h_l: block l with the Value noise injected
//                     between the q|k|v projection and attention, blocks
//                     l+1..L-1, final RMSNorm -> x_pert (one slot of a group);
//   per group         one LM-head + KL launch scores up to 16 passes against
//                     the clean logits computed once per tile, then window
//                     means and the calibration accumulator.
// Layers below l are never recomputed (prefix reuse); the same kernels on the
// same row layout make the clean and perturbed computations bitwise identical
// until the noise enters, so alpha = 0 gives KL = 0 exactly.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <functional>
#include <mutex>
#include <string>
#include <vector>

#include "rk_internal.h"

struct rk_model {
  rk_model_config cfg;
  bool bf16;
  int qkv_cols, attn_cols;
  const void* tok_emb;
  const void* lm_head;
  const float* final_norm;
  std::vector<const void*> w_qkv, w_o, w_gate_up, w_down;
  std::vector<const float*> attn_norm, mlp_norm;
  uint64_t ident;   // digest of the config and the weight pointers (state tags)
};

namespace rk {

static thread_local std::string g_error;

void set_error(const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_error = buf;
}

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Rows of a batch are int32 throughout (offsets, kernel row indices); size
// queries beyond that return 0 so no buffer plan can overflow.
static const int64_t kMaxRows = 0x7fffffff;

// FNV-1a (64-bit) over a byte range
static const uint64_t kFnvBasis = 0xcbf29ce484222325ull;
static uint64_t fnv(uint64_t h, const void* p, size_t n) {
  const unsigned char* c = (const unsigned char*)p;
  for (size_t i = 0; i < n; ++i) h = (h ^ c[i]) * 0x100000001b3ull;
  return h;
}

static size_t act_bytes(const rk_model* m) { return m->bf16 ? 2 : 4; }

// Buffers read as GEMM A operands hold whole 256-row tiles (the tile loads are
// not clamped); rows past the batch are never stored.
static int64_t pad_rows(int64_t R) { return (R + 255) / 256 * 256; }

// ----------------------------------------------------------------------------- memory plans
struct CleanPlan {
  size_t h, xf, lse, tag, total;
};

static CleanPlan clean_plan(const rk_model* m, int64_t R) {
  const int64_t d = m->cfg.d_model;
  CleanPlan p;
  size_t o = 0;
  p.h = o;   o += align256((size_t)m->cfg.n_layers * R * d * 4);
  p.xf = o;  o += align256((size_t)pad_rows(R) * d * act_bytes(m));
  p.lse = o; o += align256((size_t)R * 4);
  p.tag = o; o += 256;
  p.total = o;
  return p;
}

// State of the cached-window mode, sized for a batch of R rows (prefix plus
// window rows <= R): the prefix KV cache of every layer (K then V columns), and
// for the window rows the input of every block, the final hidden state and the
// clean log-sum-exp.
struct WinPlan {
  size_t kv, h, xf, lse, tag, total;
};

static int64_t kv_cols(const rk_model* m) { return 2 * (int64_t)m->cfg.n_kv_heads * m->cfg.head_dim; }

static WinPlan win_plan(const rk_model* m, int64_t R) {
  const int64_t d = m->cfg.d_model, L = m->cfg.n_layers;
  WinPlan p;
  size_t o = 0;
  p.kv = o;  o += align256((size_t)L * R * kv_cols(m) * act_bytes(m));
  p.h = o;   o += align256((size_t)L * R * d * 4);
  p.xf = o;  o += align256((size_t)pad_rows(R) * d * act_bytes(m));
  p.lse = o; o += align256((size_t)R * 4);
  p.tag = o; o += 256;
  p.total = o;
  return p;
}

struct WsPlan {
  size_t h, x, qkv, att, ff, xp, part, logits_c, logits_p, kl, rope, rope_pos, dbatch, sacc, tag, vpert, cpre, hloc,
      clean, total;
  bool unfused;
};

static const int kMaxSAcc = 4096;

static WsPlan ws_plan(const rk_model* m, int64_t R, int G, uint32_t flags) {
  const rk_model_config& c = m->cfg;
  const size_t a = act_bytes(m);
  WsPlan p;
  // the layer-local signal evaluates no LM head: no logits, no LM partials
  const bool local = (flags & RK_FLAG_LOCAL_SIGNAL) != 0;
  p.unfused = !local && (!m->bf16 || (flags & RK_FLAG_UNFUSED_KL));
  size_t o = 0;
  p.h = o;        o += align256((size_t)R * c.d_model * 4);
  const int64_t Rp = pad_rows(R);
  p.x = o;        o += align256((size_t)Rp * c.d_model * a);
  p.qkv = o;      o += align256((size_t)R * m->qkv_cols * a);
  p.att = o;      o += align256((size_t)Rp * m->attn_cols * a);
  p.ff = o;       o += align256((size_t)Rp * c.d_ff * a);
  p.xp = o;       o += align256((size_t)G * Rp * c.d_model * a);
  p.part = o;
  if (m->bf16 && !local) {
    // lm_chunks(rows) * rows <= min(n_vt * 128 * n_tt, (2048 + n_tt) * 128) and
    // lm_kl_chunks(rows) * rows <= min(n_vt * 256 * n_tb, (1024 + n_tb) * 256) for rows <= R
    const size_t n_vt = c.vocab / 128, n_tt = (R + 127) / 128, n_tb = (R + 255) / 256;
    const size_t bound = std::max(std::min(n_vt * 128 * n_tt, (2048 + n_tt) * 128),
                                  std::min(n_vt * 256 * n_tb, (1024 + n_tb) * 256));
    o += align256(bound * (size_t)G * 8);
  }
  p.logits_c = o;
  if (p.unfused) o += align256((size_t)R * c.vocab * 4);
  p.logits_p = o;
  if (p.unfused) o += align256((size_t)G * R * c.vocab * 4);
  p.kl = o;       o += align256((size_t)G * R * 4);
  p.rope = o;     o += align256((size_t)R * (c.head_dim / 2) * 8);   // max_len <= R positions
  p.rope_pos = o; o += align256((size_t)R * 4);
  p.dbatch = o;   o += align256((size_t)G * RK_MAX_BATCH_SEQS * 4);
  p.sacc = o;     o += align256((size_t)kMaxSAcc * 8);
  p.tag = o;      o += 256;
  p.vpert = o;
  if (flags & RK_FLAG_CACHED_WINDOW) o += align256((size_t)R * (kv_cols(m) / 2) * a);
  p.cpre = o;   // a compressed prompt cache (K and V columns)
  if (flags & RK_FLAG_CACHED_WINDOW) o += align256((size_t)R * kv_cols(m) * a);
  p.hloc = o;  // the clean output of the last block (layer-local signal)
  if (local) o += align256((size_t)R * c.d_model * 4);
  p.clean = o;
  if (flags & RK_WS_CLEAN_STATE)
    o += (flags & RK_FLAG_CACHED_WINDOW) ? win_plan(m, R).total : clean_plan(m, R).total;
  p.total = o;
  return p;
}

// Device buffers of one batch, carved from the workspace.
struct Bufs {
  float* h; void* x; void* qkv; void* att; void* ff; void* xp;
  float2* part; float* logits_c; float* logits_p; float* kl; float2* rope; int32_t* rope_pos; float* dbatch;
  double* sacc;
  uint64_t* tag;
  void* vpert;
  void* cpre;
  float* hloc;
  char* clean;
};

static Bufs carve(const WsPlan& p, void* ws) {
  char* b = (char*)ws;
  Bufs u;
  u.h = (float*)(b + p.h); u.x = b + p.x; u.qkv = b + p.qkv; u.att = b + p.att; u.ff = b + p.ff;
  u.xp = b + p.xp; u.part = (float2*)(b + p.part); u.logits_c = (float*)(b + p.logits_c);
  u.logits_p = (float*)(b + p.logits_p); u.kl = (float*)(b + p.kl); u.rope = (float2*)(b + p.rope);
  u.rope_pos = (int32_t*)(b + p.rope_pos);
  u.dbatch = (float*)(b + p.dbatch); u.sacc = (double*)(b + p.sacc); u.tag = (uint64_t*)(b + p.tag); u.vpert = b + p.vpert; u.cpre = b + p.cpre;
  u.hloc = (float*)(b + p.hloc); u.clean = b + p.clean;
  return u;
}

struct Clean {
  float* h; void* xf; float* lse;
};

static Clean clean_view(const rk_model* m, int64_t R, const void* base) {
  const CleanPlan p = clean_plan(m, R);
  char* b = (char*)base;
  return Clean{(float*)(b + p.h), b + p.xf, (float*)(b + p.lse)};
}

// Cached-window state: the window rows' part has the shape of a clean state
// (inputs h_l [L][Rw][d], final hidden, lse) plus the prefix KV cache.
struct Win {
  void* kv;   // [L][Rp][kv_cols], K columns then V columns
  Clean w;    // window rows
};

static Win win_view(const rk_model* m, int64_t R, const void* base) {
  const WinPlan p = win_plan(m, R);
  char* b = (char*)base;
  return Win{b + p.kv, Clean{(float*)(b + p.h), b + p.xf, (float*)(b + p.lse)}};
}

// ----------------------------------------------------------------------------- timing
// Event pairs around every launch of one kernel family (diagnostics only).
struct Timing {
  bool on = false;
  std::string family;
  std::vector<hipEvent_t> start, stop;
  size_t used = 0;
};
static Timing g_timing;

class Timed {
 public:
  Timed(const char* family, hipStream_t s) : s_(s) {
    if (!g_timing.on || g_timing.family != family) return;
    if (g_timing.used == g_timing.start.size()) {
      hipEvent_t a, b;
      if (hipEventCreate(&a) != hipSuccess) return;
      if (hipEventCreate(&b) != hipSuccess) { (void)hipEventDestroy(a); return; }
      g_timing.start.push_back(a);
      g_timing.stop.push_back(b);
    }
    idx_ = (long)g_timing.used++;
    (void)hipEventRecord(g_timing.start[idx_], s_);
  }
  ~Timed() {
    if (idx_ >= 0) (void)hipEventRecord(g_timing.stop[idx_], s_);
  }

 private:
  hipStream_t s_;
  long idx_ = -1;
};

// ----------------------------------------------------------------------------- passes
#define RK_TRY(expr)                                                       \
  do {                                                                     \
    hipError_t _e = (expr);                                                \
    if (_e != hipSuccess) {                                                \
      set_error("HIP error in %s: %s", #expr, hipGetErrorString(_e));      \
      return RK_ERR_HIP;                                                   \
    }                                                                      \
  } while (0)

struct Noise {
  float alpha;
  const rk_perturb_params* p;
  // joined resumed passes: the block's rows are pass slots of one->rows rows each,
  // each laid out as the single-pass table `one`; slots first .. first + n - 1
  // (the passes that start at this block) take the noise, slot first + k at alphas[k]
  const SeqTable* one = nullptr;
  int first = 0, n = 0;
  const float* alphas = nullptr;
};

// Observation queries to keep from a block (SnapKV prefill): the q columns of
// each sequence's last w rows.
struct ObsCapture {
  void* q;
  int w;
};

// Cached-window passes evaluated together (layer-synchronous batch): pass q of the
// batch owns rows [q * rw, (q + 1) * rw) of the block's buffers, and its
// attention reads layer l's prefix cache, with its own perturbed Values when l is
// the pass's layer.
struct WinBatch {
  const Win* wn;
  const SeqTable* pst;   // prefix rows: cache layout and noise keys
  const SeqTable* wst;   // the window rows of one pass
  const SeqTable* bt;    // the window rows of all n passes (pass q's sequences at q * wst->n ..)
  int n;                 // passes in the batch
  const int* layer;      // perturbed layer of each pass
  const float* alpha;
  const rk_perturb_params* p;
  int64_t rw;            // window rows per pass
  // compression damage instead of Value noise: at its layer, pass q reads the
  // n_keep retained prompt positions of every KV head, pos[q] (per sequence at
  // seq_stride), gathered from that layer's cache
  const int32_t* const* pos;
  int64_t seq_stride;
  int n_keep;
  // whole budget policies instead: at layer l, pass q attends to its own
  // compressed prompt cache, pol->keep[q][l] retained positions per KV head at
  // pol->pos[q] + pol->off[q][l] (per sequence at pol->stride[q]), or to the whole
  // cache when that count is 0
  const struct Policies* pol;
};

// Per pass of a group of whole budget policies (indexes of the group's batch).
struct Policies {
  const int32_t* pos[RK_MAX_GROUP];
  const int64_t* off[RK_MAX_GROUP];    // HOST [n_layers]
  const int32_t* keep[RK_MAX_GROUP];   // HOST [n_layers]
  int64_t stride[RK_MAX_GROUP];
};
static rk_status batch_attention(const rk_model* m, int l, const Bufs& b, const WinBatch& wb, hipStream_t s);

// One decoder block from h_in to h_out (h_out may equal h_in); `noise` perturbs
// the block's Values between the q|k|v projection and attention.
// With `pre`, the block's rows are the window rows of a cached-window batch and
// attention also reads the cached prefix; `kv_out` (if given) receives the
// block's K and V columns, row by row, and `obs` the observation queries.
static rk_status run_block(const rk_model* m, int l, const float* h_in, float* h_out, const Bufs& b,
                           const SeqTable& st, const Noise* noise, hipStream_t s, const KvPrefix* pre = nullptr,
                           void* kv_out = nullptr, const ObsCapture* obs = nullptr, const WinBatch* wb = nullptr) {
  const rk_model_config& c = m->cfg;
  const int R = st.rows, d = c.d_model;
  { Timed t("rmsnorm", s); RK_TRY(launch_rmsnorm(h_in, m->attn_norm[l], b.x, m->bf16, R, d, c.rms_eps, s)); }
  GemmArgs g{};
  g.A = b.x; g.lda = d; g.B = m->w_qkv[l]; g.ldb = d; g.M = R; g.N = m->qkv_cols; g.K = d;
  g.epi = Epi::kStoreRope; g.out = b.qkv; g.ldo = m->qkv_cols;
  g.rope_cols = (c.n_heads + c.n_kv_heads) * c.head_dim; g.head_dim = c.head_dim; g.rope_tab = b.rope;
  g.rope_pos = b.rope_pos;
  if (m->bf16) {  // the bf16 attention kernel takes queries pre-scaled to base-2 softmax units
    g.q_cols = c.n_heads * c.head_dim;
    g.q_scale = (float)(1.4426950408889634 / sqrt((double)c.head_dim));
  }
  { Timed t("gemm_qkv", s); RK_TRY(launch_gemm(g, m->bf16, s)); }
  if (kv_out) {
    const int64_t a = act_bytes(m);
    RK_TRY(launch_copy_cols(b.qkv, m->qkv_cols * a, (int64_t)c.n_heads * c.head_dim * a, kv_out, kv_cols(m) * a,
                            kv_cols(m) * a, R, s));
  }
  if (obs) RK_TRY(launch_snap_qobs(b.qkv, m->qkv_cols, st, obs->w, c.n_heads * c.head_dim, obs->q, s));
  if (noise) {
    char* v = (char*)b.qkv + (size_t)(c.n_heads + c.n_kv_heads) * c.head_dim * act_bytes(m);
    if (noise->one) {
      const size_t slot = (size_t)noise->one->rows * m->qkv_cols * act_bytes(m);
      for (int k = 0; k < noise->n; ++k) {
        Timed t("noise", s);
        RK_TRY(launch_value_noise(v + (size_t)(noise->first + k) * slot, m->bf16, m->qkv_cols, *noise->one,
                                  c.n_kv_heads, c.head_dim, l, noise->alphas[k], noise->p->seed,
                                  noise->p->protect_head, noise->p->protect_tail, s));
      }
    } else {
      Timed t("noise", s);
      RK_TRY(launch_value_noise(v, m->bf16, m->qkv_cols, st, c.n_kv_heads, c.head_dim, l, noise->alpha,
                                noise->p->seed, noise->p->protect_head, noise->p->protect_tail, s));
    }
  }
  if (wb) {
    rk_status e = batch_attention(m, l, b, *wb, s);
    if (e != RK_OK) return e;
  } else {
    Timed t("attention", s);
    RK_TRY(launch_attention(b.qkv, m->qkv_cols, b.att, m->attn_cols, st, c.n_heads, c.n_kv_heads, c.head_dim,
                            m->bf16, s, pre));
  }
  g = GemmArgs{};
  g.A = b.att; g.lda = m->attn_cols; g.B = m->w_o[l]; g.ldb = m->attn_cols; g.M = R; g.N = d; g.K = m->attn_cols;
  g.epi = Epi::kResidual; g.out = h_out; g.ldo = d; g.res = h_in; g.ldr = d;
  { Timed t("gemm_o", s); RK_TRY(launch_gemm(g, m->bf16, s)); }
  { Timed t("rmsnorm", s); RK_TRY(launch_rmsnorm(h_out, m->mlp_norm[l], b.x, m->bf16, R, d, c.rms_eps, s)); }
  g = GemmArgs{};
  g.A = b.x; g.lda = d; g.B = m->w_gate_up[l]; g.ldb = d; g.M = R; g.N = 2 * c.d_ff; g.K = d;
  g.epi = Epi::kSwiGLU; g.out = b.ff; g.ldo = c.d_ff; g.d_ff = c.d_ff;
  { Timed t("gemm_gate_up", s); RK_TRY(launch_gemm(g, m->bf16, s)); }
  g = GemmArgs{};
  g.A = b.ff; g.lda = c.d_ff; g.B = m->w_down[l]; g.ldb = c.d_ff; g.M = R; g.N = d; g.K = c.d_ff;
  g.epi = Epi::kResidual; g.out = h_out; g.ldo = d; g.res = h_out; g.ldr = d;
  { Timed t("gemm_down", s); RK_TRY(launch_gemm(g, m->bf16, s)); }
  return RK_OK;
}

// With h_last the last block's output is kept there; without lse the clean
// log-sum-exp is not formed (the layer-local signal needs neither LM head).
static rk_status reference_forward(const rk_model* m, const int32_t* tokens, const SeqTable& st, const Clean& cl,
                                   const Bufs& b, hipStream_t s, float* h_last = nullptr, bool lse = true) {
  const rk_model_config& c = m->cfg;
  const int64_t R = st.rows, d = c.d_model;
  float* last = h_last ? h_last : b.h;
  RK_TRY(launch_rope_table(b.rope, b.rope_pos, st, c.head_dim, c.rope_theta, s));
  RK_TRY(launch_embed(m->tok_emb, m->bf16, tokens, cl.h, (int)R, (int)d, s));
  for (int l = 0; l < c.n_layers; ++l) {
    float* out = (l + 1 < c.n_layers) ? cl.h + (size_t)(l + 1) * R * d : last;
    rk_status e = run_block(m, l, cl.h + (size_t)l * R * d, out, b, st, nullptr, s);
    if (e != RK_OK) return e;
  }
  RK_TRY(launch_rmsnorm(last, m->final_norm, cl.xf, m->bf16, (int)R, (int)d, c.rms_eps, s));
  if (m->bf16 && lse) {
    Timed t("lm_lse", s);
    RK_TRY(launch_lm_lse((const bf16_t*)cl.xf, (const bf16_t*)m->lm_head, (int)R, (int)d, c.vocab, b.part, cl.lse, s));
  }
  return RK_OK;
}

// Block `layer` with its Values perturbed, from the cached h_l (or from a
// recomputation of the layers below it); the output is left in b.h.
static rk_status perturbed_block(const rk_model* m, const int32_t* tokens, const SeqTable& st, const Clean& cl,
                                 int layer, float alpha, const rk_perturb_params* p, const Bufs& b, hipStream_t s) {
  const int64_t R = st.rows, d = m->cfg.d_model;
  const float* h_in = cl.h + (size_t)layer * R * d;
  if (p->flags & RK_FLAG_FULL_RECOMPUTE) {
    RK_TRY(launch_embed(m->tok_emb, m->bf16, tokens, b.h, (int)R, (int)d, s));
    for (int l = 0; l < layer; ++l) {
      rk_status e = run_block(m, l, b.h, b.h, b, st, nullptr, s);
      if (e != RK_OK) return e;
    }
    h_in = b.h;
  }
  Noise nz{alpha, p};
  return run_block(m, layer, h_in, b.h, b, st, &nz, s);
}

// PerturbedPredict up to the final normalised hidden state (written to xf_out).
static rk_status perturbed_final(const rk_model* m, const int32_t* tokens, const SeqTable& st, const Clean& cl,
                                 int layer, float alpha, const rk_perturb_params* p, void* xf_out, const Bufs& b,
                                 hipStream_t s) {
  const rk_model_config& c = m->cfg;
  const int64_t R = st.rows, d = c.d_model;
  rk_status e = perturbed_block(m, tokens, st, cl, layer, alpha, p, b, s);
  if (e != RK_OK) return e;
  for (int l = layer + 1; l < c.n_layers; ++l) {
    e = run_block(m, l, b.h, b.h, b, st, nullptr, s);
    if (e != RK_OK) return e;
  }
  RK_TRY(launch_rmsnorm(b.h, m->final_norm, xf_out, m->bf16, (int)R, (int)d, c.rms_eps, s));
  return RK_OK;
}

// A group of resumed passes, layer-synchronously (pass batching): the passes,
// ordered by their perturbed layer, join at that block from the cached clean
// block input h_l, and from then on every norm, projection, attention and
// feed-forward of a block runs once over the rows of all active passes (up to
// max_rows rows and RK_MAX_BATCH_SEQS sequences per launch; larger groups go in
// consecutive batches).  Every kernel is row-wise or per sequence, so each pass's
// result is bitwise that of perturbed_final.  Pass k's final hidden state goes
// to slot k of xp (stride pad_rows(R) rows).  The rotary table of the batch is
// rebuilt for the joined rows and restored on return.
static rk_status resumed_group_final(const rk_model* m, const int32_t* tokens, const SeqTable& st, const Clean& cl,
                                     int G, const int* layers, const float* alphas, const rk_perturb_params* p,
                                     int64_t max_rows, void* xp, const Bufs& b, hipStream_t s) {
  const rk_model_config& c = m->cfg;
  const int64_t d = c.d_model, R = st.rows, xstride = pad_rows(R) * d * act_bytes(m);
  const int L = c.n_layers;
  int B = (int)std::min<int64_t>(G, max_rows / R);
  B = std::min(B, RK_MAX_BATCH_SEQS / st.n);
  B = (int)std::min<int64_t>(B, INT32_MAX / R);   // joined row offsets are 32-bit
  if (B < 2 || (p->flags & RK_FLAG_FULL_RECOMPUTE)) {
    for (int k = 0; k < G; ++k) {
      rk_status e = perturbed_final(m, tokens, st, cl, layers[k], alphas[k], p, (char*)xp + (size_t)k * xstride, b, s);
      if (e != RK_OK) return e;
    }
    return RK_OK;
  }
  std::vector<int> order(G);
  for (int k = 0; k < G; ++k) order[k] = k;
  std::stable_sort(order.begin(), order.end(), [&](int x, int y) { return layers[x] < layers[y]; });
  for (int c0 = 0; c0 < G; c0 += B) {
    const int cb = std::min(B, G - c0);
    int lay[RK_MAX_GROUP];
    float al[RK_MAX_GROUP];
    for (int q = 0; q < cb; ++q) {
      lay[q] = layers[order[c0 + q]];
      al[q] = alphas[order[c0 + q]];
    }
    // batch table: sequence i of pass slot q at rows q * R + st.off[i]
    SeqTable bst = st;
    bst.n = cb * st.n;
    for (int q = 0; q < cb; ++q)
      for (int i = 0; i < st.n; ++i) bst.off[q * st.n + i] = (int32_t)(q * R) + st.off[i];
    bst.off[bst.n] = (int32_t)(cb * R);
    bst.rows = (int32_t)(cb * R);
    RK_TRY(launch_rope_table(b.rope, b.rope_pos, bst, c.head_dim, c.rope_theta, s));
    int active = 0;
    for (int j = lay[0]; j < L; ++j) {
      const int first = active;
      while (active < cb && lay[active] == j) {   // joins at its layer
        RK_TRY(hipMemcpyAsync(b.h + (size_t)active * R * d, cl.h + (size_t)j * R * d, (size_t)R * d * 4,
                              hipMemcpyDeviceToDevice, s));
        ++active;
      }
      SeqTable at = bst;   // the active passes' rows
      at.n = active * st.n;
      at.rows = (int32_t)(active * R);
      Noise nz{0.0f, p, &st, first, active - first, al + first};
      rk_status e = run_block(m, j, b.h, b.h, b, at, active > first ? &nz : nullptr, s);
      if (e != RK_OK) return e;
    }
    for (int q = 0; q < cb; ++q)
      RK_TRY(launch_rmsnorm(b.h + (size_t)q * R * d, m->final_norm, (char*)xp + (size_t)order[c0 + q] * xstride,
                            m->bf16, (int)R, (int)d, c.rms_eps, s));
  }
  RK_TRY(launch_rope_table(b.rope, b.rope_pos, st, c.head_dim, c.rope_theta, s));
  return RK_OK;
}

// Layer-local signal of one pass ("w/o DS" ablation): block `layer` alone with
// its Values perturbed, compared row by row with its clean output (the cached
// input of the next block, or h_last after the last block): r_out[row] =
// ||h~_{l+1} - h_{l+1}||^2 / ||h_{l+1}||^2.
static rk_status local_pass(const rk_model* m, const int32_t* tokens, const SeqTable& st, const Clean& cl, int layer,
                            float alpha, const rk_perturb_params* p, const float* h_last, float* r_out, const Bufs& b,
                            hipStream_t s) {
  const int64_t R = st.rows, d = m->cfg.d_model;
  rk_status e = perturbed_block(m, tokens, st, cl, layer, alpha, p, b, s);
  if (e != RK_OK) return e;
  const float* ref = (layer + 1 < m->cfg.n_layers) ? cl.h + (size_t)(layer + 1) * R * d : h_last;
  Timed t("local", s);
  RK_TRY(launch_local_response(b.h, ref, (int)R, (int)d, r_out, s));
  return RK_OK;
}

// KL at every position for G passes whose final hidden states sit at xp (stride R*d).
// Unfused: the clean logits must already be in logits_c; pass logits go to lp.
static rk_status score_group(const rk_model* m, const SeqTable& st, const Clean& cl, const void* xp, int G,
                             bool unfused, float* lp, float* kl, const Bufs& b, hipStream_t s) {
  const rk_model_config& c = m->cfg;
  const int64_t R = st.rows, d = c.d_model;
  if (!unfused) {
    Timed t("lm_kl", s);
    RK_TRY(launch_lm_kl((const bf16_t*)cl.xf, (const bf16_t*)xp, pad_rows(R) * d, G, (const bf16_t*)m->lm_head, (int)R, (int)d,
                        c.vocab, cl.lse, b.part, kl, s));
    return RK_OK;
  }
  for (int g = 0; g < G; ++g) {
    GemmArgs a{};
    a.A = (const char*)xp + (size_t)g * pad_rows(R) * d * act_bytes(m); a.lda = d; a.B = m->lm_head; a.ldb = d;
    a.M = (int)R; a.N = c.vocab; a.K = (int)d; a.epi = Epi::kStoreF32;
    a.out = lp + (size_t)g * R * c.vocab; a.ldo = c.vocab;
    Timed t("lm_logits", s);
    RK_TRY(launch_gemm(a, m->bf16, s));
  }
  Timed t("kl_logits", s);
  RK_TRY(launch_kl_logits(b.logits_c, lp, R * c.vocab, G, (int)R, c.vocab, kl, s));
  return RK_OK;
}

static rk_status clean_logits(const rk_model* m, const SeqTable& st, const Clean& cl, float* out, hipStream_t s) {
  const rk_model_config& c = m->cfg;
  GemmArgs a{};
  a.A = cl.xf; a.lda = c.d_model; a.B = m->lm_head; a.ldb = c.d_model;
  a.M = st.rows; a.N = c.vocab; a.K = c.d_model; a.epi = Epi::kStoreF32; a.out = out; a.ldo = c.vocab;
  RK_TRY(launch_gemm(a, m->bf16, s));
  return RK_OK;
}

// ----------------------------------------------------------------------------- cached-window mode
// The bf16 attention kernel addresses one sequence's q|k|v rows (and, in the
// cached-window mode, that sequence's cached K and V prefix, whose rows are
// narrower and fewer) through buffer descriptors with 32-bit byte offsets; a
// batch with a longer sequence is refused before any launch.
static rk_status check_span(const rk_model* m, const SeqTable& st) {
  if (!m->bf16) return RK_OK;
  const int64_t lim = (int64_t)1 << 31;
  if ((int64_t)st.max_len * m->qkv_cols * 2 >= lim) {
    set_error("a sequence of %d tokens exceeds the attention kernel's 32-bit buffer range (fewer than %lld tokens "
              "per sequence for this model)", st.max_len, (long long)((lim - 1) / ((int64_t)m->qkv_cols * 2)));
    return RK_ERR_SHAPE;
  }
  return RK_OK;
}

// Row tables of a cached-window batch: the prefix rows (P per sequence, in
// sequence order) and the window rows (T_k - P per sequence).
static rk_status window_tables(const SeqTable& st, int P, SeqTable* pst, SeqTable* wst) {
  if (P < 1) { set_error("the cached-window mode needs window_start >= 1"); return RK_ERR_ARG; }
  *pst = st;
  *wst = st;
  pst->max_len = P;
  wst->max_len = 0;
  for (int k = 0; k <= st.n; ++k) {
    pst->off[k] = k * P;
    wst->off[k] = st.off[k] - k * P;
    if (k > 0) {
      const int len = st.off[k] - st.off[k - 1];
      if (len <= P) {
        set_error("sequence %d (%d tokens) is not longer than window_start %d", k, len, P);
        return RK_ERR_SHAPE;
      }
      wst->max_len = std::max(wst->max_len, len - P);
    }
  }
  pst->rows = st.n * P;
  wst->rows = st.off[st.n] - st.n * P;
  return RK_OK;
}

// The cached prefix of layer l: K from the cache, V from the cache or from vpert.
static KvPrefix cache_prefix(const rk_model* m, const Win& wn, const SeqTable& pst, int l, const void* vpert) {
  const int64_t kc = kv_cols(m);
  const bf16_t* kv = (const bf16_t*)wn.kv + (size_t)l * pst.rows * kc;
  KvPrefix pk{};
  pk.alt_pass = -1;
  pk.k = kv;
  pk.ldk = kc;
  pk.P = pst.max_len;
  if (vpert) {
    pk.v = (const bf16_t*)vpert;
    pk.ldv = kc / 2;
  } else {
    pk.v = kv + kc / 2;
    pk.ldv = kc;
  }
  return pk;
}

// ReferencePredict of the cached-window mode: the prefixes run through every
// layer once and leave their K and V; the windows are then evaluated against the
// intact cache, keeping each block's input, the final hidden state and A_t.
static rk_status window_reference(const rk_model* m, const int32_t* tokens, const SeqTable& st, const SeqTable& pst,
                                  const SeqTable& wst, const Win& wn, const Bufs& b, hipStream_t s,
                                  float* h_last = nullptr, bool lse = true) {
  const rk_model_config& c = m->cfg;
  const int64_t d = c.d_model, Rp = pst.rows, Rw = wst.rows, kvb = kv_cols(m) * act_bytes(m);
  const int P = pst.max_len;
  RK_TRY(launch_rope_table(b.rope, b.rope_pos, pst, c.head_dim, c.rope_theta, s, 0));
  RK_TRY(launch_embed_gather(m->tok_emb, m->bf16, tokens, st, pst, 0, b.h, (int)d, s));
  for (int l = 0; l < c.n_layers; ++l) {
    rk_status e = run_block(m, l, b.h, b.h, b, pst, nullptr, s, nullptr, (char*)wn.kv + (size_t)l * Rp * kvb);
    if (e != RK_OK) return e;
  }
  RK_TRY(launch_rope_table(b.rope, b.rope_pos, wst, c.head_dim, c.rope_theta, s, P));
  RK_TRY(launch_embed_gather(m->tok_emb, m->bf16, tokens, st, wst, P, wn.w.h, (int)d, s));
  for (int l = 0; l < c.n_layers; ++l) {
    const KvPrefix pk = cache_prefix(m, wn, pst, l, nullptr);
    float* out = (l + 1 < c.n_layers) ? wn.w.h + (size_t)(l + 1) * Rw * d : (h_last ? h_last : b.h);
    rk_status e = run_block(m, l, wn.w.h + (size_t)l * Rw * d, out, b, wst, nullptr, s, &pk);
    if (e != RK_OK) return e;
  }
  RK_TRY(launch_rmsnorm(h_last ? h_last : b.h, m->final_norm, wn.w.xf, m->bf16, (int)Rw, (int)d, c.rms_eps, s));
  if (!lse) return RK_OK;
  Timed t("lm_lse", s);
  RK_TRY(launch_lm_lse((const bf16_t*)wn.w.xf, (const bf16_t*)m->lm_head, (int)Rw, (int)d, c.vocab, b.part,
                       wn.w.lse, s));
  return RK_OK;
}

// PerturbedPredict of the cached-window mode: layer `layer`'s cached prefix
// Values get the noise (a copy: the cache itself stays clean), the window rows
// resume from their input to that block and read the frozen caches above it.
// The rotary table must hold the window positions.
static rk_status window_perturbed_block(const rk_model* m, const SeqTable& pst, const SeqTable& wst, const Win& wn,
                                        int layer, float alpha, const rk_perturb_params* p, const Bufs& b,
                                        hipStream_t s) {
  const rk_model_config& c = m->cfg;
  const int64_t d = c.d_model, Rp = pst.rows, Rw = wst.rows, a = act_bytes(m), kc = kv_cols(m);
  const char* kv_l = (const char*)wn.kv + (size_t)layer * Rp * kc * a;
  RK_TRY(launch_copy_cols(kv_l, kc * a, (kc / 2) * a, b.vpert, (kc / 2) * a, (kc / 2) * a, (int)Rp, s));
  {
    Timed t("noise", s);
    RK_TRY(launch_value_noise(b.vpert, m->bf16, kc / 2, pst, c.n_kv_heads, c.head_dim, layer, alpha, p->seed,
                              p->protect_head, p->protect_tail, s));
  }
  const KvPrefix pk = cache_prefix(m, wn, pst, layer, b.vpert);
  return run_block(m, layer, wn.w.h + (size_t)layer * Rw * d, b.h, b, wst, nullptr, s, &pk);
}

static rk_status window_perturbed_final(const rk_model* m, const SeqTable& pst, const SeqTable& wst, const Win& wn,
                                        int layer, float alpha, const rk_perturb_params* p, void* xf_out,
                                        const Bufs& b, hipStream_t s) {
  const rk_model_config& c = m->cfg;
  const int64_t d = c.d_model, Rw = wst.rows;
  rk_status e = window_perturbed_block(m, pst, wst, wn, layer, alpha, p, b, s);
  if (e != RK_OK) return e;
  for (int l = layer + 1; l < c.n_layers; ++l) {
    const KvPrefix pk = cache_prefix(m, wn, pst, l, nullptr);
    if ((e = run_block(m, l, b.h, b.h, b, wst, nullptr, s, &pk)) != RK_OK) return e;
  }
  RK_TRY(launch_rmsnorm(b.h, m->final_norm, xf_out, m->bf16, (int)Rw, (int)d, c.rms_eps, s));
  return RK_OK;
}

// Layer-local signal of one cached-window pass: block `layer` on the window rows
// against the cache with its prefix Values perturbed, compared with its output
// against the intact cache (the next block's cached window input, or h_last).
static rk_status window_local_pass(const rk_model* m, const SeqTable& pst, const SeqTable& wst, const Win& wn,
                                   int layer, float alpha, const rk_perturb_params* p, const float* h_last,
                                   float* r_out, const Bufs& b, hipStream_t s) {
  const int64_t d = m->cfg.d_model, Rw = wst.rows;
  rk_status e = window_perturbed_block(m, pst, wst, wn, layer, alpha, p, b, s);
  if (e != RK_OK) return e;
  const float* ref = (layer + 1 < m->cfg.n_layers) ? wn.w.h + (size_t)(layer + 1) * Rw * d : h_last;
  Timed t("local", s);
  RK_TRY(launch_local_response(b.h, ref, (int)Rw, (int)d, r_out, s));
  return RK_OK;
}

static rk_status batch_attention(const rk_model* m, int l, const Bufs& b, const WinBatch& wb, hipStream_t s) {
  const rk_model_config& c = m->cfg;
  const int64_t a = act_bytes(m), kc = kv_cols(m), Rp = wb.pst->rows;
  int n_at_l = 0, alt = -1;
  for (int q = 0; q < wb.n; ++q)
    if (wb.layer[q] == l) { ++n_at_l; alt = q; }
  if (wb.pol) {
    // every pass reads its own (compressed or whole) prompt cache of this layer
    const char* kv_l = (const char*)wb.wn->kv + (size_t)l * Rp * kc * a;
    for (int q = 0; q < wb.n; ++q) {
      const int keep = wb.pol->keep[q][l];
      KvPrefix pk{};
      if (keep > 0) {
        RK_TRY(launch_prefix_gather(kv_l, kc, wb.pst->n, wb.pst->max_len, c.n_kv_heads, c.head_dim,
                                    wb.pol->pos[q] + wb.pol->off[q][l], wb.pol->stride[q], keep, b.cpre, s));
        pk.alt_pass = -1;
        pk.k = (const bf16_t*)b.cpre;
        pk.v = (const bf16_t*)b.cpre + kc / 2;
        pk.ldk = pk.ldv = kc;
        pk.P = keep;
      } else {
        pk = cache_prefix(m, *wb.wn, *wb.pst, l, nullptr);
      }
      Timed t("attention", s);
      RK_TRY(launch_attention((const char*)b.qkv + (size_t)q * wb.rw * m->qkv_cols * a, m->qkv_cols,
                              (char*)b.att + (size_t)q * wb.rw * m->attn_cols * a, m->attn_cols, *wb.wst, c.n_heads,
                              c.n_kv_heads, c.head_dim, m->bf16, s, &pk));
    }
    return RK_OK;
  }
  if (wb.pos) {
    // the passes ordered by layer: those below l read the full cache in one launch,
    // those starting at l (the last ones) their own compressed prompt cache
    const int full = wb.n - n_at_l;
    if (full > 0) {
      SeqTable ft = *wb.bt;
      ft.n = full * wb.wst->n;
      ft.rows = (int32_t)(full * wb.rw);
      KvPrefix pk = cache_prefix(m, *wb.wn, *wb.pst, l, nullptr);
      pk.n_seq = wb.wst->n;
      Timed t("attention", s);
      RK_TRY(launch_attention(b.qkv, m->qkv_cols, b.att, m->attn_cols, ft, c.n_heads, c.n_kv_heads, c.head_dim,
                              m->bf16, s, &pk));
    }
    const char* kv_l = (const char*)wb.wn->kv + (size_t)l * Rp * kc * a;
    for (int q = full; q < wb.n; ++q) {
      RK_TRY(launch_prefix_gather(kv_l, kc, wb.pst->n, wb.pst->max_len, c.n_kv_heads, c.head_dim, wb.pos[q],
                                  wb.seq_stride, wb.n_keep, b.cpre, s));
      KvPrefix pk{};
      pk.alt_pass = -1;
      pk.k = (const bf16_t*)b.cpre;
      pk.v = (const bf16_t*)b.cpre + kc / 2;
      pk.ldk = pk.ldv = kc;
      pk.P = wb.n_keep;
      Timed t("attention", s);
      RK_TRY(launch_attention((const char*)b.qkv + (size_t)q * wb.rw * m->qkv_cols * a, m->qkv_cols,
                              (char*)b.att + (size_t)q * wb.rw * m->attn_cols * a, m->attn_cols, *wb.wst, c.n_heads,
                              c.n_kv_heads, c.head_dim, m->bf16, s, &pk));
    }
    return RK_OK;
  }
  if (n_at_l <= 1) {
    // one launch over every pass's window rows; at most one pass reads perturbed Values
    KvPrefix pk = cache_prefix(m, *wb.wn, *wb.pst, l, nullptr);
    pk.n_seq = wb.wst->n;
    if (alt >= 0) {
      const char* kv_l = (const char*)wb.wn->kv + (size_t)l * Rp * kc * a;
      RK_TRY(launch_copy_cols(kv_l, kc * a, (kc / 2) * a, b.vpert, (kc / 2) * a, (kc / 2) * a, (int)Rp, s));
      Timed t("noise", s);
      RK_TRY(launch_value_noise(b.vpert, m->bf16, kc / 2, *wb.pst, c.n_kv_heads, c.head_dim, l, wb.alpha[alt],
                                wb.p->seed, wb.p->protect_head, wb.p->protect_tail, s));
      pk.alt_pass = alt;
      pk.v_alt = (const bf16_t*)b.vpert;
      pk.ldv_alt = kc / 2;
    }
    Timed t("attention", s);
    RK_TRY(launch_attention(b.qkv, m->qkv_cols, b.att, m->attn_cols, *wb.bt, c.n_heads, c.n_kv_heads, c.head_dim,
                            m->bf16, s, &pk));
    return RK_OK;
  }
  for (int q = 0; q < wb.n; ++q) {
    const void* vp = nullptr;
    if (wb.layer[q] == l) {   // this pass's layer: a perturbed copy of the cached prefix Values
      const char* kv_l = (const char*)wb.wn->kv + (size_t)l * Rp * kc * a;
      RK_TRY(launch_copy_cols(kv_l, kc * a, (kc / 2) * a, b.vpert, (kc / 2) * a, (kc / 2) * a, (int)Rp, s));
      Timed t("noise", s);
      RK_TRY(launch_value_noise(b.vpert, m->bf16, kc / 2, *wb.pst, c.n_kv_heads, c.head_dim, l, wb.alpha[q],
                                wb.p->seed, wb.p->protect_head, wb.p->protect_tail, s));
      vp = b.vpert;
    }
    const KvPrefix pk = cache_prefix(m, *wb.wn, *wb.pst, l, vp);
    Timed t("attention", s);
    RK_TRY(launch_attention((const char*)b.qkv + (size_t)q * wb.rw * m->qkv_cols * a, m->qkv_cols,
                            (char*)b.att + (size_t)q * wb.rw * m->attn_cols * a, m->attn_cols, *wb.wst, c.n_heads,
                            c.n_kv_heads, c.head_dim, m->bf16, s, &pk));
  }
  return RK_OK;
}

static rk_status window_compressed_final(const rk_model* m, const SeqTable& pst, const SeqTable& wst, const Win& wn,
                                         int layer, const int32_t* pos, int64_t seq_stride, int b, void* xf_out,
                                         const Bufs& bf, hipStream_t s);
static rk_status window_policy_final(const rk_model* m, const SeqTable& pst, const SeqTable& wst, const Win& wn,
                                     const int32_t* positions, const int64_t* layer_off, int64_t seq_stride,
                                     const int32_t* n_keep, void* xf_out, const Bufs& bf, hipStream_t s);

// A group of cached-window passes, layer-synchronously (pass
// batching): the passes, ordered by their perturbed layer, join the batch at that
// layer from the window's cached block input, and from then on every norm,
// projection and feed-forward of a layer runs once over the window rows of all
// active passes (up to max_rows rows and RK_MAX_BATCH_SEQS sequences per batch;
// larger groups go in consecutive batches).  Every kernel is row-wise or per pass,
// so each pass's result is bitwise that of window_perturbed_final.  Pass k's final
// hidden state goes to slot k of xp (stride pad_rows(Rw) rows).  The rotary table
// must hold the window positions; it does again on return.
static rk_status window_group_final(const rk_model* m, const SeqTable& pst, const SeqTable& wst, const Win& wn,
                                    int G, const int* layers, const float* alphas, const rk_perturb_params* p,
                                    int64_t max_rows, void* xp, const Bufs& b, hipStream_t s,
                                    const int32_t* const* pos = nullptr, int64_t seq_stride = 0, int n_keep = 0,
                                    const Policies* pol = nullptr) {
  const rk_model_config& c = m->cfg;
  const int64_t d = c.d_model, Rw = wst.rows, xstride = pad_rows(Rw) * d * act_bytes(m);
  const int L = c.n_layers, P = pst.max_len;
  int B = (int)std::min<int64_t>(G, max_rows / Rw);
  B = std::min(B, RK_MAX_BATCH_SEQS / wst.n);
  B = (int)std::min<int64_t>(B, INT32_MAX / Rw);   // joined row offsets are 32-bit
  if (B < 2) {
    for (int k = 0; k < G; ++k) {
      void* xk = (char*)xp + (size_t)k * xstride;
      rk_status e =
          pol ? window_policy_final(m, pst, wst, wn, pol->pos[k], pol->off[k], pol->stride[k], pol->keep[k], xk, b, s)
          : pos ? window_compressed_final(m, pst, wst, wn, layers[k], pos[k], seq_stride, n_keep, xk, b, s)
                : window_perturbed_final(m, pst, wst, wn, layers[k], alphas[k], p, xk, b, s);
      if (e != RK_OK) return e;
    }
    return RK_OK;
  }
  std::vector<int> order(G);
  for (int k = 0; k < G; ++k) order[k] = k;
  std::stable_sort(order.begin(), order.end(), [&](int x, int y) { return layers[x] < layers[y]; });
  for (int c0 = 0; c0 < G; c0 += B) {
    const int cb = std::min(B, G - c0);
    int lay[RK_MAX_GROUP];
    float al[RK_MAX_GROUP];
    const int32_t* ps[RK_MAX_GROUP];
    Policies pc{};
    for (int q = 0; q < cb; ++q) {
      const int k = order[c0 + q];
      lay[q] = layers[k];
      al[q] = alphas ? alphas[k] : 0.0f;
      ps[q] = pos ? pos[k] : nullptr;
      if (pol) {
        pc.pos[q] = pol->pos[k];
        pc.off[q] = pol->off[k];
        pc.keep[q] = pol->keep[k];
        pc.stride[q] = pol->stride[k];
      }
    }
    // batch table: sequence i of pass slot q at rows q * Rw + wst.off[i]
    SeqTable bst = wst;
    bst.n = cb * wst.n;
    for (int q = 0; q < cb; ++q)
      for (int i = 0; i < wst.n; ++i) bst.off[q * wst.n + i] = (int32_t)(q * Rw) + wst.off[i];
    bst.off[bst.n] = (int32_t)(cb * Rw);
    bst.rows = (int32_t)(cb * Rw);
    RK_TRY(launch_rope_table(b.rope, b.rope_pos, bst, c.head_dim, c.rope_theta, s, P));
    int active = 0;
    for (int j = lay[0]; j < L; ++j) {
      while (active < cb && lay[active] == j) {   // joins at its layer
        RK_TRY(hipMemcpyAsync(b.h + (size_t)active * Rw * d, wn.w.h + (size_t)j * Rw * d, (size_t)Rw * d * 4,
                              hipMemcpyDeviceToDevice, s));
        ++active;
      }
      SeqTable at = bst;   // the active passes' rows
      at.n = active * wst.n;
      at.rows = (int32_t)(active * Rw);
      const WinBatch wb{&wn, &pst, &wst, &at, active, lay, al, p, Rw, pos ? ps : nullptr, seq_stride, n_keep,
                        pol ? &pc : nullptr};
      rk_status e = run_block(m, j, b.h, b.h, b, at, nullptr, s, nullptr, nullptr, nullptr, &wb);
      if (e != RK_OK) return e;
    }
    for (int q = 0; q < cb; ++q)
      RK_TRY(launch_rmsnorm(b.h + (size_t)q * Rw * d, m->final_norm, (char*)xp + (size_t)order[c0 + q] * xstride,
                            m->bf16, (int)Rw, (int)d, c.rms_eps, s));
  }
  RK_TRY(launch_rope_table(b.rope, b.rope_pos, wst, c.head_dim, c.rope_theta, s, P));
  return RK_OK;
}

// Compression damage of layer `layer` (Section 2, Eq. layer-compression-damage):
// the window rows resume from their input to that block with its prompt cache
// replaced by the b retained positions of every KV head (gathered into a b-row
// cache per sequence); the caches of the other layers stay full.  The rotary
// table must hold the window positions.
static rk_status window_compressed_final(const rk_model* m, const SeqTable& pst, const SeqTable& wst, const Win& wn,
                                         int layer, const int32_t* pos, int64_t seq_stride, int b, void* xf_out,
                                         const Bufs& bf, hipStream_t s) {
  const rk_model_config& c = m->cfg;
  const int64_t d = c.d_model, Rp = pst.rows, Rw = wst.rows, a = act_bytes(m), kc = kv_cols(m);
  const char* kv_l = (const char*)wn.kv + (size_t)layer * Rp * kc * a;
  RK_TRY(launch_prefix_gather(kv_l, kc, pst.n, pst.max_len, c.n_kv_heads, c.head_dim, pos, seq_stride, b, bf.cpre,
                              s));
  KvPrefix pk{};
  pk.alt_pass = -1;
  pk.k = (const bf16_t*)bf.cpre;
  pk.v = (const bf16_t*)bf.cpre + kc / 2;
  pk.ldk = pk.ldv = kc;
  pk.P = b;
  rk_status e = run_block(m, layer, wn.w.h + (size_t)layer * Rw * d, bf.h, bf, wst, nullptr, s, &pk);
  if (e != RK_OK) return e;
  for (int l = layer + 1; l < c.n_layers; ++l) {
    pk = cache_prefix(m, wn, pst, l, nullptr);
    if ((e = run_block(m, l, bf.h, bf.h, bf, wst, nullptr, s, &pk)) != RK_OK) return e;
  }
  RK_TRY(launch_rmsnorm(bf.h, m->final_norm, xf_out, m->bf16, (int)Rw, (int)d, c.rms_eps, s));
  return RK_OK;
}

// The window rows with every layer's prompt cache compressed at once (a per-layer
// budget policy deployed, Section 4.4): block l attends to the n_keep[l] retained
// prompt positions of each KV head (positions + layer_off[l], per sequence at
// seq_stride), gathered into a compressed cache, or to the whole prompt cache when
// n_keep[l] is 0.  The window runs from block 0 (its cached input); the layers'
// caches are those of the full prefill.  The rotary table must hold the window
// positions.
static rk_status window_policy_final(const rk_model* m, const SeqTable& pst, const SeqTable& wst, const Win& wn,
                                     const int32_t* positions, const int64_t* layer_off, int64_t seq_stride,
                                     const int32_t* n_keep, void* xf_out, const Bufs& bf, hipStream_t s) {
  const rk_model_config& c = m->cfg;
  const int64_t d = c.d_model, Rp = pst.rows, Rw = wst.rows, a = act_bytes(m), kc = kv_cols(m);
  const float* h_in = wn.w.h;
  for (int l = 0; l < c.n_layers; ++l) {
    KvPrefix pk{};
    if (n_keep[l] > 0) {
      const char* kv_l = (const char*)wn.kv + (size_t)l * Rp * kc * a;
      RK_TRY(launch_prefix_gather(kv_l, kc, pst.n, pst.max_len, c.n_kv_heads, c.head_dim, positions + layer_off[l],
                                  seq_stride, n_keep[l], bf.cpre, s));
      pk.alt_pass = -1;
      pk.k = (const bf16_t*)bf.cpre;
      pk.v = (const bf16_t*)bf.cpre + kc / 2;
      pk.ldk = pk.ldv = kc;
      pk.P = n_keep[l];
    } else {
      pk = cache_prefix(m, wn, pst, l, nullptr);
    }
    rk_status e = run_block(m, l, h_in, bf.h, bf, wst, nullptr, s, &pk);
    if (e != RK_OK) return e;
    h_in = bf.h;
  }
  RK_TRY(launch_rmsnorm(bf.h, m->final_norm, xf_out, m->bf16, (int)Rw, (int)d, c.rms_eps, s));
  return RK_OK;
}

// ----------------------------------------------------------------------------- validation
static rk_status make_table(const rk_model* m, const rk_batch* bt, int first, int count, SeqTable* st) {
  if (count < 1 || count > RK_MAX_BATCH_SEQS) {
    set_error("batch holds %d sequences (1..%d allowed)", count, RK_MAX_BATCH_SEQS);
    return RK_ERR_SHAPE;
  }
  const int64_t base = bt->offsets[first];
  st->n = count;
  st->seq_index0 = bt->seq_index0 + first;
  st->max_len = 0;
  for (int k = 0; k <= count; ++k) {
    const int64_t o = bt->offsets[first + k] - base;
    if (o < 0 || o > (int64_t)0x7fffffff) { set_error("offsets out of range"); return RK_ERR_SHAPE; }
    st->off[k] = (int32_t)o;
    if (k > 0) {
      const int64_t len = bt->offsets[first + k] - bt->offsets[first + k - 1];
      if (len < 0) { set_error("offsets must be non-decreasing"); return RK_ERR_SHAPE; }
      if (len > st->max_len) st->max_len = (int32_t)len;
    }
  }
  st->rows = st->off[count];
  if (st->rows < 1) { set_error("batch has no tokens"); return RK_ERR_SHAPE; }
  return check_span(m, *st);
}

static rk_status check_batch(const rk_model* m, const rk_batch* b) {
  if (!m || !b || !b->tokens || !b->offsets) { set_error("null model, batch, tokens or offsets"); return RK_ERR_ARG; }
  if (b->n_seqs < 1) { set_error("n_seqs must be >= 1"); return RK_ERR_ARG; }
  if (b->seq_index0 < 0) { set_error("seq_index0 must be >= 0"); return RK_ERR_ARG; }
  if (b->offsets[0] != 0) { set_error("offsets[0] must be 0"); return RK_ERR_SHAPE; }
  return RK_OK;
}

// The window W_i = [window_start, T_i) of every sequence must hold a position:
// d_{i,l} is a mean over it (Eq. sample-response), undefined when it is empty.
static rk_status check_windows(const SeqTable& st, int32_t window_start) {
  for (int k = 0; k < st.n; ++k) {
    const int len = st.off[k + 1] - st.off[k];
    if (len <= window_start) {
      set_error("sequence %d (%d tokens) has an empty window: window_start %d", k, len, window_start);
      return RK_ERR_SHAPE;
    }
  }
  return RK_OK;
}

// ----------------------------------------------------------------------------- state tags
// Each state written by rk_reference_forward (window start -1) or
// rk_window_reference records which model and batch produced it: the model
// digest, the sequence lengths and the window start (host side), and a digest of
// the tokens (device side).  RK_FLAG_CHECK_STATE compares the record with the
// call's before anything is launched.
static const uint64_t kTagMagic = 0x524B535441544501ull;

static uint64_t host_ident(const rk_model* m, const SeqTable& st, int32_t window_start) {
  uint64_t h = fnv(kFnvBasis, &m->ident, sizeof(m->ident));
  h = fnv(h, &st.n, sizeof(st.n));
  h = fnv(h, st.off, sizeof(int32_t) * (size_t)(st.n + 1));
  return fnv(h, &window_start, sizeof(window_start));
}

static rk_status write_state_tag(const rk_model* m, const int32_t* tokens, const SeqTable& st, int32_t window_start,
                                 void* tag, hipStream_t s) {
  RK_TRY(launch_state_tag(tokens, st.rows, kTagMagic, host_ident(m, st, window_start), (uint64_t*)tag, s));
  return RK_OK;
}

// Synchronises the stream: the two records are read back to the host.
static rk_status check_state_tag(const rk_model* m, const int32_t* tokens, const SeqTable& st, int32_t window_start,
                                 const void* tag, uint64_t* scratch, hipStream_t s) {
  RK_TRY(launch_state_tag(tokens, st.rows, kTagMagic, host_ident(m, st, window_start), scratch, s));
  uint64_t have[4], want[4];
  RK_TRY(hipMemcpyAsync(have, tag, sizeof(have), hipMemcpyDeviceToHost, s));
  RK_TRY(hipMemcpyAsync(want, scratch, sizeof(want), hipMemcpyDeviceToHost, s));
  RK_TRY(hipStreamSynchronize(s));
  if (have[0] != kTagMagic) {
    set_error("the state was not written by rk_reference_forward or rk_window_reference");
    return RK_ERR_STATE;
  }
  if (memcmp(have, want, sizeof(have)) != 0) {
    set_error("the state belongs to another model, batch (tokens, lengths) or window start");
    return RK_ERR_STATE;
  }
  return RK_OK;
}

static rk_status check_params(const rk_perturb_params* p) {
  if (!p) { set_error("null perturbation params"); return RK_ERR_ARG; }
  if (p->window_start < 0 || p->protect_head < 0 || p->protect_tail < 0) {
    set_error("window_start / protect_head / protect_tail must be >= 0");
    return RK_ERR_ARG;
  }
  if (p->flags & ~(RK_FLAG_FULL_RECOMPUTE | RK_FLAG_UNFUSED_KL | RK_FLAG_CACHED_WINDOW | RK_FLAG_GRAPH |
                   RK_FLAG_LOCAL_SIGNAL | RK_FLAG_CHECK_STATE)) {
    set_error("unknown flags");
    return RK_ERR_ARG;
  }
  if ((p->flags & RK_FLAG_LOCAL_SIGNAL) && (p->flags & RK_FLAG_UNFUSED_KL)) {
    set_error("RK_FLAG_LOCAL_SIGNAL evaluates no LM head (RK_FLAG_UNFUSED_KL does not apply)");
    return RK_ERR_ARG;
  }
  if ((p->flags & RK_FLAG_CACHED_WINDOW) && (p->flags & RK_FLAG_FULL_RECOMPUTE)) {
    set_error("RK_FLAG_FULL_RECOMPUTE is not available in the cached-window mode");
    return RK_ERR_ARG;
  }
  return RK_OK;
}

static rk_status check_window_model(const rk_model* m) {
  if (!m->bf16) { set_error("the cached-window mode needs a bf16 model"); return RK_ERR_UNSUPPORTED; }
  return RK_OK;
}

// ----------------------------------------------------------------------------- SnapKV consumer
// Prefill state: the KV cache of every layer for all rows, then the observation
// queries of every layer.
struct SnapPlan {
  size_t kv, q, total;
};

static SnapPlan snap_plan(const rk_model* m, int64_t R, int n, int w) {
  const rk_model_config& c = m->cfg;
  SnapPlan p;
  size_t o = 0;
  p.kv = o; o += align256((size_t)c.n_layers * R * kv_cols(m) * 2);
  p.q = o;  o += align256((size_t)c.n_layers * n * w * c.n_heads * c.head_dim * 2);
  p.total = o;
  return p;
}

// Scratch of the selection: chunk partials, normalizers and every layer's votes.
struct SnapScratch {
  size_t part, cnorm, votes, total;
};

static SnapScratch snap_scratch(const rk_model* m, int64_t R, int n, int w) {
  const rk_model_config& c = m->cfg;
  SnapScratch p;
  size_t o = 0;
  p.part = o;  o += align256((size_t)c.n_layers * n * c.n_heads * w *
                             snap_chunks((int)std::min<int64_t>(R, 0x7fffffff)) * 8);
  p.cnorm = o; o += align256((size_t)c.n_layers * n * c.n_heads * w * 4);
  p.votes = o; o += align256((size_t)c.n_layers * c.n_kv_heads * R * 4);
  p.total = o;
  return p;
}

static rk_status check_snap(const rk_model* m, int w) {
  if (!m->bf16) { set_error("SnapKV selection needs a bf16 model"); return RK_ERR_UNSUPPORTED; }
  if (w < 1 || w > 64) { set_error("obs_window must be in [1, 64]"); return RK_ERR_ARG; }
  const int combos = (m->cfg.n_heads / m->cfg.n_kv_heads) * ((w + 31) / 32);
  if (combos > kSnapMaxCombos) {
    set_error("(n_heads / n_kv_heads) * ceil(obs_window / 32) = %d exceeds %d", combos, kSnapMaxCombos);
    return RK_ERR_UNSUPPORTED;
  }
  return RK_OK;
}

static rk_status check_snap_lengths(const SeqTable& st, int w) {
  for (int i = 0; i < st.n; ++i) {
    const int T = st.off[i + 1] - st.off[i];
    if (T <= w) { set_error("sequence %d (%d tokens) is not longer than obs_window %d", i, T, w); return RK_ERR_SHAPE; }
    if (T - w > kSnapMaxPrefix) {
      set_error("sequence %d: prefix of %d positions exceeds %d", i, T - w, kSnapMaxPrefix);
      return RK_ERR_UNSUPPORTED;
    }
  }
  return RK_OK;
}

// One recorded launch sequence per process: the sensitivity profile's kernels
// captured on a private stream into a HIP graph (after an eager run of the same
// call), replayed on the caller's stream while the arguments stay the same.
// With kernel timing on, the graph also holds the timing events (recorded as event
// nodes during capture); a replay re-records the same events, so the timing
// session sees the same event pairs as the captured call (timing_begin must
// precede each graphed call).
struct GraphCache {
  std::vector<uint64_t> key;
  hipGraphExec_t exec = nullptr;
  hipStream_t cap = nullptr;
  size_t timed = 0;   // timing event pairs inside the graph
};
static GraphCache g_graph;
static std::mutex g_graph_mu;   // the cache is shared by every thread of the process

template <class F>
static rk_status run_graphed(std::vector<uint64_t> key, F&& run, hipStream_t s) {
  std::lock_guard<std::mutex> lock(g_graph_mu);
  key.push_back(g_timing.on ? std::hash<std::string>()(g_timing.family) : 0);
  if (g_timing.on && g_timing.used != 0) {
    set_error("a graphed call needs a fresh timing session (rk_timing_begin) when timing is on");
    return RK_ERR_ARG;
  }
  if (g_graph.exec && g_graph.key == key) {
    RK_TRY(hipGraphLaunch(g_graph.exec, s));
    if (g_timing.on) g_timing.used = g_graph.timed;
    return RK_OK;
  }
  // first use: run eagerly (this call's results and timing events), then record
  // the same sequence for the replays; the recording reuses the timing events the
  // eager run created (no event is created while a stream is capturing)
  rk_status e = run(s);
  if (e != RK_OK) return e;
  if (!g_graph.cap) RK_TRY(hipStreamCreateWithFlags(&g_graph.cap, hipStreamNonBlocking));
  if (g_graph.exec) {
    RK_TRY(hipGraphExecDestroy(g_graph.exec));
    g_graph.exec = nullptr;
    g_graph.key.clear();
  }
  const size_t used = g_timing.used;
  g_timing.used = 0;
  RK_TRY(hipStreamBeginCapture(g_graph.cap, hipStreamCaptureModeThreadLocal));
  e = run(g_graph.cap);
  hipGraph_t graph = nullptr;
  const hipError_t ec = hipStreamEndCapture(g_graph.cap, &graph);
  const size_t timed = g_timing.used;
  g_timing.used = used;
  if (e != RK_OK) {
    if (graph) (void)hipGraphDestroy(graph);
    return e;
  }
  if (ec != hipSuccess) {
    set_error("HIP graph capture failed: %s", hipGetErrorString(ec));
    return RK_ERR_HIP;
  }
  if (g_timing.on && timed != used) {
    (void)hipGraphDestroy(graph);
    set_error("recorded launch sequence differs from the eager one");
    return RK_ERR_HIP;
  }
  hipGraphExec_t exec = nullptr;
  const hipError_t ei = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0);
  (void)hipGraphDestroy(graph);
  if (ei != hipSuccess) {
    set_error("HIP graph instantiation failed: %s", hipGetErrorString(ei));
    return RK_ERR_HIP;
  }
  g_graph.exec = exec;
  g_graph.key = key;
  g_graph.timed = g_timing.on ? used : 0;
  return RK_OK;
}

// Argument checks of the whole-profile entry points (everything but the
// workspace); on success *wp is the workspace plan for max_rows and max_group.
static rk_status check_profile(const rk_model* m, const rk_batch* calib, const int32_t* layers, int32_t n_A,
                               const float* alphas, int32_t n_alpha, const rk_perturb_params* p, int64_t max_rows,
                               int32_t max_group, const float* s_out, WsPlan* wp) {
  if (!m || !calib || !calib->tokens || !calib->offsets) { set_error("null model or calibration set"); return RK_ERR_ARG; }
  rk_status e = check_params(p);
  if (e != RK_OK) return e;
  if (calib->n_seqs < 1 || calib->seq_index0 < 0) { set_error("n_seqs must be >= 1, seq_index0 >= 0"); return RK_ERR_ARG; }
  if (calib->offsets[0] != 0) { set_error("offsets[0] must be 0"); return RK_ERR_SHAPE; }
  if (!layers || n_A < 1 || !alphas || n_alpha < 1 || !s_out) {
    set_error("null layers/alphas/s_out or empty layer/alpha set");
    return RK_ERR_ARG;
  }
  if ((int64_t)n_A * n_alpha > kMaxSAcc) { set_error("n_A * n_alpha must be <= %d", kMaxSAcc); return RK_ERR_ARG; }
  for (int j = 0; j < n_A; ++j)
    if (layers[j] < 0 || layers[j] >= m->cfg.n_layers) { set_error("layer %d out of range", layers[j]); return RK_ERR_ARG; }
  for (int a = 0; a < n_alpha; ++a)
    if (!(alphas[a] >= 0.0f) || !isfinite(alphas[a])) { set_error("alphas must be finite and >= 0"); return RK_ERR_ARG; }
  if (max_group < 1 || max_group > RK_MAX_GROUP) { set_error("max_group must be in [1, %d]", RK_MAX_GROUP); return RK_ERR_ARG; }
  if (max_rows < 1 || max_rows > kMaxRows) { set_error("max_rows must be in [1, 2^31 - 1]"); return RK_ERR_ARG; }
  const int N = calib->n_seqs;
  for (int i = 0; i < N; ++i) {
    const int64_t len = calib->offsets[i + 1] - calib->offsets[i];
    if (len < 0) { set_error("offsets must be non-decreasing"); return RK_ERR_SHAPE; }
    if (len > max_rows) { set_error("sequence %d (%lld tokens) exceeds max_rows", i, (long long)len); return RK_ERR_SHAPE; }
    if (len == 0) { set_error("sequence %d is empty", i); return RK_ERR_SHAPE; }
    if (len <= p->window_start) {
      set_error("sequence %d (%lld tokens) has an empty window: window_start %d", i, (long long)len, p->window_start);
      return RK_ERR_SHAPE;
    }
    if ((p->flags & RK_FLAG_CACHED_WINDOW) && (p->window_start < 1 || len <= p->window_start)) {
      set_error("sequence %d (%lld tokens) needs a non-empty prefix and window around window_start %d", i,
                (long long)len, p->window_start);
      return RK_ERR_SHAPE;
    }
  }
  const bool local = (p->flags & RK_FLAG_LOCAL_SIGNAL) != 0;
  const bool unfused = !local && (!m->bf16 || (p->flags & RK_FLAG_UNFUSED_KL));
  const bool cw = (p->flags & RK_FLAG_CACHED_WINDOW) != 0;
  if (cw && (e = check_window_model(m)) != RK_OK) return e;
  const uint32_t wflags = RK_WS_CLEAN_STATE | (unfused ? RK_FLAG_UNFUSED_KL : 0) | (cw ? RK_FLAG_CACHED_WINDOW : 0) |
                          (local ? RK_FLAG_LOCAL_SIGNAL : 0);
  // every batch the run will form, validated before any launch
  for (int first = 0; first < N;) {
    int count = 0;
    int64_t rows = 0;
    while (first + count < N && count < RK_MAX_BATCH_SEQS) {
      const int64_t len = calib->offsets[first + count + 1] - calib->offsets[first + count];
      if (count > 0 && rows + len > max_rows) break;
      rows += len;
      ++count;
    }
    SeqTable st, pst, wst;
    if ((e = make_table(m, calib, first, count, &st)) != RK_OK) return e;
    if (cw && (e = window_tables(st, p->window_start, &pst, &wst)) != RK_OK) return e;
    first += count;
  }
  *wp = ws_plan(m, max_rows, max_group, wflags);
  return RK_OK;
}

// The profile of a calibration set (Algorithm 1, profiling half) on a checked
// argument set, with the buffers of plan wp carved from workspace.
static rk_status profile_run(const rk_model* m, const rk_batch* calib, const int32_t* layers, int32_t n_A,
                             const float* alphas, int32_t n_alpha, const rk_perturb_params* p, int64_t max_rows,
                             int32_t max_group, float* s_out, float* d_out, const WsPlan& wp, void* workspace,
                             hipStream_t s) {
  rk_status e = RK_OK;
  const int N = calib->n_seqs;
  const bool local = (p->flags & RK_FLAG_LOCAL_SIGNAL) != 0;
  const bool unfused = !local && (!m->bf16 || (p->flags & RK_FLAG_UNFUSED_KL));
  const bool cw = (p->flags & RK_FLAG_CACHED_WINDOW) != 0;
  // Buffers are carved for max_rows; each batch uses the leading rows of each.
  const Bufs b = carve(wp, workspace);
  RK_TRY(launch_zero_f64(b.sacc, n_A * n_alpha, s));
  const int n_pass = n_A * n_alpha;
  int first = 0;
  while (first < N) {
    int count = 0;
    int64_t rows = 0;
    while (first + count < N && count < RK_MAX_BATCH_SEQS) {
      const int64_t len = calib->offsets[first + count + 1] - calib->offsets[first + count];
      if (count > 0 && rows + len > max_rows) break;
      rows += len;
      ++count;
    }
    SeqTable st;
    if ((e = make_table(m, calib, first, count, &st)) != RK_OK) return e;
    const int32_t* tokens = calib->tokens + calib->offsets[first];
    const int64_t R = st.rows;
    if (cw) {
      // cached-window mode: the same grouping over the window rows of the batch
      SeqTable pst, wst;
      if ((e = window_tables(st, p->window_start, &pst, &wst)) != RK_OK) return e;
      const Win wn = win_view(m, R, b.clean);
      if ((e = window_reference(m, tokens, st, pst, wst, wn, b, s, local ? b.hloc : nullptr, !local)) != RK_OK)
        return e;
      if (unfused && (e = clean_logits(m, wst, wn.w, b.logits_c, s)) != RK_OK) return e;
      const int64_t Rw = wst.rows;
      for (int g0 = 0; g0 < n_pass; g0 += max_group) {
        const int G = (n_pass - g0 < max_group) ? n_pass - g0 : max_group;
        PassMap pm{};
        pm.G = G;
        pm.seq_index0 = first;
        pm.d_seq_stride = n_A;
        int glay[RK_MAX_GROUP];
        float galpha[RK_MAX_GROUP];
        for (int k = 0; k < G; ++k) {
          const int idx = g0 + k, a = idx / n_A, j = idx % n_A;
          glay[k] = layers[j];
          galpha[k] = alphas[a];
          if (local &&
              (e = window_local_pass(m, pst, wst, wn, layers[j], alphas[a], p, b.hloc, b.kl + (size_t)k * Rw, b,
                                     s)) != RK_OK)
            return e;
          pm.d_base[k] = (int64_t)a * N * n_A + j;
          pm.s_index[k] = a * n_A + j;
        }
        if (!local && (e = window_group_final(m, pst, wst, wn, G, glay, galpha, p, max_rows, b.xp, b, s)) != RK_OK)
          return e;
        if (!local && (e = score_group(m, wst, wn.w, b.xp, G, unfused, b.logits_p, b.kl, b, s)) != RK_OK) return e;
        RK_TRY(launch_window_mean(b.kl, Rw, G, wst, 0, b.dbatch, s));
        RK_TRY(launch_accumulate(b.dbatch, st.n, pm, d_out, b.sacc, s));
      }
      first += count;
      continue;
    }
    const Clean cl = clean_view(m, R, b.clean);
    if ((e = reference_forward(m, tokens, st, cl, b, s, local ? b.hloc : nullptr, !local)) != RK_OK) return e;
    if (unfused && (e = clean_logits(m, st, cl, b.logits_c, s)) != RK_OK) return e;
    for (int g0 = 0; g0 < n_pass; g0 += max_group) {
      const int G = (n_pass - g0 < max_group) ? n_pass - g0 : max_group;
      PassMap pm{};
      pm.G = G;
      pm.seq_index0 = first;
      pm.d_seq_stride = n_A;
      int glay[RK_MAX_GROUP];
      float galpha[RK_MAX_GROUP];
      for (int k = 0; k < G; ++k) {
        const int idx = g0 + k, a = idx / n_A, j = idx % n_A;
        glay[k] = layers[j];
        galpha[k] = alphas[a];
        if (local &&
            (e = local_pass(m, tokens, st, cl, layers[j], alphas[a], p, b.hloc, b.kl + (size_t)k * R, b, s)) != RK_OK)
          return e;
        pm.d_base[k] = (int64_t)a * N * n_A + j;
        pm.s_index[k] = a * n_A + j;
      }
      if (!local && (e = resumed_group_final(m, tokens, st, cl, G, glay, galpha, p, max_rows, b.xp, b, s)) != RK_OK)
        return e;
      if (!local && (e = score_group(m, st, cl, b.xp, G, unfused, b.logits_p, b.kl, b, s)) != RK_OK) return e;
      RK_TRY(launch_window_mean(b.kl, R, G, st, p->window_start, b.dbatch, s));
      RK_TRY(launch_accumulate(b.dbatch, st.n, pm, d_out, b.sacc, s));
    }
    first += count;
  }
  RK_TRY(launch_finalize(b.sacc, n_pass, 1.0 / (double)N, s_out, s));
  return RK_OK;
}

// Forget the recorded sequence when its model goes away: a new model at the
// same address must never replay launches baked for the old one.
static void drop_graph(const rk_model* m) {
  std::lock_guard<std::mutex> lock(g_graph_mu);
  if (g_graph.exec && !g_graph.key.empty() && g_graph.key[0] == (uint64_t)(uintptr_t)m) {
    (void)hipGraphExecDestroy(g_graph.exec);
    g_graph.exec = nullptr;
    g_graph.key.clear();
  }
}

}  // namespace rk

using namespace rk;

// ============================================================================= C ABI
extern "C" {

const char* rk_last_error(void) { return g_error.c_str(); }

rk_status rk_timing_begin(const char* family) {
  if (!family) { set_error("null family"); return RK_ERR_ARG; }
  g_timing.on = true;
  g_timing.family = family;
  g_timing.used = 0;
  return RK_OK;
}

rk_status rk_timing_end(int64_t* launches, double* total_ms) {
  if (!launches || !total_ms) { set_error("null output"); return RK_ERR_ARG; }
  double sum = 0.0;
  for (size_t i = 0; i < g_timing.used; ++i) {
    float ms = 0.f;
    RK_TRY(hipEventSynchronize(g_timing.stop[i]));
    RK_TRY(hipEventElapsedTime(&ms, g_timing.start[i], g_timing.stop[i]));
    sum += ms;
  }
  *launches = (int64_t)g_timing.used;
  *total_ms = sum;
  g_timing.on = false;
  g_timing.used = 0;
  return RK_OK;
}

rk_status rk_model_create(const rk_model_config* cfg, const rk_model_weights* w, rk_model** out) {
  if (!cfg || !w || !out) { set_error("rk_model_create: null argument"); return RK_ERR_ARG; }
  *out = nullptr;
  const rk_model_config& c = *cfg;
  if (c.n_layers < 1 || c.d_model < 1 || c.n_heads < 1 || c.n_kv_heads < 1 || c.head_dim < 1 || c.d_ff < 1 ||
      c.vocab < 1) {
    set_error("rk_model_create: sizes must be positive");
    return RK_ERR_ARG;
  }
  if (!(c.rope_theta > 1.0f) || !isfinite(c.rope_theta) || !(c.rms_eps >= 0.0f) || !isfinite(c.rms_eps)) {
    set_error("rk_model_create: rope_theta must be > 1 and rms_eps >= 0");
    return RK_ERR_ARG;
  }
  if (c.dtype != RK_F32 && c.dtype != RK_BF16) { set_error("rk_model_create: unknown dtype"); return RK_ERR_ARG; }
  if (c.n_heads % c.n_kv_heads) { set_error("n_heads must be a multiple of n_kv_heads"); return RK_ERR_UNSUPPORTED; }
  const bool bf16 = c.dtype == RK_BF16;
  const int qkv = (c.n_heads + 2 * c.n_kv_heads) * c.head_dim, att = c.n_heads * c.head_dim;
  if (bf16 ? (c.head_dim != 64 && c.head_dim != 128) : (c.head_dim != 32 && c.head_dim != 64 && c.head_dim != 128)) {
    set_error("head_dim %d not supported for this dtype", c.head_dim);
    return RK_ERR_UNSUPPORTED;
  }
  if (c.d_model % 128 || att % 128 || qkv % 128 || c.vocab % 128 || c.d_ff % 64) {
    set_error("d_model, n_heads*head_dim, q|k|v width and vocab must be multiples of 128 and d_ff of 64");
    return RK_ERR_UNSUPPORTED;
  }
  if (!w->tok_emb || !w->lm_head || !w->final_norm || !w->w_qkv || !w->w_o || !w->w_gate_up || !w->w_down ||
      !w->attn_norm || !w->mlp_norm) {
    set_error("rk_model_create: null weight pointer");
    return RK_ERR_ARG;
  }
  for (int l = 0; l < c.n_layers; ++l)
    if (!w->w_qkv[l] || !w->w_o[l] || !w->w_gate_up[l] || !w->w_down[l] || !w->attn_norm[l] || !w->mlp_norm[l]) {
      set_error("rk_model_create: null weight pointer in layer %d", l);
      return RK_ERR_ARG;
    }
  rk_model* m = new rk_model();
  m->cfg = c;
  m->bf16 = bf16;
  m->qkv_cols = qkv;
  m->attn_cols = att;
  m->tok_emb = w->tok_emb;
  m->lm_head = w->lm_head;
  m->final_norm = w->final_norm;
  m->w_qkv.assign(w->w_qkv, w->w_qkv + c.n_layers);
  m->w_o.assign(w->w_o, w->w_o + c.n_layers);
  m->w_gate_up.assign(w->w_gate_up, w->w_gate_up + c.n_layers);
  m->w_down.assign(w->w_down, w->w_down + c.n_layers);
  m->attn_norm.assign(w->attn_norm, w->attn_norm + c.n_layers);
  m->mlp_norm.assign(w->mlp_norm, w->mlp_norm + c.n_layers);
  uint64_t h = kFnvBasis;
  const int32_t dims[8] = {c.n_layers, c.d_model, c.n_heads, c.n_kv_heads, c.head_dim, c.d_ff, c.vocab, (int32_t)c.dtype};
  h = fnv(h, dims, sizeof(dims));
  h = fnv(h, &c.rope_theta, sizeof(float));
  h = fnv(h, &c.rms_eps, sizeof(float));
  const void* top[3] = {m->tok_emb, m->lm_head, m->final_norm};
  h = fnv(h, top, sizeof(top));
  for (int l = 0; l < c.n_layers; ++l) {
    const void* lw[6] = {m->w_qkv[l], m->w_o[l], m->w_gate_up[l], m->w_down[l], m->attn_norm[l], m->mlp_norm[l]};
    h = fnv(h, lw, sizeof(lw));
  }
  m->ident = h;
  *out = m;
  return RK_OK;
}

void rk_model_destroy(rk_model* m) {
  if (!m) return;
  drop_graph(m);
  delete m;
}

size_t rk_clean_state_size(const rk_model* m, int64_t n_rows) {
  if (!m || n_rows < 1 || n_rows > kMaxRows) return 0;
  return clean_plan(m, n_rows).total;
}

size_t rk_window_state_size(const rk_model* m, int64_t n_rows) {
  if (!m || n_rows < 1 || n_rows > kMaxRows || !m->bf16) return 0;
  return win_plan(m, n_rows).total;
}

rk_status rk_window_reference(const rk_model* m, const rk_batch* batch, int32_t window_start, void* state,
                              size_t state_bytes, void* workspace, size_t ws_bytes, void* stream) {
  rk_status e = check_batch(m, batch);
  if (e != RK_OK) return e;
  if ((e = check_window_model(m)) != RK_OK) return e;
  if (!state || !workspace) { set_error("null state or workspace"); return RK_ERR_ARG; }
  SeqTable st, pst, wst;
  if ((e = make_table(m, batch, 0, batch->n_seqs, &st)) != RK_OK) return e;
  if ((e = window_tables(st, window_start, &pst, &wst)) != RK_OK) return e;
  if (state_bytes < win_plan(m, st.rows).total) { set_error("window state too small"); return RK_ERR_WORKSPACE; }
  const WsPlan wp = ws_plan(m, st.rows, 1, RK_FLAG_CACHED_WINDOW);
  if (ws_bytes < wp.total) { set_error("workspace too small (%zu < %zu)", ws_bytes, wp.total); return RK_ERR_WORKSPACE; }
  const Bufs b = carve(wp, workspace);
  hipStream_t s = (hipStream_t)stream;
  if ((e = window_reference(m, batch->tokens, st, pst, wst, win_view(m, st.rows, state), b, s)) != RK_OK) return e;
  return write_state_tag(m, batch->tokens, st, window_start, (char*)state + win_plan(m, st.rows).tag, s);
}

size_t rk_snapkv_state_size(const rk_model* m, int64_t n_rows, int32_t n_seqs, int32_t obs_window) {
  if (!m || !m->bf16 || n_rows < 1 || n_rows > kMaxRows || n_seqs < 1 || obs_window < 1) return 0;
  return snap_plan(m, n_rows, n_seqs, obs_window).total;
}

size_t rk_snapkv_workspace_size(const rk_model* m, int64_t n_rows, int32_t n_seqs, int32_t obs_window) {
  if (!m || !m->bf16 || n_rows < 1 || n_rows > kMaxRows || n_seqs < 1 || obs_window < 1) return 0;
  return std::max(ws_plan(m, n_rows, 1, 0).total, snap_scratch(m, n_rows, n_seqs, obs_window).total);
}

rk_status rk_snapkv_prefill(const rk_model* m, const rk_batch* batch, int32_t obs_window, void* state,
                            size_t state_bytes, void* workspace, size_t ws_bytes, void* stream) {
  rk_status e = check_batch(m, batch);
  if (e != RK_OK) return e;
  if ((e = check_snap(m, obs_window)) != RK_OK) return e;
  if (!state || !workspace) { set_error("null state or workspace"); return RK_ERR_ARG; }
  SeqTable st;
  if ((e = make_table(m, batch, 0, batch->n_seqs, &st)) != RK_OK) return e;
  for (int i = 0; i < st.n; ++i)
    if (st.off[i + 1] - st.off[i] <= obs_window) {
      set_error("sequence %d is not longer than obs_window %d", i, obs_window);
      return RK_ERR_SHAPE;
    }
  const SnapPlan sp = snap_plan(m, st.rows, st.n, obs_window);
  if (state_bytes < sp.total) { set_error("SnapKV state too small (%zu < %zu)", state_bytes, sp.total); return RK_ERR_WORKSPACE; }
  const WsPlan wp = ws_plan(m, st.rows, 1, 0);
  if (ws_bytes < wp.total) { set_error("workspace too small (%zu < %zu)", ws_bytes, wp.total); return RK_ERR_WORKSPACE; }
  const Bufs b = carve(wp, workspace);
  const rk_model_config& c = m->cfg;
  hipStream_t s = (hipStream_t)stream;
  const int64_t R = st.rows, d = c.d_model;
  char* kv = (char*)state + sp.kv;
  char* q = (char*)state + sp.q;
  const size_t kv_layer = (size_t)R * kv_cols(m) * 2, q_layer = (size_t)st.n * obs_window * c.n_heads * c.head_dim * 2;
  RK_TRY(launch_rope_table(b.rope, b.rope_pos, st, c.head_dim, c.rope_theta, s));
  RK_TRY(launch_embed(m->tok_emb, m->bf16, batch->tokens, b.h, (int)R, (int)d, s));
  for (int l = 0; l < c.n_layers; ++l) {
    const ObsCapture obs{q + l * q_layer, obs_window};
    if ((e = run_block(m, l, b.h, b.h, b, st, nullptr, s, nullptr, kv + l * kv_layer, &obs)) != RK_OK) return e;
  }
  return RK_OK;
}

int64_t rk_snapkv_layout(const rk_batch* batch, int32_t n_layers, const int64_t* budgets, int64_t* offsets_out) {
  if (!batch || !batch->offsets || !budgets || n_layers < 1 || batch->n_seqs < 1) return -1;
  int64_t total = 0;
  for (int i = 0; i < batch->n_seqs; ++i) {
    const int64_t T = batch->offsets[i + 1] - batch->offsets[i];
    if (T < 0) return -1;
    for (int l = 0; l < n_layers; ++l) {
      if (offsets_out) offsets_out[(int64_t)i * n_layers + l] = total;
      total += std::min(std::max(budgets[(int64_t)i * n_layers + l], (int64_t)0), T);
    }
  }
  if (offsets_out) offsets_out[(int64_t)batch->n_seqs * n_layers] = total;
  return total;
}

rk_status rk_snapkv_compress(const rk_model* m, const rk_batch* batch, const rk_snapkv_params* p,
                             const int64_t* budgets, const void* state, size_t state_bytes, int32_t* positions,
                             void* k_out, void* v_out, float* scores, void* workspace, size_t ws_bytes,
                             void* stream) {
  rk_status e = check_batch(m, batch);
  if (e != RK_OK) return e;
  if (!p || !budgets || !state || !positions || !k_out || !v_out || !workspace) {
    set_error("null params, budgets, state, outputs or workspace");
    return RK_ERR_ARG;
  }
  const int w = p->obs_window;
  if ((e = check_snap(m, w)) != RK_OK) return e;
  if (p->pool_kernel < 1 || p->pool_kernel > 31 || p->pool_kernel % 2 == 0) {
    set_error("pool_kernel must be odd and in [1, 31]");
    return RK_ERR_ARG;
  }
  if (p->pooling != RK_POOL_MAX && p->pooling != RK_POOL_AVG) { set_error("unknown pooling"); return RK_ERR_ARG; }
  SeqTable st;
  if ((e = make_table(m, batch, 0, batch->n_seqs, &st)) != RK_OK) return e;
  if ((e = check_snap_lengths(st, w)) != RK_OK) return e;
  const SnapPlan sp = snap_plan(m, st.rows, st.n, w);
  if (state_bytes < sp.total) { set_error("SnapKV state too small (%zu < %zu)", state_bytes, sp.total); return RK_ERR_WORKSPACE; }
  const SnapScratch sc = snap_scratch(m, st.rows, st.n, w);
  if (ws_bytes < sc.total) { set_error("workspace too small (%zu < %zu)", ws_bytes, sc.total); return RK_ERR_WORKSPACE; }
  const rk_model_config& c = m->cfg;
  const int L = c.n_layers;
  std::vector<int64_t> offs((size_t)st.n * L + 1);
  if (rk_snapkv_layout(batch, L, budgets, offs.data()) < 0) { set_error("bad budgets or offsets"); return RK_ERR_ARG; }
  hipStream_t s = (hipStream_t)stream;
  char* ws = (char*)workspace;
  float2* part = (float2*)(ws + sc.part);
  float* cnorm = (float*)(ws + sc.cnorm);
  float* votes = (float*)(ws + sc.votes);
  const int64_t prefix_rows = (int64_t)st.rows - (int64_t)st.n * w;
  const int64_t ldkv = kv_cols(m);
  const size_t kv_layer = (size_t)st.rows * ldkv * 2, q_layer = (size_t)st.n * w * c.n_heads * c.head_dim * 2;
  // votes of every layer, then one selection pass over all (sequence, layer) items
  {
    Timed t("snap_scores", s);
    RK_TRY(launch_snap_scores((const char*)state + sp.kv, ldkv, (int64_t)(kv_layer / 2), (const char*)state + sp.q,
                              (int64_t)(q_layer / 2), L, st, w, c.n_heads, c.n_kv_heads, c.head_dim, part, cnorm,
                              votes, prefix_rows, s));
  }
  const int n_items = st.n * L;
  std::vector<int16_t> seq(n_items), lay(n_items);
  std::vector<int32_t> keep(n_items);
  std::vector<int64_t> entry0(n_items);
  for (int i = 0; i < st.n; ++i)
    for (int l = 0; l < L; ++l) {
      const size_t j = (size_t)i * L + l;
      seq[j] = (int16_t)i;
      lay[j] = (int16_t)l;
      keep[j] = (int32_t)(offs[j + 1] - offs[j]);
      entry0[j] = offs[j] * c.n_kv_heads;
    }
  Timed t("snap_select", s);
  RK_TRY(launch_snap_select(votes, prefix_rows, (const char*)state + sp.kv, ldkv, (int64_t)(kv_layer / 2), st, w,
                            c.n_kv_heads, c.head_dim, p->pool_kernel, p->pooling == RK_POOL_AVG, n_items, seq.data(),
                            lay.data(), keep.data(), entry0.data(), positions, k_out, v_out, scores, s));
  return RK_OK;
}

}  // extern "C"

// One budget policy's arguments (see rk_policy_damage).
static rk_status check_policy(const rk_model* m, int32_t window_start, const int32_t* positions,
                              const int64_t* layer_offsets, int64_t seq_stride, const int32_t* n_keep) {
  int max_keep = 0;
  for (int l = 0; l < m->cfg.n_layers; ++l) {
    if (n_keep[l] < 0 || n_keep[l] > window_start) { set_error("n_keep[%d] must be in [0, window_start]", l); return RK_ERR_ARG; }
    if (n_keep[l] > 0 && layer_offsets[l] < 0) { set_error("layer_offsets[%d] must be >= 0", l); return RK_ERR_ARG; }
    max_keep = std::max(max_keep, (int)n_keep[l]);
  }
  if (max_keep > 0 && !positions) { set_error("null positions"); return RK_ERR_ARG; }
  if (max_keep > 0 && seq_stride < (int64_t)m->cfg.n_kv_heads * max_keep) {
    set_error("seq_stride below n_kv_heads * max(n_keep)");
    return RK_ERR_ARG;
  }
  return RK_OK;
}

// The set-up shared by the calls that evaluate a batch's window rows against its
// window state: the prefix and window tables, the size checks, the workspace
// carve-up (G passes per LM-head launch, workspace flags wf) and the window's
// rotary table (its only launch, after every check).
struct WinCall {
  SeqTable st, pst, wst;
  Bufs b;
  Win wn;
  hipStream_t s;
};

static rk_status win_call(const rk_model* m, const rk_batch* batch, int32_t window_start, const void* state,
                          size_t state_bytes, void* workspace, size_t ws_bytes, int G, uint32_t wf, void* stream,
                          WinCall* c) {
  rk_status e;
  if ((e = make_table(m, batch, 0, batch->n_seqs, &c->st)) != RK_OK) return e;
  if ((e = window_tables(c->st, window_start, &c->pst, &c->wst)) != RK_OK) return e;
  if (state_bytes < win_plan(m, c->st.rows).total) { set_error("window state too small"); return RK_ERR_WORKSPACE; }
  const WsPlan wp = ws_plan(m, c->st.rows, G, wf);
  if (ws_bytes < wp.total) { set_error("workspace too small (%zu < %zu)", ws_bytes, wp.total); return RK_ERR_WORKSPACE; }
  c->b = carve(wp, workspace);
  c->wn = win_view(m, c->st.rows, state);
  c->s = (hipStream_t)stream;
  RK_TRY(launch_rope_table(c->b.rope, c->b.rope_pos, c->wst, m->cfg.head_dim, m->cfg.rope_theta, c->s, window_start));
  return RK_OK;
}

// Scores G finished window passes (slots of b.xp) against the full-cache window
// and takes the window means: d_out[g * n_seqs + i]; logits_out selects the
// unfused LM head and receives the passes' fp32 logits.
static rk_status score_window(const rk_model* m, const WinCall& c, int G, float* logits_out, float* kl_pos,
                              float* d_out) {
  rk_status e;
  float* kl = kl_pos ? kl_pos : c.b.kl;
  const bool unfused = logits_out != nullptr;
  if (unfused && (e = clean_logits(m, c.wst, c.wn.w, c.b.logits_c, c.s)) != RK_OK) return e;
  if ((e = score_group(m, c.wst, c.wn.w, c.b.xp, G, unfused, unfused ? logits_out : c.b.logits_p, kl, c.b, c.s)) !=
      RK_OK)
    return e;
  RK_TRY(launch_window_mean(kl, c.wst.rows, G, c.wst, 0, d_out, c.s));
  return RK_OK;
}

extern "C" {

rk_status rk_compression_damage(const rk_model* m, const rk_batch* batch, int32_t window_start, int32_t layer,
                                const int32_t* positions, int64_t seq_stride, int32_t n_keep, const void* state,
                                size_t state_bytes, float* d_out, float* kl_pos, void* workspace, size_t ws_bytes,
                                void* stream) {
  rk_status e = check_batch(m, batch);
  if (e != RK_OK) return e;
  if ((e = check_window_model(m)) != RK_OK) return e;
  if (!positions || !state || !d_out || !workspace) { set_error("null positions, state, d_out or workspace"); return RK_ERR_ARG; }
  if (layer < 0 || layer >= m->cfg.n_layers) { set_error("layer %d out of range", layer); return RK_ERR_ARG; }
  if (n_keep < 1 || n_keep > window_start) { set_error("n_keep must be in [1, window_start]"); return RK_ERR_ARG; }
  if (seq_stride < (int64_t)m->cfg.n_kv_heads * n_keep) { set_error("seq_stride below n_kv_heads * n_keep"); return RK_ERR_ARG; }
  WinCall c;
  if ((e = win_call(m, batch, window_start, state, state_bytes, workspace, ws_bytes, 1, RK_FLAG_CACHED_WINDOW, stream,
                    &c)) != RK_OK)
    return e;
  if ((e = window_compressed_final(m, c.pst, c.wst, c.wn, layer, positions, seq_stride, n_keep, c.b.xp, c.b, c.s)) !=
      RK_OK)
    return e;
  return score_window(m, c, 1, nullptr, kl_pos, d_out);
}

rk_status rk_compression_damage_layers(const rk_model* m, const rk_batch* batch, int32_t window_start,
                                       const int32_t* layers, int32_t n_sel, const int32_t* positions,
                                       int64_t layer_stride, int64_t seq_stride, int32_t n_keep, const void* state,
                                       size_t state_bytes, float* d_out, float* kl_pos, void* workspace,
                                       size_t ws_bytes, void* stream) {
  rk_status e = check_batch(m, batch);
  if (e != RK_OK) return e;
  if ((e = check_window_model(m)) != RK_OK) return e;
  if (!layers || !positions || !state || !d_out || !workspace) {
    set_error("null layers, positions, state, d_out or workspace");
    return RK_ERR_ARG;
  }
  if (n_sel < 1 || n_sel > RK_MAX_GROUP) { set_error("n_layers must be in [1, %d]", RK_MAX_GROUP); return RK_ERR_ARG; }
  for (int k = 0; k < n_sel; ++k)
    if (layers[k] < 0 || layers[k] >= m->cfg.n_layers) { set_error("layer %d out of range", layers[k]); return RK_ERR_ARG; }
  if (n_keep < 1 || n_keep > window_start) { set_error("n_keep must be in [1, window_start]"); return RK_ERR_ARG; }
  if (seq_stride < (int64_t)m->cfg.n_kv_heads * n_keep) { set_error("seq_stride below n_kv_heads * n_keep"); return RK_ERR_ARG; }
  if (layer_stride < 0) { set_error("layer_stride must be >= 0"); return RK_ERR_ARG; }
  WinCall c;
  if ((e = win_call(m, batch, window_start, state, state_bytes, workspace, ws_bytes, n_sel, RK_FLAG_CACHED_WINDOW,
                    stream, &c)) != RK_OK)
    return e;
  const int32_t* ps[RK_MAX_GROUP];
  for (int k = 0; k < n_sel; ++k) ps[k] = positions + (int64_t)layers[k] * layer_stride;
  if ((e = window_group_final(m, c.pst, c.wst, c.wn, n_sel, layers, nullptr, nullptr, c.st.rows, c.b.xp, c.b, c.s, ps,
                              seq_stride, n_keep)) != RK_OK)
    return e;
  return score_window(m, c, n_sel, nullptr, kl_pos, d_out);
}

rk_status rk_policy_damage(const rk_model* m, const rk_batch* batch, int32_t window_start, const int32_t* positions,
                           const int64_t* layer_offsets, int64_t seq_stride, const int32_t* n_keep, const void* state,
                           size_t state_bytes, float* d_out, float* kl_pos, float* logits_out, void* workspace,
                           size_t ws_bytes, void* stream) {
  rk_status e = check_batch(m, batch);
  if (e != RK_OK) return e;
  if ((e = check_window_model(m)) != RK_OK) return e;
  if (!layer_offsets || !n_keep || !state || !d_out || !workspace) {
    set_error("null layer_offsets, n_keep, state, d_out or workspace");
    return RK_ERR_ARG;
  }
  if ((e = check_policy(m, window_start, positions, layer_offsets, seq_stride, n_keep)) != RK_OK) return e;
  WinCall c;
  const uint32_t wf = RK_FLAG_CACHED_WINDOW | (logits_out ? RK_FLAG_UNFUSED_KL : 0);
  if ((e = win_call(m, batch, window_start, state, state_bytes, workspace, ws_bytes, 1, wf, stream, &c)) != RK_OK)
    return e;
  if ((e = window_policy_final(m, c.pst, c.wst, c.wn, positions, layer_offsets, seq_stride, n_keep, c.b.xp, c.b,
                               c.s)) != RK_OK)
    return e;
  return score_window(m, c, 1, logits_out, kl_pos, d_out);
}

rk_status rk_policy_damage_group(const rk_model* m, const rk_batch* batch, int32_t window_start, int32_t n_policies,
                                 const int32_t* const* positions, const int64_t* layer_offsets,
                                 const int64_t* seq_stride, const int32_t* n_keep, const void* state,
                                 size_t state_bytes, float* d_out, float* kl_pos, void* workspace, size_t ws_bytes,
                                 void* stream) {
  rk_status e = check_batch(m, batch);
  if (e != RK_OK) return e;
  if ((e = check_window_model(m)) != RK_OK) return e;
  if (!positions || !layer_offsets || !seq_stride || !n_keep || !state || !d_out || !workspace) {
    set_error("null positions, layer_offsets, seq_stride, n_keep, state, d_out or workspace");
    return RK_ERR_ARG;
  }
  if (n_policies < 1 || n_policies > RK_MAX_GROUP) { set_error("n_policies must be in [1, %d]", RK_MAX_GROUP); return RK_ERR_ARG; }
  const int L = m->cfg.n_layers;
  Policies pol{};
  for (int q = 0; q < n_policies; ++q) {
    pol.pos[q] = positions[q];
    pol.off[q] = layer_offsets + (size_t)q * L;
    pol.keep[q] = n_keep + (size_t)q * L;
    pol.stride[q] = seq_stride[q];
    if ((e = check_policy(m, window_start, pol.pos[q], pol.off[q], pol.stride[q], pol.keep[q])) != RK_OK) {
      set_error("policy %d: %s", q, rk_last_error());
      return e;
    }
  }
  WinCall c;
  if ((e = win_call(m, batch, window_start, state, state_bytes, workspace, ws_bytes, n_policies,
                    RK_FLAG_CACHED_WINDOW, stream, &c)) != RK_OK)
    return e;
  const int zero[RK_MAX_GROUP] = {0};   // every policy's pass starts at block 0
  if ((e = window_group_final(m, c.pst, c.wst, c.wn, n_policies, zero, nullptr, nullptr, c.st.rows, c.b.xp, c.b, c.s,
                              nullptr, 0, 0, &pol)) != RK_OK)
    return e;
  return score_window(m, c, n_policies, nullptr, kl_pos, d_out);
}

size_t rk_workspace_size(const rk_model* m, int64_t max_rows, int32_t max_group, uint32_t flags) {
  if (!m || max_rows < 1 || max_rows > kMaxRows || max_group < 1 || max_group > RK_MAX_GROUP) return 0;
  return ws_plan(m, max_rows, max_group, flags).total;
}

rk_status rk_reference_forward(const rk_model* m, const rk_batch* batch, void* clean_state, size_t clean_bytes,
                               void* workspace, size_t ws_bytes, void* stream) {
  rk_status e = check_batch(m, batch);
  if (e != RK_OK) return e;
  if (!clean_state || !workspace) { set_error("null clean state or workspace"); return RK_ERR_ARG; }
  SeqTable st;
  if ((e = make_table(m, batch, 0, batch->n_seqs, &st)) != RK_OK) return e;
  if (clean_bytes < clean_plan(m, st.rows).total) { set_error("clean state too small"); return RK_ERR_WORKSPACE; }
  const WsPlan wp = ws_plan(m, st.rows, 1, 0);
  if (ws_bytes < wp.total) { set_error("workspace too small (%zu < %zu)", ws_bytes, wp.total); return RK_ERR_WORKSPACE; }
  const Bufs b = carve(wp, workspace);
  hipStream_t s = (hipStream_t)stream;
  if ((e = reference_forward(m, batch->tokens, st, clean_view(m, st.rows, clean_state), b, s)) != RK_OK) return e;
  return write_state_tag(m, batch->tokens, st, -1, (char*)clean_state + clean_plan(m, st.rows).tag, s);
}

rk_status rk_profile_layer(const rk_model* m, const rk_batch* batch, int32_t layer, float alpha,
                           const rk_perturb_params* p, const void* clean_state, size_t clean_bytes, float* d_out,
                           float* kl_pos, float* logits_out, void* workspace, size_t ws_bytes, void* stream) {
  rk_status e = check_batch(m, batch);
  if (e != RK_OK) return e;
  if ((e = check_params(p)) != RK_OK) return e;
  if (!clean_state || !workspace || !d_out) { set_error("null clean state, workspace or d_out"); return RK_ERR_ARG; }
  if (layer < 0 || layer >= m->cfg.n_layers) { set_error("layer %d out of range", layer); return RK_ERR_ARG; }
  if (!(alpha >= 0.0f) || !isfinite(alpha)) { set_error("alpha must be finite and >= 0"); return RK_ERR_ARG; }
  SeqTable st;
  if ((e = make_table(m, batch, 0, batch->n_seqs, &st)) != RK_OK) return e;
  if ((e = check_windows(st, p->window_start)) != RK_OK) return e;
  const bool local = (p->flags & RK_FLAG_LOCAL_SIGNAL) != 0;
  if (local && logits_out) { set_error("RK_FLAG_LOCAL_SIGNAL produces no logits"); return RK_ERR_ARG; }
  const bool unfused = !local && (!m->bf16 || logits_out || (p->flags & RK_FLAG_UNFUSED_KL));
  const uint32_t wf = (unfused ? RK_FLAG_UNFUSED_KL : 0) | (local ? RK_FLAG_LOCAL_SIGNAL : 0);
  const int L = m->cfg.n_layers;
  const int64_t d = m->cfg.d_model;
  if (p->flags & RK_FLAG_CACHED_WINDOW) {
    if ((e = check_window_model(m)) != RK_OK) return e;
    SeqTable pst, wst;
    if ((e = window_tables(st, p->window_start, &pst, &wst)) != RK_OK) return e;
    if (clean_bytes < win_plan(m, st.rows).total) { set_error("window state too small"); return RK_ERR_WORKSPACE; }
    const WsPlan wp = ws_plan(m, st.rows, 1, wf | RK_FLAG_CACHED_WINDOW);
    if (ws_bytes < wp.total) { set_error("workspace too small (%zu < %zu)", ws_bytes, wp.total); return RK_ERR_WORKSPACE; }
    const Bufs b = carve(wp, workspace);
    const Win wn = win_view(m, st.rows, clean_state);
    hipStream_t s = (hipStream_t)stream;
    if ((p->flags & RK_FLAG_CHECK_STATE) &&
        (e = check_state_tag(m, batch->tokens, st, p->window_start,
                             (const char*)clean_state + win_plan(m, st.rows).tag, b.tag, s)) != RK_OK)
      return e;
    RK_TRY(launch_rope_table(b.rope, b.rope_pos, wst, m->cfg.head_dim, m->cfg.rope_theta, s, p->window_start));
    float* kl = kl_pos ? kl_pos : b.kl;
    if (local) {
      const float* h_last = nullptr;
      if (layer + 1 == L) {  // the state keeps no output of the last block: run it clean
        const KvPrefix pk = cache_prefix(m, wn, pst, layer, nullptr);
        if ((e = run_block(m, layer, wn.w.h + (size_t)layer * wst.rows * d, b.hloc, b, wst, nullptr, s, &pk)) != RK_OK)
          return e;
        h_last = b.hloc;
      }
      if ((e = window_local_pass(m, pst, wst, wn, layer, alpha, p, h_last, kl, b, s)) != RK_OK) return e;
    } else {
      if ((e = window_perturbed_final(m, pst, wst, wn, layer, alpha, p, b.xp, b, s)) != RK_OK) return e;
      if (unfused && (e = clean_logits(m, wst, wn.w, b.logits_c, s)) != RK_OK) return e;
      if ((e = score_group(m, wst, wn.w, b.xp, 1, unfused, logits_out ? logits_out : b.logits_p, kl, b, s)) != RK_OK)
        return e;
    }
    RK_TRY(launch_window_mean(kl, wst.rows, 1, wst, 0, d_out, s));
    return RK_OK;
  }
  if (clean_bytes < clean_plan(m, st.rows).total) { set_error("clean state too small"); return RK_ERR_WORKSPACE; }
  const WsPlan wp = ws_plan(m, st.rows, 1, wf);
  if (ws_bytes < wp.total) { set_error("workspace too small (%zu < %zu)", ws_bytes, wp.total); return RK_ERR_WORKSPACE; }
  const Bufs b = carve(wp, workspace);
  const Clean cl = clean_view(m, st.rows, clean_state);
  hipStream_t s = (hipStream_t)stream;
  if ((p->flags & RK_FLAG_CHECK_STATE) &&
      (e = check_state_tag(m, batch->tokens, st, -1, (const char*)clean_state + clean_plan(m, st.rows).tag, b.tag,
                           s)) != RK_OK)
    return e;
  RK_TRY(launch_rope_table(b.rope, b.rope_pos, st, m->cfg.head_dim, m->cfg.rope_theta, s));
  float* kl = kl_pos ? kl_pos : b.kl;
  if (local) {
    const float* h_last = nullptr;
    if (layer + 1 == L) {  // the clean state keeps no output of the last block: run it clean
      if ((e = run_block(m, layer, cl.h + (size_t)layer * st.rows * d, b.hloc, b, st, nullptr, s)) != RK_OK) return e;
      h_last = b.hloc;
    }
    if ((e = local_pass(m, batch->tokens, st, cl, layer, alpha, p, h_last, kl, b, s)) != RK_OK) return e;
  } else {
    if ((e = perturbed_final(m, batch->tokens, st, cl, layer, alpha, p, b.xp, b, s)) != RK_OK) return e;
    if (unfused && (e = clean_logits(m, st, cl, b.logits_c, s)) != RK_OK) return e;
    if ((e = score_group(m, st, cl, b.xp, 1, unfused, logits_out ? logits_out : b.logits_p, kl, b, s)) != RK_OK)
      return e;
  }
  RK_TRY(launch_window_mean(kl, st.rows, 1, st, p->window_start, d_out, s));
  return RK_OK;
}

rk_status rk_sensitivity_profile(const rk_model* m, const rk_batch* calib, const int32_t* layers, int32_t n_A,
                                 const float* alphas, int32_t n_alpha, const rk_perturb_params* p, int64_t max_rows,
                                 int32_t max_group, float* s_out, float* d_out, void* workspace, size_t ws_bytes,
                                 void* stream) {
  WsPlan wp;
  rk_status e = check_profile(m, calib, layers, n_A, alphas, n_alpha, p, max_rows, max_group, s_out, &wp);
  if (e != RK_OK) return e;
  if (!workspace) { set_error("null workspace"); return RK_ERR_ARG; }
  if (ws_bytes < wp.total) { set_error("workspace too small (%zu < %zu)", ws_bytes, wp.total); return RK_ERR_WORKSPACE; }
  const int N = calib->n_seqs;
  auto run = [&](hipStream_t s) -> rk_status {
    return profile_run(m, calib, layers, n_A, alphas, n_alpha, p, max_rows, max_group, s_out, d_out, wp, workspace, s);
  };
  if (!(p->flags & RK_FLAG_GRAPH)) return run((hipStream_t)stream);
  // the key: everything the launch sequence bakes in
  std::vector<uint64_t> key;
  auto put = [&](uint64_t v) { key.push_back(v); };
  put((uint64_t)(uintptr_t)m);
  put(m->ident);   // the config (dims, dtype, rotary theta, RMSNorm eps) and the weight pointers
  put((uint64_t)(uintptr_t)m->tok_emb); put((uint64_t)(uintptr_t)m->lm_head); put((uint64_t)(uintptr_t)m->final_norm);
  for (int l = 0; l < m->cfg.n_layers; ++l) {
    put((uint64_t)(uintptr_t)m->w_qkv[l]); put((uint64_t)(uintptr_t)m->w_o[l]);
    put((uint64_t)(uintptr_t)m->w_gate_up[l]); put((uint64_t)(uintptr_t)m->w_down[l]);
    put((uint64_t)(uintptr_t)m->attn_norm[l]); put((uint64_t)(uintptr_t)m->mlp_norm[l]);
  }
  put((uint64_t)(uintptr_t)calib->tokens); put((uint64_t)N); put((uint64_t)calib->seq_index0);
  for (int i = 0; i <= N; ++i) put((uint64_t)calib->offsets[i]);
  put((uint64_t)n_A);
  for (int j = 0; j < n_A; ++j) put((uint64_t)layers[j]);
  put((uint64_t)n_alpha);
  for (int a = 0; a < n_alpha; ++a) { uint32_t u; memcpy(&u, &alphas[a], 4); put(u); }
  put(p->seed); put((uint64_t)p->window_start); put((uint64_t)p->protect_head); put((uint64_t)p->protect_tail);
  put(p->flags); put((uint64_t)max_rows); put((uint64_t)max_group);
  put((uint64_t)(uintptr_t)s_out); put((uint64_t)(uintptr_t)d_out); put((uint64_t)(uintptr_t)workspace);
  put((uint64_t)ws_bytes);
  return run_graphed(key, run, (hipStream_t)stream);
}

rk_status rk_sensitivity_profile_static(const rk_model* m, const rk_batch* calib, const int32_t* layers,
                                        int32_t n_A, const float* alphas, int32_t n_alpha,
                                        const rk_perturb_params* p, int64_t max_rows, int32_t max_group,
                                        float* s_out, float* d_out, void* stream) {
  if (p && (p->flags & RK_FLAG_GRAPH)) {
    set_error("RK_FLAG_GRAPH is not available here: recording a graph allocates");
    return RK_ERR_ARG;
  }
  WsPlan wp;
  rk_status e = check_profile(m, calib, layers, n_A, alphas, n_alpha, p, max_rows, max_group, s_out, &wp);
  if (e != RK_OK) return e;
  if (wp.total > (size_t)RK_STATIC_SCRATCH_BYTES) {
    set_error("this profile needs %zu bytes of scratch (max_rows %lld, max_group %d); the allocation-free entry "
              "point holds %zu: use rk_sensitivity_profile with a workspace", wp.total, (long long)max_rows,
              max_group, (size_t)RK_STATIC_SCRATCH_BYTES);
    return RK_ERR_WORKSPACE;
  }
  void* scratch = nullptr;
  hipError_t he = static_scratch((hipStream_t)stream, &scratch);
  if (he != hipSuccess) {
    set_error("scratch address of this device: %s", hipGetErrorString(he));
    return RK_ERR_HIP;
  }
  // a timing session would create its events on first use; this entry point's launches are not timed
  struct Untimed {
    bool was = g_timing.on;
    Untimed() { g_timing.on = false; }
    ~Untimed() { g_timing.on = was; }
  } untimed;
  return profile_run(m, calib, layers, n_A, alphas, n_alpha, p, max_rows, max_group, s_out, d_out, wp, scratch,
                     (hipStream_t)stream);
}

rk_status rk_perturb_values(const rk_model* m, const rk_batch* batch, int32_t layer, float alpha,
                            const rk_perturb_params* p, void* v, int64_t row_stride, void* stream) {
  rk_status e = check_batch(m, batch);
  if (e != RK_OK) return e;
  if ((e = check_params(p)) != RK_OK) return e;
  if (!v) { set_error("null value buffer"); return RK_ERR_ARG; }
  if (layer < 0 || layer >= m->cfg.n_layers) { set_error("layer %d out of range", layer); return RK_ERR_ARG; }
  if (!(alpha >= 0.0f) || !isfinite(alpha)) { set_error("alpha must be finite and >= 0"); return RK_ERR_ARG; }
  if (row_stride < (int64_t)m->cfg.n_kv_heads * m->cfg.head_dim) { set_error("row_stride too small"); return RK_ERR_SHAPE; }
  // four values per vector access: 8-byte (bf16) or 16-byte (fp32) aligned rows
  if (row_stride % 4 != 0 || (uintptr_t)v % (m->bf16 ? 8 : 16) != 0) {
    set_error("v must be %d-byte aligned and row_stride a multiple of 4", m->bf16 ? 8 : 16);
    return RK_ERR_ARG;
  }
  SeqTable st;
  if ((e = make_table(m, batch, 0, batch->n_seqs, &st)) != RK_OK) return e;
  const rk_model_config& c = m->cfg;
  if (c.head_dim != 32 && c.head_dim != 64 && c.head_dim != 128) { set_error("head_dim unsupported"); return RK_ERR_UNSUPPORTED; }
  RK_TRY(launch_value_noise(v, m->bf16, row_stride, st, c.n_kv_heads, c.head_dim, layer, alpha, p->seed,
                            p->protect_head, p->protect_tail, (hipStream_t)stream));
  return RK_OK;
}

}  // extern "C"
