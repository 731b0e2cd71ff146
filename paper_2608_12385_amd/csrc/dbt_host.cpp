// Host side of the decode library: argument checking, workspace layout, the
// page allocator of the single primary KV cache, and the order in which the
// kernels of prefill, boundary and continuation steps are enqueued
// (Sec. 4.4 of the Decode-Branch Transformer paper).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <functional>
#include <numeric>
#include <new>
#include <queue>
#include <string>
#include <vector>

#include "../../include/dbt.h"
#include "host_internal.h"
#include "kernels.h"

using namespace dbt;

namespace {

thread_local std::string g_err;

dbt_status fail(dbt_status s, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return s;
}

#define HIPCHK(expr)                                                                         \
  do {                                                                                       \
    hipError_t e_ = (expr);                                                                  \
    if (e_ != hipSuccess) return fail(DBT_ERR_HIP, "%s: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

constexpr int kPage = 16;
// Decode attention reads a sequence of P pages in ceil(P / target) equal
// splits; 86 pages (1376 positions) keeps the splits long enough to amortise a
// workgroup's start, and e.g. 4097 positions (257 pages) in three equal splits.
// A model with few (sequence, KV head) pairs (max_batch x n_kv below 256)
// takes shorter splits, down to 16 pages, so that its longest caches fill
// about 512 workgroups.  The target is fixed when the model is created, so a
// row's result depends only on its own query and cache.
// The fp32 kernel holds a split's scores in LDS (at most 64 pages).
constexpr int kSplitTargetBf16 = 86, kSplitMinBf16 = 16, kSplitTargetF32 = 64, kSplitWideMin = 256;
constexpr int kMixChunk = 4096;

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }
int round16(int x) { return (x + 15) / 16 * 16; }
// Decode branches (App. C.1 for more than one); 0 reads as one branch.
int n_branches(const dbt_config &c) { return c.n_branches > 1 ? c.n_branches : 1; }

// Offsets (bytes) of every workspace buffer.
struct Layout {
  int Bp_max = 0, R_max = 0, rows_max = 0, max_in = 0, nqkv = 0, f = 0;
  GemmConfig g_qkv{1, 1, 1}, g_o{1, 1, 1}, g_gu{1, 1, 1}, g_d{1, 1, 1}, g_lm{1, 1, 1};
  int split_target = 0, max_splits = 0, nch = 0, nstat = 0;
  bool wide = false;  // attention splits in eight-wave workgroups (see the layout set-up)
  bool moe = false;
  // Decode gate/up on the fused SwiGLU kernel: fixed per model (from the
  // largest stacked call), so every call of a step sums each output element
  // in the same order whatever paths it carries.
  bool glu = false;
  int fe = 0, fs = 0, amax = 0;
  GemmConfig g_sgu{1, 1, 1}, g_sd{1, 1, 1};
  size_t moe_idx = 0, moe_logits = 0, moe_w = 0, moe_aslot = 0, moe_counts = 0, moe_offsets = 0, moe_arow = 0, moe_h = 0,
         moe_y = 0, ret_idx = 0;
  size_t rope = 0, pos = 0, S = 0, Xn = 0, Xh = 0, Q = 0, O = 0, P = 0, apart = 0, astat = 0,
         logits = 0, mstats = 0, xss = 0, ret_q = 0, ret_h = 0, ret_m = 0, ret_a = 0, btok = 0, slast = 0,
         state_total = 0, total = 0;  // [0, state_total): state; [state_total, total): step buffers
};

dbt_status check_config(const dbt_config *c) {
  if (!c) return fail(DBT_ERR_ARG, "config is NULL");
  if (c->n_layers <= 0 || c->d_model <= 0 || c->n_q_heads <= 0 || c->n_kv_heads <= 0 ||
      c->head_dim <= 0 || c->vocab < 0 || c->max_batch <= 0 || c->max_pos <= 0 || c->max_prompt < 0)
    return fail(DBT_ERR_ARG, "sizes must be positive");
  if (c->dtype != DBT_F32 && c->dtype != DBT_BF16) return fail(DBT_ERR_ARG, "dtype must be DBT_F32 or DBT_BF16");
  if (c->n_q_heads % c->n_kv_heads) return fail(DBT_ERR_SHAPE, "n_q_heads %% n_kv_heads != 0");
  if (c->head_dim % 4) return fail(DBT_ERR_SHAPE, "head_dim must be a multiple of 4");
  if (c->d_model % 4) return fail(DBT_ERR_SHAPE, "d_model must be a multiple of 4");
  if (c->d_model > 32768) return fail(DBT_ERR_UNSUPPORTED, "d_model above 32768");
  if (c->max_prompt > c->max_pos) return fail(DBT_ERR_SHAPE, "max_prompt > max_pos");
  if (c->n_experts > 0) {
    if (c->dtype != DBT_BF16) return fail(DBT_ERR_UNSUPPORTED, "MoE layers run in bf16 only");
    if (c->n_experts > 256 || c->d_model > 4096 || c->d_model % 512)
      return fail(DBT_ERR_UNSUPPORTED, "MoE needs n_experts <= 256 and d_model a multiple of 512 up to 4096");
    if (c->top_k1 < 1 || c->top_k1 > 8 || c->top_k2 < 1 || c->top_k2 > 8 || c->top_k1 > c->n_experts ||
        c->top_k2 > c->n_experts)
      return fail(DBT_ERR_ARG, "top_k1/top_k2 must be in [1, min(8, n_experts)]");
    if (c->replay && c->top_k2 != c->top_k1) return fail(DBT_ERR_ARG, "router replay needs top_k2 == top_k1");
    if (c->compute_matched != 0 && c->compute_matched != 1) return fail(DBT_ERR_ARG, "compute_matched must be 0 or 1");
    if (c->d_ff_expert <= 0 || c->d_ff_expert % 128 || c->d_ff_shared < 0 || c->d_ff_shared % 128)
      return fail(DBT_ERR_UNSUPPORTED, "expert widths must be multiples of 128");
  } else if (c->d_ff <= 0) {
    return fail(DBT_ERR_ARG, "d_ff must be positive");
  } else if (c->compute_matched) {
    return fail(DBT_ERR_UNSUPPORTED, "the compute-matched variant (App. B.3) is an MoE variant");
  }
  if (c->has_embeddings && c->vocab <= 0) return fail(DBT_ERR_SHAPE, "token inputs need a vocabulary");
  if (c->max_prompt > 0 && !c->has_embeddings) return fail(DBT_ERR_SHAPE, "prefill needs token inputs");
  if (!(c->rms_eps >= 0.f) || !(c->rope_theta > 0.f)) return fail(DBT_ERR_ARG, "bad rms_eps/rope_theta");
  if (c->n_branches < 0 || c->n_branches > 3) return fail(DBT_ERR_ARG, "n_branches must be in [0, 3]");
  if (c->n_branches > 1 && c->n_experts > 0)
    return fail(DBT_ERR_UNSUPPORTED, "more than one decode branch runs with dense MLPs only");
  const int G = c->n_q_heads / c->n_kv_heads, P = 1 + n_branches(*c);
  if (P * G > 16) return fail(DBT_ERR_UNSUPPORTED, "(1 + n_branches) * query heads per KV head exceeds 16");
  if (c->head_dim > 128) return fail(DBT_ERR_UNSUPPORTED, "head_dim > 128");
  if (c->dtype == DBT_BF16) {
    const int dq = c->n_q_heads * c->head_dim, dkv = c->n_kv_heads * c->head_dim;
    if (c->head_dim != 128) return fail(DBT_ERR_UNSUPPORTED, "bf16 attention needs head_dim 128");
    if (c->d_model % 128 || dq % 128 || (c->n_experts == 0 && c->d_ff % 128))
      return fail(DBT_ERR_UNSUPPORTED, "bf16 projections need d_model, n_q*d_h, d_ff multiples of 128");
    if (dkv % 64 || c->vocab % 64) return fail(DBT_ERR_UNSUPPORTED, "bf16 projections need n_kv*d_h, vocab multiples of 64");
  }
  return DBT_OK;
}

Layout make_layout(const dbt_config *c) {
  Layout L;
  const int d = c->d_model, dq = c->n_q_heads * c->head_dim, dkv = c->n_kv_heads * c->head_dim;
  L.moe = c->n_experts > 0;
  L.fe = c->d_ff_expert;
  L.fs = L.moe ? c->d_ff_shared : 0;
  L.f = L.moe ? std::max(L.fs, 128) : c->d_ff;
  L.Bp_max = round16(c->max_batch);
  L.R_max = (1 + n_branches(*c)) * L.Bp_max;
  L.rows_max = std::max(L.R_max, c->max_prompt);
  L.max_in = std::max(std::max(d, dq), L.f);
  L.nqkv = dq + 2 * dkv;
  L.g_qkv = gemm_config(L.nqkv, d, c->dtype, std::gcd(dq, dkv), L.R_max);
  L.g_o = gemm_config(d, dq, c->dtype, d, L.R_max);
  L.g_gu = gemm_config(2 * L.f, d, c->dtype, L.f, L.R_max);
  L.g_d = gemm_config(d, L.f, c->dtype, d, L.R_max);
  L.g_lm = gemm_config(std::max(c->vocab, 1), d, c->dtype, std::max(c->vocab, 1), L.R_max);
  L.g_lm.S = 1;  // the logits are written in place (one slab)
  L.glu = !L.moe && gemm_glu_ok(L.f, L.R_max, 1 + n_branches(*c), c->dtype);
  if (L.moe && L.fs > 0) {
    L.g_sgu = gemm_config(2 * L.fs, d, c->dtype, L.fs, L.R_max);
    L.g_sd = gemm_config(d, L.fs, c->dtype, d, L.R_max);
  }
  const int maxpages = (c->max_pos + kPage - 1) / kPage;
  if (c->dtype == DBT_BF16) {
    const int pairs = c->max_batch * c->n_kv_heads;
    const int want = pairs >= 256 ? 1 : (512 + pairs - 1) / pairs;  // splits per pair
    L.split_target = std::clamp((maxpages + want - 1) / want, kSplitMinBf16, kSplitTargetBf16);
    // long caches and few (sequence, KV head) pairs: one round of eight-wave
    // workgroups, each reading up to 1024 pages, instead of several rounds
    // of four-wave ones (fewer prologues, partial stores and splits to merge)
    const int want8 = (256 + pairs - 1) / pairs;
    const int target8 = (maxpages + want8 - 1) / want8;
    if (pairs < 256 && target8 >= kSplitWideMin) {
      L.wide = true;
      L.split_target = std::min(target8, 1024);
    }
  } else {
    L.split_target = kSplitTargetF32;
  }
  L.max_splits = (maxpages + L.split_target - 1) / L.split_target;
  L.nch = c->vocab > 0 ? (c->vocab + kMixChunk - 1) / kMixChunk : 0;
  size_t part = std::max({(size_t)L.g_qkv.S * L.R_max * L.nqkv, (size_t)L.g_o.S * L.R_max * d,
                          (size_t)L.g_gu.S * L.R_max * 2 * L.f, (size_t)L.g_d.S * L.R_max * d});
  if (L.moe) part = std::max({part, (size_t)L.g_sgu.S * L.R_max * 2 * L.f, (size_t)L.g_sd.S * L.R_max * d});
  part = std::max(part, (size_t)c->max_prompt * std::max({L.nqkv, d, 2 * L.f}));
  size_t o = 0;
  auto take = [&](size_t bytes) { size_t at = o; o += align256(bytes); return at; };
  // State kept between calls: the RoPE table, positions, the primary
  // intermediates retained for a later branch evaluation, the boundary's
  // token and residual.
  L.rope = take((size_t)c->max_pos * (c->head_dim / 2) * 2 * sizeof(float));
  L.pos = take((size_t)c->max_batch * sizeof(int));
  L.ret_q = take((size_t)c->n_layers * L.Bp_max * dq * 4);
  L.ret_h = take((size_t)c->n_layers * L.Bp_max * L.f * 4);
  L.ret_m = take((size_t)c->n_layers * L.Bp_max * d * 4);
  L.ret_a = take(c->compute_matched ? (size_t)c->n_layers * L.Bp_max * d * 4 : 0);
  if (L.moe) L.ret_idx = take((size_t)c->n_layers * L.Bp_max * 8 * 4);
  L.btok = take((size_t)c->max_batch * 4);
  L.slast = take((size_t)L.Bp_max * d * 4);
  // Step buffers: written and read within one call (every element a call
  // reads is written earlier in the same call, apart from padding rows whose
  // results are never used), so any memory of this size can hold them.
  o = align256(o);
  L.state_total = o;
  L.S = take((size_t)L.rows_max * d * 4);
  L.Xn = take((size_t)L.rows_max * L.max_in * 4);
  L.Xh = take((size_t)L.rows_max * L.f * 4);
  L.Q = take((size_t)L.rows_max * dq * 4);
  L.O = take((size_t)L.rows_max * dq * 4);
  L.P = take(part * 4);
  L.apart = take((size_t)c->max_batch * c->n_kv_heads * L.max_splits * 16 * c->head_dim * 4);
  L.astat = take((size_t)c->max_batch * c->n_kv_heads * L.max_splits * 16 * 2 * 4);
  L.logits = take((size_t)L.R_max * std::max(c->vocab, 1) * 4);
  L.nstat = gemm_stats_tiles(std::max(c->vocab, 1), L.g_lm, c->dtype);
  if (L.nstat == 0) L.nstat = std::max(L.nch, 1);
  L.mstats = take((size_t)L.R_max * L.nstat * 3 * 4);
  L.xss = take((size_t)std::max(L.g_qkv.S, 1) * L.R_max * 4);
  if (L.moe) {
    L.amax = L.rows_max * 8;
    L.moe_idx = take((size_t)L.rows_max * 8 * 4);
    L.moe_logits = take((size_t)L.rows_max * 256 * 4);
    L.moe_w = take((size_t)L.rows_max * 8 * 4);
    L.moe_aslot = take((size_t)L.rows_max * 8 * 4);
    L.moe_counts = take((size_t)c->n_experts * 4);
    L.moe_offsets = take((size_t)(c->n_experts + 1) * 4);
    L.moe_arow = take((size_t)L.amax * 4);
    L.moe_h = take((size_t)L.amax * L.fe * 2);
    L.moe_y = take((size_t)L.amax * d * 4);
  }
  L.total = o;
  return L;
}

}  // namespace

struct StageTimer {
  bool on = false;
  std::vector<std::pair<hipEvent_t, hipEvent_t>> ev;
  size_t used = 0;
};

struct dbt_model {
  StageTimer timers[DBT_STAGE_COUNT];
  // Second stream for the MoE shared expert, which runs beside the routing
  // chain (created by the first MoE layer of a call that may create it;
  // default priority), and the events of its fork and join.
  hipStream_t side = nullptr;
  hipEvent_t ev_fork = nullptr, ev_join = nullptr;
  bool no_fork = false;  // the current call creates no stream (allocation-free entry point)
  ~dbt_model() {
    for (auto &t : timers)
      for (auto &e : t.ev) {
        (void)hipEventDestroy(e.first);
        (void)hipEventDestroy(e.second);
      }
    if (ev_fork) (void)hipEventDestroy(ev_fork);
    if (ev_join) (void)hipEventDestroy(ev_join);
    if (side) (void)hipStreamDestroy(side);
  }
  dbt_config cfg;
  dbt_weights w;
  std::vector<dbt_layer_weights> layers;
  char *ws = nullptr;
  Layout L;
  std::vector<float> rope_host;
  bool dev_ready = false;
  // boundary state: set by dbt_prefill(run_boundary = 0)
  const dbt_kv *bnd_kv = nullptr;
  int bnd_batch = 0;
  // Step buffers of the current call: the workspace's own step region, or
  // memory a call supplies for them (see decode_step_in).
  char *step = nullptr;
  char *p(size_t off) const { return off >= L.state_total ? step + (off - L.state_total) : ws + off; }
  template <typename T> T *at(size_t off) const { return (T *)p(off); }
};

struct dbt_kv {
  dbt_model *m;
  char *k, *v;
  int num_pages;
  int *page_table;
  int mpps;
  std::priority_queue<int, std::vector<int>, std::greater<int>> free_pages;
  std::vector<std::vector<int>> table;
  std::vector<int> len;
  struct Upd { int b, slot, page; };
  std::vector<Upd> pending;

  int take_page() {
    const int p = free_pages.top();
    free_pages.pop();
    return p;
  }
};

namespace {

size_t esize(const dbt_config &c) { return c.dtype == DBT_BF16 ? 2 : 4; }

// Records an event pair around the launches made during its lifetime when
// timing is enabled for the stage (a measurement aid; failures are ignored).
class Timed {
 public:
  Timed(dbt_model *m, int stage, hipStream_t st) : st_(st) {
    StageTimer &t = m->timers[stage];
    if (!t.on) return;
    if (t.used == t.ev.size()) {
      hipEvent_t a, b;
      if (hipEventCreate(&a) != hipSuccess) return;
      if (hipEventCreate(&b) != hipSuccess) { (void)hipEventDestroy(a); return; }
      t.ev.emplace_back(a, b);
    }
    pair_ = &t.ev[t.used++];
    (void)hipEventRecord(pair_->first, st_);
  }
  ~Timed() {
    if (pair_) (void)hipEventRecord(pair_->second, st_);
  }

 private:
  hipStream_t st_;
  std::pair<hipEvent_t, hipEvent_t> *pair_ = nullptr;
};

// K/V pages of one layer.
KVRef kv_layer(const dbt_kv *kv, int l) {
  const dbt_config &c = kv->m->cfg;
  KVRef r;
  const size_t per_layer = (size_t)kv->num_pages * c.n_kv_heads * kPage * c.head_dim * esize(c);
  r.k = kv->k + per_layer * l;
  r.v = kv->v + per_layer * l;
  r.page_table = kv->page_table;
  r.mpps = kv->mpps;
  r.n_kv = c.n_kv_heads;
  r.d_h = c.head_dim;
  return r;
}

dbt_status ensure_device(dbt_model *m, hipStream_t st) {
  if (m->dev_ready) return DBT_OK;
  HIPCHK(hipMemsetAsync(m->ws, 0, m->L.total, st));
  HIPCHK(hipMemcpyAsync(m->p(m->L.rope), m->rope_host.data(), m->rope_host.size() * sizeof(float),
                        hipMemcpyHostToDevice, st));
  m->dev_ready = true;
  return DBT_OK;
}

// Enqueue pending page-table entries and (optionally) per-sequence positions.
// With `fold` the last block is returned there instead of launched, for the
// caller to pass to the step's first kernel.
dbt_status flush(dbt_kv *kv, const int *h_pos, int npos, hipStream_t st, StepBegin *fold = nullptr) {
  dbt_model *m = kv->m;
  size_t ip = 0;
  int ipos = 0;
  if (fold) {
    fold->n_pos = fold->n_pt = 0;
    fold->b0 = 0;
  }
  while (ip < kv->pending.size() || ipos < npos) {
    StepBegin sb;
    std::memset(&sb, 0, sizeof sb);
    sb.b0 = ipos;
    sb.n_pos = std::min(64, npos - ipos);
    for (int i = 0; i < sb.n_pos; ++i) sb.pos[i] = h_pos[ipos + i];
    ipos += sb.n_pos;
    sb.n_pt = (int)std::min<size_t>(64, kv->pending.size() - ip);
    for (int i = 0; i < sb.n_pt; ++i) {
      sb.pt_b[i] = kv->pending[ip + i].b;
      sb.pt_slot[i] = kv->pending[ip + i].slot;
      sb.pt_page[i] = kv->pending[ip + i].page;
    }
    ip += sb.n_pt;
    if (fold && ip >= kv->pending.size() && ipos >= npos) {
      *fold = sb;
      break;
    }
    HIPCHK(launch_step_begin(sb, m->at<int>(m->L.pos), kv->page_table, kv->mpps, st));
  }
  kv->pending.clear();
  return DBT_OK;
}

// One layer for the active rows.  rows_layout: rows of the partial slabs.
struct LayerCall {
  Rows rows;
  int mode;
  bool retain;
  int ret_src, ret_dst;
  bool prefill;
  int seq;           // prefill: the sequence
  int rows_layout;   // prefill: T; decode: (1 + n_branches)*Bp
  bool last_norm;    // apply the next norm after the layer
  const dbt_step_out *out;  // routing outputs (MoE), may be NULL
  // layer 0 reads its rows straight from the step inputs (XNorm; no norm
  // kernel before it) when set; sb is then applied by its QKV projection
  const HIn *hin;
  const StepBegin *sb;
};

// Whether the decode step's attention kernel finishes the QKV projection
// (split-K sums, rotary embedding, query coupling, cache append) for a batch
// of B sequences whose longest cache is maxlen positions after the append.
bool attn_finishes_qkv(const dbt_model *m, int B, int maxlen, bool *single_out = nullptr);

// Whether the first layer of a layer-only model takes its rows straight from
// the step inputs (XNorm) for a decode step of B sequences.  Decided from
// the model and batch only, so the grouped, primary-only and two-pass steps
// (and a branch pass) all use the same arithmetic for a row.
bool input_fold(const dbt_model *m, const dbt_kv *kv, int B);

bool attn_finishes_qkv(const dbt_model *m, int B, int maxlen, bool *single_out) {
  const dbt_config &cf = m->cfg;
  const bool single = cf.dtype == DBT_BF16 && B * cf.n_kv_heads >= 256 && (maxlen + kPage - 1) / kPage <= 1024;
  if (single_out) *single_out = single;
  return cf.dtype == DBT_BF16 && cf.head_dim == 128 && cf.n_q_heads / cf.n_kv_heads <= (single || m->L.wide ? 8 : 4);
}

bool input_fold(const dbt_model *m, const dbt_kv *kv, int B) {
  const dbt_config &cf = m->cfg;
  if (cf.has_embeddings || cf.dtype != DBT_BF16 || cf.d_model % 128) return false;
  int maxlen = 0;
  for (int b = 0; b < B; ++b) maxlen = std::max(maxlen, kv->len[b] + 1);
  // the largest call of a step: every path's rows, or the primary's alone
  // when only it attends (compute-matched)
  const int Bp = round16(B), M = (cf.compute_matched ? 1 : 1 + n_branches(cf)) * Bp;
  return attn_finishes_qkv(m, B, maxlen) && gemm_xnorm_ok(m->L.g_qkv, M);
}

// MoE MLP of layer l for the active rows: route, dispatch, touched experts,
// shared expert (with the b coupling), combine (with the c coupling).
dbt_status run_moe_mlp(dbt_model *m, int l, const LayerCall &c, hipStream_t st) {
  const dbt_config &cf = m->cfg;
  const Layout &L = m->L;
  const dbt_layer_weights &W = m->layers[l];
  const int d = cf.d_model, fs = L.fs;
  const int xrow0 = c.rows.p0 * c.rows.Bp;
  const int M = c.rows.np * c.rows.Bp;
  const size_t es = esize(cf);
  float *P = m->at<float>(L.P), *S = m->at<float>(L.S);
  const size_t rq = (size_t)l * L.Bp_max;
  float *ret_h = m->at<float>(L.ret_h) + rq * L.f;
  float *ret_m = m->at<float>(L.ret_m) + rq * d;
  int *ret_idx = m->at<int>(L.ret_idx) + rq * 8;
  const int k2 = cf.replay ? cf.top_k1 : cf.top_k2;
  MoeRoute ro{};
  ro.Sbar = S;
  ro.g = W.mlp_norm;
  ro.eps = cf.rms_eps;
  ro.d = d;
  ro.Wr = W.router;
  ro.E = cf.n_experts;
  ro.k1 = cf.top_k1;
  ro.k2 = k2;
  ro.replay = cf.replay;
  ro.rows = c.rows;
  ro.mode = c.mode;
  ro.logits = m->at<float>(L.moe_logits);
  ro.idx = m->at<int>(L.moe_idx);
  ro.wts = m->at<float>(L.moe_w);
  ro.idx1_in = ret_idx;
  if (c.out && !c.prefill) {
    const size_t B = c.rows.B;
    ro.out_idx1 = c.out->route_idx1 ? c.out->route_idx1 + (size_t)l * B * cf.top_k1 : nullptr;
    ro.out_w1 = c.out->route_w1 ? c.out->route_w1 + (size_t)l * B * cf.top_k1 : nullptr;
    ro.out_idx2 = c.out->route_idx2 ? c.out->route_idx2 + (size_t)l * B * k2 : nullptr;
    ro.out_w2 = c.out->route_w2 ? c.out->route_w2 + (size_t)l * B * k2 : nullptr;
    const size_t E = cf.n_experts;
    ro.out_lg1 = c.out->route_logits1 ? c.out->route_logits1 + (size_t)l * B * E : nullptr;
    ro.out_lg2 = c.out->route_logits2 ? c.out->route_logits2 + (size_t)l * B * E : nullptr;
  }
  ro.ret_idx = c.retain ? ret_idx : nullptr;
  ro.ret_src = c.ret_src;
  ro.ret_dst = c.ret_dst;
  // The shared expert needs only the normed rows: it runs on a second stream
  // beside the routing chain (router, top-k, dispatch: short kernels that
  // leave most compute units idle) and the routed experts; the combine waits
  // for both.  Neither side writes what the other reads (shared: P, Xh;
  // routed: the MoE buffers).
  struct Fork {
    dbt_model *m;
    hipStream_t st;
    bool on;
    ~Fork() {
      if (!on) return;
      (void)hipEventRecord(m->ev_join, m->side);
      (void)hipStreamWaitEvent(st, m->ev_join, 0);
    }
  } fork{m, st, false};
  hipStream_t sst = st;
  const bool has_shared = fs > 0 && !(cf.compute_matched && c.mode == MODE_BRANCH);
  if (has_shared && !m->no_fork) {
    if (!m->side) {
      HIPCHK(hipStreamCreateWithFlags(&m->side, hipStreamNonBlocking));
      // device-scope release: the hand-off is between two queues of one GPU
      // (a system-scope release would also write the caches back for the host)
      HIPCHK(hipEventCreateWithFlags(&m->ev_fork, hipEventDisableTiming | hipEventReleaseToDevice));
      HIPCHK(hipEventCreateWithFlags(&m->ev_join, hipEventDisableTiming | hipEventReleaseToDevice));
    }
    HIPCHK(hipEventRecord(m->ev_fork, st));
    HIPCHK(hipStreamWaitEvent(m->side, m->ev_fork, 0));
    sst = m->side;
    fork.on = true;
  }
  // shared expert: dense SwiGLU of width fs with the b coupling on its
  // intermediate; compute-matched variant (App. B.3): primary rows only
  const bool cm = cf.compute_matched != 0;
  const Rows srows = cm ? Rows{c.rows.B, c.rows.Bp, 0, 1} : c.rows;
  const int smode = cm ? (int)MODE_PRIMARY : c.mode;
  const int sxrow0 = srows.p0 * srows.Bp, sM = srows.np * srows.Bp;
  long long stride = (long long)c.rows_layout * d;
  int S_sh = 0;
  if (fs > 0 && !(cm && c.mode == MODE_BRANCH)) {
    GemmConfig g_sgu = L.g_sgu, g_sd = L.g_sd;
    if (c.prefill) g_sgu.S = g_sd.S = 1;
    WSegs gu{{W.s_gate, W.s_up, nullptr}, {fs, fs, 0}};
    long long st_gu = (long long)c.rows_layout * 2 * fs;
    HIPCHK(launch_gemm(gu, 2 * fs, d, cf.dtype, m->p(L.Xn) + (size_t)sxrow0 * d * es, d, sM,
                       P + (size_t)sxrow0 * 2 * fs, 2 * fs, st_gu, g_sgu, sst));
    HIPCHK(launch_swiglu_finish(P, st_gu, g_sgu.S, 2 * fs, fs, smode, srows, W.b, ret_h,
                                Retain{c.retain && !cm ? ret_h : nullptr, c.ret_src, c.ret_dst}, cf.dtype,
                                m->p(L.Xh), fs, sst));
    WSegs sd{{W.s_down, nullptr, nullptr}, {d, 0, 0}};
    HIPCHK(launch_gemm(sd, d, fs, cf.dtype, m->p(L.Xh) + (size_t)sxrow0 * fs * es, fs, sM, P + (size_t)sxrow0 * d,
                       d, stride, g_sd, sst));
    S_sh = g_sd.S;
  }
  HIPCHK(launch_moe_route(ro, st));
  MoeDispatch di{};
  di.idx = ro.idx;
  di.rows = c.rows;
  di.k1 = cf.top_k1;
  di.k2 = k2;
  di.E = cf.n_experts;
  di.counts = m->at<int>(L.moe_counts);
  di.offsets = m->at<int>(L.moe_offsets);
  di.arow = m->at<int>(L.moe_arow);
  di.aslot = m->at<int>(L.moe_aslot);
  HIPCHK(launch_moe_dispatch(di, st));
  const int max_rows = c.rows.np * c.rows.B;
  {
    Timed tm(m, DBT_STAGE_GATEUP, st);
    MoeGemm g{};
    g.X = m->p(L.Xn);
    g.ldx = d;
    g.W0 = W.x_gate;
    g.W1 = W.x_up;
    g.E = cf.n_experts;
    g.N = L.fe;
    g.K = d;
    g.counts = di.counts;
    g.offsets = di.offsets;
    g.arow = di.arow;
    g.Y = m->p(L.moe_h);
    g.ldy = L.fe;
    HIPCHK(launch_moe_gemm(g, true, max_rows, st));
  }
  {
    Timed tm(m, DBT_STAGE_DOWN, st);
    MoeGemm g{};
    g.X = m->p(L.moe_h);
    g.ldx = L.fe;
    g.W0 = W.x_down;
    g.E = cf.n_experts;
    g.N = d;
    g.K = L.fe;
    g.counts = di.counts;
    g.offsets = di.offsets;
    g.arow = di.arow;
    g.Y = m->p(L.moe_y);
    g.ldy = d;
    HIPCHK(launch_moe_gemm(g, false, max_rows, st));
  }
  if (fork.on) {
    HIPCHK(hipEventRecord(m->ev_join, m->side));
    HIPCHK(hipStreamWaitEvent(st, m->ev_join, 0));
    fork.on = false;
  }
  const float *g_next = nullptr;
  if (l + 1 < cf.n_layers) g_next = m->layers[l + 1].attn_norm;
  else if (cf.vocab > 0 && c.last_norm) g_next = m->w.final_norm;
  MoeCombine cb{};
  cb.rows = c.rows;
  cb.mode = c.mode;
  cb.d = d;
  cb.k1 = cf.top_k1;
  cb.k2 = k2;
  cb.idx = ro.idx;
  cb.wts = ro.wts;
  cb.aslot = di.aslot;
  cb.Yexp = m->at<float>(L.moe_y);
  cb.part = P;
  cb.stride = stride;
  cb.S_sh = S_sh;
  cb.c = W.c;
  cb.M1_in = ret_m;  // compute-matched: the kept G1
  cb.ret = Retain{c.retain ? ret_m : nullptr, c.ret_src, c.ret_dst};
  cb.gG = cm ? W.g_shared_copy : nullptr;
  cb.S = S;
  cb.g_next = g_next;
  cb.eps = cf.rms_eps;
  cb.Xn = m->p(L.Xn);
  cb.ldx = d;
  HIPCHK(launch_moe_combine(cb, cf.dtype, st));
  return DBT_OK;
}

dbt_status run_layer(dbt_model *m, dbt_kv *kv, int l, const LayerCall &c, hipStream_t st) {
  const dbt_config &cf = m->cfg;
  const Layout &L = m->L;
  const dbt_layer_weights &W = m->layers[l];
  const int d = cf.d_model, dq = cf.n_q_heads * cf.head_dim, dkv = cf.n_kv_heads * cf.head_dim, f = L.f;
  const size_t es = esize(cf);
  const int xrow0 = c.rows.p0 * c.rows.Bp;
  const int M = c.rows.np * c.rows.Bp;
  char *Xn = m->p(L.Xn), *Xh = m->p(L.Xh), *O = m->p(L.O);
  float *P = m->at<float>(L.P), *S = m->at<float>(L.S), *Q = m->at<float>(L.Q);
  // prompt-wide rows: no reduction split (plenty of row tiles)
  auto cfg = [&](GemmConfig g) { if (c.prefill) g.S = 1; return g; };
  // A projection of the active rows: the 256-row tiled kernel over a whole
  // prompt, the weight-streaming kernel otherwise.
  auto project = [&](const WSegs &segs, int N, int K, const char *X, int ldx, int rows_M, float *Y, int ldy,
                     long long y_stride, const GemmConfig &g) -> hipError_t {
    TileGemm tg{};
    for (int i = 0; i < 3; ++i) {
      tg.w[i] = (const uint16_t *)segs.w[i];
      tg.rows[i] = segs.rows[i];
    }
    tg.N = N;
    tg.K = K;
    tg.X = (const uint16_t *)X;
    tg.ldx = ldx;
    tg.M = rows_M;
    tg.Y = Y;
    tg.ldy = ldy;
    if (c.prefill && cf.dtype == DBT_BF16 && gemm_tile_args_ok(tg, false)) return launch_gemm_tile(tg, false, st);
    return launch_gemm(segs, N, K, cf.dtype, X, ldx, rows_M, Y, ldy, y_stride, g, st);
  };
  const GemmConfig g_qkv = cfg(L.g_qkv), g_o = cfg(L.g_o), g_gu = cfg(L.g_gu), g_d = cfg(L.g_d);
  const int S_qkv = g_qkv.S, S_o = g_o.S, S_gu = g_gu.S, S_d = g_d.S;
  KVRef kvl = kv_layer(kv, l);
  const size_t rq = (size_t)l * L.Bp_max;
  float *ret_q = m->at<float>(L.ret_q) + rq * dq;
  float *ret_h = m->at<float>(L.ret_h) + rq * f;
  float *ret_m = m->at<float>(L.ret_m) + rq * d;
  // Compute-matched variant (App. B.3): attention runs on the primary rows
  // only and the branch takes g_A * A1 in the residual step.
  const bool cm = cf.compute_matched != 0;
  float *ret_a = cm ? m->at<float>(L.ret_a) + rq * d : nullptr;
  const HIn hin0 = l == 0 && c.hin ? *c.hin : HIn{};
  if (cm && c.mode == MODE_BRANCH) {
    if (hin0.h1 && c.sb) HIPCHK(launch_step_begin(*c.sb, m->at<int>(L.pos), kv->page_table, kv->mpps, st));
    HIPCHK(launch_resid_norm(P, 0, 0, d, S, W.mlp_norm, cf.rms_eps, d, cf.dtype, c.rows, Xn, d, st,
                             GatedCopy{W.g_attn_copy, ret_a, Retain{}}, hin0));
    return run_moe_mlp(m, l, c, st);
  }
  const Rows arows = cm ? Rows{c.rows.B, c.rows.Bp, 0, 1} : c.rows;
  const int amode = cm ? (int)MODE_PRIMARY : c.mode;
  const int axrow0 = arows.p0 * arows.Bp, aM = arows.np * arows.Bp;

  // 1. stacked QKV projection (branch rows need only W_Q)
  WSegs qkv{};
  int nq;
  if (amode == MODE_BRANCH) {
    qkv = WSegs{{W.wq, nullptr, nullptr}, {dq, 0, 0}};
    nq = dq;
  } else {
    qkv = WSegs{{W.wq, W.wk, W.wv}, {dq, dkv, dkv}};
    nq = L.nqkv;
  }
  long long stride = (long long)c.rows_layout * nq;
  // A whole prompt: the tiled projection applies the rotary embedding and
  // writes Q and the cache itself (no fp32 Q/K/V slab, no finish kernel).
  TileGemm tq{};
  if (c.prefill && amode == MODE_PRIMARY && cf.dtype == DBT_BF16) {
    for (int i = 0; i < 3; ++i) {
      tq.w[i] = (const uint16_t *)qkv.w[i];
      tq.rows[i] = qkv.rows[i];
    }
    tq.N = nq;
    tq.K = d;
    tq.X = (const uint16_t *)(Xn + (size_t)axrow0 * d * es);
    tq.ldx = d;
    tq.M = aM;
    tq.rope = m->at<float2>(L.rope);
    tq.Qout = Q;
    tq.kv = kvl;
    tq.seq = c.seq;
    tq.ret = c.retain && !cm ? ret_q : nullptr;
    tq.ret_src = c.ret_src;
    tq.ret_dst = c.ret_dst;
  }
  const bool qkv_fused = tq.rope && gemm_tile_args_ok(tq, false);
  // Decode on the bf16 cache: the attention kernel finishes the queries and
  // appends the cache entry itself.
  int maxlen = 0;
  if (!c.prefill)
    for (int b = 0; b < c.rows.B; ++b) maxlen = std::max(maxlen, kv->len[b] + 1);
  bool attn_single = false;
  const bool finish_in_attn = !c.prefill && attn_finishes_qkv(m, c.rows.B, maxlen, &attn_single);
  const bool xin = l == 0 && c.hin && c.hin->h1;
  if (xin && (c.prefill || !finish_in_attn || cf.dtype != DBT_BF16 || !gemm_xnorm_ok(g_qkv, aM)))
    return fail(DBT_ERR_STATE, "internal: first-layer input fold on an unsupported call");
  if (qkv_fused) {
    Timed tm(m, DBT_STAGE_QKV, st);
    HIPCHK(launch_gemm_tile(tq, false, st));
  } else if (xin) {
    XNorm xn{};
    xn.h = *c.hin;
    xn.rows = arows;
    xn.g = W.attn_norm;
    xn.ss = m->at<float>(L.xss);
    xn.ss_ld = L.R_max;
    if (c.sb) {
      xn.sb = *c.sb;
      xn.pos_arr = m->at<int>(L.pos);
      xn.page_table = kv->page_table;
      xn.mpps = kv->mpps;
    }
    Timed tm(m, DBT_STAGE_QKV, st);
    HIPCHK(launch_gemm_xnorm(qkv, nq, d, xn, aM, P + (size_t)axrow0 * nq, nq, stride, g_qkv, st));
  } else {
    Timed tm(m, DBT_STAGE_QKV, st);
    HIPCHK(project(qkv, nq, d, Xn + (size_t)axrow0 * d * es, d, aM, P + (size_t)axrow0 * nq, nq, stride, g_qkv));
  }
  QKVFinish qf{};
  qf.part = P;
  qf.split_stride = stride;
  qf.S = S_qkv;
  qf.ldp = nq;
  qf.n_q = cf.n_q_heads;
  qf.n_kv = cf.n_kv_heads;
  qf.d_h = cf.head_dim;
  qf.rows = arows;
  qf.mode = amode;
  qf.rope = m->at<float2>(L.rope);
  qf.pos_arr = c.prefill ? nullptr : m->at<int>(L.pos);
  qf.seq_fixed = c.seq;
  qf.a = W.a;
  qf.Q = Q;
  qf.Q1_in = ret_q;
  qf.ret = Retain{c.retain && !cm ? ret_q : nullptr, c.ret_src, c.ret_dst};
  qf.kv = kvl;
  qf.dtype = cf.dtype;
  if (xin) {
    qf.ss = m->at<float>(L.xss);
    qf.ss_ld = L.R_max;
    qf.ss_S = S_qkv;
    qf.d_model = d;
    qf.eps = cf.rms_eps;
  }
  if (!qkv_fused && !finish_in_attn) HIPCHK(launch_qkv_finish(qf, st));

  // 2. attention over the primary cache
  if (c.prefill) {
    HIPCHK(launch_attn_prefill(Q, dq, c.rows.B, kvl, c.seq, cf.n_q_heads, cf.dtype, O, dq, st));
  } else {
    AttnArgs aa{};
    aa.Q = Q;
    aa.kv = kvl;
    aa.pos_arr = m->at<int>(L.pos);
    aa.rows = arows;
    aa.n_q = cf.n_q_heads;
    aa.pages_per_split = L.split_target;
    aa.max_splits = L.max_splits;
    aa.opart = m->at<float>(L.apart);
    aa.ostat = m->at<float>(L.astat);
    aa.dtype = cf.dtype;
    // When the batch fills the chip (B x n_kv >= 256 workgroups), each
    // (sequence, KV head) is read by one eight-wave workgroup and no partials
    // are merged.  The choice depends on the batch, never on the branch.
    aa.single = attn_single;
    aa.wide = L.wide;
    aa.fused = finish_in_attn;
    aa.fin = qf;
    aa.O = O;
    aa.ldo = dq;
    {
      Timed tm(m, DBT_STAGE_ATTN, st);
      HIPCHK(launch_attn_decode(aa, st));
    }
    if (!aa.single) HIPCHK(launch_attn_combine(aa, O, dq, st));
  }

  // 3. output projection + residual + MLP norm
  WSegs wo{{W.wo, nullptr, nullptr}, {d, 0, 0}};
  stride = (long long)c.rows_layout * d;
  {
    Timed tm(m, DBT_STAGE_WO, st);
    HIPCHK(project(wo, d, dq, O + (size_t)axrow0 * dq * es, dq, aM, P + (size_t)axrow0 * d, d, stride, g_o));
  }
  const GatedCopy gca = cm ? GatedCopy{W.g_attn_copy, ret_a, Retain{c.retain ? ret_a : nullptr, c.ret_src, c.ret_dst}}
                           : GatedCopy{};
  HIPCHK(launch_resid_norm(P, stride, S_o, d, S, W.mlp_norm, cf.rms_eps, d, cf.dtype, c.rows, Xn, d, st, gca, hin0));

  if (L.moe) return run_moe_mlp(m, l, c, st);

  // 4. gate/up + SwiGLU + b coupling (fused into the projection's epilogue
  // when the tiles fill the chip)
  const Retain ret_h_keep{c.retain ? ret_h : nullptr, c.ret_src, c.ret_dst};
  TileGemm tg{};
  if (c.prefill && c.mode == MODE_PRIMARY && c.rows.np == 1 && cf.dtype == DBT_BF16) {
    tg.w[0] = (const uint16_t *)W.w_gate;
    tg.w[1] = (const uint16_t *)W.w_up;
    tg.rows[0] = tg.rows[1] = f;
    tg.N = f;
    tg.K = d;
    tg.X = (const uint16_t *)(Xn + (size_t)xrow0 * d * es);
    tg.ldx = d;
    tg.M = M;
    tg.H = (uint16_t *)(Xh + (size_t)xrow0 * f * es);
    tg.ldh = f;
    tg.ret = ret_h_keep.ptr;
    tg.ret_src = ret_h_keep.src_row;
    tg.ret_dst = ret_h_keep.dst_row;
  }
  if (tg.w[0] && gemm_tile_args_ok(tg, true)) {
    Timed tm(m, DBT_STAGE_GATEUP, st);
    HIPCHK(launch_gemm_tile(tg, true, st));
  } else if (c.prefill ? gemm_glu_ok(f, M, c.rows.np, cf.dtype) : L.glu) {
    const GluEpi ep{c.rows, c.mode, f, W.b, ret_h, ret_h_keep, (uint16_t *)Xh, f};
    Timed tm(m, DBT_STAGE_GATEUP, st);
    HIPCHK(launch_gemm_glu((const uint16_t *)W.w_gate, (const uint16_t *)W.w_up, f, d, Xn + (size_t)xrow0 * d * es,
                           d, M, ep, st));
  } else {
    WSegs gu{{W.w_gate, W.w_up, nullptr}, {f, f, 0}};
    stride = (long long)c.rows_layout * 2 * f;
    {
      Timed tm(m, DBT_STAGE_GATEUP, st);
      HIPCHK(launch_gemm(gu, 2 * f, d, cf.dtype, Xn + (size_t)xrow0 * d * es, d, M, P + (size_t)xrow0 * 2 * f,
                         2 * f, stride, g_gu, st));
    }
    HIPCHK(launch_swiglu_finish(P, stride, S_gu, 2 * f, f, c.mode, c.rows, W.b, ret_h, ret_h_keep, cf.dtype, Xh, f,
                                st));
  }

  // 5. down projection + c coupling + residual + next norm
  WSegs wd{{W.w_down, nullptr, nullptr}, {d, 0, 0}};
  stride = (long long)c.rows_layout * d;
  {
    Timed tm(m, DBT_STAGE_DOWN, st);
    HIPCHK(project(wd, d, f, Xh + (size_t)xrow0 * f * es, f, M, P + (size_t)xrow0 * d, d, stride, g_d));
  }
  const float *g_next = nullptr;
  if (l + 1 < cf.n_layers) g_next = m->layers[l + 1].attn_norm;
  else if (cf.vocab > 0 && c.last_norm) g_next = m->w.final_norm;
  HIPCHK(launch_down_finish(P, stride, S_d, d, d, c.mode, c.rows, W.c, ret_m,
                            Retain{c.retain ? ret_m : nullptr, c.ret_src, c.ret_dst}, S, g_next, cf.rms_eps,
                            cf.dtype, Xn, d, st));
  return DBT_OK;
}

// Step inputs for the active rows: embeddings (Eq. (7)) or given residuals,
// then the first layer's attention norm.
dbt_status load_inputs(dbt_model *m, dbt_kv *kv, const dbt_step_in *in, const int *tokens, Rows rows,
                       hipStream_t st, const StepBegin *sb = nullptr) {
  const dbt_config &cf = m->cfg;
  const Layout &L = m->L;
  const float *g0 = m->layers[0].attn_norm;
  if (cf.has_embeddings) {
    HIPCHK(launch_embed(tokens, cf.vocab, m->w.emb1, m->w.emb2, m->w.emb_norm, g0, cf.rms_eps, cf.d_model, cf.dtype, rows,
                        m->at<float>(L.S), m->p(L.Xn), cf.d_model, st, sb, m->at<int>(L.pos), kv->page_table,
                        kv->mpps));
  } else {
    HIPCHK(launch_load_hidden(in->h1_in, in->h2_in, g0, cf.rms_eps, cf.d_model, cf.dtype, rows, m->at<float>(L.S),
                              m->p(L.Xn), cf.d_model, st, sb, m->at<int>(L.pos), kv->page_table, kv->mpps));
  }
  return DBT_OK;
}

// Final norm is already in Xn (applied by the last layer); output matrix for the active rows.
dbt_status lm_head(dbt_model *m, Rows rows, hipStream_t st) {
  const dbt_config &cf = m->cfg;
  const Layout &L = m->L;
  const int xrow0 = rows.p0 * rows.Bp;
  WSegs lm{{m->w.lm_head, nullptr, nullptr}, {cf.vocab, 0, 0}};
  Timed tm(m, DBT_STAGE_LMHEAD, st);
  const bool fused = gemm_stats_tiles(cf.vocab, L.g_lm, cf.dtype) > 0;
  HIPCHK(launch_gemm(lm, cf.vocab, cf.d_model, cf.dtype, m->p(L.Xn) + (size_t)xrow0 * cf.d_model * esize(cf),
                     cf.d_model, rows.np * rows.Bp, m->at<float>(L.logits) + (size_t)xrow0 * cf.vocab, cf.vocab,
                     0, L.g_lm, st, fused ? m->at<float>(L.mstats) + (size_t)xrow0 * L.nstat * 3 : nullptr));
  return DBT_OK;
}

dbt_status readout(dbt_model *m, int B, int Bp, bool branch, dbt_step_out *out, hipStream_t st) {
  const dbt_config &cf = m->cfg;
  const Layout &L = m->L;
  if (cf.vocab <= 0) return DBT_OK;
  MixArgs mx{};
  mx.logits = m->at<float>(L.logits);
  mx.V = cf.vocab;
  const int nb = n_branches(cf);
  mx.rows = Rows{B, Bp, 0, branch ? 1 + nb : 1};
  mx.chunk = kMixChunk;
  mx.stats = m->at<float>(L.mstats);
  mx.stats_ready = gemm_stats_tiles(cf.vocab, L.g_lm, cf.dtype) > 0;
  mx.tile_w = mx.stats_ready ? gemm_tile_rows(L.g_lm) : kMixChunk;
  mx.nstat = L.nstat;
  mx.alpha = out ? out->alpha : nullptr;
  mx.next = out ? out->next_token : nullptr;
  if (mx.alpha || mx.next) {
    Timed tm(m, DBT_STAGE_MIX, st);
    HIPCHK(launch_mixture(mx, st));
  }
  if (out && out->logits1)
    HIPCHK(hipMemcpyAsync(out->logits1, m->at<float>(L.logits), (size_t)B * cf.vocab * 4, hipMemcpyDeviceToDevice, st));
  if (out && out->logits2 && branch)
    for (int j = 0; j < nb; ++j)
      HIPCHK(hipMemcpyAsync(out->logits2 + (size_t)j * B * cf.vocab, m->at<float>(L.logits) + (size_t)(1 + j) * Bp * cf.vocab,
                            (size_t)B * cf.vocab * 4, hipMemcpyDeviceToDevice, st));
  return DBT_OK;
}

// Final residual states of the branches: [n_branches][B][d].
dbt_status copy_branch_rows(dbt_model *m, float *dst, int B, int Bp, hipStream_t st) {
  if (!dst) return DBT_OK;
  const int d = m->cfg.d_model;
  for (int j = 0; j < n_branches(m->cfg); ++j)
    HIPCHK(hipMemcpyAsync(dst + (size_t)j * B * d, m->at<float>(m->L.S) + (size_t)(1 + j) * Bp * d, (size_t)B * d * 4,
                          hipMemcpyDeviceToDevice, st));
  return DBT_OK;
}

dbt_status check_model_kv(dbt_model *m, dbt_kv *kv) {
  if (!m || !kv) return fail(DBT_ERR_ARG, "model or cache is NULL");
  if (kv->m != m) return fail(DBT_ERR_ARG, "cache belongs to another model");
  return DBT_OK;
}

dbt_status check_step_in(dbt_model *m, dbt_kv *kv, const dbt_step_in *in, int need_branch_input) {
  const dbt_config &cf = m->cfg;
  if (!in) return fail(DBT_ERR_ARG, "step input is NULL");
  if (in->batch <= 0 || in->batch > cf.max_batch) return fail(DBT_ERR_ARG, "batch %d out of [1, %d]", in->batch, cf.max_batch);
  if (cf.has_embeddings) {
    if (!in->tokens) return fail(DBT_ERR_ARG, "tokens are NULL");
  } else {
    if (!in->h1_in || (need_branch_input && !in->h2_in)) return fail(DBT_ERR_ARG, "residual inputs are NULL");
  }
  int need = 0;
  for (int b = 0; b < in->batch; ++b) {
    if (kv->len[b] + 1 > cf.max_pos) return fail(DBT_ERR_SHAPE, "sequence %d would exceed max_pos", b);
    if (kv->len[b] % kPage == 0) {
      if (kv->len[b] / kPage >= kv->mpps) return fail(DBT_ERR_NO_PAGES, "sequence %d page table full", b);
      ++need;
    }
  }
  if (need > (int)kv->free_pages.size()) return fail(DBT_ERR_NO_PAGES, "need %d free pages, have %zu", need, kv->free_pages.size());
  return DBT_OK;
}

// Take pages for the new position of each sequence (batch order) and return
// the positions pos_b = len_b.
std::vector<int> begin_step(dbt_kv *kv, int B) {
  std::vector<int> pos(B);
  for (int b = 0; b < B; ++b) {
    pos[b] = kv->len[b];
    if (kv->len[b] % kPage == 0) {
      const int p = kv->take_page();
      kv->table[b].push_back(p);
      kv->pending.push_back({b, (int)kv->table[b].size() - 1, p});
    }
  }
  return pos;
}

dbt_status copy_rows(float *dst, const float *src, int B, int d, hipStream_t st) {
  if (!dst) return DBT_OK;
  HIPCHK(hipMemcpyAsync(dst, src, (size_t)B * d * 4, hipMemcpyDeviceToDevice, st));
  return DBT_OK;
}

// Branch-only pass over all layers (ungrouped pass 2 and the boundary).
dbt_status branch_pass(dbt_model *m, dbt_kv *kv, int B, int Bp, hipStream_t st, const dbt_step_out *out = nullptr,
                       const HIn *hin = nullptr) {
  LayerCall lc{};
  lc.out = out;
  lc.hin = hin;
  const int nb = n_branches(m->cfg);
  lc.rows = Rows{B, Bp, 1, nb};
  lc.mode = MODE_BRANCH;
  lc.retain = false;
  lc.ret_src = -1;
  lc.ret_dst = 0;
  lc.prefill = false;
  lc.rows_layout = (1 + nb) * Bp;
  lc.last_norm = true;
  for (int l = 0; l < m->cfg.n_layers; ++l) {
    dbt_status s = run_layer(m, kv, l, lc, st);
    if (s) return s;
  }
  if (m->cfg.vocab > 0) return lm_head(m, lc.rows, st);
  return DBT_OK;
}

dbt_status decode_step_impl(dbt_model *m, dbt_kv *kv, const dbt_step_in *in, int32_t branch_on, dbt_step_out *out,
                            dbt_stream stream) {
  dbt_status s = check_model_kv(m, kv);
  if (s) return s;
  s = check_step_in(m, kv, in, branch_on);
  if (s) return s;
  hipStream_t st = (hipStream_t)stream;
  const dbt_config &cf = m->cfg;
  const int B = in->batch, Bp = round16(B);
  if ((s = ensure_device(m, st))) return s;  // before any state changes
  m->bnd_kv = nullptr;
  std::vector<int> pos = begin_step(kv, B);
  StepBegin sb;
  if ((s = flush(kv, pos.data(), B, st, &sb))) return s;
  const bool on = branch_on != 0;
  const int nb = n_branches(cf);
  const Rows rows{B, Bp, 0, on ? 1 + nb : 1};
  const bool fold = input_fold(m, kv, B);
  const HIn hin{in->h1_in, in->h2_in, B};
  if (!fold && (s = load_inputs(m, kv, in, in->tokens, rows, st, &sb))) return s;
  LayerCall lc{};
  if (fold) {
    lc.hin = &hin;
    lc.sb = &sb;
  }
  lc.rows = rows;
  lc.mode = on ? MODE_GROUPED : MODE_PRIMARY;
  lc.retain = false;
  lc.ret_src = -1;
  lc.prefill = false;
  lc.rows_layout = (1 + nb) * Bp;
  lc.last_norm = true;
  lc.out = out;
  for (int l = 0; l < cf.n_layers; ++l)
    if ((s = run_layer(m, kv, l, lc, st))) return s;
  if (cf.vocab > 0 && (s = lm_head(m, rows, st))) return s;
  for (int b = 0; b < B; ++b) kv->len[b] += 1;
  if (out) {
    if ((s = readout(m, B, Bp, on, out, st))) return s;
    if ((s = copy_rows(out->h1_out, m->at<float>(m->L.S), B, cf.d_model, st))) return s;
    if (on && (s = copy_branch_rows(m, out->h2_out, B, Bp, st))) return s;
  }
  return DBT_OK;
}

}  // namespace

// ===========================================================================

extern "C" {

const char *dbt_last_error(void) { return g_err.c_str(); }

size_t dbt_workspace_bytes(const dbt_config *cfg) {
  if (check_config(cfg) != DBT_OK) return 0;
  return make_layout(cfg).total;
}

size_t dbt_kv_pages_bytes(const dbt_config *cfg, int32_t num_pages) {
  if (check_config(cfg) != DBT_OK || num_pages <= 0) return 0;
  return (size_t)cfg->n_layers * num_pages * cfg->n_kv_heads * kPage * cfg->head_dim * (cfg->dtype == DBT_BF16 ? 2 : 4);
}

dbt_status dbt_create(const dbt_config *cfg, const dbt_weights *w, void *workspace, dbt_model **out) {
  if (!out) return fail(DBT_ERR_ARG, "out is NULL");
  *out = nullptr;
  if (dbt_status cs = check_config(cfg)) return cs;
  if (!w || !w->h_layers) return fail(DBT_ERR_ARG, "weights are NULL");
  if (!workspace || ((uintptr_t)workspace & 255)) return fail(DBT_ERR_ARG, "workspace NULL or not 256-byte aligned");
  if (cfg->has_embeddings && (!w->emb1 || !w->emb2 || !w->emb_norm)) return fail(DBT_ERR_ARG, "embeddings are NULL");
  if (cfg->vocab > 0 && (!w->lm_head || !w->final_norm)) return fail(DBT_ERR_ARG, "output matrix or final norm is NULL");
  for (int l = 0; l < cfg->n_layers; ++l) {
    const dbt_layer_weights &L = w->h_layers[l];
    if (!L.attn_norm || !L.wq || !L.wk || !L.wv || !L.wo || !L.mlp_norm || !L.a || !L.c)
      return fail(DBT_ERR_ARG, "layer %d has a NULL parameter", l);
    if (cfg->n_experts == 0 && (!L.w_gate || !L.w_up || !L.w_down || !L.b))
      return fail(DBT_ERR_ARG, "layer %d has a NULL MLP parameter", l);
    if (cfg->n_experts > 0 && (!L.router || !L.x_gate || !L.x_up || !L.x_down))
      return fail(DBT_ERR_ARG, "layer %d has a NULL expert parameter", l);
    if (cfg->n_experts > 0 && cfg->d_ff_shared > 0 && (!L.s_gate || !L.s_up || !L.s_down || !L.b))
      return fail(DBT_ERR_ARG, "layer %d has a NULL shared-expert parameter", l);
    if (cfg->compute_matched && (!L.g_attn_copy || !L.g_shared_copy))
      return fail(DBT_ERR_ARG, "layer %d has a NULL gate of the compute-matched variant", l);
  }
  dbt_model *m = new (std::nothrow) dbt_model();
  if (!m) return fail(DBT_ERR_ARG, "out of host memory");
  m->cfg = *cfg;
  m->w = *w;
  m->layers.assign(w->h_layers, w->h_layers + cfg->n_layers);
  m->w.h_layers = nullptr;
  m->ws = (char *)workspace;
  m->L = make_layout(cfg);
  m->step = m->ws + m->L.state_total;
  // RoPE table (Eq. (8)): angle pos * theta^(-2i/d_h), evaluated in double.
  const int half = cfg->head_dim / 2;
  m->rope_host.resize((size_t)cfg->max_pos * half * 2);
  for (int p = 0; p < cfg->max_pos; ++p)
    for (int i = 0; i < half; ++i) {
      const double ang = (double)p * std::pow((double)cfg->rope_theta, -2.0 * i / cfg->head_dim);
      m->rope_host[((size_t)p * half + i) * 2 + 0] = (float)std::cos(ang);
      m->rope_host[((size_t)p * half + i) * 2 + 1] = (float)std::sin(ang);
    }
  *out = m;
  return DBT_OK;
}

dbt_status dbt_destroy(dbt_model *m) {
  delete m;
  return DBT_OK;
}

dbt_status dbt_kv_create(dbt_model *m, void *k_pages, void *v_pages, int32_t num_pages, int32_t *page_table,
                         int32_t max_pages_per_seq, dbt_kv **out) {
  if (!out) return fail(DBT_ERR_ARG, "out is NULL");
  *out = nullptr;
  if (!m || !k_pages || !v_pages || !page_table) return fail(DBT_ERR_ARG, "NULL argument");
  if (num_pages <= 0 || max_pages_per_seq <= 0) return fail(DBT_ERR_ARG, "num_pages and max_pages_per_seq must be positive");
  if ((long long)max_pages_per_seq * kPage < m->cfg.max_pos) return fail(DBT_ERR_SHAPE, "max_pages_per_seq * 16 < max_pos");
  dbt_kv *kv = new (std::nothrow) dbt_kv();
  if (!kv) return fail(DBT_ERR_ARG, "out of host memory");
  kv->m = m;
  kv->k = (char *)k_pages;
  kv->v = (char *)v_pages;
  kv->num_pages = num_pages;
  kv->page_table = page_table;
  kv->mpps = max_pages_per_seq;
  std::vector<int> all(num_pages);
  for (int i = 0; i < num_pages; ++i) all[i] = i;
  kv->free_pages = std::priority_queue<int, std::vector<int>, std::greater<int>>(std::greater<int>(), std::move(all));
  kv->table.assign(m->cfg.max_batch, {});
  kv->len.assign(m->cfg.max_batch, 0);
  *out = kv;
  return DBT_OK;
}

dbt_status dbt_kv_destroy(dbt_kv *kv) {
  delete kv;
  return DBT_OK;
}

dbt_status dbt_kv_reserve(dbt_kv *kv, int32_t b, int32_t len, int32_t *h_pages_out) {
  if (!kv) return fail(DBT_ERR_ARG, "cache is NULL");
  if (b < 0 || b >= kv->m->cfg.max_batch) return fail(DBT_ERR_ARG, "sequence %d out of range", b);
  if (len < kv->len[b]) return fail(DBT_ERR_ARG, "len %d below current length %d", len, kv->len[b]);
  if (len > kv->m->cfg.max_pos) return fail(DBT_ERR_SHAPE, "len %d exceeds max_pos", len);
  const int need_pages = (len + kPage - 1) / kPage;
  if (need_pages > kv->mpps) return fail(DBT_ERR_NO_PAGES, "page table row too short");
  const int extra = need_pages - (int)kv->table[b].size();
  if (extra > (int)kv->free_pages.size()) return fail(DBT_ERR_NO_PAGES, "need %d free pages, have %zu", extra, kv->free_pages.size());
  for (int i = 0; i < extra; ++i) {
    const int p = kv->take_page();
    kv->table[b].push_back(p);
    kv->pending.push_back({b, (int)kv->table[b].size() - 1, p});
  }
  kv->len[b] = len;
  if (h_pages_out)
    for (size_t i = 0; i < kv->table[b].size(); ++i) h_pages_out[i] = kv->table[b][i];
  if (kv->m->bnd_kv == kv) kv->m->bnd_kv = nullptr;
  return DBT_OK;
}

dbt_status dbt_kv_truncate(dbt_kv *kv, int32_t b, int32_t len) {
  if (!kv) return fail(DBT_ERR_ARG, "cache is NULL");
  if (b < 0 || b >= kv->m->cfg.max_batch) return fail(DBT_ERR_ARG, "sequence %d out of range", b);
  if (len < 0 || len > kv->len[b]) return fail(DBT_ERR_ARG, "len %d outside [0, %d]", len, kv->len[b]);
  const size_t keep = (len + kPage - 1) / kPage;
  for (size_t i = keep; i < kv->table[b].size(); ++i) kv->free_pages.push(kv->table[b][i]);
  kv->table[b].resize(keep);
  kv->len[b] = len;
  // entries of pages given back may still sit in the pending list; they are
  // harmless (a later take re-sends the slot) but drop those of this sequence
  kv->pending.erase(std::remove_if(kv->pending.begin(), kv->pending.end(),
                                   [&](const dbt_kv::Upd &u) { return u.b == b && (size_t)u.slot >= keep; }),
                    kv->pending.end());
  if (kv->m->bnd_kv == kv) kv->m->bnd_kv = nullptr;
  return DBT_OK;
}

int32_t dbt_kv_length(const dbt_kv *kv, int32_t b) {
  if (!kv || b < 0 || b >= kv->m->cfg.max_batch) return -1;
  return kv->len[b];
}

int32_t dbt_kv_pages(const dbt_kv *kv, int32_t b, int32_t *h_out, int32_t cap) {
  if (!kv || b < 0 || b >= kv->m->cfg.max_batch) return -1;
  const int n = (int)kv->table[b].size();
  for (int i = 0; i < n && i < cap && h_out; ++i) h_out[i] = kv->table[b][i];
  return n;
}

dbt_status dbt_kv_fill(dbt_kv *kv, int32_t layer, int32_t b, int32_t start, int32_t count, const void *k_src,
                       const void *v_src, dbt_stream stream) {
  if (!kv || !k_src || !v_src) return fail(DBT_ERR_ARG, "NULL argument");
  const dbt_config &cf = kv->m->cfg;
  if (layer < 0 || layer >= cf.n_layers) return fail(DBT_ERR_ARG, "layer %d out of range", layer);
  if (b < 0 || b >= cf.max_batch) return fail(DBT_ERR_ARG, "sequence %d out of range", b);
  if (start < 0 || count < 0 || start + count > kv->len[b]) return fail(DBT_ERR_ARG, "positions outside the reserved length");
  hipStream_t st = (hipStream_t)stream;
  dbt_status s = ensure_device(kv->m, st);
  if (s) return s;
  s = flush(kv, nullptr, 0, st);
  if (s) return s;
  HIPCHK(launch_kv_fill(kv_layer(kv, layer), b, start, count, k_src, v_src, cf.dtype, st));
  return DBT_OK;
}

dbt_status dbt_decode_step(dbt_model *m, dbt_kv *kv, const dbt_step_in *in, int32_t branch_on, dbt_step_out *out,
                           dbt_stream stream) {
  return decode_step_impl(m, kv, in, branch_on, out, stream);
}

dbt_status dbt_decode_step_ungrouped(dbt_model *m, dbt_kv *kv, const dbt_step_in *in, dbt_step_out *out,
                                     dbt_stream stream) {
  dbt_status s = check_model_kv(m, kv);
  if (s) return s;
  s = check_step_in(m, kv, in, 1);
  if (s) return s;
  hipStream_t st = (hipStream_t)stream;
  const dbt_config &cf = m->cfg;
  const int B = in->batch, Bp = round16(B);
  if ((s = ensure_device(m, st))) return s;  // before any state changes
  m->bnd_kv = nullptr;
  std::vector<int> pos = begin_step(kv, B);
  StepBegin sb;
  if ((s = flush(kv, pos.data(), B, st, &sb))) return s;
  // pass 1: every primary layer, keeping Q1, H1, M1
  const Rows prim{B, Bp, 0, 1};
  const bool fold = input_fold(m, kv, B);
  const HIn hin{in->h1_in, in->h2_in, B};
  if (!fold && (s = load_inputs(m, kv, in, in->tokens, prim, st, &sb))) return s;
  LayerCall lc{};
  if (fold) {
    lc.hin = &hin;
    lc.sb = &sb;
  }
  lc.rows = prim;
  lc.mode = MODE_PRIMARY;
  lc.retain = true;
  lc.ret_src = -1;
  lc.prefill = false;
  lc.rows_layout = (1 + n_branches(cf)) * Bp;
  lc.last_norm = true;
  lc.out = out;
  for (int l = 0; l < cf.n_layers; ++l)
    if ((s = run_layer(m, kv, l, lc, st))) return s;
  if (cf.vocab > 0 && (s = lm_head(m, prim, st))) return s;
  // pass 2: every branch layer
  const Rows br{B, Bp, 1, n_branches(cf)};
  if (!fold && (s = load_inputs(m, kv, in, in->tokens, br, st))) return s;
  if ((s = branch_pass(m, kv, B, Bp, st, out, fold ? &hin : nullptr))) return s;
  for (int b = 0; b < B; ++b) kv->len[b] += 1;
  if (out) {
    if ((s = readout(m, B, Bp, true, out, st))) return s;
    if ((s = copy_rows(out->h1_out, m->at<float>(m->L.S), B, cf.d_model, st))) return s;
    if ((s = copy_branch_rows(m, out->h2_out, B, Bp, st))) return s;
  }
  return DBT_OK;
}

dbt_status dbt_prefill(dbt_model *m, dbt_kv *kv, const int32_t *tokens, const int32_t *h_prompt_lens, int32_t batch,
                       int32_t run_boundary, dbt_step_out *out, dbt_stream stream) {
  dbt_status s = check_model_kv(m, kv);
  if (s) return s;
  const dbt_config &cf = m->cfg;
  if (!tokens || !h_prompt_lens) return fail(DBT_ERR_ARG, "tokens or prompt lengths NULL");
  if (cf.max_prompt <= 0) return fail(DBT_ERR_STATE, "model created without prefill support (max_prompt = 0)");
  if (batch <= 0 || batch > cf.max_batch) return fail(DBT_ERR_ARG, "batch %d out of [1, %d]", batch, cf.max_batch);
  int need = 0;
  for (int b = 0; b < batch; ++b) {
    const int T = h_prompt_lens[b];
    if (T <= 0 || T > cf.max_prompt) return fail(DBT_ERR_SHAPE, "prompt %d length %d outside [1, %d]", b, T, cf.max_prompt);
    if (kv->len[b] != 0) return fail(DBT_ERR_STATE, "sequence %d is not empty", b);
    need += (T + kPage - 1) / kPage;
  }
  if (need > (int)kv->free_pages.size()) return fail(DBT_ERR_NO_PAGES, "need %d free pages, have %zu", need, kv->free_pages.size());
  hipStream_t st = (hipStream_t)stream;
  if ((s = ensure_device(m, st))) return s;  // before any state changes
  for (int b = 0; b < batch; ++b) {  // pages for every sequence first, in batch order
    const int np = (h_prompt_lens[b] + kPage - 1) / kPage;
    for (int i = 0; i < np; ++i) {
      const int p = kv->take_page();
      kv->table[b].push_back(p);
      kv->pending.push_back({b, i, p});
    }
    kv->len[b] = h_prompt_lens[b];
  }
  if ((s = flush(kv, nullptr, 0, st))) return s;
  const Layout &L = m->L;
  const int d = cf.d_model;
  const int Bp = round16(batch);
  size_t off = 0;
  for (int b = 0; b < batch; ++b) {
    const int T = h_prompt_lens[b];
    const Rows rows{T, T, 0, 1};
    HIPCHK(launch_embed(tokens + off, cf.vocab, m->w.emb1, m->w.emb2, m->w.emb_norm, m->layers[0].attn_norm, cf.rms_eps, d,
                        cf.dtype, rows, m->at<float>(L.S), m->p(L.Xn), d, st));
    LayerCall lc{};
    lc.rows = rows;
    lc.mode = MODE_PRIMARY;
    lc.retain = true;
    lc.ret_src = T - 1;
    lc.ret_dst = b;
    lc.prefill = true;
    lc.seq = b;
    lc.rows_layout = T;
    lc.last_norm = false;
    for (int l = 0; l < cf.n_layers; ++l)
      if ((s = run_layer(m, kv, l, lc, st))) return s;
    HIPCHK(hipMemcpyAsync(m->at<float>(L.slast) + (size_t)b * d, m->at<float>(L.S) + (size_t)(T - 1) * d, d * 4,
                          hipMemcpyDeviceToDevice, st));
    HIPCHK(hipMemcpyAsync(m->at<int>(L.btok) + b, tokens + off + T - 1, 4, hipMemcpyDeviceToDevice, st));
    off += T;
  }
  // primary logits at each prompt's final position
  if (cf.vocab > 0) {
    HIPCHK(launch_rmsnorm_rows(m->at<float>(L.slast), m->w.final_norm, cf.rms_eps, d, cf.dtype, Rows{batch, 0, 0, 1},
                               m->p(L.Xn), d, st));
    if ((s = lm_head(m, Rows{batch, Bp, 0, 1}, st))) return s;
  }
  if (out) {
    if ((s = copy_rows(out->h1_out, m->at<float>(L.slast), batch, d, st))) return s;
  }
  m->bnd_kv = kv;
  m->bnd_batch = batch;
  if (run_boundary) return dbt_boundary(m, kv, batch, out, stream);
  if (out && (s = readout(m, batch, Bp, false, out, st))) return s;
  return DBT_OK;
}

dbt_status dbt_boundary(dbt_model *m, dbt_kv *kv, int32_t batch, dbt_step_out *out, dbt_stream stream) {
  dbt_status s = check_model_kv(m, kv);
  if (s) return s;
  if (m->bnd_kv != kv || batch != m->bnd_batch)
    return fail(DBT_ERR_STATE, "boundary must directly follow dbt_prefill on the same cache and batch");
  hipStream_t st = (hipStream_t)stream;
  const dbt_config &cf = m->cfg;
  const Layout &L = m->L;
  const int B = batch, Bp = round16(B);
  if ((s = ensure_device(m, st))) return s;
  std::vector<int> pos(B);
  for (int b = 0; b < B; ++b) pos[b] = kv->len[b] - 1;
  if ((s = flush(kv, pos.data(), B, st))) return s;
  const Rows br{B, Bp, 1, n_branches(cf)};
  HIPCHK(launch_embed(m->at<int>(L.btok), cf.vocab, m->w.emb1, m->w.emb2, m->w.emb_norm, m->layers[0].attn_norm, cf.rms_eps,
                      cf.d_model, cf.dtype, br, m->at<float>(L.S), m->p(L.Xn), cf.d_model, st));
  if ((s = branch_pass(m, kv, B, Bp, st))) return s;
  m->bnd_kv = nullptr;
  if (out) {
    if ((s = readout(m, B, Bp, true, out, st))) return s;
    if ((s = copy_branch_rows(m, out->h2_out, B, Bp, st))) return s;
  }
  return DBT_OK;
}

dbt_status dbt_stage_timing(dbt_model *m, int32_t stage, int32_t enable) {
  if (!m) return fail(DBT_ERR_ARG, "model is NULL");
  if (stage < 0 || stage >= DBT_STAGE_COUNT) return fail(DBT_ERR_ARG, "stage %d out of range", stage);
  m->timers[stage].on = enable != 0;
  m->timers[stage].used = 0;
  return DBT_OK;
}

double dbt_stage_time(dbt_model *m, int32_t stage, int32_t *h_launches) {
  if (!m || stage < 0 || stage >= DBT_STAGE_COUNT) return -1.0;
  StageTimer &t = m->timers[stage];
  double total = 0.0;
  for (size_t i = 0; i < t.used; ++i) {
    float ms = 0.f;
    if (hipEventSynchronize(t.ev[i].second) != hipSuccess) return -1.0;
    if (hipEventElapsedTime(&ms, t.ev[i].first, t.ev[i].second) != hipSuccess) return -1.0;
    total += ms;
  }
  if (h_launches) *h_launches = (int32_t)t.used;
  t.used = 0;
  return total;
}

}  // extern "C"

// ---------------------------------------------------------------------------
// Hooks for the allocation-free step (static_scratch.hip)
// ---------------------------------------------------------------------------
namespace dbt {

dbt_status set_error(dbt_status s, const char *msg) { return fail(s, "%s", msg); }

size_t step_bytes(const dbt_model *m) { return m->L.total - m->L.state_total; }

dbt_status decode_step_in(dbt_model *m, dbt_kv *kv, const dbt_step_in *in, int32_t branch_on, dbt_step_out *out,
                          dbt_stream stream, char *step_mem) {
  // the model's own step region again when the call returns, whatever it returns
  struct Restore {
    dbt_model *m;
    ~Restore() {
      m->step = m->ws + m->L.state_total;
      m->no_fork = false;
    }
  } restore{m};
  m->step = step_mem;
  m->no_fork = true;  // no stream of its own is created here: the shared expert stays on `stream`
  return decode_step_impl(m, kv, in, branch_on, out, stream);
}

}  // namespace dbt
