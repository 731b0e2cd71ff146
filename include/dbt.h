/*
 * dbt.h -- C ABI of the Decode-Branch Transformer decode library (gfx950).
 *
 * The method (arXiv 2608.12385, "Decode-Branch Transformers"):
 *   - a primary path that is a complete causal LM; it alone processes the
 *     prompt and writes the single persistent KV cache (Sec. 4, Sec. 4.4);
 *   - a decode branch with its own token embedding (Eq. (7)) that forms only
 *     a query, Q2~ = Q2 + a * Q1, attends to the primary keys/values
 *     (Eqs. (10)-(12)) and is coupled to the primary MLP through
 *     H2~ = H2 + b * H1 and M2 = H2~ W_D + c * M1 (Eqs. (13)-(16));
 *   - a mixture readout alpha p + (1 - alpha) q with
 *     alpha = clip(sum p^2, 0.5, 1) (Sec. 4.2, Eqs. (17)-(18));
 *   - the grouped continuation step: both paths' rows are stacked so that
 *     each shared weight tile and each primary KV page is read once for both
 *     (Sec. 4.4 "Decode", Sec. 4.5, Eq. (20));
 *   - MoE layers with independent primary/branch fan-outs k1, k2 (Sec. 5,
 *     Eq. (22)) or router replay (Sec. 4.3, Eq. (19)).
 *
 * Conventions
 *   - Every pointer argument is DEVICE memory unless its name starts with h_
 *     (host memory).  Device pointers must be 16-byte aligned.  The caller owns all device memory: weights, KV pages,
 *     page table, workspace, inputs and outputs.  The library keeps borrowed
 *     pointers, which must stay valid until the handle is destroyed.  The
 *     library itself never allocates device memory.
 *   - Calls that take a stream enqueue their work on it and return without
 *     synchronising; the caller synchronises.  Host-side bookkeeping (cache
 *     lengths, page allocation) is updated when the call returns.
 *   - Every argument, shape and state check happens before anything is
 *     enqueued.  A failing call returns a non-zero dbt_status, changes no
 *     state, and leaves a message for dbt_last_error().  HIP launch errors
 *     return DBT_ERR_HIP.  No C++ exception crosses this interface.
 *   - Calls that take no stream are host-only and need no GPU.
 *   - One model/cache pair must not be used from two threads at once.
 *
 * Storage (dtype = DBT_F32 or DBT_BF16 applies to every matrix, embedding
 * and the KV cache; vectors a, b, c and norm gains are always float32;
 * activations and accumulation are float32):
 *   - matrices are out-major: W[out][in], the input dimension contiguous;
 *   - KV pages hold 16 positions.  For layer l and page p:
 *       K: k_pages + ((l * num_pages + p) * n_kv + g) * 16 * d_h,
 *          laid out [slot 0..15][d_h]   (position-major);
 *       V: v_pages + same offset, laid out [d_h][slot 0..15] (dim-major);
 *   - page_table is int32 [max_batch][max_pages_per_seq]: entry j of
 *     sequence b is the page holding positions 16j..16j+15.
 */
#ifndef DBT_H
#define DBT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct dbt_model dbt_model;
typedef struct dbt_kv dbt_kv;
typedef void *dbt_stream; /* a hipStream_t; NULL is the default stream */

typedef enum {
  DBT_OK = 0,
  DBT_ERR_ARG = 1,         /* null pointer or out-of-range scalar */
  DBT_ERR_SHAPE = 2,       /* sizes inconsistent with the model */
  DBT_ERR_NO_PAGES = 3,    /* the page pool cannot hold the request */
  DBT_ERR_STATE = 4,       /* call out of order (e.g. boundary without prefill) */
  DBT_ERR_UNSUPPORTED = 5, /* valid configuration the library does not run */
  DBT_ERR_HIP = 6          /* HIP runtime or launch error */
} dbt_status;

enum { DBT_F32 = 0, DBT_BF16 = 1 };

/* Model shape.  n_experts = 0 selects dense SwiGLU MLPs (d_ff); otherwise
 * every layer is an MoE layer with n_experts routed SwiGLU experts of width
 * d_ff_expert, an optional shared expert of width d_ff_shared (0 = none),
 * primary fan-out top_k1 and branch fan-out top_k2 (Sec. 5, Eq. (22)).
 * replay = 1: the branch reuses the primary's selected experts with its own
 * renormalised router probabilities (Sec. 4.3, Eq. (19)); needs
 * top_k2 = top_k1.  compute_matched = 1 (MoE only): the compute-matched
 * variant of App. B.3, where the branch evaluates no attention and no shared
 * expert: its attention update is g_A * A1 and its MoE output is its own
 * routed experts plus g_G * G(N1) (the layer weights g_attn_copy,
 * g_shared_copy; a and b are unused, and c too).  vocab = 0: no output
 * matrix (layer-only models return residual states).  has_embeddings = 0:
 * steps take residual-state inputs instead of tokens.  n_branches > 1
 * (App. C.1): branch j has its own embedding table and shares the couplings
 * a, b, c and every weight; each branch reads only the primary (its Q1, H1,
 * M1 and cache); the mixture's q is the mean of the branch softmaxes.  The
 * branch tables, inputs and outputs below are then stacked [n_branches][...]
 * in branch order.  Needs (1 + n_branches) * n_q_heads / n_kv_heads <= 16. */
typedef struct {
  int32_t n_layers, d_model, n_q_heads, n_kv_heads, head_dim, d_ff, vocab;
  int32_t n_experts, d_ff_expert, d_ff_shared, top_k1, top_k2, replay;
  int32_t compute_matched; /* 0 or 1 (App. B.3) */
  int32_t n_branches;      /* decode branches, 0..3 (0 reads as 1; > 1: App. C.1, dense only) */
  int32_t dtype;          /* DBT_F32 or DBT_BF16 */
  int32_t has_embeddings; /* 1: token inputs through E1/E2 */
  int32_t max_batch;      /* sequences per call */
  int32_t max_pos;        /* positions per sequence (sizes the RoPE table) */
  int32_t max_prompt;     /* longest prompt dbt_prefill accepts (0: no prefill) */
  float rms_eps;          /* RMSNorm epsilon */
  float rope_theta;       /* RoPE base */
} dbt_config;

/* Per-layer parameters (device pointers; unused ones NULL). */
typedef struct {
  const float *attn_norm;          /* [d] */
  const void *wq;                  /* [n_q*d_h][d] */
  const void *wk;                  /* [n_kv*d_h][d] */
  const void *wv;                  /* [n_kv*d_h][d] */
  const void *wo;                  /* [d][n_q*d_h] */
  const float *mlp_norm;           /* [d] */
  const void *w_gate, *w_up;       /* dense: [d_ff][d] */
  const void *w_down;              /* dense: [d][d_ff] */
  const float *a;                  /* [n_q*d_h] query coupling, Eq. (11) */
  const float *b;                  /* [d_ff] (MoE: [d_ff_shared]) MLP coupling, Eq. (14) */
  const float *c;                  /* [d] output coupling, Eq. (15) */
  const void *router;              /* MoE: [n_experts][d] */
  const void *x_gate, *x_up;       /* MoE: [n_experts][d_ff_expert][d] */
  const void *x_down;              /* MoE: [n_experts][d][d_ff_expert] */
  const void *s_gate, *s_up;       /* MoE shared expert: [d_ff_shared][d] */
  const void *s_down;              /* MoE shared expert: [d][d_ff_shared] */
  const float *g_attn_copy;        /* compute-matched: [d] gate g_A of the attention copy */
  const float *g_shared_copy;      /* compute-matched: [d] gate g_G of the shared-expert copy */
} dbt_layer_weights;

typedef struct {
  const void *emb1;          /* [vocab][d]: primary embedding, Eq. (7) */
  const void *emb2;          /* [n_branches][vocab][d]: branch embeddings, Eq. (7) */
  const float *emb_norm;     /* [d] gain of the embedding RMSNorm */
  const float *final_norm;   /* [d] */
  const void *lm_head;       /* [vocab][d]: shared output matrix (Sec. 4.2) */
  const dbt_layer_weights *h_layers; /* HOST array [n_layers] */
} dbt_weights;

/* Inputs of one step for sequences 0..batch-1. */
typedef struct {
  const int32_t *tokens; /* [batch] (models with embeddings), else NULL */
  const float *h1_in;    /* [batch][d] primary residual input (layer-only models) */
  const float *h2_in;    /* [n_branches][batch][d] branch residual inputs (layer-only models) */
  int32_t batch;
} dbt_step_in;

/* Outputs of a step; any pointer may be NULL.  Routing arrays (MoE layers,
 * continuation steps) are [n_layers][batch][top_k] in the order selected
 * (logit descending): the selected experts I_i and their renormalised
 * weights (Sec. 3.2, Eqs. (5)-(6); Eq. (19) with replay).  route_logits1/2
 * are the float32 router logits r_i = U_i W_r^T the selection was made from,
 * [n_layers][batch][n_experts] (Sec. 3.2, Eq. (5)), so a caller can check
 * the selection against its own top-k of the same values. */
typedef struct {
  float *logits1;           /* [batch][vocab] */
  float *logits2;           /* [n_branches][batch][vocab] */
  float *alpha;             /* [batch] mixture weight (1 with the branch off) */
  int32_t *next_token;      /* [batch] greedy token of the mixture */
  float *h1_out;            /* [batch][d] final primary residual state */
  float *h2_out;            /* [n_branches][batch][d] final branch residual states */
  int32_t *route_idx1, *route_idx2;
  float *route_w1, *route_w2;
  float *route_logits1, *route_logits2;
} dbt_step_out;

/* ---- host-only calls (no GPU needed) ---------------------------------- */

/* Size in bytes of the device workspace dbt_create needs (0 on a bad config). */
size_t dbt_workspace_bytes(const dbt_config *cfg);

/* Bytes of one of the two page arrays (K or V) for num_pages pages. */
size_t dbt_kv_pages_bytes(const dbt_config *cfg, int32_t num_pages);

/* Validates cfg and the weight pointers and builds the model handle.  The
 * workspace (dbt_workspace_bytes(cfg) bytes, 256-byte aligned) holds every
 * intermediate and is owned by the caller.  Nothing is enqueued here: the
 * first call that takes a stream initialises the workspace. */
dbt_status dbt_create(const dbt_config *cfg, const dbt_weights *w, void *workspace,
                      dbt_model **out);
dbt_status dbt_destroy(dbt_model *m);

/* A paged primary KV cache (Sec. 4.4: the only persistent state; the branch
 * never writes it).  k_pages/v_pages: dbt_kv_pages_bytes() bytes each;
 * page_table: int32 [max_batch][max_pages_per_seq]. */
dbt_status dbt_kv_create(dbt_model *m, void *k_pages, void *v_pages, int32_t num_pages,
                         int32_t *page_table, int32_t max_pages_per_seq, dbt_kv **out);
dbt_status dbt_kv_destroy(dbt_kv *kv);

/* Grows sequence b to len positions (pages taken lowest free id first) so the
 * caller can fill them with dbt_kv_fill; h_pages_out (may be NULL) receives
 * the sequence's page ids, ceil(len/16) of them.  len below the current
 * length is DBT_ERR_ARG (use dbt_kv_truncate). */
dbt_status dbt_kv_reserve(dbt_kv *kv, int32_t b, int32_t len, int32_t *h_pages_out);

/* Shrinks sequence b to len positions and frees the pages past them. */
dbt_status dbt_kv_truncate(dbt_kv *kv, int32_t b, int32_t len);

/* Current length of sequence b (negative on error). */
int32_t dbt_kv_length(const dbt_kv *kv, int32_t b);

/* Copies up to cap page ids of sequence b into h_out; returns the count. */
int32_t dbt_kv_pages(const dbt_kv *kv, int32_t b, int32_t *h_out, int32_t cap);

/* Thread-local message of the last failing call. */
const char *dbt_last_error(void);

/* ---- device calls ------------------------------------------------------ */

/* Writes positions [start, start+count) of sequence b, layer `layer`, from
 * contiguous k_src/v_src [count][n_kv][d_h] (model dtype).  The positions
 * must already be reserved. */
dbt_status dbt_kv_fill(dbt_kv *kv, int32_t layer, int32_t b, int32_t start, int32_t count,
                       const void *k_src, const void *v_src, dbt_stream stream);

/* Prompt-wide prefill (Sec. 4.4, step 1): the primary path alone over every
 * prompt position; the keys/values of all positions are written to the
 * cache; the final position's Q1, H1, M1 (per layer) and primary logits are
 * kept for the boundary.  tokens: concatenated prompts [sum h_prompt_lens];
 * sequences 0..batch-1 must be empty.  run_boundary = 1 then evaluates the
 * branch once at the final prompt position (step 2; see dbt_boundary), and
 * out receives the mixture prediction of the first continuation token;
 * run_boundary = 0 fills out with the primary-only prediction. */
dbt_status dbt_prefill(dbt_model *m, dbt_kv *kv, const int32_t *tokens,
                       const int32_t *h_prompt_lens, int32_t batch, int32_t run_boundary,
                       dbt_step_out *out, dbt_stream stream);

/* The continuation boundary (Sec. 4.4, step 2): the branch alone at the final
 * prompt position, from E2 of the last prompt token and the retained primary
 * intermediates, attending to the finished prompt cache.  Writes no cache.
 * Valid only directly after dbt_prefill(run_boundary = 0) on the same cache. */
dbt_status dbt_boundary(dbt_model *m, dbt_kv *kv, int32_t batch, dbt_step_out *out,
                        dbt_stream stream);

/* One grouped continuation step (Sec. 4.4, step 3; Sec. 4.5): for every
 * sequence the primary and branch rows pass through each layer together, one
 * read of each weight tile and of each primary KV page serving both; the
 * primary appends its key/value at position len_b; the branch writes nothing
 * persistent.  branch_on = 0 runs the one-flow model (primary only, alpha = 1,
 * greedy token of p).  Sequence lengths grow by one. */
dbt_status dbt_decode_step(dbt_model *m, dbt_kv *kv, const dbt_step_in *in, int32_t branch_on,
                           dbt_step_out *out, dbt_stream stream);

/* The same step computed in two passes: every primary layer first (keeping
 * Q1, H1, M1 per layer), then every branch layer, so weights and cache pages
 * are read twice.  This is the unshared execution against which Sec. 4.4
 * ("Decode") and Sec. 4.5 (Eq. (20): decode traffic is weights plus KV
 * state, read once by the grouped step) measure grouping; it computes the
 * same definition.  Results are bit-identical to
 * dbt_decode_step(branch_on=1). */
dbt_status dbt_decode_step_ungrouped(dbt_model *m, dbt_kv *kv, const dbt_step_in *in,
                                     dbt_step_out *out, dbt_stream stream);

/* For callers that cannot allocate device memory while they step (code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation):
 * dbt_decode_step with the step's buffers (activations, split partials,
 * logits and their statistics, MoE lists) in a static device array of the
 * library instead of the model workspace's step region.  It allocates
 * nothing and calls no allocating routine; results equal
 * dbt_decode_step's bit for bit.  The array holds DBT_STATIC_SCRATCH_BYTES
 * on every GPU the library runs on, from load until the process ends; a
 * model whose step buffers need more (large vocabularies with many
 * sequences, or models sized for long prompts) gets DBT_ERR_UNSUPPORTED
 * before anything changes.  Every call on one GPU shares that GPU's array:
 * calls that overlap on one GPU (other streams, threads or models) race.
 * The model still needs its workspace for the state kept between calls. */
#define DBT_STATIC_SCRATCH_BYTES ((size_t)64 << 20)
dbt_status dbt_decode_step_noalloc(dbt_model *m, dbt_kv *kv, const dbt_step_in *in, int32_t branch_on,
                                   dbt_step_out *out, dbt_stream stream);

/* ---- stage timing -------------------------------------------------------
 * While enabled for a stage, every later device call records a HIP event pair
 * on its stream around the kernel(s) of that stage, once per launch.
 * dbt_stage_time() waits for the recorded events, returns the summed elapsed
 * milliseconds, stores the number of launches in *h_launches, and clears the
 * record.  Events are created by the library on first use and destroyed by
 * dbt_destroy.  Stages: */
enum {
  DBT_STAGE_QKV = 0,    /* stacked Q/K/V projection kernel */
  DBT_STAGE_ATTN = 1,   /* grouped decode-attention kernel (without the split merge) */
  DBT_STAGE_WO = 2,     /* attention output projection kernel */
  DBT_STAGE_GATEUP = 3, /* gate/up projection kernel */
  DBT_STAGE_DOWN = 4,   /* down projection kernel */
  DBT_STAGE_LMHEAD = 5, /* output-matrix projection kernel */
  DBT_STAGE_MIX = 6,    /* mixture readout kernels */
  DBT_STAGE_COUNT = 7
};
dbt_status dbt_stage_timing(dbt_model *m, int32_t stage, int32_t enable);
double dbt_stage_time(dbt_model *m, int32_t stage, int32_t *h_launches);

#ifdef __cplusplus
}
#endif

#endif /* DBT_H */
