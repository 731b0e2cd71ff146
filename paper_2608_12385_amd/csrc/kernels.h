// Launchers of the device kernels (internal to the library; the public
// interface is include/dbt.h).  Every launcher enqueues on `st` and returns
// hipGetLastError() of its launches.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dbt {

// Up to three stacked weight matrices that one projection reads as one
// [sum rows][K] operand (e.g. W_Q; W_K; W_V).  Unused entries have rows 0.
struct WSegs {
  const void *w[3];
  int rows[3];
};

// Which activation rows a kernel processes.  Activations of a call are laid
// out [2][Bp][width]: path p (0 primary, 1 branch) sequence b sits at
// physical row p*Bp + b, Bp = batch rounded up to 16.
struct Rows {
  int B;   // sequences
  int Bp;  // row stride between the two paths
  int p0;  // first active path
  int np;  // active paths (1 or 2)
};

enum Mode { MODE_GROUPED = 0, MODE_PRIMARY = 1, MODE_BRANCH = 2 };

// Retention of primary intermediates for a later branch evaluation.
// src_row < 0: row b of the call is kept at retained row b (all rows);
// src_row >= 0: only that row is kept, at retained row dst_row.
struct Retain {
  float *ptr;  // NULL: nothing kept
  int src_row, dst_row;
};

struct KVRef {
  void *k, *v;            // pages of this layer: k/v base + layer offset already applied
  const int *page_table;  // [max_batch][mpps]
  int mpps;               // entries per sequence
  int n_kv, d_h;
};

// ---- projections ----
struct GemmConfig {
  int RB;      // 16-row blocks per wave (a workgroup owns NW*16*RB weight rows)
  int PD;      // weight prefetch depth in 128-element chunks
  int S;       // reduction splits (one fp32 output slab per split)
  int NW = 4;  // waves per workgroup (4 or 8)
};
GemmConfig gemm_config(int n_full, int K, int dtype, int seg_gran, int max_rows);

// Gate/up projection with the SwiGLU + b-coupling epilogue fused (Eqs. (13)-(14)):
// writes the MLP intermediate H (bf16, rows p*Bp + b, leading dimension ldh)
// instead of fp32 gate/up outputs.  Branch rows take H1 from the primary rows of
// the same call (mode GROUPED) or from H1_in (mode BRANCH); primary rows are
// kept in ret when asked.  Usable when gemm_glu_ok() holds.
struct GluEpi {
  Rows rows;
  int mode;
  int f;
  const float *bvec;   // [f]
  const float *H1_in;  // [B][f] (mode BRANCH)
  Retain ret;
  uint16_t *Xh;
  int ldh;
};
bool gemm_glu_ok(int f, int M, int np, int dtype);
hipError_t launch_gemm_glu(const uint16_t *w_gate, const uint16_t *w_up, int f, int K, const void *X, int ldx, int M,
                           const GluEpi &ep, hipStream_t st);
hipError_t launch_gemm(const WSegs &segs, int N, int K, int dtype, const void *X, int ldx, int M,
                       float *Y, int ldy, long long y_split_stride, const GemmConfig &g, hipStream_t st,
                       float *row_stats = nullptr);
// Tiles per row of the statistics the output projection writes when given
// row_stats (0: this shape does not produce them).
int gemm_stats_tiles(int N, const GemmConfig &g, int dtype);
int gemm_tile_rows(const GemmConfig &g);  // weight rows (output columns) per workgroup

// Projection of a whole prompt (M >= 256 rows, K a multiple of 64, N a
// multiple of 16, bf16): 256-row tiles on the matrix cores.  Plain: Y (fp32,
// [M][ldy]) = X W^T with W the stacked segments w[0..2] (rows[0..2] rows).
// GLU: w[0] = gate, w[1] = up (N = f rows each); writes H (bf16, [M][ldh]) =
// silu(X Wg^T) * (X Wu^T), and row ret_src of H in fp32 to ret + ret_dst*N
// when ret is not NULL (ret_src < 0: every row m to ret + m*N).
// QKV (rope != NULL; bf16 cache, d_h 128, rows = positions of sequence seq,
// w = W_Q, W_K, W_V): the rotary embedding on Q and K, Q (fp32, [M][rows[0]])
// to Qout and its row ret_src to ret + ret_dst*rows[0] (when ret is not
// NULL; ret_src < 0: every row m to ret + m*rows[0]), K and V into the cache
// slots of their positions; no Y.
struct TileGemm {
  const uint16_t *w[3];
  int rows[3];
  int N, K;
  const uint16_t *X;
  int ldx, M;
  float *Y;
  int ldy;
  uint16_t *H;
  int ldh;
  float *ret;
  int ret_src, ret_dst;
  const float2 *rope;  // [max_pos][64] (cos, sin)
  float *Qout;
  KVRef kv;
  int seq;
};
bool gemm_tile_ok(int N, int K, int M, int dtype);
// Everything launch_gemm_tile requires of g (the shape test above, segment
// sizes multiples of 8 summing to N, row strides multiples of 8, element
// offsets within 32 bits); callers fall back to launch_gemm otherwise.
bool gemm_tile_args_ok(const TileGemm &g, bool glu);
hipError_t launch_gemm_tile(const TileGemm &g, bool glu, hipStream_t st);

// ---- row-wise and elementwise stages ----
struct StepBegin {
  int n_pos, b0;
  int pos[64];
  int n_pt;
  int pt_b[64], pt_slot[64], pt_page[64];
};
hipError_t launch_step_begin(const StepBegin &sb, int *pos_arr, int *page_table, int mpps,
                             hipStream_t st);

// The step's first kernel also applies `sb` (positions and new page-table
// entries) when sb is not NULL.
hipError_t launch_embed(const int *tokens, int vocab, const void *e1, const void *e2, const float *g_emb,
                        const float *g_next, float eps, int d, int dtype, Rows rows, float *S,
                        void *Xn, int ldx, hipStream_t st, const StepBegin *sb = nullptr,
                        int *pos_arr = nullptr, int *page_table = nullptr, int mpps = 0);
hipError_t launch_load_hidden(const float *h1, const float *h2, const float *g_next, float eps,
                              int d, int dtype, Rows rows, float *S, void *Xn, int ldx,
                              hipStream_t st, const StepBegin *sb = nullptr, int *pos_arr = nullptr,
                              int *page_table = nullptr, int mpps = 0);
hipError_t launch_rmsnorm_rows(const float *S, const float *g, float eps, int d, int dtype,
                               Rows rows, void *Xn, int ldx, hipStream_t st);

// The first layer of a layer-only model read straight from the step's
// residual inputs, with no norm kernel before it: RMSNorm(h) W^T =
// (1/rms(h)) (h * g) W^T, so the QKV projection stages bf16(h * g) and
// writes, per reduction split, each row's sum of squares of h over the
// split's columns; the QKV finish scales each summed output by
// 1/sqrt(sum / d + eps) and the residual step reads h as the residual.
struct HIn {
  const float *h1;  // [B][d] primary rows (NULL: not in use)
  const float *h2;  // [n_b][B][d] branch rows
  int B;
};
struct XNorm {
  HIn h;
  Rows rows;     // the call's rows: row m is path p0 + m / Bp, sequence m % Bp
  const float *g;  // [d] attention-norm gain
  float *ss;     // [S][ss_ld] per split: ss[s * ss_ld + p*Bp + b]
  int ss_ld;
  StepBegin sb;  // applied by the first workgroup (positions, page-table entries)
  int *pos_arr, *page_table, mpps;
};
// Whether launch_gemm_xnorm runs this configuration.
bool gemm_xnorm_ok(const GemmConfig &g, int M);
hipError_t launch_gemm_xnorm(const WSegs &segs, int N, int K, const XNorm &xn, int M, float *Y, int ldy,
                             long long y_split_stride, const GemmConfig &g, hipStream_t st);

struct QKVFinish {
  const float *part;
  long long split_stride;
  int S, ldp;
  int n_q, n_kv, d_h;
  Rows rows;
  int mode;
  const float2 *rope;  // [max_pos][d_h/2] (cos, sin)
  const int *pos_arr;  // decode: position of sequence b (NULL: prefill)
  int seq_fixed;       // prefill: the sequence; the row index is the position
  const float *a;
  float *Q;            // [2Bp][n_q*d_h]
  const float *Q1_in;  // branch mode: retained primary queries [*, n_q*d_h]
  Retain ret;
  KVRef kv;
  int dtype;
  // rows from XNorm: each summed output of physical row R is scaled by
  // 1/sqrt(sum_{s < ss_S} ss[s * ss_ld + R] / d_model + eps) (ss NULL: 1)
  const float *ss;
  int ss_ld, ss_S, d_model;
  float eps;
};
hipError_t launch_qkv_finish(const QKVFinish &f, hipStream_t st);

// Compute-matched variant (App. B.3): a branch row takes g * (the primary
// row's value) instead of its own.  g == NULL: the standard model.
struct GatedCopy {
  const float *g;   // [d]
  const float *in;  // [B][d] primary values (branch-only calls)
  Retain ret;       // keep the primary values for a later branch-only call
};
// hin.h1 not NULL: the residual of row (path, b) is the step input h (see
// XNorm) instead of Sres; the sum is written to Sres either way.
hipError_t launch_resid_norm(const float *part, long long split_stride, int S, int ldp, float *Sres,
                             const float *g, float eps, int d, int dtype, Rows rows, void *Xn, int ldx,
                             hipStream_t st, const GatedCopy &gc = GatedCopy{}, const HIn &hin = HIn{});

hipError_t launch_swiglu_finish(const float *part, long long split_stride, int S, int ldp, int f,
                                int mode, Rows rows, const float *bvec, const float *H1_in,
                                Retain ret, int dtype, void *Xh, int ldh, hipStream_t st);

hipError_t launch_down_finish(const float *part, long long split_stride, int S, int ldp, int d,
                              int mode, Rows rows, const float *cvec, const float *M1_in,
                              Retain ret, float *Sres, const float *g_next, float eps, int dtype,
                              void *Xn, int ldx, hipStream_t st);

// ---- attention ----
struct AttnArgs {
  const float *Q;  // [2Bp][n_q*d_h]
  KVRef kv;
  const int *pos_arr;  // length of sequence b = pos_arr[b] + 1
  Rows rows;
  int n_q;
  int pages_per_split;  // target: a sequence of P pages is read in ceil(P / target) equal splits
  int max_splits;
  float *opart;  // [B][n_kv][max_splits][16][d_h]
  float *ostat;  // [B][n_kv][max_splits][16][2]
  int dtype;
  // bf16, every sequence at most 1024 pages: one workgroup of eight waves per
  // (sequence, KV head) writes the normalised rows to O (bf16, row stride
  // ldo); no partials and no combine launch
  int single;
  void *O;
  int ldo;
  // bf16, not single: splits of up to 1024 pages in workgroups of eight waves
  // (else up to 128 pages in workgroups of four)
  int wide;
  // bf16 decode: the queries and the cache append are computed by the
  // attention kernel itself from the QKV projection's split-K slabs (fin),
  // exactly as k_qkv_finish would (one launch fewer); Q is then not read
  int fused;
  QKVFinish fin;
};
hipError_t launch_attn_decode(const AttnArgs &a, hipStream_t st);
hipError_t launch_attn_combine(const AttnArgs &a, void *O, int ldo, hipStream_t st);

// Causal attention of prompt positions 0..T-1 of one sequence (rows = positions).
hipError_t launch_attn_prefill(const float *Q, int ldq, int T, KVRef kv, int seq, int n_q,
                               int dtype, void *O, int ldo, hipStream_t st);

// ---- cache fill ----
hipError_t launch_kv_fill(KVRef kv, int seq, int start, int count, const void *ksrc,
                          const void *vsrc, int dtype, hipStream_t st);

// ---- mixture readout (Sec. 4.2) ----
struct MixArgs {
  const float *logits;  // [(1 + n_b) Bp][V]
  int V;
  Rows rows;            // np = 1 + n_b with the branches on (n_b <= 3), 1 (primary) otherwise
  int chunk;            // vocabulary entries per statistics chunk when the projection wrote none
  float *stats;         // [(1 + n_b) Bp][nstat][3] per tile (max, sum e^(z-max), sum e^(2(z-max)))
  int nstat;            // tiles per row in stats
  int tile_w;           // vocabulary entries per tile (the projection's rows per workgroup, or chunk)
  int stats_ready;      // 1: the output projection already wrote stats
  float *alpha;         // [B] or NULL
  int *next;            // [B] or NULL
};
hipError_t launch_mixture(const MixArgs &m, hipStream_t st);

// ---- MoE (Sec. 3.2, Sec. 4.3, Sec. 5) ----
// Per-row selections live in [2Bp][8] arrays (row = path*Bp + b, k <= 8).
struct MoeRoute {
  const float *Sbar;  // [2Bp][d] residual after attention (fp32)
  const float *g;     // MLP norm gain
  float eps;
  int d;
  const void *Wr;     // [E][d] bf16 router
  int E, k1, k2, replay;
  Rows rows;
  int mode;
  float *logits;      // [2Bp][256] router logits (fp32)
  int *idx;           // [2Bp][8] selected experts (logit descending)
  float *wts;         // [2Bp][8] renormalised weights
  const int *idx1_in; // branch mode + replay: retained primary selections [*, 8]
  int *out_idx1, *out_idx2;
  float *out_w1, *out_w2;  // caller outputs [B][k] of this layer (may be NULL)
  float *out_lg1, *out_lg2;  // caller router logits [B][E] of this layer (may be NULL)
  int *ret_idx;       // retained primary selections (may be NULL)
  int ret_src, ret_dst;
};
struct MoeDispatch {
  const int *idx;
  Rows rows;
  int k1, k2, E;
  int *counts;   // [E]
  int *offsets;  // [E+1]
  int *arow;     // [A] activation row of each expert-grouped assignment
  int *aslot;    // [2Bp][8] position of each (row, slot) in the expert-grouped order
};
struct MoeGemm {
  const void *X;  // gate/up: normalized MLP inputs (gathered by arow); down: expert intermediates
  int ldx;
  const void *W0, *W1;  // gate/up: x_gate, x_up; down: x_down
  int E, N, K;
  const int *counts, *offsets, *arow;
  void *Y;  // gate/up: [A][N] bf16 intermediates; down: [A][N] fp32 outputs
  int ldy;
};
struct MoeCombine {
  Rows rows;
  int mode, d, k1, k2;
  const int *idx;
  const float *wts;
  const int *aslot;
  const float *Yexp;  // [A][d]
  const float *part;  // shared-expert down projection slabs (S_sh of them)
  long long stride;
  int S_sh;
  const float *c;
  const float *M1_in;  // compute-matched: G1 (primary shared-expert output) instead
  Retain ret;          // compute-matched: keeps G1
  const float *gG;     // compute-matched variant (App. B.3): branch M2 = R2 + gG * G1; NULL otherwise
  float *S;
  const float *g_next;
  float eps;
  void *Xn;
  int ldx;
};
hipError_t launch_moe_route(const MoeRoute &a, hipStream_t st);
hipError_t launch_moe_dispatch(const MoeDispatch &a, hipStream_t st);
hipError_t launch_moe_gemm(const MoeGemm &a, bool gateup, int max_rows, hipStream_t st);
hipError_t launch_moe_combine(const MoeCombine &a, int dtype, hipStream_t st);

}  // namespace dbt
