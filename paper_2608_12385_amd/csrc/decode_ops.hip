// Row-wise stages of the decode step: embeddings (Eq. (7)), RMSNorms, the
// epilogues that finish each projection (RoPE + query coupling + cache
// append, Eqs. (8)-(11); residual adds; SwiGLU + MLP coupling, Eq. (14);
// output coupling, Eq. (15)), direct cache fill, and the mixture readout
// (Sec. 4.2, Eqs. (17)-(18)).
//
// Split-K partial slabs are always added in split order, and every reduction
// has a fixed order, so results are deterministic and a row's value does not
// depend on which other rows are active.
#include "common.h"
#include "kernels.h"

#include <algorithm>

namespace dbt {

namespace {

__device__ __forceinline__ int phys_row(const Rows &r, int path, int b) { return path * r.Bp + b; }


// ---------------------------------------------------------------------------

__global__ void k_step_begin(StepBegin sb, int *pos_arr, int *page_table, int mpps) {
  const int t = threadIdx.x;
  if (t < sb.n_pos) pos_arr[sb.b0 + t] = sb.pos[t];
  if (t < sb.n_pt) page_table[(size_t)sb.pt_b[t] * mpps + sb.pt_slot[t]] = sb.pt_page[t];
}

// Per-step positions and page-table entries travel as kernel arguments of
// the step's first kernel (no host-to-device copy); block (0,0) writes them.
__device__ __forceinline__ void apply_step_begin(const StepBegin &sb, int *pos_arr, int *page_table, int mpps) {
  if (blockIdx.x != 0 || blockIdx.y != 0 || !pos_arr) return;
  const int t = threadIdx.x;
  if (t < sb.n_pos) pos_arr[sb.b0 + t] = sb.pos[t];
  if (t < sb.n_pt) page_table[(size_t)sb.pt_b[t] * mpps + sb.pt_slot[t]] = sb.pt_page[t];
}

// Row kernels use one workgroup per row (or row pair) with float4 accesses;
// d is a multiple of 4.  st4 writes four consecutive values in dtype T.
template <typename T> __device__ __forceinline__ void st4(T *p, size_t i4, float4 v);
template <> __device__ __forceinline__ void st4<float>(float *p, size_t i4, float4 v) { ((float4 *)p)[i4] = v; }
template <> __device__ __forceinline__ void st4<uint16_t>(uint16_t *p, size_t i4, float4 v) {
  uint2 u;
  u.x = (uint32_t)f2bf(v.x) | ((uint32_t)f2bf(v.y) << 16);
  u.y = (uint32_t)f2bf(v.z) | ((uint32_t)f2bf(v.w) << 16);
  ((uint2 *)p)[i4] = u;
}
template <typename T> __device__ __forceinline__ float4 ld4(const T *p, size_t i4);
template <> __device__ __forceinline__ float4 ld4<float>(const float *p, size_t i4) { return ((const float4 *)p)[i4]; }
template <> __device__ __forceinline__ float4 ld4<uint16_t>(const uint16_t *p, size_t i4) {
  const uint2 u = ((const uint2 *)p)[i4];
  return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u), __uint_as_float(u.y << 16),
                     __uint_as_float(u.y & 0xffff0000u));
}
__device__ __forceinline__ float dot4(float4 a) { return a.x * a.x + a.y * a.y + a.z * a.z + a.w * a.w; }
__device__ __forceinline__ float4 add4(float4 a, float4 b) { return make_float4(a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w); }
__device__ __forceinline__ float4 mul4(float4 a, float s, float4 g) {
  return make_float4(a.x * s * g.x, a.y * s * g.y, a.z * s * g.z, a.w * s * g.w);
}
__device__ __forceinline__ float4 psum4(const float *part, long long stride, int S, size_t idx4) {
  float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll 4
  for (int k = 0; k < S; ++k) s = add4(s, ((const float4 *)(part + k * stride))[idx4]);
  return s;
}
// Split-K slabs 0..7 of float4 element idx4, requested as eight
// unconditional loads (slabs past S re-read slab S - 1 and are not added):
// the loads of several rows are then all in flight before the first sum
// waits, where a loop over S would wait for every outstanding load first.
__device__ __forceinline__ void slabs_issue(const float *part, long long stride, int S, size_t idx4,
                                            float4 (&v)[8]) {
#pragma unroll
  for (int k = 0; k < 8; ++k) v[k] = ((const float4 *)(part + (long long)min(k, S - 1) * stride))[idx4];
}
// ONE: a single slab (the prompt projections) takes one load; the zeros in
// the other places are not added.
template <bool ONE>
__device__ __forceinline__ void slabs_load(const float *part, long long stride, int S, size_t idx4, float4 (&v)[8]) {
  if constexpr (ONE) {
    v[0] = ((const float4 *)part)[idx4];
#pragma unroll
    for (int k = 1; k < 8; ++k) v[k] = make_float4(0.f, 0.f, 0.f, 0.f);
  } else {
    slabs_issue(part, stride, S, idx4, v);
  }
}
// Their sum in split order, the same additions as psum4 (adding +0 for the
// slabs past S leaves the bits alone: a sum 0 + v + ... is never -0).
__device__ __forceinline__ float4 slabs_sum(const float *part, long long stride, int S, size_t idx4,
                                            const float4 (&v)[8]) {
  const float4 z = make_float4(0.f, 0.f, 0.f, 0.f);
  float4 s = z;
#pragma unroll
  for (int k = 0; k < 8; ++k) s = add4(s, k < S ? v[k] : z);
  for (int k0 = 8; k0 < S; k0 += 8) {  // more than eight splits: eight more per round trip
    float4 w[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) w[k] = ((const float4 *)(part + (long long)min(k0 + k, S - 1) * stride))[idx4];
#pragma unroll
    for (int k = 0; k < 8; ++k) s = add4(s, k0 + k < S ? w[k] : z);
  }
  return s;
}

// out = x / sqrt(mean(x^2) + eps) * g (x read from global, fp32)
template <typename T>
__device__ void norm_row(const float *x, const float *g, float eps, int d, T *out, float *red) {
  float ss = 0.f;
  for (int i = threadIdx.x; i < d / 4; i += blockDim.x) ss += dot4(((const float4 *)x)[i]);
  ss = block_sum(ss, red);
  const float inv = 1.0f / sqrtf(ss / (float)d + eps);
  for (int i = threadIdx.x; i < d / 4; i += blockDim.x)
    st4<T>(out, i, mul4(((const float4 *)x)[i], inv, ((const float4 *)g)[i]));
}

// The same norm on a row a thread holds in registers: v[k] is element
// (float4) i = threadIdx.x + k * blockDim.x of the row, valid while i < d/4.
// The row is not read back from memory.
// gv[k] holds the gain of element i, loaded by the caller ahead of time
// (its load then overlaps the row's own loads or the reduction).
template <typename T, int R>
__device__ __forceinline__ void norm_regs_g(const float4 (&v)[R], const float4 (&gv)[R], float eps, int d, T *out,
                                            float *red) {
  float ss = 0.f;
#pragma unroll
  for (int k = 0; k < R; ++k)
    if (threadIdx.x + k * blockDim.x < d / 4) ss += dot4(v[k]);
  ss = block_sum(ss, red);
  const float inv = 1.0f / sqrtf(ss / (float)d + eps);
#pragma unroll
  for (int k = 0; k < R; ++k) {
    const int i = threadIdx.x + k * blockDim.x;
    if (i < d / 4) st4<T>(out, i, mul4(v[k], inv, gv[k]));
  }
}
template <typename T, int R>
__device__ __forceinline__ void norm_regs(const float4 (&v)[R], const float *g, float eps, int d, T *out,
                                          float *red) {
  float4 gv[R];
#pragma unroll
  for (int k = 0; k < R; ++k) {
    const int i = threadIdx.x + k * blockDim.x;
    gv[k] = i < d / 4 ? ((const float4 *)g)[i] : make_float4(0.f, 0.f, 0.f, 0.f);
  }
  norm_regs_g<T, R>(v, gv, eps, d, out, red);
}

// Tokens outside [0, vocab) read as a zero embedding row (no out-of-bounds read).
template <typename T, int R>
__global__ void k_embed(const int *tokens, int vocab, const T *e1, const T *e2, const float *g_emb,
                        const float *g_next, float eps, int d, Rows rows, float *S, T *Xn, int ldx, StepBegin sb,
                        int *pos_arr, int *page_table, int mpps) {
  __shared__ float red[16];
  apply_step_begin(sb, pos_arr, page_table, mpps);
  const int b = blockIdx.x, path = rows.p0 + blockIdx.y;
  const int row = phys_row(rows, path, b);
  const int tok = tokens[b];
  const bool valid = tok >= 0 && tok < vocab;
  // decode branch j >= 1 reads table j of the branch tables (App. C.1 for j >= 2)
  const T *e = (path == 0 ? e1 : e2 + (size_t)(path - 1) * vocab * d) + (size_t)(valid ? tok : 0) * d;
  float4 v[R];
  float ss = 0.f;
#pragma unroll
  for (int k = 0; k < R; ++k) {
    const int i = threadIdx.x + k * blockDim.x;
    v[k] = valid && i < d / 4 ? ld4<T>(e, i) : make_float4(0.f, 0.f, 0.f, 0.f);
    ss += dot4(v[k]);
  }
  ss = block_sum(ss, red);
  const float inv = 1.0f / sqrtf(ss / (float)d + eps);
  float4 *s = (float4 *)(S + (size_t)row * d);
#pragma unroll
  for (int k = 0; k < R; ++k) {
    const int i = threadIdx.x + k * blockDim.x;
    if (i < d / 4) {
      v[k] = mul4(v[k], inv, ((const float4 *)g_emb)[i]);
      s[i] = v[k];
    }
  }
  norm_regs<T, R>(v, g_next, eps, d, Xn + (size_t)row * ldx, red);
}

template <typename T, int R>
__global__ void k_load_hidden(const float *h1, const float *h2, const float *g_next, float eps, int d,
                              Rows rows, float *S, T *Xn, int ldx, StepBegin sb, int *pos_arr, int *page_table,
                              int mpps) {
  __shared__ float red[16];
  apply_step_begin(sb, pos_arr, page_table, mpps);
  const int b = blockIdx.x, path = rows.p0 + blockIdx.y;
  const int row = phys_row(rows, path, b);
  const float4 *h = (const float4 *)((path == 0 ? h1 : h2 + (size_t)(path - 1) * rows.B * d) + (size_t)b * d);
  float4 *s = (float4 *)(S + (size_t)row * d);
  float4 v[R], gv[R];
#pragma unroll
  for (int k = 0; k < R; ++k) {
    const int i = threadIdx.x + k * blockDim.x;
    v[k] = i < d / 4 ? h[i] : make_float4(0.f, 0.f, 0.f, 0.f);
    gv[k] = i < d / 4 ? ((const float4 *)g_next)[i] : make_float4(0.f, 0.f, 0.f, 0.f);
    if (i < d / 4) s[i] = v[k];
  }
  norm_regs_g<T, R>(v, gv, eps, d, Xn + (size_t)row * ldx, red);
}

template <typename T>
__global__ void k_rmsnorm_rows(const float *S, const float *g, float eps, int d, Rows rows, T *Xn, int ldx) {
  __shared__ float red[16];
  const int row = phys_row(rows, rows.p0 + blockIdx.y, blockIdx.x);
  norm_row<T>(S + (size_t)row * d, g, eps, d, Xn + (size_t)row * ldx, red);
}

// ---------------------------------------------------------------------------
// QKV epilogue: one thread per rotation pair (i, i + d_h/2) of a query head,
// a key head or a value head.  Primary: Q1, K1 = RoPE(.), V1; K1/V1 go to the
// cache slot of position pos (Sec. 4.4: the primary appends).  Branch:
// Q2 = RoPE(.), Q2~ = Q2 + a * Q1 (Eq. (11)); the branch writes no cache.
template <typename T>
__global__ void k_qkv_finish(QKVFinish f) {
  const int b = blockIdx.y;
  const int half = f.d_h / 2;
  const int nqp = f.n_q * half, nkp = f.n_kv * half;
  const bool prim = f.mode != MODE_BRANCH, br = f.mode != MODE_PRIMARY;
  const int total = prim ? nqp + 2 * nkp : nqp;
  const int pi = blockIdx.x * blockDim.x + threadIdx.x;
  if (pi >= total) return;
  const int pos = f.pos_arr ? f.pos_arr[b] : b;
  const int seq = f.pos_arr ? b : f.seq_fixed;
  const int dq = f.n_q * f.d_h, dkv = f.n_kv * f.d_h;
  const int r1 = phys_row(f.rows, 0, b);
  const int pb0 = f.rows.p0 > 1 ? f.rows.p0 : 1, pb1 = f.rows.p0 + f.rows.np;  // branch paths of the call
  const int i = pi % half;
  const float2 cs = f.rope[(size_t)pos * half + i];
  if (pi < nqp) {
    const int c0 = (pi / half) * f.d_h + i, c1 = c0 + half;
    float q1a = 0.f, q1b = 0.f;
    if (prim) {
      const float2 q1 = rope_pair(psum(f.part, f.split_stride, f.S, (size_t)r1 * f.ldp + c0),
                                  psum(f.part, f.split_stride, f.S, (size_t)r1 * f.ldp + c1), cs);
      q1a = q1.x;
      q1b = q1.y;
      f.Q[(size_t)r1 * dq + c0] = q1a;
      f.Q[(size_t)r1 * dq + c1] = q1b;
      if (f.ret.ptr && (f.ret.src_row < 0 || f.ret.src_row == b)) {
        const int dst = f.ret.src_row < 0 ? b : f.ret.dst_row;
        f.ret.ptr[(size_t)dst * dq + c0] = q1a;
        f.ret.ptr[(size_t)dst * dq + c1] = q1b;
      }
    } else {
      q1a = f.Q1_in[(size_t)b * dq + c0];
      q1b = f.Q1_in[(size_t)b * dq + c1];
    }
    if (br)
      for (int p = pb0; p < pb1; ++p) {  // every branch couples to Q1 with the shared a
        const int r2 = phys_row(f.rows, p, b);
        const float2 q2 = rope_pair(psum(f.part, f.split_stride, f.S, (size_t)r2 * f.ldp + c0),
                                    psum(f.part, f.split_stride, f.S, (size_t)r2 * f.ldp + c1), cs);
        f.Q[(size_t)r2 * dq + c0] = couple(f.a[c0], q1a, q2.x);
        f.Q[(size_t)r2 * dq + c1] = couple(f.a[c1], q1b, q2.y);
      }
    return;
  }
  // keys and values (primary only): cache slot of position pos
  const int page = f.kv.page_table[(size_t)seq * f.kv.mpps + pos / 16];
  const int slot = pos % 16;
  const int j = pi - nqp;
  T *kp = (T *)f.kv.k;
  T *vp = (T *)f.kv.v;
  if (j < nkp) {
    const int g = j / half;
    const int c0 = dq + g * f.d_h + i;
    const float2 k = rope_pair(psum(f.part, f.split_stride, f.S, (size_t)r1 * f.ldp + c0),
                               psum(f.part, f.split_stride, f.S, (size_t)r1 * f.ldp + c0 + half), cs);
    const size_t base = (((size_t)page * f.n_kv + g) * 16 + slot) * f.d_h;
    st<T>(kp, base + i, k.x);
    st<T>(kp, base + i + half, k.y);
  } else {
    const int g = (j - nkp) / half;
    const int c0 = dq + dkv + g * f.d_h + i;
    const float v0 = psum(f.part, f.split_stride, f.S, (size_t)r1 * f.ldp + c0);
    const float v1 = psum(f.part, f.split_stride, f.S, (size_t)r1 * f.ldp + c0 + half);
    const size_t base = ((size_t)page * f.n_kv + g) * f.d_h;
    st<T>(vp, (base + i) * 16 + slot, v0);
    st<T>(vp, (base + i + half) * 16 + slot, v1);
  }
}

// After the attention output projection: S_bar = S + A (in place), then the
// MLP input RMSNorm.  Compute-matched variant (App. B.3): a branch row adds
// g_A * A1, A1 being the primary row's projection output (both paths in the
// call) or the kept A1 (branch-only call); primary rows can keep A1.
template <typename T, int R, bool ONE = false>
__global__ void k_resid_norm(const float *part, long long stride, int S, int ldp, float *Sres,
                             const float *g, float eps, int d, Rows rows, T *Xn, int ldx, GatedCopy gc, HIn hin) {
  __shared__ float red[16];
  const int b = blockIdx.x, path = rows.p0 + blockIdx.y;
  const int row = phys_row(rows, path, b);
  float4 *s = (float4 *)(Sres + (size_t)row * d);
  // the residual: Sres, or the step input of the row (first layer, XNorm)
  const float4 *sin = hin.h1 ? (const float4 *)((path == 0 ? hin.h1 : hin.h2 + (size_t)(path - 1) * hin.B * d) +
                                                (size_t)b * d)
                             : s;
  const bool keep = gc.g && path == 0 && gc.ret.ptr && (gc.ret.src_row < 0 || gc.ret.src_row == b);
  float4 *kept = keep ? (float4 *)(gc.ret.ptr + (size_t)(gc.ret.src_row < 0 ? b : gc.ret.dst_row) * d) : nullptr;
  const int r1 = phys_row(rows, 0, b);
  float4 v[R], gv[R];
#pragma unroll
  for (int k = 0; k < R; ++k) {
    const int i = threadIdx.x + k * blockDim.x;
    v[k] = gv[k] = make_float4(0.f, 0.f, 0.f, 0.f);
    if (i >= d / 4) continue;
    gv[k] = ((const float4 *)g)[i];
    if (!gc.g || path == 0) {
      float4 sl[8];
      slabs_load<ONE>(part, stride, S, ((size_t)row * ldp) / 4 + i, sl);
      const float4 x = sin[i];
      __builtin_amdgcn_sched_barrier(0);  // the sums after every load
      const float4 a1 = slabs_sum(part, stride, S, ((size_t)row * ldp) / 4 + i, sl);
      v[k] = add4(x, a1);
      if (keep) kept[i] = a1;
    } else {
      // compute-matched branch row: S_bar2 = S2 + g_A * A1
      const float4 a1 = rows.p0 == 0 ? psum4(part, stride, S, ((size_t)r1 * ldp) / 4 + i)
                                     : ((const float4 *)(gc.in + (size_t)b * d))[i];
      const float4 ga = ((const float4 *)gc.g)[i];
      const float4 x = sin[i];
      v[k] = make_float4(x.x + ga.x * a1.x, x.y + ga.y * a1.y, x.z + ga.z * a1.z, x.w + ga.w * a1.w);
    }
    s[i] = v[k];
  }
  norm_regs_g<T, R>(v, gv, eps, d, Xn + (size_t)row * ldx, red);
}

// SwiGLU and the MLP-intermediate coupling H2~ = H2 + b * H1 (Eq. (14)).
// Gate rows are columns [0, f) of the projection, up rows [f, 2f).
template <typename T>
__global__ void k_swiglu_finish(const float *part, long long stride, int S, int ldp, int f, int mode,
                                Rows rows, const float *bvec, const float *H1_in, Retain ret, T *Xh,
                                int ldh) {
  const int b = blockIdx.y;
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= f) return;
  const bool prim = mode != MODE_BRANCH, br = mode != MODE_PRIMARY;
  const int r1 = phys_row(rows, 0, b);
  const int pb0 = rows.p0 > 1 ? rows.p0 : 1, pb1 = rows.p0 + rows.np;
  float h1;
  if (prim) {
    const float gt = psum(part, stride, S, (size_t)r1 * ldp + j);
    const float up = psum(part, stride, S, (size_t)r1 * ldp + f + j);
    h1 = gt / (1.0f + expf(-gt)) * up;
    st<T>(Xh, (size_t)r1 * ldh + j, h1);
    if (ret.ptr && (ret.src_row < 0 || ret.src_row == b))
      ret.ptr[(size_t)(ret.src_row < 0 ? b : ret.dst_row) * f + j] = h1;
  } else {
    h1 = H1_in[(size_t)b * f + j];
  }
  if (br)
    for (int p = pb0; p < pb1; ++p) {
      const int r2 = phys_row(rows, p, b);
      const float gt = psum(part, stride, S, (size_t)r2 * ldp + j);
      const float up = psum(part, stride, S, (size_t)r2 * ldp + f + j);
      const float h2 = gt / (1.0f + expf(-gt)) * up;
      st<T>(Xh, (size_t)r2 * ldh + j, h2 + bvec[j] * h1);
    }
}

// After the MLP down projection: M1, M2 = M2' + c * M1 (Eq. (15)),
// S <- S_bar + M (Eq. (16)), then the next RMSNorm (next layer's attention
// norm, or the final norm before the output matrix).
template <typename T, int R, bool ONE = false>
__global__ void k_down_finish(const float *part, long long stride, int S, int ldp, int d, int mode,
                              Rows rows, const float *cvec, const float *M1_in, Retain ret,
                              float *Sres, const float *g_next, float eps, T *Xn, int ldx) {
  __shared__ float red[16];
  // one workgroup per (sequence, path); a branch row sums the primary's
  // slabs itself (the same additions, so the same M1 bits) for its coupling
  const int b = blockIdx.x, path = rows.p0 + blockIdx.y;
  const bool prim = mode != MODE_BRANCH;
  if (path == 0 && !prim) return;
  const int r1 = phys_row(rows, 0, b), row = phys_row(rows, path, b);
  float4 *s = (float4 *)(Sres + (size_t)row * d);
  const bool keep = path == 0 && ret.ptr && (ret.src_row < 0 || ret.src_row == b);
  float4 *kept = keep ? (float4 *)(ret.ptr + (size_t)(ret.src_row < 0 ? b : ret.dst_row) * d) : nullptr;
  float4 v[R], gv[R];
#pragma unroll
  for (int k = 0; k < R; ++k) {
    const int i = threadIdx.x + k * blockDim.x;
    v[k] = gv[k] = make_float4(0.f, 0.f, 0.f, 0.f);
    if (i >= d / 4) continue;
    // every load of the element first, the slabs unconditionally (a load
    // under a condition lets the compiler start the sums before the next
    // loads): slabs of the primary row and of this row (the same row twice
    // for the primary), the residual, the coupling (a stand-in address for
    // the primary) and the kept M1 of a branch-only call
    const size_t i1 = ((size_t)r1 * ldp) / 4 + i, i2 = ((size_t)row * ldp) / 4 + i;
    float4 sl1[8], sl2[8];
    if constexpr (ONE) {
      slabs_load<true>(part, stride, S, i1, sl1);
      slabs_load<true>(part, stride, S, i2, sl2);
    } else {
#pragma unroll
      for (int k2 = 0; k2 < 8; ++k2) {
        const long long o = (long long)min(k2, S - 1) * stride;
        sl1[k2] = ((const float4 *)(part + o))[i1];
        sl2[k2] = ((const float4 *)(part + o))[i2];
      }
    }
    const float4 x = s[i];
    const float4 c = (path >= 1 ? (const float4 *)cvec : s)[i];
    if constexpr (R <= 2) gv[k] = (g_next ? (const float4 *)g_next : s)[i];  // (registers allow)
    float4 m1 = make_float4(0.f, 0.f, 0.f, 0.f);
    if (!prim) m1 = ((const float4 *)(M1_in + (size_t)b * d))[i];
    __builtin_amdgcn_sched_barrier(0);  // the sums after every load
    if (prim) m1 = slabs_sum(part, stride, S, i1, sl1);
    if (path == 0) {
      v[k] = add4(x, m1);
      if (keep) kept[i] = m1;
    } else {
      const float4 m2 = slabs_sum(part, stride, S, i2, sl2);
      const float4 t = make_float4(m2.x + c.x * m1.x, m2.y + c.y * m1.y, m2.z + c.z * m1.z, m2.w + c.w * m1.w);
      v[k] = add4(x, t);
    }
    s[i] = v[k];
  }
  if (!g_next) return;
  if constexpr (R <= 2)
    norm_regs_g<T, R>(v, gv, eps, d, Xn + (size_t)row * ldx, red);
  else
    norm_regs<T, R>(v, g_next, eps, d, Xn + (size_t)row * ldx, red);
}

// ---------------------------------------------------------------------------

template <typename E>
__global__ void k_kv_fill(KVRef kv, int seq, int start, const E *ksrc, const E *vsrc) {
  const int x = blockIdx.x, g = blockIdx.y, t = threadIdx.x;
  const int pos = start + x;
  const int page = kv.page_table[(size_t)seq * kv.mpps + pos / 16];
  const int slot = pos % 16;
  const size_t src = ((size_t)x * kv.n_kv + g) * kv.d_h + t;
  ((E *)kv.k)[(((size_t)page * kv.n_kv + g) * 16 + slot) * kv.d_h + t] = ksrc[src];
  ((E *)kv.v)[(((size_t)page * kv.n_kv + g) * kv.d_h + t) * 16 + slot] = vsrc[src];
}

// ---------------------------------------------------------------------------
// Mixture readout.  Per (row, chunk) statistics (max, sum e^(z-max),
// sum e^(2(z-max))) give, after a fixed-order merge, lse and the collision
// probability sum p^2 = sum e^(2z) / (sum e^z)^2 (Eq. (18)); then the greedy
// token of alpha p + (1 - alpha) q, lowest index on ties.

__device__ __forceinline__ void argmax_merge(float &v, int &i, float v2, int i2) {
  if (v2 > v || (v2 == v && i2 < i)) { v = v2; i = i2; }
}

__global__ void k_mix_stats(MixArgs m) {
  __shared__ float red[16];
  const int c = blockIdx.x;
  const int y = blockIdx.y;
  const int path = m.rows.p0 + y / m.rows.B, b = y % m.rows.B;
  const int row = phys_row(m.rows, path, b);
  const int nch = m.nstat;
  const int lo = c * m.chunk, hi = min(m.V, lo + m.chunk);
  const float *z = m.logits + (size_t)row * m.V;
  // each thread keeps its values in registers between the two passes
  constexpr int PER = 16;
  float v[PER];
  float mx = -INFINITY;
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    const int idx = lo + threadIdx.x + k * blockDim.x;
    v[k] = idx < hi ? z[idx] : -INFINITY;
    mx = fmaxf(mx, v[k]);
  }
  for (int idx = lo + threadIdx.x + PER * blockDim.x; idx < hi; idx += blockDim.x) mx = fmaxf(mx, z[idx]);
  mx = block_max(mx, red);
  float s1 = 0.f, s2 = 0.f;
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    const float e = expf(v[k] - mx);
    s1 += e;
    s2 += e * e;
  }
  for (int idx = lo + threadIdx.x + PER * blockDim.x; idx < hi; idx += blockDim.x) {
    const float e = expf(z[idx] - mx);
    s1 += e;
    s2 += e * e;
  }
  s1 = block_sum(s1, red);
  s2 = block_sum(s2, red);
  if (threadIdx.x == 0) {
    float *o = m.stats + ((size_t)row * nch + c) * 3;
    o[0] = mx;
    o[1] = s1;
    o[2] = s2;
  }
}

// Greedy token of the mixture (Eqs. (17)-(18)); with several decode branches
// (App. C.1) q is the mean of the branch softmaxes, (1 - alpha) / n_b *
// sum_j q_j, branches summed in order.  One wave per sequence, NP = 1 + n_b
// path rows (1: branches off).
//
// The per-tile statistics (max, sum e^(z-max), sum e^(2(z-max))) of the
// output projection give lse of each row and sum p^2 (alpha).  Not every
// entry is then read: a tile T (row maxima max1_T, max2j_T) holds no mixture
// value above
//   ub_T = alpha e^(max1_T - lse1) + (1 - alpha)/n_b sum_j e^(max2j_T - lse2j),
// while the token attaining a tile maximum proves the lower bound
//   lb = max_T max(alpha e^(max1_T - lse1), (1 - alpha)/n_b e^(max2j_T - lse2j))
// on the largest value.  Only tiles with ub_T >= lb (1 - 2^-10) are scanned
// (the margin exceeds the fp32 rounding of both sides, so a skipped entry can
// never be the fp32 argmax), and every entry of a kept tile is evaluated.
// With the branches off the value is the primary logit itself and only tiles
// attaining the row maximum are scanned.  The lowest index wins ties.  The
// kernel is short: one memory round trip for the statistics and one for up
// to 16 kept tiles (float4 loads of 8 x 4 entries per thread and path), and
// little code (a cold instruction cache is a large part of such a kernel's
// time).
template <int NP, int VEC>
__global__ __launch_bounds__(256) void k_mix_select(MixArgs m) {
  constexpr int SB = VEC == 1 ? 8 : (NP <= 2 ? 8 : 4), MAXT = 4096;
  __shared__ float red[NP][3][4];
  __shared__ float lb_s[4];
  __shared__ int list[MAXT];
  __shared__ int cnt_s[4];
  __shared__ float rv[4];
  __shared__ int ri[4];
  const int b = blockIdx.x, t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const float *st[NP];
  const float *z[NP];
#pragma unroll
  for (int j = 0; j < NP; ++j) {
    st[j] = m.stats + (size_t)(j * m.rows.Bp + b) * m.nstat * 3;
    z[j] = m.logits + (size_t)(j * m.rows.Bp + b) * m.V;
  }
  // 1. lse and sum p^2: each thread merges its tiles t + 256k online, then
  //    the workgroup merges the threads (fixed tree); the maxima of the last
  //    round stay in registers
  float M[NP], Z[NP], Y[NP], x[NP];
#pragma unroll
  for (int j = 0; j < NP; ++j) {
    M[j] = -INFINITY;
    Z[j] = Y[j] = 0.f;
  }
  for (int T = t; T - t < m.nstat; T += 256) {
    float s1[NP], s2[NP];
#pragma unroll
    for (int j = 0; j < NP; ++j) {
      x[j] = T < m.nstat ? st[j][T * 3] : -INFINITY;
      s1[j] = T < m.nstat ? st[j][T * 3 + 1] : 0.f;
      s2[j] = T < m.nstat ? st[j][T * 3 + 2] : 0.f;
    }
#pragma unroll
    for (int j = 0; j < NP; ++j) {
      const float Mn = fmaxf(M[j], x[j]);
      if (Mn == -INFINITY) continue;
      const float fo = __expf(M[j] - Mn), fn = __expf(x[j] - Mn);
      Z[j] = Z[j] * fo + s1[j] * fn;
      Y[j] = Y[j] * fo * fo + s2[j] * fn * fn;
      M[j] = Mn;
    }
  }
#pragma unroll
  for (int j = 0; j < NP; ++j) {
    const float Mw = wave_max(M[j]);
    const float f = M[j] == -INFINITY ? 0.f : __expf(M[j] - Mw);
    const float Zw = wave_sum(Z[j] * f), Yw = j == 0 ? wave_sum(Y[j] * f * f) : 0.f;
    if (lane == 0) {
      red[j][0][wave] = Mw;
      red[j][1][wave] = Zw;
      red[j][2][wave] = Yw;
    }
  }
  __syncthreads();
  float lse[NP], p2 = 0.f;
#pragma unroll
  for (int j = 0; j < NP; ++j) {
    float Mb = -INFINITY, Zb = 0.f, Yb = 0.f;
    for (int w = 0; w < 4; ++w) Mb = fmaxf(Mb, red[j][0][w]);
    for (int w = 0; w < 4; ++w) {
      const float f = red[j][0][w] == -INFINITY ? 0.f : __expf(red[j][0][w] - Mb);
      Zb += red[j][1][w] * f;
      Yb += red[j][2][w] * f * f;
    }
    lse[j] = Mb + __logf(Zb);
    if (j == 0) p2 = Yb / (Zb * Zb);
  }
  const float alpha = NP > 1 ? fminf(1.f, fmaxf(0.5f, p2)) : 1.f;
  const float wq = NP > 1 ? (1.f - alpha) / (float)(NP - 1) : 0.f;
  // 2. bounds; tile maxima from registers in the last round, else reloaded
  const int lastT = (m.nstat - 1) / 256 * 256 + t;
  auto bounds = [&](int T, float &ub, float &lo) {
    float xt[NP];
#pragma unroll
    for (int j = 0; j < NP; ++j) xt[j] = T == lastT ? x[j] : (T < m.nstat ? st[j][T * 3] : -INFINITY);
    if (T >= m.nstat) {
      ub = lo = -INFINITY;
      return;
    }
    if (NP == 1) {
      ub = lo = xt[0];
      return;
    }
    const float p1 = alpha * __expf(xt[0] - lse[0]);
    float q = 0.f;
    lo = p1;
#pragma unroll
    for (int j = 1; j < NP; ++j) {
      const float e = __expf(xt[j] - lse[j]);
      q += e;
      lo = fmaxf(lo, wq * e);
    }
    ub = p1 + wq * q;
  };
  float lb = -INFINITY;
  for (int T = t; T - t < m.nstat; T += 256) {
    float ub, lo;
    bounds(T, ub, lo);
    lb = fmaxf(lb, lo);
  }
  lb = wave_max(lb);
  if (lane == 0) lb_s[wave] = lb;
  __syncthreads();
  lb = fmaxf(fmaxf(lb_s[0], lb_s[1]), fmaxf(lb_s[2], lb_s[3]));
  const float thr = NP > 1 ? lb * (1.f - 1.f / 1024.f) : lb;
  // 3. kept tiles into the list (rounds of 256, ballot per wave), then one
  //    flattened scan, SB entries per thread per memory round trip (any
  //    order: the merge keeps the largest value, then the lowest index)
  int nkeep = 0;
  for (int T = t; T - t < m.nstat; T += 256) {
    float ub, lo;
    bounds(T, ub, lo);
    const bool keep = ub >= thr;
    const unsigned long long bal = __ballot(keep);
    if (lane == 0) cnt_s[wave] = __popcll(bal);
    __syncthreads();
    int off = nkeep;
    for (int w = 0; w < wave; ++w) off += cnt_s[w];
    if (keep && off + __popcll(bal & ((1ull << lane) - 1ull)) < MAXT)
      list[off + __popcll(bal & ((1ull << lane) - 1ull))] = T;
    nkeep += cnt_s[0] + cnt_s[1] + cnt_s[2] + cnt_s[3];
    __syncthreads();
  }
  nkeep = min(nkeep, MAXT);
  // units of VEC consecutive entries (VEC divides the tile width and V, so
  // a unit never straddles a tile or the end); loads are unconditional (an
  // entry past the list re-reads the last unit and is not merged)
  const int tw = m.tile_w, units = tw / VEC, total = nkeep * units;
  float best = -INFINITY;
  int bi = 0x7fffffff;
  for (int e0 = 0; e0 < total; e0 += 256 * SB) {
    int vi[SB];
    float a[NP][SB][VEC];
#pragma unroll
    for (int i = 0; i < SB; ++i) {
      const int e = e0 + t + 256 * i, k = e < total ? e / units : 0;
      vi[i] = e < total ? list[k] * tw + (e - k * units) * VEC : m.V;
      const int vc = min(vi[i], m.V - VEC);
#pragma unroll
      for (int j = 0; j < NP; ++j) {
        if constexpr (VEC == 4) {
          const float4 x = *(const float4 *)(z[j] + vc);
          a[j][i][0] = x.x;
          a[j][i][1] = x.y;
          a[j][i][2] = x.z;
          a[j][i][3] = x.w;
        } else {
          a[j][i][0] = z[j][vc];
        }
      }
    }
#pragma unroll
    for (int i = 0; i < SB; ++i)
#pragma unroll
      for (int c = 0; c < VEC; ++c) {
        if (vi[i] + c >= m.V) continue;
        float val = a[0][i][c];
        if (NP > 1) {
          float qs = 0.f;
#pragma unroll
          for (int j = 1; j < NP; ++j) qs += __expf(a[j][i][c] - lse[j]);
          val = alpha * __expf(a[0][i][c] - lse[0]) + wq * qs;
        }
        argmax_merge(best, bi, val, vi[i] + c);
      }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float v2 = __shfl_xor(best, o, 64);
    const int i2 = __shfl_xor(bi, o, 64);
    argmax_merge(best, bi, v2, i2);
  }
  if (lane == 0) {
    rv[wave] = best;
    ri[wave] = bi;
  }
  __syncthreads();
  if (t == 0) {
    for (int w = 1; w < 4; ++w) argmax_merge(best, bi, rv[w], ri[w]);
    if (m.next) m.next[b] = bi;
    if (m.alpha) m.alpha[b] = alpha;
  }
}

}  // namespace

// ---------------------------------------------------------------------------

hipError_t launch_step_begin(const StepBegin &sb, int *pos_arr, int *page_table, int mpps, hipStream_t st) {
  if (sb.n_pos == 0 && sb.n_pt == 0) return hipSuccess;
  hipLaunchKernelGGL(k_step_begin, dim3(1), dim3(64), 0, st, sb, pos_arr, page_table, mpps);
  return hipGetLastError();
}

static int row_threads(int d) {
  int t = (d / 4 + 63) / 64 * 64;
  return t < 64 ? 64 : t > 1024 ? 1024 : t;
}

// float4 elements per thread of the register-resident row kernels (d up to
// 32768, checked when the model is created).
static int row_regs(int d) {
  const int n = (d / 4 + row_threads(d) - 1) / row_threads(d);
  return n <= 1 ? 1 : n <= 2 ? 2 : n <= 4 ? 4 : 8;
}
#define DBT_ROW_LAUNCH(KERNEL, T, d, ...)                                                            \
  switch (row_regs(d)) {                                                                            \
    case 1: hipLaunchKernelGGL((KERNEL<T, 1>), __VA_ARGS__); break;                                 \
    case 2: hipLaunchKernelGGL((KERNEL<T, 2>), __VA_ARGS__); break;                                 \
    case 4: hipLaunchKernelGGL((KERNEL<T, 4>), __VA_ARGS__); break;                                 \
    default: hipLaunchKernelGGL((KERNEL<T, 8>), __VA_ARGS__); break;                                \
  }

// The same with the single-slab form (ONE) of a split-K row kernel.
#define DBT_ROW_LAUNCH_ONE(KERNEL, T, d, ...)                                                        \
  switch (row_regs(d)) {                                                                            \
    case 1: hipLaunchKernelGGL((KERNEL<T, 1, true>), __VA_ARGS__); break;                           \
    case 2: hipLaunchKernelGGL((KERNEL<T, 2, true>), __VA_ARGS__); break;                           \
    case 4: hipLaunchKernelGGL((KERNEL<T, 4, true>), __VA_ARGS__); break;                           \
    default: hipLaunchKernelGGL((KERNEL<T, 8, true>), __VA_ARGS__); break;                          \
  }

hipError_t launch_embed(const int *tokens, int vocab, const void *e1, const void *e2, const float *g_emb,
                        const float *g_next, float eps, int d, int dtype, Rows rows, float *S,
                        void *Xn, int ldx, hipStream_t st, const StepBegin *sb, int *pos_arr, int *page_table,
                        int mpps) {
  dim3 grid(rows.B, rows.np);
  StepBegin none;
  none.n_pos = none.n_pt = 0;
  none.b0 = 0;
  const StepBegin &s = sb ? *sb : none;
  const int threads = std::max(row_threads(d), 64);
  if (dtype == 1) {
    DBT_ROW_LAUNCH(k_embed, uint16_t, d, grid, dim3(threads), 0, st, tokens, vocab, (const uint16_t *)e1,
                   (const uint16_t *)e2, g_emb, g_next, eps, d, rows, S, (uint16_t *)Xn, ldx, s, pos_arr,
                   page_table, mpps)
  } else {
    DBT_ROW_LAUNCH(k_embed, float, d, grid, dim3(threads), 0, st, tokens, vocab, (const float *)e1,
                   (const float *)e2, g_emb, g_next, eps, d, rows, S, (float *)Xn, ldx, s, pos_arr, page_table,
                   mpps)
  }
  return hipGetLastError();
}

hipError_t launch_load_hidden(const float *h1, const float *h2, const float *g_next, float eps,
                              int d, int dtype, Rows rows, float *S, void *Xn, int ldx, hipStream_t st,
                              const StepBegin *sb, int *pos_arr, int *page_table, int mpps) {
  dim3 grid(rows.B, rows.np);
  StepBegin none;
  none.n_pos = none.n_pt = 0;
  none.b0 = 0;
  const StepBegin &s = sb ? *sb : none;
  const int threads = std::max(row_threads(d), 64);
  if (dtype == 1) {
    DBT_ROW_LAUNCH(k_load_hidden, uint16_t, d, grid, dim3(threads), 0, st, h1, h2, g_next, eps, d, rows, S,
                   (uint16_t *)Xn, ldx, s, pos_arr, page_table, mpps)
  } else {
    DBT_ROW_LAUNCH(k_load_hidden, float, d, grid, dim3(threads), 0, st, h1, h2, g_next, eps, d, rows, S,
                   (float *)Xn, ldx, s, pos_arr, page_table, mpps)
  }
  return hipGetLastError();
}

hipError_t launch_rmsnorm_rows(const float *S, const float *g, float eps, int d, int dtype, Rows rows,
                               void *Xn, int ldx, hipStream_t st) {
  dim3 grid(rows.B, rows.np);
  if (dtype == 1)
    hipLaunchKernelGGL(k_rmsnorm_rows<uint16_t>, grid, dim3(row_threads(d)), 0, st, S, g, eps, d, rows, (uint16_t *)Xn, ldx);
  else
    hipLaunchKernelGGL(k_rmsnorm_rows<float>, grid, dim3(row_threads(d)), 0, st, S, g, eps, d, rows, (float *)Xn, ldx);
  return hipGetLastError();
}

hipError_t launch_qkv_finish(const QKVFinish &f, hipStream_t st) {
  if (f.ss) return hipErrorInvalidValue;  // rows from the step inputs: finished by the attention kernel only
  const int half = f.d_h / 2;
  const int total = f.mode != MODE_BRANCH ? (f.n_q + 2 * f.n_kv) * half : f.n_q * half;
  dim3 grid((total + 255) / 256, f.rows.B);
  if (f.dtype == 1)
    hipLaunchKernelGGL(k_qkv_finish<uint16_t>, grid, dim3(256), 0, st, f);
  else
    hipLaunchKernelGGL(k_qkv_finish<float>, grid, dim3(256), 0, st, f);
  return hipGetLastError();
}

hipError_t launch_resid_norm(const float *part, long long stride, int S, int ldp, float *Sres,
                             const float *g, float eps, int d, int dtype, Rows rows, void *Xn, int ldx,
                             hipStream_t st, const GatedCopy &gc, const HIn &hin) {
  dim3 grid(rows.B, rows.np);
  if (hin.h1 && hin.B < rows.B) return hipErrorInvalidValue;
  if (dtype == 1 && S == 1) {
    DBT_ROW_LAUNCH_ONE(k_resid_norm, uint16_t, d, grid, dim3(row_threads(d)), 0, st, part, stride, S, ldp, Sres, g,
                       eps, d, rows, (uint16_t *)Xn, ldx, gc, hin)
  } else if (dtype == 1) {
    DBT_ROW_LAUNCH(k_resid_norm, uint16_t, d, grid, dim3(row_threads(d)), 0, st, part, stride, S, ldp, Sres, g, eps,
                   d, rows, (uint16_t *)Xn, ldx, gc, hin)
  } else {
    DBT_ROW_LAUNCH(k_resid_norm, float, d, grid, dim3(row_threads(d)), 0, st, part, stride, S, ldp, Sres, g, eps, d,
                   rows, (float *)Xn, ldx, gc, hin)
  }
  return hipGetLastError();
}

hipError_t launch_swiglu_finish(const float *part, long long stride, int S, int ldp, int f, int mode,
                                Rows rows, const float *bvec, const float *H1_in, Retain ret, int dtype,
                                void *Xh, int ldh, hipStream_t st) {
  dim3 grid((f + 255) / 256, rows.B);
  if (dtype == 1)
    hipLaunchKernelGGL(k_swiglu_finish<uint16_t>, grid, dim3(256), 0, st, part, stride, S, ldp, f, mode, rows,
                       bvec, H1_in, ret, (uint16_t *)Xh, ldh);
  else
    hipLaunchKernelGGL(k_swiglu_finish<float>, grid, dim3(256), 0, st, part, stride, S, ldp, f, mode, rows,
                       bvec, H1_in, ret, (float *)Xh, ldh);
  return hipGetLastError();
}

hipError_t launch_down_finish(const float *part, long long stride, int S, int ldp, int d, int mode,
                              Rows rows, const float *cvec, const float *M1_in, Retain ret, float *Sres,
                              const float *g_next, float eps, int dtype, void *Xn, int ldx, hipStream_t st) {
  dim3 grid(rows.B, rows.np);
  if (dtype == 1 && S == 1) {
    DBT_ROW_LAUNCH_ONE(k_down_finish, uint16_t, d, grid, dim3(row_threads(d)), 0, st, part, stride, S, ldp, d, mode,
                       rows, cvec, M1_in, ret, Sres, g_next, eps, (uint16_t *)Xn, ldx)
  } else if (dtype == 1) {
    DBT_ROW_LAUNCH(k_down_finish, uint16_t, d, grid, dim3(row_threads(d)), 0, st, part, stride, S, ldp, d, mode, rows,
                   cvec, M1_in, ret, Sres, g_next, eps, (uint16_t *)Xn, ldx)
  } else {
    DBT_ROW_LAUNCH(k_down_finish, float, d, grid, dim3(row_threads(d)), 0, st, part, stride, S, ldp, d, mode, rows,
                   cvec, M1_in, ret, Sres, g_next, eps, (float *)Xn, ldx)
  }
  return hipGetLastError();
}

hipError_t launch_kv_fill(KVRef kv, int seq, int start, int count, const void *ksrc, const void *vsrc,
                          int dtype, hipStream_t st) {
  if (count <= 0) return hipSuccess;
  dim3 grid(count, kv.n_kv);
  if (dtype == 1)
    hipLaunchKernelGGL(k_kv_fill<uint16_t>, grid, dim3(kv.d_h), 0, st, kv, seq, start,
                       (const uint16_t *)ksrc, (const uint16_t *)vsrc);
  else
    hipLaunchKernelGGL(k_kv_fill<uint32_t>, grid, dim3(kv.d_h), 0, st, kv, seq, start,
                       (const uint32_t *)ksrc, (const uint32_t *)vsrc);
  return hipGetLastError();
}

hipError_t launch_mixture(const MixArgs &m, hipStream_t st) {
  // k_mix_select keeps the list of kept tiles (at most 4096) in LDS
  if (m.nstat < 1 || m.nstat > 4096 || m.rows.np < 1 || m.rows.np > 4 || m.tile_w < 1) return hipErrorInvalidValue;
  if (!m.stats_ready) {
    const int nch = (m.V + m.chunk - 1) / m.chunk;
    hipLaunchKernelGGL(k_mix_stats, dim3(nch, m.rows.np * m.rows.B), dim3(256), 0, st, m);
  }
  const dim3 grid(m.rows.B), block(256);
  // float4 units when rows are 16-byte aligned and units stay inside tiles;
  // the primary alone keeps scalar loads (its scan reads about one tile, and
  // the wider loop's code costs more than it saves there)
  const bool v4 = m.rows.np > 1 && m.V % 4 == 0 && m.tile_w % 4 == 0;
  switch (m.rows.np * 2 + (v4 ? 1 : 0)) {
    case 2: hipLaunchKernelGGL((k_mix_select<1, 1>), grid, block, 0, st, m); break;
    case 4: hipLaunchKernelGGL((k_mix_select<2, 1>), grid, block, 0, st, m); break;
    case 5: hipLaunchKernelGGL((k_mix_select<2, 4>), grid, block, 0, st, m); break;
    case 6: hipLaunchKernelGGL((k_mix_select<3, 1>), grid, block, 0, st, m); break;
    case 7: hipLaunchKernelGGL((k_mix_select<3, 4>), grid, block, 0, st, m); break;
    case 8: hipLaunchKernelGGL((k_mix_select<4, 1>), grid, block, 0, st, m); break;
    default: hipLaunchKernelGGL((k_mix_select<4, 4>), grid, block, 0, st, m); break;
  }
  return hipGetLastError();
}

}  // namespace dbt
