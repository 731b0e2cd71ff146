// MoE layer of the decode step (Sec. 3.2, Eqs. (5)-(6); router replay,
// Sec. 4.3 Eq. (19); independent primary/branch fan-outs k1, k2, Sec. 5
// Eq. (22)).
//
// 1. k_moe_logits + k_moe_topk: the router logits of each sequence's primary
//    and branch rows from the fp32 MLP input (RMSNorm recomputed from S_bar),
//    top-k (logit descending, ties to the lower index) and the renormalised
//    softmax weights of the selected experts.
// 2. k_moe_dispatch: per expert, the list of (path, sequence, slot)
//    assignments in (path, sequence, slot) order; each assignment's
//    position in the expert-grouped order.
// 3. k_moe_gemm<GATEUP>: for each touched expert, its gate/up rows against
//    the gathered activation rows of all its assignments from both paths
//    (each expert weight tile is read once for the primary and branch rows
//    that selected it), SwiGLU in the epilogue.
// 4. k_moe_gemm<DOWN>: the expert down projections of the same rows.
// 5. k_moe_combine: M_i = sum over selected experts (ascending id) of
//    w_e * Expert_e(U_i) + shared expert; M2 += c * M1; S += M; next norm.
//    Compute-matched variant (App. B.3): the shared expert runs on the
//    primary rows only and M2 = R2 + g_G * G1.
// Experts no row selected are never read.
#include "common.h"
#include "kernels.h"

namespace dbt {

namespace {

__device__ __forceinline__ int prow(const Rows &r, int path, int b) { return path * r.Bp + b; }

// Router logits: workgroup = (sequence, 16 experts).  The fp32 MLP inputs
// RMSNorm(S_bar) * g of the active rows are rebuilt in LDS; wave w computes
// experts 4w..4w+3 of the group for both rows, lanes covering the model
// dimension 8 elements at a time (NIT = d / 512 pieces per lane).  Every
// load (the rows, the gain, the wave's four router rows) is issued at the
// start, so the kernel waits for memory once.
template <int NIT>
__global__ __launch_bounds__(256) void k_moe_logits(MoeRoute a) {
  __shared__ float u[2][4096 + 4];
  __shared__ float red[16];
  const int b = blockIdx.x, e0 = blockIdx.y * 16;
  const bool prim = a.mode != MODE_BRANCH, br = a.mode != MODE_PRIMARY;
  const int E = a.E;
  constexpr int d = NIT * 512, NV = (d / 4 + 255) / 256;  // float4 per thread and row
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  u32x4 wv[4][NIT];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int e = min(e0 + wave * 4 + q, E - 1);
    const uint16_t *wr = (const uint16_t *)a.Wr + (size_t)e * d;
#pragma unroll
    for (int it = 0; it < NIT; ++it) wv[q][it] = *(const u32x4 *)(wr + (it * 64 + lane) * 8);
  }
  float4 sv[2][NV], gv[NV];
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    const int i = min((int)threadIdx.x + k * 256, d / 4 - 1);
    gv[k] = ((const float4 *)a.g)[i];
#pragma unroll
    for (int p = 0; p < 2; ++p) sv[p][k] = ((const float4 *)(a.Sbar + (size_t)prow(a.rows, p, b) * d))[i];
  }
  for (int p = 0; p < 2; ++p) {
    if ((p == 0 && !prim) || (p == 1 && !br)) continue;
    float ss = 0.f;
#pragma unroll
    for (int k = 0; k < NV; ++k)
      if ((int)threadIdx.x + k * 256 < d / 4) {
        const float4 v = sv[p][k];
        ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
      }
    ss = block_sum(ss, red);
    const float inv = 1.0f / sqrtf(ss / (float)d + a.eps);
#pragma unroll
    for (int k = 0; k < NV; ++k) {
      const int i = threadIdx.x + k * 256;
      if (i < d / 4) {
        const float4 v = sv[p][k], g = gv[k];
        u[p][4 * i + 0] = v.x * inv * g.x;
        u[p][4 * i + 1] = v.y * inv * g.y;
        u[p][4 * i + 2] = v.z * inv * g.z;
        u[p][4 * i + 3] = v.w * inv * g.w;
      }
    }
  }
  __syncthreads();
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int e = e0 + wave * 4 + q;
    if (e >= E) break;
    float s0 = 0.f, s1 = 0.f;
#pragma unroll
    for (int it = 0; it < NIT; ++it) {
      const int base = (it * 64 + lane) * 8;
#pragma unroll
      for (int h = 0; h < 4; ++h) {
        const float w0 = __uint_as_float(wv[q][it][h] << 16), w1 = __uint_as_float(wv[q][it][h] & 0xffff0000u);
        if (prim) s0 = fmaf(u[0][base + 2 * h + 1], w1, fmaf(u[0][base + 2 * h], w0, s0));
        if (br) s1 = fmaf(u[1][base + 2 * h + 1], w1, fmaf(u[1][base + 2 * h], w0, s1));
      }
    }
    s0 = wave_sum(s0);
    s1 = wave_sum(s1);
    if (lane == 0) {
      if (prim) a.logits[(size_t)prow(a.rows, 0, b) * 256 + e] = s0;
      if (br) a.logits[(size_t)prow(a.rows, 1, b) * 256 + e] = s1;
      if (prim && a.out_lg1) a.out_lg1[(size_t)b * E + e] = s0;
      if (br && a.out_lg2) a.out_lg2[(size_t)b * E + e] = s1;
    }
  }
}

// Top-k per path (logit descending, ties to the lower index) by repeated wave
// argmax, and the renormalised softmax weights.  One wave per sequence.
__global__ __launch_bounds__(64) void k_moe_topk(MoeRoute a) {
  const int b = blockIdx.x, lane = threadIdx.x;
  const bool prim = a.mode != MODE_BRANCH, br = a.mode != MODE_PRIMARY;
  const int E = a.E;
  int sel0[8];
  for (int p = 0; p < 2; ++p) {
    if ((p == 0 && !prim) || (p == 1 && !br)) continue;
    const int k = p == 0 ? a.k1 : a.k2;
    const float *lg = a.logits + (size_t)prow(a.rows, p, b) * 256;
    int sel[8];
    float val[8];
    if (p == 1 && a.replay) {
      // the branch reuses the primary's experts (wave-uniform values)
      for (int j = 0; j < k; ++j) sel[j] = prim ? sel0[j] : a.idx1_in[(size_t)b * 8 + j];
      for (int j = 0; j < k; ++j) val[j] = lg[sel[j]];
    } else {
      float v[4];
      for (int q = 0; q < 4; ++q) {
        const int e = lane + 64 * q;
        v[q] = e < E ? lg[e] : -INFINITY;
      }
      for (int j = 0; j < k; ++j) {
        float best = -INFINITY;
        int bi = 0x7fffffff;
        for (int q = 0; q < 4; ++q) {
          const int e = lane + 64 * q;
          if (e < E && (v[q] > best || (v[q] == best && e < bi))) { best = v[q]; bi = e; }
        }
        for (int o = 32; o > 0; o >>= 1) {
          const float b2 = __shfl_xor(best, o, 64);
          const int i2 = __shfl_xor(bi, o, 64);
          if (b2 > best || (b2 == best && i2 < bi)) { best = b2; bi = i2; }
        }
        sel[j] = bi;
        val[j] = best;
        for (int q = 0; q < 4; ++q)
          if (lane + 64 * q == bi) v[q] = -INFINITY;
      }
    }
    if (p == 0)
      for (int j = 0; j < k; ++j) sel0[j] = sel[j];
    // softmax over all experts gathered at the selection and renormalised
    // = exp(r_e - max_sel) / sum over the selection
    float mx = -INFINITY;
    for (int j = 0; j < k; ++j) mx = fmaxf(mx, val[j]);
    float den = 0.f;
    float w[8];
    for (int j = 0; j < k; ++j) {
      w[j] = expf(val[j] - mx);
      den += w[j];
    }
    if (lane == 0) {
      const size_t r = (size_t)prow(a.rows, p, b);
      for (int j = 0; j < k; ++j) {
        a.idx[r * 8 + j] = sel[j];
        a.wts[r * 8 + j] = w[j] / den;
      }
      int *oi = p == 0 ? a.out_idx1 : a.out_idx2;
      float *ow = p == 0 ? a.out_w1 : a.out_w2;
      if (oi) for (int j = 0; j < k; ++j) oi[(size_t)b * k + j] = sel[j];
      if (ow) for (int j = 0; j < k; ++j) ow[(size_t)b * k + j] = w[j] / den;
      if (p == 0 && a.ret_idx && (a.ret_src < 0 || a.ret_src == b))
        for (int j = 0; j < k; ++j) a.ret_idx[(size_t)(a.ret_src < 0 ? b : a.ret_dst) * 8 + j] = sel[j];
    }
  }
}

// Expert-grouped order as a stable counting sort of the assignments
// (path, b, slot) by expert.  A row selects an expert at most once, so the
// assignments of expert e, in order, are the active rows that selected e, in
// row order.  Thread (e, c) owns expert e and the c-th of RC equal ranges of
// the active rows (1024 threads = RC x E rounded up to a power of two): it
// counts its range's selections of e, the counts are prefix-summed per
// expert over the ranges and across experts (one wave scan), and the thread
// then writes its range's positions.  Fixed order, no atomics.
__global__ __launch_bounds__(1024) void k_moe_dispatch(MoeDispatch a) {
  __shared__ int cnt[1024];
  __shared__ int eoff[256];
  const int t = threadIdx.x, lane = t & 63;
  const int E = a.E;
  const int epad = E <= 1 ? 1 : 1 << (32 - __clz(E - 1));
  const int RC = 1024 / epad;
  const int e = t % epad, c = t / epad;
  const int B = a.rows.B, R = a.rows.np * B;
  const int r0 = c * R / RC, r1 = (c + 1) * R / RC;
  // slot j of active row q, or -1 past the path's k (all eight slots of a
  // row in two 16-byte loads, so a range's loads are in flight together)
  auto sel = [&](int q, int (&v)[8]) {
    const int path = a.rows.p0 + q / B;
    const int k = path == 0 ? a.k1 : a.k2;
    const int4 *p = (const int4 *)(a.idx + (size_t)prow(a.rows, path, q % B) * 8);
    const int4 x = p[0], y = p[1];
    v[0] = x.x; v[1] = x.y; v[2] = x.z; v[3] = x.w; v[4] = y.x; v[5] = y.y; v[6] = y.z; v[7] = y.w;
#pragma unroll
    for (int j = 0; j < 8; ++j)
      if (j >= k) v[j] = -1;
    return prow(a.rows, path, q % B);
  };
  int n = 0;
  if (e < E)
    for (int q = r0; q < r1; ++q) {
      int v[8];
      sel(q, v);
#pragma unroll
      for (int j = 0; j < 8; ++j) n += v[j] == e;
    }
  cnt[t] = n;
  __syncthreads();
  if (t < E) {
    int acc = 0;
    for (int cc = 0; cc < RC; ++cc) {
      const int v = cnt[cc * epad + t];
      cnt[cc * epad + t] = acc;
      acc += v;
    }
    a.counts[t] = acc;
    eoff[t] = acc;
  }
  __syncthreads();
  if (t < 64) {
    // exclusive scan over experts: lane l sums experts 4l..4l+3
    int v[4], s = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int ee = 4 * lane + i;
      v[i] = ee < E ? eoff[ee] : 0;
      s += v[i];
    }
    int incl = s;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int u = __shfl_up(incl, o, 64);
      if (lane >= o) incl += u;
    }
    int off = incl - s;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int ee = 4 * lane + i;
      if (ee < E) {
        eoff[ee] = off;
        a.offsets[ee] = off;
      }
      off += v[i];
    }
    if (lane == 63) a.offsets[E] = incl;
  }
  __syncthreads();
  if (e < E) {
    int pos = eoff[e] + cnt[t];
    for (int q = r0; q < r1; ++q) {
      int v[8];
      const int row = sel(q, v);
#pragma unroll
      for (int j = 0; j < 8; ++j)
        if (v[j] == e) {
          a.arow[pos] = row;
          a.aslot[(size_t)row * 8 + j] = pos;
          ++pos;
        }
    }
  }
}

constexpr int kChunk = 128;
constexpr int kLdsRow = kChunk + 8;

// Expert projections over gathered rows.  GATEUP: workgroup = (expert,
// 64 hidden units); wave w owns hidden units h0+16w..+15 with row block 0 =
// gate rows and row block 1 = up rows, so SwiGLU is lane-local.  DOWN:
// workgroup = (expert, 64 output columns), wave w owns 16 of them.  The
// workgroup takes all rows of its expert in passes of 16*MB (one pass unless
// the expert is crowded; a further pass reads its weights again); an
// untouched expert's workgroups return before any weight read.
//
// Weight loads as in the dense projections: whole 128-byte row pieces with
// the non-temporal hint (eight rows per wave instruction), moved into the
// MFMA operand layout through the wave's LDS region half a chunk at a time.
template <int MB, bool GATEUP>
__global__ __launch_bounds__(256) void k_moe_gemm(MoeGemm a) {
  constexpr int RB = GATEUP ? 2 : 1;
  constexpr int PD = 2;
  constexpr int XR = 16 * MB;
  constexpr int PIECES = XR * (kChunk / 8);
  constexpr int PPT = (PIECES + 255) / 256;
  __shared__ uint16_t xs[PD][XR * kLdsRow];
  __shared__ int rows_s[XR];
  __shared__ u32x4 wt[4][RB * 16 * 8];
  const int tiles = a.N / 64;
  const int e = blockIdx.x / tiles, tile = blockIdx.x % tiles;
  const int Me = a.counts[e];
  if (Me <= 0) return;  // untouched expert: no weight read
  const int base = a.offsets[e];
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6, r = lane & 15, gq = lane >> 4;
  const int K = a.K, nch = K / kChunk;
  const int n0 = tile * 64 + wave * 16;
  // coalesced weight loads: row block rb, row group j (rows j*8 + lane/8 of
  // the block), 16-byte piece lane%8 of a 128-byte half chunk
  const int lr8 = lane >> 3, lp8 = lane & 7;
  const uint16_t *wrow[RB][2];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int j = 0; j < 2; ++j)
      wrow[rb][j] = (const uint16_t *)(rb == 0 ? a.W0 : a.W1) + ((size_t)e * a.N + n0 + j * 8 + lr8) * K + lp8 * 8;
  u32x4 *wreg = wt[wave];
  u32x4 w[PD][RB][4];
  u32x4 stage[PPT];
  auto wload = [&](int slot, int c) {
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          w[slot][rb][2 * h + j] = __builtin_nontemporal_load((const u32x4 *)(wrow[rb][j] + c * kChunk + h * 64));
  };
  auto xload = [&](int c) {
#pragma unroll
    for (int j = 0; j < PPT; ++j) {
      const int p = t + 256 * j;
      const int row = p >> 4, col = (p & 15) * 8;
      const int src = p < PIECES ? rows_s[row] : -1;
      stage[j] = src >= 0 ? *(const u32x4 *)((const uint16_t *)a.X + (size_t)src * a.ldx + c * kChunk + col)
                          : u32x4{0u, 0u, 0u, 0u};
    }
  };
  auto xstore = [&](int slot) {
#pragma unroll
    for (int j = 0; j < PPT; ++j) {
      const int p = t + 256 * j;
      if (p < PIECES) *(u32x4 *)(&xs[slot][(p >> 4) * kLdsRow + (p & 15) * 8]) = stage[j];
    }
  };
  for (int m0 = 0; m0 < Me; m0 += XR) {
    if (m0 > 0) __syncthreads();  // the previous pass is done with rows_s and xs
    if (t < XR) rows_s[t] = (m0 + t < Me) ? (GATEUP ? a.arow[base + m0 + t] : base + m0 + t) : -1;
    const int nb = (min(Me - m0, XR) + 15) / 16;  // live activation blocks
    __syncthreads();
    floatx4 acc[RB][MB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int cb = 0; cb < MB; ++cb) acc[rb][cb] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int u = 0; u < PD; ++u)
      if (u < nch) {
        xload(u);
        xstore(u);
        wload(u, u);
      }
    __syncthreads();
    for (int c0 = 0; c0 < nch; c0 += PD) {
#pragma unroll
      for (int u = 0; u < PD; ++u) {
        const int c = c0 + u;
        if (c < nch) {
          const bool more = c + PD < nch;
          if (more) xload(c + PD);
#pragma unroll
          for (int h = 0; h < 2; ++h) {
#pragma unroll
            for (int rb = 0; rb < RB; ++rb)
#pragma unroll
              for (int j = 0; j < 2; ++j) wreg[(rb * 16 + j * 8 + lr8) * 8 + (lp8 ^ lr8)] = w[u][rb][2 * h + j];
            wave_lds_fence();
#pragma unroll
            for (int s2 = 0; s2 < 2; ++s2) {
              const int s = 2 * h + s2;
              u32x4 wf[RB];
#pragma unroll
              for (int rb = 0; rb < RB; ++rb) wf[rb] = wreg[(rb * 16 + r) * 8 + ((4 * s2 + gq) ^ (r & 7))];
#pragma unroll
              for (int cb = 0; cb < MB; ++cb) {
                if (cb < nb) {
                  const u32x4 bx = *(const u32x4 *)(&xs[u][(cb * 16 + r) * kLdsRow + s * 32 + gq * 8]);
#pragma unroll
                  for (int rb = 0; rb < RB; ++rb)
                    acc[rb][cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                        __builtin_bit_cast(bf16x8, wf[rb]), __builtin_bit_cast(bf16x8, bx), acc[rb][cb], 0, 0, 0);
                }
              }
            }
            wave_lds_fence();
          }
          if (more) wload(u, c + PD);
          __syncthreads();
          if (more) xstore(u);
        }
      }
    }
    // lane holds D[n = n0 + 4gq + i][m = m0 + cb*16 + r]
#pragma unroll
    for (int cb = 0; cb < MB; ++cb) {
      const int m = m0 + cb * 16 + r;
      if (cb >= nb || m >= Me) continue;
      const size_t orow = (size_t)(base + m);
      if (GATEUP) {
        uint16_t h[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float g = acc[0][cb][i], up = acc[RB - 1][cb][i];
          h[i] = f2bf(g / (1.0f + expf(-g)) * up);
        }
        uint2 v;
        v.x = (uint32_t)h[0] | ((uint32_t)h[1] << 16);
        v.y = (uint32_t)h[2] | ((uint32_t)h[3] << 16);
        *(uint2 *)((uint16_t *)a.Y + orow * a.ldy + n0 + gq * 4) = v;
      } else {
        *(floatx4 *)((float *)a.Y + orow * a.ldy + n0 + gq * 4) = acc[0][cb];
      }
    }
  }
}

// Routed sum (ascending expert id) + shared expert + c coupling + residual +
// next norm.  One workgroup per sequence (both paths), float4 columns.
template <typename T>
__global__ void k_moe_combine(MoeCombine a) {
  __shared__ float red[16];
  __shared__ int sl[2][8];
  __shared__ float sw[2][8];
  const int b = blockIdx.x;
  const bool prim = a.mode != MODE_BRANCH, br = a.mode != MODE_PRIMARY;
  const int d = a.d, d4 = d / 4;
  const int r1 = prow(a.rows, 0, b), r2 = prow(a.rows, 1, b);
  if (threadIdx.x < 2) {
    // selected experts of this path in ascending id order (insertion sort, k <= 8)
    const int p = threadIdx.x;
    const int k = p == 0 ? a.k1 : a.k2;
    const int r = p == 0 ? r1 : r2;
    if ((p == 0 && prim) || (p == 1 && br)) {
      // all eight slots of the row loaded at once (the arrays hold 8 per row),
      // then an odd-even transposition sort in registers; slots >= k sort last
      int id[8], sj[8];
      float wj[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int v = a.idx[(size_t)r * 8 + j];
        id[j] = j < k ? v : 0x7fffffff;
        sj[j] = a.aslot[(size_t)r * 8 + j];
        wj[j] = a.wts[(size_t)r * 8 + j];
      }
#pragma unroll
      for (int round = 0; round < 8; ++round)
#pragma unroll
        for (int j = round & 1; j + 1 < 8; j += 2)
          if (id[j + 1] < id[j]) {
            const int ti = id[j], ts = sj[j];
            const float tw = wj[j];
            id[j] = id[j + 1];
            sj[j] = sj[j + 1];
            wj[j] = wj[j + 1];
            id[j + 1] = ti;
            sj[j + 1] = ts;
            wj[j + 1] = tw;
          }
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        sl[p][j] = j < k ? sj[j] : sj[0];  // padding: a valid row with weight 0
        sw[p][j] = j < k ? wj[j] : 0.f;
      }
    }
  }
  __syncthreads();
  float4 *s1 = (float4 *)(a.S + (size_t)r1 * d);
  float4 *s2 = (float4 *)(a.S + (size_t)r2 * d);
  const bool keep = a.ret.ptr && (a.ret.src_row < 0 || a.ret.src_row == b);
  float4 *kept = keep ? (float4 *)(a.ret.ptr + (size_t)(a.ret.src_row < 0 ? b : a.ret.dst_row) * d) : nullptr;
  // routed experts, ascending id; all eight slots (weight 0 past k: adding
  // zeros leaves the sum unchanged) so the loads are in flight together
  auto experts = [&](int p, int k, int i) {
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const float4 y = ((const float4 *)(a.Yexp + (size_t)sl[p][j] * d))[i];
      const float w = sw[p][j];
      acc.x += w * y.x;
      acc.y += w * y.y;
      acc.z += w * y.z;
      acc.w += w * y.w;
    }
    return acc;
  };
  auto shared = [&](int row, int i) {  // shared-expert slabs in split order
    float4 sh = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll 4
    for (int q = 0; q < a.S_sh; ++q) {
      const float4 v = ((const float4 *)(a.part + q * a.stride + (size_t)row * d))[i];
      sh.x += v.x;
      sh.y += v.y;
      sh.z += v.z;
      sh.w += v.w;
    }
    return sh;
  };
  const bool cm = a.gG != nullptr;  // compute-matched variant (App. B.3)
  for (int i = threadIdx.x; i < d4; i += blockDim.x) {
    float4 m1, g1;  // primary MoE output; primary shared-expert output
    if (prim) {
      const float4 r = experts(0, a.k1, i);
      g1 = shared(r1, i);
      m1 = make_float4(r.x + g1.x, r.y + g1.y, r.z + g1.z, r.w + g1.w);
      const float4 s = s1[i];
      s1[i] = make_float4(s.x + m1.x, s.y + m1.y, s.z + m1.z, s.w + m1.w);
      if (keep) kept[i] = cm ? g1 : m1;
    } else {
      m1 = g1 = ((const float4 *)(a.M1_in + (size_t)b * d))[i];
    }
    if (br) {
      const float4 r = experts(1, a.k2, i);
      const float4 s = s2[i];
      if (cm) {  // M2 = R2 + g_G * G1
        const float4 gg = ((const float4 *)a.gG)[i];
        s2[i] = make_float4(s.x + (r.x + gg.x * g1.x), s.y + (r.y + gg.y * g1.y), s.z + (r.z + gg.z * g1.z),
                            s.w + (r.w + gg.w * g1.w));
      } else {   // M2 = R2 + shared expert of the branch + c * M1
        const float4 g2 = shared(r2, i);
        const float4 c = ((const float4 *)a.c)[i];
        s2[i] = make_float4(s.x + ((r.x + g2.x) + c.x * m1.x), s.y + ((r.y + g2.y) + c.y * m1.y),
                            s.z + ((r.z + g2.z) + c.z * m1.z), s.w + ((r.w + g2.w) + c.w * m1.w));
      }
    }
  }
  if (!a.g_next) return;
  __syncthreads();
  for (int p = 0; p < 2; ++p) {
    if ((p == 0 && !prim) || (p == 1 && !br)) continue;
    const float *x = (const float *)(p == 0 ? s1 : s2);
    T *out = (T *)a.Xn + (size_t)(p == 0 ? r1 : r2) * a.ldx;
    float ss = 0.f;
    for (int i = threadIdx.x; i < d; i += blockDim.x) ss += x[i] * x[i];
    ss = block_sum(ss, red);
    const float inv = 1.0f / sqrtf(ss / (float)d + a.eps);
    for (int i = threadIdx.x; i < d; i += blockDim.x) st<T>(out, i, x[i] * inv * a.g_next[i]);
    __syncthreads();
  }
}

template <bool GATEUP>
hipError_t launch_moe_gemm_t(const MoeGemm &a, int MB, hipStream_t st) {
  dim3 grid(a.E * (a.N / 64), 1, 1);
  switch (MB) {
    case 1: hipLaunchKernelGGL((k_moe_gemm<1, GATEUP>), grid, dim3(256), 0, st, a); break;
    default: hipLaunchKernelGGL((k_moe_gemm<2, GATEUP>), grid, dim3(256), 0, st, a); break;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_moe_route(const MoeRoute &a, hipStream_t st) {
  if (a.E < 1 || a.E > 256 || a.d % 512 != 0 || a.d > 4096) return hipErrorInvalidValue;
  const dim3 grid(a.rows.B, (a.E + 15) / 16);
  switch (a.d / 512) {
    case 1: hipLaunchKernelGGL(k_moe_logits<1>, grid, dim3(256), 0, st, a); break;
    case 2: hipLaunchKernelGGL(k_moe_logits<2>, grid, dim3(256), 0, st, a); break;
    case 3: hipLaunchKernelGGL(k_moe_logits<3>, grid, dim3(256), 0, st, a); break;
    case 4: hipLaunchKernelGGL(k_moe_logits<4>, grid, dim3(256), 0, st, a); break;
    case 5: hipLaunchKernelGGL(k_moe_logits<5>, grid, dim3(256), 0, st, a); break;
    case 6: hipLaunchKernelGGL(k_moe_logits<6>, grid, dim3(256), 0, st, a); break;
    case 7: hipLaunchKernelGGL(k_moe_logits<7>, grid, dim3(256), 0, st, a); break;
    default: hipLaunchKernelGGL(k_moe_logits<8>, grid, dim3(256), 0, st, a); break;
  }
  hipLaunchKernelGGL(k_moe_topk, dim3(a.rows.B), dim3(64), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_moe_dispatch(const MoeDispatch &a, hipStream_t st) {
  if (a.E < 1 || a.E > 256) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_moe_dispatch, dim3(1), dim3(1024), 0, st, a);
  return hipGetLastError();
}

// 32-row activation passes: an expert usually gets a handful of rows; the
// rare crowded expert takes more passes (its weights are then read again).
hipError_t launch_moe_gemm(const MoeGemm &a, bool gateup, int max_rows, hipStream_t st) {
  const int MB = max_rows > 16 ? 2 : 1;
  return gateup ? launch_moe_gemm_t<true>(a, MB, st) : launch_moe_gemm_t<false>(a, MB, st);
}

hipError_t launch_moe_combine(const MoeCombine &a, int dtype, hipStream_t st) {
  if (dtype == 1)
    hipLaunchKernelGGL(k_moe_combine<uint16_t>, dim3(a.rows.B), dim3(256), 0, st, a);
  else
    hipLaunchKernelGGL(k_moe_combine<float>, dim3(a.rows.B), dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace dbt
