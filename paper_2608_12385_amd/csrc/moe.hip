// MoE layer of the decode step (Sec. 3.2, Eqs. (5)-(6); router replay,
// Sec. 4.3 Eq. (19); independent primary/branch fan-outs k1, k2, Sec. 5
// Eq. (22)).
//
// 1. k_moe_route: per sequence, the router logits of its primary and branch
//    rows from the fp32 MLP input (RMSNorm recomputed from S_bar), top-k
//    (logit descending, ties to the lower index) and the renormalised
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
// Experts no row selected are never read.
#include "common.h"
#include "kernels.h"

namespace dbt {

namespace {

__device__ __forceinline__ int prow(const Rows &r, int path, int b) { return path * r.Bp + b; }

// Router: one workgroup per sequence, 256 threads; E <= 256, k <= 8.
__global__ __launch_bounds__(256) void k_moe_route(MoeRoute a) {
  __shared__ float u[2][4096 + 4];
  __shared__ float logits[2][256];
  __shared__ float red[16];
  const int b = blockIdx.x;
  const bool prim = a.mode != MODE_BRANCH, br = a.mode != MODE_PRIMARY;
  const int d = a.d, E = a.E;
  // fp32 MLP inputs of the active rows: RMSNorm(S_bar) * g
  for (int p = 0; p < 2; ++p) {
    if ((p == 0 && !prim) || (p == 1 && !br)) continue;
    const float *s = a.Sbar + (size_t)prow(a.rows, p, b) * d;
    float ss = 0.f;
    for (int i = threadIdx.x; i < d; i += blockDim.x) ss += s[i] * s[i];
    ss = block_sum(ss, red);
    const float inv = 1.0f / sqrtf(ss / (float)d + a.eps);
    for (int i = threadIdx.x; i < d; i += blockDim.x) u[p][i] = s[i] * inv * a.g[i];
  }
  __syncthreads();
  // logits: wave w takes experts w, w+4, ...; lanes stride the model dimension
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  for (int e = wave; e < E; e += 4) {
    const uint16_t *wr = (const uint16_t *)a.Wr + (size_t)e * d;
    float s0 = 0.f, s1 = 0.f;
    for (int i = lane; i < d; i += 64) {
      const float w = bf2f(wr[i]);
      if (prim) s0 = fmaf(u[0][i], w, s0);
      if (br) s1 = fmaf(u[1][i], w, s1);
    }
    s0 = wave_sum(s0);
    s1 = wave_sum(s1);
    if (lane == 0) {
      logits[0][e] = s0;
      logits[1][e] = s1;
    }
  }
  __syncthreads();
  if (threadIdx.x >= 64) return;
  // top-k per path by repeated wave argmax over the E logits (lane holds e = lane + 64j)
  int sel0[8];
  for (int p = 0; p < 2; ++p) {
    if ((p == 0 && !prim) || (p == 1 && !br)) continue;
    const int k = p == 0 ? a.k1 : a.k2;
    int sel[8];
    float val[8];
    const bool replay = p == 1 && a.replay;
    if (replay) {
      // the branch reuses the primary's experts (wave-uniform values)
      for (int j = 0; j < k; ++j) sel[j] = prim ? sel0[j] : a.idx1_in[(size_t)b * 8 + j];
      for (int j = 0; j < k; ++j) val[j] = logits[p][sel[j]];
    } else {
      float v[4];
      for (int j = 0; j < 4; ++j) {
        const int e = lane + 64 * j;
        v[j] = e < E ? logits[p][e] : -INFINITY;
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
    // weights: softmax over the full router gathered at the selection and
    // renormalised = exp(r_e - max_sel) / sum over the selection
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

// One workgroup: thread e lists expert e's assignments in (path, b, slot) order.
__global__ void k_moe_dispatch(MoeDispatch a) {
  const int e = threadIdx.x;
  __shared__ int cnt[257];
  const int np = a.rows.np, B = a.rows.B;
  int c = 0;
  if (e < a.E) {
    for (int pp = 0; pp < np; ++pp) {
      const int p = a.rows.p0 + pp;
      const int k = p == 0 ? a.k1 : a.k2;
      for (int b = 0; b < B; ++b)
        for (int j = 0; j < k; ++j)
          if (a.idx[(size_t)prow(a.rows, p, b) * 8 + j] == e) ++c;
    }
    cnt[e] = c;
  }
  __syncthreads();
  if (e == 0) {
    int acc = 0;
    for (int i = 0; i < a.E; ++i) {
      a.offsets[i] = acc;
      acc += cnt[i];
      a.counts[i] = cnt[i];
    }
    a.offsets[a.E] = acc;
    cnt[256] = acc;
  }
  __syncthreads();
  if (e < a.E) {
    int pos = a.offsets[e];
    for (int pp = 0; pp < np; ++pp) {
      const int p = a.rows.p0 + pp;
      const int k = p == 0 ? a.k1 : a.k2;
      for (int b = 0; b < B; ++b)
        for (int j = 0; j < k; ++j) {
          const size_t r = (size_t)prow(a.rows, p, b);
          if (a.idx[r * 8 + j] == e) {
            a.arow[pos] = (int)r;
            a.aslot[r * 8 + j] = pos;
            ++pos;
          }
        }
    }
  }
}

constexpr int kChunk = 128;
constexpr int kLdsRow = kChunk + 8;

// Expert projections over gathered rows.  GATEUP: workgroup = (expert,
// 64 hidden units); wave w owns hidden units h0+16w..+15 with row block 0 =
// gate rows and row block 1 = up rows, so SwiGLU is lane-local.  DOWN:
// workgroup = (expert, 64 output columns), wave w owns 16 of them.
template <int MB, bool GATEUP>
__global__ __launch_bounds__(256) void k_moe_gemm(MoeGemm a) {
  constexpr int RB = GATEUP ? 2 : 1;
  constexpr int PD = 2;
  constexpr int XR = 16 * MB;
  constexpr int PIECES = XR * (kChunk / 8);
  constexpr int PPT = (PIECES + 255) / 256;
  __shared__ uint16_t xs[PD][XR * kLdsRow];
  __shared__ int rows_s[XR];
  const int tiles = a.N / 64;
  const int e = blockIdx.x / tiles, tile = blockIdx.x % tiles;
  const int Me = a.counts[e];
  const int m0 = blockIdx.z * XR;
  if (m0 >= Me) return;  // untouched expert (or beyond its rows): no weight read
  const int base = a.offsets[e];
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6, r = lane & 15, gq = lane >> 4;
  const int K = a.K, nch = K / kChunk;
  if (t < XR) rows_s[t] = (m0 + t < Me) ? (GATEUP ? a.arow[base + m0 + t] : base + m0 + t) : -1;
  const int nb = (min(Me - m0, XR) + 15) / 16;  // live activation blocks
  const int n0 = tile * 64 + wave * 16;
  const uint16_t *wrow[RB];
  if (GATEUP) {
    wrow[0] = (const uint16_t *)a.W0 + ((size_t)e * a.N + n0 + r) * K + gq * 8;
    wrow[RB - 1] = (const uint16_t *)a.W1 + ((size_t)e * a.N + n0 + r) * K + gq * 8;
  } else {
    wrow[0] = (const uint16_t *)a.W0 + ((size_t)e * a.N + n0 + r) * K + gq * 8;
  }
  __syncthreads();
  floatx4 acc[RB][MB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int cb = 0; cb < MB; ++cb) acc[rb][cb] = floatx4{0.f, 0.f, 0.f, 0.f};
  u32x4 w[PD][RB][4];
  u32x4 stage[PPT];
  auto wload = [&](int slot, int c) {
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int s = 0; s < 4; ++s) w[slot][rb][s] = *(const u32x4 *)(wrow[rb] + c * kChunk + s * 32);
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
        for (int s = 0; s < 4; ++s) {
#pragma unroll
          for (int cb = 0; cb < MB; ++cb) {
            if (cb < nb) {
              const u32x4 bx = *(const u32x4 *)(&xs[u][(cb * 16 + r) * kLdsRow + s * 32 + gq * 8]);
#pragma unroll
              for (int rb = 0; rb < RB; ++rb)
                acc[rb][cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                    __builtin_bit_cast(bf16x8, w[u][rb][s]), __builtin_bit_cast(bf16x8, bx), acc[rb][cb], 0, 0, 0);
            }
          }
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

// Routed sum (ascending expert id) + shared expert + c coupling + residual +
// next norm.  One workgroup per sequence (both paths).
template <typename T>
__global__ void k_moe_combine(MoeCombine a) {
  __shared__ float red[16];
  const int b = blockIdx.x;
  const bool prim = a.mode != MODE_BRANCH, br = a.mode != MODE_PRIMARY;
  const int d = a.d;
  const int r1 = prow(a.rows, 0, b), r2 = prow(a.rows, 1, b);
  // selected experts of each path in ascending id order (insertion sort, k <= 8)
  int ord[2][8];
  for (int p = 0; p < 2; ++p) {
    const int k = p == 0 ? a.k1 : a.k2;
    const int r = p == 0 ? r1 : r2;
    if ((p == 0 && !prim) || (p == 1 && !br)) continue;
    for (int j = 0; j < k; ++j) ord[p][j] = j;
    for (int j = 1; j < k; ++j)
      for (int q = j; q > 0 && a.idx[(size_t)r * 8 + ord[p][q]] < a.idx[(size_t)r * 8 + ord[p][q - 1]]; --q) {
        const int tmp = ord[p][q];
        ord[p][q] = ord[p][q - 1];
        ord[p][q - 1] = tmp;
      }
  }
  float *s1 = a.S + (size_t)r1 * d;
  float *s2 = a.S + (size_t)r2 * d;
  const bool keep = a.ret.ptr && (a.ret.src_row < 0 || a.ret.src_row == b);
  float *kept = keep ? a.ret.ptr + (size_t)(a.ret.src_row < 0 ? b : a.ret.dst_row) * d : nullptr;
  for (int i = threadIdx.x; i < d; i += blockDim.x) {
    float m1 = 0.f;
    if (prim) {
      float rsum = 0.f;
      for (int j = 0; j < a.k1; ++j) {
        const int q = ord[0][j];
        rsum += a.wts[(size_t)r1 * 8 + q] * a.Yexp[(size_t)a.aslot[(size_t)r1 * 8 + q] * d + i];
      }
      float sh = 0.f;
      for (int k = 0; k < a.S_sh; ++k) sh += a.part[k * a.stride + (size_t)r1 * d + i];
      m1 = rsum + sh;
      s1[i] += m1;
      if (keep) kept[i] = m1;
    } else {
      m1 = a.M1_in[(size_t)b * d + i];
    }
    if (br) {
      float rsum = 0.f;
      for (int j = 0; j < a.k2; ++j) {
        const int q = ord[1][j];
        rsum += a.wts[(size_t)r2 * 8 + q] * a.Yexp[(size_t)a.aslot[(size_t)r2 * 8 + q] * d + i];
      }
      float sh = 0.f;
      for (int k = 0; k < a.S_sh; ++k) sh += a.part[k * a.stride + (size_t)r2 * d + i];
      s2[i] += (rsum + sh) + a.c[i] * m1;
    }
  }
  if (!a.g_next) return;
  __syncthreads();
  for (int p = 0; p < 2; ++p) {
    if ((p == 0 && !prim) || (p == 1 && !br)) continue;
    const float *x = p == 0 ? s1 : s2;
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
  dim3 grid(a.E * (a.N / 64), 1, a.mtiles);
  switch (MB) {
    case 1: hipLaunchKernelGGL((k_moe_gemm<1, GATEUP>), grid, dim3(256), 0, st, a); break;
    case 2: hipLaunchKernelGGL((k_moe_gemm<2, GATEUP>), grid, dim3(256), 0, st, a); break;
    case 4: hipLaunchKernelGGL((k_moe_gemm<4, GATEUP>), grid, dim3(256), 0, st, a); break;
    default: hipLaunchKernelGGL((k_moe_gemm<8, GATEUP>), grid, dim3(256), 0, st, a); break;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_moe_route(const MoeRoute &a, hipStream_t st) {
  hipLaunchKernelGGL(k_moe_route, dim3(a.rows.B), dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_moe_dispatch(const MoeDispatch &a, hipStream_t st) {
  hipLaunchKernelGGL(k_moe_dispatch, dim3(1), dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_moe_gemm(const MoeGemm &a, bool gateup, int max_rows, hipStream_t st) {
  const int mb = (max_rows + 15) / 16;
  const int MB = mb >= 8 ? 8 : mb > 2 ? 4 : mb;
  MoeGemm b = a;
  b.mtiles = (max_rows + 16 * MB - 1) / (16 * MB);
  return gateup ? launch_moe_gemm_t<true>(b, MB, st) : launch_moe_gemm_t<false>(b, MB, st);
}

hipError_t launch_moe_combine(const MoeCombine &a, int dtype, hipStream_t st) {
  if (dtype == 1)
    hipLaunchKernelGGL(k_moe_combine<uint16_t>, dim3(a.rows.B), dim3(256), 0, st, a);
  else
    hipLaunchKernelGGL(k_moe_combine<float>, dim3(a.rows.B), dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace dbt
