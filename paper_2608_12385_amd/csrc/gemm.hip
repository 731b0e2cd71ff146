// Stacked-row projections Y = X W^T for the decode step (Sec. 4.4 "Decode":
// the two paths' residual rows are stacked so each weight tile is read once
// for both; Sec. 4.5, Eq. (20): the step is bound by weight + KV traffic).
//
// bf16 weights: MFMA v_mfma_f32_16x16x32_bf16.  A workgroup owns 64 weight
// rows and up to 128 activation rows; its four waves split the reduction
// dimension in 128-wide chunks and are summed through LDS in a fixed order.
// Optional split of the reduction across workgroups (grid.y) writes one fp32
// slab per split; the consumer kernel adds the slabs in split order.  The
// per-element arithmetic never depends on how many rows are stacked, so the
// primary rows come out bit-identical with or without the branch rows.
//
// fp32 weights: an LDS-tiled vector kernel (small models).
#include "common.h"
#include "kernels.h"

namespace dbt {

namespace {

constexpr int kRowsPerWG = 64;   // weight rows per workgroup
constexpr int kChunk = 128;      // reduction elements per wave iteration

__device__ __forceinline__ const uint16_t *seg_base(const WSegs &s, int n0, int &nloc) {
  nloc = n0;
  if (nloc < s.rows[0]) return (const uint16_t *)s.w[0];
  nloc -= s.rows[0];
  if (nloc < s.rows[1]) return (const uint16_t *)s.w[1];
  nloc -= s.rows[1];
  return (const uint16_t *)s.w[2];
}

template <int MB>
__global__ __launch_bounds__(256) void k_gemm_bf16(WSegs segs, int K, const uint16_t *__restrict__ X,
                                                   int ldx, int M, float *__restrict__ Y, int ldy,
                                                   long long y_split_stride, int k_per_split) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r = lane & 15, gq = lane >> 4;
  const int n0 = blockIdx.x * kRowsPerWG;
  const int split = blockIdx.y;
  const int m0 = blockIdx.z * (16 * MB);
  int nloc;
  const uint16_t *W = seg_base(segs, n0, nloc);
  const int kbeg = split * k_per_split;
  const int nchunks = k_per_split / kChunk;

  const uint16_t *wrow[4];
#pragma unroll
  for (int rb = 0; rb < 4; ++rb) wrow[rb] = W + (size_t)(nloc + rb * 16 + r) * K + kbeg + gq * 8;
  const uint16_t *xrow[MB];
  bool xval[MB];
#pragma unroll
  for (int cb = 0; cb < MB; ++cb) {
    const int m = m0 + cb * 16 + r;
    xval[cb] = m < M;
    xrow[cb] = X + (size_t)(xval[cb] ? m : 0) * ldx + kbeg + gq * 8;
  }

  floatx4 acc[4][MB];
#pragma unroll
  for (int rb = 0; rb < 4; ++rb)
#pragma unroll
    for (int cb = 0; cb < MB; ++cb) acc[rb][cb] = floatx4{0.f, 0.f, 0.f, 0.f};

  for (int c = wave; c < nchunks; c += 4) {
    const int koff = c * kChunk;
    u32x4 a[4][4];
#pragma unroll
    for (int rb = 0; rb < 4; ++rb)
#pragma unroll
      for (int s = 0; s < 4; ++s) a[rb][s] = *(const u32x4 *)(wrow[rb] + koff + s * 32);
    u32x4 bx[MB][4];
#pragma unroll
    for (int cb = 0; cb < MB; ++cb)
#pragma unroll
      for (int s = 0; s < 4; ++s)
        bx[cb][s] = xval[cb] ? *(const u32x4 *)(xrow[cb] + koff + s * 32) : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
      for (int rb = 0; rb < 4; ++rb)
#pragma unroll
        for (int cb = 0; cb < MB; ++cb)
          acc[rb][cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
              __builtin_bit_cast(bf16x8, a[rb][s]), __builtin_bit_cast(bf16x8, bx[cb][s]),
              acc[rb][cb], 0, 0, 0);
  }

  // Fixed-order sum of the four waves' partial results, 64 activation rows at a time.
  __shared__ float red[4][64][kRowsPerWG + 1];
  float *Ys = Y + (long long)split * y_split_stride;
#pragma unroll
  for (int half = 0; half < (MB + 3) / 4; ++half) {
    __syncthreads();
#pragma unroll
    for (int cbh = 0; cbh < 4; ++cbh) {
      const int cb = half * 4 + cbh;
      if (cb < MB) {
#pragma unroll
        for (int rb = 0; rb < 4; ++rb)
#pragma unroll
          for (int i = 0; i < 4; ++i) red[wave][cbh * 16 + r][rb * 16 + gq * 4 + i] = acc[rb][cb][i];
      }
    }
    __syncthreads();
    const int rows_here = min(64, 16 * MB - half * 64);
    for (int e = threadIdx.x; e < rows_here * kRowsPerWG; e += 256) {
      const int m = e / kRowsPerWG, n = e % kRowsPerWG;
      const int mg = m0 + half * 64 + m;
      if (mg < M) {
        const float v = ((red[0][m][n] + red[1][m][n]) + red[2][m][n]) + red[3][m][n];
        Ys[(size_t)mg * ldy + n0 + n] = v;
      }
    }
  }
}

// fp32: 64 output columns x 16 rows per workgroup, reduction staged through LDS.
__global__ __launch_bounds__(256) void k_gemm_f32(WSegs segs, int N, int K, const float *__restrict__ X,
                                                  int ldx, int M, float *__restrict__ Y, int ldy) {
  __shared__ float Ws[64][65];
  __shared__ float Xs[16][65];
  const int t = threadIdx.x;
  const int n0 = blockIdx.x * 64, m0 = blockIdx.y * 16;
  const int nn = t & 63, mq = t >> 6;  // 4 rows per thread: mq*4 .. mq*4+3
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
  for (int k0 = 0; k0 < K; k0 += 64) {
    __syncthreads();
    for (int e = t; e < 64 * 64; e += 256) {
      const int rr = e >> 6, kk = e & 63;
      const int n = n0 + rr, k = k0 + kk;
      float v = 0.f;
      if (n < N && k < K) {
        int nloc = n, sgi = 0;
        while (sgi < 2 && nloc >= segs.rows[sgi]) nloc -= segs.rows[sgi++];
        v = ((const float *)segs.w[sgi])[(size_t)nloc * K + k];
      }
      Ws[rr][kk] = v;
    }
    for (int e = t; e < 16 * 64; e += 256) {
      const int rr = e >> 6, kk = e & 63;
      const int m = m0 + rr, k = k0 + kk;
      Xs[rr][kk] = (m < M && k < K) ? X[(size_t)m * ldx + k] : 0.f;
    }
    __syncthreads();
#pragma unroll 8
    for (int kk = 0; kk < 64; ++kk) {
      const float w = Ws[nn][kk];
#pragma unroll
      for (int i = 0; i < 4; ++i) acc[i] = fmaf(Xs[mq * 4 + i][kk], w, acc[i]);
    }
  }
  const int n = n0 + nn;
  if (n < N) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int m = m0 + mq * 4 + i;
      if (m < M) Y[(size_t)m * ldy + n] = acc[i];
    }
  }
}

}  // namespace

// Reduction splits for a weight matrix of n_full rows and K columns.  Depends
// on the matrix shape only (never on the number of stacked rows), so every
// output element is summed in the same order whichever paths are active.
int gemm_splits(int n_full, int K, int dtype) {
  if (dtype != 1) return 1;
  const int tiles = n_full / kRowsPerWG;
  int best = 1;
  for (int S = 1; S <= 8; ++S) {
    if (K % (kChunk * S) != 0 || K / S < 4 * kChunk) continue;
    best = S;
    if (tiles * S >= 256) break;
  }
  return best;
}

hipError_t launch_gemm(const WSegs &segs, int N, int K, int dtype, const void *X, int ldx, int M,
                       float *Y, int ldy, long long y_split_stride, int S, hipStream_t st) {
  if (M <= 0 || N <= 0) return hipSuccess;
  if (dtype == 1) {
    const int mb_total = (M + 15) / 16;
    const int MB = mb_total >= 8 ? 8 : mb_total;
    dim3 grid(N / kRowsPerWG, S, (mb_total + MB - 1) / MB);
    const int kps = K / S;
    const uint16_t *Xb = (const uint16_t *)X;
    switch (MB) {
      case 1: hipLaunchKernelGGL(k_gemm_bf16<1>, grid, dim3(256), 0, st, segs, K, Xb, ldx, M, Y, ldy, y_split_stride, kps); break;
      case 2: hipLaunchKernelGGL(k_gemm_bf16<2>, grid, dim3(256), 0, st, segs, K, Xb, ldx, M, Y, ldy, y_split_stride, kps); break;
      case 3: hipLaunchKernelGGL(k_gemm_bf16<3>, grid, dim3(256), 0, st, segs, K, Xb, ldx, M, Y, ldy, y_split_stride, kps); break;
      case 4: hipLaunchKernelGGL(k_gemm_bf16<4>, grid, dim3(256), 0, st, segs, K, Xb, ldx, M, Y, ldy, y_split_stride, kps); break;
      case 5: hipLaunchKernelGGL(k_gemm_bf16<5>, grid, dim3(256), 0, st, segs, K, Xb, ldx, M, Y, ldy, y_split_stride, kps); break;
      case 6: hipLaunchKernelGGL(k_gemm_bf16<6>, grid, dim3(256), 0, st, segs, K, Xb, ldx, M, Y, ldy, y_split_stride, kps); break;
      case 7: hipLaunchKernelGGL(k_gemm_bf16<7>, grid, dim3(256), 0, st, segs, K, Xb, ldx, M, Y, ldy, y_split_stride, kps); break;
      default: hipLaunchKernelGGL(k_gemm_bf16<8>, grid, dim3(256), 0, st, segs, K, Xb, ldx, M, Y, ldy, y_split_stride, kps); break;
    }
  } else {
    dim3 grid((N + 63) / 64, (M + 15) / 16);
    hipLaunchKernelGGL(k_gemm_f32, grid, dim3(256), 0, st, segs, N, K, (const float *)X, ldx, M, Y, ldy);
  }
  return hipGetLastError();
}

}  // namespace dbt
