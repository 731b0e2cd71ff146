// Projections of a whole prompt (primary prefill, Sec. 4.4): Y = X W^T with
// thousands of activation rows, where every weight row is reused by many
// rows and the work is bound by the matrix cores, not by the weight read.
//
// Workgroup of eight waves per 256-row x BN-column output tile; the reduction
// runs in 64-element steps.  Each step's X tile (256 x 64) and W tile
// (BN x 64) are loaded once per workgroup (16-byte pieces, one register
// stage) into one of two LDS buffers while the other buffer is multiplied.
// Waves form a 4 (rows) x 2 (columns) grid; a wave owns 64 rows x BN/2
// columns and multiplies with v_mfma_f32_16x16x32_bf16, W as the A operand
// and X as the B operand, so each lane ends with four consecutive output
// columns of one row (16-byte stores).
//
// LDS rows are 128 bytes (64 bf16); the 16-byte chunk c of row r sits at
// chunk c ^ (r & 7).  Measured on gfx950 (16 waves issuing ds_read_b128 /
// ds_write_b128): the operand reads (16 consecutive rows at one chunk) and
// the staging writes (eight threads per row) then run at the conflict-free
// rate, where the unswizzled rows take 4x and c ^ ((r & 7) ^ ((r >> 3) & 1))
// 2x as long per read.
//
// Epilogues (EPI): plain fp32 output; GLU, the gate/up projection of the
// SwiGLU MLP (Eq. (13), primary rows): a tile holds BN/2 gate and the same
// BN/2 up rows, laid out so each lane holds gate and up values of the same
// (row, column), and the epilogue writes H = silu(gate) * up in bf16 (and
// keeps one row in fp32 when asked) instead of the fp32 gate/up outputs;
// QKV, the stacked Q/K/V projection of a prompt (Eq. (8), rows = positions):
// a 128-column tile is one head, laid out so each lane holds dimensions i
// and i + 64 of it (the rotary pair), and the epilogue applies the rotary
// embedding to Q and K, writes Q in fp32 (and the kept row) and K and V in
// the model dtype into the cache pages, instead of the fp32 Q/K/V outputs.
#include "common.h"
#include "kernels.h"

namespace dbt {

namespace {

constexpr int kTM = 256, kTK = 64;

__device__ __forceinline__ int swz(int row, int c) { return (c ^ (row & 7)) * 8; }

typedef __attribute__((address_space(3))) void lds_void;

enum { EPI_PLAIN = 0, EPI_GLU = 1, EPI_QKV = 2 };

template <int BN, int EPI>
__global__ __launch_bounds__(512) void k_gemm_tile(TileGemm g) {
  constexpr bool GLU = EPI == EPI_GLU, QKV = EPI == EPI_QKV;
  static_assert(!QKV || BN == 128, "one head of 128 dimensions per tile");
  constexpr int NA = BN / 32;      // 16-column tiles per wave
  constexpr int WP = BN / 64;      // W row groups (8 rows) loaded per wave per step
  __shared__ __attribute__((aligned(16))) uint16_t xs0[kTM * kTK], xs1[kTM * kTK];
  __shared__ __attribute__((aligned(16))) uint16_t ws0[BN * kTK], ws1[BN * kTK];
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int r = lane & 15, gq = lane >> 4;
  const int wm = wave & 3, wn = wave >> 2;  // wave's row block (64 rows) and column half
  const int m0 = blockIdx.y * kTM;
  const int ntile_cols = GLU ? BN / 2 : BN;
  const int n0 = blockIdx.x * ntile_cols;
  const int K = g.K;
  const int nk = K / kTK;

  // Loads go straight from global memory into LDS (global_load_lds_dwordx4):
  // one instruction of a wave fills eight whole 128-byte rows, lane l the
  // 16-byte slot l & 7 of row l >> 3, so each lane fetches the chunk that
  // the swizzle places in its slot.  X rows 32 wave + 8 i, W rows
  // 8 (WP wave + i).
  const int lrow = lane >> 3, lslot = lane & 7;
  const int lchunk = lslot ^ lrow;  // rows of a group start at multiples of 8
  // Each group of eight rows starts at a row uniform over the wave, so the
  // matrix (segment) base stays in scalar registers and a lane keeps a
  // 32-bit element offset.  Rows past the end re-read the last row.
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);
  uint32_t xo[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = min(m0 + 8 * (4 * wave_u + i) + lrow, g.M - 1);
    xo[i] = (uint32_t)row * (uint32_t)g.ldx + lchunk * 8;
  }
  const uint16_t *wb[WP];
  uint32_t wo[WP];
#pragma unroll
  for (int i = 0; i < WP; ++i) {
    const int grow = 8 * (WP * wave_u + i);  // first row of the group in the W tile
    int seg_row, row;                        // the group's first matrix row, this lane's row
    const uint16_t *base;
    if (GLU) {
      const bool up = grow >= BN / 2;
      seg_row = n0 + (up ? grow - BN / 2 : grow);
      row = min(seg_row + lrow, g.N - 1);
      base = up ? g.w[1] : g.w[0];
    } else {
      seg_row = min(n0 + grow, g.N - 1);
      row = min(n0 + grow + lrow, g.N - 1);
      base = g.w[0];
      if (seg_row >= g.rows[0]) {  // segment sizes are multiples of 8: one segment per group
        seg_row -= g.rows[0];
        row -= g.rows[0];
        base = g.w[1];
        if (seg_row >= g.rows[1]) {
          row -= g.rows[1];
          base = g.w[2];
        }
      }
    }
    wb[i] = base;
    wo[i] = (uint32_t)row * (uint32_t)K + lchunk * 8;
  }
  auto dma = [&](int kt, uint16_t *xs, uint16_t *ws) {
    const int k0 = kt * kTK;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      __builtin_amdgcn_global_load_lds((const void *)(g.X + (xo[i] + k0)), (lds_void *)(xs + (8 * (4 * wave_u + i)) * kTK),
                                       16, 0, 0);
#pragma unroll
    for (int i = 0; i < WP; ++i)
      __builtin_amdgcn_global_load_lds((const void *)(wb[i] + (wo[i] + k0)),
                                       (lds_void *)(ws + (8 * (WP * wave_u + i)) * kTK), 16, 0, 0);
  };
  // W tile row of the wave's column tile a (GLU, QKV: tiles a and a + NA/2
  // are the same columns of the tile's two halves)
  auto wrow = [&](int a) {
    if (GLU || QKV) return a < NA / 2 ? (BN / 4) * wn + 16 * a : BN / 2 + (BN / 4) * wn + 16 * (a - NA / 2);
    return (BN / 2) * wn + 16 * a;
  };

  floatx4 acc[NA][4];
#pragma unroll
  for (int a = 0; a < NA; ++a)
#pragma unroll
    for (int b = 0; b < 4; ++b) acc[a][b] = floatx4{0.f, 0.f, 0.f, 0.f};

  auto fread = [&](const uint16_t *xs, const uint16_t *ws, int s, u32x4 *xf, u32x4 *wf) {
    const int c = 4 * s + gq;
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const int row = 64 * wm + 16 * b + r;
      xf[b] = *(const u32x4 *)&xs[row * kTK + swz(row, c)];
    }
#pragma unroll
    for (int a = 0; a < NA; ++a) {
      const int row = wrow(a) + r;
      wf[a] = *(const u32x4 *)&ws[row * kTK + swz(row, c)];
    }
  };
  auto mma = [&](const u32x4 *xf, const u32x4 *wf, int a0, int a1) {
#pragma unroll
    for (int a = a0; a < a1; ++a)
#pragma unroll
      for (int b = 0; b < 4; ++b)
        acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, wf[a]),
                                                            __builtin_bit_cast(bf16x8, xf[b]), acc[a][b], 0, 0, 0);
  };
  // The first half's operand reads are issued together, its first
  // multiplies wait only for their own operands, and the second half's reads
  // are issued behind them (at most 15 LDS reads are counted in flight), so a
  // step exposes one LDS round trip instead of one per group of eight
  // multiplies; the scheduling barriers keep the compiler from sinking each
  // read to its use.
  auto compute = [&](const uint16_t *xs, const uint16_t *ws) {
    u32x4 xf0[4], wf0[NA], xf1[4], wf1[NA];
    fread(xs, ws, 0, xf0, wf0);
    __builtin_amdgcn_sched_barrier(0);
    mma(xf0, wf0, 0, NA / 2);
    __builtin_amdgcn_sched_barrier(0);
    fread(xs, ws, 1, xf1, wf1);
    __builtin_amdgcn_sched_barrier(0);
    mma(xf0, wf0, NA / 2, NA);
    mma(xf1, wf1, 0, NA);
  };

  // Step kt: wait for this wave's loads of step kt and meet at the barrier
  // (then step kt is in LDS and every wave has finished step kt - 1), load
  // step kt + 1 into the buffer step kt - 1 used, multiply step kt.  The
  // buffers are separate arrays and the loop runs in pairs of steps, so each
  // buffer is known at compile time.  A step past the end reloads the last
  // tile, which is never read.
  // (The scheduling barriers keep each step's loads in front of its
  // multiplies, where they have the whole step to land.)
  dma(0, xs0, ws0);
  for (int kt = 0; kt < nk; kt += 2) {
    __syncthreads();
    dma(min(kt + 1, nk - 1), xs1, ws1);
    __builtin_amdgcn_sched_barrier(0);
    compute(xs0, ws0);
    if (kt + 1 < nk) {  // uniform
      __syncthreads();
      dma(min(kt + 2, nk - 1), xs0, ws0);
      __builtin_amdgcn_sched_barrier(0);
      compute(xs1, ws1);
    }
  }
  __syncthreads();  // no load into LDS outlives the workgroup

  // epilogue: lane holds output rows m0 + 64 wm + 16 b + r, columns
  // (tile column of a) + 4 gq .. + 3
#pragma unroll
  for (int b = 0; b < 4; ++b) {
    const int m = m0 + 64 * wm + 16 * b + r;
    if (m >= g.M) continue;
    if (QKV) {
      // tile n0 is Q head n0/128, then K heads, then V heads
      const int dq = g.rows[0], dkv = g.rows[1];
      const int pos = m;
      const size_t page = (size_t)g.kv.page_table[(size_t)g.seq * g.kv.mpps + pos / 16];
      const int slot = pos % 16;
#pragma unroll
      for (int a = 0; a < NA / 2; ++a) {
        const int d0 = (BN / 4) * wn + 16 * a + 4 * gq;  // dimensions d0 .. d0+3 and d0+64 .. d0+67
        float x0[4], x1[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          x0[i] = acc[a][b][i];
          x1[i] = acc[a + NA / 2][b][i];
        }
        if (n0 < dq + dkv) {  // uniform over the workgroup: rotary embedding on Q and K
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float2 y = rope_pair(x0[i], x1[i], g.rope[(size_t)pos * 64 + d0 + i]);
            x0[i] = y.x;
            x1[i] = y.y;
          }
        }
        if (n0 < dq) {
          const int c0 = n0 + d0;
          *(float4 *)(g.Qout + (size_t)m * dq + c0) = float4{x0[0], x0[1], x0[2], x0[3]};
          *(float4 *)(g.Qout + (size_t)m * dq + c0 + 64) = float4{x1[0], x1[1], x1[2], x1[3]};
          if (g.ret && (g.ret_src < 0 || m == g.ret_src)) {
            float *kept = g.ret + (size_t)(g.ret_src < 0 ? m : g.ret_dst) * dq + c0;
            *(float4 *)kept = float4{x0[0], x0[1], x0[2], x0[3]};
            *(float4 *)(kept + 64) = float4{x1[0], x1[1], x1[2], x1[3]};
          }
        } else if (n0 < dq + dkv) {
          const int hd = (n0 - dq) / 128;
          uint16_t *kp = (uint16_t *)g.kv.k + ((page * g.kv.n_kv + hd) * 16 + slot) * 128;
          *(u32x2 *)(kp + d0) = u32x2{pack2(x0[0], x0[1]), pack2(x0[2], x0[3])};
          *(u32x2 *)(kp + d0 + 64) = u32x2{pack2(x1[0], x1[1]), pack2(x1[2], x1[3])};
        } else {
          const int hd = (n0 - dq - dkv) / 128;
          uint16_t *vp = (uint16_t *)g.kv.v + (page * g.kv.n_kv + hd) * 128 * 16 + slot;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            vp[(d0 + i) * 16] = f2bf(x0[i]);
            vp[(d0 + 64 + i) * 16] = f2bf(x1[i]);
          }
        }
      }
    } else if (GLU) {
      const bool keep = g.ret && (g.ret_src < 0 || m == g.ret_src);
      const int kept_row = g.ret_src < 0 ? m : g.ret_dst;
#pragma unroll
      for (int a = 0; a < NA / 2; ++a) {
        const int j = n0 + (BN / 4) * wn + 16 * a + 4 * gq;
        if (j >= g.N) continue;
        float h[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          // silu with the hardware exponential and reciprocal (v_exp_f32,
          // v_rcp_f32: about 1 ulp each, far below the bf16 rounding of H);
          // the IEEE-exact forms cost ~20 instructions per value
          const float gt = acc[a][b][i], up = acc[a + NA / 2][b][i];
          h[i] = gt * __builtin_amdgcn_rcpf(1.0f + __expf(-gt)) * up;
        }
        *(u32x2 *)(g.H + (size_t)m * g.ldh + j) =
            u32x2{(uint32_t)f2bf(h[0]) | ((uint32_t)f2bf(h[1]) << 16), (uint32_t)f2bf(h[2]) | ((uint32_t)f2bf(h[3]) << 16)};
        if (keep) *(float4 *)(g.ret + (size_t)kept_row * g.N + j) = float4{h[0], h[1], h[2], h[3]};
      }
    } else {
#pragma unroll
      for (int a = 0; a < NA; ++a) {
        const int n = n0 + (BN / 2) * wn + 16 * a + 4 * gq;
        if (n >= g.N) continue;
        *(floatx4 *)(g.Y + (size_t)m * g.ldy + n) = acc[a][b];
      }
    }
  }
}

}  // namespace

bool gemm_tile_ok(int N, int K, int M, int dtype) {
  return dtype == 1 && M >= kTM && K % kTK == 0 && N % 16 == 0;
}

bool gemm_tile_args_ok(const TileGemm &g, bool glu) {
  if (!gemm_tile_ok(g.N, g.K, g.M, 1) || g.ldx % 8 != 0) return false;
  if (!glu && (g.rows[0] % 8 != 0 || g.rows[1] % 8 != 0 || g.rows[0] + g.rows[1] + g.rows[2] != g.N)) return false;
  // the QKV epilogue: heads of 128 dimensions, Q then K then V (as many V as K heads)
  if (g.rope && (g.kv.d_h != 128 || g.rows[0] % 128 != 0 || g.rows[1] != g.kv.n_kv * 128 || g.rows[2] != g.rows[1] ||
                 !g.Qout || !g.kv.k || !g.kv.v || !g.kv.page_table))
    return false;
  // 32-bit element offsets
  return (long long)g.M * g.ldx < (1LL << 32) && (long long)g.N * g.K < (1LL << 32);
}

hipError_t launch_gemm_tile(const TileGemm &g, bool glu, hipStream_t st) {
  if (!gemm_tile_args_ok(g, glu)) return hipErrorInvalidValue;
  const int mt = (g.M + kTM - 1) / kTM;
  // One workgroup per compute unit (128 KB of LDS): the wider tile (twice the
  // multiplies per loaded byte) unless its tile count leaves more of the
  // last round of workgroups idle than the narrower one's.
  static int cus = 0;  // compute units of the current device (one device type per process)
  if (!cus) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        cus <= 0)
      cus = 256;
  }
  auto fill = [&](long long tiles) { return (double)tiles / (double)(((tiles + cus - 1) / cus) * cus); };
  const long long t256 = (long long)(g.N / 256) * mt, t128 = (long long)((g.N + 127) / 128) * mt;
  if (glu) {
    hipLaunchKernelGGL((k_gemm_tile<256, EPI_GLU>), dim3((g.N + 127) / 128, mt), dim3(512), 0, st, g);
  } else if (g.rope) {
    hipLaunchKernelGGL((k_gemm_tile<128, EPI_QKV>), dim3(g.N / 128, mt), dim3(512), 0, st, g);
  } else if (g.N % 256 == 0 && fill(t256) >= fill(t128)) {
    hipLaunchKernelGGL((k_gemm_tile<256, EPI_PLAIN>), dim3(g.N / 256, mt), dim3(512), 0, st, g);
  } else {
    hipLaunchKernelGGL((k_gemm_tile<128, EPI_PLAIN>), dim3((g.N + 127) / 128, mt), dim3(512), 0, st, g);
  }
  return hipGetLastError();
}

}  // namespace dbt
