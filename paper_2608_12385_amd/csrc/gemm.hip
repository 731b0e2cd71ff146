// Stacked-row projections Y = X W^T for the decode step (Sec. 4.4 "Decode":
// the two paths' residual rows are stacked so each weight tile is read once
// for both; Sec. 4.5, Eq. (20): the step is bound by weight + KV traffic).
//
// bf16 weights: MFMA v_mfma_f32_16x16x32_bf16.  A workgroup of NW waves owns
// NW*16*RB weight rows and up to 128 activation rows; each wave owns 16*RB of
// the weight rows and accumulates over the whole reduction range in 128-wide
// chunks.
// Optional split of the reduction across workgroups (grid.y) writes one fp32
// slab per split; the consumer kernel adds the slabs in split order.  The
// per-element arithmetic never depends on how many rows are stacked, so the
// primary rows come out bit-identical with or without the branch rows.
//
// fp32 weights: an LDS-tiled vector kernel (small models).
#include <type_traits>

#include "common.h"
#include "kernels.h"

#include <algorithm>

namespace dbt {

namespace {

constexpr int kChunk = 128;  // reduction elements per pipeline stage
constexpr int kLdsRow = kChunk + 8;  // padded LDS row of a staged activation chunk (elements)

constexpr int gcd2(int a, int b) { return b == 0 ? a : gcd2(b, a % b); }
constexpr int lcm3(int a, int b, int c) {
  const int ab = a / gcd2(a, b) * b;
  return ab / gcd2(ab, c) * c;
}

// A workgroup owns NW*16*RB consecutive weight rows of one segment (the last
// tile of a segment may be partial: its rows past the end re-read the last
// row and are not stored); wave w owns rows w*16*RB .. +16*RB and runs the
// whole reduction range of its split.  The activation chunk [16*MB rows][128]
// is staged once per workgroup in LDS (contiguous loads) and read by all waves
// in MFMA operand layout, so larger workgroups re-read the activations from
// L2 less often per weight byte.
//
// Pipeline: while chunk c is multiplied, the activations of chunk c+2 and
// the weights of chunk c+PD are loaded; the activation chunk c+1, loaded one
// step earlier, is then written to the other of two LDS slots.  Vector loads
// complete in issue order, so that write never waits for the loads just
// issued (whatever the weight depth PD), and the weights behind it stay in
// flight.
// Loads are never predicated (rows past M re-read row M-1, chunks past the
// end re-read the last one), and the loop body always runs PD chunks, so the
// compiler's wait counts stay exact across the loop's back edge.
//
// Weight loads: each wave instruction reads eight whole 128-byte row pieces
// (eight lanes per row) with the non-temporal hint, so every request is a
// full cache line that is used once and not kept; the wave then moves the
// pieces into the MFMA operand layout (16 rows x 64 bytes per instruction)
// through its own LDS region, half a chunk at a time.  Loading the operand
// layout directly would cover only half of each line per instruction, and
// the streaming read is slower that way (about 6.3 against 6.9 TB/s for a
// plain read of the output matrix).
//
// Each workgroup starts at its own chunk of the split, (tile * 7) mod chunks,
// and wraps around: workgroups running at the same time then read different
// column ranges of their rows instead of all hitting the same few memory
// channels (row strides are powers of two).  The order is a function of the
// row tile and the split only.
//
// GLU (RB = 1): each wave owns eight rows of segment 0 (gate) and the same
// eight rows of segment 1 (up) as one 16-row MFMA block, so a lane's
// accumulators for gate row n sit four lanes-groups away from those of up
// row n (lane + 32); the workgroup owns NW*8 gate rows.  Instead of storing
// Y the epilogue finishes the MLP intermediate in registers (see GluEpi):
// the branch rows' coupling partner, the primary row of the same sequence,
// is held by the same lane.
// XF: the activations are the fp32 inputs of XNorm (first layer of a
// layer-only model): each staged piece is bf16(h * g), and the workgroups of
// the first row tile write each row's sum of squares of h over their split
// (the 16 pieces of a chunk row sit in 16 consecutive lanes; summed over the
// chunks in order, then across the lanes by a fixed butterfly).
struct NoX {};
template <bool XF> using XArg = std::conditional_t<XF, XNorm, NoX>;

template <int MB, int RB, int PD, int NW, bool GLU = false, int XA = 2, bool XF = false>
__global__ __launch_bounds__(NW * 64) void k_gemm_bf16(WSegs segs, int K, const uint16_t *__restrict__ X, int ldx,
                                                       int M, float *__restrict__ Y, int ldy,
                                                       long long y_split_stride, float *__restrict__ row_stats,
                                                       GluEpi ep, XArg<XF> xa) {
  constexpr int XR = 16 * MB;
  constexpr int PIECES = XR * (kChunk / 8);  // 16-byte pieces of one activation chunk
  constexpr int PPT = (PIECES + NW * 64 - 1) / (NW * 64);
  constexpr int ROWS = NW * 16 * RB;  // weight rows per workgroup
  __shared__ uint16_t xs[2][XR * kLdsRow];
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int r = lane & 15, gq = lane >> 4;
  const int split = blockIdx.y;
  const int m0 = blockIdx.z * XR;
  // split s covers chunks [s*NC/S, (s+1)*NC/S) of the NC = K/128 chunks
  const int NC = K / kChunk, S = gridDim.y;
  const int c_lo = split * NC / S, c_hi = (split + 1) * NC / S;
  const int kbeg = c_lo * kChunk;
  const int nch = c_hi - c_lo;
  const int crot = (int)(blockIdx.x * 7u % (unsigned)nch);
  // segment of this workgroup's rows: every segment but the last holds a
  // multiple of ROWS rows; the tiles of the last one are numbered on
  int nloc = blockIdx.x * ROWS;
  const uint16_t *Wseg = (const uint16_t *)segs.w[0];
  int segrows = segs.rows[0];
  static_assert(!GLU || RB == 1, "GLU waves own one 8 + 8 row block");
  const int g0 = blockIdx.x * NW * 8 + wave * 8;  // GLU: first gate (= up) row of this wave
  if (GLU) {
    // (no segment walk: rows come from w[0] and w[1] below)
  } else if (nloc >= segs.rows[0] && segs.rows[1] > 0) {
    nloc -= segs.rows[0];
    Wseg = (const uint16_t *)segs.w[1];
    segrows = segs.rows[1];
    if (nloc >= segs.rows[1] && segs.rows[2] > 0) {
      nloc -= segs.rows[1];
      Wseg = (const uint16_t *)segs.w[2];
      segrows = segs.rows[2];
    }
  }
  const int nw = nloc + wave * 16 * RB;             // first row of this wave within the segment
  const int ny = blockIdx.x * ROWS + wave * 16 * RB;  // first output column of this wave
  // weight pointers of the coalesced loads: row block rb, row group j (rows
  // rb*16 + j*8 + lane/8), 16-byte piece lane%8 of a 128-byte half chunk
  const int lr8 = lane >> 3, lp8 = lane & 7;
  const uint16_t *wrow[RB][2];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int j = 0; j < 2; ++j)
      wrow[rb][j] = GLU ? (const uint16_t *)segs.w[j] + (size_t)min(g0 + lr8, segs.rows[0] - 1) * K + kbeg + lp8 * 8
                        : Wseg + (size_t)min(nw + rb * 16 + j * 8 + lr8, segrows - 1) * K + kbeg + lp8 * 8;
  // the wave's LDS region: RB*16 rows of one half chunk (8 pieces of 16
  // bytes); piece p of row R sits in slot p ^ (R & 7)
  __shared__ u32x4 wt[NW][RB * 16 * 8];
  u32x4 *wreg = wt[wave];
  const uint16_t *xsrc[PPT];
  const float *xsf[PPT];  // XF: the piece's fp32 input row
  int xdst[PPT], gcol[PPT];
#pragma unroll
  for (int j = 0; j < PPT; ++j) {
    const int p = t + NW * 64 * j, row = min(p >> 4, XR - 1), col = (p & 15) * 8;
    xsrc[j] = X + (size_t)min(m0 + row, M - 1) * ldx + kbeg + col;
    xdst[j] = p < PIECES ? row * kLdsRow + col : -1;
    gcol[j] = kbeg + col;
    if constexpr (XF) {
      const int mm = min(m0 + row, M - 1);
      const int path = xa.rows.p0 + mm / xa.rows.Bp, b = min(mm % xa.rows.Bp, xa.h.B - 1);
      xsf[j] = (path == 0 ? xa.h.h1 : xa.h.h2 + (size_t)(path - 1) * xa.h.B * K) + (size_t)b * K + kbeg + col;
    }
  }
  if constexpr (XF) {
    // the step's positions and new page-table entries, for the kernels after
    // this one (the first to read them is the attention)
    if (blockIdx.x == 0 && blockIdx.y == 0 && blockIdx.z == 0 && xa.pos_arr) {
      if (t < xa.sb.n_pos) xa.pos_arr[xa.sb.b0 + t] = xa.sb.pos[t];
      if (t < xa.sb.n_pt) xa.page_table[(size_t)xa.sb.pt_b[t] * xa.mpps + xa.sb.pt_slot[t]] = xa.sb.pt_page[t];
    }
  }
  float ssq[PPT];  // XF: sums of squares of the staged pieces
#pragma unroll
  for (int j = 0; j < PPT; ++j) ssq[j] = 0.f;

  floatx4 acc[RB][MB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int cb = 0; cb < MB; ++cb) acc[rb][cb] = floatx4{0.f, 0.f, 0.f, 0.f};

  static_assert(XA >= 2, "activation chunks are loaded at least two steps ahead");
  u32x4 a[PD][RB][4], stg[XA][PPT];
  // XF: h of each piece (two float4) and g of their columns (two float4:
  // every piece of a thread has the same columns, NW*64 being a multiple of 16)
  float4 stf[XF ? XA : 1][XF ? PPT : 1][2], stg_g[XF ? XA : 1][2];
  auto koff = [&](int c) {  // logical chunk c (clamped) of this workgroup's rotated order
    c = min(c, nch - 1) + crot;
    return (c >= nch ? c - nch : c) * kChunk;
  };
  auto xload = [&](int slot, int c) {
    const int ko = koff(c);
#pragma unroll
    for (int j = 0; j < PPT; ++j) {
      if constexpr (XF) {
        stf[slot][j][0] = *(const float4 *)(xsf[j] + ko);
        stf[slot][j][1] = *(const float4 *)(xsf[j] + ko + 4);
        if (j == 0) {
          stg_g[slot][0] = *(const float4 *)(xa.g + gcol[0] + ko);
          stg_g[slot][1] = *(const float4 *)(xa.g + gcol[0] + ko + 4);
        }
      } else {
        stg[slot][j] = *(const u32x4 *)(xsrc[j] + ko);
      }
    }
  };
  // a[slot][rb][2h + j]: half h of row group j of row block rb
  auto wload = [&](int slot, int c) {
    const int ko = koff(c);
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          a[slot][rb][2 * h + j] = __builtin_nontemporal_load((const u32x4 *)(wrow[rb][j] + ko + h * 64));
  };
  auto xstore = [&](int lds, int slot) {
#pragma unroll
    for (int j = 0; j < PPT; ++j)
      if (PIECES % (NW * 64) == 0 || xdst[j] >= 0) {
        if constexpr (XF) {
          const float4 u = stf[slot][j][0], v = stf[slot][j][1], gu = stg_g[slot][0], gv = stg_g[slot][1];
          ssq[j] += ((u.x * u.x + u.y * u.y) + (u.z * u.z + u.w * u.w)) +
                    ((v.x * v.x + v.y * v.y) + (v.z * v.z + v.w * v.w));
          *(u32x4 *)(&xs[lds][xdst[j]]) = u32x4{pack2(u.x * gu.x, u.y * gu.y), pack2(u.z * gu.z, u.w * gu.w),
                                                pack2(v.x * gv.x, v.y * gv.y), pack2(v.z * gv.z, v.w * gv.w)};
        } else {
          *(u32x4 *)(&xs[lds][xdst[j]]) = stg[slot][j];
        }
      }
  };
  // multiply chunk c (weight ring slot w = c % PD, LDS slot par = c & 1);
  // load the activations of chunk c+XA (register slot xc = c % XA, whose
  // chunk c went to LDS one step ago) and the weights of chunk c+PD; stage
  // chunk c+1 (register slot xn = (c+1) % XA, loaded XA-1 steps ago) into
  // the other LDS slot.  All slots are compile-time at every call.
  auto step = [&](auto guard, int c, int w, int par, int xc, int xn) {
    constexpr bool GUARD = decltype(guard)::value;  // skip loads and staging past the last chunk
    const uint16_t *xl = xs[par];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      // half h of the wave's weight rows into its LDS region (the reads of
      // the previous half were issued before: LDS operations of a wave run
      // in order)
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int j = 0; j < 2; ++j) wreg[(rb * 16 + j * 8 + lr8) * 8 + (lp8 ^ lr8)] = a[w][rb][2 * h + j];
      wave_lds_fence();
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2) {
        const int s = 2 * h + s2;
        u32x4 bx[MB], wf[RB];
#pragma unroll
        for (int cb = 0; cb < MB; ++cb) bx[cb] = *(const u32x4 *)(&xl[(cb * 16 + r) * kLdsRow + s * 32 + gq * 8]);
        // operand of row block rb: row rb*16 + r, piece 4*s2 + gq of the half
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) wf[rb] = wreg[(rb * 16 + r) * 8 + ((4 * s2 + gq) ^ (r & 7))];
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
#pragma unroll
          for (int cb = 0; cb < MB; ++cb)
            acc[rb][cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, wf[rb]),
                                                                  __builtin_bit_cast(bf16x8, bx[cb]), acc[rb][cb], 0,
                                                                  0, 0);
      }
      wave_lds_fence();
    }
    if (!GUARD || c + XA < nch) xload(xc, c + XA);
    if (!GUARD || c + PD < nch) wload(w, c + PD);
    if (!GUARD || c + 1 < nch) xstore(par ^ 1, xn);
    __syncthreads();
  };

#pragma unroll
  for (int u = 0; u < XA; ++u) xload(u, u);
#pragma unroll
  for (int u = 0; u < PD; ++u) wload(u, u);
  xstore(0, 0);
  __syncthreads();
  // rounds of P2 chunks (a common multiple of PD, XA and 2, so every ring
  // position is a constant); the round's loads are the same every time,
  // which keeps the wait counts exact across the loop's back edge
  constexpr int P2 = lcm3(PD, XA, 2);
  int c0 = 0;
  if constexpr (NW <= 8) {
    // Rounds whose loads all fall inside the split run unguarded; the last
    // steps (at most P2 + LA - 1) skip the loads past the last chunk, which
    // would otherwise re-read it and hold the waves for one more memory
    // round trip at the end (W_O 10.5 -> 9.3 us, down 29.0 -> 26.4 us by the
    // last workgroup's end).  Sixteen-wave tiles keep the plain tail: its
    // unrolled steps would exceed their 128 registers.
    constexpr int LA = PD > XA ? PD : XA;
    for (; c0 + P2 + LA <= nch; c0 += P2) {
#pragma unroll
      for (int u = 0; u < P2; ++u) step(std::false_type{}, c0 + u, u % PD, u & 1, u % XA, (u + 1) % XA);
    }
#pragma unroll
    for (int u = 0; u < P2 + LA - 1; ++u)
      if (c0 + u < nch) step(std::true_type{}, c0 + u, u % PD, u & 1, u % XA, (u + 1) % XA);
  } else {
    for (; c0 + P2 <= nch; c0 += P2) {
#pragma unroll
      for (int u = 0; u < P2; ++u) step(std::false_type{}, c0 + u, u % PD, u & 1, u % XA, (u + 1) % XA);
    }
#pragma unroll
    for (int u = 0; u + 1 < P2; ++u)
      if (c0 + u < nch) step(std::false_type{}, c0 + u, u % PD, u & 1, u % XA, (u + 1) % XA);
  }
  if constexpr (XF) {
#pragma unroll
    for (int j = 0; j < PPT; ++j) {
      float v = ssq[j];
      v += __shfl_xor(v, 1, 64);
      v += __shfl_xor(v, 2, 64);
      v += __shfl_xor(v, 4, 64);
      v += __shfl_xor(v, 8, 64);
      const int p = t + NW * 64 * j, row = p >> 4;
      if (blockIdx.x == 0 && (p & 15) == 0 && p < PIECES && m0 + row < M)
        xa.ss[(size_t)split * xa.ss_ld + xa.rows.p0 * xa.rows.Bp + m0 + row] = v;
    }
  }
  // lane holds D[n = rb*16 + 4*gq + i][m = cb*16 + r]: Y[m][n .. n+3]
  if constexpr (GLU) {
    // lane (r, gq) holds D[n = 4gq + i][m = cb*16 + r]: gate rows n < 8
    // (gq < 2), up rows n >= 8 (gq >= 2, the up value of gate row n sits in
    // lane + 32).  H = SiLU(gate) * up (Eq. (13)); branch rows add b * H1 of
    // their sequence's primary row (Eq. (14)), block cb - p*Bp/16 of the
    // same lane (primary and branches in one tile, M <= 16*MB, m0 = 0) or the
    // retained H1.
    const int Bp = ep.rows.Bp, row0 = ep.rows.p0 * Bp;
    float h[MB][4];
#pragma unroll
    for (int cb = 0; cb < MB; ++cb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float g = acc[0][cb][i];
        const float u = __shfl_xor(g, 32, 64);
        h[cb][i] = g / (1.0f + expf(-g)) * u;
      }
    if (gq >= 2) return;
    const int n = g0 + 4 * gq;  // this lane's four columns n .. n+3 of H
    if (n >= ep.f) return;
#pragma unroll
    for (int cb = 0; cb < MB; ++cb) {
      const int gm = m0 + cb * 16 + r;  // row of this call (relative to its first row)
      if (gm >= M) continue;
      const int path = ep.rows.p0 + gm / Bp, b = gm % Bp;
      if (b >= ep.rows.B) continue;
      float o[4];
      if (path == 0) {
#pragma unroll
        for (int i = 0; i < 4; ++i) o[i] = h[cb][i];
        const Retain &rt = ep.ret;
        if (rt.ptr && (rt.src_row < 0 || rt.src_row == b))
          *(float4 *)&rt.ptr[(size_t)(rt.src_row < 0 ? b : rt.dst_row) * ep.f + n] = make_float4(o[0], o[1], o[2], o[3]);
      } else {
        const float4 bv = *(const float4 *)&ep.bvec[n];
        float h1[4];
        if (ep.rows.p0 == 0) {
          // the primary row b sits in block cb - path*Bp/16 of this lane
          const int cb1 = cb - path * (Bp / 16);
#pragma unroll
          for (int c2 = 0; c2 < MB; ++c2)
            if (c2 == cb1)
#pragma unroll
              for (int i = 0; i < 4; ++i) h1[i] = h[c2][i];
        } else {
          const float4 x = *(const float4 *)&ep.H1_in[(size_t)b * ep.f + n];
          h1[0] = x.x; h1[1] = x.y; h1[2] = x.z; h1[3] = x.w;
        }
        o[0] = h[cb][0] + bv.x * h1[0];
        o[1] = h[cb][1] + bv.y * h1[1];
        o[2] = h[cb][2] + bv.z * h1[2];
        o[3] = h[cb][3] + bv.w * h1[3];
      }
      uint2 pk;
      pk.x = pack2(o[0], o[1]);
      pk.y = pack2(o[2], o[3]);
      *(uint2 *)&ep.Xh[(size_t)(row0 + gm) * ep.ldh + n] = pk;
    }
    return;
  }
  bool rvalid[RB];  // 16-row block inside its segment (else a re-read of the last row)
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) rvalid[rb] = nw + rb * 16 < segrows;
  if (row_stats) {
    // Softmax statistics of each activation row over this workgroup's valid
    // outputs (one tile): max, sum e^(y - max), sum e^(2(y - max)); waves are
    // merged in wave order.  Used by the mixture readout (no split here).
    __shared__ float smx[NW][XR], s1[NW][XR], s2[NW][XR];
#pragma unroll
    for (int cb = 0; cb < MB; ++cb) {
      float mx = -INFINITY;
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
        if (rvalid[rb])
#pragma unroll
          for (int i = 0; i < 4; ++i) mx = fmaxf(mx, acc[rb][cb][i]);
      mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      if (gq == 0) smx[wave][cb * 16 + r] = mx;
    }
    __syncthreads();
#pragma unroll
    for (int cb = 0; cb < MB; ++cb) {
      const int mm = cb * 16 + r;
      float mx = smx[0][mm];
#pragma unroll
      for (int w = 1; w < NW; ++w) mx = fmaxf(mx, smx[w][mm]);
      float e1 = 0.f, e2 = 0.f;
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
        if (rvalid[rb])
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float e = __expf(acc[rb][cb][i] - mx);  // fast exp: lse and alpha need ~1e-6
            e1 += e;
            e2 += e * e;
          }
      e1 += __shfl_xor(e1, 16, 64);
      e1 += __shfl_xor(e1, 32, 64);
      e2 += __shfl_xor(e2, 16, 64);
      e2 += __shfl_xor(e2, 32, 64);
      if (gq == 0) {
        s1[wave][mm] = e1;
        s2[wave][mm] = e2;
      }
    }
    __syncthreads();
    if (t < XR && m0 + t < M) {
      float mx = smx[0][t], a1 = s1[0][t], a2 = s2[0][t];
#pragma unroll
      for (int w = 1; w < NW; ++w) {
        mx = fmaxf(mx, smx[w][t]);
        a1 += s1[w][t];
        a2 += s2[w][t];
      }
      float *o = row_stats + ((size_t)(m0 + t) * gridDim.x + blockIdx.x) * 3;
      o[0] = mx;
      o[1] = a1;
      o[2] = a2;
    }
  }
  // Output rows are written in whole 128-byte lines: a lane's accumulators
  // hold four columns of one row, so one store instruction would cover 16
  // rows x 64 bytes; the tile goes through LDS first (rows padded by four
  // floats, so the 16 rows of one accumulator write fall in distinct banks).
  float *Ys = Y + (long long)split * y_split_stride;
  if constexpr (RB >= 2) {
    // per wave: 16 rows x RB*16 columns at a time, in its own LDS region
    constexpr int WC = RB * 16, PITCH = WC + 4, LPR = WC / 4;  // columns, pitch, lanes per row
    static_assert(GLU || 16 * PITCH * 4 <= (int)sizeof(wt[0]), "output staging exceeds the wave's region");
    float *ost = (float *)&wt[wave][0];
#pragma unroll
    for (int cb = 0; cb < MB; ++cb) {
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) *(floatx4 *)&ost[r * PITCH + rb * 16 + gq * 4] = acc[rb][cb];
      wave_lds_fence();
#pragma unroll
      for (int j = 0; j < 16 * LPR / 64; ++j) {
        const int row = j * (64 / LPR) + lane / LPR, col = (lane % LPR) * 4;
        const int m = m0 + cb * 16 + row;
        const floatx4 v = *(const floatx4 *)&ost[row * PITCH + col];
        if (m < M && rvalid[col >> 4]) *(floatx4 *)(Ys + (size_t)m * ldy + ny + col) = v;
      }
      wave_lds_fence();
    }
  } else {
    // per workgroup: the XR x ROWS tile in the activation slots (free after
    // the loop's last barrier), then each row stored by ROWS/4 threads
    constexpr int PITCH = ROWS + 4, TPR = ROWS / 4;
    static_assert(GLU || XR * PITCH * 4 <= (int)sizeof(xs), "output staging exceeds the activation slots");
    float *ost = (float *)&xs[0][0];
#pragma unroll
    for (int cb = 0; cb < MB; ++cb) *(floatx4 *)&ost[(cb * 16 + r) * PITCH + wave * 16 + gq * 4] = acc[0][cb];
    __syncthreads();
    const int nt0 = blockIdx.x * ROWS;
    for (int e = t; e < XR * TPR; e += NW * 64) {
      const int row = e / TPR, col = (e % TPR) * 4;
      const int m = m0 + row;
      if (m < M && nloc + col < segrows)
        *(floatx4 *)(Ys + (size_t)m * ldy + nt0 + col) = *(const floatx4 *)&ost[row * PITCH + col];
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

// Launch configuration of a weight matrix of n_full rows and K columns:
// row blocks per wave (RB), weight prefetch depth (PD) and reduction splits
// (S).  It depends on the matrix shape only (never on the number of stacked
// rows), so every output element is summed in the same order whichever paths
// are active.
// seg_gran: every segment boundary of the stacked matrices is a multiple of it.
GemmConfig gemm_config(int n_full, int K, int dtype, int seg_gran, int max_rows) {
  GemmConfig g{1, 1, 1, 4};
  if (dtype != 1) return g;
  if (n_full >= 65536 && seg_gran == n_full && n_full % 64 == 0) {
    // output-matrix shapes (one segment): 16 waves x 32 rows = 512 rows per
    // workgroup, so each staged activation chunk serves 512 weight rows; above
    // 64 stacked rows 8 waves x 32 (at 96 rows the sixteen-wave tile spills
    // and took 208 us against 181 us for the 8B-shape head with two branches)
    g = max_rows <= 64 ? GemmConfig{2, 1, 1, 16} : GemmConfig{2, 1, 1, 8};
  } else if (n_full >= 16384 && seg_gran % 128 == 0) {
    g = GemmConfig{2, 2, 1, 4};    // MLP up projections
  } else {
    // thin matrices: split the reduction so that at most one workgroup per
    // compute unit runs (a second round of workgroups costs a whole round);
    // the fp32 slabs of up to max_rows stacked rows never exceed the weight
    // bytes, and every split keeps at least one chunk.  Tiles of 128 rows
    // (8 waves) unless 64-row tiles (4 waves) keep more compute units busy:
    // with one workgroup per unit, eight waves keep twice the weight bytes in
    // flight, and a unit's share of a thin matrix is small enough for its
    // read to be bound by load latency rather than bandwidth.  Where both
    // fill the chip alike and eight waves would need more than eight splits,
    // the 64-row tiles win: half the fp32 slabs to write and to sum (the
    // 24-layer model's down projection: 14.4 us in 32 x 8 against 15.0 us in
    // 16 x 16, and a shorter finish).
    const int nc = K / kChunk;
    auto splits = [&](int tiles) {
      int S = 256 / tiles;
      S = std::min(S, std::max(1, K / (2 * std::max(max_rows, 1))));
      return std::max(std::min({S, 16, std::max(nc, 1)}), 1);
    };
    const int t4 = std::max(1, n_full / 64), t8 = std::max(1, n_full / 128);
    const int s4 = splits(t4), s8 = splits(t8);
    if (seg_gran % 128 == 0 && (t8 * s8 > t4 * s4 || (t8 * s8 == t4 * s4 && s8 <= 8)))
      g = GemmConfig{1, 1, s8, 8};
    else
      g = GemmConfig{1, 2, s4, 4};
  }
  return g;
}

namespace {
template <int MB>
void launch_mb(const GemmConfig &g, dim3 grid, hipStream_t st, const WSegs &segs, int K, const uint16_t *X, int ldx,
               int M, float *Y, int ldy, long long yss, float *rs) {
  const GluEpi none{};
  if (g.NW == 16)
    hipLaunchKernelGGL((k_gemm_bf16<MB, 2, 1, 16>), grid, dim3(1024), 0, st, segs, K, X, ldx, M, Y, ldy, yss, rs, none, NoX{});
  else if (g.NW == 8 && g.RB == 2)
    hipLaunchKernelGGL((k_gemm_bf16<MB, 2, 1, 8>), grid, dim3(512), 0, st, segs, K, X, ldx, M, Y, ldy, yss, rs, none, NoX{});
  else if (g.NW == 8)
    hipLaunchKernelGGL((k_gemm_bf16<MB, 1, 1, 8>), grid, dim3(512), 0, st, segs, K, X, ldx, M, Y, ldy, yss, rs, none, NoX{});
  else if (g.RB == 2)
    hipLaunchKernelGGL((k_gemm_bf16<MB, 2, 2, 4>), grid, dim3(256), 0, st, segs, K, X, ldx, M, Y, ldy, yss, rs, none, NoX{});
  else
    hipLaunchKernelGGL((k_gemm_bf16<MB, 1, 2, 4>), grid, dim3(256), 0, st, segs, K, X, ldx, M, Y, ldy, yss, rs, none, NoX{});
}

template <int MB>
void launch_glu_mb(dim3 grid, hipStream_t st, const WSegs &segs, int K, const uint16_t *X, int ldx, int M,
                   const GluEpi &ep) {
  hipLaunchKernelGGL((k_gemm_bf16<MB, 1, 2, 8, true>), grid, dim3(512), 0, st, segs, K, X, ldx, M, nullptr, 0, 0LL,
                     nullptr, ep, NoX{});
}

template <int MB>
void launch_xnorm_mb(const GemmConfig &g, dim3 grid, hipStream_t st, const WSegs &segs, int K, const XNorm &xn, int M,
                     float *Y, int ldy, long long yss) {
  const GluEpi none{};
  if (g.NW == 8)
    hipLaunchKernelGGL((k_gemm_bf16<MB, 1, 1, 8, false, 2, true>), grid, dim3(512), 0, st, segs, K, nullptr, 0, M, Y,
                       ldy, yss, nullptr, none, xn);
  else if (g.RB == 2)
    hipLaunchKernelGGL((k_gemm_bf16<MB, 2, 2, 4, false, 2, true>), grid, dim3(256), 0, st, segs, K, nullptr, 0, M, Y,
                       ldy, yss, nullptr, none, xn);
  else
    hipLaunchKernelGGL((k_gemm_bf16<MB, 1, 2, 4, false, 2, true>), grid, dim3(256), 0, st, segs, K, nullptr, 0, M, Y,
                       ldy, yss, nullptr, none, xn);
}
}  // namespace

bool gemm_xnorm_ok(const GemmConfig &g, int M) {
  // the thin-matrix shapes, up to the stacked rows whose fp32 staging still
  // fits the registers (eight waves of one row block, or four of two: 96;
  // four waves of one row block: 128)
  if (M < 1) return false;
  if (g.NW == 8 && g.RB == 1 && g.PD == 1) return M <= 96;
  if (g.NW == 4 && g.RB == 2 && g.PD == 2) return M <= 96;
  if (g.NW == 4 && g.RB == 1 && g.PD == 2) return M <= 128;
  return false;
}

static int gemm_rows_per_wg(const GemmConfig &g) { return g.NW * 16 * g.RB; }

int gemm_tile_rows(const GemmConfig &g) { return gemm_rows_per_wg(g); }

int gemm_stats_tiles(int N, const GemmConfig &g, int dtype) {
  return (dtype == 1 && g.S == 1) ? (N + gemm_rows_per_wg(g) - 1) / gemm_rows_per_wg(g) : 0;
}

// Tiles of 64 gate + 64 up rows (eight waves of 8 + 8); enough of them to
// fill the chip, and a branch row's primary partner in the same activation
// tile (M <= 128).
bool gemm_glu_ok(int f, int M, int np, int dtype) {
  return dtype == 1 && f % 64 == 0 && f / 64 >= 192 && (np == 1 || M <= 128);
}

hipError_t launch_gemm_glu(const uint16_t *w_gate, const uint16_t *w_up, int f, int K, const void *X, int ldx, int M,
                           const GluEpi &ep, hipStream_t st) {
  if (M <= 0) return hipSuccess;
  if (!gemm_glu_ok(f, M, ep.rows.np, 1)) return hipErrorInvalidValue;
  const WSegs segs{{w_gate, w_up, nullptr}, {f, f, 0}};
  const int mb_total = (M + 15) / 16;
  const int MB = mb_total >= 8 ? 8 : mb_total;
  dim3 grid(f / 64, 1, (mb_total + MB - 1) / MB);
  const uint16_t *Xb = (const uint16_t *)X;
  switch (MB) {
    case 1: launch_glu_mb<1>(grid, st, segs, K, Xb, ldx, M, ep); break;
    case 2: launch_glu_mb<2>(grid, st, segs, K, Xb, ldx, M, ep); break;
    case 3: launch_glu_mb<3>(grid, st, segs, K, Xb, ldx, M, ep); break;
    case 4: launch_glu_mb<4>(grid, st, segs, K, Xb, ldx, M, ep); break;
    case 5: launch_glu_mb<5>(grid, st, segs, K, Xb, ldx, M, ep); break;
    case 6: launch_glu_mb<6>(grid, st, segs, K, Xb, ldx, M, ep); break;
    case 7: launch_glu_mb<7>(grid, st, segs, K, Xb, ldx, M, ep); break;
    default: launch_glu_mb<8>(grid, st, segs, K, Xb, ldx, M, ep); break;
  }
  return hipGetLastError();
}

hipError_t launch_gemm_xnorm(const WSegs &segs, int N, int K, const XNorm &xn, int M, float *Y, int ldy,
                             long long y_split_stride, const GemmConfig &g, hipStream_t st) {
  if (M <= 0 || N <= 0) return hipSuccess;
  if (!gemm_xnorm_ok(g, M) || K % kChunk || !xn.h.h1 || !xn.g || !xn.ss || xn.rows.Bp < 1 || xn.h.B < 1)
    return hipErrorInvalidValue;
  const int mb_total = (M + 15) / 16;
  const int MB = mb_total >= 8 ? 8 : mb_total;
  dim3 grid((N + gemm_rows_per_wg(g) - 1) / gemm_rows_per_wg(g), g.S, (mb_total + MB - 1) / MB);
  switch (MB) {
    case 1: launch_xnorm_mb<1>(g, grid, st, segs, K, xn, M, Y, ldy, y_split_stride); break;
    case 2: launch_xnorm_mb<2>(g, grid, st, segs, K, xn, M, Y, ldy, y_split_stride); break;
    case 3: launch_xnorm_mb<3>(g, grid, st, segs, K, xn, M, Y, ldy, y_split_stride); break;
    case 4: launch_xnorm_mb<4>(g, grid, st, segs, K, xn, M, Y, ldy, y_split_stride); break;
    case 5: launch_xnorm_mb<5>(g, grid, st, segs, K, xn, M, Y, ldy, y_split_stride); break;
    case 6: launch_xnorm_mb<6>(g, grid, st, segs, K, xn, M, Y, ldy, y_split_stride); break;
    case 7: launch_xnorm_mb<7>(g, grid, st, segs, K, xn, M, Y, ldy, y_split_stride); break;
    default: launch_xnorm_mb<8>(g, grid, st, segs, K, xn, M, Y, ldy, y_split_stride); break;
  }
  return hipGetLastError();
}

hipError_t launch_gemm(const WSegs &segs, int N, int K, int dtype, const void *X, int ldx, int M, float *Y,
                       int ldy, long long y_split_stride, const GemmConfig &g, hipStream_t st, float *row_stats) {
  if (M <= 0 || N <= 0) return hipSuccess;
  if (dtype == 1) {
    const int mb_total = (M + 15) / 16;
    const int MB = mb_total >= 8 ? 8 : mb_total;
    dim3 grid((N + gemm_rows_per_wg(g) - 1) / gemm_rows_per_wg(g), g.S, (mb_total + MB - 1) / MB);
    const uint16_t *Xb = (const uint16_t *)X;
    float *rs = g.S == 1 ? row_stats : nullptr;
    switch (MB) {
      case 1: launch_mb<1>(g, grid, st, segs, K, Xb, ldx, M, Y, ldy, y_split_stride, rs); break;
      case 2: launch_mb<2>(g, grid, st, segs, K, Xb, ldx, M, Y, ldy, y_split_stride, rs); break;
      case 3: launch_mb<3>(g, grid, st, segs, K, Xb, ldx, M, Y, ldy, y_split_stride, rs); break;
      case 4: launch_mb<4>(g, grid, st, segs, K, Xb, ldx, M, Y, ldy, y_split_stride, rs); break;
      case 5: launch_mb<5>(g, grid, st, segs, K, Xb, ldx, M, Y, ldy, y_split_stride, rs); break;
      case 6: launch_mb<6>(g, grid, st, segs, K, Xb, ldx, M, Y, ldy, y_split_stride, rs); break;
      case 7: launch_mb<7>(g, grid, st, segs, K, Xb, ldx, M, Y, ldy, y_split_stride, rs); break;
      default: launch_mb<8>(g, grid, st, segs, K, Xb, ldx, M, Y, ldy, y_split_stride, rs); break;
    }
  } else {
    dim3 grid((N + 63) / 64, (M + 15) / 16);
    hipLaunchKernelGGL(k_gemm_f32, grid, dim3(256), 0, st, segs, N, K, (const float *)X, ldx, M, Y, ldy);
  }
  return hipGetLastError();
}

}  // namespace dbt
