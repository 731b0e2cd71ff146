// Causal attention over a prompt (primary prefill, Sec. 4.4): every prompt
// position attends to the cache positions at or before it, which the prefill
// has just written.  Query rows are prompt positions of one sequence.
#include "common.h"
#include "kernels.h"

namespace dbt {

namespace {

typedef __attribute__((address_space(3))) void lds_void;

// Causal attention over the prompt of one sequence on MFMA (bf16 cache,
// d_h = 128; Sec. 4.4, prefill through the primary path).  A workgroup owns
// 16 consecutive query positions and one KV head; wave w is query head
// g*G + w, so the G waves read the same K/V pages.  Each wave walks the page
// pairs up to its last position with the decode kernel's permuted score rows
// (lane: eight consecutive key positions of one page for one query), masks
// keys after the query (causal) and cache slots past the prompt, and keeps an
// online softmax per query row.  Tiles are issued longest first.
__global__ __launch_bounds__(1024) void k_attn_prefill_bf16(const float *Q, int ldq, int T, KVRef kv, int seq,
                                                           int n_q, uint16_t *O, int ldo) {
  constexpr int DH = 128;
  const int ntiles = (T + 15) >> 4;
  const int q0 = (ntiles - 1 - (int)blockIdx.x) * 16;  // longest tiles first
  const int g = blockIdx.y;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r = lane & 15, gq = lane >> 4;
  const int n_kv = kv.n_kv;
  const int G = n_q / n_kv;
  const int head = g * G + wave;
  const float scale = kLog2e / sqrtf((float)DH);
  const int qpos = q0 + r;  // query position of this lane's column
  const int qlast = min(q0 + 15, T - 1);

  u32x4 qf[4];
  {
    // row 0 stands in for positions past the prompt: the loads are
    // unconditional (all in flight at once), then zeroed
    const bool valid = qpos < T;
    const float *qp = Q + (size_t)(valid ? qpos : 0) * ldq + head * DH + gq * 8;
    float x[4][8];
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
      for (int e = 0; e < 8; ++e) x[s][e] = qp[s * 32 + e];
    const float z = valid ? 1.f : 0.f;
#pragma unroll
    for (int s = 0; s < 4; ++s)
      qf[s] = u32x4{pack2(x[s][0] * z, x[s][1] * z), pack2(x[s][2] * z, x[s][3] * z), pack2(x[s][4] * z, x[s][5] * z),
                    pack2(x[s][6] * z, x[s][7] * z)};
  }
  const uint16_t *kbase = (const uint16_t *)kv.k;
  const uint16_t *vbase = (const uint16_t *)kv.v;
  const int *ptab = kv.page_table + (size_t)seq * kv.mpps;
  float m_run = -INFINITY, l_run = 0.f;
  floatx4 acc[8];
#pragma unroll
  for (int c = 0; c < 8; ++c) acc[c] = floatx4{0.f, 0.f, 0.f, 0.f};
  const int kpage = r >> 3, kpos = 8 * ((r >> 2) & 1) + (r & 3);
  const int vpage = gq >> 1, vpos = 8 * (gq & 1);
  const int npg = (qlast >> 4) + 1;  // pages holding keys 0..qlast
  const int npairs = (npg + 1) >> 1;
  int nid0 = ptab[0], nid1 = ptab[min(1, npg - 1)];
  for (int q = 0; q < npairs; ++q) {
    const int pg0 = 2 * q;
    const int phys0 = nid0, phys1 = nid1;
    if (q + 1 < npairs) {  // page ids of the next pair
      nid0 = ptab[pg0 + 2];
      nid1 = ptab[min(pg0 + 3, npg - 1)];
    }
    const int kphys = kpage ? phys1 : phys0;
    const int vphys = vpage ? phys1 : phys0;
    const uint16_t *kp = kbase + ((size_t)kphys * n_kv + g) * 16 * DH + kpos * DH + gq * 8;
    const uint16_t *vp = vbase + ((size_t)vphys * n_kv + g) * DH * 16 + r * 16 + vpos;
    u32x4 ka[4], kb[4], vf[8];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      ka[s] = *(const u32x4 *)(kp + s * 32);
      kb[s] = *(const u32x4 *)(kp + 4 * DH + s * 32);
    }
#pragma unroll
    for (int c = 0; c < 8; ++c) vf[c] = *(const u32x4 *)(vp + c * 16 * 16);
    floatx4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      s0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, ka[s]),
                                                   __builtin_bit_cast(bf16x8, qf[s]), s0, 0, 0, 0);
      s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, kb[s]),
                                                   __builtin_bit_cast(bf16x8, qf[s]), s1, 0, 0, 0);
    }
    // key position of this lane's first score; keys after the query are masked
    const int kp0 = (pg0 + vpage) * 16 + vpos;
    const bool page_ok = pg0 + vpage < npg;
    float sc[8];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      sc[i] = (page_ok && kp0 + i <= qpos) ? s0[i] * scale : -INFINITY;
      sc[4 + i] = (page_ok && kp0 + 4 + i <= qpos) ? s1[i] * scale : -INFINITY;
    }
    float mt = sc[0];
#pragma unroll
    for (int i = 1; i < 8; ++i) mt = fmaxf(mt, sc[i]);
    mt = fmaxf(mt, __shfl_xor(mt, 16, 64));
    mt = fmaxf(mt, __shfl_xor(mt, 32, 64));
    const float m_new = fmaxf(m_run, mt);
    // a query row with no key yet in this pair keeps m = -inf: use 0 as the base
    const float m_use = m_new == -INFINITY ? 0.f : m_new;
    float p[8];
    float ps = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      p[i] = exp2f(sc[i] - m_use);
      ps += p[i];
    }
    if (__any(m_new > m_run)) {
      const float corr = m_run == -INFINITY ? 0.f : exp2f(m_run - m_new);
      l_run *= corr;
#pragma unroll
      for (int c = 0; c < 8; ++c) acc[c] = acc[c] * corr;
    }
    l_run += ps;
    m_run = m_new;
    const u32x4 pf = u32x4{pack2(p[0], p[1]), pack2(p[2], p[3]), pack2(p[4], p[5]), pack2(p[6], p[7])};
    // cache slots past the prompt (or a missing second page) may hold stale values
    const int nv = page_ok ? min(16, T - (pg0 + vpage) * 16) : 0;
    if (__any(nv < 16)) {
#pragma unroll
      for (int c = 0; c < 8; ++c) vf[c] = mask8(vf[c], vpos, nv);
    }
#pragma unroll
    for (int c = 0; c < 8; ++c)
      acc[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, vf[c]),
                                                       __builtin_bit_cast(bf16x8, pf), acc[c], 0, 0, 0);
  }
  l_run += __shfl_xor(l_run, 16, 64);
  l_run += __shfl_xor(l_run, 32, 64);
  if (qpos < T) {
    const float inv = 1.f / l_run;
    uint16_t *o = O + (size_t)qpos * ldo + head * DH;
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      const int dh = c * 16 + 4 * gq;
      *(u32x2 *)(o + dh) = u32x2{pack2(acc[c][0] * inv, acc[c][1] * inv), pack2(acc[c][2] * inv, acc[c][3] * inv)};
    }
  }
}

// Longest prompt (in 16-position pages) of the LDS-shared prefill kernel.
constexpr int kPrefillMaxPages = 1024;
// Growth of a row's score maximum (base 2) that moves its softmax base.
constexpr float kLazyMargin = 8.f;

// Causal attention over the prompt of one sequence on MFMA, K/V shared
// through LDS (bf16 cache, d_h = 128, G = n_q/n_kv dividing 16).  A
// workgroup of 16 waves covers 256/G positions of all G query heads of KV
// head g: wave w computes head g*G + (w % G) for positions
// q0 + 16*(w / G) .. +15.  Each pair of K/V pages (32 keys, 16 KB) is loaded
// once per workgroup straight into LDS (one 1 KB load per wave), two pairs
// per stage into one of two sets of buffers while the other set is
// multiplied, so every key/value is fetched once for 256 query rows.  The
// per-wave arithmetic is that of the decode kernel (permuted score rows,
// online softmax in base 2) with a causal mask per query row on the pairs
// that need one; a wave skips pairs that start after its last position.
// Position tiles are issued longest first.
template <int G>
__global__ __launch_bounds__(1024) void k_attn_prefill_wide(const float *Q, int ldq, int T, KVRef kv, int seq,
                                                            int n_q, uint16_t *O, int ldo) {
  constexpr int DH = 128, QB = 16 / G, TP = 16 * QB;  // query blocks per head, positions per workgroup
  constexpr int SP = 2;                                // pairs per stage (one barrier per stage)
  constexpr int PB = 2 * 16 * DH;                      // elements of one pair buffer (two pages)
  // Two sets of SP pair buffers, separate arrays so that the loads filling
  // one set are told apart from the reads of the other.  K: [page][key][dim]
  // with swizzled chunks; V: [page][dim][position].
  __shared__ __attribute__((aligned(16))) uint16_t kl0[SP * PB], kl1[SP * PB];
  __shared__ __attribute__((aligned(16))) uint16_t vl0[SP * PB], vl1[SP * PB];
  __shared__ int pid_s[kPrefillMaxPages];  // the sequence's page ids
  const int ntiles = (T + TP - 1) / TP;
  const int q0 = (ntiles - 1 - (int)blockIdx.x) * TP;  // longest tiles first
  const int g = blockIdx.y;
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);  // uniform: per-wave conditions stay scalar branches
  const int r = lane & 15, gq = lane >> 4;
  const int n_kv = kv.n_kv;
  const int head = g * G + wave % G;
  const int qw0 = q0 + 16 * (wave / G);    // first position of this wave
  const int qpos = qw0 + r;                // query position of this lane's column
  const int qw_last = min(qw0 + 15, T - 1);
  const int q_last = min(q0 + TP - 1, T - 1);
  const float scale = kLog2e / sqrtf((float)DH);

  u32x4 qf[4];
  {
    // row 0 stands in for positions past the prompt: all loads are issued
    // unconditionally, then zeroed
    const bool valid = qpos < T;
    const float *qp = Q + (size_t)(valid ? qpos : 0) * ldq + head * DH + gq * 8;
    float4 x[8];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      x[2 * s] = *(const float4 *)(qp + s * 32);
      x[2 * s + 1] = *(const float4 *)(qp + s * 32 + 4);
    }
    const float z = valid ? 1.f : 0.f;
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const float4 a = x[2 * s] * z, c = x[2 * s + 1] * z;
      qf[s] = u32x4{pack2(a.x, a.y), pack2(a.z, a.w), pack2(c.x, c.y), pack2(c.z, c.w)};
    }
  }
  const uint16_t *kbase = (const uint16_t *)kv.k;
  const uint16_t *vbase = (const uint16_t *)kv.v;
  const int *ptab = kv.page_table + (size_t)seq * kv.mpps;
  const int npg = (q_last >> 4) + 1;  // pages holding keys 0..q_last
  const int npairs = (npg + 1) >> 1;
  // page ids come from LDS: a page-table load in front of each K/V load
  // would make every load wait for all loads in flight
  for (int i = t; i < npg; i += 1024) pid_s[i] = ptab[i];
  __syncthreads();

  // K row j of a page holds its 16-byte chunk c at c ^ 2((j & 3) | ((j >> 3) << 2)):
  // the score operand reads rows {0..3, 8..11} (or {4..7, 12..15}) of both
  // pages at one chunk, which then run at the conflict-free rate (measured on
  // gfx950).  V rows (one dimension, 16 positions, 32 bytes) need no swizzle.
  auto kswz = [](int row) { return ((row & 3) | ((row >> 3) << 2)) << 1; };
  // Loads go straight from global memory into LDS (global_load_lds_dwordx4):
  // per pair every wave fills 1 KB, lane l the 16 bytes at l * 16 of it.
  // Waves 0..7: K rows 4 (w & 3) .. + 3 of page w >> 2 (each lane fetches the
  // chunk the swizzle places in its slot); waves 8..15: V dimensions
  // 32 ((w - 8) & 3) .. + 31 of page (w - 8) >> 2 (contiguous).
  const bool ld_k = wave < 8;
  const int lw = wave & 7, lpp = lw >> 2;
  uint32_t loff, ldst;  // lane's element offset in the page's head block; wave's offset in a pair buffer
  if (ld_k) {
    const int row = 4 * (lw & 3) + (lane >> 4);
    loff = row * DH + ((lane & 15) ^ kswz(row)) * 8;
    ldst = (lpp * 16 + 4 * (lw & 3)) * DH;
  } else {
    loff = 32 * (lw & 3) * 16 + lane * 8;
    ldst = (lpp * DH + 32 * (lw & 3)) * 16;
  }
  // pair p (a pair past the last, or a missing second page, re-reads the
  // last page: such data is never used unmasked)
  auto dma = [&](int p, uint16_t *kb, uint16_t *vb) __attribute__((always_inline)) {
    const int phys = pid_s[min(2 * min(p, npairs - 1) + lpp, npg - 1)];
    const size_t blk = ((size_t)phys * n_kv + g) * (16 * DH);  // a page's K or V block of head g
    if (ld_k)
      __builtin_amdgcn_global_load_lds((const void *)(kbase + blk + loff), (lds_void *)(kb + ldst), 16, 0, 0);
    else
      __builtin_amdgcn_global_load_lds((const void *)(vbase + blk + loff), (lds_void *)(vb + ldst), 16, 0, 0);
  };

  float m_run = -INFINITY;
  // the softmax denominator of each query row: one more value MFMA with V = 1
  // sums the same bf16 probabilities that weight the values (every row of the
  // result holds the sum of its column's query)
  floatx4 acc_l = floatx4{0.f, 0.f, 0.f, 0.f};
  const u32x4 ones = u32x4{0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u};
  floatx4 acc[8];
#pragma unroll
  for (int c = 0; c < 8; ++c) acc[c] = floatx4{0.f, 0.f, 0.f, 0.f};
  const int kpage = r >> 3, kpos = 8 * ((r >> 2) & 1) + (r & 3);
  const int vpage = gq >> 1, vpos = 8 * (gq & 1);

  // Scores of pair p (two MFMA chains over d_h); false when every key of
  // the pair comes after this wave's last position (uniform over the wave).
  auto pair_scores = [&](int p, const uint16_t *kb, floatx4 &s0, floatx4 &s1) __attribute__((always_inline)) {
    if (2 * p * 16 > qw_last) return false;
    u32x4 ka[4], kc[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      ka[s] = *(const u32x4 *)&kb[(kpage * 16 + kpos) * DH + ((s * 4 + gq) ^ kswz(kpos)) * 8];
      kc[s] = *(const u32x4 *)&kb[(kpage * 16 + kpos + 4) * DH + ((s * 4 + gq) ^ kswz(kpos + 4)) * 8];
    }
    s0 = floatx4{0.f, 0.f, 0.f, 0.f};
    s1 = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      s0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, ka[s]),
                                                   __builtin_bit_cast(bf16x8, qf[s]), s0, 0, 0, 0);
      s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, kc[s]),
                                                   __builtin_bit_cast(bf16x8, qf[s]), s1, 0, 0, 0);
    }
    return true;
  };
  // Online softmax over pair p's scores, then the value MFMAs.
  auto pair_finish = [&](int p, const uint16_t *vb, const floatx4 &s0, const floatx4 &s1) __attribute__((always_inline)) {
    const int pg0 = 2 * p;
    // value operands first: their LDS reads run under the softmax
    u32x4 vf[8];
#pragma unroll
    for (int c = 0; c < 8; ++c) vf[c] = *(const u32x4 *)&vb[(vpage * DH + c * 16 + r) * 16 + vpos];
    // every key of the pair precedes every query of the wave (uniform
    // over the wave): no causal mask
    const bool full = (pg0 + 2) * 16 <= qw0 + 1;
    // key position of this lane's first score; keys after the query are masked
    const int kp0 = (pg0 + vpage) * 16 + vpos;
    float sc[8];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      sc[i] = s0[i];
      sc[4 + i] = s1[i];
    }
    if (!full) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        if (kp0 + i > qpos) sc[i] = -INFINITY;
        if (kp0 + 4 + i > qpos) sc[4 + i] = -INFINITY;
      }
    }
    float mt = sc[0];
#pragma unroll
    for (int i = 1; i < 8; ++i) mt = fmaxf(mt, sc[i]);
    // scores in base 2: s * scale (scale > 0, so the maximum commutes)
    // Lazy rescaling: a row's base m moves only when the pair's maximum
    // exceeds it by more than kLazyMargin (base 2), so every score seen so
    // far stays <= m + kLazyMargin, the exponentials stay <= 2^kLazyMargin
    // and the accumulators are rescaled a few times per row instead of
    // whenever the maximum grows; output = acc / l with the same base, exact
    // up to rounding.  A row with no key yet keeps m = -inf (any finite
    // maximum then moves it).
    const float mt_s = rows4_max(mt) * scale;
    const bool grow = mt_s > m_run + kLazyMargin;
    const float m_new = grow ? mt_s : m_run;
    // a query row with no key yet keeps m = -inf: use 0 as the base
    const float m_use = m_new == -INFINITY ? 0.f : m_new;
    float pr[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) pr[i] = __builtin_amdgcn_exp2f(fmaf(sc[i], scale, -m_use));
    if (__any(grow)) {
      const float corr = m_run == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m_run - m_new);  // 1 where m stayed
      acc_l = acc_l * corr;
#pragma unroll
      for (int c = 0; c < 8; ++c) acc[c] = acc[c] * corr;
    }
    m_run = m_new;
    const u32x4 pf = u32x4{pack2(pr[0], pr[1]), pack2(pr[2], pr[3]), pack2(pr[4], pr[5]), pack2(pr[6], pr[7])};
    acc_l = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, ones), __builtin_bit_cast(bf16x8, pf),
                                                    acc_l, 0, 0, 0);
    // the last pair of the prompt: value slots at positions >= T (stale
    // cache slots, a missing second page) are zeroed, since 0 * NaN is NaN
    if ((pg0 + 2) * 16 > T) {
#pragma unroll
      for (int c = 0; c < 8; ++c) vf[c] = mask8(vf[c], kp0, T);
    }
#pragma unroll
    for (int c = 0; c < 8; ++c)
      acc[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, vf[c]),
                                                       __builtin_bit_cast(bf16x8, pf), acc[c], 0, 0, 0);
  };
  // Both pairs' scores first: the first pair's softmax (VALU) then runs
  // while the second pair's score MFMAs are in flight, and its value MFMAs
  // while the second pair's softmax runs.
  auto stage = [&](int st, const uint16_t *kb, const uint16_t *vb) __attribute__((always_inline)) {
    static_assert(SP == 2, "two pairs per stage");
    floatx4 a0, a1, b0, b1;
    const bool act_a = pair_scores(st * SP, kb, a0, a1);
    const bool act_b = pair_scores(st * SP + 1, kb + PB, b0, b1);
    if (act_a) pair_finish(st * SP, vb, a0, a1);
    if (act_b) pair_finish(st * SP + 1, vb + PB, b0, b1);
  };

  // Stage st: this wave's loads of stage st are waited for at the barrier
  // (then the stage is in LDS and every wave has finished stage st - 1),
  // stage st + 1 is loaded into the set stage st - 1 used, stage st is
  // multiplied.  The loop runs in pairs of stages so each set is known at
  // compile time; a stage past the last is loaded but never read.
  const int nstages = (npairs + SP - 1) / SP;
#pragma unroll
  for (int j = 0; j < SP; ++j) dma(j, kl0 + j * PB, vl0 + j * PB);
  for (int st = 0; st < nstages; st += 2) {
    __syncthreads();
#pragma unroll
    for (int j = 0; j < SP; ++j) dma((st + 1) * SP + j, kl1 + j * PB, vl1 + j * PB);
    __builtin_amdgcn_sched_barrier(0);
    stage(st, kl0, vl0);
    if (st + 1 < nstages) {  // uniform
      __syncthreads();
#pragma unroll
      for (int j = 0; j < SP; ++j) dma((st + 2) * SP + j, kl0 + j * PB, vl0 + j * PB);
      __builtin_amdgcn_sched_barrier(0);
      stage(st + 1, kl1, vl1);
    }
  }
  __syncthreads();  // no load into LDS outlives the workgroup
  const float l_run = acc_l[0];
  if (qpos < T) {
    const float inv = 1.f / l_run;
    uint16_t *o = O + (size_t)qpos * ldo + head * DH;
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      const int dh = c * 16 + 4 * gq;
      *(u32x2 *)(o + dh) = u32x2{pack2(acc[c][0] * inv, acc[c][1] * inv), pack2(acc[c][2] * inv, acc[c][3] * inv)};
    }
  }
}

// Causal attention over the prompt of one sequence: workgroup per
// (position t, KV head), keys 0..t in chunks of 256 with an online softmax.
template <typename T>
__global__ __launch_bounds__(256) void k_attn_prefill(const float *Q, int ldq, KVRef kv, int seq, int n_q,
                                                      T *O, int ldo) {
  constexpr int CH = 256;
  __shared__ float qs[16][128];
  __shared__ float sc[16][CH];
  __shared__ float red[16];
  const int t = blockIdx.x, g = blockIdx.y;
  const int n_kv = kv.n_kv, DH = kv.d_h;
  const int G = n_q / n_kv;
  const float scale = kLog2e / sqrtf((float)DH);
  const T *kb = (const T *)kv.k;
  const T *vb = (const T *)kv.v;
  const int *ptab = kv.page_table + (size_t)seq * kv.mpps;
  for (int e = threadIdx.x; e < G * DH; e += blockDim.x)
    qs[e / DH][e % DH] = Q[(size_t)t * ldq + (g * G + e / DH) * DH + e % DH];
  float acc[8], mrun[16], lrun[16];
  for (int k = 0; k < 8; ++k) acc[k] = 0.f;
  for (int j = 0; j < 16; ++j) { mrun[j] = -INFINITY; lrun[j] = 0.f; }
  const int nel = G * DH;  // <= 2048: thread owns elements threadIdx.x + 256k
  for (int c0 = 0; c0 <= t; c0 += CH) {
    const int nk = min(CH, t + 1 - c0);
    __syncthreads();
    if ((int)threadIdx.x < nk) {
      const int pos = c0 + threadIdx.x;
      const T *kr = kb + (((size_t)ptab[pos >> 4] * n_kv + g) * 16 + (pos & 15)) * DH;
      for (int j = 0; j < G; ++j) {
        float s = 0.f;
        for (int dh = 0; dh < DH; ++dh) s = fmaf(ld<T>(kr, dh), qs[j][dh], s);
        sc[j][threadIdx.x] = s * scale;
      }
    }
    __syncthreads();
    float corr[16];
    for (int j = 0; j < G; ++j) {
      float mx = -INFINITY;
      for (int k = threadIdx.x; k < nk; k += blockDim.x) mx = fmaxf(mx, sc[j][k]);
      mx = block_max(mx, red);
      const float mn = fmaxf(mrun[j], mx);
      corr[j] = exp2f(mrun[j] - mn);
      float l = 0.f;
      __syncthreads();
      for (int k = threadIdx.x; k < nk; k += blockDim.x) {
        const float pv = exp2f(sc[j][k] - mn);
        sc[j][k] = pv;
        l += pv;
      }
      l = block_sum(l, red);
      lrun[j] = lrun[j] * corr[j] + l;
      mrun[j] = mn;
    }
    __syncthreads();
    for (int k = 0; k < 8; ++k) {
      const int e = threadIdx.x + 256 * k;
      if (e >= nel) break;
      const int j = e / DH, dh = e % DH;
      float o = acc[k] * corr[j];
      for (int kk = 0; kk < nk; ++kk) {
        const int pos = c0 + kk;
        o = fmaf(sc[j][kk], ld<T>(vb, (((size_t)ptab[pos >> 4] * n_kv + g) * DH + dh) * 16 + (pos & 15)), o);
      }
      acc[k] = o;
    }
  }
  for (int k = 0; k < 8; ++k) {
    const int e = threadIdx.x + 256 * k;
    if (e >= nel) break;
    const int j = e / DH, dh = e % DH;
    st<T>(O, (size_t)t * ldo + (g * G + j) * DH + dh, acc[k] / lrun[j]);
  }
}

}  // namespace

hipError_t launch_attn_prefill(const float *Q, int ldq, int T, KVRef kv, int seq, int n_q, int dtype, void *O,
                               int ldo, hipStream_t st) {
  const int G = n_q / kv.n_kv;
  if (dtype == 1 && kv.d_h == 128 && G >= 1 && G <= 16) {
    dim3 grid((T + 15) / 16, kv.n_kv);
    switch ((T + 15) / 16 <= kPrefillMaxPages && ldq % 4 == 0 ? G : 0) {  // K/V shared by 16 waves through LDS when G divides 16
      case 1: case 2: case 4: case 8: case 16: {
        const int tp = 256 / G;  // positions per workgroup
        const dim3 wgrid((T + tp - 1) / tp, kv.n_kv);
        if (G == 1) hipLaunchKernelGGL(k_attn_prefill_wide<1>, wgrid, dim3(1024), 0, st, Q, ldq, T, kv, seq, n_q, (uint16_t *)O, ldo);
        else if (G == 2) hipLaunchKernelGGL(k_attn_prefill_wide<2>, wgrid, dim3(1024), 0, st, Q, ldq, T, kv, seq, n_q, (uint16_t *)O, ldo);
        else if (G == 4) hipLaunchKernelGGL(k_attn_prefill_wide<4>, wgrid, dim3(1024), 0, st, Q, ldq, T, kv, seq, n_q, (uint16_t *)O, ldo);
        else if (G == 8) hipLaunchKernelGGL(k_attn_prefill_wide<8>, wgrid, dim3(1024), 0, st, Q, ldq, T, kv, seq, n_q, (uint16_t *)O, ldo);
        else hipLaunchKernelGGL(k_attn_prefill_wide<16>, wgrid, dim3(1024), 0, st, Q, ldq, T, kv, seq, n_q, (uint16_t *)O, ldo);
        break;
      }
      default:
        hipLaunchKernelGGL(k_attn_prefill_bf16, grid, dim3(64 * G), 0, st, Q, ldq, T, kv, seq, n_q, (uint16_t *)O, ldo);
    }
    return hipGetLastError();
  }
  dim3 grid(T, kv.n_kv);
  if (dtype == 1)
    hipLaunchKernelGGL(k_attn_prefill<uint16_t>, grid, dim3(256), 0, st, Q, ldq, kv, seq, n_q, (uint16_t *)O, ldo);
  else
    hipLaunchKernelGGL(k_attn_prefill<float>, grid, dim3(256), 0, st, Q, ldq, kv, seq, n_q, (float *)O, ldo);
  return hipGetLastError();
}

}  // namespace dbt
