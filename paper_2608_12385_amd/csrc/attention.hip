// Grouped shared-KV decode attention (Sec. 4.1, Eqs. (9) and (12); Sec. 4.4
// "Decode": both attentions read the same primary cache).
//
// A workgroup owns one (sequence, KV head, split of the cache).  Its query
// rows are the G primary heads of that KV head followed by the G branch heads
// (2G <= 16), so each K/V page is read once for both paths.  Scores and the
// value sum run on MFMA (v_mfma_f32_16x16x32_bf16), one pair of 16-position
// pages per step.  Scores are computed as S = K Q^T by two MFMAs whose 16
// "rows" are a chosen set of positions of the pair: the first covers
// positions 8h+0..3 of page p in rows 4(2p+h)+i, the second positions
// 8h+4..7, so after both each lane (query r, group 2p+h) holds the scores of
// eight consecutive positions 8h..8h+7 of page p.  That is exactly the
// operand layout of the value MFMA O^T = V^T P^T with reduction index
// k = 8(2p+h) + j, and with V pages stored dim-major each lane loads its V^T
// operand as one 16-byte piece.  Softmax is online per split (base-2
// exponent, running max and sum), the four waves of a workgroup merge
// through LDS, and a combine kernel merges the splits in split order.  A
// sequence of P pages is read in ceil(P / target) splits of equal size (the
// last at most one page shorter per split): a function of its own length
// only, so a row's result depends only on its own query and cache, and equal
// splits keep the workgroups of a launch equally long.
#include "common.h"
#include "kernels.h"

namespace dbt {

namespace {

// Growth of a row's score maximum (base 2) that moves its softmax base.
constexpr float kLazyMargin = 8.f;

// Split s of a sequence of npages pages: pages [*pb, *pe); false when the
// sequence has fewer splits.
__device__ __forceinline__ bool split_range(int npages, int target, int s, int *pb, int *pe) {
  const int nsplit = (npages + target - 1) / target;
  if (s >= nsplit) return false;
  const int pps = (npages + nsplit - 1) / nsplit;
  *pb = s * pps;
  *pe = min(npages, *pb + pps);
  return *pb < *pe;
}

// Factor of physical row R whose QKV projection took its rows straight from
// the step inputs (XNorm): 1/rms of the row from the per-split sums of
// squares, added in split order (1 otherwise: the sums are left as they are).
__device__ __forceinline__ float row_scale(const QKVFinish &f, int R) {
  if (!f.ss) return 1.f;
  float t = 0.f;
  for (int k = 0; k < f.ss_S; ++k) t += f.ss[(size_t)k * f.ss_ld + R];
  return 1.0f / sqrtf(t / (float)f.d_model + f.eps);
}

// Requires d_h == 128 and np*G <= 16.
// <4, false>: one split of the sequence per workgroup of four waves (at most
// 128 pages, two page ids per lane), partials merged by k_attn_combine.
// <8, false>: the same with eight waves and splits of up to 1024 pages (page
// ids staged in LDS), for long sequences: one round of longer workgroups.
// <8, true> (a.single): the whole sequence in one workgroup of eight waves
// (at most 1024 pages), the waves merged in LDS and the normalised rows
// written to a.O directly.
template <int NW, bool SINGLE>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(2))) void k_attn_decode_bf16(AttnArgs a) {
  constexpr int DH = 128;
  constexpr bool LDSIDS = NW == 8;  // page ids of the split staged in LDS (else two per lane)
  static_assert(!SINGLE || LDSIDS, "the single-workgroup kernel has eight waves");
  const int split = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  const int len = a.pos_arr[b] + 1;
  const int npages = (len + 15) >> 4;
  int pb = 0, pe = npages;
  if (SINGLE && npages > 1024) return;  // excluded by the host
  if (!SINGLE && !split_range(npages, a.pages_per_split, split, &pb, &pe)) return;
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int r = lane & 15, gq = lane >> 4;
  const int n_kv = a.kv.n_kv;
  const int G = a.n_q / n_kv;
  const int nrows = a.rows.np * G;
  const int dq = a.n_q * DH;
  const float scale = kLog2e / sqrtf((float)DH);
  // page ids of the split: lane i holds pages pb + i and pb + 64 + i
  const int *ptab = a.kv.page_table + (size_t)b * a.kv.mpps;
  __shared__ int pid_s[LDSIDS ? 1024 : 1];
  int myid0 = 0, myid1 = 0;
  u32x4 qf[4];
  // Fused finish of the QKV projection (single mode, a.fused): the workgroup
  // turns the projection's split-K slabs into its query rows (qs) and the
  // primary's new cache entry of KV head g, with the slabs added in split
  // order and the same rope_pair / couple as k_qkv_finish, so the bits equal
  // the unfused path's.
  constexpr int QLD = DH + 4;  // row pitch of qs (floats): rows start on different banks
  __shared__ float qs[16][QLD];
  if constexpr (!LDSIDS) {
    myid0 = (pb + lane < pe) ? ptab[pb + lane] : 0;
    myid1 = (pb + 64 + lane < pe) ? ptab[pb + 64 + lane] : 0;
  }
  auto page_id = [&](int j) {
    if constexpr (LDSIDS) return pid_s[j];
    else return __shfl(j < 64 ? myid0 : myid1, j & 63, 64);
  };

  // Query operand: lane (query r, group gq) holds Q[r][s*32 + gq*8 .. +8].
  // Rows past the group's queries read row 0 and are zeroed: all eight
  // loads are issued at once (a load guarded per element compiles to a
  // branch and a full wait each, 32 round trips before the first page).
  if (!a.fused) {
    const bool valid = r < nrows;
    const int path = a.rows.p0 + (valid ? r / G : 0);
    const int head = g * G + (valid ? r % G : 0);
    const float *qp = a.Q + (size_t)(path * a.rows.Bp + b) * dq + head * DH + gq * 8;
    float4 x[8];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      x[2 * s] = *(const float4 *)(qp + s * 32);
      x[2 * s + 1] = *(const float4 *)(qp + s * 32 + 4);
    }
    const float z = valid ? 1.f : 0.f;
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const float4 u = x[2 * s] * z, w = x[2 * s + 1] * z;
      qf[s] = u32x4{pack2(u.x, u.y), pack2(u.z, u.w), pack2(w.x, w.y), pack2(w.z, w.w)};
    }
  }

  const uint16_t *kbase = (const uint16_t *)a.kv.k;
  const uint16_t *vbase = (const uint16_t *)a.kv.v;

  float m_run = -INFINITY, l_run = 0.f;
  floatx4 acc[8];
#pragma unroll
  for (int c = 0; c < 8; ++c) acc[c] = floatx4{0.f, 0.f, 0.f, 0.f};

  // Score-MFMA row r of this lane: page r/8, positions 8*((r/4)&1) + (r&3)
  // (first MFMA) and +4 (second).  Value operand of this lane: page gq/2,
  // positions 8*(gq&1) .. +7.
  const int kpage = r >> 3, kpos = 8 * ((r >> 2) & 1) + (r & 3);
  const int vpage = gq >> 1, vpos = 8 * (gq & 1);
  const int npairs = (pe - pb + 1) >> 1;
  const int last = pe - pb - 1;  // a missing second page re-reads the first (masked)
  // K/V of pair q into registers: each page's K (16 positions x 128) and
  // V (128 dimensions x 16) are 4 KB contiguous, read by four wave
  // instructions of 1 KB each with the non-temporal hint (whole cache lines,
  // streamed once).  raw[i], i < 8: K of page i/4, positions 4(i%4) + lane/16,
  // piece lane%16; raw[8 + i]: V of page i/4, dimensions 32(i%4) + lane/2,
  // positions 8(lane%2)..+7.  A page outside the split (pairs past the last,
  // the missing second page of an odd count) is read through an empty buffer
  // resource: zeros, no memory traffic, and no branch around the loads.
  const int pg_last = pe - pb;
  auto load_pair = [&](int q, u32x4 (&raw)[16], bool from_table, bool live = true) __attribute__((always_inline)) {
    const int j0 = 2 * q, j1 = 2 * q + 1;
    const int phys0 = __builtin_amdgcn_readfirstlane(from_table ? ptab[pb + min(j0, last)] : page_id(min(j0, last)));
    const int phys1 = __builtin_amdgcn_readfirstlane(from_table ? ptab[pb + min(j1, last)] : page_id(min(j1, last)));
    const size_t o0 = ((size_t)phys0 * n_kv + g) * 16 * DH, o1 = ((size_t)phys1 * n_kv + g) * 16 * DH;
    const int n0 = __builtin_amdgcn_readfirstlane(live && j0 < pg_last ? 16 * DH * 2 : 0);
    const int n1 = __builtin_amdgcn_readfirstlane(live && j1 < pg_last ? 16 * DH * 2 : 0);
    const auto rk0 = buf_rsrc(kbase + o0, n0), rk1 = buf_rsrc(kbase + o1, n1);
    const auto rv0 = buf_rsrc(vbase + o0, n0), rv1 = buf_rsrc(vbase + o1, n1);
    // K pages first, then V: staging waits for the K registers while the V
    // loads are still in flight (interleaved, the last K load came after
    // most V loads; 1.3 us less per benchmark step, both builds timed
    // alternately on one GPU)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      raw[i] = buf_load_nt(rk0, i * 1024 + lane * 16);
      raw[4 + i] = buf_load_nt(rk1, i * 1024 + lane * 16);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      raw[8 + i] = buf_load_nt(rv0, i * 1024 + lane * 16);
      raw[12 + i] = buf_load_nt(rv1, i * 1024 + lane * 16);
    }
  };
  // Operand layouts through the wave's LDS region (8 KB, K then V).  K: row
  // R = 16 page + position (256 bytes), piece p in slot p ^ kswz(R), so the
  // 16 rows one operand read touches (4 positions x 2 halves x 2 pages) fall
  // in distinct slots.  V: slot 2 (128 page + dim) + (half ^ bit 3 of dim),
  // so 16 consecutive dimensions at one half fall in distinct banks.
  __shared__ u32x4 kvt[NW][512];
  u32x4 *reg = kvt[wave];
  auto kswz = [](int R) { return (R & 15) ^ ((R >> 4) << 2); };
  auto stage = [&](const u32x4 (&raw)[16], u32x4 (&ka)[4], u32x4 (&kb)[4], u32x4 (&vf)[8])
      __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int R = (i >> 2) * 16 + (i & 3) * 4 + (lane >> 4);
      reg[R * 16 + ((lane & 15) ^ kswz(R))] = raw[i];
    }
    wave_lds_fence();
    const int RA = kpage * 16 + kpos, RB = RA + 4;
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      ka[s] = reg[RA * 16 + ((s * 4 + gq) ^ kswz(RA))];
      kb[s] = reg[RB * 16 + ((s * 4 + gq) ^ kswz(RB))];
    }
    wave_lds_fence();
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int dim = (i & 3) * 32 + (lane >> 1);
      reg[((i >> 2) * 128 + dim) * 2 + ((lane & 1) ^ ((dim >> 3) & 1))] = raw[8 + i];
    }
    wave_lds_fence();
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      const int dim = r + 16 * c;
      vf[c] = reg[(vpage * 128 + dim) * 2 + ((gq & 1) ^ ((dim >> 3) & 1))];
    }
    wave_lds_fence();
  };
  auto pair = [&](int q, const u32x4 (&ka)[4], const u32x4 (&kb)[4], u32x4 (&vf)[8]) __attribute__((always_inline)) {
    const int pg0 = pb + 2 * q;  // first page of the pair
    floatx4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      s0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, ka[s]),
                                                   __builtin_bit_cast(bf16x8, qf[s]), s0, 0, 0, 0);
      s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, kb[s]),
                                                   __builtin_bit_cast(bf16x8, qf[s]), s1, 0, 0, 0);
    }
    // lane (query r, gq) now holds positions vpos + 0..3 (s0) and vpos + 4..7
    // (s1) of page vpage of the pair
    // valid positions of that page (<= 0: none; a page past the split's end is not this pair's)
    const int nv = pg0 + vpage < pe ? min(16, len - (pg0 + vpage) * 16) : 0;
    float sc[8];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      sc[i] = (vpos + i < nv) ? s0[i] * scale : -INFINITY;
      sc[4 + i] = (vpos + 4 + i < nv) ? s1[i] * scale : -INFINITY;
    }
    float mt = sc[0];
#pragma unroll
    for (int i = 1; i < 8; ++i) mt = fmaxf(mt, sc[i]);
    mt = rows4_max(mt);
    // Lazy rescaling: a row's base m moves only when the pair's maximum
    // exceeds it by more than kLazyMargin (base 2), so the exponentials stay
    // <= 2^kLazyMargin and the running sums are rescaled a few times per row
    // (every pair a wave takes holds a valid position, so m is finite after
    // its first pair; the wave merge below works for any common base).
    const bool grow = mt > m_run + kLazyMargin;
    const float m_new = grow ? mt : m_run;
    float p[8];
    float ps = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      p[i] = __builtin_amdgcn_exp2f(sc[i] - m_new);
      ps += p[i];
    }
    // rescale the running sums only when some row's base moved (wave-uniform
    // test; a factor of exactly 1 for the other rows)
    if (__any(grow)) {
      const float corr = __builtin_amdgcn_exp2f(m_run - m_new);
      l_run *= corr;
#pragma unroll
      for (int c = 0; c < 8; ++c) acc[c] = acc[c] * corr;
    }
    l_run += ps;
    m_run = m_new;
    const u32x4 pf = u32x4{pack2(p[0], p[1]), pack2(p[2], p[3]), pack2(p[4], p[5]), pack2(p[6], p[7])};
    // positions past the end may hold stale values: zero them (0 * NaN)
    if (__any(nv < 16)) {
#pragma unroll
      for (int c = 0; c < 8; ++c) vf[c] = mask8(vf[c], vpos, nv);
    }
#pragma unroll
    for (int c = 0; c < 8; ++c)
      acc[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, vf[c]),
                                                       __builtin_bit_cast(bf16x8, pf), acc[c], 0, 0, 0);
  };
  // One register set of loaded pages per wave: once a pair is staged into
  // LDS, the wave's next pair loads while this one is multiplied (eight
  // waves x 16 KB in flight per workgroup).  The scheduling barrier keeps
  // the loads in front of the multiplies.
  u32x4 raw[16];
  {
    // Fused finish (a.fused): thread t < 64 G finishes the rotary pair
    // (i, i + 64) of query head g G + t / 64 on every path of the call (every
    // split of a sequence computes its queries); threads 64 G .. 64 G + 191
    // of the workgroup that holds the sequence's last page append the
    // primary's key pair / value dimension of KV head g.  All loads a thread
    // needs (its columns' slabs, the angle, the coupling, the cache page) are
    // issued before the wave's first page pair, which is requested from the
    // page table directly unless it holds the appended position; then the
    // sums wait only for the older loads and the pages stay in flight.
    // Append threads beyond the workgroup (four waves) take a second pass.
    const QKVFinish &f = a.fin;
    const int t = threadIdx.x, pos = len - 1, np = a.rows.np;
    const bool prim = f.mode != MODE_BRANCH;  // then path p0 = 0 is the primary
    const bool appends = a.fused && prim && pe == npages;
    const int hh = t / (DH / 2), i = t % (DH / 2), u = t - G * (DH / 2);
    const int c0 = (g * G + hh) * DH + i, c1 = c0 + DH / 2;
    const int dkv = n_kv * DH;
    auto at = [&](int path, int col) { return (size_t)(path * a.rows.Bp + b) * f.ldp + col; };
    int ncol = 0;
    size_t idx[4] = {0, 0, 0, 0};
    if (a.fused) {
      if (u < 0) {
#pragma unroll
        for (int pp = 0; pp < 2; ++pp)
          if (pp < np) {
            idx[2 * pp] = at(a.rows.p0 + pp, c0);
            idx[2 * pp + 1] = at(a.rows.p0 + pp, c1);
          }
        ncol = 2 * min(np, 2);
      } else if (appends && u < DH / 2) {
        idx[0] = at(0, dq + g * DH + u);
        idx[1] = at(0, dq + g * DH + u + DH / 2);
        ncol = 2;
      } else if (appends && u < DH / 2 + DH) {
        idx[0] = at(0, dq + dkv + g * DH + u - DH / 2);
        ncol = 1;
      }
    }
    // slabs 0..7 of the thread's columns, as 32 unconditional loads (a loop
    // or a guarded load here would wait for every outstanding load before
    // the first page request): slabs past S re-read slab S - 1 and columns
    // past ncol column 0, and neither is added below
#pragma unroll
    for (int j = 1; j < 4; ++j)
      if (j >= ncol) idx[j] = idx[0];
    float v[8][4];
    if (ncol > 0) {
#pragma unroll
      for (int k = 0; k < 8; ++k)
#pragma unroll
        for (int j = 0; j < 4; ++j) v[k][j] = f.part[min(k, f.S - 1) * f.split_stride + idx[j]];
    }
    // rows from the step inputs (f.ss): the row sums of squares of the
    // thread's rows (path p0 + pp; the appended entry is the primary's),
    // eight splits as unconditional loads like the slabs
    float sv[2][8];
    const int srow0 = a.rows.p0 * a.rows.Bp + b, srow1 = srow0 + a.rows.Bp;
    if (ncol > 0 && f.ss) {
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        sv[0][k] = f.ss[(size_t)min(k, f.ss_S - 1) * f.ss_ld + srow0];
        sv[1][k] = f.ss[(size_t)min(k, f.ss_S - 1) * f.ss_ld + (u < 0 && np > 1 ? srow1 : srow0)];
      }
    }
    float2 csi = make_float2(0.f, 0.f), aa = make_float2(0.f, 0.f), q1 = make_float2(0.f, 0.f);
    int page = 0;
    if (ncol > 0) {
      csi = f.rope[(size_t)pos * (DH / 2) + (u < 0 ? i : u % (DH / 2))];
      if (u < 0 && np + (prim ? 0 : 1) > 1) aa = make_float2(f.a[c0], f.a[c1]);
      if (u < 0 && !prim) q1 = make_float2(f.Q1_in[(size_t)b * dq + c0], f.Q1_in[(size_t)b * dq + c1]);
      if (u >= 0) page = ptab[pos >> 4];
    }
    const int pid0 = LDSIDS && t < pe - pb ? ptab[pb + t] : 0;
    const bool early = wave < npairs && (!appends || pb + 2 * wave + 1 < npages - 1);
    // issued by every wave (empty resources when not early: no traffic), so
    // that the waits below count the same loads on every path
    load_pair(wave, raw, true, early);
    if (ncol > 0) {
      // split-K sums in split order, as psum adds them (adding +0 for the
      // slabs past S leaves the bits alone: a sum 0 + v + ... is never -0)
      float x[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int k = 0; k < 8; ++k)
#pragma unroll
        for (int j = 0; j < 4; ++j) x[j] += k < f.S ? v[k][j] : 0.f;
      for (int k = 8; k < f.S; ++k)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          if (j < ncol) x[j] += f.part[k * f.split_stride + idx[j]];
      if (f.ss) {
        // RMSNorm of the input row applied after the projection (see XNorm)
        float rs[2];
#pragma unroll
        for (int pp = 0; pp < 2; ++pp) {
          float t2 = 0.f;
#pragma unroll
          for (int k = 0; k < 8; ++k) t2 += k < f.ss_S ? sv[pp][k] : 0.f;
          for (int k = 8; k < f.ss_S; ++k) t2 += f.ss[(size_t)k * f.ss_ld + (pp ? srow1 : srow0)];
          rs[pp] = 1.0f / sqrtf(t2 / (float)f.d_model + f.eps);
        }
        x[0] *= rs[0];
        x[1] *= rs[0];
        x[2] *= rs[1];
        x[3] *= rs[1];
      }
      if (u < 0) {
        if (prim) {
          // Q1 = RoPE(.) (Eqs. (8)-(9)), kept for a later branch pass when asked
          q1 = rope_pair(x[0], x[1], csi);
          qs[hh][i] = q1.x;
          qs[hh][i + DH / 2] = q1.y;
          const Retain &rt = f.ret;
          if (rt.ptr && (rt.src_row < 0 || rt.src_row == b)) {
            float *kp = rt.ptr + (size_t)(rt.src_row < 0 ? b : rt.dst_row) * dq;
            kp[c0] = q1.x;
            kp[c1] = q1.y;
          }
        }
        // branch rows: Q2~ = RoPE(.) + a * Q1 (Eqs. (10)-(11)); paths past
        // the first two of the call (several branches) sum their slabs here
#pragma unroll
        for (int pp = 0; pp < 2; ++pp)
          if (pp < np && !(prim && pp == 0)) {
            const float2 q2 = rope_pair(x[2 * pp], x[2 * pp + 1], csi);
            qs[pp * G + hh][i] = couple(aa.x, q1.x, q2.x);
            qs[pp * G + hh][i + DH / 2] = couple(aa.y, q1.y, q2.y);
          }
        for (int pp = 2; pp < np; ++pp) {
          const float rsp = row_scale(f, (a.rows.p0 + pp) * a.rows.Bp + b);
          const float2 q2 = rope_pair(psum(f.part, f.split_stride, f.S, at(a.rows.p0 + pp, c0)) * rsp,
                                      psum(f.part, f.split_stride, f.S, at(a.rows.p0 + pp, c1)) * rsp, csi);
          qs[pp * G + hh][i] = couple(aa.x, q1.x, q2.x);
          qs[pp * G + hh][i + DH / 2] = couple(aa.y, q1.y, q2.y);
        }
      } else if (u < DH / 2) {
        // the primary appends K = RoPE(.) and V of head g at position pos (Sec. 4.4)
        const float2 k = rope_pair(x[0], x[1], csi);
        uint16_t *kc = (uint16_t *)a.kv.k + (((size_t)page * n_kv + g) * 16 + (pos & 15)) * DH;
        kc[u] = f2bf(k.x);
        kc[u + DH / 2] = f2bf(k.y);
      } else {
        ((uint16_t *)a.kv.v)[(((size_t)page * n_kv + g) * DH + u - DH / 2) * 16 + (pos & 15)] = f2bf(x[0]);
      }
    }
    if (appends)
      for (int t2 = t + NW * 64; t2 < G * (DH / 2) + DH / 2 + DH; t2 += NW * 64) {
        const int u2 = t2 - G * (DH / 2);
        if (u2 < 0) continue;  // queries: all in the first pass (G <= NW)
        const int page2 = ptab[pos >> 4];
        const float2 cs2 = f.rope[(size_t)pos * (DH / 2) + u2 % (DH / 2)];
        const float rs0 = row_scale(f, b);
        if (u2 < DH / 2) {
          const int k0 = dq + g * DH + u2;
          const float2 k = rope_pair(psum(f.part, f.split_stride, f.S, at(0, k0)) * rs0,
                                     psum(f.part, f.split_stride, f.S, at(0, k0 + DH / 2)) * rs0, cs2);
          uint16_t *kc = (uint16_t *)a.kv.k + (((size_t)page2 * n_kv + g) * 16 + (pos & 15)) * DH;
          kc[u2] = f2bf(k.x);
          kc[u2 + DH / 2] = f2bf(k.y);
        } else {
          const float vv = psum(f.part, f.split_stride, f.S, at(0, dq + dkv + g * DH + u2 - DH / 2)) * rs0;
          ((uint16_t *)a.kv.v)[(((size_t)page2 * n_kv + g) * DH + u2 - DH / 2) * 16 + (pos & 15)] = f2bf(vv);
        }
      }
    if constexpr (LDSIDS) {
      if (threadIdx.x < pe - pb) pid_s[threadIdx.x] = pid0;
      for (int i = threadIdx.x + NW * 64; i < pe - pb; i += NW * 64) pid_s[i] = ptab[pb + i];
    }
    if (LDSIDS || a.fused) __syncthreads();  // page ids and query rows in LDS, the appended entry written
    if (!early && wave < npairs) load_pair(wave, raw, false);
  }
  if (a.fused) {
    // query operand from the rows staged above (rows past the group's are zero)
    const float z = r < nrows ? 1.f : 0.f;
    const int rq = r < nrows ? r : 0;
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const float4 u = *(const float4 *)&qs[rq][s * 32 + gq * 8] * z;
      const float4 w = *(const float4 *)&qs[rq][s * 32 + gq * 8 + 4] * z;
      qf[s] = u32x4{pack2(u.x, u.y), pack2(u.z, u.w), pack2(w.x, w.y), pack2(w.z, w.w)};
    }
  }
  // Wave w takes pairs w + NW k.  When they do not divide evenly, the waves
  // with one pair more take their last one second instead of at the end (the
  // last pair is often a single, partly filled page): its round trip then
  // overlaps the other waves' streaming rather than trailing the launch alone.
  const int per = npairs / NW, more = wave < npairs % NW && per > 0;
  auto pair_of = [&](int k) { return more && k >= 1 ? (k == 1 ? wave + per * NW : wave + (k - 1) * NW) : wave + k * NW; };
  const int cnt = per + (wave < npairs % NW ? 1 : 0);
  for (int k = 0; k < cnt; ++k) {
    u32x4 ka[4], kb[4], vf[8];
    stage(raw, ka, kb, vf);
    load_pair(k + 1 < cnt ? pair_of(k + 1) : npairs, raw, false);
    __builtin_amdgcn_sched_barrier(0);
    pair(pair_of(k), ka, kb, vf);
  }
  l_run += __shfl_xor(l_run, 16, 64);
  l_run += __shfl_xor(l_run, 32, 64);

  // merge the waves: acc holds O^T[dh = 16c + 4gq + i][query r]
  __shared__ float so[NW][DH][17];
  __shared__ float sm[NW][16], sl[NW][16];
#pragma unroll
  for (int c = 0; c < 8; ++c)
#pragma unroll
    for (int i = 0; i < 4; ++i) so[wave][c * 16 + gq * 4 + i][r] = acc[c][i];
  if (gq == 0) {
    sm[wave][r] = m_run;
    sl[wave][r] = l_run;
  }
  __syncthreads();
  const size_t obase = (((size_t)b * n_kv + g) * a.max_splits + split) * 16;
  for (int e = threadIdx.x; e < nrows * DH; e += NW * 64) {
    const int qr = e / DH, dh = e % DH;
    float mx = -INFINITY;
#pragma unroll
    for (int w = 0; w < NW; ++w) mx = fmaxf(mx, sm[w][qr]);
    float o = 0.f, l = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      if (sm[w][qr] != -INFINITY) {
        const float f = exp2f(sm[w][qr] - mx);
        o += so[w][dh][qr] * f;
        l += sl[w][qr] * f;
      }
    }
    if constexpr (SINGLE) {
      const int path = a.rows.p0 + qr / G, head = g * G + qr % G;
      ((uint16_t *)a.O)[(size_t)(path * a.rows.Bp + b) * a.ldo + head * DH + dh] = f2bf(o / l);
    } else {
      a.opart[(obase + qr) * DH + dh] = o;
      if (dh == 0) {
        a.ostat[(obase + qr) * 2 + 0] = mx;
        a.ostat[(obase + qr) * 2 + 1] = l;
      }
    }
  }
}

// fp32 cache: scores in LDS, exact two-pass softmax over the split.
__global__ __launch_bounds__(256) void k_attn_decode_f32(AttnArgs a) {
  constexpr int MAXP = 1024;  // positions per split (at most 64 pages)
  __shared__ float qs[16][128];
  __shared__ float sc[16][MAXP];
  __shared__ float red[16];
  const int split = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  const int len = a.pos_arr[b] + 1;
  const int npages = (len + 15) >> 4;
  int pb, pe;
  if (!split_range(npages, a.pages_per_split, split, &pb, &pe)) return;
  const int p_lo = pb * 16, p_hi = min(len, pe * 16);
  const int np = p_hi - p_lo;
  const int n_kv = a.kv.n_kv, DH = a.kv.d_h;
  const int G = a.n_q / n_kv;
  const int nrows = a.rows.np * G;
  const int dq = a.n_q * DH;
  const float scale = kLog2e / sqrtf((float)DH);
  const float *kb = (const float *)a.kv.k;
  const float *vb = (const float *)a.kv.v;
  const int *ptab = a.kv.page_table + (size_t)b * a.kv.mpps;
  for (int e = threadIdx.x; e < nrows * DH; e += blockDim.x) {
    const int qr = e / DH, dh = e % DH;
    const int path = a.rows.p0 + qr / G, head = g * G + qr % G;
    qs[qr][dh] = a.Q[(size_t)(path * a.rows.Bp + b) * dq + head * DH + dh];
  }
  __syncthreads();
  for (int t = threadIdx.x; t < np; t += blockDim.x) {
    const int pos = p_lo + t;
    const float *kr = kb + (((size_t)ptab[pos >> 4] * n_kv + g) * 16 + (pos & 15)) * DH;
    for (int qr = 0; qr < nrows; ++qr) {
      float s = 0.f;
      for (int dh = 0; dh < DH; ++dh) s = fmaf(kr[dh], qs[qr][dh], s);
      sc[qr][t] = s * scale;
    }
  }
  __syncthreads();
  const size_t obase = (((size_t)b * n_kv + g) * a.max_splits + split) * 16;
  for (int qr = 0; qr < nrows; ++qr) {
    float mx = -INFINITY;
    for (int t = threadIdx.x; t < np; t += blockDim.x) mx = fmaxf(mx, sc[qr][t]);
    mx = block_max(mx, red);
    float l = 0.f;
    for (int t = threadIdx.x; t < np; t += blockDim.x) {
      const float pv = exp2f(sc[qr][t] - mx);
      sc[qr][t] = pv;
      l += pv;
    }
    l = block_sum(l, red);
    if (threadIdx.x == 0) {
      a.ostat[(obase + qr) * 2 + 0] = mx;
      a.ostat[(obase + qr) * 2 + 1] = l;
    }
  }
  __syncthreads();
  for (int e = threadIdx.x; e < nrows * DH; e += blockDim.x) {
    const int qr = e / DH, dh = e % DH;
    float o = 0.f;
    for (int t = 0; t < np; ++t) {
      const int pos = p_lo + t;
      o = fmaf(sc[qr][t], vb[(((size_t)ptab[pos >> 4] * n_kv + g) * DH + dh) * 16 + (pos & 15)], o);
    }
    a.opart[(obase + qr) * DH + dh] = o;
  }
}

// Merge the splits of one (sequence, KV head) in split order and write the
// normalised head outputs to O (row path*Bp + b, column head*d_h + dh).
// One thread per (query row, 4 consecutive dims).
template <typename T>
__global__ void k_attn_combine(AttnArgs a, T *O, int ldo) {
  const int g = blockIdx.x, b = blockIdx.y;
  const int len = a.pos_arr[b] + 1;
  const int npages = (len + 15) >> 4;
  const int nsplit = (npages + a.pages_per_split - 1) / a.pages_per_split;  // as split_range
  const int n_kv = a.kv.n_kv, DH = a.kv.d_h, Q4 = DH / 4;
  const int G = a.n_q / n_kv;
  const int nrows = a.rows.np * G;
  const int e = threadIdx.x;
  if (e >= nrows * Q4) return;
  const int qr = e / Q4, d4 = e % Q4;
  const size_t base = ((size_t)b * n_kv + g) * a.max_splits;
  // (unrolled: the loads of eight splits are in flight together; a rolled
  // loop waits for each split's load before the next)
  float mx = -INFINITY;
#pragma unroll 8
  for (int s = 0; s < nsplit; ++s) mx = fmaxf(mx, a.ostat[((base + s) * 16 + qr) * 2]);
  float4 o = make_float4(0.f, 0.f, 0.f, 0.f);
  float l = 0.f;
#pragma unroll 8
  for (int s = 0; s < nsplit; ++s) {
    const size_t ix = (base + s) * 16 + qr;
    const float f = exp2f(a.ostat[ix * 2] - mx);
    const float4 v = ((const float4 *)(a.opart + ix * DH))[d4];
    o.x += v.x * f;
    o.y += v.y * f;
    o.z += v.z * f;
    o.w += v.w * f;
    l += a.ostat[ix * 2 + 1] * f;
  }
  const int path = a.rows.p0 + qr / G, head = g * G + qr % G;
  const size_t out = (size_t)(path * a.rows.Bp + b) * ldo + head * DH + d4 * 4;
  st<T>(O, out + 0, o.x / l);
  st<T>(O, out + 1, o.y / l);
  st<T>(O, out + 2, o.z / l);
  st<T>(O, out + 3, o.w / l);
}

}  // namespace

hipError_t launch_attn_decode(const AttnArgs &a, hipStream_t st) {
  // split lengths: the four-wave bf16 kernel holds two page ids per lane, the
  // eight-wave one 1024 in LDS, the fp32 one 1024 positions in LDS
  const int max_pps = a.dtype != 1 ? 64 : a.wide ? 1024 : 128;
  if (!a.single && (a.pages_per_split < 1 || a.pages_per_split > max_pps)) return hipErrorInvalidValue;
  // the fused query finish: bf16 cache, decode positions (one per
  // sequence), the same rows as the attention, every query head of a KV
  // head in the first pass (G <= waves)
  if (a.fused && !(a.dtype == 1 && a.fin.pos_arr == a.pos_arr && a.fin.d_h == 128 &&
                   a.fin.n_q == a.n_q && a.fin.n_kv == a.kv.n_kv && a.fin.rows.p0 == a.rows.p0 &&
                   a.fin.rows.np == a.rows.np && a.fin.rows.Bp == a.rows.Bp && a.fin.rows.B == a.rows.B &&
                   a.rows.np >= 1 && (a.fin.mode == MODE_BRANCH) == (a.rows.p0 >= 1) &&
                   a.n_q / a.kv.n_kv <= (a.single || a.wide ? 8 : 4)))
    return hipErrorInvalidValue;
  dim3 grid(a.max_splits, a.kv.n_kv, a.rows.B);
  if (a.dtype == 1 && a.single)
    hipLaunchKernelGGL((k_attn_decode_bf16<8, true>), dim3(1, a.kv.n_kv, a.rows.B), dim3(512), 0, st, a);
  else if (a.dtype == 1 && a.wide)
    hipLaunchKernelGGL((k_attn_decode_bf16<8, false>), grid, dim3(512), 0, st, a);
  else if (a.dtype == 1)
    hipLaunchKernelGGL((k_attn_decode_bf16<4, false>), grid, dim3(256), 0, st, a);
  else
    hipLaunchKernelGGL(k_attn_decode_f32, grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_attn_combine(const AttnArgs &a, void *O, int ldo, hipStream_t st) {
  dim3 grid(a.kv.n_kv, a.rows.B);
  const int G = a.n_q / a.kv.n_kv;
  const int threads = (a.rows.np * G * (a.kv.d_h / 4) + 63) / 64 * 64;
  if (a.dtype == 1)
    hipLaunchKernelGGL(k_attn_combine<uint16_t>, grid, dim3(threads), 0, st, a, (uint16_t *)O, ldo);
  else
    hipLaunchKernelGGL(k_attn_combine<float>, grid, dim3(threads), 0, st, a, (float *)O, ldo);
  return hipGetLastError();
}

}  // namespace dbt
