"""CPU oracle of the Decode-Branch Transformer inference path.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path imports this module;
only the tests, the smoke check and the benchmark's CPU-baseline leg do.
It shares no code with the HIP library: it receives the same seeded
parameter values (float32 arrays whose values are exactly the device's
bf16/fp32 parameters) and computes everything in float64 with NumPy.

It is written to be read against the paper (arXiv 2608.12385,
"Decode-Branch Transformers"):

* embeddings, Sec. 4, Eq. (7): S1 = RMSNorm(E1[x]), S2 = RMSNorm(E2[x]);
* asymmetric shared-KV attention, Sec. 4.1, Eqs. (8)-(12): the primary is
  plain causal self-attention; the branch forms only a query, adds a * Q1
  to it and attends to the primary keys/values;
* MLP coupling, Sec. 4.1, Eqs. (13)-(16): M1 = H1 W_D,
  H2~ = H2 + b * H1, M2 = H2~ W_D + c * M1, S <- S_bar + M;
* mixture readout, Sec. 4.2, Eqs. (17)-(18): p = softmax(z1),
  q = softmax(z2), alpha = clip(sum p^2, 0.5, 1), prediction
  alpha p + (1 - alpha) q;
* MoE routing, Sec. 3.2, Eqs. (5)-(6), router replay Sec. 4.3 Eq. (19),
  independent fan-outs k1, k2, Sec. 5 Eq. (22);
* inference schedule, Sec. 4.4: primary-only prefill writes the cache and
  keeps the final position's Q1, H1, M1; one branch evaluation at the final
  prompt position (the boundary); then continuation steps in which the
  primary appends one key/value per layer and both paths query the cache;
* compute-matched variant, App. B.3 (MoE): the branch evaluates no
  attention, A2 = g_A * A1, and its MoE output is its own routed experts
  plus g_G * G(N1), the gated primary shared-expert output (no other
  coupling term);
* more than one decode branch, App. C.1: the branch distributions are
  averaged before the mixture.

Readings taken where the paper leaves a detail open:
  R1 norm gains are shared by the two paths, one per norm site;
  R2 RMSNorm(x) = x / sqrt(mean(x^2) + eps) * gain;
  R3 rotate-half RoPE, pair (i, i + d_h/2), angle pos * theta^(-2i/d_h),
     positions 0-based and equal for both paths;
  R4 a * Q1 is added after RoPE on both queries; branch head h uses KV
     head floor(h / G) like the primary;
  R5 at step t both paths attend to positions 0..t including the key the
     primary just appended;
  R6 a final RMSNorm precedes the (untied) output matrix;
  R7 f_up is SwiGLU: SiLU(U W_gate^T) * (U W_up^T);
  R8 greedy next token = lowest index attaining the maximum of the mixture;
     with the branch off, alpha = 1;
  R9 the cache stores keys/values in the model's storage dtype (bf16 values
     are rounded to nearest even); every attention reads the stored values;
  R10 MoE: router shared by both paths; Normalize = divide by the sum;
     top-k ranks by logit with ties to the lower index; coupling b acts on
     the shared-expert intermediate, c on the whole MoE output;
  R11 pages hold 16 positions and are handed out lowest-free-id first, in
     batch order, when a sequence's length reaches a multiple of 16.
"""
from __future__ import annotations

import heapq

import numpy as np

F64 = np.float64

__all__ = [
    "rmsnorm", "rope", "silu", "softmax", "attend", "round_bf16",
    "mixture_readout", "topk", "route", "PageAllocator", "Oracle",
]


# --------------------------------------------------------------------------
# Elementary operations
# --------------------------------------------------------------------------

def rmsnorm(x, gain, eps):
    """RMSNorm over the last axis (Eq. (7) and every norm site; reading R2)."""
    x = np.asarray(x)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * gain


def rope(v, pos, theta):
    """Rotary position embedding of Eq. (8), reading R3.

    v: [..., d_h]; pos: scalar or array broadcastable to v.shape[:-1]."""
    d_h = v.shape[-1]
    half = d_h // 2
    i = np.arange(half, dtype=F64)
    inv_freq = np.power(F64(theta), -2.0 * i / d_h)
    ang = np.asarray(pos, dtype=F64)[..., None] * inv_freq
    c = np.cos(ang).astype(v.dtype)
    s = np.sin(ang).astype(v.dtype)
    x1 = v[..., :half]
    x2 = v[..., half:]
    return np.concatenate([x1 * c - x2 * s, x1 * s + x2 * c], axis=-1)


def silu(u):
    """SiLU(u) = u / (1 + exp(-u))."""
    return u / (1.0 + np.exp(-u))


def softmax(z):
    """softmax over the last axis (max-shifted)."""
    z = np.asarray(z)
    e = np.exp(z - np.max(z, axis=-1, keepdims=True))
    return e / np.sum(e, axis=-1, keepdims=True)


def attend(q, K, V):
    """One query row of scaled dot-product attention (Eq. (3)) over the keys
    it may see: weights softmax(K q / sqrt(d_h)) (max, then exp and sum in
    position order), output sum_j w_j V_j.  q: [d_h]; K, V: [T][d_h]."""
    d_h = q.shape[-1]
    s = (K @ q) / np.sqrt(F64(d_h)).astype(q.dtype)
    m = np.max(s)
    w = np.exp(s - m)
    return (w @ V) / np.sum(w)


def round_bf16(x):
    """Round to the nearest bfloat16 value, ties to even (reading R9).

    Written from the format's definition: 8 significant bits."""
    x = np.asarray(x, dtype=F64)
    m, e = np.frexp(x)                  # x = m * 2**e, 0.5 <= |m| < 1
    r = np.rint(np.ldexp(m, 8))         # 8 significant bits, half to even
    return np.ldexp(r, e - 8)


def mixture_readout(z1, z2, branch_on=True, z_branches=None):
    """Mixture readout of Sec. 4.2 (Eqs. (17)-(18)), reading R8.

    z1, z2: [V] logits.  Returns (alpha, m, next) with m the predictive
    distribution alpha p + (1 - alpha) q.  With more than one branch
    (App. C.1), pass ``z_branches`` (list of logits); q is their mean
    softmax."""
    p = softmax(z1)
    if not branch_on:
        alpha = 1.0
        m = p
    else:
        if z_branches is not None:
            q = np.mean([softmax(z) for z in z_branches], axis=0)
        else:
            q = softmax(z2)
        alpha = float(min(1.0, max(0.5, float(np.sum(p * p)))))
        m = alpha * p + (1.0 - alpha) * q
    nxt = int(np.flatnonzero(m == np.max(m))[0])
    return alpha, m, nxt


def topk(r, k):
    """Indices of the k largest router logits, ordered by logit descending,
    ties to the lower index (Eq. (5), reading R10).  Written as a full
    stable sort on (-logit, index)."""
    r = np.asarray(r)
    order = sorted(range(r.shape[0]), key=lambda e: (-r[e], e))
    return np.array(order[:k], dtype=np.int64)


def route(r, k, replay_idx=None):
    """Routing of Eq. (5)-(6) and router replay (Eq. (19)).

    Returns (indices, weights): weights are softmax(r) gathered at the
    selected indices and divided by their sum."""
    pi = softmax(r)
    idx = topk(r, k) if replay_idx is None else np.asarray(replay_idx, dtype=np.int64)
    g = pi[idx]
    return idx, g / np.sum(g)


# --------------------------------------------------------------------------
# Page allocator (reading R11)
# --------------------------------------------------------------------------

class PageAllocator:
    """Pages of ``page_size`` positions; the lowest free page id is handed
    out first.  ``table[b]`` lists sequence b's pages in position order."""

    def __init__(self, num_pages, page_size=16):
        self.num_pages = num_pages
        self.page_size = page_size
        self.free = list(range(num_pages))      # a sorted list is a min-heap
        self.table: dict[int, list[int]] = {}
        self.length: dict[int, int] = {}

    def _take(self):
        if not self.free:
            raise MemoryError("no free pages")
        return heapq.heappop(self.free)

    def pages_needed(self, length):
        return -(-length // self.page_size)

    def reserve(self, b, length):
        """Sequence b grows to ``length`` positions, taking pages as needed."""
        tab = self.table.setdefault(b, [])
        need = self.pages_needed(length) - len(tab)
        if need > len(self.free):
            raise MemoryError("no free pages")
        for _ in range(max(0, need)):
            tab.append(self._take())
        self.length[b] = max(self.length.get(b, 0), length)

    def append_one(self, b):
        """One more position for sequence b (a page is taken when the
        current length is a multiple of the page size)."""
        n = self.length.get(b, 0)
        if n % self.page_size == 0:
            self.table.setdefault(b, []).append(self._take())
        self.length[b] = n + 1
        return n

    def truncate(self, b, length):
        tab = self.table.get(b, [])
        keep = self.pages_needed(length)
        for p in tab[keep:]:
            heapq.heappush(self.free, p)
        self.table[b] = tab[:keep]
        self.length[b] = length


# --------------------------------------------------------------------------
# The model
# --------------------------------------------------------------------------

class Oracle:
    """Decode-Branch Transformer forward passes in float64.

    ``shape`` is a synth.ModelShape-like object; ``params`` maps parameter
    names (as generated by the input module) to float32 arrays.  The cache
    holds, per layer and sequence, keys and values [T][n_kv][d_h].
    """

    def __init__(self, shape, params, num_pages=1 << 20, ftype=F64):
        self.s = shape
        self.P = params
        self.ft = ftype
        self.alloc = PageAllocator(num_pages, shape.page_size)
        self.K = [dict() for _ in range(shape.n_layers)]
        self.V = [dict() for _ in range(shape.n_layers)]
        self._cache_w = {}
        self.retained = {}     # b -> dict(z1, per-layer q1/H1/M1/...) for the boundary

    # ---------------- parameter access ----------------

    def w(self, name):
        a = self._cache_w.get(name)
        if a is None:
            a = np.asarray(self.P[name]).astype(self.ft)
            if a.size * a.itemsize <= (1 << 30):
                self._cache_w[name] = a
        return a

    def lin(self, x, name):
        """x @ W^T with W stored [out][in] (converted blockwise when large)."""
        W = self.P[name]
        if W.size * 8 <= (1 << 30):
            return x @ self.w(name).T
        out = np.empty(x.shape[:-1] + (W.shape[0],), dtype=self.ft)
        blk = max(1, (1 << 25) // W.shape[1])
        for r0 in range(0, W.shape[0], blk):
            out[..., r0:r0 + blk] = x @ W[r0:r0 + blk].astype(self.ft).T
        return out

    def store(self, x):
        """Value as held in the cache (reading R9)."""
        if self.s.dtype == "bf16":
            return round_bf16(x).astype(self.ft)
        return np.asarray(x, dtype=np.float32).astype(self.ft)

    # ---------------- cache ----------------

    def length(self, b):
        return self.alloc.length.get(b, 0)

    def kv_fill(self, b, length, K_layers, V_layers):
        """Direct fill of sequence b's cache (layer-only workloads): K_layers[l]
        and V_layers[l] are [length][n_kv][d_h] arrays of stored values."""
        self.alloc.reserve(b, length)
        for l in range(self.s.n_layers):
            self.K[l][b] = np.asarray(K_layers[l]).astype(self.ft)
            self.V[l][b] = np.asarray(V_layers[l]).astype(self.ft)

    def truncate(self, b, length):
        self.alloc.truncate(b, length)
        for l in range(self.s.n_layers):
            if b in self.K[l]:
                self.K[l][b] = self.K[l][b][:length]
                self.V[l][b] = self.V[l][b][:length]

    def _append(self, l, b, pos, k, v):
        K = self.K[l].get(b)
        if K is None:
            K = np.zeros((0, self.s.n_kv_heads, self.s.head_dim), self.ft)
            V = K.copy()
        else:
            V = self.V[l][b]
        assert K.shape[0] == pos, "append position must equal cache length"
        self.K[l][b] = np.concatenate([K, self.store(k)[None]], axis=0)
        self.V[l][b] = np.concatenate([V, self.store(v)[None]], axis=0)

    # ---------------- pieces of one layer ----------------

    def embed(self, tok, path):
        """Eq. (7): RMSNorm of the path's own embedding row (path j >= 1 is
        decode branch j, table E_{j+1}; App. C.1 for j >= 2)."""
        table = f"E{path + 1}"
        e = np.asarray(self.P[table][tok]).astype(self.ft)
        return rmsnorm(e, self.w("g_emb"), self.s.rms_eps)

    def heads_attend(self, q, K, V):
        """Per-query-head attention, head h reading KV head h // G."""
        s = self.s
        G = s.n_q_heads // s.n_kv_heads
        out = np.empty_like(q)
        for h in range(s.n_q_heads):
            out[h] = attend(q[h], K[:, h // G], V[:, h // G])
        return out

    def _mlp_dense_primary(self, l, U1):
        p = f"L{l}."
        H1 = silu(self.lin(U1, p + "W_gate")) * self.lin(U1, p + "W_up")
        M1 = self.lin(H1, p + "W_down")
        return H1, M1

    def _experts(self, l, U, idx, wts):
        """sum_{e in I} w_e Expert_e(U) in ascending expert order (Eq. (6))."""
        p = f"L{l}."
        out = np.zeros(self.s.d_model, self.ft)
        for e, we in sorted(zip(idx.tolist(), wts.tolist())):
            Wg = np.asarray(self.P[p + "X_gate"][e]).astype(self.ft)
            Wu = np.asarray(self.P[p + "X_up"][e]).astype(self.ft)
            Wd = np.asarray(self.P[p + "X_down"][e]).astype(self.ft)
            h = silu(U @ Wg.T) * (U @ Wu.T)
            out = out + we * (h @ Wd.T)
        return out

    def primary_layer(self, l, b, S1, pos):
        """Primary path at one position (Eqs. (8)-(9), (13), (16)): appends the
        key/value at ``pos`` and returns the new residual plus the
        intermediates the branch reads."""
        s = self.s
        p = f"L{l}."
        N1 = rmsnorm(S1, self.w(p + "g_attn"), s.rms_eps)
        q1 = rope(self.lin(N1, p + "W_Q").reshape(s.n_q_heads, s.head_dim), pos, s.rope_theta)
        k1 = rope(self.lin(N1, p + "W_K").reshape(s.n_kv_heads, s.head_dim), pos, s.rope_theta)
        v1 = self.lin(N1, p + "W_V").reshape(s.n_kv_heads, s.head_dim)
        self._append(l, b, pos, k1, v1)
        K, V = self.K[l][b][:pos + 1], self.V[l][b][:pos + 1]
        A1 = self.lin(self.heads_attend(q1, K, V).reshape(-1), p + "W_O")
        Sb1 = S1 + A1
        U1 = rmsnorm(Sb1, self.w(p + "g_mlp"), s.rms_eps)
        inter = dict(q1=q1, A1=A1, N1=N1)
        if not s.is_moe:
            H1, M1 = self._mlp_dense_primary(l, U1)
            inter.update(H1=H1, M1=M1)
        else:
            r1 = self.lin(U1, p + "W_router")
            idx1, w1 = route(r1, s.top_k1)
            R1 = self._experts(l, U1, idx1, w1)
            if s.n_shared_experts > 0:
                Hs1 = silu(self.lin(U1, p + "S_gate")) * self.lin(U1, p + "S_up")
                G1 = self.lin(Hs1, p + "S_down")
            else:
                Hs1 = None
                G1 = np.zeros(s.d_model, self.ft)
            M1 = R1 + G1
            inter.update(H1=Hs1, M1=M1, G1=G1, r1=r1, idx1=idx1, w1=w1)
        return Sb1 + inter["M1"], inter

    def branch_layer(self, l, b, S2, pos, inter, K=None, V=None):
        """Decode branch at one position (Eqs. (10)-(12), (14)-(16)): reads the
        primary cache 0..pos and the primary intermediates; writes nothing."""
        s = self.s
        p = f"L{l}."
        if K is None:
            K, V = self.K[l][b][:pos + 1], self.V[l][b][:pos + 1]
        if s.compute_matched:
            A2 = self.w(p + "g_A") * inter["A1"]
        else:
            N2 = rmsnorm(S2, self.w(p + "g_attn"), s.rms_eps)
            q2 = rope(self.lin(N2, p + "W_Q").reshape(s.n_q_heads, s.head_dim), pos, s.rope_theta)
            q2t = q2 + self.w(p + "a").reshape(s.n_q_heads, s.head_dim) * inter["q1"]
            A2 = self.lin(self.heads_attend(q2t, K, V).reshape(-1), p + "W_O")
        Sb2 = S2 + A2
        U2 = rmsnorm(Sb2, self.w(p + "g_mlp"), s.rms_eps)
        out = dict(A2=A2)
        if not s.is_moe:
            H2 = silu(self.lin(U2, p + "W_gate")) * self.lin(U2, p + "W_up")
            H2t = H2 + self.w(p + "b") * inter["H1"]
            M2 = self.lin(H2t, p + "W_down") + self.w(p + "c") * inter["M1"]
        else:
            r2 = self.lin(U2, p + "W_router")
            if s.replay:
                idx2, w2 = route(r2, s.top_k1, replay_idx=inter["idx1"])
            else:
                idx2, w2 = route(r2, s.top_k2)
            R2 = self._experts(l, U2, idx2, w2)
            if s.compute_matched:
                # App. B.3: the branch's own routed experts plus the gated
                # primary shared-expert output, nothing else
                M2 = R2 + self.w(p + "g_G") * inter["G1"]
            else:
                if s.n_shared_experts > 0:
                    Hs2 = silu(self.lin(U2, p + "S_gate")) * self.lin(U2, p + "S_up")
                    G2 = self.lin(Hs2 + self.w(p + "b") * inter["H1"], p + "S_down")
                else:
                    G2 = np.zeros(s.d_model, self.ft)
                M2 = R2 + G2 + self.w(p + "c") * inter["M1"]
            out.update(r2=r2, idx2=idx2, w2=w2)
        return Sb2 + M2, out

    def logits(self, S):
        """Final RMSNorm and the shared output matrix (reading R6)."""
        return self.lin(rmsnorm(S, self.w("g_final"), self.s.rms_eps), "W_out")

    # ---------------- one sequence, one position ----------------

    def _inputs(self, b, token, h1, h2):
        """Residual inputs of one position: S1, and S2 (one branch) or a list
        of branch states (more branches; h2 then [n_branches][d])."""
        nb = self.s.n_branches
        if token is not None:
            if nb == 1:
                return self.embed(token, 0), self.embed(token, 1)
            return self.embed(token, 0), [self.embed(token, j) for j in range(1, nb + 1)]
        S1 = np.asarray(h1).astype(self.ft)
        if h2 is None:
            return S1, None
        if nb == 1:
            return S1, np.asarray(h2).astype(self.ft)
        return S1, [np.asarray(h2[j]).astype(self.ft) for j in range(nb)]

    def step_one(self, b, token=None, h1=None, h2=None, branch_on=True, grouped=True, readout=True):
        """Continuation step of Sec. 4.4 for sequence b at t = current length.

        grouped=True interleaves the two paths layer by layer; grouped=False
        runs every primary layer first, keeping Q1/H1/M1, then the branch.
        Both compute the same definition."""
        s = self.s
        pos = self.alloc.append_one(b)
        S1, S2 = self._inputs(b, token, h1, h2)
        if not branch_on:
            S2 = None
        many = isinstance(S2, list)          # more decode branches (App. C.1)
        Sb = S2 if many else ([S2] if S2 is not None else [])
        per_layer = []
        if grouped or not Sb:
            for l in range(s.n_layers):
                S1, inter = self.primary_layer(l, b, S1, pos)
                rec = dict(inter)
                bos = []
                for j in range(len(Sb)):     # every branch reads the same primary state
                    Sb[j], bo = self.branch_layer(l, b, Sb[j], pos, inter)
                    bos.append(bo)
                if bos:
                    rec.update(bos[0])
                    rec["branches"] = bos
                per_layer.append(rec)
        else:
            inters = []
            for l in range(s.n_layers):
                S1, inter = self.primary_layer(l, b, S1, pos)
                inters.append(inter)
            recs = [dict(inters[l]) for l in range(s.n_layers)]
            for j in range(len(Sb)):
                for l in range(s.n_layers):
                    Sb[j], bo = self.branch_layer(l, b, Sb[j], pos, inters[l])
                    if j == 0:
                        recs[l].update(bo)
                    recs[l].setdefault("branches", []).append(bo)
            per_layer = recs
        out = dict(h1=S1, h2=Sb[0] if Sb else None, layers=per_layer, pos=pos, branch_on=bool(Sb))
        if many:
            out["hb"] = Sb
        if readout:
            self._readout([out])
        return out

    def _readout(self, outs):
        """Logits and mixture for a list of per-sequence results (the output
        matrix is applied to all their rows in one product)."""
        if self.s.vocab <= 0 or not outs:
            return
        Z1 = self.logits(np.stack([o["h1"] for o in outs]))
        have2 = [o for o in outs if o["h2"] is not None]
        Z2 = self.logits(np.stack([o["h2"] for o in have2])) if have2 else None
        # further branches (App. C.1): branch j of every row in one product
        many = [o for o in have2 if "hb" in o]
        Zb = [self.logits(np.stack([o["hb"][j] for o in many]))
              for j in range(1, len(many[0]["hb"]))] if many else []
        j = jm = 0
        for i, o in enumerate(outs):
            z1 = Z1[i]
            z2 = None
            zb = None
            if o["h2"] is not None:
                z2 = Z2[j]
                j += 1
                if "hb" in o:   # more branches: q is the mean branch softmax (App. C.1)
                    zb = [z2] + [Z[jm] for Z in Zb]
                    jm += 1
                    o["zb"] = zb
            alpha, m, nxt = mixture_readout(z1, z2, branch_on=z2 is not None, z_branches=zb)
            o.update(z1=z1, z2=z2, alpha=alpha, m=m, next=nxt)

    # ---------------- batched entry points ----------------

    def decode_step(self, tokens=None, h1=None, h2=None, branch_on=True, grouped=True, batch=None):
        """One continuation step for sequences 0..B-1 (in batch order).

        tokens: [B] ints (models with embeddings) or h1/h2: [B][d] residual
        inputs (layer-only workloads).  Returns a list of per-sequence dicts."""
        B = batch if batch is not None else (len(tokens) if tokens is not None else len(h1))
        outs = []
        for b in range(B):
            outs.append(self.step_one(
                b,
                token=None if tokens is None else int(tokens[b]),
                h1=None if h1 is None else h1[b],
                h2=None if h2 is None else (h2[b] if self.s.n_branches == 1 else [h[b] for h in h2]),
                branch_on=branch_on, grouped=grouped, readout=False))
        self._readout(outs)
        return outs

    def prefill(self, prompts, run_boundary=True):
        """Primary-only prefill of each prompt (Sec. 4.4, step 1): all positions
        at once in the masked-matrix form, cache written for every position,
        the final position's Q1/H1/M1 (per layer) and z1 retained.  With
        ``run_boundary`` the branch is then evaluated once at the final prompt
        position (step 2).  Pages are reserved for all sequences first, in
        batch order."""
        for b, x in enumerate(prompts):
            self.alloc.reserve(b, len(x))
        outs = []
        for b, x in enumerate(prompts):
            x = np.asarray(x)
            T = len(x)
            S1 = self.embed(x, 0)                      # [T][d]
            keep = []
            for l in range(self.s.n_layers):
                S1, inter = self._primary_layer_full(l, S1, store_b=b)
                keep.append({k: v[T - 1] for k, v in inter.items()})
            ret = dict(layers=keep, pos=T - 1, token=int(x[-1]), h1=S1[T - 1])
            if self.s.vocab > 0:
                ret["z1"] = self.logits(S1[T - 1])
            self.retained[b] = ret
            outs.append(self.boundary(b) if run_boundary else dict(ret))
        return outs

    def boundary(self, b):
        """Branch-only evaluation at the final prompt position (Sec. 4.4,
        step 2), using the retained primary intermediates; writes no cache."""
        ret = self.retained[b]
        pos = ret["pos"]
        nb = self.s.n_branches
        Sb = [self.embed(ret["token"], j) for j in range(1, nb + 1)]
        per_layer = []
        for l in range(self.s.n_layers):
            rec = dict(ret["layers"][l])
            bos = []
            for j in range(nb):
                Sb[j], bo = self.branch_layer(l, b, Sb[j], pos, ret["layers"][l])
                bos.append(bo)
            rec.update(bos[0])
            rec["branches"] = bos
            per_layer.append(rec)
        out = dict(h1=ret["h1"], h2=Sb[0], layers=per_layer, pos=pos)
        if nb > 1:
            out["hb"] = Sb
        if self.s.vocab > 0:
            z1 = ret["z1"]
            zb = [self.logits(h) for h in Sb]
            alpha, m, nxt = mixture_readout(z1, zb[0], branch_on=True, z_branches=zb if nb > 1 else None)
            out.update(z1=z1, z2=zb[0], alpha=alpha, m=m, next=nxt)
            if nb > 1:
                out["zb"] = zb
        return out

    # ---------------- full-sequence (masked matrix) form ----------------

    def _causal(self, Q, K, V):
        """Masked-matrix causal attention over T positions, all heads:
        softmax(Q K^T / sqrt(d_h) + M_causal) V (Eq. (3)).  Q [T][n_q][d_h]."""
        s = self.s
        G = s.n_q_heads // s.n_kv_heads
        T = Q.shape[0]
        out = np.empty_like(Q)
        mask = np.triu(np.full((T, T), -np.inf), k=1)
        for h in range(s.n_q_heads):
            sc = Q[:, h] @ K[:, h // G].T / np.sqrt(F64(s.head_dim)) + mask
            out[:, h] = softmax(sc) @ V[:, h // G]
        return out

    def _primary_layer_full(self, l, S1, store_b=None):
        """Primary layer over all T positions of one sequence."""
        s = self.s
        p = f"L{l}."
        T = S1.shape[0]
        pos = np.arange(T)
        N1 = rmsnorm(S1, self.w(p + "g_attn"), s.rms_eps)
        Q1 = rope(self.lin(N1, p + "W_Q").reshape(T, s.n_q_heads, s.head_dim), pos[:, None], s.rope_theta)
        K1 = rope(self.lin(N1, p + "W_K").reshape(T, s.n_kv_heads, s.head_dim), pos[:, None], s.rope_theta)
        V1 = self.lin(N1, p + "W_V").reshape(T, s.n_kv_heads, s.head_dim)
        Ks, Vs = self.store(K1), self.store(V1)
        if store_b is not None:
            self.K[l][store_b] = Ks
            self.V[l][store_b] = Vs
        A1 = self.lin(self._causal(Q1, Ks, Vs).reshape(T, -1), p + "W_O")
        Sb1 = S1 + A1
        U1 = rmsnorm(Sb1, self.w(p + "g_mlp"), s.rms_eps)
        inter = dict(q1=Q1, A1=A1, N1=N1, K1=Ks, V1=Vs)
        if not s.is_moe:
            H1, M1 = self._mlp_dense_primary(l, U1)
            inter.update(H1=H1, M1=M1)
        else:
            Ms, Hs, Gs, Rs, Is, Ws = [], [], [], [], [], []
            for t in range(T):
                r1 = self.lin(U1[t], p + "W_router")
                idx1, w1 = route(r1, s.top_k1)
                Rs.append(r1)
                Is.append(idx1)
                Ws.append(w1)
                R1 = self._experts(l, U1[t], idx1, w1)
                if s.n_shared_experts > 0:
                    Hs1 = silu(self.lin(U1[t], p + "S_gate")) * self.lin(U1[t], p + "S_up")
                    G1 = self.lin(Hs1, p + "S_down")
                else:
                    Hs1 = np.zeros(1, self.ft)
                    G1 = np.zeros(s.d_model, self.ft)
                Ms.append(R1 + G1)
                Hs.append(Hs1)
                Gs.append(G1)
            inter.update(M1=np.array(Ms), H1=np.array(Hs), G1=np.array(Gs),
                         r1=np.array(Rs), idx1=np.array(Is), w1=np.array(Ws))
            M1 = inter["M1"]
        return Sb1 + M1, inter

    def forward_full(self, x):
        """The two-path forward over a whole sequence (the training graph of
        Sec. 4.4), dense models: every position evaluates both paths, the
        branch attends to the primary keys/values with the causal mask.
        Returns per-position z1, z2 and the final residuals.  Does not touch
        the cache."""
        s = self.s
        assert not s.is_moe
        x = np.asarray(x)
        T = len(x)
        pos = np.arange(T)
        S1 = self.embed(x, 0)
        S2 = self.embed(x, 1)
        for l in range(s.n_layers):
            p = f"L{l}."
            S1_new, inter = self._primary_layer_full(l, S1)
            if s.compute_matched:
                A2 = self.w(p + "g_A") * inter["A1"]
            else:
                N2 = rmsnorm(S2, self.w(p + "g_attn"), s.rms_eps)
                Q2 = rope(self.lin(N2, p + "W_Q").reshape(T, s.n_q_heads, s.head_dim), pos[:, None], s.rope_theta)
                Q2t = Q2 + self.w(p + "a").reshape(s.n_q_heads, s.head_dim) * inter["q1"]
                A2 = self.lin(self._causal(Q2t, inter["K1"], inter["V1"]).reshape(T, -1), p + "W_O")
            Sb2 = S2 + A2
            U2 = rmsnorm(Sb2, self.w(p + "g_mlp"), s.rms_eps)
            H2 = silu(self.lin(U2, p + "W_gate")) * self.lin(U2, p + "W_up")
            M2 = self.lin(H2 + self.w(p + "b") * inter["H1"], p + "W_down") + self.w(p + "c") * inter["M1"]
            S1, S2 = S1_new, Sb2 + M2
        out = dict(h1=S1, h2=S2)
        if s.vocab > 0:
            out["z1"] = self.logits(S1)
            out["z2"] = self.logits(S2)
        return out


def expert_assignments(idx1, idx2, n_experts):
    """For each expert, the (path, sequence) pairs that selected it, in
    (path, sequence) order.  idx1/idx2: [B][k] selected indices (idx2 may be
    None when the branch is off)."""
    out = [[] for _ in range(n_experts)]
    for path, idx in ((0, idx1), (1, idx2)):
        if idx is None:
            continue
        for b, row in enumerate(idx):
            for e in row:
                out[int(e)].append((path, b))
    return out
