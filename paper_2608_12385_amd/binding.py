"""ctypes binding of libdbt (include/dbt.h): argument marshalling only.

Every step of the decode path runs in the library's HIP kernels; PyTorch only
allocates device memory and provides the stream.  If the shared library is
missing this module raises instead of falling back to anything else.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libdbt.so")

DBT_F32, DBT_BF16 = 0, 1
STATUS = {0: "DBT_OK", 1: "DBT_ERR_ARG", 2: "DBT_ERR_SHAPE", 3: "DBT_ERR_NO_PAGES",
          4: "DBT_ERR_STATE", 5: "DBT_ERR_UNSUPPORTED", 6: "DBT_ERR_HIP"}

P = ctypes.c_void_p
I32 = ctypes.c_int32


class DbtError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"{STATUS.get(status, status)}: {msg}")
        self.status = status


class dbt_config(ctypes.Structure):
    _fields_ = [(n, I32) for n in (
        "n_layers", "d_model", "n_q_heads", "n_kv_heads", "head_dim", "d_ff", "vocab",
        "n_experts", "d_ff_expert", "d_ff_shared", "top_k1", "top_k2", "replay", "compute_matched",
        "n_branches", "dtype", "has_embeddings", "max_batch", "max_pos", "max_prompt")] + [
        ("rms_eps", ctypes.c_float), ("rope_theta", ctypes.c_float)]


class dbt_layer_weights(ctypes.Structure):
    _fields_ = [(n, P) for n in (
        "attn_norm", "wq", "wk", "wv", "wo", "mlp_norm", "w_gate", "w_up", "w_down",
        "a", "b", "c", "router", "x_gate", "x_up", "x_down", "s_gate", "s_up", "s_down",
        "g_attn_copy", "g_shared_copy")]


class dbt_weights(ctypes.Structure):
    _fields_ = [("emb1", P), ("emb2", P), ("emb_norm", P), ("final_norm", P), ("lm_head", P),
                ("h_layers", ctypes.POINTER(dbt_layer_weights))]


class dbt_step_in(ctypes.Structure):
    _fields_ = [("tokens", P), ("h1_in", P), ("h2_in", P), ("batch", I32)]


class dbt_step_out(ctypes.Structure):
    _fields_ = [(n, P) for n in ("logits1", "logits2", "alpha", "next_token", "h1_out", "h2_out",
                                 "route_idx1", "route_idx2", "route_w1", "route_w2",
                                 "route_logits1", "route_logits2")]


_lib = None

_SIGS = {
    "dbt_workspace_bytes": (ctypes.c_size_t, [ctypes.POINTER(dbt_config)]),
    "dbt_kv_pages_bytes": (ctypes.c_size_t, [ctypes.POINTER(dbt_config), I32]),
    "dbt_create": (I32, [ctypes.POINTER(dbt_config), ctypes.POINTER(dbt_weights), P, ctypes.POINTER(P)]),
    "dbt_destroy": (I32, [P]),
    "dbt_kv_create": (I32, [P, P, P, I32, P, I32, ctypes.POINTER(P)]),
    "dbt_kv_destroy": (I32, [P]),
    "dbt_kv_reserve": (I32, [P, I32, I32, ctypes.POINTER(I32)]),
    "dbt_kv_truncate": (I32, [P, I32, I32]),
    "dbt_kv_length": (I32, [P, I32]),
    "dbt_kv_pages": (I32, [P, I32, ctypes.POINTER(I32), I32]),
    "dbt_last_error": (ctypes.c_char_p, []),
    "dbt_kv_fill": (I32, [P, I32, I32, I32, I32, P, P, P]),
    "dbt_prefill": (I32, [P, P, P, ctypes.POINTER(I32), I32, I32, ctypes.POINTER(dbt_step_out), P]),
    "dbt_boundary": (I32, [P, P, I32, ctypes.POINTER(dbt_step_out), P]),
    "dbt_decode_step": (I32, [P, P, ctypes.POINTER(dbt_step_in), I32, ctypes.POINTER(dbt_step_out), P]),
    "dbt_decode_step_ungrouped": (I32, [P, P, ctypes.POINTER(dbt_step_in), ctypes.POINTER(dbt_step_out), P]),
    "dbt_decode_step_noalloc": (I32, [P, P, ctypes.POINTER(dbt_step_in), I32, ctypes.POINTER(dbt_step_out), P]),
    "dbt_stage_timing": (I32, [P, I32, I32]),
    "dbt_stage_time": (ctypes.c_double, [P, I32, ctypes.POINTER(I32)]),
}

STAGES = dict(qkv=0, attn=1, wo=2, gateup=3, down=4, lmhead=5, mix=6)


def lib():
    """The loaded libdbt.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def exported_symbols():
    return list(_SIGS)


def _check(status):
    if status != 0:
        raise DbtError(status, lib().dbt_last_error().decode())


# ----------------------------------------------------------------------------
# Same names as the C ABI
# ----------------------------------------------------------------------------

def dbt_workspace_bytes(cfg):
    return lib().dbt_workspace_bytes(ctypes.byref(cfg))


def dbt_kv_pages_bytes(cfg, num_pages):
    return lib().dbt_kv_pages_bytes(ctypes.byref(cfg), num_pages)


def dbt_create(cfg, weights, workspace_ptr):
    h = P()
    _check(lib().dbt_create(ctypes.byref(cfg), ctypes.byref(weights), P(workspace_ptr), ctypes.byref(h)))
    return h


def dbt_destroy(m):
    _check(lib().dbt_destroy(m))


def dbt_kv_create(m, k_ptr, v_ptr, num_pages, page_table_ptr, max_pages_per_seq):
    h = P()
    _check(lib().dbt_kv_create(m, P(k_ptr), P(v_ptr), num_pages, P(page_table_ptr), max_pages_per_seq,
                               ctypes.byref(h)))
    return h


def dbt_kv_destroy(kv):
    _check(lib().dbt_kv_destroy(kv))


def dbt_kv_reserve(kv, b, length):
    out = (I32 * max(1, (length + 15) // 16))()
    _check(lib().dbt_kv_reserve(kv, b, length, out))
    return list(out)[: (length + 15) // 16]


def dbt_kv_truncate(kv, b, length):
    _check(lib().dbt_kv_truncate(kv, b, length))


def dbt_kv_length(kv, b):
    return lib().dbt_kv_length(kv, b)


def dbt_kv_pages(kv, b):
    n = lib().dbt_kv_pages(kv, b, None, 0)
    out = (I32 * max(1, n))()
    lib().dbt_kv_pages(kv, b, out, n)
    return list(out)[:n]


def dbt_last_error():
    return lib().dbt_last_error().decode()


def dbt_kv_fill(kv, layer, b, start, count, k_ptr, v_ptr, stream):
    _check(lib().dbt_kv_fill(kv, layer, b, start, count, P(k_ptr), P(v_ptr), P(stream)))


def dbt_prefill(m, kv, tokens_ptr, prompt_lens, batch, run_boundary, out, stream):
    lens = (I32 * batch)(*prompt_lens)
    _check(lib().dbt_prefill(m, kv, P(tokens_ptr), lens, batch, run_boundary, ctypes.byref(out), P(stream)))


def dbt_boundary(m, kv, batch, out, stream):
    _check(lib().dbt_boundary(m, kv, batch, ctypes.byref(out), P(stream)))


def dbt_decode_step(m, kv, step_in, branch_on, out, stream):
    _check(lib().dbt_decode_step(m, kv, ctypes.byref(step_in), branch_on, ctypes.byref(out), P(stream)))


def dbt_decode_step_ungrouped(m, kv, step_in, out, stream):
    _check(lib().dbt_decode_step_ungrouped(m, kv, ctypes.byref(step_in), ctypes.byref(out), P(stream)))


def dbt_decode_step_noalloc(m, kv, step_in, branch_on, out, stream):
    _check(lib().dbt_decode_step_noalloc(m, kv, ctypes.byref(step_in), branch_on, ctypes.byref(out), P(stream)))


def dbt_stage_timing(m, stage, enable):
    _check(lib().dbt_stage_timing(m, stage, int(enable)))


def dbt_stage_time(m, stage):
    n = I32(0)
    ms = lib().dbt_stage_time(m, stage, ctypes.byref(n))
    if ms < 0:
        raise DbtError(6, "stage timing failed")
    return ms, n.value


# ----------------------------------------------------------------------------
# Session: keeps the torch-owned device buffers of one model + cache alive
# ----------------------------------------------------------------------------

def _ptr(t):
    return 0 if t is None else t.data_ptr()


class Session:
    """One model and one KV cache on a CUDA (HIP) device.

    ``shape`` is any object with the model fields (n_layers, d_model, ...,
    dtype "f32"/"bf16", has_embeddings, n_experts, ...); ``device_params``
    maps parameter names to arrays in device storage type (bf16 matrices as
    uint16 bit patterns, everything else float32):
        E1, E2, g_emb, g_final, W_out,
        L{l}.g_attn, L{l}.W_Q, L{l}.W_K, L{l}.W_V, L{l}.W_O, L{l}.g_mlp,
        L{l}.W_gate, L{l}.W_up, L{l}.W_down, L{l}.a, L{l}.b, L{l}.c.
    With n_branches > 1 the branch tables E2, E3, ... are stacked in branch
    order, and branch outputs/inputs are [n_branches][batch][...].
    """

    def __init__(self, shape, device_params, max_batch, max_pos, max_prompt=0, num_pages=None,
                 device="cuda"):
        import torch
        self.torch = torch
        self.shape = shape
        self.device = device
        s = shape
        self.cfg = dbt_config(
            n_layers=s.n_layers, d_model=s.d_model, n_q_heads=s.n_q_heads, n_kv_heads=s.n_kv_heads,
            head_dim=s.head_dim, d_ff=s.d_ff, vocab=s.vocab, n_experts=s.n_experts,
            d_ff_expert=s.d_ff_expert, d_ff_shared=s.d_ff_shared * max(0, s.n_shared_experts),
            top_k1=s.top_k1, top_k2=s.top_k2,
            replay=int(s.replay), compute_matched=int(s.compute_matched),
            n_branches=int(getattr(s, "n_branches", 1)),
            dtype=DBT_BF16 if s.dtype == "bf16" else DBT_F32,
            has_embeddings=int(s.has_embeddings), max_batch=max_batch, max_pos=max_pos,
            max_prompt=max_prompt, rms_eps=s.rms_eps, rope_theta=s.rope_theta)
        self.n_branches = max(1, int(getattr(s, "n_branches", 1)))
        self._keep = {}
        for name, arr in device_params.items():
            if self.n_branches > 1 and name.startswith("E") and name[1:].isdigit() and name != "E1":
                continue
            self._keep[name] = self._upload(arr)
        if self.n_branches > 1 and "E2" in device_params:
            self._keep["E2"] = self._upload(np.stack(
                [device_params[f"E{j + 2}"] for j in range(self.n_branches)]))
        self._layers = (dbt_layer_weights * s.n_layers)()
        names = dict(attn_norm="g_attn", wq="W_Q", wk="W_K", wv="W_V", wo="W_O", mlp_norm="g_mlp",
                     w_gate="W_gate", w_up="W_up", w_down="W_down", a="a", b="b", c="c",
                     router="W_router", x_gate="X_gate", x_up="X_up", x_down="X_down",
                     s_gate="S_gate", s_up="S_up", s_down="S_down", g_attn_copy="g_A",
                     g_shared_copy="g_G")
        for l in range(s.n_layers):
            for field, nm in names.items():
                setattr(self._layers[l], field, _ptr(self._keep.get(f"L{l}.{nm}")))
        self.weights = dbt_weights(
            emb1=_ptr(self._keep.get("E1")), emb2=_ptr(self._keep.get("E2")),
            emb_norm=_ptr(self._keep.get("g_emb")), final_norm=_ptr(self._keep.get("g_final")),
            lm_head=_ptr(self._keep.get("W_out")), h_layers=self._layers)
        ws_bytes = dbt_workspace_bytes(self.cfg)
        if ws_bytes == 0:
            raise DbtError(2, dbt_last_error())
        self.workspace = torch.empty(ws_bytes, dtype=torch.uint8, device=device)
        self.model = dbt_create(self.cfg, self.weights, self.workspace.data_ptr())
        self.max_pages_per_seq = (max_pos + 15) // 16
        if num_pages is None:
            num_pages = max_batch * self.max_pages_per_seq
        self.num_pages = num_pages
        pb = dbt_kv_pages_bytes(self.cfg, num_pages)
        self.k_pages = torch.empty(pb, dtype=torch.uint8, device=device)
        self.v_pages = torch.empty(pb, dtype=torch.uint8, device=device)
        self.page_table = torch.full((max_batch, self.max_pages_per_seq), -1, dtype=torch.int32, device=device)
        self.kv = dbt_kv_create(self.model, self.k_pages.data_ptr(), self.v_pages.data_ptr(), num_pages,
                                self.page_table.data_ptr(), self.max_pages_per_seq)

    # -- helpers --
    def _upload(self, arr):
        torch = self.torch
        a = np.ascontiguousarray(arr)
        if a.dtype == np.uint16:
            a = a.view(np.int16)
        return torch.from_numpy(a).to(self.device)

    def _br(self, *shape):
        """Shape of a branch output: [n_branches] leads only with several."""
        return shape if self.n_branches == 1 else (self.n_branches,) + shape

    @property
    def stream(self):
        return self.torch.cuda.current_stream().cuda_stream

    def close(self):
        if getattr(self, "kv", None):
            dbt_kv_destroy(self.kv)
            self.kv = None
        if getattr(self, "model", None):
            dbt_destroy(self.model)
            self.model = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def outputs(self, batch, logits=True, hidden=True, routing=False):
        """Allocates an output set; returns (dbt_step_out, dict of tensors)."""
        torch = self.torch
        s = self.shape
        t = {}
        if logits and s.vocab > 0:
            t["logits1"] = torch.empty(batch, s.vocab, dtype=torch.float32, device=self.device)
            t["logits2"] = torch.empty(*self._br(batch, s.vocab), dtype=torch.float32, device=self.device)
        if s.vocab > 0:
            t["alpha"] = torch.empty(batch, dtype=torch.float32, device=self.device)
            t["next_token"] = torch.empty(batch, dtype=torch.int32, device=self.device)
        if hidden:
            t["h1_out"] = torch.empty(batch, s.d_model, dtype=torch.float32, device=self.device)
            t["h2_out"] = torch.empty(*self._br(batch, s.d_model), dtype=torch.float32, device=self.device)
        if routing and s.n_experts > 0:
            k2 = s.top_k1 if s.replay else s.top_k2
            L = s.n_layers
            t["route_idx1"] = torch.empty(L, batch, s.top_k1, dtype=torch.int32, device=self.device)
            t["route_w1"] = torch.empty(L, batch, s.top_k1, dtype=torch.float32, device=self.device)
            t["route_idx2"] = torch.empty(L, batch, k2, dtype=torch.int32, device=self.device)
            t["route_w2"] = torch.empty(L, batch, k2, dtype=torch.float32, device=self.device)
            t["route_logits1"] = torch.empty(L, batch, s.n_experts, dtype=torch.float32, device=self.device)
            t["route_logits2"] = torch.empty(L, batch, s.n_experts, dtype=torch.float32, device=self.device)
        out = dbt_step_out(**{k: v.data_ptr() for k, v in t.items()})
        return out, t

    def step_in(self, batch, tokens=None, h1=None, h2=None):
        return dbt_step_in(tokens=_ptr(tokens), h1_in=_ptr(h1), h2_in=_ptr(h2), batch=batch)

    # -- calls --
    def reserve_fill(self, b, K_layers, V_layers):
        """Reserve len positions for sequence b and copy K/V [len][n_kv][d_h]
        (device storage type arrays, one per layer) into its pages."""
        length = int(K_layers[0].shape[0])
        pages = dbt_kv_reserve(self.kv, b, length)
        for l in range(self.shape.n_layers):
            kd = self._upload(K_layers[l])
            vd = self._upload(V_layers[l])
            dbt_kv_fill(self.kv, l, b, 0, length, kd.data_ptr(), vd.data_ptr(), self.stream)
            self.torch.cuda.current_stream().synchronize()
        return pages

    def prefill(self, prompts, run_boundary=True):
        torch = self.torch
        flat = np.concatenate([np.asarray(p, np.int32) for p in prompts])
        tok = torch.from_numpy(flat).to(self.device)
        out, t = self.outputs(len(prompts))
        dbt_prefill(self.model, self.kv, tok.data_ptr(), [len(p) for p in prompts], len(prompts),
                    int(run_boundary), out, self.stream)
        torch.cuda.current_stream().synchronize()
        return t

    def decode(self, tokens=None, h1=None, h2=None, branch_on=True, grouped=True, batch=None, logits=True):
        torch = self.torch
        tk = None if tokens is None else torch.as_tensor(np.asarray(tokens, np.int32)).to(self.device)
        h1d = None if h1 is None else torch.as_tensor(np.ascontiguousarray(h1, np.float32)).to(self.device)
        h2d = None if h2 is None else torch.as_tensor(np.ascontiguousarray(h2, np.float32)).to(self.device)
        B = batch if batch is not None else (len(tokens) if tokens is not None else h1.shape[0])
        sin = self.step_in(B, tk, h1d, h2d)
        out, t = self.outputs(B, logits=logits, routing=True)
        if grouped:
            dbt_decode_step(self.model, self.kv, sin, int(branch_on), out, self.stream)
        else:
            dbt_decode_step_ungrouped(self.model, self.kv, sin, out, self.stream)
        torch.cuda.current_stream().synchronize()
        return t
