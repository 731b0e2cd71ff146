"""Benchmark of the grouped Decode-Branch decode step on one MI355X.

Workload: one decoder layer at 8B shape (d_model 4096, 32 query / 8 KV heads
of 128, SwiGLU 14336) followed by the final norm, the shared output matrix
(vocab 128256) and the mixture readout; batch 32; every sequence holds 4096
cached positions in 16-token pages; bf16 weights and cache, fp32
accumulation; synthetic seeded weights N(0, 0.02), K/V and residual inputs
N(0, 1).  A step is one grouped primary+branch continuation step
(dbt_decode_step, branch on) over the 32 sequences; after each step the
sequences are truncated back to 4096 positions so every step sees the same
cache length.

Prints one JSON line.  value = tokens/s of the grouped step (32 continuation
tokens per step).  Also reported: the primary-only and ungrouped step times,
the branch overhead, the step's algorithmic HBM bytes and the roofline of the
dominant kernel (the output-matrix projection), timed with HIP events on the
stream it runs on, plus the CPU oracle timed on a bounded sample.

    python bench.py [--gpus 1] [--steps 20] [--warmup 5] [--no-cpu-baseline]
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

HBM_PEAK_GBPS = 8000.0
METRIC = "grouped decode step µs + tokens/s; HBM GB/s vs peak; branch overhead % vs primary-only"


def algorithmic_bytes(shape, B, L):
    """Weights touched once + live KV read once (bf16), the decode traffic
    model of Eq. (20): B_decode = B_weight + B_state."""
    d, dq, dkv, f, V = shape.d_model, shape.d_q, shape.d_kv, shape.d_ff, shape.vocab
    layer = (d * (dq + 2 * dkv) + dq * d + 2 * d * f + f * d) * 2
    head = V * d * 2
    kv = B * (L + 1) * 2 * dkv * 2
    return layer, head, kv


def time_mode(sess, B, L, h1d, h2d, mode, steps, warmup):
    import torch
    from paper_2608_12385_amd import binding
    sin = sess.step_in(B, None, h1d, h2d)
    out, _t = sess.outputs(B, logits=False, hidden=False)
    st = sess.stream

    def one():
        if mode == "ungrouped":
            binding.dbt_decode_step_ungrouped(sess.model, sess.kv, sin, out, st)
        else:
            binding.dbt_decode_step(sess.model, sess.kv, sin, 1 if mode == "grouped" else 0, out, st)
        for b in range(B):
            binding.dbt_kv_truncate(sess.kv, b, L)

    for _ in range(warmup):
        one()
    torch.cuda.synchronize()
    binding.dbt_stage_timing(sess.model, binding.STAGES["lmhead"], mode == "grouped")
    t0 = time.perf_counter()
    for _ in range(steps):
        one()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    lm_ms, lm_n = binding.dbt_stage_time(sess.model, binding.STAGES["lmhead"])
    binding.dbt_stage_timing(sess.model, binding.STAGES["lmhead"], 0)
    return (t1 - t0) / steps, lm_ms, lm_n


def cpu_baseline(shape, W, h, L, nseq):
    """The oracle as it stands, on nseq sequences of the same workload (one
    grouped step each, fresh oracle: parameter widening included)."""
    import synth
    from oracle import Oracle
    try:
        import threadpoolctl
        threads = max([i.get("num_threads", 1) for i in threadpoolctl.threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threads = os.cpu_count()
    kvs = [synth.make_kv(shape, 0, b, L, seed=3) for b in range(nseq)]
    t0 = time.perf_counter()
    orc = Oracle(shape, W.values)
    for b in range(nseq):
        (k, _), (v, _) = kvs[b]
        orc.kv_fill(b, L, [k], [v])
    outs = [orc.step_one(b, h1=h[0, b], h2=h[1, b], readout=False) for b in range(nseq)]
    orc._readout(outs)
    dt = time.perf_counter() - t0
    return dict(value=nseq / dt, unit="tokens/s", cores=int(threads), kind="oracle",
                sample=f"{nseq} of 32 sequences, one grouped step each (float64 NumPy, fresh oracle "
                       f"including parameter widening), {dt:.1f} s")


def time_workload(name, steps, warmup, **shape_kw):
    """Grouped / primary-only step times of another workload (extra report)."""
    import torch
    import synth
    from paper_2608_12385_amd import Session
    w = synth.workload(name, **shape_kw)
    shape = w["shape"]
    B = w["batch"]
    if "cache_len" in w:
        lengths = [w["cache_len"]] * B
    else:
        lengths = [int(x) for x in synth.make_lengths(4, B, w["len_lo"], w["len_hi"])]
    W = synth.make_weights(shape, seed=0)
    max_pos = max(lengths) + 16
    sess = Session(shape, {k: W.device_array(k) for k in W.values}, max_batch=B, max_pos=max_pos,
                   num_pages=sum((L + 16) // 16 + 1 for L in lengths) + B)
    for b, L in enumerate(lengths):
        (_, kb), (_, vb) = synth.make_kv(shape, 0, b, L, seed=3)
        sess.reserve_fill(b, [kb], [vb])
    del W
    h = synth.make_hidden(shape, B, step=0, seed=2)
    h1d = torch.from_numpy(np.ascontiguousarray(h[0])).cuda()
    h2d = torch.from_numpy(np.ascontiguousarray(h[1])).cuda()
    from paper_2608_12385_amd import binding
    res = {}
    for mode in ("grouped", "primary"):
        sin = sess.step_in(B, None, h1d, h2d)
        out, _t = sess.outputs(B, logits=False, hidden=False)
        def one():
            binding.dbt_decode_step(sess.model, sess.kv, sin, 1 if mode == "grouped" else 0, out, sess.stream)
            for b, L in enumerate(lengths):
                binding.dbt_kv_truncate(sess.kv, b, L)
        for _ in range(warmup):
            one()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            one()
        torch.cuda.synchronize()
        res[mode] = (time.perf_counter() - t0) / steps
    sess.close()
    d, dq, dkv = shape.d_model, shape.d_q, shape.d_kv
    attn_w = (d * (dq + 2 * dkv) + dq * d) * 2
    kv = sum(L + 1 for L in lengths) * 2 * dkv * 2
    rec = {"workload": name, "batch": B, "grouped_us": res["grouped"] * 1e6, "primary_only_us": res["primary"] * 1e6,
           "branch_overhead_pct": 100 * (res["grouped"] - res["primary"]) / res["primary"]}
    if shape.is_moe:
        rec["k1"], rec["k2"] = shape.top_k1, shape.top_k2
        rec["note"] = "bytes depend on the touched experts; see profiles"
    else:
        mlp = 3 * d * shape.d_ff * 2
        rec["algorithmic_MB"] = (attn_w + mlp + kv) / 1e6
        rec["GBps"] = (attn_w + mlp + kv) / res["grouped"] / 1e9
    return rec


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seqs", type=int, default=16)
    ap.add_argument("--all", action="store_true",
                    help="also time the long-context and MoE workloads (extra fields)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU: this build runs the decode path on a single MI355X "
              "(sharding is described, not built); use --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    import synth
    from paper_2608_12385_amd import Session

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    w = synth.workload("layer8b_bf16")
    shape = w["shape"]
    B, L = w["batch"], w["cache_len"]
    W = synth.make_weights(shape, seed=0)
    sess = Session(shape, {k: W.device_array(k) for k in W.values}, max_batch=B, max_pos=L + 16,
                   num_pages=B * ((L + 16) // 16 + 1))
    for b in range(B):
        (_, kb), (_, vb) = synth.make_kv(shape, 0, b, L, seed=3)
        sess.reserve_fill(b, [kb], [vb])
    h = synth.make_hidden(shape, B, step=0, seed=2)
    h1d = torch.from_numpy(np.ascontiguousarray(h[0])).cuda()
    h2d = torch.from_numpy(np.ascontiguousarray(h[1])).cuda()

    t_grp, lm_ms, lm_n = time_mode(sess, B, L, h1d, h2d, "grouped", args.steps, args.warmup)
    t_pri, _, _ = time_mode(sess, B, L, h1d, h2d, "primary", args.steps, args.warmup)
    t_ung, _, _ = time_mode(sess, B, L, h1d, h2d, "ungrouped", args.steps, args.warmup)

    layer_b, head_b, kv_b = algorithmic_bytes(shape, B, L)
    step_bytes = layer_b + head_b + kv_b
    x_bytes = 2 * B * shape.d_model * 2
    logit_bytes = 2 * B * shape.vocab * 4
    lm_alg = head_b + x_bytes + logit_bytes
    lm_s = (lm_ms / max(lm_n, 1)) / 1e3
    lm_gbps = lm_alg / lm_s / 1e9
    line = {
        "metric": METRIC,
        "value": B / t_grp,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": t_grp * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,0.02) weights, N(0,1) KV cache and residual inputs)",
        "config": {
            "workload": "grouped primary+branch decode step: one 8B-shape layer (d 4096, 32q/8kv x 128, "
                        "SwiGLU 14336) + final norm + LM head (vocab 128256) + mixture readout, "
                        "batch 32, KV cache 4096/sequence in 16-token pages",
            "batch": B, "cache_len": L, "page": 16,
        },
        "step_us": t_grp * 1e6,
        "primary_only_us": t_pri * 1e6,
        "ungrouped_us": t_ung * 1e6,
        "branch_overhead_pct": 100.0 * (t_grp - t_pri) / t_pri,
        "algorithmic_MB_per_step": step_bytes / 1e6,
        "step_GBps": step_bytes / t_grp / 1e9,
        "step_frac_of_peak": step_bytes / t_grp / 1e9 / HBM_PEAK_GBPS,
        "roofline": {
            "kernel": "LM-head projection (k_gemm_bf16, 64 stacked rows)",
            "bound": "hbm",
            "achieved": lm_gbps,
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": lm_gbps / HBM_PEAK_GBPS,
            "traffic": None,
            "launch_us": lm_s * 1e6,
            "algorithmic_MB_per_launch": lm_alg / 1e6,
        },
    }
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(shape, W, h, L, args.cpu_seqs)
    sess.close()
    if args.all:
        del W
        extra = [time_workload("longctx_bf16", args.steps, args.warmup)]
        for k2 in (2, 4, 8):
            extra.append(time_workload("moe_bf16", args.steps, args.warmup, top_k2=k2))
        line["other_workloads"] = extra
    print(json.dumps(line))


if __name__ == "__main__":
    main()
