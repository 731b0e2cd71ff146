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
tokens per step) over the contract's block of exactly K steps after W
warm-ups.  Then the measurement protocol: grouped, primary-only and
ungrouped steps interleaved for 100 iterations after 10 warm-ups, each step
timed by HIP events on its stream, reported as median, p10 and p90 per mode
(step_us, primary_only_us, ungrouped_us and the branch overhead are the
medians).  Also reported: the step's algorithmic HBM bytes, every stage
kernel's launch time and fraction of the HBM peak, the roofline of the
dominant kernel (the output-matrix projection: its weight bytes over its
event-timed launch), and the CPU oracle timed per mode on a bounded sample.

    python bench.py [--gpus 1] [--steps 200] [--warmup 50] [--no-cpu-baseline]
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
CALIB_BYTES = 256 << 20   # plain device copy used to calibrate the memory counters
METRIC = "grouped decode step µs + tokens/s; HBM GB/s vs peak; branch overhead % vs primary-only"


TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "lmhead_traffic_layer8b_b32_l4096.md")
GEMM_SOURCE = os.path.join(ROOT, "paper_2608_12385_amd", "csrc", "gemm.hip")
LMHEAD_KERNEL = "k_gemm_bf16<4, 2, 1, 16, false, 2, false>"   # grouped step: 64 stacked rows, 16 waves x 32 rows


def _sha256(path):
    import hashlib
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def _db(path):
    import glob
    import sqlite3
    dbs = [path] if path.endswith(".db") else sorted(glob.glob(os.path.join(path, "**", "*.db"), recursive=True))
    if not dbs:
        raise SystemExit(f"no rocpd database under {path}")
    return sqlite3.connect(dbs[0])


def _short(name):
    name = name.replace("dbt::(anonymous namespace)::", "")
    return name.split("(")[0].replace("void ", "")


def kernel_table(path):
    """Markdown table of per-kernel durations from a rocprofv3 --kernel-trace database."""
    c = _db(path)
    rows = c.execute(
        "select name, grid_x / workgroup_x, grid_y, grid_z, count(*), "
        "avg(end - start), min(end - start), max(end - start) from kernels "
        "group by name, grid_x, grid_y, grid_z order by count(*) * avg(end - start) desc"
    ).fetchall()
    out = ["| kernel | grid | launches | avg us | min us | max us |", "|---|---|---|---|---|---|"]
    for name, gx, gy, gz, n, avg, mn, mx in rows:
        out.append(f"| {_short(name)} | {gx} x {gy} x {gz} | {n} | {avg / 1e3:.2f} | {mn / 1e3:.2f} | {mx / 1e3:.2f} |")
    return "\n".join(out)


def _counter(path, counter):
    c = _db(path)
    return c.execute("select kernel_name, value from counters_collection where counter_name = ? order by dispatch_id",
                     (counter,)).fetchall()


def traffic_summary(fetch_path, write_path):
    """Memory-counter traffic, calibrated on a plain device copy, of the
    output-matrix projection and of whole grouped steps.

    Each counter (KiB per dispatch) is scaled by known bytes / counter reading of
    the 256 MiB device-to-device copies bench.py --calib-copy launches (the only
    copies of that size in the run).  The runs use --grouped-only, so every
    dispatch after the last calibration copy belongs to a grouped step; steps
    are counted by the mixture kernel (one launch per step)."""
    lines, steps = [], []
    res, step_bytes = {}, {}
    for counter, path in (("FETCH_SIZE", fetch_path), ("WRITE_SIZE", write_path)):
        vals = _counter(path, counter)
        idx = [i for i, (k, v) in enumerate(vals) if "copyBuffer" in k and v > 0.4 * CALIB_BYTES / 1024]
        if len(idx) != 3:
            raise SystemExit(f"{counter}: expected 3 calibration copies, found {len(idx)}")
        calib = [vals[i][1] for i in idx]
        factor = (CALIB_BYTES / 1024) / (sum(calib) / len(calib))
        after = vals[idx[-1] + 1:]
        lm = [v for k, v in after if _short(k) == LMHEAD_KERNEL]
        if not lm:
            raise SystemExit(f"{counter}: no {LMHEAD_KERNEL} dispatches")
        n_steps = sum(1 for k, _ in after if _short(k).startswith("k_mix_select"))
        kib = sum(lm) / len(lm)
        res[counter] = kib * 1024 * factor
        step_bytes[counter] = sum(v for _, v in after) * 1024 * factor / max(n_steps, 1)
        lines.append(f"| {counter} | {sum(calib) / len(calib):.1f} | {factor:.4f} | {len(lm)} | {kib:.1f} | "
                     f"{kib * 1024 * factor / 1e6:.1f} | {n_steps} | {step_bytes[counter] / 1e6:.1f} |")
    total = res["FETCH_SIZE"] + res["WRITE_SIZE"]
    step_total = step_bytes["FETCH_SIZE"] + step_bytes["WRITE_SIZE"]
    head = ["| counter | calibration copy reads (KiB, 256 MiB moved) | scale | LM-head dispatches | "
            "LM-head avg (KiB) | LM-head scaled (MB) | grouped steps | per step scaled (MB) |",
            "|---|---|---|---|---|---|---|---|"]
    tail = ["", f"lmhead_traffic_bytes_per_launch: {int(round(total))}",
            f"step_traffic_bytes: {int(round(step_total))}",
            f"gemm_source_sha256: {_sha256(GEMM_SOURCE)}",
            f"sources_sha256: {_sources_sha()}"]
    return "\n".join(head + lines + tail)


def _sources_sha():
    """Hash of the kernel sources a decode step runs (the prompt-only kernels
    in csrc/prefill_*.hip never run in a decode step)."""
    import hashlib
    import glob
    h = hashlib.sha256()
    for f in sorted(glob.glob(os.path.join(ROOT, "paper_2608_12385_amd", "csrc", "*"))):
        if os.path.basename(f).startswith("prefill_"):
            continue
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def recorded_traffic():
    """Counter-derived HBM bytes: (per launch of the output-matrix projection,
    per grouped step), each None when no record exists or the code it was
    measured on changed since (the projection source / all kernel sources)."""
    try:
        text = open(TRAFFIC_PROFILE).read()
    except OSError:
        return None, None
    kv = dict(l.split(": ", 1) for l in text.splitlines()
              if l.startswith(("lmhead_traffic", "step_traffic", "gemm_source", "sources_sha")))
    lm = int(kv["lmhead_traffic_bytes_per_launch"]) if kv.get("gemm_source_sha256") == _sha256(GEMM_SOURCE) else None
    st = int(kv["step_traffic_bytes"]) if ("step_traffic_bytes" in kv and
                                          kv.get("sources_sha256") == _sources_sha()) else None
    return lm, st


def algorithmic_bytes(shape, B, L):
    """Weights touched once + live KV read once (bf16), the decode traffic
    model of Eq. (20): B_decode = B_weight + B_state."""
    d, dq, dkv, f, V = shape.d_model, shape.d_q, shape.d_kv, shape.d_ff, shape.vocab
    layer = (d * (dq + 2 * dkv) + dq * d + 2 * d * f + f * d) * 2
    head = V * d * 2
    kv = B * (L + 1) * 2 * dkv * 2
    return layer, head, kv


def step_fn(sess, B, L, h1d, h2d, mode):
    """A callable that enqueues one step of `mode` (grouped, primary or
    ungrouped) and truncates every sequence back to L cached positions (host
    bookkeeping only), so that every step sees the same cache."""
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
    one.keep = (sin, out, _t)
    return one


def time_block(one, steps, warmup):
    """W untimed steps, then exactly K steps bracketed by device
    synchronisation on both sides: seconds per step."""
    import torch
    for _ in range(warmup):
        one()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        one()
    torch.cuda.synchronize()
    return (time.perf_counter() - t0) / steps


def time_interleaved(fns, iters, warmup):
    """The modes interleaved step by step (so drift in clocks or memory state
    hits every mode alike), each step bracketed by HIP events recorded on the
    stream the library launches on: per mode the list of step times (us)."""
    import torch
    names = list(fns)
    for _ in range(warmup):
        for n in names:
            fns[n]()
    torch.cuda.synchronize()
    ev = {n: [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(iters)]
          for n in names}
    for i in range(iters):
        for n in names:
            a, b = ev[n][i]
            a.record()
            fns[n]()
            b.record()
    torch.cuda.synchronize()
    return {n: [a.elapsed_time(b) * 1e3 for a, b in ev[n]] for n in names}


def dist(us):
    """median, p10 and p90 of a list of step times."""
    x = np.asarray(us, np.float64)
    return {"median": float(np.median(x)), "p10": float(np.percentile(x, 10)), "p90": float(np.percentile(x, 90)),
            "n": int(x.size)}


STAGE_NAMES = ("qkv", "attn", "wo", "gateup", "down", "lmhead", "mix")


def time_stages(sess, one, steps):
    """Average launch time (us) of every stage kernel over `steps` grouped
    steps, from HIP events the library records around each launch on its
    stream (a separate pass: the event pairs add a few us per step)."""
    import torch
    from paper_2608_12385_amd import binding
    for n in STAGE_NAMES:
        binding.dbt_stage_timing(sess.model, binding.STAGES[n], 1)
    torch.cuda.synchronize()
    for _ in range(steps):
        one()
    torch.cuda.synchronize()
    res = {}
    for n in STAGE_NAMES:
        ms, cnt = binding.dbt_stage_time(sess.model, binding.STAGES[n])
        binding.dbt_stage_timing(sess.model, binding.STAGES[n], 0)
        res[n] = ms * 1e3 / max(cnt, 1)
    return res


def stage_bytes(shape, B, L):
    """Algorithmic bytes per launch of each stage kernel at batch B, cache L:
    the weights the kernel reads once (the attention: the live cache)."""
    d, dq, dkv, f, V = shape.d_model, shape.d_q, shape.d_kv, shape.d_ff, shape.vocab
    return {"qkv": (dq + 2 * dkv) * d * 2, "attn": B * (L + 1) * 2 * dkv * 2, "wo": d * dq * 2,
            "gateup": 2 * f * d * 2, "down": d * f * 2, "lmhead": V * d * 2}


def cpu_baseline(shape, W, h, L, B, seconds_per_mode):
    """The oracle as it stands on the same workload, per mode: whole steps of
    all B sequences (each truncated back to L cached positions, as in the
    timed GPU steps) until seconds_per_mode have passed, for the grouped
    step, the primary-only step and the two-pass step.  The oracle's one-time
    parameter widening is done before the clocks start."""
    import synth
    from oracle import Oracle
    try:
        import threadpoolctl
        threads = max([i.get("num_threads", 1) for i in threadpoolctl.threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threads = os.cpu_count()
    orc = Oracle(shape, W.values)
    for b in range(B):
        (k, _), (v, _) = synth.make_kv(shape, 0, b, L, seed=3)
        orc.kv_fill(b, L, [k], [v])
    for name in list(W.values):
        orc.w(name)                      # widen the parameters once
    modes = {"grouped": dict(branch_on=True, grouped=True), "primary_only": dict(branch_on=False),
             "ungrouped": dict(branch_on=True, grouped=False)}
    per = {}
    for mode, kw in modes.items():
        steps = 0
        t0 = time.perf_counter()
        while True:
            orc.decode_step(h1=h[0], h2=h[1], **kw)
            for b in range(B):
                orc.truncate(b, L)
            steps += 1
            dt = time.perf_counter() - t0
            if dt >= seconds_per_mode or steps >= 64:
                break
        per[mode] = {"tokens_per_s": steps * B / dt, "step_s": dt / steps, "steps": steps}
    return dict(value=per["grouped"]["tokens_per_s"], unit="tokens/s", cores=int(threads), kind="oracle",
                sample=f"whole steps of all {B} sequences per mode (float64 NumPy oracle): "
                       + ", ".join(f"{m} {v['steps']} steps in {v['step_s'] * v['steps']:.1f} s"
                                   for m, v in per.items()),
                per_mode={m: v["tokens_per_s"] for m, v in per.items()})


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
    nb = max(1, shape.n_branches)
    h = synth.make_hidden(shape, B, step=0, seed=2, paths=1 + nb)
    h1d = torch.from_numpy(np.ascontiguousarray(h[0])).cuda()
    h2d = torch.from_numpy(np.ascontiguousarray(h[1] if nb == 1 else h[1:])).cuda()
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
    if nb > 1:
        rec["n_branches"] = nb
    if shape.is_moe:
        rec["k1"], rec["k2"] = shape.top_k1, shape.top_k2
        rec["compute_matched"] = bool(shape.compute_matched)
        rec["note"] = "bytes depend on the touched experts; see profiles"
    else:
        mlp = 3 * d * shape.d_ff * 2
        head = shape.vocab * d * 2
        rec["algorithmic_MB"] = (attn_w + mlp + head + kv) / 1e6
        rec["GBps"] = (attn_w + mlp + head + kv) / res["grouped"] / 1e9
    return rec


def time_full24(steps):
    """The full dense model: prefill of all prompts (primary path), then greedy
    grouped steps with the branch on, then the same number with the branch
    off (caches truncated back to the prompt), tokens fed back on the device."""
    import torch
    import synth
    from paper_2608_12385_amd import Session, binding
    w = synth.workload("full24_bf16")
    shape = w["shape"]
    B, T = w["batch"], w["prompt_len"]
    steps = steps or w["steps"]
    W = synth.make_weights(shape, seed=0)
    sess = Session(shape, {k: W.device_array(k) for k in W.values}, max_batch=B, max_pos=T + steps + 16,
                   max_prompt=T)
    del W
    prompts = [synth.make_tokens(1, 1000 + b, (T,), shape.vocab) for b in range(B)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    t = sess.prefill(prompts, run_boundary=True)
    torch.cuda.synchronize()
    t_pre = time.perf_counter() - t0
    first = t["next_token"].clone()
    res = {}
    for mode in ("on", "off"):
        for b in range(B):
            binding.dbt_kv_truncate(sess.kv, b, T)
        tok = first.clone()
        outs = [sess.outputs(B, logits=False, hidden=False) for _ in range(2)]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(steps):
            out, tt = outs[i % 2]
            binding.dbt_decode_step(sess.model, sess.kv, sess.step_in(B, tok), 1 if mode == "on" else 0, out,
                                    sess.stream)
            tok = tt["next_token"]
        torch.cuda.synchronize()
        res[mode] = time.perf_counter() - t0
    sess.close()
    return {"workload": "full24_bf16", "batch": B, "prompt_len": T, "steps": steps,
            "prefill_s": t_pre, "prefill_tokens_per_s": B * T / t_pre,
            "decode_step_us_branch_on": res["on"] / steps * 1e6, "decode_step_us_branch_off": res["off"] / steps * 1e6,
            "decode_tokens_per_s_branch_on": B * steps / res["on"],
            "decode_tokens_per_s_branch_off": B * steps / res["off"],
            "end_to_end_tokens_per_s_branch_on": B * steps / (t_pre + res["on"]),
            "end_to_end_tokens_per_s_branch_off": B * steps / (t_pre + res["off"]),
            "branch_overhead_pct": 100 * (res["on"] - res["off"]) / res["off"]}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    # the GPU's clocks settle over the first few tens of steps: warm up long
    # enough that the timed block sees the steady state (0.4 ms per step)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=8.0,
                    help="minimum CPU time of the oracle baseline per mode (whole steps)")
    ap.add_argument("--protocol-iters", type=int, default=100,
                    help="timed iterations of the interleaved three-mode measurement")
    ap.add_argument("--protocol-warmup", type=int, default=10,
                    help="untimed iterations before the interleaved measurement")
    ap.add_argument("--all", action="store_true",
                    help="also time the long-context and MoE workloads (extra fields)")
    ap.add_argument("--calib-copy", action="store_true",
                    help="launch a plain 256 MiB device copy three times first (counter calibration)")
    ap.add_argument("--grouped-only", action="store_true",
                    help="time only the grouped step (counter runs: every dispatch after the calibration "
                         "copies belongs to a grouped step)")
    ap.add_argument("--only", metavar="WORKLOAD", choices=("layer8b_bf16", "longctx_bf16", "moe_bf16", "full24_bf16",
                                                         "tp8shard_bf16"),
                    help="time only this other workload (one JSON line of its fields)")
    ap.add_argument("--top-k2", type=int, default=4, help="branch fan-out of --only moe_bf16")
    ap.add_argument("--full24-steps", type=int, default=0,
                    help="--only full24_bf16: greedy steps per mode (0: the workload's 256)")
    ap.add_argument("--branches", type=int, default=1,
                    help="--only layer8b_bf16/longctx_bf16: decode branches (App. C.1 of the paper)")
    ap.add_argument("--compute-matched", action="store_true",
                    help="--only moe_bf16: the compute-matched variant (App. B.3 of the paper)")
    ap.add_argument("--kernel-table", metavar="DB", help="print the kernel-duration table of a rocprofv3 database")
    ap.add_argument("--traffic-summary", nargs=2, metavar=("FETCH_DB", "WRITE_DB"),
                    help="print the calibrated LM-head traffic from two rocprofv3 --pmc databases")
    args = ap.parse_args()
    if args.kernel_table:
        print(kernel_table(args.kernel_table))
        return
    if args.traffic_summary:
        print(traffic_summary(*args.traffic_summary))
        return
    if args.gpus != 1:
        print("bench.py measures one GPU: the library runs the decode path on a single MI355X "
              "(sharding is described, not built); use --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    import synth
    from paper_2608_12385_amd import Session

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    if args.only == "full24_bf16":
        print(json.dumps(time_full24(args.full24_steps)))
        return
    if args.only:
        kw = ({"top_k2": args.top_k2, "compute_matched": args.compute_matched} if args.only == "moe_bf16"
              else {"n_branches": args.branches})
        print(json.dumps(time_workload(args.only, args.steps, args.warmup, **kw)))
        return
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

    if args.calib_copy:
        src = torch.empty(CALIB_BYTES // 4, dtype=torch.float32, device="cuda").fill_(1.0)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    fns = {m: step_fn(sess, B, L, h1d, h2d, m) for m in ("grouped", "primary", "ungrouped")}
    # the contract's timed block: exactly K grouped steps after W warm-ups
    t_grp = time_block(fns["grouped"], args.steps, args.warmup)
    proto = stages = None
    if not args.grouped_only:
        # the measurement protocol: the three modes interleaved, each step
        # timed by HIP events; median, p10 and p90 per mode
        us = time_interleaved(fns, args.protocol_iters, args.protocol_warmup)
        proto = {m: dist(v) for m, v in us.items()}
        paired = [100.0 * (g - p) / p for g, p in zip(us["grouped"], us["primary"])]
        proto["overhead_pct_paired"] = dist(paired)
    stages = time_stages(sess, fns["grouped"], max(args.steps, 20))

    traffic_lm, traffic_step = recorded_traffic()
    layer_b, head_b, kv_b = algorithmic_bytes(shape, B, L)
    step_bytes = layer_b + head_b + kv_b
    logit_bytes = 2 * B * shape.vocab * 4
    sb = stage_bytes(shape, B, L)
    lm_s = stages["lmhead"] / 1e6
    lm_gbps = sb["lmhead"] / lm_s / 1e9
    med = (lambda m: proto[m]["median"]) if proto else (lambda m: float("nan"))
    t_med = med("grouped") if proto else t_grp * 1e6
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
        "step_us": t_med,
        "step_us_block_mean": t_grp * 1e6,
        "primary_only_us": med("primary"),
        "ungrouped_us": med("ungrouped"),
        "branch_overhead_pct": 100.0 * (med("grouped") - med("primary")) / med("primary"),
        "protocol": None if proto is None else {
            "iterations": args.protocol_iters, "warmup": args.protocol_warmup,
            "order": "grouped, primary-only, ungrouped interleaved per iteration; HIP events per step",
            "grouped_us": proto["grouped"], "primary_only_us": proto["primary"],
            "ungrouped_us": proto["ungrouped"], "branch_overhead_pct_paired": proto["overhead_pct_paired"]},
        "algorithmic_MB_per_step": step_bytes / 1e6,
        "step_GBps": step_bytes / t_med * 1e6 / 1e9,
        "step_frac_of_peak": step_bytes / t_med * 1e6 / 1e9 / HBM_PEAK_GBPS,
        "step_traffic_MB": None if traffic_step is None else traffic_step / 1e6,
        "step_traffic_vs_algorithmic": None if traffic_step is None else traffic_step / step_bytes,
        "stages": {n: {"launch_us": stages[n],
                       **({"algorithmic_MB": sb[n] / 1e6, "GBps": sb[n] / stages[n] / 1e3,
                           "frac": sb[n] / stages[n] / 1e3 / HBM_PEAK_GBPS} if n in sb else {})}
                   for n in STAGE_NAMES},
        "stages_note": "grouped step; launch times from library HIP events on the step's stream (separate pass); "
                       "the remainder of the step is the row kernels (norms, rotary/append, split sums, "
                       "coupling) and launch gaps",
        "roofline": {
            "kernel": "LM-head projection (k_gemm_bf16, 64 stacked rows)",
            "bound": "hbm",
            "achieved": lm_gbps,
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": lm_gbps / HBM_PEAK_GBPS,
            "traffic": traffic_lm,
            "launch_us": stages["lmhead"],
            "algorithmic_MB_per_launch": sb["lmhead"] / 1e6,
            "algorithmic_note": "the output matrix read once (vocab x d_model bf16); the fp32 logits it also "
                                "writes are counted in traffic, not here",
            "logits_written_MB_per_launch": logit_bytes / 1e6,
        },
    }
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(shape, W, h, L, B, args.cpu_seconds)
    sess.close()
    if args.all:
        del W
        extra = [time_workload("longctx_bf16", args.steps, args.warmup)]
        for k2 in (2, 4, 8):
            extra.append(time_workload("moe_bf16", args.steps, args.warmup, top_k2=k2))
        extra.append(time_workload("moe_bf16", args.steps, args.warmup, top_k2=2, compute_matched=True))
        for nb in (2, 3):
            extra.append(time_workload("layer8b_bf16", args.steps, args.warmup, n_branches=nb))
        line["other_workloads"] = extra
    print(json.dumps(line))


if __name__ == "__main__":
    main()
