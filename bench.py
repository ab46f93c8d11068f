#!/usr/bin/env python3
"""Benchmark of one chunked-prefill scheduling iteration's attention step on MI355X.

A step is cp_kv_append + cp_attn_mixed over one batch of synthetic input (the
whole hot path: planner, append, prefill-MFMA, decode split-K, merge).  With
no flags it runs the Llama-3-8B-shaped mix with a 512-token budget (32 q / 8
kv heads, head_dim 128, block 16; 2 prefill chunks of 192 tokens + 128
decode rows) on one GPU and prints one JSON line.

  python bench.py [--gpus 1] [--steps K] [--warmup W] [--config N] [--all]

``--config 5`` replays the 20-iteration 70B-shaped schedule (a step is one
iteration, iterations cycle).  ``--all`` prints one line per mix.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "mixed-batch attention tokens/s + per-iteration latency; % MFMA / % HBM peak"
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E
PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
CONFIG_DESC = {
    1: "tiny mix: 4/2 heads, head_dim 64, block 16; chunks 64@0, 48@128; decodes ctx 200, 37",
    2: "Llama-3-8B attention layer, budget 512: 32/8 heads, head_dim 128, block 16; "
       "2 prefill chunks x 192 (prior ctx U[0,4096]) + 128 decode rows (ctx lognormal median 1024)",
    3: "Llama-3-8B prefill-heavy, budget 2048: 4 chunks x 480 at prior ctx 0/8192/16384/31744 "
       "+ 128 decode rows (ctx lognormal median 2048, max 32768)",
    4: "Llama-3-8B decode-dominated: 256 decode rows (70% lognormal median 512, 30% U[8k,32k]) "
       "+ one 256-token chunk at ctx 0",
    5: "70B-shaped layer (64/8 heads, head_dim 128, block 32), budget 4096: 20-iteration "
       "aging/APC schedule replay over 64 requests",
}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


# --------------------------------------------------------------------------- work accounting

def work_of(batch):
    """Algorithmic flops and HBM bytes of one step, split by kernel kind.

    prefill row (c tokens after s cached):  4*D*Hq*(c*s + c(c+1)/2) flops
    any row:  K+V of ctx keys once per kv head (4*Hkv*D*ctx bytes), q read and
              out written once (4*Hq*D*c), block-table entries (4*ceil(ctx/B))
    append:   8*Hkv*D*T bytes (new K/V read, cache slots written)
    """
    Hq, Hkv, D, B = batch.num_q_heads, batch.num_kv_heads, batch.head_dim, batch.block_size
    w = {"prefill_flops": 0, "prefill_bytes": 0, "decode_bytes": 0, "decode_flops": 0}
    for _, s, c, ctx in batch.rows.tolist():
        if c == 0:
            continue
        byt = 4 * Hkv * D * ctx + 4 * Hq * D * c + 4 * (-(-ctx // B))
        fl = 4 * D * Hq * (c * s + c * (c + 1) // 2)
        if c >= 2:
            w["prefill_flops"] += fl
            w["prefill_bytes"] += byt
        else:
            w["decode_flops"] += fl
            w["decode_bytes"] += byt
    w["append_bytes"] = 8 * Hkv * D * batch.num_tokens
    return w


def kernel_sha(name):
    with open(os.path.join(ROOT, "paper_2606_09061_amd", "csrc", name), "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def traffic_for(kernel, workload):
    """HBM bytes per launch from committed rocprofv3 counter runs, if they
    were taken on the current kernel source; else None."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    try:
        with open(path) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    ent = rec.get(f"{kernel}:{workload}")
    if not ent or ent.get("src_sha") != kernel_sha(f"{kernel}.hip"):
        return None
    return ent.get("bytes_per_launch")


# --------------------------------------------------------------------------- cpu baseline

def cpu_baseline(batches, host_caches, tensors_host, budget_s=10.0, seed=0):
    """The fp64 oracle on a uniform random sample of (token, q head) outputs of
    the first batch, timed on all host cores; tokens/s scaled from the sample."""
    import numpy as np
    import oracle

    batch = batches[0]
    kc0, vc0 = host_caches
    kc, vc = oracle.kv_append(batch, tensors_host["k_new"], tensors_host["v_new"], kc0, vc0)
    total = batch.num_tokens * batch.num_q_heads
    rng = np.random.default_rng(seed)
    pilot = rng.choice(total, size=min(total, 64), replace=False)
    t0 = time.perf_counter()
    oracle.attn(batch, tensors_host["q"], kc, vc, sel=pilot)
    per = (time.perf_counter() - t0) / len(pilot)
    n = int(min(total, max(len(pilot), budget_s / max(per, 1e-9))))
    sel = rng.choice(total, size=n, replace=False)
    t0 = time.perf_counter()
    oracle.attn(batch, tensors_host["q"], kc, vc, sel=sel)
    dt = time.perf_counter() - t0
    tok = n / batch.num_q_heads
    return {"value": tok / dt, "unit": "tokens/s", "cores": oracle.num_threads(), "kind": "oracle",
            "sample": f"{n} of {total} (token, q head) outputs drawn uniformly "
                      f"({100.0 * n / total:.1f}%), fp64, {dt:.2f} s"}


# --------------------------------------------------------------------------- gpu run

def build_inputs(cfg, device):
    import workloads as wl
    if cfg == 5:
        batches, _ = wl.replay_schedule()
        kc, vc = wl.make_caches(batches[0], device=device, fill_prior=False, seed=5000)
        steps = []
        for i, b in enumerate(batches):
            q, kn, vn, _ = wl.make_step_tensors(b, 5100 + i, device)
            steps.append({"q": q, "k_new": kn, "v_new": vn})
        shared = {"k_cache": kc, "v_cache": vc}
        return batches, steps, shared
    b = wl.make_config(cfg)
    t = wl.make_tensors(b, seed=1000 + cfg, device=device)
    steps = [{"q": t["q"], "k_new": t["k_new"], "v_new": t["v_new"]}]
    return [b], steps, {"k_cache": t["k_cache"], "v_cache": t["v_cache"]}


def run_config(cfg, steps_n, warmup, with_cpu=True, cpu_budget=10.0):
    import numpy as np
    import torch
    import paper_2606_09061_amd as cp
    from paper_2606_09061_amd import binding

    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    log(f"[bench] building inputs for mix {cfg}")
    batches, steps, shared = build_inputs(cfg, dev)
    host = None
    if with_cpu:
        host = ((shared["k_cache"].cpu().view(torch.int16).numpy().view(np.uint16),
                 shared["v_cache"].cpu().view(torch.int16).numpy().view(np.uint16)),
                {k: v.cpu() for k, v in steps[0].items()})
    descs = [cp.desc_for(b) for b in batches]
    tables = [torch.from_numpy(b.block_tables).to(dev) for b in batches]
    ws_bytes = max(cp.workspace_bytes(d, b.rows) for d, b in zip(descs, batches))
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    outs = [torch.empty(b.num_tokens, b.num_q_heads, b.head_dim, dtype=torch.bfloat16, device=dev)
            for b in batches]
    stream = torch.cuda.current_stream()

    def step(i):
        j = i % len(batches)
        b, d, t = batches[j], descs[j], steps[j]
        cp.kv_append(d, t["k_new"], t["v_new"], shared["k_cache"], shared["v_cache"], tables[j],
                     b.rows, ws, stream=stream)
        cp.attn_mixed(d, t["q"], shared["k_cache"], shared["v_cache"], tables[j], b.rows, outs[j],
                      ws, stream=stream)

    if cfg == 5:
        # the replay's caches are built by its own appends: run the iterations
        # once in order before timing so every later step reads real context
        for i in range(len(batches)):
            step(i)
    for i in range(warmup):
        step(i)
    torch.cuda.synchronize()
    log(f"[bench] warmup done ({warmup} steps); timing {steps_n} steps")
    def timed(n, detail):
        """n steps between two events on the step stream; with ``detail`` also
        an event after every step and the library's per-kernel event pairs."""
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(n + 1 if detail else 2)]
        if detail:
            binding.profile_begin()
        torch.cuda.synchronize()
        w0 = time.perf_counter()
        evs[0].record(stream)
        for i in range(n):
            step(i)
            if detail:
                evs[i + 1].record(stream)
        if not detail:
            evs[1].record(stream)
        torch.cuda.synchronize()
        wall_s = time.perf_counter() - w0
        prof_ = binding.profile_end() if detail else None
        per = (np.array([evs[i].elapsed_time(evs[i + 1]) for i in range(n)]) if detail else None)
        return float(evs[0].elapsed_time(evs[-1])), wall_s, per, prof_

    # headline region: only the two bracketing events
    total_ms, wall, _, _ = timed(steps_n, False)
    # second region, same steps: per-step latencies and per-kernel durations
    _, _, per_step, prof = timed(steps_n, True)
    tokens = sum(batches[i % len(batches)].num_tokens for i in range(steps_n))
    log(f"[bench] timed region {total_ms:.3f} ms (wall {wall * 1e3:.3f} ms)")

    # algorithmic work over the timed steps
    works = [work_of(batches[i % len(batches)]) for i in range(steps_n)]
    tot = {k: sum(w[k] for w in works) for k in works[0]}
    kern = {k: {"ms_per_step": v[0] / steps_n, "launches": v[1]} for k, v in prof.items()}
    dominant = max(("prefill", "decode"), key=lambda k: prof[k][0])
    wl_name = CONFIG_NAMES_SHORT[cfg]
    if dominant == "prefill":
        avg_ms = prof["prefill"][0] / max(1, prof["prefill"][1])
        per_launch = tot["prefill_flops"] / max(1, prof["prefill"][1])
        achieved = per_launch / (avg_ms * 1e-3) / 1e12
        roof = {"bound": "mfma", "kernel": "prefill", "achieved": achieved,
                "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s", "frac": achieved / PEAK_BF16_TFLOPS,
                "avg_launch_ms": avg_ms, "work_per_launch": per_launch}
    else:
        avg_ms = prof["decode"][0] / max(1, prof["decode"][1])
        per_launch = tot["decode_bytes"] / max(1, prof["decode"][1])
        achieved = per_launch / (avg_ms * 1e-3) / 1e9
        roof = {"bound": "hbm", "kernel": "decode", "achieved": achieved, "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": achieved / PEAK_HBM_GBS, "avg_launch_ms": avg_ms,
                "work_per_launch": per_launch}
    roof["traffic"] = traffic_for(roof["kernel"], wl_name)
    # the other kernel's fraction, for mixes where both matter
    other = {}
    if prof["prefill"][1] and dominant != "prefill":
        a = tot["prefill_flops"] / (prof["prefill"][0] * 1e-3) / 1e12
        other["prefill_tflops"] = a
        other["prefill_frac_mfma"] = a / PEAK_BF16_TFLOPS
    if prof["decode"][1] and dominant != "decode":
        a = tot["decode_bytes"] / (prof["decode"][0] * 1e-3) / 1e9
        other["decode_gbs"] = a
        other["decode_frac_hbm"] = a / PEAK_HBM_GBS

    b0 = batches[0]
    res = {
        "metric": METRIC,
        "value": tokens / (total_ms * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": steps_n,
        "warmup": warmup,
        "ms_per_step": total_ms / steps_n,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) bf16 q/k/v, seeded batch metadata and block tables)",
        "config": {"workload": f"{wl_name}: {CONFIG_DESC[cfg]}",
                   "heads_q_kv": [b0.num_q_heads, b0.num_kv_heads], "head_dim": b0.head_dim,
                   "block_size": b0.block_size,
                   "tokens_per_step": tokens / steps_n, "iterations": len(batches),
                   "parallelism": "single GPU"},
        "latency_ms": {"median": float(np.median(per_step)),
                       "p10": float(np.percentile(per_step, 10)),
                       "p90": float(np.percentile(per_step, 90))},
        "wall_ms_per_step": wall * 1e3 / steps_n,
        "kernels": kern,
        "roofline": roof,
        "other_kernel": other,
    }
    if with_cpu:
        log("[bench] timing the fp64 oracle on a host sample")
        sub = [batches[0]]
        res["cpu_baseline"] = cpu_baseline(sub, host[0], host[1], budget_s=cpu_budget)
    else:
        res["cpu_baseline"] = None
    return res


CONFIG_NAMES_SHORT = {1: "tiny", 2: "llama3-8b-budget512", 3: "llama3-8b-prefill-heavy",
                      4: "llama3-8b-decode-dominated", 5: "llama-70b-replay"}


def copy_calibration(mib, reps):
    """Plain device-to-device copies of a known size, for scaling the HBM byte
    counters (FETCH_SIZE / WRITE_SIZE) of a profiler run."""
    import torch
    n = mib << 20
    src = torch.ones(n, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes_per_launch": n, "launches": reps}), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", type=int, default=2, choices=[1, 2, 3, 4, 5])
    ap.add_argument("--all", action="store_true", help="one JSON line per mix")
    ap.add_argument("--no-cpu", action="store_true", help="skip the oracle CPU baseline")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run plain copies of MIB MiB (counter calibration)")
    args = ap.parse_args()
    if args.copy_calibration:
        copy_calibration(args.copy_calibration, args.steps)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for {args.gpus}): the attention step is "
              "measured on a single MI355X; a multi-GPU run would shard heads across GPUs with "
              "no collective inside the step and is not part of this build.", file=sys.stderr)
        sys.exit(2)
    cfgs = [1, 2, 3, 4, 5] if args.all else [args.config]
    for c in cfgs:
        res = run_config(c, args.steps, args.warmup, with_cpu=not args.no_cpu,
                         cpu_budget=args.cpu_seconds)
        print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
