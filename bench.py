#!/usr/bin/env python3
"""Benchmark of one chunked-prefill scheduling iteration's attention step on MI355X.

A step is cp_kv_append + cp_attn_mixed over one batch of synthetic input (the
whole hot path: planner, append, prefill-MFMA, decode split-K, merge), issued
as one cp_step_mixed call.  With
no flags it runs the 70B-shaped mix (64 q / 8 kv heads, head_dim 128, block
32, token budget 4096): a 20-iteration replay of an aging/APC schedule over
64 requests, one iteration per step, cycling, on one GPU, and prints one JSON
line.

  python bench.py [--gpus 1] [--steps K] [--warmup W] [--config N] [--all]
                  [--sub prefill|decode] [--cold N] [--no-cpu] [--settle S]
  python bench.py --peaks
  python bench.py --latency-table out.csv
  python bench.py --fit out.csv

``--config N`` picks another mix (1 tiny, 2 Llama-3-8B budget 512, 3 prefill-
heavy, 4 decode-dominated).  ``--all`` prints one line per mix.  ``--sub``
times only the prefill rows or only the decode rows of the mix (same pools);
``--cold`` adds steps timed after flushing the caches.  Before the warm-up the
steps run back to back for ``--settle`` seconds (default 1) so that the timed
region starts at the clock the GPU holds under load, not during its ramp from
idle.
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
    # decode rows whose work the planner placed inside the prefill launch
    w["fused_decode_bytes"] = w["decode_bytes"] if decode_fused(batch) else 0
    return w


def decode_fused(batch):
    """Whether the step runs its decode rows as decode blocks of its prefill
    launch (the plan's record lists name decode blocks)."""
    import paper_2606_09061_amd as cp
    d = cp.desc_for(batch)
    return any((cp.plan_records(d, batch.rows, w)[:, 1] == -1).any() for w in (0, 1))


def kernel_sha(*names):
    """Hash of the given sources and of every local header they include, so
    counters taken on other code are never reported."""
    import re
    csrc = os.path.join(ROOT, "paper_2606_09061_amd", "csrc")
    h, seen, todo = hashlib.sha256(), set(), list(names)
    while todo:
        fn = todo.pop(0)
        if fn in seen:
            continue
        seen.add(fn)
        with open(os.path.join(csrc, fn), "rb") as f:
            text = f.read()
        h.update(fn.encode() + b"\0" + text)
        todo += [m.decode() for m in re.findall(rb'#include\s+"([^"]+)"', text)
                 if os.path.exists(os.path.join(csrc, m.decode()))]
    return h.hexdigest()[:16]


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
    # the kernel's source with its headers, and the planner that sizes its
    # work items and key splits (both change the bytes a launch moves)
    if not ent or ent.get("src_sha") != kernel_sha(f"{kernel}.hip", "plan.cpp"):
        return None
    return ent.get("bytes_per_launch")


# --------------------------------------------------------------------------- cpu baseline

def cpu_baseline(batches, pools0, steps_host, budget_s=10.0, seed=0):
    """The fp64 oracle timed on all host cores over a uniform random sample of
    the (token, q head) outputs of every batch, in order.  Each batch's pools
    are rebuilt on the host by the oracle's own append, batch after batch, in
    ``pools0`` (written in place), so every sampled output reads the context
    it reads on the GPU.  Batch i's outputs are each drawn with probability
    f_i, set from the seconds per key read measured so far (a warmed-up pilot
    first) so that the timed work comes to about ``budget_s``; the whole job's
    time is estimated as sum(t_i / f_i) over the batches' timed calls, and
    tokens/s = all tokens / that time.  Only the attention calls are timed
    (the append is a bit copy, under 0.1 % of the oracle's work)."""
    import numpy as np
    import oracle

    rng = np.random.default_rng(seed)
    Hq = batches[0].num_q_heads

    def keys_per_output(b):  # keys each (token, head) output reads, flat t*Hq+h order
        pos = np.concatenate([np.arange(s_, s_ + c_) for _, s_, c_, _ in b.rows.tolist()] or
                             [np.zeros(0, np.int64)])
        return np.repeat(pos + 1, Hq)

    kpos = [keys_per_output(b) for b in batches]
    keys_left = float(sum(int(k.sum()) for k in kpos))
    kc, vc = pools0
    per_key, spent, keys_timed, est_total, n_out, n_all, fs = None, 0.0, 0, 0.0, 0, 0, []
    for i, b in enumerate(batches):
        kc, vc = oracle.kv_append(b, steps_host[i]["k_new"], steps_host[i]["v_new"], kc, vc,
                                  inplace=True)
        kpo = kpos[i]
        n_all += kpo.size
        if kpo.size == 0:
            continue
        if per_key is None:  # pilot on the first batch, after one warm-up call
            oracle.attn(b, steps_host[i]["q"], kc, vc, sel=rng.choice(kpo.size, 16))
            pilot = rng.choice(kpo.size, size=min(kpo.size, 256), replace=False)
            t0 = time.perf_counter()
            oracle.attn(b, steps_host[i]["q"], kc, vc, sel=pilot)
            per_key = (time.perf_counter() - t0) / max(1, int(kpo[pilot].sum()))
        f = min(1.0, max(1e-4, (budget_s - spent) / max(per_key * keys_left, 1e-9)))
        fs.append(f)
        keys_left -= float(kpo.sum())
        sel = np.nonzero(rng.random(kpo.size) < f)[0]
        if sel.size == 0:
            continue
        t0 = time.perf_counter()
        oracle.attn(b, steps_host[i]["q"], kc, vc, sel=sel)
        dt = time.perf_counter() - t0
        spent += dt
        est_total += dt / f
        keys_timed += int(kpo[sel].sum())
        per_key = spent / max(1, keys_timed)
        n_out += sel.size
    tokens = n_all / Hq
    return {"value": tokens / est_total if est_total > 0 else None, "unit": "tokens/s",
            "cores": oracle.num_threads(), "kind": "oracle",
            "sample": f"{n_out} of {n_all} (token, q head) outputs over all {len(batches)} "
                      f"batch(es), drawn with per-batch probability {min(fs):.4f}-{max(fs):.4f}; "
                      f"fp64 attention only, {spent:.2f} s timed, whole job estimated as the sum "
                      f"of each batch's time / its probability"}


# --------------------------------------------------------------------------- gpu run

SUB_MASKS = {"prefill": lambda rows: rows[:, 2] >= 2, "decode": lambda rows: rows[:, 2] == 1}


def shard_heads(b, shard):
    """The batch as one GPU of a head-sharded (tensor-parallel) group of
    ``shard`` GPUs sees it: Hq / shard q heads and Hkv / shard kv heads of
    every row, same rows, block tables and scale."""
    import dataclasses
    if shard == 1:
        return b
    if b.num_kv_heads % shard:
        raise SystemExit(f"--shard {shard} does not divide {b.num_kv_heads} kv heads")
    return dataclasses.replace(b, name=f"{b.name}-tp{shard}",
                               num_q_heads=b.num_q_heads // shard,
                               num_kv_heads=b.num_kv_heads // shard)


def build_inputs(cfg, device, sub=None, shard=1):
    """Batches, per-batch step tensors, the shared pools, and for the replay
    the full batches that fill its pools (``prime``).  ``sub`` keeps only the
    prefill rows or only the decode rows of every batch (same pools);
    ``shard`` gives one GPU's heads of a head-sharded group."""
    import workloads as wl
    if cfg == 5:
        full, _ = wl.replay_schedule()
        full = [shard_heads(b, shard) for b in full]
        kc, vc = wl.make_caches(full[0], device=device, fill_prior=False, seed=5000)
        prime = []
        for i, b in enumerate(full):
            q, kn, vn, _ = wl.make_step_tensors(b, 5100 + i, device)
            prime.append((b, {"q": q, "k_new": kn, "v_new": vn}))
        if sub is None:
            return full, [t for _, t in prime], {"k_cache": kc, "v_cache": vc}, prime
        batches, steps = [], []
        for i, b in enumerate(full):
            sb = wl.subset(b, SUB_MASKS[sub](b.rows), sub)
            q, kn, vn, _ = wl.make_step_tensors(sb, 5300 + i, device)
            batches.append(sb)
            steps.append({"q": q, "k_new": kn, "v_new": vn})
        return batches, steps, {"k_cache": kc, "v_cache": vc}, prime
    b = shard_heads(wl.make_config(cfg), shard)
    t = wl.make_tensors(b, seed=1000 + cfg, device=device)
    shared = {"k_cache": t["k_cache"], "v_cache": t["v_cache"]}
    if sub is None:
        return [b], [{"q": t["q"], "k_new": t["k_new"], "v_new": t["v_new"]}], shared, []
    sb = wl.subset(b, SUB_MASKS[sub](b.rows), sub)
    q, kn, vn, _ = wl.make_step_tensors(sb, 1050 + cfg, device)
    return [sb], [{"q": q, "k_new": kn, "v_new": vn}], shared, []


def run_config(cfg, steps_n, warmup, with_cpu=True, cpu_budget=10.0, sub=None, cold=0,
               settle_s=1.0, shard=1):
    import numpy as np
    import torch
    import paper_2606_09061_amd as cp
    from paper_2606_09061_amd import binding

    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    log(f"[bench] building inputs for mix {cfg}" + (f" ({sub} rows only)" if sub else ""))
    batches, steps, shared, prime = build_inputs(cfg, dev, sub, shard)
    descs = [cp.desc_for(b) for b in batches]
    tables = [torch.from_numpy(b.block_tables).to(dev) for b in batches]
    ws_bytes = max([cp.workspace_bytes(d, b.rows) for d, b in zip(descs, batches)] +
                   [cp.workspace_bytes(cp.desc_for(b), b.rows) for b, _ in prime])
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    outs = [torch.empty(b.num_tokens, b.num_q_heads, b.head_dim, dtype=torch.bfloat16, device=dev)
            for b in batches]
    stream = torch.cuda.current_stream()

    two_calls = os.environ.get("CP_BENCH_TWO_CALLS") == "1"

    def step(i):
        # one step: the paged append, then the attention, as cp_step_mixed
        # (one call; CP_BENCH_TWO_CALLS=1: cp_kv_append then cp_attn_mixed)
        j = i % len(batches)
        b, d, t = batches[j], descs[j], steps[j]
        if two_calls:
            cp.kv_append(d, t["k_new"], t["v_new"], shared["k_cache"], shared["v_cache"],
                         tables[j], b.rows, ws, stream=stream)
            cp.attn_mixed(d, t["q"], shared["k_cache"], shared["v_cache"], tables[j], b.rows,
                          outs[j], ws, stream=stream)
        else:
            cp.step_mixed(d, t["q"], t["k_new"], t["v_new"], shared["k_cache"], shared["v_cache"],
                          tables[j], b.rows, outs[j], ws, stream=stream)

    if prime:
        # the replay's caches are built by its own appends: run the full
        # iterations once in order before timing so every step reads real context
        for b, t in prime:
            d = cp.desc_for(b)
            bt = torch.from_numpy(b.block_tables).to(dev)
            cp.kv_append(d, t["k_new"], t["v_new"], shared["k_cache"], shared["v_cache"], bt,
                         b.rows, ws, stream=stream)
            cp.attn_mixed(d, t["q"], shared["k_cache"], shared["v_cache"], bt, b.rows,
                          torch.empty(b.num_tokens, b.num_q_heads, b.head_dim,
                                      dtype=torch.bfloat16, device=dev), ws, stream=stream)
    torch.cuda.synchronize()
    host = None
    if with_cpu and sub is None:
        if prime:
            # the replay starts from empty (all-NaN) pools; the oracle rebuilds
            # each iteration's pools from them with the iterations' own K/V
            shape_k, shape_v = shared["k_cache"].shape, shared["v_cache"].shape
            pools0 = (np.full(tuple(shape_k), 0x7FC0, np.uint16),
                      np.full(tuple(shape_v), 0x7FC0, np.uint16))
            host = ([b for b, _ in prime], pools0,
                    [{k: v.cpu() for k, v in t.items()} for _, t in prime])
        else:  # the pools as the first timed step finds them
            host = (batches, (shared["k_cache"].cpu().view(torch.int16).numpy().view(np.uint16),
                              shared["v_cache"].cpu().view(torch.int16).numpy().view(np.uint16)),
                    [{k: v.cpu() for k, v in steps[0].items()}])
    # Clock settling: the GPU idles at ~0.1 GHz and its governor takes a few
    # hundred milliseconds of continuous work to reach the clock it holds under
    # this load (~2.1 GHz on the MFMA-heavy mixes, set by the power limit;
    # up to 2.4 GHz when lightly loaded).  A timed region of a few milliseconds
    # started from idle would measure that ramp, so whole cycles of the same
    # steps run back to back for `settle_s` first (untimed, like the warm-up).
    n_settle = 0
    t_settle = time.perf_counter()
    while time.perf_counter() - t_settle < settle_s:
        for _ in range(len(batches)):
            step(n_settle)
            n_settle += 1
    torch.cuda.synchronize()
    settle_wall = time.perf_counter() - t_settle
    for i in range(warmup):
        step(i)
    torch.cuda.synchronize()
    log(f"[bench] clock settling {n_settle} steps in {settle_wall:.2f} s; "
        f"warmup done ({warmup} steps); timing {steps_n} steps")
    def timed(n, mode):
        """n steps on the step stream.  mode "total": only two bracketing
        events; "steps": an event after every step as well; "kernels": the
        library's per-kernel event pairs instead (these add GPU time)."""
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(n + 1 if mode == "steps" else 2)]
        if mode == "kernels":
            binding.profile_begin()
        torch.cuda.synchronize()
        w0 = time.perf_counter()
        evs[0].record(stream)
        for i in range(n):
            step(i)
            if mode == "steps":
                evs[i + 1].record(stream)
        if mode != "steps":
            evs[1].record(stream)
        issue_s = time.perf_counter() - w0   # host time to enqueue the n steps
        torch.cuda.synchronize()
        wall_s = time.perf_counter() - w0
        prof_ = binding.profile_end() if mode == "kernels" else None
        per = (np.array([evs[i].elapsed_time(evs[i + 1]) for i in range(n)])
               if mode == "steps" else None)
        timed.issue_s = issue_s
        return float(evs[0].elapsed_time(evs[-1])), wall_s, per, prof_

    # headline region: only the two bracketing events
    total_ms, wall, _, _ = timed(steps_n, "total")
    issue = timed.issue_s
    # host cost of a step when nothing throttles the host: groups of 6 steps
    # issued onto an idle stream (the library stages up to 8 plans ahead, so
    # none of these waits for the GPU)
    free = []
    for i in range(0, min(steps_n, 60), 6):
        torch.cuda.synchronize()
        w0 = time.perf_counter()
        for k in range(6):
            step(i + k)
        free.append((time.perf_counter() - w0) / 6)
    torch.cuda.synchronize()
    # per-step latencies (at least 100 steps), then per-kernel durations
    n_lat = max(steps_n, 100)
    _, _, per_step, _ = timed(n_lat, "steps")
    _, _, _, prof = timed(n_lat, "kernels")
    tokens = sum(batches[i % len(batches)].num_tokens for i in range(steps_n))
    log(f"[bench] timed region {total_ms:.3f} ms (wall {wall * 1e3:.3f} ms)")

    # algorithmic work over the steps of each region
    def work_over(n):
        ws_ = [work_of(batches[i % len(batches)]) for i in range(n)]
        return {k: sum(w[k] for w in ws_) for k in ws_[0]}
    tot = work_over(n_lat)
    head = work_over(steps_n)
    kern = {k: {"ms_per_step": v[0] / n_lat, "launches": v[1]} for k, v in prof.items()}
    dominant = max(("prefill", "decode"), key=lambda k: prof[k][0])
    wl_name = CONFIG_NAMES_SHORT[cfg]
    if dominant == "prefill":
        n_launch = max(1, prof["prefill"][1])
        avg_ms = prof["prefill"][0] / n_launch
        per_launch = tot["prefill_flops"] / n_launch
        achieved = per_launch / (avg_ms * 1e-3) / 1e12
        roof = {"bound": "mfma", "kernel": "prefill", "achieved": achieved,
                "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s", "frac": achieved / PEAK_BF16_TFLOPS,
                "avg_launch_ms": avg_ms, "work_per_launch": per_launch}
        if tot["fused_decode_bytes"]:
            # The launch also runs the decode rows.  Its roofline time is the
            # larger of its flops at the MFMA peak and its algorithmic bytes
            # (the prefill rows' and the fused decode rows' K/V, q and out) at
            # the HBM peak; the bound is the one that needs longer, and
            # `frac` is that time over the launch's duration.
            # `prefill_flops_frac` charges the whole launch to the flops;
            # `fused_frac_serial` is both times summed over the duration.
            byt = (tot["prefill_bytes"] + tot["fused_decode_bytes"]) / n_launch
            t_m = per_launch / (PEAK_BF16_TFLOPS * 1e12)
            t_h = byt / (PEAK_HBM_GBS * 1e9)
            if t_h > t_m:
                a = byt / (avg_ms * 1e-3) / 1e9
                roof.update({"bound": "hbm", "achieved": a, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                             "frac": a / PEAK_HBM_GBS, "work_per_launch": byt})
            roof["kernel"] = "prefill (with the step's decode rows)"
            roof["prefill_flops_per_launch"] = per_launch
            roof["prefill_flops_frac"] = achieved / PEAK_BF16_TFLOPS
            roof["fused_bytes_per_launch"] = byt
            roof["fused_frac_serial"] = (t_m + t_h) / (avg_ms * 1e-3)
    else:
        avg_ms = prof["decode"][0] / max(1, prof["decode"][1])
        per_launch = tot["decode_bytes"] / max(1, prof["decode"][1])
        achieved = per_launch / (avg_ms * 1e-3) / 1e9
        roof = {"bound": "hbm", "kernel": "decode", "achieved": achieved, "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": achieved / PEAK_HBM_GBS, "avg_launch_ms": avg_ms,
                "work_per_launch": per_launch}
    # stored counter figures belong to the whole mix at its full head count
    roof["traffic"] = (traffic_for(roof["kernel"].split()[0], wl_name)
                       if sub is None and shard == 1 else None)
    # the other kernel's fraction, for mixes where both matter
    other = {}
    # the step against the roofline: t_pf = prefill flops at the MFMA peak,
    # t_hbm = decode + append bytes at the HBM peak, per headline step
    t_pf = head["prefill_flops"] / steps_n / (PEAK_BF16_TFLOPS * 1e12)
    t_hbm = (head["decode_bytes"] + head["append_bytes"]) / steps_n / (PEAK_HBM_GBS * 1e9)
    t_step = total_ms * 1e-3 / steps_n
    roof_step = {"t_pf_us": t_pf * 1e6, "t_hbm_us": t_hbm * 1e6,
                 "serialized_frac": (t_pf + t_hbm) / t_step,
                 "overlapped_frac": max(t_pf, t_hbm) / t_step}
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
        "config": {"workload": f"{wl_name}: {CONFIG_DESC[cfg]}" + (f" [{sub} rows only]" if sub else "")
                   + (f" [one GPU of a {shard}-way head shard]" if shard > 1 else ""),
                   "heads_q_kv": [b0.num_q_heads, b0.num_kv_heads], "head_dim": b0.head_dim,
                   "block_size": b0.block_size,
                   "tokens_per_step": tokens / steps_n, "iterations": len(batches),
                   "parallelism": "single GPU"},
        "latency_ms": {"median": float(np.median(per_step)),
                       "p10": float(np.percentile(per_step, 10)),
                       "p90": float(np.percentile(per_step, 90)), "reps": n_lat},
        "wall_ms_per_step": wall * 1e3 / steps_n,
        "host_issue_ms_per_step": issue * 1e3 / steps_n,
        "host_ms_per_step_unthrottled": float(np.median(free)) * 1e3,
        "kernels": kern,
        "roofline": roof,
        "roofline_step": roof_step,
        "other_kernel": other,
        "clock_settle": {"seconds": settle_wall, "steps": n_settle},
    }
    if cold:
        # cold steps: a 1 GiB buffer is rewritten before each (outside its
        # events), which evicts the 256 MB MALL and the L2s
        flush = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
        cold_ms = []
        for i in range(cold):
            flush.zero_()
            ea, eb = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            ea.record(stream)
            step(i)
            eb.record(stream)
            eb.synchronize()
            cold_ms.append(ea.elapsed_time(eb))
        res["cold_latency_ms"] = {"median": float(np.median(cold_ms)),
                                  "p10": float(np.percentile(cold_ms, 10)),
                                  "p90": float(np.percentile(cold_ms, 90)), "reps": cold}
        del flush
    if host is not None:
        log("[bench] timing the fp64 oracle on a host sample")
        res["cpu_baseline"] = cpu_baseline(host[0], host[1], host[2], budget_s=cpu_budget)
        if cfg in (1, 2):
            import oracle
            n_all = oracle.num_threads()
            oracle.set_threads(1)
            try:
                res["cpu_baseline_1thread"] = cpu_baseline(host[0], host[1], host[2],
                                                           budget_s=cpu_budget / 3)
            finally:
                oracle.set_threads(n_all)
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


def measured_peaks(reps=20):
    """Practical peaks of this GPU beside the datasheet ones: the device
    attributes behind the datasheet figures, a register-only bf16 MFMA loop
    (constant and random operands) and a streaming non-temporal read
    (libcppeaks.so), then plain library operations: a large bf16 GEMM
    (torch.matmul), a device copy and a read-only reduction."""
    import torch
    from paper_2606_09061_amd import peaks
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream(dev)
    info = peaks.device_info(0)
    # datasheet-style peak from the attributes: 4 SIMD x 512 bf16 flop per clock per CU
    info["bf16_tflops_at_attr_clock"] = info["compute_units"] * info["clock_khz"] * 1e3 * 2048 * 2 / 1e12

    def timed_ms(fn, n=reps):
        fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for _ in range(n):
            fn()
        b.record(stream)
        b.synchronize()
        return a.elapsed_time(b) / n

    ops = torch.randn(1 << 24, device=dev, dtype=torch.float32).to(torch.bfloat16)  # 32 MiB
    blocks, threads, iters = 4 * info["compute_units"], 256, 2000
    out = torch.empty(blocks * threads, device=dev, dtype=torch.float32)
    mfma = {}
    for rnd in (0, 1):
        ms = timed_ms(lambda: peaks.mfma_loop(ops, out, blocks, threads, iters, rnd, stream), 5)
        flops = 32768.0 * 16 * iters * (threads // 64) * blocks
        mfma["random" if rnd else "constant"] = flops / (ms * 1e-3) / 1e12
    del ops, out
    big = torch.empty(1 << 31, device=dev, dtype=torch.uint8).fill_(1)
    rblocks = 8 * info["compute_units"]
    rout = torch.empty(rblocks * 256, device=dev, dtype=torch.int32)
    t_rs = timed_ms(lambda: peaks.read_stream(big, rout, rblocks, stream)) * 1e-3
    del big, rout

    def timed(fn):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        b.synchronize()
        return a.elapsed_time(b) * 1e-3 / reps

    n = 8192
    x = torch.randn(n, n, device=dev, dtype=torch.bfloat16)
    y = torch.randn(n, n, device=dev, dtype=torch.bfloat16)
    t_mm = timed(lambda: torch.matmul(x, y))
    del x, y
    m = 1 << 31  # bytes
    src = torch.ones(m, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    t_cp = timed(lambda: dst.copy_(src))
    del dst
    f = src.view(torch.float32)
    t_rd = timed(lambda: f.sum())
    return {"measured_peaks": {
        "device": info,
        "mfma_loop_bf16_tflops": mfma,
        "read_stream_2gib_gbs": (1 << 31) / t_rs / 1e9,
        "bf16_gemm_8192_tflops": 2 * n ** 3 / t_mm / 1e12,
        "copy_2gib_gbs_read_plus_write": 2 * m / t_cp / 1e9,
        "sum_2gib_read_gbs": m / t_rd / 1e9,
        "datasheet": {"bf16_tflops": PEAK_BF16_TFLOPS, "hbm_gbs": PEAK_HBM_GBS}}}


def gpu_mem_mb():
    """The four GPU-memory features of the latency predictor's raw inputs
    (Table 1): device memory used and free, and the torch caching
    allocator's allocated and reserved bytes, in MB."""
    import torch
    free, total = torch.cuda.mem_get_info()
    mb = 1.0 / (1 << 20)
    return [round((total - free) * mb, 1), round(free * mb, 1),
            round(torch.cuda.memory_allocated() * mb, 1), round(torch.cuda.memory_reserved() * mb, 1)]


LT_DECODE_ROWS = (0, 16, 64, 128, 256)
LT_DECODE_CTX = (512, 2048, 8192)
LT_CHUNKS = (0, 1, 2, 4)
LT_CHUNK_LEN = (64, 256, 512, 1024)
LT_PRIOR = (0, 4096, 16384)


def latency_table(path, reps=5, seeds=(0, 1, 2)):
    """Latency-vs-composition sweep at the Llama-3-8B shape (32/8 heads,
    head_dim 128, block 16): decode rows x decode context median x prefill
    chunks x chunk length x prior context, three seeds each.  One pre-filled
    pool serves every composition; only block tables and metadata change.
    Columns: the raw and derived batch features of the paper's latency
    predictor (Table 1, Table 2), the exact
    query-key pair count, measured append / attention / step latency, and
    Table 1's four GPU-memory features (constant here: one pool serves every
    composition)."""
    import csv
    import math
    import numpy as np
    import torch
    import paper_2606_09061_amd as cp
    import workloads as wl
    from workloads.tensors import _randn_bf16

    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    hq, hkv, d, bsz = 32, 8, 128, 16
    pool = 560_000  # blocks (37 GB of K and V): 256 rows at the 32768 clip fit
    gen = torch.Generator(device=dev)
    gen.manual_seed(7000)
    kc = _randn_bf16((pool, hkv, bsz, d), gen, dev)
    vc = _randn_bf16((pool, hkv, d, bsz), gen, dev)
    stream = torch.cuda.current_stream()
    combos = []
    for nd in LT_DECODE_ROWS:
        for med in (LT_DECODE_CTX if nd else (0,)):
            for nc in LT_CHUNKS:
                for cl in (LT_CHUNK_LEN if nc else (0,)):
                    for pr in (LT_PRIOR if nc else (0,)):
                        if nd == 0 and nc == 0:
                            continue
                        combos.extend((nd, med, nc, cl, pr, sd) for sd in seeds)
    log(f"[bench] latency table: {len(combos)} compositions x {reps} reps")
    cols = ["decode_rows_cfg", "decode_ctx_median_cfg", "chunks_cfg", "chunk_len_cfg",
            "prior_cfg", "seed", "prefill_tokens", "decode_tokens", "batch_request_count",
            "sum_decode_context_len", "max_decode_context_len", "prefill_processed_tokens",
            "max_prefill_processed_tokens", "bias", "scheduled_tokens", "avg_decode_ctx",
            "decode_ctx_interaction", "prefill_interaction", "qk_pairs_per_head",
            "append_us", "attn_us", "step_us", "host_us",
            "gpu_mem_used_mb", "gpu_mem_free_mb", "cuda_allocated_mb", "cuda_reserved_mb"]
    ws = torch.empty(1 << 20, dtype=torch.uint8, device=dev)
    with open(path, "w", newline="") as fh:
        out = csv.writer(fh)
        out.writerow(cols)
        for k, (nd, med, nc, cl, pr, sd) in enumerate(combos):
            rng = np.random.default_rng([nd, med, nc, cl, pr, sd])
            sl = []
            if nd:
                ctx = np.clip(np.round(rng.lognormal(math.log(med), 1.0, nd)), 16, 32768)
                sl += [(int(c) - 1, 1) for c in ctx]
            sl += [(pr, cl)] * nc
            b = wl.make_batch("lt", hq, hkv, d, bsz, sl, rng, pool=pool)
            q, kn, vn, _ = wl.make_step_tensors(b, 7100 + k, dev)
            desc = cp.desc_for(b)
            bt = torch.from_numpy(b.block_tables).to(dev)
            need = cp.workspace_bytes(desc, b.rows)
            if need > ws.numel():
                ws = torch.empty(need, dtype=torch.uint8, device=dev)
            o = torch.empty(b.num_tokens, hq, d, dtype=torch.bfloat16, device=dev)
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
            t_app, t_att, t_host = [], [], []
            for r in range(reps + 2):
                torch.cuda.synchronize()
                h0 = time.perf_counter()
                ev[0].record(stream)
                cp.kv_append(desc, kn, vn, kc, vc, bt, b.rows, ws, stream=stream)
                ev[1].record(stream)
                cp.attn_mixed(desc, q, kc, vc, bt, b.rows, o, ws, stream=stream)
                ev[2].record(stream)
                h1 = time.perf_counter()
                ev[2].synchronize()
                if r >= 2:
                    t_app.append(ev[0].elapsed_time(ev[1]) * 1e3)
                    t_att.append(ev[1].elapsed_time(ev[2]) * 1e3)
                    t_host.append((h1 - h0) * 1e6)
            rows = b.rows
            dec = rows[rows[:, 2] == 1]
            pf = rows[rows[:, 2] >= 2]
            pf_tok = int(pf[:, 2].sum())
            dec_tok = int(dec.shape[0])
            sum_dctx = int(dec[:, 3].sum())
            processed = int(pf[:, 1].sum())
            pairs = int(sum(int(c) * int(s0) + int(c) * (int(c) + 1) // 2 for _, s0, c, _ in pf))
            avg_dctx = sum_dctx / max(dec_tok, 1)
            app, att = float(np.median(t_app)), float(np.median(t_att))
            out.writerow([nd, med, nc, cl, pr, sd, pf_tok, dec_tok, b.n_rows, sum_dctx,
                          int(dec[:, 3].max()) if dec_tok else 0, processed,
                          int(pf[:, 1].max()) if pf.size else 0, 1, pf_tok + dec_tok,
                          round(avg_dctx, 3), round(dec_tok * avg_dctx, 3), pf_tok * processed,
                          pairs, round(app, 2), round(att, 2), round(app + att, 2),
                          round(float(np.median(t_host)), 1), *gpu_mem_mb()])
            if k % 100 == 0:
                log(f"[bench] latency table {k}/{len(combos)}")
    res = {"latency_table": path, "compositions": len(combos), "reps": reps}
    res.update(fit_latency(path))
    return res


def fit_latency(path):
    """Least-squares fits of the measured step latency on the latency
    predictor's derived batch features (Table 2 of the paper: bias,
    scheduled_tokens, avg_decode_ctx, decode_ctx_interaction,
    prefill_interaction), and on the same set with prefill_interaction
    replaced by the exact query-key pair count of the prefill rows
    (sum c*s + c(c+1)/2).  Errors are MAE, RMSE and MAPE as the paper defines
    them for its predictor; also the median step latency per (decode rows,
    prefill chunks) cell."""
    import csv
    import numpy as np
    with open(path) as fh:
        rows = list(csv.DictReader(fh))
    y = np.array([float(r["step_us"]) for r in rows])

    def cols(names):
        return np.array([[float(r[n]) for n in names] for r in rows])

    base = ["bias", "scheduled_tokens", "avg_decode_ctx", "decode_ctx_interaction"]
    fits = {}
    for name, feats in (("table2", base + ["prefill_interaction"]),
                        ("table2_exact_pairs", base + ["qk_pairs_per_head"])):
        X = cols(feats)
        scale = np.abs(X).max(axis=0)
        scale[scale == 0] = 1.0
        w, *_ = np.linalg.lstsq(X / scale, y, rcond=None)
        e = (X / scale) @ w - y
        fits[name] = {"features": feats, "mae_us": float(np.abs(e).mean()),
                      "rmse_us": float(np.sqrt((e ** 2).mean())),
                      "mape_pct": float(100.0 * np.abs(e / y).mean())}
    grid = {}
    for r, v in zip(rows, y):
        grid.setdefault((int(r["decode_rows_cfg"]), int(r["chunks_cfg"])), []).append(v)
    cells = {f"{d}x{c}": float(np.median(v)) for (d, c), v in sorted(grid.items())}
    return {"fits": fits, "median_step_us_by_decode_rows_x_chunks": cells,
            "median_host_us": float(np.median([float(r["host_us"]) for r in rows]))}


# --------------------------------------------------------------------------- closed-loop scheduling

SCHED_BASE = dict(policy=0, max_tokens=1024, max_seqs=256, max_seq_len=4096, delta=32,
                  lambda_u=1.0, lambda_o=4.0, max_active=4, min_chunk=16)
# Per engine: slots, request inter-arrival times (us) of the high / regular
# load, the short-prompt (aging) stream and the busy / quiet phases of the
# short/long (APC) stream, stream sizes, the T* quantiles swept, and the
# aging ratios alpha/|beta| (tokens of remaining work per us of waiting; a
# model round is ~100x longer than a step, so its ratios are ~100x smaller
# for the same trade-off per round).
SCHED_PROFILES = {
    "step": dict(slots=256, high=150.0, regular=1500.0, aging=40.0, apc_busy=20.0,
                 apc_quiet=200.0, n_req=1000, n_collect=600, n_collect_regular=600,
                 regular_budgets=(256, 512, 1024, 2048), targets=("mean", "p75", "p90"),
                 aging_budgets=(128, 512), aging_ratios=(0.01, 0.1), n_regular=1000,
                 workload="qwen3-8b-attention-closed-loop"),
    "model": dict(slots=128, high=15000.0, regular=150000.0, aging=4000.0, apc_busy=2000.0,
                  apc_quiet=20000.0, n_req=500, n_collect=300, n_collect_regular=150,
                  regular_budgets=(1024,), targets=("p75", "p90"), aging_budgets=(128, 512),
                  aging_ratios=(1e-4, 1e-3),
                  n_regular=160, workload="qwen3-8b-36-layer-closed-loop"),
}


def sched_experiment(out_dir, engine="step", epochs=300, parts=("lprs", "aging", "apc")):
    """Closed-loop serving under the C++ scheduler, the clock advanced by each
    round's measured latency.  engine "step": the Qwen3-8B / Llama-3-8B
    attention step alone (32/8 heads, head_dim 128, block 16, 256 slots of up
    to 4,096 tokens); engine "model": the whole 36-layer synthetic Qwen3-8B
    iteration (128 slots), the quantity the paper's predictor targets.
      1. samples: the token-budget scheduler on uniform and short/long request
         streams at several budgets and loads (the paper's offline profiling,
         Sec. 3.2.1); each round gives the 16 features and the latency;
      2. the predictor: Table 7's MLP on the weighted asymmetric Huber loss,
         8:1:1 split, test accuracy as Table 8 (and a Table-2 linear fit);
      3. LPRS (Algorithm 1) against the token budget of 1,024 (Table 9's
         comparison) at high and regular load, with APC, for B_max 1,024 and
         2,048 and T* at quantiles of the token-budget run's round latency at
         high load (and LPRS alone at the 90th percentile);
      4. Aging against FCFS (Sec. 4.2) on a short-prompt-heavy stream;
      5. APC off / on under LPRS on the 49:1 short/long mix (Table 10), T* =
         the token-budget run's mean round latency on that stream, and again
         at its 90th percentile."""
    import numpy as np
    import torch
    import workloads as wl
    from paper_2606_09061_amd import lprs, sched, serve

    P = SCHED_PROFILES[engine]
    n_req, n_collect = P["n_req"], P["n_collect"]
    HIGH, REGULAR = P["high"], P["regular"]
    os.makedirs(out_dir, exist_ok=True)
    torch.cuda.set_device(0)
    if engine == "model":
        from paper_2606_09061_amd import model as M
        eng = M.ModelEngine(M.Model(M.QWEN3_8B, max_seqs=P["slots"], max_seq_len=4096,
                                    max_tokens=2048))
    else:
        eng = serve.StepEngine(max_seqs=P["slots"], max_seq_len=4096, max_tokens=2048)

    def cfg(**kw):
        d = dict(SCHED_BASE)
        d["max_seqs"] = P["slots"]
        d.update(kw)
        return sched.make_config(**d)

    def strip(r):
        return {k: v for k, v in r.items() if not k.startswith("_")}

    out = {"workload": P["workload"], "shape": "32/8 heads, d128, B16", "engine": engine,
           "slots": P["slots"], "high_interval_us": HIGH, "regular_interval_us": REGULAR}
    serve.serve(cfg(), wl.uniform_stream(30, HIGH, seed=99), eng)  # warm-up
    log("[sched] warm-up done")

    need_model = "lprs" in parts or "apc" in parts or "lprs_sweep" in parts
    # 1. samples
    X, Y, runs = [], [], []
    plan = [(b, HIGH, "uniform") for b in (256, 512, 1024, 2048)]
    plan += [(b, REGULAR, "uniform") for b in P["regular_budgets"]]
    plan += [(256, None, "short_long"), (1024, None, "short_long")]
    for i, (bmax, iv, kind) in enumerate(plan if need_model else []):
        reqs = (wl.uniform_stream(n_collect if iv == HIGH else P["n_collect_regular"], iv,
                                  seed=10 + i) if kind == "uniform"
                else wl.short_long_stream(n_collect, busy_interval_us=5 * P["apc_busy"],
                                          quiet_interval_us=5 * P["apc_quiet"], seed=10 + i))
        t0 = time.time()
        r = serve.serve(cfg(max_tokens=bmax), reqs, eng, record=True)
        X.append(r["_features"])
        Y.append(r["_step_us"])
        runs.append({"max_tokens": bmax, "interval_us": iv, "stream": kind, "rounds": r["rounds"]})
        log(f"[sched] samples {i + 1}/{len(plan)}: B={bmax} {kind} {iv}: {r['rounds']} rounds, "
            f"{time.time() - t0:.1f}s")
    if need_model:
        model = _train_predictor(out, out_dir, X, Y, runs, epochs)
    if "lprs" in parts:
        _lprs_runs(out, P, cfg, strip, eng, model)
    if "aging" in parts:
        _aging_runs(out, P, cfg, strip, eng)
    if "apc" in parts:
        _apc_runs(out, P, cfg, strip, eng, model)
    if "lprs_sweep" in parts:
        _lprs_sweep(out, P, cfg, strip, eng, model)
    with open(os.path.join(out_dir, "sched_results.json"), "w") as fh:
        json.dump(out, fh, indent=1)
    return out


def _vs_target(r, steps, t):
    import numpy as np
    r = dict(r)
    r["target_us"] = t
    r["frac_over_target"] = float((steps > t).mean())
    r["mean_abs_dev_from_target_us"] = float(np.abs(steps - t).mean())
    return r


def _train_predictor(out, out_dir, X, Y, runs, epochs):
    import numpy as np
    from paper_2606_09061_amd import lprs, sched
    X = np.concatenate(X)
    Y = np.concatenate(Y)
    np.savetxt(os.path.join(out_dir, "samples.csv"), np.column_stack([X, Y]), delimiter=",",
               header=",".join(list(sched.FEATURES) + ["step_us"]), comments="", fmt="%.6g")
    out["samples"] = {"n": int(len(Y)), "runs": runs}

    # 2. predictor
    keep = lprs.downsample(X, Y, cap=3000, seed=0)
    X, Y = X[keep], Y[keep]
    out["samples"]["kept_after_downsampling"] = int(len(Y))
    tr, va, te = lprs.split_811(len(Y), seed=0)
    t0 = time.time()
    model = lprs.LatencyPredictor().fit(
        X[tr], Y[tr], X[va], Y[va], epochs=epochs,
        progress=lambda ep, loss: log(f"[sched] predictor epoch {ep}: val loss {loss:.5f}"))
    out["predictor"] = {"train_s": time.time() - t0, "split": [len(tr), len(va), len(te)],
                        "test": lprs.accuracy(Y[te], model.predict(X[te]))}
    lin = [sched.FEATURES.index(f) for f in ("bias", "scheduled_tokens", "avg_decode_ctx",
                                               "decode_ctx_interaction", "prefill_interaction")]
    sc = np.abs(X[tr][:, lin]).max(axis=0)
    sc[sc == 0] = 1
    w, *_ = np.linalg.lstsq(X[tr][:, lin] / sc, Y[tr], rcond=None)
    out["predictor"]["table2_linear_test"] = lprs.accuracy(Y[te], (X[te][:, lin] / sc) @ w)
    log(f"[sched] predictor: {json.dumps(out['predictor']['test'])}")
    return model


def _lprs_runs(out, P, cfg, strip, eng, model):
    import numpy as np
    import workloads as wl
    from paper_2606_09061_amd import sched, serve
    n_req, HIGH, REGULAR = P["n_req"], P["high"], P["regular"]
    vs_target = _vs_target
    cmp = {}
    reqs = wl.uniform_stream(n_req, HIGH, seed=1000)
    tb = serve.serve(cfg(max_tokens=1024), reqs, eng, record=True)
    st = tb["_step_us"]
    all_targets = {"mean": float(np.mean(st)), "p75": float(np.percentile(st, 75)),
                   "p90": float(np.percentile(st, 90))}
    targets = {k: all_targets[k] for k in P["targets"]}
    out["targets_us"] = targets
    row = {"token_budget_1024": vs_target(strip(tb), st, targets["p90"])}
    r = serve.serve(cfg(max_tokens=1024, chunking=sched.CHUNK_LPRS, target_us=targets["p90"]),
                    reqs, eng, predictor=model)
    row["lprs_B1024_T_p90"] = strip(r)
    for tname, t in targets.items():
        for bmax in (1024, 2048):
            r = serve.serve(cfg(max_tokens=bmax, chunking=sched.CHUNK_LPRS, target_us=t, apc=True),
                            reqs, eng, predictor=model)
            row[f"lprs_apc_B{bmax}_T_{tname}"] = strip(r)
        log(f"[sched] LPRS at T*={tname} ({t:.1f} us) done")
    cmp["high"] = row
    reqs = wl.uniform_stream(P["n_regular"], REGULAR, seed=1001)
    tb = serve.serve(cfg(max_tokens=1024), reqs, eng, record=True)
    row = {"token_budget_1024": vs_target(strip(tb), tb["_step_us"], targets["p90"])}
    for bmax in (1024, 2048):
        r = serve.serve(cfg(max_tokens=bmax, chunking=sched.CHUNK_LPRS, target_us=targets["p90"],
                            apc=True), reqs, eng, predictor=model)
        row[f"lprs_apc_B{bmax}_T_p90"] = strip(r)
    cmp["regular"] = row
    log("[sched] LPRS vs token budget at regular load done")
    out["lprs_vs_token_budget"] = cmp


def _lprs_sweep(out, P, cfg, strip, eng, model):
    """Sensitivity of LPRS + APC at high load to the constants the paper
    leaves open: the overflow penalty lambda_o (lambda_u = 1) and the search
    granularity delta, at T* = the token budget's 90th-percentile round."""
    import numpy as np
    import workloads as wl
    from paper_2606_09061_amd import sched, serve
    reqs = wl.uniform_stream(P["n_req"], P["high"], seed=1000)
    tb = serve.serve(cfg(max_tokens=1024), reqs, eng, record=True)
    t = float(np.percentile(tb["_step_us"], 90))
    res = {"target_us": t, "token_budget_1024": _vs_target(strip(tb), tb["_step_us"], t)}
    for lo in (1.0, 2.0, 4.0, 8.0):
        for delta in (32, 128):
            for bmax in (1024, 2048):
                r = serve.serve(cfg(max_tokens=bmax, chunking=sched.CHUNK_LPRS, target_us=t,
                                    apc=True, lambda_o=lo, delta=delta), reqs, eng,
                                predictor=model)
                res[f"lo{lo:g}_d{delta}_B{bmax}"] = strip(r)
        log(f"[sched] LPRS sweep lambda_o={lo} done")
    out["lprs_sweep"] = res


def _aging_runs(out, P, cfg, strip, eng):
    import workloads as wl
    from paper_2606_09061_amd import sched, serve
    n_req = P["n_req"]
    aging = {}
    reqs = wl.uniform_stream(n_req, P["aging"], seed=2000, max_seq_len=1024, prompt_median=19,
                             output_median=64, sigma=1.75)
    for bmax in P["aging_budgets"]:
        row = {"fcfs": strip(serve.serve(cfg(max_tokens=bmax, policy=sched.POLICY_FCFS), reqs, eng))}
        for ratio in P["aging_ratios"]:
            row[f"aging_alpha_over_beta_{ratio}"] = strip(serve.serve(
                cfg(max_tokens=bmax, policy=sched.POLICY_AGING, alpha=ratio, beta=-1.0), reqs, eng))
        aging[f"B{bmax}"] = row
    out["aging_vs_fcfs"] = aging
    log("[sched] aging vs FCFS done")


def _apc_runs(out, P, cfg, strip, eng, model):
    import numpy as np
    import workloads as wl
    from paper_2606_09061_amd import sched, serve
    n_req = P["n_req"]
    vs_target = _vs_target
    reqs = wl.short_long_stream(n_req, busy_interval_us=P["apc_busy"],
                                quiet_interval_us=P["apc_quiet"], seed=3000)
    tb = serve.serve(cfg(max_tokens=1024), reqs, eng, record=True)
    t_apc = float(np.mean(tb["_step_us"]))
    apc = {"target_us": t_apc, "token_budget_1024": vs_target(strip(tb), tb["_step_us"], t_apc)}
    for on in (False, True):
        apc["on" if on else "off"] = strip(serve.serve(
            cfg(max_tokens=1024, chunking=sched.CHUNK_LPRS, target_us=t_apc, apc=on),
            reqs, eng, predictor=model))
    # a looser target (the token budget's 90th percentile round), where LPRS
    # proposes sizeable chunks and the activity cap rather than the minimum
    # chunk decides
    t_loose = float(np.percentile(tb["_step_us"], 90))
    loose = {"target_us": t_loose}
    for on in (False, True):
        loose["on" if on else "off"] = strip(serve.serve(
            cfg(max_tokens=1024, chunking=sched.CHUNK_LPRS, target_us=t_loose, apc=on),
            reqs, eng, predictor=model))
    apc["loose_target"] = loose
    out["apc_ablation"] = apc
    log("[sched] APC ablation done")


def model_bench(reps=5, max_seqs=128, only=None):
    """Whole-iteration latency of the synthetic Qwen3-8B stack (36 layers,
    hidden 4096, 32/8 heads, d 128, FFN 12288, vocab 151936) on typical
    batches, with the per-iteration host time of issuing it."""
    import math
    import numpy as np
    import torch
    from paper_2606_09061_amd import model as M

    torch.cuda.set_device(0)
    t0 = time.time()
    m = M.Model(M.QWEN3_8B, max_seqs=max_seqs, max_seq_len=4096, max_tokens=2048, fill_caches=True)
    torch.cuda.synchronize()
    log(f"[model] built in {time.time() - t0:.1f}s, "
        f"{torch.cuda.memory_allocated() / 2**30:.1f} GiB allocated")
    rng = np.random.default_rng(0)
    ctx = np.clip(np.round(rng.lognormal(math.log(1024), 1.0, max_seqs)), 16, 4000).astype(int)
    dec = [(i, int(c) - 1, 1, int(c)) for i, c in enumerate(ctx)]
    cases = {
        "decode_128_ctx_med1024": dec,
        "decode_32_ctx_med1024": dec[:32],
        "prefill_1x1024_at_0": [(0, 0, 1024, 1024)],
        "prefill_1x1024_at_2048": [(0, 2048, 1024, 3072)],
        "prefill_2x1024_at_0": [(0, 0, 1024, 1024), (1, 0, 1024, 1024)],
        "mixed_64dec_plus_960_at_2048": dec[:64] + [(100, 2048, 960, 3008)],
        "mixed_127dec_plus_896_at_0": dec[1:] + [(0, 0, 896, 896)],
    }
    eng = M.ModelEngine(m)
    out = {"model": "qwen3-8b-synthetic", "layers": m.cfg.layers, "cases": {}}
    n_params = sum(t.numel() for L in m.layers for t in L.values()) + m.lm_head.numel()
    for name, rows in cases.items():
        if only and name not in only:
            continue
        rows = np.array(rows, np.int32)
        T = int(rows[:, 2].sum())
        for _ in range(2):
            eng.step(rows)
        gpu, host = [], []
        for _ in range(reps):
            torch.cuda.synchronize()
            h0 = time.perf_counter()
            eng.ev[0].record(eng.stream)
            m.forward(rows, eng.stream)
            eng.ev[1].record(eng.stream)
            h1 = time.perf_counter()
            eng.ev[1].synchronize()
            gpu.append(eng.ev[0].elapsed_time(eng.ev[1]))
            host.append((h1 - h0) * 1e3)
        ms = float(np.median(gpu))
        flops = 2.0 * n_params * T  # weight GEMMs only (attention excluded)
        out["cases"][name] = {"tokens": T, "rows": int(len(rows)), "gpu_ms": ms,
                              "host_issue_ms": float(np.median(host)),
                              "tokens_per_s": T / ms * 1e3,
                              "gemm_tflops": flops / (ms * 1e-3) / 1e12}
        log(f"[model] {name}: {ms:.2f} ms GPU, {np.median(host):.2f} ms host, T={T}")
    return out


def per_iteration(cfg, reps=7, settle_s=1.0):
    """Prefill and decode kernel time of every batch of mix ``cfg`` (the 20
    iterations of the replay for mix 5), measured one batch at a time with the
    library's per-kernel events after the batches have run once in order,
    with each batch's algorithmic work and the fractions of the peaks.  When
    a batch's decode rows run inside its prefill launch, "prefill_us" is that
    launch and "decode_us" is 0."""
    import numpy as np
    import torch
    import paper_2606_09061_amd as cp
    from paper_2606_09061_amd import binding

    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    batches, steps, shared, _ = build_inputs(cfg, dev)
    descs = [cp.desc_for(b) for b in batches]
    tables = [torch.from_numpy(b.block_tables).to(dev) for b in batches]
    ws = torch.empty(max(cp.workspace_bytes(d, b.rows) for d, b in zip(descs, batches)),
                     dtype=torch.uint8, device=dev)
    outs = [torch.empty(b.num_tokens, b.num_q_heads, b.head_dim, dtype=torch.bfloat16,
                        device=dev) for b in batches]
    s = torch.cuda.current_stream()

    def step(j):
        b, d, t = batches[j], descs[j], steps[j]
        cp.kv_append(d, t["k_new"], t["v_new"], shared["k_cache"], shared["v_cache"], tables[j],
                     b.rows, ws, stream=s)
        cp.attn_mixed(d, t["q"], shared["k_cache"], shared["v_cache"], tables[j], b.rows,
                      outs[j], ws, stream=s)

    for j in range(len(batches)):       # every batch once, in order (fills the replay's pools)
        step(j)
    torch.cuda.synchronize()
    t0 = time.perf_counter()            # clock settling, as in run_config
    while time.perf_counter() - t0 < settle_s:
        for j in range(len(batches)):
            step(j)
    torch.cuda.synchronize()
    times = [{"prefill": [], "decode": []} for _ in batches]
    for rep in range(reps):
        for j in range(len(batches)):
            binding.profile_begin()
            step(j)
            torch.cuda.synchronize()
            prof = binding.profile_end()
            for k in ("prefill", "decode"):
                times[j][k].append(prof[k][0] * 1e3)
        log(f"[per-iteration] rep {rep + 1}/{reps}")
    out = []
    for j, b in enumerate(batches):
        w = work_of(b)
        pf = b.rows[b.rows[:, 2] >= 2]
        t_pf = float(np.median(times[j]["prefill"][1:]))
        t_dc = float(np.median(times[j]["decode"][1:]))
        t_attn = t_pf + t_dc
        # roofline time of the attention launches: flops at the MFMA peak or
        # bytes at the HBM peak, whichever is longer
        t_roof = max(w["prefill_flops"] / (PEAK_BF16_TFLOPS * 1e12),
                     (w["prefill_bytes"] + w["decode_bytes"]) / (PEAK_HBM_GBS * 1e9))
        out.append({"iteration": j, "prefill_chunks": int(len(pf)),
                    "prefill_tokens": int(pf[:, 2].sum()),
                    "max_prior": int(pf[:, 1].max()) if len(pf) else 0,
                    "decode_rows": int((b.rows[:, 2] == 1).sum()),
                    "decode_fused": bool(w["fused_decode_bytes"]),
                    "prefill_gflop": w["prefill_flops"] / 1e9, "prefill_us": t_pf,
                    "prefill_frac_mfma": (w["prefill_flops"] / (t_pf * 1e-6) / (PEAK_BF16_TFLOPS * 1e12)
                                          if t_pf > 0 else None),
                    "decode_mb": w["decode_bytes"] / 1e6, "decode_us": t_dc,
                    "decode_frac_hbm": (w["decode_bytes"] / (t_dc * 1e-6) / (PEAK_HBM_GBS * 1e9)
                                        if t_dc > 0 else None),
                    "attention_us": t_attn,
                    "roofline_frac": t_roof / (t_attn * 1e-6) if t_attn > 0 else None})
    return {"mix": cfg, "reps": reps, "iterations": out}


FEW_TOKEN_LENS = (2, 3, 4, 8, 16)
FEW_TOKEN_PRIORS = (0, 1024, 4096)


GEMM_SHAPES = {"qkv": (6144, 4096), "o": (4096, 4096), "gate_up": (24576, 4096),
               "down": (4096, 12288)}
GEMM_ROWS = (33, 64, 128, 256, 512, 1024, 2048, 4096)


def gemm_table(reps=20):
    """The layer's projections (Qwen3-8B: hidden 4096, 32/8 heads, FFN 12288)
    on the package's tiled MFMA kernel (cpl_gemm) and on the platform BLAS
    (torch.mm -> hipBLASLt), per batch size: mean time per call over `reps`
    calls after warm-up (HIP events), and TFLOP/s.  Inputs N(0,1) bf16,
    weights N(0, 0.02)."""
    import torch
    from paper_2606_09061_amd import model as MM

    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    g = torch.Generator(device=dev).manual_seed(7)
    out = []
    only = os.environ.get("GEMM_PROJ")
    for name, (N, K) in GEMM_SHAPES.items():
        if only and name not in only.split(","):
            continue
        w = (torch.randn(N, K, generator=g, device=dev) * 0.02).to(torch.bfloat16)
        for M in GEMM_ROWS:
            a = torch.randn(M, K, generator=g, device=dev).to(torch.bfloat16)
            c1 = torch.empty(M, N, dtype=torch.bfloat16, device=dev)
            c2 = torch.empty_like(c1)
            ws = torch.empty(max(16, MM.gemm_workspace_bytes(M, N, K)), dtype=torch.uint8,
                             device=dev)
            row = {"proj": name, "M": M, "N": N, "K": K}
            for lab, fn in (("own", lambda: MM.gemm(a, w, c1, ws=ws)),
                            ("blas", lambda: torch.mm(a, w.t(), out=c2))):
                for _ in range(3):
                    fn()
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                torch.cuda.synchronize()
                e0.record()
                for _ in range(reps):
                    fn()
                e1.record()
                torch.cuda.synchronize()
                us = e0.elapsed_time(e1) * 1e3 / reps
                row[f"{lab}_us"] = us
                row[f"{lab}_tflops"] = 2.0 * M * N * K / (us * 1e-6) / 1e12
            d = (c1.float() - c2.float()).abs().max().item()
            row["max_abs_diff"] = d
            log(f"[gemm] {name} M={M}: own {row['own_us']:.1f} us, blas {row['blas_us']:.1f} us")
            out.append(row)
    return {"peak_tflops": PEAK_BF16_TFLOPS, "rows": out}


def few_token_routing(n_chunks=64, reps=20):
    """Attention time of batches of n_chunks c-token chunks (one per request,
    prior context P), routed either to the MFMA tile kernel or to the decode
    kernel one query token at a time (CP_PREFILL_MIN_LEN), at the Llama-3-8B
    (32/8 heads, block 16) and 70B (64/8 heads, block 32) shapes, head_dim 128.
    The two routings compute the same outputs; the faster one for each
    (shape, c, P) is what the planner's threshold should pick."""
    import numpy as np
    import torch
    import paper_2606_09061_amd as cp
    from paper_2606_09061_amd import binding
    import workloads as wl

    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    out = []
    # one untimed pass over both routings first (first launches load kernels)
    for hq, hkv, bsz in ((32, 8, 16), (64, 8, 32)):
        b = wl.make_batch("warm", hq, hkv, 128, bsz, [(64, 4)] * 8, np.random.default_rng(0))
        t = wl.make_tensors(b, seed=1, device=dev)
        d = cp.desc_for(b)
        ws = torch.empty(1 << 22, dtype=torch.uint8, device=dev)
        o = torch.empty(b.num_tokens, hq, 128, dtype=torch.bfloat16, device=dev)
        for min_len in ("2", "5"):
            os.environ["CP_PREFILL_MIN_LEN"] = min_len
            cp.attn_mixed(d, t["q"], t["k_cache"], t["v_cache"], t["block_tables"], b.rows, o, ws)
        os.environ.pop("CP_PREFILL_MIN_LEN", None)
    torch.cuda.synchronize()
    for hq, hkv, bsz in ((32, 8, 16), (64, 8, 32)):
        for P in FEW_TOKEN_PRIORS:
            for c in FEW_TOKEN_LENS:
                rng = np.random.default_rng([hq, P, c])
                b = wl.make_batch("few", hq, hkv, 128, bsz, [(P, c)] * n_chunks, rng)
                t = wl.make_tensors(b, seed=9000 + c, device=dev)
                d = cp.desc_for(b)
                need = cp.workspace_bytes(d, b.rows)
                os.environ["CP_PREFILL_MIN_LEN"] = str(c + 1)
                try:
                    need = max(need, cp.workspace_bytes(d, b.rows))
                finally:
                    os.environ.pop("CP_PREFILL_MIN_LEN", None)
                ws = torch.empty(need, dtype=torch.uint8, device=dev)
                o = torch.empty(b.num_tokens, hq, 128, dtype=torch.bfloat16, device=dev)
                cp.kv_append(d, t["k_new"], t["v_new"], t["k_cache"], t["v_cache"],
                             t["block_tables"], b.rows, ws)
                row = {"heads": [hq, hkv], "block": bsz, "prior": P, "chunk": c,
                       "chunks": n_chunks}
                for route, min_len in (("tile", "2"), ("decode", str(c + 1))):
                    os.environ["CP_PREFILL_MIN_LEN"] = min_len
                    try:
                        for _ in range(3):
                            cp.attn_mixed(d, t["q"], t["k_cache"], t["v_cache"], t["block_tables"],
                                          b.rows, o, ws)
                        torch.cuda.synchronize()
                        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
                        ev[0].record()
                        for _ in range(reps):
                            cp.attn_mixed(d, t["q"], t["k_cache"], t["v_cache"], t["block_tables"],
                                          b.rows, o, ws)
                        ev[1].record()
                        ev[1].synchronize()
                        row[route + "_us"] = ev[0].elapsed_time(ev[1]) * 1e3 / reps
                    finally:
                        os.environ.pop("CP_PREFILL_MIN_LEN", None)
                row["faster"] = "decode" if row["decode_us"] < row["tile_us"] else "tile"
                out.append(row)
                log(f"[few-token] {row}")
                del t, ws, o
    return {"few_token_routing": out}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=60)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", type=int, default=5, choices=[1, 2, 3, 4, 5])
    ap.add_argument("--all", action="store_true", help="one JSON line per mix")
    ap.add_argument("--no-cpu", action="store_true", help="skip the oracle CPU baseline")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--shard", type=int, default=1, choices=[1, 2, 4, 8],
                    help="run one GPU's share of a head-sharded (tensor-parallel) group of "
                         "this many GPUs: Hq / N and Hkv / N heads, same rows")
    ap.add_argument("--settle", type=float, default=1.0, metavar="SECONDS",
                    help="run the steps back to back this long before the warm-up, so the "
                         "timed region starts at the clock the GPU holds under load (0: off)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run plain copies of MIB MiB (counter calibration)")
    ap.add_argument("--sub", choices=["prefill", "decode"], default=None,
                    help="time only the prefill rows or only the decode rows of the mix")
    ap.add_argument("--cold", type=int, default=0, metavar="N",
                    help="also time N steps with the MALL and L2 flushed before each")
    ap.add_argument("--peaks", action="store_true",
                    help="only measure library GEMM / copy / read rates")
    ap.add_argument("--latency-table", default=None, metavar="CSV",
                    help="only run the latency-vs-composition sweep, written to CSV")
    ap.add_argument("--sched", default=None, metavar="DIR",
                    help="only run the closed-loop scheduling experiment, results under DIR")
    ap.add_argument("--sched-engine", choices=["step", "model"], default="step",
                    help="with --sched: the attention step alone or the whole 36-layer model")
    ap.add_argument("--sched-parts", default="lprs,aging,apc",
                    help="with --sched: comma-separated subset of lprs, aging, apc, lprs_sweep")
    ap.add_argument("--model", action="store_true",
                    help="only time whole iterations of the synthetic Qwen3-8B stack")
    ap.add_argument("--model-case", action="append", default=None,
                    help="with --model: time only this batch (repeatable)")
    ap.add_argument("--per-iteration", action="store_true",
                    help="prefill / decode kernel time of every batch of --config (mix 5: its "
                         "20 iterations) against its algorithmic work")
    ap.add_argument("--gemm", action="store_true",
                    help="the layer's projections on cpl_gemm and on the platform BLAS")
    ap.add_argument("--few-token", action="store_true",
                    help="only time few-token chunks on the tile kernel against the decode "
                         "kernel token by token")
    ap.add_argument("--fit", default=None, metavar="CSV",
                    help="only fit a latency table written earlier (no GPU)")
    args = ap.parse_args()
    if args.copy_calibration:
        copy_calibration(args.copy_calibration, args.steps)
        return
    if args.peaks:
        print(json.dumps(measured_peaks()), flush=True)
        return
    if args.latency_table:
        print(json.dumps(latency_table(args.latency_table)), flush=True)
        return
    if args.fit:
        print(json.dumps(fit_latency(args.fit)), flush=True)
        return
    if args.sched:
        print(json.dumps(sched_experiment(args.sched, engine=args.sched_engine,
                                          parts=tuple(args.sched_parts.split(",")))), flush=True)
        return
    if args.few_token:
        print(json.dumps(few_token_routing()), flush=True)
        return
    if args.gemm:
        print(json.dumps(gemm_table()), flush=True)
        return
    if args.per_iteration:
        print(json.dumps(per_iteration(args.config, settle_s=args.settle)), flush=True)
        return
    if args.model:
        print(json.dumps(model_bench(only=args.model_case)), flush=True)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for {args.gpus}): the attention step is "
              "measured on a single MI355X; a multi-GPU run would shard heads across GPUs with "
              "no collective inside the step and is not implemented here.", file=sys.stderr)
        sys.exit(2)
    cfgs = [1, 2, 3, 4, 5] if args.all else [args.config]
    for c in cfgs:
        res = run_config(c, args.steps, args.warmup, with_cpu=not args.no_cpu,
                         cpu_budget=args.cpu_seconds, sub=args.sub, cold=args.cold,
                         settle_s=args.settle, shard=args.shard)
        print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
