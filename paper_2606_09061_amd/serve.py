"""Closed-loop serving of the attention step: the C++ scheduler builds each
round's batch, the HIP library executes it on one GPU, and the measured step
latency advances the clock the scheduler sees (Sec. 3's iteration-level,
non-preemptive execution).

``StepEngine`` owns a paged KV pool with a fixed block-table row per
scheduler slot, and synthetic q / k / v rows; ``serve`` runs a request
stream to completion and returns the latency figures the paper reports
(step latency against the target, prefill and request end-to-end latency,
scheduling dynamics and APC interventions), plus the per-round predictor
features and measured latencies when asked to record them.
"""

from __future__ import annotations

import math
import time

import numpy as np

from . import binding as cp
from . import sched


def gpu_mem_mb():
    """The four GPU-memory features of Table 1, in MB: device memory in use
    and free, and the torch caching allocator's allocated and reserved bytes."""
    import torch
    free, total = torch.cuda.mem_get_info()
    mb = 1.0 / (1 << 20)
    return [(total - free) * mb, free * mb, torch.cuda.memory_allocated() * mb,
            torch.cuda.memory_reserved() * mb]


class StepEngine:
    """The attention step of one layer on one GPU, for scheduler-built batches.

    Slot s owns logical blocks [0, max_seq_len / B) mapped to a random,
    disjoint set of physical blocks.  Every round appends the batch's k/v rows
    and runs the mixed attention; the contents are synthetic (N(0,1) in bf16),
    which affects timing only through the hardware's data-dependent power."""

    def __init__(self, hq=32, hkv=8, d=128, bsz=16, max_seqs=256, max_seq_len=4096,
                 max_tokens=2048, seed=0, device=None):
        import torch
        from workloads.tensors import _randn_bf16

        self.dev = device or torch.device("cuda", 0)
        self.max_tokens = max_tokens
        mbr = -(-max_seq_len // bsz)
        nb = max_seqs * mbr
        rng = np.random.default_rng(seed)
        bt = rng.permutation(nb).astype(np.int32).reshape(max_seqs, mbr)
        self.bt = torch.from_numpy(bt).to(self.dev)
        gen = torch.Generator(device=self.dev)
        gen.manual_seed(seed)
        self.kc = _randn_bf16((nb, hkv, bsz, d), gen, self.dev)
        self.vc = _randn_bf16((nb, hkv, d, bsz), gen, self.dev)
        self.q = _randn_bf16((max_tokens, hq, d), gen, self.dev)
        self.kn = _randn_bf16((max_tokens, hkv, d), gen, self.dev)
        self.vn = _randn_bf16((max_tokens, hkv, d), gen, self.dev)
        self.out = torch.empty(max_tokens, hq, d, dtype=torch.bfloat16, device=self.dev)
        self.ws = torch.empty(64 << 20, dtype=torch.uint8, device=self.dev)
        self.desc = cp.make_desc(hq, hkv, d, bsz, nb, mbr, max_seqs, 1.0 / math.sqrt(d))
        self.stream = torch.cuda.current_stream(self.dev)
        self.ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]

    def _grow_on_demand(self, call, rows):
        import torch
        try:
            call()
        except cp.CpError as e:
            if e.code != cp.CP_ERR_WORKSPACE:
                raise
            self.ws = torch.empty(cp.workspace_bytes(self.desc, rows), dtype=torch.uint8,
                                  device=self.dev)
            call()

    def step(self, rows) -> float:
        """Runs one batch; returns the GPU time of append + attention in us."""
        import torch
        rows = np.asarray(rows, dtype=np.int32).reshape(-1, 4)
        T = int(rows[:, 2].sum())
        if T == 0:
            return 0.0
        if T > self.max_tokens:
            raise ValueError(f"batch of {T} tokens exceeds the engine's {self.max_tokens}")
        s = self.stream
        self.ev[0].record(s)
        # Each call plans the batch once.  A workspace too small is reported
        # before anything is enqueued; only then is the size asked for (a
        # second planning) and the call repeated.
        self._grow_on_demand(lambda: cp.kv_append(self.desc, self.kn[:T], self.vn[:T], self.kc,
                                                  self.vc, self.bt, rows, self.ws, stream=s), rows)
        self._grow_on_demand(lambda: cp.attn_mixed(self.desc, self.q[:T], self.kc, self.vc,
                                                   self.bt, rows, self.out[:T], self.ws, stream=s),
                             rows)
        self.ev[1].record(s)
        self.ev[1].synchronize()
        return self.ev[0].elapsed_time(self.ev[1]) * 1e3


def _pct(x, ps=(50, 90, 95, 99)):
    x = np.asarray(x, dtype=np.float64)
    if x.size == 0:
        return {f"p{p}": None for p in ps}
    return {f"p{p}": float(np.percentile(x, p)) for p in ps}


def _summary(x):
    x = np.asarray(x, dtype=np.float64)
    d = {"mean": float(x.mean()) if x.size else None}
    d.update(_pct(x))
    d["max"] = float(x.max()) if x.size else None
    return d


def serve(cfg: sched.Config, requests, engine: StepEngine, predictor=None, record=False,
          memory_features=True, max_rounds=1_000_000):
    """Runs ``requests`` [(id, arrival_us, prompt_len, max_new_tokens)] to
    completion.  The clock starts at 0 and advances by each round's measured
    step latency; when nothing is runnable it jumps to the next arrival."""
    s = sched.Scheduler(cfg)
    if predictor is not None:
        predictor.load_into(s)
    todo = sorted(requests, key=lambda r: (r[1], r[0]))
    k, now = 0, 0.0
    step_us, sched_us, n_dec, n_pf, pf_tok, pred = [], [], [], [], [], []
    feats = []
    rounds = 0
    mem = [0.0, 0.0, 0.0, 0.0]
    while k < len(todo) or s.pending():
        while k < len(todo) and todo[k][1] <= now:
            s.add_request(*todo[k])
            k += 1
        if s.pending() == 0:
            now = todo[k][1]
            continue
        if memory_features:
            mem = gpu_mem_mb()
            s.set_memory_state(mem)
        h0 = time.perf_counter()
        r = s.schedule(now)
        sched_us.append((time.perf_counter() - h0) * 1e6)
        rounds += 1
        if rounds > max_rounds:
            raise RuntimeError("serving loop exceeded its round limit")
        if len(r.rows) == 0:
            s.complete(now)
            if k < len(todo):
                now = max(now, todo[k][1])
                continue
            raise RuntimeError("scheduler returned an empty round with work pending")
        x = sched.batch_features(r.rows, mem)
        if predictor is not None:
            pred.append(float(s.predict(x[None])[0]))
        us = engine.step(r.rows)
        now += us
        s.complete(now)
        step_us.append(us)
        n_dec.append(r.n_decode)
        n_pf.append(len(r.rows) - r.n_decode)
        pf_tok.append(int(r.rows[r.n_decode:, 2].sum()))
        if record:
            feats.append(x)
    ttft, e2e, tok = [], [], 0
    for rid, arr, p, o in requests:
        info = s.request(rid)
        ttft.append(info["first_token"] - arr)
        e2e.append(info["finish"] - arr)
        tok += p + o
    st = s.stats()
    step = np.asarray(step_us)
    res = {
        "requests": len(requests), "rounds": len(step_us), "makespan_ms": now / 1e3,
        "tokens_per_s": tok / (now * 1e-6) if now > 0 else None,
        "step_us": _summary(step),
        "prefill_e2e_ms": _summary(np.asarray(ttft) / 1e3),
        "request_e2e_ms": _summary(np.asarray(e2e) / 1e3),
        "avg_decode_rows": float(np.mean(n_dec)),
        "avg_prefill_seqs": float(np.mean(n_pf)),
        "avg_prefill_chunk": float(np.sum(pf_tok) / max(1, np.sum(n_pf))),
        "avg_prefill_tokens_per_round": float(np.mean(pf_tok)),
        "sched_host_us": _summary(sched_us),
        "apc_blocked_cap": st["apc_blocked_cap"], "apc_blocked_min_chunk": st["apc_blocked_min"],
        "apc_warm_starts": st["apc_warm_starts"], "lprs_calls": st["lprs_calls"],
        "predictor_rows": st["predictor_rows"],
    }
    if cfg.chunking == sched.CHUNK_LPRS or cfg.target_us > 0:
        t = cfg.target_us
        res["target_us"] = t
        res["frac_over_target"] = float((step > t).mean())
        res["mean_abs_dev_from_target_us"] = float(np.abs(step - t).mean())
    if pred:
        e = np.asarray(pred) - step
        res["online_prediction"] = {"mae_us": float(np.abs(e).mean()),
                                    "mape_pct": float(100 * np.abs(e / step).mean()),
                                    "underestimated": float((e < 0).mean())}
    if record:
        res["_features"] = np.asarray(feats)
        res["_step_us"] = step
    return res
