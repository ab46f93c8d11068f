"""Plain reference of the scheduling layer: Aging (Sec. 3.1), LPRS
(Sec. 3.2, Algorithm 1) and APC (Sec. 3.3), in straightforward Python.

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, never by the product.  It
shares no code with the C++ scheduler (libcpsched.so); each function follows
the paper's definitions in the paper's order, with no heap, batching or
incremental state:
  * priorities are recomputed from Eq. 1 for every waiting request in every
    round and the queue is fully sorted (the naive form Sec. 3.1.4 replaces
    by a heap on Eq. 4);
  * Algorithm 1 evaluates the predictor once per candidate, in ascending c;
  * the APC rule is Eq. 12–14 written out.

Readings where the paper is silent (the same ones the product takes):
  * a row of one token is a decode row for the features, a longer row a
    prefill chunk; prefill_processed_tokens sums the chunks' start positions
    (the prompt tokens already in the cache);
  * |P_t| of Eq. 12–14 counts the prefill chunks already admitted to the
    round; |D_t| the decode rows admitted to the round;
  * equal priorities go to the earlier arrival, then to the earlier
    registered request; a request without a slot is passed over while every
    slot is taken; new requests take the lowest free slot;
  * Algorithm 1 scores that are NaN never win (both comparisons are false);
  * with APC on, the scan of a round's queue stops once |P_t| >= C_t with
    |P_t| > 0: Eq. 14 then gives 0 to every remaining candidate (C_t only
    shrinks as the round fills), so they are not scored.
"""

from __future__ import annotations

import math

import numpy as np


# ---- Table 1 and Table 2 ----------------------------------------------------

def features(rows, mem=(0.0, 0.0, 0.0, 0.0)):
    """The 16 predictor inputs of one batch, rows = [(req, start, len, ctx), ...]:
    Table 1's 11 raw statistics then Table 2's 5 derived features."""
    prefill_tokens = 0
    decode_tokens = 0
    batch_request_count = 0
    sum_decode_context_len = 0
    max_decode_context_len = 0
    prefill_processed_tokens = 0
    max_prefill_processed_tokens = 0
    for _req, start, length, ctx in rows:
        if length > 0:
            batch_request_count += 1
        if length == 1:
            decode_tokens += 1
            sum_decode_context_len += ctx
            max_decode_context_len = max(max_decode_context_len, ctx)
        elif length >= 2:
            prefill_tokens += length
            prefill_processed_tokens += start
            max_prefill_processed_tokens = max(max_prefill_processed_tokens, start)
    gpu_mem_used, gpu_mem_free, cuda_allocated, cuda_reserved = mem
    bias = 1
    scheduled_tokens = decode_tokens + prefill_tokens
    avg_decode_ctx = sum_decode_context_len / max(decode_tokens, 1)
    decode_ctx_interaction = decode_tokens * avg_decode_ctx
    prefill_interaction = prefill_tokens * prefill_processed_tokens
    return [float(v) for v in (
        prefill_tokens, decode_tokens, batch_request_count, sum_decode_context_len,
        max_decode_context_len, prefill_processed_tokens, max_prefill_processed_tokens,
        gpu_mem_used, gpu_mem_free, cuda_allocated, cuda_reserved,
        bias, scheduled_tokens, avg_decode_ctx, decode_ctx_interaction, prefill_interaction)]


# ---- the predictor f_theta (Sec. 3.2.1) ---------------------------------------

def mlp_predict(layers, x_mean, x_std, y_scale, x):
    """One feature vector through the MLP: standardise, affine layers with
    ReLU between them, scale the single output.  layers = [(W, b), ...]."""
    h = (np.asarray(x, np.float64) - np.asarray(x_mean, np.float64)) / np.asarray(x_std, np.float64)
    for i, (W, b) in enumerate(layers):
        h = np.asarray(W, np.float64) @ h + np.asarray(b, np.float64)
        if i + 1 < len(layers):
            h = np.maximum(h, 0.0)
    return float(h[0]) * y_scale


# ---- Algorithm 1 --------------------------------------------------------------

def candidate_set(h, delta):
    """Eq. 8: {1, h} together with every k*delta in [1, h]."""
    c = {1, h}
    k = 1
    while k * delta <= h:
        c.add(k * delta)
        k += 1
    return sorted(c)


def select_chunk(committed, slot, processed, remaining, max_tokens, delta, target, lambda_u,
                 lambda_o, predict, mem=(0.0, 0.0, 0.0, 0.0)):
    """Algorithm 1 for one candidate request; predict maps one feature vector
    to a latency.  Returns (c*, predicted latency of c* or nan)."""
    u = sum(r[2] for r in committed)
    h = min(remaining, max_tokens - u)                                  # Eq. 6
    if h <= 0:
        return 0, math.nan
    best_score = math.inf
    c_star = 0
    t_star_hat = math.nan
    for c in candidate_set(h, delta):                                   # Eq. 8
        x = features(list(committed) + [(slot, processed, c, processed + c)], mem)
        t_hat = predict(x)                                              # Eq. 9
        if t_hat <= target:                                             # Eq. 10
            score = lambda_u * (target - t_hat)
        else:
            score = lambda_o * (t_hat - target)
        if score < best_score:                                          # Eq. 11
            best_score, c_star, t_star_hat = score, c, t_hat
        elif score == best_score and c > c_star:
            c_star, t_star_hat = c, t_hat
    if c_star == 0 and u == 0 and h >= 1:                               # empty batch
        return 1, math.nan
    return c_star, t_star_hat


# ---- APC (Eq. 12–14) ------------------------------------------------------------

def apc(c_star, h, remaining, n_decode, n_active, committed, max_active, max_seqs, max_tokens,
        min_chunk):
    """Final chunk and reason ('accepted', 'warm_start', 'blocked_cap',
    'blocked_min_chunk')."""
    cap = min(max_active, max_seqs - n_decode, (max_tokens - committed) // min_chunk)  # Eq. 12
    m = min(remaining, min_chunk)                                                      # Eq. 13
    if n_active < cap and c_star >= m:                                                 # Eq. 14
        return c_star, "accepted"
    if c_star < m and n_active == 0:
        return min(h, m), "warm_start"
    return 0, ("blocked_cap" if c_star >= m else "blocked_min_chunk")


# ---- Aging (Eq. 1–2) ------------------------------------------------------------

def priority(alpha, beta, t, arrival, remaining):
    """Eq. 1."""
    return alpha * (t - arrival) + beta * remaining


class Scheduler:
    """Round-by-round reference scheduler with the semantics of cp_sched.h.

    cfg keys: policy ('fcfs' | 'aging'), alpha, beta, max_tokens, max_seqs,
    chunking ('budget' | 'lprs'), target, delta, lambda_u, lambda_o, apc
    (bool), max_active, min_chunk; predict is used under 'lprs'."""

    def __init__(self, cfg, predict=None, mem=(0.0, 0.0, 0.0, 0.0)):
        self.cfg = dict(cfg)
        self.predict = predict
        self.mem = mem
        self.reqs = []              # dicts, in registration order
        self.decoding = []          # request indices, in the order they started decoding
        self.free = set(range(cfg["max_seqs"]))
        self.last = None            # [(index, chunk_len)] of the batch awaiting completion
        self.counts = {"blocked_cap": 0, "blocked_min_chunk": 0, "warm_start": 0,
                       "skipped_no_slot": 0, "not_scored": 0}

    def add(self, rid, arrival, prompt_len, max_new):
        self.reqs.append({"id": rid, "arrival": arrival, "prompt": prompt_len,
                          "max_new": max_new, "processed": 0, "remaining": prompt_len,
                          "generated": 0, "slot": None, "first_token": None, "finish": None})

    def _queue(self, t):
        cfg = self.cfg
        waiting = [i for i, r in enumerate(self.reqs) if r["remaining"] > 0]
        if cfg["policy"] == "fcfs":
            return sorted(waiting, key=lambda i: (self.reqs[i]["arrival"], i))
        pri = {i: priority(cfg["alpha"], cfg["beta"], t, self.reqs[i]["arrival"],
                           self.reqs[i]["remaining"]) for i in waiting}
        return sorted(waiting, key=lambda i: (-pri[i], self.reqs[i]["arrival"], i))

    def schedule(self, t):
        """Rows [(slot, start, len, ctx)], request ids, number of decode rows."""
        cfg = self.cfg
        assert self.last is None
        rows, ids, batch = [], [], []
        u = 0
        for i in self.decoding:                                   # decode-first admission
            if u >= cfg["max_tokens"]:
                break
            r = self.reqs[i]
            pos = r["prompt"] + r["generated"] - 1
            rows.append((r["slot"], pos, 1, pos + 1))
            ids.append(r["id"])
            batch.append((i, 1))
            u += 1
        n_decode = len(rows)
        n_active = 0
        queue = self._queue(t)
        for pos_in_queue, i in enumerate(queue):
            if u >= cfg["max_tokens"] or len(rows) >= cfg["max_seqs"]:
                break
            if cfg["apc"] and n_active > 0:
                cap = min(cfg["max_active"], cfg["max_seqs"] - n_decode,
                          (cfg["max_tokens"] - u) // cfg["min_chunk"])
                if n_active >= cap:
                    # Eq. 14 gives 0 to every remaining candidate
                    self.counts["not_scored"] += len(queue) - pos_in_queue
                    break
            r = self.reqs[i]
            if r["slot"] is None and not self.free:
                self.counts["skipped_no_slot"] += 1
                continue
            h = min(r["remaining"], cfg["max_tokens"] - u)
            if cfg["chunking"] == "lprs":
                c, _ = select_chunk(rows, 0, r["processed"], r["remaining"], cfg["max_tokens"],
                                    cfg["delta"], cfg["target"], cfg["lambda_u"],
                                    cfg["lambda_o"], self.predict, self.mem)
            else:
                c = h                                             # Eq. 7
            if cfg["apc"]:
                c2, why = apc(c, h, r["remaining"], n_decode, n_active, u, cfg["max_active"],
                              cfg["max_seqs"], cfg["max_tokens"], cfg["min_chunk"])
                if why in ("blocked_cap", "blocked_min_chunk") or (why == "warm_start" and c2 != c):
                    self.counts[why] += 1
                c = c2
            if c <= 0:
                continue
            if r["slot"] is None:
                r["slot"] = min(self.free)
                self.free.remove(r["slot"])
            rows.append((r["slot"], r["processed"], c, r["processed"] + c))
            ids.append(r["id"])
            batch.append((i, c))
            r["remaining"] -= c                                   # Eq. 2
            u += c
            n_active += 1
        self.last = batch
        return rows, ids, n_decode

    def complete(self, t):
        for i, c in self.last:
            r = self.reqs[i]
            if r["processed"] < r["prompt"]:
                r["processed"] += c
                if r["processed"] < r["prompt"]:
                    continue
                r["first_token"] = t
                r["generated"] = 1
                if r["generated"] < r["max_new"]:
                    self.decoding.append(i)
                    continue
            else:
                r["generated"] += 1
                if r["generated"] < r["max_new"]:
                    continue
            r["finish"] = t
            self.free.add(r["slot"])
            if i in self.decoding:
                self.decoding.remove(i)
        self.last = None

    def pending(self):
        return sum(1 for r in self.reqs if r["finish"] is None)
