"""Seeded synthetic request streams for closed-loop serving runs.

Requests are (id, arrival_us, prompt_len, max_new_tokens) tuples; nothing
here schedules or computes.  The paper's online workloads are replays of
real traces that are not available here, so their shape is drawn instead:
  * ``uniform_stream``: requests arriving at a fixed interval (the LPRS
    workloads of Sec. 4.4: 1,000 requests at a fixed inter-arrival time,
    sequences capped at 4,096 tokens), with log-normal prompt and output
    lengths;
  * ``short_long_stream``: the APC ablation mix of Sec. 4.1, 49 short prompts
    (30–50 tokens) per long one (200–220 tokens), with arrivals whose rate
    changes over time (exponential gaps whose mean switches between a busy
    and a quiet level every 100 requests).
"""

from __future__ import annotations

import math

import numpy as np


def _lognormal_int(rng, median, n, lo, hi, sigma=1.0):
    x = rng.lognormal(mean=math.log(median), sigma=sigma, size=n)
    return np.clip(np.round(x), lo, hi).astype(np.int64)


def uniform_stream(n=1000, interval_us=1000.0, seed=0, max_seq_len=4096, prompt_median=512,
                   output_median=128, sigma=1.0):
    rng = np.random.default_rng(seed)
    prompts = _lognormal_int(rng, prompt_median, n, 16, max_seq_len - 64, sigma)
    outs = _lognormal_int(rng, output_median, n, 1, max_seq_len, sigma)
    outs = np.minimum(outs, max_seq_len - prompts)
    return [(i, float(i * interval_us), int(p), int(o)) for i, (p, o) in
            enumerate(zip(prompts, outs))]


def short_long_stream(n=1000, busy_interval_us=100.0, quiet_interval_us=1000.0, seed=0,
                      ratio=49, short=(30, 50), long=(200, 220), output_median=64,
                      max_seq_len=4096):
    rng = np.random.default_rng(seed)
    is_long = np.zeros(n, dtype=bool)
    is_long[rng.permutation(n)[: max(1, n // (ratio + 1))]] = True
    prompts = np.where(is_long, rng.integers(long[0], long[1] + 1, n),
                       rng.integers(short[0], short[1] + 1, n))
    outs = np.minimum(_lognormal_int(rng, output_median, n, 1, max_seq_len), max_seq_len - prompts)
    t, reqs = 0.0, []
    for i in range(n):
        mean = busy_interval_us if (i // 100) % 2 == 0 else quiet_interval_us
        t += float(rng.exponential(mean))
        reqs.append((i, t, int(prompts[i]), int(outs[i])))
    return reqs
