"""Pins of the scheduling reference (oracle/sched.py) against what the paper
and arithmetic fix: hand-worked feature vectors (Tables 1–2), the candidate
sets of Eq. 8, closed forms of Algorithm 1 under linear and degenerate
predictors, Eq. 12–14 case by case, the limiting orders of the aging
priority (Sec. 3.1.3), and conservation invariants of whole schedules."""

import math

import numpy as np
import pytest

from oracle import sched as ref


def test_features_hand_worked():
    # decode row: 199 cached tokens + 1 new (ctx 200); a 48-token chunk after
    # 128 cached; a first chunk of 64 tokens; an idle row of length 0.
    rows = [(0, 199, 1, 200), (1, 128, 48, 176), (2, 0, 64, 64), (3, 5, 0, 5)]
    f = ref.features(rows, (10.0, 20.0, 30.0, 40.0))
    expect = {
        "prefill_tokens": 112, "decode_tokens": 1, "batch_request_count": 3,
        "sum_decode_context_len": 200, "max_decode_context_len": 200,
        "prefill_processed_tokens": 128, "max_prefill_processed_tokens": 128,
        "gpu_mem_used_mb": 10, "gpu_mem_free_mb": 20, "cuda_allocated_mb": 30,
        "cuda_reserved_mb": 40, "bias": 1, "scheduled_tokens": 113, "avg_decode_ctx": 200,
        "decode_ctx_interaction": 200, "prefill_interaction": 112 * 128,
    }
    assert f == [float(v) for v in expect.values()]


def test_features_two_decodes_average():
    f = ref.features([(0, 99, 1, 100), (1, 299, 1, 300)])
    assert f[1] == 2 and f[3] == 400 and f[4] == 300 and f[13] == 200 and f[14] == 400
    assert f[0] == 0 and f[15] == 0 and f[12] == 2


def test_features_empty_batch():
    f = ref.features([])
    assert f[11] == 1 and sum(f) == 1  # only the bias


@pytest.mark.parametrize("h,delta,expect", [
    (100, 32, [1, 32, 64, 96, 100]), (64, 32, [1, 32, 64]), (1, 32, [1]), (31, 32, [1, 31]),
    (4, 1, [1, 2, 3, 4]), (7, 3, [1, 3, 6, 7]), (2, 2, [1, 2]),
])
def test_candidate_set_eq8(h, delta, expect):
    assert ref.candidate_set(h, delta) == expect


def _linear(a, b):
    """T_hat = a + b * scheduled_tokens."""
    return lambda x: a + b * x[12]


def _select(pred, h, target, delta=1, lam=(1.0, 4.0), committed=(), remaining=None):
    return ref.select_chunk(list(committed), 0, 0, h if remaining is None else remaining,
                            max_tokens=h + sum(r[2] for r in committed), delta=delta,
                            target=target, lambda_u=lam[0], lambda_o=lam[1], predict=pred)


@pytest.mark.parametrize("a,b,target,lu,lo", [
    (10.0, 0.5, 40.25, 1.0, 4.0), (10.0, 0.5, 40.0, 1.0, 4.0), (3.0, 0.25, 17.1, 1.0, 1.0),
    (5.0, 2.0, 70.9, 1.0, 9.0), (5.0, 2.0, 70.1, 2.0, 3.0),
])
def test_algorithm1_linear_closed_form(a, b, target, lu, lo):
    # Exhaustive candidates (delta = 1): the optimum sits at one of the two
    # integers around c_lin = (T* - a) / b, chosen by comparing the underfill
    # penalty of the lower one with the overflow penalty of the upper one.
    h = 200
    c_lin = (target - a) / b
    lo_c, hi_c = math.floor(c_lin), math.floor(c_lin) + 1
    s_lo = lu * (target - (a + b * lo_c))
    s_hi = lo * ((a + b * hi_c) - target)
    if abs(c_lin - round(c_lin)) < 1e-12:
        expect = round(c_lin)  # exact hit: score 0
    else:
        expect = hi_c if s_hi <= s_lo else lo_c
    c, t = _select(_linear(a, b), h, target, lam=(lu, lo))
    assert c == expect
    assert t == a + b * c


def test_algorithm1_reduces_to_token_budget_when_target_is_loose():
    # T* above the predicted latency of every candidate and T_hat increasing:
    # the largest candidate h wins, which is the static rule c = h (Eq. 7).
    for h in (1, 5, 33, 64, 100, 1000):
        c, _ = _select(_linear(1.0, 0.01), h, target=1e9, delta=32)
        assert c == h


def test_algorithm1_tight_target_picks_one():
    c, _ = _select(_linear(50.0, 1.0), 500, target=10.0, delta=32)
    assert c == 1


def test_algorithm1_ties_go_to_the_larger_chunk():
    c, t = _select(lambda x: 7.0, 130, target=3.0, delta=32)
    assert c == 130 and t == 7.0


def test_algorithm1_skips_without_room():
    assert ref.select_chunk([], 0, 0, 10, 0, 32, 1.0, 1.0, 4.0, _linear(0, 1))[0] == 0
    assert ref.select_chunk([], 0, 0, 0, 100, 32, 1.0, 1.0, 4.0, _linear(0, 1))[0] == 0
    full = [(0, 9, 1, 10)] * 5
    assert ref.select_chunk(full, 1, 0, 10, 5, 32, 1.0, 1.0, 4.0, _linear(0, 1))[0] == 0


def test_algorithm1_starvation_guard():
    nan = lambda x: math.nan  # noqa: E731
    # Empty batch: nothing scores, the guard returns one token.
    assert ref.select_chunk([], 0, 0, 50, 100, 32, 1.0, 1.0, 4.0, nan)[0] == 1
    # Non-empty batch: the guard does not apply.
    assert ref.select_chunk([(0, 9, 1, 10)], 1, 0, 50, 100, 32, 1.0, 1.0, 4.0, nan)[0] == 0


def test_algorithm1_asymmetry_prefers_underfill():
    # Candidates 32 and 64 straddle the target at equal distance: with
    # lambda_o > lambda_u the underfilling one wins, with the penalties
    # swapped the overflowing one does.
    pred = _linear(0.0, 1.0)
    c, _ = _select(pred, 64, target=48.0, delta=32, lam=(1.0, 4.0))
    assert c == 32
    c, _ = _select(pred, 64, target=48.0, delta=32, lam=(4.0, 1.0))
    assert c == 64


def _apc(c_star, h, r, nd, na, u, cmax=4, smax=8, bmax=100, lmin=32):
    return ref.apc(c_star, h, r, nd, na, u, cmax, smax, bmax, lmin)


def test_apc_eq12_to_14_cases():
    # C_t = min(4, 8 - 6, (100 - 40) // 32) = 1
    assert _apc(40, 60, 100, 6, 0, 40) == (40, "accepted")
    assert _apc(40, 60, 100, 6, 1, 40) == (0, "blocked_cap")
    assert _apc(10, 60, 100, 6, 0, 40) == (32, "warm_start")       # min(h, m) = 32
    assert _apc(10, 60, 100, 6, 1, 40) == (0, "blocked_min_chunk")
    # short remainder: m = min(r, L_min) = 5
    assert _apc(5, 5, 5, 0, 0, 0) == (5, "accepted")
    # budget below L_min: C_t = 0, warm start only with an empty prefill set
    assert _apc(20, 20, 200, 0, 0, 80) == (20, "warm_start")
    assert _apc(20, 20, 200, 0, 1, 80) == (0, "blocked_min_chunk")
    # slot cap: S_max - |D_t| = 0
    assert _apc(40, 92, 100, 8, 0, 8) == (0, "blocked_cap")
    # C_max reached: C_t = min(4, 8, (200 - 10) // 32 = 5) = 4
    assert _apc(32, 32, 32, 0, 4, 10, bmax=200) == (0, "blocked_cap")
    assert _apc(32, 32, 32, 0, 3, 10, bmax=200) == (32, "accepted")
    # budget term binding: C_t = min(4, 8, (100 - 10) // 32 = 2) = 2
    assert _apc(32, 32, 32, 0, 2, 10) == (0, "blocked_cap")
    assert _apc(32, 32, 32, 0, 1, 10) == (32, "accepted")


def test_priority_eq1_hand_value():
    assert ref.priority(2.0, -0.5, 10.0, 4.0, 6) == 2.0 * 6 - 0.5 * 6


def _orders(alpha, beta, arrivals, remaining, t=1000.0):
    s = ref.Scheduler(dict(policy="aging", alpha=alpha, beta=beta, max_tokens=1, max_seqs=1,
                           chunking="budget", apc=False))
    for i, (a, r) in enumerate(zip(arrivals, remaining)):
        s.add(i, a, r, 1)
    return s._queue(t)


def test_aging_limits_are_srpt_and_fcfs():
    arrivals = [0.0, 1.0, 2.0, 3.0, 4.0]
    remaining = [500, 20, 300, 5, 80]
    # alpha / |beta| tiny: shortest remaining prefill first
    assert _orders(1e-9, -1.0, arrivals, remaining) == list(np.argsort(remaining))
    # alpha / |beta| huge: arrival order
    assert _orders(1.0, -1e-9, arrivals, remaining) == [0, 1, 2, 3, 4]


def test_aging_order_is_invariant_to_the_clock():
    # The shared alpha * t drops out of every comparison (Eq. 3-4).
    rng = np.random.default_rng(0)
    arr = list(rng.integers(0, 1000, 20).astype(float))
    rem = list(rng.integers(1, 4000, 20))
    o1 = _orders(1.0, -1 / 64, arr, rem, t=1000.0)
    o2 = _orders(1.0, -1 / 64, arr, rem, t=123456.0)
    assert o1 == o2


def _run(cfg, reqs, predict=None, max_rounds=100000):
    s = ref.Scheduler(cfg, predict)
    pending = sorted(reqs, key=lambda r: r[1])
    t, k, trace = 0, 0, []
    while k < len(pending) or s.pending():
        while k < len(pending) and pending[k][1] <= t:
            s.add(*pending[k])
            k += 1
        rows, ids, nd = s.schedule(t)
        trace.append((rows, ids, nd))
        t += 1
        s.complete(t)
        assert len(trace) < max_rounds
    return s, trace


def _workload(seed, n=40):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        out.append((i, int(rng.integers(0, 60)), int(rng.integers(1, 300)), int(rng.integers(1, 20))))
    return out


@pytest.mark.parametrize("policy", ["fcfs", "aging"])
@pytest.mark.parametrize("chunking", ["budget", "lprs"])
@pytest.mark.parametrize("apc_on", [False, True])
def test_schedule_conservation(policy, chunking, apc_on):
    cfg = dict(policy=policy, alpha=1.0, beta=-1 / 64, max_tokens=256, max_seqs=12,
               chunking=chunking, target=200.0, delta=16, lambda_u=1.0, lambda_o=4.0,
               apc=apc_on, max_active=3, min_chunk=16)
    reqs = _workload(1)
    s, trace = _run(cfg, reqs, predict=_linear(20.0, 1.0))
    seen = {}
    for rows, ids, nd in trace:
        assert sum(r[2] for r in rows) <= cfg["max_tokens"]
        assert len(rows) <= cfg["max_seqs"]
        assert len({r[0] for r in rows}) == len(rows)          # distinct slots
        assert len(set(ids)) == len(ids)                       # one chunk per request
        assert all(r[2] == 1 for r in rows[:nd])
        for (slot, start, length, ctx), rid in zip(rows, ids):
            assert ctx == start + length and 0 <= slot < cfg["max_seqs"]
            seen.setdefault(rid, []).append((start, length))
    for rid, arrival, prompt, max_new in reqs:
        pos = 0
        chunks = seen[rid]
        for start, length in chunks:
            assert start == pos                                 # contiguous, in order
            pos += length
        assert pos == prompt + max_new - 1                      # prompt once, then decodes
        r = next(q for q in s.reqs if q["id"] == rid)
        assert r["first_token"] is not None and r["first_token"] > arrival
        assert r["finish"] >= r["first_token"]


def test_decode_first_admission():
    cfg = dict(policy="fcfs", alpha=1.0, beta=-1.0, max_tokens=64, max_seqs=8,
               chunking="budget", apc=False)
    s = ref.Scheduler(cfg)
    s.add(0, 0.0, 10, 50)
    s.add(1, 0.0, 500, 5)
    rows, ids, nd = s.schedule(0.0)
    assert ids == [0, 1] and rows == [(0, 0, 10, 10), (1, 0, 54, 54)] and nd == 0
    s.complete(1.0)
    rows, ids, nd = s.schedule(1.0)
    # request 0 decodes first (one token at position 10), request 1 gets the rest
    assert nd == 1 and rows[0] == (0, 10, 1, 11) and rows[1] == (1, 54, 63, 117)
