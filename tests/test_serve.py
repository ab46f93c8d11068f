"""The closed serving loop (paper_2606_09061_amd/serve.py) on the CPU, with a
stand-in engine whose step latency is a known function of the batch: the
loop's bookkeeping, and LPRS holding rounds near the target when its
predictor is exact."""

import numpy as np

import workloads as wl
from oracle import sched as ref
from paper_2606_09061_amd import sched, serve

# latency (us) = 20 + 0.25 * prefill tokens + 0.5 * decode rows
#               + 2^-10 * decode context + 2^-16 * prefill x history
_W = np.zeros((1, 16))
_W[0, 0], _W[0, 1], _W[0, 3], _W[0, 15] = 0.25, 0.5, 2.0 ** -10, 2.0 ** -16
_B = np.array([20.0])


class LinearModel:
    def load_into(self, s):
        s.set_predictor([(_W, _B)], np.zeros(16), np.ones(16), 1.0)


class FakeEngine:
    def __init__(self, noise=0.0, seed=0):
        self.rng = np.random.default_rng(seed)
        self.noise = noise
        self.batches = []

    def step(self, rows):
        self.batches.append(np.array(rows))
        x = ref.features([tuple(int(v) for v in r) for r in rows])
        t = float(_B[0] + sum(_W[0, k] * x[k] for k in range(16)))
        return t * (1.0 + self.noise * self.rng.standard_normal())


def _cfg(**kw):
    d = dict(policy=sched.POLICY_FCFS, max_tokens=512, max_seqs=64, max_seq_len=4096, delta=16)
    d.update(kw)
    return sched.make_config(**d)


def test_loop_completes_every_request():
    reqs = wl.uniform_stream(150, 20.0, seed=1, prompt_median=200, output_median=20)
    eng = FakeEngine()
    r = serve.serve(_cfg(), reqs, eng, memory_features=False, record=True)
    assert r["requests"] == 150 and r["rounds"] == len(eng.batches)
    # every prompt and output token was scheduled exactly once
    total = sum(int(b[:, 2].sum()) for b in eng.batches)
    assert total == sum(p + o - 1 for _, _, p, o in reqs)
    assert r["_features"].shape == (r["rounds"], 16)
    assert r["makespan_ms"] * 1e3 >= float(np.sum(r["_step_us"])) - 1e-6
    assert r["prefill_e2e_ms"]["p50"] <= r["request_e2e_ms"]["p50"]


def test_idle_gaps_jump_to_the_next_arrival():
    reqs = [(0, 0.0, 10, 2), (1, 1e6, 10, 2)]
    r = serve.serve(_cfg(), reqs, FakeEngine(), memory_features=False)
    assert r["makespan_ms"] > 1e3 and r["rounds"] == 4


def test_lprs_with_an_exact_predictor_holds_the_target():
    # T* = the token-budget run's mean round: LPRS (with APC against
    # one-token fragments) spreads prefill work so rounds stay near it, where
    # the token budget alternates between decode-only and full rounds.
    reqs = wl.uniform_stream(300, 10.0, seed=2, prompt_median=400, output_median=40)
    tb = serve.serve(_cfg(target_us=0.0), reqs, FakeEngine(), memory_features=False, record=True)
    t_star = float(np.mean(tb["_step_us"]))
    lp = serve.serve(_cfg(chunking=sched.CHUNK_LPRS, target_us=t_star, apc=True), reqs,
                     FakeEngine(), predictor=LinearModel(), memory_features=False)
    dev_tb = np.abs(tb["_step_us"] - t_star).mean()
    assert lp["mean_abs_dev_from_target_us"] < 0.5 * dev_tb
    assert lp["step_us"]["p99"] < 0.6 * tb["step_us"]["p99"]
    assert lp["online_prediction"]["mae_us"] < 1e-9


def test_apc_counts_interventions_and_enlarges_chunks():
    reqs = wl.short_long_stream(300, busy_interval_us=2.0, quiet_interval_us=50.0, seed=3)
    res = {}
    for on in (False, True):
        res[on] = serve.serve(_cfg(chunking=sched.CHUNK_LPRS, target_us=60.0, apc=on,
                                   max_active=2, min_chunk=16),
                              reqs, FakeEngine(), predictor=LinearModel(), memory_features=False)
    assert res[False]["apc_blocked_cap"] == 0 and res[False]["apc_blocked_min_chunk"] == 0
    assert res[True]["apc_blocked_cap"] + res[True]["apc_blocked_min_chunk"] > 0
    assert res[True]["avg_prefill_chunk"] > res[False]["avg_prefill_chunk"]


def test_step_engine_plans_once_and_grows_workspace_on_demand(monkeypatch):
    """The engine asks for the workspace size only after a call reported it
    too small (CP_ERR_WORKSPACE, nothing enqueued), then repeats that call."""
    import torch
    from paper_2606_09061_amd import binding

    eng = object.__new__(serve.StepEngine)
    eng.dev = torch.device("cpu")
    eng.desc = None
    eng.ws = torch.empty(256, dtype=torch.uint8)
    sizes = []
    monkeypatch.setattr(binding, "workspace_bytes", lambda d, r: sizes.append(1) or 4096)
    calls = []

    def call():
        calls.append(eng.ws.numel())
        if eng.ws.numel() < 4096:
            raise binding.CpError(binding.CP_ERR_WORKSPACE, "cp_attn_mixed")

    eng._grow_on_demand(call, np.zeros((1, 4), np.int32))
    assert calls == [256, 4096] and len(sizes) == 1 and eng.ws.numel() == 4096
    calls.clear()
    eng._grow_on_demand(call, np.zeros((1, 4), np.int32))   # big enough: no size query
    assert calls == [4096] and len(sizes) == 1

    def other():
        raise binding.CpError(binding.CP_ERR_BAD_META, "cp_attn_mixed")
    try:
        eng._grow_on_demand(other, np.zeros((1, 4), np.int32))
        raise AssertionError("error swallowed")
    except binding.CpError as e:
        assert e.code == binding.CP_ERR_BAD_META
