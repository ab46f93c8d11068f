"""Seeded random batches through the C ABI against the fp64 oracle.

The cases (fuzz_cases.py) mix decode rows, few-token, medium and long chunks
and empty rows over random geometries, so the planner's choices (tile width,
split grid, decode units inside the prefill launch, XCD cutting) differ from
case to case; a second set also draws the planner's CP_* settings.  Even
seeds run the step as two calls (cp_kv_append, cp_attn_mixed), odd seeds as
one cp_step_mixed call.  Outputs are compared element by element, both pools
bit for bit.
"""

import numpy as np
import pytest
import torch

import oracle
from fuzz_cases import apply_settings, draw_case, draw_settings
from gpu_util import assert_close, run_step, say, to_dev, words
from workloads import make_tensors

pytestmark = pytest.mark.gpu


def _check(batch, seed, what):
    one_call = seed % 2 == 1
    say(f"[gpu] {what}: heads {batch.num_q_heads}/{batch.num_kv_heads} D={batch.head_dim} "
        f"B={batch.block_size} rows={batch.rows[:, 1:3].tolist()} pool={batch.num_blocks} "
        f"one_call={one_call}")
    tens = make_tensors(batch, seed=95_000 + seed)
    kc_ref, vc_ref = oracle.kv_append(batch, tens["k_new"], tens["v_new"], tens["k_cache"],
                                      tens["v_cache"])
    ref = oracle.attn(batch, tens["q"], kc_ref, vc_ref)
    t = to_dev(tens)
    out = run_step(batch, t, one_call=one_call)
    torch.cuda.synchronize()
    assert np.array_equal(words(t["k_cache"]).reshape(-1), kc_ref.reshape(-1)), "K cache differs"
    assert np.array_equal(words(t["v_cache"]).reshape(-1), vc_ref.reshape(-1)), "V cache differs"
    if batch.num_tokens:
        assert_close(out, ref, what)


@pytest.mark.parametrize("seed", range(40))
def test_random_batch_matches_oracle(seed):
    _check(draw_case(seed), seed, f"fuzz seed {seed}")


@pytest.mark.parametrize("seed", range(24))
def test_random_batch_under_random_planner_settings(monkeypatch, seed):
    env = draw_settings(seed)
    apply_settings(monkeypatch, env)
    say(f"[gpu] settings {seed}: " + " ".join(f"{k}={v}" for k, v in env.items() if v is not None))
    _check(draw_case(100 + seed), seed, f"fuzz settings seed {seed}")
