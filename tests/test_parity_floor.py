"""The bf16 rounding the parity reports use for the error floor (the error of
the oracle's output rounded once to bfloat16), pinned on the CPU."""

import numpy as np
import torch

from gpu_util import bf16_rne, floor_errors


def test_bf16_rne_matches_the_library_on_float32_values():
    rng = np.random.default_rng(5)
    x = np.concatenate([rng.standard_normal(100_000), rng.uniform(-1e4, 1e4, 1000),
                        rng.standard_normal(1000) * 1e-20]).astype(np.float32)
    want = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(bf16_rne(x.astype(np.float64)), want)


def test_bf16_rne_ties_go_to_even_and_fp64_rounds_once():
    u = 2.0 ** -8  # half a unit in the last place of bf16 at 1.0
    assert bf16_rne(1 + u) == 1.0                  # tie, even neighbour below
    assert bf16_rne(1 + 3 * u) == 1 + 4 * u        # tie, even neighbour above
    assert bf16_rne(-(1 + 3 * u)) == -(1 + 4 * u)
    assert bf16_rne(1 + u + 2.0 ** -40) == 1 + 2 * u   # just past the tie
    # fp64 -> fp32 -> bf16 would round this to 1.0 twice over; once is up
    assert bf16_rne(1 + u + 2.0 ** -30) == 1 + 2 * u
    assert bf16_rne(0.0) == 0.0


def test_floor_is_half_an_ulp_at_most():
    rng = np.random.default_rng(6)
    ref = rng.standard_normal(50_000) * 0.3
    mx, mean = floor_errors(ref)
    assert mx <= np.abs(ref).max() * 2.0 ** -8 and 0 < mean < mx
