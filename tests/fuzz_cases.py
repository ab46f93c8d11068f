"""Seeded random batches and planner settings shared by the GPU fuzz test
and the CPU check of their plans.

A case draws a geometry (G = 1 to 8, D 64 or 128, block 16 or 32) and 1 to
24 rows mixing one-token decode rows, 2-15-token chunks, medium and long
chunks over prior contexts of 0 to a few thousand keys, and empty rows.  The
settings draw the planner's CP_* knobs from values its sanitizer fuzz covers;
none changes what is computed, only how the work is cut and placed.
"""

import numpy as np

from workloads import make_batch

GEOMS = [(4, 4, 64, 16), (8, 4, 128, 32), (8, 2, 64, 32), (16, 2, 128, 16),
         (32, 8, 128, 16), (64, 8, 128, 32), (16, 16, 128, 32), (32, 4, 64, 16)]
# query-key-feature products per case (well under a second of fp64 oracle time)
COST_CAP = 3.0e8

SETTINGS = {
    "CP_PREFILL_MIN_LEN": ["2", "8", "16"],
    "CP_DECODE_TARGET_ITEMS": [None, "1", "300"],
    "CP_PREFILL_TARGET_ITEMS": [None, "1", "600"],
    "CP_PREFILL_MIN_SPLIT": [None, "1", "3"],
    "CP_NUM_XCDS": [None, "1", "3"],
    "CP_PREFILL_WIDE_MIN_KEYS": [None, "0", "100000"],
    "CP_PREFILL_WIDE_MIN_ROWS": [None, "1"],
    "CP_FUSE_DECODE": ["0", "1", "2", "3", "4"],
    "CP_FUSE_NARROW": ["0", "1"],
    "CP_FUSE_UNITS_PER_CU": [None, "0.01", "4"],
    "CP_XCD_PIECE_DIV": [None, "0", "1", "9"],
    "CP_XCD_BALANCE_TOL": [None, "-1", "10"],
}


def draw_case(seed):
    rng = np.random.default_rng(90_000 + seed)
    hq, hkv, d, b = GEOMS[int(rng.integers(len(GEOMS)))]
    rows, cost = [], 0.0
    for _ in range(int(rng.integers(1, 25))):
        kind = rng.choice(["decode", "few", "medium", "long", "empty"],
                          p=[0.45, 0.15, 0.2, 0.12, 0.08])
        s = int(rng.integers(0, 3000)) if rng.random() < 0.8 else 0
        c = {"decode": 1, "few": int(rng.integers(2, 16)), "medium": int(rng.integers(16, 300)),
             "long": int(rng.integers(300, 1200)), "empty": 0}[kind]
        if kind == "empty":
            s = int(rng.integers(1, 500))
        if c and cost + c * (s + c / 2) * hq * d > COST_CAP:
            # shorten the prior context to fit the budget, or leave the row out
            s = int((COST_CAP - cost) / (c * hq * d) - c / 2)
            if s < 0:
                continue
        rows.append((s, c))
        cost += c * (s + c / 2) * hq * d
    if not any(c for _, c in rows):
        rows.append((int(rng.integers(0, 100)), 1))
    pool = None
    if rng.random() < 0.5:  # spread the rows' blocks over a larger pool
        used = sum(-(-(s + c) // b) for s, c in rows)
        pool = used + 1 + int(rng.integers(0, 4 * used + 8))
    return make_batch(f"fuzz{seed}", hq, hkv, d, b, rows, rng, pool=pool)


def draw_settings(seed):
    """CP_* variables to set (name -> value) and to clear (value None)."""
    rng = np.random.default_rng(97_000 + seed)
    return {k: v[int(rng.integers(len(v)))] for k, v in SETTINGS.items()}


def apply_settings(monkeypatch, env):
    for k, v in env.items():
        if v is None:
            monkeypatch.delenv(k, raising=False)
        else:
            monkeypatch.setenv(k, v)
