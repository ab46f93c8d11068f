"""GPU parity of the online-softmax rescale path.

Both attention kernels keep a running maximum per query row and move it
lazily: only when a later key's base-2 score exceeds it by more than 8 are
the accumulated output and sum rescaled.  With i.i.d. N(0, 1) inputs that
never happens, so these inputs are built to force it: feature 0 of every key
grows in steps with the key's position (every 48 positions the base-2 score
rises by about 12), every query holds a large weight on feature 0, and the
other features carry a little noise.  The test asserts on the host, from the
exact bf16 inputs, that every 64-key step of a prefill item after its first
(and every 16-key tile a decode wave reads after its first) holds a score
more than 8 above the maximum of the step (tile) before it, so the branch
fires on every one of them.  Outputs are compared element by element with the
fp64 oracle; pools bit for bit.

Modes cover 128- and 256-row prefill tiles, split and unsplit key ranges,
and the decode kernel split and unsplit (including few-token rows routed to
it token by token), for G in {1, 4, 8} and D in {64, 128}.
"""

import math

import numpy as np
import pytest
import torch

import oracle
import paper_2606_09061_amd as cp
from gpu_util import assert_close, run_step, say, to_dev, words
from workloads import make_batch, make_tensors

pytestmark = pytest.mark.gpu

SEG = 48          # positions per score level
STEP2 = 12.0      # base-2 score rise per level
BETA = 8.0        # weight of feature 0 in every query
NOISE = 0.25      # scale of the other query features
FIRE = 8.0        # the kernels' lazy-rescale threshold (base 2)

GEOMS = [(8, 8, 64, 16), (32, 8, 128, 16), (16, 4, 64, 32), (64, 8, 128, 32), (8, 1, 128, 16)]

# (mode, environment)
MODES = {
    "prefill-narrow-unsplit": {"CP_PREFILL_WIDE_MIN_ROWS": "100000",
                               "CP_PREFILL_MIN_SPLIT": "100000"},
    "prefill-wide-unsplit": {"CP_PREFILL_WIDE_MIN_KEYS": "0", "CP_PREFILL_MIN_SPLIT": "100000",
                             "CP_FUSE_NARROW": "0"},
    "prefill-narrow-split": {"CP_PREFILL_WIDE_MIN_ROWS": "100000", "CP_PREFILL_MIN_SPLIT": "2",
                             "CP_PREFILL_TARGET_ITEMS": "100000"},
    "prefill-wide-split": {"CP_PREFILL_WIDE_MIN_KEYS": "0", "CP_PREFILL_MIN_SPLIT": "2",
                           "CP_FUSE_NARROW": "0",
                           "CP_PREFILL_TARGET_ITEMS": "100000"},
    "decode-unsplit": {"CP_DECODE_TARGET_ITEMS": "1", "CP_PREFILL_MIN_LEN": "8"},
    "decode-split": {"CP_DECODE_TARGET_ITEMS": "100000", "CP_PREFILL_MIN_LEN": "8"},
}

ROWS = [(0, 260), (700, 130), (999, 1), (300, 1), (2000, 1), (600, 5)]


def rising_inputs(batch, seed):
    """make_tensors, then feature 0 of each key = level(position) * g and of
    each query = BETA, other query features scaled by NOISE."""
    tens = make_tensors(batch, seed=seed)
    scale2 = float(np.float32(batch.sm_scale)) * math.log2(math.e)
    g = STEP2 / (BETA * scale2)
    q = tens["q"].float()
    q[:, :, 1:] *= NOISE
    q[:, :, 0] = BETA
    tens["q"] = q.to(torch.bfloat16)
    kn = tens["k_new"].float()
    kc = tens["k_cache"]
    B = batch.block_size
    off = batch.tok_offsets()
    for r, (req, s, c, ctx) in enumerate(batch.rows.tolist()):
        pos = np.arange(ctx)
        val = torch.tensor(g * (pos // SEG), dtype=torch.float32)
        prior = pos < s
        if prior.any():
            blk = torch.from_numpy(batch.block_tables[req, pos[prior] // B].astype(np.int64))
            slot = torch.from_numpy(pos[prior] % B)
            kc[blk, :, slot, 0] = val[torch.from_numpy(prior)].to(torch.bfloat16)[:, None]
        if c:
            kn[off[r]: off[r] + c, :, 0] = val[s:][:, None]
    tens["k_new"] = kn.to(torch.bfloat16)
    return tens


def base2_scores(batch, tens, kc, vc_unused, r):
    """fp64 base-2 scores [c, Hq, ctx] of row r from the bf16 inputs (keys
    gathered from the appended pool)."""
    req, s, c, ctx = (int(x) for x in batch.rows[r])
    B, G, D = batch.block_size, batch.group, batch.head_dim
    pos = np.arange(ctx)
    kcv = kc.reshape(batch.num_blocks, batch.num_kv_heads, B, D)
    K = kcv[batch.block_tables[req, pos // B], :, pos % B, :]          # [ctx, Hkv, D] uint16
    K = (K.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    off = int(batch.tok_offsets()[r])
    q = tens["q"][off: off + c].float().numpy().astype(np.float64)   # [c, Hq, D]
    Kh = np.repeat(K, G, axis=1)                                      # [ctx, Hq, D]
    scale2 = float(np.float32(batch.sm_scale)) * math.log2(math.e)
    S = np.matmul(q.transpose(1, 0, 2), Kh.transpose(1, 2, 0))         # [Hq, c, ctx]
    return S.transpose(1, 0, 2) * scale2


def assert_rescale_fires(batch, tens, kc):
    """Every full 64-key window after the first (prefill steps) and every
    16-key tile 64 keys after another (decode waves) has a score more than
    FIRE above the earlier one's maximum, for every query that sees it."""
    fired = 0
    for r, (req, s, c, ctx) in enumerate(batch.rows.tolist()):
        if c == 0:
            continue
        S = base2_scores(batch, tens, kc, None, r)
        for j in range(c):
            p = s + j
            sp = S[j, :, : p + 1]
            # prefill: consecutive 64-key windows, the later one full
            for m in range(1, (p + 1) // 64):
                a = sp[:, 64 * (m - 1): 64 * m].max(axis=1)
                b = sp[:, 64 * m: 64 * m + 64].max(axis=1)
                assert (b > a + FIRE).all(), (r, j, m, (b - a).min())
                fired += 1
            # decode: 16-key tiles 64 keys apart, the later one possibly partial
            for t in range(0, p // 16 - 3):
                a = sp[:, 16 * t: 16 * t + 16].max(axis=1)
                b = sp[:, 16 * (t + 4): 16 * (t + 4) + 16].max(axis=1)
                assert (b > a + FIRE).all(), (r, j, t, (b - a).min())
    return fired


def check_plan_shape(batch, mode):
    d = cp.desc_for(batch)
    items = cp.plan_items(d, batch.rows)
    pf, dc = items[items[:, 0] == 0], items[items[:, 0] == 1]
    G = batch.group
    long_pf = pf[(pf[:, 7] - pf[:, 6]) >= 128]
    if mode.startswith("prefill"):
        assert len(long_pf), "no prefill item spans two steps"
        rows_per_tile = pf[:, 2] * G
        if "wide" in mode:
            assert (rows_per_tile > 128).any(), "no 256-row tile"
        else:
            assert (rows_per_tile <= 128).all(), "a 256-row tile in narrow mode"
        covered = {}
        for it in pf.tolist():
            covered.setdefault((it[1], it[5]), []).append(it)
        split = any(len(v) > 1 for v in covered.values())
        assert split == mode.endswith("-split")
    else:
        waves = dc[(dc[:, 7] - dc[:, 6]) > 64]   # a wave reads a second tile
        assert len(waves), "no decode item reaches a second tile"
        per_tok = {}
        for it in dc.tolist():
            per_tok.setdefault((it[1], it[5]), 0)
            per_tok[(it[1], it[5])] += 1
        assert (max(per_tok.values()) > 1) == (mode == "decode-split")
        assert (dc[:, 2] == 1).all()
        assert len({it[1] for it in dc.tolist()}) >= 3 + 5   # 3 decode rows + 5 few-token tokens


@pytest.mark.parametrize("mode", list(MODES))
@pytest.mark.parametrize("geom", GEOMS, ids=lambda g: "hq%d_hkv%d_d%d_b%d" % g)
def test_rescale_path_matches_oracle(monkeypatch, geom, mode):
    for k, v in MODES[mode].items():
        monkeypatch.setenv(k, v)
    hq, hkv, d, b = geom
    rng = np.random.default_rng(hq * 1000 + d + b)
    batch = make_batch("rescale", hq, hkv, d, b, ROWS, rng)
    seed = 6000 + hq + d + b
    tens = rising_inputs(batch, seed)
    kc_ref, vc_ref = oracle.kv_append(batch, tens["k_new"], tens["v_new"], tens["k_cache"],
                                      tens["v_cache"])
    fired = assert_rescale_fires(batch, tens, kc_ref)
    check_plan_shape(batch, mode)
    say(f"[gpu] rescale {mode} {geom}: T={batch.num_tokens}, {fired} window pairs fire")
    ref = oracle.attn(batch, tens["q"], kc_ref, vc_ref)
    t = to_dev(tens)
    out = run_step(batch, t)
    torch.cuda.synchronize()
    assert np.array_equal(words(t["k_cache"]).reshape(-1), kc_ref.reshape(-1)), "K cache differs"
    assert np.array_equal(words(t["v_cache"]).reshape(-1), vc_ref.reshape(-1)), "V cache differs"
    assert_close(out, ref, f"rescale {mode} {geom}")
