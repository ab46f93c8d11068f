"""The seeded input generators: reproducibility and the scheduling rules the
synthetic mixes are built from (decode-first admission, token budget, one
chunk per request, Eq. 2 bookkeeping, Eq. 4 ordering, Eq. 12-14 gating)."""

import numpy as np
import pytest
import torch

from workloads import make_batch, make_config, make_tensors, replay_schedule
from workloads.tensors import tail_slots


def _check_batch(b):
    rows = b.rows
    assert (rows[:, 3] == rows[:, 1] + rows[:, 2]).all()
    assert len(set(rows[:, 0].tolist())) == b.n_rows           # one chunk per request
    assert (rows[:, 3] <= b.max_blocks_per_req * b.block_size).all()
    assert (b.block_tables >= 0).all() and (b.block_tables < b.num_blocks).all()
    # no physical block is shared by two requests' live ranges
    seen = {}
    for req, s, c, ctx in rows.tolist():
        for blk in b.block_tables[req, : -(-ctx // b.block_size)].tolist():
            assert blk not in seen or seen[blk] == req
            seen[blk] = req
    assert b.poison_block not in seen


@pytest.mark.parametrize("n", [1, 2, 3, 4])
def test_configs_reproducible_and_valid(n):
    a, b = make_config(n), make_config(n)
    assert np.array_equal(a.rows, b.rows) and np.array_equal(a.block_tables, b.block_tables)
    _check_batch(a)


def test_config_shapes():
    c1 = make_config(1)
    assert sorted(map(tuple, c1.rows[:, 1:].tolist())) == sorted(
        [(0, 64, 64), (128, 48, 176), (199, 1, 200), (36, 1, 37)])
    c2, c3, c4 = make_config(2), make_config(3), make_config(4)
    assert c2.num_tokens == 512 and (c2.rows[:, 2] == 192).sum() == 2
    assert ((c2.rows[:, 2] == 1) & (c2.rows[:, 3] >= 16) & (c2.rows[:, 3] <= 8192)).sum() == 128
    assert c3.num_tokens == 2048
    assert sorted(c3.rows[c3.rows[:, 2] == 480, 1].tolist()) == [0, 8192, 16384, 31744]
    assert c4.num_tokens == 512 and (c4.rows[:, 2] == 1).sum() == 256
    assert (c4.rows[:, 3] <= 32768).all()
    for c in (c2, c3, c4):
        dec_first = np.nonzero(c.rows[:, 2] == 1)[0]
        assert dec_first.max() < np.nonzero(c.rows[:, 2] > 1)[0].min()   # decode rows first


def test_replay_rules():
    batches, info = replay_schedule()
    assert len(batches) == 20
    done = {}
    gen = {}
    for it, b in enumerate(batches):
        _check_batch(b)
        r = b.rows
        assert r[:, 2].sum() <= 4096                       # token budget
        is_dec = np.array([row[0] in gen and gen[row[0]] >= 1 for row in r.tolist()], bool)
        # decode rows come first and are one token
        if is_dec.any():
            assert is_dec[: is_dec.sum()].all()
            assert (r[is_dec, 2] == 1).all()
        n_pf = int((~is_dec).sum())
        assert n_pf <= 4                                    # C_max
        for req, s, c, ctx in r.tolist():
            if req in gen and gen[req] >= 1:
                assert s == info["prompts"][req] + gen[req] - 1
                gen[req] += 1
            else:
                assert s == done.get(req, 0)                 # Eq. 2: chunk starts where the last stopped
                assert req // 4 <= it                        # arrived
                done[req] = s + c
                if done[req] == info["prompts"][req]:
                    gen[req] = 1
    # max ctx and prefill depth of the replay
    assert max(int(b.rows[:, 3].max()) for b in batches) <= 32768 + 4096


def test_replay_aging_order():
    """Among prefill candidates the chosen order follows the aging key (Eq. 4)."""
    batches, info = replay_schedule(n_req=16, iters=6, budget=1024)
    prompts = info["prompts"]
    done = {}
    gen = {}
    for it, b in enumerate(batches):
        pf = [(req, s) for req, s, c, ctx in b.rows.tolist() if not (req in gen)]
        keys = [-(req // 4) - (prompts[req] - s) / 256.0 for req, s in pf]
        assert keys == sorted(keys, reverse=True) or len(set(keys)) < len(keys)
        for req, s, c, ctx in b.rows.tolist():
            if req in gen:
                gen[req] += 1
            else:
                done[req] = s + c
                if done[req] == prompts[req]:
                    gen[req] = 1


def test_tensors_poison_and_seed():
    b = make_config(1)
    t1 = make_tensors(b, seed=5)
    t2 = make_tensors(b, seed=5)
    for k in t1:
        assert torch.equal(t1[k].view(torch.int16) if t1[k].dtype == torch.bfloat16 else t1[k],
                           t2[k].view(torch.int16) if t2[k].dtype == torch.bfloat16 else t2[k])
    kc = t1["k_cache"]
    blk, slot = tail_slots(b)
    assert torch.isnan(kc[torch.from_numpy(blk), :, torch.from_numpy(slot), :].float()).all()
    unref = np.nonzero(~b.referenced)[0]
    assert torch.isnan(kc[torch.from_numpy(unref)].float()).all()
    # prior context is finite
    for req, s, c, ctx in b.rows.tolist():
        for p in range(s):
            assert torch.isfinite(kc[b.block_tables[req, p // 16], :, p % 16].float()).all()


def test_subset_keeps_rows_tables_and_pool():
    from workloads import subset
    b = make_config(2)
    dec = subset(b, b.rows[:, 2] == 1, "decode")
    pf = subset(b, b.rows[:, 2] >= 2, "prefill")
    assert dec.n_rows + pf.n_rows == b.n_rows
    assert (dec.rows[:, 2] == 1).all() and (pf.rows[:, 2] >= 2).all()
    assert dec.block_tables is b.block_tables and pf.num_blocks == b.num_blocks
    assert dec.num_tokens + pf.num_tokens == b.num_tokens


def test_make_batch_in_fixed_pool_draws_distinct_blocks():
    rng = np.random.default_rng(11)
    sl = [(1000, 1), (4095, 1), (0, 300), (8192, 64)]
    b = make_batch("pooled", 32, 8, 128, 16, sl, rng, pool=5000)
    assert b.num_blocks == 5000
    used = []
    for rid, s, c, ctx in b.rows.tolist():
        nb = -(-ctx // 16)
        used.extend(b.block_tables[rid, :nb].tolist())
    assert len(used) == len(set(used)) and max(used) < 5000 and min(used) >= 0
    assert b.poison_block not in used
    with pytest.raises(ValueError):
        make_batch("small", 32, 8, 128, 16, sl, np.random.default_rng(1), pool=10)
