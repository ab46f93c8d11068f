"""Host-only checks of libcpattn: exported symbols, validation error codes and
exact coverage of the planner's work items.  Nothing here launches a kernel."""

import ctypes
import os
import re

import numpy as np
import pytest

import paper_2606_09061_amd as cp
from paper_2606_09061_amd import binding
from workloads import make_batch, make_config, replay_schedule

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def header_functions():
    src = open(os.path.join(ROOT, "include", "cp_attn.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(cp_[a-z_]+)\s*\(", src)))


def test_library_exports_every_declared_function():
    lib = binding.load()
    names = header_functions()
    assert len(names) >= 10
    for n in names:
        assert hasattr(lib, n), f"{n} declared in cp_attn.h but not exported"
    assert sorted(binding.exported_symbols()) == names


def test_version_and_strerror():
    assert cp.version() == 10000
    for code in (0, -1, -2, -3, -4, -5):
        assert binding.strerror(code) != "unknown error"
    assert binding.strerror(-99) == "unknown error"


def _desc(**kw):
    base = dict(num_q_heads=32, num_kv_heads=8, head_dim=128, block_size=16, num_blocks=100,
                max_blocks_per_req=10, num_reqs_in_table=4, sm_scale=0.088)
    base.update(kw)
    return cp.make_desc(**base)


GOOD_ROWS = np.array([[0, 10, 5, 15], [1, 0, 1, 1]], np.int32)


@pytest.mark.parametrize("kw,code", [
    (dict(num_q_heads=0), binding.CP_ERR_INVALID_ARG),
    (dict(num_blocks=0), binding.CP_ERR_INVALID_ARG),
    (dict(num_q_heads=12, num_kv_heads=8), binding.CP_ERR_BAD_META),
    (dict(sm_scale=float("nan")), binding.CP_ERR_BAD_META),
    (dict(sm_scale=-1.0), binding.CP_ERR_BAD_META),
    (dict(sm_scale=0.0), binding.CP_ERR_BAD_META),
    (dict(sm_scale=float("inf")), binding.CP_ERR_BAD_META),
    (dict(head_dim=96), binding.CP_ERR_UNSUPPORTED),
    (dict(block_size=8), binding.CP_ERR_UNSUPPORTED),
    (dict(num_q_heads=48, num_kv_heads=3), binding.CP_ERR_UNSUPPORTED),
    (dict(num_q_heads=32, num_kv_heads=2), binding.CP_ERR_UNSUPPORTED),
])
def test_desc_validation(kw, code):
    assert cp.check_batch(_desc(**kw), GOOD_ROWS) == code


@pytest.mark.parametrize("row,code", [
    ([0, 10, -1, 9], binding.CP_ERR_BAD_META),     # negative chunk
    ([0, -1, 2, 1], binding.CP_ERR_BAD_META),      # negative start
    ([0, 10, 5, 16], binding.CP_ERR_BAD_META),     # ctx != start + len
    ([0, 150, 20, 170], binding.CP_ERR_BAD_META),  # ctx beyond the table capacity (160)
    ([7, 0, 1, 1], binding.CP_ERR_BAD_META),       # req out of range
    ([-1, 0, 1, 1], binding.CP_ERR_BAD_META),
    ([1, 3, 1, 4], binding.CP_ERR_BAD_META),       # duplicate req in one batch
])
def test_row_validation(row, code):
    rows = np.array([[1, 0, 1, 1], row], np.int32)
    assert cp.check_batch(_desc(), rows) == code


def test_good_batch_and_empty_batch_validate():
    assert cp.check_batch(_desc(), GOOD_ROWS) == 0
    assert cp.check_batch(_desc(), np.zeros((0, 4), np.int32)) == 0


def test_compute_calls_reject_before_touching_anything():
    """Bad metadata, null pointers and short workspaces are refused on the host
    (the pointers below are never dereferenced; no GPU is needed)."""
    lib = binding.load()
    d = _desc()
    bad = np.array([[0, 10, 5, 16]], np.int32)
    fake = 1 << 20  # never dereferenced
    rc = lib.cp_attn_mixed(ctypes.byref(d), fake, fake, fake, fake, bad.ctypes.data, 1, fake,
                           fake, 1 << 30, None)
    assert rc == binding.CP_ERR_BAD_META
    rc = lib.cp_kv_append(ctypes.byref(d), fake, fake, fake, fake, fake, bad.ctypes.data, 1,
                          fake, 1 << 30, None)
    assert rc == binding.CP_ERR_BAD_META
    good = GOOD_ROWS
    rc = lib.cp_attn_mixed(ctypes.byref(d), None, fake, fake, fake, good.ctypes.data, 2, fake,
                           fake, 1 << 30, None)
    assert rc == binding.CP_ERR_INVALID_ARG
    rc = lib.cp_attn_mixed(ctypes.byref(d), fake + 2, fake, fake, fake, good.ctypes.data, 2,
                           fake, fake, 1 << 30, None)
    assert rc == binding.CP_ERR_INVALID_ARG  # misaligned q
    need = cp.workspace_bytes(d, good)
    rc = lib.cp_attn_mixed(ctypes.byref(d), fake, fake, fake, fake, good.ctypes.data, 2, fake,
                           fake, need - 1, None)
    assert rc == binding.CP_ERR_WORKSPACE
    rc = lib.cp_kv_append(ctypes.byref(d), fake, fake, fake, fake, fake, good.ctypes.data, 2,
                          fake, 0, None)
    assert rc == binding.CP_ERR_WORKSPACE
    # the one-call step: the same checks, before anything is enqueued
    step = lib.cp_step_mixed
    assert step(ctypes.byref(d), fake, fake, fake, fake, fake, fake, bad.ctypes.data, 1, fake,
                fake, 1 << 30, None) == binding.CP_ERR_BAD_META
    assert step(ctypes.byref(d), fake, None, fake, fake, fake, fake, good.ctypes.data, 2, fake,
                fake, 1 << 30, None) == binding.CP_ERR_INVALID_ARG
    assert step(ctypes.byref(d), fake, fake, fake + 8, fake, fake, fake, good.ctypes.data, 2,
                fake, fake, 1 << 30, None) == binding.CP_ERR_INVALID_ARG  # misaligned v_new
    assert step(ctypes.byref(d), fake, fake, fake, fake, fake, fake, good.ctypes.data, 2, fake,
                fake, need - 1, None) == binding.CP_ERR_WORKSPACE
    # an empty batch succeeds without touching its (null) buffers
    empty = np.zeros((0, 4), np.int32)
    assert step(ctypes.byref(d), None, None, None, None, None, None, empty.ctypes.data, 0, None,
                None, 0, None) == 0
    assert lib.cp_attn_mixed(ctypes.byref(d), None, None, None, None, empty.ctypes.data, 0, None,
                             None, 0, None) == 0
    assert lib.cp_kv_append(ctypes.byref(d), None, None, None, None, None, empty.ctypes.data, 0,
                            None, 0, None) == 0


def test_workspace_bytes_zero_for_invalid():
    with pytest.raises(binding.CpError):
        cp.workspace_bytes(_desc(head_dim=96), GOOD_ROWS)


# ----------------------------------------------------------------- planner coverage

def _check_coverage(batch, min_len=2):
    """Every (token, kv head) of the batch is covered by items whose key ranges
    partition [0, end) with the token's position p < end <= ctx.  Rows of at
    least ``min_len`` tokens are prefill tiles; shorter rows are decode items,
    one per token, each ending exactly at its own causal limit p + 1."""
    d = cp.desc_for(batch)
    items = cp.plan_items(d, batch.rows)
    G = batch.group
    Hkv = batch.num_kv_heads
    off = batch.tok_offsets()
    # token -> (row, position)
    cover = {}
    for kind, tok0, ntok, pos0, req, kvh, kb, ke in items.tolist():
        assert 0 <= kvh < Hkv and ke > kb >= 0
        for j in range(ntok):
            cover.setdefault((tok0 + j, kvh), []).append((kind, kb, ke, pos0, ntok, req))
    seen = set()
    for r, (req, s, c, ctx) in enumerate(batch.rows.tolist()):
        for j in range(c):
            t = off[r] + j
            p = s + j
            for kvh in range(Hkv):
                lst = cover.get((t, kvh))
                assert lst, f"token {t} head {kvh} not covered"
                seen.add((t, kvh))
                kinds = {x[0] for x in lst}
                assert kinds == ({0} if c >= min_len else {1})
                assert all(x[5] == req for x in lst)
                ranges = sorted((x[1], x[2]) for x in lst)
                # the ranges partition [0, end) with p < end <= ctx
                assert ranges[0][0] == 0
                for a, b in zip(ranges, ranges[1:]):
                    assert a[1] == b[0], f"gap/overlap {a} {b}"
                end = ranges[-1][1]
                assert p < end <= ctx
                # every split holds a key the token may see
                for kb, ke in ranges:
                    assert kb <= p
                if c < min_len:
                    assert end == p + 1, f"decode token at {p} ends at {end}"
                    assert all(x[3] == p and x[4] == 1 for x in lst)
    assert seen == set(cover), "items cover tokens outside the batch"


@pytest.mark.parametrize("n", [1, 2, 3, 4])
def test_plan_covers_every_query_exactly_once(n):
    _check_coverage(make_config(n))


def test_plan_coverage_replay_and_ragged():
    batches, _ = replay_schedule()
    for b in batches[::4]:
        _check_coverage(b)
    rng = np.random.default_rng(3)
    for hq, hkv, d, bs in ((8, 8, 64, 16), (16, 2, 128, 32), (8, 1, 128, 16)):
        rows = [(int(s), int(c)) for s, c in zip(rng.integers(0, 5000, 12),
                                                  rng.integers(0, 700, 12))]
        rows += [(0, 1), (31, 1), (4095, 1), (7, 0)]
        _check_coverage(make_batch("ragged", hq, hkv, d, bs, rows, rng))


def test_plan_summary_counts_consistent():
    b = make_config(3)
    s = cp.plan_summary(cp.desc_for(b), b.rows)
    items = cp.plan_items(cp.desc_for(b), b.rows)
    assert s["prefill_items"] + s["decode_items"] == len(items)
    assert s["workspace_bytes"] == cp.workspace_bytes(cp.desc_for(b), b.rows)
    assert s["workspace_bytes"] >= s["partial_rows"] * (b.head_dim + 1) * 4


def test_attn_prepare_and_run_reject_bad_input():
    lib = binding.load()
    plan = binding.AttnPlan()
    bad = _desc(head_dim=96)
    r = np.ascontiguousarray(GOOD_ROWS)
    assert lib.cp_attn_prepare(ctypes.byref(bad), r.ctypes.data, 2, None, 0, None,
                               ctypes.byref(plan)) == binding.CP_ERR_UNSUPPORTED
    d = _desc()
    assert lib.cp_attn_prepare(ctypes.byref(d), r.ctypes.data, 2, None, 0, None,
                               None) == binding.CP_ERR_INVALID_ARG
    # an empty batch prepares without a workspace, and its plan runs as a no-op
    empty = np.zeros((1, 4), np.int32)
    assert lib.cp_attn_prepare(ctypes.byref(d), empty.ctypes.data, 1, None, 0, None,
                               ctypes.byref(plan)) == binding.CP_OK
    assert plan.tokens == 0
    assert lib.cp_attn_run(ctypes.byref(plan), None, None, None, None, None, None, 0,
                           None) == binding.CP_OK
    # a plan with work: missing buffers, a short workspace and offsets outside it are refused
    # before anything is launched
    plan.tokens, plan.ws_bytes, plan.n_decode = 5, 1 << 20, 1
    assert lib.cp_attn_run(ctypes.byref(plan), None, None, None, None, None, None, 1 << 20,
                           None) == binding.CP_ERR_INVALID_ARG
    assert lib.cp_attn_run(ctypes.byref(plan), 256, 256, 256, 256, 256, 256, 1024,
                           None) == binding.CP_ERR_WORKSPACE
    plan.off_decode = 2 << 20
    assert lib.cp_attn_run(ctypes.byref(plan), 256, 256, 256, 256, 256, 256, 1 << 20,
                           None) == binding.CP_ERR_INVALID_ARG
    plan.off_decode, plan.n_merge = 0, -1
    assert lib.cp_attn_run(ctypes.byref(plan), 256, 256, 256, 256, 256, 256, 1 << 20,
                           None) == binding.CP_ERR_INVALID_ARG


def test_prefill_tile_width_follows_the_step_key_range():
    # 32/8 heads: a 256-row tile holds 64 tokens, a 128-row tile 32
    d = _desc(num_blocks=4096, max_blocks_per_req=600, num_reqs_in_table=4)

    def widest(rows):
        items = cp.plan_items(d, np.array(rows, np.int32))
        return int(items[items[:, 0] == 0][:, 2].max())

    assert widest([[0, 0, 256, 256]]) == 32                 # mean key range 128: 128-row tiles
    assert widest([[0, 8192, 256, 8448]]) == 64             # 8,320: 256-row tiles
    # one width for the whole step: its token-weighted mean decides (here 4,224)
    assert widest([[0, 0, 256, 256], [1, 8192, 256, 8448]]) == 64
    assert widest([[0, 0, 2000, 2000], [1, 1200, 8, 1208]]) == 32   # (2000*1000 + 8*1204)/2008


def test_fused_split_estimate_counts_the_decode_units(monkeypatch):
    """With the decode rows inside the prefill launch, their units fill the
    launch's slots too, so a step whose decode work dominates keeps its
    prefill tiles unsplit (no merge traffic) where the prefill rows alone
    would have been split; a prefill-heavy step still splits."""
    b = make_config(2)   # 2 x 192-token chunks + 128 decode rows (decode-heavy)
    d = cp.desc_for(b)
    monkeypatch.setenv("CP_FUSE_NARROW", "0")
    fused = cp.plan_summary(d, b.rows)
    monkeypatch.setenv("CP_FUSE_DECODE", "0")
    alone = cp.plan_summary(d, b.rows)
    assert fused["prefill_items"] < alone["prefill_items"]
    monkeypatch.delenv("CP_FUSE_DECODE")
    monkeypatch.delenv("CP_FUSE_NARROW")
    b3 = make_config(3)  # prefill-heavy: long prior contexts still split (128-row tiles)
    s3 = cp.plan_summary(cp.desc_for(b3), b3.rows)
    tiles3 = 4 * -(-480 * 4 // 128) * 8
    assert s3["prefill_items"] > tiles3


def test_fused_steps_use_128_row_tiles_and_fewer_decode_units(monkeypatch):
    """A step whose decode rows run inside the prefill launch takes 128-row
    tiles (unless CP_FUSE_NARROW=0) and, when its prefill flops dominate,
    about one decode unit per CU."""
    d = _desc(num_blocks=4096, max_blocks_per_req=600, num_reqs_in_table=4)
    rows = np.array([[0, 8192, 256, 8448], [1, 9000, 1, 9001]], np.int32)

    def widest_and_units():
        items = cp.plan_items(d, rows)
        return int(items[items[:, 0] == 0][:, 2].max()), int((items[:, 0] == 1).sum())

    monkeypatch.setenv("CP_NUM_CUS", "256")
    w, units = widest_and_units()
    assert w == 32 and units <= 256
    monkeypatch.setenv("CP_FUSE_NARROW", "0")
    assert widest_and_units()[0] == 64
    monkeypatch.delenv("CP_FUSE_NARROW")
    monkeypatch.setenv("CP_FUSE_DECODE", "0")
    w, units0 = widest_and_units()
    assert w == 64 and units0 > units


FEW_TOKEN_ROWS = [(0, 2), (5, 3), (100, 2), (4000, 7), (31, 15), (16, 16), (999, 1), (0, 1),
                  (2047, 40), (3, 0)]


@pytest.mark.parametrize("min_len", [2, 3, 8, 16, 64])
def test_plan_routes_short_rows_to_decode_token_by_token(monkeypatch, min_len):
    """CP_PREFILL_MIN_LEN sends rows shorter than it to the decode kernel with
    one item list per token (its own causal limit); any value is exact."""
    monkeypatch.setenv("CP_PREFILL_MIN_LEN", str(min_len))
    rng = np.random.default_rng(min_len)
    for hq, hkv, d, bs in ((32, 8, 128, 16), (64, 8, 128, 32), (8, 8, 64, 16), (16, 2, 64, 32)):
        _check_coverage(make_batch("few", hq, hkv, d, bs, FEW_TOKEN_ROWS, rng), min_len)


@pytest.mark.parametrize("value,effective", [("1", 2), ("0", 2), ("-5", 2), ("65", 64),
                                             ("100000", 64), ("junk", 2)])
def test_prefill_min_len_is_clamped(monkeypatch, value, effective):
    monkeypatch.setenv("CP_PREFILL_MIN_LEN", value)
    rng = np.random.default_rng(4)
    rows = [(10, c) for c in (1, 2, 63, 64, 65)]
    b = make_batch("clamp", 32, 8, 128, 16, [(10 * i, c) for i, (s, c) in enumerate(rows)], rng)
    _check_coverage(b, effective)


def test_attn_run_rejects_lists_past_the_workspace():
    """Each list end (offset + length x item size) must lie inside the plan's
    workspace; a stale or edited plan is refused before any launch."""
    lib = binding.load()
    d = _desc()

    def run(**kw):
        plan = binding.AttnPlan()
        plan.desc = d
        plan.tokens, plan.ws_bytes = 5, 4096
        for k, v in kw.items():
            setattr(plan, k, v)
        return lib.cp_attn_run(ctypes.byref(plan), 256, 256, 256, 256, 256, 256, 4096, None)

    big = 4096
    assert run(off_decode=big - 64, n_decode=3) == binding.CP_ERR_INVALID_ARG     # 96 B past 4032
    assert run(off_merge=big - 32, n_merge=2) == binding.CP_ERR_INVALID_ARG
    assert run(off_prefill=big - 32, n_prefill_items=2) == binding.CP_ERR_INVALID_ARG
    assert run(off_prefill_wide=0, n_prefill_wide_items=129) == binding.CP_ERR_INVALID_ARG
    assert run(off_part_o=0, partial_rows=9) == binding.CP_ERR_INVALID_ARG        # 9 x 512 B
    assert run(off_part_lse=big - 8, partial_rows=3) == binding.CP_ERR_INVALID_ARG
    assert run(n_prefill_items=-1) == binding.CP_ERR_INVALID_ARG
    assert run(partial_rows=-1) == binding.CP_ERR_INVALID_ARG
    # decode items placed inside a prefill launch that the plan does not have
    assert run(decode_in_prefill=1, n_decode=1, off_decode=0) == binding.CP_ERR_INVALID_ARG
    assert run(decode_in_prefill=2, n_decode=1, off_decode=0, n_prefill_items=1,
               off_prefill=256) == binding.CP_ERR_INVALID_ARG
    assert run(decode_in_prefill=3) == binding.CP_ERR_INVALID_ARG
    assert run(decode_in_prefill=-1) == binding.CP_ERR_INVALID_ARG
    # empty lists may start at the very end of the workspace (nothing to
    # launch, so this runs on a CPU)
    assert run(off_prefill=big, off_prefill_wide=big, off_decode=big, off_merge=big,
               off_part_o=big, off_part_lse=big) == binding.CP_OK


def test_prepared_plan_lists_fit_its_workspace():
    for n in (2, 3, 4):
        b = make_config(n)
        d = cp.desc_for(b)
        s = cp.plan_summary(d, b.rows)
        assert s["workspace_bytes"] == cp.workspace_bytes(d, b.rows)
        assert s["workspace_bytes"] >= s["partial_rows"] * (b.head_dim + 1) * 4


def test_check_block_tables_host():
    b = make_config(2)
    d = cp.desc_for(b)
    bt = b.block_tables.copy()
    assert cp.check_block_tables(d, bt, b.rows) == binding.CP_OK
    # an entry past a row's context is never read: any value is accepted there
    req, s, c, ctx = (int(x) for x in b.rows[0])
    nb = -(-ctx // b.block_size)
    if nb < bt.shape[1]:
        bt2 = bt.copy()
        bt2[req, nb] = -7
        assert cp.check_block_tables(d, bt2, b.rows) == binding.CP_OK
    for bad in (-1, b.num_blocks, 1 << 30):
        bt2 = bt.copy()
        bt2[req, nb - 1] = bad                      # the row's last block
        assert cp.check_block_tables(d, bt2, b.rows) == binding.CP_ERR_BAD_META
        bt2 = bt.copy()
        bt2[req, 0] = bad
        assert cp.check_block_tables(d, bt2, b.rows) == binding.CP_ERR_BAD_META
    lib = binding.load()
    r = np.ascontiguousarray(b.rows)
    assert lib.cp_check_block_tables(ctypes.byref(d), None, r.ctypes.data,
                                     r.shape[0]) == binding.CP_ERR_INVALID_ARG
    assert cp.check_block_tables(_desc(head_dim=96), bt, b.rows) == binding.CP_ERR_UNSUPPORTED


def test_compute_calls_reject_bad_tables_under_debug_only_after_validation(monkeypatch):
    """With CP_DEBUG=1 a malformed batch is still refused by validation first
    (no device access happens for it, so no GPU is needed here)."""
    monkeypatch.setenv("CP_DEBUG", "1")
    lib = binding.load()
    d = _desc()
    bad = np.array([[0, 10, 5, 16]], np.int32)
    fake = 1 << 20
    assert lib.cp_attn_mixed(ctypes.byref(d), fake, fake, fake, fake, bad.ctypes.data, 1, fake,
                             fake, 1 << 30, None) == binding.CP_ERR_BAD_META


# ------------------------------------------------- decode blocks in the prefill launch

def _layouts(batch, monkeypatch, mode):
    # same tile widths, prefill split and decode split in every mode, so that
    # only the placement differs
    monkeypatch.setenv("CP_FUSE_NARROW", "0")
    monkeypatch.setenv("CP_DECODE_TARGET_ITEMS", "700")
    monkeypatch.setenv("CP_PREFILL_TARGET_ITEMS", "600")
    monkeypatch.setenv("CP_FUSE_DECODE", str(mode))
    d = cp.desc_for(batch)
    return [cp.plan_records(d, batch.rows, w) for w in (0, 1)], cp.plan_items(d, batch.rows)


def _fuse_batches():
    out = [make_config(n) for n in (1, 2, 3)]
    batches, _ = replay_schedule()
    out += [batches[i] for i in (1, 4, 9, 15, 19)]
    rng = np.random.default_rng(12)
    out.append(make_batch("wide-only", 32, 8, 128, 16,
                          [(3000, 480), (0, 1), (900, 1), (4000, 1)], rng))
    out.append(make_batch("g1", 8, 8, 64, 32, [(100, 300), (50, 2), (7, 1), (4000, 1)], rng))
    return out


@pytest.mark.parametrize("mode", [1, 2, 3, 4])
def test_decode_blocks_in_the_prefill_launch(monkeypatch, mode):
    """Placing the decode units inside the last prefill launch changes no work
    item, names every unit exactly once (one per 4-wave workgroup, two per
    8-wave one), and keeps every tile at its position modulo the XCD count
    (modes 2 and 3) or at its exact position (mode 1)."""
    X = 8
    for b in _fuse_batches():
        (n0, w0), items0 = _layouts(b, monkeypatch, 0)
        (n1, w1), items1 = _layouts(b, monkeypatch, mode)
        key = lambda a: sorted(map(tuple, a.tolist()))
        assert key(items0) == key(items1), b.name
        for recs in (n0, w0):
            assert not (recs[:, 1] < 0).any()
        n_dec = int((items0[:, 0] == 1).sum())
        has_pf = len(n0) + len(w0) > 0
        if n_dec == 0 or not has_pf:
            assert np.array_equal(n0, n1) and np.array_equal(w0, w1), b.name
            continue
        wide = len(n0) == 0
        fused, plain = (w1, w0) if wide else (n1, n0)
        other0, other1 = (n0, n1) if wide else (w0, w1)
        assert np.array_equal(other0, other1)
        marks = fused[fused[:, 1] == -1]
        per = 2 if wide else 1
        units = marks[:, 0].tolist() + [u for u in marks[:, 2].tolist() if u >= 0]
        assert sorted(units) == list(range(n_dec)), b.name
        if not wide:
            assert (marks[:, 2] == -1).all()
        assert len(marks) == -(-n_dec // per)
        tiles1 = [(i % X, tuple(r)) for i, r in enumerate(fused.tolist()) if r[1] > 0]
        tiles0 = [(i % X, tuple(r)) for i, r in enumerate(plain.tolist()) if r[1] > 0]
        assert [t for _, t in tiles1] == [t for _, t in tiles0], b.name
        if mode == 1:
            assert np.array_equal(fused[: len(plain)], plain)
            assert (fused[len(plain):, 1] == -1).all()
        else:
            assert tiles1 == tiles0, b.name
        if mode == 2:
            first_tile = min(i for i, r in enumerate(fused.tolist()) if r[1] > 0)
            assert (fused[:first_tile, 1] <= 0).all() and first_tile >= len(marks)
        if mode == 3 and len(marks) >= 2 * X and len(tiles0) >= 4 * X:
            # spread: decode blocks in both halves of the list
            pos = np.flatnonzero(fused[:, 1] == -1)
            assert pos.min() < len(fused) // 2 < pos.max()
        assert len(fused) == 0 or fused[-1, 1] != 0   # no trailing idle records


def _xcd_loads(recs, X=8):
    """Key steps of the tile records dealt to each XCD (record i runs on XCD
    i mod X)."""
    loads = np.zeros(X)
    for i, r in enumerate(recs.tolist()):
        if r[1] > 0:
            loads[i % X] += -(-(r[5] - r[4]) // 64) + 3
    return loads


def test_few_kv_groups_are_cut_across_xcds(monkeypatch):
    """With one kv head (an 8-way head shard of the 70B layer) the K/V groups
    are too few and too unequal to balance eight XCDs whole; the planner then
    cuts them into runs of tiles.  The launch keeps exactly the same tiles
    (only their positions move), every token stays covered, and the busiest
    XCD's load falls toward the mean.  Full-head batches, whose groups
    balance, keep their layout."""
    import bench
    batches, _ = replay_schedule()
    for j in (0, 3, 9, 15, 19):
        b = bench.shard_heads(batches[j], 8)
        d = cp.desc_for(b)
        monkeypatch.setenv("CP_XCD_PIECE_DIV", "0")
        whole = cp.plan_records(d, b.rows, 0)
        monkeypatch.delenv("CP_XCD_PIECE_DIV")
        cut = cp.plan_records(d, b.rows, 0)
        tiles = lambda r: sorted(map(tuple, r[r[:, 1] > 0].tolist()))
        dec = lambda r: sorted(map(tuple, r[r[:, 1] == -1].tolist()))
        assert tiles(whole) == tiles(cut), j
        assert dec(whole) == dec(cut), j
        lw, lc = _xcd_loads(whole), _xcd_loads(cut)
        assert lw.max() > 1.25 * lw.mean(), (j, lw)
        assert lc.max() < 0.8 * lw.max(), (j, lw, lc)
        _check_coverage(b)
    for j in (0, 15):
        d = cp.desc_for(batches[j])
        monkeypatch.setenv("CP_XCD_PIECE_DIV", "0")
        whole = cp.plan_records(d, batches[j].rows, 0)
        monkeypatch.delenv("CP_XCD_PIECE_DIV")
        assert np.array_equal(whole, cp.plan_records(d, batches[j].rows, 0)), j


def test_forced_xcd_pieces_keep_every_tile(monkeypatch):
    """Cutting every group (a negative tolerance: always; eighth-size pieces)
    on the other mixes moves tiles between XCDs but adds, drops and changes
    none."""
    monkeypatch.setenv("CP_XCD_BALANCE_TOL", "-1")
    monkeypatch.setenv("CP_XCD_PIECE_DIV", "8")
    cut = {(n, w): cp.plan_records(cp.desc_for(make_config(n)), make_config(n).rows, w)
           for n in (2, 3, 4) for w in (0, 1)}
    moved = 0
    monkeypatch.setenv("CP_XCD_PIECE_DIV", "0")
    for (n, w), recs in cut.items():
        whole = cp.plan_records(cp.desc_for(make_config(n)), make_config(n).rows, w)
        key = lambda r: sorted(map(tuple, r[r[:, 1] != 0].tolist()))
        assert key(whole) == key(recs), (n, w)
        moved += len(whole) != len(recs) or not np.array_equal(whole, recs)
    assert moved > 0
    monkeypatch.delenv("CP_XCD_PIECE_DIV")
    for n in (2, 3, 4):
        _check_coverage(make_config(n))


def test_shard_heads_divides_heads_and_keeps_rows():
    """`bench.py --shard N` runs one GPU's share: Hq/N and Hkv/N heads, the
    same rows, block tables and scale; N must divide the kv heads."""
    import bench
    batches, _ = replay_schedule()
    b = batches[3]
    for n in (1, 2, 4, 8):
        s = bench.shard_heads(b, n)
        assert (s.num_q_heads, s.num_kv_heads) == (b.num_q_heads // n, b.num_kv_heads // n)
        assert s.group == b.group and s.sm_scale == b.sm_scale and s.head_dim == b.head_dim
        assert np.array_equal(s.rows, b.rows) and np.array_equal(s.block_tables, b.block_tables)
    with pytest.raises(SystemExit):
        bench.shard_heads(make_config(1), 4)   # 2 kv heads


# ------------------------------------------------- the GPU fuzz cases, planned on the host

def test_gpu_fuzz_cases_plan_exactly(monkeypatch):
    """Every batch the GPU fuzz test runs, under the planner settings it runs
    it with, plans to an exact cover of its (token, kv head) key ranges."""
    from fuzz_cases import apply_settings, draw_case, draw_settings
    for seed in range(40):
        _check_coverage(draw_case(seed))
    for seed in range(24):
        env = draw_settings(seed)
        apply_settings(monkeypatch, env)
        _check_coverage(draw_case(100 + seed), int(env["CP_PREFILL_MIN_LEN"]))
