"""GPU parity of the HIP path (through the C ABI) against the fp64 oracle.

Small batches compare every output element and the whole K/V pools; the
bar is max |gpu - oracle| <= 2e-2 and mean <= 2e-3 on bf16 outputs, caches
bit-exact.  Cache slots a correct step never reads hold bf16 NaN, so any
read past a row's context or into an unreferenced block shows up.
"""

import numpy as np
import pytest
import torch

import oracle
from gpu_util import assert_close, run_step, say, to_dev, words
from workloads import Batch, make_batch, make_config, make_tensors, replay_schedule

pytestmark = pytest.mark.gpu


def _full_check(batch, seed, what):
    tens = make_tensors(batch, seed=seed)
    say(f"[gpu] {what}: rows={batch.n_rows} T={batch.num_tokens} "
        f"heads={batch.num_q_heads}/{batch.num_kv_heads} D={batch.head_dim} B={batch.block_size}")
    kc_ref, vc_ref = oracle.kv_append(batch, tens["k_new"], tens["v_new"], tens["k_cache"],
                                      tens["v_cache"])
    ref = oracle.attn(batch, tens["q"], kc_ref, vc_ref)
    t = to_dev(tens)
    out = run_step(batch, t)
    torch.cuda.synchronize()
    assert np.array_equal(words(t["k_cache"]).reshape(-1), kc_ref.reshape(-1)), "K cache differs"
    assert np.array_equal(words(t["v_cache"]).reshape(-1), vc_ref.reshape(-1)), "V cache differs"
    if batch.num_tokens:
        assert_close(out, ref, what)
    return out, ref


def test_config1_tiny_mix():
    _full_check(make_config(1), 1001, "config 1")


GEOMS = [(hq, hkv, d, b) for d in (64, 128) for b in (16, 32)
         for hq, hkv in ((4, 4), (8, 4), (8, 2), (16, 2))]


@pytest.mark.parametrize("tiles", ["planned", "wide"])
@pytest.mark.parametrize("geom", GEOMS, ids=lambda g: "hq%d_hkv%d_d%d_b%d" % g)
def test_geometry_grid(monkeypatch, geom, tiles):
    """Every supported (D, B, G); with tiles="wide" every chunk of more than
    128 rows runs on the 256-row tiles whatever the step's key range."""
    if tiles == "wide":
        monkeypatch.setenv("CP_PREFILL_WIDE_MIN_KEYS", "0")
        monkeypatch.setenv("CP_FUSE_NARROW", "0")   # wide tiles beside the decode rows too
    hq, hkv, d, b = geom
    rng = np.random.default_rng(hash(geom) % (2 ** 31))
    # a multi-tile chunk with a ragged tail, a chunk over deep context, a
    # two-token chunk, decode rows at block edges, ctx 1
    rows = [(0, 150), (300, 77), (5, 2), (b - 1, 1), (2 * b, 1), (0, 1), (257, 1), (1000, 1)]
    batch = make_batch("grid", hq, hkv, d, b, rows, rng)
    _full_check(batch, 2000 + len(str(geom)), f"grid {geom}")


def test_rows_in_any_order_and_zero_length_rows():
    rng = np.random.default_rng(7)
    rows = [(10, 40), (0, 0), (63, 1), (200, 0), (128, 130), (31, 1)]
    batch = make_batch("zeros", 32, 8, 128, 16, rows, rng)
    _full_check(batch, 3001, "zero-length rows")


@pytest.mark.parametrize("min_len", [4, 16, 64])
def test_few_token_rows_on_the_decode_kernel(monkeypatch, min_len):
    """Rows shorter than CP_PREFILL_MIN_LEN run on the decode kernel token by
    token, each token over keys up to its own position; output and pools as
    with the default routing (the oracle's)."""
    monkeypatch.setenv("CP_PREFILL_MIN_LEN", str(min_len))
    rng = np.random.default_rng(min_len)
    rows = [(0, 2), (5, 3), (100, 2), (4000, 7), (31, 15), (16, 16), (999, 1), (0, 1),
            (2047, 40), (3, 0), (1500, 63), (777, 64)]
    for hq, hkv, d, b in ((32, 8, 128, 16), (64, 8, 128, 32), (8, 8, 64, 16)):
        batch = make_batch("few", hq, hkv, d, b, rows, rng)
        _full_check(batch, 3100 + min_len + hq, f"few-token rows min_len={min_len} {(hq, hkv, d, b)}")


def test_empty_batch_is_noop():
    batch = make_batch("empty", 8, 2, 128, 16, [(5, 0)], np.random.default_rng(1))
    _full_check(batch, 3002, "empty batch")


def test_single_token_chunks_and_tiny_prefill():
    """Chunk sizes the scheduler's minimum-progress rule produces (1..8 tokens)."""
    rng = np.random.default_rng(8)
    rows = [(100, c) for c in (1, 2, 3, 5, 8)] + [(0, 2), (17, 3)]
    batch = make_batch("tiny-chunks", 32, 8, 128, 16, rows, rng)
    _full_check(batch, 3003, "tiny chunks")


def test_prepared_plan_runs_match_attn_mixed_bit_for_bit():
    # Prefill chunks long enough to be split and merged, plus decode rows with
    # split contexts: one plan, run for two "layers" (different q and pools).
    import paper_2606_09061_amd as cp
    rng = np.random.default_rng(17)
    rows = [(3000, 96), (0, 130), (8000, 1), (5000, 1), (300, 1), (12000, 40)]
    batch = make_batch("plan", 32, 8, 128, 16, rows, rng)
    d = cp.desc_for(batch)
    say(f"[gpu] prepared plan: rows={batch.n_rows} T={batch.num_tokens}")
    layers = [to_dev(make_tensors(batch, seed=s)) for s in (5101, 5102)]
    ws_a = torch.empty(cp.workspace_bytes(d, batch.rows), dtype=torch.uint8, device="cuda")
    ws_b = torch.empty_like(ws_a)
    outs_ref, outs_plan = [], []
    for t in layers:
        cp.kv_append(d, t["k_new"], t["v_new"], t["k_cache"], t["v_cache"], t["block_tables"],
                     batch.rows, ws_a)
        o = torch.empty(batch.num_tokens, 32, 128, dtype=torch.bfloat16, device="cuda")
        cp.attn_mixed(d, t["q"], t["k_cache"], t["v_cache"], t["block_tables"], batch.rows, o, ws_a)
        outs_ref.append(o)
    plan = cp.attn_prepare(d, batch.rows, ws_b)
    assert plan.tokens == batch.num_tokens and plan.n_merge > 0
    for t in layers:
        o = torch.empty(batch.num_tokens, 32, 128, dtype=torch.bfloat16, device="cuda")
        cp.attn_run(plan, t["q"], t["k_cache"], t["v_cache"], t["block_tables"], o, ws_b)
        outs_plan.append(o)
    torch.cuda.synchronize()
    for a, b in zip(outs_ref, outs_plan):
        assert torch.equal(a, b)
    with pytest.raises(cp.CpError):   # a workspace smaller than the plan's
        cp.attn_run(plan, layers[0]["q"], layers[0]["k_cache"], layers[0]["v_cache"],
                    layers[0]["block_tables"], outs_plan[0], ws_b[:256])


@pytest.mark.parametrize("fuse", ["4", "0"])
def test_prepared_plan_replays_in_a_hip_graph(monkeypatch, fuse):
    """cp_attn_run only enqueues kernels, so a caller can capture it in a HIP
    graph (the layers of a model iteration share one plan).  Each replay, with
    new q written into the captured buffer between replays and eager work and
    synchronisations around it, equals an eager run bit for bit, and the last
    equals the oracle.  fuse "4": decode rows inside the prefill launch, then
    the merge; "0": prefill, decode and merge launches."""
    import paper_2606_09061_amd as cp
    monkeypatch.setenv("CP_FUSE_DECODE", fuse)
    rng = np.random.default_rng(19)
    rows = [(3000, 96), (0, 130), (8000, 1), (5000, 1), (300, 1), (12000, 40)]
    batch = make_batch("graph", 32, 8, 128, 16, rows, rng)
    d = cp.desc_for(batch)
    say(f"[gpu] graph replay, CP_FUSE_DECODE={fuse}: rows={batch.n_rows} T={batch.num_tokens}")
    tens = make_tensors(batch, seed=5201)
    t = to_dev(tens)
    ws_app = torch.empty(cp.workspace_bytes(d, batch.rows), dtype=torch.uint8, device="cuda")
    cp.kv_append(d, t["k_new"], t["v_new"], t["k_cache"], t["v_cache"], t["block_tables"],
                 batch.rows, ws_app)
    ws = torch.empty_like(ws_app)
    plan = cp.attn_prepare(d, batch.rows, ws)
    assert plan.n_merge > 0 and plan.n_decode > 0
    assert plan.decode_in_prefill == (0 if fuse == "0" else 1)
    shape = (batch.num_tokens, 32, 128)
    out_e = torch.empty(shape, dtype=torch.bfloat16, device="cuda")
    out_g = torch.empty(shape, dtype=torch.bfloat16, device="cuda")
    run = lambda o: cp.attn_run(plan, t["q"], t["k_cache"], t["v_cache"], t["block_tables"], o, ws)
    run(out_e)  # first use of the kernels outside the capture
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        run(out_g)
    gen = torch.Generator().manual_seed(5202)
    for r in range(4):
        q_new = torch.randn(shape, generator=gen).to(torch.bfloat16)
        t["q"].copy_(q_new.to("cuda"))
        out_g.fill_(float("nan"))  # a replay must write every element
        g.replay()
        torch.cuda.synchronize()
        run(out_e)
        torch.cuda.synchronize()
        assert torch.equal(out_g, out_e), f"replay {r} differs from the eager run"
    kc_ref, vc_ref = oracle.kv_append(batch, tens["k_new"], tens["v_new"], tens["k_cache"],
                                      tens["v_cache"])
    ref = oracle.attn(batch, q_new, kc_ref, vc_ref)
    assert_close(out_g, ref, f"graph replay (CP_FUSE_DECODE={fuse})")


def test_debug_mode_rejects_out_of_range_block_ids(monkeypatch):
    """CP_DEBUG=1: a table entry outside [0, num_blocks) is found on the host
    before anything is enqueued.  The pools hold 4 blocks past the num_blocks
    the descriptor declares, and the bad entry points at one of them, so the
    memory it names exists either way."""
    import paper_2606_09061_amd as cp
    rng = np.random.default_rng(31)
    batch = make_batch("debug", 8, 2, 64, 16, [(40, 24), (70, 1)], rng)
    tens = to_dev(make_tensors(batch, seed=3201))
    for k in ("k_cache", "v_cache"):   # 4 NaN blocks past the declared pool
        pad = torch.full((4,) + tuple(tens[k].shape[1:]), float("nan"), dtype=torch.bfloat16,
                         device="cuda")
        tens[k] = torch.cat([tens[k], pad]).contiguous()
    d = cp.desc_for(batch)
    assert d.num_blocks == batch.num_blocks
    req, s, c, ctx = (int(x) for x in batch.rows[0])
    bt = tens["block_tables"].clone()
    bt[req, 1] = batch.num_blocks + 1              # declared out of range, allocated
    ws = torch.empty(cp.workspace_bytes(d, batch.rows), dtype=torch.uint8, device="cuda")
    out = torch.zeros(batch.num_tokens, 8, 64, dtype=torch.bfloat16, device="cuda")
    kc0, vc0 = tens["k_cache"].clone(), tens["v_cache"].clone()
    monkeypatch.setenv("CP_DEBUG", "1")
    say("[gpu] CP_DEBUG table check")
    with pytest.raises(cp.CpError) as e:
        cp.kv_append(d, tens["k_new"], tens["v_new"], tens["k_cache"], tens["v_cache"], bt,
                     batch.rows, ws)
    assert e.value.code == -2
    with pytest.raises(cp.CpError) as e:
        cp.attn_mixed(d, tens["q"], tens["k_cache"], tens["v_cache"], bt, batch.rows, out, ws)
    assert e.value.code == -2
    torch.cuda.synchronize()
    assert torch.equal(out, torch.zeros_like(out)), "output written after a refused call"
    assert np.array_equal(words(tens["k_cache"]), words(kc0)) and np.array_equal(
        words(tens["v_cache"]), words(vc0)), "pools written after a refused call"
    # the intact table passes the same checks and the step matches the oracle
    kc_ref, vc_ref = oracle.kv_append(batch, tens["k_new"].cpu(), tens["v_new"].cpu(),
                                      words(tens["k_cache"])[: batch.num_blocks],
                                      words(tens["v_cache"])[: batch.num_blocks])
    cp.kv_append(d, tens["k_new"], tens["v_new"], tens["k_cache"], tens["v_cache"],
                 tens["block_tables"], batch.rows, ws)
    cp.attn_mixed(d, tens["q"], tens["k_cache"], tens["v_cache"], tens["block_tables"],
                  batch.rows, out, ws)
    torch.cuda.synchronize()
    assert_close(out, oracle.attn(batch, tens["q"].cpu(), kc_ref, vc_ref), "CP_DEBUG run")


FUSE_GEOMS = [(8, 1, 128, 16), (32, 8, 128, 16), (64, 8, 128, 32), (16, 4, 64, 32), (8, 8, 64, 16)]


@pytest.mark.parametrize("width", ["narrow", "wide"])
@pytest.mark.parametrize("geom", FUSE_GEOMS, ids=lambda g: "hq%d_hkv%d_d%d_b%d" % g)
def test_decode_inside_the_prefill_launch(monkeypatch, geom, width):
    """Decode rows run as decode blocks of the prefill launch (CP_FUSE_DECODE
    1, 2, 3, 4: after, before, spread among or merged longest first with the
    tiles; 4-wave workgroups with one unit,
    8-wave ones with two, an odd unit count leaving one group idle) or in
    their own launch (0): every mode matches the oracle element by element and
    gives the same output bits as the others (the decode and prefill splits
    are pinned: fused, a step otherwise splits both differently)."""
    monkeypatch.setenv("CP_DECODE_TARGET_ITEMS", "300")
    monkeypatch.setenv("CP_PREFILL_TARGET_ITEMS", "400")
    hq, hkv, d, b = geom
    G = hq // hkv
    if width == "wide":
        monkeypatch.setenv("CP_PREFILL_WIDE_MIN_KEYS", "0")
        monkeypatch.setenv("CP_FUSE_NARROW", "0")
        chunk = max(160 // G + 1, 129)       # every chunk above 128 rows
        rows = [(3000, chunk), (0, 2 * chunk)]
    else:
        monkeypatch.setenv("CP_PREFILL_WIDE_MIN_ROWS", "100000")
        rows = [(3000, 60), (0, 150), (40, 2)]
    rows += [(b - 1, 1), (2 * b, 1), (0, 1), (6000, 1), (1000, 1)]
    rng = np.random.default_rng(hq * 100 + d + b)
    batch = make_batch("fuse-" + width, hq, hkv, d, b, rows, rng)
    tens = make_tensors(batch, seed=4000 + hq + d)
    kc_ref, vc_ref = oracle.kv_append(batch, tens["k_new"], tens["v_new"], tens["k_cache"],
                                      tens["v_cache"])
    ref = oracle.attn(batch, tens["q"], kc_ref, vc_ref)
    outs = {}
    for mode in (0, 1, 2, 3, 4):
        monkeypatch.setenv("CP_FUSE_DECODE", str(mode))
        import paper_2606_09061_amd as cp
        recs = cp.plan_records(cp.desc_for(batch), batch.rows, 1 if width == "wide" else 0)
        n_blocks = int((recs[:, 1] == -1).sum())
        assert (n_blocks > 0) == (mode > 0)
        say(f"[gpu] decode in prefill launch {width} {geom} mode {mode}: {n_blocks} decode blocks")
        t = to_dev(tens)
        out = run_step(batch, t)
        torch.cuda.synchronize()
        assert np.array_equal(words(t["k_cache"]).reshape(-1), kc_ref.reshape(-1))
        assert_close(out, ref, f"fuse {width} {geom} mode {mode}")
        outs[mode] = words(out)
    for mode in (1, 2, 3, 4):
        assert np.array_equal(outs[mode], outs[0]), f"mode {mode} differs from its own launch"


def _step_batches():
    rng = np.random.default_rng(77)
    yield "tiny", make_config(1)
    yield "ragged-70b", make_batch("step", 64, 8, 128, 32,
                                   [(3000, 60), (0, 150), (40, 2), (31, 1), (64, 1), (0, 1),
                                    (6000, 1)], rng)
    # more than 200 spans: the long span list is uploaded and the two calls run in turn
    yield "many-spans", make_batch("spans", 32, 8, 128, 16,
                                   [(int(c), 1) for c in rng.integers(0, 3000, 230)] +
                                   [(100, 40)], rng)


@pytest.mark.parametrize("which", ["tiny", "ragged-70b", "many-spans"])
def test_step_matches_append_then_attention(which):
    """cp_step_mixed (the plan copy inside the append launch) writes the same
    pools and the same output bits as cp_kv_append then cp_attn_mixed, and
    matches the oracle; two steps in a row reuse the staging slots."""
    import paper_2606_09061_amd as cp
    batch = dict(_step_batches())[which]
    tens = make_tensors(batch, seed=8800 + len(which))
    say(f"[gpu] step {which}: rows={batch.n_rows} T={batch.num_tokens}")
    kc_ref, vc_ref = oracle.kv_append(batch, tens["k_new"], tens["v_new"], tens["k_cache"],
                                      tens["v_cache"])
    ref = oracle.attn(batch, tens["q"], kc_ref, vc_ref)
    d = cp.desc_for(batch)
    a, b = to_dev(tens), to_dev(tens)
    ws_a = torch.empty(cp.workspace_bytes(d, batch.rows), dtype=torch.uint8, device="cuda")
    ws_b = torch.empty_like(ws_a)
    outs = []
    for t, ws, one_call in ((a, ws_a, False), (b, ws_b, True)):
        out = torch.empty(batch.num_tokens, batch.num_q_heads, batch.head_dim,
                          dtype=torch.bfloat16, device="cuda")
        for _ in range(2):   # the second pass appends the same tokens again (same bits)
            if one_call:
                cp.step_mixed(d, t["q"], t["k_new"], t["v_new"], t["k_cache"], t["v_cache"],
                              t["block_tables"], batch.rows, out, ws)
            else:
                cp.kv_append(d, t["k_new"], t["v_new"], t["k_cache"], t["v_cache"],
                             t["block_tables"], batch.rows, ws)
                cp.attn_mixed(d, t["q"], t["k_cache"], t["v_cache"], t["block_tables"],
                              batch.rows, out, ws)
        outs.append(out)
    torch.cuda.synchronize()
    assert np.array_equal(words(b["k_cache"]).reshape(-1), kc_ref.reshape(-1))
    assert np.array_equal(words(b["v_cache"]).reshape(-1), vc_ref.reshape(-1))
    assert np.array_equal(words(outs[0]), words(outs[1])), "step differs from the two calls"
    assert_close(outs[1], ref, f"step {which}")


@pytest.mark.parametrize("it,shard", [(9, 8), (4, 4), (0, 8)])
def test_xcd_pieces_change_no_output_bit(monkeypatch, it, shard):
    """A head-sharded replay iteration (1 or 2 kv heads) has too few K/V groups
    to balance the XCDs whole, so the planner cuts them into runs of tiles:
    the output matches the oracle element by element and equals the uncut
    layout's bit for bit (workgroups move, no work changes)."""
    import bench
    batches, _ = replay_schedule()
    batch = bench.shard_heads(batches[it], shard)
    tens = make_tensors(batch, seed=4400 + it)
    kc_ref, vc_ref = oracle.kv_append(batch, tens["k_new"], tens["v_new"], tens["k_cache"],
                                      tens["v_cache"])
    ref = oracle.attn(batch, tens["q"], kc_ref, vc_ref)
    outs = {}
    for div in ("0", "4"):
        monkeypatch.setenv("CP_XCD_PIECE_DIV", div)
        say(f"[gpu] replay it {it} shard {shard}: CP_XCD_PIECE_DIV={div}")
        t = to_dev(tens)
        out = run_step(batch, t, one_call=True)
        torch.cuda.synchronize()
        assert np.array_equal(words(t["k_cache"]).reshape(-1), kc_ref.reshape(-1))
        assert_close(out, ref, f"replay it {it} shard {shard} div {div}")
        outs[div] = words(out)
    assert np.array_equal(outs["0"], outs["4"])
