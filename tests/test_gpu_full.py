"""Full-size GPU parity: the benchmark's mixes in the benchmark's launch
configuration (the same cp_step_mixed call, the same plans), checked against
the fp64 oracle; the large-pool and long-context cases take the two calls.  Whole K/V pools are compared bit for bit after the append, and every
output element (all T x Hq x D of each mix and of each of the replay's 20
iterations) is compared with the oracle's; max and mean errors are printed
per mix and per iteration.
"""

import numpy as np
import pytest
import torch

import oracle
from gpu_util import assert_close, run_step, say, words
from workloads import Batch, make_batch, make_caches, make_config, make_step_tensors, make_tensors
from workloads import replay_schedule

pytestmark = pytest.mark.gpu


def check_all(batch, out_gpu, q_host, kc_ref, vc_ref, what):
    """Every output element against the oracle's."""
    ref = oracle.attn(batch, q_host, kc_ref, vc_ref)
    return assert_close(out_gpu, ref, f"{what} (all {ref.size} elements)")


@pytest.mark.parametrize("n", [2, 3, 4])
def test_full_size_mix(n):
    batch = make_config(n)
    say(f"[gpu] mix {n}: rows={batch.n_rows} T={batch.num_tokens} blocks={batch.num_blocks}")
    dev = torch.device("cuda", 0)
    t = make_tensors(batch, seed=7000 + n, device=dev)
    host = {k: v.cpu() for k, v in t.items() if k in ("q", "k_new", "v_new")}
    kc0, vc0 = words(t["k_cache"]), words(t["v_cache"])
    out = run_step(batch, t, one_call=True)
    torch.cuda.synchronize()
    kc_ref, vc_ref = oracle.kv_append(batch, host["k_new"], host["v_new"], kc0, vc0)
    del kc0, vc0
    assert np.array_equal(words(t["k_cache"]).reshape(-1), kc_ref.reshape(-1)), "K pool differs"
    assert np.array_equal(words(t["v_cache"]).reshape(-1), vc_ref.reshape(-1)), "V pool differs"
    check_all(batch, out, host["q"], kc_ref, vc_ref, f"mix {n}")


def test_replay_twenty_iterations_lockstep():
    batches, info = replay_schedule()
    dev = torch.device("cuda", 0)
    kc, vc = make_caches(batches[0], device=dev, fill_prior=False)
    kc_ref, vc_ref = words(kc), words(vc)
    for i, b in enumerate(batches):
        q, kn, vn, _ = make_step_tensors(b, 9000 + i, dev)
        t = {"q": q, "k_new": kn, "v_new": vn, "k_cache": kc, "v_cache": vc,
             "block_tables": torch.from_numpy(b.block_tables).to(dev)}
        say(f"[gpu] replay iteration {i}: rows={b.n_rows} T={b.num_tokens}")
        out = run_step(b, t, one_call=True)
        torch.cuda.synchronize()
        kc_ref, vc_ref = oracle.kv_append(b, kn.cpu(), vn.cpu(), kc_ref, vc_ref, inplace=True)
        check_all(b, out, q.cpu(), kc_ref, vc_ref, f"replay it {i}")
        if i in (0, 9, 19):
            assert np.array_equal(words(kc).reshape(-1), kc_ref.reshape(-1)), f"K pool it {i}"
            assert np.array_equal(words(vc).reshape(-1), vc_ref.reshape(-1)), f"V pool it {i}"


def test_block_ids_beyond_2g_elements():
    """Blocks whose element offset exceeds 2^31 (pool > 4 GiB per cache)."""
    hq, hkv, d, bsz = 32, 8, 128, 16
    per_block = hkv * bsz * d
    nb = (1 << 31) // per_block + 4096              # 135168 blocks, 4.4 GB per cache
    rows = [(3000, 200), (5000, 1), (777, 1), (0, 40)]
    rng = np.random.default_rng(21)
    need = [-(-(s + c) // bsz) for s, c in rows]
    ids = rng.permutation(np.arange(nb - 2048, nb - 1))[: sum(need)]  # beyond 2^31 elements
    assert ids.min() * per_block > (1 << 31)
    mbr = max(need)
    bt = np.full((len(rows), mbr), nb - 1, np.int32)
    k = 0
    rr = np.zeros((len(rows), 4), np.int32)
    for i, (s, c) in enumerate(rows):
        bt[i, : need[i]] = ids[k: k + need[i]]
        k += need[i]
        rr[i] = (i, s, c, s + c)
    big = Batch("bigpool", hq, hkv, d, bsz, rr, bt, nb, nb - 1)
    # the oracle sees the same data through a compact pool (block ids remapped)
    remap = {int(b): j for j, b in enumerate(ids)}
    bt_small = np.vectorize(lambda x: remap.get(int(x), 0))(bt).astype(np.int32)
    small = Batch("compact", hq, hkv, d, bsz, rr, bt_small, len(ids), 0)
    ref_t = make_tensors(small, seed=555)           # compact pool holds every referenced block
    dev = torch.device("cuda", 0)
    say(f"[gpu] big pool: {nb} blocks, max element offset {int(ids.max()) * per_block:.3e}")
    kc = torch.full((nb, hkv, bsz, d), float("nan"), dtype=torch.bfloat16, device=dev)
    vc = torch.full((nb, hkv, d, bsz), float("nan"), dtype=torch.bfloat16, device=dev)
    idx = torch.from_numpy(ids.astype(np.int64)).to(dev)
    kc[idx] = ref_t["k_cache"].to(dev)
    vc[idx] = ref_t["v_cache"].to(dev)
    t = {"q": ref_t["q"].to(dev), "k_new": ref_t["k_new"].to(dev), "v_new": ref_t["v_new"].to(dev),
         "k_cache": kc, "v_cache": vc, "block_tables": torch.from_numpy(bt).to(dev)}
    out = run_step(big, t)
    torch.cuda.synchronize()
    kc_ref, vc_ref = oracle.kv_append(small, ref_t["k_new"], ref_t["v_new"], ref_t["k_cache"],
                                      ref_t["v_cache"])
    assert np.array_equal(words(kc[idx]).reshape(-1), kc_ref.reshape(-1))
    assert np.array_equal(words(vc[idx]).reshape(-1), vc_ref.reshape(-1))
    assert bool(torch.isnan(kc[nb - 1].float()).all()), "poison block written"
    assert bool(torch.isnan(vc[nb - 1].float()).all()), "poison block written"
    ref = oracle.attn(small, ref_t["q"], kc_ref, vc_ref)
    assert_close(out, ref, "big pool")


def test_long_context_prefill_unsplit(monkeypatch):
    """A chunk over 70k cached keys with the planner told not to split key
    ranges: each prefill workgroup walks ~4400 blocks of one request."""
    monkeypatch.setenv("CP_PREFILL_MIN_SPLIT", "100000")
    rng = np.random.default_rng(21)
    batch = make_batch("long", 32, 8, 128, 16, [(70_000, 300), (3000, 1)], rng)
    say(f"[gpu] long context: rows={batch.n_rows} T={batch.num_tokens} blocks={batch.num_blocks}")
    dev = torch.device("cuda", 0)
    t = make_tensors(batch, seed=7100, device=dev)
    host = {k: v.cpu() for k, v in t.items() if k in ("q", "k_new", "v_new")}
    kc0, vc0 = words(t["k_cache"]), words(t["v_cache"])
    out = run_step(batch, t)
    torch.cuda.synchronize()
    kc_ref, vc_ref = oracle.kv_append(batch, host["k_new"], host["v_new"], kc0, vc0)
    del kc0, vc0
    assert np.array_equal(words(t["k_cache"]).reshape(-1), kc_ref.reshape(-1)), "K pool differs"
    assert np.array_equal(words(t["v_cache"]).reshape(-1), vc_ref.reshape(-1)), "V pool differs"
    check_all(batch, out, host["q"], kc_ref, vc_ref, "long context")


@pytest.mark.parametrize("shard", [8, 2])
def test_replay_head_shard_lockstep(shard):
    """One GPU's share of the replay under an N-way head shard (the shapes
    `bench.py --shard N` measures: 64/N q heads, 8/N kv heads, where few K/V
    groups make the planner cut them across XCDs), all 20 iterations in
    order through cp_step_mixed, every output element against the oracle."""
    import bench
    batches, _ = replay_schedule()
    batches = [bench.shard_heads(b, shard) for b in batches]
    dev = torch.device("cuda", 0)
    kc, vc = make_caches(batches[0], device=dev, fill_prior=False)
    kc_ref, vc_ref = words(kc), words(vc)
    for i, b in enumerate(batches):
        q, kn, vn, _ = make_step_tensors(b, 9500 + i, dev)
        t = {"q": q, "k_new": kn, "v_new": vn, "k_cache": kc, "v_cache": vc,
             "block_tables": torch.from_numpy(b.block_tables).to(dev)}
        say(f"[gpu] replay shard {shard} iteration {i}: rows={b.n_rows} T={b.num_tokens}")
        out = run_step(b, t, one_call=True)
        torch.cuda.synchronize()
        kc_ref, vc_ref = oracle.kv_append(b, kn.cpu(), vn.cpu(), kc_ref, vc_ref, inplace=True)
        check_all(b, out, q.cpu(), kc_ref, vc_ref, f"replay shard {shard} it {i}")
    assert np.array_equal(words(kc).reshape(-1), kc_ref.reshape(-1))
    assert np.array_equal(words(vc).reshape(-1), vc_ref.reshape(-1))


@pytest.mark.parametrize("geom", [(32, 32, 64, 16), (16, 8, 128, 16), (32, 16, 64, 32)],
                         ids=lambda g: "hq%d_hkv%d_d%d_b%d" % g)
def test_replay_other_geometries_lockstep(geom):
    """The 20-iteration replay at other head counts, head sizes and block
    sizes (G = 1 with D = 64 and B = 16, G = 2 with B = 16, G = 2 with D = 64
    and B = 32), all iterations in order through cp_step_mixed, every output
    element against the oracle: the fused launches, key splits and XCD
    dealing at full length for geometries the benchmark's mixes do not use."""
    hq, hkv, d, bsz = geom
    batches, _ = replay_schedule(hq=hq, hkv=hkv, d=d, bsz=bsz)
    dev = torch.device("cuda", 0)
    kc, vc = make_caches(batches[0], device=dev, fill_prior=False)
    kc_ref, vc_ref = words(kc), words(vc)
    for i, b in enumerate(batches):
        q, kn, vn, _ = make_step_tensors(b, 9700 + i, dev)
        t = {"q": q, "k_new": kn, "v_new": vn, "k_cache": kc, "v_cache": vc,
             "block_tables": torch.from_numpy(b.block_tables).to(dev)}
        say(f"[gpu] replay {geom} iteration {i}: rows={b.n_rows} T={b.num_tokens}")
        out = run_step(b, t, one_call=True)
        torch.cuda.synchronize()
        kc_ref, vc_ref = oracle.kv_append(b, kn.cpu(), vn.cpu(), kc_ref, vc_ref, inplace=True)
        check_all(b, out, q.cpu(), kc_ref, vc_ref, f"replay {geom} it {i}")
    assert np.array_equal(words(kc).reshape(-1), kc_ref.reshape(-1))
    assert np.array_equal(words(vc).reshape(-1), vc_ref.reshape(-1))
