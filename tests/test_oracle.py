"""Pins of the fp64 oracle against things other than itself.

* a hand-derived worked example (tests/golden/two_key_worked_example.json);
* a dense-matrix brute force (oracle/dense.py) and torch's SDPA in float64
  with an explicit boolean mask (a library routine), on tiny batches;
* closed forms: ctx 1 returns V_0; q = 0 or equal keys give the mean of V;
  a dominant key returns its V;
* exact fp64 invariants: chunked == unchunked prefill, a decode row equals the
  last row of a full prefill, block-table permutation, row order, GQA
  replication and batch independence;
* the append: gather(append(x)) == x bit for bit, other slots untouched;
* mutation checks: plausible mistakes planted in a copy of the oracle source
  (on the CPU) must each fail at least one of these pins.
"""

import json
import math
import os

import numpy as np
import pytest
import torch

import oracle
from oracle import dense
from workloads import Batch, make_batch, make_config, make_tensors, replay_schedule

HERE = os.path.dirname(os.path.abspath(__file__))


def bits(x):
    """float array -> bf16 words (RNE)."""
    t = torch.as_tensor(np.asarray(x, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def words(t):
    return t.contiguous().view(torch.int16).numpy().view(np.uint16)


def run_step(batch, tens, lib=None):
    """oracle append then attention; returns (out, kc, vc)."""
    kc, vc = oracle.kv_append(batch, tens["k_new"], tens["v_new"], tens["k_cache"],
                              tens["v_cache"], lib=lib)
    out = oracle.attn(batch, tens["q"], kc, vc, lib=lib)
    return out, kc, vc


def random_batch(rng, hq, hkv, d, bsz, starts_lens, n_spare=3):
    return make_batch("rand", hq, hkv, d, bsz, starts_lens, rng, n_spare=n_spare)


# ---------------------------------------------------------------- worked example

def _golden_batch():
    g = json.load(open(os.path.join(HERE, "golden", "two_key_worked_example.json")))
    geo = g["geometry"]
    keys = np.array(g["keys"])
    vals = np.array(g["values"])
    qv = np.array(g["query"])
    # one request, the three keys already cached at positions 0..2; three
    # separate single-token rows query positions 0, 1, 2 (three requests that
    # share identical pages through their block tables)
    B = geo["B"]
    nb = 2
    kc = np.zeros((nb, 1, B, 2), np.float32)
    vc = np.zeros((nb, 1, 2, B), np.float32)
    for p in range(3):
        kc[p // B, 0, p % B] = keys[p]
        vc[p // B, 0, :, p % B] = vals[p]
    bt = np.array([[0, 1], [0, 1], [0, 1]], np.int32)
    rows = np.array([[0, 0, 1, 1], [1, 1, 1, 2], [2, 2, 1, 3]], np.int32)
    batch = Batch("golden", 1, 1, 2, B, rows, bt, nb, 1, sm_scale=geo["sm_scale"])
    q = np.tile(qv, (3, 1, 1))
    return g, batch, bits(q), bits(kc), bits(vc)


def test_golden_worked_example():
    g, batch, q, kc, vc = _golden_batch()
    out = oracle.attn(batch, q, kc, vc)
    e = math.e
    for pos, exprs in g["expected_by_position"].items():
        want = [eval(x, {"e": e}) for x in exprs]
        np.testing.assert_allclose(out[int(pos), 0], want, rtol=0, atol=1e-15)


# ---------------------------------------------------------------- brute force

def _tiny_cases():
    yield make_config(1)
    rng = np.random.default_rng(11)
    yield random_batch(rng, 8, 2, 64, 16, [(0, 33), (17, 5), (40, 1), (0, 1), (63, 2)])
    yield random_batch(rng, 4, 4, 128, 32, [(31, 1), (5, 40), (0, 64)])
    yield random_batch(rng, 8, 1, 64, 16, [(100, 9), (0, 1), (15, 1), (16, 1)])


@pytest.mark.parametrize("case", range(4))
def test_oracle_vs_dense_bruteforce(case):
    batch = list(_tiny_cases())[case]
    tens = make_tensors(batch, seed=100 + case)
    out, kc, vc = run_step(batch, tens)
    ref = dense.dense_attention(batch, words(tens["q"]), kc, vc)
    assert np.isfinite(out).all()
    np.testing.assert_allclose(out, ref, rtol=0, atol=1e-12)


@pytest.mark.parametrize("case", range(4))
def test_oracle_vs_torch_sdpa_float64(case):
    batch = list(_tiny_cases())[case]
    tens = make_tensors(batch, seed=200 + case)
    out, kc, vc = run_step(batch, tens)
    kcf = dense.bf16_to_f64(kc).reshape(batch.num_blocks, batch.num_kv_heads,
                                       batch.block_size, batch.head_dim)
    vcf = dense.bf16_to_f64(vc).reshape(batch.num_blocks, batch.num_kv_heads,
                                       batch.head_dim, batch.block_size)
    q = tens["q"].to(torch.float64)
    G = batch.group
    off = 0
    for req, s, c, ctx in batch.rows.tolist():
        K, V = dense.gather_kv(kcf, vcf, batch.block_tables[req], ctx, batch.block_size)
        K = torch.from_numpy(np.ascontiguousarray(K)).permute(1, 0, 2)  # [Hkv, ctx, D]
        V = torch.from_numpy(np.ascontiguousarray(V)).permute(1, 0, 2)
        K = K.repeat_interleave(G, dim=0)
        V = V.repeat_interleave(G, dim=0)
        Q = q[off: off + c].permute(1, 0, 2)                             # [Hq, c, D]
        mask = torch.arange(ctx)[None, :] <= (s + torch.arange(c))[:, None]
        ref = torch.nn.functional.scaled_dot_product_attention(
            Q, K, V, attn_mask=mask, scale=float(np.float32(batch.sm_scale)))
        np.testing.assert_allclose(out[off: off + c], ref.permute(1, 0, 2).numpy(),
                                   rtol=0, atol=1e-12)
        off += c


# ---------------------------------------------------------------- closed forms

def _single_request(hq, hkv, d, bsz, ctx, q, K, V, start, length, scale=None):
    """Batch with one request whose keys 0..ctx-1 are given as float arrays
    [ctx, Hkv, D]; the row is (start, length)."""
    nb = -(-ctx // bsz)
    kc = np.full((nb, hkv, bsz, d), np.nan, np.float32)
    vc = np.full((nb, hkv, d, bsz), np.nan, np.float32)
    for p in range(ctx):
        kc[p // bsz, :, p % bsz, :] = K[p]
        vc[p // bsz, :, :, p % bsz] = V[p]
    bt = np.arange(nb, dtype=np.int32)[None, :]
    rows = np.array([[0, start, length, start + length]], np.int32)
    b = Batch("single", hq, hkv, d, bsz, rows, bt, nb, 0, sm_scale=scale or 0.0)
    return b, bits(q), bits(kc), bits(vc)


def test_ctx_one_returns_v0():
    rng = np.random.default_rng(3)
    K = rng.standard_normal((1, 2, 64))
    V = rng.standard_normal((1, 2, 64))
    q = rng.standard_normal((1, 4, 64))
    b, qw, kc, vc = _single_request(4, 2, 64, 16, 1, q, K, V, 0, 1)
    out = oracle.attn(b, qw, kc, vc)
    vb = dense.bf16_to_f64(bits(V))
    for h in range(4):
        assert np.array_equal(out[0, h], vb[0, h // 2])


@pytest.mark.parametrize("mode", ["zero_q", "equal_keys"])
def test_uniform_weights_give_mean_of_v(mode):
    rng = np.random.default_rng(4)
    ctx = 45
    V = rng.standard_normal((ctx, 2, 64))
    if mode == "zero_q":
        K = rng.standard_normal((ctx, 2, 64))
        q = np.zeros((12, 4, 64))
    else:
        K = np.tile(rng.standard_normal((1, 2, 64)), (ctx, 1, 1))
        q = rng.standard_normal((12, 4, 64))
    b, qw, kc, vc = _single_request(4, 2, 64, 16, ctx, q, K, V, ctx - 12, 12)
    out = oracle.attn(b, qw, kc, vc)
    vb = dense.bf16_to_f64(bits(V))
    for j in range(12):
        p = ctx - 12 + j
        for h in range(4):
            np.testing.assert_allclose(out[j, h], vb[: p + 1, h // 2].mean(axis=0),
                                       rtol=0, atol=1e-13)


def test_dominant_key_returns_its_value():
    rng = np.random.default_rng(5)
    ctx, d = 20, 64
    qv = np.zeros(d)
    qv[:4] = 8.0
    K = np.zeros((ctx, 1, d))
    K[7, 0, :4] = 8.0  # score 256 * scale = 32 above every other key
    V = rng.standard_normal((ctx, 1, d))
    b, qw, kc, vc = _single_request(1, 1, d, 16, ctx, qv[None, None, :], K, V, ctx - 1, 1)
    out = oracle.attn(b, qw, kc, vc)
    vb = dense.bf16_to_f64(bits(V))
    np.testing.assert_allclose(out[0, 0], vb[7, 0], rtol=0, atol=1e-12)


# ---------------------------------------------------------------- invariants

def _prompt_pages(rng, hkv, d, bsz, n):
    return rng.standard_normal((n, hkv, d)), rng.standard_normal((n, hkv, d))


def test_chunked_equals_unchunked_exactly():
    """A prompt processed in chunks gives, token for token, exactly the fp64
    output of processing it in one chunk (each chunk appended before it attends)."""
    rng = np.random.default_rng(6)
    hq, hkv, d, bsz, n = 8, 2, 64, 16, 77
    Kf, Vf = _prompt_pages(rng, hkv, d, bsz, n)
    qf = rng.standard_normal((n, hq, d))
    nb = -(-n // bsz)
    perm = rng.permutation(nb + 2).astype(np.int32)
    bt = perm[None, :nb]
    kc0 = bits(np.full((nb + 2, hkv, bsz, d), np.nan))
    vc0 = bits(np.full((nb + 2, hkv, d, bsz), np.nan))
    kn, vn, qw = bits(Kf), bits(Vf), bits(qf)

    def run(chunks):
        kc, vc = kc0, vc0
        outs = []
        for s, c in chunks:
            b = Batch("p", hq, hkv, d, bsz, np.array([[0, s, c, s + c]]), bt, nb + 2, int(perm[nb]))
            kc, vc = oracle.kv_append(b, kn[s: s + c], vn[s: s + c], kc, vc)
            outs.append(oracle.attn(b, qw[s: s + c], kc, vc))
        return np.concatenate(outs), kc, vc

    full, kc_full, vc_full = run([(0, n)])
    for cuts in ([(0, 1), (1, 30), (31, 46)], [(i, 1) for i in range(n)], [(0, 16), (16, 61)]):
        got, kc, vc = run(cuts)
        assert np.array_equal(got, full)
        assert np.array_equal(kc, kc_full) and np.array_equal(vc, vc_full)


def test_decode_row_equals_last_prefill_row():
    rng = np.random.default_rng(7)
    hq, hkv, d, bsz, n = 4, 1, 128, 32, 70
    Kf, Vf = _prompt_pages(rng, hkv, d, bsz, n)
    qf = rng.standard_normal((n, hq, d))
    b, qw, kc, vc = _single_request(hq, hkv, d, bsz, n, qf, Kf, Vf, 0, n)
    full = oracle.attn(b, qw, kc, vc)
    for p in (0, 31, 32, 69):
        bd = Batch("d", hq, hkv, d, bsz, np.array([[0, p, 1, p + 1]]), b.block_tables,
                   b.num_blocks, 0)
        dec = oracle.attn(bd, qw[p: p + 1], kc, vc)
        assert np.array_equal(dec[0], full[p])


def _permute_pool(batch, kc, vc, perm):
    """Moves physical block b to perm[b] and rewrites the tables to match."""
    nb = batch.num_blocks
    kc2 = np.empty_like(kc).reshape(nb, -1)
    vc2 = np.empty_like(vc).reshape(nb, -1)
    kc2[perm] = kc.reshape(nb, -1)
    vc2[perm] = vc.reshape(nb, -1)
    bt = perm[batch.block_tables].astype(np.int32)
    b2 = Batch(batch.name, batch.num_q_heads, batch.num_kv_heads, batch.head_dim,
               batch.block_size, batch.rows, bt, nb, int(perm[batch.poison_block]),
               sm_scale=batch.sm_scale)
    return b2, kc2.reshape(-1), vc2.reshape(-1)


def test_block_table_permutation_invariance():
    batch = make_config(1)
    tens = make_tensors(batch, seed=8)
    out, kc, vc = run_step(batch, tens)
    perm = np.random.default_rng(8).permutation(batch.num_blocks)
    b2, kc2, vc2 = _permute_pool(batch, kc, vc, perm)
    out2 = oracle.attn(b2, tens["q"], kc2, vc2)
    assert np.array_equal(out, out2)


def test_row_order_and_batch_independence():
    batch = make_config(1)
    tens = make_tensors(batch, seed=9)
    out, kc, vc = run_step(batch, tens)
    off = batch.tok_offsets()
    q = words(tens["q"])
    order = [2, 0, 3, 1]
    rows2 = batch.rows[order]
    q2 = np.concatenate([q[off[r]: off[r + 1]] for r in order])
    b2 = Batch("reord", 4, 2, 64, 16, rows2, batch.block_tables, batch.num_blocks,
               batch.poison_block)
    out2 = oracle.attn(b2, q2, kc, vc)
    want = np.concatenate([out[off[r]: off[r + 1]] for r in order])
    assert np.array_equal(out2, want)
    for r in range(batch.n_rows):
        b1 = Batch("one", 4, 2, 64, 16, batch.rows[r: r + 1], batch.block_tables,
                   batch.num_blocks, batch.poison_block)
        o1 = oracle.attn(b1, q[off[r]: off[r + 1]], kc, vc)
        assert np.array_equal(o1, out[off[r]: off[r + 1]])


def test_gqa_replication_invariance():
    """Copying each kv head G times and running with G = 1 changes nothing."""
    batch = make_config(1)
    tens = make_tensors(batch, seed=10)
    out, kc, vc = run_step(batch, tens)
    G = batch.group
    kcr = kc.reshape(batch.num_blocks, 2, 16, 64).repeat(G, axis=1)
    vcr = vc.reshape(batch.num_blocks, 2, 64, 16).repeat(G, axis=1)
    b2 = Batch("rep", 4, 4, 64, 16, batch.rows, batch.block_tables, batch.num_blocks,
               batch.poison_block)
    out2 = oracle.attn(b2, tens["q"], kcr, vcr)
    assert np.array_equal(out, out2)


def test_selection_matches_full_output():
    batch = make_config(1)
    tens = make_tensors(batch, seed=12)
    out, kc, vc = run_step(batch, tens)
    sel = np.random.default_rng(12).choice(batch.num_tokens * 4, 50, replace=False)
    got = oracle.attn(batch, tens["q"], kc, vc, sel=sel)
    assert np.array_equal(got, out.reshape(-1, 64)[sel])


# ---------------------------------------------------------------- append

@pytest.mark.parametrize("cfg", ["tiny", "replay"])
def test_append_gather_roundtrip_and_untouched(cfg):
    if cfg == "tiny":
        batch = make_config(1)
        tens = make_tensors(batch, seed=13)
        kc0, vc0 = words(tens["k_cache"]), words(tens["v_cache"])
    else:
        batches, _ = replay_schedule(n_req=6, iters=3, budget=300, hq=8, hkv=2, d=64, bsz=16)
        batch = batches[1]
        tens = make_tensors(batch, seed=14, fill_prior=True, poison=True)
        kc0, vc0 = words(tens["k_cache"]), words(tens["v_cache"])
    kc, vc = oracle.kv_append(batch, tens["k_new"], tens["v_new"], kc0, vc0)
    # gather back the new tokens
    B, Hkv, D = batch.block_size, batch.num_kv_heads, batch.head_dim
    kc4 = kc.reshape(batch.num_blocks, Hkv, B, D)
    vc4 = vc.reshape(batch.num_blocks, Hkv, D, B)
    kn, vn = words(tens["k_new"]), words(tens["v_new"])
    touched = np.zeros((batch.num_blocks, B), bool)
    off = 0
    for req, s, c, ctx in batch.rows.tolist():
        pos = np.arange(s, s + c)
        blk = batch.block_tables[req][pos // B]
        assert np.array_equal(kc4[blk, :, pos % B, :], kn[off: off + c])
        assert np.array_equal(vc4[blk, :, :, pos % B], vn[off: off + c])
        touched[blk, pos % B] = True
        off += c
    k0 = kc0.reshape(batch.num_blocks, Hkv, B, D)
    v0 = vc0.reshape(batch.num_blocks, Hkv, D, B)
    bi, si = np.nonzero(~touched)
    assert np.array_equal(kc4[bi, :, si, :], k0[bi, :, si, :])
    assert np.array_equal(vc4[bi, :, :, si], v0[bi, :, :, si])
    kd, vd = dense.dense_append(batch, kn, vn, kc0, vc0)
    assert np.array_equal(kd.reshape(-1), kc.reshape(-1))
    assert np.array_equal(vd.reshape(-1), vc.reshape(-1))


def test_oracle_rejects_bad_metadata():
    batch = make_config(1)
    tens = make_tensors(batch, seed=15)
    bad = batch.rows.copy()
    bad[0, 3] += 1
    b2 = Batch("bad", 4, 2, 64, 16, bad, batch.block_tables, batch.num_blocks, 0)
    with pytest.raises(ValueError):
        oracle.attn(b2, tens["q"], tens["k_cache"], tens["v_cache"])


# ---------------------------------------------------------------- mutations

MUTATIONS = {
    "causal_off_by_one": ("const int n_keys = pos + 1;", "const int n_keys = pos + (pos > 0 ? 0 : 1);"),
    "gqa_modulo": ("const int kvh = h / (g->Hq / g->Hkv);", "const int kvh = h % g->Hkv;"),
    "scale_dropped": ("s[i] = scale * dot;", "s[i] = dot;"),
    "v_layout_transposed": ("return (((size_t)blk * g->Hkv + h) * g->D + d) * g->B + slot;",
                            "return (((size_t)blk * g->Hkv + h) * g->B + slot) * g->D + d;"),
    "block_index_wrong": ("return bt[(size_t)req * g->MBR + pos / g->B];",
                          "return bt[(size_t)req * g->MBR + (pos / g->B + 1) % g->MBR];"),
    "denominator_dropped": ("o[d] /= denom;", "o[d] /= 1.0;"),
    "weights_unexponentiated": ("const double w = exp(s[i] - smax);", "const double w = s[i] - smax + 1.0;"),
    "append_slot_shift": ("k_cache[k_slot(&g, blk, h, pos % B, d)] = k_new[src];",
                          "k_cache[k_slot(&g, blk, h, (pos + 1) % B, d)] = k_new[src];"),
    "query_row_wrong": ("const int pos = rows[4 * r + 1] + (int)(t - off[r]);",
                        "const int pos = rows[4 * r + 3] - 1;"),
}


def _pins_pass(lib):
    """A fast subset of the pins above, run against a given oracle build."""
    try:
        _, batch, q, kc, vc = _golden_batch()
        g = json.load(open(os.path.join(HERE, "golden", "two_key_worked_example.json")))
        out = oracle.attn(batch, q, kc, vc, lib=lib)
        for pos, exprs in g["expected_by_position"].items():
            want = [eval(x, {"e": math.e}) for x in exprs]
            if not np.allclose(out[int(pos), 0], want, rtol=0, atol=1e-15):
                return False
        for case, batch in enumerate(_tiny_cases()):
            tens = make_tensors(batch, seed=300 + case)
            kn, vn = words(tens["k_new"]), words(tens["v_new"])
            kc0, vc0 = words(tens["k_cache"]), words(tens["v_cache"])
            kc, vc = oracle.kv_append(batch, kn, vn, kc0, vc0, lib=lib)
            kd, vd = dense.dense_append(batch, kn, vn, kc0, vc0)
            if not (np.array_equal(kd.reshape(-1), kc.reshape(-1))
                    and np.array_equal(vd.reshape(-1), vc.reshape(-1))):
                return False
            out = oracle.attn(batch, tens["q"], kc, vc, lib=lib)
            ref = dense.dense_attention(batch, words(tens["q"]), kd, vd)
            if not np.allclose(out, ref, rtol=0, atol=1e-12):
                return False
    except ValueError:
        return False
    return True


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_planted_mistake_is_caught(name, tmp_path):
    src = open(oracle.SRC).read()
    old, new = MUTATIONS[name]
    assert src.count(old) == 1, f"mutation anchor for {name} not found once"
    mutated = tmp_path / "mut.c"
    mutated.write_text(src.replace(old, new))
    so = str(tmp_path / "libmut.so")
    oracle.build(str(mutated), so)
    lib = oracle.load(so)
    assert not _pins_pass(lib), f"planted mistake '{name}' passed every pin"


def test_unmutated_oracle_passes_pin_subset():
    assert _pins_pass(oracle.load())


def test_inplace_append_equals_copying_append():
    """The in-place form of the oracle's append writes the same pools."""
    import numpy as np
    import oracle
    from workloads import make_config, make_tensors
    b = make_config(1)
    t = make_tensors(b, seed=77)
    kc, vc = oracle.kv_append(b, t["k_new"], t["v_new"], t["k_cache"], t["v_cache"])
    k2 = t["k_cache"].view(__import__("torch").int16).numpy().view(np.uint16).copy()
    v2 = t["v_cache"].view(__import__("torch").int16).numpy().view(np.uint16).copy()
    k3, v3 = oracle.kv_append(b, t["k_new"], t["v_new"], k2, v2, inplace=True)
    assert k3 is k2 and v3 is v2
    assert np.array_equal(k2, kc) and np.array_equal(v2, vc)
