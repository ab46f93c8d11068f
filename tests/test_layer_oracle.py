"""Pins of the decoder-layer reference (oracle/layer.py) against closed forms
and invariants of RMSNorm, rotary embedding and SwiGLU."""

import math

import numpy as np
import pytest

from oracle import layer as ref


def test_rmsnorm_closed_forms():
    w = np.linspace(0.5, 2.0, 8)
    # a constant row normalises to sign * w (up to eps)
    y = ref.rmsnorm(np.full((1, 8), -3.0), w, 1e-12)
    assert np.allclose(y[0], -w, rtol=1e-10)
    # scale invariance for positive factors
    rng = np.random.default_rng(0)
    x = rng.normal(size=(4, 32))
    assert np.allclose(ref.rmsnorm(x, 1.0, 1e-12), ref.rmsnorm(7.5 * x, 1.0, 1e-12), rtol=1e-10)
    # unit root-mean-square output with unit weights
    assert np.allclose(np.sqrt((ref.rmsnorm(x, 1.0, 0.0) ** 2).mean(axis=1)), 1.0)
    # hand value: x = (3, 4): mean square 12.5
    assert np.allclose(ref.rmsnorm(np.array([[3.0, 4.0]]), 1.0, 0.0),
                       [[3 / math.sqrt(12.5), 4 / math.sqrt(12.5)]])


def test_rope_identity_at_zero_and_norm_preserving():
    rng = np.random.default_rng(1)
    x = rng.normal(size=(5, 3, 64))
    assert np.allclose(ref.rope(x, np.zeros(5), 1e6), x)
    y = ref.rope(x, np.array([1, 17, 300, 4095, 32767]), 1e6)
    assert np.allclose(np.linalg.norm(y, axis=-1), np.linalg.norm(x, axis=-1))


def test_rope_first_pair_turns_by_the_position():
    # d = 0 has frequency theta^0 = 1: the pair (x0, x_half) turns by pos radians.
    x = np.zeros((1, 1, 8))
    x[0, 0, 0] = 1.0
    y = ref.rope(x, np.array([0.5]), 10000.0)
    assert np.isclose(y[0, 0, 0], math.cos(0.5)) and np.isclose(y[0, 0, 4], math.sin(0.5))


def test_rope_scores_depend_on_relative_position_only():
    rng = np.random.default_rng(2)
    q = rng.normal(size=(1, 1, 128))
    k = rng.normal(size=(1, 1, 128))
    def score(pq, pk):
        return float(ref.rope(q, [pq], 1e6)[0, 0] @ ref.rope(k, [pk], 1e6)[0, 0])
    assert math.isclose(score(10, 3), score(1010, 1003), rel_tol=1e-9, abs_tol=1e-9)
    assert math.isclose(score(500, 0), score(4000, 3500), rel_tol=1e-9, abs_tol=1e-9)


def test_silu_and_swiglu_values():
    assert ref.silu(0.0) == 0.0
    assert math.isclose(float(ref.silu(1.0)), 1 / (1 + math.exp(-1)))
    assert math.isclose(float(ref.silu(40.0)), 40.0, rel_tol=1e-15)
    assert abs(float(ref.silu(-40.0))) < 1e-15
    gu = np.array([[1.0, -2.0, 3.0, 0.5]])
    assert np.allclose(ref.swiglu(gu), [[ref.silu(1.0) * 3.0, ref.silu(-2.0) * 0.5]])


def test_qkv_split_layout():
    hq, hkv, D = 2, 1, 4
    qkv = np.arange((hq + 2 * hkv) * D, dtype=float)[None] + 1.0
    q, k, v = ref.qkv_rope(qkv, np.ones(D), np.ones(D), np.zeros(1), hq, hkv, D, 1e4, 0.0)
    assert np.allclose(v[0, 0], qkv[0, 12:16])
    assert np.allclose(q[0, 1], ref.rmsnorm(qkv[0, 4:8], 1.0, 0.0))
    assert np.allclose(k[0, 0], ref.rmsnorm(qkv[0, 8:12], 1.0, 0.0))


def test_attention_single_key_returns_its_value():
    q = np.ones((1, 2, 4))
    k = np.zeros((1, 1, 4))
    v = np.arange(4.0).reshape(1, 1, 4)
    out = ref.attention(q, k, v, [(0, 0, 1, 1)], {0: np.zeros((0, 1, 4))},
                        {0: np.zeros((0, 1, 4))}, 0.5)
    assert np.allclose(out[0, 0], v[0, 0]) and np.allclose(out[0, 1], v[0, 0])


def test_attention_equal_keys_average_values():
    rng = np.random.default_rng(3)
    q = rng.normal(size=(1, 1, 8))
    pk = np.tile(rng.normal(size=(1, 1, 8)), (5, 1, 1))
    pv = rng.normal(size=(5, 1, 8))
    out = ref.attention(q, pk[:1], pv[4:5], [(0, 4, 1, 5)], {0: pk}, {0: pv}, 0.3)
    assert np.allclose(out[0, 0], pv.mean(axis=0)[0])


def test_decoder_layer_with_zero_projections_is_identity():
    H, hq, hkv, D, I = 16, 2, 1, 8, 12
    rng = np.random.default_rng(4)
    wts = {"in_norm": np.ones(H), "qkv": rng.normal(size=((hq + 2 * hkv) * D, H)),
           "q_norm": np.ones(D), "k_norm": np.ones(D), "o": np.zeros((H, hq * D)),
           "post_norm": np.ones(H), "gate_up": rng.normal(size=(2 * I, H)),
           "down": np.zeros((H, I))}
    x = rng.normal(size=(3, H))
    rows = [(0, 0, 3, 3)]
    out, k, v = ref.decoder_layer(x, wts, rows, {0: np.zeros((0, hkv, D))},
                                  {0: np.zeros((0, hkv, D))}, hq, hkv, D, 1e6, 1e-6, 0.35)
    assert np.allclose(out, x)
    assert k.shape == (3, hkv, D) and v.shape == (3, hkv, D)


def test_layer_library_exports_every_declared_function():
    import os
    import re
    from paper_2606_09061_amd import model as M
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    src = open(os.path.join(root, "include", "cp_layer.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    names = sorted(set(re.findall(r"\b(cpl_[a-z_]+)\s*\(", src)))
    assert names == sorted(M.exported_symbols())
    lib = M.load()
    for n in names:
        assert hasattr(lib, n)


def test_positions_of_rows():
    from paper_2606_09061_amd.model import positions_of
    rows = np.array([[3, 7, 2, 9], [0, 0, 0, 0], [1, 199, 1, 200], [2, 0, 3, 3]])
    assert positions_of(rows).tolist() == [7, 8, 199, 0, 1, 2]
    assert positions_of(np.zeros((0, 4))).tolist() == []


def test_skinny_dispatch_follows_measured_table():
    from paper_2606_09061_amd.model import skinny_faster
    qkv, o, gate_up, down = (6144, 4096), (4096, 4096), (24576, 4096), (4096, 12288)
    for n, k in (qkv, o, gate_up, down):
        assert skinny_faster(1, n, k) and skinny_faster(16, n, k)
        assert not skinny_faster(33, n, k) and not skinny_faster(128, n, k)
    assert skinny_faster(32, *qkv) and skinny_faster(32, *gate_up) and skinny_faster(32, *down)
    assert not skinny_faster(1, 1000, 256) and not skinny_faster(1, 64, 320)   # unsupported shapes


def test_gemm_validates_before_launching():
    """cpl_gemm refuses unsupported shapes, aliasing and misalignment on the
    host, before touching the device (so this runs without a GPU)."""
    from paper_2606_09061_amd import model as M
    lib = M.load()
    a, w, c = 1 << 20, 2 << 20, 3 << 20      # aligned stand-in addresses, never dereferenced

    def bad(a_, w_, r_, c_, m, n, k, ws=None):
        return lib.cpl_gemm(a_, w_, r_, c_, m, n, k, ws, 1 << 20, None)
    assert bad(a, w, None, c, 0, 128, 32) != 0       # M = 0
    assert bad(a, w, None, c, 8, 96, 32) != 0        # N % 128
    assert bad(a, w, None, c, 8, 128, 48) != 0       # K % 32
    assert bad(a, w, None, a, 8, 128, 32) != 0       # a aliases c
    assert bad(a, w, None, w, 8, 128, 32) != 0       # w aliases c
    assert bad(a + 8, w, None, c, 8, 128, 32) != 0   # misaligned a
    assert bad(a, w, c + 4, c, 8, 128, 32) != 0      # misaligned residual
    assert bad(a, w, None, c, 8, 128, 32, ws=c + 8) != 0   # misaligned workspace
    assert bad(None, w, None, c, 8, 128, 32) != 0    # null
    # the workspace a full split needs: none for a grid that fills the GPU
    assert lib.cpl_gemm_workspace_bytes(4096, 6144, 4096) == 0
    assert lib.cpl_gemm_workspace_bytes(64, 4096, 4096) > 0
    assert lib.cpl_gemm_workspace_bytes(8, 96, 32) == 0
