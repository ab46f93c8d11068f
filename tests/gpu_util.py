"""Shared helpers of the GPU tests: run the step through the C ABI and
compare it with the fp64 oracle."""

import sys

import numpy as np
import torch

import oracle
import paper_2606_09061_amd as cp

MAX_ABS = 2e-2   # max |gpu - oracle| over bf16 outputs
MEAN_ABS = 2e-3  # mean |gpu - oracle|


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def check_shapes(batch, t):
    T, Hq, Hkv, D, B, NB = (batch.num_tokens, batch.num_q_heads, batch.num_kv_heads,
                           batch.head_dim, batch.block_size, batch.num_blocks)
    assert tuple(t["q"].shape) == (T, Hq, D)
    assert tuple(t["k_new"].shape) == (T, Hkv, D) and tuple(t["v_new"].shape) == (T, Hkv, D)
    assert tuple(t["k_cache"].shape) == (NB, Hkv, B, D)
    assert tuple(t["v_cache"].shape) == (NB, Hkv, D, B)
    bt = t["block_tables"]
    assert tuple(bt.shape) == (batch.num_reqs_in_table, batch.max_blocks_per_req)
    assert bt.dtype == torch.int32
    btn = batch.block_tables
    for req, s, c, ctx in batch.rows.tolist():
        nb = -(-ctx // B)
        assert (btn[req, :nb] >= 0).all() and (btn[req, :nb] < NB).all()


def run_step(batch, t, out=None, ws=None, stream=None, one_call=False):
    """cp_kv_append then cp_attn_mixed on device tensors ``t`` (caches updated
    in place); with ``one_call``, the same step as one cp_step_mixed call, the
    call the benchmark times."""
    check_shapes(batch, t)
    d = cp.desc_for(batch)
    if out is None:
        out = torch.empty(batch.num_tokens, batch.num_q_heads, batch.head_dim,
                          dtype=torch.bfloat16, device=t["q"].device)
    if ws is None:
        ws = torch.empty(max(256, cp.workspace_bytes(d, batch.rows)), dtype=torch.uint8,
                         device=t["q"].device)
    if one_call:
        cp.step_mixed(d, t["q"], t["k_new"], t["v_new"], t["k_cache"], t["v_cache"],
                      t["block_tables"], batch.rows, out, ws, stream=stream)
        return out
    cp.kv_append(d, t["k_new"], t["v_new"], t["k_cache"], t["v_cache"], t["block_tables"],
                 batch.rows, ws, stream=stream)
    cp.attn_mixed(d, t["q"], t["k_cache"], t["v_cache"], t["block_tables"], batch.rows, out, ws,
                  stream=stream)
    return out


def to_dev(t, dev="cuda"):
    return {k: v.to(dev) for k, v in t.items()}


def words(x):
    return x.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


def errors(gpu_out, ref):
    g = gpu_out.detach().cpu().float().numpy().astype(np.float64).reshape(ref.shape)
    assert np.isfinite(g).all(), "non-finite GPU output"
    e = np.abs(g - ref)
    return float(e.max()) if e.size else 0.0, float(e.mean()) if e.size else 0.0


def bf16_rne(x):
    """fp64 values rounded once to the nearest bfloat16 (8 significant bits),
    ties to even; exact for the normal range the attention outputs live in."""
    m, e = np.frexp(np.asarray(x, dtype=np.float64))
    return np.ldexp(np.round(np.ldexp(m, 8)), e - 8)


def floor_errors(ref):
    """max and mean |bf16(oracle) - oracle|: the error of a perfectly rounded
    bf16 output, the floor under any bf16 result."""
    e = np.abs(bf16_rne(ref) - ref)
    return float(e.max()) if e.size else 0.0, float(e.mean()) if e.size else 0.0


def assert_close(gpu_out, ref, what=""):
    mx, mean = errors(gpu_out, ref)
    fmx, fmean = floor_errors(ref)
    say(f"  {what}: max_abs={mx:.3e} mean_abs={mean:.3e} "
        f"(oracle rounded to bf16: max {fmx:.3e} mean {fmean:.3e})")
    assert mx <= MAX_ABS and mean <= MEAN_ABS, f"{what}: max {mx:.3e} mean {mean:.3e}"
    return mx, mean
