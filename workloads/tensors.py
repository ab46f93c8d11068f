"""Seeded bf16 tensors for a :class:`~workloads.configs.Batch`.

Values are fp32 draws from N(0, 1) rounded to bf16 (round-to-nearest-even,
torch's conversion).  Layouts are the library's:

    q            [T][Hq][D]
    k_new, v_new [T][Hkv][D]
    k_cache      [NB][Hkv][B][D]      (token-major rows inside a block)
    v_cache      [NB][Hkv][D][B]      (feature-major rows inside a block)

Cache slots that a correct step never reads hold bf16 NaN (0x7FC0): every
block no request references, and, in referenced blocks, every slot at a
logical position >= chunk_start (not yet written when the step starts; the
append fills [chunk_start, ctx) and the tail past ctx stays NaN).
"""

from __future__ import annotations

import numpy as np
import torch

_CHUNK = 1 << 26  # elements per randn call; bounds the fp32 temporary


def _randn_bf16(shape, gen, device):
    n = int(np.prod(shape))
    out = torch.empty(n, dtype=torch.bfloat16, device=device)
    for s in range(0, n, _CHUNK):
        e = min(n, s + _CHUNK)
        out[s:e] = torch.randn(e - s, generator=gen, device=device, dtype=torch.float32)
    return out.view(*shape)


def tail_slots(batch):
    """(block, slot) of every logical position in [chunk_start, n_blocks*B) of every row."""
    B = batch.block_size
    blks, slots = [], []
    for rid, s, c, ctx in batch.rows:
        nb = -(-int(ctx) // B)
        if nb == 0:
            continue
        p = np.arange(int(s), nb * B, dtype=np.int64)
        blks.append(batch.block_tables[int(rid), p // B].astype(np.int64))
        slots.append(p % B)
    if not blks:
        return np.zeros(0, np.int64), np.zeros(0, np.int64)
    return np.concatenate(blks), np.concatenate(slots)


def make_step_tensors(batch, seed, device="cpu"):
    """q, k_new, v_new for one iteration (draw order: q, k_new, v_new)."""
    gen = torch.Generator(device=device)
    gen.manual_seed(int(seed))
    T, Hq, Hkv, D = batch.num_tokens, batch.num_q_heads, batch.num_kv_heads, batch.head_dim
    q = _randn_bf16((T, Hq, D), gen, device)
    k_new = _randn_bf16((T, Hkv, D), gen, device)
    v_new = _randn_bf16((T, Hkv, D), gen, device)
    return q, k_new, v_new, gen


def make_caches(batch, gen=None, device="cpu", fill_prior=True, poison=True, seed=None):
    """K and V pools: N(0,1) prior context (or all NaN if ``fill_prior`` is False),
    NaN in unreferenced blocks and in every slot at or past each row's chunk_start."""
    if gen is None and fill_prior:
        gen = torch.Generator(device=device)
        gen.manual_seed(int(seed))
    NB, Hkv, B, D = batch.num_blocks, batch.num_kv_heads, batch.block_size, batch.head_dim
    if fill_prior:
        kc = _randn_bf16((NB, Hkv, B, D), gen, device)
        vc = _randn_bf16((NB, Hkv, D, B), gen, device)
    else:
        kc = torch.full((NB, Hkv, B, D), float("nan"), dtype=torch.bfloat16, device=device)
        vc = torch.full((NB, Hkv, D, B), float("nan"), dtype=torch.bfloat16, device=device)
    if poison and fill_prior:
        nan = torch.tensor(float("nan"), dtype=torch.bfloat16, device=device)
        if batch.referenced is not None:
            unref = torch.from_numpy(np.nonzero(~batch.referenced)[0]).to(device)
            if unref.numel():
                kc[unref] = nan
                vc[unref] = nan
        blk, slot = tail_slots(batch)
        if blk.size:
            bt_ = torch.from_numpy(blk).to(device)
            st_ = torch.from_numpy(slot).to(device)
            kc[bt_, :, st_, :] = nan
            vc[bt_, :, :, st_] = nan
    return kc, vc


def make_tensors(batch, seed, device="cpu", fill_prior=True, poison=True):
    """All inputs of one step: dict with q, k_new, v_new, k_cache, v_cache
    (bf16, on ``device``) and block_tables (int32)."""
    q, k_new, v_new, gen = make_step_tensors(batch, seed, device)
    kc, vc = make_caches(batch, gen, device, fill_prior=fill_prior, poison=poison)
    bt = torch.from_numpy(batch.block_tables).to(device)
    return {"q": q, "k_new": k_new, "v_new": v_new, "k_cache": kc, "v_cache": vc,
            "block_tables": bt}
