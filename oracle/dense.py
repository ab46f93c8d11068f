"""Dense-matrix brute force for tiny batches (numpy float64).

TEST INFRASTRUCTURE ONLY.  A second formulation of the same step, written
independently of ``cp_oracle.c``: for each row, gather the request's pages
into dense K and V in logical order, form the full score matrix, apply an
explicit bottom-right causal mask (query j of a chunk that starts at
position chunk_start may see keys 0..chunk_start+j), softmax along keys and
multiply by V.  Used to pin the C oracle; too slow for real sizes.
"""

from __future__ import annotations

import numpy as np


def bf16_to_f64(words) -> np.ndarray:
    """Raw bf16 words (uint16) -> float64 (exact widening)."""
    w = np.asarray(words).view(np.uint16).astype(np.uint32) << 16
    return w.view(np.float32).astype(np.float64)


def gather_kv(k_cache_f, v_cache_f, bt_row, ctx, block_size):
    """Dense [ctx, Hkv, D] K and V of one request from float K/V pools
    (k pool [NB][Hkv][B][D], v pool [NB][Hkv][D][B])."""
    pos = np.arange(ctx)
    blk = np.asarray(bt_row)[pos // block_size]
    slot = pos % block_size
    K = k_cache_f[blk, :, slot, :]          # [ctx, Hkv, D]
    V = v_cache_f[blk, :, :, slot]          # [ctx, Hkv, D]
    return K, V


def causal_mask(chunk_start, chunk_len, ctx):
    """Boolean [chunk_len, ctx]: True where query j may attend key i."""
    j = np.arange(chunk_len)[:, None]
    i = np.arange(ctx)[None, :]
    return i <= chunk_start + j


def dense_attention(batch, q_words, kc_words, vc_words):
    """[T, Hq, D] float64 output of the whole batch."""
    q = bf16_to_f64(q_words).reshape(batch.num_tokens, batch.num_q_heads, batch.head_dim)
    kc = bf16_to_f64(kc_words).reshape(batch.num_blocks, batch.num_kv_heads,
                                       batch.block_size, batch.head_dim)
    vc = bf16_to_f64(vc_words).reshape(batch.num_blocks, batch.num_kv_heads,
                                       batch.head_dim, batch.block_size)
    G = batch.group
    scale = float(np.float32(batch.sm_scale))
    out = np.zeros_like(q)
    off = 0
    for req, start, length, ctx in batch.rows.tolist():
        if length == 0:
            continue
        K, V = gather_kv(kc, vc, batch.block_tables[req], ctx, batch.block_size)
        mask = causal_mask(start, length, ctx)
        for h in range(batch.num_q_heads):
            Q = q[off: off + length, h, :]                     # [len, D]
            S = scale * (Q @ K[:, h // G, :].T)                # [len, ctx]
            S = np.where(mask, S, -np.inf)
            S = S - S.max(axis=1, keepdims=True)
            P = np.exp(S)
            P = P / P.sum(axis=1, keepdims=True)
            out[off: off + length, h, :] = P @ V[:, h // G, :]
        off += length
    return out


def dense_append(batch, kn_words, vn_words, kc_words, vc_words):
    """Scatter of the step's new K/V rows into copies of the pools (uint16)."""
    B, Hkv, D = batch.block_size, batch.num_kv_heads, batch.head_dim
    kc = np.array(kc_words, dtype=np.uint16).reshape(batch.num_blocks, Hkv, B, D)
    vc = np.array(vc_words, dtype=np.uint16).reshape(batch.num_blocks, Hkv, D, B)
    kn = np.asarray(kn_words, dtype=np.uint16).reshape(-1, Hkv, D)
    vn = np.asarray(vn_words, dtype=np.uint16).reshape(-1, Hkv, D)
    off = 0
    for req, start, length, _ in batch.rows.tolist():
        pos = np.arange(start, start + length)
        blk = batch.block_tables[req][pos // B]
        slot = pos % B
        kc[blk, :, slot, :] = kn[off: off + length]
        vc[blk, :, :, slot] = vn[off: off + length]
        off += length
    return kc, vc
