"""fp64 reference of the decoder layer around the attention step.

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, never by the product.  It
shares no code with libcplayer.so or the package's model code.  Each
function is the plain definition (numpy float64, inputs widened exactly from
bf16 where they come as bf16 words):

  * rmsnorm:   y = x * w / sqrt(mean(x^2) + eps) over the last axis;
  * qkv_rope:  split of the fused projection into q, k, v heads; per-head
               RMSNorm of q and k; rotation of the pairs (d, d + D/2) by the
               angle pos * theta^(-2d/D) (the Qwen3 / Llama rotary layout);
  * swiglu:    silu(gate) * up, silu(g) = g / (1 + exp(-g));
  * decoder_layer: x + O(attn(...)) then + down(swiglu(gate_up(rmsnorm))),
               with causal attention over the request's cached keys (earlier
               positions read from the paged pools, this batch's from the
               new rows) - the same bottom-right alignment as the step.

The paper does not describe the model; these follow the published Qwen3
architecture.
"""

from __future__ import annotations

import numpy as np


def bf16_to_f64(words) -> np.ndarray:
    w = np.asarray(words).view(np.uint16).astype(np.uint32) << 16
    return w.view(np.float32).astype(np.float64)


def rmsnorm(x, w, eps):
    x = np.asarray(x, np.float64)
    return x * np.asarray(w, np.float64) / np.sqrt((x * x).mean(axis=-1, keepdims=True) + eps)


def rope(x, positions, theta):
    """Rotates [T, H, D] by position: pairs (d, d + D/2), angle pos * theta^(-2d/D)."""
    x = np.asarray(x, np.float64)
    D = x.shape[-1]
    half = D // 2
    inv_freq = theta ** (-2.0 * np.arange(half) / D)
    ang = np.asarray(positions, np.float64)[:, None] * inv_freq[None, :]      # [T, half]
    c, s = np.cos(ang)[:, None, :], np.sin(ang)[:, None, :]
    a, b = x[..., :half], x[..., half:]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


def qkv_rope(qkv, q_norm_w, k_norm_w, positions, hq, hkv, D, theta, eps):
    qkv = np.asarray(qkv, np.float64).reshape(-1, hq + 2 * hkv, D)
    q = rope(rmsnorm(qkv[:, :hq], q_norm_w, eps), positions, theta)
    k = rope(rmsnorm(qkv[:, hq:hq + hkv], k_norm_w, eps), positions, theta)
    v = qkv[:, hq + hkv:].copy()
    return q, k, v


def silu(g):
    g = np.asarray(g, np.float64)
    return g / (1.0 + np.exp(-g))


def swiglu(gu):
    gu = np.asarray(gu, np.float64)
    inter = gu.shape[-1] // 2
    return silu(gu[..., :inter]) * gu[..., inter:]


def positions_of(rows):
    return np.concatenate([np.arange(s, s + c) for _, s, c, _ in rows if c > 0] or
                          [np.zeros(0, np.int64)])


def attention(q, k_new, v_new, rows, prior_k, prior_v, sm_scale):
    """Causal attention of the batch's queries.  q [T, Hq, D]; k_new, v_new
    [T, Hkv, D]; prior_k[req], prior_v[req]: [ctx_prior, Hkv, D] keys and values
    of the positions before the row's chunk.  Returns [T, Hq, D]."""
    T, Hq, D = q.shape
    Hkv = k_new.shape[1]
    G = Hq // Hkv
    out = np.zeros_like(q)
    off = 0
    for req, start, length, ctx in rows:
        if length == 0:
            continue
        K = np.concatenate([prior_k[req][:start], k_new[off:off + length]], axis=0)
        V = np.concatenate([prior_v[req][:start], v_new[off:off + length]], axis=0)
        for j in range(length):
            p = start + j
            for h in range(Hq):
                s = sm_scale * (K[:p + 1, h // G] @ q[off + j, h])
                w = np.exp(s - s.max())
                out[off + j, h] = (w @ V[:p + 1, h // G]) / w.sum()
        off += length
    return out


def decoder_layer(x, wts, rows, prior_k, prior_v, hq, hkv, D, theta, eps, sm_scale):
    """One layer.  wts: dict of float64 arrays in_norm [H], qkv [(hq+2hkv)D, H],
    q_norm [D], k_norm [D], o [H, hq D], post_norm [H], gate_up [2I, H],
    down [H, I] (row-major [out, in]).  Returns (x_out, k_new, v_new)."""
    x = np.asarray(x, np.float64)
    pos = positions_of(rows)
    h = rmsnorm(x, wts["in_norm"], eps)
    q, k, v = qkv_rope(h @ wts["qkv"].T, wts["q_norm"], wts["k_norm"], pos, hq, hkv, D, theta,
                       eps)
    a = attention(q, k, v, rows, prior_k, prior_v, sm_scale)
    x = x + a.reshape(len(x), hq * D) @ wts["o"].T
    h = rmsnorm(x, wts["post_norm"], eps)
    x = x + swiglu(h @ wts["gate_up"].T) @ wts["down"].T
    return x, k, v
