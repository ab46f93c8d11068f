"""A Qwen3-style decoder stack around the attention step, on one GPU.

The paper's predictor and target latency T* refer to a whole model iteration
(Sec. 3.2.1; Sec. 4.4 uses Qwen3-8B with T* = 105 ms), so this module runs the
scheduler's batch through every layer of such a model with synthetic weights:

    embedding -> L x [RMSNorm -> QKV GEMM -> cpl_qkv_rope -> cp_kv_append ->
    cp_attn_mixed -> O GEMM (+ residual) -> RMSNorm -> gate/up GEMM ->
    cpl_swiglu -> down GEMM (+ residual)] -> RMSNorm -> LM head on each row's
    last token -> argmax

Projections of small batches (up to 32 tokens) run in this package's skinny
GEMM kernel, the rest as library GEMMs (torch.mm / addmm, i.e. hipBLASLt);
every other step runs in this package's HIP kernels
(libcplayer.so for the element-wise parts, libcpattn.so for append and
attention).  Each layer has
its own paged KV pool; all layers share one block table, whose row s maps
slot s's logical blocks to physical blocks (a random permutation, so pages
are scattered).  Weights are N(0, 0.02) in bf16, norms 1.
"""

from __future__ import annotations

import ctypes
import math
import os
from dataclasses import dataclass

import numpy as np

from . import binding as cp

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libcplayer.so")

_lib = None


def load():
    """Loads libcplayer.so; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it first "
                           "(python -m paper_2606_09061_amd.build)")
    lib = ctypes.CDLL(LIB_PATH)
    P, I32, F, D = ctypes.c_void_p, ctypes.c_int32, ctypes.c_float, ctypes.c_double
    lib.cpl_rmsnorm.argtypes = [P, P, P, I32, I32, F, P]
    lib.cpl_qkv_rope.argtypes = [P, P, P, P, I32, I32, I32, I32, D, F, P, P, P, P]
    lib.cpl_swiglu.argtypes = [P, P, I32, I32, P]
    lib.cpl_gemm_skinny.argtypes = [P, P, P, P, I32, I32, I32, P]
    lib.cpl_gemm.argtypes = [P, P, P, P, I32, I32, I32, P, ctypes.c_size_t, P]
    lib.cpl_gemm_workspace_bytes.argtypes = [I32, I32, I32]
    lib.cpl_gemm_workspace_bytes.restype = ctypes.c_size_t
    for f in (lib.cpl_rmsnorm, lib.cpl_qkv_rope, lib.cpl_swiglu, lib.cpl_gemm_skinny, lib.cpl_gemm):
        f.restype = ctypes.c_int
    _lib = lib
    return lib


def exported_symbols():
    return ["cpl_rmsnorm", "cpl_qkv_rope", "cpl_swiglu", "cpl_gemm_skinny", "cpl_gemm",
            "cpl_gemm_workspace_bytes"]


def _check(rc, what):
    if rc != 0:
        raise cp.CpError(rc, what)


def _s(stream):
    return cp._stream(stream)


def _dense(*ts):
    for t in ts:
        if not t.is_contiguous():
            raise cp.CpError(cp.CP_ERR_INVALID_ARG, "layer kernels take dense tensors")


def rmsnorm(x, w, out, eps, stream=None):
    """out = RMSNorm(x) * w over the last axis (bf16 tensors; out may be x)."""
    _dense(x, w, out)
    n, width = x.shape[0], x.shape[-1]
    _check(load().cpl_rmsnorm(x.data_ptr(), w.data_ptr(), out.data_ptr(), n, width, eps,
                              _s(stream)), "cpl_rmsnorm")


def qkv_rope(qkv, q_norm_w, k_norm_w, positions, hq, hkv, head_dim, theta, eps, q, k, v,
             stream=None):
    """Splits qkv [T, (hq+2hkv)*D] into q [T, hq, D], k, v [T, hkv, D] with
    per-head RMSNorm and rotary embedding of q and k (positions: int32 [T])."""
    _dense(qkv, q_norm_w, k_norm_w, positions, q, k, v)
    _check(load().cpl_qkv_rope(qkv.data_ptr(), q_norm_w.data_ptr(), k_norm_w.data_ptr(),
                               positions.data_ptr(), qkv.shape[0], hq, hkv, head_dim,
                               float(theta), eps, q.data_ptr(), k.data_ptr(), v.data_ptr(),
                               _s(stream)), "cpl_qkv_rope")


def swiglu(gu, out, stream=None):
    """out [T, I] = silu(gu[:, :I]) * gu[:, I:]."""
    _dense(gu, out)
    _check(load().cpl_swiglu(gu.data_ptr(), out.data_ptr(), gu.shape[0], out.shape[-1],
                             _s(stream)), "cpl_swiglu")


# Where the skinny kernel beats the library GEMM on MI355X.  Per launch, with
# the weights evicted from the caches beforehand (a model iteration streams
# 15 GB of weights), at one row: QKV 24.0 -> 14.2 us, O 21.0 -> 11.1, gate/up
# 79.3 -> 34.0, down 40.8 -> 23.5, LM head 288 -> 178; at 32 rows still
# 1.19-1.97x on all five.  A whole 36-layer decode iteration with this
# dispatch against the library alone: 1.29x at 1 row, 1.23x at 8, 1.18x at
# 16, 1.08x at 24, 1.03x at 32, even at 40 rows (each 32-column slice
# re-reads the activations), hence no skinny kernel above 32 rows.
def skinny_faster(m, n, k):
    if n % 32 or k % 256 or m < 1:
        return False
    return m <= 32


def gemm_skinny(a, w, out, residual=None, stream=None):
    """out [M, N] = a [M, K] @ w [N, K]^T (+ residual, which may be out itself)."""
    _dense(a, w, out)
    if residual is not None:
        _dense(residual)
    M, K = a.shape
    N = w.shape[0]
    _check(load().cpl_gemm_skinny(a.data_ptr(), w.data_ptr(),
                                  residual.data_ptr() if residual is not None else None,
                                  out.data_ptr(), M, N, K, _s(stream)), "cpl_gemm_skinny")


def gemm_workspace_bytes(m, n, k):
    """Device bytes cpl_gemm uses to split K for this shape (0: no split)."""
    return int(load().cpl_gemm_workspace_bytes(m, n, k))


def gemm(a, w, out, residual=None, stream=None, ws=None):
    """out [M, N] = a [M, K] @ w [N, K]^T (+ residual, which may be out itself),
    on the package's LDS-tiled MFMA kernel (cpl_gemm).  ``ws``: a uint8 device
    tensor for the split over K (allocated here when None and needed)."""
    import torch
    _dense(a, w, out)
    if residual is not None:
        _dense(residual)
    M, K = a.shape
    N = w.shape[0]
    need = gemm_workspace_bytes(M, N, K)
    if ws is None and need:
        ws = torch.empty(need, dtype=torch.uint8, device=a.device)
    _check(load().cpl_gemm(a.data_ptr(), w.data_ptr(),
                           residual.data_ptr() if residual is not None else None,
                           out.data_ptr(), M, N, K, ws.data_ptr() if ws is not None else None,
                           ws.numel() if ws is not None else 0, _s(stream)), "cpl_gemm")


def project_attn(a, w, out, residual=None, stream=None, ws=None):
    """The QKV and output projections around the attention step, always on
    the package's kernels: the skinny kernel up to 32 rows, the tiled MFMA
    GEMM above (``ws``: its split-K workspace, see gemm)."""
    M, K = a.shape
    N = w.shape[0]
    if skinny_faster(M, N, K):
        gemm_skinny(a, w, out, residual, stream)
    elif N % 128 == 0 and K % 32 == 0:
        gemm(a, w, out, residual, stream, ws)
    else:
        raise ValueError(f"projection {M}x{N}x{K}: the kernels need N % 128 == 0 and K % 32 == 0")


def project(a, w, out, residual=None, stream=None):
    """a @ w^T into out (+ residual): the skinny kernel where it is faster
    (small batches, moderate projections), the platform BLAS otherwise.
    The feed-forward and LM-head projections use it."""
    import torch
    M, K = a.shape
    N = w.shape[0]
    if skinny_faster(M, N, K):
        gemm_skinny(a, w, out, residual, stream)
    elif residual is None:
        torch.mm(a, w.t(), out=out)
    elif residual is out:
        out.addmm_(a, w.t())
    else:
        torch.addmm(residual, a, w.t(), out=out)


@dataclass
class ModelConfig:
    hidden: int = 4096
    layers: int = 36
    hq: int = 32
    hkv: int = 8
    head_dim: int = 128
    inter: int = 12288
    vocab: int = 151936
    eps: float = 1e-6
    theta: float = 1e6
    block_size: int = 16


QWEN3_8B = ModelConfig()


def positions_of(rows) -> np.ndarray:
    """Absolute position of every scheduled token, in row order."""
    rows = np.asarray(rows).reshape(-1, 4)
    lens = rows[:, 2].astype(np.int64)
    if lens.sum() == 0:
        return np.zeros(0, np.int32)
    base = np.repeat(rows[:, 1].astype(np.int64) - np.concatenate([[0], np.cumsum(lens)[:-1]]),
                     lens)
    return (base + np.arange(lens.sum())).astype(np.int32)


class Model:
    """Synthetic-weight decoder stack with per-layer paged KV pools."""

    def __init__(self, cfg: ModelConfig = QWEN3_8B, max_seqs=128, max_seq_len=4096,
                 max_tokens=2048, seed=0, device=None, lm_head=True, fill_caches=False):
        import torch
        from workloads.tensors import _randn_bf16

        self.cfg = c = cfg
        self.dev = device or torch.device("cuda", 0)
        self.max_tokens = max_tokens
        gen = torch.Generator(device=self.dev)
        gen.manual_seed(seed)

        def w(*shape):
            t = _randn_bf16(shape, gen, self.dev)
            return t.mul_(0.02)

        def ones(n):
            return torch.ones(n, dtype=torch.bfloat16, device=self.dev)

        H, D = c.hidden, c.head_dim
        nqkv = (c.hq + 2 * c.hkv) * D
        self.layers = [dict(in_norm=ones(H), qkv=w(nqkv, H), q_norm=ones(D), k_norm=ones(D),
                            o=w(H, c.hq * D), post_norm=ones(H), gate_up=w(2 * c.inter, H),
                            down=w(H, c.inter)) for _ in range(c.layers)]
        self.embed = w(c.vocab, H)
        self.final_norm = ones(H)
        self.lm_head = w(c.vocab, H) if lm_head else None
        mbr = -(-max_seq_len // c.block_size)
        nb = max_seqs * mbr
        rng = np.random.default_rng(seed)
        self.bt = torch.from_numpy(rng.permutation(nb).astype(np.int32).reshape(max_seqs, mbr)
                                   ).to(self.dev)
        # Serving writes every position before attention reads it, so pools may
        # start unwritten; fill_caches draws N(0,1) contents for benchmarks
        # that attend to context they never appended.
        if fill_caches:
            self.kc = [_randn_bf16((nb, c.hkv, c.block_size, D), gen, self.dev)
                       for _ in range(c.layers)]
            self.vc = [_randn_bf16((nb, c.hkv, D, c.block_size), gen, self.dev)
                       for _ in range(c.layers)]
        else:
            self.kc = [torch.empty(nb, c.hkv, c.block_size, D, dtype=torch.bfloat16,
                                   device=self.dev) for _ in range(c.layers)]
            self.vc = [torch.empty(nb, c.hkv, D, c.block_size, dtype=torch.bfloat16,
                                   device=self.dev) for _ in range(c.layers)]
        self.desc = cp.make_desc(c.hq, c.hkv, D, c.block_size, nb, mbr, max_seqs,
                                 1.0 / math.sqrt(D))
        T = max_tokens

        def buf(*shape):
            return torch.empty(*shape, dtype=torch.bfloat16, device=self.dev)

        self.x, self.h = buf(T, H), buf(T, H)
        self.qkv = buf(T, nqkv)
        self.q, self.k, self.v = buf(T, c.hq, D), buf(T, c.hkv, D), buf(T, c.hkv, D)
        self.attn = buf(T, c.hq, D)
        self.gu, self.act = buf(T, 2 * c.inter), buf(T, c.inter)
        self.pos_host = torch.zeros(T, dtype=torch.int32).pin_memory()
        self.pos_copied = torch.cuda.Event()   # the last upload out of pos_host is done
        self.pos = torch.zeros(T, dtype=torch.int32, device=self.dev)
        self.tokens = torch.randint(0, c.vocab, (T,), generator=gen, device=self.dev)
        self.ws = torch.empty(64 << 20, dtype=torch.uint8, device=self.dev)      # attention plan
        # split-K partials of the QKV / output projections (grown on demand)
        self.ws_gemm = torch.empty(256, dtype=torch.uint8, device=self.dev)
        # an append item covers one row's tokens inside one block: at most
        # max_tokens + max_seqs items of 16 bytes, so the append never needs more
        self.ws_append = torch.empty(16 * (max_tokens + max_seqs) + 256, dtype=torch.uint8,
                                     device=self.dev)

    def forward(self, rows, stream=None):
        """Runs one iteration for the batch ``rows`` [(slot, start, len, ctx)];
        returns the greedy next token of every row (device int64 [n_rows]), or
        None when the model has no LM head."""
        import torch
        c = self.cfg
        rows = np.ascontiguousarray(np.asarray(rows, dtype=np.int32).reshape(-1, 4))
        T = int(rows[:, 2].sum())
        if T == 0:
            return None
        if T > self.max_tokens:
            raise ValueError(f"batch of {T} tokens exceeds the model's {self.max_tokens}")
        s = stream or torch.cuda.current_stream(self.dev)
        pos = positions_of(rows)
        self.pos_copied.synchronize()   # the previous iteration's upload has left pos_host
        self.pos_host[:T].numpy()[:] = pos
        with torch.cuda.stream(s):
            self.pos[:T].copy_(self.pos_host[:T], non_blocking=True)
            self.pos_copied.record(s)
            x, h = self.x[:T], self.h[:T]
            torch.index_select(self.embed, 0, self.tokens[:T], out=x)
            qkv, q, k, v, attn = self.qkv[:T], self.q[:T], self.k[:T], self.v[:T], self.attn[:T]
            gu, act = self.gu[:T], self.act[:T]
            # every layer attends with the same rows: plan once, run per layer
            # (the plan is built once per iteration; only a workspace that is
            # too small costs a second planning, to learn the size)
            try:
                plan = cp.attn_prepare(self.desc, rows, self.ws, stream=s)
            except cp.CpError as e:
                if e.code != cp.CP_ERR_WORKSPACE:
                    raise
                self.ws = torch.empty(cp.workspace_bytes(self.desc, rows), dtype=torch.uint8,
                                      device=self.dev)
                plan = cp.attn_prepare(self.desc, rows, self.ws, stream=s)
            need = max(gemm_workspace_bytes(T, qkv.shape[1], c.hidden),
                       gemm_workspace_bytes(T, c.hidden, c.hq * c.head_dim)) if T > 32 else 0
            if need > self.ws_gemm.numel():
                self.ws_gemm = torch.empty(need, dtype=torch.uint8, device=self.dev)
            for L, kc, vc in zip(self.layers, self.kc, self.vc):
                rmsnorm(x, L["in_norm"], h, c.eps, s)
                project_attn(h, L["qkv"], qkv, None, s, self.ws_gemm)
                qkv_rope(qkv, L["q_norm"], L["k_norm"], self.pos, c.hq, c.hkv, c.head_dim,
                         c.theta, c.eps, q, k, v, s)
                cp.kv_append(self.desc, k, v, kc, vc, self.bt, rows, self.ws_append, stream=s)
                cp.attn_run(plan, q, kc, vc, self.bt, attn, self.ws, stream=s)
                project_attn(attn.view(T, c.hq * c.head_dim), L["o"], x, x, s, self.ws_gemm)
                rmsnorm(x, L["post_norm"], h, c.eps, s)
                project(h, L["gate_up"], gu, None, s)
                swiglu(gu, act, s)
                project(act, L["down"], x, x, s)
            if self.lm_head is None:
                return None
            last = torch.from_numpy(np.cumsum(rows[:, 2]).astype(np.int64) - 1)
            last = last[rows[:, 2] > 0].to(self.dev, non_blocking=True)
            hl = torch.empty(len(last), c.hidden, dtype=torch.bfloat16, device=self.dev)
            rmsnorm(x.index_select(0, last), self.final_norm, hl, c.eps, s)
            logits = torch.empty(len(last), c.vocab, dtype=torch.bfloat16, device=self.dev)
            project(hl, self.lm_head, logits, None, s)
            return torch.argmax(logits, dim=-1)


class ModelEngine:
    """StepEngine-compatible wrapper: one scheduler round = one model iteration."""

    def __init__(self, model: Model):
        import torch
        self.model = model
        self.max_tokens = model.max_tokens
        self.stream = torch.cuda.current_stream(model.dev)
        self.ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]

    def step(self, rows) -> float:
        rows = np.asarray(rows, dtype=np.int32).reshape(-1, 4)
        if int(rows[:, 2].sum()) == 0:
            return 0.0
        self.ev[0].record(self.stream)
        self.model.forward(rows, self.stream)
        self.ev[1].record(self.stream)
        self.ev[1].synchronize()
        return self.ev[0].elapsed_time(self.ev[1]) * 1e3
