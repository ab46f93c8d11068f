"""fp64 CPU oracle for the mixed prefill/decode paged-attention step.

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, the smoke check and the
benchmark's CPU-baseline leg, never by the product library.  It shares no
code with the HIP path; both consume the seeded inputs of ``workloads``.

Two independent formulations live here:
  * ``cp_oracle.c`` (built into ``liboracle.so``): the per-(row, query, head)
    definition of paged causal attention in fp64, plus the paged append;
  * ``dense.py``: a dense-matrix brute force (gather the pages, build an
    explicit bottom-right causal mask, softmax) in numpy float64, used to pin
    the C oracle on tiny inputs.
"""

from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(_HERE, "cp_oracle.c")
LIB = os.path.join(_HERE, "liboracle.so")
CFLAGS = ["-O2", "-fopenmp", "-ffp-contract=off", "-std=c11", "-Wall", "-Wextra",
          "-shared", "-fPIC"]

_lib = None


def build(src=SRC, out=LIB, extra=()):
    """Compiles the oracle with gcc (no GPU code involved)."""
    cmd = ["gcc", *CFLAGS, *extra, src, "-o", out + ".tmp", "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


def _bind(lib):
    i32, f32, i64 = ctypes.c_int, ctypes.c_float, ctypes.c_int64
    vp = ctypes.c_void_p
    lib.oracle_kv_append.argtypes = [i32] * 6 + [vp] * 6 + [i32]
    lib.oracle_kv_append.restype = i32
    lib.oracle_attn.argtypes = [i32] * 7 + [f32] + [vp] * 5 + [i32, vp, i64, vp]
    lib.oracle_attn.restype = i32
    lib.oracle_num_threads.argtypes = []
    lib.oracle_num_threads.restype = i32
    lib.oracle_set_threads.argtypes = [i32]
    lib.oracle_set_threads.restype = None
    return lib


def load(path=None):
    """Loads liboracle.so, building it first if it is missing or stale."""
    global _lib
    if path is not None:
        return _bind(ctypes.CDLL(path))
    if _lib is None:
        if not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
            build()
        _lib = _bind(ctypes.CDLL(LIB))
    return _lib


def _u16(x):
    """bf16 tensor / uint16 array -> contiguous uint16 numpy view (raw bits)."""
    if hasattr(x, "detach"):
        import torch
        x = x.detach().to("cpu").contiguous().view(torch.int16).numpy()
    return np.ascontiguousarray(x).view(np.uint16)


def _ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p)


def kv_append(batch, k_new, v_new, k_cache, v_cache, lib=None, inplace=False):
    """Returns (k_cache, v_cache) uint16 arrays with the step's tokens written:
    new copies, or with ``inplace`` the given C-contiguous uint16 numpy arrays
    themselves (no copy of the pools)."""
    lib = lib or load()
    kn, vn = _u16(k_new), _u16(v_new)
    if inplace:
        for a in (k_cache, v_cache):
            if not (isinstance(a, np.ndarray) and a.dtype == np.uint16 and a.flags.c_contiguous):
                raise TypeError("inplace append needs C-contiguous uint16 numpy pools")
        kc, vc = k_cache, v_cache
    else:
        kc, vc = _u16(k_cache).copy(), _u16(v_cache).copy()
    bt = np.ascontiguousarray(batch.block_tables, dtype=np.int32)
    rows = np.ascontiguousarray(batch.rows, dtype=np.int32)
    rc = lib.oracle_kv_append(batch.num_kv_heads, batch.head_dim, batch.block_size,
                              batch.num_blocks, batch.num_reqs_in_table,
                              batch.max_blocks_per_req, _ptr(kn), _ptr(vn), _ptr(kc),
                              _ptr(vc), _ptr(bt), _ptr(rows), batch.n_rows)
    if rc != 0:
        raise ValueError(f"oracle_kv_append rejected the batch (code {rc})")
    return kc, vc


def attn(batch, q, k_cache, v_cache, sel=None, lib=None, sm_scale=None):
    """fp64 attention output: [T, Hq, D] or, with ``sel`` (flat t*Hq+h indices), [n_sel, D]."""
    lib = lib or load()
    qq, kc, vc = _u16(q), _u16(k_cache), _u16(v_cache)
    bt = np.ascontiguousarray(batch.block_tables, dtype=np.int32)
    rows = np.ascontiguousarray(batch.rows, dtype=np.int32)
    T, Hq, D = batch.num_tokens, batch.num_q_heads, batch.head_dim
    scale = batch.sm_scale if sm_scale is None else sm_scale
    if sel is None:
        out = np.empty((T, Hq, D), dtype=np.float64)
        sp, n_sel = None, 0
    else:
        sel = np.ascontiguousarray(sel, dtype=np.int64)
        out = np.empty((sel.size, D), dtype=np.float64)
        sp, n_sel = _ptr(sel), sel.size
    rc = lib.oracle_attn(Hq, batch.num_kv_heads, D, batch.block_size, batch.num_blocks,
                         batch.num_reqs_in_table, batch.max_blocks_per_req,
                         ctypes.c_float(scale), _ptr(qq), _ptr(kc), _ptr(vc), _ptr(bt),
                         _ptr(rows), batch.n_rows, sp, n_sel, _ptr(out))
    if rc != 0:
        raise ValueError(f"oracle_attn rejected the batch (code {rc})")
    return out


def num_threads(lib=None):
    return (lib or load()).oracle_num_threads()


def set_threads(n, lib=None):
    (lib or load()).oracle_set_threads(int(n))
