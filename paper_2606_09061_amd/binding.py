"""ctypes binding of libcpattn.so: argument marshalling only.

Every step of the attention path runs in the library's HIP kernels; this
module turns torch tensors into device pointers, the row metadata into the
packed host array, and error codes into exceptions.  There is no fallback:
if the library is not built, every call raises.
"""

from __future__ import annotations

import ctypes
import os

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libcpattn.so")

CP_OK = 0
CP_ERR_INVALID_ARG = -1
CP_ERR_BAD_META = -2
CP_ERR_WORKSPACE = -3
CP_ERR_UNSUPPORTED = -4
CP_ERR_HIP = -5


class CpError(RuntimeError):
    def __init__(self, code, what):
        self.code = code
        super().__init__(f"{what}: {strerror(code)} ({code})")


class Desc(ctypes.Structure):
    """cp_attn_desc"""

    _fields_ = [
        ("num_q_heads", ctypes.c_int32),
        ("num_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("block_size", ctypes.c_int32),
        ("num_blocks", ctypes.c_int32),
        ("max_blocks_per_req", ctypes.c_int32),
        ("num_reqs_in_table", ctypes.c_int32),
        ("sm_scale", ctypes.c_float),
    ]


class AttnPlan(ctypes.Structure):
    """cp_attn_plan: a batch's attention plan, prepared once, run per layer."""

    _fields_ = [("desc", Desc), ("tokens", ctypes.c_int64), ("ws_bytes", ctypes.c_int64),
                ("n_prefill_items", ctypes.c_int32), ("n_prefill_wide_items", ctypes.c_int32),
                ("n_decode", ctypes.c_int32), ("n_merge", ctypes.c_int32)] + [
        (n, ctypes.c_int64) for n in ("off_prefill", "off_prefill_wide", "off_decode",
                                      "off_merge", "off_part_o", "off_part_lse",
                                      "partial_rows")] + [
        ("decode_in_prefill", ctypes.c_int32), ("reserved", ctypes.c_int32)]


_lib = None


def load():
    """Loads the built library; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(
            f"{LIB_PATH} is missing: build the HIP extension first "
            "(python -m paper_2606_09061_amd.build)")
    lib = ctypes.CDLL(LIB_PATH)
    vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    dp = ctypes.POINTER(Desc)
    lib.cp_version.argtypes, lib.cp_version.restype = [], ctypes.c_int
    lib.cp_strerror.argtypes, lib.cp_strerror.restype = [ctypes.c_int], ctypes.c_char_p
    lib.cp_workspace_bytes.argtypes, lib.cp_workspace_bytes.restype = [dp, vp, i32], sz
    lib.cp_check_batch.argtypes, lib.cp_check_batch.restype = [dp, vp, i32], ctypes.c_int
    lib.cp_check_block_tables.argtypes = [dp, vp, vp, i32]
    lib.cp_check_block_tables.restype = ctypes.c_int
    lib.cp_kv_append.argtypes = [dp, vp, vp, vp, vp, vp, vp, i32, vp, sz, vp]
    lib.cp_kv_append.restype = ctypes.c_int
    lib.cp_attn_mixed.argtypes = [dp, vp, vp, vp, vp, vp, i32, vp, vp, sz, vp]
    lib.cp_attn_mixed.restype = ctypes.c_int
    lib.cp_attn_prepare.argtypes = [dp, vp, i32, vp, sz, vp, vp]
    lib.cp_attn_prepare.restype = ctypes.c_int
    lib.cp_attn_run.argtypes = [vp, vp, vp, vp, vp, vp, vp, sz, vp]
    lib.cp_attn_run.restype = ctypes.c_int
    lib.cp_plan_summary.argtypes = [dp, vp, i32, vp]
    lib.cp_plan_summary.restype = ctypes.c_int
    lib.cp_plan_items.argtypes = [dp, vp, i32, vp, i64]
    lib.cp_plan_items.restype = i64
    lib.cp_step_mixed.argtypes = [dp, vp, vp, vp, vp, vp, vp, vp, i32, vp, vp, ctypes.c_size_t, vp]
    lib.cp_step_mixed.restype = ctypes.c_int
    lib.cp_plan_records.argtypes = [dp, vp, i32, i32, vp, i64]
    lib.cp_plan_records.restype = i64
    lib.cp_noalloc_init.argtypes, lib.cp_noalloc_init.restype = [], ctypes.c_int
    lib.cp_attn_mixed_noalloc.argtypes = [dp, vp, vp, vp, vp, vp, i32, vp, vp]
    lib.cp_attn_mixed_noalloc.restype = ctypes.c_int
    lib.cp_profile_begin.argtypes, lib.cp_profile_begin.restype = [], ctypes.c_int
    lib.cp_profile_end.argtypes, lib.cp_profile_end.restype = [vp, vp], ctypes.c_int
    _lib = lib
    return lib


def exported_symbols():
    return ["cp_version", "cp_strerror", "cp_workspace_bytes", "cp_check_batch",
            "cp_check_block_tables", "cp_kv_append",
            "cp_attn_mixed", "cp_attn_prepare", "cp_attn_run", "cp_plan_summary", "cp_plan_items",
            "cp_plan_records", "cp_step_mixed",
            "cp_noalloc_init", "cp_attn_mixed_noalloc", "cp_profile_begin", "cp_profile_end"]


def strerror(code: int) -> str:
    try:
        return load().cp_strerror(int(code)).decode()
    except RuntimeError:
        return f"code {code}"


def version() -> int:
    return load().cp_version()


def make_desc(num_q_heads, num_kv_heads, head_dim, block_size, num_blocks, max_blocks_per_req,
              num_reqs_in_table, sm_scale) -> Desc:
    return Desc(int(num_q_heads), int(num_kv_heads), int(head_dim), int(block_size),
                int(num_blocks), int(max_blocks_per_req), int(num_reqs_in_table), float(sm_scale))


def desc_for(batch) -> Desc:
    """Desc of a workloads.Batch-like object."""
    return make_desc(batch.num_q_heads, batch.num_kv_heads, batch.head_dim, batch.block_size,
                     batch.num_blocks, batch.max_blocks_per_req, batch.num_reqs_in_table,
                     batch.sm_scale)


def _rows(rows) -> np.ndarray:
    r = np.ascontiguousarray(rows, dtype=np.int32).reshape(-1, 4)
    return r


def _ptr(x):
    """Device/host pointer of a tensor, an int address or None."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def check_batch(desc: Desc, rows) -> int:
    r = _rows(rows)
    return load().cp_check_batch(ctypes.byref(desc), r.ctypes.data, r.shape[0])


def check_block_tables(desc: Desc, block_tables_host, rows) -> int:
    """cp_check_block_tables on a host copy of the table (numpy int32)."""
    r = _rows(rows)
    bt = np.ascontiguousarray(block_tables_host, dtype=np.int32)
    return load().cp_check_block_tables(ctypes.byref(desc), bt.ctypes.data, r.ctypes.data,
                                        r.shape[0])


def workspace_bytes(desc: Desc, rows) -> int:
    r = _rows(rows)
    n = load().cp_workspace_bytes(ctypes.byref(desc), r.ctypes.data, r.shape[0])
    if n == 0:
        raise CpError(check_batch(desc, rows), "cp_workspace_bytes")
    return int(n)


def kv_append(desc: Desc, k_new, v_new, k_cache, v_cache, block_tables, rows, ws, ws_bytes=None,
              stream=None) -> None:
    r = _rows(rows)
    nbytes = ws.numel() * ws.element_size() if ws_bytes is None else ws_bytes
    rc = load().cp_kv_append(ctypes.byref(desc), _ptr(k_new), _ptr(v_new), _ptr(k_cache),
                             _ptr(v_cache), _ptr(block_tables), r.ctypes.data, r.shape[0],
                             _ptr(ws), nbytes, _stream(stream))
    if rc != CP_OK:
        raise CpError(rc, "cp_kv_append")


def attn_mixed(desc: Desc, q, k_cache, v_cache, block_tables, rows, out, ws, ws_bytes=None,
               stream=None) -> None:
    r = _rows(rows)
    nbytes = ws.numel() * ws.element_size() if ws_bytes is None else ws_bytes
    rc = load().cp_attn_mixed(ctypes.byref(desc), _ptr(q), _ptr(k_cache), _ptr(v_cache),
                              _ptr(block_tables), r.ctypes.data, r.shape[0], _ptr(out), _ptr(ws),
                              nbytes, _stream(stream))
    if rc != CP_OK:
        raise CpError(rc, "cp_attn_mixed")


def step_mixed(desc: Desc, q, k_new, v_new, k_cache, v_cache, block_tables, rows, out, ws,
               ws_bytes=None, stream=None) -> None:
    """cp_step_mixed: kv_append then attn_mixed in one call (the attention
    plan's copy shares the append's launch)."""
    r = _rows(rows)
    nbytes = ws.numel() * ws.element_size() if ws_bytes is None else ws_bytes
    rc = load().cp_step_mixed(ctypes.byref(desc), _ptr(q), _ptr(k_new), _ptr(v_new),
                              _ptr(k_cache), _ptr(v_cache), _ptr(block_tables), r.ctypes.data,
                              r.shape[0], _ptr(out), _ptr(ws), nbytes, _stream(stream))
    if rc != CP_OK:
        raise CpError(rc, "cp_step_mixed")


def attn_prepare(desc: Desc, rows, ws, ws_bytes=None, stream=None) -> AttnPlan:
    """Plans the batch once and uploads the plan into ws (cp_attn_prepare)."""
    r = _rows(rows)
    nbytes = ws.numel() * ws.element_size() if ws_bytes is None else ws_bytes
    plan = AttnPlan()
    rc = load().cp_attn_prepare(ctypes.byref(desc), r.ctypes.data, r.shape[0], _ptr(ws), nbytes,
                                _stream(stream), ctypes.byref(plan))
    if rc != CP_OK:
        raise CpError(rc, "cp_attn_prepare")
    return plan


def attn_run(plan: AttnPlan, q, k_cache, v_cache, block_tables, out, ws, ws_bytes=None,
             stream=None) -> None:
    """cp_attn_mixed for a batch prepared by attn_prepare in the same workspace."""
    nbytes = ws.numel() * ws.element_size() if ws_bytes is None else ws_bytes
    rc = load().cp_attn_run(ctypes.byref(plan), _ptr(q), _ptr(k_cache), _ptr(v_cache),
                            _ptr(block_tables), _ptr(out), _ptr(ws), nbytes, _stream(stream))
    if rc != CP_OK:
        raise CpError(rc, "cp_attn_run")


NOALLOC_SCRATCH_BYTES = 64 << 20   # CP_NOALLOC_SCRATCH_BYTES
NOALLOC_PLAN_BYTES = 1 << 20       # CP_NOALLOC_PLAN_BYTES


def noalloc_init() -> None:
    """cp_noalloc_init on the current device."""
    rc = load().cp_noalloc_init()
    if rc != CP_OK:
        raise CpError(rc, "cp_noalloc_init")


def attn_mixed_noalloc(desc: Desc, q, k_cache, v_cache, block_tables, rows, out,
                       stream=None) -> None:
    """cp_attn_mixed_noalloc: cp_attn_mixed on the library's static scratch."""
    r = _rows(rows)
    rc = load().cp_attn_mixed_noalloc(ctypes.byref(desc), _ptr(q), _ptr(k_cache), _ptr(v_cache),
                                      _ptr(block_tables), r.ctypes.data, r.shape[0], _ptr(out),
                                      _stream(stream))
    if rc != CP_OK:
        raise CpError(rc, "cp_attn_mixed_noalloc")


def plan_summary(desc: Desc, rows) -> dict:
    r = _rows(rows)
    c = np.zeros(6, dtype=np.int64)
    rc = load().cp_plan_summary(ctypes.byref(desc), r.ctypes.data, r.shape[0], c.ctypes.data)
    if rc != CP_OK:
        raise CpError(rc, "cp_plan_summary")
    keys = ["prefill_items", "decode_items", "merge_groups", "partial_rows", "workspace_bytes",
            "decode_split_blocks"]
    return dict(zip(keys, (int(x) for x in c)))


def plan_records(desc: Desc, rows, which: int) -> np.ndarray:
    """[n, 8] int32: one prefill launch's records in dispatch order (which 0:
    128-row tiles, 1: 256-row tiles); columns tok0, n_tok, pos0, req, key
    begin, key end, part, kv head (n_tok 0: idle, -1: decode block)."""
    r = _rows(rows)
    lib = load()
    n = lib.cp_plan_records(ctypes.byref(desc), r.ctypes.data, r.shape[0], int(which), None, 0)
    if n < 0:
        raise CpError(int(n), "cp_plan_records")
    out = np.zeros((max(n, 1), 8), dtype=np.int32)
    n2 = lib.cp_plan_records(ctypes.byref(desc), r.ctypes.data, r.shape[0], int(which),
                             out.ctypes.data, n)
    assert n2 == n
    return out[:n]


def plan_items(desc: Desc, rows) -> np.ndarray:
    """[n, 8] int32: kind, tok0, n_tok, pos0, req, kv head, key begin, key end."""
    r = _rows(rows)
    lib = load()
    n = lib.cp_plan_items(ctypes.byref(desc), r.ctypes.data, r.shape[0], None, 0)
    if n < 0:
        raise CpError(int(n), "cp_plan_items")
    out = np.zeros((max(n, 1), 8), dtype=np.int32)
    n2 = lib.cp_plan_items(ctypes.byref(desc), r.ctypes.data, r.shape[0], out.ctypes.data, n)
    assert n2 == n
    return out[:n]


KERNEL_KINDS = ("append", "prefill", "decode", "merge")


def profile_begin() -> None:
    rc = load().cp_profile_begin()
    if rc != CP_OK:
        raise CpError(rc, "cp_profile_begin")


def profile_end() -> dict:
    """{kind: (total_ms, launches)} of the kernels launched since profile_begin()."""
    ms = np.zeros(4, dtype=np.float64)
    n = np.zeros(4, dtype=np.int64)
    rc = load().cp_profile_end(ms.ctypes.data, n.ctypes.data)
    if rc != CP_OK:
        raise CpError(rc, "cp_profile_end")
    return {k: (float(ms[i]), int(n[i])) for i, k in enumerate(KERNEL_KINDS)}
