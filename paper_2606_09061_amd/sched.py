"""ctypes binding of libcpsched.so (include/cp_sched.h): argument marshalling only.

The scheduler itself (Aging heap, Algorithm 1, APC rule, batch features and
the predictor's forward pass) runs in the C++ library; this module converts
numpy arrays and Python values and turns error codes into exceptions.
"""

from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libcpsched.so")

NUM_FEATURES = 16
FEATURES = (
    "prefill_tokens", "decode_tokens", "batch_request_count",
    "sum_decode_context_len", "max_decode_context_len",
    "prefill_processed_tokens", "max_prefill_processed_tokens",
    "gpu_mem_used_mb", "gpu_mem_free_mb", "cuda_allocated_mb", "cuda_reserved_mb",
    "bias", "scheduled_tokens", "avg_decode_ctx", "decode_ctx_interaction",
    "prefill_interaction",
)
POLICY_FCFS, POLICY_AGING = 0, 1
CHUNK_TOKEN_BUDGET, CHUNK_LPRS = 0, 1
APC_REASONS = ("accepted", "warm_start", "blocked_cap", "blocked_min_chunk")
_ERRORS = {-1: "invalid argument", -2: "capacity", -3: "no predictor loaded",
           -4: "call out of order", -5: "host allocation failed"}


class SchedError(RuntimeError):
    def __init__(self, code, what):
        self.code = code
        super().__init__(f"{what}: {_ERRORS.get(code, 'error')} ({code})")


class Config(ctypes.Structure):
    """cps_config"""

    _fields_ = [
        ("policy", ctypes.c_int32), ("alpha", ctypes.c_double), ("beta", ctypes.c_double),
        ("max_tokens", ctypes.c_int32), ("max_seqs", ctypes.c_int32),
        ("max_seq_len", ctypes.c_int32), ("chunking", ctypes.c_int32),
        ("target_us", ctypes.c_double), ("delta", ctypes.c_int32),
        ("lambda_u", ctypes.c_double), ("lambda_o", ctypes.c_double),
        ("apc", ctypes.c_int32), ("max_active", ctypes.c_int32), ("min_chunk", ctypes.c_int32),
    ]


class Stats(ctypes.Structure):
    """cps_stats"""

    _fields_ = [(n, ctypes.c_int64) for n in (
        "rounds", "decode_rows", "prefill_rows", "prefill_tokens", "lprs_calls",
        "predictor_rows", "apc_blocked_cap", "apc_blocked_min", "apc_warm_starts",
        "skipped_no_slot", "apc_not_scored", "finished")]


class RequestInfo(ctypes.Structure):
    """cps_request_info"""

    _fields_ = [("arrival", ctypes.c_double), ("first_token", ctypes.c_double),
                ("finish", ctypes.c_double)] + [
        (n, ctypes.c_int32) for n in ("prompt_len", "max_new_tokens", "processed", "generated",
                                      "chunks", "slot")]


_lib = None


def load():
    """Loads the built library; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it first "
                           "(python -m paper_2606_09061_amd.build)")
    lib = ctypes.CDLL(LIB_PATH)
    P, I32, I64, D = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_double
    sig = {
        "cps_create": (P, [P, P]),
        "cps_destroy": (None, [P]),
        "cps_set_predictor": (ctypes.c_int, [P, I32, P, P, P, P, P, D]),
        "cps_set_memory_state": (ctypes.c_int, [P, P]),
        "cps_add_request": (ctypes.c_int, [P, I64, D, I32, I32]),
        "cps_schedule": (ctypes.c_int, [P, D, P, P, I32, P, P]),
        "cps_complete": (ctypes.c_int, [P, D]),
        "cps_get_stats": (ctypes.c_int, [P, P]),
        "cps_request": (ctypes.c_int, [P, I64, P]),
        "cps_pending": (I64, [P]),
        "cps_batch_features": (ctypes.c_int, [P, I32, P, P]),
        "cps_predict": (ctypes.c_int, [P, P, I32, P]),
        "cps_select_chunk": (ctypes.c_int, [P, P, I32, I32, I32, I32, P, P]),
        "cps_apc_decide": (ctypes.c_int, [P, I32, I32, I32, I32, I32, I32, P, P]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _check(code, what):
    if code != 0:
        raise SchedError(code, what)


def _ptr(a):
    return a.ctypes.data if a is not None and a.size else None


def _rows(rows):
    r = np.ascontiguousarray(np.asarray(rows, dtype=np.int32).reshape(-1, 4))
    return r


def make_config(policy=POLICY_AGING, alpha=1.0, beta=-1.0 / 256.0, max_tokens=1024,
                max_seqs=256, max_seq_len=4096, chunking=CHUNK_TOKEN_BUDGET, target_us=0.0,
                delta=32, lambda_u=1.0, lambda_o=4.0, apc=False, max_active=4,
                min_chunk=32) -> Config:
    return Config(policy, alpha, beta, max_tokens, max_seqs, max_seq_len, chunking, target_us,
                  delta, lambda_u, lambda_o, int(bool(apc)), max_active, min_chunk)


def batch_features(rows, mem=(0.0, 0.0, 0.0, 0.0)) -> np.ndarray:
    """The 16 predictor inputs of one batch given as (req, start, len, ctx) rows."""
    r = _rows(rows)
    m = np.ascontiguousarray(mem, dtype=np.float64)
    out = np.zeros(NUM_FEATURES, dtype=np.float64)
    _check(load().cps_batch_features(_ptr(r), len(r), m.ctypes.data, out.ctypes.data),
           "cps_batch_features")
    return out


def apc_decide(cfg: Config, c_star, h, remaining, n_decode, n_active, committed):
    """Eq. 12–14 for one candidate: (chunk, reason name)."""
    c, why = ctypes.c_int32(), ctypes.c_int32()
    _check(load().cps_apc_decide(ctypes.byref(cfg), c_star, h, remaining, n_decode, n_active,
                                 committed, ctypes.byref(c), ctypes.byref(why)), "cps_apc_decide")
    return c.value, APC_REASONS[why.value]


@dataclass
class Round:
    rows: np.ndarray       # int32 [n, 4]: slot, chunk_start, chunk_len, ctx_len
    ids: np.ndarray        # int64 [n]: request ids
    n_decode: int


class Scheduler:
    """One cps_sched instance."""

    def __init__(self, cfg: Config):
        lib = load()
        err = ctypes.c_int(0)
        self.cfg = cfg
        self._h = lib.cps_create(ctypes.byref(cfg), ctypes.byref(err))
        if not self._h:
            raise SchedError(err.value, "cps_create")
        self._rows = np.zeros((max(cfg.max_seqs, 1), 4), dtype=np.int32)
        self._ids = np.zeros(max(cfg.max_seqs, 1), dtype=np.int64)

    def close(self):
        if getattr(self, "_h", None):
            load().cps_destroy(self._h)
            self._h = None

    __del__ = close

    def set_predictor(self, weights, x_mean, x_std, y_scale):
        """weights: [(W [out, in], b [out]), ...] of the MLP, first input 16, last output 1."""
        dims = np.array([weights[0][0].shape[1]] + [W.shape[0] for W, _ in weights], np.int32)
        w = np.ascontiguousarray(np.concatenate([np.asarray(W, np.float64).ravel() for W, _ in weights]))
        b = np.ascontiguousarray(np.concatenate([np.asarray(B, np.float64).ravel() for _, B in weights]))
        mu = np.ascontiguousarray(x_mean, dtype=np.float64)
        sd = np.ascontiguousarray(x_std, dtype=np.float64)
        _check(load().cps_set_predictor(self._h, len(weights), dims.ctypes.data, w.ctypes.data,
                                        b.ctypes.data, mu.ctypes.data, sd.ctypes.data,
                                        float(y_scale)), "cps_set_predictor")

    def set_memory_state(self, mem):
        m = np.ascontiguousarray(mem, dtype=np.float64)
        _check(load().cps_set_memory_state(self._h, m.ctypes.data), "cps_set_memory_state")

    def add_request(self, rid, arrival, prompt_len, max_new_tokens):
        _check(load().cps_add_request(self._h, int(rid), float(arrival), int(prompt_len),
                                      int(max_new_tokens)), "cps_add_request")

    def schedule(self, now) -> Round:
        n, nd = ctypes.c_int32(), ctypes.c_int32()
        _check(load().cps_schedule(self._h, float(now), self._rows.ctypes.data,
                                   self._ids.ctypes.data, len(self._ids), ctypes.byref(n),
                                   ctypes.byref(nd)), "cps_schedule")
        return Round(self._rows[:n.value].copy(), self._ids[:n.value].copy(), nd.value)

    def complete(self, now):
        _check(load().cps_complete(self._h, float(now)), "cps_complete")

    def stats(self) -> dict:
        s = Stats()
        _check(load().cps_get_stats(self._h, ctypes.byref(s)), "cps_get_stats")
        return {n: getattr(s, n) for n, _ in Stats._fields_}

    def request(self, rid) -> dict:
        r = RequestInfo()
        _check(load().cps_request(self._h, int(rid), ctypes.byref(r)), "cps_request")
        return {n: getattr(r, n) for n, _ in RequestInfo._fields_}

    def pending(self) -> int:
        return int(load().cps_pending(self._h))

    def predict(self, X) -> np.ndarray:
        x = np.ascontiguousarray(np.asarray(X, np.float64).reshape(-1, NUM_FEATURES))
        out = np.zeros(len(x), dtype=np.float64)
        _check(load().cps_predict(self._h, _ptr(x), len(x), _ptr(out)), "cps_predict")
        return out

    def select_chunk(self, committed, slot, processed, remaining):
        """Algorithm 1 for one candidate: (c*, predicted latency or nan)."""
        r = _rows(committed)
        c, t = ctypes.c_int32(), ctypes.c_double()
        _check(load().cps_select_chunk(self._h, _ptr(r), len(r), int(slot), int(processed),
                                       int(remaining), ctypes.byref(c), ctypes.byref(t)),
               "cps_select_chunk")
        return c.value, t.value
