"""ctypes wrapper of the CPU oracle -- TEST INFRASTRUCTURE ONLY.

Arrays are numpy, float32 for tensors (bf16 inputs widened exactly) and int32
for indices.  The wrapper only marshals arguments; all arithmetic happens in
retopk_oracle.c.
"""
from __future__ import annotations

import ctypes as C
import os
from dataclasses import dataclass

import numpy as np

from . import build as _build

REUSE, FALLBACK, REFRESH, COLD = 0, 1, 2, 3
PATH_NAMES = {REUSE: "reuse", FALLBACK: "fallback", REFRESH: "refresh", COLD: "cold"}


class OrcConfig(C.Structure):
    _fields_ = [
        ("batch", C.c_int32), ("n_q_heads", C.c_int32), ("n_kv_heads", C.c_int32),
        ("head_dim", C.c_int32), ("max_len", C.c_int64), ("k", C.c_int32),
        ("cache_cap", C.c_int32), ("r", C.c_int32), ("window", C.c_int32),
        ("tau", C.c_float), ("refresh", C.c_int32), ("retrieval", C.c_int32),
    ]


class OrcInfo(C.Structure):
    _fields_ = [
        ("path", C.c_void_p), ("rho_max", C.c_void_p), ("retrieved", C.c_void_p),
        ("n_cand", C.c_void_p), ("cand", C.c_void_p), ("sel_score", C.c_void_p),
    ]


_LIB = None


def load(path: str | None = None):
    """Load (building first if needed) the oracle shared library.  The environment
    variable RETOPK_ORACLE_LIB names another build of it (the sanitizer test)."""
    global _LIB
    if path is None and _LIB is not None:
        return _LIB
    default = path is None
    path = path or os.environ.get("RETOPK_ORACLE_LIB") or _build.LIB
    if not os.path.exists(path) and path == _build.LIB:
        _build.build()
    lib = C.CDLL(path)
    P = C.c_void_p
    lib.orc_create.argtypes = [C.POINTER(OrcConfig), C.POINTER(P)]
    lib.orc_create.restype = C.c_int
    lib.orc_destroy.argtypes = [P]
    lib.orc_destroy.restype = None
    lib.orc_prefill_init.argtypes = [P, P, C.c_int32, P, P, C.c_int64, P]
    lib.orc_prefill_init.restype = C.c_int
    lib.orc_decode_step.argtypes = [P, P, P, P, C.c_int64, P, P, C.POINTER(OrcInfo), P]
    lib.orc_decode_step.restype = C.c_int
    lib.orc_exact.argtypes = [C.POINTER(OrcConfig), P, P, P, C.c_int64, P, P, P, P]
    lib.orc_exact.restype = C.c_int
    lib.orc_get_state.argtypes = [P, P, P, P, C.POINTER(C.c_int64), C.POINTER(C.c_int64)]
    lib.orc_get_state.restype = C.c_int
    lib.orc_set_state.argtypes = [P, P, P, P, C.c_int64, C.c_int64]
    lib.orc_set_state.restype = C.c_int
    lib.orc_scores.argtypes = [P, P, C.c_int32, C.c_int64, P, P]
    lib.orc_scores.restype = None
    lib.orc_normalize.argtypes = [P, C.c_int32, P]
    lib.orc_normalize.restype = None
    lib.orc_attend.argtypes = [P, P, P, C.c_int32, C.c_int64, P, P]
    lib.orc_attend.restype = None
    if default:
        _LIB = lib
    return lib


def _ptr(a: np.ndarray | None):
    if a is None:
        return None
    assert a.flags["C_CONTIGUOUS"], "oracle arrays must be C-contiguous"
    return a.ctypes.data


def _f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


@dataclass
class Params:
    batch: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    max_len: int
    k: int
    cache_cap: int
    r: int
    window: int
    tau: float
    refresh: int
    retrieval: int = 0     # 0: the R most similar entries (Eq. 7); 1: the R most recent

    def cstruct(self) -> OrcConfig:
        return OrcConfig(self.batch, self.n_q_heads, self.n_kv_heads, self.head_dim,
                         self.max_len, self.k, self.cache_cap, self.r, self.window,
                         self.tau, self.refresh, self.retrieval)

    @property
    def cand_cap(self) -> int:
        return self.r * self.k + self.window

    @property
    def heads(self) -> int:
        return self.batch * self.n_q_heads


@dataclass
class StepInfo:
    path: np.ndarray
    rho_max: np.ndarray
    retrieved: np.ndarray
    n_cand: np.ndarray
    cand: np.ndarray
    sel_score: np.ndarray


class Oracle:
    """Stateful ReTopK oracle over all (sequence, query head) pairs."""

    def __init__(self, p: Params, lib_path: str | None = None):
        self.p = p
        self.lib = load(lib_path)
        self._cfg = p.cstruct()
        h = C.c_void_p()
        rc = self.lib.orc_create(C.byref(self._cfg), C.byref(h))
        if rc != 0:
            raise ValueError(f"orc_create failed ({rc})")
        self.h = h

    def close(self):
        if self.h:
            self.lib.orc_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def prefill_init(self, q_tail, k, v, prefill_len: int, head_mask=None):
        q_tail, k, v = _f32(q_tail), _f32(k), _f32(v)
        mask = None if head_mask is None else np.ascontiguousarray(head_mask, dtype=np.uint8)
        rc = self.lib.orc_prefill_init(self.h, _ptr(q_tail), q_tail.shape[-2], _ptr(k), _ptr(v),
                                       prefill_len, _ptr(mask))
        if rc != 0:
            raise ValueError(f"orc_prefill_init failed ({rc})")

    def decode_step(self, q, k, v, length: int, head_mask=None):
        """Returns (out [B,Hq,d], sel [B,Hq,K], StepInfo)."""
        p = self.p
        q, k, v = _f32(q), _f32(k), _f32(v)
        out = np.zeros((p.batch, p.n_q_heads, p.head_dim), np.float32)
        sel = np.full((p.batch, p.n_q_heads, p.k), -1, np.int32)
        info = StepInfo(
            path=np.full(p.heads, -1, np.int8),
            rho_max=np.full(p.heads, np.nan, np.float64),
            retrieved=np.full((p.heads, p.r), -1, np.int32),
            n_cand=np.zeros(p.heads, np.int32),
            cand=np.full((p.heads, p.cand_cap), -1, np.int32),
            sel_score=np.full((p.heads, p.k), np.nan, np.float32),
        )
        ci = OrcInfo(_ptr(info.path), _ptr(info.rho_max), _ptr(info.retrieved),
                     _ptr(info.n_cand), _ptr(info.cand), _ptr(info.sel_score))
        mask = None if head_mask is None else np.ascontiguousarray(head_mask, dtype=np.uint8)
        rc = self.lib.orc_decode_step(self.h, _ptr(q), _ptr(k), _ptr(v), length, _ptr(out),
                                      _ptr(sel), C.byref(ci), _ptr(mask))
        if rc != 0:
            raise ValueError(f"orc_decode_step failed ({rc})")
        return out, sel, info

    def get_state(self):
        p = self.p
        e = p.heads * p.cache_cap
        qbar = np.zeros((p.heads, p.cache_cap, p.head_dim), np.float32)
        supp = np.zeros((p.heads, p.cache_cap, p.k), np.int32)
        cnt = np.zeros((p.heads, p.cache_cap), np.int32)
        n_ins, t_dec = C.c_int64(), C.c_int64()
        assert e >= 0
        self.lib.orc_get_state(self.h, _ptr(qbar), _ptr(supp), _ptr(cnt), C.byref(n_ins),
                               C.byref(t_dec))
        return dict(qbar=qbar, supp=supp, cnt=cnt, n_inserted=n_ins.value, t_dec=t_dec.value)

    def set_state(self, qbar, supp, cnt, n_inserted: int, t_dec: int):
        qbar = _f32(qbar)
        supp = np.ascontiguousarray(supp, dtype=np.int32)
        cnt = np.ascontiguousarray(cnt, dtype=np.int32)
        rc = self.lib.orc_set_state(self.h, _ptr(qbar), _ptr(supp), _ptr(cnt), n_inserted, t_dec)
        if rc != 0:
            raise ValueError(f"orc_set_state failed ({rc})")


def exact(p: Params, q, k, v, length: int, head_mask=None, lib_path: str | None = None):
    """Stateless Exact Top-K attention. Returns (out, sel, sel_score)."""
    lib = load(lib_path)
    q, k, v = _f32(q), _f32(k), _f32(v)
    out = np.zeros((p.batch, p.n_q_heads, p.head_dim), np.float32)
    sel = np.full((p.batch, p.n_q_heads, p.k), -1, np.int32)
    sc = np.full((p.batch, p.n_q_heads, p.k), np.nan, np.float32)
    mask = None if head_mask is None else np.ascontiguousarray(head_mask, dtype=np.uint8)
    cfg = p.cstruct()
    rc = lib.orc_exact(C.byref(cfg), _ptr(q), _ptr(k), _ptr(v), length, _ptr(out), _ptr(sel),
                       _ptr(sc), _ptr(mask))
    if rc != 0:
        raise ValueError(f"orc_exact failed ({rc})")
    return out, sel, sc


def scores(q, krows, idx, lib_path: str | None = None) -> np.ndarray:
    """Ranked fp32 scores of rows `idx` of krows [n, d] against q [d]."""
    lib = load(lib_path)
    q = _f32(q)
    krows = _f32(krows)
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    out = np.zeros(idx.shape[0], np.float32)
    lib.orc_scores(_ptr(q), _ptr(krows), q.shape[-1], idx.shape[0], _ptr(idx), _ptr(out))
    return out


def attend(q, krows, vrows, idx, lib_path: str | None = None) -> np.ndarray:
    """Eq. 10 + Eq. 12 over the index set `idx` (rows of krows/vrows [n, d])."""
    lib = load(lib_path)
    q, krows, vrows = _f32(q), _f32(krows), _f32(vrows)
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    out = np.zeros(q.shape[-1], np.float32)
    lib.orc_attend(_ptr(q), _ptr(krows), _ptr(vrows), q.shape[-1], idx.shape[0], _ptr(idx),
                   _ptr(out))
    return out


def normalize(q, lib_path: str | None = None) -> np.ndarray:
    lib = load(lib_path)
    q = _f32(q)
    out = np.zeros_like(q)
    lib.orc_normalize(_ptr(q), q.shape[-1], _ptr(out))
    return out
