"""ctypes binding of libretopk.so (include/retopk.h).

Argument marshalling only: every step of the decode path runs in the gfx950
kernels of the library.  Tensor arguments are torch tensors on the GPU (any
object with ``data_ptr()``) or raw device addresses; streams are torch streams,
raw ``hipStream_t`` values, or None for torch's current stream.
"""
from __future__ import annotations

import ctypes as C
import os

from . import build as _build

RETOPK_F32, RETOPK_BF16 = 0, 1
REUSE, FALLBACK, REFRESH, COLD = 0, 1, 2, 3
PATH_NAMES = {REUSE: "reuse", FALLBACK: "fallback", REFRESH: "refresh", COLD: "cold"}
STATUS = {0: "ok", -1: "invalid argument", -2: "unsupported shape", -3: "device out of memory",
          -4: "HIP runtime error", -5: "call out of order or handle broken",
          -6: "workspace larger than the fixed scratch"}

# Every symbol include/retopk.h declares.
EXPORTS = ("retopk_create", "retopk_destroy", "retopk_prefill_init", "retopk_decode_step",
           "exact_topk_attention", "exact_topk_attention_noalloc", "full_attention",
           "retopk_stream_read", "retopk_stats",
           "retopk_get_state",
           "retopk_set_state",
           "retopk_profile", "retopk_profile_read", "retopk_kernel_name",
           "retopk_status_string")


class RetopkError(RuntimeError):
    def __init__(self, fn: str, code: int, detail: str = ""):
        super().__init__(f"{fn}: {STATUS.get(code, code)} ({code})" + (f": {detail}" if detail else ""))
        self.code = code


def _check_tensor(fn: str, name: str, x, numel: int, itemsize: int):
    """A torch tensor argument must be on the GPU, contiguous, of the element size
    the call expects and at least as large as the layout the call indexes; the
    call is refused (RETOPK_ERR_ARG) before reaching the library otherwise.  Raw
    addresses (ints) and None pass unchecked."""
    if x is None or isinstance(x, int) or not hasattr(x, "is_cuda"):
        return
    if not x.is_cuda:
        raise RetopkError(fn, -1, f"{name} is not a GPU tensor")
    if not x.is_contiguous():
        raise RetopkError(fn, -1, f"{name} is not contiguous")
    if x.element_size() != itemsize:
        raise RetopkError(fn, -1, f"{name} has {x.element_size()}-byte elements, {itemsize} expected")
    if x.numel() < numel:
        raise RetopkError(fn, -1, f"{name} has {x.numel()} elements, {numel} expected")


class retopk_config(C.Structure):
    _fields_ = [("batch", C.c_int32), ("n_q_heads", C.c_int32), ("n_kv_heads", C.c_int32),
                ("head_dim", C.c_int32), ("max_len", C.c_int64), ("k", C.c_int32),
                ("cache_cap", C.c_int32), ("r", C.c_int32), ("window", C.c_int32),
                ("tau", C.c_float), ("refresh", C.c_int32), ("dtype", C.c_int32),
                ("retrieval", C.c_int32)]


class retopk_stats_t(C.Structure):
    _fields_ = [(n, C.c_uint64) for n in ("steps", "head_steps", "reuse", "fallback", "refresh",
                                          "cold", "kv_group_scans", "cand_sum", "cand_max")]


class retopk_debug(C.Structure):
    _fields_ = [("path", C.c_void_p), ("rho_max", C.c_void_p), ("retrieved", C.c_void_p),
                ("n_cand", C.c_void_p), ("cand", C.c_void_p)]


_LIB = None


def load(path: str | None = None):
    """Load the built library.  Raises if it has not been built: there is no
    fallback implementation.  The environment variable RETOPK_LIB names another
    build of it (the host-sanitizer test)."""
    global _LIB
    if _LIB is not None and path is None:
        return _LIB
    default = path is None
    path = path or os.environ.get("RETOPK_LIB") or _build.LIB
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with __graft_entry__.build() "
                           "(hipcc --offload-arch=gfx950)")
    lib = C.CDLL(path)
    P, I32, I64 = C.c_void_p, C.c_int32, C.c_int64
    sig = {
        "retopk_create": ([C.POINTER(retopk_config), C.POINTER(P)], C.c_int),
        "retopk_destroy": ([P], C.c_int),
        "retopk_prefill_init": ([P, P, I32, P, P, I64, P], C.c_int),
        "retopk_decode_step": ([P, P, P, P, I64, P, P, C.POINTER(retopk_debug), P], C.c_int),
        "exact_topk_attention": ([P, P, P, P, I64, P, P, P], C.c_int),
        "exact_topk_attention_noalloc": ([C.POINTER(retopk_config), P, P, P, I64, P, P, P],
                                         C.c_int),
        "full_attention": ([P, P, P, P, I64, P, P], C.c_int),
        "retopk_stream_read": ([P, I64, P, P], C.c_int),
        "retopk_stats": ([P, C.POINTER(retopk_stats_t)], C.c_int),
        "retopk_get_state": ([P, P, P, P, C.POINTER(I64), C.POINTER(I64)], C.c_int),
        "retopk_set_state": ([P, P, P, P, I64, I64], C.c_int),
        "retopk_profile": ([P, I32], C.c_int),
        "retopk_profile_read": ([P, I32, P, P], C.c_int),
        "retopk_kernel_name": ([I32], C.c_char_p),
        "retopk_status_string": ([C.c_int], C.c_char_p),
    }
    for name, (args, res) in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    if default:
        _LIB = lib
    return lib


def _addr(x):
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(s):
    if s is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(s, int):
        return s
    return s.cuda_stream


def _check(fn: str, rc: int):
    if rc != 0:
        raise RetopkError(fn, rc)


def make_config(batch, n_q_heads, n_kv_heads, head_dim, max_len, k, cache_cap, r, window, tau,
                refresh, dtype, retrieval=0) -> retopk_config:
    dt = {"f32": RETOPK_F32, "bf16": RETOPK_BF16}.get(dtype, dtype)
    return retopk_config(batch, n_q_heads, n_kv_heads, head_dim, max_len, k, cache_cap, r,
                         window, tau, refresh, dt, retrieval)


# ---------------------------------------------------------------------------
# Functions with the C names
# ---------------------------------------------------------------------------

def retopk_create(cfg: retopk_config) -> int:
    h = C.c_void_p()
    _check("retopk_create", load().retopk_create(C.byref(cfg), C.byref(h)))
    return h.value


def retopk_destroy(h: int) -> None:
    _check("retopk_destroy", load().retopk_destroy(h))


def retopk_prefill_init(h, q_tail, n, k, v, prefill_len, stream=None) -> None:
    _check("retopk_prefill_init", load().retopk_prefill_init(
        h, _addr(q_tail), n, _addr(k), _addr(v), prefill_len, _stream(stream)))


def retopk_decode_step(h, q, k, v, length, out, sel=None, dbg: dict | None = None,
                       stream=None) -> None:
    d = None
    if dbg is not None:
        d = retopk_debug(_addr(dbg.get("path")), _addr(dbg.get("rho_max")),
                         _addr(dbg.get("retrieved")), _addr(dbg.get("n_cand")),
                         _addr(dbg.get("cand")))
    _check("retopk_decode_step", load().retopk_decode_step(
        h, _addr(q), _addr(k), _addr(v), length, _addr(out), _addr(sel),
        C.byref(d) if d is not None else None, _stream(stream)))


def exact_topk_attention(h, q, k, v, length, out, sel=None, stream=None) -> None:
    _check("exact_topk_attention", load().exact_topk_attention(
        h, _addr(q), _addr(k), _addr(v), length, _addr(out), _addr(sel), _stream(stream)))


def exact_topk_attention_noalloc(cfg: retopk_config, q, k, v, length, out, sel=None,
                                 stream=None) -> None:
    """exact_topk_attention without a handle, on the library's fixed scratch."""
    _check_io("exact_topk_attention_noalloc", _cfg_dict(cfg), q=q, k=k, v=v, out=out, sel=sel)
    _check("exact_topk_attention_noalloc", load().exact_topk_attention_noalloc(
        C.byref(cfg), _addr(q), _addr(k), _addr(v), length, _addr(out), _addr(sel),
        _stream(stream)))


def full_attention(h, q, k, v, length, out, stream=None) -> None:
    _check("full_attention", load().full_attention(
        h, _addr(q), _addr(k), _addr(v), length, _addr(out), _stream(stream)))


def retopk_stream_read(src, nbytes: int, sink, stream=None) -> None:
    """Read nbytes at src once (the streaming-read ceiling; a measurement aid)."""
    _check("retopk_stream_read", load().retopk_stream_read(_addr(src), nbytes, _addr(sink),
                                                            _stream(stream)))


def retopk_stats(h) -> dict:
    st = retopk_stats_t()
    _check("retopk_stats", load().retopk_stats(h, C.byref(st)))
    return {n: int(getattr(st, n)) for n, _ in retopk_stats_t._fields_}


def retopk_get_state(h, qbar=None, supp=None, cnt=None):
    """Fills numpy arrays (host) and returns (n_inserted, t_dec)."""
    n_ins, t_dec = C.c_int64(), C.c_int64()
    P = lambda a: None if a is None else a.ctypes.data  # noqa: E731
    _check("retopk_get_state", load().retopk_get_state(h, P(qbar), P(supp), P(cnt),
                                                       C.byref(n_ins), C.byref(t_dec)))
    return n_ins.value, t_dec.value


def retopk_set_state(h, qbar, supp, cnt, n_inserted: int, t_dec: int) -> None:
    import numpy as np
    qbar = np.ascontiguousarray(qbar, np.float32)
    supp = np.ascontiguousarray(supp, np.int32)
    cnt = np.ascontiguousarray(cnt, np.int32)
    _check("retopk_set_state", load().retopk_set_state(
        h, qbar.ctypes.data, supp.ctypes.data, cnt.ctypes.data, n_inserted, t_dec))


def retopk_profile(h, enable: bool) -> None:
    _check("retopk_profile", load().retopk_profile(h, 1 if enable else 0))


def retopk_kernel_name(kid: int) -> str | None:
    r = load().retopk_kernel_name(kid)
    return r.decode() if r is not None else None


def retopk_profile_read(h) -> dict:
    """{kernel name: (launches, total ms)} over the recording window."""
    n = 0
    while retopk_kernel_name(n) is not None:
        n += 1
    launches = (C.c_uint64 * n)()
    ms = (C.c_double * n)()
    _check("retopk_profile_read", load().retopk_profile_read(h, n, launches, ms))
    return {retopk_kernel_name(i): (int(launches[i]), float(ms[i])) for i in range(n)}


def retopk_status_string(code: int) -> str:
    return load().retopk_status_string(code).decode()


def _cfg_dict(cfg: retopk_config) -> dict:
    return {n: getattr(cfg, n) for n, _ in retopk_config._fields_}


def _check_io(fn: str, c: dict, q=None, k=None, v=None, out=None, sel=None, q_tail=None,
              n_tail: int = 0):
    """Layout checks of the tensor arguments against the configuration c (see
    include/retopk.h: q [B, Hq, d], k and v [B, Hkv, max_len, d], out [B, Hq, d]
    float32, sel [B, Hq, K] int32, q_tail [B, Hq, n, d])."""
    dt = c["dtype"]
    es = 2 if dt in ("bf16", RETOPK_BF16) else 4
    bhq = c["batch"] * c["n_q_heads"]
    d = c["head_dim"]
    _check_tensor(fn, "q", q, bhq * d, es)
    kv = c["batch"] * c["n_kv_heads"] * c["max_len"] * d
    _check_tensor(fn, "k", k, kv, es)
    _check_tensor(fn, "v", v, kv, es)
    _check_tensor(fn, "out", out, bhq * d, 4)
    _check_tensor(fn, "sel", sel, bhq * c["k"], 4)
    _check_tensor(fn, "q_tail", q_tail, bhq * n_tail * d, es)


# ---------------------------------------------------------------------------
# Convenience wrapper
# ---------------------------------------------------------------------------

class Handle:
    """Owns one retopk handle.  Construct from keyword config fields."""

    def __init__(self, **cfg):
        self.cfg = dict(cfg)
        self.h = retopk_create(make_config(**cfg))

    def close(self):
        if self.h:
            retopk_destroy(self.h)
            self.h = None

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def prefill_init(self, q_tail, n, k, v, prefill_len, stream=None):
        _check_io("retopk_prefill_init", self.cfg, k=k, v=v, q_tail=q_tail, n_tail=n)
        retopk_prefill_init(self.h, q_tail, n, k, v, prefill_len, stream)

    def decode_step(self, q, k, v, length, out, sel=None, dbg=None, stream=None):
        _check_io("retopk_decode_step", self.cfg, q=q, k=k, v=v, out=out, sel=sel)
        retopk_decode_step(self.h, q, k, v, length, out, sel, dbg, stream)

    def exact(self, q, k, v, length, out, sel=None, stream=None):
        _check_io("exact_topk_attention", self.cfg, q=q, k=k, v=v, out=out, sel=sel)
        exact_topk_attention(self.h, q, k, v, length, out, sel, stream)

    def full(self, q, k, v, length, out, stream=None):
        _check_io("full_attention", self.cfg, q=q, k=k, v=v, out=out)
        full_attention(self.h, q, k, v, length, out, stream)

    def stats(self):
        return retopk_stats(self.h)

    def get_state(self):
        import numpy as np
        c = self.cfg
        bh = c["batch"] * c["n_q_heads"]
        qbar = np.zeros((bh, c["cache_cap"], c["head_dim"]), np.float32)
        supp = np.zeros((bh, c["cache_cap"], c["k"]), np.int32)
        cnt = np.zeros((bh, c["cache_cap"]), np.int32)
        n_ins, t_dec = retopk_get_state(self.h, qbar, supp, cnt)
        return dict(qbar=qbar, supp=supp, cnt=cnt, n_inserted=n_ins, t_dec=t_dec)

    def set_state(self, qbar, supp, cnt, n_inserted, t_dec):
        import numpy as np
        c = self.cfg
        bh = c["batch"] * c["n_q_heads"]
        want = {"qbar": (bh, c["cache_cap"], c["head_dim"]), "supp": (bh, c["cache_cap"], c["k"]),
                "cnt": (bh, c["cache_cap"])}
        for name, arr in (("qbar", qbar), ("supp", supp), ("cnt", cnt)):
            if tuple(np.shape(arr)) != want[name]:
                raise RetopkError("retopk_set_state", -1,
                                  f"{name} has shape {tuple(np.shape(arr))}, {want[name]} expected")
        retopk_set_state(self.h, qbar, supp, cnt, n_inserted, t_dec)

    def profile(self, enable=True):
        retopk_profile(self.h, enable)

    def profile_read(self):
        return retopk_profile_read(self.h)
