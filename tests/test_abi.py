"""The C ABI library loads, exports every function include/retopk.h declares, and
rejects bad arguments on the host before touching a device (no GPU needed)."""
import ctypes as C
import os
import re

import pytest

from paper_2607_27692_amd import build as B
from paper_2607_27692_amd import retopk as R

HEADER = os.path.join(os.path.dirname(os.path.dirname(__file__)), "include", "retopk.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(B.LIB):
        B.build()
    return R.load()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b([a-z_]+)\s*\(", text)) - {"if", "sizeof"})


def test_header_and_binding_agree():
    assert declared_functions() == sorted(R.EXPORTS)


def test_every_declared_symbol_is_exported(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_status_strings(lib):
    for code in (0, -1, -2, -3, -4, -5, -6):
        assert R.retopk_status_string(code) == R.STATUS[code]
    assert [R.retopk_kernel_name(i) for i in range(8)] == [
        "retopk_sim", "retopk_score", "retopk_scan", "retopk_filter", "retopk_final",
        "dense_chunk", "dense_merge", "prefill_score"]
    assert R.retopk_kernel_name(8) is None and R.retopk_kernel_name(-1) is None


def _cfg(**kw):
    base = dict(batch=1, n_q_heads=32, n_kv_heads=8, head_dim=128, max_len=4096, k=256,
                cache_cap=256, r=4, window=128, tau=0.8, refresh=32, dtype="bf16")
    base.update(kw)
    return R.make_config(**base)


@pytest.mark.parametrize("bad, code", [
    (dict(batch=0), -1), (dict(n_q_heads=30), -1), (dict(n_kv_heads=0), -1),
    (dict(max_len=0), -1), (dict(max_len=1 << 31), -1), (dict(k=0), -1),
    (dict(cache_cap=-1), -1), (dict(r=0), -1), (dict(window=-1), -1), (dict(refresh=-1), -1),
    (dict(tau=float("nan")), -1), (dict(tau=float("inf")), -1), (dict(dtype=7), -1),
    (dict(retrieval=2), -1), (dict(retrieval=-1), -1),
    (dict(head_dim=96), -2), (dict(n_q_heads=32, n_kv_heads=2), -2), (dict(k=4096), -2),
    (dict(r=64), -2), (dict(cache_cap=8192), -2), (dict(max_len=(1 << 24) + 1), -2),
    (dict(batch=65), -2),
])
def test_create_rejects_bad_config(lib, bad, code):
    h = C.c_void_p()
    cfg = _cfg(**bad)
    assert lib.retopk_create(C.byref(cfg), C.byref(h)) == code
    assert h.value is None


def test_null_arguments(lib):
    assert lib.retopk_create(None, None) == -1
    assert lib.retopk_destroy(None) == 0
    assert lib.retopk_decode_step(None, 16, 16, 16, 1, 16, None, None, None) == -1
    assert lib.exact_topk_attention(None, 16, 16, 16, 1, 16, None, None) == -1
    assert lib.full_attention(None, 16, 16, 16, 1, 16, None) == -1
    # argument checks of the streaming read happen before any HIP call
    assert lib.retopk_stream_read(None, 16, 16, None) == -1
    assert lib.retopk_stream_read(16, 16, None, None) == -1
    assert lib.retopk_stream_read(16, 24, 16, None) == -1      # not a multiple of 16
    assert lib.retopk_stream_read(8, 16, 16, None) == -1       # not 16-byte aligned
    assert lib.retopk_stream_read(16, 0, 16, None) == -1
    assert lib.retopk_prefill_init(None, 16, 1, 16, 16, 1, None) == -1
    st = R.retopk_stats_t()
    assert lib.retopk_stats(None, C.byref(st)) == -1
    assert lib.retopk_profile(None, 1) == -1


def test_noalloc_entry_point_checks_on_the_host(lib):
    """exact_topk_attention_noalloc validates its configuration and arguments, and
    refuses a call whose workspace exceeds the fixed scratch, before any device
    work (no GPU needed)."""
    fn = lib.exact_topk_attention_noalloc
    ok = _cfg(max_len=131328)
    assert fn(None, 16, 16, 16, 1, 16, None, None) == -1                  # no config
    bad = _cfg(batch=0)
    assert fn(C.byref(bad), 16, 16, 16, 1, 16, None, None) == -1
    unsup = _cfg(head_dim=96)
    assert fn(C.byref(unsup), 16, 16, 16, 1, 16, None, None) == -2
    assert fn(C.byref(ok), None, 16, 16, 1, 16, None, None) == -1         # null q
    assert fn(C.byref(ok), 16, 16, 16, 1, None, None, None) == -1        # null out
    assert fn(C.byref(ok), 8, 16, 16, 1, 16, None, None) == -1           # misaligned q
    assert fn(C.byref(ok), 16, 16, 16, 0, 16, None, None) == -1          # len 0
    assert fn(C.byref(ok), 16, 16, 16, 131329, 16, None, None) == -1     # len > max_len
    # 128 heads at 64K (the 4-sequence layer) need about 108 MB of workspace
    big = _cfg(batch=4, max_len=65792)
    assert fn(C.byref(big), 16, 16, 16, 65792, 16, None, None) == -6
    # the same heads at 16K fit: that call would reach the device, so it is not made here
    assert R.retopk_status_string(-6) == R.STATUS[-6]


def test_noalloc_workspace_formula():
    """The workspace size documented in include/retopk.h for the fixed scratch: the
    128K layer of 32 query heads fits, the 4-sequence 64K layer does not."""
    def need(bh, length):
        r = 4096 * -(-length // 4096)
        parts = [bh * r * 4, bh * r * 8, bh * 8192, bh * (r // 4096) * 4, bh * 32]
        return sum(-(-p // 256) * 256 for p in parts)
    limit = 64 << 20
    assert need(32, 131328) <= limit < need(128, 65792)
    assert abs(need(32, 131328) / 1e6 - 52.2) < 0.1


class _FakeTensor:
    """Stands in for a torch tensor in the binding's argument checks."""
    def __init__(self, numel, itemsize, cuda=True, contiguous=True):
        self.is_cuda, self._n, self._i, self._c = cuda, numel, itemsize, contiguous

    def numel(self):
        return self._n

    def element_size(self):
        return self._i

    def is_contiguous(self):
        return self._c


def test_binding_checks_tensor_layouts():
    """The Python binding refuses tensors that are on the host, not contiguous, of the
    wrong element size or smaller than the layout the call indexes, before calling
    the library (RETOPK_ERR_ARG); raw addresses pass through to the library's own
    checks."""
    c = dict(batch=1, n_q_heads=4, n_kv_heads=2, head_dim=64, max_len=100, k=8, dtype="bf16")
    ok = dict(q=_FakeTensor(4 * 64, 2), k=_FakeTensor(2 * 100 * 64, 2),
              v=_FakeTensor(2 * 100 * 64, 2), out=_FakeTensor(4 * 64, 4), sel=_FakeTensor(32, 4))
    R._check_io("f", c, **ok)
    R._check_io("f", c, q=16, k=16, v=16, out=16, sel=None)     # raw addresses
    for name, bad in (("q", _FakeTensor(4 * 64, 2, cuda=False)),
                      ("k", _FakeTensor(2 * 100 * 64, 2, contiguous=False)),
                      ("v", _FakeTensor(2 * 100 * 64, 4)),
                      ("out", _FakeTensor(4 * 64 - 1, 4)),
                      ("sel", _FakeTensor(31, 4))):
        with pytest.raises(R.RetopkError) as e:
            R._check_io("f", c, **dict(ok, **{name: bad}))
        assert e.value.code == -1 and name in str(e.value)
    with pytest.raises(R.RetopkError):
        R._check_io("f", c, q_tail=_FakeTensor(4 * 3 * 64 - 1, 2), n_tail=3)
