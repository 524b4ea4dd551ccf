"""Argument and call-order errors of the C ABI on a live handle: they are caught on
the host before any kernel is launched, return the documented status and leave the
handle usable."""
import numpy as np
import pytest

from gpu_harness import handle_of, params_of, to_dev, torch_cuda
from paper_2607_27692_amd import retopk as R
from paper_2607_27692_amd.inputs import WORKLOADS, make_inputs

pytestmark = pytest.mark.gpu


def _status(exc):
    return exc.value.code


def test_errors_leave_the_handle_usable():
    torch = torch_cuda()
    w = WORKLOADS["tiny"]
    print("error paths", flush=True)
    inp = make_inputs(w)
    p = params_of(w)
    h = handle_of(p, w.dtype)
    q_tail, q_dec, k, v = (to_dev(inp.q_tail_raw), to_dev(inp.q_dec_raw), to_dev(inp.k_raw),
                           to_dev(inp.v_raw))
    out = torch.empty((w.batch, w.n_q_heads, w.head_dim), dtype=torch.float32, device="cuda")
    sel = torch.empty((w.batch, w.n_q_heads, w.k), dtype=torch.int32, device="cuda")
    with pytest.raises(R.RetopkError) as e:          # prefill longer than the KV allocation
        h.prefill_init(q_tail, w.cache_cap, k, v, w.max_len + 1)
    assert _status(e) == -1
    h.prefill_init(q_tail, w.cache_cap, k, v, w.prompt_len)
    h.decode_step(q_dec[0], k, v, w.step_len(0), out, sel)
    for bad_len in (0, w.max_len + 1):
        with pytest.raises(R.RetopkError) as e:
            h.decode_step(q_dec[1], k, v, bad_len, out, sel)
        assert _status(e) == -1
    with pytest.raises(R.RetopkError) as e:          # the context never shrinks
        h.decode_step(q_dec[1], k, v, w.step_len(0) - 1, out, sel)
    assert _status(e) == -5
    misaligned = out.view(-1)[1:]                    # a 4-byte offset
    with pytest.raises(R.RetopkError) as e:          # refused by the binding (too small)
        h.decode_step(q_dec[1], k, v, w.step_len(1), misaligned, sel)
    assert _status(e) == -1
    with pytest.raises(R.RetopkError) as e:          # and, as a raw address, by the library
        R.retopk_decode_step(h.h, q_dec[1], k, v, w.step_len(1), misaligned.data_ptr(), sel)
    assert _status(e) == -1
    with pytest.raises(R.RetopkError) as e:          # a host tensor never reaches the library
        h.decode_step(q_dec[1].cpu(), k, v, w.step_len(1), out, sel)
    assert _status(e) == -1
    with pytest.raises(R.RetopkError) as e:
        h.exact(q_dec[1], k, v, w.max_len + 1, out, sel)
    assert _status(e) == -1
    # the handle still steps: the rejected calls changed nothing
    before = h.stats()
    h.decode_step(q_dec[1], k, v, w.step_len(1), out, sel)
    torch.cuda.synchronize()
    after = h.stats()
    assert after["steps"] == before["steps"] + 1
    assert np.isfinite(out.cpu().numpy()).all()
    h.close()


def test_set_state_rejects_invalid_caches():
    """retopk_set_state checks every counted support index, every count and every q_bar
    value on the host: an invalid cache returns -1 and leaves the state as it was; a
    valid one is taken, and the handle steps from it as from the state it was read as."""
    torch = torch_cuda()
    w = WORKLOADS["tiny"]
    print("set_state validation", flush=True)
    inp = make_inputs(w)
    p = params_of(w)
    h = handle_of(p, w.dtype)
    q_tail, q_dec, k, v = (to_dev(inp.q_tail_raw), to_dev(inp.q_dec_raw), to_dev(inp.k_raw),
                           to_dev(inp.v_raw))
    out = torch.empty((w.batch, w.n_q_heads, w.head_dim), dtype=torch.float32, device="cuda")
    h.prefill_init(q_tail, w.cache_cap, k, v, w.prompt_len)
    h.decode_step(q_dec[0], k, v, w.step_len(0), out)
    st = h.get_state()
    good = (st["qbar"], st["supp"], st["cnt"], st["n_inserted"], st["t_dec"])

    def bad(field, edit, n_ins=st["n_inserted"], t_dec=st["t_dec"]):
        arrs = {key: st[key].copy() for key in ("qbar", "supp", "cnt")}
        if field:
            edit(arrs[field])
        with pytest.raises(R.RetopkError) as e:
            h.set_state(arrs["qbar"], arrs["supp"], arrs["cnt"], n_ins, t_dec)
        assert _status(e) == -1

    bad("cnt", lambda a: a.__setitem__((0, 3), w.k + 1))               # count above K
    bad("cnt", lambda a: a.__setitem__((0, 3), -1))                    # negative count
    bad("supp", lambda a: a.__setitem__((0, 5, 0), w.max_len))         # index past max_len
    bad("supp", lambda a: a.__setitem__((0, 5, 1), -7))                # negative counted index
    bad("qbar", lambda a: a.__setitem__((0, 2, 4), np.nan))            # non-finite q_bar
    bad(None, None, n_ins=-1)
    bad(None, None, t_dec=-1)
    after = h.get_state()                                              # unchanged
    for key in ("qbar", "supp", "cnt", "n_inserted", "t_dec"):
        assert np.array_equal(after[key], st[key])
    # the valid state is taken; stepping from it equals stepping on
    h.decode_step(q_dec[1], k, v, w.step_len(1), out)
    torch.cuda.synchronize()
    ref = out.cpu().numpy().copy()
    h.set_state(*good)
    h.decode_step(q_dec[1], k, v, w.step_len(1), out)
    torch.cuda.synchronize()
    assert np.array_equal(out.cpu().numpy(), ref)
    h.close()
