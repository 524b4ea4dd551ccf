"""exact_topk_attention_noalloc, the entry point for callers that cannot allocate
device memory, against exact_topk_attention on a handle: the same supports
(bit-exact) and outputs within the bf16 tolerance, on two calls in a row on the
library's fixed scratch, the second with a smaller input (fewer rows), so that
nothing the first call left in the scratch may reach the second's result.  The
first call is the 128K layer of 32 query heads on 8 KV heads (52 MB of the
scratch); its KV group 0 is also compared with the oracle."""
import numpy as np
import pytest

from gpu_harness import (OUT_TOL, Tally, check_output, check_selection, handle_of, params_of,
                         rel_err, to_dev, torch_cuda)
from oracle import oracle as O
from paper_2607_27692_amd.inputs import WORKLOADS, make_inputs

pytestmark = pytest.mark.gpu


def test_noalloc_matches_the_handle_entry_point():
    torch = torch_cuda()
    from paper_2607_27692_amd import retopk as R
    w = WORKLOADS["128k"]
    print(f"no-alloc exact {w.name}", flush=True)
    inp = make_inputs(w)
    p = params_of(w)
    q, k, v = to_dev(inp.q_dec_raw), to_dev(inp.k_raw), to_dev(inp.v_raw)
    cfg = R.make_config(batch=w.batch, n_q_heads=w.n_q_heads, n_kv_heads=w.n_kv_heads,
                        head_dim=w.head_dim, max_len=w.max_len, k=w.k, cache_cap=w.cache_cap,
                        r=w.r, window=w.window, tau=w.tau, refresh=w.refresh, dtype=w.dtype)
    h = handle_of(p, w.dtype)
    shape = (w.batch, w.n_q_heads, w.head_dim)
    out_a = torch.empty(shape, dtype=torch.float32, device="cuda")
    out_b = torch.empty(shape, dtype=torch.float32, device="cuda")
    sel_a = torch.empty((w.batch, w.n_q_heads, w.k), dtype=torch.int32, device="cuda")
    sel_b = torch.empty((w.batch, w.n_q_heads, w.k), dtype=torch.int32, device="cuda")
    # the full headline length, then a smaller ragged one (not a multiple of any tile)
    for t, length in ((0, w.step_len(0)), (1, 9001)):
        print(f"  call {t}: len {length}", flush=True)
        R.exact_topk_attention_noalloc(cfg, q[t], k, v, length, out_a, sel_a)
        h.exact(q[t], k, v, length, out_b, sel_b)
        torch.cuda.synchronize()
        ga, gb = sel_a.cpu().numpy(), sel_b.cpu().numpy()
        oa, ob = out_a.cpu().numpy(), out_b.cpu().numpy()
        assert np.array_equal(ga, gb), f"call {t}: supports differ"
        err = rel_err(oa, ob)
        print(f"  call {t}: supports equal, output error {err:.3g} "
              f"({'bitwise' if np.array_equal(oa, ob) else 'not bitwise'})", flush=True)
        assert err <= OUT_TOL[w.dtype]
        if t == 0:
            # KV group 0 against the oracle (the same bar as the exact-path tests)
            mask = np.zeros(p.heads, np.uint8)
            mask[:w.group] = 1
            kf, vf = inp.k, inp.v          # widened to fp32 once
            o_out, o_sel, _ = O.exact(p, inp.q_dec[t], kf, vf, length, head_mask=mask)
            tally = Tally()
            kr, vr = kf[0, 0, :length], vf[0, 0, :length]
            universe = np.arange(length, dtype=np.int32)
            for hh in range(w.group):
                qh = inp.q_dec[t][0, hh]
                us = O.scores(qh, kr, universe)
                g = check_selection(ga[0, hh], o_sel[0, hh], universe, us, f"head {hh}", tally)
                check_output(oa[0, hh], qh, kr, vr, g, o_out[0, hh],
                             np.array_equal(g, o_sel[0, hh][o_sel[0, hh] >= 0]), w.dtype,
                             f"head {hh}", tally)
            print(f"  oracle: {tally}", flush=True)
    h.close()
