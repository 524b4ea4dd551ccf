"""Pins of the CPU oracle against facts that do not come from the oracle itself.

Each test names the passage of the paper it follows.  Sources of truth used here:
hand-derived closed forms (tests/golden/hand_small.yaml), textbook special cases
(K >= len turns Exact Top-K attention into dense softmax attention, computed with
scipy), brute force on tiny inputs with numpy sorting and set algebra, and the
invariants the paper states (window inside the candidate set, candidate bound of
Eq. 14, exact recovery when the exact support lies in the candidates, FIFO cache).
"""
import math
import os

import numpy as np
import pytest
import scipy.special
import yaml

from oracle import oracle as O
from paper_2607_27692_amd.inputs import WORKLOADS, make_inputs

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "hand_small.yaml")
PATHS = {"reuse": O.REUSE, "fallback": O.FALLBACK, "refresh": O.REFRESH, "cold": O.COLD}


def _closed(expr: str) -> float:
    return float(eval(expr, {"__builtins__": {}}, {"e": math.e, "nan": math.nan}))


def _params(**kw) -> O.Params:
    base = dict(batch=1, n_q_heads=1, n_kv_heads=1, head_dim=4, max_len=6, k=2, cache_cap=3,
                r=1, window=1, tau=0.5, refresh=0)
    base.update(kw)
    return O.Params(**base)


@pytest.fixture(scope="module")
def golden():
    with open(GOLDEN) as f:
        return yaml.safe_load(f)


# ---------------------------------------------------------------------------
# Hand-derived worked examples
# ---------------------------------------------------------------------------

def test_golden_exact(oracle_lib, golden):
    """Eq. 1, Eq. 4, Eq. 12 on the hand-built case."""
    k = np.array(golden["keys"], np.float32)[None, None]
    v = np.array(golden["values"], np.float32)[None, None]
    q = np.array(golden["exact"]["q"], np.float32)[None, None]
    for case in golden["exact"]["cases"]:
        p = _params(k=case["k"])
        out, sel, _ = O.exact(p, q, k, v, 6)
        assert sel[0, 0].tolist() == case["sel"], case
        want = np.array([_closed(s) for s in case["out"]])
        np.testing.assert_allclose(out[0, 0], want, rtol=2e-7, atol=1e-7)


def test_golden_reuse(oracle_lib, golden):
    """Eq. 5-13 and the insertion rule of Sec. 3.4 on the hand-built state."""
    g = golden["reuse"]
    k = np.array(golden["keys"], np.float32)[None, None]
    v = np.array(golden["values"], np.float32)[None, None]
    for case in g["cases"]:
        p = _params(k=g["k"], cache_cap=g["cache_cap"], r=g["r"], window=g["window"],
                    tau=case["tau"], refresh=case["refresh"])
        orc = O.Oracle(p)
        qbar = np.array(g["state"]["qbar"], np.float32)[None]
        supp = np.array(g["state"]["supp"], np.int32)[None]
        cnt = np.full((1, g["cache_cap"]), g["k"], np.int32)
        orc.set_state(qbar, supp, cnt, g["state"]["n_inserted"], case["t_dec"])
        q = np.array(case["q"], np.float32)[None, None]
        out, sel, info = orc.decode_step(q, k, v, 6)
        name = case["name"]
        assert info.path[0] == PATHS[case["path"]], name
        rm = _closed(case["rho_max"])
        if math.isnan(rm):
            assert math.isnan(info.rho_max[0]), name
        else:
            assert abs(info.rho_max[0] - rm) < 1e-7, name
        nret = len(case["retrieved"])
        assert info.retrieved[0, :nret].tolist() == case["retrieved"], name
        assert (info.retrieved[0, nret:] == -1).all(), name
        assert info.n_cand[0] == len(case["cand"]), name
        assert info.cand[0, :len(case["cand"])].tolist() == case["cand"], name
        assert sel[0, 0].tolist() == case["sel"], name
        want = np.array([_closed(s) for s in case["out"]])
        np.testing.assert_allclose(out[0, 0], want, rtol=2e-7, atol=1e-7, err_msg=name)
        st = orc.get_state()
        slot = case["insert_slot"]
        qn = np.array(case["q"], np.float64)
        np.testing.assert_allclose(st["qbar"][0, slot], qn / np.linalg.norm(qn), rtol=1e-7)
        assert st["supp"][0, slot].tolist() == case["sel"], name
        assert st["n_inserted"] == g["state"]["n_inserted"] + 1
        assert st["t_dec"] == case["t_dec"] + 1
        orc.close()


# ---------------------------------------------------------------------------
# Exact Top-K: textbook special cases and brute force
# ---------------------------------------------------------------------------

def _rand_case(rng, B, Hq, Hkv, d, L, integer=False):
    shape_q = (B, Hq, d)
    shape_kv = (B, Hkv, L, d)
    if integer:
        q = rng.integers(-2, 3, shape_q).astype(np.float32)
        k = rng.integers(-2, 3, shape_kv).astype(np.float32)
    else:
        q = rng.standard_normal(shape_q).astype(np.float32)
        k = rng.standard_normal(shape_kv).astype(np.float32)
    v = rng.standard_normal(shape_kv).astype(np.float32)
    return q, k, v


@pytest.mark.parametrize("B,Hq,Hkv,d,L", [(1, 1, 1, 8, 5), (2, 4, 2, 16, 33), (1, 6, 3, 64, 70)])
def test_dense_limit(oracle_lib, B, Hq, Hkv, d, L):
    """K >= len: Exact Top-K attention is dense softmax attention (Eq. 12 over every key)."""
    rng = np.random.default_rng(1)
    q, k, v = _rand_case(rng, B, Hq, Hkv, d, L)
    for K in (L, L + 7):
        p = _params(batch=B, n_q_heads=Hq, n_kv_heads=Hkv, head_dim=d, max_len=L, k=K)
        out, sel, _ = O.exact(p, q, k, v, L)
        G = Hq // Hkv
        for b in range(B):
            for h in range(Hq):
                s = (k[b, h // G].astype(np.float64) @ q[b, h].astype(np.float64)) / math.sqrt(d)
                dense = scipy.special.softmax(s) @ v[b, h // G].astype(np.float64)
                np.testing.assert_allclose(out[b, h], dense, rtol=1e-5, atol=1e-6)
                assert sel[b, h, :L].tolist() == list(range(L))
                assert (sel[b, h, L:] == -1).all()


@pytest.mark.parametrize("integer", [False, True])
def test_exact_bruteforce(oracle_lib, integer):
    """Eq. 1: the K largest scores, ties to the lower index (numpy lexsort brute force).
    Integer-valued inputs force many exact ties at the K-th boundary."""
    rng = np.random.default_rng(2 + integer)
    for trial in range(12):
        B, Hkv, G = 1 + trial % 2, 1 + trial % 3, 1 + (trial // 3) % 2
        Hq, d = Hkv * G, (4, 8, 64)[trial % 3]
        L = int(rng.integers(1, 90))
        K = int(rng.integers(1, 40))
        q, k, v = _rand_case(rng, B, Hq, Hkv, d, L, integer)
        p = _params(batch=B, n_q_heads=Hq, n_kv_heads=Hkv, head_dim=d, max_len=L, k=K)
        out, sel, sc = O.exact(p, q, k, v, L)
        for b in range(B):
            for h in range(Hq):
                kk = k[b, h // G].astype(np.float64)
                dots = (kk @ q[b, h].astype(np.float64)).astype(np.float32)
                s = dots * np.float32(1 / math.sqrt(d))
                order = np.lexsort((np.arange(L), -s.astype(np.float64)))
                top = np.sort(order[:min(K, L)])
                assert sel[b, h, :len(top)].tolist() == top.tolist()
                assert (sel[b, h, len(top):] == -1).all()
                np.testing.assert_array_equal(sc[b, h, :len(top)], s[top])
                w = scipy.special.softmax(s[top].astype(np.float64))
                np.testing.assert_allclose(out[b, h], w @ v[b, h // G][top].astype(np.float64),
                                           rtol=1e-5, atol=1e-6)


def test_all_equal_scores_take_lowest_indices(oracle_lib):
    """Tie-break (score desc, index asc): identical keys select indices 0..K-1."""
    L, d, K = 50, 8, 7
    k = np.ones((1, 1, L, d), np.float32)
    v = np.arange(L * d, dtype=np.float32).reshape(1, 1, L, d)
    q = np.ones((1, 1, d), np.float32)
    p = _params(head_dim=d, max_len=L, k=K)
    out, sel, _ = O.exact(p, q, k, v, L)
    assert sel[0, 0].tolist() == list(range(K))
    np.testing.assert_allclose(out[0, 0], v[0, 0, :K].mean(0), rtol=1e-6)


def test_negative_zero_ties_positive_zero(oracle_lib):
    """A -0.0 score ranks equal to +0.0, so the lower index wins."""
    d = 4
    k = np.array([[0, 0, 0, 0], [-1, 0, 0, 0], [1, 0, 0, 0]], np.float32)[None, None]
    q = np.array([0, 1, 0, 0], np.float32)[None, None]           # all scores are +-0
    k[0, 0, 1, 1] = -0.0
    v = np.eye(3, 4, dtype=np.float32)[None, None]
    p = _params(head_dim=d, max_len=3, k=1)
    _, sel, _ = O.exact(p, q, k, v, 3)
    assert sel[0, 0].tolist() == [0]
    q2 = np.array([-1, 0, 0, 0], np.float32)[None, None]         # scores 0, 0.5, -0.5
    _, sel2, _ = O.exact(_params(head_dim=d, max_len=3, k=2), q2, k, v, 3)
    assert sel2[0, 0].tolist() == [0, 1]


def test_one_hot_values_expose_weights(oracle_lib):
    """With v_i = e_i the output is the weight vector of Eq. 12: zero outside the
    support, positive on it, summing to 1, with ratios exp(s_i - s_j)."""
    rng = np.random.default_rng(4)
    L, K = 40, 9
    d = L
    k = rng.standard_normal((1, 1, L, d)).astype(np.float32)
    q = rng.standard_normal((1, 1, d)).astype(np.float32)
    v = np.eye(L, dtype=np.float32)[None, None]
    p = _params(head_dim=d, max_len=L, k=K)
    out, sel, sc = O.exact(p, q, k, v, L)
    w = out[0, 0].astype(np.float64)
    chosen = sel[0, 0]
    mask = np.zeros(L, bool)
    mask[chosen] = True
    assert (w[~mask] == 0).all() and (w[mask] > 0).all()
    assert abs(w.sum() - 1) < 1e-6
    s = sc[0, 0].astype(np.float64)
    for a in range(1, K):
        assert abs(math.log(w[chosen[a]] / w[chosen[0]]) - (s[a] - s[0])) < 1e-5


@pytest.mark.parametrize("Hq, Hkv", [(4, 2), (14, 2), (9, 3)])
def test_gqa_head_mapping(oracle_lib, Hq, Hkv):
    """Query head h reads KV head h // (Hq / Hkv): zero keys and constant values in the
    last KV head make exactly its G query heads return that constant (G = 2, and the
    group sizes 7 and 3 that are not powers of two)."""
    rng = np.random.default_rng(5)
    B, d, L = 1, 8, 20
    G = Hq // Hkv
    q, k, v = _rand_case(rng, B, Hq, Hkv, d, L)
    k[0, Hkv - 1] = 0
    v[0, Hkv - 1] = 3.25
    p = _params(batch=B, n_q_heads=Hq, n_kv_heads=Hkv, head_dim=d, max_len=L, k=5)
    out, sel, _ = O.exact(p, q, k, v, L)
    np.testing.assert_array_equal(out[0, Hq - G:], 3.25)
    for h in range(Hq - G, Hq):
        assert sel[0, h].tolist() == [0, 1, 2, 3, 4]
    for h in range(Hq - G):
        assert not np.allclose(out[0, h], 3.25)


# ---------------------------------------------------------------------------
# Trajectory on the small workload: invariants and brute force per step
# ---------------------------------------------------------------------------

def _workload_params(w, **kw) -> O.Params:
    base = dict(batch=w.batch, n_q_heads=w.n_q_heads, n_kv_heads=w.n_kv_heads,
                head_dim=w.head_dim, max_len=w.max_len, k=w.k, cache_cap=w.cache_cap, r=w.r,
                window=w.window, tau=w.tau, refresh=w.refresh)
    base.update(kw)
    return O.Params(**base)


@pytest.fixture(scope="module")
def tiny():
    return make_inputs(WORKLOADS["tiny"])


def _run(w, inp, p, n_steps=None, prefill=True, check=None):
    orc = O.Oracle(p)
    if prefill:
        orc.prefill_init(inp.q_tail, inp.k, inp.v, w.prompt_len)
    rows = []
    for t in range(n_steps or w.steps):
        before = orc.get_state() if check else None
        out, sel, info = orc.decode_step(inp.q_dec[t], inp.k, inp.v, w.step_len(t))
        rows.append((out, sel, info))
        if check:
            check(t, before, out, sel, info)
    return orc, rows


def test_prefill_inserts_causal_exact_supports(oracle_lib, tiny):
    """Sec. 3.3: the cache starts from the final C prompt queries, each with its exact
    support over its causal prefix, in FIFO order."""
    w = tiny.w
    p = _workload_params(w)
    orc = O.Oracle(p)
    orc.prefill_init(tiny.q_tail, tiny.k, tiny.v, w.prompt_len)
    st = orc.get_state()
    assert st["n_inserted"] == w.cache_cap and st["t_dec"] == 0
    for u in range(0, w.cache_cap, 7):
        pos = w.prompt_len - w.cache_cap + u
        q = tiny.q_tail[:, :, u]
        _, sel, _ = O.exact(p, q, tiny.k, tiny.v, pos + 1)
        assert st["supp"][0, u].tolist() == sel[0, 0].tolist()
        qn = q[0, 0].astype(np.float64)
        np.testing.assert_allclose(st["qbar"][0, u], qn / np.linalg.norm(qn), rtol=2e-7,
                                   atol=1e-8)


def test_trajectory_invariants(oracle_lib, tiny):
    """Per reuse step: Eq. 8 window inside the candidates, Eq. 14 bound, candidates
    equal the brute-force union of the retrieved supports (Eq. 9), Top-R equals the
    brute-force ranking of cosine similarities (Eq. 6, Eq. 7), the rerank equals a
    brute-force Top-K over the candidates (Eq. 11), exact recovery when the exact
    support lies inside the candidates (Sec. 3.3), and every output is a convex
    combination of the selected value rows (Eq. 12)."""
    w = tiny.w
    p = _workload_params(w)
    G = w.group
    seen = {"reuse": 0, "fallback": 0, "refresh": 0}

    def check(t, before, out, sel, info):
        L = w.step_len(t)
        path = int(info.path[0])
        q = tiny.q_dec[t][0, 0]
        kk = tiny.k[0, 0 // G][:L].astype(np.float64)
        vv = tiny.v[0, 0 // G][:L]
        chosen = sel[0, 0][sel[0, 0] >= 0]
        assert len(chosen) == min(w.k, L if path != O.REUSE else info.n_cand[0])
        assert (np.diff(chosen) > 0).all()
        # convex combination of the selected rows
        lo, hi = vv[chosen].min(0), vv[chosen].max(0)
        assert (out[0, 0] >= lo - 1e-6).all() and (out[0, 0] <= hi + 1e-6).all()
        s_all = (kk @ q.astype(np.float64)).astype(np.float32) * np.float32(1 / math.sqrt(w.head_dim))
        exact_top = np.sort(np.lexsort((np.arange(L), -s_all.astype(np.float64)))[:w.k])
        if path != O.REUSE:
            assert chosen.tolist() == exact_top.tolist()
            if path == O.REFRESH:
                seen["refresh"] += 1
            else:
                seen["fallback"] += 1
            return
        seen["reuse"] += 1
        n = int(info.n_cand[0])
        cand = info.cand[0, :n]
        assert (info.cand[0, n:] == -1).all()
        assert n <= w.r * w.k + w.window
        assert (np.diff(cand) > 0).all() and cand[0] >= 0 and cand[-1] < L
        window = np.arange(max(0, L - w.window), L)
        assert np.isin(window, cand).all()
        # Top-R by brute force over the cached normalised queries
        nv = min(before["n_inserted"], w.cache_cap)
        qb = q.astype(np.float64) / np.linalg.norm(q.astype(np.float64))
        rho = before["qbar"][0, :nv].astype(np.float64) @ qb
        age = (before["n_inserted"] - 1 - np.arange(nv)) % w.cache_cap
        ret = np.lexsort((age, -rho))[:min(w.r, nv)]
        assert abs(info.rho_max[0] - rho.max()) < 1e-6
        gaps = np.abs(rho[:, None] - rho[None, :]) + np.eye(nv)
        if gaps.min() > 1e-6:   # no near-tie anywhere: the ranking is unambiguous
            assert info.retrieved[0, :len(ret)].tolist() == ret.tolist()
        # Union of the retrieved supports and the window
        r_slots = info.retrieved[0][info.retrieved[0] >= 0]
        union = set(window.tolist())
        for s in r_slots:
            union.update(before["supp"][0, s, :before["cnt"][0, s]].tolist())
        assert cand.tolist() == sorted(union)
        # Rerank: brute-force Top-K over the candidates
        sc = s_all[cand]
        top = np.sort(cand[np.lexsort((cand, -sc.astype(np.float64)))[:w.k]])
        assert chosen.tolist() == top.tolist()
        # Exact recovery
        if np.isin(exact_top, cand).all():
            assert chosen.tolist() == exact_top.tolist()

    _run(w, tiny, p, check=check)
    assert seen["reuse"] > 10 and seen["fallback"] > 0 and seen["refresh"] == (w.steps - 1) // w.refresh


def test_exact_recovery(oracle_lib, tiny):
    """Sec. 3.3: if the exact support lies inside the candidate set, the rerank returns
    exactly that support.  The cache is built so that slot 0 holds the current query
    with its exact support; the step then reuses it and must reproduce Exact Top-K
    bit for bit.  Dropping one support index that the window does not cover must
    change the result."""
    w = tiny.w
    p = _workload_params(w)
    rng = np.random.default_rng(11)
    C, K = w.cache_cap, w.k
    for t in (0, 9, 33, 63):
        L = w.step_len(t)
        q = tiny.q_dec[t]
        out_e, sel_e, _ = O.exact(p, q, tiny.k, tiny.v, L)
        qbar = rng.standard_normal((1, C, w.head_dim)).astype(np.float32)
        qbar /= np.linalg.norm(qbar, axis=-1, keepdims=True)
        supp = np.sort(rng.integers(0, L - w.window, (1, C, K)), axis=-1).astype(np.int32)
        qbar[0, 0] = O.normalize(q[0, 0])
        supp[0, 0] = sel_e[0, 0]
        cnt = np.full((1, C), K, np.int32)
        orc = O.Oracle(p)
        orc.set_state(qbar, supp, cnt, C, 1)
        out, sel, info = orc.decode_step(q, tiny.k, tiny.v, L)
        assert info.path[0] == O.REUSE and info.retrieved[0, 0] == 0
        np.testing.assert_array_equal(sel, sel_e)
        np.testing.assert_array_equal(out, out_e)
        outside = [i for i in sel_e[0, 0] if i < L - w.window]
        if outside:
            drop = outside[0]
            keep = [i for i in sel_e[0, 0] if i != drop]
            supp[0, 0] = np.array(keep + [keep[-1]], np.int32)
            cnt[0, 0] = K - 1
            supp[0, 1:] = np.minimum(supp[0, 1:], 0)     # other slots cover only key 0
            cnt[0, 1:] = 1
            orc2 = O.Oracle(p)
            orc2.set_state(qbar, supp, cnt, C, 1)
            _, sel2, _ = orc2.decode_step(q, tiny.k, tiny.v, L)
            assert drop not in sel2[0, 0].tolist()


def test_fifo_holds_last_entries(oracle_lib, tiny):
    """Eq. 5 (bounded FIFO of capacity C) with insertion after every step (Sec. 3.4):
    after n > C inserts slot s holds insert j with j = s (mod C), the latest such."""
    w = tiny.w.with_(cache_cap=8)
    p = _workload_params(w, tau=1.5)       # every step exact, so each insert is known
    orc = O.Oracle(p)
    sels = []
    n = 21
    for t in range(n):
        _, sel, _ = orc.decode_step(tiny.q_dec[t], tiny.k, tiny.v, w.step_len(t))
        sels.append(sel[0, 0].copy())
    st = orc.get_state()
    assert st["n_inserted"] == n
    for s in range(8):
        j = max(j for j in range(n) if j % 8 == s)
        assert st["supp"][0, s].tolist() == sels[j].tolist()
        qn = tiny.q_dec[j][0, 0].astype(np.float64)
        np.testing.assert_allclose(st["qbar"][0, s], qn / np.linalg.norm(qn), rtol=2e-7, atol=1e-8)


def test_forced_fallback_equals_exact(oracle_lib, tiny):
    """tau > 1 (no cosine reaches it): every step takes the exact path, so ReTopK is
    Exact Top-K attention step for step (Eq. 13)."""
    w = tiny.w
    p = _workload_params(w, tau=1.5)
    _, rows = _run(w, tiny, p, n_steps=20)
    for t, (out, sel, info) in enumerate(rows):
        assert info.path[0] in (O.FALLBACK, O.REFRESH)
        out_e, sel_e, _ = O.exact(p, tiny.q_dec[t], tiny.k, tiny.v, w.step_len(t))
        np.testing.assert_array_equal(sel, sel_e)
        np.testing.assert_array_equal(out, out_e)


def test_zero_capacity_is_always_cold_exact(oracle_lib, tiny):
    """C = 0 (no cache): every step is a cold exact step."""
    w = tiny.w
    p = _workload_params(w, cache_cap=0)
    _, rows = _run(w, tiny, p, n_steps=10)
    for t, (out, sel, info) in enumerate(rows):
        assert info.path[0] == O.COLD
        out_e, sel_e, _ = O.exact(p, tiny.q_dec[t], tiny.k, tiny.v, w.step_len(t))
        np.testing.assert_array_equal(sel, sel_e)
        np.testing.assert_array_equal(out, out_e)


def test_no_fallback_when_tau_is_minus_one(oracle_lib, tiny):
    """tau = -1 disables the similarity fallback (Tab. 3); only refreshes are exact."""
    w = tiny.w
    p = _workload_params(w, tau=-1.0)
    _, rows = _run(w, tiny, p)
    paths = [int(r[2].path[0]) for r in rows]
    assert O.FALLBACK not in paths
    assert paths.count(O.REFRESH) == (w.steps - 1) // w.refresh


@pytest.mark.parametrize("P", [0, 1, 2, 5, 16])
def test_refresh_schedule(oracle_lib, tiny, P):
    """Eq. 13: refresh at t_dec in {T_r, 2T_r, ...}, none when T_r = 0; with a 0-based
    t_dec that is floor((T-1)/T_r) refreshes in T steps."""
    w = tiny.w
    p = _workload_params(w, tau=-1.0, refresh=P)
    _, rows = _run(w, tiny, p, n_steps=33)
    got = [t for t, r in enumerate(rows) if r[2].path[0] == O.REFRESH]
    want = [t for t in range(33) if P > 0 and t > 0 and t % P == 0]
    assert got == want
    assert len(got) == (0 if P == 0 else (33 - 1) // P)


def test_refresh_share_matches_paper_path_mix(oracle_lib):
    """The paper's path mix (Sec. 4.2, operator breakdown) reports reuse + fallback of
    87.5 + 11.9 = 99.4 % at 16K and 88.9 + 10.5 = 99.4 % at 128K over 512 decode
    steps with T_r = 128: refreshes are 0.6 % of steps.  With refresh at t_dec =
    128, 256, 384 (0-based t_dec) that is 3/512 = 0.59 %; a 1-based reading would give
    4/512 = 0.78 % (99.2 %).  Runs the oracle for 512 steps on a minimal head."""
    rng = np.random.default_rng(7)
    d, L0, T = 4, 16, 512
    k = rng.standard_normal((1, 1, L0 + T, d)).astype(np.float32)
    v = rng.standard_normal((1, 1, L0 + T, d)).astype(np.float32)
    p = _params(head_dim=d, max_len=L0 + T, k=2, cache_cap=4, r=1, window=2, tau=-1.0,
                refresh=128)
    orc = O.Oracle(p)
    paths = []
    for t in range(T):
        q = rng.standard_normal((1, 1, d)).astype(np.float32)
        _, _, info = orc.decode_step(q, k, v, L0 + t + 1)
        paths.append(int(info.path[0]))
    n_ref = paths.count(O.REFRESH)
    assert n_ref == 3
    assert round(100 * (T - n_ref) / T, 1) == round(87.5 + 11.9, 1) == round(88.9 + 10.5, 1)


def test_window_only_reuse_when_supports_empty(oracle_lib):
    """W only (retrieved supports hold no index): the candidate set is the window and
    the rerank keeps its best K (Eq. 8-11)."""
    rng = np.random.default_rng(9)
    d, L = 8, 30
    k = rng.standard_normal((1, 1, L, d)).astype(np.float32)
    v = rng.standard_normal((1, 1, L, d)).astype(np.float32)
    q = rng.standard_normal((1, 1, d)).astype(np.float32)
    p = _params(head_dim=d, max_len=L, k=3, cache_cap=2, r=2, window=6, tau=-1.0)
    orc = O.Oracle(p)
    qb = np.tile(q[0, 0] / np.linalg.norm(q[0, 0]), (1, 2, 1)).astype(np.float32)
    orc.set_state(qb, np.full((1, 2, 3), -1, np.int32), np.zeros((1, 2), np.int32), 2, 0)
    out, sel, info = orc.decode_step(q, k, v, L)
    assert info.path[0] == O.REUSE
    assert info.cand[0, :info.n_cand[0]].tolist() == list(range(L - 6, L))
    s = O.scores(q[0, 0], k[0, 0], np.arange(L - 6, L))
    best = np.sort(np.arange(L - 6, L)[np.lexsort((np.arange(6), -s.astype(np.float64)))[:3]])
    assert sel[0, 0].tolist() == best.tolist()


def test_attend_on_given_set_matches_exact(oracle_lib, golden):
    """orc_attend over the exact support reproduces the exact output, and over the
    hand case's index sets gives the closed forms of Eq. 12."""
    k = np.array(golden["keys"], np.float32)
    v = np.array(golden["values"], np.float32)
    q = np.array(golden["exact"]["q"], np.float32)
    for case in golden["exact"]["cases"]:
        idx = np.array([i for i in case["sel"] if i >= 0], np.int32)
        want = np.array([_closed(s) for s in case["out"]])
        np.testing.assert_allclose(O.attend(q, k, v, idx[::-1].copy()), want, rtol=2e-7, atol=1e-7)


def test_recent_r_retrieval(oracle_lib, tiny):
    """Recent-R retrieval (the component ablation, Table 3): on every reuse step the
    retrieved entries are the R most recent insertions, newest first; rho_max is
    the best similarity among them and decides the fallback (Eq. 13); candidates
    are the union of their supports and the window (Eq. 8-9)."""
    w = tiny.w
    p = _workload_params(w, retrieval=1)
    seen = {"reuse": 0, "fallback": 0}

    def check(t, before, out, sel, info):
        L = w.step_len(t)
        path = int(info.path[0])
        if path not in (O.REUSE, O.FALLBACK):
            return
        nv = min(before["n_inserted"], w.cache_cap)
        recent = [(before["n_inserted"] - 1 - i) % w.cache_cap for i in range(min(w.r, nv))]
        q = tiny.q_dec[t][0, 0].astype(np.float64)
        qb = q / np.linalg.norm(q)
        rho = before["qbar"][0, :nv].astype(np.float64) @ qb
        assert abs(info.rho_max[0] - rho[recent].max()) < 1e-6
        assert (path == O.FALLBACK) == (info.rho_max[0] < w.tau)
        if path == O.FALLBACK:
            seen["fallback"] += 1
            return
        seen["reuse"] += 1
        assert info.retrieved[0, :len(recent)].tolist() == recent
        union = set(range(max(0, L - w.window), L))
        for s in recent:
            union.update(before["supp"][0, s, :before["cnt"][0, s]].tolist())
        n = int(info.n_cand[0])
        assert info.cand[0, :n].tolist() == sorted(union)

    _run(w, tiny, p, check=check)
    assert seen["reuse"] > 10 and seen["fallback"] > 0


def test_recent_r_equals_similarity_when_all_entries_are_retrieved(oracle_lib, tiny):
    """With R = C both retrieval rules retrieve every cached entry, so the two
    trajectories coincide step for step (same paths, supports and outputs)."""
    w = tiny.w
    a = _run(w, tiny, _workload_params(w, r=w.cache_cap))[1]
    b = _run(w, tiny, _workload_params(w, r=w.cache_cap, retrieval=1))[1]
    for (oa, sa, ia), (ob, sb, ib) in zip(a, b):
        assert np.array_equal(ia.path, ib.path)
        assert np.array_equal(sa, sb)
        assert np.array_equal(oa, ob)


def test_top_r_retrieval_bruteforce(oracle_lib, tiny):
    """Eq. 6-7 by brute force on every step that computes similarities: rho_c is the
    cosine of q with each valid cached q_bar (computed here in float64 from the
    stored fp32 rows), rho_max their maximum, and the retrieved entries the R most
    similar, ties to the newer insertion, most similar first; the candidates are
    the union of their supports and the window (Eq. 8-9)."""
    w = tiny.w
    p = _workload_params(w)
    seen = {"reuse": 0, "fallback": 0}

    def check(t, before, out, sel, info):
        path = int(info.path[0])
        if path not in (O.REUSE, O.FALLBACK):
            return
        nv = min(before["n_inserted"], w.cache_cap)
        q = tiny.q_dec[t][0, 0].astype(np.float64)
        qb = (q / np.sqrt((q * q).sum())).astype(np.float32).astype(np.float64)
        rho = before["qbar"][0, :nv].astype(np.float64) @ qb
        age = [(before["n_inserted"] - 1 - s) % w.cache_cap for s in range(nv)]
        order = sorted(range(nv), key=lambda s: (-rho[s], age[s]))
        assert abs(info.rho_max[0] - rho.max()) <= 1e-12 * max(1.0, abs(rho.max()))
        assert (path == O.FALLBACK) == (rho.max() < w.tau)
        if path == O.FALLBACK:
            seen["fallback"] += 1
            return
        seen["reuse"] += 1
        n_ret = min(w.r, nv)
        assert info.retrieved[0, :n_ret].tolist() == order[:n_ret]
        L = w.step_len(t)
        union = set(range(max(0, L - w.window), L))
        for s in order[:n_ret]:
            union.update(before["supp"][0, s, :before["cnt"][0, s]].tolist())
        n = int(info.n_cand[0])
        assert info.cand[0, :n].tolist() == sorted(union)

    _run(w, tiny, p, check=check)
    assert seen["reuse"] > 10 and seen["fallback"] > 0


def test_softmax_v_is_a_convex_combination(oracle_lib, tiny):
    """Eq. 12: the output is a convex combination of the selected value rows, so
    every coordinate lies between the smallest and the largest selected value of
    that coordinate (a wrong normalisation or sign breaks this)."""
    w = tiny.w
    p = _workload_params(w)
    for t in (0, 7, 31):
        L = w.step_len(t)
        out, sel, _ = O.exact(p, tiny.q_dec[t], tiny.k, tiny.v, L)
        idx = sel[0, 0][sel[0, 0] >= 0]
        vs = tiny.v[0, 0, idx].astype(np.float64)
        o = out[0, 0].astype(np.float64)
        slack = 1e-6 * np.abs(vs).max()
        assert (o >= vs.min(axis=0) - slack).all() and (o <= vs.max(axis=0) + slack).all()
        assert len(idx) == min(w.k, L)
