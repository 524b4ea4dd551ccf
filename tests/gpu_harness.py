"""Shared helpers of the GPU parity tests: device upload, handles, and the
comparison rules between the HIP path and the CPU oracle.

Comparison rules (per sequence, query head and step):
  * selected index sets must be equal, except when the oracle's K-th and (K+1)-th
    scores differ by at most REL_GAP relative; then the GPU set is accepted if
    every index it selected scores (in the oracle) at least s_K - tol and every
    index it left out at most s_K + tol ("near tie");
  * outputs are compared with the oracle's output on the GPU's own support:
    max_j |o - o_ref| / max_j |o_ref| <= OUT_TOL[dtype];
  * paths must match unless |rho_max - tau| <= REL_GAP; retrieved slots must match
    unless the cosine similarities involved tie within RHO_TIE.
"""
from __future__ import annotations

import numpy as np
import pytest

from oracle import oracle as O

REL_GAP = 1e-5
RHO_TIE = 1e-9
OUT_TOL = {"f32": 1e-5, "bf16": 2e-3}


def torch_cuda():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    return torch


def to_dev(raw: np.ndarray):
    torch = torch_cuda()
    if raw.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(raw).view(np.int16)).to("cuda")
    return torch.from_numpy(np.ascontiguousarray(raw)).to("cuda")


def params_of(w, **kw) -> O.Params:
    base = dict(batch=w.batch, n_q_heads=w.n_q_heads, n_kv_heads=w.n_kv_heads,
                head_dim=w.head_dim, max_len=w.max_len, k=w.k, cache_cap=w.cache_cap, r=w.r,
                window=w.window, tau=w.tau, refresh=w.refresh)
    base.update(kw)
    return O.Params(**base)


def handle_of(p: O.Params, dtype: str):
    from paper_2607_27692_amd import retopk as R
    return R.Handle(batch=p.batch, n_q_heads=p.n_q_heads, n_kv_heads=p.n_kv_heads,
                    head_dim=p.head_dim, max_len=p.max_len, k=p.k, cache_cap=p.cache_cap,
                    r=p.r, window=p.window, tau=p.tau, refresh=p.refresh, dtype=dtype,
                    retrieval=p.retrieval)


def debug_buffers(p: O.Params):
    torch = torch_cuda()
    bh = p.heads
    return dict(
        path=torch.full((bh,), -9, dtype=torch.int8, device="cuda"),
        rho_max=torch.full((bh,), float("nan"), dtype=torch.float64, device="cuda"),
        retrieved=torch.full((bh, p.r), -9, dtype=torch.int32, device="cuda"),
        n_cand=torch.full((bh,), -9, dtype=torch.int32, device="cuda"),
        cand=torch.full((bh, p.cand_cap), -9, dtype=torch.int32, device="cuda"),
    )


def rel_err(o, ref) -> float:
    o = np.asarray(o, np.float64)
    ref = np.asarray(ref, np.float64)
    scale = np.abs(ref).max()
    return float(np.abs(o - ref).max() / (scale if scale > 0 else 1.0))


class Tally:
    def __init__(self):
        self.exact = 0
        self.near_tie = 0
        self.path_tie = 0
        self.rho_tie = 0
        self.max_out_err = 0.0

    def __repr__(self):
        return (f"exact={self.exact} near_tie={self.near_tie} path_tie={self.path_tie} "
                f"rho_tie={self.rho_tie} max_out_err={self.max_out_err:.3g}")


def check_selection(gsel, osel, universe, uscores, where: str, tally: Tally) -> np.ndarray:
    """gsel / osel: K-long, -1 padded, ascending.  universe: candidate indices with
    their oracle scores uscores.  Returns the GPU support (validated)."""
    g = gsel[gsel >= 0]
    o = osel[osel >= 0]
    assert (np.diff(g) > 0).all(), f"{where}: GPU support not strictly ascending"
    if g.shape == o.shape and (g == o).all():
        tally.exact += 1
        return g
    assert g.shape == o.shape, f"{where}: support sizes {g.size} vs {o.size}"
    score = dict(zip(universe.tolist(), uscores.tolist()))
    assert all(i in score for i in g.tolist()), f"{where}: GPU picked an index outside the universe"
    in_o = np.isin(universe, o)
    s_k = uscores[in_o].min()
    s_next = uscores[~in_o].max()
    tol = REL_GAP * max(abs(float(s_k)), 1e-30)
    assert s_k - s_next <= tol, (
        f"{where}: support differs and the K-boundary gap {s_k - s_next:.3g} exceeds {tol:.3g}")
    in_g = np.isin(universe, g)
    assert (uscores[in_g] >= s_k - tol).all() and (uscores[~in_g] <= s_k + tol).all(), (
        f"{where}: GPU support is not a valid near-tie choice")
    tally.near_tie += 1
    return g


def check_output(gout, q, kr, vr, g, oout, exact_set: bool, dtype: str, where: str,
                 tally: Tally):
    ref = oout if exact_set else O.attend(q, kr, vr, g)
    e = rel_err(gout, ref)
    tally.max_out_err = max(tally.max_out_err, e)
    assert e <= OUT_TOL[dtype], f"{where}: output error {e:.3g} > {OUT_TOL[dtype]}"


def divergence_is_near_tie(info, bh: int, q, krows, length: int, k: int, tau: float,
                           r: int, pre_qbar, n_valid: int) -> bool:
    """True when the oracle's own step for head bh sits on a near-tie that lets a
    correct GPU step differ from it: the path decision within REL_GAP of tau, the
    R-th and (R+1)-th cosine similarities within RHO_TIE (pre_qbar: the head's
    cached queries before the step), or the K-th and (K+1)-th candidate scores
    within REL_GAP relative.  Then either choice is valid and the trajectories may
    part."""
    path = int(info.path[bh])
    if path in (O.REUSE, O.FALLBACK) and abs(float(info.rho_max[bh]) - tau) <= REL_GAP:
        return True
    if path == O.REUSE and n_valid > r:
        rho = np.sort(pre_qbar[:n_valid].astype(np.float64) @
                      O.normalize(q).astype(np.float64))[::-1]
        if rho[r - 1] - rho[r] <= RHO_TIE:
            return True
    if path == O.REUSE:
        universe = info.cand[bh, :int(info.n_cand[bh])]
    else:
        universe = np.arange(length, dtype=np.int32)
    if universe.size <= k:
        return False
    s = np.sort(O.scores(q, krows, universe))[::-1]
    return float(s[k - 1] - s[k]) <= REL_GAP * max(abs(float(s[k - 1])), 1e-30)
