"""ReTopK decode-step benchmark on one MI355X.

One step = one ReTopK decode step over every query head of the layer (the whole
hot path: similarity recall, path rule, candidate union, candidate or
full-history scoring, Top-K, Softmax-V, cache insert).  The default workload is
the 128K-context layer: 32 query / 8 KV heads, d = 128, bf16, K = 512, cache
capacity 512, r = 8, W = 256, tau = 0.8, refresh period 64, 256 decode steps, on
synthetic clustered keys and query walks (paper_2607_27692_amd/inputs.py).

Timing: inputs are resident in HBM before timing starts.  Prefill
initialisation is untimed.  Each timed step is bracketed by HIP events on the
launch stream; between steps a 1 GiB buffer is read (outside the events) so that
every step starts with cold L2 and MALL caches, as it would between two layers of
a model.  The flush reads rather than writes, so no dirty lines are left to be
written back during the timed step.  The Exact Top-K baseline (exact_topk_attention) runs over
the same queries and lengths under the same protocol.  Kernel durations come
from the library's own event profiling over the timed steps.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, published
COPY_BYTES = 256 << 20
METRIC = "µs per decode step (all heads) + speedup vs Exact Top-K, 128K ctx, K=512"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=256)
    ap.add_argument("--warmup", type=int, default=16)
    ap.add_argument("--workload", default="128k")
    ap.add_argument("--warm", action="store_true", help="no cache flush between steps")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--dump-steps", default="", metavar="FILE",
                    help="write the per-step times of the timed passes (JSON)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--copy-calibration", action="store_true",
                    help="after the passes, run a plain 256 MiB device copy 8 times, so that "
                         "a hardware-counter run can scale FETCH_SIZE / WRITE_SIZE by what "
                         "they read for a copy of known size")
    ap.add_argument("--summarize", nargs=3, metavar=("TRACE_DIR", "FETCH_DIR", "WRITE_DIR"),
                    help="no GPU work: turn the csv output of a rocprofv3 kernel-trace run and "
                         "of a FETCH_SIZE and a WRITE_SIZE counter run of this script (with "
                         "--copy-calibration) into the text summaries under profiles/")
    ap.add_argument("--fidelity", type=int, default=0, metavar="STEPS",
                    help="instead of timing, run STEPS decode steps from the prefill "
                         "initialisation and report how close ReTopK's supports and outputs "
                         "are to Exact Top-K's and to full attention's (support recall, "
                         "retained attention mass, output cosine), overall and on the "
                         "reuse path")
    ap.add_argument("--layers", type=int, default=0, metavar="L",
                    help="instead of the one-layer protocol, decode with L independent layers "
                         "(each its own keys, values, queries and ReTopK state) one after the "
                         "other per token, as a model does, and report ms per token over the L "
                         "layers for ReTopK, Exact Top-K and full attention (no cache flush: "
                         "rotating the layers' key and value rows defeats the caches)")
    ap.add_argument("--contexts", default="", metavar="N1,N2,...",
                    help="instead of the one-layer protocol, time the --workload layer (by "
                         "default the headline one) at each prompt length given (ReTopK, "
                         "Exact Top-K and full attention, cold "
                         "caches, --steps decode steps each, at most 64) and print one JSON "
                         "line with the per-length table (latency against context length)")
    ap.add_argument("--ablation", action="store_true",
                    help="instead of the one-layer protocol, run the component-ablation "
                         "settings (Table 3) and the paper's default settings on the 128K "
                         "layer: us per step, exact-path share, candidates, speedup against "
                         "Exact Top-K and support recall, one JSON line")
    return ap.parse_args()


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def main():
    args = parse()
    if args.summarize:
        summarize(args, *args.summarize)
        return
    if args.gpus != 1:
        print(f"bench.py: this build runs on exactly one GPU (asked for {args.gpus}); the "
              "multi-GPU layout is a design note only", file=sys.stderr)
        sys.exit(2)
    if args.fidelity:
        fidelity(args)
        return
    if args.layers:
        layers(args)
        return
    if args.contexts:
        contexts(args)
        return
    if args.ablation:
        ablation(args)
        return
    import torch

    from paper_2607_27692_amd import retopk as R
    from paper_2607_27692_amd.inputs import WORKLOADS, make_inputs

    w = WORKLOADS[args.workload]
    K_steps = min(args.steps, w.steps)
    torch.cuda.set_device(0)
    t0 = time.time()
    inp = make_inputs(w)
    log(f"[bench] inputs {w.name} generated in {time.time() - t0:.1f}s")

    def dev(raw):
        if raw.dtype == np.uint16:
            return torch.from_numpy(raw.view(np.int16)).to("cuda")
        return torch.from_numpy(raw).to("cuda")

    q_tail, q_dec, k, v = (dev(inp.q_tail_raw), dev(inp.q_dec_raw), dev(inp.k_raw),
                           dev(inp.v_raw))
    cfg = dict(batch=w.batch, n_q_heads=w.n_q_heads, n_kv_heads=w.n_kv_heads,
               head_dim=w.head_dim, max_len=w.max_len, k=w.k, cache_cap=w.cache_cap, r=w.r,
               window=w.window, tau=w.tau, refresh=w.refresh, dtype=w.dtype)
    out = torch.empty((w.batch, w.n_q_heads, w.head_dim), dtype=torch.float32, device="cuda")
    sel = torch.empty((w.batch, w.n_q_heads, w.k), dtype=torch.int32, device="cuda")
    flush = torch.ones(1 << 28, dtype=torch.float32, device="cuda")   # 1 GiB
    sink = torch.zeros((), dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()

    def fresh_handle():
        h = R.Handle(**cfg)
        h.prefill_init(q_tail, w.cache_cap, k, v, w.prompt_len)
        return h

    # ---- warm-up (separate handle, then discarded) --------------------------
    h = fresh_handle()
    for t in range(min(args.warmup, w.steps)):
        h.decode_step(q_dec[t], k, v, w.step_len(t), out, sel)
        h.exact(q_dec[t], k, v, w.step_len(t), out, sel)
        h.full(q_dec[t], k, v, w.step_len(t), out)
    # the timing loop's own machinery once (the flush's reduction and add kernels,
    # timing events), so that no first-call cost of the host lands in a timed step
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    for _ in range(2):
        sink.add_(flush.sum())
        e0.record(stream)
        e1.record(stream)
    torch.cuda.synchronize()
    e0.elapsed_time(e1)
    h.close()
    log("[bench] warm-up done")

    # ---- prefill initialisation (Sec. 3.3), timed once on its own handle -------
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    h = R.Handle(**cfg)
    h.profile(True)
    h.prefill_init(q_tail, w.cache_cap, k, v, w.prompt_len)
    torch.cuda.synchronize()
    pf_ms = (time.perf_counter() - t0) * 1e3
    pf_prof = h.profile_read()
    h.profile(False)
    h.close()
    log(f"[bench] prefill initialisation: {pf_ms:.2f} ms")

    def timed(run, profile, flush_between=None):
        """One pass over the timed steps on a fresh handle (prefill untimed)."""
        if flush_between is None:
            flush_between = not args.warm
        handle = fresh_handle()
        st0 = handle.stats()
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(K_steps)]
        handle.profile(profile)
        torch.cuda.synchronize()
        # a head start for the host: the GPU reads the flush buffer twice first, so
        # each step is queued before the GPU reaches it (host latency never enters
        # the events)
        sink.add_(flush.sum())
        sink.add_(flush.sum())
        wall0 = time.perf_counter()
        for t in range(K_steps):
            if flush_between:
                sink.add_(flush.sum())
            ev[t][0].record(stream)
            run(handle, t)
            ev[t][1].record(stream)
        torch.cuda.synchronize()
        wall = time.perf_counter() - wall0
        prof = handle.profile_read() if profile else {}
        handle.profile(False)
        st1 = handle.stats()
        handle.close()
        ms = np.array([a.elapsed_time(b) for a, b in ev])
        return ms, wall, prof, {k_: st1[k_] - st0[k_] for k_ in st1}

    retopk_run = lambda hh, t: hh.decode_step(q_dec[t], k, v, w.step_len(t), out, sel)  # noqa
    exact_run = lambda hh, t: hh.exact(q_dec[t], k, v, w.step_len(t), out, sel)  # noqa
    full_run = lambda hh, t: hh.full(q_dec[t], k, v, w.step_len(t), out)  # noqa

    # ---- ReTopK, then the Exact Top-K baseline on the same queries and lengths ---
    r_ms, r_wall, _, st = timed(retopk_run, False)
    log(f"[bench] ReTopK: {r_ms.mean() * 1e3:.1f} us/step (median {np.median(r_ms) * 1e3:.1f})")
    e_ms, e_wall, _, _ = timed(exact_run, False)
    log(f"[bench] Exact: {e_ms.mean() * 1e3:.1f} us/step (median {np.median(e_ms) * 1e3:.1f})")
    f_ms, _, _, _ = timed(full_run, False)
    log(f"[bench] Full attention: {f_ms.mean() * 1e3:.1f} us/step")
    # Same passes again with every kernel dispatch timed (events attached to the
    # dispatch packets); the trajectory is deterministic, so the kernels match.
    _, _, r_prof, st_p = timed(retopk_run, True)
    _, _, e_prof, _ = timed(exact_run, True)
    _, _, f_prof, _ = timed(full_run, True)
    assert st_p == st, "profiled pass diverged from the timed pass"
    # The same two passes back to back, without the flush (warm caches).
    rw_ms = timed(retopk_run, False, flush_between=False)[0]
    ew_ms = timed(exact_run, False, flush_between=False)[0]
    log(f"[bench] warm: ReTopK {rw_ms.mean() * 1e3:.1f} us/step, Exact {ew_ms.mean() * 1e3:.1f}")
    # The kind of every timed step (the trajectory is deterministic): an untimed
    # pass that reads the counters after each step.
    hh = fresh_handle()
    kinds, prev = [], hh.stats()
    for t in range(K_steps):
        retopk_run(hh, t)
        cur = hh.stats()
        dlt = {k_: cur[k_] - prev[k_] for k_ in cur}
        prev = cur
        kinds.append("refresh" if dlt["refresh"] else ("no_scan" if dlt["kv_group_scans"] == 0 else
                     ("one_scan" if dlt["kv_group_scans"] == 1 else "scans_2plus")))
    hh.close()
    kinds = np.array(kinds)
    step_types = {kd: dict(steps=int((kinds == kd).sum()), **step_stats(r_ms[kinds == kd]))
                  for kd in ("no_scan", "one_scan", "scans_2plus", "refresh") if (kinds == kd).any()}
    slow = int(np.argmax(r_ms))
    log(f"[bench] slowest ReTopK step: {slow} ({kinds[slow]}, {r_ms[slow] * 1e3:.1f} us); "
        f"first steps (us): {' '.join(f'{x * 1e3:.1f}' for x in r_ms[:12])}")
    if args.dump_steps:
        with open(args.dump_steps, "w") as f:
            json.dump({"retopk_us": (r_ms * 1e3).round(2).tolist(),
                       "exact_us": (e_ms * 1e3).round(2).tolist(),
                       "kinds": kinds.tolist()}, f)

    # ---- algorithmic bytes ------------------------------------------------------
    e = 2 if w.dtype == "bf16" else 4
    d = w.head_dim
    lens = np.array([w.step_len(t) for t in range(K_steps)], np.float64)
    BH = w.batch * w.n_q_heads
    head_steps = st["head_steps"]
    reuse = st["reuse"]
    fallback = st["fallback"]
    refresh = st["refresh"]
    scans = st["kv_group_scans"]
    cand_sum = st["cand_sum"]
    exact_heads = head_steps - reuse
    mean_len = lens.mean()
    # Per step: q, V rows of the support, output, cache insert for every head;
    # cached queries and supports read on reuse; key rows scanned or gathered.
    C_valid = w.cache_cap
    per_head_fixed = d * e + w.k * d * e + d * 4 + d * 4 + w.k * 4
    retopk_bytes = (head_steps * per_head_fixed
                    + (reuse + fallback) * C_valid * d * 4
                    + reuse * w.r * w.k * 4
                    + cand_sum * d * e
                    + scans * mean_len * d * e)
    exact_bytes = K_steps * (w.batch * w.n_kv_heads * mean_len * d * e
                             + BH * (w.k * d * e + d * e + d * 4))
    r_us, e_us = r_ms.mean() * 1e3, e_ms.mean() * 1e3
    step_gbs = retopk_bytes / K_steps / (r_us * 1e-6) / 1e9
    exact_gbs = exact_bytes / K_steps / (e_us * 1e-6) / 1e9

    # Dominant kernel of the ReTopK pass and its algorithmic bytes per launch: the
    # bytes the method has to read for the heads that launch serves (key rows
    # scanned or gathered, cached queries, support lists, value rows); buffers
    # internal to this implementation (scores, survivor lists) are not counted.
    # Refresh steps run every head as a full scan (retopk_scan); the other steps
    # launch retopk_sim and retopk_score.
    refresh_steps = refresh // BH if BH else 0
    select_steps = K_steps - refresh_steps
    scans_select = scans - refresh_steps * w.batch * w.n_kv_heads
    roof = None
    if r_prof:
        dom = max(r_prof, key=lambda n: r_prof[n][1])
        launches, tot_ms = r_prof[dom]
        if dom == "retopk_score":
            kbytes = (scans_select * mean_len * d * e + cand_sum * d * e
                      + reuse * w.r * w.k * 4 + select_steps * BH * d * e)
        elif dom == "retopk_sim":
            kbytes = select_steps * BH * (C_valid * d * 4 + d * e)
        elif dom == "retopk_final":
            kbytes = head_steps * (w.k * d * e + d * 4)
        elif dom == "retopk_scan":
            kbytes = refresh_steps * w.batch * w.n_kv_heads * mean_len * d * e
        else:
            kbytes = exact_heads * mean_len * 4
        ach = kbytes / launches / (tot_ms / launches * 1e-3) / 1e9
        roof = {"kernel": dom, "bound": "hbm", "achieved": round(ach, 1),
                "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(ach / HBM_PEAK_GBS, 4),
                "traffic": traffic_per_launch(dom, w.name),
                "avg_launch_us": round(tot_ms / launches * 1e3, 2), "launches": launches,
                "bytes_per_launch": round(kbytes / launches)}
    exact_roof = None
    if e_prof and e_prof.get("retopk_scan", (0, 0))[0]:
        launches, tot_ms = e_prof["retopk_scan"]
        scan_bytes = K_steps * w.batch * w.n_kv_heads * mean_len * d * e
        ach = scan_bytes / (tot_ms * 1e-3) / 1e9
        exact_roof = {"kernel": "retopk_scan", "bound": "hbm", "achieved": round(ach, 1),
                      "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(ach / HBM_PEAK_GBS, 4),
                      "traffic": traffic_per_launch("retopk_scan", w.name),
                      "bytes_per_launch": round(scan_bytes / launches),
                      "avg_launch_us": round(tot_ms / launches * 1e3, 2)}

    # Full attention: every key and value row once per step.
    f_us = f_ms.mean() * 1e3
    full_bytes = w.batch * w.n_kv_heads * mean_len * d * e * 2 + BH * (d * e + d * 4)
    full_roof = None
    if f_prof and f_prof.get("dense_chunk", (0, 0))[0]:
        launches, tot_ms = f_prof["dense_chunk"]
        fb = K_steps * w.batch * w.n_kv_heads * mean_len * d * e * 2
        ach = fb / (tot_ms * 1e-3) / 1e9
        full_roof = {"kernel": "dense_chunk", "bound": "hbm", "achieved": round(ach, 1),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(ach / HBM_PEAK_GBS, 4),
                     "traffic": traffic_per_launch("dense_chunk", w.name),
                     "avg_launch_us": round(tot_ms / launches * 1e3, 2),
                     "bytes_per_launch": round(fb / launches)}

    # Prefill: 2 d flops per (position, head, causal key) on the matrix cores.
    n_pf = w.cache_cap
    pf_flops = 2.0 * d * BH * sum(w.prompt_len - n_pf + u + 1 for u in range(n_pf))
    pf_score = pf_prof.get("prefill_score", (0, 0.0))
    prefill = {"ms": round(pf_ms, 3), "positions": n_pf,
               "kernels": {n: {"launches": l, "ms": round(ms, 3)} for n, (l, ms) in
                           pf_prof.items() if l},
               "prefill_score_tflops": round(pf_flops / (pf_score[1] * 1e-3) / 1e12, 1)
               if pf_score[0] else None}

    # ---- the practical HBM read ceiling: a plain streaming read of 1 GiB -------
    sink32 = torch.zeros(1, dtype=torch.int32, device="cuda")
    nbytes = flush.numel() * flush.element_size()
    for _ in range(2):
        R.retopk_stream_read(flush, nbytes, sink32)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record(stream)
    for _ in range(10):
        R.retopk_stream_read(flush, nbytes, sink32)
    ev1.record(stream)
    torch.cuda.synchronize()
    stream_gbs = 10 * nbytes / (ev0.elapsed_time(ev1) * 1e-3) / 1e9
    log(f"[bench] streaming read: {stream_gbs:.0f} GB/s")
    for rf in (roof, exact_roof, full_roof):
        if rf:
            rf["stream_read_gbs"] = round(stream_gbs, 1)
            rf["frac_of_stream_read"] = round(rf["achieved"] / stream_gbs, 4)

    # ---- CPU baseline: the oracle on a bounded sample ------------------------
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(w, inp, args.cpu_seconds,
                           round(cand_sum / reuse, 1) if reuse else None)

    res = {
        "metric": METRIC,
        "value": round(r_us, 2),
        "unit": "us/step",
        "n_gpus": 1,
        "steps": K_steps,
        "warmup": args.warmup,
        "ms_per_step": round(r_us / 1e3, 5),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if w.dtype == "bf16" else "f32",
        "data": "synthetic",
        "config": {"workload": w.name, "batch": w.batch, "q_heads": w.n_q_heads,
                   "kv_heads": w.n_kv_heads, "head_dim": w.head_dim,
                   "context": w.prompt_len, "k": w.k, "cache_cap": w.cache_cap, "r": w.r,
                   "window": w.window, "tau": w.tau, "refresh": w.refresh,
                   "cache_state": "warm" if args.warm else "cold (1 GiB read between steps)"},
        "speedup_vs_exact": round(e_us / r_us, 3),
        "exact_us_per_step": round(e_us, 2),
        "full_attention_us_per_step": round(f_us, 2),
        "speedup_vs_full_attention": round(f_us / r_us, 3),
        "full_hbm_frac": round(full_bytes / (f_us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
        "retopk_us_median": round(float(np.median(r_ms)) * 1e3, 2),
        "retopk_us_p90": round(float(np.percentile(r_ms, 90)) * 1e3, 2),
        "retopk_us_max": round(float(r_ms.max()) * 1e3, 2),
        "retopk_slowest_step": {"step": slow, "kind": str(kinds[slow])},
        "exact_us_median": round(float(np.median(e_ms)) * 1e3, 2),
        "exact_us_p90": round(float(np.percentile(e_ms, 90)) * 1e3, 2),
        "exact_us_max": round(float(e_ms.max()) * 1e3, 2),
        "fallback_rate": round(fallback / head_steps, 4) if head_steps else None,
        "refresh_share": round(refresh / head_steps, 4) if head_steps else None,
        "cold_head_steps": int(st["cold"]),
        "mean_candidates": round(cand_sum / reuse, 1) if reuse else None,
        "max_candidates": st["cand_max"],
        "wall_s_exact": round(e_wall, 4),
        "kv_group_scans_per_step": round(scans / K_steps, 3),
        "step_hbm_gbs": round(step_gbs, 1),
        "step_hbm_frac": round(step_gbs / HBM_PEAK_GBS, 4),
        "exact_hbm_gbs": round(exact_gbs, 1),
        "exact_hbm_frac": round(exact_gbs / HBM_PEAK_GBS, 4),
        "wall_s_timed": round(r_wall, 4),
        "kernels_retopk": {n: {"launches": l, "avg_us": round(ms / l * 1e3, 2) if l else None}
                           for n, (l, ms) in r_prof.items()},
        "kernels_exact": {n: {"launches": l, "avg_us": round(ms / l * 1e3, 2) if l else None}
                          for n, (l, ms) in e_prof.items()},
        "roofline": roof,
        "exact_roofline": exact_roof,
        "full_attention_roofline": full_roof,
        "prefill_init": prefill,
        "step_types": step_types,
        "warm_caches": {"retopk_us_per_step": round(float(rw_ms.mean()) * 1e3, 2),
                        "exact_us_per_step": round(float(ew_ms.mean()) * 1e3, 2),
                        "speedup_vs_exact": round(float(ew_ms.mean() / rw_ms.mean()), 3)},
        "cpu_baseline": cpu,
    }
    print(json.dumps(res), flush=True)
    if args.copy_calibration:
        src = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(8):
            sink.add_(flush.sum())
            dst.copy_(src)
        torch.cuda.synchronize()
        log(f"[bench] copy calibration: 8 x {COPY_BYTES} bytes")


def step_stats(ms) -> dict:
    """Mean, median, 90th percentile and maximum of per-step times given in ms, in us."""
    ms = np.asarray(ms, np.float64)
    return {"us_mean": round(float(ms.mean()) * 1e3, 2),
            "us_median": round(float(np.median(ms)) * 1e3, 2),
            "us_p90": round(float(np.percentile(ms, 90)) * 1e3, 2),
            "us_max": round(float(ms.max()) * 1e3, 2)}


def kernel_source_digest() -> str:
    path = os.path.join(ROOT, "paper_2607_27692_amd", "csrc", "retopk_kernels.hip")
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def traffic_per_launch(kernel: str, workload: str):
    """Measured HBM bytes per launch of `kernel` (FETCH_SIZE + WRITE_SIZE, scaled
    by a copy of known size), from the counter summary kept under profiles/;
    None when there is none or the kernel source has changed since it was taken."""
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel}_{workload}.txt")
    if not os.path.exists(path):
        return None
    fields = {}
    with open(path) as f:
        for line in f:
            if ":" in line and not line.startswith("#"):
                key, val = line.split(":", 1)
                fields[key.strip()] = val.strip()
    if fields.get("kernel_source_sha256") != kernel_source_digest():
        return None
    try:
        return int(float(fields["traffic_bytes_per_launch"]))
    except (KeyError, ValueError):
        return None


def cpu_baseline(w, inp, seconds: float, gpu_mean_candidates=None):
    """The oracle, single-threaded and pinned to one host core, on KV group 0's
    query heads: Exact Top-K steps, then ReTopK decode steps from a seeded cache
    state, until about `seconds` of CPU time is spent; scaled to all heads of the
    layer.  The seeded supports are drawn half from the query's key cluster and
    half uniformly, so their unions are larger than those of the GPU's own
    trajectory; the sample's mean candidate count is reported beside the GPU's."""
    from oracle import oracle as O
    from paper_2607_27692_amd.inputs import make_support_state

    G = w.group
    heads = list(range(G))
    mask = np.zeros(w.batch * w.n_q_heads, np.uint8)
    mask[heads] = 1
    p = O.Params(w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.max_len, w.k, w.cache_cap,
                 w.r, w.window, w.tau, w.refresh)
    kf, vf = inp.k, inp.v
    supp, cnt = make_support_state(inp, heads=heads)
    qbar = np.zeros((w.batch * w.n_q_heads, w.cache_cap, w.head_dim), np.float32)
    for hh in heads:
        qbar[hh] = np.stack([O.normalize(inp.q_tail[0, hh, u]) for u in range(w.cache_cap)])
    orc = O.Oracle(p)
    orc.set_state(qbar, supp, cnt, w.cache_cap, 1)
    # pin this thread to one core of those the process may use, for the timed work
    allowed = sorted(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else []
    core = allowed[0] if allowed else None
    if core is not None:
        os.sched_setaffinity(0, {core})
    try:
        t0 = time.thread_time()
        n_ex = 0
        while n_ex < 2 or (time.thread_time() - t0 < seconds / 2 and n_ex < w.steps):
            O.exact(p, inp.q_dec[n_ex], kf, vf, w.step_len(n_ex), head_mask=mask)
            n_ex += 1
        ex_s = (time.thread_time() - t0) / n_ex
        t1 = time.thread_time()
        n_st, cand, n_reuse = 0, 0, 0
        while n_st < 2 or (time.thread_time() - t1 < seconds / 2 and n_st < w.steps):
            _, _, info = orc.decode_step(inp.q_dec[n_st], kf, vf, w.step_len(n_st),
                                         head_mask=mask)
            n_st += 1
            ru = info.path[heads] == O.REUSE
            cand += int(info.n_cand[heads][ru].sum())
            n_reuse += int(ru.sum())
        st_s = (time.thread_time() - t1) / n_st
    finally:
        if core is not None:
            os.sched_setaffinity(0, set(allowed))
    scale = (w.batch * w.n_q_heads) / len(heads)
    return {"value": round(st_s * scale * 1e6, 1), "unit": "us/step", "cores": 1,
            "kind": "oracle",
            "exact_us_per_step": round(ex_s * scale * 1e6, 1),
            "sample": (f"oracle (plain C, 1 thread pinned to core {core}) on the {len(heads)} "
                       f"query heads of KV group 0, {n_st} ReTopK steps from a seeded cache "
                       f"state and {n_ex} Exact Top-K steps, scaled x{scale:g} to all heads"),
            "pinned_core": core,
            "mean_candidates": round(cand / n_reuse, 1) if n_reuse else None,
            "gpu_mean_candidates": gpu_mean_candidates,
            "cpu": _cpu_model(), "host_cores": os.cpu_count()}


def _cpu_model() -> str:
    """The host CPU's model name (from /proc/cpuinfo where there is one)."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or platform.machine()


# ---- fidelity diagnostics ------------------------------------------------------
def support_recall(sel, exact_sel) -> float:
    """|S_hat & S| / |S| for two -1 padded supports (the overlap measure of Eq. 2
    applied to the selected and the exact support)."""
    a = set(int(i) for i in sel if i >= 0)
    b = set(int(i) for i in exact_sel if i >= 0)
    return len(a & b) / max(len(b), 1)


def retained_mass(sel, probs) -> float:
    """Share of the full-attention probability mass on the selected positions."""
    idx = np.asarray([i for i in sel if i >= 0], dtype=np.int64)
    return float(np.asarray(probs, np.float64)[idx].sum())


def cosine(x, y) -> float:
    x = np.asarray(x, np.float64).ravel()
    y = np.asarray(y, np.float64).ravel()
    den = np.linalg.norm(x) * np.linalg.norm(y)
    return float(x @ y / den) if den > 0 else 1.0


def fidelity(args):
    """ReTopK against Exact Top-K and full attention on the GPU, step by step from
    the prefill initialisation: support recall (Eq. 2), retained attention mass,
    attention-distribution cosine and head-output cosine, as the paper reports
    them for its fidelity analysis (Sec. 4.2)."""
    import torch

    from paper_2607_27692_amd import retopk as R
    from paper_2607_27692_amd.inputs import WORKLOADS, make_inputs

    w = WORKLOADS[args.workload]
    steps = min(args.fidelity, w.steps)
    torch.cuda.set_device(0)
    inp = make_inputs(w)

    def dev(raw):
        if raw.dtype == np.uint16:
            return torch.from_numpy(raw.view(np.int16)).to("cuda")
        return torch.from_numpy(raw).to("cuda")

    q_tail, q_dec, k, v = (dev(inp.q_tail_raw), dev(inp.q_dec_raw), dev(inp.k_raw),
                           dev(inp.v_raw))
    cfg = dict(batch=w.batch, n_q_heads=w.n_q_heads, n_kv_heads=w.n_kv_heads,
               head_dim=w.head_dim, max_len=w.max_len, k=w.k, cache_cap=w.cache_cap, r=w.r,
               window=w.window, tau=w.tau, refresh=w.refresh, dtype=w.dtype)
    h = R.Handle(**cfg)
    h.prefill_init(q_tail, w.cache_cap, k, v, w.prompt_len)
    BH = w.batch * w.n_q_heads
    out_r = torch.empty((w.batch, w.n_q_heads, w.head_dim), dtype=torch.float32, device="cuda")
    out_e = torch.empty_like(out_r)
    sel_r = torch.empty((w.batch, w.n_q_heads, w.k), dtype=torch.int32, device="cuda")
    sel_e = torch.empty_like(sel_r)
    path = torch.empty(BH, dtype=torch.int8, device="cuda")
    scale = 1.0 / np.sqrt(w.head_dim)
    rows = []   # (path, recall, mass_r, mass_e, dist_cos, out_cos_exact, out_cos_full)
    for t in range(steps):
        L = w.step_len(t)
        h.decode_step(q_dec[t], k, v, L, out_r, sel_r, {"path": path})
        h.exact(q_dec[t], k, v, L, out_e, sel_e)
        torch.cuda.synchronize()
        sr, se = sel_r.cpu().numpy(), sel_e.cpu().numpy()
        orr, oe = out_r.cpu().numpy(), out_e.cpu().numpy()
        pth = path.cpu().numpy()
        for b in range(w.batch):
            for g in range(w.n_kv_heads):
                # full attention in fp32 as the reference
                as32 = (lambda x: x.view(torch.bfloat16).float()) if w.dtype == "bf16" else (
                    lambda x: x.float())
                kf, vf = as32(k[b, g, :L]), as32(v[b, g, :L])
                qf = as32(q_dec[t][b, g * w.group:(g + 1) * w.group])
                probs = torch.softmax((qf @ kf.T) * scale, dim=-1)
                full = (probs @ vf).cpu().numpy()
                probs = probs.cpu().numpy()
                for j in range(w.group):
                    hq = g * w.group + j
                    sel = sr[b, hq]
                    idx = sel[sel >= 0]
                    sparse = np.zeros(L)
                    sparse[idx] = probs[j][idx] / probs[j][idx].sum()
                    rows.append((int(pth[b * w.n_q_heads + hq]), support_recall(sel, se[b, hq]),
                                 retained_mass(sel, probs[j]), retained_mass(se[b, hq], probs[j]),
                                 cosine(sparse, probs[j]), cosine(orr[b, hq], oe[b, hq]),
                                 cosine(orr[b, hq], full[j])))
        log(f"[fidelity] step {t + 1}/{steps}")
    h.close()
    a = np.array(rows, dtype=np.float64)
    names = ["support_recall", "retained_mass", "exact_retained_mass",
             "attention_distribution_cosine", "output_cosine_vs_exact", "output_cosine_vs_full"]

    def summary(mask):
        return {n: round(float(a[mask, i + 1].mean()), 5) for i, n in enumerate(names)} | {
            "head_steps": int(mask.sum())}

    reuse = a[:, 0] == 0   # RETOPK_REUSE
    print(json.dumps({"fidelity": {"workload": w.name, "steps": steps, "data": "synthetic",
                                   "all": summary(np.ones(len(a), bool)),
                                   "reuse_path": summary(reuse)}}), flush=True)


# ---- component ablation (Table 3) ----------------------------------------------
ABLATION = [  # label, config changes (the same inputs for every setting)
    ("retopk", {}),
    ("recent_r", {"retrieval": 1}),
    ("r1", {"r": 1}),
    ("c1", {"cache_cap": 1}),
    ("tau_minus1", {"tau": -1.0}),
    ("no_refresh", {"refresh": 0}),
    ("no_window", {"window": 0}),
    ("paper_defaults", {"cache_cap": 32, "r": 4, "window": 32, "tau": 0.85, "refresh": 128}),
]


def ablation(args):
    """The settings of the paper's component ablation (Table 3) on the 128K layer,
    each on the same keys, values and queries (the prefill uses the last C prompt
    queries): mean us per step (cold caches), the share of head-steps on the exact
    path, mean candidates per reuse head, the speedup against Exact Top-K, and the
    support recall against Exact Top-K over the first steps."""
    import torch

    from paper_2607_27692_amd import retopk as R
    from paper_2607_27692_amd.inputs import WORKLOADS, make_inputs

    w = WORKLOADS[args.workload]
    steps = min(args.steps, w.steps)
    rsteps = min(16, steps)
    torch.cuda.set_device(0)
    inp = make_inputs(w)

    def dev(raw):
        if raw.dtype == np.uint16:
            return torch.from_numpy(np.ascontiguousarray(raw).view(np.int16)).to("cuda")
        return torch.from_numpy(np.ascontiguousarray(raw)).to("cuda")

    q_dec, k, v = dev(inp.q_dec_raw), dev(inp.k_raw), dev(inp.v_raw)
    flush = torch.ones(1 << 28, dtype=torch.float32, device="cuda")
    sink = torch.zeros((), dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()
    base = dict(batch=w.batch, n_q_heads=w.n_q_heads, n_kv_heads=w.n_kv_heads,
                head_dim=w.head_dim, max_len=w.max_len, k=w.k, cache_cap=w.cache_cap, r=w.r,
                window=w.window, tau=w.tau, refresh=w.refresh, dtype=w.dtype)
    out = torch.empty((w.batch, w.n_q_heads, w.head_dim), dtype=torch.float32, device="cuda")
    sel = torch.empty((w.batch, w.n_q_heads, w.k), dtype=torch.int32, device="cuda")

    def timed(run):
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(steps)]
        torch.cuda.synchronize()
        sink.add_(flush.sum())   # a head start for the host (see the main pass)
        sink.add_(flush.sum())
        for t in range(steps):
            sink.add_(flush.sum())
            ev[t][0].record(stream)
            run(t)
            ev[t][1].record(stream)
        torch.cuda.synchronize()
        return np.array([a.elapsed_time(b) for a, b in ev]) * 1e3

    # Exact Top-K: time, and its supports for the recall
    he = R.Handle(**base)
    exact_sel = []
    for t in range(rsteps):
        he.exact(q_dec[t], k, v, w.step_len(t), out, sel)
        exact_sel.append(sel.cpu().numpy().copy())
    e_us = timed(lambda t: he.exact(q_dec[t], k, v, w.step_len(t), out, sel)).mean()
    he.close()
    rows = []
    for label, change in ABLATION:
        cfg = dict(base, **change)
        C = cfg["cache_cap"]
        q_tail = dev(inp.q_tail_raw[:, :, w.cache_cap - C:])
        # support recall over the first steps, then the timed pass, each from the prefill
        h = R.Handle(**cfg)
        h.prefill_init(q_tail, C, k, v, w.prompt_len)
        rec = []
        for t in range(rsteps):
            h.decode_step(q_dec[t], k, v, w.step_len(t), out, sel)
            s_ = sel.cpu().numpy()
            rec += [support_recall(s_[b, hq], exact_sel[t][b, hq])
                    for b in range(w.batch) for hq in range(w.n_q_heads)]
        h.close()
        h = R.Handle(**cfg)
        h.prefill_init(q_tail, C, k, v, w.prompt_len)
        st0 = h.stats()
        r_us = timed(lambda t: h.decode_step(q_dec[t], k, v, w.step_len(t), out, sel))
        st = {k_: v_ - st0[k_] for k_, v_ in h.stats().items()}
        h.close()
        hs = st["head_steps"]
        row = {"setting": label, **change, "us_per_step": round(float(r_us.mean()), 2),
               "speedup_vs_exact": round(float(e_us / r_us.mean()), 3),
               "exact_path_share": round((st["fallback"] + st["refresh"] + st["cold"]) / hs, 4),
               "fallback_rate": round(st["fallback"] / hs, 4),
               "mean_candidates": round(st["cand_sum"] / st["reuse"], 1) if st["reuse"] else None,
               "support_recall": round(float(np.mean(rec)), 4)}
        rows.append(row)
        log(f"[ablation] {row}")
    print(json.dumps({"ablation": rows, "workload": w.name, "steps": steps,
                      "recall_steps": rsteps, "exact_us_per_step": round(float(e_us), 2),
                      "data": "synthetic", "cache_state": "cold (1 GiB read between steps)"}),
          flush=True)


# ---- latency against context length -------------------------------------------
def contexts(args):
    """The --workload layer (by default the headline one: 32 query / 8 KV heads,
    d = 128, bf16, K = 512, C = 512, R = 8, W = 256, tau = 0.8, T_r = 64), with one
    key cluster per K keys, at each prompt length: mean us per step of
    ReTopK, Exact Top-K and full attention under the cold-cache protocol, the
    fallback rate and the KV-group scans per step.  The reuse path's work does not
    depend on the context length; the exact path's grows with it (Sec. 4.3)."""
    import torch

    from paper_2607_27692_amd import retopk as R
    from paper_2607_27692_amd.inputs import WORKLOADS, make_inputs

    base = WORKLOADS[args.workload]
    steps = max(1, min(args.steps, 64))
    torch.cuda.set_device(0)
    flush = torch.ones(1 << 28, dtype=torch.float32, device="cuda")
    sink = torch.zeros((), dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()
    dev = lambda raw: torch.from_numpy(raw.view(np.int16)).to("cuda")  # noqa: E731
    rows = []
    for n_ctx in [int(x) for x in args.contexts.split(",") if x]:
        # as many key clusters as keys / K, so that a cluster is about one support
        w = base.with_(name=f"{n_ctx // 1024}k", prompt_len=n_ctx, steps=steps,
                       n_centers=max(1, n_ctx // base.k))
        t0 = time.time()
        inp = make_inputs(w)
        q_tail, q_dec, k, v = (dev(inp.q_tail_raw), dev(inp.q_dec_raw), dev(inp.k_raw),
                               dev(inp.v_raw))
        del inp
        cfg = dict(batch=w.batch, n_q_heads=w.n_q_heads, n_kv_heads=w.n_kv_heads,
                   head_dim=w.head_dim, max_len=w.max_len, k=w.k, cache_cap=w.cache_cap,
                   r=w.r, window=w.window, tau=w.tau, refresh=w.refresh, dtype=w.dtype)
        out = torch.empty((w.batch, w.n_q_heads, w.head_dim), dtype=torch.float32,
                          device="cuda")
        sel = torch.empty((w.batch, w.n_q_heads, w.k), dtype=torch.int32, device="cuda")

        def one_pass(kind, prefill):
            h = R.Handle(**cfg)
            if prefill:
                h.prefill_init(q_tail, w.cache_cap, k, v, w.prompt_len)
            ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                  for _ in range(steps)]
            st0 = h.stats()
            torch.cuda.synchronize()
            sink.add_(flush.sum())   # a head start for the host (see the main pass)
            sink.add_(flush.sum())
            for t in range(steps):
                sink.add_(flush.sum())
                ev[t][0].record(stream)
                if kind == "retopk":
                    h.decode_step(q_dec[t], k, v, w.step_len(t), out, sel)
                elif kind == "exact":
                    h.exact(q_dec[t], k, v, w.step_len(t), out, sel)
                else:
                    h.full(q_dec[t], k, v, w.step_len(t), out)
                ev[t][1].record(stream)
            torch.cuda.synchronize()
            st1 = h.stats()
            h.close()
            ms = np.array([a.elapsed_time(b) for a, b in ev])
            return ms, {k_: st1[k_] - st0[k_] for k_ in st1}

        one_pass("retopk", True)     # warm-up: kernels loaded, allocator primed
        r_ms, st = one_pass("retopk", True)
        e_ms, _ = one_pass("exact", False)
        f_ms, _ = one_pass("full", False)
        row = {"context": n_ctx, "retopk_us": round(float(r_ms.mean()) * 1e3, 2),
               "retopk_us_median": round(float(np.median(r_ms)) * 1e3, 2),
               "exact_us": round(float(e_ms.mean()) * 1e3, 2),
               "full_attention_us": round(float(f_ms.mean()) * 1e3, 2),
               "speedup_vs_exact": round(float(e_ms.mean() / r_ms.mean()), 3),
               "fallback_rate": round(st["fallback"] / st["head_steps"], 4),
               "kv_group_scans_per_step": round(st["kv_group_scans"] / steps, 3)}
        rows.append(row)
        log(f"[contexts] {n_ctx}: {row} ({time.time() - t0:.1f}s)")
        del q_tail, q_dec, k, v
        torch.cuda.empty_cache()
    print(json.dumps({"contexts": rows, "steps": steps, "data": "synthetic", "dtype": "bf16",
                      "config": {"workload": base.name, "batch": base.batch,
                                 "q_heads": base.n_q_heads,
                                 "kv_heads": base.n_kv_heads, "head_dim": base.head_dim,
                                 "k": base.k, "cache_cap": base.cache_cap, "r": base.r,
                                 "window": base.window, "tau": base.tau,
                                 "refresh": base.refresh},
                      "cache_state": "cold (1 GiB read between steps)"}), flush=True)


# ---- several layers per token ---------------------------------------------------
def _layer_inputs(job):
    """Worker: the raw arrays of one layer (the workload drawn from its own seed)."""
    from paper_2607_27692_amd.inputs import WORKLOADS, make_inputs
    name, seed = job
    inp = make_inputs(WORKLOADS[name], seed=seed)
    return seed, inp.q_tail_raw, inp.q_dec_raw, inp.k_raw, inp.v_raw


def layers(args):
    """ms per token over L layers: token t runs decode step t of layer 0, 1, ..,
    L-1 in turn (each layer its own handle, keys, values and queries, layer l
    drawn from seed l), the way the paper reports decode latency per token over a
    model's layers (Table 4).  The Exact Top-K and full-attention passes run the
    same layers and tokens.  Each token is bracketed by HIP events; there is no
    flush, since L layers' key and value rows exceed the caches."""
    import multiprocessing as mp

    from paper_2607_27692_amd.inputs import WORKLOADS
    w = WORKLOADS[args.workload]
    L = args.layers
    T = min(args.steps, w.steps)
    # Generate on the host before this process touches the GPU (the workers are
    # forked), then upload layer by layer.
    t0 = time.time()
    n_proc = max(1, min(L, 16, os.cpu_count() or 1))
    ctx = mp.get_context("fork")
    pool = ctx.Pool(n_proc)
    import torch

    from paper_2607_27692_amd import retopk as R
    lay = [None] * L

    def dev(raw):
        if raw.dtype == np.uint16:
            return torch.from_numpy(raw.view(np.int16)).to("cuda")
        return torch.from_numpy(raw).to("cuda")

    for seed, qt, qd, kr, vr in pool.imap_unordered(_layer_inputs, [(w.name, l) for l in range(L)]):
        lay[seed] = (dev(qt), dev(qd), dev(kr), dev(vr))
        del qt, qd, kr, vr
        log(f"[layers] layer {seed} resident ({L - lay.count(None)}/{L})")
    pool.close()
    pool.join()
    log(f"[layers] inputs of {L} layers generated and uploaded in {time.time() - t0:.1f}s")
    torch.cuda.set_device(0)
    cfg = dict(batch=w.batch, n_q_heads=w.n_q_heads, n_kv_heads=w.n_kv_heads,
               head_dim=w.head_dim, max_len=w.max_len, k=w.k, cache_cap=w.cache_cap, r=w.r,
               window=w.window, tau=w.tau, refresh=w.refresh, dtype=w.dtype)
    out = torch.empty((w.batch, w.n_q_heads, w.head_dim), dtype=torch.float32, device="cuda")
    sel = torch.empty((w.batch, w.n_q_heads, w.k), dtype=torch.int32, device="cuda")
    stream = torch.cuda.current_stream()

    def handles():
        hs = []
        for qt, _, kk, vv in lay:
            hh = R.Handle(**cfg)
            hh.prefill_init(qt, w.cache_cap, kk, vv, w.prompt_len)
            hs.append(hh)
        torch.cuda.synchronize()
        return hs

    def decode(hh, l, t):
        _, qd, kk, vv = lay[l]
        hh.decode_step(qd[t], kk, vv, w.step_len(t), out, sel)

    def exact(hh, l, t):
        _, qd, kk, vv = lay[l]
        hh.exact(qd[t], kk, vv, w.step_len(t), out, sel)

    def full(hh, l, t):
        _, qd, kk, vv = lay[l]
        hh.full(qd[t], kk, vv, w.step_len(t), out)

    def run(fn, hs, n_tokens):
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(n_tokens)]
        torch.cuda.synchronize()
        for t in range(n_tokens):
            ev[t][0].record(stream)
            for l in range(L):
                fn(hs[l], l, t)
            ev[t][1].record(stream)
        torch.cuda.synchronize()
        return np.array([a.elapsed_time(b) for a, b in ev])

    # warm-up on throwaway handles, then fresh handles for the timed ReTopK pass
    hs = handles()
    for fn in (decode, exact, full):
        run(fn, hs, min(args.warmup, T))
    for hh in hs:
        hh.close()
    log("[layers] warm-up done")
    hs = handles()
    st0 = [hh.stats() for hh in hs]
    r_ms = run(decode, hs, T)
    st = {k_: sum(hh.stats()[k_] - s0[k_] for hh, s0 in zip(hs, st0)) for k_ in st0[0]}
    log(f"[layers] ReTopK: {r_ms.mean():.3f} ms/token")
    e_ms = run(exact, hs, T)
    log(f"[layers] Exact: {e_ms.mean():.3f} ms/token")
    f_ms = run(full, hs, T)
    log(f"[layers] Full attention: {f_ms.mean():.3f} ms/token")
    for hh in hs:
        hh.close()
    hsteps = st["head_steps"]
    print(json.dumps({
        "metric": f"ms per token over {L} layers (all heads of each layer), "
                  f"{w.prompt_len // 1024}K ctx, K={w.k}",
        "value": round(float(r_ms.mean()), 4), "unit": "ms/token", "n_gpus": 1,
        "layers": L, "tokens": T, "warmup": args.warmup, "higher_is_better": False,
        "dtype": "bf16" if w.dtype == "bf16" else "f32", "data": "synthetic",
        "config": {"workload": w.name, "layers": L, "batch": w.batch, "q_heads": w.n_q_heads,
                   "kv_heads": w.n_kv_heads, "head_dim": w.head_dim, "context": w.prompt_len,
                   "k": w.k, "cache_cap": w.cache_cap, "r": w.r, "window": w.window,
                   "tau": w.tau, "refresh": w.refresh},
        "retopk_ms_per_token": round(float(r_ms.mean()), 4),
        "retopk_ms_median": round(float(np.median(r_ms)), 4),
        "exact_ms_per_token": round(float(e_ms.mean()), 4),
        "full_attention_ms_per_token": round(float(f_ms.mean()), 4),
        "speedup_vs_exact": round(float(e_ms.mean() / r_ms.mean()), 3),
        "speedup_vs_full_attention": round(float(f_ms.mean() / r_ms.mean()), 3),
        "retopk_us_per_layer": round(float(r_ms.mean()) * 1e3 / L, 2),
        "exact_us_per_layer": round(float(e_ms.mean()) * 1e3 / L, 2),
        "full_attention_us_per_layer": round(float(f_ms.mean()) * 1e3 / L, 2),
        "fallback_rate": round(st["fallback"] / hsteps, 4) if hsteps else None,
        "refresh_share": round(st["refresh"] / hsteps, 4) if hsteps else None,
        "kv_group_scans_per_layer_step": round(st["kv_group_scans"] / (T * L), 3),
    }), flush=True)


# ---- profiler summaries -------------------------------------------------------
SYMBOLS = {  # kernel symbol prefix -> name used by the library's own profiling
    "void retopk::k_sim<": "retopk_sim",
    "retopk::k_filter(": "retopk_filter",
    "void retopk::k_final<": "retopk_final",
    "void retopk::k_dense<": "dense_chunk",
    "void retopk::k_dense_merge<": "dense_merge",
    "void retopk::k_pf_score<": "prefill_score",
    "void retopk::k_scan_list<": "retopk_scan",
}


def _lib_name(symbol: str):
    if symbol.startswith("void retopk::k_score<"):
        # every build of k_score: <dtype, d, heads per group, selects>
        return "retopk_score" if symbol.split(">(", 1)[0].endswith("true") else "retopk_scan"
    for prefix, name in SYMBOLS.items():
        if symbol.startswith(prefix):
            return name
    return None


def _read_csv(path):
    import csv
    with open(path) as f:
        return list(csv.DictReader(f))


def _passes(names, w, steps, warmup):
    """Splits the library's dispatches (in dispatch order) into the bench's
    passes.  Every pass starts on a fresh handle whose prefill issues a
    prefill_score, filter, final triple per launch of prompt-tail positions (a
    scan, filter, final triple per position for f32); a decode step that selects
    issues sim, score, filter, final, any other step or an Exact Top-K step
    scan, filter, final, and a full-attention step dense_chunk, dense_merge.
    The warm-up runs one step of each kind per warm-up step, then one handle
    runs the timed prefill alone; after the six passes come the two warm-cache
    passes and the untimed pass that labels the step kinds.  Returns (label, first, end) positions of each
    pass's step dispatches, and the (first, end) positions of the timed prefill's
    dispatches."""
    plan = [("warm-up", 3 * min(warmup, w.steps)), ("prefill", 0), ("retopk timed", steps),
            ("exact timed", steps), ("full timed", steps), ("retopk profiled", steps),
            ("exact profiled", steps), ("full profiled", steps), ("retopk warm", steps),
            ("exact warm", steps), ("step kinds", steps)]
    units = {"retopk_sim": ["retopk_sim", "retopk_score", "retopk_filter", "retopk_final"],
             "retopk_scan": ["retopk_scan", "retopk_filter", "retopk_final"],
             "dense_chunk": ["dense_chunk", "dense_merge"]}
    out, i = [], 0
    pf = ["prefill_score", "retopk_filter", "retopk_final"]
    prefill = None
    n_pf = None      # triples per prefill: every handle's prefill is the same
    for label, n_units in plan:
        p0 = i
        if names[i] == "prefill_score":
            if n_pf is None:   # the first handle's prefill is followed by steps
                n_pf = 0
                while names[i + 3 * n_pf:i + 3 * n_pf + 3] == pf:
                    n_pf += 1
            for _ in range(n_pf):
                assert names[i:i + 3] == pf, f"unexpected prefill at {i}"
                i += 3
        else:
            for _ in range(w.cache_cap):
                assert names[i:i + 3] == units["retopk_scan"], f"unexpected prefill at {i}"
                i += 3
        if label == "prefill":
            prefill = (p0, i)
        start = i
        for _ in range(n_units):
            unit = units.get(names[i])
            assert unit and names[i:i + len(unit)] == unit, f"unexpected step at {i}"
            i += len(unit)
        out.append((label, start, i))
    assert i == len(names), "dispatches left over"
    return out, prefill


def summarize(args, trace_dir, fetch_dir, write_dir):
    import glob
    from paper_2607_27692_amd.inputs import WORKLOADS
    w = WORKLOADS[args.workload]
    steps = min(args.steps, w.steps)
    trace = _read_csv(glob.glob(os.path.join(trace_dir, "*kernel_trace.csv"))[0])
    stats = _read_csv(glob.glob(os.path.join(trace_dir, "*kernel_stats.csv"))[0])
    trace.sort(key=lambda r: int(r["Dispatch_Id"]))
    lib = [(r, _lib_name(r["Kernel_Name"])) for r in trace]
    lib = [(r, n) for r, n in lib if n]
    names = [n for _, n in lib]
    passes, prefill = _passes(names, w, steps, args.warmup)
    dur = lambda r: (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3  # noqa: E731

    wflag = "" if w.name == "128k" else f" --workload {w.name}"
    lines = [f"# Kernel durations, {w.name} workload, rocprofv3 kernel trace",
             "command: cd /tmp && export TMPDIR=/tmp && rocprofv3 --kernel-trace --stats -f csv "
             f"-d <out>/kt -o kt -- python3 -u <repo>/bench.py --no-cpu-baseline{wflag}",
             f"summary: python bench.py --summarize <out>/kt <out>/pmc_fetch <out>/pmc_write{wflag}",
             "",
             "## rocprofv3 --stats (every dispatch of the run: prefills, warm-up and all passes)",
             f"{'kernel':60s} {'library name':14s} {'calls':>6s} {'avg_us':>9s} {'min_us':>9s} {'max_us':>9s} {'share':>7s}"]
    for r in stats:
        name = _lib_name(r["Name"]) or ""
        lines.append(f"{r['Name'][:60]:60s} {name:14s} {int(r['Calls']):6d} "
                     f"{float(r['AverageNs']) / 1e3:9.2f} {float(r['MinNs']) / 1e3:9.2f} "
                     f"{float(r['MaxNs']) / 1e3:9.2f} {float(r['Percentage']):6.2f}%")
    lines += ["", f"## per pass, decode-step dispatches only ({steps} steps per pass)",
              f"{'pass':18s} {'kernel':14s} {'launches':>8s} {'avg_us':>9s}"]
    for label, a, b in passes:
        acc = {}
        for r, n in lib[a:b]:
            acc.setdefault(n, []).append(dur(r))
        for n in ("retopk_sim", "retopk_score", "retopk_scan", "retopk_filter", "retopk_final",
                  "dense_chunk", "dense_merge"):
            if n in acc:
                v = acc[n]
                lines.append(f"{label:18s} {n:14s} {len(v):8d} {sum(v) / len(v):9.2f}")
    acc = {}
    for r, n in lib[prefill[0]:prefill[1]]:
        acc.setdefault(n, []).append(dur(r))
    lines += ["", f"## prefill initialisation, {w.cache_cap} prompt-tail positions (timed handle)",
              f"{'kernel':14s} {'launches':>8s} {'avg_us':>9s} {'sum_us':>9s}"]
    for n, v in acc.items():
        lines.append(f"{n:14s} {len(v):8d} {sum(v) / len(v):9.2f} {sum(v):9.1f}")
    kt_path = os.path.join(ROOT, "profiles", f"kernels_{w.name}.txt")

    # ---- counters: FETCH_SIZE / WRITE_SIZE, scaled by the copy calibration ----
    def counters(d):
        rows = _read_csv(glob.glob(os.path.join(d, "*counter_collection.csv"))[0])
        rows.sort(key=lambda r: int(r["Dispatch_Id"]))
        libr = [(float(r["Counter_Value"]), _lib_name(r["Kernel_Name"])) for r in rows]
        copies = [float(r["Counter_Value"]) for r in rows
                  if r["Kernel_Name"].startswith("__amd_rocclr_copyBuffer")]
        return [(v, n) for v, n in libr if n], copies
    fetch, fcopy = counters(fetch_dir)
    write, wcopy = counters(write_dir)
    assert [n for _, n in fetch] == names == [n for _, n in write], "dispatch sequences differ"
    copy_kib = COPY_BYTES / 1024
    f_big = [v for v in fcopy if v > copy_kib / 4]
    w_big = [v for v in wcopy if v > copy_kib / 4]
    f_factor = copy_kib / (sum(f_big) / len(f_big))
    w_factor = copy_kib / (sum(w_big) / len(w_big))
    digest = kernel_source_digest()
    written = [kt_path]
    by_label = {lab: i for i, (lab, _, _) in enumerate(passes)}
    for kernel, label in (("retopk_score", "retopk timed"), ("retopk_scan", "exact timed"),
                          ("dense_chunk", "full timed")):
        pass_idx = by_label[label]
        _, a, b = passes[pass_idx]
        fv = [v for v, n in fetch[a:b] if n == kernel]
        wv = [v for v, n in write[a:b] if n == kernel]
        fk, wk = sum(fv) / len(fv), sum(wv) / len(wv)
        traffic = (fk * f_factor + wk * w_factor) * 1024
        out = [f"# HBM traffic per launch of {kernel}, {w.name} workload, rocprofv3 counters",
               "command_fetch: cd /tmp && export TMPDIR=/tmp && timeout -s KILL 300 rocprofv3 "
               "--pmc FETCH_SIZE -f csv -d <out>/pmc_fetch -o pmc -- python3 -u <repo>/bench.py "
               f"--no-cpu-baseline --copy-calibration{wflag}",
               "command_write: the same with --pmc WRITE_SIZE -d <out>/pmc_write",
               f"summary: python bench.py --summarize <out>/kt <out>/pmc_fetch <out>/pmc_write{wflag}",
               f"copy_bytes: {COPY_BYTES}",
               f"copy_fetch_kib: {sum(f_big) / len(f_big):.1f}",
               f"copy_write_kib: {sum(w_big) / len(w_big):.1f}",
               f"fetch_factor: {f_factor:.4f}",
               f"write_factor: {w_factor:.4f}",
               f"pass: {passes[pass_idx][0]} (first timed pass)",
               f"launches: {len(fv)}",
               f"fetch_kib_per_launch: {fk:.1f}",
               f"write_kib_per_launch: {wk:.1f}",
               f"traffic_bytes_per_launch: {traffic:.0f}",
               f"kernel_source_sha256: {digest}"]
        path = os.path.join(ROOT, "profiles", f"traffic_{kernel}_{w.name}.txt")
        with open(path, "w") as f:
            f.write("\n".join(out) + "\n")
        written.append(path)
        lines.append(f"traffic {kernel}: {traffic / 1e6:.2f} MB per launch "
                     f"(fetch {fk:.0f} KiB x {f_factor:.3f}, write {wk:.0f} KiB x {w_factor:.3f})")
    with open(kt_path, "w") as f:
        f.write("\n".join(lines) + "\n")
    for p_ in written:
        log(f"[bench] wrote {p_}")


if __name__ == "__main__":
    main()
