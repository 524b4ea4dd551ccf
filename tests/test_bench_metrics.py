"""Host logic of the benchmark: the fidelity measures it reports (support recall,
retained mass, cosine) on hand-made inputs, the split of a profile into passes,
the one-GPU guard and the traffic lookup."""
import os
import sys

import numpy as np

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
import bench  # noqa: E402


def test_support_recall():
    assert bench.support_recall([1, 2, 3, -1], [1, 2, 3, -1]) == 1.0
    assert bench.support_recall([1, 2, 5, 6], [1, 2, 3, 4]) == 0.5
    assert bench.support_recall([-1, -1], [7, 8]) == 0.0


def test_retained_mass():
    p = np.array([0.5, 0.25, 0.125, 0.125])
    assert bench.retained_mass([0, 1, -1], p) == 0.75
    assert bench.retained_mass([0, 1, 2, 3], p) == 1.0


def test_cosine():
    assert abs(bench.cosine([1, 0], [1, 0]) - 1.0) < 1e-12
    assert abs(bench.cosine([1, 0], [0, 1])) < 1e-12
    assert abs(bench.cosine([1, 1], [2, 2]) - 1.0) < 1e-12


def _dispatches(w, steps, warmup, n_pf, exact_heads_at=()):
    """A dispatch-name sequence in the order bench.py issues it: every handle's
    batched prefill (n_pf triples), the warm-up's three step kinds per step, the
    timed prefill alone, the six passes, the two warm passes and the labelling
    pass."""
    pf = ["prefill_score", "retopk_filter", "retopk_final"]
    sel = ["retopk_sim", "retopk_score", "retopk_filter", "retopk_final"]
    scan = ["retopk_scan", "retopk_filter", "retopk_final"]
    dense = ["dense_chunk", "dense_merge"]
    names = pf * n_pf
    for t in range(min(warmup, w.steps)):
        names += (scan if t in exact_heads_at else sel) + scan + dense
    names += pf * n_pf                                   # the timed prefill
    for kind in ("retopk", "exact", "full", "retopk", "exact", "full", "retopk", "exact",
                 "retopk"):
        names += pf * n_pf
        for t in range(steps):
            names += {"retopk": scan if t in exact_heads_at else sel, "exact": scan,
                      "full": dense}[kind]
    return names


def test_passes_split_the_dispatch_sequence():
    from paper_2607_27692_amd.inputs import WORKLOADS
    w = WORKLOADS["128k"]
    steps, warmup, n_pf = 5, 2, 13
    names = _dispatches(w, steps, warmup, n_pf, exact_heads_at=(3,))
    passes, prefill = bench._passes(names, w, steps, warmup)
    labels = [p[0] for p in passes]
    assert labels == ["warm-up", "prefill", "retopk timed", "exact timed", "full timed",
                      "retopk profiled", "exact profiled", "full profiled", "retopk warm",
                      "exact warm", "step kinds"]
    assert prefill[1] - prefill[0] == 3 * n_pf
    assert names[prefill[0]:prefill[1]] == ["prefill_score", "retopk_filter", "retopk_final"] * n_pf
    by = {p[0]: (p[1], p[2]) for p in passes}
    a, b = by["retopk timed"]
    assert b - a == 4 * (steps - 1) + 3                  # one refresh-like step
    a, b = by["exact timed"]
    assert names[a:b] == ["retopk_scan", "retopk_filter", "retopk_final"] * steps
    a, b = by["full timed"]
    assert names[a:b] == ["dense_chunk", "dense_merge"] * steps
    assert by["prefill"][0] == by["prefill"][1]          # no steps in the prefill pass


def test_more_than_one_gpu_is_refused():
    """bench.py --gpus N with N > 1 exits with a message before touching a GPU."""
    import subprocess
    r = subprocess.run([sys.executable, os.path.join(os.path.dirname(bench.__file__), "bench.py"),
                        "--gpus", "2"], capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "exactly one GPU" in r.stderr
    assert r.stdout == ""


def test_traffic_is_reported_only_for_the_profiled_source(monkeypatch):
    """The measured traffic of a kernel comes from its counter summary only while the
    kernel source still has the digest recorded with it."""
    path = os.path.join(bench.ROOT, "profiles", "traffic_retopk_score_128k.txt")
    with open(path) as f:
        fields = dict(line.split(":", 1) for line in f if ":" in line)
    digest = fields["kernel_source_sha256"].strip()
    expected = int(float(fields["traffic_bytes_per_launch"]))
    monkeypatch.setattr(bench, "kernel_source_digest", lambda: digest)
    assert bench.traffic_per_launch("retopk_score", "128k") == expected
    monkeypatch.setattr(bench, "kernel_source_digest", lambda: "0" * 64)
    assert bench.traffic_per_launch("retopk_score", "128k") is None
    assert bench.traffic_per_launch("no_such_kernel", "128k") is None


def test_trace_symbols_name_every_score_build():
    # The decode step's scoring launch and the scan-only launch are two builds of
    # one kernel template, for every dtype, head dim and group size.
    for dt in ("unsigned short", "float"):
        for d in (64, 128):
            for g in (1, 2, 4, 8):
                sym = f"void retopk::k_score<{dt}, {d}, {g}, %s>(retopk::StepArgs, retopk::Ws)"
                assert bench._lib_name(sym % "true") == "retopk_score"
                assert bench._lib_name(sym % "false") == "retopk_scan"
    assert bench._lib_name("void retopk::k_final<unsigned short, 128, true>(a)") == "retopk_final"
    assert bench._lib_name("void at::native::reduce_kernel<512, 1>(x)") is None
