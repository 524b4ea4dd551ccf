"""The fidelity measures the benchmark reports (support recall, retained mass,
cosine), on hand-made inputs."""
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
