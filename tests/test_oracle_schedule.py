"""Pins for the pipeline timing oracle against the paper's statements (CPU only)."""
import numpy as np

from oracle import schedule


def test_overlap_leaves_one_layer_of_load_when_compute_dominates():
    # Sec. 4.3: with per-layer load below per-layer compute, only about one
    # layer's transfer, C1/n, stays exposed.
    n, c, p = 32, 0.4, 1.0
    makespan, exposed = schedule.simulate([c] * n, [p] * n)
    assert abs(exposed - c) < 1e-12
    assert abs(exposed - (n * c) / n) < 1e-12


def test_synchronous_cost_is_eq1():
    # Eq. 1: loading N1 cached tokens' KV and offloading N2 new tokens' KV costs
    # C1 in total regardless of the hit ratio; compute costs (N2/N) C2.
    N, N1 = 8192, 4096
    N2 = N - N1
    C1, C2 = 0.5, 4.0
    load = (N1 / N) * C1
    offload = (N2 / N) * C1
    compute = (N2 / N) * C2
    assert abs((load + offload + compute) - (C1 + (N2 / N) * C2)) < 1e-12
    assert abs(schedule.synchronous([load], [compute + offload]) - (C1 + (N2 / N) * C2)) < 1e-12


def test_copy_bound_pipeline_exposes_nearly_all_load():
    n, c, p = 32, 1.22, 0.057
    makespan, exposed = schedule.simulate([c] * n, [p] * n)
    assert abs(makespan - (n * c + p)) < 1e-9
    assert exposed / n > 0.95 * c
