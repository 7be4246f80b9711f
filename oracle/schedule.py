"""Oracle for the two-stream layer pipeline's timing (Sec. 4.3, Eq. 1).

TEST INFRASTRUCTURE (see the package docstring). An explicit event-by-event
simulation of two in-order queues: the copy queue runs the layer loads back to
back; the compute queue runs layer l's work once layer l-1's work is done and
layer l's load has landed. Used to pin the closed-form bound the benchmark
reports as the least exposure any schedule can reach.
"""
from __future__ import annotations

from typing import Sequence, Tuple


def simulate(load_ms: Sequence[float], compute_ms: Sequence[float]) -> Tuple[float, float]:
    """Returns (makespan, exposed) where exposed = makespan - sum(compute).

    Both queues start at time 0 with every load already enqueued.
    """
    n = len(load_ms)
    assert len(compute_ms) == n
    copy_free = 0.0
    compute_free = 0.0
    for l in range(n):
        load_done = copy_free + load_ms[l]
        copy_free = load_done
        start = max(compute_free, load_done)
        compute_free = start + compute_ms[l]
    return compute_free, compute_free - sum(compute_ms)


def synchronous(load_ms: Sequence[float], compute_ms: Sequence[float]) -> float:
    """No overlap: all loads, then all compute (the synchronous cost of Eq. 1)."""
    return sum(load_ms) + sum(compute_ms)
