"""CPU: the benchmark's measurement arithmetic against independent formulations
(brute-force pair counting, the oracle's event-by-event two-queue schedule, the
permutation flow-shop recurrence, the oracle planner's block-pair list)."""

import pytest

import bench
from oracle import datamove as odm
from oracle import schedule as osched
from paper_2603_23049_amd import synth


def _pairs_brute(prefix_lens, suffix_lens):
    n = 0
    for p, s in zip(prefix_lens, suffix_lens):
        for i in range(s):                 # suffix row i sits at position p + i
            for j in range(p + s):
                n += j <= p + i
    return n


@pytest.mark.parametrize("pl,sl", [([0], [1]), ([1], [1]), ([17, 0, 256], [5, 64, 3]), ([15, 16], [63, 2])])
def test_attention_flops_counts_causal_pairs(pl, sl):
    assert bench.attention_flops(pl, sl, 8, 64) == 4 * 64 * 8 * _pairs_brute(pl, sl)


def test_attention_flops_of_the_benchmark_layer():
    b = synth.l8b_layer()
    assert bench.attention_flops(b.prefix_lens, b.suffix_lens, b.num_q_heads, b.head_dim) == 70_875_348_992


@pytest.mark.parametrize("c,p,n", [(1.2, 0.07, 32), (1.22, 2.43, 32), (2.14, 0.87, 80), (1.0, 1.0, 5), (0.5, 3.0, 1)])
def test_two_queue_bound_matches_event_simulation(c, p, n):
    makespan, _ = osched.simulate([c] * n, [p] * n)
    assert bench.flow_shop_exposure(c, p, n) == pytest.approx(makespan - n * p, rel=1e-12, abs=1e-12)


def _flow_shop_recurrence(times, n):
    """Completion time of job n-1 on the last machine, jobs in order, each machine in
    order: C[i][k] = max(C[i-1][k], C[i][k-1]) + t_k."""
    prev = [0.0] * len(times)
    for _ in range(n):
        cur = []
        for k, t in enumerate(times):
            cur.append(max(prev[k], cur[k - 1] if k else 0.0) + t)
        prev = cur
    return prev[-1]


@pytest.mark.parametrize("times,n", [((1.2, 2.4, 1.8), 32), ((0.1, 0.2, 0.3), 7), ((3.0, 1.0, 1.0), 4),
                                     ((1.0, 1.0, 1.0), 1)])
def test_three_queue_bound_matches_recurrence(times, n):
    assert bench.flow_shop3_makespan(*times, n) == pytest.approx(_flow_shop_recurrence(times, n), rel=1e-12)


@pytest.mark.parametrize("mk", [synth.tiny, synth.l8b_layer, synth.l70b_pipe80])
def test_load_bytes_equal_the_planned_block_pairs(mk):
    b = mk()
    src, dst, slots, cu = odm.plan(b.prefix_lens, b.suffix_lens, b.block_tables, b.host_blocks, b.block_size)
    block_bytes = b.block_size * b.num_kv_heads * b.head_dim * 2
    assert bench.load_bytes(b.prefix_lens, b.num_kv_heads, b.head_dim) == 2 * len(src) * block_bytes
    assert bench.append_bytes(b.T, b.num_kv_heads, b.head_dim) == 2 * 2 * len(slots) * b.num_kv_heads * b.head_dim * 2
