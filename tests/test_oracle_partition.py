"""Pins of the exhaustive partitioner (appendix "Memory-constrained pipeline
partitioning") against hand-solved instances and an independent textbook
method for the unconstrained case."""
import numpy as np
import pytest

from oracle import partition as op

INF = float("inf")


def test_classic_linear_partition():
    # The textbook instance: 1..9 over 3 workers; the best largest sum is 17
    # ({1..5} = 15, {6, 7} = 13, {8, 9} = 17), reached by that split only.
    t = list(range(1, 10))
    feas, best, cuts = op.partition(t, [0] * 9, [0] * 9, 3, INF)
    assert feas and best == 17
    assert cuts == [(0, 5, 7, 9)]


def test_uniform_layers_split_evenly():
    feas, best, cuts = op.partition([1.0] * 8, [0] * 8, [0] * 8, 4, INF)
    assert feas and best == 2.0 and cuts == [(0, 2, 4, 6, 8)]


def test_in_flight_weights_move_layers_downstream():
    # 4 equal layers, 2 stages, activations only: stage 1 holds w_1 = 2
    # micro-batches, stage 2 holds one. With a = 1 per layer and B = 2, an even
    # split needs 2 * 2 = 4 on stage 1 (too much); 1 + 3 needs 2 and 3 (too
    # much); no split fits. With B = 3: only (1 | 3) fits, time 3.
    t, s, a = [1.0] * 4, [0.0] * 4, [1.0] * 4
    feas, best, cuts = op.partition(t, s, a, 2, 3.0)
    assert feas and best == 3.0 and cuts == [(0, 1, 4)]
    # at B = 4 the balanced split fits again
    feas, best, cuts = op.partition(t, s, a, 2, 4.0)
    assert feas and best == 2.0 and cuts == [(0, 2, 4)]


def test_static_bytes_are_paid_once():
    # static bytes do not scale with w_j: s = 1 per layer, a = 0, B = 2 allows
    # at most two layers per stage whatever the stage position
    feas, best, cuts = op.partition([1.0, 5.0, 1.0, 1.0], [1.0] * 4, [0.0] * 4, 2, 2.0)
    assert feas and best == 6.0 and cuts == [(0, 2, 4)]


def test_fallback_minimises_overshoot_then_time():
    # B = 2 with a = 1 per layer, 3 layers on 2 stages: (1 | 2) gives memories
    # (2, 2) and fits; B = 1.5 fits nothing. Overshoots: (1 | 2) -> (0.5, 0.5),
    # (2 | 1) -> (2.5, 0). The fallback keeps (1 | 2).
    t, s, a = [1.0, 1.0, 1.0], [0.0] * 3, [1.0] * 3
    feas, best, cuts = op.partition(t, s, a, 2, 1.5)
    assert not feas and best == (0.5, 2.0) and cuts == [(0, 1, 3)]
    # equal overshoot, different time: static bytes 1 per layer, B = 2, so
    # 5 layers on 2 stages overshoot by 1 at best, with (2 | 3) or (3 | 2);
    # times [1, 1, 1, 5, 1] give 7 and 6, and the fallback keeps (3 | 2)
    feas, best, cuts = op.partition([1.0, 1.0, 1.0, 5.0, 1.0], [1.0] * 5, [0.0] * 5, 2, 2.0)
    assert not feas and best == (1.0, 6.0) and cuts == [(0, 3, 5)]


def _greedy_min_max(t, N):
    """Textbook method for min-max linear partition: binary search over the
    answer among all contiguous sums, with a greedy fill as the test."""
    L = len(t)
    cand = sorted({sum(t[i:j]) for i in range(L) for j in range(i + 1, L + 1)})

    def stages_needed(cap):
        n, acc = 1, 0.0
        for x in t:
            if x > cap:
                return INF
            if acc + x > cap:
                n, acc = n + 1, x
            else:
                acc += x
        return n

    lo, hi = 0, len(cand) - 1
    while lo < hi:
        mid = (lo + hi) // 2
        if stages_needed(cand[mid]) <= N:
            hi = mid
        else:
            lo = mid + 1
    return cand[lo]


@pytest.mark.parametrize("seed", range(12))
def test_unconstrained_matches_greedy_binary_search(seed):
    r = np.random.default_rng(seed)
    L = int(r.integers(3, 10))
    N = int(r.integers(1, L + 1))
    t = [float(x) for x in r.integers(1, 20, size=L)]
    feas, best, cuts = op.partition(t, [0.0] * L, [0.0] * L, N, INF)
    assert feas and best == _greedy_min_max(t, N)
    for c in cuts:
        assert c[0] == 0 and c[-1] == L and all(x < y for x, y in zip(c, c[1:]))


def test_partition_count_is_binomial():
    from math import comb
    for L in range(1, 9):
        for N in range(1, L + 1):
            assert sum(1 for _ in op.all_partitions(L, N)) == comb(L - 1, N - 1)
