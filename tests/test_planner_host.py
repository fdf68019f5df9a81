"""The library's host-only stage planning calls against the exhaustive oracle
(partitioner) and the paper's printed numbers (Eqs. 3-5). No device work."""
import json
import math
import os

import numpy as np
import pytest

from oracle import partition as opart

binding = pytest.importorskip("paper_2606_07881_amd.binding",
                              reason="libpaci_stage.so not built (python -m paper_2606_07881_amd.build)")
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
INF = float("inf")


def _instance(seed):
    """Integer-valued profiles (exact sums) with budgets from loose to infeasible."""
    r = np.random.default_rng(seed)
    L = int(r.integers(2, 11))
    N = int(r.integers(1, min(L, 6) + 1))
    t = r.integers(1, 30, size=L).astype(float)
    s = r.integers(0, 8, size=L).astype(float)
    a = r.integers(0, 5, size=L).astype(float)
    total = s.sum() + N * a.sum()
    budget = [INF, float(r.integers(1, int(total) + 2)), float(r.integers(0, 4))][seed % 3]
    return t, s, a, N, budget


@pytest.mark.parametrize("seed", range(60))
def test_partition_matches_exhaustive_search(seed):
    t, s, a, N, budget = _instance(seed)
    cuts, mt, mo = binding.partition(t, s, a, N, budget)
    feas, best, opt = opart.partition(list(t), list(s), list(a), N, budget)
    if feas:
        assert mo == 0.0 and mt == best
    else:
        assert mo > 0.0 and (mo, mt) == best
    assert tuple(int(c) for c in cuts) in opt     # one of the optimal partitions


def test_partition_on_a_stage_profile():
    # 24 equal blocks (GPT-2-medium depth) plus a heavier embedding layer and
    # LM-head layer, 4 stages; activation bytes dominate, so the first stage
    # (w_1 = 4 in flight) is given fewer blocks when the budget binds.
    t = [3.0] + [10.0] * 24 + [12.0]
    s = [200.0] + [50.0] * 24 + [200.0]
    a = [8.0] + [40.0] * 24 + [60.0]
    cuts_free, mt_free, mo_free = binding.partition(t, s, a, 4, INF)
    assert mo_free == 0.0 and mt_free == opart.partition(t, s, a, 4, INF)[1]
    # at this budget the optimum is unique: embedding + 4 blocks on the first
    # stage, 7 blocks + LM head on the last
    cuts, mt, mo = binding.partition(t, s, a, 4, 1100.0)
    assert mo == 0.0 and mt == 80.0 and cuts.tolist() == [0, 5, 11, 19, 26]
    assert opart.partition(t, s, a, 4, 1100.0) == (True, 80.0, [(0, 5, 11, 19, 26)])
    mem = [sum(s[cuts[j]:cuts[j + 1]]) + (4 - j) * sum(a[cuts[j]:cuts[j + 1]]) for j in range(4)]
    assert max(mem) <= 1100.0 and mt > mt_free


def test_partition_rejects_bad_arguments():
    with pytest.raises(binding.PaciError):
        binding.partition([1.0, 2.0], [0.0, 0.0], [0.0, 0.0], 3)        # more stages than layers
    with pytest.raises(binding.PaciError):
        binding.partition([1.0, -2.0], [0.0, 0.0], [0.0, 0.0], 1)       # negative time
    with pytest.raises(binding.PaciError):
        binding.partition([1.0, 2.0], [0.0, math.nan], [0.0, 0.0], 1)
    with pytest.raises(binding.PaciError):
        binding.partition([1.0, 2.0], [0.0, 0.0], [0.0, 0.0], 1, math.nan)
    with pytest.raises(binding.PaciError):
        binding.partition([1.0, 2.0], [0.0, 0.0], [0.0, 0.0], 1, -1.0)
    with pytest.raises(binding.PaciError):
        binding.partition([1.0, 2.0], [0.0, 0.0], [0.0, 0.0], 0)


def test_efficiency_formulas_reproduce_the_papers_numbers():
    with open(os.path.join(GOLDEN, "efficiency_worked_values.json")) as fh:
        for c in json.load(fh)["cases"]:
            assert binding.lib.paci_eta_flush(c["m"], c["N"]) == pytest.approx(c["eta_flush"], rel=1e-12)
            assert binding.lib.paci_eta_interleaved(c["m"], c["N"], c["V"]) == pytest.approx(c["eta_inter"],
                                                                                            rel=1e-12)
    with open(os.path.join(GOLDEN, "table1_projection.json")) as fh:
        for c in json.load(fh)["columns"]:
            proj = binding.lib.paci_throughput_proxy(c["flush"], c["m"], c["gpus"])
            assert abs(proj - c["paci"]) <= 0.005 + 1e-9, c
    assert math.isnan(binding.lib.paci_eta_flush(0, 4))
    assert math.isnan(binding.lib.paci_eta_interleaved(4, 4, 0))
