"""The drift workloads separate Eq. (1) from weight stashing (oracle only).

Eq. (1) (Sec. 3.1; appendix "PyTorch modifications for asynchronous
execution"): a stale backward differentiates the activations of its forward at
the parameters current when it runs. Weight stashing (PipeDream's remedy, which
PACI does not use) would differentiate at the forward's parameters instead. A
GPU parity test can only tell the two apart if, on its workload, they differ by
more than the tolerance. For every workload of the drift parity tests this
checks, with the oracle alone and under the same forced G as the GPU test uses
(here the oracle's own), that
* every stale backward's input gradient differs between the two readings by at
  least 5 tolerances;
* in every window with a stale backward, at least half of the G tensors do, and
  the largest gap is at least 5 tolerances;
so that the GPU test's requirement (3 tolerances away from stashing, within 1
of the oracle) cannot be met by a stage that stashed its weights.
"""
import numpy as np
import pytest

from parity import DRIFT, Inputs, drift_cfg, oracle_replay, rel_err, tol
from oracle import stage as ostage


@pytest.mark.parametrize("name", sorted(DRIFT))
def test_drift_workload_separates_current_from_stashed_weights(name):
    c = drift_cfg(name)
    inp = Inputs(c, 1, c["M"])
    o = oracle_replay(c, inp)
    Gs = o["G"]
    stash = ostage.replay_with_version_store(c, inp.oracle_params(), c["K"], c["delay"], inp.x,
                                             None if c["kind"] == "last" else inp.dy,
                                             inp.tgt if c["kind"] == "last" else None, backward_at="forward",
                                             grad_hook=lambda s, G: {n: Gs[s][n].copy() for n in G})
    t = tol(c, "grad")
    stale = [i for i in range(c["M"]) if o["tB"][i] > o["tF"][i]]
    assert stale, "the workload has no stale backward"
    if c["kind"] != "first":
        gaps = [rel_err(stash["grad_in"][i], o["grad_in"][i]) / t for i in stale]
        assert min(gaps) >= 5.0, f"input-gradient gap only {min(gaps):.2f} tolerances"
    for s in range(len(Gs)):
        if not any(o["tB"][i] == s for i in stale):
            # no stale backward in this window: both readings agree exactly
            for n in Gs[s]:
                assert np.array_equal(stash["G"][s][n], Gs[s][n])
            continue
        gaps = {n: rel_err(stash["G"][s][n], Gs[s][n]) / t for n in Gs[s]}
        assert max(gaps.values()) >= 5.0, gaps
        assert sum(g >= 5.0 for g in gaps.values()) >= len(gaps) / 2, gaps


def test_stash_and_current_agree_without_drift():
    """At delay 0 no backward is stale, so the two readings are the same
    replay, bit for bit (a check of the stash variant itself)."""
    c = drift_cfg("drift_ragged_bf16")
    c["delay"] = 0
    inp = Inputs(c, 1, 8)
    cur = ostage.replay_with_version_store(c, inp.oracle_params(), c["K"], 0, inp.x, inp.dy, None)
    st = ostage.replay_with_version_store(c, inp.oracle_params(), c["K"], 0, inp.x, inp.dy, None,
                                          backward_at="forward")
    for a, b in zip(cur["grad_in"], st["grad_in"]):
        assert np.array_equal(a, b)
