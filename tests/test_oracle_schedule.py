"""Pins of the oracle's schedule: Alg. 1 counters, stamps and the bound of Eq. (2)."""
import json
import os

import pytest

from oracle import pipeline, schedule


GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_canonical_order_tiny_stage_by_hand():
    # Alg. 1 at K = 4, delay = 3 (stage 0 of a 4-stage pipeline), M = 16, written
    # out by hand: four warm-up forwards, then B_j / update after every 4th B /
    # F_{j+4}; the last three backwards drain the pipeline.
    ev = schedule.canonical_events(16, 4, 3)
    expect = ("F0 F1 F2 F3 B0 F4 B1 F5 B2 F6 B3 S F7 B4 F8 B5 F9 B6 F10 B7 S F11 "
              "B8 F12 B9 F13 B10 F14 B11 S F15 B12 B13 B14 B15 S")
    assert schedule.events_to_string(ev) == expect


@pytest.mark.parametrize("M,K,delay", [(16, 4, 3), (64, 8, 3), (64, 8, 0), (128, 16, 7),
                                       (10, 1, 0), (10, 3, 5), (7, 2, 9), (1, 1, 0), (0, 2, 1)])
def test_counters_match_closed_form_stamps(M, K, delay):
    ev = schedule.canonical_events(M, K, delay)
    assert len(ev) == 2 * M + M // K
    tF, tB, delta, n_upd = schedule.run_events(ev, K, delay)
    cF, cB, cD = schedule.closed_form_stamps(M, K, delay)
    assert (tF, tB, delta) == (cF, cB, cD)
    assert n_upd == M // K
    assert all(0 <= d <= schedule.delta_bound(delay, K) for d in delta)


@pytest.mark.parametrize("M,K,delay,total", [(16, 4, 3, 9), (64, 8, 3, 21), (64, 8, 0, 0),
                                             (128, 16, 7, 49)])
def test_total_crossings_of_the_stage_workloads(M, K, delay, total):
    # When K divides M and delay <= K every window after the first is crossed
    # by exactly `delay` backwards: sum Delta = delay * (M/K - 1).
    _, _, delta, _ = schedule.run_events(schedule.canonical_events(M, K, delay), K, delay)
    assert sum(delta) == total == delay * (M // K - 1)
    assert max(delta) == (1 if delay else 0)


def test_protocol_errors():
    sc = schedule.StageCounters(K=2, delay=1)
    sc.forward(0)
    with pytest.raises(schedule.ProtocolError):
        sc.forward(2)                       # out of order
    sc.forward(1)
    with pytest.raises(schedule.ProtocolError):
        sc.forward(2)                       # q = 2 > delay: backpressure
    with pytest.raises(schedule.ProtocolError):
        sc.backward(1)                      # backwards are FIFO
    with pytest.raises(schedule.ProtocolError):
        sc.step()                           # not due
    sc.backward(0)
    sc.backward(1)
    assert sc.step_due
    with pytest.raises(schedule.ProtocolError):
        sc.forward(2)                       # update pending
    assert sc.step() == 1
    with pytest.raises(schedule.ProtocolError):
        sc.backward(2)                      # no forward pending


@pytest.mark.parametrize("M", [6, 8])
@pytest.mark.parametrize("K", [1, 2, 3, 4])
@pytest.mark.parametrize("delay", [0, 1, 2, 3, 5])
def test_bound_holds_over_every_admissible_interleaving(M, K, delay):
    """Eq. (2) by brute force: no interleaving Alg. 1 admits exceeds ceil(delay/K),
    and the canonical order reaches the bound whenever M leaves room for it."""
    worst = schedule.max_delta_brute_force(M, K, delay)
    bound = schedule.delta_bound(delay, K)
    assert worst <= bound
    _, _, delta, _ = schedule.run_events(schedule.canonical_events(M, K, delay), K, delay)
    assert max(delta) <= worst
    if M >= K + delay:
        assert max(delta) == bound


def test_bound_needs_the_admission_rule():
    # Without the admission rule a stage may run arbitrarily far ahead and the
    # bound of Eq. (2) no longer holds.
    assert schedule.max_delta_brute_force(10, 2, 3, admission=False) == 4 > schedule.delta_bound(3, 2)


def test_brute_force_enumerates_all_orders():
    # delay >= M - 1 and K > M: every ballot sequence of M forwards and M
    # backwards is admissible, so the count is the Catalan number C_M.
    assert [schedule.count_orders(M, M + 1, M) for M in range(1, 8)] == [1, 2, 5, 14, 42, 132, 429]
    # delay = 0 forces strict alternation.
    assert schedule.count_orders(7, 3, 0) == 1


def test_paper_worked_bounds():
    with open(os.path.join(GOLDEN, "bound_worked_values.json")) as fh:
        cases = json.load(fh)["cases"]
    for c in cases:
        # first stage: i = 1, downstream depth N - 1
        assert schedule.delta_bound(c["N"] - 1, c["a"]) == c["delta_max"], c["cite"]


def test_paper_worked_bound_n8_brute_force():
    # Sec. 4.2: for an 8-stage pipeline the first stage (delay 7) crosses at most
    # 2 updates at a = 4 and 1 at a = 8; every admissible order respects it and
    # the canonical order attains it.
    assert schedule.max_delta_brute_force(11, 4, 7) == 2
    assert schedule.max_delta_brute_force(10, 8, 7) == 1


def test_bubble_efficiency_worked_values():
    with open(os.path.join(GOLDEN, "efficiency_worked_values.json")) as fh:
        cases = json.load(fh)["cases"]
    for c in cases:
        assert pipeline.eta_flush(c["m"], c["N"]) == pytest.approx(c["eta_flush"], rel=1e-12)
        assert pipeline.eta_interleaved(c["m"], c["N"], c["V"]) == pytest.approx(c["eta_inter"], rel=1e-12)


def test_table1_projection():
    with open(os.path.join(GOLDEN, "table1_projection.json")) as fh:
        cols = json.load(fh)["columns"]
    for c in cols:
        proj = pipeline.paci_throughput_proxy(c["flush"], c["m"], c["gpus"])
        assert abs(proj - c["paci"]) <= 0.005 + 1e-9, c


def test_flush_order_by_hand():
    # Synchronous 1F1B with a flush at K = 4: at delay 3 each window fills the
    # stage, drains it and updates; at delay 1 it alternates after one warm-up.
    assert schedule.events_to_string(schedule.flush_events(8, 4, 3)) == \
        "F0 F1 F2 F3 B0 B1 B2 B3 S F4 F5 F6 F7 B4 B5 B6 B7 S"
    assert schedule.events_to_string(schedule.flush_events(8, 4, 1)) == \
        "F0 F1 B0 F2 B1 F3 B2 B3 S F4 F5 B4 F6 B5 F7 B6 B7 S"
    # a trailing partial window has no update
    assert schedule.events_to_string(schedule.flush_events(5, 2, 0)) == "F0 B0 F1 B1 S F2 B2 F3 B3 S F4 B4"


@pytest.mark.parametrize("M,K,delay", [(16, 4, 3), (64, 8, 3), (128, 16, 7), (10, 3, 5), (7, 2, 9), (0, 2, 1)])
def test_flush_order_has_no_crossings(M, K, delay):
    """Alg. 1's counters accept the flush order (it never exceeds the admission
    window) and stamp every micro-batch with Delta = 0, against sum Delta =
    delay * (M/K - 1) for the asynchronous order when delay <= K divides M."""
    ev = schedule.flush_events(M, K, delay)
    assert len(ev) == 2 * M + M // K
    tF, tB, delta, n_upd = schedule.run_events(ev, K, delay)
    assert delta == [0] * M and n_upd == M // K
    assert tF == [i // K for i in range(M)] == tB


@pytest.mark.parametrize("M,K,delay", [(6, 2, 1), (6, 3, 2), (8, 4, 3), (6, 1, 2)])
def test_flush_order_is_one_of_the_admissible_interleavings(M, K, delay):
    # the synchronous order is a special case of Alg. 1: a stage that waits
    flush = schedule.flush_events(M, K, delay)
    assert any(list(o) == flush for o in schedule.all_admissible_orders(M, K, delay))
