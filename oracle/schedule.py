"""Stage event rule, version stamps and the inconsistency bound (test infrastructure).

Notation: the paper's stage i of N (one-indexed) has downstream depth N - i; here
that depth is ``delay``. Its accumulation factor a is ``K``. A stage admits a
forward only while its unresolved-forward counter q satisfies q <= delay
(Sec. 3.2 and the appendix "Inconsistency bound"), counts local backwards in c
and applies one optimizer update when c reaches K, resetting c (Alg. 1). The
version t is the number of local updates applied so far (appendix "Pipeline
setup and notation"); a micro-batch's stamps are the versions its forward and
backward ran at, and Delta = t^B - t^F.

Events are tuples ("F", i), ("B", i) or ("S", None).
"""


class ProtocolError(Exception):
    """An event that Alg. 1 does not admit at this point."""


class StageCounters:
    """The counters of Alg. 1 for one stage, with FIFO micro-batch order.

    Forwards arrive in micro-batch order and each backward belongs to the
    oldest unresolved forward (1F1B). The update is due as soon as the K-th
    backward of a window completes and must be applied before any further event.
    """

    def __init__(self, K, delay):
        if K < 1 or delay < 0:
            raise ValueError("K >= 1 and delay >= 0 required")
        self.K, self.delay = K, delay
        self.t = 0          # version: local updates applied so far
        self.c = 0          # backwards in the current accumulation window
        self.q = 0          # forwards whose backward has not returned
        self.next_f = 0
        self.next_b = 0
        self.tF, self.tB = {}, {}

    @property
    def step_due(self):
        return self.c == self.K

    def forward(self, mb):
        if self.step_due:
            raise ProtocolError("update pending")
        if mb != self.next_f:
            raise ProtocolError("forward out of order")
        if not self.q <= self.delay:          # admission rule q_i <= N - i
            raise ProtocolError("backpressure")
        self.tF[mb] = self.t
        self.next_f += 1
        self.q += 1
        return self.t

    def backward(self, mb):
        if self.step_due:
            raise ProtocolError("update pending")
        if mb != self.next_b or self.next_b >= self.next_f:
            raise ProtocolError("backward out of order")
        self.tB[mb] = self.t
        self.next_b += 1
        self.c += 1
        self.q -= 1
        return self.t

    def step(self):
        if not self.step_due:
            raise ProtocolError("update not due")
        self.c = 0
        self.t += 1
        return self.t


def canonical_events(M, K, delay):
    """The steady asynchronous 1F1B order of one stage.

    Warm-up forwards F_0 .. F_min(delay, M-1), then for every j: B_j, the update
    if j+1 is a multiple of K, and F_{j+delay+1} while micro-batches remain.
    Each forward is issued as soon as the admission rule allows it and each
    update right after the backward that completes its window (Alg. 1).
    """
    ev = [("F", i) for i in range(min(delay + 1, M))]
    for j in range(M):
        ev.append(("B", j))
        if (j + 1) % K == 0:
            ev.append(("S", None))
        if j + delay + 1 < M:
            ev.append(("F", j + delay + 1))
    return ev


def flush_events(M, K, delay):
    """Synchronous 1F1B with a flush (Sec. 2, Eq. (3)) seen at one stage.

    Each window of K micro-batches runs on its own: the stage's first forwards
    (up to delay + 1 of them, the warm-up of the 1F1B order), then one backward
    and, while the window has one left, one forward; the update follows the
    window's last backward, and the next window starts only after it. Every
    forward and backward of a window then sees the same version (Delta = 0).
    A trailing partial window gets no update.
    """
    ev = []
    for a in range(0, M, K):
        b = min(M, a + K)
        ev += [("F", i) for i in range(a, min(a + delay + 1, b))]
        for j in range(a, b):
            ev.append(("B", j))
            if j + delay + 1 < b:
                ev.append(("F", j + delay + 1))
        if b - a == K:
            ev.append(("S", None))
    return ev


def run_events(events, K, delay):
    """Drive StageCounters through ``events``; return (tF, tB, delta, n_updates)."""
    sc = StageCounters(K, delay)
    for kind, i in events:
        if kind == "F":
            sc.forward(i)
        elif kind == "B":
            sc.backward(i)
        else:
            sc.step()
    M = sc.next_f
    tF = [sc.tF[i] for i in range(M)]
    tB = [sc.tB[i] for i in range(sc.next_b)]
    return tF, tB, [b - f for f, b in zip(tF, tB)], sc.t


def closed_form_stamps(M, K, delay):
    """Stamps of the canonical order in closed form.

    Before F_i the backwards B_0 .. B_{i-delay-1} are done, so t^F(i) =
    floor(max(0, i - delay) / K); before B_i exactly i backwards are done, so
    t^B(i) = floor(i / K).
    """
    tF = [max(0, i - delay) // K for i in range(M)]
    tB = [i // K for i in range(M)]
    return tF, tB, [b - f for f, b in zip(tF, tB)]


def delta_bound(delay, K):
    """Eq. (2): Delta <= ceil((N - i) / a) = ceil(delay / K)."""
    return -(-delay // K)


def all_admissible_orders(M, K, delay, admission=True):
    """Every interleaving of one stage's events that Alg. 1 can produce.

    Forwards in micro-batch order, backwards in micro-batch order, B_j only
    after F_j, a forward only while q <= delay (unless ``admission`` is False),
    and the update immediately after each K-th backward. Yields event lists.
    Exponential; meant for M up to about 10.
    """
    def rec(nf, nb, c, prefix):
        if nb == M:
            yield list(prefix)
            return
        if nf < M and (not admission or nf - nb <= delay):
            prefix.append(("F", nf))
            yield from rec(nf + 1, nb, c, prefix)
            prefix.pop()
        if nb < nf:
            prefix.append(("B", nb))
            if c + 1 == K:
                prefix.append(("S", None))
                yield from rec(nf, nb + 1, 0, prefix)
                prefix.pop()
            else:
                yield from rec(nf, nb + 1, c + 1, prefix)
            prefix.pop()
    yield from rec(0, 0, 0, [])


def max_delta_brute_force(M, K, delay, admission=True):
    """Largest Delta over every admissible interleaving (see all_admissible_orders).

    Stamps are counted directly from the event list (updates seen before each
    event), independently of StageCounters.
    """
    worst = 0
    for ev in all_admissible_orders(M, K, delay, admission):
        t, tF = 0, {}
        for kind, i in ev:
            if kind == "S":
                t += 1
            elif kind == "F":
                tF[i] = t
            else:
                worst = max(worst, t - tF[i])
    return worst


def count_orders(M, K, delay):
    return sum(1 for _ in all_admissible_orders(M, K, delay))


def events_to_string(ev):
    return " ".join("S" if k == "S" else f"{k}{i}" for k, i in ev)


__all__ = [
    "ProtocolError", "StageCounters", "canonical_events", "run_events",
    "closed_form_stamps", "delta_bound", "all_admissible_orders",
    "max_delta_brute_force", "count_orders", "events_to_string",
]
