"""Memory-constrained pipeline partitioning (appendix "Memory-constrained
pipeline partitioning"), by exhaustive search. Test infrastructure only.

L layers with forward times t_l, static bytes s_l and per-micro-batch
activation bytes a_l are cut into N contiguous non-empty stages G_1 .. G_N.
Stage j (1-based) holds w_j = N - j + 1 micro-batches in flight under 1F1B,
so its memory is M_j = sum_{l in G_j} s_l + w_j * sum_{l in G_j} a_l. The
partition minimises the largest stage time max_j T(G_j) subject to M_j <= B
for every j. When no partition fits, the fallback minimises the pair
(largest overshoot max_j max(0, M_j - B), largest stage time) in
lexicographic order.

Every partition is enumerated (C(L-1, N-1) of them), so this is for small L.
"""
import itertools


def stage_costs(t, s, a, cuts, budget):
    """Per-stage (time, memory, overshoot) for cut points 0 = c_0 < ... < c_N = L."""
    N = len(cuts) - 1
    out = []
    for j in range(1, N + 1):
        lo, hi = cuts[j - 1], cuts[j]
        w = N - j + 1
        time = sum(t[lo:hi])
        mem = sum(s[lo:hi]) + w * sum(a[lo:hi])
        out.append((time, mem, max(0.0, mem - budget)))
    return out


def all_partitions(L, N):
    """Every cut vector (c_0 = 0, c_1, ..., c_N = L) with non-empty stages."""
    for inner in itertools.combinations(range(1, L), N - 1):
        yield (0,) + inner + (L,)


def partition(t, s, a, N, budget):
    """Returns (feasible, best objective, list of every optimal cut vector).

    Objective: max stage time when some partition fits the budget; otherwise
    the pair (max overshoot, max stage time)."""
    L = len(t)
    if not (1 <= N <= L):
        raise ValueError("need 1 <= N <= L")
    scored = []
    for cuts in all_partitions(L, N):
        c = stage_costs(t, s, a, cuts, budget)
        fits = all(mem <= budget for _, mem, _ in c)
        scored.append((cuts, fits, max(x[0] for x in c), max(x[2] for x in c)))
    feas = [x for x in scored if x[1]]
    if feas:
        best = min(x[2] for x in feas)
        return True, best, [x[0] for x in feas if x[2] == best]
    best = min((x[3], x[2]) for x in scored)
    return False, best, [x[0] for x in scored if (x[3], x[2]) == best]
