"""Pipeline-efficiency formulas of Sec. 3.3-3.4 (test infrastructure).

Only used to pin values the paper prints (Table 1 and the worked numbers of
Sec. 3.3); nothing in the stage computation depends on them.
"""


def eta_flush(m, N):
    """Eq. (3): bubble efficiency of synchronous 1F1B with a flush, m / (m + N - 1)."""
    return m / (m + N - 1)


def eta_interleaved(m, N, V):
    """Eq. (4): efficiency of interleaved 1F1B with V virtual stages, mV / (mV + N - 1)."""
    return m * V / (m * V + N - 1)


def paci_throughput_proxy(t_flush, m, N):
    """Eq. (5): projected PACI throughput, T_flush / eta_flush(m, N)."""
    return t_flush / eta_flush(m, N)
