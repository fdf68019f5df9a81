"""Pins of the oracle's activation-checkpointed stage (appendix "Activation
checkpointing"): a backward recomputes its stage's activations under the
version current at that time and differentiates them there."""
import numpy as np
import pytest

from oracle import stage
from test_oracle_stage import _cfg, _data


def _run(cfg, params, xs, dys, tg, K, delay, recompute):
    return stage.replay(cfg, params, K, delay, xs, grad_outs=None if cfg["kind"] == "last" else dys,
                        targets=tg if cfg["kind"] == "last" else None, recompute=recompute)


@pytest.mark.parametrize("kind", ["middle", "first", "last"])
def test_checkpointed_without_delay_equals_stored(kind):
    """delay = 0: every backward runs at its forward's version, so recomputing
    the activations gives the stored ones bit for bit."""
    cfg = _cfg(kind=kind)
    params, xs, dys, tg = _data(cfg, 6, seed=3)
    a = _run(cfg, params, xs, dys, tg, 3, 0, recompute=False)
    b = _run(cfg, params, xs, dys, tg, 3, 0, recompute=True)
    for i in range(6):
        assert np.array_equal(np.asarray(a["out"][i]), np.asarray(b["out"][i]))
        if a["grad_in"][i] is not None:
            assert np.array_equal(a["grad_in"][i], b["grad_in"][i])
    for w in range(2):
        for n in a["G"][w]:
            assert np.array_equal(a["G"][w][n], b["G"][w][n]), n
            assert np.array_equal(a["theta"][w][n], b["theta"][w][n]), n


def _version(params, rec, t):
    return {n: np.asarray(v, dtype=np.float64) for n, v in params.items()} if t == 0 else rec["theta"][t - 1]


def _inner(cfg, theta, x, dy):
    out, _ = stage.stage_fwd(cfg, theta, x)
    return float(np.sum(out * dy))


def test_checkpointed_backward_is_the_gradient_at_the_current_version():
    """With delay 2 and K 2 some backwards cross an update. For every one of them
    the input gradient is the derivative of <dy, F(x; theta)> at the backward's
    version (central differences along a random direction), and each window's
    G is the sum over its micro-batches of the parameter derivative at each one's
    backward version."""
    cfg = _cfg(kind="middle")
    M, K, delay, eps = 6, 2, 2, 1e-5
    params, xs, dys, tg = _data(cfg, M, seed=5)
    rec = _run(cfg, params, xs, dys, tg, K, delay, recompute=True)
    r = np.random.default_rng(11)
    stale = [i for i in range(M) if rec["tB"][i] > rec["tF"][i]]
    assert stale, "the workload must contain stale backwards"
    for i in range(M):
        th = _version(params, rec, rec["tB"][i])
        u = r.standard_normal(xs[i].shape)
        fd = (_inner(cfg, th, xs[i] + eps * u, dys[i]) - _inner(cfg, th, xs[i] - eps * u, dys[i])) / (2 * eps)
        got = float(np.sum(rec["grad_in"][i] * u))
        assert abs(got - fd) <= 1e-6 * max(1.0, abs(fd)), (i, got, fd)
    for w in range(M // K):
        U = {n: r.standard_normal(np.shape(v)) for n, v in params.items()}
        fd = 0.0
        for i in range(w * K, (w + 1) * K):
            th = _version(params, rec, rec["tB"][i])
            plus = {n: th[n] + eps * U[n] for n in th}
            minus = {n: th[n] - eps * U[n] for n in th}
            fd += (_inner(cfg, plus, xs[i], dys[i]) - _inner(cfg, minus, xs[i], dys[i])) / (2 * eps)
        got = sum(float(np.sum(rec["G"][w][n] * U[n])) for n in U)
        assert abs(got - fd) <= 1e-6 * max(1.0, abs(fd)), (w, got, fd)


def test_checkpointed_and_stored_differ_exactly_on_stale_backwards():
    """The two variants agree until a stale gradient has entered an update (here:
    the backwards at version 0) and differ on every stale backward (Sec. 3.1
    against the appendix)."""
    cfg = _cfg(kind="middle")
    M, K, delay = 6, 2, 2
    params, xs, dys, tg = _data(cfg, M, seed=7)
    a = _run(cfg, params, xs, dys, tg, K, delay, recompute=False)
    b = _run(cfg, params, xs, dys, tg, K, delay, recompute=True)
    for i in range(M):
        diff = np.abs(a["grad_in"][i] - b["grad_in"][i]).max() / np.abs(a["grad_in"][i]).max()
        if b["tB"][i] == 0:
            assert diff == 0.0, i
        else:
            assert diff > 1e-4, (i, diff)
