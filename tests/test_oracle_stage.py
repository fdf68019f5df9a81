"""Pins of the oracle's stage replay and AdamW against invariants the method fixes."""
import numpy as np
import pytest
import torch

from oracle import adamw, schedule, stage

BASE = dict(kind="middle", n_layers=2, d_model=8, n_heads=2, head_dim=4, d_ff=16, seq=5,
            micro_batch=2, vocab=11, max_pos=6, ln_eps=1e-5,
            lr=1e-2, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1)


def _cfg(**kw):
    c = dict(BASE)
    c.update(kw)
    return c


def _data(cfg, M, seed=0):
    r = np.random.default_rng(seed)
    params = {}
    for n, s in stage.param_shapes(cfg):
        leaf = n.split(".")[-1]
        params[n] = (1.0 + 0.1 * r.standard_normal(s)) if leaf.endswith("_g") else 0.2 * r.standard_normal(s)
    T, d = cfg["micro_batch"] * cfg["seq"], cfg["d_model"]
    if cfg["kind"] == "first":
        xs = [r.integers(0, cfg["vocab"], size=(cfg["micro_batch"], cfg["seq"])) for _ in range(M)]
    else:
        xs = [r.standard_normal((T, d)) for _ in range(M)]
    dys = [0.1 * r.standard_normal((T, d)) for _ in range(M)]
    tg = [r.integers(0, cfg["vocab"], size=(cfg["micro_batch"], cfg["seq"])) for _ in range(M)]
    return params, xs, dys, tg


def _sync_loop(cfg, params, xs, dys, tg, K):
    """Plain synchronous training: forward and backward of K micro-batches at the
    same parameters, sum their gradients, one AdamW update; repeat."""
    names = [n for n, _ in stage.param_shapes(cfg)]
    th = {n: params[n].astype(float).copy() for n in names}
    m = {n: np.zeros_like(th[n]) for n in names}
    v = {n: np.zeros_like(th[n]) for n in names}
    outs, gins, Gs, thetas = [], [], [], []
    for w in range(len(xs) // K):
        G = {n: np.zeros_like(th[n]) for n in names}
        for i in range(w * K, (w + 1) * K):
            tgt = tg[i] if cfg["kind"] == "last" else None
            out, saved = stage.stage_fwd(cfg, th, xs[i], tgt)
            gin, g = stage.stage_bwd(cfg, th, saved, dys[i], K, ids=xs[i] if cfg["kind"] == "first" else None)
            outs.append(out)
            gins.append(gin)
            for n in names:
                G[n] += g[n]
        Gs.append(G)
        for n in names:
            wd = cfg["weight_decay"] if stage.decayed(n) else 0.0
            th[n], m[n], v[n] = adamw.adamw_update(th[n], G[n], m[n], v[n], w + 1, cfg["lr"],
                                                   cfg["beta1"], cfg["beta2"], cfg["eps"], wd)
        thetas.append({n: th[n].copy() for n in names})
    return outs, gins, Gs, thetas


def _replay(cfg, params, xs, dys, tg, K, delay):
    return stage.replay(cfg, params, K, delay, xs, grad_outs=None if cfg["kind"] == "last" else dys,
                        targets=tg if cfg["kind"] == "last" else None)


@pytest.mark.parametrize("kind", ["middle", "first", "last"])
@pytest.mark.parametrize("K", [1, 3])
def test_no_delay_equals_synchronous_accumulation(kind, K):
    """delay = 0: every backward directly follows its forward, so the replay is
    ordinary gradient accumulation over K micro-batches (K = 1: a plain
    synchronous fwd; bwd; AdamW loop)."""
    cfg = _cfg(kind=kind)
    M = 2 * K
    params, xs, dys, tg = _data(cfg, M)
    rec = _replay(cfg, params, xs, dys, tg, K, 0)
    outs, gins, Gs, thetas = _sync_loop(cfg, params, xs, dys, tg, K)
    for i in range(M):
        np.testing.assert_allclose(rec["out"][i], outs[i], rtol=1e-13, atol=1e-13)
        if kind != "first":
            np.testing.assert_allclose(rec["grad_in"][i], gins[i], rtol=1e-13, atol=1e-13)
    for s in range(M // K):
        for n in thetas[s]:
            np.testing.assert_allclose(rec["G"][s][n], Gs[s][n], rtol=1e-13, atol=1e-15)
            np.testing.assert_allclose(rec["theta"][s][n], thetas[s][n], rtol=1e-13, atol=1e-15)
    assert rec["delta"] == [0] * M


@pytest.mark.parametrize("delay", [1, 3, 5])
def test_zero_learning_rate_makes_delay_irrelevant(delay):
    """lr = 0: parameters never change, so every accumulated G equals the
    synchronous one whatever the delay."""
    cfg = _cfg(lr=0.0)
    K, M = 2, 6
    params, xs, dys, tg = _data(cfg, M, seed=1)
    rec = _replay(cfg, params, xs, dys, tg, K, delay)
    _, _, Gs, _ = _sync_loop(cfg, params, xs, dys, tg, K)
    for s in range(M // K):
        for n in Gs[s]:
            np.testing.assert_allclose(rec["G"][s][n], Gs[s][n], rtol=1e-13, atol=1e-15)


@pytest.mark.parametrize("kind", ["middle", "first", "last"])
def test_replay_equals_version_store_formulation(kind):
    """The in-place replay (single parameter copy, activations stored at forward
    time) equals a second formulation that keeps every parameter version,
    recomputes each forward at theta^(t^F) and differentiates at theta^(t^B).
    Differentiating at theta^(t^F) instead (weight stashing) gives a different
    trajectory, so the drift of Eq. (1) is exercised."""
    cfg = _cfg(kind=kind)
    K, delay, M = 2, 3, 8
    params, xs, dys, tg = _data(cfg, M, seed=2)
    go = None if kind == "last" else dys
    tgs = tg if kind == "last" else None
    rec = stage.replay(cfg, params, K, delay, xs, go, tgs)
    alt = stage.replay_with_version_store(cfg, params, K, delay, xs, go, tgs, backward_at="current")
    stash = stage.replay_with_version_store(cfg, params, K, delay, xs, go, tgs, backward_at="forward")
    assert max(rec["delta"]) == 2
    for i in range(M):
        np.testing.assert_allclose(rec["out"][i], alt["out"][i], rtol=1e-12, atol=1e-14)
        if kind != "first":
            np.testing.assert_allclose(rec["grad_in"][i], alt["grad_in"][i], rtol=1e-12, atol=1e-14)
    diff = 0.0
    for s in range(M // K):
        for n in rec["theta"][s]:
            np.testing.assert_allclose(rec["theta"][s][n], alt["theta"][s][n], rtol=1e-12, atol=1e-14)
            diff = max(diff, np.abs(rec["theta"][s][n] - stash["theta"][s][n]).max())
    assert diff > 1e-6


def test_replay_stamps_match_closed_forms():
    cfg = _cfg()
    K, delay, M = 3, 4, 9
    params, xs, dys, tg = _data(cfg, M, seed=3)
    rec = _replay(cfg, params, xs, dys, tg, K, delay)
    tF, tB, d = schedule.closed_form_stamps(M, K, delay)
    assert rec["tF"] == tF and rec["tB"] == tB and rec["delta"] == d
    assert rec["final_version"] == M // K


def test_stage_refuses_what_alg1_refuses():
    cfg = _cfg()
    params, xs, dys, _ = _data(cfg, 4)
    st = stage.Stage(cfg, params, K=2, delay=0)
    st.forward(0, xs[0])
    with pytest.raises(schedule.ProtocolError):
        st.forward(1, xs[1])              # q = 1 > delay = 0
    _, _, due = st.backward(0, dys[0])
    assert not due
    st.forward(1, xs[1])
    _, _, due = st.backward(1, dys[1])
    assert due
    with pytest.raises(schedule.ProtocolError):
        st.forward(2, xs[2])
    assert st.step() == 1


def test_adamw_first_step_closed_form():
    # From zero moments, step 1: m_hat = g, v_hat = g^2, so the update is
    # theta (1 - lr wd) - lr g / (|g| + eps).
    r = np.random.default_rng(4)
    th, g = r.standard_normal(1000), r.standard_normal(1000)
    lr, wd, eps = 1e-3, 0.1, 1e-8
    new, m, v = adamw.adamw_update(th, g, 0 * th, 0 * th, 1, lr, 0.9, 0.95, eps, wd)
    np.testing.assert_allclose(new, th * (1 - lr * wd) - lr * g / (np.abs(g) + eps), rtol=1e-14, atol=1e-18)
    np.testing.assert_allclose(m, 0.1 * g, rtol=1e-15)
    np.testing.assert_allclose(v, 0.05 * g * g, rtol=1e-14)


@pytest.mark.parametrize("wd", [0.0, 0.1])
def test_adamw_matches_torch_optim(wd):
    r = np.random.default_rng(5)
    th = r.standard_normal(257)
    p = torch.tensor(th.copy(), requires_grad=True)
    opt = torch.optim.AdamW([p], lr=1e-3, betas=(0.9, 0.95), eps=1e-8, weight_decay=wd)
    m, v = np.zeros_like(th), np.zeros_like(th)
    for t in range(1, 7):
        g = r.standard_normal(257) * (10.0 ** -t)
        p.grad = torch.tensor(g)
        opt.step()
        th, m, v = adamw.adamw_update(th, g, m, v, t, 1e-3, 0.9, 0.95, 1e-8, wd)
        np.testing.assert_allclose(th, p.detach().numpy(), rtol=1e-13, atol=1e-16)


def test_adamw_direction_bound():
    # The bound is attained by a constant gradient sequence at step 1 (|u| = 1)
    # and is never exceeded by random sequences.
    assert adamw.direction_bound(1, 0.9, 0.95) == pytest.approx(1.0)
    r = np.random.default_rng(6)
    for t in range(1, 9):
        bound = adamw.direction_bound(t, 0.9, 0.95)
        for _ in range(200):
            gs = r.standard_normal(t) * np.exp(r.standard_normal(t) * 3)
            m = v = 0.0
            for j, g in enumerate(gs, 1):
                m, v = 0.9 * m + 0.1 * g, 0.95 * v + 0.05 * g * g
            u = (m / (1 - 0.9 ** t)) / np.sqrt(v / (1 - 0.95 ** t))
            assert abs(u) <= bound * (1 + 1e-12)


def test_lr_schedule_closed_forms():
    """Linear warmup to the peak, cosine decay to lr_min_ratio * peak, then flat;
    no schedule (lr_total = 0) keeps the constant rate."""
    c = dict(lr=1e-3, lr_warmup=2, lr_total=10, lr_min_ratio=0.1)
    assert adamw.lr_at(c, 1) == pytest.approx(0.5e-3, rel=1e-15)
    assert adamw.lr_at(c, 2) == pytest.approx(1e-3, rel=1e-15)
    assert adamw.lr_at(c, 6) == pytest.approx(1e-3 * (0.1 + 0.9 * 0.5), rel=1e-14)   # halfway down the cosine
    assert adamw.lr_at(c, 10) == pytest.approx(1e-4, rel=1e-14)
    assert adamw.lr_at(c, 25) == pytest.approx(1e-4, rel=1e-14)
    assert adamw.lr_at(dict(lr=3e-4), 7) == 3e-4


def test_lr_schedule_matches_torch_schedulers():
    """Each phase against PyTorch's own scheduler: update t <= W runs at LinearLR's
    rate after t - 1 steps (from peak / W to the peak over W - 1 steps); update
    t > W at CosineAnnealingLR's rate after t - W steps (T_max = N - W, down to
    lr_min_ratio * peak)."""
    W, N, r, peak = 3, 17, 0.1, 2e-3
    c = dict(lr=peak, lr_warmup=W, lr_total=N, lr_min_ratio=r)

    def rates(make, n):
        p = torch.nn.Parameter(torch.zeros(1))
        opt = torch.optim.SGD([p], lr=peak)
        sched = make(opt)
        out = []
        for _ in range(n):
            out.append(opt.param_groups[0]["lr"])
            opt.step()
            sched.step()
        return out

    warm = rates(lambda o: torch.optim.lr_scheduler.LinearLR(o, start_factor=1.0 / W, end_factor=1.0,
                                                             total_iters=W - 1), W)
    cos = rates(lambda o: torch.optim.lr_scheduler.CosineAnnealingLR(o, T_max=N - W, eta_min=r * peak), N - W + 1)
    for t in range(1, W + 1):
        assert adamw.lr_at(c, t) == pytest.approx(warm[t - 1], rel=1e-12), t
    for t in range(W + 1, N + 1):
        assert adamw.lr_at(c, t) == pytest.approx(cos[t - W], rel=1e-9), t


def test_nonfinite_gradient_skips_the_update():
    """A window whose G holds a NaN changes no parameter or moment, clears G and
    still advances the version; the next update is AdamW's first (bias
    correction step 1, the closed form of test_adamw_first_step_closed_form)."""
    cfg = _cfg(kind="middle", weight_decay=0.1)
    params, xs, dys, tg = _data(cfg, 6, seed=9)

    def hook(s, G):
        if s == 0:
            G = {n: g.copy() for n, g in G.items()}
            G["h0.w_qkv"].flat[3] = np.nan
        return G

    rec = stage.replay(cfg, params, 2, 1, xs, grad_outs=dys, grad_hook=hook)
    st = rec["stage"]
    assert st.skipped == 1 and st.applied == 2 and rec["final_version"] == 3
    for n in params:
        assert np.array_equal(rec["theta"][0][n], np.asarray(params[n], np.float64)), n
        assert not np.any(rec["m"][0][n]) and not np.any(rec["v"][0][n]), n
    lr, wd = cfg["lr"], cfg["weight_decay"]
    for n in params:
        g = rec["G"][1][n]
        th0 = np.asarray(params[n], np.float64)
        first = (th0 * (1 - lr * wd) if stage.decayed(n) else th0) - lr * g / (np.abs(g) + cfg["eps"])
        np.testing.assert_allclose(rec["theta"][1][n], first, rtol=1e-12, atol=1e-15)


@pytest.mark.parametrize("kind", ["middle", "last"])
def test_flush_order_equals_synchronous_training(kind):
    """The synchronous 1F1B-with-flush order, at any delay, is plain synchronous
    gradient accumulation: the replay equals the fwd; bwd; AdamW loop, while the
    asynchronous order at the same delay differs after the first update."""
    cfg = _cfg(kind=kind)
    K, delay, M = 2, 3, 6
    params, xs, dys, tg = _data(cfg, M, seed=4)
    go = None if kind == "last" else dys
    tgs = tg if kind == "last" else None
    rec = stage.replay(cfg, params, K, delay, xs, go, tgs, events=schedule.flush_events(M, K, delay))
    outs, gins, Gs, thetas = _sync_loop(cfg, params, xs, dys, tg, K)
    assert rec["delta"] == [0] * M
    for i in range(M):
        np.testing.assert_allclose(rec["out"][i], outs[i], rtol=1e-13, atol=1e-13)
        np.testing.assert_allclose(rec["grad_in"][i], gins[i], rtol=1e-13, atol=1e-13)
    for s in range(M // K):
        for n in thetas[s]:
            np.testing.assert_allclose(rec["theta"][s][n], thetas[s][n], rtol=1e-13, atol=1e-15)
    paci = stage.replay(cfg, params, K, delay, xs, go, tgs)
    assert sum(paci["delta"]) > 0
    assert max(np.abs(paci["theta"][-1][n] - thetas[-1][n]).max() for n in thetas[-1]) > 1e-6
