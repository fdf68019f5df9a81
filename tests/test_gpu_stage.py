"""GPU parity of the PACI stage against the oracle, through the C ABI only."""
import numpy as np
import pytest

from parity import (DRIFT, Inputs, adamw_np, compare_replays, drift_cfg, drift_check, forced_oracle, free_report,
                    gpu_replay, oracle_replay, rel_err, small_cfg, stash_oracle, to_host, to_torch, tol, unflatten)
from oracle import schedule as osched
from oracle import stage as ostage
from paper_2606_07881_amd import configs, inputs

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def binding():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    from paper_2606_07881_amd import binding as b
    return b


def _one_event_pair(binding, c, seed=0):
    """F_0 then B_0 at version 0; returns GPU and oracle (out, grad_in, G)."""
    import torch
    inp = Inputs(c, seed, 1)
    st = binding.Stage(c, K=2, delay=0 if c.get("fused_head") else 1)   # a fused head needs delay 0
    st.load_params(inp.params)
    T, d = c["micro_batch"] * c["seq"], c["d_model"]
    x = to_torch(inp.x_dev[0])
    tg = to_torch(inp.tgt[0]) if c["kind"] == "last" else None
    out = torch.zeros(1, dtype=torch.float32, device="cuda") if c["kind"] == "last" else \
        torch.zeros(T, d, dtype=st.act_dtype, device="cuda")
    assert st.forward(0, x, out, tg) == 0
    go = None if c["kind"] == "last" else to_torch(inp.dy_dev[0])
    gi = None if c["kind"] == "first" else torch.zeros(T, d, dtype=st.act_dtype, device="cuda")
    v, due = st.backward(0, go, gi)
    assert v == 0 and not due
    G = unflatten(c, st.read(binding.GRADS))
    st.sync()
    g_out = to_host(out)
    g_in = None if gi is None else to_host(gi)
    st.close()
    theta = inp.oracle_params()
    o_out, saved = ostage.stage_fwd(c, theta, inp.x[0], inp.tgt[0] if c["kind"] == "last" else None)
    o_in, o_G = ostage.stage_bwd(c, theta, saved, None if c["kind"] == "last" else inp.dy[0], 2,
                                 ids=inp.x[0] if c["kind"] == "first" else None)
    return (g_out, g_in, G), (o_out, o_in, o_G)


@pytest.mark.parametrize("name", ["tiny_fp32", "ragged_bf16", "ragged_fp32", "win_bf16", "dh128_bf16", "dh32_bf16",
                                  "dh64_fp32", "first_bf16", "last_bf16", "first_fp32", "last_fp32",
                                  "fused_last_bf16", "drop_ragged_fp32", "drop_first_bf16"])
def test_first_forward_backward(binding, name):
    c = configs.get("tiny_fp32") if name == "tiny_fp32" else small_cfg(name)
    (g_out, g_in, G), (o_out, o_in, o_G) = _one_event_pair(binding, c)
    e = rel_err(np.atleast_1d(g_out).ravel(), np.atleast_1d(o_out).ravel())
    print(f"{name}: out {e:.2e}", flush=True)
    assert e <= tol(c, "act")
    if o_in is not None:
        e = rel_err(g_in, o_in)
        print(f"{name}: grad_in {e:.2e}", flush=True)
        assert e <= tol(c, "grad")
    worst = max(rel_err(G[n], o_G[n]) for n in o_G)
    print(f"{name}: worst G {worst:.2e}", flush=True)
    for n in o_G:
        assert rel_err(G[n], o_G[n]) <= tol(c, "grad"), n


def _fmt(rep):
    return {k: (f"{v:.2e}" if isinstance(v, float) else v) for k, v in rep.items()}


@pytest.mark.parametrize("name", ["tiny_fp32", "ragged_bf16", "ragged_fp32", "win_bf16", "win8_bf16", "winsplit_bf16",
                                  "acc8_bf16", "wide_bf16", "tall_bf16", "xcd_bf16", "dh128_bf16",
                                  "dh32_bf16", "first_bf16", "last_bf16", "first_fp32", "last_fp32",
                                  "ckpt_tiny_fp32", "ckpt_ragged_bf16", "ckpt_win_bf16", "ckpt_first_bf16",
                                  "ckpt_last_bf16", "sched_bf16", "fused_last_bf16", "ckpt_fused_last_bf16",
                                  "drop_tiny_fp32", "drop_ragged_bf16", "drop_ragged_fp32", "drop_win_bf16",
                                  "drop_dh128_bf16", "drop_dh32_bf16", "drop_first_bf16", "drop_last_bf16",
                                  "drop_first_fp32", "drop_last_fp32", "ckpt_drop_ragged_bf16",
                                  "drop_fused_last_bf16", "lastv_bf16", "fused_lastv_bf16"])
def test_replay_parity(binding, name):
    """The whole asynchronous 1F1B replay, gradient-forced: stamps bit-exact;
    every output, input gradient, accumulated G and the state after every AdamW
    update at the tolerance, with no allowance after an update."""
    c = configs.get("tiny_fp32") if name == "tiny_fp32" else small_cfg(name)
    inp = Inputs(c, 1, c["M"])
    print(f"{name}: replay of {c['M']} micro-batches", flush=True)
    g = gpu_replay(c, inp)
    o = forced_oracle(c, inp, g)
    rep = compare_replays(c, g, o, theta0=inp.params)
    print(name, "forced", _fmt(rep), flush=True)
    print(name, "free-running (reported only)", _fmt(free_report(c, g, oracle_replay(c, inp))), flush=True)
    assert g["counters"]["version"] == c["M"] // c["K"]


@pytest.mark.parametrize("name", sorted(DRIFT))
def test_drift_parity(binding, name):
    """Eq. (1) at a raised learning rate: every stale backward reads the
    current parameters. The forced replay matches at the tolerance, and every
    stale input gradient and window sum lies at least 3 tolerances away from
    what weight stashing (backward at the forward's parameters) gives."""
    c = drift_cfg(name)
    inp = Inputs(c, 1, c["M"])
    print(f"{name}: replay of {c['M']} micro-batches, lr {c['lr']}", flush=True)
    g = gpu_replay(c, inp)
    o = forced_oracle(c, inp, g)
    rep = compare_replays(c, g, o, theta0=inp.params)
    checked, closest = drift_check(c, g, o, stash_oracle(c, inp, g))
    print(name, "forced", _fmt(rep), f"stash checks {checked}, closest {closest:.1f} tolerances", flush=True)
    assert checked > 0


def test_window_flush_on_read(binding):
    """Windowed weight gradients (bf16, T a multiple of 64): reading G after the
    first backward of every window adds the products so far; the rest follow at
    the update, and every G, theta, m and v still match the oracle."""
    c = small_cfg("win8_bf16")
    inp = Inputs(c, 4, c["M"])
    g = gpu_replay(c, inp, read_mid=True)
    o = forced_oracle(c, inp, g)
    rep = compare_replays(c, g, o, theta0=inp.params)
    print("win8_bf16 read_mid", _fmt(rep), flush=True)
    assert g["counters"]["version"] == c["M"] // c["K"]


def test_stage_run_equals_event_calls(binding):
    """paci_stage_run (the schedule driver) against the same events issued one by one."""
    import torch
    c = small_cfg("ragged_bf16")
    inp = Inputs(c, 2, c["M"])
    g = gpu_replay(c, inp)
    T, d, M = c["micro_batch"] * c["seq"], c["d_model"], c["M"]
    st = binding.Stage(c)
    st.load_params(inp.params)
    x_all = torch.stack([to_torch(a) for a in inp.x_dev])
    dy_all = torch.stack([to_torch(a) for a in inp.dy_dev])
    out_all = torch.zeros(M, T, d, dtype=st.act_dtype, device="cuda")
    gin_all = torch.zeros(M, T, d, dtype=st.act_dtype, device="cuda")
    stamps = st.run(M, x_all, dy_all, out_all, gin_all)
    st.sync()
    tF, tB, dl = osched.closed_form_stamps(M, c["K"], c["delay"])
    assert stamps[:, 0].tolist() == tF and stamps[:, 1].tolist() == tB and stamps[:, 2].tolist() == dl
    for i in range(M):
        assert rel_err(to_host(out_all[i]), g["out"][i]) <= 1e-2
        assert rel_err(to_host(gin_all[i]), g["grad_in"][i]) <= 1e-2
    theta = unflatten(c, st.read(binding.PARAMS))
    for n in theta:
        assert np.abs(theta[n] - g["theta"][-1][n]).max() <= 2 * c["lr"] * (M // c["K"]) + 1e-6
    # a second replay needs fresh counters
    with pytest.raises(binding.PaciError) as ei:
        st.run(M, x_all, dy_all)
    assert ei.value.code == binding.E_ORDER
    st.reset_counters()
    st.run(M, x_all, dy_all)
    st.sync()
    assert st.counters()["version"] == M // c["K"]
    st.close()


def test_protocol_errors_leave_state_unchanged(binding):
    import torch
    c = small_cfg("dh32_bf16")
    inp = Inputs(c, 3, 4)
    T, d = c["micro_batch"] * c["seq"], c["d_model"]
    st = binding.Stage(c, K=2, delay=1)
    st.load_params(inp.params)
    xs = [to_torch(a) for a in inp.x_dev]
    dys = [to_torch(a) for a in inp.dy_dev]
    outs = [torch.zeros(T, d, dtype=st.act_dtype, device="cuda") for _ in range(4)]
    assert st.try_forward(1, xs[1], outs[1]) == binding.E_ORDER
    assert st.try_backward(0, dys[0]) == binding.E_ORDER
    assert st.try_step() == binding.E_NOT_DUE
    st.forward(0, xs[0], outs[0])
    st.forward(1, xs[1], outs[1])
    sentinel = torch.full((T, d), 7.0, dtype=st.act_dtype, device="cuda")
    outs[2].copy_(sentinel)
    before = st.counters()
    assert st.try_forward(2, xs[2], outs[2]) == binding.E_BACKPRESSURE
    assert st.counters() == before
    st.sync()
    assert torch.equal(outs[2], sentinel)          # no device work was enqueued
    assert st.backward(0, dys[0]) == (0, False)
    st.forward(2, xs[2], outs[2])
    assert st.backward(1, dys[1]) == (0, True)
    assert st.try_forward(3, xs[3], outs[3]) == binding.E_STEP_PENDING
    assert st.try_backward(2, dys[2]) == binding.E_STEP_PENDING
    assert st.step() == 1
    assert st.counters()["c"] == 0
    # null pointers are refused
    assert st.try_forward(3, None, outs[3]) == binding.E_INVAL
    assert st.try_backward(2, None) == binding.E_INVAL
    st.close()


def test_nonfinite_gradient_skips_the_update(binding):
    """A window whose G holds a NaN or an infinity: the step leaves theta, m and v
    bit-for-bit unchanged, clears G and still advances the version; the next
    window's update is AdamW's first (bias correction and rate schedule at
    update 1) on the GPU's own G, as the oracle's guard defines it."""
    import torch
    c = small_cfg("sched_bf16")
    inp = Inputs(c, 5, 4)
    T, d = c["micro_batch"] * c["seq"], c["d_model"]
    st = binding.Stage(c, K=2, delay=1)
    st.load_params(inp.params)
    xs = [to_torch(a) for a in inp.x_dev]
    dys = [to_torch(a) for a in inp.dy_dev]
    out = torch.zeros(T, d, dtype=st.act_dtype, device="cuda")

    def window(i0):
        for i in (i0, i0 + 1):
            st.forward(i, xs[i], out)
            v, due = st.backward(i, dys[i])
        assert due

    window(0)
    th0, m0, v0 = st.read(binding.PARAMS), st.read(binding.EXP_AVG), st.read(binding.EXP_AVG_SQ)
    G = st.read(binding.GRADS)
    assert np.isfinite(G).all()
    G[7] = np.nan
    G[-3] = np.inf
    st.load(binding.GRADS, G)
    assert st.step() == 1
    assert st.updates() == (0, 1)
    assert np.array_equal(st.read(binding.PARAMS).view(np.uint32), th0.view(np.uint32))
    assert np.array_equal(st.read(binding.EXP_AVG).view(np.uint32), m0.view(np.uint32))
    assert np.array_equal(st.read(binding.EXP_AVG_SQ).view(np.uint32), v0.view(np.uint32))
    assert not st.read(binding.GRADS).any()

    window(2)
    G2 = unflatten(c, st.read(binding.GRADS))
    assert st.step() == 2
    assert st.updates() == (1, 1)
    th0d = unflatten(c, th0)
    th, m, v = (unflatten(c, st.read(w)) for w in (binding.PARAMS, binding.EXP_AVG, binding.EXP_AVG_SQ))
    for n in th:
        g = np.asarray(G2[n], np.float64)
        th_x, m_x, v_x = adamw_np(np.asarray(th0d[n], np.float64), g, np.zeros_like(g), np.zeros_like(g), 1, c,
                                  ostage.decayed(n))
        e = max(rel_err(th[n], th_x), rel_err(m[n], m_x), rel_err(v[n], v_x))
        assert e <= 1e-5, f"{n}: update after a skipped one differs from AdamW's first: {e:.3e}"
    st.reset_counters()
    assert st.updates() == (0, 0)
    st.close()


@pytest.mark.parametrize("name", ["sched_bf16", "win_bf16", "dh64_fp32"])
def test_nonfinite_gradient_from_a_backward(binding, name):
    """A NaN that reaches G through a backward (in the output gradient of a
    window's last micro-batch) skips that window's update: parameters and
    moments bit for bit unchanged, G reads zero afterwards, and the next
    window's update is AdamW's first on its own G (the default stage takes the
    block matrices' flag from the last backward's weight-gradient products,
    the windowed and fp32 stages from the guard pass over all of G)."""
    import torch
    c = small_cfg(name)
    K = c["K"]
    inp = Inputs(c, 9, 2 * K)
    T, d = c["micro_batch"] * c["seq"], c["d_model"]
    st = binding.Stage(c, K=K, delay=1)
    st.load_params(inp.params)
    xs = [to_torch(a) for a in inp.x_dev]
    dys = [to_torch(a) for a in inp.dy_dev]
    dys[K - 1][3, 5] = float("nan")
    out = torch.zeros(T, d, dtype=st.act_dtype, device="cuda")
    th0, m0, v0 = st.read(binding.PARAMS), st.read(binding.EXP_AVG), st.read(binding.EXP_AVG_SQ)

    def window(i0):
        st.forward(i0, xs[i0], out)
        for i in range(i0, i0 + K):
            if i + 1 < i0 + K:
                st.forward(i + 1, xs[i + 1], out)
            v, due = st.backward(i, dys[i])
        assert due

    window(0)
    assert st.step() == 1
    assert st.updates() == (0, 1)
    assert np.array_equal(st.read(binding.PARAMS).view(np.uint32), th0.view(np.uint32))
    assert np.array_equal(st.read(binding.EXP_AVG).view(np.uint32), m0.view(np.uint32))
    assert np.array_equal(st.read(binding.EXP_AVG_SQ).view(np.uint32), v0.view(np.uint32))
    assert not st.read(binding.GRADS).any()
    window(K)
    G2 = unflatten(c, st.read(binding.GRADS))
    assert all(np.isfinite(g).all() for g in G2.values())
    assert st.step() == 2
    assert st.updates() == (1, 1)
    th0d = unflatten(c, th0)
    th, m, v = (unflatten(c, st.read(w)) for w in (binding.PARAMS, binding.EXP_AVG, binding.EXP_AVG_SQ))
    for n in th:
        g = np.asarray(G2[n], np.float64)
        th_x, m_x, v_x = adamw_np(np.asarray(th0d[n], np.float64), g, np.zeros_like(g), np.zeros_like(g), 1, c,
                                  ostage.decayed(n))
        e = max(rel_err(th[n], th_x), rel_err(m[n], m_x), rel_err(v[n], v_x))
        assert e <= 1e-5, f"{n}: {e:.3e}"
    st.close()


@pytest.mark.parametrize("name", ["dh32_bf16", "tiny_fp32"])
def test_flush_schedule_parity(binding, name):
    """Synchronous 1F1B with a flush per window (Delta = 0 everywhere): the
    event calls against the oracle replaying the same order, then the native
    driver paci_stage_run_events on that order against the event calls."""
    import torch
    c = small_cfg(name) if name != "tiny_fp32" else configs.get(name)
    M, K, delay = c["M"], c["K"], c["delay"]
    inp = Inputs(c, 6, M)
    ev = osched.flush_events(M, K, delay)
    g = gpu_replay(c, inp, events=ev)
    o = forced_oracle(c, inp, g, events=ev)
    rep = compare_replays(c, g, o, theta0=inp.params)
    print(name, "flush", _fmt(rep), flush=True)
    assert g["delta"] == [0] * M

    kinds, idx = binding.schedule(M, K, delay, flush=True)
    T, d = c["micro_batch"] * c["seq"], c["d_model"]
    st = binding.Stage(c, K, delay)
    st.load_params(inp.params)
    x_all = torch.stack([to_torch(a) for a in inp.x_dev])
    dy_all = torch.stack([to_torch(a) for a in inp.dy_dev])
    out_all = torch.zeros(M, T, d, dtype=st.act_dtype, device="cuda")
    gin_all = torch.zeros(M, T, d, dtype=st.act_dtype, device="cuda")
    stamps = st.run_events(kinds, idx, x_all, dy_all, out_all, gin_all)
    st.sync()
    assert stamps[:, 0].tolist() == [i // K for i in range(M)] == stamps[:, 1].tolist()
    assert stamps[:, 2].tolist() == [0] * M
    lim = 1e-2 if c["dtype"] == "bf16" else 1e-5
    for i in range(M):
        assert rel_err(to_host(out_all[i]), g["out"][i]) <= lim
        assert rel_err(to_host(gin_all[i]), g["grad_in"][i]) <= lim
    theta = unflatten(c, st.read(binding.PARAMS))
    for n in theta:
        # fp32 atomics make G differ in its last bits between runs, and AdamW's
        # normalized step can turn that into up to 2 lr per update where G ~ 0
        assert np.abs(theta[n] - g["theta"][-1][n]).max() <= 2 * c["lr"] * (M // K) + 1e-6
    # a malformed list is refused before any event runs
    st.reset_counters()
    before = st.read(binding.PARAMS)
    bad = np.array([0, 1, 7], np.int32)
    with pytest.raises(binding.PaciError) as ei:
        st.run_events(bad, np.array([0, 0, 0], np.int32), x_all, dy_all)
    assert ei.value.code == binding.E_INVAL
    assert st.counters()["next_f"] == 0
    assert np.array_equal(st.read(binding.PARAMS), before)
    st.close()


@pytest.mark.parametrize("name", ["drop_ragged_fp32", "drop_win_bf16", "drop_first_fp32"])
def test_dropout_masks_in_every_window(binding, name):
    """lr = 0 keeps the parameters fixed, so every window's G, output and input
    gradient must match the oracle at the base tolerance with no allowance for
    downstream drift: the masks of every micro-batch (keyed by its index) agree."""
    c = small_cfg(name, lr=0.0)
    inp = Inputs(c, 3, c["M"])
    g = gpu_replay(c, inp)
    o = oracle_replay(c, inp)
    ta, tg = tol(c, "act"), tol(c, "grad")
    for i in range(c["M"]):
        assert rel_err(np.atleast_1d(g["out"][i]), np.atleast_1d(o["out"][i])) <= ta, f"out[{i}]"
        if o["grad_in"][i] is not None:
            assert rel_err(g["grad_in"][i], o["grad_in"][i]) <= ta, f"grad_in[{i}]"
    worst = 0.0
    for s in range(len(o["G"])):
        for n in o["G"][s]:
            e = rel_err(g["G"][s][n], o["G"][s][n])
            worst = max(worst, e)
            assert e <= tg, f"G[{n}] of window {s + 1}: {e:.3e}"
    print(name, "lr=0 worst G over all windows", f"{worst:.2e}", flush=True)


@pytest.mark.parametrize("name", ["win_bf16", "ragged_fp32"])
def test_trailing_partial_window(binding, name):
    """M not a multiple of K: the updates of the full windows, then the last
    window's backwards leave their gradients in G with no update (no implicit
    step); reading G adds a windowed stage's pending products first. lr = 0
    keeps the parameters fixed, so the pending G compares at the base
    tolerance."""
    import torch
    c = small_cfg(name, lr=0.0)
    K = c["K"]
    M = 2 * K + 1
    inp = Inputs(c, 7, M)
    g = gpu_replay(c, inp)
    o = oracle_replay(c, inp)
    assert g["tB"] == o["tB"] and g["tF"] == o["tF"] and len(g["G"]) == len(o["G"]) == 2
    assert g["counters"]["version"] == 2 and g["counters"]["c"] == 1
    st = binding.Stage(c, K, c["delay"])
    st.load_params(inp.params)
    x_all = torch.stack([to_torch(a) for a in inp.x_dev])
    dy_all = torch.stack([to_torch(a) for a in inp.dy_dev])
    st.run(M, x_all, dy_all)
    G = unflatten(c, st.read(binding.GRADS))
    assert st.counters()["c"] == 1
    st.close()
    tg = tol(c, "grad")
    for n, ref in o["stage"].G.items():
        e = rel_err(G[n], ref)
        assert e <= tg, f"pending G[{n}]: {e:.3e}"


@pytest.mark.parametrize("name", ["drop_ragged_fp32", "win_bf16"])
def test_checkpoint_resume_continues_the_run(binding, name):
    """A drained stage saved (parameters, moments, counters, update counts) and
    restored into a fresh stage with paci_stage_resume continues as the
    original: the same stamps and update counts, and the same parameters up to
    the run-to-run spread of fp32 atomic sums (dropout masks follow the
    micro-batch index, the AdamW step count follows the applied updates)."""
    import torch
    c = small_cfg(name)
    K, delay = c["K"], c["delay"]
    M1, M2 = 2 * K, K
    inp = Inputs(c, 8, M1 + M2)
    x_all = torch.stack([to_torch(a) for a in inp.x_dev])
    dy_all = torch.stack([to_torch(a) for a in inp.dy_dev])
    kinds, idx = binding.schedule(M2, K, delay)
    idx = np.where(kinds < 2, idx + M1, idx).astype(np.int32)   # micro-batches M1 .. M1 + M2 - 1

    a = binding.Stage(c, K, delay)
    a.load_params(inp.params)
    a.run(M1, x_all, dy_all)
    ck = {w: a.read(w) for w in (binding.PARAMS, binding.EXP_AVG, binding.EXP_AVG_SQ)}
    cnt, upd = a.counters(), a.updates()
    assert cnt["q"] == 0 and cnt["c"] == 0 and cnt["version"] == M1 // K and upd == (M1 // K, 0)
    st_a = a.run_events(kinds, idx, x_all, dy_all)

    b = binding.Stage(c, K, delay)
    for w, arr in ck.items():
        b.load(w, arr)
    b.resume(cnt["version"], cnt["next_f"], *upd)
    st_b = b.run_events(kinds, idx, x_all, dy_all)
    assert np.array_equal(st_a[M1:], st_b[M1:])
    assert a.counters() == b.counters() and a.updates() == b.updates() == ((M1 + M2) // K, 0)
    th_a, th_b = a.read(binding.PARAMS).astype(np.float64), b.read(binding.PARAMS).astype(np.float64)
    # where rounding flips the sign of a near-zero G element, AdamW moves it by up to 2 lr
    d_ab = np.abs(th_a - th_b)
    assert d_ab.max() <= 2 * c["lr"] * (M2 // K) + 1e-6
    # AdamW's step count went on: resuming at step 1 instead changes the
    # update of every parameter (bias correction 1 - beta^1 against 1 - beta^3)
    cfresh = binding.Stage(c, K, delay)
    for w, arr in ck.items():
        cfresh.load(w, arr)
    cfresh.resume(cnt["version"], cnt["next_f"], 0, 0)
    cfresh.run_events(kinds, idx, x_all, dy_all)
    d_ac = np.abs(cfresh.read(binding.PARAMS).astype(np.float64) - th_a)
    print(name, f"resume vs run: mean |dtheta| {d_ab.mean():.2e}; wrong step count: {d_ac.mean():.2e}", flush=True)
    assert d_ac.mean() > 20 * d_ab.mean() + 1e-6
    # resuming is refused while micro-batches are in flight
    with pytest.raises(binding.PaciError) as ei:
        d = binding.Stage(c, K, delay)
        d.load_params(inp.params)
        d.forward(0, x_all[0], torch.zeros_like(x_all[0]))
        d.resume(0, 0, 0)
    assert ei.value.code == binding.E_ORDER
    for s in (a, b, cfresh, d):
        s.close()
