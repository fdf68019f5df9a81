"""Shared helpers of the GPU parity tests (not collected by pytest).

The GPU side is driven only through the C ABI (paper_2606_07881_amd.binding);
the expected side is only the oracle. Both consume the same seeded inputs
from paper_2606_07881_amd.inputs.

Error metric (per tensor): e(x, r) = max|x - r| / max|r| (absolute when r == 0).
Tolerances: fp32 stages 1e-4 everywhere; bf16 stages 2e-2 on activations and
the loss, 3e-2 on gradients, parameters and moments. No other allowance.

Protocol (gradient-forced). AdamW's first update moves each weight by about
lr * sign(G): where |G| is near eps its derivative is lr / eps, so two G that
agree within the tolerance can still move a near-zero element by up to 2 lr in
opposite directions, and every later quantity inherits that. So the oracle
replays the same event list with one change: just before each update it
substitutes the GPU's accumulated G for its own (after comparing the two).
From then on both sides hold the same parameter versions up to fp32 rounding,
and every quantity of the replay is compared at the tolerance above:
* version stamps, update count: exactly;
* every stage output and every input gradient;
* the accumulated G before every update (the oracle's own sum of its own
  backwards, against the GPU's);
* the parameters and both moments after every update;
* every AdamW update also as a property of the GPU's own state: the
  parameters and moments it writes equal AdamW applied to the parameters, G
  and moments it read (1e-5).
The free-running oracle (its own G at every update) is reported beside it,
with the number of elements whose G sign differs at the first update; it is
printed, not asserted.

Drift (Eq. (1)): for the workloads in DRIFT the tests also replay the oracle
with weight stashing (every backward at the parameters of its forward, under
the same forced G) and require the GPU's stale input gradients and window
sums to lie at least 3 tolerances away from that result; the CPU tests check
with the oracle alone that these workloads separate the two readings by at
least 5 tolerances, so a stage that stashed weights could not pass.
"""
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from oracle import adamw as oadamw  # noqa: E402
from oracle import schedule as osched  # noqa: E402
from oracle import stage as ostage  # noqa: E402
from paper_2606_07881_amd import configs, inputs  # noqa: E402

def tol(c, kind):
    if c["dtype"] == "fp32":
        return 1e-4
    return 2e-2 if kind == "act" else 3e-2


def rel_err(x, r):
    x = np.asarray(x, np.float64)
    r = np.asarray(r, np.float64)
    assert x.shape == r.shape, (x.shape, r.shape)
    if x.size == 0:
        return 0.0
    if not np.all(np.isfinite(x)):
        return float("inf")
    den = np.abs(r).max()
    num = np.abs(x - r).max()
    return float(num / den) if den > 0 else float(num)


def small_cfg(name, **kw):
    """Parity workloads small enough for the oracle (seconds), spanning several
    tiles with ragged tails. ``ckpt_<name>``: workload <name> on an
    activation-checkpointed stage; ``fused_<name>``: a last stage whose LM head
    keeps no logits (the oracle is the same function); ``drop_<name>``: with
    dropout 0.1 at every site."""
    if name.startswith("ckpt_"):
        base = name[len("ckpt_"):]
        c = configs.get(base) if base == "tiny_fp32" else small_cfg(base)
        c.update(recompute=1, window=0, **kw)   # a checkpointed stage keeps no window
        return c
    if name.startswith("fused_"):
        c = small_cfg(name[len("fused_"):])
        c.update(fused_head=1, **kw)
        return c
    if name.startswith("drop_"):   # the paper's dropout rate at every site
        base = name[len("drop_"):]
        c = configs.get(base) if base == "tiny_fp32" else small_cfg(base)
        c.update(dropout=0.1, dropout_seed=2606, **kw)
        return c
    base = {
        # ragged in tokens (T = 400), model width (192 = 1.5 GEMM tiles) and keys (S = 200)
        "ragged_bf16": dict(kind="middle", n_layers=2, d_model=192, n_heads=3, head_dim=64, d_ff=768, seq=200,
                            micro_batch=2, K=4, delay=3, M=12, dtype="bf16"),
        "ragged_fp32": dict(kind="middle", n_layers=2, d_model=96, n_heads=3, head_dim=32, d_ff=320, seq=100,
                            micro_batch=2, K=3, delay=2, M=9, dtype="fp32"),
        # the learning-rate schedule: warmup over the first update, cosine to 10% by the third
        "sched_bf16": dict(kind="middle", n_layers=1, d_model=128, n_heads=2, head_dim=64, d_ff=256, seq=64,
                           micro_batch=2, K=2, delay=1, M=8, dtype="bf16", lr=3e-3, lr_warmup=1, lr_total=3,
                           lr_min_ratio=0.1),
        # T = 128 (a multiple of 64): bf16 weight gradients windowed over K = 3 micro-batches
        "win_bf16": dict(kind="middle", n_layers=2, d_model=128, n_heads=2, head_dim=64, d_ff=384, seq=64,
                         micro_batch=2, K=3, delay=2, M=9, dtype="bf16", window=1),
        # 8 micro-batches of T = 1024 per window: the window GEMMs split the 8192
        # contracted rows 8 ways, each split one activation segment
        "win8_bf16": dict(kind="middle", n_layers=1, d_model=128, n_heads=2, head_dim=64, d_ff=256, seq=512,
                          micro_batch=2, K=8, delay=2, M=16, dtype="bf16", window=1),
        # T = 320, K = 7: the 2240 contracted rows of a window split in two at row
        # 1152, inside the fourth activation segment (rows 960 .. 1279), as the
        # full-size window products split mid-segment
        "winsplit_bf16": dict(kind="middle", n_layers=1, d_model=128, n_heads=2, head_dim=64, d_ff=256, seq=160,
                              micro_batch=2, K=7, delay=2, M=14, dtype="bf16", window=1),
        # FFN width 2304 at T = 4096: the FFN1 forward and FFN2 input-gradient products
        # have 288 tiles of 256 x 128, more than the 256 CUs (a second, partial round)
        "wide_bf16": dict(kind="middle", n_layers=1, d_model=256, n_heads=4, head_dim=64, d_ff=2304, seq=512,
                          micro_batch=8, K=2, delay=1, M=6, dtype="bf16"),
        # T = 4000, FFN width 4064, d 96: the FFN1 forward and FFN2 input-gradient
        # products run on 256 x 256 tiles (16 x 16 = 256 tiles, whole rounds of the
        # 256 CUs), both with a ragged last row and column tile, and their
        # contraction over d = 96 ends in a partial k-step
        "tall_bf16": dict(kind="middle", n_layers=1, d_model=96, n_heads=3, head_dim=32, d_ff=4064, seq=500,
                          micro_batch=8, K=2, delay=1, M=3, dtype="bf16"),
        # d 512, FFN 2048: every weight's tile grid of the grouped weight-gradient launch
        # splits into 8 equal blocks, one per XCD (W_qkv 6 x 4 and W_o 2 x 4 tiles of 256 x 128)
        "xcd_bf16": dict(kind="middle", n_layers=1, d_model=512, n_heads=8, head_dim=64, d_ff=2048, seq=128,
                         micro_batch=2, K=2, delay=1, M=4, dtype="bf16"),
        # the same shapes as win8_bf16 on the default stage (per-backward accumulation)
        "acc8_bf16": dict(kind="middle", n_layers=1, d_model=128, n_heads=2, head_dim=64, d_ff=256, seq=512,
                          micro_batch=2, K=8, delay=2, M=16, dtype="bf16"),
        "dh128_bf16": dict(kind="middle", n_layers=1, d_model=256, n_heads=2, head_dim=128, d_ff=512, seq=160,
                           micro_batch=2, K=2, delay=1, M=6, dtype="bf16"),
        "dh32_bf16": dict(kind="middle", n_layers=1, d_model=128, n_heads=4, head_dim=32, d_ff=256, seq=96,
                          micro_batch=3, K=3, delay=2, M=9, dtype="bf16"),
        "dh64_fp32": dict(kind="middle", n_layers=1, d_model=128, n_heads=2, head_dim=64, d_ff=256, seq=80,
                          micro_batch=2, K=2, delay=1, M=4, dtype="fp32"),
        "first_bf16": dict(kind="first", n_layers=1, d_model=128, n_heads=2, head_dim=64, d_ff=512, seq=100,
                           micro_batch=2, vocab=1000, max_pos=128, K=2, delay=2, M=6, dtype="bf16"),
        "last_bf16": dict(kind="last", n_layers=1, d_model=128, n_heads=2, head_dim=64, d_ff=512, seq=100,
                          micro_batch=2, vocab=1000, max_pos=128, K=2, delay=0, M=4, dtype="bf16"),
        "first_fp32": dict(kind="first", n_layers=1, d_model=64, n_heads=2, head_dim=32, d_ff=128, seq=40,
                           micro_batch=2, vocab=301, max_pos=64, K=2, delay=1, M=4, dtype="fp32"),
        "last_fp32": dict(kind="last", n_layers=1, d_model=64, n_heads=2, head_dim=32, d_ff=128, seq=40,
                          micro_batch=2, vocab=301, max_pos=64, K=2, delay=0, M=4, dtype="fp32"),
        # a vocabulary smaller than one 64-column group of the fused head's statistics
        "lastv_bf16": dict(kind="last", n_layers=1, d_model=128, n_heads=2, head_dim=64, d_ff=256, seq=72,
                           micro_batch=2, vocab=37, max_pos=128, K=2, delay=0, M=4, dtype="bf16"),
    }[name]
    c = configs.get("tiny_fp32")
    c.update(vocab=0, max_pos=0)
    c.update(base)
    c.update(kw)
    c["name"] = name
    return c


# Workloads whose stale backwards separate Eq. (1) (current parameters) from
# weight stashing by at least 5 tolerances (checked with the oracle alone in
# tests/test_oracle_drift.py): raised learning rates make one update move the
# weights enough. Name -> (small_cfg workload, overrides).
DRIFT = {
    "drift_ragged_bf16": ("ragged_bf16", dict(lr=1e-2)),           # default store, 2 blocks, K 4, delay 3
    "drift_acc8_bf16": ("acc8_bf16", dict(lr=3e-2)),               # default store, T 1024, K 8
    "drift_win8_bf16": ("win8_bf16", dict(lr=3e-2)),               # windowed weight gradients
    "drift_winsplit_bf16": ("winsplit_bf16", dict(lr=3e-2)),       # windowed, splits inside segments
    "drift_first_bf16": ("first_bf16", dict(lr=1e-2)),             # first stage (embedding gradients)
    "drift_last_bf16": ("last_bf16", dict(lr=1e-2, delay=2)),      # last stage with two in flight
}


def drift_cfg(name):
    base, over = DRIFT[name]
    c = small_cfg(base, **over)
    c["name"] = name
    return c


# ---- inputs ------------------------------------------------------------------------------------
class Inputs:
    """Seeded inputs of M micro-batches as oracle values and device bits."""

    def __init__(self, c, seed, M):
        self.c, self.seed, self.M = c, seed, M
        self.params = inputs.make_params(c, seed)
        self.x, self.x_dev, self.dy, self.dy_dev, self.ids, self.tgt = [], [], [], [], [], []
        for i in range(M):
            if c["kind"] == "first":
                ids = inputs.make_ids(c, seed, i)
                self.x.append(ids)
                self.x_dev.append(ids)
            else:
                v, b = inputs.make_x(c, seed, i)
                self.x.append(v.astype(np.float64))
                self.x_dev.append(b)
            if c["kind"] == "last":
                t = inputs.make_targets(c, seed, i)
                self.tgt.append(t)
            else:
                v, b = inputs.make_dy(c, seed, i)
                self.dy.append(v.astype(np.float64))
                self.dy_dev.append(b)

    def oracle_params(self):
        return {k: v.astype(np.float64) for k, v in self.params.items()}


def to_torch(a):
    import torch
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16).copy()).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def to_host(t):
    import torch
    if t.dtype == torch.bfloat16:
        return t.float().cpu().numpy().astype(np.float64)
    return t.cpu().numpy().astype(np.float64)


def unflatten(c, flat, table=None):
    out = {}
    off = 0
    for name, shape, _ in inputs.param_specs(c):
        n = int(np.prod(shape))
        out[name] = flat[off:off + n].reshape(shape).astype(np.float64)
        off += n
    return out


# ---- GPU replay, driven event by event through the C ABI --------------------------------------
def gpu_replay(c, inp, events=None, K=None, delay=None, read_mid=False):
    """read_mid: also read G (and drop it) after the first backward of every window."""
    import torch
    from paper_2606_07881_amd import binding
    K = c["K"] if K is None else K
    delay = c["delay"] if delay is None else delay
    M = inp.M
    st = binding.Stage(c, K, delay)
    st.load_params(inp.params)
    if events is None:
        kinds, idx = binding.schedule(M, K, delay)
        events = [("F", int(i)) if k == 0 else ("B", int(i)) if k == 1 else ("S", None) for k, i in zip(kinds, idx)]
    T, d = c["micro_batch"] * c["seq"], c["d_model"]
    act = st.act_dtype
    rec = dict(out=[None] * M, grad_in=[None] * M, tF=[None] * M, tB=[None] * M, G=[], theta=[], m=[], v=[])
    outs, gins, xs, dys, tgs = {}, {}, {}, {}, {}
    for kind, i in events:
        if kind == "F":
            xs[i] = to_torch(inp.x_dev[i])
            if c["kind"] == "last":
                tgs[i] = to_torch(inp.tgt[i])
                outs[i] = torch.zeros(1, dtype=torch.float32, device="cuda")
            else:
                outs[i] = torch.zeros(T, d, dtype=act, device="cuda")
            rec["tF"][i] = st.forward(i, xs[i], outs[i], tgs.get(i))
        elif kind == "B":
            go = None
            if c["kind"] != "last":
                dys[i] = to_torch(inp.dy_dev[i])
                go = dys[i]
            gi = None
            if c["kind"] != "first":
                gins[i] = torch.zeros(T, d, dtype=act, device="cuda")
                gi = gins[i]
            rec["tB"][i], _ = st.backward(i, go, gi)
            if read_mid and i % K == 0:
                st.read(binding.GRADS)
        else:
            rec["G"].append(unflatten(c, st.read(binding.GRADS)))
            st.step()
            rec["theta"].append(unflatten(c, st.read(binding.PARAMS)))
            rec["m"].append(unflatten(c, st.read(binding.EXP_AVG)))
            rec["v"].append(unflatten(c, st.read(binding.EXP_AVG_SQ)))
    st.sync()
    for i in range(M):
        if i in outs:
            rec["out"][i] = to_host(outs[i])[0] if c["kind"] == "last" else to_host(outs[i])
        if i in gins:
            rec["grad_in"][i] = to_host(gins[i])
    rec["delta"] = [None if f is None or b is None else b - f for f, b in zip(rec["tF"], rec["tB"])]
    rec["counters"] = st.counters()
    st.close()
    return rec


def oracle_replay(c, inp, events=None, K=None, delay=None, grad_hook=None):
    K = c["K"] if K is None else K
    delay = c["delay"] if delay is None else delay
    return ostage.replay(c, inp.oracle_params(), K, delay, inp.x,
                         grad_outs=None if c["kind"] == "last" else inp.dy,
                         targets=inp.tgt if c["kind"] == "last" else None, events=events, grad_hook=grad_hook,
                         recompute=bool(c.get("recompute", 0)))


def adamw_np(theta, G, m, v, step, c, decay):
    """The AdamW update (decoupled decay first, bias-corrected moments, eps outside
    the root) in float64, used to check a GPU update against the GPU's own state."""
    lr, b1, b2, eps, wd = oadamw.lr_at(c, step), c["beta1"], c["beta2"], c["eps"], c["weight_decay"]
    th = theta * (1.0 - lr * wd) if decay else theta.copy()
    m = b1 * m + (1 - b1) * G
    v = b2 * v + (1 - b2) * G * G
    th = th - (lr / (1 - b1 ** step)) * m / (np.sqrt(v) / np.sqrt(1 - b2 ** step) + eps)
    return th, m, v


# ---- comparison ----------------------------------------------------------------------------------
def _force(g):
    """grad_hook substituting the GPU's accumulated G before each update."""
    Gs = g["G"]

    def hook(s, G):
        return {n: np.asarray(Gs[s][n], np.float64).copy() for n in G}
    return hook


def forced_oracle(c, inp, g, events=None):
    """The oracle replay of the same events with the GPU's G at every update."""
    return oracle_replay(c, inp, events=events, grad_hook=_force(g))


def stash_oracle(c, inp, g, events=None):
    """Weight stashing under the same forced G: every backward at the
    parameters of its own forward (not the method; see Eq. (1))."""
    return ostage.replay_with_version_store(c, inp.oracle_params(), c["K"], c["delay"], inp.x,
                                            None if c["kind"] == "last" else inp.dy,
                                            inp.tgt if c["kind"] == "last" else None, backward_at="forward",
                                            events=events, grad_hook=_force(g))


def compare_replays(c, g, o, theta0=None):
    """Asserts parity of a GPU replay ``g`` with the forced oracle replay ``o``
    (forced_oracle) at the tolerances, everywhere; returns the error report.
    theta0: the initial parameters (dict), for the property check of the first update."""
    assert g["tF"] == o["tF"] and g["tB"] == o["tB"], "version stamps differ"
    assert g["delta"] == o["delta"]
    assert len(g["G"]) == len(o["G"]), "number of updates differs"
    t_act, t_grad = tol(c, "act"), tol(c, "grad")
    worst = dict(out=0.0, grad_in=0.0, out_after_update=0.0, grad_in_after_update=0.0, G=0.0, G_after_update=0.0,
                 theta=0.0, m=0.0, v=0.0, adamw_property=0.0)
    for i in range(len(o["out"])):
        if o["out"][i] is not None:
            e = rel_err(np.atleast_1d(g["out"][i]), np.atleast_1d(o["out"][i]))
            key = "out_after_update" if (o["tF"][i] or 0) > 0 else "out"
            worst[key] = max(worst[key], e)
            assert e <= t_act, f"output of micro-batch {i} (t^F {o['tF'][i]}): {e:.3e}"
        if o["grad_in"][i] is not None:
            e = rel_err(g["grad_in"][i], o["grad_in"][i])
            key = "grad_in_after_update" if (o["tB"][i] or 0) > 0 else "grad_in"
            worst[key] = max(worst[key], e)
            assert e <= t_grad, f"input gradient of micro-batch {i} (t^F {o['tF'][i]}, t^B {o['tB'][i]}): {e:.3e}"
    names = [n for n, _, _ in inputs.param_specs(c)]
    for s in range(len(o["G"])):
        for n in names:
            gg = g["G"][s][n]
            e = rel_err(gg, o["G"][s][n])
            key = "G" if s == 0 else "G_after_update"
            worst[key] = max(worst[key], e)
            assert e <= t_grad, f"G[{n}] before update {s + 1}: {e:.3e}"
            for key in ("theta", "m", "v"):
                e = rel_err(g[key][s][n], o[key][s][n])
                worst[key] = max(worst[key], e)
                assert e <= t_grad, f"{key}[{n}] after update {s + 1}: {e:.3e}"
            # the update as a property of the GPU's own state
            if s == 0:
                th_prev = None if theta0 is None else np.asarray(theta0[n], np.float64)
                m_prev = np.zeros_like(gg)
                v_prev = np.zeros_like(gg)
            else:
                th_prev, m_prev, v_prev = g["theta"][s - 1][n], g["m"][s - 1][n], g["v"][s - 1][n]
            if th_prev is not None:
                th_x, m_x, v_x = adamw_np(th_prev, gg, m_prev, v_prev, s + 1, c, ostage.decayed(n))
                e = max(rel_err(g["theta"][s][n], th_x), rel_err(g["m"][s][n], m_x), rel_err(g["v"][s][n], v_x))
                worst["adamw_property"] = max(worst["adamw_property"], e)
                assert e <= 1e-5, f"AdamW update {s + 1} of {n} differs from the formula on its own state: {e:.3e}"
    return worst


def free_report(c, g, free):
    """Errors of the GPU replay against the free-running oracle (its own G at
    every update), for the record: the largest error after the first update per
    quantity, and the number of G elements whose sign differs at update 1."""
    rep = dict(out=0.0, grad_in=0.0, G=0.0, theta=0.0)
    for i in range(len(free["out"])):
        if free["out"][i] is not None and (free["tF"][i] or 0) > 0:
            rep["out"] = max(rep["out"], rel_err(np.atleast_1d(g["out"][i]), np.atleast_1d(free["out"][i])))
        if free["grad_in"][i] is not None and (free["tB"][i] or 0) > 0:
            rep["grad_in"] = max(rep["grad_in"], rel_err(g["grad_in"][i], free["grad_in"][i]))
    for s in range(len(free["G"])):
        for n in free["G"][s]:
            if s > 0:
                rep["G"] = max(rep["G"], rel_err(g["G"][s][n], free["G"][s][n]))
            rep["theta"] = max(rep["theta"], rel_err(g["theta"][s][n], free["theta"][s][n]))
    rep["G_sign_flips_update_1"] = int(sum(int(np.sum(np.sign(g["G"][0][n]) != np.sign(free["G"][0][n])))
                                           for n in free["G"][0])) if free["G"] else 0
    return rep


def drift_check(c, g, o, stash, factor=3.0, min_gap=5.0):
    """Eq. (1) discriminated: every stale backward's input gradient, and each
    G tensor of a window with a stale backward whose forced-oracle gap to weight
    stashing is at least ``min_gap`` tolerances, lie ``factor`` tolerances or
    more away from the weight-stash result. Returns (checked, closest) with
    closest in tolerances."""
    t = tol(c, "grad")
    closest, checked = float("inf"), 0
    for i in range(len(o["grad_in"])):
        if o["grad_in"][i] is None or not (o["tB"][i] > o["tF"][i]):
            continue
        e = rel_err(g["grad_in"][i], stash["grad_in"][i]) / t
        closest = min(closest, e)
        checked += 1
        assert e >= factor, f"input gradient of stale micro-batch {i} only {e:.2f} tolerances from weight stashing"
    for s in range(len(o["G"])):
        stale = [i for i in range(len(o["tB"])) if o["tB"][i] == s and o["tF"][i] is not None and o["tF"][i] < s]
        if not stale:
            continue
        for n in o["G"][s]:
            if rel_err(o["G"][s][n], stash["G"][s][n]) / t < min_gap:
                continue
            e = rel_err(g["G"][s][n], stash["G"][s][n]) / t
            closest = min(closest, e)
            checked += 1
            assert e >= factor, f"G[{n}] of window {s + 1} only {e:.2f} tolerances from weight stashing"
    return checked, closest
