"""Shared helpers of the GPU parity tests (not collected by pytest).

The GPU side is driven only through the C ABI (paper_2606_07881_amd.binding);
the expected side is only the oracle. Both consume the same seeded inputs
from paper_2606_07881_amd.inputs.

Error metric (per tensor): e(x, r) = max|x - r| / max|r| (absolute when r == 0).
Tolerances: fp32 stages 1e-4 everywhere; bf16 stages 2e-2 on activations and
the loss, 3e-2 on gradients, parameters and moments.

What is compared, and how:
* version stamps, update count: exactly;
* every output whose forward, and every input gradient whose backward, ran
  before the first update, every accumulated G and the moments m, v after
  every update: the tolerance above;
* every AdamW update, as a property of the GPU's own state: the parameters
  and moments it writes equal the AdamW formula applied to the parameters,
  G and moments it read (1e-5);
* parameters against the oracle after every update: elementwise wherever the
  Adam step lr * m_hat / (sqrt(v_hat) + eps) is well conditioned, i.e.
  sqrt(v_hat) + eps of the oracle exceeds 3 / tol times the largest
  discrepancy of that element's G seen so far (so that discrepancy moves the
  step by at most a third of the tolerance). Elsewhere (the first update moves a weight by about
  lr * sign(G), so a tiny G within its tolerance may flip it) several results
  are correct and the element is only checked for validity: within
  2 * lr * (sum of the largest possible Adam steps) of the oracle;
* everything downstream of the first update (outputs and input gradients of
  events that ran at an updated version, later G, m, v, parameters): that
  tolerance, widened to twice the oracle's own sensitivity where that is
  larger. The sensitivity is the oracle-only change of each of these
  quantities when every accumulated G is perturbed, before each update, by
  Gaussian noise of the stage dtype's rounding error times its largest
  element: 2^-8 for bf16 operands, 2^-20 (16 units of the last place) for
  fp32 accumulation.
  AdamW's normalized first steps amplify such differences: where |G| is near
  eps the update's derivative is lr / eps, and where G is small it
  behaves like lr * sign(G).
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

SENS_RHO = {"bf16": 2.0 ** -8, "fp32": 2.0 ** -20}   # G perturbation relative to max|G|


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
        c.update(recompute=1, **kw)
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
                         micro_batch=2, K=3, delay=2, M=9, dtype="bf16"),
        # 8 micro-batches of T = 1024 per window: the window GEMMs split the 8192
        # contracted rows 8 ways, one split per XCD
        "win8_bf16": dict(kind="middle", n_layers=1, d_model=128, n_heads=2, head_dim=64, d_ff=256, seq=512,
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


def oracle_sensitivity(c, inp, ref, seed=12345, events=None, draws=2):
    """Oracle-only change of every compared quantity when each accumulated G is
    perturbed by Gaussian noise of SENS_RHO[dtype] * max|G| before each update
    (``events``: the event list ``ref`` was replayed with, default canonical).
    The largest change over ``draws`` independent perturbations is kept: after
    AdamW's first step (a sign per element) the change comes from the few G
    elements near zero whose sign the noise flips, which one draw can
    undercount. Returns dict(out=[...], grad_in=[...], G=[{name: e}], m=...,
    v=..., theta=...)."""
    rho = SENS_RHO[c["dtype"]]
    out = None
    for k in range(draws):
        rng = np.random.default_rng(seed + k)

        def hook(s, G):
            return {n: g + rho * np.abs(g).max() * rng.standard_normal(g.shape) for n, g in G.items()}

        pert = oracle_replay(c, inp, events=events, grad_hook=hook)
        one = dict(out=[], grad_in=[], G=[], m=[], v=[], theta=[])
        for i in range(len(ref["out"])):
            one["out"].append(rel_err(np.atleast_1d(pert["out"][i]), np.atleast_1d(ref["out"][i])))
            one["grad_in"].append(0.0 if ref["grad_in"][i] is None else rel_err(pert["grad_in"][i], ref["grad_in"][i]))
        for s in range(len(ref["G"])):
            # G of update s as the perturbed trajectory saw it (before its own perturbation)
            for key in ("G", "m", "v", "theta"):
                one[key].append({n: rel_err(pert[key][s][n], ref[key][s][n]) for n in ref[key][s]})
        if out is None:
            out = one
            continue
        for key in ("out", "grad_in"):
            out[key] = [max(a, b) for a, b in zip(out[key], one[key])]
        for key in ("G", "m", "v", "theta"):
            out[key] = [{n: max(a[n], b[n]) for n in a} for a, b in zip(out[key], one[key])]
    return out


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
def compare_replays(c, g, o, sens=None, theta0=None):
    """Asserts parity of a GPU replay ``g`` with an oracle replay ``o``; returns the error report.

    sens: oracle_sensitivity() output (allowances downstream of the first update);
    theta0: the initial parameters (dict), for the property check of the first update.
    """
    rep = {}
    M = len(o["out"])
    assert g["tF"] == o["tF"] and g["tB"] == o["tB"], "version stamps differ"
    assert g["delta"] == o["delta"]
    assert len(g["G"]) == len(o["G"]), "number of updates differs"
    t_act, t_grad = tol(c, "act"), tol(c, "grad")

    def lim(base, allowance, downstream):
        return max(base, 2.0 * allowance) if (downstream and sens is not None) else base

    worst = dict(out=0.0, grad_in=0.0, out_after_update=0.0, grad_in_after_update=0.0, G=0.0, G_after_update=0.0,
                 theta=0.0, m=0.0, v=0.0, adamw_property=0.0)
    for i in range(M):
        after_f = (o["tF"][i] or 0) > 0       # forward ran at an updated version
        after_b = (o["tB"][i] or 0) > 0       # backward ran at an updated version
        if o["out"][i] is not None:
            e = rel_err(np.atleast_1d(g["out"][i]), np.atleast_1d(o["out"][i]))
            key = "out_after_update" if after_f else "out"
            worst[key] = max(worst[key], e)
            L = lim(t_act, sens["out"][i] if sens else 0.0, after_f)
            assert e <= L, f"output of micro-batch {i}: {e:.3e} (limit {L:.3e})"
        if o["grad_in"][i] is not None:
            e = rel_err(g["grad_in"][i], o["grad_in"][i])
            key = "grad_in_after_update" if after_b else "grad_in"
            worst[key] = max(worst[key], e)
            L = lim(t_grad, sens["grad_in"][i] if sens else 0.0, after_b)
            assert e <= L, f"input gradient of micro-batch {i}: {e:.3e} (limit {L:.3e})"
    names = [n for n, _, _ in inputs.param_specs(c)]
    b1, b2 = c["beta1"], c["beta2"]
    masked = {n: None for n in names}
    gerr = {n: None for n in names}
    n_masked = n_total = 0
    budget = 0.0
    for s in range(len(o["G"])):
        budget += 2.0 * oadamw.lr_at(c, s + 1) * oadamw.direction_bound(s + 1, b1, b2)
        for n in names:
            sv = (lambda key: sens[key][s][n]) if sens else (lambda key: 0.0)
            gg, og = g["G"][s][n], o["G"][s][n]
            e = rel_err(gg, og)
            worst["G" if s == 0 else "G_after_update"] = max(worst["G" if s == 0 else "G_after_update"], e)
            L = lim(t_grad, sv("G"), s > 0)
            assert e <= L, f"G[{n}] before update {s + 1}: {e:.3e} (limit {L:.3e})"
            d = np.abs(gg - og)
            gerr[n] = d if gerr[n] is None else np.maximum(gerr[n], d)
            for key in ("m", "v"):
                e = rel_err(g[key][s][n], o[key][s][n])
                worst[key] = max(worst[key], e)
                L = lim(t_grad, sv(key), s > 0)
                assert e <= L, f"{key}[{n}] after update {s + 1}: {e:.3e} (limit {L:.3e})"
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
            # parameters against the oracle
            vhat = o["v"][s][n] / (1.0 - b2 ** (s + 1))
            amb = np.sqrt(vhat) + c["eps"] < (3.0 / t_grad) * gerr[n]
            masked[n] = amb if masked[n] is None else (masked[n] | amb)
            th_g, th_o = g["theta"][s][n], o["theta"][s][n]
            keep = ~masked[n]
            den = np.abs(th_o).max()
            if keep.any():
                diff = np.abs(th_g - th_o)[keep].max()
                e = float(diff / den) if den > 0 else float(diff)
                worst["theta"] = max(worst["theta"], e)
                L = lim(t_grad, sv("theta"), s > 0)
                assert e <= L, f"theta[{n}] after update {s + 1}: {e:.3e} (limit {L:.3e})"
            if masked[n].any():
                dev = np.abs(th_g - th_o)[masked[n]].max()
                assert dev <= budget + t_grad * den, f"theta[{n}] invalid at an ill-conditioned element: {dev:.3e}"
            n_masked += int(masked[n].sum())
            n_total += masked[n].size
    rep.update(worst)
    rep["ill_conditioned_fraction"] = n_masked / max(n_total, 1)
    return rep
