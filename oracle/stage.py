"""One PACI stage and the replay of its event list, float64 (test infrastructure).

A stage holds a single parameter copy theta, a gradient accumulator G, the AdamW
moments and the counters of Alg. 1 (appendix "Stage-level execution rule").
Forward F_m stores the activations its backward needs; backward B_m computes
the local gradient and the input gradient, adds the local gradient to G, and
after every K-th backward the stage applies one AdamW update with G and clears
G (Alg. 1, accumulate / update / reset). There is no weight stash
(appendix "Memory and synchronization properties").

Drift semantics (Eq. (1), Sec. 3.1, and the appendix "PyTorch modifications"):
a backward differentiates the activations saved by its own forward, while every
parameter it reads is the version current when it runs. Activations that depend
on parameters are therefore saved at forward time, never recomputed.

With ``recompute=True`` the stage follows the activation-checkpointed variant
(appendix "Activation checkpointing"): a forward keeps only its stage input
(and the targets or token ids), and the backward first recomputes the stage's
activations under the version current at that time, then differentiates them
at that same version. The output gradient is still the one the pipeline
delivered for the original forward.

Parameter naming and order (nn.Linear weights are [out, in]):
  first stage prefix  wte [V, d], wpe [max_pos, d]
  block l             h{l}.ln1_g, h{l}.ln1_b, h{l}.w_qkv [3d, d], h{l}.b_qkv,
                      h{l}.w_o [d, d], h{l}.b_o, h{l}.ln2_g, h{l}.ln2_b,
                      h{l}.w_1 [f, d], h{l}.b_1, h{l}.w_2 [d, f], h{l}.b_2
  last stage suffix   lnf_g, lnf_b, w_lm [V, d]
Weight decay applies to the w_* matrices only (no decay on biases, LayerNorm
parameters or embeddings, appendix "Detailed experimental setup").
"""
import numpy as np

from . import adamw, dropout, model
from .schedule import StageCounters, canonical_events

BLOCK_PARAMS = ("ln1_g", "ln1_b", "w_qkv", "b_qkv", "w_o", "b_o",
                "ln2_g", "ln2_b", "w_1", "b_1", "w_2", "b_2")


def param_shapes(cfg):
    """Ordered (name, shape) list of a stage's parameters."""
    d, f, V, P = cfg["d_model"], cfg["d_ff"], cfg.get("vocab", 0), cfg.get("max_pos", 0)
    out = []
    if cfg["kind"] == "first":
        out += [("wte", (V, d)), ("wpe", (P, d))]
    per = {"ln1_g": (d,), "ln1_b": (d,), "w_qkv": (3 * d, d), "b_qkv": (3 * d,),
           "w_o": (d, d), "b_o": (d,), "ln2_g": (d,), "ln2_b": (d,),
           "w_1": (f, d), "b_1": (f,), "w_2": (d, f), "b_2": (d,)}
    for l in range(cfg["n_layers"]):
        out += [(f"h{l}.{n}", per[n]) for n in BLOCK_PARAMS]
    if cfg["kind"] == "last":
        out += [("lnf_g", (d,)), ("lnf_b", (d,)), ("w_lm", (V, d))]
    return out


def decayed(name):
    return name.split(".")[-1].startswith("w_")


def _drop_masks(cfg, mb, block):
    """Keep masks of one block for micro-batch ``mb`` (None without dropout)."""
    p = cfg.get("dropout", 0.0)
    if not p:
        return None
    seed, mu, S, H, d = cfg.get("dropout_seed", 0), cfg["micro_batch"], cfg["seq"], cfg["n_heads"], cfg["d_model"]
    T = mu * S
    return dict(scale=dropout.scale(p),
                attn=dropout.keep_attention(seed, mb, block, mu, H, S, p),
                proj=dropout.keep_elementwise(seed, mb, block, dropout.SITE_PROJ, T, d, p),
                ffn=dropout.keep_elementwise(seed, mb, block, dropout.SITE_FFN, T, d, p))


def stage_fwd(cfg, theta, inp, targets=None, mb=0):
    """F_i at parameters ``theta``. Returns (output, saved).

    middle: inp is x [T, d], output y [T, d]; first: inp is ids [mu, S];
    last: output is the mean cross-entropy of the micro-batch. With
    cfg["dropout"] = p > 0 the masks of micro-batch ``mb`` are applied
    (oracle/dropout.py); the embedding sum of a first stage is dropped too.
    """
    saved = {"blocks": []}
    if cfg["kind"] == "first":
        x = model.embed_fwd(inp, theta["wte"], theta["wpe"])
        if cfg.get("dropout", 0.0):
            p = cfg["dropout"]
            keep = dropout.keep_elementwise(cfg.get("dropout_seed", 0), mb, 0, dropout.SITE_EMBED, x.shape[0],
                                            x.shape[1], p)
            saved["embed_drop"] = keep * dropout.scale(p)
            x = x * saved["embed_drop"]
    else:
        x = inp
    for l in range(cfg["n_layers"]):
        p = {n: theta[f"h{l}.{n}"] for n in BLOCK_PARAMS}
        x, s = model.block_fwd(x, p, cfg, _drop_masks(cfg, mb, l))
        saved["blocks"].append(s)
    if cfg["kind"] == "last":
        loss, saved["head"] = model.head_fwd(x, targets, theta["lnf_g"], theta["lnf_b"],
                                             theta["w_lm"], cfg["ln_eps"])
        return loss, saved
    return x, saved


def stage_bwd(cfg, theta, saved, grad_out, K, ids=None):
    """Backward of stage_fwd from ``saved`` at parameters ``theta``.

    Returns (grad_in, grads). For the last stage the seed is
    (softmax(z) - onehot(target)) / (T * K): the micro-batch loss is a mean over
    its T tokens and K micro-batches make one update. grad_in is None for the
    first stage (its input is token ids).
    """
    g = {}
    if cfg["kind"] == "last":
        T = cfg["micro_batch"] * cfg["seq"]
        dy, g["lnf_g"], g["lnf_b"], g["w_lm"] = model.head_bwd(
            saved["head"], theta["lnf_g"], theta["w_lm"], 1.0 / (T * K))
    else:
        dy = grad_out
    for l in reversed(range(cfg["n_layers"])):
        p = {n: theta[f"h{l}.{n}"] for n in BLOCK_PARAMS}
        dy, gl = model.block_bwd(dy, saved["blocks"][l], p, cfg)
        for n, v in gl.items():
            g[f"h{l}.{n}"] = v
    if cfg["kind"] == "first":
        if "embed_drop" in saved:
            dy = dy * saved["embed_drop"]
        g["wte"], g["wpe"] = model.embed_bwd(dy, ids, cfg["vocab"], cfg["max_pos"])
        return None, g
    return dy, g


class Stage:
    """Alg. 1 for one stage over float64 state."""

    def __init__(self, cfg, params, K, delay, recompute=False):
        self.cfg, self.K, self.delay, self.recompute = cfg, K, delay, recompute
        self.names = [n for n, _ in param_shapes(cfg)]
        self.theta = {n: np.array(params[n], dtype=np.float64) for n in self.names}
        self.G = {n: np.zeros_like(self.theta[n]) for n in self.names}
        self.m = {n: np.zeros_like(self.theta[n]) for n in self.names}
        self.v = {n: np.zeros_like(self.theta[n]) for n in self.names}
        self.counters = StageCounters(K, delay)
        self.saved = {}
        self.ids = {}
        self.applied = self.skipped = 0   # updates applied / skipped by the non-finite guard

    @property
    def version(self):
        return self.counters.t

    def forward(self, mb, inp, targets=None):
        """F_mb: returns (output, t^F). Stores the activations until B_mb."""
        version = self.counters.forward(mb)
        out, saved = stage_fwd(self.cfg, self.theta, inp, targets, mb=mb)
        # checkpointed: keep the input only (the activations are dropped here)
        self.saved[mb] = (inp, targets) if self.recompute else saved
        if self.cfg["kind"] == "first":
            self.ids[mb] = inp
        return out, version

    def backward(self, mb, grad_out=None):
        """B_mb at the current parameters: returns (grad_in, t^B, update_due)."""
        version = self.counters.backward(mb)
        saved = self.saved.pop(mb)
        if self.recompute:   # the activations again (same dropout masks), under the current version
            _, saved = stage_fwd(self.cfg, self.theta, saved[0], saved[1], mb=mb)
        grad_in, g = stage_bwd(self.cfg, self.theta, saved, grad_out, self.K, ids=self.ids.pop(mb, None))
        for n, v in g.items():
            self.G[n] += v
        return grad_in, version, self.counters.step_due

    def step(self):
        """AdamW with the accumulated G, then G <- 0; returns the new version.

        Non-finite guard (the paper implements no handling of invalid gradients,
        Sec. "Limitations"): if any element of G is not finite, no parameter
        or moment changes; G is still cleared and the version still advances,
        so the stamps remain a function of the event order alone. AdamW's
        bias correction and the rate schedule count applied updates only."""
        c = self.cfg
        if not all(np.all(np.isfinite(g)) for g in self.G.values()):
            self.skipped += 1
            for n in self.names:
                self.G[n] = np.zeros_like(self.G[n])
            return self.counters.step()
        self.applied += 1
        t_adam = self.applied
        lr = adamw.lr_at(c, t_adam)
        for n in self.names:
            wd = c["weight_decay"] if decayed(n) else 0.0
            self.theta[n], self.m[n], self.v[n] = adamw.adamw_update(
                self.theta[n], self.G[n], self.m[n], self.v[n], t_adam,
                lr, c["beta1"], c["beta2"], c["eps"], wd)
            self.G[n] = np.zeros_like(self.G[n])
        return self.counters.step()


def _copy(d):
    return {k: v.copy() for k, v in d.items()}


def replay(cfg, params, K, delay, inputs, grad_outs=None, targets=None, events=None, grad_hook=None,
           recompute=False):
    """Run ``events`` (default: the canonical asynchronous 1F1B order) on a Stage.

    inputs[i] is micro-batch i's stage input, grad_outs[i] its output gradient
    (middle and first stages) and targets[i] its token targets (last stage).
    Returns a dict with per-micro-batch outputs, input gradients and stamps,
    and per update the G it consumed and theta, m, v after it.
    ``grad_hook(update_index, G)``, if given, may replace G just before each
    update (the recorded G is the one before the hook); tests use it to
    measure how strongly the trajectory after an update depends on small
    changes of the accumulated gradient. ``recompute`` selects the
    activation-checkpointed stage (see the module docstring).
    """
    M = len(inputs)
    if events is None:
        events = canonical_events(M, K, delay)
    st = Stage(cfg, params, K, delay, recompute=recompute)
    rec = dict(out=[None] * M, grad_in=[None] * M, tF=[None] * M, tB=[None] * M,
               G=[], theta=[], m=[], v=[], events=list(events))
    for kind, i in events:
        if kind == "F":
            tgt = targets[i] if targets is not None else None
            rec["out"][i], rec["tF"][i] = st.forward(i, inputs[i], tgt)
        elif kind == "B":
            go = grad_outs[i] if grad_outs is not None else None
            rec["grad_in"][i], rec["tB"][i], _ = st.backward(i, go)
        else:
            rec["G"].append(_copy(st.G))
            if grad_hook is not None:
                st.G = grad_hook(len(rec["G"]) - 1, st.G)
            st.step()
            rec["theta"].append(_copy(st.theta))
            rec["m"].append(_copy(st.m))
            rec["v"].append(_copy(st.v))
    rec["delta"] = [b - f for f, b in zip(rec["tF"], rec["tB"])]
    rec["final_version"] = st.version
    rec["stage"] = st
    return rec


def replay_with_version_store(cfg, params, K, delay, inputs, grad_outs=None, targets=None,
                              backward_at="current", events=None, grad_hook=None):
    """The same trajectory computed a second way, for cross-checking ``replay``.

    Keeps every parameter version theta^(0), theta^(1), ... and no activation
    store. At B_i it re-runs the forward of micro-batch i at theta^(t^F(i)) to
    obtain the activations, then differentiates at theta^(t^B(i))
    (``backward_at="current"``, Eq. (1)) or at theta^(t^F(i))
    (``backward_at="forward"``, weight stashing; not PACI, used to show that
    the drift is exercised). Versions are counted from the event list itself
    (default: the canonical order). ``grad_hook(update_index, G)`` may replace
    G just before each update, as in ``replay``; the recorded G is the one
    before the hook.
    """
    M = len(inputs)
    if events is None:
        events = canonical_events(M, K, delay)
    names = [n for n, _ in param_shapes(cfg)]
    versions = [{n: np.array(params[n], dtype=np.float64) for n in names}]
    G = {n: np.zeros_like(versions[0][n]) for n in names}
    m = {n: np.zeros_like(versions[0][n]) for n in names}
    v = {n: np.zeros_like(versions[0][n]) for n in names}
    tF, out, grad_in, thetas, Gs = {}, [None] * M, [None] * M, [], []
    for kind, i in events:
        t = len(versions) - 1
        if kind == "F":
            tF[i] = t
            tgt = targets[i] if targets is not None else None
            out[i], _ = stage_fwd(cfg, versions[t], inputs[i], tgt, mb=i)
        elif kind == "B":
            tgt = targets[i] if targets is not None else None
            _, saved = stage_fwd(cfg, versions[tF[i]], inputs[i], tgt, mb=i)
            at = versions[t] if backward_at == "current" else versions[tF[i]]
            go = grad_outs[i] if grad_outs is not None else None
            ids = inputs[i] if cfg["kind"] == "first" else None
            grad_in[i], g = stage_bwd(cfg, at, saved, go, K, ids=ids)
            for n in names:
                G[n] = G[n] + g[n]
        else:
            Gs.append(_copy(G))
            if grad_hook is not None:
                G = grad_hook(len(Gs) - 1, G)
            new = {}
            for n in names:
                wd = cfg["weight_decay"] if decayed(n) else 0.0
                new[n], m[n], v[n] = adamw.adamw_update(
                    versions[t][n], G[n], m[n], v[n], t + 1,
                    adamw.lr_at(cfg, t + 1), cfg["beta1"], cfg["beta2"], cfg["eps"], wd)
                G[n] = np.zeros_like(G[n])
            versions.append(new)
            thetas.append(new)
    return dict(out=out, grad_in=grad_in, theta=thetas, G=Gs)
