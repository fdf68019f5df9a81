"""Pins of the oracle's stage function: finite differences, special cases, and
torch fp64 autograd as an independent implementation (including the paper's
own mechanism for backwards at a newer parameter version)."""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import model, stage

TINY = dict(kind="middle", n_layers=2, d_model=8, n_heads=2, head_dim=4, d_ff=32, seq=5,
            micro_batch=2, vocab=11, max_pos=7, ln_eps=1e-5)


def _cfg(**kw):
    c = dict(TINY)
    c.update(kw)
    return c


def _params(cfg, seed, std=0.3, bias_std=0.1):
    """Random parameters (non-trivial gammas and biases so every term matters)."""
    r = np.random.default_rng(seed)
    p = {}
    for name, shape in stage.param_shapes(cfg):
        leaf = name.split(".")[-1]
        if leaf.endswith("_g"):
            p[name] = 1.0 + 0.2 * r.standard_normal(shape)
        elif leaf.startswith("b_") or leaf.endswith("_b"):
            p[name] = bias_std * r.standard_normal(shape)
        else:
            p[name] = std * r.standard_normal(shape)
    return p


def _stage_input(cfg, r):
    if cfg["kind"] == "first":
        return r.integers(0, cfg["vocab"], size=(cfg["micro_batch"], cfg["seq"]))
    return r.standard_normal((cfg["micro_batch"] * cfg["seq"], cfg["d_model"]))


def _scalar(cfg, theta, inp, g, tgt):
    out, _ = stage.stage_fwd(cfg, theta, inp, tgt)
    return out if cfg["kind"] == "last" else float((out * g).sum())


@pytest.mark.parametrize("kind", ["middle", "first", "last"])
def test_gradients_match_central_differences(kind):
    cfg = _cfg(kind=kind)
    r = np.random.default_rng(1)
    theta = _params(cfg, 2)
    inp = _stage_input(cfg, r)
    T = cfg["micro_batch"] * cfg["seq"]
    g = r.standard_normal((T, cfg["d_model"]))
    tgt = r.integers(0, cfg["vocab"], size=(cfg["micro_batch"], cfg["seq"])) if kind == "last" else None
    out, saved = stage.stage_fwd(cfg, theta, inp, tgt)
    K = 1
    grad_in, grads = stage.stage_bwd(cfg, theta, saved, None if kind == "last" else g, K,
                                     ids=inp if kind == "first" else None)
    h = 1e-6
    rr = np.random.default_rng(3)
    for name, arr in theta.items():
        # every element of small tensors, a random sample of large ones
        idx = list(np.ndindex(arr.shape))
        if len(idx) > 40:
            idx = [idx[i] for i in rr.choice(len(idx), 40, replace=False)]
        for ix in idx:
            old = arr[ix]
            arr[ix] = old + h
            fp = _scalar(cfg, theta, inp, g, tgt)
            arr[ix] = old - h
            fm = _scalar(cfg, theta, inp, g, tgt)
            arr[ix] = old
            fd = (fp - fm) / (2 * h)
            assert abs(grads[name][ix] - fd) <= 1e-7 * max(1.0, abs(fd)) + 1e-8, (name, ix, grads[name][ix], fd)
    if kind != "first":
        for _ in range(30):
            ix = (rr.integers(T), rr.integers(cfg["d_model"]))
            old = inp[ix]
            inp[ix] = old + h
            fp = _scalar(cfg, theta, inp, g, tgt)
            inp[ix] = old - h
            fm = _scalar(cfg, theta, inp, g, tgt)
            inp[ix] = old
            fd = (fp - fm) / (2 * h)
            assert abs(grad_in[ix] - fd) <= 1e-7 * max(1.0, abs(fd)) + 1e-8


def test_single_key_attention_returns_v():
    # S = 1: each query sees only its own key, softmax is 1, o = v.
    r = np.random.default_rng(0)
    mu, H, dh = 3, 2, 4
    qkv = r.standard_normal((mu, 3 * H * dh))
    o, lse = model.attention_fwd(qkv, mu, 1, H, dh)
    np.testing.assert_array_equal(o, qkv[:, 2 * H * dh:])
    q, k = qkv[:, :H * dh].reshape(mu, H, dh), qkv[:, H * dh:2 * H * dh].reshape(mu, H, dh)
    np.testing.assert_allclose(lse[:, :, 0], (q * k).sum(-1) / math.sqrt(dh), rtol=1e-14)


def test_first_query_attends_to_itself_only():
    r = np.random.default_rng(1)
    mu, S, H, dh = 2, 6, 2, 4
    qkv = r.standard_normal((mu * S, 3 * H * dh))
    o, _ = model.attention_fwd(qkv, mu, S, H, dh)
    for b in range(mu):
        np.testing.assert_allclose(o[b * S], qkv[b * S, 2 * H * dh:], rtol=1e-13)


def test_zero_weights_give_residual_plus_biases():
    cfg = _cfg()
    r = np.random.default_rng(2)
    p = {n: np.zeros(s) for n, s in stage.param_shapes(cfg)}
    for l in range(cfg["n_layers"]):
        p[f"h{l}.b_o"] = r.standard_normal(cfg["d_model"])
        p[f"h{l}.b_2"] = r.standard_normal(cfg["d_model"])
        p[f"h{l}.ln1_g"] = np.ones(cfg["d_model"])
        p[f"h{l}.ln2_g"] = np.ones(cfg["d_model"])
    x = r.standard_normal((cfg["micro_batch"] * cfg["seq"], cfg["d_model"]))
    y, _ = stage.stage_fwd(cfg, p, x)
    expect = x + sum(p[f"h{l}.b_o"] + p[f"h{l}.b_2"] for l in range(cfg["n_layers"]))
    np.testing.assert_allclose(y, expect, rtol=1e-14, atol=1e-14)


def test_layernorm_of_constant_row_is_beta():
    beta = np.arange(6.0)
    n, mean, rstd = model.layernorm_fwd(np.full((3, 6), 2.5), np.ones(6) * 3.0, beta, 1e-5)
    np.testing.assert_allclose(n, np.broadcast_to(beta, (3, 6)), atol=1e-12)
    np.testing.assert_allclose(mean, 2.5)
    np.testing.assert_allclose(rstd, 1 / math.sqrt(1e-5))


def test_uniform_logits_cross_entropy_is_log_vocab():
    # W_lm = 0 makes every logit 0: the loss is ln V exactly, for V = 50257 too.
    V, d, T = 50257, 8, 6
    r = np.random.default_rng(3)
    y = r.standard_normal((T, d))
    tgt = r.integers(0, V, size=(1, T))
    loss, s = model.head_fwd(y, tgt, np.ones(d), np.zeros(d), np.zeros((V, d)), 1e-5)
    assert loss == pytest.approx(math.log(V), rel=1e-14)
    assert math.log(V) == pytest.approx(10.8249, abs=5e-5)
    # softmax - onehot sums to zero over the vocabulary, so the LM-head gradient
    # summed over its rows vanishes.
    _, _, _, g_w = model.head_bwd(s, np.ones(d), np.zeros((V, d)), 1.0 / T)
    np.testing.assert_allclose(g_w.sum(axis=0), 0.0, atol=1e-11)


def test_embedding_gradient_of_repeated_token_is_row_sum():
    ids = np.array([[3, 1, 3], [3, 0, 2]])
    r = np.random.default_rng(4)
    dx = r.standard_normal((6, 4))
    g_wte, g_wpe = model.embed_bwd(dx, ids, vocab=5, max_pos=4)
    np.testing.assert_allclose(g_wte[3], dx[0] + dx[2] + dx[3])
    np.testing.assert_allclose(g_wte[4], 0.0)
    np.testing.assert_allclose(g_wpe[1], dx[1] + dx[4])
    np.testing.assert_allclose(g_wpe[3], 0.0)


# ---------------------------------------------------------------------------
# torch fp64 autograd: an independent implementation of the same stage
# ---------------------------------------------------------------------------
def _torch_stage(cfg, P, inp, tgt):
    """The stage written with torch.nn.functional library ops."""
    mu, S, H, dh, d = cfg["micro_batch"], cfg["seq"], cfg["n_heads"], cfg["head_dim"], cfg["d_model"]
    if cfg["kind"] == "first":
        x = (F.embedding(inp, P["wte"]) + P["wpe"][:S][None]).reshape(mu * S, d)
    else:
        x = inp
    for l in range(cfg["n_layers"]):
        g = lambda n: P[f"h{l}.{n}"]
        n1 = F.layer_norm(x, (d,), g("ln1_g"), g("ln1_b"), cfg["ln_eps"])
        qkv = F.linear(n1, g("w_qkv"), g("b_qkv"))
        q, k, v = [qkv[:, j * d:(j + 1) * d].reshape(mu, S, H, dh).transpose(1, 2) for j in range(3)]
        o = F.scaled_dot_product_attention(q, k, v, is_causal=True)
        o = o.transpose(1, 2).reshape(mu * S, d)
        x1 = x + F.linear(o, g("w_o"), g("b_o"))
        n2 = F.layer_norm(x1, (d,), g("ln2_g"), g("ln2_b"), cfg["ln_eps"])
        x = x1 + F.linear(F.gelu(F.linear(n2, g("w_1"), g("b_1")), approximate="tanh"), g("w_2"), g("b_2"))
    if cfg["kind"] == "last":
        nf = F.layer_norm(x, (d,), P["lnf_g"], P["lnf_b"], cfg["ln_eps"])
        return F.cross_entropy(F.linear(nf, P["w_lm"]), tgt.reshape(-1))
    return x


@pytest.mark.parametrize("kind", ["middle", "first", "last"])
def test_matches_torch_autograd(kind):
    cfg = _cfg(kind=kind, seq=7, vocab=13)
    r = np.random.default_rng(5)
    theta = _params(cfg, 6)
    inp = _stage_input(cfg, r)
    T = cfg["micro_batch"] * cfg["seq"]
    g = r.standard_normal((T, cfg["d_model"]))
    tgt = r.integers(0, cfg["vocab"], size=(cfg["micro_batch"], cfg["seq"]))
    K = 3
    out, saved = stage.stage_fwd(cfg, theta, inp, tgt if kind == "last" else None)
    gin, grads = stage.stage_bwd(cfg, theta, saved, g, K, ids=inp if kind == "first" else None)

    P = {n: torch.tensor(v, requires_grad=True) for n, v in theta.items()}
    tin = torch.tensor(inp) if kind == "first" else torch.tensor(inp, requires_grad=True)
    tout = _torch_stage(cfg, P, tin, torch.tensor(tgt))
    if kind == "last":
        (tout / K).backward()
        assert out == pytest.approx(tout.item(), rel=1e-12)
    else:
        tout.backward(torch.tensor(g))
        np.testing.assert_allclose(out, tout.detach().numpy(), rtol=1e-11, atol=1e-12)
    for n in theta:
        np.testing.assert_allclose(grads[n], P[n].grad.numpy(), rtol=1e-9, atol=1e-12, err_msg=n)
    if kind != "first":
        np.testing.assert_allclose(gin, tin.grad.numpy(), rtol=1e-9, atol=1e-12)


@pytest.mark.parametrize("kind", ["middle", "last"])
def test_stale_backward_matches_paper_mechanism(kind):
    """Eq. (1) as the paper implements it: autograd's saved tensors from a forward
    at theta0, parameters then overwritten in place without a version bump
    (``.data``), backward at the new values. The oracle's backward from the
    activations saved at theta0 with parameters theta1 must agree."""
    cfg = _cfg(kind=kind, seq=6, vocab=9)
    r = np.random.default_rng(7)
    th0 = _params(cfg, 8)
    th1 = {n: v + 0.05 * r.standard_normal(v.shape) for n, v in th0.items()}
    inp = _stage_input(cfg, r)
    T = cfg["micro_batch"] * cfg["seq"]
    g = r.standard_normal((T, cfg["d_model"]))
    tgt = r.integers(0, cfg["vocab"], size=(cfg["micro_batch"], cfg["seq"]))

    _, saved = stage.stage_fwd(cfg, th0, inp, tgt if kind == "last" else None)
    gin, grads = stage.stage_bwd(cfg, th1, saved, g, 1)

    P = {n: torch.tensor(v, requires_grad=True) for n, v in th0.items()}
    tin = torch.tensor(inp, requires_grad=True)
    tout = _torch_stage(cfg, P, tin, torch.tensor(tgt))
    for n in P:
        P[n].data.copy_(torch.tensor(th1[n]))
    if kind == "last":
        tout.backward()
    else:
        tout.backward(torch.tensor(g))
    for n in th0:
        np.testing.assert_allclose(grads[n], P[n].grad.numpy(), rtol=1e-9, atol=1e-12, err_msg=n)
    np.testing.assert_allclose(gin, tin.grad.numpy(), rtol=1e-9, atol=1e-12)
    # and the drift is real: differentiating at theta0 gives something else
    gin0, _ = stage.stage_bwd(cfg, th0, saved, g, 1)
    assert np.abs(gin0 - gin).max() > 1e-3 * np.abs(gin).max()
