"""Pins of the oracle's dropout: the generator against its published
known-answer vectors, the mask statistics, and the stage with dropout against
finite differences and torch fp64 autograd with the same masks."""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import dropout, stage

TINY = dict(kind="middle", n_layers=2, d_model=8, n_heads=2, head_dim=4, d_ff=32, seq=6,
            micro_batch=2, vocab=11, max_pos=7, ln_eps=1e-5, dropout=0.25, dropout_seed=1234,
            lr=1e-2, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1)


def _cfg(**kw):
    c = dict(TINY)
    c.update(kw)
    return c


def _params(cfg, seed):
    r = np.random.default_rng(seed)
    p = {}
    for name, shape in stage.param_shapes(cfg):
        leaf = name.split(".")[-1]
        p[name] = (1.0 + 0.2 * r.standard_normal(shape)) if leaf.endswith("_g") else 0.3 * r.standard_normal(shape)
    return p


def _input(cfg, r):
    if cfg["kind"] == "first":
        return r.integers(0, cfg["vocab"], size=(cfg["micro_batch"], cfg["seq"]))
    return r.standard_normal((cfg["micro_batch"] * cfg["seq"], cfg["d_model"]))


def test_philox_known_answers():
    # Known-answer vectors of Philox4x32-10 published with the generator's
    # reference implementation (Random123): counter, key -> output.
    cases = [((0, 0, 0, 0), (0, 0), (0x6627E8D5, 0xE169C58D, 0xBC57AC4C, 0x9B00DBD8)),
             ((0xFFFFFFFF,) * 4, (0xFFFFFFFF, 0xFFFFFFFF), (0x408F276D, 0x41C83B0E, 0xA20BC7C6, 0x6D5451FD)),
             ((0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344), (0xA4093822, 0x299F31D0),
              (0xD16CFE09, 0x94FDCCEB, 0x5001E420, 0x24126EA1))]
    for ctr, key, want in cases:
        got = dropout.philox4x32_10(*ctr, *key)
        assert tuple(int(w) for w in got) == want


def test_threshold_and_scale():
    assert dropout.threshold(0.1) == 6554          # float32(0.1) * 65536 = 6553.6...
    assert dropout.threshold(0.0) == 0
    assert dropout.threshold(0.5) == 32768
    assert dropout.scale(0.5) == 2.0


@pytest.mark.parametrize("p", [0.1, 0.5])
def test_keep_fraction_is_binomial(p):
    keep = dropout.keep_elementwise(7, 3, 1, dropout.SITE_FFN, 256, 512, p)
    n = keep.size
    q = 1.0 - dropout.threshold(p) / 65536.0
    assert abs(keep.mean() - q) <= 5.0 * math.sqrt(q * (1 - q) / n)
    att = dropout.keep_attention(7, 3, 1, 2, 2, 128, p)
    assert abs(att.mean() - q) <= 5.0 * math.sqrt(q * (1 - q) / att.size)


def test_masks_depend_on_every_index():
    base = dropout.keep_elementwise(1, 0, 0, dropout.SITE_PROJ, 64, 64, 0.5)
    for other in [dropout.keep_elementwise(2, 0, 0, dropout.SITE_PROJ, 64, 64, 0.5),
                  dropout.keep_elementwise(1, 1, 0, dropout.SITE_PROJ, 64, 64, 0.5),
                  dropout.keep_elementwise(1, 0, 1, dropout.SITE_PROJ, 64, 64, 0.5),
                  dropout.keep_elementwise(1, 0, 0, dropout.SITE_FFN, 64, 64, 0.5)]:
        assert 0.4 < (base != other).mean() < 0.6
    a = dropout.keep_attention(1, 0, 0, 2, 2, 32, 0.5)
    assert 0.4 < (a[0, 0] != a[0, 1]).mean() < 0.6 and 0.4 < (a[0, 0] != a[1, 0]).mean() < 0.6
    # neighbouring elements draw different 16-bit values (no value is reused)
    assert 0.4 < (base[:, 0::2] != base[:, 1::2]).mean() < 0.6
    assert 0.4 < (a[0, 0, 0::2] != a[0, 0, 1::2]).mean() < 0.6


@pytest.mark.parametrize("kind", ["middle", "first", "last"])
def test_zero_rate_is_no_dropout(kind):
    cfg = _cfg(kind=kind, dropout=0.0)
    plain = {k: v for k, v in cfg.items() if not k.startswith("dropout")}
    r = np.random.default_rng(0)
    theta = _params(cfg, 1)
    inp = _input(cfg, r)
    tgt = r.integers(0, cfg["vocab"], size=(cfg["micro_batch"], cfg["seq"]))
    a, _ = stage.stage_fwd(cfg, theta, inp, tgt if kind == "last" else None, mb=5)
    b, _ = stage.stage_fwd(plain, theta, inp, tgt if kind == "last" else None)
    np.testing.assert_array_equal(a, b)


def _scalar(cfg, theta, inp, g, tgt, mb):
    out, _ = stage.stage_fwd(cfg, theta, inp, tgt, mb=mb)
    return out if cfg["kind"] == "last" else float((out * g).sum())


@pytest.mark.parametrize("kind", ["middle", "first", "last"])
def test_gradients_with_dropout_match_central_differences(kind):
    """For a fixed micro-batch the masks are constants, so the stage is smooth;
    the backward's masked branch gradients, masked attention probabilities and
    masked embedding gradient must agree with central differences."""
    cfg = _cfg(kind=kind)
    mb = 3
    r = np.random.default_rng(1)
    theta = _params(cfg, 2)
    inp = _input(cfg, r)
    T = cfg["micro_batch"] * cfg["seq"]
    g = r.standard_normal((T, cfg["d_model"]))
    tgt = r.integers(0, cfg["vocab"], size=(cfg["micro_batch"], cfg["seq"])) if kind == "last" else None
    _, saved = stage.stage_fwd(cfg, theta, inp, tgt, mb=mb)
    grad_in, grads = stage.stage_bwd(cfg, theta, saved, None if kind == "last" else g, 1,
                                     ids=inp if kind == "first" else None)
    h = 1e-6
    rr = np.random.default_rng(3)
    for name, arr in theta.items():
        idx = list(np.ndindex(arr.shape))
        if len(idx) > 25:
            idx = [idx[i] for i in rr.choice(len(idx), 25, replace=False)]
        for ix in idx:
            old = arr[ix]
            arr[ix] = old + h
            fp = _scalar(cfg, theta, inp, g, tgt, mb)
            arr[ix] = old - h
            fm = _scalar(cfg, theta, inp, g, tgt, mb)
            arr[ix] = old
            fd = (fp - fm) / (2 * h)
            assert abs(grads[name][ix] - fd) <= 1e-7 * max(1.0, abs(fd)) + 1e-8, (name, ix, grads[name][ix], fd)
    if kind != "first":
        for _ in range(20):
            ix = (rr.integers(T), rr.integers(cfg["d_model"]))
            old = inp[ix]
            inp[ix] = old + h
            fp = _scalar(cfg, theta, inp, g, tgt, mb)
            inp[ix] = old - h
            fm = _scalar(cfg, theta, inp, g, tgt, mb)
            inp[ix] = old
            fd = (fp - fm) / (2 * h)
            assert abs(grad_in[ix] - fd) <= 1e-7 * max(1.0, abs(fd)) + 1e-8


def _torch_stage(cfg, P, inp, tgt, masks):
    """The stage with torch library ops; dropout as multiplication by the given
    keep masks (the probabilities are formed by torch.softmax)."""
    mu, S, H, dh, d = cfg["micro_batch"], cfg["seq"], cfg["n_heads"], cfg["head_dim"], cfg["d_model"]
    sc = dropout.scale(cfg["dropout"])
    if cfg["kind"] == "first":
        x = (F.embedding(inp, P["wte"]) + P["wpe"][:S][None]).reshape(mu * S, d) * masks["embed"] * sc
    else:
        x = inp
    causal = torch.ones(S, S, dtype=torch.bool).tril()
    for l in range(cfg["n_layers"]):
        g = lambda n: P[f"h{l}.{n}"]
        m = masks["blocks"][l]
        n1 = F.layer_norm(x, (d,), g("ln1_g"), g("ln1_b"), cfg["ln_eps"])
        qkv = F.linear(n1, g("w_qkv"), g("b_qkv"))
        q, k, v = [qkv[:, j * d:(j + 1) * d].reshape(mu, S, H, dh).transpose(1, 2) for j in range(3)]
        s = (q @ k.transpose(-1, -2).contiguous()) / math.sqrt(dh)
        prob = torch.softmax(s.masked_fill(~causal, float("-inf")), dim=-1) * m["attn"] * sc
        o = (prob @ v).transpose(1, 2).reshape(mu * S, d)
        x1 = x + F.linear(o, g("w_o"), g("b_o")) * m["proj"] * sc
        n2 = F.layer_norm(x1, (d,), g("ln2_g"), g("ln2_b"), cfg["ln_eps"])
        hid = F.gelu(F.linear(n2, g("w_1"), g("b_1")), approximate="tanh")
        x = x1 + F.linear(hid, g("w_2"), g("b_2")) * m["ffn"] * sc
    if cfg["kind"] == "last":
        nf = F.layer_norm(x, (d,), P["lnf_g"], P["lnf_b"], cfg["ln_eps"])
        return F.cross_entropy(F.linear(nf, P["w_lm"]), tgt.reshape(-1))
    return x


@pytest.mark.parametrize("kind", ["middle", "first", "last"])
def test_dropout_stage_matches_torch_autograd(kind):
    cfg = _cfg(kind=kind, seq=7, vocab=13)
    mb, K = 6, 2
    r = np.random.default_rng(5)
    theta = _params(cfg, 6)
    inp = _input(cfg, r)
    T, d, p = cfg["micro_batch"] * cfg["seq"], cfg["d_model"], cfg["dropout"]
    g = r.standard_normal((T, d))
    tgt = r.integers(0, cfg["vocab"], size=(cfg["micro_batch"], cfg["seq"]))
    out, saved = stage.stage_fwd(cfg, theta, inp, tgt if kind == "last" else None, mb=mb)
    gin, grads = stage.stage_bwd(cfg, theta, saved, g, K, ids=inp if kind == "first" else None)

    seed = cfg["dropout_seed"]
    masks = {"embed": torch.tensor(dropout.keep_elementwise(seed, mb, 0, dropout.SITE_EMBED, T, d, p),
                                   dtype=torch.float64),
             "blocks": [{"attn": torch.tensor(dropout.keep_attention(seed, mb, l, cfg["micro_batch"], cfg["n_heads"],
                                                                     cfg["seq"], p), dtype=torch.float64),
                         "proj": torch.tensor(dropout.keep_elementwise(seed, mb, l, dropout.SITE_PROJ, T, d, p),
                                              dtype=torch.float64),
                         "ffn": torch.tensor(dropout.keep_elementwise(seed, mb, l, dropout.SITE_FFN, T, d, p),
                                             dtype=torch.float64)}
                        for l in range(cfg["n_layers"])]}
    P = {n: torch.tensor(v, requires_grad=True) for n, v in theta.items()}
    tin = torch.tensor(inp) if kind == "first" else torch.tensor(inp, requires_grad=True)
    tout = _torch_stage(cfg, P, tin, torch.tensor(tgt), masks)
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


def test_masks_follow_the_micro_batch_not_the_version():
    """A replay with dropout: the checkpointed stage (forward recomputed in the
    backward) equals the stored one at delay 0, so both draw the same masks
    for a micro-batch; different micro-batches see different masks."""
    cfg = _cfg()
    r = np.random.default_rng(9)
    theta = _params(cfg, 10)
    xs = [_input(cfg, r) for _ in range(4)]
    dys = [0.1 * r.standard_normal((cfg["micro_batch"] * cfg["seq"], cfg["d_model"])) for _ in range(4)]
    a = stage.replay(cfg, theta, 2, 0, xs, dys)
    b = stage.replay(cfg, theta, 2, 0, xs, dys, recompute=True)
    for i in range(4):
        np.testing.assert_array_equal(a["out"][i], b["out"][i])
        np.testing.assert_array_equal(a["grad_in"][i], b["grad_in"][i])
    y0, _ = stage.stage_fwd(cfg, theta, xs[0], mb=0)
    y1, _ = stage.stage_fwd(cfg, theta, xs[0], mb=1)
    assert np.abs(y0 - y1).max() > 1e-3
