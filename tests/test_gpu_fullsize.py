"""Parity at the full workload sizes, sampled, through the C ABI.

At these sizes the oracle cannot replay a schedule, so the GPU runs the
canonical asynchronous 1F1B events up to B_K, the first backward after the
first update, at the full shapes and in the same launch configuration as the
benchmark. Checked against what the oracle computes from single sequences
(sequences of a micro-batch are independent, and by causality a prefix of a
sequence depends on that prefix only):

* F_0: outputs of the first and the last sequence (prefix of P tokens), at
  version 0; LAST: the micro-batch loss (all its sequences);
* B_0: the input gradient of sequence 0 at version 0 (full sequence);
* the first update, as a property of the GPU's own state: theta_1, m_1, v_1
  equal AdamW applied to theta_0 and the G the GPU accumulated;
* the G of the last block's output bias after the first window equals the sum
  of every output gradient of that window (MIDDLE and FIRST);
* GPT-2-medium-shaped middle stage (default and windowed weight gradients):
  every G tensor of the last block after the first window, against the oracle
  accumulated sequence by sequence (64 sequences, each a forward through all
  blocks and the last block's backward at version 0); this reaches the weight
  gradient products at their full shapes and split counts;
* B_K: the input gradient of sequence 0 with activations saved at version
  t^F(K) and the parameters of version 1 (the GPU's theta_1): for delay > 0
  this is the stale backward of the method (activations of version 0,
  weights of version 1); on a checkpointed stage the activations are
  recomputed at version 1 as well;
* F_(K+delay): outputs of sequence 0 (prefix) at version 1;
* every version stamp, exactly; every output finite.
"""
import numpy as np
import pytest

from parity import rel_err, to_host, to_torch, tol, unflatten, adamw_np
from oracle import model
from oracle import schedule as osched
from oracle import stage as ostage
from paper_2606_07881_amd import configs, inputs

pytestmark = pytest.mark.gpu

FULL = ["gpt2s_mid_bf16", "gpt2m_mid_bf16", "gpt2m_first_bf16", "gpt2m_last_bf16", "gpt1p3b_pos0_bf16",
        "gpt2m_mid_bf16+ckpt",    # +ckpt: the same workload on an activation-checkpointed stage
        "gpt2m_last_bf16+fused",  # +fused: the last stage with the fused LM head (no logits kept)
        "gpt2m_mid_bf16+window"]  # +window: windowed weight gradients (K + delay activation slots)
EXTRA = {"+ckpt": {"recompute": 1}, "+fused": {"fused_head": 1}, "+window": {"window": 1}}
LAST_BLOCK_G = {"gpt2m_mid_bf16"}   # workloads whose last block's G is compared in full
PREFIX = 256   # tokens of a sequence whose forward is checked where the whole one is not needed


@pytest.fixture(scope="module")
def binding():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    from paper_2606_07881_amd import binding as b
    return b


def seq_cfg(c, S=None):
    s = dict(c)
    s["micro_batch"] = 1
    if S is not None:
        s["seq"] = S
    return s


def seq_input(c, x_mb, b, S=None):
    """Sequence b of a micro-batch's stage input (first S tokens) for the oracle."""
    S = c["seq"] if S is None else S
    if c["kind"] == "first":
        return x_mb[b:b + 1, :S]
    return x_mb.reshape(c["micro_batch"], c["seq"], -1)[b, :S].astype(np.float64)


def seq_rows(c, a, b, S=None):
    """Rows of sequence b (first S tokens) of a [T, d] array."""
    S = c["seq"] if S is None else S
    return a.reshape(c["micro_batch"], c["seq"], -1)[b, :S]


_ORACLE_G = {}


def oracle_last_block_G(c, seed, theta0):
    """G of the last block after the first window (micro-batches 0 .. K-1, all
    at version 0): the sum over their sequences of the last block's parameter
    gradients, each from a forward through every block and the last block's
    backward. Middle stage, no dropout. Cached per workload shape."""
    key = (c["name"].split("+")[0], seed)
    if key in _ORACLE_G:
        return _ORACLE_G[key]
    L, K, mu = c["n_layers"], c["K"], c["micro_batch"]
    cs = seq_cfg(c)
    blocks = [{n: theta0[f"h{l}.{n}"] for n in ostage.BLOCK_PARAMS} for l in range(L)]
    acc = None
    for i in range(K):
        xm = inputs.make_x(c, seed, i)[0]
        dym = inputs.make_dy(c, seed, i)[0]
        for b in range(mu):
            x = seq_input(c, xm, b)
            for l in range(L):
                x, saved = model.block_fwd(x, blocks[l], cs, None)
            _, g = model.block_bwd(seq_rows(c, dym, b).astype(np.float64), saved, blocks[L - 1], cs)
            acc = g if acc is None else {n: acc[n] + g[n] for n in g}
        print(f"  oracle: last block G, micro-batch {i + 1}/{K} accumulated", flush=True)
    _ORACLE_G[key] = acc
    return acc


def oracle_grad_in(c, theta_f, theta_b, x_seq, dy_seq, tgt_seq):
    """Input gradient of one sequence: activations saved at theta_f, backward at theta_b."""
    cs = seq_cfg(c)
    _, saved = ostage.stage_fwd(cs, theta_f, x_seq, tgt_seq)
    gin, _ = ostage.stage_bwd(cs, theta_b, saved, dy_seq, c["K"], ids=x_seq if c["kind"] == "first" else None)
    if c["kind"] == "last":
        gin = gin / c["micro_batch"]   # the loss is the mean over all mu * S tokens of the micro-batch
    return gin


@pytest.mark.timeout(900)   # the oracle's last-block G takes about 100 s of host time
@pytest.mark.parametrize("name", FULL)
def test_fullsize_sampled(binding, name):
    import torch
    c = configs.get(name.split("+")[0], **next((v for k, v in EXTRA.items() if name.endswith(k)), {}))
    K, delay, seed = c["K"], c["delay"], 0
    T, d, mu = c["micro_batch"] * c["seq"], c["d_model"], c["micro_batch"]
    kind = c["kind"]
    ta, tg = tol(c, "act"), tol(c, "grad")
    print(f"{name}: T={T} d={d} K={K} delay={delay}", flush=True)

    # events of the canonical order up to and including B_K
    assert c["M"] > K + delay
    events = []
    for e in osched.canonical_events(c["M"], K, delay):
        events.append(e)
        if e == ("B", K):
            break
    n_mb = 1 + max(i for k, i in events if k == "F")

    params0 = inputs.make_params(c, seed)
    st = binding.Stage(c)
    st.load_params(params0)
    act = st.act_dtype
    x_host, x_dev, dy_dev, tg_host, tg_dev = {}, {}, {}, {}, {}
    for i in range(n_mb):
        if kind == "first":
            x_host[i] = inputs.make_ids(c, seed, i)
            x_dev[i] = to_torch(x_host[i])
        else:
            v, bits = inputs.make_x(c, seed, i)
            x_host[i] = v
            x_dev[i] = to_torch(bits)
        if kind == "last":
            tg_host[i] = inputs.make_targets(c, seed, i)
            tg_dev[i] = to_torch(tg_host[i])
    dy_host = {}
    if kind != "last":
        for i in range(K + 1):
            v, bits = inputs.make_dy(c, seed, i)
            dy_host[i] = v
            dy_dev[i] = to_torch(bits)

    outs, gins, tF, tB = {}, {}, {}, {}
    G1 = theta1 = m1 = v1 = None
    for kd, i in events:
        if kd == "F":
            outs[i] = torch.zeros(1, dtype=torch.float32, device="cuda") if kind == "last" else \
                torch.empty(T, d, dtype=act, device="cuda")
            tF[i] = st.forward(i, x_dev[i], outs[i], tg_dev.get(i))
        elif kd == "B":
            gins[i] = None if kind == "first" else torch.empty(T, d, dtype=act, device="cuda")
            tB[i], due = st.backward(i, dy_dev.get(i), gins[i])
            assert due == ((i + 1) % K == 0)
            if i not in (0, K):
                gins[i] = None        # only B_0 and B_K are compared; free the rest
        else:
            G1 = st.read(binding.GRADS)
            assert st.step() == 1
            theta1 = st.read(binding.PARAMS)
            m1 = st.read(binding.EXP_AVG)
            v1 = st.read(binding.EXP_AVG_SQ)
    st.sync()
    cf, cb, _ = osched.closed_form_stamps(c["M"], K, delay)
    for i in tF:
        assert tF[i] == cf[i], ("t^F", i)
    for i in tB:
        assert tB[i] == cb[i], ("t^B", i)
    assert st.counters()["version"] == 1

    theta0 = {k: v.astype(np.float64) for k, v in params0.items()}
    th1 = unflatten(c, theta1)

    # the first update as a property of the GPU's state
    flat0 = inputs.flat_params(c, params0).astype(np.float64)
    G1d = G1.astype(np.float64)
    off = 0
    worst = 0.0
    for pname, shape, _ in inputs.param_specs(c):
        n = int(np.prod(shape))
        sl = slice(off, off + n)
        ref_t, ref_m, ref_v = adamw_np(flat0[sl], G1d[sl], np.zeros(n), np.zeros(n), 1, c, ostage.decayed(pname))
        for got, ref in ((theta1[sl], ref_t), (m1[sl], ref_m), (v1[sl], ref_v)):
            e = rel_err(got, ref)
            worst = max(worst, e)
            assert e <= 1e-5, (pname, e)
        off += n
    print(f"{name}: AdamW step 1 property {worst:.2e}", flush=True)
    assert np.all(np.isfinite(G1))

    # G of the last block's output bias: the sum of the window's output gradients
    if kind != "last":
        L = c["n_layers"]
        Gd = unflatten(c, G1)
        ref = sum(dy_host[i].astype(np.float64).sum(0) for i in range(K))
        e = rel_err(Gd[f"h{L - 1}.b_2"], ref)
        print(f"{name}: G b_2 of the last block {e:.2e}", flush=True)
        assert e <= 1e-4

    # every G tensor of the last block against the oracle
    if name.split("+")[0] in LAST_BLOCK_G and not c.get("recompute"):
        L = c["n_layers"]
        ref = oracle_last_block_G(c, seed, theta0)
        Gd = unflatten(c, G1)
        for n, r in ref.items():
            e = rel_err(Gd[f"h{L - 1}.{n}"], r)
            print(f"{name}: G h{L - 1}.{n} after the first window {e:.2e}", flush=True)
            assert e <= tg, n

    # F_0 at version 0
    out0 = to_host(outs[0])
    assert np.all(np.isfinite(out0))
    if kind == "last":
        ref = np.mean([ostage.stage_fwd(seq_cfg(c), theta0, seq_input(c, x_host[0], b), tg_host[0][b:b + 1])[0]
                       for b in range(mu)])
        e = rel_err(np.atleast_1d(out0[0]), np.atleast_1d(ref))
        print(f"{name}: loss of micro-batch 0 {out0[0]:.6f} vs {ref:.6f} ({e:.2e})", flush=True)
        assert e <= ta
    else:
        for b in (0, mu - 1):
            ref, _ = ostage.stage_fwd(seq_cfg(c, PREFIX), theta0, seq_input(c, x_host[0], b, PREFIX))
            e = rel_err(seq_rows(c, out0, b, PREFIX), ref)
            print(f"{name}: F_0 sequence {b} prefix {e:.2e}", flush=True)
            assert e <= ta

    # B_0 at version 0, and B_K with saved activations of version t^F(K) and parameters of version 1
    versions = {0: theta0, 1: th1}
    for i in (0, K):
        if kind == "first":
            continue    # no input gradient
        gin = to_host(gins[i])
        assert np.all(np.isfinite(gin))
        t_act = tB[i] if c.get("recompute") else tF[i]   # the version the activations are from
        ref = oracle_grad_in(c, versions[t_act], versions[tB[i]], seq_input(c, x_host[i], 0),
                             None if kind == "last" else seq_rows(c, dy_host[i], 0).astype(np.float64),
                             tg_host[i][0:1] if kind == "last" else None)
        e = rel_err(seq_rows(c, gin, 0), ref)
        print(f"{name}: B_{i} (t^F={tF[i]}, t^B={tB[i]}) grad_in sequence 0 {e:.2e}", flush=True)
        assert e <= tg
        if tB[i] > tF[i] and not c.get("recompute"):
            # Eq. (1) against weight stashing: the same saved activations
            # differentiated at the forward's parameters. One update moves the
            # weights by about lr along sign(G), which changes this input
            # gradient by about 10 tolerances at the GPT-2-medium shapes; the
            # GPU's result must lie at least 3 tolerances from the stash result
            # and at least 3 times farther from it than from Eq. (1)'s.
            stash = oracle_grad_in(c, versions[tF[i]], versions[tF[i]], seq_input(c, x_host[i], 0),
                                   None if kind == "last" else seq_rows(c, dy_host[i], 0).astype(np.float64),
                                   tg_host[i][0:1] if kind == "last" else None)
            e_st = rel_err(seq_rows(c, gin, 0), stash)
            print(f"{name}: B_{i} distance from weight stashing {e_st:.2e} ({e_st / max(e, 1e-30):.1f}x the "
                  f"distance from Eq. (1))", flush=True)
            assert e_st >= 3.0 * tg and e_st >= 3.0 * e

    # the last forward, at version 1
    j = max(i for k, i in events if k == "F")
    assert tF[j] == 1
    outj = to_host(outs[j])
    assert np.all(np.isfinite(outj))
    if kind != "last":
        ref, _ = ostage.stage_fwd(seq_cfg(c, PREFIX), th1, seq_input(c, x_host[j], 0, PREFIX))
        e = rel_err(seq_rows(c, outj, 0, PREFIX), ref)
        print(f"{name}: F_{j} (version 1) sequence 0 prefix {e:.2e}", flush=True)
        assert e <= ta
    st.close()
