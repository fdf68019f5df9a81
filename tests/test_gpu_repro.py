"""Two-run reproducibility at the full workload sizes: a race check.

Every floating-point atomic of the library adds into the gradient arena G
(split-K weight gradients, bias and LayerNorm column sums, the column sums
fused into GEMM and attention epilogues, the embedding scatter-add). Nothing
else reads G before the first update, so up to that update every other result
is a fixed-order computation: the forwards F_0 .. F_(K-1+delay), the input
gradients of B_0 .. B_(K-1) and the last stage's losses must come out bit for
bit the same when the same inputs go through two fresh stages. A missing
barrier, an LDS hazard or a read of memory another workgroup is still writing
shows up here as a difference. G itself is compared to the rounding that a
different order of fp32 additions allows.
"""
import numpy as np
import pytest

from parity import rel_err, to_torch, unflatten
from oracle import schedule as osched
from paper_2606_07881_amd import configs, inputs

pytestmark = pytest.mark.gpu

CASES = ["gpt2m_mid_bf16", "gpt2m_first_bf16", "gpt2m_last_bf16", "gpt2m_last_bf16+fused",
         "gpt2m_mid_bf16+ckpt+drop", "gpt1p3b_pos0_bf16"]
EXTRA = {"ckpt": {"recompute": 1}, "fused": {"fused_head": 1}, "drop": {"dropout": 0.1, "dropout_seed": 7}}
G_TOL = 1e-5   # relative to a tensor's largest |G|; fp32 sums in another order differ by a few ulps


@pytest.fixture(scope="module")
def binding():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    from paper_2606_07881_amd import binding as b
    return b


def first_window(binding, c, params, x_dev, dy_dev, tg_dev):
    """Runs the canonical events up to the first update on a fresh stage; returns
    the forward outputs, the input gradients and G read before the update."""
    import torch
    T, d, K, kind = c["micro_batch"] * c["seq"], c["d_model"], c["K"], c["kind"]
    st = binding.Stage(c)
    st.load_params(params)
    outs, gins = {}, {}
    for kd, i in osched.canonical_events(c["M"], K, c["delay"]):
        if kd == "F":
            outs[i] = torch.zeros(1, dtype=torch.float32, device="cuda") if kind == "last" else \
                torch.empty(T, d, dtype=st.act_dtype, device="cuda")
            assert st.forward(i, x_dev[i], outs[i], tg_dev.get(i)) == 0
        elif kd == "B":
            gins[i] = None if kind == "first" else torch.empty(T, d, dtype=st.act_dtype, device="cuda")
            st.backward(i, dy_dev.get(i), gins[i])
        else:
            G = st.read(binding.GRADS)
            break
    st.sync()
    st.close()
    return outs, gins, G


@pytest.mark.parametrize("name", CASES)
def test_two_runs_identical(binding, name):
    import torch
    base, *flags = name.split("+")
    over = {}
    for f in flags:
        over.update(EXTRA[f])
    c = configs.get(base, **over)
    K, delay, seed, kind = c["K"], c["delay"], 0, c["kind"]
    print(f"{name}: T={c['micro_batch'] * c['seq']} d={c['d_model']} K={K} delay={delay}", flush=True)
    params = inputs.make_params(c, seed)
    n_mb = K + delay
    x_dev, dy_dev, tg_dev = {}, {}, {}
    for i in range(n_mb):
        x_dev[i] = to_torch(inputs.make_ids(c, seed, i)) if kind == "first" else to_torch(inputs.make_x(c, seed, i)[1])
        if kind == "last":
            tg_dev[i] = to_torch(inputs.make_targets(c, seed, i))
        elif i < K:
            dy_dev[i] = to_torch(inputs.make_dy(c, seed, i)[1])

    outs_a, gins_a, G_a = first_window(binding, c, params, x_dev, dy_dev, tg_dev)
    outs_b, gins_b, G_b = first_window(binding, c, params, x_dev, dy_dev, tg_dev)

    assert sorted(outs_a) == list(range(n_mb))
    for i in outs_a:
        assert torch.isfinite(outs_a[i]).all(), ("F", i)
        assert torch.equal(outs_a[i].view(torch.uint8), outs_b[i].view(torch.uint8)), ("F", i)
    for i in gins_a:
        if gins_a[i] is not None:
            assert torch.equal(gins_a[i].view(torch.uint8), gins_b[i].view(torch.uint8)), ("B", i)
    print(f"{name}: {len(outs_a)} forwards and {len(gins_a)} backwards bit-identical", flush=True)

    assert np.all(np.isfinite(G_a))
    ga, gb = unflatten(c, G_a), unflatten(c, G_b)
    worst = max(rel_err(gb[k], ga[k]) for k in ga)
    n_equal = int(np.count_nonzero(G_a.view(np.uint32) == G_b.view(np.uint32)))
    print(f"{name}: G worst relative difference {worst:.2e}, {n_equal / G_a.size:.1%} of entries equal", flush=True)
    assert worst <= G_TOL
