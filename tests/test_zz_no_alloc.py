"""paci_stage_backward_static against paci_stage_backward, through the C ABI.

The variant takes the attention backward's (lse2, D) pairs from the library's
static per-GPU scratch instead of the stage arena. Two calls in a row on the
same GPU, the second with a smaller stage (fewer queries, so the static buffer
still holds the first call's larger contents past the second's end): each
must give the input gradient of the arena-backed backward bit for bit (no
atomic sums feed it) and the same accumulated G within the tolerance (the bias
column sums use fp32 atomics), and the stamps and counters must agree.
"""
import numpy as np
import pytest

from parity import Inputs, rel_err, small_cfg, to_host, to_torch, tol, unflatten

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def binding():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    from paper_2606_07881_amd import binding as b
    return b


def _pair(binding, c, seed):
    """One forward and backward of micro-batch 0 on twin stages: arena-backed
    backward on the first, the static variant on the second."""
    import torch
    inp = Inputs(c, seed, 1)
    T, d = c["micro_batch"] * c["seq"], c["d_model"]
    res = []
    for static in (False, True):
        st = binding.Stage(c, K=2, delay=1)
        st.load_params(inp.params)
        out = torch.zeros(T, d, dtype=st.act_dtype, device="cuda")
        assert st.forward(0, to_torch(inp.x_dev[0]), out) == 0
        gin = torch.zeros(T, d, dtype=st.act_dtype, device="cuda")
        fn = st.backward_static if static else st.backward
        v, due = fn(0, to_torch(inp.dy_dev[0]), gin)
        assert v == 0 and not due
        G = unflatten(c, st.read(binding.GRADS))
        st.sync()
        res.append((to_host(gin), G, st.counters()))
        st.close()
    return res


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_static_backward_matches_arena_backward(binding, dtype):
    big = small_cfg("ragged_bf16" if dtype == "bf16" else "ragged_fp32")
    small = dict(big, seq=big["seq"] // 2 + 4, micro_batch=1, name=big["name"] + "_small")
    for c, seed in ((big, 11), (small, 12)):    # the second call has fewer queries
        print(f"static backward: {c['name']} mu={c['micro_batch']} S={c['seq']} H={c['n_heads']}", flush=True)
        (gin_a, G_a, cnt_a), (gin_s, G_s, cnt_s) = _pair(binding, c, seed)
        assert cnt_a == cnt_s
        assert np.array_equal(gin_a, gin_s), "input gradients differ"
        worst = max(rel_err(G_s[n], G_a[n]) for n in G_a)
        print(f"  grad_in bit-identical, worst G difference {worst:.2e}", flush=True)
        assert worst <= tol(c, "grad")


def test_static_backward_refuses_beyond_the_buffer(binding):
    """A stage whose pairs exceed 8 MiB: PACI_E_SCRATCH, counters unchanged."""
    import torch
    c2 = small_cfg("dh32_bf16", micro_batch=64, seq=1024, n_heads=32, head_dim=32, d_model=1024)
    assert 2 * c2["micro_batch"] * c2["n_heads"] * 1024 * 4 == 16 << 20   # pairs: 16 MiB
    st = binding.Stage(c2, K=2, delay=1)
    T, d = c2["micro_batch"] * c2["seq"], c2["d_model"]
    x = torch.zeros(T, d, dtype=st.act_dtype, device="cuda")
    out = torch.zeros_like(x)
    assert st.forward(0, x, out) == 0
    before = st.counters()
    with pytest.raises(binding.PaciError) as ei:
        st.backward_static(0, torch.zeros_like(x), torch.zeros_like(x))
    assert ei.value.code == binding.E_SCRATCH
    assert st.counters() == before
    st.backward(0, torch.zeros_like(x), torch.zeros_like(x))
    st.close()
