"""The C-ABI library on the host: it loads, exports every declared symbol, and its
host-only parts (schedule, protocol object, parameter table, arena sizing)
agree with the oracle bit for bit. No device work is issued."""
import ctypes
import itertools

import numpy as np
import pytest

from oracle import schedule as osched
from oracle import stage as ostage
from paper_2606_07881_amd import configs, inputs

binding = pytest.importorskip("paper_2606_07881_amd.binding",
                              reason="libpaci_stage.so not built (python -m paper_2606_07881_amd.build)")


def test_every_declared_symbol_is_exported():
    names = binding.header_symbols()
    assert "paci_stage_init" in names and "paci_stage_run" in names and "paci_fsm_step" in names
    missing = [n for n in names if not hasattr(binding.lib, n)]
    assert not missing, missing
    assert len(names) >= 25


def test_status_strings():
    for code in [0, 1] + list(range(-1, -10, -1)):
        assert binding.strerror(code) != "unknown status"


@pytest.mark.parametrize("M,K,delay", [(16, 4, 3), (64, 8, 3), (64, 8, 0), (128, 16, 7), (5, 1, 0),
                                       (7, 3, 9), (0, 1, 0), (1, 2, 0), (13, 5, 2)])
def test_schedule_matches_oracle(M, K, delay):
    kinds, idx = binding.schedule(M, K, delay)
    ev = osched.canonical_events(M, K, delay)
    lib_ev = [("F", int(i)) if k == 0 else ("B", int(i)) if k == 1 else ("S", None) for k, i in zip(kinds, idx)]
    assert lib_ev == ev


def test_schedule_rejects_bad_arguments():
    n = ctypes.c_int(0)
    k = np.zeros(4, np.int32)
    p = k.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
    assert binding.lib.paci_schedule(10, 2, 1, p, p, 4, ctypes.byref(n)) == binding.E_INVAL
    assert n.value == 25                       # required capacity still reported
    assert binding.lib.paci_schedule(10, 0, 1, p, p, 100, ctypes.byref(n)) == binding.E_INVAL
    assert binding.lib.paci_schedule(-1, 1, 1, p, p, 100, ctypes.byref(n)) == binding.E_INVAL


def _drive(events, K, delay):
    f = binding.Fsm(K, delay)
    tF, tB = {}, {}
    for kind, i in events:
        if kind == "F":
            r, v = f.forward(i)
            assert r == 0
            tF[i] = v
        elif kind == "B":
            r, v = f.backward(i)
            assert r in (0, 1)
            assert (r == 1) == (len(tB) % K == K - 1)
            tB[i] = v
        else:
            r, v = f.step()
            assert r == 0
    M = len(tF)
    return [tF[i] for i in range(M)], [tB[i] for i in range(M)], f.counters()


@pytest.mark.parametrize("M,K,delay", [(16, 4, 3), (64, 8, 3), (64, 8, 0), (128, 16, 7), (12, 5, 4)])
def test_protocol_stamps_bit_exact_vs_oracle(M, K, delay):
    ev = osched.canonical_events(M, K, delay)
    tF, tB, c = _drive(ev, K, delay)
    oF, oB, _, n_upd = osched.run_events(ev, K, delay)
    assert tF == oF and tB == oB
    assert c["version"] == n_upd == M // K
    assert sum(b - f for f, b in zip(tF, tB)) == sum(b - f for f, b in zip(oF, oB))


def test_protocol_on_every_admissible_interleaving():
    # every order Alg. 1 admits for M = 7, K = 2, delay = 2 gives the oracle's stamps
    n = 0
    for ev in osched.all_admissible_orders(7, 2, 2):
        tF, tB, _ = _drive(ev, 2, 2)
        oF, oB, _, _ = osched.run_events(ev, 2, 2)
        assert (tF, tB) == (oF, oB)
        assert max(b - f for f, b in zip(tF, tB)) <= osched.delta_bound(2, 2)
        n += 1
    assert n > 100


def test_protocol_errors_match_oracle():
    """Random event streams: the library refuses exactly what the oracle refuses,
    with the matching code, and a refused event changes nothing."""
    rng = np.random.default_rng(0)
    codes = {"update pending": binding.E_STEP_PENDING, "forward out of order": binding.E_ORDER,
             "backpressure": binding.E_BACKPRESSURE, "backward out of order": binding.E_ORDER,
             "update not due": binding.E_NOT_DUE}
    for K, delay in itertools.product([1, 2, 3], [0, 1, 3]):
        f = binding.Fsm(K, delay)
        o = osched.StageCounters(K, delay)
        for _ in range(300):
            kind = rng.integers(3)
            mb = int(o.next_f if kind == 0 else o.next_b) + int(rng.integers(-1, 2)) * (rng.random() < 0.2)
            before = f.counters()
            try:
                if kind == 0:
                    want = o.forward(mb)
                elif kind == 1:
                    want = o.backward(mb)
                else:
                    want = o.step()
                err = None
            except osched.ProtocolError as e:
                err = codes[str(e)]
            if kind == 0:
                r, v = f.forward(mb)
            elif kind == 1:
                r, v = f.backward(mb)
            else:
                r, v = f.step()
            if err is None:
                assert r >= 0 and v == want
            else:
                assert r == err
                assert f.counters() == before
            c = f.counters()
            assert (c["version"], c["c"], c["q"], c["next_f"], c["next_b"]) == (o.t, o.c, o.q, o.next_f, o.next_b)


@pytest.mark.parametrize("name", list(configs.CONFIGS))
def test_parameter_table_matches_canonical_order(name):
    c = configs.get(name)
    table = binding.param_table(c)
    specs = inputs.param_specs(c)
    assert [t["name"] for t in table] == [n for n, _, _ in specs]
    off = 0
    for t, (n, shape, _) in zip(table, specs):
        assert t["offset"] == off and t["numel"] == int(np.prod(shape))
        assert t["decay"] == ostage.decayed(n)
        off += t["numel"]


def test_arena_sizes_and_shape_validation():
    c = configs.get("gpt2m_mid_bf16")
    b = binding.arena_bytes(c)
    P = sum(int(np.prod(s)) for _, s, _ in inputs.param_specs(c))
    # fp32 theta, G, m, v + bf16 copy + (delay+1) activation slots
    assert b > 18 * P + 4 * 8192 * 1024 * 2 * 6 * 8
    assert b < 64 * 2 ** 30
    bad = [dict(d_model=1000), dict(head_dim=48, n_heads=4, d_model=192), dict(kind="middle", dtype="fp32",
                                                                               head_dim=128, n_heads=8,
                                                                               d_model=1024)]
    expect = [binding.E_INVAL, binding.E_UNSUPPORTED, binding.E_UNSUPPORTED]
    for over, code in zip(bad, expect):
        cc = configs.get("gpt2m_mid_bf16", **over)
        s = binding.shapes(cc)
        out = ctypes.c_size_t(0)
        assert binding.lib.paci_stage_arena_bytes(ctypes.byref(s), 8, 3, ctypes.byref(out)) == code
    s = binding.shapes(c)
    out = ctypes.c_size_t(0)
    assert binding.lib.paci_stage_arena_bytes(ctypes.byref(s), 0, 3, ctypes.byref(out)) == binding.E_INVAL
    assert binding.lib.paci_stage_arena_bytes(ctypes.byref(s), 8, -1, ctypes.byref(out)) == binding.E_INVAL
    first = configs.get("gpt2m_first_bf16", seq=2048)
    s = binding.shapes(first)
    assert binding.lib.paci_stage_arena_bytes(ctypes.byref(s), 8, 3, ctypes.byref(out)) == binding.E_INVAL


def test_init_refuses_bad_arguments_without_device_work():
    c = configs.get("tiny_fp32")
    s = binding.shapes(c)
    h = ctypes.c_void_p()
    # null arena, misaligned arena, arena too small: all refused before any HIP call
    assert binding.lib.paci_stage_init(ctypes.byref(s), 4, 3, None, 1 << 20, None, ctypes.byref(h)) == binding.E_INVAL
    assert binding.lib.paci_stage_init(ctypes.byref(s), 4, 3, ctypes.c_void_p(0x1001), 1 << 20, None,
                                       ctypes.byref(h)) == binding.E_INVAL
    assert binding.lib.paci_stage_init(ctypes.byref(s), 4, 3, ctypes.c_void_p(0x100000), 16, None,
                                       ctypes.byref(h)) == binding.E_NOMEM


@pytest.mark.parametrize("M,K,delay", [(16, 4, 3), (64, 8, 3), (64, 8, 0), (128, 16, 7), (5, 1, 0),
                                       (7, 3, 9), (0, 1, 0), (1, 2, 0), (13, 5, 2)])
def test_flush_schedule_matches_oracle(M, K, delay):
    kinds, idx = binding.schedule(M, K, delay, flush=True)
    ev = osched.flush_events(M, K, delay)
    lib_ev = [("F", int(i)) if k == 0 else ("B", int(i)) if k == 1 else ("S", None) for k, i in zip(kinds, idx)]
    assert lib_ev == ev
    n = ctypes.c_int(0)
    k = np.zeros(1, np.int32)
    p = k.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
    if len(ev) > 1:
        assert binding.lib.paci_schedule_flush(M, K, delay, p, p, 1, ctypes.byref(n)) == binding.E_INVAL
        assert n.value == len(ev)
    assert binding.lib.paci_schedule_flush(M, 0, delay, p, p, 1, ctypes.byref(n)) == binding.E_INVAL


def test_fused_head_validation_and_memory():
    """The fused LM head keeps no [T, V] logits: the GPT-2-medium-shaped last
    stage's arena shrinks by the fp32 logits of every slot; it is refused off
    a bf16 last stage and for a stage with delay > 0."""
    out = ctypes.c_size_t(0)
    c = configs.get("gpt2m_last_bf16")
    s = binding.shapes(c)
    assert binding.lib.paci_stage_arena_bytes(ctypes.byref(s), c["K"], c["delay"], ctypes.byref(out)) == 0
    plain = out.value
    s = binding.shapes(dict(c, fused_head=1))
    assert binding.lib.paci_stage_arena_bytes(ctypes.byref(s), c["K"], c["delay"], ctypes.byref(out)) == 0
    fused = out.value
    T, ldz = c["micro_batch"] * c["seq"], (c["vocab"] + 63) // 64 * 64
    slots = c["delay"] + 1             # the default store: the micro-batches in flight
    partials = 8 * T * (ldz // 64) + 4 * T
    assert plain - fused >= slots * 4 * T * ldz - partials - 4096
    assert plain - fused <= slots * 4 * T * ldz
    for over, code in [(dict(kind="middle"), binding.E_UNSUPPORTED), (dict(dtype="fp32"), binding.E_UNSUPPORTED),
                       (dict(fused_head=2), binding.E_INVAL)]:
        s = binding.shapes(dict(dict(c, fused_head=1), **over))
        s.fused_head = over.get("fused_head", 1)
        assert binding.lib.paci_stage_arena_bytes(ctypes.byref(s), 8, 0, ctypes.byref(out)) == code
    s = binding.shapes(dict(c, fused_head=1))
    assert binding.lib.paci_stage_arena_bytes(ctypes.byref(s), 8, 1, ctypes.byref(out)) == binding.E_INVAL


def test_static_backward_rejects_a_stage_beyond_its_scratch():
    """paci_stage_backward_static: the attention scratch of a stage must fit the
    library's 8 MiB static buffer; the host-side size check refuses larger ones
    before any device work (a null handle is refused first)."""
    v = ctypes.c_int(-1)
    assert binding.lib.paci_stage_backward_static(None, 0, None, None, ctypes.byref(v)) == binding.E_INVAL
    assert binding.strerror(binding.E_SCRATCH) != "unknown status"
