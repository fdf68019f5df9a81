"""The seeded input generators: determinism, distributions, bf16 rounding and
agreement of the parameter list with the oracle's."""
import numpy as np
import pytest

from oracle import stage
from paper_2606_07881_amd import configs, inputs


@pytest.mark.parametrize("name", list(configs.CONFIGS))
def test_param_list_matches_oracle(name):
    c = configs.get(name)
    a = [(n, tuple(s)) for n, s, _ in inputs.param_specs(c)]
    b = [(n, tuple(s)) for n, s in stage.param_shapes(c)]
    assert a == b


def test_bf16_rounding_is_nearest_even():
    vals = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -2.5, 1e-30, 3.0e38], np.float32)
    bits = inputs.bf16_bits(vals)
    # 1 + 2^-8 is a tie between 1 and 1 + 2^-7: even mantissa (1.0) wins;
    # 1 + 3*2^-8 ties between 1 + 2^-7 and 1 + 2^-6: 1 + 2^-6 (even) wins.
    assert list(inputs.bf16_to_f32(bits)[:4]) == [1.0, 1.0, 1.0 + 2 ** -6, -2.5]
    x = np.random.default_rng(0).standard_normal(10000).astype(np.float32)
    r = inputs.bf16_round(x)
    assert np.all(np.abs(r - x) <= np.abs(x) * 2.0 ** -8)


def test_streams_are_deterministic_and_distinct():
    c = configs.get("tiny_fp32")
    a, _ = inputs.make_x(c, 0, 3)
    b, _ = inputs.make_x(c, 0, 3)
    d, _ = inputs.make_dy(c, 0, 3)
    np.testing.assert_array_equal(a, b)
    assert not np.array_equal(a, inputs.make_x(c, 0, 4)[0])
    assert abs(a.std() - 1.0) < 0.02 and abs(d.std() - 0.01) < 2e-4
    p = inputs.make_params(c, 0)
    assert abs(p["h0.w_qkv"].std() - 0.02) < 1e-3
    assert np.all(p["h1.ln2_g"] == 1) and np.all(p["h1.b_2"] == 0)


def test_bf16_stage_inputs_are_bf16_exact():
    c = configs.get("tiny_fp32", dtype="bf16")
    x, bits = inputs.make_x(c, 1, 0)
    assert bits.dtype == np.uint16
    np.testing.assert_array_equal(inputs.bf16_to_f32(bits), x)
