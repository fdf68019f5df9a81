"""Seeded synthetic inputs shared by the tests, the benchmark and the oracle checks.

This module holds no arithmetic of the method. It draws the initial parameters
and the per-micro-batch stage inputs, output gradients, token ids and targets
from counter-keyed PCG64 streams, so that micro-batch i can be generated on its
own and both sides of a parity check see identical bits.

Recipe (the paper's GPT-2 Medium pretraining on OpenWebText is replaced by
synthetic data with these distributions):
  weights and embeddings ~ N(0, 0.02^2), biases 0, LayerNorm gamma 1, beta 0;
  stage input activations ~ N(0, 1); output gradients ~ N(0, 0.01^2);
  token ids and targets i.i.d. uniform on [0, vocab).
Normals are drawn in float32. For bf16 stages the activations and gradients
are rounded to bf16 (round to nearest even) before use, and both sides consume
the rounded values.

Streams: key (seed, stream, index) with stream 0 = parameters, 1 = stage inputs,
2 = output gradients, 3 = token ids, 4 = targets, and index = micro-batch.
"""
import numpy as np

STREAM_PARAMS, STREAM_X, STREAM_DY, STREAM_IDS, STREAM_TGT = range(5)


def rng(seed, stream, index=0):
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, stream, index])))


def bf16_bits(a):
    """Round float32 values to bf16 (nearest, ties to even); return uint16 bits."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    r = ((u >> 16) & 1) + np.uint32(0x7FFF)
    return ((u + r) >> 16).astype(np.uint16)


def bf16_to_f32(bits):
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def bf16_round(a):
    return bf16_to_f32(bf16_bits(a))


def param_specs(c):
    """Ordered (name, shape, init) of the stage parameters (init: normal/zeros/ones)."""
    d, f, V, P = c["d_model"], c["d_ff"], c.get("vocab", 0), c.get("max_pos", 0)
    out = []
    if c["kind"] == "first":
        out += [("wte", (V, d), "normal"), ("wpe", (P, d), "normal")]
    for l in range(c["n_layers"]):
        out += [(f"h{l}.ln1_g", (d,), "ones"), (f"h{l}.ln1_b", (d,), "zeros"),
                (f"h{l}.w_qkv", (3 * d, d), "normal"), (f"h{l}.b_qkv", (3 * d,), "zeros"),
                (f"h{l}.w_o", (d, d), "normal"), (f"h{l}.b_o", (d,), "zeros"),
                (f"h{l}.ln2_g", (d,), "ones"), (f"h{l}.ln2_b", (d,), "zeros"),
                (f"h{l}.w_1", (f, d), "normal"), (f"h{l}.b_1", (f,), "zeros"),
                (f"h{l}.w_2", (d, f), "normal"), (f"h{l}.b_2", (d,), "zeros")]
    if c["kind"] == "last":
        out += [("lnf_g", (d,), "ones"), ("lnf_b", (d,), "zeros"), ("w_lm", (V, d), "normal")]
    return out


def make_params(c, seed=0, std=0.02):
    """Initial parameters as float32 arrays, drawn in canonical order from one stream."""
    g = rng(seed, STREAM_PARAMS)
    out = {}
    for name, shape, init in param_specs(c):
        if init == "normal":
            out[name] = (g.standard_normal(shape, dtype=np.float32) * np.float32(std)).astype(np.float32)
        elif init == "ones":
            out[name] = np.ones(shape, np.float32)
        else:
            out[name] = np.zeros(shape, np.float32)
    return out


def flat_params(c, params):
    return np.concatenate([params[n].reshape(-1) for n, _, _ in param_specs(c)]).astype(np.float32)


def _normal(c, seed, stream, i, std):
    T, d = c["micro_batch"] * c["seq"], c["d_model"]
    a = rng(seed, stream, i).standard_normal((T, d), dtype=np.float32)
    if std != 1.0:
        a *= np.float32(std)
    return a


def make_x(c, seed, i):
    """Stage input of micro-batch i: N(0, 1), [T, d]. Returns (values f32, device bits).

    device bits are uint16 bf16 for bf16 stages, the float32 array otherwise.
    """
    a = _normal(c, seed, STREAM_X, i, 1.0)
    if c["dtype"] == "bf16":
        b = bf16_bits(a)
        return bf16_to_f32(b), b
    return a, a


def make_dy(c, seed, i):
    """Output gradient of micro-batch i: N(0, 0.01^2), [T, d]; same return convention."""
    a = _normal(c, seed, STREAM_DY, i, 1e-2)
    if c["dtype"] == "bf16":
        b = bf16_bits(a)
        return bf16_to_f32(b), b
    return a, a


def make_ids(c, seed, i):
    return rng(seed, STREAM_IDS, i).integers(0, c["vocab"], size=(c["micro_batch"], c["seq"]),
                                             dtype=np.int32)


def make_targets(c, seed, i):
    return rng(seed, STREAM_TGT, i).integers(0, c["vocab"], size=(c["micro_batch"], c["seq"]),
                                             dtype=np.int32)
