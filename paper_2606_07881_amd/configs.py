"""Stage workloads, named by what they are.

Each entry describes one pipeline stage: its kind (middle, first or last stage
of the pipeline), block shapes, micro-batch size, accumulation factor K, delay
(micro-batches in flight = downstream depth N - i of the paper), number of
micro-batches M in one replay, arithmetic dtype and AdamW settings.

The paper trains GPT-2 Medium (24 blocks, d 1024, 16 heads, seq 1024) split over
8 stages with BF16 and AdamW (betas 0.9/0.95, eps 1e-8, weight decay 0.1); the
stage workloads below use its block shapes and optimizer, with a constant
learning rate of 1e-3 and no dropout.
"""
import copy

_ADAMW = dict(lr=1e-3, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1, ln_eps=1e-5)


def _cfg(name, kind, L, d, h, dh, f, S, mu, K, delay, M, dtype, vocab=0, max_pos=0):
    assert d == h * dh
    c = dict(name=name, kind=kind, n_layers=L, d_model=d, n_heads=h, head_dim=dh, d_ff=f,
             seq=S, micro_batch=mu, vocab=vocab, max_pos=max_pos, K=K, delay=delay, M=M,
             dtype=dtype)
    c.update(_ADAMW)
    return c


CONFIGS = {
    # 2 blocks, d 128, 4x32 heads, FFN 512, seq 64, micro-batch 4; stage 0 of 4.
    "tiny_fp32": _cfg("tiny_fp32", "middle", 2, 128, 4, 32, 512, 64, 4, 4, 3, 16, "fp32"),
    # GPT-2-small-shaped middle stage: 3 blocks, d 768, 12x64, FFN 3072, seq 1024.
    "gpt2s_mid_bf16": _cfg("gpt2s_mid_bf16", "middle", 3, 768, 12, 64, 3072, 1024, 8, 8, 3, 64, "bf16"),
    # GPT-2-medium-shaped middle stage: 6 blocks, d 1024, 16x64, FFN 4096, seq 1024.
    "gpt2m_mid_bf16": _cfg("gpt2m_mid_bf16", "middle", 6, 1024, 16, 64, 4096, 1024, 8, 8, 3, 64, "bf16"),
    # First and last stage of a 4-stage GPT-2-medium-shaped pipeline.
    "gpt2m_first_bf16": _cfg("gpt2m_first_bf16", "first", 6, 1024, 16, 64, 4096, 1024, 8, 8, 3, 64,
                             "bf16", vocab=50257, max_pos=1024),
    "gpt2m_last_bf16": _cfg("gpt2m_last_bf16", "last", 6, 1024, 16, 64, 4096, 1024, 8, 8, 0, 64,
                            "bf16", vocab=50257, max_pos=1024),
    # 1.3B-class stage at position 0 of 8: 3 blocks, d 2048, 16x128, FFN 8192, seq 2048.
    "gpt1p3b_pos0_bf16": _cfg("gpt1p3b_pos0_bf16", "middle", 3, 2048, 16, 128, 8192, 2048, 4, 16, 7,
                              128, "bf16"),
}

# The workload the benchmark times: the GPT-2-medium-shaped bf16 middle stage.
BENCH_CONFIG = "gpt2m_mid_bf16"


def get(name, **overrides):
    c = copy.deepcopy(CONFIGS[name])
    c.update(overrides)
    if "name" not in overrides:
        c["name"] = name if not overrides else name + "+" + ",".join(f"{k}={v}" for k, v in overrides.items())
    return c


def tokens_per_microbatch(c):
    return c["micro_batch"] * c["seq"]


def algorithmic_flop_per_microbatch(c):
    """Forward + backward FLOP of one micro-batch through the stage.

    Per block the four linear layers cost 2*T*(4 d^2 + 2 d f) forward and twice
    that backward. Causal attention costs 2*T*S*d forward (QK^T and PV over the
    keys at or before each query: half of the dense 4*T*S*d) and 4*T*S*d
    backward (dV, dP, dQ, dK), recomputation not counted. The last stage adds
    the LM head, 6*T*d*V.
    """
    T, d, f, S, L = tokens_per_microbatch(c), c["d_model"], c["d_ff"], c["seq"], c["n_layers"]
    gemm = 6 * T * (4 * d * d + 2 * d * f)
    attn = 6 * T * S * d
    total = L * (gemm + attn)
    if c["kind"] == "last":
        total += 6 * T * d * c["vocab"]
    return total
