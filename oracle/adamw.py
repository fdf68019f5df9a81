"""AdamW, float64 (test infrastructure).

The paper trains with AdamW (appendix "Detailed experimental setup",
Optimization and training): beta1 = 0.9, beta2 = 0.95, eps = 1e-8, weight decay
0.1 with no decay on biases, LayerNorm parameters or embeddings. The update is
the decoupled form of Loshchilov and Hutter as implemented by PyTorch's AdamW:
the decay multiplies the parameter first, then the bias-corrected Adam
direction is subtracted, with eps added outside the square root.
"""
import math

import numpy as np


def adamw_update(theta, grad, m, v, step, lr, beta1, beta2, eps, weight_decay):
    """One AdamW update at local step ``step`` (1 for the first update).

    theta <- theta * (1 - lr * weight_decay)
    m     <- beta1 m + (1 - beta1) grad
    v     <- beta2 v + (1 - beta2) grad^2
    theta <- theta - lr * (m / (1 - beta1^step)) / (sqrt(v / (1 - beta2^step)) + eps)

    Returns new (theta, m, v); the inputs are not modified.
    """
    theta = theta * (1.0 - lr * weight_decay)
    m = beta1 * m + (1.0 - beta1) * grad
    v = beta2 * v + (1.0 - beta2) * grad * grad
    mhat = m / (1.0 - beta1 ** step)
    vhat = v / (1.0 - beta2 ** step)
    return theta - lr * mhat / (np.sqrt(vhat) + eps), m, v


def lr_at(cfg, step):
    """Learning rate of update ``step`` (1 for the first update).

    The paper's recipe (appendix "Detailed experimental setup") warms the rate
    up linearly over the first 1% of the updates and then decays it along a
    cosine to 10% of the peak. Read here as: with W = lr_warmup and
    N = lr_total updates (N = 0: the constant rate cfg["lr"]),
      step <= W:  lr * step / W
      step >  W:  lr * (r + (1 - r) * (1 + cos(pi * p)) / 2),
                  p = min(1, (step - W) / (N - W)), r = lr_min_ratio.
    """
    peak = cfg["lr"]
    total = int(cfg.get("lr_total", 0))
    if total <= 0:
        return peak
    warm = int(cfg.get("lr_warmup", 0))
    r = float(cfg.get("lr_min_ratio", 0.1))
    if step <= warm:
        return peak * step / warm
    p = min(1.0, (step - warm) / max(1, total - warm))
    return peak * (r + (1.0 - r) * 0.5 * (1.0 + math.cos(math.pi * p)))


def direction_bound(step, beta1, beta2):
    """Largest |m_hat / sqrt(v_hat)| any gradient sequence can produce at ``step``.

    By Cauchy-Schwarz, |sum_j b1^(t-j) g_j| <= sqrt(sum_j (b1^2/b2)^(t-j))
    * sqrt(sum_j b2^(t-j) g_j^2), so |m_hat| / sqrt(v_hat) <= (1-b1)/(1-b1^t)
    * sqrt((1-b2^t)/(1-b2)) * sqrt(sum_{k<t} (b1^2/b2)^k). Used to state which
    parameter values are valid where the update direction is not determined by
    the gradient within its tolerance.
    """
    r = beta1 * beta1 / beta2
    s = sum(r ** k for k in range(step))
    return (1.0 - beta1) / (1.0 - beta1 ** step) * math.sqrt((1.0 - beta2 ** step) / (1.0 - beta2)) * math.sqrt(s)
