"""float64 forward/backward of the stage function F_i (test infrastructure).

The paper trains GPT-2 Medium (Sec. 4.1, "Experimental setup"); a stage F_i is a
contiguous run of pre-LN decoder blocks, optionally preceded by the token and
position embeddings (first stage) or followed by the final LayerNorm, the LM
head and the cross-entropy loss (last stage). The paper names no kernels, so
each op here is its textbook definition:

* LayerNorm: biased variance over the feature axis, eps inside the square root,
  affine gamma/beta.
* GELU: the tanh approximation used by GPT-2.
* attention: softmax(q k^T / sqrt(dh)) v with keys restricted to positions at
  or before the query (causal), per sequence and head.
* linear layers follow nn.Linear: weight [out, in], y = x W^T + b.

Backward functions take the *saved* activations of the forward and the
parameters to differentiate at as separate arguments, because under Eq. (1) of
Sec. 3.1 the two may come from different parameter versions (the parameters
are the ones current when the backward runs, see the appendix "PyTorch
modifications for asynchronous execution").

Arrays are float64 numpy arrays. Activations are 2-D [T, d] with the T = mu*S
tokens of a micro-batch in sequence-major order (token t = b*S + s).
"""
import math

import numpy as np


# ----------------------------------------------------------------------------
# LayerNorm
# ----------------------------------------------------------------------------
def layernorm_fwd(x, gamma, beta, eps):
    """n = (x - mean) * rstd * gamma + beta over the last axis (biased variance).

    Returns (n, mean, rstd) with mean and rstd of shape [T].
    """
    mean = x.mean(axis=-1)
    xc = x - mean[:, None]
    var = (xc * xc).mean(axis=-1)
    rstd = 1.0 / np.sqrt(var + eps)
    xhat = xc * rstd[:, None]
    return xhat * gamma[None, :] + beta[None, :], mean, rstd


def layernorm_bwd(dn, x, mean, rstd, gamma):
    """Backward of layernorm_fwd at the given gamma.

    xhat is rebuilt from the saved input and statistics (it holds no
    parameter). With g = dn * gamma, the input gradient is
        dx = rstd * (g - mean(g) - xhat * mean(g * xhat)),
    and the affine gradients are dgamma = sum_t dn * xhat, dbeta = sum_t dn.
    """
    xhat = (x - mean[:, None]) * rstd[:, None]
    g = dn * gamma[None, :]
    dx = rstd[:, None] * (g - g.mean(axis=-1, keepdims=True)
                          - xhat * (g * xhat).mean(axis=-1, keepdims=True))
    return dx, (dn * xhat).sum(axis=0), dn.sum(axis=0)


# ----------------------------------------------------------------------------
# GELU (tanh form)
# ----------------------------------------------------------------------------
_GELU_C = math.sqrt(2.0 / math.pi)
_GELU_A = 0.044715


def gelu(u):
    """0.5 u (1 + tanh(sqrt(2/pi) (u + 0.044715 u^3)))."""
    return 0.5 * u * (1.0 + np.tanh(_GELU_C * (u + _GELU_A * u ** 3)))


def gelu_grad(u):
    """d gelu / du, the derivative of the expression in gelu()."""
    th = np.tanh(_GELU_C * (u + _GELU_A * u ** 3))
    return 0.5 * (1.0 + th) + 0.5 * u * (1.0 - th * th) * _GELU_C * (1.0 + 3.0 * _GELU_A * u * u)


# ----------------------------------------------------------------------------
# causal attention
# ----------------------------------------------------------------------------
def _heads(qkv, mu, S, n_heads, head_dim):
    """Split the fused [T, 3d] projection into q, k, v of shape [mu, H, S, dh].

    Columns [0, d) hold q, [d, 2d) hold k and [2d, 3d) hold v; head h owns
    columns h*dh .. (h+1)*dh - 1 of each.
    """
    d = n_heads * head_dim
    parts = []
    for j in range(3):
        m = qkv[:, j * d:(j + 1) * d].reshape(mu, S, n_heads, head_dim)
        parts.append(m.transpose(0, 2, 1, 3))
    return parts


def _merge(o):
    """[mu, H, S, dh] -> [T, H*dh] (inverse of the head split)."""
    mu, H, S, dh = o.shape
    return o.transpose(0, 2, 1, 3).reshape(mu * S, H * dh)


def attention_fwd(qkv, mu, S, n_heads, head_dim, keep=None, drop_scale=1.0):
    """o = softmax(q k^T / sqrt(dh) + causal mask) v for every sequence and head.

    With ``keep`` [mu, H, S, S] (dropout on the probabilities) the product
    uses P * keep * drop_scale. Returns o as [T, d] and the per-row
    log-sum-exp of the scaled scores, lse [mu, H, S] (of the undropped ones).
    """
    q, k, v = _heads(qkv, mu, S, n_heads, head_dim)
    scale = 1.0 / math.sqrt(head_dim)
    future = np.triu(np.ones((S, S), dtype=bool), k=1)
    o = np.empty_like(q)
    lse = np.empty((mu, n_heads, S))
    for b in range(mu):
        for h in range(n_heads):
            s = (q[b, h] @ k[b, h].T) * scale
            s[future] = -np.inf
            smax = s.max(axis=1, keepdims=True)
            e = np.exp(s - smax)
            rowsum = e.sum(axis=1, keepdims=True)
            P = e / rowsum
            if keep is not None:
                P = P * keep[b, h] * drop_scale
            o[b, h] = P @ v[b, h]
            lse[b, h] = (smax + np.log(rowsum))[:, 0]
    return _merge(o), lse


def attention_bwd(do_, qkv, lse, mu, S, n_heads, head_dim, keep=None, drop_scale=1.0):
    """Backward of attention_fwd; returns d(qkv) as [T, 3d].

    P is rebuilt from q, k and the saved log-sum-exp (it holds no parameter).
    With dP = dO V^T: dV = P^T dO, dS = P * (dP - rowsum(dP * P)),
    dQ = dS K / sqrt(dh), dK = dS^T Q / sqrt(dh). With dropout (``keep``),
    M = keep * drop_scale: dV = (P M)^T dO and dP = (dO V^T) M.
    """
    q, k, v = _heads(qkv, mu, S, n_heads, head_dim)
    d = n_heads * head_dim
    dO = do_.reshape(mu, S, n_heads, head_dim).transpose(0, 2, 1, 3)
    scale = 1.0 / math.sqrt(head_dim)
    future = np.triu(np.ones((S, S), dtype=bool), k=1)
    dq, dk, dv = np.empty_like(q), np.empty_like(k), np.empty_like(v)
    for b in range(mu):
        for h in range(n_heads):
            s = (q[b, h] @ k[b, h].T) * scale
            s[future] = -np.inf
            P = np.exp(s - lse[b, h][:, None])
            Mk = 1.0 if keep is None else keep[b, h] * drop_scale
            dv[b, h] = (P * Mk).T @ dO[b, h]
            dP = (dO[b, h] @ v[b, h].T) * Mk
            dS = P * (dP - (dP * P).sum(axis=1, keepdims=True))
            dq[b, h] = (dS @ k[b, h]) * scale
            dk[b, h] = (dS.T @ q[b, h]) * scale
    out = np.empty((mu * S, 3 * d))
    out[:, 0:d] = _merge(dq)
    out[:, d:2 * d] = _merge(dk)
    out[:, 2 * d:3 * d] = _merge(dv)
    return out


# ----------------------------------------------------------------------------
# one pre-LN decoder block
# ----------------------------------------------------------------------------
def block_fwd(x, p, cfg, drop=None):
    """y = x1 + W2 gelu(W1 LN2(x1) + b1) + b2,  x1 = x + Wo attn(Wqkv LN1(x) + bqkv) + bo.

    ``p`` maps the block's parameter names (ln1_g, ln1_b, w_qkv, b_qkv, w_o,
    b_o, ln2_g, ln2_b, w_1, b_1, w_2, b_2) to arrays. ``drop`` (optional) holds
    the dropout keep masks of this block and micro-batch, {"attn", "proj",
    "ffn"}, and their scale: the attention probabilities and the two branch
    outputs (before their residual adds) are multiplied by keep * scale.
    Returns (y, saved), where ``saved`` holds every activation (and mask) the
    backward reads.
    """
    mu, S, H, dh, eps = cfg["micro_batch"], cfg["seq"], cfg["n_heads"], cfg["head_dim"], cfg["ln_eps"]
    sc = 1.0 if drop is None else drop["scale"]
    n1, mean1, rstd1 = layernorm_fwd(x, p["ln1_g"], p["ln1_b"], eps)
    qkv = n1 @ p["w_qkv"].T + p["b_qkv"]
    o, lse = attention_fwd(qkv, mu, S, H, dh, None if drop is None else drop["attn"], sc)
    z1 = o @ p["w_o"].T + p["b_o"]
    x1 = x + (z1 if drop is None else z1 * drop["proj"] * sc)
    n2, mean2, rstd2 = layernorm_fwd(x1, p["ln2_g"], p["ln2_b"], eps)
    u = n2 @ p["w_1"].T + p["b_1"]
    a = gelu(u)
    z2 = a @ p["w_2"].T + p["b_2"]
    y = x1 + (z2 if drop is None else z2 * drop["ffn"] * sc)
    saved = dict(x=x, mean1=mean1, rstd1=rstd1, n1=n1, qkv=qkv, o=o, lse=lse,
                 x1=x1, mean2=mean2, rstd2=rstd2, n2=n2, u=u, a=a, drop=drop)
    return y, saved


def block_bwd(dy, s, p, cfg):
    """Backward of block_fwd from saved activations ``s`` at parameters ``p``.

    Returns (dx, grads) with grads keyed like the parameters. Weight gradients
    read only saved activations; every parameter that the backward reads (the
    weights of the input-gradient products and the LayerNorm gammas) is taken
    from ``p``.
    """
    mu, S, H, dh = cfg["micro_batch"], cfg["seq"], cfg["n_heads"], cfg["head_dim"]
    drop = s.get("drop")
    g = {}
    # y = x1 + drop(a W2^T + b2): the branch sees dy * keep * scale
    g2 = dy if drop is None else dy * drop["ffn"] * drop["scale"]
    g["w_2"] = g2.T @ s["a"]
    g["b_2"] = g2.sum(axis=0)
    du = (g2 @ p["w_2"]) * gelu_grad(s["u"])
    # u = n2 W1^T + b1
    g["w_1"] = du.T @ s["n2"]
    g["b_1"] = du.sum(axis=0)
    dn2 = du @ p["w_1"]
    dx1_ln, g["ln2_g"], g["ln2_b"] = layernorm_bwd(dn2, s["x1"], s["mean2"], s["rstd2"], p["ln2_g"])
    dx1 = dy + dx1_ln
    # x1 = x + drop(o Wo^T + bo)
    g1 = dx1 if drop is None else dx1 * drop["proj"] * drop["scale"]
    g["w_o"] = g1.T @ s["o"]
    g["b_o"] = g1.sum(axis=0)
    do_ = g1 @ p["w_o"]
    dqkv = attention_bwd(do_, s["qkv"], s["lse"], mu, S, H, dh, None if drop is None else drop["attn"],
                         1.0 if drop is None else drop["scale"])
    # qkv = n1 Wqkv^T + bqkv
    g["w_qkv"] = dqkv.T @ s["n1"]
    g["b_qkv"] = dqkv.sum(axis=0)
    dn1 = dqkv @ p["w_qkv"]
    dx_ln, g["ln1_g"], g["ln1_b"] = layernorm_bwd(dn1, s["x"], s["mean1"], s["rstd1"], p["ln1_g"])
    return dx1 + dx_ln, g


# ----------------------------------------------------------------------------
# first stage: token + learned position embedding
# ----------------------------------------------------------------------------
def embed_fwd(ids, wte, wpe):
    """x[b*S + s] = wte[ids[b, s]] + wpe[s]."""
    mu, S = ids.shape
    return (wte[ids] + wpe[None, :S, :]).reshape(mu * S, wte.shape[1])


def embed_bwd(dx, ids, vocab, max_pos):
    """Gradients of embed_fwd: rows of wte receive the sum over every position
    holding that id (duplicates add); wpe row s receives the sum over sequences."""
    mu, S = ids.shape
    d = dx.shape[1]
    g_wte = np.zeros((vocab, d))
    np.add.at(g_wte, ids.reshape(-1), dx)
    g_wpe = np.zeros((max_pos, d))
    g_wpe[:S] = dx.reshape(mu, S, d).sum(axis=0)
    return g_wte, g_wpe


# ----------------------------------------------------------------------------
# last stage: final LayerNorm, LM head, mean softmax cross-entropy
# ----------------------------------------------------------------------------
def head_fwd(y, targets, lnf_g, lnf_b, w_lm, eps):
    """z = LN_f(y) W_lm^T;  loss = mean_t (logsumexp(z_t) - z_t[target_t]).

    Returns (loss, saved).
    """
    nf, meanf, rstdf = layernorm_fwd(y, lnf_g, lnf_b, eps)
    z = nf @ w_lm.T
    zmax = z.max(axis=1, keepdims=True)
    lse = (zmax + np.log(np.exp(z - zmax).sum(axis=1, keepdims=True)))[:, 0]
    tgt = targets.reshape(-1)
    loss = float(np.mean(lse - z[np.arange(z.shape[0]), tgt]))
    return loss, dict(y=y, meanf=meanf, rstdf=rstdf, nf=nf, z=z, lse=lse, targets=tgt)


def head_bwd(s, lnf_g, w_lm, seed_scale):
    """Backward of head_fwd scaled by ``seed_scale``.

    dz = seed_scale * (softmax(z) - onehot(target)); then the LM-head products
    and the final LayerNorm backward at the given (current) lnf_g and w_lm.
    Returns (dy, g_lnf_g, g_lnf_b, g_w_lm).
    """
    z, tgt = s["z"], s["targets"]
    dz = np.exp(z - s["lse"][:, None])
    dz[np.arange(z.shape[0]), tgt] -= 1.0
    dz *= seed_scale
    g_w_lm = dz.T @ s["nf"]
    dnf = dz @ w_lm
    dy, g_g, g_b = layernorm_bwd(dnf, s["y"], s["meanf"], s["rstdf"], lnf_g)
    return dy, g_g, g_b, g_w_lm
