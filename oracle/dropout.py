"""Dropout masks from a counter-based generator (test infrastructure).

The paper trains with dropout 0.1 (appendix "Detailed experimental setup").
GPT-2 applies it at four places, all of them kept here: the embedding sum (first
stage), the attention probabilities, and the outputs of the attention
projection and of the FFN before each residual add. Inverted dropout keeps an
element with probability 1 - p and scales the kept ones by 1 / (1 - p).

Masks must be identical in a forward, in its backward (which may run under a
newer parameter version but uses the same micro-batch) and in a recomputed
forward, so every keep bit is a pure function of (seed, micro-batch, block,
site, element), drawn from Philox4x32-10 (Salmon, Moraes, Dror and Shaw,
"Parallel random numbers: as easy as 1, 2, 3", SC 2011): 10 rounds of two
32 x 32 -> 64-bit multiplications on a 4-word counter with a 2-word key bumped
by the Weyl constants between rounds.

Element -> bits (the GPU derives the same bits from the same definition):
  key            (seed, micro-batch index)
  site word      (block << 2) | site, site 0 embedding, 1 attention, 2 projection, 3 FFN
  element-wise   element e = t * d + j of a [T, d] tensor:
                 counter (e >> 3 mod 2^32, e >> 35, 0, site word); 16-bit value
                 (e & 1) of output word (e >> 1) & 3
  attention      probability (b, h, query q, key k), bh = b * H + h:
                 counter (k >> 2, q >> 1, bh, site word); 16-bit value (k & 1)
                 of output word 2 (q & 1) + ((k >> 1) & 1)
A value v keeps its element when v >= thr, thr = floor(p * 65536 + 1/2) with p
rounded to float32 first.
"""
import math

import numpy as np

M0, M1 = 0xD2511F53, 0xCD9E8D57      # Philox4x32 multipliers
W0, W1 = 0x9E3779B9, 0xBB67AE85      # key increments (Weyl sequence)
MASK32 = np.uint64(0xFFFFFFFF)

SITE_EMBED, SITE_ATTN, SITE_PROJ, SITE_FFN = 0, 1, 2, 3


def philox4x32_10(c0, c1, c2, c3, k0, k1):
    """Philox4x32-10 on arrays of counter words (any broadcastable shapes)."""
    c = [np.asarray(x, dtype=np.uint64) & MASK32 for x in (c0, c1, c2, c3)]
    k0 = np.uint64(k0 & 0xFFFFFFFF)
    k1 = np.uint64(k1 & 0xFFFFFFFF)
    for r in range(10):
        if r:
            k0 = (k0 + np.uint64(W0)) & MASK32
            k1 = (k1 + np.uint64(W1)) & MASK32
        p0 = np.uint64(M0) * c[0]
        p1 = np.uint64(M1) * c[2]
        hi0, lo0 = p0 >> np.uint64(32), p0 & MASK32
        hi1, lo1 = p1 >> np.uint64(32), p1 & MASK32
        c = [hi1 ^ c[1] ^ k0, lo1, hi0 ^ c[3] ^ k1, lo0]
    return c


def threshold(p):
    return int(math.floor(float(np.float32(p)) * 65536.0 + 0.5))


def scale(p):
    return 1.0 / (1.0 - float(np.float32(p)))


def site_word(block, site):
    return (block << 2) | site


def keep_elementwise(seed, mb, block, site, T, d, p):
    """Keep mask [T, d] of an element-wise site."""
    e = np.arange(T * d, dtype=np.uint64)
    words = philox4x32_10(e >> np.uint64(3), e >> np.uint64(35), np.zeros_like(e),
                          np.full_like(e, site_word(block, site)), seed, mb)
    widx = ((e >> np.uint64(1)) & np.uint64(3)).astype(np.int64)
    w = np.choose(widx, words)
    v = (w >> (np.uint64(16) * (e & np.uint64(1)))) & np.uint64(0xFFFF)
    return (v >= threshold(p)).reshape(T, d)


def keep_attention(seed, mb, block, mu, H, S, p):
    """Keep mask [mu, H, S (query), S (key)] of the attention probabilities."""
    q = np.arange(S, dtype=np.uint64)[:, None]
    k = np.arange(S, dtype=np.uint64)[None, :]
    out = np.empty((mu, H, S, S), dtype=bool)
    thr = threshold(p)
    widx = (np.uint64(2) * (q & np.uint64(1)) + ((k >> np.uint64(1)) & np.uint64(1))).astype(np.int64)
    shift = np.uint64(16) * (k & np.uint64(1))
    for b in range(mu):
        for h in range(H):
            words = philox4x32_10(k >> np.uint64(2), q >> np.uint64(1), np.uint64(b * H + h),
                                  np.uint64(site_word(block, SITE_ATTN)), seed, mb)
            words = [np.broadcast_to(w, (S, S)) for w in words]
            w = np.choose(np.broadcast_to(widx, (S, S)), words)
            out[b, h] = ((w >> shift) & np.uint64(0xFFFF)) >= thr
    return out
