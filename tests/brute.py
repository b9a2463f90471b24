"""Brute-force NumPy/SciPy references for tiny inputs (fp64), used to pin the oracle.

These work on the *dense* per-request K arrays the workload generator keeps, so they do not
go through the block table at all, and they use library routines (``numpy.matmul``,
``scipy.special.softmax`` / ``logsumexp``, ``numpy.lexsort``,
``sliding_window_view``) instead of hand-written loops.
"""
import numpy as np
from numpy.lib.stride_tricks import sliding_window_view
from scipy.special import logsumexp, softmax


def f32(bits):
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def attention_probs(q_bits, k_bits, sm_scale, causal):
    """Full attention matrix per query head: P[j, g, t] (fp64), masked entries 0.

    q_bits [n, Hq, D], k_bits [L, Hkv, D] (bf16 bits); query j sits at position L - n + j.
    """
    q = f32(q_bits).astype(np.float64)
    k = f32(k_bits).astype(np.float64)
    n, Hq, D = q.shape
    L, Hkv, _ = k.shape
    G = Hq // Hkv
    P = np.zeros((n, Hq, L))
    for g in range(Hq):
        logits = sm_scale * (q[:, g, :] @ k[:, g // G, :].T)   # [n, L]
        if causal:
            pos = L - n + np.arange(n)
            mask = np.arange(L)[None, :] > pos[:, None]
            logits = np.where(mask, -np.inf, logits)
        P[:, g, :] = softmax(logits, axis=1)
    return P


def lse(q_bits, k_bits, sm_scale, causal):
    q = f32(q_bits).astype(np.float64)
    k = f32(k_bits).astype(np.float64)
    n, Hq, D = q.shape
    L, Hkv, _ = k.shape
    G = Hq // Hkv
    out = np.zeros((n, Hq))
    for g in range(Hq):
        logits = sm_scale * (q[:, g, :] @ k[:, g // G, :].T)
        if causal:
            pos = L - n + np.arange(n)
            logits = np.where(np.arange(L)[None, :] > pos[:, None], -np.inf, logits)
        out[:, g] = logsumexp(logits, axis=1)
    return out


def scores(q_bits, k_bits, sm_scale, causal, agg="sum"):
    """[Hkv, L] fp64 aggregate of the attention matrix."""
    P = attention_probs(q_bits, k_bits, sm_scale, causal)
    n, Hq, L = P.shape
    Hkv = k_bits.shape[1]
    G = Hq // Hkv
    Pg = P.reshape(n, Hkv, G, L)
    if agg == "sum":
        return Pg.sum(axis=(0, 2))
    return Pg.max(axis=2).sum(axis=0) / max(n, 1)


def pool(x, w):
    """Centred max-pool with -inf padding (window w odd)."""
    h = w // 2
    pad = np.concatenate([np.full(h, -np.inf, np.float32), np.asarray(x, np.float32),
                          np.full(h, -np.inf, np.float32)])
    return sliding_window_view(pad, w).max(axis=1).astype(np.float32)


def topk_ascending(v, k):
    """The k entries with the largest value, ties to the lower index, sorted ascending."""
    v = np.asarray(v)
    order = np.lexsort((np.arange(v.shape[0]), -v.astype(np.float64)))
    return np.sort(order[:k]).astype(np.int32)
