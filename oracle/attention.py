"""Softmax attention over a dequantised cache (oracle).

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

A decode step is one query per head attending over the stored tokens of its
layer's cache (§2.1: a layer uses its own query and reads its anchor's keys and
values; GQA query head h reads KV head h / (Hq/Hkv)).  Everything here is fp64.

Pins: brute-force loops on tiny inputs, scipy's softmax, T = 1 gives the single
value row, q = 0 gives the mean of the values, invariance under a permutation
of the tokens, and a split of the tokens merged by log-sum-exp equals one pass.
"""
import numpy as np


def softmax_attention(q: np.ndarray, K: np.ndarray, V: np.ndarray, scale: float) -> np.ndarray:
    """q [H, D], K [T, D], V [T, Dv] -> [H, Dv]; p = softmax(scale q.K^T) over the
    T tokens; T = 0 gives zeros."""
    q = np.asarray(q, dtype=np.float64)
    K = np.asarray(K, dtype=np.float64)
    V = np.asarray(V, dtype=np.float64)
    if K.shape[0] == 0:
        return np.zeros((q.shape[0], V.shape[1]))
    s = scale * (q @ K.T)
    s = s - s.max(axis=1, keepdims=True)
    p = np.exp(s)
    return (p @ V) / p.sum(axis=1, keepdims=True)


def partial_attention(q, K, V, scale):
    """One split's (m, l, o): m = max score, l = sum exp(s - m), o = sum exp(s - m) v
    (unnormalised).  Empty splits give m = -inf, l = 0, o = 0."""
    q = np.asarray(q, dtype=np.float64)
    if K.shape[0] == 0:
        return (np.full(q.shape[0], -np.inf), np.zeros(q.shape[0]),
                np.zeros((q.shape[0], V.shape[1])))
    s = scale * (q @ np.asarray(K, np.float64).T)
    m = s.max(axis=1)
    p = np.exp(s - m[:, None])
    return m, p.sum(axis=1), p @ np.asarray(V, np.float64)


def lse_merge(parts):
    """Merge split partials: m* = max m_i, l* = sum l_i e^(m_i - m*),
    o = sum o_i e^(m_i - m*) / l*."""
    ms = np.stack([p[0] for p in parts])
    mstar = ms.max(axis=0)
    w = np.where(np.isfinite(ms), np.exp(ms - mstar), 0.0)
    l = sum(wi * p[1] for wi, p in zip(w, parts))
    o = sum(wi[:, None] * p[2] for wi, p in zip(w, parts))
    with np.errstate(invalid="ignore", divide="ignore"):
        return np.where(l[:, None] > 0, o / l[:, None], 0.0)


def gqa_attention(q: np.ndarray, K: np.ndarray, V: np.ndarray, scale: float) -> np.ndarray:
    """q [Hq, D]; K, V [Hkv, T, D] -> [Hq, D]; head h reads KV head h // (Hq/Hkv)."""
    Hq, Hkv = q.shape[0], K.shape[0]
    G = Hq // Hkv
    out = np.zeros((Hq, V.shape[2]))
    for kv in range(Hkv):
        out[kv * G:(kv + 1) * G] = softmax_attention(q[kv * G:(kv + 1) * G], K[kv], V[kv], scale)
    return out
