"""Query-aware token selection at prefill, as the paper's eviction baseline (oracle).

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

The paper's configurations do not drop positions, so an evictor can run on the
same cache and the reductions multiply (§3.4); it pairs them with SnapKV keeping
one position in four or eight, and its eviction implementations sum attention
over a 32-query observation window (App. F.3, eviction implementations).  What is
computed here, per sequence and KV head, from the keys K [n, D] of the prompt and
the queries of its last W = 32 positions (both after RoPE):

  * window query w sits at position n - W + w and attends causally: its
    probabilities are softmax_t(scale q_w . k_t) over t = 0 .. n - W + w;
  * the importance of position t is the sum of those probabilities over the W
    window queries and over the G query heads that read the KV head;
  * the W window positions are always kept; the other keep - W positions are the
    prefix positions (t < n - W) of largest importance, ties going to the lower
    position; the keep list is in increasing order (the eviction gather's input).

The paper names no pooling of the importances, so there is none.  Everything is
fp64 from the given (bf16-valued) inputs.

Pins (tests/test_oracle_snapkv.py): explicit loops on a tiny input; every
softmax row sums to one, so the importances of all n positions add up to G W;
scale 0 gives the closed form sum_w 1 / (n - W + w + 1) per head for every prefix
position; causality (the last position is seen by one window query only);
permuting the prefix keys permutes their importances; keep = n keeps everything
and keep = W only the window; a planted key aligned with the window queries is
kept; equal importances keep the lowest positions.
"""
import numpy as np

WINDOW = 32


def importance(q_obs: np.ndarray, K: np.ndarray, scale: float, window: int = WINDOW) -> np.ndarray:
    """q_obs [Hq, W, D] (the window queries), K [Hkv, n, D] -> importance [Hkv, n]
    (fp64): sum over the G query heads of a KV head and the W window queries of
    their causal softmax probabilities."""
    q = np.asarray(q_obs, dtype=np.float64)
    K = np.asarray(K, dtype=np.float64)
    Hq, W, _ = q.shape
    Hkv, n, _ = K.shape
    assert W == window and n >= W and Hq % Hkv == 0
    G = Hq // Hkv
    pos = n - W + np.arange(W)                      # absolute position of each window query
    visible = np.arange(n)[None, :] <= pos[:, None]  # [W, n] causal mask
    imp = np.zeros((Hkv, n))
    for h in range(Hkv):
        for g in range(G):
            s = scale * (q[h * G + g] @ K[h].T)      # [W, n]
            s = np.where(visible, s, -np.inf)
            s = s - s.max(axis=1, keepdims=True)
            p = np.exp(s)
            p /= p.sum(axis=1, keepdims=True)
            imp[h] += p.sum(axis=0)
    return imp


def select(imp: np.ndarray, keep: int, window: int = WINDOW) -> np.ndarray:
    """importance [n] -> kept positions [keep] (int32, increasing): the window plus
    the keep - W prefix positions of largest importance (ties: lower position)."""
    n = imp.shape[0]
    assert window <= keep <= n
    prefix = n - window
    order = sorted(range(prefix), key=lambda t: (-imp[t], t))
    chosen = sorted(order[:keep - window]) + list(range(prefix, n))
    return np.asarray(chosen, dtype=np.int32)


def keep_list(q_obs: np.ndarray, K: np.ndarray, scale: float, keep: int, window: int = WINDOW) -> np.ndarray:
    """[Hkv, keep] kept positions of one sequence."""
    imp = importance(q_obs, K, scale, window)
    return np.stack([select(imp[h], keep, window) for h in range(imp.shape[0])])


# ---------------------------------------------------------------------------
# MLA layers (§2.1 "Rank", App. C.2): the latent is shared by every head, so a
# sequence keeps one list of positions for all heads.  Head h's key at position t is
# [W_UK[h] c_t ; k^R_t] (the latent at its full width r, before the layer keeps
# its first d coordinates); its window queries are [q_nope ; q_rope].  The
# importance of a position sums the causal softmax probabilities over the 32
# window queries of every query head; the selection rule is the one above.
# ---------------------------------------------------------------------------

def importance_mla(q_obs: np.ndarray, C: np.ndarray, R: np.ndarray, W_UK: np.ndarray, scale: float,
                   window: int = WINDOW) -> np.ndarray:
    """q_obs [Hq, W, nope + d_R] (each head's window queries: no-RoPE part, then the
    RoPE part), C [n, r] latent, R [n, d_R] positional keys, W_UK [Hq, nope, r] ->
    importance [n] (fp64), the keys reconstructed per head."""
    q = np.asarray(q_obs, dtype=np.float64)
    C = np.asarray(C, dtype=np.float64)
    R = np.asarray(R, dtype=np.float64)
    Wk = np.asarray(W_UK, dtype=np.float64)
    Hq, W, qw = q.shape
    n, dR = R.shape
    nope = qw - dR
    assert W == window and n >= W and Wk.shape[:2] == (Hq, nope)
    pos = n - W + np.arange(W)
    visible = np.arange(n)[None, :] <= pos[:, None]
    imp = np.zeros(n)
    for h in range(Hq):
        K = np.concatenate([C @ Wk[h].T, R], axis=1)  # [n, nope + d_R]: head h's keys
        s = scale * (q[h] @ K.T)                      # [W, n]
        s = np.where(visible, s, -np.inf)
        s = s - s.max(axis=1, keepdims=True)
        p = np.exp(s)
        p /= p.sum(axis=1, keepdims=True)
        imp += p.sum(axis=0)
    return imp


def keep_list_mla(q_obs, C, R, W_UK, scale: float, keep: int, window: int = WINDOW) -> np.ndarray:
    """[keep] kept positions of one sequence of an MLA layer."""
    return select(importance_mla(q_obs, C, R, W_UK, scale, window), keep, window)
