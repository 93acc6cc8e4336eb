"""Pins of the oracle's query-aware token selection (oracle.snapkv)."""
import numpy as np
import pytest

from oracle import snapkv as S

W = S.WINDOW


def _inputs(seed, Hq=4, Hkv=2, n=80, D=16):
    rng = np.random.default_rng(seed)
    return rng.standard_normal((Hq, W, D)), rng.standard_normal((Hkv, n, D))


def test_importance_matches_explicit_loops():
    q, K = _inputs(1, Hq=2, Hkv=1, n=40, D=4)
    scale = 0.7
    n = K.shape[1]
    want = np.zeros(n)
    for g in range(2):
        for w in range(W):
            last = n - W + w
            sc = [scale * sum(q[g, w, c] * K[0, t, c] for c in range(4)) for t in range(last + 1)]
            m = max(sc)
            e = [np.exp(x - m) for x in sc]
            z = sum(e)
            for t in range(last + 1):
                want[t] += e[t] / z
    assert np.allclose(S.importance(q, K, scale)[0], want, rtol=1e-12, atol=1e-14)


def test_importances_add_up_to_heads_times_window():
    q, K = _inputs(2)
    imp = S.importance(q, K, 0.3)
    assert np.allclose(imp.sum(axis=1), 2 * W, rtol=1e-12)


def test_scale_zero_closed_form():
    q, K = _inputs(3, n=70)
    imp = S.importance(q, K, 0.0)
    n = 70
    per_head = sum(1.0 / (n - W + w + 1) for w in range(W))
    assert np.allclose(imp[:, :n - W], 2 * per_head, rtol=1e-12)
    # window position n - W + j is seen by window queries j .. W - 1
    for j in range(W):
        want = 2 * sum(1.0 / (n - W + w + 1) for w in range(j, W))
        assert np.allclose(imp[:, n - W + j], want, rtol=1e-12)


def test_causality_last_position():
    q, K = _inputs(4)
    n = K.shape[1]
    imp = S.importance(q, K, 0.5)
    for h in range(2):
        p_last = 0.0
        for g in range(2):
            s = 0.5 * (q[2 * h + g, W - 1] @ K[h].T)
            e = np.exp(s - s.max())
            p_last += e[-1] / e.sum()
        assert np.isclose(imp[h, n - 1], p_last, rtol=1e-12)


def test_prefix_permutation_permutes_importance():
    q, K = _inputs(5)
    n = K.shape[1]
    perm = np.random.default_rng(6).permutation(n - W)
    K2 = K.copy()
    K2[:, :n - W] = K[:, perm]
    a, b = S.importance(q, K, 0.4), S.importance(q, K2, 0.4)
    assert np.allclose(b[:, :n - W], a[:, perm], rtol=1e-12)
    assert np.allclose(b[:, n - W:], a[:, n - W:], rtol=1e-12)


def test_keep_all_and_window_only():
    q, K = _inputs(7)
    n = K.shape[1]
    assert np.array_equal(S.keep_list(q, K, 0.3, n), np.tile(np.arange(n), (2, 1)))
    assert np.array_equal(S.keep_list(q, K, 0.3, W), np.tile(np.arange(n - W, n), (2, 1)))


def test_planted_key_is_kept():
    q, K = _inputs(8)
    n = K.shape[1]
    K[0, 17] = 50.0 * q[0:2].sum(axis=(0, 1)) / np.linalg.norm(q[0:2].sum(axis=(0, 1)))
    kl = S.keep_list(q, K, 1.0, W + 1)
    assert kl[0, 0] == 17 and np.array_equal(kl[0, 1:], np.arange(n - W, n))


@pytest.mark.parametrize("keep", [W + 1, W + 10, 60])
def test_ties_keep_lowest_positions(keep):
    q, K = _inputs(9)
    K[:] = 0.0  # every visible score equal: prefix importances all equal
    kl = S.keep_list(q, K, 1.0, keep)
    n = K.shape[1]
    want = np.concatenate([np.arange(keep - W), np.arange(n - W, n)])
    assert np.array_equal(kl[0], want) and np.array_equal(kl[1], want)


def test_keep_list_is_sorted_unique_and_holds_window():
    q, K = _inputs(10, n=200)
    kl = S.keep_list(q, K, 0.25, 100)
    for h in range(2):
        assert np.all(np.diff(kl[h]) > 0)
        assert set(range(200 - W, 200)) <= set(kl[h].tolist())


# --- MLA layers: one keep list per sequence, the heads sharing the latent ---------

def _mla_inputs(seed, Hq=3, n=60, r=12, nope=4, dR=2):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((Hq, W, nope + dR)), rng.standard_normal((n, r)), rng.standard_normal((n, dR)),
            rng.standard_normal((Hq, nope, r)) / np.sqrt(r))


def test_mla_importance_matches_explicit_loops():
    q, C, R, Wk = _mla_inputs(11, Hq=2, n=36, r=6, nope=3, dR=2)
    scale, n = 0.6, C.shape[0]
    want = np.zeros(n)
    for h in range(2):
        for w in range(W):
            last = n - W + w
            sc = []
            for t in range(last + 1):
                key = [sum(Wk[h, i, c] * C[t, c] for c in range(6)) for i in range(3)] + [R[t, 0], R[t, 1]]
                sc.append(scale * sum(q[h, w, j] * key[j] for j in range(5)))
            m = max(sc)
            e = [np.exp(x - m) for x in sc]
            z = sum(e)
            for t in range(last + 1):
                want[t] += e[t] / z
    assert np.allclose(S.importance_mla(q, C, R, Wk, scale), want, rtol=1e-12, atol=1e-14)


def test_mla_importance_reduces_to_multi_head_attention():
    """W_UK[h] reading a slice of the latent of its own: head h's keys are that slice
    and the positional keys, so the MLA importance is the sum over heads of the
    (pinned) per-KV-head importance with one query head per KV head."""
    Hq, n, nope, dR = 3, 50, 4, 2
    rng = np.random.default_rng(12)
    q = rng.standard_normal((Hq, W, nope + dR))
    C = rng.standard_normal((n, Hq * nope))
    R = rng.standard_normal((n, dR))
    Wk = np.zeros((Hq, nope, Hq * nope))
    for h in range(Hq):
        Wk[h, :, h * nope:(h + 1) * nope] = np.eye(nope)
    K = np.stack([np.concatenate([C[:, h * nope:(h + 1) * nope], R], axis=1) for h in range(Hq)])
    want = S.importance(q, K, 0.45).sum(axis=0)
    assert np.allclose(S.importance_mla(q, C, R, Wk, 0.45), want, rtol=1e-12)


def test_mla_importance_positional_part_alone():
    """No-RoPE queries of zero: only the shared positional keys score, as one KV head
    read by all query heads."""
    q, C, R, Wk = _mla_inputs(13)
    q[:, :, :4] = 0.0
    want = S.importance(q[:, :, 4:], R[None], 0.8)[0]
    assert np.allclose(S.importance_mla(q, C, R, Wk, 0.8), want, rtol=1e-12)


def test_mla_importance_mass_and_scale_zero():
    q, C, R, Wk = _mla_inputs(14, Hq=4, n=70)
    assert np.isclose(S.importance_mla(q, C, R, Wk, 0.3).sum(), 4 * W, rtol=1e-12)
    imp0 = S.importance_mla(q, C, R, Wk, 0.0)
    n = 70
    closed = 4 * sum(1.0 / (n - W + w + 1) for w in range(W))
    assert np.allclose(imp0[:n - W], closed, rtol=1e-12)
    kl = S.keep_list_mla(q, C, R, Wk, 0.3, 40)
    assert kl.shape == (40,) and np.all(np.diff(kl) > 0) and np.array_equal(kl[-W:], np.arange(n - W, n))
