"""Pins of the oracle's selector forward pass (oracle.selector)."""
import numpy as np

from oracle import selector as S

W = S.WIDTH


def _block(rng, scale=0.05, zero=False):
    def m(*shape):
        return np.zeros(shape) if zero else rng.standard_normal(shape) * scale
    return {"ln1_g": np.ones(W), "ln1_b": np.zeros(W), "w_qkv": m(W, 3 * W), "b_qkv": m(3 * W),
            "w_o": m(W, W), "b_o": m(W), "ln2_g": np.ones(W), "ln2_b": np.zeros(W),
            "w_1": m(W, S.FFN), "b_1": m(S.FFN), "w_2": m(S.FFN, W), "b_2": m(W)}


def _weights(rng, d_model=64, L=6, zero_blocks=False):
    return {"w_in": rng.standard_normal((d_model, W)) * 0.1, "b_in": rng.standard_normal(W) * 0.1,
            "blocks": [_block(rng, zero=zero_blocks) for _ in range(2)],
            "w_head": rng.standard_normal((L, W, S.N_ACTIONS)) * 0.1, "b_head": np.zeros((L, S.N_ACTIONS))}


def test_zero_blocks_are_identity():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((10, W))
    p = _block(rng, zero=True)
    assert np.array_equal(S.block(x, p), x)


def test_attention_over_identical_positions_returns_the_value():
    rng = np.random.default_rng(2)
    row = rng.standard_normal(W)
    x = np.tile(row, (7, 1))
    w_qkv, b_qkv = rng.standard_normal((W, 3 * W)), rng.standard_normal(3 * W)
    eye = np.eye(W)
    out = S.attention(x, w_qkv, b_qkv, eye, np.zeros(W))
    v = (row @ w_qkv + b_qkv)[2 * W:]
    assert np.allclose(out, np.tile(v, (7, 1)), rtol=1e-12, atol=1e-12)


def test_attention_and_layernorm_match_loops():
    rng = np.random.default_rng(3)
    x = rng.standard_normal((5, W))
    g, b = rng.standard_normal(W), rng.standard_normal(W)
    ln = S.layer_norm(x, g, b)
    for t in range(5):
        mu = sum(x[t]) / W
        var = sum((xi - mu) ** 2 for xi in x[t]) / W
        assert np.allclose(ln[t], [(x[t, c] - mu) / np.sqrt(var + 1e-5) * g[c] + b[c] for c in range(W)])
    w_qkv, b_qkv = rng.standard_normal((W, 3 * W)) * 0.1, rng.standard_normal(3 * W) * 0.1
    out = S.attention(x, w_qkv, b_qkv, np.eye(W), np.zeros(W))
    qkv = x @ w_qkv + b_qkv
    for h in range(S.HEADS):
        for t in range(5):
            sc = [sum(qkv[t, 64 * h + c] * qkv[u, W + 64 * h + c] for c in range(64)) / 8.0 for u in range(5)]
            e = np.exp(np.array(sc) - max(sc))
            want = sum(e[u] * qkv[u, 2 * W + 64 * h:2 * W + 64 * (h + 1)] for u in range(5)) / e.sum()
            assert np.allclose(out[t, 64 * h:64 * (h + 1)], want, rtol=1e-10)


def test_feature_is_token_order_invariant():
    rng = np.random.default_rng(4)
    w = _weights(rng)
    emb = rng.standard_normal((20, 64))
    perm = rng.permutation(20)
    assert np.allclose(S.feature(emb, w), S.feature(emb[perm], w), rtol=1e-10, atol=1e-12)


def test_layer_zero_never_inherits_and_biases_steer_the_argmax():
    rng = np.random.default_rng(5)
    w = _weights(rng)
    w["w_head"][:] = 0.0
    w["b_head"][:, 0] = 10.0  # every layer prefers depth ...
    emb = rng.standard_normal((9, 64))
    pl = S.plan(emb, w)
    assert pl[0] != (1, 16) and all(a == (1, 16) for a in pl[1:])
    w["b_head"][:] = 0.0
    w["b_head"][:, 3] = 5.0  # ... or int4
    assert all(a == (0, 4) for a in S.plan(emb, w))
