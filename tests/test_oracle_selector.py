"""Pins of the oracle's selector forward pass (oracle.selector) against App. B and
the mathematics, independent of the oracle's own formulas."""
import numpy as np
import pytest
import torch

from oracle import selector as S

W, DH = S.WIDTH, S.HEAD_DIM


def _random_weights(rng, d_model=64, L=6, n_actions=S.N_ACTIONS_FULL, scale=0.05, zero_blocks=False):
    shapes = S.weight_shapes(d_model, L, n_actions)

    def draw(shape, key):
        if key.startswith("g_"):
            return 1.0 + 0.1 * rng.standard_normal(shape)
        if zero_blocks:
            return np.zeros(shape)
        return rng.standard_normal(shape) * scale

    w = {k: draw(v, k) for k, v in shapes.items() if k != "blocks"}
    w["w_in"] = rng.standard_normal(shapes["w_in"]) / np.sqrt(d_model)
    w["blocks"] = [{k: draw(v, k) for k, v in b.items()} for b in shapes["blocks"]]
    return w


# App. B prints the selector's size with 17 actions per layer for six backbones.
# Embedding widths H are those of the public model configurations; L from the
# backbone table.
PRINTED = [("Qwen2.5-1.5B", 1536, 28, 2.61e6), ("Qwen2.5-3B", 2048, 36, 2.78e6),
           ("Qwen2.5-7B", 3584, 28, 3.14e6), ("Qwen2.5-14B", 5120, 48, 3.62e6),
           ("Qwen2.5-32B", 5120, 64, 3.69e6), ("Mistral-7B / OLMo-3-7B", 4096, 32, 3.29e6)]


def _count(shapes):
    n = 0
    for k, v in shapes.items():
        if k == "blocks":
            n += sum(int(np.prod(s)) for b in v for s in b.values())
        else:
            n += int(np.prod(v))
    return n


@pytest.mark.parametrize("name,H,L,printed", PRINTED)
def test_parameter_count_matches_appendix(name, H, L, printed):
    shapes = S.weight_shapes(H, L, S.N_ACTIONS_FULL)
    n = _count(shapes)
    assert round(n / 1e4) == round(printed / 1e4), (name, n)  # three significant figures
    heads = int(np.prod(shapes["w_head"])) + int(np.prod(shapes["b_head"]))
    assert 122e3 <= round(heads, -3) <= 280e3  # "the per-layer heads account for 122k-280k"


def test_head_parameter_range_endpoints():
    lo = [_count({"w_head": S.weight_shapes(H, L)["w_head"], "b_head": S.weight_shapes(H, L)["b_head"]})
          for _, H, L, _ in PRINTED]
    assert round(min(lo), -3) == 122e3 and round(max(lo), -3) == 280e3


def test_the_shapes_are_the_ones_consumed():
    rng = np.random.default_rng(0)
    w = _random_weights(rng, d_model=96, L=5)
    z = S.logits(rng.standard_normal((7, 96)), w)
    assert z.shape == (5, S.N_ACTIONS_FULL) and np.isfinite(z[1:]).all()


def test_rms_norm_loops_and_torch():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((5, W)) * 3.0
    g = rng.standard_normal(W)
    got = S.rms_norm(x, g)
    for t in range(5):
        ms = sum(xi * xi for xi in x[t]) / W
        assert np.allclose(got[t], [x[t, c] / np.sqrt(ms + 1e-6) * g[c] for c in range(W)], rtol=1e-13)
    ref = torch.nn.functional.rms_norm(torch.from_numpy(x), (W,), torch.from_numpy(g), eps=1e-6).numpy()
    assert np.allclose(got, ref, rtol=1e-12, atol=1e-12)
    ones = S.rms_norm(x, np.ones(W))
    assert np.allclose(np.sqrt((ones ** 2).mean(axis=1)), 1.0, atol=1e-6)  # unit RMS
    assert np.allclose(S.rms_norm(7.5 * x, g), got, rtol=1e-6)  # scale invariant (up to eps)


def test_swiglu_loops_and_torch():
    rng = np.random.default_rng(2)
    n = rng.standard_normal((3, W))
    p = {"w_gate": rng.standard_normal((S.FFN, W)) * 0.05, "w_up": rng.standard_normal((S.FFN, W)) * 0.05,
         "w_down": rng.standard_normal((W, S.FFN)) * 0.05}
    got = S.swiglu(n, p)
    for t in range(3):
        hid = []
        for j in range(S.FFN):
            a = sum(p["w_gate"][j, c] * n[t, c] for c in range(W))
            b = sum(p["w_up"][j, c] * n[t, c] for c in range(W))
            hid.append(a / (1.0 + np.exp(-a)) * b)
        want = [sum(p["w_down"][o, j] * hid[j] for j in range(S.FFN)) for o in range(W)]
        assert np.allclose(got[t], want, rtol=1e-10, atol=1e-12)
    tn = torch.from_numpy(n)
    ref = (torch.nn.functional.silu(tn @ torch.from_numpy(p["w_gate"]).T) * (tn @ torch.from_numpy(p["w_up"]).T)) \
        @ torch.from_numpy(p["w_down"]).T
    assert np.allclose(got, ref.numpy(), rtol=1e-12, atol=1e-13)
    # SiLU(0) = 0: a zero gate gives a zero feed-forward output whatever W_up is
    p0 = dict(p, w_gate=np.zeros_like(p["w_gate"]))
    assert np.array_equal(S.swiglu(n, p0), np.zeros((3, W)))


def test_rope_is_a_complex_rotation_of_channel_pairs():
    rng = np.random.default_rng(3)
    x = rng.standard_normal((9, DH))
    pos = np.array([0, 1, 2, 5, 17, 100, 1000, 4095, 32767])
    got = S.rope(x, pos)
    zc = (x[:, :32] + 1j * x[:, 32:]) * np.exp(1j * pos[:, None] * 10000.0 ** (-np.arange(32) / 32.0))
    assert np.allclose(got[:, :32], zc.real, rtol=1e-12, atol=1e-12)
    assert np.allclose(got[:, 32:], zc.imag, rtol=1e-12, atol=1e-12)
    assert np.allclose(np.linalg.norm(got, axis=1), np.linalg.norm(x, axis=1), rtol=1e-13)
    assert np.array_equal(S.rope(x[:1], [0]), x[:1])  # position 0: identity
    # channel 0 pairs with channel 32 at frequency 1 rad per position
    e0 = np.zeros((1, DH)); e0[0, 0] = 1.0
    r = S.rope(e0, [1])
    assert np.isclose(r[0, 0], np.cos(1.0)) and np.isclose(r[0, 32], np.sin(1.0)) and abs(r[0, 1:32]).max() == 0


def _block_params(rng, scale=0.08):
    return {k: (1.0 + 0.1 * rng.standard_normal(v) if k.startswith("g_") else rng.standard_normal(v) * scale)
            for k, v in S.weight_shapes(64, 1)["blocks"][0].items()}


def test_attention_without_rotation_matches_torch_sdpa():
    rng = np.random.default_rng(4)
    n = rng.standard_normal((11, W))
    p = _block_params(rng)
    got = S.attention(n, p, np.zeros(11))  # every position 0: RoPE is the identity
    tn = torch.from_numpy(n)
    q = (tn @ torch.from_numpy(p["w_q"]).T).reshape(11, 4, DH).transpose(0, 1)
    k = (tn @ torch.from_numpy(p["w_k"]).T).reshape(11, 4, DH).transpose(0, 1)
    v = (tn @ torch.from_numpy(p["w_v"]).T).reshape(11, 4, DH).transpose(0, 1)
    o = torch.nn.functional.scaled_dot_product_attention(q, k, v)  # scale 1/sqrt(64), no mask
    ref = o.transpose(0, 1).reshape(11, W) @ torch.from_numpy(p["w_o"]).T
    assert np.allclose(got, ref.numpy(), rtol=1e-10, atol=1e-12)


def test_attention_depends_only_on_relative_positions():
    rng = np.random.default_rng(5)
    n = rng.standard_normal((13, W))
    p = _block_params(rng)
    base = np.arange(13)
    a = S.attention(n, p, base)
    for shift in (1, 37, 5000):
        assert np.allclose(S.attention(n, p, base + shift), a, rtol=1e-8, atol=1e-10)
    # ... but not on absolute order: reversing the positions changes it
    assert not np.allclose(S.attention(n, p, base[::-1].copy()), a, atol=1e-6)


def test_attention_over_identical_tokens_returns_their_value():
    rng = np.random.default_rng(6)
    row = rng.standard_normal(W)
    n = np.tile(row, (7, 1))
    p = _block_params(rng)
    p["w_o"] = np.eye(W)
    out = S.attention(n, p, np.arange(7))
    assert np.allclose(out, np.tile(p["w_v"] @ row, (7, 1)), rtol=1e-12, atol=1e-12)


def test_zero_weight_block_is_identity():
    rng = np.random.default_rng(7)
    x = rng.standard_normal((10, W))
    p = {k: (np.ones(v) if k.startswith("g_") else np.zeros(v))
         for k, v in S.weight_shapes(64, 1)["blocks"][0].items()}
    assert np.array_equal(S.block(x, p, np.arange(10)), x)


def test_zero_blocks_reduce_to_normalised_mean():
    rng = np.random.default_rng(8)
    w = _random_weights(rng, zero_blocks=True)
    emb = rng.standard_normal((6, 64))
    x = emb @ w["w_in"].T
    want = (x / np.sqrt((x ** 2).mean(axis=1, keepdims=True) + 1e-6) * w["g_final"]).mean(axis=0)
    assert np.allclose(S.feature(emb, w), want, rtol=1e-12)


def test_feature_depends_on_token_order_and_is_bidirectional():
    rng = np.random.default_rng(9)
    w = _random_weights(rng, scale=0.1)
    emb = rng.standard_normal((20, 64))
    perm = rng.permutation(20)
    assert not np.allclose(S.feature(emb, w), S.feature(emb[perm], w), atol=1e-9)
    # the first position's block output sees the last token (no causal mask)
    p = w["blocks"][0]
    x = emb @ w["w_in"].T
    y1 = S.block(x, p, np.arange(20))
    x2 = x.copy()
    x2[-1] += 1.0
    assert not np.allclose(S.block(x2, p, np.arange(20))[0], y1[0], atol=1e-9)


def test_layer_zero_never_inherits_and_biases_steer_the_argmax():
    rng = np.random.default_rng(10)
    w = _random_weights(rng)
    w["w_head"][:] = 0.0
    w["b_head"][:] = 0.0
    w["b_head"][:, 0] = 10.0  # every layer prefers depth ...
    emb = rng.standard_normal((9, 64))
    acts = S.actions(emb, w)
    assert acts[0] != 0 and all(a == 0 for a in acts[1:])
    assert all(a != 0 for a in S.actions(emb, w, depth=False))  # ... unless depth is masked
    w["b_head"][:] = 0.0
    w["b_head"][:, 1] = 5.0  # App. B's initial bias: the least compressed action
    assert all(S.action_config(a) == (0, 1, 16) for a in S.actions(emb, w))
    w["b_head"][:] = 0.0
    w["b_head"][:, 1 + 4 * 2 + 2] = 5.0  # d = r/4 at 4 bits
    assert all(S.action_config(a) == (0, 4, 4) for a in S.actions(emb, w))


def test_action_space_is_eq3():
    assert len(S.ACTIONS) == 4 * 4 + 1 and S.ACTIONS[0][0] == 1
    produced = {(a[1], a[2]) for a in S.ACTIONS[1:]}
    assert produced == {(j, b) for j in (1, 2, 4, 8) for b in (2, 4, 8, 16)}
    assert [a[2] for a in S.ACTIONS[1:S.N_ACTIONS_GQA]] == [16, 8, 4, 2] and all(
        a[1] == 1 for a in S.ACTIONS[1:S.N_ACTIONS_GQA])


def test_film_zero_is_identity_and_affine():
    rng = np.random.default_rng(11)
    w = _random_weights(rng)
    emb = rng.standard_normal((5, 64))
    z = S.feature(emb, w)
    assert np.array_equal(S.feature(emb, w, film=(np.zeros(W), np.zeros(W))), z)
    g, b = rng.standard_normal(W), rng.standard_normal(W)
    assert np.allclose(S.feature(emb, w, film=(g, b)), z + z * g + b, rtol=1e-13)
