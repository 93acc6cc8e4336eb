"""Pins of the oracle's attention, depth sharing, eviction and cache round trip."""
import math

import numpy as np
import pytest
import torch
from scipy.special import softmax as sp_softmax

from oracle import attention as A
from oracle import cache as C
from oracle import plan as P
from oracle import quant as Q


def _brute(q, K, V, scale):
    """Softmax attention with explicit Python loops (tiny inputs only)."""
    H, T, Dv = len(q), len(K), len(V[0])
    out = []
    for h in range(H):
        s = [scale * sum(q[h][c] * K[t][c] for c in range(len(q[h]))) for t in range(T)]
        m = max(s)
        e = [math.exp(x - m) for x in s]
        z = sum(e)
        out.append([sum(e[t] * V[t][c] for t in range(T)) / z for c in range(Dv)])
    return np.array(out)


def test_softmax_attention_brute_force():
    rng = np.random.default_rng(0)
    q, K, V = rng.standard_normal((3, 5)), rng.standard_normal((7, 5)), rng.standard_normal((7, 4))
    got = A.softmax_attention(q, K, V, 0.7)
    assert np.allclose(got, _brute(q.tolist(), K.tolist(), V.tolist(), 0.7), rtol=1e-12, atol=1e-13)
    ref = sp_softmax(0.7 * q @ K.T, axis=1) @ V
    assert np.allclose(got, ref, rtol=1e-12, atol=1e-13)


def test_special_cases():
    rng = np.random.default_rng(1)
    K, V = rng.standard_normal((9, 6)), rng.standard_normal((9, 6))
    q = rng.standard_normal((2, 6))
    assert np.allclose(A.softmax_attention(q, K[:1], V[:1], 1.0), V[:1].repeat(2, 0))
    assert np.allclose(A.softmax_attention(np.zeros((1, 6)), K, V, 1.0), V.mean(0, keepdims=True))
    perm = rng.permutation(9)
    assert np.allclose(A.softmax_attention(q, K, V, 0.3), A.softmax_attention(q, K[perm], V[perm], 0.3))
    assert np.all(A.softmax_attention(q, K[:0], V[:0], 1.0) == 0)


@pytest.mark.parametrize("cuts", [[0, 9], [0, 4, 9], [0, 1, 2, 9], [0, 0, 5, 9]])
def test_split_lse_merge_equals_single_pass(cuts):
    rng = np.random.default_rng(2)
    K, V, q = rng.standard_normal((9, 6)), rng.standard_normal((9, 5)), rng.standard_normal((3, 6)) * 4
    parts = [A.partial_attention(q, K[a:b], V[a:b], 0.5) for a, b in zip(cuts[:-1], cuts[1:])]
    assert np.allclose(A.lse_merge(parts), A.softmax_attention(q, K, V, 0.5), rtol=1e-12, atol=1e-14)


def test_gqa_head_mapping_brute_force():
    rng = np.random.default_rng(3)
    Hq, Hkv, T, D = 6, 2, 5, 4
    q, K, V = rng.standard_normal((Hq, D)), rng.standard_normal((Hkv, T, D)), rng.standard_normal((Hkv, T, D))
    got = A.gqa_attention(q, K, V, 0.9)
    for h in range(Hq):
        kv = h // 3
        assert np.allclose(got[h], _brute([q[h].tolist()], K[kv].tolist(), V[kv].tolist(), 0.9)[0])


def _bf16_inputs(seed, shape, scale=1.0):
    g = torch.Generator().manual_seed(seed)
    x = (torch.randn(shape, generator=g) * scale).to(torch.bfloat16)
    return x.float().numpy()


@pytest.mark.parametrize("n", [1, 31, 32, 77, 96])
def test_bf16_layer_recovers_input_exactly(n):
    """b = 16 on bf16 inputs stores them unchanged (the uncompressed model, §2.2),
    including the tail of n % 32 tokens."""
    dims = P.Dims(P.GQA, 1, 4, 2, 64, batch=2, max_tokens=96)
    K, V = _bf16_inputs(0, (2, 2, n, 64)), _bf16_inputs(1, (2, 2, n, 64))
    reg = C.compress_layer(dims, 16, K, V)
    arena = reg
    Kh, Vh = C.dequant_layer(dims, [P.Action(bits=16)], arena, 0, n)
    assert np.array_equal(Kh, K) and np.array_equal(Vh, V)
    q = _bf16_inputs(2, (1, 2, 4, 64))
    out = C.decode_step(dims, [P.Action(bits=16)], arena, q, n, 0.125)
    for b in range(2):
        assert np.allclose(out[0, b], A.gqa_attention(q[0, b], K[b], V[b], 0.125), rtol=1e-13)


@pytest.mark.parametrize("qs", [P.KIVI32, P.SYMROW, P.GROUP64])
@pytest.mark.parametrize("bits", [2, 4, 8])
def test_cache_roundtrip_matches_direct_quantiser(qs, bits):
    """Compress -> bytes -> dequantise equals quantising the groups directly."""
    D, n = 64, 70
    dims = P.Dims(P.GQA, 1, 2, 1, D, qscheme=qs, batch=1, max_tokens=96)
    K, V = _bf16_inputs(5, (1, 1, n, D), 2.0), _bf16_inputs(6, (1, 1, n, D))
    reg = C.compress_layer(dims, bits, K, V)
    Kh, Vh = C.dequant_layer(dims, [P.Action(bits=bits)], reg, 0, n)
    k, v = K[0, 0], V[0, 0]
    for blk in range(2):
        kb, vb = k[32 * blk:32 * blk + 32], v[32 * blk:32 * blk + 32]
        if qs == P.KIVI32:
            u, s, z = Q.kivi_quantize(kb.T, bits)
            assert np.array_equal(Kh[0, 0, 32 * blk:32 * blk + 32], Q.kivi_dequantize(u, s[:, None], z[:, None]).T)
            u, s, z = Q.kivi_quantize(vb.reshape(32, D // 32, 32), bits)
            ref = Q.kivi_dequantize(u, s[..., None], z[..., None]).reshape(32, D)
        elif qs == P.GROUP64:
            u, s, z = Q.kivi_quantize(kb.reshape(32, D // 64, 64), bits)
            assert np.array_equal(Kh[0, 0, 32 * blk:32 * blk + 32],
                                  Q.kivi_dequantize(u, s[..., None], z[..., None]).reshape(32, D))
            u, s, z = Q.kivi_quantize(vb.reshape(32, D // 64, 64), bits)
            ref = Q.kivi_dequantize(u, s[..., None], z[..., None]).reshape(32, D)
        else:
            u, s = Q.symrow_quantize(kb, bits)
            assert np.array_equal(Kh[0, 0, 32 * blk:32 * blk + 32], Q.symrow_dequantize(u, s[:, None], bits))
            u, s = Q.symrow_quantize(vb, bits)
            ref = Q.symrow_dequantize(u, s[:, None], bits)
        assert np.array_equal(Vh[0, 0, 32 * blk:32 * blk + 32], ref)
    assert np.array_equal(Kh[0, 0, 64:], K[0, 0, 64:]) and np.array_equal(Vh[0, 0, 64:], V[0, 0, 64:])


def test_depth_inheritor_reads_anchor():
    """§2.1: an inheriting layer attends over its anchor's cache with its own query;
    with the anchor's query it reproduces the anchor's output exactly."""
    dims = P.Dims(P.GQA, 3, 4, 2, 64, batch=1, max_tokens=64)
    plan = [P.Action(bits=4), P.Action(inherit=True), P.Action(bits=8)]
    Ks = [_bf16_inputs(10 + l, (1, 2, 64, 64)) for l in range(3)]
    Vs = [_bf16_inputs(20 + l, (1, 2, 64, 64)) for l in range(3)]
    arena = C.compress_arena(dims, plan, Ks, Vs)
    q = _bf16_inputs(30, (3, 1, 4, 64))
    q[1] = q[0]
    out = C.decode_step(dims, plan, arena, q, 64, 0.125)
    assert np.array_equal(out[0], out[1])
    q2 = q.copy()
    q2[1] = _bf16_inputs(31, (1, 4, 64))
    out2 = C.decode_step(dims, plan, arena, q2, 64, 0.125)
    Kh, Vh = C.dequant_layer(dims, plan, arena, 0, 64)
    assert np.allclose(out2[1, 0], A.gqa_attention(q2[1, 0], Kh[0], Vh[0], 0.125))


def test_eviction_equals_masked_attention():
    """§3 long context: evicting positions then attending equals attention over the
    uncompressed cache with those positions masked out (b = 16, exact)."""
    n, keep = 100, 45
    dims = P.Dims(P.GQA, 1, 2, 1, 64, batch=1, max_tokens=n, keep_tokens=keep)
    K, V = _bf16_inputs(40, (1, 1, n, 64)), _bf16_inputs(41, (1, 1, n, 64))
    rng = np.random.default_rng(7)
    kidx = np.sort(rng.choice(n, keep, replace=False))[None, None]
    reg = C.compress_layer(dims, 16, K, V, kidx)
    q = _bf16_inputs(42, (1, 1, 2, 64))
    out = C.decode_step(dims, [P.Action(bits=16)], reg, q, keep, 0.125)
    s = 0.125 * q[0, 0].astype(np.float64) @ K[0, 0].T.astype(np.float64)
    mask = np.full(n, -np.inf)
    mask[kidx[0, 0]] = 0
    ref = sp_softmax(s + mask, axis=1) @ V[0, 0]
    assert np.allclose(out[0, 0], ref, rtol=1e-12, atol=1e-14)
    # keeping every position is the identity
    dims_all = P.Dims(P.GQA, 1, 2, 1, 64, batch=1, max_tokens=n, keep_tokens=n)
    reg_all = C.compress_layer(dims_all, 16, K, V, np.arange(n)[None, None])
    dims_none = P.Dims(P.GQA, 1, 2, 1, 64, batch=1, max_tokens=n)
    assert np.array_equal(reg_all, C.compress_layer(dims_none, 16, K, V))
