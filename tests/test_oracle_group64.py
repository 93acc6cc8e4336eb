"""Pins of the oracle's GROUP64 scheme: the grouped asymmetric per-token quantiser
with groups of 64 channels (App. C.3's on-device grouped cache, 3.56x at 4 bits),
keys and values alike."""
import numpy as np
import pytest

from oracle import cache as C
from oracle import layout as LY
from oracle import plan as P
from oracle import quant as Q


def _dims(D, n_cap=64):
    return P.Dims(P.GQA, 1, 2, 1, D, qscheme=P.GROUP64, batch=1, max_tokens=n_cap)


@pytest.mark.parametrize("bits", [2, 4, 8])
def test_block_size_gives_the_papers_bits_per_element(bits):
    """8 bytes x block / (32 tokens x 2 D values) = b + 32/64: 4.5 bits at b = 4, the
    3.56x of App. C.3's on-device figure."""
    for D in (64, 128):
        per = 8 * P.block_bytes(_dims(D), bits) / (32 * 2 * D)
        assert per == bits + 0.5
    assert round(16 / (4 + 0.5), 2) == 3.56
    assert P.realized_bits(P.GROUP64, 4, 64, 0, 16384) == 4.5


@pytest.mark.parametrize("D", [64, 128])
def test_meta_maps_are_bijections(D):
    ki, vi = LY.g64_kmeta_index(D), LY.g64_vmeta_index(D)
    assert np.array_equal(np.sort(ki.ravel()), np.arange(D))
    assert np.array_equal(np.sort(vi.ravel()), np.arange(D))


def test_meta_index_worked_by_hand():
    """D = 128 (two groups): the K scale of token 21 (tile 1, kg 1, e 1) in group 1 sits
    at ((1*4 + 1)*2*2 + 1*2 + 0)*4 + 1 = 89; its V zero (s = 5: 16*(5/4) + 4*1 + 1 = 21)
    at ((1*2 + 1)*4 + 1)*8 + 5 = 109."""
    assert LY.g64_kmeta_index(128)[0, 21, 1] == 89
    assert LY.g64_vmeta_index(128)[1, 21, 1] == 109


@pytest.mark.parametrize("bits", [2, 4, 8])
def test_groups_are_64_channels_of_one_token_brute_force(bits):
    """Loops over one block: each (token, 64-channel group) of K and V gets its own
    fp16 scale (max - min)/(2^b - 1) and zero (the minimum); dequantised values are
    u s + z within s/2 of the input; a spike at channel 64 of one token changes only
    that token's second group."""
    D = 128
    rng = np.random.default_rng(40 + bits)
    K = rng.standard_normal((1, 1, 32, D)).astype(np.float32)
    V = rng.standard_normal((1, 1, 32, D)).astype(np.float32)
    dims = _dims(D)
    Kh, Vh = C.dequant_layer(dims, [P.Action(bits=bits)], C.compress_layer(dims, bits, K, V), 0, 32)
    for X, Xh in ((K, Kh), (V, Vh)):
        for t in range(32):
            for g in range(2):
                grp = [float(X[0, 0, t, c]) for c in range(64 * g, 64 * g + 64)]
                mn, mx = min(grp), max(grp)
                s = float(np.float16(np.float32(np.float32(mx) - np.float32(mn)) / np.float32(2 ** bits - 1)))
                z = float(np.float16(mn))
                for c in range(64):
                    xh = float(Xh[0, 0, t, 64 * g + c])
                    u = (xh - z) / s
                    assert u == round(u) and 0 <= u <= 2 ** bits - 1
                    if z <= grp[c] <= z + s * (2 ** bits - 1):
                        assert abs(grp[c] - xh) <= s / 2 * (1 + 1e-6)
    K2 = K.copy()
    K2[0, 0, 7, 64] = 50.0
    K2h, _ = C.dequant_layer(dims, [P.Action(bits=bits)], C.compress_layer(dims, bits, K2, V), 0, 32)
    diff = np.argwhere(K2h[0, 0] != Kh[0, 0])
    assert diff.size and set(map(tuple, diff[:, :1].tolist())) == {(7,)} and diff[:, 1].min() >= 64


def test_only_gqa_with_64_channel_multiples():
    assert P.validate(P.Dims(P.GQA, 1, 2, 1, 96, qscheme=P.GROUP64), [P.Action(bits=4)]) is not None
    assert P.validate(_dims(64), [P.Action(bits=4)]) is None
