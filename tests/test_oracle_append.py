"""Pins of the oracle's decode-time append (oracle.cache.append_token,
oracle.mla.append_token).

The append rule (new token into the bf16 tail; the token that fills the tail
completes a 32-token group, quantised into the next full block) has one checkable
consequence that does not depend on how either side is written: appending tokens
one at a time to a stream must give the same stored tokens as writing the whole
sequence at prefill, once the inputs are bf16 values (the tail's precision).  The
one-shot write is pinned by the quantiser and layout pins; here both paths run on
the same tokens and must agree byte for byte on every full block and on every
valid tail token, for every bit-width and both schemes, starting from an empty
stream, from a ragged tail and from a block boundary.
"""
import numpy as np
import pytest

from oracle import cache as OC
from oracle import layout as LY
from oracle import mla as OM
from oracle import plan as P
from oracle import quant as Q


def _bf16_rows(rng, n, w, outliers=True):
    x = rng.standard_normal((n, w)).astype(np.float32)
    if outliers:
        x *= np.exp(rng.standard_normal(w)).astype(np.float32)[None, :]
    return Q.round_bf16(x)


def _gqa_stored(dims, bits, stream, n):
    """(full blocks, valid tail tokens K, V) of a GQA stream holding n tokens."""
    blocks, tail = LY.split_stream(dims, bits, stream, n)
    kt, vt = LY.unpack_bf16_blocks(tail[None], dims.head_dim)
    nt = n % P.GROUP
    return blocks.copy(), kt[0, :nt].copy(), vt[0, :nt].copy()


@pytest.mark.parametrize("qs", [P.KIVI32, P.SYMROW], ids=["kivi32", "symrow"])
@pytest.mark.parametrize("bits", [2, 4, 8, 16])
@pytest.mark.parametrize("n0", [0, 7, 32])
def test_gqa_append_equals_prefill_write(qs, bits, n0):
    D, n1 = 64, 70
    dims = P.Dims(P.GQA, 1, 2, 1, D, qscheme=qs, batch=1, max_tokens=96)
    rng = np.random.default_rng(1000 + 10 * bits + n0 + qs)
    K, V = _bf16_rows(rng, n1, D), _bf16_rows(rng, n1, D, outliers=False)
    stream = OC.compress_stream(dims, bits, K[:n0], V[:n0])
    for n in range(n0, n1):
        stream = OC.append_token(dims, bits, stream, n, K[n], V[n])
        if n + 1 in (n0 + 1, 32, 33, 64, n1):
            ref = OC.compress_stream(dims, bits, K[:n + 1], V[:n + 1])
            for got, want in zip(_gqa_stored(dims, bits, stream, n + 1), _gqa_stored(dims, bits, ref, n + 1)):
                assert np.array_equal(got, want), f"differs after appending token {n}"
    Kh, Vh = OC.dequant_stream(dims, bits, stream, n1)
    Kr, Vr = OC.dequant_stream(dims, bits, OC.compress_stream(dims, bits, K, V), n1)
    assert np.array_equal(Kh, Kr) and np.array_equal(Vh, Vr)


def test_gqa_append_rounds_fp32_input_to_bf16():
    """fp32 tokens are stored as their bf16 values: appending x equals appending
    bf16(x), and a completed group equals the prefill write of the bf16 values."""
    D = 64
    dims = P.Dims(P.GQA, 1, 2, 1, D, batch=1, max_tokens=64)
    rng = np.random.default_rng(7)
    K = rng.standard_normal((32, D)).astype(np.float32)
    V = rng.standard_normal((32, D)).astype(np.float32)
    s32 = OC.compress_stream(dims, 4, K[:0], V[:0])
    s16 = s32.copy()
    for n in range(32):
        s32 = OC.append_token(dims, 4, s32, n, K[n], V[n])
        s16 = OC.append_token(dims, 4, s16, n, Q.round_bf16(K[n]), Q.round_bf16(V[n]))
    assert np.array_equal(s32, s16)
    ref = OC.compress_stream(dims, 4, Q.round_bf16(K), Q.round_bf16(V))
    assert np.array_equal(_gqa_stored(dims, 4, s32, 32)[0], _gqa_stored(dims, 4, ref, 32)[0])


def test_gqa_append_flush_writes_only_its_block():
    """The token that completes a group changes block n // 32 and nothing before it."""
    D, bits = 64, 2
    dims = P.Dims(P.GQA, 1, 2, 1, D, batch=1, max_tokens=96)
    rng = np.random.default_rng(11)
    K, V = _bf16_rows(rng, 64, D), _bf16_rows(rng, 64, D)
    s = OC.compress_stream(dims, bits, K[:63], V[:63])
    s2 = OC.append_token(dims, bits, s, 63, K[63], V[63])
    blk = P.block_bytes(dims, bits)
    assert np.array_equal(s2[:blk], s[:blk])
    assert not np.array_equal(s2[blk:2 * blk], s[blk:2 * blk])


def _mla_dims(qs, d_max=128):
    return P.Dims(P.MLA, 1, 4, 1, 128, latent_dim=d_max, rope_dim=64, nope_dim=16, v_dim=8,
                  qscheme=qs, batch=1, max_tokens=96)


def _mla_stored(dims, bits, d, stream, n):
    W = d + dims.rope_dim
    blk = P.block_bytes(dims, bits, d)
    nb = n // P.GROUP
    t0 = (dims.stored_cap // P.GROUP) * blk
    tail = OM.unpack_bf16_block(stream[None, t0:t0 + P.tail_bytes(dims, d)], W)[0]
    return stream[:nb * blk].copy(), tail[:n % P.GROUP].copy()


@pytest.mark.parametrize("qs", [P.KIVI32, P.SYMROW], ids=["kivi32", "symrow"])
@pytest.mark.parametrize("bits", [2, 4, 8, 16])
@pytest.mark.parametrize("d", [128, 64])
def test_mla_append_equals_prefill_write(qs, bits, d):
    dims = _mla_dims(qs)
    rng = np.random.default_rng(2000 + bits + d + qs)
    n0, n1 = 5, 69
    C, R = _bf16_rows(rng, n1, dims.latent_dim, outliers=False), _bf16_rows(rng, n1, 64, outliers=False)
    stream = OM.compress_stream(dims, bits, d, C[:n0], R[:n0])
    for n in range(n0, n1):
        stream = OM.append_token(dims, bits, d, stream, n, C[n], R[n])
        if n + 1 in (6, 32, 33, 64, n1):
            ref = OM.compress_stream(dims, bits, d, C[:n + 1], R[:n + 1])
            for got, want in zip(_mla_stored(dims, bits, d, stream, n + 1), _mla_stored(dims, bits, d, ref, n + 1)):
                assert np.array_equal(got, want), f"differs after appending token {n}"
    Ch, Rh = OM.dequant_stream(dims, bits, d, stream, n1)
    Cr, Rr = OM.dequant_stream(dims, bits, d, OM.compress_stream(dims, bits, d, C, R), n1)
    assert np.array_equal(Ch, Cr) and np.array_equal(Rh, Rr)
