"""Pins of the oracle's quantisers (App. C.3) and arena layout."""
import os

import numpy as np
import pytest
import torch

from oracle import layout as LY
from oracle import plan as P
from oracle import quant as Q

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _special_f32(rng, n):
    x = (rng.standard_normal(n) * 10.0 ** rng.integers(-6, 4, n)).astype(np.float32)
    # force exact bf16 ties (low 16 bits 0x8000) and fp16 ties on a share of the values
    bits = x.view(np.uint32).copy()
    bits[: n // 4] = (bits[: n // 4] & 0xFFFF0000) | 0x8000
    return bits.view(np.float32)


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    x = _special_f32(rng, 20000)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(Q.bf16_bits(x), ref)


def test_f16_rounding_matches_torch():
    rng = np.random.default_rng(1)
    x = rng.standard_normal(20000).astype(np.float32) * np.float32(100)
    x[:5000] = (np.rint(x[:5000] * 2048) + 0.5) / 2048  # ties at the fp16 spacing near 1..2
    ref = torch.from_numpy(x).to(torch.float16).numpy()
    assert np.array_equal(Q.f16(x).view(np.uint16), ref.view(np.uint16))


def test_kivi_ramp_closed_form():
    """A ramp 0..31 at 4 bits: zero 0, scale fp16(31/15), codes rint(x/scale),
    every one of the 16 levels used."""
    x = np.arange(32, dtype=np.float32)[None]
    u, s, z = Q.kivi_quantize(x, 4)
    assert float(z[0]) == 0.0
    assert s[0] == np.float16(31.0 / 15.0)
    assert np.array_equal(u[0], np.rint(x[0] / np.float32(s[0])).astype(np.int64))
    assert set(u[0].tolist()) == set(range(16))


def test_kivi_constant_group():
    """A constant group has scale 0: codes 0 and x_hat = zero = fp16(c)."""
    x = np.full((3, 32), np.float32(0.3))
    u, s, z = Q.kivi_quantize(x, 2)
    assert np.all(u == 0) and np.all(s == 0)
    xh = Q.kivi_dequantize(u, s[:, None], z[:, None])
    assert np.all(xh == np.float32(np.float16(0.3)))


@pytest.mark.parametrize("bits", [2, 4, 8])
def test_kivi_error_bound(bits):
    """|x - x_hat| <= s/2 + |min - zero| + (2^b - 1)|s_exact - s| + fp32 rounding."""
    rng = np.random.default_rng(bits)
    x = (rng.standard_normal((4000, 32)) * np.exp(rng.standard_normal((4000, 1)))).astype(np.float32)
    u, s, z = Q.kivi_quantize(x, bits)
    xh = Q.kivi_dequantize(u, s[:, None], z[:, None]).astype(np.float64)
    mn, mx = x.min(1).astype(np.float64), x.max(1).astype(np.float64)
    s64 = s.astype(np.float64)
    exact = (mx - mn) / (2 ** bits - 1)
    bound = s64 / 2 + np.abs(mn - z.astype(np.float64)) + (2 ** bits - 1) * np.abs(exact - s64)
    err = np.abs(x.astype(np.float64) - xh)
    assert np.all(err <= bound[:, None] * (1 + 1e-6) + 1e-6 * np.abs(x))
    assert u.min() >= 0 and u.max() <= 2 ** bits - 1


@pytest.mark.parametrize("bits", [2, 4, 8])
def test_kivi_idempotent_given_metadata(bits):
    """Re-quantising x_hat with the same scale and zero returns the same codes."""
    rng = np.random.default_rng(10 + bits)
    x = rng.standard_normal((2000, 32)).astype(np.float32)
    u, s, z = Q.kivi_quantize(x, bits)
    xh = Q.kivi_dequantize(u, s[:, None], z[:, None])
    sf, zf = s.astype(np.float32)[:, None], z.astype(np.float32)[:, None]
    u2 = np.clip(np.rint((xh - zf) / sf), 0, 2 ** bits - 1).astype(np.int64)
    assert np.array_equal(u, u2)
    # a full re-quantisation (new min/max) reproduces codes and metadata
    u3, s3, z3 = Q.kivi_quantize(xh, bits)
    assert np.array_equal(u3, u) and np.array_equal(s3, s) and np.array_equal(z3, z)


def test_symrow_two_bit_has_three_levels():
    """App. C.3: at two bits the symmetric quantiser has three levels."""
    rng = np.random.default_rng(3)
    x = rng.standard_normal((500, 128)).astype(np.float32)
    u, sb = Q.symrow_quantize(x, 2)
    assert set(np.unique(u).tolist()) == {1, 2, 3}
    xh = Q.symrow_dequantize(u, sb[:, None], 2)
    for r in range(50):
        assert len(np.unique(xh[r])) <= 3
    # the largest magnitude maps to +-1 * s, s = bf16(max|x|)
    i = np.abs(x).argmax(1)
    s = Q.bf16_value(sb)
    assert np.all(np.abs(xh[np.arange(500), i]) == s)


@pytest.mark.parametrize("bits", [2, 4, 8])
def test_symrow_idempotent_and_bound(bits):
    rng = np.random.default_rng(20 + bits)
    x = (rng.standard_normal((1000, 128)) * 3).astype(np.float32)
    u, sb = Q.symrow_quantize(x, bits)
    xh = Q.symrow_dequantize(u, sb[:, None], bits)
    u2, sb2 = Q.symrow_quantize(xh, bits)
    assert np.array_equal(u, u2) and np.array_equal(sb, sb2)
    q = 2 ** (bits - 1) - 1
    s = Q.bf16_value(sb).astype(np.float64)[:, None]
    amax = np.abs(x).max(1, keepdims=True).astype(np.float64)
    bound = s / 2 + q * np.abs(amax / q - s)  # bf16 rounding of the scale may clip the max
    assert np.all(np.abs(x - xh.astype(np.float64)) <= bound * (1 + 1e-6))
    assert u.min() >= 1 and u.max() <= 2 ** bits - 1


def test_symrow_zero_row():
    u, sb = Q.symrow_quantize(np.zeros((2, 128), np.float32), 4)
    assert np.all(u == 8) and np.all(sb == 0)


# ---------------------------------------------------------------------------
# layout
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("D", [64, 128])
@pytest.mark.parametrize("bits", [2, 4, 8])
def test_code_maps_are_bijections(D, bits):
    ka, va = LY.code_bitaddr(D, bits)
    cb = 4 * D * bits * 8  # bits of one code region
    assert np.array_equal(np.sort(ka.ravel()), np.arange(0, cb, bits))
    assert np.array_equal(np.sort(va.ravel()), np.arange(cb, 2 * cb, bits))


@pytest.mark.parametrize("D", [64, 128])
def test_bf16_maps_and_vmeta_are_bijections(D):
    ka, va = LY.bf16_byteaddr(D)
    assert np.array_equal(np.sort(ka.ravel()), np.arange(0, 64 * D, 2))
    assert np.array_equal(np.sort(va.ravel()), np.arange(64 * D, 128 * D, 2))
    vi = LY.kivi_vmeta_index(D)
    assert np.array_equal(np.sort(vi.ravel()), np.arange(2 * D))


def test_layout_examples_worked_by_hand():
    with open(os.path.join(GOLD, "layout_examples.txt")) as f:
        rows = [ln.split() for ln in f if ln.strip() and not ln.startswith("#")]
    assert rows
    for D, b, which, t, c, addr in rows:
        ka, va = LY.code_bitaddr(int(D), int(b))
        got = (ka if which == "K" else va)[int(t), int(c)]
        assert got == int(addr), (D, b, which, t, c)


@pytest.mark.parametrize("qs", [P.KIVI32, P.SYMROW, P.GROUP64])
@pytest.mark.parametrize("D", [64, 128])
@pytest.mark.parametrize("bits", [2, 4, 8])
def test_pack_unpack_roundtrip_all_codes(qs, D, bits):
    rng = np.random.default_rng(bits * D)
    dims = P.Dims(P.GQA, 1, 1, 1, D, qscheme=qs)
    n = 3
    f = {"uk": rng.integers(0, 2 ** bits, (n, 32, D)), "uv": rng.integers(0, 2 ** bits, (n, 32, D))}
    f["uk"][0].flat[: 2 ** bits] = np.arange(2 ** bits)  # every code value appears
    if qs == P.KIVI32:
        f.update(ks=rng.standard_normal((n, D)).astype(np.float16),
                 kz=rng.standard_normal((n, D)).astype(np.float16),
                 vs=rng.standard_normal((n, 32, D // 32)).astype(np.float16),
                 vz=rng.standard_normal((n, 32, D // 32)).astype(np.float16))
    elif qs == P.GROUP64:
        f.update({k: rng.standard_normal((n, 32, D // 64)).astype(np.float16) for k in ("ks", "kz", "vs", "vz")})
    else:
        f.update(ks=rng.integers(0, 2 ** 16, (n, 32)).astype(np.uint16),
                 vs=rng.integers(0, 2 ** 16, (n, 32)).astype(np.uint16))
    raw = LY.pack_quant_blocks(dims, bits, f)
    assert raw.shape == (n, P.block_bytes(dims, bits))
    g = LY.unpack_quant_blocks(dims, bits, raw)
    for key in f:
        assert np.array_equal(np.asarray(g[key]).view(np.uint16) if g[key].dtype == np.float16
                              else g[key], np.asarray(f[key]).view(np.uint16)
                              if f[key].dtype == np.float16 else f[key]), key
