"""Cache quantisers of App. C.3 (oracle).

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

Three schemes:
  * SYMROW — the paper's own quantiser (App. B "Quantization", App. C.3):
    symmetric, one scale per stored vector set by its largest magnitude,
    q = 2^(b-1) - 1, s = max|x| / q, code = clip(round(x / s), -q, q),
    x_hat = code * s.  The scale is held in bf16, one per 128-element
    token-head row (the App. C.3 table caption).
  * KIVI32 — the grouped asymmetric quantiser App. C.3 contrasts it with: a
    scale and a zero point per group, all 2^b levels.  Groups: keys per channel
    over 32 consecutive stored tokens, values per token over 32 consecutive
    channels; scale and zero in fp16.
  * GROUP64 — the same grouped asymmetric quantiser with per-token groups of 64
    consecutive channels for keys and values alike (App. C.3's on-device grouped
    cache: 4 + 32/64 = 4.5 bits per element at 4 bits, 3.56x); kivi_quantize over
    such groups.

Readings where the paper is silent: rounding is
round-half-to-even; the scale is rounded to its storage type before codes are
computed; the zero point is the fp16 of the group minimum; a group with a zero
scale gets code 0 (so x_hat = zero, or 0 for SYMROW); the arithmetic is the fp32
chain written below.

Pins: closed forms for ramps and constant groups, the three levels of 2-bit
SYMROW, the |x - x_hat| <= s/2 bound for unclipped values, idempotent
re-quantisation, and the bf16/fp16 roundings against torch's conversions.
"""
import numpy as np

F32 = np.float32


def bf16_bits(x) -> np.ndarray:
    """Round fp32 values to bf16 (round-to-nearest-even), returning the 16-bit
    patterns.  NaN maps to the canonical quiet NaN."""
    x = np.asarray(x, dtype=F32)
    b = x.view(np.uint32).astype(np.uint64)
    r = (b + 0x7FFF + ((b >> 16) & 1)) >> 16
    r = np.where(np.isnan(x), 0x7FC0, r)
    return r.astype(np.uint16)


def bf16_value(bits16) -> np.ndarray:
    """fp32 value of bf16 bit patterns (exact)."""
    return (np.asarray(bits16, dtype=np.uint16).astype(np.uint32) << 16).view(F32)


def round_bf16(x) -> np.ndarray:
    return bf16_value(bf16_bits(x))


def f16(x) -> np.ndarray:
    """Round fp32 values to fp16 (numpy's conversion rounds to nearest even)."""
    return np.asarray(x, dtype=F32).astype(np.float16)


def kivi_quantize(x: np.ndarray, bits: int):
    """Grouped asymmetric quantisation along the last axis (one group per row).

    Returns (u, scale16, zero16): integer codes in [0, 2^b - 1] (int64), and the
    fp16 scale and zero of each group.  All arithmetic is fp32 as in the chain
    mn = min x, mx = max x, s = fp16((mx - mn) / (2^b - 1)), z = fp16(mn),
    u = clamp(rint((x - z) / s), 0, 2^b - 1), or 0 where s == 0."""
    x = np.asarray(x, dtype=F32)
    levels = F32(2 ** bits - 1)
    mn = x.min(axis=-1)
    mx = x.max(axis=-1)
    s16 = f16((mx - mn) / levels)
    z16 = f16(mn)
    s = s16.astype(F32)[..., None]
    z = z16.astype(F32)[..., None]
    with np.errstate(divide="ignore", invalid="ignore"):
        t = (x - z) / s
    u = np.clip(np.rint(t), F32(0), levels)
    u = np.where(s == 0, F32(0), u)
    return u.astype(np.int64), s16, z16


def kivi_dequantize(u, scale16, zero16) -> np.ndarray:
    """x_hat = fmaf(u, s, z): the exact u*s + z (exact in fp64 for fp16 s, z and
    u < 2^8) rounded once to fp32.  scale16/zero16 broadcast against u."""
    s = np.asarray(scale16, dtype=np.float16).astype(np.float64)
    z = np.asarray(zero16, dtype=np.float16).astype(np.float64)
    return (np.asarray(u, dtype=np.float64) * s + z).astype(F32)


def symrow_quantize(x: np.ndarray, bits: int):
    """Symmetric quantisation along the last axis (one row per scale).

    Returns (u, scale_bf16_bits): stored codes u = code + 2^(b-1) (int64) and the
    bf16 bit pattern of each row's scale.  s = bf16(max|x| / q) in fp32;
    code = clamp(rint(x / s), -q, q), or 0 where s == 0."""
    x = np.asarray(x, dtype=F32)
    q = F32(2 ** (bits - 1) - 1)
    amax = np.abs(x).max(axis=-1)
    sb = bf16_bits(amax / q)
    s = bf16_value(sb)[..., None]
    with np.errstate(divide="ignore", invalid="ignore"):
        t = x / s
    code = np.clip(np.rint(t), -q, q)
    code = np.where(s == 0, F32(0), code)
    return code.astype(np.int64) + 2 ** (bits - 1), sb


def symrow_dequantize(u, scale_bits, bits: int) -> np.ndarray:
    """x_hat = code * s with code = u - 2^(b-1); exact in fp32 (|code| < 2^7 and
    s has 8 significant bits)."""
    s = bf16_value(scale_bits).astype(np.float64)
    code = np.asarray(u, dtype=np.int64) - 2 ** (bits - 1)
    return (code.astype(np.float64) * s).astype(F32)
