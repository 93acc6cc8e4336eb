"""Arena byte layout of one (sequence, KV head) stream (oracle).

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

This is the storage layout documented in include/kvk.h, restated from its text:
the paper fixes what is stored per token (codes, scale, zero point, §2.1 and
App. C.3) but not where; the library chooses the order so that its decode kernel
loads each lane's operands with wide contiguous loads.  The oracle writes and
reads the bytes through explicit (token, channel) -> address maps built by
enumerating the header's slot rules, so that the two sides agree only through
the documented layout.

Pins: every map is a bijection onto the region it describes (no two values share
a bit, no bit is left over), pack/unpack round-trips every code value of every
bit-width, and the block sizes give the App. C.3 bits-per-element figures.
"""
from functools import lru_cache

import numpy as np

from .plan import GROUP, GROUP64, KIVI32, SYMROW, Dims, block_bytes, stream_bytes, tail_bytes


def _lanes():
    for lam in range(64):
        yield lam, lam // 16, lam % 16


@lru_cache(maxsize=None)
def k_slots(D: int):
    """K slot map: lane lam=16kg+i, tile tau, sub-chunk j, slot s -> token
    16 tau + i, channel 32 j + 8 kg + s.  Returns a list of tuples
    (tau, lam, j, s, token, channel)."""
    out = []
    for tau in range(2):
        for lam, kg, i in _lanes():
            for j in range(D // 32):
                for s in range(8):
                    out.append((tau, lam, j, s, 16 * tau + i, 32 * j + 8 * kg + s))
    return out


@lru_cache(maxsize=None)
def v_slots(D: int):
    """V slot map: lane lam=16kg+i, tile m, slot s -> channel 16 m + i, token
    16 (s/4) + 4 kg + (s%4).  Returns tuples (lam, m, s, token, channel)."""
    out = []
    for lam, kg, i in _lanes():
        for m in range(D // 16):
            for s in range(8):
                out.append((lam, m, s, 16 * (s // 4) + 4 * kg + (s % 4), 16 * m + i))
    return out


def part_byte(P: int, lam: int, o: int) -> int:
    """Byte of a part that holds byte o of lane lam's P-byte share: shares longer
    than 16 bytes are dealt to the 64 lanes in 16-byte pieces (piece o // 16 of
    every lane, in lane order, then the next piece); shorter shares are stored
    one lane after another."""
    if P > 16:
        return 1024 * (o // 16) + 16 * lam + o % 16
    return lam * P + o


def _bit_in_chunk(bits: int, x: int, s: int) -> int:
    """Bit offset of slot s relative to the start of its chunk's 32-bit word (or
    of the chunk for b = 8), chunk index x (j or m)."""
    if bits == 8:
        return 8 * s
    if bits == 4:
        return 16 * (s % 2) + 4 * (s // 2)
    if bits == 2:
        return 16 * (s % 2) + 2 * (s // 2) + 8 * (x % 2)
    raise ValueError(bits)


@lru_cache(maxsize=None)
def code_bitaddr(D: int, bits: int):
    """Bit addresses (from the block start) of every K and V code: two int64
    arrays [32 tokens, D channels]."""
    kaddr = np.full((32, D), -1, dtype=np.int64)
    for tau, lam, j, s, t, c in k_slots(D):
        chunk = 2 * D * bits * tau + part_byte(D * bits // 32, lam, j * bits)
        word = chunk - (j % 2) * bits if bits == 2 else chunk
        kaddr[t, c] = 8 * word + _bit_in_chunk(bits, j, s)
    vaddr = np.full((32, D), -1, dtype=np.int64)
    vbase = 4 * D * bits
    for lam, m, s, t, c in v_slots(D):
        chunk = vbase + part_byte(D * bits // 16, lam, m * bits)
        word = chunk - (m % 2) * bits if bits == 2 else chunk
        vaddr[t, c] = 8 * word + _bit_in_chunk(bits, m, s)
    return kaddr, vaddr


@lru_cache(maxsize=None)
def bf16_byteaddr(D: int):
    """Byte addresses of every K and V bf16 value of a bf16 block: [32, D] each."""
    kaddr = np.full((32, D), -1, dtype=np.int64)
    for tau, lam, j, s, t, c in k_slots(D):
        kaddr[t, c] = 32 * D * tau + part_byte(D // 2, lam, 16 * j + 2 * s)
    vaddr = np.full((32, D), -1, dtype=np.int64)
    for lam, m, s, t, c in v_slots(D):
        vaddr[t, c] = 64 * D + part_byte(D, lam, 16 * m + 2 * s)
    return kaddr, vaddr


@lru_cache(maxsize=None)
def kivi_vmeta_index(D: int):
    """V-meta fp16 index for (w, token, group): ((g*2 + w)*4 + kg)*8 + s where
    token = 16 (s/4) + 4 kg + (s%4).  Returns int64 [2, 32, D/32]."""
    idx = np.full((2, 32, D // 32), -1, dtype=np.int64)
    for g in range(D // 32):
        for w in range(2):
            for kg in range(4):
                for s in range(8):
                    t = 16 * (s // 4) + 4 * kg + (s % 4)
                    idx[w, t, g] = ((g * 2 + w) * 4 + kg) * 8 + s
    return idx


def g64_kmeta_index(D: int):
    """GROUP64 K-meta fp16 index for (w, token, group): ((tau*4 + kg)*NG*2 + g*2 + w)*4 + e
    where token = 16 tau + 4 kg + e and NG = D/64.  Returns int64 [2, 32, NG]."""
    NG = D // 64
    idx = np.full((2, 32, NG), -1, dtype=np.int64)
    for tau in range(2):
        for kg in range(4):
            for g in range(NG):
                for w in range(2):
                    for e in range(4):
                        idx[w, 16 * tau + 4 * kg + e, g] = ((tau * 4 + kg) * NG * 2 + g * 2 + w) * 4 + e
    return idx


def g64_vmeta_index(D: int):
    """GROUP64 V-meta fp16 index for (w, token, group): ((g*2 + w)*4 + kg)*8 + s where
    token = 16 (s/4) + 4 kg + (s%4), g over the D/64 groups.  Returns int64 [2, 32, D/64]."""
    idx = np.full((2, 32, D // 64), -1, dtype=np.int64)
    for g in range(D // 64):
        for w in range(2):
            for kg in range(4):
                for s in range(8):
                    t = 16 * (s // 4) + 4 * kg + (s % 4)
                    idx[w, t, g] = ((g * 2 + w) * 4 + kg) * 8 + s
    return idx


def _pack_bits(u: np.ndarray, addr: np.ndarray, bits: int, nbytes: int) -> np.ndarray:
    """Scatter codes u [n, 32, D] to bit addresses addr [32, D] of n regions of
    nbytes bytes each; returns uint8 [n, nbytes]."""
    n = u.shape[0]
    nwords = nbytes // 4
    flat_addr = addr.reshape(-1)
    word = flat_addr // 32
    shift = (flat_addr % 32).astype(np.uint64)
    vals = u.reshape(n, flat_addr.size).astype(np.uint64) << shift
    order = np.argsort(word, kind="stable")
    per = 32 // bits
    assert np.array_equal(word[order], np.repeat(np.arange(nwords), per)), "layout not dense"
    words = vals[:, order].reshape(n, nwords, per).sum(axis=-1)
    return np.ascontiguousarray(words.astype(np.uint32)).view(np.uint8).reshape(n, nbytes)


def _unpack_bits(raw: np.ndarray, addr: np.ndarray, bits: int) -> np.ndarray:
    """Inverse of _pack_bits: raw uint8 [n, nbytes] -> codes int64 [n, 32, D]."""
    n = raw.shape[0]
    words = np.ascontiguousarray(raw).view(np.uint32).reshape(n, raw.shape[1] // 4).astype(np.int64)
    flat_addr = addr.reshape(-1)
    vals = (words[:, flat_addr // 32] >> (flat_addr % 32)) & ((1 << bits) - 1)
    return vals.reshape(n, *addr.shape)


def _put_u16(region: np.ndarray, byte_addr: np.ndarray, vals: np.ndarray):
    """region uint8 [n, R]; write uint16 vals [n, ...] at byte addresses [...]."""
    a = byte_addr.reshape(-1)
    v = vals.reshape(vals.shape[0], a.size).astype(np.uint16)
    region[:, a] = (v & 0xFF).astype(np.uint8)
    region[:, a + 1] = (v >> 8).astype(np.uint8)


def _get_u16(region: np.ndarray, byte_addr: np.ndarray) -> np.ndarray:
    a = byte_addr.reshape(-1)
    v = region[:, a].astype(np.uint16) | (region[:, a + 1].astype(np.uint16) << 8)
    return v.reshape(region.shape[0], *byte_addr.shape)


# ---------------------------------------------------------------------------
# Blocks
# ---------------------------------------------------------------------------

def pack_bf16_blocks(kb: np.ndarray, vb: np.ndarray) -> np.ndarray:
    """kb, vb: uint16 bf16 patterns [n, 32, D] -> uint8 [n, 128 D]."""
    n, _, D = kb.shape
    out = np.zeros((n, 128 * D), dtype=np.uint8)
    ka, va = bf16_byteaddr(D)
    _put_u16(out, ka, kb)
    _put_u16(out, va, vb)
    return out


def unpack_bf16_blocks(raw: np.ndarray, D: int):
    ka, va = bf16_byteaddr(D)
    return _get_u16(raw, ka), _get_u16(raw, va)


def pack_quant_blocks(dims: Dims, bits: int, f: dict) -> np.ndarray:
    """Quantised blocks.  f holds 'uk', 'uv' int [n, 32, D] and, for KIVI32,
    'ks', 'kz' fp16 [n, D], 'vs', 'vz' fp16 [n, 32, D/32]; for GROUP64, 'ks', 'kz',
    'vs', 'vz' fp16 [n, 32, D/64]; for SYMROW, 'ks', 'vs' bf16 bit patterns uint16
    [n, 32]."""
    D = dims.head_dim
    n = f["uk"].shape[0]
    out = np.zeros((n, block_bytes(dims, bits)), dtype=np.uint8)
    ka, va = code_bitaddr(D, bits)
    cb = 4 * D * bits
    out[:, :cb] = _pack_bits(f["uk"], ka, bits, cb)
    out[:, cb:2 * cb] = _pack_bits(f["uv"], va - 8 * cb, bits, cb)
    mb = 2 * cb
    if dims.qscheme == KIVI32:
        ch = np.arange(D)
        _put_u16(out, mb + 2 * ch, f["ks"].view(np.uint16))
        _put_u16(out, mb + 2 * D + 2 * ch, f["kz"].view(np.uint16))
        vi = kivi_vmeta_index(D)
        _put_u16(out, mb + 4 * D + 2 * vi[0], f["vs"].view(np.uint16))
        _put_u16(out, mb + 4 * D + 2 * vi[1], f["vz"].view(np.uint16))
    elif dims.qscheme == GROUP64:
        ki, vi = g64_kmeta_index(D), g64_vmeta_index(D)
        _put_u16(out, mb + 2 * ki[0], f["ks"].view(np.uint16))
        _put_u16(out, mb + 2 * ki[1], f["kz"].view(np.uint16))
        _put_u16(out, mb + 2 * D + 2 * vi[0], f["vs"].view(np.uint16))
        _put_u16(out, mb + 2 * D + 2 * vi[1], f["vz"].view(np.uint16))
    else:
        t = np.arange(32)
        _put_u16(out, mb + 2 * t, f["ks"])
        _put_u16(out, mb + 64 + 2 * t, f["vs"])
    return out


def unpack_quant_blocks(dims: Dims, bits: int, raw: np.ndarray) -> dict:
    D = dims.head_dim
    ka, va = code_bitaddr(D, bits)
    cb = 4 * D * bits
    f = {"uk": _unpack_bits(raw[:, :cb], ka, bits),
         "uv": _unpack_bits(raw[:, cb:2 * cb], va - 8 * cb, bits)}
    mb = 2 * cb
    if dims.qscheme == KIVI32:
        ch = np.arange(D)
        f["ks"] = _get_u16(raw, mb + 2 * ch).view(np.float16)
        f["kz"] = _get_u16(raw, mb + 2 * D + 2 * ch).view(np.float16)
        vi = kivi_vmeta_index(D)
        f["vs"] = _get_u16(raw, mb + 4 * D + 2 * vi[0]).view(np.float16)
        f["vz"] = _get_u16(raw, mb + 4 * D + 2 * vi[1]).view(np.float16)
    elif dims.qscheme == GROUP64:
        ki, vi = g64_kmeta_index(D), g64_vmeta_index(D)
        f["ks"] = _get_u16(raw, mb + 2 * ki[0]).view(np.float16)
        f["kz"] = _get_u16(raw, mb + 2 * ki[1]).view(np.float16)
        f["vs"] = _get_u16(raw, mb + 2 * D + 2 * vi[0]).view(np.float16)
        f["vz"] = _get_u16(raw, mb + 2 * D + 2 * vi[1]).view(np.float16)
    else:
        t = np.arange(32)
        f["ks"] = _get_u16(raw, mb + 2 * t)
        f["vs"] = _get_u16(raw, mb + 64 + 2 * t)
    return f


# ---------------------------------------------------------------------------
# Streams
# ---------------------------------------------------------------------------

def assemble_stream(dims: Dims, bits: int, blocks: np.ndarray, tail: np.ndarray) -> np.ndarray:
    """Concatenate full blocks [nb, blk] and the bf16 tail block [128 D] into a
    stream of stream_bytes, zero-padded (unused blocks and padding are zero)."""
    sb = stream_bytes(dims, bits)
    out = np.zeros(sb, dtype=np.uint8)
    blk = block_bytes(dims, bits)
    nb = blocks.shape[0]
    out[:nb * blk] = blocks.reshape(-1)
    cap_blocks = dims.stored_cap // GROUP
    t0 = cap_blocks * blk
    out[t0:t0 + tail_bytes(dims)] = tail
    return out


def split_stream(dims: Dims, bits: int, stream: np.ndarray, n_stored: int):
    """Return (full blocks uint8 [n_stored//32, blk], tail block uint8 [128 D])."""
    blk = block_bytes(dims, bits)
    nb = n_stored // GROUP
    blocks = stream[:nb * blk].reshape(nb, blk)
    t0 = (dims.stored_cap // GROUP) * blk
    return blocks, stream[t0:t0 + tail_bytes(dims)]


__all__ = [
    "k_slots", "v_slots", "code_bitaddr", "bf16_byteaddr", "kivi_vmeta_index", "g64_kmeta_index",
    "g64_vmeta_index",
    "pack_bf16_blocks", "unpack_bf16_blocks", "pack_quant_blocks", "unpack_quant_blocks",
    "assemble_stream", "split_stream", "SYMROW",
]
