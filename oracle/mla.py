"""The rank axis: MLA latent caches, their storage and their attention (oracle).

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

What an MLA layer stores (§2.1 "Rank", App. C.2): per token a latent c of width r,
shared by every head, and a positional key k^R of width d_R, held after RoPE.  A
layer that keeps width d stores only c[:d] (App. C.2: training zeroes the
coordinates after d with a prefix mask, a deployed kernel writes only the first
d).  Precision composes with rank (§2.2, eq. (1): cost (d + d_R) b):
  * KIVI32: the grouped asymmetric quantiser of App. C.3 with groups of 32
    consecutive stored channels of one token (the d latent coordinates followed
    by the d_R positional ones; d and d_R are multiples of 32);
  * SYMROW: the paper's own quantiser, one bf16 scale per stored vector, that is
    one for c[:d] and one for k^R of each token.
A layer at b = 16 stores the bf16 values.  The fp32 chains are those of
oracle/quant.py.

Attention (§2.1, App. C.2).  Head h has its own up-projections W_UK_h
[nope, r] and W_UV_h [v, r].  Its content key of token t is W_UK_h c_t, its
value W_UV_h c_t, its key the concatenation [W_UK_h c_t ; k^R_t], and its query
[q_nope_h ; q_rope_h].  The oracle attends with exactly these reconstructed keys
and values, the latent zero-padded beyond d.  Because the content key undergoes
no RoPE the projection can be moved onto the query (App. C.2); the absorbed form
is written out separately and agrees with the reconstruction to rounding, which
is one of the pins.

Storage layout: the one documented in include/kvk.h (MLA section), restated from
its text as explicit (token, channel) -> address maps: inside a block, bytes are
ordered by slots of 8 channels of one token, slot S = (T NK + K) 64 + i + 16 g for
token 16 T + i and channels 32 K + 8 g .. + 7.

Low-rank projection on write (§2.1 "Rank", App. C.2): the latent of a layer is the
down-projection of the token's hidden state, of which a layer keeping width d
computes and stores only the first d coordinates (project_latent); it is held in
bf16 and then written as any latent input.

Pins (tests/test_oracle_mla.py): absorbed == reconstructed; prefix mask ==
truncation; the projection: an identity map returns the hidden state's first d
coordinates, keeping d is the prefix of keeping r, brute-force sums on a tiny
input, single rounding to bf16 with ties to even, and the projected write equals
the latent-input write of the projected latent; a full-rank MLA whose up-projections select disjoint latent slices is
multi-head attention over those slices (checked against the GQA oracle); T = 1
gives W_UV c_0; q = 0 gives W_UV of the mean latent; the layout maps are
bijections; the quantiser closed forms; block sizes against eq. (1) plus the
stated metadata.
"""
from functools import lru_cache

import numpy as np

from . import attention as att
from . import quant
from .plan import (GROUP, KIVI32, MLA, Dims, anchor_of, arena_offsets, block_bytes, layer_bytes,
                   stored_width, stream_bytes, tail_bytes)

F32 = np.float32


# ---------------------------------------------------------------------------
# Layout of one 32-token block (include/kvk.h, MLA section)
# ---------------------------------------------------------------------------

def slot_index(W: int) -> np.ndarray:
    """Slot S of (token t, stored channel c) in a block: int64 [32, W].  With tile
    T = t // 16, row i = t % 16, k-step K = c // 32 (NK = W / 32 of them) and
    sub-group g = (c // 8) % 4:  S = (T NK + K) 64 + i + 16 g.  A slot holds 8
    consecutive channels c = 32 K + 8 g + s, s = c % 8."""
    NK = W // 32
    t = np.arange(32)[:, None]
    c = np.arange(W)[None, :]
    return (t // 16 * NK + c // 32) * 64 + t % 16 + 16 * (c // 8 % 4)


@lru_cache(maxsize=None)
def code_bitaddr(W: int, bits: int) -> np.ndarray:
    """Bit address, from the block start, of the code of (token t, stored channel
    c): int64 [32, W], on 32-bit little-endian words:
      b = 8: slot S fills words 2 S, 2 S + 1; position s at word 2 S + s // 4,
             bit 8 (s % 4);
      b = 4: slot S is word S; position s at bit 16 (s % 2) + 4 (s // 2);
      b = 2: sub-groups g = 2 y + x of (t, K) share word ((T NK + K) 16 + i) 2 + y;
             position s at bit 16 (s % 2) + 2 (s // 2) + 8 x."""
    NK = W // 32
    t = np.arange(32)[:, None]
    c = np.arange(W)[None, :]
    S = slot_index(W)
    s, g = c % 8, c // 8 % 4
    if bits == 8:
        word, bit = 2 * S + s // 4, 8 * (s % 4)
    elif bits == 4:
        word, bit = S, 16 * (s % 2) + 4 * (s // 2)
    else:
        word = ((t // 16 * NK + c // 32) * 16 + t % 16) * 2 + g // 2
        bit = 16 * (s % 2) + 2 * (s // 2) + 8 * (g % 2)
    return (32 * word + bit).astype(np.int64)


def kivi_meta_offset(W: int) -> np.ndarray:
    """Byte offset, from the start of the metadata, of the (scale, zero) pair of
    (token t, channel group K): int64 [32, W / 32] = 4 ((T NK + K) 16 + i)."""
    NK = W // 32
    t = np.arange(32)[:, None]
    K = np.arange(NK)[None, :]
    return 4 * ((t // 16 * NK + K) * 16 + t % 16)


def codes_bytes(W: int, bits: int) -> int:
    return 32 * W * bits // 8


def _pack(u: np.ndarray, addr: np.ndarray, bits: int, nbytes: int) -> np.ndarray:
    """Codes u [n, 32, W] -> uint8 [n, nbytes], each code placed at its bit
    address.  The map must cover every bit of the region exactly once."""
    n = u.shape[0]
    nwords = nbytes // 4
    flat = addr.reshape(-1)
    word = flat // 32
    vals = u.reshape(n, flat.size).astype(np.uint64) << (flat % 32).astype(np.uint64)
    order = np.argsort(word, kind="stable")
    per = 32 // bits
    assert np.array_equal(word[order], np.repeat(np.arange(nwords), per)), "layout not dense"
    words = vals[:, order].reshape(n, nwords, per).sum(axis=-1)  # disjoint bits: sum == or
    return np.ascontiguousarray(words.astype(np.uint32)).view(np.uint8).reshape(n, nbytes)


def _unpack(raw: np.ndarray, addr: np.ndarray, bits: int) -> np.ndarray:
    n = raw.shape[0]
    words = np.ascontiguousarray(raw).view(np.uint32).reshape(n, raw.shape[1] // 4).astype(np.int64)
    flat = addr.reshape(-1)
    return ((words[:, flat // 32] >> (flat % 32)) & ((1 << bits) - 1)).reshape(n, *addr.shape)


def _u16_put(region, byte_off, vals):
    v = np.asarray(vals).astype(np.uint16)
    region[..., byte_off] = (v & 0xFF).astype(np.uint8)
    region[..., byte_off + 1] = (v >> 8).astype(np.uint8)


def _u16_get(region, byte_off):
    return region[..., byte_off].astype(np.uint16) | (region[..., byte_off + 1].astype(np.uint16) << 8)


def _bf16_index(W: int) -> np.ndarray:
    """bf16 element index (2-byte units) of (t, c) in a bf16 block: 8 S + c % 8."""
    return 8 * slot_index(W) + np.arange(W)[None, :] % 8


def pack_bf16_block(x16: np.ndarray) -> np.ndarray:
    """bf16 patterns [n, 32, W] -> uint8 [n, 64 W]: the 8 values of slot S at bytes
    16 S .. 16 S + 15."""
    n, _, W = x16.shape
    out = np.zeros((n, 32 * W), dtype=np.uint16)
    out[:, _bf16_index(W).reshape(-1)] = x16.astype(np.uint16).reshape(n, 32 * W)
    return out.view(np.uint8).reshape(n, 64 * W)


def unpack_bf16_block(raw: np.ndarray, W: int) -> np.ndarray:
    n = raw.shape[0]
    v = np.ascontiguousarray(raw[:, :64 * W]).view(np.uint16).reshape(n, 32 * W)
    return v[:, _bf16_index(W).reshape(-1)].reshape(n, 32, W)


# ---------------------------------------------------------------------------
# Quantisation of stored rows
# ---------------------------------------------------------------------------

def quantise_rows(dims: Dims, bits: int, d: int, X: np.ndarray) -> dict:
    """X fp32 [n, 32, W] (W = d + d_R stored channels) -> fields of n blocks."""
    n, _, W = X.shape
    if dims.qscheme == KIVI32:
        u, s, z = quant.kivi_quantize(X.reshape(n, 32, W // 32, 32), bits)
        return {"u": u.reshape(n, 32, W), "s": s, "z": z}  # s, z fp16 [n, 32, W/32]
    ul, sl = quant.symrow_quantize(X[..., :d], bits)
    ur, sr = quant.symrow_quantize(X[..., d:], bits)
    return {"u": np.concatenate([ul, ur], axis=-1), "sl": sl, "sr": sr}  # bf16 bits [n, 32]


def dequantise_rows(dims: Dims, bits: int, d: int, f: dict) -> np.ndarray:
    n, _, W = f["u"].shape
    if dims.qscheme == KIVI32:
        u = f["u"].reshape(n, 32, W // 32, 32)
        return quant.kivi_dequantize(u, f["s"][..., None], f["z"][..., None]).reshape(n, 32, W)
    lat = quant.symrow_dequantize(f["u"][..., :d], f["sl"][..., None], bits)
    rope = quant.symrow_dequantize(f["u"][..., d:], f["sr"][..., None], bits)
    return np.concatenate([lat, rope], axis=-1)


def pack_quant_blocks(dims: Dims, bits: int, f: dict) -> np.ndarray:
    """[codes: 32 W b / 8 bytes][meta]: KIVI32 meta holds per token t, per group K
    of 32 stored channels, the fp16 scale then the fp16 zero at
    kivi_meta_offset(W)[t, K]; SYMROW meta holds per token the bf16 scale of c[:d]
    then that of k^R at byte 4 t."""
    n, _, W = f["u"].shape
    cb = codes_bytes(W, bits)
    out = np.zeros((n, block_bytes(dims, bits, W - dims.rope_dim)), dtype=np.uint8)
    out[:, :cb] = _pack(f["u"], code_bitaddr(W, bits), bits, cb)
    if dims.qscheme == KIVI32:
        off = cb + kivi_meta_offset(W)
        _u16_put(out, off, f["s"].view(np.uint16))
        _u16_put(out, off + 2, f["z"].view(np.uint16))
    else:
        off = cb + 4 * np.arange(32)
        _u16_put(out, off, f["sl"])
        _u16_put(out, off + 2, f["sr"])
    return out


def unpack_quant_blocks(dims: Dims, bits: int, d: int, raw: np.ndarray) -> dict:
    W = d + dims.rope_dim
    cb = codes_bytes(W, bits)
    f = {"u": _unpack(raw[:, :cb], code_bitaddr(W, bits), bits)}
    if dims.qscheme == KIVI32:
        off = cb + kivi_meta_offset(W)
        f["s"] = _u16_get(raw, off).view(np.float16)
        f["z"] = _u16_get(raw, off + 2).view(np.float16)
    else:
        off = cb + 4 * np.arange(32)
        f["sl"] = _u16_get(raw, off)
        f["sr"] = _u16_get(raw, off + 2)
    return f


# ---------------------------------------------------------------------------
# Streams (one per sequence)
# ---------------------------------------------------------------------------

def compress_stream(dims: Dims, bits: int, d: int, C: np.ndarray, R: np.ndarray) -> np.ndarray:
    """Stored tokens of one sequence: latent C [n, >= d] and positional key
    R [n, d_R] (fp32 values) -> stream bytes.  Only C[:, :d] is written."""
    X = np.concatenate([np.asarray(C, F32)[:, :d], np.asarray(R, F32)], axis=1)
    n, W = X.shape
    nb, nt = divmod(n, GROUP)
    Xf = X[:nb * GROUP].reshape(nb, GROUP, W)
    if bits == 16:
        blocks = pack_bf16_block(quant.bf16_bits(Xf))
    else:
        blocks = pack_quant_blocks(dims, bits, quantise_rows(dims, bits, d, Xf))
    tail = np.zeros((1, GROUP, W), dtype=np.uint16)
    tail[0, :nt] = quant.bf16_bits(X[nb * GROUP:])
    sb = stream_bytes(dims, bits, d)
    out = np.zeros(sb, dtype=np.uint8)
    blk = block_bytes(dims, bits, d)
    out[:nb * blk] = blocks.reshape(-1)
    t0 = (dims.stored_cap // GROUP) * blk
    out[t0:t0 + tail_bytes(dims, d)] = pack_bf16_block(tail)[0]
    return out


def append_token(dims: Dims, bits: int, d: int, stream: np.ndarray, n_stored: int, c_tok, r_tok) -> np.ndarray:
    """Decode-time append of the token at position n_stored (latent c_tok [>= d],
    positional key r_tok [d_R]) to one MLA stream, by the rule of the GQA append
    (oracle.cache.append_token): the stored row [c[:d] ; k^R], rounded to bf16,
    enters tail slot n_stored % 32, and the token that fills the tail completes a
    group that is written, from its bf16 rows, as full block n_stored // 32.
    Returns the new stream bytes (the input is not modified)."""
    W = d + dims.rope_dim
    out = np.array(stream, dtype=np.uint8, copy=True)
    blk = block_bytes(dims, bits, d)
    t0 = (dims.stored_cap // GROUP) * blk
    tb = tail_bytes(dims, d)
    tail = unpack_bf16_block(out[None, t0:t0 + tb], W)  # [1, 32, W] bf16 patterns
    slot = n_stored % GROUP
    row = np.concatenate([np.asarray(c_tok, F32)[:d], np.asarray(r_tok, F32)])
    tail[0, slot] = quant.bf16_bits(row)
    if slot < GROUP - 1:
        out[t0:t0 + tb] = pack_bf16_block(tail)[0]
        return out
    j = n_stored // GROUP
    if bits == 16:
        block = pack_bf16_block(tail)[0]
    else:
        block = pack_quant_blocks(dims, bits, quantise_rows(dims, bits, d, quant.bf16_value(tail)))[0]
    out[j * blk:(j + 1) * blk] = block
    return out


def dequant_stream(dims: Dims, bits: int, d: int, stream: np.ndarray, n_stored: int):
    """Stream bytes -> (C_hat [n_stored, d], R_hat [n_stored, d_R]) fp32."""
    W = d + dims.rope_dim
    blk = block_bytes(dims, bits, d)
    nb, nt = divmod(n_stored, GROUP)
    raw = stream[:nb * blk].reshape(nb, blk)
    if bits == 16:
        X = quant.bf16_value(unpack_bf16_block(raw, W))
    else:
        X = dequantise_rows(dims, bits, d, unpack_quant_blocks(dims, bits, d, raw))
    t0 = (dims.stored_cap // GROUP) * blk
    tail = quant.bf16_value(unpack_bf16_block(stream[None, t0:t0 + tail_bytes(dims, d)], W))[0]
    X = np.concatenate([X.reshape(-1, W), tail[:nt]])
    return X[:, :d], X[:, d:]


def compress_layer(dims: Dims, bits: int, d: int, C: np.ndarray, R: np.ndarray,
                   keep=None) -> np.ndarray:
    """C [B, n, r], R [B, n, d_R] -> the layer's region (B streams).  keep
    [B, n_keep]: the stored stream is the tokens at these positions, in order."""
    sb = stream_bytes(dims, bits, d)
    out = np.zeros(layer_bytes(dims, bits, d), dtype=np.uint8)
    for b in range(C.shape[0]):
        c, r = C[b], R[b]
        if keep is not None:
            idx = np.sort(np.asarray(keep[b]))
            c, r = c[idx], r[idx]
        out[b * sb:(b + 1) * sb] = compress_stream(dims, bits, d, c, r)
    return out


# ---------------------------------------------------------------------------
# Low-rank projection on write (§2.1 "Rank", App. C.2)
# ---------------------------------------------------------------------------

def round_bf16_exact(x) -> np.ndarray:
    """fp64 values rounded once to bf16 (nearest, ties to even), returned as fp64.
    Values stay well inside the bf16 normal range here."""
    x = np.ascontiguousarray(np.asarray(x, np.float64))
    b = x.view(np.uint64)
    lsb = (b >> np.uint64(45)) & np.uint64(1)  # last kept mantissa bit (7 of 52 kept)
    r = ((b + np.uint64((1 << 44) - 1) + lsb) >> np.uint64(45)) << np.uint64(45)
    return r.view(np.float64)


def project_latent(X, W_DKV, d: int) -> np.ndarray:
    """The latent a layer keeping width d stores for tokens X [n, H]: the first d
    coordinates of the down-projection, c[:d] = W_DKV[:d, :] x per token (App. C.2:
    a deployed kernel computes only those), exact in fp64 and rounded once to bf16
    (the latent is held in bf16 before the cache write quantises it).  W_DKV
    [r, H]: row i maps a token's hidden state to latent coordinate i."""
    c = np.asarray(X, np.float64) @ np.asarray(W_DKV, np.float64)[:d].T
    return round_bf16_exact(c)


def compress_layer_projected(dims: Dims, bits: int, d: int, X: np.ndarray, W_DKV: np.ndarray, R: np.ndarray,
                             keep=None) -> np.ndarray:
    """X [B, n, H] hidden states, R [B, n, d_R] positional keys -> the layer's region:
    the latent of every token projected to its first d coordinates, then written
    exactly as a latent input is (truncation, quantiser, layout)."""
    C = np.stack([project_latent(X[b], W_DKV, d) for b in range(X.shape[0])])
    return compress_layer(dims, bits, d, C, R, keep)


def compress_arena(dims: Dims, plan, Cs, Rs, keeps=None) -> np.ndarray:
    offs, total = arena_offsets(dims, plan)
    arena = np.zeros(total, dtype=np.uint8)
    for l, a in enumerate(plan):
        if a.inherit:
            continue
        reg = compress_layer(dims, a.bits, a.rank, Cs[l], Rs[l], None if keeps is None else keeps[l])
        arena[offs[l]:offs[l] + reg.size] = reg
    return arena


def dequant_layer(dims: Dims, plan, arena: np.ndarray, layer: int, n_stored: int):
    """(C_hat [B, n, d], R_hat [B, n, d_R]) of the cache `layer` reads."""
    a = anchor_of(plan)[layer]
    offs, _ = arena_offsets(dims, plan)
    bits, d = plan[a].bits, plan[a].rank
    sb = stream_bytes(dims, bits, d)
    Cs, Rs = [], []
    for b in range(dims.batch):
        s = offs[a] + b * sb
        c, r = dequant_stream(dims, bits, d, arena[s:s + sb], n_stored)
        Cs.append(c)
        Rs.append(r)
    return np.stack(Cs), np.stack(Rs)


# ---------------------------------------------------------------------------
# Attention
# ---------------------------------------------------------------------------

def attention_reconstructed(q_nope, q_rope, Chat, Rhat, W_UK, W_UV, scale):
    """Explicit reconstruction (§2.1, App. C.2).  q_nope [H, nope], q_rope [H, d_R],
    Chat [T, d], Rhat [T, d_R], W_UK [H, nope, r], W_UV [H, v, r] -> [H, v].
    The latent is zero-padded from d to r; head h attends with keys
    [W_UK_h c_t ; k^R_t] and values W_UV_h c_t."""
    H, _, r = W_UK.shape
    T, d = Chat.shape
    C = np.zeros((T, r))
    C[:, :d] = Chat
    out = np.zeros((H, W_UV.shape[1]))
    for h in range(H):
        K = np.concatenate([C @ np.asarray(W_UK[h], np.float64).T, np.asarray(Rhat, np.float64)], axis=1)
        V = C @ np.asarray(W_UV[h], np.float64).T
        q = np.concatenate([q_nope[h], q_rope[h]])[None]
        out[h] = att.softmax_attention(q, K, V, scale)[0]
    return out


def attention_absorbed(q_nope, q_rope, Chat, Rhat, W_UK, W_UV, scale):
    """The same attention with the projections moved onto the query and the
    output (App. C.2): q~_h = W_UK_h[:, :d]^T q_nope_h; scores
    scale (q~_h . c_t + q_rope_h . k^R_t); o_lat = softmax . C; o_h = W_UV_h[:, :d] o_lat."""
    H = W_UK.shape[0]
    T, d = Chat.shape
    C = np.asarray(Chat, np.float64)
    R = np.asarray(Rhat, np.float64)
    out = np.zeros((H, W_UV.shape[1]))
    if T == 0:
        return out
    for h in range(H):
        qt = np.asarray(W_UK[h], np.float64)[:, :d].T @ np.asarray(q_nope[h], np.float64)
        s = scale * (C @ qt + R @ np.asarray(q_rope[h], np.float64))
        p = np.exp(s - s.max())
        olat = (p @ C) / p.sum()
        out[h] = np.asarray(W_UV[h], np.float64)[:, :d] @ olat
    return out


def decode_step(dims: Dims, plan, arena: np.ndarray, q: np.ndarray, w_uk: np.ndarray,
                w_uv: np.ndarray, n_stored: int, scale: float, l0: int = 0, l1=None,
                absorbed: bool = False) -> np.ndarray:
    """q [l1-l0, B, Hq, nope + d_R], w_uk [l1-l0, Hq, nope, r], w_uv [l1-l0, Hq, v, r]
    -> out fp64 [l1-l0, B, Hq, v]: each layer's own query and up-projections against
    its anchor's stored latent (§2.1).  absorbed=True evaluates the same attention
    in the absorbed form (cheaper for long contexts; pinned equal to the
    reconstruction)."""
    assert dims.kind == MLA
    l1 = dims.n_layers if l1 is None else l1
    anc = anchor_of(plan)
    nope = dims.nope_dim
    out = np.zeros((l1 - l0, dims.batch, dims.n_q_heads, dims.v_dim))
    cache = {}
    for l in range(l0, l1):
        a = anc[l]
        if a not in cache:
            cache[a] = dequant_layer(dims, plan, arena, a, n_stored)
        Ch, Rh = cache[a]
        for b in range(dims.batch):
            qb = np.asarray(q[l - l0, b], np.float64)
            f = attention_absorbed if absorbed else attention_reconstructed
            out[l - l0, b] = f(qb[:, :nope], qb[:, nope:], Ch[b], Rh[b], w_uk[l - l0], w_uv[l - l0], scale)
    return out


__all__ = ["code_bitaddr", "codes_bytes", "quantise_rows", "dequantise_rows", "pack_quant_blocks",
           "unpack_quant_blocks", "pack_bf16_block", "unpack_bf16_block", "compress_stream",
           "dequant_stream", "compress_layer", "compress_arena", "dequant_layer",
           "attention_reconstructed", "attention_absorbed", "decode_step", "stored_width"]
