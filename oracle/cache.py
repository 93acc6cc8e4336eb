"""Compress a layer to arena bytes and run a decode step from them (oracle).

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

Write side (§2.1, App. C.3): an anchor layer stores, per (sequence, KV head),
its keys and values — after an optional eviction gather (§3 long context: the
evictor runs on the same cache) — as 32-token blocks quantised by the table's
scheme (or bf16 at b = 16) plus a bf16 tail of the last n % 32 tokens.  An
inheriting layer stores nothing.

Read side: dequantise the anchor's stream and attend (§2.1).

Parity: dequantised values and arena bytes are defined exactly by the rules in
include/kvk.h and are pinned through the quantiser and layout pins; attention
outputs on compressed caches have no printed values in the paper (parity of
those values rests on the attention pins plus this composition).
"""
import numpy as np

from . import attention as att
from . import layout, quant
from .plan import (GROUP, GROUP64, KIVI32, Dims, anchor_of, arena_offsets, block_bytes, layer_bytes, stream_bytes,
                   tail_bytes)

F32 = np.float32


def quantise_blocks(dims: Dims, bits: int, K: np.ndarray, V: np.ndarray) -> dict:
    """K, V fp32 [nb, 32, D] -> the fields of nb quantised blocks."""
    D = dims.head_dim
    nb = K.shape[0]
    if dims.qscheme == KIVI32:
        uk, ks, kz = quant.kivi_quantize(np.swapaxes(K, 1, 2), bits)  # groups: channel x 32 tokens
        uv, vs, vz = quant.kivi_quantize(V.reshape(nb, 32, D // 32, 32), bits)  # token x 32 ch
        return {"uk": np.swapaxes(uk, 1, 2), "uv": uv.reshape(nb, 32, D),
                "ks": ks, "kz": kz, "vs": vs, "vz": vz}
    if dims.qscheme == GROUP64:  # keys and values alike: token x 64 consecutive channels
        uk, ks, kz = quant.kivi_quantize(K.reshape(nb, 32, D // 64, 64), bits)
        uv, vs, vz = quant.kivi_quantize(V.reshape(nb, 32, D // 64, 64), bits)
        return {"uk": uk.reshape(nb, 32, D), "uv": uv.reshape(nb, 32, D),
                "ks": ks, "kz": kz, "vs": vs, "vz": vz}
    uk, ks = quant.symrow_quantize(K, bits)  # one row = a token's D channels
    uv, vs = quant.symrow_quantize(V, bits)
    return {"uk": uk, "uv": uv, "ks": ks, "vs": vs}


def dequantise_blocks(dims: Dims, bits: int, f: dict):
    """Fields of nb quantised blocks -> K_hat, V_hat fp32 [nb, 32, D]."""
    D = dims.head_dim
    nb = f["uk"].shape[0]
    if dims.qscheme == KIVI32:
        kh = quant.kivi_dequantize(f["uk"], f["ks"][:, None, :], f["kz"][:, None, :])
        uv = f["uv"].reshape(nb, 32, D // 32, 32)
        vh = quant.kivi_dequantize(uv, f["vs"][..., None], f["vz"][..., None]).reshape(nb, 32, D)
        return kh, vh
    if dims.qscheme == GROUP64:
        uk = f["uk"].reshape(nb, 32, D // 64, 64)
        uv = f["uv"].reshape(nb, 32, D // 64, 64)
        kh = quant.kivi_dequantize(uk, f["ks"][..., None], f["kz"][..., None]).reshape(nb, 32, D)
        vh = quant.kivi_dequantize(uv, f["vs"][..., None], f["vz"][..., None]).reshape(nb, 32, D)
        return kh, vh
    kh = quant.symrow_dequantize(f["uk"], f["ks"][..., None], bits)
    vh = quant.symrow_dequantize(f["uv"], f["vs"][..., None], bits)
    return kh, vh


def compress_stream(dims: Dims, bits: int, K: np.ndarray, V: np.ndarray) -> np.ndarray:
    """One stream's stored tokens K, V [n, D] (fp32 values) -> stream bytes."""
    n, D = K.shape
    nb, nt = divmod(n, GROUP)
    K = np.asarray(K, dtype=F32)
    V = np.asarray(V, dtype=F32)
    Kf = K[:nb * GROUP].reshape(nb, GROUP, D)
    Vf = V[:nb * GROUP].reshape(nb, GROUP, D)
    if bits == 16:
        blocks = layout.pack_bf16_blocks(quant.bf16_bits(Kf), quant.bf16_bits(Vf))
    else:
        blocks = layout.pack_quant_blocks(dims, bits, quantise_blocks(dims, bits, Kf, Vf))
    kt = np.zeros((1, GROUP, D), dtype=np.uint16)
    vt = np.zeros((1, GROUP, D), dtype=np.uint16)
    kt[0, :nt] = quant.bf16_bits(K[nb * GROUP:])
    vt[0, :nt] = quant.bf16_bits(V[nb * GROUP:])
    tail = layout.pack_bf16_blocks(kt, vt)[0]
    return layout.assemble_stream(dims, bits, blocks, tail)


def dequant_stream(dims: Dims, bits: int, stream: np.ndarray, n_stored: int):
    """Stream bytes -> K_hat, V_hat fp32 [n_stored, D]."""
    D = dims.head_dim
    blocks, tail = layout.split_stream(dims, bits, stream, n_stored)
    nb = blocks.shape[0]
    if bits == 16:
        kb, vb = layout.unpack_bf16_blocks(blocks, D)
        kh, vh = quant.bf16_value(kb), quant.bf16_value(vb)
    else:
        kh, vh = dequantise_blocks(dims, bits, layout.unpack_quant_blocks(dims, bits, blocks))
    kt, vt = layout.unpack_bf16_blocks(tail[None], D)
    nt = n_stored - nb * GROUP
    K = np.concatenate([kh.reshape(-1, D), quant.bf16_value(kt[0, :nt])])
    V = np.concatenate([vh.reshape(-1, D), quant.bf16_value(vt[0, :nt])])
    return K, V


def append_token(dims: Dims, bits: int, stream: np.ndarray, n_stored: int, k_tok, v_tok) -> np.ndarray:
    """Decode-time append of the token at position n_stored to one stream.

    The plan holds for the whole generation (§2.3), so the stream keeps its
    configuration.  The new token (key and value [D], rounded to bf16) goes to slot
    n_stored % 32 of the bf16 tail, the window of recent tokens kept in full
    precision (App. C.3).  When that slot is the last one, the 32 tail tokens form a
    complete group: they are quantised from their bf16 values into full block
    n_stored // 32 by the block quantiser of the prefill write, and the tail is
    empty again.  Returns the new stream bytes (the input is not modified)."""
    D = dims.head_dim
    out = np.array(stream, dtype=np.uint8, copy=True)
    blk = block_bytes(dims, bits)
    t0 = (dims.stored_cap // GROUP) * blk
    kt, vt = layout.unpack_bf16_blocks(out[None, t0:t0 + tail_bytes(dims)], D)
    slot = n_stored % GROUP
    kt[0, slot] = quant.bf16_bits(np.asarray(k_tok, F32))
    vt[0, slot] = quant.bf16_bits(np.asarray(v_tok, F32))
    if slot < GROUP - 1:
        out[t0:t0 + tail_bytes(dims)] = layout.pack_bf16_blocks(kt, vt)[0]
        return out
    j = n_stored // GROUP
    if bits == 16:
        block = layout.pack_bf16_blocks(kt, vt)[0]
    else:
        Kg = quant.bf16_value(kt)  # [1, 32, D] fp32
        Vg = quant.bf16_value(vt)
        block = layout.pack_quant_blocks(dims, bits, quantise_blocks(dims, bits, Kg, Vg))[0]
    out[j * blk:(j + 1) * blk] = block
    return out


def gather_kept(X: np.ndarray, keep: np.ndarray) -> np.ndarray:
    """Eviction: the stored stream is X at the kept positions, in increasing order."""
    return X[np.sort(np.asarray(keep))]


def compress_layer(dims: Dims, bits: int, K: np.ndarray, V: np.ndarray, keep=None) -> np.ndarray:
    """K, V [B, Hkv, n, D] -> the layer's region bytes (B*Hkv streams)."""
    B, H = K.shape[:2]
    sb = stream_bytes(dims, bits)
    out = np.zeros(layer_bytes(dims, bits), dtype=np.uint8)
    for b in range(B):
        for h in range(H):
            k, v = K[b, h], V[b, h]
            if keep is not None:
                k, v = gather_kept(k, keep[b, h]), gather_kept(v, keep[b, h])
            s = b * H + h
            out[s * sb:(s + 1) * sb] = compress_stream(dims, bits, k, v)
    return out


def compress_arena(dims: Dims, plan, Ks, Vs, keeps=None) -> np.ndarray:
    """Whole arena for per-layer inputs Ks[l], Vs[l] (ignored for inheritors)."""
    offs, total = arena_offsets(dims, plan)
    arena = np.zeros(total, dtype=np.uint8)
    for l, a in enumerate(plan):
        if a.inherit:
            continue
        reg = compress_layer(dims, a.bits, Ks[l], Vs[l], None if keeps is None else keeps[l])
        arena[offs[l]:offs[l] + reg.size] = reg
    return arena


def dequant_layer(dims: Dims, plan, arena: np.ndarray, layer: int, n_stored: int):
    """K_hat, V_hat fp32 [B, Hkv, n_stored, D] of the cache `layer` reads."""
    a = anchor_of(plan)[layer]
    offs, _ = arena_offsets(dims, plan)
    bits = plan[a].bits
    sb = stream_bytes(dims, bits)
    B, H, D = dims.batch, dims.n_kv_heads, dims.head_dim
    Kh = np.zeros((B, H, n_stored, D), dtype=F32)
    Vh = np.zeros_like(Kh)
    for b in range(B):
        for h in range(H):
            s = offs[a] + (b * H + h) * sb
            Kh[b, h], Vh[b, h] = dequant_stream(dims, bits, arena[s:s + sb], n_stored)
    return Kh, Vh


def decode_step(dims: Dims, plan, arena: np.ndarray, q: np.ndarray, n_stored: int,
                scale: float, l0: int = 0, l1=None) -> np.ndarray:
    """q [l1-l0, B, Hq, D] -> out fp64 [l1-l0, B, Hq, D]: each layer's own query
    attends over its anchor's dequantised cache (§2.1)."""
    l1 = dims.n_layers if l1 is None else l1
    anc = anchor_of(plan)
    out = np.zeros((l1 - l0, dims.batch, dims.n_q_heads, dims.head_dim))
    cachebuf = {}
    for l in range(l0, l1):
        a = anc[l]
        if a not in cachebuf:
            cachebuf[a] = dequant_layer(dims, plan, arena, a, n_stored)
        Kh, Vh = cachebuf[a]
        for b in range(dims.batch):
            out[l - l0, b] = att.gqa_attention(np.asarray(q[l - l0, b], np.float64),
                                               Kh[b], Vh[b], scale)
    return out


def compress_arena_batched(dims: Dims, plans, Ks, Vs, keeps=None) -> np.ndarray:
    """Arena of a batch with per-sequence plans: Ks[l], Vs[l] [B, Hkv, n, D]; the
    arena of sequence b (plans[b], its rows of the inputs) at its base."""
    from .plan import batched_arena_bases, sequence_dims
    sd = sequence_dims(dims)
    bases, total = batched_arena_bases(dims, plans)
    arena = np.zeros(total, dtype=np.uint8)
    for b, pl in enumerate(plans):
        sub = compress_arena(sd, pl, [None if K is None else K[b:b + 1] for K in Ks],
                             [None if V is None else V[b:b + 1] for V in Vs],
                             None if keeps is None else [None if k is None else k[b:b + 1] for k in keeps])
        arena[bases[b]:bases[b] + sub.size] = sub
    return arena


def decode_step_batched(dims: Dims, plans, arena: np.ndarray, q: np.ndarray, n_stored: int,
                        scale: float, l0: int = 0, l1=None) -> np.ndarray:
    """q [l1-l0, B, Hq, D] -> out fp64 [l1-l0, B, Hq, D]: sequence b decodes its own
    arena with its own plan (the uniform decode step of a one-sequence table)."""
    from .plan import batched_arena_bases, sequence_dims
    l1 = dims.n_layers if l1 is None else l1
    sd = sequence_dims(dims)
    bases, _ = batched_arena_bases(dims, plans)
    out = np.zeros((l1 - l0, dims.batch, dims.n_q_heads, dims.head_dim))
    for b, pl in enumerate(plans):
        size = arena_offsets(sd, pl)[1]
        out[:, b:b + 1] = decode_step(sd, pl, arena[bases[b]:bases[b] + size], q[:, b:b + 1], n_stored,
                                      scale, l0, l1)
    return out
