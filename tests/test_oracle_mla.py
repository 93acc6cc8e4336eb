"""Pins of the oracle's rank axis (MLA latent caches, App. C.2, §2.1, §2.2)."""
import math
import os

import numpy as np
import pytest
import torch

from oracle import attention as A
from oracle import mla as M
from oracle import plan as P
from oracle import quant as Q

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "mla_layout_examples.txt")


def _dims(d_max=64, qs=P.KIVI32, B=2, T=96, keep=0, H=4):
    return P.Dims(P.MLA, 3, H, 1, 128, latent_dim=d_max, rope_dim=64, nope_dim=16, v_dim=8,
                  qscheme=qs, batch=B, max_tokens=T, keep_tokens=keep)


def _golden():
    rows = []
    for line in open(GOLDEN):
        line = line.strip()
        if line and not line.startswith("#"):
            rows.append(line.split())
    return rows


# ---------------------------------------------------------------------------
# Layout
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("W", [96, 128, 192, 320, 576])
@pytest.mark.parametrize("bits", [2, 4, 8])
def test_code_map_is_a_bijection(W, bits):
    """Every code gets b bits of its own and the codes fill the code region."""
    addr = M.code_bitaddr(W, bits).reshape(-1)
    occupied = (addr[:, None] + np.arange(bits)[None, :]).reshape(-1)
    assert occupied.min() == 0 and occupied.size == 32 * W * bits
    assert np.unique(occupied).size == occupied.size


@pytest.mark.parametrize("W", [96, 128, 192, 320, 576])
def test_slot_bf16_and_meta_maps_are_bijections(W):
    """Slots hold 8 channels of one token each and cover 4 W slots; the bf16 block
    and the KIVI32 (scale, zero) pairs fill their regions exactly once."""
    S = M.slot_index(W)
    assert np.array_equal(np.sort(np.unique(S)), np.arange(4 * W))
    assert np.all(np.bincount(S.reshape(-1)) == 8)
    rows, cols = np.nonzero(S == S[17, 40 % W])
    assert np.unique(rows).size == 1 and np.ptp(cols) == 7
    b16 = (8 * S + np.arange(W)[None, :] % 8).reshape(-1)
    assert np.array_equal(np.sort(b16), np.arange(32 * W))
    meta = M.kivi_meta_offset(W).reshape(-1)
    assert np.array_equal(np.sort(meta), 4 * np.arange(32 * W // 32))


def test_layout_hand_examples():
    dims = {s: _dims(qs=(P.KIVI32 if s == "kivi" else P.SYMROW)) for s in ("kivi", "symrow", "bf16")}
    n = 0
    for row in _golden():
        if row[0] == "code":
            W, bits, t, c, want = map(int, row[1:])
            assert M.code_bitaddr(W, bits)[t, c] == want, row
        elif row[0] == "bf16":
            W, t, c, want = map(int, row[1:])
            x = np.zeros((1, 32, W), dtype=np.uint16)
            x[0, t, c] = 0x3F00  # bf16 0.5: low byte zero
            nz = np.nonzero(M.pack_bf16_block(x)[0])[0]
            assert nz.size == 1 and nz[0] == want + 1, (row, nz)  # little-endian: high byte second
            assert M.unpack_bf16_block(M.pack_bf16_block(x), W)[0, t, c] == 0x3F00
        elif row[0] == "meta":
            scheme, W, bits, t, g, field, want = row[1], int(row[2]), int(row[3]), int(row[4]), int(row[5]), row[6], int(row[7])
            # place a marker in one field through the packer and find its byte
            u = np.zeros((1, 32, W), dtype=np.int64)
            d = W - 64
            dm = P.Dims(P.MLA, 1, 4, 1, 128, latent_dim=d, rope_dim=64, nope_dim=16, v_dim=8,
                        qscheme=P.KIVI32 if scheme == "kivi" else P.SYMROW, max_tokens=32)
            if scheme == "kivi":
                f = {"u": u, "s": np.zeros((1, 32, W // 32), np.float16), "z": np.zeros((1, 32, W // 32), np.float16)}
                f["s" if field == "scale" else "z"][0, t, g] = np.float16(1.0)  # 0x3C00
            else:
                f = {"u": u, "sl": np.zeros((1, 32), np.uint16), "sr": np.zeros((1, 32), np.uint16)}
                f["sl" if field == "latent" else "sr"][0, t] = 0x3F00  # bf16 0.5: low byte zero
            raw = M.pack_quant_blocks(dm, bits, f)[0]
            nz = np.nonzero(raw)[0]
            assert nz.size == 1 and nz[0] == want + 1, (row, nz)  # little-endian: high byte second
        elif row[0] == "blocksize":
            scheme, d, dR, bits, want = row[1], int(row[2]), int(row[3]), int(row[4]), int(row[5])
            dm = P.Dims(P.MLA, 1, 4, 1, 128, latent_dim=d, rope_dim=dR, nope_dim=16, v_dim=8,
                        qscheme=P.SYMROW if scheme == "symrow" else P.KIVI32, max_tokens=32)
            assert P.block_bytes(dm, bits, d) == want, row
        n += 1
    assert n > 20


@pytest.mark.parametrize("bits", [2, 4, 8])
@pytest.mark.parametrize("qs", [P.KIVI32, P.SYMROW])
def test_pack_unpack_every_code_value(bits, qs):
    W, d = 160, 96
    dims = P.Dims(P.MLA, 1, 4, 1, 128, latent_dim=96, rope_dim=64, qscheme=qs, max_tokens=32)
    rng = np.random.default_rng(bits)
    u = rng.integers(0, 2 ** bits, (3, 32, W))
    u[0].reshape(-1)[:2 ** bits] = np.arange(2 ** bits)
    if qs == P.KIVI32:
        f = {"u": u, "s": rng.standard_normal((3, 32, W // 32)).astype(np.float16),
             "z": rng.standard_normal((3, 32, W // 32)).astype(np.float16)}
    else:
        f = {"u": u, "sl": rng.integers(0, 2 ** 16, (3, 32)).astype(np.uint16),
             "sr": rng.integers(0, 2 ** 16, (3, 32)).astype(np.uint16)}
    raw = M.pack_quant_blocks(dims, bits, f)
    back = M.unpack_quant_blocks(dims, bits, d, raw)
    for k in f:
        assert np.array_equal(np.asarray(back[k]).view(np.uint16) if k != "u" else back[k],
                              np.asarray(f[k]).view(np.uint16) if k != "u" else f[k]), k


def test_block_bits_are_eq1_cost_plus_metadata():
    """eq. (1): a (d, b) layer costs (d + d_R) b bits per token; the stored block adds
    exactly the stated metadata: 32 bits per 32-channel group (KIVI32) or two bf16
    scales per token (SYMROW); bf16 adds nothing."""
    for d in (64, 128, 256, 512):
        for bits in (2, 4, 8, 16):
            for qs in (P.KIVI32, P.SYMROW):
                dims = P.Dims(P.MLA, 1, 32, 4, 128, latent_dim=512, rope_dim=64, qscheme=qs, max_tokens=32)
                per_token = P.block_bytes(dims, bits, d) * 8 / 32
                c = P.cost_bits(dims, P.Action(bits=bits, rank=d))
                assert c == (d + 64) * bits
                if bits == 16:
                    meta = 0
                elif qs == P.KIVI32:
                    meta = 32 * (d + 64) // 32
                else:
                    meta = 32
                assert per_token == c + meta


def test_table_ratios_match_printed_mla_ranges():
    """eq. (2) on an MLA table at the Qwen2.5-14B geometry of App. C.1
    ((L, 2 n_kv d_h, r) = (48, 2048, 1024), d_R = 64): a plan at full width and
    16 bits gives the printed rho_min 1.88; all layers at (r/8, 2) the printed
    rank+precision maximum 85.3; one such anchor read by every layer 4096."""
    dims = P.Dims(P.MLA, 48, 40, 8, 128, latent_dim=1024, rope_dim=64, nope_dim=128, v_dim=128,
                  max_tokens=32)
    full = [P.Action(bits=16, rank=1024)] * 48
    assert round(P.rho(dims, full), 2) == 1.88
    low = [P.Action(bits=2, rank=128)] * 48
    assert round(P.rho(dims, low), 1) == 85.3
    deep = [P.Action(bits=2, rank=128)] + [P.Action(inherit=True)] * 47
    assert P.rho(dims, deep) == 4096


# ---------------------------------------------------------------------------
# Quantisers on MLA rows
# ---------------------------------------------------------------------------

def test_kivi_groups_are_32_channels_of_one_token():
    """A ramp 0..31 over one group at 4 bits gives s = fp16(31/15), z = 0 and the
    codes rint(i / s); a constant group gives s = 0 and codes 0; groups do not mix
    (each token and group has its own pair)."""
    dims = _dims(d_max=64)
    X = np.zeros((1, 32, 128), np.float32)
    X[0, 3, 32:64] = np.arange(32)
    X[0, 4, :] = 7.0
    f = M.quantise_rows(dims, 4, 64, X)
    s = np.float16(np.float32(31) / np.float32(15))
    assert f["s"][0, 3, 1] == s and f["z"][0, 3, 1] == 0
    assert np.array_equal(f["u"][0, 3, 32:64], np.rint(np.arange(32, dtype=np.float32) / np.float32(s)))
    assert np.all(f["s"][0, 4] == 0) and np.all(f["u"][0, 4] == 0) and np.all(f["z"][0, 4] == 7)
    Xh = M.dequantise_rows(dims, 4, 64, f)
    assert np.all(Xh[0, 4] == 7.0)


def test_symrow_scales_latent_and_rope_separately():
    """One scale per stored vector (App. C.3, §2.1): the latent row and the
    positional key row of a token each get max|x| / q in bf16."""
    dims = _dims(d_max=64, qs=P.SYMROW)
    X = np.zeros((1, 32, 128), np.float32)
    X[0, 0, :64] = np.linspace(-3.0, 1.0, 64)
    X[0, 0, 64:] = np.linspace(-0.5, 0.25, 64)
    f = M.quantise_rows(dims, 4, 64, X)
    assert Q.bf16_value(f["sl"][0, 0]) == Q.round_bf16(np.float32(3.0) / np.float32(7))
    assert Q.bf16_value(f["sr"][0, 0]) == Q.round_bf16(np.float32(0.5) / np.float32(7))
    Xh = M.dequantise_rows(dims, 4, 64, f)
    assert np.max(np.abs(Xh[0, 0, 64:] - X[0, 0, 64:])) <= Q.bf16_value(f["sr"][0, 0]) / 2 + 1e-7


@pytest.mark.parametrize("bits", [2, 4, 8])
@pytest.mark.parametrize("qs", [P.KIVI32, P.SYMROW])
def test_requantise_dequantised_rows_is_idempotent(bits, qs):
    dims = _dims(d_max=64, qs=qs)
    X = np.random.default_rng(bits).standard_normal((4, 32, 128)).astype(np.float32)
    f = M.quantise_rows(dims, bits, 64, X)
    Xh = M.dequantise_rows(dims, bits, 64, f)
    g = M.quantise_rows(dims, bits, 64, Xh)
    if qs == P.SYMROW:
        assert np.array_equal(g["u"], f["u"])
    else:  # re-quantising with the stored metadata reproduces the codes
        s = f["s"].astype(np.float32)[..., None]
        z = f["z"].astype(np.float32)[..., None]
        t = (Xh.reshape(4, 32, 4, 32) - z) / s
        u = np.clip(np.rint(t), 0, 2 ** bits - 1).reshape(4, 32, 128)
        assert np.array_equal(u, f["u"])


# ---------------------------------------------------------------------------
# Streams
# ---------------------------------------------------------------------------

def _bf16(seed, shape, scale=1.0):
    g = torch.Generator().manual_seed(seed)
    return (torch.randn(shape, generator=g) * scale).to(torch.bfloat16).float().numpy()


@pytest.mark.parametrize("n", [1, 31, 32, 70, 96])
def test_bf16_full_rank_recovers_input_exactly(n):
    """b = 16 on bf16 inputs at full width stores the latent and k^R unchanged, tail included."""
    dims = _dims(d_max=64)
    C, R = _bf16(1, (n, 64)), _bf16(2, (n, 64))
    st = M.compress_stream(dims, 16, 64, C, R)
    Ch, Rh = M.dequant_stream(dims, 16, 64, st, n)
    assert np.array_equal(Ch, C) and np.array_equal(Rh, R)


@pytest.mark.parametrize("bits", [2, 4, 8])
def test_truncated_write_stores_only_first_d(bits):
    """A (d, b) layer writes c[:d]: the stream is the same whatever c holds beyond d."""
    dims = _dims(d_max=128)
    C, R = _bf16(3, (64, 128)), _bf16(4, (64, 64))
    C2 = C.copy()
    C2[:, 32:] = 99.0
    assert np.array_equal(M.compress_stream(dims, bits, 32, C, R), M.compress_stream(dims, bits, 32, C2, R))
    assert M.compress_stream(dims, bits, 32, C, R).size == P.stream_bytes(dims, bits, 32)


# ---------------------------------------------------------------------------
# Attention
# ---------------------------------------------------------------------------

def _rand_mla(seed, H=3, nope=8, v=6, r=16, dR=4, T=11):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((H, nope)), rng.standard_normal((H, dR)), rng.standard_normal((T, r)),
            rng.standard_normal((T, dR)), rng.standard_normal((H, nope, r)) / 4, rng.standard_normal((H, v, r)) / 4)


@pytest.mark.parametrize("d", [4, 8, 16])
def test_absorbed_equals_reconstructed(d):
    qn, qr, C, R, WK, WV = _rand_mla(5)
    a = M.attention_absorbed(qn, qr, C[:, :d], R, WK, WV, 0.4)
    b = M.attention_reconstructed(qn, qr, C[:, :d], R, WK, WV, 0.4)
    assert np.allclose(a, b, rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("bits", [4, 16])
def test_prefix_mask_equals_truncation(bits):
    """App. C.2: training zeroes coordinates after d (prefix mask) at full shape; a
    deployed kernel writes only c[:d].  A full-width bf16 cache of the masked latent
    gives the same attention as the truncated cache (exactly at b = 16; at b = 4 the
    masked coordinates quantise in their own groups, so the kept groups match)."""
    dims = _dims(d_max=128)
    C, R = _bf16(6, (70, 128)), _bf16(7, (70, 64))
    rng = np.random.default_rng(8)
    qn, qr = rng.standard_normal((4, 16)), rng.standard_normal((4, 64))
    WK, WV = rng.standard_normal((4, 16, 128)) / 8, rng.standard_normal((4, 8, 128)) / 8
    Cm = C.copy()
    Cm[:, 64:] = 0.0
    full = M.dequant_stream(dims, bits, 128, M.compress_stream(dims, bits, 128, Cm, R), 70)
    trunc = M.dequant_stream(dims, bits, 64, M.compress_stream(dims, bits, 64, C, R), 70)
    assert np.array_equal(full[0][:, :64], trunc[0]) and np.all(full[0][:, 64:] == 0)
    a = M.attention_reconstructed(qn, qr, full[0], full[1], WK, WV, 0.1)
    b = M.attention_reconstructed(qn, qr, trunc[0], trunc[1], WK, WV, 0.1)
    assert np.array_equal(a, b) or np.allclose(a, b, rtol=1e-14, atol=1e-15)


def test_selection_weights_reduce_to_multi_head_attention():
    """With r = H * nope and W_UK_h = W_UV_h selecting latent slice h, head h is
    ordinary attention with keys [c_t[slice h] ; k^R_t] and values c_t[slice h]
    (scipy softmax on explicitly sliced operands)."""
    from scipy.special import softmax
    H, nope, dR, T = 3, 4, 2, 9
    rng = np.random.default_rng(9)
    C, R = rng.standard_normal((T, H * nope)), rng.standard_normal((T, dR))
    qn, qr = rng.standard_normal((H, nope)), rng.standard_normal((H, dR))
    W = np.zeros((H, nope, H * nope))
    for h in range(H):
        W[h, :, h * nope:(h + 1) * nope] = np.eye(nope)
    got = M.attention_reconstructed(qn, qr, C, R, W, W, 0.6)
    for h in range(H):
        Ch = C[:, h * nope:(h + 1) * nope]
        s = 0.6 * (Ch @ qn[h] + R @ qr[h])
        assert np.allclose(got[h], softmax(s) @ Ch, rtol=1e-12, atol=1e-14)


def test_special_cases():
    qn, qr, C, R, WK, WV = _rand_mla(10, T=7)
    one = M.attention_reconstructed(qn, qr, C[:1, :8], R[:1], WK, WV, 1.0)
    for h in range(3):
        assert np.allclose(one[h], WV[h][:, :8] @ C[0, :8], rtol=1e-12)
    z = M.attention_reconstructed(np.zeros_like(qn), np.zeros_like(qr), C[:, :8], R, WK, WV, 1.0)
    for h in range(3):
        assert np.allclose(z[h], WV[h][:, :8] @ C[:, :8].mean(0), rtol=1e-12)
    perm = np.random.default_rng(0).permutation(7)
    a = M.attention_absorbed(qn, qr, C[:, :8], R, WK, WV, 0.3)
    b = M.attention_absorbed(qn, qr, C[perm, :8], R[perm], WK, WV, 0.3)
    assert np.allclose(a, b, rtol=1e-12)
    assert np.all(M.attention_absorbed(qn, qr, C[:0, :8], R[:0], WK, WV, 1.0) == 0)


def test_split_merge_of_absorbed_scores():
    """Splitting the tokens and merging by log-sum-exp gives the one-pass latent output."""
    qn, qr, C, R, WK, WV = _rand_mla(11, T=13)
    d = 16
    qt = np.stack([WK[h][:, :d].T @ qn[h] for h in range(3)])
    key = np.concatenate([C, R], axis=1)
    qq = np.concatenate([qt, qr], axis=1)
    parts = [A.partial_attention(qq, key[a:b], C[a:b], 0.5) for a, b in [(0, 5), (5, 6), (6, 13)]]
    assert np.allclose(A.lse_merge(parts), A.softmax_attention(qq, key, C, 0.5), rtol=1e-12)


def test_decode_step_depth_and_eviction():
    """Depth: an inheritor given its anchor's query and up-projections reproduces
    the anchor's output exactly.  Eviction: the stored stream is the kept positions."""
    dims = P.Dims(P.MLA, 3, 4, 1, 128, latent_dim=64, rope_dim=64, nope_dim=16, v_dim=8,
                  qscheme=P.KIVI32, batch=2, max_tokens=80, keep_tokens=40)
    plan = [P.Action(bits=4, rank=64), P.Action(inherit=True), P.Action(bits=16, rank=32)]
    rng = np.random.default_rng(12)
    Cs = [_bf16(20 + l, (2, 80, 64)) for l in range(3)]
    Rs = [_bf16(30 + l, (2, 80, 64)) for l in range(3)]
    keeps = [np.stack([np.sort(rng.choice(80, 40, replace=False)) for _ in range(2)]) for _ in range(3)]
    arena = M.compress_arena(dims, plan, Cs, Rs, keeps)
    q = rng.standard_normal((3, 2, 4, 80))
    WK = rng.standard_normal((3, 4, 16, 64)) / 8
    WV = rng.standard_normal((3, 4, 8, 64)) / 8
    q[1], WK[1], WV[1] = q[0], WK[0], WV[0]
    out = M.decode_step(dims, plan, arena, q, WK, WV, 40, 0.1)
    assert np.array_equal(out[1], out[0])
    # layer 2 (bf16, d = 32) against attention over the kept bf16 rows
    for b in range(2):
        idx = keeps[2][b]
        ref = M.attention_reconstructed(q[2, b, :, :16], q[2, b, :, 16:], Cs[2][b][idx, :32],
                                        Rs[2][b][idx], WK[2], WV[2], 0.1)
        assert np.allclose(out[2, b], ref, rtol=1e-12, atol=1e-14)


# --- low-rank projection on write ------------------------------------------------

def test_projection_identity_returns_the_prefix():
    rng = np.random.default_rng(900)
    H, r = 96, 64
    X = Q.round_bf16(rng.standard_normal((10, H)).astype(np.float32)).astype(np.float64)
    W = np.zeros((r, H))
    W[:, :r] = np.eye(r)
    for d in (8, 32, 64):
        assert np.array_equal(M.project_latent(X, W, d), X[:, :d])


def test_projection_keeping_d_is_the_prefix_of_keeping_r():
    rng = np.random.default_rng(901)
    X, W = rng.standard_normal((7, 40)), rng.standard_normal((32, 40))
    full = M.project_latent(X, W, 32)
    for d in (4, 8, 16):
        assert np.array_equal(M.project_latent(X, W, d), full[:, :d])


def test_projection_brute_force_and_rounding():
    rng = np.random.default_rng(902)
    X, W = rng.standard_normal((3, 5)), rng.standard_normal((4, 5))
    got = M.project_latent(X, W, 4)
    for t in range(3):
        for i in range(4):
            exact = sum(W[i, k] * X[t, k] for k in range(5))
            # the nearest bf16 (8 significant bits): neighbours 2^(e-7) apart
            e = np.floor(np.log2(abs(exact)))
            ulp = 2.0 ** (e - 7)
            lo = np.floor(exact / ulp) * ulp
            cand = [lo, lo + ulp]
            assert got[t, i] in cand and abs(got[t, i] - exact) <= ulp / 2 + 1e-300
    # ties go to the even neighbour: 1 + 2^-8 -> 1, 1 + 3 * 2^-8 -> 1 + 2^-6
    one = np.ones((1, 1))
    assert M.project_latent(one, np.array([[1 + 2.0 ** -8]]), 1)[0, 0] == 1.0
    assert M.project_latent(one, np.array([[1 + 3 * 2.0 ** -8]]), 1)[0, 0] == 1 + 2.0 ** -6
    assert M.project_latent(one, np.array([[1 + 2.0 ** -8 + 2.0 ** -30]]), 1)[0, 0] == 1 + 2.0 ** -7


@pytest.mark.parametrize("bits", [16, 8, 4, 2])
@pytest.mark.parametrize("qs", [P.KIVI32, P.SYMROW])
def test_projected_write_is_the_latent_write_of_the_projection(bits, qs):
    rng = np.random.default_rng(903 + bits)
    B, n, H, r, d = 2, 70, 64, 64, 32
    dims = P.Dims(P.MLA, 1, 8, 1, 64, latent_dim=r, rope_dim=64, nope_dim=64, v_dim=64, qscheme=qs,
                   batch=B, max_tokens=96)
    X = rng.standard_normal((B, n, H))
    W = rng.standard_normal((r, H)) / 8.0
    R = Q.round_bf16(rng.standard_normal((B, n, 64)).astype(np.float32))
    C = np.stack([M.project_latent(X[b], W, d) for b in range(B)])
    assert np.array_equal(M.compress_layer_projected(dims, bits, d, X, W, R),
                          M.compress_layer(dims, bits, d, C, R))
