"""GPU parity of the decode-time append (kvk_append_token) against the oracle's
append rule, through the C ABI.

Bit-exact: every full block and every valid tail token of each anchor's streams
after a sequence of appends that crosses several group boundaries (the oracle
replays the same appends with oracle.cache.append_token / oracle.mla.append_token,
starting from its own prefill write).  Decode after the appends: max|diff| <=
2e-3 * max|out| against oracle attention over the oracle's appended streams.
"""
import numpy as np
import pytest
import torch

from oracle import cache as OC
from oracle import layout as LY
from oracle import mla as OM
from oracle import plan as OP
from paper_2609_37988_amd import kvk, synth

from gpu_common import DEV, TOL, Case, oracle_rows, rel_err, say
from test_gpu_mla import SCALE, MlaCase

pytestmark = pytest.mark.gpu


def _np(x):
    return x.detach().float().cpu().numpy()


def _gqa_valid(odims, bits, stream, n):
    blocks, tail = LY.split_stream(odims, bits, stream, n)
    kt, vt = LY.unpack_bf16_blocks(tail[None], odims.head_dim)
    return blocks, kt[0, :n % 32], vt[0, :n % 32]


def _gqa_append_case(qs, bits_a, bits_b, D, dtype, n0, n1, seed):
    """Layers: anchor (bits_a), inheritor, anchor (bits_b).  Prefill n0 tokens, then
    append tokens n0 .. n1-1 one call per token over all three layers."""
    B, Hkv, Hq = 2, 2, 6
    case = Case(3, Hq, Hkv, D, B, n1 + 8, [(0, bits_a), (1, 16), (0, bits_b)], qscheme=qs)
    inputs = {}
    for l in (0, 2):
        k, v = synth.kv_random(seed + l, B, Hkv, n1, D, dtype=dtype)
        inputs[l] = (k, v)
        if n0 > 0:
            case.compress(l, k[:, :, :n0].to(DEV), v[:, :, :n0].to(DEV), n0)
    for n in range(n0, n1):
        kn = torch.randn((3, B, Hkv, D), dtype=torch.float32).to(dtype)  # row 1 (inheritor) is not read
        vn = torch.randn((3, B, Hkv, D), dtype=torch.float32).to(dtype)
        for l in (0, 2):
            kn[l], vn[l] = inputs[l][0][:, :, n], inputs[l][1][:, :, n]
        kvk.append_token(case.table, 0, 3, kn.to(DEV).contiguous(), vn.to(DEV).contiguous(), n, case.arena)
    # the oracle replays the appends from its own prefill write
    streams = {}
    for l in (0, 2):
        bits = case.plan[l].bits
        kn, vn = _np(inputs[l][0]), _np(inputs[l][1])
        for b in range(B):
            for h in range(Hkv):
                st = OC.compress_stream(case.odims, bits, kn[b, h, :n0], vn[b, h, :n0])
                for n in range(n0, n1):
                    st = OC.append_token(case.odims, bits, st, n, kn[b, h, n], vn[b, h, n])
                streams[(l, b, h)] = st
                got = case.stream_bytes_host(l, b, h)
                for x, y in zip(_gqa_valid(case.odims, bits, got, n1), _gqa_valid(case.odims, bits, st, n1)):
                    assert np.array_equal(x, y), f"stored tokens differ (layer {l}, b {b}, h {h})"
    return case, streams


@pytest.mark.parametrize("qs", [kvk.KIVI32, kvk.SYMROW, kvk.GROUP64], ids=["kivi32", "symrow", "group64"])
@pytest.mark.parametrize("bits_a,bits_b", [(16, 2), (8, 4), (4, 16), (2, 8)])
def test_gqa_append_matches_oracle_and_decodes(qs, bits_a, bits_b):
    """29 prefilled tokens, 70 appends (group boundaries at 32, 64 and 96), d_h 128."""
    say(f"case gqa append qs={qs} bits={bits_a},{bits_b}")
    n0, n1, D = 29, 99, 128
    case, streams = _gqa_append_case(qs, bits_a, bits_b, D, torch.bfloat16, n0, n1, 300 + bits_a)
    q = synth.q_random(310 + bits_b, 3, 2, 6, D)
    out = _np(case.decode(q.to(DEV), n1, 1.0 / np.sqrt(D)))
    qn = _np(q).astype(np.float64)
    ref = np.zeros_like(out, dtype=np.float64)
    for l in range(3):
        a = case.info.anchor_of[l]
        for b in range(2):
            for h in range(2):
                ref[l, b, 3 * h:3 * h + 3] = oracle_rows(case.odims, case.plan[a].bits, streams[(a, b, h)], n1,
                                                         qn[l, b, 3 * h:3 * h + 3], 1.0 / np.sqrt(D))
    err = rel_err(out, ref)
    say(f"  max|diff| / max|out| = {err:.2e}")
    assert err <= TOL


def test_gqa_append_from_empty_fp32_input():
    """No prefill; 40 fp32 tokens appended (stored as their bf16 values), d_h 64."""
    say("case gqa append from empty, fp32 input")
    _gqa_append_case(kvk.KIVI32, 4, 8, 64, torch.float32, 0, 40, 400)


def test_generation_loop_decode_append():
    """Three steps of decode at n, append token n, decode at n + 1: every decode
    matches the oracle over the oracle's appended streams (steps cross a group
    boundary at 32)."""
    say("case gqa generation loop")
    D, B, Hkv, Hq, n0 = 128, 1, 2, 4, 30
    case = Case(2, Hq, Hkv, D, B, 64, [(0, 4), (1, 16)])
    k, v = synth.kv_random(500, B, Hkv, n0 + 3, D)
    case.compress(0, k[:, :, :n0].to(DEV), v[:, :, :n0].to(DEV), n0)
    kn, vn = _np(k), _np(v)
    st = {h: OC.compress_stream(case.odims, 4, kn[0, h, :n0], vn[0, h, :n0]) for h in range(Hkv)}
    for step in range(3):
        n = n0 + step
        q = synth.q_random(510 + step, 2, B, Hq, D)
        out = _np(case.decode(q.to(DEV), n, 1.0 / np.sqrt(D)))
        qn = _np(q).astype(np.float64)
        for l in range(2):
            for h in range(Hkv):
                ref = oracle_rows(case.odims, 4, st[h], n, qn[l, 0, 2 * h:2 * h + 2], 1.0 / np.sqrt(D))
                assert rel_err(out[l, 0, 2 * h:2 * h + 2], ref) <= TOL, f"step {step} layer {l}"
        kt = torch.zeros((2, B, Hkv, D), dtype=torch.bfloat16)
        vt = torch.zeros((2, B, Hkv, D), dtype=torch.bfloat16)
        kt[0], vt[0] = k[:, :, n], v[:, :, n]
        kvk.append_token(case.table, 0, 2, kt.to(DEV), vt.to(DEV), n, case.arena)
        for h in range(Hkv):
            st[h] = OC.append_token(case.odims, 4, st[h], n, kn[0, h, n], vn[0, h, n])


def _mla_valid(odims, bits, d, stream, n):
    W = d + odims.rope_dim
    blk = OP.block_bytes(odims, bits, d)
    t0 = (odims.stored_cap // 32) * blk
    tail = OM.unpack_bf16_block(stream[None, t0:t0 + OP.tail_bytes(odims, d)], W)[0]
    return stream[:(n // 32) * blk], tail[:n % 32]


@pytest.mark.parametrize("qs", [kvk.KIVI32, kvk.SYMROW], ids=["kivi32", "symrow"])
def test_mla_append_matches_oracle_and_decodes(qs):
    """MLA stack: bf16 d 512, inheritor, int4 d 256, int2 d 64; 27 prefilled tokens
    and 40 appends (boundaries at 32 and 64)."""
    say(f"case mla append qs={qs}")
    plan = [(0, 16, 512), (1, 16, 0), (0, 4, 256), (0, 2, 64)]
    B, r, n0, n1 = 2, 512, 27, 67
    c = MlaCase(4, 32, r, B, 96, plan, qscheme=qs)
    inputs = {}
    for l in (0, 2, 3):
        C, R = synth.latent_random(600 + l, B, n1, r), synth.latent_random(610 + l, B, n1, 64)
        inputs[l] = (C, R)
        c.compress(l, C[:, :n0], R[:, :n0], n0)
    for n in range(n0, n1):
        Cn = torch.zeros((4, B, r), dtype=torch.bfloat16)
        Rn = torch.zeros((4, B, 64), dtype=torch.bfloat16)
        for l in (0, 2, 3):
            Cn[l], Rn[l] = inputs[l][0][:, n], inputs[l][1][:, n]
        kvk.append_token(c.table, 0, 4, Cn.to(DEV), Rn.to(DEV), n, c.arena)
    offs, total = OP.arena_offsets(c.odims, c.oplan)
    oarena = np.zeros(total, dtype=np.uint8)
    for l in (0, 2, 3):
        a = c.oplan[l]
        Cn, Rn = _np(inputs[l][0]), _np(inputs[l][1])
        sb = OP.stream_bytes(c.odims, a.bits, a.rank)
        for b in range(B):
            st = OM.compress_stream(c.odims, a.bits, a.rank, Cn[b, :n0], Rn[b, :n0])
            for n in range(n0, n1):
                st = OM.append_token(c.odims, a.bits, a.rank, st, n, Cn[b, n], Rn[b, n])
            off = offs[l] + b * sb
            oarena[off:off + sb] = st
            got = c.arena[off:off + sb].cpu().numpy()
            for x, y in zip(_mla_valid(c.odims, a.bits, a.rank, got, n1), _mla_valid(c.odims, a.bits, a.rank, st, n1)):
                assert np.array_equal(x, y), f"stored tokens differ (layer {l}, b {b})"
    q = synth.q_random(620, 4, B, 32, 192)
    wk = synth.weights_random(621, 4, 32, 128, r)
    wv = synth.weights_random(622, 4, 32, 128, r)
    out = _np(c.decode(q, wk, wv, n1, SCALE))
    ref = OM.decode_step(c.odims, c.oplan, oarena, _np(q).astype(np.float64), _np(wk).astype(np.float64),
                         _np(wv).astype(np.float64), n1, SCALE)
    err = rel_err(out, ref)
    say(f"  max|diff| / max|out| = {err:.2e}")
    assert err <= TOL
