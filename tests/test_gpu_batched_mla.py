"""GPU parity of MLA tables whose sequences carry their own plans (§2.3: a plan per
input sequence; eq. (3)'s actions with the rank axis, so kept widths, bit-widths
and depth differ between sequences), through the C ABI.

Sequence b is stored exactly as a one-sequence table of its plan stores it (bytes
against the oracle), decodes as its own one-sequence batch (the oracle's decode of
that sequence within 2e-3 * max|out|, and bit for bit what a one-sequence table of
its plan returns), and tokens appended at decode time leave the cache the prefill of
the same tokens writes (decode outputs bit for bit).
"""
import numpy as np
import pytest
import torch

from oracle import mla as OM
from oracle import plan as OP
from paper_2609_37988_amd import kvk, synth

from gpu_common import TOL, rel_err, say

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
SCALE = 1.0 / np.sqrt(192.0)
PLANS = [[(0, 16, 512), (1, 16, 0), (0, 4, 256), (0, 8, 128)],
         [(0, 4, 64), (0, 2, 512), (1, 16, 0), (1, 16, 0)],
         [(0, 8, 256), (1, 16, 0), (0, 16, 128), (0, 4, 512)]]
L, HQ, R, B = 4, 32, 512, 3


def _np(x):
    return x.detach().float().cpu().numpy()


def _dims(batch, n_cap, qs=kvk.KIVI32):
    return kvk.make_dims(kvk.MLA, L, HQ, 4, 128, R, 64, 128, 128, qscheme=qs, batch=batch, max_tokens=n_cap)


def _inputs(n, seed=0):
    return [(synth.latent_random(seed + 10 + l, B, n, R), synth.latent_random(seed + 20 + l, B, n, 64)) for l in range(L)]


def _decode(t, q, wk, wv, n):
    d = t.dims
    out = torch.full((L, d.batch, HQ, 128), float("nan"), dtype=torch.float32, device=DEV)
    ws = torch.full((kvk.workspace_bytes(t, 0, L),), 0xFF, dtype=torch.uint8, device=DEV)
    kvk.decode_setup(t, 0, L, ws)  # the per-sequence work list (a no-op for one plan)
    kvk.decode_attention(t, 0, L, q.to(DEV).contiguous(), n, SCALE, _arena(t), out, ws,
                         w_uk=kvk.mla_weights_for_library(wk.to(DEV)), w_uv=wv.to(DEV).contiguous())
    return out


_ARENAS = {}


def _arena(t):
    return _ARENAS[id(t)]


def _new(t):
    _ARENAS[id(t)] = torch.zeros(max(kvk.table_query(t).arena_bytes, 256), dtype=torch.uint8, device=DEV)
    return _ARENAS[id(t)]


@pytest.mark.parametrize("qs", [kvk.KIVI32, kvk.SYMROW], ids=["kivi32", "symrow"])
def test_per_sequence_mla_plans(qs):
    """3 sequences x 4 layers, 150 tokens (4 blocks + a 22-token tail)."""
    say(f"case batched mla qs={qs}")
    n = 150
    t = kvk.layer_table_batched(_dims(B, 160, qs), [kvk.make_plan(p) for p in PLANS])
    arena = _new(t)
    inp = _inputs(n)
    for l in range(L):
        kvk.compress_layer(t, l, inp[l][0].to(DEV), inp[l][1].to(DEV), n, None, arena)
    od = OP.Dims(OP.MLA, L, HQ, 4, 128, latent_dim=R, rope_dim=64, nope_dim=128, v_dim=128, qscheme=qs,
                 batch=B, max_tokens=160)
    sd = OP.sequence_dims(od)
    oplans = [[OP.Action(bool(a), bb, r) for a, bb, r in p] for p in PLANS]
    bases, _ = OP.batched_arena_bases(od, oplans)
    q = synth.q_random(30, L, B, HQ, 192)
    wk = synth.weights_random(31, L, HQ, 128, R)
    wv = synth.weights_random(32, L, HQ, 128, R)
    out = _decode(t, q, wk, wv, n)
    got_arena = arena.cpu().numpy()
    for b in range(B):
        offs, total = OP.arena_offsets(sd, oplans[b])
        ref = np.zeros(total, dtype=np.uint8)
        for l in range(L):
            a = oplans[b][l]
            if a.inherit:
                continue
            reg = OM.compress_layer(sd, a.bits, a.rank, _np(inp[l][0][b:b + 1]), _np(inp[l][1][b:b + 1]))
            ref[offs[l]:offs[l] + reg.size] = reg
        assert np.array_equal(got_arena[bases[b]:bases[b] + total], ref), f"sequence {b} bytes differ"
        want = OM.decode_step(sd, oplans[b], ref, _np(q[:, b:b + 1]).astype(np.float64),
                              _np(wk).astype(np.float64), _np(wv).astype(np.float64), n, SCALE)
        err = rel_err(_np(out[:, b:b + 1]), want)
        say(f"  sequence {b}: max|diff| / max|out| = {err:.2e}")
        assert err <= TOL
        # bit for bit what a one-sequence table of its plan returns
        one = kvk.layer_table(_dims(1, 160, qs), kvk.make_plan(PLANS[b]))
        a1 = _new(one)
        for l in range(L):
            kvk.compress_layer(one, l, inp[l][0][b:b + 1].to(DEV), inp[l][1][b:b + 1].to(DEV), n, None, a1)
        assert torch.equal(_decode(one, q[:, b:b + 1], wk, wv, n)[:, 0], out[:, b]), f"sequence {b}"
    # the test dequantiser: sequence b's latent at b n r, rows of its own width
    for l in range(L):
        c = torch.full((B * n * R,), float("nan"), dtype=torch.float32, device=DEV)
        r = torch.empty((B * n * 64,), dtype=torch.float32, device=DEV)
        kvk.debug_dequantize(t, l, n, arena, c, r)
        for b in range(B):
            info = kvk.table_sequence_query(t, b)
            dd = PLANS[b][info.anchor_of[l]][2]
            offs, total = OP.arena_offsets(sd, oplans[b])
            Cr, Rr = OM.dequant_layer(sd, oplans[b], got_arena[bases[b]:bases[b] + total], l, n)
            assert np.array_equal(_np(c[b * n * R:b * n * R + n * dd]).reshape(n, dd), Cr[0])
            assert np.array_equal(_np(r[b * n * 64:(b + 1) * n * 64]).reshape(n, 64), Rr[0])


def test_per_sequence_mla_append_equals_prefill():
    """62 tokens prefilled, then 3 appended one at a time (the second completes block 1):
    every sequence decodes bit for bit as after a prefill of the same 65 tokens."""
    say("case batched mla append")
    n0, n = 62, 65
    inp = _inputs(n, seed=100)
    full = kvk.layer_table_batched(_dims(B, 96), [kvk.make_plan(p) for p in PLANS])
    part = kvk.layer_table_batched(_dims(B, 96), [kvk.make_plan(p) for p in PLANS])
    af, ap = _new(full), _new(part)
    for l in range(L):
        kvk.compress_layer(full, l, inp[l][0].to(DEV), inp[l][1].to(DEV), n, None, af)
        kvk.compress_layer(part, l, inp[l][0][:, :n0].contiguous().to(DEV), inp[l][1][:, :n0].contiguous().to(DEV),
                           n0, None, ap)
    for pos in range(n0, n):
        lat = torch.stack([inp[l][0][:, pos] for l in range(L)]).contiguous().to(DEV)   # [L, B, r]
        rop = torch.stack([inp[l][1][:, pos] for l in range(L)]).contiguous().to(DEV)   # [L, B, 64]
        kvk.append_token(part, 0, L, lat, rop, pos, ap)
    q = synth.q_random(130, L, B, HQ, 192)
    wk = synth.weights_random(131, L, HQ, 128, R)
    wv = synth.weights_random(132, L, HQ, 128, R)
    assert torch.equal(_decode(part, q, wk, wv, n), _decode(full, q, wk, wv, n))


def test_per_sequence_mla_projected_write():
    """The projected write on a per-sequence table stores, per sequence, the bytes of
    the same write on a one-sequence table of its plan (hidden width 256, 70 tokens)."""
    say("case batched mla projected write")
    n, H = 70, 256
    t = kvk.layer_table_batched(_dims(B, 96), [kvk.make_plan(p) for p in PLANS])
    arena = _new(t)
    X = synth.latent_random(200, B, n, H).to(DEV)
    W = synth.weights_random(201, 1, 1, R, H)[0, 0].contiguous().to(DEV)
    Rk = synth.latent_random(202, B, n, 64).to(DEV)
    for l in range(L):
        kvk.compress_layer_project(t, l, X, W, Rk, n, None, arena)
    got = arena.cpu().numpy()
    for b in range(B):
        one = kvk.layer_table(_dims(1, 96), kvk.make_plan(PLANS[b]))
        a1 = _new(one)
        for l in range(L):
            kvk.compress_layer_project(one, l, X[b:b + 1].contiguous(), W, Rk[b:b + 1].contiguous(), n, None, a1)
        base = kvk.table_sequence_query(t, b).layer_offset
        info1 = kvk.table_query(one)
        for l in range(L):
            if PLANS[b][l][0]:
                continue
            nb = info1.layer_bytes[l]
            assert np.array_equal(got[base[l]:base[l] + nb], a1[info1.layer_offset[l]:info1.layer_offset[l] + nb].cpu().numpy())


def test_per_sequence_projected_write_keep_lists_beyond_one_launch():
    """70 sequences (more than one launch serves) with their own keep lists (32 of 40
    positions, out of order): each sequence's bytes equal the same write on a
    one-sequence table of its plan given its own rows and keep list."""
    say("case batched mla projected write, 70 sequences, keep lists")
    nb, n, H, keep = 70, 40, 256, 32
    plans = [PLANS[b % len(PLANS)] for b in range(nb)]
    dims = kvk.make_dims(kvk.MLA, L, HQ, 4, 128, R, 64, 128, 128, qscheme=kvk.KIVI32, batch=nb,
                         max_tokens=n, keep_tokens=keep)
    t = kvk.layer_table_batched(dims, [kvk.make_plan(p) for p in plans])
    arena = _new(t)
    X = synth.latent_random(210, nb, n, H).to(DEV)
    W = synth.weights_random(211, 1, 1, R, H)[0, 0].contiguous().to(DEV)
    Rk = synth.latent_random(212, nb, n, 64).to(DEV)
    g = np.random.default_rng(213)
    K = torch.from_numpy(np.stack([g.permutation(n)[:keep] for _ in range(nb)]).astype(np.int32)).to(DEV)
    for l in range(L):
        kvk.compress_layer_project(t, l, X, W, Rk, n, K, arena)
    got = arena.cpu().numpy()
    d1 = kvk.make_dims(kvk.MLA, L, HQ, 4, 128, R, 64, 128, 128, qscheme=kvk.KIVI32, batch=1,
                       max_tokens=n, keep_tokens=keep)
    for b in range(nb):
        one = kvk.layer_table(d1, kvk.make_plan(plans[b]))
        a1 = _new(one)
        for l in range(L):
            kvk.compress_layer_project(one, l, X[b:b + 1].contiguous(), W, Rk[b:b + 1].contiguous(), n,
                                       K[b:b + 1].contiguous(), a1)
        base = kvk.table_sequence_query(t, b).layer_offset
        info1 = kvk.table_query(one)
        for l in range(L):
            if plans[b][l][0]:
                continue
            nbytes = info1.layer_bytes[l]
            assert np.array_equal(got[base[l]:base[l] + nbytes],
                                  a1[info1.layer_offset[l]:info1.layer_offset[l] + nbytes].cpu().numpy()), (b, l)


def _one_table_decode(plan, inp_b, q_b, wk, wv, n, cap, qs=kvk.KIVI32):
    """Decode of one sequence through a one-sequence table of its plan."""
    one = kvk.layer_table(kvk.make_dims(kvk.MLA, len(plan), HQ, 4, 128, R, 64, 128, 128, qscheme=qs, batch=1,
                                        max_tokens=cap), kvk.make_plan(plan))
    a1 = _new(one)
    for l, (c, r) in enumerate(inp_b):
        kvk.compress_layer(one, l, c.to(DEV), r.to(DEV), n, None, a1)
    nl = len(plan)
    out = torch.full((nl, 1, HQ, 128), float("nan"), dtype=torch.float32, device=DEV)
    ws = torch.full((kvk.workspace_bytes(one, 0, nl),), 0xFF, dtype=torch.uint8, device=DEV)
    kvk.decode_attention(one, 0, nl, q_b.to(DEV).contiguous(), n, SCALE, a1, out, ws,
                         w_uk=kvk.mla_weights_for_library(wk.to(DEV)), w_uv=wv.to(DEV).contiguous())
    return out


def test_per_sequence_mla_batched_launch_many_items():
    """8 sequences x 6 layers (every kept width and bit-width, depth groups of up to 3),
    5000 of 8192 tokens stored: the list is laid out for the capacity (3 splits of the
    4-bit width-512 streams) and the call runs 2; the split phase and the merge called
    separately; every sequence bit for bit its one-sequence table's decode, two of them
    against the oracle."""
    say("case batched mla many items")
    nl, B8, n, cap = 6, 8, 5000, 8192
    rng = np.random.default_rng(77)
    widths, bits = [512, 256, 128, 64], [16, 8, 4, 2]
    plans = []
    for b in range(B8):
        p, l = [], 0
        while l < nl:
            g = int(rng.integers(1, 4)) if l > 0 else 1
            p.append((0, int(rng.choice(bits)), int(rng.choice(widths))))
            p += [(1, 16, 0)] * (min(g, nl - l) - 1)
            l += min(g, nl - l)
        plans.append(p)
    plans[0][0] = (0, 4, 512)  # a 4-bit full-width anchor (several splits)
    d = kvk.make_dims(kvk.MLA, nl, HQ, 4, 128, R, 64, 128, 128, batch=B8, max_tokens=cap)
    t = kvk.layer_table_batched(d, [kvk.make_plan(p) for p in plans])
    arena = _new(t)
    inp = [(synth.latent_random(900 + l, B8, n, R), synth.latent_random(950 + l, B8, n, 64)) for l in range(nl)]
    for l in range(nl):
        kvk.compress_layer(t, l, inp[l][0].to(DEV), inp[l][1].to(DEV), n, None, arena)
    q = synth.q_random(901, nl, B8, HQ, 192)
    wk = synth.weights_random(902, nl, HQ, 128, R)
    wv = synth.weights_random(903, nl, HQ, 128, R)
    wk_lib, wv_d = kvk.mla_weights_for_library(wk.to(DEV)), wv.to(DEV).contiguous()
    ws = torch.full((kvk.workspace_bytes(t, 0, nl),), 0xFF, dtype=torch.uint8, device=DEV)
    kvk.decode_setup(t, 0, nl, ws)
    out = torch.full((nl, B8, HQ, 128), float("nan"), dtype=torch.float32, device=DEV)
    kvk.decode_attention(t, 0, nl, q.to(DEV), n, SCALE, arena, out, ws, w_uk=wk_lib, w_uv=wv_d)
    out2 = torch.full_like(out, float("nan"))
    kvk.decode_splits(t, 0, nl, q.to(DEV), n, SCALE, arena, ws, w_uk=wk_lib, w_uv=wv_d)
    kvk.decode_merge(t, 0, nl, q.to(DEV), n, SCALE, arena, ws, out2, w_uk=wk_lib, w_uv=wv_d)
    assert torch.equal(out, out2)
    for b in range(B8):
        ref = _one_table_decode(plans[b], [(inp[l][0][b:b + 1].contiguous(), inp[l][1][b:b + 1].contiguous())
                                           for l in range(nl)], q[:, b:b + 1], wk, wv, n, cap)
        assert torch.equal(ref[:, 0], out[:, b]), f"sequence {b} differs from its one-sequence table"
    od = OP.Dims(OP.MLA, nl, HQ, 4, 128, latent_dim=R, rope_dim=64, nope_dim=128, v_dim=128, batch=B8,
                 max_tokens=cap)
    sd = OP.sequence_dims(od)
    oplans = [[OP.Action(bool(a), bb, r) for a, bb, r in p] for p in plans]
    bases, _ = OP.batched_arena_bases(od, oplans)
    got_arena = arena.cpu().numpy()
    for b in (0, 5):
        offs, total = OP.arena_offsets(sd, oplans[b])
        want = OM.decode_step(sd, oplans[b], got_arena[bases[b]:bases[b] + total], _np(q[:, b:b + 1]).astype(np.float64),
                              _np(wk).astype(np.float64), _np(wv).astype(np.float64), n, SCALE)
        err = rel_err(_np(out[:, b:b + 1]), want)
        say(f"  sequence {b}: max|diff| / max|out| = {err:.2e}")
        assert err <= TOL


def test_per_sequence_mla_needs_setup_and_its_list():
    """A per-sequence MLA decode needs kvk_decode_setup of the same workspace and layer
    range; a workspace whose list was overwritten since makes the kernels return NaN
    outputs and read nothing through it."""
    say("case batched mla setup")
    n = 100
    t = kvk.layer_table_batched(_dims(B, 128), [kvk.make_plan(p) for p in PLANS])
    arena = _new(t)
    inp = _inputs(n, seed=300)
    for l in range(L):
        kvk.compress_layer(t, l, inp[l][0].to(DEV), inp[l][1].to(DEV), n, None, arena)
    q = synth.q_random(301, L, B, HQ, 192).to(DEV)
    wk = kvk.mla_weights_for_library(synth.weights_random(302, L, HQ, 128, R).to(DEV))
    wv = synth.weights_random(303, L, HQ, 128, R).to(DEV).contiguous()
    ws = torch.zeros(kvk.workspace_bytes(t, 0, L), dtype=torch.uint8, device=DEV)
    out = torch.zeros((L, B, HQ, 128), dtype=torch.float32, device=DEV)
    with pytest.raises(kvk.KvkError, match="kvk_decode_setup"):
        kvk.decode_attention(t, 0, L, q, n, SCALE, arena, out, ws, w_uk=wk, w_uv=wv)
    kvk.decode_setup(t, 1, L, ws)
    with pytest.raises(kvk.KvkError, match="kvk_decode_setup"):
        kvk.decode_attention(t, 0, L, q, n, SCALE, arena, out, ws, w_uk=wk, w_uv=wv)
    kvk.decode_setup(t, 0, L, ws)
    kvk.decode_attention(t, 0, L, q, n, SCALE, arena, out, ws, w_uk=wk, w_uv=wv)
    torch.cuda.synchronize()
    assert torch.isfinite(out).all()
    ws[:256].zero_()  # the list's header overwritten
    kvk.decode_attention(t, 0, L, q, n, SCALE, arena, out, ws, w_uk=wk, w_uv=wv)
    torch.cuda.synchronize()
    assert torch.isnan(out).all()


def test_per_sequence_mla_14b_latent_shape():
    """Qwen2.5-14B's latent shape (40 heads padded to two 32-head chunks, r 1024 + 64):
    per-sequence plans with width-1024 anchors (the wide kernel reading its items from
    the workspace), depth and every bit-width; every sequence bit for bit its
    one-sequence table's decode, one against the oracle."""
    say("case batched mla 14b latent")
    nl, B3, n, cap, hq, r = 3, 3, 150, 160, 40, 1024
    plans = [[(0, 16, 1024), (1, 16, 0), (0, 4, 256)],
             [(0, 8, 512), (0, 4, 1024), (1, 16, 0)],
             [(0, 2, 1024), (0, 16, 128), (0, 8, 1024)]]
    d = kvk.make_dims(kvk.MLA, nl, hq, 8, 128, r, 64, 128, 128, batch=B3, max_tokens=cap)
    t = kvk.layer_table_batched(d, [kvk.make_plan(p) for p in plans])
    arena = _new(t)
    inp = [(synth.latent_random(1300 + l, B3, n, r), synth.latent_random(1350 + l, B3, n, 64)) for l in range(nl)]
    for l in range(nl):
        kvk.compress_layer(t, l, inp[l][0].to(DEV), inp[l][1].to(DEV), n, None, arena)
    q = synth.q_random(1301, nl, B3, hq, 192)
    wk = synth.weights_random(1302, nl, hq, 128, r)
    wv = synth.weights_random(1303, nl, hq, 128, r)
    ws = torch.full((kvk.workspace_bytes(t, 0, nl),), 0xFF, dtype=torch.uint8, device=DEV)
    kvk.decode_setup(t, 0, nl, ws)
    out = torch.full((nl, B3, hq, 128), float("nan"), dtype=torch.float32, device=DEV)
    kvk.decode_attention(t, 0, nl, q.to(DEV), n, SCALE, arena, out, ws,
                         w_uk=kvk.mla_weights_for_library(wk.to(DEV)), w_uv=wv.to(DEV).contiguous())
    for b in range(B3):
        one = kvk.layer_table(kvk.make_dims(kvk.MLA, nl, hq, 8, 128, r, 64, 128, 128, batch=1, max_tokens=cap),
                              kvk.make_plan(plans[b]))
        a1 = _new(one)
        for l in range(nl):
            kvk.compress_layer(one, l, inp[l][0][b:b + 1].contiguous().to(DEV), inp[l][1][b:b + 1].contiguous().to(DEV),
                               n, None, a1)
        o1 = torch.full((nl, 1, hq, 128), float("nan"), dtype=torch.float32, device=DEV)
        w1 = torch.full((kvk.workspace_bytes(one, 0, nl),), 0xFF, dtype=torch.uint8, device=DEV)
        kvk.decode_attention(one, 0, nl, q[:, b:b + 1].contiguous().to(DEV), n, SCALE, a1, o1, w1,
                             w_uk=kvk.mla_weights_for_library(wk.to(DEV)), w_uv=wv.to(DEV).contiguous())
        assert torch.equal(o1[:, 0], out[:, b]), f"sequence {b} differs from its one-sequence table"
    od = OP.Dims(OP.MLA, nl, hq, 8, 128, latent_dim=r, rope_dim=64, nope_dim=128, v_dim=128, batch=B3,
                 max_tokens=cap)
    sd = OP.sequence_dims(od)
    oplans = [[OP.Action(bool(a), bb, rr) for a, bb, rr in p] for p in plans]
    bases, _ = OP.batched_arena_bases(od, oplans)
    got = arena.cpu().numpy()
    b = 2
    offs, total = OP.arena_offsets(sd, oplans[b])
    want = OM.decode_step(sd, oplans[b], got[bases[b]:bases[b] + total], _np(q[:, b:b + 1]).astype(np.float64),
                          _np(wk).astype(np.float64), _np(wv).astype(np.float64), n, SCALE)
    err = rel_err(_np(out[:, b:b + 1]), want)
    say(f"  sequence {b}: max|diff| / max|out| = {err:.2e}")
    assert err <= TOL
