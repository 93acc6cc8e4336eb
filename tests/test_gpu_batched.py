"""GPU parity of batches whose sequences carry their own plans (kvk_layer_table_batched)
against the oracle (oracle.cache.compress_arena_batched / decode_step_batched).

Bit-exact: every stored stream of every sequence (its own plan's anchors) and the
dequantised values.  Decode (one launch for the whole batch): max|diff| <=
2e-3 * max|out|.
"""
import numpy as np
import pytest
import torch

from oracle import cache as OC
from oracle import layout as LY
from oracle import plan as OP
from paper_2609_37988_amd import kvk, synth

from gpu_common import DEV, TOL, meaningful, rel_err, say

pytestmark = pytest.mark.gpu

PLANS = [
    [(0, 4), (1, 16), (0, 8), (1, 16), (0, 2), (1, 16)],
    [(0, 16), (0, 2), (1, 16), (1, 16), (1, 16), (0, 4)],
    [(0, 8), (0, 8), (0, 4), (0, 16), (1, 16), (1, 16)],
    [(0, 2), (1, 16), (1, 16), (1, 16), (1, 16), (1, 16)],
]


class BatchCase:
    def __init__(self, plans, Hq, Hkv, D, max_tokens, qscheme=kvk.KIVI32, keep=0):
        B, L = len(plans), len(plans[0])
        self.B, self.L = B, L
        self.dims = kvk.make_dims(kvk.GQA, L, Hq, Hkv, D, qscheme=qscheme, batch=B, max_tokens=max_tokens,
                                  keep_tokens=keep)
        self.table = kvk.layer_table_batched(self.dims, [kvk.make_plan(p) for p in plans])
        self.info = kvk.table_query(self.table)
        self.arena = torch.zeros(max(self.info.arena_bytes, 256), dtype=torch.uint8, device=DEV)
        self.od = OP.Dims(OP.GQA, L, Hq, Hkv, D, qscheme=qscheme, batch=B, max_tokens=max_tokens, keep_tokens=keep)
        self.oplans = [[OP.Action(bool(a), b) for a, b in p] for p in plans]

    def workspace(self, l0, l1):
        """A workspace set up once for the range (the per-sequence work list at its head)."""
        if not hasattr(self, "_ws"):
            self._ws = {}
        if (l0, l1) not in self._ws:
            ws = torch.full((max(kvk.workspace_bytes(self.table, l0, l1), 256),), 0xFF, dtype=torch.uint8,
                            device=DEV)
            kvk.decode_setup(self.table, l0, l1, ws)
            self._ws[(l0, l1)] = ws
        return self._ws[(l0, l1)]

    def decode(self, q, n, scale, l0=0, l1=None):
        l1 = self.L if l1 is None else l1
        d = self.dims
        out = torch.full((l1 - l0, d.batch, d.n_q_heads, d.head_dim), float("nan"), dtype=torch.float32,
                         device=DEV)
        kvk.decode_attention(self.table, l0, l1, q.to(DEV).contiguous(), n, scale, self.arena, out,
                             self.workspace(l0, l1))
        return out.cpu().numpy()

    def check_streams(self, oarena, n):
        bases, _ = OP.batched_arena_bases(self.od, self.oplans)
        sd = OP.sequence_dims(self.od)
        host = self.arena.cpu().numpy()
        for b in range(self.B):
            si = kvk.table_sequence_query(self.table, b)
            for l, a in enumerate(self.oplans[b]):
                if a.inherit:
                    continue
                for h in range(self.dims.n_kv_heads):
                    off = si.layer_offset[l] + h * si.stream_bytes[l]
                    got = host[off:off + si.stream_bytes[l]]
                    want = oarena[off:off + si.stream_bytes[l]]
                    assert np.array_equal(meaningful(sd, a.bits, got, n), meaningful(sd, a.bits, want, n)), \
                        f"stream differs (b {b}, layer {l}, h {h})"


def _inputs(case, n, seed, keep=None):
    Ks, Vs = [], []
    for l in range(case.L):
        k, v = synth.kv_random(seed + l, case.B, case.dims.n_kv_heads, n, case.dims.head_dim)
        Ks.append(k)
        Vs.append(v)
    return Ks, Vs


@pytest.mark.parametrize("qs", [kvk.KIVI32, kvk.SYMROW], ids=["kivi32", "symrow"])
def test_batched_plans_match_oracle(qs):
    """4 sequences, 6 layers, each sequence its own plan (every bit-width, inheritors),
    ragged length 300; one decode over all layers and one over layers 1..4."""
    say(f"case batched plans qs={qs}")
    n, D = 300, 128
    c = BatchCase(PLANS, 8, 2, D, 320, qscheme=qs)
    Ks, Vs = _inputs(c, n, 1100 + qs)
    for l in range(c.L):
        kvk.compress_layer(c.table, l, Ks[l].to(DEV), Vs[l].to(DEV), n, None, c.arena)
    oarena = OC.compress_arena_batched(c.od, c.oplans, [K.float().numpy() for K in Ks],
                                       [V.float().numpy() for V in Vs])
    c.check_streams(oarena, n)
    q = synth.q_random(1150, c.L, c.B, 8, D)
    scale = 1.0 / np.sqrt(D)
    out = c.decode(q, n, scale)
    ref = OC.decode_step_batched(c.od, c.oplans, oarena, q.float().numpy().astype(np.float64), n, scale)
    err = rel_err(out, ref)
    say(f"  max|diff| / max|out| = {err:.2e}")
    assert err <= TOL
    sub = c.decode(q[1:5], n, scale, 1, 5)
    ref_sub = OC.decode_step_batched(c.od, c.oplans, oarena, q[1:5].float().numpy().astype(np.float64), n,
                                     scale, 1, 5)
    assert rel_err(sub, ref_sub) <= TOL
    # dequantised values of every sequence equal the oracle's
    kd = torch.empty((c.B, 2, n, D), dtype=torch.float32, device=DEV)
    vd = torch.empty_like(kd)
    for l in range(c.L):
        kvk.debug_dequantize(c.table, l, n, c.arena, kd, vd)
        for b in range(c.B):
            sd = OP.sequence_dims(c.od)
            bases, _ = OP.batched_arena_bases(c.od, c.oplans)
            Kr, Vr = OC.dequant_layer(sd, c.oplans[b], oarena[bases[b]:], l, n)
            assert np.array_equal(kd[b].cpu().numpy(), Kr[0]) and np.array_equal(vd[b].cpu().numpy(), Vr[0])


def test_write_of_more_sequences_than_one_launch_serves():
    """70 sequences with their own plans (layer 0 int4 in every plan: 70 sequences of
    one bit-width, more than the 64 one write launch serves; layer 1 int2 or bf16 by
    sequence), ragged length 90: every stream bit-exact against the oracle's write."""
    say("case batched write, 70 sequences")
    n, D = 90, 64
    plans = [[(0, 4), (0, 2 if b % 2 == 0 else 16)] for b in range(70)]
    c = BatchCase(plans, 2, 1, D, 96)
    Ks, Vs = _inputs(c, n, 1300)
    for l in range(c.L):
        kvk.compress_layer(c.table, l, Ks[l].to(DEV), Vs[l].to(DEV), n, None, c.arena)
    oarena = OC.compress_arena_batched(c.od, c.oplans, [K.float().numpy() for K in Ks],
                                       [V.float().numpy() for V in Vs])
    c.check_streams(oarena, n)


def test_equal_plans_agree_with_one_plan():
    """All sequences on the same plan: the per-sequence batch decodes like the table
    with that one plan (within the tolerance; its splits differ)."""
    say("case batched = uniform")
    n, D, plan = 500, 128, PLANS[0]
    c = BatchCase([plan] * 3, 8, 2, D, 512)
    u = kvk.layer_table(c.dims, kvk.make_plan(plan))
    ua = torch.zeros(kvk.table_query(u).arena_bytes, dtype=torch.uint8, device=DEV)
    Ks, Vs = _inputs(c, n, 1200)
    for l in range(c.L):
        kvk.compress_layer(c.table, l, Ks[l].to(DEV), Vs[l].to(DEV), n, None, c.arena)
        kvk.compress_layer(u, l, Ks[l].to(DEV), Vs[l].to(DEV), n, None, ua)
    q = synth.q_random(1201, c.L, 3, 8, D)
    out = c.decode(q, n, 1.0 / np.sqrt(D))
    uo = torch.empty((c.L, 3, 8, D), dtype=torch.float32, device=DEV)
    ws = torch.empty(kvk.workspace_bytes(u, 0, c.L), dtype=torch.uint8, device=DEV)
    kvk.decode_setup(u, 0, c.L, ws)  # a no-op for a one-plan table
    kvk.decode_attention(u, 0, c.L, q.to(DEV), n, 1.0 / np.sqrt(D), ua, uo, ws)
    assert rel_err(out, uo.cpu().numpy()) <= TOL


def test_batched_eviction_write():
    """Per-sequence plans with eviction: keep 200 of 260 positions per (sequence, KV
    head); every sequence's streams equal the oracle's gathered write."""
    say("case batched eviction")
    n, keep, D = 260, 200, 64
    c = BatchCase(PLANS, 4, 2, D, n, keep=keep)
    Ks, Vs = _inputs(c, n, 1300)
    keeps = [synth.keep_random(1310 + l, c.B, 2, n, keep) for l in range(c.L)]
    for l in range(c.L):
        kvk.compress_layer(c.table, l, Ks[l].to(DEV), Vs[l].to(DEV), n, keeps[l].to(DEV), c.arena)
    oarena = OC.compress_arena_batched(c.od, c.oplans, [K.float().numpy() for K in Ks],
                                       [V.float().numpy() for V in Vs], [k.numpy() for k in keeps])
    c.check_streams(oarena, keep)
    q = synth.q_random(1320, c.L, c.B, 4, D)
    out = c.decode(q, keep, 0.125)
    ref = OC.decode_step_batched(c.od, c.oplans, oarena, q.float().numpy().astype(np.float64), keep, 0.125)
    assert rel_err(out, ref) <= TOL


def _oracle_arena_at(c, Ks, Vs, n0, n):
    """The oracle's batched arena after a prefill of n0 tokens and appends up to n."""
    bases, total = OP.batched_arena_bases(c.od, c.oplans)
    sd = OP.sequence_dims(c.od)
    oarena = np.zeros(total, dtype=np.uint8)
    for b in range(c.B):
        si = kvk.table_sequence_query(c.table, b)
        for l, a in enumerate(c.oplans[b]):
            if a.inherit:
                continue
            for h in range(c.dims.n_kv_heads):
                kn, vn = Ks[l][b, h].float().numpy(), Vs[l][b, h].float().numpy()
                st = OC.compress_stream(sd, a.bits, kn[:n0], vn[:n0])
                for i in range(n0, n):
                    st = OC.append_token(sd, a.bits, st, i, kn[i], vn[i])
                off = si.layer_offset[l] + h * si.stream_bytes[l]
                oarena[off:off + st.size] = st
    return oarena


def test_generation_decodes_every_step_on_one_setup():
    """Per-sequence plans through a generation: one kvk_decode_setup, then decode and
    append alternate for 40 steps from 250 prefilled tokens (group boundaries at 256
    and 288, a tail-only step would need fewer than 32 tokens); the decode at 250,
    255, 256, 257, 288 and 289 tokens equals the oracle's at that length.  The work
    list is laid out for the capacity, so nothing is copied per step."""
    say("case batched generation")
    n0, n1, D = 250, 290, 64
    c = BatchCase(PLANS, 4, 2, D, 320)
    Ks, Vs = _inputs(c, n1, 1450)
    for l in range(c.L):
        kvk.compress_layer(c.table, l, Ks[l][:, :, :n0].contiguous().to(DEV),
                           Vs[l][:, :, :n0].contiguous().to(DEV), n0, None, c.arena)
    c.workspace(0, c.L)  # the one set-up
    checks = {250, 255, 256, 257, 288, 289}
    for i in range(n0, n1):
        if i in checks:
            q = synth.q_random(1460 + i, c.L, c.B, 4, D)
            out = c.decode(q, i, 0.125)
            ref = OC.decode_step_batched(c.od, c.oplans, _oracle_arena_at(c, Ks, Vs, n0, i),
                                         q.float().numpy().astype(np.float64), i, 0.125)
            err = rel_err(out, ref)
            say(f"  step {i}: max|diff| / max|out| = {err:.2e}")
            assert err <= TOL
        kt = torch.stack([K[:, :, i] for K in Ks]).contiguous()  # [L, B, Hkv, D]
        vt = torch.stack([V[:, :, i] for V in Vs]).contiguous()
        kvk.append_token(c.table, 0, c.L, kt.to(DEV), vt.to(DEV), i, c.arena)


def test_setup_is_required_and_bound_to_its_range():
    """A per-sequence decode needs kvk_decode_setup of the same workspace and layer
    range; a set-up of another range on that workspace replaces it; a workspace whose
    list was overwritten since gives NaN outputs (the kernels read nothing through
    it)."""
    say("case batched setup rules")
    n, D = 100, 64
    c = BatchCase(PLANS, 4, 2, D, 128)
    Ks, Vs = _inputs(c, n, 1480)
    for l in range(c.L):
        kvk.compress_layer(c.table, l, Ks[l].to(DEV), Vs[l].to(DEV), n, None, c.arena)
    q = synth.q_random(1481, c.L, c.B, 4, D).to(DEV)
    out = torch.zeros((c.L, c.B, 4, D), dtype=torch.float32, device=DEV)
    ws = torch.zeros(kvk.workspace_bytes(c.table, 0, c.L), dtype=torch.uint8, device=DEV)
    with pytest.raises(kvk.KvkError, match="kvk_decode_setup"):
        kvk.decode_attention(c.table, 0, c.L, q, n, 0.125, c.arena, out, ws)
    kvk.decode_setup(c.table, 0, c.L, ws)
    kvk.decode_attention(c.table, 0, c.L, q, n, 0.125, c.arena, out, ws)
    good = out.clone()
    sub = torch.zeros((3, c.B, 4, D), dtype=torch.float32, device=DEV)
    with pytest.raises(kvk.KvkError, match="kvk_decode_setup"):
        kvk.decode_attention(c.table, 1, 4, q[1:4].contiguous(), n, 0.125, c.arena, sub, ws)
    kvk.decode_setup(c.table, 1, 4, ws)  # replaces the record of [0, L)
    kvk.decode_attention(c.table, 1, 4, q[1:4].contiguous(), n, 0.125, c.arena, sub, ws)
    assert torch.equal(sub, good[1:4])
    with pytest.raises(kvk.KvkError, match="kvk_decode_setup"):
        kvk.decode_attention(c.table, 0, c.L, q, n, 0.125, c.arena, out, ws)
    kvk.decode_setup(c.table, 0, c.L, ws)
    ws.zero_()  # the list is gone, the record remains
    kvk.decode_attention(c.table, 0, c.L, q, n, 0.125, c.arena, out, ws)
    torch.cuda.synchronize()
    assert torch.isnan(out).all()


def test_per_sequence_decode_step_in_a_graph():
    """A per-sequence decode step (after its set-up) captured in a HIP graph: the call
    copies nothing and does not synchronise, so it records; three replays, each after
    new queries are written into the captured buffer, equal the eager decode."""
    say("case batched decode in a graph")
    n, D = 300, 128
    c = BatchCase(PLANS, 8, 2, D, 320)
    Ks, Vs = _inputs(c, n, 1490)
    for l in range(c.L):
        kvk.compress_layer(c.table, l, Ks[l].to(DEV), Vs[l].to(DEV), n, None, c.arena)
    ws = c.workspace(0, c.L)
    qbuf = synth.q_random(1491, c.L, c.B, 8, D).to(DEV)
    out = torch.zeros((c.L, c.B, 8, D), dtype=torch.float32, device=DEV)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):  # warm-up on the capture stream
        kvk.decode_attention(c.table, 0, c.L, qbuf, n, 0.088, c.arena, out, ws)
    torch.cuda.current_stream().wait_stream(side)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        kvk.decode_attention(c.table, 0, c.L, qbuf, n, 0.088, c.arena, out, ws)
    for r in range(3):
        qbuf.copy_(synth.q_random(1500 + r, c.L, c.B, 8, D).to(DEV))
        graph.replay()
        torch.cuda.synchronize()
        want = c.decode(qbuf.clone(), n, 0.088)
        assert np.array_equal(out.cpu().numpy(), want), f"replay {r} differs from the eager decode"


def test_batched_append():
    """Per-sequence plans: 250 prefilled tokens, then 40 appended (group boundaries at
    256 and 288); stored blocks and tail tokens equal the oracle's appends, decode at
    290 within tolerance."""
    say("case batched append")
    n0, n_app, D = 250, 40, 64
    n1 = n0 + n_app
    c = BatchCase(PLANS, 4, 2, D, 300)
    Ks, Vs = _inputs(c, n1, 1400)
    for l in range(c.L):
        kvk.compress_layer(c.table, l, Ks[l][:, :, :n0].contiguous().to(DEV),
                           Vs[l][:, :, :n0].contiguous().to(DEV), n0, None, c.arena)
    for i in range(n0, n1):
        kt = torch.stack([K[:, :, i] for K in Ks]).contiguous()  # [L, B, Hkv, D]
        vt = torch.stack([V[:, :, i] for V in Vs]).contiguous()
        kvk.append_token(c.table, 0, c.L, kt.to(DEV), vt.to(DEV), i, c.arena)
    bases, total = OP.batched_arena_bases(c.od, c.oplans)
    sd = OP.sequence_dims(c.od)
    oarena = np.zeros(total, dtype=np.uint8)
    host = c.arena.cpu().numpy()
    for b in range(c.B):
        si = kvk.table_sequence_query(c.table, b)
        for l, a in enumerate(c.oplans[b]):
            if a.inherit:
                continue
            for h in range(2):
                kn, vn = Ks[l][b, h].float().numpy(), Vs[l][b, h].float().numpy()
                st = OC.compress_stream(sd, a.bits, kn[:n0], vn[:n0])
                for i in range(n0, n1):
                    st = OC.append_token(sd, a.bits, st, i, kn[i], vn[i])
                off = si.layer_offset[l] + h * si.stream_bytes[l]
                oarena[off:off + st.size] = st
                got = host[off:off + si.stream_bytes[l]]
                gb, gt = LY.split_stream(sd, a.bits, got, n1)
                wb, wt = LY.split_stream(sd, a.bits, st, n1)
                assert np.array_equal(gb, wb), f"blocks differ (b {b}, layer {l}, h {h})"
                gk, gv = LY.unpack_bf16_blocks(gt[None], D)
                wk, wv = LY.unpack_bf16_blocks(wt[None], D)
                nt = n1 % 32
                assert np.array_equal(gk[0, :nt], wk[0, :nt]) and np.array_equal(gv[0, :nt], wv[0, :nt])
    q = synth.q_random(1499, c.L, c.B, 4, D)
    out = c.decode(q, n1, 0.125)
    ref = OC.decode_step_batched(c.od, c.oplans, oarena, q.float().numpy().astype(np.float64), n1, 0.125)
    err = rel_err(out, ref)
    say(f"  max|diff| / max|out| = {err:.2e}")
    assert err <= TOL


def test_batched_append_past_one_launch():
    """Per-sequence append with more (sequence, anchor) items than one launch takes
    (120): 32 sequences with 5 anchors each in 6 layers (160 items, two launches),
    60 prefilled tokens and 8 appended across the group boundary at 64; every stored
    block and tail token equals the oracle's appends, decode within tolerance."""
    say("case batched append, 160 items")
    B, n0, n1, D = 32, 60, 68, 64
    plans = [synth.plan_mixed(1600 + b, 6, 1) for b in range(B)]
    c = BatchCase(plans, 4, 2, D, 96)
    assert sum(not a for p in plans for a, _ in p) > 120
    Ks, Vs = _inputs(c, n1, 1650)
    for l in range(c.L):
        kvk.compress_layer(c.table, l, Ks[l][:, :, :n0].contiguous().to(DEV),
                           Vs[l][:, :, :n0].contiguous().to(DEV), n0, None, c.arena)
    for i in range(n0, n1):
        kt = torch.stack([K[:, :, i] for K in Ks]).contiguous()
        vt = torch.stack([V[:, :, i] for V in Vs]).contiguous()
        kvk.append_token(c.table, 0, c.L, kt.to(DEV), vt.to(DEV), i, c.arena)
    oarena = _oracle_arena_at(c, Ks, Vs, n0, n1)
    sd = OP.sequence_dims(c.od)
    host = c.arena.cpu().numpy()
    for b in range(B):
        si = kvk.table_sequence_query(c.table, b)
        for l, a in enumerate(c.oplans[b]):
            if a.inherit:
                continue
            for h in range(2):
                off = si.layer_offset[l] + h * si.stream_bytes[l]
                gb, gt = LY.split_stream(sd, a.bits, host[off:off + si.stream_bytes[l]], n1)
                wb, wt = LY.split_stream(sd, a.bits, oarena[off:off + si.stream_bytes[l]], n1)
                assert np.array_equal(gb, wb), f"blocks differ (b {b}, layer {l}, h {h})"
                gk, gv = LY.unpack_bf16_blocks(gt[None], D)
                wk, wv = LY.unpack_bf16_blocks(wt[None], D)
                nt = n1 % 32
                assert np.array_equal(gk[0, :nt], wk[0, :nt]) and np.array_equal(gv[0, :nt], wv[0, :nt])
    q = synth.q_random(1699, c.L, B, 4, D)
    out = c.decode(q, n1, 0.125)
    ref = OC.decode_step_batched(c.od, c.oplans, oarena, q.float().numpy().astype(np.float64), n1, 0.125)
    err = rel_err(out, ref)
    say(f"  max|diff| / max|out| = {err:.2e}")
    assert err <= TOL
