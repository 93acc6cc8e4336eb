"""Full-size parity: the benchmark workloads at their real sizes, in the launch
configuration bench.py times (all layers of the plan in one decode call), checked on
sampled streams and output rows that the oracle computes one by one.

For each sampled (layer, sequence, KV head): the layer's inputs are regenerated from
the seeded generator, the anchor's stream is compressed by the oracle and compared
byte for byte with the GPU arena, and the G output rows of that layer are compared
with the oracle's attention (max|diff| <= 2e-3 * max|out| over the sampled rows).
"""
import numpy as np
import pytest
import torch

from oracle import cache as OC
from oracle import plan as OP
from paper_2609_37988_amd import kvk, synth

from gpu_common import TOL, meaningful, oracle_rows, say

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _run_workload(w, n_samples, seed, cover_bits=False):
    n_tok = w.tokens
    n_stored = w.keep_tokens if w.keep_tokens else n_tok
    dims = kvk.make_dims(kvk.GQA, w.n_layers, w.n_q_heads, w.n_kv_heads, w.head_dim, qscheme=w.qscheme,
                         batch=w.batch, max_tokens=n_tok, keep_tokens=w.keep_tokens)
    table = kvk.layer_table(dims, kvk.make_plan(w.plan))
    info = kvk.table_query(table)
    arena = torch.empty(info.arena_bytes, dtype=torch.uint8, device=DEV)
    for l in range(w.n_layers):
        if w.plan[l][0]:
            continue
        k, v = synth.kv_layer(w, l, device=DEV)
        keep = synth.keep_positions(w, l, device=DEV) if w.keep_tokens else None
        kvk.compress_layer(table, l, k, v, n_tok, keep, arena)
        del k, v, keep
    q = synth.queries(w, w.n_layers, device=DEV)
    out = torch.empty((w.n_layers, w.batch, w.n_q_heads, w.head_dim), dtype=torch.float32, device=DEV)
    ws = torch.empty(kvk.workspace_bytes(table, 0, w.n_layers), dtype=torch.uint8, device=DEV)
    kvk.decode_attention(table, 0, w.n_layers, q, n_stored, w.softmax_scale(), arena, out, ws)
    torch.cuda.synchronize()

    od = OP.Dims(OP.GQA, w.n_layers, w.n_q_heads, w.n_kv_heads, w.head_dim, qscheme=w.qscheme,
                 batch=w.batch, max_tokens=n_tok, keep_tokens=w.keep_tokens)
    G = w.n_q_heads // w.n_kv_heads
    rng = np.random.default_rng(seed)
    got_rows, ref_rows = [], []
    picks = []
    if cover_bits:  # one reading layer of an anchor of every bit-width in the plan first
        for bits in sorted({w.plan[info.anchor_of[l]][1] for l in range(w.n_layers)}):
            ls = [l for l in range(w.n_layers) if w.plan[info.anchor_of[l]][1] == bits]
            picks.append(ls[int(rng.integers(len(ls)))])
    picks += [int(rng.integers(w.n_layers)) for _ in range(max(0, n_samples - len(picks)))]
    for l in picks:
        b = int(rng.integers(w.batch))
        h = int(rng.integers(w.n_kv_heads))
        a = info.anchor_of[l]
        bits = w.plan[a][1]
        say(f"  sample layer {l} (anchor {a}, {bits} bits) b {b} kv head {h}")
        k, v = synth.kv_layer(w, a, device=DEV)
        ks, vs = k[b, h].float().cpu().numpy(), v[b, h].float().cpu().numpy()
        del k, v
        if w.keep_tokens:
            keep = synth.keep_positions(w, a, device=DEV)[b, h].cpu().numpy()
            ks, vs = OC.gather_kept(ks, keep), OC.gather_kept(vs, keep)
        ref_stream = OC.compress_stream(od, bits, ks, vs)
        sb = info.stream_bytes[a]
        off = info.layer_offset[a] + (b * w.n_kv_heads + h) * sb
        gpu_stream = arena[off:off + sb].cpu().numpy()
        assert np.array_equal(meaningful(od, bits, gpu_stream, n_stored),
                              meaningful(od, bits, ref_stream, n_stored)), f"stream bytes differ: {(l, b, h)}"
        qrows = q[l, b, h * G:(h + 1) * G].float().cpu().numpy().astype(np.float64)
        ref_rows.append(oracle_rows(od, bits, ref_stream, n_stored, qrows, w.softmax_scale()))
        got_rows.append(out[l, b, h * G:(h + 1) * G].cpu().numpy())
    got, ref = np.stack(got_rows), np.stack(ref_rows)
    err = np.abs(got - ref).max() / np.abs(ref).max()
    say(f"  max|diff| / max|out| = {err:.2e}")
    assert err <= TOL
    del arena, ws, out
    torch.cuda.empty_cache()


@pytest.mark.parametrize("variant", [None, "bf16"], ids=["int4", "bf16"])
def test_qwen7b_shaped_stack(variant):
    """28 layers, 28/4 heads, batch 8, context 8192."""
    w = synth.workload(1, variant)
    say(f"case {w.name}")
    _run_workload(w, 6, 11)


def test_qwen14b_shaped_mixed_stack():
    """The benchmark workload: 48 layers, 40/8 heads, batch 32, context 8192, mixed plan."""
    w = synth.workload(2)
    say(f"case {w.name}")
    _run_workload(w, 8, 12)


@pytest.mark.parametrize("qs", [kvk.SYMROW, kvk.GROUP64], ids=["symrow", "group64"])
def test_qwen14b_shaped_mixed_stack_other_quantisers(qs):
    """The benchmark workload with the paper's own quantiser (SYMROW: one bf16 scale per
    stored row, App. B / App. C.3) and with the grouped per-token one (GROUP64): every
    bit-width of the plan sampled, stream bytes bit-exact, rows within tolerance."""
    w = synth.workload(2)
    w.qscheme = qs
    say(f"case {w.name} qscheme {qs}")
    _run_workload(w, 8, 15 + qs, cover_bits=True)


@pytest.mark.parametrize("qs", [kvk.SYMROW, kvk.GROUP64], ids=["symrow", "group64"])
def test_qwen7b_shaped_int4_other_quantisers(qs):
    """28 layers of int4 (Qwen2.5-7B shape) with SYMROW and GROUP64 (App. C.3's 3.56x)."""
    w = synth.workload(1)
    w.qscheme = qs
    say(f"case {w.name} qscheme {qs}")
    _run_workload(w, 6, 21 + qs)


def test_qwen14b_shaped_one_anchor_for_all_layers():
    """Depth's extreme at full size (App. C.1): layer 0's int4 cache read by all 48
    layers (240 query rows per KV head: 16 chunk waves in 4 workgroups per split),
    batch 32, context 8192, in the launch shape the benchmark times."""
    w = synth.workload(2, "one-anchor-4")
    say(f"case {w.name}")
    _run_workload(w, 6, 17)


def test_qwen14b_shaped_128k_eviction():
    """48 layers, batch 4, context 131072 with half the positions kept, int2/int4 plan."""
    w = synth.workload(4)
    say(f"case {w.name}")
    _run_workload(w, 4, 14)


@pytest.mark.parametrize("variant", [None, "int4", "depth", "int4-depth", "14b", "14b-int4"],
                         ids=["bf16", "int4", "depth", "int4-depth", "14b-bf16", "14b-int4"])
def test_mla_shaped_stack(variant):
    """The MLA-style stacks at full size (32 layers, 32 heads, latent 512 + 64,
    batch 16, context 16384; and Qwen2.5-14B's latent shape: 48 layers, 40 heads,
    latent 1024 + 64, batch 32, context 8192), kept to per-layer widths, one decode
    call over all layers; sampled (layer, sequence) streams bit-exact and their
    output heads within tolerance (oracle in the absorbed form, pinned equal to the
    reconstruction).  A layer reading a full-width anchor is always sampled."""
    from oracle import mla as OM
    w = synth.mla_workload(variant)
    say(f"case {w.name}")
    n = w.tokens
    dims = kvk.make_dims(kvk.MLA, w.n_layers, w.n_q_heads, w.ref_kv_heads, w.ref_head_dim, w.latent_dim,
                         w.rope_dim, w.nope_dim, w.v_dim, qscheme=w.qscheme, batch=w.batch, max_tokens=n)
    table = kvk.layer_table(dims, kvk.make_plan(w.plan))
    info = kvk.table_query(table)
    arena = torch.empty(info.arena_bytes, dtype=torch.uint8, device=DEV)
    for l in range(w.n_layers):
        c, r = synth.mla_layer(w, l, device=DEV)
        kvk.compress_layer(table, l, c, r, n, None, arena)
        del c, r
    q = synth.mla_queries(w, w.n_layers, device=DEV)
    wk, wv = synth.mla_weights(w, w.n_layers, device=DEV)
    out = torch.empty((w.n_layers, w.batch, w.n_q_heads, w.v_dim), dtype=torch.float32, device=DEV)
    ws = torch.empty(kvk.workspace_bytes(table, 0, w.n_layers), dtype=torch.uint8, device=DEV)
    kvk.decode_attention(table, 0, w.n_layers, q, n, w.softmax_scale(), arena, out, ws,
                         w_uk=kvk.mla_weights_for_library(wk), w_uv=wv)
    torch.cuda.synchronize()
    od = OP.Dims(OP.MLA, w.n_layers, w.n_q_heads, w.ref_kv_heads, w.ref_head_dim, latent_dim=w.latent_dim,
                 rope_dim=w.rope_dim, nope_dim=w.nope_dim, v_dim=w.v_dim, qscheme=w.qscheme, batch=w.batch,
                 max_tokens=n)
    rng = np.random.default_rng(13)
    got_rows, ref_rows = [], []
    readers = [l for l in range(w.n_layers) if w.plan[l][0]]  # inheriting layers (depth variants)
    picks = [readers[int(rng.integers(len(readers)))] for _ in range(2)] if readers else []
    full = [l for l in range(w.n_layers) if w.plan[info.anchor_of[l]][2] == w.latent_dim]
    if full:
        picks.append(full[int(rng.integers(len(full)))])
    picks += [int(rng.integers(w.n_layers)) for _ in range(4 - len(picks))]
    for l in picks:
        b = int(rng.integers(w.batch))
        a = info.anchor_of[l]
        _, bits, d = w.plan[a]
        say(f"  sample layer {l} (anchor {a}: d {d}, {bits} bits) b {b}")
        c, r = synth.mla_layer(w, a, device=DEV)
        cs, rs = c[b].float().cpu().numpy(), r[b].float().cpu().numpy()
        del c, r
        ref_stream = OM.compress_stream(od, bits, d, cs, rs)
        sb = info.stream_bytes[a]
        off = info.layer_offset[a] + b * sb
        assert np.array_equal(arena[off:off + sb].cpu().numpy(), ref_stream), f"stream bytes differ: {(l, b)}"
        C, R = OM.dequant_stream(od, bits, d, ref_stream, n)
        qb = q[l, b].float().cpu().numpy().astype(np.float64)
        ref_rows.append(OM.attention_absorbed(qb[:, :w.nope_dim], qb[:, w.nope_dim:], C, R,
                                              wk[l].float().cpu().numpy(), wv[l].float().cpu().numpy(),
                                              w.softmax_scale()))
        got_rows.append(out[l, b].cpu().numpy())
    got, ref = np.stack(got_rows), np.stack(ref_rows)
    err = np.abs(got - ref).max() / np.abs(ref).max()
    say(f"  max|diff| / max|out| = {err:.2e}")
    assert err <= TOL
    del arena, ws, out
    torch.cuda.empty_cache()


def test_qwen14b_shaped_append_last_group():
    """Decode-time append at the benchmark's size and launch shape: the 14B mixed
    stack prefilled with 8160 tokens, then 32 appended tokens (one kvk_append_token
    call per token over all 48 layers, the last one completing block 255), then one
    decode over all layers at 8192.  Sampled streams equal the oracle's prefill of
    8160 tokens followed by its appends of the same 32 tokens; sampled output rows
    match the oracle's attention over them."""
    w = synth.workload(2)
    say(f"case {w.name} + 32 appended tokens")
    n_tok, n0 = w.tokens, w.tokens - 32
    dims = kvk.make_dims(kvk.GQA, w.n_layers, w.n_q_heads, w.n_kv_heads, w.head_dim, qscheme=w.qscheme,
                         batch=w.batch, max_tokens=n_tok)
    table = kvk.layer_table(dims, kvk.make_plan(w.plan))
    info = kvk.table_query(table)
    arena = torch.empty(info.arena_bytes, dtype=torch.uint8, device=DEV)
    for l in range(w.n_layers):
        if w.plan[l][0]:
            continue
        k, v = synth.kv_layer(w, l, device=DEV)
        kvk.compress_layer(table, l, k[:, :, :n0].contiguous(), v[:, :, :n0].contiguous(), n0, None, arena)
        del k, v
    kn, vn = synth.kv_random(77, w.n_layers * w.batch, w.n_kv_heads, 32, w.head_dim, device=DEV)
    kn = kn.reshape(w.n_layers, w.batch, w.n_kv_heads, 32, w.head_dim)
    vn = vn.reshape(w.n_layers, w.batch, w.n_kv_heads, 32, w.head_dim)
    for i in range(32):
        kvk.append_token(table, 0, w.n_layers, kn[:, :, :, i].contiguous(), vn[:, :, :, i].contiguous(), n0 + i,
                         arena)
    q = synth.queries(w, w.n_layers, device=DEV)
    out = torch.empty((w.n_layers, w.batch, w.n_q_heads, w.head_dim), dtype=torch.float32, device=DEV)
    ws = torch.empty(kvk.workspace_bytes(table, 0, w.n_layers), dtype=torch.uint8, device=DEV)
    kvk.decode_attention(table, 0, w.n_layers, q, n_tok, w.softmax_scale(), arena, out, ws)
    torch.cuda.synchronize()
    od = OP.Dims(OP.GQA, w.n_layers, w.n_q_heads, w.n_kv_heads, w.head_dim, qscheme=w.qscheme,
                 batch=w.batch, max_tokens=n_tok)
    G = w.n_q_heads // w.n_kv_heads
    rng = np.random.default_rng(15)
    got_rows, ref_rows = [], []
    for _ in range(6):
        l, b, h = int(rng.integers(w.n_layers)), int(rng.integers(w.batch)), int(rng.integers(w.n_kv_heads))
        a = info.anchor_of[l]
        bits = w.plan[a][1]
        say(f"  sample layer {l} (anchor {a}, {bits} bits) b {b} kv head {h}")
        k, v = synth.kv_layer(w, a, device=DEV)
        ks, vs = k[b, h, :n0].float().cpu().numpy(), v[b, h, :n0].float().cpu().numpy()
        del k, v
        st = OC.compress_stream(od, bits, ks, vs)
        kt, vt = kn[a, b, h].float().cpu().numpy(), vn[a, b, h].float().cpu().numpy()
        for i in range(32):
            st = OC.append_token(od, bits, st, n0 + i, kt[i], vt[i])
        sb = info.stream_bytes[a]
        off = info.layer_offset[a] + (b * w.n_kv_heads + h) * sb
        blocks_gpu = arena[off:off + sb].cpu().numpy()[:(n_tok // 32) * OP.block_bytes(od, bits)]
        assert np.array_equal(blocks_gpu, st[:blocks_gpu.size]), f"stream blocks differ: {(l, b, h)}"
        qrows = q[l, b, h * G:(h + 1) * G].float().cpu().numpy().astype(np.float64)
        ref_rows.append(oracle_rows(od, bits, st, n_tok, qrows, w.softmax_scale()))
        got_rows.append(out[l, b, h * G:(h + 1) * G].cpu().numpy())
    got, ref = np.stack(got_rows), np.stack(ref_rows)
    err = np.abs(got - ref).max() / np.abs(ref).max()
    say(f"  max|diff| / max|out| = {err:.2e}")
    assert err <= TOL
    del arena, ws, out
    torch.cuda.empty_cache()


def test_snapkv_at_128k():
    """The query-aware keep list at the eviction workload's size (batch 4, 131072
    positions, 8 KV heads, 40 query heads, keep 65536) on one anchor's keys:
    sampled streams' importances within 1e-4 of the oracle's largest, the selection
    exactly the rule applied to the kernel's importances, and any difference from
    the oracle's own selection at its threshold."""
    from oracle import snapkv as S
    w = synth.workload(4)
    say(f"case snapkv {w.name}")
    n, keep, G = w.tokens, w.keep_tokens, w.n_q_heads // w.n_kv_heads
    dims = kvk.make_dims(kvk.GQA, w.n_layers, w.n_q_heads, w.n_kv_heads, w.head_dim, batch=w.batch,
                         max_tokens=n, keep_tokens=keep)
    table = kvk.layer_table(dims, kvk.make_plan(w.plan))
    k, _ = synth.kv_layer(w, 0, device=DEV)
    q = synth.q_random(4242, w.batch, w.n_q_heads, 32, w.head_dim, device=DEV)
    keep_out = torch.empty((w.batch, w.n_kv_heads, keep), dtype=torch.int32, device=DEV)
    imp = torch.empty((w.batch, w.n_kv_heads, n), dtype=torch.float32, device=DEV)
    ws = torch.empty(kvk.snapkv_workspace_bytes(table, n), dtype=torch.uint8, device=DEV)
    kvk.snapkv_select(table, 0, k, q, n, w.softmax_scale(), keep_out, ws, importance=imp)
    torch.cuda.synchronize()
    rng = np.random.default_rng(16)
    for _ in range(2):
        b, h = int(rng.integers(w.batch)), int(rng.integers(w.n_kv_heads))
        say(f"  sample b {b} kv head {h}")
        kb = k[b, h:h + 1].float().cpu().numpy().astype(np.float64)
        qb = q[b, h * G:(h + 1) * G].float().cpu().numpy().astype(np.float64)
        ref = S.importance(qb, kb, w.softmax_scale())[0]
        got = imp[b, h].cpu().numpy()
        top = ref.max()
        assert np.abs(got - ref).max() <= 1e-4 * top
        kl = keep_out[b, h].cpu().numpy()
        assert np.array_equal(kl, S.select(got.astype(np.float64), keep))
        diff = np.setxor1d(kl, S.select(ref, keep))
        if diff.size:
            theta = np.sort(ref[:n - 32])[::-1][keep - 33]
            assert np.all(np.abs(ref[diff] - theta) <= 1e-4 * top)
    del k, ws, imp
    torch.cuda.empty_cache()


def test_mla_per_sequence_plans_full_size():
    """The benchmark's per-sequence MLA workload (16 sequences of 16384 tokens, each its
    own 32-layer plan of kept widths, 512 anchors) in the one batched launch per phase:
    two sampled sequences decode bit for bit as their one-sequence tables do."""
    w = synth.mla_workload(None)
    plans = synth.mla_plans_per_sequence(w)
    say(f"case {w.name} per-sequence plans")
    n = w.tokens
    dims = kvk.make_dims(kvk.MLA, w.n_layers, w.n_q_heads, w.ref_kv_heads, w.ref_head_dim, w.latent_dim,
                         w.rope_dim, w.nope_dim, w.v_dim, qscheme=w.qscheme, batch=w.batch, max_tokens=n)
    table = kvk.layer_table_batched(dims, [kvk.make_plan(p) for p in plans])
    arena = torch.empty(kvk.table_query(table).arena_bytes, dtype=torch.uint8, device=DEV)
    for l in range(w.n_layers):
        c, r = synth.mla_layer(w, l, device=DEV)
        kvk.compress_layer(table, l, c, r, n, None, arena)
        del c, r
    q = synth.mla_queries(w, w.n_layers, device=DEV)
    wk, wv = synth.mla_weights(w, w.n_layers, device=DEV)
    wk = kvk.mla_weights_for_library(wk)
    out = torch.full((w.n_layers, w.batch, w.n_q_heads, w.v_dim), float("nan"), dtype=torch.float32, device=DEV)
    ws = torch.empty(kvk.workspace_bytes(table, 0, w.n_layers), dtype=torch.uint8, device=DEV)
    kvk.decode_setup(table, 0, w.n_layers, ws)
    kvk.decode_attention(table, 0, w.n_layers, q, n, w.softmax_scale(), arena, out, ws, w_uk=wk, w_uv=wv)
    torch.cuda.synchronize()
    del arena, ws
    torch.cuda.empty_cache()
    one_dims = kvk.make_dims(kvk.MLA, w.n_layers, w.n_q_heads, w.ref_kv_heads, w.ref_head_dim, w.latent_dim,
                             w.rope_dim, w.nope_dim, w.v_dim, qscheme=w.qscheme, batch=1, max_tokens=n)
    for b in (0, 9):
        one = kvk.layer_table(one_dims, kvk.make_plan(plans[b]))
        a1 = torch.empty(kvk.table_query(one).arena_bytes, dtype=torch.uint8, device=DEV)
        for l in range(w.n_layers):
            c, r = synth.mla_layer(w, l, device=DEV)
            kvk.compress_layer(one, l, c[b:b + 1].contiguous(), r[b:b + 1].contiguous(), n, None, a1)
            del c, r
        o1 = torch.full((w.n_layers, 1, w.n_q_heads, w.v_dim), float("nan"), dtype=torch.float32, device=DEV)
        w1 = torch.empty(kvk.workspace_bytes(one, 0, w.n_layers), dtype=torch.uint8, device=DEV)
        kvk.decode_attention(one, 0, w.n_layers, q[:, b:b + 1].contiguous(), n, w.softmax_scale(), a1, o1, w1,
                             w_uk=wk, w_uv=wv)
        torch.cuda.synchronize()
        assert torch.isfinite(o1).all()
        assert torch.equal(o1[:, 0], out[:, b]), f"sequence {b} differs from its one-sequence table"
        say(f"  sequence {b}: bit for bit")
        del a1, w1
        torch.cuda.empty_cache()
