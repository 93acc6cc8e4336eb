"""Host side of the C ABI (no GPU): exports, plan tables, accounting, error codes."""
import ctypes
import os
import re

import pytest

from oracle import plan as P
from paper_2609_37988_amd import kvk, synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _header_functions():
    with open(os.path.join(ROOT, "include", "kvk.h")) as f:
        text = f.read()
    return sorted(set(re.findall(r"\b(kvk_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_function():
    lib = kvk.load()
    declared = _header_functions()
    assert declared, "no declarations found"
    for name in declared:
        assert hasattr(lib, name), name
    assert set(declared) == set(kvk.exported_symbols())
    assert "gfx950" in kvk.version()


def _oracle_dims(d):
    return P.Dims(d.kind, d.n_layers, d.n_q_heads, d.n_kv_heads, d.head_dim, qscheme=d.qscheme,
                  batch=d.batch, max_tokens=d.max_tokens, keep_tokens=d.keep_tokens)


def _table_for(w):
    d = kvk.make_dims(kvk.GQA, w.n_layers, w.n_q_heads, w.n_kv_heads, w.head_dim, qscheme=w.qscheme,
                      batch=w.batch, max_tokens=w.tokens, keep_tokens=w.keep_tokens)
    plan = kvk.make_plan(w.plan)
    return d, plan, kvk.layer_table(d, plan)


@pytest.mark.parametrize("cfg", [0, 1, 2, 4])
@pytest.mark.parametrize("qs", [kvk.KIVI32, kvk.SYMROW, kvk.GROUP64])
def test_table_matches_oracle_accounting(cfg, qs):
    w = synth.workload(cfg)
    w.qscheme = qs
    d, plan, t = _table_for(w)
    inf = kvk.table_query(t)
    od = _oracle_dims(d)
    oplan = [P.Action(bool(a.inherit), a.bits) for a in plan]
    assert P.validate(od, oplan) is None
    assert inf.anchor_of == P.anchor_of(oplan)
    offs, total = P.arena_offsets(od, oplan)
    assert inf.layer_offset == offs and inf.arena_bytes == total
    for l, a in enumerate(oplan):
        if not a.inherit:
            assert inf.layer_bytes[l] == P.layer_bytes(od, a.bits)
            assert inf.stream_bytes[l] == P.stream_bytes(od, a.bits)
        assert inf.layer_cost_bits[l] == P.cost_bits(od, a)
    assert inf.rho == pytest.approx(P.rho(od, oplan), rel=1e-15)
    alg = P.read_bytes(od, oplan, 0, od.n_layers, od.stored_cap)
    assert inf.rho_realized == pytest.approx(P.bf16_full_bytes(od) / alg, rel=1e-12)
    assert inf.n_anchors == sum(1 for a in oplan if not a.inherit)
    for n in (0, 1, 33, od.stored_cap):
        for l0, l1 in ((0, od.n_layers), (1, min(5, od.n_layers)), (od.n_layers - 1, od.n_layers)):
            if l1 > l0:
                assert kvk.read_bytes(t, l0, l1, n) == P.read_bytes(od, oplan, l0, l1, n)


def test_headline_plans():
    """The 14B-shaped 128k plan is 16x by eq. (2) (32x with half the positions kept);
    the 14B-shaped mixed plan has 16 inheriting layers."""
    w4 = synth.workload(4)
    t4 = _table_for(w4)[2]
    i4 = kvk.table_query(t4)
    assert i4.rho == pytest.approx(16.0) and i4.n_anchors == 20
    assert i4.rho * w4.tokens / w4.keep_tokens == pytest.approx(32.0)
    w2 = synth.workload(2)
    assert sum(e[0] for e in w2.plan) == 16 and w2.plan[0][0] == 0


def _gold(name):
    with open(os.path.join(ROOT, "tests", "golden", name)) as f:
        return [ln.split() for ln in f if ln.strip() and not ln.startswith("#")]


def test_realized_bits_entry_point_matches_table():
    for scheme, g, b, bpe, _ in _gold("realized_bits_table.txt"):
        if scheme == "symrow":
            got = kvk.realized_bits(kvk.SYMROW, int(b), int(g), 0, 2048)
        else:
            got = kvk.realized_bits(kvk.KIVI32, int(b), int(g), 128, 2048)
        assert round(got, 3) == pytest.approx(float(bpe))
    assert kvk.realized_bits(kvk.KIVI32, 3, 32, 0, 10) < 0


AXES = {
    "precision": (True, False, False), "depth": (False, False, True),
    "depth+precision": (True, False, True), "rank": (False, True, False),
    "rank+precision": (True, True, False), "depth+rank": (False, True, True),
    "depth+rank+precision": (True, True, True),
}


def test_rho_range_entry_point_matches_table():
    for row in _gold("ranges_table.txt"):
        prec, rank, depth = AXES[row[0]]
        mla = row[1] == "MLA"
        for (L, width, r), cols in (((48, 2048, 1024), row[4:6]), ((36, 512, 256), row[7:9])):
            lo, hi = kvk.rho_range(L, width, r, 64, mla, prec, rank, depth)
            for got, printed in ((lo, cols[0]), (hi, cols[1])):
                nd = len(printed.split(".")[1]) if "." in printed else 0
                assert round(got, nd) == pytest.approx(float(printed))


def _expect(status, fn, *args):
    with pytest.raises(kvk.KvkError) as e:
        fn(*args)
    assert e.value.status == status, str(e.value)
    assert kvk.last_error()


def test_invalid_plans_and_dims():
    good = kvk.make_dims(kvk.GQA, 3, 8, 2, 128, batch=2, max_tokens=100)
    ok_plan = kvk.make_plan([(0, 4), (1, 16), (0, 2)])
    kvk.layer_table(good, ok_plan)
    _expect(kvk.ERR_INVALID, kvk.layer_table, good, kvk.make_plan([(1, 16), (0, 4), (0, 4)]))
    _expect(kvk.ERR_INVALID, kvk.layer_table, good, kvk.make_plan([(0, 3), (0, 4), (0, 4)]))
    _expect(kvk.ERR_INVALID, kvk.layer_table, good, kvk.make_plan([(0, 4, 256), (0, 4), (0, 4)]))
    mla_plan = kvk.make_plan([(0, 4, 512), (1, 16, 0), (0, 2, 128)])
    _expect(kvk.ERR_UNSUPPORTED, kvk.layer_table, kvk.make_dims(kvk.MLA, 3, 12, 2, 128, 512, 64, 128, 128,
                                                                batch=1, max_tokens=8), mla_plan)
    _expect(kvk.ERR_UNSUPPORTED, kvk.layer_table, kvk.make_dims(kvk.MLA, 3, 32, 2, 128, 2048, 64, 128, 128,
                                                                batch=1, max_tokens=8),
            kvk.make_plan([(0, 4, 2048), (1, 16, 0), (0, 2, 256)]))
    # Qwen2.5-14B's heads (40 query heads) at its full latent width 1024 + 64
    kvk.layer_table(kvk.make_dims(kvk.MLA, 3, 40, 8, 128, 1024, 64, 128, 128, batch=1, max_tokens=8),
                    kvk.make_plan([(0, 4, 1024), (1, 16, 0), (0, 2, 128)]))
    _expect(kvk.ERR_UNSUPPORTED, kvk.layer_table, kvk.make_dims(kvk.GQA, 3, 8, 2, 96, max_tokens=8), ok_plan)
    # streams above 2 GiB (bf16 K and V of d_h 128: 512 bytes per token; a width-1024
    # bf16 latent: 2176) are refused; just below the limit they are accepted
    big_gqa = kvk.make_plan([(0, 16), (1, 16), (0, 2)])
    _expect(kvk.ERR_UNSUPPORTED, kvk.layer_table, kvk.make_dims(kvk.GQA, 3, 8, 2, 128, max_tokens=5_000_000), big_gqa)
    kvk.layer_table(kvk.make_dims(kvk.GQA, 3, 8, 2, 128, max_tokens=4_000_000), big_gqa)
    _expect(kvk.ERR_UNSUPPORTED, kvk.layer_table,
            kvk.make_dims(kvk.MLA, 3, 40, 8, 128, 1024, 64, 128, 128, batch=1, max_tokens=1_000_000),
            kvk.make_plan([(0, 16, 1024), (1, 16, 0), (0, 2, 128)]))
    _expect(kvk.ERR_INVALID, kvk.layer_table, kvk.make_dims(kvk.GQA, 3, 6, 4, 128, max_tokens=8), ok_plan)
    _expect(kvk.ERR_INVALID, kvk.layer_table,
            kvk.make_dims(kvk.GQA, 3, 8, 2, 128, max_tokens=8, keep_tokens=9), ok_plan)
    _expect(kvk.ERR_INVALID, kvk.layer_table, kvk.make_dims(kvk.GQA, 0, 8, 2, 128, max_tokens=8), ok_plan)
    # every eq. (3) plan is accepted, including one anchor serving all layers
    # (App. C.1's depth extreme): 64 layers x 8 query heads per KV head = 512 rows
    d64 = kvk.make_dims(kvk.GQA, 64, 64, 8, 128, max_tokens=64)
    one = kvk.table_query(kvk.layer_table(d64, kvk.make_plan([(0, 2)] + [(1, 16)] * 63)))
    assert one.n_anchors == 1 and all(a == 0 for a in one.anchor_of[:64])


def _raw(status, name, *args):
    lib = kvk.load()
    assert getattr(lib, name)(*args) == status, kvk.last_error()
    if status != kvk.OK:
        assert kvk.last_error()


def test_entry_points_reject_bad_arguments_without_launching():
    """Validation happens on the host before any launch: these calls pass non-null
    dummy pointers that no kernel ever sees."""
    d = kvk.make_dims(kvk.GQA, 2, 4, 1, 64, batch=1, max_tokens=64)
    t = kvk.layer_table(d, kvk.make_plan([(0, 8), (1, 16)]))
    h, P = t.handle, ctypes.c_void_p
    f = P(256)
    I, B = kvk.ERR_INVALID, kvk.ERR_BUFFER
    _raw(I, "kvk_compress_layer", h, 5, f, f, kvk.BF16, 64, None, f, None)     # layer
    _raw(I, "kvk_compress_layer", h, 0, f, f, kvk.BF16, 65, None, f, None)     # n_tokens
    _raw(I, "kvk_compress_layer", h, 0, f, f, kvk.BF16, 64, f, f, None)        # keep without eviction
    _raw(I, "kvk_compress_layer", h, 0, None, f, kvk.BF16, 64, None, f, None)  # NULL input
    _raw(I, "kvk_compress_layer", h, 0, f, f, 7, 64, None, f, None)            # dtype
    _raw(kvk.OK, "kvk_compress_layer", h, 1, f, f, kvk.BF16, 64, None, f, None)  # inheritor: no-op
    _raw(I, "kvk_compress_layer", h, 0, P(264), f, kvk.BF16, 64, None, f, None)  # K not 16-byte aligned
    _raw(I, "kvk_compress_layer", h, 0, f, P(260), kvk.BF16, 64, None, f, None)  # V not 16-byte aligned
    _raw(I, "kvk_decode_attention", h, 1, 1, f, kvk.BF16, 64, 0.1, None, None, f, f, f, 1 << 20, None)
    _raw(I, "kvk_decode_attention", h, 0, 2, f, kvk.BF16, 65, 0.1, None, None, f, f, f, 1 << 20, None)
    _raw(I, "kvk_decode_attention", h, 0, 2, f, kvk.BF16, 64, 0.1, f, None, f, f, f, 1 << 20, None)
    _raw(I, "kvk_decode_attention", h, 0, 2, P(264), kvk.BF16, 64, 0.1, None, None, f, f, f, 1 << 20, None)
    _raw(B, "kvk_decode_attention", h, 0, 2, f, kvk.BF16, 64, 0.1, None, None, f, f, f, 16, None)
    _raw(I, "kvk_decode_attention", h, 0, 2, f, kvk.BF16, 64, float("nan"), None, None, f, f, f, 1 << 20, None)
    _raw(I, "kvk_debug_dequantize", h, 0, 65, f, f, f, None)
    assert kvk.workspace_bytes(t, 0, 2) > 0
    _raw(I, "kvk_append_token", h, 0, 3, f, f, kvk.BF16, 10, f, None)        # layer range
    _raw(I, "kvk_append_token", h, 1, 1, f, f, kvk.BF16, 10, f, None)        # empty range
    _raw(I, "kvk_append_token", h, 0, 2, f, f, kvk.BF16, 64, f, None)        # stream full (cap 64)
    _raw(I, "kvk_append_token", h, 0, 2, f, f, kvk.BF16, -1, f, None)        # negative position
    _raw(I, "kvk_append_token", h, 0, 2, None, f, kvk.BF16, 10, f, None)     # NULL input
    _raw(I, "kvk_append_token", h, 0, 2, f, f, 7, 10, f, None)               # dtype
    _raw(I, "kvk_append_token", h, 0, 2, P(264), f, kvk.BF16, 10, f, None)   # K not 16-byte aligned
    _raw(I, "kvk_append_token", h, 0, 2, f, f, kvk.BF16, 10, P(260), None)   # arena not 16-byte aligned
    _raw(kvk.OK, "kvk_append_token", h, 1, 2, f, f, kvk.BF16, 63, f, None)   # inheritors only: no-op


def test_snapkv_rejects_bad_arguments_without_launching():
    P = ctypes.c_void_p
    f = P(256)
    I, U, B = kvk.ERR_INVALID, kvk.ERR_UNSUPPORTED, kvk.ERR_BUFFER
    ev = kvk.layer_table(kvk.make_dims(kvk.GQA, 2, 10, 2, 128, batch=1, max_tokens=256, keep_tokens=64),
                         kvk.make_plan([(0, 4), (1, 16)]))
    need = kvk.snapkv_workspace_bytes(ev, 256)
    assert need > 0
    h = ev.handle
    _raw(I, "kvk_snapkv_select", h, 0, f, f, kvk.BF16, 63, 0.1, f, None, f, need, None)     # n < keep
    _raw(I, "kvk_snapkv_select", h, 0, f, f, kvk.BF16, 257, 0.1, f, None, f, need, None)    # n > max
    _raw(I, "kvk_snapkv_select", h, 2, f, f, kvk.BF16, 256, 0.1, f, None, f, need, None)    # layer
    _raw(I, "kvk_snapkv_select", h, 0, None, f, kvk.BF16, 256, 0.1, f, None, f, need, None)  # NULL keys
    _raw(U, "kvk_snapkv_select", h, 0, f, f, kvk.F32, 256, 0.1, f, None, f, need, None)     # fp32
    _raw(I, "kvk_snapkv_select", h, 0, P(264), f, kvk.BF16, 256, 0.1, f, None, f, need, None)  # align
    _raw(B, "kvk_snapkv_select", h, 0, f, f, kvk.BF16, 256, 0.1, f, None, f, need - 1, None)
    _raw(kvk.OK, "kvk_snapkv_select", h, 1, f, f, kvk.BF16, 256, 0.1, f, None, f, need, None)  # inheritor
    no_ev = kvk.layer_table(kvk.make_dims(kvk.GQA, 1, 4, 1, 128, batch=1, max_tokens=256), kvk.make_plan([(0, 4)]))
    _raw(I, "kvk_snapkv_select", no_ev.handle, 0, f, f, kvk.BF16, 256, 0.1, f, None, f, need, None)
    wide = kvk.layer_table(kvk.make_dims(kvk.GQA, 1, 18, 2, 128, batch=1, max_tokens=256, keep_tokens=64),
                           kvk.make_plan([(0, 4)]))
    _raw(U, "kvk_snapkv_select", wide.handle, 0, f, f, kvk.BF16, 256, 0.1, f, None, f, 1 << 30, None)  # G 9


def test_binding_rejects_mis_sized_tensors():
    import torch
    d = kvk.make_dims(kvk.GQA, 1, 4, 1, 64, batch=1, max_tokens=64)
    t = kvk.layer_table(d, kvk.make_plan([(0, 8)]))
    k = torch.zeros(1, 1, 63, 64, dtype=torch.bfloat16)
    arena = torch.zeros(16, dtype=torch.uint8)
    with pytest.raises(ValueError):
        kvk.compress_layer(t, 0, k, k, 64, None, arena)
    q = torch.zeros(1, 1, 4, 64, dtype=torch.bfloat16)
    with pytest.raises(ValueError):
        kvk.decode_attention(t, 0, 1, q, 64, 0.1, arena, torch.zeros(1, 1, 4, 63), arena)


# ---------------------------------------------------------------------------
# MLA tables (rank axis)
# ---------------------------------------------------------------------------

def _mla_dims(w):
    return kvk.make_dims(kvk.MLA, w.n_layers, w.n_q_heads, w.ref_kv_heads, w.ref_head_dim, w.latent_dim,
                         w.rope_dim, w.nope_dim, w.v_dim, qscheme=w.qscheme, batch=w.batch,
                         max_tokens=w.tokens, keep_tokens=w.keep_tokens)


def _mla_oracle_dims(w):
    return P.Dims(P.MLA, w.n_layers, w.n_q_heads, w.ref_kv_heads, w.ref_head_dim, latent_dim=w.latent_dim,
                  rope_dim=w.rope_dim, nope_dim=w.nope_dim, v_dim=w.v_dim, qscheme=w.qscheme, batch=w.batch,
                  max_tokens=w.tokens, keep_tokens=w.keep_tokens)


@pytest.mark.parametrize("variant,inherit", [(None, 0), ("int4", 0), ("int4", 10)])
@pytest.mark.parametrize("qs", [kvk.KIVI32, kvk.SYMROW])
def test_mla_table_matches_oracle_accounting(variant, inherit, qs):
    w = synth.mla_workload(variant)
    w.qscheme = qs
    if inherit:
        w.plan = synth.plan_ranks(77, w.n_layers, w.latent_dim, 4, n_inherit=inherit)
    t = kvk.layer_table(_mla_dims(w), kvk.make_plan(w.plan))
    inf = kvk.table_query(t)
    od = _mla_oracle_dims(w)
    oplan = [P.Action(bool(i), b, r) for i, b, r in w.plan]
    assert P.validate(od, oplan) is None
    assert inf.anchor_of == P.anchor_of(oplan)
    offs, total = P.arena_offsets(od, oplan)
    assert inf.layer_offset == offs and inf.arena_bytes == total
    for l, a in enumerate(oplan):
        if not a.inherit:
            assert inf.layer_bytes[l] == P.layer_bytes(od, a.bits, a.rank)
            assert inf.stream_bytes[l] == P.stream_bytes(od, a.bits, a.rank)
        assert inf.layer_cost_bits[l] == P.cost_bits(od, a)
    assert inf.rho == pytest.approx(P.rho(od, oplan), rel=1e-15)
    alg = P.read_bytes(od, oplan, 0, od.n_layers, od.stored_cap)
    assert inf.rho_realized == pytest.approx(P.bf16_full_bytes(od) / alg, rel=1e-12)
    for n in (0, 1, 33, od.stored_cap):
        for l0, l1 in ((0, od.n_layers), (3, 9), (od.n_layers - 1, od.n_layers)):
            assert kvk.read_bytes(t, l0, l1, n) == P.read_bytes(od, oplan, l0, l1, n)
    assert kvk.workspace_bytes(t, 0, od.n_layers) == inf.workspace_bytes > 0


def test_mla_workload_bytes():
    """The MLA-style workload: 32 layers of bf16 latents at widths drawn from
    {512, 256, 128, 64} + 64 hold about 5.1 GB at 16 x 16384 tokens."""
    w = synth.mla_workload()
    t = kvk.layer_table(_mla_dims(w), kvk.make_plan(w.plan))
    alg = kvk.read_bytes(t, 0, w.n_layers, w.tokens)
    assert alg == sum(w.batch * w.tokens * (r + 64) * 2 for _, _, r in w.plan)
    assert 4.5e9 < alg < 5.7e9


def test_mla_invalid_plans_and_dims():
    def dims(**kw):
        a = dict(n_layers=2, Hq=32, Hkv=4, hd=128, r=512, rope=64, nope=128, v=128)
        a.update(kw)
        return kvk.make_dims(kvk.MLA, a["n_layers"], a["Hq"], a["Hkv"], a["hd"], a["r"], a["rope"], a["nope"],
                             a["v"], batch=1, max_tokens=64)
    ok = kvk.make_plan([(0, 4, 512), (1, 16, 0)])
    kvk.layer_table(dims(), ok)
    _expect(kvk.ERR_INVALID, kvk.layer_table, dims(), kvk.make_plan([(0, 4, 100), (1, 16, 0)]))
    _expect(kvk.ERR_INVALID, kvk.layer_table, dims(), kvk.make_plan([(0, 4, 0), (1, 16, 0)]))
    _expect(kvk.ERR_INVALID, kvk.layer_table, dims(r=300), ok)
    _expect(kvk.ERR_INVALID, kvk.layer_table, dims(Hkv=0), ok)
    _expect(kvk.ERR_UNSUPPORTED, kvk.layer_table, dims(rope=32), ok)
    _expect(kvk.ERR_UNSUPPORTED, kvk.layer_table, dims(Hq=20), ok)
    kvk.layer_table(dims(Hq=16), ok)
    kvk.layer_table(dims(Hq=40), ok)
    _expect(kvk.ERR_UNSUPPORTED, kvk.layer_table, dims(nope=100), ok)
    _expect(kvk.ERR_UNSUPPORTED, kvk.layer_table, dims(r=2048), kvk.make_plan([(0, 4, 2048), (1, 16, 0)]))
    kvk.layer_table(dims(r=1024), kvk.make_plan([(0, 4, 1024), (1, 16, 0)]))
    kvk.layer_table(dims(r=1024), kvk.make_plan([(0, 4, 512), (0, 2, 128)]))
    g64 = kvk.make_dims(kvk.MLA, 2, 32, 4, 128, 512, 64, 128, 128, qscheme=kvk.GROUP64, batch=1, max_tokens=64)
    _expect(kvk.ERR_UNSUPPORTED, kvk.layer_table, g64, ok)  # the per-token 64-channel scheme is GQA-only


def test_mla_entry_points_reject_bad_arguments_without_launching():
    d = kvk.make_dims(kvk.MLA, 2, 32, 4, 128, 256, 64, 128, 128, batch=1, max_tokens=64)
    t = kvk.layer_table(d, kvk.make_plan([(0, 8, 128), (1, 16, 0)]))
    h, Pv = t.handle, ctypes.c_void_p
    f = Pv(256)
    I, B = kvk.ERR_INVALID, kvk.ERR_BUFFER
    need = kvk.workspace_bytes(t, 0, 2)
    _raw(I, "kvk_decode_attention", h, 0, 2, f, kvk.BF16, 64, 0.1, None, f, f, f, f, need, None)  # no w_uk
    _raw(I, "kvk_decode_attention", h, 0, 2, f, kvk.BF16, 64, 0.1, f, None, f, f, f, need, None)  # no w_uv
    _raw(I, "kvk_decode_attention", h, 0, 2, f, kvk.BF16, 65, 0.1, f, f, f, f, f, need, None)    # n_stored
    _raw(I, "kvk_decode_attention", h, 0, 2, f, kvk.BF16, 64, 0.1, Pv(264), f, f, f, f, need, None)  # align
    _raw(B, "kvk_decode_attention", h, 0, 2, f, kvk.BF16, 64, 0.1, f, f, f, f, f, need - 1, None)
    _raw(B, "kvk_decode_splits", h, 0, 2, f, kvk.BF16, 64, 0.1, f, f, f, f, need - 1, None)
    _raw(I, "kvk_compress_layer", h, 0, f, f, kvk.BF16, 65, None, f, None)
    _raw(I, "kvk_compress_layer", h, 0, Pv(264), f, kvk.BF16, 64, None, f, None)  # latent misaligned
    _raw(kvk.OK, "kvk_compress_layer", h, 1, f, f, kvk.BF16, 64, None, f, None)  # inheritor: no-op
    _raw(I, "kvk_append_token", h, 0, 2, f, f, kvk.BF16, 64, f, None)        # stream full
    _raw(I, "kvk_append_token", h, 0, 2, f, Pv(264), kvk.BF16, 10, f, None)  # k^R misaligned
    _raw(kvk.OK, "kvk_append_token", h, 1, 2, f, f, kvk.BF16, 10, f, None)   # inheritors only: no-op


def test_batched_table_accounting_matches_oracle():
    """Per-sequence plans: sequence b's region starts at the oracle's base_b, its
    per-layer offsets and stream sizes are those of its one-sequence table, and the
    algorithmic read bytes are the sum over the sequences."""
    from oracle import plan as OP
    plans = [[(0, 4), (1, 16), (0, 8), (0, 2)], [(0, 16), (0, 2), (1, 16), (1, 16)],
             [(0, 8), (0, 8), (0, 4), (1, 16)]]
    d = kvk.make_dims(kvk.GQA, 4, 8, 2, 128, batch=3, max_tokens=300)
    t = kvk.layer_table_batched(d, [kvk.make_plan(p) for p in plans])
    od = OP.Dims(OP.GQA, 4, 8, 2, 128, batch=3, max_tokens=300)
    oplans = [[OP.Action(bool(a), b) for a, b in p] for p in plans]
    bases, total = OP.batched_arena_bases(od, oplans)
    info = kvk.table_query(t)
    assert info.arena_bytes == total and info.n_anchors == 8 and info.workspace_bytes > 0
    sd = OP.sequence_dims(od)
    for b in range(3):
        si = kvk.table_sequence_query(t, b)
        offs, _ = OP.arena_offsets(sd, oplans[b])
        assert si.layer_offset == [o + bases[b] if o >= 0 else -1 for o in offs]
        assert si.anchor_of == OP.anchor_of(oplans[b])
        for l, (inh, bits) in enumerate(plans[b]):
            if not inh:
                assert si.stream_bytes[l] == OP.stream_bytes(sd, bits)
    for n in (0, 31, 200, 300):
        assert kvk.read_bytes(t, 0, 4, n) == OP.read_bytes_batched(od, oplans, 0, 4, n)
        assert kvk.read_bytes(t, 1, 3, n) == OP.read_bytes_batched(od, oplans, 1, 3, n)


def test_batched_table_rejects_bad_input():
    d = kvk.make_dims(kvk.GQA, 2, 4, 1, 128, batch=2, max_tokens=64)
    with pytest.raises(kvk.KvkError):
        kvk.layer_table_batched(d, [kvk.make_plan([(0, 4), (1, 16)]), kvk.make_plan([(1, 16), (0, 4)])])
    with pytest.raises(kvk.KvkError):
        kvk.layer_table_batched(d, [kvk.make_plan([(0, 4), (1, 16)]), kvk.make_plan([(0, 3), (1, 16)])])
    m = kvk.make_dims(kvk.MLA, 2, 32, 4, 128, 256, 64, 128, 128, batch=2, max_tokens=64)
    with pytest.raises(kvk.KvkError):  # a kept width outside {r/8 .. r} in one sequence's plan
        kvk.layer_table_batched(m, [kvk.make_plan([(0, 8, 128), (1, 16, 0)]), kvk.make_plan([(0, 8, 100), (1, 16, 0)])])
    kvk.layer_table_batched(m, [kvk.make_plan([(0, 8, 128), (1, 16, 0)]), kvk.make_plan([(0, 2, 32), (0, 16, 256)])])
    t = kvk.layer_table_batched(d, [kvk.make_plan([(0, 4), (1, 16)]), kvk.make_plan([(0, 8), (0, 2)])])
    with pytest.raises(kvk.KvkError):
        kvk.table_sequence_query(t, 2)
    u = kvk.layer_table(d, kvk.make_plan([(0, 4), (1, 16)]))
    with pytest.raises(kvk.KvkError):
        kvk.table_sequence_query(u, 0)


def test_host_buffers_are_refused_before_any_launch():
    """A kernel given a pageable host address would fault the GPU: the binding refuses
    host tensors, and the C entry points refuse buffers the HIP runtime does not map
    for the GPU (checked after the size checks, before any launch)."""
    import numpy as np
    import torch
    d = kvk.make_dims(kvk.GQA, 1, 4, 1, 64, batch=1, max_tokens=64)
    t = kvk.layer_table(d, kvk.make_plan([(0, 8)]))
    k = torch.zeros(1, 1, 64, 64, dtype=torch.bfloat16)
    arena = torch.zeros(kvk.table_query(t).arena_bytes, dtype=torch.uint8)
    with pytest.raises(ValueError, match="GPU tensors"):
        kvk.compress_layer(t, 0, k, k, 64, None, arena)
    host = np.zeros(1 << 16, dtype=np.uint8)
    base = host.ctypes.data + (-host.ctypes.data) % 256  # aligned host addresses
    P = ctypes.c_void_p
    hk, ha = P(base), P(base + 16384)
    _raw(kvk.ERR_INVALID, "kvk_compress_layer", t.handle, 0, hk, hk, kvk.BF16, 64, None, ha, None)
    assert "GPU-accessible" in kvk.last_error()
    _raw(kvk.ERR_INVALID, "kvk_decode_attention", t.handle, 0, 1, hk, kvk.BF16, 64, 0.1, None, None, ha, ha,
         P(base + 32768), 1 << 14, None)
    assert "GPU-accessible" in kvk.last_error()
    _raw(kvk.ERR_INVALID, "kvk_append_token", t.handle, 0, 1, hk, hk, kvk.BF16, 10, ha, None)


def test_per_sequence_decode_needs_its_setup():
    """A per-sequence table's decode reads its work list from the workspace that
    kvk_decode_setup wrote: without that set-up the call fails before any launch
    (and copies nothing)."""
    d = kvk.make_dims(kvk.GQA, 2, 4, 1, 64, batch=2, max_tokens=64)
    t = kvk.layer_table_batched(d, [kvk.make_plan([(0, 16), (1, 16)]), kvk.make_plan([(0, 4), (0, 8)])])
    f, P = ctypes.c_void_p(1 << 20), ctypes.c_void_p
    _raw(kvk.ERR_INVALID, "kvk_decode_attention", t.handle, 0, 2, f, kvk.BF16, 64, 0.1, None, None, f, f,
         P(1 << 21), 1 << 20, None)
    assert "kvk_decode_setup" in kvk.last_error()
    _raw(kvk.ERR_INVALID, "kvk_decode_splits", t.handle, 0, 2, f, kvk.BF16, 64, 0.1, None, None, f,
         P(1 << 21), 1 << 20, None)
    _raw(kvk.ERR_INVALID, "kvk_decode_setup", t.handle, 0, 3, P(1 << 21), 1 << 20, None)  # range
    _raw(kvk.ERR_BUFFER, "kvk_decode_setup", t.handle, 0, 2, P(1 << 21), 16, None)         # workspace size
    one = kvk.layer_table(d, kvk.make_plan([(0, 16), (1, 16)]))
    _raw(kvk.OK, "kvk_decode_setup", one.handle, 0, 2, P(1 << 21), 16, None)  # one plan: nothing to write


def test_mla_weight_entry_points_reject_bad_arguments():
    """kvk_set_mla_weights and kvk_mla_arrange_w_uk validate before touching memory;
    an MLA decode that passes no weights needs attached ones."""
    import ctypes
    Pv = ctypes.c_void_p
    f = Pv(256)
    I = kvk.ERR_INVALID
    g = kvk.layer_table(kvk.make_dims(kvk.GQA, 2, 8, 2, 128, max_tokens=64), kvk.make_plan([(0, 4), (1, 16)]))
    _raw(I, "kvk_set_mla_weights", g.handle, f, f)                     # GQA table
    m = kvk.layer_table(kvk.make_dims(kvk.MLA, 2, 32, 4, 128, 256, 64, 128, 128, batch=1, max_tokens=64),
                        kvk.make_plan([(0, 8, 128), (1, 16, 0)]))
    _raw(I, "kvk_set_mla_weights", m.handle, f, None)                  # one of the two
    _raw(I, "kvk_set_mla_weights", m.handle, Pv(264), f)               # misaligned
    _raw(kvk.OK, "kvk_set_mla_weights", m.handle, None, None)          # detaching is always allowed
    need = kvk.workspace_bytes(m, 0, 2)
    _raw(I, "kvk_decode_attention", m.handle, 0, 2, f, kvk.BF16, 64, 0.1, None, None, f, f, f, need, None)
    _raw(I, "kvk_mla_arrange_w_uk", None, 2, 32, 128, 256, f, None)     # NULL input
    _raw(I, "kvk_mla_arrange_w_uk", f, 2, 32, 100, 256, Pv(512), None)  # nope not a multiple of 32
    _raw(I, "kvk_mla_arrange_w_uk", f, 0, 32, 128, 256, Pv(512), None)  # no layers
    _raw(I, "kvk_mla_arrange_w_uk", f, 2, 32, 128, 256, f, None)        # output aliases the input


def test_batched_mla_table_accounting_matches_oracle():
    """Per-sequence MLA plans (kept widths, bit-widths and depth differing per
    sequence): bases, per-layer offsets and read bytes as the oracle's one-sequence
    tables give them; the workspace holds the work list and every sequence's own MLA
    workspace."""
    from oracle import plan as OP
    plans = [[(0, 4, 512), (1, 16, 0), (0, 8, 128)], [(0, 16, 64), (0, 2, 256), (1, 16, 0)],
             [(0, 8, 256), (0, 8, 256), (0, 4, 512)]]
    d = kvk.make_dims(kvk.MLA, 3, 32, 4, 128, 512, 64, 128, 128, batch=3, max_tokens=300)
    t = kvk.layer_table_batched(d, [kvk.make_plan(p) for p in plans])
    od = OP.Dims(OP.MLA, 3, 32, 4, 128, latent_dim=512, rope_dim=64, nope_dim=128, v_dim=128, batch=3,
                 max_tokens=300)
    oplans = [[OP.Action(bool(a), b, r) for a, b, r in p] for p in plans]
    bases, total = OP.batched_arena_bases(od, oplans)
    info = kvk.table_query(t)
    assert info.arena_bytes == total and info.n_anchors == 7
    sd = OP.sequence_dims(od)
    one_ws = 0
    for b in range(3):
        si = kvk.table_sequence_query(t, b)
        offs, _ = OP.arena_offsets(sd, oplans[b])
        assert si.layer_offset == [o + bases[b] if o >= 0 else -1 for o in offs]
        one = kvk.layer_table(kvk.make_dims(kvk.MLA, 3, 32, 4, 128, 512, 64, 128, 128, batch=1, max_tokens=300),
                              kvk.make_plan(plans[b]))
        one_ws += kvk.workspace_bytes(one, 0, 3)
    # the work list (rows and items, a few KiB) at the head, then every sequence's own
    assert one_ws < kvk.workspace_bytes(t, 0, 3) <= one_ws + (16 << 10)
    assert kvk.read_bytes(t, 0, 3, 250) == OP.read_bytes_batched(od, oplans, 0, 3, 250)
