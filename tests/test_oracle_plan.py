"""Pins of the oracle's plan and storage accounting against what the paper prints.

Every expected number here is the paper's (fixtures under tests/golden/ cite the
table they come from) or follows from the paper's own statements.
"""
import math
import os

import pytest

from oracle import plan as P

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _rows(name):
    with open(os.path.join(GOLD, name)) as f:
        return [ln.split() for ln in f if ln.strip() and not ln.startswith("#")]


AXES = {
    "precision": (True, False, False), "depth": (False, False, True),
    "depth+precision": (True, False, True), "rank": (False, True, False),
    "rank+precision": (True, True, False), "depth+rank": (False, True, True),
    "depth+rank+precision": (True, True, True),
}


def _digits(printed: str) -> int:
    return len(printed.split(".")[1]) if "." in printed else 0


@pytest.mark.parametrize("row", _rows("ranges_table.txt"), ids=lambda r: r[0])
def test_eq5_matches_ranges_table(row):
    """App. C.1 table: eq. (5) ranges and |A|^L plan counts for both geometries."""
    name, backbone, actions = row[0], row[1], int(row[2])
    prec, rank, depth = AXES[name]
    mla = backbone == "MLA"
    assert P.n_actions(mla, prec, rank, depth) == actions
    for (L, width, r), cols in (((48, 2048, 1024), row[3:6]), ((36, 512, 256), row[6:9])):
        plans_log10, rmin_p, rmax_p = int(cols[0]), cols[1], cols[2]
        assert round(L * math.log10(actions)) == plans_log10
        rmin, rmax = P.rho_range(L, width, r, 64, mla, prec, rank, depth)
        assert round(rmin, _digits(rmin_p)) == pytest.approx(float(rmin_p))
        assert round(rmax, _digits(rmax_p)) == pytest.approx(float(rmax_p))


@pytest.mark.parametrize("row", _rows("realized_bits_table.txt"), ids=lambda r: "-".join(r[:3]))
def test_storage_accounting_matches_table(row):
    """App. C.3 table: bits/element with metadata (and a 128-token bf16 window in a
    2048 context for KIVI) and rho = 16 / bits."""
    scheme, g, b, bpe, rho = row[0], int(row[1]), int(row[2]), float(row[3]), float(row[4])
    if scheme == "symrow":
        got = P.realized_bits(P.SYMROW, b, g, 0, 2048)
    else:
        got = P.realized_bits(P.KIVI32, b, g, 128, 2048)
    assert round(got, 3) == pytest.approx(bpe)
    assert round(16 / got, 2) == pytest.approx(rho)


def test_storage_accounting_text_figures():
    """App. C.3 text: 2-bit g=128 without the window gives 7.11x; at 16k 4-bit
    g=128 uses 4.34 bits (3.7x).  §4: MLX's grouped 4-bit cache is 3.56x."""
    assert round(16 / P.realized_bits(P.KIVI32, 2, 128, 0, 2048), 2) == 7.11
    b16k = P.realized_bits(P.KIVI32, 4, 128, 128, 16384)
    assert round(b16k, 2) == 4.34 and round(16 / b16k, 1) == 3.7
    assert round(16 / P.realized_bits(P.KIVI32, 4, 64, 0, 1), 2) == 3.56


def test_paper_cache_sizes():
    """§1: Qwen2.5-14B caches 192 KiB per token; 32 sequences of 8k fill 48 GiB."""
    d = P.Dims(P.GQA, 48, 40, 8, 128, batch=32, max_tokens=8192)
    assert d.n_layers * d.kv_width * 2 == 192 * 1024
    assert P.bf16_full_bytes(d) == 48 * 2 ** 30


def test_on_device_factors():
    """§4: rank 128 on the 14B geometry is 10.7x, 12 groups of 4 layers 4x, the
    composition of 4-bit, rank 128 and depth 152x; Fig. 1's maximum is 8 x 10.7 x 48."""
    d = P.Dims(P.MLA, 48, 40, 8, 128, latent_dim=1024, rope_dim=64)
    rank128 = [P.Action(bits=16, rank=128)] * 48
    assert round(P.rho(d, rank128), 1) == 10.7
    gqa = P.Dims(P.GQA, 48, 40, 8, 128)
    depth4 = [P.Action(inherit=(l % 4 != 0), bits=16) for l in range(48)]
    assert P.rho(gqa, depth4) == 4.0
    four_bit = 16 / P.realized_bits(P.KIVI32, 4, 64, 0, 1)
    assert round(four_bit * P.rho(d, rank128) * P.rho(gqa, depth4)) == 152
    one_anchor = [P.Action(bits=2, rank=128)] + [P.Action(inherit=True)] * 47
    assert P.rho(d, one_anchor) == 4096.0


def test_anchor_resolution_and_validation():
    """§2.1 nearest-earlier anchor; §2.2 layer 1 must own a cache; eq. (3)."""
    pl = [P.Action(bits=4), P.Action(inherit=True), P.Action(inherit=True), P.Action(bits=2),
          P.Action(inherit=True)]
    assert P.anchor_of(pl) == [0, 0, 0, 3, 3]
    d = P.Dims(P.GQA, 5, 8, 2, 64)
    assert P.validate(d, pl) is None
    assert P.validate(d, [P.Action(inherit=True)] + pl[1:]) is not None
    assert P.validate(d, [P.Action(bits=3)] + pl[1:]) is not None
    m = P.Dims(P.MLA, 2, 8, 2, 64, latent_dim=512, rope_dim=64)
    assert P.validate(m, [P.Action(bits=4, rank=64), P.Action(bits=8, rank=512)]) is None
    assert P.validate(m, [P.Action(bits=4, rank=96), P.Action(inherit=True)]) is not None


def test_eq1_eq2_gqa_bf16_is_uncompressed():
    """§2.2: a GQA layer at b = 16 costs exactly C0 / L, so rho = 1."""
    d = P.Dims(P.GQA, 28, 28, 4, 128)
    pl = [P.Action(bits=16)] * 28
    assert P.cost_bits(d, pl[0]) * 28 == P.c0_bits(d)
    assert P.rho(d, pl) == 1.0


def test_eviction_composition_factor():
    """§3 long context: ratios multiply; a plan of 20 anchors (16 int2 + 4 int4)
    over 48 layers is 16x by eq. (2), and keeping half the positions doubles it."""
    d = P.Dims(P.GQA, 48, 40, 8, 128)
    pl = ([P.Action(bits=2), P.Action(inherit=True)] * 12 +
          [P.Action(bits=2), P.Action(inherit=True), P.Action(inherit=True)] * 4 +
          [P.Action(bits=4), P.Action(inherit=True), P.Action(inherit=True)] * 4)
    assert len(pl) == 48
    assert P.rho(d, pl) == pytest.approx(48 * 16 / (16 * 2 + 4 * 4))
    assert P.rho(d, pl) * 2 == pytest.approx(32.0)


def test_block_sizes_give_table_bits():
    """Our block layout stores exactly the App. C.3 bits per element: SYMROW
    b + 1/8 (d_h = 128), KIVI32 b + 1 (scale and zero of 16 bits per 32)."""
    for b in (2, 4, 8):
        ds = P.Dims(P.GQA, 1, 1, 1, 128, qscheme=P.SYMROW)
        assert P.block_bytes(ds, b) * 8 / (32 * 2 * 128) == P.realized_bits(P.SYMROW, b, 128, 0, 1)
        dk = P.Dims(P.GQA, 1, 1, 1, 128, qscheme=P.KIVI32)
        assert P.block_bytes(dk, b) * 8 / (32 * 2 * 128) == P.realized_bits(P.KIVI32, b, 32, 0, 1)
    assert P.block_bytes(dk, 16) * 8 / (32 * 2 * 128) == 16
