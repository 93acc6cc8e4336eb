"""GPU parity of depth sharing at the paper's extremes (§2.1 depth, eq. (3), App. C.1
eq. (5)): anchors read by more query rows than one 64-row workgroup holds, up to one
anchor serving every layer.  Each layer attends with its own query to its anchor's
cache; the outputs are compared with the oracle (max|diff| <= 2e-3 * max|out|), and
two layers given the same query return bitwise equal outputs wherever their rows
sit among the anchor's row chunks.
"""
import numpy as np
import pytest
import torch

from paper_2609_37988_amd import kvk, synth

from gpu_common import DEV, TOL, Case, oracle_rows, oracle_stream, rel_err, say

pytestmark = pytest.mark.gpu


def _check(L, Hq, Hkv, D, B, T, plan, qs, seed):
    G = Hq // Hkv
    c = Case(L, Hq, Hkv, D, B, (T + 31) // 32 * 32, plan, qscheme=qs)
    inputs = {}
    for l, (inh, bits) in enumerate(plan):
        if inh:
            continue
        k, v = synth.kv_random(seed + l, B, Hkv, T, D)
        c.compress(l, k.to(DEV), v.to(DEV), T)
        inputs[l] = (k.float().numpy(), v.float().numpy(), bits)
    q = synth.q_random(seed + 100, L, B, Hq, D)
    group0 = [l for l in range(L) if c.info.anchor_of[l] == 0]
    same = [group0[-1], group0[len(group0) // 2]]  # these layers ask layer 0's questions
    for l in same:
        q[l] = q[0]
    scale = 1.0 / np.sqrt(D)
    out = c.decode(q.to(DEV), T, scale).cpu().numpy()
    assert all(np.array_equal(out[l], out[0]) for l in same), \
        "equal queries of layers sharing an anchor gave different outputs"
    got, ref = [], []
    for (a, b, h) in {(c.info.anchor_of[l], b, h) for l in range(L) for b in range(B) for h in range(Hkv)}:
        K, V, bits = inputs[a]
        st = oracle_stream(c.odims, bits, K[b, h], V[b, h])
        readers = [l for l in range(L) if c.info.anchor_of[l] == a]
        rows = np.concatenate([q[l, b, h * G:(h + 1) * G].float().numpy() for l in readers]).astype(np.float64)
        ref.append(oracle_rows(c.odims, bits, st, T, rows, scale))
        got.append(np.concatenate([out[l, b, h * G:(h + 1) * G] for l in readers]))
    err = rel_err(np.concatenate(got), np.concatenate(ref))
    say(f"  max|diff| / max|out| = {err:.2e}")
    assert err <= TOL


@pytest.mark.parametrize("qs,bits", [(kvk.KIVI32, 16), (kvk.KIVI32, 8), (kvk.KIVI32, 4), (kvk.KIVI32, 2),
                                     (kvk.SYMROW, 4), (kvk.GROUP64, 2)])
def test_one_anchor_serves_all_48_layers(qs, bits):
    """Qwen2.5-14B heads (40 / 8, d_h 128): layer 0 is the only anchor, its cache read
    by all 48 layers (240 query rows per KV head: 16 chunk waves in 4 workgroups);
    1000 tokens (31 blocks and an 8-token tail)."""
    say(f"case depth: one anchor for 48 layers, qs={qs} bits={bits}")
    _check(48, 40, 8, 128, 2, 1000, [(0, bits)] + [(1, 16)] * 47, qs, 3000 + bits)


def test_long_and_short_groups_mixed():
    """Qwen2.5-7B heads (28 / 4, G 7): a 10-layer group (70 rows, just past one
    workgroup), a 2-layer group, a 16-layer group of int2 (112 rows)."""
    say("case depth: groups of 10, 2, 16 layers at G 7")
    plan = [(0, 4)] + [(1, 16)] * 9 + [(0, 8), (1, 16)] + [(0, 2)] + [(1, 16)] * 15
    _check(28, 28, 4, 128, 3, 333, plan, kvk.KIVI32, 3100)


def test_sixty_four_layers_one_anchor_g8():
    """The largest plan the table takes: 64 layers on one anchor with 8 query heads
    per KV head (512 rows: 32 chunk waves in 8 workgroups), d_h 64."""
    say("case depth: 64 layers x G 8 on one anchor, d_h 64")
    _check(64, 16, 2, 64, 1, 200, [(0, 8)] + [(1, 16)] * 63, kvk.KIVI32, 3200)
