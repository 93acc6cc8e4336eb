"""GPU parity of the query-aware keep list (kvk_snapkv_select) against the oracle
(oracle.snapkv), through the C ABI.

- Importances: max|diff| <= 1e-4 * max importance (the kernel's scores are bf16
  products accumulated in fp32; the oracle is fp64).
- Selection, exact: the kernel's keep list equals the oracle's selection rule
  applied to the kernel's own importances (the top-k decision taken in the
  kernel's precision).
- Against the oracle's own keep list: any position kept by one side only has an
  oracle importance within 1e-4 * max of the selection threshold.
- Structure: keep_tokens positions per stream, increasing, the window included.
"""
import numpy as np
import pytest
import torch

from oracle import snapkv as S
from paper_2609_37988_amd import kvk, synth

from gpu_common import DEV, TOL, Case, oracle_rows, oracle_stream, rel_err, say

pytestmark = pytest.mark.gpu
W = 32


def _run(B, Hq, Hkv, D, n, keep, seed, zero_keys=False):
    G = Hq // Hkv
    case = Case(1, Hq, Hkv, D, B, n, [(0, 4)], keep=keep)
    k, _ = synth.kv_random(seed, B, Hkv, n, D)
    if zero_keys:
        k = torch.zeros_like(k)
    q = synth.q_random(seed + 1, B, Hq, W, D)  # [B, Hq, 32, D]
    scale = 1.0 / np.sqrt(D)
    keep_out = torch.full((B, Hkv, keep), -1, dtype=torch.int32, device=DEV)
    imp = torch.empty((B, Hkv, n), dtype=torch.float32, device=DEV)
    ws = torch.empty(kvk.snapkv_workspace_bytes(case.table, n), dtype=torch.uint8, device=DEV)
    kvk.snapkv_select(case.table, 0, k.to(DEV).contiguous(), q.to(DEV).contiguous(), n, scale, keep_out, ws,
                      importance=imp)
    torch.cuda.synchronize()
    kn = k.float().numpy().astype(np.float64)
    qn = q.float().numpy().astype(np.float64)
    return case, k, q, scale, keep_out.cpu().numpy(), imp.cpu().numpy(), kn, qn


def _check(B, Hkv, n, keep, keep_gpu, imp_gpu, kn, qn, scale):
    for b in range(B):
        imp_or = S.importance(qn[b], kn[b], scale)
        top = imp_or.max()
        assert np.abs(imp_gpu[b] - imp_or).max() <= 1e-4 * top, "importance differs"
        for h in range(Hkv):
            kl = keep_gpu[b, h]
            assert kl.shape[0] == keep and np.all(np.diff(kl) > 0), "not increasing"
            assert np.array_equal(kl[keep - W:], np.arange(n - W, n)), "window not kept"
            assert np.array_equal(kl, S.select(imp_gpu[b, h].astype(np.float64), keep)), \
                f"selection differs from the rule on the kernel's importances (b {b}, h {h})"
            ref = S.select(imp_or[h], keep)
            diff = np.setxor1d(kl, ref)
            if diff.size:
                pre = np.sort(imp_or[h][:n - W])[::-1]
                theta = pre[keep - W - 1] if keep > W else np.inf
                assert np.all(np.abs(imp_or[h][diff] - theta) <= 1e-4 * top), \
                    f"positions {diff[:8]} differ away from the threshold"


@pytest.mark.parametrize("Hq,Hkv,D,n,keep", [
    (10, 2, 128, 300, 150),     # G 5 (the 14B group), ragged length, one chunk
    (10, 2, 128, 4500, 1125),   # three chunks, keep 1/4
    (8, 1, 128, 2100, 263),     # G 8 (the widest), chunk boundary just past 2048
    (4, 4, 64, 777, 400),       # G 1, d_h 64
])
def test_snapkv_matches_oracle(Hq, Hkv, D, n, keep):
    say(f"case snapkv Hq={Hq} Hkv={Hkv} D={D} n={n} keep={keep}")
    B = 2
    case, k, q, scale, keep_gpu, imp_gpu, kn, qn = _run(B, Hq, Hkv, D, n, keep, 700 + n)
    _check(B, Hkv, n, keep, keep_gpu, imp_gpu, kn, qn, scale)


@pytest.mark.parametrize("n,keep", [(40, 32), (40, 40), (33, 33), (96, 50)])
def test_snapkv_edges(n, keep):
    """Window only, keep everything, a single prefix position, and a small ragged case."""
    say(f"case snapkv edge n={n} keep={keep}")
    case, k, q, scale, keep_gpu, imp_gpu, kn, qn = _run(1, 10, 2, 128, n, keep, 800 + n + keep)
    _check(1, 2, n, keep, keep_gpu, imp_gpu, kn, qn, scale)
    if keep == n:
        assert np.array_equal(keep_gpu[0, 0], np.arange(n))


def test_snapkv_ties_keep_lowest_positions():
    """Zero keys: every prefix position has the same importance, so the lowest ones
    are kept; the importances of all positions add up to G * 32."""
    say("case snapkv ties")
    n, keep = 500, 100
    case, k, q, scale, keep_gpu, imp_gpu, kn, qn = _run(1, 10, 2, 128, n, keep, 900, zero_keys=True)
    want = np.concatenate([np.arange(keep - W), np.arange(n - W, n)])
    for h in range(2):
        assert np.array_equal(keep_gpu[0, h], want)
        assert abs(imp_gpu[0, h].sum() - 5 * W) <= 1e-3


def test_snapkv_ties_across_selection_slices():
    """Zero keys over 9000 positions: the selection runs on three slices of each
    stream, and the lowest keep - 32 = 4000 prefix positions (equal importances,
    the threshold tie running across the first slice boundary) are kept in order."""
    say("case snapkv ties across slices")
    n, keep = 9000, 4032
    case, k, q, scale, keep_gpu, imp_gpu, kn, qn = _run(1, 10, 2, 128, n, keep, 960, zero_keys=True)
    want = np.concatenate([np.arange(keep - W), np.arange(n - W, n)])
    for h in range(2):
        assert np.array_equal(keep_gpu[0, h], want)


def test_snapkv_keep_list_drives_the_eviction_write():
    """The selected positions go to kvk_compress_layer as keep_idx; decode over the
    evicted int4 cache matches the oracle's attention over the same positions."""
    say("case snapkv -> eviction write -> decode")
    B, Hq, Hkv, D, n, keep = 2, 10, 2, 128, 1000, 500
    case, k, q, scale, keep_gpu, imp_gpu, kn, qn = _run(B, Hq, Hkv, D, n, keep, 950)
    _, v = synth.kv_random(951, B, Hkv, n, D)
    case.compress(0, k.to(DEV), v.to(DEV), n, torch.from_numpy(keep_gpu).to(DEV))
    qd = synth.q_random(952, 1, B, Hq, D)
    out = case.decode(qd.to(DEV), keep, scale).cpu().numpy()
    vn = v.float().numpy()
    qdn = qd.float().numpy().astype(np.float64)
    ref = np.zeros_like(out, dtype=np.float64)
    for b in range(B):
        for h in range(Hkv):
            st = oracle_stream(case.odims, 4, k[b, h].float().numpy(), vn[b, h], keep_gpu[b, h])
            ref[0, b, 5 * h:5 * h + 5] = oracle_rows(case.odims, 4, st, keep, qdn[0, b, 5 * h:5 * h + 5], scale)
    err = rel_err(out, ref)
    say(f"  max|diff| / max|out| = {err:.2e}")
    assert err <= TOL
