"""GPU parity of the MLA query-aware keep list (kvk_snapkv_select_mla) against the
oracle (oracle.snapkv.importance_mla), through the C ABI.

- Importances: max|diff| <= 2e-3 * max importance (the window queries are absorbed
  into fp16, q~ = W_UK^T q_nope, and scored against the latent with fp16 products
  accumulated in fp32; the oracle reconstructs every head's keys in fp64).
- Selection, exact: the kernel's keep list equals the oracle's selection rule
  applied to the kernel's own importances (the decision taken in its precision).
- Against the oracle's own keep list: a position kept by one side only has an
  oracle importance within 2e-3 * max of the selection threshold.
- Structure: keep_tokens positions per sequence, increasing, the window included.
"""
import numpy as np
import pytest
import torch

from oracle import snapkv as S
from paper_2609_37988_amd import kvk, synth

from gpu_common import say

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
W = 32
TOL_IMP = 2e-3


def _table(Hq, r, B, n, keep, L=1, plan=None):
    d = kvk.make_dims(kvk.MLA, L, Hq, 4, 128, r, 64, 128, 128, batch=B, max_tokens=n, keep_tokens=keep)
    return kvk.layer_table(d, kvk.make_plan(plan or [(0, 4, r)]))


def _run(Hq, r, B, n, keep, seed, attach=False):
    t = _table(Hq, r, B, n, keep)
    C = synth.latent_random(seed, B, n, r)
    R = synth.latent_random(seed + 1, B, n, 64)
    q = synth.q_random(seed + 2, B, W, Hq, 192)  # [B, 32, Hq, nope + 64]
    wk = synth.weights_random(seed + 3, 1, Hq, 128, r)  # [1, Hq, nope, r]
    wk_lib = kvk.mla_weights_for_library(wk.to(DEV))
    scale = 1.0 / np.sqrt(192.0)
    keep_out = torch.full((B, keep), -1, dtype=torch.int32, device=DEV)
    imp = torch.empty((B, n), dtype=torch.float32, device=DEV)
    ws = torch.empty(kvk.snapkv_workspace_bytes(t, n), dtype=torch.uint8, device=DEV)
    if attach:
        wv = synth.weights_random(seed + 4, 1, Hq, 128, r).to(DEV).contiguous()
        kvk.set_mla_weights(t, wk_lib, wv)
        kvk.snapkv_select_mla(t, 0, C.to(DEV), R.to(DEV), q.to(DEV), n, scale, keep_out, ws, importance=imp)
    else:
        kvk.snapkv_select_mla(t, 0, C.to(DEV), R.to(DEV), q.to(DEV), n, scale, keep_out, ws, w_uk=wk_lib[0],
                              importance=imp)
    torch.cuda.synchronize()
    return (keep_out.cpu().numpy(), imp.cpu().numpy(), C.float().numpy(), R.float().numpy(),
            q.float().numpy(), wk[0].float().numpy(), scale)


def _check(B, n, keep, keep_gpu, imp_gpu, C, R, q, wk, scale):
    for b in range(B):
        imp_or = S.importance_mla(np.transpose(q[b], (1, 0, 2)), C[b], R[b], wk, scale)
        top = imp_or.max()
        err = np.abs(imp_gpu[b] - imp_or).max() / top
        say(f"  sequence {b}: importance max|diff| / max = {err:.2e}")
        assert err <= TOL_IMP, "importance differs"
        kl = keep_gpu[b]
        assert kl.shape[0] == keep and np.all(np.diff(kl) > 0), "not increasing"
        assert np.array_equal(kl[keep - W:], np.arange(n - W, n)), "window not kept"
        assert np.array_equal(kl, S.select(imp_gpu[b].astype(np.float64), keep)), \
            f"selection differs from the rule on the kernel's importances (b {b})"
        ref = S.select(imp_or, keep)
        diff = np.setxor1d(kl, ref)
        if diff.size:
            pre = np.sort(imp_or[:n - W])[::-1]
            theta = pre[keep - W - 1] if keep > W else np.inf
            assert np.all(np.abs(imp_or[diff] - theta) <= TOL_IMP * top), \
                f"positions {diff[:8]} differ away from the threshold"


@pytest.mark.parametrize("Hq,r,n,keep", [
    (32, 512, 300, 150),    # the 32-layer stack's heads and width, one chunk plus a ragged tail
    (40, 1024, 600, 200),   # Qwen2.5-14B's heads (padded to 64 inside) and width, three chunks
    (16, 256, 777, 400),    # a narrow latent, 16 heads (one padded chunk)
])
def test_snapkv_mla_matches_oracle(Hq, r, n, keep):
    say(f"case snapkv mla Hq={Hq} r={r} n={n} keep={keep}")
    B = 2
    keep_gpu, imp_gpu, C, R, q, wk, scale = _run(Hq, r, B, n, keep, 1500 + n)
    _check(B, n, keep, keep_gpu, imp_gpu, C, R, q, wk, scale)


@pytest.mark.parametrize("n,keep", [(40, 32), (40, 40), (33, 33), (96, 50)])
def test_snapkv_mla_edges(n, keep):
    """Window only, keep everything, a single prefix position, a small ragged case;
    the weights attached to the table."""
    say(f"case snapkv mla edges n={n} keep={keep}")
    keep_gpu, imp_gpu, C, R, q, wk, scale = _run(32, 512, 1, n, keep, 1600 + n, attach=True)
    _check(1, n, keep, keep_gpu, imp_gpu, C, R, q, wk, scale)


def test_snapkv_mla_full_size_properties():
    """The 32-layer latent stack's shape (B 16, 16384 tokens, 32 heads, r 512), one
    layer, keeping a quarter: deterministic, every sequence's importances add up to
    32 heads x 32 window queries, the keep lists follow the rule on the kernel's
    importances and hold the window."""
    say("case snapkv mla full size")
    B, n, Hq, r, keep = 16, 16384, 32, 512, 4096
    t = _table(Hq, r, B, n, keep)
    C = synth.latent_random(1700, B, n, r, device=DEV)
    R = synth.latent_random(1701, B, n, 64, device=DEV)
    q = synth.q_random(1702, B, W, Hq, 192, device=DEV)
    wk = kvk.mla_weights_for_library(synth.weights_random(1703, 1, Hq, 128, r, device=DEV))[0]
    ws = torch.empty(kvk.snapkv_workspace_bytes(t, n), dtype=torch.uint8, device=DEV)
    outs = []
    for _ in range(2):
        keep_out = torch.empty((B, keep), dtype=torch.int32, device=DEV)
        imp = torch.empty((B, n), dtype=torch.float32, device=DEV)
        kvk.snapkv_select_mla(t, 0, C, R, q, n, 1.0 / np.sqrt(192.0), keep_out, ws, w_uk=wk, importance=imp)
        outs.append((keep_out.cpu().numpy(), imp.cpu().numpy()))
    assert np.array_equal(outs[0][0], outs[1][0]) and np.array_equal(outs[0][1], outs[1][1])
    keep_gpu, imp_gpu = outs[0]
    mass = imp_gpu.astype(np.float64).sum(axis=1)
    say(f"  mass: {mass.min():.4f} .. {mass.max():.4f} (want {Hq * W})")
    assert np.allclose(mass, Hq * W, rtol=1e-4)
    for b in range(B):
        kl = keep_gpu[b]
        assert np.array_equal(kl[keep - W:], np.arange(n - W, n))
        assert np.array_equal(kl, S.select(imp_gpu[b].astype(np.float64), keep))
