"""GPU parity of the MLA write with the down-projection on the matrix cores
(§2.1 "Rank", App. C.2), through the C ABI.

Three checks per case:
  * the bf16 latent the kernel stored (latent_out) against the oracle's exact
    projection: equal to it rounded once to bf16 for all but a small share of the
    values (fp32 accumulation can cross a bf16 rounding boundary), and everywhere
    within the bound of an fp32 sum of H products followed by one bf16 rounding,
    |got - c| <= 2^-8 (|c| + g) + g with g = H 2^-24 sum_k |x_k w_k| (bf16
    products are exact in fp32; near-cancelling sums can be several ulps off);
  * the arena bytes bit-exact against the oracle's write of the kernel's own
    latent (the quantiser and the layout are integer work once the latent is fixed);
  * decode attention over the projected cache within 2e-3 * max|out| of the
    oracle's cache built from the exact projection.
"""
import numpy as np
import pytest
import torch

from oracle import mla as OM
from paper_2609_37988_amd import kvk, synth

from gpu_common import TOL, rel_err, say
from test_gpu_mla import DEV, SCALE, MlaCase, _np

pytestmark = pytest.mark.gpu

MAX_OFF_SHARE = 0.01


def _check_latent(got, X, W, d):
    """got [n, d] (fp32 copies of bf16) against the exact projection of X [n, H]."""
    H = X.shape[1]
    c = np.asarray(X, np.float64) @ np.asarray(W, np.float64)[:d].T
    g = H * 2.0 ** -24 * (np.abs(np.asarray(X, np.float64)) @ np.abs(np.asarray(W, np.float64))[:d].T)
    err = np.abs(got.astype(np.float64) - c)
    assert np.all(err <= 2.0 ** -8 * (np.abs(c) + g) + g), "latent outside the fp32-sum error bound"
    off = float(np.mean(got.astype(np.float64) != OM.project_latent(X, W, d)))
    say(f"  latent: {off:.2e} of values differ from the once-rounded projection, "
        f"max err / bound {float(np.max(err / (2.0 ** -8 * (np.abs(c) + g) + g))):.2f}")
    assert off <= MAX_OFF_SHARE


def _run(H, d, bits, qs, n, B=2, keep=0, seed=0, decode=True, r=512):
    c = MlaCase(1, 32, r, B, n if keep else (n + 31) // 32 * 32, [(0, bits, d)], qscheme=qs, keep=keep)
    X = synth.latent_random(seed + 1, B, n, H)
    W = synth.weights_random(seed + 2, 1, 1, r, H)[0, 0].contiguous()
    R = synth.latent_random(seed + 3, B, n, 64)
    kidx = synth.keep_random(seed + 4, B, 1, n, keep).reshape(B, keep) if keep else None
    ns = keep if keep else n
    lat = torch.full((B, ns, d), float("nan"), dtype=torch.bfloat16, device=DEV)
    kvk.compress_layer_project(c.table, 0, X.to(DEV), W.to(DEV), R.to(DEV), n,
                               None if kidx is None else kidx.to(DEV), c.arena, lat)
    got_lat = _np(lat)
    Xn, Wn, Rn = _np(X), _np(W), _np(R)
    kn = None if kidx is None else kidx.numpy()
    Xs = np.concatenate([Xn[b] if kn is None else Xn[b, kn[b]] for b in range(B)])
    _check_latent(got_lat.reshape(-1, d), Xs, Wn, d)
    # Bytes: the oracle's write of the kernel's latent (stored tokens, in order).
    Rs = Rn if kn is None else np.stack([Rn[b, kn[b]] for b in range(B)])
    ref = OM.compress_layer(c.odims, bits, d, got_lat, Rs)
    off, nb = c.info.layer_offset[0], c.info.layer_bytes[0]
    assert np.array_equal(c.arena[off:off + nb].cpu().numpy(), ref), "arena bytes differ"
    if not decode:
        return
    # Attention over the projected cache vs the oracle's cache of the exact projection.
    full = np.zeros((B, n, r), np.float32)
    for b in range(B):
        full[b, :, :d] = OM.project_latent(Xn[b], Wn, d)
    c.inputs[0] = (full, Rn, kn)
    q = synth.q_random(seed + 5, 1, B, 32, 192)
    wk = synth.weights_random(seed + 6, 1, 32, 128, r)
    wv = synth.weights_random(seed + 7, 1, 32, 128, r)
    out = _np(c.decode(q, wk, wv, ns, SCALE))
    err = rel_err(out, c.oracle_out(q, wk, wv, ns, SCALE))
    say(f"  decode max|diff| / max|out| = {err:.2e}")
    assert err <= TOL


@pytest.mark.parametrize("qs", [kvk.KIVI32, kvk.SYMROW], ids=["kivi32", "symrow"])
@pytest.mark.parametrize("bits", [16, 8, 4, 2])
@pytest.mark.parametrize("d", [64, 512])
def test_project_ragged(qs, bits, d):
    """Model width 512, 200 tokens (6 full blocks + an 8-token tail), B 2."""
    say(f"case project H=512 d={d} bits={bits} qs={qs}")
    _run(512, d, bits, qs, 200, seed=100 + bits + d)


@pytest.mark.parametrize("r,d", [(256, 32), (512, 128), (512, 256)])
def test_project_other_widths(r, d):
    """The remaining kept widths (32 needs r 256) at 4 bits, model width 256, 70 tokens."""
    say(f"case project H=256 r={r} d={d}")
    _run(256, d, 4, kvk.KIVI32, 70, seed=200 + d, r=r)


@pytest.mark.parametrize("keep", [150, 128])
def test_project_eviction(keep):
    """Stored tokens are a sorted subset of 300 (150: a ragged tail; 128: whole
    groups, an empty tail): the kernel projects only them."""
    say(f"case project eviction {keep} of 300")
    _run(384, 256, 4, kvk.KIVI32, 300, keep=keep, seed=300 + keep)


def test_project_short_and_inheritor():
    """Fewer tokens than one block (tail only); an inheriting layer is a no-op."""
    say("case project tail only")
    _run(512, 128, 8, kvk.KIVI32, 9, seed=400)
    c = MlaCase(2, 32, 512, 1, 32, [(0, 16, 512), (1, 16, 0)])
    before = c.arena.clone()
    X = synth.latent_random(1, 1, 10, 64).to(DEV)
    W = synth.weights_random(2, 1, 1, 512, 64)[0, 0].contiguous().to(DEV)
    R = synth.latent_random(3, 1, 10, 64).to(DEV)
    kvk.compress_layer_project(c.table, 1, X, W, R, 10, None, c.arena)
    assert torch.equal(c.arena, before)


@pytest.mark.parametrize("qs,d", [(kvk.KIVI32, 512), (kvk.SYMROW, 256)], ids=["kivi32-512", "symrow-256"])
def test_project_full_size_sample(qs, d):
    """The 32-layer latent stack's layer write at full size: B 16, 16384 tokens, r 512,
    model width 2048 (DeepSeek-V2-Lite's), int4.  Sampled: the latent of 96 tokens
    against the exact projection, and two whole sequences' streams against the
    oracle's write of the kernel's latent."""
    say(f"case project full-size B=16 n=16384 H=2048 d={d} qs={qs} int4")
    B, n, H, r = 16, 16384, 2048, 512
    c = MlaCase(1, 32, r, B, n, [(0, 4, d)], qscheme=qs)
    X = synth.latent_random(501, B, n, H, device=DEV)
    W = synth.weights_random(502, 1, 1, r, H, device=DEV)[0, 0].contiguous()
    R = synth.latent_random(503, B, n, 64, device=DEV)
    lat = torch.empty((B, n, d), dtype=torch.bfloat16, device=DEV)
    kvk.compress_layer_project(c.table, 0, X, W, R, n, None, c.arena, lat)
    torch.cuda.synchronize()
    rng = np.random.default_rng(7)
    bs, ts = rng.integers(B, size=96), rng.integers(n, size=96)
    _check_latent(_np(lat[bs, ts]), _np(X[bs, ts]), _np(W), d)
    off, sb = c.info.layer_offset[0], c.info.stream_bytes[0]
    for b in (0, int(rng.integers(1, B))):
        ref = OM.compress_stream(c.odims, 4, d, _np(lat[b]), _np(R[b]))
        got = c.arena[off + b * sb:off + (b + 1) * sb].cpu().numpy()
        assert np.array_equal(got, ref), f"stream {b} bytes differ"


def test_project_refusals():
    """Host-side rejections: GQA tables, d_model not a multiple of 32."""
    c = MlaCase(1, 32, 512, 1, 32, [(0, 16, 512)])
    X = torch.zeros((1, 4, 40), dtype=torch.bfloat16, device=DEV)
    W = torch.zeros((512, 40), dtype=torch.bfloat16, device=DEV)
    R = torch.zeros((1, 4, 64), dtype=torch.bfloat16, device=DEV)
    with pytest.raises(kvk.KvkError):
        kvk.compress_layer_project(c.table, 0, X, W, R, 4, None, c.arena)
