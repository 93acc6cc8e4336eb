"""GPU parity of the selector forward pass (kvk_selector_forward) against the oracle
(oracle.selector), through the C ABI.

Tolerance on the logits, derived from the roundings the kernels take: on its way
through the two blocks a prompt position's activations are rounded to bf16 six
times per block (the normalised input of each sublayer, the rotated q and k and
the value, the attention probabilities, the attention output, the SwiGLU hidden
layer): twelve roundings, each an independent relative error uniform within
+-2^-9 (standard deviation 2^-9 / sqrt 3).  Their root sum of squares is
sqrt(12 / 3) * 2^-9 = 2^-8 of an activation; everything else (fp32 accumulation,
the fp32 RoPE table formed in fp64, the fp32 pooling and heads) is two orders
below.  The logits are compared within 2^-8 of the largest logit.  The actions
are the argmax of the kernel's own logits exactly (the decision in the kernel's
precision), and equal the oracle's on every layer whose two best oracle logits are
further apart than twice the tolerance; the share of layers so checked is printed
and must be at least half.
"""
import numpy as np
import pytest
import torch

from oracle import selector as S
from paper_2609_37988_amd import kvk

from gpu_common import DEV, say

pytestmark = pytest.mark.gpu
TOL_SEL = 2.0 ** -8
W, F = 256, 1024


def _bf16(x):
    return torch.from_numpy(np.asarray(x, np.float32)).to(torch.bfloat16)


def _weights(seed, d_model, L, A):
    """Oracle weights (bf16 values as float64) and the packed bf16 vector of kvk.h."""
    rng = np.random.default_rng(seed)

    def mat(n_out, n_in, gain=1.0):
        return _bf16(rng.standard_normal((n_out, n_in)) * gain / np.sqrt(n_in))

    def gain_vec():
        return _bf16(1.0 + 0.1 * rng.standard_normal(W))

    w_in = mat(W, d_model)
    packed, blocks = [w_in], []
    for _ in range(2):
        p = {"g_attn": gain_vec(), "w_q": mat(W, W, 1.5), "w_k": mat(W, W, 1.5), "w_v": mat(W, W),
             "w_o": mat(W, W), "g_ffn": gain_vec(), "w_gate": mat(F, W), "w_up": mat(F, W),
             "w_down": mat(W, F)}
        packed += [p[k] for k in S.BLOCK_KEYS]
        blocks.append({k: v.double().numpy() for k, v in p.items()})
    g_final = gain_vec()
    w_head = mat(L * A, W).reshape(L, A, W)
    b_head = _bf16(0.1 * rng.standard_normal((L, A)))
    packed += [g_final, w_head, b_head]
    ow = {"w_in": w_in.double().numpy(), "blocks": blocks, "g_final": g_final.double().numpy(),
          "w_head": w_head.double().numpy(), "b_head": b_head.double().numpy()}
    vec = torch.cat([t.reshape(-1) for t in packed]).contiguous()
    assert vec.numel() == kvk.selector_weight_elems(d_model, L, A)
    return ow, vec


def _run(d_model, L, A, packed, emb, depth=True, film=None):
    T = emb.shape[0]
    actions = torch.empty(L, dtype=torch.int32, device=DEV)
    logits = torch.empty((L, A), dtype=torch.float32, device=DEV)
    ws = torch.empty(kvk.selector_workspace_bytes(d_model, L, T), dtype=torch.uint8, device=DEV)
    kvk.selector_forward(d_model, L, packed, emb, actions, ws, logits=logits, n_actions=A, depth=depth,
                         film=film)
    torch.cuda.synchronize()
    return logits.cpu().numpy().astype(np.float64), actions.cpu().numpy()


def _compare(got, act, ref, depth=True):
    assert np.isneginf(got[0, 0]) and np.isneginf(ref[0, 0])
    if not depth:
        assert np.isneginf(got[:, 0]).all()
    fin = np.isfinite(ref)
    assert np.array_equal(fin, np.isfinite(got))
    top = np.abs(ref[fin]).max()
    err = np.abs(got[fin] - ref[fin]).max() / top
    assert np.array_equal(act, np.argmax(got, axis=1)), "actions are not the argmax of the kernel's logits"
    assert act[0] != 0, "layer 0 inherits"
    srt = np.sort(ref, axis=1)
    clear = (srt[:, -1] - srt[:, -2]) > 2 * TOL_SEL * top
    say(f"  max|diff| / max|logit| = {err:.2e}; argmax checked on {clear.sum()} of {len(clear)} layers")
    assert err <= TOL_SEL
    assert np.array_equal(act[clear], np.argmax(ref, axis=1)[clear])
    assert clear.mean() >= 0.5
    return err


@pytest.mark.parametrize("T,L,A,depth,film", [(100, 48, 17, True, False), (1000, 48, 5, True, True),
                                              (3000, 48, 17, False, False), (1, 64, 17, True, False),
                                              (300, 7, 5, True, True), (257, 28, 17, True, True)])
def test_selector_matches_oracle(T, L, A, depth, film):
    """d_model 512: the input map takes 2 or 4 splits over K at these lengths; T = 1,
    257 and 300 leave ragged key tiles and row tiles."""
    d_model = 512
    say(f"case selector T={T} L={L} A={A} depth={depth} film={film}")
    ow, packed = _weights(1500 + T, d_model, L, A)
    rng = np.random.default_rng(1600 + T)
    emb = _bf16(rng.standard_normal((T, d_model)))
    fv = None
    if film:
        fv = (0.3 * rng.standard_normal(W), 0.3 * rng.standard_normal(W))
    ft = torch.from_numpy(np.stack(fv).astype(np.float32)).to(DEV) if film else None
    got, act = _run(d_model, L, A, packed.to(DEV), emb.to(DEV), depth=depth, film=ft)
    ref = S.logits(emb.double().numpy(), ow, depth=depth,
                   film=None if fv is None else (ft[0].double().cpu().numpy(), ft[1].double().cpu().numpy()))
    _compare(got, act, ref, depth)


def test_selector_positions_matter():
    """Reversing the prompt changes the kernel's logits by far more than the tolerance,
    as it changes the oracle's (rotary positions; a model without them is invariant)."""
    d_model, L, A, T = 512, 16, 17, 200
    say(f"case selector reversed prompt T={T}")
    ow, packed = _weights(1900, d_model, L, A)
    emb = _bf16(np.random.default_rng(1901).standard_normal((T, d_model)))
    z1, _ = _run(d_model, L, A, packed.to(DEV), emb.to(DEV))
    z2, a2 = _run(d_model, L, A, packed.to(DEV), emb.flip(0).contiguous().to(DEV))
    ref2 = S.logits(emb.flip(0).double().numpy(), ow)
    fin = np.isfinite(z1)
    top = np.abs(z1[fin]).max()
    say(f"  reversed: max|diff| / max|logit| = {np.abs(z2[fin] - z1[fin]).max() / top:.2e}")
    assert np.abs(z2[fin] - z1[fin]).max() > 10 * TOL_SEL * top
    _compare(z2, a2, ref2)


def test_selector_14b_width_8k_matches_oracle():
    """The 14B embedding width (5120) and 48 layers at 8192 prompt tokens, the launch
    shape the benchmark times (the input map and the down projection split over K,
    4 key splits in the attention): logits against the oracle, actions the argmax."""
    d_model, L, A, T = 5120, 48, 5, 8192
    say(f"case selector d_model {d_model} T={T}")
    ow, packed = _weights(1700, d_model, L, A)
    emb = _bf16(np.random.default_rng(1701).standard_normal((T, d_model)))
    got, act = _run(d_model, L, A, packed.to(DEV), emb.to(DEV))
    ref = S.logits(emb.double().numpy(), ow)
    _compare(got, act, ref)


def test_selector_32k_properties():
    """32768 prompt tokens at the 14B width with 17 actions (the oracle's attention
    would take minutes): two calls bit-identical (split-K partials summed in a fixed
    order), actions the argmax of finite logits, and a prompt of one token repeated
    32768 times giving the logits of that token alone (identical rows attend to
    their common value whatever their positions, so every row stays the one-token
    row), within the tolerance."""
    d_model, L, A, T = 5120, 48, 17, 32768
    say(f"case selector d_model {d_model} T={T} properties")
    _, packed = _weights(1800, d_model, L, A)
    packed = packed.to(DEV)
    g = torch.Generator(device=DEV)
    g.manual_seed(1801)
    emb = torch.randn((T, d_model), generator=g, device=DEV).to(torch.bfloat16)
    z1, a1 = _run(d_model, L, A, packed, emb)
    z2, a2 = _run(d_model, L, A, packed, emb)
    assert np.array_equal(z1, z2) and np.array_equal(a1, a2), "not deterministic"
    fin = np.isfinite(z1)
    assert fin.sum() == L * A - 1 and np.isneginf(z1[0, 0])
    assert np.array_equal(a1, np.argmax(z1, axis=1)) and a1[0] != 0
    row = emb[12345:12346]
    zr, _ = _run(d_model, L, A, packed, row.expand(T, d_model).contiguous())
    z0, _ = _run(d_model, L, A, packed, row.contiguous())
    top = np.abs(z0[fin]).max()
    err = np.abs(zr[fin] - z0[fin]).max() / top
    say(f"  repeated token vs single token: max|diff| / max|logit| = {err:.2e}")
    assert err <= TOL_SEL


def test_selector_rejects_bad_sizes():
    with pytest.raises(Exception):
        kvk.selector_weight_elems(512, 8, 1)
    with pytest.raises(Exception):
        kvk.selector_weight_elems(500, 8, 5)
