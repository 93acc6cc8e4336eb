"""GPU parity of the selector forward pass (kvk_selector_forward) against the oracle
(oracle.selector), through the C ABI.

Tolerance on the logits, derived from the arithmetic: the kernels round ten
activations per prompt position to bf16 on their way into the matrix cores (per
block: the two normalised inputs, q/k/v, the attention output, the feed-forward
hidden layer), each a relative error of at most 2^-9; accumulated in fp32 they stay
well below 2e-2 of the largest logit.  The actions are the argmax of the kernel's own
logits exactly (the decision in the kernel's precision), and they equal the oracle's
wherever the oracle's two best logits of a layer are further apart than twice that.
"""
import numpy as np
import pytest
import torch

from oracle import selector as S
from paper_2609_37988_amd import kvk

from gpu_common import DEV, say

pytestmark = pytest.mark.gpu
TOL_SEL = 2e-2
W, F = 256, 1024


def _bf16(x):
    return torch.from_numpy(np.asarray(x, np.float32)).to(torch.bfloat16)


def _weights(seed, d_model, L):
    """Oracle weights ([in, out], bf16 values as float64) and the packed bf16 vector."""
    rng = np.random.default_rng(seed)

    def mat(fan_in, fan_out):
        return _bf16(rng.standard_normal((fan_in, fan_out)) / np.sqrt(fan_in))

    def vec(n, mean=0.0, sd=0.05):
        return _bf16(mean + sd * rng.standard_normal(n))

    w_in, b_in = mat(d_model, W), vec(W)
    blocks, packed = [], [w_in.T.reshape(-1), b_in]
    for _ in range(2):
        p = {"ln1_g": vec(W, 1.0, 0.1), "ln1_b": vec(W), "w_qkv": mat(W, 3 * W), "b_qkv": vec(3 * W),
             "w_o": mat(W, W), "b_o": vec(W), "ln2_g": vec(W, 1.0, 0.1), "ln2_b": vec(W),
             "w_1": mat(W, F), "b_1": vec(F), "w_2": mat(F, W), "b_2": vec(W)}
        for key in ("ln1_g", "ln1_b", "w_qkv", "b_qkv", "w_o", "b_o", "ln2_g", "ln2_b", "w_1", "b_1", "w_2", "b_2"):
            t = p[key]
            packed.append(t.T.reshape(-1) if t.dim() == 2 else t)
        blocks.append({k: v.double().numpy() for k, v in p.items()})
    w_head = _bf16(rng.standard_normal((L, W, 5)) / np.sqrt(W))
    b_head = vec(L * 5, 0.0, 0.1).reshape(L, 5)
    packed += [w_head.reshape(-1), b_head.reshape(-1)]
    ow = {"w_in": w_in.double().numpy(), "b_in": b_in.double().numpy(), "blocks": blocks,
          "w_head": w_head.double().numpy(), "b_head": b_head.double().numpy()}
    return ow, torch.cat([t.reshape(-1) for t in packed]).contiguous()


@pytest.mark.parametrize("T,L", [(100, 48), (1000, 48), (3000, 48), (1, 64), (300, 7)])
def test_selector_matches_oracle(T, L):
    d_model = 512
    say(f"case selector T={T} L={L}")
    ow, packed = _weights(1500 + T, d_model, L)
    assert packed.numel() == kvk.selector_weight_elems(d_model, L)
    rng = np.random.default_rng(1600 + T)
    emb = _bf16(rng.standard_normal((T, d_model)))
    logits = torch.empty((L, 5), dtype=torch.float32, device=DEV)
    actions = torch.empty(L, dtype=torch.int32, device=DEV)
    ws = torch.empty(kvk.selector_workspace_bytes(d_model, L, T), dtype=torch.uint8, device=DEV)
    kvk.selector_forward(d_model, L, packed.to(DEV), emb.to(DEV), actions, ws, logits=logits)
    torch.cuda.synchronize()
    got = logits.cpu().numpy().astype(np.float64)
    ref = S.logits(emb.double().numpy(), ow)
    assert np.isneginf(got[0, 0]) and np.isneginf(ref[0, 0])
    fin = np.isfinite(ref)
    top = np.abs(ref[fin]).max()
    err = np.abs(got[fin] - ref[fin]).max() / top
    say(f"  max|diff| / max|logit| = {err:.2e}")
    assert err <= TOL_SEL
    act = actions.cpu().numpy()
    assert np.array_equal(act, np.argmax(got, axis=1)), "actions are not the argmax of the kernel's logits"
    assert act[0] != 0, "layer 0 inherits"
    oact = np.argmax(ref, axis=1)
    srt = np.sort(ref, axis=1)
    clear = (srt[:, -1] - srt[:, -2]) > 2 * TOL_SEL * top
    assert np.array_equal(act[clear], oact[clear])


def _run(d_model, L, packed, emb, logits=None):
    T = emb.shape[0]
    actions = torch.empty(L, dtype=torch.int32, device=DEV)
    if logits is None:
        logits = torch.empty((L, 5), dtype=torch.float32, device=DEV)
    ws = torch.empty(kvk.selector_workspace_bytes(d_model, L, T), dtype=torch.uint8, device=DEV)
    kvk.selector_forward(d_model, L, packed, emb, actions, ws, logits=logits)
    torch.cuda.synchronize()
    return logits.cpu().numpy().astype(np.float64), actions.cpu().numpy()


def test_selector_14b_width_8k_matches_oracle():
    """The 14B embedding width (5120) and 48 layers at 8192 prompt tokens, the launch
    shape the benchmark times (the input map and the second feed-forward matrix split
    4 ways over K): logits against the oracle, actions the argmax."""
    d_model, L, T = 5120, 48, 8192
    say(f"case selector d_model {d_model} T={T}")
    ow, packed = _weights(1700, d_model, L)
    emb = _bf16(np.random.default_rng(1701).standard_normal((T, d_model)))
    got, act = _run(d_model, L, packed.to(DEV), emb.to(DEV))
    ref = S.logits(emb.double().numpy(), ow)
    fin = np.isfinite(ref)
    top = np.abs(ref[fin]).max()
    err = np.abs(got[fin] - ref[fin]).max() / top
    say(f"  max|diff| / max|logit| = {err:.2e}")
    assert err <= TOL_SEL
    assert np.array_equal(act, np.argmax(got, axis=1)) and act[0] != 0


def test_selector_32k_properties():
    """32768 prompt tokens at the 14B width (the oracle's attention would take minutes):
    finite logits whose argmax are the actions, two calls bit-identical (the split-K
    partials are summed in a fixed order), and the logits unchanged within the parity
    tolerance when the prompt's tokens are permuted (the feature is a time average of
    a bidirectional model without positions)."""
    d_model, L, T = 5120, 48, 32768
    say(f"case selector d_model {d_model} T={T} properties")
    _, packed = _weights(1800, d_model, L)
    packed = packed.to(DEV)
    g = torch.Generator(device=DEV)
    g.manual_seed(1801)
    emb = torch.randn((T, d_model), generator=g, device=DEV).to(torch.bfloat16)
    z1, a1 = _run(d_model, L, packed, emb)
    z2, a2 = _run(d_model, L, packed, emb)
    assert np.array_equal(z1, z2) and np.array_equal(a1, a2), "not deterministic"
    fin = np.isfinite(z1)
    assert fin.sum() == L * 5 - 1 and np.isneginf(z1[0, 0])
    assert np.array_equal(a1, np.argmax(z1, axis=1)) and a1[0] != 0
    perm = torch.randperm(T, generator=g, device=DEV)
    zp, _ = _run(d_model, L, packed, emb[perm].contiguous())
    top = np.abs(z1[fin]).max()
    err = np.abs(zp[fin] - z1[fin]).max() / top
    say(f"  permuted: max|diff| / max|logit| = {err:.2e}")
    assert err <= TOL_SEL
