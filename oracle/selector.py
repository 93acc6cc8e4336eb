"""The selector's forward pass: prompt -> per-layer cache configuration (oracle).

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

§2.3: a selector maps the T input tokens to one action per layer.  A small shared
sequence model ingests the backbone's own token embeddings through two bidirectional
transformer blocks; its outputs are averaged over time; one linear head per layer
maps that feature to logits over the action space; evaluation takes the plain
argmax, with the depth action's logit forced to -inf where depth is not allowed
(always at the first layer).  The evaluated selectors hold 2.6-3.7M parameters
(§2.3); the paper reports about 3 ms per prompt on an H100 from 2k to 32k tokens
(Fig. prefill).

Readings where the paper is silent (the library follows the same):
  * width 256, 4 heads of 64, feed-forward 1024 with tanh-approximated GELU,
    pre-normalisation (LayerNorm, eps 1e-5, with gain and bias) and residuals;
  * the embeddings (width d_model) enter through a linear map to 256 with bias;
    no positional encoding (the feature is a time average);
  * attention is softmax(q k / 8) over every position (bidirectional);
  * GQA action space: index 0 = inherit (depth), 1..4 = bf16, int8, int4, int2;
  * every weight is an input (synthetic here; the paper's are trained).
Everything is fp64 from the given values (bf16 weights and embeddings).

Pins (tests/test_oracle_selector.py): a block with zero weights is the identity
(the residual path); attention over identical positions returns their value; the
pooled feature is invariant to permuting the tokens; explicit loops on a tiny
input for attention and LayerNorm; layer 0 never inherits; the argmax follows
planted head biases.
"""
import numpy as np

WIDTH = 256
HEADS = 4
FFN = 1024
N_ACTIONS = 5
ACTIONS = [(1, 16), (0, 16), (0, 8), (0, 4), (0, 2)]  # (inherit, bits) by action index


def layer_norm(x, g, b, eps=1e-5):
    x = np.asarray(x, np.float64)
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps) * g + b


def gelu(x):
    return 0.5 * x * (1.0 + np.tanh(np.sqrt(2.0 / np.pi) * (x + 0.044715 * x ** 3)))


def attention(x, w_qkv, b_qkv, w_o, b_o):
    """Bidirectional multi-head attention over x [T, 256]."""
    T = x.shape[0]
    qkv = x @ w_qkv + b_qkv  # [T, 768]
    q, k, v = qkv[:, :WIDTH], qkv[:, WIDTH:2 * WIDTH], qkv[:, 2 * WIDTH:]
    dh = WIDTH // HEADS
    out = np.zeros((T, WIDTH))
    for h in range(HEADS):
        sl = slice(h * dh, (h + 1) * dh)
        s = q[:, sl] @ k[:, sl].T / np.sqrt(dh)
        s = s - s.max(axis=1, keepdims=True)
        p = np.exp(s)
        p /= p.sum(axis=1, keepdims=True)
        out[:, sl] = p @ v[:, sl]
    return out @ w_o + b_o


def block(x, p):
    """Pre-normalised transformer block; p holds ln1_g, ln1_b, w_qkv, b_qkv, w_o, b_o,
    ln2_g, ln2_b, w_1, b_1, w_2, b_2 (weights [in, out])."""
    h = x + attention(layer_norm(x, p["ln1_g"], p["ln1_b"]), p["w_qkv"], p["b_qkv"], p["w_o"], p["b_o"])
    return h + gelu(layer_norm(h, p["ln2_g"], p["ln2_b"]) @ p["w_1"] + p["b_1"]) @ p["w_2"] + p["b_2"]


def feature(emb, w):
    """emb [T, d_model] -> the time-averaged feature [256]."""
    x = np.asarray(emb, np.float64) @ w["w_in"] + w["b_in"]
    for p in w["blocks"]:
        x = block(x, p)
    return x.mean(axis=0)


def logits(emb, w):
    """[n_layers, 5] logits; the depth action of layer 0 at -inf."""
    f = feature(emb, w)
    z = np.einsum("c,lca->la", f, np.asarray(w["w_head"], np.float64)) + w["b_head"]
    z[0, 0] = -np.inf
    return z


def plan(emb, w):
    """Per-layer (inherit, bits) by argmax (lowest index on ties)."""
    return [ACTIONS[int(np.argmax(r))] for r in logits(emb, w)]
