"""The selector's forward pass: prompt -> per-layer cache configuration (oracle).

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

What it computes (§2.3 and App. B "Selector architecture"):
  * the backbone's token embeddings [T, H] are mapped linearly to width 256;
  * two bidirectional transformer blocks follow; each has
      - an attention sublayer of 4 heads of width 64, with rotary position
        embeddings applied to the queries and the keys,
      - a SwiGLU feed-forward sublayer of inner width 1024,
      - an RMSNorm before each sublayer and a residual connection around each;
  * a final RMSNorm follows the second block;
  * the output is averaged over the T tokens into z (256 wide);
  * optionally the budget conditioning of App. B (FiLM) maps z to z * (1 + gamma) + beta
    (the MLP producing gamma, beta from the target ratio is outside this function);
  * each of the L layers has its own linear head (with bias) giving |A| logits;
  * the depth action's logit is -inf at the first layer and at every layer when
    depth is not in the selector's action space (§2.3); evaluation takes the argmax.

Readings where the paper is silent (the library follows the same):
  * RoPE: the position of token t is t (0 .. T-1); base 10000 (RoFormer's);
    rotate-half pairing, channel i with channel i + 32 of a 64-wide head, at
    frequency base^(-2i/64), i = 0 .. 31 (the convention of the Qwen2.5 family the
    selector serves); applied to q and k after their projections, v untouched;
  * attention scale 1/sqrt(64); softmax over every position (bidirectional);
  * RMSNorm: x / sqrt(mean(x^2) + 1e-6) * g, a gain and no bias;
  * SwiGLU: W_down (SiLU(W_gate n) * W_up n), SiLU(x) = x / (1 + e^-x);
  * no bias in the trunk's linear maps (input map, q, k, v, o, gate, up, down);
    the heads carry biases (App. B initialises them);
  * action index order: 0 = inherit; 1 + 4 j + k = produce with kept width
    r / 2^j and b = 16 / 2^k bits (j, k = 0 .. 3), so index 1 is the least
    compressed action; a GQA selector (precision and depth) uses the first five.
Weight matrices are [out][in].  Everything is fp64 from the given values.

Pins (tests/test_oracle_selector.py): the parameter count of this weight set
matches every count App. B prints (2.61 - 3.69M over six backbones, heads
122k - 280k); RMSNorm and SwiGLU against explicit loops and torch's own
rms_norm / silu; RoPE against complex rotation, norm preservation, the identity
at position 0; attention with all positions at 0 against torch's
scaled_dot_product_attention; shifting every position by a constant leaves the
attention unchanged; identical tokens return their value; a block with zero
weights is the identity; the feature depends on token order; layer 0 never
inherits; a masked depth action is never chosen; planted biases steer the argmax;
FiLM with zero scale and shift is the identity.
"""
import numpy as np

WIDTH = 256
HEADS = 4
HEAD_DIM = 64
FFN = 1024
RMS_EPS = 1e-6
ROPE_BASE = 10000.0

# Composed action space (eq. (3)): index -> (inherit, rank divisor 2^j, bits)
ACTIONS = [(1, 1, 16)] + [(0, 1 << j, 16 >> k) for j in range(4) for k in range(4)]
N_ACTIONS_FULL = len(ACTIONS)        # 17
N_ACTIONS_GQA = 5                    # inherit, 16, 8, 4, 2 bits at full width
BLOCK_KEYS = ("g_attn", "w_q", "w_k", "w_v", "w_o", "g_ffn", "w_gate", "w_up", "w_down")


def rms_norm(x, g, eps=RMS_EPS):
    x = np.asarray(x, np.float64)
    return x / np.sqrt((x * x).mean(axis=-1, keepdims=True) + eps) * np.asarray(g, np.float64)


def silu(x):
    return x / (1.0 + np.exp(-x))


def rope_angles(positions):
    """[T, 32] angles m * theta_i."""
    i = np.arange(HEAD_DIM // 2, dtype=np.float64)
    theta = ROPE_BASE ** (-2.0 * i / HEAD_DIM)
    return np.asarray(positions, np.float64)[:, None] * theta[None, :]


def rope(x, positions):
    """Rotate-half RoPE of x [T, 64]: channels (i, i + 32) rotated by m * theta_i."""
    a = rope_angles(positions)
    c, s = np.cos(a), np.sin(a)
    x1, x2 = x[:, :HEAD_DIM // 2], x[:, HEAD_DIM // 2:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=1)


def attention(n, p, positions):
    """Bidirectional multi-head attention over the normalised rows n [T, 256]."""
    q, k, v = n @ p["w_q"].T, n @ p["w_k"].T, n @ p["w_v"].T
    out = np.zeros_like(q)
    for h in range(HEADS):
        sl = slice(h * HEAD_DIM, (h + 1) * HEAD_DIM)
        qh, kh = rope(q[:, sl], positions), rope(k[:, sl], positions)
        s = qh @ kh.T / np.sqrt(HEAD_DIM)
        s = s - s.max(axis=1, keepdims=True)
        e = np.exp(s)
        out[:, sl] = (e / e.sum(axis=1, keepdims=True)) @ v[:, sl]
    return out @ p["w_o"].T


def swiglu(n, p):
    return (silu(n @ p["w_gate"].T) * (n @ p["w_up"].T)) @ p["w_down"].T


def block(x, p, positions):
    """Pre-norm block: x + Attn(RMSNorm(x)), then + SwiGLU(RMSNorm(.))."""
    h = x + attention(rms_norm(x, p["g_attn"]), p, positions)
    return h + swiglu(rms_norm(h, p["g_ffn"]), p)


def feature(emb, w, film=None, positions=None):
    """emb [T, H] -> z [256]; film = (gamma, beta) or None."""
    emb = np.asarray(emb, np.float64)
    pos = np.arange(emb.shape[0]) if positions is None else positions
    x = emb @ np.asarray(w["w_in"], np.float64).T
    for p in w["blocks"]:
        x = block(x, p, pos)
    z = rms_norm(x, w["g_final"]).mean(axis=0)
    if film is not None:
        gamma, beta = film
        z = z * (1.0 + np.asarray(gamma, np.float64)) + np.asarray(beta, np.float64)
    return z


def logits(emb, w, depth=True, film=None):
    """[L, |A|] logits; the depth action (index 0) -inf at layer 0, or everywhere
    when depth is not in the action space."""
    z = feature(emb, w, film)
    out = np.einsum("lac,c->la", np.asarray(w["w_head"], np.float64), z) + np.asarray(w["b_head"], np.float64)
    out[0, 0] = -np.inf
    if not depth:
        out[:, 0] = -np.inf
    return out


def actions(emb, w, depth=True, film=None):
    """Per-layer action index by argmax (the lowest index on ties)."""
    return [int(np.argmax(r)) for r in logits(emb, w, depth, film)]


def action_config(index):
    """(inherit, rank divisor, bits) of a composed-space action index."""
    return ACTIONS[index]


def weight_shapes(d_model, n_layers, n_actions=N_ACTIONS_FULL):
    """Shapes of every weight the functions above consume ([out][in] matrices)."""
    blk = {"g_attn": (WIDTH,), "w_q": (WIDTH, WIDTH), "w_k": (WIDTH, WIDTH), "w_v": (WIDTH, WIDTH),
           "w_o": (WIDTH, WIDTH), "g_ffn": (WIDTH,), "w_gate": (FFN, WIDTH), "w_up": (FFN, WIDTH),
           "w_down": (WIDTH, FFN)}
    return {"w_in": (WIDTH, d_model), "blocks": [dict(blk), dict(blk)], "g_final": (WIDTH,),
            "w_head": (n_layers, n_actions, WIDTH), "b_head": (n_layers, n_actions)}
