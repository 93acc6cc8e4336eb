"""Plans, anchors, cost model and storage accounting (oracle).

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

Follows §2.1 (anchors: a layer either owns a cache or inherits from the nearest
anchor before it), §2.2 eq. (1) (cost per action), eq. (2) (compression ratio
against the bf16 GQA cache, metadata excluded as §3 states), eq. (3) (action
space), App. C.1 eq. (5) (range of ratios) and App. C.3 (storage cost with
quantisation metadata).

Pins: eq. (5) against every row of the App. C.1 ranges table; the storage
accounting against every row of the App. C.3 table; the §1 cache size of
Qwen2.5-14B (192 KiB/token, 48 GiB for 32 x 8k); the §4 on-device factors.
"""
from dataclasses import dataclass
from typing import List, Optional, Sequence

BITS = (2, 4, 8, 16)
GROUP = 32
GQA, MLA = 0, 1
KIVI32, SYMROW, GROUP64 = 0, 1, 2


@dataclass(frozen=True)
class Action:
    inherit: bool = False
    bits: int = 16
    rank: int = 0


@dataclass(frozen=True)
class Dims:
    kind: int
    n_layers: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    latent_dim: int = 0
    rope_dim: int = 0
    nope_dim: int = 0
    v_dim: int = 0
    qscheme: int = KIVI32
    batch: int = 1
    max_tokens: int = 1
    keep_tokens: int = 0

    @property
    def group_size(self) -> int:
        """Query heads per KV head (GQA)."""
        return self.n_q_heads // self.n_kv_heads

    @property
    def kv_width(self) -> int:
        """Cached scalars per token per layer of the GQA model, 2 n_kv d_h (§2.1)."""
        return 2 * self.n_kv_heads * self.head_dim

    @property
    def stored_cap(self) -> int:
        return self.keep_tokens if self.keep_tokens > 0 else self.max_tokens


def rank_set(latent_dim: int) -> List[int]:
    """eq. (3): D = {r/8, r/4, r/2, r}."""
    return [latent_dim // 8, latent_dim // 4, latent_dim // 2, latent_dim]


def validate(dims: Dims, plan: Sequence[Action]) -> Optional[str]:
    """Return None if the plan is valid, else a reason.

    Layer 1 of the paper (index 0 here) must own a cache (§2.2, and §2.3 forces
    its inherit logit to -inf); every other action must lie in eq. (3)'s set.
    """
    if len(plan) != dims.n_layers:
        return "plan length != n_layers"
    if plan[0].inherit:
        return "layer 0 must own a cache"
    if dims.qscheme == GROUP64 and (dims.kind != GQA or dims.head_dim % 64):
        return "GROUP64 needs a GQA table with head_dim a multiple of 64"
    for a in plan:
        if a.inherit:
            continue
        if a.bits not in BITS:
            return "bits not in {2,4,8,16}"
        if dims.kind == GQA:
            if a.rank not in (0, dims.kv_width):
                return "GQA has no rank axis"
        else:
            if a.rank not in rank_set(dims.latent_dim):
                return "rank not in {r/8, r/4, r/2, r}"
    return None


def anchor_of(plan: Sequence[Action]) -> List[int]:
    """§2.1: each layer reads its own cache if it produces one, else the nearest
    producing layer before it."""
    out, last = [], -1
    for l, a in enumerate(plan):
        if not a.inherit:
            last = l
        out.append(last)
    return out


def cost_bits(dims: Dims, a: Action) -> int:
    """eq. (1): 0 for inherit, (d + d_R) b otherwise; for GQA d = 2 n_kv d_h, d_R = 0."""
    if a.inherit:
        return 0
    if dims.kind == GQA:
        return dims.kv_width * a.bits
    return (a.rank + dims.rope_dim) * a.bits


def c0_bits(dims: Dims) -> int:
    """eq. (2): C0 = L * 2 n_kv d_h * 16."""
    return dims.n_layers * dims.kv_width * 16


def rho(dims: Dims, plan: Sequence[Action]) -> float:
    """eq. (2): C0 / sum_l c(a_l)."""
    return c0_bits(dims) / sum(cost_bits(dims, a) for a in plan)


def rho_range(n_layers: int, kv_width: int, latent_dim: int, rope_dim: int, mla: bool,
              precision: bool, rank: bool, depth: bool):
    """App. C.1 eq. (5).  The extrema run over cache-producing actions; with depth
    the maximum puts the cheapest action on a single anchor."""
    bits = BITS if precision else (16,)
    if mla:
        widths = rank_set(latent_dim) if rank else [latent_dim]
        costs = [(d + rope_dim) * b for d in widths for b in bits]
    else:
        costs = [kv_width * b for b in bits]
    c0 = n_layers * kv_width * 16
    rmin = c0 / (n_layers * max(costs))
    rmax = c0 / min(costs) if depth else c0 / (n_layers * min(costs))
    return rmin, rmax


def n_actions(mla: bool, precision: bool, rank: bool, depth: bool) -> int:
    """eq. (3): |A| = |D| |B| (+1 with depth)."""
    nb = 4 if precision else 1
    nd = 4 if (mla and rank) else 1
    return nd * nb + (1 if depth else 0)


def realized_bits(qscheme: int, bits: int, group: int, window: int, context: int,
                  row: int = 128) -> float:
    """App. C.3 storage accounting: bits per cached element including metadata and
    a bf16 residual window.  The grouped scheme stores a 16-bit scale and a 16-bit
    zero per `group` elements; the paper's own scheme one bf16 scale per `row`."""
    if qscheme == SYMROW:
        per = bits + 16.0 / row
    else:
        per = bits + 32.0 / group
    return (per * (context - window) + 16.0 * window) / context


# ---------------------------------------------------------------------------
# Arena geometry (the layout rules of include/kvk.h, restated)
# ---------------------------------------------------------------------------

def round256(n: int) -> int:
    return (n + 255) // 256 * 256


def stored_width(dims: Dims, rank: int) -> int:
    """MLA: scalars stored per token by a layer that keeps width d = rank, namely
    the first d latent coordinates and the positional key, d + d_R (§2.1, App. C.2)."""
    return rank + dims.rope_dim


def block_bytes(dims: Dims, bits: int, rank: int = 0) -> int:
    """Bytes of one 32-token block of one stream.  GQA: a (b, KV head) stream
    holding K and V of width D; MLA: a (b) stream holding d + d_R scalars per
    token."""
    if dims.kind == MLA:
        W = stored_width(dims, rank)
        if bits == 16:
            return 64 * W
        if dims.qscheme == KIVI32:
            return 4 * W * (bits + 1)
        return 4 * W * bits + 128
    D = dims.head_dim
    if bits == 16:
        return 128 * D
    if dims.qscheme == KIVI32:
        return 8 * D * (bits + 1)
    if dims.qscheme == GROUP64:
        return 8 * D * bits + 4 * D  # codes + fp16 (scale, zero) per 64 channels of a token, K and V
    return 8 * D * bits + 128


def tail_bytes(dims: Dims, rank: int = 0) -> int:
    if dims.kind == MLA:
        return 64 * stored_width(dims, rank)
    return 128 * dims.head_dim


def stream_bytes(dims: Dims, bits: int, rank: int = 0) -> int:
    nb = dims.stored_cap // GROUP
    return round256(nb * block_bytes(dims, bits, rank) + tail_bytes(dims, rank))


def streams_per_layer(dims: Dims) -> int:
    """GQA: one stream per (sequence, KV head); MLA: one per sequence (the latent
    is shared by every head, §2.1)."""
    return dims.batch * (dims.n_kv_heads if dims.kind == GQA else 1)


def layer_bytes(dims: Dims, bits: int, rank: int = 0) -> int:
    return streams_per_layer(dims) * stream_bytes(dims, bits, rank)


def arena_offsets(dims: Dims, plan: Sequence[Action]):
    """Byte offset of each anchor's region (anchors in layer order, from 0), -1 for
    inheritors, and the arena size (the regions' total)."""
    offs, cur = [], 0
    for a in plan:
        if a.inherit:
            offs.append(-1)
        else:
            offs.append(cur)
            cur += round256(layer_bytes(dims, a.bits, a.rank))
    return offs, cur


def read_bytes_stream(dims: Dims, bits: int, n_stored: int, rank: int = 0) -> int:
    """Algorithmic bytes a decode step reads from one stream holding n_stored
    tokens: the full blocks plus the bf16 values of the tail tokens."""
    nb, nt = divmod(n_stored, GROUP)
    per_tail_token = 2 * stored_width(dims, rank) if dims.kind == MLA else 4 * dims.head_dim
    return nb * block_bytes(dims, bits, rank) + nt * per_tail_token


def read_bytes(dims: Dims, plan: Sequence[Action], l0: int, l1: int, n_stored: int) -> int:
    """Algorithmic bytes of one decode step over [l0, l1): every distinct anchor
    read by the range, read once."""
    anc = anchor_of(plan)
    used = sorted(set(anc[l] for l in range(l0, l1)))
    per = streams_per_layer(dims)
    return sum(per * read_bytes_stream(dims, plan[a].bits, n_stored, plan[a].rank) for a in used)


def bf16_full_bytes(dims: Dims) -> int:
    """Uncompressed bf16 GQA cache of all L layers at the full prefill length."""
    return dims.n_layers * dims.batch * dims.max_tokens * dims.kv_width * 2


# ---------------------------------------------------------------------------
# Per-sequence plans in one batch (§2.3: the selector maps each input sequence to
# its own plan; eq. (4) takes the realized cost per sequence i).
# ---------------------------------------------------------------------------

def sequence_dims(dims: Dims) -> Dims:
    """The dims of one sequence of a batch (batch 1, everything else equal)."""
    from dataclasses import replace
    return replace(dims, batch=1)


def batched_arena_bases(dims: Dims, plans) -> tuple:
    """A batch whose sequences carry their own plans stores, for sequence b, the
    arena of a one-sequence table with plans[b] at base_b; the bases are the
    running sums of those arenas, each rounded up to 256 bytes.  Returns (bases,
    total)."""
    sd = sequence_dims(dims)
    bases, cur = [], 0
    for pl in plans:
        bases.append(cur)
        cur += round256(arena_offsets(sd, pl)[1])
    return bases, cur


def read_bytes_batched(dims: Dims, plans, l0: int, l1: int, n_stored: int) -> int:
    """Algorithmic bytes of a decode step over [l0, l1) of a per-sequence batch: each
    sequence reads its own distinct anchors once."""
    sd = sequence_dims(dims)
    return sum(read_bytes(sd, pl, l0, l1, n_stored) for pl in plans)
