"""Reference oracle for the KV-Kaizen compressed-cache decode path.

TEST INFRASTRUCTURE ONLY.  This package is a plain, slow, CPU implementation of
what the library computes, written from the paper (arXiv 2609.37988) and from the
storage layout documented in include/kvk.h.  Only tests/, the smoke check in
__graft_entry__.py and the CPU-baseline leg of bench.py may import it.  The
product path (paper_2609_37988_amd) never imports, links or executes anything in
here, and this package imports nothing from the product path: the two share no
code.

Arithmetic conventions:
  * Where the library works in IEEE fp32 (the quantiser chain), the oracle does
    the same operation in numpy float32, whose + - * / are correctly rounded;
    this equals "compute in fp64, then round to fp32" for a single operation.
  * Conversions to fp16 use numpy's round-to-nearest-even; conversions to bf16
    are written out below (round-to-nearest-even on the fp32 bit pattern).
  * Attention is computed in fp64 from the dequantised cache.

Modules:
  plan      — plan validation, anchors, eq. (1), (2), (5), storage accounting
  quant     — App. C.3 quantisers (KIVI32 grouped asymmetric, SYMROW symmetric)
  layout    — the arena byte layout (pack / unpack)
  attention — softmax attention, split/LSE merge, depth, eviction
  cache     — compress a layer to arena bytes and decode a step from them
  mla       — the rank axis: MLA latent caches, their storage and attention
  snapkv    — query-aware token selection at prefill (the eviction composed with)
  selector  — the selector forward pass (prompt embeddings -> per-layer plan)

Parity status per function is stated in each module's docstring.
"""
from . import plan, quant, layout, attention, cache, mla, snapkv, selector  # noqa: F401
