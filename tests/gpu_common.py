"""Helpers shared by the GPU tests: build a table, compress, decode, and run the
oracle on the same seeded inputs."""
import sys

import numpy as np
import torch

from oracle import attention as OA
from oracle import cache as OC
from oracle import plan as OP
from paper_2609_37988_amd import kvk

DEV = "cuda:0"


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


class Case:
    """A table plus its device buffers."""

    def __init__(self, n_layers, Hq, Hkv, D, B, max_tokens, plan, qscheme=kvk.KIVI32, keep=0):
        self.dims = kvk.make_dims(kvk.GQA, n_layers, Hq, Hkv, D, qscheme=qscheme, batch=B,
                                  max_tokens=max_tokens, keep_tokens=keep)
        self.plan = kvk.make_plan(plan)
        self.table = kvk.layer_table(self.dims, self.plan)
        self.info = kvk.table_query(self.table)
        self.arena = torch.zeros(max(self.info.arena_bytes, 256), dtype=torch.uint8, device=DEV)
        self.odims = OP.Dims(OP.GQA, n_layers, Hq, Hkv, D, qscheme=qscheme, batch=B,
                             max_tokens=max_tokens, keep_tokens=keep)
        self.oplan = [OP.Action(bool(a.inherit), a.bits) for a in self.plan]

    def compress(self, layer, k, v, n_tokens, keep=None):
        kvk.compress_layer(self.table, layer, k.contiguous(), v.contiguous(), n_tokens,
                           None if keep is None else keep.contiguous(), self.arena)

    def decode(self, q, n_stored, scale, l0=0, l1=None):
        l1 = self.dims.n_layers if l1 is None else l1
        d = self.dims
        # NaN-filled output and workspace: a read of anything the kernels did not write shows
        out = torch.full((l1 - l0, d.batch, d.n_q_heads, d.head_dim), float("nan"), dtype=torch.float32, device=DEV)
        ws = torch.full((max(kvk.workspace_bytes(self.table, l0, l1), 256),), 0xFF, dtype=torch.uint8, device=DEV)
        kvk.decode_attention(self.table, l0, l1, q.contiguous(), n_stored, scale, self.arena, out, ws)
        return out

    def dequant(self, layer, n_stored):
        d = self.dims
        shape = (d.batch, d.n_kv_heads, max(n_stored, 1), d.head_dim)
        k = torch.empty(shape, dtype=torch.float32, device=DEV)
        v = torch.empty(shape, dtype=torch.float32, device=DEV)
        kvk.debug_dequantize(self.table, layer, n_stored, self.arena, k, v)
        return k[:, :, :n_stored], v[:, :, :n_stored]

    def stream_bytes_host(self, layer, b, h):
        """The meaningful bytes (full blocks + tail block) of one stream, from the GPU arena."""
        a = self.info.anchor_of[layer]
        sb = self.info.stream_bytes[a]
        off = self.info.layer_offset[a] + (b * self.dims.n_kv_heads + h) * sb
        return self.arena[off:off + sb].cpu().numpy()


def meaningful(odims, bits, stream: np.ndarray, n_stored: int) -> np.ndarray:
    """Concatenate the full blocks and the tail block of a stream's bytes."""
    blocks, tail = OC.layout.split_stream(odims, bits, stream, n_stored)
    return np.concatenate([blocks.reshape(-1), tail])


def oracle_stream(odims, bits, k: np.ndarray, v: np.ndarray, keep=None):
    """Oracle bytes of one stream from its input rows (after eviction if keep)."""
    if keep is not None:
        k, v = OC.gather_kept(k, keep), OC.gather_kept(v, keep)
    return OC.compress_stream(odims, bits, k, v)


def oracle_rows(odims, bits, stream, n_stored, q_rows: np.ndarray, scale: float):
    """Attention of q_rows [R, D] over one oracle stream."""
    K, V = OC.dequant_stream(odims, bits, stream, n_stored)
    return OA.softmax_attention(q_rows, K, V, scale)


def rel_err(got: np.ndarray, ref: np.ndarray) -> float:
    m = np.abs(ref).max()
    return float(np.abs(got - ref).max() / (m if m > 0 else 1.0))


TOL = 2e-3  # max|diff| <= 2e-3 * max|out| (fp32 accumulation)
