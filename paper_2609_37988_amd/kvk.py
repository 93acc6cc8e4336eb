"""Python binding of libkvk (ctypes): argument marshalling only.

Every function here calls the C ABI of include/kvk.h with the same name minus
the `kvk_` prefix.  Device buffers are torch tensors on the current HIP device;
the binding passes their data pointers and the current stream.  All compute runs
in the library's HIP kernels.  If libkvk.so has not been built, loading fails
with an error (there is no fallback path).
"""
import ctypes
import os
from dataclasses import dataclass
from typing import List, Optional, Sequence

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libkvk.so")
MAX_LAYERS = 64

OK, ERR_INVALID, ERR_UNSUPPORTED, ERR_DEVICE, ERR_BUFFER = 0, -1, -2, -3, -4
GQA, MLA = 0, 1
KIVI32, SYMROW, GROUP64 = 0, 1, 2
BF16, F32 = 0, 1


class Dims(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "kind", "n_layers", "n_q_heads", "n_kv_heads", "head_dim", "latent_dim", "rope_dim",
        "nope_dim", "v_dim", "qscheme", "batch", "max_tokens", "keep_tokens")]


class Action(ctypes.Structure):
    _fields_ = [("inherit", ctypes.c_int32), ("bits", ctypes.c_int32), ("rank", ctypes.c_int32)]


class TableInfo(ctypes.Structure):
    _fields_ = [
        ("arena_bytes", ctypes.c_int64), ("workspace_bytes", ctypes.c_int64),
        ("n_anchors", ctypes.c_int32), ("stored_tokens_cap", ctypes.c_int32),
        ("cost_bits_per_token", ctypes.c_double), ("c0_bits_per_token", ctypes.c_double),
        ("rho", ctypes.c_double), ("rho_realized", ctypes.c_double),
        ("anchor_of", ctypes.c_int32 * MAX_LAYERS), ("layer_offset", ctypes.c_int64 * MAX_LAYERS),
        ("layer_bytes", ctypes.c_int64 * MAX_LAYERS), ("stream_bytes", ctypes.c_int64 * MAX_LAYERS),
        ("layer_cost_bits", ctypes.c_double * MAX_LAYERS),
        ("layer_bits_per_elt", ctypes.c_double * MAX_LAYERS),
    ]


class KvkError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"kvk status {status}: {msg}")
        self.status = status


_lib = None


def load() -> ctypes.CDLL:
    """Load libkvk.so (built in-tree by paper_2609_37988_amd.build)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: run `python -m paper_2609_37988_amd.build`")
        lib = ctypes.CDLL(LIB_PATH)
        P, I32, I64, F = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float
        sig = {
            "kvk_layer_table": (I32, [ctypes.POINTER(Dims), ctypes.POINTER(Action), ctypes.POINTER(P)]),
            "kvk_table_query": (I32, [P, ctypes.POINTER(TableInfo)]),
            "kvk_table_destroy": (None, [P]),
            "kvk_workspace_bytes": (I32, [P, I32, I32, ctypes.POINTER(ctypes.c_size_t)]),
            "kvk_layer_table_batched": (I32, [P, P, ctypes.POINTER(P)]),
            "kvk_table_sequence_query": (I32, [P, I32, P]),
            "kvk_compress_layer": (I32, [P, I32, P, P, I32, I32, P, P, P]),
            "kvk_compress_layer_project": (I32, [P, I32, P, P, I32, P, I32, P, P, P, P]),
            "kvk_mla_arrange_w_uk": (I32, [P, I32, I32, I32, I32, P, P]),
            "kvk_set_mla_weights": (I32, [P, P, P]),
            "kvk_snapkv_select_mla": (I32, [P, I32, P, P, P, P, I32, F, P, P, P, ctypes.c_size_t, P]),
            "kvk_append_token": (I32, [P, I32, I32, P, P, I32, I32, P, P]),
            "kvk_snapkv_workspace_bytes": (I32, [P, I32, ctypes.POINTER(ctypes.c_size_t)]),
            "kvk_selector_weight_elems": (I64, [I32, I32, I32]),
            "kvk_selector_workspace_bytes": (I32, [I32, I32, I32, ctypes.POINTER(ctypes.c_size_t)]),
            "kvk_selector_forward": (I32, [I32, I32, I32, I32, P, P, I32, P, P, P, P, ctypes.c_size_t, P]),
            "kvk_snapkv_select": (I32, [P, I32, P, P, I32, I32, F, P, P, P, ctypes.c_size_t, P]),
            "kvk_decode_attention": (I32, [P, I32, I32, P, I32, I32, F, P, P, P, P, P, ctypes.c_size_t, P]),
            "kvk_decode_splits": (I32, [P, I32, I32, P, I32, I32, F, P, P, P, P, ctypes.c_size_t, P]),
            "kvk_decode_attention_noalloc": (I32, [P, I32, I32, P, I32, I32, F, P, P, P, P, P]),
            "kvk_decode_setup": (I32, [P, I32, I32, P, ctypes.c_size_t, P]),
            "kvk_decode_merge": (I32, [P, I32, I32, P, I32, I32, F, P, P, P, P, ctypes.c_size_t, P, P]),
            "kvk_read_bytes": (I32, [P, I32, I32, I32, ctypes.POINTER(ctypes.c_int64)]),
            "kvk_debug_dequantize": (I32, [P, I32, I32, P, P, P, P]),
            "kvk_realized_bits": (ctypes.c_double, [I32, I32, I32, I64, I64]),
            "kvk_rho_range": (I32, [I32, I32, I32, I32, I32, I32, ctypes.POINTER(ctypes.c_double),
                                    ctypes.POINTER(ctypes.c_double)]),
            "kvk_last_error": (ctypes.c_char_p, []),
            "kvk_version": (ctypes.c_char_p, []),
        }
        for name, (res, args) in sig.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
    return _lib


def exported_symbols() -> List[str]:
    """Names of the C entry points the binding expects libkvk to export."""
    return ["kvk_layer_table", "kvk_layer_table_batched", "kvk_table_sequence_query", "kvk_table_query", "kvk_table_destroy", "kvk_workspace_bytes",
            "kvk_compress_layer", "kvk_compress_layer_project", "kvk_mla_arrange_w_uk", "kvk_set_mla_weights",
            "kvk_snapkv_select_mla",
            "kvk_append_token", "kvk_snapkv_workspace_bytes", "kvk_snapkv_select",
            "kvk_selector_weight_elems", "kvk_selector_workspace_bytes", "kvk_selector_forward",
            "kvk_decode_attention", "kvk_decode_splits", "kvk_decode_merge", "kvk_decode_attention_noalloc", "kvk_decode_setup",
            "kvk_read_bytes", "kvk_debug_dequantize",
            "kvk_realized_bits", "kvk_rho_range", "kvk_last_error", "kvk_version"]


def last_error() -> str:
    return load().kvk_last_error().decode()


def version() -> str:
    return load().kvk_version().decode()


def _check(st: int):
    if st != OK:
        raise KvkError(st, last_error())


def _ptr(t: Optional[torch.Tensor]):
    """The device address of a GPU tensor (every buffer the library's kernels read or
    write); a tensor in host memory is refused here, before the call."""
    if t is None:
        return None
    _need(t.is_cuda, "buffers must be GPU tensors (got a tensor on the host)")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


@dataclass
class Info:
    arena_bytes: int
    workspace_bytes: int
    n_anchors: int
    stored_tokens_cap: int
    cost_bits_per_token: float
    c0_bits_per_token: float
    rho: float
    rho_realized: float
    anchor_of: List[int]
    layer_offset: List[int]
    layer_bytes: List[int]
    stream_bytes: List[int]
    layer_cost_bits: List[float]
    layer_bits_per_elt: List[float]


class Table:
    """Owning handle of a kvk_table."""

    def __init__(self, handle: ctypes.c_void_p, dims: Dims, plan: Sequence[Action]):
        self._h = handle
        self.dims = dims
        self.plan = list(plan)
        self.mla_weights = None  # (w_uk, w_uv) attached by set_mla_weights
        self.plans = None        # per-sequence plans (layer_table_batched)

    @property
    def handle(self):
        return self._h

    def __del__(self):
        if getattr(self, "_h", None) and _lib is not None:
            _lib.kvk_table_destroy(self._h)
            self._h = None


def make_dims(kind=GQA, n_layers=1, n_q_heads=1, n_kv_heads=1, head_dim=128, latent_dim=0,
              rope_dim=0, nope_dim=0, v_dim=0, qscheme=KIVI32, batch=1, max_tokens=1,
              keep_tokens=0) -> Dims:
    return Dims(kind, n_layers, n_q_heads, n_kv_heads, head_dim, latent_dim, rope_dim, nope_dim,
                v_dim, qscheme, batch, max_tokens, keep_tokens)


def make_plan(entries: Sequence[tuple]) -> List[Action]:
    """entries: (inherit, bits) or (inherit, bits, rank) per layer."""
    out = []
    for e in entries:
        inherit, bits = int(e[0]), int(e[1])
        rank = int(e[2]) if len(e) > 2 else 0
        out.append(Action(inherit, bits, rank))
    return out


def layer_table(dims: Dims, plan: Sequence[Action]) -> Table:
    lib = load()
    arr = (Action * max(1, len(plan)))(*plan)
    h = ctypes.c_void_p()
    _check(lib.kvk_layer_table(ctypes.byref(dims), arr, ctypes.byref(h)))
    return Table(h, dims, plan)


def layer_table_batched(dims: Dims, plans: Sequence[Sequence[Action]]) -> Table:
    """A batch whose sequences carry their own plans: plans[b] is sequence b's plan."""
    _need(len(plans) == dims.batch and all(len(p) == dims.n_layers for p in plans),
          "plans must hold batch plans of n_layers actions")
    flat = [a for p in plans for a in p]
    arr = (Action * len(flat))(*flat)
    h = ctypes.c_void_p()
    _check(load().kvk_layer_table_batched(ctypes.byref(dims), arr, ctypes.byref(h)))
    t = Table(h, dims, plans[0])
    t.plans = [list(p) for p in plans]
    return t


def _info(inf, L) -> Info:
    return Info(inf.arena_bytes, inf.workspace_bytes, inf.n_anchors, inf.stored_tokens_cap,
                inf.cost_bits_per_token, inf.c0_bits_per_token, inf.rho, inf.rho_realized,
                list(inf.anchor_of[:L]), list(inf.layer_offset[:L]), list(inf.layer_bytes[:L]),
                list(inf.stream_bytes[:L]), list(inf.layer_cost_bits[:L]),
                list(inf.layer_bits_per_elt[:L]))


def table_sequence_query(t: Table, b: int) -> Info:
    """Per-sequence plans: sequence b's accounting, layer offsets absolute in the arena."""
    inf = TableInfo()
    _check(load().kvk_table_sequence_query(t.handle, b, ctypes.byref(inf)))
    return _info(inf, t.dims.n_layers)


def table_query(t: Table) -> Info:
    inf = TableInfo()
    _check(load().kvk_table_query(t.handle, ctypes.byref(inf)))
    L = t.dims.n_layers
    return Info(inf.arena_bytes, inf.workspace_bytes, inf.n_anchors, inf.stored_tokens_cap,
                inf.cost_bits_per_token, inf.c0_bits_per_token, inf.rho, inf.rho_realized,
                list(inf.anchor_of[:L]), list(inf.layer_offset[:L]), list(inf.layer_bytes[:L]),
                list(inf.stream_bytes[:L]), list(inf.layer_cost_bits[:L]),
                list(inf.layer_bits_per_elt[:L]))


def workspace_bytes(t: Table, layer_begin: int, layer_end: int) -> int:
    out = ctypes.c_size_t()
    _check(load().kvk_workspace_bytes(t.handle, layer_begin, layer_end, ctypes.byref(out)))
    return out.value


def _dtype_code(x: torch.Tensor) -> int:
    if x.dtype == torch.bfloat16:
        return BF16
    if x.dtype == torch.float32:
        return F32
    raise TypeError(f"unsupported dtype {x.dtype}")


def _nbytes(x) -> int:
    return x.numel() * x.element_size()


def _need(cond: bool, msg: str):
    if not cond:
        raise ValueError(msg)


def _q_width(d: Dims) -> int:
    """Per-head query width: d_h (GQA) or nope_dim + rope_dim (MLA)."""
    return d.nope_dim + d.rope_dim if d.kind == MLA else d.head_dim


def _out_width(d: Dims) -> int:
    """Per-head output width: d_h (GQA) or v_dim (MLA)."""
    return d.v_dim if d.kind == MLA else d.head_dim


def mla_weights_for_library(w_uk: torch.Tensor, stream=None) -> torch.Tensor:
    """W_UK [layers, Hq, nope, r] in the model's layout -> the latent-major layout the
    library reads ([layers, Hq, r, nope]), by kvk_mla_arrange_w_uk; done once at
    weight load."""
    _need(w_uk.dtype == torch.bfloat16 and w_uk.is_contiguous() and w_uk.dim() == 4,
          "w_uk must be contiguous bf16 [layers, Hq, nope, r]")
    L, H, nope, r = w_uk.shape
    out = torch.empty((L, H, r, nope), dtype=torch.bfloat16, device=w_uk.device)
    _check(load().kvk_mla_arrange_w_uk(_ptr(w_uk), L, H, nope, r, _ptr(out), _stream(stream)))
    return out


def set_mla_weights(t: Table, w_uk: Optional[torch.Tensor], w_uv: Optional[torch.Tensor]):
    """Attach all-layer weights to an MLA table (w_uk as mla_weights_for_library
    returns it, w_uv [layers, Hq, v, r]); None for both detaches.  The table keeps
    references so the tensors outlive their use."""
    d = t.dims
    if w_uk is not None or w_uv is not None:
        _need(w_uk is not None and w_uv is not None, "pass both weights or neither")
        _need(w_uk.dtype == torch.bfloat16 and w_uv.dtype == torch.bfloat16 and w_uk.is_contiguous()
              and w_uv.is_contiguous(), "w_uk / w_uv must be contiguous bf16")
        _need(w_uk.numel() == d.n_layers * d.n_q_heads * d.latent_dim * d.nope_dim and
              w_uv.numel() == d.n_layers * d.n_q_heads * d.v_dim * d.latent_dim,
              "attached weights cover every layer of the table")
    _check(load().kvk_set_mla_weights(t.handle, _ptr(w_uk), _ptr(w_uv)))
    t.mla_weights = None if w_uk is None else (w_uk, w_uv)


def _check_weights(t: Table, nl: int, w_uk, w_uv):
    d = t.dims
    if d.kind != MLA:
        _need(w_uk is None and w_uv is None, "w_uk / w_uv are for MLA tables only")
        return
    if w_uk is None and w_uv is None and t.mla_weights is not None:
        return  # the weights attached to the table
    _need(w_uk is not None and w_uv is not None, "an MLA table needs w_uk and w_uv")
    _need(w_uk.dtype == torch.bfloat16 and w_uv.dtype == torch.bfloat16 and w_uk.is_contiguous()
          and w_uv.is_contiguous(), "w_uk / w_uv must be contiguous bf16")
    _need(w_uk.numel() == nl * d.n_q_heads * d.latent_dim * d.nope_dim,
          "w_uk size must be layers*Hq*latent_dim*nope_dim (W_UK transposed, latent-major)")
    _need(w_uv.numel() == nl * d.n_q_heads * d.v_dim * d.latent_dim,
          "w_uv size must be layers*Hq*v_dim*latent_dim")


def compress_layer(t: Table, layer: int, k: torch.Tensor, v: torch.Tensor, n_tokens: int,
                   keep_idx: Optional[torch.Tensor], arena: torch.Tensor, stream=None):
    """GQA: k, v [B, Hkv, n_tokens, d_h].  MLA: k = latent [B, n_tokens, r], v = positional
    key [B, n_tokens, d_R].  Contiguous bf16/fp32 on the device."""
    d = t.dims
    _need(k.dtype == v.dtype and k.is_contiguous() and v.is_contiguous(),
          "k and v must be contiguous tensors of one dtype")
    if d.kind == MLA:
        _need(k.numel() == d.batch * n_tokens * d.latent_dim and v.numel() == d.batch * n_tokens * d.rope_dim,
              "latent size must be B*n_tokens*r and k^R size B*n_tokens*d_R")
        streams = d.batch
    else:
        _need(k.numel() == v.numel() == d.batch * d.n_kv_heads * n_tokens * d.head_dim,
              "k/v size must be B*Hkv*n_tokens*d_h")
        streams = d.batch * d.n_kv_heads
    if keep_idx is not None:
        _need(keep_idx.dtype == torch.int32 and keep_idx.is_contiguous(),
              "keep_idx must be a contiguous int32 tensor")
        _need(keep_idx.numel() == streams * d.keep_tokens, "keep_idx size must be streams*keep_tokens")
    _need(_nbytes(arena) >= table_query(t).arena_bytes, "arena smaller than arena_bytes")
    _check(load().kvk_compress_layer(t.handle, layer, _ptr(k), _ptr(v), _dtype_code(k), n_tokens,
                                     _ptr(keep_idx), _ptr(arena), _stream(stream)))


def compress_layer_project(t: Table, layer: int, x: torch.Tensor, w_dkv: torch.Tensor, k_rope: torch.Tensor,
                           n_tokens: int, keep_idx: Optional[torch.Tensor], arena: torch.Tensor,
                           latent_out: Optional[torch.Tensor] = None, stream=None):
    """MLA prefill write from hidden states: x [B, n_tokens, d_model] bf16, w_dkv
    [r, d_model] bf16, k_rope [B, n_tokens, 64] bf16; latent_out (optional) bf16
    [B, n_stored, d] receives the projected latent."""
    d = t.dims
    _need(d.kind == MLA, "an MLA table is required")
    _need(x.dtype == torch.bfloat16 and x.is_contiguous() and x.dim() == 3 and x.shape[0] == d.batch and
          x.shape[1] == n_tokens, "x must be contiguous bf16 [B, n_tokens, d_model]")
    _need(w_dkv.dtype == torch.bfloat16 and w_dkv.is_contiguous() and w_dkv.shape == (d.latent_dim, x.shape[2]),
          "w_dkv must be contiguous bf16 [r, d_model]")
    _need(k_rope.dtype == torch.bfloat16 and k_rope.is_contiguous() and
          k_rope.numel() == d.batch * n_tokens * d.rope_dim, "k_rope must be contiguous bf16 [B, n_tokens, 64]")
    if keep_idx is not None:
        _need(keep_idx.dtype == torch.int32 and keep_idx.is_contiguous() and
              keep_idx.numel() == d.batch * d.keep_tokens, "keep_idx must be int32 [B, keep_tokens]")
    if latent_out is not None:
        _need(latent_out.dtype == torch.bfloat16 and latent_out.is_contiguous(), "latent_out must be contiguous bf16")
    _need(_nbytes(arena) >= table_query(t).arena_bytes, "arena smaller than arena_bytes")
    _check(load().kvk_compress_layer_project(t.handle, layer, _ptr(x), _ptr(w_dkv), x.shape[2], _ptr(k_rope),
                                             n_tokens, _ptr(keep_idx), _ptr(arena), _ptr(latent_out),
                                             _stream(stream)))


def append_token(t: Table, layer_begin: int, layer_end: int, k: torch.Tensor, v: torch.Tensor,
                 n_stored: int, arena: torch.Tensor, stream=None):
    """Append one decoded token at position n_stored to every anchor in
    [layer_begin, layer_end).  GQA: k, v [layers, B, Hkv, d_h].  MLA: k = latent
    [layers, B, r], v = positional key [layers, B, d_R].  Contiguous bf16/fp32 on the
    device; the rows of inheriting layers are not read."""
    d = t.dims
    nl = layer_end - layer_begin
    _need(k.dtype == v.dtype and k.is_contiguous() and v.is_contiguous(),
          "k and v must be contiguous tensors of one dtype")
    if d.kind == MLA:
        _need(k.numel() == nl * d.batch * d.latent_dim and v.numel() == nl * d.batch * d.rope_dim,
              "latent size must be layers*B*r and k^R size layers*B*d_R")
    else:
        _need(k.numel() == v.numel() == nl * d.batch * d.n_kv_heads * d.head_dim,
              "k/v size must be layers*B*Hkv*d_h")
    _need(_nbytes(arena) >= table_query(t).arena_bytes, "arena smaller than arena_bytes")
    _check(load().kvk_append_token(t.handle, layer_begin, layer_end, _ptr(k), _ptr(v), _dtype_code(k),
                                   n_stored, _ptr(arena), _stream(stream)))


def snapkv_workspace_bytes(t: Table, n_tokens: int) -> int:
    out = ctypes.c_size_t(0)
    _check(load().kvk_snapkv_workspace_bytes(t.handle, n_tokens, ctypes.byref(out)))
    return out.value


def snapkv_select(t: Table, layer: int, k: torch.Tensor, q_obs: torch.Tensor, n_tokens: int, scale: float,
                  keep_out: torch.Tensor, workspace: torch.Tensor, importance: Optional[torch.Tensor] = None,
                  stream=None):
    """Query-aware keep list of one anchor layer at prefill.  k [B, Hkv, n_tokens, d_h]
    and q_obs [B, Hq, 32, d_h] (the last 32 prompt positions' queries) bf16; keep_out
    int32 [B, Hkv, keep_tokens]; importance (optional) fp32 [B, Hkv, n_tokens]."""
    d = t.dims
    _need(k.dtype == q_obs.dtype == torch.bfloat16 and k.is_contiguous() and q_obs.is_contiguous(),
          "k and q_obs must be contiguous bf16 tensors")
    _need(k.numel() == d.batch * d.n_kv_heads * n_tokens * d.head_dim, "k size must be B*Hkv*n_tokens*d_h")
    _need(q_obs.numel() == d.batch * d.n_q_heads * 32 * d.head_dim, "q_obs size must be B*Hq*32*d_h")
    _need(keep_out.dtype == torch.int32 and keep_out.is_contiguous() and
          keep_out.numel() == d.batch * d.n_kv_heads * d.keep_tokens, "keep_out must be int32 B*Hkv*keep_tokens")
    if importance is not None:
        _need(importance.dtype == torch.float32 and importance.is_contiguous() and
              importance.numel() == d.batch * d.n_kv_heads * n_tokens, "importance must be fp32 B*Hkv*n_tokens")
    _check(load().kvk_snapkv_select(t.handle, layer, _ptr(k), _ptr(q_obs), _dtype_code(k), n_tokens, float(scale),
                                    _ptr(keep_out), _ptr(importance), _ptr(workspace), _nbytes(workspace),
                                    _stream(stream)))


def snapkv_select_mla(t: Table, layer: int, latent: torch.Tensor, k_rope: torch.Tensor, q_obs: torch.Tensor,
                      n_tokens: int, scale: float, keep_out: torch.Tensor, workspace: torch.Tensor,
                      w_uk: Optional[torch.Tensor] = None, importance: Optional[torch.Tensor] = None, stream=None):
    """MLA keep list of one anchor layer at prefill, one list per sequence.  latent
    [B, n_tokens, r], k_rope [B, n_tokens, 64], q_obs [B, 32, Hq, nope + 64] bf16;
    w_uk [Hq, r, nope] (this layer's, as mla_weights_for_library arranges it) or None
    for the attached weights; keep_out int32 [B, keep_tokens]; importance (optional)
    fp32 [B, n_tokens]."""
    d = t.dims
    _need(d.kind == MLA, "an MLA table is required")
    _need(latent.dtype == k_rope.dtype == q_obs.dtype == torch.bfloat16 and latent.is_contiguous() and
          k_rope.is_contiguous() and q_obs.is_contiguous(), "latent, k_rope and q_obs must be contiguous bf16")
    _need(latent.numel() == d.batch * n_tokens * d.latent_dim and k_rope.numel() == d.batch * n_tokens * d.rope_dim,
          "latent must be B*n_tokens*r and k_rope B*n_tokens*64")
    _need(q_obs.numel() == d.batch * 32 * d.n_q_heads * (d.nope_dim + d.rope_dim), "q_obs must be B*32*Hq*(nope+64)")
    if w_uk is not None:
        _need(w_uk.dtype == torch.bfloat16 and w_uk.is_contiguous() and
              w_uk.numel() == d.n_q_heads * d.latent_dim * d.nope_dim, "w_uk must be bf16 [Hq, r, nope]")
    else:
        _need(t.mla_weights is not None, "pass w_uk or attach the weights (set_mla_weights)")
    _need(keep_out.dtype == torch.int32 and keep_out.is_contiguous() and keep_out.numel() == d.batch * d.keep_tokens,
          "keep_out must be int32 B*keep_tokens")
    if importance is not None:
        _need(importance.dtype == torch.float32 and importance.is_contiguous() and
              importance.numel() == d.batch * n_tokens, "importance must be fp32 B*n_tokens")
    _check(load().kvk_snapkv_select_mla(t.handle, layer, _ptr(latent), _ptr(k_rope), _ptr(q_obs), _ptr(w_uk),
                                        n_tokens, float(scale), _ptr(keep_out), _ptr(importance), _ptr(workspace),
                                        _nbytes(workspace), _stream(stream)))


# Composed action space (eq. (3)): index 0 = inherit, 1 + 4 j + k = produce with
# kept width r / 2^j at 16 / 2^k bits; a GQA selector uses the first five.
SELECTOR_ACTIONS = [(1, 1, 16)] + [(0, 1 << j, 16 >> k) for j in range(4) for k in range(4)]
SELECTOR_ACTIONS_GQA = 5


def selector_weight_elems(d_model: int, n_layers: int, n_actions: int = SELECTOR_ACTIONS_GQA) -> int:
    n = int(load().kvk_selector_weight_elems(d_model, n_layers, n_actions))
    _need(n > 0, f"selector sizes d_model {d_model}, n_layers {n_layers}, n_actions {n_actions}")
    return n


def selector_workspace_bytes(d_model: int, n_layers: int, n_tokens: int) -> int:
    out = ctypes.c_size_t(0)
    _check(load().kvk_selector_workspace_bytes(d_model, n_layers, n_tokens, ctypes.byref(out)))
    return out.value


def selector_forward(d_model: int, n_layers: int, weights: torch.Tensor, emb: torch.Tensor,
                     actions: torch.Tensor, workspace: torch.Tensor, logits: Optional[torch.Tensor] = None,
                     n_actions: int = SELECTOR_ACTIONS_GQA, depth: bool = True,
                     film: Optional[torch.Tensor] = None, stream=None):
    """emb [n_tokens, d_model] bf16; weights packed bf16 (see kvk.h); actions int32
    [n_layers]; logits (optional) fp32 [n_layers, n_actions]; film (optional) fp32
    [2, 256]: the budget scale gamma and shift beta applied to the pooled feature."""
    _need(emb.dtype == torch.bfloat16 and emb.is_contiguous() and emb.dim() == 2 and emb.shape[1] == d_model,
          "emb must be contiguous bf16 [n_tokens, d_model]")
    _need(weights.dtype == torch.bfloat16 and weights.is_contiguous() and
          weights.numel() == selector_weight_elems(d_model, n_layers, n_actions),
          "weights must be the packed bf16 vector")
    _need(actions.dtype == torch.int32 and actions.numel() == n_layers, "actions must be int32 [n_layers]")
    if logits is not None:
        _need(logits.dtype == torch.float32 and logits.is_contiguous() and logits.numel() == n_layers * n_actions,
              "logits must be fp32 [n_layers, n_actions]")
    if film is not None:
        _need(film.dtype == torch.float32 and film.is_contiguous() and film.numel() == 2 * 256,
              "film must be fp32 [2, 256]")
    _check(load().kvk_selector_forward(d_model, n_layers, n_actions, 1 if depth else 0, _ptr(weights), _ptr(emb),
                                       emb.shape[0], _ptr(film), _ptr(logits), _ptr(actions), _ptr(workspace),
                                       _nbytes(workspace), _stream(stream)))


def decode_attention(t: Table, layer_begin: int, layer_end: int, q: torch.Tensor, n_stored: int,
                     scale: float, arena: torch.Tensor, out: torch.Tensor, workspace: torch.Tensor,
                     w_uk: Optional[torch.Tensor] = None, w_uv: Optional[torch.Tensor] = None,
                     stream=None):
    """q: [layers, B, Hq, d_h] (MLA: [layers, B, Hq, nope + d_R]) bf16/fp32; out fp32
    [layers, B, Hq, d_h] (MLA: v_dim); w_uk: MLA W_UK transposed [layers, Hq, r, nope]
    and w_uv [layers, Hq, v, r], bf16 (see mla_weights_for_library)."""
    d = t.dims
    nl = layer_end - layer_begin
    _need(q.is_contiguous() and out.is_contiguous() and out.dtype == torch.float32,
          "q must be contiguous; out contiguous fp32")
    _need(q.numel() == nl * d.batch * d.n_q_heads * _q_width(d), "q size must be layers*B*Hq*width")
    _need(out.numel() == nl * d.batch * d.n_q_heads * _out_width(d), "out size must be layers*B*Hq*width")
    _check_weights(t, nl, w_uk, w_uv)
    _need(_nbytes(arena) >= table_query(t).arena_bytes, "arena smaller than arena_bytes")
    _check(load().kvk_decode_attention(
        t.handle, layer_begin, layer_end, _ptr(q), _dtype_code(q), n_stored, float(scale),
        _ptr(w_uk), _ptr(w_uv), _ptr(arena), _ptr(out), _ptr(workspace),
        workspace.numel() * workspace.element_size(), _stream(stream)))


def decode_setup(t: Table, layer_begin: int, layer_end: int, workspace: torch.Tensor, stream=None):
    """Once per (table, layer range, workspace) before decoding a per-sequence table:
    writes the work list to the head of the workspace (synchronises the stream)."""
    _check(load().kvk_decode_setup(t.handle, layer_begin, layer_end, _ptr(workspace), _nbytes(workspace),
                                   _stream(stream)))


NOALLOC_SCRATCH_BYTES = 64 << 20  # KVK_NOALLOC_SCRATCH_BYTES


def decode_attention_noalloc(t: Table, layer_begin: int, layer_end: int, q: torch.Tensor, n_stored: int,
                             scale: float, arena: torch.Tensor, out: torch.Tensor,
                             w_uk: Optional[torch.Tensor] = None, w_uv: Optional[torch.Tensor] = None,
                             stream=None):
    """decode_attention without a workspace: the library's static device scratch
    holds the split partials (calls that overlap on one GPU race)."""
    d = t.dims
    nl = layer_end - layer_begin
    _need(q.is_contiguous() and out.is_contiguous() and out.dtype == torch.float32,
          "q must be contiguous; out contiguous fp32")
    _need(q.numel() == nl * d.batch * d.n_q_heads * _q_width(d), "q size must be layers*B*Hq*width")
    _need(out.numel() == nl * d.batch * d.n_q_heads * _out_width(d), "out size must be layers*B*Hq*width")
    _check_weights(t, nl, w_uk, w_uv)
    _need(_nbytes(arena) >= table_query(t).arena_bytes, "arena smaller than arena_bytes")
    _check(load().kvk_decode_attention_noalloc(
        t.handle, layer_begin, layer_end, _ptr(q), _dtype_code(q), n_stored, float(scale),
        _ptr(w_uk), _ptr(w_uv), _ptr(arena), _ptr(out), _stream(stream)))


def decode_splits(t: Table, layer_begin: int, layer_end: int, q: torch.Tensor, n_stored: int,
                  scale: float, arena: torch.Tensor, workspace: torch.Tensor,
                  w_uk: Optional[torch.Tensor] = None, w_uv: Optional[torch.Tensor] = None,
                  stream=None):
    """First phase of decode_attention: split partials into `workspace`."""
    d = t.dims
    nl = layer_end - layer_begin
    _need(q.is_contiguous() and q.numel() == nl * d.batch * d.n_q_heads * _q_width(d),
          "q must be contiguous, layers*B*Hq*width")
    _check_weights(t, nl, w_uk, w_uv)
    _need(_nbytes(arena) >= table_query(t).arena_bytes, "arena smaller than arena_bytes")
    _check(load().kvk_decode_splits(
        t.handle, layer_begin, layer_end, _ptr(q), _dtype_code(q), n_stored, float(scale),
        _ptr(w_uk), _ptr(w_uv), _ptr(arena), _ptr(workspace), _nbytes(workspace), _stream(stream)))


def decode_merge(t: Table, layer_begin: int, layer_end: int, q: torch.Tensor, n_stored: int,
                 scale: float, arena: torch.Tensor, workspace: torch.Tensor, out: torch.Tensor,
                 w_uk: Optional[torch.Tensor] = None, w_uv: Optional[torch.Tensor] = None,
                 stream=None):
    """Second phase of decode_attention: merge of the split partials (GQA: with the
    tail tokens; MLA: then the W_UV up-projection)."""
    d = t.dims
    nl = layer_end - layer_begin
    _need(q.is_contiguous() and q.numel() == nl * d.batch * d.n_q_heads * _q_width(d),
          "q must be contiguous, layers*B*Hq*width")
    _need(out.is_contiguous() and out.dtype == torch.float32 and
          out.numel() == nl * d.batch * d.n_q_heads * _out_width(d),
          "out must be contiguous fp32, layers*B*Hq*width")
    _check_weights(t, nl, w_uk, w_uv)
    _need(_nbytes(arena) >= table_query(t).arena_bytes, "arena smaller than arena_bytes")
    _check(load().kvk_decode_merge(
        t.handle, layer_begin, layer_end, _ptr(q), _dtype_code(q), n_stored, float(scale),
        _ptr(w_uk), _ptr(w_uv), _ptr(arena), _ptr(workspace), _nbytes(workspace), _ptr(out),
        _stream(stream)))


def read_bytes(t: Table, layer_begin: int, layer_end: int, n_stored: int) -> int:
    out = ctypes.c_int64()
    _check(load().kvk_read_bytes(t.handle, layer_begin, layer_end, n_stored, ctypes.byref(out)))
    return out.value


def debug_dequantize(t: Table, layer: int, n_stored: int, arena: torch.Tensor, k_out: torch.Tensor,
                     v_out: torch.Tensor, stream=None):
    """GQA: k_out, v_out fp32 [B, Hkv, n_stored, d_h].  MLA: k_out = latent fp32
    [B, n_stored, d] (the anchor's kept width), v_out = k^R fp32 [B, n_stored, d_R];
    under per-sequence plans sequence b's latent starts at b * n_stored * r, in rows
    of its own anchor's kept width."""
    d = t.dims
    n = max(n_stored, 0)
    if d.kind == MLA and getattr(t, "plans", None) is not None:
        nk, nv = d.batch * n * d.latent_dim, d.batch * n * d.rope_dim
    elif d.kind == MLA:
        a = table_query(t).anchor_of[layer]
        nk, nv = d.batch * n * t.plan[a].rank, d.batch * n * d.rope_dim
    else:
        nk = nv = d.batch * d.n_kv_heads * n * d.head_dim
    _need(k_out.dtype == torch.float32 and v_out.dtype == torch.float32, "outputs must be fp32")
    _need(k_out.numel() >= nk and v_out.numel() >= nv, "outputs smaller than the dequantised cache")
    _need(_nbytes(arena) >= table_query(t).arena_bytes, "arena smaller than arena_bytes")
    _check(load().kvk_debug_dequantize(t.handle, layer, n_stored, _ptr(arena), _ptr(k_out),
                                       _ptr(v_out), _stream(stream)))


def realized_bits(qscheme: int, bits: int, group: int, window: int, context: int) -> float:
    return load().kvk_realized_bits(qscheme, bits, group, window, context)


def rho_range(n_layers: int, kv_width: int, latent_dim: int, rope_dim: int, mla: bool,
              precision: bool, rank: bool, depth: bool):
    lo, hi = ctypes.c_double(), ctypes.c_double()
    axes = (1 if precision else 0) | (2 if rank else 0) | (4 if depth else 0)
    _check(load().kvk_rho_range(n_layers, kv_width, latent_dim, rope_dim, int(mla), axes,
                                ctypes.byref(lo), ctypes.byref(hi)))
    return lo.value, hi.value
