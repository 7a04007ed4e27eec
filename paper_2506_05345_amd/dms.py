"""Python binding of libdms (include/dms.h).

The functions named ``dms_*`` mirror the C entry points one to one and only
marshal arguments: device pointers may be given as integers or as tensors
(their ``data_ptr()``), streams as integers, ``torch.cuda.Stream`` objects or
None (the current stream).  :class:`DmsCache` is plumbing on top: it lets
PyTorch allocate the caller-owned buffers the library works in.

There is no fallback: if ``libdms.so`` is missing the first call raises.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libdms.so")

DMS_OK = 0
DMS_ERR_INVALID = -1
DMS_ERR_UNSUPPORTED = -2
DMS_ERR_HIP = -3
DMS_ERR_OUT_OF_PAGES = -4
DMS_ERR_CAPACITY = -5
DMS_ERR_BAD_SEQ = -6
DMS_ERR_SCRATCH = -7


class DmsConfig(ctypes.Structure):
    _fields_ = [
        ("num_layers", ctypes.c_int32),
        ("max_seqs", ctypes.c_int32),
        ("num_kv_heads", ctypes.c_int32),
        ("group_size", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("window", ctypes.c_int32),
        ("page_size", ctypes.c_int32),
        ("num_pages", ctypes.c_int32),
        ("max_pages_per_head", ctypes.c_int32),
        ("max_chunk_tokens", ctypes.c_int32),
        ("softmax_scale", ctypes.c_float),
        ("eviction", ctypes.c_int32),
        ("decision_source", ctypes.c_int32),
        ("decision_bias", ctypes.c_float),
        ("kv_format", ctypes.c_int32),
        ("quest_page_budget", ctypes.c_int32),
    ]


class DmsTrainConfig(ctypes.Structure):
    _fields_ = [
        ("batch", ctypes.c_int32),
        ("seq_len", ctypes.c_int32),
        ("num_kv_heads", ctypes.c_int32),
        ("group_size", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("window", ctypes.c_int32),
        ("softmax_scale", ctypes.c_float),
    ]


DMS_EVICT_DELAYED = 0
DMS_EVICT_IMMEDIATE = 1
DMS_DECIDE_CALLER = 0
DMS_DECIDE_QUERY = 1
DMS_KV_BF16 = 0
DMS_KV_FP8 = 1
DMS_KV_MLA = 2
MLA_ROW_DIM = 576      # latent (512) + rotary key (64)
MLA_LATENT_DIM = 512


class DmsStateOffsets(ctypes.Structure):
    _fields_ = [(n, ctypes.c_size_t) for n in
                ("status", "layer0", "layer_stride", "pos", "len", "ring", "page_table",
                 "slot_meta", "stack", "top", "page_bounds")]


class DmsError(RuntimeError):
    def __init__(self, code: int, where: str = ""):
        self.code = code
        super().__init__(f"{where}: {dms_strerror(code)} ({code})")


_lib = None
_VP = ctypes.c_void_p
_I = ctypes.c_int
_SZ = ctypes.c_size_t

_SIGS = {
    "dms_layout": (_I, [ctypes.POINTER(DmsConfig), ctypes.POINTER(_SZ), ctypes.POINTER(_SZ),
                        ctypes.POINTER(_SZ), ctypes.POINTER(_SZ)]),
    "dms_state_layout": (_I, [ctypes.POINTER(DmsConfig), ctypes.POINTER(DmsStateOffsets)]),
    "dms_create": (_I, [ctypes.POINTER(DmsConfig), _VP, ctypes.POINTER(_VP), _VP,
                        ctypes.POINTER(_VP)]),
    "dms_destroy": (_I, [_VP]),
    "dms_init_state": (_I, [_VP, _VP]),
    "dms_seq_reset": (_I, [_VP, _I, _I, _VP, _VP]),
    "dms_append": (_I, [_VP, _I, _I, _VP, _VP, _VP, _VP, _VP]),
    "dms_decode": (_I, [_VP, _I, _I, _VP, _VP, _VP, _VP]),
    "dms_decode_step": (_I, [_VP, _I, _I, _VP, _VP, _VP, _VP, _VP, _VP, _VP]),
    "dms_append_chunk": (_I, [_VP, _I, _I, _VP, _VP, _I, _I, _VP, _VP, _VP, _VP]),
    "dms_prefill_chunk": (_I, [_VP, _I, _I, _VP, _VP, _I, _I, _VP, _VP, _VP, _VP, _VP, _VP]),
    "dms_decode_step_q": (_I, [_VP, _I, _I, _VP, _VP, _VP, _VP, _VP, _VP, _VP]),
    "dms_decode_step_static": (_I, [_VP, _I, _I, _VP, _VP, _VP, _VP, _VP, _VP, _VP]),
    "dms_prefill_chunk_q": (_I, [_VP, _I, _I, _VP, _VP, _I, _I, _VP, _VP, _VP, _VP, _VP, _VP]),
    "dms_retained_lengths": (_I, [_VP, _I, _I, _VP, _VP, _VP]),
    "dms_quest_selection": (_I, [_VP, _I, _VP, _VP, _VP]),
    "dms_export_state": (_I, [_VP, _I, _VP, _SZ, _VP]),
    "dms_status": (_I, [_VP, _VP]),
    "dms_clear_status": (_I, [_VP, _VP]),
    "dms_profile_start": (_I, [_VP, _I]),
    "dms_profile_stop": (_I, [_VP, ctypes.POINTER(ctypes.c_float), ctypes.POINTER(_I)]),
    "dms_strerror": (ctypes.c_char_p, [_I]),
    "dms_train_workspace": (_I, [ctypes.POINTER(DmsTrainConfig), ctypes.POINTER(_SZ)]),
    "dms_train_attention_fwd": (_I, [ctypes.POINTER(DmsTrainConfig), _VP, _VP, _VP, _VP, _VP, _VP,
                                     _VP, _VP]),
    "dms_train_attention_bwd": (_I, [ctypes.POINTER(DmsTrainConfig), _VP, _VP, _VP, _VP, _VP, _VP,
                                     _VP, _VP, _VP, _VP, _VP, _VP, _VP]),
    "dms_gumbel_sigmoid_fwd": (_I, [_I, _VP, _VP, ctypes.c_float, _VP, _VP]),
    "dms_gumbel_sigmoid_bwd": (_I, [_I, _VP, _VP, ctypes.c_float, _VP, _VP]),
}


def lib():
    """Load libdms.so (built in-tree); raises if it is missing."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run __graft_entry__.build()")
        h = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            fn = getattr(h, name)
            fn.restype = res
            fn.argtypes = args
        _lib = h
    return _lib


def _ptr(x):
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if hasattr(x, "data_ptr"):
        return x.data_ptr()
    raise TypeError(f"cannot pass {type(x)} as a pointer")


def _stream(s):
    if s is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(s, int):
        return s
    return s.cuda_stream


def _check(rc, where):
    if rc != DMS_OK:
        raise DmsError(rc, where)


# Configuration of every live context (by handle), for the argument checks.
_CTX_CFG = {}

_BF16 = "bf16"
_U8 = "uint8"
_I32 = "int32"
_F32 = "float32"


def _args(where, *specs):
    """Check tensor arguments before their addresses are handed to the library.
    Each spec is (tensor, name, element type, minimum element count).  Element
    types of all arguments are checked first, then that each is a contiguous
    GPU tensor with enough elements.  Integers (raw device addresses) and None
    pass through; the library checks null pointers itself."""
    if all(x is None or isinstance(x, int) for x, *_ in specs):
        return
    import torch
    kinds = {_BF16: torch.bfloat16, _U8: torch.uint8, _I32: torch.int32, _F32: torch.float32}
    live = []
    for x, name, kind, count in specs:
        if x is None or isinstance(x, int):
            continue
        if not isinstance(x, torch.Tensor):
            raise TypeError(f"{where}: {name} must be a tensor or a device address, got {type(x)}")
        if x.dtype != kinds[kind]:
            raise DmsError(DMS_ERR_INVALID, f"{where}: {name} must be {kind}, got {x.dtype}")
        live.append((x, name, count))
    for x, name, count in live:
        if not x.is_cuda:
            raise DmsError(DMS_ERR_INVALID, f"{where}: {name} must be a GPU tensor")
        if not x.is_contiguous():
            raise DmsError(DMS_ERR_INVALID, f"{where}: {name} must be contiguous")
        if x.numel() < count:
            raise DmsError(DMS_ERR_INVALID,
                           f"{where}: {name} holds {x.numel()} elements, needs {count}")


def _arg(x, name, kind, count, where):
    _args(where, (x, name, kind, count))


def _dims(ctx):
    """(Hkv, Hq, d, output row width) of a context's configuration, or None for
    a handle this module did not create."""
    c = _CTX_CFG.get(ctx)
    if c is None:
        return None
    out_d = MLA_LATENT_DIM if c.kv_format == DMS_KV_MLA else c.head_dim
    return c.num_kv_heads, c.num_kv_heads * c.group_size, c.head_dim, out_d


def _check_kv_args(ctx, where, n, rows, seq_ids=None, cu=None, k=None, v=None, flags=None,
                   q=None, out=None, decisions=None):
    """seq_ids [n] and cu_seqlens [n + 1] int32; per-row tensors for `rows`
    rows (tokens of a chunk, or one per sequence)."""
    specs = [(seq_ids, "seq_ids", _I32, n), (cu, "cu_seqlens", _I32, n + 1)]
    dims = _dims(ctx)
    if dims is not None:
        H, Hq, D, Dout = dims
        specs += [(k, "k", _BF16, rows * H * D), (v, "v", _BF16, rows * H * D),
                  (flags, "flags", _U8, rows * H), (decisions, "decisions_out", _U8, rows * H),
                  (q, "q", _BF16, rows * Hq * D), (out, "out", _F32, rows * Hq * Dout)]
    _args(where, *specs)


def make_config(num_layers, max_seqs, num_kv_heads, group_size, head_dim, window,
                page_size, num_pages, max_pages_per_head, max_chunk_tokens=0,
                softmax_scale=0.0, eviction=DMS_EVICT_DELAYED,
                decision_source=DMS_DECIDE_CALLER, decision_bias=-5.0,
                kv_format=DMS_KV_BF16, quest_page_budget=0) -> DmsConfig:
    return DmsConfig(num_layers, max_seqs, num_kv_heads, group_size, head_dim, window,
                     page_size, num_pages, max_pages_per_head, max_chunk_tokens,
                     softmax_scale, eviction, decision_source, decision_bias, kv_format,
                     quest_page_budget)


# ---------------------------------------------------------------------------
# Entry points (same names as the C ABI)
# ---------------------------------------------------------------------------

def dms_layout(cfg: DmsConfig):
    a, b, c, d = _SZ(), _SZ(), _SZ(), _SZ()
    _check(lib().dms_layout(ctypes.byref(cfg), ctypes.byref(a), ctypes.byref(b),
                            ctypes.byref(c), ctypes.byref(d)), "dms_layout")
    return a.value, b.value, c.value, d.value


def dms_state_layout(cfg: DmsConfig) -> DmsStateOffsets:
    o = DmsStateOffsets()
    _check(lib().dms_state_layout(ctypes.byref(cfg), ctypes.byref(o)), "dms_state_layout")
    return o


def dms_create(cfg: DmsConfig, meta, pools, workspace):
    arr = (_VP * cfg.num_layers)(*[_ptr(p) for p in pools])
    out = _VP()
    _check(lib().dms_create(ctypes.byref(cfg), _ptr(meta), arr, _ptr(workspace),
                            ctypes.byref(out)), "dms_create")
    _CTX_CFG[out.value] = DmsConfig.from_buffer_copy(cfg)
    return out.value


def dms_destroy(ctx):
    _check(lib().dms_destroy(ctx), "dms_destroy")
    _CTX_CFG.pop(ctx, None)


def dms_init_state(ctx, stream=None):
    _check(lib().dms_init_state(ctx, _stream(stream)), "dms_init_state")


def dms_seq_reset(ctx, layer, n, seq_ids, stream=None):
    _arg(seq_ids, "seq_ids", _I32, n, "dms_seq_reset")
    _check(lib().dms_seq_reset(ctx, layer, n, _ptr(seq_ids), _stream(stream)), "dms_seq_reset")


def dms_append(ctx, layer, n, seq_ids, k, v, flags, stream=None):
    _check_kv_args(ctx, "dms_append", n, n, seq_ids=seq_ids, k=k, v=v, flags=flags)
    _check(lib().dms_append(ctx, layer, n, _ptr(seq_ids), _ptr(k), _ptr(v), _ptr(flags),
                            _stream(stream)), "dms_append")


def dms_decode(ctx, layer, n, seq_ids, q, out, stream=None):
    _check_kv_args(ctx, "dms_decode", n, n, seq_ids=seq_ids, q=q, out=out)
    _check(lib().dms_decode(ctx, layer, n, _ptr(seq_ids), _ptr(q), _ptr(out), _stream(stream)),
           "dms_decode")


def dms_decode_step(ctx, layer, n, seq_ids, q, k, v, flags, out, stream=None):
    _check_kv_args(ctx, "dms_decode_step", n, n, seq_ids=seq_ids, k=k, v=v, flags=flags, q=q,
                   out=out)
    _check(lib().dms_decode_step(ctx, layer, n, _ptr(seq_ids), _ptr(q), _ptr(k), _ptr(v),
                                 _ptr(flags), _ptr(out), _stream(stream)), "dms_decode_step")


def dms_decode_step_static(ctx, layer, n, seq_ids, q, k, v, flags, out, stream=None):
    _check_kv_args(ctx, "dms_decode_step_static", n, n, seq_ids=seq_ids, k=k, v=v, flags=flags,
                   q=q, out=out)
    _check(lib().dms_decode_step_static(ctx, layer, n, _ptr(seq_ids), _ptr(q), _ptr(k), _ptr(v),
                                        _ptr(flags), _ptr(out), _stream(stream)),
           "dms_decode_step_static")


def dms_decode_step_q(ctx, layer, n, seq_ids, q, k, v, decisions_out, out, stream=None):
    _check_kv_args(ctx, "dms_decode_step_q", n, n, seq_ids=seq_ids, k=k, v=v, q=q, out=out,
                   decisions=decisions_out)
    _check(lib().dms_decode_step_q(ctx, layer, n, _ptr(seq_ids), _ptr(q), _ptr(k), _ptr(v),
                                   _ptr(decisions_out), _ptr(out), _stream(stream)),
           "dms_decode_step_q")


def dms_append_chunk(ctx, layer, n, seq_ids, cu_seqlens, total_tokens, max_seqlen, k, v, flags,
                     stream=None):
    _check_kv_args(ctx, "dms_append_chunk", n, total_tokens, seq_ids=seq_ids, cu=cu_seqlens, k=k,
                   v=v, flags=flags)
    _check(lib().dms_append_chunk(ctx, layer, n, _ptr(seq_ids), _ptr(cu_seqlens), total_tokens,
                                  max_seqlen, _ptr(k), _ptr(v), _ptr(flags), _stream(stream)),
           "dms_append_chunk")


def dms_prefill_chunk(ctx, layer, n, seq_ids, cu_seqlens, total_tokens, max_seqlen, q, k, v,
                      flags, out, stream=None):
    _check_kv_args(ctx, "dms_prefill_chunk", n, total_tokens, seq_ids=seq_ids, cu=cu_seqlens, k=k,
                   v=v, flags=flags, q=q, out=out)
    _check(lib().dms_prefill_chunk(ctx, layer, n, _ptr(seq_ids), _ptr(cu_seqlens), total_tokens,
                                   max_seqlen, _ptr(q), _ptr(k), _ptr(v), _ptr(flags), _ptr(out),
                                   _stream(stream)), "dms_prefill_chunk")


def dms_prefill_chunk_q(ctx, layer, n, seq_ids, cu_seqlens, total_tokens, max_seqlen, q, k, v,
                        decisions_out, out, stream=None):
    _check_kv_args(ctx, "dms_prefill_chunk_q", n, total_tokens, seq_ids=seq_ids, cu=cu_seqlens,
                   k=k, v=v, q=q, out=out, decisions=decisions_out)
    _check(lib().dms_prefill_chunk_q(ctx, layer, n, _ptr(seq_ids), _ptr(cu_seqlens), total_tokens,
                                     max_seqlen, _ptr(q), _ptr(k), _ptr(v), _ptr(decisions_out),
                                     _ptr(out), _stream(stream)), "dms_prefill_chunk_q")


def dms_retained_lengths(ctx, layer, n, seq_ids, out, stream=None):
    dims = _dims(ctx)
    _args("dms_retained_lengths", (seq_ids, "seq_ids", _I32, n),
          (out, "out", _I32, n * dims[0] if dims else 0))
    _check(lib().dms_retained_lengths(ctx, layer, n, _ptr(seq_ids), _ptr(out), _stream(stream)),
           "dms_retained_lengths")


def dms_quest_selection(ctx, n, pages_out, count_out, stream=None):
    c = _CTX_CFG.get(ctx)
    if c is not None:
        _args("dms_quest_selection",
              (pages_out, "pages_out", _I32, n * c.num_kv_heads * max(c.quest_page_budget, 1)),
              (count_out, "count_out", _I32, n * c.num_kv_heads))
    _check(lib().dms_quest_selection(ctx, n, _ptr(pages_out), _ptr(count_out), _stream(stream)),
           "dms_quest_selection")


def dms_export_state(ctx, layer, nbytes, stream=None) -> np.ndarray:
    buf = np.empty(nbytes, dtype=np.uint8)
    _check(lib().dms_export_state(ctx, layer, buf.ctypes.data, nbytes, _stream(stream)),
           "dms_export_state")
    return buf


def dms_status(ctx, stream=None) -> int:
    return lib().dms_status(ctx, _stream(stream))


def dms_clear_status(ctx, stream=None):
    _check(lib().dms_clear_status(ctx, _stream(stream)), "dms_clear_status")


def dms_profile_start(ctx, max_launches):
    _check(lib().dms_profile_start(ctx, max_launches), "dms_profile_start")


DMS_PROFILE_DECODE = 0
DMS_PROFILE_PREFILL = 1


def dms_profile_stop(ctx):
    """Returns {kind: (total milliseconds, launches recorded)} for the decode
    and prefill-attention kernels."""
    ms, n = (ctypes.c_float * 2)(), (_I * 2)()
    _check(lib().dms_profile_stop(ctx, ms, n), "dms_profile_stop")
    return {DMS_PROFILE_DECODE: (ms[0], n[0]), DMS_PROFILE_PREFILL: (ms[1], n[1])}


def dms_strerror(code: int) -> str:
    return lib().dms_strerror(code).decode()


# ---------------------------------------------------------------------------
# PyTorch-owned buffers
# ---------------------------------------------------------------------------

@dataclass
class LayerStateView:
    """One layer's exported state as NumPy arrays (see dms_state_offsets)."""
    pos: np.ndarray
    L: np.ndarray
    ring_slot: np.ndarray
    ring_flag: np.ndarray
    page_table: np.ndarray
    slot_pos: np.ndarray
    slot_flag: np.ndarray
    stack: np.ndarray
    top: int


class DmsCache:
    """Device buffers for one context, allocated by PyTorch on ``device``."""

    def __init__(self, cfg: DmsConfig, device="cuda", pool_pages=None):
        import torch
        self.cfg = cfg
        self.meta_bytes, self.pool_bytes, self.ws_bytes, self.page_bytes = dms_layout(cfg)
        self.offsets = dms_state_layout(cfg)
        self.meta = torch.empty(self.meta_bytes, dtype=torch.uint8, device=device)
        self.pools = [torch.empty(self.pool_bytes, dtype=torch.uint8, device=device)
                      for _ in range(cfg.num_layers)]
        self.workspace = torch.empty(max(self.ws_bytes, 1), dtype=torch.uint8, device=device)
        self.ctx = dms_create(cfg, self.meta, self.pools, self.workspace)
        dms_init_state(self.ctx)

    def close(self):
        if self.ctx:
            dms_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def export(self, layer) -> LayerStateView:
        c, o = self.cfg, self.offsets
        raw = dms_export_state(self.ctx, layer, o.layer_stride)
        S, H, w = c.max_seqs, c.num_kv_heads, c.window
        maxp, P = c.max_pages_per_head, c.page_size

        def arr(off, count):
            return raw[off: off + 4 * count].view(np.int32)

        ring = arr(o.ring, S * H * w).reshape(S, H, w).view(np.uint32)
        meta = arr(o.slot_meta, S * H * maxp * P).reshape(S, H, maxp * P).view(np.uint32)
        top = int(arr(o.top, 1)[0])
        return LayerStateView(
            pos=arr(o.pos, S).copy(),
            L=arr(o.len, S * H).reshape(S, H).copy(),
            ring_slot=(ring & 0x7FFFFFFF).astype(np.int64),
            ring_flag=(ring >> 31).astype(np.uint8),
            page_table=arr(o.page_table, S * H * maxp).reshape(S, H, maxp).astype(np.int64),
            slot_pos=(meta & 0x7FFFFFFF).astype(np.int64),
            slot_flag=(meta >> 31).astype(np.uint8),
            stack=arr(o.stack, c.num_pages)[:top].astype(np.int64),
            top=top,
        )

    def pool_page_kv(self, layer, page):
        """One page on the host: bf16 pages give (K [P, d], V [P, d]) bit patterns
        (uint16); latent pages give (rows [P, d], their latent part [P, 512]);
        FP8 pages give (K codes, V codes [P, d] uint8, K scales, V scales
        [P] float32)."""
        raw = self.pools[layer][page * self.page_bytes:(page + 1) * self.page_bytes].cpu().numpy()
        if self.cfg.kv_format == DMS_KV_FP8:
            return unpack_page_fp8(raw, self.cfg.page_size, self.cfg.head_dim)
        if self.cfg.kv_format == DMS_KV_MLA:
            rows = unpack_page_mla(raw.view(np.uint16), self.cfg.page_size, self.cfg.head_dim)
            return rows, rows[:, :MLA_LATENT_DIM]
        return unpack_page(raw.view(np.uint16), self.cfg.page_size, self.cfg.head_dim)


def unpack_page(u16, P, D):
    """Decode one page (uint16 words, fragment-ordered tiles of dms.h) into K, V [P, D]."""
    tiles = np.asarray(u16).reshape(P // 32, 2, D * 32)
    j = np.arange(32)[:, None]
    e = np.arange(D)[None, :]
    h, r = (j // 4) % 2, 4 * (j // 8) + j % 4
    koff = ((((e // 32) * 2 + h) * 4 + (e // 8) % 4) * 16 + r) * 8 + e % 8
    voff = (((e // 16) * 4 + j // 8) * 16 + e % 16) * 8 + j % 8
    k = tiles[:, 0][:, koff].reshape(P, D)
    v = tiles[:, 1][:, voff].reshape(P, D)
    return k, v


def unpack_page_mla(u16, P, D):
    """Decode one latent-attention page (uint16 words) into its rows [P, D]:
    tiles of 32 rows in the key order of the bf16 pages, no value part."""
    tiles = np.asarray(u16).reshape(P // 32, D * 32)
    j = np.arange(32)[:, None]
    e = np.arange(D)[None, :]
    h, r = (j // 4) % 2, 4 * (j // 8) + j % 4
    koff = ((((e // 32) * 2 + h) * 4 + (e // 8) % 4) * 16 + r) * 8 + e % 8
    return tiles[:, koff].reshape(P, D)


def unpack_page_fp8(raw, P, D):
    """Decode one FP8 page (bytes, layout of dms.h) into K codes, V codes [P, D]
    (uint8) and K scales, V scales [P] (float32)."""
    tb = 64 * D + 256
    tiles = np.asarray(raw, np.uint8).reshape(P // 32, tb)
    j = np.arange(32)[:, None]
    e = np.arange(D)[None, :]
    h, r = (j // 4) % 2, 4 * (j // 8) + j % 4
    koff = (e // 64) * 2048 + h * 1024 + (16 * ((e // 8) % 4) + r) * 16 + 8 * ((e // 32) % 2) + e % 8
    voff = 32 * D + (e // 32) * 1024 + (16 * (j // 8) + e % 16) * 16 + 8 * ((e // 16) % 2) + j % 8
    soff = 64 * D + (np.arange(32) // 8) * 64 + (np.arange(32) % 8) * 4
    k = tiles[:, koff].reshape(P, D)
    v = tiles[:, voff].reshape(P, D)
    sc = tiles[:, soff[:, None] + np.arange(4)[None, :]].reshape(P // 32, 32, 4)
    ks = np.ascontiguousarray(sc).view(np.float32).reshape(P)
    sv = tiles[:, soff[:, None] + 32 + np.arange(4)[None, :]].reshape(P // 32, 32, 4)
    vs = np.ascontiguousarray(sv).view(np.float32).reshape(P)
    return k, v, ks, vs


# ---------------------------------------------------------------------------
# Training-time attention (continuous decisions)
# ---------------------------------------------------------------------------

def make_train_config(batch, seq_len, num_kv_heads, group_size, head_dim, window,
                      softmax_scale=0.0) -> DmsTrainConfig:
    return DmsTrainConfig(batch, seq_len, num_kv_heads, group_size, head_dim, window, softmax_scale)


def dms_train_workspace(cfg: DmsTrainConfig) -> int:
    n = _SZ()
    _check(lib().dms_train_workspace(ctypes.byref(cfg), ctypes.byref(n)), "dms_train_workspace")
    return n.value


def _check_train_args(cfg, where, **t):
    B, T, H, g, D = cfg.batch, cfg.seq_len, cfg.num_kv_heads, cfg.group_size, cfg.head_dim
    rows_q, rows_k = B * T * H * g, B * T * H
    spec = {"q": (_BF16, rows_q * D), "dout": (_BF16, rows_q * D), "k": (_BF16, rows_k * D),
            "v": (_BF16, rows_k * D), "alpha": (_F32, rows_k), "out": (_F32, rows_q * D),
            "lse": (_F32, rows_q), "dq": (_F32, rows_q * D), "dk": (_F32, rows_k * D),
            "dv": (_F32, rows_k * D), "dalpha": (_F32, rows_k)}
    specs = [(x, name, *spec[name]) for name, x in t.items() if name != "workspace"]
    ws = t.get("workspace")
    if ws is not None and not isinstance(ws, int):
        # the size is only known for a valid configuration (else the library refuses it)
        need = dms_train_workspace(cfg) if cfg.batch >= 1 and cfg.seq_len >= 1 else 0
        specs.append((ws, "workspace", _U8, need))
    _args(where, *specs)


def dms_train_attention_fwd(cfg, q, k, v, alpha, out, lse, workspace, stream=None):
    _check_train_args(cfg, "dms_train_attention_fwd", q=q, k=k, v=v, alpha=alpha, out=out,
                      lse=lse, workspace=workspace)
    _check(lib().dms_train_attention_fwd(ctypes.byref(cfg), _ptr(q), _ptr(k), _ptr(v), _ptr(alpha),
                                         _ptr(out), _ptr(lse), _ptr(workspace), _stream(stream)),
           "dms_train_attention_fwd")


def dms_train_attention_bwd(cfg, q, k, v, alpha, out, lse, dout, dq, dk, dv, dalpha, workspace,
                            stream=None):
    _check_train_args(cfg, "dms_train_attention_bwd", q=q, k=k, v=v, alpha=alpha, out=out,
                      lse=lse, dout=dout, dq=dq, dk=dk, dv=dv, dalpha=dalpha, workspace=workspace)
    _check(lib().dms_train_attention_bwd(ctypes.byref(cfg), _ptr(q), _ptr(k), _ptr(v), _ptr(alpha),
                                         _ptr(out), _ptr(lse), _ptr(dout), _ptr(dq), _ptr(dk),
                                         _ptr(dv), _ptr(dalpha), _ptr(workspace), _stream(stream)),
           "dms_train_attention_bwd")


def dms_gumbel_sigmoid_fwd(n, logits, u, tau, alpha, stream=None):
    _args("dms_gumbel_sigmoid_fwd", (logits, "logits", _F32, n), (u, "u", _F32, n),
          (alpha, "alpha", _F32, n))
    _check(lib().dms_gumbel_sigmoid_fwd(n, _ptr(logits), _ptr(u), tau, _ptr(alpha), _stream(stream)),
           "dms_gumbel_sigmoid_fwd")


def dms_gumbel_sigmoid_bwd(n, alpha, dalpha, tau, dlogits, stream=None):
    _args("dms_gumbel_sigmoid_bwd", (alpha, "alpha", _F32, n), (dalpha, "dalpha", _F32, n),
          (dlogits, "dlogits", _F32, n))
    _check(lib().dms_gumbel_sigmoid_bwd(n, _ptr(alpha), _ptr(dalpha), tau, _ptr(dlogits),
                                        _stream(stream)), "dms_gumbel_sigmoid_bwd")
