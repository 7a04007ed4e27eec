"""C ABI checks that need no GPU: the library loads, exports every function
declared in include/dms.h, and rejects bad configurations and arguments on
the host before any HIP call."""
import ctypes
import os
import re

import pytest

from paper_2506_05345_amd import dms

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "dms.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(dms_[a-z_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    lib = ctypes.CDLL(dms.LIB_PATH)
    names = _declared()
    assert len(names) >= 15
    for n in names:
        assert hasattr(lib, n), n
    # and the binding wraps each of them under the same name
    for n in names:
        assert hasattr(dms, n), n


def _cfg(**kw):
    base = dict(num_layers=2, max_seqs=4, num_kv_heads=2, group_size=2, head_dim=64, window=16,
                page_size=64, num_pages=32, max_pages_per_head=16, max_chunk_tokens=256)
    base.update(kw)
    return dms.make_config(**base)


@pytest.mark.parametrize("kw,code", [
    (dict(window=0), dms.DMS_ERR_INVALID),
    (dict(window=-3), dms.DMS_ERR_INVALID),
    (dict(head_dim=96), dms.DMS_ERR_UNSUPPORTED),
    (dict(head_dim=0), dms.DMS_ERR_INVALID),
    (dict(group_size=17), dms.DMS_ERR_UNSUPPORTED),
    (dict(group_size=0), dms.DMS_ERR_INVALID),
    (dict(page_size=48), dms.DMS_ERR_INVALID),
    (dict(page_size=16), dms.DMS_ERR_INVALID),
    (dict(num_layers=0), dms.DMS_ERR_INVALID),
    (dict(max_seqs=70000), dms.DMS_ERR_INVALID),
    (dict(num_pages=0), dms.DMS_ERR_INVALID),
    (dict(max_chunk_tokens=-1), dms.DMS_ERR_INVALID),
    (dict(softmax_scale=float("nan")), dms.DMS_ERR_INVALID),
    (dict(softmax_scale=float("inf")), dms.DMS_ERR_INVALID),
    (dict(eviction=2), dms.DMS_ERR_INVALID),
    (dict(eviction=-1), dms.DMS_ERR_INVALID),
    (dict(decision_source=2), dms.DMS_ERR_INVALID),
    (dict(decision_source=1, decision_bias=float("nan")), dms.DMS_ERR_INVALID),
    (dict(decision_source=1, decision_bias=float("inf")), dms.DMS_ERR_INVALID),
    (dict(kv_format=3), dms.DMS_ERR_INVALID),
    (dict(quest_page_budget=-1), dms.DMS_ERR_INVALID),
    (dict(quest_page_budget=17), dms.DMS_ERR_INVALID),                     # > max_pages_per_head
    (dict(quest_page_budget=4, max_pages_per_head=5000), dms.DMS_ERR_UNSUPPORTED),
    (dict(kv_format=-1), dms.DMS_ERR_INVALID),
    # split-K partial accumulators past 2 GiB (32-bit buffer offsets), for every page format
    (dict(max_seqs=65536, num_kv_heads=8, group_size=16, head_dim=128), dms.DMS_ERR_UNSUPPORTED),
    (dict(max_seqs=65536, num_kv_heads=8, group_size=16, head_dim=128, kv_format=1),
     dms.DMS_ERR_UNSUPPORTED),
    (dict(max_seqs=32768, num_kv_heads=16, group_size=16, head_dim=64), dms.DMS_ERR_UNSUPPORTED),
    (dict(max_seqs=65536, num_kv_heads=1, group_size=16, head_dim=576, kv_format=2),
     dms.DMS_ERR_UNSUPPORTED),
    (dict(max_seqs=8192, num_kv_heads=1, group_size=128, head_dim=576, kv_format=2),
     dms.DMS_ERR_UNSUPPORTED),
])
def test_bad_configuration(kw, code):
    rc = dms.lib().dms_layout(ctypes.byref(_cfg(**kw)), None, None, None, None)
    assert rc == code


# Largest-partials configurations below the 2 GiB bound: (U + S * Hkv) * g * row * 4
# bytes, U = 8192 decode waves (1024 work units for latent rows).
@pytest.mark.parametrize("kw", [
    dict(max_seqs=4096, num_kv_heads=8, group_size=16, head_dim=128),
    dict(max_seqs=65536, num_kv_heads=8, group_size=1, head_dim=128, kv_format=1),
    dict(max_seqs=8192, num_kv_heads=1, group_size=16, head_dim=576, kv_format=2),
    dict(max_seqs=60000, num_kv_heads=1, group_size=16, head_dim=576, kv_format=2),
    dict(max_seqs=4096, num_kv_heads=1, group_size=128, head_dim=576, kv_format=2),
])
def test_partial_area_just_below_the_bound_is_accepted(kw):
    cfg = _cfg(**kw)
    latent = kw.get("kv_format") == 2
    row, units = (512, 1024) if latent else (kw["head_dim"], 8192)
    need = (units + cfg.max_seqs * cfg.num_kv_heads) * cfg.group_size * row * 4
    assert need < 2 ** 31
    m, p, w, pg = dms.dms_layout(cfg)
    assert w >= need


def test_layout_sizes():
    m, p, w, pg = dms.dms_layout(_cfg())
    assert pg == 2 * 64 * 64 * 2 and p == 32 * pg
    o = dms.dms_state_layout(_cfg())
    assert m == o.layer0 + 2 * o.layer_stride
    # arrays are disjoint and ordered inside a layer's region
    offs = [o.pos, o.len, o.ring, o.page_table, o.slot_meta, o.stack, o.top]
    assert offs == sorted(offs) and o.top < o.layer_stride


def test_host_side_argument_errors_change_nothing():
    # fake device pointers: every call below must fail validation before any
    # HIP call, so nothing is dereferenced
    cfg = _cfg()
    L = dms.lib()
    assert L.dms_create(ctypes.byref(cfg), None, (ctypes.c_void_p * 2)(1, 2), 3,
                        ctypes.byref(ctypes.c_void_p())) == dms.DMS_ERR_INVALID
    assert L.dms_create(ctypes.byref(cfg), 1, (ctypes.c_void_p * 2)(1, None), 3,
                        ctypes.byref(ctypes.c_void_p())) == dms.DMS_ERR_INVALID
    ctx = dms.dms_create(cfg, 0x1000, [0x2000, 0x3000], 0x4000)
    try:
        P = 0x100
        assert L.dms_append(ctx, 2, 1, P, P, P, P, None) == dms.DMS_ERR_INVALID      # layer
        assert L.dms_append(ctx, -1, 1, P, P, P, P, None) == dms.DMS_ERR_INVALID
        assert L.dms_append(ctx, 0, 0, P, P, P, P, None) == dms.DMS_ERR_INVALID      # n
        assert L.dms_append(ctx, 0, 5, P, P, P, P, None) == dms.DMS_ERR_INVALID      # n > max_seqs
        assert L.dms_append(ctx, 0, 1, None, P, P, P, None) == dms.DMS_ERR_INVALID   # seq ids
        assert L.dms_append(ctx, 0, 1, P, None, P, P, None) == dms.DMS_ERR_INVALID
        assert L.dms_decode(ctx, 0, 1, P, P, None, None) == dms.DMS_ERR_INVALID      # out
        assert L.dms_decode_step(ctx, 0, 1, P, P, P, P, None, P, None) == dms.DMS_ERR_INVALID
        # chunk sizes: total over max_chunk_tokens, max_seqlen > total, missing cu
        assert L.dms_append_chunk(ctx, 0, 1, P, P, 257, 257, P, P, P, None) == dms.DMS_ERR_INVALID
        assert L.dms_append_chunk(ctx, 0, 1, P, P, 10, 11, P, P, P, None) == dms.DMS_ERR_INVALID
        assert L.dms_append_chunk(ctx, 0, 1, P, None, 10, 10, P, P, P, None) == dms.DMS_ERR_INVALID
        assert L.dms_append_chunk(ctx, 0, 1, P, P, -1, 0, P, P, P, None) == dms.DMS_ERR_INVALID
        assert L.dms_append_chunk(ctx, 0, 1, P, P, 0, 0, P, P, P, None) == dms.DMS_OK  # empty: no-op
        assert L.dms_prefill_chunk(ctx, 0, 1, P, P, 10, 10, None, P, P, P, P, None) == dms.DMS_ERR_INVALID
        assert L.dms_seq_reset(ctx, 2, 1, P, None) == dms.DMS_ERR_INVALID
        assert L.dms_seq_reset(ctx, -2, 1, P, None) == dms.DMS_ERR_INVALID
        assert L.dms_retained_lengths(ctx, 0, 1, P, None, None) == dms.DMS_ERR_INVALID
        assert L.dms_export_state(ctx, 0, P, 4, None) == dms.DMS_ERR_INVALID          # too small
        assert L.dms_profile_start(ctx, 0) == dms.DMS_ERR_INVALID
        assert L.dms_profile_stop(ctx, None, None) == dms.DMS_ERR_INVALID            # no session
        assert L.dms_status(None, None) == dms.DMS_ERR_INVALID
    finally:
        dms.dms_destroy(ctx)
    assert L.dms_destroy(None) == dms.DMS_ERR_INVALID


def test_decision_source_selects_the_entry_points():
    """Caller-flag and query-decision entry points reject the other mode on
    the host (fake pointers: nothing may be launched or dereferenced)."""
    L = dms.lib()
    P = 0x100
    ctx = dms.dms_create(_cfg(), 0x1000, [0x2000, 0x3000], 0x4000)
    try:
        assert L.dms_decode_step_q(ctx, 0, 1, P, P, P, P, None, P, None) == dms.DMS_ERR_INVALID
        assert L.dms_prefill_chunk_q(ctx, 0, 1, P, P, 10, 10, P, P, P, None, P, None) == dms.DMS_ERR_INVALID
    finally:
        dms.dms_destroy(ctx)
    ctx = dms.dms_create(_cfg(decision_source=dms.DMS_DECIDE_QUERY, eviction=dms.DMS_EVICT_IMMEDIATE),
                         0x1000, [0x2000, 0x3000], 0x4000)
    try:
        assert L.dms_decode_step(ctx, 0, 1, P, P, P, P, P, P, None) == dms.DMS_ERR_INVALID
        assert L.dms_prefill_chunk(ctx, 0, 1, P, P, 10, 10, P, P, P, P, P, None) == dms.DMS_ERR_INVALID
        # query mode: q, k, v and out are required; decisions_out may be NULL
        assert L.dms_decode_step_q(ctx, 0, 1, P, None, P, P, None, P, None) == dms.DMS_ERR_INVALID
        assert L.dms_decode_step_q(ctx, 0, 1, P, P, P, P, None, None, None) == dms.DMS_ERR_INVALID
        assert L.dms_prefill_chunk_q(ctx, 0, 1, P, P, 10, 10, None, P, P, None, P, None) == dms.DMS_ERR_INVALID
        assert L.dms_prefill_chunk_q(ctx, 0, 1, P, P, 0, 0, P, P, P, None, P, None) == dms.DMS_OK
    finally:
        dms.dms_destroy(ctx)


def test_error_strings():
    for code in (0, -1, -2, -3, -4, -5, -6):
        assert dms.dms_strerror(code) and dms.dms_strerror(code) != "unknown error code"
    assert dms.dms_strerror(-99) == "unknown error code"


def _bf16_offsets(j, e, D):
    """Byte offsets of key and value element (j, e) in a bf16 tile (include/dms.h)."""
    h, r = (j // 4) % 2, 4 * (j // 8) + j % 4
    k = ((((e // 32) * 2 + h) * 4 + (e // 8) % 4) * 16 + r) * 16 + (e % 8) * 2
    v = 64 * D + (((e // 16) * 4 + j // 8) * 16 + e % 16) * 16 + (j % 8) * 2
    return k, v


def test_bf16_tile_offsets_are_a_bijection():
    # every key and value element of a tile has its own 2-byte cell, and the
    # cells fill the 128 * D bytes exactly
    import numpy as np
    for D in (64, 128):
        j = np.arange(32)[:, None]
        e = np.arange(D)[None, :]
        k, v = _bf16_offsets(j, e, D)
        cells = np.concatenate([k.ravel(), v.ravel()])
        assert (cells % 2 == 0).all()
        assert np.array_equal(np.sort(cells), np.arange(0, 128 * D, 2))
        # the 8 dims of one key piece (and 8 slots of one value piece) are contiguous
        assert (np.diff(k.reshape(32, D // 8, 8), axis=2) == 2).all()
        assert (np.diff(v.T.reshape(D, 4, 8), axis=2) == 2).all()


def test_unpack_page_matches_documented_offsets():
    # element (j, e) of tile t at the documented key / value offsets
    import numpy as np
    P, D = 64, 128
    words = np.zeros(P * D * 2, np.uint16)
    for s in (0, 5, 12, 31, 32, 45, 63):
        t, j = divmod(s, 32)
        for e in (0, 7, 9, 31, 32, 100, 127):
            base = t * 128 * D
            ko, vo = _bf16_offsets(j, e, D)
            words[(base + ko) // 2] = 1000 + s * 200 + e
            words[(base + vo) // 2] = 3 * (1000 + s * 200 + e)
    k, v = dms.unpack_page(words, P, D)
    for s in (0, 5, 12, 31, 32, 45, 63):
        for e in (0, 7, 9, 31, 32, 100, 127):
            assert k[s, e] == 1000 + s * 200 + e
            assert v[s, e] == 3 * (1000 + s * 200 + e)


def _tcfg(**kw):
    base = dict(batch=2, seq_len=100, num_kv_heads=2, group_size=4, head_dim=128, window=16,
                softmax_scale=0.0)
    base.update(kw)
    return dms.make_train_config(**base)


@pytest.mark.parametrize("kw,code", [
    (dict(batch=0), dms.DMS_ERR_INVALID),
    (dict(seq_len=0), dms.DMS_ERR_INVALID),
    (dict(num_kv_heads=0), dms.DMS_ERR_INVALID),
    (dict(group_size=0), dms.DMS_ERR_INVALID),
    (dict(group_size=17), dms.DMS_ERR_UNSUPPORTED),
    (dict(head_dim=64), dms.DMS_ERR_UNSUPPORTED),
    (dict(window=0), dms.DMS_ERR_INVALID),
    (dict(softmax_scale=float("nan")), dms.DMS_ERR_INVALID),
    (dict(softmax_scale=float("inf")), dms.DMS_ERR_INVALID),
    (dict(batch=1 << 20, seq_len=1 << 20), dms.DMS_ERR_INVALID),
    (dict(batch=40000, num_kv_heads=2, seq_len=1), dms.DMS_ERR_INVALID),
])
def test_bad_train_configuration(kw, code):
    rc = dms.lib().dms_train_workspace(ctypes.byref(_tcfg(**kw)), None)
    assert rc == code


def test_train_workspace_and_host_side_errors():
    n = dms.dms_train_workspace(_tcfg())
    # at least the K and V tiles of every head, padded to 32 tokens
    assert n >= 2 * 2 * 2 * 4 * 128 * 128
    assert dms.dms_train_workspace(_tcfg(seq_len=200)) > n
    assert dms.dms_train_workspace(_tcfg(softmax_scale=-1.0)) == n
    L = dms.lib()
    assert L.dms_train_attention_fwd(None, *([None] * 8)) == dms.DMS_ERR_INVALID
    assert L.dms_train_attention_fwd(ctypes.byref(_tcfg()), *([None] * 8)) == dms.DMS_ERR_INVALID
    assert L.dms_train_attention_bwd(ctypes.byref(_tcfg()), *([None] * 13)) == dms.DMS_ERR_INVALID
    for fn in (L.dms_gumbel_sigmoid_fwd, L.dms_gumbel_sigmoid_bwd):
        assert fn(-1, None, None, ctypes.c_float(1.0), None, None) == dms.DMS_ERR_INVALID
        assert fn(4, None, None, ctypes.c_float(0.0), None, None) == dms.DMS_ERR_INVALID
        assert fn(4, None, None, ctypes.c_float(float("nan")), None, None) == dms.DMS_ERR_INVALID
        assert fn(4, None, None, ctypes.c_float(1.0), None, None) == dms.DMS_ERR_INVALID
        assert fn(0, None, None, ctypes.c_float(1.0), None, None) == dms.DMS_OK


def test_fp8_pages_layout_and_host_checks():
    """FP8 pages are P/32 tiles of 64 d + 256 bytes laid out as include/dms.h
    documents."""
    import numpy as np
    for D in (64, 128):
        for P in (32, 64, 256):
            _, pool, _, pg = dms.dms_layout(_cfg(kv_format=dms.DMS_KV_FP8, head_dim=D, page_size=P))
            assert pg == P // 32 * (64 * D + 256) and pool == pg * _cfg().num_pages
    # documented offsets (include/dms.h) -> unpack_page_fp8
    P, D = 64, 128
    raw = np.zeros(P // 32 * (64 * D + 256), np.uint8)
    for s_ in (0, 5, 31, 32, 63):
        t, j = divmod(s_, 32)
        base = t * (64 * D + 256)
        h, r = (j // 4) % 2, 4 * (j // 8) + j % 4
        for e in (0, 7, 31, 32, 64, 100, 127):
            ko = (e // 64) * 2048 + h * 1024 + (16 * ((e // 8) % 4) + r) * 16 + 8 * ((e // 32) % 2) + e % 8
            vo = 32 * D + (e // 32) * 1024 + (16 * (j // 8) + e % 16) * 16 + 8 * ((e // 16) % 2) + j % 8
            raw[base + ko] = (s_ + e) % 251
            raw[base + vo] = (3 * s_ + e) % 251
        so = 64 * D + (j // 8) * 64 + (j % 8) * 4
        raw[base + so: base + so + 4] = np.array([2.0 ** -s_], np.float32).view(np.uint8)
        raw[base + so + 32: base + so + 36] = np.array([2.0 ** s_], np.float32).view(np.uint8)
    k, v, ks, vs = dms.unpack_page_fp8(raw, P, D)
    for s_ in (0, 5, 31, 32, 63):
        assert ks[s_] == 2.0 ** -s_ and vs[s_] == 2.0 ** s_
        for e in (0, 7, 31, 32, 64, 100, 127):
            assert k[s_, e] == (s_ + e) % 251 and v[s_, e] == (3 * s_ + e) % 251


def test_quest_layout_and_host_checks():
    """Page bounds live in each layer's state only with a budget; the
    selection export rejects contexts without one (fake pointers)."""
    o0 = dms.dms_state_layout(_cfg())
    o1 = dms.dms_state_layout(_cfg(quest_page_budget=4))
    assert o0.page_bounds == 0 and o1.page_bounds > o1.top
    assert o1.layer_stride - o0.layer_stride >= _cfg().num_pages * 2 * 64 * 2
    L = dms.lib()
    P = 0x100
    ctx = dms.dms_create(_cfg(), 0x1000, [0x2000, 0x3000], 0x4000)
    try:
        assert L.dms_quest_selection(ctx, 1, P, P, None) == dms.DMS_ERR_INVALID
    finally:
        dms.dms_destroy(ctx)
    ctx = dms.dms_create(_cfg(quest_page_budget=4), 0x1000, [0x2000, 0x3000], 0x4000)
    try:
        assert L.dms_quest_selection(ctx, 0, P, P, None) == dms.DMS_ERR_INVALID
        assert L.dms_quest_selection(ctx, 5, P, P, None) == dms.DMS_ERR_INVALID   # > max_seqs
        assert L.dms_quest_selection(ctx, 1, None, P, None) == dms.DMS_ERR_INVALID
    finally:
        dms.dms_destroy(ctx)
    assert L.dms_quest_selection(None, 1, P, P, None) == dms.DMS_ERR_INVALID



def test_latent_pages_layout_and_host_checks():
    """Latent-attention pools: one KV head of 576-dim rows, P/32 tiles of
    64 * 576 bytes in the bf16 key order; the unsupported combinations are
    refused on the host."""
    import numpy as np
    mla = dict(kv_format=dms.DMS_KV_MLA, head_dim=dms.MLA_ROW_DIM, num_kv_heads=1, group_size=16)
    for P in (32, 64, 256):
        _, pool, ws, pg = dms.dms_layout(_cfg(page_size=P, **mla))
        assert pg == P * dms.MLA_ROW_DIM * 2 and pool == pg * _cfg().num_pages
    for kw in (dict(head_dim=128), dict(num_kv_heads=2), dict(quest_page_budget=2),
               dict(decision_source=dms.DMS_DECIDE_QUERY)):
        rc = dms.lib().dms_layout(ctypes.byref(_cfg(**{**mla, **kw})), None, None, None, None)
        assert rc == dms.DMS_ERR_UNSUPPORTED, kw
    # 576-dim rows only exist in latent pools
    rc = dms.lib().dms_layout(ctypes.byref(_cfg(head_dim=dms.MLA_ROW_DIM)), None, None, None, None)
    assert rc == dms.DMS_ERR_UNSUPPORTED
    # up to 128 query heads share a latent row (DeepSeek-V2), in groups of 16
    lat = {k: v for k, v in mla.items() if k != "group_size"}
    for g in (17, 40, 128):
        rc = dms.lib().dms_layout(ctypes.byref(_cfg(group_size=g, **lat)), None, None, None, None)
        assert rc == dms.DMS_OK, g
    rc = dms.lib().dms_layout(ctypes.byref(_cfg(group_size=129, **lat)), None, None, None, None)
    assert rc == dms.DMS_ERR_UNSUPPORTED
    # the workspace grows with the group: partial rows, (max, sum) slots of
    # the group rounded up to 16, one arrival counter per head group
    ws16 = dms.dms_layout(_cfg(group_size=16, **lat))[2]
    ws128 = dms.dms_layout(_cfg(group_size=128, **lat))[2]
    assert ws128 > 7 * ws16
    # documented offsets (include/dms.h): the bf16 key formula, tiles of 64 d bytes
    P, D = 64, dms.MLA_ROW_DIM
    words = np.zeros(P * D, np.uint16)
    for s_ in (0, 5, 31, 32, 63):
        t, j = divmod(s_, 32)
        h, r = (j // 4) % 2, 4 * (j // 8) + j % 4
        for e in (0, 7, 31, 32, 100, 511, 512, 575):
            off = t * 64 * D + ((((e // 32) * 2 + h) * 4 + (e // 8) % 4) * 16 + r) * 16 + (e % 8) * 2
            words[off // 2] = 1 + s_ * 1000 + e
    rows = dms.unpack_page_mla(words, P, D)
    for s_ in (0, 5, 31, 32, 63):
        for e in (0, 7, 31, 32, 100, 511, 512, 575):
            assert rows[s_, e] == 1 + s_ * 1000 + e
    # latent pools: prefill with caller decisions takes no value rows (v may be
    # NULL, the other arguments may not); decisions from q are refused, all
    # before any device work
    L = dms.lib()
    ctx = dms.dms_create(_cfg(**mla), 0x1000, [0x2000, 0x3000], 0x4000)
    try:
        X = 0x100
        assert L.dms_prefill_chunk(ctx, 0, 1, X, X, 4, 4, None, X, None, X, X, None) == dms.DMS_ERR_INVALID
        assert L.dms_prefill_chunk(ctx, 0, 1, X, X, 4, 4, X, None, None, X, X, None) == dms.DMS_ERR_INVALID
        assert L.dms_prefill_chunk_q(ctx, 0, 1, X, X, 4, 4, X, X, None, X, X, None) == dms.DMS_ERR_UNSUPPORTED
    finally:
        dms.dms_destroy(ctx)


def test_binding_checks_tensor_arguments_before_the_call():
    """The Python binding refuses tensors of the wrong element type, on the
    host, non-contiguous or too small before handing their addresses to the
    library (which cannot see them); raw integer addresses pass through."""
    import torch
    cfg = _cfg()    # Hkv = 2, g = 2, d = 64
    ctx = dms.dms_create(cfg, 0x1000, [0x2000, 0x3000], 0x4000)
    try:
        n = 2
        sid = torch.zeros(n, dtype=torch.int32)
        q = torch.zeros((n, 4, 64), dtype=torch.bfloat16)
        k = torch.zeros((n, 2, 64), dtype=torch.bfloat16)
        fl = torch.zeros((n, 2), dtype=torch.uint8)
        out = torch.zeros((n, 4, 64), dtype=torch.float32)

        def code(fn, *a):
            with pytest.raises(dms.DmsError) as e:
                fn(*a)
            return e.value.code, str(e.value)

        # element types
        c, msg = code(dms.dms_decode_step, ctx, 0, n, sid.to(torch.int64), q, k, k, fl, out, 0)
        assert c == dms.DMS_ERR_INVALID and "seq_ids must be int32" in msg
        c, msg = code(dms.dms_decode_step, ctx, 0, n, sid, q.float(), k, k, fl, out, 0)
        assert c == dms.DMS_ERR_INVALID and ": q must be bf16" in msg
        c, msg = code(dms.dms_decode_step, ctx, 0, n, sid, q, k, k, fl.to(torch.int32), out, 0)
        assert "flags must be uint8" in msg
        c, msg = code(dms.dms_decode_step, ctx, 0, n, sid, q, k, k, fl, out.to(torch.bfloat16), 0)
        assert "out must be float32" in msg
        c, msg = code(dms.dms_train_attention_fwd, dms.make_train_config(1, 4, 2, 2, 128, 2),
                      q, k, k, out, out, out.to(torch.bfloat16), 0x100)
        assert "lse must be float32" in msg
        # right types, but host memory
        c, msg = code(dms.dms_decode_step, ctx, 0, n, sid, q, k, k, fl, out, 0)
        assert c == dms.DMS_ERR_INVALID and "GPU" in msg
        # raw addresses are not inspected (the library validates nulls and sizes it can see)
        assert dms.lib().dms_decode_step(ctx, 0, n, 0x100, 0x100, 0x100, 0x100, 0x100, None,
                                         None) == dms.DMS_ERR_INVALID
    finally:
        dms.dms_destroy(ctx)
    assert ctx not in dms._CTX_CFG


@pytest.mark.gpu
def test_binding_refuses_small_or_strided_gpu_tensors():
    import torch
    cfg = _cfg()
    cache = dms.DmsCache(cfg, device="cuda")
    try:
        n = 2
        sid = torch.arange(n, dtype=torch.int32, device="cuda")
        q = torch.zeros((n, 4, 64), dtype=torch.bfloat16, device="cuda")
        k = torch.zeros((n, 2, 64), dtype=torch.bfloat16, device="cuda")
        fl = torch.zeros((n, 2), dtype=torch.uint8, device="cuda")
        out = torch.zeros((n, 4, 64), dtype=torch.float32, device="cuda")
        with pytest.raises(dms.DmsError, match="needs"):
            dms.dms_decode_step(cache.ctx, 0, n, sid, q[:1], k, k, fl, out)
        with pytest.raises(dms.DmsError, match="contiguous"):
            dms.dms_decode_step(cache.ctx, 0, n, sid, q, k, k, fl,
                                torch.zeros((n, 64, 4), device="cuda").transpose(1, 2))
        with pytest.raises(dms.DmsError, match="needs"):
            dms.dms_append_chunk(cache.ctx, 0, 1, sid[:1], sid[:1], 2, 2, k, k, fl)  # cu too short
        torch.cuda.synchronize()
        assert dms.dms_status(cache.ctx) == 0
    finally:
        cache.close()
