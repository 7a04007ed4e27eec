"""GPU parity of the DMS-masked chunked prefill (dms_prefill_chunk): outputs
of every chunk query against dense masked attention over the full history
(max-abs 1e-2), and the committed state against the oracle replay (bit-exact),
for several group sizes, head sizes, windows, eviction rates and chunkings."""
import numpy as np
import pytest

from dms_testlib import (ATOL, SeqInputs, bf16_to_f32, compare_pool, compare_pool_fp8, compare_state,
                         to_dev)
from oracle import PagedKVOracle, dense_dms_attention, fake_quantize_fp8

pytestmark = pytest.mark.gpu


def _run(cfg_kw, seqs, lens, chunks, seed, p, q_scale=1.0, override=None, fp8=False, nan_pools=False):
    """Prefill every sequence to lens[s] tokens in calls of chunks[c] tokens
    per sequence; check each call's outputs and the state after it.  With
    fp8 the pages are E4M3 and every key and value (cached or in the chunk)
    is attended in its quantized form; pools and workspace start as NaN
    bytes (also with nan_pools for bf16 pages: the slots past a head's live
    length, read with its last cached tile, then hold NaNs)."""
    import torch
    from paper_2506_05345_amd import dms
    cfg = dms.make_config(kv_format=dms.DMS_KV_FP8 if fp8 else dms.DMS_KV_BF16, **cfg_kw)
    cache = dms.DmsCache(cfg)
    if fp8 or nan_pools:
        for pl in cache.pools:
            pl.fill_(0xFF)
        cache.workspace.fill_(0xFF)
        dms.dms_init_state(cache.ctx)
        torch.cuda.synchronize()
    kvq = fake_quantize_fp8 if fp8 else (lambda x: x)
    H, g, D, w = cfg.num_kv_heads, cfg.group_size, cfg.head_dim, cfg.window
    inp = {s: SeqInputs(seed, 0, s, lens[s], H, g, D, p, q_scale=q_scale) for s in seqs}
    if override:
        override(inp)
    orc = PagedKVOracle(cfg.max_seqs, H, w, cfg.page_size, cfg.num_pages,
                        cfg.max_pages_per_head, D, kv_format="fp8" if fp8 else "bf16")
    cur = {s: 0 for s in seqs}
    worst = 0.0
    ci = 0
    while any(cur[s] < lens[s] for s in seqs):
        C = chunks[ci % len(chunks)]
        ci += 1
        ls = [min(C, lens[s] - cur[s]) for s in seqs]
        cu = np.concatenate([[0], np.cumsum(ls)]).astype(np.int32)
        sl = lambda arr, s, l: arr[cur[s]:cur[s] + l]
        q = np.concatenate([sl(inp[s].q, s, l) for s, l in zip(seqs, ls)])
        k = np.concatenate([sl(inp[s].k, s, l) for s, l in zip(seqs, ls)])
        v = np.concatenate([sl(inp[s].v, s, l) for s, l in zip(seqs, ls)])
        f = np.concatenate([sl(inp[s].flags, s, l) for s, l in zip(seqs, ls)])
        out = torch.full((int(cu[-1]), H * g, D), float("nan"), device="cuda")
        dms.dms_prefill_chunk(cache.ctx, 0, len(seqs), to_dev(np.array(seqs, np.int32)),
                              to_dev(cu), int(cu[-1]), int(max(ls)), to_dev(q), to_dev(k),
                              to_dev(v), to_dev(f), out)
        torch.cuda.synchronize()
        assert dms.dms_status(cache.ctx) == 0
        got = out.cpu().numpy()
        for i, (s, l) in enumerate(zip(seqs, ls)):
            if l == 0:
                continue
            tq = np.arange(cur[s], cur[s] + l)
            ref = dense_dms_attention(bf16_to_f32(inp[s].q[tq]), kvq(bf16_to_f32(inp[s].k[:tq[-1] + 1])),
                                      kvq(bf16_to_f32(inp[s].v[:tq[-1] + 1])), inp[s].flags[:tq[-1] + 1],
                                      w, g, t_query=tq)
            err = np.abs(got[cu[i]:cu[i + 1]] - ref).max()
            worst = max(worst, err)
            assert err <= ATOL, (s, cur[s], err)
        orc.append_chunk(seqs, [sl(inp[s].flags, s, l) for s, l in zip(seqs, ls)],
                         [bf16_to_f32(sl(inp[s].k, s, l)) for s, l in zip(seqs, ls)],
                         [bf16_to_f32(sl(inp[s].v, s, l)) for s, l in zip(seqs, ls)])
        for s, l in zip(seqs, ls):
            cur[s] += l
        compare_state(cache.export(0), orc, seqs)
    if fp8:
        compare_pool_fp8(cache, orc, seqs)
    else:
        compare_pool(cache, 0, cache.export(0), seqs, inp)
    cache.close()
    return worst


@pytest.mark.parametrize("chunks", [[512], [37], [200, 1, 64, 311]])
def test_tiny_config_prefill(chunks):
    """1 sequence, 2 KV heads x group 2, d=64, 512 tokens, w=16, p=1/2, seed 0."""
    worst = _run(dict(num_layers=1, max_seqs=1, num_kv_heads=2, group_size=2, head_dim=64,
                      window=16, page_size=64, num_pages=32, max_pages_per_head=16,
                      max_chunk_tokens=512), [0], {0: 512}, chunks, 0, 0.5)
    print(f"max abs err {worst:.3e}")


@pytest.mark.parametrize("d,g,w,P,p", [
    (128, 5, 256, 64, 0.875), (128, 6, 8, 32, 0.875), (128, 7, 20, 64, 0.75),
    (64, 1, 1, 32, 0.5), (64, 3, 5, 128, 0.9), (128, 8, 64, 64, 0.5),
    (128, 16, 33, 256, 0.875), (64, 2, 16, 64, 0.0), (128, 4, 12, 64, 1.0)])
def test_ragged_prefill(d, g, w, P, p):
    H = 2
    seqs = [2, 0, 3]
    lens = {2: 900, 0: 130, 3: 611}
    _run(dict(num_layers=1, max_seqs=4, num_kv_heads=H, group_size=g, head_dim=d, window=w,
              page_size=P, num_pages=300, max_pages_per_head=64, max_chunk_tokens=3 * 400),
         seqs, lens, [400, 77], 31, p)


@pytest.mark.parametrize("d,g,w,P,chunks", [(128, 5, 256, 64, [400, 77]), (64, 3, 5, 32, [37, 200]),
                                            (128, 8, 16, 256, [129])])
def test_ragged_prefill_nan_pools(d, g, w, P, chunks):
    """bf16 pages over NaN bytes: every ragged last cache tile brings stale
    NaN rows into LDS, which must leave no trace in the outputs."""
    H = 2
    seqs = [2, 0, 3]
    lens = {2: 700, 0: 95, 3: 411}
    _run(dict(num_layers=1, max_seqs=4, num_kv_heads=H, group_size=g, head_dim=d, window=w,
              page_size=P, num_pages=300, max_pages_per_head=64, max_chunk_tokens=3 * 400),
         seqs, lens, chunks, 57, 0.75, nan_pools=True)


def test_prefill_peaked_and_needle():
    def needle(inp):
        x = inp[0]
        x.k[:] = 0
        x.q[:] = 0
        x.q[:, :, 0] = 0x447A      # 1000.0: every query looks for dim 0
        x.k[10, 0, 0] = 0x3F80     # kept needle
        x.flags[10] = 0
        x.v[10, 0, :] = 0x4000
        x.k[300, 0, 0] = 0x3F80    # flagged needle, leaves the window at 316
        x.flags[300] = 1
        x.v[300, 0, :] = 0xC000
    _run(dict(num_layers=1, max_seqs=1, num_kv_heads=1, group_size=4, head_dim=128, window=16,
              page_size=64, num_pages=64, max_pages_per_head=16, max_chunk_tokens=512),
         [0], {0: 700}, [256, 100], 41, 0.875, override=needle)
    _run(dict(num_layers=1, max_seqs=1, num_kv_heads=2, group_size=5, head_dim=128, window=64,
              page_size=64, num_pages=64, max_pages_per_head=16, max_chunk_tokens=512),
         [0], {0: 600}, [300], 43, 0.875, q_scale=8.0)


def test_prefill_then_decode_matches_decode_only_path():
    """The state after dms_prefill_chunk equals the state after
    dms_append_chunk of the same tokens, and decode continues correctly."""
    import torch
    from paper_2506_05345_amd import dms
    kw = dict(num_layers=2, max_seqs=2, num_kv_heads=2, group_size=3, head_dim=128, window=32,
              page_size=64, num_pages=64, max_pages_per_head=16, max_chunk_tokens=600)
    cfg = dms.make_config(**kw)
    cache = dms.DmsCache(cfg)
    seqs = [1, 0]
    inp = {s: SeqInputs(51, 0, s, 400, 2, 3, 128, 0.8) for s in seqs}
    cu = np.array([0, 300, 600], np.int32)
    cat = lambda name: np.concatenate([getattr(inp[s], name)[:300] for s in seqs])
    out = torch.empty((600, 6, 128), device="cuda")
    sid = to_dev(np.array(seqs, np.int32))
    dms.dms_prefill_chunk(cache.ctx, 0, 2, sid, to_dev(cu), 600, 300, to_dev(cat("q")),
                          to_dev(cat("k")), to_dev(cat("v")), to_dev(cat("flags")), out)
    dms.dms_append_chunk(cache.ctx, 1, 2, sid, to_dev(cu), 600, 300, to_dev(cat("k")),
                         to_dev(cat("v")), to_dev(cat("flags")))
    torch.cuda.synchronize()
    assert dms.dms_status(cache.ctx) == 0
    a, b = cache.export(0), cache.export(1)
    for f in ("pos", "L", "ring_slot", "ring_flag", "page_table", "stack"):
        assert np.array_equal(getattr(a, f), getattr(b, f)), f
    for s in seqs:          # slot owners are defined below L only
        for h in range(2):
            L = a.L[s, h]
            assert np.array_equal(a.slot_pos[s, h, :L], b.slot_pos[s, h, :L])
            assert np.array_equal(a.slot_flag[s, h, :L], b.slot_flag[s, h, :L])
    for t in range(300, 310):
        outs = []
        for layer in (0, 1):
            o = torch.empty((2, 6, 128), device="cuda")
            st = lambda name: to_dev(np.stack([getattr(inp[s], name)[t] for s in seqs]))
            dms.dms_decode_step(cache.ctx, layer, 2, sid, st("q"), st("k"), st("v"), st("flags"), o)
            outs.append(o)
        torch.cuda.synchronize()
        assert torch.equal(outs[0], outs[1])
    cache.close()


@pytest.mark.parametrize("d,g,w,P,p,chunks", [
    (128, 5, 256, 64, 0.875, [400, 77]), (64, 2, 16, 32, 0.5, [37]), (128, 16, 33, 256, 0.75, [200, 1, 311]),
    (64, 7, 1, 128, 0.9, [400])])
def test_ragged_prefill_fp8(d, g, w, P, p, chunks):
    """FP8 pages: cached keys come from E4M3 pages (ragged last tiles over NaN
    bytes), in-chunk keys from E4M3 workspace tiles; codes of the committed
    slots bit-exact."""
    H = 2
    seqs = [2, 0, 3]
    lens = {2: 900, 0: 130, 3: 611}
    _run(dict(num_layers=1, max_seqs=4, num_kv_heads=H, group_size=g, head_dim=d, window=w,
              page_size=P, num_pages=300, max_pages_per_head=64, max_chunk_tokens=3 * 400),
         seqs, lens, chunks, 33, p, fp8=True)


def test_prefill_fp8_peaked():
    _run(dict(num_layers=1, max_seqs=1, num_kv_heads=2, group_size=5, head_dim=128, window=64,
              page_size=64, num_pages=64, max_pages_per_head=16, max_chunk_tokens=512),
         [0], {0: 600}, [300], 43, 0.875, q_scale=8.0, fp8=True)


def test_prefill_many_heads_unordered_work_items():
    """70 sequences x 8 KV heads: 560 (sequence, head) rows, more than the
    head ranking takes, so grid rows keep the call's order; 2 query blocks
    per row give 1120 work items, more than the chip holds workgroups, so
    the resident workgroups take most items from the counter."""
    seqs = list(range(70))
    lens = {s: 60 + (s % 7) for s in seqs}
    _run(dict(num_layers=1, max_seqs=70, num_kv_heads=8, group_size=5, head_dim=128, window=32,
              page_size=64, num_pages=70 * 8 * 3, max_pages_per_head=4, max_chunk_tokens=70 * 40),
         seqs, lens, [40], 71, 0.75)


@pytest.mark.parametrize("d,g,fp8", [(64, 16, False), (128, 5, True)])
def test_prefill_ranked_rows_counter_items(d, g, fp8):
    """Few heads but many query blocks: the rows are ranked by work and the
    items outnumber the resident workgroups (800 items at d = 64, g = 16 on
    bf16 pages; 320 at d = 128, g = 5 on FP8 pages, one workgroup per CU);
    unequal histories so the ranking reorders the rows."""
    H = 4 if not fp8 else 8
    seqs = [1, 3, 0, 2]
    lens = {1: 900, 3: 640, 0: 1000, 2: 700}
    chunk = 400 if not fp8 else 500
    _run(dict(num_layers=1, max_seqs=4, num_kv_heads=H, group_size=g, head_dim=d, window=48,
              page_size=64, num_pages=4 * H * 18, max_pages_per_head=18, max_chunk_tokens=4 * chunk),
         seqs, lens, [chunk], 83, 0.8, fp8=fp8)
