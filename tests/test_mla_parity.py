"""GPU parity of decode over a latent-attention (MLA) cache against the CPU
oracle: one KV head of 576-dim rows (512 latent + 64 rotary key), every query
head in its group, outputs of 512 latent dims.  Bookkeeping and stored rows
bit-exact; outputs within 1e-2 max-abs (bf16 rows and queries, fp32
accumulation)."""
import math

import numpy as np
import pytest

import dms_synth as sy
from dms_testlib import ATOL, bf16_to_f32, compare_state, to_dev
from oracle import PagedKVOracle, mla_attention, visible, visible_immediate

pytestmark = pytest.mark.gpu

ROW, LATENT = 576, 512


class MlaInputs:
    """Seeded rows [T, 1, 576], queries [T, g, 576] (bf16 bits) and flags
    [T, 1] of one sequence."""

    def __init__(self, seed, seq, T, g, p):
        pos = np.arange(T)
        self.flags = sy.flags_np(seed, p, 0, seq, np.zeros((1, 1), np.int64), pos[:, None])
        hk, dk = sy.wide_coords(np.zeros((1, 1, 1), np.int64), np.arange(ROW)[None, None, :], ROW)
        hq, dq = sy.wide_coords(np.arange(g)[None, :, None], np.arange(ROW)[None, None, :], ROW)
        pp = pos[:, None, None]
        self.k = sy.token_vectors_np(seed, sy.STREAM_K, 0, seq, hk, pp, dk)
        self.q = sy.token_vectors_np(seed, sy.STREAM_Q, 0, seq, hq, pp, dq)


def _torch():
    import torch
    return torch


def _mk(max_seqs, g, w, P, num_pages, maxp, max_chunk=4096, mode="delayed"):
    from paper_2506_05345_amd import dms
    cfg = dms.make_config(num_layers=1, max_seqs=max_seqs, num_kv_heads=1, group_size=g,
                          head_dim=ROW, window=w, page_size=P, num_pages=num_pages,
                          max_pages_per_head=maxp, max_chunk_tokens=max_chunk,
                          eviction=dms.DMS_EVICT_IMMEDIATE if mode == "immediate" else dms.DMS_EVICT_DELAYED,
                          kv_format=dms.DMS_KV_MLA)
    cache = dms.DmsCache(cfg)
    orc = PagedKVOracle(max_seqs, 1, w, P, num_pages, maxp, ROW, mode=mode)
    return dms, cfg, cache, orc


def _append_chunks(dms, cache, orc, seqs, inp, start, stop, chunk, with_v=False):
    torch = _torch()
    cur = dict(start)
    while any(cur[s] < stop[s] for s in seqs):
        lens = [min(chunk, stop[s] - cur[s]) for s in seqs]
        cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
        fl = np.concatenate([inp[s].flags[cur[s]:cur[s] + l] for s, l in zip(seqs, lens)])
        kk = np.concatenate([inp[s].k[cur[s]:cur[s] + l] for s, l in zip(seqs, lens)])
        sid = to_dev(np.array(seqs, np.int32))
        kd = to_dev(kk)
        dms.dms_append_chunk(cache.ctx, 0, len(seqs), sid, to_dev(cu), int(cu[-1]), int(max(lens)),
                             kd, kd if with_v else None, to_dev(fl))
        rows = [bf16_to_f32(inp[s].k[cur[s]:cur[s] + l]) for s, l in zip(seqs, lens)]
        orc.append_chunk(seqs, [inp[s].flags[cur[s]:cur[s] + l] for s, l in zip(seqs, lens)], rows, rows)
        for s, l in zip(seqs, lens):
            cur[s] += l
        torch.cuda.synchronize()
        assert dms.dms_status(cache.ctx) == 0


def _dense_ref(inp, s, t, w, g):
    """Definition route: masked absorbed attention over the full history."""
    T = t + 1
    rows = bf16_to_f32(inp[s].k[:T, 0]).astype(np.float64)
    mask = np.asarray(visible(t, np.arange(T), inp[s].flags[:T, 0], w), dtype=bool)
    q = bf16_to_f32(inp[s].q[t]).astype(np.float64)
    return mla_attention(q, rows, np.broadcast_to(mask, (g, T)), LATENT, 1.0 / math.sqrt(ROW))


def _decode_steps(dms, cache, orc, seqs, inp, t_from, nsteps, g, dense_every=0):
    torch = _torch()
    cfg = cache.cfg
    sid = to_dev(np.array(seqs, np.int32))
    for step in range(nsteps):
        ts = {s: t_from[s] + step for s in seqs}
        q = np.stack([inp[s].q[ts[s]] for s in seqs])
        k = np.stack([inp[s].k[ts[s]] for s in seqs])
        f = np.stack([inp[s].flags[ts[s]] for s in seqs])
        out = torch.full((len(seqs), g, LATENT), float("nan"), device="cuda")
        dms.dms_decode_step(cache.ctx, 0, len(seqs), sid, to_dev(q), to_dev(k), None, to_dev(f), out)
        torch.cuda.synchronize()
        assert dms.dms_status(cache.ctx) == 0
        kf = bf16_to_f32(k)
        orc.append(seqs, f, kf, kf)
        ref = orc.decode_latent(seqs, bf16_to_f32(q), LATENT)
        got = out.cpu().numpy()
        err = np.abs(got - ref).max()
        assert err <= ATOL, (step, err)
        if dense_every and step % dense_every == 0:
            for i, s in enumerate(seqs):
                dref = _dense_ref(inp, s, ts[s], cfg.window, g)
                assert np.abs(got[i] - dref).max() <= ATOL, (step, s)


def _compare_rows(cache, orc, seqs):
    """Every live slot holds the row bits of the position that owns it."""
    view = cache.export(0)
    P = cache.cfg.page_size
    pages = {}
    for s in seqs:
        L = int(view.L[s, 0])
        for slot in range(L):
            pg = int(view.page_table[s, 0, slot // P])
            if pg not in pages:
                pages[pg] = cache.pool_page_kv(0, pg)[0]
            got = bf16_to_f32(pages[pg][slot % P])
            assert np.array_equal(got, orc.k_store[s, 0, slot].astype(np.float32)), (s, slot)
    return view


@pytest.mark.parametrize("g", [128, 40, 16, 5, 1])
def test_mla_ragged_chunks_then_decode(g):
    """Ragged histories (1 token .. a few thousand) appended in chunks, then
    decode steps that append one row each: state, rows and outputs."""
    lens = [1, 31, 33, 100, 513, 2100]
    seqs = list(range(len(lens)))
    w, P = 32, 64
    dms, cfg, cache, orc = _mk(len(lens), g, w, P, num_pages=len(lens) * 48, maxp=48, max_chunk=2048)
    inp = {s: MlaInputs(17, s, lens[s] + 40, g, 0.5) for s in seqs}
    _append_chunks(dms, cache, orc, seqs, inp, {s: 0 for s in seqs}, {s: lens[s] for s in seqs}, 256)
    view = _compare_rows(cache, orc, seqs)
    compare_state(view, orc, seqs)
    _decode_steps(dms, cache, orc, seqs, inp, {s: lens[s] for s in seqs}, 24, g, dense_every=8)
    view = _compare_rows(cache, orc, seqs)
    compare_state(view, orc, seqs)
    cache.close()


def test_mla_decode_without_append_and_separate_appends():
    """dms_append (no value rows) then dms_decode: the same outputs as the
    fused step; empty sequences give zeros."""
    torch = _torch()
    g, w, P = 16, 16, 32
    lens = [70, 0, 300]
    seqs = [0, 1, 2]
    dms, cfg, cache, orc = _mk(3, g, w, P, num_pages=64, maxp=16)
    inp = {s: MlaInputs(23, s, lens[s] + 8, g, 0.7) for s in seqs}
    live = [s for s in seqs if lens[s] > 0]
    _append_chunks(dms, cache, orc, live, inp, {s: 0 for s in live}, {s: lens[s] for s in live}, 64,
                   with_v=True)
    sid = to_dev(np.array(live, np.int32))
    for step in range(4):
        k = np.stack([inp[s].k[lens[s] + step] for s in live])
        f = np.stack([inp[s].flags[lens[s] + step] for s in live])
        dms.dms_append(cache.ctx, 0, len(live), sid, to_dev(k), None, to_dev(f))
        kf = bf16_to_f32(k)
        orc.append(live, f, kf, kf)
        q = np.stack([inp[s].q[lens[s] + step] for s in seqs])
        out = torch.full((3, g, LATENT), float("nan"), device="cuda")
        dms.dms_decode(cache.ctx, 0, 3, to_dev(np.array(seqs, np.int32)), to_dev(q), out)
        torch.cuda.synchronize()
        assert dms.dms_status(cache.ctx) == 0
        got = out.cpu().numpy()
        assert np.all(got[1] == 0.0)
        ref = orc.decode_latent(live, bf16_to_f32(q[[0, 2]]), LATENT)
        assert np.abs(got[[0, 2]] - ref).max() <= ATOL, step
    compare_state(cache.export(0), orc, live)
    cache.close()


@pytest.mark.parametrize("g", [16, 128])
def test_mla_long_heads_split_over_many_waves(g):
    """Two sequences of ~24K retained rows each (~750 tiles apiece over the
    decode units): every head is split over hundreds of units and merged, per
    group of 16 query heads, by the block that completes it.  Pools and
    workspace start as NaN bytes."""
    torch = _torch()
    w, P, T = 64, 64, 25000
    dms, cfg, cache, orc = _mk(2, g, w, P, num_pages=2 * (T // P + 8), maxp=T // P + 8)
    for p in cache.pools:
        p.fill_(0xFF)
    cache.workspace.fill_(0xFF)
    dms.dms_init_state(cache.ctx)
    torch.cuda.synchronize()
    inp = {s: MlaInputs(31, s, T + 4, g, 0.05) for s in (0, 1)}
    _append_chunks(dms, cache, orc, [0, 1], inp, {0: 0, 1: 0}, {0: T, 1: T - 777}, 2048)
    view = cache.export(0)
    assert view.L[:2, 0].min() > 20000
    compare_state(view, orc, [0, 1])
    _decode_steps(dms, cache, orc, [0, 1], inp, {0: T, 1: T - 777}, 3, g)
    cache.close()


def _prefill_run(g, seqs, lens, chunks, seed, p, w, P, nan_fill=False, then_decode=0, mode="delayed"):
    """Prefill every sequence to lens[s] tokens in calls of chunks[c] tokens
    per sequence (dms_prefill_chunk over latent rows): each call's outputs
    against dense masked absorbed attention over the full history, the state
    and stored rows after it against the oracle replay; then decode steps."""
    torch = _torch()
    maxp = max(lens.values()) // P + 4 + then_decode // P
    dms, cfg, cache, orc = _mk(max(seqs) + 1, g, w, P, num_pages=len(seqs) * maxp, maxp=maxp,
                               max_chunk=len(seqs) * max(chunks), mode=mode)
    if nan_fill:
        for pl in cache.pools:
            pl.fill_(0xFF)
        cache.workspace.fill_(0xFF)
        dms.dms_init_state(cache.ctx)
        torch.cuda.synchronize()
    inp = {s: MlaInputs(seed, s, lens[s] + then_decode, g, p) for s in seqs}
    scale = 1.0 / math.sqrt(ROW)
    cur = {s: 0 for s in seqs}
    ci = 0
    worst = 0.0
    while any(cur[s] < lens[s] for s in seqs):
        C = chunks[ci % len(chunks)]
        ci += 1
        ls = [min(C, lens[s] - cur[s]) for s in seqs]
        cu = np.concatenate([[0], np.cumsum(ls)]).astype(np.int32)
        q = np.concatenate([inp[s].q[cur[s]:cur[s] + l] for s, l in zip(seqs, ls)])
        k = np.concatenate([inp[s].k[cur[s]:cur[s] + l] for s, l in zip(seqs, ls)])
        f = np.concatenate([inp[s].flags[cur[s]:cur[s] + l] for s, l in zip(seqs, ls)])
        out = torch.full((int(cu[-1]), g, LATENT), float("nan"), device="cuda")
        dms.dms_prefill_chunk(cache.ctx, 0, len(seqs), to_dev(np.array(seqs, np.int32)), to_dev(cu),
                              int(cu[-1]), int(max(ls)), to_dev(q), to_dev(k), None, to_dev(f), out)
        torch.cuda.synchronize()
        assert dms.dms_status(cache.ctx) == 0
        got = out.cpu().numpy()
        for i, (s, l) in enumerate(zip(seqs, ls)):
            if l == 0:
                continue
            T = cur[s] + l
            rows = bf16_to_f32(inp[s].k[:T, 0]).astype(np.float64)
            qs = bf16_to_f32(inp[s].q[cur[s]:T]).astype(np.float64)
            for x in range(l):
                t = cur[s] + x
                if mode == "immediate":
                    mask = np.asarray(visible_immediate(t, np.arange(t + 1), inp[s].flags[:, 0], w), dtype=bool)
                else:
                    mask = np.asarray(visible(t, np.arange(t + 1), inp[s].flags[:t + 1, 0], w), dtype=bool)
                ref = mla_attention(qs[x], rows[:t + 1], np.broadcast_to(mask, (g, t + 1)), LATENT, scale)
                err = float(np.abs(got[cu[i] + x] - ref).max())
                worst = max(worst, err)
                assert err <= ATOL, (s, t, err)
        rows_f = [bf16_to_f32(inp[s].k[cur[s]:cur[s] + l]) for s, l in zip(seqs, ls)]
        orc.append_chunk(seqs, [inp[s].flags[cur[s]:cur[s] + l] for s, l in zip(seqs, ls)], rows_f, rows_f)
        for s, l in zip(seqs, ls):
            cur[s] += l
        view = _compare_rows(cache, orc, seqs)
        compare_state(view, orc, seqs)
    if then_decode:
        _decode_steps(dms, cache, orc, seqs, inp, {s: lens[s] for s in seqs}, then_decode, g, dense_every=4)
    cache.close()
    return worst


@pytest.mark.parametrize("g,w,P,p,chunks", [
    (16, 32, 64, 0.75, [256, 37]), (5, 16, 32, 0.5, [300]), (1, 8, 64, 0.9, [129, 64]),
    (40, 64, 64, 0.875, [200]), (128, 24, 64, 0.75, [96, 160])])
def test_mla_prefill_ragged_chunks(g, w, P, p, chunks):
    """Chunked prefill over latent rows: ragged histories, several chunkings,
    query groups below, at and above 16 heads (ragged groups of 16)."""
    lens = {2: 700, 0: 131, 1: 402} if g <= 40 else {1: 300, 0: 97}
    worst = _prefill_run(g, sorted(lens), lens, chunks, 53 + g, p, w, P)
    print(f"[mla prefill] g={g} max abs err {worst:.2e}", flush=True)


def test_mla_prefill_immediate_eviction():
    """The immediate-eviction timing (a token's own decision evicts the token
    w positions back, Sec. 5.3): cached keys hidden by decisions inside the
    chunk, chunk keys by later chunk decisions."""
    lens = {0: 600, 1: 333}
    _prefill_run(16, [0, 1], lens, [150, 64], 81, 0.7, 32, 64, mode="immediate")


def test_mla_prefill_on_nan_pools_then_decode():
    """Pools and workspace start as NaN bytes (stale rows of freed pages and
    the workspace's unused tiles must never reach an output); decode steps
    after the prefill continue from the committed state."""
    _prefill_run(16, [0, 1], {0: 500, 1: 260}, [200], 71, 0.8, 32, 64, nan_fill=True, then_decode=12)


def test_mla_prefill_q_is_refused():
    """Decisions from the query are not combined with latent rows."""
    from paper_2506_05345_amd import dms
    _, cfg, cache, _ = _mk(1, 16, 16, 32, 8, 4)
    torch = _torch()
    x = torch.zeros(16 * ROW, dtype=torch.bfloat16, device="cuda")
    cu = torch.tensor([0, 4], dtype=torch.int32, device="cuda")
    dec = torch.zeros(4, dtype=torch.uint8, device="cuda")
    out = torch.zeros(4 * 16 * LATENT, dtype=torch.float32, device="cuda")
    sid = torch.zeros(1, dtype=torch.int32, device="cuda")
    with pytest.raises(dms.DmsError):
        dms.dms_prefill_chunk_q(cache.ctx, 0, 1, sid, cu, 4, 4, x, x, None, dec, out)
    cache.close()


def test_mla_graph_replays_match_eager():
    """Latent-attention decode steps (two layers) captured once into a HIP
    graph and replayed with eager work in between: every replay equals an
    eager run of the same step on an identical cache, outputs bitwise and
    state bit-exact (split heads merge partials in unit order whichever
    block completes them)."""
    torch = _torch()
    from paper_2506_05345_amd import dms
    g, w, P, T0, REPLAYS = 16, 16, 64, 700, 4
    seqs = [2, 0, 1]
    kw = dict(num_layers=2, max_seqs=3, num_kv_heads=1, group_size=g, head_dim=ROW, window=w,
              page_size=P, num_pages=120, max_pages_per_head=32, max_chunk_tokens=3 * T0,
              kv_format=dms.DMS_KV_MLA)
    cfg = dms.make_config(**kw)
    eager, graphed = dms.DmsCache(cfg), dms.DmsCache(cfg)
    inp = {s: MlaInputs(67, s, T0 + REPLAYS, g, 0.6) for s in seqs}
    sid = to_dev(np.array(seqs, np.int32))
    cu = to_dev(np.array([0, T0, 2 * T0, 3 * T0], np.int32))
    kk = to_dev(np.concatenate([inp[s].k[:T0] for s in seqs]))
    ff = to_dev(np.concatenate([inp[s].flags[:T0] for s in seqs]))
    for c in (eager, graphed):
        for layer in (0, 1):
            dms.dms_append_chunk(c.ctx, layer, 3, sid, cu, 3 * T0, T0, kk, None, ff)
    torch.cuda.synchronize()
    qb = torch.empty((3, g, ROW), dtype=torch.bfloat16, device="cuda")
    kb = torch.empty((3, 1, ROW), dtype=torch.bfloat16, device="cuda")
    fb = torch.empty((3, 1), dtype=torch.uint8, device="cuda")
    outs = [torch.empty((3, g, LATENT), device="cuda") for _ in range(2)]

    def fill(t):
        qb.copy_(to_dev(np.stack([inp[s].q[t] for s in seqs])))
        kb.copy_(to_dev(np.stack([inp[s].k[t] for s in seqs])))
        fb.copy_(to_dev(np.stack([inp[s].flags[t] for s in seqs])))

    def step(c):
        for layer in (0, 1):
            dms.dms_decode_step(c.ctx, layer, 3, sid, qb, kb, None, fb, outs[layer])

    fill(T0)
    torch.cuda.synchronize()
    gr = torch.cuda.CUDAGraph()
    with torch.cuda.graph(gr):
        step(graphed)
    torch.cuda.synchronize()
    for r in range(REPLAYS):
        fill(T0 + r)
        torch.cuda.synchronize()
        gr.replay()
        torch.cuda.synchronize()
        got = [o.clone() for o in outs]
        step(eager)
        torch.cuda.synchronize()
        for layer in (0, 1):
            assert torch.equal(got[layer], outs[layer]), (r, layer)
            a, b = eager.export(layer), graphed.export(layer)
            for f in ("pos", "L", "ring_slot", "ring_flag", "page_table", "stack"):
                assert np.array_equal(getattr(a, f), getattr(b, f)), (r, layer, f)
        assert dms.dms_status(graphed.ctx) == 0 and dms.dms_status(eager.ctx) == 0
        _ = torch.ones(1000, device="cuda").sum().item()
    eager.close()
    graphed.close()
