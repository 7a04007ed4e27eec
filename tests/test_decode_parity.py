"""GPU parity of the decode path (append + split-K decode + combine) and of
chunk commits against the CPU oracle: bookkeeping bit-exact, outputs within
1e-2 max-abs (bf16 inputs, fp32 accumulation)."""
import numpy as np
import pytest

from dms_testlib import ATOL, SeqInputs, bf16_to_f32, compare_pool, compare_state, to_dev
from oracle import PagedKVOracle, dense_dms_attention

pytestmark = pytest.mark.gpu


def _torch():
    import torch
    return torch


def _mk(cfg_kw):
    from paper_2506_05345_amd import dms
    cfg = dms.make_config(**cfg_kw)
    return dms, cfg, dms.DmsCache(cfg)


def _oracle_for(cfg):
    return PagedKVOracle(cfg.max_seqs, cfg.num_kv_heads, cfg.window, cfg.page_size,
                         cfg.num_pages, cfg.max_pages_per_head, cfg.head_dim)


def _append_chunks(dms, cache, orc, seqs, inputs, start, stop, chunk):
    """Append positions start[s] .. stop[s]-1 of every sequence in pieces of
    at most `chunk` tokens, one call per piece (all sequences together)."""
    torch = _torch()
    cur = dict(start)
    while any(cur[s] < stop[s] for s in seqs):
        lens = [min(chunk, stop[s] - cur[s]) for s in seqs]
        cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
        fl = np.concatenate([inputs[s].flags[cur[s]:cur[s] + l] for s, l in zip(seqs, lens)])
        kk = np.concatenate([inputs[s].k[cur[s]:cur[s] + l] for s, l in zip(seqs, lens)])
        vv = np.concatenate([inputs[s].v[cur[s]:cur[s] + l] for s, l in zip(seqs, lens)])
        sid = to_dev(np.array(seqs, np.int32))
        dms.dms_append_chunk(cache.ctx, 0, len(seqs), sid, to_dev(cu), int(cu[-1]), int(max(lens)),
                             to_dev(kk), to_dev(vv), to_dev(fl))
        orc.append_chunk(seqs, [inputs[s].flags[cur[s]:cur[s] + l] for s, l in zip(seqs, lens)],
                         [bf16_to_f32(inputs[s].k[cur[s]:cur[s] + l]) for s, l in zip(seqs, lens)],
                         [bf16_to_f32(inputs[s].v[cur[s]:cur[s] + l]) for s, l in zip(seqs, lens)])
        for s, l in zip(seqs, lens):
            cur[s] += l
        torch.cuda.synchronize()
        assert dms.dms_status(cache.ctx) == 0


def _decode_steps(dms, cache, orc, seqs, inputs, t_from, nsteps, g, check_every=1, dense_check=True):
    """Run nsteps decode steps; compare state and outputs against the oracle."""
    torch = _torch()
    cfg = cache.cfg
    Hq = cfg.num_kv_heads * g
    sid = to_dev(np.array(seqs, np.int32))
    worst = 0.0
    for step in range(nsteps):
        ts = {s: t_from[s] + step for s in seqs}
        q = np.stack([inputs[s].q[ts[s]] for s in seqs])
        k = np.stack([inputs[s].k[ts[s]] for s in seqs])
        v = np.stack([inputs[s].v[ts[s]] for s in seqs])
        f = np.stack([inputs[s].flags[ts[s]] for s in seqs])
        out = torch.full((len(seqs), Hq, cfg.head_dim), float("nan"), device="cuda")
        dms.dms_decode_step(cache.ctx, 0, len(seqs), sid, to_dev(q), to_dev(k), to_dev(v),
                            to_dev(f), out)
        torch.cuda.synchronize()
        assert dms.dms_status(cache.ctx) == 0
        orc.append(seqs, f, bf16_to_f32(k), bf16_to_f32(v))
        ref = orc.decode(seqs, bf16_to_f32(q), g)
        got = out.cpu().numpy()
        err = np.abs(got - ref).max()
        worst = max(worst, err)
        assert err <= ATOL, (step, err)
        if dense_check and step % 16 == 0:
            # mask route over the full history (definition of the output)
            for i, s in enumerate(seqs):
                t = ts[s]
                dref = dense_dms_attention(bf16_to_f32(inputs[s].q[t:t + 1]),
                                           bf16_to_f32(inputs[s].k[:t + 1]),
                                           bf16_to_f32(inputs[s].v[:t + 1]),
                                           inputs[s].flags[:t + 1], cfg.window, g, t_query=[t])
                assert np.abs(got[i] - dref[0]).max() <= ATOL
        if step % check_every == 0 or step == nsteps - 1:
            view = cache.export(0)
            compare_state(view, orc, seqs)
    return worst


@pytest.mark.parametrize("chunk", [512, 37])
def test_tiny_config_prefill_then_decode(chunk):
    """1 sequence, 2 KV heads x group 2, d=64, 512-token context then 64 decode
    steps, w=16, flags Bernoulli(1/2), seed 0."""
    dms, cfg, cache = _mk(dict(num_layers=1, max_seqs=1, num_kv_heads=2, group_size=2,
                               head_dim=64, window=16, page_size=64, num_pages=32,
                               max_pages_per_head=16, max_chunk_tokens=512))
    inp = {0: SeqInputs(0, 0, 0, 576, 2, 2, 64, 0.5)}
    orc = _oracle_for(cfg)
    _append_chunks(dms, cache, orc, [0], inp, {0: 0}, {0: 512}, chunk)
    view = cache.export(0)
    compare_state(view, orc, [0])
    compare_pool(cache, 0, view, [0], inp)
    worst = _decode_steps(dms, cache, orc, [0], inp, {0: 512}, 64, 2)
    compare_pool(cache, 0, cache.export(0), [0], inp)
    print(f"max abs err {worst:.3e}")


@pytest.mark.parametrize("d,g,w,P,p", [(128, 6, 8, 32, 0.875), (128, 5, 20, 64, 0.75),
                                       (64, 7, 3, 128, 0.5), (128, 16, 256, 256, 0.875),
                                       (64, 1, 1, 32, 0.9)])
def test_ragged_multi_sequence(d, g, w, P, p):
    """Several sequences of different lengths, called out of id order, chunk
    sizes that are not multiples of the page or tile, then decode."""
    H = 2
    seqs = [3, 0, 2]
    dms, cfg, cache = _mk(dict(num_layers=1, max_seqs=4, num_kv_heads=H, group_size=g,
                               head_dim=d, window=w, page_size=P, num_pages=400,
                               max_pages_per_head=64, max_chunk_tokens=3 * 300))
    lens = {3: 700, 0: 95, 2: 333}
    inp = {s: SeqInputs(11, 0, s, lens[s] + 40, H, g, d, p) for s in seqs}
    orc = _oracle_for(cfg)
    _append_chunks(dms, cache, orc, seqs, inp, {s: 0 for s in seqs}, lens, 300)
    view = cache.export(0)
    compare_state(view, orc, seqs)
    compare_pool(cache, 0, view, seqs, inp)
    _decode_steps(dms, cache, orc, seqs, inp, lens, 40, g, check_every=7)
    compare_pool(cache, 0, cache.export(0), seqs, inp)


def test_qwen3_8b_shape_window_512():
    """The Qwen3-8B attention shape of the sweeps (8 KV heads x group 4,
    head_dim 128) with its window w = 512 (Sec. 5.2): contexts below, at and
    well past the window, chunks that are not multiples of the page, then
    decode steps across the window boundary of the shortest sequence."""
    H, g, d, w, P = 8, 4, 128, 512, 64
    seqs = [4, 1, 0, 3, 2]
    lens = {4: 300, 1: 511, 0: 512, 3: 1900, 2: 3700}
    dms, cfg, cache = _mk(dict(num_layers=1, max_seqs=5, num_kv_heads=H, group_size=g,
                               head_dim=d, window=w, page_size=P, num_pages=5 * H * 70,
                               max_pages_per_head=70, max_chunk_tokens=5 * 700))
    inp = {s: SeqInputs(29, 0, s, lens[s] + 240, H, g, d, 0.875) for s in seqs}
    orc = _oracle_for(cfg)
    _append_chunks(dms, cache, orc, seqs, inp, {s: 0 for s in seqs}, lens, 700)
    view = cache.export(0)
    compare_state(view, orc, seqs)
    compare_pool(cache, 0, view, seqs, inp)
    # 230 steps take sequence 4 from 300 past the window (512) and the others further
    _decode_steps(dms, cache, orc, seqs, inp, lens, 230, g, check_every=23)
    compare_pool(cache, 0, cache.export(0), seqs, inp)
    cache.close()


def test_many_heads_multi_pass_planner():
    """320 sequences x 4 KV heads = 1280 heads per call: more heads than one
    planning block has threads, so the multi-pass planner runs; ragged short
    contexts, some heads longer than one decode wave's share."""
    H, g, d, w, P = 4, 2, 64, 16, 32
    rng = np.random.default_rng(77)
    seqs = [int(s) for s in rng.permutation(320)]
    lens = {s: int(rng.integers(1, 260)) for s in seqs}
    lens[seqs[5]] = 3000          # one long sequence: its heads span several waves
    dms, cfg, cache = _mk(dict(num_layers=1, max_seqs=320, num_kv_heads=H, group_size=g,
                               head_dim=d, window=w, page_size=P, num_pages=12000,
                               max_pages_per_head=128, max_chunk_tokens=320 * 256))
    inp = {s: SeqInputs(13, 0, s, lens[s] + 6, H, g, d, 0.6) for s in seqs}
    orc = _oracle_for(cfg)
    _append_chunks(dms, cache, orc, seqs, inp, {s: 0 for s in seqs}, lens, 256)
    compare_state(cache.export(0), orc, seqs)
    _decode_steps(dms, cache, orc, seqs, inp, lens, 6, g, check_every=2, dense_check=False)
    cache.close()


@pytest.mark.parametrize("nseq", [3, 20, 25])
def test_short_heads_split_over_workgroups(nseq):
    """Small calls whose heads all fit one workgroup's share: 12, 80 and 100
    call heads are split over 4, 3 and 2 workgroups per head (one folded
    partial each, merged by the last); heads of 1-3 tiles leave parts without
    tiles."""
    H, g, d, w, P = 4, 2, 64, 16, 32
    rng = np.random.default_rng(90 + nseq)
    seqs = [int(s) for s in rng.permutation(nseq)]
    lens = {s: int(rng.integers(1, 600)) for s in seqs}
    for s in seqs[:3]:
        lens[s] = int(rng.integers(1, 90))   # one to three tiles
    dms, cfg, cache = _mk(dict(num_layers=1, max_seqs=nseq, num_kv_heads=H, group_size=g,
                               head_dim=d, window=w, page_size=P, num_pages=4000,
                               max_pages_per_head=64, max_chunk_tokens=nseq * 600))
    inp = {s: SeqInputs(91, 0, s, lens[s] + 8, H, g, d, 0.7) for s in seqs}
    orc = _oracle_for(cfg)
    _append_chunks(dms, cache, orc, seqs, inp, {s: 0 for s in seqs}, lens, 600)
    compare_state(cache.export(0), orc, seqs)
    _decode_steps(dms, cache, orc, seqs, inp, lens, 8, g, check_every=3, dense_check=False)
    compare_pool(cache, 0, cache.export(0), seqs, inp)
    cache.close()


def test_decode_from_empty_cache_token_by_token():
    """Every token through dms_decode_step from position 0 (first steps have a
    single visible key, the output is that value exactly up to rounding)."""
    dms, cfg, cache = _mk(dict(num_layers=1, max_seqs=2, num_kv_heads=3, group_size=4,
                               head_dim=128, window=5, page_size=32, num_pages=64,
                               max_pages_per_head=16))
    seqs = [1, 0]
    inp = {s: SeqInputs(5, 0, s, 150, 3, 4, 128, 0.6) for s in seqs}
    orc = _oracle_for(cfg)
    _decode_steps(dms, cache, orc, seqs, inp, {0: 0, 1: 0}, 150, 4, check_every=5)


@pytest.mark.parametrize("variant", ["peaked", "v_const", "needle"])
def test_value_variants(variant):
    torch = _torch()
    dms, cfg, cache = _mk(dict(num_layers=1, max_seqs=1, num_kv_heads=1, group_size=4,
                               head_dim=128, window=16, page_size=64, num_pages=64,
                               max_pages_per_head=32, max_chunk_tokens=1024))
    T = 1000
    inp = SeqInputs(21, 0, 0, T + 1, 1, 4, 128, 0.875, q_scale=8.0 if variant == "peaked" else 1.0)
    if variant == "v_const":
        inp.v[:] = 0x3F80  # 1.0
    if variant == "needle":
        # a kept key and an evicted key both aligned with the last query
        inp.k[:] = 0
        inp.q[T] = 0
        inp.q[T, :, 0] = 0x447A  # 1000.0
        inp.k[100, 0, 0] = 0x3F80
        inp.flags[100] = 0
        inp.v[100, 0, :] = 0x4000  # 2.0
        inp.k[200, 0, 0] = 0x3F80
        inp.flags[200] = 1
        inp.v[200, 0, :] = 0xC000  # -2.0
    orc = _oracle_for(cfg)
    _append_chunks(dms, cache, orc, [0], {0: inp}, {0: 0}, {0: T}, 1024)
    _decode_steps(dms, cache, orc, [0], {0: inp}, {0: T}, 1, 4)
    if variant in ("v_const", "needle"):
        out = torch.empty((1, 4, 128), device="cuda")
        dms.dms_decode(cache.ctx, 0, 1, to_dev(np.array([0], np.int32)), to_dev(inp.q[T][None]), out)
        torch.cuda.synchronize()
        o = out.cpu().numpy()
        if variant == "v_const":
            assert np.abs(o - 1.0).max() < 4e-3
        else:
            assert np.abs(o[0, 0] - 2.0).max() < 1e-2  # the kept needle, nothing of -2


def test_out_of_pages_is_sticky_and_changes_nothing():
    torch = _torch()
    dms, cfg, cache = _mk(dict(num_layers=1, max_seqs=2, num_kv_heads=2, group_size=2,
                               head_dim=64, window=4, page_size=32, num_pages=5,
                               max_pages_per_head=8, max_chunk_tokens=256))
    inp = {s: SeqInputs(3, 0, s, 200, 2, 2, 64, 0.0) for s in (0, 1)}
    orc = _oracle_for(cfg)
    # 60 kept tokens: 2 pages per head, slots 60..63 still free in the last page
    _append_chunks(dms, cache, orc, [0], inp, {0: 0}, {0: 60}, 64)
    before = cache.export(0)
    # sequence 1 needs 2 more pages (one per head): only 1 left
    sid = to_dev(np.array([1], np.int32))
    cu = to_dev(np.array([0, 10], np.int32))
    dms.dms_append_chunk(cache.ctx, 0, 1, sid, cu, 10, 10, to_dev(inp[1].k[:10]),
                         to_dev(inp[1].v[:10]), to_dev(inp[1].flags[:10]))
    assert dms.dms_status(cache.ctx) == dms.DMS_ERR_OUT_OF_PAGES
    after = cache.export(0)
    for f in ("pos", "L", "ring_slot", "page_table", "slot_pos", "stack"):
        assert np.array_equal(getattr(before, f), getattr(after, f)), f
    # later calls are no-ops while the status is set; outputs untouched
    out = torch.full((1, 4, 64), 7.0, device="cuda")
    s0 = to_dev(np.array([0], np.int32))
    dms.dms_decode_step(cache.ctx, 0, 1, s0, to_dev(inp[0].q[60][None]), to_dev(inp[0].k[60][None]),
                        to_dev(inp[0].v[60][None]), to_dev(inp[0].flags[60][None]), out)
    torch.cuda.synchronize()
    assert (out == 7.0).all()
    assert cache.export(0).pos[0] == 60
    dms.dms_clear_status(cache.ctx)
    assert dms.dms_status(cache.ctx) == 0
    _decode_steps(dms, cache, orc, [0], inp, {0: 60}, 4, 2)
    # the fifth step needs a page per head again: one is left, two are needed
    dms.dms_decode_step(cache.ctx, 0, 1, s0, to_dev(inp[0].q[64][None]), to_dev(inp[0].k[64][None]),
                        to_dev(inp[0].v[64][None]), to_dev(inp[0].flags[64][None]), out)
    assert dms.dms_status(cache.ctx) == dms.DMS_ERR_OUT_OF_PAGES
    compare_state(cache.export(0), orc, [0, 1])


def test_bad_sequence_ids_set_status():
    dms, cfg, cache = _mk(dict(num_layers=1, max_seqs=3, num_kv_heads=1, group_size=1,
                               head_dim=64, window=4, page_size=32, num_pages=8,
                               max_pages_per_head=4))
    z = to_dev(np.zeros((2, 1, 64), np.uint16))
    f = to_dev(np.zeros((2, 1), np.uint8))
    for ids in ([0, 0], [1, 3], [-1, 0]):
        dms.dms_append(cache.ctx, 0, 2, to_dev(np.array(ids, np.int32)), z, z, f)
        assert dms.dms_status(cache.ctx) == dms.DMS_ERR_BAD_SEQ
        assert cache.export(0).pos.tolist() == [0, 0, 0]
        dms.dms_clear_status(cache.ctx)


def test_seq_reset_returns_pages_in_order():
    dms, cfg, cache = _mk(dict(num_layers=2, max_seqs=3, num_kv_heads=2, group_size=2,
                               head_dim=64, window=4, page_size=32, num_pages=40,
                               max_pages_per_head=8, max_chunk_tokens=600))
    seqs = [2, 0, 1]
    inp = {s: SeqInputs(8, 0, s, 200, 2, 2, 64, 0.3) for s in seqs}
    orc = _oracle_for(cfg)
    _append_chunks(dms, cache, orc, seqs, inp, {s: 0 for s in seqs}, {2: 150, 0: 90, 1: 199}, 200)
    dms.dms_seq_reset(cache.ctx, 0, 2, to_dev(np.array([0, 2], np.int32)))
    orc.seq_reset([0, 2])
    view = cache.export(0)
    compare_state(view, orc, [0, 1, 2])
    # reuse after reset
    _append_chunks(dms, cache, orc, [2], inp, {2: 0}, {2: 120}, 120)
    compare_state(cache.export(0), orc, [0, 1, 2])


@pytest.mark.parametrize("lens", [(40, 97, 130), (300, 5, 1)])
def test_merge_ignores_stale_workspace(lens):
    """Fewer tiles than decode waves, so heads split over spans that include
    waves with no tiles (their partial slots are never written): a workspace
    filled with NaN bytes beforehand must not reach the outputs.  Spans of up
    to 4 waves take the register merge, longer ones the batched merge."""
    torch = _torch()
    dms, cfg, cache = _mk(dict(num_layers=1, max_seqs=3, num_kv_heads=2, group_size=3,
                               head_dim=128, window=8, page_size=32, num_pages=64,
                               max_pages_per_head=16, max_chunk_tokens=3 * 300))
    cache.workspace.fill_(0xFF)
    dms.dms_init_state(cache.ctx)     # re-zeroes only what the library keeps between calls
    torch.cuda.synchronize()
    seqs = [2, 0, 1]
    ln = dict(zip(seqs, lens))
    inp = {s: SeqInputs(51, 0, s, ln[s] + 8, 2, 3, 128, 0.5) for s in seqs}
    orc = _oracle_for(cfg)
    _append_chunks(dms, cache, orc, seqs, inp, {s: 0 for s in seqs}, ln, 300)
    _decode_steps(dms, cache, orc, seqs, inp, ln, 8, 3, check_every=4)


@pytest.mark.parametrize("fmt", ["bf16", "fp8"])
def test_long_heads_split_over_hundreds_of_waves(fmt):
    """Two heads of ~24K retained tokens each: ~1500 tiles over the 1024 decode
    waves, so every head is split over hundreds of waves and its merge runs
    the batched path over several batches of 64 partials, at the end of the
    waves that complete it.  Flags mostly 0 so the heads stay long.  Pools and
    workspace start as NaN bytes, so a stale partial or slot would show."""
    torch = _torch()
    from paper_2506_05345_amd import dms as dmsmod
    H, g, d, w, P = 2, 4, 128, 64, 64
    T = 26000
    kw = dict(num_layers=1, max_seqs=1, num_kv_heads=H, group_size=g, head_dim=d, window=w,
              page_size=P, num_pages=2 * (T // P + 8), max_pages_per_head=T // P + 8,
              max_chunk_tokens=4096)
    if fmt == "fp8":
        kw["kv_format"] = dmsmod.DMS_KV_FP8
    dms, cfg, cache = _mk(kw)
    for p in cache.pools:
        p.fill_(0xFF)
    cache.workspace.fill_(0xFF)
    dms.dms_init_state(cache.ctx)
    torch.cuda.synchronize()
    inp = {0: SeqInputs(29, 0, 0, T + 4, H, g, d, 0.05)}
    orc = PagedKVOracle(cfg.max_seqs, H, w, P, cfg.num_pages, cfg.max_pages_per_head, d,
                        kv_format=fmt)
    _append_chunks(dms, cache, orc, [0], inp, {0: 0}, {0: T}, 4096)
    view = cache.export(0)
    assert view.L[0].min() > 20000
    compare_state(view, orc, [0])
    _decode_steps(dms, cache, orc, [0], inp, {0: T}, 3, g, dense_check=False)
    cache.close()
