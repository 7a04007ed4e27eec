"""GPU parity of page retrieval within the retained set (Quest on top of DMS)
against the CPU oracle: page bounds bit-exact (bf16 min / max of the stored
keys of every live page), the selection equal to the oracle's top-budget
pages wherever the float32 scores cannot reorder them (else checked valid
within the float32 rounding bound), and decode outputs within 1e-2 of
float64 attention over the live slots of the pages the GPU selected."""
import numpy as np
import pytest

from dms_testlib import ATOL, SeqInputs, bf16_to_f32, compare_state, to_dev
from oracle import PagedKVOracle, masked_attention, quest_page_scores, quest_select

pytestmark = pytest.mark.gpu


def _mk(B, fp8=False, **kw):
    import torch
    from paper_2506_05345_amd import dms
    cfg = dms.make_config(quest_page_budget=B, kv_format=dms.DMS_KV_FP8 if fp8 else dms.DMS_KV_BF16, **kw)
    cache = dms.DmsCache(cfg)
    cache.workspace.fill_(0xFF)   # stale bytes must not matter
    dms.dms_init_state(cache.ctx)
    torch.cuda.synchronize()
    orc = PagedKVOracle(cfg.max_seqs, cfg.num_kv_heads, cfg.window, cfg.page_size, cfg.num_pages,
                        cfg.max_pages_per_head, cfg.head_dim, kv_format="fp8" if fp8 else "bf16")
    return dms, cfg, cache, orc


def _bounds_from_export(cache, layer=0):
    from paper_2506_05345_amd import dms
    o = cache.offsets
    raw = dms.dms_export_state(cache.ctx, layer, o.layer_stride)
    c = cache.cfg
    n = c.num_pages * 2 * c.head_dim
    u16 = raw[o.page_bounds:o.page_bounds + 2 * n].view(np.uint16).reshape(c.num_pages, 2, c.head_dim)
    return bf16_to_f32(u16).astype(np.float64)


def _head_pages(orc, s, h, P):
    L = int(orc.L[s, h])
    k = orc.k_store[s, h, :L]
    npg = -(-L // P)
    lo = np.stack([k[i * P:min(L, (i + 1) * P)].min(axis=0) for i in range(npg)])
    hi = np.stack([k[i * P:min(L, (i + 1) * P)].max(axis=0) for i in range(npg)])
    return L, k, lo, hi


def _check_bounds(cache, orc, seqs):
    c = cache.cfg
    P = c.page_size
    got = _bounds_from_export(cache)
    view = cache.export(0)
    for s in seqs:
        for h in range(c.num_kv_heads):
            L, _, lo, hi = _head_pages(orc, s, h, P)
            for i in range(lo.shape[0]):
                pg = int(view.page_table[s, h, i])
                assert np.array_equal(got[pg, 0], lo[i]) and np.array_equal(got[pg, 1], hi[i]), (s, h, i)


def _check_step(dms, cache, orc, seqs, q_bf16, out, g):
    """Selection and outputs of the last decode call."""
    import torch
    c = cache.cfg
    H, P, B, D = c.num_kv_heads, c.page_size, c.quest_page_budget, c.head_dim
    n = len(seqs)
    pages = torch.empty((n * H, B), dtype=torch.int32, device="cuda")
    counts = torch.empty(n * H, dtype=torch.int32, device="cuda")
    dms.dms_quest_selection(cache.ctx, n, pages, counts)
    torch.cuda.synchronize()
    pages, counts = pages.cpu().numpy(), counts.cpu().numpy()
    q = bf16_to_f32(q_bf16).astype(np.float64)
    got = out.cpu().numpy()
    exact = ambiguous = 0
    for i, s in enumerate(seqs):
        for h in range(H):
            hh = i * H + h
            L, k, lo, hi = _head_pages(orc, s, h, P)
            qg = q[i, h * g:(h + 1) * g]
            sel = pages[hh, :counts[hh]]
            assert list(pages[hh, counts[hh]:]) == [-1] * (B - counts[hh])
            npg = lo.shape[0]
            ref_sel = quest_select(quest_page_scores(qg, lo, hi), B)
            if npg <= B:
                assert list(sel) == list(range(npg))
            elif list(sel) == list(ref_sel):
                exact += 1
            else:
                # only near-ties may differ: float32 sums of 128 exact products
                u = quest_page_scores(qg, lo, hi)
                mag = np.max(np.abs(qg)[:, None, :] * np.maximum(np.abs(lo), np.abs(hi))[None], axis=0).sum(-1)
                tol = 1e-5 * mag.max() + 1e-30
                assert len(sel) == B and np.all(np.diff(sel) > 0)
                rest = np.setdiff1d(np.arange(npg), sel)
                assert u[sel].min() >= u[rest].max() - tol, (s, h, sel, ref_sel)
                ambiguous += 1
            slots = np.concatenate([np.arange(p * P, min(L, (p + 1) * P)) for p in sel])
            ref = masked_attention(qg, k[slots], orc.v_store[s, h, slots], np.ones((g, len(slots)), bool),
                                   1 / np.sqrt(D))
            err = np.abs(got[i, h * g:(h + 1) * g] - ref).max()
            assert err <= ATOL, (s, h, err)
    return exact, ambiguous


def _append_chunks(dms, cache, orc, seqs, inputs, lens, chunk):
    import torch
    cur = {s: 0 for s in seqs}
    while any(cur[s] < lens[s] for s in seqs):
        ls = [min(chunk, lens[s] - cur[s]) for s in seqs]
        cu = np.concatenate([[0], np.cumsum(ls)]).astype(np.int32)
        cat = lambda name: np.concatenate([getattr(inputs[s], name)[cur[s]:cur[s] + l] for s, l in zip(seqs, ls)])
        dms.dms_append_chunk(cache.ctx, 0, len(seqs), to_dev(np.array(seqs, np.int32)), to_dev(cu),
                             int(cu[-1]), int(max(ls)), to_dev(cat("k")), to_dev(cat("v")), to_dev(cat("flags")))
        orc.append_chunk(seqs, [inputs[s].flags[cur[s]:cur[s] + l] for s, l in zip(seqs, ls)],
                         [bf16_to_f32(inputs[s].k[cur[s]:cur[s] + l]) for s, l in zip(seqs, ls)],
                         [bf16_to_f32(inputs[s].v[cur[s]:cur[s] + l]) for s, l in zip(seqs, ls)])
        for s, l in zip(seqs, ls):
            cur[s] += l
        torch.cuda.synchronize()
        assert dms.dms_status(cache.ctx) == 0


def _decode_steps(dms, cache, orc, seqs, inputs, t0, nsteps, g, fused=True, check_bounds_every=4):
    import torch
    c = cache.cfg
    sid = to_dev(np.array(seqs, np.int32))
    tot_exact = tot_amb = 0
    for step in range(nsteps):
        ts = {s: t0[s] + step for s in seqs}
        q = np.stack([inputs[s].q[ts[s]] for s in seqs])
        k = np.stack([inputs[s].k[ts[s]] for s in seqs])
        v = np.stack([inputs[s].v[ts[s]] for s in seqs])
        f = np.stack([inputs[s].flags[ts[s]] for s in seqs])
        out = torch.full((len(seqs), c.num_kv_heads * g, c.head_dim), float("nan"), device="cuda")
        if fused:
            dms.dms_decode_step(cache.ctx, 0, len(seqs), sid, to_dev(q), to_dev(k), to_dev(v), to_dev(f), out)
        else:
            dms.dms_append(cache.ctx, 0, len(seqs), sid, to_dev(k), to_dev(v), to_dev(f))
            dms.dms_decode(cache.ctx, 0, len(seqs), sid, to_dev(q), out)
        torch.cuda.synchronize()
        assert dms.dms_status(cache.ctx) == 0
        orc.append(seqs, f, bf16_to_f32(k), bf16_to_f32(v))
        e, a = _check_step(dms, cache, orc, seqs, q, out, g)
        tot_exact += e
        tot_amb += a
        if step % check_bounds_every == 0 or step == nsteps - 1:
            _check_bounds(cache, orc, seqs)
            compare_state(cache.export(0), orc, seqs)
    return tot_exact, tot_amb


@pytest.mark.parametrize("d,g,w,P,p,B", [(128, 5, 16, 32, 0.75, 3), (64, 2, 4, 64, 0.5, 2),
                                         (128, 16, 40, 32, 0.875, 2), (64, 7, 1, 32, 0.9, 1)])
def test_chunk_then_decode_steps(d, g, w, P, p, B):
    """Ragged heads (some within the budget, most beyond it): bounds after
    chunk commits and after every decode step's append, selection, outputs."""
    H = 2
    seqs = [3, 0, 2]
    dms, cfg, cache, orc = _mk(B, num_layers=1, max_seqs=4, num_kv_heads=H, group_size=g, head_dim=d,
                               window=w, page_size=P, num_pages=400, max_pages_per_head=64,
                               max_chunk_tokens=3 * 300)
    lens = {3: 701, 0: 40, 2: 333}
    inp = {s: SeqInputs(61, 0, s, lens[s] + 24, H, g, d, p) for s in seqs}
    _append_chunks(dms, cache, orc, seqs, inp, lens, 300)
    _check_bounds(cache, orc, seqs)
    exact, amb = _decode_steps(dms, cache, orc, seqs, inp, lens, 24, g)
    print(f"selections equal to the oracle's: {exact}, near-tie differences: {amb}")
    assert exact > 0


def test_append_then_decode_path_and_fp8_pages():
    """dms_append (scatter) + dms_decode, FP8 pages: bounds of dequantized keys."""
    H, g, d, P = 2, 4, 128, 32
    seqs = [1, 0]
    dms, cfg, cache, orc = _mk(2, fp8=True, num_layers=1, max_seqs=2, num_kv_heads=H, group_size=g,
                               head_dim=d, window=8, page_size=P, num_pages=64, max_pages_per_head=16,
                               max_chunk_tokens=600)
    lens = {1: 250, 0: 90}
    inp = {s: SeqInputs(62, 0, s, lens[s] + 30, H, g, d, 0.7) for s in seqs}
    _append_chunks(dms, cache, orc, seqs, inp, lens, 300)
    _decode_steps(dms, cache, orc, seqs, inp, lens, 30, g, fused=False)


def test_budget_covering_every_page_is_dense_decode():
    import torch
    from paper_2506_05345_amd import dms as dmsmod
    H, g, d, P = 2, 3, 128, 64
    kw = dict(num_layers=1, max_seqs=2, num_kv_heads=H, group_size=g, head_dim=d, window=16,
              page_size=P, num_pages=64, max_pages_per_head=16, max_chunk_tokens=1000)
    dms, cfg, cache, orc = _mk(16, **kw)
    dense = dmsmod.DmsCache(dmsmod.make_config(**kw))
    seqs = [0, 1]
    lens = {0: 400, 1: 977}
    inp = {s: SeqInputs(63, 0, s, lens[s] + 2, H, g, d, 0.6) for s in seqs}
    orc2 = PagedKVOracle(2, H, 16, P, 64, 16, d)
    _append_chunks(dms, cache, orc, seqs, inp, lens, 500)
    _append_chunks(dmsmod, dense, orc2, seqs, inp, lens, 500)
    sid = to_dev(np.array(seqs, np.int32))
    q = to_dev(np.stack([inp[s].q[lens[s]] for s in seqs]))
    a = torch.empty((2, H * g, d), device="cuda")
    b = torch.empty((2, H * g, d), device="cuda")
    dms.dms_decode(cache.ctx, 0, 2, sid, q, a)
    dmsmod.dms_decode(dense.ctx, 0, 2, sid, q, b)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


def test_many_heads_multi_pass_planner():
    """320 sequences x 4 KV heads: more heads than one planning block has
    threads, so the multi-pass planner plans over the selected pages."""
    H, g, d, P, B = 4, 2, 64, 32, 2
    rng = np.random.default_rng(71)
    seqs = [int(s) for s in rng.permutation(320)]
    lens = {s: int(rng.integers(1, 300)) for s in seqs}
    dms, cfg, cache, orc = _mk(B, num_layers=1, max_seqs=320, num_kv_heads=H, group_size=g, head_dim=d,
                               window=8, page_size=P, num_pages=12000, max_pages_per_head=32,
                               max_chunk_tokens=320 * 300)
    inp = {s: SeqInputs(72, 0, s, lens[s] + 3, H, g, d, 0.5) for s in seqs}
    _append_chunks(dms, cache, orc, seqs, inp, lens, 300)
    exact, amb = _decode_steps(dms, cache, orc, seqs, inp, lens, 3, g, check_bounds_every=2)
    assert exact > 100


def test_query_decisions_read_the_zeroed_neuron():
    """Decisions from the borrowed neuron (App. C): selection scores and
    attention both read that element as 0."""
    import torch
    from oracle import query_decisions, zero_borrowed_neuron
    H, g, d, P, B = 2, 4, 128, 32, 2
    dms, cfg, cache, orc = _mk(B, num_layers=1, max_seqs=2, num_kv_heads=H, group_size=g, head_dim=d,
                               window=8, page_size=P, num_pages=64, max_pages_per_head=16,
                               max_chunk_tokens=600, decision_source=1, decision_bias=0.0)
    seqs = [1, 0]
    lens = {1: 300, 0: 180}
    inp = {s: SeqInputs(73, 0, s, lens[s] + 10, H, g, d, 0.5) for s in seqs}
    for s in seqs:   # decisions as the library will take them: from q
        inp[s].flags[:] = query_decisions(bf16_to_f32(inp[s].q), g, 0.0)
    _append_chunks(dms, cache, orc, seqs, inp, lens, 300)
    sid = to_dev(np.array(seqs, np.int32))
    for step in range(10):
        ts = {s: lens[s] + step for s in seqs}
        q = np.stack([inp[s].q[ts[s]] for s in seqs])
        k = np.stack([inp[s].k[ts[s]] for s in seqs])
        v = np.stack([inp[s].v[ts[s]] for s in seqs])
        out = torch.full((2, H * g, d), float("nan"), device="cuda")
        dec = torch.empty((2, H), dtype=torch.uint8, device="cuda")
        dms.dms_decode_step_q(cache.ctx, 0, 2, sid, to_dev(q), to_dev(k), to_dev(v), dec, out)
        torch.cuda.synchronize()
        assert dms.dms_status(cache.ctx) == 0
        f = np.stack([inp[s].flags[ts[s]] for s in seqs])
        assert np.array_equal(dec.cpu().numpy(), f)
        orc.append(seqs, f, bf16_to_f32(k), bf16_to_f32(v))
        qz = zero_borrowed_neuron(bf16_to_f32(q), g)
        from dms_synth import f32_to_bf16_bits_np
        _check_step(dms, cache, orc, seqs, f32_to_bf16_bits_np(qz.astype(np.float32)), out, g)

