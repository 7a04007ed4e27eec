"""GPU parity of the decision modes against the CPU oracle:

* immediate eviction (Sec. 5.3 ablation: the decision made at step j + w
  evicts token j) through decode steps, chunk appends and masked prefill;
* decisions read from the borrowed query neuron (Sec. 3.2 rounding, App. C:
  round(sigmoid(q[first head of group][0] + b)), the neuron then zeroed for
  attention) through dms_decode_step_q / dms_prefill_chunk_q.

Decisions and bookkeeping are compared bit-exactly, outputs within 1e-2."""
import numpy as np
import pytest

import oracle
from dms_testlib import ATOL, SeqInputs, bf16_to_f32, compare_pool, compare_state, to_dev
from oracle import PagedKVOracle, dense_dms_attention

pytestmark = pytest.mark.gpu


def _setup(mode, decide, bias=-0.3, **kw):
    from paper_2506_05345_amd import dms
    cfg_kw = dict(num_layers=1, max_seqs=4, num_kv_heads=2, group_size=3, head_dim=128, window=16,
                  page_size=32, num_pages=256, max_pages_per_head=64, max_chunk_tokens=3 * 300)
    cfg_kw.update(kw)
    cfg = dms.make_config(**cfg_kw,
                          eviction=dms.DMS_EVICT_IMMEDIATE if mode == "immediate" else dms.DMS_EVICT_DELAYED,
                          decision_source=dms.DMS_DECIDE_QUERY if decide else dms.DMS_DECIDE_CALLER,
                          decision_bias=bias)
    cache = dms.DmsCache(cfg)
    orc = PagedKVOracle(cfg.max_seqs, cfg.num_kv_heads, cfg.window, cfg.page_size, cfg.num_pages,
                        cfg.max_pages_per_head, cfg.head_dim, mode=mode)
    return dms, cfg, cache, orc


def _use_query_decisions(inputs, g, bias):
    """Replace each sequence's flags by the decisions its queries give."""
    for x in inputs.values():
        x.flags = oracle.query_decisions(bf16_to_f32(x.q), g, bias)


def _append(dms, cache, orc, seqs, inputs, lo, hi):
    import torch
    lens = [hi[s] - lo[s] for s in seqs]
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    cat = lambda name: np.concatenate([getattr(inputs[s], name)[lo[s]:hi[s]] for s in seqs])
    dms.dms_append_chunk(cache.ctx, 0, len(seqs), to_dev(np.array(seqs, np.int32)), to_dev(cu),
                         int(cu[-1]), int(max(lens)), to_dev(cat("k")), to_dev(cat("v")),
                         to_dev(cat("flags")))
    orc.append_chunk(seqs, [inputs[s].flags[lo[s]:hi[s]] for s in seqs],
                     [bf16_to_f32(inputs[s].k[lo[s]:hi[s]]) for s in seqs],
                     [bf16_to_f32(inputs[s].v[lo[s]:hi[s]]) for s in seqs])
    torch.cuda.synchronize()
    assert dms.dms_status(cache.ctx) == 0


def _decode(dms, cfg, cache, orc, seqs, inputs, t0, steps, decide, mode):
    import torch
    g = cfg.group_size
    sid = to_dev(np.array(seqs, np.int32))
    for step in range(steps):
        ts = {s: t0[s] + step for s in seqs}
        q = np.stack([inputs[s].q[ts[s]] for s in seqs])
        k = np.stack([inputs[s].k[ts[s]] for s in seqs])
        v = np.stack([inputs[s].v[ts[s]] for s in seqs])
        f = np.stack([inputs[s].flags[ts[s]] for s in seqs])
        out = torch.full((len(seqs), cfg.num_kv_heads * g, cfg.head_dim), float("nan"), device="cuda")
        if decide:
            dec = torch.full((len(seqs), cfg.num_kv_heads), 7, dtype=torch.uint8, device="cuda")
            dms.dms_decode_step_q(cache.ctx, 0, len(seqs), sid, to_dev(q), to_dev(k), to_dev(v),
                                  dec, out)
        else:
            dms.dms_decode_step(cache.ctx, 0, len(seqs), sid, to_dev(q), to_dev(k), to_dev(v),
                                to_dev(f), out)
        torch.cuda.synchronize()
        assert dms.dms_status(cache.ctx) == 0
        if decide:
            assert np.array_equal(dec.cpu().numpy(), f), step
        orc.append(seqs, f, bf16_to_f32(k), bf16_to_f32(v))
        qa = oracle.zero_borrowed_neuron(bf16_to_f32(q), g) if decide else bf16_to_f32(q)
        got = out.cpu().numpy()
        assert np.abs(got - orc.decode(seqs, qa, g)).max() <= ATOL, step
        if step % 8 == 0:
            for i, s in enumerate(seqs):
                t = ts[s]
                qd = bf16_to_f32(inputs[s].q[t:t + 1])
                if decide:
                    qd = oracle.zero_borrowed_neuron(qd, g)
                ref = dense_dms_attention(qd, bf16_to_f32(inputs[s].k[:t + 1]),
                                          bf16_to_f32(inputs[s].v[:t + 1]), inputs[s].flags[:t + 1],
                                          cfg.window, g, t_query=[t], mode=mode)
                assert np.abs(got[i] - ref[0]).max() <= ATOL, (step, s)
        compare_state(cache.export(0), orc, seqs)


@pytest.mark.parametrize("mode,decide,w,P,p,bias", [
    ("immediate", False, 16, 32, 0.5, 0.0),
    ("immediate", False, 5, 64, 0.9, 0.0),
    ("immediate", False, 1, 32, 0.7, 0.0),
    ("delayed", True, 16, 32, 0.0, -0.3),
    ("delayed", True, 7, 64, 0.0, 0.8),
    ("immediate", True, 12, 32, 0.0, 0.2),
])
def test_decode_steps(mode, decide, w, P, p, bias):
    dms, cfg, cache, orc = _setup(mode, decide, bias, window=w, page_size=P)
    seqs = [2, 0, 3]
    T0 = {2: 150, 0: 37, 3: 96}
    steps = 40
    inputs = {s: SeqInputs(71 + s, 0, s, T0[s] + steps, 2, 3, 128, p) for s in seqs}
    if decide:
        _use_query_decisions(inputs, 3, bias)
    _append(dms, cache, orc, seqs, inputs, {s: 0 for s in seqs}, T0)
    compare_state(cache.export(0), orc, seqs)
    _decode(dms, cfg, cache, orc, seqs, inputs, T0, steps, decide, mode)
    compare_pool(cache, 0, cache.export(0), seqs, inputs)
    cache.close()


def _prefill(mode, decide, w, P, p, bias, chunks, d=128, g=3, decisions_buffer=True):
    import torch
    dms, cfg, cache, orc = _setup(mode, decide, bias, window=w, page_size=P, head_dim=d, group_size=g)
    H = cfg.num_kv_heads
    seqs = [1, 3, 0]
    lens = {1: 420, 3: 77, 0: 260}
    inputs = {s: SeqInputs(300 + s, 0, s, lens[s], H, g, d, p) for s in seqs}
    if decide:
        _use_query_decisions(inputs, g, bias)
    cur = {s: 0 for s in seqs}
    ci = 0
    while any(cur[s] < lens[s] for s in seqs):
        C = chunks[ci % len(chunks)]
        ci += 1
        ls = [min(C, lens[s] - cur[s]) for s in seqs]
        cu = np.concatenate([[0], np.cumsum(ls)]).astype(np.int32)
        cat = lambda name: np.concatenate([getattr(inputs[s], name)[cur[s]:cur[s] + l]
                                           for s, l in zip(seqs, ls)])
        T = int(cu[-1])
        out = torch.full((T, H * g, d), float("nan"), device="cuda")
        sid = to_dev(np.array(seqs, np.int32))
        if decide:
            dec = torch.full((T, H), 7, dtype=torch.uint8, device="cuda") if decisions_buffer else None
            dms.dms_prefill_chunk_q(cache.ctx, 0, len(seqs), sid, to_dev(cu), T, int(max(ls)),
                                    to_dev(cat("q")), to_dev(cat("k")), to_dev(cat("v")), dec, out)
        else:
            dms.dms_prefill_chunk(cache.ctx, 0, len(seqs), sid, to_dev(cu), T, int(max(ls)),
                                  to_dev(cat("q")), to_dev(cat("k")), to_dev(cat("v")),
                                  to_dev(cat("flags")), out)
        torch.cuda.synchronize()
        assert dms.dms_status(cache.ctx) == 0
        if decide and decisions_buffer:
            assert np.array_equal(dec.cpu().numpy(), cat("flags"))
        got = out.cpu().numpy()
        for i, (s, l) in enumerate(zip(seqs, ls)):
            if l == 0:
                continue
            tq = np.arange(cur[s], cur[s] + l)
            qq = bf16_to_f32(inputs[s].q[tq])
            if decide:
                qq = oracle.zero_borrowed_neuron(qq, g)
            # the history the queries may see, plus the decisions of later
            # chunk positions (immediate eviction reads decision j + w)
            hist = tq[-1] + 1
            ref = dense_dms_attention(qq, bf16_to_f32(inputs[s].k[:hist]), bf16_to_f32(inputs[s].v[:hist]),
                                      inputs[s].flags[:hist], w, g, t_query=tq, mode=mode)
            err = np.abs(got[cu[i]:cu[i + 1]] - ref).max()
            assert err <= ATOL, (s, cur[s], err)
        orc.append_chunk(seqs, [inputs[s].flags[cur[s]:cur[s] + l] for s, l in zip(seqs, ls)],
                         [bf16_to_f32(inputs[s].k[cur[s]:cur[s] + l]) for s, l in zip(seqs, ls)],
                         [bf16_to_f32(inputs[s].v[cur[s]:cur[s] + l]) for s, l in zip(seqs, ls)])
        for s, l in zip(seqs, ls):
            cur[s] += l
        compare_state(cache.export(0), orc, seqs)
    compare_pool(cache, 0, cache.export(0), seqs, inputs)
    cache.close()


@pytest.mark.parametrize("w,P,p,chunks,d,g", [
    (16, 32, 0.5, [300], 128, 3),
    (40, 64, 0.8, [100, 7, 64], 128, 5),
    (3, 32, 0.6, [33], 64, 2),
    (64, 64, 0.9, [128, 129], 128, 4),
])
def test_immediate_prefill(w, P, p, chunks, d, g):
    _prefill("immediate", False, w, P, p, 0.0, chunks, d, g)


@pytest.mark.parametrize("mode,bias,chunks", [
    ("delayed", -0.3, [300]), ("delayed", 0.9, [50, 128]), ("immediate", 0.1, [64, 300]),
])
def test_query_decisions_prefill(mode, bias, chunks):
    _prefill(mode, True, 16, 32, 0.0, bias, chunks)


def test_query_decisions_prefill_without_output_buffer():
    _prefill("delayed", True, 16, 32, 0.0, 0.2, [100, 300], decisions_buffer=False)


def test_query_mode_attend_only_zeroes_the_neuron():
    import torch
    dms, cfg, cache, orc = _setup("delayed", True, 0.0)
    seqs = [1, 2]
    inputs = {s: SeqInputs(900 + s, 0, s, 120, 2, 3, 128, 0.5) for s in seqs}
    # a large borrowed neuron would dominate the scores if it were not zeroed
    for x in inputs.values():
        x.q[:, ::3, 0] = 0x4480   # 1024.0
    _append(dms, cache, orc, seqs, inputs, {s: 0 for s in seqs}, {s: 120 for s in seqs})
    q = np.stack([inputs[s].q[119] for s in seqs])
    out = torch.full((2, 6, 128), float("nan"), device="cuda")
    dms.dms_decode(cache.ctx, 0, 2, to_dev(np.array(seqs, np.int32)), to_dev(q), out)
    torch.cuda.synchronize()
    assert dms.dms_status(cache.ctx) == 0
    ref = orc.decode(seqs, oracle.zero_borrowed_neuron(bf16_to_f32(q), 3), 3)
    assert np.abs(out.cpu().numpy() - ref).max() <= ATOL
    cache.close()
