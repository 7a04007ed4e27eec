"""HIP-graph capture of decode steps: a captured sequence of dms_decode_step
calls (two layers) is replayed several times, with eager work and
synchronisations in between, and every replay must match an eager run of the
same steps on an identical cache -- outputs bitwise, state bit-exact."""
import numpy as np
import pytest

from dms_testlib import SeqInputs, to_dev

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("fp8,budget", [(False, 0), (True, 0), (False, 2), (True, 2)])
def test_graph_replays_match_eager(fp8, budget):
    """Dense and page-retrieval steps (budget 2 of ~3 pages per head), bf16 and
    FP8 pages: the retrieval step is six launches per layer, all captured."""
    import torch
    from paper_2506_05345_amd import dms
    kw = dict(num_layers=2, max_seqs=3, num_kv_heads=2, group_size=5, head_dim=128, window=16,
              page_size=64, num_pages=200, max_pages_per_head=32, max_chunk_tokens=3 * 600,
              kv_format=dms.DMS_KV_FP8 if fp8 else dms.DMS_KV_BF16, quest_page_budget=budget)
    cfg = dms.make_config(**kw)
    eager, graphed = dms.DmsCache(cfg), dms.DmsCache(cfg)
    seqs = [2, 0, 1]
    T0, REPLAYS = 500, 5
    inp = {s: SeqInputs(61, 0, s, T0 + REPLAYS, 2, 5, 128, 0.75) for s in seqs}
    sid = to_dev(np.array(seqs, np.int32))
    cu = to_dev(np.array([0, T0, 2 * T0, 3 * T0], np.int32))
    cat = lambda name: to_dev(np.concatenate([getattr(inp[s], name)[:T0] for s in seqs]))
    for c in (eager, graphed):
        for layer in (0, 1):
            dms.dms_append_chunk(c.ctx, layer, 3, sid, cu, 3 * T0, T0, cat("k"), cat("v"), cat("flags"))
    torch.cuda.synchronize()
    # static input buffers the graph reads; refilled before every replay
    qb = torch.empty((3, 10, 128), dtype=torch.bfloat16, device="cuda")
    kb = torch.empty((3, 2, 128), dtype=torch.bfloat16, device="cuda")
    vb = torch.empty_like(kb)
    fb = torch.empty((3, 2), dtype=torch.uint8, device="cuda")
    outs = [torch.empty((3, 10, 128), device="cuda") for _ in range(2)]

    def fill(t):
        qb.copy_(to_dev(np.stack([inp[s].q[t] for s in seqs])))
        kb.copy_(to_dev(np.stack([inp[s].k[t] for s in seqs])))
        vb.copy_(to_dev(np.stack([inp[s].v[t] for s in seqs])))
        fb.copy_(to_dev(np.stack([inp[s].flags[t] for s in seqs])))

    def step(c):
        for layer in (0, 1):
            dms.dms_decode_step(c.ctx, layer, 3, sid, qb, kb, vb, fb, outs[layer])

    fill(T0)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step(graphed)
    torch.cuda.synchronize()
    # capture recorded the launches without running them: both caches agree
    assert np.array_equal(eager.export(0).pos, graphed.export(0).pos)
    for r in range(REPLAYS):
        fill(T0 + r)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = [o.clone() for o in outs]
        step(eager)                      # eager reference of the same step
        torch.cuda.synchronize()
        for layer in (0, 1):
            assert torch.equal(got[layer], outs[layer]), (r, layer)
            a, b = eager.export(layer), graphed.export(layer)
            for f in ("pos", "L", "ring_slot", "ring_flag", "page_table", "stack"):
                assert np.array_equal(getattr(a, f), getattr(b, f)), (r, layer, f)
        assert dms.dms_status(graphed.ctx) == 0 and dms.dms_status(eager.ctx) == 0
        _ = torch.ones(1000, device="cuda").sum().item()   # unrelated eager work between replays
    eager.close()
    graphed.close()
