"""dms_decode_step_static (planner output, split-K partials and arrival
counters in the library's static device scratch, nothing allocated) against
dms_decode_step (over the context's workspace) and against the CPU oracle:
two contexts with identical state take identical decode steps, one through
each entry point.  dms_decode_step may split a call differently (its fused
launch sizes the wave count to the call), so the two outputs agree up to
float32 reassociation: both within 1e-2 of each other and of the oracle's
replay; bookkeeping bit-exact on both sides.  Two calls in a row, the second with
fewer sequences, then a call from a third context of another shape on the
same GPU (the scratch keeps the last call's contents)."""
import numpy as np
import pytest

from dms_testlib import ATOL, SeqInputs, bf16_to_f32, compare_state, to_dev
from oracle import PagedKVOracle

pytestmark = pytest.mark.gpu


def _setup(fmt, S, H, g, d, w, lengths, seed):
    import torch
    from paper_2506_05345_amd import dms
    P = 64
    maxp = (max(lengths) + 8) // P + 2
    cfg = dms.make_config(1, S, H, g, d, w, P, S * H * maxp + 8, maxp, 4096, kv_format=fmt)
    caches = []
    for _ in range(2):
        c = dms.DmsCache(cfg)
        # stale bytes everywhere a call might read by mistake
        for p in c.pools:
            p.fill_(0xFF)
        c.workspace.fill_(0xFF)
        dms.dms_init_state(c.ctx)
        caches.append(c)
    T = max(lengths) + 4
    inputs = {s: SeqInputs(seed, 0, s, T, H, g, d, 0.75) for s in range(S)}
    orc = PagedKVOracle(S, H, w, P, cfg.num_pages, maxp, d,
                        kv_format="fp8" if fmt == dms.DMS_KV_FP8 else "bf16")
    seqs = list(range(S))
    cur = [0] * S
    while any(cur[s] < lengths[s] for s in seqs):
        # the same chunks on both contexts and in the oracle (page pops follow calls)
        lens = [min(4096 // S, lengths[s] - cur[s]) for s in seqs]
        cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
        fl = np.concatenate([inputs[s].flags[cur[s]:cur[s] + l] for s, l in zip(seqs, lens)])
        kk = np.concatenate([inputs[s].k[cur[s]:cur[s] + l] for s, l in zip(seqs, lens)])
        vv = np.concatenate([inputs[s].v[cur[s]:cur[s] + l] for s, l in zip(seqs, lens)])
        for c in caches:
            dms.dms_append_chunk(c.ctx, 0, S, to_dev(np.array(seqs, np.int32)), to_dev(cu),
                                 int(cu[-1]), int(max(lens)), to_dev(kk), to_dev(vv), to_dev(fl))
        orc.append_chunk(seqs, [inputs[s].flags[cur[s]:cur[s] + l] for s, l in zip(seqs, lens)],
                         [bf16_to_f32(inputs[s].k[cur[s]:cur[s] + l]) for s, l in zip(seqs, lens)],
                         [bf16_to_f32(inputs[s].v[cur[s]:cur[s] + l]) for s, l in zip(seqs, lens)])
        for s, l in zip(seqs, lens):
            cur[s] += l
    torch.cuda.synchronize()
    for c in caches:
        assert dms.dms_status(c.ctx) == 0
    return dms, cfg, caches, inputs, orc


def _step_both(dms, cfg, caches, inputs, orc, seqs, pos):
    """One decode step of `seqs` (position pos[s]) on cache 0 through
    dms_decode_step and on cache 1 through dms_decode_step_static."""
    import torch
    g = cfg.group_size
    Hq, d = cfg.num_kv_heads * g, cfg.head_dim
    sid = to_dev(np.array(seqs, np.int32))
    q = np.stack([inputs[s].q[pos[s]] for s in seqs])
    k = np.stack([inputs[s].k[pos[s]] for s in seqs])
    v = np.stack([inputs[s].v[pos[s]] for s in seqs])
    f = np.stack([inputs[s].flags[pos[s]] for s in seqs])
    outs = []
    for i, c in enumerate(caches):
        out = torch.full((len(seqs), Hq, d), float("nan"), device="cuda")
        fn = dms.dms_decode_step if i == 0 else dms.dms_decode_step_static
        print(f"[no-alloc] {fn.__name__} n={len(seqs)} fmt={cfg.kv_format}", flush=True)
        fn(c.ctx, 0, len(seqs), sid, to_dev(q), to_dev(k), to_dev(v), to_dev(f), out)
        torch.cuda.synchronize()
        assert dms.dms_status(c.ctx) == 0
        outs.append(out.cpu().numpy())
    orc.append(seqs, f, bf16_to_f32(k), bf16_to_f32(v))
    ref = orc.decode(seqs, bf16_to_f32(q), g)
    assert np.isfinite(outs[0]).all() and np.isfinite(outs[1]).all()
    assert float(np.abs(outs[0] - outs[1]).max()) <= ATOL
    err = float(np.abs(outs[1] - ref).max())
    assert err <= ATOL, err
    assert float(np.abs(outs[0] - ref).max()) <= ATOL
    v0, v1 = caches[0].export(0), caches[1].export(0)
    compare_state(v1, orc, range(cfg.max_seqs))
    compare_state(v0, orc, range(cfg.max_seqs))
    for s in seqs:
        pos[s] += 1
    return err


@pytest.mark.parametrize("fmt", [0, 1])
def test_static_scratch_decode_matches_workspace_decode(fmt):
    # ragged histories: heads split over many waves (batched merge), over a
    # few (register merge) and heads inside one wave; a 1-token history
    lengths = [3900, 2600, 700, 33, 1, 1900, 1250, 3100]
    dms, cfg, caches, inputs, orc = _setup(fmt, 8, 4, 5, 128, 64, lengths, seed=71 + fmt)
    pos = {s: lengths[s] for s in range(8)}
    try:
        # two calls in a row, the second with fewer sequences (other order)
        _step_both(dms, cfg, caches, inputs, orc, [0, 1, 2, 3, 4, 5, 6, 7], pos)
        _step_both(dms, cfg, caches, inputs, orc, [6, 1, 3], pos)
        _step_both(dms, cfg, caches, inputs, orc, [0, 1, 2, 3, 4, 5, 6, 7], pos)
    finally:
        for c in caches:
            c.close()


def test_static_scratch_shared_by_contexts_of_another_shape():
    # a context of another shape (head_dim 64, group 3) uses the same GPU's
    # scratch right after the calls of the test above or of a fresh process
    dms, cfg, caches, inputs, orc = _setup(0, 5, 3, 3, 64, 16, [500, 2000, 17, 3000, 64], seed=5)
    pos = {s: l for s, l in enumerate([500, 2000, 17, 3000, 64])}
    try:
        _step_both(dms, cfg, caches, inputs, orc, [4, 3, 2, 1, 0], pos)
        _step_both(dms, cfg, caches, inputs, orc, [3], pos)
    finally:
        for c in caches:
            c.close()


def test_static_scratch_refuses_calls_beyond_its_size():
    import torch
    from paper_2506_05345_amd import dms
    # 4096 sequences x 8 KV heads x group 16 at head_dim 128 need ~290 MB of partials
    cfg = dms.make_config(1, 4096, 8, 16, 128, 16, 32, 8, 1, 0)
    cache = dms.DmsCache(cfg)
    try:
        n = 4096
        sid = torch.arange(n, dtype=torch.int32, device="cuda")
        q = torch.zeros((n, 128, 128), dtype=torch.bfloat16, device="cuda")
        kv = torch.zeros((n, 8, 128), dtype=torch.bfloat16, device="cuda")
        fl = torch.zeros((n, 8), dtype=torch.uint8, device="cuda")
        out = torch.zeros((n, 128, 128), dtype=torch.float32, device="cuda")
        with pytest.raises(dms.DmsError) as e:
            dms.dms_decode_step_static(cache.ctx, 0, n, sid, q, kv, kv, fl, out)
        assert e.value.code == dms.DMS_ERR_SCRATCH
        torch.cuda.synchronize()
        # nothing was enqueued: the state is untouched
        assert dms.dms_status(cache.ctx) == 0
        assert int(cache.export(0).pos.max()) == 0
        # unsupported page formats are refused on the host
    finally:
        cache.close()
    cfg = dms.make_config(1, 2, 1, 4, 576, 16, 64, 8, 2, 0, kv_format=dms.DMS_KV_MLA)
    cache = dms.DmsCache(cfg)
    try:
        assert dms.lib().dms_decode_step_static(cache.ctx, 0, 1, 0x100, 0x100, 0x100, 0x100, 0x100,
                                                0x100, None) == dms.DMS_ERR_UNSUPPORTED
    finally:
        cache.close()
