"""GPU parity of FP8 (E4M3, power-of-two row scales) KV pages against the CPU
oracle: bookkeeping bit-exact, every live slot's codes and scales bit-exact
(the quantization is an integer decision taken in float32 on both sides),
decode outputs within 1e-2 max-abs of float64 attention over the dequantized
rows."""
import numpy as np
import pytest

from dms_testlib import ATOL, SeqInputs, bf16_to_f32, compare_pool_fp8, compare_state, to_dev
from oracle import PagedKVOracle, dense_dms_attention, fake_quantize_fp8

pytestmark = pytest.mark.gpu


def _mk(**kw):
    import torch
    from paper_2506_05345_amd import dms
    cfg = dms.make_config(kv_format=dms.DMS_KV_FP8, **kw)
    cache = dms.DmsCache(cfg)
    # freed or never-written slots hold arbitrary bytes: fill every pool with
    # NaN codes and NaN scales so that reading one shows up in the outputs
    for p in cache.pools:
        p.fill_(0xFF)
    cache.workspace.fill_(0xFF)
    dms.dms_init_state(cache.ctx)
    torch.cuda.synchronize()
    orc = PagedKVOracle(cfg.max_seqs, cfg.num_kv_heads, cfg.window, cfg.page_size, cfg.num_pages,
                        cfg.max_pages_per_head, cfg.head_dim, kv_format="fp8")
    return dms, cfg, cache, orc


def _compare_pool_fp8(cache, orc, seqs, layer=0):
    compare_pool_fp8(cache, orc, seqs, layer)


def _append_chunks(dms, cache, orc, seqs, inputs, start, stop, chunk):
    import torch
    cur = dict(start)
    while any(cur[s] < stop[s] for s in seqs):
        lens = [min(chunk, stop[s] - cur[s]) for s in seqs]
        cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
        fl = np.concatenate([inputs[s].flags[cur[s]:cur[s] + l] for s, l in zip(seqs, lens)])
        kk = np.concatenate([inputs[s].k[cur[s]:cur[s] + l] for s, l in zip(seqs, lens)])
        vv = np.concatenate([inputs[s].v[cur[s]:cur[s] + l] for s, l in zip(seqs, lens)])
        dms.dms_append_chunk(cache.ctx, 0, len(seqs), to_dev(np.array(seqs, np.int32)), to_dev(cu),
                             int(cu[-1]), int(max(lens)), to_dev(kk), to_dev(vv), to_dev(fl))
        orc.append_chunk(seqs, [inputs[s].flags[cur[s]:cur[s] + l] for s, l in zip(seqs, lens)],
                         [bf16_to_f32(inputs[s].k[cur[s]:cur[s] + l]) for s, l in zip(seqs, lens)],
                         [bf16_to_f32(inputs[s].v[cur[s]:cur[s] + l]) for s, l in zip(seqs, lens)])
        for s, l in zip(seqs, lens):
            cur[s] += l
        torch.cuda.synchronize()
        assert dms.dms_status(cache.ctx) == 0


def _decode_steps(dms, cache, orc, seqs, inputs, t_from, nsteps, g, fused=True, dense_every=16):
    """Decode steps (fused append + attention, or dms_append then dms_decode);
    outputs against the oracle's fp8 replay and, every `dense_every` steps,
    against dense attention over the fake-quantized full history."""
    import torch
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
        if fused:
            dms.dms_decode_step(cache.ctx, 0, len(seqs), sid, to_dev(q), to_dev(k), to_dev(v),
                                to_dev(f), out)
        else:
            dms.dms_append(cache.ctx, 0, len(seqs), sid, to_dev(k), to_dev(v), to_dev(f))
            dms.dms_decode(cache.ctx, 0, len(seqs), sid, to_dev(q), out)
        torch.cuda.synchronize()
        assert dms.dms_status(cache.ctx) == 0
        orc.append(seqs, f, bf16_to_f32(k), bf16_to_f32(v))
        ref = orc.decode(seqs, bf16_to_f32(q), g)
        got = out.cpu().numpy()
        err = np.abs(got - ref).max()
        worst = max(worst, err)
        assert err <= ATOL, (step, err)
        if dense_every and step % dense_every == 0:
            for i, s in enumerate(seqs):
                t = ts[s]
                dref = dense_dms_attention(bf16_to_f32(inputs[s].q[t:t + 1]),
                                           fake_quantize_fp8(bf16_to_f32(inputs[s].k[:t + 1])),
                                           fake_quantize_fp8(bf16_to_f32(inputs[s].v[:t + 1])),
                                           inputs[s].flags[:t + 1], cfg.window, g, t_query=[t])
                assert np.abs(got[i] - dref[0]).max() <= ATOL
    return worst


@pytest.mark.parametrize("d,g,w,P,p", [(128, 5, 16, 64, 0.875), (64, 2, 3, 32, 0.5),
                                       (128, 16, 40, 256, 0.75), (64, 7, 1, 128, 0.9)])
def test_chunk_commit_and_decode(d, g, w, P, p):
    """Ragged sequences called out of id order: chunk commits (pool codes and
    scales bit-exact), then fused decode steps with ragged last tiles."""
    H = 2
    seqs = [3, 0, 2]
    dms, cfg, cache, orc = _mk(num_layers=1, max_seqs=4, num_kv_heads=H, group_size=g, head_dim=d,
                               window=w, page_size=P, num_pages=300, max_pages_per_head=64,
                               max_chunk_tokens=3 * 300)
    lens = {3: 701, 0: 95, 2: 333}
    inp = {s: SeqInputs(31, 0, s, lens[s] + 40, H, g, d, p) for s in seqs}
    _append_chunks(dms, cache, orc, seqs, inp, {s: 0 for s in seqs}, lens, 300)
    compare_state(cache.export(0), orc, seqs)
    _compare_pool_fp8(cache, orc, seqs)
    worst = _decode_steps(dms, cache, orc, seqs, inp, lens, 40, g)
    compare_state(cache.export(0), orc, seqs)
    _compare_pool_fp8(cache, orc, seqs)
    print(f"max abs err {worst:.3e}")


def test_append_then_decode_token_by_token():
    """Every token through dms_append (scatter path) and dms_decode from
    position 0: single-key steps, tiles filling one slot at a time."""
    dms, cfg, cache, orc = _mk(num_layers=1, max_seqs=2, num_kv_heads=3, group_size=4, head_dim=128,
                               window=5, page_size=32, num_pages=64, max_pages_per_head=16)
    seqs = [1, 0]
    inp = {s: SeqInputs(5, 0, s, 120, 3, 4, 128, 0.6) for s in seqs}
    _decode_steps(dms, cache, orc, seqs, inp, {0: 0, 1: 0}, 120, 4, fused=False, dense_every=7)
    compare_state(cache.export(0), orc, seqs)
    _compare_pool_fp8(cache, orc, seqs)


def test_reset_pages_reused_with_stale_codes():
    """A released sequence's pages (holding its codes) are popped by another
    sequence whose last tiles are partial: stale slots must not leak in."""
    import torch
    dms, cfg, cache, orc = _mk(num_layers=1, max_seqs=2, num_kv_heads=2, group_size=3, head_dim=64,
                               window=4, page_size=64, num_pages=40, max_pages_per_head=16,
                               max_chunk_tokens=600)
    inp0 = SeqInputs(41, 0, 0, 600, 2, 3, 64, 0.3)
    _append_chunks(dms, cache, orc, [0], {0: inp0}, {0: 0}, {0: 600}, 600)
    dms.dms_seq_reset(cache.ctx, 0, 1, to_dev(np.array([0], np.int32)))
    orc.seq_reset([0])
    torch.cuda.synchronize()
    inp1 = SeqInputs(42, 0, 1, 200, 2, 3, 64, 0.5)
    _append_chunks(dms, cache, orc, [1], {1: inp1}, {1: 0}, {1: 77}, 77)
    _decode_steps(dms, cache, orc, [1], {1: inp1}, {1: 77}, 30, 3)
    _compare_pool_fp8(cache, orc, [1])


@pytest.mark.parametrize("variant", ["peaked", "v_const", "needle", "zero_rows"])
def test_value_variants(variant):
    import torch
    dms, cfg, cache, orc = _mk(num_layers=1, max_seqs=1, num_kv_heads=1, group_size=4, head_dim=128,
                               window=16, page_size=64, num_pages=64, max_pages_per_head=32,
                               max_chunk_tokens=1024)
    T = 1000
    inp = SeqInputs(21, 0, 0, T + 1, 1, 4, 128, 0.875, q_scale=8.0 if variant == "peaked" else 1.0)
    if variant == "v_const":
        inp.v[:] = 0x3F80        # 1.0: stored exactly (code 256 at scale 2^-8)
    if variant == "needle":
        inp.k[:] = 0
        inp.q[T] = 0
        inp.q[T, :, 0] = 0x447A  # 1000.0
        inp.k[100, 0, 0] = 0x3F80
        inp.flags[100] = 0
        inp.v[100, 0, :] = 0x4000  # 2.0
        inp.k[200, 0, 0] = 0x3F80
        inp.flags[200] = 1
        inp.v[200, 0, :] = 0xC000  # -2.0
    if variant == "zero_rows":
        inp.k[::3] = 0             # all-zero rows: exponent 0, codes 0
        inp.v[1::3] = 0
    _append_chunks(dms, cache, orc, [0], {0: inp}, {0: 0}, {0: T}, 1024)
    _compare_pool_fp8(cache, orc, [0])
    _decode_steps(dms, cache, orc, [0], {0: inp}, {0: T}, 1, 4)
    if variant in ("v_const", "needle"):
        out = torch.empty((1, 4, 128), device="cuda")
        dms.dms_decode(cache.ctx, 0, 1, to_dev(np.array([0], np.int32)), to_dev(inp.q[T][None]), out)
        torch.cuda.synchronize()
        o = out.cpu().numpy()
        if variant == "v_const":
            assert np.abs(o - 1.0).max() < 4e-3
        else:
            assert np.abs(o[0, 0] - 2.0).max() < 1e-2
