"""Parity at the full sizes of the other synthetic workloads, one layer each,
in the benchmark's launch configuration (one decode wave per SIMD, 64-token
pages).  Bookkeeping of every head is compared bit-exactly with the oracle's
replay; sampled outputs against dense masked attention over the full history.

* Qwen-R1-1.5B-shaped: 32 sequences x 2 KV heads (group 6), 8192-token prompt
  through the masked chunked prefill, then all 256 decode steps; w=256,
  flags Bernoulli(7/8).
* Qwen-R1-7B-shaped: 64 sequences x 4 KV heads (group 7), contexts uniform in
  [4096, 32768], decode steps; w=256, flags Bernoulli(3/4).
* Heterogeneous stress (32B attention shape): 32 sequences x 8 KV heads
  (group 5), per-(sequence, head) eviction rate ~ Beta(7,1), contexts
  log-uniform in [1K, 128K]; one mixed step = 4096-token masked prefill for
  4 sequences plus a decode step for the other 28; w in {64, 256}.
"""
import numpy as np
import pytest

import dms_synth as sy
from dms_testlib import ATOL, bf16_to_f32, compare_state
from fullsize_lib import (Workload, build, check_decode_sample, closed_form_L,
                          decode_step_inputs, to_bf16_dev)
from oracle import PagedKVOracle, dense_dms_attention_head

pytestmark = pytest.mark.gpu


def _cache(dms, wl, lens_final, chunk_tokens):
    pages = 0
    maxp = 0
    for s in range(wl.B):
        L = closed_form_L(wl, s, int(lens_final[s]))
        need = (L + wl.P - 1) // wl.P
        pages += int(need.sum())
        maxp = max(maxp, int(need.max()))
    cfg = dms.make_config(1, wl.B, wl.H, wl.g, wl.D, wl.w, wl.P, pages + 16, maxp + 2, chunk_tokens)
    orc = PagedKVOracle(wl.B, wl.H, wl.w, wl.P, pages + 16, maxp + 2, wl.D, store_values=False)
    return dms.DmsCache(cfg), orc


def _decode(dms, cache, wl, orc, seqs, positions):
    import torch
    q, k, v, f = decode_step_inputs(wl, seqs, positions)
    out = torch.full((len(seqs), wl.H * wl.g, wl.D), float("nan"), device="cuda")
    sid = torch.as_tensor(np.asarray(seqs, np.int32), device="cuda")
    dms.dms_decode_step(cache.ctx, 0, len(seqs), sid, to_bf16_dev(q), to_bf16_dev(k),
                        to_bf16_dev(v), torch.from_numpy(f).cuda(), out)
    torch.cuda.synchronize()
    assert dms.dms_status(cache.ctx) == 0
    orc.append(list(seqs), f)
    return q, out.cpu().numpy()


def test_qwen_r1_1p5b_prefill_then_256_decode_steps():
    import torch
    from paper_2506_05345_amd import dms
    B, H, g, D, w, T, STEPS = 32, 2, 6, 128, 256, 8192, 256
    wl = Workload(1, 0, B, H, g, D, w, [T] * B, [[sy.dyadic_threshold(7 / 8)] * H] * B)
    cache, orc = _cache(dms, wl, [T + STEPS] * B, B * T)
    dev = "cuda"
    # the whole 8192-token prompt of every sequence in one masked prefill call
    seq_t = torch.arange(B, device=dev).repeat_interleave(T)
    pos_t = torch.arange(T, device=dev).repeat(B)
    heads = torch.arange(H, device=dev)
    qh = torch.arange(H * g, device=dev)
    dd = torch.arange(D, device=dev)
    vec = lambda stream, hs: sy.token_vectors_torch(wl.seed, stream, 0, seq_t[:, None, None],
                                                    hs[None, :, None], pos_t[:, None, None],
                                                    dd[None, None, :], dev)
    q, k, v = vec(sy.STREAM_Q, qh), vec(sy.STREAM_K, heads), vec(sy.STREAM_V, heads)
    f = wl.flags_dev(seq_t[:, None], heads[None, :], pos_t[:, None], dev)
    cu = torch.arange(B + 1, dtype=torch.int32, device=dev) * T
    out = torch.full((B * T, H * g, D), float("nan"), device=dev)
    sid = torch.arange(B, dtype=torch.int32, device=dev)
    dms.dms_prefill_chunk(cache.ctx, 0, B, sid, cu, B * T, T, q, k, v, f, out)
    torch.cuda.synchronize()
    assert dms.dms_status(cache.ctx) == 0
    fh = f.cpu().numpy()
    orc.append_chunk(list(range(B)), [fh[s * T:(s + 1) * T] for s in range(B)])
    compare_state(cache.export(0), orc, range(B))
    # sampled prefill outputs, including the first and last positions
    for (s, h) in [(0, 0), (13, 1), (31, 1)]:
        tq = np.array([0, 1, 255, 256, 257, 4000, 8190, 8191])
        kh = wl.vec_host(sy.STREAM_K, s, h, np.arange(T))
        vh = wl.vec_host(sy.STREAM_V, s, h, np.arange(T))
        fl = wl.flags_host(s, np.arange(T))[:, h]
        qq = np.stack([sy.token_vectors_np(wl.seed, sy.STREAM_Q, 0, s, h * g + np.arange(g)[:, None],
                                           t, np.arange(D)[None, :]) for t in tq])
        ref = dense_dms_attention_head(bf16_to_f32(qq), bf16_to_f32(kh), bf16_to_f32(vh), fl, w, tq)
        got = out[torch.as_tensor(s * T + tq, device=dev)][:, h * g:(h + 1) * g].cpu().numpy()
        assert np.abs(got - ref).max() <= ATOL
    del q, k, v, out
    # all 256 decode steps
    for step in range(STEPS):
        t = T + step
        q_bits, got = _decode(dms, cache, wl, orc, list(range(B)), [t] * B)
        if step % 64 == 0 or step == STEPS - 1:
            compare_state(cache.export(0), orc, range(B))
            for (s, h) in [(5, 0), (30, 1)]:
                check_decode_sample(wl, got[s, h * g:(h + 1) * g], q_bits[s, h * g:(h + 1) * g], s, h, t)
    assert np.array_equal(cache.export(0).L, np.stack([closed_form_L(wl, s, T + STEPS) for s in range(B)]))
    cache.close()


def test_qwen_r1_7b_ragged_contexts():
    from paper_2506_05345_amd import dms
    B, H, g, D, w, STEPS = 64, 4, 7, 128, 256, 3
    ctx = np.random.default_rng(2).integers(4096, 32768 + 1, size=B)
    wl = Workload(2, 0, B, H, g, D, w, ctx, [[sy.dyadic_threshold(3 / 4)] * H] * B)
    cache, orc = _cache(dms, wl, ctx + STEPS, 4096 * B)
    build(dms, cache, wl, orc, np.zeros(B, np.int64), ctx, 4096)
    view = cache.export(0)
    compare_state(view, orc, range(B))
    assert np.array_equal(view.L, np.stack([closed_form_L(wl, s, int(ctx[s])) for s in range(B)]))
    for step in range(STEPS):
        q_bits, got = _decode(dms, cache, wl, orc, list(range(B)), ctx + step)
    compare_state(cache.export(0), orc, range(B))
    longest, shortest = int(np.argmax(ctx)), int(np.argmin(ctx))
    for (s, h) in [(longest, 3), (shortest, 0), (17, 2)]:
        t = int(ctx[s]) + STEPS - 1
        check_decode_sample(wl, got[s, h * g:(h + 1) * g], q_bits[s, h * g:(h + 1) * g], s, h, t)
    cache.close()


@pytest.mark.parametrize("w,seed", [(64, 4), (256, 5)])
def test_heterogeneous_stress_mixed_step(w, seed):
    import torch
    from paper_2506_05345_amd import dms
    B, H, g, D, C = 32, 8, 5, 128, 4096
    rng = np.random.default_rng(seed)
    ctx = np.exp(rng.uniform(np.log(1024), np.log(131072), size=B)).astype(np.int64)
    thr = sy.beta71_rates_np(seed, 0, np.arange(B)[:, None], np.arange(H)[None, :])
    wl = Workload(seed, 0, B, H, g, D, w, ctx, thr)
    prefill = np.arange(28, 32)
    decode = np.arange(28)
    final = ctx.copy()
    final[prefill] += C
    final[decode] += 1
    cache, orc = _cache(dms, wl, final, max(4096 * B, C * len(prefill)))
    build(dms, cache, wl, orc, np.zeros(B, np.int64), ctx, 4096)
    view = cache.export(0)
    compare_state(view, orc, range(B))
    L = view.L
    assert L.max() / L.mean() > 4          # heads really are ragged
    # mixed step: masked prefill of 4096 tokens for 4 sequences ...
    dev = "cuda"
    seq_t = torch.as_tensor(prefill, device=dev).repeat_interleave(C)
    pos_t = torch.cat([torch.arange(int(ctx[s]), int(ctx[s]) + C, device=dev) for s in prefill])
    heads = torch.arange(H, device=dev)
    dd = torch.arange(D, device=dev)
    vec = lambda stream, hs: sy.token_vectors_torch(wl.seed, stream, 0, seq_t[:, None, None],
                                                    hs[None, :, None], pos_t[:, None, None],
                                                    dd[None, None, :], dev)
    q, k, v = vec(sy.STREAM_Q, torch.arange(H * g, device=dev)), vec(sy.STREAM_K, heads), vec(sy.STREAM_V, heads)
    f = wl.flags_dev(seq_t[:, None], heads[None, :], pos_t[:, None], dev)
    cu = torch.arange(len(prefill) + 1, dtype=torch.int32, device=dev) * C
    out = torch.full((len(prefill) * C, H * g, D), float("nan"), device=dev)
    dms.dms_prefill_chunk(cache.ctx, 0, len(prefill), torch.as_tensor(prefill.astype(np.int32), device=dev),
                          cu, len(prefill) * C, C, q, k, v, f, out)
    fh = f.cpu().numpy()
    orc.append_chunk(list(prefill), [fh[i * C:(i + 1) * C] for i in range(len(prefill))])
    # ... and a decode step for the other 28 (pages are popped in call order)
    q_bits, got = _decode(dms, cache, wl, orc, list(decode), ctx[decode])
    compare_state(cache.export(0), orc, range(B))
    # sampled decode outputs (longest-context decode head included)
    s_long = int(decode[np.argmax(ctx[decode])])
    for (s, h) in [(s_long, 0), (3, 7)]:
        check_decode_sample(wl, got[s, h * g:(h + 1) * g], q_bits[s, h * g:(h + 1) * g], s, h, int(ctx[s]))
    # sampled prefill outputs
    for i, h in [(0, 2), (3, 6)]:
        s = int(prefill[i])
        T = int(ctx[s]) + C
        kh = wl.vec_host(sy.STREAM_K, s, h, np.arange(T))
        vh = wl.vec_host(sy.STREAM_V, s, h, np.arange(T))
        fl = wl.flags_host(s, np.arange(T))[:, h]
        loc = np.array([0, 1, w - 1, w, 2000, C - 1])
        tq = int(ctx[s]) + loc
        qq = np.stack([sy.token_vectors_np(wl.seed, sy.STREAM_Q, 0, s, h * g + np.arange(g)[:, None],
                                           t, np.arange(D)[None, :]) for t in tq])
        ref = dense_dms_attention_head(bf16_to_f32(qq), bf16_to_f32(kh), bf16_to_f32(vh), fl, w, tq)
        gotp = out[torch.as_tensor(i * C + loc, device=dev)][:, h * g:(h + 1) * g].cpu().numpy()
        assert np.abs(gotp - ref).max() <= ATOL
    cache.close()
