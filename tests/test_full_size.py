"""Parity at the full Qwen-R1-32B-shaped size, one layer, in the launch
configuration the benchmark times: 128 sequences x 8 KV heads (group 5,
head_dim 128), 32768 context tokens appended in 4096-token chunks, w=256,
flags Bernoulli(7/8), then decode steps.

Checked: every head's bookkeeping bit-exactly against the oracle's replay
(retained lengths, positions, rings, page tables, slot owners, free stack);
the decode outputs of every query head of 16 sequences spread over the batch
and of every head whose tiles the planner spreads over three or more decode
waves, against dense masked attention over the full history (max-abs 1e-2);
and, on sampled (sequence, KV head) pairs, the pool contents at every live
slot."""
import numpy as np
import pytest

import dms_synth as sy
from dms_testlib import ATOL, bf16_to_f32, compare_state
from oracle import PagedKVOracle, dense_dms_attention_head

pytestmark = pytest.mark.gpu

SEED, LAYER = 3, 5
B, H, G, D, W, P, CTX, CHUNK, P_EVICT = 128, 8, 5, 128, 256, 64, 32768, 4096, 7 / 8
STEPS = 3
SAMPLES = [(0, 0), (17, 3), (64, 7), (127, 5), (90, 1), (33, 6)]
FULL_SEQS = list(range(0, B, 8))   # every query head of these sequences


def wave_spans(L, waves):
    """Decode waves holding each head's tiles, as the planner splits the call:
    the heads' 32-slot tiles laid end to end in call order, wave w taking
    tiles [w * total / W, (w + 1) * total / W).  L [n, H] retained lengths."""
    tiles = (L.reshape(-1).astype(np.int64) + 31) // 32
    cum = np.concatenate([[0], np.cumsum(tiles)])
    total = int(cum[-1])
    bounds = np.arange(waves + 1, dtype=np.int64) * total // waves
    first = np.searchsorted(bounds, cum[:-1], side="right") - 1          # bounds[w] <= c0
    last = np.searchsorted(bounds[1:], cum[1:], side="left")             # bounds[w + 1] >= c1
    return (last - first + 1).reshape(L.shape)


def test_full_size_layer():
    import torch
    from paper_2506_05345_amd import dms

    dev = "cuda"
    seqs_np = np.arange(B)
    # host flags of every (seq, head, position): the oracle replays them
    pos_all = np.arange(CTX + STEPS)
    flags_host = sy.flags_np(SEED, P_EVICT, LAYER, seqs_np[:, None, None],
                             np.arange(H)[None, None, :], pos_all[None, :, None])   # [B, T, H]
    L0 = np.minimum(W, CTX) + (flags_host[:, : CTX - W] == 0).sum(axis=1)
    maxp = int((L0.max() + STEPS + P - 1) // P) + 1
    num_pages = int(((L0 + STEPS + P - 1) // P).sum()) + 16
    cfg = dms.make_config(1, B, H, G, D, W, P, num_pages, maxp, CHUNK * B)
    cache = dms.DmsCache(cfg)
    orc = PagedKVOracle(B, H, W, P, num_pages, maxp, D, store_values=False)
    sid = torch.arange(B, dtype=torch.int32, device=dev)
    seqs_t = torch.arange(B, device=dev)
    heads_t = torch.arange(H, device=dev)
    for c0 in range(0, CTX, CHUNK):
        k = sy.seq_chunk_vectors_torch(SEED, sy.STREAM_K, LAYER, seqs_np, H, c0, CHUNK, D, dev)
        v = sy.seq_chunk_vectors_torch(SEED, sy.STREAM_V, LAYER, seqs_np, H, c0, CHUNK, D, dev)
        pos = torch.arange(c0, c0 + CHUNK, device=dev)
        f = sy.flags_torch(SEED, P_EVICT, LAYER, seqs_t[:, None, None], heads_t[None, None, :],
                           pos[None, :, None], dev)
        assert np.array_equal(f.cpu().numpy(), flags_host[:, c0:c0 + CHUNK])
        cu = torch.arange(B + 1, dtype=torch.int32, device=dev) * CHUNK
        dms.dms_append_chunk(cache.ctx, 0, B, sid, cu, B * CHUNK, CHUNK,
                             k.reshape(B * CHUNK, H, D), v.reshape(B * CHUNK, H, D),
                             f.reshape(B * CHUNK, H))
        orc.append_chunk(list(range(B)), [flags_host[s, c0:c0 + CHUNK] for s in range(B)])
        del k, v
    torch.cuda.synchronize()
    assert dms.dms_status(cache.ctx) == 0
    view = cache.export(0)
    assert np.array_equal(view.L, L0)                  # closed form
    compare_state(view, orc, range(B))                 # full bookkeeping

    # decode steps with the benchmark's launch configuration
    dd = np.arange(D)
    for step in range(STEPS):
        t = CTX + step
        q = sy.token_vectors_np(SEED, sy.STREAM_Q, LAYER, seqs_np[:, None, None],
                                np.arange(H * G)[None, :, None], t, dd[None, None, :])
        k = sy.token_vectors_np(SEED, sy.STREAM_K, LAYER, seqs_np[:, None, None],
                                np.arange(H)[None, :, None], t, dd[None, None, :])
        v = sy.token_vectors_np(SEED, sy.STREAM_V, LAYER, seqs_np[:, None, None],
                                np.arange(H)[None, :, None], t, dd[None, None, :])
        f = np.ascontiguousarray(flags_host[:, t])
        to = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(dev).view(torch.bfloat16)
        out = torch.full((B, H * G, D), float("nan"), device=dev)
        dms.dms_decode_step(cache.ctx, 0, B, sid, to(q), to(k), to(v), torch.from_numpy(f).to(dev), out)
        torch.cuda.synchronize()
        assert dms.dms_status(cache.ctx) == 0
        orc.append(list(range(B)), f)
        got = out.cpu().numpy()
        assert np.isfinite(got).all()
        view = cache.export(0)
        compare_state(view, orc, range(B))
        if step == STEPS - 1:
            # every query head of FULL_SEQS, every head spread over >= 3 waves
            props = torch.cuda.get_device_properties(0)
            n_waves = min(props.multi_processor_count * 4, 8192)
            span = wave_spans(view.L, n_waves)
            check = sorted({(s, h) for s in FULL_SEQS for h in range(H)} |
                           {(int(s), int(h)) for s, h in zip(*np.nonzero(span >= 3))} |
                           set(SAMPLES))
            print(f"[full-size] comparing {len(check)} KV heads ({int((span >= 3).sum())} over "
                  f">= 3 waves, widest {int(span.max())}) at t={t}", flush=True)
            worst = 0.0
            by_seq = {}
            for (s, h) in check:
                by_seq.setdefault(s, []).append(h)
            for s, hs in by_seq.items():
                kd = sy.seq_chunk_vectors_torch(SEED, sy.STREAM_K, LAYER, [s], H, 0, t + 1, D, dev)
                vd = sy.seq_chunk_vectors_torch(SEED, sy.STREAM_V, LAYER, [s], H, 0, t + 1, D, dev)
                ks, vs = kd[0].float().cpu().numpy(), vd[0].float().cpu().numpy()
                del kd, vd
                for h in hs:
                    ref = dense_dms_attention_head(bf16_to_f32(q[s, h * G:(h + 1) * G])[None],
                                                   ks[:, h], vs[:, h], flags_host[s, : t + 1, h],
                                                   W, [t])[0]
                    err = float(np.abs(got[s, h * G:(h + 1) * G] - ref).max())
                    assert err <= ATOL, (s, h, int(span[s, h]), err)
                    worst = max(worst, err)
            print(f"[full-size] worst max-abs error {worst:.2e}", flush=True)
            for (s, h) in SAMPLES:
                hist = np.arange(t + 1)
                kh = sy.head_sequence_np(SEED, sy.STREAM_K, LAYER, s, h, hist, D)
                vh = sy.head_sequence_np(SEED, sy.STREAM_V, LAYER, s, h, hist, D)
                ref = dense_dms_attention_head(bf16_to_f32(q[s, h * G:(h + 1) * G])[None],
                                               bf16_to_f32(kh), bf16_to_f32(vh),
                                               flags_host[s, : t + 1, h], W, [t])[0]
                err = np.abs(got[s, h * G:(h + 1) * G] - ref).max()
                assert err <= ATOL, (s, h, err)
                # pool contents of every live slot of this head
                Lh = int(view.L[s, h])
                pages = view.page_table[s, h, : (Lh + P - 1) // P]
                for i, pg in enumerate(pages):
                    kk, vv = cache.pool_page_kv(0, int(pg))
                    slots = np.arange(i * P, min((i + 1) * P, Lh))
                    owners = view.slot_pos[s, h, slots]
                    assert np.array_equal(kk[slots - i * P], kh[owners])
                    assert np.array_equal(vv[slots - i * P], vh[owners])
    cache.close()
