"""Parity of latent-attention (MLA) decode at the benchmark's full sizes, one
layer, in the launch configuration the benchmark times: 128 sequences, one
latent KV head of 576-dim rows shared by 16 query heads (DeepSeek-V2-Lite)
or 128 (DeepSeek-V2: eight head groups of 16), 32768 context tokens
appended in 4096-token chunks, w=256, flags Bernoulli(7/8), then decode
steps.

Checked: the bookkeeping of every sequence bit-exactly against the oracle's
replay, and, on sampled sequences, the stored rows at every live slot and the
decode outputs against dense masked absorbed attention over the full history
(max-abs 1e-2)."""
import math

import numpy as np
import pytest

import dms_synth as sy
from dms_testlib import ATOL, bf16_to_f32, compare_state
from oracle import PagedKVOracle, mla_attention, visible

pytestmark = pytest.mark.gpu

SEED, LAYER = 4, 11
B, ROW, LATENT, W, P, CTX, CHUNK, P_EVICT = 128, 576, 512, 256, 64, 32768, 4096, 7 / 8
STEPS = 3
SAMPLES = [0, 17, 64, 127, 90, 33]


def _rows_np(seq, positions):
    hh, dd = sy.wide_coords(np.zeros((1, 1), np.int64), np.arange(ROW)[None, :], ROW)
    return sy.token_vectors_np(SEED, sy.STREAM_K, LAYER, seq, hh, np.asarray(positions)[:, None], dd)


@pytest.mark.parametrize("G", [16, 128], ids=["deepseek-v2-lite", "deepseek-v2"])
def test_full_size_latent_layer(G):
    import torch
    from paper_2506_05345_amd import dms

    dev = "cuda"
    seqs_np = np.arange(B)
    pos_all = np.arange(CTX + STEPS)
    flags_host = sy.flags_np(SEED, P_EVICT, LAYER, seqs_np[:, None, None], np.zeros((1, 1, 1), np.int64),
                             pos_all[None, :, None])                        # [B, T, 1]
    L0 = np.minimum(W, CTX) + (flags_host[:, : CTX - W] == 0).sum(axis=1)
    maxp = int((L0.max() + STEPS + P - 1) // P) + 1
    num_pages = int(((L0 + STEPS + P - 1) // P).sum()) + 16
    cfg = dms.make_config(1, B, 1, G, ROW, W, P, num_pages, maxp, CHUNK * B, kv_format=dms.DMS_KV_MLA)
    cache = dms.DmsCache(cfg)
    orc = PagedKVOracle(B, 1, W, P, num_pages, maxp, ROW, store_values=False)
    sid = torch.arange(B, dtype=torch.int32, device=dev)
    seqs_t = torch.arange(B, device=dev)
    hk, dk = sy.wide_coords(torch.zeros((1, 1, 1), dtype=torch.int64, device=dev),
                            torch.arange(ROW, device=dev)[None, None, :], ROW)
    for c0 in range(0, CTX, CHUNK):
        pos = torch.arange(c0, c0 + CHUNK, device=dev)
        k = sy.token_vectors_torch(SEED, sy.STREAM_K, LAYER, seqs_t[:, None, None], hk, pos[None, :, None],
                                   dk, dev)                                 # [B, CHUNK, ROW]
        f = sy.flags_torch(SEED, P_EVICT, LAYER, seqs_t[:, None, None], 0, pos[None, :, None], dev)
        assert np.array_equal(f.cpu().numpy(), flags_host[:, c0:c0 + CHUNK])
        cu = torch.arange(B + 1, dtype=torch.int32, device=dev) * CHUNK
        dms.dms_append_chunk(cache.ctx, 0, B, sid, cu, B * CHUNK, CHUNK, k.reshape(B * CHUNK, 1, ROW),
                             None, f.reshape(B * CHUNK, 1))
        orc.append_chunk(list(range(B)), [flags_host[s, c0:c0 + CHUNK] for s in range(B)])
        del k
    torch.cuda.synchronize()
    assert dms.dms_status(cache.ctx) == 0
    view = cache.export(0)
    assert np.array_equal(view.L[:, 0], L0[:, 0])      # closed form
    compare_state(view, orc, range(B))                 # full bookkeeping

    hq, dq = sy.wide_coords(np.arange(G)[None, :, None], np.arange(ROW)[None, None, :], ROW)
    to = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(dev).view(torch.bfloat16)
    for step in range(STEPS):
        t = CTX + step
        q = sy.token_vectors_np(SEED, sy.STREAM_Q, LAYER, seqs_np[:, None, None], hq, t, dq)   # [B, G, ROW]
        k = np.stack([_rows_np(s, [t]) for s in range(B)])                                   # [B, 1, ROW]
        f = np.ascontiguousarray(flags_host[:, t])
        out = torch.full((B, G, LATENT), float("nan"), device=dev)
        dms.dms_decode_step(cache.ctx, 0, B, sid, to(q), to(k), None, torch.from_numpy(f).to(dev), out)
        torch.cuda.synchronize()
        assert dms.dms_status(cache.ctx) == 0
        orc.append(list(range(B)), f)
        got = out.cpu().numpy()
        assert np.isfinite(got).all()
        view = cache.export(0)
        compare_state(view, orc, range(B))
        if step == STEPS - 1:
            for s in SAMPLES:
                hist = np.arange(t + 1)
                rows = _rows_np(s, hist)
                mask = np.asarray(visible(t, hist, flags_host[s, : t + 1, 0], W), dtype=bool)
                ref = mla_attention(bf16_to_f32(q[s]), bf16_to_f32(rows), np.broadcast_to(mask, (G, t + 1)),
                                    LATENT, 1.0 / math.sqrt(ROW))
                err = np.abs(got[s] - ref).max()
                assert err <= ATOL, (s, err)
                # stored rows of every live slot of this sequence
                Lh = int(view.L[s, 0])
                pages = view.page_table[s, 0, : (Lh + P - 1) // P]
                for i, pg in enumerate(pages):
                    kk, _ = cache.pool_page_kv(0, int(pg))
                    slots = np.arange(i * P, min((i + 1) * P, Lh))
                    owners = view.slot_pos[s, 0, slots]
                    assert np.array_equal(kk[slots - i * P], rows[owners])
    cache.close()
