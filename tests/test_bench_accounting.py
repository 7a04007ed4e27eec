"""The benchmark's own arithmetic against the oracle's accountant: the
prefill flop count of the heterogeneous stress step and the App. I step model
of the sweeps.  CPU only (bench.py is imported, nothing is launched)."""
import numpy as np
import pytest
import torch

import bench
from oracle import latency_model as lm
from oracle import visibility_mask


@pytest.mark.parametrize("w", [1, 4, 16, 64])
def test_chunk_visible_counts_match_oracle_mask(w):
    # several (sequence, head) histories with cached tokens before the chunk
    # (none, fewer than w, more than w), then a chunk of C tokens
    rng = np.random.default_rng(100 + w)
    n, H, C = 3, 2, 90
    pos0 = np.array([0, max(0, w - 1), 3 * w + 11])
    T = int(pos0.max()) + C
    flags = (rng.uniform(size=(n, T, H)) < 0.6).astype(np.uint8)
    L0 = np.zeros((n, H), np.int64)
    want = np.zeros((n, C, H), np.int64)
    for s in range(n):
        for h in range(H):
            m = visibility_mask(flags[s, : pos0[s] + C, h], w)
            L0[s, h] = m[pos0[s] - 1].sum() if pos0[s] > 0 else 0
            want[s, :, h] = m[pos0[s]: pos0[s] + C].sum(axis=1)
    pos = torch.as_tensor(pos0[:, None] + np.arange(C)[None, :])
    back = torch.zeros((n, C, H), dtype=torch.uint8)
    for s in range(n):
        for c in range(C):
            t = pos0[s] + c
            if t >= w:
                back[s, c] = torch.as_tensor(flags[s, t - w])
    got = bench.chunk_visible_counts(torch.as_tensor(L0), pos, back, w)
    assert np.array_equal(got.numpy(), want)
    g, d = 5, 128
    assert bench.prefill_flops(got, g, d) == lm.prefill_attention_flops(want, g, d)


@pytest.mark.parametrize("name", sorted(bench.SWEEP_SHAPES))
def test_app_i_estimate_matches_oracle_model(name):
    sh = bench.SWEEP_SHAPES[name]
    params = dict(n=sh["layers"], d=sh["d"], d_ff=sh["d_ff"], d_kv=sh["kv_heads"] * sh["head_dim"],
                  V=sh["V"])
    peak_flops, peak_bw = bench.MFMA_PEAK_FLOPS, bench.HBM_PEAK_GBS * 1e9
    for B, L in [(1, 0), (1, 1), (32, 4096), (128, 4448.5), (2045, 4320)]:
        lat, share, weights = bench.app_i_estimate(sh, B, L)
        assert lat == pytest.approx(lm.latency(B, L, peak_flops, peak_bw, **params), rel=1e-12)
        assert weights == lm.reads(B, 0, **params)
        kv = lm.reads(B, L, **params) - lm.reads(B, 0, **params)
        assert share == pytest.approx(kv / peak_bw / lat, rel=1e-12)


def test_latent_prefill_and_decode_flops_decompose_into_the_pinned_accountant():
    # the oracle's accountant counts 4 d flops per visible (query, key) pair
    # and query head: 2 d for q . k and 2 d for p . v.  A latent row scores
    # over all 576 dims and contributes its 512 latent dims as the value.
    rng = np.random.default_rng(7)
    vis = torch.as_tensor(rng.integers(0, 5000, size=(3, 17, 1)))
    for g in (1, 16, 40, 128):
        want = lm.prefill_attention_flops(vis.numpy(), g, 576) / 2 + lm.prefill_attention_flops(vis.numpy(), g, 512) / 2
        assert bench.mla_prefill_flops(vis, g) == want
        # per retained row of one decode step: the same per-pair count
        wl = dict(head_dim=576, group=g, kv_format=bench.MLA)
        assert bench.attend_flops(wl) == lm.prefill_attention_flops(np.ones(1), g, 576) / 2 + \
            lm.prefill_attention_flops(np.ones(1), g, 512) / 2
    # standard rows: 4 d per pair
    assert bench.attend_flops(dict(head_dim=128, group=5)) == lm.prefill_attention_flops(np.ones(1), 5, 128)
