"""Pins of the oracle's latent-attention (MLA) decode, CPU only.

The absorbed form the oracle writes out (a head scores a cached row
[c_j ; k_rope_j] with [W_UK^T q_nope ; q_rope] and returns the weighted sum
of the latents c_j) must equal DeepSeek-V2's attention computed the
non-absorbed way: per-head keys [W_UK c_j ; k_rope_j], values W_UV c_j, and
W_UV applied to the absorbed output.  The reference route below runs torch's
scaled_dot_product_attention in float64 on explicit per-head keys and
values, so it shares no arithmetic with the oracle.
"""
import math

import numpy as np
import pytest
import torch

from oracle import PagedKVOracle, mla_attention, visible

LATENT, ROPE, NOPE, DV = 512, 64, 128, 128


def _mla_inputs(seed, T, H):
    rng = np.random.default_rng(seed)
    c = rng.standard_normal((T, LATENT))
    k_rope = rng.standard_normal((T, ROPE))
    w_uk = rng.standard_normal((H, NOPE, LATENT)) / math.sqrt(LATENT)
    w_uv = rng.standard_normal((H, DV, LATENT)) / math.sqrt(LATENT)
    q_nope = rng.standard_normal((H, NOPE))
    q_rope = rng.standard_normal((H, ROPE))
    return c, k_rope, w_uk, w_uv, q_nope, q_rope


def _non_absorbed(c, k_rope, w_uk, w_uv, q_nope, q_rope, mask, scale):
    """Per-head keys / values materialized, attention by torch SDPA (float64)."""
    H = w_uk.shape[0]
    out = np.empty((H, DV))
    for h in range(H):
        k = np.concatenate([c @ w_uk[h].T, k_rope], axis=1)          # [T, 192]
        v = c @ w_uv[h].T                                             # [T, 128]
        q = np.concatenate([q_nope[h], q_rope[h]])[None]              # [1, 192]
        o = torch.nn.functional.scaled_dot_product_attention(
            torch.from_numpy(q)[None], torch.from_numpy(k)[None], torch.from_numpy(v)[None],
            attn_mask=torch.from_numpy(mask[None, None]), scale=scale)
        out[h] = o[0, 0].numpy()
    return out


def _absorbed(c, k_rope, w_uk, w_uv, q_nope, q_rope, mask, scale):
    rows = np.concatenate([c, k_rope], axis=1)                        # [T, 576]
    qa = np.concatenate([np.einsum("hnl,hn->hl", w_uk, q_nope), q_rope], axis=1)   # [H, 576]
    lat = mla_attention(qa, rows, np.broadcast_to(mask, (qa.shape[0], rows.shape[0])), LATENT, scale)
    return np.einsum("hvl,hl->hv", w_uv, lat)


@pytest.mark.parametrize("T,H,w,p", [(1, 4, 4, 0.0), (40, 16, 8, 0.5), (300, 16, 16, 0.9),
                                     (200, 128, 32, 0.7)])
def test_absorbed_form_equals_explicit_mla(T, H, w, p):
    c, k_rope, w_uk, w_uv, q_nope, q_rope = _mla_inputs(T * 7 + H, T, H)
    flags = (np.random.default_rng(T).random(T) < p).astype(np.uint8)
    t = T - 1
    mask = np.asarray(visible(t, np.arange(T), flags, w), dtype=bool)
    scale = 1.0 / math.sqrt(NOPE + ROPE)
    ref = _non_absorbed(c, k_rope, w_uk, w_uv, q_nope, q_rope, mask, scale)
    got = _absorbed(c, k_rope, w_uk, w_uv, q_nope, q_rope, mask, scale)
    np.testing.assert_allclose(got, ref, rtol=1e-10, atol=1e-12)


def test_absorbed_form_needs_the_rotary_part_and_the_latent_values():
    """The pin above fails for the plausible slips: scoring without the
    rotary dims, or taking values from the wrong end of the row."""
    T, H = 50, 8
    c, k_rope, w_uk, w_uv, q_nope, q_rope = _mla_inputs(3, T, H)
    mask = np.ones(T, bool)
    scale = 1.0 / math.sqrt(NOPE + ROPE)
    ref = _non_absorbed(c, k_rope, w_uk, w_uv, q_nope, q_rope, mask, scale)
    no_rope = _absorbed(c, np.zeros_like(k_rope), w_uk, w_uv, q_nope, q_rope, mask, scale)
    assert np.abs(no_rope - ref).max() > 1e-3
    # values taken from the last 512 dims of the row instead of the latent
    rows = np.concatenate([c, k_rope], axis=1)
    qa = np.concatenate([np.einsum("hnl,hn->hl", w_uk, q_nope), q_rope], axis=1)
    s_ = (qa @ rows.T) * scale
    pr = np.exp(s_ - s_.max(axis=1, keepdims=True))
    tail = (pr @ rows[:, -LATENT:]) / pr.sum(axis=1, keepdims=True)
    assert np.abs(np.einsum("hvl,hl->hv", w_uv, tail) - ref).max() > 1e-3
    # and the right slice reproduces it (the slips above are what the pin sees)
    head = (pr @ rows[:, :LATENT]) / pr.sum(axis=1, keepdims=True)
    np.testing.assert_allclose(np.einsum("hvl,hl->hv", w_uv, head), ref, rtol=1e-10, atol=1e-12)


def test_latent_replay_decode_equals_dense_masked_history():
    """The paged replay with one KV head of latent rows attends exactly the
    keys visible under DMS (brute force over the full history)."""
    T, w, P, Hq = 200, 16, 32, 4
    rng = np.random.default_rng(11)
    rows = rng.standard_normal((T, LATENT + ROPE))
    flags = (rng.random(T) < 0.7).astype(np.uint8)
    orc = PagedKVOracle(1, 1, w, P, 64, 16, LATENT + ROPE)
    for t in range(T):
        orc.append([0], flags[t][None, None], rows[t][None, None], rows[t][None, None])
    q = rng.standard_normal((1, Hq, LATENT + ROPE))
    got = orc.decode_latent([0], q, LATENT)
    mask = np.asarray(visible(T - 1, np.arange(T), flags, w), dtype=bool)
    scale = 1.0 / math.sqrt(LATENT + ROPE)
    s = (q[0] @ rows.T) * scale
    s = np.where(mask[None], s, -np.inf)
    pr = np.exp(s - s.max(axis=1, keepdims=True))
    ref = (pr @ rows[:, :LATENT]) / pr.sum(axis=1, keepdims=True)
    np.testing.assert_allclose(got[0], ref, rtol=1e-12, atol=1e-12)
    assert orc.L[0, 0] == mask.sum()
