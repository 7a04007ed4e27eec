"""Byte / flop accounting for one decode step.  TEST INFRASTRUCTURE ONLY.

Appendix I of the paper models one autoregressive step of a Llama-3-style
model: FLOPS(B, L) (major matrix-vector products, 2 flops per MAC), HBM
Reads(B, L) at 2 bytes per parameter, and latency as the max of the two over
the device peaks (ideal overlap).  Only the key/value term 4 n B L d_kv grows
with batch and context.  The DMS decode path reads exactly the retained
tokens, so its algorithmic KV bytes are that term with L replaced by each
head's retained count (the paper's "KV-cache token reads" metric of Sec. 5.1
times the bytes per token).

Reading of the printed appendix: the non-KV read term is written with
4 d d_ff where the printed constant 1.50e10 only follows with 4 d d_kv (the
attention K/V projections); the printed FLOPS constant 1.45e9 B disagrees
with the equation, which gives 1.50e10 B.  ``reads`` takes the d_kv reading
by default and keeps the literal one behind ``literal_dff=True``.
"""
from __future__ import annotations

__all__ = ["LLAMA31_8B", "flops", "reads", "latency", "kv_read_bytes",
           "decode_attention_flops", "prefill_attention_flops"]

# Parameter table of Appendix I (Llama 3.1 8B).
LLAMA31_8B = dict(n=32, d=4096, d_ff=14336, d_kv=1024, V=128256)


def flops(B, L, n, d, d_ff, d_kv, V):
    """Eq. for FLOPS(B, L): per layer 6 d d_ff (MLP) + 4 d^2 (Q, O) + 4 d d_kv (K, V)
    + 4 d L (attention scores and weighted sum), per token of the batch; plus the
    2 d V logits."""
    return n * B * (6 * d * d_ff + 4 * d * d + 4 * d * d_kv + 4 * d * L) + 2 * B * d * V


def reads(B, L, n, d, d_ff, d_kv, V, literal_dff=False):
    """Eq. for Reads(B, L) in bytes at 16-bit precision."""
    kv_proj = 4 * d * (d_ff if literal_dff else d_kv)
    return n * (6 * d * d_ff + 4 * d * d + kv_proj + 4 * B * L * d_kv) + 2 * d * V


def latency(B, L, peak_flops, peak_bw, **params):
    """Per-step latency under ideal overlap: max(FLOPS / peak, Reads / bandwidth)."""
    return max(flops(B, L, **params) / peak_flops, reads(B, L, **params) / peak_bw)


def kv_read_bytes(retained_lengths, head_dim, bytes_per_elem=2):
    """Algorithmic HBM bytes of one decode attention pass: every retained token
    of every (sequence, KV head) contributes one key and one value row."""
    total = 0
    for L in _flat(retained_lengths):
        total += int(L) * 2 * head_dim * bytes_per_elem
    return total


def decode_attention_flops(retained_lengths, group, head_dim):
    """q.k and p.v for every query head of the group: 4 d flops per (query head, token)."""
    return sum(int(L) for L in _flat(retained_lengths)) * group * 4 * head_dim


def prefill_attention_flops(visible_counts, group, head_dim):
    """Same per-(query head, visible key) cost, summed over the chunk's queries.
    ``visible_counts`` lists, per (query position, KV head), the number of keys
    visible to that query."""
    return sum(int(c) for c in _flat(visible_counts)) * group * 4 * head_dim


def _flat(x):
    try:
        import numpy as np
        return np.asarray(x).reshape(-1).tolist()
    except Exception:  # pragma: no cover
        return list(x)
