"""Pins for the byte / flop accountant against the printed coefficients of
Appendix I (Llama 3.1 8B)."""
import numpy as np
import pytest

from oracle import latency_model as lm

P = lm.LLAMA31_8B


def test_kv_read_coefficient():
    # printed 1.31e5 * B * L bytes
    per_BL = lm.reads(1, 1, **P) - lm.reads(1, 0, **P)
    assert per_BL == 4 * P["n"] * P["d_kv"] == 131072
    assert round(per_BL / 1e5, 2) == 1.31


def test_attention_flop_coefficient():
    # printed 5.24e5 * B * L
    per_BL = lm.flops(1, 1, **P) - lm.flops(1, 0, **P)
    assert per_BL == 524288 and round(per_BL / 1e5, 2) == 5.24


def test_constant_read_term_and_parameter_count():
    # printed 1.50e10 bytes; Reads(1, 0) / 2 is about 7.5 B parameters
    r0 = lm.reads(1, 0, **P)
    assert round(r0 / 1e10, 2) == 1.50
    assert round(r0 / 2 / 1e9, 1) == 7.5
    # the literal 4 d d_ff term would give 2.20e10 instead
    assert round(lm.reads(1, 0, literal_dff=True, **P) / 1e10, 2) == 2.20


def test_constant_flop_term_follows_equation():
    # the equation gives 1.50e10 per sequence (the printed 1.45e9 does not follow)
    assert round(lm.flops(1, 0, **P) / 1e10, 2) == 1.50


def test_latency_is_max_of_compute_and_memory():
    B, L = 64, 8192
    t = lm.latency(B, L, 989.5e12, 3.35e12, **P)
    assert t == pytest.approx(max(lm.flops(B, L, **P) / 989.5e12, lm.reads(B, L, **P) / 3.35e12))
    # memory bound at this size
    assert lm.reads(B, L, **P) / 3.35e12 > lm.flops(B, L, **P) / 989.5e12


def test_retained_kv_bytes_reduce_to_appendix_term():
    # with every head retaining L tokens the accountant equals the 4 n B L d_kv
    # term (d_kv = kv heads * head_dim), per layer and summed over layers
    n, B, Hkv, d, L = 3, 5, 8, 128, 777
    lengths = [[[L] * Hkv] * B] * n
    assert lm.kv_read_bytes(lengths, d) == 4 * n * B * L * Hkv * d


def test_decode_flops_per_byte_is_group_size():
    # q.k and p.v: 4 d flops per (query head, token); 4 d bytes per token
    for g in (2, 5, 6, 7):
        assert lm.decode_attention_flops([100], g, 128) / lm.kv_read_bytes([100], 128) == g


# ----------------------------------------------------------------------------
# Prefill flop accounting
# ----------------------------------------------------------------------------

def _llama_prefill_flops_per_token(L, fn=None):
    """Attention flops of one query at position L - 1 with every earlier key
    kept, summed over the 32 layers of the App. I model (8 KV heads x group 4,
    head_dim 128, so d = 4096 and d_kv = 1024)."""
    from oracle import visibility_mask
    fn = fn or lm.prefill_attention_flops
    counts = visibility_mask(np.zeros(L, np.uint8), 16).sum(axis=1)[L - 1]
    return P["n"] * fn([counts] * 8, 4, 128)


def test_prefill_flops_reduce_to_appendix_attention_term():
    # with all decisions 0 the visible keys of the query at position L - 1 are
    # the L causal ones, and App. I's attention term is 4 d L per layer
    # (printed 5.24e5 * B * L for Llama 3.1 8B)
    for L in (1, 37, 4096):
        assert _llama_prefill_flops_per_token(L) == lm.flops(1, L, **P) - lm.flops(1, 0, **P)
        assert _llama_prefill_flops_per_token(L) == 524288 * L


@pytest.mark.parametrize("w,p", [(1, 0.5), (4, 0.5), (16, 7 / 8), (64, 0.25)])
def test_prefill_flops_equal_decode_flops_summed_over_positions(w, p):
    # prefill query t sees exactly the keys a decode step at t reads (the
    # retained tokens, closed form min(w, t+1) + #{j <= t-w kept})
    from oracle import visibility_mask
    rng = np.random.default_rng(w)
    T, g, d = 300, 5, 128
    flags = (rng.uniform(size=T) < p).astype(np.uint8)
    counts = visibility_mask(flags, w).sum(axis=1)
    closed = [min(w, t + 1) + int(np.sum(flags[: max(0, t - w + 1)] == 0)) for t in range(T)]
    assert counts.tolist() == closed
    assert lm.prefill_attention_flops(counts, g, d) == sum(
        lm.decode_attention_flops([c], g, d) for c in closed)


@pytest.mark.parametrize("mutant", ["two_d", "no_group", "hkv_for_group"])
def test_planted_prefill_flop_mistake_is_caught(monkeypatch, mutant):
    bad = {"two_d": lambda c, g, d: sum(int(x) for x in np.ravel(c)) * g * 2 * d,
           "no_group": lambda c, g, d: sum(int(x) for x in np.ravel(c)) * 4 * d,
           "hkv_for_group": lambda c, g, d: sum(int(x) for x in np.ravel(c)) * 8 * 4 * d}[mutant]
    monkeypatch.setattr(lm, "prefill_attention_flops", bad)
    with pytest.raises(AssertionError):
        test_prefill_flops_reduce_to_appendix_attention_term()
