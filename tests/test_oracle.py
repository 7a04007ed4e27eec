"""Pins for the CPU oracle: each test checks it against something other than
itself -- the paper's worked example, closed forms, textbook / library
routines that special cases reduce to, and brute force on tiny inputs."""
import math
import os

import numpy as np
import pytest
import torch

import oracle
from oracle import (PagedKVOracle, OutOfPages, additive_mask, dense_dms_attention,
                    dense_dms_attention_head, masked_attention, retained_count,
                    visibility_mask)

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ----------------------------------------------------------------------------
# Fig. 1b worked example
# ----------------------------------------------------------------------------

def _load_fig1b():
    rows = {}
    with open(os.path.join(GOLDEN, "fig1b_mask_w4.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            name, *cells = line.split()
            rows[name] = cells
    return rows


def _fig1b_matches(mask_fn, w, T=10):
    """Compare mask_fn(alpha, w) with the printed rows; the figure's label
    alpha_K belongs to key column K - 1."""
    rng = np.random.default_rng(0)
    alpha = rng.uniform(0.05, 0.95, size=T)
    M = mask_fn(alpha, w)
    n = T - 1
    cols = [0, 1, 2, n]
    rowpos = {"q0": 0, "q1": 1, "q2": 2, "q3": 3, "q4": 4, "q5": 5, "qn": n}
    for name, cells in _load_fig1b().items():
        t = rowpos[name]
        for j, cell in zip(cols, cells):
            if cell == "0":
                want = 0.0
            elif cell == "-inf":
                want = -np.inf
            else:
                want = math.log(1.0 - alpha[int(cell[1:]) - 1])
            if not (M[t, j] == want or (np.isfinite(want) and abs(M[t, j] - want) < 1e-12)):
                return False
    return True


def test_fig1b_worked_example_w4():
    assert _fig1b_matches(additive_mask, 4)


@pytest.mark.parametrize("w", [2, 3, 5, 6])
def test_fig1b_rejects_other_windows(w):
    # The printed pattern pins the exclusive window reading at w = 4; an
    # inclusive boundary is the exclusive rule at w + 1 and fails here too.
    assert not _fig1b_matches(additive_mask, w)


def test_binary_alpha_mask_equals_visibility_predicate():
    # At alpha in {0, 1}: log(1 - 0) = 0 keeps the key, log(1 - 1) = -inf hides it.
    rng = np.random.default_rng(1)
    for w in (1, 3, 8):
        flags = rng.integers(0, 2, size=23)
        M = additive_mask(flags.astype(float), w)
        assert np.array_equal(np.isfinite(M), visibility_mask(flags, w))
        assert np.all(M[np.isfinite(M)] == 0.0)


# ----------------------------------------------------------------------------
# Brute force: the eviction process written as events
# ----------------------------------------------------------------------------

def _simulate_eviction(flags, w):
    """Literal event simulation of delayed eviction: at step t the tokens
    flagged at step t - w leave the cache, then token t enters.  Returns the
    live position set after each step."""
    live, history = [], []
    for t in range(len(flags)):
        live = [j for j in live if not (flags[j] and t - j >= w)]
        live.append(t)
        history.append(sorted(live))
    return history


@pytest.mark.parametrize("seed", range(40))
def test_bruteforce_live_sets(seed):
    rng = np.random.default_rng(seed)
    w = int(rng.integers(1, 20))
    T = int(rng.integers(1, 120))
    p = rng.uniform(0, 1)
    flags = (rng.uniform(size=T) < p).astype(np.uint8)
    hist = _simulate_eviction(flags, w)
    mask = visibility_mask(flags, w)
    orc = PagedKVOracle(1, 1, w, 4, 64, 64, 2, store_values=False)
    for t in range(T):
        assert sorted(np.nonzero(mask[t])[0].tolist()) == hist[t]
        orc.append([0], flags[t][None, None])
        assert sorted(orc.live_positions(0, 0).tolist()) == hist[t]
        # closed form of the retained count
        closed = min(w, t + 1) + int(np.sum(flags[: max(0, t - w + 1)] == 0))
        assert retained_count(flags, w, t) == closed == orc.L[0, 0]


# ----------------------------------------------------------------------------
# Special cases that reduce to textbook attention
# ----------------------------------------------------------------------------

def _torch_sdpa(q, k, v, bool_mask):
    # q [Hq, T, d] ... library routine, float64 on the CPU
    return torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q), torch.from_numpy(k), torch.from_numpy(v),
        attn_mask=torch.from_numpy(bool_mask)).numpy()


def _rand_qkv(rng, T, Hq, Hkv, d):
    q = rng.standard_normal((T, Hq, d))
    k = rng.standard_normal((T, Hkv, d))
    v = rng.standard_normal((T, Hkv, d))
    return q, k, v


def _expand_kv(x, g):
    return np.repeat(x, g, axis=1)


@pytest.mark.parametrize("g", [1, 3])
def test_all_kept_is_causal_attention(g):
    rng = np.random.default_rng(2)
    T, Hkv, d, w = 37, 2, 16, 5
    q, k, v = _rand_qkv(rng, T, Hkv * g, Hkv, d)
    out = dense_dms_attention(q, k, v, np.zeros((T, Hkv), np.uint8), w, g)
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q).transpose(0, 1), torch.from_numpy(_expand_kv(k, g)).transpose(0, 1),
        torch.from_numpy(_expand_kv(v, g)).transpose(0, 1), is_causal=True).transpose(0, 1).numpy()
    np.testing.assert_allclose(out, ref, atol=1e-12)


@pytest.mark.parametrize("w", [1, 4, 9])
def test_all_flagged_is_sliding_window_attention(w):
    rng = np.random.default_rng(3)
    T, Hkv, g, d = 41, 2, 2, 8
    q, k, v = _rand_qkv(rng, T, Hkv * g, Hkv, d)
    out = dense_dms_attention(q, k, v, np.ones((T, Hkv), np.uint8), w, g)
    ones = torch.ones(T, T, dtype=torch.bool)
    band = (torch.tril(ones) & ~torch.tril(ones, diagonal=-w)).numpy()   # t - w < j <= t
    ref = _torch_sdpa(q.transpose(1, 0, 2), _expand_kv(k, g).transpose(1, 0, 2),
                      _expand_kv(v, g).transpose(1, 0, 2), band).transpose(1, 0, 2)
    np.testing.assert_allclose(out, ref, atol=1e-12)


def test_window_covering_history_is_causal_for_any_flags():
    rng = np.random.default_rng(4)
    T, Hkv, g, d = 30, 1, 4, 8
    q, k, v = _rand_qkv(rng, T, Hkv * g, Hkv, d)
    flags = rng.integers(0, 2, size=(T, Hkv)).astype(np.uint8)
    out = dense_dms_attention(q, k, v, flags, T, g)
    causal = dense_dms_attention(q, k, v, np.zeros_like(flags), 1, g)
    np.testing.assert_allclose(out, causal, atol=1e-12)


def test_masked_attention_matches_library_with_random_mask():
    rng = np.random.default_rng(5)
    Tq, Tk, d = 9, 31, 12
    q = rng.standard_normal((Tq, d))
    k = rng.standard_normal((Tk, d))
    v = rng.standard_normal((Tk, d))
    mask = rng.uniform(size=(Tq, Tk)) < 0.4
    mask[:, 3] = True
    out = masked_attention(q, k, v, mask, 1.0 / math.sqrt(d))
    ref = _torch_sdpa(q[None], k[None], v[None], mask[None])[0]
    np.testing.assert_allclose(out, ref, atol=1e-12)


def test_one_visible_key_returns_its_value_and_constant_v():
    rng = np.random.default_rng(6)
    d = 8
    q = rng.standard_normal((1, 2, d))
    k = rng.standard_normal((1, 1, d))
    v = rng.standard_normal((1, 1, d))
    out = dense_dms_attention(q, k, v, np.ones((1, 1), np.uint8), 1, 2)
    np.testing.assert_array_equal(out[0, 0], v[0, 0])
    T = 20
    q, k, _ = _rand_qkv(rng, T, 2, 1, d)
    out = dense_dms_attention(q * 4, k, np.ones((T, 1, d)), rng.integers(0, 2, (T, 1)), 3, 2)
    np.testing.assert_allclose(out, 1.0, atol=1e-14)


def test_needle_retained_vs_evicted():
    # One kept key and one evicted key both aligned with q: the output is the
    # kept value and carries nothing of the evicted one.
    d, T, w = 16, 12, 2
    k = np.zeros((T, 1, d))
    v = np.zeros((T, 1, d))
    q = np.zeros((1, 1, d))
    q[0, 0, 0] = 40.0
    k[2, 0, 0] = 1.0
    v[2, 0, 1] = 1.0       # kept needle
    k[5, 0, 0] = 1.0
    v[5, 0, 2] = 1.0       # flagged needle, out of the window at t = 11
    flags = np.ones((T, 1), np.uint8)
    flags[2] = 0
    out = dense_dms_attention(q, k, v, flags, w, 1, t_query=[T - 1])
    assert out[0, 0, 1] > 0.99 and out[0, 0, 2] == 0.0


# ----------------------------------------------------------------------------
# Bookkeeping: compact route vs mask route, invariances
# ----------------------------------------------------------------------------

def _run_decode_compare(seed, w, P, T, Hkv, g, d, p):
    rng = np.random.default_rng(seed)
    n = 3
    flags = (rng.uniform(size=(n, T, Hkv)) < p).astype(np.uint8)
    q = rng.standard_normal((n, T, Hkv * g, d))
    k = rng.standard_normal((n, T, Hkv, d))
    v = rng.standard_normal((n, T, Hkv, d))
    orc = PagedKVOracle(4, Hkv, w, P, 4 * Hkv * (T // P + 2), T // P + 2, d)
    seqs = [2, 0, 3]
    for t in range(T):
        orc.append(seqs, flags[:, t], k[:, t], v[:, t])
        got = orc.decode(seqs, q[:, t], g)
        for i in range(n):
            ref = dense_dms_attention(q[i, t:t + 1], k[i, :t + 1], v[i, :t + 1],
                                      flags[i, :t + 1], w, g, t_query=[t])
            np.testing.assert_allclose(got[i], ref[0], atol=1e-12)
    return orc, flags


@pytest.mark.parametrize("w,P,p", [(1, 2, 0.5), (4, 4, 0.5), (7, 8, 0.875), (16, 4, 0.25)])
def test_compact_route_equals_mask_route(w, P, p):
    _run_decode_compare(7, w, P, 40, 2, 2, 8, p)


def test_pool_contents_hold_owner_inputs():
    rng = np.random.default_rng(8)
    T, H, d, w = 50, 2, 4, 5
    flags = (rng.uniform(size=(T, H)) < 0.7).astype(np.uint8)
    k = rng.standard_normal((T, H, d))
    v = rng.standard_normal((T, H, d))
    orc = PagedKVOracle(1, H, w, 4, 64, 32, d)
    for t in range(T):
        orc.append([0], flags[t][None], k[t][None], v[t][None])
    for h in range(H):
        for slot in range(orc.L[0, h]):
            j = orc.slot_pos[0, h, slot]
            assert np.array_equal(orc.k_store[0, h, slot], k[j, h])
            assert np.array_equal(orc.v_store[0, h, slot], v[j, h])
            assert orc.slot_flag[0, h, slot] == flags[j, h]


def test_attention_invariant_to_slot_order():
    rng = np.random.default_rng(9)
    orc, _ = _run_decode_compare(10, 3, 4, 25, 1, 3, 8, 0.6)
    q = rng.standard_normal((3, 8))
    base = orc.attend(2, 0, q)
    n = orc.L[2, 0]
    perm = rng.permutation(n)
    orc.k_store[2, 0, :n] = orc.k_store[2, 0, perm]
    orc.v_store[2, 0, :n] = orc.v_store[2, 0, perm]
    np.testing.assert_allclose(orc.attend(2, 0, q), base, atol=1e-13)


def test_gqa_group_equals_repeated_single_heads():
    rng = np.random.default_rng(11)
    T, Hkv, g, d, w = 19, 2, 3, 8, 4
    q, k, v = _rand_qkv(rng, T, Hkv * g, Hkv, d)
    flags = rng.integers(0, 2, (T, Hkv)).astype(np.uint8)
    grouped = dense_dms_attention(q, k, v, flags, w, g)
    single = dense_dms_attention(q, _expand_kv(k, g), _expand_kv(v, g), np.repeat(flags, g, axis=1), w, 1)
    np.testing.assert_allclose(grouped, single, atol=1e-13)


def _state(orc):
    return (orc.pos.copy(), orc.L.copy(), orc.ring_slot.copy(), orc.ring_flag.copy(),
            orc.page_table.copy(), orc.free_stack(), orc.slot_pos.copy(), orc.slot_flag.copy())


@pytest.mark.parametrize("w", [1, 5, 16])
def test_chunk_size_invariance(w):
    rng = np.random.default_rng(12)
    T, H, P = 600, 3, 8
    seqs = [1, 0]
    flags = (rng.uniform(size=(2, T, H)) < 0.8).astype(np.uint8)
    states = []
    for C in (1, 7, w, 512):
        orc = PagedKVOracle(2, H, w, P, 2 * H * (T // P + 1), T // P + 1, 2, store_values=False)
        for c0 in range(0, T, C):
            orc.append_chunk(seqs, [flags[0, c0:c0 + C], flags[1, c0:c0 + C]])
        states.append(_state(orc))
    # Per-head slot state is invariant; page ids depend on how pops interleave
    # across calls (pop order is per call), so only the set of pages in use
    # and the stack height are invariant.
    for s in states[1:]:
        for idx in (0, 1, 2, 3, 6, 7):
            assert np.array_equal(states[0][idx], s[idx])
        assert len(s[5]) == len(states[0][5])
        assert sorted(s[4][s[4] >= 0].tolist()) == sorted(states[0][4][states[0][4] >= 0].tolist())


def test_ragged_chunk_call_equals_separate_calls():
    rng = np.random.default_rng(13)
    H, w, P = 2, 3, 4
    f0 = (rng.uniform(size=(9, H)) < 0.5).astype(np.uint8)
    f1 = (rng.uniform(size=(4, H)) < 0.5).astype(np.uint8)
    a = PagedKVOracle(2, H, w, P, 64, 16, 2, store_values=False)
    a.append_chunk([1, 0], [f0, f1])
    b = PagedKVOracle(2, H, w, P, 64, 16, 2, store_values=False)
    b.append_chunk([1], [f0])
    b.append_chunk([0], [f1])
    for x, y in zip(_state(a), _state(b)):
        assert np.array_equal(x, y)


def test_pop_order_hand_derived():
    # P = 2, w = 2, two heads, no flags: every head takes fresh slots 0, 1, 2, ...
    # and needs a page at slots 0 and 2.  One call appends 3 tokens to seq 1
    # then 1 token to seq 0 (call order [1, 0]): pops go
    #   seq 1 head 0: pages 0 (slot 0), 1 (slot 2)
    #   seq 1 head 1: pages 2, 3
    #   seq 0 head 0: page 4;   seq 0 head 1: page 5
    orc = PagedKVOracle(2, 2, 2, 2, 8, 4, 1, store_values=False)
    orc.append_chunk([1, 0], [np.zeros((3, 2), np.uint8), np.zeros((1, 2), np.uint8)])
    assert orc.page_table[1, 0, :2].tolist() == [0, 1]
    assert orc.page_table[1, 1, :2].tolist() == [2, 3]
    assert orc.page_table[0, 0, 0] == 4 and orc.page_table[0, 1, 0] == 5
    assert orc.top == 2 and orc.free_stack().tolist() == [7, 6]
    # reset of seq 1 pushes head 0's pages then head 1's, page-table order
    orc.seq_reset([1])
    assert orc.free_stack().tolist() == [7, 6, 0, 1, 2, 3]
    orc.append([1], np.zeros((1, 2), np.uint8))
    assert orc.page_table[1, 0, 0] == 3 and orc.page_table[1, 1, 0] == 2


def test_recycled_slot_hand_derived():
    # w = 2: tokens 0 (flagged) and 1; token 2 takes token 0's slot 0; token 3
    # (token 1 unflagged) takes fresh slot 2.
    orc = PagedKVOracle(1, 1, 2, 4, 4, 4, 1, store_values=False)
    for f in (1, 0, 0, 0):
        orc.append([0], np.array([[f]], np.uint8))
    assert orc.L[0, 0] == 3
    assert orc.slot_pos[0, 0, :3].tolist() == [2, 1, 3]


def test_out_of_pages_is_all_or_nothing():
    orc = PagedKVOracle(2, 1, 2, 2, 3, 4, 1, store_values=False)
    orc.append_chunk([0], [np.zeros((4, 1), np.uint8)])    # 2 pages
    before = _state(orc)
    with pytest.raises(OutOfPages):
        orc.append_chunk([1, 0], [np.zeros((2, 1), np.uint8), np.zeros((1, 1), np.uint8)])
    for a, b in zip(before, _state(orc)):
        assert np.array_equal(a, b)


# ----------------------------------------------------------------------------
# Planted mistakes: each plausible slip in the oracle fails at least one pin
# ----------------------------------------------------------------------------

def _pins_pass():
    """A compact set of the pins above; False as soon as one fails."""
    try:
        assert _fig1b_matches(oracle.dms_oracle.additive_mask, 4)
        rng = np.random.default_rng(21)
        flags = (rng.uniform(size=30) < 0.5).astype(np.uint8)
        hist = _simulate_eviction(flags, 3)
        m = oracle.dms_oracle.visibility_mask(flags, 3)
        for t in range(30):
            assert sorted(np.nonzero(m[t])[0].tolist()) == hist[t]
        test_all_kept_is_causal_attention(3)
        test_all_flagged_is_sliding_window_attention(4)
        test_masked_attention_matches_library_with_random_mask()
        _run_decode_compare(3, 3, 2, 12, 1, 2, 4, 0.5)
        test_pop_order_hand_derived()
        test_recycled_slot_hand_derived()
    except AssertionError:
        return False
    return True


def test_pins_pass_unmodified():
    assert _pins_pass()


@pytest.mark.parametrize("mutant", ["inclusive_window", "flags_ignored", "flag_inverted",
                                    "transposed_scores", "no_scale", "r1_reuse_any",
                                    "pop_bottom"])
def test_planted_mistake_is_caught(monkeypatch, mutant):
    mod = oracle.dms_oracle
    if mutant == "inclusive_window":
        monkeypatch.setattr(mod, "visible", lambda t, j, f, w: (j <= t) & ((j >= t - w) | (f == 0)))
        monkeypatch.setattr(mod, "additive_mask", lambda a, w: _orig_additive(a, w + 1))
    elif mutant == "flags_ignored":
        monkeypatch.setattr(mod, "visible", lambda t, j, f, w: (j <= t) | (f > 1))
    elif mutant == "flag_inverted":
        monkeypatch.setattr(mod, "visible", lambda t, j, f, w: (j <= t) & ((j > t - w) | (f == 1)))
    elif mutant == "transposed_scores":
        def bad(q, k, v, mask, scale):
            q = np.asarray(q, np.float64); k = np.asarray(k, np.float64)
            s = (q @ k.T) * scale
            s = np.where(mask, s, -np.inf)
            e = np.where(mask, np.exp(s - s.max(axis=0, keepdims=True)), 0.0)
            return (e @ np.asarray(v, np.float64)) / e.sum(axis=1, keepdims=True)
        monkeypatch.setattr(mod, "masked_attention", bad)
    elif mutant == "no_scale":
        monkeypatch.setattr(mod, "masked_attention", lambda q, k, v, m, s: _orig_masked(q, k, v, m, 1.0))
    elif mutant == "r1_reuse_any":
        # reuse token t-w's slot regardless of its flag
        orig = mod.PagedKVOracle.append_chunk

        def bad_append(self, seq_ids, flags_list, k_list=None, v_list=None):
            self.ring_flag[:] = 1
            return orig(self, seq_ids, flags_list, k_list, v_list)
        monkeypatch.setattr(mod.PagedKVOracle, "append_chunk", bad_append)
    elif mutant == "pop_bottom":
        orig_init = mod.PagedKVOracle.__init__

        def bad_init(self, *a, **kw):
            orig_init(self, *a, **kw)
            self.stack = self.stack[::-1].copy()
        monkeypatch.setattr(mod.PagedKVOracle, "__init__", bad_init)
    assert not _pins_pass()


_orig_additive = oracle.dms_oracle.additive_mask
_orig_masked = oracle.dms_oracle.masked_attention
