"""Pins for the oracle's inference-time decisions (Sec. 3.2 rounding, the
borrowed query neuron of App. C) and for the immediate-eviction ablation
(Sec. 5.3): literal rounded sigmoid, perturbation of the borrowed neuron,
attention with the neuron dimension removed, and a literal event simulation
of immediate eviction with its closed-form retained count."""
import math

import numpy as np
import pytest

import oracle
from oracle import PagedKVOracle, masked_attention

BF16_5_PLUS = 5.03125    # next bf16 value above 5.0


def _bf16(x):
    """Round float32 values to bf16 (round to nearest even), returned as float32."""
    u = np.asarray(x, np.float32).view(np.uint32).astype(np.uint64)
    u = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    return u.astype(np.uint32).view(np.float32)


# ----------------------------------------------------------------------------
# alpha_bin = round(sigmoid(logit))
# ----------------------------------------------------------------------------

def test_alpha_bin_is_rounded_sigmoid():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.normal(0, 6, 5000), rng.normal(0, 1e-3, 1000),
                        [-30.0, -5.0, -1e-9, 1e-9, 5.0, 30.0]])
    x = x[np.abs(x) > 1e-12]        # float64 sigmoid of |x| < 1e-16 is exactly 1/2
    literal = np.array([int(round(1.0 / (1.0 + math.exp(-v)))) for v in x])
    assert np.array_equal(oracle.alpha_bin(x), literal)


def test_alpha_bin_tie_keeps_the_token():
    # sigmoid(0) = 1/2: the reading is "keep" (decision 0)
    assert oracle.alpha_bin(0.0) == 0
    assert oracle.alpha_bin(np.float32(np.nextafter(np.float32(0), np.float32(1)))) == 1


# ----------------------------------------------------------------------------
# the borrowed neuron: element 0 of the first query head of each group
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("g,H", [(1, 3), (2, 2), (5, 4), (16, 1)])
def test_decision_reads_only_the_borrowed_neuron(g, H):
    rng = np.random.default_rng(g * 10 + H)
    d = 8
    q = _bf16(rng.normal(0, 3, (6, H * g, d)))
    base = oracle.query_decisions(q, g, -5.0)
    assert base.shape == (6, H)
    # any other element: no change
    for (n, qh, e) in [(0, 1 % (H * g), 0), (2, 0, 3), (5, H * g - 1, d - 1)]:
        if qh % g == 0 and e == 0:
            continue
        q2 = q.copy()
        q2[n, qh, e] = 1e4 if base[n, qh // g] == 0 else -1e4
        assert np.array_equal(oracle.query_decisions(q2, g, -5.0), base)
    # the borrowed neuron of head h around the threshold -b = 5: flips only (n, h)
    for h in range(H):
        for val, want in [(5.0, 0), (BF16_5_PLUS, 1), (4.96875, 0), (-5.0, 0), (60.0, 1)]:
            q2 = q.copy()
            q2[3, h * g, 0] = val
            got = oracle.query_decisions(q2, g, -5.0)
            assert got[3, h] == want
            other = np.ones_like(base, bool)
            other[3, h] = False
            assert np.array_equal(got[other], base[other])


def test_zero_neuron_with_training_offset_keeps():
    # with b = -5 a silent neuron keeps the token (alpha ~ sigmoid(-5) ~ 0.007)
    q = np.zeros((1, 4, 8), np.float32)
    assert oracle.query_decisions(q, 2, -5.0).tolist() == [[0, 0]]
    assert oracle.query_decisions(q, 2, 0.5).tolist() == [[1, 1]]


def test_zeroed_neuron_attention_drops_that_dimension():
    """Attention of the first head of each group after zeroing equals
    attention over dims 1..d-1 (same 1/sqrt(d) scale); other heads unchanged."""
    rng = np.random.default_rng(3)
    g, H, d, T = 3, 2, 16, 25
    q = rng.normal(0, 2, (H * g, d))
    k = rng.normal(0, 1, (T, d))
    v = rng.normal(0, 1, (T, d))
    mask = np.ones((1, T), bool)
    scale = 1 / math.sqrt(d)
    qz = oracle.zero_borrowed_neuron(q, g)
    for qh in range(H * g):
        got = masked_attention(qz[qh][None], k, v, mask, scale)
        if qh % g == 0:
            s = (k[:, 1:] @ q[qh, 1:]) * scale
            p = np.exp(s - s.max())
            want = (p @ v) / p.sum()
        else:
            want = masked_attention(q[qh][None], k, v, mask, scale)[0]
        assert np.allclose(got[0], want, atol=1e-12)
    assert np.array_equal(q[:, 1:], qz[:, 1:])


# ----------------------------------------------------------------------------
# immediate eviction
# ----------------------------------------------------------------------------

def _simulate_immediate(alpha, w):
    """Literal events: at step t the decision alpha_t evicts token t - w (if
    any and still present), then token t enters.  Live set after each step."""
    live, hist = [], []
    for t in range(len(alpha)):
        if t >= w and alpha[t]:
            live = [j for j in live if j != t - w]
        live.append(t)
        hist.append(sorted(live))
    return hist


@pytest.mark.parametrize("seed", range(30))
def test_bruteforce_immediate_live_sets(seed):
    rng = np.random.default_rng(100 + seed)
    w = int(rng.integers(1, 17))
    T = int(rng.integers(1, 110))
    alpha = (rng.uniform(size=T) < rng.uniform()).astype(np.uint8)
    hist = _simulate_immediate(alpha, w)
    mask = oracle.visibility_mask(alpha, w, mode="immediate")
    orc = PagedKVOracle(1, 1, w, 4, 64, 64, 2, store_values=False, mode="immediate")
    for t in range(T):
        assert sorted(np.nonzero(mask[t])[0].tolist()) == hist[t]
        orc.append([0], alpha[t][None, None])
        assert sorted(orc.live_positions(0, 0).tolist()) == hist[t]
        closed = min(w, t + 1) + sum(1 for j in range(0, t - w + 1) if alpha[j + w] == 0)
        assert oracle.retained_count(alpha, w, t, mode="immediate") == closed == orc.L[0, 0]


def test_immediate_differs_from_delayed():
    # token 0 flagged, token w kept: delayed evicts token 0 at step w,
    # immediate keeps it (alpha_w = 0)
    w = 3
    alpha = np.array([1, 0, 0, 0, 0], np.uint8)
    d = oracle.visibility_mask(alpha, w)
    im = oracle.visibility_mask(alpha, w, mode="immediate")
    assert not d[3, 0] and im[3, 0]


def test_immediate_chunk_size_invariance():
    rng = np.random.default_rng(9)
    H, w, T = 2, 5, 90
    alpha = (rng.uniform(size=(T, H)) < 0.6).astype(np.uint8)
    states = []
    for chunks in ([T], [7] * 13, [1] * T, [40, 3, 47]):
        orc = PagedKVOracle(1, H, w, 8, 64, 32, 2, store_values=False, mode="immediate")
        c0 = 0
        for c in chunks:
            c = min(c, T - c0)
            if c <= 0:
                break
            orc.append_chunk([0], [alpha[c0:c0 + c]])
            c0 += c
        states.append((orc.L.copy(), orc.slot_pos.copy(), orc.ring_slot.copy()))
    for st in states[1:]:
        for a, b in zip(states[0], st):
            assert np.array_equal(a, b)


# ----------------------------------------------------------------------------
# planted mistakes
# ----------------------------------------------------------------------------

def _pins_pass():
    try:
        test_alpha_bin_is_rounded_sigmoid()
        test_alpha_bin_tie_keeps_the_token()
        test_decision_reads_only_the_borrowed_neuron(5, 4)
        test_zeroed_neuron_attention_drops_that_dimension()
        for seed in range(6):
            test_bruteforce_immediate_live_sets(seed)
    except AssertionError:
        return False
    return True


def test_pins_pass_unmodified():
    assert _pins_pass()


@pytest.mark.parametrize("mutant", ["tie_evicts", "last_head_of_group", "no_offset",
                                    "immediate_uses_own_decision", "zero_all_heads",
                                    "replay_uses_delayed_rule"])
def test_planted_mistake_is_caught(monkeypatch, mutant):
    mod = oracle.dms_oracle
    if mutant == "tie_evicts":
        monkeypatch.setattr(mod, "alpha_bin", lambda x: (np.asarray(x) >= 0).astype(np.uint8))
    elif mutant == "last_head_of_group":
        monkeypatch.setattr(mod, "query_decisions", lambda q, g, b: mod.alpha_bin(
            np.asarray(q)[..., g - 1::g, 0].astype(np.float32) + np.float32(b)))
    elif mutant == "no_offset":
        monkeypatch.setattr(mod, "query_decisions", lambda q, g, b: mod.alpha_bin(
            np.asarray(q)[..., ::g, 0].astype(np.float32)))
    elif mutant == "immediate_uses_own_decision":
        monkeypatch.setattr(mod, "visible_immediate",
                            lambda t, j, a, w: mod.visible(t, j, np.asarray(a)[np.asarray(j) * 0 + np.asarray(j)], w))
    elif mutant == "zero_all_heads":
        def bad(q, g):
            q = np.array(q, dtype=np.float64, copy=True)
            q[..., 0] = 0.0
            return q
        monkeypatch.setattr(mod, "zero_borrowed_neuron", bad)
    elif mutant == "replay_uses_delayed_rule":
        orig = mod.PagedKVOracle.__init__

        def bad_init(self, *a, **kw):
            orig(self, *a, **kw)
            self.mode = "delayed"
        monkeypatch.setattr(mod.PagedKVOracle, "__init__", bad_init)
    # the tests above import names through the package; route them to the module
    monkeypatch.setattr(oracle, "alpha_bin", mod.alpha_bin)
    monkeypatch.setattr(oracle, "query_decisions", mod.query_decisions)
    monkeypatch.setattr(oracle, "zero_borrowed_neuron", mod.zero_borrowed_neuron)
    monkeypatch.setattr(oracle, "visibility_mask", mod.visibility_mask)
    assert not _pins_pass()
