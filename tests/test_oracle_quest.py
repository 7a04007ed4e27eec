"""Pins for the Quest-within-DMS oracle: the page bound equals the maximum of
q.k over the box of the page's keys (brute force over all corners), bounds
every live key's score, selection equals a brute-force sort with ties to the
lower index, a budget that covers every page is dense attention, and planted
mistakes fail."""
import itertools

import numpy as np
import pytest

import oracle
from oracle import quest


def _corner_max(q, lo, hi):
    """max over all 2^d corners of the box lo <= k <= hi of q.k (a linear
    function attains its maximum over a box at a corner)."""
    best = -np.inf
    for bits in itertools.product((0, 1), repeat=len(lo)):
        k = np.where(np.array(bits) == 1, hi, lo)
        best = max(best, float(q @ k))
    return best


def test_bound_is_the_box_maximum():
    rng = np.random.default_rng(1)
    for _ in range(40):
        d, g = 7, 3
        keys = rng.normal(size=(rng.integers(1, 9), d))
        lo, hi = quest.page_bounds(keys)
        q = rng.normal(size=(g, d))
        u = quest.quest_page_scores(q, lo[None], hi[None])[0]
        assert np.isclose(u, max(_corner_max(qh, lo, hi) for qh in q), rtol=0, atol=1e-12)


def test_bound_covers_every_live_key():
    rng = np.random.default_rng(2)
    d, g, n = 32, 5, 20
    pages = [rng.normal(size=(rng.integers(1, 17), d)) * rng.uniform(0.1, 3) for _ in range(n)]
    lo = np.stack([quest.page_bounds(p)[0] for p in pages])
    hi = np.stack([quest.page_bounds(p)[1] for p in pages])
    q = rng.normal(size=(g, d))
    u = quest.quest_page_scores(q, lo, hi)
    for i, p in enumerate(pages):
        assert (q @ p.T).max() <= u[i] + 1e-12
    # a single-key page: the bound is that key's best score exactly
    k = rng.normal(size=(1, d))
    lo1, hi1 = quest.page_bounds(k)
    assert np.isclose(quest.quest_page_scores(q, lo1[None], hi1[None])[0], (q @ k[0]).max(), atol=1e-12)


def test_selection_is_top_k_with_ties_to_the_lower_index():
    s = np.array([1.0, 5.0, 3.0, 5.0, 2.0, 3.0, 0.5])
    assert list(quest.quest_select(s, 1)) == [1]
    assert list(quest.quest_select(s, 2)) == [1, 3]
    assert list(quest.quest_select(s, 3)) == [1, 2, 3]        # 3.0 at 2 beats 3.0 at 5
    assert list(quest.quest_select(s, 4)) == [1, 2, 3, 5]
    assert list(quest.quest_select(s, 7)) == list(range(7))
    assert list(quest.quest_select(s, 100)) == list(range(7))
    rng = np.random.default_rng(3)
    for _ in range(50):
        n = int(rng.integers(1, 40))
        sc = rng.integers(0, 6, n).astype(float)           # many ties
        b = int(rng.integers(1, 45))
        got = list(quest.quest_select(sc, b))
        # brute force: every selected score >= every unselected one, ties by index
        ref = sorted(sorted(range(n), key=lambda i: (-sc[i], i))[:min(b, n)])
        assert got == ref


def test_full_budget_is_dense_attention():
    rng = np.random.default_rng(4)
    L, d, g, P = 150, 16, 3, 32
    k, v = rng.normal(size=(L, d)), rng.normal(size=(L, d))
    q = rng.normal(size=(g, d))
    out, sel = quest.quest_attend_head(q, k, v, P, budget=5)
    assert list(sel) == [0, 1, 2, 3, 4]
    ref = oracle.masked_attention(q, k, v, np.ones((g, L), bool), 1 / np.sqrt(d))
    assert np.allclose(out, ref, atol=1e-12)


def test_restricted_attention_reads_only_selected_pages():
    rng = np.random.default_rng(5)
    L, d, g, P, B = 200, 16, 2, 32, 2
    k, v = rng.normal(size=(L, d)), rng.normal(size=(L, d))
    # page 4 holds a key aligned with the query: it must be selected
    q = rng.normal(size=(g, d))
    k[4 * P + 3] = 6 * q[0] / np.linalg.norm(q[0])
    out, sel = quest.quest_attend_head(q, k, v, P, B)
    assert 4 in sel and len(sel) == B
    slots = np.concatenate([np.arange(i * P, min(L, (i + 1) * P)) for i in sel])
    ref = oracle.masked_attention(q, k[slots], v[slots], np.ones((g, len(slots)), bool), 1 / np.sqrt(d))
    assert np.allclose(out, ref, atol=1e-12)


# ----------------------------------------------------------------------------
# planted mistakes
# ----------------------------------------------------------------------------

def _pins_pass():
    try:
        test_bound_is_the_box_maximum()
        test_bound_covers_every_live_key()
        test_selection_is_top_k_with_ties_to_the_lower_index()
        test_full_budget_is_dense_attention()
    except AssertionError:
        return False
    return True


def test_pins_pass_unmodified():
    assert _pins_pass()


@pytest.mark.parametrize("mutant", ["min_of_products", "sum_over_heads", "abs_bound", "ties_high",
                                    "first_key_bounds"])
def test_planted_mistake_is_caught(monkeypatch, mutant):
    orig_scores, orig_select, orig_bounds = quest.quest_page_scores, quest.quest_select, quest.page_bounds
    if mutant == "min_of_products":
        def f(q, lo, hi):
            q = np.asarray(q, np.float64)[:, None, :]
            return np.minimum(q * np.asarray(lo)[None], q * np.asarray(hi)[None]).sum(-1).max(0)
        monkeypatch.setattr(quest, "quest_page_scores", f)
    elif mutant == "sum_over_heads":
        def f(q, lo, hi):
            q = np.asarray(q, np.float64)[:, None, :]
            return np.maximum(q * np.asarray(lo)[None], q * np.asarray(hi)[None]).sum(-1).sum(0)
        monkeypatch.setattr(quest, "quest_page_scores", f)
    elif mutant == "abs_bound":
        def f(q, lo, hi):
            q = np.abs(np.asarray(q, np.float64))[:, None, :]
            m = np.maximum(np.abs(np.asarray(lo)), np.abs(np.asarray(hi)))[None]
            return (q * m).sum(-1).max(0)
        monkeypatch.setattr(quest, "quest_page_scores", f)
    elif mutant == "ties_high":
        def f(scores, budget):
            s = np.asarray(scores, np.float64)
            n = len(s)
            if n <= budget:
                return np.arange(n)
            order = sorted(range(n), key=lambda i: (-s[i], -i))
            return np.sort(np.array(order[:budget]))
        monkeypatch.setattr(quest, "quest_select", f)
    elif mutant == "first_key_bounds":
        monkeypatch.setattr(quest, "page_bounds", lambda k: orig_bounds(np.asarray(k)[:1]))
    assert not _pins_pass()
