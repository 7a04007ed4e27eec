"""Quest-style page retrieval within the DMS retained set.  TEST
INFRASTRUCTURE ONLY.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may use
this module; the GPU library never calls it and shares no code with it.

The paper notes that DMS compresses the KV cache while Quest (query-aware
page selection) retrieves cache items, so the two are orthogonal and could be
combined (App. A).  Quest keeps, per page of keys, the channel-wise minimum
and maximum; for a query q the largest score any key of the page can reach is
bounded by  U = sum_i max(q_i * lo_i, q_i * hi_i)  (each term bounds q_i k_i
over the box lo <= k <= hi).  A decode step attends only the pages with the
largest bounds.

Readings used here (the paper gives no combined scheme):
* the retrieval unit is the cache's own page: P slots of one KV head, whose
  live slots hold retained tokens of any positions (DMS reuses the slots of
  evicted tokens);
* lo / hi are the exact channel-wise min / max over the page's live slots
  (slots below the head's retained length L) of the keys as stored;
* one selection per KV head, shared by its g query heads (the group reads
  each page once): a page's score is the maximum of U over the group;
* the top `budget` pages by score are attended, ties going to the lower
  page index; a head with at most `budget` pages attends all of them;
* selection applies to decode steps; prefill attends densely.
"""
from __future__ import annotations

import math

import numpy as np

__all__ = ["page_bounds", "quest_page_scores", "quest_select", "quest_attend_head"]


def page_bounds(keys_live):
    """Channel-wise (min, max) of the live keys of one page, [n, d] -> ([d], [d])."""
    k = np.asarray(keys_live, np.float64)
    return k.min(axis=0), k.max(axis=0)


def quest_page_scores(q_group, lo, hi):
    """Score of each page for a query group: q_group [g, d], lo / hi [npages, d]
    -> [npages] = max over the g heads of sum_i max(q_i lo_i, q_i hi_i)."""
    q = np.asarray(q_group, np.float64)[:, None, :]            # [g, 1, d]
    lo = np.asarray(lo, np.float64)[None]                       # [1, n, d]
    hi = np.asarray(hi, np.float64)[None]
    u = np.maximum(q * lo, q * hi).sum(axis=-1)                 # [g, n]
    return u.max(axis=0)


def quest_select(scores, budget):
    """Page indices attended: the `budget` largest scores (ties -> lower index),
    in ascending index order; all pages when there are at most `budget`."""
    s = np.asarray(scores, np.float64)
    n = s.shape[0]
    if n <= budget:
        return np.arange(n)
    order = sorted(range(n), key=lambda i: (-s[i], i))
    return np.sort(np.array(order[:budget], np.int64))


def quest_attend_head(q_group, keys, values, P, budget, scale=None):
    """Decode attention of one KV head's query group over the live slots
    (keys / values [L, d] in slot order) restricted to the selected pages.
    Returns (output [g, d], selected page indices)."""
    q = np.asarray(q_group, np.float64)
    k = np.asarray(keys, np.float64)
    v = np.asarray(values, np.float64)
    L, d = k.shape
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    npages = -(-L // P)
    lo = np.empty((npages, d))
    hi = np.empty((npages, d))
    for i in range(npages):
        lo[i], hi[i] = page_bounds(k[i * P:min(L, (i + 1) * P)])
    sel = quest_select(quest_page_scores(q, lo, hi), budget)
    slots = np.concatenate([np.arange(i * P, min(L, (i + 1) * P)) for i in sel])
    s = q @ k[slots].T * scale
    s -= s.max(axis=1, keepdims=True)
    p = np.exp(s)
    return (p @ v[slots]) / p.sum(axis=1, keepdims=True), sel
