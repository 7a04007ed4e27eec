"""Plain, slow CPU oracle for DMS inference.  TEST INFRASTRUCTURE ONLY.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may use
this module.  It shares no code with the GPU library and never imports it.

What it computes (paper: "Inference-Time Hyper-Scaling with KV Cache
Compression", arxiv 2506.05345):

* Visibility of key j to query t under DMS with binary decisions.  Sec. 3.1
  ("Eviction Decisions", "Delayed Eviction via Sliding Window") builds the
  additive mask M_alpha of Fig. 1b: -inf above the diagonal, 0 for the w most
  recent positions, log(1 - alpha_j) elsewhere.  Sec. 3.2 rounds alpha to
  {0, 1} at inference, where log(1 - 1) = -inf hides the key and log(1) = 0
  keeps it.  So key j is visible to query t iff j <= t and (j > t - w or
  alpha_j = 0).
* Dense masked softmax attention in float64 over the full history with that
  mask, grouped-query heads sharing one KV head (Sec. 4 notes all evaluated
  models use GQA; the eviction decision is per KV head, Sec. 3.1).
* The KV-cache bookkeeping of Sec. 3.2 ("Performance Considerations" of the
  inference paragraph): a flagged token is removed w steps after it was
  flagged and an incoming token overwrites its slot; pages belong to one
  attention head.  The oracle replays this token by token (rule R1 below) on
  a paged per-head layout and exposes every piece of state for bit-exact
  comparison.

Readings of points the paper leaves open (each is also listed in the design
notes):

* Window boundary: "available until t + w" is exclusive -- key j is visible
  to queries j .. j + w - 1.  This reproduces Fig. 1b with w = 4, whose
  column k_j carries the 1-based label alpha_{j+1}.
* Rule R1 (which slot an incoming token takes): token t reuses the slot of
  token t - w when t >= w and token t - w was flagged; otherwise it takes the
  next fresh slot L of its head (L += 1), and a fresh slot that starts a page
  (slot % page_size == 0) pops a page from the free stack.
* Free stack: initially stack[i] = num_pages - 1 - i with top = num_pages, so
  pops return pages 0, 1, 2, ... .  Within one call pops happen in the order
  (sequence in call order, KV head ascending, position ascending).  A reset
  pushes each head's pages in page-table order, heads ascending.
* Softmax scale 1/sqrt(head_dim); query head q reads KV head q // group.
* A call that would pop more pages than the stack holds fails as a whole
  (OutOfPages) and changes nothing.

Latent attention (MLA; the paper names it as a direction for DMS, Sec. 6,
without a scheme).  Reading: an MLA layer caches one row per token shared by
all query heads -- the compressed latent c_t followed by the decoupled rotary
key -- so DMS treats it as a single KV head whose group is every query head
and evicts rows by the same rule.  Decode is the absorbed form of
DeepSeek-V2's attention: the query arrives already mapped into the latent
space (W_UK^T q_nope) and followed by its rotary part; a head scores row j
by q . row_j over the full row and outputs the softmax-weighted sum of the
rows' latent parts (W_UV is applied afterwards by the model).  ``mla_attention``
writes that out; the tests pin it to the non-absorbed form with explicit
per-head keys [W_UK c_j ; k_rope_j] and values W_UV c_j.

Decisions at inference and the eviction-timing ablation:

* Sec. 3.2 rounds the decision to alpha_bin = round(sigmoid(logit)).  The
  logit of a token for one KV head is the first neuron of the first query
  head of its group plus the offset b (App. C borrows that neuron; Sec. 3.1
  adds b, -5 in training).  After the decision is read, App. C sets that
  neuron to 0 for attention.  Readings: the logit is formed in float32 from
  the bf16 query value; sigmoid(0) = 1/2 rounds to 0 (the token is kept).
* Immediate eviction (Sec. 5.3 ablation): the decision made at step t + w
  evicts token t at that step, so key j is hidden from query t iff
  j + w <= t and alpha_{j+w} = 1.  In the replay, token t takes token
  t - w's slot iff t >= w and token t's own decision is 1.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

from .kv_fp8 import dequantize_rows_fp8, quantize_rows_fp8

__all__ = [
    "visible", "visible_immediate", "visibility_mask", "additive_mask", "retained_count",
    "alpha_bin", "query_decisions", "zero_borrowed_neuron",
    "masked_attention", "dense_dms_attention", "dense_dms_attention_head",
    "mla_attention", "OutOfPages", "PagedKVOracle",
]


# ----------------------------------------------------------------------------
# Visibility (Sec. 3.1 mask M_alpha and delayed eviction; Sec. 3.2 binarisation)
# ----------------------------------------------------------------------------

def visible(t, j, flag_j, w):
    """Key j visible to query t: causal, and either inside the window or kept.

    Works elementwise on NumPy arrays (broadcasting) as well as on scalars.
    """
    return (j <= t) & ((j > t - w) | (flag_j == 0))


def visible_immediate(t, j, alpha, w):
    """Key j visible to query t under immediate eviction (Sec. 5.3): the
    decision alpha_{j+w}, made at step j + w, evicts token j at that step.

    alpha holds the decisions of positions 0 .. T-1 (T > t); elementwise over
    arrays of t and j.
    """
    alpha = np.asarray(alpha)
    j = np.asarray(j)
    at = j + w
    decided = at <= t
    evicted = decided & (alpha[np.clip(at, 0, alpha.shape[0] - 1)] == 1)
    return (j <= t) & ~evicted


def visibility_mask(flags: np.ndarray, w: int, mode: str = "delayed") -> np.ndarray:
    """Boolean [T, T] mask, row = query position, column = key position."""
    flags = np.asarray(flags)
    T = flags.shape[0]
    t = np.arange(T)[:, None]
    j = np.arange(T)[None, :]
    if mode == "immediate":
        return np.asarray(visible_immediate(t, j, flags, w), dtype=bool)
    return np.asarray(visible(t, j, flags[None, :], w), dtype=bool)


def additive_mask(alpha: np.ndarray, w: int) -> np.ndarray:
    """M_alpha of Fig. 1b for continuous decisions alpha_j in [0, 1].

    Entry (t, j): -inf if j > t; 0 if j lies among the w most recent positions
    (t - w < j <= t); log(1 - alpha_j) otherwise.
    """
    alpha = np.asarray(alpha, dtype=np.float64)
    T = alpha.shape[0]
    m = np.full((T, T), -np.inf)
    with np.errstate(divide="ignore"):
        for t in range(T):
            for j in range(t + 1):
                m[t, j] = 0.0 if j > t - w else math.log(1.0 - alpha[j]) if alpha[j] < 1.0 else -np.inf
    return m


def retained_count(flags: np.ndarray, w: int, t: int, mode: str = "delayed") -> int:
    """Number of keys visible to query t, counted straight from the predicate."""
    if mode == "immediate":
        return sum(1 for j in range(t + 1) if visible_immediate(t, j, flags, w))
    return sum(1 for j in range(t + 1) if visible(t, j, int(flags[j]), w))


# ----------------------------------------------------------------------------
# Decisions from the borrowed query neuron (Sec. 3.2 rounding, App. C)
# ----------------------------------------------------------------------------

def alpha_bin(logit):
    """round(sigmoid(logit)) in {0, 1}.  sigmoid is increasing and equals 1/2
    at 0, so the rounded value is 1 exactly when logit > 0; the tie (logit 0)
    keeps the token."""
    return (np.asarray(logit) > 0).astype(np.uint8)


def query_decisions(q, group, bias):
    """Decisions of tokens for every KV head from their queries.

    q [..., Hq, d] (bf16 values as floats): KV head h reads element 0 of query
    head h * group (the first head of its group) and adds the offset b; the
    sum is formed in float32.  Returns uint8 [..., Hq // group].
    """
    first = np.asarray(q)[..., ::group, 0].astype(np.float32)
    return alpha_bin(first + np.float32(bias))


def zero_borrowed_neuron(q, group):
    """Copy of q [..., Hq, d] with element 0 of the first query head of every
    group set to 0 (App. C: the neuron no longer takes part in attention)."""
    q = np.array(q, dtype=np.float64, copy=True)
    q[..., ::group, 0] = 0.0
    return q


# ----------------------------------------------------------------------------
# Dense attention
# ----------------------------------------------------------------------------

def masked_attention(q, k, v, mask, scale) -> np.ndarray:
    """softmax(scale * q k^T restricted to mask) v, in float64.

    q [Tq, d], k [Tk, d], v [Tk, d], mask bool [Tq, Tk] (every row needs at
    least one True).
    """
    q = np.asarray(q, np.float64)
    k = np.asarray(k, np.float64)
    v = np.asarray(v, np.float64)
    s = (q @ k.T) * scale
    s = np.where(mask, s, -np.inf)
    m = s.max(axis=1, keepdims=True)
    p = np.where(mask, np.exp(s - m), 0.0)
    return (p @ v) / p.sum(axis=1, keepdims=True)


def mla_attention(q, rows, mask, latent, scale) -> np.ndarray:
    """Absorbed-form latent attention, float64: softmax(scale * q rows^T
    restricted to mask) rows[:, :latent].

    q [Tq, d] (latent-space query then rotary query), rows [Tk, d] (latent
    then rotary key), mask bool [Tq, Tk].  Returns [Tq, latent].
    """
    rows = np.asarray(rows, np.float64)
    return masked_attention(q, rows, rows[:, :latent], mask, scale)


def dense_dms_attention_head(q_rows, k_hist, v_hist, flags_hist, w, t_query, scale=None,
                             mode="delayed"):
    """One KV head, its query group, several query positions, full history.

    q_rows [Nq, g, d]: the g query heads of the group at each query position.
    k_hist, v_hist [T, d]: keys / values of positions 0 .. T-1 of this head.
    flags_hist [T]: binary decision of each position.
    t_query [Nq]: position of each query (< T).
    mode: "delayed" (Sec. 3.1) or "immediate" (Sec. 5.3 ablation).
    Returns [Nq, g, d] float64.
    """
    q_rows = np.asarray(q_rows, np.float64)
    Nq, g, d = q_rows.shape
    T = np.asarray(k_hist).shape[0]
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    flags_hist = np.asarray(flags_hist)
    out = np.empty((Nq, g, d))
    j = np.arange(T)
    for i, t in enumerate(np.asarray(t_query)):
        if mode == "immediate":
            row = np.asarray(visible_immediate(t, j, flags_hist, w), dtype=bool)
        else:
            row = np.asarray(visible(t, j, flags_hist, w), dtype=bool)
        out[i] = masked_attention(q_rows[i], k_hist, v_hist,
                                  np.broadcast_to(row, (g, T)), scale)
    return out


def dense_dms_attention(q, k, v, flags, w, group, t_query=None, scale=None, mode="delayed"):
    """One sequence, all heads.  q [Nq, Hq, d] at positions t_query (default
    0..Nq-1), k / v [T, Hkv, d], flags [T, Hkv].  Returns [Nq, Hq, d]."""
    q = np.asarray(q, np.float64)
    Nq, Hq, d = q.shape
    Hkv = Hq // group
    if t_query is None:
        t_query = np.arange(Nq)
    out = np.empty((Nq, Hq, d))
    for h in range(Hkv):
        out[:, h * group:(h + 1) * group] = dense_dms_attention_head(
            q[:, h * group:(h + 1) * group], np.asarray(k)[:, h], np.asarray(v)[:, h],
            np.asarray(flags)[:, h], w, t_query, scale, mode)
    return out


# ----------------------------------------------------------------------------
# Paged per-head KV bookkeeping (Sec. 3.2), token-sequential replay
# ----------------------------------------------------------------------------

class OutOfPages(RuntimeError):
    pass


@dataclass
class _Dims:
    max_seqs: int
    num_kv_heads: int
    window: int
    page_size: int
    num_pages: int
    max_pages_per_head: int
    head_dim: int


class PagedKVOracle:
    """Token-by-token replay of DMS cache management for one layer.

    State (all NumPy, exported as-is for comparison):
      pos[s]                    tokens appended to sequence s
      L[s, h]                   retained (= live) slots of head h
      ring_slot[s, h, w]        slot of the token at position p, index p % w
      ring_flag[s, h, w]        its decision
      page_table[s, h, i]       page holding slots i*P .. i*P+P-1
      stack[num_pages], top     free-page stack
      slot_pos[s, h, slot]      position of the token held by a live slot
      slot_flag[s, h, slot]     its decision
    With ``store_values`` the K / V rows of every live slot are kept too.
    mode "delayed": token t reuses token t - w's slot iff that token's own
    decision was 1; mode "immediate": iff token t's decision is 1.
    kv_format "fp8": every stored row is quantized on append (E4M3 codes and
    a power-of-two row exponent, see ``kv_fp8``); k_codes / k_exp and
    v_codes / v_exp hold them and k_store / v_store the dequantized rows that
    attention reads.
    """

    def __init__(self, max_seqs, num_kv_heads, window, page_size, num_pages,
                 max_pages_per_head, head_dim, store_values=True, mode="delayed",
                 kv_format="bf16"):
        if window < 1:
            raise ValueError("window must be >= 1")
        if mode not in ("delayed", "immediate"):
            raise ValueError("mode must be 'delayed' or 'immediate'")
        if kv_format not in ("bf16", "fp8"):
            raise ValueError("kv_format must be 'bf16' or 'fp8'")
        self.mode = mode
        self.kv_format = kv_format
        self.dims = _Dims(max_seqs, num_kv_heads, window, page_size, num_pages,
                          max_pages_per_head, head_dim)
        S, H, w = max_seqs, num_kv_heads, window
        max_slots = max_pages_per_head * page_size
        self.pos = np.zeros(S, np.int64)
        self.L = np.zeros((S, H), np.int64)
        self.ring_slot = np.full((S, H, w), -1, np.int64)
        self.ring_flag = np.zeros((S, H, w), np.uint8)
        self.page_table = np.full((S, H, max_pages_per_head), -1, np.int64)
        self.stack = np.arange(num_pages - 1, -1, -1, dtype=np.int64)
        self.top = num_pages
        self.slot_pos = np.full((S, H, max_slots), -1, np.int64)
        self.slot_flag = np.zeros((S, H, max_slots), np.uint8)
        self.store_values = store_values
        if store_values:
            self.k_store = np.zeros((S, H, max_slots, head_dim), np.float64)
            self.v_store = np.zeros((S, H, max_slots, head_dim), np.float64)
            if kv_format == "fp8":
                self.k_codes = np.zeros((S, H, max_slots, head_dim), np.uint8)
                self.v_codes = np.zeros((S, H, max_slots, head_dim), np.uint8)
                self.k_exp = np.zeros((S, H, max_slots), np.int64)
                self.v_exp = np.zeros((S, H, max_slots), np.int64)

    # -- the append rule ------------------------------------------------------
    def append_chunk(self, seq_ids, flags_list, k_list=None, v_list=None):
        """Append C_i tokens to each listed sequence (all heads).

        flags_list[i]: [C_i, H] decisions; k_list[i], v_list[i]: [C_i, H, d].
        Tokens are processed in position order for every head; the result is
        the same as appending them one at a time.
        """
        D = self.dims
        P, w, H = D.page_size, D.window, D.num_kv_heads
        seq_ids = [int(s) for s in seq_ids]
        if len(set(seq_ids)) != len(seq_ids):
            raise ValueError("duplicate sequence ids")
        pos = self.pos.copy()
        L = self.L.copy()
        ring_slot = self.ring_slot.copy()
        ring_flag = self.ring_flag.copy()
        slot_pos = self.slot_pos.copy()
        slot_flag = self.slot_flag.copy()
        writes = []          # (seq rows, slots, active call indices, c) for stored values
        page_events = []     # (i, h, page_index) needing a fresh page
        flags_all = [np.asarray(f).reshape(-1, H) for f in flags_list]
        lens = np.array([f.shape[0] for f in flags_all], np.int64)
        sid = np.array(seq_ids, np.int64)
        hs = np.arange(H)
        # Every sequence (and head) is independent; step all of them through
        # their own positions side by side, one chunk offset c at a time.
        for c in range(int(lens.max(initial=0))):
            act = np.nonzero(lens > c)[0]
            s = sid[act]
            t = pos[s]                                   # [na]
            e = t % w
            f = np.stack([flags_all[i][c] for i in act])   # [na, H]
            prev_slot = ring_slot[s[:, None], hs[None, :], e[:, None]]
            prev_flag = ring_flag[s[:, None], hs[None, :], e[:, None]]
            if self.mode == "immediate":
                reuse = (t >= w)[:, None] & (f == 1)        # token t evicts token t-w now
            else:
                reuse = (t >= w)[:, None] & (prev_flag == 1)   # token t-w was flagged
            slot = np.where(reuse, prev_slot, L[s])
            fresh = ~reuse
            if np.any(slot >= D.max_pages_per_head * P):
                raise OutOfPages("head exceeds max_pages_per_head")
            for a, h in zip(*np.nonzero(fresh & (slot % P == 0))):
                page_events.append((int(act[a]), int(h), int(slot[a, h] // P)))
            L[s] += fresh
            ring_slot[s[:, None], hs[None, :], e[:, None]] = slot
            ring_flag[s[:, None], hs[None, :], e[:, None]] = f
            slot_pos[s[:, None], hs[None, :], slot] = t[:, None]
            slot_flag[s[:, None], hs[None, :], slot] = f
            if self.store_values and k_list is not None:
                writes.append((s, slot.copy(), act, c))
            pos[s] = t + 1
        # pops: sequence in call order, head ascending, position (= page) ascending
        page_events.sort()
        if len(page_events) > self.top:
            raise OutOfPages(f"need {len(page_events)} pages, {self.top} free")
        page_table = self.page_table.copy()
        top = self.top
        for (i, h, pidx) in page_events:
            top -= 1
            page_table[seq_ids[i], h, pidx] = self.stack[top]
        # commit
        self.pos, self.L = pos, L
        self.ring_slot, self.ring_flag = ring_slot, ring_flag
        self.slot_pos, self.slot_flag = slot_pos, slot_flag
        self.page_table, self.top = page_table, top
        for (s, slot, act, c) in writes:
            for r, i in enumerate(act):
                kr = np.asarray(k_list[i], np.float64).reshape(-1, H, D.head_dim)[c]
                vr = np.asarray(v_list[i], np.float64).reshape(-1, H, D.head_dim)[c]
                if self.kv_format == "fp8":
                    kc, ke = quantize_rows_fp8(kr)
                    vc, ve = quantize_rows_fp8(vr)
                    self.k_codes[s[r], hs, slot[r]] = kc
                    self.v_codes[s[r], hs, slot[r]] = vc
                    self.k_exp[s[r], hs, slot[r]] = ke
                    self.v_exp[s[r], hs, slot[r]] = ve
                    kr = dequantize_rows_fp8(kc, ke)
                    vr = dequantize_rows_fp8(vc, ve)
                self.k_store[s[r], hs, slot[r]] = kr
                self.v_store[s[r], hs, slot[r]] = vr

    def append(self, seq_ids, flags, k=None, v=None):
        """One token per listed sequence: flags [n, H], k / v [n, H, d]."""
        n = len(seq_ids)
        fl = [np.asarray(flags)[i][None] for i in range(n)]
        kl = None if k is None else [np.asarray(k)[i][None] for i in range(n)]
        vl = None if v is None else [np.asarray(v)[i][None] for i in range(n)]
        self.append_chunk(seq_ids, fl, kl, vl)

    def seq_reset(self, seq_ids):
        """Return every page of the listed sequences to the stack and clear them."""
        D = self.dims
        P = D.page_size
        for s in seq_ids:
            for h in range(D.num_kv_heads):
                npages = -(-int(self.L[s, h]) // P)
                for i in range(npages):
                    self.stack[self.top] = self.page_table[s, h, i]
                    self.top += 1
                self.page_table[s, h, :] = -1
                self.slot_pos[s, h, :] = -1
                self.slot_flag[s, h, :] = 0
            self.pos[s] = 0
            self.L[s] = 0
            self.ring_slot[s] = -1
            self.ring_flag[s] = 0

    # -- attention over the live slots (compact route) -------------------------
    def live_positions(self, s, h):
        return self.slot_pos[s, h, : self.L[s, h]].copy()

    def attend(self, s, h, q_group, scale=None):
        """Plain softmax over the live slots of head h: q_group [g, d] -> [g, d]."""
        n = int(self.L[s, h])
        q = np.asarray(q_group, np.float64)
        if scale is None:
            scale = 1.0 / math.sqrt(q.shape[-1])
        k = self.k_store[s, h, :n]
        v = self.v_store[s, h, :n]
        return masked_attention(q, k, v, np.ones((q.shape[0], n), bool), scale)

    def decode_latent(self, seq_ids, q, latent, scale=None):
        """Latent-attention decode (one KV head holding the rows, every query
        head in its group): q [n, Hq, d] -> [n, Hq, latent]."""
        q = np.asarray(q, np.float64)
        n, Hq, d = q.shape
        if scale is None:
            scale = 1.0 / math.sqrt(d)
        out = np.empty((n, Hq, latent))
        for i, s in enumerate(seq_ids):
            L = int(self.L[s, 0])
            out[i] = mla_attention(q[i], self.k_store[s, 0, :L], np.ones((Hq, L), bool), latent, scale)
        return out

    def decode(self, seq_ids, q, group, scale=None):
        """q [n, Hq, d] -> [n, Hq, d]: each query head over its KV head's live slots."""
        q = np.asarray(q, np.float64)
        n, Hq, d = q.shape
        out = np.empty((n, Hq, d))
        for i, s in enumerate(seq_ids):
            for h in range(Hq // group):
                out[i, h * group:(h + 1) * group] = self.attend(s, h, q[i, h * group:(h + 1) * group], scale)
        return out

    def free_stack(self):
        return self.stack[: self.top].copy()
