"""Full-size parity harness: one layer of a workload built on the device from
the counter-based generators, replayed by the oracle for every head, with
sampled outputs checked against dense masked attention over the full history."""
from __future__ import annotations

import numpy as np

import dms_synth as sy
from dms_testlib import ATOL, bf16_to_f32, compare_state
from oracle import PagedKVOracle, dense_dms_attention_head


class Workload:
    """One layer: per-sequence contexts and per-(seq, head) 24-bit eviction
    thresholds; flags, keys, values and queries come from the hash."""

    def __init__(self, seed, layer, B, H, g, D, w, contexts, thresholds, P=64):
        self.seed, self.layer = seed, layer
        self.B, self.H, self.g, self.D, self.w, self.P = B, H, g, D, w, P
        self.ctx = np.asarray(contexts, np.int64)
        self.thr = np.asarray(thresholds, np.int64).reshape(B, H)

    def flags_host(self, s, positions):
        """[len(positions), H] flags of sequence s."""
        pos = np.asarray(positions)[:, None]
        return sy.flags_rate_np(self.seed, self.thr[s][None, :], self.layer, s,
                                np.arange(self.H)[None, :], pos)

    def flags_dev(self, seqs_t, heads_t, pos_t, dev):
        import torch
        thr = torch.as_tensor(self.thr, device=dev)
        return sy.flags_rate_torch(self.seed, thr[seqs_t, heads_t], self.layer, seqs_t, heads_t,
                                   pos_t, dev)

    def vec_host(self, stream, s, head, positions):
        return sy.head_sequence_np(self.seed, stream, self.layer, s, head, positions, self.D)


def build(dms, cache, wl: Workload, orc: PagedKVOracle, starts, stops, chunk, dev="cuda"):
    """Append positions starts[s] .. stops[s]-1 of every sequence through
    dms_append_chunk in pieces of `chunk`, replaying them in the oracle."""
    import torch
    B, H, D = wl.B, wl.H, wl.D
    seqs = np.arange(B)
    cur = np.asarray(starts, np.int64).copy()
    stops = np.asarray(stops, np.int64)
    sid = torch.arange(B, dtype=torch.int32, device=dev)
    heads_t = torch.arange(H, device=dev)
    while (cur < stops).any():
        lens = np.minimum(chunk, stops - cur)
        cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
        T = int(cu[-1])
        seq_of = np.repeat(seqs, lens)
        pos = np.concatenate([np.arange(cur[s], cur[s] + lens[s]) for s in seqs])
        seq_t = torch.as_tensor(seq_of, device=dev)
        pos_t = torch.as_tensor(pos, device=dev)
        k = sy.token_vectors_torch(wl.seed, sy.STREAM_K, wl.layer, seq_t[:, None, None],
                                   heads_t[None, :, None], pos_t[:, None, None],
                                   torch.arange(D, device=dev)[None, None, :], dev)
        v = sy.token_vectors_torch(wl.seed, sy.STREAM_V, wl.layer, seq_t[:, None, None],
                                   heads_t[None, :, None], pos_t[:, None, None],
                                   torch.arange(D, device=dev)[None, None, :], dev)
        f = wl.flags_dev(seq_t[:, None], heads_t[None, :], pos_t[:, None], dev)
        dms.dms_append_chunk(cache.ctx, 0, B, sid, torch.as_tensor(cu, device=dev), T,
                             int(lens.max()), k, v, f)
        host_f = f.cpu().numpy()
        orc.append_chunk(list(seqs), [host_f[cu[i]:cu[i + 1]] for i in range(B)])
        cur += lens
        del k, v
    torch.cuda.synchronize()
    assert dms.dms_status(cache.ctx) == 0


def closed_form_L(wl: Workload, s, T):
    """Retained count of every head of sequence s after T tokens."""
    if T <= wl.w:
        return np.full(wl.H, T)
    f = wl.flags_host(s, np.arange(T - wl.w))
    return wl.w + (f == 0).sum(axis=0)


def check_decode_sample(wl: Workload, got, q_bits, s, h, t):
    """Outputs of the g query heads of (s, h) at position t vs dense attention."""
    hist = np.arange(t + 1)
    kh = wl.vec_host(sy.STREAM_K, s, h, hist)
    vh = wl.vec_host(sy.STREAM_V, s, h, hist)
    fh = wl.flags_host(s, hist)[:, h]
    g = wl.g
    ref = dense_dms_attention_head(bf16_to_f32(q_bits)[None], bf16_to_f32(kh), bf16_to_f32(vh),
                                   fh, wl.w, [t])[0]
    err = np.abs(got - ref).max()
    assert err <= ATOL, (s, h, t, err)
    return err


def decode_step_inputs(wl: Workload, seqs, positions):
    """q [n, Hq, d], k / v [n, H, d] bits and flags [n, H] at per-sequence positions."""
    H, g, D = wl.H, wl.g, wl.D
    seqs = np.asarray(seqs)
    pos = np.asarray(positions)
    dd = np.arange(D)[None, None, :]
    q = sy.token_vectors_np(wl.seed, sy.STREAM_Q, wl.layer, seqs[:, None, None],
                            np.arange(H * g)[None, :, None], pos[:, None, None], dd)
    k = sy.token_vectors_np(wl.seed, sy.STREAM_K, wl.layer, seqs[:, None, None],
                            np.arange(H)[None, :, None], pos[:, None, None], dd)
    v = sy.token_vectors_np(wl.seed, sy.STREAM_V, wl.layer, seqs[:, None, None],
                            np.arange(H)[None, :, None], pos[:, None, None], dd)
    f = np.stack([wl.flags_host(s, [p])[0] for s, p in zip(seqs, pos)])
    return q, k, v, f


def to_bf16_dev(bits, dev="cuda"):
    import torch
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(dev).view(torch.bfloat16)
