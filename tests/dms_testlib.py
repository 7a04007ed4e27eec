"""Helpers shared by the GPU parity tests: seeded inputs, a GPU cache driven
through the C ABI binding, and element-by-element state comparison against
the CPU oracle."""
from __future__ import annotations

import numpy as np

import dms_synth as sy
from oracle import PagedKVOracle

ATOL = 1e-2   # outputs vs oracle (bf16 q/k/v, fp32 accumulate)


def bf16_to_f32(bits):
    return sy.bf16_bits_to_f32_np(bits)


class SeqInputs:
    """Host-side seeded inputs of one sequence for positions 0 .. T-1.

    flags [T, Hkv] u8, k / v [T, Hkv, d] and q [T, Hq, d] as bf16 bit patterns.
    """

    def __init__(self, seed, layer, seq, T, Hkv, g, d, p, q_scale=1.0):
        pos = np.arange(T)
        self.flags = sy.flags_np(seed, p, layer, seq, np.arange(Hkv)[None, :], pos[:, None])
        hd = np.arange(Hkv)[None, :, None]
        qd = np.arange(Hkv * g)[None, :, None]
        dim = np.arange(d)[None, None, :]
        pp = pos[:, None, None]
        self.k = sy.token_vectors_np(seed, sy.STREAM_K, layer, seq, hd, pp, dim)
        self.v = sy.token_vectors_np(seed, sy.STREAM_V, layer, seq, hd, pp, dim)
        self.q = sy.token_vectors_np(seed, sy.STREAM_Q, layer, seq, qd, pp, dim)
        if q_scale != 1.0:
            self.q = sy.f32_to_bf16_bits_np(bf16_to_f32(self.q) * np.float32(q_scale))


def to_dev(x, dtype=None):
    import torch
    a = np.ascontiguousarray(x)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).cuda().view(torch.bfloat16)
    return torch.from_numpy(a).cuda()


def compare_state(view, orc: PagedKVOracle, seqs, check_pages=True):
    """Bit-exact comparison of a GPU layer state against the oracle for the
    given sequences (plus the whole free stack)."""
    D = orc.dims
    P, w = D.page_size, D.window
    for s in seqs:
        assert view.pos[s] == orc.pos[s], (s, view.pos[s], orc.pos[s])
        assert np.array_equal(view.L[s], orc.L[s]), (s, view.L[s], orc.L[s])
        t = int(orc.pos[s])
        for p in range(max(0, t - w), t):
            e = p % w
            assert np.array_equal(view.ring_slot[s, :, e], orc.ring_slot[s, :, e]), (s, p)
            assert np.array_equal(view.ring_flag[s, :, e], orc.ring_flag[s, :, e]), (s, p)
        for h in range(D.num_kv_heads):
            L = int(orc.L[s, h])
            npg = -(-L // P)
            if check_pages:
                assert np.array_equal(view.page_table[s, h, :npg], orc.page_table[s, h, :npg]), (s, h)
            assert np.array_equal(view.slot_pos[s, h, :L], orc.slot_pos[s, h, :L]), (s, h)
            assert np.array_equal(view.slot_flag[s, h, :L], orc.slot_flag[s, h, :L]), (s, h)
    if check_pages:
        assert view.top == orc.top
        assert np.array_equal(view.stack, orc.free_stack())


def compare_pool(cache, layer, view, seqs, inputs_by_seq):
    """Every live slot holds the K / V bits of the position that owns it."""
    import torch
    from paper_2506_05345_amd.dms import unpack_page
    c = cache.cfg
    P, Dm = c.page_size, c.head_dim
    raw = cache.pools[layer].view(torch.int16).cpu().numpy().view(np.uint16)
    words = raw.reshape(c.num_pages, -1)
    decoded = {}
    for s in seqs:
        inp = inputs_by_seq[s]
        for h in range(c.num_kv_heads):
            L = int(view.L[s, h])
            for slot in range(L):
                pg = int(view.page_table[s, h, slot // P])
                if pg not in decoded:
                    decoded[pg] = unpack_page(words[pg], P, Dm)
                kk, vv = decoded[pg]
                owner = view.slot_pos[s, h, slot]
                assert np.array_equal(kk[slot % P], inp.k[owner, h]), (s, h, slot)
                assert np.array_equal(vv[slot % P], inp.v[owner, h]), (s, h, slot)


def compare_pool_fp8(cache, orc, seqs, layer=0):
    """FP8 pages: codes and scales of every live slot equal the oracle's
    quantization of the row its owner appended (bit-exact)."""
    view = cache.export(layer)
    c = cache.cfg
    P = c.page_size
    pages = {}
    for s in seqs:
        for h in range(c.num_kv_heads):
            L = int(view.L[s, h])
            for slot in range(L):
                pg = int(view.page_table[s, h, slot // P])
                if pg not in pages:
                    pages[pg] = cache.pool_page_kv(layer, pg)
                kc, vc, ks, vs = pages[pg]
                row = slot % P
                assert np.array_equal(kc[row], orc.k_codes[s, h, slot]), (s, h, slot)
                assert np.array_equal(vc[row], orc.v_codes[s, h, slot]), (s, h, slot)
                assert ks[row] == 2.0 ** orc.k_exp[s, h, slot], (s, h, slot)
                assert vs[row] == 2.0 ** orc.v_exp[s, h, slot], (s, h, slot)
