"""Seeded synthetic inputs for the DMS decode / prefill path.

This module is shared by the tests, the CPU oracle's callers and the benchmark.
It holds none of the method's arithmetic: it only turns (seed, tensor, index)
triples into input values -- eviction flags, and bf16 query / key / value
elements -- so that the same element can be regenerated independently on the
host (NumPy) and on the device (PyTorch) without either side handing data to
the other.

Generator
---------
Every element is a function of a 64-bit counter, hashed with the SplitMix64
output function (Steele, Lea & Flood, "Fast splittable pseudorandom number
generators", OOPSLA 2014; constants as published by Vigna for splitmix64.c):

    z = x + 0x9E3779B97F4A7C15
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9
    z = (z ^ (z >> 27)) * 0x94D049BB133111EB
    z = z ^ (z >> 31)

The counter of an element is ``base(seed, stream) + index`` where ``base`` is
the hash of ``seed * 2**8 + stream`` and ``index`` packs the element's logical
coordinates with fixed strides (``FLAG_INDEX`` / ``VEC_INDEX`` below), so the
value of, say, the key of (layer 3, sequence 17, KV head 5, position 30000,
dim 64) does not depend on how many sequences or positions a run has.

* Flags: Bernoulli(p) with ``flag = (hash >> 40) < round(p * 2**24)``; exact
  for dyadic p such as 1/2, 3/4, 7/8.
* Values: Irwin-Hall(4) approximation of N(0, 1): the four 16-bit fields of the
  hash are summed, centred and scaled by 1/sd in float32 (exact integer sum,
  one IEEE multiply), then rounded to bfloat16 with round-to-nearest-even.
  Values lie in [-3.47, 3.47].

Both implementations (NumPy ``*_np`` and PyTorch ``*_torch``) are checked
against each other element by element in the test suite.
"""
from __future__ import annotations

import math

import numpy as np

# stream ids
STREAM_FLAGS = 1
STREAM_K = 2
STREAM_V = 3
STREAM_Q = 4
STREAM_RATE = 5

# Fixed coordinate strides (bits): layer 8 | seq 12 | head 6 | pos 24 (| dim 8).
POS_BITS = 24
HEAD_BITS = 6
SEQ_BITS = 12
DIM_BITS = 8

_GOLDEN = 0x9E3779B97F4A7C15
_M1 = 0xBF58476D1CE4E5B9
_M2 = 0x94D049BB133111EB
_MASK64 = (1 << 64) - 1

# Irwin-Hall(4) of 16-bit uniforms: mean 4*65535/2, var 4*(65536**2-1)/12
_IH_MEAN = 2 * 65535
_IH_INV_SD = np.float32(1.0 / math.sqrt(4.0 * (65536.0 ** 2 - 1.0) / 12.0))


def _to_signed64(x: int) -> int:
    x &= _MASK64
    return x - (1 << 64) if x >> 63 else x


def splitmix64_int(x: int) -> int:
    """Scalar SplitMix64 output function on Python ints (reference form)."""
    z = (x + _GOLDEN) & _MASK64
    z = ((z ^ (z >> 30)) * _M1) & _MASK64
    z = ((z ^ (z >> 27)) * _M2) & _MASK64
    return z ^ (z >> 31)


def stream_base(seed: int, stream: int) -> int:
    return splitmix64_int(((seed & 0xFFFFFFFFFFFF) << 8) | (stream & 0xFF))


def flag_index(layer, seq, head, pos):
    """Packed counter index of a per-token quantity (flags)."""
    return (((layer * (1 << SEQ_BITS) + seq) * (1 << HEAD_BITS) + head) << POS_BITS) + pos


def vec_index(layer, seq, head, pos, dim):
    """Packed counter index of a per-token vector element (q / k / v)."""
    return (flag_index(layer, seq, head, pos) << DIM_BITS) + dim


def dyadic_threshold(p: float) -> int:
    return int(round(p * (1 << 24)))


# ----------------------------------------------------------------------------
# NumPy implementation
# ----------------------------------------------------------------------------

def splitmix64_np(x: np.ndarray) -> np.ndarray:
    x = x.astype(np.uint64, copy=False)
    with np.errstate(over="ignore"):
        z = x + np.uint64(_GOLDEN)
        z = (z ^ (z >> np.uint64(30))) * np.uint64(_M1)
        z = (z ^ (z >> np.uint64(27))) * np.uint64(_M2)
        return z ^ (z >> np.uint64(31))


def _counters_np(seed, stream, index):
    with np.errstate(over="ignore"):
        return np.uint64(stream_base(seed, stream)) + np.asarray(index, dtype=np.uint64)


def flags_np(seed, p, layer, seq, head, pos) -> np.ndarray:
    """uint8 Bernoulli(p) flags at broadcast coordinates."""
    idx = flag_index(np.asarray(layer, np.uint64), np.asarray(seq, np.uint64),
                     np.asarray(head, np.uint64), np.asarray(pos, np.uint64))
    h = splitmix64_np(_counters_np(seed, STREAM_FLAGS, idx))
    return ((h >> np.uint64(40)) < np.uint64(dyadic_threshold(p))).astype(np.uint8)


def flags_rate_np(seed, rate_threshold, layer, seq, head, pos) -> np.ndarray:
    """Flags with a per-coordinate 24-bit threshold (heterogeneous eviction rates)."""
    idx = flag_index(np.asarray(layer, np.uint64), np.asarray(seq, np.uint64),
                     np.asarray(head, np.uint64), np.asarray(pos, np.uint64))
    h = splitmix64_np(_counters_np(seed, STREAM_FLAGS, idx))
    return ((h >> np.uint64(40)) < np.asarray(rate_threshold, np.uint64)).astype(np.uint8)


def uniform01_np(seed, stream, index) -> np.ndarray:
    """float64 uniforms in [0, 1) with 53 random bits (host-side draws only)."""
    h = splitmix64_np(_counters_np(seed, stream, index))
    return (h >> np.uint64(11)).astype(np.float64) * (1.0 / (1 << 53))


def f32_to_bf16_bits_np(x: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 bit pattern, round to nearest even (finite inputs)."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = b + np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))
    return (r >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32_np(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint32) << np.uint32(16)).view(np.float32)


def normal_bf16_bits_np(seed, stream, index) -> np.ndarray:
    h = splitmix64_np(_counters_np(seed, stream, index))
    m = np.uint64(0xFFFF)
    s = ((h & m) + ((h >> np.uint64(16)) & m) + ((h >> np.uint64(32)) & m)
         + (h >> np.uint64(48))).astype(np.int64) - _IH_MEAN
    f = s.astype(np.float32) * _IH_INV_SD
    return f32_to_bf16_bits_np(f)


def token_vectors_np(seed, stream, layer, seq, head, pos, dim) -> np.ndarray:
    """bf16 bit patterns (uint16) of vector elements at broadcast coordinates."""
    idx = vec_index(np.asarray(layer, np.uint64), np.asarray(seq, np.uint64),
                    np.asarray(head, np.uint64), np.asarray(pos, np.uint64),
                    np.asarray(dim, np.uint64))
    return normal_bf16_bits_np(seed, stream, idx)


def wide_coords(head, dim, width):
    """Coordinates of element ``dim`` of a vector of ``width`` > 256 elements
    (rows of a latent-attention cache, 576 wide): the dim field holds 8 bits,
    so the vector is split into ceil(width / 256) sub-heads.  Works on ints,
    NumPy arrays and torch tensors; returns (head, dim) for the generators."""
    nsub = -(-width // (1 << DIM_BITS))
    return head * nsub + dim // (1 << DIM_BITS), dim % (1 << DIM_BITS)


def head_sequence_np(seed, stream, layer, seq, head, positions, head_dim) -> np.ndarray:
    """[len(positions), head_dim] bf16 bits of one head's vectors at the given positions."""
    pos = np.asarray(positions, np.uint64)[:, None]
    dim = np.arange(head_dim, dtype=np.uint64)[None, :]
    return token_vectors_np(seed, stream, layer, seq, head, pos, dim)


def beta71_rates_np(seed, layer, seq, head) -> np.ndarray:
    """Per-(layer, seq, head) eviction rate p ~ Beta(7, 1) by inverse CDF p = u**(1/7).

    Returned as 24-bit integer thresholds (the exact value both sides compare against).
    """
    idx = flag_index(np.asarray(layer, np.uint64), np.asarray(seq, np.uint64),
                     np.asarray(head, np.uint64), np.uint64(0))
    u = uniform01_np(seed, STREAM_RATE, idx)
    return np.floor(u ** (1.0 / 7.0) * (1 << 24)).astype(np.int64)


# ----------------------------------------------------------------------------
# PyTorch implementation (device-side generation for large workloads)
# ----------------------------------------------------------------------------

def _t():
    import torch
    return torch


def _lshr(x, s):
    """Logical right shift of an int64 tensor holding 64-bit patterns."""
    return (x >> s) & ((1 << (64 - s)) - 1)


def splitmix64_torch(x):
    z = x + _to_signed64(_GOLDEN)
    z = (z ^ _lshr(z, 30)) * _to_signed64(_M1)
    z = (z ^ _lshr(z, 27)) * _to_signed64(_M2)
    return z ^ _lshr(z, 31)


def flags_torch(seed, p, layer, seq, head, pos, device):
    """uint8 flags; ``seq``, ``head``, ``pos`` are broadcastable int64 tensors or ints."""
    torch = _t()
    as_t = lambda a: torch.as_tensor(a, dtype=torch.int64, device=device)
    idx = flag_index(as_t(layer), as_t(seq), as_t(head), as_t(pos))
    h = splitmix64_torch(idx + _to_signed64(stream_base(seed, STREAM_FLAGS)))
    return (_lshr(h, 40) < dyadic_threshold(p)).to(torch.uint8)


def flags_rate_torch(seed, rate_threshold, layer, seq, head, pos, device):
    torch = _t()
    as_t = lambda a: torch.as_tensor(a, dtype=torch.int64, device=device)
    idx = flag_index(as_t(layer), as_t(seq), as_t(head), as_t(pos))
    h = splitmix64_torch(idx + _to_signed64(stream_base(seed, STREAM_FLAGS)))
    return (_lshr(h, 40) < as_t(rate_threshold)).to(torch.uint8)


def token_vectors_torch(seed, stream, layer, seq, head, pos, dim, device):
    """bfloat16 tensor of vector elements at broadcast coordinates."""
    torch = _t()
    as_t = lambda a: torch.as_tensor(a, dtype=torch.int64, device=device)
    idx = vec_index(as_t(layer), as_t(seq), as_t(head), as_t(pos), as_t(dim))
    h = splitmix64_torch(idx + _to_signed64(stream_base(seed, stream)))
    s = ((h & 0xFFFF) + (_lshr(h, 16) & 0xFFFF) + (_lshr(h, 32) & 0xFFFF)
         + _lshr(h, 48)) - _IH_MEAN
    f = s.to(torch.float32) * float(_IH_INV_SD)
    return f.to(torch.bfloat16)


def chunk_vectors_torch(seed, stream, layer, seqs, heads, pos0, ntok, head_dim, device,
                        max_elems=1 << 26):
    """[ntok, len(seqs), heads, head_dim] bf16, token-major (the library's varlen layout
    for equal-length chunks), generated in slabs of at most ``max_elems`` elements."""
    torch = _t()
    seqs_t = torch.as_tensor(seqs, dtype=torch.int64, device=device)
    out = torch.empty((ntok, len(seqs), heads, head_dim), dtype=torch.bfloat16, device=device)
    per_tok = len(seqs) * heads * head_dim
    step = max(1, max_elems // per_tok)
    hh = torch.arange(heads, device=device, dtype=torch.int64)[None, None, :, None]
    dd = torch.arange(head_dim, device=device, dtype=torch.int64)[None, None, None, :]
    ss = seqs_t[None, :, None, None]
    for t0 in range(0, ntok, step):
        t1 = min(ntok, t0 + step)
        pp = torch.arange(pos0 + t0, pos0 + t1, device=device, dtype=torch.int64)[:, None, None, None]
        out[t0:t1] = token_vectors_torch(seed, stream, layer, ss, hh, pp, dd, device)
    return out


def seq_chunk_vectors_torch(seed, stream, layer, seqs, heads, pos0, ntok, head_dim, device,
                            max_elems=1 << 26):
    """[len(seqs), ntok, heads, head_dim] bf16: positions pos0 .. pos0+ntok-1 of
    every listed sequence, sequence-major (the varlen layout of equal-length
    chunks), generated in slabs of at most ``max_elems`` elements."""
    torch = _t()
    seqs_t = torch.as_tensor(seqs, dtype=torch.int64, device=device)
    out = torch.empty((len(seqs), ntok, heads, head_dim), dtype=torch.bfloat16, device=device)
    per_seq_tok = heads * head_dim
    step = max(1, max_elems // (per_seq_tok * ntok))
    hh = torch.arange(heads, device=device, dtype=torch.int64)[None, None, :, None]
    dd = torch.arange(head_dim, device=device, dtype=torch.int64)[None, None, None, :]
    pp = torch.arange(pos0, pos0 + ntok, device=device, dtype=torch.int64)[None, :, None, None]
    for i0 in range(0, len(seqs), step):
        ss = seqs_t[i0:i0 + step][:, None, None, None]
        out[i0:i0 + step] = token_vectors_torch(seed, stream, layer, ss, hh, pp, dd, device)
    return out
