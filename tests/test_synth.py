"""The seeded input generators: published test vector, NumPy vs PyTorch
agreement element by element, and the distributions they claim."""
import numpy as np
import torch

import dms_synth as sy


def test_splitmix64_published_sequence():
    # SplitMix64 seeded with 1234567 (state advanced by the golden gamma
    # before each output), as published with the reference generator.
    state, out = 1234567, []
    for _ in range(5):
        out.append(sy.splitmix64_int(state))
        state = (state + 0x9E3779B97F4A7C15) & ((1 << 64) - 1)
    assert out == [6457827717110365317, 3203168211198807973, 9817491932198370423,
                   4593380528125082431, 16408922859458223821]


def test_numpy_and_torch_hash_agree():
    x = np.array([0, 1, 2**40 + 7, 2**63 + 5, 2**64 - 1], dtype=np.uint64)
    a = sy.splitmix64_np(x)
    b = sy.splitmix64_torch(torch.from_numpy(x.view(np.int64))).numpy().view(np.uint64)
    assert np.array_equal(a, b)
    assert [int(v) for v in a] == [sy.splitmix64_int(int(v)) for v in x]


def test_flags_numpy_torch_agree_and_rate():
    seqs = np.arange(5)[:, None, None]
    heads = np.arange(3)[None, :, None]
    pos = np.arange(4000)[None, None, :]
    for p in (0.5, 0.75, 0.875):
        a = sy.flags_np(7, p, 2, seqs, heads, pos)
        b = sy.flags_torch(7, p, 2, torch.from_numpy(seqs), torch.from_numpy(heads),
                           torch.from_numpy(pos), "cpu").numpy()
        assert np.array_equal(a, b)
        assert abs(a.mean() - p) < 0.01


def test_vectors_numpy_torch_agree_and_moments():
    pos = np.arange(300)[:, None]
    dim = np.arange(128)[None, :]
    a = sy.token_vectors_np(3, sy.STREAM_K, 1, 9, 2, pos, dim)
    b = sy.token_vectors_torch(3, sy.STREAM_K, 1, 9, 2, torch.from_numpy(pos),
                               torch.from_numpy(dim), "cpu")
    assert np.array_equal(a, b.view(torch.int16).numpy().view(np.uint16))
    f = sy.bf16_bits_to_f32_np(a)
    assert abs(f.mean()) < 0.02 and abs(f.std() - 1.0) < 0.02
    assert np.abs(f).max() < 3.5


def test_chunk_generator_layout():
    x = sy.chunk_vectors_torch(5, sy.STREAM_V, 0, [3, 1], 2, 10, 6, 8, "cpu", max_elems=64)
    for t in range(6):
        for i, s in enumerate([3, 1]):
            for h in range(2):
                ref = sy.token_vectors_np(5, sy.STREAM_V, 0, s, h, 10 + t, np.arange(8))
                assert np.array_equal(x[t, i, h].view(torch.int16).numpy().view(np.uint16), ref)


def test_bf16_rounding_is_nearest_even():
    x = np.array([1.0, 1.0 + 2**-8, 1.0 + 3 * 2**-8, -2.5, 3.0e-3], dtype=np.float32)
    bits = sy.f32_to_bf16_bits_np(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(bits, ref)
    assert sy.bf16_bits_to_f32_np(bits)[1] == 1.0           # tie rounds to even
    assert sy.bf16_bits_to_f32_np(bits)[2] == 1.0 + 2**-6   # tie rounds up to even


def test_beta71_rates():
    r = sy.beta71_rates_np(4, 0, np.arange(256)[:, None], np.arange(8)[None, :]) / 2**24
    # Beta(7, 1) has mean 7/8
    assert abs(r.mean() - 0.875) < 0.02 and r.min() > 0.2 and r.max() < 1.0


def test_wide_vectors_have_distinct_coordinates():
    """576-wide rows: every (head, element) pair of up to 16 heads maps to its
    own generator coordinate, so no two elements of any rows share a draw."""
    import numpy as np
    import dms_synth as sy
    heads = np.arange(16)[:, None]
    dims = np.arange(576)[None, :]
    h, d = sy.wide_coords(heads, dims, 576)
    assert d.max() < 256 and h.max() < (1 << sy.HEAD_BITS)
    keys = (h << sy.DIM_BITS) + d
    assert len(np.unique(keys)) == 16 * 576
    v = sy.token_vectors_np(5, sy.STREAM_K, 0, 0, h, 7, d)
    assert len(np.unique(v)) > 1000
