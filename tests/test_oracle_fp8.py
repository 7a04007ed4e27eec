"""Pins for the FP8 (OCP E4M3) KV quantization oracle: values the format
definition fixes, brute-force nearest-value rounding with ties to even,
brute-force search for the row exponent, error bounds, and planted
mistakes."""
import numpy as np
import pytest

import oracle
from oracle import kv_fp8

ALL = np.arange(256)


def test_spot_values_of_the_format():
    # (code, value) fixed by the E4M3 layout: bias 7, 3 mantissa bits, subnormals below 2^-6
    table = {0x00: 0.0, 0x01: 2.0 ** -9, 0x07: 7 * 2.0 ** -9, 0x08: 2.0 ** -6, 0x30: 0.5,
             0x38: 1.0, 0x39: 1.125, 0x3F: 1.875, 0x40: 2.0, 0x78: 256.0, 0x7E: 448.0,
             0xB8: -1.0, 0xFE: -448.0}
    for c, val in table.items():
        assert kv_fp8.e4m3_decode(c) == val, hex(c)
    assert np.isnan(kv_fp8.e4m3_decode(0x7F)) and np.isnan(kv_fp8.e4m3_decode(0xFF))
    assert np.signbit(kv_fp8.e4m3_decode(0x80)) and kv_fp8.e4m3_decode(0x80) == 0.0


def test_codes_are_ordered_and_mirrored():
    v = kv_fp8.e4m3_decode(ALL)
    pos = v[:0x7F]
    assert np.all(np.diff(pos) > 0)                       # 0x00 .. 0x7E strictly increasing
    assert np.array_equal(v[0x80:0xFF], -pos)
    # 126 positive finite values: 7 subnormals and 15 binades x 8 minus the NaN slot
    assert np.count_nonzero(pos > 0) == 126


def test_encode_inverts_decode_on_every_finite_code():
    v = kv_fp8.e4m3_decode(ALL)
    fin = ~np.isnan(v)
    assert np.array_equal(kv_fp8.e4m3_encode(v[fin]), ALL[fin].astype(np.uint8))


def _nearest_even(x):
    """Brute force: the finite code nearest to x, ties to the even code."""
    v = kv_fp8.e4m3_decode(np.arange(0x7F))
    a = np.abs(np.asarray(x, np.float64))
    d = np.abs(a[:, None] - v[None, :])
    best = d == d.min(axis=1, keepdims=True)
    codes = np.arange(0x7F)
    pick = np.where(best.sum(axis=1) == 1, np.argmax(best, axis=1),
                    np.where(best & (codes % 2 == 0), codes, 10 ** 6).min(axis=1))
    return (pick | np.where(np.signbit(x), 0x80, 0)).astype(np.uint8)


def _rounding_inputs():
    v = np.sort(kv_fp8.e4m3_decode(np.arange(0x7F)))
    mids = (v[1:] + v[:-1]) / 2
    f32 = mids.astype(np.float32)
    rng = np.random.default_rng(5)
    x = np.concatenate([v, mids, np.nextafter(f32, np.float32(1e9)), np.nextafter(f32, np.float32(-1e9)),
                        rng.uniform(0, 448, 4000), rng.uniform(0, 2.0 ** -5, 4000)])
    x = np.concatenate([x, -x, [-0.0]]).astype(np.float32).astype(np.float64)
    return x[np.abs(x) <= 448]


def test_encode_is_round_to_nearest_even_by_brute_force():
    x = _rounding_inputs()
    assert np.array_equal(kv_fp8.e4m3_encode(x), _nearest_even(x))


def test_encode_rejects_out_of_range():
    for bad in (448.5, -1000.0, np.inf, np.nan):
        with pytest.raises(ValueError):
            kv_fp8.e4m3_encode(np.array([bad]))


def test_row_exponent_is_the_smallest_that_fits():
    rng = np.random.default_rng(6)
    amax = np.concatenate([448.0 * 2.0 ** np.arange(-20, 10), 224.0 * 2.0 ** np.arange(-20, 10),
                           np.nextafter(448.0 * 2.0 ** np.arange(-20, 10), np.inf),
                           np.exp(rng.uniform(-30, 20, 2000)), [1.0, 0.875, 2.0 ** -133]])
    e = kv_fp8.fp8_row_exponent(amax)
    for a, ei in zip(amax, e):
        # brute force over a window of candidates
        cands = [k for k in range(-200, 200) if a * 2.0 ** -k <= 448.0]
        assert ei == min(cands), (a, ei)
    assert kv_fp8.fp8_row_exponent(0.0) == 0


def test_quantized_rows_land_in_range_and_within_half_a_step():
    rng = np.random.default_rng(7)
    x = rng.normal(size=(500, 128)) * np.exp(rng.uniform(-8, 8, (500, 1)))
    x = x.astype(np.float32).astype(np.float64)
    codes, e = kv_fp8.quantize_rows_fp8(x)
    q = kv_fp8.e4m3_decode(codes)
    xs = x * np.exp2(-e.astype(np.float64))[:, None]            # exact scaling
    # the largest element of each row scales into (224, 448] and rounds into [224, 448]
    smax = np.abs(xs).max(axis=1)
    assert np.all((smax > 224) & (smax <= 448))
    qmax = np.abs(q).max(axis=1)
    assert np.all((qmax >= 224) & (qmax <= 448))
    step = np.where(np.abs(xs) >= 2.0 ** -6, np.exp2(np.floor(np.log2(np.maximum(np.abs(xs), 2.0 ** -6))) - 3),
                    2.0 ** -9)
    assert np.all(np.abs(q - xs) <= step / 2)
    # dequantized = code value times the power-of-two scale, exactly
    assert np.array_equal(kv_fp8.dequantize_rows_fp8(codes, e), q * np.exp2(e.astype(np.float64))[:, None])
    # zero rows stay zero with exponent 0
    c0, e0 = kv_fp8.quantize_rows_fp8(np.zeros((2, 8)))
    assert np.all(c0 == 0) and np.all(e0 == 0)


# ----------------------------------------------------------------------------
# planted mistakes
# ----------------------------------------------------------------------------

def _pins_pass():
    try:
        test_spot_values_of_the_format()
        test_encode_inverts_decode_on_every_finite_code()
        test_encode_is_round_to_nearest_even_by_brute_force()
        test_row_exponent_is_the_smallest_that_fits()
        test_quantized_rows_land_in_range_and_within_half_a_step()
    except AssertionError:
        return False
    return True


def test_pins_pass_unmodified():
    assert _pins_pass()


@pytest.mark.parametrize("mutant", ["bias8", "half_up", "truncate", "exponent_plus_one", "no_subnormals"])
def test_planted_mistake_is_caught(monkeypatch, mutant):
    orig_dec, orig_enc, orig_exp = kv_fp8.e4m3_decode, kv_fp8.e4m3_encode, kv_fp8.fp8_row_exponent
    if mutant == "bias8":   # the FNUZ variant's exponent bias
        monkeypatch.setattr(kv_fp8, "e4m3_decode", lambda c: orig_dec(c) / 2.0)
    elif mutant == "half_up":
        def enc(x):
            x = np.asarray(x, np.float64)
            c = orig_enc(x).astype(np.int64)
            v = orig_dec(c)
            up = np.nextafter(np.abs(v), np.inf)
            # a tie that went down to an even code goes up instead
            nxt = orig_dec(np.minimum((c & 0x7F) + 1, 0x7E))
            tie = np.abs(np.abs(x) - (np.abs(v) + nxt) / 2) == 0
            return np.where(tie & (np.abs(x) > np.abs(v)) & (up > 0), c + 1, c).astype(np.uint8)
        monkeypatch.setattr(kv_fp8, "e4m3_encode", enc)
    elif mutant == "truncate":
        def enc(x):
            x = np.asarray(x, np.float64)
            v = orig_dec(np.arange(0x7F))
            idx = np.searchsorted(v, np.abs(x), side="right") - 1
            return (idx | np.where(np.signbit(x), 0x80, 0)).astype(np.uint8)
        monkeypatch.setattr(kv_fp8, "e4m3_encode", enc)
    elif mutant == "exponent_plus_one":
        monkeypatch.setattr(kv_fp8, "fp8_row_exponent", lambda a: orig_exp(a) + 1)
    elif mutant == "no_subnormals":
        def enc(x):
            c = orig_enc(x)
            return np.where((c & 0x78) == 0, c & 0x80, c).astype(np.uint8)
        monkeypatch.setattr(kv_fp8, "e4m3_encode", enc)
    assert not _pins_pass()


def test_paged_replay_in_fp8_attends_the_quantized_history():
    """The fp8 replay's compact route equals dense masked attention over the
    row-wise fake-quantized history, and its stored codes are those rows'."""
    rng = np.random.default_rng(8)
    H, g, d, w, T = 2, 3, 16, 5, 40
    k = rng.normal(size=(T, H, d)) * 3
    v = rng.normal(size=(T, H, d))
    flags = (rng.uniform(size=(T, H)) < 0.6).astype(np.uint8)
    q = rng.normal(size=(T, H * g, d))
    orc = oracle.PagedKVOracle(1, H, w, 8, 64, 16, d, kv_format="fp8")
    kq, vq = oracle.fake_quantize_fp8(k), oracle.fake_quantize_fp8(v)
    for t in range(T):
        orc.append([0], flags[t][None], k[t][None], v[t][None])
        got = orc.decode([0], q[t][None], g)[0]
        ref = oracle.dense_dms_attention(q[t][None], kq[: t + 1], vq[: t + 1], flags[: t + 1], w, g,
                                         t_query=[t])[0]
        assert np.allclose(got, ref, rtol=0, atol=1e-12)
    for h in range(H):
        n = int(orc.L[0, h])
        pos = orc.live_positions(0, h)
        codes, e = oracle.quantize_rows_fp8(k[pos, h])
        assert np.array_equal(orc.k_codes[0, h, :n], codes) and np.array_equal(orc.k_exp[0, h, :n], e)
