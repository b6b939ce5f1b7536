"""Pins of the oracle's quantizer (Sec. 5.2) against facts fixed outside the oracle:
a worked example derived by hand from the paper's figure, published generator
outputs, closed-form invariants, and the paper's stated sum widths / sizes."""
import json
import os

import numpy as np
import pytest

from oracle import hack_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rand_f16(seed, shape, scale=1.0):
    g = np.random.default_rng(seed)
    return (g.standard_normal(shape, dtype=np.float32) * np.float32(scale)).astype(np.float16)


def test_worked_example_last_v_block():
    """Sec. 5.3 figure: [-2.1, 1.7] then -2.9 appended below the old minimum."""
    ex = json.load(open(os.path.join(GOLDEN, "v_last_group.json")))
    for key in ("old_block", "new_block"):
        blk = ex[key]
        c, m, s, tot = O.quantize_partition(np.array(blk["values"], np.float16), ex["bits"])
        assert list(c) == blk["codes"]
        assert float(m) == blk["min"]
        assert float(s) == blk["scale"]
        assert tot == sum(blk["codes"])
    # the appended value lies below the old minimum: the open block's range changes
    assert np.float16(ex["new_block"]["values"][2]) < ex["old_block"]["min"]


def test_splitmix64_published_outputs():
    """Reference outputs of SplitMix64 seeded with 0: the first two draws."""
    out = O.splitmix64(np.array([0, 0x9E3779B97F4A7C15], np.uint64))
    assert int(out[0]) == 0xE220A8397B1DCDAF
    assert int(out[1]) == 0x6E789E6AA1B965F4


@pytest.mark.parametrize("bits", [2, 4, 8])
def test_code_range_and_extremes(bits):
    x = _rand_f16(1, (200, 32))
    c, m, s, tot = O.quantize_partition(x, bits)
    q = (1 << bits) - 1
    assert c.min() >= 0 and c.max() <= q
    # nearest rounding maps the minimum to 0 and the maximum to 2^b - 1
    rows = np.arange(x.shape[0])
    assert np.all(c[rows, np.argmin(x, axis=1)] == 0)
    assert np.all(c[rows, np.argmax(x, axis=1)] == q)
    assert np.all(c.sum(axis=1) == tot)
    assert np.all(m == x.min(axis=1).astype(np.float32))


@pytest.mark.parametrize("bits", [2, 4, 8])
def test_reconstruction_error_nearest(bits):
    x = _rand_f16(2, (500, 64), scale=3.0)
    c, m, s, _ = O.quantize_partition(x, bits)
    xhat = s[:, None].astype(np.float64) * c + m[:, None]
    err = np.abs(x.astype(np.float64) - xhat)
    assert np.all(err <= s[:, None] * (0.5 + 2.0 ** -14))


@pytest.mark.parametrize("bits", [2, 4])
def test_nearest_grid_point(bits):
    """Each code is the grid point closest to x: neighbours c-1 and c+1 are not closer."""
    x = _rand_f16(3, (300, 32))
    c, m, s, _ = O.quantize_partition(x, bits)
    xf = x.astype(np.float64)
    s = s[:, None].astype(np.float64)
    m = m[:, None].astype(np.float64)
    d0 = np.abs(xf - (m + s * c))
    q = (1 << bits) - 1
    for step in (-1, 1):
        cn = c + step
        ok = (cn >= 0) & (cn <= q)
        dn = np.abs(xf - (m + s * cn))
        assert np.all(d0[ok] <= dn[ok] + 1e-6 * s.repeat(32, 1)[ok])


def test_scale_is_fp16_rounded_up():
    x = _rand_f16(4, (1000, 32))
    _, m, s, _ = O.quantize_partition(x, 2)
    true = (x.max(axis=1).astype(np.float64) - x.min(axis=1)) / 3.0
    assert np.all(s >= true * (1 - 2.0 ** -23))
    assert np.all(s.astype(np.float16).astype(np.float32) == s)          # representable in fp16
    below = np.nextafter(s.astype(np.float16), np.float16(0)).astype(np.float64)
    assert np.all(below < true * (1 + 2.0 ** -22))                       # the next fp16 down is too small


def test_power_of_two_scaling():
    """x -> 4x is exact in fp16: codes unchanged, min and scale scale by 4."""
    x = _rand_f16(5, (100, 32))
    c1, m1, s1, _ = O.quantize_partition(x, 4)
    c2, m2, s2, _ = O.quantize_partition((x.astype(np.float32) * 4).astype(np.float16), 4)
    assert np.array_equal(c1, c2)
    assert np.array_equal(m2, m1 * 4) and np.array_equal(s2, s1 * 4)


def test_constant_partition():
    x = np.full((3, 32), 1.25, np.float16)
    c, m, s, tot = O.quantize_partition(x, 2)
    assert np.all(c == 0) and np.all(s == 0) and np.all(m == 1.25) and np.all(tot == 0)


def test_stochastic_error_and_unbiasedness():
    x = _rand_f16(6, (1, 32))
    bits = 2
    c0, m, s, _ = O.quantize_partition(x, bits)
    t = (x.astype(np.float64) - float(m[0])) / float(s[0])
    draws = []
    for seed in range(4000):
        u = O.stochastic_threshold(seed, O.STREAM_K, np.arange(32))
        c, m2, s2, _ = O.quantize_partition(x, bits, rounding=O.STOCHASTIC, u=u[None, :])
        assert m2[0] == m[0] and s2[0] == s[0]
        err = np.abs(x.astype(np.float64) - (float(s[0]) * c + float(m[0])))
        assert np.all(err < float(s[0]) * (1 + 2.0 ** -14))
        draws.append(c[0])
    mean = np.mean(draws, axis=0)
    # E[c] = t; standard error <= 0.5/sqrt(4000) ~ 0.008
    assert np.max(np.abs(mean - t[0])) < 0.04


def test_stochastic_thresholds_uniform():
    u = O.stochastic_threshold(123, O.STREAM_V, np.arange(100000))
    assert u.min() >= 0 and u.max() < 1
    assert abs(u.mean() - 0.5) < 0.01
    assert abs((u < 0.25).mean() - 0.25) < 0.01


def test_sum_width_matches_paper():
    """Sec. 5.3: Pi=64 with 2 bits needs at most 8 bits per sum; Sec. 6: Pi=128 with
    2 bits needs 9 bits and is stored as INT16."""
    assert 64 * 3 < 256 and O.sum_bytes(2, 64) == 1
    assert 128 * 3 >= 256 and O.sum_bytes(2, 128) == 2
    assert O.sum_bytes(2, 32) == 1 and O.sum_bytes(4, 16) == 1 and O.sum_bytes(4, 32) == 2


def test_compressed_size_matches_paper():
    """Sec. 7.2: compressed KV is about 15% of fp16 (2-bit codes, Pi=64, fp16 min/scale);
    Sec. 6: INT16 sums are about 5% of the quantized KV (2-bit, Pi=128)."""
    pi = 64
    per_partition = pi * 2 // 8 + 4          # codes + fp16 min + fp16 scale
    assert per_partition / (pi * 2) == 0.15625
    pi = 128
    assert abs(2 / (pi * 2 // 8 + 4) - 0.05) < 0.01


def test_pack_lsb_first():
    assert list(O.pack_codes([1, 2, 3, 0], 2)) == [0x39]
    assert list(O.pack_codes([0xA, 0x5], 4)) == [0x5A]
    g = np.random.default_rng(7)
    for bits in (2, 4, 8):
        c = g.integers(0, 1 << bits, size=(5, 64))
        assert np.array_equal(O.unpack_codes(O.pack_codes(c, bits), bits), c)


# --- planted mistakes: each variant must be caught by one of the pins above -----------
def _floor_quantizer(x, bits, meta="f16", rounding=0, u=None):
    c, m, s, tot = O.quantize_partition(x, bits, meta, rounding, u)
    xf = np.asarray(x).astype(np.float32)
    t = (xf - m[..., None]) / np.where(s == 0, 1, s)[..., None]
    c = np.minimum(np.floor(t), (1 << bits) - 1).astype(np.int64)
    return c, m, s, c.sum(-1)


def _round_to_nearest_scale(x, bits, meta="f16", rounding=0, u=None):
    xf = np.asarray(x).astype(np.float32)
    lo = xf.min(-1)
    s = ((xf.max(-1) - lo) / np.float32((1 << bits) - 1)).astype(np.float16).astype(np.float32)
    t = (xf - lo[..., None]) * (1 / s[..., None])
    c = np.rint(t).astype(np.int64)            # no clamp, scale rounded to nearest
    return c, lo, s, c.sum(-1)


def test_planted_mistakes_are_caught(monkeypatch):
    ex = json.load(open(os.path.join(GOLDEN, "v_last_group.json")))
    x = np.array(ex["new_block"]["values"], np.float16)
    c, _, _, _ = _floor_quantizer(x, 2)
    assert list(c) != ex["new_block"]["codes"]           # floor rounding fails the worked example
    xr = _rand_f16(8, (2000, 32))
    c, m, s, _ = _round_to_nearest_scale(xr, 2)
    assert c.max() > 3 or np.any(s < (xr.max(1).astype(np.float64) - xr.min(1)) / 3)   # range pin fails


# ---- the requantizing open block (the alternative to requantization elimination, R15) ----
def test_requantizing_append_reproduces_the_worked_example():
    """Sec. 5.3's figure: the open block holds -2.1 and 1.7 (codes 0, 3); appending -2.9
    (below the old minimum) through dequantize -> add -> quantize gives the hand-derived
    block of tests/golden (codes 1, 3, 0 with the new min and the fp16-rounded-up scale)."""
    ex = json.load(open(os.path.join(GOLDEN, "v_last_group.json")))
    v = np.zeros((2, 32), np.float16)
    v[:, 0] = np.array(ex["old_block"]["values"], np.float16)
    sq = O.quantize_sequence(np.zeros((2, 32), np.float16), v, ex["bits"], 32)
    assert list(sq.v_codes[0, :2, 0]) == ex["old_block"]["codes"]
    new = np.zeros(32, np.float16)
    new[0] = ex["new_block"]["values"][2]
    sq2 = O.append_requantizing(sq, np.zeros(32, np.float16), new, ex["bits"])
    assert list(sq2.v_codes[0, :3, 0]) == ex["new_block"]["codes"]
    assert float(sq2.v_min[0, 0]) == ex["new_block"]["min"]
    assert float(sq2.v_scale[0, 0]) == ex["new_block"]["scale"]
    assert sq2.v_sum[0, 0] == sum(ex["new_block"]["codes"]) and sq2.v_count[0] == 3


def test_requantizing_append_matches_fresh_quantization_where_nothing_was_requantized():
    """K rows never depend on the open block; a token that opens a new block (n = 1) and
    a block closed from a fresh start agree with quantizing the longer sequence."""
    k = _rand_f16(3, (70, 128))
    v = _rand_f16(4, (70, 128))
    sq = O.quantize_sequence(k[:64], v[:64], 2, 32)
    sq = O.append_requantizing(sq, k[64], v[64], 2)           # opens block 2 with one token
    ref = O.quantize_sequence(k[:65], v[:65], 2, 32)
    for f in ("k_codes", "k_min", "k_scale", "k_sum", "v_codes", "v_min", "v_scale", "v_sum", "v_count"):
        assert np.array_equal(getattr(sq, f), getattr(ref, f)), f
    for t in range(65, 70):
        sq = O.append_requantizing(sq, k[t], v[t], 2)
    ref = O.quantize_sequence(k[:70], v[:70], 2, 32)
    assert np.array_equal(sq.k_codes, ref.k_codes) and np.array_equal(sq.k_scale, ref.k_scale)
    assert np.array_equal(sq.v_codes[:2], ref.v_codes[:2])      # closed blocks untouched


def test_requantizing_error_accumulates_within_its_bound():
    """Building a block by 32 requantizing appends keeps every earlier rounding error:
    each element's error |x - x_hat| stays within the sum of s/2 over the quantizations it
    went through, and on average exceeds the error of quantizing the originals once."""
    bits, Pi, d = 2, 32, 128
    k = _rand_f16(5, (Pi, d))
    v = _rand_f16(6, (Pi, d))
    sq = O.quantize_sequence(k[:0], v[:0], bits, Pi)
    bound = np.zeros((Pi, d))
    for t in range(Pi):
        sq = O.append_requantizing(sq, k[t], v[t], bits)
        bound[:t + 1] += sq.v_scale[0][None, :] * (0.5 + 2.0 ** -14)
    vhat = sq.v_codes[0] * sq.v_scale[0][None, :] + sq.v_min[0][None, :]
    err = np.abs(vhat - v.astype(np.float64))
    # every step also rounds the dequantized values to fp16 (half an ulp of |x| <= 2^-11 |x|)
    assert np.all(err <= bound + Pi * 2.0 ** -11 * (np.abs(v.astype(np.float64)) + 8.0))
    once = O.quantize_sequence(k, v, bits, Pi)
    err_once = np.abs(once.v_codes[0] * once.v_scale[0][None, :] + once.v_min[0][None, :] - v.astype(np.float64))
    assert err.mean() > err_once.mean()
