"""Pins of the nested bit-plane format oracle: closed forms (an exactly
representable 16-level row), the nesting of codes and LUTs, the squared-error
order of the two precisions, a bit-by-bit placement check of the page
layout, and the page sizes of Eq. 3."""
import os

import numpy as np

import oracle
from oracle import apl


def test_sixteen_levels_are_recovered_exactly():
    rng = np.random.default_rng(0)
    R, K = 4, 256
    lo = np.array([-0.5, -1.0, 0.25, -0.0625])
    step = np.array([1 / 15, 2 / 15, 1 / 60, 1 / 120])
    lev = rng.integers(0, 16, (R, K))
    lev[:, :16] = np.arange(16)                      # every level present
    v = lo[:, None] + step[:, None] * lev
    v16 = np.array([[oracle.round_nearest16(float(x), oracle.BF16) for x in row] for row in v], np.uint16)
    vv = oracle.decode16(v16, oracle.BF16).astype(np.float64)
    codes, c4, c8 = apl.quantize_rows(vv)
    np.testing.assert_array_equal(codes >> 4, lev)
    np.testing.assert_array_equal(codes & 15, 0)      # equal members: every split keeps child 0
    levels = np.array([np.unique(row) for row in vv])
    np.testing.assert_array_equal(c4, levels)
    np.testing.assert_array_equal(c8, np.repeat(c4, 16, axis=1))


def test_nesting_and_error_order():
    rng = np.random.default_rng(1)
    R, K = 16, 512
    v16 = synth_bf16(rng.standard_normal((R, K)) * 0.02)
    v = oracle.decode16(v16, oracle.BF16).astype(np.float64)
    codes, c4, c8 = apl.quantize_rows(v)
    # the 4-bit code is the nearest level-4 centroid (the seed's final assignment)
    d = np.abs(v[:, :, None] - c4[:, None, :])
    np.testing.assert_array_equal(codes >> 4, np.argmin(d, axis=2))
    # level-8 centroids refine level 4: per row, the squared error does not grow
    r = np.arange(R)[:, None]
    e4 = ((v - c4[r, codes >> 4]) ** 2).sum(axis=1)
    e8 = ((v - c8[r, codes]) ** 2).sum(axis=1)
    assert np.all(e8 <= e4) and np.all(e8 < 0.05 * e4)
    # every value lies within its 8-bit cluster's span around the centroid
    assert np.all(np.abs(v - c8[r, codes]) <= np.abs(v - c4[r, codes >> 4]) + (v.max() - v.min()))


def synth_bf16(x):
    return np.array([[oracle.round_nearest16(float(t), oracle.BF16) for t in row] for row in x], np.uint16)


def test_plane_layout_bit_placement():
    R, K = 32, 256
    for (r, k, code) in [(0, 0, 0x80), (17, 131, 0x01), (31, 255, 0xA5), (5, 77, 0x3C)]:
        codes = np.zeros((R, K), np.uint8)
        codes[r, k] = code
        buf = apl.encode_page(codes, np.zeros((R, 16), np.uint16), np.zeros((R, 256), np.uint16))
        rk8 = R * K // 8
        rt, kb = r // 16, k // 128
        kk = k % 128
        i, lg, q = kk // 32, (kk % 32) // 8, kk % 8
        lane = 16 * lg + r % 16
        t = rt * (K // 128) + kb
        want = np.zeros_like(buf)
        for j in range(8):
            if (code >> (7 - j)) & 1:
                base = j * rk8 if j < 4 else 4 * rk8 + 32 * R + (j - 4) * rk8
                bitpos = 8 * i + q
                want[base + 256 * t + 4 * lane + bitpos // 8] |= 1 << (bitpos % 8)
        np.testing.assert_array_equal(buf, want)
        for bits in (8, 4):
            c, _ = apl.decode_page(buf, R, K, bits)
            assert c[r, k] == code >> (8 - bits) and np.count_nonzero(c) == (1 if code >> (8 - bits) else 0)


def test_page_sizes_eq3():
    R, K = 128, 4096
    assert apl.page_bytes(R, K, 8) == R * K + 32 * R + 512 * R
    assert apl.page_bytes(R, K, 4) == R * K // 2 + 32 * R
    # dropping planes 4-7 and the 8-bit LUT releases exactly the page tail
    assert apl.page_bytes(R, K, 8) - apl.page_bytes(R, K, 4) == R * K // 2 + 512 * R
    assert apl.page_bytes(R, K, 4) % 256 == 0 and apl.page_bytes(R, K, 8) % 256 == 0


def test_dequant_uses_the_committed_precision():
    rng = np.random.default_rng(3)
    R, K = 16, 128
    v = oracle.decode16(synth_bf16(rng.standard_normal((R, K)) * 0.02), oracle.BF16).astype(np.float64)
    codes, c4, c8 = apl.quantize_rows(v)
    l4, l8 = apl.lut16(c4, oracle.BF16), apl.lut16(c8, oracle.BF16)
    buf = apl.encode_page(codes, l4, l8)
    for bits, lut in ((8, l8), (4, l4)):
        c, lt = apl.decode_page(buf, R, K, bits)
        np.testing.assert_array_equal(lt, lut)
        w = apl.dequant(codes, lt, bits)
        np.testing.assert_array_equal(w, np.take_along_axis(lut, (codes >> (8 - bits)).astype(np.int64), 1))


def _golden(name):
    out = {}
    for line in open(os.path.join(os.path.dirname(__file__), "golden", name)):
        line = line.split("#", 1)[0].strip()
        if "=" in line:
            k, v = line.split("=", 1)
            out[k.strip()] = v.split()
    return out


def test_split_level_matches_hand_worked_example():
    """The one-bit split (child initialisation, exactly 4 Lloyd iterations,
    strict nearness for child 1, empty parent) reproduces the hand-worked
    example in tests/golden/apl_split_example.txt bit for bit."""
    from fractions import Fraction
    g = _golden("apl_split_example.txt")
    v = np.array([[float(x) for x in g["values"]]])
    a = np.array([[int(x) for x in g["parents"]]])
    c = np.array([[float(x) for x in g["centroids"]]])
    codes, ch = apl.split_level(v, a, c)
    assert codes.tolist() == [[int(x) for x in g["codes"]]]
    want = [float(Fraction(x)) for x in g["child_centroids"]]
    assert ch.tolist() == [want]


def test_split_iteration_count_is_visible():
    """The example discriminates the iteration count: 3 or 5 Lloyd
    iterations give other codes than the 4 the reading fixes."""
    g = _golden("apl_split_example.txt")
    v = np.array([[float(x) for x in g["values"]]])
    a = np.array([[int(x) for x in g["parents"]]])
    c = np.array([[float(x) for x in g["centroids"]]])
    want = [int(x) for x in g["codes"]]
    saved = apl.SPLIT_ITERS
    try:
        for n in (3, 5):
            apl.SPLIT_ITERS = n
            codes, _ = apl.split_level(v, a, c)
            assert codes.tolist() != [want], n
    finally:
        apl.SPLIT_ITERS = saved
