"""Pins of the oracle's 16-bit formats and group-wise RTN quantizer.

Each check compares the oracle with something other than itself: numpy/torch
conversions, exact rational arithmetic (``fractions``), brute force over all
codes, or constructed inputs whose exact answer is known in closed form.
"""
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle

F16, BF16 = oracle.F16, oracle.BF16


def _bf16_bits(x32: np.ndarray) -> np.ndarray:
    return torch.from_numpy(np.ascontiguousarray(x32, np.float32)).to(torch.bfloat16) \
        .view(torch.int16).numpy().view(np.uint16)


def _val(h: int, fmt: int) -> float:
    """Value of a 16-bit pattern via numpy / torch (independent of the oracle)."""
    if fmt == F16:
        return float(np.array([h], np.uint16).view(np.float16)[0])
    return float(torch.tensor([h], dtype=torch.int32).to(torch.int16).view(torch.bfloat16).float()[0])


def _frac16(h: int, fmt: int) -> Fraction:
    return Fraction(_val(h, fmt))


# ---------------------------------------------------------------------------
# 16-bit formats
# ---------------------------------------------------------------------------

def test_decode16_matches_numpy_and_torch_for_every_pattern():
    pats = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    f16 = pats.view(np.float16).astype(np.float64)
    o = oracle.decode16(pats, F16)
    fin = np.isfinite(f16)
    assert np.array_equal(o[fin], f16[fin])
    assert np.array_equal(np.isnan(o), np.isnan(f16))
    b16 = torch.from_numpy(pats.view(np.int16).copy()).view(torch.bfloat16).double().numpy()
    o = oracle.decode16(pats, BF16)
    fin = np.isfinite(b16)
    assert np.array_equal(o[fin], b16[fin])
    assert np.array_equal(np.isnan(o), np.isnan(b16))


def _neighbors_f16(x: float):
    """(largest f16 <= x, smallest f16 >= x) via numpy's RNE cast and nextafter."""
    n = np.float16(np.float32(x))
    lo = n if float(n) <= x else np.nextafter(n, np.float16(-np.inf))
    hi = n if float(n) >= x else np.nextafter(n, np.float16(np.inf))
    return float(lo), float(hi)


def _bf16_step(h: int, up: bool) -> int:
    """Adjacent bf16 pattern in value order (sign-magnitude stepping)."""
    neg = h & 0x8000
    mag = h & 0x7FFF
    if mag == 0:
        return 0x0001 if up else 0x8001
    if (not neg) == up:
        return h + 1
    return h - 1


def _neighbors_bf16(x: float):
    h = int(_bf16_bits(np.array([x], np.float32))[0])
    v = _val(h, BF16)
    lo = h if v <= x else _bf16_step(h, up=False)
    hi = h if v >= x else _bf16_step(h, up=True)
    return _val(lo, BF16), _val(hi, BF16)


@pytest.mark.parametrize("fmt", [F16, BF16])
def test_directed_rounding_brackets_value(fmt):
    rng = np.random.default_rng(11)
    xs = np.concatenate([rng.standard_normal(3000).astype(np.float32) * 0.05,
                         rng.standard_normal(500).astype(np.float32) * 1e-6,
                         rng.standard_normal(500).astype(np.float32) * 300,
                         np.array([0.0, 1.0, -1.0, 0.1, -0.1, 2 ** -14, 65504.0], np.float32)])
    if fmt == F16:
        xs = xs[np.abs(xs) < 60000]
    nb = _neighbors_f16 if fmt == F16 else _neighbors_bf16
    for x in xs.tolist():
        lo, hi = nb(x)
        assert _val(oracle.round_down16(x, fmt), fmt) == lo, x
        assert _val(oracle.round_up16(x, fmt), fmt) == hi, x


@pytest.mark.parametrize("fmt", [F16, BF16])
def test_zero_rounds_to_positive_zero(fmt):
    assert oracle.round_down16(0.0, fmt) == 0
    assert oracle.round_down16(-0.0, fmt) == 0
    assert oracle.round_up16(-0.0, fmt) == 0


@pytest.mark.parametrize("fmt", [F16, BF16])
def test_next_up_and_nearest(fmt):
    rng = np.random.default_rng(5)
    xs = rng.standard_normal(2000).astype(np.float32) * 0.1
    for x in xs.tolist():
        h = oracle.round_down16(x, fmt)
        up = oracle.next_up16(h, fmt)
        assert _val(up, fmt) > _val(h, fmt)
        if fmt == BF16:
            assert up == _bf16_step(h, up=True) or (h == 0 and up == 1)
        # nearest-even agrees with the library casts on fp32 inputs
        ref = int(np.float16(x).view(np.uint16)) if fmt == F16 else int(_bf16_bits(np.array([x], np.float32))[0])
        got = oracle.round_nearest16(x, fmt)
        assert _val(got, fmt) == _val(ref, fmt)


# ---------------------------------------------------------------------------
# quantizer
# ---------------------------------------------------------------------------

def _exact_check_group(v32: np.ndarray, bits: int, sdt: int, slack: bool = True):
    """P2-style bounds in exact rational arithmetic."""
    Q = (1 << bits) - 1
    c, sb, zb = oracle.quantize_group(v32, bits, sdt)
    s, z = _frac16(sb, sdt), _frac16(zb, sdt)
    vs = [Fraction(float(x)) for x in v32]
    lo, hi = min(vs), max(vs)
    assert z <= lo
    # z is the largest sdt value <= lo: the next one up is above lo
    assert _frac16(oracle.next_up16(zb, sdt), sdt) > lo or z == lo
    assert c.max() <= Q
    if s == 0:
        assert hi == z and np.all(c == 0)
        return c, s, z
    r = Fraction(float(np.float32(np.float32(hi) - np.float32(z))))
    assert s * Q >= r
    # s is the smallest sdt value whose Q multiple covers r
    prev = oracle.round_down16(float(np.nextafter(np.float32(float(s)), np.float32(0))), sdt)
    assert _frac16(prev, sdt) * Q < r
    for x, ci in zip(vs, c.tolist()):
        err = abs(x - (z + ci * s))
        bound = s / 2 + (Fraction(1, 2 ** 22) * (x - z) if slack else 0)
        assert err <= bound, (float(x), ci, float(s), float(z))
    assert z + Q * s >= hi - (Fraction(1, 2 ** 22) * (hi - z) if slack else 0)
    return c, s, z


@pytest.mark.parametrize("sdt", [F16, BF16])
@pytest.mark.parametrize("bits", [8, 4])
@pytest.mark.parametrize("G", [64, 128])
def test_quantize_error_bound_exact(sdt, bits, G):
    """P2: |v - (z + c s)| <= s/2 (plus fp32 rounding slack), z <= min, z + Q s >= max."""
    rng = np.random.default_rng(100 + bits + G + sdt)
    fmt = sdt
    for _ in range(40):
        v = rng.standard_normal(G).astype(np.float32) * np.float32(0.02)
        v = oracle.decode16(oracle_round_to(v, fmt), fmt).astype(np.float32)
        _exact_check_group(v, bits, sdt)


def oracle_round_to(v32, fmt):
    if fmt == F16:
        return v32.astype(np.float16).view(np.uint16)
    return _bf16_bits(v32)


@pytest.mark.parametrize("sdt", [F16, BF16])
@pytest.mark.parametrize("bits", [8, 4])
def test_quantize_error_bound_no_slack_on_exact_grid(sdt, bits):
    """On inputs where every fp32 step is exact the bound is exactly s/2."""
    rng = np.random.default_rng(7 + bits + sdt)
    for _ in range(60):
        # small-integer multiples of 2^-10: differences and quotients by a
        # power-of-two-times-small-odd scale stay exact or round harmlessly
        v = (rng.integers(-300, 300, size=32) * 2.0 ** -10).astype(np.float32)
        _exact_check_group(v, bits, sdt, slack=False)


@pytest.mark.parametrize("sdt", [F16, BF16])
@pytest.mark.parametrize("bits", [8, 4])
def test_quantize_brute_force_argmin(sdt, bits):
    """P3: for tiny groups each code is the nearest grid point (ties to even)."""
    Q = (1 << bits) - 1
    rng = np.random.default_rng(31 + bits + sdt)
    checked = 0
    for _ in range(300):
        G = int(rng.integers(2, 9))
        v = rng.standard_normal(G).astype(np.float32) * np.float32(0.05)
        v = oracle.decode16(oracle_round_to(v, sdt), sdt).astype(np.float32)
        c, sb, zb = oracle.quantize_group(v, bits, sdt)
        s, z = _frac16(sb, sdt), _frac16(zb, sdt)
        if s == 0:
            continue
        for x, ci in zip(v.tolist(), c.tolist()):
            t = (Fraction(x) - z) / s
            frac = t - int(t)
            if abs(frac - Fraction(1, 2)) < Fraction(1, 2 ** 18):
                continue          # a near-tie where one fp32 rounding may decide
            errs = [abs(Fraction(x) - (z + k * s)) for k in range(Q + 1)]
            best = min(errs)
            cands = [k for k in range(Q + 1) if errs[k] == best]
            want = cands[0] if len(cands) == 1 else [k for k in cands if k % 2 == 0][0]
            assert ci == want
            checked += 1
    assert checked > 500


@pytest.mark.parametrize("sdt", [F16, BF16])
@pytest.mark.parametrize("bits", [8, 4])
def test_quantize_arithmetic_progression(sdt, bits):
    """P4: v_j = z0 + j s0 (representable) quantizes to (j, s0, z0)."""
    Q = (1 << bits) - 1
    rng = np.random.default_rng(3 + bits)
    for _ in range(30):
        s0 = float(np.float32(2.0 ** int(rng.integers(-12, -5)) * (1 + int(rng.integers(0, 8)) / 8)))
        z0 = -float(rng.integers(1, 64)) * 2.0 ** -8
        if sdt == BF16:
            s0 = _val(oracle.round_down16(s0, BF16), BF16)
        v = np.array([z0 + j * s0 for j in range(Q + 1)], np.float32)
        assert all(Fraction(float(x)) == Fraction(z0) + j * Fraction(s0) for j, x in enumerate(v))
        perm = rng.permutation(Q + 1)
        c, sb, zb = oracle.quantize_group(v[perm], bits, sdt)
        assert _val(sb, sdt) == s0 and _val(zb, sdt) == z0
        assert np.array_equal(c, perm.astype(np.uint8))


@pytest.mark.parametrize("sdt", [F16, BF16])
def test_degenerate_group(sdt):
    """A constant group that the zero represents exactly: s = +0, codes 0."""
    v = np.full(64, 0.25, np.float32)
    c, sb, zb = oracle.quantize_group(v, 4, sdt)
    assert sb == 0 and _val(zb, sdt) == 0.25 and not c.any()
    # not representable in sdt -> a real step, all codes still reproduce within s/2
    v = np.full(64, np.float32(0.1), np.float32)
    _exact_check_group(v, 4, sdt)


@pytest.mark.parametrize("sdt,bits", [(F16, 8), (F16, 4), (BF16, 4)])
def test_requant_fixed_point(sdt, bits):
    """P5: Q_b(deq(Q_b(v))) == Q_b(v) when the first pass uses codes 0 and Q."""
    Q = (1 << bits) - 1
    rng = np.random.default_rng(17 + bits + sdt)
    n_fixed = 0
    for _ in range(200):
        v = rng.standard_normal(128).astype(np.float32) * np.float32(0.02)
        v = oracle.decode16(oracle_round_to(v, sdt), sdt).astype(np.float32)
        c, sb, zb = oracle.quantize_group(v, bits, sdt)
        if c.min() != 0 or c.max() != Q:
            continue
        d = oracle.dequant_values(c[None, :], np.array([[sb]], np.uint16),
                                  np.array([[zb]], np.uint16), 128, sdt)[0]
        # the precondition of the argument: the dequantized values are exact
        s, z = _frac16(sb, sdt), _frac16(zb, sdt)
        assert all(Fraction(float(x)) == z + int(ci) * s for x, ci in zip(d, c))
        c2, sb2, zb2 = oracle.quantize_group(d, bits, sdt)
        assert (sb2, zb2) == (sb, zb) and np.array_equal(c2, c)
        n_fixed += 1
    assert n_fixed > 100


def test_requant_value_level_bf16_int8():
    """bf16 scales with 8-bit codes: a second pass moves each value by at most s/2."""
    rng = np.random.default_rng(99)
    for _ in range(100):
        v = rng.standard_normal(128).astype(np.float32) * np.float32(0.02)
        v = oracle.decode16(_bf16_bits(v), BF16).astype(np.float32)
        c, sb, zb = oracle.quantize_group(v, 8, BF16)
        d1 = oracle.dequant_values(c[None], np.array([[sb]], np.uint16), np.array([[zb]], np.uint16), 128, BF16)[0]
        c2, sb2, zb2 = oracle.quantize_group(d1, 8, BF16)
        d2 = oracle.dequant_values(c2[None], np.array([[sb2]], np.uint16), np.array([[zb2]], np.uint16), 128, BF16)[0]
        s2 = _frac16(sb2, BF16)
        for a, b in zip(d1.tolist(), d2.tolist()):
            assert abs(Fraction(a) - Fraction(b)) <= s2 / 2 + Fraction(1, 2 ** 22) * abs(Fraction(a))


def test_dequant_formula():
    """O4: fl32(z + c s) for every code of a random group."""
    for sdt in (F16, BF16):
        c, sb, zb = oracle.quantize_group(np.linspace(-0.05, 0.07, 128, dtype=np.float32), 8, sdt)
        for ci in range(256):
            want = np.float32(np.float32(_val(zb, sdt)) + np.float32(ci) * np.float32(_val(sb, sdt)))
            assert oracle.lib().or_dequant(ci, sb, zb, sdt) == want


def test_page_quantize_is_groupwise():
    """A page quantizes each (row, group) independently along K."""
    rng = np.random.default_rng(1)
    w = oracle_round_to(rng.standard_normal((4, 256)).astype(np.float32) * 0.02, BF16)
    c, s, z = oracle.quantize_page16(w, BF16, 64, 4, BF16)
    v = oracle.decode16(w, BF16).astype(np.float32)
    for r in range(4):
        for g in range(4):
            cg, sg, zg = oracle.quantize_group(v[r, g * 64:(g + 1) * 64], 4, BF16)
            assert np.array_equal(c[r, g * 64:(g + 1) * 64], cg)
            assert (s[r, g], z[r, g]) == (sg, zg)


def test_requant_8_to_4_uses_dequantized_source():
    rng = np.random.default_rng(2)
    w = oracle_round_to(rng.standard_normal((2, 128)).astype(np.float32) * 0.02, BF16)
    c8, s8, z8 = oracle.quantize_page16(w, BF16, 128, 8, BF16)
    c4, s4, z4 = oracle.requant_page(c8, s8, z8, 128, BF16, 4)
    d = oracle.dequant_values(c8, s8, z8, 128, BF16)
    r4 = oracle.quantize_page_f32(d, 128, 4, BF16)
    assert all(np.array_equal(a, b) for a, b in zip((c4, s4, z4), r4))
