"""Pins of the page byte format and Eq. 3's released-memory accounting.

The encoder is checked against an independent forward (scatter) construction of
the same layout written here, against a hand-derived golden example, and the
page sizes against the closed forms of Eq. 3 (Sec. 3.1).
"""
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _scatter_encode(codes, s, z, G, bits):
    """Place each code directly at its byte/bit position (forward construction)."""
    R, K = codes.shape
    code_bytes = R * K if bits == 8 else R * K // 2
    out = np.zeros(code_bytes + 4 * R * (K // G), np.uint8)
    for r in range(R):
        for k in range(K):
            blk, within = divmod(k, 128)
            rho, q = divmod(within, 8)
            p = 4 * (rho % 4) + rho // 4            # run position of run rho
            if bits == 8:
                out[r * K + blk * 128 + 8 * p + q] = codes[r, k]
            else:
                t, hi = divmod(q, 2)
                bit = 4 * t + 16 * hi
                word = r * (K // 2) + blk * 64 + 4 * p
                out[word + bit // 8] |= (int(codes[r, k]) & 15) << (bit % 8)
    for r in range(R):
        for g in range(K // G):
            i = code_bytes + 4 * (g * R + r)
            out[i:i + 2] = np.array([s[r, g]], np.uint16).view(np.uint8)
            out[i + 2:i + 4] = np.array([z[r, g]], np.uint16).view(np.uint8)
    return out


@pytest.mark.parametrize("bits", [8, 4])
@pytest.mark.parametrize("R,K,G", [(2, 128, 64), (3, 256, 128), (1, 384, 128)])
def test_encoder_matches_scatter_construction(bits, R, K, G):
    rng = np.random.default_rng(R * K + bits)
    codes = rng.integers(0, 1 << bits, size=(R, K)).astype(np.uint8)
    s = rng.integers(0, 65536, size=(R, K // G)).astype(np.uint16)
    z = rng.integers(0, 65536, size=(R, K // G)).astype(np.uint16)
    enc = oracle.encode_page(codes, s, z, G, bits)
    assert np.array_equal(enc, _scatter_encode(codes, s, z, G, bits))
    c2, s2, z2 = oracle.decode_page(enc, R, K, G, bits)
    assert np.array_equal(c2, codes) and np.array_equal(s2, s) and np.array_equal(z2, z)


def _read_golden(name):
    vals = {}
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.split("#")[0].strip()
            if line:
                k, v = line.split("=")
                vals[k.strip()] = v.strip()
    return vals


def test_golden_int4_and_int8_layout():
    """Hand-derived bytes of a one-row page with codes (k + k div 8) mod 2^bits."""
    g = _read_golden("page_format_example.txt")
    K = 128
    k = np.arange(K)
    c4 = ((k + k // 8) % 16).astype(np.uint8)[None]
    c8 = ((k + k // 8) % 256).astype(np.uint8)[None]
    sz = np.zeros((1, 1), np.uint16)
    e4 = oracle.encode_page(c4, sz, sz, 128, 4)
    e8 = oracle.encode_page(c8, sz, sz, 128, 8)
    assert e4[0:4].tobytes().hex() == g["int4_word_p0"]
    assert e4[4:8].tobytes().hex() == g["int4_word_p1"]
    assert e8[0:8].tobytes().hex() == g["int8_run_p0"]
    assert e8[8:16].tobytes().hex() == g["int8_run_p1"]


def test_page_sizes_eq3_closed_form():
    """M^16 = 2RK, M^8 = RK + 4R K/G, M^4 = RK/2 + 4R K/G; Delta = M^b - M^b'."""
    R, G = 128, 128
    assert oracle.page_bytes(R, 4096, G, 16) == 1_048_576
    assert oracle.page_bytes(R, 4096, G, 4) == 278_528
    assert oracle.delta_bytes(R, 4096, G, 16, 4) == 770_048
    assert oracle.page_bytes(R, 14336, G, 16) == 3_670_016
    assert oracle.page_bytes(R, 14336, G, 4) == 974_848
    assert oracle.delta_bytes(R, 14336, G, 16, 4) == 2_695_168
    assert oracle.delta_bytes(R, 4096, G, 8, 4) == R * 4096 // 2
    # downshift workload: 112 + 112 gate/up pages and 32 down pages go 16 -> 4
    assert 224 * 770_048 + 32 * 2_695_168 == 258_736_128
    for b in (16, 8, 4):
        assert oracle.page_bytes(64, 512, 64, b) % 256 == 0


def test_encoded_size_matches_page_bytes():
    for bits in (8, 4):
        for (R, K, G) in [(64, 256, 64), (128, 4096, 128), (64, 1408, 128)]:
            c = np.zeros((R, K), np.uint8)
            s = np.zeros((R, K // G), np.uint16)
            assert oracle.encode_page(c, s, s, G, bits).size == oracle.page_bytes(R, K, G, bits)
