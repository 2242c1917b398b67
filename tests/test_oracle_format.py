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


def _lane_step(r, k):
    """(tile index pieces, lane, step, position in run) of value (r, k)."""
    tau, lc = divmod(r, 16)
    beta, within = divmod(k, 128)
    i, rest = divmod(within, 32)
    lg, q = divmod(rest, 8)
    return tau, beta, 16 * lg + lc, i, q


def _scatter_encode(codes, s, z, G, bits):
    """Place each code directly at its byte/bit position (forward construction)."""
    R, K = codes.shape
    nkb = K // 128
    code_bytes = R * K if bits == 8 else R * K // 2
    out = np.zeros(code_bytes + 4 * R * (K // G), np.uint8)
    for r in range(R):
        for k in range(K):
            tau, beta, l, i, q = _lane_step(r, k)
            tile = tau * nkb + beta
            if bits == 8:
                out[tile * 2048 + 1024 * (i // 2) + 16 * l + 8 * (i % 2) + q] = codes[r, k]
            else:
                t, hi = divmod(q, 2)
                bit = 4 * t + 16 * hi
                word = tile * 1024 + 16 * l + 4 * i
                out[word + bit // 8] |= (int(codes[r, k]) & 15) << (bit % 8)
    for r in range(R):
        for g in range(K // G):
            i = code_bytes + 4 * (g * R + r)
            out[i:i + 2] = np.array([s[r, g]], np.uint16).view(np.uint8)
            out[i + 2:i + 4] = np.array([z[r, g]], np.uint16).view(np.uint8)
    return out


def _scatter_encode16(w):
    R, K = w.shape
    nkb = K // 128
    out = np.zeros(2 * R * K, np.uint8)
    for r in range(R):
        for k in range(K):
            tau, beta, l, i, q = _lane_step(r, k)
            o = (tau * nkb + beta) * 4096 + 1024 * i + 16 * l + 2 * q
            out[o:o + 2] = np.array([w[r, k]], np.uint16).view(np.uint8)
    return out


@pytest.mark.parametrize("bits", [8, 4])
@pytest.mark.parametrize("R,K,G", [(16, 128, 64), (32, 256, 128), (48, 384, 128)])
def test_encoder_matches_scatter_construction(bits, R, K, G):
    rng = np.random.default_rng(R * K + bits)
    codes = rng.integers(0, 1 << bits, size=(R, K)).astype(np.uint8)
    s = rng.integers(0, 65536, size=(R, K // G)).astype(np.uint16)
    z = rng.integers(0, 65536, size=(R, K // G)).astype(np.uint16)
    enc = oracle.encode_page(codes, s, z, G, bits)
    assert np.array_equal(enc, _scatter_encode(codes, s, z, G, bits))
    c2, s2, z2 = oracle.decode_page(enc, R, K, G, bits)
    assert np.array_equal(c2, codes) and np.array_equal(s2, s) and np.array_equal(z2, z)


@pytest.mark.parametrize("R,K", [(16, 128), (32, 384)])
def test_encoder16_matches_scatter_construction(R, K):
    w = np.random.default_rng(R + K).integers(0, 65536, size=(R, K)).astype(np.uint16)
    enc = oracle.encode_page16(w)
    assert np.array_equal(enc, _scatter_encode16(w))
    assert np.array_equal(oracle.decode_page16(enc, R, K), w)


def _read_golden(name):
    vals = {}
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.split("#")[0].strip()
            if line:
                k, v = line.split("=")
                vals[k.strip()] = v.strip()
    return vals


def test_golden_tiled_layout():
    """Hand-derived bytes of a one-tile page (16 rows x 128 values)."""
    g = _read_golden("page_format_example.txt")
    r = np.arange(16)[:, None]
    k = np.arange(128)[None, :]
    sz = np.zeros((16, 1), np.uint16)
    e4 = oracle.encode_page(((r + k) % 16).astype(np.uint8), sz, sz, 128, 4)
    e8 = oracle.encode_page(((r + k) % 256).astype(np.uint8), sz, sz, 128, 8)
    e16 = oracle.encode_page16((r * 256 + k).astype(np.uint16))
    assert e4[0:4].tobytes().hex() == g["int4_lane0_step0"]
    assert e4[16:20].tobytes().hex() == g["int4_lane1_step0"]
    assert e4[260:264].tobytes().hex() == g["int4_lane16_step1"]
    assert e8[24:32].tobytes().hex() == g["int8_lane1_step1"]
    assert e8[1296:1304].tobytes().hex() == g["int8_lane17_step2"]
    assert e16[3104:3120].tobytes().hex() == g["v16_lane2_step3"]


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
    assert oracle.encode_page16(np.zeros((16, 128), np.uint16)).size == oracle.page_bytes(16, 128, 128, 16)


def test_encoded_size_matches_page_bytes():
    for bits in (8, 4):
        for (R, K, G) in [(64, 256, 64), (128, 4096, 128), (64, 1408, 128)]:
            c = np.zeros((R, K), np.uint8)
            s = np.zeros((R, K // G), np.uint16)
            assert oracle.encode_page(c, s, s, G, bits).size == oracle.page_bytes(R, K, G, bits)
