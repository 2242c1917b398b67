"""Oracle of the nested bit-plane page format (test infrastructure only).

Sec. 2-3 of the paper build on any-precision weights: a linear-block holds
non-uniform codes whose top b bits form its b-bit code, stored as bit-planes,
with one lookup table (LUT) of reconstruction values per row and precision;
lowering a block's bitwidth drops its lowest bit-planes (no requantization),
and only the LUT of the committed precision is read. The paper leaves the
quantizer to the cited any-precision method; the deterministic reading used
here (also in the design notes):

* codes have 8 bits; supported precisions are 8 and 4 (planes 0-3 give the
  4-bit code, planes 0-7 the 8-bit code; plane 0 is the most significant);
* 4-bit seed, per row: 16 centroids initialised at lo + (hi - lo)(2j+1)/32
  (lo, hi the row's minimum and maximum), then 8 Lloyd iterations (assign
  each value to the nearest centroid, ties to the lower index; replace each
  centroid with the mean of its members, summed in order of k; an empty
  cluster keeps its centroid), then a final assignment;
* upscaling one bit at a time (levels 5..8): every parent cluster p with
  members (its values under the current assignment) gets two children
  initialised at (lo_p + m_p)/2 and (m_p + hi_p)/2 (m_p the members' mean),
  4 Lloyd iterations among the members, then a final assignment; code
  2p + child. A parent without members passes its centroid to both children;
* LUT_b[r][c] = the level-b centroid rounded to the activation dtype (nearest
  even); a weight at precision b reconstructs as LUT_b[r][code >> (8 - b)].

All arithmetic is float64 with sums accumulated from +0.0 in order of k, so
any implementation that keeps that order reproduces it bit for bit. Only the test suite, the smoke check and the benchmark's CPU leg may
import this module; it shares no code with the library.

Page layout of an R x K block (R a multiple of 16, K of 128), byte offsets:
  planes 0-3 at 0 (plane j at j RK/8), LUT_4 at RK/2 (R x 16 entries,
  row-major), planes 4-7 after it, LUT_8 after them (R x 256 entries).
Inside a plane, the 16-row x 128-value tile t = rt (K/128) + kb occupies
256 bytes at 256 t: lane l (0..63) owns the 32-bit word at 4 l, whose bit
8 i + q holds code bit (7 - j) of row 16 rt + l mod 16, column
128 kb + 32 i + 8 (l div 16) + q (i < 4, q < 8) -- the order in which a
64-lane wave feeds 16 x 32 matrix-core fragments.
"""
from __future__ import annotations

from typing import Tuple

import numpy as np

SEED_BITS = 4
MAX_BITS = 8
SEED_ITERS = 8
SPLIT_ITERS = 4


def _assign(v: np.ndarray, c: np.ndarray) -> np.ndarray:
    """Nearest centroid per value (ties to the lower index); v [R,K], c [R,J]."""
    d = np.abs(v[:, :, None] - c[:, None, :])
    return np.argmin(d, axis=2)


def _cluster_sums(v: np.ndarray, a: np.ndarray, J: int) -> Tuple[np.ndarray, np.ndarray]:
    """Per row and cluster: member count and the members' sum, accumulated from
    +0.0 one value at a time in order of k (np.add.at is unbuffered and adds
    in index order)."""
    R, K = v.shape
    rows = np.repeat(np.arange(R), K)
    s = np.zeros((R, J))
    np.add.at(s, (rows, a.reshape(-1)), v.reshape(-1))
    n = np.zeros((R, J), np.int64)
    np.add.at(n, (rows, a.reshape(-1)), 1)
    return n, s


def _update(c: np.ndarray, n: np.ndarray, s: np.ndarray) -> np.ndarray:
    """Lloyd update: each non-empty cluster's centroid becomes its mean."""
    c = c.copy()
    nz = n > 0
    c[nz] = s[nz] / n[nz]
    return c


def split_level(v: np.ndarray, a: np.ndarray, c: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """One bit of upscaling. v [R,K] values, a [R,K] their parent cluster
    (0 .. P-1), c [R,P] the parent centroids. Every parent p with members gets
    two children initialised at (lo_p + m_p)/2 and (m_p + hi_p)/2 (lo_p, hi_p,
    m_p the members' minimum, maximum and mean); SPLIT_ITERS Lloyd iterations
    move each member between its parent's two children (child 1 only when it
    is strictly nearer); a final assignment gives the code 2p + child. A
    parent without members passes its centroid to both children. Returns
    (codes [R,K], child centroids [R,2P])."""
    R, K = v.shape
    P = c.shape[1]
    r = np.arange(R)[:, None]
    # parent statistics: members' count, sum (in order of k), minimum, maximum
    n, s = _cluster_sums(v, a, P)
    pmin = np.full((R, P), np.inf)
    pmax = np.full((R, P), -np.inf)
    rows = np.repeat(np.arange(R), K)
    np.minimum.at(pmin, (rows, a.reshape(-1)), v.reshape(-1))
    np.maximum.at(pmax, (rows, a.reshape(-1)), v.reshape(-1))
    has = n > 0
    mean = np.where(has, s / np.maximum(n, 1), c)
    ch = np.empty((R, 2 * P))
    ch[:, 0::2] = np.where(has, (pmin + mean) / 2.0, c)
    ch[:, 1::2] = np.where(has, (mean + pmax) / 2.0, c)
    for _ in range(SPLIT_ITERS):
        pick = (np.abs(v - ch[r, 2 * a + 1]) < np.abs(v - ch[r, 2 * a])).astype(np.int64)
        ch = _update(ch, *_cluster_sums(v, 2 * a + pick, 2 * P))
    pick = (np.abs(v - ch[r, 2 * a + 1]) < np.abs(v - ch[r, 2 * a])).astype(np.int64)
    return 2 * a + pick, ch


def quantize_rows(v: np.ndarray) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """(8-bit codes [R,K] uint8, level-4 centroids [R,16], level-8 centroids
    [R,256]) of rows v (float64, the 16-bit weights' values)."""
    v = np.asarray(v, np.float64)
    lo, hi = v.min(axis=1), v.max(axis=1)
    c = lo[:, None] + (hi - lo)[:, None] * ((2.0 * np.arange(16) + 1.0) / 32.0)[None, :]
    for _ in range(SEED_ITERS):
        a = _assign(v, c)
        c = _update(c, *_cluster_sums(v, a, 16))
    a = _assign(v, c)
    c4 = c.copy()
    for _level in range(SEED_BITS + 1, MAX_BITS + 1):
        a, c = split_level(v, a, c)
    return a.astype(np.uint8), c4, c


def lut16(c: np.ndarray, fmt: int) -> np.ndarray:
    """Centroids rounded to the 16-bit activation dtype (nearest even), as bit patterns."""
    from oracle import round_nearest16
    flat = np.asarray(c, np.float64).reshape(-1)
    return np.array([round_nearest16(float(x), fmt) for x in flat], np.uint16).reshape(np.shape(c))


def page_bytes(R: int, K: int, bits: int) -> int:
    """Eq. 3's M^b of a nested bit-plane block: b planes and the LUTs up to b."""
    rk8 = R * K // 8
    if bits == 4:
        return 4 * rk8 + 32 * R
    if bits == 8:
        return 8 * rk8 + 32 * R + 512 * R
    raise ValueError("bits must be 8 or 4")


def lut4_offset(R: int, K: int) -> int:
    return 4 * (R * K // 8)


def encode_page(codes: np.ndarray, lut4: np.ndarray, lut8: np.ndarray) -> np.ndarray:
    """The 8-bit page bytes (layout in the module docstring)."""
    R, K = codes.shape
    rk8 = R * K // 8
    out = np.zeros(page_bytes(R, K, 8), np.uint8)
    nkb = K // 128
    for j in range(8):
        base = j * rk8 if j < 4 else 4 * rk8 + 32 * R + (j - 4) * rk8
        bit = ((codes >> (7 - j)) & 1).astype(np.uint32)
        words = np.zeros((R // 16, nkb, 64), np.uint32)
        for l in range(64):
            r = np.arange(R // 16) * 16 + (l % 16)
            for i in range(4):
                for q in range(8):
                    k = np.arange(nkb) * 128 + 32 * i + 8 * (l // 16) + q
                    words[:, :, l] |= bit[r][:, k] << np.uint32(8 * i + q)
        out[base:base + rk8] = words.reshape(-1).view(np.uint8)
    off4 = 4 * rk8
    out[off4:off4 + 32 * R] = np.ascontiguousarray(lut4, np.uint16).reshape(-1).view(np.uint8)
    off8 = 8 * rk8 + 32 * R
    out[off8:off8 + 512 * R] = np.ascontiguousarray(lut8, np.uint16).reshape(-1).view(np.uint8)
    return out


def decode_page(buf: np.ndarray, R: int, K: int, bits: int) -> Tuple[np.ndarray, np.ndarray]:
    """(codes at the given precision [R,K], that precision's LUT [R, 2^bits]) from page bytes."""
    rk8 = R * K // 8
    nkb = K // 128
    codes = np.zeros((R, K), np.uint32)
    for j in range(bits):
        base = j * rk8 if j < 4 else 4 * rk8 + 32 * R + (j - 4) * rk8
        words = np.frombuffer(buf[base:base + rk8].tobytes(), np.uint32).reshape(R // 16, nkb, 64)
        for l in range(64):
            r = np.arange(R // 16) * 16 + (l % 16)
            for i in range(4):
                for q in range(8):
                    k = np.arange(nkb) * 128 + 32 * i + 8 * (l // 16) + q
                    b = (words[:, :, l] >> np.uint32(8 * i + q)) & 1
                    codes[np.ix_(r, k)] |= b << np.uint32(bits - 1 - j)
    if bits == 4:
        lut = np.frombuffer(buf[4 * rk8:4 * rk8 + 32 * R].tobytes(), np.uint16).reshape(R, 16)
    else:
        off8 = 8 * rk8 + 32 * R
        lut = np.frombuffer(buf[off8:off8 + 512 * R].tobytes(), np.uint16).reshape(R, 256)
    return codes.astype(np.uint8), lut


def dequant(codes8: np.ndarray, lut: np.ndarray, bits: int) -> np.ndarray:
    """16-bit reconstruction (bit patterns) at precision bits: LUT_b[r][code >> (8 - b)]."""
    idx = (codes8.astype(np.int64) >> (8 - bits))
    return np.take_along_axis(np.asarray(lut), idx, axis=1).astype(np.uint16)
