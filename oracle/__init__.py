"""CPU oracle for the paged mixed-bit MoE hot path (test infrastructure only).

Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
import this package. It wraps ``pw_oracle.c`` (plain C, built with gcc) via
ctypes and never touches the HIP library. See ``pw_oracle.c`` for what each
function computes and which passage of the paper defines it.

Precision: quantizer decisions in fp32 as the format defines them; routing
weights, SwiGLU and the expert matmuls in fp64.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import List, Optional, Sequence, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "pw_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

GATE, UP, DOWN = 0, 1, 2
F16, BF16 = 0, 1

_c_u8p = np.ctypeslib.ndpointer(dtype=np.uint8, flags="C_CONTIGUOUS")
_c_u16p = np.ctypeslib.ndpointer(dtype=np.uint16, flags="C_CONTIGUOUS")
_c_i32p = np.ctypeslib.ndpointer(dtype=np.int32, flags="C_CONTIGUOUS")
_c_f32p = np.ctypeslib.ndpointer(dtype=np.float32, flags="C_CONTIGUOUS")
_c_f64p = np.ctypeslib.ndpointer(dtype=np.float64, flags="C_CONTIGUOUS")


def build(force: bool = False) -> str:
    """Compile the oracle shared library with gcc (idempotent unless forced)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp",
                               "-ffp-contract=off", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib():
    global _lib
    if _lib is not None:
        return _lib
    build()
    L = ctypes.CDLL(_LIB)
    L.or_init.argtypes = []
    L.or_decode16.argtypes = [ctypes.c_uint16, ctypes.c_int]
    L.or_decode16.restype = ctypes.c_double
    L.or_round_down16.argtypes = [ctypes.c_float, ctypes.c_int]
    L.or_round_down16.restype = ctypes.c_uint16
    L.or_round_up16.argtypes = [ctypes.c_float, ctypes.c_int]
    L.or_round_up16.restype = ctypes.c_uint16
    L.or_next_up16.argtypes = [ctypes.c_uint16, ctypes.c_int]
    L.or_next_up16.restype = ctypes.c_uint16
    L.or_round_nearest16.argtypes = [ctypes.c_double, ctypes.c_int]
    L.or_round_nearest16.restype = ctypes.c_uint16
    L.or_quantize_group.argtypes = [_c_f32p, ctypes.c_int, ctypes.c_int, ctypes.c_int, _c_u8p,
                                    ctypes.POINTER(ctypes.c_uint16), ctypes.POINTER(ctypes.c_uint16)]
    L.or_dequant.argtypes = [ctypes.c_uint8, ctypes.c_uint16, ctypes.c_uint16, ctypes.c_int]
    L.or_dequant.restype = ctypes.c_float
    L.or_quantize_page_f32.argtypes = [_c_f32p] + [ctypes.c_int] * 5 + [_c_u8p, _c_u16p, _c_u16p]
    L.or_quantize_page16.argtypes = [_c_u16p] + [ctypes.c_int] * 6 + [_c_u8p, _c_u16p, _c_u16p]
    L.or_requant_page.argtypes = [_c_u8p, _c_u16p, _c_u16p] + [ctypes.c_int] * 5 + \
        [_c_u8p, _c_u16p, _c_u16p]
    L.or_page_bytes.argtypes = [ctypes.c_int] * 4
    L.or_page_bytes.restype = ctypes.c_uint64
    L.or_delta_bytes.argtypes = [ctypes.c_int] * 5
    L.or_delta_bytes.restype = ctypes.c_uint64
    L.or_encode_page.argtypes = [_c_u8p, _c_u16p, _c_u16p] + [ctypes.c_int] * 4 + [_c_u8p]
    L.or_decode_page.argtypes = [_c_u8p] + [ctypes.c_int] * 4 + [_c_u8p, _c_u16p, _c_u16p]
    L.or_encode_page16.argtypes = [_c_u16p, ctypes.c_int, ctypes.c_int, _c_u8p]
    L.or_decode_page16.argtypes = [_c_u8p, ctypes.c_int, ctypes.c_int, _c_u16p]
    L.or_route.argtypes = [_c_f32p] + [ctypes.c_int] * 4 + [_c_i32p, _c_f64p]
    L.or_permute.argtypes = [_c_i32p] + [ctypes.c_int] * 3 + [_c_i32p] * 4
    L.or_routing_mass.argtypes = [_c_i32p, _c_f64p] + [ctypes.c_int] * 3 + [_c_f64p]
    L.or_moe_forward.argtypes = (
        [_c_u16p] + [ctypes.c_int] * 9 + [_c_i32p, _c_f64p]
        + [_c_u16p, _c_i32p, _c_u8p, _c_u16p, _c_u16p] * 3
        + [ctypes.c_int, ctypes.c_int, _c_i32p, ctypes.c_int, _c_f64p])
    L.or_threads.restype = ctypes.c_int
    L.or_set_threads.argtypes = [ctypes.c_int]
    L.or_init()
    _lib = L
    return L


# ---------------------------------------------------------------------------
# scalar helpers
# ---------------------------------------------------------------------------

_dec_tables = {}


def decode16(bits, fmt: int) -> np.ndarray:
    """Exact values of 16-bit patterns, as float64."""
    if fmt not in _dec_tables:
        L = lib()
        _dec_tables[fmt] = np.array([L.or_decode16(h, fmt) for h in range(65536)], np.float64)
    flat = np.asarray(bits, dtype=np.uint16).ravel()
    return _dec_tables[fmt][flat].reshape(np.shape(bits))


def round_down16(x: float, fmt: int) -> int:
    return int(lib().or_round_down16(float(x), fmt))


def round_up16(x: float, fmt: int) -> int:
    return int(lib().or_round_up16(float(x), fmt))


def next_up16(h: int, fmt: int) -> int:
    return int(lib().or_next_up16(int(h), fmt))


def round_nearest16(x: float, fmt: int) -> int:
    return int(lib().or_round_nearest16(float(x), fmt))


# ---------------------------------------------------------------------------
# quantizer
# ---------------------------------------------------------------------------

def quantize_group(v: np.ndarray, bits: int, sdt: int) -> Tuple[np.ndarray, int, int]:
    """Quantize one group of fp32 values. Returns (codes uint8, s bits, z bits)."""
    v = np.ascontiguousarray(v, dtype=np.float32)
    c = np.zeros(v.size, dtype=np.uint8)
    s = ctypes.c_uint16()
    z = ctypes.c_uint16()
    lib().or_quantize_group(v, v.size, bits, sdt, c, ctypes.byref(s), ctypes.byref(z))
    return c, int(s.value), int(z.value)


def dequant_values(codes: np.ndarray, s: np.ndarray, z: np.ndarray, G: int, sdt: int) -> np.ndarray:
    """fl32(z + c*s) for a [R][K] page with scale/zero [R][K/G] (fp32 result)."""
    sv = decode16(s, sdt).astype(np.float32)
    zv = decode16(z, sdt).astype(np.float32)
    sk = np.repeat(sv, G, axis=1)
    zk = np.repeat(zv, G, axis=1)
    prod = codes.astype(np.float32) * sk          # exact
    return (zk + prod).astype(np.float32)


def quantize_page16(w16: np.ndarray, fmt16: int, G: int, bits: int, sdt: int):
    """Quantize a [R][K] page of 16-bit values. Returns (codes, s, z)."""
    w16 = np.ascontiguousarray(w16, dtype=np.uint16)
    R, K = w16.shape
    c = np.zeros((R, K), np.uint8)
    s = np.zeros((R, K // G), np.uint16)
    z = np.zeros((R, K // G), np.uint16)
    lib().or_quantize_page16(w16, fmt16, R, K, G, bits, sdt, c, s, z)
    return c, s, z


def quantize_page_f32(v: np.ndarray, G: int, bits: int, sdt: int):
    v = np.ascontiguousarray(v, dtype=np.float32)
    R, K = v.shape
    c = np.zeros((R, K), np.uint8)
    s = np.zeros((R, K // G), np.uint16)
    z = np.zeros((R, K // G), np.uint16)
    lib().or_quantize_page_f32(v, R, K, G, bits, sdt, c, s, z)
    return c, s, z


def requant_page(codes, s, z, G: int, sdt: int, bits_out: int):
    """Requantize a quantized page to a lower bitwidth from its dequantized values."""
    codes = np.ascontiguousarray(codes, np.uint8)
    R, K = codes.shape
    c2 = np.zeros((R, K), np.uint8)
    s2 = np.zeros((R, K // G), np.uint16)
    z2 = np.zeros((R, K // G), np.uint16)
    lib().or_requant_page(codes, np.ascontiguousarray(s, np.uint16), np.ascontiguousarray(z, np.uint16),
                          R, K, G, sdt, bits_out, c2, s2, z2)
    return c2, s2, z2


# ---------------------------------------------------------------------------
# page byte format
# ---------------------------------------------------------------------------

def page_bytes(R: int, K: int, G: int, bits: int) -> int:
    return int(lib().or_page_bytes(R, K, G, bits))


def delta_bytes(R: int, K: int, G: int, b: int, bp: int) -> int:
    """Eq. 3: bytes released when a block goes from b to b' bits."""
    return int(lib().or_delta_bytes(R, K, G, b, bp))


def encode_page(codes, s, z, G: int, bits: int) -> np.ndarray:
    codes = np.ascontiguousarray(codes, np.uint8)
    R, K = codes.shape
    out = np.zeros(page_bytes(R, K, G, bits), np.uint8)
    lib().or_encode_page(codes, np.ascontiguousarray(s, np.uint16), np.ascontiguousarray(z, np.uint16),
                         R, K, G, bits, out)
    return out


def encode_page16(w16) -> np.ndarray:
    """Bytes of a 16-bit page ([R][K] values) in the tiled pool layout."""
    w16 = np.ascontiguousarray(w16, np.uint16)
    R, K = w16.shape
    out = np.zeros(2 * R * K, np.uint8)
    lib().or_encode_page16(w16, R, K, out)
    return out


def decode_page16(buf: np.ndarray, R: int, K: int) -> np.ndarray:
    buf = np.ascontiguousarray(buf, np.uint8)
    assert buf.size >= 2 * R * K
    w = np.zeros((R, K), np.uint16)
    lib().or_decode_page16(buf, R, K, w)
    return w


def decode_page(buf: np.ndarray, R: int, K: int, G: int, bits: int):
    buf = np.ascontiguousarray(buf, np.uint8)
    assert buf.size >= page_bytes(R, K, G, bits)
    c = np.zeros((R, K), np.uint8)
    s = np.zeros((R, K // G), np.uint16)
    z = np.zeros((R, K // G), np.uint16)
    lib().or_decode_page(buf, R, K, G, bits, c, s, z)
    return c, s, z


# ---------------------------------------------------------------------------
# routing
# ---------------------------------------------------------------------------

def route(logits: np.ndarray, K: int, renorm: int = 1) -> Tuple[np.ndarray, np.ndarray]:
    """Top-K expert ids [T,K] int32 and routing weights [T,K] float64."""
    logits = np.ascontiguousarray(logits, np.float32)
    T, E = logits.shape
    ids = np.zeros((T, K), np.int32)
    w = np.zeros((T, K), np.float64)
    lib().or_route(logits, T, E, K, renorm, ids, w)
    return ids, w


def route_shared(logits: np.ndarray, K: int, n_shared: int, gate: Optional[np.ndarray] = None,
                 renorm: int = 1) -> Tuple[np.ndarray, np.ndarray]:
    """Routing of a layer whose last n_shared experts are shared experts
    (Table 1 of the paper: MoE layers with experts every token uses beside
    the routed ones). logits [T, E] covers the routed experts only; each
    token gets its routed top-K (as route()) followed by the shared experts
    E .. E + n_shared - 1 with weight gate[t, j] (1 without a gate). The
    layer output is then the plain weighted sum over all K + n_shared
    columns: the routed mixture plus each shared expert's FFN times its gate
    (the reading taken here; the paper does not spell the combination out).
    Returns ids [T, K + n_shared] int32 and weights float64."""
    ids, w = route(logits, K, renorm)
    T, E = np.shape(logits)
    sid = np.tile(np.arange(E, E + n_shared, dtype=np.int32), (T, 1))
    if gate is None:
        sw = np.ones((T, n_shared), np.float64)
    else:
        sw = np.asarray(gate, np.float32).astype(np.float64).reshape(T, n_shared)
    return (np.ascontiguousarray(np.concatenate([ids, sid], axis=1), np.int32),
            np.ascontiguousarray(np.concatenate([w, sw], axis=1)))


def permute(ids: np.ndarray, E: int):
    """(counts[E], offsets[E+1], sorted_slot[S], slot_pos[S]) for slot s = t*K + k."""
    ids = np.ascontiguousarray(ids, np.int32)
    T, K = ids.shape
    S = T * K
    counts = np.zeros(E, np.int32)
    offsets = np.zeros(E + 1, np.int32)
    ss = np.zeros(S, np.int32)
    sp = np.zeros(S, np.int32)
    lib().or_permute(ids, T, K, E, counts, offsets, ss, sp)
    return counts, offsets, ss, sp


def threads() -> int:
    """OpenMP threads the oracle's parallel loops use."""
    return int(lib().or_threads())


def set_threads(n: int) -> None:
    """Threads for the oracle's later parallel loops (for timing the oracle)."""
    lib().or_set_threads(int(n))


def routing_mass(ids: np.ndarray, w: np.ndarray, E: int) -> np.ndarray:
    """Eq. 1: each expert's share of the total routing weight."""
    ids = np.ascontiguousarray(ids, np.int32)
    T, K = ids.shape
    m = np.zeros(E, np.float64)
    lib().or_routing_mass(ids, np.ascontiguousarray(w, np.float64), T, K, E, m)
    return m


# ---------------------------------------------------------------------------
# a layer: every page at its committed bitwidth
# ---------------------------------------------------------------------------

class OracleLayer:
    """The oracle's own copy of a paged layer.

    ``w16[p]`` holds the 16-bit source weights of projection p ([E,F,H] for
    gate/up, [E,H,F] for down); ``bits[p]`` the committed bitwidth per page
    [E, nrb]. Quantized pages are quantized here, by the oracle, from w16.
    """

    def __init__(self, E, H, F, R, G, act, sdt, w16: Sequence[np.ndarray], bits: Sequence[np.ndarray]):
        self.E, self.H, self.F, self.R, self.G, self.act, self.sdt = E, H, F, R, G, act, sdt
        self.w16 = [np.ascontiguousarray(w, np.uint16) for w in w16]
        self.bits = [np.ascontiguousarray(b, np.int32).copy() for b in bits]
        self.codes, self.s, self.z = [], [], []
        for p in range(3):
            rows, cols = self.w16[p].shape[1:]
            self.codes.append(np.zeros((E, rows, cols), np.uint8))
            self.s.append(np.zeros((E, rows, cols // G), np.uint16))
            self.z.append(np.zeros((E, rows, cols // G), np.uint16))
            for e in range(E):
                for rb in range(rows // R):
                    b = int(self.bits[p][e, rb])
                    if b != 16:
                        self._set_page(p, e, rb, *quantize_page16(self._rows16(p, e, rb), act, G, b, sdt))

    def _rows16(self, p, e, rb):
        return self.w16[p][e, rb * self.R:(rb + 1) * self.R]

    def _set_page(self, p, e, rb, c, s, z):
        sl = slice(rb * self.R, (rb + 1) * self.R)
        self.codes[p][e, sl] = c
        self.s[p][e, sl] = s
        self.z[p][e, sl] = z

    def page(self, p, e, rb):
        """(bits, codes, s, z) of a quantized page, or (16, w16 rows, None, None)."""
        sl = slice(rb * self.R, (rb + 1) * self.R)
        b = int(self.bits[p][e, rb])
        if b == 16:
            return 16, self.w16[p][e, sl], None, None
        return b, self.codes[p][e, sl], self.s[p][e, sl], self.z[p][e, sl]

    def page_image(self, p, e, rb) -> np.ndarray:
        """The page's bytes in the pool format."""
        b, c, s, z = self.page(p, e, rb)
        if b == 16:
            return encode_page16(c)
        return encode_page(c, s, z, self.G, b)

    def requant(self, p, e, rb, new_bits) -> int:
        """Lower page (p, e, rb) to new_bits; returns Eq. 3's released bytes."""
        b = int(self.bits[p][e, rb])
        if new_bits == b:
            return 0
        if new_bits > b:
            raise ValueError("raising a bitwidth needs a reload")
        if b == 16:
            q = quantize_page16(self._rows16(p, e, rb), self.act, self.G, new_bits, self.sdt)
        else:
            _, c, s, z = self.page(p, e, rb)
            q = requant_page(c, s, z, self.G, self.sdt, new_bits)
        self._set_page(p, e, rb, *q)
        self.bits[p][e, rb] = new_bits
        K = self.w16[p].shape[2]
        return delta_bytes(self.R, K, self.G, b, new_bits)

    def forward(self, x16: np.ndarray, ids: np.ndarray, w: np.ndarray, h_round: bool = False,
                tokens: Optional[Sequence[int]] = None, w_round: bool = False) -> np.ndarray:
        """y [T,H] float64 for the listed tokens (all by default); other rows 0.

        h_round: round the SwiGLU output to the activation format before the
        down projection. w_round: read a quantized weight as its fp32 value
        z + c*s rounded to the activation format (16-bit pages unchanged)."""
        x16 = np.ascontiguousarray(x16, np.uint16)
        T = x16.shape[0]
        K = ids.shape[1]
        tok = np.arange(T, dtype=np.int32) if tokens is None else np.asarray(tokens, np.int32)
        y = np.zeros((T, self.H), np.float64)
        args = []
        for p in range(3):
            args += [self.w16[p], self.bits[p], self.codes[p], self.s[p], self.z[p]]
        lib().or_moe_forward(x16, T, self.H, self.F, self.E, K, self.R, self.G, self.act, self.sdt,
                             np.ascontiguousarray(ids, np.int32), np.ascontiguousarray(w, np.float64),
                             *args, int(h_round), int(w_round), np.ascontiguousarray(tok), int(tok.size), y)
        return y

    def active_weight_bytes(self, counts: np.ndarray) -> int:
        """Bytes of every page (data plus scale/zero) of experts with routed slots."""
        tot = 0
        for p in range(3):
            K = self.w16[p].shape[2]
            for e in range(self.E):
                if counts[e] == 0:
                    continue
                for b in self.bits[p][e]:
                    tot += page_bytes(self.R, K, self.G, int(b))
        return tot
