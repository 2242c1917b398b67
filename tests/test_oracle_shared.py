"""Pins of the shared-expert reading in the oracle (experts every token uses
beside the routed ones, Table 1 of the paper: 60 routed + 4 shared, 128
routed + 1 shared): the layer output is the routed mixture plus each shared
expert's FFN times a per-token gate.

- Qwen-style fused shared expert: four shared experts of width F under one
  gate equal one shared expert of width 4F whose gate/up rows and down
  columns are the four stacked (SwiGLU is separable over its hidden units),
  with mixed-bit pages too (groups along K never straddle the experts).
- Routed experts with W_up = 0 contribute exactly 0: the layer reduces to the
  gated shared FFNs, checked against a textbook float64 numpy FFN.
- A zero gate gives the routed-only layer bit for bit.
- The routing columns: routed top-K as the plain router, then E .. E+n-1.
"""
import numpy as np
import pytest

import oracle
from paper_2607_16184_amd import synth

F16 = oracle.F16


def _w16(rng, E, rows, cols, fmt=F16):
    return synth.to16(rng.standard_normal((E, rows, cols)).astype(np.float32) * np.float32(0.05), fmt)


def _layer(E, H, F, R, G, w16, bits):
    return oracle.OracleLayer(E, H, F, R, G, F16, F16, w16, bits)


def _ffn(x, wg, wu, wd):
    """Textbook SwiGLU FFN in float64: W_down (silu(W_gate x) * W_up x)."""
    g = x @ wg.T
    u = x @ wu.T
    return (g / (1.0 + np.exp(-g)) * u) @ wd.T


def test_route_shared_columns():
    rng = np.random.default_rng(1)
    T, E, K, n = 9, 6, 2, 3
    logits = rng.standard_normal((T, E)).astype(np.float32)
    gate = rng.uniform(0, 1, (T, n)).astype(np.float32)
    ids, w = oracle.route_shared(logits, K, n, gate)
    rid, rw = oracle.route(logits, K)
    assert ids.shape == (T, K + n) and np.array_equal(ids[:, :K], rid) and np.array_equal(w[:, :K], rw)
    assert np.array_equal(ids[:, K:], np.tile(np.arange(E, E + n), (T, 1)))
    assert np.array_equal(w[:, K:], gate.astype(np.float64))
    _, w1 = oracle.route_shared(logits, K, n)
    assert np.all(w1[:, K:] == 1.0)
    # the permutation over E + n experts gives each shared expert every token
    counts, off, ss, sp = oracle.permute(ids, E + n)
    assert np.all(counts[E:] == T)


@pytest.mark.parametrize("bits_mode", ["16", "mixed"])
def test_four_shared_experts_equal_one_fused_expert(bits_mode):
    rng = np.random.default_rng(2)
    T, H, F, R, G, n = 12, 128, 128, 64, 64, 4
    wg, wu, wd = _w16(rng, n, F, H), _w16(rng, n, F, H), _w16(rng, n, H, F)
    if bits_mode == "16":
        bg = bu = np.full((n, F // R), 16)
        bd = np.full((n, H // R), 16)
    else:
        bg = rng.choice([16, 8, 4], (n, F // R))
        bu = rng.choice([16, 8, 4], (n, F // R))
        bd = np.tile(rng.choice([16, 8, 4], (1, H // R)), (n, 1))   # one bitwidth per fused down row block
    sep = _layer(n, H, F, R, G, [wg, wu, wd], [bg, bu, bd])
    # the fused expert: gate/up rows stacked, down columns stacked
    fg = wg.reshape(1, n * F, H)
    fu = wu.reshape(1, n * F, H)
    fd = np.concatenate([wd[j] for j in range(n)], axis=1)[None]
    fus = _layer(1, H, n * F, R, G, [fg, fu, fd],
                 [bg.reshape(1, -1), bu.reshape(1, -1), bd[:1]])
    x16 = synth.to16(rng.standard_normal((T, H)).astype(np.float32), F16)
    gate = rng.uniform(0, 1, T).astype(np.float32)
    # one gate for the four shared experts (as the fused expert has one)
    ids_s = np.tile(np.arange(n, dtype=np.int32), (T, 1))
    w_s = np.tile(gate.astype(np.float64)[:, None], (1, n))
    ids_f = np.zeros((T, 1), np.int32)
    w_f = gate.astype(np.float64)[:, None]
    y_s = sep.forward(x16, ids_s, w_s)
    y_f = fus.forward(x16, ids_f, w_f)
    assert np.abs(y_s - y_f).max() <= 1e-12 * np.abs(y_f).max()


def test_zeroed_routed_experts_leave_the_shared_ffn():
    rng = np.random.default_rng(3)
    T, E, n, K, H, F, R, G = 7, 6, 2, 2, 128, 128, 64, 64
    Et = E + n
    wg, wu, wd = _w16(rng, Et, F, H), _w16(rng, Et, F, H), _w16(rng, Et, H, F)
    wu[:E] = 0                                  # routed experts: W_up = 0
    bits = [np.full((Et, F // R), 16), np.full((Et, F // R), 16), np.full((Et, H // R), 16)]
    L = _layer(Et, H, F, R, G, [wg, wu, wd], bits)
    logits = rng.standard_normal((T, E)).astype(np.float32)
    gate = rng.uniform(0, 1, (T, n)).astype(np.float32)
    ids, w = oracle.route_shared(logits, K, n, gate)
    x16 = synth.to16(rng.standard_normal((T, H)).astype(np.float32), F16)
    y = L.forward(x16, ids, w)
    x = oracle.decode16(x16, F16)
    dec = [oracle.decode16(a, F16) for a in (wg, wu, wd)]
    want = np.zeros((T, H))
    for j in range(n):
        want += gate[:, j].astype(np.float64)[:, None] * _ffn(x, dec[0][E + j], dec[1][E + j], dec[2][E + j])
    assert np.abs(y - want).max() <= 1e-12 * np.abs(want).max()


def test_zero_gate_gives_the_routed_layer():
    rng = np.random.default_rng(4)
    T, E, n, K, H, F, R, G = 10, 8, 1, 2, 128, 256, 64, 64
    Et = E + n
    w16 = [_w16(rng, Et, F, H), _w16(rng, Et, F, H), _w16(rng, Et, H, F)]
    bits = [rng.choice([16, 8, 4], (Et, F // R)), rng.choice([16, 8, 4], (Et, F // R)),
            rng.choice([16, 8, 4], (Et, H // R))]
    L = _layer(Et, H, F, R, G, w16, bits)
    logits = rng.standard_normal((T, E)).astype(np.float32)
    ids, w = oracle.route_shared(logits, K, n, np.zeros((T, n), np.float32))
    rid, rw = oracle.route(logits, K)
    x16 = synth.to16(rng.standard_normal((T, H)).astype(np.float32), F16)
    assert np.array_equal(L.forward(x16, ids, w), L.forward(x16, rid, rw))
