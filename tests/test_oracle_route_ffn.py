"""Pins of the oracle's router, token permutation and paged expert forward.

Router (Sec. 2.1): top-K of E logits, ties to the lower index, weights
renormalised over the selected K. Routing mass: Eq. 1. Expert forward and
output accumulation (Sec. 3.3): checked against a textbook dense MoE in numpy
float64, special cases with closed forms, and the permutation against numpy's
stable sort.
"""
import numpy as np
import pytest
import scipy.special

import oracle
from paper_2607_16184_amd import synth

F16, BF16 = oracle.F16, oracle.BF16


# ---------------------------------------------------------------------------
# router
# ---------------------------------------------------------------------------

def test_route_matches_brute_force_sort():
    rng = np.random.default_rng(0)
    for E, K in [(8, 2), (64, 6), (5, 5), (16, 1)]:
        lg = rng.standard_normal((200, E)).astype(np.float32)
        lg[:20, :3] = 0.5                          # force ties
        ids, w = oracle.route(lg, K)
        for t in range(lg.shape[0]):
            order = sorted(range(E), key=lambda e: (-float(lg[t, e]), e))[:K]
            assert ids[t].tolist() == order
            a = np.exp(lg[t, order].astype(np.float64) - lg[t, order[0]])
            np.testing.assert_allclose(w[t], a / a.sum(), rtol=1e-15)


def test_route_full_topk_is_softmax():
    """K = E: the renormalised weights are the full softmax."""
    rng = np.random.default_rng(1)
    lg = rng.standard_normal((50, 8)).astype(np.float32)
    ids, w = oracle.route(lg, 8)
    sm = scipy.special.softmax(lg.astype(np.float64), axis=1)
    np.testing.assert_allclose(w, np.take_along_axis(sm, ids.astype(np.int64), 1), rtol=1e-14)


def test_route_unrenormalised_is_softmax_probability():
    rng = np.random.default_rng(2)
    lg = rng.standard_normal((50, 8)).astype(np.float32)
    ids, w = oracle.route(lg, 2, renorm=0)
    sm = scipy.special.softmax(lg.astype(np.float64), axis=1)
    np.testing.assert_allclose(w, np.take_along_axis(sm, ids.astype(np.int64), 1), rtol=1e-14)


def test_route_special_cases():
    lg = np.zeros((4, 8), np.float32)
    ids, w = oracle.route(lg, 3)
    assert (ids == np.array([0, 1, 2])).all()
    np.testing.assert_allclose(w, 1.0 / 3.0, rtol=0, atol=1e-16)
    lg[2, 6] = 100.0
    ids, w = oracle.route(lg, 2)
    assert ids[2, 0] == 6 and w[2, 0] > 0.999999
    rng = np.random.default_rng(3)
    lg = rng.standard_normal((100, 64)).astype(np.float32)
    _, w = oracle.route(lg, 6)
    np.testing.assert_allclose(w.sum(1), 1.0, rtol=0, atol=1e-14)
    assert np.all(np.diff(w, axis=1) <= 0)


def test_routing_mass_eq1():
    """Eq. 1: with K = 1 every weight is 1, so the mass is the selection frequency."""
    rng = np.random.default_rng(4)
    lg = rng.standard_normal((300, 8)).astype(np.float32)
    ids, w = oracle.route(lg, 1)
    m = oracle.routing_mass(ids, w, 8)
    np.testing.assert_allclose(m, np.bincount(ids.ravel(), minlength=8) / 300.0, rtol=1e-14)
    ids, w = oracle.route(lg, 2)
    m = oracle.routing_mass(ids, w, 8)
    want = np.array([w[ids == e].sum() for e in range(8)]) / w.sum()
    np.testing.assert_allclose(m, want, rtol=1e-13)
    assert abs(m.sum() - 1.0) < 1e-14


# ---------------------------------------------------------------------------
# permutation
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("T,E,K", [(16, 8, 2), (512, 64, 6), (1, 4, 4), (100, 8, 1)])
def test_permute_invariants_and_stable_sort(T, E, K):
    rng = np.random.default_rng(T + E)
    ids, _ = oracle.route(rng.standard_normal((T, E)).astype(np.float32), K)
    counts, offsets, ss, sp = oracle.permute(ids, E)
    flat = ids.ravel()
    assert counts.sum() == T * K
    assert np.array_equal(counts, np.bincount(flat, minlength=E))
    assert offsets[0] == 0 and np.array_equal(np.diff(offsets), counts)
    assert np.array_equal(np.sort(ss), np.arange(T * K))
    assert np.array_equal(ss, np.argsort(flat, kind="stable"))
    assert np.array_equal(sp[ss], np.arange(T * K))
    for e in range(E):
        seg = ss[offsets[e]:offsets[e + 1]]
        assert np.all(flat[seg] == e) and np.all(np.diff(seg) > 0)


# ---------------------------------------------------------------------------
# paged expert forward
# ---------------------------------------------------------------------------

def _dense_moe(x, Wg, Wu, Wd, ids, w, h_round_fmt=None):
    """Textbook dense MoE in float64: y_t = sum_k w_tk Wd_e (silu(Wg_e x) * Wu_e x)."""
    T = x.shape[0]
    y = np.zeros((T, Wd.shape[1]))
    for t in range(T):
        for k in range(ids.shape[1]):
            e = ids[t, k]
            g = np.einsum("fh,h->f", Wg[e], x[t])
            u = np.einsum("fh,h->f", Wu[e], x[t])
            h = g * scipy.special.expit(g) * u
            if h_round_fmt == F16:
                h = h.astype(np.float16).astype(np.float64)
            y[t] += w[t, k] * np.einsum("nf,f->n", Wd[e], h)
    return y


def _small_cfg(**kw):
    base = dict(cfg_id=90, name="t", E=4, K=2, H=256, F=128, T=6, R=64, G=64,
                act=F16, sdt=F16, mix=None, shuffle_pool=False)
    base.update(kw)
    return synth.LayerConfig(**base)


def _layer(cfg, bits=None):
    w16 = [synth.expert_weights(cfg, p) for p in range(3)]
    if bits is None:
        bits = synth.bitmap(cfg)
    return oracle.OracleLayer(cfg.E, cfg.H, cfg.F, cfg.R, cfg.G, cfg.act, cfg.sdt, w16, bits), w16


def _dequantized_dense(L: oracle.OracleLayer, p):
    """Dense [E, rows, cols] float64 weights read at each page's bitwidth."""
    W = oracle.decode16(L.w16[p], L.act).copy()
    E, rows, cols = W.shape
    for e in range(E):
        for rb in range(rows // L.R):
            b, c, s, z = L.page(p, e, rb)
            if b != 16:
                sv = np.repeat(oracle.decode16(s, L.sdt), L.G, axis=1)
                zv = np.repeat(oracle.decode16(z, L.sdt), L.G, axis=1)
                W[e, rb * L.R:(rb + 1) * L.R] = zv + c.astype(np.float64) * sv
    return W


def test_all_16bit_pages_equal_textbook_moe():
    """P1: every page at 16 bits -> the plain dense MoE."""
    cfg = _small_cfg()
    bits = [np.full((cfg.E, cfg.nrb(p)), 16, np.int32) for p in range(3)]
    L, w16 = _layer(cfg, bits)
    x16 = synth.activations(cfg)
    ids, w = oracle.route(synth.logits(cfg), cfg.K)
    y = L.forward(x16, ids, w)
    x = oracle.decode16(x16, F16)
    ref = _dense_moe(x, *(oracle.decode16(a, F16) for a in w16), ids, w)
    np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-12 * np.abs(ref).max())


def test_mixed_pages_equal_dense_moe_of_dequantized_weights():
    """Each row is read at its own page's bitwidth (row-block indexing)."""
    cfg = _small_cfg(E=3, H=256, F=192, T=5)
    L, _ = _layer(cfg)
    assert len({int(b) for p in range(3) for b in L.bits[p].ravel()}) == 3
    x16 = synth.activations(cfg)
    ids, w = oracle.route(synth.logits(cfg), cfg.K)
    y = L.forward(x16, ids, w)
    ref = _dense_moe(oracle.decode16(x16, F16), *(_dequantized_dense(L, p) for p in range(3)), ids, w)
    np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-12 * np.abs(ref).max())
    yr = L.forward(x16, ids, w, h_round=True)
    refr = _dense_moe(oracle.decode16(x16, F16), *(_dequantized_dense(L, p) for p in range(3)), ids, w,
                      h_round_fmt=F16)
    np.testing.assert_allclose(yr, refr, rtol=1e-9, atol=1e-9 * np.abs(refr).max())


def _bf16_rne(a32):
    """float32 -> bfloat16 value (round to nearest even), by the bit formula."""
    u = np.asarray(a32, np.float32).view(np.uint32).astype(np.uint64)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    return r.astype(np.uint32).view(np.float32).astype(np.float64)


@pytest.mark.parametrize("act", [F16, BF16])
def test_w_round_equals_dense_moe_of_rounded_weights(act):
    """w_round: a quantized weight enters as fl32(z + c*s) rounded to the
    activation format; 16-bit pages are unchanged. Reference: numpy's own
    float32 / float16 conversions (bfloat16 by the round-to-nearest-even bit
    formula) applied to the dense dequantized weights."""
    cfg = _small_cfg(E=3, H=256, F=192, T=5, act=act, sdt=act)
    L, _ = _layer(cfg)
    x16 = synth.activations(cfg)
    ids, w = oracle.route(synth.logits(cfg), cfg.K)
    dense = []
    for p in range(3):
        W = _dequantized_dense(L, p)
        q = np.repeat(np.stack([np.array(L.bits[p][e]) for e in range(cfg.E)]) != 16, cfg.R, axis=1)
        W32 = W.astype(np.float32)
        Wr = W32.astype(np.float16).astype(np.float64) if act == F16 else _bf16_rne(W32)
        dense.append(np.where(q[:, :, None], Wr, W))
        assert (dense[-1] != W).any()
    y = L.forward(x16, ids, w, w_round=True)
    ref = _dense_moe(oracle.decode16(x16, act), *dense, ids, w)
    np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-12 * np.abs(ref).max())
    # with every page at 16 bits the option changes nothing
    bits16 = [np.full((cfg.E, cfg.nrb(p)), 16, np.int32) for p in range(3)]
    L16, _ = _layer(cfg, bits16)
    assert np.array_equal(L16.forward(x16, ids, w, w_round=True), L16.forward(x16, ids, w))


def test_zero_up_projection_gives_zero_output():
    """P9: W_up = 0 -> h = 0 -> y = 0 exactly."""
    cfg = _small_cfg()
    w16 = [synth.expert_weights(cfg, p) for p in range(3)]
    w16[1][:] = 0
    bits = [np.full((cfg.E, cfg.nrb(p)), 16, np.int32) for p in range(3)]
    L = oracle.OracleLayer(cfg.E, cfg.H, cfg.F, cfg.R, cfg.G, cfg.act, cfg.sdt, w16, bits)
    ids, w = oracle.route(synth.logits(cfg), cfg.K)
    assert not L.forward(synth.activations(cfg), ids, w).any()


def test_single_expert_is_plain_ffn():
    """P9: one expert, K = 1, weight 1 -> the plain SwiGLU FFN."""
    cfg = _small_cfg(E=1, K=1)
    bits = [np.full((1, cfg.nrb(p)), 16, np.int32) for p in range(3)]
    L, w16 = _layer(cfg, bits)
    x16 = synth.activations(cfg)
    ids, w = oracle.route(synth.logits(cfg), 1)
    assert np.all(w == 1.0)
    y = L.forward(x16, ids, w)
    x = oracle.decode16(x16, F16)
    Wg, Wu, Wd = (oracle.decode16(a, F16)[0] for a in w16)
    g, u = x @ Wg.T, x @ Wu.T
    ref = (g / (1 + np.exp(-g)) * u) @ Wd.T
    np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-12 * np.abs(ref).max())


def test_token_subset_matches_full_forward():
    cfg = _small_cfg()
    L, _ = _layer(cfg)
    x16 = synth.activations(cfg)
    ids, w = oracle.route(synth.logits(cfg), cfg.K)
    full = L.forward(x16, ids, w)
    sub = L.forward(x16, ids, w, tokens=[4, 1])
    assert np.array_equal(sub[[1, 4]], full[[1, 4]])
    assert not sub[[0, 2, 3, 5]].any()


def test_layer_requant_semantics():
    """Lowering: no-op at equal bits, error when raising, Eq. 3 bytes released."""
    cfg = _small_cfg()
    bits = [np.full((cfg.E, cfg.nrb(p)), 16, np.int32) for p in range(3)]
    L, w16 = _layer(cfg, bits)
    assert L.requant(0, 1, 0, 16) == 0
    K = cfg.H
    assert L.requant(0, 1, 0, 8) == oracle.page_bytes(64, K, 64, 16) - oracle.page_bytes(64, K, 64, 8)
    with pytest.raises(ValueError):
        L.requant(0, 1, 0, 16)
    assert L.requant(0, 1, 0, 4) == (64 * K) // 2
    # 16 -> 4 directly equals quantizing the 16-bit rows
    L.requant(2, 0, 1, 4)
    c, s, z = oracle.quantize_page16(w16[2][0, 64:128], F16, 64, 4, F16)
    _, c2, s2, z2 = L.page(2, 0, 1)
    assert np.array_equal(c, c2) and np.array_equal(s, s2) and np.array_equal(z, z2)
