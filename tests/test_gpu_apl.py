"""Nested bit-plane pages on the GPU (any-precision weights: Sec. 2.2 and 3.1).

Checked: every quantized page is byte-identical to the oracle's (codes,
bit-planes and both LUTs); the forward through the streaming kernel matches
the oracle's dense MoE of the reconstructed 16-bit weights; lowering 8 -> 4
bits runs no kernel, keeps the page prefix, frees exactly the page tail
(Eq. 3), and the forward then follows the 4-bit LUTs; unsupported moves are
refused.
"""
import numpy as np
import pytest

import oracle
from oracle import apl
from helpers import case, oracle_layer, rel_err, say, to_dev, to_dev16, y16_values
from paper_2607_16184_amd import pw, synth

pytestmark = pytest.mark.gpu

TOL16, TOL32 = 2e-2, 1e-3


def _oracle_pages(cfg, w16, bits):
    """{(e, p, rb): (8-bit page bytes, codes8, lut4, lut8)} for every quantized block."""
    out = {}
    for p in range(3):
        for e in range(cfg.E):
            for rb in range(cfg.nrb(p)):
                if bits[p][e, rb] == 16:
                    continue
                rows = w16[p][e, rb * cfg.R:(rb + 1) * cfg.R]
                v = oracle.decode16(rows, cfg.act).astype(np.float64)
                codes, c4, c8 = apl.quantize_rows(v)
                l4, l8 = apl.lut16(c4, cfg.act), apl.lut16(c8, cfg.act)
                out[(e, p, rb)] = (apl.encode_page(codes, l4, l8), codes, l4, l8)
    return out


def _effective_w16(cfg, w16, bits, pages):
    """16-bit weights the kernels must reproduce: LUT values of each quantized block."""
    eff = [np.array(w, copy=True) for w in w16]
    for (e, p, rb), (_, codes, l4, l8) in pages.items():
        b = int(bits[p][e, rb])
        eff[p][e, rb * cfg.R:(rb + 1) * cfg.R] = apl.dequant(codes, l8 if b == 8 else l4, b)
    return eff


def _layer(cfg, w16, bits, slack=0.25):
    from paper_2607_16184_amd.layer import PagedLayer
    R = cfg.R
    need = 0
    for p in range(3):
        K = cfg.F if p == 2 else cfg.H
        for b in np.asarray(bits[p]).ravel():
            need += pw.pw_page_bytes(cfg, p, 16) if b == 16 else apl.page_bytes(R, K, int(b))
    L = PagedLayer(cfg, int(need * (1 + slack)) + 4096)
    order = synth.pool_order(cfg)
    L.load_pages(w16, bits, [pg for pg in order if bits[pg[1]][pg[0], pg[2]] == 16])
    L.load_pages_apl(w16, [(e, p, rb, int(bits[p][e, rb])) for (e, p, rb) in order if bits[p][e, rb] != 16])
    return L


def _forward_check(L, cfg, eff, T=None):
    import torch
    logits = synth.logits(cfg, T=T)
    x16 = synth.activations(cfg, T=T)
    O = oracle_layer(cfg, eff, [np.full_like(b, 16) for b in synth.bitmap(cfg)])
    routing = L.route(to_dev(logits), cfg.K)
    x = to_dev16(x16)
    y16 = L.forward(x, routing)
    y32 = L.forward(x, routing, out_fp32=True)
    torch.cuda.synchronize()
    ids, w = oracle.route(logits, cfg.K)
    r1 = O.forward(x16, ids, w, h_round=False)
    r2 = O.forward(x16, ids, w, h_round=True)
    return rel_err(y16_values(y16, cfg.act), r1), rel_err(y32.cpu().numpy(), r2)


@pytest.mark.parametrize("act", [oracle.F16, oracle.BF16])
def test_apl_pages_bit_exact_and_forward(act):
    cfg, w16, bits, _ = case("tiny", act=act, sdt=act)
    say("bit-plane pages: tiny layer act %d, quantize %d blocks" % (act, sum(int((b != 16).sum()) for b in bits)))
    L = _layer(cfg, w16, bits)
    pages = _oracle_pages(cfg, w16, bits)
    for (e, p, rb), (buf, _, _, _) in pages.items():
        got = L.page_image(e, p, rb)
        want = buf[:got.size]
        K = cfg.F if p == 2 else cfg.H
        assert got.size == apl.page_bytes(cfg.R, K, int(bits[p][e, rb]))
        if not np.array_equal(got, want):
            b = int(bits[p][e, rb])
            gc, gl = apl.decode_page(got, cfg.R, K, b)
            wc, wl = apl.decode_page(want, cfg.R, K, b)
            raise AssertionError("page %s: %d code and %d LUT mismatches" % ((e, p, rb), (gc != wc).sum(),
                                                                          (gl != wl).sum()))
        assert L.entry(e, p, rb).rsv == pw.PW_FMT_APL
    eff = _effective_w16(cfg, w16, bits, pages)
    for T in (None, 200):
        say("bit-plane forward T=%s" % T)
        e16, e32 = _forward_check(L, cfg, eff, T)
        assert e16 <= TOL16 and e32 <= TOL32, (T, e16, e32)
    L.close()


def test_apl_downshift_drops_planes():
    import torch
    cfg, w16, bits, _ = case("tiny")
    say("bit-plane downshift 8 -> 4")
    L = _layer(cfg, w16, bits)
    pages = _oracle_pages(cfg, w16, bits)
    eight = [k for k in pages if bits[k[1]][k[0], k[2]] == 8]
    free0 = L.stats()[1]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    pw.pw_profile_read(L.handle, reset=True)
    pw.pw_profile_enable(L.handle, True)
    delta = L.requant(eight, 4, stream=side)
    want = sum(apl.page_bytes(cfg.R, cfg.F if p == 2 else cfg.H, 8) - apl.page_bytes(cfg.R, cfg.F if p == 2 else cfg.H, 4)
               for (e, p, rb) in eight)
    assert delta == want
    assert L.commit() == len(eight)
    torch.cuda.synchronize()
    pw.pw_profile_enable(L.handle, False)
    assert pw.pw_profile_read(L.handle, reset=True)[1][pw.PW_PH_REQUANT] == 0   # no requant kernel ran
    L.reclaim()
    assert L.stats()[1] - free0 == want
    bits4 = [b.copy() for b in bits]
    for (e, p, rb) in eight:
        bits4[p][e, rb] = 4
        ent = L.entry(e, p, rb)
        assert ent.bits == 4 and ent.rsv == pw.PW_FMT_APL
        got = L.page_image(e, p, rb)
        assert np.array_equal(got, pages[(e, p, rb)][0][:got.size])
    e16, e32 = _forward_check(L, cfg, _effective_w16(cfg, w16, bits4, pages))
    assert e16 <= TOL16 and e32 <= TOL32, (e16, e32)
    # refused moves: a plane page to 16 bits; the same bitwidth is a no-op
    blk = eight[0]
    with pytest.raises(pw.PWError) as ei:
        L.requant([blk], 16)
    assert ei.value.status == 4
    assert L.requant([blk], 4) == 0
    L.close()


def _slot(n):
    return (n + 255) // 256 * 256


def test_apl_offload_drop_reload():
    """Sec. 3.1's page states with bit-plane pages: the 8-bit pages are copied
    to host memory, lowered in place to 4 bits (tail freed), and raised back
    from their host copies; each state's pages are byte-identical to the
    oracle's and the forward follows the committed precision."""
    import torch
    cfg, w16, bits, _ = case("tiny")
    say("bit-plane offload, 8 -> 4 drop, reload")
    # a reload takes a fresh 8-bit slot while the 4-bit prefix is still held
    # (the freed tails are smaller than a page): room for every raised page
    L = _layer(cfg, w16, bits, slack=1.0)
    pages = _oracle_pages(cfg, w16, bits)
    eight = [k for k in pages if bits[k[1]][k[0], k[2]] == 8]
    kdim = lambda p: cfg.F if p == 2 else cfg.H
    host_need = sum(_slot(apl.page_bytes(cfg.R, kdim(p), 8)) for (_, p, _) in eight)
    L.set_host_pool(host_need)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    L.offload(eight, stream=side)
    assert L.host_pool_stats() == (host_need, host_need)
    L.offload(eight, stream=side)                                      # same bitwidth: no-op
    delta = L.requant(eight, 4, stream=side)
    assert delta == sum(apl.page_bytes(cfg.R, kdim(p), 8) - apl.page_bytes(cfg.R, kdim(p), 4) for (_, p, _) in eight)
    assert L.commit() == len(eight)
    torch.cuda.synchronize()
    L.reclaim()
    bits4 = [b.copy() for b in bits]
    for (e, p, rb) in eight:
        bits4[p][e, rb] = 4
        assert L.host_copy_info(e, p, rb) == (8, True)
    e16, e32 = _forward_check(L, cfg, _effective_w16(cfg, w16, bits4, pages))
    assert e16 <= TOL16 and e32 <= TOL32, (e16, e32)

    say("bit-plane reload 4 -> 8")
    added = L.reload(eight, stream=side)
    assert added == delta
    for (e, p, rb) in eight:
        assert L.entry(e, p, rb).state == pw.PW_PAGE_RELOAD_PENDING
    assert L.commit() == len(eight)
    torch.cuda.synchronize()
    L.reclaim()
    for (e, p, rb) in eight:
        ent = L.entry(e, p, rb)
        assert ent.bits == 8 and ent.rsv == pw.PW_FMT_APL and ent.state == pw.PW_PAGE_RESIDENT
        got = L.page_image(e, p, rb)
        assert got.size == apl.page_bytes(cfg.R, kdim(p), 8)
        assert np.array_equal(got, pages[(e, p, rb)][0]), (e, p, rb)
    e16, e32 = _forward_check(L, cfg, _effective_w16(cfg, w16, bits, pages))
    assert e16 <= TOL16 and e32 <= TOL32, (e16, e32)
    # raising again from a copy of the committed bitwidth is refused
    with pytest.raises(pw.PWError) as ei:
        L.reload([eight[0]], stream=side)
    assert ei.value.status == 4
    torch.cuda.synchronize()
    L.close()


def test_apl_load_errors():
    import torch
    cfg, w16, bits, _ = case("tiny")
    say("bit-plane load errors")
    from paper_2607_16184_amd.layer import PagedLayer
    L = PagedLayer(cfg, 4 << 20)
    with pytest.raises(pw.PWError) as ei:
        L.load_pages_apl(w16, [(0, 0, 0, 16)])
    assert ei.value.status == 1
    L.load_pages_apl(w16, [(0, 0, 0, 8)])
    with pytest.raises(pw.PWError) as ei:
        L.load_pages_apl(w16, [(0, 0, 0, 4)])
    assert ei.value.status == 3
    torch.cuda.synchronize()
    L.close()


def test_apl_wide_range_and_degenerate_rows():
    """The quantizer sums a row's values in any order when every partial sum
    is exact (the row's largest magnitude times K within 2^53 of its
    smallest value's unit); rows beyond that bound take the one-thread form,
    which sums in order of k. Here, in bf16 blocks of each projection: rows
    holding 2^-100-sized values beside ordinary weights (beyond the bound),
    a row of zeros, a constant row, and a row of two values. Every page is
    byte-identical to the oracle's, in both precisions."""
    cfg, w16, bits, _ = case("tiny", act=synth.BF16, sdt=synth.BF16)
    w16 = [np.array(w, copy=True) for w in w16]
    rng = np.random.default_rng(3)
    enc = lambda x: oracle.round_nearest16(float(x), synth.BF16)
    touched = []
    for p in range(3):
        for b in (8, 4):
            e, rb = next((e, rb) for e in range(cfg.E) for rb in range(cfg.nrb(p)) if bits[p][e, rb] == b)
            r0 = rb * cfg.R
            K = w16[p].shape[2]
            tiny = [enc(x) for x in rng.choice([1e-30, -3e-31, 7e-29], size=K // 8)]
            cols = rng.choice(K, size=K // 8, replace=False)
            w16[p][e, r0, cols] = tiny                          # beyond the exact-sum bound
            w16[p][e, r0 + 1, :] = 0                            # zeros
            w16[p][e, r0 + 2, :] = enc(0.25)                    # constant
            w16[p][e, r0 + 3, :] = np.where(np.arange(K) % 3 == 0, enc(-0.5), enc(0.125))   # two values
            touched.append((e, p, rb))
    say("bit-plane pages with wide-range and degenerate rows: %d blocks" % len(touched))
    L = _layer(cfg, w16, bits)
    pages = _oracle_pages(cfg, w16, bits)
    for (e, p, rb), (buf, _, _, _) in pages.items():
        got = L.page_image(e, p, rb)
        want = buf[:got.size]
        if not np.array_equal(got, want):
            K = cfg.F if p == 2 else cfg.H
            b = int(bits[p][e, rb])
            gc, gl = apl.decode_page(got, cfg.R, K, b)
            wc, wl = apl.decode_page(want, cfg.R, K, b)
            raise AssertionError("page %s: %d code and %d LUT mismatches" % ((e, p, rb), (gc != wc).sum(),
                                                                          (gl != wl).sum()))
    L.close()


def test_apl_mixtral_sampled_pages():
    """The Mixtral-shaped decode layer with its quantized pages as bit-plane
    pages (the configuration the benchmark times): sampled pages of every
    projection and both precisions are byte-identical to the oracle's
    (rows of 4096 and 14336 values, bf16 LUTs)."""
    import torch
    cfg = synth.CONFIGS["mixtral_decode"]
    w16 = [synth.expert_weights(cfg, p) for p in range(3)]
    bits = synth.bitmap(cfg)
    say("bit-plane pages: Mixtral decode layer")
    L = _layer(cfg, w16, bits, slack=0.05)
    rng = np.random.default_rng(7)
    picks = []
    for p, b in ((0, 8), (1, 4), (2, 8), (2, 4)):
        cand = [(e, p, rb) for e in range(cfg.E) for rb in range(cfg.nrb(p)) if bits[p][e, rb] == b]
        picks.append(cand[int(rng.integers(len(cand)))])
    for (e, p, rb) in picks:
        say("oracle page %s" % ((e, p, rb),))
        rows = w16[p][e, rb * cfg.R:(rb + 1) * cfg.R]
        codes, c4, c8 = apl.quantize_rows(oracle.decode16(rows, cfg.act).astype(np.float64))
        want = apl.encode_page(codes, apl.lut16(c4, cfg.act), apl.lut16(c8, cfg.act))
        got = L.page_image(e, p, rb)
        assert np.array_equal(got, want[:got.size]), (e, p, rb)
    # the step runs (streaming kernel) and is deterministic
    logits, x16 = synth.logits(cfg), synth.activations(cfg)
    routing = L.route(to_dev(logits), cfg.K)
    x = to_dev16(x16)
    y1 = L.forward(x, routing, out_fp32=True)
    y2 = L.forward(x, routing, out_fp32=True)
    torch.cuda.synchronize()
    assert torch.equal(y1, y2) and bool(torch.isfinite(y1).all())
    L.close()


def test_apl_mixtral_forward_full():
    """The Mixtral-shaped decode layer (4096/14336, 64 tokens) with two
    bit-plane pages per projection and precision and every other page 16-bit:
    the layer then runs the streaming kernel for both GEMMs with 32-slot tiles
    and the down projection split over K, as the benchmark's bit-plane leg
    does. Every token of the output is compared with the oracle's dense MoE of
    the reconstructed weights."""
    import torch
    cfg = synth.CONFIGS["mixtral_decode"]
    w16 = [synth.expert_weights(cfg, p) for p in range(3)]
    bits = [np.full_like(b, 16) for b in synth.bitmap(cfg)]
    rng = np.random.default_rng(11)
    for p in range(3):
        cand = [(e, rb) for e in range(cfg.E) for rb in range(cfg.nrb(p))]
        pick = rng.permutation(len(cand))[:4]
        for j, i in enumerate(pick):
            e, rb = cand[i]
            bits[p][e, rb] = 8 if j < 2 else 4
    say("bit-plane Mixtral forward: 12 bit-plane pages, rest 16-bit")
    L = _layer(cfg, w16, bits, slack=0.05)
    pages = _oracle_pages(cfg, w16, bits)
    assert len(pages) == 12
    for (e, p, rb), (buf, _, _, _) in pages.items():
        got = L.page_image(e, p, rb)
        assert np.array_equal(got, buf[:got.size]), (e, p, rb)
    eff = _effective_w16(cfg, w16, bits, pages)
    say("bit-plane Mixtral forward: oracle on all 64 tokens")
    e16, e32 = _forward_check(L, cfg, eff)
    assert e16 <= TOL16 and e32 <= TOL32, (e16, e32)
    torch.cuda.synchronize()
    L.close()
