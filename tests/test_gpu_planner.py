"""Routing statistics on the GPU and the planner driving requantization
(Sec. 3.2, Alg. 1; Eq. 1).

Checked: per-expert slot counts exactly; routing-weighted sums within the
routing-weight tolerance (the kernel's weights and the oracle's differ by
ulps of exp); norms and their maximum to 1e-12; accumulation over calls;
run-to-run bit identity; and an end-to-end step where the library's plan
equals the oracle planner's, and the requantized pages are bit-exact.
"""
import numpy as np
import pytest

import oracle
from oracle import planner as P
from helpers import case, gpu_layer, oracle_layer, say, to_dev, to_dev16
from paper_2607_16184_amd import pw, synth

pytestmark = pytest.mark.gpu


def _oracle_stats(rows64, row_of_slot, logits, K, E):
    ids, w = oracle.route(logits, K)
    _, off, ss, _ = oracle.permute(ids, E)
    return P.routing_stats(rows64, row_of_slot(ss, off), w, off, ss)


def _compare(got, want):
    got = np.asarray(got)
    np.testing.assert_array_equal(got[:, 1], want[:, 1])                          # counts
    np.testing.assert_allclose(got[:, 4], want[:, 4], rtol=1e-12, atol=0)         # max norm
    scale = np.maximum(np.abs(want[:, [0, 2, 3]]), 1e-300)
    assert np.all(np.abs(got[:, [0, 2, 3]] - want[:, [0, 2, 3]]) <= 2e-6 * scale + 1e-12), (got, want)


@pytest.mark.parametrize("name", ["tiny", "mixtral_decode", "mixtral_prefill"])
def test_routing_stats_gate_up_input(name):
    import torch
    cfg = synth.CONFIGS[name]
    say("routing stats of x: %s" % name)
    from paper_2607_16184_amd.layer import PagedLayer
    L = PagedLayer(cfg, 1 << 20)
    logits, x16 = synth.logits(cfg), synth.activations(cfg)
    routing = L.route(to_dev(logits), cfg.K)
    x = to_dev16(x16)
    st = L.routing_stats(x, routing)
    st2 = L.routing_stats(x, routing)
    torch.cuda.synchronize()
    assert torch.equal(st, st2)                                                   # bit-identical runs
    x64 = synth.from16(x16, cfg.act).astype(np.float64)
    want = _oracle_stats(x64, lambda ss, off: ss // cfg.K, logits, cfg.K, cfg.E)
    _compare(st.cpu().numpy(), want)
    # accumulation over two steps: sums add, the maximum stays
    acc = L.routing_stats(x, routing, out=st.clone(), accumulate=True)
    torch.cuda.synchronize()
    a, b = acc.cpu().numpy(), st.cpu().numpy()
    np.testing.assert_array_equal(a[:, [0, 1, 2, 3]], 2 * b[:, [0, 1, 2, 3]])
    np.testing.assert_array_equal(a[:, 4], b[:, 4])
    L.close()


def test_routing_stats_down_input_by_position():
    import torch
    cfg = synth.CONFIGS["tiny"]
    say("routing stats of expert-major rows")
    from paper_2607_16184_amd.layer import PagedLayer
    L = PagedLayer(cfg, 1 << 20)
    logits = synth.logits(cfg)
    S = cfg.T * cfg.K
    rng = np.random.default_rng(11)
    h16 = synth.to16(rng.standard_normal((S, cfg.F)).astype(np.float32), cfg.act)
    routing = L.route(to_dev(logits), cfg.K)
    st = L.routing_stats(to_dev16(h16), routing, rows_by_position=True)
    torch.cuda.synchronize()
    h64 = synth.from16(h16, cfg.act).astype(np.float64)
    want = _oracle_stats(h64, lambda ss, off: np.arange(len(ss)), logits, cfg.K, cfg.E)
    _compare(st.cpu().numpy(), want)
    L.close()


def test_routing_stats_no_tokens():
    import torch
    cfg = synth.CONFIGS["tiny"]
    say("routing stats with no tokens")
    from paper_2607_16184_amd.layer import PagedLayer
    L = PagedLayer(cfg, 1 << 20)
    routing = L.route(torch.zeros((0, cfg.E), dtype=torch.float32, device="cuda"), cfg.K)
    st = torch.full((cfg.E, 5), 7.0, dtype=torch.float64, device="cuda")
    L.routing_stats(torch.zeros((0, cfg.H), dtype=torch.int16, device="cuda"), routing, out=st)
    torch.cuda.synchronize()
    assert torch.count_nonzero(st) == 0
    L.close()


def _config():
    return dict(bucket_frac=[0.25, 0.75], mult=[6.0, 1.0], floors=[[8, 8], [8, 4], [4, 4]],
                alpha=0.5, rho_min=-0.5, rho_max=0.5, eps=1e-9)


def test_planner_drives_requant():
    """One planner step on the tiny layer under KV pressure: the library's plan
    (from GPU statistics) equals the oracle planner's (from its own routing and
    statistics); applying it lowers exactly those blocks, the requantized
    pages are bit-exact and the pool gains the plan's bytes."""
    import torch
    cfg, w16, _, order = case("tiny")
    bits = [np.full((cfg.E, cfg.nrb(p)), 16, np.int32) for p in range(3)]
    for p in range(3):
        bits[p][::3] = 8                                                          # some blocks start at 8
    say("planner step on the tiny layer")
    L = gpu_layer(cfg, w16, bits, order, slack=1.0)
    O = oracle_layer(cfg, w16, bits)
    rng = np.random.default_rng(21)
    n = L.n_entries
    sens = np.sort(rng.gamma(1.0, 1.0, (n, 3)), 1)
    hw, ha, hc = rng.normal(0, 0.01, (2, 2, 3)), rng.normal(0, 0.2, (2, 2)), rng.uniform(0.3, 1.0, (2, 2))
    kw = _config()
    planner = L.planner(sens, pw.planner_config(head_w=hw, head_a=ha, head_c=hc, **kw))
    logits, x16 = synth.logits(cfg), synth.activations(cfg)
    routing = L.route(to_dev(logits), cfg.K)
    st = L.routing_stats(to_dev16(x16), routing)
    planner.add_request(st, None, 1.0)
    kvb = 96 * 1024
    r = planner.step(L, free_blocks=1, free_threshold=3, kv_block_bytes=kvb)   # D = 3 blocks
    assert r.triggered == 1 and r.target == 3 * kvb

    # the oracle's plan from its own statistics
    nrb = L.n_entries // (cfg.E * 3)
    units, q = [], []
    for i in range(n):
        e, rem = divmod(i, 3 * nrb)
        p, rb = divmod(rem, nrb)
        valid = rb < cfg.nrb(p)
        kd = cfg.F if p == 2 else cfg.H
        units.append(P.Unit(e, 1 if p == 2 else 0, tuple(oracle.page_bytes(cfg.R, kd, cfg.G, b) for b in (16, 8, 4)),
                            tuple(float(v) for v in sens[i])))
        q.append(int(bits[p][e, rb]) if valid else 0)
    x64 = synth.from16(x16, cfg.act).astype(np.float64)
    sto = _oracle_stats(x64, lambda ss, off: ss // cfg.K, logits, cfg.K, cfg.E)
    m, pg = P.mass_and_features(sto)
    D, plans, best = P.plan_step(P.Config(head_w=hw, head_a=ha, head_c=hc, **kw), units, q, m,
                                 np.stack([pg, np.zeros_like(pg)], 1), 1, 3, kvb)
    assert r.stage == best.stage and r.bytes == best.nbytes
    got = planner.plan()
    assert {u: (f, t) for (u, f, t, _) in got} == best.final()

    free0 = L.stats()[1]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    delta = planner.apply(L, stream=side)
    assert delta == best.nbytes
    assert L.commit() == len(got)
    torch.cuda.synchronize()
    L.reclaim()
    assert L.stats()[1] - free0 == delta
    for (u, f, t, _) in got:
        e, rem = divmod(u, 3 * nrb)
        p, rb = divmod(rem, nrb)
        assert L.entry(e, p, rb).bits == t
        O.requant(p, e, rb, t)
        assert np.array_equal(L.page_image(e, p, rb), O.page_image(p, e, rb)), (e, p, rb)
    # a second step on the lowered table plans from the new bitwidths
    r2 = planner.step(L, free_blocks=1, free_threshold=3, kv_block_bytes=kvb)
    for (u, f, t, _) in planner.plan():
        e, rem = divmod(u, 3 * nrb)
        p, rb = divmod(rem, nrb)
        assert f == L.entry(e, p, rb).bits
    planner.close()
    L.close()
