"""Runtime downshift on the GPU (Sec. 3.1 offload order, Sec. 3.3 asynchronous
page movement, Eq. 3): requantize chunks of 16-bit pages to int4 on a side
stream while decode steps run on the main stream, commit at step boundaries,
reclaim the old slots.

Checked: every requantized page is bit-exact against the oracle; the pool
gains exactly sum(Delta) bytes; every step's output (17 tokens each) matches
the oracle run with the table committed at that step; after the switch the
layer computes bit-identical outputs to a layer built directly at the
post-switch bitwidths.
"""
import numpy as np
import pytest

import oracle
from helpers import assert_all_pages_equal, case, gpu_layer, oracle_layer, rel_err, say, to_dev, to_dev16
from paper_2607_16184_amd import synth

pytestmark = pytest.mark.gpu


def _step(L, cfg, s, out_fp32=True):
    lg, x16 = synth.step_inputs(cfg, s)
    r = L.route(to_dev(lg), cfg.K)
    return L.forward(to_dev16(x16), r, out_fp32=out_fp32), lg, x16


def test_downshift_under_decode():
    import torch
    cfg, w16, bits, order = case("downshift")
    plan = synth.downshift_plan(cfg, list(bits))
    assert len(plan) == 8 and all(len(c) == 32 for c in plan)
    say("downshift: build layer")
    L = gpu_layer(cfg, w16, bits, order, slack=0.1)
    O = oracle_layer(cfg, w16, bits)
    side = torch.cuda.Stream()
    free0 = L.stats()[1]
    want_delta = 0
    toks = list(range(0, cfg.T, 4)) + [cfg.T - 1]
    for s, chunk in enumerate(plan):
        say("downshift: step %d, requant chunk of %d pages" % (s, len(chunk)))
        # the requant is ordered after everything already on the main stream
        side.wait_stream(torch.cuda.current_stream())
        delta = L.requant(chunk, 4, stream=side)
        y, lg, x16 = _step(L, cfg, s)                  # overlaps the requant
        # the step saw the table committed before it (its own chunk is still
        # pending): the oracle holds exactly chunks 0 .. s-1 here
        ids, w = oracle.route(lg, cfg.K)
        r2 = O.forward(x16, ids, w, h_round=True, tokens=toks)
        err = rel_err(y.cpu().numpy()[toks], r2[toks])
        assert err <= 1e-3, (s, err)
        for (e, p, rb) in chunk:
            want_delta += O.requant(p, e, rb, 4)
        assert delta == sum(oracle.delta_bytes(cfg.R, cfg.kdim(p), cfg.G, 16, 4) for (_, p, _) in chunk)
        assert L.commit() == len(chunk)                # step boundary
        L.reclaim()
    torch.cuda.synchronize()
    L.reclaim()
    assert want_delta == 258_736_128
    assert L.stats()[1] - free0 == want_delta          # Eq. 3, exactly
    say("downshift: every downshifted page")
    assert assert_all_pages_equal(L, O, cfg, [b for c in plan for b in c]) == 256
    # the step after the last commit reads every int4 page
    ya, lg, x16 = _step(L, cfg, 39)
    ids, w = oracle.route(lg, cfg.K)
    r2 = O.forward(x16, ids, w, h_round=True, tokens=toks)
    assert rel_err(ya.cpu().numpy()[toks], r2[toks]) <= 1e-3
    say("downshift: compare with a layer built at the post-switch bitwidths")
    post = [b.copy() for b in bits]
    for chunk in plan:
        for (e, p, rb) in chunk:
            post[p][e, rb] = 4
    L2 = gpu_layer(cfg, w16, post, order)
    ya, _, _ = _step(L, cfg, 40)
    yb, _, _ = _step(L2, cfg, 40)
    torch.cuda.synchronize()
    assert torch.equal(ya, yb)
    L.close()
    L2.close()
