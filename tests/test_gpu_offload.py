"""Page offload and reload on the GPU (Sec. 3.1 page states and offload
order): a block's page is copied to pinned host memory before the block is
lowered, and a reload raises it back from that copy.

Checked: the lowered pages are bit-exact against the oracle's requantization;
after the reload every page is byte-identical to the oracle's page of the
original bitwidth and the layer's forward output equals (bit for bit) what it
was before the offload; the pool regains its layout's byte count; the error
paths leave the table unchanged.
"""
import numpy as np
import pytest

import oracle
from helpers import case, gpu_layer, oracle_layer, say, to_dev, to_dev16
from paper_2607_16184_amd import synth

pytestmark = pytest.mark.gpu


def _slot(n):
    return (n + 255) // 256 * 256


def _forward(L, cfg, logits, x16):
    routing = L.route(to_dev(logits), cfg.K)
    x = to_dev16(x16)
    return L.forward(x, routing), L.forward(x, routing, out_fp32=True)


def _pages_equal(L, O, pages):
    for (e, p, rb) in pages:
        assert np.array_equal(L.page_image(e, p, rb), O.page_image(p, e, rb)), (e, p, rb)


@pytest.mark.parametrize("src,low", [(16, 4), (8, 4), (16, 8)])
def test_offload_lower_reload_round_trip(src, low):
    import torch
    cfg, w16, _, order = case("tiny")
    bits = [np.full((cfg.E, cfg.nrb(p)), src, np.int32) for p in range(3)]
    say("offload/reload %d->%d->%d" % (src, low, src))
    L = gpu_layer(cfg, w16, bits, order, slack=1.0)
    O = oracle_layer(cfg, w16, bits)
    O0 = oracle_layer(cfg, w16, bits)
    logits, x16 = synth.logits(cfg), synth.activations(cfg)
    y16_0, y32_0 = _forward(L, cfg, logits, x16)
    torch.cuda.synchronize()
    used0 = L.stats()[0]
    blocks = [pg for i, pg in enumerate(order) if i % 2 == 1]
    kdim = lambda p: cfg.F if p == 2 else cfg.H
    host_need = sum(_slot(oracle.page_bytes(cfg.R, kdim(p), cfg.G, src)) for (_, p, _) in blocks)
    L.set_host_pool(host_need)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    L.offload(blocks, stream=side)
    assert L.host_pool_stats() == (host_need, host_need)
    delta = L.requant(blocks, low, stream=side)
    want = sum(O.requant(p, e, rb, low) for (e, p, rb) in blocks)
    assert delta == want
    assert L.commit() == len(blocks)
    torch.cuda.synchronize()
    _pages_equal(L, O, order)
    assert L.reclaim() > 0
    for (e, p, rb) in blocks:
        assert L.host_copy_info(e, p, rb) == (src, True)

    say("reload %d->%d" % (low, src))
    added = L.reload(blocks, stream=side)
    assert added == sum(oracle.page_bytes(cfg.R, kdim(p), cfg.G, src) -
                        oracle.page_bytes(cfg.R, kdim(p), cfg.G, low) for (_, p, _) in blocks)
    e0, p0, rb0 = blocks[0]
    ent = L.entry(e0, p0, rb0)
    assert ent.bits == low and ent.state == 3          # the lower page is served until the commit
    assert L.commit() == len(blocks)
    torch.cuda.synchronize()
    ent = L.entry(e0, p0, rb0)
    assert ent.bits == src and ent.state == 1
    _pages_equal(L, O0, order)
    y16_1, y32_1 = _forward(L, cfg, logits, x16)
    torch.cuda.synchronize()
    assert torch.equal(y16_0, y16_1) and torch.equal(y32_0, y32_1)
    L.reclaim()
    assert L.stats()[0] == used0
    for (e, p, rb) in blocks:
        L.drop_host_copy(e, p, rb)
    L.reclaim()
    assert L.host_pool_stats() == (host_need, 0)
    L.close()


def test_offload_reload_errors():
    import torch
    from paper_2607_16184_amd.pw import PWError
    cfg, w16, _, order = case("tiny")
    bits = [np.full((cfg.E, cfg.nrb(p)), 16, np.int32) for p in range(3)]
    say("offload/reload error paths")
    L = gpu_layer(cfg, w16, bits, order, slack=0.0)
    blk = order[0]
    with pytest.raises(PWError) as ei:
        L.offload([blk])
    assert ei.value.status == 6                         # no host pool
    one = _slot(oracle.page_bytes(cfg.R, cfg.F if blk[1] == 2 else cfg.H, cfg.G, 16))
    L.set_host_pool(one)
    with pytest.raises(PWError) as ei:
        L.reload([blk])
    assert ei.value.status == 6                         # no host copy
    with pytest.raises(PWError) as ei:
        L.offload([order[0], order[1]])
    assert ei.value.status == 2                         # host pool too small: nothing copied
    assert L.host_pool_stats()[1] == 0
    L.offload([blk])
    torch.cuda.synchronize()
    with pytest.raises(PWError) as ei:
        L.reload([blk])
    assert ei.value.status == 4                         # the copy is not above the committed bitwidth
    assert L.entry(*blk).state == 1
    L.close()
