"""The whole step (route, paged GEMMs, combine) captured in a HIP graph and
replayed: every replay is bit-identical to the eager step, for each GEMM path
(decode kernels, streaming kernel, LDS-tiled kernel), with eager work on the
same stream between replays. Nothing in the step allocates or clears memory
with a memset, so the captured launches are the eager ones."""
import pytest

from helpers import case, gpu_layer, say, to_dev, to_dev16
from paper_2607_16184_amd import synth

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("T,chains", [(16, 2), (16, 1), (300, 2), (1000, 2)])
def test_graph_replay_matches_eager(T, chains):
    """Captured with two chains (two graph branches at decode sizes) or one."""
    import torch
    from paper_2607_16184_amd.layer import PagedLayer
    cfg, w16, bits, order = case("tiny", T=T)
    say("graph replay tiny T=%d chains=%d" % (T, chains))
    L = gpu_layer(cfg, w16, bits, order)
    L.set_chains(chains)
    logits, x = to_dev(synth.logits(cfg)), to_dev16(synth.activations(cfg))
    rbuf = PagedLayer.routing_buffers(cfg.T, cfg.E, cfg.K)
    y = torch.empty((cfg.T, cfg.H), dtype=torch.float32, device="cuda")

    def step():
        L.forward(x, L.route(logits, cfg.K, out=rbuf), out_fp32=True, y=y)

    step()
    torch.cuda.synchronize()
    want = y.clone()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    other = torch.empty_like(y)
    for r in range(3):
        y.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(y, want), r
        L.forward(x, L.route(logits, cfg.K), out_fp32=True, y=other)   # eager work in between
        torch.cuda.synchronize()
        assert torch.equal(other, want), r
    L.close()


@pytest.mark.parametrize("T", [16, 100])
def test_graph_replay_shared_experts(T):
    """A layer with shared experts: their GEMMs run on the layer's own stream,
    forked from the caller's and joined before the combine, so the captured
    graph has two branches. Every replay is bit-identical to the eager step,
    with eager steps (which fork and join again) between the replays."""
    import torch
    from paper_2607_16184_amd.layer import PagedLayer
    cfg, w16, bits, order = case("tiny_shared", T=T)
    say("graph replay, shared experts, T=%d" % T)
    L = gpu_layer(cfg, w16, bits, order)
    L.set_shared_experts(cfg.n_shared)
    logits, x = to_dev(synth.logits(cfg)), to_dev16(synth.activations(cfg))
    gate = to_dev(synth.shared_gate(cfg))
    Kt = cfg.K + cfg.n_shared
    rbuf = PagedLayer.routing_buffers(cfg.T, cfg.E, Kt)
    y = torch.empty((cfg.T, cfg.H), dtype=torch.float32, device="cuda")

    def step(out):
        L.forward(x, L.route_shared(logits, cfg.K, cfg.n_shared, gate=gate, out=rbuf), out_fp32=True, y=out)

    step(y)
    torch.cuda.synchronize()
    want = y.clone()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step(y)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step(y)
    other = torch.empty_like(y)
    for r in range(3):
        y.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(y, want), r
        step(other)                                        # eager work in between
        torch.cuda.synchronize()
        assert torch.equal(other, want), r
    L.close()


@pytest.mark.parametrize("T", [16, 40, 100])
def test_chains_bit_identical(T):
    """The routed experts as one chain or as two concurrent chains (the
    second on the layer's stream) give the same bits, 16-bit and fp32 out."""
    import torch
    cfg, w16, bits, order = case("tiny", T=T)
    say("one chain vs two chains, tiny T=%d" % T)
    L = gpu_layer(cfg, w16, bits, order)
    logits, x = to_dev(synth.logits(cfg)), to_dev16(synth.activations(cfg))
    routing = L.route(logits, cfg.K)
    out = {}
    for chains in (1, 2):
        L.set_chains(chains)
        out[chains] = (L.forward(x, routing).clone(), L.forward(x, routing, out_fp32=True).clone())
    torch.cuda.synchronize()
    assert torch.equal(out[1][0], out[2][0]) and torch.equal(out[1][1], out[2][1])
    from paper_2607_16184_amd import pw
    for bad in (0, 3):
        with pytest.raises(pw.PWError) as ei:
            L.set_chains(bad)
        assert ei.value.status == pw.PW_EINVAL
    L.close()


@pytest.mark.parametrize("T,kw", [(16, {}), (100, {}), (600, dict(F=4096, n_shared=4, E=12))])
def test_chains_bit_identical_shared(T, kw):
    """With shared experts the shared range runs on the layer's stream beside
    the routed one (two chains) or after it (one chain): same bits. T = 100
    puts the shared range on the streaming kernel, T = 600 (4 shared experts
    of F = 4096) on the tiled one."""
    import torch
    cfg, w16, bits, order = case("tiny_shared", T=T, **kw)
    say("one chain vs two chains with shared experts, T=%d" % T)
    L = gpu_layer(cfg, w16, bits, order)
    L.set_shared_experts(cfg.n_shared)
    logits, x = to_dev(synth.logits(cfg, T=T)), to_dev16(synth.activations(cfg, T=T))
    gate = to_dev(synth.shared_gate(cfg, T=T))
    routing = L.route_shared(logits, cfg.K, cfg.n_shared, gate=gate)
    out = {}
    for chains in (1, 2):
        L.set_chains(chains)
        out[chains] = (L.forward(x, routing).clone(), L.forward(x, routing, out_fp32=True).clone())
    torch.cuda.synchronize()
    assert torch.equal(out[1][0], out[2][0]) and torch.equal(out[1][1], out[2][1])
    L.close()
