"""The whole step (route, paged GEMMs, combine) captured in a HIP graph and
replayed: every replay is bit-identical to the eager step, for each GEMM path
(decode kernels, streaming kernel, LDS-tiled kernel), with eager work on the
same stream between replays. Nothing in the step allocates or clears memory
with a memset, so the captured launches are the eager ones."""
import pytest

from helpers import case, gpu_layer, say, to_dev, to_dev16
from paper_2607_16184_amd import synth

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("T", [16, 300, 1000])
def test_graph_replay_matches_eager(T):
    import torch
    from paper_2607_16184_amd.layer import PagedLayer
    cfg, w16, bits, order = case("tiny", T=T)
    say("graph replay tiny T=%d" % T)
    L = gpu_layer(cfg, w16, bits, order)
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
