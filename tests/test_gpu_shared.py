"""Shared experts on the GPU (Table 1 of the paper: MoE layers with experts
every token uses beside the routed ones). The layer's last n_shared experts
are declared shared; routing appends them to every token with a per-token
gate; the GEMM runs routed and shared experts as separate launches, each on
the kernels suited to its slots per expert. Checked against the oracle:
routing ids, offsets and slot order bit-exact, weights within 1e-6; pages
byte-identical; outputs within 2e-2 (16-bit) and 1e-3 (fp32).

The fp32 output is compared with the oracle's reading of each range's
kernels: the decode kernels (up to 48 expected slots per expert) never round
a weight, the streaming and tiled kernels read a quantized weight rounded to
the activation dtype, so the oracle output is the sum of the routed columns'
forward and the shared columns' forward, each in its kernels' reading.
"""
import numpy as np
import pytest

import oracle
from helpers import assert_all_pages_equal, case, gpu_layer, oracle_layer, rel_err, say, to_dev, to_dev16, y16_values
from paper_2607_16184_amd import synth

pytestmark = pytest.mark.gpu

TOL16, TOL32 = 2e-2, 1e-3


def _rounds(expect):
    """Whether the kernels serving `expect` slots per expert read quantized
    weights rounded to the activation dtype (streaming and tiled kernels)."""
    return expect > 48


def _check(L, O, cfg, T, with_gate, tokens=None):
    import torch
    Er, K, n = cfg.E_routed, cfg.K, cfg.n_shared
    logits = synth.logits(cfg, T=T)
    x16 = synth.activations(cfg, T=T)
    gate = synth.shared_gate(cfg, T=T) if with_gate else None
    routing = L.route_shared(to_dev(logits), K, n, gate=to_dev(gate) if gate is not None else None)
    x = to_dev16(x16)
    y16 = L.forward(x, routing)
    y32 = L.forward(x, routing, out_fp32=True)
    torch.cuda.synchronize()
    ids, w = oracle.route_shared(logits, K, n, gate)
    _, off, ss, sp = oracle.permute(ids, cfg.E)
    S = T * (K + n)
    assert np.array_equal(routing[0].cpu().numpy(), ids)
    assert np.abs(routing[1].cpu().numpy() - w).max() <= 1e-6
    assert np.array_equal(routing[2].cpu().numpy(), off)
    assert np.array_equal(routing[3].cpu().numpy()[:S], ss)
    assert np.array_equal(routing[4].cpu().numpy()[:S], sp)
    tok = list(range(T)) if tokens is None else list(tokens)
    r1 = O.forward(x16, ids, w, h_round=False, tokens=tok)
    rr = _rounds((T * K + Er - 1) // Er)
    rs = _rounds(T)
    r2 = (O.forward(x16, ids[:, :K], w[:, :K], h_round=True, tokens=tok, w_round=rr)
          + O.forward(x16, ids[:, K:], w[:, K:], h_round=True, tokens=tok, w_round=rs))
    e16 = rel_err(y16_values(y16, cfg.act)[tok], r1[tok])
    e32 = rel_err(y32.cpu().numpy()[tok], r2[tok])
    return e16, e32


# T = 16: both ranges on the decode kernels; T = 100: routed on the decode
# kernels (25 slots per expert), shared on the streaming kernel (100);
# T = 300: routed and shared on the streaming kernel (75 and 300 slots per
# expert; two shared experts fill too few 256 x 256 tiles for the tiled one,
# so the tiled kernel runs the shared range only where the tiles fill the
# chip, as in test_shared_experts_tiled)
@pytest.mark.parametrize("T", [16, 100, 300])
@pytest.mark.parametrize("with_gate", [False, True])
def test_tiny_shared_experts(T, with_gate):
    cfg, w16, bits, order = case("tiny_shared")
    say("shared experts: tiny layer 8 + 2, T=%d, gate=%s" % (T, with_gate))
    L = gpu_layer(cfg, w16, bits, order)
    L.set_shared_experts(cfg.n_shared)
    O = oracle_layer(cfg, w16, bits)
    e16, e32 = _check(L, O, cfg, T, with_gate)
    assert e16 <= TOL16 and e32 <= TOL32, (T, e16, e32)
    L.close()


def test_shared_experts_tiled():
    """Shared experts on the tiled kernel: 4 shared experts of a tiny layer
    with F = 4096 at T = 600 fill 4 x 3 x 32 = 384 tiles of 256 x 256."""
    cfg, w16, bits, order = case("tiny_shared", F=4096, n_shared=4, E=12, T=600)
    say("shared experts: tiled shared range, T=600")
    L = gpu_layer(cfg, w16, bits, order)
    L.set_shared_experts(cfg.n_shared)
    O = oracle_layer(cfg, w16, bits)
    e16, e32 = _check(L, O, cfg, cfg.T, True, tokens=list(range(0, 600, 7)) + [599])
    assert e16 <= TOL16 and e32 <= TOL32, (e16, e32)
    L.close()


def test_shared_experts_after_downshift():
    """A shared expert's pages are lowered and committed like a routed one's."""
    import torch
    cfg, w16, bits, order = case("tiny_shared")
    L = gpu_layer(cfg, w16, bits, order, slack=0.5)
    L.set_shared_experts(cfg.n_shared)
    O = oracle_layer(cfg, w16, bits)
    blocks = [(e, p, rb) for e in range(cfg.E_routed, cfg.E) for p in range(3) for rb in range(cfg.nrb(p))
              if bits[p][e, rb] == 16]
    say("shared experts: downshift %d shared-expert pages to int4" % len(blocks))
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    L.requant(blocks, 4, stream=side)
    assert L.commit() == len(blocks)
    for (e, p, rb) in blocks:
        O.requant(p, e, rb, 4)
    torch.cuda.synchronize()
    L.reclaim()
    assert_all_pages_equal(L, O, cfg, blocks)
    e16, e32 = _check(L, O, cfg, 100, True)
    assert e16 <= TOL16 and e32 <= TOL32, (e16, e32)
    L.close()


def test_shared_argument_checks():
    import torch
    from paper_2607_16184_amd import pw
    cfg, w16, bits, order = case("tiny_shared")
    L = gpu_layer(cfg, w16, bits, order)
    say("shared experts: argument checks")
    with pytest.raises(pw.PWError) as ei:
        L.set_shared_experts(cfg.E)                 # no routed expert left
    assert ei.value.status == pw.PW_EINVAL
    L.set_shared_experts(cfg.n_shared)
    with pytest.raises(pw.PWError) as ei:           # K must count the shared columns too
        pw.pw_workspace_bytes(L.handle, 16, cfg.n_shared)
    assert ei.value.status == pw.PW_EINVAL
    with pytest.raises(pw.PWError) as ei:           # E + n_shared above 256
        pw.pw_route_topk_shared(256, 4, 250, 2, 1, 8, 0, 256, 256, 256, 256, 256,
                                torch.cuda.current_stream().cuda_stream)
    assert ei.value.status == pw.PW_EINVAL
    torch.cuda.synchronize()
    L.close()


def test_qwen_shared_full():
    """Qwen1.5-MoE-shaped layer (60 routed + 4 shared experts, top-4, 2048 /
    1408, 128 tokens, gated shared experts): every page byte and every token
    of the output. The routed experts run the decode kernels (9 slots per
    expert), the shared ones the streaming kernel (128 each: four experts
    would fill only 44 of the tiled kernel's 256 x 256 tiles)."""
    cfg, w16, bits, order = case("qwen_shared")
    say("shared experts: Qwen-shaped layer, build (%d pages)" % len(order))
    L = gpu_layer(cfg, w16, bits, order)
    L.set_shared_experts(cfg.n_shared)
    O = oracle_layer(cfg, w16, bits)
    assert assert_all_pages_equal(L, O, cfg) == len(order)
    say("shared experts: Qwen-shaped layer, forward and oracle on 128 tokens")
    e16, e32 = _check(L, O, cfg, cfg.T, True)
    assert e16 <= TOL16 and e32 <= TOL32, (e16, e32)
    L.close()
