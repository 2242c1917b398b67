"""The allocation-free forward (pw_moe_paged_gemm_noalloc): the workspace
comes from the library's static device array instead of the caller's. Its
output must equal the workspace entry point's bit for bit (same kernels, same
summation order) and match the oracle to the parity bar, on two calls in a
row, the second with fewer tokens than the first, so the second call runs on
what the first left in the array."""
import numpy as np
import pytest

import oracle
from helpers import case, gpu_layer, oracle_layer, rel_err, say, to_dev, to_dev16, y16_values
from paper_2607_16184_amd import pw, synth

pytestmark = pytest.mark.gpu

TOL16, TOL32 = 2e-2, 1e-3


def _noalloc(L, x, routing, out_fp32):
    import torch
    ids, w, offsets, ss, sp = routing
    T, K = ids.shape
    y = torch.empty((T, L.cfg.H), dtype=torch.float32 if out_fp32 else torch.int16, device=x.device)
    pw.pw_moe_paged_gemm_noalloc(L.handle, x.data_ptr(), T, K, w.data_ptr(), offsets.data_ptr(), ss.data_ptr(),
                                 sp.data_ptr(), y.data_ptr(), int(out_fp32),
                                 torch.cuda.current_stream().cuda_stream)
    return y


def _check(L, O, cfg, T):
    import torch
    logits = synth.logits(cfg, T=T)
    x16 = synth.activations(cfg, T=T)
    routing = L.route(to_dev(logits), cfg.K)
    x = to_dev16(x16)
    y32n = _noalloc(L, x, routing, True)
    y16n = _noalloc(L, x, routing, False)
    y32 = L.forward(x, routing, out_fp32=True)
    y16 = L.forward(x, routing)
    torch.cuda.synchronize()
    assert torch.equal(y32n, y32) and torch.equal(y16n, y16)
    ids, w = oracle.route(logits, cfg.K)
    r1 = O.forward(x16, ids, w, h_round=False)
    r2 = O.forward(x16, ids, w, h_round=True)
    e16 = rel_err(y16_values(y16n, cfg.act), r1)
    e32 = rel_err(y32n.cpu().numpy(), r2)
    assert e16 <= TOL16 and e32 <= TOL32, (T, e16, e32)


def test_noalloc_matches_workspace_entry_point():
    import torch
    cfg, w16, bits, order = case("tiny")
    L = gpu_layer(cfg, w16, bits, order)
    O = oracle_layer(cfg, w16, bits)
    # 300 tokens (600 slots, 75 per expert: streaming kernel), then 16 tokens
    # (decode kernels, split down projection) on what the first call left
    for T in (300, 16):
        say("no-alloc forward: tiny layer, T=%d" % T)
        _check(L, O, cfg, T)
    L.close()


def test_noalloc_refuses_oversized_calls():
    import torch
    cfg, w16, bits, order = case("tiny")
    L = gpu_layer(cfg, w16, bits, order)
    T = 40000     # 80000 slots: 2 KiB of workspace each, above 64 MiB
    assert pw.pw_workspace_bytes(L.handle, T, cfg.K) > 64 << 20
    say("no-alloc forward: oversized call is refused")
    with pytest.raises(pw.PWError) as ei:
        pw.pw_moe_paged_gemm_noalloc(L.handle, 256, T, cfg.K, 256, 256, 256, 256, 256, 1,
                                     torch.cuda.current_stream().cuda_stream)
    assert ei.value.status == pw.PW_ENOMEM
    assert "static scratch" in pw.pw_last_error()
    torch.cuda.synchronize()
    L.close()
