"""The ceiling probes run through the C ABI: every read workgroup completes,
bad arguments are rejected, and the MFMA probe's result is finite and the
same in every workgroup (its operands are the same constants)."""
import numpy as np
import pytest

from helpers import say

pytestmark = pytest.mark.gpu


def test_read_probe_covers_every_workgroup():
    import torch
    from paper_2607_16184_amd import pw
    nblk, nbytes = 64, 64 * 32768 * 3
    say("read probe %d bytes, %d workgroups" % (nbytes, nblk))
    buf = torch.ones(nbytes, dtype=torch.uint8, device="cuda")
    out = torch.zeros(2 * nblk, dtype=torch.int32, device="cuda")
    pw.pw_probe_read(buf.data_ptr(), nbytes, nblk, out.data_ptr(), torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    assert out[nblk:].cpu().numpy().tolist() == [1] * nblk


def test_probe_argument_errors():
    import torch
    from paper_2607_16184_amd import pw
    buf = torch.ones(32768, dtype=torch.uint8, device="cuda")
    out = torch.zeros(4, dtype=torch.int32, device="cuda")
    st = torch.cuda.current_stream().cuda_stream
    with pytest.raises(RuntimeError):
        pw.pw_probe_read(buf.data_ptr(), 1000, 1, out.data_ptr(), st)      # not a multiple of 32768
    with pytest.raises(RuntimeError):
        pw.pw_probe_mfma(0, 1, out.data_ptr(), st)                           # iters < 1


def test_mfma_probe_value():
    import torch
    from paper_2607_16184_amd import pw
    iters, nblk = 3, 2
    say("MFMA probe iters=%d" % iters)
    out = torch.zeros(nblk, dtype=torch.float32, device="cuda")
    pw.pw_probe_mfma(iters, nblk, out.data_ptr(), torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    v = out.cpu().numpy()
    assert np.all(np.isfinite(v)) and np.all(v > 0)
    assert v[0] == v[1]
