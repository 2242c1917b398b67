"""The C-ABI library loads and exports every entry point that include/pw.h
declares; host-only calls answer without a GPU."""
import ctypes
import os
import re

import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "pw.h")


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(pw_[a-z0-9_]+)\s*\(", src)))


def test_header_declares_the_boundary():
    names = _declared()
    for n in ("pw_route_topk", "pw_moe_paged_gemm", "pw_requant_block", "pw_commit",
              "pw_reclaim", "pw_layer_create", "pw_layer_load_page"):
        assert n in names


def test_library_exports_every_declared_symbol():
    from paper_2607_16184_amd import pw
    lib = ctypes.CDLL(pw.LIB_PATH)
    missing = [n for n in _declared() if not hasattr(lib, n)]
    assert not missing, missing


def test_page_bytes_match_eq3():
    from paper_2607_16184_amd import pw
    for (E, H, F, R, G) in [(8, 4096, 14336, 128, 128), (64, 2048, 1408, 64, 128), (8, 256, 512, 64, 64)]:
        d = pw.pw_layer_desc(E, H, F, R, G, pw.PW_BF16, pw.PW_BF16)
        assert pw.pw_table_entries(d) == E * 3 * max(F, H) // R
        for proj, K in ((pw.PW_GATE, H), (pw.PW_UP, H), (pw.PW_DOWN, F)):
            for b in (16, 8, 4):
                assert pw.pw_page_bytes(d, proj, b) == oracle.page_bytes(R, K, G, b)


def test_host_validation_without_gpu():
    from paper_2607_16184_amd import pw
    with pytest.raises(pw.PWError) as ei:
        pw.pw_route_topk(0, 4, 8, 9, 1, 0, 0, 0, 0, 0, 0)        # K > E
    assert ei.value.status == pw.PW_EINVAL
    with pytest.raises(pw.PWError) as ei:
        pw.pw_page_bytes(pw.pw_layer_desc(8, 256, 500, 64, 64, 0, 0), 0, 16)   # F % R
    assert ei.value.status == pw.PW_EINVAL
    with pytest.raises(pw.PWError):
        pw.pw_page_bytes(pw.pw_layer_desc(8, 256, 512, 64, 64, 0, 0), 0, 5)
    with pytest.raises(pw.PWError) as ei:
        pw.pw_layer_create(pw.pw_layer_desc(8, 256, 512, 64, 64, 0, 0), 0, 0, 0)
    assert ei.value.status == pw.PW_EINVAL
    assert "null" in pw.pw_last_error()


@pytest.mark.parametrize("G", [32, 96, 192, 384, 1024])
def test_group_size_outside_the_kernels_set_is_refused(G):
    """The kernels index groups with shifts and masks: only G = 64, 128, 256,
    512 are accepted; any other value is refused before a layer exists."""
    from paper_2607_16184_amd import pw
    d = pw.pw_layer_desc(8, 3072, 6144, 128, G, pw.PW_BF16, pw.PW_BF16)
    with pytest.raises(pw.PWError) as ei:
        pw.pw_page_bytes(d, pw.PW_GATE, 8)
    assert ei.value.status == pw.PW_EINVAL
    assert "G must be" in pw.pw_last_error()


@pytest.mark.parametrize("G", [64, 128, 256, 512])
def test_power_of_two_group_sizes_are_accepted(G):
    from paper_2607_16184_amd import pw
    d = pw.pw_layer_desc(8, 3072, 6144, 128, G, pw.PW_BF16, pw.PW_BF16)
    assert pw.pw_page_bytes(d, pw.PW_GATE, 4) == oracle.page_bytes(128, 3072, G, 4)
