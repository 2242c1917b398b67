"""ctypes binding of libpagedweight.so (C ABI in include/pw.h).

Argument marshalling only: every step of the hot path runs in the library's
HIP kernels. Functions keep the C names; pointers are integers (device
addresses, e.g. ``tensor.data_ptr()``) and streams are ``hipStream_t`` handles
as integers (``torch.cuda.current_stream().cuda_stream``). A non-OK status
raises :class:`PWError` carrying ``pw_last_error()``.

Importing this module loads the library and raises if it cannot be loaded;
there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from typing import Sequence, Tuple

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libpagedweight.so")

PW_OK, PW_EINVAL, PW_ENOMEM, PW_EBUSY, PW_EUNSUPPORTED, PW_EHIP, PW_ESTATE = range(7)
PW_F16, PW_BF16 = 0, 1
PW_GATE, PW_UP, PW_DOWN = 0, 1, 2
PW_PAGE_ABSENT, PW_PAGE_RESIDENT, PW_PAGE_REQUANT_PENDING, PW_PAGE_RELOAD_PENDING = 0, 1, 2, 3
PW_PH_GATEUP, PW_PH_DOWN, PW_PH_COMBINE, PW_PH_REQUANT, PW_NPHASE = 0, 1, 2, 3, 4


class pw_page_entry(ctypes.Structure):
    _fields_ = [("data_off", ctypes.c_uint64), ("sz_off", ctypes.c_uint64),
                ("bits", ctypes.c_uint8), ("state", ctypes.c_uint8),
                ("rsv", ctypes.c_uint16), ("gen", ctypes.c_uint32)]


class pw_layer_desc(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int) for n in ("E", "H", "F", "R", "G", "act", "sdt")]


class PWError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__("%s: %s" % (_status_name(status), msg))
        self.status = status


def _load():
    if not os.path.exists(LIB_PATH):
        from . import build as _build
        _build.build_all()
    L = ctypes.CDLL(LIB_PATH)
    vp, i32, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t
    P = ctypes.POINTER
    sig = {
        "pw_table_entries": (sz, [P(pw_layer_desc)]),
        "pw_page_bytes": (i32, [P(pw_layer_desc), i32, i32, P(sz)]),
        "pw_layer_create": (i32, [P(pw_layer_desc), vp, sz, vp, P(vp)]),
        "pw_layer_destroy": (i32, [vp]),
        "pw_layer_load_page": (i32, [vp, i32, i32, i32, i32, vp, vp]),
        "pw_route_topk": (i32, [vp, i32, i32, i32, i32, vp, vp, vp, vp, vp, vp]),
        "pw_workspace_bytes": (i32, [vp, i32, i32, P(sz)]),
        "pw_moe_paged_gemm": (i32, [vp, vp, i32, i32, vp, vp, vp, vp, vp, i32, vp, sz, vp]),
        "pw_requant_block": (i32, [vp, i32, i32, i32, i32, vp, P(sz)]),
        "pw_requant_blocks": (i32, [vp, i32, P(i32), P(i32), P(i32), P(i32), vp, P(sz)]),
        "pw_layer_set_host_pool": (i32, [vp, vp, sz]),
        "pw_offload_block": (i32, [vp, i32, i32, i32, vp]),
        "pw_offload_blocks": (i32, [vp, i32, P(i32), P(i32), P(i32), vp]),
        "pw_reload_block": (i32, [vp, i32, i32, i32, vp, P(sz)]),
        "pw_reload_blocks": (i32, [vp, i32, P(i32), P(i32), P(i32), vp, P(sz)]),
        "pw_drop_host_copy": (i32, [vp, i32, i32, i32]),
        "pw_host_copy_info": (i32, [vp, i32, i32, i32, P(i32), P(i32)]),
        "pw_host_pool_stats": (i32, [vp, P(sz), P(sz)]),
        "pw_commit": (i32, [vp, vp, P(i32)]),
        "pw_reclaim": (i32, [vp, P(sz)]),
        "pw_page_info": (i32, [vp, i32, i32, i32, P(pw_page_entry)]),
        "pw_pool_stats": (i32, [vp, P(sz), P(sz), P(sz)]),
        "pw_profile_enable": (i32, [vp, i32]),
        "pw_profile_read": (i32, [vp, P(ctypes.c_double), P(ctypes.c_int64), i32]),
        "pw_last_error": (ctypes.c_char_p, []),
        "pw_status_str": (ctypes.c_char_p, [i32]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(L, name)
        fn.restype = res
        fn.argtypes = args
    return L


_lib = _load()


def _status_name(s: int) -> str:
    return _lib.pw_status_str(s).decode()


def _check(status: int):
    if status != PW_OK:
        raise PWError(status, _lib.pw_last_error().decode())


def _desc(d) -> pw_layer_desc:
    if isinstance(d, pw_layer_desc):
        return d
    return pw_layer_desc(d.E, d.H, d.F, d.R, d.G, d.act, d.sdt)


# --------------------------------------------------------------------------
# C ABI, one wrapper per entry point
# --------------------------------------------------------------------------

def pw_table_entries(desc) -> int:
    return int(_lib.pw_table_entries(ctypes.byref(_desc(desc))))


def pw_page_bytes(desc, proj: int, bits: int) -> int:
    out = ctypes.c_size_t()
    _check(_lib.pw_page_bytes(ctypes.byref(_desc(desc)), proj, bits, ctypes.byref(out)))
    return out.value


def pw_layer_create(desc, pool_ptr: int, pool_bytes: int, table_ptr: int) -> int:
    h = ctypes.c_void_p()
    _check(_lib.pw_layer_create(ctypes.byref(_desc(desc)), pool_ptr, pool_bytes, table_ptr,
                                ctypes.byref(h)))
    return h.value


def pw_layer_destroy(layer: int):
    _check(_lib.pw_layer_destroy(layer))


def pw_layer_load_page(layer: int, e: int, proj: int, rb: int, bits: int, rows16_ptr: int, stream: int):
    _check(_lib.pw_layer_load_page(layer, e, proj, rb, bits, rows16_ptr, stream))


def pw_route_topk(logits_ptr: int, T: int, E: int, K: int, renorm: int, ids_ptr: int, w_ptr: int,
                  offsets_ptr: int, sorted_slot_ptr: int, slot_pos_ptr: int, stream: int):
    _check(_lib.pw_route_topk(logits_ptr, T, E, K, renorm, ids_ptr, w_ptr, offsets_ptr,
                              sorted_slot_ptr, slot_pos_ptr, stream))


def pw_workspace_bytes(layer: int, T: int, K: int) -> int:
    out = ctypes.c_size_t()
    _check(_lib.pw_workspace_bytes(layer, T, K, ctypes.byref(out)))
    return out.value


def pw_moe_paged_gemm(layer: int, x_ptr: int, T: int, K: int, w_ptr: int, offsets_ptr: int,
                      sorted_slot_ptr: int, slot_pos_ptr: int, y_ptr: int, out_fp32: int,
                      ws_ptr: int, ws_bytes: int, stream: int):
    _check(_lib.pw_moe_paged_gemm(layer, x_ptr, T, K, w_ptr, offsets_ptr, sorted_slot_ptr,
                                  slot_pos_ptr, y_ptr, out_fp32, ws_ptr, ws_bytes, stream))


def pw_requant_block(layer: int, e: int, proj: int, rb: int, new_bits: int, stream: int) -> int:
    d = ctypes.c_size_t()
    _check(_lib.pw_requant_block(layer, e, proj, rb, new_bits, stream, ctypes.byref(d)))
    return d.value


def pw_requant_blocks(layer: int, es: Sequence[int], projs: Sequence[int], rbs: Sequence[int],
                      new_bits: Sequence[int], stream: int) -> int:
    n = len(es)
    arr = ctypes.c_int * max(n, 1)
    d = ctypes.c_size_t()
    _check(_lib.pw_requant_blocks(layer, n, arr(*es), arr(*projs), arr(*rbs), arr(*new_bits),
                                  stream, ctypes.byref(d)))
    return d.value


def pw_layer_set_host_pool(layer: int, host_ptr: int, host_bytes: int):
    _check(_lib.pw_layer_set_host_pool(layer, host_ptr, host_bytes))


def pw_offload_block(layer: int, e: int, proj: int, rb: int, stream: int):
    _check(_lib.pw_offload_block(layer, e, proj, rb, stream))


def pw_offload_blocks(layer: int, es: Sequence[int], projs: Sequence[int], rbs: Sequence[int], stream: int):
    n = len(es)
    arr = ctypes.c_int * max(n, 1)
    _check(_lib.pw_offload_blocks(layer, n, arr(*es), arr(*projs), arr(*rbs), stream))


def pw_reload_block(layer: int, e: int, proj: int, rb: int, stream: int) -> int:
    d = ctypes.c_size_t()
    _check(_lib.pw_reload_block(layer, e, proj, rb, stream, ctypes.byref(d)))
    return d.value


def pw_reload_blocks(layer: int, es: Sequence[int], projs: Sequence[int], rbs: Sequence[int], stream: int) -> int:
    n = len(es)
    arr = ctypes.c_int * max(n, 1)
    d = ctypes.c_size_t()
    _check(_lib.pw_reload_blocks(layer, n, arr(*es), arr(*projs), arr(*rbs), stream, ctypes.byref(d)))
    return d.value


def pw_drop_host_copy(layer: int, e: int, proj: int, rb: int):
    _check(_lib.pw_drop_host_copy(layer, e, proj, rb))


def pw_host_copy_info(layer: int, e: int, proj: int, rb: int) -> Tuple[int, bool]:
    bits, ready = ctypes.c_int(), ctypes.c_int()
    _check(_lib.pw_host_copy_info(layer, e, proj, rb, ctypes.byref(bits), ctypes.byref(ready)))
    return bits.value, bool(ready.value)


def pw_host_pool_stats(layer: int) -> Tuple[int, int]:
    c, u = ctypes.c_size_t(), ctypes.c_size_t()
    _check(_lib.pw_host_pool_stats(layer, ctypes.byref(c), ctypes.byref(u)))
    return c.value, u.value


def pw_commit(layer: int, stream: int) -> int:
    n = ctypes.c_int()
    _check(_lib.pw_commit(layer, stream, ctypes.byref(n)))
    return n.value


def pw_reclaim(layer: int) -> int:
    b = ctypes.c_size_t()
    _check(_lib.pw_reclaim(layer, ctypes.byref(b)))
    return b.value


def pw_page_info(layer: int, e: int, proj: int, rb: int) -> pw_page_entry:
    out = pw_page_entry()
    _check(_lib.pw_page_info(layer, e, proj, rb, ctypes.byref(out)))
    return out


def pw_pool_stats(layer: int) -> Tuple[int, int, int]:
    u, f, l = ctypes.c_size_t(), ctypes.c_size_t(), ctypes.c_size_t()
    _check(_lib.pw_pool_stats(layer, ctypes.byref(u), ctypes.byref(f), ctypes.byref(l)))
    return u.value, f.value, l.value


def pw_profile_enable(layer: int, on: bool):
    _check(_lib.pw_profile_enable(layer, int(bool(on))))


def pw_profile_read(layer: int, reset: bool = True):
    ms = (ctypes.c_double * PW_NPHASE)()
    cnt = (ctypes.c_int64 * PW_NPHASE)()
    _check(_lib.pw_profile_read(layer, ms, cnt, int(bool(reset))))
    return list(ms), list(cnt)


def pw_last_error() -> str:
    return _lib.pw_last_error().decode()
