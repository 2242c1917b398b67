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

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libpagedweight.so")

PW_OK, PW_EINVAL, PW_ENOMEM, PW_EBUSY, PW_EUNSUPPORTED, PW_EHIP, PW_ESTATE = range(7)
PW_F16, PW_BF16 = 0, 1
PW_GATE, PW_UP, PW_DOWN = 0, 1, 2
PW_PAGE_ABSENT, PW_PAGE_RESIDENT, PW_PAGE_REQUANT_PENDING, PW_PAGE_RELOAD_PENDING = 0, 1, 2, 3
PW_PH_GATEUP, PW_PH_DOWN, PW_PH_COMBINE, PW_PH_REQUANT, PW_PH_GEMM, PW_NPHASE = 0, 1, 2, 3, 4, 5


class pw_page_entry(ctypes.Structure):
    _fields_ = [("data_off", ctypes.c_uint64), ("sz_off", ctypes.c_uint64),
                ("bits", ctypes.c_uint8), ("state", ctypes.c_uint8),
                ("rsv", ctypes.c_uint16), ("gen", ctypes.c_uint32)]


class pw_layer_desc(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int) for n in ("E", "H", "F", "R", "G", "act", "sdt")]


PW_FMT_RTN, PW_FMT_APL = 0, 1
PW_PLAN_MAX_BUCKETS = 8
PW_PLAN_MAX_STAGES = 8


class pw_planner_config(ctypes.Structure):
    _fields_ = [("n_buckets", ctypes.c_int),
                ("bucket_frac", ctypes.c_double * PW_PLAN_MAX_BUCKETS),
                ("mult", ctypes.c_double * PW_PLAN_MAX_BUCKETS),
                ("n_stages", ctypes.c_int),
                ("floor_bits", (ctypes.c_int * PW_PLAN_MAX_BUCKETS) * PW_PLAN_MAX_STAGES),
                ("alpha", ctypes.c_double), ("rho_min", ctypes.c_double), ("rho_max", ctypes.c_double),
                ("eps", ctypes.c_double),
                ("head_w", ((ctypes.c_double * 3) * 2) * 2),
                ("head_a", (ctypes.c_double * 2) * 2),
                ("head_c", (ctypes.c_double * 2) * 2)]


class pw_plan_summary(ctypes.Structure):
    _fields_ = [("target", ctypes.c_uint64), ("bytes", ctypes.c_uint64), ("damage", ctypes.c_double),
                ("triggered", ctypes.c_int), ("stage", ctypes.c_int), ("n_steps", ctypes.c_int),
                ("n_units", ctypes.c_int)]


class PWError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__("%s: %s" % (_status_name(status), msg))
        self.status = status


def _load():
    # The library binds to whatever HIP runtime the process has loaded. PyTorch
    # ships its own copy: load it first, so the library and PyTorch share one
    # runtime (two runtimes in one process do not both reach the device).
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
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
        "pw_probe_read": (i32, [vp, sz, i32, vp, vp]),
        "pw_probe_mfma": (i32, [i32, i32, vp, vp]),
        "pw_workspace_bytes": (i32, [vp, i32, i32, P(sz)]),
        "pw_moe_paged_gemm": (i32, [vp, vp, i32, i32, vp, vp, vp, vp, vp, i32, vp, sz, vp]),
        "pw_layer_set_shared_experts": (i32, [vp, i32]),
        "pw_layer_set_chains": (i32, [vp, i32]),
        "pw_route_topk_shared": (i32, [vp, i32, i32, i32, i32, i32, vp, vp, vp, vp, vp, vp, vp]),
        "pw_moe_paged_gemm_noalloc": (i32, [vp, vp, i32, i32, vp, vp, vp, vp, vp, i32, vp]),
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
        "pw_apl_workspace_bytes": (i32, [vp, i32, P(sz)]),
        "pw_layer_load_pages_apl": (i32, [vp, i32, P(i32), P(i32), P(i32), P(i32), P(vp), vp, sz, vp]),
        "pw_routing_stats": (i32, [vp, i32, i32, i32, i32, vp, vp, vp, i32, i32, i32, vp, vp, i32, vp]),
        "pw_planner_create": (i32, [i32, i32, P(i32), P(i32), P(ctypes.c_uint64), P(ctypes.c_double),
                                    P(pw_planner_config), P(vp)]),
        "pw_planner_destroy": (None, [vp]),
        "pw_planner_add_request": (i32, [vp, P(ctypes.c_double), P(ctypes.c_double), ctypes.c_double]),
        "pw_planner_clear_requests": (i32, [vp]),
        "pw_planner_step": (i32, [vp, P(i32), i32, i32, ctypes.c_uint64, P(pw_plan_summary)]),
        "pw_planner_plan": (i32, [vp, i32, i32, i32, P(i32), P(i32), P(i32), P(ctypes.c_uint64), P(i32)]),
        "pw_planner_create_for_layer": (i32, [vp, P(ctypes.c_double), P(pw_planner_config), P(vp)]),
        "pw_planner_step_layer": (i32, [vp, vp, i32, i32, ctypes.c_uint64, P(pw_plan_summary)]),
        "pw_planner_apply": (i32, [vp, vp, vp, P(sz)]),
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


def pw_probe_read(buf_ptr: int, nbytes: int, nblocks: int, out_ptr: int, stream: int):
    _check(_lib.pw_probe_read(buf_ptr, nbytes, nblocks, out_ptr, stream))


def pw_probe_mfma(iters: int, nblocks: int, out_ptr: int, stream: int):
    _check(_lib.pw_probe_mfma(iters, nblocks, out_ptr, stream))


def pw_workspace_bytes(layer: int, T: int, K: int) -> int:
    out = ctypes.c_size_t()
    _check(_lib.pw_workspace_bytes(layer, T, K, ctypes.byref(out)))
    return out.value


def pw_moe_paged_gemm(layer: int, x_ptr: int, T: int, K: int, w_ptr: int, offsets_ptr: int,
                      sorted_slot_ptr: int, slot_pos_ptr: int, y_ptr: int, out_fp32: int,
                      ws_ptr: int, ws_bytes: int, stream: int):
    _check(_lib.pw_moe_paged_gemm(layer, x_ptr, T, K, w_ptr, offsets_ptr, sorted_slot_ptr,
                                  slot_pos_ptr, y_ptr, out_fp32, ws_ptr, ws_bytes, stream))


def pw_layer_set_shared_experts(layer: int, n_shared: int):
    _check(_lib.pw_layer_set_shared_experts(layer, n_shared))


def pw_layer_set_chains(layer: int, chains: int):
    _check(_lib.pw_layer_set_chains(layer, chains))


def pw_route_topk_shared(logits_ptr: int, T: int, E: int, K: int, renorm: int, n_shared: int, gate_ptr: int,
                         ids_ptr: int, w_ptr: int, offsets_ptr: int, sorted_slot_ptr: int, slot_pos_ptr: int,
                         stream: int):
    _check(_lib.pw_route_topk_shared(logits_ptr, T, E, K, renorm, n_shared, gate_ptr or None, ids_ptr, w_ptr,
                                     offsets_ptr, sorted_slot_ptr, slot_pos_ptr, stream))


def pw_moe_paged_gemm_noalloc(layer: int, x_ptr: int, T: int, K: int, w_ptr: int, offsets_ptr: int,
                              sorted_slot_ptr: int, slot_pos_ptr: int, y_ptr: int, out_fp32: int,
                              stream: int):
    _check(_lib.pw_moe_paged_gemm_noalloc(layer, x_ptr, T, K, w_ptr, offsets_ptr, sorted_slot_ptr,
                                          slot_pos_ptr, y_ptr, out_fp32, stream))


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


# --------------------------------------------------------------------------
# routing statistics and the runtime planner (Sec. 3.2, Alg. 1)
# --------------------------------------------------------------------------

def pw_routing_stats(rows_ptr: int, act: int, n_rows: int, dim: int, rows_by_position: int, w_ptr: int,
                     offsets_ptr: int, sorted_slot_ptr: int, T: int, E: int, K: int, norm2_ptr: int,
                     stats_ptr: int, accumulate: int, stream: int):
    _check(_lib.pw_routing_stats(rows_ptr, act, n_rows, dim, rows_by_position, w_ptr, offsets_ptr,
                                 sorted_slot_ptr, T, E, K, norm2_ptr, stats_ptr, accumulate, stream))


def planner_config(bucket_frac, mult, floors, alpha=1.0, rho_min=-1.0, rho_max=1.0, eps=1e-9,
                   head_w=None, head_a=None, head_c=None) -> pw_planner_config:
    """Fills a pw_planner_config; floors is [stage][bucket]; head_* indexed [u][step]."""
    c = pw_planner_config()
    c.n_buckets = len(bucket_frac)
    c.n_stages = len(floors)
    for j, (f, m) in enumerate(zip(bucket_frac, mult)):
        c.bucket_frac[j] = float(f)
        c.mult[j] = float(m)
    for s_, row in enumerate(floors):
        for j, b in enumerate(row):
            c.floor_bits[s_][j] = int(b)
    c.alpha, c.rho_min, c.rho_max, c.eps = float(alpha), float(rho_min), float(rho_max), float(eps)
    for u in range(2):
        for t in range(2):
            for k in range(3):
                c.head_w[u][t][k] = 0.0 if head_w is None else float(head_w[u][t][k])
            c.head_a[u][t] = 0.0 if head_a is None else float(head_a[u][t])
            c.head_c[u][t] = 1.0 if head_c is None else float(head_c[u][t])
    return c


def _dp(a):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def pw_planner_create(n_experts: int, unit_expert, unit_type, unit_bytes, unit_sens, cfg) -> int:
    ue = np.ascontiguousarray(unit_expert, np.int32)
    ut = np.ascontiguousarray(unit_type, np.int32)
    ub = np.ascontiguousarray(unit_bytes, np.uint64).reshape(-1)
    us = np.ascontiguousarray(unit_sens, np.float64).reshape(-1)
    h = ctypes.c_void_p()
    _check(_lib.pw_planner_create(n_experts, len(ue), ue.ctypes.data_as(ctypes.POINTER(ctypes.c_int)),
                                  ut.ctypes.data_as(ctypes.POINTER(ctypes.c_int)),
                                  ub.ctypes.data_as(ctypes.POINTER(ctypes.c_uint64)), _dp(us),
                                  ctypes.byref(cfg), ctypes.byref(h)))
    return h.value


def pw_planner_destroy(p: int):
    _lib.pw_planner_destroy(p)


def pw_planner_add_request(p: int, stats_gate_up, stats_down, kv_weight: float):
    sg = np.ascontiguousarray(stats_gate_up, np.float64)
    sd = None if stats_down is None else np.ascontiguousarray(stats_down, np.float64)
    _check(_lib.pw_planner_add_request(p, _dp(sg), None if sd is None else _dp(sd), float(kv_weight)))


def pw_planner_clear_requests(p: int):
    _check(_lib.pw_planner_clear_requests(p))


def pw_planner_step(p: int, unit_bits, free_blocks: int, free_threshold: int, kv_block_bytes: int) -> pw_plan_summary:
    q = np.ascontiguousarray(unit_bits, np.int32)
    out = pw_plan_summary()
    _check(_lib.pw_planner_step(p, q.ctypes.data_as(ctypes.POINTER(ctypes.c_int)), free_blocks, free_threshold,
                                kv_block_bytes, ctypes.byref(out)))
    return out


def pw_planner_plan(p: int, stage: int = -1, steps: bool = False):
    """[(unit, from_bits, to_bits, bytes)] of a stage's plan (-1: the selected one)."""
    n = ctypes.c_int()
    _check(_lib.pw_planner_plan(p, stage, int(steps), 0, None, None, None, None, ctypes.byref(n)))
    m = n.value
    u, f, t = (np.zeros(max(m, 1), np.int32) for _ in range(3))
    b = np.zeros(max(m, 1), np.uint64)
    ip = lambda a: a.ctypes.data_as(ctypes.POINTER(ctypes.c_int))
    _check(_lib.pw_planner_plan(p, stage, int(steps), m, ip(u), ip(f), ip(t),
                                b.ctypes.data_as(ctypes.POINTER(ctypes.c_uint64)), ctypes.byref(n)))
    return [(int(u[k]), int(f[k]), int(t[k]), int(b[k])) for k in range(m)]


def pw_planner_create_for_layer(layer: int, sens, cfg) -> int:
    s_ = np.ascontiguousarray(sens, np.float64).reshape(-1)
    h = ctypes.c_void_p()
    _check(_lib.pw_planner_create_for_layer(layer, _dp(s_), ctypes.byref(cfg), ctypes.byref(h)))
    return h.value


def pw_planner_step_layer(p: int, layer: int, free_blocks: int, free_threshold: int,
                          kv_block_bytes: int) -> pw_plan_summary:
    out = pw_plan_summary()
    _check(_lib.pw_planner_step_layer(p, layer, free_blocks, free_threshold, kv_block_bytes, ctypes.byref(out)))
    return out


def pw_planner_apply(p: int, layer: int, stream: int) -> int:
    d = ctypes.c_size_t()
    _check(_lib.pw_planner_apply(p, layer, stream, ctypes.byref(d)))
    return d.value


# --------------------------------------------------------------------------
# nested bit-plane pages
# --------------------------------------------------------------------------

def pw_apl_workspace_bytes(layer: int, n: int) -> int:
    out = ctypes.c_size_t()
    _check(_lib.pw_apl_workspace_bytes(layer, n, ctypes.byref(out)))
    return out.value


def pw_layer_load_pages_apl(layer: int, es, projs, rbs, bits, row_ptrs, ws_ptr: int, ws_bytes: int, stream: int):
    n = len(es)
    arr = ctypes.c_int * max(n, 1)
    ptrs = (ctypes.c_void_p * max(n, 1))(*row_ptrs)
    _check(_lib.pw_layer_load_pages_apl(layer, n, arr(*es), arr(*projs), arr(*rbs), arr(*bits), ptrs, ws_ptr,
                                        ws_bytes, stream))
