"""Device buffers around the C ABI: a paged layer held in torch memory.

PyTorch supplies device memory and streams only. Every computation (quantize,
route, GEMM, combine, requant, commit) is a call into libpagedweight.so.
"""
from __future__ import annotations

from typing import Dict, Iterable, List, Optional, Sequence, Tuple

import numpy as np
import torch

from . import pw
from .synth import DOWN, GATE, UP, LayerConfig

ENTRY_BYTES = 24


def _stream(s: Optional[torch.cuda.Stream] = None) -> int:
    return (s or torch.cuda.current_stream()).cuda_stream


def _aligned_empty(nbytes: int, device, align: int = 256) -> Tuple[torch.Tensor, int]:
    """A uint8 device buffer and the first address in it aligned to ``align``."""
    t = torch.empty(nbytes + align, dtype=torch.uint8, device=device)
    p = t.data_ptr()
    return t, (p + align - 1) // align * align


class PagedLayer:
    """One MoE layer whose expert weights live as pages in a device pool."""

    def __init__(self, cfg: LayerConfig, pool_bytes: int, device="cuda"):
        self.cfg = cfg
        self.device = torch.device(device)
        self.desc = pw.pw_layer_desc(cfg.E, cfg.H, cfg.F, cfg.R, cfg.G, cfg.act, cfg.sdt)
        self.pool_bytes = int(pool_bytes)
        self._pool_t, self.pool_ptr = _aligned_empty(self.pool_bytes, self.device)
        self.n_entries = pw.pw_table_entries(self.desc)
        self._table_t, self.table_ptr = _aligned_empty(self.n_entries * ENTRY_BYTES, self.device)
        torch.cuda.synchronize(self.device)
        self.handle = pw.pw_layer_create(self.desc, self.pool_ptr, self.pool_bytes, self.table_ptr)
        self._ws = None
        self._ws_ptr = 0
        self._ws_bytes = 0

    # -- construction ------------------------------------------------------
    @staticmethod
    def pool_bytes_for(cfg: LayerConfig, bits: Sequence[np.ndarray], slack: float = 0.0) -> int:
        tot = 0
        for p in (GATE, UP, DOWN):
            for b in np.asarray(bits[p]).ravel():
                tot += (pw.pw_page_bytes(cfg, p, int(b)) + 255) // 256 * 256
        return int(tot * (1.0 + slack)) + 256

    def load_pages(self, w16: Sequence[np.ndarray], bits: Sequence[np.ndarray],
                   order: Iterable[Tuple[int, int, int]], stream=None):
        """Upload the 16-bit weights and place every page at its bitwidth.

        ``w16[p]`` is the [E, rows, cols] uint16 array of projection p; pages
        are placed in ``order`` (which fixes their pool addresses).
        """
        st = _stream(stream)
        cfg = self.cfg
        dev = []
        for p in (GATE, UP, DOWN):
            dev.append(torch.from_numpy(np.ascontiguousarray(w16[p]).view(np.int16)).to(self.device))
        for (e, p, rb) in order:
            rows, cols = w16[p].shape[1:]
            off = ((e * rows + rb * cfg.R) * cols) * 2
            pw.pw_layer_load_page(self.handle, e, p, rb, int(bits[p][e, rb]), dev[p].data_ptr() + off, st)
        torch.cuda.current_stream().synchronize() if stream is None else stream.synchronize()
        del dev

    def load_pages_apl(self, w16: Sequence[np.ndarray], pages: Iterable[Tuple[int, int, int, int]],
                       stream=None):
        """Quantize blocks into nested bit-plane pages: pages = [(e, p, rb, bits)]
        with bits 8 or 4, placed in that order (pw_layer_load_pages_apl)."""
        st = _stream(stream)
        cfg = self.cfg
        pages = list(pages)
        if not pages:
            return
        dev = [torch.from_numpy(np.ascontiguousarray(w16[p]).view(np.int16)).to(self.device) for p in (GATE, UP, DOWN)]
        chunk = 32
        ws_bytes = pw.pw_apl_workspace_bytes(self.handle, min(chunk, len(pages)))
        ws_t, ws_ptr = _aligned_empty(ws_bytes, self.device)
        for i in range(0, len(pages), chunk):
            part = pages[i:i + chunk]
            ptrs = []
            for (e, p, rb, b) in part:
                rows, cols = w16[p].shape[1:]
                ptrs.append(dev[p].data_ptr() + ((e * rows + rb * cfg.R) * cols) * 2)
            es, ps, rbs, bs = zip(*part)
            pw.pw_layer_load_pages_apl(self.handle, list(es), list(ps), list(rbs), list(bs), ptrs, ws_ptr,
                                       ws_bytes, st)
        torch.cuda.current_stream().synchronize() if stream is None else stream.synchronize()
        del dev, ws_t

    # -- hot path ------------------------------------------------------------
    @staticmethod
    def routing_buffers(T: int, E: int, K: int, device="cuda"):
        """(ids [T,K], w [T,K], offsets [E+1], sorted_slot [S], slot_pos [S])."""
        return (torch.empty((T, K), dtype=torch.int32, device=device),
                torch.empty((T, K), dtype=torch.float32, device=device),
                torch.empty(E + 1, dtype=torch.int32, device=device),
                torch.empty(max(T * K, 1), dtype=torch.int32, device=device),
                torch.empty(max(T * K, 1), dtype=torch.int32, device=device))

    def route(self, logits: torch.Tensor, K: int, renorm: int = 1, stream=None, out=None):
        T, E = logits.shape
        ids, w, offsets, ss, sp = out if out is not None else self.routing_buffers(T, E, K, logits.device)
        pw.pw_route_topk(logits.data_ptr(), T, E, K, renorm, ids.data_ptr(), w.data_ptr(),
                         offsets.data_ptr(), ss.data_ptr(), sp.data_ptr(), _stream(stream))
        return ids, w, offsets, ss, sp

    def set_shared_experts(self, n_shared: int):
        """Declare the layer's last n_shared experts as shared experts."""
        pw.pw_layer_set_shared_experts(self.handle, n_shared)
        self.n_shared = n_shared

    def set_chains(self, chains: int):
        """1 or 2 concurrent expert chains for decode-sized GEMM calls."""
        pw.pw_layer_set_chains(self.handle, chains)

    def route_shared(self, logits: torch.Tensor, K: int, n_shared: int, gate: torch.Tensor = None,
                     renorm: int = 1, stream=None, out=None):
        """Routed top-K over logits [T, E_routed] plus n_shared shared columns
        (weights from gate [T, n_shared] fp32, or 1): [T, K + n_shared] routing."""
        T, E = logits.shape
        Kt = K + n_shared
        ids, w, offsets, ss, sp = out if out is not None else self.routing_buffers(T, E + n_shared, Kt,
                                                                                   logits.device)
        pw.pw_route_topk_shared(logits.data_ptr(), T, E, K, renorm, n_shared,
                                gate.data_ptr() if gate is not None else 0, ids.data_ptr(), w.data_ptr(),
                                offsets.data_ptr(), ss.data_ptr(), sp.data_ptr(), _stream(stream))
        return ids, w, offsets, ss, sp

    def workspace(self, T: int, K: int) -> Tuple[int, int]:
        need = pw.pw_workspace_bytes(self.handle, T, K)
        if need > self._ws_bytes:
            self._ws, self._ws_ptr = _aligned_empty(need, self.device)
            self._ws_bytes = need
        return self._ws_ptr, self._ws_bytes

    def forward(self, x: torch.Tensor, routing, out_fp32: bool = False, y: torch.Tensor = None,
                stream=None) -> torch.Tensor:
        ids, w, offsets, ss, sp = routing
        T, K = ids.shape
        if y is None:
            y = torch.empty((T, self.cfg.H), dtype=torch.float32 if out_fp32 else torch.int16,
                            device=x.device)
        ws_ptr, ws_bytes = self.workspace(T, K)
        pw.pw_moe_paged_gemm(self.handle, x.data_ptr(), T, K, w.data_ptr(), offsets.data_ptr(),
                             ss.data_ptr(), sp.data_ptr(), y.data_ptr(), int(out_fp32),
                             ws_ptr, ws_bytes, _stream(stream))
        return y

    # -- planner observations (Sec. 3.2) ------------------------------------
    def routing_stats(self, rows: torch.Tensor, routing, rows_by_position: bool = False,
                      out: torch.Tensor = None, accumulate: bool = False, stream=None) -> torch.Tensor:
        """[E, 5] float64 routing statistics of one step (pw_routing_stats):
        rows = x [T, H] (gate/up input, one row per token) or the SwiGLU rows
        [T K, F] in expert-major slot order (down input, rows_by_position)."""
        ids, w, offsets, ss, _ = routing
        T, K = ids.shape
        if out is None:
            out = torch.zeros((self.cfg.E, 5), dtype=torch.float64, device=rows.device)
        norm2 = torch.empty(max(rows.shape[0], 1), dtype=torch.float64, device=rows.device)
        pw.pw_routing_stats(rows.data_ptr(), self.cfg.act, rows.shape[0], rows.shape[1], int(rows_by_position),
                            w.data_ptr(), offsets.data_ptr(), ss.data_ptr(), T, self.cfg.E, K, norm2.data_ptr(),
                            out.data_ptr(), int(accumulate), _stream(stream))
        return out

    def hidden_rows(self, T: int, K: int) -> torch.Tensor:
        """The SwiGLU output of the last forward, [T K, F] 16-bit, expert-major
        slot order (a view of the workspace)."""
        self.workspace(T, K)
        off = self._ws_ptr - self._ws.data_ptr()
        n = T * K * self.cfg.F
        return self._ws[off:off + 2 * n].view(torch.int16).view(T * K, self.cfg.F)

    def planner(self, sens: np.ndarray, cfg) -> "Planner":
        """A runtime planner over this layer's table entries (sens: [entries, 3])."""
        return Planner(pw.pw_planner_create_for_layer(self.handle, sens, cfg))

    # -- runtime downshift -------------------------------------------------
    def requant(self, blocks: Sequence[Tuple[int, int, int]], new_bits: int, stream=None) -> int:
        if not blocks:
            return 0
        es, ps, rbs = zip(*blocks)
        return pw.pw_requant_blocks(self.handle, list(es), list(ps), list(rbs),
                                    [new_bits] * len(blocks), _stream(stream))

    # -- host copies (offload / reload) ---------------------------------------
    def set_host_pool(self, host_bytes: int):
        """Give the layer a pinned host pool of ``host_bytes`` for page copies."""
        self._host_t = torch.empty(int(host_bytes) + 256, dtype=torch.uint8, pin_memory=True)
        p = self._host_t.data_ptr()
        self.host_ptr = (p + 255) // 256 * 256
        pw.pw_layer_set_host_pool(self.handle, self.host_ptr, int(host_bytes))

    def offload(self, blocks: Sequence[Tuple[int, int, int]], stream=None):
        if not blocks:
            return
        es, ps, rbs = zip(*blocks)
        pw.pw_offload_blocks(self.handle, list(es), list(ps), list(rbs), _stream(stream))

    def reload(self, blocks: Sequence[Tuple[int, int, int]], stream=None) -> int:
        if not blocks:
            return 0
        es, ps, rbs = zip(*blocks)
        return pw.pw_reload_blocks(self.handle, list(es), list(ps), list(rbs), _stream(stream))

    def drop_host_copy(self, e: int, p: int, rb: int):
        pw.pw_drop_host_copy(self.handle, e, p, rb)

    def host_copy_info(self, e: int, p: int, rb: int):
        return pw.pw_host_copy_info(self.handle, e, p, rb)

    def host_pool_stats(self):
        return pw.pw_host_pool_stats(self.handle)

    def commit(self, stream=None) -> int:
        return pw.pw_commit(self.handle, _stream(stream))

    def reclaim(self) -> int:
        return pw.pw_reclaim(self.handle)

    # -- inspection --------------------------------------------------------
    def entry(self, e: int, p: int, rb: int) -> pw.pw_page_entry:
        return pw.pw_page_info(self.handle, e, p, rb)

    def page_image(self, e: int, p: int, rb: int) -> np.ndarray:
        """The page's bytes as stored in the pool (host copy)."""
        ent = self.entry(e, p, rb)
        if ent.rsv & 0xFF == pw.PW_FMT_APL:
            R, K = self.cfg.R, (self.cfg.F if p == DOWN else self.cfg.H)
            n = R * K * int(ent.bits) // 8 + 32 * R + (512 * R if ent.bits == 8 else 0)
        else:
            n = pw.pw_page_bytes(self.desc, p, int(ent.bits))
        base = self.pool_ptr - self._pool_t.data_ptr() + ent.data_off
        return self._pool_t[base:base + n].cpu().numpy()

    def device_table(self) -> np.ndarray:
        off = self.table_ptr - self._table_t.data_ptr()
        return self._table_t[off:off + self.n_entries * ENTRY_BYTES].cpu().numpy()

    def stats(self):
        return pw.pw_pool_stats(self.handle)

    def close(self):
        if self.handle:
            torch.cuda.synchronize(self.device)
            pw.pw_layer_destroy(self.handle)
            self.handle = 0

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Planner:
    """Host-side runtime planner (Alg. 1); see pw_planner_* in include/pw.h."""

    def __init__(self, handle: int):
        self.handle = handle

    def add_request(self, stats_gate_up, stats_down=None, kv_weight: float = 1.0):
        g = stats_gate_up.cpu().numpy() if isinstance(stats_gate_up, torch.Tensor) else stats_gate_up
        d = stats_down.cpu().numpy() if isinstance(stats_down, torch.Tensor) else stats_down
        pw.pw_planner_add_request(self.handle, g, d, kv_weight)

    def clear_requests(self):
        pw.pw_planner_clear_requests(self.handle)

    def step(self, layer: PagedLayer, free_blocks: int, free_threshold: int, kv_block_bytes: int):
        return pw.pw_planner_step_layer(self.handle, layer.handle, free_blocks, free_threshold, kv_block_bytes)

    def plan(self, stage: int = -1, steps: bool = False):
        return pw.pw_planner_plan(self.handle, stage, steps)

    def apply(self, layer: PagedLayer, stream=None) -> int:
        return pw.pw_planner_apply(self.handle, layer.handle, _stream(stream))

    def close(self):
        if self.handle:
            pw.pw_planner_destroy(self.handle)
            self.handle = 0

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
