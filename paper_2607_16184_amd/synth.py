"""Seeded synthetic inputs for the paged mixed-bit MoE layer.

This module only draws random numbers and lays them out. It holds none of the
method's arithmetic (no routing, no quantization, no matmul), so both the CPU
oracle's tests and the GPU path may consume what it returns.

Workloads stand in for the paper's evaluated models (Table 1): Mixtral-8x7B's
expert shape with top-2 routing, and a fine-grained many-expert layer for the
Qwen1.5-MoE / Gemma regime. The paper's datasets and trained weights are not
used; every tensor here is drawn from a seeded normal distribution.

Seeds: ``np.random.default_rng(1000 * cfg_id + stream)`` with streams
0 logits, 1 per-expert logit bias, 2 activations, 3/4/5 gate/up/down weights,
6 bitwidth map, 7 pool order, 8 downshift page selection, 9 shared-expert
gates, and 100 + s for the logits and activations of decode step s in the
downshift workload.

16-bit values are produced by round-to-nearest-even from fp32 draws and are
returned as raw uint16 bit patterns; no consumer re-rounds them.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional, Tuple

import numpy as np

GATE, UP, DOWN = 0, 1, 2
PROJ_NAMES = ("gate", "up", "down")
F16, BF16 = 0, 1


@dataclasses.dataclass(frozen=True)
class LayerConfig:
    """Shape and input recipe of one synthetic MoE layer."""

    cfg_id: int
    name: str
    E: int                  # experts of the layer (routed, then n_shared shared)
    K: int                  # routed top-k
    H: int                  # hidden size
    F: int                  # expert FFN size
    T: int                  # tokens per step
    R: int                  # rows per page (row-block height)
    G: int                  # quantization group size along the reduction dim
    act: int                # F16 or BF16 (activations and 16-bit pages)
    sdt: int                # F16 or BF16 (scale / zero dtype)
    mix: Optional[Tuple[float, float, float]]  # stratified (16, 8, 4) fractions; None = iid
    bias_sd: float = 0.0    # per-expert router logit bias sd (load skew)
    shuffle_pool: bool = True
    # runtime downshift workload
    steps: int = 0
    downshift_frac: float = 0.0
    downshift_bits: int = 4
    downshift_chunks: int = 0
    # shared experts: the last n_shared of the E experts, used by every token
    n_shared: int = 0

    @property
    def S(self) -> int:
        return self.T * (self.K + self.n_shared)

    @property
    def E_routed(self) -> int:
        return self.E - self.n_shared

    def nrb(self, proj: int) -> int:
        """Row-blocks (pages) per expert for a projection."""
        return (self.F if proj != DOWN else self.H) // self.R

    def kdim(self, proj: int) -> int:
        """Reduction length of a projection's rows."""
        return self.H if proj != DOWN else self.F

    def with_tokens(self, T: int) -> "LayerConfig":
        return dataclasses.replace(self, T=T)


def _cfg(**kw) -> LayerConfig:
    return LayerConfig(**kw)


CONFIGS: Dict[str, LayerConfig] = {
    # 8 experts, top-2, 256/512, 16 tokens, fp16, 64-row pages, iid {16,8,4}, G=64
    "tiny": _cfg(cfg_id=1, name="tiny", E=8, K=2, H=256, F=512, T=16, R=64, G=64,
                 act=F16, sdt=F16, mix=None),
    # Mixtral-shaped decode: 8 experts top-2, 4096/14336, 64 tokens bf16,
    # 128-row pages, 50/25/25 mix, G=128, pool order shuffled
    "mixtral_decode": _cfg(cfg_id=2, name="mixtral_decode", E=8, K=2, H=4096, F=14336,
                           T=64, R=128, G=128, act=BF16, sdt=BF16,
                           mix=(0.5, 0.25, 0.25)),
    # Mixtral-shaped prefill: 4096 tokens, router bias N(0, 0.5) for load skew
    "mixtral_prefill": _cfg(cfg_id=3, name="mixtral_prefill", E=8, K=2, H=4096, F=14336,
                            T=4096, R=128, G=128, act=BF16, sdt=BF16,
                            mix=(0.5, 0.25, 0.25), bias_sd=0.5),
    # fine-grained: 64 experts top-6, 2048/1408, 512 tokens, 64-row pages, 25/25/50
    "finegrained": _cfg(cfg_id=4, name="finegrained", E=64, K=6, H=2048, F=1408,
                        T=512, R=64, G=128, act=BF16, sdt=BF16,
                        mix=(0.25, 0.25, 0.5)),
    # runtime downshift: the Mixtral decode layer over 32 steps; 25% of the
    # 16-bit pages of each projection go to int4 in 8 chunks
    "downshift": _cfg(cfg_id=5, name="downshift", E=8, K=2, H=4096, F=14336,
                      T=64, R=128, G=128, act=BF16, sdt=BF16,
                      mix=(0.5, 0.25, 0.25), steps=32, downshift_frac=0.25,
                      downshift_bits=4, downshift_chunks=8),
    # shared experts, shaped like Qwen1.5-MoE's layer (Table 1: 60 routed +
    # 4 shared experts, top-4; hidden 2048, expert FFN 1408): 128 decode
    # tokens, 64-row pages 25/25/50, a per-token gate per shared expert
    "qwen_shared": _cfg(cfg_id=6, name="qwen_shared", E=64, K=4, H=2048, F=1408,
                        T=128, R=64, G=128, act=BF16, sdt=BF16,
                        mix=(0.25, 0.25, 0.5), n_shared=4),
    # tiny layer with 8 routed + 2 shared experts (parity cases)
    "tiny_shared": _cfg(cfg_id=7, name="tiny_shared", E=10, K=2, H=256, F=512, T=16, R=64, G=64,
                        act=F16, sdt=F16, mix=None, n_shared=2),
}


def rng(cfg: LayerConfig, stream: int) -> np.random.Generator:
    return np.random.default_rng(1000 * cfg.cfg_id + stream)


def to16(a: np.ndarray, fmt: int) -> np.ndarray:
    """Round fp32 values to fp16 / bf16 (nearest-even); return uint16 bits."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    if fmt == F16:
        return a.astype(np.float16).view(np.uint16)
    import torch  # CPU conversion only
    return torch.from_numpy(a).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def from16(bits: np.ndarray, fmt: int) -> np.ndarray:
    """Widen uint16 bit patterns to fp32 values (exact)."""
    bits = np.ascontiguousarray(bits, dtype=np.uint16)
    if fmt == F16:
        return bits.view(np.float16).astype(np.float32)
    return (bits.astype(np.uint32) << 16).view(np.float32)


def logits(cfg: LayerConfig, stream: int = 0, T: Optional[int] = None) -> np.ndarray:
    """Router logits [T, E_routed] fp32 ~ N(0,1), plus a per-expert N(0, bias_sd) bias."""
    T = cfg.T if T is None else T
    lg = rng(cfg, stream).standard_normal((T, cfg.E_routed), dtype=np.float32)
    if cfg.bias_sd > 0:
        b = rng(cfg, 1).standard_normal(cfg.E_routed, dtype=np.float32) * np.float32(cfg.bias_sd)
        lg = (lg + b[None, :]).astype(np.float32)
    return np.ascontiguousarray(lg)


def shared_gate(cfg: LayerConfig, T: Optional[int] = None) -> np.ndarray:
    """Per-token gates of the shared experts [T, n_shared] fp32 ~ U(0, 1) (the
    range of a sigmoid gate), drawn from stream 9."""
    T = cfg.T if T is None else T
    return np.ascontiguousarray(rng(cfg, 9).uniform(0.0, 1.0, (T, cfg.n_shared)).astype(np.float32))


def activations(cfg: LayerConfig, T: Optional[int] = None) -> np.ndarray:
    """Activations x [T, H] as 16-bit bits of dtype ``cfg.act``, ~ N(0,1)."""
    T = cfg.T if T is None else T
    return to16(rng(cfg, 2).standard_normal((T, cfg.H), dtype=np.float32), cfg.act)


def step_inputs(cfg: LayerConfig, step: int) -> Tuple[np.ndarray, np.ndarray]:
    """Fresh (logits [T,E] fp32, x [T,H] 16-bit) for decode step ``step``."""
    g = np.random.default_rng(1000 * cfg.cfg_id + 100 + step)
    lg = g.standard_normal((cfg.T, cfg.E), dtype=np.float32)
    x = to16(g.standard_normal((cfg.T, cfg.H), dtype=np.float32), cfg.act)
    return np.ascontiguousarray(lg), x


def expert_weights(cfg: LayerConfig, proj: int) -> np.ndarray:
    """Weights of one projection for all experts, 16-bit bits of dtype ``cfg.act``.

    gate/up: [E, F, H]; down: [E, H, F]. Row-major, a row is one output feature.
    Drawn ~ N(0, 0.02) expert by expert from stream 3/4/5.
    """
    g = rng(cfg, 3 + proj)
    rows, cols = (cfg.F, cfg.H) if proj != DOWN else (cfg.H, cfg.F)
    out = np.empty((cfg.E, rows, cols), dtype=np.uint16)
    for e in range(cfg.E):
        w = g.standard_normal((rows, cols), dtype=np.float32)
        w *= np.float32(0.02)
        out[e] = to16(w, cfg.act)
    return out


def bitmap(cfg: LayerConfig) -> List[np.ndarray]:
    """Initial bitwidth of every page: list over proj of int arrays [E, nrb]."""
    g = rng(cfg, 6)
    out = []
    for proj in (GATE, UP, DOWN):
        n = cfg.E * cfg.nrb(proj)
        if cfg.mix is None:
            b = g.choice(np.array([16, 8, 4]), size=n)
        else:
            n16 = int(round(cfg.mix[0] * n))
            n8 = int(round(cfg.mix[1] * n))
            n4 = n - n16 - n8
            b = np.array([16] * n16 + [8] * n8 + [4] * n4)
            b = b[g.permutation(n)]
        out.append(b.reshape(cfg.E, cfg.nrb(proj)).astype(np.int32))
    return out


def page_list(cfg: LayerConfig) -> List[Tuple[int, int, int]]:
    """Every page (e, proj, rb) in canonical order."""
    return [(e, p, rb) for p in (GATE, UP, DOWN) for e in range(cfg.E)
            for rb in range(cfg.nrb(p))]


def pool_order(cfg: LayerConfig) -> List[Tuple[int, int, int]]:
    """Order in which pages are placed into the pool (seeded shuffle)."""
    pages = page_list(cfg)
    if not cfg.shuffle_pool:
        return pages
    perm = rng(cfg, 7).permutation(len(pages))
    return [pages[i] for i in perm]


def downshift_plan(cfg: LayerConfig, bits: List[np.ndarray]) -> List[List[Tuple[int, int, int]]]:
    """Chunks of pages (e, proj, rb) to lower to ``cfg.downshift_bits``.

    Takes ``downshift_frac`` of the 16-bit pages of each projection, chosen by a
    seeded shuffle, and splits them into ``downshift_chunks`` equal chunks.
    """
    g = rng(cfg, 8)
    chosen = []
    for proj in (GATE, UP, DOWN):
        cand = [(e, proj, rb) for e in range(cfg.E) for rb in range(cfg.nrb(proj))
                if bits[proj][e, rb] == 16]
        n = int(round(cfg.downshift_frac * len(cand)))
        perm = g.permutation(len(cand))[:n]
        chosen.extend(cand[i] for i in perm)
    order = g.permutation(len(chosen))
    chosen = [chosen[i] for i in order]
    nch = max(cfg.downshift_chunks, 1)
    per = (len(chosen) + nch - 1) // nch
    return [chosen[i * per:(i + 1) * per] for i in range(nch)]


def page_rows(w: np.ndarray, cfg: LayerConfig, e: int, proj: int, rb: int) -> np.ndarray:
    """View of the R rows of page (e, proj, rb) from a projection array."""
    return w[e, rb * cfg.R:(rb + 1) * cfg.R]
