"""Shared test helpers: seeded cases, oracle/GPU layer construction, metrics."""
import functools
import os
import sys

import numpy as np

import oracle
from paper_2607_16184_amd import synth


@functools.lru_cache(maxsize=4)
def case(name: str, **overrides):
    """(cfg, w16 per proj, bits per proj, pool order) of a named workload."""
    cfg = synth.CONFIGS[name]
    if overrides:
        import dataclasses
        cfg = dataclasses.replace(cfg, **overrides)
    w16 = tuple(synth.expert_weights(cfg, p) for p in range(3))
    bits = tuple(synth.bitmap(cfg))
    order = tuple(synth.pool_order(cfg))
    return cfg, w16, bits, order


def oracle_layer(cfg, w16, bits):
    return oracle.OracleLayer(cfg.E, cfg.H, cfg.F, cfg.R, cfg.G, cfg.act, cfg.sdt,
                              list(w16), [np.array(b) for b in bits])


def gpu_layer(cfg, w16, bits, order, slack=0.0):
    from paper_2607_16184_amd.layer import PagedLayer
    L = PagedLayer(cfg, PagedLayer.pool_bytes_for(cfg, bits, slack))
    L.load_pages(w16, bits, order)
    return L


def rel_err(y, r):
    """max |y - r| / max |r| over the tensor."""
    y = np.asarray(y, np.float64)
    r = np.asarray(r, np.float64)
    return float(np.abs(y - r).max() / max(np.abs(r).max(), 1e-300))


def y16_values(y_t, act):
    """Kernel 16-bit output (int16 tensor of bit patterns) as float64."""
    return synth.from16(y_t.cpu().numpy().view(np.uint16), act).astype(np.float64)


def to_dev16(a16):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a16).view(np.int16)).cuda()


def to_dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def say(msg):
    """Name the case before a GPU step, flushed (survives a lost box)."""
    sys.stdout.write("[case] %s\n" % msg)
    sys.stdout.flush()


def assert_all_pages_equal(L, O, cfg, blocks=None):
    """Every page (or the listed (e, p, rb) blocks) of GPU layer L byte-identical
    to the oracle layer O's page image. The pool is copied to the host once."""
    pool = L._pool_t.cpu().numpy()
    base = L.pool_ptr - L._pool_t.data_ptr()
    if blocks is None:
        blocks = [(e, p, rb) for p in range(3) for e in range(cfg.E) for rb in range(cfg.nrb(p))]
    bad = []
    for (e, p, rb) in blocks:
        ent = L.entry(e, p, rb)
        want = O.page_image(p, e, rb)
        assert int(ent.bits) == int(O.bits[p][e, rb]), (e, p, rb)
        got = pool[base + ent.data_off:base + ent.data_off + want.size]
        if not np.array_equal(got, want):
            bad.append((e, p, rb))
    assert not bad, "%d of %d pages differ, first %s" % (len(bad), len(blocks), bad[:4])
    return len(blocks)
