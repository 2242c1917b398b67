"""Host-side protocol on the CPU: slot allocator, page-table mirror and the
requant -> commit -> reclaim order (Sec. 3.1 offload: the lower bitwidth is
committed before the old pages are freed; Sec. 3.3: commits at safe
boundaries), driven by a simulated event clock. Errors leave state unchanged.
"""
import ctypes
import os

import pytest

import oracle
from oracle import apl

HERE = os.path.dirname(os.path.abspath(__file__))
LIBP = os.path.join(os.path.dirname(HERE), "paper_2607_16184_amd", "libpw_hosttest.so")


class Entry(ctypes.Structure):
    _fields_ = [("data_off", ctypes.c_uint64), ("sz_off", ctypes.c_uint64), ("bits", ctypes.c_uint8),
                ("state", ctypes.c_uint8), ("rsv", ctypes.c_uint16), ("gen", ctypes.c_uint32)]


class Desc(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int) for n in ("E", "H", "F", "R", "G", "act", "sdt")]


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(LIBP):
        from paper_2607_16184_amd import build
        build.build_hosttest()
    lib = ctypes.CDLL(LIBP)
    lib.pwt_create.restype = ctypes.c_void_p
    lib.pwt_create.argtypes = [ctypes.POINTER(Desc), ctypes.c_uint64]
    lib.pwt_destroy.argtypes = [ctypes.c_void_p]
    lib.pwt_load.argtypes = [ctypes.c_void_p] + [ctypes.c_int] * 4
    lib.pwt_load_apl.argtypes = [ctypes.c_void_p] + [ctypes.c_int] * 4
    ip = ctypes.POINTER(ctypes.c_int)
    lib.pwt_requant.argtypes = [ctypes.c_void_p, ctypes.c_int, ip, ip, ip, ip,
                                ctypes.POINTER(ctypes.c_uint64), ctypes.POINTER(ctypes.c_uint64)]
    lib.pwt_commit.restype = ctypes.c_uint64
    lib.pwt_commit.argtypes = [ctypes.c_void_p, ip]
    lib.pwt_complete.argtypes = [ctypes.c_void_p, ctypes.c_uint64]
    lib.pwt_reclaim.restype = ctypes.c_uint64
    lib.pwt_reclaim.argtypes = [ctypes.c_void_p]
    lib.pwt_entry.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.POINTER(Entry)]
    u64p = ctypes.POINTER(ctypes.c_uint64)
    lib.pwt_stats.argtypes = [ctypes.c_void_p, u64p, u64p, u64p, u64p]
    lib.pwt_all_present.argtypes = [ctypes.c_void_p]
    lib.pwt_set_host_pool.argtypes = [ctypes.c_void_p, ctypes.c_uint64]
    lib.pwt_offload.argtypes = [ctypes.c_void_p, ctypes.c_int, ip, ip, ip, u64p]
    lib.pwt_reload.argtypes = [ctypes.c_void_p, ctypes.c_int, ip, ip, ip, u64p, u64p]
    lib.pwt_drop_host_copy.argtypes = [ctypes.c_void_p] + [ctypes.c_int] * 3
    lib.pwt_host_copy.argtypes = [ctypes.c_void_p] + [ctypes.c_int] * 3 + [ip, u64p, u64p]
    lib.pwt_host_stats.argtypes = [ctypes.c_void_p, u64p, u64p]
    lib.pwt_last_error.restype = ctypes.c_char_p
    return lib


R, G, E, H, F = 64, 64, 2, 256, 512
PW_FMT_APL = 1


class Layer:
    def __init__(self, lib, pool_bytes):
        self.lib = lib
        self.h = lib.pwt_create(ctypes.byref(Desc(E, H, F, R, G, 1, 1)), pool_bytes)
        assert self.h

    def load(self, e, p, rb, b):
        return self.lib.pwt_load(self.h, e, p, rb, b)

    def load_apl(self, e, p, rb, b):
        return self.lib.pwt_load_apl(self.h, e, p, rb, b)

    def requant(self, blocks, nb):
        n = len(blocks)
        arr = ctypes.c_int * max(n, 1)
        es, ps, rbs = (zip(*blocks) if n else ((), (), ()))
        d, ev = ctypes.c_uint64(), ctypes.c_uint64()
        st = self.lib.pwt_requant(self.h, n, arr(*es), arr(*ps), arr(*rbs), arr(*([nb] * n)),
                                  ctypes.byref(d), ctypes.byref(ev))
        return st, d.value, ev.value

    def commit(self):
        n = ctypes.c_int()
        ev = self.lib.pwt_commit(self.h, ctypes.byref(n))
        return n.value, ev

    def entry(self, e, p, rb):
        x = Entry()
        assert self.lib.pwt_entry(self.h, e, p, rb, ctypes.byref(x)) == 0
        return x

    def stats(self):
        v = [ctypes.c_uint64() for _ in range(4)]
        self.lib.pwt_stats(self.h, *[ctypes.byref(x) for x in v])
        return [x.value for x in v]

    def _batch(self, blocks):
        n = len(blocks)
        arr = ctypes.c_int * max(n, 1)
        es, ps, rbs = (zip(*blocks) if n else ((), (), ()))
        return n, arr(*es), arr(*ps), arr(*rbs)

    def offload(self, blocks):
        ev = ctypes.c_uint64()
        st = self.lib.pwt_offload(self.h, *self._batch(blocks), ctypes.byref(ev))
        return st, ev.value

    def reload(self, blocks):
        a, ev = ctypes.c_uint64(), ctypes.c_uint64()
        st = self.lib.pwt_reload(self.h, *self._batch(blocks), ctypes.byref(a), ctypes.byref(ev))
        return st, a.value, ev.value

    def host_copy(self, e, p, rb):
        b, off, ev = ctypes.c_int(), ctypes.c_uint64(), ctypes.c_uint64()
        assert self.lib.pwt_host_copy(self.h, e, p, rb, ctypes.byref(b), ctypes.byref(off), ctypes.byref(ev)) == 0
        return b.value, off.value, ev.value

    def host_stats(self):
        c, u = ctypes.c_uint64(), ctypes.c_uint64()
        self.lib.pwt_host_stats(self.h, ctypes.byref(c), ctypes.byref(u))
        return c.value, u.value

    def close(self):
        self.lib.pwt_destroy(self.h)


def pages():
    return [(e, p, rb) for e in range(E) for p in range(3) for rb in range((F if p < 2 else H) // R)]


def _load_all(Lx, bits=16):
    for (e, p, rb) in pages():
        assert Lx.load(e, p, rb, bits) == 0


def test_allocator_and_load(L):
    need = sum(oracle.page_bytes(R, H if p < 2 else F, G, 16) for (_, p, _) in pages())
    Lx = Layer(L, need)
    _load_all(Lx)
    assert L.pwt_all_present(Lx.h) == 1
    used, free, largest, _ = Lx.stats()
    assert used == need and free == 0
    assert Lx.load(0, 0, 0, 16) == 3          # PW_EBUSY: already present
    offs = sorted((Lx.entry(*pg).data_off, oracle.page_bytes(R, H if pg[1] < 2 else F, G, 16))
                  for pg in pages())
    for (a, n), (b, _) in zip(offs, offs[1:]):
        assert a + n <= b                     # slots never overlap
    Lx.close()


def test_pool_exhaustion_leaves_state_unchanged(L):
    Lx = Layer(L, 4 * 65536)
    assert Lx.load(0, 0, 0, 16) == 0          # 32 KiB
    before = Lx.stats()
    st, d, ev = Lx.requant([(0, 0, 0)], 8)
    assert st == 0
    Lx2 = Layer(L, oracle.page_bytes(R, H, G, 16))
    assert Lx2.load(0, 0, 0, 16) == 0
    assert Lx2.load(0, 0, 1, 4) == 2          # PW_ENOMEM
    st, d, ev = Lx2.requant([(0, 0, 0)], 4)
    assert st == 2 and Lx2.entry(0, 0, 0).bits == 16 and Lx2.entry(0, 0, 0).state == 1
    Lx.close()
    Lx2.close()


def test_requant_commit_reclaim_order(L):
    need = sum(oracle.page_bytes(R, H if p < 2 else F, G, 16) for (_, p, _) in pages())
    Lx = Layer(L, 2 * need)
    _load_all(Lx)
    old = Lx.entry(1, 2, 3)
    free0 = Lx.stats()[1]
    st, delta, ev = Lx.requant([(1, 2, 3)], 4)
    assert st == 0 and delta == oracle.delta_bytes(R, F, G, 16, 4)
    cur = Lx.entry(1, 2, 3)
    # offload: nothing is published before the commit
    assert (cur.bits, cur.data_off, cur.state) == (16, old.data_off, 2)
    assert Lx.requant([(1, 2, 3)], 8)[0] == 3  # PW_EBUSY while pending
    n, cev = Lx.commit()
    assert n == 1 and cev != 0
    cur = Lx.entry(1, 2, 3)
    assert cur.bits == 4 and cur.gen == old.gen + 1 and cur.data_off != old.data_off and cur.state == 1
    # the old slot is retired, not freed, until the commit has completed
    assert L.pwt_reclaim(Lx.h) == 0
    L.pwt_complete(Lx.h, cev)
    assert L.pwt_reclaim(Lx.h) == oracle.page_bytes(R, F, G, 16)
    assert Lx.stats()[1] - free0 == delta      # Eq. 3: the pool gained exactly Delta
    assert Lx.stats()[3] == 0                  # every event released
    Lx.close()


def test_requant_rules(L):
    need = sum(oracle.page_bytes(R, H if p < 2 else F, G, 16) for (_, p, _) in pages())
    Lx = Layer(L, 2 * need)
    _load_all(Lx, bits=8)
    st, d, ev = Lx.requant([(0, 0, 0)], 8)     # same bits: no-op
    assert st == 0 and d == 0 and ev == 0 and Lx.commit()[0] == 0
    assert Lx.requant([(0, 0, 0)], 16)[0] == 4  # raising: PW_EUNSUPPORTED
    assert Lx.requant([(0, 0, 0)], 5)[0] == 1
    assert Lx.requant([(0, 0, 0), (0, 0, 0)], 4)[0] == 1   # duplicate in a batch
    assert Lx.requant([(0, 0, 99)], 4)[0] == 1
    free0 = Lx.stats()[1]
    # a failing batch rolls back the slots of the earlier blocks
    assert Lx.requant([(0, 0, 0), (0, 1, 0), (5, 0, 0)], 4)[0] == 1
    assert Lx.stats()[1] == free0 and Lx.entry(0, 0, 0).state == 1
    st, d, ev = Lx.requant([(0, 0, 0), (1, 2, 0)], 4)
    assert st == 0 and d == oracle.delta_bytes(R, H, G, 8, 4) + oracle.delta_bytes(R, F, G, 8, 4)
    n, cev = Lx.commit()
    assert n == 2
    L.pwt_complete(Lx.h, cev)
    assert L.pwt_reclaim(Lx.h) == oracle.page_bytes(R, H, G, 8) + oracle.page_bytes(R, F, G, 8)
    assert Lx.stats()[1] - free0 == d
    Lx.close()


def test_allocator_coalesces(L):
    one = oracle.page_bytes(R, H, G, 16)
    Lx = Layer(L, 3 * one)
    for rb in range(3):
        assert Lx.load(0, 0, rb, 16) == 0
    for rb in range(3):
        st, _, _ = Lx.requant([(0, 0, rb)], 4)
        assert st == 2                          # pool full: ENOMEM, nothing changed
    Lx.close()
    Lx = Layer(L, 4 * one)
    for rb in range(3):
        assert Lx.load(0, 0, rb, 16) == 0
    for rb in (0, 2, 1):
        assert Lx.requant([(0, 0, rb)], 4)[0] == 0
        n, cev = Lx.commit()
        L.pwt_complete(Lx.h, cev)
        Lx.reclaim = L.pwt_reclaim(Lx.h)
    used, free, largest, _ = Lx.stats()
    assert used == 3 * ((oracle.page_bytes(R, H, G, 4) + 255) // 256 * 256)
    assert largest >= 2 * one                  # freed neighbours merged
    Lx.close()


def _slot(nbytes):
    return (nbytes + 255) // 256 * 256


def test_offload_lower_reload_cycle(L):
    """Sec. 3.1: the 16-bit page goes to host memory before the block is
    lowered; a later reload raises it back. The reload is published by a
    commit, the lower page retires only after that commit completed, and the
    host slot stays until its last transfer finished."""
    need = sum(oracle.page_bytes(R, H if p < 2 else F, G, 16) for (_, p, _) in pages())
    Lx = Layer(L, 2 * need)
    _load_all(Lx)
    L.pwt_set_host_pool(Lx.h, need)
    p16, p4 = oracle.page_bytes(R, F, G, 16), oracle.page_bytes(R, F, G, 4)
    st, oev = Lx.offload([(1, 2, 3), (0, 0, 0)])
    assert st == 0 and oev != 0
    assert Lx.host_copy(1, 2, 3)[0] == 16 and Lx.host_copy(1, 2, 3)[2] == oev
    assert Lx.host_stats() == (need, _slot(p16) + _slot(oracle.page_bytes(R, H, G, 16)))
    assert Lx.offload([(1, 2, 3)]) == (0, 0)            # a copy at this bitwidth exists: no-op
    old = Lx.entry(1, 2, 3)
    assert Lx.requant([(1, 2, 3)], 4)[0] == 0
    n, cev = Lx.commit()
    L.pwt_complete(Lx.h, cev)
    assert L.pwt_reclaim(Lx.h) == p16
    free0 = Lx.stats()[1]
    low = Lx.entry(1, 2, 3)
    assert low.bits == 4 and low.gen == old.gen + 1
    # raise it back
    st, added, rev = Lx.reload([(1, 2, 3)])
    assert st == 0 and added == p16 - p4 and rev not in (0, oev)
    cur = Lx.entry(1, 2, 3)
    assert (cur.bits, cur.data_off, cur.state) == (4, low.data_off, 3)   # reload pending, 4-bit page served
    assert Lx.stats()[1] == free0 - _slot(p16)
    assert Lx.requant([(1, 2, 3)], 8)[0] == 3            # EBUSY while the reload is pending
    assert Lx.offload([(1, 2, 3)])[0] == 3
    assert Lx.reload([(1, 2, 3)])[0] == 3
    assert Lx.host_copy(1, 2, 3)[2] == rev               # the host slot now waits for the reload
    n, cev2 = Lx.commit()
    assert n == 1
    cur = Lx.entry(1, 2, 3)
    assert (cur.bits, cur.state, cur.gen) == (16, 1, low.gen + 1) and cur.data_off != low.data_off
    assert L.pwt_reclaim(Lx.h) == 0                      # the 4-bit page retires on the commit
    L.pwt_complete(Lx.h, cev2)
    assert L.pwt_reclaim(Lx.h) == p4
    assert Lx.stats()[1] == free0 - _slot(p16) + _slot(p4)
    assert Lx.reload([(1, 2, 3)])[0] == 4                # copy not above the committed bitwidth
    # dropping the copy frees its host slot once the reload's transfer is done
    used0 = Lx.host_stats()[1]
    assert L.pwt_drop_host_copy(Lx.h, 1, 2, 3) == 0
    assert Lx.host_copy(1, 2, 3)[0] == 0
    L.pwt_reclaim(Lx.h)
    assert Lx.host_stats()[1] == used0
    L.pwt_complete(Lx.h, rev)
    L.pwt_reclaim(Lx.h)
    assert Lx.host_stats()[1] == used0 - _slot(p16)
    assert L.pwt_drop_host_copy(Lx.h, 0, 0, 0) == 0
    L.pwt_complete(Lx.h, oev)
    L.pwt_reclaim(Lx.h)
    assert Lx.host_stats()[1] == 0 and Lx.stats()[3] == 0   # every slot and event released
    Lx.close()


def test_bitplane_offload_lower_reload_cycle(L):
    """Sec. 3.1 with nested bit-plane pages (Sec. 3.2, Eq. 3): the host copy
    is the whole committed page (planes and LUTs), the 8 -> 4 drop frees the
    page tail in place, and the reload brings the whole 8-bit page back into
    a fresh slot, with LUT_4 right after planes 0-3 as in a loaded page."""
    K = H                                              # gate rows read H inputs
    a8, a4 = apl.page_bytes(R, K, 8), apl.page_bytes(R, K, 4)
    assert a8 == R * K + 544 * R and a4 == R * K // 2 + 32 * R
    Lx = Layer(L, 3 * _slot(a8) + _slot(oracle.page_bytes(R, K, G, 16)))
    assert Lx.load_apl(0, 0, 0, 8) == 0 and Lx.load_apl(0, 0, 1, 4) == 0
    assert Lx.load_apl(0, 0, 0, 8) == 3                # already present
    assert Lx.load_apl(0, 0, 2, 16) == 1               # bit-plane pages hold 8 or 4 bits
    assert Lx.load(1, 0, 0, 16) == 0
    ld = Lx.entry(0, 0, 0)
    assert (ld.bits, ld.rsv, ld.sz_off) == (8, PW_FMT_APL, ld.data_off + R * K // 2)
    L.pwt_set_host_pool(Lx.h, 4 * _slot(a8))
    st, oev = Lx.offload([(0, 0, 0), (0, 0, 1)])
    assert st == 0 and oev != 0
    assert Lx.host_stats()[1] == _slot(a8) + _slot(a4)  # each copy is its committed page
    assert Lx.host_copy(0, 0, 0)[0] == 8 and Lx.host_copy(0, 0, 1)[0] == 4
    assert Lx.offload([(0, 0, 0)]) == (0, 0)            # same bitwidth and format: no-op
    # 8 -> 4 in place: the slot keeps planes 0-3 and LUT_4, the tail retires after the commit
    st, d, _ = Lx.requant([(0, 0, 0)], 4)
    assert st == 0 and d == a8 - a4
    n, cev = Lx.commit()
    assert n == 1 and L.pwt_reclaim(Lx.h) == 0
    L.pwt_complete(Lx.h, cev)
    assert L.pwt_reclaim(Lx.h) == a8 - a4
    low = Lx.entry(0, 0, 0)
    assert (low.bits, low.rsv, low.data_off, low.sz_off, low.gen) == (4, PW_FMT_APL, ld.data_off, ld.sz_off, 2)
    assert Lx.requant([(0, 0, 0)], 8)[0] == 4           # raising needs the host copy
    free0 = Lx.stats()[1]
    st, added, rev = Lx.reload([(0, 0, 0)])
    assert st == 0 and added == a8 - a4 and rev not in (0, oev)
    assert Lx.entry(0, 0, 0).state == 3 and Lx.stats()[1] == free0 - _slot(a8)
    n, cev2 = Lx.commit()
    cur = Lx.entry(0, 0, 0)
    assert (cur.bits, cur.rsv, cur.state, cur.gen) == (8, PW_FMT_APL, 1, 3)
    assert cur.data_off != low.data_off and cur.sz_off == cur.data_off + R * K // 2
    L.pwt_complete(Lx.h, cev2)
    assert L.pwt_reclaim(Lx.h) == a4                    # the 4-bit prefix retires
    assert Lx.stats()[1] == free0 - _slot(a8) + _slot(a4)
    # a 4-bit page has no higher copy to reload; offloading it again at 4 bits replaces nothing
    assert Lx.reload([(0, 0, 1)])[0] == 4
    # the reloaded page can be lowered again, and a copy of the lower page replaces the 8-bit one
    assert Lx.requant([(0, 0, 0)], 4)[0] == 0
    n, cev3 = Lx.commit()
    L.pwt_complete(Lx.h, cev3)
    L.pwt_complete(Lx.h, rev)
    L.pwt_reclaim(Lx.h)
    st, oev2 = Lx.offload([(0, 0, 0)])
    assert st == 0 and Lx.host_copy(0, 0, 0)[0] == 4
    L.pwt_complete(Lx.h, oev)
    L.pwt_complete(Lx.h, oev2)
    L.pwt_reclaim(Lx.h)
    assert Lx.host_stats()[1] == 2 * _slot(a4)
    assert Lx.reload([(0, 0, 0)])[0] == 4               # copy not above the committed bitwidth
    for blk in ((0, 0, 0), (0, 0, 1)):
        assert L.pwt_drop_host_copy(Lx.h, *blk) == 0
    L.pwt_reclaim(Lx.h)
    assert Lx.host_stats()[1] == 0 and Lx.stats()[3] == 0
    Lx.close()


def test_offload_reload_errors(L):
    one16, one8 = oracle.page_bytes(R, H, G, 16), oracle.page_bytes(R, H, G, 8)
    Lx = Layer(L, 2 * one16 + one8)
    assert Lx.offload([(0, 0, 0)])[0] == 6               # no host pool: ESTATE
    L.pwt_set_host_pool(Lx.h, one16 + 256)
    assert Lx.offload([(0, 0, 0)])[0] == 6               # page absent
    assert Lx.load(0, 0, 0, 16) == 0 and Lx.load(0, 0, 1, 16) == 0
    assert Lx.reload([(0, 0, 0)])[0] == 6                # no host copy
    assert Lx.offload([(0, 0, 0), (0, 0, 0)])[0] == 1    # duplicate in a batch
    # a batch that does not fit leaves no host slot behind
    assert Lx.offload([(0, 0, 0), (0, 0, 1)])[0] == 2
    assert Lx.host_stats()[1] == 0 and Lx.host_copy(0, 0, 0)[0] == 0
    st, oev = Lx.offload([(0, 0, 0)])
    assert st == 0
    # lower to 8 bits; then the pool is too full to take a 16-bit page back
    assert Lx.requant([(0, 0, 0)], 8)[0] == 0
    n, cev = Lx.commit()
    L.pwt_complete(Lx.h, cev)
    L.pwt_reclaim(Lx.h)
    assert Lx.load(0, 1, 0, 16) == 0
    free0 = Lx.stats()[1]
    before = Lx.entry(0, 0, 0)
    assert Lx.reload([(0, 0, 0)])[0] == 2                # device pool: ENOMEM, nothing changed
    after = Lx.entry(0, 0, 0)
    assert (after.bits, after.state, after.data_off) == (8, 1, before.data_off) and Lx.stats()[1] == free0
    # offloading the 8-bit page replaces the 16-bit copy (its slot waits for its transfer)
    assert Lx.offload([(0, 0, 0)])[0] == 2               # the host pool holds the 16-bit copy
    assert L.pwt_drop_host_copy(Lx.h, 0, 0, 0) == 0
    L.pwt_complete(Lx.h, oev)
    L.pwt_reclaim(Lx.h)
    st, oev2 = Lx.offload([(0, 0, 0)])
    assert st == 0 and Lx.host_copy(0, 0, 0)[0] == 8
    assert Lx.reload([(0, 0, 0)])[0] == 4                # the copy is not of a higher bitwidth
    Lx.close()
