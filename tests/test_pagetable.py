"""Host-side page table of the paged cache (the C++ that libws.so runs before
every launch), exercised on the CPU through libws_host.so.  Checks the
bookkeeping the block-causal mask relies on (Wan-Streamer v0.2, Fig. 1
caption; Sec. 2.1 history commit; Sec. 3 cache update per unit)."""
import ctypes
import os

import numpy as np
import pytest

OK, OUT_OF_PAGES, UNKNOWN, COMMITTED, SHAPE = 0, 1, 2, 3, 4
COND, VIDEO, AUDIO = 0, 1, 2


@pytest.fixture(scope="module")
def lib():
    from paper_2607_04443_amd import _build
    if not os.path.exists(_build.HOST_LIB_PATH):
        _build.build()
    L = ctypes.CDLL(_build.HOST_LIB_PATH)
    L.wsh_create.restype = ctypes.c_void_p
    L.wsh_create.argtypes = [ctypes.c_int32, ctypes.c_int32]
    L.wsh_destroy.argtypes = [ctypes.c_void_p]
    L.wsh_acquire.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                              ctypes.POINTER(ctypes.c_int32)]
    L.wsh_commit.argtypes = [ctypes.c_void_p, ctypes.c_int32]
    L.wsh_evict_before.argtypes = [ctypes.c_void_p, ctypes.c_int32]
    L.wsh_release.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32]
    L.wsh_reset.argtypes = [ctypes.c_void_p]
    L.wsh_free_pages.argtypes = [ctypes.c_void_p]
    L.wsh_version.argtypes = [ctypes.c_void_p]
    L.wsh_version.restype = ctypes.c_uint64
    L.wsh_n_segments.argtypes = [ctypes.c_void_p]
    L.wsh_visible.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32, ctypes.c_uint32,
                              ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32]
    L.wsh_segment_pages.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32,
                                    ctypes.c_void_p, ctypes.c_int32]
    return L


class PT:
    def __init__(self, lib, max_pages):
        self.L = lib
        self.h = lib.wsh_create(64, max_pages)

    def acquire(self, unit, kind, n):
        created = ctypes.c_int32()
        st = self.L.wsh_acquire(self.h, unit, kind, n, ctypes.byref(created))
        return st, bool(created.value)

    def visible(self, q_unit, min_unit=-(2 ** 31), kind_mask=0b011):
        cap = 4096
        p = np.zeros(cap, np.int32)
        n = np.zeros(cap, np.int32)
        cnt = self.L.wsh_visible(self.h, q_unit, min_unit, kind_mask, p.ctypes.data, n.ctypes.data,
                                 cap)
        return p[:cnt].copy(), n[:cnt].copy()

    def pages(self, unit, kind):
        p = np.zeros(1024, np.int32)
        cnt = self.L.wsh_segment_pages(self.h, unit, kind, p.ctypes.data, 1024)
        return None if cnt < 0 else p[:cnt].copy()

    def free(self):
        return self.L.wsh_free_pages(self.h)

    def __del__(self):
        self.L.wsh_destroy(self.h)


def test_allocation_and_tail_pages(lib):
    pt = PT(lib, 100)
    assert pt.acquire(0, COND, 256) == (OK, True)
    assert pt.acquire(0, VIDEO, 920) == (OK, True)
    assert len(pt.pages(0, COND)) == 4 and len(pt.pages(0, VIDEO)) == 15
    assert pt.free() == 100 - 19
    p, n = pt.visible(0)
    assert list(n) == [64] * 4 + [64] * 14 + [24]
    assert len(set(p)) == 19
    assert sum(n) == 256 + 920


def test_rewrite_keeps_pages_and_version(lib):
    pt = PT(lib, 50)
    pt.acquire(3, VIDEO, 100)
    before = pt.pages(3, VIDEO)
    v0 = lib.wsh_version(pt.h)
    assert pt.acquire(3, VIDEO, 100) == (OK, False)
    assert np.array_equal(pt.pages(3, VIDEO), before)
    assert lib.wsh_version(pt.h) == v0
    assert pt.acquire(3, VIDEO, 99)[0] == SHAPE
    lib.wsh_commit(pt.h, 3)
    assert pt.acquire(3, VIDEO, 100)[0] == COMMITTED


def test_out_of_pages_changes_nothing(lib):
    pt = PT(lib, 10)
    assert pt.acquire(0, COND, 64 * 8)[0] == OK
    v = lib.wsh_version(pt.h)
    assert pt.acquire(0, VIDEO, 64 * 3)[0] == OUT_OF_PAGES
    assert pt.free() == 2 and lib.wsh_version(pt.h) == v
    assert pt.pages(0, VIDEO) is None


def test_block_causal_window_and_kinds(lib):
    pt = PT(lib, 200)
    pt.acquire(0, COND, 64)
    for u in range(4):
        pt.acquire(u, VIDEO, 70)   # 2 pages, tail of 6
        pt.acquire(u, AUDIO, 4)    # 1 page of 4
    # video queries of unit 2: cond + video units 0..2
    p, n = pt.visible(2)
    assert sum(n) == 64 + 3 * 70
    # audio queries of unit 3, all kinds
    p, n = pt.visible(3, kind_mask=0b111)
    assert sum(n) == 64 + 4 * 74
    # window: units >= 2 only, cond kept
    p, n = pt.visible(3, min_unit=2, kind_mask=0b111)
    assert sum(n) == 64 + 2 * 74
    # a cond slice of a later unit is not visible yet
    pt.acquire(5, COND, 10)
    p, n = pt.visible(3, kind_mask=0b001)
    assert sum(n) == 64
    p, n = pt.visible(5, kind_mask=0b001)
    assert sum(n) == 74
    # creation order: cond first, then unit 0 video, ...
    p, n = pt.visible(0, kind_mask=0b011)
    assert np.array_equal(p[:1], pt.pages(0, COND)) and np.array_equal(p[1:], pt.pages(0, VIDEO))


def test_evict_and_release_free_exact_pages(lib):
    pt = PT(lib, 64)
    pt.acquire(0, COND, 128)
    for u in range(5):
        pt.acquire(u, VIDEO, 130)
    freed_pages = set(pt.pages(0, VIDEO)) | set(pt.pages(1, VIDEO))
    free0 = pt.free()
    assert lib.wsh_evict_before(pt.h, 2) == 2
    assert pt.free() == free0 + 6
    assert pt.pages(0, VIDEO) is None and pt.pages(0, COND) is not None
    # the freed pages are reused, lowest ids first
    pt.acquire(5, VIDEO, 130)
    assert set(pt.pages(5, VIDEO)) <= freed_pages | set(range(64))
    assert lib.wsh_release(pt.h, 0, COND) == OK
    assert lib.wsh_release(pt.h, 0, COND) == UNKNOWN
    lib.wsh_reset(pt.h)
    assert pt.free() == 64 and lib.wsh_n_segments(pt.h) == 0


def test_pages_never_shared(lib):
    rng = np.random.default_rng(0)
    pt = PT(lib, 300)
    live = {}
    for step in range(200):
        u = int(rng.integers(0, 30))
        kind = int(rng.integers(0, 3))
        if rng.random() < 0.6:
            st, created = pt.acquire(u, kind, int(rng.integers(1, 400)))
            if st == OK and created:
                live[(u, kind)] = True
        elif (u, kind) in live:
            assert lib.wsh_release(pt.h, u, kind) == OK
            del live[(u, kind)]
        owned = [pt.pages(*key) for key in live]
        allp = np.concatenate(owned) if owned else np.zeros(0)
        assert len(allp) == len(set(allp.tolist()))
        assert pt.free() == 300 - len(allp)
