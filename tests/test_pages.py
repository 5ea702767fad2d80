"""KV page allocator of continuous batching (include/vfm_pages.h), on the
host: hand-worked sequences of reserve / release, a plain Python model of
the free stack driven through thousands of random operations, the pool's
invariants, and errors that leave the state unchanged."""
import numpy as np
import pytest

from paper_2606_09643_amd import binding as B


def test_fresh_pool_hands_out_pages_in_order_and_reuses_released_first():
    a = B.PageAllocator(n_pages=8, page_size=16, max_seqs=3, max_pages=4)
    a.reserve(0, 20)                       # 2 pages: 0, 1
    a.reserve(1, 16)                       # 1 page: 2
    a.reserve(0, 32)                       # still 2 pages: no-op
    a.reserve(0, 33)                       # third page: 3
    assert a.table([0, 1, 2], 4).tolist() == [[0, 1, 3, -1], [2, -1, -1, -1], [-1] * 4]
    assert a.count(0) == (3, 4)
    a.release(0)
    assert a.count(0) == (0, 7)
    a.reserve(2, 40)                       # the released sequence's pages, its first page first
    assert a.table([2], 3).tolist() == [[0, 1, 3]]
    a.reserve(1, 0)                        # zero tokens: nothing to add
    assert a.count(1) == (1, 4)


class _Model:
    """The allocator written out with Python lists."""

    def __init__(self, n_pages, page_size, max_seqs, max_pages):
        self.free = list(range(n_pages - 1, -1, -1))     # top = last element
        self.ps, self.mp = page_size, max_pages
        self.pages = [[] for _ in range(max_seqs)]

    def reserve(self, s, n):
        need = -(-n // self.ps)
        extra = need - len(self.pages[s])
        if extra <= 0:
            return True
        if need > self.mp or extra > len(self.free):
            return False
        for _ in range(extra):
            self.pages[s].append(self.free.pop())
        return True

    def release(self, s):
        for p in reversed(self.pages[s]):
            self.free.append(p)
        self.pages[s] = []


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_random_operations_match_the_list_model(seed):
    rng = np.random.default_rng(seed)
    n_pages, ps, n_seq, mp = 64, 16, 12, 10
    a = B.PageAllocator(n_pages, ps, n_seq, mp)
    m = _Model(n_pages, ps, n_seq, mp)
    tokens = [0] * n_seq
    for _ in range(4000):
        s = int(rng.integers(n_seq))
        if rng.random() < 0.15:
            a.release(s)
            m.release(s)
            tokens[s] = 0
        else:
            n = tokens[s] + int(rng.integers(0, 40))
            ok = a.try_reserve(s, n)
            assert ok == m.reserve(s, n)
            if ok:
                tokens[s] = n
        tab = a.table(np.arange(n_seq), mp)
        for q in range(n_seq):
            held = [x for x in tab[q] if x >= 0]
            assert held == m.pages[q]
        owned = [x for row in tab for x in row if x >= 0]
        assert len(owned) == len(set(owned))                    # no page held twice
        assert len(owned) + a.count(0)[1] == n_pages           # held + free = pool


def test_errors_leave_the_state_unchanged():
    a = B.PageAllocator(n_pages=4, page_size=16, max_seqs=2, max_pages=3)
    a.reserve(0, 40)                                           # 3 pages
    before = a.state.copy()
    lib = B.lib()
    st = a.state.ctypes.data
    assert lib.vfm_pages_reserve(st, 1, 40) == B.VFM_ERR_SHAPE     # 3 pages wanted, 1 free
    assert lib.vfm_pages_reserve(st, 0, 64) == B.VFM_ERR_SHAPE     # above max_pages
    assert lib.vfm_pages_reserve(st, 2, 1) == B.VFM_ERR_TASK
    assert lib.vfm_pages_reserve(st, 0, -1) == B.VFM_ERR_SHAPE
    assert lib.vfm_pages_release(st, -1) == B.VFM_ERR_TASK
    out = np.zeros((1, 2), np.int32)
    seqs = np.array([0], np.int32)
    assert lib.vfm_pages_table(st, seqs.ctypes.data, 1, out.ctypes.data, 2) == B.VFM_ERR_SHAPE
    assert np.array_equal(a.state, before)
    assert lib.vfm_pages_reserve(None, 0, 1) == B.VFM_ERR_ARG
    junk = np.zeros(64, np.int64)                              # never initialised
    assert lib.vfm_pages_reserve(junk.ctypes.data, 0, 1) == B.VFM_ERR_ARG
    bad = B.vfm_pages_config(0, 16, 1, 1)
    n = B.C.c_size_t()
    assert lib.vfm_pages_state_size(B.C.byref(bad), B.C.byref(n)) == B.VFM_ERR_SHAPE
