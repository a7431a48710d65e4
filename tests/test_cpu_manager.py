"""The multi-threaded host memory manager (the benchmark's on-CPU comparison baseline)
gives exactly the oracle's state: random allocation / release rounds on several
thread counts, the ring wrapping, and an all-or-nothing refusal (CPU only)."""
import numpy as np
import pytest

from baselines import cpu_manager as cm


@pytest.mark.parametrize("threads", [1, 3, 8])
def test_matches_oracle_over_rounds(orc, threads):
    rng = np.random.default_rng(70 + threads)
    tables, num_pages = 37, 1500
    L = orc.layout(max_seq_len=700)
    oc = orc.Cache(L, num_pages, tables, 1, ring=rng.permutation(num_pages), with_pool=False)
    m = cm.Manager(oc.table, oc.pages, oc.len, oc.ring, oc.ring_ptr, (16, 32), threads)
    try:
        for rnd in range(25):
            free = int(oc.ring_ptr[1] - oc.ring_ptr[0])
            dem = np.zeros((tables, 2), np.int32)
            for t in range(tables):
                room = L.p_max - int(oc.pages[t].sum())
                a = int(rng.integers(0, max(1, min(room, 2 * free // tables) + 1)))
                hi = int(rng.integers(0, a + 1))
                dem[t] = hi, a - hi
            orc.alloc_pages(oc, dem)
            assert m.alloc(dem) == 0
            oc.len[:] = np.maximum(oc.pages * np.array([16, 32]) - rng.integers(0, 16, (tables, 2)), 0)
            oc.len[oc.pages == 0] = 0
            m.len[:] = oc.len
            rel = (rng.random((tables, L.p_max)) < rng.random()).astype(np.uint8)
            orc.compact(oc, rel)
            m.compact(rel)
            for f, o in (("table", oc.table), ("pages", oc.pages), ("len", oc.len),
                         ("ring", oc.ring), ("ring_ptr", oc.ring_ptr)):
                assert np.array_equal(getattr(m, f), o), "round %d: %s" % (rnd, f)
        assert oc.ring_ptr[1] > num_pages   # the ring wrapped
        # refusals change nothing
        snap = {f: getattr(m, f).copy() for f in ("table", "pages", "ring", "ring_ptr")}
        dem = np.zeros((tables, 2), np.int32)
        dem[3, 1] = int(m.ring_ptr[1] - m.ring_ptr[0]) + 1
        assert m.alloc(dem) == 1 and m.status[0] & 1
        dem[:] = 0
        dem[5, 0] = L.p_max
        assert m.alloc(dem) == 1 and m.status[0] & 2
        for f, v in snap.items():
            assert np.array_equal(getattr(m, f), v), f
    finally:
        m.close()
