"""Host-side checks of the seeded input generators (no method arithmetic)."""
import numpy as np

from paper_2010_12635_amd import inputs as I


def test_er_exact_edge_count_and_simple():
    s, d = I.er_graph(300, 1200, np.random.default_rng(0))
    assert s.size == 1200
    assert np.all(s != d)
    pairs = set(zip(np.minimum(s, d).tolist(), np.maximum(s, d).tolist()))
    assert len(pairs) == 1200
    assert s.min() >= 0 and max(s.max(), d.max()) < 300


def test_decode_upper_pairs_bijective():
    s = 37
    idx = np.arange(s * (s - 1) // 2)
    i, j = I._decode_upper_pairs(idx, s)
    assert np.all(i < j) and np.all(j < s)
    assert len(set(zip(i.tolist(), j.tolist()))) == idx.size


def test_ba_edge_count_and_degrees():
    n, m = 2000, 4
    s, d = I.ba_graph(n, m, np.random.default_rng(1))
    assert s.size == m * (n - m)
    assert np.all(s > d)                       # every edge joins a new vertex to an older one
    # no repeated edge from the same new vertex
    for v in (m, 100, n - 1):
        assert len(set(d[s == v].tolist())) == m
    deg = np.bincount(np.r_[s, d], minlength=n)
    assert deg.max() > 10 * m                  # hubs appear


def test_sbm_block_structure():
    s, d, block = I.sbm_graph(1024, 8, 0.05, 0.001, np.random.default_rng(2))
    same = block[s] == block[d]
    assert same.mean() > 0.7
    assert np.all(s != d)


def test_rmat_skew_and_range():
    s, d = I.rmat_graph(12, 8, 0.57, 0.19, 0.19, np.random.default_rng(3))
    n = 1 << 12
    assert s.size == 8 * n and s.max() < n and d.max() < n
    deg = np.bincount(np.r_[s, d], minlength=n)
    assert deg.max() > 20 * deg.mean()


def test_workload_is_seeded():
    a = I.workload("er2k", 5)
    b = I.workload("er2k", 5)
    c = I.workload("er2k", 6)
    assert np.array_equal(a["src"], b["src"]) and np.array_equal(a["X"], b["X"])
    assert not np.array_equal(a["src"], c["src"])
    x = a["X"]
    assert 0.005 < (x != 0).mean() < 0.015 and x.min() >= 0 and x.max() < 1
    assert a["mask"].sum() == 140
