"""Pins for the CPU oracle: each test checks it against something other than
itself -- brute force, closed forms, invariants, finite differences or an
independent library routine -- so that a dropped term, a wrong sign or
index, or a transposed operand fails at least one of them."""
import json
import math
import os

import numpy as np
import pytest
import scipy.sparse as sp
from hypothesis import given, settings, strategies as st

from oracle import gcn_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------- graph / CSR

def brute_csr(n, src, dst):
    """Set-based construction of the neighbour lists of A + I."""
    nbrs = [set([i]) for i in range(n)]
    for u, v in zip(src, dst):
        if u != v:
            nbrs[u].add(v)
            nbrs[v].add(u)
    rowptr = [0]
    cols = []
    for i in range(n):
        cols.extend(sorted(nbrs[i]))
        rowptr.append(len(cols))
    return np.array(rowptr), np.array(cols)


@settings(max_examples=60, deadline=None)
@given(st.integers(1, 12).flatmap(
    lambda n: st.tuples(st.just(n), st.lists(st.tuples(st.integers(0, n - 1), st.integers(0, n - 1)), max_size=40))))
def test_csr_matches_brute_force(case):
    n, edges = case
    src = [e[0] for e in edges]
    dst = [e[1] for e in edges]
    g = O.graph(n, np.array(src, np.int32), np.array(dst, np.int32))
    rp, ci = brute_csr(n, src, dst)
    assert np.array_equal(g.rowptr, rp)
    assert np.array_equal(g.colidx, ci)
    assert g.deg.sum() == g.nnz


def test_csr_matches_scipy():
    rng = np.random.default_rng(3)
    n = 300
    src = rng.integers(0, n, 2000)
    dst = rng.integers(0, n, 2000)
    g = O.graph(n, src, dst)
    keep = src != dst
    m = sp.coo_matrix((np.ones(keep.sum() * 2), (np.r_[src[keep], dst[keep]], np.r_[dst[keep], src[keep]])),
                      shape=(n, n)).tocsr()
    m.data[:] = 1.0
    m = m + sp.identity(n, format="csr")
    m.sum_duplicates()
    m.sort_indices()
    assert np.array_equal(g.rowptr, m.indptr)
    assert np.array_equal(g.colidx, m.indices)
    # sum of degrees = 2E + n
    e_undirected = len({(min(a, b), max(a, b)) for a, b in zip(src, dst) if a != b})
    assert g.nnz == 2 * e_undirected + n


def test_out_of_range_rejected():
    with pytest.raises(ValueError):
        O.graph(4, np.array([0, 4]), np.array([1, 2]))
    with pytest.raises(ValueError):
        O.graph(4, np.array([-1]), np.array([1]))


def test_empty_graph_is_identity():
    g = O.graph(5, np.zeros(0, np.int32), np.zeros(0, np.int32))
    assert np.array_equal(O.dense_adj(g), np.eye(5))


def _golden():
    with open(os.path.join(GOLDEN, "closed_forms.json")) as f:
        return json.load(f)


def _dense_of(case):
    e = np.array(case["edges"])
    g = O.graph(case["n"], e[:, 0], e[:, 1])
    return O.dense_adj(g)


def test_closed_forms():
    gold = _golden()
    assert np.allclose(_dense_of(gold["K2"]), np.array(gold["K2"]["A_hat"]), rtol=0, atol=1e-15)
    s6 = 1 / math.sqrt(6)
    p3 = np.array([[0.5, s6, 0], [s6, 1 / 3, s6], [0, s6, 0.5]])
    assert np.allclose(_dense_of(gold["P3"]), p3, rtol=0, atol=1e-15)
    a = _dense_of(gold["star_K1_4"])
    assert a[0, 0] == pytest.approx(1 / 5, abs=1e-15)
    assert np.allclose(a[0, 1:], 1 / math.sqrt(10), atol=1e-15)
    assert np.allclose(np.diag(a)[1:], 0.5, atol=1e-15)
    assert np.allclose(a[1:, 1:] - np.diag(np.diag(a)[1:]), 0.0)
    c5 = gold["C5"]
    adj = np.eye(5)
    for u, v in c5["edges"]:
        adj[u, v] = adj[v, u] = 1
    assert np.allclose(_dense_of(c5), adj / 3, atol=1e-15)
    assert np.allclose(_dense_of(gold["K4"]), np.full((4, 4), 0.25), atol=1e-15)


def test_invariants_random_graph():
    rng = np.random.default_rng(7)
    n = 120
    src = rng.integers(0, n, 500)
    dst = rng.integers(0, n, 500)
    g = O.graph(n, src, dst)
    a = O.dense_adj(g)
    assert np.array_equal(a, a.T)                          # exact symmetry
    d = np.sqrt(g.deg.astype(np.float64))
    assert np.allclose(a @ d, d, rtol=1e-13)               # A_hat D^1/2 1 = D^1/2 1
    ev = np.linalg.eigvalsh(a)
    assert ev.max() == pytest.approx(1.0, abs=1e-12)
    assert ev.min() > -1.0 - 1e-12


def test_regular_graph_row_sums():
    # 3-regular circulant on 20 vertices plus loops: each row sums to 1
    n = 20
    src = np.r_[np.arange(n), np.arange(n)]
    dst = np.r_[(np.arange(n) + 1) % n, (np.arange(n) + 10) % n]
    g = O.graph(n, src, dst)
    assert np.all(g.deg == 4)
    assert np.allclose(O.dense_adj(g).sum(axis=1), 1.0, atol=1e-15)


def test_dinv_f32_is_rounded_fp64():
    g = O.graph(6, np.array([0, 0, 0, 1]), np.array([1, 2, 3, 2]))
    want = np.array([np.float32(1.0 / math.sqrt(float(d))) for d in g.deg], np.float32)
    assert np.array_equal(O.dinv_f32(g), want)


def test_transpose_matches_scipy():
    rng = np.random.default_rng(11)
    n = 50
    g = O.graph(n, rng.integers(0, n, 150), rng.integers(0, n, 150))
    vals = rng.standard_normal(g.nnz)                      # deliberately non-symmetric values
    gt, vt = O.transpose_csr(g, vals)
    m = sp.csr_matrix((vals, g.colidx, g.rowptr), shape=(n, n)).T.tocsr()
    m.sort_indices()
    assert np.array_equal(gt.rowptr, m.indptr)
    assert np.array_equal(gt.colidx, m.indices)
    assert np.allclose(vt, m.data, rtol=0, atol=0)


def test_spmm_matches_scipy_and_dense():
    rng = np.random.default_rng(5)
    n = 80
    g = O.graph(n, rng.integers(0, n, 300), rng.integers(0, n, 300))
    vals = O.norm_values(g)
    x = rng.standard_normal((n, 9))
    y = O.spmm(g, vals, x)
    ref = sp.csr_matrix((vals, g.colidx, g.rowptr), shape=(n, n)) @ x
    assert np.allclose(y, ref, rtol=1e-13, atol=1e-13)
    assert np.allclose(y, O.dense_adj(g) @ x, rtol=1e-13, atol=1e-13)
    # row blocks of a few entries (rows split across no block, a block per
    # row for rows longer than the budget) give the same sums
    for be in (1, 7, 64):
        assert np.array_equal(O.spmm(g, vals, x, block_entries=be), y)


def test_spmm_general_csr_with_empty_rows():
    # a CSR that is not of the form A + I: empty rows (first, inner, last),
    # repeated columns, rectangular use of X's rows
    rng = np.random.default_rng(11)
    n = 40
    counts = rng.integers(0, 6, n)
    counts[[0, 17, 18, n - 1]] = 0
    rowptr = np.zeros(n + 1, np.int64)
    np.cumsum(counts, out=rowptr[1:])
    colidx = rng.integers(0, n, rowptr[-1]).astype(np.int32)
    vals = rng.standard_normal(rowptr[-1])
    g = O.Graph(n, rowptr, colidx)
    x = rng.standard_normal((n, 5))
    ref = sp.csr_matrix((vals, colidx, rowptr), shape=(n, n)) @ x
    for be in (1, 3, 1 << 22):
        y = O.spmm(g, vals, x, block_entries=be)
        assert np.allclose(y, ref, rtol=1e-13, atol=1e-13)
        assert np.all(y[[0, 17, 18, n - 1]] == 0)


# ---------------------------------------------------------------- dropout RNG

def test_philox_matches_numpy():
    # numpy's Philox is Philox-4x64-10; it increments the counter before
    # producing a block, so block(c) == philox(c + 1).
    for ctr, key in [([0, 0, 0, 0], [0, 0]), ([5, 7, 9, 11], [123, 456]),
                     ([2**40 + 3, 2**33, 17, 2**62], [2**63 + 5, 2**61 + 9])]:
        bg = np.random.Philox(counter=np.array(ctr, np.uint64), key=np.array(key, np.uint64))
        ref = bg.random_raw(4)
        c1 = np.array([ctr], np.uint64)
        c1[0, 0] += np.uint64(1)
        mine = O.philox4x64(c1, np.array([key], np.uint64))[0]
        assert [int(x) for x in mine] == [int(x) for x in ref]


def test_dropout_p0_keeps_all_and_fraction():
    assert O.dropout_keep(1, 0, 0, 10, 7, 0.0).all()
    keep = O.dropout_keep(123, 1, 3, 500, 40, 0.5)
    n = keep.size
    frac = keep.mean()
    assert abs(frac - 0.5) < 5 * math.sqrt(0.25 / n)       # binomial 5-sigma
    keep3 = O.dropout_keep(123, 1, 3, 500, 40, 0.3)
    assert abs(keep3.mean() - 0.7) < 5 * math.sqrt(0.21 / n)
    # different epoch / layer / seed give different masks
    assert (keep != O.dropout_keep(123, 1, 4, 500, 40, 0.5)).mean() > 0.4
    assert (keep != O.dropout_keep(123, 2, 3, 500, 40, 0.5)).mean() > 0.4
    assert (keep != O.dropout_keep(124, 1, 3, 500, 40, 0.5)).mean() > 0.4


def test_philox4x32_known_answers():
    # the generator's published known-answer vectors (tests/golden)
    path = os.path.join(os.path.dirname(__file__), "golden", "philox4x32_10_kat.txt")
    rows = [ln.split() for ln in open(path) if ln.strip() and not ln.startswith("#")]
    assert len(rows) == 3
    for r in rows:
        v = [int(x, 16) for x in r]
        got = O.philox4x32(np.array([v[0:4]], np.uint64), np.array([v[4:6]], np.uint64))[0]
        assert [int(x) for x in got] == v[6:10]


def test_philox4x32_rounds_and_key_schedule():
    # brute force with Python integers of one round structure, independent of
    # numpy's uint64 arithmetic: 7 rounds at a random counter and key
    M0, M1, W0, W1 = 0xD2511F53, 0xCD9E8D57, 0x9E3779B9, 0xBB67AE85
    c = [0x01234567, 0x89ABCDEF, 0xDEADBEEF, 0x0BADF00D]
    k = [0xCAFEBABE, 0x12345678]
    x, kk = list(c), list(k)
    for r in range(7):
        p0, p1 = M0 * x[0], M1 * x[2]
        x = [(p1 >> 32) ^ x[1] ^ kk[0], p1 & 0xFFFFFFFF, (p0 >> 32) ^ x[3] ^ kk[1], p0 & 0xFFFFFFFF]
        kk = [(kk[0] + W0) & 0xFFFFFFFF, (kk[1] + W1) & 0xFFFFFFFF]
    got = O.philox4x32(np.array([c], np.uint64), np.array([k], np.uint64), rounds=7)[0]
    assert [int(v) for v in got] == x


def test_dropout_word_layout():
    # element e uses word e % 4 of block e // 4, counter (b lo, b hi, epoch,
    # layer), key (seed lo, seed hi): check two blocks by hand
    seed, layer, epoch = (7 << 32) + 99, 2, 5
    thr = int(math.floor(0.5 * 2**32))
    keep = O.dropout_keep(seed, layer, epoch, 4, 8, 0.5)  # 32 elements, blocks 6, 7 = row 3
    words = []
    for b in (6, 7):
        out = O.philox4x32(np.array([[b, 0, epoch, layer]], np.uint64), np.array([[99, 7]], np.uint64))[0]
        words += [int(x) for x in out]
    assert [bool(w >= thr) for w in words] == keep[3].tolist()
    # a block index past 2^32 carries into counter word 1
    e = np.array([(2**32 + 5) * 4 + 1], np.uint64)
    out = O.philox4x32(np.array([[5, 1, epoch, layer]], np.uint64), np.array([[99, 7]], np.uint64))[0]
    assert int(O.dropout_words(seed, layer, epoch, e)[0]) == int(out[1])


def test_dropout_scales_kept_by_two():
    rng = np.random.default_rng(0)
    n, f = 64, 16
    g = O.graph(n, np.zeros(0, np.int32), np.zeros(0, np.int32))   # A_hat = I
    h = rng.standard_normal((n, 8))
    w = rng.standard_normal((8, f))
    _, z, out = O.layer_fwd(g, O.norm_values(g), h, w, None, "relu", 0.5, True, 7, 1, 0)
    keep = O.dropout_keep(7, 1, 0, n, f, 0.5)
    assert np.array_equal(out[keep], 2.0 * np.maximum(z, 0)[keep])
    assert np.all(out[~keep] == 0)


# ---------------------------------------------------------------- layer math

def _small_problem(seed=0, n=40, fin=6, fh=5, c=4, e=90):
    rng = np.random.default_rng(seed)
    g = O.graph(n, rng.integers(0, n, e), rng.integers(0, n, e))
    vals = O.norm_values(g)
    x = rng.standard_normal((n, fin))
    w1 = rng.standard_normal((fin, fh)) * 0.5
    b1 = rng.standard_normal(fh) * 0.1
    w2 = rng.standard_normal((fh, c)) * 0.5
    b2 = rng.standard_normal(c) * 0.1
    y = rng.integers(0, c, n)
    mask = rng.random(n) < 0.6
    return rng, g, vals, x, w1, b1, w2, b2, y, mask


def test_identity_graph_reduces_to_dense_layer():
    rng = np.random.default_rng(2)
    n = 30
    g = O.graph(n, np.zeros(0, np.int32), np.zeros(0, np.int32))
    h = rng.standard_normal((n, 7))
    w = rng.standard_normal((7, 3))
    b = rng.standard_normal(3)
    s, z, out = O.layer_fwd(g, O.norm_values(g), h, w, b, "relu", 0.0)
    ref = np.einsum("ik,kj->ij", h, w) + b
    assert np.allclose(z, ref, rtol=1e-14)
    assert np.allclose(out, np.maximum(ref, 0))


def test_featureless_input_gives_weights():
    # X = I (the paper's default featureless input): S = W
    rng = np.random.default_rng(4)
    n = 12
    g = O.graph(n, rng.integers(0, n, 20), rng.integers(0, n, 20))
    w = rng.standard_normal((n, 5))
    s, z, _ = O.layer_fwd(g, O.norm_values(g), np.eye(n), w, None, "none")
    assert np.array_equal(s, w)
    assert np.allclose(z, O.dense_adj(g) @ w, rtol=1e-13)


def test_dense_and_csr_forward_agree():
    _, g, vals, x, w1, b1, *_ = _small_problem(1)
    a = O.dense_adj(g, vals)
    for act in ("relu", "none"):
        r1 = O.layer_fwd(g, vals, x, w1, b1, act, 0.5, True, 3, 0, 1)
        r2 = O.layer_fwd(g, vals, x, w1, b1, act, 0.5, True, 3, 0, 1, dense=a)
        for u, v in zip(r1, r2):
            assert np.allclose(u, v, rtol=1e-13, atol=1e-13)


def test_permutation_equivariance():
    _, g, vals, x, w1, b1, *_ = _small_problem(3)
    n = g.n
    perm = np.random.default_rng(9).permutation(n)
    inv = np.argsort(perm)
    rows = g.rows()
    # relabel vertex v -> inv[v]
    src = inv[rows]
    dst = inv[g.colidx]
    gp = O.graph(n, src, dst)
    _, z, _ = O.layer_fwd(g, vals, x, w1, b1, "none")
    _, zp, _ = O.layer_fwd(gp, O.norm_values(gp), x[perm], w1, b1, "none")
    assert np.allclose(zp, z[perm], rtol=1e-12, atol=1e-12)


def test_adjoint_identity():
    rng, g, vals, *_ = _small_problem(5)
    vals = rng.standard_normal(g.nnz)                      # generic, non-symmetric A
    x = rng.standard_normal((g.n, 3))
    y = rng.standard_normal((g.n, 3))
    gt, vt = O.transpose_csr(g, vals)
    lhs = np.sum(O.spmm(g, vals, x) * y)
    rhs = np.sum(x * O.spmm(gt, vt, y))
    assert lhs == pytest.approx(rhs, rel=1e-12)


def test_softmax_ce_closed_forms():
    n, c = 10, 7
    z = np.full((n, c), 0.3)
    y = np.arange(n) % c
    mask = np.zeros(n, bool)
    mask[[1, 4, 6]] = True
    loss, d, nc = O.softmax_ce(z, y, mask, loss_scale=8.0)
    assert loss == pytest.approx(math.log(c), rel=1e-15)
    want = np.zeros((n, c))
    for i in np.flatnonzero(mask):
        want[i] = 1.0 / c
        want[i, y[i]] -= 1.0
    assert np.allclose(d, want * 8.0 / 3, rtol=1e-14, atol=1e-16)
    # uniform logits: arg-max ties resolve to class 0
    assert nc == int(np.sum(y[mask] == 0))


def _loss_of(params, g, vals, x, y, mask, p, seed):
    w1, b1, w2, b2 = params
    _, _, h1 = O.layer_fwd(g, vals, x, w1, b1, "relu", p, True, seed, 0, 0)
    _, z2, _ = O.layer_fwd(g, vals, h1, w2, b2, "none")
    return O.softmax_ce(z2, y, mask)[0]


def test_two_layer_gradients_finite_difference():
    _, g, vals, x, w1, b1, w2, b2, y, mask = _small_problem(6)
    p, seed = 0.5, 77
    params = [w1, b1, w2, b2]
    s1, z1, h1 = O.layer_fwd(g, vals, x, w1, b1, "relu", p, True, seed, 0, 0)
    _, z2, _ = O.layer_fwd(g, vals, h1, w2, b2, "none")
    _, dz2, _ = O.softmax_ce(z2, y, mask)
    _, dw2, db2, dz1 = O.layer_bwd(g, vals, h1, w2, dz2, "relu", p)
    _, dw1, db1, _ = O.layer_bwd(g, vals, x, w1, dz1, "none", 0.0, need_dh=False)
    assert np.min(np.abs(z1)) > 1e-4                       # away from ReLU kinks
    grads = [dw1, db1, dw2, db2]
    h = 1e-6
    rng = np.random.default_rng(0)
    for k, (par, gr) in enumerate(zip(params, grads)):
        flat = par.reshape(-1)
        for idx in rng.choice(flat.size, size=min(flat.size, 8), replace=False):
            old = flat[idx]
            flat[idx] = old + h
            lp = _loss_of(params, g, vals, x, y, mask, p, seed)
            flat[idx] = old - h
            lm = _loss_of(params, g, vals, x, y, mask, p, seed)
            flat[idx] = old
            fd = (lp - lm) / (2 * h)
            assert gr.reshape(-1)[idx] == pytest.approx(fd, rel=1e-5, abs=1e-9), (k, idx)


def test_input_gradient_finite_difference():
    # gradient w.r.t. the layer input H through a non-symmetric A
    rng, g, vals, x, w1, b1, *_ = _small_problem(8)
    vals = rng.uniform(0.1, 1.0, g.nnz)
    r = rng.standard_normal((g.n, w1.shape[1]))

    def f(xx):
        return np.sum(O.layer_fwd(g, vals, xx, w1, b1, "none")[1] * r)

    _, dw, db, dx = O.layer_bwd(g, vals, x, w1, r, "none", 0.0)
    h = 1e-6
    for i, j in [(0, 0), (5, 2), (17, 4), (33, 1)]:
        xp = x.copy(); xp[i, j] += h
        xm = x.copy(); xm[i, j] -= h
        assert dx[i, j] == pytest.approx((f(xp) - f(xm)) / (2 * h), rel=1e-6, abs=1e-9)
    assert np.allclose(db, r.sum(axis=0))


def test_relu_dropout_mask_in_backward():
    # dZ_below is zero exactly where H is zero and scaled by 1/(1-p) elsewhere
    rng = np.random.default_rng(12)
    n = 16
    g = O.graph(n, np.zeros(0, np.int32), np.zeros(0, np.int32))
    h = np.maximum(rng.standard_normal((n, 4)), 0) * 2.0
    w = rng.standard_normal((4, 3))
    dz = rng.standard_normal((n, 3))
    _, _, _, dzb = O.layer_bwd(g, O.norm_values(g), h, w, dz, "relu", 0.5)
    dh = dz @ w.T
    assert np.all(dzb[h == 0] == 0)
    assert np.allclose(dzb[h > 0], 2.0 * dh[h > 0], rtol=1e-15)


# ---------------------------------------------------------------- optimiser

def test_adam_first_step_closed_form():
    g = np.array([3.0, -0.5, 1e-3, -7.0])
    st_ = O.AdamState(4)
    sc = O.LossScaler(scale=1024.0)
    w0 = np.array([1.0, 2.0, 3.0, 4.0])
    w1, applied = O.adam_step(w0, g * 1024.0, st_, sc, lr=0.01)
    assert applied
    # m_hat = g, v_hat = g^2: every coordinate moves by lr * g / (|g| + eps)
    assert np.allclose(w1, w0 - 0.01 * g / (np.abs(g) + 1e-8), rtol=1e-15)


def test_adam_constant_gradient_closed_form_over_many_steps():
    # a constant gradient g keeps m_t = (1 - b1^t) g and v_t = (1 - b2^t) g^2,
    # so the bias-corrected moments are exactly g and g^2 at every step t and
    # each step moves theta by lr * g / (|g| + eps) (Kingma & Ba); after T
    # steps theta_T = theta_0 - T lr g / (|g| + eps).  A dropped bias
    # correction, a swapped beta or a missing square root breaks this from
    # the second step on.
    g = np.array([3.0, -0.5, 1e-3, -7.0, 1e-8, -2e-8])
    w0 = np.array([1.0, 2.0, 3.0, 4.0, 5.0, 6.0])
    st_ = O.AdamState(g.size)
    sc = O.LossScaler(scale=256.0, interval=10**9)
    w = w0
    T = 25
    for t in range(T):
        w, applied = O.adam_step(w, g * 256.0, st_, sc, lr=0.01)
        assert applied
    assert st_.t == T
    assert np.allclose(w, w0 - T * 0.01 * g / (np.abs(g) + 1e-8), rtol=1e-13, atol=0)


def test_adam_overflow_skips_and_backs_off():
    st_ = O.AdamState(3)
    sc = O.LossScaler(scale=2.0**16)
    w0 = np.array([1.0, 2.0, 3.0])
    w1, applied = O.adam_step(w0, np.array([1.0, np.inf, 0.0]), st_, sc)
    assert not applied and np.array_equal(w1, w0)
    assert sc.scale == 2.0**15 and st_.t == 0
    w2, applied = O.adam_step(w0, np.array([np.nan, 0, 0]), st_, sc)
    assert not applied and sc.scale == 2.0**14


def test_loss_scaler_script():
    sc = O.LossScaler(scale=4.0, interval=3, min_scale=1.0, max_scale=16.0)
    seq = [False, False, False, True, True, True, False, False, False, False, False, False,
           False, False, False, False, False, False]
    states = []
    for ov in seq:
        sc.update(ov)
        states.append((sc.scale, sc.good))
    assert states[:3] == [(4.0, 1), (4.0, 2), (8.0, 0)]
    assert states[3:6] == [(4.0, 0), (2.0, 0), (1.0, 0)]           # clamps at min
    assert states[6:9] == [(1.0, 1), (1.0, 2), (2.0, 0)]
    assert states[9:15] == [(2.0, 1), (2.0, 2), (4.0, 0), (4.0, 1), (4.0, 2), (8.0, 0)]
    assert states[15:18] == [(8.0, 1), (8.0, 2), (16.0, 0)]
    sc.update(False); sc.update(False); sc.update(False)
    assert sc.scale == 16.0                                         # clamps at max


# ------------------------------------------- storage rounding, O3 optimiser

def _binary16_values():
    """Every finite non-negative binary16 value from the format's fields:
    (-1)^s 2^(E - 15) (1 + f / 1024) for E in 1..30, 2^-14 (f / 1024) for E = 0."""
    E = np.arange(32)[:, None]
    f = np.arange(1024)[None, :]
    normal = np.exp2(E - 15.0) * (1.0 + f / 1024.0)
    sub = np.exp2(-14.0) * (f / 1024.0)
    vals = np.where(E == 0, sub, normal)[:31].ravel()
    return np.sort(vals)


def test_round_to_binary16_fixed_points_and_midpoints():
    v = _binary16_values()
    assert v[-1] == 65504.0 and v[1] == 2.0**-24
    assert np.array_equal(O.round_to(v, "f16"), v)
    assert np.array_equal(O.round_to(-v, "f16"), -v)
    # the midpoint of two neighbours rounds to the one with an even fraction
    # field (the even multiple of the local spacing); just off the midpoint,
    # to the nearer one
    lo, hi = v[:-1], v[1:]
    mid = (lo + hi) / 2.0
    spacing = hi - lo
    even_lo = np.mod(np.round(lo / spacing), 2.0) == 0.0
    assert np.array_equal(O.round_to(mid, "f16"), np.where(even_lo, lo, hi))
    assert np.array_equal(O.round_to(mid - spacing / 8, "f16"), lo)
    assert np.array_equal(O.round_to(mid + spacing / 8, "f16"), hi)


def test_round_to_binary16_hand_values():
    cases = [(65504.0, 65504.0), (65519.99, 65504.0), (65520.0, np.inf),      # tie above the max: to even (overflow)
             (1e6, np.inf), (2.0**-24, 2.0**-24), (2.0**-25, 0.0),           # tie at the bottom: to even (zero)
             (3 * 2.0**-26, 2.0**-24), (1 + 2.0**-11, 1.0), (1 + 3 * 2.0**-11, 1 + 2.0**-9),
             (1e-8, 0.0), (0.1, 0.0999755859375), (-0.1, -0.0999755859375)]
    x = np.array([c[0] for c in cases])
    want = np.array([c[1] for c in cases])
    assert np.array_equal(O.round_to(x, "f16"), want)
    z = O.round_to(np.array([-0.0, np.inf, -np.inf, np.nan]), "f16")
    assert np.signbit(z[0]) and z[1] == np.inf and z[2] == -np.inf and np.isnan(z[3])


def test_round_storage_f16_matches_numpy_conversion():
    rng = np.random.default_rng(3)
    x = (rng.standard_normal(200_000) * np.exp2(rng.uniform(-30, 18, 200_000))).astype(np.float32)
    with np.errstate(over="ignore"):
        want = x.astype(np.float16).astype(np.float64)
    assert np.array_equal(O.round_storage(x, "f16"), want)


def test_round_storage_bf16_two_formulations_agree():
    rng = np.random.default_rng(4)
    with np.errstate(over="ignore"):
        x = (rng.standard_normal(200_000) * np.exp2(rng.uniform(-140, 127, 200_000))).astype(np.float32)
    x = np.concatenate([x, np.float32([3.4028235e38, -3.4028235e38, 1e-45, 0.0, -0.0, np.inf])])
    a = O.round_storage(x, "bf16")          # encoding-level rounding
    b = O.round_to(x.astype(np.float64), "bf16")   # spacing-level rounding
    assert np.array_equal(a, b)
    hand = O.round_storage(np.float32([1 + 2.0**-8, 1 + 3 * 2.0**-8, 0.1, 3.4028235e38]), "bf16")
    assert np.array_equal(hand, [1.0, 1.015625, 0.10009765625, np.inf])
    assert np.isnan(O.round_storage(np.float32([np.nan]), "bf16")[0])


def test_adam_half_first_step_large_gradient_matches_adam():
    # |g| well inside binary16's range: the O3 step lands within rounding of
    # the exact first Adam step, w - lr g / (|g| + eps)
    g = np.array([0.5, -0.75, 0.25, 1.0])
    w0 = O.round_to(np.array([1.0, -2.0, 0.3, 0.05]), "f16")
    z = np.zeros(4)
    w1, m1, v1 = O.adam_step_half(w0, g.astype(np.float32), z, z, 1, "f16", lr=0.01)
    exact = w0 - 0.01 * g / (np.abs(g) + 1e-8)
    ulp = np.exp2(np.floor(np.log2(np.abs(exact))) - 10)
    assert np.all(np.abs(w1 - exact) <= 2 * ulp)
    assert np.array_equal(O.round_to(w1, "f16"), w1)


def test_adam_half_small_gradient_underflows_to_infinity():
    # (1 - b2) g^2 = 1e-3 * (1e-3)^2 = 1e-9 lies below half of binary16's
    # smallest subnormal 2^-24 (about 6e-8), so v rounds to 0; eps = 1e-8
    # rounds to 0 too, and the update m_hat / 0 is infinite
    w0 = np.array([1.0, 1.0])
    g = np.float32([1e-3, -1e-3])
    w1, m1, v1 = O.adam_step_half(w0, g, np.zeros(2), np.zeros(2), 1, "f16")
    assert np.array_equal(v1, [0.0, 0.0])
    assert w1[0] == -np.inf and w1[1] == np.inf
    # with zero gradient and zero moments the update is 0 / 0
    w2, _, _ = O.adam_step_half(w0, np.float32([0.0, 0.0]), np.zeros(2), np.zeros(2), 1, "f16")
    assert np.all(np.isnan(w2))
    # bf16 has binary32's exponent range: the same step stays finite and
    # within rounding of the exact step
    w3, _, v3 = O.adam_step_half(w0, g, np.zeros(2), np.zeros(2), 1, "bf16")
    assert np.all(v3 > 0)
    assert np.all(np.abs(w3 - (1.0 - 0.01 * np.sign(g))) <= 2 * 2.0**-8)


def test_adam_half_first_moment_is_binary32_then_binary16():
    """O3 reading: each elementwise line is evaluated in binary32, one
    rounding per arithmetic operation, and the line's result is rounded to
    binary16.  A case where that differs from rounding the line's exact
    value once, derived with integers:

    b1 = binary32(0.9) = 15099494 * 2^-24, so 1 - b1 = 1677722 * 2^-24
    (exact: the operands are within a factor 2).  Take m = -1355 * 2^-11
    = -0.66162109375 and g = 5 * 2^-4 = 0.3125 (both binary16).
      b1 * m        = -20459814370 * 2^-35 exactly (35 bits); in binary32
                      (24 bits: multiples of 2^11 units) -20459814912 * 2^-35.
      (1 - b1) * g  = 8388610 * 2^-28 = 1073742080 * 2^-35 (exact in binary32).
      binary32 sum  = -19386072832 * 2^-35, rounded to a multiple of 2^11:
                      -19386073088 * 2^-35 = -1155.5 * 2^-11, which is the
                      midpoint of the binary16 neighbours -1155 * 2^-11 and
                      -1156 * 2^-11; ties to even give -1156 * 2^-11.
      exact sum     = -19386072290 * 2^-35 = -1155.49995... * 2^-11, which
                      rounds once to -1155 * 2^-11.
    So m' = -0.564453125 under the binary32 reading and -0.56396484375
    under round-once."""
    bm = 15099494 * -1355                       # b1 * m in units of 2^-35
    assert bm == -20459814370
    q, r = divmod(-bm, 2048)                    # binary32 keeps 24 bits: 2^11-unit multiples
    bm32 = -(q + (r > 1024 or (r == 1024 and q % 2 == 1))) * 2048
    assert bm32 == -20459814912
    og = (2**24 - 15099494) * 5 * 128           # (1 - b1) g in units of 2^-35
    assert og == 1073742080
    q, r = divmod(-(bm32 + og), 2048)
    s32 = -(q + (r > 1024 or (r == 1024 and q % 2 == 1))) * 2048
    assert s32 == -1155 * 2**24 - 2**23          # exactly the binary16 midpoint
    assert (bm + og) > s32                      # the exact sum lies above it (towards -1155)
    m1 = np.array([-1355 * 2.0**-11])
    w1, m2, v2 = O.adam_step_half(np.array([0.5]), np.float32([0.3125]), m1, np.array([0.25]), 2, "f16")
    assert m2[0] == -1156 * 2.0**-11 == -0.564453125


def test_adam_half_tracks_fp64_adam_for_large_gradients():
    rng = np.random.default_rng(5)
    n = 64
    w = O.round_to(rng.uniform(-1, 1, n), "f16")
    m = np.zeros(n)
    v = np.zeros(n)
    ref = w.copy()
    st_ = O.AdamState(n)
    sc = O.LossScaler(scale=1.0)
    for t in range(1, 4):
        g = (rng.choice([-1, 1], n) * rng.uniform(0.1, 1.0, n)).astype(np.float32)
        w, m, v = O.adam_step_half(w, g, m, v, t, "f16", lr=0.001)
        ref, _ = O.adam_step(ref, g.astype(np.float64), st_, sc, lr=0.001)
    # three updates of about lr each: binary16 rounding of w (spacing
    # <= 2^-11 on [-1, 1]) bounds the difference
    assert np.max(np.abs(w - ref)) <= 4 * 2.0**-11


def test_sampled_graph_helpers_match_full_graph():
    rng = np.random.default_rng(21)
    n = 400
    src = rng.integers(0, n, 3000)
    dst = rng.integers(0, n, 3000)
    g = O.graph(n, src, dst)
    assert np.array_equal(O.graph_degrees(n, src, dst), g.deg)
    rows = [0, 5, 17, 399]
    nb = O.graph_rows(n, src, dst, rows)
    for r in rows:
        assert np.array_equal(nb[r], g.colidx[g.rowptr[r]:g.rowptr[r + 1]])


def test_dropout_keep_rows_matches_full_mask():
    full = O.dropout_keep(77, 3, 9, 50, 13, 0.4)
    rows = [0, 7, 49, 23]
    assert np.array_equal(O.dropout_keep_rows(77, 3, 9, rows, 13, 0.4), full[rows])


def test_norm_adj_matvec_matches_csr_product():
    rng = np.random.default_rng(22)
    n = 300
    src = rng.integers(0, n, 2000)
    dst = rng.integers(0, n, 2000)
    g = O.graph(n, src, dst)
    y = rng.standard_normal((n, 3))
    want = O.spmm(g, O.norm_values(g), y)
    assert np.allclose(O.norm_adj_matvec(n, src, dst, y), want, rtol=1e-13, atol=1e-13)
    assert np.allclose(O.norm_adj_matvec(n, src, dst, y[:, 0]), want[:, 0], rtol=1e-13, atol=1e-13)


# ------------------------------------------------------ link prediction (Eq. 2)

def _numpy_philox_block(ctr, key):
    """One Philox-4x64-10 block from numpy's generator (an implementation
    independent of the oracle's): numpy increments the counter before it
    produces a block (ctr[0] >= 1 here, so no carry)."""
    c = np.array(ctr, np.uint64)
    assert c[0] >= 1
    c[0] -= np.uint64(1)
    return np.random.Philox(counter=c, key=np.array(key, np.uint64)).random_raw(4)


def test_sample_pairs_draws_and_layout():
    rng = np.random.default_rng(31)
    n = 1000
    eu = rng.integers(0, n, 300).astype(np.int32)
    ev = (eu + 1 + rng.integers(0, n - 1, 300)).astype(np.int32) % n
    seed, epoch, n_pos, n_neg = 2**40 + 7, 3, 500, 700
    u, v = O.sample_pairs(seed, epoch, n, eu, ev, n_pos, n_neg)
    # pairs by hand from numpy's Philox: positives 1 and n_pos - 1, negatives n_pos and last
    for k in (1, n_pos - 1, n_pos, n_pos + n_neg - 1):
        w = _numpy_philox_block([k, epoch, 0, 0], [seed, O.PAIR_STREAM])
        if k < n_pos:
            e = int(w[0]) % eu.size
            assert (u[k], v[k]) == (eu[e], ev[e])
        else:
            uu = int(w[0]) % n
            assert (u[k], v[k]) == (uu, (uu + 1 + int(w[1]) % (n - 1)) % n)
    # positives are training edges; negatives are distinct vertices in range
    edges = set(zip(eu.tolist(), ev.tolist()))
    assert all((a, b) in edges for a, b in zip(u[:n_pos].tolist(), v[:n_pos].tolist()))
    assert np.all(u[n_pos:] != v[n_pos:]) and u.min() >= 0 and v.max() < n
    # roughly uniform negatives (mean of a uniform id over [0, n) within 5 sigma)
    sd = math.sqrt((n * n - 1) / 12 / n_neg)
    assert abs(u[n_pos:].mean() - (n - 1) / 2) < 5 * sd
    # another epoch gives other pairs
    u2, _ = O.sample_pairs(seed, epoch + 1, n, eu, ev, n_pos, n_neg)
    assert (u2 != u).mean() > 0.9


def test_pair_loss_closed_forms():
    rng = np.random.default_rng(32)
    n, f, n_pos, n_neg = 50, 6, 30, 40
    u = rng.integers(0, n, n_pos + n_neg)
    v = (u + 1 + rng.integers(0, n - 1, n_pos + n_neg)) % n
    # Z = 0: every score 0, loss = log 2, g = S (1/2 - y) / K
    loss, s, g = O.pair_loss(np.zeros((n, f)), u, v, n_pos, loss_scale=8.0)
    assert s.tolist() == [0.0] * u.size
    assert abs(loss - math.log(2.0)) < 1e-15
    y = (np.arange(u.size) < n_pos)
    assert np.allclose(g, 8.0 * (0.5 - y) / u.size, rtol=0, atol=1e-17)
    # textbook binary cross-entropy -[y log p + (1 - y) log (1 - p)], p = sigmoid(s)
    z = 0.4 * rng.standard_normal((n, f))
    loss, s, g = O.pair_loss(z, u, v, n_pos)
    p = 1.0 / (1.0 + np.exp(-s))
    want = -np.mean(np.where(y, np.log(p), np.log(1.0 - p)))
    assert abs(loss - want) < 1e-12
    assert np.allclose(s, [z[a] @ z[b] for a, b in zip(u, v)], rtol=1e-13, atol=1e-13)
    # large scores stay finite (stable softplus / sigmoid)
    zz = np.zeros((n, f)); zz[:, 0] = 40.0
    loss, s, g = O.pair_loss(zz, u, v, n_pos)
    assert np.isfinite(loss) and np.all(np.isfinite(g))
    assert abs(loss - n_neg * 1600.0 / u.size) < 1e-9    # negatives pay ~s, positives ~0


def test_pair_gradient_finite_differences():
    rng = np.random.default_rng(33)
    n, f, n_pos, n_neg = 20, 5, 25, 25
    u = rng.integers(0, n, n_pos + n_neg)
    v = (u + 1 + rng.integers(0, n - 1, n_pos + n_neg)) % n
    z = 0.5 * rng.standard_normal((n, f))
    _, _, g = O.pair_loss(z, u, v, n_pos)
    dz = O.pair_backward(n, z, u, v, g)
    h = 1e-6
    for r, c in [(0, 0), (3, 2), (int(u[0]), 4), (int(v[7]), 1), (19, 3)]:
        zp, zm = z.copy(), z.copy()
        zp[r, c] += h
        zm[r, c] -= h
        fd = (O.pair_loss(zp, u, v, n_pos)[0] - O.pair_loss(zm, u, v, n_pos)[0]) / (2 * h)
        assert abs(dz[r, c] - fd) < 1e-8, (r, c, dz[r, c], fd)
    # rows that appear in no pair get zero
    unused = np.setdiff1d(np.arange(n), np.concatenate([u, v]))
    assert np.all(dz[unused] == 0)


def test_auc_ap_match_sklearn():
    from sklearn.metrics import average_precision_score, roc_auc_score
    rng = np.random.default_rng(34)
    for p, q in [(50, 70), (200, 200), (7, 3)]:
        sp = np.round(rng.standard_normal(p) + 0.7, 1)     # rounded: many ties
        sn = np.round(rng.standard_normal(q), 1)
        auc, ap = O.auc_ap(sp, sn)
        y = np.r_[np.ones(p), np.zeros(q)]
        sc = np.r_[sp, sn]
        assert abs(auc - roc_auc_score(y, sc)) < 1e-12
        assert abs(ap - average_precision_score(y, sc)) < 1e-12
    assert O.auc_ap([2.0, 3.0], [0.0, 1.0]) == (1.0, 1.0)
    assert O.auc_ap([0.0], [1.0])[0] == 0.0
