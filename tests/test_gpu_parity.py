"""GPU parity: every libgcn call against the CPU fp64 oracle on the same
seeded inputs.  Integer outputs are compared bit-exactly; floating-point
outputs to the tolerances in tests/parity.py (fp32: 1e-5 normwise; fp16:
2e-2 per element with the tensor RMS as floor; bf16: 1e-1 provisional)."""
import numpy as np
import pytest
import torch

from oracle import gcn_oracle as O
from paper_2010_12635_amd import gcn as G
from paper_2010_12635_amd import inputs as I
from paper_2010_12635_amd.model import DeviceGraph, GCN2, round8
from tests.parity import assert_close, f32, hub_graph, tol_for

pytestmark = pytest.mark.gpu

PRECS = [G.GCN_F32, G.GCN_F16, G.GCN_BF16]
PNAME = {0: "f32", 1: "f16", 2: "bf16"}


def dev():
    return torch.device("cuda:0")


def to_dev(a, prec, ld=None):
    a = np.asarray(a, np.float32)
    n, f = a.shape
    ld = ld or round8(f)
    t = torch.zeros((n, ld), dtype=G.torch_dtype(prec), device=dev())
    t[:, :f] = torch.as_tensor(a).to(dev()).to(G.torch_dtype(prec))
    return t


def host(t, f=None):
    # the logical columns only (padding may hold any bits)
    if f is not None:
        t = t[:, :f]
    return t.float().cpu().numpy().astype(np.float64)


def rounded(a, prec):
    """The values the device actually holds for a host array in `prec`."""
    return torch.as_tensor(np.asarray(a, np.float32)).to(G.torch_dtype(prec)).float().numpy().astype(np.float64)


# ------------------------------------------------------------- normalize ----

@pytest.mark.parametrize("index", [G.GCN_I32, G.GCN_I64])
def test_normalize_bit_exact(index):
    n = 6000
    # one hub above the LDS sort limit (4096), medium hubs, many small rows
    src, dst = hub_graph(n, 20000, [(7, 5000), (100, 700), (200, 90), (300, 64)], seed=1)
    g = O.graph(n, src, dst)
    dg = DeviceGraph(n, src, dst, prec=G.GCN_F32, index=index, schedule=False)
    rp, ci = dg.csr_host()
    assert dg.nnz == g.nnz
    assert np.array_equal(rp, g.rowptr)
    assert np.array_equal(ci, g.colidx)
    assert np.array_equal(dg.deg.cpu().numpy(), g.deg)
    assert np.array_equal(dg.dinv.cpu().numpy(), O.dinv_f32(g))
    vals = dg.values[: dg.nnz].cpu().numpy().astype(np.float64)
    assert np.max(np.abs(vals - O.norm_values(g)) / O.norm_values(g)) < 3e-7
    # run-to-run identical
    dg2 = DeviceGraph(n, src, dst, prec=G.GCN_F32, index=index, schedule=False)
    assert np.array_equal(dg2.csr_host()[1], ci)


def untile(flat, n, prec):
    """Row-major n x n from the tiled operand layout documented in gcn.h."""
    kc = 16 if prec == G.GCN_F32 else 32
    ve = kc // 4
    nc = (n + kc - 1) // kc
    i = np.arange(n)[:, None]
    j = np.arange(n)[None, :]
    off = (((i // 64) * nc + j // kc) * 4 + (i % 64) // 16) * (16 * kc) + ((j % kc) // ve * 16 + i % 16) * ve + j % ve
    assert flat.size == ((n + 63) // 64) * 64 * nc * kc
    return flat[off]


@pytest.mark.parametrize("prec", [G.GCN_F16, G.GCN_F32, G.GCN_BF16], ids=lambda p: PNAME[p])
@pytest.mark.parametrize("tiled", [False, True], ids=["rowmajor", "tiled"])
def test_normalize_dense(prec, tiled):
    n = 700
    src, dst = hub_graph(n, 3000, [(3, 300)], seed=2)
    g = O.graph(n, src, dst)
    dg = DeviceGraph(n, src, dst, prec=prec, dense=True, tiled=tiled)
    want = O.dense_adj(g)
    if tiled:
        flat = dg.dense.float().cpu().numpy().astype(np.float64)
        got = untile(flat, n, prec)
        # padding entries (outside n x n) are zero
        assert np.count_nonzero(flat) == np.count_nonzero(got)
    else:
        got = dg.dense[:, :n].float().cpu().numpy().astype(np.float64)
    assert np.array_equal(got != 0, want != 0)
    assert_close(got, want, prec, "dense A_hat")


def test_normalize_empty_and_bad_ids():
    dg = DeviceGraph(37, np.zeros(0, np.int32), np.zeros(0, np.int32), prec=G.GCN_F32)
    rp, ci = dg.csr_host()
    assert np.array_equal(rp, np.arange(38)) and np.array_equal(ci, np.arange(37))
    assert np.all(dg.dinv.cpu().numpy() == 1.0)
    with pytest.raises(G.GcnError) as e:
        DeviceGraph(10, np.array([0, 3], np.int32), np.array([1, 10], np.int32))
    assert e.value.status == 8


def _expected_pieces(g, heavy, chunk, parts):
    """Pieces of the heavy rows as the schedule defines them: each row's
    entries cut where the column range floor(c P / n) changes, then every
    `chunk` entries; returns (first entry of each piece, pieces per row)."""
    n = g.n
    begs, counts = [], []
    for r in heavy:
        a0, a1 = int(g.rowptr[r]), int(g.rowptr[r + 1])
        cols = g.colidx[a0:a1].astype(np.int64)
        rng = cols * parts // n
        cuts = [a0 + int(np.searchsorted(rng, q + 1, side="left")) for q in range(parts - 1)]
        bounds = [a0] + cuts + [a1]
        k0 = len(begs)
        for a, b in zip(bounds[:-1], bounds[1:]):
            begs.extend(range(a, b, chunk))
        counts.append(len(begs) - k0)
    return np.array(begs, np.int64), np.array(counts, np.int64)


@pytest.mark.parametrize("parts", [1, 8, 16])
def test_schedule_lists_heavy_rows(parts):
    n = 3000
    # hub 1234 has more than GCN_FIX_BIG_PIECES pieces of 64 entries; about
    # 2 % of the vertices are isolated
    src, dst = hub_graph(n, 3000, [(5, 400), (17, 120), (2999, 1000), (1234, 4000)], seed=3)
    g = O.graph(n, src, dst)
    dg = DeviceGraph(n, src, dst, prec=G.GCN_F16, heavy_threshold=32, chunk_nnz=64, col_parts=parts)
    a = dg.adj
    assert a.col_parts == parts
    heavy = np.flatnonzero(g.deg > 32)
    assert a.n_heavy == heavy.size
    # read the schedule arrays back through their device addresses
    base = dg.sched
    off = lambda p: (p - base.data_ptr())
    rd = lambda ptr, count, dt, sz: base[off(ptr): off(ptr) + sz * count].view(dt).cpu().numpy()
    rows = rd(a.heavy_rows, a.n_heavy, torch.int32, 4)
    assert np.array_equal(rows, heavy)
    want_beg, want_cnt = _expected_pieces(g, heavy, 64, parts)
    cho = rd(a.heavy_chunk_off, a.n_heavy + 1, torch.int32, 4)
    assert np.array_equal(cho, np.concatenate([[0], np.cumsum(want_cnt)]))
    assert a.n_chunks == want_beg.size
    beg = rd(a.chunk_beg, a.n_chunks + 1, torch.int64, 8)
    assert np.array_equal(beg[:-1], want_beg) and beg[-1] == g.nnz
    owner = rd(a.chunk_heavy, a.n_chunks, torch.int32, 4)
    assert np.array_equal(owner, np.repeat(np.arange(heavy.size), want_cnt))
    # light rows: every row with deg <= threshold exactly once, degree
    # non-increasing (below 2^20 rows the order is one global degree order)
    perm = rd(a.row_perm, a.n_light, torch.int32, 4)
    light = np.flatnonzero(g.deg <= 32)
    assert a.n_light == light.size
    assert np.array_equal(np.sort(perm), light)
    assert np.all(np.diff(g.deg[perm]) <= 0)
    # the rows of one entry (isolated vertices) are the last n_light_single
    assert a.n_light_single == np.count_nonzero(g.deg[light] == 1) > 0
    assert np.all(g.deg[perm[a.n_light - a.n_light_single:]] == 1)
    # launch order: every piece once, first columns in non-decreasing
    # buckets, the pieces of column range q in chunk_order[part_off[q] ..
    # part_off[q + 1]), and part_slots the most pieces of one XCD
    order = rd(a.chunk_order, a.n_chunks, torch.int32, 4)
    assert np.array_equal(np.sort(order), np.arange(a.n_chunks))
    first_col = g.colidx[want_beg].astype(np.int64)
    assert np.all(np.diff(first_col[order] * 4096 // n) >= 0)
    # 16-byte descriptors: light rows {first entry, row, length} in row_perm
    # order; pieces {first entry, row, length | 2^31 for a row's only piece}
    # in launch order, and the launch position of every piece
    ld = rd(a.row_desc, a.n_light * 4, torch.int32, 4).reshape(-1, 4)
    assert np.array_equal(ld[:, 0].astype(np.uint32).astype(np.int64) + (ld[:, 1].astype(np.int64) << 32),
                          g.rowptr[perm])
    assert np.array_equal(ld[:, 2], perm) and np.array_equal(ld[:, 3], g.deg[perm])
    pd = rd(a.piece_desc, a.n_chunks * 4, torch.int32, 4).reshape(-1, 4)
    ends = np.minimum(beg[1:], g.rowptr[heavy[owner] + 1])
    single = np.repeat(want_cnt == 1, want_cnt)
    assert np.array_equal(pd[:, 0].astype(np.uint32).astype(np.int64) + (pd[:, 1].astype(np.int64) << 32),
                          want_beg[order])
    assert np.array_equal(pd[:, 2], heavy[owner][order])
    lenf = pd[:, 3].astype(np.uint32)
    assert np.array_equal(lenf & 0x7FFFFFFF, (ends - want_beg)[order]) and np.array_equal(lenf >> 31, single[order])
    pos = rd(a.piece_pos, a.n_chunks, torch.int32, 4)
    assert np.array_equal(order[pos], np.arange(a.n_chunks))
    if parts > 1:
        po = rd(a.part_off, parts + 1, torch.int64, 8)
        assert po[0] == 0 and po[-1] == a.n_chunks and np.all(np.diff(po) >= 0)
        for q in range(parts):
            assert np.all(first_col[order[po[q]:po[q + 1]]] * parts // n == q)
            # a piece never crosses its range: its last entry is in range q too
            last = np.minimum(beg[1:], g.rowptr[heavy[owner] + 1])[order[po[q]:po[q + 1]]] - 1
            assert np.all(g.colidx[last].astype(np.int64) * parts // n == q)
        per_xcd = [sum(po[q + 1] - po[q] for q in range(x, parts, 8)) for x in range(8)]
        assert a.part_slots == max(per_xcd)
    else:
        assert a.part_slots == a.n_chunks
    # rows for the fix-up: every heavy row of several pieces once, those of
    # more than GCN_FIX_BIG_PIECES pieces first, each group ascending
    big = np.flatnonzero(want_cnt > G.FIX_BIG_PIECES)
    small = np.flatnonzero((want_cnt >= 2) & (want_cnt <= G.FIX_BIG_PIECES))
    assert a.n_fix_big == big.size and a.n_fix == big.size + small.size
    fix = rd(a.fix_rows, a.n_fix, torch.int32, 4)
    assert np.array_equal(fix, np.concatenate([big, small]))


# ------------------------------------------------------------ layer fwd ----

# hub rows of 7, 2 and 1 chunk(s) at the tests' chunk size (96 entries)
HUBS = [(1, 600), (2, 150), (3, 70)]
# heavy rows of one chunk only: every heavy row is stored by its chunk and
# no fix-up pass runs
HUBS_ONE_CHUNK = [(3, 70), (5, 60)]


def _layer_case(n, f_in, f_out, seed, hubs=HUBS, m_random=None):
    rng = np.random.default_rng(seed)
    src, dst = hub_graph(n, 4 * n if m_random is None else m_random, hubs, seed)
    g = O.graph(n, src, dst)
    h = rng.standard_normal((n, f_in)).astype(np.float32)
    w = (rng.standard_normal((f_in, f_out)) / np.sqrt(f_in)).astype(np.float32)
    b = (0.1 * rng.standard_normal(f_out)).astype(np.float32)
    return g, src, dst, h, w, b


FWD_CASES = [
    # (n, f_in, f_out, act, p, adjacency storage)
    (3000, 500, 64, G.GCN_ACT_RELU, 0.5, "csr"),
    (3000, 128, 7, G.GCN_ACT_NONE, 0.0, "csr"),
    (2100, 40, 130, G.GCN_ACT_RELU, 0.3, "csr"),
    (2100, 40, 130, G.GCN_ACT_RELU, 0.3, "csr_dinv"),
    (1800, 72, 24, G.GCN_ACT_RELU, 0.5, "csr_onechunk"),
    (3000, 500, 64, G.GCN_ACT_RELU, 0.5, "csr_parts"),
    (2100, 40, 130, G.GCN_ACT_RELU, 0.3, "csr_parts"),
    (3000, 128, 7, G.GCN_ACT_NONE, 0.0, "csr_smallpieces"),
    # rows wider than one lane group (2 column blocks in 16-bit, 3 in fp32),
    # a hub of more than GCN_FIX_BIG_PIECES pieces, dropout in the fix-up
    (2000, 24, 600, G.GCN_ACT_RELU, 0.5, "csr_smallpieces"),
    (3001, 64, 130, G.GCN_ACT_RELU, 0.5, "csr_isolated"),
    (2003, 40, 7, G.GCN_ACT_NONE, 0.0, "csr_isolated_dinv"),
    (1500, 500, 64, G.GCN_ACT_RELU, 0.5, "tiled"),
    (1500, 64, 32, G.GCN_ACT_NONE, 0.0, "tiled"),
    (1003, 40, 7, G.GCN_ACT_NONE, 0.0, "tiled"),
    (777, 16, 130, G.GCN_ACT_RELU, 0.5, "tiled"),
    # wide features: the MFMA-bound dense kernel (128 x 64 and 128 x 128 per wave)
    (1300, 40, 200, G.GCN_ACT_RELU, 0.5, "tiled"),
    (777, 24, 520, G.GCN_ACT_RELU, 0.3, "tiled"),
    (2048, 16, 256, G.GCN_ACT_NONE, 0.0, "tiled"),
    # few 256-wide tiles and a long k loop: the tiles' k loops cut into
    # ranges whose fp32 partials a reduction adds (2 ranges in 16-bit, 4 in fp32)
    (8200, 40, 200, G.GCN_ACT_RELU, 0.5, "tiled"),
    (1500, 500, 64, G.GCN_ACT_RELU, 0.5, "dense"),
    (1003, 40, 7, G.GCN_ACT_NONE, 0.0, "dense"),
    (777, 16, 130, G.GCN_ACT_RELU, 0.5, "dense"),
]


CSR_STORAGES = ("csr", "csr_dinv", "csr_onechunk", "csr_parts", "csr_smallpieces", "csr_isolated",
                "csr_isolated_dinv")
# storages whose graph has about half its vertices isolated (one-entry rows
# for the bundled path, bundles with 1 .. 4 live rows)
SPARSE_STORAGES = ("csr_isolated", "csr_isolated_dinv")


def _graph_for(n, src, dst, prec, storage):
    # "csr": heavy rows cut every 96 entries, one column range;
    # "csr_dinv": CSR without stored values, every edge weight formed from dinv;
    # "csr_onechunk": CSR whose heavy rows are all one piece;
    # "csr_parts": 16 column ranges (the XCD-mapped launch);
    # "csr_smallpieces": 8 column ranges and pieces of 8 entries, so that a
    # hub has dozens of pieces for the fix-up to add
    csr = storage in CSR_STORAGES
    parts = {"csr_parts": 16, "csr_smallpieces": 8}.get(storage, 1)
    chunk = 8 if storage == "csr_smallpieces" else 96
    return DeviceGraph(n, src, dst, prec=prec, dense=not csr, tiled=storage == "tiled",
                       values=storage not in ("csr_dinv", "csr_isolated_dinv"), heavy_threshold=48, chunk_nnz=chunk,
                       col_parts=parts)


@pytest.mark.parametrize("prec", PRECS, ids=lambda p: PNAME[p])
@pytest.mark.parametrize("case", FWD_CASES, ids=lambda c: f"n{c[0]}_{c[1]}x{c[2]}_act{c[3]}_p{c[4]}_{c[5]}")
def test_layer_fwd(prec, case):
    n, f_in, f_out, act, p, storage = case
    dense = storage not in CSR_STORAGES
    g, src, dst, h, w, b = _layer_case(n, f_in, f_out, seed=n + f_in,
                                       hubs=HUBS_ONE_CHUNK if storage == "csr_onechunk" else HUBS,
                                       m_random=n // 3 if storage in SPARSE_STORAGES else None)
    dg = _graph_for(n, src, dst, prec, storage)
    L = G.GcnLayer(f_in, f_out, round8(f_in), round8(f_out), act, p, 3, 0)
    H, W = to_dev(h, prec), to_dev(w, prec, round8(f_out))
    bias = torch.as_tensor(b).to(dev())
    S = torch.empty((n, round8(f_out)), dtype=G.torch_dtype(prec), device=dev())
    Hout = torch.empty_like(S)
    ov = torch.zeros(1, dtype=torch.int32, device=dev())
    ws = torch.empty(G.gcn_layer_workspace_size(dg.adj, L, prec), dtype=torch.uint8, device=dev())
    seed, epoch = 1234567, 5
    G.gcn_layer_fwd(dg.adj, L, prec, True, H, W, bias, seed, epoch, S, Hout, ov, ws)
    torch.cuda.synchronize()
    hr, wr = rounded(h, prec), rounded(w, prec)
    vals = O.norm_values(g)
    p32 = f32(p)     # the ABI takes dropout_p as binary32
    s_o, z_o, out_o = O.layer_fwd(g, vals, hr, wr, b, "relu" if act else "none", p32, True, seed, 3, epoch,
                                  dense=O.dense_adj(g, vals) if dense else None)
    assert_close(host(S, f_out), s_o, prec, "S = H W")
    assert_close(host(Hout, f_out), out_o, prec, "H_out")
    assert int(ov.item()) == 0
    if p > 0:   # dropout decisions are bit-identical: zero pattern of kept positives matches
        keep = O.dropout_keep(seed, 3, epoch, n, f_out, p32)
        got = host(Hout, f_out)
        # positions whose sign no rounding of the device path can flip
        pos = z_o > (1e-3 if prec == 0 else 10 * tol_for(prec) * np.sqrt(np.mean(z_o * z_o)))
        assert np.array_equal(got[pos] != 0, keep[pos])


# neighbour rows wider than 256 bytes from a table of more than 128 MiB:
# the aggregation gathers them in 256-byte column blocks (grid y), heavy-row
# pieces and their fix-up included; bias and ReLU in the epilogue
@pytest.mark.parametrize("prec,n", [(G.GCN_F32, 70_000), (G.GCN_F16, 140_000)], ids=["f32", "f16"])
def test_aggregate_wide_rows_of_a_large_table(prec, n):
    F = 520
    assert n * F * (4 if prec == G.GCN_F32 else 2) > 128 << 20
    rng = np.random.default_rng(n)
    src, dst = hub_graph(n, 4 * n, HUBS, n)
    g = O.graph(n, src, dst)
    x = rng.standard_normal((n, F)).astype(np.float32)
    b = (0.1 * rng.standard_normal(F)).astype(np.float32)
    dg = DeviceGraph(n, src, dst, prec=prec, heavy_threshold=48, chunk_nnz=96)
    assert dg.adj.n_fix > 0
    X = to_dev(x, prec)
    Y = torch.empty_like(X)
    ov = torch.zeros(1, dtype=torch.int32, device=dev())
    ws = torch.empty(G.gcn_aggregate_workspace_size(dg.adj, F, prec), dtype=torch.uint8, device=dev())
    G.gcn_aggregate(dg.adj, F, prec, X, F, torch.as_tensor(b).to(dev()), G.GCN_ACT_RELU, 0.0, 0, 0, 0, 0,
                    Y, F, ov, ws)
    torch.cuda.synchronize()
    z = O.spmm(g, O.norm_values(g), rounded(x, prec)) + b.astype(np.float64)[None, :]
    assert_close(host(Y, F), np.maximum(z, 0.0), prec, "relu(A_hat X + b)")
    assert int(ov.item()) == 0


def test_dropout_threshold_uses_binary32_p():
    """The keep threshold is floor(p * 2^32) of the binary32 p the ABI takes.

    p64 is chosen (from the oracle's Philox words) so that for one element e
    the threshold of p64 itself lies at or below its word w while the
    threshold of float32(p64) lies above it: the device must drop e, as the
    oracle does when given the binary32 value, although the oracle given
    p64 would keep it.  Every other decision must match too.  Graph without
    edges (A_hat = I), H = 1, W = I: Z = 1 everywhere, so H_out is zero
    exactly where an element is dropped."""
    n, f, seed, layer, epoch = 64, 8, 987654321, 2, 11
    e_all = np.arange(n * f, dtype=np.uint64)
    words = O.dropout_words(seed, layer, epoch, e_all)
    # binary32 spacing in [1/4, 1/2) is 2^-25, i.e. 128 threshold units
    cand = [int(e) for e in e_all if 2**30 <= int(words[e]) < 2**31 and int(words[e]) % 128 >= 70]
    assert cand, "no suitable element for this seed"
    e = cand[0]
    w = int(words[e])
    p32 = (w // 128 + 1) / 2.0**25                      # smallest binary32 above w / 2^32
    p64 = p32 - 0.45 / 2.0**25                          # rounds to p32 in binary32
    assert f32(p64) == p32 and np.floor(p64 * 2.0**32) <= w < np.floor(p32 * 2.0**32)
    keep64 = O.dropout_keep(seed, layer, epoch, n, f, p64)
    keep32 = O.dropout_keep(seed, layer, epoch, n, f, f32(p64))
    assert keep64.reshape(-1)[e] and not keep32.reshape(-1)[e]
    empty = np.zeros(0, np.int32)
    for prec in PRECS:
        dg = DeviceGraph(n, empty, empty, prec=prec)
        L = G.GcnLayer(f, f, 8, 8, G.GCN_ACT_RELU, p64, layer, 0)
        H, W = to_dev(np.ones((n, f)), prec), to_dev(np.eye(f), prec)
        S = torch.empty((n, 8), dtype=G.torch_dtype(prec), device=dev())
        Hout = torch.empty_like(S)
        ov = torch.zeros(1, dtype=torch.int32, device=dev())
        ws = torch.empty(G.gcn_layer_workspace_size(dg.adj, L, prec), dtype=torch.uint8, device=dev())
        G.gcn_layer_fwd(dg.adj, L, prec, True, H, W, None, seed, epoch, S, Hout, ov, ws)
        torch.cuda.synchronize()
        got = host(Hout, f) != 0
        assert np.array_equal(got, keep32), PNAME[prec]


# ------------------------------------------------------------ layer bwd ----

BWD_CASES = [
    (3000, 500, 64, G.GCN_ACT_NONE, 0.0, "csr"),
    (3000, 64, 7, G.GCN_ACT_RELU, 0.5, "csr"),
    (2100, 130, 40, G.GCN_ACT_RELU, 0.3, "csr"),
    (3000, 64, 7, G.GCN_ACT_RELU, 0.5, "csr_dinv"),
    (1800, 24, 72, G.GCN_ACT_RELU, 0.5, "csr_onechunk"),
    (3000, 64, 7, G.GCN_ACT_RELU, 0.5, "csr_parts"),
    (2100, 130, 40, G.GCN_ACT_RELU, 0.3, "csr_smallpieces"),
    (2000, 40, 600, G.GCN_ACT_RELU, 0.5, "csr"),
    (3001, 130, 40, G.GCN_ACT_RELU, 0.3, "csr_isolated"),
    (1500, 64, 32, G.GCN_ACT_RELU, 0.5, "tiled"),
    (1003, 130, 7, G.GCN_ACT_RELU, 0.5, "tiled"),
    (1003, 130, 7, G.GCN_ACT_RELU, 0.5, "dense"),
    (777, 40, 130, G.GCN_ACT_RELU, 0.5, "tiled"),   # three 64-feature groups, ragged tail
    (1300, 200, 300, G.GCN_ACT_RELU, 0.5, "tiled"),  # wide G_S = A_hat dZ
    (600, 64, 448, G.GCN_ACT_NONE, 0.0, "tiled"),
    (8200, 24, 520, G.GCN_ACT_RELU, 0.5, "tiled"),   # G_S = A_hat dZ over k ranges
]


@pytest.mark.parametrize("prec", PRECS, ids=lambda p: PNAME[p])
@pytest.mark.parametrize("case", BWD_CASES, ids=lambda c: f"n{c[0]}_{c[1]}x{c[2]}_below{c[3]}_p{c[4]}_{c[5]}")
def test_layer_bwd(prec, case):
    n, f_in, f_out, act_below, p, storage = case
    dense = storage not in CSR_STORAGES
    g, src, dst, h, w, _ = _layer_case(n, f_in, f_out, seed=7 * n + f_out,
                                       hubs=HUBS_ONE_CHUNK if storage == "csr_onechunk" else HUBS,
                                       m_random=n // 3 if storage in SPARSE_STORAGES else None)
    rng = np.random.default_rng(n)
    if act_below == G.GCN_ACT_RELU:   # H as produced by ReLU + dropout: exact zeros
        h = np.where(rng.random(h.shape) < 0.5, 0.0, np.abs(h) * 2).astype(np.float32)
    dz = (rng.standard_normal((n, f_out)) * 8.0).astype(np.float32)
    dg = _graph_for(n, src, dst, prec, storage)
    L = G.GcnLayer(f_in, f_out, round8(f_in), round8(f_out), G.GCN_ACT_NONE, 0.0, 0, 0)
    H, W, dZ = to_dev(h, prec), to_dev(w, prec, round8(f_out)), to_dev(dz, prec)
    dW = torch.full((f_in, round8(f_out)), 7.0, dtype=torch.float32, device=dev())
    db = torch.full((round8(f_out),), 7.0, dtype=torch.float32, device=dev())
    dZb = torch.empty((n, round8(f_in)), dtype=G.torch_dtype(prec), device=dev())
    dbb = torch.full((round8(f_in),), 7.0, dtype=torch.float32, device=dev())
    GS = torch.empty((n, round8(f_out)), dtype=G.torch_dtype(prec), device=dev())
    ov = torch.zeros(1, dtype=torch.int32, device=dev())
    ws = torch.empty(G.gcn_layer_workspace_size(dg.adj, L, prec), dtype=torch.uint8, device=dev())
    G.gcn_layer_bwd(dg.adj, L, prec, H, W, dZ, act_below, p, dW, db, dZb, GS, ov, ws, dbias_below=dbb)
    torch.cuda.synchronize()
    hr, wr, dzr = rounded(h, prec), rounded(w, prec), rounded(dz, prec)
    vals = O.norm_values(g)
    gs_o, dw_o, db_o, dzb_o = O.layer_bwd(g, vals, hr, wr, dzr, "relu" if act_below else "none", f32(p),
                                          dense=O.dense_adj(g, vals) if dense else None)
    assert_close(host(GS, f_out), gs_o, prec, "G_S")
    assert_close(dW.cpu().numpy()[:, :f_out], dw_o, prec, "dW")
    assert np.all(dW.cpu().numpy()[:, f_out:] == 0)
    assert_close(db.cpu().numpy()[:f_out], db_o, prec, "db")
    assert np.all(db.cpu().numpy()[f_out:] == 0)
    assert_close(host(dZb, f_in), dzb_o, prec, "dZ_below")
    # the bias gradient of the layer below: the column sums of dZ_below as
    # stored (checked against the stored values summed in fp64, to fp32
    # summation error, and against the oracle's exact dZ_below)
    stored = host(dZb, f_in).astype(np.float64)
    got_bb = dbb.cpu().numpy()
    assert np.all(np.abs(got_bb[:f_in] - stored.sum(0)) <= 2e-5 * np.abs(stored).sum(0) + 1e-30)
    assert np.all(got_bb[f_in:] == 0)
    assert_close(got_bb[:f_in], dzb_o.sum(0), prec, "db_below")
    assert int(ov.item()) == 0


def test_bwd_power_of_two_scale_invariance():
    """fp32: scaling dZ by 2^k scales G_S, dW, db, dZ_below by exactly 2^k."""
    prec = G.GCN_F32
    n, f_in, f_out = 1200, 40, 24
    g, src, dst, h, w, _ = _layer_case(n, f_in, f_out, seed=99)
    dz = np.random.default_rng(3).standard_normal((n, f_out)).astype(np.float32)
    dg = DeviceGraph(n, src, dst, prec=prec, heavy_threshold=48, chunk_nnz=96)
    L = G.GcnLayer(f_in, f_out, round8(f_in), round8(f_out), G.GCN_ACT_NONE, 0.0, 0, 0)
    ws = torch.empty(G.gcn_layer_workspace_size(dg.adj, L, prec), dtype=torch.uint8, device=dev())
    outs = []
    for k in (0, 12):
        dZ = to_dev(dz * (2.0 ** k), prec)
        dW = torch.empty((f_in, round8(f_out)), dtype=torch.float32, device=dev())
        db = torch.empty((round8(f_out),), dtype=torch.float32, device=dev())
        dZb = torch.empty((n, round8(f_in)), dtype=torch.float32, device=dev())
        GS = torch.empty((n, round8(f_out)), dtype=torch.float32, device=dev())
        G.gcn_layer_bwd(dg.adj, L, prec, to_dev(h, prec), to_dev(w, prec, round8(f_out)), dZ, G.GCN_ACT_RELU,
                        0.5, dW, db, dZb, GS, None, ws)
        outs.append([t.cpu() for t in (GS, dW, db, dZb)])
    for a, b in zip(*outs):
        assert torch.equal(a * 4096.0, b)


# ----------------------------------------------------------------- loss ----

@pytest.mark.parametrize("prec", PRECS, ids=lambda p: PNAME[p])
@pytest.mark.parametrize("C,n", [(7, 5000), (40, 5000), (64, 5000), (32, 5000),
                                 # more than 16384 row groups: four rows per lane group and iteration
                                 (64, 600_003), (40, 600_003),
                                 # more than 4096 workgroups with C not a multiple of 8: the
                                 # column-sum partials (rows padded to 8) summed in two stages
                                 (7, 1_200_003)])
def test_loss(prec, C, n):
    rng = np.random.default_rng(C)
    z = (rng.standard_normal((n, C)) * 3).astype(np.float32)
    y = rng.integers(0, C, n).astype(np.int32)
    mask = (rng.random(n) < 0.3).astype(np.uint8)
    ld = round8(C)
    Z = to_dev(z, prec)
    dZ = torch.empty_like(Z)
    scale = torch.tensor([1024.0], device=dev())
    loss = torch.zeros(1, device=dev())
    nc = torch.zeros(1, dtype=torch.int32, device=dev())
    ws = torch.empty(G.gcn_loss_workspace_size(n, C), dtype=torch.uint8, device=dev())
    dcs = torch.full((ld,), 7.0, dtype=torch.float32, device=dev())
    G.gcn_loss(n, C, ld, prec, Z, torch.as_tensor(y).to(dev()), torch.as_tensor(mask).to(dev()), int(mask.sum()),
               scale, loss, dZ, nc, None, ws, dlogits_colsum=dcs)
    torch.cuda.synchronize()
    zr = rounded(z, prec)
    l_o, d_o, nc_o = O.softmax_ce(zr, y, mask, 1024.0)
    assert abs(loss.item() - l_o) <= (1e-5 if prec == 0 else 1e-4) * max(1.0, abs(l_o))
    assert_close(host(dZ, C), d_o, prec, "dlogits")
    assert np.all(host(dZ)[:, C:] == 0)
    assert nc.item() == nc_o
    # column sums of dlogits (the output layer's bias gradient): against the
    # stored values summed in fp64, to fp32 summation error, and the oracle
    stored = host(dZ, C).astype(np.float64)
    got = dcs.cpu().numpy()
    assert np.all(np.abs(got[:C] - stored.sum(0)) <= 2e-5 * np.abs(stored).sum(0) + 1e-30)
    assert np.all(got[C:] == 0)
    assert_close(got[:C], d_o.sum(0), prec, "dlogits column sums")


# ------------------------------------------------------------ optimiser ----

# a few workgroups and a grid of several hundred: same state sequence
@pytest.mark.parametrize("P", [5000, 70001])
def test_optimizer_matches_oracle_and_skips_on_overflow(P):
    rng = np.random.default_rng(0)
    w0 = rng.standard_normal(P).astype(np.float32)
    g0 = (rng.standard_normal(P) * 65536).astype(np.float32)
    master = torch.as_tensor(w0).to(dev())
    grad = torch.as_tensor(g0).to(dev())
    m = torch.zeros(P, device=dev())
    v = torch.zeros(P, device=dev())
    working = torch.empty(P, dtype=torch.float16, device=dev())
    state = torch.zeros(4, dtype=torch.int32, device=dev())
    state.view(torch.float32)[0] = 65536.0
    ov = torch.zeros(1, dtype=torch.int32, device=dev())
    cfg = G.GcnAdamConfig(0.01, 0.9, 0.999, 1e-8, 0.5, 2.0, 3, 1.0, 2.0**24)
    sc = O.LossScaler(65536.0, 0.5, 2.0, 3, 1.0, 2.0**24)
    ad = O.AdamState(P)
    w_o = w0.astype(np.float64)
    for step in range(4):
        gs = g0 * (1 + step)
        grad.copy_(torch.as_tensor(gs))
        G.gcn_optimizer_step(P, master, grad, m, v, working, G.GCN_F16, cfg, state, ov)
        w_o, applied = O.adam_step(w_o, gs.astype(np.float64), ad, sc, lr=0.01)
        torch.cuda.synchronize()
        assert_close(master.cpu().numpy(), w_o, 0, f"master step {step}")
        assert np.array_equal(working.cpu().numpy(), master.cpu().numpy().astype(np.float16))
        st = state.cpu()
        assert float(st.view(torch.float32)[0]) == sc.scale and int(st[1]) == sc.good
    # overflow: weights bit-unchanged, scale halved, flag cleared
    before = master.clone()
    bad = g0.copy()
    bad[P - 1] = np.inf
    grad.copy_(torch.as_tensor(bad))
    G.gcn_optimizer_step(P, master, grad, m, v, working, G.GCN_F16, cfg, state, ov)
    sc.update(True)
    torch.cuda.synchronize()
    assert torch.equal(master, before)
    st = state.cpu()
    assert float(st.view(torch.float32)[0]) == sc.scale and int(st[3]) == 1 and ov.item() == 0
    # overflow flagged by an earlier kernel
    ov.fill_(1)
    grad.copy_(torch.as_tensor(g0))
    G.gcn_optimizer_step(P, master, grad, m, v, working, G.GCN_F16, cfg, state, ov)
    torch.cuda.synchronize()
    assert torch.equal(master, before) and int(state.cpu()[3]) == 2


# ------------------------------------------------------- full training step ----

def _oracle_step(g, x, y, mask, w1, b1, w2, b2, p, seed, epoch, scale):
    vals = O.norm_values(g)
    _, _, h1 = O.layer_fwd(g, vals, x, w1, b1, "relu", p, True, seed, 0, epoch)
    _, z2, _ = O.layer_fwd(g, vals, h1, w2, b2, "none", 0.0, True, seed, 1, epoch)
    loss, dz2, nc = O.softmax_ce(z2, y, mask, scale)
    _, dw2, db2, dz1 = O.layer_bwd(g, vals, h1, w2, dz2, "relu", p)
    _, dw1, db1, _ = O.layer_bwd(g, vals, x, w1, dz1, "none", 0.0, need_dh=False)
    return loss, nc, dw1, db1, dw2, db2, h1, z2


@pytest.mark.parametrize("prec", PRECS, ids=lambda p: PNAME[p])
def test_full_step_er2k(prec):
    """One forward + loss + backward step of the tiny 2-layer workload
    (ER n=2048, 512 -> 16 -> 7, 140-vertex train mask, dropout 0.5)."""
    wl = I.workload("er2k", 0)
    n = wl["n"]
    g = O.graph(n, wl["src"], wl["dst"])
    dg = DeviceGraph(n, wl["src"], wl["dst"], prec=prec)
    scale = 65536.0 if prec else 1.0
    m = GCN2(dg, wl["X"], wl["labels"], wl["mask"], wl["W1"], wl["W2"], prec=prec, dropout=0.5,
             seed=wl["dropout_seed"], loss_scale=scale)
    m.forward(epoch=0)
    m.loss_and_backward()
    torch.cuda.synchronize()
    x, w1, w2 = rounded(wl["X"], prec), rounded(wl["W1"], prec), rounded(wl["W2"], prec)
    loss, nc, dw1, db1, dw2, db2, h1, z2 = _oracle_step(g, x, wl["labels"], wl["mask"], w1, wl["b1"], w2,
                                                        wl["b2"], 0.5, wl["dropout_seed"], 0, scale)
    assert abs(m.loss.item() - loss) <= (1e-5 if prec == 0 else 2e-3) * abs(loss)
    assert_close(host(m.H1, 16), h1, prec, "H1")
    assert_close(host(m.Z2, 7), z2, prec, "Z2")
    # gradients through a chain of 16-bit roundings: compared per element in
    # fp32 mode, normwise (same bound) in 16-bit modes (see design notes)
    grads = [(m.dW1().cpu().numpy()[:, :16], dw1, "dW1"), (m.db1().cpu().numpy()[:16], db1, "db1"),
             (m.dW2().cpu().numpy()[:, :7], dw2, "dW2"), (m.db2().cpu().numpy()[:7], db2, "db2")]
    for got, want, name in grads:
        if prec == 0:
            assert_close(got, want, 0, name)
        else:
            err = np.max(np.abs(got - want)) / np.max(np.abs(want))
            assert err <= (2e-2 if prec == 1 else 1e-1), f"{name}: normwise {err}"
    assert m.overflow.item() == 0


def test_full_step_deterministic():
    wl = I.workload("er2k", 1)
    n = wl["n"]
    res = []
    for _ in range(2):
        dg = DeviceGraph(n, wl["src"], wl["dst"], prec=G.GCN_F16, heavy_threshold=16, chunk_nnz=16)
        m = GCN2(dg, wl["X"], wl["labels"], wl["mask"], wl["W1"], wl["W2"], prec=G.GCN_F16,
                 seed=wl["dropout_seed"])
        for ep in range(3):
            m.step(ep)
        torch.cuda.synchronize()
        res.append((m.master.cpu(), m.H1.cpu(), m.loss.cpu()))
    for a, b in zip(*res):
        assert torch.equal(a, b)
