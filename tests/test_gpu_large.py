"""Launch geometry at n = 2^26 + 3 vertices, past the point where one
work-item per wave-sized row slot no longer fits a single dispatch
dimension (2^32 work-items): the one-wave-per-row kernels of the CSR
construction, the light-row aggregation and the loss walk their rows in
loops over a capped grid, and these tests check their results there.

* CSR: degrees and row pointers of every row bit-exact against the oracle;
  sampled rows' column lists and dinv bit-exact.
* Layer forward (64 -> 64, ReLU, dropout 0.5): sampled output rows against
  the oracle's per-row formula.
* Loss on all-zero logits: the closed form loss = log C, dlogits =
  S (1/C - onehot) / n, n_correct = #{labels == 0} (arg-max ties take the
  lowest class)."""
import numpy as np
import pytest
import torch

from oracle import gcn_oracle as O
from paper_2010_12635_amd import gcn as G
from paper_2010_12635_amd.model import DeviceGraph, round8
from tests.parity import assert_close

pytestmark = pytest.mark.gpu

N = (1 << 26) + 3


@pytest.fixture(scope="module")
def big():
    rng = np.random.default_rng(11)
    e = 200_000
    src = rng.integers(0, N, e).astype(np.int32)
    dst = rng.integers(0, N, e).astype(np.int32)
    hub = 12345                                   # one heavy row (> 512 entries)
    nb = rng.choice(N, 3000, replace=False).astype(np.int32)
    src = np.concatenate([src, np.full(nb.size, hub, np.int32)])
    dst = np.concatenate([dst, nb])
    print(f"[large] n={N}: normalize", flush=True)
    dg = DeviceGraph(N, src, dst, prec=G.GCN_F16, index=G.GCN_I64)
    torch.cuda.synchronize()
    deg = O.graph_degrees(N, src, dst)
    rows = np.unique(np.concatenate([[0, hub, N - 1], np.argsort(deg)[-5:], rng.choice(N, 40, replace=False)]))
    yield dict(dg=dg, src=src, dst=dst, deg=deg, rows=rows, nbrs=O.graph_rows(N, src, dst, rows))
    del dg
    torch.cuda.empty_cache()


def test_csr_at_2pow26(big):
    dg, deg = big["dg"], big["deg"]
    assert dg.nnz == int(deg.sum())
    assert np.array_equal(dg.deg.cpu().numpy(), deg)
    rp = dg.rowptr.cpu().numpy()
    assert rp[0] == 0 and np.array_equal(np.diff(rp), deg.astype(np.int64))
    dinv = dg.dinv.cpu().numpy()
    for r in big["rows"]:
        got = dg.colidx[int(rp[r]): int(rp[r + 1])].cpu().numpy()
        assert np.array_equal(got, big["nbrs"][int(r)]), r
        assert dinv[r] == np.float32(1.0 / np.sqrt(np.float64(deg[r])))
    assert dg.adj.n_heavy == int((deg > 512).sum()) >= 1
    # light-row schedule: every light row once; the rows of several entries
    # in blocks of 4096 consecutive ids, decreasing degree inside a block,
    # then the rows of one entry
    a = dg.adj
    base = dg.sched
    o = a.row_perm - base.data_ptr()
    perm = base[o: o + 4 * a.n_light].view(torch.int32).cpu().numpy()
    light = deg <= 512
    assert a.n_light == int(light.sum())
    assert a.n_light_single == int((deg == 1).sum()) > 0
    multi = perm[: a.n_light - a.n_light_single]
    assert np.all(deg[perm[a.n_light - a.n_light_single:]] == 1) and np.all(deg[multi] > 1)
    blk = multi.astype(np.int64) // 4096
    assert np.all(np.diff(blk) >= 0)
    same = np.diff(blk) == 0
    assert np.all(np.diff(deg[multi].astype(np.int64))[same] <= 0)
    assert np.all(light[perm]) and np.unique(perm).size == perm.size


def test_layer_fwd_at_2pow26(big):
    dg, deg, rows, nbrs = big["dg"], big["deg"], big["rows"], big["nbrs"]
    f = 64
    print(f"[large] layer fwd {f} -> {f}", flush=True)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(5)
    X = torch.empty((N, f), dtype=torch.float16, device="cuda")
    for lo in range(0, N, 1 << 24):
        hi = min(lo + (1 << 24), N)
        X[lo:hi] = torch.randn((hi - lo, f), generator=gen, device="cuda").half()
    w = (np.random.default_rng(6).standard_normal((f, f)) / np.sqrt(f)).astype(np.float32)
    W = torch.as_tensor(w).cuda().half()
    L = G.GcnLayer(f, f, f, f, G.GCN_ACT_RELU, 0.5, 0, 0)
    S = torch.empty((N, f), dtype=torch.float16, device="cuda")
    Hout = torch.empty_like(S)
    ov = torch.zeros(1, dtype=torch.int32, device="cuda")
    ws = torch.empty(G.gcn_layer_workspace_size(dg.adj, L, G.GCN_F16), dtype=torch.uint8, device="cuda")
    seed, epoch = 99, 3
    G.gcn_layer_fwd(dg.adj, L, G.GCN_F16, True, X, W, None, seed, epoch, S, Hout, ov, ws)
    torch.cuda.synchronize()
    need = np.unique(np.concatenate([nbrs[int(r)] for r in rows]))
    xs = dict(zip(need.tolist(), X[torch.as_tensor(need).cuda()].float().cpu().numpy().astype(np.float64)))
    wr = W.float().cpu().numpy().astype(np.float64)
    d = 1.0 / np.sqrt(deg.astype(np.float64))
    keep = O.dropout_keep_rows(seed, 0, epoch, rows, f, 0.5)
    want = np.empty((rows.size, f))
    for t, r in enumerate(rows):
        nb = nbrs[int(r)]
        z = sum((d[r] * d[c]) * (xs[int(c)] @ wr) for c in nb)
        want[t] = np.where(keep[t], np.maximum(z, 0.0) * 2.0, 0.0)
    got = Hout[torch.as_tensor(rows).cuda()].float().cpu().numpy().astype(np.float64)
    assert_close(got, want, G.GCN_F16, "H_out sampled rows at n = 2^26 + 3")
    assert ov.item() == 0


def test_loss_closed_form_at_2pow26():
    C, ld = 64, 64
    print("[large] loss", flush=True)
    labels_h = np.random.default_rng(7).integers(0, C, N).astype(np.int32)
    labels = torch.as_tensor(labels_h).cuda()
    logits = torch.zeros((N, ld), dtype=torch.float16, device="cuda")
    dl = torch.empty_like(logits)
    scale = torch.tensor([1024.0], device="cuda")
    loss = torch.zeros(1, device="cuda")
    nc = torch.zeros(1, dtype=torch.int32, device="cuda")
    ov = torch.zeros(1, dtype=torch.int32, device="cuda")
    ws = torch.empty(G.gcn_loss_workspace_size(N, C), dtype=torch.uint8, device="cuda")
    G.gcn_loss(N, C, ld, G.GCN_F16, logits, labels, None, N, scale, loss, dl, nc, ov, ws)
    torch.cuda.synchronize()
    assert abs(loss.item() - np.log(C)) <= 1e-5 * np.log(C)
    assert nc.item() == int((labels_h == 0).sum())
    rows = np.unique(np.concatenate([[0, N - 1], np.random.default_rng(8).choice(N, 64, replace=False)]))
    got = dl[torch.as_tensor(rows).cuda()].float().cpu().numpy().astype(np.float64)
    want = np.full((rows.size, C), 1.0 / C)
    want[np.arange(rows.size), labels_h[rows]] -= 1.0
    want *= 1024.0 / N
    assert_close(got, want, G.GCN_F16, "dlogits sampled rows")
    assert ov.item() == 0
