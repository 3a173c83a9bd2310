"""The featureless input of the paper's run-time experiments (Section
"Run-Time and Memory Usage Analysis": X = I, model sizes up to 2048) and the
MFMA-bound dense aggregation it leads to.

* identity_input layers: forward and backward against the oracle's layer
  with h = I (a dense identity), CSR and tiled dense A_hat, 16-bit and fp32;
  dW = G_S widened, padding zero; the argument checks (f_in != n,
  dZ_below given).
* The dense aggregation at full size, one shape per workgroup tile of the
  MFMA kernel: the benchmark's widest (n = 32768, F = 2048, the launch the
  model-size sweep times, 256 x 256 tiles), shapes whose tile count falls
  below the compute-unit count (256 x 128 and 128 x 128 tiles, ragged n and
  F), 256 x 256 tiles with ragged n and F in fp16 and fp32, and an fp32
  256 x 128 shape: sampled output rows against the oracle's per-row
  formula."""
import numpy as np
import pytest
import torch

from oracle import gcn_oracle as O
from paper_2010_12635_amd import gcn as G
from paper_2010_12635_amd.model import DeviceGraph, round8
from tests.parity import assert_close, hub_graph

pytestmark = pytest.mark.gpu

PNAME = {0: "f32", 1: "f16", 2: "bf16"}


def dev():
    return torch.device("cuda")


def to_dev(a, prec, ld=None):
    a = np.asarray(a, np.float32)
    n, f = a.shape
    t = torch.zeros((n, ld or round8(f)), dtype=G.torch_dtype(prec), device=dev())
    t[:, :f] = torch.as_tensor(a).to(dev()).to(G.torch_dtype(prec))
    return t


def rounded(a, prec):
    return torch.as_tensor(np.asarray(a, np.float32)).to(G.torch_dtype(prec)).float().numpy().astype(np.float64)


@pytest.mark.parametrize("prec", [G.GCN_F16, G.GCN_F32, G.GCN_BF16], ids=lambda p: PNAME[p])
@pytest.mark.parametrize("storage", ["csr", "tiled"])
@pytest.mark.parametrize("f_out", [40, 256])
def test_identity_input_layer(prec, storage, f_out):
    n = 700
    print(f"[featureless] {PNAME[prec]} {storage} n={n} f_out={f_out}", flush=True)
    rng = np.random.default_rng(f_out)
    src, dst = hub_graph(n, 4 * n, [(3, 300)], 5)
    g = O.graph(n, src, dst)
    w = (rng.standard_normal((n, f_out)) / np.sqrt(n)).astype(np.float32)
    b = (0.1 * rng.standard_normal(f_out)).astype(np.float32)
    dz = (rng.standard_normal((n, f_out)) * 4.0).astype(np.float32)
    dg = DeviceGraph(n, src, dst, prec=prec, dense=storage != "csr")
    ldo = round8(f_out) + 8                     # padding beyond the last vector
    L = G.GcnLayer(n, f_out, round8(n), ldo, G.GCN_ACT_RELU, 0.5, 2, 1)
    W = to_dev(w, prec, ldo)
    bias = torch.as_tensor(b).to(dev())
    Hout = torch.empty((n, ldo), dtype=G.torch_dtype(prec), device=dev())
    ov = torch.zeros(1, dtype=torch.int32, device=dev())
    ws = torch.empty(G.gcn_layer_workspace_size(dg.adj, L, prec), dtype=torch.uint8, device=dev())
    seed, epoch = 77, 4
    G.gcn_layer_fwd(dg.adj, L, prec, True, None, W, bias, seed, epoch, None, Hout, ov, ws)
    torch.cuda.synchronize()
    vals = O.norm_values(g)
    dense = O.dense_adj(g, vals) if storage != "csr" else None
    eye = np.eye(n)
    wr = rounded(w, prec)
    _, _, out_o = O.layer_fwd(g, vals, eye, wr, b, "relu", 0.5, True, seed, 2, epoch, dense=dense)
    assert_close(Hout.float().cpu().numpy()[:, :f_out], out_o, prec, "H_out (X = I)")
    # backward (input layer: no dZ_below)
    dZ = to_dev(dz, prec, ldo)
    GS = torch.empty((n, ldo), dtype=G.torch_dtype(prec), device=dev())
    dW = torch.full((n, ldo), 7.0, dtype=torch.float32, device=dev())
    db = torch.full((ldo,), 7.0, dtype=torch.float32, device=dev())
    G.gcn_layer_bwd(dg.adj, L, prec, None, W, dZ, G.GCN_ACT_NONE, 0.0, dW, db, None, GS, ov, ws)
    torch.cuda.synchronize()
    gs_o, dw_o, db_o, _ = O.layer_bwd(g, vals, eye, wr, rounded(dz, prec), "none", 0.0, dense=dense)
    assert_close(GS.float().cpu().numpy()[:, :f_out], gs_o, prec, "G_S")
    dwh = dW.cpu().numpy()
    assert_close(dwh[:, :f_out], dw_o, prec, "dW = G_S")
    assert np.array_equal(dwh[:, :f_out], GS.float().cpu().numpy()[:, :f_out])   # exactly the widened G_S
    assert np.all(dwh[:, f_out:] == 0)
    assert_close(db.cpu().numpy()[:f_out], db_o, prec, "db")
    assert int(ov.item()) == 0
    # argument checks
    with pytest.raises(G.GcnError):
        G.gcn_layer_bwd(dg.adj, L, prec, None, W, dZ, G.GCN_ACT_NONE, 0.0, dW, db, Hout, GS, ov, ws)
    L_bad = G.GcnLayer(n - 8, f_out, round8(n - 8), ldo, G.GCN_ACT_RELU, 0.5, 2, 1)
    with pytest.raises(G.GcnError):
        G.gcn_layer_fwd(dg.adj, L_bad, prec, True, None, W, bias, seed, epoch, None, Hout, ov, ws)


@pytest.mark.parametrize("n,F,prec", [
    (32768, 2048, G.GCN_F16),   # 256 x 256 workgroup tiles
    (16384, 520, G.GCN_BF16),   # 256 x 128: 192 tiles of 256 x 256 would not fill the chip
    (32768, 256, G.GCN_F32),    # 256 x 128, fp32 MFMA
    (6000, 1000, G.GCN_F16),    # 128 x 128, ragged rows and columns
    (33000, 600, G.GCN_F16),    # 256 x 256 with ragged rows and columns (bias of the lanes past F)
    (33000, 600, G.GCN_F32),    # the same tiles in fp32 (four 16x16x4 steps per fragment pair)
], ids=["n32768_F2048_f16", "n16384_F520_bf16", "n32768_F256_f32", "n6000_F1000_f16", "n33000_F600_f16",
        "n33000_F600_f32"])
def test_wide_dense_aggregation_at_full_size(n, F, prec):
    print(f"[wide] n={n} F={F} tiled {PNAME[prec]}", flush=True)
    rng = np.random.default_rng(21)
    src = rng.integers(0, n, 8 * n).astype(np.int32)
    dst = rng.integers(0, n, 8 * n).astype(np.int32)
    dg = DeviceGraph(n, src, dst, prec=prec, dense=True)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(3)
    ld = round8(F)
    X = torch.randn((n, ld), generator=gen, device="cuda").to(G.torch_dtype(prec))
    Y = torch.empty_like(X)
    bias = torch.as_tensor((0.1 * rng.standard_normal(F)).astype(np.float32)).to(dev())
    ov = torch.zeros(1, dtype=torch.int32, device=dev())
    ws = torch.empty(G.gcn_aggregate_workspace_size(dg.adj, F, prec), dtype=torch.uint8, device=dev())
    G.gcn_aggregate(dg.adj, F, prec, X, ld, bias, G.GCN_ACT_RELU, 0.0, 0, 0, 0, 0, Y, ld, ov, ws)
    torch.cuda.synchronize()
    deg = O.graph_degrees(n, src, dst)
    rows = np.unique(np.concatenate([[0, 255, 256, n - 1], rng.choice(n, 60, replace=False)]))
    nbrs = O.graph_rows(n, src, dst, rows)
    d = 1.0 / np.sqrt(deg.astype(np.float64))
    need = np.unique(np.concatenate([nbrs[int(r)] for r in rows]))
    xs = dict(zip(need.tolist(), X[torch.as_tensor(need).cuda(), :F].float().cpu().numpy().astype(np.float64)))
    bh = bias.cpu().numpy().astype(np.float64)
    want = np.stack([np.maximum(sum(d[r] * d[c] * xs[int(c)] for c in nbrs[int(r)]) + bh, 0.0) for r in rows])
    got = Y[torch.as_tensor(rows).cuda(), :F].float().cpu().numpy().astype(np.float64)
    assert_close(got, want, prec, f"Y sampled rows at n = {n}, F = {F}")
    assert int(ov.item()) == 0
