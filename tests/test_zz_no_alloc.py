"""gcn_layer_bwd_noalloc (scratch in the library's fixed device array)
against gcn_layer_bwd (caller workspace): identical outputs, bit for bit,
on two calls in a row, the second on a smaller graph and narrower layer
(so that stale contents of the shared array from the first call would
show), for CSR with heavy-row chunks and for tiled dense A_hat."""
import numpy as np
import pytest
import torch

from paper_2010_12635_amd import gcn as G
from paper_2010_12635_amd.model import DeviceGraph, round8
from tests.parity import hub_graph

pytestmark = pytest.mark.gpu

HUBS = [(3, 900), (17, 400), (40, 120)]


def _case(n, f_in, f_out, prec, storage, seed):
    rng = np.random.default_rng(seed)
    src, dst = hub_graph(n, 4 * n, HUBS, seed)
    dg = DeviceGraph(n, src, dst, prec=prec, dense=storage == "tiled", heavy_threshold=48, chunk_nnz=96)
    dt = G.torch_dtype(prec)

    def dev(a, ld):
        t = torch.zeros((a.shape[0], ld), dtype=dt, device="cuda")
        t[:, : a.shape[1]] = torch.as_tensor(a).cuda().to(dt)
        return t

    h = np.where(rng.random((n, f_in)) < 0.5, 0.0, rng.random((n, f_in)) * 2).astype(np.float32)
    w = (rng.standard_normal((f_in, f_out)) / np.sqrt(f_in)).astype(np.float32)
    dz = (rng.standard_normal((n, f_out)) * 8.0).astype(np.float32)
    L = G.GcnLayer(f_in, f_out, round8(f_in), round8(f_out), G.GCN_ACT_NONE, 0.0, 0, 0)
    return dg, L, dev(h, round8(f_in)), dev(w, round8(f_out)), dev(dz, round8(f_out))


def _outputs(n, L, prec):
    dt = G.torch_dtype(prec)
    return dict(dW=torch.full((L.f_in, L.ld_out), 7.0, dtype=torch.float32, device="cuda"),
                db=torch.full((L.ld_out,), 7.0, dtype=torch.float32, device="cuda"),
                dZb=torch.zeros((n, L.ld_in), dtype=dt, device="cuda"),
                dbb=torch.full((L.ld_in,), 7.0, dtype=torch.float32, device="cuda"),
                GS=torch.zeros((n, L.ld_out), dtype=dt, device="cuda"),
                ov=torch.zeros(1, dtype=torch.int32, device="cuda"))


@pytest.mark.parametrize("prec", [G.GCN_F32, G.GCN_F16])
@pytest.mark.parametrize("storage", ["csr", "tiled"])
def test_noalloc_matches_workspace_call_twice(prec, storage):
    for k, (n, f_in, f_out) in enumerate([(3000, 130, 40), (1100, 24, 7)]):
        print(f"[noalloc] {storage} prec={prec} call {k}: n={n} {f_in}x{f_out}", flush=True)
        dg, L, H, W, dZ = _case(n, f_in, f_out, prec, storage, seed=17 + k)
        need = G.gcn_layer_workspace_size(dg.adj, L, prec)
        assert need <= G.NOALLOC_SCRATCH_BYTES
        ref = _outputs(n, L, prec)
        ws = torch.empty(need, dtype=torch.uint8, device="cuda")
        G.gcn_layer_bwd(dg.adj, L, prec, H, W, dZ, G.GCN_ACT_RELU, 0.5, ref["dW"], ref["db"], ref["dZb"], ref["GS"],
                        ref["ov"], ws, dbias_below=ref["dbb"])
        got = _outputs(n, L, prec)
        G.gcn_layer_bwd_noalloc(dg.adj, L, prec, H, W, dZ, G.GCN_ACT_RELU, 0.5, got["dW"], got["db"], got["dZb"],
                                got["GS"], got["ov"], dbias_below=got["dbb"])
        torch.cuda.synchronize()
        for key in ref:
            assert torch.equal(ref[key], got[key]), (storage, prec, k, key)
        assert got["ov"].item() == 0
