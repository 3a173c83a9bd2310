"""Link prediction (graph auto-encoder, Eq. (2) on sampled pairs): the
pair sampler bit-exact against the oracle's Philox draws, the pair loss,
its backward scatter and the AUC/AP metrics against the oracle, invalid
ids, determinism, and one full training step of the auto-encoder."""
import numpy as np
import pytest
import torch

from oracle import gcn_oracle as O
from paper_2010_12635_amd import gcn as G
from paper_2010_12635_amd import inputs as I
from paper_2010_12635_amd.model import DeviceGraph, GAE2, round8
from tests.parity import assert_close, tol_for

pytestmark = pytest.mark.gpu

PRECS = [G.GCN_F32, G.GCN_F16, G.GCN_BF16]
PNAME = {G.GCN_F32: "f32", G.GCN_F16: "f16", G.GCN_BF16: "bf16"}


def dev(a, dt=None):
    t = torch.as_tensor(np.ascontiguousarray(a))
    return t.cuda() if dt is None else t.cuda().to(dt)


def z_dev(z, prec, ld):
    t = torch.zeros((z.shape[0], ld), dtype=G.torch_dtype(prec), device="cuda")
    t[:, : z.shape[1]] = torch.as_tensor(z).cuda().to(t.dtype)
    t[:, z.shape[1]:] = float("nan")          # padding columns must be ignored
    return t


def host(t, f):
    return t.float().cpu().numpy()[:, :f].astype(np.float64)


def test_sample_pairs_bit_exact():
    rng = np.random.default_rng(40)
    n, m = 5000, 3000
    eu = rng.integers(0, n, m).astype(np.int32)
    ev = ((eu + 1 + rng.integers(0, n - 1, m)) % n).astype(np.int32)
    n_pos, n_neg, seed = 3001, 4093, (1 << 40) + 7
    pu = torch.empty(n_pos + n_neg, dtype=torch.int32, device="cuda")
    pv = torch.empty_like(pu)
    for epoch in (0, 3):
        G.gcn_sample_pairs(n, dev(eu), dev(ev), n_pos, n_neg, seed, epoch, pu, pv)
        ou, ov = O.sample_pairs(seed, epoch, n, eu, ev, n_pos, n_neg)
        assert np.array_equal(pu.cpu().numpy(), ou) and np.array_equal(pv.cpu().numpy(), ov)
    # negatives only (no edge list needed)
    G.gcn_sample_pairs(n, None, None, 0, 100, seed, 1, pu, pv)
    ou, ov = O.sample_pairs(seed, 1, n, eu, ev, 0, 100)
    assert np.array_equal(pu[:100].cpu().numpy(), ou) and np.array_equal(pv[:100].cpu().numpy(), ov)


def _pairs(n, n_pos, n_neg, seed):
    rng = np.random.default_rng(seed)
    eu = rng.integers(0, n, 4 * n).astype(np.int32)
    ev = ((eu + 1 + rng.integers(0, n - 1, 4 * n)) % n).astype(np.int32)
    return O.sample_pairs(seed, 2, n, eu, ev, n_pos, n_neg)


@pytest.mark.parametrize("prec", PRECS, ids=lambda p: PNAME[p])
@pytest.mark.parametrize("F", [64, 130, 7])
def test_pair_loss_matches_oracle(prec, F):
    n, n_pos, n_neg = 3000, 2500, 3100
    rng = np.random.default_rng(41 + F)
    z = (0.3 * rng.standard_normal((n, F))).astype(np.float32)
    u, v = _pairs(n, n_pos, n_neg, 42 + F)
    ld = round8(F)
    Z = z_dev(z, prec, ld)
    zr = host(Z, F)
    K = n_pos + n_neg
    loss = torch.zeros(1, device="cuda")
    scores = torch.empty(K, device="cuda")
    g = torch.empty(K, device="cuda")
    ov = torch.zeros(1, dtype=torch.int32, device="cuda")
    scale = torch.tensor([256.0], device="cuda")
    ws = torch.empty(G.gcn_pair_loss_workspace_size(K), dtype=torch.uint8, device="cuda")
    G.gcn_pair_loss(n, F, ld, prec, Z, dev(u), dev(v), n_pos, n_neg, scale, loss, scores, g, ov, ws)
    torch.cuda.synchronize()
    l_o, s_o, g_o = O.pair_loss(zr, u, v, n_pos, loss_scale=256.0)
    # fp32 arithmetic on identical inputs: fp32 tolerance whatever the storage type
    assert_close(scores.cpu().numpy().astype(np.float64), s_o, G.GCN_F32, "scores")
    assert_close(g.cpu().numpy().astype(np.float64), g_o, G.GCN_F32, "g")
    assert abs(loss.item() - l_o) <= 1e-5 * abs(l_o)
    assert ov.item() == 0


@pytest.mark.parametrize("prec", PRECS, ids=lambda p: PNAME[p])
@pytest.mark.parametrize("F", [64, 130])
def test_pair_backward_matches_oracle(prec, F):
    n, n_pos, n_neg = 2000, 3000, 3000
    rng = np.random.default_rng(43 + F)
    z = (0.5 * rng.standard_normal((n, F))).astype(np.float32)
    u, v = _pairs(n, n_pos, n_neg, 44 + F)
    K = n_pos + n_neg
    gk = (rng.standard_normal(K) * 1e-3).astype(np.float32)
    ld = round8(F)
    Z = z_dev(z, prec, ld)
    dZ = torch.full((n, ld), 7.0, dtype=G.torch_dtype(prec), device="cuda")
    ov = torch.zeros(1, dtype=torch.int32, device="cuda")
    ws = torch.empty(G.gcn_pair_backward_workspace_size(n, K, F), dtype=torch.uint8, device="cuda")
    G.gcn_pair_backward(n, F, ld, prec, Z, dev(u), dev(v), K, dev(gk), dZ, ld, ov, ws)
    torch.cuda.synchronize()
    want = O.pair_backward(n, host(Z, F), u, v, gk.astype(np.float64))
    assert_close(host(dZ, F), want, prec, "dZ")
    assert torch.all(dZ[:, F:].float() == 0)
    assert ov.item() == 0
    # run-to-run identical (fixed summation order per row)
    first = dZ.clone()
    G.gcn_pair_backward(n, F, ld, prec, Z, dev(u), dev(v), K, dev(gk), dZ, ld, ov, ws)
    torch.cuda.synchronize()
    assert torch.equal(first, dZ)


@pytest.mark.parametrize("prec", [G.GCN_F32, G.GCN_F16])
@pytest.mark.parametrize("n,hub_pairs,K", [(100_003, 5000, 9000), (300, 0, 0), (5000, 700, 700), (70_000, 3, 257)])
def test_pair_backward_hub_rows_and_edges(prec, n, hub_pairs, K):
    """Rows whose entries span many 64-entry blocks (a hub in thousands of
    pairs), rows in no pair, no pairs at all, three radix passes (n > 2^16)
    and entry counts just past a block boundary."""
    F = 64
    print(f"[pair-bwd] prec={prec} n={n} hub={hub_pairs} K={K}", flush=True)
    rng = np.random.default_rng(n + K)
    z = (0.5 * rng.standard_normal((n, F))).astype(np.float32)
    u = rng.integers(0, n, K).astype(np.int32)
    v = rng.integers(0, n, K).astype(np.int32)
    if hub_pairs:
        u[:hub_pairs] = 7
        v[hub_pairs // 2: hub_pairs] = n - 1
    gk = (rng.standard_normal(K) * 1e-2).astype(np.float32)
    ld = F
    Z = z_dev(z, prec, ld)
    dZ = torch.full((n, ld), 7.0, dtype=G.torch_dtype(prec), device="cuda")
    ov = torch.zeros(1, dtype=torch.int32, device="cuda")
    ws = torch.empty(G.gcn_pair_backward_workspace_size(n, K, F), dtype=torch.uint8, device="cuda")
    du = dev(u) if K else None
    dv = dev(v) if K else None
    dg = dev(gk) if K else None
    G.gcn_pair_backward(n, F, ld, prec, Z, du, dv, K, dg, dZ, ld, ov, ws)
    torch.cuda.synchronize()
    want = O.pair_backward(n, host(Z, F), u, v, gk.astype(np.float64))
    assert_close(host(dZ, F), want, prec, "dZ")
    assert ov.item() == 0
    first = dZ.clone()
    G.gcn_pair_backward(n, F, ld, prec, Z, du, dv, K, dg, dZ, ld, ov, ws)
    torch.cuda.synchronize()
    assert torch.equal(first, dZ)


def test_pair_invalid_ids_are_skipped():
    n, F, ld = 100, 16, 16
    z = np.random.default_rng(45).standard_normal((n, F)).astype(np.float32)
    u = np.array([1, 2, n, 4, -1], np.int32)
    v = np.array([5, n + 3, 7, 8, 9], np.int32)
    Z = z_dev(z, G.GCN_F32, ld)
    loss = torch.zeros(1, device="cuda")
    scores = torch.empty(5, device="cuda")
    g = torch.empty(5, device="cuda")
    ov = torch.zeros(1, dtype=torch.int32, device="cuda")
    ws = torch.empty(G.gcn_pair_loss_workspace_size(5), dtype=torch.uint8, device="cuda")
    G.gcn_pair_loss(n, F, ld, G.GCN_F32, Z, dev(u), dev(v), 2, 3, None, loss, scores, g, ov, ws)
    torch.cuda.synchronize()
    assert ov.item() == 1
    gh, sh = g.cpu().numpy(), scores.cpu().numpy()
    assert np.all(gh[[1, 2, 4]] == 0) and np.all(np.isnan(sh[[1, 2, 4]]))
    ok = [0, 3]
    _, s_o, _ = O.pair_loss(z.astype(np.float64), u[ok], v[ok], 1)
    assert np.allclose(sh[ok], s_o, rtol=1e-5, atol=1e-6)
    # the backward pass ignores them as well
    dZ = torch.empty((n, ld), device="cuda")
    ov.zero_()
    bws = torch.empty(G.gcn_pair_backward_workspace_size(n, 5, F), dtype=torch.uint8, device="cuda")
    gk = np.array([0.5, 1.0, 1.0, -0.25, 1.0], np.float32)
    G.gcn_pair_backward(n, F, ld, G.GCN_F32, Z, dev(u), dev(v), 5, dev(gk), dZ, ld, ov, bws)
    torch.cuda.synchronize()
    want = O.pair_backward(n, z.astype(np.float64), u[ok], v[ok], gk[ok].astype(np.float64))
    assert_close(dZ.cpu().numpy().astype(np.float64), want, G.GCN_F32, "dZ with skipped pairs")


@pytest.mark.parametrize("P,N", [(1000, 1500), (37, 5), (300, 300), (4000, 6003), (1, 1)])
def test_pair_metrics_match_oracle(P, N):
    rng = np.random.default_rng(46 + P)
    sp = np.round(rng.standard_normal(P) + 0.8, 1).astype(np.float32)   # rounded: ties
    sn = np.round(rng.standard_normal(N), 1).astype(np.float32)
    scores = dev(np.concatenate([sp, sn]))
    out = torch.empty(2, dtype=torch.float64, device="cuda")
    ws = torch.empty(G.gcn_pair_metrics_workspace_size(P, N), dtype=torch.uint8, device="cuda")
    G.gcn_pair_metrics(scores, P, N, out, ws)
    auc, ap = out.cpu().tolist()
    auc_o, ap_o = O.auc_ap(sp.astype(np.float64), sn.astype(np.float64))
    assert auc == auc_o                    # an exact count over P x N
    assert abs(ap - ap_o) <= 1e-12


def _metrics(sp, sn):
    P, N = sp.size, sn.size
    scores = dev(np.concatenate([sp, sn]).astype(np.float32))
    out = torch.empty(2, dtype=torch.float64, device="cuda")
    ws = torch.empty(G.gcn_pair_metrics_workspace_size(P, N), dtype=torch.uint8, device="cuda")
    G.gcn_pair_metrics(scores, P, N, out, ws)
    return out.cpu().tolist()


def test_pair_metrics_ties_signed_zero_and_extremes():
    # every score equal: AUC 1/2, AP = P / (P + N)
    auc, ap = _metrics(np.full(70, 0.25, np.float32), np.full(130, 0.25, np.float32))
    assert auc == 0.5 and abs(ap - 70 / 200) <= 1e-15
    # -0 and +0 are equal scores; negative, denormal and large magnitudes order as floats
    sp = np.array([-0.0, 0.0, 1e-42, -1e-42, 3.0e38, -2.5, 7.0], np.float32)
    sn = np.array([0.0, -0.0, -1e-42, 2e-42, -3.0e38, -2.5, 7.0, 6.999999], np.float32)
    auc, ap = _metrics(sp, sn)
    auc_o, ap_o = O.auc_ap(sp.astype(np.float64), sn.astype(np.float64))
    assert auc == auc_o and abs(ap - ap_o) <= 1e-12
    # perfect and reversed separation
    assert _metrics(np.array([2.0, 3.0], np.float32), np.array([-1.0, 0.5, 1.0], np.float32)) == [1.0, 1.0]
    auc, ap = _metrics(np.array([-2.0, -3.0], np.float32), np.array([-1.0, 0.5, 1.0], np.float32))
    auc_o, ap_o = O.auc_ap(np.array([-2.0, -3.0]), np.array([-1.0, 0.5, 1.0]))
    assert auc == 0.0 and abs(ap - ap_o) <= 1e-15


@pytest.mark.parametrize("prec", [G.GCN_F32, G.GCN_F16], ids=lambda p: PNAME[p])
def test_gae_step_matches_oracle(prec):
    wl = I.gae_workload(0, n_override=2048)
    n = wl["n"]
    n_pos, n_neg, seed = 4000, 4000, 77
    print(f"[gae] n={n} train edges {wl['train_u'].size}", flush=True)
    dg = DeviceGraph(n, wl["train_u"], wl["train_v"], prec=prec, heavy_threshold=48, chunk_nnz=96)
    m = GAE2(dg, wl["X"], wl["W1"], wl["W2"], wl["train_u"], wl["train_v"], prec=prec, n_pos=n_pos, n_neg=n_neg,
             seed=seed, loss_scale=256.0 if prec else 1.0)
    m.encode()
    m.loss_and_backward(epoch=5)
    torch.cuda.synchronize()
    assert m.overflow.item() == 0
    # oracle on the same rounded inputs, layer by layer
    g = O.graph(n, wl["train_u"], wl["train_v"])
    vals = O.norm_values(g)
    rnd = lambda a: torch.as_tensor(np.asarray(a, np.float32)).to(G.torch_dtype(prec)).float().numpy().astype(np.float64)
    x, w1, w2 = rnd(wl["X"]), rnd(wl["W1"]), rnd(wl["W2"])
    _, _, h1 = O.layer_fwd(g, vals, x, w1, np.zeros(w1.shape[1]), "relu", 0.0, True)
    h1r = host(m.H1, m.f_h)
    assert_close(h1r, h1, prec, "H1")
    _, _, z = O.layer_fwd(g, vals, h1r, w2, np.zeros(w2.shape[1]), "none", 0.0, True)
    zr = host(m.Z, m.f_e)
    assert_close(zr, z, prec, "Z")
    u, v = O.sample_pairs(seed, 5, n, wl["train_u"], wl["train_v"], n_pos, n_neg)
    assert np.array_equal(m.pair_u.cpu().numpy(), u) and np.array_equal(m.pair_v.cpu().numpy(), v)
    scale = 256.0 if prec else 1.0
    l_o, _, g_o = O.pair_loss(zr, u, v, n_pos, loss_scale=scale)
    assert abs(m.loss.item() - l_o) <= 1e-5 * abs(l_o)
    # the per-pair gradient (fp32 on the device in every mode)
    assert_close(m.pair_g.cpu().numpy().astype(np.float64), g_o, G.GCN_F32, "pair gradient")
    dz = O.pair_backward(n, zr, u, v, g_o)
    dzr = host(m.dZ, m.f_e)
    assert_close(dzr, dz, prec, "dZ")
    _, dw2, db2, dz1 = O.layer_bwd(g, vals, h1r, rnd(m.W2w().float().cpu().numpy()[:, :m.f_e]), dzr, "relu", 0.0)
    assert_close(m.dW2().cpu().numpy()[:, :m.f_e].astype(np.float64), dw2, prec, "dW2")
    dz1r = host(m.dZ1, m.f_h)
    assert_close(dz1r, dz1, prec, "dZ1")
    _, dw1, _, _ = O.layer_bwd(g, vals, x, w1, dz1r, "none", 0.0)
    assert_close(m.dW1().cpu().numpy()[:, :m.f_h].astype(np.float64), dw1, prec, "dW1")


def test_gae_trains_and_scores_held_out_pairs():
    wl = I.gae_workload(1, n_override=4096)
    n = wl["n"]
    dg = DeviceGraph(n, wl["train_u"], wl["train_v"], prec=G.GCN_F16)
    m = GAE2(dg, wl["X"], wl["W1"], wl["W2"], wl["train_u"], wl["train_v"], prec=G.GCN_F16, n_pos=16384,
             n_neg=16384, seed=3)
    auc0, ap0, loss0 = m.evaluate(wl["test_u"], wl["test_v"], wl["n_test_pos"])
    for ep in range(60):
        m.step(ep)
    auc1, ap1, loss1 = m.evaluate(wl["test_u"], wl["test_v"], wl["n_test_pos"])
    print(f"[gae] AUC {auc0:.3f} -> {auc1:.3f}, AP {ap0:.3f} -> {ap1:.3f}, "
          f"held-out loss {loss0:.3f} -> {loss1:.3f}", flush=True)
    assert m.scaler_state()["skipped"] <= 2
    assert loss1 < loss0 and auc1 > 0.6 and ap1 > 0.6


def test_pair_path_at_full_size():
    """The link-prediction calls at the benchmark's size (R-MAT scale 17
    training edges, 2^20 + 2^20 pairs, F = 64, fp16): the pairs bit-exact,
    sampled scores and gradients against the oracle's per-pair formula, the
    mean loss over all pairs, and sampled rows of dZ (the hubs among them)
    against the oracle's per-row sum."""
    wl = I.gae_workload(0)
    n, F = wl["n"], 64
    n_pos = n_neg = 1 << 20
    K = n_pos + n_neg
    print(f"[gae-full] n={n} K={K}", flush=True)
    eu, ev = wl["train_u"], wl["train_v"]
    pu = torch.empty(K, dtype=torch.int32, device="cuda")
    pv = torch.empty_like(pu)
    G.gcn_sample_pairs(n, dev(eu), dev(ev), n_pos, n_neg, 11, 4, pu, pv)
    u, v = O.sample_pairs(11, 4, n, eu, ev, n_pos, n_neg)
    assert np.array_equal(pu.cpu().numpy(), u) and np.array_equal(pv.cpu().numpy(), v)
    rng = np.random.default_rng(12)
    z = (0.3 * rng.standard_normal((n, F))).astype(np.float32)
    Z = z_dev(z, G.GCN_F16, F)
    zr = host(Z, F)
    scale = torch.tensor([1024.0], device="cuda")
    loss = torch.zeros(1, device="cuda")
    scores = torch.empty(K, device="cuda")
    g = torch.empty(K, device="cuda")
    ov = torch.zeros(1, dtype=torch.int32, device="cuda")
    ws = torch.empty(G.gcn_pair_loss_workspace_size(K), dtype=torch.uint8, device="cuda")
    G.gcn_pair_loss(n, F, F, G.GCN_F16, Z, pu, pv, n_pos, n_neg, scale, loss, scores, g, ov, ws)
    torch.cuda.synchronize()
    s_all = np.einsum("ij,ij->i", zr[u], zr[v])
    y = (np.arange(K) < n_pos).astype(np.float64)
    want_loss = np.mean(np.logaddexp(0.0, s_all) - y * s_all)
    assert abs(loss.item() - want_loss) <= 1e-4 * abs(want_loss)
    ks = np.unique(np.concatenate([[0, n_pos - 1, n_pos, K - 1], rng.choice(K, 500, replace=False)]))
    sg, gg = scores.cpu().numpy()[ks], g.cpu().numpy()[ks]
    assert np.allclose(sg, s_all[ks], rtol=1e-4, atol=1e-4)
    want_g = (1.0 / (1.0 + np.exp(-s_all[ks])) - y[ks]) * 1024.0 / K
    assert np.allclose(gg, want_g, rtol=1e-4, atol=1e-9)
    # backward: sampled rows, hubs included
    gk = g.cpu().numpy().astype(np.float64)
    dZ = torch.empty((n, F), dtype=torch.float16, device="cuda")
    bws = torch.empty(G.gcn_pair_backward_workspace_size(n, K, F), dtype=torch.uint8, device="cuda")
    G.gcn_pair_backward(n, F, F, G.GCN_F16, Z, pu, pv, K, g, dZ, F, ov, bws)
    torch.cuda.synchronize()
    cnt = np.bincount(u, minlength=n) + np.bincount(v, minlength=n)
    rows = np.unique(np.concatenate([np.argsort(cnt)[-5:], rng.choice(n, 40, replace=False),
                                     np.flatnonzero(cnt == 0)[:3]]))
    got = dZ[torch.as_tensor(rows).cuda()].float().cpu().numpy().astype(np.float64)
    want = np.stack([(gk[u == r, None] * zr[v[u == r]]).sum(0) + (gk[v == r, None] * zr[u[v == r]]).sum(0)
                     for r in rows])
    assert_close(got, want, G.GCN_F16, "dZ sampled rows at full size")
    assert ov.item() == 0
