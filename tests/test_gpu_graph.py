"""A training epoch captured into a HIP graph and replayed gives, replay by
replay, the same bits as eager training: the dropout counter read on the
device from the loss-scale state equals the epoch the host would pass, and
nothing in the captured epoch depends on host state.  Eager work and
synchronisations run between the replays, and every replay is compared."""
import numpy as np
import pytest
import torch

from paper_2010_12635_amd import gcn as G
from paper_2010_12635_amd import inputs as I
from paper_2010_12635_amd.model import DeviceGraph, GCN2

pytestmark = pytest.mark.gpu

PARAMS = ("master", "working", "m", "v", "scaler")


def _state(m):
    """Parameters, optimiser state, loss, gradients and the logical columns
    of the activations (padding columns of outputs are not specified)."""
    return dict(master=m.master, working=m.working, m=m.m, v=m.v, scaler=m.scaler, grad=m.grad, loss=m.loss,
                H1=m.H1[:, :m.f_h], Z2=m.Z2[:, :m.C], dZ2=m.dZ2[:, :m.C], dZ1=m.dZ1[:, :m.f_h])


def _model(wl, prec, device_epoch):
    spec = wl["spec"]
    dg = DeviceGraph(wl["n"], wl["src"], wl["dst"], prec=prec, dense=spec.dense_adj)
    return GCN2(dg, wl["X"], wl["labels"], wl["mask"], wl["W1"], wl["W2"], wl["b1"], wl["b2"], prec=prec,
                dropout=spec.dropout, seed=wl["dropout_seed"], loss_scale=spec.loss_scale0 if prec else 1.0,
                device_epoch=device_epoch)


@pytest.mark.parametrize("prec", [G.GCN_F16, G.GCN_F32], ids=["f16", "f32"])
@pytest.mark.parametrize("name,n", [("er2k", None), ("ba200k", 6000), ("sbm16k_dense", 2048)])
def test_graph_replay_matches_eager(name, n, prec):
    print(f"[graph] {name} n={n} prec={prec}", flush=True)
    wl = I.workload(name, 0, n_override=n)
    host = _model(wl, prec, device_epoch=False)       # epoch passed by the host
    dev = _model(wl, prec, device_epoch=True)          # epoch read on the device, eager
    rep = _model(wl, prec, device_epoch=True)          # the same, captured and replayed
    rep.capture()
    torch.cuda.synchronize()
    for t in PARAMS:                                   # capturing ran nothing
        assert torch.equal(getattr(rep, t), getattr(dev, t)), t
    for k in range(6):
        host.step(k)
        dev.step(k)
        rep.replay()
        torch.cuda.synchronize()
        junk = torch.arange(4096, device="cuda", dtype=torch.float32).sum()   # eager work between replays
        assert float(junk) == 4096 * 4095 / 2
        sa, sb, sc = _state(host), _state(dev), _state(rep)
        for t in sa:
            assert torch.equal(sa[t], sb[t]), (k, t, "device counter")
            assert torch.equal(sa[t], sc[t]), (k, t, "graph replay")
    st = rep.scaler_state()
    assert st["step"] + st["skipped"] == 6
    assert np.isfinite(float(rep.loss.item()))


def test_capture_needs_device_epoch():
    wl = I.workload("er2k", 0)
    m = _model(wl, G.GCN_F16, device_epoch=False)
    with pytest.raises(ValueError):
        m.capture()
