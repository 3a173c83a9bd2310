"""GPU parity of the precision-level calls (gcn_cast, gcn_optimizer_step_half)
and the training behaviour of the optimisation levels O0-O3 of Section
"Background and Motivation".

* gcn_cast: bit-exact against the oracle's round_storage for fp32 -> 16 bit
  (ties, subnormals, overflow, NaN, infinities), exact widening, strided
  blocks whose padding columns stay untouched, flat buffers with a ragged
  tail; the flag is raised exactly when an output is not finite.
* gcn_optimizer_step_half: one-step maps against the oracle's
  adam_step_half, fed the device state of the previous step; both evaluate
  every operation in binary32 with one rounding each and round its result
  to 16 bits, so the bar is bit equality (NaN positions included).
* Levels: on a small SBM (dense and CSR A_hat) O0, O1 and O2 learn, O1 and
  O2 agree (the same roundings in a different order of casts), O3's first
  update is infinite for most weights and training collapses; peak device
  memory orders as O1 > O0 > O2 >= O3 with a dense A_hat."""
import numpy as np
import pytest
import torch

from oracle import gcn_oracle as O
from paper_2010_12635_amd import gcn as G
from paper_2010_12635_amd import inputs as I
from paper_2010_12635_amd.model import DeviceGraph, GCN2

pytestmark = pytest.mark.gpu

PNAME = {G.GCN_F16: "f16", G.GCN_BF16: "bf16"}


def dev():
    return torch.device("cuda")


def _special_f32(rng, n):
    """Random fp32 values over the whole 16-bit range plus hand-picked
    ties, subnormals, overflow and non-finite values."""
    x = (rng.standard_normal(n) * np.exp2(rng.uniform(-30, 18, n))).astype(np.float32)
    hand = np.float32([65504, 65519.99, 65520, 1e6, 2.0**-24, 2.0**-25, 3 * 2.0**-26, 1 + 2.0**-11,
                       1 + 3 * 2.0**-11, 1 + 2.0**-8, 1 + 3 * 2.0**-8, 1e-8, 0.1, -0.0, np.inf, -np.inf, np.nan,
                       3.4028235e38, 1e-45])
    x[: hand.size] = hand
    return x


def _bits_equal(got, want):
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    nan = np.isnan(want)
    return np.array_equal(np.isnan(got), nan) and np.array_equal(got[~nan], want[~nan]) and \
        np.array_equal(np.signbit(got[~nan]), np.signbit(want[~nan]))


@pytest.mark.parametrize("prec", [G.GCN_F16, G.GCN_BF16])
@pytest.mark.parametrize("count", [1, 7, 8, 1_000_003])
def test_cast_flat_matches_oracle(prec, count):
    print(f"[cast] flat {PNAME[prec]} count={count}", flush=True)
    x = _special_f32(np.random.default_rng(count), max(count, 32))[:count]
    src = torch.as_tensor(x).to(dev())
    dst = torch.full((count + 8,), 7.0, dtype=G.torch_dtype(prec), device=dev())
    ov = torch.zeros(1, dtype=torch.int32, device=dev())
    G.gcn_cast(1, count, G.GCN_F32, src, 0, prec, dst, 0, ov)
    torch.cuda.synchronize()
    got = dst.float().cpu().numpy()
    want = O.round_storage(x, PNAME[prec])
    assert _bits_equal(got[:count], want)
    assert np.all(got[count:] == 7.0)
    assert ov.item() == int(not np.all(np.isfinite(want)))
    # widening back is exact
    back = torch.empty(count, dtype=torch.float32, device=dev())
    ov.zero_()
    G.gcn_cast(1, count, prec, dst, 0, G.GCN_F32, back, 0, ov)
    torch.cuda.synchronize()
    assert _bits_equal(back.cpu().numpy(), want)


@pytest.mark.parametrize("src_prec,dst_prec", [(G.GCN_F32, G.GCN_F16), (G.GCN_F32, G.GCN_BF16),
                                               (G.GCN_F16, G.GCN_F32), (G.GCN_F16, G.GCN_BF16),
                                               (G.GCN_BF16, G.GCN_F16), (G.GCN_F16, G.GCN_F16)])
def test_cast_strided_block(src_prec, dst_prec):
    rows, cols, lds, ldd = 1037, 45, 48, 56
    print(f"[cast] block {rows}x{cols} {src_prec}->{dst_prec}", flush=True)
    rng = np.random.default_rng(9)
    x = np.clip(rng.standard_normal((rows, lds)) * 3.0, -6e4, 6e4).astype(np.float32)
    names = {G.GCN_F32: "f32", G.GCN_F16: "f16", G.GCN_BF16: "bf16"}
    xs = O.round_storage(x, names[src_prec]) if src_prec != G.GCN_F32 else x.astype(np.float64)
    src = torch.as_tensor(xs.astype(np.float32)).to(dev()).to(G.torch_dtype(src_prec))
    dst = torch.full((rows, ldd), -3.0, dtype=G.torch_dtype(dst_prec), device=dev())
    G.gcn_cast(rows, cols, src_prec, src, lds, dst_prec, dst, ldd, None)
    torch.cuda.synchronize()
    got = dst.float().cpu().numpy()
    want = O.round_storage(xs[:, :cols].astype(np.float32), names[dst_prec])
    assert _bits_equal(got[:, :cols], want)
    assert np.all(got[:, cols:] == -3.0)


@pytest.mark.parametrize("prec", [G.GCN_F16, G.GCN_BF16])
@pytest.mark.parametrize("P", [5000, 70001])
def test_half_optimizer_matches_oracle(prec, P):
    print(f"[adam-half] {PNAME[prec]} P={P}", flush=True)
    rng = np.random.default_rng(P)
    dt = G.torch_dtype(prec)
    w0 = O.round_storage(rng.uniform(-1, 1, P).astype(np.float32), PNAME[prec])
    w = torch.as_tensor(w0.astype(np.float32)).to(dev()).to(dt)
    m = torch.zeros(P, dtype=dt, device=dev())
    v = torch.zeros(P, dtype=dt, device=dev())
    widened = torch.empty(P, dtype=torch.float32, device=dev())
    grad = torch.empty(P, dtype=torch.float32, device=dev())
    state = torch.zeros(4, dtype=torch.int32, device=dev())
    state.view(torch.float32)[0] = 1.0
    ov = torch.zeros(1, dtype=torch.int32, device=dev())
    cfg = G.GcnAdamConfig(0.01, 0.9, 0.999, 1e-8, 0.5, 2.0, 2000, 1.0, 2.0**24)
    for step in range(1, 5):
        g = (rng.choice([-1.0, 1.0], P) * np.exp2(rng.uniform(-17, 0, P))).astype(np.float32)
        g[::97] = 0.0
        if step == 2:
            g[5] = np.inf
        grad.copy_(torch.as_tensor(g))
        wb, mb, vb = (t.float().cpu().numpy().astype(np.float64) for t in (w, m, v))
        G.gcn_optimizer_step_half(P, w, grad, m, v, widened, prec, cfg, state, ov)
        torch.cuda.synchronize()
        wo, mo, vo = O.adam_step_half(wb, g, mb, vb, step, PNAME[prec], 0.01, 0.9, 0.999, 1e-8)
        for name, t_, want in (("m", m, mo), ("v", v, vo), ("w", w, wo)):
            got = t_.float().cpu().numpy()
            if not _bits_equal(got, want):
                bad = np.flatnonzero(~((got == want) | (np.isnan(got) & np.isnan(want))))
                raise AssertionError(f"{name} step {step}: {bad.size} of {P} differ, first at {bad[:3]}: "
                                     f"got {got[bad[:3]]}, want {want[bad[:3]]}")
        assert _bits_equal(widened.cpu().numpy(), w.float().cpu().numpy())
        st = state.cpu()
        assert int(st[2]) == step and int(st[3]) == (1 if step >= 2 else 0) and ov.item() == 0
        assert float(st.view(torch.float32)[0]) == 1.0


def test_half_optimizer_underflow_is_infinite():
    # the binary16 instability: |g| = 1e-3 gives v = 0, eps rounds to 0, the
    # update is infinite; bf16 keeps the same step finite
    P = 64
    for prec, finite in ((G.GCN_F16, False), (G.GCN_BF16, True)):
        dt = G.torch_dtype(prec)
        w = torch.ones(P, dtype=dt, device=dev())
        m = torch.zeros(P, dtype=dt, device=dev())
        v = torch.zeros(P, dtype=dt, device=dev())
        grad = torch.full((P,), 1e-3, dtype=torch.float32, device=dev())
        state = torch.zeros(4, dtype=torch.int32, device=dev())
        ov = torch.zeros(1, dtype=torch.int32, device=dev())
        cfg = G.GcnAdamConfig(0.01, 0.9, 0.999, 1e-8, 0.5, 2.0, 2000, 1.0, 2.0**24)
        G.gcn_optimizer_step_half(P, w, grad, m, v, None, prec, cfg, state, ov)
        torch.cuda.synchronize()
        got = w.float().cpu().numpy()
        if finite:
            assert np.all(np.abs(got - 0.99) <= 2 * 2.0**-8)
        else:
            assert np.all(got == -np.inf) and np.all(v.float().cpu().numpy() == 0.0)


# --------------------------------------------------------------- levels

def _train(wl, level, epochs, dense):
    prec = G.GCN_F32 if level == "O0" else G.GCN_F16
    gprec = G.GCN_F32 if level in ("O0", "O1") else G.GCN_F16
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    torch.cuda.reset_peak_memory_stats()
    base = torch.cuda.memory_allocated()
    dg = DeviceGraph(wl["n"], wl["src"], wl["dst"], prec=gprec, dense=dense,
                     tiled=False if level == "O1" else None)
    m = GCN2(dg, wl["X"], wl["labels"], wl["mask"], wl["W1"], wl["W2"], wl["b1"], wl["b2"], prec=prec,
             dropout=0.0, seed=wl["dropout_seed"], loss_scale=1024.0, level=level)
    losses = []
    w1_first = None
    for ep in range(epochs):
        m.step(ep)
        losses.append(float(m.loss.item()))
        if ep == 0:
            w1_first = m.working[: m.f_in * m.ld_h].float().cpu().numpy()
    acc = int(m.n_correct.item()) / m.n_mask
    peak = torch.cuda.max_memory_allocated() - base
    st = m.scaler_state()
    del m, dg
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return dict(losses=np.array(losses), acc=acc, peak=peak, w1_first=w1_first, state=st)


@pytest.fixture(scope="module")
def small_sbm():
    return I.workload("sbm16k_dense", 0, n_override=2048)


@pytest.mark.parametrize("dense", [True, False])
def test_levels_training_behaviour(small_sbm, dense):
    wl = small_sbm
    runs = {}
    for level in ("O0", "O1", "O2", "O3"):
        print(f"[levels] {level} dense={dense}", flush=True)
        runs[level] = _train(wl, level, 100, dense)
        r = runs[level]
        print(f"[levels] {level}: loss {r['losses'][0]:.4f} -> {r['losses'][-1]:.4f}, acc {r['acc']:.4f}, "
              f"peak {r['peak']}, scaler {r['state']}", flush=True)
    chance = 1.0 / wl["spec"].classes
    l0 = runs["O0"]["losses"]
    assert l0[-1] < 0.5 * l0[0] and runs["O0"]["acc"] > 2 * chance
    for level in ("O1", "O2"):
        r = runs[level]
        assert np.all(np.isfinite(r["losses"])), level
        assert abs(r["losses"][-1] - l0[-1]) <= 0.1 * l0[-1] + 1e-3, (level, r["losses"][-1], l0[-1])
        assert abs(r["acc"] - runs["O0"]["acc"]) <= 0.05, (level, r["acc"])
    # O1 and O2 round the same values at the same points
    assert np.allclose(runs["O1"]["losses"], runs["O2"]["losses"], rtol=1e-2, atol=1e-3)
    # O3: the first update sends most first-layer weights to +-inf or NaN ...
    w1 = runs["O3"]["w1_first"]
    assert np.mean(~np.isfinite(w1)) > 0.5
    # ... and training collapses
    r3 = runs["O3"]
    assert (not np.isfinite(r3["losses"][-1])) or r3["acc"] < chance + 0.1
    if dense:
        p = {k: r["peak"] for k, r in runs.items()}
        print(f"[levels] peak bytes {p}", flush=True)
        assert p["O1"] > p["O0"] > p["O2"] >= p["O3"]
