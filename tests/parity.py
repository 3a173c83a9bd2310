"""Shared helpers of the GPU parity tests: tolerances and small graphs."""
import numpy as np

# fp32 mode: normwise max relative error per tensor
TOL_F32 = 1e-5
# 16-bit storage / fp32 accumulation: per element, floor at the tensor RMS
TOL_F16 = 2e-2
TOL_BF16 = 1e-1


def f32(x):
    """x rounded to binary32, as the C ABI receives float arguments (e.g.
    dropout_p): the oracle is given the value the library actually sees."""
    return float(np.float32(x))


def tol_for(prec):
    return {0: TOL_F32, 1: TOL_F16, 2: TOL_BF16}[prec]


def assert_close(got, want, prec, what=""):
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    assert got.shape == want.shape, (what, got.shape, want.shape)
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    if prec == 0:
        den = np.max(np.abs(want))
        err = np.max(np.abs(got - want)) / (den if den > 0 else 1.0)
        assert err <= TOL_F32, f"{what}: normwise rel err {err:.3e} > {TOL_F32}"
    else:
        tol = tol_for(prec)
        rms = np.sqrt(np.mean(want * want)) if want.size else 0.0
        bound = tol * np.maximum(np.abs(want), rms)
        bad = np.abs(got - want) > bound
        if bad.any():
            i = np.argmax(np.abs(got - want) / np.maximum(bound, 1e-300))
            raise AssertionError(f"{what}: {bad.sum()} of {bad.size} elements out of tolerance {tol}; "
                                 f"worst at {np.unravel_index(i, got.shape)}: got {got.flat[i]}, want {want.flat[i]}")


def hub_graph(n, m_random, hubs, seed):
    """Raw undirected edge list with repeats, reversed pairs, self-loops and
    a few hubs: hubs = list of (vertex, number of random neighbours)."""
    rng = np.random.default_rng(seed)
    src = [rng.integers(0, n, m_random)]
    dst = [rng.integers(0, n, m_random)]
    for v, k in hubs:
        nb = rng.integers(0, n, k)
        src.append(np.full(k, v))
        dst.append(nb)
    s = np.concatenate(src)
    d = np.concatenate(dst)
    # repeats in both orientations and explicit self-loops
    s = np.concatenate([s, d[:50], np.arange(10)])
    d = np.concatenate([d, s[:50], np.arange(10)])
    return s.astype(np.int32), d.astype(np.int32)
