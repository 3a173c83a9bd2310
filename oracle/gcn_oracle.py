"""CPU fp64 oracle for the GCN training hot path.

TEST INFRASTRUCTURE ONLY.  This module is the slow, plain reference that the
HIP library is checked against.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import it; the product path never does.  It
shares no code with the HIP path (no kernels, headers, helpers or constant
tables) and imports nothing from the library package.

What it computes follows the paper's statement of the problem
(Section "Graph Convolutions", Eq. (1); Section "Background and Motivation",
optimisation levels O0 and O2; Section "Reduced Precision Changes") together
with the readings recorded in the design notes for everything the paper
leaves open:

* graph(): undirected graph G=(V,E) given as unordered vertex pairs; input
  self-loops and repeated pairs are dropped, each edge is stored in both
  directions and one self-loop per vertex is added (A + I).
* norm_values(): A_hat = D^-1/2 (A + I) D^-1/2, D counting the self-loop
  (the renormalised adjacency of Kipf & Welling, which the paper cites for
  the normalised adjacency it feeds to every layer).
* layer_fwd(): one layer of Eq. (1) read as A_hat (H W) + b, then ReLU and
  inverted dropout on hidden layers, identity on the output layer.
* softmax_ce(): masked mean softmax cross-entropy with a scaled gradient.
* layer_bwd(): the exact gradients of layer_fwd.
* adam_step() / LossScaler: fp32 master weights updated by Adam on unscaled
  gradients, dynamic loss scaling that skips a step and halves the scale on
  overflow and doubles it after a run of good steps (O1/O2 description).
* round_to() / round_storage(): rounding to the 16-bit storage types
  (the casts of the O1 cast policy and of every 16-bit tensor).
* adam_step_half(): the O3 level, Adam with parameters and moments held in
  16 bits and no loss scale, each elementwise operation rounded.
* philox4x32(), philox4x64(): the counter-based generators (Salmon et al.,
  SC'11) that draw the dropout keep decisions (4x32, the generator behind
  PyTorch's GPU dropout, the framework the paper trains with) and the
  decoder's pairs (4x64).
* Link prediction (Section "Graph Auto-Encoders", Eq. (2): the decoder
  sigma(Z Z^T) read on sampled vertex pairs): sample_pairs() draws an
  epoch's positive and negative pairs, pair_loss() scores them by inner
  products and takes the mean logistic (binary cross-entropy) loss and its
  gradient per pair, pair_backward() scatters that gradient into dZ, and
  auc_ap() gives the area under the ROC curve and the average precision
  of held-out pairs (the paper's link-prediction metrics).

Every floating-point quantity is float64.  Parity status: every function
here is pinned by the CPU tests (brute force, closed forms, invariants,
finite differences, library special cases); none is "parity unpinned".
"""
from __future__ import annotations

import numpy as np

__all__ = [
    "Graph", "graph", "norm_values", "dinv_f32", "dense_adj", "transpose_csr",
    "spmm", "philox4x32", "philox4x64", "dropout_words", "dropout_keep", "layer_fwd", "softmax_ce",
    "graph_degrees", "graph_rows", "dropout_keep_rows", "norm_adj_matvec",
    "layer_bwd", "adam_step", "LossScaler", "AdamState",
    "PAIR_STREAM", "sample_pairs", "pair_loss", "pair_backward", "auc_ap",
    "round_to", "round_storage", "adam_step_half",
]


# ---------------------------------------------------------------------------
# Graph and normalised adjacency
# ---------------------------------------------------------------------------

class Graph:
    """Canonical CSR of A + I: rows sorted, columns sorted and unique."""

    def __init__(self, n, rowptr, colidx):
        self.n = int(n)
        self.rowptr = rowptr          # int64 [n+1]
        self.colidx = colidx          # int32 [nnz]

    @property
    def nnz(self):
        return int(self.rowptr[-1])

    @property
    def deg(self):
        """Degree of A + I (the self-loop counts once)."""
        return np.diff(self.rowptr).astype(np.int32)

    def rows(self):
        """Row index of every stored entry."""
        return np.repeat(np.arange(self.n, dtype=np.int64), np.diff(self.rowptr))


def graph(n, src, dst):
    """Build the canonical CSR of A + I from an undirected edge list.

    The paper's graphs are undirected with edges as unordered vertex pairs
    (Section "Introduction", footnote on A); pairs are therefore taken as
    sets {u, v}: a pair and its reverse are the same edge, repeats collapse,
    and u == v pairs are dropped because the self-loop of every vertex is
    added exactly once afterwards (the "+ I" of the renormalised adjacency).
    Vertex ids outside [0, n) raise ValueError.
    """
    src = np.asarray(src, dtype=np.int64)
    dst = np.asarray(dst, dtype=np.int64)
    if src.shape != dst.shape:
        raise ValueError("src and dst differ in length")
    if src.size and (src.min() < 0 or dst.min() < 0 or src.max() >= n or dst.max() >= n):
        raise ValueError("vertex id out of range")
    keep = src != dst
    lo = np.minimum(src[keep], dst[keep])
    hi = np.maximum(src[keep], dst[keep])
    pairs = np.unique(lo * n + hi)                      # each undirected edge once
    u, v = pairs // n, pairs % n
    loops = np.arange(n, dtype=np.int64)
    rows = np.concatenate([u, v, loops])
    cols = np.concatenate([v, u, loops])
    order = np.lexsort((cols, rows))                    # by row, then column
    rows, cols = rows[order], cols[order]
    counts = np.bincount(rows, minlength=n)
    rowptr = np.zeros(n + 1, np.int64)
    np.cumsum(counts, out=rowptr[1:])
    return Graph(n, rowptr, cols.astype(np.int32))


def _undirected_pairs(n, src, dst):
    """Distinct unordered pairs {u, v}, u != v, as sorted int64 keys u*n+v (u<v)."""
    src = np.asarray(src, dtype=np.int64)
    dst = np.asarray(dst, dtype=np.int64)
    if src.size and (src.min() < 0 or dst.min() < 0 or src.max() >= n or dst.max() >= n):
        raise ValueError("vertex id out of range")
    keep = src != dst
    return np.unique(np.minimum(src[keep], dst[keep]) * n + np.maximum(src[keep], dst[keep]))


def graph_degrees(n, src, dst):
    """Degrees of A + I (as in graph()) without building the CSR: each
    distinct unordered pair adds one to both endpoints, plus one self-loop."""
    pairs = _undirected_pairs(n, src, dst)
    deg = np.bincount(pairs // n, minlength=n) + np.bincount(pairs % n, minlength=n) + 1
    return deg.astype(np.int32)


def graph_rows(n, src, dst, rows):
    """Sorted neighbour lists (self-loop included) of the selected rows of
    A + I, as in graph(); for checks of sampled rows of large graphs."""
    pairs = _undirected_pairs(n, src, dst)
    u, v = pairs // n, pairs % n
    out = {}
    for r in rows:
        nb = np.concatenate([v[u == r], u[v == r], [r]])
        out[int(r)] = np.sort(nb)
    return out


def norm_adj_matvec(n, src, dst, y):
    """A_hat y (fp64) for a vector or n x k block y, straight from the
    distinct unordered pairs: (A_hat y)_i = d_i^-1/2 (d_i^-1/2 y_i +
    sum over pairs {i, j} of d_j^-1/2 y_j)."""
    pairs = _undirected_pairs(n, src, dst)
    u, v = pairs // n, pairs % n
    deg = np.bincount(u, minlength=n) + np.bincount(v, minlength=n) + 1
    d = 1.0 / np.sqrt(deg.astype(np.float64))
    y = np.asarray(y, np.float64)
    yy = y.reshape(n, -1)
    acc = d[:, None] * yy
    for c in range(yy.shape[1]):
        acc[:, c] += np.bincount(u, weights=d[v] * yy[v, c], minlength=n)
        acc[:, c] += np.bincount(v, weights=d[u] * yy[u, c], minlength=n)
    return (d[:, None] * acc).reshape(y.shape)


def dinv_f32(g: Graph):
    """D^-1/2 rounded once to float32 from the fp64 value 1/sqrt(deg)."""
    return (1.0 / np.sqrt(g.deg.astype(np.float64))).astype(np.float32)


def norm_values(g: Graph):
    """Stored values of A_hat = D^-1/2 (A+I) D^-1/2 (fp64), one per CSR entry."""
    d = 1.0 / np.sqrt(g.deg.astype(np.float64))
    return d[g.rows()] * d[g.colidx.astype(np.int64)]


def dense_adj(g: Graph, values=None):
    """A_hat as a dense n x n fp64 array (the paper's own storage, Section
    "Reduced Precision Changes": every tensor was cast to dense)."""
    if values is None:
        values = norm_values(g)
    a = np.zeros((g.n, g.n), np.float64)
    a[g.rows(), g.colidx.astype(np.int64)] = values
    return a


def transpose_csr(g: Graph, values):
    """CSR of the transpose, built by swapping row and column of every entry.
    Used by the backward pass so that it does not rely on A_hat being
    symmetric."""
    rows = g.rows()
    cols = g.colidx.astype(np.int64)
    order = np.lexsort((rows, cols))
    t_rows, t_cols, t_vals = cols[order], rows[order], values[order]
    counts = np.bincount(t_rows, minlength=g.n)
    rowptr = np.zeros(g.n + 1, np.int64)
    np.cumsum(counts, out=rowptr[1:])
    return Graph(g.n, rowptr, t_cols.astype(np.int32)), t_vals


def spmm(g: Graph, values, x, block_entries=1 << 22):
    """Y = A X for A in CSR (fp64): Y[i] = sum over stored (i, j) of a_ij X[j].

    Rows are taken in consecutive blocks of about ``block_entries`` stored
    entries (at least one row per block), so that the products a_ij X[j]
    held at once stay bounded on graphs with many millions of entries; each
    row's terms are summed in entry order."""
    x = np.asarray(x, np.float64)
    values = np.asarray(values, np.float64)
    rp = np.asarray(g.rowptr, np.int64)
    y = np.zeros((g.n, x.shape[1]), np.float64)
    r0 = 0
    while r0 < g.n:
        # last row r1 whose block still holds at most block_entries entries
        r1 = int(np.searchsorted(rp, rp[r0] + block_entries, side="right")) - 1
        r1 = min(max(r1, r0 + 1), g.n)
        p0, p1 = int(rp[r0]), int(rp[r1])
        if p1 > p0:
            prod = values[p0:p1, None] * x[g.colidx[p0:p1].astype(np.int64)]
            counts = np.diff(rp[r0:r1 + 1])
            live = counts > 0
            starts = rp[r0:r1][live] - p0
            y[r0:r1][live] = np.add.reduceat(prod, starts, axis=0)
        r0 = r1
    return y


# ---------------------------------------------------------------------------
# Counter-based RNGs: Philox-4x64-10 (the decoder's pairs) and Philox-4x32-10
# (dropout) (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as easy as
# 1, 2, 3", SC'11)
# ---------------------------------------------------------------------------

_M64 = (1 << 64) - 1
_PHILOX_M0 = 0xD2E7470EE14C6C93
_PHILOX_M1 = 0xCA5A826395121157
_PHILOX_W0 = 0x9E3779B97F4A7C15
_PHILOX_W1 = 0xBB67AE8584CAA73B


def _mulhilo64(a, b):
    """Full 128-bit product of uint64 arrays a*b split into (hi, lo), via
    32-bit halves (numpy has no 128-bit integers)."""
    mask32 = np.uint64(0xFFFFFFFF)
    s32 = np.uint64(32)
    a = a.astype(np.uint64)
    b = np.uint64(b) if np.isscalar(b) else b.astype(np.uint64)
    a_lo, a_hi = a & mask32, a >> s32
    b_lo, b_hi = b & mask32, b >> s32
    ll = a_lo * b_lo
    lh = a_lo * b_hi
    hl = a_hi * b_lo
    hh = a_hi * b_hi
    mid = (ll >> s32) + (lh & mask32) + (hl & mask32)
    lo = (ll & mask32) | ((mid & mask32) << s32)
    hi = hh + (lh >> s32) + (hl >> s32) + (mid >> s32)
    return hi, lo


def philox4x64(ctr, key, rounds=10):
    """Philox-4x64 with ``rounds`` rounds.  ctr: uint64 array [..., 4];
    key: uint64 array [..., 2].  Returns uint64 [..., 4].

    Each round multiplies words 0 and 2 by the two round multipliers, forms
    the new state (hi(M1*x2) ^ x1 ^ k0, lo(M1*x2), hi(M0*x0) ^ x3 ^ k1,
    lo(M0*x0)), and the key is bumped by the two Weyl constants between
    rounds."""
    with np.errstate(over="ignore"):
        c = np.array(ctr, dtype=np.uint64, copy=True)
        k = np.array(key, dtype=np.uint64, copy=True)
        x0, x1, x2, x3 = c[..., 0], c[..., 1], c[..., 2], c[..., 3]
        k0, k1 = k[..., 0], k[..., 1]
        for r in range(rounds):
            hi0, lo0 = _mulhilo64(x0, _PHILOX_M0)
            hi1, lo1 = _mulhilo64(x2, _PHILOX_M1)
            x0, x1, x2, x3 = hi1 ^ x1 ^ k0, lo1, hi0 ^ x3 ^ k1, lo0
            if r + 1 < rounds:
                k0 = k0 + np.uint64(_PHILOX_W0)
                k1 = k1 + np.uint64(_PHILOX_W1)
        return np.stack([x0, x1, x2, x3], axis=-1)


_P32_M0 = 0xD2511F53
_P32_M1 = 0xCD9E8D57
_P32_W0 = 0x9E3779B9
_P32_W1 = 0xBB67AE85


def philox4x32(ctr, key, rounds=10):
    """Philox-4x32 with ``rounds`` rounds.  ctr: array [..., 4] of 32-bit
    words, key: [..., 2] (any integer dtype; values taken mod 2^32).  Returns
    uint64 [..., 4] holding the four 32-bit output words.

    Each round forms the 64-bit products M0*x0 and M1*x2 (exact in uint64),
    the new state (hi(M1*x2) ^ x1 ^ k0, lo(M1*x2), hi(M0*x0) ^ x3 ^ k1,
    lo(M0*x0)), and bumps the key by the two Weyl constants mod 2^32 between
    rounds."""
    mask = np.uint64(0xFFFFFFFF)
    s32 = np.uint64(32)
    c = np.array(ctr, dtype=np.uint64, copy=True) & mask
    k = np.array(key, dtype=np.uint64, copy=True) & mask
    x0, x1, x2, x3 = c[..., 0], c[..., 1], c[..., 2], c[..., 3]
    k0, k1 = k[..., 0], k[..., 1]
    for r in range(rounds):
        p0 = x0 * np.uint64(_P32_M0)
        p1 = x2 * np.uint64(_P32_M1)
        x0, x1, x2, x3 = (p1 >> s32) ^ x1 ^ k0, p1 & mask, (p0 >> s32) ^ x3 ^ k1, p0 & mask
        if r + 1 < rounds:
            k0 = (k0 + np.uint64(_P32_W0)) & mask
            k1 = (k1 + np.uint64(_P32_W1)) & mask
    return np.stack([x0, x1, x2, x3], axis=-1)


def dropout_words(seed, layer_id, epoch, e):
    """The 32-bit dropout word of each element linear index e (uint64 array):
    word e % 4 of the Philox-4x32-10 block with counter (b mod 2^32,
    b div 2^32, epoch mod 2^32, layer_id), b = e div 4, and key
    (seed mod 2^32, seed div 2^32 mod 2^32)."""
    e = np.asarray(e, np.uint64)
    b = e >> np.uint64(2)
    mask = np.uint64(0xFFFFFFFF)
    ctr = np.empty(e.shape + (4,), np.uint64)
    ctr[..., 0] = b & mask
    ctr[..., 1] = b >> np.uint64(32)
    ctr[..., 2] = np.uint64(int(epoch) & 0xFFFFFFFF)
    ctr[..., 3] = np.uint64(int(layer_id) & 0xFFFFFFFF)
    key = np.empty(e.shape + (2,), np.uint64)
    key[..., 0] = np.uint64(int(seed) & 0xFFFFFFFF)
    key[..., 1] = np.uint64((int(seed) >> 32) & 0xFFFFFFFF)
    out = philox4x32(ctr, key)
    w = (e & np.uint64(3)).astype(np.int64)
    return np.take_along_axis(out, w[..., None], axis=-1)[..., 0]


def dropout_keep(seed, layer_id, epoch, n, f, p):
    """Keep mask (bool n x f) of inverted dropout with drop probability p.

    Element (i, j) has linear index e = i*f + j over the logical width f and
    is kept iff its word (dropout_words) >= floor(p * 2^32)."""
    e = np.arange(n * f, dtype=np.uint64)
    thr = np.uint64(int(np.floor(p * 4294967296.0)))
    return (dropout_words(seed, layer_id, epoch, e) >= thr).reshape(n, f)


def dropout_keep_rows(seed, layer_id, epoch, rows, f, p):
    """dropout_keep() restricted to the given rows (same element indexing
    e = i*f + j over the logical width f)."""
    rows = np.asarray(rows, np.int64)
    e = (rows[:, None] * f + np.arange(f, dtype=np.int64)[None, :]).astype(np.uint64)
    thr = np.uint64(int(np.floor(p * 4294967296.0)))
    return dropout_words(seed, layer_id, epoch, e) >= thr


# ---------------------------------------------------------------------------
# Layer forward / backward, loss
# ---------------------------------------------------------------------------

def layer_fwd(g: Graph, values, h, w, b, act="relu", p=0.0, training=True,
              seed=0, layer_id=0, epoch=0, dense=None):
    """One GCN layer, Eq. (1): S = H W, Z = A_hat S + b; hidden layers apply
    ReLU then inverted dropout (kept entries scaled by 1/(1-p)), the output
    layer returns Z unchanged.  ``dense`` (optional n x n fp64) replaces the
    CSR product by the dense one.  Returns (S, Z, H_out), all fp64."""
    h = np.asarray(h, np.float64)
    w = np.asarray(w, np.float64)
    s = h @ w
    z = (dense @ s) if dense is not None else spmm(g, values, s)
    if b is not None:
        z = z + np.asarray(b, np.float64)[None, :]
    if act == "relu":
        out = np.maximum(z, 0.0)
        if training and p > 0.0:
            keep = dropout_keep(seed, layer_id, epoch, g.n, w.shape[1], p)
            out = np.where(keep, out / (1.0 - p), 0.0)
    elif act == "none":
        out = z
    else:
        raise ValueError(act)
    return s, z, out


def softmax_ce(logits, labels, mask=None, loss_scale=1.0):
    """Masked mean softmax cross-entropy.

    loss = mean over masked rows i of (logsumexp(z_i) - z_i[y_i]);
    dlogits = loss_scale * (softmax(z_i) - onehot(y_i)) / |mask| on masked
    rows and 0 elsewhere; n_correct counts masked rows whose arg-max (lowest
    index on ties) equals the label.  Returns (loss, dlogits, n_correct)."""
    z = np.asarray(logits, np.float64)
    n, c = z.shape
    m = np.ones(n, bool) if mask is None else np.asarray(mask).astype(bool)
    cnt = int(m.sum())
    zmax = z.max(axis=1, keepdims=True)
    ez = np.exp(z - zmax)
    se = ez.sum(axis=1, keepdims=True)
    lse = zmax[:, 0] + np.log(se[:, 0])
    y = np.asarray(labels, np.int64)
    per_row = lse - z[np.arange(n), y]
    loss = per_row[m].sum() / cnt if cnt else 0.0
    sm = ez / se
    onehot = np.zeros_like(z)
    onehot[np.arange(n), y] = 1.0
    d = (sm - onehot) * (loss_scale / cnt if cnt else 0.0)
    d[~m] = 0.0
    n_correct = int((np.argmax(z, axis=1) == y)[m].sum())
    return loss, d, n_correct


def layer_bwd(g: Graph, values, h, w, dz, act_below="relu", p_below=0.0, dense=None,
              need_dh=True):
    """Gradients of layer_fwd given dZ (gradient w.r.t. Z = A_hat S + b).

    G_S = A_hat^T dZ (explicit transpose, no symmetry assumed);
    dW = H^T G_S; db = column sums of dZ; dH = G_S W^T; and, when H was
    produced by ReLU + inverted dropout, dZ_below = dH * [H > 0] / (1 - p)
    (the ReLU derivative at 0 is taken as 0).  Returns (G_S, dW, db,
    dZ_below or None)."""
    h = np.asarray(h, np.float64)
    w = np.asarray(w, np.float64)
    dz = np.asarray(dz, np.float64)
    if dense is not None:
        gs = dense.T @ dz
    else:
        gt, vt = transpose_csr(g, values)
        gs = spmm(gt, vt, dz)
    dw = h.T @ gs
    db = dz.sum(axis=0)
    dzb = None
    if need_dh:
        dh = gs @ w.T
        if act_below == "relu":
            dzb = np.where(h > 0.0, dh / (1.0 - p_below), 0.0)
        elif act_below == "none":
            dzb = dh
        else:
            raise ValueError(act_below)
    return gs, dw, db, dzb


# ---------------------------------------------------------------------------
# Optimiser with fp32 master weights and dynamic loss scaling
# ---------------------------------------------------------------------------

class LossScaler:
    """Dynamic loss scale state machine (O1/O2 "dynamic loss scaling"):
    on overflow skip the update and multiply the scale by ``backoff``
    (not below ``min_scale``) and reset the good-step counter; otherwise
    count the good step and multiply the scale by ``growth`` (not above
    ``max_scale``) after ``interval`` consecutive good steps."""

    def __init__(self, scale=65536.0, backoff=0.5, growth=2.0, interval=2000,
                 min_scale=1.0, max_scale=16777216.0):
        self.scale = float(scale)
        self.backoff, self.growth, self.interval = backoff, growth, interval
        self.min_scale, self.max_scale = min_scale, max_scale
        self.good = 0
        self.skipped = 0

    def update(self, overflow: bool) -> bool:
        """Advance one step; returns True when the parameter update applies."""
        if overflow:
            self.scale = max(self.scale * self.backoff, self.min_scale)
            self.good = 0
            self.skipped += 1
            return False
        self.good += 1
        if self.good == self.interval:
            self.scale = min(self.scale * self.growth, self.max_scale)
            self.good = 0
        return True


class AdamState:
    def __init__(self, size):
        self.m = np.zeros(size, np.float64)
        self.v = np.zeros(size, np.float64)
        self.t = 0


def adam_step(master, grad_scaled, state: AdamState, scaler: LossScaler,
              lr=0.01, beta1=0.9, beta2=0.999, eps=1e-8):
    """One optimiser step on the fp32 master weights (as fp64 here).

    overflow = any non-finite scaled gradient.  On overflow nothing but the
    scaler changes.  Otherwise g = grad / scale and Adam (Kingma & Ba) with
    bias correction: m = b1 m + (1-b1) g, v = b2 v + (1-b2) g^2,
    theta -= lr * (m / (1-b1^t)) / (sqrt(v / (1-b2^t)) + eps).
    Returns (new master, applied)."""
    grad_scaled = np.asarray(grad_scaled, np.float64)
    overflow = not np.all(np.isfinite(grad_scaled))
    scale = scaler.scale
    applied = scaler.update(overflow)
    if not applied:
        return np.array(master, np.float64, copy=True), False
    g = grad_scaled / scale
    state.t += 1
    state.m = beta1 * state.m + (1.0 - beta1) * g
    state.v = beta2 * state.v + (1.0 - beta2) * g * g
    mhat = state.m / (1.0 - beta1 ** state.t)
    vhat = state.v / (1.0 - beta2 ** state.t)
    new = np.asarray(master, np.float64) - lr * mhat / (np.sqrt(vhat) + eps)
    return new, True


# ---------------------------------------------------------------------------
# Storage rounding and the pure 16-bit optimiser (optimisation level O3)
# ---------------------------------------------------------------------------

_FORMATS = {            # fraction bits, smallest normal exponent, largest finite value
    "f16": (10, -14, 65504.0),
    "bf16": (7, -126, 255.0 * 2.0 ** 120),
}


def round_to(z, prec):
    """float64 values ``z`` rounded to the 16-bit format ``prec`` ("f16":
    IEEE 754 binary16; "bf16": 8 exponent bits, 7 fraction bits) with
    round-to-nearest, ties to even, straight from the exact value.

    Written out from the formats' definition: around |z| the representable
    values are spaced 2^(e - p) apart, with p the fraction bits and
    e = max(floor(log2 |z|), e_min) (the subnormal range shares the
    spacing of the smallest binade); z / spacing is rounded to the nearest
    integer, ties to the even one; a result beyond the largest finite value
    becomes infinity.  NaN, infinities and signed zeros pass through."""
    if prec == "f32":
        return np.asarray(z, np.float32).astype(np.float64)
    p, emin, vmax = _FORMATS[prec]
    z = np.asarray(z, np.float64)
    out = z.copy()
    fin = np.isfinite(z) & (z != 0.0)
    if np.any(fin):
        a = np.abs(z[fin])
        e = np.floor(np.log2(a))
        # floor(log2) of a float64 can be off by one next to powers of two
        e = np.where(np.exp2(e) > a, e - 1.0, e)
        e = np.where(np.exp2(e + 1.0) <= a, e + 1.0, e)
        e = np.maximum(e, float(emin))
        spacing = np.exp2(e - p)
        q = a / spacing                  # exact: division by a power of two
        lo = np.floor(q)
        frac = q - lo
        up = (frac > 0.5) | ((frac == 0.5) & (np.mod(lo, 2.0) == 1.0))
        mag = (lo + up) * spacing
        out[fin] = np.copysign(np.where(mag > vmax, np.inf, mag), z[fin])
    return out


def round_storage(x, prec):
    """Values of float32 array ``x`` stored in a 16-bit type (the cast of
    the O1 cast lists and of every 16-bit tensor), as float64.
    "f16": round_to(x, "f16").  "bf16": the upper half of the binary32
    encoding after rounding its lower 16 bits to nearest, ties to even
    (NaN stays NaN) -- the encoding-level statement of the same rounding.
    "f32": x itself."""
    x32 = np.asarray(x, np.float32)
    if prec == "bf16":
        b = x32.view(np.uint32).astype(np.uint64)
        r = ((b + np.uint64(0x7FFF) + ((b >> np.uint64(16)) & np.uint64(1))) >> np.uint64(16)) << np.uint64(16)
        out = r.astype(np.uint32).view(np.float32).astype(np.float64)
        out[np.isnan(x32)] = np.nan
        return out
    return round_to(x32.astype(np.float64), prec)


def adam_step_half(w, grad, m, v, t, prec="f16", lr=0.01, beta1=0.9, beta2=0.999, eps=1e-8):
    """One Adam step of optimisation level O3 (Section "Background and
    Motivation": every operation in 16 bits): parameters and both moments
    are held in the storage type ``prec``, there is no master copy and no
    loss scale, and a non-finite value is applied like any other.

    Reading: an elementwise operation on 16-bit tensors is evaluated in
    single precision (IEEE binary32, one rounding per arithmetic operation,
    no fused multiply-add) and its result rounded to the storage type.
    Each line is one such operation, r() the rounding to ``prec``:
        g  = r(grad)
        m' = r(b1 * m + (1 - b1) * g)
        v' = r(b2 * v + ((1 - b2) * g) * g)
        mh = r(m' / c1),  c1 = 1 - b1^t
        vh = r(v' / c2),  c2 = 1 - b2^t
        d  = r(r(sqrt(vh)) + eps)
        w' = r(w - r((lr * mh) / d))
    The hyper-parameters are binary32 values; the bias corrections c1, c2
    are 1 - b^t evaluated exactly (here in float64) and rounded to binary32.
    t >= 1 is the step number of this update.
    Returns (w', m', v') as float64 arrays of representable values."""
    f32 = np.float32

    def r(z):     # binary32 result -> storage type
        return f32(round_to(np.asarray(z, f32).astype(np.float64), prec)) if np.ndim(z) == 0 else \
            round_to(np.asarray(z, f32).astype(np.float64), prec).astype(f32)

    lr, b1, b2, eps = (f32(z) for z in (lr, beta1, beta2, eps))
    c1 = f32(1.0 - float(b1) ** t)
    c2 = f32(1.0 - float(b2) ** t)
    w = np.asarray(w, np.float64).astype(f32)
    m = np.asarray(m, np.float64).astype(f32)
    v = np.asarray(v, np.float64).astype(f32)
    with np.errstate(divide="ignore", invalid="ignore", over="ignore"):
        g = r(np.asarray(grad, f32))
        m2 = r(b1 * m + (f32(1) - b1) * g)
        v2 = r(b2 * v + ((f32(1) - b2) * g) * g)
        mh = r(m2 / c1)
        vh = r(v2 / c2)
        d = r(r(np.sqrt(vh)) + eps)
        w2 = r(w - r((lr * mh) / d))
    return w2.astype(np.float64), m2.astype(np.float64), v2.astype(np.float64)


# ---------------------------------------------------------------------------
# Link prediction: Eq. (2) on sampled pairs
# ---------------------------------------------------------------------------

PAIR_STREAM = 0x50414952   # second key word of the pair sampler's Philox stream


def sample_pairs(seed, epoch, n, edge_u, edge_v, n_pos, n_neg):
    """Pairs of one training epoch of the decoder.  Pair k (0 <= k <
    n_pos + n_neg) takes the Philox-4x64-10 block with key (seed,
    PAIR_STREAM) and counter (k, epoch, 0, 0), outputs w0, w1:
      k <  n_pos: the training edge e = w0 mod n_edges, (u, v) = (edge_u[e], edge_v[e]);
      k >= n_pos: u = w0 mod n, v = (u + 1 + (w1 mod (n - 1))) mod n, so v != u.
    Returns int32 arrays u, v; pairs k < n_pos are positives (label 1)."""
    total = n_pos + n_neg
    ctr = np.zeros((total, 4), np.uint64)
    ctr[:, 0] = np.arange(total, dtype=np.uint64)
    ctr[:, 1] = np.uint64(epoch)
    key = np.zeros((total, 2), np.uint64)
    key[:, 0] = np.uint64(seed & _M64)
    key[:, 1] = np.uint64(PAIR_STREAM)
    out = philox4x64(ctr, key)
    w0, w1 = out[:, 0], out[:, 1]
    edge_u = np.asarray(edge_u, np.int64)
    edge_v = np.asarray(edge_v, np.int64)
    u = np.empty(total, np.int64)
    v = np.empty(total, np.int64)
    e = (w0[:n_pos] % np.uint64(edge_u.size)).astype(np.int64)
    u[:n_pos], v[:n_pos] = edge_u[e], edge_v[e]
    un = w0[n_pos:] % np.uint64(n)
    u[n_pos:] = un.astype(np.int64)
    v[n_pos:] = ((un + np.uint64(1) + w1[n_pos:] % np.uint64(n - 1)) % np.uint64(n)).astype(np.int64)
    return u.astype(np.int32), v.astype(np.int32)


def _softplus(x):
    return np.maximum(x, 0.0) + np.log1p(np.exp(-np.abs(x)))


def _sigmoid(x):
    out = np.empty_like(x)
    pos = x >= 0
    out[pos] = 1.0 / (1.0 + np.exp(-x[pos]))
    ex = np.exp(x[~pos])
    out[~pos] = ex / (1.0 + ex)
    return out


def pair_loss(Z, u, v, n_pos, loss_scale=1.0):
    """Decoder of Eq. (2) on pairs: score s_k = <Z[u_k], Z[v_k]>, label
    y_k = 1 for k < n_pos else 0, loss = mean_k BCE(sigmoid(s_k), y_k)
    = mean_k softplus(s_k) - y_k s_k, gradient per pair
    g_k = loss_scale * (sigmoid(s_k) - y_k) / K (K = number of pairs).
    Returns (loss, scores, g)."""
    z = np.asarray(Z, np.float64)
    u = np.asarray(u, np.int64)
    v = np.asarray(v, np.int64)
    s = np.einsum("kf,kf->k", z[u], z[v])
    y = (np.arange(u.size) < n_pos).astype(np.float64)
    loss = float(np.mean(_softplus(s) - y * s))
    g = loss_scale * (_sigmoid(s) - y) / u.size
    return loss, s, g


def pair_backward(n, Z, u, v, g):
    """dZ of sum_k g_k s_k with s_k = <Z[u_k], Z[v_k]>: row r collects
    g_k Z[v_k] for every pair with u_k = r and g_k Z[u_k] for every pair
    with v_k = r.  Rows in no pair are 0."""
    z = np.asarray(Z, np.float64)
    u = np.asarray(u, np.int64)
    v = np.asarray(v, np.int64)
    g = np.asarray(g, np.float64)
    dz = np.zeros((n, z.shape[1]))
    np.add.at(dz, u, g[:, None] * z[v])
    np.add.at(dz, v, g[:, None] * z[u])
    return dz


def auc_ap(scores_pos, scores_neg):
    """Link-prediction metrics from the scores of positive and negative
    pairs, by their definitions (brute force over all pairs of scores):
    AUC = P(score of a random positive > score of a random negative), ties
    counting 1/2; AP = mean over positives i of the precision among all
    pairs scoring >= s_i."""
    sp = np.asarray(scores_pos, np.float64)
    sn = np.asarray(scores_neg, np.float64)
    gt = (sp[:, None] > sn[None, :]).sum()
    eq = (sp[:, None] == sn[None, :]).sum()
    auc = (gt + 0.5 * eq) / (sp.size * sn.size)
    pos_ge = (sp[None, :] >= sp[:, None]).sum(axis=1)
    all_ge = pos_ge + (sn[None, :] >= sp[:, None]).sum(axis=1)
    ap = float(np.mean(pos_ge / all_ge))
    return float(auc), ap
