"""Seeded synthetic inputs for the GCN workloads.

This module only *draws* inputs: raw edge lists, feature matrices, labels,
train masks and initial weights.  It holds none of the method's arithmetic
(no self-loop handling, no symmetrisation, no normalisation, no layer math),
so that the CPU oracle and the HIP path can both be fed from it without
sharing any computation.

Every generator takes a ``numpy.random.Generator``; ``workload()`` spawns one
independent stream per input kind from ``SeedSequence(seed)``.

Graph models (the paper's run-time study uses Barabasi-Albert graphs,
Section "Datasets"; the other models stand in for the shapes of the
workloads this library is measured on):

* ``er_graph``    Erdos-Renyi G(n, M): M distinct undirected edges, no self-loops.
* ``sbm_graph``   stochastic block model, contiguous equal blocks, one
                  independent Bernoulli draw per unordered vertex pair.
* ``ba_graph``    Barabasi-Albert preferential attachment: m isolated seed
                  vertices, the first new vertex links to all of them, every
                  later vertex to m distinct earlier vertices drawn with
                  probability proportional to degree; m*(n-m) edges.
* ``rmat_graph``  R-MAT recursive quadrant sampling, edge_factor*n samples,
                  then a random relabelling of the vertices.  Samples may
                  repeat and may be self-loops: the adjacency normalisation
                  removes both.
"""
from __future__ import annotations

from dataclasses import dataclass, field
import numpy as np

__all__ = [
    "er_graph", "sbm_graph", "ba_graph", "rmat_graph", "rmat_graph_device", "scale_workload_device",
    "link_split", "gae_workload",
    "features", "uniform_labels", "train_mask", "glorot_uniform",
    "WorkloadSpec", "SPECS", "workload",
]


def _decode_upper_pairs(idx: np.ndarray, s: int):
    """Map linear indices of the strict upper triangle of an s x s matrix
    (row-major over pairs (i, j), i < j) back to (i, j)."""
    idx = idx.astype(np.int64)
    # row i holds s-1-i pairs; first index of row i is i*(2s-i-1)/2
    i = np.floor(((2 * s - 1) - np.sqrt((2 * s - 1) ** 2 - 8.0 * idx)) / 2).astype(np.int64)
    first = i * (2 * s - i - 1) // 2
    # guard against floating error at row boundaries
    over = idx < first
    i[over] -= 1
    first = i * (2 * s - i - 1) // 2
    nxt = (i + 1) * (2 * s - i - 2) // 2
    under = idx >= nxt
    i[under] += 1
    first = i * (2 * s - i - 1) // 2
    j = idx - first + i + 1
    return i, j


def er_graph(n: int, m_edges: int, rng: np.random.Generator):
    """G(n, M): ``m_edges`` distinct unordered pairs {u, v}, u != v, uniformly
    at random.  Returns (src, dst) int32, one entry per undirected edge."""
    npairs = n * (n - 1) // 2
    if m_edges > npairs:
        raise ValueError("more edges than vertex pairs")
    idx = rng.choice(npairs, size=m_edges, replace=False)
    i, j = _decode_upper_pairs(idx, n)
    return i.astype(np.int32), j.astype(np.int32)


def sbm_graph(n: int, blocks: int, p_in: float, p_out: float, rng: np.random.Generator):
    """Stochastic block model with contiguous equal blocks (block(v) = v // (n/blocks)).
    Each unordered pair is an edge independently with probability p_in (same
    block) or p_out (different blocks); drawn per block pair as a binomial
    count followed by a uniform choice of that many distinct pairs, which has
    the same distribution.  Returns (src, dst) int32 and the block id of every
    vertex."""
    if n % blocks:
        raise ValueError("n must be a multiple of the number of blocks")
    s = n // blocks
    srcs, dsts = [], []
    for bi in range(blocks):
        for bj in range(bi, blocks):
            if bi == bj:
                npairs = s * (s - 1) // 2
                k = rng.binomial(npairs, p_in)
                idx = rng.choice(npairs, size=k, replace=False)
                i, j = _decode_upper_pairs(idx, s)
                srcs.append(bi * s + i)
                dsts.append(bi * s + j)
            else:
                npairs = s * s
                k = rng.binomial(npairs, p_out)
                idx = rng.choice(npairs, size=k, replace=False)
                srcs.append(bi * s + idx // s)
                dsts.append(bj * s + idx % s)
    src = np.concatenate(srcs).astype(np.int32)
    dst = np.concatenate(dsts).astype(np.int32)
    block = (np.arange(n) // s).astype(np.int32)
    return src, dst, block


def ba_graph(n: int, m: int, rng: np.random.Generator):
    """Barabasi-Albert preferential attachment (Barabasi & Albert 1999), the
    paper's synthetic run-time graphs.  Returns (src, dst) int32 with
    m*(n-m) undirected edges."""
    if not (1 <= m < n):
        raise ValueError("need 1 <= m < n")
    n_edges = m * (n - m)
    src = np.empty(n_edges, np.int32)
    dst = np.empty(n_edges, np.int32)
    # every endpoint of every edge so far: sampling uniformly from it is
    # sampling proportionally to degree
    pool = np.empty(2 * n_edges, np.int32)
    pool_len = 0
    targets = np.arange(m, dtype=np.int32)
    e = 0
    for v in range(m, n):
        src[e:e + m] = v
        dst[e:e + m] = targets
        e += m
        pool[pool_len:pool_len + m] = targets
        pool[pool_len + m:pool_len + 2 * m] = v
        pool_len += 2 * m
        if v + 1 == n:
            break
        chosen: list[int] = []
        seen = set()
        while len(chosen) < m:
            draws = pool[rng.integers(0, pool_len, size=2 * m)]
            for t in draws.tolist():
                if t not in seen:
                    seen.add(t)
                    chosen.append(t)
                    if len(chosen) == m:
                        break
        targets = np.asarray(chosen, dtype=np.int32)
    return src, dst


def rmat_graph(scale: int, edge_factor: int, a: float, b: float, c: float,
               rng: np.random.Generator):
    """R-MAT (Chakrabarti et al. 2004): edge_factor * 2^scale samples, each
    choosing one quadrant per bit level with probabilities (a, b, c, d), then
    a uniform random relabelling of the 2^scale vertices.  Raw samples are
    returned: repeats and self-loops included."""
    n = 1 << scale
    n_samples = edge_factor * n
    src = np.zeros(n_samples, np.int64)
    dst = np.zeros(n_samples, np.int64)
    ab = a + b
    abc = a + b + c
    chunk = 1 << 22
    for lo in range(0, n_samples, chunk):
        hi = min(lo + chunk, n_samples)
        s = np.zeros(hi - lo, np.int64)
        d = np.zeros(hi - lo, np.int64)
        for bit in range(scale):
            r = rng.random(hi - lo)
            down = r >= ab                       # quadrant c or d: row bit set
            right = ((r >= a) & (r < ab)) | (r >= abc)   # quadrant b or d: column bit set
            s |= down.astype(np.int64) << bit
            d |= right.astype(np.int64) << bit
        src[lo:hi] = s
        dst[lo:hi] = d
    perm = rng.permutation(n)
    return perm[src].astype(np.int32), perm[dst].astype(np.int32)


def rmat_graph_device(scale: int, edge_factor: int, a: float, b: float, c: float, seed: int,
                      device="cuda", chunk: int = 1 << 27):
    """The R-MAT recipe of rmat_graph drawn on the device with torch's
    generator (seeded by ``seed``), for graphs too large to draw on the host:
    per sample and bit level one uniform draw picks the quadrant, then a
    uniform random relabelling.  Returns int32 device tensors (raw samples,
    repeats and self-loops included).  Not the same stream as rmat_graph."""
    import torch
    n = 1 << scale
    n_samples = edge_factor * n
    gen = torch.Generator(device=device)
    gen.manual_seed(int(seed))
    src = torch.empty(n_samples, dtype=torch.int32, device=device)
    dst = torch.empty(n_samples, dtype=torch.int32, device=device)
    ab, abc = a + b, a + b + c
    for lo in range(0, n_samples, chunk):
        hi = min(lo + chunk, n_samples)
        s = torch.zeros(hi - lo, dtype=torch.int32, device=device)
        d = torch.zeros(hi - lo, dtype=torch.int32, device=device)
        for bit in range(scale):
            r = torch.rand(hi - lo, generator=gen, device=device)
            s |= (r >= ab).to(torch.int32) << bit
            d |= (((r >= a) & (r < ab)) | (r >= abc)).to(torch.int32) << bit
            del r
        src[lo:hi] = s
        dst[lo:hi] = d
        del s, d
    perm = torch.randperm(n, generator=gen, device=device, dtype=torch.int32)
    for lo in range(0, n_samples, chunk):
        hi = min(lo + chunk, n_samples)
        src[lo:hi] = perm[src[lo:hi].long()]
        dst[lo:hi] = perm[dst[lo:hi].long()]
    del perm
    return src, dst


def scale_workload_device(scale: int, seed: int, f_in: int = 128, hidden: int = 128, classes: int = 64,
                          dtype=None, device="cuda"):
    """The scale-test workload (R-MAT scale ``scale``, edge factor 16,
    (0.57, 0.19, 0.19, 0.05); features N(0,1); uniform labels over
    ``classes``; every vertex in the training mask; Glorot-uniform weights)
    with the graph, features and labels drawn on the device.  X is returned
    as n x round8(f_in) in ``dtype`` with zero padding columns."""
    import torch
    dtype = dtype or torch.float16
    src, dst = rmat_graph_device(scale, 16, 0.57, 0.19, 0.19, seed, device)
    n = 1 << scale
    gen = torch.Generator(device=device)
    gen.manual_seed(int(seed) + 1)
    ld = (f_in + 7) // 8 * 8
    X = torch.zeros((n, ld), dtype=dtype, device=device)
    step = 1 << 22
    for lo in range(0, n, step):
        hi = min(lo + step, n)
        X[lo:hi, :f_in] = torch.randn((hi - lo, f_in), generator=gen, device=device).to(dtype)
    labels = torch.randint(0, classes, (n,), generator=gen, device=device, dtype=torch.int32)
    mask = torch.ones(n, dtype=torch.uint8, device=device)
    w_rng = np.random.default_rng(seed)
    W1 = glorot_uniform(f_in, hidden, w_rng)
    W2 = glorot_uniform(hidden, classes, w_rng)
    return dict(n=n, src=src, dst=dst, X=X, labels=labels, mask=mask, W1=W1, W2=W2,
                b1=np.zeros(hidden, np.float32), b2=np.zeros(classes, np.float32),
                dropout_seed=int(seed) * 7919 + 1)


def features(n: int, f: int, kind: str, rng: np.random.Generator, density: float = 1.0):
    """Feature matrix (float32).  kind 'normal': N(0,1); kind 'uniform':
    U[0,1) kept with probability ``density`` (rest exactly 0)."""
    if kind == "normal":
        x = rng.standard_normal((n, f), dtype=np.float32)
    elif kind == "uniform":
        x = rng.random((n, f), dtype=np.float32)
        if density < 1.0:
            x *= (rng.random((n, f)) < density)
    else:
        raise ValueError(kind)
    return x


def uniform_labels(n: int, classes: int, rng: np.random.Generator):
    return rng.integers(0, classes, size=n, dtype=np.int64).astype(np.int32)


def train_mask(n: int, k: int | None, rng: np.random.Generator):
    """uint8 mask with k vertices chosen without replacement (all if k is None)."""
    m = np.zeros(n, np.uint8)
    if k is None:
        m[:] = 1
    else:
        m[rng.choice(n, size=k, replace=False)] = 1
    return m


def glorot_uniform(fan_in: int, fan_out: int, rng: np.random.Generator):
    """Glorot & Bengio uniform init, U(-a, a) with a = sqrt(6 / (fan_in + fan_out))."""
    a = np.sqrt(6.0 / (fan_in + fan_out))
    return rng.uniform(-a, a, size=(fan_in, fan_out)).astype(np.float32)


@dataclass(frozen=True)
class WorkloadSpec:
    """One synthetic workload: graph recipe, layer widths and training recipe."""
    name: str
    graph: str
    graph_args: tuple
    f_in: int
    hidden: int
    classes: int
    feat_kind: str = "normal"
    feat_density: float = 1.0
    labels: str = "uniform"          # 'uniform' or 'block'
    mask_k: int | None = None        # None: every vertex is in the train mask
    dropout: float = 0.5
    epochs: int = 1
    dense_adj: bool = False
    index64: bool = False
    lr: float = 0.01
    loss_scale0: float = 65536.0
    extra: dict = field(default_factory=dict)


SPECS = {
    # tiny 2-layer vertex classification, Cora-like shape (7 classes, 140 labels)
    "er2k": WorkloadSpec("er2k", "er", (2048, 8192), 512, 16, 7, "uniform", 0.01,
                         mask_k=140, epochs=1),
    # dense-adjacency 2-layer GCN on a 32-block SBM
    "sbm16k_dense": WorkloadSpec("sbm16k_dense", "sbm", (16384, 32, 0.01, 0.0002), 500, 64, 32,
                                 labels="block", epochs=200, dense_adj=True),
    # sparse 2-layer GCN on a Barabasi-Albert graph
    "ba200k": WorkloadSpec("ba200k", "ba", (200000, 8), 128, 128, 40, epochs=100),
    # GAE encoder shape on an R-MAT graph (scale 17)
    "rmat17": WorkloadSpec("rmat17", "rmat", (17, 16, 0.57, 0.19, 0.19), 256, 256, 64,
                           epochs=100),
    # scale test on an R-MAT graph (scale 21), 64-bit row pointers
    "rmat21": WorkloadSpec("rmat21", "rmat", (21, 16, 0.57, 0.19, 0.19), 128, 128, 64,
                           epochs=20, index64=True),
}


def _graph(spec: WorkloadSpec, rng):
    if spec.graph == "er":
        n, m = spec.graph_args
        s, d = er_graph(n, m, rng)
        return n, s, d, None
    if spec.graph == "sbm":
        n, blocks, p_in, p_out = spec.graph_args
        s, d, block = sbm_graph(n, blocks, p_in, p_out, rng)
        return n, s, d, block
    if spec.graph == "ba":
        n, m = spec.graph_args
        s, d = ba_graph(n, m, rng)
        return n, s, d, None
    if spec.graph == "rmat":
        scale, ef, a, b, c = spec.graph_args
        s, d = rmat_graph(scale, ef, a, b, c, rng)
        return 1 << scale, s, d, None
    raise ValueError(spec.graph)


def workload(spec: WorkloadSpec | str, seed: int = 0, *, n_override: int | None = None):
    """Draw every input of a workload from ``SeedSequence(seed)``.

    Returns a dict: n, src, dst (raw undirected edge samples, int32),
    X (n x f_in float32), labels (int32), mask (uint8), W1, W2 (float32,
    Glorot-uniform), b1, b2 (zeros), dropout seed (uint64).
    ``n_override`` shrinks ER/BA/SBM/R-MAT graphs (keeping the recipe) for
    small parity cases."""
    if isinstance(spec, str):
        spec = SPECS[spec]
    if n_override is not None:
        spec = _shrunk(spec, n_override)
    ss = np.random.SeedSequence(seed)
    g_rng, x_rng, y_rng, m_rng, w_rng, d_rng = [np.random.default_rng(s) for s in ss.spawn(6)]
    n, src, dst, block = _graph(spec, g_rng)
    X = features(n, spec.f_in, spec.feat_kind, x_rng, spec.feat_density)
    if spec.labels == "block":
        labels = block.copy()
    else:
        labels = uniform_labels(n, spec.classes, y_rng)
    mask = train_mask(n, spec.mask_k if (spec.mask_k is None or spec.mask_k <= n) else None, m_rng)
    W1 = glorot_uniform(spec.f_in, spec.hidden, w_rng)
    W2 = glorot_uniform(spec.hidden, spec.classes, w_rng)
    dseed = int(d_rng.integers(0, 2**63 - 1, dtype=np.int64))
    return dict(spec=spec, n=n, src=src, dst=dst, X=X, labels=labels, mask=mask,
                W1=W1, W2=W2, b1=np.zeros(spec.hidden, np.float32),
                b2=np.zeros(spec.classes, np.float32), dropout_seed=dseed)


def table1_workload(n: int, model_size: int, seed: int = 0, classes: int = 16, m: int = 8):
    """One point of the paper's run-time sweep (Table 1): a Barabasi-Albert
    graph of n vertices (m edges per new vertex), featureless input X = I
    (returned as X = None), a 2-layer GCN n -> model_size -> classes,
    uniform labels on every vertex, Glorot-uniform weights."""
    ss = np.random.SeedSequence([seed, n, model_size])
    g_rng, y_rng, w_rng, d_rng = [np.random.default_rng(s) for s in ss.spawn(4)]
    src, dst = ba_graph(n, m, g_rng)
    labels = uniform_labels(n, classes, y_rng)
    spec = WorkloadSpec(f"table1_n{n}_d{model_size}", "ba", (n, m), n, model_size, classes, feat_kind="identity",
                        epochs=5, dense_adj=True)
    return dict(spec=spec, n=n, src=src, dst=dst, X=None, labels=labels, mask=np.ones(n, np.uint8),
                W1=glorot_uniform(n, model_size, w_rng), W2=glorot_uniform(model_size, classes, w_rng),
                b1=np.zeros(model_size, np.float32), b2=np.zeros(classes, np.float32),
                dropout_seed=int(d_rng.integers(0, 2**63 - 1, dtype=np.int64)))


def _shrunk(spec: WorkloadSpec, n: int) -> WorkloadSpec:
    from dataclasses import replace
    if spec.graph == "er":
        m = spec.graph_args[1] * n // spec.graph_args[0]
        return replace(spec, graph_args=(n, max(m, 1)))
    if spec.graph == "sbm":
        _, blocks, p_in, p_out = spec.graph_args
        blocks = min(blocks, max(1, n // 16))
        n = (n // blocks) * blocks
        scale_up = spec.graph_args[0] / n
        return replace(spec, graph_args=(n, blocks, min(1.0, p_in * scale_up), min(1.0, p_out * scale_up)))
    if spec.graph == "ba":
        return replace(spec, graph_args=(n, spec.graph_args[1]))
    if spec.graph == "rmat":
        scale = max(1, int(np.log2(n)))
        return replace(spec, graph_args=(scale,) + tuple(spec.graph_args[1:]))
    raise ValueError(spec.graph)


def link_split(n: int, src, dst, test_frac: float, rng: np.random.Generator):
    """Held-out split for link prediction: the distinct undirected edges
    (self-loops and repeats of the raw samples dropped) are shuffled, a
    ``test_frac`` share becomes the test positives and the rest the training
    edges; as many test negatives are drawn uniformly among vertex pairs
    that are not edges (distinct, u < v).  Returns (train_u, train_v,
    test_u, test_v, n_test_pos) with the test positives first."""
    src = np.asarray(src, np.int64)
    dst = np.asarray(dst, np.int64)
    keep = src != dst
    a, b = np.minimum(src[keep], dst[keep]), np.maximum(src[keep], dst[keep])
    key = np.unique(a * n + b)
    key = key[rng.permutation(key.size)]
    n_test = int(round(test_frac * key.size))
    test_pos, train = key[:n_test], key[n_test:]
    edges = np.sort(key)
    neg = np.empty(0, np.int64)
    while neg.size < n_test:
        m = 2 * (n_test - neg.size) + 16
        u = rng.integers(0, n, m)
        v = rng.integers(0, n, m)
        ok = u != v
        k = np.minimum(u, v)[ok] * n + np.maximum(u, v)[ok]
        pos = np.searchsorted(edges, k)
        is_edge = (pos < edges.size) & (edges[np.minimum(pos, edges.size - 1)] == k)
        k = k[~is_edge]
        neg = np.unique(np.concatenate([neg, k]))
    neg = neg[rng.permutation(neg.size)][:n_test]
    test = np.concatenate([test_pos, neg])
    return ((train // n).astype(np.int32), (train % n).astype(np.int32),
            (test // n).astype(np.int32), (test % n).astype(np.int32), n_test)


def gae_workload(seed: int = 0, *, n_override: int | None = None, test_frac: float = 0.1):
    """The link-prediction workload (graph auto-encoder): the R-MAT scale-17
    graph of SPECS["rmat17"] (edge factor 16), features 256 N(0,1), encoder
    256 -> 256 -> 64; 10 % of the distinct edges held out as test positives
    with as many non-edges as test negatives.  Adds train_u/train_v (the
    encoder's graph and the pool of training positives), test_u/test_v and
    n_test_pos to the workload dict."""
    wl = workload("rmat17", seed, n_override=n_override)
    rng = np.random.default_rng(np.random.SeedSequence(seed).spawn(7)[6])
    tu, tv, eu, ev, nt = link_split(wl["n"], wl["src"], wl["dst"], test_frac, rng)
    wl.update(train_u=tu, train_v=tv, test_u=eu, test_v=ev, n_test_pos=nt)
    return wl
