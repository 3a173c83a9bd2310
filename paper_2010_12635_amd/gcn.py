"""Python binding of libgcn (ctypes).

Argument marshalling only: every computation runs in the HIP kernels of
``libgcn.so``.  PyTorch supplies device memory (tensors) and the stream.
The functions keep the C names (``gcn_normalize``, ``gcn_layer_fwd`` ...)
and take torch tensors where the C call takes device pointers.  If the
library is missing, loading fails with an error: there is no fallback.
"""
from __future__ import annotations

import ctypes
import os

import torch

__all__ = [
    "GCN_F32", "GCN_F16", "GCN_BF16", "GCN_I32", "GCN_I64", "GCN_CSR", "GCN_DENSE",
    "GCN_ACT_NONE", "GCN_ACT_RELU", "GCN_DENSE_TILED", "gcn_dense_tiled_elems", "gcn_densify", "GcnError", "GcnAdj", "GcnLayer", "GcnScaler",
    "GcnAdamConfig", "lib", "LIB_PATH", "EXPORTED", "torch_dtype",
    "gcn_status_string", "gcn_abi_version", "gcn_normalize_workspace_size", "gcn_normalize",
    "gcn_schedule_size", "gcn_schedule", "gcn_layer_workspace_size", "gcn_layer_fwd",
    "gcn_layer_bwd", "gcn_layer_bwd_noalloc", "gcn_loss_workspace_size", "gcn_loss", "gcn_optimizer_step",
    "gcn_transform_workspace_size", "gcn_transform", "gcn_aggregate_workspace_size", "gcn_aggregate",
    "gcn_sample_pairs", "gcn_pair_loss_workspace_size", "gcn_pair_loss", "gcn_pair_backward_workspace_size",
    "gcn_pair_backward", "gcn_pair_metrics_workspace_size", "gcn_pair_metrics",
]

GCN_F32, GCN_F16, GCN_BF16 = 0, 1, 2
GCN_I32, GCN_I64 = 0, 1
GCN_CSR, GCN_DENSE, GCN_DENSE_TILED = 0, 1, 2
GCN_ACT_NONE, GCN_ACT_RELU = 0, 1

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libgcn.so")

# every symbol declared in include/gcn.h
EXPORTED = (
    "gcn_status_string", "gcn_abi_version", "gcn_normalize_workspace_size", "gcn_normalize",
    "gcn_schedule_size", "gcn_schedule", "gcn_layer_workspace_size", "gcn_layer_fwd",
    "gcn_layer_bwd", "gcn_layer_bwd_noalloc", "gcn_loss_workspace_size", "gcn_loss", "gcn_optimizer_step",
    "gcn_transform_workspace_size", "gcn_transform", "gcn_aggregate_workspace_size", "gcn_aggregate",
    "gcn_dense_tiled_elems", "gcn_densify",
    "gcn_sample_pairs", "gcn_pair_loss_workspace_size", "gcn_pair_loss", "gcn_pair_backward_workspace_size",
    "gcn_pair_backward", "gcn_pair_metrics_workspace_size", "gcn_pair_metrics",
    "gcn_cast", "gcn_optimizer_step_half",
)

_DTYPES = {GCN_F32: torch.float32, GCN_F16: torch.float16, GCN_BF16: torch.bfloat16}


def torch_dtype(prec: int) -> torch.dtype:
    return _DTYPES[prec]


class GcnError(RuntimeError):
    def __init__(self, status: int, where: str):
        super().__init__(f"{where}: {gcn_status_string(status)}")
        self.status = status


class GcnAdj(ctypes.Structure):
    _fields_ = [
        ("n", ctypes.c_int64), ("nnz", ctypes.c_int64),
        ("format", ctypes.c_int32), ("index", ctypes.c_int32),
        ("value_prec", ctypes.c_int32), ("reserved0", ctypes.c_int32),
        ("rowptr", ctypes.c_void_p), ("colidx", ctypes.c_void_p), ("values", ctypes.c_void_p),
        ("dinv", ctypes.c_void_p), ("dense", ctypes.c_void_p), ("ld_dense", ctypes.c_int64),
        ("heavy_threshold", ctypes.c_int64), ("chunk_nnz", ctypes.c_int64),
        ("n_heavy", ctypes.c_int64), ("n_chunks", ctypes.c_int64),
        ("heavy_rows", ctypes.c_void_p), ("heavy_chunk_off", ctypes.c_void_p),
        ("chunk_heavy", ctypes.c_void_p), ("n_light", ctypes.c_int64), ("row_perm", ctypes.c_void_p),
        ("chunk_order", ctypes.c_void_p), ("chunk_beg", ctypes.c_void_p), ("part_off", ctypes.c_void_p),
        ("col_parts", ctypes.c_int64), ("part_slots", ctypes.c_int64),
        ("piece_desc", ctypes.c_void_p), ("piece_pos", ctypes.c_void_p), ("row_desc", ctypes.c_void_p),
        ("n_light_single", ctypes.c_int64),
        ("n_fix", ctypes.c_int64), ("n_fix_big", ctypes.c_int64), ("fix_rows", ctypes.c_void_p),
    ]


class GcnLayer(ctypes.Structure):
    _fields_ = [
        ("f_in", ctypes.c_int64), ("f_out", ctypes.c_int64),
        ("ld_in", ctypes.c_int64), ("ld_out", ctypes.c_int64),
        ("act", ctypes.c_int32), ("dropout_p", ctypes.c_float),
        ("layer_id", ctypes.c_int32), ("identity_input", ctypes.c_int32),
        ("epoch_from", ctypes.c_void_p),
    ]


class GcnScaler(ctypes.Structure):
    _fields_ = [("scale", ctypes.c_float), ("good_steps", ctypes.c_int32),
                ("step", ctypes.c_int32), ("skipped", ctypes.c_int32)]


class GcnAdamConfig(ctypes.Structure):
    _fields_ = [("lr", ctypes.c_float), ("beta1", ctypes.c_float), ("beta2", ctypes.c_float),
                ("eps", ctypes.c_float), ("backoff", ctypes.c_float), ("growth", ctypes.c_float),
                ("interval", ctypes.c_int32), ("min_scale", ctypes.c_float),
                ("max_scale", ctypes.c_float)]


ABI_VERSION = 11          # GCN_ABI_VERSION of the structs and signatures here
FIX_BIG_PIECES = 32       # GCN_FIX_BIG_PIECES

_lib = None


def lib():
    """Load libgcn.so (built in-tree by ``__graft_entry__.build()``)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"libgcn.so not found at {LIB_PATH}: build it first "
                           "(python -c 'import __graft_entry__ as g; g.build()')")
    L = ctypes.CDLL(LIB_PATH)
    P, I64, I32, SZ = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_size_t
    PSZ = ctypes.POINTER(ctypes.c_size_t)
    PI64 = ctypes.POINTER(ctypes.c_int64)
    PADJ = ctypes.POINTER(GcnAdj)
    PLAY = ctypes.POINTER(GcnLayer)
    sig = {
        "gcn_status_string": (ctypes.c_char_p, [I32]),
        "gcn_abi_version": (I32, []),
        "gcn_normalize_workspace_size": (I32, [I64, I64, PSZ]),
        "gcn_normalize": (I32, [I64, I64, P, P, I32, P, P, I64, P, P, I32, P, P, I64, PI64, P, SZ, P]),
        "gcn_schedule_size": (I32, [I64, I64, I64, I64, I64, PSZ]),
        "gcn_schedule": (I32, [PADJ, I64, I64, I64, P, SZ, P]),
        "gcn_layer_workspace_size": (I32, [PADJ, PLAY, I32, PSZ]),
        "gcn_layer_fwd": (I32, [PADJ, PLAY, I32, I32, P, P, P, ctypes.c_uint64, ctypes.c_uint64,
                                P, P, P, P, SZ, P]),
        "gcn_layer_bwd": (I32, [PADJ, PLAY, I32, P, P, P, I32, ctypes.c_float, P, P, P, P, P, P, P,
                                SZ, P]),
        "gcn_layer_bwd_noalloc": (I32, [PADJ, PLAY, I32, P, P, P, I32, ctypes.c_float, P, P, P, P, P, P, P]),
        "gcn_loss_workspace_size": (I32, [I64, I64, PSZ]),
        "gcn_loss": (I32, [I64, I64, I64, I32, P, P, P, I64, P, P, P, P, P, P, P, SZ, P]),
        "gcn_optimizer_step": (I32, [I64, P, P, P, P, P, I32, ctypes.POINTER(GcnAdamConfig), P, P, P]),
        "gcn_transform_workspace_size": (I32, [I64, I64, I64, I32, PSZ]),
        "gcn_transform": (I32, [I64, I64, I64, I32, P, I64, P, I64, P, I64, P, P, SZ, P]),
        "gcn_aggregate_workspace_size": (I32, [PADJ, I64, I32, PSZ]),
        "gcn_dense_tiled_elems": (I32, [I64, I32, PI64]),
        "gcn_densify": (I32, [PADJ, I32, I32, P, I64, P]),
        "gcn_aggregate": (I32, [PADJ, I64, I32, P, I64, P, I32, ctypes.c_float, I32, ctypes.c_uint64, I32,
                                ctypes.c_uint64, P, I64, P, P, SZ, P]),
        "gcn_sample_pairs": (I32, [I64, P, P, I64, I64, I64, ctypes.c_uint64, ctypes.c_uint64, P, P, P]),
        "gcn_pair_loss_workspace_size": (I32, [I64, PSZ]),
        "gcn_pair_loss": (I32, [I64, I64, I64, I32, P, P, P, I64, I64, P, P, P, P, P, P, SZ, P]),
        "gcn_pair_backward_workspace_size": (I32, [I64, I64, I64, PSZ]),
        "gcn_pair_backward": (I32, [I64, I64, I64, I32, P, P, P, I64, P, P, I64, P, P, SZ, P]),
        "gcn_pair_metrics_workspace_size": (I32, [I64, I64, PSZ]),
        "gcn_pair_metrics": (I32, [P, I64, I64, P, P, SZ, P]),
        "gcn_cast": (I32, [I64, I64, I32, P, I64, I32, P, I64, P, P]),
        "gcn_optimizer_step_half": (I32, [I64, P, P, P, P, P, I32, ctypes.POINTER(GcnAdamConfig), P, P, P]),
    }
    for name, (res, args) in sig.items():
        f = getattr(L, name)
        f.restype = res
        f.argtypes = args
    if L.gcn_abi_version() != ABI_VERSION:
        raise RuntimeError(f"{LIB_PATH} has ABI version {L.gcn_abi_version()}, this binding expects "
                           f"{ABI_VERSION}: rebuild it")
    _lib = L
    return L


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream=None):
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


def _check(status, where):
    if status != 0:
        raise GcnError(status, where)


def gcn_status_string(status: int) -> str:
    return lib().gcn_status_string(status).decode()


def gcn_abi_version() -> int:
    return lib().gcn_abi_version()


def gcn_normalize_workspace_size(n: int, num_edges: int) -> int:
    b = ctypes.c_size_t(0)
    _check(lib().gcn_normalize_workspace_size(n, num_edges, ctypes.byref(b)), "gcn_normalize_workspace_size")
    return b.value


def gcn_normalize(n, src, dst, index, rowptr, colidx, deg, dinv, value_prec, values, dense, ld_dense,
                  workspace, stream=None) -> int:
    """Returns nnz.  Tensors are device tensors (see include/gcn.h)."""
    nnz = ctypes.c_int64(0)
    ne = 0 if src is None else src.numel()
    st = lib().gcn_normalize(n, ne, _ptr(src), _ptr(dst), index, _ptr(rowptr), _ptr(colidx), colidx.numel(),
                             _ptr(deg), _ptr(dinv), value_prec, _ptr(values), _ptr(dense), ld_dense,
                             ctypes.byref(nnz), _ptr(workspace), workspace.numel() * workspace.element_size(),
                             _stream(stream))
    _check(st, "gcn_normalize")
    return nnz.value


def gcn_schedule_size(n, nnz, heavy_threshold=0, chunk_nnz=0, col_parts=0) -> int:
    b = ctypes.c_size_t(0)
    _check(lib().gcn_schedule_size(n, nnz, heavy_threshold, chunk_nnz, col_parts, ctypes.byref(b)),
           "gcn_schedule_size")
    return b.value


def gcn_schedule(adj: GcnAdj, sched, heavy_threshold=0, chunk_nnz=0, col_parts=0, stream=None):
    st = lib().gcn_schedule(ctypes.byref(adj), heavy_threshold, chunk_nnz, col_parts, _ptr(sched),
                            sched.numel() * sched.element_size(), _stream(stream))
    _check(st, "gcn_schedule")


def gcn_layer_workspace_size(adj: GcnAdj, layer: GcnLayer, prec: int) -> int:
    b = ctypes.c_size_t(0)
    _check(lib().gcn_layer_workspace_size(ctypes.byref(adj), ctypes.byref(layer), prec, ctypes.byref(b)),
           "gcn_layer_workspace_size")
    return b.value


def gcn_layer_fwd(adj, layer, prec, training, H, W, bias, seed, epoch, S, H_out, overflow, workspace,
                  stream=None):
    st = lib().gcn_layer_fwd(ctypes.byref(adj), ctypes.byref(layer), prec, int(training), _ptr(H), _ptr(W),
                             _ptr(bias), seed & 0xFFFFFFFFFFFFFFFF, epoch, _ptr(S), _ptr(H_out), _ptr(overflow),
                             _ptr(workspace), workspace.numel() * workspace.element_size(), _stream(stream))
    _check(st, "gcn_layer_fwd")


def gcn_layer_bwd(adj, layer, prec, H, W, dZ, act_below, p_below, dW, dbias, dZ_below, GS, overflow,
                  workspace, stream=None, dbias_below=None):
    st = lib().gcn_layer_bwd(ctypes.byref(adj), ctypes.byref(layer), prec, _ptr(H), _ptr(W), _ptr(dZ),
                             act_below, p_below, _ptr(dW), _ptr(dbias), _ptr(dZ_below), _ptr(dbias_below),
                             _ptr(GS), _ptr(overflow), _ptr(workspace), workspace.numel() * workspace.element_size(),
                             _stream(stream))
    _check(st, "gcn_layer_bwd")


NOALLOC_SCRATCH_BYTES = 64 << 20    # GCN_NOALLOC_SCRATCH_BYTES


def gcn_layer_bwd_noalloc(adj, layer, prec, H, W, dZ, act_below, p_below, dW, dbias, dZ_below, GS, overflow,
                          stream=None, dbias_below=None):
    st = lib().gcn_layer_bwd_noalloc(ctypes.byref(adj), ctypes.byref(layer), prec, _ptr(H), _ptr(W), _ptr(dZ),
                                     act_below, p_below, _ptr(dW), _ptr(dbias), _ptr(dZ_below),
                                     _ptr(dbias_below), _ptr(GS), _ptr(overflow), _stream(stream))
    _check(st, "gcn_layer_bwd_noalloc")


def gcn_loss_workspace_size(n, C) -> int:
    b = ctypes.c_size_t(0)
    _check(lib().gcn_loss_workspace_size(n, C, ctypes.byref(b)), "gcn_loss_workspace_size")
    return b.value


def gcn_loss(n, C, ld, prec, logits, labels, mask, n_mask, loss_scale, loss, dlogits, n_correct, overflow,
             workspace, stream=None, dlogits_colsum=None):
    st = lib().gcn_loss(n, C, ld, prec, _ptr(logits), _ptr(labels), _ptr(mask), n_mask, _ptr(loss_scale),
                        _ptr(loss), _ptr(dlogits), _ptr(dlogits_colsum), _ptr(n_correct), _ptr(overflow),
                        _ptr(workspace), workspace.numel() * workspace.element_size(), _stream(stream))
    _check(st, "gcn_loss")


def gcn_optimizer_step(count, master, grad, m, v, working, prec, cfg: GcnAdamConfig, state, overflow,
                       stream=None):
    st = lib().gcn_optimizer_step(count, _ptr(master), _ptr(grad), _ptr(m), _ptr(v), _ptr(working), prec,
                                  ctypes.byref(cfg), _ptr(state), _ptr(overflow), _stream(stream))
    _check(st, "gcn_optimizer_step")


def gcn_optimizer_step_half(count, w, grad, m, v, widened, prec, cfg: GcnAdamConfig, state, overflow,
                            stream=None):
    st = lib().gcn_optimizer_step_half(count, _ptr(w), _ptr(grad), _ptr(m), _ptr(v), _ptr(widened), prec,
                                       ctypes.byref(cfg), _ptr(state), _ptr(overflow), _stream(stream))
    _check(st, "gcn_optimizer_step_half")


def gcn_cast(rows, cols, src_prec, src, ld_src, dst_prec, dst, ld_dst, overflow=None, stream=None):
    st = lib().gcn_cast(rows, cols, src_prec, _ptr(src), ld_src, dst_prec, _ptr(dst), ld_dst, _ptr(overflow),
                        _stream(stream))
    _check(st, "gcn_cast")


def gcn_transform_workspace_size(n, f_in, f_out, prec) -> int:
    b = ctypes.c_size_t(0)
    _check(lib().gcn_transform_workspace_size(n, f_in, f_out, prec, ctypes.byref(b)), "gcn_transform_workspace_size")
    return b.value


def gcn_transform(n, f_in, f_out, prec, H, ld_in, W, ld_w, S, ld_s, overflow, workspace, stream=None):
    st = lib().gcn_transform(n, f_in, f_out, prec, _ptr(H), ld_in, _ptr(W), ld_w, _ptr(S), ld_s, _ptr(overflow),
                             _ptr(workspace), 0 if workspace is None else workspace.numel() * workspace.element_size(),
                             _stream(stream))
    _check(st, "gcn_transform")


def gcn_aggregate_workspace_size(adj, F, prec) -> int:
    b = ctypes.c_size_t(0)
    _check(lib().gcn_aggregate_workspace_size(ctypes.byref(adj), F, prec, ctypes.byref(b)),
           "gcn_aggregate_workspace_size")
    return b.value


def gcn_aggregate(adj, F, prec, X, ldx, bias, act, dropout_p, training, seed, layer_id, epoch, Y, ldy, overflow,
                  workspace, stream=None):
    st = lib().gcn_aggregate(ctypes.byref(adj), F, prec, _ptr(X), ldx, _ptr(bias), act, dropout_p, int(training),
                             seed & 0xFFFFFFFFFFFFFFFF, layer_id, epoch, _ptr(Y), ldy, _ptr(overflow),
                             _ptr(workspace), 0 if workspace is None else workspace.numel() * workspace.element_size(),
                             _stream(stream))
    _check(st, "gcn_aggregate")


def gcn_dense_tiled_elems(n, prec) -> int:
    e = ctypes.c_int64(0)
    _check(lib().gcn_dense_tiled_elems(n, prec, ctypes.byref(e)), "gcn_dense_tiled_elems")
    return e.value


def gcn_densify(adj, fmt, value_prec, dense, ld_dense, stream=None):
    _check(lib().gcn_densify(ctypes.byref(adj), fmt, value_prec, _ptr(dense), ld_dense, _stream(stream)),
           "gcn_densify")


# ------------------------------------------------------- link prediction ----

def gcn_sample_pairs(n, edge_u, edge_v, n_pos, n_neg, seed, epoch, pair_u, pair_v, stream=None):
    n_edges = 0 if edge_u is None else edge_u.numel()
    _check(lib().gcn_sample_pairs(n, _ptr(edge_u), _ptr(edge_v), n_edges, n_pos, n_neg,
                                  seed & 0xFFFFFFFFFFFFFFFF, epoch, _ptr(pair_u), _ptr(pair_v), _stream(stream)),
           "gcn_sample_pairs")


def gcn_pair_loss_workspace_size(n_pairs) -> int:
    b = ctypes.c_size_t(0)
    _check(lib().gcn_pair_loss_workspace_size(n_pairs, ctypes.byref(b)), "gcn_pair_loss_workspace_size")
    return b.value


def gcn_pair_loss(n, F, ld, prec, Z, pair_u, pair_v, n_pos, n_neg, loss_scale, loss, scores, g, overflow,
                  workspace, stream=None):
    st = lib().gcn_pair_loss(n, F, ld, prec, _ptr(Z), _ptr(pair_u), _ptr(pair_v), n_pos, n_neg, _ptr(loss_scale),
                             _ptr(loss), _ptr(scores), _ptr(g), _ptr(overflow), _ptr(workspace),
                             workspace.numel() * workspace.element_size(), _stream(stream))
    _check(st, "gcn_pair_loss")


def gcn_pair_backward_workspace_size(n, n_pairs, F) -> int:
    b = ctypes.c_size_t(0)
    _check(lib().gcn_pair_backward_workspace_size(n, n_pairs, F, ctypes.byref(b)), "gcn_pair_backward_workspace_size")
    return b.value


def gcn_pair_backward(n, F, ld, prec, Z, pair_u, pair_v, n_pairs, g, dZ, ldz, overflow, workspace, stream=None):
    st = lib().gcn_pair_backward(n, F, ld, prec, _ptr(Z), _ptr(pair_u), _ptr(pair_v), n_pairs, _ptr(g), _ptr(dZ),
                                 ldz, _ptr(overflow), _ptr(workspace), workspace.numel() * workspace.element_size(),
                                 _stream(stream))
    _check(st, "gcn_pair_backward")


def gcn_pair_metrics_workspace_size(n_pos, n_neg) -> int:
    b = ctypes.c_size_t(0)
    _check(lib().gcn_pair_metrics_workspace_size(n_pos, n_neg, ctypes.byref(b)), "gcn_pair_metrics_workspace_size")
    return b.value


def gcn_pair_metrics(scores, n_pos, n_neg, auc_ap, workspace, stream=None):
    st = lib().gcn_pair_metrics(_ptr(scores), n_pos, n_neg, _ptr(auc_ap), _ptr(workspace),
                                workspace.numel() * workspace.element_size(), _stream(stream))
    _check(st, "gcn_pair_metrics")
