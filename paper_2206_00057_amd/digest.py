"""Thin Python binding of ``libdigest.so`` (the C ABI declared in include/digest.h).

Functions carry the C names.  They only marshal arguments: tensors become
device pointers (after dtype/device/size checks that keep every kernel
inside the buffers it is given), the stream defaults to torch's current
stream, and a negative status raises ``DigestError``.  All computation runs
in the HIP library; if it is not built, importing this module fails loudly.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
# DIGEST_LIBRARY names another build of the same ABI (e.g. the host-only
# sanitizer build); by default the in-tree libdigest.so.
LIB_PATH = os.environ.get("DIGEST_LIBRARY") or os.path.join(_PKG, "libdigest.so")

OK, EINVAL, ENOMEM, EHIP, ESTATE = 0, -1, -2, -3, -4
MODEL_GCN, MODEL_GAT = 0, 1
ACT_RELU, ACT_IDENTITY = 0, 1
PUSH_BOUNDARY, PUSH_ALL_OWNED = 0, 1
PULL_ROWS, PULL_AGGREGATE = 0, 1

_lib = None


class DigestError(RuntimeError):
    def __init__(self, status, message):
        super().__init__(f"digest status {status}: {message}")
        self.status = status


def lib():
    """Load libdigest.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run `python -m paper_2206_00057_amd.build` "
                               "(or __graft_entry__.build())")
        L = ctypes.CDLL(LIB_PATH)
        P, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
        st = ctypes.c_int
        sig = {
            "digest_last_error": ([], ctypes.c_char_p),
            "digest_partition_create": ([i64, P, P, P, P, i64, P, i64, i32, P, P], st),
            "digest_partition_destroy": ([P], None),
            "digest_partition_query": ([P, P, P, P, P], st),
            "digest_partition_bind_workspace": ([P, P, sz, P], st),
            "digest_partition_export_maps": ([P, P, P, P], st),
            "digest_partition_export_transpose": ([P, P, P, P], st),
            "digest_partition_read_halo": ([P, i32, P, P], st),
            "digest_pull": ([P, i32, P, P], st),
            "digest_partition_set_pull_mode": ([P, i32], st),
            "digest_push": ([P, i32, P, P, i32, P], st),
            "digest_layer_forward": ([P, i32, P, P, P, i32, P], st),
            "digest_layer_backward": ([P, i32, P, P, P, P, P, P, P], st),
            "digest_softmax_xent": ([P, P, P, P, P, P], st),
            "digest_softmax_xent_static": ([i64, i32, P, P, P, P, P], st),
            "digest_sgd_average": ([P, P, i32, i64, ctypes.c_float, P], st),
            "digest_halo_gradient": ([P, i32, P, P, P, P, P], st),
            "digest_layer_backward_halo": ([P, i32, P, P, P, P, P, P, P, P], st),
            "digest_gat_query": ([P, P], st),
            "digest_gat_bind_workspace": ([P, P, sz, P], st),
            "digest_gat_forward": ([P, i32, P, P, P, ctypes.c_float, P, i32, P], st),
            "digest_gat_backward": ([P, i32, P, P, P, P, P, P, P, P, P], st),
            "digest_push_add": ([P, i32, P, P, P], st),
            "digest_pull_add": ([P, i32, P, P, P], st),
            "digest_sync_period": ([i32, i64, P, P], st),
            "digest_profile_enable": ([P, i32], st),
            "digest_profile_read": ([P, P, P], st),
            "digest_profile_kernel_count": ([], i32),
            "digest_profile_kernel_name": ([i32], ctypes.c_char_p),
            "digest_partition_plan": ([P, i32, P], st),
            "digest_profile_model": ([P, i32, P, P, P], st),
        }
        for name, (args, res) in sig.items():
            f = getattr(L, name)
            f.argtypes = args
            f.restype = res
        _lib = L
    return _lib


def _check(status):
    if status != OK:
        raise DigestError(status, lib().digest_last_error().decode())


def _np(a, dtype):
    a = np.ascontiguousarray(a, dtype=dtype)
    return a, a.ctypes.data_as(ctypes.c_void_p)


def _stream(stream):
    if stream is None:
        import torch
        return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, int):
        return ctypes.c_void_p(stream)
    return ctypes.c_void_p(stream.cuda_stream)


def _dev(t, dtype, numel, name):
    """Device pointer of a contiguous CUDA tensor with exactly ``numel`` elements."""
    import torch
    if t is None:
        raise ValueError(f"{name} is required")
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a CUDA tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if t.numel() != numel:
        raise ValueError(f"{name} has {t.numel()} elements, expected {numel}")
    return ctypes.c_void_p(t.data_ptr())


class Partition:
    """Handle of one partition (wraps ``digest_partition*``)."""

    def __init__(self, handle, n_global, n_own, n_halo, widths):
        self.handle = ctypes.c_void_p(handle)
        self.n_global = n_global
        self.n_own = n_own
        self.n_halo = n_halo
        self.widths = list(widths)
        self.L = len(self.widths) - 1
        self.workspace = None
        q = digest_partition_query(self)
        self.n_boundary = q["n_boundary"]
        self.nnz = q["nnz"]
        self.nnz_in = q["nnz_in"]
        self.workspace_bytes = q["workspace_bytes"]

    def __del__(self):
        try:
            digest_partition_destroy(self)
        except Exception:
            pass


def digest_partition_create(n_global, indptr, indices, values, owned, halo, widths):
    indptr, p_indptr = _np(indptr, np.int64)
    indices, p_indices = _np(indices, np.int64)
    values, p_values = _np(values, np.float32)
    owned, p_owned = _np(owned, np.int64)
    halo, p_halo = _np(halo, np.int64)
    widths, p_widths = _np(widths, np.int32)
    if indptr.shape[0] != owned.shape[0] + 1:
        raise ValueError("indptr must have n_owned + 1 entries")
    nnz = int(indptr[-1]) if indptr.size else 0
    if indices.shape[0] < nnz or values.shape[0] < nnz:
        raise ValueError("indices/values shorter than indptr[-1]")
    out = ctypes.c_void_p()
    _check(lib().digest_partition_create(int(n_global), p_indptr, p_indices, p_values, p_owned,
                                         owned.shape[0], p_halo, halo.shape[0],
                                         widths.shape[0] - 1, p_widths, ctypes.byref(out)))
    return Partition(out.value, int(n_global), owned.shape[0], halo.shape[0], widths.tolist())


def digest_partition_destroy(p):
    if p.handle:
        lib().digest_partition_destroy(p.handle)
        p.handle = ctypes.c_void_p()


def digest_partition_query(p):
    nb, nnz, nnz_in = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
    ws = ctypes.c_size_t()
    _check(lib().digest_partition_query(p.handle, ctypes.byref(nb), ctypes.byref(nnz),
                                        ctypes.byref(nnz_in), ctypes.byref(ws)))
    return {"n_boundary": nb.value, "nnz": nnz.value, "nnz_in": nnz_in.value,
            "workspace_bytes": ws.value}


def digest_partition_bind_workspace(p, workspace, stream=None):
    """Bind a CUDA uint8 tensor of at least ``p.workspace_bytes`` bytes."""
    import torch
    if not isinstance(workspace, torch.Tensor) or not workspace.is_cuda:
        raise TypeError("workspace must be a CUDA tensor")
    nbytes = workspace.numel() * workspace.element_size()
    _check(lib().digest_partition_bind_workspace(p.handle, ctypes.c_void_p(workspace.data_ptr()),
                                                 nbytes, _stream(stream)))
    p.workspace = workspace


def digest_partition_export_maps(p):
    col = np.empty(p.nnz, np.int32)
    bgid = np.empty(p.n_boundary, np.int64)
    bloc = np.empty(p.n_boundary, np.int32)
    _check(lib().digest_partition_export_maps(p.handle, col.ctypes.data_as(ctypes.c_void_p),
                                              bgid.ctypes.data_as(ctypes.c_void_p),
                                              bloc.ctypes.data_as(ctypes.c_void_p)))
    return col, bgid, bloc


def digest_partition_export_transpose(p):
    ptr = np.empty(p.n_own + 1, np.int64)
    src = np.empty(p.nnz_in, np.int32)
    val = np.empty(p.nnz_in, np.float32)
    _check(lib().digest_partition_export_transpose(p.handle, ptr.ctypes.data_as(ctypes.c_void_p),
                                                   src.ctypes.data_as(ctypes.c_void_p),
                                                   val.ctypes.data_as(ctypes.c_void_p)))
    return ptr, src, val


def digest_partition_read_halo(p, level, out, stream=None):
    import torch
    _check_level(p, level, 0)
    ptr = _dev(out, torch.float32, p.n_halo * p.widths[level], "out")
    _check(lib().digest_partition_read_halo(p.handle, int(level), ptr, _stream(stream)))


def _check_level(p, level, lo):
    if not (lo <= level < p.L):
        raise DigestError(EINVAL, f"level {level} outside [{lo}, {p.L})")


def _check_layer(p, layer):
    if not (1 <= layer <= p.L):
        raise DigestError(EINVAL, f"layer {layer} outside [1, {p.L}]")


def digest_partition_set_pull_mode(p, mode):
    _check(lib().digest_partition_set_pull_mode(p.handle, int(mode)))


def digest_pull(p, level, store, stream=None):
    import torch
    _check_level(p, level, 0)
    ptr = _dev(store, torch.float32, p.n_global * p.widths[level], "store")
    _check(lib().digest_pull(p.handle, int(level), ptr, _stream(stream)))


def digest_push(p, level, h_own, store, mode=PUSH_BOUNDARY, stream=None):
    import torch
    _check_level(p, level, 1)
    d = p.widths[level]
    ph = _dev(h_own, torch.float32, p.n_own * d, "h_own")
    ps = _dev(store, torch.float32, p.n_global * d, "store")
    _check(lib().digest_push(p.handle, int(level), ph, ps, int(mode), _stream(stream)))


def digest_layer_forward(p, layer, h_in, w, h_out, act, stream=None):
    import torch
    _check_layer(p, layer)
    di, do = p.widths[layer - 1], p.widths[layer]
    a = _dev(h_in, torch.float32, p.n_own * di, "h_in")
    b = _dev(w, torch.float32, di * do, "w")
    c = _dev(h_out, torch.float32, p.n_own * do, "h_out")
    _check(lib().digest_layer_forward(p.handle, int(layer), a, b, c, int(act), _stream(stream)))


def digest_layer_backward(p, layer, h_in, h_out, dh_out, w, dw, dh_in=None, stream=None):
    import torch
    _check_layer(p, layer)
    di, do = p.widths[layer - 1], p.widths[layer]
    x = _dev(h_in, torch.float32, p.n_own * di, "h_in")
    a = _dev(h_out, torch.float32, p.n_own * do, "h_out")
    b = _dev(dh_out, torch.float32, p.n_own * do, "dh_out")
    c = _dev(w, torch.float32, di * do, "w")
    e = _dev(dw, torch.float32, di * do, "dw")
    f = _dev(dh_in, torch.float32, p.n_own * di, "dh_in") if dh_in is not None else None
    _check(lib().digest_layer_backward(p.handle, int(layer), x, a, b, c, e, f, _stream(stream)))


def digest_layer_backward_halo(p, layer, h_in, h_out, dh_out, w, dw, dh_in, dh_halo,
                               stream=None):
    """digest_layer_backward plus dh_halo = P_out^T D W^T (layer 2..L)."""
    import torch
    _check_layer(p, layer)
    di, do = p.widths[layer - 1], p.widths[layer]
    _check(lib().digest_layer_backward_halo(
        p.handle, int(layer), _dev(h_in, torch.float32, p.n_own * di, "h_in"),
        _dev(h_out, torch.float32, p.n_own * do, "h_out"),
        _dev(dh_out, torch.float32, p.n_own * do, "dh_out"),
        _dev(w, torch.float32, di * do, "w"), _dev(dw, torch.float32, di * do, "dw"),
        _dev(dh_in, torch.float32, p.n_own * di, "dh_in"),
        _dev(dh_halo, torch.float32, p.n_halo * di, "dh_halo"), _stream(stream)))


GAT_SLOPE = 0.2   # the GAT model's LeakyReLU slope


def digest_gat_query(p):
    """Bytes of the partition's GAT workspace."""
    n = ctypes.c_size_t(0)
    _check(lib().digest_gat_query(p.handle, ctypes.byref(n)))
    return int(n.value)


def digest_gat_bind_workspace(p, workspace, stream=None):
    """Bind a CUDA tensor of at least digest_gat_query(p) bytes."""
    import torch
    if not isinstance(workspace, torch.Tensor) or not workspace.is_cuda:
        raise TypeError("GAT workspace must be a CUDA tensor")
    nbytes = workspace.numel() * workspace.element_size()
    _check(lib().digest_gat_bind_workspace(p.handle, ctypes.c_void_p(workspace.data_ptr()),
                                           nbytes, _stream(stream)))
    p.gat_workspace = workspace   # kept alive with the handle


def digest_gat_forward(p, layer, h_in, w, att, h_out, act, slope=GAT_SLOPE, stream=None):
    import torch
    _check_layer(p, layer)
    di, do = p.widths[layer - 1], p.widths[layer]
    _check(lib().digest_gat_forward(
        p.handle, int(layer), _dev(h_in, torch.float32, p.n_own * di, "h_in"),
        _dev(w, torch.float32, di * do, "w"), _dev(att, torch.float32, do * 2, "att"),
        ctypes.c_float(slope), _dev(h_out, torch.float32, p.n_own * do, "h_out"), int(act),
        _stream(stream)))


def digest_gat_backward(p, layer, h_in, h_out, dh_out, w, att, dw, datt, dh_in=None,
                        stream=None):
    import torch
    _check_layer(p, layer)
    di, do = p.widths[layer - 1], p.widths[layer]
    _check(lib().digest_gat_backward(
        p.handle, int(layer), _dev(h_in, torch.float32, p.n_own * di, "h_in"),
        _dev(h_out, torch.float32, p.n_own * do, "h_out"),
        _dev(dh_out, torch.float32, p.n_own * do, "dh_out"),
        _dev(w, torch.float32, di * do, "w"), _dev(att, torch.float32, do * 2, "att"),
        _dev(dw, torch.float32, di * do, "dw"), _dev(datt, torch.float32, do * 2, "datt"),
        _dev(dh_in, torch.float32, p.n_own * di, "dh_in") if dh_in is not None else None,
        _stream(stream)))


def digest_softmax_xent(p, logits, labels, dlogits, loss, stream=None):
    import torch
    C = p.widths[-1]
    a = _dev(logits, torch.float32, p.n_own * C, "logits")
    b = _dev(labels, torch.int32, p.n_own, "labels")
    c = _dev(dlogits, torch.float32, p.n_own * C, "dlogits")
    d = _dev(loss, torch.float32, 1, "loss")
    _check(lib().digest_softmax_xent(p.handle, a, b, c, d, _stream(stream)))


def digest_softmax_xent_static(logits, labels, dlogits, loss, stream=None):
    """The loss head without a partition or workspace (for callers that
    cannot allocate): logits [n, C], labels int32 [n], dlogits [n, C], loss
    [1]; partial sums in the library's fixed device array."""
    import torch
    if logits.dim() != 2:
        raise ValueError("logits must be [n, C]")
    n, C = int(logits.shape[0]), int(logits.shape[1])
    _check(lib().digest_softmax_xent_static(
        n, C, _dev(logits, torch.float32, n * C, "logits"),
        _dev(labels, torch.int32, n, "labels"), _dev(dlogits, torch.float32, n * C, "dlogits"),
        _dev(loss, torch.float32, 1, "loss"), _stream(stream)))


def digest_halo_gradient(p, layer, h_out, dh_out, w, dh_halo, stream=None):
    """dh_halo = P_out^T D W^T for the halo rows of level layer-1."""
    import torch
    _check_layer(p, layer)
    d_in, d_out = p.widths[layer - 1], p.widths[layer]
    _check(lib().digest_halo_gradient(
        p.handle, int(layer), _dev(h_out, torch.float32, p.n_own * d_out, "h_out"),
        _dev(dh_out, torch.float32, p.n_own * d_out, "dh_out"),
        _dev(w, torch.float32, d_in * d_out, "w"),
        _dev(dh_halo, torch.float32, p.n_halo * d_in, "dh_halo"), _stream(stream)))


def digest_push_add(p, level, dh_halo, gstore, stream=None):
    """gstore[halo] += dh_halo (level 1..L-1)."""
    import torch
    _check_level(p, level, 1)
    d = p.widths[level]
    _check(lib().digest_push_add(p.handle, int(level),
                                 _dev(dh_halo, torch.float32, p.n_halo * d, "dh_halo"),
                                 _dev(gstore, torch.float32, p.n_global * d, "gstore"),
                                 _stream(stream)))


def digest_pull_add(p, level, gstore, dh_own, stream=None):
    """dh_own += gstore[owned]; gstore[owned] = 0 (level 1..L-1)."""
    import torch
    _check_level(p, level, 1)
    d = p.widths[level]
    _check(lib().digest_pull_add(p.handle, int(level),
                                 _dev(gstore, torch.float32, p.n_global * d, "gstore"),
                                 _dev(dh_own, torch.float32, p.n_own * d, "dh_own"),
                                 _stream(stream)))


def digest_sgd_average(w, grads, lr, stream=None):
    """w -= lr * mean(grads), the average of the local models (Algorithm 1, AGG)."""
    import torch
    if not grads:
        raise ValueError("need at least one gradient")
    n = w.numel()
    pw = _dev(w, torch.float32, n, "w")
    ptrs = (ctypes.c_void_p * len(grads))(*[_dev(g, torch.float32, n, f"grads[{m}]").value
                                            for m, g in enumerate(grads)])
    _check(lib().digest_sgd_average(pw, ptrs, len(grads), n, float(lr), _stream(stream)))


def digest_sync_period(K, iteration):
    a, b = ctypes.c_int32(), ctypes.c_int32()
    _check(lib().digest_sync_period(int(K), int(iteration), ctypes.byref(a), ctypes.byref(b)))
    return bool(a.value), bool(b.value)


def digest_profile_enable(p, on=True):
    _check(lib().digest_profile_enable(p.handle, 1 if on else 0))


def kernel_names():
    L = lib()
    return [L.digest_profile_kernel_name(i).decode() for i in range(L.digest_profile_kernel_count())]


def digest_profile_read(p):
    """Per (kernel kind, layer slot): {"kind.lN": (total ms, launches)} since the
    last read (synchronises).  Slot = layer for layer kernels, level for
    pull/push, L for the loss head; entries without launches are omitted."""
    n = lib().digest_profile_kernel_count()
    slots = p.L + 1
    ms = np.zeros(n * slots, np.float64)
    cnt = np.zeros(n * slots, np.int64)
    _check(lib().digest_profile_read(p.handle, ms.ctypes.data_as(ctypes.c_void_p),
                                     cnt.ctypes.data_as(ctypes.c_void_p)))
    out = {}
    for i, name in enumerate(kernel_names()):
        for sl in range(slots):
            j = i * slots + sl
            if cnt[j]:
                out[f"{name}.l{sl}"] = (float(ms[j]), int(cnt[j]))
    return out


class LayerPlan(ctypes.Structure):
    """``digest_layer_plan`` of include/digest.h."""
    _fields_ = [("transform_first", ctypes.c_int32), ("forward_narrow", ctypes.c_int32),
                ("dw_slices", ctypes.c_int32), ("dgrad_narrow_first", ctypes.c_int32),
                ("dgrad_fused", ctypes.c_int32), ("tiers_fwd", ctypes.c_int32),
                ("tiers_bwd", ctypes.c_int32), ("tier_rows_fwd", ctypes.c_int32),
                ("tier_rows_bwd", ctypes.c_int32), ("tier_entries_fwd", ctypes.c_int64),
                ("tier_entries_bwd", ctypes.c_int64), ("forward_fused", ctypes.c_int32),
                ("backward_fused", ctypes.c_int32)]


def digest_partition_plan(p, layer):
    """The library's launch plan of ``layer`` as a dict of the C fields."""
    _check_layer(p, layer)
    out = LayerPlan()
    _check(lib().digest_partition_plan(p.handle, int(layer), ctypes.byref(out)))
    return {name: int(getattr(out, name)) for name, _ in LayerPlan._fields_}


def digest_profile_model(p, model=MODEL_GCN):
    """Algorithmic (bytes, flops, sparse entries) of one launch of each
    (kernel kind, slot) a round makes, keyed like ``digest_profile_read``;
    kinds the round does not launch are omitted."""
    n = lib().digest_profile_kernel_count()
    slots = p.L + 1
    b = np.zeros(n * slots, np.float64)
    f = np.zeros(n * slots, np.float64)
    e = np.zeros(n * slots, np.int64)
    _check(lib().digest_profile_model(p.handle, int(model), b.ctypes.data_as(ctypes.c_void_p),
                                      f.ctypes.data_as(ctypes.c_void_p),
                                      e.ctypes.data_as(ctypes.c_void_p)))
    out = {}
    for i, name in enumerate(kernel_names()):
        for sl in range(slots):
            j = i * slots + sl
            if b[j] or f[j] or e[j]:
                out[f"{name}.l{sl}"] = (float(b[j]), float(f[j]), int(e[j]))
    return out
