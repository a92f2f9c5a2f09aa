"""CPU oracle for one DIGEST partition's GCN layer (arXiv 2206.00057).

TEST INFRASTRUCTURE ONLY.  Only the tests, ``__graft_entry__.smoke()`` and the
CPU leg of ``bench.py`` may import this package.  It shares no code with the
HIP library in ``paper_2206_00057_amd`` and imports nothing from it: inputs
arrive as plain numpy arrays.

The arithmetic lives in ``digest_oracle.c`` (plain C, double accumulation);
this module compiles it with gcc on first use and marshals numpy arrays.

What each function follows in the paper:
  - ``partition_maps`` / ``owned_transpose``: Eq. 2 (in/out-of-subgraph split),
    the halo and push sets of Sec. 3.2, P_in of Eq. 5.
  - ``pull`` / ``push``: the pull and push operations of Sec. 3.2.
  - ``aggregate`` / ``transform`` / ``OraclePartition.forward``: Eq. 5 (Eq. 4).
  - ``softmax_xent``: the local loss of Eq. 3 with cross entropy.
  - ``layer_backward``: Eq. 6 completed by the chain rule of the GCN backward
    (Appendix A.3), halo rows held constant.
  - ``sync_period``: the pull/push conditions of Algorithm 1.
  - ``gat_forward`` / ``gat_backward``: the stale-representation layer of
    Eq. 4 with the attention aggregation of the GAT model the experiments
    train (single head), and its chain-rule backward, halo rows constant.

Every function is pinned by ``tests/test_oracle_pins.py`` against
brute-force set algebra, dense matrices, scipy/torch fp64 routines, closed
forms, finite differences and the golden fixtures in ``tests/golden/``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "digest_oracle.c")
_LIB_DIR = os.path.join(_HERE, "_build")
_LIB = os.path.join(_LIB_DIR, "liboracle.so")

RELU = 0
IDENTITY = 1

_lock = threading.Lock()
_lib = None


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (fp64, no fast-math) and return the path."""
    os.makedirs(_LIB_DIR, exist_ok=True)
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + f".tmp{os.getpid()}"
        subprocess.check_call(
            ["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared", "-Wall",
             "-Werror", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    with _lock:
        if _lib is None:
            lib = ctypes.CDLL(build())
            i64, i32, f32, f64 = ctypes.c_int64, ctypes.c_int32, ctypes.c_float, ctypes.c_double
            P = ctypes.c_void_p
            lib.oracle_num_threads.restype = ctypes.c_int
            lib.oracle_set_num_threads.argtypes = [ctypes.c_int]
            lib.oracle_set_num_threads.restype = ctypes.c_int
            lib.oracle_partition_maps.argtypes = [i64, P, P, i64, P, i64, P, P, P, P]
            lib.oracle_partition_maps.restype = ctypes.c_int
            lib.oracle_owned_transpose.argtypes = [i64, P, P, P, P, P, P]
            lib.oracle_owned_transpose.restype = i64
            lib.oracle_pull.argtypes = [P, i64, i64, P, P]
            lib.oracle_push.argtypes = [P, i64, P, i64, P, P]
            lib.oracle_aggregate.argtypes = [i64, P, P, P, P, P, i64, P]
            lib.oracle_transform.argtypes = [i64, i64, i64, P, P, ctypes.c_int, P]
            lib.oracle_softmax_xent.argtypes = [i64, i64, P, P, P, ctypes.POINTER(f64)]
            lib.oracle_softmax_xent.restype = ctypes.c_int
            lib.oracle_layer_backward.argtypes = [i64, P, P, P, P, P, i64, i64, P, P, P,
                                                  ctypes.c_int, P, P]
            lib.oracle_sync_period.argtypes = [i32, i64, ctypes.POINTER(i32), ctypes.POINTER(i32)]
            lib.oracle_sync_period.restype = ctypes.c_int
            lib.oracle_sgd_average.argtypes = [P, P, i32, i64, f32]
            lib.oracle_halo_gradient.argtypes = [i64, i64, P, P, P, i64, i64, P, P, P,
                                                 ctypes.c_int, P]
            lib.oracle_sgd_average.restype = ctypes.c_int
            lib.oracle_gat_forward.argtypes = [i64, i64, P, P, P, P, i64, i64, P, P, f64,
                                               ctypes.c_int, P, P]
            lib.oracle_gat_backward.argtypes = [i64, i64, P, P, P, P, i64, i64, P, P, f64,
                                                ctypes.c_int, P, P, P, P, P]
            del f32
            _lib = lib
    return _lib


def num_threads() -> int:
    return int(_load().oracle_num_threads())


def set_num_threads(n: int) -> int:
    """Thread count of the oracle's OpenMP loops from now on; returns it."""
    return int(_load().oracle_set_num_threads(int(n)))


def _c(a, dtype):
    a = np.ascontiguousarray(a, dtype=dtype)
    return a


def _p(a):
    return a.ctypes.data_as(ctypes.c_void_p) if a is not None else None


class OracleError(ValueError):
    pass


def partition_maps(n_global, indptr, indices, owned, halo):
    """Local column numbering and the boundary (pushed) rows.

    Returns ``(col_local int32[nnz], boundary_local int32[n_boundary])``.
    Raises ``OracleError`` on malformed input.
    """
    indptr = _c(indptr, np.int64)
    indices = _c(indices, np.int64)
    owned = _c(owned, np.int64)
    halo = _c(halo, np.int64)
    n_own = owned.shape[0]
    if indptr.shape[0] != n_own + 1:
        raise OracleError("indptr length must be n_own + 1")
    col_local = np.empty(indices.shape[0], np.int32)
    boundary = np.empty(max(n_own, 1), np.int32)
    nb = ctypes.c_int64(0)
    rc = _load().oracle_partition_maps(
        int(n_global), _p(indptr), _p(indices), n_own, _p(owned), halo.shape[0],
        _p(halo), _p(col_local), _p(boundary), ctypes.byref(nb))
    if rc != 0:
        raise OracleError("invalid partition description")
    return col_local, boundary[: nb.value].copy()


def owned_transpose(n_own, indptr, col_local, values):
    """CSR of P_in^T: ``(t_indptr int64[n_own+1], t_src int32, t_vals float32)``."""
    indptr = _c(indptr, np.int64)
    col_local = _c(col_local, np.int32)
    values = _c(values, np.float32)
    t_indptr = np.empty(n_own + 1, np.int64)
    t_src = np.empty(max(col_local.shape[0], 1), np.int32)
    t_vals = np.empty(max(col_local.shape[0], 1), np.float32)
    nnz_in = _load().oracle_owned_transpose(n_own, _p(indptr), _p(col_local), _p(values),
                                            _p(t_indptr), _p(t_src), _p(t_vals))
    return t_indptr, t_src[:nnz_in].copy(), t_vals[:nnz_in].copy()


def pull(store, halo):
    store = _c(store, np.float32)
    halo = _c(halo, np.int64)
    d = store.shape[1]
    out = np.empty((halo.shape[0], d), np.float32)
    _load().oracle_pull(_p(store), d, halo.shape[0], _p(halo), _p(out))
    return out


def push(h_own, owned, rows, store):
    """Overwrite ``store`` (in place) at ``owned[rows]`` with ``h_own[rows]``."""
    h_own = _c(h_own, np.float32)
    owned = _c(owned, np.int64)
    rows = _c(rows, np.int32)
    assert store.dtype == np.float32 and store.flags.c_contiguous
    _load().oracle_push(_p(h_own), h_own.shape[1], _p(owned), rows.shape[0], _p(rows), _p(store))
    return store


def aggregate(indptr, col_local, values, h_own, halo_buf):
    indptr = _c(indptr, np.int64)
    col_local = _c(col_local, np.int32)
    values = _c(values, np.float32)
    h_own = _c(h_own, np.float32)
    d = h_own.shape[1]
    halo_buf = _c(halo_buf if halo_buf is not None else np.zeros((0, d), np.float32), np.float32)
    n_own = indptr.shape[0] - 1
    out = np.empty((n_own, d), np.float32)
    _load().oracle_aggregate(n_own, _p(indptr), _p(col_local), _p(values), _p(h_own),
                             _p(halo_buf), d, _p(out))
    return out


def transform(ah, w, act):
    ah = _c(ah, np.float32)
    w = _c(w, np.float32)
    n, d_in = ah.shape
    assert w.shape[0] == d_in
    out = np.empty((n, w.shape[1]), np.float32)
    _load().oracle_transform(n, d_in, w.shape[1], _p(ah), _p(w), int(act), _p(out))
    return out


def softmax_xent(logits, labels):
    """Returns ``(loss float, dlogits float32[n, C])``."""
    logits = _c(logits, np.float32)
    labels = _c(labels, np.int32)
    n, C = logits.shape
    d = np.empty_like(logits)
    loss = ctypes.c_double(0.0)
    rc = _load().oracle_softmax_xent(n, C, _p(logits), _p(labels), _p(d), ctypes.byref(loss))
    if rc != 0:
        raise OracleError("label outside [0, C)")
    return loss.value, d


def layer_backward(indptr, col_local, values, h_own, halo_buf, w, h_out, dh_out, act,
                   want_dh_in=True):
    """Returns ``(dw float32[d_in, d_out], dh_in float32[n_own, d_in] or None)``."""
    indptr = _c(indptr, np.int64)
    col_local = _c(col_local, np.int32)
    values = _c(values, np.float32)
    h_own = _c(h_own, np.float32)
    d_in = h_own.shape[1]
    halo_buf = _c(halo_buf if halo_buf is not None else np.zeros((0, d_in), np.float32),
                  np.float32)
    w = _c(w, np.float32)
    h_out = _c(h_out, np.float32)
    dh_out = _c(dh_out, np.float32)
    n_own = indptr.shape[0] - 1
    d_out = w.shape[1]
    dw = np.empty((d_in, d_out), np.float32)
    dh_in = np.empty((n_own, d_in), np.float32) if want_dh_in else None
    _load().oracle_layer_backward(n_own, _p(indptr), _p(col_local), _p(values), _p(h_own),
                                  _p(halo_buf), d_in, d_out, _p(w), _p(h_out), _p(dh_out),
                                  int(act), _p(dw), _p(dh_in))
    return dw, dh_in


def sync_period(K, r):
    """Algorithm 1 schedule: ``(do_pull, do_push)`` for round ``r`` (1-based)."""
    a, b = ctypes.c_int32(0), ctypes.c_int32(0)
    rc = _load().oracle_sync_period(int(K), int(r), ctypes.byref(a), ctypes.byref(b))
    if rc != 0:
        raise OracleError("K and r must be >= 1")
    return bool(a.value), bool(b.value)


def halo_gradient(indptr, col_local, values, n_halo, w, h_out, dh_out, act):
    """The appendix's stale-gradient term P_out^T D W^T: float32 [n_halo, d_in]."""
    indptr = _c(indptr, np.int64)
    col_local = _c(col_local, np.int32)
    values = _c(values, np.float32)
    w = _c(w, np.float32)
    h_out = _c(h_out, np.float32)
    dh_out = _c(dh_out, np.float32)
    n_own = indptr.shape[0] - 1
    d_in, d_out = w.shape
    out = np.empty((int(n_halo), d_in), np.float32)
    _load().oracle_halo_gradient(n_own, int(n_halo), _p(indptr), _p(col_local), _p(values),
                                 d_in, d_out, _p(w), _p(h_out), _p(dh_out), int(act), _p(out))
    return out


GAT_SLOPE = 0.2   # LeakyReLU slope of the attention scores (the GAT model's value)


def _gat_common(indptr, col_local, h_own, halo_buf, w, att):
    indptr = _c(indptr, np.int64)
    col_local = _c(col_local, np.int32)
    h_own = _c(h_own, np.float32)
    w = _c(w, np.float32)
    att = _c(att, np.float32)
    d_in, d_out = w.shape
    halo_buf = _c(halo_buf if halo_buf is not None else np.zeros((0, d_in), np.float32),
                  np.float32)
    if att.shape != (d_out, 2):
        raise OracleError("att must be [d_out, 2] (source, target columns)")
    return indptr, col_local, h_own, halo_buf, w, att, d_in, d_out


def gat_forward(indptr, col_local, h_own, halo_buf, w, att, act, slope=GAT_SLOPE,
                want_alpha=False):
    """GAT layer forward with stale halo rows: float32 h_out [n_own, d_out]
    (and the attention weights in CSR entry order with want_alpha)."""
    indptr, col_local, h_own, halo_buf, w, att, d_in, d_out = _gat_common(
        indptr, col_local, h_own, halo_buf, w, att)
    n_own = indptr.shape[0] - 1
    out = np.empty((n_own, d_out), np.float32)
    alpha = np.empty(int(indptr[-1]), np.float32) if want_alpha else None
    _load().oracle_gat_forward(n_own, halo_buf.shape[0], _p(indptr), _p(col_local), _p(h_own),
                               _p(halo_buf), d_in, d_out, _p(w), _p(att), float(slope),
                               int(act), _p(out), _p(alpha) if want_alpha else None)
    return (out, alpha) if want_alpha else out


def gat_backward(indptr, col_local, h_own, halo_buf, w, att, h_out, dh_out, act,
                 slope=GAT_SLOPE, want_dh_in=True):
    """Returns (dw [d_in, d_out], datt [d_out, 2], dh_in [n_own, d_in] or None)."""
    indptr, col_local, h_own, halo_buf, w, att, d_in, d_out = _gat_common(
        indptr, col_local, h_own, halo_buf, w, att)
    n_own = indptr.shape[0] - 1
    h_out = _c(h_out, np.float32)
    dh_out = _c(dh_out, np.float32)
    dw = np.empty((d_in, d_out), np.float32)
    datt = np.empty((d_out, 2), np.float32)
    dh_in = np.empty((n_own, d_in), np.float32) if want_dh_in else None
    _load().oracle_gat_backward(n_own, halo_buf.shape[0], _p(indptr), _p(col_local), _p(h_own),
                                _p(halo_buf), d_in, d_out, _p(w), _p(att), float(slope),
                                int(act), _p(h_out), _p(dh_out), _p(dw), _p(datt),
                                _p(dh_in) if want_dh_in else None)
    return dw, datt, dh_in


def push_add(gstore, halo, dh_halo):
    """gstore[halo[j]] += dh_halo[j] (float32 adds; ``halo`` ids distinct)."""
    halo = _c(halo, np.int64)
    gstore[halo] = gstore[halo] + _c(dh_halo, np.float32)
    return gstore


def pull_add(gstore, owned, dh_own):
    """dh_own += gstore[owned]; gstore[owned] = 0.  Returns the new dh_own."""
    owned = _c(owned, np.int64)
    out = _c(dh_own, np.float32) + gstore[owned]
    gstore[owned] = 0.0
    return out


def sgd_average(w, grads, lr):
    """Algorithm 1's global update (AGG): the average of the M local models
    ``w - lr * grads[m]``; returns the new float32 ``w``."""
    w = _c(w, np.float32).copy()
    gs = [_c(g, np.float32) for g in grads]
    for g in gs:
        if g.shape != w.shape:
            raise OracleError("gradient shape differs from the parameter's")
    ptrs = (ctypes.c_void_p * max(len(gs), 1))(*[g.ctypes.data for g in gs])
    rc = _load().oracle_sgd_average(_p(w), ptrs, len(gs), w.size, float(lr))
    if rc != 0:
        raise OracleError("need at least one gradient")
    return w


class OraclePartition:
    """One partition's state, mirroring the library's call sequence.

    ``indptr/indices/values`` are the CSR rows of P (global column ids) for the
    owned nodes, in ``owned`` order; ``halo`` lists the out-of-partition
    neighbours; ``widths`` are d_0..d_L.
    """

    def __init__(self, n_global, indptr, indices, values, owned, halo, widths):
        self.n_global = int(n_global)
        self.indptr = _c(indptr, np.int64)
        self.values = _c(values, np.float32)
        self.owned = _c(owned, np.int64)
        self.halo = _c(halo, np.int64)
        self.widths = [int(x) for x in widths]
        self.L = len(self.widths) - 1
        self.n_own = self.owned.shape[0]
        self.n_halo = self.halo.shape[0]
        self.col_local, self.boundary = partition_maps(n_global, indptr, indices, owned, halo)
        self.t_indptr, self.t_src, self.t_vals = owned_transpose(
            self.n_own, self.indptr, self.col_local, self.values)
        self.halo_buf = {}

    @property
    def nnz(self):
        return int(self.indptr[-1])

    @property
    def nnz_in(self):
        return int(self.t_indptr[-1])

    def pull(self, level, store):
        self.halo_buf[level] = pull(store, self.halo)
        return self.halo_buf[level]

    def push(self, level, h_own, store, all_owned=False):
        rows = np.arange(self.n_own, dtype=np.int32) if all_owned else self.boundary
        return push(h_own, self.owned, rows, store)

    def aggregate(self, layer, h_in):
        return aggregate(self.indptr, self.col_local, self.values, h_in,
                         self.halo_buf.get(layer - 1))

    def forward(self, layer, h_in, w, act):
        return transform(self.aggregate(layer, h_in), w, act)

    def backward(self, layer, h_in, w, h_out, dh_out, act, want_dh_in=None):
        if want_dh_in is None:
            want_dh_in = layer > 1
        return layer_backward(self.indptr, self.col_local, self.values, h_in,
                              self.halo_buf.get(layer - 1), w, h_out, dh_out, act,
                              want_dh_in=want_dh_in)

    def halo_gradient(self, layer, w, h_out, dh_out, act):
        return halo_gradient(self.indptr, self.col_local, self.values, self.n_halo, w, h_out,
                             dh_out, act)

    def gat_forward(self, layer, h_in, w, att, act, slope=GAT_SLOPE, want_alpha=False):
        return gat_forward(self.indptr, self.col_local, h_in, self.halo_buf.get(layer - 1), w,
                           att, act, slope, want_alpha)

    def gat_backward(self, layer, h_in, w, att, h_out, dh_out, act, slope=GAT_SLOPE,
                     want_dh_in=None):
        if want_dh_in is None:
            want_dh_in = layer > 1
        return gat_backward(self.indptr, self.col_local, h_in, self.halo_buf.get(layer - 1), w,
                            att, h_out, dh_out, act, slope, want_dh_in)


class OracleTrainer:
    """Algorithm 1 (synchronous mode) over every subgraph, one after another
    at each layer: in round r every subgraph starts from the global W; for
    each layer l, if r mod K == 0 and l >= 2 every subgraph pulls level l-1,
    then every subgraph computes layer l, then, if (r-1) mod K == 0 and
    l < L, every subgraph pushes level l; then every subgraph computes its
    local loss (Eq. 3) and gradients, and AGG averages the M locally updated
    models.  ``parts`` carry owned / halo / CSR rows (global columns).

    grad_exchange adds the appendix's stale-gradient term: after the
    backward of layer l >= 2 (all subgraphs, layer by layer), every subgraph's
    halo gradient P_out^T D W^T is added into a per-level gradient store and
    each owner adds its rows to its input gradient -- in the same round
    ("fresh") or one round later ("stale", the t-1 of the appendix).  With
    "none" (reading A8) halo rows get no gradient.

    model="gat" runs the GAT layer over stale halo rows instead of Eq. 5;
    AGG then averages the attention matrices ``atts`` as well as W."""

    def __init__(self, n_global, parts, widths, X, labels, Ws, lr, K, grad_exchange="none",
                 model="gcn", atts=None):
        if grad_exchange not in ("none", "fresh", "stale"):
            raise OracleError("grad_exchange is none, fresh or stale")
        if model not in ("gcn", "gat"):
            raise OracleError("model is gcn or gat")
        if model == "gat" and (atts is None or len(atts) != len(widths) - 1):
            raise OracleError("a GAT model needs one attention matrix per layer")
        if model == "gat" and grad_exchange != "none":
            raise OracleError("the halo-gradient exchange is defined for GCN layers")
        self.model = model
        self.att = [_c(a, np.float32).copy() for a in atts] if model == "gat" else None
        self.widths = [int(x) for x in widths]
        self.L = len(self.widths) - 1
        self.lr, self.K = float(lr), int(K)
        self.grad_exchange = grad_exchange
        self.gstores = [None] + [np.zeros((int(n_global), self.widths[l]), np.float32)
                                 for l in range(1, self.L)]
        self.ops = [OraclePartition(n_global, p.indptr, p.indices, p.values, p.owned, p.halo,
                                    widths) for p in parts]
        self.X = _c(X, np.float32)
        self.x_own = [self.X[p.owned] for p in parts]
        self.y_own = [_c(labels, np.int32)[p.owned] for p in parts]
        self.W = [_c(w, np.float32).copy() for w in Ws]
        self.stores = [self.X] + [np.zeros((int(n_global), self.widths[l]), np.float32)
                                  for l in range(1, self.L)]
        self.logits = [None] * len(parts)
        self.losses = [None] * len(parts)

    def act(self, layer):
        return RELU if layer < self.L else IDENTITY

    def _forward(self, op, l, h):
        if self.model == "gat":
            return op.gat_forward(l, h, self.W[l - 1], self.att[l - 1], self.act(l))
        return op.forward(l, h, self.W[l - 1], self.act(l))

    def init_stores(self):
        """One forward of every subgraph at the current W, pulling before and
        pushing after every layer, then every halo level pulled."""
        for op in self.ops:
            op.pull(0, self.stores[0])
        h = list(self.x_own)
        for l in range(1, self.L):
            if l >= 2:
                for op in self.ops:
                    op.pull(l - 1, self.stores[l - 1])
            h = [self._forward(op, l, h[m]) for m, op in enumerate(self.ops)]
            for m, op in enumerate(self.ops):
                self.stores[l] = op.push(l, h[m], self.stores[l])
        for op in self.ops:
            for lev in range(1, self.L):
                op.pull(lev, self.stores[lev])

    def round(self, r):
        do_pull, do_push = sync_period(self.K, r)
        outs = [[None] * (self.L + 1) for _ in self.ops]
        for m in range(len(self.ops)):
            outs[m][0] = self.x_own[m]
        for l in range(1, self.L + 1):
            if do_pull and l >= 2:
                for op in self.ops:
                    op.pull(l - 1, self.stores[l - 1])
            for m, op in enumerate(self.ops):
                outs[m][l] = self._forward(op, l, outs[m][l - 1])
            if do_push and l <= self.L - 1:
                for m, op in enumerate(self.ops):
                    self.stores[l] = op.push(l, outs[m][l], self.stores[l])
        grads = [[None] * len(self.ops) for _ in range(self.L)]
        agrads = [[None] * len(self.ops) for _ in range(self.L)]
        dh = [None] * len(self.ops)
        for m in range(len(self.ops)):
            self.logits[m] = outs[m][self.L]
            self.losses[m], dh[m] = softmax_xent(outs[m][self.L], self.y_own[m])
        for l in range(self.L, 0, -1):
            dh_in = [None] * len(self.ops)
            for m, op in enumerate(self.ops):
                if self.model == "gat":
                    grads[l - 1][m], agrads[l - 1][m], dh_in[m] = op.gat_backward(
                        l, outs[m][l - 1], self.W[l - 1], self.att[l - 1], outs[m][l], dh[m],
                        self.act(l), want_dh_in=l > 1)
                else:
                    grads[l - 1][m], dh_in[m] = op.backward(l, outs[m][l - 1], self.W[l - 1],
                                                            outs[m][l], dh[m], self.act(l),
                                                            want_dh_in=l > 1)
            if l > 1 and self.grad_exchange != "none":
                hg = [op.halo_gradient(l, self.W[l - 1], outs[m][l], dh[m], self.act(l))
                      for m, op in enumerate(self.ops)]
                gs = self.gstores[l - 1]
                if self.grad_exchange == "fresh":
                    for m, op in enumerate(self.ops):
                        push_add(gs, op.halo, hg[m])
                    for m, op in enumerate(self.ops):
                        dh_in[m] = pull_add(gs, op.owned, dh_in[m])
                else:   # last round's halo gradients, then this round's for the next
                    for m, op in enumerate(self.ops):
                        dh_in[m] = pull_add(gs, op.owned, dh_in[m])
                    for m, op in enumerate(self.ops):
                        push_add(gs, op.halo, hg[m])
            dh = dh_in
        self.W = [sgd_average(self.W[l], grads[l], self.lr) for l in range(self.L)]
        if self.model == "gat":   # AGG of the attention parameters too
            self.att = [sgd_average(self.att[l], agrads[l], self.lr) for l in range(self.L)]
        return float(np.mean(self.losses))

