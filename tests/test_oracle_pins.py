"""Pins for the CPU oracle: checks against what the paper and mathematics fix,
never against the oracle itself.

  * set algebra on dense adjacency (halo set, local numbering, push set,
    symmetric-graph boundary identity, push-then-pull round trip);
  * a hand-derived worked example (tests/golden/path4_worked.txt);
  * single partition == plain GCN (scipy.sparse + numpy, float64);
  * sync interval 1 with a freshly pushed store == full-graph GCN rows;
  * dense brute force P[O, :] @ H_mixed @ W on graphs with <= 64 nodes;
  * backward vs torch float64 autograd with the stale rows detached, and
    exact central differences of linear functionals;
  * loss vs closed forms and torch's cross entropy in float64;
  * the schedule vs the table written out from Algorithm 1.
"""
import numpy as np
import pytest
import scipy.sparse as sp
import torch

import oracle
from paper_2206_00057_amd import synth


def tiny_cfg(n=48, blocks=4, cap=8, widths=(5, 6, 3), classes=3, **kw):
    return synth.scaled(synth.CONFIGS["tiny"], n, blocks=blocks, cap=cap, widths=widths,
                        classes=classes, **kw)


def dense(g):
    return sp.csr_matrix((g.values.astype(np.float64), g.indices, g.indptr),
                         shape=(g.n, g.n)).toarray()


def rel_close(a, b, rtol=2e-6, atol=1e-7):
    np.testing.assert_allclose(np.asarray(a, np.float64), np.asarray(b, np.float64),
                               rtol=rtol, atol=atol)


# --------------------------------------------------------------------------
# maps (Eq. 2; Sec. 3.2)
# --------------------------------------------------------------------------

@pytest.mark.parametrize("seed", [0, 1, 2])
def test_maps_match_set_algebra(seed):
    cfg = tiny_cfg()
    g = synth.make_graph(cfg, seed=seed)
    A = dense(g)
    for m in range(cfg.blocks):
        p = synth.make_partition(cfg, g, m)
        O = list(p.owned)
        Oset = set(O)
        # halo: every out-of-partition neighbour of an owned node
        brute_halo = sorted({u for v in O for u in range(g.n) if A[v, u] != 0 and u not in Oset})
        assert list(p.halo) == brute_halo
        col_local, boundary = oracle.partition_maps(g.n, p.indptr, p.indices, p.owned, p.halo)
        local = {v: i for i, v in enumerate(O)}
        local.update({u: len(O) + j for j, u in enumerate(brute_halo)})
        assert col_local.tolist() == [local[int(c)] for c in p.indices]
        brute_bnd = [i for i, v in enumerate(O) if any(A[v, u] != 0 and u not in Oset
                                                       for u in range(g.n))]
        assert boundary.tolist() == brute_bnd


def test_boundary_is_what_other_partitions_pull():
    """On a symmetric graph, the push set of m equals V_m intersected with the
    union of the other partitions' halo sets."""
    cfg = tiny_cfg(n=64)
    g = synth.make_graph(cfg, seed=5)
    parts = [synth.make_partition(cfg, g, m) for m in range(cfg.blocks)]
    for m, p in enumerate(parts):
        _, bnd = oracle.partition_maps(g.n, p.indptr, p.indices, p.owned, p.halo)
        others = set()
        for q, pq in enumerate(parts):
            if q != m:
                others |= set(pq.halo.tolist())
        assert set(p.owned[bnd].tolist()) == set(p.owned.tolist()) & others


def test_owned_transpose_dense_and_order():
    cfg = tiny_cfg(n=64)
    g = synth.make_graph(cfg, seed=7)
    p = synth.make_partition(cfg, g, 1)
    col_local, _ = oracle.partition_maps(g.n, p.indptr, p.indices, p.owned, p.halo)
    n = p.n_own
    t_indptr, t_src, t_vals = oracle.owned_transpose(n, p.indptr, col_local, p.values)
    A = dense(g)
    P_in = A[np.ix_(p.owned, p.owned)]
    T = sp.csr_matrix((t_vals.astype(np.float64), t_src, t_indptr), shape=(n, n)).toarray()
    np.testing.assert_array_equal(T, P_in.T)
    for c in range(n):
        srcs = t_src[t_indptr[c]:t_indptr[c + 1]]
        assert np.all(np.diff(srcs) >= 0)
    # P is symmetric, so the owned block is too
    np.testing.assert_array_equal(T, P_in)


def test_maps_reject_malformed():
    cfg = tiny_cfg()
    g = synth.make_graph(cfg, seed=0)
    p = synth.make_partition(cfg, g, 0)
    ok = (g.n, p.indptr, p.indices, p.owned, p.halo)
    oracle.partition_maps(*ok)
    bad_halo = p.halo[1:]                                        # a column neither owned nor halo
    with pytest.raises(oracle.OracleError):
        oracle.partition_maps(g.n, p.indptr, p.indices, p.owned, bad_halo)
    with pytest.raises(oracle.OracleError):                      # owned and halo overlap
        oracle.partition_maps(g.n, p.indptr, p.indices, p.owned, np.append(p.halo, p.owned[0]))
    with pytest.raises(oracle.OracleError):                      # duplicate owned id
        oracle.partition_maps(g.n, p.indptr, p.indices, np.append(p.owned[:-1], p.owned[0]), p.halo)
    with pytest.raises(oracle.OracleError):                      # id out of range
        oracle.partition_maps(int(max(p.halo.max(), p.owned.max())), p.indptr, p.indices,
                              p.owned, p.halo)
    bad_ptr = p.indptr.copy()
    bad_ptr[2] = bad_ptr[1] - 1
    with pytest.raises(oracle.OracleError):                      # non-monotone indptr
        oracle.partition_maps(g.n, bad_ptr, p.indices, p.owned, p.halo)


# --------------------------------------------------------------------------
# worked example (golden)
# --------------------------------------------------------------------------

def test_worked_path_example(golden):
    f = golden("path4_worked.txt")
    iv = lambda k: np.array([int(x) for x in f[k]], np.int64)
    fv = lambda k: np.array([float(x) for x in f[k]], np.float64)
    s6 = np.sqrt(6.0)
    values = np.array([1 / 2, 1 / s6, 1 / s6, 1 / 3, 1 / 3], np.float32)
    owned, halo = iv("owned"), iv("halo")
    op = oracle.OraclePartition(int(f["n_global"][0]), iv("indptr"), iv("indices"), values,
                                owned, halo, [1, 1])
    assert op.col_local.tolist() == iv("col_local").tolist()
    assert op.boundary.tolist() == iv("boundary").tolist()
    assert op.t_indptr.tolist() == iv("t_indptr").tolist()
    assert op.t_src.tolist() == iv("t_src").tolist()
    store = np.zeros((4, 1), np.float32)
    store[2, 0] = float(f["store_row_2"][0])
    store[3, 0] = 1e6          # node 3 is not a neighbour: must not leak in
    op.pull(0, store)
    h = fv("h_own").astype(np.float32).reshape(2, 1)
    w = fv("w").astype(np.float32).reshape(1, 1)
    ah = op.aggregate(1, h)
    rel_close(ah[:, 0], fv("ah"))
    out = op.forward(1, h, w, oracle.IDENTITY)
    rel_close(out[:, 0], fv("h_out"))
    dw, dh = op.backward(1, h, w, out, np.ones((2, 1), np.float32), oracle.IDENTITY,
                         want_dh_in=True)
    rel_close(dw.ravel(), fv("dw"))
    rel_close(dh[:, 0], fv("dh_in"))


# --------------------------------------------------------------------------
# forward (Eq. 5)
# --------------------------------------------------------------------------

def scipy_gcn(g, X, Ws):
    """Plain full-graph GCN in float64 with scipy: ReLU hidden layers, identity logits."""
    P = sp.csr_matrix((g.values.astype(np.float64), g.indices, g.indptr), shape=(g.n, g.n))
    H = [X.astype(np.float64)]
    for l, W in enumerate(Ws):
        Z = (P @ H[-1]) @ W.astype(np.float64)
        H.append(np.maximum(Z, 0) if l < len(Ws) - 1 else Z)
    return H


def test_single_partition_is_plain_gcn():
    cfg = synth.scaled(synth.CONFIGS["tiny"], 400, widths=(12, 10, 4), classes=4)
    g = synth.make_graph(cfg, seed=3)
    X = synth.features(cfg)
    Ws = synth.weights(cfg)
    ref = scipy_gcn(g, X, Ws)
    owned = np.arange(g.n, dtype=np.int64)
    op = oracle.OraclePartition(g.n, g.indptr, g.indices, g.values, owned,
                                np.zeros(0, np.int64), cfg.widths)
    assert op.boundary.size == 0 and op.n_halo == 0
    h = X
    for l, W in enumerate(Ws, start=1):
        act = oracle.RELU if l < cfg.layers else oracle.IDENTITY
        h = op.forward(l, h, W, act)
        rel_close(h, ref[l], rtol=1e-5, atol=1e-6)


@pytest.mark.parametrize("part", [0, 2])
def test_sync_interval_one_fresh_store_equals_full_graph(part):
    """With the store pushed at the current weights, P_in H_in + P_out H~_out = P_m H:
    the partition's outputs are the full-graph GCN rows of its nodes."""
    cfg = synth.CONFIGS["tiny"]
    g = synth.make_graph(cfg)
    X, Ws = synth.features(cfg), synth.weights(cfg)
    ref = scipy_gcn(g, X, Ws)
    p = synth.make_partition(cfg, g, part)
    op = oracle.OraclePartition(g.n, p.indptr, p.indices, p.values, p.owned, p.halo, cfg.widths)
    stores = [X] + [ref[l].astype(np.float32) for l in range(1, cfg.layers)]
    h = X[p.owned]
    for l, W in enumerate(Ws, start=1):
        op.pull(l - 1, stores[l - 1])
        act = oracle.RELU if l < cfg.layers else oracle.IDENTITY
        h = op.forward(l, h, W, act)
        rel_close(h, ref[l][p.owned], rtol=1e-5, atol=1e-6)


@pytest.mark.parametrize("seed", [0, 1])
def test_dense_bruteforce_with_stale_store(seed):
    cfg = tiny_cfg(n=60, blocks=3, widths=(7, 9, 5), classes=5)
    g = synth.make_graph(cfg, seed=seed)
    A = dense(g)
    p = synth.make_partition(cfg, g, 1)
    op = oracle.OraclePartition(g.n, p.indptr, p.indices, p.values, p.owned, p.halo, cfg.widths)
    rng = np.random.default_rng(seed + 100)
    W = rng.standard_normal((7, 9)).astype(np.float32)
    h_own = rng.standard_normal((p.n_own, 7)).astype(np.float32)
    store = rng.standard_normal((g.n, 7)).astype(np.float32)       # stale rows, all nodes
    op.pull(0, store)
    Hmix = store.astype(np.float64).copy()
    Hmix[p.owned] = h_own
    Z = A[p.owned] @ Hmix @ W.astype(np.float64)
    rel_close(op.forward(1, h_own, W, oracle.IDENTITY), Z, rtol=1e-5, atol=1e-6)
    rel_close(op.forward(1, h_own, W, oracle.RELU), np.maximum(Z, 0), rtol=1e-5, atol=1e-6)
    # a dropped halo term would make the output independent of the store
    store2 = store.copy()
    store2[p.halo] += 1.0
    op.pull(0, store2)
    assert not np.allclose(op.forward(1, h_own, W, oracle.IDENTITY), Z, atol=1e-3)


# --------------------------------------------------------------------------
# push / pull (Sec. 3.2)
# --------------------------------------------------------------------------

def test_push_then_pull_round_trip():
    cfg = tiny_cfg(n=64, widths=(3, 4, 2))
    g = synth.make_graph(cfg, seed=9)
    H = np.random.default_rng(1).standard_normal((g.n, 4)).astype(np.float32)
    store = np.full((g.n, 4), np.nan, np.float32)
    parts = [synth.make_partition(cfg, g, m) for m in range(cfg.blocks)]
    ops = [oracle.OraclePartition(g.n, p.indptr, p.indices, p.values, p.owned, p.halo, cfg.widths)
           for p in parts]
    for p, op in zip(parts, ops):
        op.push(1, H[p.owned], store)
    for p, op in zip(parts, ops):
        np.testing.assert_array_equal(op.pull(1, store), H[p.halo])
    # rows nobody reads stay untouched
    touched = set()
    for p, op in zip(parts, ops):
        touched |= set(p.owned[op.boundary].tolist())
    untouched = np.array(sorted(set(range(g.n)) - touched), np.int64)
    assert np.all(np.isnan(store[untouched]))
    # the paper-literal variant pushes every owned row
    store_all = np.zeros((g.n, 4), np.float32)
    for p, op in zip(parts, ops):
        op.push(1, H[p.owned], store_all, all_owned=True)
    np.testing.assert_array_equal(store_all, H)


# --------------------------------------------------------------------------
# backward (Eq. 6, Appendix A.3)
# --------------------------------------------------------------------------

def torch_layer_grads(A, p, h_own, stale, W, dh_out, relu):
    P = torch.tensor(A[p.owned], dtype=torch.float64)
    Hin = torch.tensor(h_own, dtype=torch.float64, requires_grad=True)
    Hst = torch.tensor(stale, dtype=torch.float64)          # constants: no gradient
    Wt = torch.tensor(W, dtype=torch.float64, requires_grad=True)
    Hmix = torch.zeros(A.shape[0], h_own.shape[1], dtype=torch.float64)
    Hmix = Hmix.index_copy(0, torch.tensor(p.halo), Hst)
    Hmix = Hmix.index_copy(0, torch.tensor(p.owned), Hin)
    Z = P @ Hmix @ Wt
    out = torch.relu(Z) if relu else Z
    (out * torch.tensor(dh_out, dtype=torch.float64)).sum().backward()
    return Wt.grad.numpy(), Hin.grad.numpy(), out.detach().numpy()


@pytest.mark.parametrize("relu", [True, False])
def test_backward_vs_torch_autograd(relu):
    cfg = tiny_cfg(n=64, widths=(6, 5, 3))
    g = synth.make_graph(cfg, seed=11)
    A = dense(g)
    p = synth.make_partition(cfg, g, 2)
    rng = np.random.default_rng(7)
    h_own = rng.standard_normal((p.n_own, 6)).astype(np.float32)
    stale = rng.standard_normal((p.n_halo, 6)).astype(np.float32)
    W = rng.standard_normal((6, 5)).astype(np.float32)
    dh = rng.standard_normal((p.n_own, 5)).astype(np.float32)
    op = oracle.OraclePartition(g.n, p.indptr, p.indices, p.values, p.owned, p.halo, cfg.widths)
    store = np.zeros((g.n, 6), np.float32)
    store[p.halo] = stale
    op.pull(1, store)
    act = oracle.RELU if relu else oracle.IDENTITY
    out = op.forward(2, h_own, W, act)
    dW_ref, dH_ref, out_ref = torch_layer_grads(A, p, h_own, stale, W, dh, relu)
    rel_close(out, out_ref, rtol=1e-5, atol=1e-6)
    dW, dH = op.backward(2, h_own, W, out, dh, act)
    rel_close(dW, dW_ref, rtol=1e-5, atol=1e-6)
    rel_close(dH, dH_ref, rtol=1e-5, atol=1e-6)
    # first layer: no input gradient requested
    _, none = oracle.layer_backward(op.indptr, op.col_local, op.values, h_own, op.halo_buf[1],
                                    W, out, dh, act, want_dh_in=False)
    assert none is None


def test_backward_exact_central_differences():
    """With identity activation the functional f = sum(dH_out * H_out) is linear
    in W and in H_in, so a central difference with step 1 is exact up to
    rounding of the float outputs."""
    cfg = tiny_cfg(n=48, widths=(4, 3, 2))
    g = synth.make_graph(cfg, seed=4)
    p = synth.make_partition(cfg, g, 0)
    op = oracle.OraclePartition(g.n, p.indptr, p.indices, p.values, p.owned, p.halo, cfg.widths)
    rng = np.random.default_rng(3)
    store = rng.standard_normal((g.n, 4)).astype(np.float32)
    op.pull(0, store)
    h = rng.standard_normal((p.n_own, 4)).astype(np.float32)
    W = rng.standard_normal((4, 3)).astype(np.float32)
    dh = rng.standard_normal((p.n_own, 3)).astype(np.float32)
    f = lambda hh, WW: float(np.sum(dh.astype(np.float64) *
                                    op.forward(1, hh, WW, oracle.IDENTITY).astype(np.float64)))
    out = op.forward(1, h, W, oracle.IDENTITY)
    dW, dH = op.backward(1, h, W, out, dh, oracle.IDENTITY, want_dh_in=True)
    for a in range(4):
        for b in range(3):
            Wp, Wm = W.copy(), W.copy()
            Wp[a, b] += 1.0
            Wm[a, b] -= 1.0
            assert abs((f(h, Wp) - f(h, Wm)) / 2 - dW[a, b]) < 1e-4 * (1 + abs(dW[a, b]))
    for i in range(0, p.n_own, 3):
        for c in range(4):
            hp, hm = h.copy(), h.copy()
            hp[i, c] += 1.0
            hm[i, c] -= 1.0
            assert abs((f(hp, W) - f(hm, W)) / 2 - dH[i, c]) < 1e-4 * (1 + abs(dH[i, c]))


# --------------------------------------------------------------------------
# loss (Eq. 3)
# --------------------------------------------------------------------------

def test_loss_closed_form_uniform_logits():
    n, C = 10, 7
    labels = np.arange(n, dtype=np.int32) % C
    loss, d = oracle.softmax_xent(np.zeros((n, C), np.float32), labels)
    assert abs(loss - np.log(C)) < 1e-12
    expect = np.full((n, C), 1.0 / C)
    expect[np.arange(n), labels] -= 1.0
    rel_close(d, expect / n, rtol=1e-6, atol=1e-9)


def test_loss_two_class_closed_form():
    z = np.array([[0.3, -1.2], [2.0, 0.5]], np.float32)
    y = np.array([0, 0], np.int32)
    loss, _ = oracle.softmax_xent(z, y)
    expect = np.mean(np.log1p(np.exp(z[:, 1].astype(np.float64) - z[:, 0])))
    assert abs(loss - expect) < 1e-12


def test_loss_vs_torch_cross_entropy():
    rng = np.random.default_rng(0)
    z = (3 * rng.standard_normal((50, 41))).astype(np.float32)
    y = rng.integers(0, 41, 50).astype(np.int32)
    loss, d = oracle.softmax_xent(z, y)
    zt = torch.tensor(z, dtype=torch.float64, requires_grad=True)
    lt = torch.nn.functional.cross_entropy(zt, torch.tensor(y, dtype=torch.long))
    lt.backward()
    assert abs(loss - lt.item()) < 1e-12
    rel_close(d, zt.grad.numpy(), rtol=1e-6, atol=1e-9)
    with pytest.raises(oracle.OracleError):
        oracle.softmax_xent(z, np.full(50, 41, np.int32))


# --------------------------------------------------------------------------
# schedule (Algorithm 1)
# --------------------------------------------------------------------------

def test_schedule_matches_algorithm_table(golden):
    rows = []
    import os
    from conftest import ROOT
    with open(os.path.join(ROOT, "tests", "golden", "alg1_schedule.txt")) as fh:
        for line in fh:
            line = line.split("#", 1)[0].split()
            if line:
                rows.append(tuple(int(x) for x in line))
    assert len(rows) > 20
    for K, r, pull, push in rows:
        assert oracle.sync_period(K, r) == (bool(pull), bool(push)), (K, r)
    with pytest.raises(oracle.OracleError):
        oracle.sync_period(0, 1)
    with pytest.raises(oracle.OracleError):
        oracle.sync_period(3, 0)


def test_repeated_entries_in_any_order_sum_like_a_dense_matrix():
    """A CSR row may list its columns in any order and repeat a column: the
    aggregation is the product with the dense matrix whose entry is the sum
    of the repeats (checked against a dense numpy product in float64)."""
    cfg = synth.CONFIGS["tiny"]
    g = synth.make_graph(cfg)
    base = synth.make_partition(cfg, g, 1)
    p = synth.scramble_rows(base, seed=3, repeat_frac=0.4, long_row=200)
    col, _ = oracle.partition_maps(g.n, p.indptr, p.indices, p.owned, p.halo)
    d = 9
    h_own = synth.normal((p.n_own, d), seed=1)
    halo = synth.normal((p.n_halo, d), seed=2)
    got = oracle.aggregate(p.indptr, col, p.values, h_own, halo)
    dense = np.zeros((p.n_own, p.n_own + p.n_halo))
    rows = np.repeat(np.arange(p.n_own), np.diff(p.indptr))
    np.add.at(dense, (rows, col), p.values.astype(np.float64))
    ref = dense @ np.vstack([h_own, halo]).astype(np.float64)
    np.testing.assert_allclose(got, ref, rtol=1e-6, atol=1e-6)
    assert p.nnz > base.nnz
