"""Pins for the oracle's GAT layer with stale halo rows (the stale-
representation layer of Eq. 4 with an attention aggregation), against what
the mathematics fixes, never against the oracle itself:

  * zero attention vectors give uniform attention over each row's entries:
    h_out = act(D^-1 S [H; H~] W) with S the 0/1 structure (dense numpy);
  * attention weights sum to one: when every local input row is the same
    vector x, every output row is act(x W) whatever the attention vectors;
  * with LeakyReLU slope 1 the target score adds the same constant to every
    entry of a row, so it cancels in the softmax: the output does not
    depend on the target column of att;
  * forward and every gradient (dW, datt, dH_own) against an independent
    dense float64 implementation (masked softmax over a dense score matrix)
    differentiated by torch autograd, the stale halo rows detached;
  * a partition whose halo rows hold the current full-graph rows computes
    the full-graph GAT rows of its owned nodes;
  * an owned row without entries gives act(0) and no gradient.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2206_00057_amd import synth

RELU, IDENT = oracle.RELU, oracle.IDENTITY


def small(widths=(12, 10, 6), n=240, blocks=4, seed=3, part=1):
    cfg = synth.scaled(synth.CONFIGS["tiny"], n, blocks=blocks, cap=16, widths=widths,
                       classes=widths[-1])
    g = synth.make_graph(cfg, seed=seed)
    p = synth.make_partition(cfg, g, part)
    op = oracle.OraclePartition(g.n, p.indptr, p.indices, p.values, p.owned, p.halo,
                                cfg.widths)
    return cfg, g, p, op


def structure(op):
    """Dense 0/1 matrix of the owned rows over all local columns."""
    S = np.zeros((op.n_own, op.n_own + op.n_halo))
    for i in range(op.n_own):
        for k in range(op.indptr[i], op.indptr[i + 1]):
            S[i, op.col_local[k]] += 1.0
    return S


def torch_gat(S, x_all, n_own, W, att, act, slope):
    """Dense GAT in float64: scores over every (owned row, local column)
    pair, masked to the entries of S before the softmax."""
    z = x_all @ W
    s = z @ att[:, 0]
    t = z[:n_own] @ att[:, 1]
    e = torch.nn.functional.leaky_relu(t[:, None] + s[None, :], negative_slope=slope)
    mask = torch.from_numpy(S > 0)
    e = e.masked_fill(~mask, float("-inf"))
    alpha = torch.softmax(e, dim=1)
    alpha = torch.nan_to_num(alpha, nan=0.0)   # rows without entries
    o = alpha @ z
    return torch.relu(o) if act == RELU else o


def rand(shape, seed, scale=1.0):
    return (np.random.default_rng(seed).standard_normal(shape) * scale).astype(np.float32)


@pytest.mark.parametrize("act", [RELU, IDENT])
def test_zero_attention_is_mean_aggregation(act):
    cfg, g, p, op = small()
    d_in, d_out = cfg.widths[0], cfg.widths[1]
    h = rand((op.n_own, d_in), 1)
    halo = rand((op.n_halo, d_in), 2)
    W = rand((d_in, d_out), 3, 0.4)
    out = oracle.gat_forward(op.indptr, op.col_local, h, halo, W, np.zeros((d_out, 2)), act)
    S = structure(op)
    ref = (S / S.sum(1, keepdims=True)) @ np.vstack([h, halo]).astype(np.float64) @ W
    if act == RELU:
        ref = np.maximum(ref, 0.0)
    np.testing.assert_allclose(out, ref, rtol=1e-5, atol=1e-6)


def test_attention_sums_to_one():
    cfg, g, p, op = small()
    d_in, d_out = cfg.widths[0], cfg.widths[1]
    x = rand((d_in,), 4)
    h = np.tile(x, (op.n_own, 1))
    halo = np.tile(x, (op.n_halo, 1))
    W = rand((d_in, d_out), 5, 0.4)
    att = rand((d_out, 2), 6, 2.0)
    out, alpha = oracle.gat_forward(op.indptr, op.col_local, h, halo, W, att, IDENT,
                                    want_alpha=True)
    np.testing.assert_allclose(out, np.tile(x.astype(np.float64) @ W, (op.n_own, 1)),
                               rtol=1e-5, atol=1e-6)
    rows = np.add.reduceat(alpha.astype(np.float64), op.indptr[:-1])
    np.testing.assert_allclose(rows, 1.0, rtol=1e-6)


def test_target_score_cancels_at_slope_one():
    cfg, g, p, op = small()
    d_in, d_out = cfg.widths[0], cfg.widths[1]
    h, halo = rand((op.n_own, d_in), 7), rand((op.n_halo, d_in), 8)
    W = rand((d_in, d_out), 9, 0.4)
    att = rand((d_out, 2), 10, 1.0)
    att2 = att.copy()
    att2[:, 1] = rand((d_out,), 11, 3.0)
    a = oracle.gat_forward(op.indptr, op.col_local, h, halo, W, att, IDENT, slope=1.0)
    b = oracle.gat_forward(op.indptr, op.col_local, h, halo, W, att2, IDENT, slope=1.0)
    np.testing.assert_allclose(a, b, rtol=1e-5, atol=1e-6)
    # at the GAT slope the target column does matter
    c = oracle.gat_forward(op.indptr, op.col_local, h, halo, W, att, IDENT)
    d = oracle.gat_forward(op.indptr, op.col_local, h, halo, W, att2, IDENT)
    assert np.abs(c - d).max() > 1e-3


@pytest.mark.parametrize("act", [RELU, IDENT])
@pytest.mark.parametrize("widths", [(12, 10, 6), (5, 3, 2)])
def test_forward_and_gradients_match_dense_autograd(act, widths):
    cfg, g, p, op = small(widths=widths)
    d_in, d_out = cfg.widths[0], cfg.widths[1]
    h, halo = rand((op.n_own, d_in), 12), rand((op.n_halo, d_in), 13)
    W = rand((d_in, d_out), 14, 0.5)
    att = rand((d_out, 2), 15, 1.0)
    G = rand((op.n_own, d_out), 16)
    slope = oracle.GAT_SLOPE
    S = structure(op)

    ht = torch.tensor(h, dtype=torch.float64, requires_grad=True)
    Wt = torch.tensor(W, dtype=torch.float64, requires_grad=True)
    at = torch.tensor(att, dtype=torch.float64, requires_grad=True)
    halo_t = torch.tensor(halo, dtype=torch.float64)          # stale rows: constants
    out_t = torch_gat(S, torch.cat([ht, halo_t]), op.n_own, Wt, at, act, slope)
    (out_t * torch.tensor(G, dtype=torch.float64)).sum().backward()

    # the scores take both signs, so both LeakyReLU branches are exercised
    z = np.vstack([h, halo]).astype(np.float64) @ W
    pre = (z[:op.n_own] @ att[:, 1])[:, None] + (z @ att[:, 0])[None, :]
    assert (pre[S > 0] > 0).any() and (pre[S > 0] < 0).any()

    out = oracle.gat_forward(op.indptr, op.col_local, h, halo, W, att, act)
    np.testing.assert_allclose(out, out_t.detach().numpy(), rtol=1e-5, atol=1e-6)
    dw, datt, dh = oracle.gat_backward(op.indptr, op.col_local, h, halo, W, att, out, G, act)
    np.testing.assert_allclose(dw, Wt.grad.numpy(), rtol=1e-5, atol=1e-5)
    np.testing.assert_allclose(datt, at.grad.numpy(), rtol=1e-5, atol=1e-5)
    np.testing.assert_allclose(dh, ht.grad.numpy(), rtol=1e-5, atol=1e-5)


def test_fresh_halo_rows_give_full_graph_rows():
    cfg, g, p, op = small(widths=(12, 10, 6), part=2)
    d_in, d_out = cfg.widths[0], cfg.widths[1]
    X = rand((g.n, d_in), 17)
    W = rand((d_in, d_out), 18, 0.5)
    att = rand((d_out, 2), 19, 1.0)
    # the whole graph as one partition
    full = oracle.OraclePartition(g.n, g.indptr, g.indices, g.values, np.arange(g.n),
                                  np.zeros(0, np.int64), cfg.widths)
    ref = full.gat_forward(1, X, W, att, RELU)
    out = oracle.gat_forward(op.indptr, op.col_local, X[p.owned], X[p.halo], W, att, RELU)
    np.testing.assert_allclose(out, ref[p.owned], rtol=1e-5, atol=1e-6)
    # and a stale halo row changes the rows that read it, only those
    halo2 = X[p.halo].copy()
    halo2[0] += 1.0
    out2 = oracle.gat_forward(op.indptr, op.col_local, X[p.owned], halo2, W, att, RELU)
    reads = np.zeros(op.n_own, bool)
    for i in range(op.n_own):
        reads[i] = (op.col_local[op.indptr[i]:op.indptr[i + 1]] == op.n_own).any()
    assert reads.any()
    np.testing.assert_array_equal(out2[~reads], out[~reads])
    assert np.abs(out2[reads] - out[reads]).max() > 1e-4


def test_empty_row_gives_zero_and_no_gradient():
    # two owned rows over three local columns (one halo); row 1 is empty
    indptr = np.array([0, 2, 2], np.int64)
    col_local = np.array([0, 2], np.int32)
    h = rand((2, 4), 20)
    halo = rand((1, 4), 21)
    W = rand((4, 3), 22)
    att = rand((3, 2), 23)
    out = oracle.gat_forward(indptr, col_local, h, halo, W, att, IDENT)
    assert not out[1].any()
    dw, datt, dh = oracle.gat_backward(indptr, col_local, h, halo, W, att, out,
                                       np.ones((2, 3), np.float32), IDENT)
    # row 1 reads nothing and nobody reads it: its input gradient is zero
    assert not dh[1].any()
    assert np.abs(dh[0]).max() > 0


def test_backward_does_not_depend_on_the_thread_count():
    """Every sum of the GAT backward has one order whatever the thread count:
    one thread and several give the same bits, on rows longer than one
    column block of the parallel scatter."""
    cfg = synth.scaled(synth.CONFIGS["tiny"], 1500, widths=(20, 24, 6), classes=6)
    g = synth.make_graph(cfg, seed=9)
    p = synth.make_partition(cfg, g, 1)
    op = oracle.OraclePartition(g.n, p.indptr, p.indices, p.values, p.owned, p.halo,
                                cfg.widths)
    assert np.diff(op.indptr).max() > 64 and op.n_own + op.n_halo > 4 * 64
    h, halo = rand((op.n_own, 20), 30), rand((op.n_halo, 20), 31)
    W, att = rand((20, 24), 32, 0.3), rand((24, 2), 33, 0.5)
    G = rand((op.n_own, 24), 34)
    out = oracle.gat_forward(op.indptr, op.col_local, h, halo, W, att, RELU)
    before = oracle.num_threads()
    try:
        results = []
        for n in (1, 3, max(before, 4)):
            oracle.set_num_threads(n)
            results.append(oracle.gat_backward(op.indptr, op.col_local, h, halo, W, att, out,
                                               G, RELU))
    finally:
        oracle.set_num_threads(before)
    for other in results[1:]:
        for a, b in zip(results[0], other):
            np.testing.assert_array_equal(np.asarray(a).view(np.uint32),
                                          np.asarray(b).view(np.uint32))
