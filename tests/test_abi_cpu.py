"""Host-side checks of libdigest.so that need no GPU: every symbol of
include/digest.h is exported, the index maps built by digest_partition_create
match the oracle bit for bit, malformed inputs are rejected with the
documented status, calls before a workspace is bound fail with
DIGEST_ESTATE, and the schedule matches Algorithm 1.  No kernel is launched."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
from conftest import ROOT
from paper_2206_00057_amd import digest as D
from paper_2206_00057_amd import synth


def header_functions():
    text = open(os.path.join(ROOT, "include", "digest.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(digest_[a-z_]+)\s*\(", text)))


def test_library_exports_every_header_symbol():
    names = header_functions()
    assert len(names) >= 16
    L = D.lib()
    for n in names:
        assert hasattr(L, n), n


def _tiny_partition(part=0, cfg=None):
    cfg = cfg or synth.CONFIGS["tiny"]
    g = synth.make_graph(cfg)
    return cfg, g, synth.make_partition(cfg, g, part)


@pytest.mark.parametrize("part", [0, 3])
def test_maps_bit_exact_vs_oracle(part):
    cfg, g, p = _tiny_partition(part)
    h = D.digest_partition_create(g.n, p.indptr, p.indices, p.values, p.owned, p.halo, cfg.widths)
    col, bgid, bloc = D.digest_partition_export_maps(h)
    o_col, o_bnd = oracle.partition_maps(g.n, p.indptr, p.indices, p.owned, p.halo)
    np.testing.assert_array_equal(col, o_col)
    np.testing.assert_array_equal(bloc, o_bnd)
    np.testing.assert_array_equal(bgid, p.owned[o_bnd])
    t_ptr, t_src, t_val = D.digest_partition_export_transpose(h)
    o_ptr, o_src, o_val = oracle.owned_transpose(p.n_own, p.indptr, o_col, p.values)
    np.testing.assert_array_equal(t_ptr, o_ptr)
    np.testing.assert_array_equal(t_src, o_src)
    np.testing.assert_array_equal(t_val.view(np.uint32), o_val.view(np.uint32))
    assert h.nnz == p.nnz and h.nnz_in == o_ptr[-1] and h.n_boundary == o_bnd.size
    assert h.workspace_bytes > 0 and h.workspace_bytes % 256 == 0


def test_maps_with_duplicates_and_unreferenced_halo():
    # row 0: owned 0 twice (summed), halo 5; row 1: owned 0; halo 7 unreferenced
    indptr = np.array([0, 3, 4])
    indices = np.array([0, 0, 5, 0])
    values = np.array([0.5, 0.25, 1.0, 2.0], np.float32)
    owned, halo = np.array([0, 3]), np.array([5, 7])
    h = D.digest_partition_create(8, indptr, indices, values, owned, halo, [4, 4])
    col, bgid, bloc = D.digest_partition_export_maps(h)
    assert col.tolist() == [0, 0, 2, 0]
    assert bloc.tolist() == [0] and bgid.tolist() == [0]
    o_col, o_bnd = oracle.partition_maps(8, indptr, indices, owned, halo)
    assert o_col.tolist() == col.tolist() and o_bnd.tolist() == bloc.tolist()
    t_ptr, t_src, t_val = D.digest_partition_export_transpose(h)
    assert t_ptr.tolist() == [0, 3, 3] and t_src.tolist() == [0, 0, 1]
    assert t_val.tolist() == [0.5, 0.25, 2.0]


def test_empty_partition_is_valid():
    h = D.digest_partition_create(10, np.array([0]), np.zeros(0), np.zeros(0, np.float32),
                                  np.zeros(0), np.zeros(0), [3, 2])
    assert h.nnz == 0 and h.n_boundary == 0 and h.nnz_in == 0


def expect_status(status, fn, *a, **kw):
    with pytest.raises(D.DigestError) as e:
        fn(*a, **kw)
    assert e.value.status == status, str(e.value)


def test_create_rejects_malformed_input():
    cfg, g, p = _tiny_partition()
    mk = lambda **kw: D.digest_partition_create(
        kw.get("n", g.n), kw.get("indptr", p.indptr), kw.get("indices", p.indices),
        kw.get("values", p.values), kw.get("owned", p.owned), kw.get("halo", p.halo),
        kw.get("widths", cfg.widths))
    mk()
    E = D.EINVAL
    expect_status(E, mk, halo=p.halo[1:])                              # column not owned/halo
    expect_status(E, mk, halo=np.append(p.halo, p.owned[3]))           # owned and halo overlap
    expect_status(E, mk, owned=np.append(p.owned[:-1], p.owned[0]))    # repeated owned id
    expect_status(E, mk, halo=np.append(p.halo[:-1], p.halo[0]))       # repeated halo id
    expect_status(E, mk, n=int(max(p.halo.max(), p.owned.max())))      # id out of range
    bad = p.indptr.copy()
    bad[5] = bad[4] - 1
    expect_status(E, mk, indptr=bad)                                   # decreasing indptr
    bad = p.indptr.copy()
    bad[0] = 1
    expect_status(E, mk, indptr=bad)                                   # indptr[0] != 0
    expect_status(E, mk, widths=[64, 0, 16])                           # width 0
    expect_status(E, mk, widths=[64])                                  # no layer
    neg = p.indices.copy()
    neg[7] = -3
    expect_status(E, mk, indices=neg)                                  # negative id
    expect_status(E, mk, n=0)


def test_device_calls_without_workspace_fail_with_estate():
    cfg, g, p = _tiny_partition()
    h = D.digest_partition_create(g.n, p.indptr, p.indices, p.values, p.owned, p.halo, cfg.widths)
    L = D.lib()
    fake = ctypes.c_void_p(256)   # never dereferenced: the state check comes first
    assert L.digest_pull(h.handle, 0, fake, None) == D.ESTATE
    assert L.digest_push(h.handle, 1, fake, fake, 0, None) == D.ESTATE
    assert L.digest_layer_forward(h.handle, 1, fake, fake, fake, 0, None) == D.ESTATE
    assert L.digest_layer_backward(h.handle, 1, fake, fake, fake, fake, fake, None, None) == D.ESTATE
    assert L.digest_softmax_xent(h.handle, fake, fake, fake, fake, None) == D.ESTATE
    assert L.digest_halo_gradient(h.handle, 2, fake, fake, fake, fake, None) == D.ESTATE
    assert L.digest_push_add(h.handle, 1, fake, fake, None) == D.ESTATE
    assert L.digest_pull_add(h.handle, 1, fake, fake, None) == D.ESTATE
    assert L.digest_layer_backward_halo(h.handle, 2, fake, fake, fake, fake, fake, fake, fake,
                                        None) == D.ESTATE
    assert L.digest_halo_gradient(None, 2, fake, fake, fake, fake, None) == D.EINVAL
    assert L.digest_push_add(None, 1, fake, fake, None) == D.EINVAL
    assert L.digest_pull(None, 0, fake, None) == D.EINVAL
    assert b"workspace" in L.digest_last_error() or b"handle" in L.digest_last_error()
    # binding rejects misaligned or short workspaces before touching the device
    assert L.digest_partition_bind_workspace(h.handle, ctypes.c_void_p(4), 1 << 30, None) == D.EINVAL
    assert L.digest_partition_bind_workspace(h.handle, ctypes.c_void_p(256), 16, None) == D.ENOMEM


def test_sgd_average_rejects_bad_arguments_before_any_device_work():
    L = D.lib()
    fake = ctypes.c_void_p(256)   # never dereferenced: the checks come first
    ptrs = (ctypes.c_void_p * 65)(*([256] * 65))
    assert L.digest_sgd_average(fake, ptrs, 0, 10, ctypes.c_float(0.1), None) == D.EINVAL
    assert L.digest_sgd_average(fake, ptrs, 65, 10, ctypes.c_float(0.1), None) == D.EINVAL
    assert L.digest_sgd_average(fake, ptrs, 2, -1, ctypes.c_float(0.1), None) == D.EINVAL
    assert L.digest_sgd_average(None, ptrs, 2, 10, ctypes.c_float(0.1), None) == D.EINVAL
    nulls = (ctypes.c_void_p * 2)(256, None)
    assert L.digest_sgd_average(fake, nulls, 2, 10, ctypes.c_float(0.1), None) == D.EINVAL
    assert b"NULL" in L.digest_last_error()
    # nothing to update: no device work, OK
    assert L.digest_sgd_average(None, None, 1, 0, ctypes.c_float(0.1), None) == D.OK


def test_sync_period_matches_algorithm_and_oracle(golden):
    f = os.path.join(ROOT, "tests", "golden", "alg1_schedule.txt")
    for line in open(f):
        line = line.split("#", 1)[0].split()
        if line:
            K, r, pull, push = map(int, line)
            assert D.digest_sync_period(K, r) == (bool(pull), bool(push))
    for K in (1, 2, 3, 7, 10, 20):
        for r in range(1, 3 * K + 2):
            assert D.digest_sync_period(K, r) == oracle.sync_period(K, r)
    expect_status(D.EINVAL, D.digest_sync_period, 0, 1)
    expect_status(D.EINVAL, D.digest_sync_period, 4, 0)


def test_profile_kernel_names():
    names = D.kernel_names()
    assert len(names) == D.lib().digest_profile_kernel_count()
    assert "spmm_fwd" in names and "gemm_fwd_relu" in names and "pull_gather" in names


def test_launch_plan_and_cost_model():
    """The plan query reports the library's product order and split counts,
    and the per-launch cost model covers exactly the kinds a round launches,
    with the compulsory bytes of the copies and aggregations."""
    cfg, g, p = _tiny_partition(0)
    h = D.digest_partition_create(g.n, p.indptr, p.indices, p.values, p.owned, p.halo, cfg.widths)
    pl1, pl2 = D.digest_partition_plan(h, 1), D.digest_partition_plan(h, 2)
    assert pl1["transform_first"] == 0 and pl1["dw_slices"] >= 1   # ReLU layers aggregate first
    assert pl2["transform_first"] == 1   # 64 -> 16 identity: narrower gathers pay
    with pytest.raises(D.DigestError):
        D.digest_partition_plan(h, 0)
    with pytest.raises(D.DigestError):
        D.digest_partition_plan(h, cfg.layers + 1)
    n, nh, nb = p.n_own, p.n_halo, h.n_boundary
    assert 0 < nb < n and h.nnz_in < h.nnz
    # the forward's operand: the owned-column entries, plus one entry per
    # boundary row for its halo aggregate; the pull's: the halo entries
    nnz_s, nnz_b = h.nnz_in + nb, h.nnz - h.nnz_in
    gcn = D.digest_profile_model(h, D.MODEL_GCN)
    assert gcn["pull_gather.l0"][0] == 8 * nh * cfg.widths[0] + 4 * nh
    assert gcn["push_scatter.l1"][0] == 8 * nb * cfg.widths[1] + 8 * nb
    di, dh, do = cfg.widths
    for lev, d in ((0, di), (1, dh)):
        assert gcn[f"halo_aggregate.l{lev}"] == (
            4 * (nb + 1) + 8 * nnz_b + 4 * (nh + nb) * d, 0.0, nnz_b)
    assert gcn["spmm_fwd.l1"] == (4 * (n + 1) + 8 * nnz_s + 4 * (n + nb) * di + 4 * n * di, 0.0,
                                  nnz_s)
    assert gcn["gemm_fwd_relu.l1"][1] == 2.0 * n * di * cfg.widths[1]
    # the transform-first layer 2 multiplies the owned and the boundary rows
    assert gcn["gemm_fwd_relu.l2"][1] == 2.0 * (n + nb) * dh * do
    assert gcn["gemm_dw_splitk.l2"][1] == 2.0 * (n + nb) * dh * do
    assert gcn["spmm_bwd_transposed.l2"][2] == h.nnz_in
    assert gcn["boundary_rows.l2"][0] == 8 * nb * do + 4 * nb
    assert not any(k.startswith("gat_") for k in gcn)
    assert "softmax_xent.l2" in gcn and "loss_mean.l2" in gcn
    gat = D.digest_profile_model(h, D.MODEL_GAT)
    assert gat["gat_aggregate.l2"][2] == h.nnz and "spmm_fwd.l1" not in gat
    assert not any(k.startswith("halo_aggregate") for k in gat)
    L = D.lib()
    buf = (ctypes.c_double * 1000)()
    cnt = (ctypes.c_int64 * 1000)()
    assert L.digest_profile_model(h.handle, 7, buf, buf, cnt) == D.EINVAL
    assert L.digest_profile_model(h.handle, 0, None, buf, cnt) == D.EINVAL


def test_pull_mode_and_its_cost_model():
    """The aggregate-only pull mode drops the pull's row gather from the cost
    model (the halo aggregate reads the store instead); unknown modes and a
    NULL handle are refused."""
    cfg, g, p = _tiny_partition(0)
    h = D.digest_partition_create(g.n, p.indptr, p.indices, p.values, p.owned, p.halo, cfg.widths)
    rows = D.digest_profile_model(h, D.MODEL_GCN)
    assert "pull_gather.l0" in rows and "halo_aggregate.l0" in rows
    D.digest_partition_set_pull_mode(h, D.PULL_AGGREGATE)
    agg = D.digest_profile_model(h, D.MODEL_GCN)
    assert not any(k.startswith("pull_gather") for k in agg)
    assert agg["halo_aggregate.l1"] == rows["halo_aggregate.l1"]
    D.digest_partition_set_pull_mode(h, D.PULL_ROWS)
    assert "pull_gather.l1" in D.digest_profile_model(h, D.MODEL_GCN)
    for bad in (-1, 2, 7):
        expect_status(D.EINVAL, D.digest_partition_set_pull_mode, h, bad)
    assert D.lib().digest_partition_set_pull_mode(None, D.PULL_ROWS) == D.EINVAL


def test_tier_plan_follows_the_overrides(monkeypatch):
    """Tiers are planned at create: a forced count with a small L2 budget
    gives that many tiers of budget / 128 rows (256-wide rows: one 32-float
    slice per XCD), a zero budget none; the tiers' entries are part of the
    operand."""
    widths = [256, 256, 7]
    cfg = synth.scaled(synth.CONFIGS["tiny"], 2000, widths=widths, classes=7)
    g = synth.make_graph(cfg)
    p = synth.make_partition(cfg, g, 0)
    monkeypatch.setenv("DIGEST_SPMM_TIERS", "2")
    monkeypatch.setenv("DIGEST_SPMM_TIER_BYTES", "4096")
    h = D.digest_partition_create(g.n, p.indptr, p.indices, p.values, p.owned, p.halo, widths)
    pl = D.digest_partition_plan(h, 1)
    assert pl["tiers_fwd"] == 2 and pl["tier_rows_fwd"] == 32
    assert 0 < pl["tier_entries_fwd"] < h.nnz
    pl2 = D.digest_partition_plan(h, 2)
    if not pl2["transform_first"]:
        assert pl2["tiers_bwd"] == 2 and 0 < pl2["tier_entries_bwd"] < h.nnz_in
    monkeypatch.setenv("DIGEST_SPMM_TIER_BYTES", "0")
    h0 = D.digest_partition_create(g.n, p.indptr, p.indices, p.values, p.owned, p.halo, widths)
    assert D.digest_partition_plan(h0, 1)["tiers_fwd"] == 0
    assert h0.workspace_bytes < h.workspace_bytes


def test_fused_forward_plan_and_cost_model(monkeypatch):
    """The fused forward is planned for aggregate-first layers of 65..256
    input floats whose product is the MFMA GEMM, at 16,384 owned rows or
    more (DIGEST_FUSE=2: any count, 0: never); its cost model splits the
    aggregation at 64 entries per row into the long-row pass and the fused
    pass (entries, distinct sources, the long rows read back, the short
    rows' AH written, W, the output) and drops the separate GEMM."""
    widths = [256, 256, 7]
    cfg = synth.scaled(synth.CONFIGS["large"], 4000, widths=widths, classes=7)
    g = synth.make_graph(cfg, seed=7)
    p = synth.make_partition(cfg, g, 1)

    def create():
        return D.digest_partition_create(g.n, p.indptr, p.indices, p.values, p.owned, p.halo,
                                         widths)

    monkeypatch.delenv("DIGEST_FUSE", raising=False)
    h = create()
    assert D.digest_partition_plan(h, 1)["forward_fused"] == 0   # too few rows
    monkeypatch.setenv("DIGEST_FUSE", "2")
    assert D.digest_partition_plan(h, 1)["forward_fused"] == 1
    assert D.digest_partition_plan(h, 2)["forward_fused"] == 0   # 7 outputs: narrow product
    # the forward's operand: row i's owned-column entries, then, for a row
    # with halo entries (boundary row b), one entry reading column n_own + b
    n = p.n_own
    pos = {int(v): i for i, v in enumerate(p.owned)}
    rows = np.repeat(np.arange(n), np.diff(p.indptr))
    local = np.array([pos.get(int(c), -1) for c in p.indices])
    inn = local >= 0
    bnd = np.unique(rows[~inn])
    s_rows = np.concatenate([rows[inn], bnd])
    s_cols = np.concatenate([local[inn], n + np.arange(bnd.size)])
    lens = np.bincount(s_rows, minlength=n)
    assert lens.sum() == h.nnz_in + h.n_boundary
    long_rows = lens > 64
    assert long_rows.any() and (~long_rows).any()
    src_short = np.unique(s_cols[~long_rows[s_rows]]).size
    src_long = np.unique(s_cols[long_rows[s_rows]]).size
    di, do = widths[0], widths[1]
    nl, el = int(long_rows.sum()), int(lens[long_rows].sum())
    nnz_s = int(lens.sum())
    m = D.digest_profile_model(h, D.MODEL_GCN)
    assert "gemm_fwd_relu.l1" not in m
    assert m["spmm_fwd.l1"] == (8 * nl + 8 * el + 4 * src_long * di + 4 * nl * di, 0.0, el)
    assert m["spmm_gemm_fwd.l1"] == (
        4 * (n + 1) + 8 * (nnz_s - el) + 4 * src_short * di + 4 * nl * di + 4 * (n - nl) * di +
        4 * di * do + 4 * n * do, 2.0 * n * di * do, nnz_s - el)
    monkeypatch.setenv("DIGEST_FUSE", "0")
    assert D.digest_partition_plan(h, 1)["forward_fused"] == 0
    assert "gemm_fwd_relu.l1" in D.digest_profile_model(h, D.MODEL_GCN)


def test_fused_input_gradient_plan_and_cost_model(monkeypatch):
    """The input gradient of a ReLU aggregate-first layer >= 2 with 65..256
    output floats is planned as one fused pass over P_in^T (rows split at 64
    entries) after D is formed once; the weight gradient then reads D
    without the mask, and the separate input-gradient GEMM is gone."""
    widths = [100, 256, 256, 7]
    cfg = synth.scaled(synth.CONFIGS["large"], 4000, widths=widths, classes=7)
    g = synth.make_graph(cfg, seed=7)
    p = synth.make_partition(cfg, g, 1)
    monkeypatch.setenv("DIGEST_FUSE", "2")
    h = D.digest_partition_create(g.n, p.indptr, p.indices, p.values, p.owned, p.halo, widths)
    assert D.digest_partition_plan(h, 2)["backward_fused"] == 1
    assert D.digest_partition_plan(h, 1)["backward_fused"] == 0   # no input gradient
    assert D.digest_partition_plan(h, 3)["backward_fused"] == 0   # identity layer
    # P_in^T: the owned-to-owned entries, by source row
    pos = {int(v): i for i, v in enumerate(p.owned)}
    rows = np.repeat(np.arange(p.n_own), np.diff(p.indptr))
    inn = np.array([int(c) in pos for c in p.indices])
    src = rows[inn]
    dst = np.array([pos[int(c)] for c in p.indices[inn]])
    lens = np.bincount(dst, minlength=p.n_own)
    long_rows = lens > 64
    assert long_rows.any() and (~long_rows).any()
    src_short = np.unique(src[~long_rows[dst]]).size
    src_long = np.unique(src[long_rows[dst]]).size
    n, di, do = p.n_own, widths[1], widths[2]
    nl, el = int(long_rows.sum()), int(lens[long_rows].sum())
    m = D.digest_profile_model(h, D.MODEL_GCN)
    assert "gemm_dgrad.l2" not in m
    assert m["relu_mask.l2"][0] == 12 * n * do and m["transpose_w.l2"][0] == 8 * di * do
    assert m["spmm_bwd_transposed.l2"] == (8 * nl + 8 * el + 4 * src_long * do + 4 * nl * do,
                                           0.0, el)
    assert m["spmm_gemm_bwd.l2"] == (
        4 * (n + 1) + 8 * (h.nnz_in - el) + 4 * src_short * do + 4 * nl * do + 4 * di * do +
        4 * n * di, 2.0 * n * di * do, h.nnz_in - el)
    assert m["gemm_dw_splitk.l2"][0] == 4 * (n * di + n * do + di * do)
    monkeypatch.setenv("DIGEST_FUSE", "0")
    assert D.digest_partition_plan(h, 2)["backward_fused"] == 0
    assert "gemm_dgrad.l2" in D.digest_profile_model(h, D.MODEL_GCN)
    # rows of 65..128 floats are fused too (two lane groups per row), rows of
    # 64 floats or fewer go to the narrow kernels
    monkeypatch.setenv("DIGEST_FUSE", "2")
    for d_in, fused in ((100, 1), (65, 1), (64, 0)):
        h2 = D.digest_partition_create(g.n, p.indptr, p.indices, p.values, p.owned, p.halo,
                                       [d_in, 256, 7])
        assert D.digest_partition_plan(h2, 1)["forward_fused"] == fused, d_in
