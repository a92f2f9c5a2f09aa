"""GPU parity of every library call against the CPU oracle, on identical
seeded inputs from ``paper_2206_00057_amd.synth`` (no oracle input ever comes
from the GPU).

Bars: index maps, pull and push contents bit-exact; activations, gradients
and the loss within rtol 1e-4 / atol 1e-5 element-wise, plus a scale-aware
bound max|gpu - oracle| / max|oracle| (gradients scale like 1/n_own, where
atol alone says little).  Cases span several tiles with ragged tails, odd
widths, rows longer than one aggregation work item, an empty partition, a
partition without halo, and the small GCN workload end to end over several
rounds of Algorithm 1 with sync intervals 1 and 5.
"""
import numpy as np
import pytest

import oracle
from paper_2206_00057_amd import synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

RTOL, ATOL = 1e-4, 1e-5
SCALE_TOL = 2e-5


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def D():
    from paper_2206_00057_amd import digest
    return digest


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host(t):
    torch.cuda.synchronize()
    return t.detach().cpu().numpy()


def assert_close(gpu, ref, name, rtol=RTOL, atol=ATOL, scale_tol=SCALE_TOL):
    g = np.asarray(gpu, np.float64)
    r = np.asarray(ref, np.float64)
    assert g.shape == r.shape, name
    assert np.all(np.isfinite(g)), f"{name}: non-finite GPU values"
    err = np.abs(g - r)
    bad = err > atol + rtol * np.abs(r)
    peak = float(np.abs(r).max()) if r.size else 0.0
    scale = float(err.max()) / peak if r.size and peak > 0 else 0.0
    assert not bad.any(), (f"{name}: {int(bad.sum())}/{bad.size} outside rtol/atol, "
                           f"max err {err.max():.3e}, scale err {scale:.3e}")
    assert scale <= scale_tol, f"{name}: scale err {scale:.3e} > {scale_tol}"
    return scale


def assert_bits(gpu, ref, name):
    g = np.ascontiguousarray(gpu)
    r = np.ascontiguousarray(ref)
    assert g.shape == r.shape, name
    np.testing.assert_array_equal(g.view(np.uint32), r.view(np.uint32), err_msg=name)


class Case:
    """A partition with its library handle, oracle twin and seeded inputs."""

    def __init__(self, cfg, g, part, label="", ws_fill=None):
        self.cfg, self.g, self.part = cfg, g, part
        self.label = label or cfg.name
        self.widths = list(cfg.widths)
        self.L = len(self.widths) - 1
        Dm = D()
        self.h = Dm.digest_partition_create(g.n, part.indptr, part.indices, part.values,
                                            part.owned, part.halo, self.widths)
        self.ws = torch.empty(max(self.h.workspace_bytes, 256), dtype=torch.uint8, device="cuda")
        if ws_fill is not None:   # every workspace byte set before the library writes any
            self.ws.fill_(ws_fill)
        Dm.digest_partition_bind_workspace(self.h, self.ws)
        self.op = oracle.OraclePartition(g.n, part.indptr, part.indices, part.values,
                                         part.owned, part.halo, self.widths)
        self.n = part.n_own

    def store(self, level):
        if level == 0:
            return synth.features(self.cfg)
        return synth.relu_normal((self.g.n, self.widths[level]), seed=20 + level)

    def layer_input(self, layer):
        if layer == 1:
            return synth.features(self.cfg)[self.part.owned]
        return synth.relu_normal((self.n, self.widths[layer - 1]), seed=10 + layer)

    def upstream(self, layer):
        return synth.normal((self.n, self.widths[layer]), seed=30 + layer,
                            scale=1.0 / max(self.n, 1))

    def act(self, layer):
        return oracle.RELU if layer < self.L else oracle.IDENTITY


def check_pull(c, level, store=None):
    Dm = D()
    store = c.store(level) if store is None else store
    Dm.digest_pull(c.h, level, dev(store))
    out = torch.empty(c.part.n_halo, c.widths[level], device="cuda")
    Dm.digest_partition_read_halo(c.h, level, out)
    assert_bits(host(out), c.op.pull(level, store), f"{c.label} pull level {level}")


def check_push(c, level):
    Dm = D()
    base = synth.normal((c.g.n, c.widths[level]), seed=40 + level)
    h_own = synth.normal((c.n, c.widths[level]), seed=50 + level)
    for mode, all_owned in ((Dm.PUSH_BOUNDARY, False), (Dm.PUSH_ALL_OWNED, True)):
        s = dev(base)
        Dm.digest_push(c.h, level, dev(h_own), s, mode)
        ref = c.op.push(level, h_own, base.copy(), all_owned=all_owned)
        assert_bits(host(s), ref, f"{c.label} push level {level} mode {mode}")


def check_layer(c, layer, check_dh_in=True):
    """Forward and backward of one layer on seeded inputs, vs the oracle."""
    Dm = D()
    if c.part.n_halo:
        store = c.store(layer - 1)
        Dm.digest_pull(c.h, layer - 1, dev(store))
        c.op.pull(layer - 1, store)
    h_in = c.layer_input(layer)
    W = synth.weights(c.cfg)[layer - 1]
    act = c.act(layer)
    out = torch.empty(c.n, c.widths[layer], device="cuda")
    Dm.digest_layer_forward(c.h, layer, dev(h_in), dev(W), out, act)
    ref_out = c.op.forward(layer, h_in, W, act)
    assert_close(host(out), ref_out, f"{c.label} forward layer {layer}")
    # backward: mask and upstream gradient from the oracle / the generator
    dh = c.upstream(layer)
    dw = torch.empty(W.shape, device="cuda")
    want = check_dh_in and layer > 1
    dh_in = torch.empty(c.n, c.widths[layer - 1], device="cuda") if want else None
    Dm.digest_layer_backward(c.h, layer, dev(h_in), dev(ref_out), dev(dh), dev(W), dw, dh_in)
    ref_dw, ref_dh_in = c.op.backward(layer, h_in, W, ref_out, dh, act, want_dh_in=want)
    assert_close(host(dw), ref_dw, f"{c.label} dW layer {layer}")
    if want:
        assert_close(host(dh_in), ref_dh_in, f"{c.label} dH_in layer {layer}")


def check_loss(c, seed=60):
    Dm = D()
    C = c.widths[-1]
    logits = synth.normal((c.n, C), seed=seed, scale=3.0)
    y = synth.labels(c.cfg)[c.part.owned]
    dl = torch.empty(c.n, C, device="cuda")
    loss = torch.empty(1, device="cuda")
    Dm.digest_softmax_xent(c.h, dev(logits), dev(y), dl, loss)
    ref_loss, ref_dl = oracle.softmax_xent(logits, y)
    assert_close(host(dl), ref_dl, f"{c.label} dlogits")
    assert abs(float(host(loss)[0]) - ref_loss) <= ATOL + RTOL * abs(ref_loss)


# ---------------------------------------------------------------------------
# the small GCN workload (2,000 nodes, 64 -> 64 -> 16), every call
# ---------------------------------------------------------------------------

@pytest.fixture(scope="module")
def tiny_graph():
    cfg = synth.CONFIGS["tiny"]
    return cfg, synth.make_graph(cfg)


@pytest.fixture(scope="module", params=[0, 3])
def tiny(request, tiny_graph):
    cfg, g = tiny_graph
    return Case(cfg, g, synth.make_partition(cfg, g, request.param),
                label=f"tiny/part{request.param}")


def test_tiny_pull_push_bit_exact(tiny):
    for level in range(tiny.L):
        check_pull(tiny, level)
    for level in range(1, tiny.L):
        check_push(tiny, level)


@pytest.mark.parametrize("layer", [1, 2])
def test_tiny_layer(tiny, layer):
    check_layer(tiny, layer)


def test_tiny_loss(tiny):
    # repeated calls on one handle reuse its loss partials
    for seed in (60, 62, 63):
        check_loss(tiny, seed)


def test_tiny_bad_label_gives_nan_and_zero_rows(tiny):
    Dm = D()
    C = tiny.widths[-1]
    logits = synth.normal((tiny.n, C), seed=61)
    y = synth.labels(tiny.cfg)[tiny.part.owned].copy()
    y[5] = C
    dl = torch.full((tiny.n, C), 7.0, device="cuda")
    loss = torch.empty(1, device="cuda")
    Dm.digest_softmax_xent(tiny.h, dev(logits), dev(y), dl, loss)
    assert np.isnan(host(loss)[0])
    out = host(dl)
    assert np.all(out[5] == 0)
    ref_loss, ref_dl = oracle.softmax_xent(logits[np.arange(tiny.n) != 5],
                                           y[np.arange(tiny.n) != 5])
    # the other rows keep their value (normalised by the full row count)
    assert_close(out[np.arange(tiny.n) != 5] * tiny.n,
                 ref_dl * (tiny.n - 1), "dlogits with one bad label")


def test_determinism_bitwise(tiny):
    Dm = D()
    store = tiny.store(0)
    Dm.digest_pull(tiny.h, 0, dev(store))
    x = dev(tiny.layer_input(1))
    W = dev(synth.weights(tiny.cfg)[0])
    outs, dws = [], []
    for _ in range(2):
        out = torch.empty(tiny.n, tiny.widths[1], device="cuda")
        Dm.digest_layer_forward(tiny.h, 1, x, W, out, Dm.ACT_RELU)
        dw = torch.empty(W.shape, device="cuda")
        Dm.digest_layer_backward(tiny.h, 1, x, out, dev(tiny.upstream(1)), W, dw, None)
        outs.append(host(out))
        dws.append(host(dw))
    assert_bits(outs[0], outs[1], "forward run twice")
    assert_bits(dws[0], dws[1], "dW run twice")


# ---------------------------------------------------------------------------
# shapes: odd widths, ragged tiles, long rows, empty and halo-free partitions
# ---------------------------------------------------------------------------

WIDTHS = [(1, 1, 1), (3, 5, 2), (7, 41, 47), (602, 47, 7), (100, 256, 41), (64, 64, 16),
          (33, 130, 9), (500, 256, 7), (16, 24, 70), (20, 40, 100), (8, 12, 130),
          (8, 40, 24), (8, 100, 60)]


@pytest.mark.parametrize("widths", WIDTHS, ids=lambda w: "x".join(map(str, w)))
def test_widths(widths):
    cfg = synth.scaled(synth.CONFIGS["tiny"], 1200, widths=widths, classes=widths[-1])
    g = synth.make_graph(cfg, seed=1)
    c = Case(cfg, g, synth.make_partition(cfg, g, 1), label=f"widths{widths}")
    for level in range(c.L):
        check_pull(c, level)
    for layer in (1, 2):
        check_layer(c, layer)
    check_loss(c)


def test_long_rows_split_into_items():
    """Rows with more entries than one work item (lognormal, mean ~490)."""
    cfg = synth.scaled(synth.CONFIGS["dense"], 8000, widths=(96, 40, 5), classes=5)
    g = synth.make_graph(cfg, seed=2)
    part = synth.make_partition(cfg, g, 0)
    assert np.diff(part.indptr).max() > 1000
    c = Case(cfg, g, part, label="long-rows")
    for layer in (1, 2):
        check_layer(c, layer)


def test_relu_narrowing_layer_uses_masked_dgrad():
    cfg = synth.scaled(synth.CONFIGS["tiny"], 1200, widths=(48, 20, 3), classes=3)
    g = synth.make_graph(cfg, seed=4)
    c = Case(cfg, g, synth.make_partition(cfg, g, 2), label="relu-narrow")
    check_layer(c, 1, check_dh_in=True)
    # dh_in of layer 1 (ReLU, narrowing) is also defined by the API
    Dm = D()
    h_in = c.layer_input(1)
    W = synth.weights(cfg)[0]
    out = torch.empty(c.n, 20, device="cuda")
    Dm.digest_layer_forward(c.h, 1, dev(h_in), dev(W), out, Dm.ACT_RELU)
    ref_out = c.op.forward(1, h_in, W, oracle.RELU)
    dh = c.upstream(1)
    dw = torch.empty(W.shape, device="cuda")
    dh_in = torch.empty(c.n, 48, device="cuda")
    Dm.digest_layer_backward(c.h, 1, dev(h_in), dev(ref_out), dev(dh), dev(W), dw, dh_in)
    ref_dw, ref_dh = c.op.backward(1, h_in, W, ref_out, dh, oracle.RELU, want_dh_in=True)
    assert_close(host(dh_in), ref_dh, "relu-narrow dH_in")


def test_single_partition_no_halo():
    cfg = synth.scaled(synth.CONFIGS["tiny"], 900, widths=(16, 24, 5), classes=5)
    g = synth.make_graph(cfg, seed=6)
    part = synth.extract_partition(g, np.arange(g.n, dtype=np.int64))
    assert part.n_halo == 0
    c = Case(cfg, g, part, label="no-halo")
    assert c.h.n_boundary == 0
    for layer in (1, 2):
        check_layer(c, layer)


def test_halo_aggregate_follows_pulls():
    """The halo rows reach the GCN forward through their aggregate, formed
    when a level is pulled: a second pull from another store changes the
    next forward and backward, a store written after the pull does not
    (the rows are stale until the next pull), and a partition with a GAT
    workspace (whose pulls skip the aggregate) forms it in the forward.
    Layer 1 aggregates first (ReLU), layer 2 multiplies first (identity)."""
    Dm = D()
    cfg = synth.scaled(synth.CONFIGS["tiny"], 1500, widths=(36, 40, 12), classes=12)
    g = synth.make_graph(cfg, seed=9)
    c = Case(cfg, g, synth.make_partition(cfg, g, 2), label="halo-aggregate", ws_fill=255)
    assert 0 < c.h.n_boundary < c.n
    assert Dm.digest_partition_plan(c.h, 1)["transform_first"] == 0
    assert Dm.digest_partition_plan(c.h, 2)["transform_first"] == 1

    def run(layer, store, label, write_after=None):
        gstore = dev(store)
        Dm.digest_pull(c.h, layer - 1, gstore)
        c.op.pull(layer - 1, store)
        if write_after is not None:   # the store changes, the pulled rows do not
            gstore.copy_(dev(write_after))
        h_in = c.layer_input(layer)
        W = synth.weights(c.cfg)[layer - 1]
        act = c.act(layer)
        out = torch.empty(c.n, c.widths[layer], device="cuda")
        Dm.digest_layer_forward(c.h, layer, dev(h_in), dev(W), out, act)
        ref_out = c.op.forward(layer, h_in, W, act)
        assert_close(host(out), ref_out, f"{label} forward layer {layer}")
        dh = c.upstream(layer)
        dw = torch.empty(W.shape, device="cuda")
        dh_in = torch.empty(c.n, c.widths[layer - 1], device="cuda") if layer > 1 else None
        Dm.digest_layer_backward(c.h, layer, dev(h_in), dev(ref_out), dev(dh), dev(W), dw,
                                 dh_in)
        ref_dw, ref_dh_in = c.op.backward(layer, h_in, W, ref_out, dh, act,
                                          want_dh_in=layer > 1)
        assert_close(host(dw), ref_dw, f"{label} dW layer {layer}")
        if layer > 1:
            assert_close(host(dh_in), ref_dh_in, f"{label} dH_in layer {layer}")

    for layer in (1, 2):
        a = synth.relu_normal((g.n, c.widths[layer - 1]), seed=70 + layer)
        b = synth.relu_normal((g.n, c.widths[layer - 1]), seed=75 + layer) + 0.5
        run(layer, a, "first pull")
        run(layer, b, "second pull", write_after=a)
    gat_ws = torch.empty(max(Dm.digest_gat_query(c.h), 256), dtype=torch.uint8, device="cuda")
    Dm.digest_gat_bind_workspace(c.h, gat_ws)
    for layer in (1, 2):
        a = synth.relu_normal((g.n, c.widths[layer - 1]), seed=80 + layer)
        run(layer, a, "GAT workspace bound")


def test_pull_aggregate_mode():
    """In the aggregate-only pull mode a pull forms the halo aggregate from
    the store's rows (here 42 floats wide, not a multiple of 4) and keeps no
    halo rows: forward and backward (with the halo gradient too) still match
    the oracle after each pull, the calls that read halo rows refuse, and
    switching back to the rows mode needs a new pull."""
    Dm = D()
    cfg = synth.scaled(synth.CONFIGS["tiny"], 1500, widths=(36, 42, 12), classes=12)
    g = synth.make_graph(cfg, seed=9)
    c = Case(cfg, g, synth.make_partition(cfg, g, 2), label="pull-aggregate", ws_fill=255)
    assert 0 < c.h.n_boundary < c.n
    assert Dm.digest_partition_plan(c.h, 2)["transform_first"] == 1
    Dm.digest_partition_set_pull_mode(c.h, Dm.PULL_AGGREGATE)
    for layer in (1, 2):
        check_layer(c, layer)   # pulls store(layer - 1) first
        b = synth.relu_normal((g.n, c.widths[layer - 1]), seed=85 + layer) + 0.25
        Dm.digest_pull(c.h, layer - 1, dev(b))
        c.op.pull(layer - 1, b)
        h_in = c.layer_input(layer)
        W = synth.weights(c.cfg)[layer - 1]
        out = torch.empty(c.n, c.widths[layer], device="cuda")
        Dm.digest_layer_forward(c.h, layer, dev(h_in), dev(W), out, c.act(layer))
        ref = c.op.forward(layer, h_in, W, c.act(layer))
        assert_close(host(out), ref, f"second pull forward layer {layer}")
    # the halo variant of the (transform-first) backward needs no halo rows
    h_in = c.layer_input(2)
    W = synth.weights(c.cfg)[1]
    ref = c.op.forward(2, h_in, W, c.act(2))
    dh = c.upstream(2)
    dw = torch.empty(W.shape, device="cuda")
    dh_in = torch.empty(c.n, c.widths[1], device="cuda")
    dh_halo = torch.full((c.part.n_halo, c.widths[1]), float("nan"), device="cuda")
    Dm.digest_layer_backward_halo(c.h, 2, dev(h_in), dev(ref), dev(dh), dev(W), dw, dh_in,
                                  dh_halo)
    ref_dw, ref_dh = c.op.backward(2, h_in, W, ref, dh, c.act(2), want_dh_in=True)
    assert_close(host(dw), ref_dw, "aggregate mode, halo variant dW")
    assert_close(host(dh_in), ref_dh, "aggregate mode, halo variant dH_in")
    assert_close(host(dh_halo), c.op.halo_gradient(2, W, ref, dh, c.act(2)),
                 "aggregate mode, halo gradient")
    # the calls that read halo rows refuse
    with pytest.raises(Dm.DigestError) as e:
        Dm.digest_partition_read_halo(c.h, 1, torch.empty(c.part.n_halo, c.widths[1],
                                                           device="cuda"))
    assert e.value.status == Dm.ESTATE
    gat_ws = torch.empty(max(Dm.digest_gat_query(c.h), 256), dtype=torch.uint8, device="cuda")
    Dm.digest_gat_bind_workspace(c.h, gat_ws)
    att = synth.normal((c.widths[1], 2), seed=5)
    with pytest.raises(Dm.DigestError) as e:
        Dm.digest_gat_forward(c.h, 1, dev(c.layer_input(1)), dev(synth.weights(c.cfg)[0]),
                              dev(att), torch.empty(c.n, c.widths[1], device="cuda"),
                              Dm.ACT_RELU)
    assert e.value.status == Dm.ESTATE
    # back to the rows mode: every level must be pulled again
    Dm.digest_partition_set_pull_mode(c.h, Dm.PULL_ROWS)
    with pytest.raises(Dm.DigestError) as e:
        Dm.digest_layer_forward(c.h, 2, dev(h_in), dev(W), torch.empty(c.n, c.widths[2],
                                                                       device="cuda"),
                                c.act(2))
    assert e.value.status == Dm.ESTATE
    check_pull(c, 1)
    check_layer(c, 2)


# ReLU layers computed transform-first, relu(P_s (H W)), where the output
# is much narrower than the input: 600 -> 62 (D formed once, padded to 64
# floats) and 300 -> 11 (the narrow epilogue writes dH_in from the gather of
# D's 11 columns, rows 12 floats apart)
RELU_TF = [(24, 600, 62, 7), (24, 300, 11, 5)]


@pytest.mark.parametrize("widths", RELU_TF, ids=lambda w: "x".join(map(str, w)))
def test_relu_transform_first(widths):
    Dm = D()
    cfg = synth.scaled(synth.CONFIGS["tiny"], 1500, widths=widths, classes=widths[-1])
    g = synth.make_graph(cfg, seed=6)
    c = Case(cfg, g, synth.make_partition(cfg, g, 1), label=f"relu-tf{widths}", ws_fill=255)
    pl = Dm.digest_partition_plan(c.h, 2)
    assert pl["transform_first"] == 1 and c.act(2) == oracle.RELU
    assert pl["dgrad_fused"] == (1 if widths[2] <= 16 else 0)
    for layer in range(1, c.L + 1):
        check_layer(c, layer)
    Dm.digest_partition_set_pull_mode(c.h, Dm.PULL_AGGREGATE)
    check_layer(c, 2)


def test_empty_partition():
    Dm = D()
    h = Dm.digest_partition_create(10, np.array([0]), np.zeros(0), np.zeros(0, np.float32),
                                   np.zeros(0), np.zeros(0), [3, 2])
    ws = torch.empty(max(h.workspace_bytes, 256), dtype=torch.uint8, device="cuda")
    Dm.digest_partition_bind_workspace(h, ws)
    Dm.digest_pull(h, 0, torch.zeros(10, 3, device="cuda"))
    e = torch.empty(0, 3, device="cuda")
    out = torch.empty(0, 2, device="cuda")
    W = torch.ones(3, 2, device="cuda")
    Dm.digest_layer_forward(h, 1, e, W, out, Dm.ACT_IDENTITY)
    dw = torch.full((3, 2), 5.0, device="cuda")
    Dm.digest_layer_backward(h, 1, e, out, out, W, dw, e)
    assert np.all(host(dw) == 0)
    loss = torch.full((1,), 3.0, device="cuda")
    Dm.digest_softmax_xent(h, out, torch.empty(0, dtype=torch.int32, device="cuda"), out, loss)
    assert host(loss)[0] == 0


def test_state_errors_on_device():
    Dm = D()
    cfg = synth.CONFIGS["tiny"]
    g = synth.make_graph(cfg)
    part = synth.make_partition(cfg, g, 0)
    c = Case(cfg, g, part)
    W = dev(synth.weights(cfg)[1])
    x = torch.zeros(c.n, 64, device="cuda")
    out = torch.empty(c.n, 16, device="cuda")
    with pytest.raises(Dm.DigestError) as e:       # level 1 never pulled
        Dm.digest_layer_forward(c.h, 2, x, W, out, Dm.ACT_IDENTITY)
    assert e.value.status == Dm.ESTATE
    with pytest.raises(Dm.DigestError) as e:       # no forward of layer 2 yet
        Dm.digest_layer_backward(c.h, 2, x, out, out, W, torch.empty(64, 16, device="cuda"), None)
    assert e.value.status == Dm.ESTATE
    # a pull of level 1 between the forward and the backward of layer 2
    store1 = torch.zeros(g.n, 64, device="cuda")
    Dm.digest_pull(c.h, 1, store1)
    Dm.digest_layer_forward(c.h, 2, x, W, out, Dm.ACT_IDENTITY)
    dw = torch.empty(64, 16, device="cuda")
    Dm.digest_layer_backward(c.h, 2, x, out, out, W, dw, None)   # fine
    Dm.digest_pull(c.h, 1, store1)
    with pytest.raises(Dm.DigestError) as e:
        Dm.digest_layer_backward(c.h, 2, x, out, out, W, dw, None)
    assert e.value.status == Dm.ESTATE
    with pytest.raises(Dm.DigestError) as e:       # push of level 0 is not a stale level
        Dm.digest_push(c.h, 0, x, torch.zeros(g.n, 64, device="cuda"))
    assert e.value.status == Dm.EINVAL


# ---------------------------------------------------------------------------
# Algorithm 1 over several rounds (the small workload), sync interval 1 and 5
# ---------------------------------------------------------------------------

def _full_forward_oracle(g, X, Ws, L):
    allp = oracle.OraclePartition(g.n, g.indptr, g.indices, g.values,
                                  np.arange(g.n, dtype=np.int64), np.zeros(0, np.int64),
                                  [X.shape[1]] + [w.shape[1] for w in Ws])
    hs = [X]
    for l in range(1, L + 1):
        hs.append(allp.forward(l, hs[-1], Ws[l - 1], oracle.RELU if l < L else oracle.IDENTITY))
    return hs


@pytest.mark.parametrize("overlap_io", [False, True], ids=["in-line-io", "overlapped-io"])
@pytest.mark.parametrize("K", [1, 5])
def test_rounds_of_algorithm1(tiny_graph, K, overlap_io):
    """Each side runs its own rounds: the other partitions are played by a
    full-graph forward at the current weights whose boundary rows are pushed
    at every push round; the partition itself pulls/pushes per the schedule
    and applies SGD.  Compared round by round."""
    from paper_2206_00057_amd import step
    Dm = D()
    cfg, g = tiny_graph
    part = synth.make_partition(cfg, g, 0)
    L = cfg.layers
    X = synth.features(cfg)
    Ws = synth.weights(cfg)
    y = synth.labels(cfg)[part.owned]
    lr = 0.5
    # shared start: stores initialised by one full-graph forward at the initial W
    init = _full_forward_oracle(g, X, Ws, L)
    o_stores = [X] + [init[l].copy() for l in range(1, L)]
    g_stores = [dev(X)] + [dev(init[l]) for l in range(1, L)]
    op = oracle.OraclePartition(g.n, part.indptr, part.indices, part.values, part.owned,
                                part.halo, cfg.widths)
    gp = step.GpuPartition(g.n, part, cfg.widths, overlap_io=overlap_io)
    for lev in range(L):
        op.pull(lev, o_stores[lev])
    gp.pull_all(g_stores)
    oW = [w.copy() for w in Ws]
    gW = [dev(w) for w in Ws]
    x_own = X[part.owned]
    gx = dev(x_own)
    gy = dev(y)
    others = np.setdiff1d(np.arange(g.n), part.owned)
    for r in range(1, 3 * K + 2):
        do_pull, do_push = Dm.digest_sync_period(K, r)
        assert (do_pull, do_push) == oracle.sync_period(K, r)
        if do_push:   # the other partitions push their rows computed at the current W
            o_full = _full_forward_oracle(g, X, oW, L)
            for l in range(1, L):
                o_stores[l][others] = o_full[l][others]
            # the GPU side gets the same emulated rows from its own weights, via the library
            gfull = step.GpuPartition(g.n, synth.extract_partition(g, np.arange(g.n)), cfg.widths)
            gfull.pull_all([dev(X)] + [torch.zeros(g.n, cfg.widths[l], device="cuda")
                                       for l in range(1, L)])
            gfull.forward(dev(X), gW)
            idx = torch.from_numpy(others).cuda()
            for l in range(1, L):
                g_stores[l][idx] = gfull.H[l][idx]
        # oracle round
        h = x_own
        outs = []
        for l in range(1, L + 1):
            if do_pull and l >= 2:
                op.pull(l - 1, o_stores[l - 1])
            act = oracle.RELU if l < L else oracle.IDENTITY
            outs.append((h, op.forward(l, h, oW[l - 1], act)))
            h = outs[-1][1]
            if do_push and l <= L - 1:
                op.push(l, h, o_stores[l])
        o_loss, dh = oracle.softmax_xent(h, y)
        o_dw = [None] * L
        for l in range(L, 0, -1):
            act = oracle.RELU if l < L else oracle.IDENTITY
            o_dw[l - 1], dh_in = op.backward(l, outs[l - 1][0], oW[l - 1], outs[l - 1][1], dh,
                                             act, want_dh_in=l > 1)
            dh = dh_in
        # GPU round
        gp.round(r, K, gx, gW, g_stores, gy)
        assert_close(host(gp.H[L]), outs[-1][1], f"K={K} round {r} logits")
        assert abs(float(host(gp.loss)[0]) - o_loss) <= ATOL + RTOL * abs(o_loss)
        for l in range(1, L + 1):
            assert_close(host(gp.dW[l]), o_dw[l - 1], f"K={K} round {r} dW{l}",
                         scale_tol=1e-4)
        for l in range(1, L):
            assert_close(host(g_stores[l]), o_stores[l], f"K={K} round {r} store level {l}")
        # SGD on both sides
        for l in range(L):
            oW[l] = (oW[l] - np.float32(lr) * o_dw[l]).astype(np.float32)
            gW[l].sub_(lr * gp.dW[l + 1])


@pytest.mark.parametrize("overlap_io", [False, True], ids=["in-line-io", "overlapped-io"])
def test_graph_replay_matches_eager(tiny_graph, overlap_io):
    from paper_2206_00057_amd import step
    cfg, g = tiny_graph
    part = synth.make_partition(cfg, g, 1)
    L = cfg.layers
    X = synth.features(cfg)
    stores = [dev(X)] + [dev(synth.relu_normal((g.n, cfg.widths[l]), 20 + l))
                         for l in range(1, L)]
    Ws = [dev(w) for w in synth.weights(cfg)]
    y = dev(synth.labels(cfg)[part.owned])
    x = dev(X[part.owned])
    gp = step.GpuPartition(g.n, part, cfg.widths, overlap_io=overlap_io)
    gp.pull_all(stores)
    K = 3
    eager = {}
    for r in (1, 2, 3):
        gp.round(r, K, x, Ws, stores, y)
        eager[r] = (host(gp.H[L]).copy(), [host(gp.dW[l]).copy() for l in range(1, L + 1)])
    gp.capture(K, x, Ws, stores, y)
    for rep in range(3):
        for r in (1, 2, 3):
            gp.H[L].zero_()
            for l in range(1, L + 1):
                gp.dW[l].zero_()
            gp.replay(r, K)
            torch.cuda.synchronize()
            _ = torch.ones(1000, device="cuda").sum().item()   # eager work between replays
            assert_bits(host(gp.H[L]), eager[r][0], f"replay {rep} round {r} logits")
            for l in range(1, L + 1):
                assert_bits(host(gp.dW[l]), eager[r][1][l - 1], f"replay {rep} round {r} dW{l}")


def test_profile_instrumentation(tiny_graph):
    from paper_2206_00057_amd import step
    Dm = D()
    cfg, g = tiny_graph
    part = synth.make_partition(cfg, g, 0)
    gp = step.GpuPartition(g.n, part, cfg.widths)
    stores = [dev(synth.features(cfg))] + [dev(synth.relu_normal((g.n, 64), 21))]
    gp.pull_all(stores)
    Ws = [dev(w) for w in synth.weights(cfg)]
    Dm.digest_profile_enable(gp.p, True)
    gp.round(1, 1, dev(synth.features(cfg)[part.owned]), Ws, stores,
             dev(synth.labels(cfg)[part.owned]))
    prof = Dm.digest_profile_read(gp.p)
    Dm.digest_profile_enable(gp.p, False)
    # tiny workload: layer 1 aggregates first; layer 2 (64 -> 16, identity) transforms first
    assert prof["spmm_fwd.l1"][1] == 1 and prof["spmm_fwd.l2"][1] == 1
    assert prof["gemm_fwd_relu.l1"][1] == 1 and prof["gemm_fwd_relu.l2"][1] == 1
    # the GCN partition's pulls keep the halo aggregate alone (no row gather)
    assert prof["halo_aggregate.l1"][1] == 1 and "pull_gather.l1" not in prof
    assert prof["push_scatter.l1"][1] == 1 and prof["boundary_rows.l2"][1] == 1
    assert prof["softmax_xent.l2"][1] == 1 and prof["loss_mean.l2"][1] == 1
    assert prof["gemm_dw_splitk.l1"][1] == 1 and prof["gemm_dw_splitk.l2"][1] == 1
    assert prof["spmm_bwd_transposed.l2"][1] == 1 and "spmm_bwd_transposed.l1" not in prof
    assert all(ms >= 0 for ms, _ in prof.values())
    assert Dm.digest_profile_read(gp.p) == {}


# ---------------------------------------------------------------------------
# CSR rows in any column order, with repeated (row, column) entries: the
# header lets callers pass them (repeats are summed), and the oracle follows
# the same CSR, so every call must still match it
# ---------------------------------------------------------------------------

# (widths, what layer 2 runs): transform-first identity with the fused
# narrow epilogue (64 -> 16), aggregate-first identity on the GEMM (40 -> 48)
SCRAMBLED = [(64, 64, 16), (24, 40, 48)]


@pytest.mark.parametrize("widths", SCRAMBLED, ids=lambda w: "x".join(map(str, w)))
def test_scrambled_rows_with_repeats(widths):
    from paper_2206_00057_amd import digest as Dm
    cfg = synth.scaled(synth.CONFIGS["tiny"], 2000, widths=widths, classes=widths[-1])
    g = synth.make_graph(cfg)
    base = synth.make_partition(cfg, g, 1)
    part = synth.scramble_rows(base, seed=7, repeat_frac=0.3, long_row=300)
    rows = np.diff(part.indptr)
    assert rows.max() >= 300 and part.nnz > base.nnz
    assert any(np.any(np.diff(part.indices[part.indptr[i]:part.indptr[i + 1]]) <= 0)
               for i in range(part.n_own))
    c = Case(cfg, g, part, label=f"scrambled {widths}")
    for layer in (1, 2):
        check_layer(c, layer)
    # the halo gradient of layer 2, standalone and from the fused backward
    W = synth.weights(cfg)[1]
    h_in = c.layer_input(2)
    for act in (oracle.RELU, oracle.IDENTITY):
        out = torch.empty(c.n, widths[2], device="cuda")
        Dm.digest_layer_forward(c.h, 2, dev(h_in), dev(W), out, act)
        h_out = c.op.forward(2, h_in, W, act)
        dh = c.upstream(2)
        ref_halo = c.op.halo_gradient(2, W, h_out, dh, act)
        got = torch.full((part.n_halo, widths[1]), float("nan"), device="cuda")
        Dm.digest_halo_gradient(c.h, 2, dev(h_out), dev(dh), dev(W), got)
        assert_close(host(got), ref_halo, f"{c.label} halo gradient act {act}")
        dw = torch.empty(W.shape, device="cuda")
        dh_in = torch.empty(c.n, widths[1], device="cuda")
        got2 = torch.full((part.n_halo, widths[1]), float("nan"), device="cuda")
        Dm.digest_layer_backward_halo(c.h, 2, dev(h_in), dev(h_out), dev(dh), dev(W), dw, dh_in,
                                      got2)
        ref_dw, ref_dh = c.op.backward(2, h_in, W, h_out, dh, act)
        assert_close(host(dw), ref_dw, f"{c.label} fused dW act {act}")
        assert_close(host(dh_in), ref_dh, f"{c.label} fused dh_in act {act}")
        assert_close(host(got2), ref_halo, f"{c.label} fused halo gradient act {act}")


def test_empty_partition_with_halo_gives_zero_halo_gradient():
    """No owned rows but unreferenced halo ids: the fused backward's halo
    gradient is zero (as digest_halo_gradient gives), and dW is zero."""
    from paper_2206_00057_amd import digest as Dm
    widths = [8, 12, 5]
    halo = np.array([3, 7, 11], np.int64)
    h = Dm.digest_partition_create(20, np.zeros(1, np.int64), np.zeros(0, np.int64),
                                   np.zeros(0, np.float32), np.zeros(0, np.int64), halo, widths)
    ws = torch.empty(max(h.workspace_bytes, 256), dtype=torch.uint8, device="cuda")
    Dm.digest_partition_bind_workspace(h, ws)
    Dm.digest_pull(h, 1, dev(synth.normal((20, widths[1]), seed=3)))
    W = dev(synth.normal((widths[1], widths[2]), seed=4))
    empty = torch.empty(0, device="cuda")
    Dm.digest_layer_forward(h, 2, empty, W, empty, Dm.ACT_IDENTITY)
    dw = torch.full((widths[1], widths[2]), float("nan"), device="cuda")
    dh_halo = torch.full((3, widths[1]), float("nan"), device="cuda")
    Dm.digest_layer_backward_halo(h, 2, empty, empty, empty, W, dw, empty, dh_halo)
    assert not host(dh_halo).any() and not host(dw).any()


# ---------------------------------------------------------------------------
# tiered aggregation: sliced passes over the most-read source rows, then the
# rest, each adding into the output (forced here on small graphs)
# ---------------------------------------------------------------------------

# (widths, what is tiered): float4 slices at 256 (one slice per XCD) and 264
# (a partial second slice group), forward and transposed; float2 slices at
# 602 (three slice groups per XCD)
TIERED = [(256, 264, 258, 7), (602, 300, 41)]


@pytest.mark.parametrize("widths", TIERED, ids=lambda w: "x".join(map(str, w)))
def test_tiered_aggregation_matches_oracle(widths, monkeypatch):
    from paper_2206_00057_amd import digest as Dm
    monkeypatch.setenv("DIGEST_SPMM_TIERS", "3")
    monkeypatch.setenv("DIGEST_SPMM_TIER_BYTES", "8192")
    cfg = synth.scaled(synth.CONFIGS["tiny"], 2000, widths=widths, classes=widths[-1])
    g = synth.make_graph(cfg)
    part = synth.scramble_rows(synth.make_partition(cfg, g, 1), seed=5, repeat_frac=0.1,
                               long_row=400)
    c = Case(cfg, g, part, label=f"tiered {widths}")
    plan = Dm.digest_partition_plan(c.h, 1)
    assert plan["tiers_fwd"] == 3 and 0 < plan["tier_entries_fwd"] < part.nnz, plan
    if len(widths) == 4:
        plan2 = Dm.digest_partition_plan(c.h, 2)
        assert plan2["tiers_fwd"] == 3 and plan2["tiers_bwd"] == 3, plan2
    for layer in range(1, c.L + 1):
        check_layer(c, layer)


def test_tiering_off_gives_one_pass(monkeypatch):
    """DIGEST_SPMM_TIER_BYTES=0 plans no tiers; the results agree with the
    tiered plan's within the float32 bar (the sums are ordered differently)."""
    from paper_2206_00057_amd import digest as Dm
    widths = (256, 264, 7)
    cfg = synth.scaled(synth.CONFIGS["tiny"], 2000, widths=widths, classes=widths[-1])
    g = synth.make_graph(cfg)
    part = synth.make_partition(cfg, g, 2)
    outs = []
    for env in ({"DIGEST_SPMM_TIER_BYTES": "0"},
                {"DIGEST_SPMM_TIER_BYTES": "8192", "DIGEST_SPMM_TIERS": "2"}):
        for k in ("DIGEST_SPMM_TIER_BYTES", "DIGEST_SPMM_TIERS"):
            monkeypatch.delenv(k, raising=False)
        for k, v in env.items():
            monkeypatch.setenv(k, v)
        c = Case(cfg, g, part, label=str(env))
        assert (Dm.digest_partition_plan(c.h, 1)["tiers_fwd"] > 0) == ("DIGEST_SPMM_TIERS" in env)
        x = c.layer_input(1)
        W = synth.weights(cfg)[0]
        Dm.digest_pull(c.h, 0, dev(c.store(0)))
        out = torch.empty(c.n, widths[1], device="cuda")
        Dm.digest_layer_forward(c.h, 1, dev(x), dev(W), out, Dm.ACT_RELU)
        outs.append(host(out))
    assert_close(outs[1], outs[0], "tiered vs one pass")


# ---------------------------------------------------------------------------
# tall products (6,000 owned rows) -- forward (ReLU epilogue), input
# gradient (masked A, W read transposed), rows padded past an odd K, and the
# halo-gradient product
# ---------------------------------------------------------------------------

TALL = [(100, 256, 256, 47), (602, 256, 41), (500, 256, 7), (33, 130, 9, 70)]


@pytest.mark.parametrize("widths", TALL, ids=lambda w: "x".join(map(str, w)))
def test_tall_products(widths):
    from paper_2206_00057_amd import digest as Dm
    cfg = synth.scaled(synth.CONFIGS["tiny"], 24000, widths=widths, classes=widths[-1])
    g = synth.make_graph(cfg, seed=3)
    c = Case(cfg, g, synth.make_partition(cfg, g, 1), label=f"tall{widths}")
    assert c.n >= 4096
    for layer in range(1, c.L + 1):
        check_layer(c, layer)
    # the halo gradient of layer 2 (ReLU or identity, as the layer's act)
    W = synth.weights(cfg)[1]
    h_in = c.layer_input(2)
    act = c.act(2)
    out = torch.empty(c.n, widths[2], device="cuda")
    Dm.digest_layer_forward(c.h, 2, dev(h_in), dev(W), out, act)
    h_out = c.op.forward(2, h_in, W, act)
    dh = c.upstream(2)
    got = torch.full((c.part.n_halo, widths[1]), float("nan"), device="cuda")
    Dm.digest_halo_gradient(c.h, 2, dev(h_out), dev(dh), dev(W), got)
    assert_close(host(got), c.op.halo_gradient(2, W, h_out, dh, act), f"{c.label} halo gradient")


# ---------------------------------------------------------------------------
# the fused forward and input gradient (each 32-row tile aggregated into LDS
# and multiplied by W or W^T there), forced at small sizes: rows of 65..128
# floats (two lane groups per row) and of 129..256, a padded width, column
# counts that leave partial 64-column blocks and a second 256-column pass,
# two fused layers, rows long enough for the long-row pass (lognormal
# degrees: all of them; Zipf degrees up to 4,096: a third of the entries);
# results against the oracle and the two-pass path, and bit for bit from one
# fused run to the next (rows are dealt to the waves in a fixed order, each
# summed by one wave in a fixed order)
# ---------------------------------------------------------------------------

FUSED = [((256, 256, 256, 47), "tiny", 1200), ((130, 100, 70), "tiny", 1200),
         ((133, 130, 9, 70), "tiny", 1200), ((256, 300, 7), "tiny", 1200),
         ((256, 256, 7), "dense", 2000), ((256, 256, 256, 47), "large", 8000),
         ((100, 200, 256, 7), "large", 8000), ((64, 140, 150, 5), "tiny", 1200),
         ((72, 96, 80, 5), "large", 8000)]


@pytest.mark.parametrize("widths,base,n", FUSED,
                         ids=lambda v: "x".join(map(str, v)) if isinstance(v, tuple) else str(v))
def test_fused_forward(widths, base, n, monkeypatch):
    Dm = D()
    cfg = synth.scaled(synth.CONFIGS[base], n, widths=widths, classes=widths[-1])
    g = synth.make_graph(cfg, seed=7)
    part = synth.make_partition(cfg, g, 1)
    monkeypatch.setenv("DIGEST_FUSE", "2")
    c = Case(cfg, g, part, label=f"fused{widths}")
    plans = [Dm.digest_partition_plan(c.h, l) for l in range(1, c.L + 1)]
    assert any(pl["forward_fused"] or pl["backward_fused"] for pl in plans)
    for layer in range(1, c.L + 1):
        check_layer(c, layer)
    # the input gradient of layer 2 (ReLU, aggregate first), fused or not
    if c.L >= 3:
        x2 = dev(c.layer_input(2))
        W2 = dev(synth.weights(cfg)[1])
        dh2 = dev(c.upstream(2))
        if c.part.n_halo:
            Dm.digest_pull(c.h, 1, dev(c.store(1)))
        got2 = {}
        for mode in ("2", "0", "2b"):
            monkeypatch.setenv("DIGEST_FUSE", mode[0])
            out2 = torch.empty(c.n, widths[2], device="cuda")
            Dm.digest_layer_forward(c.h, 2, x2, W2, out2, Dm.ACT_RELU)
            dw2 = torch.empty(W2.shape, device="cuda")
            dhin = torch.empty(c.n, widths[1], device="cuda")
            Dm.digest_layer_backward(c.h, 2, x2, out2, dh2, W2, dw2, dhin)
            got2[mode] = (host(dw2), host(dhin))
        for i, what in enumerate(("dW", "dH_in")):
            assert_close(got2["2"][i], got2["0"][i], f"{c.label} fused vs two-pass layer-2 {what}",
                         rtol=1e-5, atol=1e-6)
            assert_bits(got2["2"][i], got2["2b"][i], f"{c.label} fused layer-2 {what} run twice")
    # the same forward and weight gradient of layer 1, fused and not
    x = dev(c.layer_input(1))
    W = dev(synth.weights(cfg)[0])
    dh = dev(c.upstream(1))
    Dm.digest_pull(c.h, 0, dev(c.store(0)))
    got = {}
    for mode in ("2", "0", "2b"):
        monkeypatch.setenv("DIGEST_FUSE", mode[0])
        out = torch.empty(c.n, widths[1], device="cuda")
        Dm.digest_layer_forward(c.h, 1, x, W, out, Dm.ACT_RELU)
        dw = torch.empty(W.shape, device="cuda")
        Dm.digest_layer_backward(c.h, 1, x, out, dh, W, dw, None)
        got[mode] = (host(out), host(dw))
    assert_close(got["2"][0], got["0"][0], f"{c.label} fused vs two-pass forward",
                 rtol=1e-5, atol=1e-6)
    assert_close(got["2"][1], got["0"][1], f"{c.label} fused vs two-pass dW",
                 rtol=1e-5, atol=1e-6)
    assert_bits(got["2"][0], got["2b"][0], f"{c.label} fused forward run twice")
    assert_bits(got["2"][1], got["2b"][1], f"{c.label} fused dW run twice")


# ---------------------------------------------------------------------------
# padding columns of the library's buffers hold NaN (the workspace is filled
# with 0xFF bytes before binding): rows of widths that are not a multiple of
# 4 floats are read as whole vectors, and nothing of the padding may reach
# an output -- GEMMs over a padded K (30 -> 100, the 70-wide last layer's
# padded gradient), the narrow products, the aggregations and the halo reads
# ---------------------------------------------------------------------------

PADDED = [(30, 100, 70), (30, 80, 9), (602, 47, 7), (33, 130, 9, 70)]


@pytest.mark.parametrize("widths", PADDED, ids=lambda w: "x".join(map(str, w)))
def test_nan_padding_never_reaches_outputs(widths):
    cfg = synth.scaled(synth.CONFIGS["tiny"], 1200, widths=widths, classes=widths[-1])
    g = synth.make_graph(cfg, seed=6)
    c = Case(cfg, g, synth.make_partition(cfg, g, 1), label=f"nanpad{widths}", ws_fill=255)
    for level in range(c.L):
        check_pull(c, level)
    for layer in range(1, c.L + 1):
        check_layer(c, layer)
    check_loss(c)


# ---------------------------------------------------------------------------
# the weight gradient on the library's side stream, concurrent with the
# input-gradient chain (forced at every size here): results, and graph
# capture with replays, must not change
# ---------------------------------------------------------------------------

# (widths, fuse): layer 2 aggregate-first with ReLU, the weight gradient next
# to the transposed aggregation of D W^T (24 -> 40 -> 48 -> 7); an identity
# layer aggregated at its narrower output width first (24 -> 40 -> 36); and
# the fused passes forced (a ReLU layer of 96 floats fused in both
# directions, 100 -> 96 -> 96 -> 7), so that the weight gradient's fork sits
# after the formed D and beside the fused input gradient; and a
# transform-first layer 24 floats wide (48 -> 96 -> 24), whose weight
# gradient runs beside G W^T
SIDE = [((24, 40, 48, 7), "0"), ((24, 40, 36), "0"), ((100, 96, 96, 7), "2"),
        ((48, 96, 24), "0")]


@pytest.mark.parametrize("widths,fuse", SIDE,
                         ids=lambda v: "x".join(map(str, v)) if isinstance(v, tuple) else v)
def test_side_stream_backward(widths, fuse, monkeypatch):
    from paper_2206_00057_amd import step
    monkeypatch.setenv("DIGEST_SIDE_STREAM", "2")
    monkeypatch.setenv("DIGEST_FUSE", fuse)
    cfg = synth.scaled(synth.CONFIGS["tiny"], 1200, widths=widths, classes=widths[-1])
    g = synth.make_graph(cfg, seed=4)
    part = synth.make_partition(cfg, g, 2)
    c = Case(cfg, g, part, label=f"side{widths}")
    Dm = D()
    if fuse == "2":
        assert Dm.digest_partition_plan(c.h, 2)["forward_fused"] == 1
        assert Dm.digest_partition_plan(c.h, 2)["backward_fused"] == 1
    if widths == (48, 96, 24):
        pl = Dm.digest_partition_plan(c.h, 2)
        assert pl["transform_first"] == 1 and pl["dgrad_fused"] == 0
    for layer in range(1, c.L + 1):
        check_layer(c, layer)
    # rounds: eager, then captured and replayed (bit for bit)
    L = cfg.layers
    X = synth.features(cfg)
    stores = [dev(X)] + [dev(synth.relu_normal((g.n, cfg.widths[l]), 20 + l))
                         for l in range(1, L)]
    Ws = [dev(w) for w in synth.weights(cfg)]
    y = dev(synth.labels(cfg)[part.owned])
    x = dev(X[part.owned])
    gp = step.GpuPartition(g.n, part, cfg.widths)
    gp.pull_all(stores)
    K = 2
    eager = {}
    for r in (1, 2):
        gp.round(r, K, x, Ws, stores, y)
        eager[r] = [host(gp.dW[l]).copy() for l in range(1, L + 1)] + [host(gp.dH[1]).copy()]
    gp.capture(K, x, Ws, stores, y)
    for rep in range(3):
        for r in (1, 2):
            for l in range(1, L + 1):
                gp.dW[l].zero_()
            gp.replay(r, K)
            torch.cuda.synchronize()
            _ = torch.ones(1000, device="cuda").sum().item()   # eager work between replays
            got = [host(gp.dW[l]) for l in range(1, L + 1)] + [host(gp.dH[1])]
            for i, (a, b) in enumerate(zip(got, eager[r])):
                assert_bits(a, b, f"replay {rep} round {r} output {i}")
