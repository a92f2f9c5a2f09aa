"""GPU parity at the full sizes of the four large workloads (Flickr-, Reddit-
and OGB-Products-shaped synthetic graphs, and the halo-dominated permutation
partition), in the same library calls the benchmark times: pull and push
contents bit-exact; every layer's forward and backward, the fused backward
with the halo gradient, and the loss head within rtol 1e-4 / atol 1e-5 plus
the scale-aware bound, over all outputs; Algorithm 1's rounds over all eight
Flickr-shaped subgraphs against the oracle trainer
(the oracle finishes these in seconds with its threads); and the GAT layer
over stale halo rows on the three workloads the GAT benchmark times, every
layer's forward and backward over all outputs."""
import time

import numpy as np
import pytest

from paper_2206_00057_amd import synth
from test_gpu_parity import (Case, assert_close, check_layer, check_loss, check_pull, check_push,
                             dev, host, torch)
import test_gpu_gat
import oracle

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

_graphs = {}


def check_backward_halo(c, layer):
    """The trainer's fused backward of a layer above the first, with the
    halo gradient P_out^T D W^T (Appendix A.3's stale-gradient term): dW,
    dH_in and dH_halo against the oracle."""
    from paper_2206_00057_amd import digest as Dm
    h_in = c.layer_input(layer)
    W = synth.weights(c.cfg)[layer - 1]
    act = c.act(layer)
    d_in, d_out = c.widths[layer - 1], c.widths[layer]
    out = torch.empty(c.n, d_out, device="cuda")
    Dm.digest_layer_forward(c.h, layer, dev(h_in), dev(W), out, act)
    ref_out = c.op.forward(layer, h_in, W, act)
    dh = c.upstream(layer)
    dw = torch.empty(d_in, d_out, device="cuda")
    dh_in = torch.empty(c.n, d_in, device="cuda")
    dh_halo = torch.full((c.part.n_halo, d_in), float("nan"), device="cuda")
    Dm.digest_layer_backward_halo(c.h, layer, dev(h_in), dev(ref_out), dev(dh), dev(W), dw,
                                  dh_in, dh_halo)
    ref_dw, ref_dh = c.op.backward(layer, h_in, W, ref_out, dh, act)
    ref_halo = c.op.halo_gradient(layer, W, ref_out, dh, act)
    assert_close(host(dw), ref_dw, f"{c.label} fused dW layer {layer}")
    assert_close(host(dh_in), ref_dh, f"{c.label} fused dH_in layer {layer}")
    assert_close(host(dh_halo), ref_halo, f"{c.label} dH_halo layer {layer}")


def graph_for(cfg):
    key = (cfg.n, cfg.blocks, cfg.degree, cfg.shape, cfg.cap, cfg.p_intra, cfg.c)
    if key not in _graphs:
        _graphs.clear()
        t = time.time()
        _graphs[key] = synth.make_graph(cfg)
        print(f"[graph {cfg.name}: {time.time() - t:.1f}s]", flush=True)
    return _graphs[key]


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", ["medium", "dense", "large", "halo"])
def test_full_size_workload(name):
    cfg = synth.CONFIGS[name]
    g = graph_for(cfg)
    part = synth.make_partition(cfg, g, 0)
    c = Case(cfg, g, part, label=name)
    print(f"[{name}] {synth.shape_stats(cfg, g, part)}", flush=True)
    for level in range(c.L):
        t = time.time()
        check_pull(c, level)
        print(f"[{name}] pull level {level} ok {time.time() - t:.1f}s", flush=True)
    for level in range(1, c.L):
        t = time.time()
        check_push(c, level)
        print(f"[{name}] push level {level} ok {time.time() - t:.1f}s", flush=True)
    for layer in range(1, c.L + 1):
        t = time.time()
        check_layer(c, layer)
        print(f"[{name}] layer {layer} fwd+bwd ok {time.time() - t:.1f}s", flush=True)
        if layer > 1 and c.part.n_halo:
            t = time.time()
            check_backward_halo(c, layer)   # level layer-1 as check_layer pulled it
            print(f"[{name}] layer {layer} halo gradient ok {time.time() - t:.1f}s", flush=True)
    check_loss(c)
    print(f"[{name}] loss ok", flush=True)
    del c
    torch.cuda.empty_cache()


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", ["medium", "dense", "large"])
def test_full_size_gat_workload(name):
    """Every GAT layer of the workload, on the partition the benchmark times:
    each level pulled from a seeded store, then the layer's forward and
    backward (dW, datt, dH_in) on both sides, the inputs on the dyadic grid
    that makes every LeakyReLU branch decision exact."""
    cfg = synth.CONFIGS[name]
    g = graph_for(cfg)
    part = synth.make_partition(cfg, g, 0)
    c = test_gpu_gat.Case(g.n, part, cfg.widths, seed=5)
    L = len(cfg.widths) - 1
    print(f"[{name} gat] {synth.shape_stats(cfg, g, part)}", flush=True)
    for layer in range(1, L + 1):
        t = time.time()
        store = synth.relu_normal((g.n, cfg.widths[layer - 1]), seed=70 + layer)
        c.pull(layer - 1, test_gpu_gat.dyadic(store, test_gpu_gat.X_BITS))
        act = oracle.RELU if layer < L else oracle.IDENTITY
        c.layer(layer, act, f"{name} gat layer {layer}", grid=True)
        print(f"[{name} gat] layer {layer} fwd+bwd ok {time.time() - t:.1f}s", flush=True)
    del c
    torch.cuda.empty_cache()


@pytest.mark.timeout(900)
@pytest.mark.parametrize("mode,rounds", [("none", 11), ("fresh", 3)])
def test_full_size_trainer_rounds(mode, rounds):
    """Algorithm 1 over all eight subgraphs of the Flickr-shaped workload
    (the configuration `bench.py --train` times), sync interval 10: rounds
    1..11 take the initial push, the pull of round 10 and the push of round
    11. Each round's logits of every subgraph, the global W and the stores
    are checked against the oracle trainer running its own trajectory."""
    from test_gpu_trainer import _setup
    cfg = synth.CONFIGS["medium"]
    K = cfg.sync_periods[0]
    g, parts, tr, ot = _setup(cfg, K=K, lr=0.1, grad_exchange=mode)
    tr.init_stores()
    ot.init_stores()
    for lev in range(1, cfg.layers):
        assert_close(host(tr.stores[lev]), ot.stores[lev], f"initial store level {lev}")
    for r in range(1, rounds + 1):
        t = time.time()
        tr.round(r)
        o_loss = ot.round(r)
        for m, gp in enumerate(tr.gps):
            assert_close(host(gp.H[cfg.layers]), ot.logits[m], f"{mode} round {r} logits m={m}",
                         scale_tol=1e-4)
        assert abs(tr.mean_loss() - o_loss) <= 1e-5 + 1e-4 * abs(o_loss)
        for l in range(cfg.layers):
            assert_close(host(tr.W[l]), ot.W[l], f"{mode} round {r} W{l + 1}", scale_tol=1e-4)
        for lev in range(1, cfg.layers):
            assert_close(host(tr.stores[lev]), ot.stores[lev], f"{mode} round {r} store {lev}",
                         scale_tol=1e-4)
        print(f"[medium trainer {mode}] round {r} ok, loss {o_loss:.6f} {time.time() - t:.1f}s",
              flush=True)
