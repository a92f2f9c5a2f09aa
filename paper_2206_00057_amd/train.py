"""DIGEST training of every subgraph of a graph on one GPU (Algorithm 1,
synchronous mode), the subgraphs taking turns on one stream and sharing one
device-resident representation store per stale level.

Round r (1-based), sync interval K, M subgraphs:

    every subgraph starts from the global parameters W
    for l = 1..L:
        if r mod K == 0 and l >= 2: every subgraph pulls level l-1
        every subgraph runs the forward of layer l
        if (r-1) mod K == 0 and l <= L-1: every subgraph pushes level l
    every subgraph: loss head, backward of layers L..1 -> dW_m
    W <- W - lr * (1/M) sum_m dW_m        (AGG of the M local models)

The subgraphs advance layer by layer together (all forwards of layer l, then
all pushes of level l, then the pulls of level l before layer l+1; the
backward likewise, layer L down to 1), the synchronous barrier of
Algorithm 1 at layer granularity.  With K = 1 every
halo row a subgraph reads was pushed by its owner earlier in the same round,
so each subgraph's forward equals the full-graph GCN forward on its rows
(P_m = P_in + P_out with fresh halo rows).  With K > 1 the halo rows are the
stale ones of the last push round.

grad_exchange adds the appendix's stale-gradient term: after the backward of
layer l >= 2, every subgraph's halo gradient P_out^T D W^T goes into a
per-level gradient store (digest_push_add) and each owner adds its rows to
its input gradient (digest_pull_add) -- in the same round ("fresh": with
K = 1 the mean of the subgraphs' gradients is then the full-graph gradient)
or one round later ("stale", the t-1 of the appendix).  "none" keeps halo
rows as constants.

model="gat" trains GAT layers over stale halo rows instead of Eq. 5; AGG
then averages the attention matrices as well as W.

All arithmetic runs in libdigest.so (the layers, pulls, pushes, loss heads
and the parameter averaging); this module owns the buffers and orders the
calls.  ``capture`` records one round per pull/push pattern into a HIP graph.
"""
from __future__ import annotations

import torch

from . import digest as D
from .step import GpuPartition


def boundary_push_mode(gps, parts):
    """DIGEST_PUSH_BOUNDARY when every halo node of every subgraph is a
    boundary row of its owner (so pushing boundary rows writes every row
    anyone pulls; this holds when the graph is structurally symmetric),
    else DIGEST_PUSH_ALL_OWNED, the paper's push of every owned row."""
    import numpy as np
    pushed = np.concatenate([D.digest_partition_export_maps(gp.p)[1] for gp in gps] +
                            [np.zeros(0, np.int64)])
    pulled = np.concatenate([np.asarray(p.halo, np.int64) for p in parts] +
                            [np.zeros(0, np.int64)])
    return D.PUSH_BOUNDARY if np.isin(pulled, pushed).all() else D.PUSH_ALL_OWNED


class DigestTrainer:
    def __init__(self, n_global, parts, widths, x, labels, weights, lr, K, device="cuda",
                 grad_exchange="none", model="gcn", atts=None):
        """parts: synth-style partitions (owned, halo, CSR rows) covering the
        graph; x: device [n_global, d_0] features; labels: device int32
        [n_global]; weights: device float32 tensors W_1..W_L (the global
        parameters, updated in place by every round)."""
        if not 1 <= len(parts) <= 64:
            raise ValueError("between 1 and 64 subgraphs")
        if grad_exchange not in ("none", "fresh", "stale"):
            raise ValueError("grad_exchange is none, fresh or stale")
        if model == "gat" and grad_exchange != "none":
            raise ValueError("the halo-gradient exchange is defined for GCN layers")
        self.grad_exchange = grad_exchange
        self.model = model
        self.att = atts   # GAT: device [d_l, 2] attention matrices, updated in place
        self.widths = [int(w) for w in widths]
        self.L = len(self.widths) - 1
        self.n_global = int(n_global)
        self.lr, self.K = float(lr), int(K)
        self.W = weights
        # pulls keep the halo aggregate alone for GCN layers, the halo rows
        # for GAT layers (GpuPartition's default)
        self.gps = [GpuPartition(n_global, p, widths, device=device, model=model, atts=atts)
                    for p in parts]
        self.push_mode = boundary_push_mode(self.gps, parts)
        idx = [torch.from_numpy(p.owned).to(device) for p in parts]
        self.x_own = [x.index_select(0, i).contiguous() for i in idx]
        self.y_own = [labels.index_select(0, i).contiguous() for i in idx]
        f32 = dict(dtype=torch.float32, device=device)
        # the shared store: level 0 is the static features, levels 1..L-1 stale
        self.stores = [x] + [torch.zeros(n_global, self.widths[l], **f32)
                             for l in range(1, self.L)]
        self.losses = torch.zeros(len(parts), **f32)
        if grad_exchange != "none":
            # gradient stores (levels 1..L-1) and each subgraph's halo gradients
            self.gstores = [None] + [torch.zeros(n_global, self.widths[l], **f32)
                                     for l in range(1, self.L)]
            self.dh_halo = [[None] + [torch.empty(p.n_halo, self.widths[l], **f32)
                                      for l in range(1, self.L)] for p in parts]
        self.graphs = {}
        # aggregation entries per round: GCN forward nnz and backward nnz_in
        # (layers >= 2); GAT forward and transposed backward nnz per layer
        if model == "gat":
            self.edges_per_round = sum(2 * gp.p.nnz * self.L for gp in self.gps)
        else:
            self.edges_per_round = sum(gp.p.nnz + (gp.p.nnz_in if l > 1 else 0)
                                       for gp in self.gps for l in range(1, self.L + 1))

    def act(self, layer):
        return D.ACT_RELU if layer < self.L else D.ACT_IDENTITY

    def _fwd(self, gp, l, h):
        if self.model == "gat":
            D.digest_gat_forward(gp.p, l, h, self.W[l - 1], self.att[l - 1], gp.H[l], self.act(l))
        else:
            D.digest_layer_forward(gp.p, l, h, self.W[l - 1], gp.H[l], self.act(l))

    def init_stores(self):
        """Fill the store with one forward of all subgraphs at the current W
        with fresh halo rows (a round-0 pass that pulls before and pushes
        after every layer), then give every subgraph all its halo levels."""
        for gp in self.gps:
            D.digest_pull(gp.p, 0, self.stores[0])
        h = list(self.x_own)
        for l in range(1, self.L):
            for m, gp in enumerate(self.gps):
                if l >= 2:
                    D.digest_pull(gp.p, l - 1, self.stores[l - 1])
                self._fwd(gp, l, h[m])
            for gp in self.gps:
                D.digest_push(gp.p, l, gp.H[l], self.stores[l], self.push_mode)
            h = [gp.H[l] for gp in self.gps]
        for gp in self.gps:
            for lev in range(1, self.L):
                D.digest_pull(gp.p, lev, self.stores[lev])

    def _round(self, do_pull, do_push):
        h = list(self.x_own)
        for l in range(1, self.L + 1):
            if do_pull and l >= 2:
                for gp in self.gps:
                    D.digest_pull(gp.p, l - 1, self.stores[l - 1])
            for m, gp in enumerate(self.gps):
                self._fwd(gp, l, h[m])
            if do_push and l <= self.L - 1:
                for gp in self.gps:
                    D.digest_push(gp.p, l, gp.H[l], self.stores[l], self.push_mode)
            h = [gp.H[l] for gp in self.gps]
        for m, gp in enumerate(self.gps):
            D.digest_softmax_xent(gp.p, gp.H[self.L], self.y_own[m], gp.dH[self.L],
                                  self.losses[m:m + 1])
        exch = self.grad_exchange != "none"
        for l in range(self.L, 0, -1):
            for m, gp in enumerate(self.gps):
                dh_in = gp.dH[l - 1] if l > 1 else None
                h_in = gp.H[l - 1] if l > 1 else self.x_own[m]
                if self.model == "gat":
                    D.digest_gat_backward(gp.p, l, h_in, gp.H[l], gp.dH[l], self.W[l - 1],
                                          self.att[l - 1], gp.dW[l], gp.dAtt[l], dh_in)
                elif exch and l > 1:
                    # the halo gradient comes out of the backward's own products
                    D.digest_layer_backward_halo(gp.p, l, h_in, gp.H[l], gp.dH[l],
                                                 self.W[l - 1], gp.dW[l], dh_in,
                                                 self.dh_halo[m][l - 1])
                else:
                    D.digest_layer_backward(gp.p, l, h_in, gp.H[l], gp.dH[l], self.W[l - 1],
                                            gp.dW[l], dh_in)
            if exch and l > 1:
                self._exchange(l)
        for l in range(1, self.L + 1):
            D.digest_sgd_average(self.W[l - 1], [gp.dW[l] for gp in self.gps], self.lr)
            if self.model == "gat":
                D.digest_sgd_average(self.att[l - 1], [gp.dAtt[l] for gp in self.gps], self.lr)

    def _exchange(self, l):
        """The halo gradients of layer l (from the backward) into the level
        l-1 store and back to the owners' input gradients (fresh: this
        round's; stale: last round's)."""
        gs = self.gstores[l - 1]
        if self.grad_exchange == "fresh":
            for m, gp in enumerate(self.gps):
                D.digest_push_add(gp.p, l - 1, self.dh_halo[m][l - 1], gs)
            for gp in self.gps:
                D.digest_pull_add(gp.p, l - 1, gs, gp.dH[l - 1])
        else:
            for gp in self.gps:
                D.digest_pull_add(gp.p, l - 1, gs, gp.dH[l - 1])
            for m, gp in enumerate(self.gps):
                D.digest_push_add(gp.p, l - 1, self.dh_halo[m][l - 1], gs)

    def round(self, r):
        """Round r (1-based), eagerly."""
        self._round(*D.digest_sync_period(self.K, r))

    def capture(self):
        """Record one HIP graph per pull/push pattern of the schedule.  The
        warm-up and the captures run rounds, so they also train: the caller
        restores W (and the store) afterwards if it needs a fixed start."""
        patterns = sorted({D.digest_sync_period(self.K, r) for r in range(1, 2 * self.K + 1)})
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            for pat in patterns:
                self._round(*pat)
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        for pat in patterns:
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                self._round(*pat)
            self.graphs[pat] = g
        torch.cuda.synchronize()

    def replay(self, r):
        self.graphs[D.digest_sync_period(self.K, r)].replay()

    def mean_loss(self):
        """Average of the subgraphs' local losses of the last round (Eq. 3)."""
        return float(self.losses.mean())
