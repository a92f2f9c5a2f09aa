"""One DIGEST training round of one partition on the GPU, as a sequence of
library calls (Algorithm 1's inner loop for a single subgraph), for the GCN
layer of Eq. 5 or the GAT layer over stale halo rows:

    for l = 1..L:   pull level l-1 if the schedule says so (levels >= 1),
                    layer forward, push level l if the schedule says so
                    (levels 1..L-1)
    loss head
    for l = L..1:   layer backward

All arithmetic runs in libdigest.so; this module only owns the device
buffers (PyTorch tensors) and orders the calls.  With overlap_io, pulls and
pushes run on a second stream next to the layer computation, as the paper's
system design overlaps representation I/O with the forward pass (Sec. 3.2):
a pull of level l-1 only has to finish before layer l starts, and a push of
level l only has to start after layer l.  With the store in the same HBM as
the layers' operands both sides are bandwidth-bound and the overlap does not
shorten a round, so the default keeps them in line on the caller's stream.
``capture``
records the round into a HIP graph (one graph per distinct pull/push
pattern of the schedule) so that replays cost one launch.
"""
from __future__ import annotations

import torch

from . import digest as D


class GpuPartition:
    def __init__(self, n_global, part, widths, device="cuda", overlap_io=False, model="gcn",
                 atts=None, pull_mode=None):
        """model "gcn" (Eq. 5) or "gat" (the attention layer over stale halo
        rows; atts are its per-layer [d_l, 2] attention matrices).
        pull_mode: what a pull keeps (D.PULL_ROWS or D.PULL_AGGREGATE); by
        default the halo aggregate alone for the GCN layer, the halo rows
        for the GAT layer, which reads them."""
        if model not in ("gcn", "gat"):
            raise ValueError("model is gcn or gat")
        if model == "gat" and (atts is None or len(atts) != len(widths) - 1):
            raise ValueError("a GAT model needs one attention matrix per layer")
        self.model, self.atts = model, atts
        self.widths = [int(w) for w in widths]
        self.L = len(self.widths) - 1
        self.device = device
        self.p = D.digest_partition_create(n_global, part.indptr, part.indices, part.values,
                                           part.owned, part.halo, self.widths)
        if pull_mode is None:
            pull_mode = D.PULL_AGGREGATE if model == "gcn" else D.PULL_ROWS
        D.digest_partition_set_pull_mode(self.p, pull_mode)
        n = self.p.n_own
        self.n_own = n
        self.workspace = torch.empty(max(self.p.workspace_bytes, 256), dtype=torch.uint8,
                                     device=device)
        D.digest_partition_bind_workspace(self.p, self.workspace)
        if model == "gat":
            self.gat_workspace = torch.empty(max(D.digest_gat_query(self.p), 256),
                                             dtype=torch.uint8, device=device)
            D.digest_gat_bind_workspace(self.p, self.gat_workspace)
        f32 = dict(dtype=torch.float32, device=device)
        # H[l]: output of layer l (H[0] is the caller's input rows); dH[l] its gradient
        self.H = [None] + [torch.empty(n, self.widths[l], **f32) for l in range(1, self.L + 1)]
        self.dH = [None] + [torch.empty(n, self.widths[l], **f32) for l in range(1, self.L + 1)]
        self.dW = [None] + [torch.empty(self.widths[l - 1], self.widths[l], **f32)
                            for l in range(1, self.L + 1)]
        self.dAtt = ([None] + [torch.empty(self.widths[l], 2, **f32) for l in range(1, self.L + 1)]
                     if model == "gat" else None)
        self.loss = torch.zeros(1, **f32)
        self.graphs = {}
        # pulls and pushes: on their own stream (default priority) next to the
        # layers, or in line on the caller's stream
        self.overlap_io = overlap_io
        self.io = torch.cuda.Stream(device=device) if overlap_io else None
        self.pull_done = [torch.cuda.Event() for _ in range(self.L)]

    def act(self, layer):
        return D.ACT_RELU if layer < self.L else D.ACT_IDENTITY

    def _layer(self, l, h, W, stream=None):
        if self.model == "gat":
            D.digest_gat_forward(self.p, l, h, W, self.atts[l - 1], self.H[l], self.act(l),
                                 stream=stream)
        else:
            D.digest_layer_forward(self.p, l, h, W, self.H[l], self.act(l), stream=stream)

    def pull_all(self, stores):
        """Initial pull of every level (level 0 = features)."""
        for lev in range(self.L):
            D.digest_pull(self.p, lev, stores[lev])

    def forward(self, x_own, Ws, stores=None, do_pull=False, do_push=False):
        self.x_own = x_own
        if not self.overlap_io:
            return self._forward_in_line(x_own, Ws, stores, do_pull, do_push)
        main = torch.cuda.current_stream()
        pulled = do_pull and self.L >= 2
        if pulled:
            # every scheduled pull starts now, on the I/O stream
            self.io.wait_stream(main)
            with torch.cuda.stream(self.io):
                for lev in range(1, self.L):
                    D.digest_pull(self.p, lev, stores[lev], stream=self.io)
                    self.pull_done[lev].record(self.io)
        h = x_own
        for l in range(1, self.L + 1):
            if pulled and l >= 2:
                main.wait_event(self.pull_done[l - 1])
            self._layer(l, h, Ws[l - 1])
            if do_push and l <= self.L - 1:
                self.io.wait_stream(main)
                with torch.cuda.stream(self.io):
                    D.digest_push(self.p, l, self.H[l], stores[l], stream=self.io)
            h = self.H[l]
        if pulled or do_push:
            main.wait_stream(self.io)
        return self.H[self.L]

    def _forward_in_line(self, x_own, Ws, stores, do_pull, do_push):
        h = x_own
        for l in range(1, self.L + 1):
            if do_pull and l >= 2:
                D.digest_pull(self.p, l - 1, stores[l - 1])
            self._layer(l, h, Ws[l - 1])
            if do_push and l <= self.L - 1:
                D.digest_push(self.p, l, self.H[l], stores[l])
            h = self.H[l]
        return self.H[self.L]

    def backward(self, Ws, labels):
        D.digest_softmax_xent(self.p, self.H[self.L], labels, self.dH[self.L], self.loss)
        for l in range(self.L, 0, -1):
            dh_in = self.dH[l - 1] if l > 1 else None
            h_in = self.H[l - 1] if l > 1 else self.x_own
            if self.model == "gat":
                D.digest_gat_backward(self.p, l, h_in, self.H[l], self.dH[l], Ws[l - 1],
                                      self.atts[l - 1], self.dW[l], self.dAtt[l], dh_in)
            else:
                D.digest_layer_backward(self.p, l, h_in, self.H[l], self.dH[l], Ws[l - 1],
                                        self.dW[l], dh_in)

    def round(self, r, K, x_own, Ws, stores, labels):
        """Round r (1-based) with sync interval K, eagerly."""
        do_pull, do_push = D.digest_sync_period(K, r)
        self.forward(x_own, Ws, stores, do_pull, do_push)
        self.backward(Ws, labels)

    def capture(self, K, x_own, Ws, stores, labels):
        """Record one HIP graph per pull/push pattern that the schedule uses."""
        patterns = sorted({D.digest_sync_period(K, r) for r in range(1, 2 * K + 1)})
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):   # warm-up outside capture
            for pat in patterns:
                self.forward(x_own, Ws, stores, *pat)
                self.backward(Ws, labels)
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        for pat in patterns:
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                self.forward(x_own, Ws, stores, *pat)
                self.backward(Ws, labels)
            self.graphs[(K, pat)] = g
        torch.cuda.synchronize()

    def replay(self, r, K):
        self.graphs[(K, D.digest_sync_period(K, r))].replay()
