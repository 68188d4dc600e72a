"""One SGD-momentum training step of the LeNet-style network, on the GPU library.

conv(1->32, 5x5, p2)+relu -> max-pool 2x2/2 -> conv(32->64, 5x5, p2)+relu ->
max-pool 2x2/2 -> affine 3136->512 + relu -> affine 512->10 -> softmax +
cross-entropy; backward in reverse order; then v <- mu v - lr g and
theta <- theta + v for the eight parameter tensors (paper, Section 2: the NN
library's layers, its minibatch training loop and SGD with momentum).  Each
conv+relu+pool runs as one fused call forward.  Backward, the pool backward
(relu mask folded in) writes the conv-output gradient and the plain conv
backward passes read it; with fused_pool_backward=True the conv passes
instead take the pool's gradient, argmax and pooled values directly (the
relu mask and the pool routing built while staging), so the conv-output
gradients are never stored (less memory, a slower step at this size).

All activations, gradients and the workspaces (backward-filter partials,
affine split partials) are allocated once; ``step`` only enqueues library
calls (about twenty launches, one of them the optimizer update over the flat
parameter buffer) on the current stream and, for the weight gradients of
affine 1 and conv2, on a second stream that joins the current one before the
step returns; it returns the loss as a device scalar.
"""
from __future__ import annotations

import torch

from . import dmlnn

PARAM_ORDER = ("W1", "b1", "W2", "b2", "W3", "b3", "W4", "b4")


class LeNetTrainer:
    def __init__(self, params: dict, N: int = 64, lr: float = 0.01, mu: float = 0.9,
                 dtype=torch.float64, device="cuda", fused_pool_backward: bool = False):
        self.N, self.lr, self.mu = N, lr, mu
        # False: the pool backward runs as its own kernel (max_pool2d_bwd_relu)
        # into a stored conv-output gradient, which the plain conv backward
        # calls read (the faster step at batch 64); True: the conv backward
        # passes read the pool gradients directly (no conv-output gradients)
        self.fused_pool_backward = fused_pool_backward
        kw = dict(dtype=dtype, device=device)
        # Parameters, gradients and velocities each live in one flat buffer (the
        # tensors are contiguous views into it), so the optimizer update of all
        # eight tensors is a single elementwise launch.
        shapes = {k: tuple(torch.as_tensor(params[k]).shape) for k in PARAM_ORDER}
        sizes = {k: int(torch.Size(sh).numel()) for k, sh in shapes.items()}
        total = sum(sizes.values())
        self.p_flat = torch.empty(total, **kw)
        self.g_flat = torch.empty(total, **kw)
        self.v_flat = torch.zeros(total, **kw)
        self.p, self.g, self.v = {}, {}, {}
        off = 0
        for k in PARAM_ORDER:
            n = sizes[k]
            for d, flat in ((self.p, self.p_flat), (self.g, self.g_flat), (self.v, self.v_flat)):
                d[k] = flat[off:off + n].view(shapes[k])
            self.p[k].copy_(torch.as_tensor(params[k]).to(**kw))
            off += n
        e = lambda *s: torch.empty(*s, **kw)  # noqa: E731
        i32 = lambda *s: torch.empty(*s, dtype=torch.int32, device=device)  # noqa: E731
        # conv outputs are never stored: the pools run in the convolutions'
        # epilogues and the pool backward folds in the relu mask (pooled > 0)
        self.p1, self.i1 = e(N, 32 * 196), i32(N, 32 * 196)
        self.p2, self.i2 = e(N, 64 * 49), i32(N, 64 * 49)
        self.h, self.s = e(N, 512), e(N, 10)
        self.loss, self.ds = e(1), e(N, 10)
        self.dh, self.dp2, self.dp1 = e(N, 512), e(N, 3136), e(N, 32 * 196)
        if not fused_pool_backward:
            self.dc2, self.dc1 = e(N, 64 * 196), e(N, 32 * 784)
        ws1 = dmlnn.conv2d_backward_filter_workspace_size(dtype, N, 1, 28, 28, 32, 5, 5, 1, 2)
        ws2 = dmlnn.conv2d_backward_filter_workspace_size(dtype, N, 32, 14, 14, 64, 5, 5, 1, 2)
        self.ws1 = torch.empty(ws1, dtype=torch.uint8, device=device)
        self.ws2 = torch.empty(ws2, dtype=torch.uint8, device=device)
        # split-reduction partials of the affine products: one buffer for the
        # current stream's products, one for the second stream's (affine 1 dW)
        wa = max(dmlnn.affine_workspace_size(dtype, N, 3136, 512),
                 dmlnn.affine_workspace_size(dtype, N, 512, 10))
        self.wsa = torch.empty(wa, dtype=torch.uint8, device=device)
        self.wsa_side = torch.empty(wa, dtype=torch.uint8, device=device)
        # the loss shares of softmax_xent's blocks (none at batch <= 64: one block)
        self.wss = torch.empty(dmlnn.softmax_xent_workspace_size(dtype, N, 10), dtype=torch.uint8,
                               device=device)
        # The weight gradients of affine 1 and conv2 run on a second stream
        # (default priority), beside the data-gradient chain (affine 1 dX, pool
        # backward, conv2 backward_data, ...): they only share read-only inputs,
        # and each kernel is too small to fill the GPU alone
        self.side = torch.cuda.Stream(device=device)
        self.ev_fork1, self.ev_fork2, self.ev_join = (torch.cuda.Event() for _ in range(3))
        self.two_streams = True

    def forward_backward(self, X, Y):
        p, g = self.p, self.g
        # Streams and events are passed explicitly (no stream contexts, no
        # events created per step): the step is a few dozen short launches, and
        # the host time to enqueue them is part of its time.
        ms = torch.cuda.current_stream()
        two = self.two_streams
        ss = self.side if two else ms
        dmlnn.conv2d_forward_pool(X, p["W1"], p["b1"], 1, 28, 28, 5, 5, 1, 2, 2, 2, 2, 0,
                                  pooled=self.p1, argmax=self.i1, stream=ms)
        dmlnn.conv2d_forward_pool(self.p1, p["W2"], p["b2"], 32, 14, 14, 5, 5, 1, 2, 2, 2, 2, 0,
                                  pooled=self.p2, argmax=self.i2, stream=ms)
        dmlnn.affine_fwd(self.p2, p["W3"], p["b3"], relu=True, out=self.h, workspace=self.wsa,
                         stream=ms)
        dmlnn.affine_fwd(self.h, p["W4"], p["b4"], relu=False, out=self.s, workspace=self.wsa,
                         stream=ms)
        dmlnn.softmax_xent(self.s, Y, want_probs=False, loss=self.loss, dscores=self.ds,
                           workspace=self.wss, stream=ms)
        # dh comes out masked by h > 0 (the relu backward of affine 1, folded
        # into this product), so affine 1's backward reads no mask
        dmlnn.affine_bwd(self.ds, self.h, p["W4"], None, dX=self.dh, dW=g["W4"], db=g["b4"],
                         workspace=self.wsa, relu_input=True, stream=ms)
        if two:  # fork: dh is ready
            self.ev_fork1.record(ms)
            ss.wait_event(self.ev_fork1)
        dmlnn.affine_bwd(self.dh, self.p2, p["W3"], None, want_dX=False, dW=g["W3"],
                         db=g["b3"], workspace=self.wsa_side, stream=ss)
        dmlnn.affine_bwd(self.dh, self.p2, p["W3"], None, dX=self.dp2, want_dW=False,
                         want_db=False, workspace=self.wsa, stream=ms)
        if self.fused_pool_backward:
            if two:  # fork: dp2 is ready
                self.ev_fork2.record(ms)
                ss.wait_event(self.ev_fork2)
            dmlnn.conv2d_backward_filter_pooled(self.p1, self.dp2, self.i2, self.p2, 32, 14,
                                                14, 5, 5, 1, 2, 64, 2, 2, 2, 0,
                                                workspace=self.ws2, dW=g["W2"], db=g["b2"],
                                                stream=ss)
            dmlnn.conv2d_backward_data_pooled(p["W2"], self.dp2, self.i2, self.p2, 32, 14, 14, 5,
                                              5, 1, 2, 2, 2, 2, 0, dX=self.dp1, stream=ms)
            dmlnn.conv2d_backward_filter_pooled(X, self.dp1, self.i1, self.p1, 1, 28, 28, 5, 5, 1,
                                                2, 32, 2, 2, 2, 0, workspace=self.ws1,
                                                dW=g["W1"], db=g["b1"], stream=ms)
        else:
            dmlnn.max_pool2d_bwd_relu(self.dp2, self.i2, self.p2, 64, 14, 14, 2, 2, 2, 0,
                                      dX=self.dc2, stream=ms)
            if two:  # fork: dc2 is ready
                self.ev_fork2.record(ms)
                ss.wait_event(self.ev_fork2)
            dmlnn.conv2d_backward_filter(self.p1, self.dc2, None, 32, 14, 14, 5, 5, 1, 2, 64,
                                         workspace=self.ws2, dW=g["W2"], db=g["b2"], stream=ss)
            dmlnn.conv2d_backward_data(p["W2"], self.dc2, None, 32, 14, 14, 5, 5, 1, 2,
                                       dX=self.dp1, stream=ms)
            dmlnn.max_pool2d_bwd_relu(self.dp1, self.i1, self.p1, 32, 28, 28, 2, 2, 2, 0,
                                      dX=self.dc1, stream=ms)
            dmlnn.conv2d_backward_filter(X, self.dc1, None, 1, 28, 28, 5, 5, 1, 2, 32,
                                         workspace=self.ws1, dW=g["W1"], db=g["b1"], stream=ms)
        # join: the optimizer reads the side stream's gradients, and the next
        # step's forward overwrites p1 and p2, which the side stream reads
        if two:
            self.ev_join.record(ss)
            ms.wait_event(self.ev_join)
        return self.loss

    def step(self, X, Y):
        loss = self.forward_backward(X, Y)
        dmlnn.sgd_momentum_update(self.p_flat, self.g_flat, self.v_flat, self.lr, self.mu)
        return loss

    # --- HIP graph form of the step ----------------------------------------
    # The step is a fixed sequence of launches on fixed buffers, so it can be
    # recorded once into a HIP graph and replayed: one submission instead of
    # seventeen, and no host work between kernels.  The batch is read from
    # static input buffers (copy a new batch into them before a replay).
    def capture(self, X, Y, warmup: int = 1):
        """Record one training step reading X, Y (copied into static buffers).
        The warm-up steps run eagerly first (they update the parameters)."""
        self.X_static = X.clone()
        self.Y_static = Y.clone()
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            for _ in range(warmup):  # kernel attributes and occupancy queries happen here
                self.step(self.X_static, self.Y_static)
        torch.cuda.current_stream().wait_stream(side)
        # The graph holds the single-stream form of the step: replayed, the
        # two-stream form ran its branches one after the other with extra
        # dependency overhead (0.343 ms against 0.333 ms single-stream).
        self.graph = torch.cuda.CUDAGraph()
        self.two_streams = False
        try:
            with torch.cuda.graph(self.graph):
                self.graph_loss = self.step(self.X_static, self.Y_static)
        finally:
            self.two_streams = True
        return self.graph

    def replay(self, X=None, Y=None):
        """One training step from the recorded graph (optionally on a new batch)."""
        if X is not None:
            self.X_static.copy_(X)
        if Y is not None:
            self.Y_static.copy_(Y)
        self.graph.replay()
        return self.graph_loss


class LeNetScorer:
    """Forward-only batched scoring of the same network (the paper's parfor-style
    scoring: every minibatch is independent, Section 3 "Distributed
    Operations"), on one GPU: the batches are dealt round-robin to ``streams``
    HIP streams, each with its own activation buffers, so the small per-batch
    kernels of different batches overlap.  Returns the class probabilities."""

    def __init__(self, params: dict, batch: int = 64, streams: int = 4,
                 dtype=torch.float64, device="cuda"):
        kw = dict(dtype=dtype, device=device)
        self.batch, self.dtype, self.device = batch, dtype, device
        self.p = {k: torch.as_tensor(v).to(**kw).contiguous() for k, v in params.items()}
        self.streams = [torch.cuda.Stream(device=device) for _ in range(streams)]
        e = lambda *s: torch.empty(*s, **kw)  # noqa: E731
        i32 = lambda *s: torch.empty(*s, dtype=torch.int32, device=device)  # noqa: E731
        B = batch
        wa = max(dmlnn.affine_workspace_size(dtype, B, 3136, 512),
                 dmlnn.affine_workspace_size(dtype, B, 512, 10))
        self.buf = [dict(p1=e(B, 32 * 196), i1=i32(B, 32 * 196),
                         p2=e(B, 64 * 49), i2=i32(B, 64 * 49),
                         h=e(B, 512), s=e(B, 10),
                         ws=torch.empty(wa, dtype=torch.uint8, device=device))
                    for _ in range(streams)]

    def _forward(self, X, out, b):
        p = self.p
        dmlnn.conv2d_forward_pool(X, p["W1"], p["b1"], 1, 28, 28, 5, 5, 1, 2, 2, 2, 2, 0,
                                  pooled=b["p1"], argmax=b["i1"])
        dmlnn.conv2d_forward_pool(b["p1"], p["W2"], p["b2"], 32, 14, 14, 5, 5, 1, 2, 2, 2, 2, 0,
                                  pooled=b["p2"], argmax=b["i2"])
        dmlnn.affine_fwd(b["p2"], p["W3"], p["b3"], relu=True, out=b["h"], workspace=b["ws"])
        dmlnn.affine_fwd(b["h"], p["W4"], p["b4"], relu=False, out=b["s"], workspace=b["ws"])
        dmlnn.softmax_fwd(b["s"], probs=out)

    def score(self, X):
        """X: M x 784 on the device (M a multiple of the batch size)."""
        M = X.shape[0]
        if M % self.batch:
            raise ValueError(f"{M} rows is not a multiple of the batch size {self.batch}")
        probs = torch.empty((M, 10), dtype=self.dtype, device=self.device)
        main = torch.cuda.current_stream()
        for s in self.streams:
            s.wait_stream(main)  # X and the parameters are ready
        for k in range(M // self.batch):
            j = k % len(self.streams)
            lo = k * self.batch
            with torch.cuda.stream(self.streams[j]):
                self._forward(X[lo:lo + self.batch], probs[lo:lo + self.batch], self.buf[j])
        for s in self.streams:
            main.wait_stream(s)
        return probs
