"""Benchmark: conv2d forward + backward_filter + backward_data (bias_add and relu
fused) of the ResNet-shaped layer N=256, C=64, 56x56, F=64, 3x3, stride 1, pad 1,
in fp64 on one MI355X, as GFLOP/s and a fraction of the fp64 matrix-core peak.

    python bench.py [--gpus 1] [--steps K] [--warmup W]

One step = the three conv passes over one batch already resident in HBM.  The
timed region is bracketed by device synchronisations; per-pass durations come
from HIP events recorded on the stream the kernels are launched on.  Also
reported (extra keys): the fp32 mode of the same layer, the LeNet-style
training step (batch 64, fp64) in images/s, and the oracle timed on a bounded
sample of the same layer on the host's cores.  Prints one JSON line.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import platform
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_F64_MFMA = 78.6      # TFLOP/s, MI355X dense fp64 matrix
PEAK_F32_MFMA = 157.3     # TFLOP/s, MI355X dense fp32 matrix
PEAK_HBM_TBPS = 8.0       # TB/s, MI355X HBM3E
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "conv_hbm_traffic_resnet_fp64.txt")


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu", action="store_true", help="skip the oracle baseline")
    ap.add_argument("--separate-mask", action="store_true",
                    help="time the step with both backward passes applying the relu mask "
                         "(no masked gradient handed from backward_filter to backward_data)")
    ap.add_argument("--zero-skip-probe", action="store_true",
                    help="only run the config 2 zero-skip measurement (for counter runs)")
    ap.add_argument("--only-f64", action="store_true",
                    help="skip the fp32, LeNet, other-config and other-kernel extras")
    ap.add_argument("--only-f32", action="store_true",
                    help="only time the fp32 mode of the ResNet-shaped layer (for counter runs)")
    ap.add_argument("--only-aux", action="store_true",
                    help="only time the bandwidth-bound ops and the copy calibration (for "
                         "counter runs)")
    ap.add_argument("--only-lenet", action="store_true",
                    help="only time the LeNet training step (for kernel-trace runs)")
    ap.add_argument("--lenet-trace", choices=("fused", "unfused"),
                    help="only run the LeNet step in one form, eager and on one stream, so a "
                         "kernel trace of the run adds up to the step (fused: the conv backward "
                         "passes read the pool gradients; unfused: pool backward kernels first)")
    return ap.parse_args()


def kernel_source_sha() -> str:
    h = hashlib.sha256()
    for name in ("conv_igemm.hip", "conv_wgrad.hip", "common.hpp"):
        with open(os.path.join(ROOT, "paper_1802_04647_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic(pass_name: str):
    """HBM bytes per launch from the committed rocprofv3 counter summary, or None
    when absent or taken on a different kernel source."""
    try:
        with open(TRAFFIC_FILE) as f:
            text = f.read()
    except OSError:
        return None
    m = re.search(r"^source_sha=(\w+)", text, re.M)
    if not m or m.group(1) != kernel_source_sha():
        return None
    m = re.search(rf"^{pass_name}_hbm_bytes_per_launch=([0-9.eE+]+)", text, re.M)
    return float(m.group(1)) if m else None


def conv_step_timing(dtype_name, steps, warmup, emit=True):
    """The three passes of the ResNet-shaped layer, timed.  emit: backward_filter
    also writes the relu-masked gradient it stages (conv2d_backward_filter_emit)
    and backward_data takes it with no mask; else both passes take dout and the
    mask."""
    import torch
    from paper_1802_04647_amd import dmlnn
    from paper_1802_04647_amd.inputs import SHAPES, conv_layer_inputs

    s = SHAPES["resnet_conv"]
    tdt = torch.float64 if dtype_name == "f64" else torch.float32
    X0, W0, b0, dout0 = conv_layer_inputs("resnet_conv")
    dev = lambda a: torch.from_numpy(a).to(device="cuda", dtype=tdt)  # noqa: E731
    X, W, b, dout = dev(X0), dev(W0), dev(b0), dev(dout0)
    del X0, dout0
    a = (s.C, s.Hin, s.Win, s.Hf, s.Wf, s.stride, s.pad)
    out = torch.empty((s.N, s.F * s.Hout * s.Wout), dtype=tdt, device="cuda")
    dW = torch.empty_like(W)
    db = torch.empty_like(b)
    dX = torch.empty_like(X)
    ws = torch.empty(dmlnn.conv2d_backward_filter_workspace_size(tdt, *s.args()),
                     dtype=torch.uint8, device="cuda")
    g = torch.empty_like(dout) if emit else None

    def step(ev=None):
        if ev is not None:
            ev[0].record()
        dmlnn.conv2d_forward(X, W, b, *a, relu=True, out=out)
        if ev is not None:
            ev[1].record()
        dmlnn.conv2d_backward_filter(X, dout, out, *a, s.F, workspace=ws, dW=dW, db=db, g_out=g)
        if ev is not None:
            ev[2].record()
        if emit:
            dmlnn.conv2d_backward_data(W, g, None, *a, dX=dX)
        else:
            dmlnn.conv2d_backward_data(W, dout, out, *a, dX=dX)
        if ev is not None:
            ev[3].record()

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(steps)]
    t0 = time.perf_counter()
    for k in range(steps):
        step(evs[k])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    per = {"forward": 0.0, "backward_filter": 0.0, "backward_data": 0.0}
    for ev in evs:
        per["forward"] += ev[0].elapsed_time(ev[1])
        per["backward_filter"] += ev[1].elapsed_time(ev[2])
        per["backward_data"] += ev[2].elapsed_time(ev[3])
    per = {k: v / steps for k, v in per.items()}          # ms per launch
    flops = s.flops_per_pass()
    return dict(wall_s=wall, per_pass_ms=per, flops_per_pass=flops, N=s.N)


def lenet_timing(steps=50, warmup=10):
    import torch
    from paper_1802_04647_amd.inputs import lenet_train_inputs
    from paper_1802_04647_amd.lenet import LeNetTrainer

    X, Y, params = lenet_train_inputs()
    Xd = torch.from_numpy(X).cuda()
    Yd = torch.from_numpy(Y).cuda()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def eager_ms(tr):
        for _ in range(warmup):
            tr.step(Xd, Yd)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(steps):
            tr.step(Xd, Yd)
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / steps

    # the conv backward passes reading the pool gradients directly (the
    # step's form), and the pool backward as its own kernel, for comparison
    ms = eager_ms(LeNetTrainer(params))
    # the step's forms: conv backward from the pool gradients (fused) or after
    # the pool backward kernel (unfused), on one stream or two
    forms = {}
    for fused in (True, False):
        for two in (True, False):
            tr = LeNetTrainer(params, fused_pool_backward=fused)
            tr.two_streams = two
            forms[f"{'fused' if fused else 'unfused'}_{'two' if two else 'one'}_streams"] = \
                eager_ms(tr)
    # the same step recorded once as a HIP graph and replayed
    gtr = LeNetTrainer(params)
    gtr.capture(Xd, Yd, warmup=2)
    for _ in range(warmup):
        gtr.replay()
    torch.cuda.synchronize()
    e0.record()
    for _ in range(steps):
        gtr.replay()
    e1.record()
    torch.cuda.synchronize()
    gms = e0.elapsed_time(e1) / steps
    return dict(ms_per_step=ms, images_per_s=64.0 / (ms / 1e3), graph_ms_per_step=gms,
                graph_images_per_s=64.0 / (gms / 1e3), forms_ms_per_step=forms)


def lenet_trace(fused, steps, warmup):
    """The LeNet step in one form, eager on one stream (kernels back to back)."""
    import torch
    from paper_1802_04647_amd.inputs import lenet_train_inputs
    from paper_1802_04647_amd.lenet import LeNetTrainer

    X, Y, params = lenet_train_inputs()
    tr = LeNetTrainer(params, fused_pool_backward=fused)
    tr.two_streams = False
    Xd, Yd = torch.from_numpy(X).cuda(), torch.from_numpy(Y).cuda()
    for _ in range(warmup):
        tr.step(Xd, Yd)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        tr.step(Xd, Yd)
    e1.record()
    torch.cuda.synchronize()
    return {"form": "fused" if fused else "unfused", "streams": 1, "steps": steps,
            "ms_per_step": round(e0.elapsed_time(e1) / steps, 4)}


def _median_ms(fn, reps=20, warmup=5, with_min=False):
    """Median (and min) over reps of HIP-event timings on the current stream."""
    import torch
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(reps)]
    for e0, e1 in evs:
        e0.record()
        fn()
        e1.record()
    torch.cuda.synchronize()
    ts = sorted(e0.elapsed_time(e1) for e0, e1 in evs)
    return (ts[len(ts) // 2], ts[0]) if with_min else ts[len(ts) // 2]


def scoring_timing(M=4096):
    """Forward-only LeNet scoring of M images in batches of 64, on 1 and 4 streams."""
    import torch
    from paper_1802_04647_amd.inputs import lenet_train_inputs, sparse_uniform, streams
    from paper_1802_04647_amd.lenet import LeNetScorer

    _, _, params = lenet_train_inputs()
    g_x, g_mask = streams(977)[:2]
    X = torch.from_numpy(sparse_uniform(g_mask, g_x, (M, 784), keep=0.2)).cuda()
    res = {"images": M, "batch": 64, "dtype": "f64"}
    for ns in (1, 4):
        sc = LeNetScorer(params, batch=64, streams=ns)
        ms = _median_ms(lambda: sc.score(X), reps=5, warmup=2)
        res[f"streams_{ns}"] = {"ms": round(ms, 3), "images_per_s": round(M / (ms / 1e3), 1)}
    return res


def horizontal_fusion_timing():
    """Three 3x3 filter banks (16, 16 and 32 filters) over one 256 x 64 x 28x28
    input: one horizontally fused launch (the banks fill one 64-row tile, so each
    input tile is staged once for all of them) against three conv2d_forward
    calls (fp64)."""
    import torch
    from paper_1802_04647_amd import dmlnn

    g = torch.Generator(device="cuda").manual_seed(7)
    N, C, H, Fs = 256, 64, 28, (16, 16, 32)
    X = torch.relu(torch.randn((N, C * H * H), dtype=torch.float64, device="cuda", generator=g))
    Ws = [torch.randn((F, C * 9), dtype=torch.float64, device="cuda", generator=g) * 0.06
          for F in Fs]
    bs = [torch.zeros(F, dtype=torch.float64, device="cuda") for F in Fs]
    outs = [torch.empty((N, F * H * H), dtype=torch.float64, device="cuda") for F in Fs]
    Wcat, bcat = torch.cat(Ws).contiguous(), torch.cat(bs).contiguous()
    a = (C, H, H, 3, 3, 1, 1)
    fused = _median_ms(lambda: dmlnn.conv2d_forward_multi(X, Ws, bs, *a, outs=outs, Wcat=Wcat,
                                                          bcat=bcat))
    sep = _median_ms(lambda: [dmlnn.conv2d_forward(X, W, b, *a, out=o)
                              for W, b, o in zip(Ws, bs, outs)])
    flops = 2.0 * N * sum(Fs) * H * H * C * 9
    return {"shape": "256 x 64 x 28x28, banks of 16, 16 and 32 filters 3x3 p1, fp64",
            "fused_ms": round(fused, 4), "separate_ms": round(sep, 4),
            "fused_tflops": round(flops / (fused / 1e3) / 1e12, 3),
            "separate_tflops": round(flops / (sep / 1e3) / 1e12, 3)}


def pooled_backward_timing():
    """Backward of conv -> relu -> 2x2/2 max-pool on the ResNet-shaped layer
    (256 x 64 x 56x56, 64 filters 3x3 p1, fp64): both conv backward passes
    reading the pool's gradient, argmax and pooled values directly, against the
    pool backward kernel storing the conv-output gradient (411 MB) that the two
    passes then read."""
    import torch
    from paper_1802_04647_amd import dmlnn
    from paper_1802_04647_amd.inputs import SHAPES, conv_layer_inputs

    s = SHAPES["resnet_conv"]
    X0, W0, b0, _ = conv_layer_inputs("resnet_conv")
    X, W, b = (torch.from_numpy(v).cuda() for v in (X0, W0, b0))
    a = (s.C, s.Hin, s.Win, s.Hf, s.Wf, s.stride, s.pad)
    _, pooled, argmax, Hp, Wp = dmlnn.conv2d_forward_pool(X, W, b, *a, 2, 2, 2, 0)
    g = torch.Generator(device="cuda").manual_seed(13)
    dpool = torch.randn(pooled.shape, dtype=torch.float64, device="cuda", generator=g)
    ws = torch.empty(dmlnn.conv2d_backward_filter_workspace_size(torch.float64, *s.args()),
                     dtype=torch.uint8, device="cuda")
    dW, db = torch.empty_like(W), torch.empty_like(b)
    dX = torch.empty_like(X)
    dc = torch.empty((s.N, s.F * s.Hout * s.Wout), dtype=torch.float64, device="cuda")

    def fused():
        dmlnn.conv2d_backward_filter_pooled(X, dpool, argmax, pooled, *a, s.F, 2, 2, 2, 0,
                                            workspace=ws, dW=dW, db=db)
        dmlnn.conv2d_backward_data_pooled(W, dpool, argmax, pooled, *a, 2, 2, 2, 0, dX=dX)

    def unfused():
        dmlnn.max_pool2d_bwd_relu(dpool, argmax, pooled, s.F, s.Hout, s.Wout, 2, 2, 2, 0, dX=dc)
        dmlnn.conv2d_backward_filter(X, dc, None, *a, s.F, workspace=ws, dW=dW, db=db)
        dmlnn.conv2d_backward_data(W, dc, None, *a, dX=dX)

    f_ms = _median_ms(fused, reps=10, warmup=3)
    u_ms = _median_ms(unfused, reps=10, warmup=3)
    return {"shape": "256 x 64 x 56x56, 64 filters 3x3 p1, then relu and 2x2/2 max-pool, fp64",
            "fused_ms": round(f_ms, 4), "unfused_ms": round(u_ms, 4)}


def sparse_conv_timing():
    """conv2d forward of a CSR input against the dense forward of the same matrix:
    the LeNet conv1 layer (64 x 1x28x28, ~80% zeros) and a 256 x 16x56x56 input
    with 98% zeros (fp64)."""
    import numpy as np
    import torch
    from paper_1802_04647_amd import dmlnn
    from paper_1802_04647_amd.inputs import SHAPES, conv_layer_inputs

    def csr_of(Xd):
        # host-side CSR construction of the benchmark input (not timed)
        X = Xd.cpu().numpy()
        nz = X != 0
        rowptr = np.concatenate([[0], np.cumsum(nz.sum(axis=1))]).astype(np.int32)
        cols = np.nonzero(nz)[1].astype(np.int32)
        return (torch.from_numpy(rowptr).cuda(), torch.from_numpy(cols).cuda(),
                Xd[torch.from_numpy(nz).cuda()].contiguous())

    res = {}
    s = SHAPES["lenet_conv1"]
    X0, W0, b0, _ = conv_layer_inputs("lenet_conv1")
    cases = [("lenet_conv1", s, torch.from_numpy(X0).cuda(), torch.from_numpy(W0).cuda(),
              torch.from_numpy(b0).cuda())]
    g = torch.Generator(device="cuda").manual_seed(11)
    N, C, H, F = 256, 16, 56, 32
    Xs = torch.randn((N, C * H * H), dtype=torch.float64, device="cuda", generator=g)
    Xs[torch.rand(Xs.shape, device="cuda", generator=g) < 0.98] = 0.0
    from paper_1802_04647_amd.inputs import ConvShape
    cases.append(("sparse_98pct_256x16x56x56", ConvShape(N, C, H, H, F, 3, 3, 1, 1), Xs,
                  torch.randn((F, C * 9), dtype=torch.float64, device="cuda", generator=g) * 0.1,
                  torch.zeros(F, dtype=torch.float64, device="cuda")))
    for name, s, X, W, b in cases:
        rowptr, cols, vals = csr_of(X)
        a = (s.C, s.Hin, s.Win, s.Hf, s.Wf, s.stride, s.pad)
        out = torch.empty((s.N, s.F * s.Hout * s.Wout), dtype=torch.float64, device="cuda")
        ri = torch.empty(s.N * s.C * s.Hin + 1, dtype=torch.int32, device="cuda")
        csr_ms = _median_ms(lambda: dmlnn.conv2d_forward_csr(rowptr, cols, vals, W, b, *a,
                                                             out=out, row_index=ri))
        dense_ms = _median_ms(lambda: dmlnn.conv2d_forward(X, W, b, *a, out=out))
        res[name] = {"density": round(vals.numel() / X.numel(), 4), "csr_ms": round(csr_ms, 4),
                     "dense_ms": round(dense_ms, 4),
                     "csr_bytes": int(vals.numel() * 12 + rowptr.numel() * 4),
                     "dense_bytes": int(X.numel() * 8)}
    return res


def _reach_counts(H, Hf, S, P, Hout):
    """For each input row h: the number of output rows whose window covers h."""
    import numpy as np
    cnt = np.zeros(H, dtype=np.int64)
    for oh in range(Hout):
        for i in range(Hf):
            h = oh * S + i - P
            if 0 <= h < H:
                cnt[h] += 1
    return cnt


def zero_skip_timing():
    """The three conv passes with the zero-fragment skip off and on, on the
    workloads of configs 2, 3 and 5 with their own zeros, plus a structured-zero
    supplement (config 2's draw with a 6-pixel zero border), fp64.  Config 3's
    backward passes take the pooled gradient (>= 75% zeros) with the conv output
    as relu mask; the others the workload's dout and mask.  Per pass: median ms
    of each mode; the forward also reports the nnz-based algorithmic work
    2*F*sum over non-zero inputs of the outputs each reaches.  (The MFMA counts
    of each mode come from a counter run of --zero-skip-probe.)"""
    import numpy as np
    import torch
    from paper_1802_04647_amd import dmlnn
    from paper_1802_04647_amd.inputs import SHAPES, conv_layer_inputs

    def workload(name, structured=False):
        s = SHAPES[name]
        X0, W0, b0, d0 = conv_layer_inputs(name)
        if structured:
            Xs = X0.reshape(s.N, s.C, s.Hin, s.Win).copy()
            for sl in (np.s_[:, :, :6, :], np.s_[:, :, -6:, :], np.s_[:, :, :, :6], np.s_[:, :, :, -6:]):
                Xs[sl] = 0.0
            X0 = Xs.reshape(s.N, -1)
        return s, X0, W0, b0, d0

    res = {}
    for label, name, structured in (("config2", "lenet_conv1", False),
                                    ("config2_structured_zeros", "lenet_conv1", True),
                                    ("config3", "lenet_conv2", False),
                                    ("config5", "resnet_conv", False)):
        s, X0, W0, b0, d0 = workload(name, structured)
        a = (s.C, s.Hin, s.Win, s.Hf, s.Wf, s.stride, s.pad)
        X, W, b = (torch.from_numpy(np.ascontiguousarray(v)).cuda() for v in (X0, W0, b0))
        out = torch.empty((s.N, s.F * s.Hout * s.Wout), dtype=torch.float64, device="cuda")
        dmlnn.conv2d_forward(X, W, b, *a, out=out)
        if name == "lenet_conv2":
            # the pooled gradient routed back through the 2x2/2 pool of the output
            _, idx, _, _ = dmlnn.max_pool2d_fwd(out, s.F, s.Hout, s.Wout, 2, 2, 2, 0)
            dout = dmlnn.max_pool2d_bwd(torch.from_numpy(d0).cuda(), idx, s.F, s.Hout, s.Wout,
                                        2, 2, 2, 0)
        else:
            dout = torch.from_numpy(d0).cuda()
        dW, db, dX = torch.empty_like(W), torch.empty_like(b), torch.empty_like(X)
        ws = torch.empty(dmlnn.conv2d_backward_filter_workspace_size(torch.float64, *s.args()),
                         dtype=torch.uint8, device="cuda")
        rh = _reach_counts(s.Hin, s.Hf, s.stride, s.pad, s.Hout)
        rw = _reach_counts(s.Win, s.Wf, s.stride, s.pad, s.Wout)
        nz = X0.reshape(s.N, s.C, s.Hin, s.Win) != 0
        nnz_flops = 2.0 * s.F * float((nz * np.outer(rh, rw)).sum())
        row = {"x_zero_fraction": round(float(np.mean(X0 == 0)), 4),
               "g_zero_fraction": round(float(((dout == 0) | (out <= 0)).double().mean()), 4),
               "dense_gflop_per_pass": round(s.flops_per_pass() / 1e9, 4),
               "forward_nnz_gflop": round(nnz_flops / 1e9, 4)}
        fns = {"forward": lambda: dmlnn.conv2d_forward(X, W, b, *a, out=out),
               "backward_filter": lambda: dmlnn.conv2d_backward_filter(
                   X, dout, out, *a, s.F, workspace=ws, dW=dW, db=db),
               "backward_data": lambda: dmlnn.conv2d_backward_data(W, dout, out, *a, dX=dX)}
        reps = 10 if name == "resnet_conv" else 20
        for pname, fn in fns.items():
            for mode in (0, 1):
                prev = dmlnn.set_zero_skip(mode)
                ms = _median_ms(fn, reps=reps, warmup=3)
                dmlnn.set_zero_skip(prev)
                row.setdefault(pname, {})["skip_ms" if mode else "dense_ms"] = round(ms, 4)
        res[label] = row
    return res


def conv_config_timing():
    """Per-pass GFLOP/s of the LeNet conv layers (configs 2 and 3) in fp64 and fp32."""
    import torch
    from paper_1802_04647_amd import dmlnn
    from paper_1802_04647_amd.inputs import SHAPES, conv_layer_inputs

    res = {}
    for name in ("lenet_conv1", "lenet_conv2"):
        s = SHAPES[name]
        X0, W0, b0, dout0 = conv_layer_inputs(name)
        if dout0.size != s.N * s.F * s.Hout * s.Wout:
            # config 3's stored upstream gradient is the pooled one; the conv
            # passes take one of the conv output's shape
            import numpy as np
            dout0 = np.random.default_rng(3).standard_normal((s.N, s.F * s.Hout * s.Wout))
        res[name] = {}
        for dtn, tdt, peak in (("f64", torch.float64, PEAK_F64_MFMA),
                               ("f32", torch.float32, PEAK_F32_MFMA)):
            dev = lambda v: torch.from_numpy(v).to(device="cuda", dtype=tdt)  # noqa: E731
            X, W, b, dout = dev(X0), dev(W0), dev(b0), dev(dout0)
            a = (s.C, s.Hin, s.Win, s.Hf, s.Wf, s.stride, s.pad)
            out = torch.empty((s.N, s.F * s.Hout * s.Wout), dtype=tdt, device="cuda")
            dW, db, dX = torch.empty_like(W), torch.empty_like(b), torch.empty_like(X)
            ws = torch.empty(dmlnn.conv2d_backward_filter_workspace_size(tdt, *s.args()),
                             dtype=torch.uint8, device="cuda")
            dmlnn.conv2d_forward(X, W, b, *a, relu=True, out=out)
            fns = {
                "forward": lambda: dmlnn.conv2d_forward(X, W, b, *a, relu=True, out=out),
                "backward_filter": lambda: dmlnn.conv2d_backward_filter(
                    X, dout, out, *a, s.F, workspace=ws, dW=dW, db=db),
                "backward_data": lambda: dmlnn.conv2d_backward_data(W, dout, out, *a, dX=dX),
            }
            flops = s.flops_per_pass()
            res[name][dtn] = {}
            for pname, fn in fns.items():
                ms, mn = _median_ms(fn, with_min=True)
                tf = flops / (ms / 1e3) / 1e12
                res[name][dtn][pname] = {"ms": round(ms, 4), "min_ms": round(mn, 4),
                                         "tflops": round(tf, 3),
                                         "pct_of_mfma_peak": round(100 * tf / peak, 2),
                                         "images_per_s": round(s.N / (ms / 1e3), 1)}
    return res


def aux_kernel_timing():
    """HBM rate of the bandwidth-bound ops (bytes each operand moves once, over the
    median launch time), and the affine GEMMs of the LeNet step in TFLOP/s."""
    import torch
    from paper_1802_04647_amd import dmlnn

    f64 = torch.float64
    res = {}

    def hbm(name, nbytes, fn, note):
        ms = _median_ms(fn)
        gbps = nbytes / (ms / 1e3) / 1e9
        res[name] = {"ms": round(ms, 4), "bytes": int(nbytes), "gbps": round(gbps, 1),
                     "pct_of_hbm_peak": round(100 * gbps / (PEAK_HBM_TBPS * 1e3), 2),
                     "shape": note}

    g = torch.Generator(device="cuda").manual_seed(1802)
    # bias_add_relu on the ResNet activation shape (256 x 64*56*56)
    X = torch.randn((256, 64 * 3136), dtype=f64, device="cuda", generator=g)
    b = torch.randn(64, dtype=f64, device="cuda", generator=g)
    out = torch.empty_like(X)
    hbm("bias_add_relu", 2 * X.numel() * 8 + 64 * 8,
        lambda: dmlnn.bias_add_relu(X, b, 64, 3136, relu=True, out=out),
        "256 x (64*56*56) fp64, separate output")
    # max_pool2d 2x2/2 on the same activation
    pout = torch.empty((256, 64 * 28 * 28), dtype=f64, device="cuda")
    idx = torch.empty((256, 64 * 28 * 28), dtype=torch.int32, device="cuda")
    hbm("max_pool2d_fwd", X.numel() * 8 + pout.numel() * 12,
        lambda: dmlnn.max_pool2d_fwd(X, 64, 56, 56, 2, 2, 2, 0, out=pout, argmax=idx),
        "256 x 64 x 56x56 -> 28x28, 2x2 stride 2, fp64 + int32 argmax")
    dX = torch.empty_like(X)
    hbm("max_pool2d_bwd", pout.numel() * 12 + X.numel() * 8,
        lambda: dmlnn.max_pool2d_bwd(pout, idx, 64, 56, 56, 2, 2, 2, 0, dX=dX),
        "256 x 64 x 28x28 -> 56x56 gather, fp64")
    del X, out, pout, idx, dX
    # LeNet pool2 (config 3): latency-bound size
    Xs = torch.randn((64, 64 * 196), dtype=f64, device="cuda", generator=g)
    ps = torch.empty((64, 64 * 49), dtype=f64, device="cuda")
    ids = torch.empty((64, 64 * 49), dtype=torch.int32, device="cuda")
    hbm("max_pool2d_fwd_lenet", Xs.numel() * 8 + ps.numel() * 12,
        lambda: dmlnn.max_pool2d_fwd(Xs, 64, 14, 14, 2, 2, 2, 0, out=ps, argmax=ids),
        "64 x 64 x 14x14 -> 7x7 (config 3), fp64; 8.8 MB, resident in the 256 MB MALL "
        "across reps")
    # SGD-momentum over the LeNet parameter count (config 4)
    n = 1663370
    th = torch.randn(n, dtype=f64, device="cuda", generator=g)
    gr = torch.randn(n, dtype=f64, device="cuda", generator=g)
    v = torch.zeros(n, dtype=f64, device="cuda")
    hbm("sgd_momentum_update", 5 * n * 8,
        lambda: dmlnn.sgd_momentum_update(th, gr, v, 0.01, 0.9),
        "1,663,370 fp64 parameters (LeNet), theta/grad/v read, theta/v written")
    # softmax + cross-entropy (config 4)
    S = torch.randn((64, 10), dtype=f64, device="cuda", generator=g)
    Y = torch.zeros((64, 10), dtype=f64, device="cuda")
    Y[torch.arange(64), torch.arange(64) % 10] = 1.0
    loss = torch.empty(1, dtype=f64, device="cuda")
    dS = torch.empty_like(S)
    P = torch.empty_like(S)
    hbm("softmax_xent", 4 * S.numel() * 8 + 8,
        lambda: dmlnn.softmax_xent(S, Y, loss=loss, dscores=dS, probs=P),
        "64 x 10 fp64 (config 4): latency-bound")
    # the same op over a large batch: the rows spread over 2048 blocks
    NL = 1 << 21
    SL = torch.randn((NL, 10), dtype=f64, device="cuda", generator=g)
    YL = torch.zeros((NL, 10), dtype=f64, device="cuda")
    YL[torch.arange(NL, device="cuda"), torch.arange(NL, device="cuda") % 10] = 1.0
    dSL, PL = torch.empty_like(SL), torch.empty_like(SL)
    wsl = torch.empty(dmlnn.softmax_xent_workspace_size(f64, NL, 10), dtype=torch.uint8,
                      device="cuda")
    hbm("softmax_xent_large", 4 * SL.numel() * 8 + 8,
        lambda: dmlnn.softmax_xent(SL, YL, loss=loss, dscores=dSL, probs=PL, workspace=wsl),
        f"{NL} x 10 fp64, scores and labels read, probs and dscores written")
    del SL, YL, dSL, PL
    # affine 3136 -> 512 of the LeNet step (config 4), fp64 MFMA
    A = torch.randn((64, 3136), dtype=f64, device="cuda", generator=g)
    Wa = torch.randn((3136, 512), dtype=f64, device="cuda", generator=g) * 0.02
    ba = torch.zeros(512, dtype=f64, device="cuda")
    oa = torch.empty((64, 512), dtype=f64, device="cuda")
    dA, dWa, dba = torch.empty_like(A), torch.empty_like(Wa), torch.empty_like(ba)
    go = torch.randn((64, 512), dtype=f64, device="cuda", generator=g)
    wsa = torch.empty(dmlnn.affine_workspace_size(f64, 64, 3136, 512), dtype=torch.uint8,
                      device="cuda")
    dmlnn.affine_fwd(A, Wa, ba, relu=True, out=oa, workspace=wsa)
    for nm, fn, fl in (("affine_fwd", lambda: dmlnn.affine_fwd(A, Wa, ba, relu=True, out=oa,
                                                               workspace=wsa),
                        2 * 64 * 3136 * 512),
                       ("affine_bwd", lambda: dmlnn.affine_bwd(go, A, Wa, out_fwd=oa, dX=dA,
                                                               dW=dWa, db=dba, workspace=wsa),
                        2 * 2 * 64 * 3136 * 512)):
        ms = _median_ms(fn)
        tf = fl / (ms / 1e3) / 1e12
        res[nm] = {"ms": round(ms, 4), "tflops": round(tf, 3),
                   "pct_of_fp64_mfma_peak": round(100 * tf / PEAK_F64_MFMA, 2),
                   "shape": "64 x 3136 . 3136 x 512 fp64 (config 4)"}
    return res


def copy_calibration(nbytes=1 << 30, reps=5):
    """A plain device-to-device copy of known size: the achievable HBM rate, and the
    reference kernel whose FETCH_SIZE / WRITE_SIZE counters calibrate the byte
    counts of the conv kernels."""
    import torch
    x = torch.ones(nbytes // 8, dtype=torch.float64, device="cuda")
    y = torch.empty_like(x)
    y.copy_(x)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        y.copy_(x)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    return {"bytes_moved": 2 * nbytes, "ms": round(ms, 4), "gbps": round(2 * nbytes / ms / 1e6, 1)}


def cpu_baseline(target_s=12.0):
    """The oracle (plain nested loops, OpenMP over independent outputs) on a bounded
    sample of the same layer: the three passes over n images."""
    import numpy as np  # noqa: F401
    import oracle
    from paper_1802_04647_amd.inputs import SHAPES, conv_layer_inputs

    s = SHAPES["resnet_conv"]
    cores = len(os.sched_getaffinity(0))
    oracle.set_threads(cores)
    a = (s.C, s.Hin, s.Win, s.Hf, s.Wf, s.stride, s.pad)

    def run(n):
        X, W, b, dout = conv_layer_inputs("resnet_conv", N=n)
        t = time.perf_counter()
        out, _, _ = oracle.conv2d_forward(X, W, b, *a)
        oracle.conv2d_backward_filter(X, dout, out, *a, s.F)
        oracle.conv2d_backward_data(W, dout, out, *a)
        return time.perf_counter() - t

    t1 = run(1)
    n = int(max(1, min(s.N, round(target_s / max(t1, 1e-3)))))
    t = run(n) if n > 1 else t1
    flops = 3 * 2.0 * n * s.F * s.Hout * s.Wout * s.K
    cpu = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            m = re.search(r"model name\s*:\s*(.*)", f.read())
            cpu = m.group(1).strip() if m else platform.processor()
    except OSError:
        pass
    return {"value": round(flops / t / 1e9, 3), "unit": "GFLOP/s", "cores": oracle.get_threads(),
            "kind": "oracle",
            "sample": f"fwd+bwd_filter+bwd_data of the 64->64 56x56 3x3 layer on {n} of 256 "
                      f"images, fp64, {t:.2f} s wall, {cpu}"}


def cpu_baselines_lenet(target_s=4.0):
    """The oracle on bounded samples of the LeNet-scale workloads: the three conv
    passes of each LeNet layer (fp64 GFLOP/s) and the whole training step
    (images/s), each on as many images as fit about target_s seconds."""
    import numpy as np
    import oracle
    from oracle import lenet as lenet_oracle
    from paper_1802_04647_amd.inputs import SHAPES, conv_layer_inputs, lenet_train_inputs

    cores = len(os.sched_getaffinity(0))
    oracle.set_threads(cores)
    res = {}
    for name in ("lenet_conv1", "lenet_conv2"):
        s = SHAPES[name]
        a = (s.C, s.Hin, s.Win, s.Hf, s.Wf, s.stride, s.pad)

        def run(n):
            X, W, b, _ = conv_layer_inputs(name, N=n)
            dout = np.random.default_rng(3).standard_normal((n, s.F * s.Hout * s.Wout))
            t = time.perf_counter()
            out, _, _ = oracle.conv2d_forward(X, W, b, *a)
            oracle.conv2d_backward_filter(X, dout, out, *a, s.F)
            oracle.conv2d_backward_data(W, dout, out, *a)
            return time.perf_counter() - t

        t1 = run(1)
        n = int(max(1, min(s.N, round(target_s / max(t1, 1e-3)))))
        t = run(n) if n > 1 else t1
        res[name] = {"value": round(3 * 2.0 * n * s.F * s.Hout * s.Wout * s.K / t / 1e9, 3),
                     "unit": "GFLOP/s", "cores": oracle.get_threads(), "kind": "oracle",
                     "sample": f"fwd+bwd_filter+bwd_data on {n} of {s.N} images, fp64, "
                               f"{t:.2f} s wall"}

    def step(n):
        X, Y, params = lenet_train_inputs(n)
        vel = lenet_oracle.zero_velocities(params)
        t = time.perf_counter()
        lenet_oracle.train_step(X, Y, params, vel)
        return time.perf_counter() - t

    t1 = step(1)
    n = int(max(1, min(64, round(target_s / max(t1, 1e-3)))))
    t = step(n) if n > 1 else t1
    res["lenet_train"] = {"value": round(n / t, 2), "unit": "images/s",
                          "cores": oracle.get_threads(), "kind": "oracle",
                          "sample": f"one SGD-momentum training step on {n} of 64 images, fp64, "
                                    f"{t:.2f} s wall"}
    return res


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); this library has "
              "no multi-GPU path (how the layer would shard is described in its design notes).",
              file=sys.stderr)
        sys.exit(2)
    import torch
    if not torch.cuda.is_available():
        print("no GPU available", file=sys.stderr)
        sys.exit(1)

    if args.zero_skip_probe:
        print(json.dumps({"zero_skip": zero_skip_timing()}), flush=True)
        return
    if args.only_f32:
        r32 = conv_step_timing("f32", args.steps, args.warmup)
        print(json.dumps({"f32_per_pass_ms": {k: round(v, 4) for k, v in
                                              r32["per_pass_ms"].items()}}), flush=True)
        return
    if args.only_aux:
        print(json.dumps({"aux_kernels": aux_kernel_timing(), "hbm_copy": copy_calibration()}),
              flush=True)
        return
    if args.lenet_trace:
        print(json.dumps({"lenet_trace": lenet_trace(args.lenet_trace == "fused", args.steps,
                                                     args.warmup)}), flush=True)
        return
    if args.only_lenet:
        lt = lenet_timing()
        forms = lt.pop("forms_ms_per_step")
        out = {k: round(v, 4) for k, v in lt.items()}
        out["forms_ms_per_step"] = {k: round(v, 4) for k, v in forms.items()}
        print(json.dumps({"lenet_training": out}), flush=True)
        return
    r = conv_step_timing("f64", args.steps, args.warmup, emit=not args.separate_mask)
    N, F3 = r["N"], 3 * r["flops_per_pass"]
    ms_step = r["wall_s"] * 1e3 / args.steps
    gflops = F3 / (ms_step / 1e3) / 1e9
    per = r["per_pass_ms"]
    dom = max(per, key=per.get)
    achieved = r["flops_per_pass"] / (per[dom] / 1e3) / 1e12
    sum_ms = sum(per.values())
    rec = {
        "metric": "conv2d fwd+bwd GFLOP/s and % of MFMA peak (fp64); training images/sec",
        "value": round(gflops, 1),
        "unit": "GFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64",
        "data": "synthetic (seeded relu(N(0,1)) activations, He-normal filters, N(0,1) upstream "
                "gradient)",
        "config": {"workload": "resnet_conv: conv2d 64->64, 56x56, 3x3, stride 1, pad 1, "
                               "bias_add+relu fused; forward + backward_filter + backward_data"
                               + ("" if args.separate_mask else
                                  " (backward_filter hands the relu-masked gradient to "
                                  "backward_data)"),
                   "global_batch": N, "seq_len": None, "parallelism": "single GPU"},
        "pct_of_fp64_mfma_peak": round(100.0 * gflops / 1e3 / PEAK_F64_MFMA, 2),
        "images_per_s": round(N / (ms_step / 1e3), 1),
        "per_pass_ms": {k: round(v, 4) for k, v in per.items()},
        "per_pass_tflops": {k: round(r["flops_per_pass"] / (v / 1e3) / 1e12, 3)
                            for k, v in per.items()},
        "event_sum_ms": round(sum_ms, 4),
        "roofline": {"bound": "mfma", "kernel": f"conv2d_{dom}", "achieved": round(achieved, 3),
                     "peak": PEAK_F64_MFMA, "unit": "TFLOP/s",
                     "frac": round(achieved / PEAK_F64_MFMA, 4),
                     "traffic": measured_traffic(dom)},
    }
    rec["hbm_copy"] = copy_calibration()
    if not args.only_f64 and not args.separate_mask:
        rs = conv_step_timing("f64", args.steps, args.warmup, emit=False)
        rec["separate_mask"] = {"ms_per_step": round(rs["wall_s"] * 1e3 / args.steps, 4),
                                "per_pass_ms": {k: round(v, 4) for k, v in
                                                rs["per_pass_ms"].items()}}
    if not args.only_f64:
        r32 = conv_step_timing("f32", args.steps, args.warmup)
        ms32 = r32["wall_s"] * 1e3 / args.steps
        rec["f32_mode"] = {"gflops": round(3 * r32["flops_per_pass"] / (ms32 / 1e3) / 1e9, 1),
                           "ms_per_step": round(ms32, 4),
                           "pct_of_fp32_mfma_peak": round(
                               100.0 * 3 * r32["flops_per_pass"] / (ms32 / 1e3) / 1e12
                               / PEAK_F32_MFMA, 2),
                           "per_pass_ms": {k: round(v, 4) for k, v in r32["per_pass_ms"].items()}}
        lt = lenet_timing()
        rec["lenet_training"] = {"batch": 64, "dtype": "f64",
                                 "ms_per_step": round(lt["ms_per_step"], 4),
                                 "images_per_s": round(lt["images_per_s"], 1),
                                 "hip_graph_ms_per_step": round(lt["graph_ms_per_step"], 4),
                                 "hip_graph_images_per_s": round(lt["graph_images_per_s"], 1),
                                 "forms_ms_per_step": {k: round(v, 4) for k, v in
                                                       lt["forms_ms_per_step"].items()}}
        rec["lenet_scoring"] = scoring_timing()
        rec["conv_configs"] = conv_config_timing()
        rec["horizontal_fusion"] = horizontal_fusion_timing()
        rec["pooled_backward"] = pooled_backward_timing()
        rec["sparse_conv"] = sparse_conv_timing()
        rec["zero_skip"] = zero_skip_timing()
        rec["aux_kernels"] = aux_kernel_timing()
    if not args.no_cpu:
        rec["cpu_baseline"] = cpu_baseline()
        if not args.only_f64:
            rec["cpu_baselines_lenet"] = cpu_baselines_lenet()
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
