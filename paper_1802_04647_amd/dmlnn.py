"""Thin Python binding of libdmlnn.so (the C ABI in include/dmlnn.h).

Argument marshalling only: every function checks that its tensors are
contiguous device tensors of one floating dtype (float64 or float32), passes
their device pointers, sizes and torch's current HIP stream to the C entry
point of the same name, and raises :class:`DmlnnError` with the library's
message on a nonzero status.  Outputs not supplied by the caller are allocated
with ``torch.empty`` on the inputs' device (torch is used only for memory and
streams).  Every computation runs in the library's HIP kernels; there is no
fallback: if the library is missing, the first call raises.

Layer-level signatures follow the paper's DML layers (Section 2 and 3):
``conv2d_forward(X, W, b, C, Hin, Win, Hf, Wf, stride, pad)`` etc., with N and F
taken from the row counts of X and W.
"""
from __future__ import annotations

import ctypes
import os
import re

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libdmlnn.so")
HEADER_PATH = os.path.join(os.path.dirname(_HERE), "include", "dmlnn.h")

F64, F32 = 0, 1
_DT = {torch.float64: F64, torch.float32: F32}


class DmlnnError(RuntimeError):
    def __init__(self, name, status, msg):
        super().__init__(f"{name} failed with status {status}: {msg}")
        self.status = status


_lib = None
_vp = ctypes.c_void_p


class ConvPlan(ctypes.Structure):
    """dmlnn_conv_plan of include/dmlnn.h."""
    _fields_ = [(n, ctypes.c_int) for n in (
        "kernel", "zero_skip", "tile_m", "tile_pixels", "blocks", "chunk", "k_split", "splits",
        "window_width", "window_rows")] + [("lds_bytes", ctypes.c_size_t),
                                           ("workspace_bytes", ctypes.c_size_t)] + [
        (n, ctypes.c_int) for n in ("tile_stride", "k_chunk", "slice_stride", "stage_bytes",
                                    "window_bytes", "slice_bytes", "slice_vec", "g_stride",
                                    "row_slices", "pipelined", "fused", "row_staged")]


KERNELS = {1: "igemm_dma", 2: "igemm_reg", 3: "small_m", 4: "resident", 5: "wgrad_ring",
           6: "wgrad_tiles", 7: "wgrad_pool_sparse"}
PASSES = {"forward": 0, "backward_filter": 1, "backward_data": 2}
_i = ctypes.c_int


def load():
    """Load libdmlnn.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    # DMLNN_LIBRARY: another build of the same library (the host-sanitized copy
    # that the CPU sanitizer tests load)
    path = os.environ.get("DMLNN_LIBRARY") or LIB_PATH
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with "
                           "`python -m paper_1802_04647_amd.build`")
    lib = ctypes.CDLL(path)
    sig = {
        "conv2d_out_dim": (_i, [_i] * 4),
        "conv2d_forward": (_i, [_i, _vp, _vp, _vp, _vp] + [_i] * 10 + [_vp]),
        "conv2d_backward_filter_workspace_size": (ctypes.c_size_t, [_i] * 10),
        "conv2d_backward_filter": (_i, [_i, _vp, _vp, _vp, _vp, _vp] + [_i] * 9
                                   + [_vp, ctypes.c_size_t, _vp]),
        "conv2d_backward_filter_emit": (_i, [_i, _vp, _vp, _vp, _vp, _vp, _vp] + [_i] * 9
                                        + [_vp, ctypes.c_size_t, _vp]),
        "conv2d_backward_data": (_i, [_i, _vp, _vp, _vp, _vp] + [_i] * 9 + [_vp]),
        "conv2d_backward_filter_noalloc": (_i, [_i, _vp, _vp, _vp, _vp, _vp] + [_i] * 9 + [_vp]),
        "conv2d_backward_filter_pooled": (_i, [_i] + [_vp] * 6 + [_i] * 13
                                          + [_vp, ctypes.c_size_t, _vp]),
        "conv2d_backward_data_pooled": (_i, [_i] + [_vp] * 5 + [_i] * 13 + [_vp]),
        "dmlnn_set_zero_skip": (_i, [_i]),
        "bias_add_relu": (_i, [_i, _vp, _vp, _vp] + [_i] * 4 + [_vp]),
        "max_pool2d_fwd": (_i, [_i, _vp, _vp, _vp] + [_i] * 8 + [_vp]),
        "max_pool2d_bwd": (_i, [_i, _vp, _vp, _vp] + [_i] * 8 + [_vp]),
        "affine_workspace_size": (ctypes.c_size_t, [_i] * 4),
        "affine_plan": (_i, [_i] * 5 + [ctypes.c_size_t] + [ctypes.POINTER(_i)] * 3),
        "affine_fwd": (_i, [_i, _vp, _vp, _vp, _vp] + [_i] * 4 + [_vp, ctypes.c_size_t, _vp]),
        "affine_bwd": (_i, [_i, _vp, _vp, _vp, _vp, _vp, _vp, _vp] + [_i] * 4
                       + [_vp, ctypes.c_size_t, _vp]),
        "softmax_xent": (_i, [_i, _vp, _vp, _vp, _vp, _vp, _i, _i, _vp, ctypes.c_size_t, _vp]),
        "softmax_xent_workspace_size": (ctypes.c_size_t, [_i, _i, _i]),
        "sgd_momentum_update": (_i, [_i, _vp, _vp, _vp, ctypes.c_double, ctypes.c_double,
                                     ctypes.c_longlong, _vp]),
        "softmax_fwd": (_i, [_i, _vp, _vp, _i, _i, _vp]),
        "conv2d_forward_pool": (_i, [_i] + [_vp] * 6 + [_i] * 14 + [_vp]),
        "conv2d_forward_multi": (_i, [_i, _vp, _vp, _vp, _vp, _vp] + [_i] * 10 + [_vp]),
        "conv2d_forward_csr": (_i, [_i, _vp, _vp, _vp, _i, _vp, _vp, _vp, _vp] + [_i] * 10
                               + [_vp]),
        "max_pool2d_bwd_relu": (_i, [_i, _vp, _vp, _vp, _vp] + [_i] * 8 + [_vp]),
        "sgd_update": (_i, [_i, _vp, _vp, ctypes.c_double, ctypes.c_longlong, _vp]),
        "sgd_nesterov_update": (_i, [_i, _vp, _vp, _vp, ctypes.c_double, ctypes.c_double,
                                     ctypes.c_longlong, _vp]),
        "adagrad_update": (_i, [_i, _vp, _vp, _vp, ctypes.c_double, ctypes.c_double,
                                ctypes.c_longlong, _vp]),
        "rmsprop_update": (_i, [_i, _vp, _vp, _vp] + [ctypes.c_double] * 3
                           + [ctypes.c_longlong, _vp]),
        "adam_update": (_i, [_i, _vp, _vp, _vp, _vp] + [ctypes.c_double] * 4
                        + [ctypes.c_longlong, ctypes.c_longlong, _vp]),
        "count_nonzero": (_i, [_i, _vp, ctypes.c_longlong, _vp, _vp]),
        "conv2d_plan": (_i, [_i] * 12 + [ctypes.POINTER(ConvPlan)]),
        "conv2d_plan_fused": (_i, [_i] * 17 + [ctypes.POINTER(ConvPlan)]),
        "conv2d_zero_skip_choice": (_i, [_i, _i, ctypes.c_longlong] + [_i] * 9),
        "dmlnn_last_error": (ctypes.c_char_p, []),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def header_symbols():
    """Names of the entry points declared in include/dmlnn.h."""
    with open(HEADER_PATH) as f:
        text = f.read()
    return re.findall(r"^DMLNN_API\s+(?:const\s+)?\w+\s*\**\s*(\w+)\s*\(", text, re.M)


def last_error() -> str:
    return load().dmlnn_last_error().decode()


def _check(name, rc):
    if rc != 0:
        raise DmlnnError(name, rc, last_error())


def _dtype(*ts):
    dt = None
    for t in ts:
        if t is None:
            continue
        d = _DT.get(t.dtype)
        if d is None:
            raise TypeError(f"unsupported dtype {t.dtype}; use float64 or float32")
        if dt is not None and d != dt:
            raise TypeError("all floating tensors of a call must share one dtype")
        dt = d
    return dt


def _p(t):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("dmlnn tensors must live on the GPU")
    if not t.is_contiguous():
        raise ValueError("dmlnn tensors must be contiguous")
    return t.data_ptr()


def _need(t, n, name):
    """Host-side guard: a buffer must hold exactly the elements the call will touch."""
    if t is not None and t.numel() != n:
        raise ValueError(f"{name} has {t.numel()} elements, the call needs {n}")


def _stream(stream=None):
    """The HIP stream a call is enqueued on: `stream` (a torch.cuda.Stream) when
    given, else the current stream.  Every call takes an optional stream=, so a
    caller that switches streams per call need not enter a stream context."""
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return stream.cuda_stream


def _empty(shape, like, dtype=None):
    return torch.empty(shape, dtype=dtype or like.dtype, device=like.device)


def conv2d_out_dim(Hin, Hf, stride, pad) -> int:
    return int(load().conv2d_out_dim(Hin, Hf, stride, pad))


def set_zero_skip(mode: int) -> int:
    """0 = dense, 1 = wavefront-ballot zero skip.  Returns the previous mode."""
    r = load().dmlnn_set_zero_skip(int(mode))
    if r < 0:
        raise ValueError(f"invalid zero-skip mode {mode}")
    return r


def conv2d_plan(dtype, pass_name, N, C, Hin, Win, F, Hf, Wf, stride, pad, zero_skip=0) -> dict:
    """The kernel and tiling a conv2d pass would take (host-only query, no GPU
    needed); ``kernel`` is named as in ``KERNELS``."""
    dt = _DT[dtype] if isinstance(dtype, torch.dtype) else int(dtype)
    plan = ConvPlan()
    _check("conv2d_plan", load().conv2d_plan(dt, PASSES[pass_name], N, C, Hin, Win, F, Hf, Wf,
                                             stride, pad, int(zero_skip), ctypes.byref(plan)))
    d = {name: getattr(plan, name) for name, _ in ConvPlan._fields_}
    d["kernel"] = KERNELS[plan.kernel]
    return d


FORMS = {"plain": 0, "pool_epilogue": 1, "pooled_source": 2, "csr_input": 3, "banks": 4}


def conv2d_plan_fused(dtype, pass_name, form, N, C, Hin, Win, F, Hf, Wf, stride, pad,
                      pool=(0, 0, 0, 0), zero_skip=0) -> dict:
    """conv2d_plan for a fused call: ``form`` as in ``FORMS``, ``pool`` =
    (pool_h, pool_w, pool_stride, pool_pad) for the two pool forms."""
    dt = _DT[dtype] if isinstance(dtype, torch.dtype) else int(dtype)
    plan = ConvPlan()
    ph, pw, ps, pp = pool
    _check("conv2d_plan_fused",
           load().conv2d_plan_fused(dt, PASSES[pass_name], FORMS[form], ph, pw, ps, pp, N, C, Hin,
                                    Win, F, Hf, Wf, stride, pad, int(zero_skip),
                                    ctypes.byref(plan)))
    d = {name: getattr(plan, name) for name, _ in ConvPlan._fields_}
    d["kernel"] = KERNELS[plan.kernel]
    return d


def conv2d_zero_skip_choice(dtype, pass_name, nnz, N, C, Hin, Win, F, Hf, Wf, stride, pad) -> int:
    """The zero-skip mode (0 or 1) the library's nnz rule picks for a pass whose
    staged operand has ``nnz`` non-zeros (host only)."""
    dt = _DT[dtype] if isinstance(dtype, torch.dtype) else int(dtype)
    r = load().conv2d_zero_skip_choice(dt, PASSES[pass_name], int(nnz), N, C, Hin, Win, F, Hf, Wf,
                                       stride, pad)
    if r < 0:
        raise ValueError("conv2d_zero_skip_choice: invalid arguments")
    return r


# ------------------------------------------------------------------------- conv2d
def conv2d_forward(X, W, b, C, Hin, Win, Hf, Wf, stride, pad, relu=True, out=None, stream=None):
    """out = relu(conv2d(X, W) + b): N x (F*Hout*Wout).  Returns (out, Hout, Wout)."""
    dt = _dtype(X, W, b, out)
    N, F = X.shape[0], W.shape[0]
    Hout, Wout = conv2d_out_dim(Hin, Hf, stride, pad), conv2d_out_dim(Win, Wf, stride, pad)
    if out is None:
        out = _empty((N, F * max(Hout, 0) * max(Wout, 0)), X)
    _need(X, N * C * Hin * Win, "X")
    _need(W, F * C * Hf * Wf, "W")
    _need(b, F, "b")
    _need(out, N * F * max(Hout, 0) * max(Wout, 0), "out")
    _check("conv2d_forward", load().conv2d_forward(
        dt, _p(X), _p(W), _p(b), _p(out), N, C, Hin, Win, F, Hf, Wf, stride, pad,
        int(bool(relu)), _stream(stream)))
    return out, Hout, Wout


def conv2d_backward_filter_workspace_size(dtype, N, C, Hin, Win, F, Hf, Wf, stride, pad) -> int:
    dt = _DT[dtype] if isinstance(dtype, torch.dtype) else int(dtype)
    return int(load().conv2d_backward_filter_workspace_size(dt, N, C, Hin, Win, F, Hf, Wf,
                                                            stride, pad))


def conv2d_backward_filter(X, dout, out_fwd, C, Hin, Win, Hf, Wf, stride, pad, F,
                           want_db=True, workspace=None, dW=None, db=None, g_out=None,
                           stream=None):
    """Returns (dW F x C*Hf*Wf, db F or None); out_fwd None means no relu mask.
    With g_out (an N x F*Hout*Wout buffer, possibly dout itself) the masked
    gradient is written there too (conv2d_backward_filter_emit), ready to be
    conv2d_backward_data's dout with out_fwd None."""
    dt = _dtype(X, dout, out_fwd, dW, db, g_out)
    N = X.shape[0]
    need = conv2d_backward_filter_workspace_size(dt, N, C, Hin, Win, F, Hf, Wf, stride, pad)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=X.device)
    if dW is None:
        dW = _empty((F, C * Hf * Wf), X)
    if db is None and want_db:
        db = _empty((F,), X)
    Hout, Wout = conv2d_out_dim(Hin, Hf, stride, pad), conv2d_out_dim(Win, Wf, stride, pad)
    _need(X, N * C * Hin * Win, "X")
    _need(dout, N * F * max(Hout, 0) * max(Wout, 0), "dout")
    _need(out_fwd, N * F * max(Hout, 0) * max(Wout, 0), "out_fwd")
    _need(dW, F * C * Hf * Wf, "dW")
    _need(db, F, "db")
    if g_out is not None:
        _need(g_out, N * F * max(Hout, 0) * max(Wout, 0), "g_out")
        _check("conv2d_backward_filter_emit", load().conv2d_backward_filter_emit(
            dt, _p(X), _p(dout), _p(out_fwd), _p(dW), _p(db), _p(g_out), N, C, Hin, Win, F, Hf,
            Wf, stride, pad, _p(workspace), workspace.numel() * workspace.element_size(),
            _stream(stream)))
        return dW, db
    _check("conv2d_backward_filter", load().conv2d_backward_filter(
        dt, _p(X), _p(dout), _p(out_fwd), _p(dW), _p(db), N, C, Hin, Win, F, Hf, Wf,
        stride, pad, _p(workspace), workspace.numel() * workspace.element_size(), _stream(stream)))
    return dW, db


def conv2d_backward_filter_noalloc(X, dout, out_fwd, C, Hin, Win, Hf, Wf, stride, pad, F, dW,
                                   db=None, stream=None):
    """conv2d_backward_filter with the library's own device scratch instead of a
    workspace: allocates nothing (dW, and db if wanted, are supplied)."""
    dt = _dtype(X, dout, out_fwd, dW, db)
    N = X.shape[0]
    Hout, Wout = conv2d_out_dim(Hin, Hf, stride, pad), conv2d_out_dim(Win, Wf, stride, pad)
    _need(X, N * C * Hin * Win, "X")
    _need(dout, N * F * max(Hout, 0) * max(Wout, 0), "dout")
    _need(out_fwd, N * F * max(Hout, 0) * max(Wout, 0), "out_fwd")
    _need(dW, F * C * Hf * Wf, "dW")
    _need(db, F, "db")
    _check("conv2d_backward_filter_noalloc", load().conv2d_backward_filter_noalloc(
        dt, _p(X), _p(dout), _p(out_fwd), _p(dW), _p(db), N, C, Hin, Win, F, Hf, Wf, stride, pad,
        _stream(stream)))
    return dW, db


def _pool_out(Hout, Wout, pool_h, pool_w, pool_stride, pool_pad):
    return (conv2d_out_dim(Hout, pool_h, pool_stride, pool_pad),
            conv2d_out_dim(Wout, pool_w, pool_stride, pool_pad))


def conv2d_backward_filter_pooled(X, dpool, argmax, pooled, C, Hin, Win, Hf, Wf, stride, pad, F,
                                  pool_h, pool_w, pool_stride, pool_pad, want_db=True,
                                  workspace=None, dW=None, db=None, stream=None):
    """Filter and bias gradients of conv -> relu -> max-pool from the pool's
    upstream gradient (dpool), argmax and pooled values.  Returns (dW, db)."""
    dt = _dtype(X, dpool, pooled, dW, db)
    N = X.shape[0]
    need = conv2d_backward_filter_workspace_size(dt, N, C, Hin, Win, F, Hf, Wf, stride, pad)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=X.device)
    if dW is None:
        dW = _empty((F, C * Hf * Wf), X)
    if db is None and want_db:
        db = _empty((F,), X)
    Hout, Wout = conv2d_out_dim(Hin, Hf, stride, pad), conv2d_out_dim(Win, Wf, stride, pad)
    Hp, Wp = _pool_out(Hout, Wout, pool_h, pool_w, pool_stride, pool_pad)
    _need(X, N * C * Hin * Win, "X")
    for t, name in ((dpool, "dpool"), (argmax, "argmax"), (pooled, "pooled")):
        _need(t, N * F * max(Hp, 0) * max(Wp, 0), name)
    if argmax.dtype != torch.int32:
        raise TypeError("argmax must be int32")
    _need(dW, F * C * Hf * Wf, "dW")
    _need(db, F, "db")
    _check("conv2d_backward_filter_pooled", load().conv2d_backward_filter_pooled(
        dt, _p(X), _p(dpool), _p(argmax), _p(pooled), _p(dW), _p(db), N, C, Hin, Win, F, Hf, Wf,
        stride, pad, pool_h, pool_w, pool_stride, pool_pad, _p(workspace),
        workspace.numel() * workspace.element_size(), _stream(stream)))
    return dW, db


def conv2d_backward_data_pooled(W, dpool, argmax, pooled, C, Hin, Win, Hf, Wf, stride, pad,
                                pool_h, pool_w, pool_stride, pool_pad, dX=None, stream=None):
    """Input gradient of conv -> relu -> max-pool from the pool's upstream
    gradient (dpool), argmax and pooled values: N x C*Hin*Win."""
    dt = _dtype(W, dpool, pooled, dX)
    N, F = dpool.shape[0], W.shape[0]
    Hout, Wout = conv2d_out_dim(Hin, Hf, stride, pad), conv2d_out_dim(Win, Wf, stride, pad)
    Hp, Wp = _pool_out(Hout, Wout, pool_h, pool_w, pool_stride, pool_pad)
    if dX is None:
        dX = _empty((N, C * Hin * Win), W)
    _need(W, F * C * Hf * Wf, "W")
    for t, name in ((dpool, "dpool"), (argmax, "argmax"), (pooled, "pooled")):
        _need(t, N * F * max(Hp, 0) * max(Wp, 0), name)
    if argmax.dtype != torch.int32:
        raise TypeError("argmax must be int32")
    _need(dX, N * C * Hin * Win, "dX")
    _check("conv2d_backward_data_pooled", load().conv2d_backward_data_pooled(
        dt, _p(W), _p(dpool), _p(argmax), _p(pooled), _p(dX), N, C, Hin, Win, F, Hf, Wf, stride,
        pad, pool_h, pool_w, pool_stride, pool_pad, _stream(stream)))
    return dX


def conv2d_backward_data(W, dout, out_fwd, C, Hin, Win, Hf, Wf, stride, pad, dX=None, stream=None):
    """Returns dX, N x (C*Hin*Win)."""
    dt = _dtype(W, dout, out_fwd, dX)
    N, F = dout.shape[0], W.shape[0]
    if dX is None:
        dX = _empty((N, C * Hin * Win), dout)
    Hout, Wout = conv2d_out_dim(Hin, Hf, stride, pad), conv2d_out_dim(Win, Wf, stride, pad)
    _need(W, F * C * Hf * Wf, "W")
    _need(dout, N * F * max(Hout, 0) * max(Wout, 0), "dout")
    _need(out_fwd, N * F * max(Hout, 0) * max(Wout, 0), "out_fwd")
    _need(dX, N * C * Hin * Win, "dX")
    _check("conv2d_backward_data", load().conv2d_backward_data(
        dt, _p(W), _p(dout), _p(out_fwd), _p(dX), N, C, Hin, Win, F, Hf, Wf, stride, pad,
        _stream(stream)))
    return dX


# -------------------------------------------------------------------------- others
def bias_add_relu(X, b, C, HW, relu=True, out=None, stream=None):
    dt = _dtype(X, b, out)
    if out is None:
        out = torch.empty_like(X)
    _need(X, X.shape[0] * C * HW, "X")
    _need(b, C, "b")
    _need(out, X.numel(), "out")
    _check("bias_add_relu", load().bias_add_relu(dt, _p(X), _p(b), _p(out), X.shape[0], C, HW,
                                                  int(bool(relu)), _stream(stream)))
    return out


def max_pool2d_fwd(X, C, Hin, Win, Hf, Wf, stride, pad, out=None, argmax=None, stream=None):
    """Returns (out, argmax int32, Hout, Wout)."""
    dt = _dtype(X, out)
    N = X.shape[0]
    Hout, Wout = conv2d_out_dim(Hin, Hf, stride, pad), conv2d_out_dim(Win, Wf, stride, pad)
    cols = C * max(Hout, 0) * max(Wout, 0)
    if out is None:
        out = _empty((N, cols), X)
    if argmax is None:
        argmax = _empty((N, cols), X, dtype=torch.int32)
    _need(X, N * C * Hin * Win, "X")
    _need(out, N * cols, "out")
    _need(argmax, N * cols, "argmax")
    _check("max_pool2d_fwd", load().max_pool2d_fwd(dt, _p(X), _p(out), _p(argmax), N, C, Hin,
                                                    Win, Hf, Wf, stride, pad, _stream(stream)))
    return out, argmax, Hout, Wout


def max_pool2d_bwd(dout, argmax, C, Hin, Win, Hf, Wf, stride, pad, dX=None, stream=None):
    dt = _dtype(dout, dX)
    if argmax.dtype != torch.int32:
        raise TypeError("argmax must be int32")
    N = dout.shape[0]
    if dX is None:
        dX = _empty((N, C * Hin * Win), dout)
    Hout, Wout = conv2d_out_dim(Hin, Hf, stride, pad), conv2d_out_dim(Win, Wf, stride, pad)
    _need(dout, N * C * max(Hout, 0) * max(Wout, 0), "dout")
    _need(argmax, N * C * max(Hout, 0) * max(Wout, 0), "argmax")
    _need(dX, N * C * Hin * Win, "dX")
    _check("max_pool2d_bwd", load().max_pool2d_bwd(dt, _p(dout), _p(argmax), _p(dX), N, C, Hin,
                                                    Win, Hf, Wf, stride, pad, _stream(stream)))
    return dX


def conv2d_forward_pool(X, W, b, C, Hin, Win, Hf, Wf, stride, pad, pool_h, pool_w, pool_stride,
                        pool_pad, relu=True, out=None, pooled=None, argmax=None, keep_out=False,
                        stream=None):
    """relu(conv + b) then max-pool in one call.  Returns (out or None, pooled, argmax,
    Hp, Wp); the conv output is only materialised when out is given or keep_out."""
    dt = _dtype(X, W, b, out, pooled)
    N, F = X.shape[0], W.shape[0]
    Hout = conv2d_out_dim(Hin, Hf, stride, pad)
    Wout = conv2d_out_dim(Win, Wf, stride, pad)
    Hp = conv2d_out_dim(Hout, pool_h, pool_stride, pool_pad)
    Wp = conv2d_out_dim(Wout, pool_w, pool_stride, pool_pad)
    _need(X, N * C * Hin * Win, "X")
    _need(W, F * C * Hf * Wf, "W")
    _need(b, F, "b")
    if out is None and keep_out:
        out = _empty((N, F * max(Hout, 0) * max(Wout, 0)), X)
    _need(out, N * F * max(Hout, 0) * max(Wout, 0), "out")
    if pooled is None:
        pooled = _empty((N, F * max(Hp, 0) * max(Wp, 0)), X)
    if argmax is None:
        argmax = _empty((N, F * max(Hp, 0) * max(Wp, 0)), X, torch.int32)
    _need(pooled, N * F * max(Hp, 0) * max(Wp, 0), "pooled")
    _need(argmax, N * F * max(Hp, 0) * max(Wp, 0), "argmax")
    _check("conv2d_forward_pool", load().conv2d_forward_pool(
        dt, _p(X), _p(W), _p(b), _p(out), _p(pooled), _p(argmax), N, C, Hin, Win, F, Hf, Wf,
        stride, pad, int(relu), pool_h, pool_w, pool_stride, pool_pad, _stream(stream)))
    return out, pooled, argmax, Hp, Wp


def conv2d_forward_csr(rowptr, colidx, vals, W, b, C, Hin, Win, Hf, Wf, stride, pad, relu=True,
                       out=None, row_index=None, stream=None):
    """conv2d forward of a CSR input (N x C*Hin*Win; int32 rowptr/colidx on the device)."""
    dt = _dtype(vals, W, b, out)
    N, F = rowptr.numel() - 1, W.shape[0]
    nnz = colidx.numel()
    if rowptr.dtype != torch.int32 or colidx.dtype != torch.int32:
        raise TypeError("rowptr and colidx must be int32")
    _need(vals, nnz, "vals")
    _need(W, F * C * Hf * Wf, "W")
    _need(b, F, "b")
    Hout = conv2d_out_dim(Hin, Hf, stride, pad)
    Wout = conv2d_out_dim(Win, Wf, stride, pad)
    if out is None:
        out = _empty((N, F * max(Hout, 0) * max(Wout, 0)), W)
    if row_index is None:
        row_index = torch.empty(N * C * Hin + 1, dtype=torch.int32, device=W.device)
    _need(out, N * F * max(Hout, 0) * max(Wout, 0), "out")
    _need(row_index, N * C * Hin + 1, "row_index")
    _check("conv2d_forward_csr", load().conv2d_forward_csr(
        dt, _p(rowptr), _p(colidx) if nnz else None, _p(vals) if nnz else None, nnz,
        _p(row_index), _p(W), _p(b), _p(out), N, C, Hin, Win, F, Hf, Wf, stride, pad,
        int(relu), _stream(stream)))
    return out


def conv2d_forward_multi(X, Ws, bs, C, Hin, Win, Hf, Wf, stride, pad, relu=True, outs=None,
                         Wcat=None, bcat=None, stream=None):
    """Several filter banks over one input in one launch.  Ws / bs: lists of the
    banks' filters (F_b x C*Hf*Wf) and biases (or None).  Wcat / bcat may pass the
    stacked copies already made; returns the list of outputs."""
    dt = _dtype(X, *Ws)
    N, nb = X.shape[0], len(Ws)
    Fs = [int(W.shape[0]) for W in Ws]
    Hout = conv2d_out_dim(Hin, Hf, stride, pad)
    Wout = conv2d_out_dim(Win, Wf, stride, pad)
    _need(X, N * C * Hin * Win, "X")
    for W, F in zip(Ws, Fs):
        _need(W, F * C * Hf * Wf, "W")
    if Wcat is None:
        Wcat = torch.cat([W.reshape(F, -1) for W, F in zip(Ws, Fs)]).contiguous()
    if bcat is None and bs is not None and any(b is not None for b in bs):
        bcat = torch.cat([b if b is not None else torch.zeros(F, dtype=X.dtype, device=X.device)
                          for b, F in zip(bs, Fs)]).contiguous()
    if outs is None:
        outs = [_empty((N, F * max(Hout, 0) * max(Wout, 0)), X) for F in Fs]
    for o, F in zip(outs, Fs):
        _need(o, N * F * max(Hout, 0) * max(Wout, 0), "out")
    ptrs = (ctypes.c_void_p * nb)(*[_p(o) for o in outs])
    fs = (ctypes.c_int * nb)(*Fs)
    _check("conv2d_forward_multi", load().conv2d_forward_multi(
        dt, _p(X), _p(Wcat), _p(bcat), ctypes.cast(ptrs, ctypes.c_void_p),
        ctypes.cast(fs, ctypes.c_void_p), nb, N, C, Hin, Win, Hf, Wf, stride, pad, int(relu),
        _stream(stream)))
    return outs


def max_pool2d_bwd_relu(dout, argmax, pooled, C, Hin, Win, Hf, Wf, stride, pad, dX=None,
                        stream=None):
    """Pool backward with the preceding relu's mask (pooled > 0) folded in."""
    dt = _dtype(dout, pooled, dX)
    N = dout.shape[0]
    Hout = conv2d_out_dim(Hin, Hf, stride, pad)
    Wout = conv2d_out_dim(Win, Wf, stride, pad)
    if dX is None:
        dX = _empty((N, C * Hin * Win), dout)
    n_out = N * C * max(Hout, 0) * max(Wout, 0)
    _need(dout, n_out, "dout")
    _need(argmax, n_out, "argmax")
    _need(pooled, n_out, "pooled")
    _need(dX, N * C * Hin * Win, "dX")
    _check("max_pool2d_bwd_relu", load().max_pool2d_bwd_relu(
        dt, _p(dout), _p(argmax), _p(pooled), _p(dX), N, C, Hin, Win, Hf, Wf, stride, pad,
        _stream(stream)))
    return dX


def affine_workspace_size(dtype, N, D, M) -> int:
    dt = _DT[dtype] if isinstance(dtype, torch.dtype) else int(dtype)
    return int(load().affine_workspace_size(dt, N, D, M))


AFFINE_PRODUCTS = {"forward": 0, "dX": 1, "dW": 2}


def affine_plan(dtype, product, N, D, M, workspace_bytes):
    """The launch shape of one affine product (host only): a dict of tile
    (output tile edge), waves (per block, splitting its k range) and splits
    (blocks per tile along k)."""
    dt = _DT[dtype] if isinstance(dtype, torch.dtype) else int(dtype)
    t, w, s = ctypes.c_int(), ctypes.c_int(), ctypes.c_int()
    _check("affine_plan", load().affine_plan(dt, AFFINE_PRODUCTS[product], N, D, M,
                                              workspace_bytes, ctypes.byref(t), ctypes.byref(w),
                                              ctypes.byref(s)))
    return {"tile": t.value, "waves": w.value, "splits": s.value}


def _affine_ws(X, N, D, M, workspace):
    """The caller's workspace (None: a fresh one of the full size; an empty
    tensor: none, the products run unsplit) as (pointer, bytes)."""
    if workspace is None:
        nb = affine_workspace_size(X.dtype, N, D, M)
        workspace = torch.empty(nb, dtype=torch.uint8, device=X.device) if nb else None
    if workspace is None or workspace.numel() == 0:
        return None, 0
    return _p(workspace), workspace.numel() * workspace.element_size()


def affine_fwd(X, W, b, relu=False, out=None, workspace=None, stream=None):
    dt = _dtype(X, W, b, out)
    N, D = X.shape
    M = W.shape[1]
    if out is None:
        out = _empty((N, M), X)
    _need(W, D * M, "W")
    _need(b, M, "b")
    _need(out, N * M, "out")
    ws, nb = _affine_ws(X, N, D, M, workspace)
    _check("affine_fwd", load().affine_fwd(dt, _p(X), _p(W), _p(b), _p(out), N, D, M,
                                            int(bool(relu)), ws, nb, _stream(stream)))
    return out


def affine_bwd(dout, X, W, out_fwd=None, want_dX=True, want_db=True, dX=None, dW=None, db=None,
               want_dW=True, workspace=None, relu_input=False, stream=None):
    """Returns [dX, dW, db] (each None when not wanted).  relu_input: dX is
    also multiplied by (X > 0) (X is a relu output)."""
    dt = _dtype(dout, X, W, out_fwd, dX, dW, db)
    N, D = X.shape
    M = W.shape[1]
    if dX is None and want_dX:
        dX = _empty((N, D), X)
    if dW is None and want_dW:
        dW = _empty((D, M), X)
    if db is None and want_db:
        db = _empty((M,), X)
    _need(W, D * M, "W")
    _need(dout, N * M, "dout")
    _need(out_fwd, N * M, "out_fwd")
    _need(dX, N * D, "dX")
    _need(dW, D * M, "dW")
    _need(db, M, "db")
    ws, nb = _affine_ws(X, N, D, M, workspace) if (dX is not None or dW is not None) else (None, 0)
    _check("affine_bwd", load().affine_bwd(dt, _p(dout), _p(X), _p(W), _p(out_fwd), _p(dX),
                                            _p(dW), _p(db), N, D, M, int(bool(relu_input)), ws,
                                            nb, _stream(stream)))
    return dX, dW, db


def softmax_xent_workspace_size(dtype, N, K) -> int:
    """Bytes of workspace softmax_xent spreads its rows over (0: one block)."""
    dt = _DT[dtype] if isinstance(dtype, torch.dtype) else int(dtype)
    return int(load().softmax_xent_workspace_size(dt, N, K))


def softmax_xent(scores, Y, want_probs=True, loss=None, dscores=None, probs=None, stream=None,
                 workspace=None):
    """Returns (loss as a 1-element device tensor, dscores, probs-or-None).
    workspace: None (a fresh one of the full size), a byte tensor, or an
    empty tensor (none: one block does the call)."""
    dt = _dtype(scores, Y, loss, dscores, probs)
    N, K = scores.shape
    if loss is None:
        loss = _empty((1,), scores)
    if dscores is None:
        dscores = torch.empty_like(scores)
    if probs is None and want_probs:
        probs = torch.empty_like(scores)
    _need(Y, N * K, "Y")
    _need(dscores, N * K, "dscores")
    _need(probs, N * K, "probs")
    _need(loss, 1, "loss")
    if workspace is None:
        nb = softmax_xent_workspace_size(dt, N, K)
        workspace = torch.empty(nb, dtype=torch.uint8, device=scores.device) if nb else None
    ws, nb = (None, 0) if workspace is None or workspace.numel() == 0 else (
        _p(workspace), workspace.numel() * workspace.element_size())
    _check("softmax_xent", load().softmax_xent(dt, _p(scores), _p(Y), _p(probs), _p(dscores),
                                                _p(loss), N, K, ws, nb, _stream(stream)))
    return loss, dscores, probs


def softmax_fwd(scores, probs=None, stream=None):
    """Row-wise softmax of an N x K matrix."""
    dt = _dtype(scores, probs)
    N, K = scores.shape
    if probs is None:
        probs = _empty((N, K), scores)
    _need(probs, N * K, "probs")
    _check("softmax_fwd", load().softmax_fwd(dt, _p(scores), _p(probs), N, K, _stream(stream)))
    return probs


def sgd_momentum_update(theta, grad, v, lr, mu, stream=None):
    """In place: v <- mu v - lr grad; theta <- theta + v."""
    dt = _dtype(theta, grad, v)
    _need(grad, theta.numel(), "grad")
    _need(v, theta.numel(), "v")
    _check("sgd_momentum_update", load().sgd_momentum_update(
        dt, _p(theta), _p(grad), _p(v), float(lr), float(mu), theta.numel(), _stream(stream)))
    return theta, v


def sgd_update(theta, grad, lr, stream=None):
    """In place: theta <- theta - lr grad."""
    dt = _dtype(theta, grad)
    _need(grad, theta.numel(), "grad")
    _check("sgd_update", load().sgd_update(dt, _p(theta), _p(grad), float(lr), theta.numel(),
                                           _stream(stream)))
    return theta


def sgd_nesterov_update(theta, grad, v, lr, mu, stream=None):
    """In place: v' = mu v - lr grad; theta <- theta - mu v + (1 + mu) v'; v <- v'."""
    dt = _dtype(theta, grad, v)
    _need(grad, theta.numel(), "grad")
    _need(v, theta.numel(), "v")
    _check("sgd_nesterov_update", load().sgd_nesterov_update(
        dt, _p(theta), _p(grad), _p(v), float(lr), float(mu), theta.numel(), _stream(stream)))
    return theta, v


def adagrad_update(theta, grad, cache, lr, eps=1e-6, stream=None):
    """In place: cache += grad^2; theta -= lr grad / (sqrt(cache) + eps)."""
    dt = _dtype(theta, grad, cache)
    _need(grad, theta.numel(), "grad")
    _need(cache, theta.numel(), "cache")
    _check("adagrad_update", load().adagrad_update(
        dt, _p(theta), _p(grad), _p(cache), float(lr), float(eps), theta.numel(), _stream(stream)))
    return theta, cache


def rmsprop_update(theta, grad, cache, lr, decay=0.99, eps=1e-6, stream=None):
    """In place: cache = decay cache + (1-decay) grad^2; theta -= lr grad / (sqrt(cache) + eps)."""
    dt = _dtype(theta, grad, cache)
    _need(grad, theta.numel(), "grad")
    _need(cache, theta.numel(), "cache")
    _check("rmsprop_update", load().rmsprop_update(
        dt, _p(theta), _p(grad), _p(cache), float(lr), float(decay), float(eps), theta.numel(),
        _stream(stream)))
    return theta, cache


def adam_update(theta, grad, m, v, lr, beta1=0.9, beta2=0.999, eps=1e-8, t=1, stream=None):
    """In place, step t >= 1: m, v moments; theta -= lr_t m / (sqrt(v) + eps),
    lr_t = lr sqrt(1 - beta2^t) / (1 - beta1^t)."""
    dt = _dtype(theta, grad, m, v)
    _need(grad, theta.numel(), "grad")
    _need(m, theta.numel(), "m")
    _need(v, theta.numel(), "v")
    _check("adam_update", load().adam_update(
        dt, _p(theta), _p(grad), _p(m), _p(v), float(lr), float(beta1), float(beta2), float(eps),
        int(t), theta.numel(), _stream(stream)))
    return theta, m, v


def count_nonzero(X, out=None, stream=None):
    """Number of non-zero entries, as a 1-element int64 device tensor."""
    dt = _dtype(X)
    if out is None:
        out = _empty((1,), X, dtype=torch.int64)
    if out.dtype != torch.int64 or out.numel() < 1:
        raise ValueError("out must be an int64 tensor with at least one element")
    _check("count_nonzero", load().count_nonzero(dt, _p(X), X.numel(), _p(out), _stream(stream)))
    return out
