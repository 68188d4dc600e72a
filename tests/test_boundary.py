"""The C ABI boundary on the CPU: the library loads, exports every entry point
that include/dmlnn.h declares, and rejects bad arguments on the host with the
documented status codes before launching anything.  No GPU is needed and no
pointer is ever dereferenced: every call below fails validation, except the
ones marked, which pass it and therefore run only on hosts without a GPU, where
the device check stops them."""
import ctypes

import pytest

from paper_1802_04647_amd import dmlnn

OK, ERR_ARG, ERR_NULL, ERR_DTYPE, ERR_WS, ERR_DEVICE = 0, 1, 2, 3, 4, 5
FAKE = 0x1000  # never dereferenced: every call using it fails validation first


@pytest.fixture(scope="module")
def lib():
    return dmlnn.load()


def test_exports_every_declared_symbol(lib):
    names = dmlnn.header_symbols()
    expected = {"conv2d_out_dim", "conv2d_forward", "conv2d_backward_filter_workspace_size",
                "conv2d_backward_filter", "conv2d_backward_data", "dmlnn_set_zero_skip",
                "bias_add_relu", "max_pool2d_fwd", "max_pool2d_bwd", "affine_fwd", "affine_bwd",
                "affine_workspace_size", "softmax_xent_workspace_size",
                "softmax_xent", "sgd_momentum_update", "count_nonzero", "dmlnn_last_error"}
    assert expected <= set(names)
    for n in names:
        assert hasattr(lib, n), n


def test_out_dim(lib):
    assert lib.conv2d_out_dim(56, 3, 1, 1) == 56
    assert lib.conv2d_out_dim(28, 5, 1, 2) == 28
    assert lib.conv2d_out_dim(28, 2, 2, 0) == 14
    assert lib.conv2d_out_dim(7, 3, 2, 0) == 3
    assert lib.conv2d_out_dim(2, 3, 1, 0) <= 0
    assert lib.conv2d_out_dim(5, 3, 0, 0) <= 0
    assert lib.conv2d_out_dim(5, 3, 1, -1) <= 0


def test_workspace_size(lib):
    f = lib.conv2d_backward_filter_workspace_size
    w64 = f(0, 256, 64, 56, 56, 64, 3, 3, 1, 1)
    w32 = f(1, 256, 64, 56, 56, 64, 3, 3, 1, 1)
    # splits x (F*K + F) elements of the dtype; the split count follows the
    # kernel's per-CU occupancy bound (fp32 blocks take half the LDS)
    FK = 64 * 576 + 64
    assert w64 > 0 and w32 > 0 and w64 % (8 * FK) == 0 and w32 % (4 * FK) == 0
    assert f(0, 4, 1, 8, 8, 2, 3, 3, 1, 1) > 0
    assert f(7, 4, 1, 8, 8, 2, 3, 3, 1, 1) == 0          # bad dtype
    assert f(0, 0, 1, 8, 8, 2, 3, 3, 1, 1) == 0          # N = 0
    assert f(0, 4, 1, 2, 2, 2, 3, 3, 1, 0) == 0          # no window fits


def _conv_fwd(lib, dt=0, X=FAKE, W=FAKE, out=FAKE, N=2, C=1, H=8, Wd=8, F=2, Hf=3, Wf=3, s=1,
              p=1, relu=1):
    return lib.conv2d_forward(dt, X, W, None, out, N, C, H, Wd, F, Hf, Wf, s, p, relu, None)


def test_conv_forward_validation(lib):
    assert _conv_fwd(lib, dt=2) == ERR_DTYPE
    assert _conv_fwd(lib, X=None) == ERR_NULL
    assert _conv_fwd(lib, out=None) == ERR_NULL
    assert "required" in dmlnn.last_error()
    assert _conv_fwd(lib, N=0) == ERR_ARG
    assert _conv_fwd(lib, s=0) == ERR_ARG
    assert _conv_fwd(lib, p=-1) == ERR_ARG
    assert _conv_fwd(lib, H=2, Hf=5, p=0) == ERR_ARG
    assert _conv_fwd(lib, relu=2) == ERR_ARG
    assert _conv_fwd(lib, N=70000, C=64, H=100, Wd=100) == ERR_ARG   # > 2^31 elements


def test_conv_backward_validation(lib):
    bf = lib.conv2d_backward_filter
    need = lib.conv2d_backward_filter_workspace_size(0, 2, 1, 8, 8, 2, 3, 3, 1, 1)
    assert bf(0, FAKE, FAKE, None, FAKE, None, 2, 1, 8, 8, 2, 3, 3, 1, 1, None, need, None) == ERR_WS
    assert bf(0, FAKE, FAKE, None, FAKE, None, 2, 1, 8, 8, 2, 3, 3, 1, 1, FAKE, need - 1,
              None) == ERR_WS
    assert "workspace" in dmlnn.last_error()
    assert bf(0, None, FAKE, None, FAKE, None, 2, 1, 8, 8, 2, 3, 3, 1, 1, FAKE, need,
              None) == ERR_NULL
    assert bf(5, FAKE, FAKE, None, FAKE, None, 2, 1, 8, 8, 2, 3, 3, 1, 1, FAKE, need,
              None) == ERR_DTYPE
    # the masked-gradient form: g_out is required and may not overlap X, dW,
    # db or the workspace (dout itself is allowed); each call fails validation
    be = lib.conv2d_backward_filter_emit
    X, dout, dW, g, ws = 0x10000, 0x20000, 0x30000, 0x40000, 0x50000
    args = (2, 1, 8, 8, 2, 3, 3, 1, 1)
    assert be(0, X, dout, None, dW, None, None, *args, ws, need, None) == ERR_NULL
    assert be(0, X, dout, None, dW, None, X + 8, *args, ws, need, None) == ERR_ARG
    assert "overlaps" in dmlnn.last_error()
    assert be(0, X, dout, None, dW, None, dW, *args, ws, need, None) == ERR_ARG
    assert be(0, X, dout, None, dW, None, ws + 64, *args, ws, need, None) == ERR_ARG
    assert be(0, X, dout, None, dW, None, g, *args, ws, need - 1, None) == ERR_WS
    assert be(0, X, dout, None, dW, None, g, 2, 1, 8, 8, 2, 3, 3, 0, 1, ws, need, None) == ERR_ARG
    bd = lib.conv2d_backward_data
    assert bd(0, FAKE, FAKE, None, None, 2, 1, 8, 8, 2, 3, 3, 1, 1, None) == ERR_NULL
    assert bd(0, FAKE, FAKE, None, FAKE, 2, 1, 8, 8, 2, 3, 3, 0, 1, None) == ERR_ARG


def test_other_validation(lib):
    assert lib.bias_add_relu(0, None, None, FAKE, 2, 3, 4, 1, None) == ERR_NULL
    assert lib.bias_add_relu(0, FAKE, None, FAKE, 2, 0, 4, 1, None) == ERR_ARG
    assert lib.max_pool2d_fwd(0, FAKE, FAKE, None, 1, 1, 4, 4, 2, 2, 2, 0, None) == ERR_NULL
    assert lib.max_pool2d_fwd(0, FAKE, FAKE, FAKE, 1, 1, 4, 4, 2, 2, 2, 2, None) == ERR_ARG
    assert lib.max_pool2d_bwd(1, FAKE, FAKE, FAKE, 1, 1, 4, 4, 2, 2, 0, 0, None) == ERR_ARG
    assert lib.affine_fwd(0, FAKE, FAKE, None, FAKE, 0, 3, 4, 0, None, 0, None) == ERR_ARG
    assert lib.affine_bwd(0, FAKE, FAKE, FAKE, None, None, None, None, 2, 3, 4, 0, None, 0,
                          None) == ERR_NULL
    assert lib.affine_bwd(0, None, FAKE, FAKE, None, FAKE, FAKE, None, 2, 3, 4, 0, None, 0,
                          None) == ERR_NULL
    assert lib.softmax_xent(0, FAKE, FAKE, None, FAKE, None, 2, 3, None, 0, None) == ERR_NULL
    assert lib.sgd_momentum_update(0, FAKE, FAKE, FAKE, 0.1, 0.9, 0, None) == ERR_ARG
    assert lib.count_nonzero(3, FAKE, 10, FAKE, None) == ERR_DTYPE


def test_affine_workspace(lib):
    """The split-reduction workspace: sized from the products that split (the
    batch-64 3136 -> 512 forward: seven splits of 64 x 512 partials), none for
    products whose tiles fill the GPU, and a workspace that is misaligned or
    overlaps a tensor of the call is rejected before anything runs."""
    assert lib.affine_workspace_size(0, 64, 3136, 512) == 7 * 64 * 512 * 8
    assert lib.affine_workspace_size(1, 64, 3136, 512) == 7 * 64 * 512 * 4
    assert lib.affine_workspace_size(0, 64, 512, 10) == 0
    assert lib.affine_workspace_size(0, 0, 3, 4) == 0
    assert lib.affine_workspace_size(4, 2, 3, 4) == 0
    X, W, out, ws = 0x100000, 0x200000, 0x300000, 0x400000
    assert lib.affine_fwd(0, X, W, None, out, 2, 3, 4, 0, ws + 4, 64, None) == ERR_ARG
    assert lib.affine_fwd(0, X, W, None, out, 2, 3, 4, 0, out - 32, 64, None) == ERR_ARG
    assert lib.affine_bwd(0, X, W, out, None, ws, None, None, 2, 3, 4, 0, ws + 8, 64,
                          None) == ERR_ARG
    assert "workspace" in dmlnn.last_error()
    # relu_input: a flag, and dX may not overlap the X it is masked by
    assert lib.affine_bwd(0, X, W, out, None, ws, None, None, 2, 3, 4, 2, None, 0,
                          None) == ERR_ARG
    assert lib.affine_bwd(0, X, W, out, None, W + 8, None, None, 2, 3, 4, 1, None, 0,
                          None) == ERR_ARG
    assert "relu_input" in dmlnn.last_error()


def test_softmax_xent_workspace(lib):
    """One element per block of 16 x (64 / sw) rows (sw = the power of two
    segment a row takes), up to 2048 blocks; none when one block covers the
    batch (the LeNet step's 64 x 10); bad workspaces rejected before any launch."""
    f = lib.softmax_xent_workspace_size
    assert f(0, 64, 10) == 0                        # 64 rows a block at K = 10
    assert f(0, 65, 10) == 2 * 8
    assert f(1, 65, 10) == 2 * 4
    assert f(0, 1024, 1) == 0 and f(0, 1025, 1) == 2 * 8
    assert f(0, 17, 130) == 2 * 8                   # 16 rows a block at K > 64
    assert f(0, 1 << 20, 10) == 2048 * 8            # capped
    assert f(0, 0, 10) == 0 and f(3, 100, 10) == 0  # bad sizes, bad dtype
    S, Y, dS, loss, ws = 0x100000, 0x200000, 0x300000, 0x400000, 0x500000
    assert lib.softmax_xent(0, S, Y, None, dS, loss, 100, 10, ws + 4, 64, None) == ERR_ARG
    assert "workspace" in dmlnn.last_error()
    assert lib.softmax_xent(0, S, Y, None, dS, loss, 100, 10, dS + 800, 64, None) == ERR_ARG
    assert lib.softmax_xent(0, S, Y, None, dS, loss, 100, 10, loss - 8, 64, None) == ERR_ARG


def test_zero_skip_mode(lib):
    prev = lib.dmlnn_set_zero_skip(1)
    try:
        assert lib.dmlnn_set_zero_skip(0) == 1
        assert lib.dmlnn_set_zero_skip(7) == -1
    finally:
        lib.dmlnn_set_zero_skip(prev)


def _skip_on_gpu_host():
    # Calls below pass validation with never-allocated pointers: on a host with
    # a GPU they would launch kernels on those addresses, so they run only where
    # the device check stops them.
    import torch
    if torch.cuda.device_count() > 0:
        pytest.skip("a GPU is present: a call that passes validation would launch")


def test_no_device_is_reported_not_crashed(lib):
    # Without a GPU a valid call must return DMLNN_ERR_DEVICE rather than abort.
    _skip_on_gpu_host()
    assert _conv_fwd(lib) == ERR_DEVICE
    assert dmlnn.last_error() != ""


def test_affine_bwd_accepts_any_single_output(lib):
    # Any one of dX, dW, db alone is a valid request: validation passes and only
    # the device check (no GPU here) stops the call.
    _skip_on_gpu_host()
    for outs in ((FAKE, None, None), (None, FAKE, None), (None, None, FAKE)):
        assert lib.affine_bwd(0, FAKE, FAKE, FAKE, None, *outs, 2, 3, 4, 0, None, 0,
                              None) == ERR_DEVICE


def test_binding_rejects_host_tensors():
    import torch
    X = torch.zeros(2, 64, dtype=torch.float64)
    W = torch.zeros(2, 9, dtype=torch.float64)
    with pytest.raises(ValueError):
        dmlnn.conv2d_forward(X, W, None, 1, 8, 8, 3, 3, 1, 1)
    with pytest.raises(TypeError):
        dmlnn.conv2d_forward(X.half(), W.half(), None, 1, 8, 8, 3, 3, 1, 1)


def test_optimizer_validation(lib):
    d = ctypes.c_double
    assert lib.sgd_update(0, None, FAKE, d(0.1), 10, None) == ERR_NULL
    assert lib.sgd_update(5, FAKE, FAKE, d(0.1), 10, None) == ERR_DTYPE
    assert lib.sgd_update(0, FAKE, FAKE, d(0.1), 0, None) == ERR_ARG
    assert lib.sgd_nesterov_update(0, FAKE, FAKE, None, d(0.1), d(0.9), 10, None) == ERR_NULL
    assert lib.adagrad_update(0, FAKE, FAKE, FAKE, d(0.1), d(-1.0), 10, None) == ERR_ARG
    assert lib.rmsprop_update(0, FAKE, FAKE, FAKE, d(0.1), d(1.5), d(1e-6), 10, None) == ERR_ARG
    assert lib.rmsprop_update(0, FAKE, FAKE, None, d(0.1), d(0.9), d(1e-6), 10, None) == ERR_NULL
    adam = lib.adam_update
    assert adam(0, FAKE, FAKE, FAKE, FAKE, d(1e-3), d(0.9), d(0.999), d(1e-8), 0, 10, None) \
        == ERR_ARG                                                       # t = 0
    assert adam(0, FAKE, FAKE, FAKE, FAKE, d(1e-3), d(1.0), d(0.999), d(1e-8), 1, 10, None) \
        == ERR_ARG                                                       # beta1 = 1
    assert adam(0, FAKE, FAKE, FAKE, None, d(1e-3), d(0.9), d(0.999), d(1e-8), 1, 10, None) \
        == ERR_NULL


def test_noalloc_backward_filter_validation(lib):
    f = lib.conv2d_backward_filter_noalloc
    # a layer whose split partials (5x5 filters over 256 channels, 61-wide rows:
    # the tiled kernel) exceed the scratch: rejected before anything else happens
    big = (64, 256, 8, 61, 64, 5, 5, 1, 2)
    assert lib.conv2d_backward_filter_workspace_size(0, *big) > 80 * 2 ** 20
    assert f(0, FAKE, FAKE, None, FAKE, None, *big, None) == ERR_WS
    assert "scratch" in dmlnn.last_error()
    # the benchmark layer's partials fit
    assert lib.conv2d_backward_filter_workspace_size(0, 256, 64, 56, 56, 64, 3, 3, 1, 1) \
        <= 80 * 2 ** 20
    assert f(0, None, FAKE, None, FAKE, None, 2, 1, 8, 8, 2, 3, 3, 1, 1, None) == ERR_NULL
    assert f(0, FAKE, FAKE, None, None, None, 2, 1, 8, 8, 2, 3, 3, 1, 1, None) == ERR_NULL
    assert f(9, FAKE, FAKE, None, FAKE, None, 2, 1, 8, 8, 2, 3, 3, 1, 1, None) == ERR_DTYPE
    assert f(0, FAKE, FAKE, None, FAKE, None, 2, 1, 8, 8, 2, 3, 3, 0, 1, None) == ERR_ARG


def test_pooled_backward_validation(lib):
    bf, bd = lib.conv2d_backward_filter_pooled, lib.conv2d_backward_data_pooled
    conv = (2, 3, 10, 10, 8, 3, 3, 1, 1)           # 10x10 conv output
    need = lib.conv2d_backward_filter_workspace_size(0, *conv)
    # overlapping windows (stride 2 < 3) and padded pools are refused
    assert bd(0, FAKE, FAKE, FAKE, FAKE, FAKE, *conv, 3, 3, 2, 0, None) == ERR_ARG
    assert "overlap" in dmlnn.last_error()
    assert bd(0, FAKE, FAKE, FAKE, FAKE, FAKE, *conv, 2, 2, 2, 1, None) == ERR_ARG
    assert bf(0, FAKE, FAKE, FAKE, FAKE, FAKE, None, *conv, 3, 3, 2, 0, FAKE, need,
              None) == ERR_ARG
    # missing pool inputs, workspace, bad dtype
    assert bd(0, FAKE, FAKE, None, FAKE, FAKE, *conv, 2, 2, 2, 0, None) == ERR_NULL
    assert bf(0, FAKE, FAKE, FAKE, None, FAKE, None, *conv, 2, 2, 2, 0, FAKE, need,
              None) == ERR_NULL
    assert bf(0, FAKE, FAKE, FAKE, FAKE, FAKE, None, *conv, 2, 2, 2, 0, FAKE, need - 1,
              None) == ERR_WS
    assert bd(6, FAKE, FAKE, FAKE, FAKE, FAKE, *conv, 2, 2, 2, 0, None) == ERR_DTYPE
    # a window larger than the conv output
    assert bd(0, FAKE, FAKE, FAKE, FAKE, FAKE, *conv, 11, 11, 11, 0, None) == ERR_ARG
