"""Kernel selection on the host (no GPU): the plan query reports which kernel
form each conv2d pass takes, its tiling and the backward_filter workspace."""
import pytest
import torch

from paper_1802_04647_amd import dmlnn
from paper_1802_04647_amd.inputs import SHAPES, ConvShape
from test_gpu_zero_skip import CASES as SKIP_CASES

PASSES = ("forward", "backward_filter", "backward_data")
DT = {"f64": torch.float64, "f32": torch.float32}


def test_skip_cases_reach_every_form():
    """The zero-skip GPU cases take every kernel form that has a skip
    instantiation: the LDS-DMA implicit GEMM (plain, two- and four-way k split,
    32- and 224-pixel tiles) and the register-staged one, forward and backward,
    and both backward_filter kernels."""
    seen = set()
    for s in SKIP_CASES:
        for dt in DT.values():
            for pname in PASSES:
                p = dmlnn.conv2d_plan(dt, pname, *s.args(), zero_skip=1)
                assert p["zero_skip"] == 1, (s, dt, pname, p)
                seen.add((pname, p["kernel"], p["k_split"], p["tile_pixels"] > 32))
    want = {(pn, "igemm_dma", ks, False) for pn in ("forward", "backward_data") for ks in (1, 2, 4)}
    want |= {(pn, "igemm_dma", 1, True) for pn in ("forward", "backward_data")}
    want |= {(pn, "igemm_reg", 1, False) for pn in ("forward", "backward_data")}
    assert want <= seen, want - seen
    assert {k[1] for k in seen if k[0] == "backward_filter"} == {"wgrad_ring", "wgrad_tiles"}


def test_forms_without_a_skip_variant_report_it():
    # at most four output rows: the vector-ALU kernel, identical under either mode
    p = dmlnn.conv2d_plan(torch.float64, "backward_data", *SHAPES["lenet_conv1"].args(), zero_skip=1)
    assert p["kernel"] == "small_m" and p["zero_skip"] == 0
    # the filter-resident forward has no skip form: the skip mode takes the DMA kernel
    s = SHAPES["lenet_conv2"]
    assert dmlnn.conv2d_plan(torch.float64, "forward", *s.args())["kernel"] == "resident"
    p = dmlnn.conv2d_plan(torch.float64, "forward", *s.args(), zero_skip=1)
    assert p["kernel"] == "igemm_dma" and p["zero_skip"] == 1


def test_benchmark_layer_plan():
    s = SHAPES["resnet_conv"]
    for dt in DT.values():
        f = dmlnn.conv2d_plan(dt, "forward", *s.args())
        d = dmlnn.conv2d_plan(dt, "backward_data", *s.args())
        w = dmlnn.conv2d_plan(dt, "backward_filter", *s.args())
        assert f["kernel"] == d["kernel"] == "igemm_dma"
        assert f["tile_pixels"] == d["tile_pixels"] == 224 and f["chunk"] == 4
        assert w["kernel"] == "wgrad_ring" and w["chunk"] == 576
        assert max(f["lds_bytes"], d["lds_bytes"]) <= 80 * 1024      # two blocks per CU
        assert w["lds_bytes"] <= 160 * 1024


@pytest.mark.parametrize("name", sorted(SHAPES))
@pytest.mark.parametrize("dt", ["f64", "f32"])
def test_workspace_is_the_launchable_splits(name, dt):
    """The workspace holds exactly the partials of the most splits a launch
    uses: splits x (F*K + F) elements."""
    s = SHAPES[name]
    p = dmlnn.conv2d_plan(DT[dt], "backward_filter", *s.args())
    tsz = 8 if dt == "f64" else 4
    assert p["splits"] >= 1
    assert p["workspace_bytes"] == p["splits"] * (s.F * s.K + s.F) * tsz
    assert p["workspace_bytes"] == dmlnn.conv2d_backward_filter_workspace_size(DT[dt], *s.args())


def test_ring_staging_forms():
    """How the row ring stages its next input row: fp32 at stride 1 by LDS DMA
    into an Hf + 1 slot ring (and the g tile a row a wave), fp64 at stride 1 a
    row a wave through registers in an Hf slot ring, and any dtype at stride 2
    an element a thread; the pooled source's g tile has its own staging."""
    s1 = SHAPES["resnet_conv"]
    s2 = ConvShape(2, 64, 6, 24, 5, 3, 3, 2, 1)
    for s, dt, want_rs, want_rows in ((s1, "f32", 4 | 2, s1.Hf + 1), (s1, "f64", 1, s1.Hf),
                                      (s2, "f32", 0, s2.Hf), (s2, "f64", 0, s2.Hf)):
        p = dmlnn.conv2d_plan(DT[dt], "backward_filter", *s.args())
        assert p["kernel"] == "wgrad_ring"
        assert (p["row_staged"], p["window_rows"]) == (want_rs, want_rows), (s, dt, p)
    s3 = ConvShape(2, 40, 12, 12, 48, 3, 3, 1, 1)
    p = dmlnn.conv2d_plan_fused(DT["f32"], "backward_filter", "pooled_source", *s3.args(),
                                pool=(2, 2, 2, 0))
    assert p["kernel"] == "wgrad_ring" and p["row_staged"] == 4 and p["window_rows"] == 4


def test_benchmark_layer_workspace_bound():
    s = SHAPES["resnet_conv"]
    for dt in DT.values():
        assert dmlnn.conv2d_backward_filter_workspace_size(dt, *s.args()) <= 80 * 10 ** 6


def test_images_of_2gib_take_the_register_path():
    """Per-image source tensors of 2 GiB or more cannot be addressed by the
    32-bit byte offsets of the LDS-DMA and filter-resident kernels: such layers
    take the register-staged kernel (fp64 here; the same image is 1 GiB in
    fp32).  backward_data stages the gradient (16 channels here), not X."""
    s = ConvShape(1, 4096, 256, 256, 16, 3, 3, 1, 1)
    assert s.C * s.Hin * s.Win * 8 >= 2 ** 31
    assert dmlnn.conv2d_plan(torch.float64, "forward", *s.args())["kernel"] == "igemm_reg"
    assert dmlnn.conv2d_plan(torch.float32, "forward", *s.args())["kernel"] == "igemm_dma"
    assert dmlnn.conv2d_plan(torch.float64, "backward_data", *s.args())["kernel"] == "igemm_dma"


def test_plan_validation():
    lib = dmlnn.load()
    plan = dmlnn.ConvPlan()
    import ctypes
    assert lib.conv2d_plan(0, 3, 1, 1, 8, 8, 2, 3, 3, 1, 1, 0, ctypes.byref(plan)) == 1   # pass
    assert lib.conv2d_plan(0, 0, 1, 1, 8, 8, 2, 3, 3, 1, 1, 2, ctypes.byref(plan)) == 1   # mode
    assert lib.conv2d_plan(0, 0, 1, 1, 8, 8, 2, 3, 3, 1, 1, 0, None) == 2
    assert lib.conv2d_plan(4, 0, 1, 1, 8, 8, 2, 3, 3, 1, 1, 0, ctypes.byref(plan)) == 3
    assert lib.conv2d_plan(0, 0, 1, 1, 2, 2, 2, 3, 3, 1, 0, 0, ctypes.byref(plan)) == 1   # no window


def test_zero_skip_choice_follows_density():
    s = SHAPES["resnet_conv"]
    n = s.N * s.C * s.Hin * s.Win
    ch = lambda p, nnz, s=s: dmlnn.conv2d_zero_skip_choice(torch.float64, p, nnz, *s.args())  # noqa
    assert ch("forward", int(0.5 * n)) == 0        # the config's 50% density: no fragment skips
    assert ch("forward", int(0.01 * n)) == 1       # (0.99)^64 = 0.53 of fragments all zero
    assert ch("forward", 0) == 1
    assert ch("forward", int(0.045 * n)) == 1 and ch("forward", int(0.047 * n)) == 0
    assert ch("backward_filter", int(0.01 * n)) == 1
    # kernels with no skip form in the dense mode: never the skip mode
    s1, s2 = SHAPES["lenet_conv1"], SHAPES["lenet_conv2"]
    n1 = s1.N * s1.C * s1.Hin * s1.Win
    assert ch("forward", 0, s1) == 1            # LDS-DMA forward: a skip form
    assert ch("backward_data", 0, s1) == 0      # small-M vector backward_data (one channel)
    assert ch("backward_filter", int(0.01 * n1), s1) == 1
    assert ch("forward", 0, s2) == 0            # filter-resident forward
    with pytest.raises(ValueError):
        ch("forward", n + 1)
    with pytest.raises(ValueError):
        ch("forward", -1)


def test_fused_plan_query():
    """conv2d_plan_fused reports the kernels the fused calls take, and rejects
    a form that does not apply to the pass or a pool it cannot fuse."""
    s = SHAPES["lenet_conv2"]
    pool = (2, 2, 2, 0)
    f = dmlnn.conv2d_plan_fused(torch.float64, "forward", "pool_epilogue", *s.args(), pool=pool)
    assert f["fused"] == 1 and f["kernel"] == "resident"
    d = dmlnn.conv2d_plan_fused(torch.float64, "backward_data", "pooled_source", *s.args(),
                                pool=pool)
    assert d["fused"] == 1 and d["kernel"] == "igemm_dma" and d["zero_skip"] == 0
    w = dmlnn.conv2d_plan_fused(torch.float64, "backward_filter", "pooled_source", *s.args(),
                                pool=pool)
    assert w["kernel"] == dmlnn.conv2d_plan(torch.float64, "backward_filter", *s.args())["kernel"]
    # a padded pool is not fused: the call runs the plain conv, then the pool
    u = dmlnn.conv2d_plan_fused(torch.float64, "forward", "pool_epilogue", *s.args(),
                                pool=(3, 3, 2, 1))
    assert u["fused"] == 0
    # the CSR input always takes the register-staged kernel's direct staging
    c = dmlnn.conv2d_plan_fused(torch.float32, "forward", "csr_input", *s.args())
    assert c["kernel"] == "igemm_reg" and c["pipelined"] == 0
    for args in [("forward", "pooled_source", pool), ("backward_data", "pool_epilogue", pool),
                 ("backward_filter", "csr_input", (0, 0, 0, 0)),
                 ("backward_data", "pooled_source", (3, 3, 2, 0))]:
        with pytest.raises(RuntimeError):
            dmlnn.conv2d_plan_fused(torch.float64, args[0], args[1], *s.args(), pool=args[2])
