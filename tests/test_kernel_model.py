"""The kernels' index arithmetic, modelled on the CPU for every conv shape
the GPU tests and the benchmark launch (kernel_model.py): LDS regions and
accesses in bounds, global accesses inside their tensors, exact divisions,
staging slots that cover what is read, the right operand in every fragment
and every output written once -- with the tiling the library reports for
each shape, pass, precision, zero-skip mode and fused form.  An index or plan
change that would fault or read stale data on the GPU fails here first.
"""
import ast
import glob
import os

import pytest
import torch

import kernel_model as km
from paper_1802_04647_amd import dmlnn
from paper_1802_04647_amd.inputs import SHAPES, ConvShape

HERE = os.path.dirname(os.path.abspath(__file__))
PASSES = ("forward", "backward_filter", "backward_data")
DT = {"f64": torch.float64, "f32": torch.float32}


def _literal_shapes():
    """Every ConvShape(...) with literal arguments in the GPU test files."""
    found = set()
    for path in sorted(glob.glob(os.path.join(HERE, "test_gpu_*.py")) +
                       glob.glob(os.path.join(HERE, "test_zz_*.py"))):
        with open(path) as f:
            tree = ast.parse(f.read())
        for node in ast.walk(tree):
            if (isinstance(node, ast.Call) and getattr(node.func, "id", None) == "ConvShape"
                    and all(isinstance(a, ast.Constant) for a in node.args)
                    and len(node.args) == 9):
                found.add(ConvShape(*(a.value for a in node.args)))
    return found


def _cases():
    """(shape, form, pool) for every conv launch of the GPU tests, the LeNet
    step and the benchmark."""
    from test_gpu_fusion import CASES as POOL_CASES, HCASES, PB_CASES
    from test_gpu_sparse import CASES as SPARSE_CASES
    cases = set()
    plain = _literal_shapes() | set(SHAPES.values())
    plain |= {ConvShape(2, *s.args()[1:]) for s in SHAPES.values()}  # tests that take N = 2
    for s in plain:
        if s.F > 0:
            cases.add((s, "plain", None))
    for s, ph, pw, ps in POOL_CASES:
        cases.add((s, "pool_epilogue", (ph, pw, ps, 0)))
    for s, ph, pw, ps in PB_CASES:
        cases.add((s, "pooled_source", (ph, pw, ps, 0)))
    for s0, Fs in HCASES:
        cases.add((ConvShape(s0.N, s0.C, s0.Hin, s0.Win, sum(Fs), s0.Hf, s0.Wf, s0.stride,
                             s0.pad), "banks", None))
        for F in Fs:  # unfused banks run as plain forwards
            cases.add((ConvShape(s0.N, s0.C, s0.Hin, s0.Win, F, s0.Hf, s0.Wf, s0.stride,
                                 s0.pad), "plain", None))
    for s, _ in SPARSE_CASES:
        cases.add((s, "csr_input", None))
    cases.add((SHAPES["lenet_conv1"], "csr_input", None))
    for name in ("lenet_conv1", "lenet_conv2"):  # the fused LeNet step, batch 64 and 100
        for n in (SHAPES[name].N, 100):
            s = ConvShape(n, *SHAPES[name].args()[1:])
            cases.add((s, "plain", None))
            cases.add((s, "pool_epilogue", (2, 2, 2, 0)))
            cases.add((s, "pooled_source", (2, 2, 2, 0)))
    return sorted(cases, key=lambda c: (str(c[0]), c[1]))


CASES = _cases()
FORM_PASSES = {"plain": PASSES, "pool_epilogue": ("forward",), "csr_input": ("forward",),
               "banks": ("forward",), "pooled_source": ("backward_filter", "backward_data")}


def _plan(s, dt, pname, form, pool, zs):
    if form == "plain":
        return dmlnn.conv2d_plan(DT[dt], pname, *s.args(), zero_skip=zs)
    return dmlnn.conv2d_plan_fused(DT[dt], pname, form, *s.args(), pool=pool or (0, 0, 0, 0),
                                   zero_skip=zs)


def test_cases_cover_the_gpu_tests():
    shapes = {c[0] for c in CASES}
    assert len(shapes) > 60
    assert SHAPES["resnet_conv"] in shapes
    assert {c[1] for c in CASES} == set(FORM_PASSES)


@pytest.mark.parametrize("dt", ["f64", "f32"])
@pytest.mark.parametrize("case", CASES, ids=lambda c: f"{c[0]}-{c[1]}")
def test_kernel_indices(case, dt):
    s, form, pool = case
    seen = set()
    for pname in FORM_PASSES[form]:
        for zs in (0, 1):
            p = _plan(s, dt, pname, form, pool, zs)
            key = (pname, tuple(sorted((k, v) for k, v in p.items() if k != "zero_skip")))
            if key in seen:  # the skip mode changes no index
                continue
            seen.add(key)
            km.check_conv(s, pname, dt, p, form=form, pool=pool)


def test_every_kernel_and_form_is_modelled():
    kinds = set()
    for s, form, pool in CASES:
        for pname in FORM_PASSES[form]:
            p = _plan(s, "f64", pname, form, pool, 0)
            kinds.add((p["kernel"], form if p.get("fused", 1) else "plain"))
    for k in km.MODELS:
        assert any(k == kk for kk, _ in kinds), k
    for want in [("igemm_dma", "pool_epilogue"), ("resident", "pool_epilogue"),
                 ("igemm_dma", "pooled_source"), ("igemm_reg", "pooled_source"),
                 ("small_m", "pooled_source"), ("wgrad_ring", "pooled_source"),
                 ("wgrad_tiles", "pooled_source"), ("wgrad_pool_sparse", "pooled_source"),
                 ("igemm_reg", "csr_input"),
                 ("igemm_dma", "banks")]:
        assert want in kinds, want


# ------------------------------------------------------- planted mistakes
# The model must reject a plan that does not match what the kernels index:
# each case shrinks or shifts one field of a real plan.
PLANTS = [
    ("resnet_conv", "forward", "lds_bytes", -256, "outside the block"),
    ("resnet_conv", "forward", "window_rows", -1, "window rows"),
    ("resnet_conv", "backward_data", "slice_bytes", -256, "stage layout"),
    ("resnet_conv", "forward", "tile_stride", 32, "tile of"),
    ("lenet_conv2", "backward_data", "k_chunk", 4, "k per chunk"),
    ("resnet_conv", "backward_filter", "lds_bytes", -8, "LDS size"),
    ("resnet_conv", "backward_filter", "workspace_bytes", -8, "workspace size"),
    ("lenet_conv2", "backward_filter", "window_rows", -1, "LDS size"),
    ("lenet_conv1", "backward_data", "window_rows", -1, "LDS size"),
    ("lenet_conv2", "forward", "slice_stride", -2, "slice layout"),
    ("resnet_conv", "backward_filter", "row_staged", 2, "row staging"),
    ("resnet_conv", "backward_filter", "row_staged", -1, "row staging"),
]


@pytest.mark.parametrize("plant", PLANTS, ids=lambda p: f"{p[0]}-{p[1]}-{p[2]}{p[3]:+d}")
def test_model_rejects_a_wrong_plan(plant):
    name, pname, field, delta, msg = plant
    s = SHAPES[name]
    p = dict(dmlnn.conv2d_plan(torch.float64, pname, *s.args()))
    km.check_conv(s, pname, "f64", p)  # the real plan passes
    p[field] += delta
    with pytest.raises(km.ModelError, match=msg):
        km.check_conv(s, pname, "f64", p)


def test_model_rejects_a_short_window_of_the_right_size():
    """A backward_filter plan whose window holds one row fewer than a tile
    reads, with its LDS size made to match: the row check reports it."""
    s = SHAPES["lenet_conv2"]
    p = dict(dmlnn.conv2d_plan(torch.float64, "backward_filter", *s.args()))
    nch_alloc = (p["chunk"] - 1) // (s.Hf * s.Wf) + 2
    p["window_rows"] -= 1
    p["lds_bytes"] = 8 * (64 * p["g_stride"] + nch_alloc * p["window_rows"] * p["window_width"])
    with pytest.raises(km.ModelError, match="window rows"):
        km.check_conv(s, "backward_filter", "f64", p)


def test_model_rejects_wrong_divisions():
    with pytest.raises(km.ModelError, match="inexact"):
        km.div_magic([1 << 31], 3)            # beyond the magic multiplier's exact range
    with pytest.raises(km.ModelError, match="numerator"):
        km.div_small([1 << 23], 7)
    assert list(km.div_small([0, 5, 4194303], 7)) == [0, 0, 599186]
    assert list(km.div_magic([0, 65535, 4095], 56)) == [0, 1170, 73]


def test_model_rejects_an_unstaged_operand():
    """A fragment that reads an LDS slot the staging never wrote (a DMA that
    stops one instruction short) is reported."""
    s = SHAPES["lenet_conv2"]
    p = dict(dmlnn.conv2d_plan(torch.float64, "backward_data", *s.args()))
    g = km.gemm_view(s, "backward_data")
    Wpad = p["window_width"]
    real = km.tile_rows

    def short(q0, qend, Qw, S, Hf):  # the window holds one row fewer than the tile reads
        return real(q0, qend, Qw, S, Hf) - 1

    km.tile_rows = short
    try:
        with pytest.raises(km.ModelError):
            km.model_igemm_dma(g, p, 8, "plain")
    finally:
        km.tile_rows = real
    assert Wpad > 0
