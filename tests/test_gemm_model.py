"""The affine kernel's index arithmetic, modelled on the CPU (gemm_model.py)
for every affine shape the GPU tests and the LeNet step launch, in both
dtypes, with the full workspace, a two-split workspace and none."""
import pytest
import torch

import gemm_model as gm
from kernel_model import ModelError
from paper_1802_04647_amd import dmlnn
from test_gpu_ops import AFFINE, SPLIT

SHAPES = sorted(set(AFFINE) | set(SPLIT) | {(20, 96, 40), (64, 512, 10), (64, 3136, 512),
                                             (100, 512, 10), (100, 3136, 512),
                                             (33, 70, 65), (5, 7, 3)})
DT = {"f64": torch.float64, "f32": torch.float32}


@pytest.mark.parametrize("dt", ["f64", "f32"])
@pytest.mark.parametrize("shape", SHAPES, ids=str)
def test_gemm_indices(shape, dt):
    N, D, M = shape
    tsz = 8 if dt == "f64" else 4
    full = dmlnn.affine_workspace_size(DT[dt], N, D, M)
    for ws in {full, 2 * max(N * M, N * D, D * M) * tsz, 0}:
        for product in ("forward", "dX", "dW"):
            plan = dmlnn.affine_plan(DT[dt], product, N, D, M, ws)
            gm.check_gemm(product, N, D, M, tsz, plan, ws)


def test_plans_take_both_tiles_and_splits():
    seen = set()
    for N, D, M in SHAPES:
        for product in ("forward", "dX", "dW"):
            full = dmlnn.affine_workspace_size(torch.float64, N, D, M)
            p = dmlnn.affine_plan(torch.float64, product, N, D, M, full)
            seen.add((p["tile"], p["splits"] > 1, p["waves"] > 1))
    assert {t for t, _, _ in seen} == {16, 32}
    assert any(s for _, s, _ in seen) and any(w for _, _, w in seen)


def test_model_rejects_a_wrong_plan():
    N, D, M = 64, 3136, 512
    p = dmlnn.affine_plan(torch.float64, "forward", N, D, M,
                          dmlnn.affine_workspace_size(torch.float64, N, D, M))
    assert p["splits"] > 1
    with pytest.raises(ModelError, match="workspace"):
        gm.check_gemm("forward", N, D, M, 8, p, 0)
    with pytest.raises(ModelError, match="plan"):
        gm.check_gemm("forward", N, D, M, 8, dict(p, tile=48), 1 << 40)


def test_plan_query_validation():
    with pytest.raises(dmlnn.DmlnnError):
        dmlnn.affine_plan(torch.float64, "forward", 0, 3, 4, 0)
