"""The LeNet training step recorded as a HIP graph and replayed: every replay
must equal the eager step bitwise (same kernels, same order, deterministic
reductions), with eager work and synchronisations between the replays and a
new batch copied into the static inputs halfway.  The eager step runs its
weight gradients on a second stream and the graph holds the single-stream form,
so this also checks that the two forms agree bitwise."""
import numpy as np
import pytest
import torch

from gpu_util import dev
from paper_1802_04647_amd.inputs import lenet_train_inputs, sparse_uniform, streams
from paper_1802_04647_amd.lenet import LeNetTrainer

pytestmark = pytest.mark.gpu


def test_lenet_graph_replay_matches_eager():
    X, Y, params = lenet_train_inputs()
    Xd, Yd = dev(X, "f64"), dev(Y, "f64")
    g_x, g_mask = streams(991)[:2]
    X2 = dev(sparse_uniform(g_mask, g_x, X.shape, keep=0.2), "f64")
    Y2 = torch.roll(Yd, 1, dims=0).contiguous()
    eager = LeNetTrainer(params)
    graphed = LeNetTrainer(params)
    graphed.capture(Xd, Yd, warmup=1)      # one eager warm-up step inside
    eager.step(Xd, Yd)
    torch.cuda.synchronize()
    assert torch.equal(eager.p_flat, graphed.p_flat)
    for k in range(4):
        xb, yb = (Xd, Yd) if k < 2 else (X2, Y2)
        le = eager.step(xb, yb)
        lg = graphed.replay(xb, yb)
        torch.cuda.synchronize()
        junk = torch.randn(1000, device="cuda").sum()          # eager work between replays
        torch.cuda.synchronize()
        assert torch.isfinite(junk)
        assert torch.equal(le, lg), k
        assert torch.equal(eager.p_flat, graphed.p_flat), k
        assert torch.equal(eager.v_flat, graphed.v_flat), k
    assert not np.isnan(graphed.graph_loss.item())
