"""Forward-only scoring on the GPU: the softmax_fwd entry point and the
multi-stream LeNet scorer, against the oracle."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import assert_close, dev, host, rounded
from oracle.lenet import forward_probs
from paper_1802_04647_amd import dmlnn
from paper_1802_04647_amd.inputs import lenet_train_inputs, sparse_uniform, streams
from paper_1802_04647_amd.lenet import LeNetScorer

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("dt", ["f64", "f32"])
@pytest.mark.parametrize("N,K", [(64, 10), (1000, 10), (37, 1), (5, 100), (3, 64), (130, 33)])
def test_softmax_fwd(N, K, dt):
    r = np.random.default_rng(N * 131 + K)
    S = rounded(r.standard_normal((N, K)) * 4, dt)
    P = dmlnn.softmax_fwd(dev(S, dt))
    torch.cuda.synchronize()
    ref = oracle.softmax_forward(S)
    assert_close(host(P), ref, dt, "probs")


def _images(M):
    g_x, g_mask = streams(977)[:2]
    return sparse_uniform(g_mask, g_x, (M, 784), keep=0.2)


def test_lenet_scoring_matches_oracle_and_is_stream_independent():
    _, _, params = lenet_train_inputs()
    X = _images(320)                      # five batches of 64
    Xd = torch.from_numpy(X).cuda()
    p3 = LeNetScorer(params, batch=64, streams=3).score(Xd)
    p1 = LeNetScorer(params, batch=64, streams=1).score(Xd)
    torch.cuda.synchronize()
    assert torch.equal(p1, p3)            # same kernels per batch, whatever the stream
    ref = forward_probs(X, params)
    assert_close(host(p3), ref, "f64", "probs")
    np.testing.assert_allclose(host(p3).sum(axis=1), 1.0, rtol=1e-12)
