"""Pin the oracle's composed LeNet training step to torch autograd + torch.optim.SGD
(CPU, float64).  This checks the layer order, the relu/pool gradient routing and
the momentum form together, on the same shapes as the training workload (batch
reduced to keep the CPU suite quick)."""
import numpy as np
import torch
import torch.nn.functional as tF

from oracle import lenet as lenet_oracle
from paper_1802_04647_amd.inputs import lenet_train_inputs


def _torch_step(X, Y, params, steps, lr=0.01, mu=0.9):
    N = X.shape[0]
    t = {k: torch.nn.Parameter(torch.from_numpy(v.copy())) for k, v in params.items()}
    opt = torch.optim.SGD(list(t.values()), lr=lr, momentum=mu)
    losses = []
    for _ in range(steps):
        opt.zero_grad()
        x = torch.from_numpy(X).reshape(N, 1, 28, 28)
        h = torch.relu(tF.conv2d(x, t["W1"].reshape(32, 1, 5, 5), t["b1"], padding=2))
        h = tF.max_pool2d(h, 2, 2)
        h = torch.relu(tF.conv2d(h, t["W2"].reshape(64, 32, 5, 5), t["b2"], padding=2))
        h = tF.max_pool2d(h, 2, 2).reshape(N, -1)
        h = torch.relu(h @ t["W3"] + t["b3"])
        s = h @ t["W4"] + t["b4"]
        loss = tF.cross_entropy(s, torch.from_numpy(Y.argmax(1)))
        loss.backward()
        opt.step()
        losses.append(loss.item())
    return losses, {k: v.detach().numpy() for k, v in t.items()}


def test_lenet_three_steps_match_torch():
    X, Y, params = lenet_train_inputs(N=8)
    vel = lenet_oracle.zero_velocities(params)
    p = params
    losses = []
    for _ in range(3):
        loss, p, vel, _, _ = lenet_oracle.train_step(X, Y, p, vel)
        losses.append(loss)
    tl, tp = _torch_step(X, Y, params, 3)
    assert np.allclose(losses, tl, rtol=1e-12, atol=0)
    for k in lenet_oracle.PARAM_ORDER:
        d = np.max(np.abs(p[k] - tp[k])) / max(np.max(np.abs(tp[k])), 1e-300)
        assert d < 1e-12, (k, d)
