"""Oracle against hand-worked examples and its stored results (CPU only)."""
import json
import math
import os

import numpy as np

import oracle
from paper_1802_04647_amd.inputs import SHAPES, conv_layer_inputs

GOLD = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _load(name):
    with open(os.path.join(GOLD, name)) as f:
        return json.load(f)


def test_hand_worked_conv():
    g = _load("hand_conv_3x3_2x2.json")
    a = (g["C"], g["Hin"], g["Win"], g["Hf"], g["Wf"], g["stride"], g["pad"])
    X, W, b = (np.array(g[k], dtype=np.float64) for k in ("X", "W", "b"))
    out, _, _ = oracle.conv2d_forward(X, W, b, *a, relu=True)
    assert np.array_equal(out, np.array(g["out"]))
    dout = np.array(g["dout"], dtype=np.float64)
    dW, db = oracle.conv2d_backward_filter(X, dout, out, *a, 1)
    dX = oracle.conv2d_backward_data(W, dout, out, *a)
    assert np.array_equal(dW, np.array(g["dW"]))
    assert np.array_equal(db, np.array(g["db"]))
    assert np.array_equal(dX, np.array(g["dX"]))


def test_hand_worked_pool():
    g = _load("hand_pool_4x4.json")
    a = (g["C"], g["Hin"], g["Win"], g["Hf"], g["Wf"], g["stride"], g["pad"])
    X = np.array(g["X"], dtype=np.float64)
    out, idx, _, _ = oracle.max_pool2d_fwd(X, *a)
    assert np.array_equal(out, np.array(g["out"]))
    assert np.array_equal(idx, np.array(g["argmax"]))
    dX = oracle.max_pool2d_bwd(np.array(g["dout"], dtype=np.float64), idx, *a)
    assert np.array_equal(dX, np.array(g["dX"]))


def test_softmax_uniform_closed_form():
    g = _load("softmax_uniform_closed_form.json")
    Y = np.eye(g["K"])[g["labels"]]
    loss, dS, P = oracle.softmax_xent(np.zeros((g["N"], g["K"])), Y)
    assert abs(loss - g["loss"]) < 1e-15 and abs(g["loss"] - math.log(10)) < 1e-15
    assert np.allclose(P, g["p"], rtol=0, atol=1e-16)
    assert np.allclose(dS, (g["p"] - Y) / g["N"], rtol=0, atol=1e-17)


def test_stored_small_conv_results_unchanged():
    g = _load("conv_small_fp64.json")
    s = SHAPES["conv_small"]
    X, W, b, dout = conv_layer_inputs("conv_small")
    a = (s.C, s.Hin, s.Win, s.Hf, s.Wf, s.stride, s.pad)
    out, _, _ = oracle.conv2d_forward(X, W, b, *a, relu=True)
    dW, db = oracle.conv2d_backward_filter(X, dout, out, *a, s.F)
    dX = oracle.conv2d_backward_data(W, dout, out, *a)
    for k, v in (("out", out), ("dW", dW), ("db", db), ("dX", dX)):
        assert np.array_equal(v, np.array(g[k])), k
