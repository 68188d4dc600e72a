"""Write the stored oracle results for the small conv workload (N=4, C=1, 8x8, F=2
3x3 s1 p1) to conv_small_fp64.json.  Calls only the oracle and the seeded input
generator; the stored file locks the oracle against accidental change.

Run from the repository root:  python tests/golden/make_golden.py
"""
import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import oracle  # noqa: E402
from paper_1802_04647_amd.inputs import SHAPES, conv_layer_inputs  # noqa: E402


def main():
    s = SHAPES["conv_small"]
    X, W, b, dout = conv_layer_inputs("conv_small")
    a = (s.C, s.Hin, s.Win, s.Hf, s.Wf, s.stride, s.pad)
    out, _, _ = oracle.conv2d_forward(X, W, b, *a, relu=True)
    dW, db = oracle.conv2d_backward_filter(X, dout, out, *a, s.F)
    dX = oracle.conv2d_backward_data(W, dout, out, *a)
    rec = {"about": "oracle results for the small conv workload; inputs from "
                    "paper_1802_04647_amd.inputs.conv_layer_inputs('conv_small'); "
                    "written by tests/golden/make_golden.py",
           "out": out.tolist(), "dW": dW.tolist(), "db": db.tolist(), "dX": dX.tolist()}
    with open(os.path.join(HERE, "conv_small_fp64.json"), "w") as f:
        json.dump(rec, f, indent=0)


if __name__ == "__main__":
    main()
