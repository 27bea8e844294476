"""Writes tests/golden/oracle_tiny.json from the CPU oracle only.

The paper prints no worked numeric example of the box filter, its table or its
gradients, so no stored value here comes from the paper.  This file freezes
the oracle's output on two tiny seeded cases (an integer-corner case, exact in
int64, and a sub-pixel case in fp64) so that any later change to the oracle's
arithmetic shows up as a diff of a committed file.

Run:  python tests/golden/make_golden.py
"""
import json
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import oracle as O  # noqa: E402


def cases():
    rng = np.random.default_rng(2019)
    xi = rng.integers(-8, 9, size=(1, 2, 5, 6)).astype(np.int32)
    bi = np.array([[[0.0, 0.0, 1.5, 1.5], [2.5, -0.5, 1.0, 2.0]],
                   [[-1.5, 1.0, 2.0, 0.5], [0.0, 0.0, 0.5, 0.5]]], dtype=np.float32)
    xf = rng.standard_normal((1, 1, 5, 4)).astype(np.float32)
    bf = np.array([[[0.3, -0.45, 1.2, 0.8], [-1.7, 0.9, 0.55, 2.1]]], dtype=np.float32)
    gf = rng.standard_normal((1, 2, 5, 4)).astype(np.float32)
    return xi, bi, xf, bf, gf


def main():
    xi, bi, xf, bf, gf = cases()
    out = {
        "note": "written by tests/golden/make_golden.py from the CPU oracle",
        "int_case": {"x": xi.tolist(), "boxes": bi.tolist(),
                     "sat": O.sat_exclusive(xi).tolist(),
                     "y": O.box_forward(xi, bi).tolist()},
        "float_case": {"x": xf.tolist(), "boxes": bf.tolist(), "grad_y": gf.tolist(),
                       "y": O.box_forward(xf, bf).tolist(),
                       "grad_x": O.box_backward_input(gf, bf, 5, 4).tolist(),
                       "grad_boxes": O.box_backward_params(xf, gf, bf).tolist()},
    }
    with open(os.path.join(HERE, "oracle_tiny.json"), "w") as f:
        json.dump(out, f, indent=1)


if __name__ == "__main__":
    main()
