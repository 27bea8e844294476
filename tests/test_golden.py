"""The oracle reproduces its frozen tiny cases, and a hand-worked Eq. 1 case."""
import json
import os

import numpy as np

import oracle as O

HERE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def test_oracle_reproduces_frozen_cases():
    with open(os.path.join(HERE, "oracle_tiny.json")) as f:
        g = json.load(f)
    ic = g["int_case"]
    x = np.array(ic["x"], dtype=np.int32)
    bx = np.array(ic["boxes"], dtype=np.float32)
    np.testing.assert_array_equal(O.sat_exclusive(x), np.array(ic["sat"]))
    np.testing.assert_array_equal(O.box_forward(x, bx), np.array(ic["y"]))
    fc = g["float_case"]
    x = np.array(fc["x"], dtype=np.float32)
    bx = np.array(fc["boxes"], dtype=np.float32)
    gy = np.array(fc["grad_y"], dtype=np.float32)
    np.testing.assert_allclose(O.box_forward(x, bx), fc["y"], rtol=0, atol=1e-12)
    np.testing.assert_allclose(O.box_backward_input(gy, bx, 5, 4), fc["grad_x"], rtol=0, atol=1e-12)
    np.testing.assert_allclose(O.box_backward_params(x, gy, bx), fc["grad_boxes"], rtol=0, atol=1e-11)


def test_hand_worked_three_by_three():
    """Eq. 1 by hand on I = [[1,2,3],[4,5,6],[7,8,9]] with the centred 3x3 box
    (cx = cy = 0, rx = ry = 3/2, i.e. x_l = y_l = -1, x_h = y_h = 1):
    corner (0,0) sums 1+2+4+5 = 12, the centre sums everything = 45, the top
    middle sums 1+2+3+4+5+6 = 21, the bottom right sums 5+6+8+9 = 28.
    Its exclusive table has last row 0, 12, 27, 45 (running sums of the
    column totals 12, 15, 18)."""
    x = np.arange(1, 10, dtype=np.int32).reshape(1, 1, 3, 3)
    bx = np.array([[[0.0, 0.0, 1.5, 1.5]]], dtype=np.float32)
    y = O.box_forward(x, bx)[0, 0]
    assert y[0, 0] == 12 and y[1, 1] == 45 and y[0, 1] == 21 and y[2, 2] == 28
    assert list(O.sat_exclusive(x)[0, 0, 3]) == [0, 12, 27, 45]
    # half a pixel wider on the right (rx = 1.75, cx = 0.25): the centre pixel
    # now also takes half of a column outside the image -> still 45.
    bx2 = np.array([[[0.25, 0.0, 1.75, 1.5]]], dtype=np.float32)
    y2 = O.box_forward(x.astype(np.float32), bx2)[0, 0]
    assert y2[1, 1] == 45.0
    # and at the left column it gains half of column 2: 12 + (3+6)/2 = 16.5
    assert y2[0, 0] == 16.5
