"""The oracle still reproduces the frozen small-view fixture (regression pin)."""
import json
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))


def test_oracle_reproduces_golden_fixture(orc):
    import sys
    sys.path.insert(0, os.path.join(HERE, "golden"))
    import make_golden
    ref = json.load(open(os.path.join(HERE, "golden", "oracle_small_view.json")))["data"]
    got = make_golden.compute()
    for k in ("radius", "rect", "depth_bits", "conic_f32_bits", "keys", "vals", "n_contrib_row16"):
        assert got[k] == ref[k], k
    for k in ("rgb", "img_row16", "grad_mean", "grad_log_scale", "grad_quat", "grad_opacity", "grad_sh"):
        np.testing.assert_allclose(got[k], ref[k], rtol=1e-10, atol=1e-16, err_msg=k)
    assert abs(got["loss"] - ref["loss"]) < 1e-12
