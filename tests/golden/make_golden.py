"""Writes tests/golden/oracle_small_view.json from the oracle only.

The fixture freezes the oracle's projection, render and gradients for a
seeded 6-primitive, SH-degree-3 scene seen by a 40x32 camera (one training
view as the paper's Section 2.1 describes it: render, image loss, backward).
It is a regression pin: any later change to the oracle's arithmetic shows up
as a diff of this file and needs a stated reason.

Run from the repository root:  python tests/golden/make_golden.py
"""
import json
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from paper_2607_19893_amd import scenes  # noqa: E402


def compute():
    sc = scenes.random_scene(7, 6, 3, extent=0.5, ls_mu=-2.3, ls_sd=0.3, depth=3.0)
    cam = scenes.look_at((0.0, 0.0, 0.0), (0.0, 0.0, 1.0), (0.0, -1.0, 0.0), 40, 32, 60.0)
    tgt = scenes.make_target(40, 32, 7, 0, "uniform")
    m = [np.zeros_like(a) for _, a in sc.groups()]
    v = [np.zeros_like(a) for _, a in sc.groups()]
    r = oracle.train_view(sc, cam, tgt, m, v, 1)
    g = r.grads.full(sc.n)
    return {
        "radius": r.proj.radius.tolist(),
        "rect": r.proj.rect.tolist(),
        "depth_bits": r.proj.depth.view(np.uint32).tolist(),
        "conic_f32_bits": r.proj.conic_f32.view(np.uint32).reshape(-1).tolist(),
        "rgb": r.proj.rgb.reshape(-1).tolist(),
        "keys": [int(k) for k in r.keys],
        "vals": r.vals.tolist(),
        "img_row16": r.render.img[:, 16, :].reshape(-1).tolist(),
        "n_contrib_row16": r.render.n_contrib[16].tolist(),
        "loss": r.loss,
        "grad_mean": g[0].reshape(-1).tolist(),
        "grad_log_scale": g[1].reshape(-1).tolist(),
        "grad_quat": g[2].reshape(-1).tolist(),
        "grad_opacity": g[3].reshape(-1).tolist(),
        "grad_sh": g[4].reshape(-1).tolist(),
    }


if __name__ == "__main__":
    out = os.path.join(os.path.dirname(os.path.abspath(__file__)), "oracle_small_view.json")
    with open(out, "w") as f:
        json.dump({"source": "tests/golden/make_golden.py (oracle only); one training view as in the "
                             "paper's Section 2.1", "data": compute()}, f, indent=0)
    print("wrote", out)
