"""Runs the C oracle end to end on small seeded inputs (a child process of
the sanitizer test, with the AddressSanitizer/UBSan build of gs_oracle.c
loaded through GS_ORACLE_LIB): one training view, a task unit of two views,
the planted-mistake switch, the SH basis functions, and a render whose
pairs include capped and clamped primitives."""
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import oracle as orc                                   # noqa: E402
from paper_2607_19893_amd import scenes                # noqa: E402

assert os.environ.get("GS_ORACLE_LIB") and orc.lib()._name == os.environ["GS_ORACLE_LIB"]

for deg, n, seed in ((0, 1500, 1), (3, 800, 2)):
    sc = scenes.random_scene(seed, n, deg)
    cam = scenes.look_at((0.0, 0.0, -3.0), (0.0, 0.0, 0.0), (0.0, -1.0, 0.0), 96, 64, 60.0)
    # some opaque primitives (alpha at the 0.99 cap) and negative colours (clamped)
    sc.opacity[: n // 10] = 8.0
    sc.sh[n // 10: n // 5, 0] = -3.0
    tgt = np.random.default_rng(seed).uniform(0, 1, (3, cam.height, cam.width)).astype(np.float32)
    m = [np.zeros_like(a) for _, a in sc.groups()]
    v = [np.zeros_like(a) for _, a in sc.groups()]
    out = orc.train_view(sc, cam, tgt, m, v, 1)
    cam2 = scenes.look_at((0.5, 0.0, -3.0), (0.0, 0.0, 0.0), (0.0, -1.0, 0.0), 80, 72, 55.0)
    tgt2 = np.random.default_rng(seed + 7).uniform(0, 1, (3, cam2.height, cam2.width)).astype(np.float32)
    orc.train_unit(sc, [cam, cam2], [tgt, tgt2], m, v, 1)
    pr = orc.project(sc, cam, 0)
    vis = orc.visible(pr.tiles)
    rn = orc.render(vis, pr, cam)
    orc.ambiguous_pixels(rn)
    for k in (1, 7, 22, 24, 26):
        orc.set_mutation(k)
        orc.render(vis, pr, cam)
    orc.set_mutation(0)
print("ok")
