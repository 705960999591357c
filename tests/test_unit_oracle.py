"""Pins of the oracle's task unit (several views, one optimizer step; Section
2.1): its gradient is the gradient of the sum of the views' losses, checked
by central finite differences of the fp64 forward over two cameras that see
different subsets of a tiny scene; a one-view unit is the training view; the
union rows and the accumulated evidence follow the views' visible sets."""
import numpy as np
import pytest

from paper_2607_19893_amd import scenes
from test_oracle_pins import _forward_loss, _perturbed
from parity_util import target_of


def two_cameras(W=40, H=32):
    """Two narrow cameras turned apart: the second one misses part of the scene."""
    a = scenes.look_at((0.0, 0.0, 0.0), (-0.45, 0.0, 3.0), (0.0, -1.0, 0.0), W, H, 22.0)
    b = scenes.look_at((0.1, -0.1, 0.0), (0.45, 0.05, 3.0), (0.0, -1.0, 0.0), W, H, 22.0)
    return [a, b]


def check_unit_fd(o, seed=6, n=8, deg=2, tol=1e-5):
    rng = np.random.default_rng(seed)
    cams = two_cameras()
    sc = scenes.random_scene(seed, n, deg, extent=0.6, ls_mu=-2.3, ls_sd=0.3, depth=3.0)
    sc.opacity[:] = np.clip(sc.opacity, -2.0, 2.0)
    ws = [rng.standard_normal((3, c.height, c.width)) for c in cams]
    union, grads, gnorm, views = o.unit_gradients(sc, cams, dL_list=ws, mode=1)
    vis_sets = [set(v[0].tolist()) for v in views]
    assert vis_sets[0] != vis_sets[1]                       # the views see different primitives
    names = ["mean", "log_scale", "quat", "opacity", "sh"]
    full = {}
    for name, G in zip(names, grads):
        a = np.zeros((n, G.shape[1]))
        a[union.astype(np.int64)] = G
        full[name] = a

    def total(s):
        Ls, sigs = zip(*(_forward_loss(o, s, c, w) for c, w in zip(cams, ws)))
        return sum(Ls), sigs

    base, base_sig = total(sc)
    checked = skipped = 0
    for name in names:
        flat = getattr(sc, name).reshape(n, -1)
        an = full[name]
        for j in range(n):
            for c in range(flat.shape[1]):
                x0 = float(flat[j, c])
                h = 2e-5 * max(1.0, abs(x0))
                vals, steps, ok = [], [], True
                for sgn in (+1, -1):
                    s2, xs = _perturbed(sc, name, j, c, sgn * h)
                    L, sig = total(s2)
                    ok &= sig == base_sig
                    vals.append(L); steps.append(xs - x0)
                if not ok:
                    skipped += 1
                    continue
                fd = (vals[0] - vals[1]) / (steps[0] - steps[1])
                scale = max(abs(fd), abs(an[j, c]), 1e-7 * np.abs(an).max())
                assert abs(fd - an[j, c]) <= tol * scale, (name, j, c, fd, an[j, c])
                checked += 1
    assert checked > 0.8 * (checked + skipped) and checked > 100, (checked, skipped)


def check_unit_rows(o):
    w = scenes.tiny(n=400)
    cams = [w.cameras[0], scenes.look_at((1.5, 0.0, -3.5), (0.5, 0.0, 0.0), (0.0, -1.0, 0.0), 96, 64, 40.0)]
    tg = [target_of(w, 0)[:, :c.height, :c.width] for c in cams]
    union, grads, gnorm, views = o.unit_gradients(w.scene, cams, targets=tg)
    v0, v1 = views[0][0], views[1][0]
    np.testing.assert_array_equal(union, np.union1d(v0, v1).astype(np.uint32))
    only0 = np.setdiff1d(v0, v1)
    assert only0.size > 0
    # a primitive only one view sees carries exactly that view's gradient and evidence
    single = o.unit_gradients(w.scene, cams[:1], targets=tg[:1])
    r_u = np.searchsorted(union, only0)
    r_s = np.searchsorted(single[0], only0)
    for G, S in zip(grads, single[1]):
        np.testing.assert_array_equal(G[r_u], S[r_s])
    np.testing.assert_array_equal(gnorm[only0.astype(np.int64)], single[2][only0.astype(np.int64)])


def test_unit_gradient_finite_differences(orc):
    check_unit_fd(orc)


def test_unit_rows(orc):
    check_unit_rows(orc)


def test_one_view_unit_is_the_training_view(orc):
    w = scenes.tiny(n=500)
    cam = w.cameras[0]
    m0 = [np.zeros_like(a).reshape(w.scene.n, -1) for _, a in w.scene.groups()]
    v0 = [np.zeros_like(a) for a in m0]
    u = orc.train_unit(w.scene, [cam], [target_of(w, 0)], m0, v0, 1)
    t = orc.train_view(w.scene, cam, target_of(w, 0), m0, v0, 1)
    np.testing.assert_array_equal(u.union, t.vis)
    for a, b in zip(u.grads, t.grads.groups()):
        np.testing.assert_array_equal(a, b)
    for a, b in zip(u.deltas, t.deltas):
        np.testing.assert_array_equal(a, b)
    np.testing.assert_array_equal(u.msg, t.msg)


def test_unit_planted_mistake_is_caught(orc):
    orc.set_mutation(15)                                   # view rows taken as union rows
    try:
        with pytest.raises(AssertionError):
            check_unit_fd(orc)
    finally:
        orc.set_mutation(0)
