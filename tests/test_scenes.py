"""Host-side workload helpers: the spatial (Morton) storage order of the
primitive pool is a permutation that follows the Z-order curve, and storing
the pool in it changes no rendered result (CPU oracle)."""
import numpy as np
import pytest

from paper_2607_19893_amd import scenes


def _morton_ref(q):
    """Bit-by-bit interleave of three 21-bit integers (x in bit 0, y in bit 1, z in bit 2)."""
    c = 0
    for b in range(21):
        c |= ((int(q[0]) >> b) & 1) << (3 * b) | ((int(q[1]) >> b) & 1) << (3 * b + 1) | \
             ((int(q[2]) >> b) & 1) << (3 * b + 2)
    return c


def test_morton_codes_interleave_bits():
    rng = np.random.default_rng(0)
    q = rng.integers(0, 2 ** 21, (300, 3))
    got = scenes._spread3(q[:, 0]) | (scenes._spread3(q[:, 1]) << np.uint64(1)) | \
        (scenes._spread3(q[:, 2]) << np.uint64(2))
    assert [int(g) for g in got] == [_morton_ref(r) for r in q]


def test_morton_codes_quantize_the_bounding_box():
    m = np.array([[0.0, 0.0, 0.0], [1.0, 1.0, 1.0], [1.0, 0.0, 0.0], [0.0, 1.0, 0.0], [0.0, 0.0, 1.0]], np.float32)
    c = scenes.morton_codes(m)
    top = 2 ** 21 - 1
    assert int(c[0]) == 0
    assert int(c[1]) == _morton_ref((top, top, top))
    assert [int(x) for x in c[2:]] == [_morton_ref((top, 0, 0)), _morton_ref((0, top, 0)), _morton_ref((0, 0, top))]


def test_spatial_order_is_a_sorting_permutation():
    rng = np.random.default_rng(1)
    m = rng.uniform(-5, 5, (50000, 3)).astype(np.float32)
    m[100:200] = m[100]                                    # equal codes keep their given order
    p = scenes.spatial_order(m)
    assert np.array_equal(np.sort(p), np.arange(m.shape[0]))
    c = scenes.morton_codes(m)[p]
    assert np.all(c[1:] >= c[:-1])
    ties = p[np.isin(p, np.arange(100, 200))]
    assert np.all(np.diff(ties) > 0)
    # a small box of space falls into few runs of consecutive positions
    inside = np.flatnonzero(np.all(np.abs(m[p] - 2.5) < 1.0, axis=1))
    runs = 1 + int(np.count_nonzero(np.diff(inside) > 1))
    assert inside.size > 20 and runs < inside.size / 2


def test_permuted_scene_renders_the_same(orc):
    w = scenes.tiny(n=3000)
    cam = w.cameras[0]
    perm = scenes.spatial_order(w.scene.mean)
    ws = scenes.spatially_ordered(w)
    assert np.array_equal(ws.scene.mean, w.scene.mean[perm]) and np.array_equal(ws.scene.sh, w.scene.sh[perm])
    assert np.array_equal(ws.target(0), w.target(0))
    r0 = orc.render(orc.visible(orc.project(w.scene, cam, 0).tiles), orc.project(w.scene, cam, 0), cam)
    p1 = orc.project(ws.scene, cam, 0)
    r1 = orc.render(orc.visible(p1.tiles), p1, cam)
    np.testing.assert_allclose(r1.img, r0.img, rtol=1e-12, atol=1e-15)
    np.testing.assert_array_equal(r1.active[np.argsort(perm)], r0.active)


def test_perturbed_copy_is_one_scene_in_any_storage_order():
    """The ring workload's targets are renders of a perturbed copy: the copy
    of the spatially ordered pool is the copy of the generated pool, rows
    permuted the same way (each primitive keeps its own noise), and it differs
    from the pool itself by the stated noise scales."""
    w = scenes.ring(n=5000, width=64, height=48)
    assert w.target_kind == "perturbed"
    ws = scenes.spatially_ordered(w)
    a, b = w.target_scene(), ws.target_scene()
    for x, y in zip(a.groups(), b.groups()):
        np.testing.assert_array_equal(x[1][ws.perm], y[1])
    d = (a.mean - w.scene.mean).std(), (a.opacity - w.scene.opacity).std(), (a.sh - w.scene.sh).std()
    assert abs(d[0] - 0.02) < 0.002 and abs(d[1] - 0.5) < 0.05 and abs(d[2] - 0.05) < 0.005
    with pytest.raises(ValueError):
        w.target(0)
    img = w.target(0, render=lambda sc, cam: np.full((3, cam.height, cam.width), 0.25, np.float32))
    assert img.shape == (3, 48, 64) and img.dtype == np.float32
