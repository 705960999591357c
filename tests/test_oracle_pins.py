"""Pins of the CPU oracle against facts that do not come from the oracle itself.

Each check is a plain function so that the mutation test at the bottom can
re-run it with a deliberate mistake switched on inside the oracle and see it
fail.  Sources of truth used here:
  * closed forms of special cases (one on-axis Gaussian, two stacked ones, an
    isotropic off-axis Gaussian, the image moments of a rotated anisotropic
    Gaussian, points on a camera's axes);
  * a library routine (scipy's complex spherical harmonics, torch's Adam and
    L1 loss);
  * quadrature (orthonormality of the SH basis);
  * brute force on tiny inputs (sorted pairs, visible ids);
  * central finite differences of the fp64 forward (every gradient).
"""
import dataclasses
import math

import numpy as np
import pytest

from paper_2607_19893_amd import scenes

SQRT_PI2 = 2.0 * math.sqrt(math.pi)


def axis_camera(w=64, h=64, fov=60.0):
    """Camera at the origin looking down +z; R is the identity."""
    return scenes.look_at((0.0, 0.0, 0.0), (0.0, 0.0, 1.0), (0.0, -1.0, 0.0), w, h, fov)


def make_scene(means, scales, quats, opac, rgb=None, sh=None, deg=0):
    means = np.asarray(means, np.float64).reshape(-1, 3)
    n = means.shape[0]
    ls = np.log(np.broadcast_to(np.asarray(scales, np.float64), (n, 3)))
    q = np.broadcast_to(np.asarray(quats, np.float64), (n, 4))
    op = np.broadcast_to(np.asarray(opac, np.float64), (n,))
    logit = np.log(op / (1.0 - op))
    K = (deg + 1) ** 2
    if sh is None:
        sh = np.zeros((n, K, 3))
        rgb = np.broadcast_to(np.asarray(rgb, np.float64), (n, 3))
        sh[:, 0, :] = (rgb - 0.5) * SQRT_PI2
    return scenes.Scene(mean=means.astype(np.float32), log_scale=ls.astype(np.float32),
                        quat=np.ascontiguousarray(q, np.float32), opacity=logit.astype(np.float32),
                        sh=np.ascontiguousarray(sh, np.float32), sh_degree=deg)


def pixel_grid(cam):
    ys, xs = np.meshgrid(np.arange(cam.height) + 0.5, np.arange(cam.width) + 0.5, indexing="ij")
    return xs, ys


def tile_mask(cam, rect):
    x0, y0, x1, y1 = rect
    xs, ys = pixel_grid(cam)
    tx, ty = (xs // 16).astype(int), (ys // 16).astype(int)
    return (tx >= x0) & (tx < x1) & (ty >= y0) & (ty < y1)


# ---------------------------------------------------------------------------
# spherical harmonics
# ---------------------------------------------------------------------------

def real_sh_scipy(l, m, theta, phi):
    from scipy.special import sph_harm_y
    if m > 0:
        return math.sqrt(2.0) * sph_harm_y(l, m, theta, phi).real
    if m < 0:
        return math.sqrt(2.0) * sph_harm_y(l, -m, theta, phi).imag
    return sph_harm_y(l, 0, theta, phi).real


def sh_oracle(orc, dirs, deg=3):
    import ctypes
    dirs = np.ascontiguousarray(dirs, np.float64)
    out = np.zeros((dirs.shape[0], 16))
    orc.lib().orc_sh_basis(deg, dirs.ctypes.data_as(ctypes.c_void_p), dirs.shape[0],
                           out.ctypes.data_as(ctypes.c_void_p))
    return out


def sh_oracle_grad(orc, dirs, deg=3):
    import ctypes
    dirs = np.ascontiguousarray(dirs, np.float64)
    out = np.zeros((dirs.shape[0], 16, 3))
    orc.lib().orc_sh_basis_grad(deg, dirs.ctypes.data_as(ctypes.c_void_p), dirs.shape[0],
                                out.ctypes.data_as(ctypes.c_void_p))
    return out


def check_sh_vs_scipy(orc):
    rng = np.random.default_rng(5)
    theta = np.arccos(rng.uniform(-1, 1, 200))
    phi = rng.uniform(0, 2 * math.pi, 200)
    d = np.stack([np.sin(theta) * np.cos(phi), np.sin(theta) * np.sin(phi), np.cos(theta)], 1)
    Y = sh_oracle(orc, d)
    for l in range(4):
        for m in range(-l, l + 1):
            ref = real_sh_scipy(l, m, theta, phi)
            np.testing.assert_allclose(Y[:, l * l + l + m], ref, atol=1e-13, err_msg=f"l={l} m={m}")


def test_sh_matches_scipy(orc):
    check_sh_vs_scipy(orc)


def test_sh_orthonormal_by_quadrature(orc):
    xg, wg = np.polynomial.legendre.leggauss(16)
    nphi = 32
    phi = 2 * math.pi * np.arange(nphi) / nphi
    Z, P = np.meshgrid(xg, phi, indexing="ij")
    W = np.meshgrid(wg, np.full(nphi, 2 * math.pi / nphi), indexing="ij")
    w = (W[0] * W[1]).reshape(-1)
    st = np.sqrt(1 - Z ** 2)
    d = np.stack([st * np.cos(P), st * np.sin(P), Z], -1).reshape(-1, 3)
    Y = sh_oracle(orc, d)
    G = (Y * w[:, None]).T @ Y
    np.testing.assert_allclose(G, np.eye(16), atol=1e-12)
    assert abs(Y[0, 0] - 1.0 / SQRT_PI2) < 1e-15


def test_sh_gradient_finite_difference(orc):
    rng = np.random.default_rng(6)
    d = rng.standard_normal((20, 3))
    d /= np.linalg.norm(d, axis=1, keepdims=True)
    G = sh_oracle_grad(orc, d)
    h = 1e-6
    for i in range(3):
        e = np.zeros(3); e[i] = h
        dp = d + e; dp /= np.linalg.norm(dp, axis=1, keepdims=True)
        dm = d - e; dm /= np.linalg.norm(dm, axis=1, keepdims=True)
        fd = (sh_oracle(orc, dp) - sh_oracle(orc, dm)) / (2 * h)
        # d normalize(d)/dd_i at |d| = 1 is (e_i - d d_i): the polynomial
        # gradient contracted with it is the derivative along the sphere
        an = np.einsum("nkj,nj->nk", G, (np.eye(3)[i][None, :] - d * d[:, i:i + 1]))
        np.testing.assert_allclose(an, fd, atol=1e-7)


# ---------------------------------------------------------------------------
# projection and compositing closed forms
# ---------------------------------------------------------------------------

def check_single_gaussian(orc, mode, o=0.8, s=0.2, W=64):
    """One on-axis isotropic Gaussian: the image is rgb * min(0.99, o exp(-rho^2 / (2 var)))
    with var = (fx s / z)^2 + 0.3, inside the tile rectangle where alpha >= 1/255."""
    cam = axis_camera(W, W, 60.0)
    z, rgb = 4.0, (0.7, 0.2, 0.45)
    sc = make_scene([[0.0, 0.0, z]], [s, s, s], [1, 0, 0, 0], o, rgb=rgb)
    pr = orc.project(sc, cam, mode)
    vis = orc.visible(pr.tiles)
    assert list(vis) == [0]
    fx = float(np.float64(np.float32(cam.fx)))
    s32 = float(np.float32(math.exp(float(np.float32(math.log(s))))))
    var = (fx * s32 / z) ** 2 + 0.3
    np.testing.assert_allclose(pr.conic[0], [1 / var, 0.0, 1 / var], rtol=2e-6, atol=1e-9)
    np.testing.assert_allclose(pr.mean2d[0], [cam.cx, cam.cy], atol=1e-5)
    r = math.ceil(3 * math.sqrt(var + math.sqrt(0.1)))
    assert pr.radius[0] == r
    rect = [max(0, math.floor((cam.cx - r) / 16)), max(0, math.floor((cam.cy - r) / 16)),
            min(cam.tiles_x, math.floor((cam.cx + r + 15) / 16)), min(cam.tiles_y, math.floor((cam.cy + r + 15) / 16))]
    assert list(pr.rect[0]) == rect
    rn = orc.render(vis, pr, cam)
    xs, ys = pixel_grid(cam)
    g = o * np.exp(-0.5 * ((xs - cam.cx) ** 2 + (ys - cam.cy) ** 2) / var)
    alpha = np.minimum(0.99, g)
    inc = tile_mask(cam, rect) & (alpha >= 1 / 255)
    safe = np.abs(g - 1 / 255) / (1 / 255) > 1e-4
    rgb32 = np.float32((np.asarray(rgb) - 0.5) * SQRT_PI2).astype(np.float64) / SQRT_PI2 + 0.5
    for ch in range(3):
        exp_img = np.where(inc, rgb32[ch] * alpha, 0.0)
        np.testing.assert_allclose(rn.img[ch][safe], exp_img[safe], rtol=1e-5, atol=1e-12)
    np.testing.assert_allclose(rn.T_final[safe], np.where(inc, 1 - alpha, 1.0)[safe], rtol=1e-5)
    assert inc.sum() > 50
    return g, rn, rgb32, cam, sc, pr, vis


@pytest.mark.parametrize("mode", [0, 1])
def test_single_gaussian_closed_form(orc, mode):
    check_single_gaussian(orc, mode)


def check_capped_closed_form(orc, mode=1):
    """alpha = min(0.99, o e^-sigma): with o = 0.995 the pixels where
    o e^-sigma >= 0.99 render exactly 0.99 * rgb and keep T = 1 - 0.99; the
    capped-pair signature marks exactly those pixels (the one pair is at list
    position 0, so its entry is 1)."""
    g, rn, rgb32, cam, sc, pr, vis = check_single_gaussian(orc, mode, o=0.995, s=1.0, W=128)
    core = g >= 0.99
    assert core.sum() >= 12, core.sum()
    for ch in range(3):
        assert np.all(rn.img[ch][core] == 0.99 * rgb32[ch])
    assert np.all(rn.T_final[core] == 1.0 - 0.99)
    away = np.abs(g - 0.99) > 1e-9
    assert np.array_equal((rn.capped_sig > 0)[away], core[away])
    assert set(np.unique(rn.capped_sig)) <= {0, 1}


def test_alpha_cap_closed_form(orc):
    check_capped_closed_form(orc, 1)
    check_capped_closed_form(orc, 0)


def check_clamped_colour(orc, mode=1):
    """rgb = max(0, SH(d) + 0.5): a Gaussian whose red sum is -0.3 renders
    exactly 0 in red everywhere, carries clamp bit 0, and leaves the other
    channels as the closed form says."""
    cam = axis_camera(64, 64, 60.0)
    sc = make_scene([[0.0, 0.0, 4.0]], [0.2] * 3, [1, 0, 0, 0], 0.8, rgb=(-0.3, 0.4, 0.6))
    pr = orc.project(sc, cam, mode)
    vis = orc.visible(pr.tiles)
    assert list(vis) == [0]
    assert pr.clamp[0] == 1
    assert pr.rgb[0, 0] == 0.0
    np.testing.assert_allclose(pr.rgb[0, 1:], [0.4, 0.6], rtol=1e-6)
    rn = orc.render(vis, pr, cam)
    assert np.all(rn.img[0] == 0.0)
    assert rn.img[1].max() > 0.3 and rn.img[2].max() > 0.45


def test_colour_clamp_closed_form(orc):
    check_clamped_colour(orc, 1)
    check_clamped_colour(orc, 0)


def check_capped_backward(orc):
    """Zero derivative through a pair held at the cap: with the upstream
    gradient non-zero only on pixels where the single Gaussian of
    check_capped_closed_form is capped (T = 1, nothing behind, bg = 0), the
    derivatives w.r.t. u, v, the conic and the opacity are exactly 0, and the
    colour derivative is sum over those pixels of alpha T w = 0.99 * sum w."""
    g, rn, rgb32, cam, sc, pr, vis = check_single_gaussian(orc, 1, o=0.995, s=1.0, W=128)
    core = g >= 0.99 * (1 + 1e-9)
    rng = np.random.default_rng(4)
    w = np.zeros((3, cam.height, cam.width))
    w[:, core] = rng.uniform(0.5, 1.5, (3, int(core.sum())))
    g2, _ = orc.render_backward(vis, pr, cam, w)
    assert np.all(g2[0, :6] == 0.0), g2[0, :6]
    np.testing.assert_allclose(g2[0, 6:], 0.99 * w[:, core].sum(axis=1), rtol=1e-14)


def test_capped_pair_backward_is_zero(orc):
    check_capped_backward(orc)


def _stack_at_pixel(orc, opacities):
    """Gaussians stacked on the centre of pixel (8, 8) of a 16 x 16 image (one
    tile), front to back in the given order, each seen there with sigma = 0,
    so that its alpha at that pixel is its opacity exactly."""
    n = len(opacities)
    pr = orc.Projection(radius=np.full(n, 8, np.int32), tiles=np.ones(n, np.uint32),
                        rect=np.tile(np.array([0, 0, 1, 1], np.int32), (n, 1)),
                        depth=np.arange(1, n + 1, dtype=np.float32),
                        mean2d=np.tile([8.5, 8.5], (n, 1)), conic=np.tile([4.0, 0.0, 4.0], (n, 1)),
                        mean2d_f32=np.tile(np.float32([8.5, 8.5]), (n, 1)),
                        conic_f32=np.tile(np.float32([4.0, 0.0, 4.0]), (n, 1)),
                        opacity=np.asarray(opacities, np.float64), rgb=np.full((n, 3), 0.5),
                        clamp=np.zeros(n, np.uint8), clamp_margin=np.full(n, np.inf),
                        jclamp_margin=np.full(n, np.inf))
    cam = dataclasses.make_dataclass("Cam", ["width", "height"])(16, 16)
    w = np.zeros((3, 16, 16))
    w[0, 8, 8] = 1.0
    return pr, cam, w, np.arange(n, dtype=np.uint32)


def test_alternative_outcome_of_banded_decisions(orc):
    """The backward's alternative pass takes the other outcome of each failed
    decision within its band and no other.  d L / d r of a pair at the one
    pixel with dL/dR = 1 is alpha T when it is included and 0 when not."""
    a_min = 1.0 / 255.0
    # an alpha test failing within the band: left out, included by the alternative
    for rel, inside in ((0.5 * orc.AMB_ALPHA, True), (2.0 * orc.AMB_ALPHA, False)):
        o = a_min * (1.0 - rel)
        pr, cam, w, vis = _stack_at_pixel(orc, [o])
        g0, _ = orc.render_backward(vis, pr, cam, w)
        g1, _ = orc.render_backward(vis, pr, cam, w, alternative=True)
        assert g0[0, 6] == 0.0
        assert g1[0, 6] == (o if inside else 0.0)
    # a termination test within the band: the fourth pair's T (1e-3 behind
    # three pairs of alpha 0.9) would fall just under 1e-4, so the pixel stops
    # there; the alternative includes it and stops at the fifth, whose test
    # lies far outside the band.  The pairs in front gain the fourth's colour
    # in their suffix: d L / d o_k there is T_k (c - S_k / (1 - alpha_k)).
    T3 = 1.0
    for _ in range(3):
        T3 *= 1.0 - 0.9
    for rel, inside in ((0.5 * orc.AMB_T, True), (2.0 * orc.AMB_T, False)):
        a4 = 1.0 - 1e-4 * (1.0 - rel) / T3
        pr, cam, w, vis = _stack_at_pixel(orc, [0.9, 0.9, 0.9, a4, 0.5])
        g0, _ = orc.render_backward(vis, pr, cam, w)
        g1, _ = orc.render_backward(vis, pr, cam, w, alternative=True)
        assert g0[3, 6] == 0.0 and g0[4, 6] == 0.0
        assert g1[4, 6] == 0.0
        if not inside:
            np.testing.assert_array_equal(g1, g0)
            continue
        assert math.isclose(g1[3, 6], a4 * T3, rel_tol=1e-12)
        # the suffix behind the third pair gains the fourth's 0.5 a4 T3 in the
        # alternative, so its d L / d o differs by -0.5 a4 T3 / (1 - 0.9)
        diff = g1[2, 5] - g0[2, 5]
        assert math.isclose(diff, -0.5 * a4 * T3 / (1.0 - 0.9), rel_tol=1e-9), diff


def test_two_layer_composite(orc):
    cam = axis_camera(64, 64, 60.0)
    sc = make_scene([[0.0, 0.0, 3.0], [0.0, 0.0, 5.0]], [[0.04] * 3, [0.12] * 3], [1, 0, 0, 0],
                    [0.6, 0.8], rgb=[[0.9, 0.1, 0.3], [0.2, 0.6, 0.8]])
    pr = orc.project(sc, cam, 1)
    vis = orc.visible(pr.tiles)
    rn = orc.render(vis, pr, cam)
    xs, ys = pixel_grid(cam)
    alphas, incs, gs = [], [], []
    for j in range(2):
        A = pr.conic[j, 0]
        gj = pr.opacity[j] * np.exp(-0.5 * A * ((xs - cam.cx) ** 2 + (ys - cam.cy) ** 2))
        a = np.minimum(0.99, gj)
        inc = tile_mask(cam, pr.rect[j]) & (a >= 1 / 255)
        alphas.append(np.where(inc, a, 0.0)); gs.append(gj)
    safe = np.ones_like(xs, bool)
    for gj in gs:
        safe &= np.abs(gj - 1 / 255) / (1 / 255) > 1e-6
    for ch in range(3):
        e = pr.rgb[0, ch] * alphas[0] + pr.rgb[1, ch] * alphas[1] * (1 - alphas[0])
        np.testing.assert_allclose(rn.img[ch][safe], e[safe], rtol=1e-12, atol=1e-15)


def check_offaxis_isotropic(orc, mode):
    cam = axis_camera(128, 96, 60.0)
    pts = [[0.4, -0.3, 3.0], [-0.7, 0.5, 5.0], [1.0, 0.8, 4.0]]
    s = 0.03
    sc = make_scene(pts, [s, s, s], [1, 0, 0, 0], 0.5, rgb=(0.5, 0.5, 0.5))
    pr = orc.project(sc, cam, mode)
    fx, fy = cam.fx, cam.fy
    s32 = float(np.float32(math.exp(float(np.float32(math.log(s))))))
    for j, (x, y, z) in enumerate(pts):
        x, y, z = [float(np.float32(c)) for c in (x, y, z)]
        assert abs(pr.mean2d[j, 0] - (fx * x / z + cam.cx)) < 2e-4
        assert abs(pr.mean2d[j, 1] - (fy * y / z + cam.cy)) < 2e-4
        a = s32 ** 2 * (fx ** 2 / z ** 2 + fx ** 2 * x ** 2 / z ** 4) + 0.3
        b = s32 ** 2 * fx * fy * x * y / z ** 4
        c = s32 ** 2 * (fy ** 2 / z ** 2 + fy ** 2 * y ** 2 / z ** 4) + 0.3
        D = a * c - b * b
        np.testing.assert_allclose(pr.conic[j], [c / D, -b / D, a / D], rtol=1e-5)


@pytest.mark.parametrize("mode", [0, 1])
def test_offaxis_isotropic_closed_form(orc, mode):
    check_offaxis_isotropic(orc, mode)


def check_camera_axes(orc):
    """A look-at camera maps its target to the principal point, and offsets
    along its right / down vectors to pure u / v shifts of fx*d/dist."""
    rng = np.random.default_rng(11)
    for _ in range(5):
        eye = rng.uniform(-5, 5, 3)
        tgt = rng.uniform(-1, 1, 3)
        cam = scenes.look_at(eye, tgt, (0.0, 0.0, 1.0), 200, 150, 55.0)
        dist = float(np.linalg.norm(tgt - eye))
        right = cam.R[0].astype(np.float64)
        down = cam.R[1].astype(np.float64)
        pts = [tgt, tgt + 0.2 * right, tgt + 0.2 * down]
        sc = make_scene(pts, [0.01] * 3, [1, 0, 0, 0], 0.5, rgb=(0.5, 0.5, 0.5))
        pr = orc.project(sc, cam, 0)
        assert np.all(pr.radius > 0)
        np.testing.assert_allclose(pr.mean2d[0], [cam.cx, cam.cy], atol=2e-3)
        np.testing.assert_allclose(pr.mean2d[1], [cam.cx + cam.fx * 0.2 / dist, cam.cy], atol=2e-3)
        np.testing.assert_allclose(pr.mean2d[2], [cam.cx, cam.cy + cam.fy * 0.2 / dist], atol=2e-3)
        np.testing.assert_allclose(pr.depth[0], dist, rtol=1e-6)


def test_camera_axes(orc):
    check_camera_axes(orc)


def check_rotated_moments(orc, mode=1):
    """Image moments of one rotated anisotropic Gaussian.

    With opacity o < 0.99 the rendered alpha is o*exp(-sigma) on the region
    sigma <= c = ln(255 o) (and that region lies inside the 3-sigma tile
    rectangle).  The alpha-weighted centroid is the projected mean and the
    alpha-weighted covariance is Sigma2D * E[sigma], E[sigma] =
    (1 - (1+c) e^-c) / (1 - e^-c) for sigma ~ Exp(1) truncated at c.
    Sigma2D = (f/z)^2 Rz diag(s1^2, s2^2) Rz^T + 0.3 I for a rotation by theta
    about the optical axis: the ellipse's major axis points along
    (cos theta, sin theta) in (right, down) image coordinates.
    """
    cam = axis_camera(256, 256, 60.0)
    th, z, s1, s2, o = 0.6, 6.0, 0.3, 0.1, 0.3
    q = [math.cos(th / 2), 0.0, 0.0, math.sin(th / 2)]
    sc = make_scene([[0.0, 0.0, z]], [s1, s2, 0.1], q, o, rgb=(1.0, 0.5, 0.5))
    pr = orc.project(sc, cam, mode)
    vis = orc.visible(pr.tiles)
    rn = orc.render(vis, pr, cam)
    a = rn.img[0] / pr.rgb[0, 0]
    xs, ys = pixel_grid(cam)
    wsum = a.sum()
    mu = np.array([(a * xs).sum() / wsum, (a * ys).sum() / wsum])
    dx, dy = xs - mu[0], ys - mu[1]
    M = np.array([[(a * dx * dx).sum(), (a * dx * dy).sum()], [(a * dx * dy).sum(), (a * dy * dy).sum()]]) / wsum
    c = math.log(255 * o)
    Es = (1 - (1 + c) * math.exp(-c)) / (1 - math.exp(-c))
    f = cam.fx / z
    Rz = np.array([[math.cos(th), -math.sin(th)], [math.sin(th), math.cos(th)]])
    S2 = f * f * Rz @ np.diag([s1 * s1, s2 * s2]) @ Rz.T + 0.3 * np.eye(2)
    np.testing.assert_allclose(mu, [cam.cx, cam.cy], atol=1e-3)
    np.testing.assert_allclose(M, S2 * Es, rtol=1.5e-2, atol=0.02 * np.abs(S2 * Es).max())


def test_rotated_anisotropic_moments(orc):
    check_rotated_moments(orc, 1)
    check_rotated_moments(orc, 0)


def test_culling(orc):
    cam = axis_camera(64, 64, 60.0)
    sc = make_scene([[0.0, 0.0, -1.0], [0.0, 0.0, 0.1], [40.0, 0.0, 2.0], [0.1, 0.1, 3.0]],
                    [0.05] * 3, [1, 0, 0, 0], 0.5, rgb=(0.5, 0.5, 0.5))
    for mode in (0, 1):
        pr = orc.project(sc, cam, mode)
        assert list(pr.radius[:3]) == [0, 0, 0] and list(pr.tiles[:3]) == [0, 0, 0]
        assert pr.radius[3] > 0
        assert list(orc.visible(pr.tiles)) == [3]


def test_visible_matches_nonzero(orc):
    rng = np.random.default_rng(3)
    for dt in (np.uint8, np.uint32):
        a = (rng.random(5000) < 0.3).astype(dt) * rng.integers(1, 5, 5000).astype(dt)
        np.testing.assert_array_equal(orc.visible(a), np.flatnonzero(a))
    assert orc.visible(np.zeros(10, np.uint32)).size == 0


def test_sorted_pairs_brute_force(orc):
    w = scenes.tiny(n=300)
    cam = w.cameras[0]
    pr = orc.project(w.scene, cam, 0)
    vis = orc.visible(pr.tiles)
    keys, vals, ranges = orc.sorted_pairs(vis, pr, cam)
    pairs = []
    for j in vis:
        x0, y0, x1, y1 = pr.rect[j]
        for ty in range(y0, y1):
            for tx in range(x0, x1):
                db = int(np.float32(pr.depth[j]).view(np.uint32))
                pairs.append(((ty * cam.tiles_x + tx) << 32 | db, int(j)))
    pairs.sort()
    assert [p[0] for p in pairs] == [int(k) for k in keys]
    assert [p[1] for p in pairs] == [int(v) for v in vals]
    for t in range(cam.num_tiles):
        sel = [i for i, p in enumerate(pairs) if p[0] >> 32 == t]
        if sel:
            assert ranges[t, 0] == sel[0] and ranges[t, 1] == sel[-1] + 1
        else:
            assert ranges[t, 0] == ranges[t, 1]


def test_render_invariants(orc):
    w = scenes.tiny()
    cam = w.cameras[0]
    pr = orc.project(w.scene, cam, 0)
    vis = orc.visible(pr.tiles)
    keys, vals, ranges = orc.sorted_pairs(vis, pr, cam)
    rn = orc.render(vis, pr, cam)
    assert rn.T_final.min() >= 1e-4 and rn.T_final.max() <= 1.0
    maxc = pr.rgb[vis].max(axis=0)
    for ch in range(3):
        assert np.all(rn.img[ch] <= maxc[ch] * (1 - rn.T_final) + 1e-12)
    ty, tx = np.meshgrid(np.arange(cam.height) // 16, np.arange(cam.width) // 16, indexing="ij")
    t = ty * cam.tiles_x + tx
    L = (ranges[:, 1] - ranges[:, 0])[t]
    assert np.all(rn.n_contrib <= L) and np.all(rn.n_hits <= rn.n_contrib)
    assert np.all(rn.active[rn.active > 0] <= (pr.tiles > 0)[rn.active > 0])
    assert set(np.flatnonzero(rn.active)) <= set(vis)
    # every included pixel has one hit at least where n_contrib > 0
    assert np.all((rn.n_contrib > 0) == (rn.n_hits > 0))


def test_fp32_geometry_agrees_with_fp64(orc):
    for w in (scenes.tiny(), scenes.ring(n=20000)):
        for cam in w.cameras[:3]:
            p32 = orc.project(w.scene, cam, 0)
            p64 = orc.project(w.scene, cam, 1)
            both = (p32.radius > 0) & (p64.radius > 0)
            assert ((p32.radius > 0) != (p64.radius > 0)).sum() <= max(2, 1e-4 * w.scene.n)
            np.testing.assert_allclose(p32.mean2d[both], p64.mean2d[both], rtol=1e-6, atol=1e-3)
            scale = np.abs(p64.conic[both]).max(axis=1, keepdims=True)
            np.testing.assert_allclose(p32.conic[both], p64.conic[both], atol=1e-4 * scale.max(), rtol=1e-4)
            diff = (p32.rect[both] != p64.rect[both]).any(axis=1) | (p32.radius[both] != p64.radius[both])
            assert diff.sum() <= max(2, 2e-4 * both.sum())
            np.testing.assert_allclose(p32.depth[both], p64.depth[both], rtol=1e-6)


# ---------------------------------------------------------------------------
# gradients: central finite differences of the fp64 forward
# ---------------------------------------------------------------------------

def _forward_loss(orc, sc, cam, wimg):
    pr = orc.project(sc, cam, 1)
    vis = orc.visible(pr.tiles)
    rn = orc.render(vis, pr, cam)
    # the decision signature: culling, rectangles, colour clamps, which pairs
    # each pixel includes and which of them sit at the 0.99 cap
    sig = (tuple(pr.radius), tuple(map(tuple, pr.rect)), tuple(pr.clamp), rn.n_contrib.tobytes(), rn.n_hits.tobytes(),
           rn.capped_sig.tobytes())
    return float((rn.img * wimg).sum()), sig


def check_fd_gradients(orc, seed=0, n=6, deg=3, W=40, H=32, tol=1e-5):
    rng = np.random.default_rng(seed)
    cam = axis_camera(W, H, 60.0)
    sc = scenes.random_scene(seed, n, deg, extent=0.5, ls_mu=-2.3, ls_sd=0.3, depth=3.0)
    sc.opacity[:] = np.clip(sc.opacity, -2.0, 2.0)    # stay clear of the 0.99 cap
    wimg = rng.standard_normal((3, H, W))
    return fd_check(orc, sc, cam, wimg, tol)


def fd_check(orc, sc, cam, wimg, tol=1e-5):
    """Every parameter's analytic gradient of sum(wimg * img) against a central
    finite difference of the fp64 forward, skipping elements whose +-h steps
    change the decision signature.  Returns the number of elements checked."""
    n = sc.n
    pr = orc.project(sc, cam, 1)
    vis = orc.visible(pr.tiles)
    g2, _ = orc.render_backward(vis, pr, cam, wimg)
    gr = orc.project_backward(sc, cam, vis, g2, pr)
    names = ["mean", "log_scale", "quat", "opacity", "sh"]
    an_groups = dict(zip(names, gr.full(n)))
    base_loss, base_sig = _forward_loss(orc, sc, cam, wimg)
    checked = skipped = 0
    for name in names:
        arr = getattr(sc, name)
        flat = arr.reshape(n, -1)
        an = an_groups[name]
        for j in range(n):
            for c in range(flat.shape[1]):
                x0 = float(flat[j, c])
                h = 1e-4 * max(1.0, abs(x0))
                vals, steps = [], []
                ok = True
                for sgn in (+1, -1):
                    # the forward reads fp32 parameters: use the fp32-rounded step
                    sc2, xs = _perturbed(sc, name, j, c, sgn * h)
                    L, sig = _forward_loss(orc, sc2, cam, wimg)
                    ok &= (sig == base_sig)
                    vals.append(L); steps.append(xs - x0)
                if not ok:
                    skipped += 1
                    continue
                fd = (vals[0] - vals[1]) / (steps[0] - steps[1])
                ref = an[j, c]
                scale = max(abs(fd), abs(ref), 1e-7 * np.abs(an).max())
                assert abs(fd - ref) <= tol * scale, (name, j, c, fd, ref)
                checked += 1
    assert checked > 0.8 * (checked + skipped), (checked, skipped)
    return checked


def _perturbed(sc, name, j, c, h):
    arr = getattr(sc, name).copy()
    flat = arr.reshape(sc.n, -1)
    flat[j, c] = np.float32(float(flat[j, c]) + h)
    kw = {k: getattr(sc, k) for k in ("mean", "log_scale", "quat", "opacity", "sh")}
    kw[name] = arr
    return scenes.Scene(sh_degree=sc.sh_degree, **kw), float(flat[j, c])


def test_fd_gradients(orc):
    # steps of 1e-4 relative: truncation error O(h^2) ~ 1e-8 relative
    assert check_fd_gradients(orc, seed=0) > 50
    assert check_fd_gradients(orc, seed=1, n=4, deg=1) > 20


def cap_clamp_scene():
    """Three wide Gaussians at degree 1 in front of a 64x64 camera: two with
    opacity logits 6 and 7.5 (o = 0.9975, 0.99945) whose cores reach the 0.99
    cap, one at logit 0.5; the first also has a red channel whose SH sum is
    negative (clamped).  Cores are >= 15 px apart, so no pixel holds two
    capped pairs (their product would sit on the 1e-4 termination threshold)."""
    rng = np.random.default_rng(21)
    cam = axis_camera(64, 64, 60.0)
    means = np.array([[-0.75, -0.45, 3.0], [0.8, 0.35, 3.3], [0.1, 0.7, 3.8]])
    ls = np.log(np.array([[0.5, 0.65, 0.55], [0.6, 0.5, 0.45], [0.4, 0.55, 0.5]]))
    q = rng.standard_normal((3, 4))
    q /= np.linalg.norm(q, axis=1, keepdims=True)
    logit = np.array([6.0, 7.5, 0.5])
    sh = np.zeros((3, 4, 3))
    sh[:, 0, :] = rng.uniform(0.2, 0.8, (3, 3))
    sh[:, 1:, :] = rng.normal(0.0, 0.05, (3, 3, 3))
    sh[0, 0, 0] = (-0.35 - 0.5) * SQRT_PI2          # red SH sum about -0.35 (clamped)
    sc = scenes.Scene(mean=means.astype(np.float32), log_scale=ls.astype(np.float32),
                      quat=q.astype(np.float32), opacity=logit.astype(np.float32), sh=sh.astype(np.float32),
                      sh_degree=1)
    wimg = rng.standard_normal((3, cam.height, cam.width))
    return sc, cam, wimg


def check_fd_cap_clamp(orc):
    """Finite differences on a scene with capped pairs and a clamped channel:
    no derivative flows through a capped pair (w.r.t. opacity and sigma) nor
    through a clamped colour channel (w.r.t. its SH and the view direction)."""
    sc, cam, wimg = cap_clamp_scene()
    pr = orc.project(sc, cam, 1)
    assert pr.clamp[0] & 1 and pr.rgb[0, 0] == 0.0
    rn = orc.render(orc.visible(pr.tiles), pr, cam)
    assert (rn.capped_sig > 0).sum() >= 6, (rn.capped_sig > 0).sum()
    return fd_check(orc, sc, cam, wimg)


def test_fd_gradients_at_cap_and_clamp(orc):
    assert check_fd_cap_clamp(orc) > 50


def check_grad_norm_fd(orc):
    """g(p) = ||dL/d(u, v)||_2: finite differences of the render w.r.t. each
    visible primitive's pixel mean (rectangles and candidate lists held
    fixed), compared with the 2D gradient and with grad_norm."""
    sc, cam, wimg = cap_clamp_scene()
    pr = orc.project(sc, cam, 1)
    vis = orc.visible(pr.tiles)
    g2, _ = orc.render_backward(vis, pr, cam, wimg)
    gr = orc.project_backward(sc, cam, vis, g2, pr)

    def loss_sig(p):
        rn = orc.render(vis, p, cam)
        return float((rn.img * wimg).sum()), (rn.n_contrib.tobytes(), rn.n_hits.tobytes(), rn.capped_sig.tobytes())

    _, base_sig = loss_sig(pr)
    for row, j in enumerate(vis):
        fd = []
        for c in range(2):
            h = 1e-5
            vals = []
            for sgn in (+1, -1):
                p2 = dataclasses.replace(pr, mean2d=pr.mean2d.copy())
                p2.mean2d[j, c] += sgn * h
                L, sig = loss_sig(p2)
                assert sig == base_sig
                vals.append(L)
            fd.append((vals[0] - vals[1]) / (2 * h))
        np.testing.assert_allclose(g2[j, :2], fd, rtol=1e-6, atol=1e-9 * np.abs(fd).max())
        assert abs(gr.grad_norm[row] - math.hypot(*fd)) <= 1e-6 * math.hypot(*fd), (row, gr.grad_norm[row], fd)
    return vis.size


def test_grad_norm_is_l2_of_uv_gradient(orc):
    assert check_grad_norm_fd(orc) == 3


# ---------------------------------------------------------------------------
# loss, Adam, pack/apply against library routines / identities
# ---------------------------------------------------------------------------

def test_l1_matches_torch(orc):
    import torch
    rng = np.random.default_rng(0)
    img = rng.random((3, 17, 23)).astype(np.float32)
    tgt = rng.random((3, 17, 23)).astype(np.float32)
    tgt[0, 0, :5] = img[0, 0, :5]          # exact ties: sign(0) = 0
    loss, g, _ = orc.loss_l1(img, tgt)
    ti = torch.tensor(img.astype(np.float64), requires_grad=True)
    tl = torch.nn.functional.l1_loss(ti, torch.tensor(tgt.astype(np.float64)))
    tl.backward()
    assert abs(loss - tl.item()) < 1e-14
    np.testing.assert_allclose(g, ti.grad.numpy(), rtol=1e-7)
    assert np.all(g[0, 0, :5] == 0)


def check_adam_vs_torch(orc, steps=4):
    import torch
    rng = np.random.default_rng(1)
    n, cols = 50, 7
    p0 = rng.standard_normal((n, cols))
    rows = np.sort(rng.choice(n, 20, replace=False))
    lr, b1, b2, eps = 1e-2, 0.9, 0.999, 1e-15
    # full set: torch on all rows
    tp = torch.tensor(p0.copy(), requires_grad=True)
    opt = torch.optim.Adam([tp], lr=lr, betas=(b1, b2), eps=eps, foreach=False)
    p, m, v = p0.copy(), np.zeros_like(p0), np.zeros_like(p0)
    for t in range(1, steps + 1):
        g = rng.standard_normal((n, cols))
        opt.zero_grad(); tp.grad = torch.tensor(g); opt.step()
        p, m, v, _ = orc.adam(p, g, m, v, np.arange(n), t, lr, b1, b2, eps)
    np.testing.assert_allclose(p, tp.detach().numpy(), rtol=1e-12, atol=1e-14)
    # subset: torch sees only the visible rows; the rest must stay bit-identical
    ts = torch.tensor(p0[rows].copy(), requires_grad=True)
    opt = torch.optim.Adam([ts], lr=lr, betas=(b1, b2), eps=eps, foreach=False)
    p, m, v = p0.copy(), np.zeros_like(p0), np.zeros_like(p0)
    for t in range(1, steps + 1):
        g = rng.standard_normal((n, cols))
        opt.zero_grad(); ts.grad = torch.tensor(g[rows]); opt.step()
        p, m, v, d = orc.adam(p, g, m, v, rows, t, lr, b1, b2, eps)
    np.testing.assert_allclose(p[rows], ts.detach().numpy(), rtol=1e-12, atol=1e-14)
    rest = np.setdiff1d(np.arange(n), rows)
    assert np.array_equal(p[rest], p0[rest])


def test_adam_matches_torch(orc):
    check_adam_vs_torch(orc)


def test_pack_apply_roundtrip(orc):
    rng = np.random.default_rng(2)
    n = 100
    groups = [rng.standard_normal((n, c)).astype(np.float32) for c in (3, 3, 4, 1, 48)]
    idx = np.sort(rng.choice(n, 37, replace=False)).astype(np.uint32)
    msg = orc.delta_pack(idx, groups, version=9)
    assert msg[1] == 37 and msg[2] == 9 and msg[3] == 59
    tgt = [np.zeros_like(g) for g in groups]
    out, ver = orc.delta_apply(msg, tgt, "overwrite", np.zeros(n, np.uint32))
    for a, g in zip(out, groups):
        assert np.array_equal(a[idx], g[idx])
        rest = np.setdiff1d(np.arange(n), idx)
        assert np.all(a[rest] == 0)
    assert np.all(ver[idx] == 9) and ver.sum() == 9 * idx.size
    base = [rng.standard_normal((n, c)).astype(np.float32) for c in (3, 3, 4, 1, 48)]
    out, _ = orc.delta_apply(msg, base, "add")
    for a, b, g in zip(out, base, groups):
        assert np.array_equal(a[idx], b[idx] + g[idx])
    empty = orc.delta_pack(np.zeros(0, np.uint32), groups, version=1)
    out, _ = orc.delta_apply(empty, base, "add")
    assert all(np.array_equal(a, b) for a, b in zip(out, base))


# ---------------------------------------------------------------------------
# the pins above catch plausible mistakes planted in the oracle
# ---------------------------------------------------------------------------

MUTATIONS = {
    1: lambda o: check_single_gaussian(o, 0),        # dilation dropped
    2: lambda o: check_offaxis_isotropic(o, 0),      # sign of the J02 term
    3: lambda o: check_camera_axes(o),               # camera rotation transposed
    4: lambda o: check_rotated_moments(o, 0),        # sign of the conic cross term in sigma
    5: lambda o: check_fd_gradients(o, seed=0),      # dC/dalpha without 1/(1-alpha)
    6: lambda o: check_sh_vs_scipy(o),               # sign of one SH basis function
    7: lambda o: check_adam_vs_torch(o),             # Adam without bias correction
    22: lambda o: check_capped_closed_form(o, 1),    # alpha cap at 0.999 instead of 0.99
    23: lambda o: check_clamped_colour(o, 1),        # colour clamp max(0, .) dropped
    24: lambda o: check_capped_backward(o),          # derivative passed through capped pairs
    25: lambda o: check_grad_norm_fd(o),             # grad_norm as |du| + |dv| instead of the 2-norm
    26: lambda o: check_fd_cap_clamp(o),             # colour gradient through a clamped channel
}
# the finite-difference scene catches the capped-pair mistake on its own too
FD_ALSO = {24: check_fd_cap_clamp}


@pytest.mark.parametrize("k", sorted(MUTATIONS))
def test_planted_mistake_is_caught(orc, k):
    orc.set_mutation(k)
    try:
        with pytest.raises(AssertionError):
            MUTATIONS[k](orc)
        if k in FD_ALSO:
            with pytest.raises(AssertionError):
                FD_ALSO[k](orc)
    finally:
        orc.set_mutation(0)
