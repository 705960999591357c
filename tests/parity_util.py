"""Comparison rules shared by the GPU parity tests.

Bars (derivations in the design notes):
  * integers, ids, keys, ranges, messages: bit-exact;
  * rendered pixels: |gpu - oracle| <= 1e-4 * max(|oracle|, PIX_FLOOR);
  * gradients and updated parameters: |gpu - oracle| <= 2e-3 * max(|oracle|, floor)
    + SUM_EPS * M, where M carries the sums of |per-pixel terms| through the
    chain rule (an fp32 sum's rounding error is relative to them) and
    floor = GRAD_FLOOR_FRAC * (99th percentile of |oracle| over the group),
    plus a normwise check ||gpu - oracle|| / ||oracle|| <= 2e-3.  The
    comparison reports how many elements pass only because of the floor or
    only because of the summation term.
Pixels / primitives whose result depends on a threshold decision that the
fp32 kernel may take differently from the fp64 oracle are excluded from the
element-wise check and reported; their share is bounded by AMB_SHARE.
"""
import numpy as np

PIX_RTOL = 1e-4
PIX_FLOOR = 0.05
GRAD_RTOL = 2e-3
GRAD_FLOOR_FRAC = 1e-2
SUM_EPS = 1e-5      # fp32 summation error relative to the summed magnitudes
AMB_SHARE = 1e-4    # largest share of pixels a threshold band may leave out


def assert_pixels(gpu, ref, mask=None, name="img"):
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    err = np.abs(gpu - ref)
    tol = PIX_RTOL * np.maximum(np.abs(ref), PIX_FLOOR)
    bad = err > tol
    if mask is not None:
        bad &= mask
    nbad = int(bad.sum())
    assert nbad == 0, "%s: %d entries beyond 1e-4 relative (max err %.3g at ref %.3g)" % (
        name, nbad, err[bad].max(), ref[bad][np.argmax(err[bad])])
    return float(err[mask].max()) if mask is not None and mask.any() else float(err.max())


def grad_floor(ref):
    a = np.abs(np.asarray(ref, np.float64)).reshape(-1)
    if a.size == 0:
        return 0.0
    return GRAD_FLOOR_FRAC * float(np.quantile(a, 0.99)) + 1e-30


def assert_grads(gpu, ref, rows_ok, name, rtol=GRAD_RTOL, floor=None, mag=None, slack=None):
    """Element-wise on rows_ok (bool per row), normwise on the same rows.
    mag: per-element summed magnitudes (oracle.gradient_magnitudes); adds
    SUM_EPS * mag to the element-wise bound.  slack: a per-element absolute
    allowance added to the bound (the part of the gradient that comes from
    pixels whose decisions may go either way); the normwise check then
    covers the elements whose error stays within the plain bound."""
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    g, r = gpu[rows_ok], ref[rows_ok]
    if r.size == 0:
        return {}
    if floor is None:
        fl = grad_floor(r)
    elif np.ndim(floor) == 0:
        fl = floor
    else:
        fl = np.asarray(floor, np.float64)[rows_ok]
    err = np.abs(g - r)
    tol = rtol * np.maximum(np.abs(r), fl)
    sum_term = SUM_EPS * np.asarray(mag, np.float64)[rows_ok] if mag is not None else 0.0
    tol = tol + sum_term
    plain = err <= tol
    if slack is not None:
        tol = tol + np.asarray(slack, np.float64)[rows_ok]
    bad = err > tol
    inn = plain if slack is not None else np.ones_like(plain)
    nrm = float(np.linalg.norm((g - r)[inn]) / max(np.linalg.norm(r[inn]), 1e-300))
    stats = {"max_rel": float((err / np.maximum(np.abs(r), fl)).max()), "norm_rel": nrm, "bad": int(bad.sum())}
    # how many elements pass only because of the floor, only because of the summation term
    stats["need_floor"] = int(((err > rtol * np.abs(r) + sum_term) & ~bad).sum())
    stats["need_sum_term"] = int(((err > rtol * np.maximum(np.abs(r), fl)) & plain).sum())
    stats["need_slack"] = int((~plain & ~bad).sum())
    stats["n"] = int(err.size)
    assert bad.sum() == 0, "%s: %d elements beyond %.0e relative (floor %.3g): worst err %.3g ref %.3g" % (
        name, int(bad.sum()), rtol, float(np.max(fl)), err[bad].max(), r[bad][np.argmax(err[bad])])
    assert nrm <= rtol, "%s: normwise error %.3g" % (name, nrm)
    return stats


def order_code(n):
    """The dispatch code of a tile's pair count that gs_bin_sort documents:
    the count itself below 16, then 16 steps per octave, 255 from 2^19 on."""
    n = int(n)
    if n < 16:
        return n
    e = n.bit_length() - 1
    return 255 if e > 18 else 16 * (e - 3) + ((n >> (e - 4)) & 15)


def expected_tile_order(ranges):
    """Tile ids by dispatch code descending, equal codes by ascending id."""
    ranges = np.asarray(ranges, np.int64).reshape(-1, 2)
    codes = np.array([order_code(e - s) for s, e in ranges], np.int64)
    return np.lexsort((np.arange(codes.size), -codes)).astype(np.uint32)


def oracle_render(scene, cam):
    """The oracle's image of a scene from a camera (fp32), for targets that are
    renders of a workload's perturbed copy."""
    import oracle as orc
    pr = orc.project(scene, cam, 0)
    return orc.render(orc.visible(pr.tiles), pr, cam).img.astype(np.float32)


def target_of(w, view):
    """A workload's target image for a view, renders made by the oracle."""
    return w.target(view, render=oracle_render)
