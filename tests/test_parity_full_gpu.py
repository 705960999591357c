"""End-to-end parity of one training view at the five full workload sizes
against the CPU oracle on the same seeded inputs, with the pool stored in
the spatial order the benchmark uses.

Two passes over views 0, 1 and the last of each workload (tiny has one
view), each from the same initial pool and Adam state:

  1. every visible primitive's gradient: projection, visible set, bin sort,
     the fused forward + L1, then the backward with the oracle's upstream
     gradient, zeroed at the pixels whose threshold decisions lie within the
     oracle's bands (a pixel's decisions reach the gradients only through
     its own upstream gradient);
  2. the benchmark's training step itself (ViewTrainer.step with the
     overlapped commit, exactly as bench.py times it): visible set, pairs and
     ranges bit-exact, the realized active set equal to pass 1's, image, dL/dimg bit-exact against the sign of the GPU
     image's difference from the target, the step's gradient rows against the
     oracle's backward of that same dL/dimg on every visible primitive whose
     inclusion in no pixel lies within a decision band (the bound of each
     element widened by twice the magnitude that the ambiguous pixels' own
     terms reach it with; the primitives left out, at most 1% of the rows,
     were checked in pass 1), the Adam steps staged as the version-1 message,
     the parameters, and the replica the overlapped commit wrote.

The first Adam step (t = 1, zero moments, eps = 1e-15) gives
delta = -lr * g / (|g| + eps): elements whose oracle gradient is above the
gradient floor must match to the 2e-3 bar; elements below it may carry
either sign of lr (their gradient is at the fp32 noise level of the
backward), so they are checked for |delta_gpu - delta_oracle| <= 2 lr.
"""
import sys
import time

import numpy as np
import pytest

from parity_util import AMB_SHARE, GRAD_RTOL, assert_grads, assert_pixels, expected_tile_order, grad_floor
from parity_util import target_of

pytestmark = [pytest.mark.gpu, pytest.mark.slow]


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


WORKLOADS = ["tiny", "ring", "room", "spiral", "aerial"]
# views checked per workload: the first two and the last (tiny has one camera);
# each starts from the same initial pool and Adam state
VIEWS = {"tiny": (0,), "ring": (0, 1, -1), "room": (0, 1, -1), "spiral": (0, 1, -1), "aerial": (0, 1, -1)}
CASES = [(name, v) for name in WORKLOADS for v in VIEWS[name]]


def _group_rows(tr, V):
    return tr.rows_by_group(tr.grad_rows, V)


_WORKLOAD_CACHE = {}


def _workload(name):
    """The workload in the bench's storage order, built once per test session."""
    from paper_2607_19893_amd import scenes
    if name not in _WORKLOAD_CACHE:
        _WORKLOAD_CACHE.clear()
        _WORKLOAD_CACHE[name] = scenes.spatially_ordered(scenes.workload(name))
    return _WORKLOAD_CACHE[name]


@pytest.mark.timeout(1100)
@pytest.mark.parametrize("name,view", CASES)
def test_full_view(name, view, orc):
    import torch
    from paper_2607_19893_amd.pipeline import ViewTrainer, to_u32
    assert torch.cuda.is_available()
    t0 = time.time()
    w = _workload(name)                                      # the pool in the bench's storage order
    view = view % len(w.cameras)
    cam = w.cameras[view]
    n = w.scene.n
    H, W = cam.height, cam.width
    _say(name, "view %d, n=%d (workload ready in %.1fs)" % (view, n, time.time() - t0))
    tr = ViewTrainer(w.scene, capacity=1, max_width=W, max_height=H, lr=w.lr, with_keys=True)
    tr.ensure_capacity([cam])
    tgt = target_of(w, view)
    tr.set_target(tgt)

    # oracle: projection, visible set, pairs, render, and the ambiguous pixels
    t0 = time.time()
    pr = orc.project(w.scene, cam, 0)
    vis_o = orc.visible(pr.tiles)
    keys_o, vals_o, ranges_o = orc.sorted_pairs(vis_o, pr, cam)
    rn = orc.render(vis_o, pr, cam)
    amb = orc.ambiguous_pixels(rn)
    _say(name, "oracle forward in %.1fs; ambiguous pixels %d of %d" % (time.time() - t0, int(amb.sum()), amb.size))
    assert amb.mean() <= AMB_SHARE

    # ---- 1. every visible primitive's gradient, with the ambiguous pixels' dL zeroed
    tr.status.zero_()
    tr.project(cam); tr.visible(); tr.bin_sort(); tr.raster_fwd_l1(active=True)
    torch.cuda.synchronize()
    assert to_u32(tr.status)[0] == 0
    _, dL_o, _ = orc.loss_l1(rn.img.astype(np.float32), tgt)
    dLm = np.where(amb[None], 0.0, dL_o).astype(np.float32)
    tr.set_dL(dLm)
    tr.raster_bwd(grad2d=True)
    torch.cuda.synchronize()
    V = int(to_u32(tr.counts[0:1])[0])
    vis = to_u32(tr.vis_idx)[:V].copy()
    np.testing.assert_array_equal(vis, vis_o)
    act = tr.active.cpu().numpy()[:n].copy()
    t0 = time.time()
    g2m, flagm, gabs = orc.render_backward(vis_o, pr, cam, dLm.astype(np.float64), want_abs=True)
    grm = orc.project_backward(w.scene, cam, vis_o, g2m, pr)
    mags, mag_norm = orc.gradient_magnitudes(w.scene, cam, vis_o, gabs, pr)
    _say(name, "oracle backward in %.1fs" % (time.time() - t0))
    # the realized active set: a flag may differ only where an ambiguous pixel looked
    diff = np.flatnonzero(act != rn.active)
    assert np.all(flagm[diff] & orc.FLAG_AMB_PIXEL), diff[:10]
    ok_rows = ((flagm[vis] & orc.FLAG_NEAR_CAP) == 0) & (pr.clamp_margin[vis] > 1e-5) & (pr.jclamp_margin[vis] > 1e-5)
    _say(name, "dL zeroed at %d pixels; gradient rows checked %d of %d" % (int(amb.sum()), int(ok_rows.sum()), V))
    assert ok_rows.mean() > 0.999
    for gname, gp, go, mg in zip(["mean", "log_scale", "quat", "opacity", "sh"], _group_rows(tr, V), grm.groups(),
                                 mags):
        st = assert_grads(gp, go, ok_rows, "grad." + gname, mag=mg)
        _say(name, gname, st)
    st = assert_grads(tr.grad_norm.cpu().numpy()[vis.astype(np.int64)], grm.grad_norm, ok_rows, "grad_norm",
                      mag=mag_norm)
    _say(name, "grad_norm", st)

    # ---- 2. the benchmark's step: fused forward + L1, split backward, Adam staged
    # as version 1 in ring slot 1, its commit on the second stream
    tr.status.zero_()
    tr.step(cam, step=1, version=1, overlap=True)
    tr.flush_apply()
    torch.cuda.synchronize()
    assert to_u32(tr.status)[0] == 0
    assert int(to_u32(tr.ring_state)[0]) == 1
    assert int(to_u32(tr.counts[0:1])[0]) == V
    np.testing.assert_array_equal(to_u32(tr.vis_idx)[:V], vis_o)
    M = int(to_u32(tr.counts[1:2])[0])
    assert M == keys_o.size
    np.testing.assert_array_equal(tr.keys.cpu().numpy()[:M].view(np.uint64), keys_o)
    np.testing.assert_array_equal(to_u32(tr.vals)[:M], vals_o)
    T = cam.num_tiles
    np.testing.assert_array_equal(to_u32(tr.ranges)[:2 * T].reshape(T, 2), ranges_o)
    np.testing.assert_array_equal(to_u32(tr.tile_order)[:T], expected_tile_order(ranges_o))
    _say(name, "V=%d M=%d bit-exact" % (V, M))
    # the realized active set: the ids of the flags the forward of pass 1 set, in
    # ascending order; the step's compaction leaves every flag cleared
    A = int(to_u32(tr.counts[2:3])[0])
    np.testing.assert_array_equal(to_u32(tr.act_idx)[:A], np.flatnonzero(act))
    assert int(tr.active[:n].max()) == 0
    _say(name, "realized active set %d of %d visible" % (A, V))
    img = tr.img.view(-1)[:3 * H * W].cpu().numpy().reshape(3, H, W)
    assert_pixels(img, rn.img, np.broadcast_to(~amb, img.shape), "img")
    fT = tr.final_T.view(-1)[:H * W].cpu().numpy().reshape(H, W)
    assert_pixels(fT, rn.T_final, ~amb, "final_T")
    nc = to_u32(tr.n_contrib)[:H * W].reshape(H, W)
    np.testing.assert_array_equal(nc[~amb], rn.n_contrib[~amb])
    # the loss gradient: the sign of the GPU image's difference from the target, bit for bit
    loss_g, dL_g, _ = orc.loss_l1(img, tgt)
    dL = tr.dL.view(-1)[:3 * H * W].cpu().numpy().reshape(3, H, W)
    np.testing.assert_array_equal(dL, dL_g.astype(np.float32))
    assert abs(tr.loss.item() - loss_g) <= 1e-6 * loss_g
    loss_o, _, _ = orc.loss_l1(rn.img.astype(np.float32), tgt)
    assert abs(loss_g - loss_o) <= 1e-5 * loss_o
    # the step's gradient rows against the oracle's backward of the same dL/dimg;
    # an ambiguous pixel's terms may differ on the two sides (its decisions
    # may go either way), so each element's bound takes twice the magnitude
    # of the terms those pixels contribute to it (their sum of |terms| carried
    # through the chain rule), the larger of that magnitude in the oracle's own
    # pass and in the pass that takes the other outcome of each banded decision
    # (which also holds the pairs the oracle left out there)
    t0 = time.time()
    g2, flag, gabs = orc.render_backward(vis_o, pr, cam, dL_g, want_abs=True)
    gr = orc.project_backward(w.scene, cam, vis_o, g2, pr)
    mags, _ = orc.gradient_magnitudes(w.scene, cam, vis_o, gabs, pr)
    dL_amb = np.where(amb[None], dL_g, 0.0)
    _, _, gabs_amb = orc.render_backward(vis_o, pr, cam, dL_amb, want_abs=True)
    mags_amb, _ = orc.gradient_magnitudes(w.scene, cam, vis_o, gabs_amb, pr)
    _, _, gabs_alt = orc.render_backward(vis_o, pr, cam, dL_amb, want_abs=True, alternative=True)
    mags_alt, _ = orc.gradient_magnitudes(w.scene, cam, vis_o, gabs_alt, pr)
    _say(name, "oracle backward of the step's dL in %.1fs" % (time.time() - t0))
    g_gpu = _group_rows(tr, V)
    grown = sum(int(np.any(mb > ma, axis=1).sum()) for ma, mb in zip(mags_amb, mags_alt))
    _say(name, "rows whose bound the other outcomes widen: %d of %d" % (grown, V))
    for gname, gp, go, mg, ma, mb in zip(["mean", "log_scale", "quat", "opacity", "sh"], g_gpu, gr.groups(), mags,
                                         mags_amb, mags_alt):
        st = assert_grads(gp, go, ok_rows, "step grad." + gname, mag=mg, slack=2.0 * np.maximum(ma, mb))
        _say(name, "step", gname, st)
    # the Adam steps are compared where no ambiguous pixel reached the row
    sure_rows = ok_rows & (flag[vis] == 0)
    _say(name, "step rows no ambiguous pixel examined: %d of %d" % (int(sure_rows.sum()), V))
    # the Adam steps, staged as the message of version 1 in ring slot 1
    rows = vis.astype(np.int64)
    p0 = [a.reshape(n, -1) for _, a in w.scene.groups()]
    lr = w.lr
    deltas = [orc.adam_rows(p[rows], g, np.zeros_like(g), np.zeros_like(g), 1, lr)[3] for p, g in zip(p0, gr.groups())]
    msg_o = orc.delta_message(vis_o, [d.astype(np.float32) for d in deltas], 1)
    msg = tr.msgs[1].cpu().numpy().view(np.uint32)
    head = 8 + 8 + V
    np.testing.assert_array_equal(msg[:head], msg_o[:head])
    r0 = (head + 3) // 4 * 4
    rows_gpu = msg[r0:r0 + V * tr.row_len].view(np.float32).reshape(V, tr.row_len)
    offs = np.cumsum([0] + tr.cols)
    for gi, (p, d_orc, g_orc) in enumerate(zip(tr.params, deltas, gr.groups())):
        d_gpu = rows_gpu[:, offs[gi]:offs[gi + 1]].astype(np.float64)
        sure = sure_rows[:, None] & (np.abs(g_orc) > grad_floor(g_orc))
        err = np.abs(d_gpu - d_orc)
        assert np.all(err[sure] <= GRAD_RTOL * lr), (gi, err[sure].max())
        assert np.all(err <= 2 * lr * (1 + GRAD_RTOL)), (gi, err.max())
        # the parameter moved by exactly the staged step (one fp32 add)
        pn = p.cpu().numpy()[rows]
        np.testing.assert_array_equal(pn, (p0[gi][rows] + rows_gpu[:, offs[gi]:offs[gi + 1]]).astype(np.float32))
    # the replica received exactly the published rows (one fp32 add each) from the overlapped commit
    for r, gi in zip(tr.replica, range(5)):
        np.testing.assert_array_equal(r.cpu().numpy()[rows],
                                      (p0[gi][rows] + rows_gpu[:, offs[gi]:offs[gi + 1]]).astype(np.float32))
    assert np.all(to_u32(tr.version)[rows] == 1)
    untouched = np.setdiff1d(np.arange(n), rows)[:100000]
    for r, gi in zip(tr.replica, range(5)):
        np.testing.assert_array_equal(r.cpu().numpy()[untouched], p0[gi][untouched])
    _say(name, "ok")
