"""GPU parity of a task unit of two views (Section 2.1: a small batch of
views whose gradients and evidence accumulate over the union of their scopes,
then one optimizer step): union of the visible sets bit-exact, the summed
gradient rows and accumulated |dL/d(u,v)| within the gradient bar, the Adam
step over the union and its message; small workloads with ragged image sides
and the full room workload (1M primitives, 1920x1080)."""
import sys

import numpy as np
import pytest

from parity_util import GRAD_RTOL, assert_grads, grad_floor
from parity_util import target_of

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def u32(t):
    return t.detach().cpu().numpy().view(np.uint32)


def workloads():
    from paper_2607_19893_amd import scenes
    return {
        "room-60k-392x216": lambda: scenes.room(n=60000, width=392, height=216),
        "ring-20k-328x184": lambda: scenes.ring(n=20000, width=328, height=184),
        "room-1M-1920x1080": lambda: scenes.workload("room"),
    }


@pytest.mark.parametrize("case", list(workloads().keys()))
def test_unit_of_two_views(case, orc):
    import torch
    from paper_2607_19893_amd import scenes
    from paper_2607_19893_amd.pipeline import ViewTrainer
    assert torch.cuda.is_available()
    w = workloads()[case]()
    cams = w.cameras[:2]
    n = w.scene.n
    tr = ViewTrainer(w.scene, capacity=1, max_width=max(c.width for c in cams),
                     max_height=max(c.height for c in cams), lr=w.lr)
    tr.ensure_capacity(cams)
    # upstream gradients with each view's ambiguous pixels zeroed (decided by the oracle)
    dLm, vis_o = [], []
    for k, cam in enumerate(cams):
        dL = scenes.make_upstream_grad(cam.width, cam.height, 17 + k)
        pr = orc.project(w.scene, cam, 0)
        vis = orc.visible(pr.tiles)
        rn = orc.render(vis, pr, cam)
        amb = orc.ambiguous_pixels(rn)
        dLm.append(np.where(amb[None], 0.0, dL).astype(np.float32).astype(np.float64))
        vis_o.append(vis)
    tr.status.zero_()
    tr.unit_scopes(cams)
    for k, cam in enumerate(cams):
        tr.unit_view_backward(k, cam, dL=dLm[k].astype(np.float32))
    torch.cuda.synchronize()
    assert u32(tr.status)[0] == 0
    # union: bit-exact
    U = int(u32(tr.union_count)[0])
    union = u32(tr.union_idx)[:U].copy()
    np.testing.assert_array_equal(union, np.union1d(vis_o[0], vis_o[1]).astype(np.uint32))
    _say(case, "views see %d and %d primitives, union %d" % (vis_o[0].size, vis_o[1].size, U))
    # summed gradients over union rows
    ref_union, grads, gnorm, views = orc.unit_gradients(w.scene, cams, dL_list=dLm)
    np.testing.assert_array_equal(ref_union, union)
    mags = [np.zeros_like(g) for g in grads]
    mag_norm = np.zeros(n)
    ok = np.ones(U, bool)
    for view, cam in zip(views, cams):
        vis, pr, dL = view[0], view[1], view[3]
        g2, flag2, gabs = orc.render_backward(vis, pr, cam, dL, want_abs=True)
        m, mn = orc.gradient_magnitudes(w.scene, cam, vis, gabs, pr)
        rows = np.searchsorted(union, vis)
        for M, mm in zip(mags, m):
            M[rows] += mm
        mag_norm[vis.astype(np.int64)] += mn
        bad = ((flag2[vis] & orc.FLAG_NEAR_CAP) != 0) | (pr.clamp_margin[vis] <= 1e-5) | (pr.jclamp_margin[vis] <= 1e-5)
        ok[rows[bad]] = False
    _say(case, "union rows outside the element-wise check:", int((~ok).sum()))
    assert (~ok).sum() <= max(5, 1e-3 * U)
    for name, gp, go, mg in zip(["mean", "log_scale", "quat", "opacity", "sh"], tr.rows_by_group(tr.grad_rows, U),
                                grads, mags):
        st = assert_grads(gp, go, ok, "unit grad." + name, mag=mg)
        _say(case, name, st)
    # padding columns stay zero
    if tr.ld > tr.row_len:
        assert float(tr.grad_rows[:U, tr.row_len:].abs().max()) == 0.0
    ui = union.astype(np.int64)
    assert_grads(tr.grad_norm.cpu().numpy()[ui], gnorm[ui], ok, "unit grad_norm", mag=mag_norm[ui])
    # one Adam step over the union, staged as the message of version 1, then committed
    msg = tr.msgs[1]
    from paper_2607_19893_amd import gsmi
    gsmi.gs_sparse_adam_publish(tr.adam_arr, 5, tr.union_idx, tr.union_count[0:1], n, tr.grad_rows, tr.ld, tr.m,
                                tr.v, tr.ld, 1, tr.beta1, tr.beta2, tr.eps, 1, msg, tr.status)
    tr.commit(1)
    torch.cuda.synchronize()
    assert u32(tr.status)[0] == 0
    m0 = [np.zeros((n, c)) for c in tr.cols]
    res = orc.train_unit(w.scene, cams, None, m0, [np.zeros_like(a) for a in m0], 1, lr=w.lr, dL_list=dLm)
    got = u32(msg)
    head = 8 + 8 + U
    np.testing.assert_array_equal(got[:head], res.msg[:head])
    r0 = (head + 3) // 4 * 4
    rows_gpu = got[r0:r0 + U * tr.row_len].view(np.float32).reshape(U, tr.row_len)
    offs = np.cumsum([0] + tr.cols)
    lr = w.lr
    for gi, (d_orc, g_orc) in enumerate(zip(res.deltas, res.grads)):
        d_gpu = rows_gpu[:, offs[gi]:offs[gi + 1]].astype(np.float64)
        sure = ok[:, None] & (np.abs(g_orc) > grad_floor(g_orc))
        err = np.abs(d_gpu - d_orc)
        assert np.all(err[sure] <= GRAD_RTOL * lr), (gi, err[sure].max())
        assert np.all(err <= 2 * lr * (1 + GRAD_RTOL)), (gi, err.max())
    # the replica received the unit's steps; versions name the unit's version on the union
    for p, r in zip(tr.params, tr.replica):
        assert torch.equal(p, r)
    ver = u32(tr.version)
    assert np.all(ver[ui] == 1) and int((ver != 0).sum()) == U


def test_unit_step_end_to_end(orc):
    """step_unit with L1 losses over several consecutive units: statuses stay
    clear, versions advance, the replica tracks the parameters bit for bit."""
    import torch
    from paper_2607_19893_amd import scenes
    from paper_2607_19893_amd.pipeline import ViewTrainer
    w = scenes.room(n=60000, width=392, height=216)
    tr = ViewTrainer(w.scene, capacity=1, max_width=392, max_height=216, lr=w.lr)
    tr.ensure_capacity(w.cameras[:6])
    targets = [torch.from_numpy(target_of(w, i).reshape(-1)).cuda() for i in range(6)]
    for u in range(3):
        tr.step_unit(w.cameras[2 * u:2 * u + 2], step=u + 1, version=u + 1, targets=targets[2 * u:2 * u + 2])
    torch.cuda.synchronize()
    assert u32(tr.status)[0] == 0
    assert u32(tr.ring_state)[0] == 3
    for p, r in zip(tr.params, tr.replica):
        assert torch.equal(p, r)
    assert u32(tr.version).max() == 3
