"""GPU parity: every C-ABI entry point against the CPU oracle on the same
seeded inputs (run on an MI355X; `-m gpu`).

Small cases span several tiles and ragged tails (image sides that are not
multiples of 16); the full-size cases are the five workloads in the exact
launch configuration the benchmark times.
"""
import sys

import numpy as np
import pytest

from parity_util import AMB_SHARE, assert_grads, assert_pixels, expected_tile_order
from parity_util import target_of

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def torch_gpu():
    import torch
    assert torch.cuda.is_available(), "GPU parity tests need an MI355X"
    return torch


def small_cases():
    from paper_2607_19893_amd import scenes
    return {
        "tiny-10k-256": lambda: scenes.tiny(),
        "ring-20k-328x184": lambda: scenes.ring(n=20000, width=328, height=184),
        "room-60k-392x216": lambda: scenes.room(n=60000, width=392, height=216),
    }


CASES = list(small_cases().keys())
_CACHE = {}


def get_case(name):
    if name not in _CACHE:
        _CACHE[name] = small_cases()[name]()
    return _CACHE[name]


def trainer_for(w, torch_gpu, capacity=None, packed=True):
    from paper_2607_19893_amd.pipeline import ViewTrainer
    tr = ViewTrainer(w.scene, capacity=capacity or 1, max_width=max(c.width for c in w.cameras),
                     max_height=max(c.height for c in w.cameras), with_keys=True, packed=packed)
    if capacity is None:
        tr.ensure_capacity(w.cameras[:2])
    return tr


def u32(t):
    from paper_2607_19893_amd.pipeline import to_u32
    return to_u32(t)


# ---------------------------------------------------------------------------
# stage by stage
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("case", CASES)
def test_project_visible_sort(case, torch_gpu, orc):
    w = get_case(case)
    _say("case", case, "n", w.scene.n)
    tr = trainer_for(w, torch_gpu)
    for vi, cam in enumerate(w.cameras[:2]):
        tr.status.zero_()
        tr.project(cam)
        tr.visible()
        tr.bin_sort()
        torch_gpu.cuda.synchronize()
        assert u32(tr.status)[0] == 0
        ref = orc.project(w.scene, cam, 0)
        n = w.scene.n
        rad = tr.radius.cpu().numpy()[:n]
        tiles = u32(tr.tiles)[:n]
        np.testing.assert_array_equal(rad, ref.radius)
        np.testing.assert_array_equal(tiles, ref.tiles)
        vis_ref = orc.visible(ref.tiles)
        V = int(u32(tr.counts[0:1])[0])
        vis = u32(tr.vis_idx)[:V]
        np.testing.assert_array_equal(vis, vis_ref)
        rect = tr.rect.cpu().numpy().view(np.uint16)[:n]
        np.testing.assert_array_equal(rect[vis].astype(np.int32), ref.rect[vis])
        np.testing.assert_array_equal(tr.depth.cpu().numpy()[vis].view(np.uint32), ref.depth[vis].view(np.uint32))
        np.testing.assert_array_equal(tr.mean2d.cpu().numpy()[vis].view(np.uint32), ref.mean2d_f32[vis].view(np.uint32))
        co = tr.conic.cpu().numpy()[vis]
        np.testing.assert_array_equal(co[:, :3].view(np.uint32), ref.conic_f32[vis].view(np.uint32))
        # the opacity is the fp64 sigmoid rounded once: within half an fp32 ulp
        np.testing.assert_allclose(co[:, 3], ref.opacity[vis], rtol=2.0 ** -24 * (1 + 1e-9), atol=0)
        rgb = tr.rgb.cpu().numpy()[vis]
        np.testing.assert_allclose(rgb, ref.rgb[vis], rtol=1e-5, atol=2e-6)
        cl = tr.clamp.cpu().numpy()[vis]
        sure = ref.clamp_margin[vis] > 1e-5
        np.testing.assert_array_equal(cl[sure], ref.clamp[vis][sure])
        # sorted pairs
        keys_ref, vals_ref, ranges_ref = orc.sorted_pairs(vis_ref, ref, cam)
        M = int(u32(tr.counts[1:2])[0])
        assert M == keys_ref.size
        np.testing.assert_array_equal(u32(tr.vals)[:M], vals_ref)
        np.testing.assert_array_equal(tr.keys.cpu().numpy()[:M].view(np.uint64), keys_ref)
        T = cam.num_tiles
        np.testing.assert_array_equal(u32(tr.ranges)[:2 * T].reshape(T, 2), ranges_ref)
        np.testing.assert_array_equal(u32(tr.tile_order)[:T], expected_tile_order(ranges_ref))
        # emission offsets: exclusive sums of tiles in visible-set (ascending id) order
        order = vis_ref
        offs = np.concatenate([[0], np.cumsum(ref.tiles[order].astype(np.int64))[:-1]])
        np.testing.assert_array_equal(u32(tr.pair_offset)[order], offs)
        # pair_emit: sorted position -> emission position, a permutation under which
        # sorted pair i is tile number k of its primitive's rectangle (row-major),
        # emitted at pair_offset[id] + k
        emit = u32(tr.pair_emit)[:M].astype(np.int64)
        assert np.array_equal(np.sort(emit), np.arange(M))
        gid_of_e = np.repeat(order, ref.tiles[order].astype(np.int64))
        np.testing.assert_array_equal(gid_of_e[emit], vals_ref)
        k_local = np.arange(M) - np.repeat(offs, ref.tiles[order].astype(np.int64))
        rc = ref.rect[gid_of_e]
        wdt = rc[:, 2] - rc[:, 0]
        tile_e = (rc[:, 1] + k_local // wdt) * cam.tiles_x + rc[:, 0] + k_local % wdt
        np.testing.assert_array_equal(tile_e[emit], (keys_ref >> np.uint64(32)).astype(np.int64))
        _say(case, "view", vi, "V", V, "M", M, "ok")


@pytest.mark.parametrize("case", CASES)
def test_raster_forward(case, torch_gpu, orc):
    w = get_case(case)
    tr = trainer_for(w, torch_gpu)
    cam = w.cameras[0]
    tr.project(cam); tr.visible(); tr.bin_sort(); tr.raster_fwd(active=True)
    torch_gpu.cuda.synchronize()
    ref = orc.project(w.scene, cam, 0)
    vis = orc.visible(ref.tiles)
    rn = orc.render(vis, ref, cam)
    H, W = cam.height, cam.width
    img = tr.img.view(-1)[:3 * H * W].cpu().numpy().reshape(3, H, W)
    amb = orc.ambiguous_pixels(rn)
    ok = ~amb
    _say(case, "ambiguous pixels", int(amb.sum()), "of", amb.size)
    assert amb.mean() <= AMB_SHARE
    assert_pixels(img, rn.img, np.broadcast_to(ok, img.shape), "img")
    fT = tr.final_T.view(-1)[:H * W].cpu().numpy().reshape(H, W)
    assert_pixels(fT, rn.T_final, ok, "final_T")
    nc = u32(tr.n_contrib)[:H * W].reshape(H, W)
    np.testing.assert_array_equal(nc[ok], rn.n_contrib[ok])
    # the realized active set: a flag may differ only for a primitive that an
    # ambiguous pixel examined
    act = tr.active.cpu().numpy()[:w.scene.n]
    _, flag = orc.render_backward(vis, ref, cam, np.zeros((3, H, W)))
    diff = np.flatnonzero(act != rn.active)
    assert np.all(flag[diff] & orc.FLAG_AMB_PIXEL), diff[:10]


@pytest.mark.parametrize("case", CASES)
def test_loss_l1(case, torch_gpu, orc):
    w = get_case(case)
    tr = trainer_for(w, torch_gpu)
    cam = w.cameras[0]
    tgt = target_of(w, 0)
    tr.project(cam); tr.visible(); tr.bin_sort(); tr.raster_fwd()
    tr.set_target(tgt)
    tr.loss_l1()
    torch_gpu.cuda.synchronize()
    H, W = cam.height, cam.width
    img = tr.img.view(-1)[:3 * H * W].cpu().numpy().reshape(3, H, W)
    loss, g, _ = orc.loss_l1(img, tgt)
    dL = tr.dL.view(-1)[:3 * H * W].cpu().numpy().reshape(3, H, W)
    np.testing.assert_array_equal(dL, g.astype(np.float32))
    assert abs(tr.loss.item() - loss) <= 1e-5 * abs(loss)


@pytest.mark.parametrize("case", CASES)
def test_raster_fwd_l1_matches_separate_calls(case, torch_gpu, orc):
    """gs_raster_fwd_l1 = gs_raster_fwd then gs_loss_l1: image, transmittance,
    contributor counts, active flags and dL/dimg bit for bit; the loss to the
    last fp32 bits (tile partial sums instead of 2048-element blocks)."""
    w = get_case(case)
    tr = trainer_for(w, torch_gpu)
    cam = w.cameras[0]
    tr.set_target(target_of(w, 0))
    tr.project(cam); tr.visible(); tr.bin_sort()
    tr.raster_fwd(active=True); tr.loss_l1()
    torch_gpu.cuda.synchronize()
    ref = [t.clone() for t in (tr.img, tr.final_T, tr.n_contrib, tr.dL, tr.active)]
    loss_ref = float(tr.loss.item())
    for t in (tr.img, tr.final_T, tr.n_contrib, tr.dL, tr.active, tr.loss):
        t.fill_(7)
    tr.raster_fwd_l1(active=True)
    torch_gpu.cuda.synchronize()
    H, W = cam.height, cam.width
    for a, b, k in zip((tr.img, tr.final_T, tr.n_contrib, tr.dL, tr.active), ref, (3 * H * W, H * W, H * W,
                                                                                   3 * H * W, w.scene.n)):
        assert torch_gpu.equal(a.reshape(-1)[:k], b.reshape(-1)[:k])
    assert abs(float(tr.loss.item()) - loss_ref) <= 1e-6 * abs(loss_ref)


def masked_upstream(orc, w, cam, dL, loss_margin=None):
    """dL with the ambiguous pixels zeroed: a pixel's decisions reach the
    gradients only through its own upstream gradient, so with dL = 0 there the
    fp32 and fp64 sides must agree on every primitive."""
    ref = orc.project(w.scene, cam, 0)
    vis = orc.visible(ref.tiles)
    rn = orc.render(vis, ref, cam)
    amb = orc.ambiguous_pixels(rn, loss_margin)
    return np.where(amb[None, :, :], 0.0, np.asarray(dL, np.float64)), amb, ref, vis


def bwd_compare(w, tr, orc, ref, vis, dL_masked, case):
    cam = tr.cam
    g2, flag, gabs = orc.render_backward(vis, ref, cam, dL_masked, want_abs=True)
    gr = orc.project_backward(w.scene, cam, vis, g2, ref)
    mags, mag_norm = orc.gradient_magnitudes(w.scene, cam, vis, gabs, ref)
    rows = vis.astype(np.int64)
    ok = np.zeros(w.scene.n, bool)
    ok[vis] = True
    ok &= (flag & orc.FLAG_NEAR_CAP) == 0
    ok &= ref.clamp_margin > 1e-5
    ok &= ref.jclamp_margin > 1e-5
    nskip = int(vis.size - ok.sum())
    _say(case, "primitives outside the element-wise check (cap / clamp margins):", nskip, "of", vis.size)
    assert nskip <= max(5, 1e-3 * vis.size)
    g2_gpu = tr.grad2d.cpu().numpy()[:w.scene.n]
    stats = {}
    names = ["du", "dv", "dA", "dB", "dC", "dop", "dr", "dg", "db"]
    for c, nm in enumerate(names):
        stats[nm] = assert_grads(g2_gpu[:, c], g2[:, c], ok, "grad2d." + nm, mag=gabs[:, c])
    okr = ok[rows]
    V = vis.size
    assert int(u32(tr.counts[0:1])[0]) == V
    for name, gp, go, mg in zip(["mean", "log_scale", "quat", "opacity", "sh"], tr.rows_by_group(tr.grad_rows, V),
                                gr.groups(), mags):
        stats[name] = assert_grads(gp, go, okr, "grad." + name, mag=mg)
    # the padding columns of every gradient row are zero
    assert float(tr.grad_rows[:V, tr.row_len:].abs().max()) == 0.0 if tr.ld > tr.row_len else True
    gn = tr.grad_norm.cpu().numpy()[rows]
    stats["grad_norm"] = assert_grads(gn, gr.grad_norm, okr, "grad_norm", mag=mag_norm)
    _say(case, {k: (round(v.get("max_rel", 0), 6), round(v.get("norm_rel", 0), 8)) for k, v in stats.items()})
    _say(case, "elements passing only by the floor / the summation term:",
         {k: (v.get("need_floor"), v.get("need_sum_term"), v.get("n")) for k, v in stats.items()})
    return gr


@pytest.mark.parametrize("case", CASES)
def test_raster_backward(case, torch_gpu, orc):
    from paper_2607_19893_amd import scenes
    w = get_case(case)
    tr = trainer_for(w, torch_gpu)
    cam = w.cameras[0]
    dL = scenes.make_upstream_grad(cam.width, cam.height, 17)
    dLm, amb, ref, vis = masked_upstream(orc, w, cam, dL)
    _say(case, "ambiguous pixels zeroed in dL:", int(amb.sum()))
    tr.project(cam); tr.visible(); tr.bin_sort(); tr.raster_fwd()
    tr.set_dL(dLm.astype(np.float32))
    tr.raster_bwd(grad2d=True)
    torch_gpu.cuda.synchronize()
    bwd_compare(w, tr, orc, ref, vis, dLm.astype(np.float32).astype(np.float64), case)


def _adam_case(n=5000, K=1234, seed=3):
    from paper_2607_19893_amd import scenes
    rng = np.random.default_rng(seed)
    cols = [3, 3, 4, 1, 48]
    p = [rng.standard_normal((n, c)).astype(np.float32) for c in cols]
    g = [(rng.standard_normal((n, c)) * 1e-3).astype(np.float32) for c in cols]
    mv = [scenes.adam_state(5, n, c) for c in cols]
    idx = np.sort(rng.choice(n, K, replace=False)).astype(np.uint32)
    lrs = [1e-3, 2e-3, 1e-3, 5e-2, 2.5e-3]
    return cols, p, g, mv, idx, lrs


def _rows_table(groups, ld, rows=None):
    """Concatenate per-group arrays [*, cols] (optionally gathered at rows) into a [*, ld] table."""
    parts = [a if rows is None else a[rows] for a in groups]
    t = np.concatenate(parts, axis=1)
    out = np.zeros((t.shape[0], ld), np.float32)
    out[:, :t.shape[1]] = t
    return out


def _split(table, cols):
    offs = np.cumsum([0] + cols)
    return [table[:, offs[i]:offs[i + 1]] for i in range(len(cols))]


class _AdamGpu:
    """Device state of one sparse-Adam case: pool groups, compact gradient rows, moment tables."""

    def __init__(self, cols, p, g, mv, idx, lrs, ld=64):
        import torch
        from paper_2607_19893_amd import gsmi
        dev = torch.device("cuda")
        self.cols, self.ld, self.n = cols, ld, p[0].shape[0]
        self.P = [torch.from_numpy(a.copy()).to(dev) for a in p]
        gt = _rows_table(g, ld, idx.astype(np.int64))
        self.G = torch.from_numpy(gt if gt.shape[0] else np.zeros((1, ld), np.float32)).to(dev)
        self.M = torch.from_numpy(_rows_table([a[0] for a in mv], ld)).to(dev)
        self.Vv = torch.from_numpy(_rows_table([a[1] for a in mv], ld)).to(dev)
        self.D = torch.zeros(max(1, idx.size), ld, device=dev)
        self.arr = gsmi.make_adam_groups([(a, lr) for a, lr in zip(self.P, lrs)])
        self.I = torch.from_numpy(idx.view(np.int32).copy() if idx.size else np.zeros(1, np.int32)).to(dev)
        self.cnt = torch.tensor([idx.size], dtype=torch.int32, device=dev)
        self.K = idx.size

    def adam(self, step):
        from paper_2607_19893_amd import gsmi
        gsmi.gs_sparse_adam(self.arr, 5, self.I, self.cnt, self.n, self.G, self.ld, self.M, self.Vv, self.ld, step,
                            0.9, 0.999, 1e-15, self.D, self.ld)

    def publish(self, step, version, msg, status):
        from paper_2607_19893_amd import gsmi
        gsmi.gs_sparse_adam_publish(self.arr, 5, self.I, self.cnt, self.n, self.G, self.ld, self.M, self.Vv, self.ld,
                                    step, 0.9, 0.999, 1e-15, version, msg, status)


def adam_step_floor(m_old, g, v_new, step, lr, beta1=0.9, beta2=0.999, eps=1e-15):
    """Per element, the magnitude the fp32 rounding error of an Adam step is
    relative to: m = b1 m + (1 - b1) g rounds relative to b1 |m| + (1 - b1) |g|
    (the two terms can cancel), and the step scales m by
    (lr / (1 - b1^t)) / (sqrt(v / (1 - b2^t)) + eps)."""
    m_old, g, v_new = (np.asarray(a, np.float64) for a in (m_old, g, v_new))
    fm = beta1 * np.abs(m_old) + (1 - beta1) * np.abs(g)
    return lr / (1 - beta1 ** step) * fm / (np.sqrt(v_new / (1 - beta2 ** step)) + eps)


def test_sparse_adam(torch_gpu, orc):
    import torch
    cols, p, g, mv, idx, lrs = _adam_case()
    n = p[0].shape[0]
    st = _AdamGpu(cols, p, g, mv, idx, lrs)
    rows = np.zeros(n, bool); rows[idx] = True
    for step in (1, 7):
        st.adam(step)
        torch.cuda.synchronize()
        m_gpu = _split(st.M.cpu().numpy()[:n], cols)
        v_gpu = _split(st.Vv.cpu().numpy()[:n], cols)
        d_gpu = _split(st.D.cpu().numpy()[:idx.size], cols)
        assert float(st.M[:, sum(cols):].abs().max()) == 0.0     # padding columns untouched
        for k in range(5):
            pr, mr, vr, dr = orc.adam(p[k], g[k], mv[k][0], mv[k][1], idx, step, lrs[k], 0.9, 0.999, 1e-15)
            gp = st.P[k].cpu().numpy()
            np.testing.assert_array_equal(gp[~rows], p[k][~rows])        # untouched rows
            np.testing.assert_array_equal(m_gpu[k][~rows], mv[k][0][~rows])
            # fp32 rounding of b*m + (1-b)*g is relative to the operands' magnitudes
            g64 = g[k].astype(np.float64)
            fm = 0.9 * np.abs(mv[k][0]) + 0.1 * np.abs(g64)
            fv = 0.999 * np.abs(mv[k][1]) + 0.001 * g64 * g64
            assert_grads(m_gpu[k], mr, rows, "m%d" % k, rtol=1e-5, floor=fm)
            assert_grads(v_gpu[k], vr, rows, "v%d" % k, rtol=1e-5, floor=fv)
            rr = idx.astype(np.int64)
            assert_grads(d_gpu[k], dr, np.ones(idx.size, bool), "delta%d" % k, rtol=2e-5,
                         floor=adam_step_floor(mv[k][0][rr], g[k][rr], vr[rr], step, lrs[k]))
            assert_grads(gp, pr, rows, "p%d" % k, rtol=1e-6)
            p[k], mv[k] = pr.astype(np.float32), (mr.astype(np.float32), vr.astype(np.float32))
        # continue from the oracle's state
        for k in range(5):
            st.P[k].copy_(torch.from_numpy(p[k]))
        st.M.copy_(torch.from_numpy(_rows_table([a[0] for a in mv], st.ld)))
        st.Vv.copy_(torch.from_numpy(_rows_table([a[1] for a in mv], st.ld)))


@pytest.mark.parametrize("K", [0, 1, 777, 5000])
def test_sparse_adam_publish(K, torch_gpu, orc):
    """The fused update + staging: same parameters and moments as gs_sparse_adam bit for bit, a message whose
    header and ids equal the oracle's and whose rows are the oracle's steps (and gs_sparse_adam's, bit for bit)."""
    import torch
    from paper_2607_19893_amd import gsmi
    cols, p, g, mv, idx, lrs = _adam_case(K=K, seed=11 + K)
    n = p[0].shape[0]
    a = _AdamGpu(cols, p, g, mv, idx, lrs)
    b = _AdamGpu(cols, p, g, mv, idx, lrs)
    row_len = sum(cols)
    nbytes = gsmi.gs_delta_msg_bytes(K, row_len, len(cols))
    msg = torch.full(((nbytes + 15) // 16 * 4,), -1, dtype=torch.int32, device="cuda")
    status = torch.zeros(4, dtype=torch.int32, device="cuda")
    a.adam(3)
    b.publish(3, 42, msg, status)
    torch.cuda.synchronize()
    assert int(status[0]) == 0
    for k in range(5):
        assert torch.equal(a.P[k], b.P[k])
    assert torch.equal(a.M, b.M) and torch.equal(a.Vv, b.Vv)
    words = msg.cpu().numpy().view(np.uint32)[:nbytes // 4]
    deltas, floors = [], []
    rr = idx.astype(np.int64)
    for k in range(5):
        _, _, vr, dr = orc.adam(p[k], g[k], mv[k][0], mv[k][1], idx, 3, lrs[k], 0.9, 0.999, 1e-15)
        full = np.zeros((n, cols[k]))
        full[rr] = dr
        deltas.append(full)
        floors.append(adam_step_floor(mv[k][0][rr], g[k][rr], vr[rr], 3, lrs[k]))
    ref = orc.delta_pack(idx, deltas, 42)
    head = ref.size - K * row_len
    np.testing.assert_array_equal(words[:head], ref[:head])
    rows_gpu = words[head:].view(np.float32).reshape(K, row_len)
    np.testing.assert_array_equal(rows_gpu, a.D.cpu().numpy()[:K, :row_len])
    rows_orc = np.concatenate([d[idx.astype(np.int64)] for d in deltas], axis=1) if K else np.zeros((0, row_len))
    fl = np.concatenate(floors, axis=1) if K else np.zeros((0, row_len))
    assert_grads(rows_gpu.astype(np.float64), rows_orc, np.ones(K, bool), "msg rows", rtol=2e-5, floor=fl)
    # too small a buffer: nothing is written, the required size is reported
    if K > 0:
        c = _AdamGpu(cols, p, g, mv, idx, lrs)
        small = torch.zeros(((nbytes - 16) // 4,), dtype=torch.int32, device="cuda")
        st2 = torch.zeros(4, dtype=torch.int32, device="cuda")
        c.publish(3, 42, small, st2)
        torch.cuda.synchronize()
        s2 = st2.cpu().numpy().view(np.uint32)
        assert s2[0] & gsmi.GS_DEV_MSG_OVERFLOW and s2[1] == nbytes
        assert int(small.abs().max()) == 0
        for k in range(5):
            np.testing.assert_array_equal(c.P[k].cpu().numpy(), p[k])
        np.testing.assert_array_equal(c.M.cpu().numpy(), _rows_table([x[0] for x in mv], c.ld))


def test_delta_pack_apply(torch_gpu, orc):
    import torch
    from paper_2607_19893_amd import gsmi
    rng = np.random.default_rng(4)
    dev = torch.device("cuda")
    for n, K, cols in ((1000, 333, [3, 3, 4, 1, 48]), (64, 0, [3, 3, 4, 1, 3]), (70000, 70000, [3, 3, 4, 1, 48])):
        src = [rng.standard_normal((n, c)).astype(np.float32) for c in cols]
        dst0 = [rng.standard_normal((n, c)).astype(np.float32) for c in cols]
        idx = np.sort(rng.choice(n, K, replace=False)).astype(np.uint32)
        S = [torch.from_numpy(a).to(dev) for a in src]
        I = torch.from_numpy(idx.view(np.int32).copy() if K else np.zeros(1, np.int32)).to(dev)
        cnt = torch.tensor([K], dtype=torch.int32, device=dev)
        nbytes = gsmi.gs_delta_msg_bytes(K, sum(cols), len(cols))
        msg = torch.zeros((nbytes + 15) // 4, dtype=torch.int32, device=dev)
        st = torch.zeros(4, dtype=torch.int32, device=dev)
        gsmi.gs_delta_pack(I, cnt, n, gsmi.make_groups(S), len(cols), 5, msg, st)
        torch.cuda.synchronize()
        assert st.cpu().numpy()[0] == 0
        ref = orc.delta_pack(idx, src, 5)
        got = msg.cpu().numpy().view(np.uint32)[:ref.size]
        np.testing.assert_array_equal(got, ref)
        for mode, name in ((gsmi.GS_APPLY_ADD, "add"), (gsmi.GS_APPLY_OVERWRITE, "overwrite")):
            Dd = [torch.from_numpy(a.copy()).to(dev) for a in dst0]
            ver = torch.zeros(n, dtype=torch.int32, device=dev)
            gsmi.gs_delta_apply(msg, gsmi.make_groups(Dd), len(cols), n, n, mode, ver, st)
            torch.cuda.synchronize()
            out, vref = orc.delta_apply(ref, dst0, name, np.zeros(n, np.uint32))
            for a, b in zip(Dd, out):
                np.testing.assert_array_equal(a.cpu().numpy().view(np.uint32), b.view(np.uint32))
            np.testing.assert_array_equal(ver.cpu().numpy().view(np.uint32), vref)
    # overflow: capacity too small -> flag + required bytes, no header written
    msg = torch.zeros(16, dtype=torch.int32, device=dev)
    st = torch.zeros(4, dtype=torch.int32, device=dev)
    gsmi.gs_delta_pack(I, cnt, n, gsmi.make_groups(S), len(cols), 5, msg, st)
    torch.cuda.synchronize()
    s = st.cpu().numpy().view(np.uint32)
    assert s[0] & gsmi.GS_DEV_MSG_OVERFLOW and s[1] == gsmi.gs_delta_msg_bytes(K, sum(cols), len(cols))
    # mismatch: a destination with different widths is refused and left untouched
    good = torch.zeros((gsmi.gs_delta_msg_bytes(K, sum(cols), len(cols)) + 15) // 4, dtype=torch.int32, device=dev)
    st.zero_()
    gsmi.gs_delta_pack(I, cnt, n, gsmi.make_groups(S), len(cols), 5, good, st)
    wrong = [torch.zeros(n, c, device=dev) for c in (3, 3, 4, 1, 45)]
    gsmi.gs_delta_apply(good, gsmi.make_groups(wrong), 5, n, n, gsmi.GS_APPLY_ADD, None, st)
    torch.cuda.synchronize()
    assert st.cpu().numpy()[0] & gsmi.GS_DEV_MSG_MISMATCH
    assert all(float(t.abs().sum()) == 0.0 for t in wrong)


def test_long_tile_lists(torch_gpu, orc):
    """Tiles whose pair lists exceed the per-tile LDS sort (thousands of wide
    primitives over the image centre) take the global-memory path; the order
    is still exactly (tile, depth bits, id), including equal depths."""
    from paper_2607_19893_amd import scenes
    rng = np.random.default_rng(21)
    w = scenes.tiny(n=9000)
    sc = w.scene
    sc.mean[:] = (rng.standard_normal((sc.n, 3)) * [0.05, 0.05, 0.3]).astype(np.float32)
    sc.mean[:3000, 2] = 0.5                      # equal depths: ties broken by id
    sc.log_scale[:] = np.float32(-2.5)
    tr = trainer_for(w, torch_gpu)
    cam = w.cameras[0]
    tr.status.zero_()
    tr.project(cam); tr.visible(); tr.bin_sort()
    torch_gpu.cuda.synchronize()
    assert u32(tr.status)[0] == 0
    ref = orc.project(sc, cam, 0)
    vis_ref = orc.visible(ref.tiles)
    keys_ref, vals_ref, ranges_ref = orc.sorted_pairs(vis_ref, ref, cam)
    lengths = ranges_ref[:, 1].astype(np.int64) - ranges_ref[:, 0]
    _say("longest tile list", int(lengths.max()), "tiles above 2048:", int((lengths > 2048).sum()))
    assert lengths.max() > 2048
    M = int(u32(tr.counts[1:2])[0])
    assert M == keys_ref.size
    np.testing.assert_array_equal(u32(tr.vals)[:M], vals_ref)
    np.testing.assert_array_equal(tr.keys.cpu().numpy()[:M].view(np.uint64), keys_ref)
    T = cam.num_tiles
    np.testing.assert_array_equal(u32(tr.ranges)[:2 * T].reshape(T, 2), ranges_ref)
    order = u32(tr.tile_order)[:T]
    np.testing.assert_array_equal(order, expected_tile_order(ranges_ref))
    assert lengths[order[0]] == lengths.max()


# (tile x, tile y, primitives, short ties, long run): one cluster per tile
# class of the per-tile depth sort, from one wave with one key per lane up to
# tiles longer than a workgroup's register sort (two runs merged, 2049..4096
# pairs) and longer than two runs (global memory).  Short ties: an eighth of
# the primitives copy a neighbour's mean (runs of equal depth bits of a few
# pairs); long run: that many primitives share one mean (a run longer than
# the in-place placement takes).
DEPTH_SORT_CLUSTERS = [(1, 1, 40, True, 0), (3, 1, 40, False, 0), (5, 1, 100, True, 0), (7, 1, 200, True, 0),
                       (9, 1, 400, True, 0), (11, 1, 400, False, 0), (13, 1, 230, False, 0),
                       (1, 5, 1000, False, 0), (5, 5, 1000, True, 0), (9, 5, 1800, False, 0),
                       (13, 5, 3000, False, 0), (3, 9, 700, True, 0), (7, 9, 300, False, 80),
                       (11, 9, 900, False, 100), (1, 13, 2300, True, 0), (5, 13, 2600, False, 300),
                       (9, 13, 4500, True, 0)]


def test_depth_sort_paths(torch_gpu, orc):
    """Tiles of every size class of the per-tile sort (one wave with 1, 2, 4
    or 8 keys per lane, a workgroup up to 2048 keys, two merged runs up to
    4096, global memory beyond), with and without pairs of equal depth bits
    (copies of a primitive's mean): the order is exactly (tile, depth bits,
    id) in every class."""
    from paper_2607_19893_amd import scenes
    rng = np.random.default_rng(33)
    n_bg = 1500
    n = n_bg + sum(c[2] for c in DEPTH_SORT_CLUSTERS)
    w = scenes.tiny(n=n)
    sc = w.scene
    cam = w.cameras[0]
    R = np.asarray(cam.R, np.float64)
    k = n_bg
    for tx, ty, cnt, ties, run in DEPTH_SORT_CLUSTERS:
        # pixels inside the tile (away from its edges), camera depths in [2, 6]
        u = tx * 16 + 8 + rng.uniform(-3, 3, cnt)
        v = ty * 16 + 8 + rng.uniform(-3, 3, cnt)
        z = rng.uniform(2.0, 6.0, cnt)
        pc = np.stack([(u - cam.cx) * z / cam.fx, (v - cam.cy) * z / cam.fy, z], 1)
        mean = (pc - np.asarray(cam.t, np.float64)) @ R           # R^T (p - t)
        if ties:
            dup = rng.choice(cnt, cnt // 8, replace=False)
            mean[dup] = mean[(dup + 1) % cnt]
        mean[1:run] = mean[0]
        sc.mean[k:k + cnt] = mean.astype(np.float32)
        k += cnt
    sc.log_scale[n_bg:] = np.float32(-5.5)
    tr = trainer_for(w, torch_gpu)
    tr.status.zero_()
    tr.project(cam); tr.visible(); tr.bin_sort()
    torch_gpu.cuda.synchronize()
    assert u32(tr.status)[0] == 0
    ref = orc.project(sc, cam, 0)
    vis_ref = orc.visible(ref.tiles)
    keys_ref, vals_ref, ranges_ref = orc.sorted_pairs(vis_ref, ref, cam)
    T = cam.num_tiles
    lengths = ranges_ref[:, 1].astype(np.int64) - ranges_ref[:, 0]
    tied, longest = 0, []
    for t in range(T):
        kk = keys_ref[ranges_ref[t, 0]:ranges_ref[t, 1]] & np.uint64(0xFFFFFFFF)
        tied += int(kk.size != np.unique(kk).size)
        longest.append(int(np.unique(kk, return_counts=True)[1].max()) if kk.size else 0)
    for tx, ty, cnt, ties, run in DEPTH_SORT_CLUSTERS:
        t = ty * cam.tiles_x + tx
        _say("cluster tile (%d,%d): %d pairs, longest run of equal depth bits %d" % (tx, ty, lengths[t], longest[t]))
    _say("tiles with equal depth bits:", tied)
    cl = [lengths[ty * cam.tiles_x + tx] for tx, ty, _, _, _ in DEPTH_SORT_CLUSTERS]
    assert min(cl) <= 64 and max(cl) > 4096 and any(512 <= c <= 2048 for c in cl)
    assert sum(2048 < c <= 4096 for c in cl) >= 3
    assert any(256 < c < 512 for c in cl) and tied >= 4
    runs = {(tx, ty): longest[ty * cam.tiles_x + tx] for tx, ty, _, _, _ in DEPTH_SORT_CLUSTERS}
    assert runs[(7, 9)] > 64 and runs[(11, 9)] > 64 and 2 <= runs[(9, 1)] <= 64 and 2 <= runs[(5, 5)] <= 64
    M = int(u32(tr.counts[1:2])[0])
    assert M == keys_ref.size
    np.testing.assert_array_equal(tr.keys.cpu().numpy()[:M].view(np.uint64), keys_ref)
    np.testing.assert_array_equal(u32(tr.vals)[:M], vals_ref)
    np.testing.assert_array_equal(u32(tr.ranges)[:2 * T].reshape(T, 2), ranges_ref)
    np.testing.assert_array_equal(u32(tr.tile_order)[:T], expected_tile_order(ranges_ref))
    # emission offsets, and the sorted -> emission map: sorted pair i is tile number
    # (ty - y0) * (x1 - x0) + (tx - x0) of primitive vals[i]'s rectangle
    off_ref = np.cumsum(ref.tiles[vis_ref].astype(np.int64)) - ref.tiles[vis_ref]
    np.testing.assert_array_equal(u32(tr.pair_offset)[vis_ref], off_ref)
    tile = (keys_ref >> np.uint64(32)).astype(np.int64)
    rc = ref.rect[vals_ref].astype(np.int64)
    local = (tile // cam.tiles_x - rc[:, 1]) * (rc[:, 2] - rc[:, 0]) + (tile % cam.tiles_x - rc[:, 0])
    full = np.zeros(sc.n, np.int64)
    full[vis_ref] = off_ref
    np.testing.assert_array_equal(u32(tr.pair_emit)[:M], full[vals_ref] + local)


def test_pair_overflow_flag(torch_gpu, orc):
    """Capacity below the pair count: the flag and the required count are set."""
    w = get_case("tiny-10k-256")
    tr = trainer_for(w, torch_gpu, capacity=1000)
    tr.status.zero_()
    tr.project(w.cameras[0]); tr.visible(); tr.bin_sort()
    torch_gpu.cuda.synchronize()
    s = u32(tr.status)
    M = int(u32(tr.counts[1:2])[0])
    assert s[0] & 1 and s[1] == M and M > 1000
    assert np.all(u32(tr.ranges) == 0)
    T = w.cameras[0].num_tiles
    np.testing.assert_array_equal(u32(tr.tile_order)[:T], np.arange(T))


def test_pair_overflow_leaves_state_untouched(torch_gpu, orc):
    """A training step whose pair list overflows its capacity changes no
    state: the backward finds no pair slot of the view (the slot buffer holds
    another view's values here), so every gradient row it writes is zero;
    Adam + staging sees the overflow flag in the shared device status and
    writes nothing; the commit then finds no message of the version and
    refuses.  Parameters, moments, message slots, replica and versions stay
    bit-identical."""
    torch = torch_gpu
    w = get_case("tiny-10k-256")
    tr = trainer_for(w, torch, capacity=1000)
    tr.set_target(target_of(w, 0))
    tr.ws_bwd.view(torch.float32).fill_(1.0)        # stale slots of an earlier view
    tr.grad_rows.fill_(7.0)
    snap = lambda: [t.clone() for t in (*tr.params, tr.m, tr.v, *tr.msgs, *tr.replica, tr.version, tr.ring_state)]
    before = snap()
    tr.status.zero_()
    tr.step(w.cameras[0], step=1, version=1)
    torch.cuda.synchronize()
    s = u32(tr.status)
    M = int(u32(tr.counts[1:2])[0])
    assert M > 1000 and s[0] & 1 and s[1] >= M
    assert s[0] & 4                                  # the commit refused: no message of version 1
    V = int(u32(tr.counts[0:1])[0])
    assert V > 0
    assert np.all(tr.grad_rows[:V].cpu().numpy() == 0.0)
    assert np.all(u32(tr.pair_offset)[u32(tr.vis_idx)[:V]] == 0xFFFFFFFF)
    for a, b in zip(before, snap()):
        assert torch.equal(a, b)


def test_zero_tile_ids_in_the_visible_list(torch_gpu, orc):
    """gs_bin_sort over an id list that also holds primitives with no tile
    (here every id, 90% of them culled, so one 2048-pair emission block spans
    far more ranks than its LDS staging holds): the same pairs, order,
    ranges, dispatch order and emission map as over the visible set."""
    from paper_2607_19893_amd import scenes
    torch = torch_gpu
    w = scenes.tiny(n=20000)
    w.scene.mean[np.arange(w.scene.n) % 10 != 0, 2] = -10.0     # behind the camera
    tr = trainer_for(w, torch, capacity=1 << 16)
    cam = w.cameras[0]
    T = cam.num_tiles
    tr.status.zero_()
    tr.project(cam); tr.visible(); tr.bin_sort()
    torch.cuda.synchronize()
    V = int(u32(tr.counts[0:1])[0])
    M = int(u32(tr.counts[1:2])[0])
    assert 1500 < V <= 2000 and M > 2048
    ref = [u32(t)[:k].copy() for t, k in ((tr.vals, M), (tr.pair_emit, M), (tr.ranges, 2 * T), (tr.tile_order, T))]
    keys = tr.keys.cpu().numpy()[:M].copy()
    vis = u32(tr.vis_idx)[:V].copy()
    off = u32(tr.pair_offset)[vis].copy()
    for t in (tr.vals, tr.pair_emit, tr.ranges, tr.tile_order, tr.keys, tr.pair_offset):
        t.fill_(-1)
    n = w.scene.n
    tr.vis_idx.copy_(torch.arange(n, dtype=torch.int32, device=tr.vis_idx.device))
    tr.counts[0:1].fill_(n)
    tr.bin_sort()
    torch.cuda.synchronize()
    assert u32(tr.status)[0] == 0 and int(u32(tr.counts[1:2])[0]) == M
    got = [u32(t)[:k] for t, k in ((tr.vals, M), (tr.pair_emit, M), (tr.ranges, 2 * T), (tr.tile_order, T))]
    for a, b in zip(ref, got):
        np.testing.assert_array_equal(a, b)
    np.testing.assert_array_equal(tr.keys.cpu().numpy()[:M], keys)
    np.testing.assert_array_equal(u32(tr.pair_offset)[vis], off)


def test_offsets_over_many_rank_blocks(torch_gpu, orc):
    """gs_bin_sort over a list of 9M ids of which one in a thousand has tiles:
    the offsets pass then adds up more than 4096 per-block tile sums (two
    rounds of 16-byte loads per thread) for every block's offset and for the
    pair total, and must give the same pairs, order, ranges and emission map
    as over the visible set alone."""
    from paper_2607_19893_amd import scenes
    torch = torch_gpu
    n = 9_000_000
    assert (n + 2047) // 2048 > 4096
    w = scenes.tiny(n=n)
    w.scene.mean[np.arange(n) % 1000 != 0, 2] = -10.0      # behind the camera
    tr = trainer_for(w, torch, capacity=1 << 16)
    cam = w.cameras[0]
    T = cam.num_tiles
    tr.status.zero_()
    tr.project(cam); tr.visible(); tr.bin_sort()
    torch.cuda.synchronize()
    V = int(u32(tr.counts[0:1])[0])
    M = int(u32(tr.counts[1:2])[0])
    assert 8000 < V <= 9000 and 2048 < M <= 1 << 16
    ref = [u32(t)[:k].copy() for t, k in ((tr.vals, M), (tr.pair_emit, M), (tr.ranges, 2 * T), (tr.tile_order, T))]
    vis = u32(tr.vis_idx)[:V].copy()
    off = u32(tr.pair_offset)[vis].copy()
    tiles = u32(tr.tiles)[vis].astype(np.int64)
    for t in (tr.vals, tr.pair_emit, tr.ranges, tr.tile_order, tr.pair_offset):
        t.fill_(-1)
    tr.vis_idx.copy_(torch.arange(n, dtype=torch.int32, device=tr.vis_idx.device))
    tr.counts[0:1].fill_(n)
    tr.bin_sort()
    torch.cuda.synchronize()
    assert u32(tr.status)[0] == 0 and int(u32(tr.counts[1:2])[0]) == M
    got = [u32(t)[:k] for t, k in ((tr.vals, M), (tr.pair_emit, M), (tr.ranges, 2 * T), (tr.tile_order, T))]
    for a, b in zip(ref, got):
        np.testing.assert_array_equal(a, b)
    np.testing.assert_array_equal(u32(tr.pair_offset)[vis], off)
    # the offsets are the exclusive prefix of the visible ids' tile counts
    np.testing.assert_array_equal(off, np.concatenate([[0], np.cumsum(tiles)[:-1]]).astype(np.uint32))


def test_projection_near_the_image_border(torch_gpu, orc):
    """Primitives centred up to 300 pixels past every border of the image,
    with one long scale axis, random rotations and camera depths from 0.3 to
    20: radius, tile counts and rectangles equal the oracle's bit for bit, so
    the projection's early off-screen cull (a bound on the radius from the
    largest scale) rejects exactly the primitives whose rectangle is empty."""
    from paper_2607_19893_amd import scenes
    rng = np.random.default_rng(41)
    n = 200_000
    w = scenes.tiny(n=n)
    cam = w.cameras[0]
    u = rng.uniform(-300.0, cam.width + 300.0, n)
    v = rng.uniform(-300.0, cam.height + 300.0, n)
    z = np.exp(rng.uniform(np.log(0.3), np.log(20.0), n))
    pc = np.stack([(u - cam.cx) * z / cam.fx, (v - cam.cy) * z / cam.fy, z], 1)
    R = np.asarray(cam.R, np.float64)
    w.scene.mean[:] = ((pc - np.asarray(cam.t, np.float64)) @ R).astype(np.float32)   # R^T (p - t)
    ls = rng.normal(-3.0, 1.0, (n, 3))
    ls[:, 0] += rng.uniform(0.0, 3.0, n)
    w.scene.log_scale[:] = ls.astype(np.float32)
    tr = trainer_for(w, torch_gpu, capacity=1 << 20)
    tr.project(cam)
    torch_gpu.cuda.synchronize()
    ref = orc.project(w.scene, cam, 0)
    np.testing.assert_array_equal(tr.radius.cpu().numpy()[:n], ref.radius)
    np.testing.assert_array_equal(u32(tr.tiles)[:n], ref.tiles)
    vis = np.flatnonzero(ref.tiles)
    rect = tr.rect.cpu().numpy().view(np.uint16)[:n]
    np.testing.assert_array_equal(rect[vis].astype(np.int32), ref.rect[vis])
    outside = (u < 0) | (u >= cam.width) | (v < 0) | (v >= cam.height)
    reach = int((outside & (ref.tiles > 0)).sum())
    _say("centres outside the image: %d, of which %d reach a tile" % (int(outside.sum()), reach))
    assert reach > 1000 and int((outside & (ref.tiles == 0)).sum()) > 10000


def test_clearing_compaction(torch_gpu, orc):
    """GS_PRED_U8_NONZERO_CLEAR gives the ascending ids of the nonzero flags (as
    GS_PRED_U8_NONZERO does) and leaves every flag at 0, through gs_visible_set
    and gs_visible_set_noalloc, on lengths with a ragged last block; a second
    call then finds nothing."""
    from paper_2607_19893_amd import gsmi as gs
    torch = torch_gpu
    rng = np.random.default_rng(7)
    for n in (300_001, 5, 3 * 2048):
        f = np.where(rng.random(n) < 0.3, rng.integers(1, 256, n), 0).astype(np.uint8)
        want = np.flatnonzero(f).astype(np.uint32)
        for noalloc in (False, True):
            flags = torch.from_numpy(f.copy()).cuda()
            out = torch.zeros(n, dtype=torch.int32, device="cuda")
            cnt = torch.zeros(1, dtype=torch.int32, device="cuda")
            ws = torch.zeros(gs.gs_workspace_bytes(gs.GS_WS_VISIBLE_SET, n, 0, 0, 0), dtype=torch.uint8,
                             device="cuda")
            for rep in range(2):
                if noalloc:
                    gs.gs_visible_set_noalloc(gs.GS_PRED_U8_NONZERO_CLEAR, flags, n, out, cnt)
                else:
                    gs.gs_visible_set(gs.GS_PRED_U8_NONZERO_CLEAR, flags, n, out, cnt, ws)
                torch.cuda.synchronize()
                c = int(u32(cnt)[0])
                if rep == 0:
                    assert c == want.size, (n, noalloc, c, want.size)
                    np.testing.assert_array_equal(u32(out)[:c], want)
                    assert int(flags.max()) == 0
                else:
                    assert c == 0


def test_empty_and_degenerate(torch_gpu, orc):
    """All primitives behind the camera: empty visible set, empty image."""
    from paper_2607_19893_amd import scenes
    w = scenes.tiny(n=500)
    w.scene.mean[:, 2] = -10.0
    tr = trainer_for(w, torch_gpu, capacity=1024)
    tr.set_target(target_of(w, 0))
    tr.step(w.cameras[0], step=1)
    torch_gpu.cuda.synchronize()
    assert int(u32(tr.counts[0:1])[0]) == 0 and int(u32(tr.counts[1:2])[0]) == 0
    assert int(u32(tr.counts[2:3])[0]) == 0                 # no realized active primitive
    hw = w.cameras[0].width * w.cameras[0].height
    assert float(tr.img.view(-1)[:3 * hw].abs().max()) == 0.0
    assert float(tr.final_T.view(-1)[:hw].min()) == 1.0
    T = w.cameras[0].num_tiles
    np.testing.assert_array_equal(u32(tr.tile_order)[:T], np.arange(T))


@pytest.mark.parametrize("case", ["room-60k-392x216", "ring-20k-328x184"])
def test_dispatch_order_changes_no_result(case, torch_gpu, orc):
    """The raster kernels in the longest-first tile order and in row-major
    order give the same image, transmittance, contributor counts, active
    flags, pair statistics, loss, dL/dimg and gradients, bit for bit."""
    w = get_case(case)
    runs = []
    for longest_first in (True, False):
        tr = trainer_for(w, torch_gpu)
        tr.longest_first = longest_first
        cam = w.cameras[1]
        tr.set_target(target_of(w, 1))
        tr.pair_stats.zero_()
        tr.project(cam); tr.visible(); tr.bin_sort()
        tr.raster_fwd(active=True, stats=True)
        out = [t.clone() for t in (tr.img, tr.final_T, tr.n_contrib, tr.active, tr.pair_stats)]
        tr.raster_fwd_l1()
        tr.raster_bwd(grad2d=True)
        torch_gpu.cuda.synchronize()
        out += [t.clone() for t in (tr.loss, tr.dL, tr.grad_rows, tr.grad2d, tr.grad_norm)]
        order = u32(tr.tile_order)[:cam.num_tiles]
        assert np.array_equal(np.sort(order), np.arange(cam.num_tiles))
        runs.append(out)
    for a, b in zip(*runs):
        assert torch_gpu.equal(a, b)


def test_tile_order_large_image(torch_gpu, orc):
    """An image of more than 32768 tiles (4100x2320: 37265) takes the tile
    order's scanned path: ranges, pair order and tile order bit-exact, and
    the forward image the same in either dispatch order."""
    from paper_2607_19893_amd import scenes
    w = scenes.ring(n=20000, width=4100, height=2320)
    cam = w.cameras[0]
    T = cam.num_tiles
    assert T > 32768
    ref = orc.project(w.scene, cam, 0)
    vis_ref = orc.visible(ref.tiles)
    keys_ref, vals_ref, ranges_ref = orc.sorted_pairs(vis_ref, ref, cam)
    imgs = []
    for longest_first in (True, False):
        tr = trainer_for(w, torch_gpu)
        tr.longest_first = longest_first
        tr.status.zero_()
        tr.project(cam); tr.visible(); tr.bin_sort(); tr.raster_fwd()
        torch_gpu.cuda.synchronize()
        assert u32(tr.status)[0] == 0
        M = int(u32(tr.counts[1:2])[0])
        assert M == keys_ref.size
        np.testing.assert_array_equal(u32(tr.vals)[:M], vals_ref)
        np.testing.assert_array_equal(u32(tr.ranges)[:2 * T].reshape(T, 2), ranges_ref)
        np.testing.assert_array_equal(u32(tr.tile_order)[:T], expected_tile_order(ranges_ref))
        imgs.append(tr.img.view(-1)[:3 * cam.width * cam.height].clone())
    assert torch_gpu.equal(imgs[0], imgs[1])


def test_backward_halves_match_combined(torch_gpu, orc):
    """gs_raster_bwd_pixels + gs_raster_bwd_project give gs_raster_bwd's result bit for bit."""
    w = get_case("room-60k-392x216")
    tr = trainer_for(w, torch_gpu)
    cam = w.cameras[0]
    tr.set_target(target_of(w, 0))
    tr.project(cam); tr.visible(); tr.bin_sort(); tr.raster_fwd(); tr.loss_l1()
    tr.raster_bwd(grad2d=True)
    torch_gpu.cuda.synchronize()
    ref = [tr.grad_rows.clone(), tr.grad2d.clone(), tr.grad_norm.clone()]
    tr.grad_rows.zero_(); tr.grad2d.zero_(); tr.grad_norm.zero_()
    tr.raster_bwd_pixels()
    tr.raster_bwd_project(grad2d=True)
    torch_gpu.cuda.synchronize()
    got = [tr.grad_rows, tr.grad2d, tr.grad_norm]
    for a, b in zip(got, ref):
        assert torch_gpu.equal(a, b)


def test_step_matches_phase_calls(torch_gpu, orc):
    """The training step's prepared-argument launches give the phase-by-phase
    calls' results bit for bit (parameters, moments, replica, versions, image,
    gradients, realized active ids, and the flags, which both leave cleared),
    over two views of two cameras."""
    w = get_case("room-60k-392x216")
    runs = []
    for fast in (True, False):
        tr = trainer_for(w, torch_gpu)
        for s, cam in enumerate(w.cameras[:2], start=1):
            tgt = torch_gpu.from_numpy(target_of(w, s - 1).reshape(-1)).cuda()
            if fast:
                tr.step(cam, step=s, version=s, target=tgt)
            else:
                tr.project(cam); tr.visible(); tr.bin_sort(); tr.raster_fwd_l1(tgt, active=True); tr.active_set()
                tr.raster_bwd_pixels(); tr.raster_bwd_project(); tr.adam_publish(s, s, tr.msgs[s & 1]); tr.commit(s)
        torch_gpu.cuda.synchronize()
        assert int(u32(tr.status)[0]) == 0
        A = int(u32(tr.counts[2:3])[0])
        assert A > 0
        runs.append([t.clone() for t in tr.params] + [tr.m.clone(), tr.v.clone()] +
                    [t.clone() for t in tr.replica] + [tr.version.clone(), tr.img.clone(), tr.grad_rows.clone(),
                                                       tr.active.clone(), tr.act_idx[:A].clone()])
    for a, b in zip(*runs):
        assert torch_gpu.equal(a, b)


def test_overlapped_publication_matches_sequential(torch_gpu, orc):
    """Applies on the second stream (deferred into the next view) leave parameters, moments,
    replica and publication versions bit-identical to the one-stream schedule, over several views."""
    w = get_case("room-60k-392x216")
    cam = w.cameras[0]
    runs = []
    for overlap in (False, True):
        tr = trainer_for(w, torch_gpu)
        tr.set_target(target_of(w, 0))
        for s in range(1, 6):
            tr.step(cam, step=s, version=s, overlap=overlap)
        tr.flush_apply()
        torch_gpu.cuda.synchronize()
        assert int(u32(tr.status)[0]) == 0
        runs.append([t.clone() for t in tr.params] + [tr.m.clone(), tr.v.clone()] +
                    [t.clone() for t in tr.replica] + [tr.version.clone()])
    for a, b in zip(*runs):
        assert torch_gpu.equal(a, b)
    # the replica received every step as published: the same fp32 adds as the parameters,
    # so replica and parameters are bit-identical; versions name the last publishing view
    ver = u32(runs[1][-1])
    assert (ver > 0).sum() > 0 and ver.max() == 5
    for p, r in zip(runs[1][:5], runs[1][7:12]):
        assert torch_gpu.equal(p, r)


@pytest.mark.parametrize("case", ["room-60k-392x216", "tiny-10k-256"])
def test_record_table_matches_dense_groups(case, torch_gpu, orc):
    """quat, log_scale and opacity held as column views of one strided head
    table give the dense five-tensor layout's results bit for bit:
    projection, image, gradients, moments, parameters, replica and versions
    over three views, at SH degree 3 and 0; the row strides change only
    addresses, never arithmetic."""
    w = get_case(case)
    runs = []
    for packed in (True, False):
        tr = trainer_for(w, torch_gpu, packed=packed)
        assert (tr.head is not None) == packed
        if packed:
            assert tr.params[1].stride(0) == tr.params[2].stride(0) == tr.params[3].stride(0) == 8
            assert tr.params[1].data_ptr() == tr.params[2].data_ptr() + 16
        for s in range(1, 4):
            k = (s - 1) % len(w.cameras)
            tgt = torch_gpu.from_numpy(target_of(w, k).reshape(-1)).cuda()
            tr.step(w.cameras[k], step=s, version=s, target=tgt)
        tr.flush_apply()
        torch_gpu.cuda.synchronize()
        assert int(u32(tr.status)[0]) == 0
        runs.append([t.clone() for t in tr.params] + [tr.m.clone(), tr.v.clone()] +
                    [t.clone() for t in tr.replica] +
                    [tr.version.clone(), tr.img.clone(), tr.grad_rows.clone(), tr.conic.clone(), tr.rgb.clone()])
    for a, b in zip(*runs):
        assert torch_gpu.equal(a, b)
