"""CPU oracle for one 3DGS training view -- TEST INFRASTRUCTURE ONLY.

Only the test suite, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg
of ``bench.py`` may import this package.  It shares no code with the HIP path
(``paper_2607_19893_amd``): the renderer, its derivative and the projection are
in ``gs_oracle.c`` (plain C, fp64 except the fp32 geometry that decides
integers, see that file's header); the L1 loss, Adam and the pending-update
pack/apply are plain numpy below.

What each stage follows:
  * one training view draws a single camera, scores it with an image loss,
    and changes just the primitives that took part (paper Section 2.1); the renderer is
    the cited 3D Gaussian Splatting method;
  * the loss is L1 over all 3*H*W pixel channels;
  * the update is Adam (Kingma & Ba) with torch.optim.Adam's bias-corrected
    form, applied to the rows of the visible set only;
  * pending updates are staged rows of primitive state that a later consumer
    commits (Section 4.3, Shadow Graph steps 3-5): pack gathers the rows of
    an ascending index list into one message, apply adds or copies them into
    a replica and stamps the message version per primitive.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
import subprocess
import time
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "gs_oracle.c")
# GS_ORACLE_LIB names another build of gs_oracle.c to load (the sanitizer
# test's instrumented one); it is used as it is, never rebuilt here.
_LIB_OVERRIDE = os.environ.get("GS_ORACLE_LIB")
_LIB = _LIB_OVERRIDE or os.path.join(_HERE, "liborc.so")
TILE = 16


def build(force: bool = True) -> str:
    """Compile the C part (plain gcc, no FMA contraction, no fast-math)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-fopenmp", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared",
               "-std=gnu11", _SRC, "-o", tmp, "-lm"]
        subprocess.check_call(cmd)
        os.replace(tmp, _LIB)
    return _LIB


class _Cam(ctypes.Structure):
    _fields_ = [("width", ctypes.c_int32), ("height", ctypes.c_int32),
                ("fx", ctypes.c_float), ("fy", ctypes.c_float), ("cx", ctypes.c_float), ("cy", ctypes.c_float),
                ("tan_fovx", ctypes.c_float), ("tan_fovy", ctypes.c_float), ("near_z", ctypes.c_float),
                ("R", ctypes.c_float * 9), ("t", ctypes.c_float * 3), ("campos", ctypes.c_float * 3)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not _LIB_OVERRIDE and (not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC)):
            build(force=True)
        L = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        i32, i64, f64 = ctypes.c_int32, ctypes.c_int64, ctypes.c_double
        L.orc_project.argtypes = [i32, i32, P, P, P, P, P, ctypes.POINTER(_Cam), i32] + [P] * 13
        L.orc_project.restype = None
        L.orc_visible.argtypes = [i32, P, i32, P]
        L.orc_visible.restype = i64
        L.orc_sorted_pairs.argtypes = [i64, P, P, P, i32, i32, P, P, P]
        L.orc_sorted_pairs.restype = i64
        L.orc_render.argtypes = [i64, P, P, P, P, P, P, P, i32, i32, P, P, P, P, P, P, P, P, P]
        L.orc_render.restype = None
        L.orc_render_backward.argtypes = [i64, P, P, P, P, P, P, P, i32, i32, P, P, i32, P, P, f64, f64, f64, P, f64,
                                          P, i32]
        L.orc_render_backward.restype = None
        L.orc_project_backward.argtypes = [i32, i32, P, P, P, P, P, ctypes.POINTER(_Cam), i64, P, P, P,
                                           P, P, P, P, P, P]
        L.orc_project_backward.restype = None
        L.orc_sh_basis.argtypes = [i32, P, i32, P]
        L.orc_sh_basis_grad.argtypes = [i32, P, i32, P]
        L.orc_set_mutation.argtypes = [i32]
        L.orc_num_threads.restype = i32
        _lib = L
    return _lib


def _p(a: np.ndarray):
    assert a.flags["C_CONTIGUOUS"], "oracle arrays must be C-contiguous"
    return a.ctypes.data_as(ctypes.c_void_p)


def _cam(c) -> _Cam:
    cc = _Cam()
    cc.width, cc.height = int(c.width), int(c.height)
    for k in ("fx", "fy", "cx", "cy", "tan_fovx", "tan_fovy", "near_z"):
        setattr(cc, k, float(getattr(c, k)))
    R = np.asarray(c.R, np.float32).reshape(9)
    for i in range(9):
        cc.R[i] = float(R[i])
    for i in range(3):
        cc.t[i] = float(np.float32(c.t[i]))
        cc.campos[i] = float(np.float32(c.campos[i]))
    return cc


def set_mutation(k: int) -> None:
    """Switch on deliberate mistake k in the oracle (0 = off); tests only."""
    lib().orc_set_mutation(int(k))
    global _MUT
    _MUT = int(k)


_MUT = 0


def num_threads() -> int:
    return int(lib().orc_num_threads())


def _f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


# ---------------------------------------------------------------------------
# stages
# ---------------------------------------------------------------------------

@dataclasses.dataclass
class Projection:
    radius: np.ndarray
    tiles: np.ndarray
    rect: np.ndarray
    depth: np.ndarray
    mean2d: np.ndarray       # fp64 (widened fp32 in mode 0)
    conic: np.ndarray
    mean2d_f32: np.ndarray
    conic_f32: np.ndarray
    opacity: np.ndarray      # fp64
    rgb: np.ndarray          # fp64
    clamp: np.ndarray
    clamp_margin: np.ndarray
    jclamp_margin: np.ndarray


def project(scene, cam, mode: int = 0) -> Projection:
    """EWA projection + SH colour of every primitive (mode 0: fp32 geometry, 1: fp64)."""
    n, deg = scene.n, scene.sh_degree
    mean, ls, q, lo, sh = (_f32(scene.mean), _f32(scene.log_scale), _f32(scene.quat),
                           _f32(scene.opacity), _f32(scene.sh))
    out = Projection(radius=np.zeros(n, np.int32), tiles=np.zeros(n, np.uint32), rect=np.zeros((n, 4), np.int32),
                     depth=np.zeros(n, np.float32), mean2d=np.zeros((n, 2)), conic=np.zeros((n, 3)),
                     mean2d_f32=np.zeros((n, 2), np.float32), conic_f32=np.zeros((n, 3), np.float32),
                     opacity=np.zeros(n), rgb=np.zeros((n, 3)), clamp=np.zeros(n, np.uint8),
                     clamp_margin=np.full(n, np.inf), jclamp_margin=np.full(n, np.inf))
    cc = _cam(cam)
    lib().orc_project(n, deg, _p(mean), _p(ls), _p(q), _p(lo), _p(sh), ctypes.byref(cc), int(mode),
                      _p(out.radius), _p(out.tiles), _p(out.rect), _p(out.depth), _p(out.mean2d), _p(out.conic),
                      _p(out.mean2d_f32), _p(out.conic_f32), _p(out.opacity), _p(out.rgb), _p(out.clamp),
                      _p(out.clamp_margin), _p(out.jclamp_margin))
    return out


def visible(src: np.ndarray) -> np.ndarray:
    """Ascending ids whose predicate value is non-zero (u8 or u32 input)."""
    src = np.ascontiguousarray(src)
    eb = src.dtype.itemsize
    assert eb in (1, 4)
    idx = np.zeros(max(1, src.size), np.uint32)
    c = lib().orc_visible(int(src.size), _p(src), eb, _p(idx))
    return idx[:c].copy()


def sorted_pairs(vis: np.ndarray, proj: Projection, cam):
    """All (tile<<32 | depth bits, id) pairs sorted; per-tile [start, end)."""
    vis = np.ascontiguousarray(vis, np.uint32)
    m = int(proj.tiles[vis].astype(np.int64).sum())
    keys = np.zeros(max(1, m), np.uint64)
    vals = np.zeros(max(1, m), np.uint32)
    T = cam.tiles_x * cam.tiles_y
    ranges = np.zeros((T, 2), np.uint32)
    got = lib().orc_sorted_pairs(vis.size, _p(vis), _p(proj.rect), _p(proj.depth), cam.tiles_x, cam.tiles_y,
                                 _p(keys), _p(vals), _p(ranges))
    assert got == m
    return keys[:m].copy(), vals[:m].copy(), ranges


@dataclasses.dataclass
class Render:
    img: np.ndarray          # [3,H,W] fp64
    T_final: np.ndarray
    n_contrib: np.ndarray
    active: np.ndarray
    margin_alpha: np.ndarray
    margin_T: np.ndarray
    n_hits: np.ndarray
    capped_sig: np.ndarray   # [H,W]: sum of (list position + 1) of the included pairs at the 0.99 cap


def render(vis, proj: Projection, cam, bg=(0.0, 0.0, 0.0)) -> Render:
    W, H = cam.width, cam.height
    n = proj.radius.size
    vis = np.ascontiguousarray(vis, np.uint32)
    bg = np.ascontiguousarray(bg, np.float64)
    r = Render(img=np.zeros((3, H, W)), T_final=np.zeros((H, W)), n_contrib=np.zeros((H, W), np.uint32),
               active=np.zeros(n, np.uint8), margin_alpha=np.zeros((H, W)), margin_T=np.zeros((H, W)),
               n_hits=np.zeros((H, W), np.uint32), capped_sig=np.zeros((H, W), np.uint32))
    lib().orc_render(vis.size, _p(vis), _p(proj.rect), _p(proj.depth), _p(proj.mean2d), _p(proj.conic),
                     _p(proj.opacity), _p(proj.rgb), W, H, _p(bg), _p(r.img), _p(r.T_final), _p(r.n_contrib),
                     _p(r.active), _p(r.margin_alpha), _p(r.margin_T), _p(r.n_hits), _p(r.capped_sig))
    return r


# Bands inside which a threshold decision of an fp32 renderer may go either
# way relative to this fp64 oracle, each about twice the largest error of the
# fp32 quantity measured over 20 full-size views of the five workloads:
#   * relative distance of o*exp(-sigma) from 1/255 and from the 0.99 cap:
#     alpha (fp32 opacity, sigma and exponential) within 4.8e-7 relative;
#   * relative distance of T*(1-alpha) from 1e-4: the fp32 transmittance
#     within 7.5e-6 relative (alpha's rounding, amplified by alpha / (1 -
#     alpha) for dense pairs, dominates the per-step rounding of T);
#   * absolute distance |img - target| of the loss sign: pixels within 8e-7.
AMB_ALPHA = 1e-6
AMB_T = 1.5e-5
AMB_CAP = 1e-6
AMB_LOSS = 2e-6


FLAG_AMB_PIXEL = 1   # examined by a pixel whose decisions or loss sign are within the bands
FLAG_NEAR_CAP = 2    # has an included pair within AMB_CAP of the 0.99 alpha cap


def ambiguous_pixels(rnd: "Render", loss_margin=None, amb_alpha=AMB_ALPHA, amb_T=AMB_T, amb_loss=AMB_LOSS):
    """[H,W] mask of pixels whose result (or loss sign) the fp32 kernel may decide differently."""
    amb = (rnd.margin_alpha < amb_alpha) | (rnd.margin_T < amb_T)
    if loss_margin is not None:
        amb |= (np.abs(np.asarray(loss_margin)) < amb_loss).any(axis=0)
    return amb


def render_backward(vis, proj: Projection, cam, dL_dimg, bg=(0.0, 0.0, 0.0), loss_margin=None,
                    amb_alpha=AMB_ALPHA, amb_T=AMB_T, amb_cap=AMB_CAP, amb_loss=AMB_LOSS, want_abs=False,
                    alternative=False):
    """d loss / d(u, v, A, B, C, opacity, rgb) per visible primitive, plus flags
    (FLAG_AMB_PIXEL | FLAG_NEAR_CAP bits per primitive).  alternative=True takes
    the other outcome of every failed decision within the (amb_alpha, amb_T)
    bands: such a pair is included and such a termination test does not stop
    the pixel (what a computation in another precision may do instead)."""
    W, H = cam.width, cam.height
    n = proj.radius.size
    vis = np.ascontiguousarray(vis, np.uint32)
    bg = np.ascontiguousarray(bg, np.float64)
    g = np.ascontiguousarray(dL_dimg, np.float64).reshape(3, H, W)
    grad2d = np.zeros((n, 9))
    flag = np.zeros(n, np.uint8)
    gabs = np.zeros((n, 9)) if want_abs else None
    lm = None if loss_margin is None else np.ascontiguousarray(loss_margin, np.float64).reshape(3, H, W)
    lib().orc_render_backward(vis.size, _p(vis), _p(proj.rect), _p(proj.depth), _p(proj.mean2d), _p(proj.conic),
                              _p(proj.opacity), _p(proj.rgb), W, H, _p(bg), _p(g), n, _p(grad2d), _p(flag),
                              float(amb_alpha), float(amb_T), float(amb_cap),
                              None if lm is None else _p(lm), float(amb_loss), None if gabs is None else _p(gabs),
                              int(bool(alternative)))
    if want_abs:
        return grad2d, flag, gabs
    return grad2d, flag


@dataclasses.dataclass
class Grads:
    """Parameter gradients of the visible rows only: row a belongs to primitive vis[a]."""
    vis: np.ndarray
    mean: np.ndarray
    log_scale: np.ndarray
    quat: np.ndarray
    opacity: np.ndarray
    sh: np.ndarray
    grad_norm: np.ndarray

    def groups(self):
        v = self.vis.size
        return [self.mean.reshape(v, 3), self.log_scale.reshape(v, 3), self.quat.reshape(v, 4),
                self.opacity.reshape(v, 1), self.sh.reshape(v, -1)]

    def full(self, n):
        """Scatter into [n, cols] arrays (zeros elsewhere)."""
        out = []
        for g in self.groups():
            a = np.zeros((n, g.shape[1]))
            a[self.vis.astype(np.int64)] = g
            out.append(a)
        return out


def project_backward(scene, cam, vis, grad2d, proj: Projection) -> Grads:
    n, deg = scene.n, scene.sh_degree
    K = (deg + 1) ** 2
    vis = np.ascontiguousarray(vis, np.uint32)
    v = vis.size
    g = Grads(vis=vis, mean=np.zeros((v, 3)), log_scale=np.zeros((v, 3)), quat=np.zeros((v, 4)), opacity=np.zeros(v),
              sh=np.zeros((v, K, 3)), grad_norm=np.zeros(v))
    cc = _cam(cam)
    lib().orc_project_backward(n, deg, _p(_f32(scene.mean)), _p(_f32(scene.log_scale)), _p(_f32(scene.quat)),
                               _p(_f32(scene.opacity)), _p(_f32(scene.sh)), ctypes.byref(cc), vis.size, _p(vis),
                               _p(np.ascontiguousarray(grad2d, np.float64)), _p(proj.clamp),
                               _p(g.mean), _p(g.log_scale), _p(g.quat), _p(g.opacity), _p(g.sh), _p(g.grad_norm))
    return g


def gradient_magnitudes(scene, cam, vis, grad2d_abs, proj: Projection):
    """Per element of the parameter gradients: sum_c |d g_k / d g2d_c| * S_c, with
    S_c = grad2d_abs[:, c] the sum of |per-pixel terms| of 2D component c.

    The chain from the 2D gradient to the parameters is linear per primitive,
    so its Jacobian columns are the chain applied to unit vectors.  An error
    that is relative to S_c in each 2D component reaches the parameters scaled
    by these magnitudes.  Returns compact rows (one per visible primitive) per
    group, plus the grad_norm entry |S_u| + |S_v|.
    """
    vis = np.ascontiguousarray(vis, np.uint32)
    rows = vis.astype(np.int64)
    acc = None
    for c in range(9):
        g2 = np.zeros_like(grad2d_abs)
        g2[rows, c] = grad2d_abs[rows, c]
        gr = project_backward(scene, cam, vis, g2, proj)
        parts = [np.abs(a) for a in gr.groups()]
        acc = parts if acc is None else [x + y for x, y in zip(acc, parts)]
    return acc, grad2d_abs[rows, 0] + grad2d_abs[rows, 1]


def loss_l1(img, target):
    """L = mean |img - target| over all 3*H*W entries; dL/dimg = sign(img - target) / (3HW).

    img and target are the fp32 images both sides see; the sign is taken on
    their exact difference; the scale 1/(3HW) is the fp32-rounded constant.
    """
    img64 = np.asarray(img, np.float64)
    t64 = np.asarray(target, np.float64)
    d = img64 - t64
    inv = np.float32(1.0 / d.size)
    return float(np.abs(d).mean()), (np.sign(d) * np.float64(inv)), d


def adam_rows(p, g, m, v, step, lr, beta1=0.9, beta2=0.999, eps=1e-15):
    """torch.optim.Adam update of the given rows (all fp64): returns (p, m, v, delta).

    m <- b1 m + (1-b1) g ; v <- b2 v + (1-b2) g^2
    delta = -(lr / (1 - b1^t)) * m / (sqrt(v) / sqrt(1 - b2^t) + eps) ; p <- p + delta
    """
    p, g, m, v = (np.asarray(a, np.float64) for a in (p, g, m, v))
    m = beta1 * m + (1.0 - beta1) * g
    v = beta2 * v + (1.0 - beta2) * g * g
    bc1 = 1.0 - beta1 ** step
    bc2 = 1.0 - beta2 ** step
    if _MUT == 7:
        bc1 = bc2 = 1.0
    delta = -(lr / bc1) * m / (np.sqrt(v) / np.sqrt(bc2) + eps)
    return p + delta, m, v, delta


def adam(p, g, m, v, rows, step, lr, beta1=0.9, beta2=0.999, eps=1e-15):
    """torch.optim.Adam update of rows `rows` of one parameter group (fp64).

    m <- b1 m + (1-b1) g ; v <- b2 v + (1-b2) g^2
    delta = -(lr / (1 - b1^t)) * m / (sqrt(v) / sqrt(1 - b2^t) + eps) ; p <- p + delta
    Rows outside `rows` are returned unchanged.  Returns (p, m, v, delta[rows]).
    """
    p = np.array(p, np.float64, copy=True)
    m = np.array(m, np.float64, copy=True)
    v = np.array(v, np.float64, copy=True)
    rows = np.asarray(rows, np.int64)
    p[rows], m[rows], v[rows], delta = adam_rows(p[rows], np.asarray(g, np.float64)[rows], m[rows], v[rows], step,
                                                 lr, beta1, beta2, eps)
    return p, m, v, delta


MSG_MAGIC = 0x47534D31  # "GSM1"


def delta_message(idx, row_groups, version):
    """Message for ids `idx` whose rows are given (row a of each group belongs to idx[a]).

    Layout: 8 header words (magic, count, version, row_len, n_groups, 0, 0, 0),
    the group widths (padded with zeros to a multiple of 4 words), the K ids,
    zero padding to a 16-byte boundary, then K rows of row_len fp32 values
    (each row = the groups' rows concatenated in group order).
    """
    idx = np.asarray(idx, np.uint32)
    cols = [int(a.shape[1]) for a in row_groups]
    row_len = sum(cols)
    hdr = np.zeros(8, np.uint32)
    hdr[0], hdr[1], hdr[2], hdr[3], hdr[4] = MSG_MAGIC, idx.size, version, row_len, len(row_groups)
    colw = np.zeros(((len(row_groups) + 3) // 4) * 4, np.uint32)
    colw[:len(row_groups)] = cols
    rows = np.concatenate([np.asarray(a, np.float32) for a in row_groups], axis=1) \
        if idx.size else np.zeros((0, row_len), np.float32)
    head = 8 + colw.size + idx.size
    pad = np.zeros((-head) % 4, np.uint32)
    return np.concatenate([hdr, colw, idx, pad, np.ascontiguousarray(rows).reshape(-1).view(np.uint32)])


def delta_pack(idx, groups, version):
    """Gather rows `idx` of full [n, cols] groups into one message (see delta_message)."""
    idx = np.asarray(idx, np.uint32)
    return delta_message(idx, [np.asarray(a, np.float32)[idx.astype(np.int64)] for a in groups], version)


def delta_apply(msg, groups, mode, version_arr=None):
    """ADD (fp32 p += row) or OVERWRITE (copy) every message row into `groups`; stamp versions."""
    msg = np.asarray(msg, np.uint32)
    assert msg[0] == MSG_MAGIC
    K, version, row_len, ng = int(msg[1]), int(msg[2]), int(msg[3]), int(msg[4])
    ncw = ((ng + 3) // 4) * 4
    cols = [int(c) for c in msg[8:8 + ng]]
    off = 8 + ncw
    idx = msg[off:off + K].astype(np.int64)
    r0 = (off + K + 3) // 4 * 4
    rows = msg[r0:r0 + K * row_len].view(np.float32).reshape(K, row_len)
    out = []
    c0 = 0
    for a, c in zip(groups, cols):
        a = np.array(a, np.float32, copy=True)
        r = rows[:, c0:c0 + c]
        if mode == "add":
            a[idx] = (a[idx].astype(np.float64) + r.astype(np.float64)).astype(np.float32)
        else:
            a[idx] = r
        out.append(a)
        c0 += c
    if version_arr is not None:
        version_arr = np.array(version_arr, np.uint32, copy=True)
        version_arr[idx] = version
    return out, version_arr


# ---------------------------------------------------------------------------
# one whole view
# ---------------------------------------------------------------------------

@dataclasses.dataclass
class ViewResult:
    proj: Projection
    vis: np.ndarray
    keys: Optional[np.ndarray]
    vals: Optional[np.ndarray]
    ranges: Optional[np.ndarray]
    render: Render
    loss: float
    dL_dimg: np.ndarray
    loss_margin: np.ndarray
    grad2d: np.ndarray
    flag: np.ndarray
    grads: Grads
    new_params: list      # visible rows only (row a = primitive vis[a]), fp64
    new_m: list
    new_v: list
    deltas: list
    msg: Optional[np.ndarray]
    times: dict


def train_view(scene, cam, target, m_groups, v_groups, step, lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-15,
               with_pairs=True, with_msg=True, version=1, dL_dimg=None):
    """Projection -> visible set -> pairs -> render -> L1 -> backward -> Adam -> pack (one view).

    The loss sign is taken on the fp32-rounded rendered image (the precision
    the kernel decides it in); pass dL_dimg to bypass the loss.
    """
    tm = {}
    t0 = time.perf_counter()
    proj = project(scene, cam, 0)
    tm["project"] = time.perf_counter() - t0
    t0 = time.perf_counter()
    vis = visible(proj.tiles)
    tm["visible"] = time.perf_counter() - t0
    keys = vals = ranges = None
    if with_pairs:
        t0 = time.perf_counter()
        keys, vals, ranges = sorted_pairs(vis, proj, cam)
        tm["pairs"] = time.perf_counter() - t0
    t0 = time.perf_counter()
    rnd = render(vis, proj, cam)
    tm["render"] = time.perf_counter() - t0
    if dL_dimg is None:
        loss, dL, diff = loss_l1(rnd.img.astype(np.float32), target)
        lm = diff
    else:
        loss, dL, lm = float("nan"), np.asarray(dL_dimg, np.float64), None
    t0 = time.perf_counter()
    grad2d, flag = render_backward(vis, proj, cam, dL, loss_margin=lm)
    tm["render_backward"] = time.perf_counter() - t0
    t0 = time.perf_counter()
    grads = project_backward(scene, cam, vis, grad2d, proj)
    tm["project_backward"] = time.perf_counter() - t0
    t0 = time.perf_counter()
    params = [a for _, a in scene.groups()]
    rows = vis.astype(np.int64)
    newp, newm, newv, deltas = [], [], [], []
    for p, g, m, v in zip(params, grads.groups(), m_groups, v_groups):
        pn, mn, vn, d = adam_rows(p[rows], g, m[rows], v[rows], step, lr, beta1, beta2, eps)
        newp.append(pn); newm.append(mn); newv.append(vn); deltas.append(d)
    tm["adam"] = time.perf_counter() - t0
    msg = None
    if with_msg:
        t0 = time.perf_counter()
        msg = delta_message(vis, [d.astype(np.float32) for d in deltas], version)
        tm["pack"] = time.perf_counter() - t0
    return ViewResult(proj, vis, keys, vals, ranges, rnd, loss, dL, lm, grad2d, flag, grads, newp, newm, newv,
                      deltas, msg, tm)


# ---------------------------------------------------------------------------
# primitive scopes: hazard sets and throughput-first admission (Section 4.3)
# ---------------------------------------------------------------------------
# Scopes are sets of primitive ids (Section 2.1: the dependency unit is the
# primitive index).  Here they are plain Python sets built from id arrays; the
# results are returned as ascending uint32 arrays.

GATE_NO_DELAY = 0        # D+ is empty: there is no RAW wait to admit
GATE_ADMIT = 1           # both admission tests pass: B may read the last published versions
GATE_WAIT_RHO = 2        # |D+| / |R+(B)| > tau
GATE_WAIT_NO_ACTIVE = 3  # C_A is empty: the gradient gate cannot be evaluated
GATE_WAIT_MISSING = 4    # a delayed primitive has no producer evidence
GATE_WAIT_SECOND = 5     # a delayed primitive already carries another producer's skipped update
GATE_WAIT_GRADIENT = 6   # a delayed primitive's ||g_A|| exceeds tau times the active-set mean


def _idset(a):
    return set(int(x) for x in np.asarray(a, np.int64).reshape(-1))


def _sorted_u32(s):
    return np.array(sorted(s), dtype=np.uint32)


def scope_conflicts(RA, WA, RB, WB):
    """Quality-first primitive-state hazards between an earlier unit A and a
    later unit B (Section 4.3, "Quality-first path"), from their conservative
    read and update scopes:
        C_WAW = W+(B) & W+(A)
        C_RAW = (R+(B) - W+(B)) & W+(A)
        C_WAR = W+(B) & (R+(A) - W+(A))
    Returns (waw, raw, war) as ascending id arrays."""
    RA, WA, RB, WB = (_idset(x) for x in (RA, WA, RB, WB))
    waw = WB & WA
    raw = (RB - WB) & WA
    war = WB & (RA - WA)
    if _MUT == 8:
        raw = RB & WA                      # planted: B's own update scope not excluded
    if _MUT == 9:
        war = WA & (RB - WB)               # planted: A and B swapped
    return _sorted_u32(waw), _sorted_u32(raw), _sorted_u32(war)


@dataclasses.dataclass
class GateResult:
    admit: int
    reason: int
    n_delayed: int
    n_read: int
    n_active: int
    n_missing: int
    n_second: int
    rho: float
    mean_g: float
    max_g: float
    threshold: float


def admission_gate(RB, D, CA, g, tau, evidence=None, skip=None, producer_version=0):
    """Throughput-first admission of a delayed read (Section 4.3,
    "Throughput-first path") for the delayed-read set D = C_RAW(A, B).

      * D empty (which includes an empty R+(B)): nothing to admit (GATE_NO_DELAY);
      * rho = |D| / |R+(B)| must not exceed tau;
      * the gradient gate needs a non-empty active set C_A and producer
        evidence for every delayed primitive (`evidence`: the ids whose
        ||g_A|| the producer reported; None means C_A);
      * publication metadata (`skip`, per primitive: the version of a pending
        update an admitted read has already skipped, 0 if none) must show no
        other producer's skipped update on a delayed primitive, so a read
        never passes over more than one pending (unpublished) update;
      * every delayed p needs ||g_A(p)|| <= tau * (1/|C_A|) sum_{q in C_A} ||g_A(q)||.
    Tests are taken in the order listed; the first that fails names the reason.
    g is indexed by primitive id.  The sum is exact (math.fsum), the mean and
    the threshold are then rounded to fp64 once each.

    Returns (GateResult, skip'): on admission skip'[p] = producer_version for
    every p in D; otherwise skip' equals skip."""
    import math
    RB, D, CA = _idset(RB), _idset(D), _idset(CA)
    E = CA if evidence is None else _idset(evidence)
    g = np.asarray(g, np.float32)
    nD, nR, nC = len(D), len(RB), len(CA)
    rho = (nD / nR) if nR > 0 else 0.0
    missing = sum(1 for p in D if p not in E)
    second = 0
    if skip is not None:
        second = sum(1 for p in D if int(skip[p]) != 0 and int(skip[p]) != int(producer_version))
    sum_g = math.fsum(float(g[q]) for q in CA)
    mean_g = sum_g / nC if nC > 0 else 0.0
    if _MUT == 10 and nD > 0:
        mean_g = math.fsum(float(g[q]) for q in D) / nD     # planted: mean over the delayed set
    thr = float(tau) * mean_g
    max_g = max((float(g[p]) for p in D), default=0.0)
    if nD == 0:
        reason = GATE_NO_DELAY
    elif rho > tau or (_MUT == 11 and rho >= tau):
        reason = GATE_WAIT_RHO
    elif nC == 0:
        reason = GATE_WAIT_NO_ACTIVE
    elif missing:
        reason = GATE_WAIT_MISSING
    elif second and _MUT != 12:
        reason = GATE_WAIT_SECOND
    elif max_g > thr:
        reason = GATE_WAIT_GRADIENT
    else:
        reason = GATE_ADMIT
    admit = 1 if reason in (GATE_NO_DELAY, GATE_ADMIT) else 0
    new_skip = None
    if skip is not None:
        new_skip = np.array(skip, np.uint32, copy=True)
        if reason == GATE_ADMIT:
            for p in D:
                new_skip[p] = producer_version
    return GateResult(admit, reason, nD, nR, nC, missing, second, rho, mean_g, max_g, thr), new_skip


def scope_bitmap(ids, n):
    """A set of ids as uint32 words, bit (i & 31) of word (i >> 5), ids >= n
    dropped (the scope layout of the C boundary; used to compare with it)."""
    ids = np.asarray(ids, np.int64).reshape(-1)
    ids = ids[(ids >= 0) & (ids < n)]
    words = np.zeros((int(n) + 31) // 32, np.uint32)
    np.bitwise_or.at(words, ids >> 5, (np.uint32(1) << (ids & 31).astype(np.uint32)))
    return words


def scope_ids(words, n):
    """Inverse of scope_bitmap: the ascending ids whose bit is set (ids < n)."""
    words = np.asarray(words, np.uint32)
    bits = ((words[:, None] >> np.arange(32, dtype=np.uint32)[None, :]) & 1).reshape(-1)
    return np.flatnonzero(bits[:int(n)]).astype(np.uint32)


# ---------------------------------------------------------------------------
# versioned two-slot staging (Section 4.3, Shadow Graph steps 3-4 and the
# per-primitive publication metadata of the throughput-first path)
# ---------------------------------------------------------------------------

COMMIT_OK = 0
COMMIT_MISMATCH = 4      # the slot does not hold a well-formed message of this version for these groups
COMMIT_ORDER = 8         # the version is not the one after the last committed version


def parse_message(msg):
    """(K, version, row_len, cols, ids, rows) of a message (see delta_message)."""
    msg = np.asarray(msg, np.uint32)
    K, version, row_len, ng = int(msg[1]), int(msg[2]), int(msg[3]), int(msg[4])
    ncw = ((ng + 3) // 4) * 4
    cols = [int(c) for c in msg[8:8 + ng]]
    off = 8 + ncw
    ids = msg[off:off + K].astype(np.int64)
    r0 = (off + K + 3) // 4 * 4
    rows = msg[r0:r0 + K * row_len].view(np.float32).reshape(K, row_len)
    return K, version, row_len, cols, ids, rows


def publish_commit(ring_state, slots, version, groups, mode, prim_version, skip=None, n_rows=None):
    """Commit the update staged for `version` in slot (version & 1) of a
    two-slot ring into a replica (Shadow Graph step 4: the produced slot is
    committed once its publication condition holds).

      * the slot must hold a message with this version, the replica's group
        widths and ids below n_rows, else COMMIT_MISMATCH;
      * versions are committed in order: ring_state[0] (the last committed
        version) must be version - 1, else COMMIT_ORDER;
      * a row is applied (ADD: one fp32 add; OVERWRITE: copy) only if the
        primitive's published version is older than `version`, and then
        stamped with it; rows already at or past it are left as they are;
      * skip metadata naming this version is cleared for every row of the
        message: the update a delayed read skipped is now published.
    On any failure nothing changes.  Returns (groups, prim_version, skip,
    ring_state, flags) with ring_state = [committed, applied, left, 0]."""
    ring_state = np.array(ring_state, np.uint32, copy=True)
    msg = np.asarray(slots[version & 1], np.uint32)
    n_rows = int(groups[0].shape[0]) if n_rows is None else int(n_rows)
    ok = int(msg[0]) == MSG_MAGIC and int(msg[2]) == int(version)
    if ok:
        K, v, row_len, cols, ids, rows = parse_message(msg)
        ok = cols == [int(a.shape[1]) for a in groups] and bool(np.all(ids < n_rows))
    if not ok:
        return groups, prim_version, skip, ring_state, COMMIT_MISMATCH
    if int(ring_state[0]) + 1 != int(version):
        return groups, prim_version, skip, ring_state, COMMIT_ORDER
    prim_version = np.array(prim_version, np.uint32, copy=True)
    newer = prim_version[ids] < version
    if _MUT == 14:
        newer = np.ones(ids.size, bool)        # planted: published versions not checked
    take = ids[newer]
    out = []
    c0 = 0
    for a, c in zip(groups, cols):
        a = np.array(a, np.float32, copy=True)
        r = rows[newer, c0:c0 + c]
        if mode == "add":
            a[take] = (a[take].astype(np.float64) + r.astype(np.float64)).astype(np.float32)
        else:
            a[take] = r
        out.append(a)
        c0 += c
    prim_version[take] = version
    if skip is not None:
        skip = np.array(skip, np.uint32, copy=True)
        hit = ids[skip[ids] == version]
        if _MUT != 13:                         # planted (13): markers never cleared
            skip[hit] = 0
    ring_state[0] = version
    ring_state[1] = int(newer.sum())
    ring_state[2] = int((~newer).sum())
    return out, prim_version, skip, ring_state, COMMIT_OK


# ---------------------------------------------------------------------------
# a task unit of several views (Section 2.1)
# ---------------------------------------------------------------------------

@dataclasses.dataclass
class UnitResult:
    union: np.ndarray          # ascending union of the views' visible sets
    grads: list                # per group [|union|, cols] fp64: the views' gradients summed
    grad_norm: np.ndarray      # [n]: sum over the views of |dL/d(u,v)| (visible views only)
    views: list                # per view: (vis, proj, render, dL_dimg, loss, flag)
    new_params: list           # union rows, fp64
    new_m: list
    new_v: list
    deltas: list
    msg: Optional[np.ndarray]


def unit_gradients(scene, cams, targets=None, dL_list=None, mode=0):
    """Gradient of a task unit: the sum over its views of each view's loss
    gradient (a task unit groups a few training views, and its active
    set and gradient evidence are the union and accumulation over its views,
    Section 2.1).  Each view's loss is the L1 mean of that view (targets), or
    its upstream image gradient is given (dL_list).  Rows are those of the
    ascending union of the views' visible sets.  mode selects the projection's
    geometry (0: the fixed-order fp32 geometry, 1: fp64).  Returns (union,
    grads per group by union row, grad_norm by id, per-view records)."""
    n = scene.n
    views = []
    for k, cam in enumerate(cams):
        proj = project(scene, cam, mode)
        vis = visible(proj.tiles)
        rnd = render(vis, proj, cam)
        if dL_list is None:
            loss, dL, lm = loss_l1(rnd.img.astype(np.float32), targets[k])
        else:
            loss, dL, lm = float("nan"), np.asarray(dL_list[k], np.float64), None
        g2, flag = render_backward(vis, proj, cam, dL, loss_margin=lm)
        gr = project_backward(scene, cam, vis, g2, proj)
        views.append((vis, proj, rnd, dL, loss, flag, gr, lm))
    union = np.unique(np.concatenate([v[0] for v in views]).astype(np.int64)).astype(np.uint32) \
        if views else np.zeros(0, np.uint32)
    cols = [3, 3, 4, 1, 3 * (scene.sh_degree + 1) ** 2]
    grads = [np.zeros((union.size, c)) for c in cols]
    gnorm = np.zeros(n)
    for vis, proj, rnd, dL, loss, flag, gr, lm in views:
        rows = np.searchsorted(union, vis)
        if _MUT == 15:
            rows = np.arange(vis.size)             # planted: view rows taken as union rows
        for G, g in zip(grads, gr.groups()):
            G[rows] += g
        gnorm[vis.astype(np.int64)] += gr.grad_norm
    return union, grads, gnorm, views


def train_unit(scene, cams, targets, m_groups, v_groups, step, lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-15,
               version=1, dL_list=None, with_msg=True):
    """A task unit: the views' gradients summed over the union of their visible
    sets, then one Adam step over that union (rows outside it untouched) and
    its steps staged as one message."""
    union, grads, gnorm, views = unit_gradients(scene, cams, targets, dL_list)
    rows = union.astype(np.int64)
    params = [a.reshape(scene.n, -1) for _, a in scene.groups()]
    newp, newm, newv, deltas = [], [], [], []
    for p, g, m, v in zip(params, grads, m_groups, v_groups):
        pn, mn, vn, d = adam_rows(p[rows], g, np.asarray(m).reshape(scene.n, -1)[rows],
                                  np.asarray(v).reshape(scene.n, -1)[rows], step, lr, beta1, beta2, eps)
        newp.append(pn); newm.append(mn); newv.append(vn); deltas.append(d)
    msg = delta_message(union, [d.astype(np.float32) for d in deltas], version) if with_msg else None
    return UnitResult(union, grads, gnorm, [v[:6] for v in views], newp, newm, newv, deltas, msg)


# the ahead-of-time planner (Sections 4.1.1 and 4.2)
from .planner import (RLG, Partition, Schedule, group_cycle, jaccard, lp_partition, rlg_build,  # noqa: E402
                      score, sds_order, track_sets)
