"""One training view on the GPU, driven through the C ABI.

`ViewTrainer` owns the device buffers of one primitive pool (parameters,
gradients, Adam moments, projection outputs, pair lists, images, workspaces,
a replica and the publication message) and calls the gs_* entry points in
phase order.  torch is used for allocation, host<->device copies and the
stream only; every step of the path runs in libgsmi's kernels.
"""
from __future__ import annotations

import numpy as np
import torch

from . import gsmi

GROUPS = ("mean", "log_scale", "quat", "opacity", "sh")


def _u32(n, device):
    return torch.zeros(max(1, int(n)), dtype=torch.int32, device=device)


def to_u32(t) -> np.ndarray:
    return t.detach().cpu().numpy().view(np.uint32)


HEAD_OFF = {"quat": 0, "log_scale": 4, "opacity": 7}   # columns of the 32-byte head record
HEAD_LD = 8


def alloc_groups(host, deg, n, device, packed=True):
    """Device parameter groups in GROUPS order from host arrays.

    dense: five tensors.  packed: quat, log_scale and opacity as column views
    of one [n, 8] head table (32 bytes a primitive: the projection reads quat
    and log_scale for every primitive in front of the camera, and the
    optimizer and the commit update the three together, so one segment
    serves them instead of three partial ones), the means and the SH
    coefficients dense ([n, 3]: read for every primitive; [n, 3K]: 192-byte
    rows at SH degree 3, whole 64-byte segments)."""
    k3 = 3 * (deg + 1) ** 2
    cols = [3, 3, 4, 1, k3]
    arrs = [torch.from_numpy(np.ascontiguousarray(a, np.float32).reshape(n, c)) for a, c in zip(host, cols)]
    if not packed:
        return [a.to(device) for a in arrs], None
    head = torch.zeros(max(1, n), HEAD_LD, device=device)
    views = [arrs[0].to(device)]
    for name, a, c in zip(GROUPS[1:4], arrs[1:4], cols[1:4]):
        v = head[:n, HEAD_OFF[name]:HEAD_OFF[name] + c]
        v.copy_(a.to(device))
        views.append(v)
    views.append(arrs[4].to(device))
    return views, head


class ViewTrainer:
    def __init__(self, scene, capacity: int = 0, max_width: int = 0, max_height: int = 0, device="cuda",
                 lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-15, with_replica=True, with_keys=False, packed=True):
        self.dev = torch.device(device)
        self.n = int(scene.n)
        self.deg = int(scene.sh_degree)
        self.K = (self.deg + 1) ** 2
        self.cols = [3, 3, 4, 1, 3 * self.K]
        self.row_len = sum(self.cols)
        # gradient rows, moments and step rows: one row per primitive (moments)
        # or per visible row (gradients, steps), padded to 16/32/64 floats
        self.ld = next(w for w in (16, 32, 64) if w >= self.row_len)
        self.col_off = [sum(self.cols[:i]) for i in range(len(self.cols))]
        self.lr, self.beta1, self.beta2, self.eps = lr, beta1, beta2, eps
        n = self.n
        host = [scene.mean, scene.log_scale, scene.quat, scene.opacity, scene.sh]
        # parameters: quat / log_scale / opacity in one head table beside dense
        # means and SH (packed), or five dense tensors; the replica has the same layout
        self.packed = packed
        self.params, self.head = alloc_groups(host, self.deg, n, self.dev, packed)
        self.grad_rows = torch.zeros(max(1, n), self.ld, device=self.dev)
        self.m = torch.zeros(max(1, n), self.ld, device=self.dev)
        self.v = torch.zeros(max(1, n), self.ld, device=self.dev)
        self.delta_rows = torch.zeros(max(1, n), self.ld, device=self.dev)
        self.replica, self.replica_head = (alloc_groups(host, self.deg, n, self.dev, packed) if with_replica
                                            else (None, None))
        self.version = _u32(n, self.dev)
        # projection
        self.radius = _u32(n, self.dev)
        self.tiles = _u32(n, self.dev)
        self.rect = torch.zeros(max(1, n), 4, dtype=torch.int16, device=self.dev)
        self.depth = torch.zeros(max(1, n), device=self.dev)
        self.mean2d = torch.zeros(max(1, n), 2, device=self.dev)
        self.conic = torch.zeros(max(1, n), 4, device=self.dev)
        self.rgb = torch.zeros(max(1, n), 3, device=self.dev)
        self.clamp = torch.zeros(max(1, n), dtype=torch.uint8, device=self.dev)
        self.active = torch.zeros(max(1, n), dtype=torch.uint8, device=self.dev)
        # True while every active flag is 0: the step's compaction of the flags
        # (active_set) clears them, so the next marking forward needs no fill
        self._active_clean = True
        self.vis_idx = _u32(n, self.dev)
        self.act_idx = _u32(n, self.dev)
        self.counts = _u32(8, self.dev)          # [0] V, [1] M, [2] active count
        self.status = _u32(4, self.dev)
        self.pair_offset = _u32(n, self.dev)
        self.grad2d = torch.zeros(max(1, n), 9, device=self.dev)
        self.grad_norm = torch.zeros(max(1, n), device=self.dev)
        self.loss = torch.zeros(1, device=self.dev)
        self.pair_stats = torch.zeros(4, dtype=torch.int64, device=self.dev)
        self.with_keys = with_keys
        self.ws_vis = torch.zeros(gsmi.gs_workspace_bytes(gsmi.GS_WS_VISIBLE_SET, n), dtype=torch.uint8,
                                  device=self.dev)
        self.capacity = 0
        self.width = self.height = 0
        self.longest_first = True   # raster workgroups take the tiles in gs_bin_sort's dispatch order
        self._set_image(max(1, max_width), max(1, max_height))
        self._set_capacity(max(1, capacity))
        self.scene_s = gsmi.make_scene(n, self.deg, *self.params)
        self.proj_s = gsmi.make_proj(self.radius, self.tiles, self.rect, self.depth, self.mean2d, self.conic,
                                     self.rgb, self.clamp)
        self.adam_arr = gsmi.make_adam_groups([(p, lr) for p in self.params])
        self.params_arr = gsmi.make_groups(self.params)
        self.replica_arr = gsmi.make_groups(self.replica) if with_replica else None
        # the two-slot publication ring: version v is staged in msgs[v & 1]
        self.msgs = [torch.zeros((gsmi.gs_delta_msg_bytes(n, self.row_len, 5) + 15) // 16 * 4, dtype=torch.int32,
                                 device=self.dev) for _ in range(2)]
        self.msg = self.msgs[0]
        self.ring_state = _u32(8, self.dev)
        self.ring = gsmi.make_ring(self.msgs, self.ring_state)
        self.ring_bg = gsmi.make_ring(self.msgs, self.ring_state, background=True)
        self.skip = None            # per-primitive skip metadata of admitted delayed reads (optional)

    # -- buffers -------------------------------------------------------------
    def _set_image(self, w, h):
        if w <= self.width and h <= self.height:
            return
        self.width, self.height = max(w, self.width), max(h, self.height)
        w, h = self.width, self.height
        T = ((w + 15) // 16) * ((h + 15) // 16)
        self.img = torch.zeros(3, h, w, device=self.dev)
        self.final_T = torch.zeros(h, w, device=self.dev)
        self.n_contrib = torch.zeros(h * w, dtype=torch.int32, device=self.dev)
        self.dL = torch.zeros(3, h, w, device=self.dev)
        self.target = torch.zeros(3, h, w, device=self.dev)
        self.ranges = _u32(2 * T, self.dev)
        self.tile_order = _u32(T, self.dev)
        self.ws_loss = torch.zeros(gsmi.gs_workspace_bytes(gsmi.GS_WS_LOSS, 0, 0, w, h), dtype=torch.uint8,
                                   device=self.dev)
        self.ws_fwd_l1 = torch.zeros(gsmi.gs_workspace_bytes(gsmi.GS_WS_RASTER_FWD_L1, 0, 0, w, h),
                                     dtype=torch.uint8, device=self.dev)
        if self.capacity:
            self._set_capacity(self.capacity, force=True)

    def _set_capacity(self, cap, force=False):
        if cap <= self.capacity and not force:
            return
        self.capacity = int(cap)
        self.vals = _u32(cap, self.dev)
        self.pair_emit = _u32(cap, self.dev)
        self.keys = torch.zeros(max(1, cap), dtype=torch.int64, device=self.dev) if self.with_keys else None
        self.ws_sort = torch.zeros(gsmi.gs_workspace_bytes(gsmi.GS_WS_BIN_SORT, self.n, cap, self.width,
                                                           self.height), dtype=torch.uint8, device=self.dev)
        self.ws_bwd = torch.zeros(gsmi.gs_workspace_bytes(gsmi.GS_WS_RASTER_BWD, self.n, cap), dtype=torch.uint8,
                                  device=self.dev)

    def _view(self, cam):
        """Image tensors cropped to this camera (views of the max-size buffers)."""
        w, h = cam.width, cam.height
        self._set_image(w, h)
        return w, h

    # -- phases --------------------------------------------------------------
    def project(self, cam):
        self._view(cam)
        self.cam_c = gsmi.make_camera(cam)
        self.cam = cam
        gsmi.gs_project(self.scene_s, self.cam_c, self.proj_s)

    def visible(self):
        gsmi.gs_visible_set(gsmi.GS_PRED_U32_NONZERO, self.tiles, self.n, self.vis_idx, self.counts[0:1], self.ws_vis)

    def bin_sort(self):
        w, h = self.cam.width, self.cam.height
        gsmi.gs_bin_sort(self.proj_s, self.n, self.vis_idx, self.counts[0:1], w, h, self.capacity, self.vals,
                         self.ranges, self.pair_offset, self.pair_emit, self.keys, self.counts[1:2], self.status,
                         self.ws_sort, tile_order=self.tile_order)

    def _order(self):
        return self.tile_order if self.longest_first else None

    def _img_views(self):
        w, h = self.cam.width, self.cam.height
        hw = w * h
        img = self.img.view(-1)[:3 * hw]
        fT = self.final_T.view(-1)[:hw]
        nc = self.n_contrib[:hw]
        dL = self.dL.view(-1)[:3 * hw]
        tgt = self.target.view(-1)[:3 * hw]
        return img, fT, nc, dL, tgt

    def raster_fwd(self, bg=(0.0, 0.0, 0.0), active=True, stats=False):
        img, fT, nc, _, _ = self._img_views()
        if active:
            self._mark_active()
        gsmi.gs_raster_fwd(self.proj_s, self.n, self.vals, self.ranges, self.cam.width, self.cam.height, bg, img, fT,
                           nc, self.active if active else None, self.pair_stats if stats else None,
                           tile_order=self._order())

    def raster_fwd_l1(self, target=None, bg=(0.0, 0.0, 0.0), active=False):
        """Forward raster and the L1 loss in one pass (target: device tensor of 3*H*W floats, or None for the
        set_target buffer)."""
        img, fT, nc, dL, tgt = self._img_views()
        if active:
            self._mark_active()
        gsmi.gs_raster_fwd_l1(self.proj_s, self.n, self.vals, self.ranges, self.cam.width, self.cam.height, bg,
                              tgt if target is None else target, img, fT, nc, self.active if active else None,
                              self.loss, dL, self.ws_fwd_l1, tile_order=self._order())

    def set_target(self, target_np):
        """Copy a [3,H,W] target into the target buffer (planar, first 3*H*W floats)."""
        a = np.ascontiguousarray(target_np, np.float32)
        self._set_image(a.shape[2], a.shape[1])
        self.target.view(-1)[:a.size].copy_(torch.from_numpy(a.reshape(-1)))

    def loss_l1(self, target=None):
        """target: a device tensor holding 3*H*W floats, or None for the set_target buffer."""
        img, _, _, dL, tgt = self._img_views()
        gsmi.gs_loss_l1(img, tgt if target is None else target, self.cam.width, self.cam.height, self.loss, dL,
                        self.ws_loss)

    def set_dL(self, dL_np):
        """Copy a [3,H,W] upstream image gradient into the dL buffer."""
        a = np.ascontiguousarray(dL_np, np.float32)
        self._set_image(a.shape[2], a.shape[1])
        self.dL.view(-1)[:a.size].copy_(torch.from_numpy(a.reshape(-1)))

    def raster_bwd(self, bg=(0.0, 0.0, 0.0), grad2d=True):
        _, fT, nc, dL, _ = self._img_views()
        gsmi.gs_raster_bwd(self.scene_s, self.cam_c, self.proj_s, self.vals, self.ranges, self.pair_offset,
                           self.pair_emit, self.vis_idx, self.counts[0:1], self.capacity, fT, nc, dL, bg,
                           self.grad_rows, self.ld, self.grad2d if grad2d else None, self.grad_norm, self.ws_bwd,
                           tile_order=self._order())

    def raster_bwd_pixels(self, bg=(0.0, 0.0, 0.0)):
        _, fT, nc, dL, _ = self._img_views()
        gsmi.gs_raster_bwd_pixels(self.proj_s, self.cam_c, self.vals, self.ranges, self.pair_emit, self.capacity, fT,
                                  nc, dL, bg, self.ws_bwd, tile_order=self._order())

    def raster_bwd_project(self, grad2d=False):
        gsmi.gs_raster_bwd_project(self.scene_s, self.cam_c, self.proj_s, self.pair_offset,
                                   self.vis_idx, self.counts[0:1], self.capacity, self.grad_rows, self.ld,
                                   self.grad2d if grad2d else None, self.grad_norm, self.ws_bwd)

    def _mark_active(self):
        """Before a forward that marks active flags: zero them unless the last
        compaction cleared them."""
        if not self._active_clean:
            self.active.zero_()
        self._active_clean = False

    def active_set(self):
        """The realized active set C_i: ids of the flags the last forward set, in
        ascending order (act_idx, count in counts[2]); the compaction also
        clears the flags it reads."""
        gsmi.gs_visible_set(gsmi.GS_PRED_U8_NONZERO_CLEAR, self.active, self.n, self.act_idx, self.counts[2:3],
                            self.ws_vis)
        self._active_clean = True

    def adam(self, step):
        """Sparse Adam over the visible rows; the steps go to delta_rows."""
        gsmi.gs_sparse_adam(self.adam_arr, 5, self.vis_idx, self.counts[0:1], self.n, self.grad_rows, self.ld, self.m,
                            self.v, self.ld, step, self.beta1, self.beta2, self.eps, self.delta_rows, self.ld)

    def adam_publish(self, step, version, msg=None):
        """Sparse Adam over the visible rows, its steps staged as a message."""
        gsmi.gs_sparse_adam_publish(self.adam_arr, 5, self.vis_idx, self.counts[0:1], self.n, self.grad_rows,
                                    self.ld, self.m, self.v, self.ld, step, self.beta1, self.beta2, self.eps,
                                    version, self.msg if msg is None else msg, self.status)

    def pack_params(self, version):
        """Stage the current parameter rows of the visible set (for an overwrite replica)."""
        gsmi.gs_delta_pack(self.vis_idx, self.counts[0:1], self.n, self.params_arr, 5, version, self.msg,
                           self.status)

    # -- task units of several views --------------------------------------------
    _SLOT_ATTRS = ("radius", "tiles", "rect", "depth", "mean2d", "conic", "rgb", "clamp", "vis_idx", "counts",
                   "proj_s")

    def view_slot(self, k):
        """Switch the projection outputs, visible set and counts to those of view k of a task unit (each
        view of a unit keeps its own until the unit's backward is done; pair lists and images are reused)."""
        if not hasattr(self, "_slots"):
            self._slots = [{a: getattr(self, a) for a in self._SLOT_ATTRS}]
        while len(self._slots) <= k:
            n, dev = self.n, self.dev
            d = dict(radius=_u32(n, dev), tiles=_u32(n, dev), rect=torch.zeros(max(1, n), 4, dtype=torch.int16, device=dev),
                     depth=torch.zeros(max(1, n), device=dev), mean2d=torch.zeros(max(1, n), 2, device=dev),
                     conic=torch.zeros(max(1, n), 4, device=dev), rgb=torch.zeros(max(1, n), 3, device=dev),
                     clamp=torch.zeros(max(1, n), dtype=torch.uint8, device=dev), vis_idx=_u32(n, dev),
                     counts=_u32(8, dev))
            d["proj_s"] = gsmi.make_proj(d["radius"], d["tiles"], d["rect"], d["depth"], d["mean2d"], d["conic"],
                                         d["rgb"], d["clamp"])
            self._slots.append(d)
        for a, t in self._slots[k].items():
            setattr(self, a, t)

    def _unit_buffers(self):
        if getattr(self, "union_scope", None) is None:
            self.union_scope = _u32(gsmi.scope_words(self.n), self.dev)
            self.union_idx = _u32(self.n, self.dev)
            self.union_count = _u32(4, self.dev)

    def unit_scopes(self, cams):
        """Project every view of a unit into its own slot, and form the unit's union of visible sets."""
        self._unit_buffers()
        for k, cam in enumerate(cams):
            self.view_slot(k)
            self.project(cam)
            self.visible()
            gsmi.gs_scope_from_pred(gsmi.GS_PRED_U32_NONZERO, self.tiles, self.n, 1 if k else 0, self.union_scope)
        gsmi.gs_visible_set(gsmi.GS_PRED_BITMAP, self.union_scope, self.n, self.union_idx, self.union_count[0:1],
                            self.ws_vis)

    def unit_view_backward(self, k, cam, target=None, dL=None):
        """Render view k of the unit (its slot holds its projection), take its L1 loss (or a given upstream
        gradient) and add its gradient into the unit's rows."""
        self.view_slot(k)
        self.cam, self.cam_c = cam, gsmi.make_camera(cam)
        self.bin_sort()
        if dL is None:
            self.raster_fwd_l1(target)
        else:
            self.raster_fwd(active=False)
            self.set_dL(dL)
        self.raster_bwd_pixels()
        gsmi.gs_raster_bwd_project_accum(self.scene_s, self.cam_c, self.proj_s, self.pair_offset, self.vis_idx,
                                         self.counts[0:1], self.capacity, self.union_idx, self.union_count[0:1],
                                         1 if k == 0 else 0, self.grad_rows, self.ld, self.grad_norm, self.ws_bwd)

    def step_unit(self, cams, step, version, targets=None):
        """One task unit: every view rendered and back-propagated, the gradients summed over the union of the
        views' visible sets, one sparse Adam over that union staged as the message of `version`, and its
        commit to the replica."""
        self.unit_scopes(cams)
        for k, cam in enumerate(cams):
            self.unit_view_backward(k, cam, target=None if targets is None else targets[k])
        self.view_slot(0)
        msg = self.msgs[version & 1]
        gsmi.gs_sparse_adam_publish(self.adam_arr, 5, self.union_idx, self.union_count[0:1], self.n, self.grad_rows,
                                    self.ld, self.m, self.v, self.ld, step, self.beta1, self.beta2, self.eps,
                                    version, msg, self.status)
        self.commit(version)

    # -- host views of compact rows ------------------------------------------
    def rows_by_group(self, t, count):
        """Per-group numpy arrays [count, cols] of a [*, ld] row table (gradients, moments, steps)."""
        a = t[:count].cpu().numpy()
        return [a[:, o:o + c] for o, c in zip(self.col_off, self.cols)]

    def set_state(self, m_groups, v_groups):
        """Fill the moment tables from per-group [n, cols] arrays."""
        m = np.zeros((max(1, self.n), self.ld), np.float32)
        v = np.zeros((max(1, self.n), self.ld), np.float32)
        for o, c, a, b in zip(self.col_off, self.cols, m_groups, v_groups):
            m[:self.n, o:o + c] = a.reshape(self.n, c)
            v[:self.n, o:o + c] = b.reshape(self.n, c)
        self.m.copy_(torch.from_numpy(m))
        self.v.copy_(torch.from_numpy(v))

    def apply(self, mode=gsmi.GS_APPLY_ADD, msg=None):
        gsmi.gs_delta_apply(self.msg if msg is None else msg, self.replica_arr, 5, self.n, self.n, mode,
                            self.version, self.status)

    def commit(self, version, mode=gsmi.GS_APPLY_ADD, background=False):
        """Commit the update staged for `version` (in msgs[version & 1]) into the replica, in version order
        (background: it runs beside compute on the second stream)."""
        gsmi.gs_publish_commit(self.ring_bg if background else self.ring, version, self.replica_arr, 5, self.n,
                               self.n, mode, self.version, self.skip, self.status)

    def enable_overlap(self):
        """Run each view's apply to the replica on a second stream (default
        priority), started once the next view's loss is done on the device, so
        that it runs beside that view's backward raster (arithmetic-bound, light
        on HBM), which reads projection outputs, not the replica.  Messages alternate between two buffers; a view's staging waits
        until the apply that read its buffer two views earlier has finished."""
        if getattr(self, "apply_stream", None) is not None:
            return
        self.apply_stream = torch.cuda.Stream(device=self.dev)
        self.pub_ev = [torch.cuda.Event(), torch.cuda.Event()]
        self.app_ev = [torch.cuda.Event(), torch.cuda.Event()]
        self._pending = None
        self.front_ev = torch.cuda.Event()

    def flush_apply(self, after=None, staged=False):
        """Issue the deferred apply of the last view, if any (overlap mode); it
        starts on the device once its message is staged and, if given, once the
        event `after` has been reached.  staged: `after` was recorded on the
        current stream behind the view's staging, so waiting for it covers the
        staging too (no event of its own: each one is a marker the device
        processes between two kernels)."""
        pend = getattr(self, "_pending", None)
        if pend is None:
            return
        self._pending = None
        version, ev = pend
        k = version & 1
        if not (staged and after is not None):
            # the current stream has issued the view's staging: mark its position
            self.pub_ev[k].record(torch.cuda.current_stream())
        with torch.cuda.stream(self.apply_stream):
            if not (staged and after is not None):
                self.apply_stream.wait_event(self.pub_ev[k])
            if after is not None:
                self.apply_stream.wait_event(after)
            if ev and ev[-2] is not None:
                ev[-2].record(self.apply_stream)
            self.commit(version, background=True)
            self.app_ev[k].record(self.apply_stream)
            if ev and ev[-1] is not None:
                ev[-1].record(self.apply_stream)

    # -- whole view ----------------------------------------------------------
    APPLY_AFTER = 3       # overlap mode: a view's apply starts once the next view's loss is done
    PHASES = ("project", "visible", "bin_sort", "raster_fwd_l1", "raster_bwd_pixels", "raster_bwd_project",
              "adam_publish", "apply")

    def _fwd_step(self, target, active):
        """The step's forward + L1; with active, also the realized active set (flags from the forward,
        compacted into act_idx, its size in counts[2])."""
        self.raster_fwd_l1(target, active=active)
        if active:
            self.active_set()

    def step(self, cam, step, version=1, publish=True, active=True, target=None, events=None, overlap=False):
        """Project, visible set, bin+sort, forward, L1 (and the realized active set: the primitives some
        pixel included, when active), backward, Adam staged as the message of `version` in
        ring slot version & 1, and its commit to the replica (versions must follow each other by one).
        publish=False runs plain Adam (steps to delta_rows) and no commit.
        target: device tensor (3*H*W) or None for the set_target buffer.
        events: optional list of len(PHASES)+1 torch.cuda.Event recorded around the phases (None entries
        are skipped: each recorded event is a marker the device processes between two kernels).
        overlap: apply on the second stream, deferred into the next step (enable_overlap; call
        flush_apply after the last step); events then holds len(PHASES)+2 events: the first
        len(PHASES) bracket the other phases on the current stream, the last two bracket the
        apply on the second stream."""
        ev = events

        def mark(i):
            if ev and ev[i] is not None:
                ev[i].record()

        if overlap and publish:
            self.enable_overlap()
            k = version & 1
            msg = self.msgs[k]
            main = torch.cuda.current_stream()
            calls = (lambda: self.project(cam), self.visible, self.bin_sort,
                     lambda: self._fwd_step(target, active), self.raster_bwd_pixels,
                     self.raster_bwd_project)
            mark(0)
            for i, fn in enumerate(calls):
                fn()
                mark(i + 1)
                if i == self.APPLY_AFTER:
                    # the previous view's apply, once this view reaches that phase on the device
                    self.front_ev.record(main)
                    self.flush_apply(after=self.front_ev, staged=True)
            main.wait_event(self.app_ev[k])          # the commit that read this slot two versions ago
            self.adam_publish(step, version, msg)
            mark(len(calls) + 1)
            self._pending = (version, ev)
            return
        calls = (lambda: self.project(cam), self.visible, self.bin_sort,
                 lambda: self._fwd_step(target, active), self.raster_bwd_pixels, self.raster_bwd_project,
                 (lambda: self.adam_publish(step, version, self.msgs[version & 1])) if publish
                 else (lambda: self.adam(step)),
                 (lambda: self.commit(version)) if publish else (lambda: None))
        mark(0)
        for i, fn in enumerate(calls):
            fn()
            mark(i + 1)

    def ensure_capacity(self, cams, margin=1.25):
        """Size the pair buffers for the given cameras (synchronizes)."""
        need = 0
        for cam in cams:
            self.project(cam)
            self.visible()
            self.status.zero_()
            self.bin_sort()
            torch.cuda.synchronize()
            need = max(need, int(to_u32(self.counts[1:2])[0]))
        if need > self.capacity:
            self._set_capacity(int(need * margin) + 1024)
        self.status.zero_()
        return need

    def host_status(self):
        return to_u32(self.status)
