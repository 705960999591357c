"""Thin ctypes binding of libgsmi (include/gsmi.h): same names, argument
marshalling only.  Tensors are torch tensors on the GPU; their data pointers
and the current HIP stream are handed to the C ABI unchanged.

Importing this module loads the in-tree libgsmi.so and fails loudly if it is
missing; there is no CPU fallback.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libgsmi.so")

if not os.path.exists(LIB_PATH):
    raise ImportError("libgsmi.so is not built (run __graft_entry__.build() or "
                      "python -m paper_2607_19893_amd.build); there is no fallback path")

_lib = ctypes.CDLL(LIB_PATH)

P = ctypes.c_void_p
i32, u32, i64, f32, sz = ctypes.c_int32, ctypes.c_uint32, ctypes.c_int64, ctypes.c_float, ctypes.c_size_t

GS_OK, GS_ERR_INVALID_ARG, GS_ERR_UNSUPPORTED, GS_ERR_WORKSPACE, GS_ERR_HIP = range(5)
GS_WS_VISIBLE_SET, GS_WS_BIN_SORT, GS_WS_RASTER_BWD, GS_WS_LOSS, GS_WS_SCOPE, GS_WS_RASTER_FWD_L1 = 1, 2, 3, 4, 5, 6
GS_PRED_U32_NONZERO, GS_PRED_U8_NONZERO, GS_PRED_BITMAP, GS_PRED_U8_NONZERO_CLEAR = 0, 1, 2, 3
(GS_GATE_NO_DELAY, GS_GATE_ADMIT, GS_GATE_WAIT_RHO, GS_GATE_WAIT_NO_ACTIVE, GS_GATE_WAIT_MISSING, GS_GATE_WAIT_SECOND,
 GS_GATE_WAIT_GRADIENT) = range(7)
GS_APPLY_ADD, GS_APPLY_OVERWRITE = 0, 1
GS_DEV_PAIR_OVERFLOW, GS_DEV_MSG_OVERFLOW, GS_DEV_MSG_MISMATCH, GS_DEV_MSG_ORDER = 1, 2, 4, 8
GS_MSG_MAGIC = 0x47534D31
GS_MAX_GROUPS = 8


class gs_scene(ctypes.Structure):
    _fields_ = [("n", i32), ("sh_degree", i32), ("mean", P), ("log_scale", P), ("quat", P), ("opacity", P),
                ("sh", P), ("ld_mean", i32), ("ld_log_scale", i32), ("ld_quat", i32), ("ld_opacity", i32),
                ("ld_sh", i32)]


class gs_camera(ctypes.Structure):
    _fields_ = [("width", i32), ("height", i32), ("fx", f32), ("fy", f32), ("cx", f32), ("cy", f32),
                ("tan_fovx", f32), ("tan_fovy", f32), ("near_z", f32), ("R", f32 * 9), ("t", f32 * 3),
                ("campos", f32 * 3)]


class gs_proj(ctypes.Structure):
    _fields_ = [("radius", P), ("tiles", P), ("rect", P), ("depth", P), ("mean2d", P), ("conic_opacity", P),
                ("rgb", P), ("clamp", P)]


class gs_adam_group(ctypes.Structure):
    _fields_ = [("p", P), ("cols", i32), ("lr", f32), ("ld", i32)]


class gs_group(ctypes.Structure):
    _fields_ = [("ptr", P), ("cols", i32), ("ld", i32)]


class gs_ring(ctypes.Structure):
    _fields_ = [("slot", P * 2), ("slot_bytes", sz), ("state", P), ("background", i32)]


class gs_gate_args(ctypes.Structure):
    _fields_ = [("active", P), ("evidence", P), ("g", P), ("skip", P), ("producer_version", u32),
                ("tau", ctypes.c_double)]


class gs_gate_result(ctypes.Structure):
    """Mirror of the device-side result record (64 bytes)."""
    _fields_ = [("admit", u32), ("reason", u32), ("n_read", u32), ("n_delayed", u32), ("n_active", u32),
                ("n_missing", u32), ("n_second", u32), ("reserved", u32), ("rho", ctypes.c_double),
                ("mean_g", ctypes.c_double), ("max_g", ctypes.c_double), ("threshold", ctypes.c_double)]


def scope_words(n) -> int:
    return (int(n) + 31) // 32


_lib.gs_abi_version.restype = i32
# the structs above mirror this version of the header; a library built from
# another one would read them with a different layout
ABI_VERSION = 4
if _lib.gs_abi_version() != ABI_VERSION:
    raise ImportError("libgsmi ABI version %d, binding expects %d: rebuild the library"
                      % (_lib.gs_abi_version(), ABI_VERSION))
_lib.gs_status_string.restype = ctypes.c_char_p
_lib.gs_status_string.argtypes = [i32]
_lib.gs_last_error.restype = ctypes.c_char_p
_lib.gs_workspace_bytes.restype = sz
_lib.gs_workspace_bytes.argtypes = [i32, i32, u32, i32, i32]
_lib.gs_delta_msg_bytes.restype = sz
_lib.gs_delta_msg_bytes.argtypes = [u32, i32, i32]
_lib.gs_project.argtypes = [ctypes.POINTER(gs_scene), ctypes.POINTER(gs_camera), ctypes.POINTER(gs_proj), P]
_lib.gs_visible_set.argtypes = [i32, P, i32, P, P, P, sz, P]
_lib.gs_visible_set_noalloc.argtypes = [i32, P, i32, P, P, P]
_lib.gs_bin_sort.argtypes = [ctypes.POINTER(gs_proj), i32, P, P, i32, i32, u32, P, P, P, P, P, P, P, P, P, sz, P]
_lib.gs_raster_fwd.argtypes = [ctypes.POINTER(gs_proj), i32, P, P, P, i32, i32, P, P, P, P, P, P, P]
_lib.gs_loss_l1.argtypes = [P, P, i32, i32, P, P, P, sz, P]
_lib.gs_raster_fwd_l1.argtypes = [ctypes.POINTER(gs_proj), i32, P, P, P, i32, i32, P, P, P, P, P, P, P, P, P, sz, P]
_lib.gs_raster_bwd.argtypes = [ctypes.POINTER(gs_scene), ctypes.POINTER(gs_camera), ctypes.POINTER(gs_proj), P, P, P,
                               P, P, P, P, u32, P, P, P, P, P, i32, P, P, P, sz, P]
_lib.gs_raster_bwd_pixels.argtypes = [ctypes.POINTER(gs_proj), ctypes.POINTER(gs_camera), P, P, P, P, u32, P, P, P,
                                      P, P, sz, P]
_lib.gs_raster_bwd_project.argtypes = [ctypes.POINTER(gs_scene), ctypes.POINTER(gs_camera), ctypes.POINTER(gs_proj),
                                       P, P, P, u32, P, i32, P, P, P, sz, P]
_lib.gs_raster_bwd_project_accum.argtypes = [ctypes.POINTER(gs_scene), ctypes.POINTER(gs_camera),
                                             ctypes.POINTER(gs_proj), P, P, P, u32, P, P, i32, P, i32, P, P, sz, P]
_lib.gs_sparse_adam.argtypes = [ctypes.POINTER(gs_adam_group), i32, P, P, i32, P, i32, P, P, i32, i32,
                                ctypes.c_double, ctypes.c_double, ctypes.c_double, P, i32, P]
_lib.gs_sparse_adam_publish.argtypes = [ctypes.POINTER(gs_adam_group), i32, P, P, i32, P, i32, P, P, i32, i32,
                                        ctypes.c_double, ctypes.c_double, ctypes.c_double, u32, P, sz, P, P]
_lib.gs_delta_pack.argtypes = [P, P, i32, ctypes.POINTER(gs_group), i32, u32, P, sz, P, P]
_lib.gs_delta_apply.argtypes = [P, sz, ctypes.POINTER(gs_group), i32, i32, i32, i32, P, P, P]
_lib.gs_publish_commit.argtypes = [ctypes.POINTER(gs_ring), u32, ctypes.POINTER(gs_group), i32, i32, i32, i32, P, P,
                                   P, P]
_lib.gs_scope_from_ids.argtypes = [P, P, i32, i32, i32, P, P]
_lib.gs_scope_from_pred.argtypes = [i32, P, i32, i32, P, P]
_lib.gs_scope_conflicts.argtypes = [P, P, P, P, i32, P, P, P, P, P, P, P, P, sz, P]
_lib.gs_admission_gate.argtypes = [P, P, ctypes.POINTER(gs_gate_args), i32, P, P, sz, P]
_lib.gs_rlg_build.argtypes = [i32, i32, P, P, i32, i32, P, P, P, ctypes.c_int64, P]
_lib.gs_lp_partition.argtypes = [i32, P, P, P, P, i32, i32, P, P, P]
_lib.gs_sds_order.argtypes = [i32, P, i32, P, P, P, P, i32, P, P, P, P, P, P]
for _name in ("gs_project", "gs_visible_set", "gs_visible_set_noalloc", "gs_bin_sort", "gs_raster_fwd", "gs_loss_l1", "gs_raster_bwd",
              "gs_raster_bwd_pixels", "gs_raster_bwd_project", "gs_sparse_adam", "gs_sparse_adam_publish",
              "gs_delta_pack", "gs_delta_apply", "gs_scope_from_ids", "gs_scope_from_pred", "gs_scope_conflicts",
              "gs_admission_gate", "gs_publish_commit", "gs_raster_bwd_project_accum", "gs_raster_fwd_l1",
              "gs_rlg_build", "gs_lp_partition", "gs_sds_order"):
    getattr(_lib, _name).restype = i32

EXPORTS = ["gs_abi_version", "gs_status_string", "gs_last_error", "gs_workspace_bytes", "gs_delta_msg_bytes",
           "gs_project", "gs_visible_set", "gs_visible_set_noalloc", "gs_bin_sort", "gs_raster_fwd", "gs_loss_l1",
           "gs_raster_bwd", "gs_raster_bwd_pixels", "gs_raster_bwd_project", "gs_sparse_adam", "gs_sparse_adam_publish",
           "gs_delta_pack", "gs_delta_apply", "gs_scope_from_ids", "gs_scope_from_pred", "gs_scope_conflicts",
           "gs_admission_gate", "gs_publish_commit", "gs_raster_bwd_project_accum", "gs_raster_fwd_l1",
           "gs_rlg_build", "gs_lp_partition", "gs_sds_order"]


class GsmiError(RuntimeError):
    def __init__(self, fn, status):
        self.status = status
        msg = _lib.gs_last_error().decode()
        super().__init__("%s -> %s: %s" % (fn, _lib.gs_status_string(status).decode(), msg))


def _check(fn, st):
    if st != GS_OK:
        raise GsmiError(fn, st)
    return st


def ptr(t):
    """Device pointer of a tensor (or None)."""
    if t is None:
        return None
    return ctypes.c_void_p(t.data_ptr())


def current_stream():
    import torch
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def make_camera(cam) -> gs_camera:
    c = gs_camera()
    c.width, c.height = int(cam.width), int(cam.height)
    for k in ("fx", "fy", "cx", "cy", "tan_fovx", "tan_fovy", "near_z"):
        setattr(c, k, float(getattr(cam, k)))
    R = [float(x) for x in cam.R.reshape(9)]
    for i in range(9):
        c.R[i] = R[i]
    for i in range(3):
        c.t[i] = float(cam.t[i])
        c.campos[i] = float(cam.campos[i])
    return c


def row_stride(t) -> int:
    """Floats between consecutive rows of a parameter group: the first-dim
    stride of a tensor whose rows are contiguous (a dense tensor or a column
    range of a wider table)."""
    if t is None or t.numel() == 0:
        return 0
    per_row = t[0].numel() if t.dim() > 1 else 1
    if t.dim() > 1 and not t[0].is_contiguous():
        raise ValueError("rows of a parameter group must be contiguous")
    return int(t.stride(0)) if t.shape[0] > 1 else per_row


def make_scene(n, sh_degree, mean, log_scale, quat, opacity, sh) -> gs_scene:
    return gs_scene(int(n), int(sh_degree), ptr(mean), ptr(log_scale), ptr(quat), ptr(opacity), ptr(sh),
                    row_stride(mean), row_stride(log_scale), row_stride(quat), row_stride(opacity), row_stride(sh))


def make_proj(radius, tiles, rect, depth, mean2d, conic_opacity, rgb, clamp) -> gs_proj:
    return gs_proj(ptr(radius), ptr(tiles), ptr(rect), ptr(depth), ptr(mean2d), ptr(conic_opacity), ptr(rgb),
                   ptr(clamp))


# ---- the entry points -------------------------------------------------------

def gs_abi_version() -> int:
    return int(_lib.gs_abi_version())


def gs_status_string(s: int) -> str:
    return _lib.gs_status_string(int(s)).decode()


def gs_last_error() -> str:
    return _lib.gs_last_error().decode()


def gs_workspace_bytes(which, n, capacity=0, width=0, height=0) -> int:
    return int(_lib.gs_workspace_bytes(int(which), int(n), int(capacity), int(width), int(height)))


def gs_delta_msg_bytes(count, row_len, n_groups) -> int:
    return int(_lib.gs_delta_msg_bytes(int(count), int(row_len), int(n_groups)))


def gs_project(scene: gs_scene, cam: gs_camera, proj: gs_proj, stream=None):
    return _check("gs_project", _lib.gs_project(ctypes.byref(scene), ctypes.byref(cam), ctypes.byref(proj),
                                                stream if stream is not None else current_stream()))


def gs_visible_set(kind, src, n, out_idx, out_count, ws, stream=None):
    return _check("gs_visible_set", _lib.gs_visible_set(int(kind), ptr(src), int(n), ptr(out_idx), ptr(out_count),
                                                        ptr(ws), ws.numel() * ws.element_size() if ws is not None else 0,
                                                        stream if stream is not None else current_stream()))


def gs_visible_set_noalloc(kind, src, n, out_idx, out_count, stream=None):
    return _check("gs_visible_set_noalloc",
                  _lib.gs_visible_set_noalloc(int(kind), ptr(src), int(n), ptr(out_idx), ptr(out_count),
                                              stream if stream is not None else current_stream()))


GS_NOALLOC_SCRATCH_BYTES = 262144
GS_NOALLOC_MAX_N = 134215680


def gs_bin_sort(proj: gs_proj, n, vis_idx, vis_count, width, height, capacity, vals, ranges, pair_offset,
                pair_emit, keys, num_pairs, status, ws, stream=None, tile_order=None):
    return _check("gs_bin_sort", _lib.gs_bin_sort(ctypes.byref(proj), int(n), ptr(vis_idx), ptr(vis_count),
                                                  int(width), int(height), int(capacity), ptr(vals), ptr(ranges),
                                                  ptr(tile_order), ptr(pair_offset), ptr(pair_emit), ptr(keys),
                                                  ptr(num_pairs), ptr(status), ptr(ws),
                                                  ws.numel() * ws.element_size(),
                                                  stream if stream is not None else current_stream()))


def _bg(bg):
    arr = (ctypes.c_float * 3)(*[float(x) for x in bg])
    return arr


def gs_raster_fwd(proj: gs_proj, n, vals, ranges, width, height, bg, img, final_T, n_contrib, active=None,
                  pair_stats=None, stream=None, tile_order=None):
    b = _bg(bg)
    return _check("gs_raster_fwd", _lib.gs_raster_fwd(ctypes.byref(proj), int(n), ptr(vals), ptr(ranges),
                                                      ptr(tile_order), int(width), int(height), ctypes.cast(b, P),
                                                      ptr(img), ptr(final_T), ptr(n_contrib), ptr(active),
                                                      ptr(pair_stats),
                                                      stream if stream is not None else current_stream()))


def gs_raster_fwd_l1(proj: gs_proj, n, vals, ranges, width, height, bg, target, img, final_T, n_contrib, active, loss,
                     dL_dimg, ws, stream=None, tile_order=None):
    b = _bg(bg)
    return _check("gs_raster_fwd_l1", _lib.gs_raster_fwd_l1(
        ctypes.byref(proj), int(n), ptr(vals), ptr(ranges), ptr(tile_order), int(width), int(height),
        ctypes.cast(b, P), ptr(target), ptr(img), ptr(final_T), ptr(n_contrib), ptr(active), ptr(loss),
        ptr(dL_dimg), ptr(ws),
        ws.numel() * ws.element_size(), stream if stream is not None else current_stream()))


def gs_loss_l1(img, target, width, height, loss, dL_dimg, ws, stream=None):
    return _check("gs_loss_l1", _lib.gs_loss_l1(ptr(img), ptr(target), int(width), int(height), ptr(loss),
                                                ptr(dL_dimg), ptr(ws), ws.numel() * ws.element_size(),
                                                stream if stream is not None else current_stream()))


def gs_raster_bwd(scene: gs_scene, cam: gs_camera, proj: gs_proj, vals, ranges, pair_offset, pair_emit, vis_idx,
                  vis_count, capacity, final_T, n_contrib, dL_dimg, bg, grad_rows, grad_ld, grad2d, grad_norm, ws,
                  stream=None, tile_order=None):
    b = _bg(bg)
    return _check("gs_raster_bwd", _lib.gs_raster_bwd(ctypes.byref(scene), ctypes.byref(cam), ctypes.byref(proj),
                                                      ptr(vals), ptr(ranges), ptr(tile_order), ptr(pair_offset),
                                                      ptr(pair_emit), ptr(vis_idx), ptr(vis_count), int(capacity),
                                                      ptr(final_T),
                                                      ptr(n_contrib), ptr(dL_dimg), ctypes.cast(b, P),
                                                      ptr(grad_rows), int(grad_ld), ptr(grad2d), ptr(grad_norm),
                                                      ptr(ws), ws.numel() * ws.element_size(),
                                                      stream if stream is not None else current_stream()))


def gs_raster_bwd_pixels(proj: gs_proj, cam: gs_camera, vals, ranges, pair_emit, capacity, final_T, n_contrib, dL_dimg,
                         bg, ws, stream=None, tile_order=None):
    b = _bg(bg)
    return _check("gs_raster_bwd_pixels", _lib.gs_raster_bwd_pixels(
        ctypes.byref(proj), ctypes.byref(cam), ptr(vals), ptr(ranges), ptr(tile_order), ptr(pair_emit), int(capacity),
        ptr(final_T), ptr(n_contrib), ptr(dL_dimg), ctypes.cast(b, P), ptr(ws), ws.numel() * ws.element_size(),
        stream if stream is not None else current_stream()))


def gs_raster_bwd_project(scene: gs_scene, cam: gs_camera, proj: gs_proj, pair_offset, vis_idx, vis_count,
                          capacity, grad_rows, grad_ld, grad2d, grad_norm, ws, stream=None):
    return _check("gs_raster_bwd_project", _lib.gs_raster_bwd_project(
        ctypes.byref(scene), ctypes.byref(cam), ctypes.byref(proj), ptr(pair_offset), ptr(vis_idx),
        ptr(vis_count), int(capacity), ptr(grad_rows), int(grad_ld), ptr(grad2d), ptr(grad_norm), ptr(ws),
        ws.numel() * ws.element_size(), stream if stream is not None else current_stream()))


def gs_raster_bwd_project_accum(scene: gs_scene, cam: gs_camera, proj: gs_proj, pair_offset, vis_idx, vis_count,
                                capacity, union_idx, union_count, first, grad_rows, grad_ld, grad_norm, ws, stream=None):
    return _check("gs_raster_bwd_project_accum", _lib.gs_raster_bwd_project_accum(
        ctypes.byref(scene), ctypes.byref(cam), ctypes.byref(proj), ptr(pair_offset), ptr(vis_idx), ptr(vis_count),
        int(capacity), ptr(union_idx), ptr(union_count), int(first), ptr(grad_rows), int(grad_ld), ptr(grad_norm),
        ptr(ws), ws.numel() * ws.element_size(), stream if stream is not None else current_stream()))


def make_adam_groups(groups):
    """groups: list of (p [n, cols] tensor, lr)."""
    arr = (gs_adam_group * len(groups))()
    for i, (p, lr) in enumerate(groups):
        arr[i] = gs_adam_group(ptr(p), int(p.shape[1]), float(lr), row_stride(p))
    return arr


def gs_sparse_adam(groups_arr, n_groups, idx, count, max_rows, grad_rows, grad_ld, m, v, state_ld, step, beta1,
                   beta2, eps, delta_rows=None, delta_ld=0, stream=None):
    return _check("gs_sparse_adam", _lib.gs_sparse_adam(
        groups_arr, int(n_groups), ptr(idx), ptr(count), int(max_rows), ptr(grad_rows), int(grad_ld), ptr(m), ptr(v),
        int(state_ld), int(step), float(beta1), float(beta2), float(eps), ptr(delta_rows), int(delta_ld),
        stream if stream is not None else current_stream()))


def gs_sparse_adam_publish(groups_arr, n_groups, idx, count, max_rows, grad_rows, grad_ld, m, v, state_ld, step,
                           beta1, beta2, eps, version, msg, status, stream=None):
    return _check("gs_sparse_adam_publish", _lib.gs_sparse_adam_publish(
        groups_arr, int(n_groups), ptr(idx), ptr(count), int(max_rows), ptr(grad_rows), int(grad_ld), ptr(m), ptr(v),
        int(state_ld), int(step), float(beta1), float(beta2), float(eps), int(version), ptr(msg),
        msg.numel() * msg.element_size(), ptr(status), stream if stream is not None else current_stream()))


def make_groups(tensors):
    arr = (gs_group * len(tensors))()
    for i, t in enumerate(tensors):
        arr[i] = gs_group(ptr(t), int(t.shape[1]), row_stride(t))
    return arr


def gs_delta_pack(idx, count, max_rows, groups_arr, n_groups, version, msg, status, stream=None):
    return _check("gs_delta_pack", _lib.gs_delta_pack(ptr(idx), ptr(count), int(max_rows), groups_arr, int(n_groups),
                                                      int(version), ptr(msg), msg.numel() * msg.element_size(),
                                                      ptr(status), stream if stream is not None else current_stream()))


def gs_delta_apply(msg, groups_arr, n_groups, n_rows, max_rows, mode, prim_version, status, stream=None):
    return _check("gs_delta_apply", _lib.gs_delta_apply(ptr(msg), msg.numel() * msg.element_size(), groups_arr,
                                                        int(n_groups), int(n_rows),
                                                        int(max_rows), int(mode), ptr(prim_version), ptr(status),
                                                        stream if stream is not None else current_stream()))


def make_ring(slots, state, background=False) -> gs_ring:
    """slots: two device tensors of equal byte size (slot v & 1 holds version v); state: >= 8 uint32 words;
    background: the commit runs beside compute on another stream (one workgroup per compute unit)."""
    nb = min(t.numel() * t.element_size() for t in slots)
    r = gs_ring()
    r.slot[0], r.slot[1] = slots[0].data_ptr(), slots[1].data_ptr()
    r.slot_bytes = nb
    r.state = state.data_ptr()
    r.background = 1 if background else 0
    return r


def gs_publish_commit(ring: gs_ring, version, groups_arr, n_groups, n_rows, max_rows, mode, prim_version, skip, status,
                      stream=None):
    return _check("gs_publish_commit", _lib.gs_publish_commit(
        ctypes.byref(ring), int(version), groups_arr, int(n_groups), int(n_rows), int(max_rows), int(mode),
        ptr(prim_version), ptr(skip), ptr(status), stream if stream is not None else current_stream()))


def gs_scope_from_ids(idx, count, max_rows, n, accumulate, scope, stream=None):
    return _check("gs_scope_from_ids", _lib.gs_scope_from_ids(ptr(idx), ptr(count), int(max_rows), int(n),
                                                              int(accumulate), ptr(scope),
                                                              stream if stream is not None else current_stream()))


def gs_scope_from_pred(kind, src, n, accumulate, scope, stream=None):
    return _check("gs_scope_from_pred", _lib.gs_scope_from_pred(int(kind), ptr(src), int(n), int(accumulate),
                                                                ptr(scope),
                                                                stream if stream is not None else current_stream()))


def gs_scope_conflicts(RA, WA, RB, WB, n, waw, raw_, war, waw_idx, raw_idx, war_idx, counts, ws, stream=None):
    return _check("gs_scope_conflicts", _lib.gs_scope_conflicts(
        ptr(RA), ptr(WA), ptr(RB), ptr(WB), int(n), ptr(waw), ptr(raw_), ptr(war), ptr(waw_idx), ptr(raw_idx),
        ptr(war_idx), ptr(counts), ptr(ws), ws.numel() * ws.element_size() if ws is not None else 0,
        stream if stream is not None else current_stream()))


def make_gate_args(active, g, tau, evidence=None, skip=None, producer_version=0) -> gs_gate_args:
    return gs_gate_args(ptr(active), ptr(evidence), ptr(g), ptr(skip), int(producer_version), float(tau))


def gs_admission_gate(RB, D, args: gs_gate_args, n, result, ws, stream=None):
    """result: a device tensor of >= 64 bytes (see gate_result_from)."""
    return _check("gs_admission_gate", _lib.gs_admission_gate(
        ptr(RB), ptr(D), ctypes.byref(args), int(n), ptr(result), ptr(ws),
        ws.numel() * ws.element_size() if ws is not None else 0,
        stream if stream is not None else current_stream()))


def gate_result_from(buf) -> gs_gate_result:
    """Decode a result record copied to the host (bytes-like or a tensor)."""
    if hasattr(buf, "cpu"):
        buf = buf.detach().cpu().numpy().tobytes()
    return gs_gate_result.from_buffer_copy(bytes(buf)[:ctypes.sizeof(gs_gate_result)])


def raw():
    """The loaded ctypes library (for tests of argument validation)."""
    return _lib


# ---- the ahead-of-time planner (host arrays) --------------------------------

def _np(a, dtype):
    """A C-contiguous numpy array of dtype and its pointer (kept alive by the caller)."""
    import numpy as np
    a = np.ascontiguousarray(a, dtype=dtype)
    return a, ctypes.c_void_p(a.ctypes.data)


class PlanGraph:
    """The retained relative locality graph in CSR form (numpy arrays)."""

    def __init__(self, edge_ptr, edge_dst, edge_w):
        self.edge_ptr, self.edge_dst, self.edge_w = edge_ptr, edge_dst, edge_w

    def ptrs(self):
        return (ctypes.c_void_p(self.edge_ptr.ctypes.data), ctypes.c_void_p(self.edge_dst.ctypes.data),
                ctypes.c_void_p(self.edge_w.ctypes.data))


def gs_rlg_build(item_ptr, item_tracks, n_tracks, track_cap, top_k) -> PlanGraph:
    import numpy as np
    ip, ip_p = _np(item_ptr, np.int64)
    it, it_p = _np(item_tracks if len(item_tracks) else np.zeros(1, np.int32), np.int32)
    n = ip.size - 1
    cap = 2 * n * int(top_k) if top_k > 0 else 0
    for _ in range(2):
        eptr = np.zeros(n + 1, np.int64)
        edst = np.zeros(max(cap, 1), np.int32)
        ew = np.zeros(max(cap, 1), np.float64)
        ne = ctypes.c_int64(0)
        st = _lib.gs_rlg_build(int(n), int(n_tracks), ip_p, it_p, int(track_cap), int(top_k),
                               ctypes.c_void_p(eptr.ctypes.data), ctypes.c_void_p(edst.ctypes.data),
                               ctypes.c_void_p(ew.ctypes.data), int(cap), ctypes.byref(ne))
        if st == GS_ERR_WORKSPACE and cap < ne.value:
            cap = int(ne.value)
            continue
        _check("gs_rlg_build", st)
        return PlanGraph(eptr, edst[:ne.value].copy(), ew[:ne.value].copy())
    raise GsmiError("gs_rlg_build", GS_ERR_WORKSPACE)


def gs_lp_partition(position, graph: PlanGraph, K, max_iters):
    """Returns (group [n] int32, coupling [K, K] float64, rounds run)."""
    import numpy as np
    pos, pos_p = _np(np.asarray(position, np.float64).reshape(-1, 3), np.float64)
    n = pos.shape[0]
    group = np.zeros(max(n, 1), np.int32)
    coupling = np.zeros((K, K), np.float64)
    it = ctypes.c_int32(0)
    ep, ed, ew = graph.ptrs()
    _check("gs_lp_partition", _lib.gs_lp_partition(int(n), pos_p, ep, ed, ew, int(K), int(max_iters),
                                                   ctypes.c_void_p(group.ctypes.data),
                                                   ctypes.c_void_p(coupling.ctypes.data), ctypes.byref(it)))
    return group[:n], coupling, int(it.value)


def gs_sds_order(group, coupling, graph: PlanGraph, unit_size):
    """Returns (cycle, order, unit_group, transition) as numpy arrays."""
    import numpy as np
    g, g_p = _np(group, np.int32)
    K = int(np.asarray(coupling).shape[0])
    C, C_p = _np(coupling, np.float64)
    n = g.size
    units = -(-n // int(unit_size)) if n else 0
    cycle = np.zeros(K, np.int32)
    order = np.zeros(max(n, 1), np.int32)
    ug = np.zeros(max(units, 1), np.int32)
    tr = np.zeros(max(units, 1), np.float64)
    nc, nu = ctypes.c_int32(0), ctypes.c_int32(0)
    ep, ed, ew = graph.ptrs()
    _check("gs_sds_order", _lib.gs_sds_order(int(n), g_p, K, C_p, ep, ed, ew, int(unit_size),
                                             ctypes.c_void_p(cycle.ctypes.data), ctypes.byref(nc),
                                             ctypes.c_void_p(order.ctypes.data), ctypes.c_void_p(ug.ctypes.data),
                                             ctypes.c_void_p(tr.ctypes.data), ctypes.byref(nu)))
    assert nu.value == units
    return cycle[:nc.value], order[:n], ug[:units], tr[:units]
