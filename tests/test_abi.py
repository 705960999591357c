"""The C-ABI library loads, exports every entry point include/gsmi.h declares,
and rejects bad arguments synchronously (host-side checks, no GPU needed)."""
import ctypes
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_symbols():
    src = open(os.path.join(ROOT, "include", "gsmi.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(gs_[a-z0-9_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def gs():
    from paper_2607_19893_amd import gsmi
    return gsmi


def test_exports_every_declared_symbol(gs):
    names = declared_symbols()
    assert len(names) >= 16
    for nm in names:
        assert hasattr(gs.raw(), nm), nm
        assert nm in gs.EXPORTS, nm
    assert gs.gs_abi_version() == gs.ABI_VERSION == 4


def test_noalloc_limits_match_header(gs):
    src = open(os.path.join(ROOT, "include", "gsmi.h")).read()
    d = dict(re.findall(r"#define (GS_NOALLOC_\w+) (\d+)", src))
    assert int(d["GS_NOALLOC_SCRATCH_BYTES"]) == gs.GS_NOALLOC_SCRATCH_BYTES
    assert int(d["GS_NOALLOC_MAX_N"]) == gs.GS_NOALLOC_MAX_N
    # the compaction needs one count per 2048 ids plus one word
    assert (gs.GS_NOALLOC_MAX_N // 2048 + 1) * 4 == gs.GS_NOALLOC_SCRATCH_BYTES
    assert gs.gs_workspace_bytes(gs.GS_WS_VISIBLE_SET, gs.GS_NOALLOC_MAX_N) <= gs.GS_NOALLOC_SCRATCH_BYTES
    assert gs.gs_workspace_bytes(gs.GS_WS_VISIBLE_SET, gs.GS_NOALLOC_MAX_N + 1) > gs.GS_NOALLOC_SCRATCH_BYTES


def test_status_strings(gs):
    assert gs.gs_status_string(0) == "ok"
    assert "workspace" in gs.gs_status_string(3)


def test_null_and_range_arguments_rejected(gs):
    L = gs.raw()
    assert L.gs_project(None, None, None, None) == gs.GS_ERR_INVALID_ARG
    assert "null scene" in gs.gs_last_error()
    sc = gs.gs_scene(10, 4, 1, 1, 16, 1, 16)
    cam = gs.gs_camera()
    pr = gs.gs_proj(16, 16, 16, 16, 16, 16, 16, 16)
    assert L.gs_project(ctypes.byref(sc), ctypes.byref(cam), ctypes.byref(pr), None) == gs.GS_ERR_INVALID_ARG
    assert "sh_degree" in gs.gs_last_error()
    sc.sh_degree = 3
    cam.width = 40000
    assert L.gs_project(ctypes.byref(sc), ctypes.byref(cam), ctypes.byref(pr), None) == gs.GS_ERR_UNSUPPORTED
    assert L.gs_visible_set(7, None, 0, None, None, None, 0, None) == gs.GS_ERR_INVALID_ARG
    assert L.gs_visible_set(4, None, 0, None, None, None, 0, None) == gs.GS_ERR_INVALID_ARG
    assert L.gs_visible_set(gs.GS_PRED_U8_NONZERO_CLEAR, 12, 100, 16, 16, 256, 1 << 20,
                            None) == gs.GS_ERR_INVALID_ARG                 # flags must be 8-byte aligned
    assert "misaligned" in gs.gs_last_error()
    assert L.gs_scope_from_pred(gs.GS_PRED_U8_NONZERO_CLEAR, 16, 100, 0, 16, None) == gs.GS_ERR_INVALID_ARG
    assert L.gs_visible_set(0, 16, 100, 16, 16, 256, 0, None) == gs.GS_ERR_WORKSPACE
    # workspaces are 256-byte aligned (the per-block counts are read 16 bytes at a time)
    assert L.gs_visible_set(0, 16, 100, 16, 16, 16, 1 << 20, None) == gs.GS_ERR_INVALID_ARG
    assert "aligned" in gs.gs_last_error()
    assert L.gs_bin_sort(ctypes.byref(pr), 10, 16, 16, 64, 64, 0, None, 16, None, 16, None, None, 16, 16, 16, 1 << 20,
                         None) == gs.GS_ERR_INVALID_ARG
    assert "aligned" in gs.gs_last_error()
    # the no-allocation variant: sizes beyond its fixed workspace are refused before any HIP call
    assert L.gs_visible_set_noalloc(0, 16, gs.GS_NOALLOC_MAX_N + 1, 16, 16, None) == gs.GS_ERR_UNSUPPORTED
    assert "GS_NOALLOC_MAX_N" in gs.gs_last_error()
    assert L.gs_visible_set_noalloc(4, 16, 100, 16, 16, None) == gs.GS_ERR_INVALID_ARG
    assert L.gs_visible_set_noalloc(0, 16, -1, 16, 16, None) == gs.GS_ERR_INVALID_ARG
    assert L.gs_visible_set_noalloc(0, 16, 100, 16, None, None) == gs.GS_ERR_INVALID_ARG
    A = (16, 16, 10, 16, 64, 16, 16, 64)          # idx, count, max_rows, grad_rows, grad_ld, m, v, state_ld
    assert L.gs_sparse_adam(None, 0, *A, 1, 0.9, 0.999, 1e-15, None, 0, None) == gs.GS_ERR_INVALID_ARG
    grp = (gs.gs_adam_group * 1)(gs.gs_adam_group(16, 70, 1e-3))
    assert L.gs_sparse_adam(grp, 1, *A, 1, 0.9, 0.999, 1e-15, None, 0, None) == gs.GS_ERR_UNSUPPORTED
    grp[0].cols = 3
    assert L.gs_sparse_adam(grp, 1, *A, 0, 0.9, 0.999, 1e-15, None, 0, None) == gs.GS_ERR_INVALID_ARG
    assert "step" in gs.gs_last_error()
    assert L.gs_sparse_adam(grp, 1, 16, 16, 10, 16, 2, 16, 16, 64, 1, 0.9, 0.999, 1e-15, None, 0,
                            None) == gs.GS_ERR_INVALID_ARG
    assert "grad_ld" in gs.gs_last_error()
    assert L.gs_sparse_adam(grp, 1, *A, 1, 0.9, 0.999, 1e-15, 16, 2, None) == gs.GS_ERR_INVALID_ARG
    assert "delta_ld" in gs.gs_last_error()
    assert L.gs_sparse_adam_publish(grp, 1, *A, 1, 0.9, 0.999, 1e-15, 1, None, 1024, 16,
                                    None) == gs.GS_ERR_INVALID_ARG
    assert L.gs_sparse_adam_publish(grp, 1, *A, 1, 0.9, 0.999, 1e-15, 1, 8, 1024, 16, None) == gs.GS_ERR_INVALID_ARG
    assert "aligned" in gs.gs_last_error()
    # gradient rows of the backward: leading dimension a multiple of 4, at least the row length
    sc3 = gs.gs_scene(10, 3, 16, 16, 16, 16, 16)
    cam3 = gs.gs_camera()
    assert L.gs_raster_bwd_project(ctypes.byref(sc3), ctypes.byref(cam3), ctypes.byref(pr), 16, 16, 16, 100, 16,
                                   58, None, None, 256, 1 << 20, None) == gs.GS_ERR_INVALID_ARG
    assert "grad_ld" in gs.gs_last_error()
    g = (gs.gs_group * 1)(gs.gs_group(16, 3))
    assert L.gs_delta_apply(16, 4096, g, 1, 10, 10, 5, None, 16, None) == gs.GS_ERR_INVALID_ARG
    assert L.gs_delta_apply(16, 8, g, 1, 10, 10, 0, None, 16, None) == gs.GS_ERR_INVALID_ARG
    assert L.gs_delta_pack(16, 16, 10, g, 1, 1, 8, 1024, 16, None) == gs.GS_ERR_INVALID_ARG  # misaligned msg
    assert L.gs_loss_l1(None, None, 4, 4, None, None, None, 0, None) == gs.GS_ERR_INVALID_ARG
    # row strides of the parameter groups: at least the group's width, quat and sh a multiple of 4
    cam.width = 64
    for field, bad, word in (("ld_mean", 2, "ld_mean"), ("ld_quat", 6, "ld_quat"), ("ld_sh", 44, "ld_sh"),
                             ("ld_sh", 50, "ld_sh"), ("ld_sh", 3, "ld_sh"), ("ld_log_scale", 1, "ld_log_scale"),
                             ("ld_opacity", -1, "ld_opacity")):
        scl = gs.gs_scene(10, 3, 16, 16, 16, 16, 16)
        setattr(scl, field, bad)
        assert L.gs_project(ctypes.byref(scl), ctypes.byref(cam), ctypes.byref(pr), None) == gs.GS_ERR_INVALID_ARG
        assert word in gs.gs_last_error()
    grp[0].ld = 2
    assert L.gs_sparse_adam(grp, 1, *A, 1, 0.9, 0.999, 1e-15, None, 0, None) == gs.GS_ERR_INVALID_ARG
    assert "ld 2 below cols 3" in gs.gs_last_error()
    g[0].ld = 1
    assert L.gs_delta_apply(16, 4096, g, 1, 10, 10, 0, None, 16, None) == gs.GS_ERR_INVALID_ARG
    assert "ld 1 below cols 3" in gs.gs_last_error()
    g[0].ld = 0
    # fused forward + loss: workspace sized per tile
    assert L.gs_raster_fwd_l1(ctypes.byref(pr), 10, 16, 16, None, 256, 256, 16, 16, 16, 16, 16, None, 16, 16, 16, 0,
                              None) == gs.GS_ERR_WORKSPACE
    assert L.gs_raster_fwd_l1(ctypes.byref(pr), 10, 16, 16, None, 256, 256, 16, None, 16, 16, 16, None, 16, 16, 16,
                              1 << 20,
                              None) == gs.GS_ERR_INVALID_ARG
    assert gs.gs_workspace_bytes(gs.GS_WS_RASTER_FWD_L1, 0, 0, 1920, 1080) >= 4 * 120 * 68
    # versioned commit of a ring slot
    ring = gs.gs_ring()
    ring.slot[0], ring.slot[1], ring.slot_bytes, ring.state = 16, 32, 4096, 16
    g5 = (gs.gs_group * 1)(gs.gs_group(16, 3))
    assert L.gs_publish_commit(None, 1, g5, 1, 10, 10, 0, 16, None, 16, None) == gs.GS_ERR_INVALID_ARG
    assert L.gs_publish_commit(ctypes.byref(ring), 0, g5, 1, 10, 10, 0, 16, None, 16, None) == gs.GS_ERR_INVALID_ARG
    assert "version 0" in gs.gs_last_error()
    assert L.gs_publish_commit(ctypes.byref(ring), 1, g5, 1, 10, 10, 0, None, None, 16, None) == gs.GS_ERR_INVALID_ARG
    assert L.gs_publish_commit(ctypes.byref(ring), 1, g5, 1, 10, 10, 3, 16, None, 16, None) == gs.GS_ERR_INVALID_ARG
    ring.slot[1] = 40
    assert L.gs_publish_commit(ctypes.byref(ring), 1, g5, 1, 10, 10, 0, 16, None, 16, None) == gs.GS_ERR_INVALID_ARG
    assert "aligned" in gs.gs_last_error()
    ring.slot[1], ring.slot_bytes = 32, 8
    assert L.gs_publish_commit(ctypes.byref(ring), 1, g5, 1, 10, 10, 0, 16, None, 16, None) == gs.GS_ERR_INVALID_ARG
    # scopes, hazards and admission
    assert L.gs_scope_from_ids(None, None, 5, 100, 0, 16, None) == gs.GS_ERR_INVALID_ARG
    assert L.gs_scope_from_ids(16, 16, 5, -1, 0, 16, None) == gs.GS_ERR_INVALID_ARG
    assert L.gs_scope_from_pred(5, 16, 100, 0, 16, None) == gs.GS_ERR_INVALID_ARG
    assert L.gs_scope_from_pred(0, None, 100, 0, 16, None) == gs.GS_ERR_INVALID_ARG
    assert L.gs_scope_conflicts(16, 16, 16, 16, 100, None, None, None, None, None, None, None, 16, 1 << 20,
                                None) == gs.GS_ERR_INVALID_ARG
    assert L.gs_scope_conflicts(16, 16, 16, None, 100, None, None, None, None, None, None, 16, 16, 1 << 20,
                                None) == gs.GS_ERR_INVALID_ARG
    assert L.gs_scope_conflicts(16, 16, 16, 16, 1 << 20, None, None, None, None, None, None, 16, 16, 0,
                                None) == gs.GS_ERR_WORKSPACE
    args = gs.gs_gate_args(16, None, 16, None, 0, 1.5)
    assert L.gs_admission_gate(16, 16, ctypes.byref(args), 100, 16, 16, 1 << 20, None) == gs.GS_ERR_INVALID_ARG
    assert "tau" in gs.gs_last_error()
    args = gs.gs_gate_args(16, None, 16, 16, 0, 0.2)
    assert L.gs_admission_gate(16, 16, ctypes.byref(args), 100, 16, 16, 1 << 20, None) == gs.GS_ERR_INVALID_ARG
    assert "producer version" in gs.gs_last_error()
    args = gs.gs_gate_args(None, None, 16, None, 0, 0.2)
    assert L.gs_admission_gate(16, 16, ctypes.byref(args), 100, 16, 16, 1 << 20, None) == gs.GS_ERR_INVALID_ARG
    args = gs.gs_gate_args(16, None, 16, None, 0, 0.2)
    assert L.gs_admission_gate(16, 16, ctypes.byref(args), 1 << 20, 16, 16, 0, None) == gs.GS_ERR_WORKSPACE


def test_workspace_sizes_monotone(gs):
    a = gs.gs_workspace_bytes(gs.GS_WS_BIN_SORT, 1000, 5000, 256, 256)
    b = gs.gs_workspace_bytes(gs.GS_WS_BIN_SORT, 2000, 10000, 256, 256)
    assert 0 < a < b and a % 256 == 0
    assert gs.gs_workspace_bytes(gs.GS_WS_RASTER_BWD, 0, 100) >= 9 * 4 * 100
    # the backward's workspace holds one padded 9-float slot per pair of the capacity
    assert gs.gs_workspace_bytes(gs.GS_WS_RASTER_BWD, 1000, 100) >= 12 * 4 * 100
    assert gs.gs_workspace_bytes(gs.GS_WS_RASTER_BWD, 0, 5000) > gs.gs_workspace_bytes(gs.GS_WS_RASTER_BWD, 0, 100)
    assert gs.gs_workspace_bytes(99, 10, 10) == 0
    assert 0 < gs.gs_workspace_bytes(gs.GS_WS_SCOPE, 100) <= gs.gs_workspace_bytes(gs.GS_WS_SCOPE, 10_000_000)


def test_message_size_matches_oracle_layout(gs, orc):
    rng = np.random.default_rng(0)
    for K, cols in ((0, [3]), (1, [3, 3, 4, 1, 48]), (37, [3, 3, 4, 1, 3]), (1000, [1, 2, 3, 4, 5, 6, 7, 8])):
        groups = [rng.standard_normal((max(K, 1) + 5, c)).astype(np.float32) for c in cols]
        msg = orc.delta_pack(np.arange(K, dtype=np.uint32), groups, 3)
        assert gs.gs_delta_msg_bytes(K, sum(cols), len(cols)) == msg.size * 4
