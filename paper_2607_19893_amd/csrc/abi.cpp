// C-ABI entry points: synchronous argument validation, then the launches.
// No entry point allocates, frees or synchronizes.
#include <hip/hip_runtime.h>

#include <atomic>
#include <cstdarg>
#include <cstdio>
#include <cstring>

#include "internal.h"

namespace gsmi {

// The device-property cache: compute units per device, filled on first use.
uint32_t compute_units() {
    static std::atomic<uint32_t> cache[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0) return 0;
    if (dev >= 64) {
        int v = 0;
        return hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess ? (uint32_t)v : 0;
    }
    uint32_t c = cache[dev].load(std::memory_order_relaxed);
    if (c == 0) {
        int v = 0;
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0) return 0;
        c = (uint32_t)v;
        cache[dev].store(c, std::memory_order_relaxed);
    }
    return c;
}

}  // namespace gsmi

namespace {

thread_local char g_err[256] = "";

gs_status fail(gs_status s, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return s;
}

gs_status ok() {
    g_err[0] = 0;
    return GS_OK;
}

gs_status hip_status(hipError_t e, const char* what) {
    if (e != hipSuccess) return fail(GS_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
    return ok();
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

#define GS_REQUIRE(cond, ...)                                   \
    do {                                                        \
        if (!(cond)) return fail(GS_ERR_INVALID_ARG, __VA_ARGS__); \
    } while (0)

gs_status check_scene(const gs_scene* s, const char* what) {
    GS_REQUIRE(s != nullptr, "%s: null scene", what);
    GS_REQUIRE(s->n >= 0, "%s: n < 0", what);
    GS_REQUIRE(s->sh_degree >= 0 && s->sh_degree <= GS_MAX_SH_DEGREE, "%s: sh_degree %d outside 0..3", what,
               s->sh_degree);
    if (s->n > 0) {
        GS_REQUIRE(s->mean && s->log_scale && s->quat && s->opacity && s->sh, "%s: null parameter pointer", what);
        GS_REQUIRE(aligned(s->quat, 16) && aligned(s->sh, 16), "%s: quat and sh must be 16-byte aligned", what);
    }
    const int32_t K3 = 3 * (s->sh_degree + 1) * (s->sh_degree + 1);
    GS_REQUIRE(s->ld_mean == 0 || s->ld_mean >= 3, "%s: ld_mean %d below 3", what, s->ld_mean);
    GS_REQUIRE(s->ld_log_scale == 0 || s->ld_log_scale >= 3, "%s: ld_log_scale %d below 3", what, s->ld_log_scale);
    GS_REQUIRE(s->ld_opacity >= 0, "%s: ld_opacity < 0", what);
    GS_REQUIRE(s->ld_quat == 0 || (s->ld_quat >= 4 && s->ld_quat % 4 == 0),
               "%s: ld_quat %d must be a multiple of 4 and >= 4", what, s->ld_quat);
    GS_REQUIRE(s->ld_sh == 0 || s->ld_sh == K3 || (s->ld_sh > K3 && s->ld_sh % 4 == 0),
               "%s: ld_sh %d must be %d or a multiple of 4 above it", what, s->ld_sh, K3);
    return GS_OK;
}

gs_status check_camera(const gs_camera* c, const char* what) {
    if (c == nullptr) return fail(GS_ERR_INVALID_ARG, "%s: null camera", what);
    if (c->width < 0 || c->height < 0) return fail(GS_ERR_INVALID_ARG, "%s: negative image size", what);
    if (c->width > GS_MAX_IMAGE_SIDE || c->height > GS_MAX_IMAGE_SIDE)
        return fail(GS_ERR_UNSUPPORTED, "%s: image side above %d", what, GS_MAX_IMAGE_SIDE);
    return GS_OK;
}

gs_status check_proj(const gs_proj* p, bool need_all, const char* what) {
    GS_REQUIRE(p != nullptr, "%s: null proj", what);
    GS_REQUIRE(p->tiles && p->rect && p->depth && p->mean2d && p->conic_opacity && p->rgb, "%s: null proj array",
               what);
    if (need_all) GS_REQUIRE(p->radius && p->clamp, "%s: null proj array", what);
    GS_REQUIRE(aligned(p->rect, 8) && aligned(p->mean2d, 8) && aligned(p->conic_opacity, 16),
               "%s: proj arrays misaligned (rect 8, mean2d 8, conic_opacity 16 bytes)", what);
    return GS_OK;
}

int32_t scene_row_len(const gs_scene* s) { return 11 + 3 * (s->sh_degree + 1) * (s->sh_degree + 1); }

gs_status check_grad_rows(const gs_scene* s, const float* grad_rows, int32_t grad_ld, const char* what) {
    GS_REQUIRE(grad_rows != nullptr || s->n == 0, "%s: null grad_rows", what);
    GS_REQUIRE(aligned(grad_rows, 16), "%s: grad_rows must be 16-byte aligned", what);
    GS_REQUIRE(grad_ld % 4 == 0 && grad_ld >= scene_row_len(s), "%s: grad_ld %d must be a multiple of 4 and >= %d",
               what, grad_ld, scene_row_len(s));
    return GS_OK;
}

}  // namespace

extern "C" {

int32_t gs_abi_version(void) { return GSMI_ABI_VERSION; }

const char* gs_status_string(int32_t s) {
    switch (s) {
        case GS_OK: return "ok";
        case GS_ERR_INVALID_ARG: return "invalid argument";
        case GS_ERR_UNSUPPORTED: return "unsupported size";
        case GS_ERR_WORKSPACE: return "workspace too small";
        case GS_ERR_HIP: return "HIP runtime error";
        default: return "unknown status";
    }
}

const char* gs_last_error(void) { return g_err; }

size_t gs_workspace_bytes(int32_t which, int32_t n, uint32_t capacity, int32_t width, int32_t height) {
    if (n < 0 || width < 0 || height < 0) return 0;
    switch (which) {
        case GS_WS_VISIBLE_SET: return gsmi::visible_ws_bytes(n);
        case GS_WS_BIN_SORT: return gsmi::binsort_ws_bytes(n, capacity, width, height);
        case GS_WS_RASTER_BWD: return gsmi::raster_bwd_ws_bytes(n, capacity);
        case GS_WS_LOSS: return gsmi::loss_ws_bytes(width, height);
        case GS_WS_SCOPE: return gsmi::scope_ws_bytes(n);
        case GS_WS_RASTER_FWD_L1: return gsmi::raster_fwd_l1_ws_bytes(width, height);
        default: return 0;
    }
}

size_t gs_delta_msg_bytes(uint32_t count, int32_t row_len, int32_t n_groups) {
    if (row_len < 0 || n_groups < 0) return 0;
    return gsmi::delta_msg_bytes(count, row_len, n_groups);
}

gs_status gs_project(const gs_scene* scene, const gs_camera* cam, const gs_proj* out, void* stream) {
    gs_status s;
    if ((s = check_scene(scene, "gs_project")) != GS_OK) return s;
    if ((s = check_camera(cam, "gs_project")) != GS_OK) return s;
    if ((s = check_proj(out, true, "gs_project")) != GS_OK) return s;
    const gsmi::CamArgs c = gsmi::make_cam_args(cam);
    return hip_status(gsmi::launch_project(*scene, c, *out, static_cast<hipStream_t>(stream)), "gs_project");
}

gs_status gs_visible_set(int32_t kind, const void* src, int32_t n, uint32_t* out_idx, uint32_t* out_count, void* ws,
                         size_t ws_bytes, void* stream) {
    GS_REQUIRE(kind == GS_PRED_U32_NONZERO || kind == GS_PRED_U8_NONZERO || kind == GS_PRED_BITMAP ||
                   kind == GS_PRED_U8_NONZERO_CLEAR,
               "gs_visible_set: bad kind %d", kind);
    GS_REQUIRE(n >= 0, "gs_visible_set: n < 0");
    GS_REQUIRE(out_count != nullptr, "gs_visible_set: null out_count");
    if (n > 0) {
        GS_REQUIRE(src && out_idx && ws, "gs_visible_set: null pointer");
        GS_REQUIRE(aligned(ws, 256), "gs_visible_set: workspace must be 256-byte aligned");
        GS_REQUIRE(aligned(src, kind == GS_PRED_U32_NONZERO ? 16 : (kind == GS_PRED_BITMAP ? 4 : 8)),
                   "gs_visible_set: src misaligned");
    }
    if (ws_bytes < gsmi::visible_ws_bytes(n)) return fail(GS_ERR_WORKSPACE, "gs_visible_set: workspace too small");
    return hip_status(gsmi::launch_visible(kind, src, n, out_idx, out_count, ws, static_cast<hipStream_t>(stream)),
                      "gs_visible_set");
}

gs_status gs_visible_set_noalloc(int32_t kind, const void* src, int32_t n, uint32_t* out_idx, uint32_t* out_count,
                                 void* stream) {
    GS_REQUIRE(kind == GS_PRED_U32_NONZERO || kind == GS_PRED_U8_NONZERO || kind == GS_PRED_BITMAP ||
                   kind == GS_PRED_U8_NONZERO_CLEAR,
               "gs_visible_set_noalloc: bad kind %d", kind);
    GS_REQUIRE(n >= 0, "gs_visible_set_noalloc: n < 0");
    if (n > GS_NOALLOC_MAX_N)
        return fail(GS_ERR_UNSUPPORTED, "gs_visible_set_noalloc: n = %d above GS_NOALLOC_MAX_N (%d)", n,
                    GS_NOALLOC_MAX_N);
    GS_REQUIRE(out_count != nullptr, "gs_visible_set_noalloc: null out_count");
    if (n > 0) {
        GS_REQUIRE(src && out_idx, "gs_visible_set_noalloc: null pointer");
        GS_REQUIRE(aligned(src, kind == GS_PRED_U32_NONZERO ? 16 : (kind == GS_PRED_BITMAP ? 4 : 8)),
                   "gs_visible_set_noalloc: src misaligned");
    }
    static_assert(GS_NOALLOC_SCRATCH_BYTES % 256 == 0, "scratch size");
    if (gsmi::visible_ws_bytes(n) > GS_NOALLOC_SCRATCH_BYTES)
        return fail(GS_ERR_UNSUPPORTED, "gs_visible_set_noalloc: n = %d needs more than the fixed workspace", n);
    hipError_t e = hipSuccess;
    void* ws = gsmi::noalloc_scratch(&e);
    if (ws == nullptr) return hip_status(e == hipSuccess ? hipErrorInvalidSymbol : e, "gs_visible_set_noalloc");
    return hip_status(gsmi::launch_visible(kind, src, n, out_idx, out_count, ws, static_cast<hipStream_t>(stream)),
                      "gs_visible_set_noalloc");
}

gs_status gs_bin_sort(const gs_proj* proj, int32_t n, const uint32_t* vis_idx, const uint32_t* vis_count,
                      int32_t width, int32_t height, uint32_t capacity, uint32_t* vals, uint32_t* ranges,
                      uint32_t* tile_order, uint32_t* pair_offset, uint32_t* pair_emit, uint64_t* keys,
                      uint32_t* num_pairs, gs_device_status* status, void* ws, size_t ws_bytes, void* stream) {
    gs_status s;
    if ((s = check_proj(proj, false, "gs_bin_sort")) != GS_OK) return s;
    GS_REQUIRE(n >= 0 && width >= 0 && height >= 0, "gs_bin_sort: negative size");
    if (width > GS_MAX_IMAGE_SIDE || height > GS_MAX_IMAGE_SIDE)
        return fail(GS_ERR_UNSUPPORTED, "gs_bin_sort: image side above %d", GS_MAX_IMAGE_SIDE);
    GS_REQUIRE(vis_idx && vis_count && ranges && pair_offset && num_pairs && status && ws,
               "gs_bin_sort: null pointer");
    GS_REQUIRE(capacity == 0 || (vals && pair_emit), "gs_bin_sort: null vals / pair_emit");
    GS_REQUIRE(aligned(ws, 256), "gs_bin_sort: workspace must be 256-byte aligned");
    if (ws_bytes < gsmi::binsort_ws_bytes(n, capacity, width, height))
        return fail(GS_ERR_WORKSPACE, "gs_bin_sort: workspace too small");
    return hip_status(gsmi::launch_binsort(*proj, n, vis_idx, vis_count, width, height, capacity, vals, ranges,
                                           tile_order, pair_offset, pair_emit, keys, num_pairs, status, ws,
                                           static_cast<hipStream_t>(stream)),
                      "gs_bin_sort");
}

gs_status gs_raster_fwd(const gs_proj* proj, int32_t n, const uint32_t* vals, const uint32_t* ranges,
                        const uint32_t* tile_order, int32_t width, int32_t height, const float* bg, float* img,
                        float* final_T, uint32_t* n_contrib, uint8_t* active, uint64_t* pair_stats, void* stream) {
    gs_status s;
    if ((s = check_proj(proj, false, "gs_raster_fwd")) != GS_OK) return s;
    GS_REQUIRE(n >= 0 && width >= 0 && height >= 0, "gs_raster_fwd: negative size");
    if (width > GS_MAX_IMAGE_SIDE || height > GS_MAX_IMAGE_SIDE)
        return fail(GS_ERR_UNSUPPORTED, "gs_raster_fwd: image side above %d", GS_MAX_IMAGE_SIDE);
    GS_REQUIRE(vals && ranges && bg && img && final_T && n_contrib, "gs_raster_fwd: null pointer");
    GS_REQUIRE(pair_stats == nullptr || aligned(pair_stats, 8), "gs_raster_fwd: pair_stats misaligned");
    return hip_status(gsmi::launch_raster_fwd(*proj, vals, ranges, tile_order, width, height, bg, img, final_T,
                                              n_contrib, active, pair_stats, static_cast<hipStream_t>(stream)),
                      "gs_raster_fwd");
}

gs_status gs_raster_fwd_l1(const gs_proj* proj, int32_t n, const uint32_t* vals, const uint32_t* ranges,
                           const uint32_t* tile_order, int32_t width, int32_t height, const float* bg,
                           const float* target, float* img, float* final_T, uint32_t* n_contrib, uint8_t* active,
                           float* loss, float* dL_dimg, void* ws,
                           size_t ws_bytes, void* stream) {
    gs_status s;
    if ((s = check_proj(proj, false, "gs_raster_fwd_l1")) != GS_OK) return s;
    GS_REQUIRE(n >= 0 && width >= 0 && height >= 0, "gs_raster_fwd_l1: negative size");
    if (width > GS_MAX_IMAGE_SIDE || height > GS_MAX_IMAGE_SIDE)
        return fail(GS_ERR_UNSUPPORTED, "gs_raster_fwd_l1: image side above %d", GS_MAX_IMAGE_SIDE);
    GS_REQUIRE(vals && ranges && bg && target && img && final_T && n_contrib && loss && dL_dimg && ws,
               "gs_raster_fwd_l1: null pointer");
    if (ws_bytes < gsmi::raster_fwd_l1_ws_bytes(width, height))
        return fail(GS_ERR_WORKSPACE, "gs_raster_fwd_l1: workspace too small");
    return hip_status(gsmi::launch_raster_fwd_l1(*proj, vals, ranges, tile_order, width, height, bg, target, img,
                                                 final_T, n_contrib, active, loss, dL_dimg, ws,
                                                 static_cast<hipStream_t>(stream)),
                      "gs_raster_fwd_l1");
}

gs_status gs_loss_l1(const float* img, const float* target, int32_t width, int32_t height, float* loss,
                     float* dL_dimg, void* ws, size_t ws_bytes, void* stream) {
    GS_REQUIRE(width >= 0 && height >= 0, "gs_loss_l1: negative size");
    GS_REQUIRE(img && target && loss && dL_dimg && ws, "gs_loss_l1: null pointer");
    if (ws_bytes < gsmi::loss_ws_bytes(width, height)) return fail(GS_ERR_WORKSPACE, "gs_loss_l1: workspace too small");
    return hip_status(gsmi::launch_loss_l1(img, target, width, height, loss, dL_dimg, ws,
                                           static_cast<hipStream_t>(stream)),
                      "gs_loss_l1");
}

gs_status gs_raster_bwd(const gs_scene* scene, const gs_camera* cam, const gs_proj* proj, const uint32_t* vals,
                        const uint32_t* ranges, const uint32_t* tile_order, const uint32_t* pair_offset,
                        const uint32_t* pair_emit, const uint32_t* vis_idx, const uint32_t* vis_count,
                        uint32_t capacity, const float* final_T, const uint32_t* n_contrib, const float* dL_dimg,
                        const float* bg, float* grad_rows, int32_t grad_ld, float* grad2d, float* grad_norm, void* ws,
                        size_t ws_bytes, void* stream) {
    gs_status s;
    if ((s = check_scene(scene, "gs_raster_bwd")) != GS_OK) return s;
    if ((s = check_grad_rows(scene, grad_rows, grad_ld, "gs_raster_bwd")) != GS_OK) return s;
    if ((s = check_camera(cam, "gs_raster_bwd")) != GS_OK) return s;
    if ((s = check_proj(proj, true, "gs_raster_bwd")) != GS_OK) return s;
    GS_REQUIRE(vals && ranges && pair_offset && pair_emit && vis_idx && vis_count && final_T && n_contrib && dL_dimg &&
                   bg && ws,
               "gs_raster_bwd: null pointer");
    GS_REQUIRE(aligned(ws, 256), "gs_raster_bwd: workspace must be 256-byte aligned");
    if (ws_bytes < gsmi::raster_bwd_ws_bytes(scene->n, capacity))
        return fail(GS_ERR_WORKSPACE, "gs_raster_bwd: workspace too small");
    const gsmi::CamArgs c = gsmi::make_cam_args(cam);
    return hip_status(gsmi::launch_raster_bwd(*scene, c, *proj, vals, ranges, tile_order, pair_offset, pair_emit,
                                              vis_idx, vis_count, capacity, final_T, n_contrib, dL_dimg, bg,
                                              grad_rows, grad_ld, grad2d, grad_norm, ws, 3,
                                              static_cast<hipStream_t>(stream)),
                      "gs_raster_bwd");
}

gs_status gs_raster_bwd_pixels(const gs_proj* proj, const gs_camera* cam, const uint32_t* vals, const uint32_t* ranges,
                               const uint32_t* tile_order, const uint32_t* pair_emit, uint32_t capacity,
                               const float* final_T, const uint32_t* n_contrib, const float* dL_dimg, const float* bg,
                               void* ws, size_t ws_bytes, void* stream) {
    gs_status s;
    if ((s = check_camera(cam, "gs_raster_bwd_pixels")) != GS_OK) return s;
    if ((s = check_proj(proj, false, "gs_raster_bwd_pixels")) != GS_OK) return s;
    GS_REQUIRE(vals && ranges && pair_emit && final_T && n_contrib && dL_dimg && bg && ws,
               "gs_raster_bwd_pixels: null pointer");
    GS_REQUIRE(aligned(ws, 256), "gs_raster_bwd_pixels: workspace must be 256-byte aligned");
    if (ws_bytes < gsmi::raster_bwd_ws_bytes(0, capacity))
        return fail(GS_ERR_WORKSPACE, "gs_raster_bwd_pixels: workspace too small");
    const gsmi::CamArgs c = gsmi::make_cam_args(cam);
    gs_scene none = {0, 0, nullptr, nullptr, nullptr, nullptr, nullptr};
    return hip_status(gsmi::launch_raster_bwd(none, c, *proj, vals, ranges, tile_order, nullptr, pair_emit, nullptr,
                                              nullptr, capacity, final_T, n_contrib, dL_dimg, bg, nullptr, 0, nullptr,
                                              nullptr, ws, 1, static_cast<hipStream_t>(stream)),
                      "gs_raster_bwd_pixels");
}

gs_status gs_raster_bwd_project(const gs_scene* scene, const gs_camera* cam, const gs_proj* proj,
                                const uint32_t* pair_offset, const uint32_t* vis_idx,
                                const uint32_t* vis_count, uint32_t capacity, float* grad_rows, int32_t grad_ld,
                                float* grad2d, float* grad_norm, void* ws, size_t ws_bytes, void* stream) {
    gs_status s;
    if ((s = check_scene(scene, "gs_raster_bwd_project")) != GS_OK) return s;
    if ((s = check_grad_rows(scene, grad_rows, grad_ld, "gs_raster_bwd_project")) != GS_OK) return s;
    if ((s = check_camera(cam, "gs_raster_bwd_project")) != GS_OK) return s;
    if ((s = check_proj(proj, true, "gs_raster_bwd_project")) != GS_OK) return s;
    GS_REQUIRE(pair_offset && vis_idx && vis_count && ws, "gs_raster_bwd_project: null pointer");
    GS_REQUIRE(aligned(ws, 256), "gs_raster_bwd_project: workspace must be 256-byte aligned");
    if (ws_bytes < gsmi::raster_bwd_ws_bytes(scene->n, capacity))
        return fail(GS_ERR_WORKSPACE, "gs_raster_bwd_project: workspace too small");
    const gsmi::CamArgs c = gsmi::make_cam_args(cam);
    const float bg0[3] = {0.0f, 0.0f, 0.0f};
    return hip_status(gsmi::launch_raster_bwd(*scene, c, *proj, nullptr, nullptr, nullptr, pair_offset, nullptr,
                                              vis_idx, vis_count, capacity, nullptr, nullptr, nullptr, bg0, grad_rows,
                                              grad_ld, grad2d, grad_norm, ws, 2, static_cast<hipStream_t>(stream)),
                      "gs_raster_bwd_project");
}

gs_status gs_raster_bwd_project_accum(const gs_scene* scene, const gs_camera* cam, const gs_proj* proj,
                                      const uint32_t* pair_offset, const uint32_t* vis_idx, const uint32_t* vis_count,
                                      uint32_t capacity, const uint32_t* union_idx, const uint32_t* union_count,
                                      int32_t first, float* grad_rows, int32_t grad_ld, float* grad_norm, void* ws,
                                      size_t ws_bytes, void* stream) {
    gs_status s;
    if ((s = check_scene(scene, "gs_raster_bwd_project_accum")) != GS_OK) return s;
    if ((s = check_grad_rows(scene, grad_rows, grad_ld, "gs_raster_bwd_project_accum")) != GS_OK) return s;
    if ((s = check_camera(cam, "gs_raster_bwd_project_accum")) != GS_OK) return s;
    if ((s = check_proj(proj, true, "gs_raster_bwd_project_accum")) != GS_OK) return s;
    GS_REQUIRE(pair_offset && vis_idx && vis_count && union_idx && union_count && ws,
               "gs_raster_bwd_project_accum: null pointer");
    GS_REQUIRE(aligned(ws, 256), "gs_raster_bwd_project_accum: workspace must be 256-byte aligned");
    if (ws_bytes < gsmi::raster_bwd_ws_bytes(scene->n, capacity))
        return fail(GS_ERR_WORKSPACE, "gs_raster_bwd_project_accum: workspace too small");
    const gsmi::CamArgs c = gsmi::make_cam_args(cam);
    const float bg0[3] = {0.0f, 0.0f, 0.0f};
    return hip_status(gsmi::launch_raster_bwd(*scene, c, *proj, nullptr, nullptr, nullptr, pair_offset, nullptr,
                                              vis_idx, vis_count, capacity, nullptr, nullptr, nullptr, bg0, grad_rows,
                                              grad_ld, nullptr, grad_norm, ws, 2, static_cast<hipStream_t>(stream),
                                              union_idx, union_count, first != 0),
                      "gs_raster_bwd_project_accum");
}

static gs_status check_adam(const gs_adam_group* groups, int32_t n_groups, const uint32_t* idx, const uint32_t* count,
                            int32_t max_rows, const float* grad_rows, int32_t grad_ld, const float* m, const float* v,
                            int32_t state_ld, int32_t step, double beta1, double beta2, double eps,
                            const char* what) {
    GS_REQUIRE(groups && n_groups > 0 && n_groups <= GS_MAX_GROUPS, "%s: 1..%d groups", what, GS_MAX_GROUPS);
    GS_REQUIRE(idx && count, "%s: null index list", what);
    GS_REQUIRE(grad_rows && m && v, "%s: null gradient or moment table", what);
    GS_REQUIRE(max_rows >= 0, "%s: max_rows < 0", what);
    GS_REQUIRE(step >= 1, "%s: step must be >= 1", what);
    GS_REQUIRE(beta1 >= 0.0 && beta1 < 1.0 && beta2 >= 0.0 && beta2 < 1.0, "%s: betas outside [0,1)", what);
    GS_REQUIRE(eps >= 0.0, "%s: eps < 0", what);
    int32_t row_len = 0;
    for (int i = 0; i < n_groups; ++i) {
        GS_REQUIRE(groups[i].p, "%s: group %d null", what, i);
        GS_REQUIRE(groups[i].cols > 0, "%s: group %d cols <= 0", what, i);
        GS_REQUIRE(groups[i].ld == 0 || groups[i].ld >= groups[i].cols, "%s: group %d ld %d below cols %d", what, i,
                   groups[i].ld, groups[i].cols);
        row_len += groups[i].cols;
    }
    if (row_len > 64) return fail(GS_ERR_UNSUPPORTED, "%s: row length %d above 64", what, row_len);
    GS_REQUIRE(grad_ld >= row_len && state_ld >= row_len, "%s: grad_ld and state_ld must be >= row length %d", what,
               row_len);
    return GS_OK;
}

gs_status gs_sparse_adam(const gs_adam_group* groups, int32_t n_groups, const uint32_t* idx, const uint32_t* count,
                         int32_t max_rows, const float* grad_rows, int32_t grad_ld, float* m, float* v,
                         int32_t state_ld, int32_t step, double beta1, double beta2, double eps, float* delta_rows,
                         int32_t delta_ld, void* stream) {
    gs_status s = check_adam(groups, n_groups, idx, count, max_rows, grad_rows, grad_ld, m, v, state_ld, step, beta1,
                             beta2, eps, "gs_sparse_adam");
    if (s != GS_OK) return s;
    int32_t row_len = 0;
    for (int i = 0; i < n_groups; ++i) row_len += groups[i].cols;
    GS_REQUIRE(delta_rows == nullptr || delta_ld >= row_len, "gs_sparse_adam: delta_ld must be >= row length %d",
               row_len);
    return hip_status(gsmi::launch_sparse_adam(groups, n_groups, idx, count, max_rows, grad_rows, grad_ld, m, v,
                                               state_ld, step, beta1, beta2, eps, delta_rows, delta_ld,
                                               static_cast<hipStream_t>(stream)),
                      "gs_sparse_adam");
}

gs_status gs_sparse_adam_publish(const gs_adam_group* groups, int32_t n_groups, const uint32_t* idx,
                                 const uint32_t* count, int32_t max_rows, const float* grad_rows, int32_t grad_ld,
                                 float* m, float* v, int32_t state_ld, int32_t step, double beta1, double beta2,
                                 double eps, uint32_t version, void* msg, size_t msg_capacity,
                                 gs_device_status* status, void* stream) {
    gs_status s = check_adam(groups, n_groups, idx, count, max_rows, grad_rows, grad_ld, m, v, state_ld, step, beta1,
                             beta2, eps, "gs_sparse_adam_publish");
    if (s != GS_OK) return s;
    GS_REQUIRE(msg && status, "gs_sparse_adam_publish: null message or status");
    GS_REQUIRE(aligned(msg, 16), "gs_sparse_adam_publish: msg must be 16-byte aligned");
    return hip_status(gsmi::launch_sparse_adam_publish(groups, n_groups, idx, count, max_rows, grad_rows, grad_ld, m,
                                                       v, state_ld, step, beta1, beta2, eps, version, msg,
                                                       msg_capacity, status, static_cast<hipStream_t>(stream)),
                      "gs_sparse_adam_publish");
}

static gs_status check_groups(const gs_group* g, int32_t n, const char* what) {
    GS_REQUIRE(g && n > 0 && n <= GS_MAX_GROUPS, "%s: 1..%d groups", what, GS_MAX_GROUPS);
    int32_t rl = 0;
    for (int i = 0; i < n; ++i) {
        GS_REQUIRE(g[i].ptr && g[i].cols > 0, "%s: group %d invalid", what, i);
        GS_REQUIRE(g[i].ld == 0 || g[i].ld >= g[i].cols, "%s: group %d ld %d below cols %d", what, i, g[i].ld,
                   g[i].cols);
        rl += g[i].cols;
    }
    if (rl > 64) return fail(GS_ERR_UNSUPPORTED, "%s: row length %d above 64", what, rl);
    return GS_OK;
}

gs_status gs_delta_pack(const uint32_t* idx, const uint32_t* count, int32_t max_rows, const gs_group* src,
                        int32_t n_groups, uint32_t version, void* msg, size_t msg_capacity, gs_device_status* status,
                        void* stream) {
    gs_status s;
    if ((s = check_groups(src, n_groups, "gs_delta_pack")) != GS_OK) return s;
    GS_REQUIRE(idx && count && msg && status, "gs_delta_pack: null pointer");
    GS_REQUIRE(max_rows >= 0, "gs_delta_pack: max_rows < 0");
    GS_REQUIRE(aligned(msg, 16), "gs_delta_pack: msg must be 16-byte aligned");
    return hip_status(gsmi::launch_delta_pack(idx, count, max_rows, src, n_groups, version, msg, msg_capacity, status,
                                              static_cast<hipStream_t>(stream)),
                      "gs_delta_pack");
}

gs_status gs_delta_apply(const void* msg, size_t msg_capacity, const gs_group* dst, int32_t n_groups, int32_t n_rows,
                         int32_t max_rows, int32_t mode, uint32_t* prim_version, gs_device_status* status,
                         void* stream) {
    gs_status s;
    if ((s = check_groups(dst, n_groups, "gs_delta_apply")) != GS_OK) return s;
    GS_REQUIRE(msg && status, "gs_delta_apply: null pointer");
    GS_REQUIRE(msg_capacity >= gsmi::delta_msg_bytes(0, 0, n_groups), "gs_delta_apply: message buffer below header size");
    GS_REQUIRE(mode == GS_APPLY_ADD || mode == GS_APPLY_OVERWRITE, "gs_delta_apply: bad mode %d", mode);
    GS_REQUIRE(n_rows >= 0 && max_rows >= 0, "gs_delta_apply: negative size");
    GS_REQUIRE(aligned(msg, 16), "gs_delta_apply: msg must be 16-byte aligned");
    return hip_status(gsmi::launch_delta_apply(msg, msg_capacity, dst, n_groups, n_rows, max_rows, mode, prim_version, status,
                                               static_cast<hipStream_t>(stream)),
                      "gs_delta_apply");
}

gs_status gs_publish_commit(const gs_ring* ring, uint32_t version, const gs_group* dst, int32_t n_groups,
                            int32_t n_rows, int32_t max_rows, int32_t mode, uint32_t* prim_version, uint32_t* skip,
                            gs_device_status* status, void* stream) {
    gs_status s;
    if ((s = check_groups(dst, n_groups, "gs_publish_commit")) != GS_OK) return s;
    GS_REQUIRE(ring && ring->slot[0] && ring->slot[1] && ring->state, "gs_publish_commit: null ring");
    GS_REQUIRE(aligned(ring->slot[0], 16) && aligned(ring->slot[1], 16), "gs_publish_commit: slots must be 16-byte aligned");
    GS_REQUIRE(ring->slot_bytes >= gsmi::delta_msg_bytes(0, 0, n_groups),
               "gs_publish_commit: slots below the message header size");
    GS_REQUIRE(prim_version && status, "gs_publish_commit: null prim_version / status");
    GS_REQUIRE(version >= 1, "gs_publish_commit: version 0");
    GS_REQUIRE(mode == GS_APPLY_ADD || mode == GS_APPLY_OVERWRITE, "gs_publish_commit: bad mode %d", mode);
    GS_REQUIRE(n_rows >= 0 && max_rows >= 0, "gs_publish_commit: negative size");
    return hip_status(gsmi::launch_publish_commit(*ring, version, dst, n_groups, n_rows, max_rows, mode, prim_version,
                                                  skip, status, static_cast<hipStream_t>(stream)),
                      "gs_publish_commit");
}

gs_status gs_scope_from_ids(const uint32_t* idx, const uint32_t* count, int32_t max_rows, int32_t n,
                            int32_t accumulate, uint32_t* scope, void* stream) {
    GS_REQUIRE(n >= 0 && max_rows >= 0, "gs_scope_from_ids: negative size");
    if (n == 0) return ok();
    GS_REQUIRE(scope != nullptr, "gs_scope_from_ids: null scope");
    GS_REQUIRE(max_rows == 0 || (idx && count), "gs_scope_from_ids: null idx / count");
    return hip_status(gsmi::launch_scope_from_ids(idx, count, max_rows, n, accumulate != 0, scope,
                                                  static_cast<hipStream_t>(stream)),
                      "gs_scope_from_ids");
}

gs_status gs_scope_from_pred(int32_t kind, const void* src, int32_t n, int32_t accumulate, uint32_t* scope,
                             void* stream) {
    GS_REQUIRE(kind == GS_PRED_U32_NONZERO || kind == GS_PRED_U8_NONZERO, "gs_scope_from_pred: bad kind %d", kind);
    GS_REQUIRE(n >= 0, "gs_scope_from_pred: n < 0");
    if (n == 0) return ok();
    GS_REQUIRE(src && scope, "gs_scope_from_pred: null pointer");
    return hip_status(gsmi::launch_scope_from_pred(kind, src, n, accumulate != 0, scope,
                                                   static_cast<hipStream_t>(stream)),
                      "gs_scope_from_pred");
}

gs_status gs_scope_conflicts(const uint32_t* RA, const uint32_t* WA, const uint32_t* RB, const uint32_t* WB,
                             int32_t n, uint32_t* waw, uint32_t* raw, uint32_t* war, uint32_t* waw_idx,
                             uint32_t* raw_idx, uint32_t* war_idx, uint32_t* counts, void* ws, size_t ws_bytes,
                             void* stream) {
    GS_REQUIRE(n >= 0, "gs_scope_conflicts: n < 0");
    GS_REQUIRE(counts != nullptr, "gs_scope_conflicts: null counts");
    if (n > 0) GS_REQUIRE(RA && WA && RB && WB && ws, "gs_scope_conflicts: null scope or workspace");
    if (ws_bytes < gsmi::scope_ws_bytes(n)) return fail(GS_ERR_WORKSPACE, "gs_scope_conflicts: workspace too small");
    return hip_status(gsmi::launch_scope_conflicts(RA, WA, RB, WB, n, waw, raw, war, waw_idx, raw_idx, war_idx,
                                                   counts, ws, static_cast<hipStream_t>(stream)),
                      "gs_scope_conflicts");
}

gs_status gs_admission_gate(const uint32_t* RB, const uint32_t* D, const gs_gate_args* args, int32_t n,
                            gs_gate_result* result, void* ws, size_t ws_bytes, void* stream) {
    GS_REQUIRE(n >= 0, "gs_admission_gate: n < 0");
    GS_REQUIRE(args != nullptr && result != nullptr && ws != nullptr, "gs_admission_gate: null pointer");
    GS_REQUIRE(args->tau >= 0.0 && args->tau <= 1.0, "gs_admission_gate: tau outside [0, 1]");
    GS_REQUIRE(args->skip == nullptr || args->producer_version != 0,
               "gs_admission_gate: metadata given without a producer version");
    if (n > 0) GS_REQUIRE(RB && D && args->active && args->g, "gs_admission_gate: null scope or evidence");
    if (ws_bytes < gsmi::scope_ws_bytes(n)) return fail(GS_ERR_WORKSPACE, "gs_admission_gate: workspace too small");
    return hip_status(gsmi::launch_admission_gate(RB, D, *args, n, result, ws, static_cast<hipStream_t>(stream)),
                      "gs_admission_gate");
}

gs_status gs_rlg_build(int32_t n_items, int32_t n_tracks, const int64_t* item_ptr, const int32_t* item_tracks,
                       int32_t track_cap, int32_t top_k, int64_t* edge_ptr, int32_t* edge_dst, double* edge_w,
                       int64_t edge_capacity, int64_t* n_edges) {
    GS_REQUIRE(n_items >= 0 && n_tracks >= 0, "gs_rlg_build: negative size");
    GS_REQUIRE(item_ptr && edge_ptr && n_edges, "gs_rlg_build: null pointer");
    GS_REQUIRE(item_tracks || item_ptr[n_items] == 0, "gs_rlg_build: null item_tracks");
    GS_REQUIRE(edge_capacity >= 0 && ((edge_dst && edge_w) || edge_capacity == 0),
               "gs_rlg_build: null edge arrays");
    char msg[160] = "";
    const int s = gsmi::rlg_build(n_items, n_tracks, item_ptr, item_tracks, track_cap, top_k, edge_ptr, edge_dst,
                                  edge_w, edge_capacity, n_edges, msg, sizeof msg);
    if (s == GS_ERR_WORKSPACE)
        return fail(GS_ERR_WORKSPACE, "gs_rlg_build: %lld edge entries needed, %lld available",
                    (long long)*n_edges, (long long)edge_capacity);
    if (s != GS_OK) return fail((gs_status)s, "gs_rlg_build: %s", msg);
    return ok();
}

gs_status gs_lp_partition(int32_t n_items, const double* position, const int64_t* edge_ptr,
                          const int32_t* edge_dst, const double* edge_w, int32_t K, int32_t max_iters,
                          int32_t* group, double* coupling, int32_t* iters_run) {
    GS_REQUIRE(n_items >= 0, "gs_lp_partition: n_items < 0");
    GS_REQUIRE(K >= 1 && max_iters >= 1, "gs_lp_partition: K and max_iters must be >= 1");
    GS_REQUIRE(edge_ptr && coupling && iters_run, "gs_lp_partition: null pointer");
    if (n_items > 0) GS_REQUIRE(position && group, "gs_lp_partition: null pointer");
    GS_REQUIRE(edge_ptr[n_items] == 0 || (edge_dst && edge_w), "gs_lp_partition: null edge arrays");
    char msg[160] = "";
    const int s = gsmi::lp_partition(n_items, position, edge_ptr, edge_dst, edge_w, K, max_iters, group, coupling,
                                     iters_run, msg, sizeof msg);
    if (s != GS_OK) return fail((gs_status)s, "gs_lp_partition: %s", msg);
    return ok();
}

gs_status gs_sds_order(int32_t n_items, const int32_t* group, int32_t K, const double* coupling,
                       const int64_t* edge_ptr, const int32_t* edge_dst, const double* edge_w, int32_t unit_size,
                       int32_t* cycle, int32_t* n_cycle, int32_t* order, int32_t* unit_group, double* transition,
                       int32_t* n_units) {
    GS_REQUIRE(n_items >= 0, "gs_sds_order: n_items < 0");
    GS_REQUIRE(K >= 1 && unit_size >= 1, "gs_sds_order: K and unit_size must be >= 1");
    GS_REQUIRE(coupling && edge_ptr && cycle && n_cycle && n_units, "gs_sds_order: null pointer");
    if (n_items > 0) GS_REQUIRE(group && order && unit_group && transition, "gs_sds_order: null pointer");
    GS_REQUIRE(edge_ptr[n_items] == 0 || (edge_dst && edge_w), "gs_sds_order: null edge arrays");
    char msg[160] = "";
    const int s = gsmi::sds_order(n_items, group, K, coupling, edge_ptr, edge_dst, edge_w, unit_size, cycle,
                                  n_cycle, order, unit_group, transition, n_units, msg, sizeof msg);
    if (s != GS_OK) return fail((gs_status)s, "gs_sds_order: %s", msg);
    return ok();
}

}  // extern "C"
