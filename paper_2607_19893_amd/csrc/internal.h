// Launch wrappers shared between the kernel files and the C-ABI layer.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/gsmi.h"
#include "planner.h"

namespace gsmi {

struct CamArgs {
    int32_t width, height, tiles_x, tiles_y;
    float fx, fy, cx, cy, tan_fovx, tan_fovy, near_z;
    float R[9];
    float t[3];
    float campos[3];
};

CamArgs make_cam_args(const gs_camera* c);

// Row strides (floats) of the pool's groups, the dense widths filled in for 0.
struct SceneLd {
    int32_t mean, log_scale, quat, opacity, sh;
    int32_t head;   // 1: log_scale and opacity are floats 4..7 of quat's 16-byte-aligned row
};

inline SceneLd scene_ld(const gs_scene& s) {
    const int32_t K3 = 3 * (s.sh_degree + 1) * (s.sh_degree + 1);
    SceneLd l;
    l.mean = s.ld_mean ? s.ld_mean : 3;
    l.log_scale = s.ld_log_scale ? s.ld_log_scale : 3;
    l.quat = s.ld_quat ? s.ld_quat : 4;
    l.opacity = s.ld_opacity ? s.ld_opacity : 1;
    l.sh = s.ld_sh ? s.ld_sh : K3;
    l.head = s.log_scale == s.quat + 4 && s.opacity == s.quat + 7 && l.log_scale == l.quat &&
             l.opacity == l.quat && l.quat % 4 == 0;
    return l;
}

// Compute units of the current device (cached per device; 0 if the query fails).
uint32_t compute_units();

// project.hip
hipError_t launch_project(const gs_scene& s, const CamArgs& cam, const gs_proj& out, hipStream_t st);

// compact.hip
size_t visible_ws_bytes(int32_t n);
hipError_t launch_visible(int kind, const void* src, int32_t n, uint32_t* out_idx, uint32_t* out_count, void* ws,
                          hipStream_t st);
hipError_t launch_fill_u32(uint32_t* p, uint32_t value, size_t n, hipStream_t st);
// Device address of the fixed visible-set workspace on the current device
// (GS_NOALLOC_SCRATCH_BYTES, 256-byte aligned); nullptr with *err set if the
// lookup fails.  Allocates nothing.
void* noalloc_scratch(hipError_t* err);

// binsort.hip
size_t binsort_ws_bytes(int32_t n, uint32_t capacity, int32_t width, int32_t height);
hipError_t launch_binsort(const gs_proj& proj, int32_t n, const uint32_t* vis_idx, const uint32_t* vis_count,
                          int32_t width, int32_t height, uint32_t capacity, uint32_t* vals, uint32_t* ranges,
                          uint32_t* tile_order, uint32_t* pair_offset, uint32_t* pair_emit, uint64_t* keys,
                          uint32_t* num_pairs, gs_device_status* status, void* ws, hipStream_t st);

// raster.hip
hipError_t launch_raster_fwd(const gs_proj& proj, const uint32_t* vals, const uint32_t* ranges,
                             const uint32_t* tile_order, int32_t width, int32_t height, const float bg[3],
                             float* img, float* final_T, uint32_t* n_contrib, uint8_t* active, uint64_t* pair_stats,
                             hipStream_t st);
size_t raster_fwd_l1_ws_bytes(int32_t width, int32_t height);
hipError_t launch_raster_fwd_l1(const gs_proj& proj, const uint32_t* vals, const uint32_t* ranges,
                                const uint32_t* tile_order, int32_t width, int32_t height, const float bg[3],
                                const float* target, float* img, float* final_T, uint32_t* n_contrib, uint8_t* active,
                                float* loss, float* dL, void* ws, hipStream_t st);
size_t loss_ws_bytes(int32_t width, int32_t height);
hipError_t launch_loss_l1(const float* img, const float* target, int32_t width, int32_t height, float* loss,
                          float* dL, void* ws, hipStream_t st);
size_t raster_bwd_ws_bytes(int32_t n, uint32_t capacity);
hipError_t launch_raster_bwd(const gs_scene& scene, const CamArgs& cam, const gs_proj& proj, const uint32_t* vals,
                             const uint32_t* ranges, const uint32_t* tile_order, const uint32_t* pair_offset,
                             const uint32_t* pair_emit,
                             const uint32_t* vis_idx, const uint32_t* vis_count, uint32_t capacity,
                             const float* final_T, const uint32_t* n_contrib, const float* dL_dimg, const float bg[3],
                             float* grad_rows, int32_t grad_ld, float* grad2d, float* grad_norm, void* ws, int stages,
                             hipStream_t st, const uint32_t* union_idx = nullptr,
                             const uint32_t* union_count = nullptr, int first = 0);

// adam.hip
hipError_t launch_sparse_adam(const gs_adam_group* groups, int32_t n_groups, const uint32_t* idx,
                              const uint32_t* count, int32_t max_rows, const float* grad_rows, int32_t grad_ld,
                              float* m, float* v, int32_t state_ld, int32_t step, double beta1, double beta2,
                              double eps, float* delta_rows, int32_t delta_ld, hipStream_t st);
hipError_t launch_sparse_adam_publish(const gs_adam_group* groups, int32_t n_groups, const uint32_t* idx,
                                      const uint32_t* count, int32_t max_rows, const float* grad_rows,
                                      int32_t grad_ld, float* m, float* v, int32_t state_ld, int32_t step,
                                      double beta1, double beta2, double eps, uint32_t version, void* msg,
                                      size_t msg_capacity, gs_device_status* status, hipStream_t st);

// scope.hip
size_t scope_ws_bytes(int32_t n);
hipError_t launch_scope_from_ids(const uint32_t* idx, const uint32_t* count, int32_t max_rows, int32_t n,
                                 int32_t accumulate, uint32_t* scope, hipStream_t st);
hipError_t launch_scope_from_pred(int kind, const void* src, int32_t n, int32_t accumulate, uint32_t* scope,
                                  hipStream_t st);
hipError_t launch_scope_conflicts(const uint32_t* RA, const uint32_t* WA, const uint32_t* RB, const uint32_t* WB,
                                  int32_t n, uint32_t* waw, uint32_t* raw, uint32_t* war, uint32_t* waw_idx,
                                  uint32_t* raw_idx, uint32_t* war_idx, uint32_t* counts, void* ws, hipStream_t st);
hipError_t launch_admission_gate(const uint32_t* RB, const uint32_t* D, const gs_gate_args& a, int32_t n,
                                 gs_gate_result* result, void* ws, hipStream_t st);

// delta.hip
size_t delta_msg_bytes(uint64_t count, int32_t row_len, int32_t n_groups);
hipError_t launch_delta_pack(const uint32_t* idx, const uint32_t* count, int32_t max_rows, const gs_group* src,
                             int32_t n_groups, uint32_t version, void* msg, size_t msg_capacity,
                             gs_device_status* status, hipStream_t st);
hipError_t launch_publish_commit(const gs_ring& ring, uint32_t version, const gs_group* dst, int32_t n_groups,
                                 int32_t n_rows, int32_t max_rows, int32_t mode, uint32_t* prim_version,
                                 uint32_t* skip, gs_device_status* status, hipStream_t st);
hipError_t launch_delta_apply(const void* msg, size_t msg_capacity, const gs_group* dst, int32_t n_groups,
                              int32_t n_rows, int32_t max_rows, int32_t mode, uint32_t* prim_version,
                              gs_device_status* status, hipStream_t st);

}  // namespace gsmi
