/*
 * gsmi.h -- C ABI of the MI355X (gfx950) 3D Gaussian Splatting training-view
 * hot path: one view of point-based neural rendering training on one GPU's
 * share of the primitive pool, plus the primitive-indexed publication steps
 * that a primitive-level synchronization runtime drives.
 *
 * The paper frames a training view as: render one camera, compute an image
 * loss, back-propagate, and update only the primitives that participate; the
 * pool is a set of aligned per-primitive tensors whose dependency unit is the
 * primitive index (Introduction; Section 2.1).  The renderer is the cited
 * 3D Gaussian Splatting method.  Each call below is one phase of that view
 * (Section 4.1.2 lists the phases: scope extraction, preprocessing,
 * rendering, backward, communication, optimizer update) or one of the
 * runtime's publication steps (Section 4.3, Shadow Graph; Section 5 hooks).
 *
 * Conventions for every call:
 *  - All array pointers are DEVICE pointers owned by the caller; the library
 *    never allocates, frees, or keeps them.  Host-side structs (gs_scene,
 *    gs_camera, gs_proj, gs_group, gs_adam_group) are read during the call
 *    only.
 *  - Every call is asynchronous on `stream` (a hipStream_t passed as void*;
 *    NULL = the default stream) and never synchronizes the host.
 *  - Argument problems are reported synchronously as a gs_status and nothing
 *    is enqueued.  Data-dependent conditions found on the device (a pair list
 *    or message larger than its buffer, a message that does not match its
 *    destination) are reported through a gs_device_status in device memory;
 *    the outputs of that call are then undefined and the caller retries with
 *    larger buffers after its next synchronization.
 *  - Counts produced on the device (visible-set size, pair count) stay on the
 *    device; later calls read them from there.
 *  - Row-major layouts: a "[n,c]" array holds row i at elements [i*c, i*c+c);
 *    "[n,c] with leading dimension ld" (written [n,ld]) at [i*ld, i*ld+c).
 *  - Thread safety: calls on different streams may run concurrently if they
 *    do not share output buffers.
 */
#ifndef GSMI_H
#define GSMI_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define GSMI_ABI_VERSION 4
#define GS_TILE 16            /* pixels per tile side */
#define GS_MAX_SH_DEGREE 3
#define GS_MAX_GROUPS 8
#define GS_MAX_IMAGE_SIDE 32768

typedef enum {
    GS_OK = 0,
    GS_ERR_INVALID_ARG = 1,   /* null pointer, negative size, bad enum, ... */
    GS_ERR_UNSUPPORTED = 2,   /* size beyond a documented limit */
    GS_ERR_WORKSPACE = 3,     /* workspace smaller than gs_workspace_bytes() */
    GS_ERR_HIP = 4            /* the HIP runtime refused a launch */
} gs_status;

/* Device-side error channel (16 bytes of device memory, caller-zeroed). */
typedef struct {
    uint32_t flags;           /* OR of GS_DEV_* */
    uint32_t required;        /* elements (pairs) or bytes (messages) needed */
    uint32_t reserved[2];
} gs_device_status;

#define GS_DEV_PAIR_OVERFLOW 1u     /* gs_bin_sort: pairs > capacity */
#define GS_DEV_MSG_OVERFLOW 2u      /* gs_delta_pack, gs_sparse_adam_publish: message > msg_capacity */
#define GS_DEV_MSG_MISMATCH 4u      /* gs_delta_apply, gs_publish_commit: bad magic / widths / ids / version */
#define GS_DEV_MSG_ORDER 8u         /* gs_publish_commit: not the version after the last committed one */

/*
 * Primitive pool Theta (Section 2.1): five aligned fp32 tensors, one row per
 * primitive.
 *   mean      [n,3] world position
 *   log_scale [n,3] log standard deviation per axis
 *   quat      [n,4] rotation quaternion (w,x,y,z), any non-zero length
 *   opacity   [n]   opacity logit
 *   sh        [n,(sh_degree+1)^2,3] colour coefficients, coefficient
 *             k = l*l + l + m (m = -l..l), channel fastest
 * Row i of a group starts ld_<group> floats after row i-1 (0 = the group's
 * width, a dense tensor), so groups may be column ranges of one table: with
 * quat, log_scale and opacity as floats 0..3, 4..6 and 7 of a [n, 8] table
 * (ld 8 for all three) a primitive's geometry and opacity are one 32-byte
 * record, read and updated as one memory segment.  quat and sh
 * must be 16-byte aligned; ld_quat a multiple of 4, ld_sh the dense width
 * 3(sh_degree+1)^2 or a multiple of 4 above it.
 */
typedef struct {
    int32_t n;
    int32_t sh_degree;        /* 0..3 */
    float* mean;
    float* log_scale;
    float* quat;
    float* opacity;
    float* sh;
    int32_t ld_mean, ld_log_scale, ld_quat, ld_opacity, ld_sh;
} gs_scene;

/*
 * Pinhole camera (host struct, by pointer): world-to-camera rotation R
 * (row-major; rows = right, down, forward), translation t, centre campos,
 * focal lengths, principal point, tangents of the half fields of view and
 * the near plane.  Pixel (i,k) is centred at (i+0.5, k+0.5).
 */
typedef struct {
    int32_t width, height;
    float fx, fy, cx, cy;
    float tan_fovx, tan_fovy;
    float near_z;
    float R[9];
    float t[3];
    float campos[3];
} gs_camera;

/*
 * Per-primitive projection results ([n] rows; device).  Culled primitives
 * have radius = 0 and tiles = 0; their other rows are not written.
 *   radius        [n]   int32   3-sigma pixel radius
 *   tiles         [n]   uint32  number of 16x16 tiles the radius touches
 *   rect          [n,4] uint16  tile rectangle x0,y0,x1,y1 (half-open)
 *   depth         [n]   fp32    camera-space z
 *   mean2d        [n,2] fp32    pixel-space mean
 *   conic_opacity [n,4] fp32    inverse 2D covariance (A,B,C) and opacity
 *   rgb           [n,3] fp32    view-dependent colour
 *   clamp         [n]   uint8   bit c set: colour channel c was clamped at 0
 */
typedef struct {
    int32_t* radius;
    uint32_t* tiles;
    uint16_t* rect;
    float* depth;
    float* mean2d;
    float* conic_opacity;
    float* rgb;
    uint8_t* clamp;
} gs_proj;

/* ---------------------------------------------------------------------- */

int32_t gs_abi_version(void);
const char* gs_status_string(int32_t status);
/* Message of the last synchronous error on this thread ("" if none). */
const char* gs_last_error(void);

enum {
    GS_WS_VISIBLE_SET = 1,
    GS_WS_BIN_SORT = 2,
    GS_WS_RASTER_BWD = 3,
    GS_WS_LOSS = 4,
    GS_WS_SCOPE = 5,
    GS_WS_RASTER_FWD_L1 = 6
};
/*
 * Workspace bytes a call needs, for a pool of n primitives, a pair capacity
 * (gs_bin_sort, gs_raster_bwd) and an image size.  Workspaces are caller-
 * owned device memory, 256-byte aligned; only the gs_raster_bwd_pixels ->
 * gs_raster_bwd_project pair hands data from one call to the next.
 */
size_t gs_workspace_bytes(int32_t which, int32_t n, uint32_t capacity, int32_t width, int32_t height);

/*
 * Phase "preprocessing" (Section 4.1.2; P in Figure 6): EWA projection of
 * every primitive of `scene` into `cam`, with spherical-harmonic colour
 * evaluated along the viewing direction.  The geometry that decides radius,
 * tile rectangle and depth is computed in fp32 in a fixed operation order
 * (no fused multiply-add) so that it is reproducible bit for bit:
 *   p = R mu + t (cull if p_z <= near_z); s = exp(log_scale); Sigma = (Rq S)(Rq S)^T
 *   J from p with x/z, y/z clamped to +-1.3 tan_fov; Sigma2D = J R Sigma R^T J^T + 0.3 I
 *   conic = Sigma2D^-1 (cull if det <= 0); r = ceil(3 sqrt(mid + sqrt(max(0.1, mid^2 - det))))
 *   u = fx p_x/p_z + cx, v = fy p_y/p_z + cy; rectangle from (u +- r)/16 (cull if empty)
 * opacity = sigmoid(logit); rgb = max(0, SH(d) + 0.5), d = (mu - campos)/|mu - campos|.
 * Errors: GS_ERR_INVALID_ARG on null pointers, n < 0, degree outside 0..3;
 * GS_ERR_UNSUPPORTED if width/height exceed GS_MAX_IMAGE_SIDE.
 */
gs_status gs_project(const gs_scene* scene, const gs_camera* cam, const gs_proj* out, void* stream);

/*
 * Scope extraction (Section 4.1.2) and the pre-observation / post-backward
 * scope hooks (Section 5): ordered stream compaction of a per-primitive
 * predicate into ascending primitive ids.  With `tiles` from gs_project the
 * result is the projection-visible set (a superset of the realized active
 * set C_i of Section 2.1); with the active flags of gs_raster_fwd it is C_i
 * itself; any caller mask works the same way.
 *   kind: GS_PRED_U32_NONZERO (src is uint32[n]), GS_PRED_U8_NONZERO (uint8[n])
 *     or GS_PRED_BITMAP (src is a scope bitmap, see gs_scope_from_ids);
 *     GS_PRED_U8_NONZERO_CLEAR compacts uint8[n] flags as GS_PRED_U8_NONZERO
 *     and also sets every flag it finds nonzero back to 0: flags that a
 *     forward marks afresh for each view then need no separate clear before
 *     the next marking.  src is then written, so it must be writable device
 *     memory (it is declared const for the kinds that only read it).
 *   src: 16-byte aligned for GS_PRED_U32_NONZERO, 8 for the uint8 kinds, 4
 *     for the bitmap (else GS_ERR_INVALID_ARG)
 *   out_idx [n] uint32 (the first *out_count entries are written)
 *   out_count: one uint32 on the device
 *   ws: gs_workspace_bytes(GS_WS_VISIBLE_SET, n, 0, 0, 0) bytes, 256-byte
 *     aligned (else GS_ERR_INVALID_ARG)
 */
enum { GS_PRED_U32_NONZERO = 0, GS_PRED_U8_NONZERO = 1, GS_PRED_BITMAP = 2, GS_PRED_U8_NONZERO_CLEAR = 3 };
gs_status gs_visible_set(int32_t kind, const void* src, int32_t n, uint32_t* out_idx, uint32_t* out_count,
                         void* ws, size_t ws_bytes, void* stream);

/*
 * gs_visible_set for callers that cannot allocate device memory: code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc.
 * Same arguments and results as gs_visible_set, without the workspace: the
 * compaction's block counts live in a fixed buffer of
 * GS_NOALLOC_SCRATCH_BYTES that the library holds on every GPU it runs on
 * until the process ends (looked up, not allocated, on the first call on each
 * device).  The call allocates nothing.
 *   n <= GS_NOALLOC_MAX_N, else GS_ERR_UNSUPPORTED and nothing is enqueued.
 * Every call on one GPU shares that GPU's buffer, which keeps the last call's
 * contents (each call writes every word it reads, so nothing needs clearing):
 * calls that can overlap on one GPU (different streams, or threads without
 * ordering) race, and the caller must serialize them.
 */
#define GS_NOALLOC_SCRATCH_BYTES 262144
#define GS_NOALLOC_MAX_N 134215680    /* (GS_NOALLOC_SCRATCH_BYTES / 4 - 1) blocks of 2048 ids */
gs_status gs_visible_set_noalloc(int32_t kind, const void* src, int32_t n, uint32_t* out_idx, uint32_t* out_count,
                                 void* stream);

/*
 * Phase "rendering", part 1 (Section 4.1.2): duplicate every visible
 * primitive once per touched tile and order the (tile, primitive) pairs by
 * (tile, depth, primitive id).  Equal depths keep ascending ids.
 *   vis_idx/vis_count: ascending visible ids (gs_visible_set on `tiles`); ids
 *     whose tile count is 0 may be in the list too (they emit no pair)
 *   capacity: length of vals (and keys); more pairs set GS_DEV_PAIR_OVERFLOW,
 *     emit no pair (every range empty) and set pair_offset to 0xFFFFFFFF for
 *     the listed ids, so that gs_raster_bwd_project reads no pair slot and
 *     writes zero gradient rows
 *   vals   [capacity] uint32  primitive id of every sorted pair
 *   ranges [T,2] uint32       [start, end) of each tile's pairs, T = tiles in the image
 *   tile_order [T] uint32 or NULL: a dispatch order for the per-tile kernels,
 *                             the tile ids by pair count descending (counts
 *                             compared through an 8-bit code: exact below 16,
 *                             then 16 steps per octave, one code from 2^19 on),
 *                             equal codes by ascending id.  It changes no result
 *                             of any call that takes it; it lets the longest
 *                             tiles start first.  Written even when there are
 *                             no pairs (then it is 0..T-1).
 *   pair_offset [n] uint32    per visible primitive: first of its pairs in
 *                             emission order (primitives in ascending id order, each one's
 *                             rectangle row-major); read by gs_raster_bwd
 *   pair_emit [capacity] uint32  emission position of every sorted pair
 *                             (pair_offset[id] + tile number in id's rectangle)
 *   keys   [capacity] uint64 or NULL: (tile << 32) | bits(depth) per sorted pair
 *   num_pairs: one uint32 on the device (the pair count, also on overflow)
 *   ws: gs_workspace_bytes(GS_WS_BIN_SORT, n, capacity, width, height) bytes,
 *     256-byte aligned (else GS_ERR_INVALID_ARG)
 */
gs_status gs_bin_sort(const gs_proj* proj, int32_t n, const uint32_t* vis_idx, const uint32_t* vis_count,
                      int32_t width, int32_t height, uint32_t capacity, uint32_t* vals, uint32_t* ranges,
                      uint32_t* tile_order, uint32_t* pair_offset, uint32_t* pair_emit, uint64_t* keys,
                      uint32_t* num_pairs, gs_device_status* status, void* ws, size_t ws_bytes, void* stream);

/*
 * Phase "rendering", part 2 (R in Figure 6): front-to-back alpha blending of
 * each pixel over its tile's sorted pairs.  Per pair: sigma = A dx^2/2 +
 * B dx dy + C dy^2/2 (dx = u - px, pixel centres at +0.5), skipped if
 * sigma < 0; alpha = min(0.99, o e^-sigma), skipped if alpha < 1/255; the pixel
 * stops before a pair that would take T(1-alpha) below 1e-4.
 *   img [3,H,W] fp32 planar = sum alpha T rgb + T_final bg
 *   final_T [H,W] fp32; n_contrib [H,W] uint32 = 1 + position (within the tile's
 *   range) of the last included pair, 0 if none
 *   active [n] uint8 or NULL: set to 1 for every primitive included in at least
 *   one pixel (never cleared: zero it before the call)
 *   pair_stats [4] uint64 or NULL (accumulated: zero it before the call):
 *   += number of (pixel, pair) evaluations, of included pairs, of (row, pair)
 *   steps the kernel executed (a row is 16 pixels of a tile row, the unit the
 *   kernel walks pairs in), and of those steps in which at least one pixel
 *   included the pair
 *   bg: 3 floats on the HOST
 *   tile_order [T] uint32 or NULL: the order in which workgroups take the
 *   tiles (gs_bin_sort's tile_order, any permutation of 0..T-1, or NULL for
 *   row-major); results do not depend on it.  Entries >= T are skipped.
 */
gs_status gs_raster_fwd(const gs_proj* proj, int32_t n, const uint32_t* vals, const uint32_t* ranges,
                        const uint32_t* tile_order, int32_t width, int32_t height, const float* bg, float* img,
                        float* final_T, uint32_t* n_contrib, uint8_t* active, uint64_t* pair_stats, void* stream);

/*
 * gs_raster_fwd followed by gs_loss_l1 in one pass over the image (the
 * render and the image loss of one training view, Section 2.1): img, final_T,
 * n_contrib and active are gs_raster_fwd's; dL_dimg is gs_loss_l1's, bit for
 * bit (the same fp32 comparison per channel); loss is the same mean, summed
 * per 16x16 tile and then over the tiles in fp64, so it can differ from
 * gs_loss_l1's value in the last fp32 bits.
 *   target [3,H,W] fp32; loss: one float on the device; tile_order as in gs_raster_fwd
 *   ws: gs_workspace_bytes(GS_WS_RASTER_FWD_L1, 0, 0, W, H) bytes
 */
gs_status gs_raster_fwd_l1(const gs_proj* proj, int32_t n, const uint32_t* vals, const uint32_t* ranges,
                           const uint32_t* tile_order, int32_t width, int32_t height, const float* bg,
                           const float* target, float* img, float* final_T, uint32_t* n_contrib, uint8_t* active,
                           float* loss, float* dL_dimg, void* ws, size_t ws_bytes, void* stream);

/*
 * Image loss (Section 2.1): L = mean over all 3*H*W entries of |img - target|;
 * dL_dimg = sign(img - target) / (3HW) with sign(0) = 0.
 *   loss: one float on the device; ws: gs_workspace_bytes(GS_WS_LOSS, 0, 0, W, H)
 */
gs_status gs_loss_l1(const float* img, const float* target, int32_t width, int32_t height, float* loss,
                     float* dL_dimg, void* ws, size_t ws_bytes, void* stream);

/*
 * Phase "backward" (B in Figure 6; Shadow Graph step 2 of Section 4.3): the
 * analytic derivative of the rendered view, first w.r.t. each pair's 2D
 * quantities (replayed back to front per pixel from final_T and n_contrib),
 * summed per primitive in a fixed order, then
 * chained through projection and colour to the parameters.  grad_norm is the
 * per-primitive gradient evidence g(p) of Section 2.1 that the post-backward
 * hook of Section 5 reports: |dL/d(u,v)| of this view.
 *   grad_rows [V,grad_ld] fp32: one record per visible row r (the r-th entry
 *     of vis_idx, V = *vis_count): [dmean 3, dlog_scale 3, dquat 4, dopacity 1,
 *     dsh 3(L+1)^2] (row_len = 11 + 3(L+1)^2 floats, the pool's groups in
 *     order); columns row_len..grad_ld-1 are set to 0.  grad_ld is a multiple
 *     of 4 and >= row_len; grad_rows is 16-byte aligned and holds n rows.
 *   grad2d [n,9] fp32 or NULL: (du, dv, dA, dB, dC, dopacity, dr, dg, db) per visible id
 *   grad_norm [n] fp32 or NULL (visible ids)
 *   ws: gs_workspace_bytes(GS_WS_RASTER_BWD, n, capacity, W, H); capacity as in gs_bin_sort
 *   tile_order: as in gs_raster_fwd (the per-pixel replay's dispatch order)
 */
gs_status gs_raster_bwd(const gs_scene* scene, const gs_camera* cam, const gs_proj* proj, const uint32_t* vals,
                        const uint32_t* ranges, const uint32_t* tile_order, const uint32_t* pair_offset,
                        const uint32_t* pair_emit, const uint32_t* vis_idx, const uint32_t* vis_count,
                        uint32_t capacity, const float* final_T, const uint32_t* n_contrib, const float* dL_dimg,
                        const float* bg, float* grad_rows, int32_t grad_ld, float* grad2d, float* grad_norm, void* ws,
                        size_t ws_bytes, void* stream);

/*
 * The two halves of gs_raster_bwd, for callers that schedule or time them
 * separately.  gs_raster_bwd_pixels runs the per-pixel replay and leaves one
 * 9-float derivative per (tile, primitive) pair in the workspace, at the
 * pair's emission position;
 * gs_raster_bwd_project sums each visible primitive's pairs and applies the
 * chain rule.  The same workspace (gs_workspace_bytes(GS_WS_RASTER_BWD, ...))
 * must be passed to both, on the same stream or with the ordering ensured by
 * the caller; it carries the pair derivatives from the first call to the
 * second.  Arguments mean what they mean in gs_raster_bwd.
 */
gs_status gs_raster_bwd_pixels(const gs_proj* proj, const gs_camera* cam, const uint32_t* vals,
                               const uint32_t* ranges, const uint32_t* tile_order, const uint32_t* pair_emit,
                               uint32_t capacity, const float* final_T, const uint32_t* n_contrib,
                               const float* dL_dimg, const float* bg, void* ws, size_t ws_bytes, void* stream);
gs_status gs_raster_bwd_project(const gs_scene* scene, const gs_camera* cam, const gs_proj* proj,
                                const uint32_t* pair_offset, const uint32_t* vis_idx,
                                const uint32_t* vis_count, uint32_t capacity, float* grad_rows, int32_t grad_ld,
                                float* grad2d, float* grad_norm, void* ws, size_t ws_bytes, void* stream);

/*
 * A task unit of several views (Section 2.1: a task unit is a small batch of
 * training views whose scopes, active sets and gradient evidence are unions
 * and accumulations over its views): gs_raster_bwd_project for one view of
 * the unit, adding into the unit's gradient instead of writing a view's.
 *   union_idx/union_count: the unit's ascending union of visible sets (e.g.
 *     gs_scope_from_pred over the views' tile counts, then gs_visible_set with
 *     GS_PRED_BITMAP); it must contain this view's visible ids (ids missing
 *     from it are left out)
 *   grad_rows [*,grad_ld]: row u accumulates the gradient of union_idx[u]
 *     (same record layout as gs_raster_bwd); grad_norm [n]: grad_norm[id]
 *     accumulates |dL/d(u,v)| of each view (the unit's g_U evidence), or NULL
 *   first != 0 (the unit's first view): the |U| rows (all grad_ld columns) and
 *     grad_norm at the union ids are cleared before this view's terms are added
 * Other arguments as in gs_raster_bwd_project (its workspace, written by
 * gs_raster_bwd_pixels for this view).  Views must be added one after the
 * other (same stream); the result is the fp32 sum of the views' gradients in
 * view order.
 */
gs_status gs_raster_bwd_project_accum(const gs_scene* scene, const gs_camera* cam, const gs_proj* proj,
                                      const uint32_t* pair_offset, const uint32_t* vis_idx, const uint32_t* vis_count,
                                      uint32_t capacity, const uint32_t* union_idx, const uint32_t* union_count,
                                      int32_t first, float* grad_rows, int32_t grad_ld, float* grad_norm, void* ws,
                                      size_t ws_bytes, void* stream);

/*
 * Optimizer update (U in Figure 6; Shadow Graph step 5): Adam on the rows in
 * idx only (only the primitives a view sees are updated, Introduction), torch.optim.Adam
 * form with one global step t >= 1:
 *   m = b1 m + (1-b1) g;  v = b2 v + (1-b2) g^2
 *   delta = -(lr/(1-b1^t)) m / (sqrt(v)/sqrt(1-b2^t) + eps);  p += delta
 * The hyper-parameters are taken in fp64; b, 1-b, the bias corrections and
 * lr/(1-b1^t) are formed in fp64 and rounded to fp32 once (the arithmetic per
 * element is fp32).
 *   groups: the pool tensors p [n,cols] with their learning rates; a row's
 *     columns are the groups' columns concatenated (row_len = sum of cols <= 64)
 *   idx/count: the ascending ids to update (*count on the device, <= max_rows,
 *     which also sizes the launch)
 *   grad_rows [*,grad_ld]: row r holds the gradient of primitive idx[r] (the
 *     layout gs_raster_bwd writes); grad_ld >= row_len
 *   m, v [n,state_ld]: the moments, one row per primitive id (columns in
 *     group order); state_ld >= row_len
 *   delta_rows [*,delta_ld] or NULL: row r receives the step of idx[r] -- the
 *     pending update that a later publication carries; delta_ld >= row_len
 * Rows not in idx are not touched.  Errors: GS_ERR_INVALID_ARG for null
 * pointers, step < 1, betas outside [0,1), eps < 0, or a leading dimension
 * below row_len; GS_ERR_UNSUPPORTED for row_len > 64.
 */
typedef struct {
    float* p;                 /* [n, cols] with leading dimension ld */
    int32_t cols;
    float lr;
    int32_t ld;               /* floats between rows (0 = cols) */
} gs_adam_group;

gs_status gs_sparse_adam(const gs_adam_group* groups, int32_t n_groups, const uint32_t* idx,
                         const uint32_t* count, int32_t max_rows, const float* grad_rows, int32_t grad_ld, float* m,
                         float* v, int32_t state_ld, int32_t step, double beta1, double beta2, double eps,
                         float* delta_rows, int32_t delta_ld, void* stream);

/*
 * The optimizer update fused with the staging of its pending update (Shadow
 * Graph steps 3 and 5 of Section 4.3): the same update as gs_sparse_adam, and
 * the steps of the updated rows written as one publication message (layout
 * below; ids = idx, rows = the steps), byte for byte the message that
 * gs_delta_pack would build from gs_sparse_adam's delta_rows scattered back to
 * the pool layout.  If the message would not fit in msg_capacity bytes,
 * NOTHING is written (parameters, moments and message stay as they were) and
 * GS_DEV_MSG_OVERFLOW is set with the required bytes, so the call can be
 * repeated with a larger buffer.  If `status` already carries
 * GS_DEV_PAIR_OVERFLOW (the view's gs_bin_sort, given the same status, ran out
 * of pair capacity, so its gradient is incomplete), nothing is written either;
 * clear the status before the next view.  msg is 16-byte aligned.
 */
gs_status gs_sparse_adam_publish(const gs_adam_group* groups, int32_t n_groups, const uint32_t* idx,
                                 const uint32_t* count, int32_t max_rows, const float* grad_rows, int32_t grad_ld,
                                 float* m, float* v, int32_t state_ld, int32_t step, double beta1, double beta2,
                                 double eps, uint32_t version, void* msg, size_t msg_capacity,
                                 gs_device_status* status, void* stream);

/*
 * Staged publication (Shadow Graph steps 3-4 of Section 4.3; publication
 * callback of Section 5): pack gathers the rows of an ascending primitive id
 * list (e.g. the updated set, or the part of it a later task may observe)
 * from n_groups row-major tensors into one contiguous message; apply commits
 * a message into a replica and stamps the per-primitive publication version
 * (the publication metadata of Section 4.3's throughput-first path).
 *
 * Message layout (uint32 words, little endian):
 *   [0] magic 0x47534D31  [1] count K  [2] version  [3] row_len (sum of cols)
 *   [4] n_groups  [5..7] 0
 *   [8 .. 8+G) cols of each group, G = n_groups rounded up to a multiple of 4
 *   then K ids, then zero padding to a 16-byte boundary, then K rows of
 *   row_len fp32 values (each row = the groups' rows concatenated).
 *   gs_delta_msg_bytes(K, row_len, n_groups) gives the size.
 */
typedef struct {
    float* ptr;               /* [rows, cols] with leading dimension ld */
    int32_t cols;
    int32_t ld;               /* floats between rows (0 = cols) */
} gs_group;

#define GS_MSG_MAGIC 0x47534D31u
size_t gs_delta_msg_bytes(uint32_t count, int32_t row_len, int32_t n_groups);

gs_status gs_delta_pack(const uint32_t* idx, const uint32_t* count, int32_t max_rows, const gs_group* src,
                        int32_t n_groups, uint32_t version, void* msg, size_t msg_capacity,
                        gs_device_status* status, void* stream);

/* mode: GS_APPLY_ADD (one fp32 add per element) or GS_APPLY_OVERWRITE (copy).
 * msg_capacity: bytes readable at msg.  prim_version [n_rows] uint32 or NULL.
 * A bad magic, group widths that differ from dst, a count above max_rows, a
 * message longer than msg_capacity or an id >= n_rows set GS_DEV_MSG_MISMATCH
 * and nothing is written.  max_rows also sizes the launch. */
enum { GS_APPLY_ADD = 0, GS_APPLY_OVERWRITE = 1 };
gs_status gs_delta_apply(const void* msg, size_t msg_capacity, const gs_group* dst, int32_t n_groups, int32_t n_rows,
                         int32_t max_rows, int32_t mode, uint32_t* prim_version, gs_device_status* status,
                         void* stream);

/*
 * Versioned two-slot publication ring (Section 4.3, Shadow Graph steps 3-4:
 * updates are staged in a shared two-slot ring that is also the
 * communication source, and a slot is committed once its publication
 * condition holds; throughput-first path: per-primitive publication metadata
 * so that no read passes over more than one pending update).
 *   slot[0], slot[1]: device message buffers of slot_bytes each, 16-byte
 *     aligned; the update of version v is staged (gs_sparse_adam_publish or
 *     gs_delta_pack with that version) in slot[v & 1]
 *   state: 8 uint32 of device memory, zeroed by the caller once before the
 *     first commit: [0] last committed version, [1] rows applied and [2] rows
 *     left by the last commit, [3] reserved, [4..7] the library's (keep zero)
 * gs_publish_commit commits version `version` from slot[version & 1] into the
 * replica dst:
 *   - the slot must hold a message of this version whose group widths match
 *     dst, with count <= max_rows and ids < n_rows, else GS_DEV_MSG_MISMATCH;
 *   - versions commit in order: state[0] must be version - 1, else
 *     GS_DEV_MSG_ORDER (a repeated or early commit);
 *   - a row is applied (GS_APPLY_ADD: one fp32 add; GS_APPLY_OVERWRITE: copy)
 *     only if prim_version[id] < version, and prim_version[id] is then set to
 *     version; rows already at or past it are left (counted in state[2]);
 *   - skip[id] == version is cleared to 0 for every row of the message (the
 *     update that delayed reads skipped is now published; see
 *     gs_admission_gate);
 *   - on success state[0] = version.
 * After a flagged refusal nothing is written (replica, versions, skip, state).
 *   prim_version [n_rows] uint32 (required); skip [n_rows] uint32 or NULL
 * Errors: GS_ERR_INVALID_ARG for null pointers, misaligned slots, slots
 * smaller than a message header, version 0, a bad mode or group list;
 * GS_ERR_UNSUPPORTED for rows longer than 64 floats.
 */
typedef struct {
    void* slot[2];
    size_t slot_bytes;
    uint32_t* state;
    int32_t background;       /* nonzero: the commit is meant to run beside compute-bound work on another
                                 stream and is launched with one workgroup per compute unit, taking a
                                 small share of every CU instead of all of them */
} gs_ring;

gs_status gs_publish_commit(const gs_ring* ring, uint32_t version, const gs_group* dst, int32_t n_groups,
                            int32_t n_rows, int32_t max_rows, int32_t mode, uint32_t* prim_version, uint32_t* skip,
                            gs_device_status* status, void* stream);

/*
 * Primitive scopes (Section 2.1: the dependency unit is the primitive index;
 * a task unit's conservative read and update scopes R+ and W+, its realized
 * active set C and gradient evidence g).  A scope is a bitmap over primitive
 * ids: bit (i & 31) of uint32 word (i >> 5), GS_SCOPE_WORDS(n) words, device
 * memory.  Bits at or beyond n are ignored on input and written as 0.
 *
 * gs_scope_from_ids: the scope of ids idx[0 .. min(*count, max_rows)) (any
 * order; ids >= n are ignored).  accumulate = 0 clears the scope first,
 * accumulate = 1 adds the ids to it (the union over a task unit's views,
 * R+(U) = union of R+_i, Section 2.1).  count is one uint32 on the device.
 * gs_scope_from_pred: the same from a per-primitive predicate array
 * (GS_PRED_U32_NONZERO: uint32[n], GS_PRED_U8_NONZERO: uint8[n]), e.g. the
 * tile counts of gs_project (projection-visible scope) or the active flags of
 * gs_raster_fwd (realized active set).
 * Errors: GS_ERR_INVALID_ARG for null pointers, n < 0, a bad kind.
 */
#define GS_SCOPE_WORDS(n) (((uint32_t)(n) + 31u) / 32u)
gs_status gs_scope_from_ids(const uint32_t* idx, const uint32_t* count, int32_t max_rows, int32_t n,
                            int32_t accumulate, uint32_t* scope, void* stream);
gs_status gs_scope_from_pred(int32_t kind, const void* src, int32_t n, int32_t accumulate, uint32_t* scope,
                             void* stream);

/*
 * Quality-first primitive-state hazards (Section 4.3, "Quality-first path")
 * between an earlier task unit A and a later unit B:
 *   C_WAW = W+(B) & W+(A)
 *   C_RAW = (R+(B) \ W+(B)) & W+(A)
 *   C_WAR = W+(B) & (R+(A) \ W+(A))
 * RAW and WAW ids wait for A's publication, WAR ids for the end of A's
 * state-observing phase; with all three empty B may proceed.
 *   RA, WA, RB, WB: the four scopes (bitmaps of GS_SCOPE_WORDS(n) words)
 *   waw, raw, war: output bitmaps, each may be NULL
 *   waw_idx, raw_idx, war_idx: the same sets as ascending ids ([n] uint32
 *     each, the first count entries written), each may be NULL
 *   counts: 4 uint32 on the device: |C_WAW|, |C_RAW|, |C_WAR|, |R+(B)|
 *   ws: gs_workspace_bytes(GS_WS_SCOPE, n, 0, 0, 0) bytes
 * Errors: GS_ERR_INVALID_ARG for a null scope, counts or workspace, n < 0;
 * GS_ERR_WORKSPACE.
 */
gs_status gs_scope_conflicts(const uint32_t* RA, const uint32_t* WA, const uint32_t* RB, const uint32_t* WB,
                             int32_t n, uint32_t* waw, uint32_t* raw, uint32_t* war, uint32_t* waw_idx,
                             uint32_t* raw_idx, uint32_t* war_idx, uint32_t* counts, void* ws, size_t ws_bytes,
                             void* stream);

/*
 * Throughput-first admission of B's delayed reads (Section 4.3,
 * "Throughput-first path") for the delayed-read set D+ = C_RAW(A, B).  The
 * tests, in this order (the first that fails names the reason):
 *   D+ empty (also when R+(B) is empty): nothing to admit -> GS_GATE_NO_DELAY
 *   rho = |D+| / |R+(B)| <= tau                       else GS_GATE_WAIT_RHO
 *   C_A non-empty                                     else GS_GATE_WAIT_NO_ACTIVE
 *   every delayed id has producer evidence            else GS_GATE_WAIT_MISSING
 *   no delayed id's publication metadata names another producer's skipped
 *   update (no read passes over two pending updates)   else GS_GATE_WAIT_SECOND
 *   max over D+ of ||g_A(p)|| <= tau * mean over C_A of ||g_A(q)||
 *                                                     else GS_GATE_WAIT_GRADIENT
 *   -> GS_GATE_ADMIT
 * rho, the mean (an fp64 sum of the fp32 magnitudes) and the threshold are
 * formed in fp64.  On GS_GATE_ADMIT, skip[p] = producer_version for every p in
 * D+ (the per-primitive publication metadata; gs_publish_commit clears
 * it when that version is published).
 *   RB, D: scopes (bitmaps); args->active: the scope C_A; args->evidence: the
 *     scope of ids whose ||g_A|| the producer reported, or NULL for C_A;
 *     args->g: [n] fp32 ||g_A(p)|| by id (finite, >= 0; read at ids in C_A or
 *     D+ only; gs_raster_bwd's grad_norm is this for the visible ids);
 *     args->skip: [n] uint32 metadata, or NULL (no metadata: that test passes
 *     and nothing is stamped); args->tau in [0, 1]
 *   result: one gs_gate_result in device memory
 *   ws: gs_workspace_bytes(GS_WS_SCOPE, n, 0, 0, 0) bytes
 * Errors: GS_ERR_INVALID_ARG for null pointers, n < 0, tau outside [0, 1],
 * skip without a non-zero producer_version; GS_ERR_WORKSPACE.
 */
enum {
    GS_GATE_NO_DELAY = 0,
    GS_GATE_ADMIT = 1,
    GS_GATE_WAIT_RHO = 2,
    GS_GATE_WAIT_NO_ACTIVE = 3,
    GS_GATE_WAIT_MISSING = 4,
    GS_GATE_WAIT_SECOND = 5,
    GS_GATE_WAIT_GRADIENT = 6
};

typedef struct {
    const uint32_t* active;
    const uint32_t* evidence;
    const float* g;
    uint32_t* skip;
    uint32_t producer_version;
    double tau;
} gs_gate_args;

typedef struct {
    uint32_t admit;           /* 1 for GS_GATE_NO_DELAY and GS_GATE_ADMIT */
    uint32_t reason;          /* GS_GATE_* */
    uint32_t n_read;          /* |R+(B)| */
    uint32_t n_delayed;       /* |D+| */
    uint32_t n_active;        /* |C_A| */
    uint32_t n_missing;       /* delayed ids without evidence */
    uint32_t n_second;        /* delayed ids whose metadata names another producer */
    uint32_t reserved;
    double rho;               /* |D+| / |R+(B)|, 0 if R+(B) is empty */
    double mean_g;            /* mean of ||g_A|| over C_A, 0 if empty */
    double max_g;             /* max of ||g_A|| over D+, 0 if empty */
    double threshold;         /* tau * mean_g */
} gs_gate_result;

gs_status gs_admission_gate(const uint32_t* RB, const uint32_t* D, const gs_gate_args* args, int32_t n,
                            gs_gate_result* result, void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Ahead-of-time planner (host).  The three calls below run on the CPU over
 * host memory, synchronously, before training; they take no stream and
 * allocate host scratch internally.  Views are items 0..n-1.  Results are
 * deterministic: they do not depend on the number of threads used.
 * ------------------------------------------------------------------------ */

/*
 * Relative locality graph (Section 4.1.1, Eq. 1).  The weight of views i and
 * j is the Jaccard similarity |P_i & P_j| / |P_i | P_j| of their track sets
 * (0 for an empty union; a missing edge means weight 0, not independence).
 * Shared-track counts are taken through the inverse track -> view mapping.
 * Tracks seen by more than track_cap views are outliers and are left out
 * of every view's set (track_cap <= 0: no cap).  Each view keeps its top_k
 * strongest neighbours (weight descending, then view id ascending;
 * top_k <= 0 keeps all) and an edge is retained when either end keeps it,
 * so the graph is symmetric.
 *
 *   item_ptr [n_items+1]  CSR offsets into item_tracks, item_ptr[0] = 0
 *   item_tracks           track ids of each view, strictly ascending,
 *                         in [0, n_tracks)
 *   edge_ptr [n_items+1]  out: CSR offsets of the retained graph
 *   edge_dst, edge_w      out: neighbours (ascending) and weights in (0, 1],
 *                         edge_capacity entries available
 *   n_edges               out: entries the graph needs
 * At most 2 * n_items * top_k entries when top_k > 0.  Errors:
 * GS_ERR_INVALID_ARG for null pointers or a malformed track list;
 * GS_ERR_WORKSPACE (with *n_edges set, outputs untouched) if edge_capacity is
 * too small.
 */
gs_status gs_rlg_build(int32_t n_items, int32_t n_tracks, const int64_t* item_ptr, const int32_t* item_tracks,
                       int32_t track_cap, int32_t top_k, int64_t* edge_ptr, int32_t* edge_dst, double* edge_w,
                       int64_t edge_capacity, int64_t* n_edges);

/*
 * Logical partitioning (Section 4.2, LP): K balanced groups of views by
 * k-means over the camera centres.  Seeds are view 0 and then, one at a
 * time, the view farthest from every seed so far (squared distance, lowest
 * id on ties).  Each round assigns (distance, view, group) triples in
 * ascending order, each group taking at most ceil(n / K) views, and moves
 * each centre to its members' mean (summed in ascending view order).  It
 * stops when a round repeats the previous assignment or after max_iters
 * rounds.  The groups are then refined on the graph, so that strong coupling
 * stays within groups (the goal Section 4.2 sets for a partition): in passes
 * over the views in ascending order (at most 16, until one moves nothing), a
 * view moves to the group its edges weigh most towards (weights summed by
 * ascending neighbour; lowest group on ties) when that exceeds the weight
 * towards its own group, keeping every group size within floor(n / K) - s ..
 * ceil(n / K) + s, s = max(1, ceil(n / K) / 16).  The region-level coupling
 * summary coupling[a*K + b] is the sum
 * of the retained edge weights between groups a and b (within group a for
 * a = b), summed by ascending view, then neighbour.
 *
 *   position [n_items,3]  camera centres (finite)
 *   edge_*                a graph from gs_rlg_build (or any symmetric one
 *                         with ascending neighbours and weights in (0, 1])
 *   group [n_items]       out: group of each view
 *   coupling [K*K]        out
 *   iters_run             out: assignment rounds run
 * Errors: GS_ERR_INVALID_ARG for null pointers, K < 1, max_iters < 1, a
 * non-finite centre or a malformed graph.
 */
gs_status gs_lp_partition(int32_t n_items, const double* position, const int64_t* edge_ptr,
                          const int32_t* edge_dst, const double* edge_w, int32_t K, int32_t max_iters,
                          int32_t* group, double* coupling, int32_t* iters_run);

/*
 * Static data scheduling (Section 4.2, SDS, Eq. 2).  The traversal starts
 * at the lowest-numbered non-empty group and repeatedly moves to the
 * unvisited non-empty group least coupled to the last one (lowest id on
 * ties).  Task units of unit_size views take turns over that cycle.  Each
 * unit is filled from its group with the views of lowest score
 * s(v | U_prev) = sum of w_uv over the previous unit (view id breaks ties),
 * and topped up from the next groups of the cycle when its group runs out,
 * so every unit but the last has unit_size views.  transition[t] is the
 * largest retained weight between units t-1 and t (0 for t = 0).
 *
 *   group [n_items]       from gs_lp_partition (values in [0, K))
 *   coupling [K*K]        the region-level summary
 *   cycle [K]             out: the traversal, -1 after its n_cycle entries
 *   order [n_items]       out: the views, unit after unit
 *   unit_group, transition  out: [ceil(n_items / unit_size)] each
 * Errors: GS_ERR_INVALID_ARG for null pointers, K < 1, unit_size < 1, a
 * group outside [0, K) or a malformed graph.
 */
gs_status gs_sds_order(int32_t n_items, const int32_t* group, int32_t K, const double* coupling,
                       const int64_t* edge_ptr, const int32_t* edge_dst, const double* edge_w, int32_t unit_size,
                       int32_t* cycle, int32_t* n_cycle, int32_t* order, int32_t* unit_group, double* transition,
                       int32_t* n_units);

#ifdef __cplusplus
}
#endif
#endif /* GSMI_H */
