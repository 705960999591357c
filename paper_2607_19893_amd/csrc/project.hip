// Preprocessing phase: EWA projection + spherical-harmonic colour, one thread
// per primitive.
//
// The geometry that decides integers (radius, tile rectangle) and the depth
// used in sort keys is evaluated in fp32 in one fixed order with no
// contraction into fused multiply-adds (this file is built with
// -ffp-contract=off and the pragma below), IEEE division and square root,
// and exp of the log-scales taken in fp64 and rounded once.  That makes it
// reproducible bit for bit on any IEEE machine that follows the same order.
#include "common.h"
#include "internal.h"

#pragma clang fp contract(off)

namespace gsmi {

namespace {

// Real SH basis (Condon-Shortley phase) on the unit sphere, degrees 0..3.
constexpr float kY0 = 0.28209479177387814f;
constexpr float kY1 = 0.48860251190291992f;
constexpr float kY2a = 1.0925484305920792f;
constexpr float kY2b = 0.31539156525252005f;
constexpr float kY2c = 0.54627421529603959f;
constexpr float kY3a = 0.59004358992664352f;
constexpr float kY3b = 2.8906114426405538f;
constexpr float kY3c = 0.45704579946446572f;
constexpr float kY3d = 0.37317633259011546f;
constexpr float kY3e = 1.4453057213202769f;

__device__ __forceinline__ void sh_basis(int deg, float x, float y, float z, float* Y) {
    Y[0] = kY0;
    if (deg < 1) return;
    Y[1] = -kY1 * y;
    Y[2] = kY1 * z;
    Y[3] = -kY1 * x;
    if (deg < 2) return;
    const float xx = x * x, yy = y * y, zz = z * z;
    Y[4] = kY2a * (x * y);
    Y[5] = -kY2a * (y * z);
    Y[6] = kY2b * (2.0f * zz - xx - yy);
    Y[7] = -kY2a * (x * z);
    Y[8] = kY2c * (xx - yy);
    if (deg < 3) return;
    Y[9] = -kY3a * y * (3.0f * xx - yy);
    Y[10] = kY3b * (x * y) * z;
    Y[11] = -kY3c * y * (4.0f * zz - xx - yy);
    Y[12] = kY3d * z * (2.0f * zz - 3.0f * xx - 3.0f * yy);
    Y[13] = -kY3c * x * (4.0f * zz - xx - yy);
    Y[14] = kY3e * z * (xx - yy);
    Y[15] = -kY3a * x * (xx - 3.0f * yy);
}

template <int DEG>
__global__ void __launch_bounds__(GS_BLOCK) k_project(
    int32_t n, const float* __restrict__ mean, const float* __restrict__ log_scale,
    const float* __restrict__ quat, const float* __restrict__ opacity, const float* __restrict__ sh, SceneLd ld, CamArgs c,
    int32_t* __restrict__ radius, uint32_t* __restrict__ tiles, ushort4* __restrict__ rect,
    float* __restrict__ depth, float2* __restrict__ mean2d, float4* __restrict__ conic_opacity,
    float* __restrict__ rgb, uint8_t* __restrict__ clampm) {
    const int32_t i = blockIdx.x * GS_BLOCK + threadIdx.x;
    if (i >= n) return;
    const float* mrow = mean + (size_t)i * ld.mean;
    const float mx = mrow[0], my = mrow[1], mz = mrow[2];

    // camera space
    const float p0 = ((c.R[0] * mx + c.R[1] * my) + c.R[2] * mz) + c.t[0];
    const float p1 = ((c.R[3] * mx + c.R[4] * my) + c.R[5] * mz) + c.t[1];
    const float p2 = ((c.R[6] * mx + c.R[7] * my) + c.R[8] * mz) + c.t[2];
    if (!(p2 > c.near_z)) {
        radius[i] = 0;
        tiles[i] = 0;
        return;
    }
    float l0, l1, l2, logit;
    if (ld.head) {
        // the record's head: one 16-byte load for log_scale and the opacity logit
        const float4 h = *reinterpret_cast<const float4*>(quat + (size_t)i * ld.quat + 4);
        l0 = h.x; l1 = h.y; l2 = h.z; logit = h.w;
    } else {
        const float* lrow = log_scale + (size_t)i * ld.log_scale;
        l0 = lrow[0]; l1 = lrow[1]; l2 = lrow[2];
        logit = 0.0f;
    }
    const float s0 = (float)exp((double)l0);
    const float s1 = (float)exp((double)l1);
    const float s2 = (float)exp((double)l2);
    const float lx = 1.3f * c.tan_fovx, ly = 1.3f * c.tan_fovy;
    const float u = c.fx * (p0 / p2) + c.cx;
    const float v = c.fy * (p1 / p2) + c.cy;
    const float fTX = (float)c.tiles_x, fTY = (float)c.tiles_y;
    {
        // Off-screen primitives leave before their rotation is read.  The 2D
        // covariance's larger eigenvalue is at most |J|_F^2 smax^2 + 0.3 (J the
        // clamped projection Jacobian, Sigma's spectral norm smax^2), and the
        // radius rule below adds at most sqrt(0.1) to it, so 3 sqrt of that bound
        // (with 0.1% and 2 pixels to spare for rounding) is at least the radius.
        // The rectangle only grows with the radius: if it is empty at the bound,
        // the full rule would find it empty too and write the same zeros.
        const float smax = fmaxf(s0, fmaxf(s1, s2));
        const float jx = c.fx / p2, jy = c.fy / p2;
        const float jf2 = jx * jx * (1.0f + lx * lx) + jy * jy * (1.0f + ly * ly);
        const float rb = 3.0f * sqrtf(jf2 * (smax * smax) + 0.62f) * 1.001f + 2.0f;
        const int bx0 = (int)floorf(fminf(fmaxf((u - rb) / 16.0f, 0.0f), fTX));
        const int bx1 = (int)floorf(fminf(fmaxf(((u + rb) + 15.0f) / 16.0f, 0.0f), fTX));
        const int by0 = (int)floorf(fminf(fmaxf((v - rb) / 16.0f, 0.0f), fTY));
        const int by1 = (int)floorf(fminf(fmaxf(((v + rb) + 15.0f) / 16.0f, 0.0f), fTY));
        if ((bx1 - bx0) * (by1 - by0) <= 0) {
            radius[i] = 0;
            tiles[i] = 0;
            return;
        }
    }

    // 3D covariance  Sigma = (Rq S)(Rq S)^T
    const float4 q = *reinterpret_cast<const float4*>(quat + (size_t)i * ld.quat);
    const float qn = sqrtf(((q.x * q.x + q.y * q.y) + q.z * q.z) + q.w * q.w);
    const float w = q.x / qn, x = q.y / qn, y = q.z / qn, z = q.w / qn;
    float Rq[3][3];
    Rq[0][0] = 1.0f - 2.0f * (y * y + z * z);
    Rq[0][1] = 2.0f * (x * y - w * z);
    Rq[0][2] = 2.0f * (x * z + w * y);
    Rq[1][0] = 2.0f * (x * y + w * z);
    Rq[1][1] = 1.0f - 2.0f * (x * x + z * z);
    Rq[1][2] = 2.0f * (y * z - w * x);
    Rq[2][0] = 2.0f * (x * z - w * y);
    Rq[2][1] = 2.0f * (y * z + w * x);
    Rq[2][2] = 1.0f - 2.0f * (x * x + y * y);
    const float sc[3] = {s0, s1, s2};
    float M[3][3];
#pragma unroll
    for (int a = 0; a < 3; ++a)
#pragma unroll
        for (int b = 0; b < 3; ++b) M[a][b] = Rq[a][b] * sc[b];
    float S[3][3];
#pragma unroll
    for (int a = 0; a < 3; ++a)
#pragma unroll
        for (int b = a; b < 3; ++b) {
            S[a][b] = (M[a][0] * M[b][0] + M[a][1] * M[b][1]) + M[a][2] * M[b][2];
            S[b][a] = S[a][b];
        }

    // EWA: Sigma2D = (J Rcam) Sigma (J Rcam)^T + 0.3 I
    const float rx = p0 / p2, ry = p1 / p2;
    const float xc = fminf(lx, fmaxf(-lx, rx)) * p2;
    const float yc = fminf(ly, fmaxf(-ly, ry)) * p2;
    const float j00 = c.fx / p2;
    const float j02 = -(c.fx * xc) / (p2 * p2);
    const float j11 = c.fy / p2;
    const float j12 = -(c.fy * yc) / (p2 * p2);
    float T0[3], T1[3];
#pragma unroll
    for (int k = 0; k < 3; ++k) {
        T0[k] = j00 * c.R[k] + j02 * c.R[6 + k];
        T1[k] = j11 * c.R[3 + k] + j12 * c.R[6 + k];
    }
    float U0[3], U1[3];
#pragma unroll
    for (int k = 0; k < 3; ++k) {
        U0[k] = (T0[0] * S[0][k] + T0[1] * S[1][k]) + T0[2] * S[2][k];
        U1[k] = (T1[0] * S[0][k] + T1[1] * S[1][k]) + T1[2] * S[2][k];
    }
    const float a = ((U0[0] * T0[0] + U0[1] * T0[1]) + U0[2] * T0[2]) + 0.3f;
    const float b = (U0[0] * T1[0] + U0[1] * T1[1]) + U0[2] * T1[2];
    const float cc = ((U1[0] * T1[0] + U1[1] * T1[1]) + U1[2] * T1[2]) + 0.3f;
    const float det = a * cc - b * b;
    if (!(det > 0.0f)) {
        radius[i] = 0;
        tiles[i] = 0;
        return;
    }
    const float cA = cc / det, cB = -(b / det), cC = a / det;
    const float mid = 0.5f * (a + cc);
    const float lam = mid + sqrtf(fmaxf(0.1f, mid * mid - det));
    const float rf = ceilf(3.0f * sqrtf(lam));
    const int x0 = (int)floorf(fminf(fmaxf((u - rf) / 16.0f, 0.0f), fTX));
    const int x1 = (int)floorf(fminf(fmaxf(((u + rf) + 15.0f) / 16.0f, 0.0f), fTX));
    const int y0 = (int)floorf(fminf(fmaxf((v - rf) / 16.0f, 0.0f), fTY));
    const int y1 = (int)floorf(fminf(fmaxf(((v + rf) + 15.0f) / 16.0f, 0.0f), fTY));
    const int nt = (x1 - x0) * (y1 - y0);
    if (nt <= 0) {
        radius[i] = 0;
        tiles[i] = 0;
        return;
    }
    radius[i] = (int)fminf(rf, 1073741824.0f);
    tiles[i] = (uint32_t)nt;
    rect[i] = make_ushort4((unsigned short)x0, (unsigned short)y0, (unsigned short)x1, (unsigned short)y1);
    depth[i] = p2;
    mean2d[i] = make_float2(u, v);

    // appearance (fp32, not part of any integer decision)
    if (!ld.head) logit = opacity[(size_t)i * ld.opacity];
    // the sigmoid in fp64, rounded to fp32 once: the blending's transmittance
    // error grows with alpha / (1 - alpha) times alpha's relative error, and a
    // two-ulp fp32 sigmoid was a third of that error
    const float o = (float)(1.0 / (1.0 + exp(-(double)logit)));
    conic_opacity[i] = make_float4(cA, cB, cC, o);
    float dx = mx - c.campos[0], dy = my - c.campos[1], dz = mz - c.campos[2];
    const float inv = 1.0f / sqrtf(dx * dx + dy * dy + dz * dz);
    dx *= inv; dy *= inv; dz *= inv;
    constexpr int K = (DEG + 1) * (DEG + 1);
    float Y[16];
    sh_basis(DEG, dx, dy, dz, Y);
    // the row's coefficients, as float4 loads when a row is a whole number of them
    float co[3 * K];
    if constexpr ((3 * K) % 4 == 0) {
        const float4* s4 = reinterpret_cast<const float4*>(sh + (size_t)i * ld.sh);
#pragma unroll
        for (int k = 0; k < 3 * K / 4; ++k) {
            const float4 v4 = s4[k];
            co[4 * k] = v4.x; co[4 * k + 1] = v4.y; co[4 * k + 2] = v4.z; co[4 * k + 3] = v4.w;
        }
    } else {
#pragma unroll
        for (int k = 0; k < 3 * K; ++k) co[k] = sh[(size_t)i * ld.sh + k];
    }
    float acc0 = 0.5f, acc1 = 0.5f, acc2 = 0.5f;
#pragma unroll
    for (int k = 0; k < K; ++k) {
        acc0 = fmaf(co[3 * k + 0], Y[k], acc0);
        acc1 = fmaf(co[3 * k + 1], Y[k], acc1);
        acc2 = fmaf(co[3 * k + 2], Y[k], acc2);
    }
    uint8_t cm = (uint8_t)((acc0 < 0.0f ? 1 : 0) | (acc1 < 0.0f ? 2 : 0) | (acc2 < 0.0f ? 4 : 0));
    rgb[3 * i + 0] = fmaxf(acc0, 0.0f);
    rgb[3 * i + 1] = fmaxf(acc1, 0.0f);
    rgb[3 * i + 2] = fmaxf(acc2, 0.0f);
    clampm[i] = cm;
}

}  // namespace

CamArgs make_cam_args(const gs_camera* c) {
    CamArgs a;
    a.width = c->width;
    a.height = c->height;
    a.tiles_x = (c->width + GS_TILE - 1) / GS_TILE;
    a.tiles_y = (c->height + GS_TILE - 1) / GS_TILE;
    a.fx = c->fx; a.fy = c->fy; a.cx = c->cx; a.cy = c->cy;
    a.tan_fovx = c->tan_fovx; a.tan_fovy = c->tan_fovy; a.near_z = c->near_z;
    for (int i = 0; i < 9; ++i) a.R[i] = c->R[i];
    for (int i = 0; i < 3; ++i) { a.t[i] = c->t[i]; a.campos[i] = c->campos[i]; }
    return a;
}

hipError_t launch_project(const gs_scene& s, const CamArgs& cam, const gs_proj& o, hipStream_t st) {
    if (s.n == 0) return hipSuccess;
    const dim3 grid(div_up(s.n, GS_BLOCK));
#define GS_LAUNCH_PROJECT(D)                                                                                   \
    hipLaunchKernelGGL(k_project<D>, grid, dim3(GS_BLOCK), 0, st, s.n, s.mean, s.log_scale, s.quat, s.opacity,   \
                       s.sh, scene_ld(s), cam, o.radius, o.tiles, reinterpret_cast<ushort4*>(o.rect), o.depth,   \
                       reinterpret_cast<float2*>(o.mean2d), reinterpret_cast<float4*>(o.conic_opacity), o.rgb,  \
                       o.clamp)
    switch (s.sh_degree) {
        case 0: GS_LAUNCH_PROJECT(0); break;
        case 1: GS_LAUNCH_PROJECT(1); break;
        case 2: GS_LAUNCH_PROJECT(2); break;
        default: GS_LAUNCH_PROJECT(3); break;
    }
#undef GS_LAUNCH_PROJECT
    return hipGetLastError();
}

}  // namespace gsmi
