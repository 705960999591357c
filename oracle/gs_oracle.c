/*
 * CPU oracle for one 3D Gaussian Splatting training view.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, loads or
 * calls this file; only the test suite, the smoke check and the CPU-baseline
 * leg of the benchmark do.  It shares no source with the HIP path.
 *
 * The paper (Section 2.1) describes a PBNR training view as: render one
 * camera, compute an image loss, back-propagate and update only the
 * primitives that participate.  The renderer itself is the cited 3D Gaussian
 * Splatting method (Introduction, citation of 3DGS); this file writes that
 * method out as plainly as possible:
 *
 *   orc_project          EWA projection of every primitive + SH colour
 *   orc_visible          ascending ids of a per-primitive predicate
 *   orc_sorted_pairs     every (tile, depth, id) pair, sorted by qsort
 *   orc_render           per pixel: its candidates sorted by (depth, id),
 *                        then front-to-back compositing in fp64
 *   orc_render_backward  per pixel: the exact derivative of that composite,
 *                        with the transmittances kept from a forward replay
 *   orc_project_backward per primitive: chain rule back to the parameters
 *
 * Precision.  Everything continuous is fp64.  The one exception is the
 * projection geometry that decides integers (radius, tile rectangle, the
 * depth bits inside a sort key): that decision is taken in fp32 with a fixed
 * operation order (no fused multiply-add, IEEE division and square root),
 * because the kernel takes it in fp32; mode 1 of orc_project evaluates the
 * same geometry in fp64 instead and is used to pin the fp32 path and for
 * finite differences.  The fp32 geometry order is:
 *
 *   p_k  = ((R[k][0]*mx + R[k][1]*my) + R[k][2]*mz) + t[k]; cull if !(p_2 > near)
 *   s_k  = (float)exp((double)log_scale_k)
 *   q    = q / sqrt(((w*w + x*x) + y*y) + z*z), rotation matrix Rq from q
 *   M_ij = Rq_ij * s_j;  S_ij = (M_i0*M_j0 + M_i1*M_j1) + M_i2*M_j2
 *   xc   = min(lx, max(-lx, p_0/p_2)) * p_2  with lx = 1.3f*tan_fovx (same for y)
 *   J    = [fx/p_2, 0, -(fx*xc)/(p_2*p_2); 0, fy/p_2, -(fy*yc)/(p_2*p_2)]
 *   T    = J * Rcam (2x3);  U = T*S;  a = U0.T0 + 0.3, b = U0.T1, c = U1.T1 + 0.3
 *   D    = a*c - b*b; cull if !(D > 0); conic = (c/D, -(b/D), a/D)
 *   mid  = 0.5*(a+c); lam = mid + sqrt(max(0.1, mid*mid - D)); r = ceil(3*sqrt(lam))
 *   u    = fx*(p_0/p_2) + cx;  v = fy*(p_1/p_2) + cy
 *   x0   = floor(clamp((u - r)/16, 0, TX));  x1 = floor(clamp(((u + r) + 15)/16, 0, TX))
 *   (y likewise); tiles = (x1-x0)*(y1-y0); cull if tiles == 0
 *
 * Parity that no identity pins: none in this file -- every function is
 * checked by the CPU test suite against closed forms, brute force, finite
 * differences or a library routine.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORC_TILE 16

typedef struct {
    int32_t width, height;
    float fx, fy, cx, cy, tan_fovx, tan_fovy, near_z;
    float R[9];      /* world -> camera, row-major */
    float t[3];
    float campos[3];
} orc_camera;

/* Deliberate mistakes, switched on only by the test that checks that the
 * pins catch them (0 = none). */
static int g_mutation = 0;
void orc_set_mutation(int m) { g_mutation = m; }

int orc_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* ------------------------------------------------------------------------ */
/* Real spherical harmonics, from their definition.                          */
/*                                                                           */
/* Y_lm(d) = (-1)^|m| sqrt(2 - [m==0]) N_l|m| P_l^(|m|)(z) * B_m(x, y)       */
/*   N_lm = sqrt((2l+1)/(4 pi) * (l-m)!/(l+m)!)                              */
/*   P_l^(m) = m-th derivative of the Legendre polynomial P_l                */
/*   B_m = Re((x+iy)^m) for m > 0, 1 for m = 0, Im((x+iy)^|m|) for m < 0     */
/* i.e. the real basis built from the associated Legendre functions with the */
/* Condon-Shortley phase.  Coefficient k = l*l + l + m.                       */
/* ------------------------------------------------------------------------ */

#define ORC_MAXL 3
#define ORC_MAXK 16

static double g_leg[ORC_MAXL + 2][ORC_MAXL + 2];     /* P_l coefficients, power j */
static double g_norm[ORC_MAXL + 1][ORC_MAXL + 1];    /* (-1)^m sqrt(2-[m==0]) N_lm */
static int g_sh_ready = 0;

static double factorial(int n) { double f = 1.0; for (int i = 2; i <= n; ++i) f *= i; return f; }

static void sh_init(void)
{
    if (g_sh_ready) return;
    memset(g_leg, 0, sizeof g_leg);
    g_leg[0][0] = 1.0;
    g_leg[1][1] = 1.0;
    /* Bonnet recurrence: (l+1) P_{l+1} = (2l+1) z P_l - l P_{l-1} */
    for (int l = 1; l + 1 <= ORC_MAXL + 1; ++l)
        for (int j = 0; j <= ORC_MAXL + 1; ++j) {
            double zp = (j > 0) ? g_leg[l][j - 1] : 0.0;
            g_leg[l + 1][j] = ((2 * l + 1) * zp - l * g_leg[l - 1][j]) / (l + 1);
        }
    for (int l = 0; l <= ORC_MAXL; ++l)
        for (int m = 0; m <= l; ++m) {
            double n = sqrt((2.0 * l + 1.0) / (4.0 * M_PI) * factorial(l - m) / factorial(l + m));
            double s = (m & 1) ? -1.0 : 1.0;
            g_norm[l][m] = s * (m == 0 ? 1.0 : sqrt(2.0)) * n;
        }
    g_sh_ready = 1;
}

/* value of the m-th derivative of P_l at z */
static double legendre_deriv(int l, int m, double z)
{
    double acc = 0.0, zp = 1.0;
    for (int j = m; j <= l; ++j) {
        double c = g_leg[l][j];
        for (int k = 0; k < m; ++k) c *= (double)(j - k);
        acc += c * zp;
        zp *= z;
    }
    return acc;
}

/* Re/Im of (x + i y)^m */
static void cpow_xy(double x, double y, int m, double* re, double* im)
{
    double a = 1.0, b = 0.0;
    for (int k = 0; k < m; ++k) { double na = a * x - b * y; double nb = a * y + b * x; a = na; b = nb; }
    *re = a; *im = b;
}

/* Y[k] and, if grad != NULL, dY[k]/d(x,y,z) of the polynomial extension. */
static void sh_eval(int deg, const double d[3], double* Y, double (*grad)[3])
{
    sh_init();
    const double x = d[0], y = d[1], z = d[2];
    for (int l = 0; l <= deg; ++l)
        for (int m = -l; m <= l; ++m) {
            int am = m < 0 ? -m : m;
            int k = l * l + l + m;
            double P = legendre_deriv(l, am, z);
            double re, im;
            cpow_xy(x, y, am, &re, &im);
            double B = (m > 0) ? re : (m < 0 ? im : 1.0);
            double c = g_norm[l][am];
            if (g_mutation == 6 && l == 1 && m == 1) c = -c;
            Y[k] = c * P * B;
            if (grad) {
                /* d/dx (x+iy)^m = m (x+iy)^(m-1);  d/dy = i m (x+iy)^(m-1) */
                double dBx = 0.0, dBy = 0.0;
                if (am > 0) {
                    double re1, im1;
                    cpow_xy(x, y, am - 1, &re1, &im1);
                    if (m > 0) { dBx = am * re1; dBy = -am * im1; }
                    else       { dBx = am * im1; dBy = am * re1; }
                }
                double dP = (am + 1 <= l) ? legendre_deriv(l, am + 1, z) : 0.0;
                grad[k][0] = c * P * dBx;
                grad[k][1] = c * P * dBy;
                grad[k][2] = c * dP * B;
            }
        }
}

void orc_sh_basis(int deg, const double* dirs, int n, double* out)
{
    for (int i = 0; i < n; ++i) sh_eval(deg, dirs + 3 * i, out + (size_t)ORC_MAXK * i, NULL);
}

void orc_sh_basis_grad(int deg, const double* dirs, int n, double* out)
{
    for (int i = 0; i < n; ++i) {
        double Y[ORC_MAXK];
        sh_eval(deg, dirs + 3 * i, Y, (double (*)[3])(out + (size_t)ORC_MAXK * 3 * i));
    }
}

/* ------------------------------------------------------------------------ */
/* Projection                                                                */
/* ------------------------------------------------------------------------ */

static void quat_to_rot_d(const double q[4], double Rq[3][3])
{
    double w = q[0], x = q[1], y = q[2], z = q[3];
    Rq[0][0] = 1.0 - 2.0 * (y * y + z * z); Rq[0][1] = 2.0 * (x * y - w * z);       Rq[0][2] = 2.0 * (x * z + w * y);
    Rq[1][0] = 2.0 * (x * y + w * z);       Rq[1][1] = 1.0 - 2.0 * (x * x + z * z); Rq[1][2] = 2.0 * (y * z - w * x);
    Rq[2][0] = 2.0 * (x * z - w * y);       Rq[2][1] = 2.0 * (y * z + w * x);       Rq[2][2] = 1.0 - 2.0 * (x * x + y * y);
}

typedef struct {
    int culled;
    int radius;
    int rect[4];          /* x0, y0, x1, y1 (tiles, half-open) */
    float depth;          /* camera-space z in fp32 (sort key) */
    double u, v, A, B, C; /* pixel mean and conic used by the compositor */
    float u32, v32, conic32[3];
    double jclamp_margin; /* distance of p_x/p_z, p_y/p_z from the 1.3*tan clamp, relative */
} orc_geom;

/* fp32 geometry with the fixed operation order in the file header. */
static orc_geom geom_f32(const float* m, const float* ls, const float* q, const orc_camera* c)
{
    orc_geom g;
    memset(&g, 0, sizeof g);
    const float* R = c->R;
    float Rc[9];
    for (int i = 0; i < 9; ++i) Rc[i] = R[i];
    if (g_mutation == 3) {  /* transposed camera rotation */
        for (int i = 0; i < 3; ++i) for (int j = 0; j < 3; ++j) Rc[3 * i + j] = R[3 * j + i];
    }
    float p0 = ((Rc[0] * m[0] + Rc[1] * m[1]) + Rc[2] * m[2]) + c->t[0];
    float p1 = ((Rc[3] * m[0] + Rc[4] * m[1]) + Rc[5] * m[2]) + c->t[1];
    float p2 = ((Rc[6] * m[0] + Rc[7] * m[1]) + Rc[8] * m[2]) + c->t[2];
    if (!(p2 > c->near_z)) { g.culled = 1; return g; }

    float s0 = (float)exp((double)ls[0]);
    float s1 = (float)exp((double)ls[1]);
    float s2 = (float)exp((double)ls[2]);
    float qw = q[0], qx = q[1], qy = q[2], qz = q[3];
    float nq = sqrtf(((qw * qw + qx * qx) + qy * qy) + qz * qz);
    qw = qw / nq; qx = qx / nq; qy = qy / nq; qz = qz / nq;
    float Rq[3][3];
    Rq[0][0] = 1.0f - 2.0f * (qy * qy + qz * qz);
    Rq[0][1] = 2.0f * (qx * qy - qw * qz);
    Rq[0][2] = 2.0f * (qx * qz + qw * qy);
    Rq[1][0] = 2.0f * (qx * qy + qw * qz);
    Rq[1][1] = 1.0f - 2.0f * (qx * qx + qz * qz);
    Rq[1][2] = 2.0f * (qy * qz - qw * qx);
    Rq[2][0] = 2.0f * (qx * qz - qw * qy);
    Rq[2][1] = 2.0f * (qy * qz + qw * qx);
    Rq[2][2] = 1.0f - 2.0f * (qx * qx + qy * qy);
    float Mm[3][3];
    const float s[3] = {s0, s1, s2};
    for (int i = 0; i < 3; ++i) for (int j = 0; j < 3; ++j) Mm[i][j] = Rq[i][j] * s[j];
    float S[3][3];
    for (int i = 0; i < 3; ++i)
        for (int j = i; j < 3; ++j) {
            S[i][j] = (Mm[i][0] * Mm[j][0] + Mm[i][1] * Mm[j][1]) + Mm[i][2] * Mm[j][2];
            S[j][i] = S[i][j];
        }

    float lx = 1.3f * c->tan_fovx, ly = 1.3f * c->tan_fovy;
    float rx = p0 / p2, ry = p1 / p2;
    float xc = fminf(lx, fmaxf(-lx, rx)) * p2;
    float yc = fminf(ly, fmaxf(-ly, ry)) * p2;
    float j00 = c->fx / p2;
    float j02 = -(c->fx * xc) / (p2 * p2);
    float j11 = c->fy / p2;
    float j12 = -(c->fy * yc) / (p2 * p2);
    if (g_mutation == 2) j02 = -j02;
    float T[2][3];
    for (int k = 0; k < 3; ++k) {
        T[0][k] = j00 * Rc[k] + j02 * Rc[6 + k];
        T[1][k] = j11 * Rc[3 + k] + j12 * Rc[6 + k];
    }
    float U[2][3];
    for (int i = 0; i < 2; ++i)
        for (int k = 0; k < 3; ++k) U[i][k] = (T[i][0] * S[0][k] + T[i][1] * S[1][k]) + T[i][2] * S[2][k];
    float dil = (g_mutation == 1) ? 0.0f : 0.3f;
    float a = ((U[0][0] * T[0][0] + U[0][1] * T[0][1]) + U[0][2] * T[0][2]) + dil;
    float b = (U[0][0] * T[1][0] + U[0][1] * T[1][1]) + U[0][2] * T[1][2];
    float cc = ((U[1][0] * T[1][0] + U[1][1] * T[1][1]) + U[1][2] * T[1][2]) + dil;
    float D = a * cc - b * b;
    if (!(D > 0.0f)) { g.culled = 1; return g; }
    float cA = cc / D, cB = -(b / D), cC = a / D;
    float mid = 0.5f * (a + cc);
    float lam = mid + sqrtf(fmaxf(0.1f, mid * mid - D));
    float rf = ceilf(3.0f * sqrtf(lam));
    float u = c->fx * (p0 / p2) + c->cx;
    float v = c->fy * (p1 / p2) + c->cy;
    int TX = (c->width + ORC_TILE - 1) / ORC_TILE, TY = (c->height + ORC_TILE - 1) / ORC_TILE;
    float fTX = (float)TX, fTY = (float)TY;
    int x0 = (int)floorf(fminf(fmaxf((u - rf) / 16.0f, 0.0f), fTX));
    int x1 = (int)floorf(fminf(fmaxf(((u + rf) + 15.0f) / 16.0f, 0.0f), fTX));
    int y0 = (int)floorf(fminf(fmaxf((v - rf) / 16.0f, 0.0f), fTY));
    int y1 = (int)floorf(fminf(fmaxf(((v + rf) + 15.0f) / 16.0f, 0.0f), fTY));
    if ((x1 - x0) * (y1 - y0) <= 0) { g.culled = 1; return g; }
    g.radius = (int)fminf(rf, 1073741824.0f);
    g.rect[0] = x0; g.rect[1] = y0; g.rect[2] = x1; g.rect[3] = y1;
    g.depth = p2;
    g.u32 = u; g.v32 = v;
    g.conic32[0] = cA; g.conic32[1] = cB; g.conic32[2] = cC;
    g.u = u; g.v = v; g.A = cA; g.B = cB; g.C = cC;
    double mx = fabs(fabs((double)rx) - lx) / lx, my = fabs(fabs((double)ry) - ly) / ly;
    g.jclamp_margin = mx < my ? mx : my;
    return g;
}

/* The same geometry evaluated in fp64 (rect decided in fp64 too). */
static orc_geom geom_f64(const float* mf, const float* lsf, const float* qf, const orc_camera* c)
{
    orc_geom g;
    memset(&g, 0, sizeof g);
    double R[9];
    for (int i = 0; i < 9; ++i) R[i] = c->R[i];
    double m[3] = {mf[0], mf[1], mf[2]};
    double p[3];
    for (int k = 0; k < 3; ++k) p[k] = R[3 * k] * m[0] + R[3 * k + 1] * m[1] + R[3 * k + 2] * m[2] + (double)c->t[k];
    if (!(p[2] > (double)c->near_z)) { g.culled = 1; return g; }
    double s[3] = {exp((double)lsf[0]), exp((double)lsf[1]), exp((double)lsf[2])};
    double q[4] = {qf[0], qf[1], qf[2], qf[3]};
    double nq = sqrt(q[0] * q[0] + q[1] * q[1] + q[2] * q[2] + q[3] * q[3]);
    for (int i = 0; i < 4; ++i) q[i] /= nq;
    double Rq[3][3];
    quat_to_rot_d(q, Rq);
    double S[3][3];
    for (int i = 0; i < 3; ++i)
        for (int j = 0; j < 3; ++j) {
            double acc = 0.0;
            for (int k = 0; k < 3; ++k) acc += Rq[i][k] * s[k] * Rq[j][k] * s[k];
            S[i][j] = acc;
        }
    double lx = 1.3 * (double)c->tan_fovx, ly = 1.3 * (double)c->tan_fovy;
    double rx = p[0] / p[2], ry = p[1] / p[2];
    double xc = fmin(lx, fmax(-lx, rx)) * p[2], yc = fmin(ly, fmax(-ly, ry)) * p[2];
    double fx = c->fx, fy = c->fy;
    double J[2][3] = {{fx / p[2], 0.0, -fx * xc / (p[2] * p[2])}, {0.0, fy / p[2], -fy * yc / (p[2] * p[2])}};
    double T[2][3];
    for (int i = 0; i < 2; ++i)
        for (int k = 0; k < 3; ++k) T[i][k] = J[i][0] * R[k] + J[i][1] * R[3 + k] + J[i][2] * R[6 + k];
    double cov[2][2];
    for (int i = 0; i < 2; ++i)
        for (int j = 0; j < 2; ++j) {
            double acc = 0.0;
            for (int k = 0; k < 3; ++k) for (int l = 0; l < 3; ++l) acc += T[i][k] * S[k][l] * T[j][l];
            cov[i][j] = acc;
        }
    double a = cov[0][0] + 0.3, b = cov[0][1], cc = cov[1][1] + 0.3;
    double D = a * cc - b * b;
    if (!(D > 0.0)) { g.culled = 1; return g; }
    double mid = 0.5 * (a + cc);
    double lam = mid + sqrt(fmax(0.1, mid * mid - D));
    double rf = ceil(3.0 * sqrt(lam));
    double u = fx * (p[0] / p[2]) + c->cx, v = fy * (p[1] / p[2]) + c->cy;
    int TX = (c->width + ORC_TILE - 1) / ORC_TILE, TY = (c->height + ORC_TILE - 1) / ORC_TILE;
    int x0 = (int)floor(fmin(fmax((u - rf) / 16.0, 0.0), TX));
    int x1 = (int)floor(fmin(fmax((u + rf + 15.0) / 16.0, 0.0), TX));
    int y0 = (int)floor(fmin(fmax((v - rf) / 16.0, 0.0), TY));
    int y1 = (int)floor(fmin(fmax((v + rf + 15.0) / 16.0, 0.0), TY));
    if ((x1 - x0) * (y1 - y0) <= 0) { g.culled = 1; return g; }
    g.radius = (int)fmin(rf, 1073741824.0);
    g.rect[0] = x0; g.rect[1] = y0; g.rect[2] = x1; g.rect[3] = y1;
    g.depth = (float)p[2];
    g.u = u; g.v = v; g.A = cc / D; g.B = -b / D; g.C = a / D;
    g.u32 = (float)u; g.v32 = (float)v;
    g.conic32[0] = (float)g.A; g.conic32[1] = (float)g.B; g.conic32[2] = (float)g.C;
    double mx = fabs(fabs(rx) - lx) / lx, my = fabs(fabs(ry) - ly) / ly;
    g.jclamp_margin = mx < my ? mx : my;
    return g;
}

/*
 * Project every primitive.  mode 0: fp32 geometry (the kernel's decision
 * precision); mode 1: fp64 geometry.  Culled primitives get radius = 0 and
 * tiles = 0 and nothing else is written for them.
 *
 * Colour: rgb_ch = max(0, sum_k sh[k][ch] Y_k(d) + 0.5) with
 * d = (mean - campos)/|mean - campos|; clamp bit ch set when the sum + 0.5 is
 * negative; clamp_margin = min_ch |sum + 0.5|.
 */
void orc_project(int n, int deg, const float* mean, const float* ls, const float* quat, const float* logit,
                 const float* sh, const orc_camera* cam, int mode,
                 int32_t* radius, uint32_t* tiles, int32_t* rect, float* depth,
                 double* mean2d, double* conic, float* mean2d_f32, float* conic_f32,
                 double* opacity, double* rgb, uint8_t* clamp, double* clamp_margin, double* jclamp_margin)
{
    sh_init();
    const int K = (deg + 1) * (deg + 1);
#pragma omp parallel for schedule(static)
    for (int i = 0; i < n; ++i) {
        orc_geom g = (mode == 0) ? geom_f32(mean + 3 * i, ls + 3 * i, quat + 4 * i, cam)
                                 : geom_f64(mean + 3 * i, ls + 3 * i, quat + 4 * i, cam);
        if (g.culled) { radius[i] = 0; tiles[i] = 0; continue; }
        radius[i] = g.radius;
        tiles[i] = (uint32_t)((g.rect[2] - g.rect[0]) * (g.rect[3] - g.rect[1]));
        for (int k = 0; k < 4; ++k) rect[4 * i + k] = g.rect[k];
        depth[i] = g.depth;
        mean2d[2 * i] = g.u; mean2d[2 * i + 1] = g.v;
        conic[3 * i] = g.A; conic[3 * i + 1] = g.B; conic[3 * i + 2] = g.C;
        mean2d_f32[2 * i] = g.u32; mean2d_f32[2 * i + 1] = g.v32;
        for (int k = 0; k < 3; ++k) conic_f32[3 * i + k] = g.conic32[k];
        jclamp_margin[i] = g.jclamp_margin;
        opacity[i] = 1.0 / (1.0 + exp(-(double)logit[i]));
        double d[3], nrm = 0.0;
        for (int k = 0; k < 3; ++k) { d[k] = (double)mean[3 * i + k] - (double)cam->campos[k]; nrm += d[k] * d[k]; }
        nrm = sqrt(nrm);
        for (int k = 0; k < 3; ++k) d[k] /= nrm;
        double Y[ORC_MAXK];
        sh_eval(deg, d, Y, NULL);
        uint8_t cm = 0;
        double marg = 1e300;
        for (int ch = 0; ch < 3; ++ch) {
            double acc = 0.0;
            for (int k = 0; k < K; ++k) acc += (double)sh[((size_t)i * K + k) * 3 + ch] * Y[k];
            acc += 0.5;
            if (fabs(acc) < marg) marg = fabs(acc);
            if (acc < 0.0 && g_mutation != 23) { cm |= (uint8_t)(1u << ch); acc = 0.0; }
            rgb[3 * i + ch] = acc;
        }
        clamp[i] = cm;
        clamp_margin[i] = marg;
    }
}

/* Ascending ids i with src[i] != 0 (elem_bytes = 1 or 4).  Returns the count. */
int64_t orc_visible(int n, const void* src, int elem_bytes, uint32_t* idx)
{
    int64_t c = 0;
    for (int i = 0; i < n; ++i) {
        int on = (elem_bytes == 1) ? (((const uint8_t*)src)[i] != 0) : (((const uint32_t*)src)[i] != 0);
        if (on) idx[c++] = (uint32_t)i;
    }
    return c;
}

/* ------------------------------------------------------------------------ */
/* Sorted (tile, depth, id) pairs                                            */
/* ------------------------------------------------------------------------ */

typedef struct { uint64_t key; uint32_t val; } orc_pair;

static int cmp_pair(const void* pa, const void* pb)
{
    const orc_pair* a = (const orc_pair*)pa;
    const orc_pair* b = (const orc_pair*)pb;
    if (a->key != b->key) return a->key < b->key ? -1 : 1;
    if (a->val != b->val) return a->val < b->val ? -1 : 1;
    return 0;
}

static uint32_t fbits(float f) { uint32_t u; memcpy(&u, &f, 4); return u; }

/*
 * Every pair (tile, j) with tile in rect_j for j in vis; key = tile << 32 |
 * bits(depth_j); sorted by (key, j).  ranges[2*t] = start, [2*t+1] = end.
 * Returns the number of pairs (keys/vals must hold that many).
 */
int64_t orc_sorted_pairs(int64_t nvis, const uint32_t* vis, const int32_t* rect, const float* depth,
                         int TX, int TY, uint64_t* keys, uint32_t* vals, uint32_t* ranges)
{
    int64_t m = 0;
    for (int64_t a = 0; a < nvis; ++a) {
        const int32_t* r = rect + 4 * (size_t)vis[a];
        m += (int64_t)(r[2] - r[0]) * (r[3] - r[1]);
    }
    orc_pair* P = (orc_pair*)malloc(sizeof(orc_pair) * (size_t)(m > 0 ? m : 1));
    int64_t w = 0;
    for (int64_t a = 0; a < nvis; ++a) {
        uint32_t j = vis[a];
        const int32_t* r = rect + 4 * (size_t)j;
        for (int ty = r[1]; ty < r[3]; ++ty)
            for (int tx = r[0]; tx < r[2]; ++tx) {
                P[w].key = ((uint64_t)(uint32_t)(ty * TX + tx) << 32) | fbits(depth[j]);
                P[w].val = j;
                ++w;
            }
    }
    qsort(P, (size_t)m, sizeof(orc_pair), cmp_pair);
    for (int t = 0; t < TX * TY; ++t) { ranges[2 * t] = 0; ranges[2 * t + 1] = 0; }
    for (int64_t i = 0; i < m; ++i) {
        keys[i] = P[i].key;
        vals[i] = P[i].val;
        uint32_t t = (uint32_t)(P[i].key >> 32);
        if (i == 0 || (uint32_t)(P[i - 1].key >> 32) != t) ranges[2 * t] = (uint32_t)i;
        ranges[2 * t + 1] = (uint32_t)(i + 1);
    }
    free(P);
    return m;
}

/* ------------------------------------------------------------------------ */
/* Per-pixel compositing                                                     */
/* ------------------------------------------------------------------------ */

typedef struct {
    int64_t nvis;
    const uint32_t* vis;
    const int32_t* rect;
    const float* depth;
    const double* mean2d;
    const double* conic;
    const double* opacity;
    const double* rgb;
    int W, H, TX, TY;
    double bg[3];
} orc_scene2d;

typedef struct { float depth; uint32_t j; } orc_cand;

static int cmp_cand(const void* pa, const void* pb)
{
    const orc_cand* a = (const orc_cand*)pa;
    const orc_cand* b = (const orc_cand*)pb;
    uint32_t da = fbits(a->depth), db = fbits(b->depth);
    if (da != db) return da < db ? -1 : 1;
    if (a->j != b->j) return a->j < b->j ? -1 : 1;
    return 0;
}

/* Candidates of tile (tx, ty): every visible j whose rectangle holds the
 * tile, in (depth bits, id) order.  Returns the count. */
static int tile_candidates(const orc_scene2d* s, int tx, int ty, orc_cand* out)
{
    int c = 0;
    for (int64_t a = 0; a < s->nvis; ++a) {
        uint32_t j = s->vis[a];
        const int32_t* r = s->rect + 4 * (size_t)j;
        if (tx >= r[0] && tx < r[2] && ty >= r[1] && ty < r[3]) {
            out[c].depth = s->depth[j];
            out[c].j = j;
            ++c;
        }
    }
    qsort(out, (size_t)c, sizeof(orc_cand), cmp_cand);
    return c;
}

static int max_tile_list(const orc_scene2d* s)
{
    int T = s->TX * s->TY;
    int* cnt = (int*)calloc((size_t)T, sizeof(int));
    for (int64_t a = 0; a < s->nvis; ++a) {
        const int32_t* r = s->rect + 4 * (size_t)s->vis[a];
        for (int ty = r[1]; ty < r[3]; ++ty)
            for (int tx = r[0]; tx < r[2]; ++tx) cnt[ty * s->TX + tx]++;
    }
    int mx = 1;
    for (int t = 0; t < T; ++t) if (cnt[t] > mx) mx = cnt[t];
    free(cnt);
    return mx;
}

#define ORC_ALPHA_MIN (1.0 / 255.0)
#define ORC_T_MIN 1e-4
#define ORC_ALPHA_MAX 0.99

/* One entry of a pixel's front-to-back pass. */
typedef struct {
    int pos;          /* index in the tile's candidate list */
    double alpha, T;  /* alpha and the transmittance in front of it */
    double g;         /* o * exp(-sigma) before the 0.99 cap */
    double e;         /* exp(-sigma) */
    double dx, dy;
    int capped;
} orc_hit;

typedef struct {
    double C[3];
    double T;          /* final transmittance */
    int n_contrib;     /* 1 + list position of the last included pair (0 if none) */
    int n_seen;        /* list entries examined (terminated pixels stop early) */
    double margin_alpha, margin_T, margin_cap;
    int nhit;
    uint32_t capped_sig;  /* sum of (list position + 1) over the included pairs at the 0.99 cap */
} orc_pixres;

/* Front-to-back pass of pixel (px, py) over candidates L[0..nl).  With alt
 * set, every decision within its band (an alpha test within band_alpha of
 * 1/255, a termination test within band_T of 1e-4) that fails is taken the
 * other way: such a pair is included, and such a test does not stop the pass.
 * That is the outcome a computation in another precision may reach instead. */
static orc_pixres composite_pixel(const orc_scene2d* s, const orc_cand* L, int nl, int px, int py, orc_hit* hits,
                                  int alt, double band_alpha, double band_T)
{
    orc_pixres r;
    memset(&r, 0, sizeof r);
    r.margin_alpha = r.margin_T = r.margin_cap = 1e300;
    double T = 1.0;
    double C[3] = {0.0, 0.0, 0.0};
    double cx = px + 0.5, cy = py + 0.5;
    const double amax = (g_mutation == 22) ? 0.999 : ORC_ALPHA_MAX;
    int k;
    for (k = 0; k < nl; ++k) {
        uint32_t j = L[k].j;
        double dx = s->mean2d[2 * j] - cx, dy = s->mean2d[2 * j + 1] - cy;
        double A = s->conic[3 * j], B = s->conic[3 * j + 1], Cc = s->conic[3 * j + 2];
        double Bterm = (g_mutation == 4) ? -B * dx * dy : B * dx * dy;
        double sigma = 0.5 * A * dx * dx + Bterm + 0.5 * Cc * dy * dy;
        if (sigma < 0.0) continue;
        double e = exp(-sigma);
        double gval = s->opacity[j] * e;
        double ma = fabs(gval - ORC_ALPHA_MIN) / ORC_ALPHA_MIN;
        if (ma < r.margin_alpha) r.margin_alpha = ma;
        double mc = fabs(gval - amax) / amax;
        if (mc < r.margin_cap) r.margin_cap = mc;
        double alpha = gval < amax ? gval : amax;
        if (alpha < ORC_ALPHA_MIN && !(alt && ma < band_alpha)) continue;
        double Tn = T * (1.0 - alpha);
        double mt = fabs(Tn - ORC_T_MIN) / ORC_T_MIN;
        if (mt < r.margin_T) r.margin_T = mt;
        if (Tn < ORC_T_MIN && !(alt && mt < band_T)) { ++k; break; }
        if (hits) {
            orc_hit* h = &hits[r.nhit];
            h->pos = k; h->alpha = alpha; h->T = T; h->g = gval; h->e = e; h->dx = dx; h->dy = dy;
            h->capped = !(gval < amax);
        }
        if (!(gval < amax)) r.capped_sig += (uint32_t)(k + 1);
        r.nhit++;
        for (int ch = 0; ch < 3; ++ch) C[ch] += alpha * T * s->rgb[3 * j + ch];
        T = Tn;
        r.n_contrib = k + 1;
    }
    r.n_seen = k;
    for (int ch = 0; ch < 3; ++ch) r.C[ch] = C[ch] + T * s->bg[ch];
    r.T = T;
    return r;
}

/*
 * Render.  Outputs (any may be NULL except img):
 *   img [3,H,W] fp64 planar; T_final [H,W]; n_contrib [H,W];
 *   active [n] set to 1 for every primitive included in at least one pixel;
 *   margin_alpha / margin_T [H,W]: smallest relative distance of any
 *   decision of the pixel from its threshold (1/255 on alpha, 1e-4 on T);
 *   n_hits [H,W]: number of pairs included in the pixel;
 *   capped_sig [H,W]: sum of (list position + 1) over the pixel's included
 *   pairs whose o*exp(-sigma) reaches the 0.99 cap (0 if none), so that a
 *   finite-difference step can tell when a pair crosses the cap.
 */
void orc_render(int64_t nvis, const uint32_t* vis, const int32_t* rect, const float* depth,
                const double* mean2d, const double* conic, const double* opacity, const double* rgb,
                int W, int H, const double* bg,
                double* img, double* T_final, uint32_t* n_contrib, uint8_t* active,
                double* margin_alpha, double* margin_T, uint32_t* n_hits, uint32_t* capped_sig)
{
    orc_scene2d s = {nvis, vis, rect, depth, mean2d, conic, opacity, rgb, W, H,
                     (W + ORC_TILE - 1) / ORC_TILE, (H + ORC_TILE - 1) / ORC_TILE, {bg[0], bg[1], bg[2]}};
    int maxl = max_tile_list(&s);
    int T = s.TX * s.TY;
#pragma omp parallel
    {
        orc_cand* L = (orc_cand*)malloc(sizeof(orc_cand) * (size_t)maxl);
        orc_hit* hits = (orc_hit*)malloc(sizeof(orc_hit) * (size_t)maxl);
#pragma omp for schedule(dynamic, 1)
        for (int t = 0; t < T; ++t) {
            int tx = t % s.TX, ty = t / s.TX;
            int nl = tile_candidates(&s, tx, ty, L);
            for (int py = ty * ORC_TILE; py < (ty + 1) * ORC_TILE && py < H; ++py)
                for (int px = tx * ORC_TILE; px < (tx + 1) * ORC_TILE && px < W; ++px) {
                    orc_pixres r = composite_pixel(&s, L, nl, px, py, active ? hits : NULL, 0, 0.0, 0.0);
                    size_t p = (size_t)py * W + px;
                    for (int ch = 0; ch < 3; ++ch) img[(size_t)ch * W * H + p] = r.C[ch];
                    if (T_final) T_final[p] = r.T;
                    if (n_contrib) n_contrib[p] = (uint32_t)r.n_contrib;
                    if (margin_alpha) margin_alpha[p] = r.margin_alpha;
                    if (margin_T) margin_T[p] = r.margin_T;
                    if (n_hits) n_hits[p] = (uint32_t)r.nhit;
                    if (capped_sig) capped_sig[p] = r.capped_sig;
                    if (active)
                        for (int h = 0; h < r.nhit; ++h) active[L[hits[h].pos].j] = 1;  /* benign same-value store */
                }
        }
        free(L);
        free(hits);
    }
}

/*
 * Exact derivative of the render w.r.t. the per-primitive 2D quantities.
 *
 * For pixel colour C = sum_k alpha_k T_k c_k + T_end bg with
 * T_{k+1} = T_k (1 - alpha_k):
 *   dC/dc_k     = alpha_k T_k
 *   dC/dalpha_k = T_k c_k - S_k / (1 - alpha_k),  S_k = sum_{m>k} alpha_m T_m c_m + T_end bg
 * alpha = min(0.99, o e^-sigma): d/do = e^-sigma, d/dsigma = -alpha (zero when capped)
 * sigma = A dx^2/2 + B dx dy + C dy^2/2, dx = u - px, dy = v - py.
 * Pairs that were skipped (alpha < 1/255) or cut off by termination carry no
 * derivative (the decisions are locally constant).
 *
 * grad2d[9*j] = (du, dv, dA, dB, dC, dopacity, dr, dg, db), summed over the
 * pixels in a fixed tile order (deterministic).  Rows of invisible primitives
 * are zeroed.  flag[j] (if not NULL) gets bit 0 when j was examined by a
 * pixel whose margins fall below (amb_alpha, amb_T), or whose loss sign is
 * close (|loss_margin| < amb_loss, if loss_margin != NULL), bit 1 when one
 * of its included pairs sits within amb_cap of the 0.99 cap (where the
 * derivative w.r.t. opacity and sigma jumps).  grad2d_abs (if not NULL)
 * receives the per-component sums of |per-pixel term| (the magnitude an
 * fp32 summation's rounding error is proportional to).  With alt set, every
 * pixel takes the other outcome of each decision within the (amb_alpha, amb_T)
 * bands that failed (see composite_pixel), so the terms, their magnitudes and
 * the flags are those of that alternative pass.
 */
void orc_render_backward(int64_t nvis, const uint32_t* vis, const int32_t* rect, const float* depth,
                         const double* mean2d, const double* conic, const double* opacity, const double* rgb,
                         int W, int H, const double* bg, const double* dL_dimg, int n,
                         double* grad2d, uint8_t* flag, double amb_alpha, double amb_T, double amb_cap,
                         const double* loss_margin, double amb_loss, double* grad2d_abs, int alt)
{
    orc_scene2d s = {nvis, vis, rect, depth, mean2d, conic, opacity, rgb, W, H,
                     (W + ORC_TILE - 1) / ORC_TILE, (H + ORC_TILE - 1) / ORC_TILE, {bg[0], bg[1], bg[2]}};
    int maxl = max_tile_list(&s);
    int T = s.TX * s.TY;
    /* per-tile accumulators so that the final sum has a fixed order */
    int64_t* toff = (int64_t*)malloc(sizeof(int64_t) * (size_t)(T + 1));
    {
        int* cnt = (int*)calloc((size_t)T, sizeof(int));
        for (int64_t a = 0; a < nvis; ++a) {
            const int32_t* r = rect + 4 * (size_t)vis[a];
            for (int ty = r[1]; ty < r[3]; ++ty)
                for (int tx = r[0]; tx < r[2]; ++tx) cnt[ty * s.TX + tx]++;
        }
        toff[0] = 0;
        for (int t = 0; t < T; ++t) toff[t + 1] = toff[t] + cnt[t];
        free(cnt);
    }
    double* acc = (double*)calloc((size_t)toff[T] * 9 + 1, sizeof(double));
    double* aab = grad2d_abs ? (double*)calloc((size_t)toff[T] * 9 + 1, sizeof(double)) : NULL;
    uint32_t* accj = (uint32_t*)malloc(sizeof(uint32_t) * (size_t)(toff[T] + 1));
    uint8_t* accf = (uint8_t*)calloc((size_t)toff[T] + 1, 1);
    const size_t HW = (size_t)W * H;
#pragma omp parallel
    {
        orc_cand* L = (orc_cand*)malloc(sizeof(orc_cand) * (size_t)maxl);
        orc_hit* hits = (orc_hit*)malloc(sizeof(orc_hit) * (size_t)maxl);
#pragma omp for schedule(dynamic, 1)
        for (int t = 0; t < T; ++t) {
            int tx = t % s.TX, ty = t / s.TX;
            int nl = tile_candidates(&s, tx, ty, L);
            double* ta = acc + (size_t)toff[t] * 9;
            double* tb = aab ? aab + (size_t)toff[t] * 9 : NULL;
            uint8_t* tf = accf + toff[t];
            for (int k = 0; k < nl; ++k) accj[toff[t] + k] = L[k].j;
            for (int py = ty * ORC_TILE; py < (ty + 1) * ORC_TILE && py < H; ++py)
                for (int px = tx * ORC_TILE; px < (tx + 1) * ORC_TILE && px < W; ++px) {
                    orc_pixres r = composite_pixel(&s, L, nl, px, py, hits, alt, amb_alpha, amb_T);
                    size_t p = (size_t)py * W + px;
                    double gC[3] = {dL_dimg[p], dL_dimg[HW + p], dL_dimg[2 * HW + p]};
                    int amb = (r.margin_alpha < amb_alpha) || (r.margin_T < amb_T);
                    if (loss_margin)
                        for (int ch = 0; ch < 3; ++ch) if (fabs(loss_margin[ch * HW + p]) < amb_loss) amb = 1;
                    if (amb) {
                        int upto = (r.margin_T < amb_T) ? nl : r.n_seen;
                        for (int k = 0; k < upto; ++k) tf[k] |= 1;
                    }
                    /* suffix sum S, walking back to front */
                    double S[3] = {r.T * bg[0], r.T * bg[1], r.T * bg[2]};
                    for (int h = r.nhit - 1; h >= 0; --h) {
                        const orc_hit* e = &hits[h];
                        uint32_t j = L[e->pos].j;
                        double* g = ta + (size_t)e->pos * 9;
                        const double* c = rgb + 3 * (size_t)j;
                        double term[9] = {0, 0, 0, 0, 0, 0, 0, 0, 0};
                        double dalpha = 0.0;
                        for (int ch = 0; ch < 3; ++ch) {
                            double sk = (g_mutation == 5) ? S[ch] : S[ch] / (1.0 - e->alpha);
                            dalpha += gC[ch] * (e->T * c[ch] - sk);
                            term[6 + ch] = gC[ch] * e->alpha * e->T;
                        }
                        if (fabs(e->g - ORC_ALPHA_MAX) / ORC_ALPHA_MAX < amb_cap) tf[e->pos] |= 2;
                        if (!e->capped || g_mutation == 24) {
                            double A = conic[3 * j], B = conic[3 * j + 1], Cc = conic[3 * j + 2];
                            term[5] = dalpha * e->e;
                            double dsig = -dalpha * e->alpha;
                            term[0] = dsig * (A * e->dx + B * e->dy);
                            term[1] = dsig * (B * e->dx + Cc * e->dy);
                            term[2] = dsig * 0.5 * e->dx * e->dx;
                            term[3] = dsig * e->dx * e->dy;
                            term[4] = dsig * 0.5 * e->dy * e->dy;
                        }
                        for (int q = 0; q < 9; ++q) g[q] += term[q];
                        if (tb)
                            for (int q = 0; q < 9; ++q) tb[(size_t)e->pos * 9 + q] += fabs(term[q]);
                        for (int ch = 0; ch < 3; ++ch) S[ch] += e->alpha * e->T * c[ch];
                    }
                }
        }
        free(L);
        free(hits);
    }
    for (int64_t a = 0; a < nvis; ++a) {
        memset(grad2d + 9 * (size_t)vis[a], 0, 9 * sizeof(double));
        if (grad2d_abs) memset(grad2d_abs + 9 * (size_t)vis[a], 0, 9 * sizeof(double));
        if (flag) flag[vis[a]] = 0;
    }
    for (int64_t i = 0; i < toff[T]; ++i) {
        uint32_t j = accj[i];
        for (int c = 0; c < 9; ++c) grad2d[9 * (size_t)j + c] += acc[9 * (size_t)i + c];
        if (aab)
            for (int c = 0; c < 9; ++c) grad2d_abs[9 * (size_t)j + c] += aab[9 * (size_t)i + c];
        if (flag) flag[j] |= accf[i];
    }
    (void)n;
    free(acc); free(aab); free(accj); free(accf); free(toff);
}

/* ------------------------------------------------------------------------ */
/* Projection backward (fp64 chain rule)                                     */
/* ------------------------------------------------------------------------ */

/*
 * For each visible j = vis[row]: from grad2d[9*j] = (du, dv, dA, dB, dC, do,
 * dr, dg, db) to the parameter gradients, written to `row` of the compact
 * outputs (dmean [nvis,3], dls [nvis,3], dquat [nvis,4], dlogit [nvis],
 * dsh [nvis,K,3], grad_norm [nvis]).  The geometry is re-evaluated in fp64.
 *   opacity:  dlogit = do * o (1 - o)
 *   colour:   channels with the clamp bit carry no gradient; dsh[k][ch] = dc_ch Y_k(d);
 *             d(view dir) -> d(mean) through d = (mu - campos)/|mu - campos|
 *   conic:    Q = inv(Sigma2D): dSigma2D = -Q dQ Q with dQ = [[dA, dB/2], [dB/2, dC]]
 *   Sigma2D = T Sigma T^T (+0.3 I):  dSigma = T^T dS2 T,  dT = 2 dS2 T Sigma
 *   T = J Rcam, J from p = Rcam mu + t with the 1.3 tan clamp (clamped
 *   coordinates carry no derivative w.r.t. p_x, p_y)
 *   u = fx p_x/p_z + cx, v = fy p_y/p_z + cy
 *   Sigma = M M^T, M = Rq diag(s): dM = 2 dSigma M; ds_j = sum_i dM_ij Rq_ij; dls = ds s
 *   Rq(q/|q|): dq = (dqn - qn (qn . dqn)) / |q|
 * grad_norm[j] = |(du, dv)|.
 */
void orc_project_backward(int n, int deg, const float* mean, const float* ls, const float* quat, const float* logit,
                          const float* sh, const orc_camera* cam, int64_t nvis, const uint32_t* vis,
                          const double* grad2d, const uint8_t* clamp,
                          double* dmean, double* dls, double* dquat, double* dlogit, double* dsh, double* grad_norm)
{
    sh_init();
    const int K = (deg + 1) * (deg + 1);
    (void)n;
#pragma omp parallel for schedule(static)
    for (int64_t row = 0; row < nvis; ++row) {
        const size_t j = vis[row];
        const double* g2 = grad2d + 9 * j;
        double R[9];
        for (int i = 0; i < 9; ++i) R[i] = cam->R[i];
        double mu[3] = {mean[3 * j], mean[3 * j + 1], mean[3 * j + 2]};
        double p[3];
        for (int k = 0; k < 3; ++k) p[k] = R[3 * k] * mu[0] + R[3 * k + 1] * mu[1] + R[3 * k + 2] * mu[2] + (double)cam->t[k];
        double s[3] = {exp((double)ls[3 * j]), exp((double)ls[3 * j + 1]), exp((double)ls[3 * j + 2])};
        double qraw[4] = {quat[4 * j], quat[4 * j + 1], quat[4 * j + 2], quat[4 * j + 3]};
        double nq = sqrt(qraw[0] * qraw[0] + qraw[1] * qraw[1] + qraw[2] * qraw[2] + qraw[3] * qraw[3]);
        double q[4] = {qraw[0] / nq, qraw[1] / nq, qraw[2] / nq, qraw[3] / nq};
        double Rq[3][3];
        quat_to_rot_d(q, Rq);
        double Mm[3][3];
        for (int i = 0; i < 3; ++i) for (int k = 0; k < 3; ++k) Mm[i][k] = Rq[i][k] * s[k];
        double Sig[3][3];
        for (int i = 0; i < 3; ++i)
            for (int k = 0; k < 3; ++k) Sig[i][k] = Mm[i][0] * Mm[k][0] + Mm[i][1] * Mm[k][1] + Mm[i][2] * Mm[k][2];
        const double fx = cam->fx, fy = cam->fy;
        const double lx = 1.3 * (double)cam->tan_fovx, ly = 1.3 * (double)cam->tan_fovy;
        double rx = p[0] / p[2], ry = p[1] / p[2];
        int clx = (rx < -lx) || (rx > lx), cly = (ry < -ly) || (ry > ly);
        double xr = fmin(lx, fmax(-lx, rx)), yr = fmin(ly, fmax(-ly, ry));
        double tz = p[2];
        double J[2][3] = {{fx / tz, 0.0, -fx * xr / tz}, {0.0, fy / tz, -fy * yr / tz}};
        double T[2][3];
        for (int i = 0; i < 2; ++i)
            for (int k = 0; k < 3; ++k) T[i][k] = J[i][0] * R[k] + J[i][1] * R[3 + k] + J[i][2] * R[6 + k];
        double cov[2][2];
        for (int i = 0; i < 2; ++i)
            for (int k = 0; k < 2; ++k) {
                double acc = 0.0;
                for (int u = 0; u < 3; ++u) for (int v = 0; v < 3; ++v) acc += T[i][u] * Sig[u][v] * T[k][v];
                cov[i][k] = acc;
            }
        double a = cov[0][0] + 0.3, b = cov[0][1], c = cov[1][1] + 0.3;
        double D = a * c - b * b;
        double Q[2][2] = {{c / D, -b / D}, {-b / D, a / D}};
        double gQ[2][2] = {{g2[2], 0.5 * g2[3]}, {0.5 * g2[3], g2[4]}};
        double tmp[2][2], gS2[2][2];
        for (int i = 0; i < 2; ++i)
            for (int k = 0; k < 2; ++k) tmp[i][k] = gQ[i][0] * Q[0][k] + gQ[i][1] * Q[1][k];
        for (int i = 0; i < 2; ++i)
            for (int k = 0; k < 2; ++k) gS2[i][k] = -(Q[i][0] * tmp[0][k] + Q[i][1] * tmp[1][k]);
        /* dSigma = T^T gS2 T ; dT = 2 gS2 T Sigma */
        double gSig[3][3];
        for (int u = 0; u < 3; ++u)
            for (int v = 0; v < 3; ++v) {
                double acc = 0.0;
                for (int i = 0; i < 2; ++i) for (int k = 0; k < 2; ++k) acc += T[i][u] * gS2[i][k] * T[k][v];
                gSig[u][v] = acc;
            }
        double gT[2][3];
        for (int i = 0; i < 2; ++i)
            for (int v = 0; v < 3; ++v) {
                double acc = 0.0;
                for (int k = 0; k < 2; ++k) for (int u = 0; u < 3; ++u) acc += gS2[i][k] * T[k][u] * Sig[u][v];
                gT[i][v] = 2.0 * acc;
            }
        double gJ00 = 0, gJ02 = 0, gJ11 = 0, gJ12 = 0;
        for (int k = 0; k < 3; ++k) {
            gJ00 += gT[0][k] * R[k];
            gJ02 += gT[0][k] * R[6 + k];
            gJ11 += gT[1][k] * R[3 + k];
            gJ12 += gT[1][k] * R[6 + k];
        }
        double gp[3] = {0.0, 0.0, 0.0};
        /* J00 = fx/tz, J11 = fy/tz */
        gp[2] += gJ00 * (-fx / (tz * tz)) + gJ11 * (-fy / (tz * tz));
        /* J02 = -fx*xr/tz with xr = px/tz unless clamped */
        if (clx) gp[2] += gJ02 * (fx * xr / (tz * tz));
        else { gp[0] += gJ02 * (-fx / (tz * tz)); gp[2] += gJ02 * (2.0 * fx * p[0] / (tz * tz * tz)); }
        if (cly) gp[2] += gJ12 * (fy * yr / (tz * tz));
        else { gp[1] += gJ12 * (-fy / (tz * tz)); gp[2] += gJ12 * (2.0 * fy * p[1] / (tz * tz * tz)); }
        /* pixel mean */
        gp[0] += g2[0] * fx / tz;
        gp[1] += g2[1] * fy / tz;
        gp[2] += -g2[0] * fx * p[0] / (tz * tz) - g2[1] * fy * p[1] / (tz * tz);
        double gmu[3];
        for (int k = 0; k < 3; ++k) gmu[k] = R[k] * gp[0] + R[3 + k] * gp[1] + R[6 + k] * gp[2];
        /* Sigma = M M^T */
        double gM[3][3];
        for (int i = 0; i < 3; ++i)
            for (int k = 0; k < 3; ++k) gM[i][k] = 2.0 * (gSig[i][0] * Mm[0][k] + gSig[i][1] * Mm[1][k] + gSig[i][2] * Mm[2][k]);
        double gRq[3][3];
        for (int i = 0; i < 3; ++i) for (int k = 0; k < 3; ++k) gRq[i][k] = gM[i][k] * s[k];
        for (int k = 0; k < 3; ++k) {
            double gs = gM[0][k] * Rq[0][k] + gM[1][k] * Rq[1][k] + gM[2][k] * Rq[2][k];
            dls[3 * row + k] = gs * s[k];
        }
        double w = q[0], x = q[1], y = q[2], z = q[3];
        double gq[4];
        gq[0] = 2.0 * (-z * gRq[0][1] + y * gRq[0][2] + z * gRq[1][0] - x * gRq[1][2] - y * gRq[2][0] + x * gRq[2][1]);
        gq[1] = 2.0 * (y * gRq[0][1] + z * gRq[0][2] + y * gRq[1][0] - 2.0 * x * gRq[1][1] - w * gRq[1][2]
                       + z * gRq[2][0] + w * gRq[2][1] - 2.0 * x * gRq[2][2]);
        gq[2] = 2.0 * (-2.0 * y * gRq[0][0] + x * gRq[0][1] + w * gRq[0][2] + x * gRq[1][0] + z * gRq[1][2]
                       - w * gRq[2][0] + z * gRq[2][1] - 2.0 * y * gRq[2][2]);
        gq[3] = 2.0 * (-2.0 * z * gRq[0][0] - w * gRq[0][1] + x * gRq[0][2] + w * gRq[1][0] - 2.0 * z * gRq[1][1]
                       + y * gRq[1][2] + x * gRq[2][0] + y * gRq[2][1]);
        double qd = q[0] * gq[0] + q[1] * gq[1] + q[2] * gq[2] + q[3] * gq[3];
        for (int k = 0; k < 4; ++k) dquat[4 * row + k] = (gq[k] - q[k] * qd) / nq;
        /* opacity */
        double o = 1.0 / (1.0 + exp(-(double)logit[j]));
        dlogit[row] = g2[5] * o * (1.0 - o);
        /* colour */
        double dv[3], nrm = 0.0;
        for (int k = 0; k < 3; ++k) { dv[k] = mu[k] - (double)cam->campos[k]; nrm += dv[k] * dv[k]; }
        nrm = sqrt(nrm);
        double d[3] = {dv[0] / nrm, dv[1] / nrm, dv[2] / nrm};
        double Y[ORC_MAXK], dY[ORC_MAXK][3];
        sh_eval(deg, d, Y, dY);
        double gd[3] = {0.0, 0.0, 0.0};
        for (int ch = 0; ch < 3; ++ch) {
            double gc = ((clamp[j] >> ch & 1) && g_mutation != 26) ? 0.0 : g2[6 + ch];
            for (int k = 0; k < K; ++k) {
                dsh[((size_t)row * K + k) * 3 + ch] = gc * Y[k];
                double cf = sh[(j * K + k) * 3 + ch];
                gd[0] += gc * cf * dY[k][0];
                gd[1] += gc * cf * dY[k][1];
                gd[2] += gc * cf * dY[k][2];
            }
        }
        double dd = gd[0] * d[0] + gd[1] * d[1] + gd[2] * d[2];
        for (int k = 0; k < 3; ++k) gmu[k] += (gd[k] - d[k] * dd) / nrm;
        for (int k = 0; k < 3; ++k) dmean[3 * row + k] = gmu[k];
        grad_norm[row] = (g_mutation == 25) ? fabs(g2[0]) + fabs(g2[1]) : sqrt(g2[0] * g2[0] + g2[1] * g2[1]);
    }
}
