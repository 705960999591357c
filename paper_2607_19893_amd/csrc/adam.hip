// Optimizer update over the visible rows only (sparse Adam).
//
// Layout: one primitive row spans all parameter groups (3+3+4+1+48 = 59
// floats at SH degree 3).  A wave takes floor(64 / row_len) rows at a time;
// lane l owns column l % row_len of sub-row l / row_len, so the lanes of one
// row read each group's contiguous row segment together.  The group and
// column of every lane are fixed once; the loop over rows is grid-strided.
// Bound by HBM: 16 bytes read (p, g, m, v) and 12-16 written per element.
#include "common.h"
#include "internal.h"

namespace gsmi {

namespace {

struct AdamArgs {
    float* p[GS_MAX_GROUPS];
    const float* g[GS_MAX_GROUPS];
    float* m[GS_MAX_GROUPS];
    float* v[GS_MAX_GROUPS];
    float* d[GS_MAX_GROUPS];
    int32_t cols[GS_MAX_GROUPS];
    float step[GS_MAX_GROUPS];     // lr / (1 - beta1^t)
    int32_t n_groups;
    int32_t row_len;
    int32_t rows_per_wave;
    float beta1, beta2, one_m_b1, one_m_b2, sqrt_bc2, eps;
};

__global__ void __launch_bounds__(GS_BLOCK) k_sparse_adam(AdamArgs a, const uint32_t* __restrict__ idx,
                                                          const uint32_t* __restrict__ count) {
    const int lane = lane_id();
    const int sub = lane / a.row_len;
    const int col = lane - sub * a.row_len;
    if (sub >= a.rows_per_wave) return;
    int grp = 0, c = col;
    while (grp + 1 < a.n_groups && c >= a.cols[grp]) {
        c -= a.cols[grp];
        ++grp;
    }
    float* __restrict__ P = a.p[grp];
    const float* __restrict__ G = a.g[grp];
    float* __restrict__ Mm = a.m[grp];
    float* __restrict__ Vv = a.v[grp];
    float* __restrict__ D = a.d[grp];
    const int cols = a.cols[grp];
    const float step = a.step[grp];
    const uint32_t K = *count;
    const uint32_t waves = gridDim.x * (GS_BLOCK / GS_WAVE);
    const uint32_t wave = blockIdx.x * (GS_BLOCK / GS_WAVE) + threadIdx.x / GS_WAVE;
    for (uint32_t r = wave * a.rows_per_wave + sub; r < K; r += waves * a.rows_per_wave) {
        const size_t o = (size_t)idx[r] * cols + c;
        const float gr = G[o];
        const float mn = a.beta1 * Mm[o] + a.one_m_b1 * gr;
        const float vn = a.beta2 * Vv[o] + a.one_m_b2 * gr * gr;
        const float den = sqrtf(vn) / a.sqrt_bc2 + a.eps;
        const float delta = -step * (mn / den);
        Mm[o] = mn;
        Vv[o] = vn;
        P[o] = P[o] + delta;
        if (D) D[o] = delta;
    }
}

}  // namespace

hipError_t launch_sparse_adam(const gs_adam_group* groups, int32_t n_groups, const uint32_t* idx,
                              const uint32_t* count, int32_t max_rows, int32_t step, double beta1, double beta2,
                              double eps, hipStream_t st) {
    AdamArgs a = {};
    int32_t row_len = 0;
    const double bc1 = 1.0 - pow(beta1, (double)step);
    const double bc2 = 1.0 - pow(beta2, (double)step);
    for (int i = 0; i < n_groups; ++i) {
        a.p[i] = groups[i].p;
        a.g[i] = groups[i].g;
        a.m[i] = groups[i].m;
        a.v[i] = groups[i].v;
        a.d[i] = groups[i].delta;
        a.cols[i] = groups[i].cols;
        a.step[i] = (float)((double)groups[i].lr / bc1);
        row_len += groups[i].cols;
    }
    a.n_groups = n_groups;
    a.row_len = row_len;
    a.rows_per_wave = GS_WAVE / row_len;
    a.beta1 = (float)beta1;
    a.beta2 = (float)beta2;
    a.one_m_b1 = (float)(1.0 - beta1);
    a.one_m_b2 = (float)(1.0 - beta2);
    a.sqrt_bc2 = (float)sqrt(bc2);
    a.eps = (float)eps;
    if (max_rows <= 0) return hipSuccess;
    const uint64_t waves_needed = div_up((uint64_t)max_rows, (uint64_t)a.rows_per_wave);
    uint32_t blocks = div_up(waves_needed, GS_BLOCK / GS_WAVE);
    if (blocks > 8192) blocks = 8192;
    hipLaunchKernelGGL(k_sparse_adam, dim3(blocks), dim3(GS_BLOCK), 0, st, a, idx, count);
    return hipGetLastError();
}

}  // namespace gsmi
