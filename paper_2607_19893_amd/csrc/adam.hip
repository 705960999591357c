// Optimizer update over the visible rows only (sparse Adam), optionally fused
// with the staging of its pending update as a publication message.
//
// Layout: a primitive's row spans all parameter groups (3+3+4+1+48 = 59
// floats at SH degree 3).  The gradient arrives as compact rows (row r ->
// primitive idx[r]) and the moments are row-major tables indexed by id, so a
// row's g, m and v are each one contiguous segment; only the parameters keep
// the pool's per-group tensors.  A wave takes floor(64 / row_len) rows at a
// time and lane l owns column l % row_len of sub-row l / row_len.  Each lane
// works on kUnroll rows per iteration, issuing all their loads before any
// arithmetic, so that enough rows are in flight to cover HBM latency.
#include "common.h"
#include "internal.h"

namespace gsmi {

namespace {

constexpr int kUnroll = 4;

struct AdamArgs {
    float* p[GS_MAX_GROUPS];
    int32_t cols[GS_MAX_GROUPS];
    int32_t ld[GS_MAX_GROUPS];     // row stride of each parameter group
    float step[GS_MAX_GROUPS];     // lr / (1 - beta1^t)
    int32_t n_groups;
    int32_t row_len;
    int32_t rows_per_wave;
    const float* g;
    int32_t gld;
    float* m;
    float* v;
    int32_t sld;
    float* d;                      // step rows (row r), or nullptr
    int32_t dld;
    uint32_t* msg;                 // publication message (PUBLISH only)
    uint64_t msg_capacity;
    uint32_t version;
    gs_device_status* status;
    float beta1, beta2, one_m_b1, one_m_b2, sqrt_bc2, eps;
};

// UNI (rows of more than 32 floats, one row per wave): the row index and its
// id are wave-uniform, so the id comes from a scalar load and stays in scalar
// registers.
template <bool PUBLISH, bool UNI>
__global__ void __launch_bounds__(GS_BLOCK) k_sparse_adam(AdamArgs a, const uint32_t* __restrict__ idx,
                                                          const uint32_t* __restrict__ count) {
    const uint32_t K = *count;
    float* __restrict__ drows = a.d;
    int32_t dld = a.dld;
    uint32_t* __restrict__ ids = nullptr;
    if (PUBLISH) {
        // the view's pair list overflowed (same device status as its
        // gs_bin_sort): its gradient is incomplete, so nothing is written
        if (a.status->flags & GS_DEV_PAIR_OVERFLOW) return;
        const uint64_t need = msg_bytes(K, a.row_len, a.n_groups);
        if (need > a.msg_capacity) {
            // all or nothing: no block touches parameters, moments or message
            if (blockIdx.x == 0 && threadIdx.x == 0) {
                atomicOr(&a.status->flags, GS_DEV_MSG_OVERFLOW);
                atomicMax(&a.status->required, (uint32_t)(need > 0xFFFFFFFFull ? 0xFFFFFFFFull : need));
            }
            return;
        }
        const uint32_t gw = (uint32_t)((a.n_groups + 3) / 4) * 4;
        const uint64_t row0 = msg_words_before_rows(K, a.n_groups);
        if (blockIdx.x == 0) {
            const uint32_t t = threadIdx.x;
            if (t < 8 + gw) {
                uint32_t val = 0;
                if (t == 0) val = GS_MSG_MAGIC;
                else if (t == 1) val = K;
                else if (t == 2) val = a.version;
                else if (t == 3) val = (uint32_t)a.row_len;
                else if (t == 4) val = (uint32_t)a.n_groups;
                else if (t >= 8 && t - 8 < (uint32_t)a.n_groups) val = (uint32_t)a.cols[t - 8];
                a.msg[t] = val;
            } else if (t < 8 + gw + 4) {
                const uint64_t pw = 8 + gw + K + (t - 8 - gw);     // zero padding between ids and rows
                if (pw < row0) a.msg[pw] = 0;
            }
        }
        ids = a.msg + 8 + gw;
        drows = reinterpret_cast<float*>(a.msg + row0);
        dld = a.row_len;
    }
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
    const int pld = a.ld[grp];
    const float step = a.step[grp];
    const float* __restrict__ G = a.g;
    float* __restrict__ Mm = a.m;
    float* __restrict__ Vv = a.v;
    const uint32_t waves = gridDim.x * (GS_BLOCK / GS_WAVE);
    const uint32_t wave = __builtin_amdgcn_readfirstlane(blockIdx.x * (GS_BLOCK / GS_WAVE) + threadIdx.x / GS_WAVE);
    const uint32_t rpw = UNI ? 1u : (uint32_t)a.rows_per_wave;
    const uint32_t stride = waves * rpw;
    for (uint32_t r0 = wave * rpw + (UNI ? 0u : (uint32_t)sub); r0 < K; r0 += kUnroll * stride) {
        uint32_t id[kUnroll], rr[kUnroll];
        float gr[kUnroll], mo[kUnroll], vo[kUnroll], po[kUnroll];
        // loads are unconditional (rows past the end re-read row 0, K >= 1 here)
        // and all issued before any use
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const uint32_t r = r0 + u * stride;
            rr[u] = r < K ? r : 0u;
            id[u] = idx[rr[u]];
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            gr[u] = G[(size_t)rr[u] * a.gld + col];
            mo[u] = Mm[(size_t)id[u] * a.sld + col];
            vo[u] = Vv[(size_t)id[u] * a.sld + col];
            po[u] = P[(size_t)id[u] * pld + c];
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            loaded(gr[u]);
            loaded(mo[u]);
            loaded(vo[u]);
            loaded(po[u]);
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const uint32_t r = r0 + u * stride;
            if (r < K) {
                const float mn = a.beta1 * mo[u] + a.one_m_b1 * gr[u];
                const float vn = a.beta2 * vo[u] + a.one_m_b2 * gr[u] * gr[u];
                const float den = sqrtf(vn) / a.sqrt_bc2 + a.eps;
                const float delta = -step * (mn / den);
                Mm[(size_t)id[u] * a.sld + col] = mn;
                Vv[(size_t)id[u] * a.sld + col] = vn;
                // a plain rounded add of the published step (this file is built
                // without contraction): a replica that adds the message's rows stays
                // bit-identical to the parameters
                P[(size_t)id[u] * pld + c] = po[u] + delta;
                if (drows) drows[(size_t)r * dld + col] = delta;
                if (PUBLISH && col == 0) ids[r] = id[u];
            }
        }
    }
}

AdamArgs make_args(const gs_adam_group* groups, int32_t n_groups, const float* grad_rows, int32_t grad_ld, float* m,
                   float* v, int32_t state_ld, int32_t step, double beta1, double beta2, double eps) {
    AdamArgs a = {};
    int32_t row_len = 0;
    const double bc1 = 1.0 - pow(beta1, (double)step);
    const double bc2 = 1.0 - pow(beta2, (double)step);
    for (int i = 0; i < n_groups; ++i) {
        a.p[i] = groups[i].p;
        a.cols[i] = groups[i].cols;
        a.ld[i] = groups[i].ld ? groups[i].ld : groups[i].cols;
        a.step[i] = (float)((double)groups[i].lr / bc1);
        row_len += groups[i].cols;
    }
    a.n_groups = n_groups;
    a.row_len = row_len;
    a.rows_per_wave = GS_WAVE / row_len;
    a.g = grad_rows;
    a.gld = grad_ld;
    a.m = m;
    a.v = v;
    a.sld = state_ld;
    a.beta1 = (float)beta1;
    a.beta2 = (float)beta2;
    a.one_m_b1 = (float)(1.0 - beta1);
    a.one_m_b2 = (float)(1.0 - beta2);
    a.sqrt_bc2 = (float)sqrt(bc2);
    a.eps = (float)eps;
    return a;
}

uint32_t adam_blocks(int32_t max_rows, int32_t rows_per_wave) {
    const uint64_t waves_needed = div_up(div_up((uint64_t)max_rows, (uint64_t)rows_per_wave), kUnroll);
    uint32_t blocks = div_up(waves_needed, GS_BLOCK / GS_WAVE);
    if (blocks > 8192) blocks = 8192;
    return blocks > 0 ? blocks : 1;
}

}  // namespace

hipError_t launch_sparse_adam(const gs_adam_group* groups, int32_t n_groups, const uint32_t* idx,
                              const uint32_t* count, int32_t max_rows, const float* grad_rows, int32_t grad_ld,
                              float* m, float* v, int32_t state_ld, int32_t step, double beta1, double beta2,
                              double eps, float* delta_rows, int32_t delta_ld, hipStream_t st) {
    AdamArgs a = make_args(groups, n_groups, grad_rows, grad_ld, m, v, state_ld, step, beta1, beta2, eps);
    a.d = delta_rows;
    a.dld = delta_ld;
    if (max_rows <= 0) return hipSuccess;
    const dim3 grid(adam_blocks(max_rows, a.rows_per_wave));
    if (a.rows_per_wave == 1)
        hipLaunchKernelGGL((k_sparse_adam<false, true>), grid, dim3(GS_BLOCK), 0, st, a, idx, count);
    else
        hipLaunchKernelGGL((k_sparse_adam<false, false>), grid, dim3(GS_BLOCK), 0, st, a, idx, count);
    return hipGetLastError();
}

hipError_t launch_sparse_adam_publish(const gs_adam_group* groups, int32_t n_groups, const uint32_t* idx,
                                      const uint32_t* count, int32_t max_rows, const float* grad_rows,
                                      int32_t grad_ld, float* m, float* v, int32_t state_ld, int32_t step,
                                      double beta1, double beta2, double eps, uint32_t version, void* msg,
                                      size_t msg_capacity, gs_device_status* status, hipStream_t st) {
    AdamArgs a = make_args(groups, n_groups, grad_rows, grad_ld, m, v, state_ld, step, beta1, beta2, eps);
    a.msg = static_cast<uint32_t*>(msg);
    a.msg_capacity = (uint64_t)msg_capacity;
    a.version = version;
    a.status = status;
    // launched even for max_rows == 0: the (empty) message header is still written
    const dim3 grid(adam_blocks(max_rows > 0 ? max_rows : 1, a.rows_per_wave));
    if (a.rows_per_wave == 1)
        hipLaunchKernelGGL((k_sparse_adam<true, true>), grid, dim3(GS_BLOCK), 0, st, a, idx, count);
    else
        hipLaunchKernelGGL((k_sparse_adam<true, false>), grid, dim3(GS_BLOCK), 0, st, a, idx, count);
    return hipGetLastError();
}

}  // namespace gsmi
