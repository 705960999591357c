// Staged publication of pending updates: pack the rows of an ascending id
// list into one message, and commit a message into a replica (add or copy),
// stamping the per-primitive publication version; the versioned commit of a
// two-slot ring checks the order of versions and each primitive's published
// version and clears the skip markers of delayed reads.
//
// Same lane layout as the optimizer: one row per floor(64/row_len) lanes,
// lane -> (group, column) fixed once, grid-strided rows.  Message writes are
// contiguous; source/destination rows are gathered/scattered by id.
#include "common.h"
#include "internal.h"

namespace gsmi {

namespace {

struct GroupArgs {
    float* ptr[GS_MAX_GROUPS];
    int32_t cols[GS_MAX_GROUPS];
    int32_t ld[GS_MAX_GROUPS];     // row stride of each group
    int32_t n_groups;
    int32_t row_len;
    int32_t rows_per_wave;
};

__device__ __forceinline__ void lane_group(const GroupArgs& a, int lane, int& sub, int& grp, int& c) {
    sub = lane / a.row_len;
    c = lane - sub * a.row_len;
    grp = 0;
    while (grp + 1 < a.n_groups && c >= a.cols[grp]) {
        c -= a.cols[grp];
        ++grp;
    }
}

// Rows are taken kRowsInFlight at a time per lane group, with all their loads
// issued before any store: a row's gather depends on its id, so one row per
// iteration would leave each wave waiting two memory latencies per row.
constexpr int kRowsInFlight = 8;

template <bool UNI>
__global__ void __launch_bounds__(GS_BLOCK) k_pack(GroupArgs a, const uint32_t* __restrict__ idx,
                                                   const uint32_t* __restrict__ count, uint32_t version,
                                                   uint32_t* __restrict__ msg, uint64_t capacity,
                                                   gs_device_status* __restrict__ status) {
    const uint32_t K = *count;
    const uint64_t need = msg_bytes(K, a.row_len, a.n_groups);
    if (need > capacity) {
        if (blockIdx.x == 0 && threadIdx.x == 0 && status) {
            atomicOr(&status->flags, GS_DEV_MSG_OVERFLOW);
            atomicMax(&status->required, (uint32_t)(need > 0xFFFFFFFFull ? 0xFFFFFFFFull : need));
        }
        return;
    }
    const uint64_t gw = (uint64_t)((a.n_groups + 3) / 4) * 4;
    if (blockIdx.x == 0 && threadIdx.x < 8 + gw) {
        const uint32_t t = threadIdx.x;
        uint32_t v = 0;
        if (t == 0) v = GS_MSG_MAGIC;
        else if (t == 1) v = K;
        else if (t == 2) v = version;
        else if (t == 3) v = (uint32_t)a.row_len;
        else if (t == 4) v = (uint32_t)a.n_groups;
        else if (t >= 8 && t - 8 < (uint32_t)a.n_groups) v = (uint32_t)a.cols[t - 8];
        msg[t] = v;
    }
    uint32_t* __restrict__ ids = msg + 8 + gw;
    const uint64_t row0 = msg_words_before_rows(K, a.n_groups);
    // zero padding between the ids and the rows
    if (blockIdx.x == 0 && threadIdx.x < 4) {
        const uint64_t pw = 8 + gw + K + threadIdx.x;
        if (pw < row0) msg[pw] = 0;
    }
    float* __restrict__ rows = reinterpret_cast<float*>(msg + row0);
    const int lane = lane_id();
    int sub, grp, c;
    lane_group(a, lane, sub, grp, c);
    if (sub >= a.rows_per_wave) return;
    const float* __restrict__ src = a.ptr[grp];
    const int gld = a.ld[grp];
    const int col = lane - sub * a.row_len;
    const uint32_t rpw = UNI ? 1u : (uint32_t)a.rows_per_wave;
    const uint32_t waves = gridDim.x * (GS_BLOCK / GS_WAVE);
    const uint32_t wave = __builtin_amdgcn_readfirstlane(blockIdx.x * (GS_BLOCK / GS_WAVE) + threadIdx.x / GS_WAVE);
    for (uint32_t r0 = wave * rpw * kRowsInFlight; r0 < K; r0 += waves * rpw * kRowsInFlight) {
        uint32_t rr[kRowsInFlight], id[kRowsInFlight];
        float val[kRowsInFlight];
#pragma unroll
        for (int u = 0; u < kRowsInFlight; ++u) {
            const uint32_t r = r0 + (uint32_t)u * rpw + (UNI ? 0u : (uint32_t)sub);
            rr[u] = r < K ? r : K - 1u;           // past the end: re-read the last row, store nothing
        }
#pragma unroll
        for (int u = 0; u < kRowsInFlight; ++u) id[u] = idx[rr[u]];
#pragma unroll
        for (int u = 0; u < kRowsInFlight; ++u) val[u] = src[(size_t)id[u] * gld + c];
#pragma unroll
        for (int u = 0; u < kRowsInFlight; ++u) loaded(val[u]);
#pragma unroll
        for (int u = 0; u < kRowsInFlight; ++u) {
            const uint32_t r = r0 + (uint32_t)u * rpw + (UNI ? 0u : (uint32_t)sub);
            if (r < K) {
                if (col == 0) ids[r] = id[u];
                rows[(size_t)r * a.row_len + col] = val[u];
            }
        }
    }
}

// Header and id check; sets GS_DEV_MSG_MISMATCH when the message cannot be applied.
__global__ void __launch_bounds__(GS_BLOCK) k_apply_check(GroupArgs a, const uint32_t* __restrict__ msg,
                                                          uint64_t msg_capacity, int32_t n_rows, int32_t max_rows,
                                                          gs_device_status* __restrict__ status) {
    bool bad = false;
    const uint32_t K = msg[1];
    if (msg[0] != GS_MSG_MAGIC || msg[3] != (uint32_t)a.row_len || msg[4] != (uint32_t)a.n_groups ||
        K > (uint32_t)max_rows || msg_bytes(K, a.row_len, a.n_groups) > msg_capacity)
        bad = true;
    if (!bad && blockIdx.x == 0 && threadIdx.x < (uint32_t)a.n_groups)
        if (msg[8 + threadIdx.x] != (uint32_t)a.cols[threadIdx.x]) bad = true;
    if (!bad) {
        const uint64_t gw = (uint64_t)((a.n_groups + 3) / 4) * 4;
        const uint32_t* ids = msg + 8 + gw;
        for (uint32_t r = blockIdx.x * GS_BLOCK + threadIdx.x; r < K; r += gridDim.x * GS_BLOCK)
            if (ids[r] >= (uint32_t)n_rows) bad = true;
    }
    if (bad) atomicOr(&status->flags, GS_DEV_MSG_MISMATCH);
}

template <bool UNI>
__global__ void __launch_bounds__(GS_BLOCK) k_apply(GroupArgs a, const uint32_t* __restrict__ msg, int32_t mode,
                                                    uint32_t* __restrict__ prim_version,
                                                    const gs_device_status* __restrict__ status) {
    if (status->flags & GS_DEV_MSG_MISMATCH) return;
    const uint32_t K = msg[1];
    const uint32_t version = msg[2];
    const uint64_t gw = (uint64_t)((a.n_groups + 3) / 4) * 4;
    const uint32_t* __restrict__ ids = msg + 8 + gw;
    const float* __restrict__ rows = reinterpret_cast<const float*>(msg + msg_words_before_rows(K, a.n_groups));
    const int lane = lane_id();
    int sub, grp, c;
    lane_group(a, lane, sub, grp, c);
    if (sub >= a.rows_per_wave) return;
    float* __restrict__ dst = a.ptr[grp];
    const int gld = a.ld[grp];
    const int col = lane - sub * a.row_len;
    const bool add = mode == GS_APPLY_ADD;
    const uint32_t rpw = UNI ? 1u : (uint32_t)a.rows_per_wave;
    const uint32_t waves = gridDim.x * (GS_BLOCK / GS_WAVE);
    const uint32_t wave = __builtin_amdgcn_readfirstlane(blockIdx.x * (GS_BLOCK / GS_WAVE) + threadIdx.x / GS_WAVE);
    for (uint32_t r0 = wave * rpw * kRowsInFlight; r0 < K; r0 += waves * rpw * kRowsInFlight) {
        uint32_t rr[kRowsInFlight], id[kRowsInFlight];
        float val[kRowsInFlight], old[kRowsInFlight];
#pragma unroll
        for (int u = 0; u < kRowsInFlight; ++u) {
            const uint32_t r = r0 + (uint32_t)u * rpw + (UNI ? 0u : (uint32_t)sub);
            rr[u] = r < K ? r : K - 1u;           // past the end: re-read the last row, store nothing
        }
#pragma unroll
        for (int u = 0; u < kRowsInFlight; ++u) {
            id[u] = ids[rr[u]];
            val[u] = rows[(size_t)rr[u] * a.row_len + col];
        }
#pragma unroll
        for (int u = 0; u < kRowsInFlight; ++u) old[u] = add ? dst[(size_t)id[u] * gld + c] : 0.0f;
#pragma unroll
        for (int u = 0; u < kRowsInFlight; ++u) {
            loaded(val[u]);
            loaded(old[u]);
        }
#pragma unroll
        for (int u = 0; u < kRowsInFlight; ++u) {
            const uint32_t r = r0 + (uint32_t)u * rpw + (UNI ? 0u : (uint32_t)sub);
            if (r < K) {
                dst[(size_t)id[u] * gld + c] = add ? old[u] + val[u] : val[u];
                if (col == 0 && prim_version) prim_version[id[u]] = version;
            }
        }
    }
}

// Commit of a ring slot (Shadow Graph step 4): the message check above plus
// the slot's version and the commit order; then the rows of primitives whose
// published version is older than the message's, each stamped with it, and
// the skip markers that name this version cleared; finally the ring's
// committed version and the counts of applied / left rows.
__global__ void k_commit_order(const uint32_t* __restrict__ msg, uint32_t version,
                               const uint32_t* __restrict__ ring_state, gs_device_status* __restrict__ status) {
    if (msg[2] != version) atomicOr(&status->flags, GS_DEV_MSG_MISMATCH);
    else if (ring_state[0] + 1u != version) atomicOr(&status->flags, GS_DEV_MSG_ORDER);
}

// UNI (rows of more than 32 floats, one row per wave): the row index and
// its id are wave-uniform, so the id comes from a scalar load and stays in
// scalar registers, which leaves room for the rows in flight.
template <bool UNI>
__global__ void __launch_bounds__(GS_BLOCK) k_commit(GroupArgs a, const uint32_t* __restrict__ msg, int32_t mode,
                                                     uint32_t* __restrict__ prim_version, uint32_t* __restrict__ skip,
                                                     uint32_t* __restrict__ ring_state,
                                                     const gs_device_status* __restrict__ status) {
    if (status->flags & (GS_DEV_MSG_MISMATCH | GS_DEV_MSG_ORDER)) return;
    const uint32_t K = msg[1];
    const uint32_t version = msg[2];
    const uint64_t gw = (uint64_t)((a.n_groups + 3) / 4) * 4;
    const uint32_t* __restrict__ ids = msg + 8 + gw;
    const float* __restrict__ rows = reinterpret_cast<const float*>(msg + msg_words_before_rows(K, a.n_groups));
    const int lane = lane_id();
    int sub, grp, c;
    lane_group(a, lane, sub, grp, c);
    const bool in_row = sub < a.rows_per_wave;
    if (!in_row) grp = c = 0;                  // spare lanes read row 0's first column and store nothing
    float* __restrict__ dst = a.ptr[grp];
    const int gld = a.ld[grp];
    const int col = in_row ? lane - sub * a.row_len : 0;
    const uint32_t rpw = UNI ? 1u : (uint32_t)a.rows_per_wave;
    const uint32_t waves = gridDim.x * (GS_BLOCK / GS_WAVE);
    const uint32_t wave = __builtin_amdgcn_readfirstlane(blockIdx.x * (GS_BLOCK / GS_WAVE) + threadIdx.x / GS_WAVE);
    uint32_t left = 0;
    // every lane of the wave runs the same number of iterations (rows are
    // strided by whole waves), so the wave-level count below sees all lanes.
    // Loads are unconditional (rows past the end read row 0; every id was
    // checked against n_rows), so they are all in flight before the first use.
    for (uint32_t r0 = wave * rpw * kRowsInFlight; r0 < K; r0 += waves * rpw * kRowsInFlight) {
        uint32_t rr[kRowsInFlight], id[kRowsInFlight], pv[kRowsInFlight], sk[kRowsInFlight];
        float val[kRowsInFlight], old[kRowsInFlight];
        bool ok[kRowsInFlight];
#pragma unroll
        for (int u = 0; u < kRowsInFlight; ++u) {
            const uint32_t r = r0 + (uint32_t)u * rpw + (UNI ? 0u : (uint32_t)sub);
            ok[u] = in_row && r < K;
            rr[u] = r < K ? r : 0u;
        }
#pragma unroll
        for (int u = 0; u < kRowsInFlight; ++u) id[u] = ids[rr[u]];
#pragma unroll
        for (int u = 0; u < kRowsInFlight; ++u) {
            // every lane of the row reads the version before lane 0 stamps it
            pv[u] = prim_version[id[u]];
            val[u] = rows[(size_t)rr[u] * a.row_len + col];
            old[u] = dst[(size_t)id[u] * gld + c];
            sk[u] = skip ? skip[id[u]] : 0u;
        }
#pragma unroll
        for (int u = 0; u < kRowsInFlight; ++u) {
            loaded(pv[u]);
            loaded(val[u]);
            loaded(old[u]);
            loaded(sk[u]);
        }
#pragma unroll
        for (int u = 0; u < kRowsInFlight; ++u) {
            if (!ok[u]) continue;
            const bool newer = pv[u] < version;
            if (newer) dst[(size_t)id[u] * gld + c] = (mode == GS_APPLY_ADD) ? (old[u] + val[u]) : val[u];
            if (col == 0) {
                if (newer)
                    prim_version[id[u]] = version;
                else
                    ++left;
                if (skip && sk[u] == version) skip[id[u]] = 0u;
            }
        }
    }
    // rows left behind are rare (a later version already published them):
    // only waves that saw one touch the shared counter
    left = wave_sum_u32(left);
    if (lane == 0 && left) atomicAdd(&ring_state[5], left);
}

__global__ void k_commit_finish(const uint32_t* __restrict__ msg, uint32_t version, uint32_t* __restrict__ ring_state,
                                const gs_device_status* __restrict__ status) {
    if (status->flags & (GS_DEV_MSG_MISMATCH | GS_DEV_MSG_ORDER)) return;
    const uint32_t left = ring_state[5];
    ring_state[0] = version;
    ring_state[1] = msg[1] - left;
    ring_state[2] = left;
    ring_state[5] = 0u;
}

GroupArgs make_group_args(const gs_group* g, int32_t n) {
    GroupArgs a = {};
    int32_t rl = 0;
    for (int i = 0; i < n; ++i) {
        a.ptr[i] = g[i].ptr;
        a.cols[i] = g[i].cols;
        a.ld[i] = g[i].ld ? g[i].ld : g[i].cols;
        rl += g[i].cols;
    }
    a.n_groups = n;
    a.row_len = rl;
    a.rows_per_wave = rl > 0 ? GS_WAVE / rl : 0;
    return a;
}

// Blocks for a row loop over up to max_rows rows, rows_per_iter rows per wave
// iteration: enough to cover the rows once, at most 8 resident blocks per
// compute unit (the loop strides over the rest).
uint32_t row_blocks(int32_t max_rows, int32_t rows_per_iter) {
    if (max_rows <= 0 || rows_per_iter <= 0) return 1;
    uint32_t b = div_up(div_up((uint64_t)max_rows, (uint64_t)rows_per_iter), GS_BLOCK / GS_WAVE);
    const uint32_t cus = compute_units();
    const uint32_t cap = cus > 0 ? 8u * cus : 2048u;
    return b > cap ? cap : (b == 0 ? 1 : b);
}

}  // namespace

hipError_t launch_publish_commit(const gs_ring& ring, uint32_t version, const gs_group* dst, int32_t n_groups,
                                 int32_t n_rows, int32_t max_rows, int32_t mode, uint32_t* prim_version,
                                 uint32_t* skip, gs_device_status* status, hipStream_t st) {
    const GroupArgs a = make_group_args(dst, n_groups);
    const uint32_t* msg = static_cast<const uint32_t*>(ring.slot[version & 1u]);
    uint32_t cb = div_up((uint64_t)(max_rows > 0 ? max_rows : 1), GS_BLOCK);
    if (cb > 4096) cb = 4096;
    hipLaunchKernelGGL(k_apply_check, dim3(cb), dim3(GS_BLOCK), 0, st, a, msg, (uint64_t)ring.slot_bytes, n_rows,
                       max_rows, status);
    hipLaunchKernelGGL(k_commit_order, dim3(1), dim3(1), 0, st, msg, version, ring.state, status);
    uint32_t blocks = row_blocks(max_rows, a.rows_per_wave * kRowsInFlight);
    if (ring.background) {
        const uint32_t cus = compute_units();
        if (cus > 0 && blocks > cus) blocks = cus;
    }
    if (a.rows_per_wave == 1)
        hipLaunchKernelGGL(k_commit<true>, dim3(blocks), dim3(GS_BLOCK), 0, st, a, msg, mode, prim_version, skip,
                           ring.state, status);
    else
        hipLaunchKernelGGL(k_commit<false>, dim3(blocks), dim3(GS_BLOCK), 0, st, a, msg, mode, prim_version, skip,
                           ring.state, status);
    hipLaunchKernelGGL(k_commit_finish, dim3(1), dim3(1), 0, st, msg, version, ring.state, status);
    return hipGetLastError();
}

size_t delta_msg_bytes(uint64_t count, int32_t row_len, int32_t n_groups) {
    return (size_t)msg_bytes(count, row_len, n_groups);
}

hipError_t launch_delta_pack(const uint32_t* idx, const uint32_t* count, int32_t max_rows, const gs_group* src,
                             int32_t n_groups, uint32_t version, void* msg, size_t msg_capacity,
                             gs_device_status* status, hipStream_t st) {
    const GroupArgs a = make_group_args(src, n_groups);
    const dim3 grid(row_blocks(max_rows, a.rows_per_wave * kRowsInFlight));
    if (a.rows_per_wave == 1)
        hipLaunchKernelGGL(k_pack<true>, grid, dim3(GS_BLOCK), 0, st, a, idx, count, version,
                           static_cast<uint32_t*>(msg), (uint64_t)msg_capacity, status);
    else
        hipLaunchKernelGGL(k_pack<false>, grid, dim3(GS_BLOCK), 0, st, a, idx, count, version,
                           static_cast<uint32_t*>(msg), (uint64_t)msg_capacity, status);
    return hipGetLastError();
}

hipError_t launch_delta_apply(const void* msg, size_t msg_capacity, const gs_group* dst, int32_t n_groups,
                              int32_t n_rows, int32_t max_rows, int32_t mode, uint32_t* prim_version,
                              gs_device_status* status, hipStream_t st) {
    const GroupArgs a = make_group_args(dst, n_groups);
    uint32_t cb = div_up((uint64_t)(max_rows > 0 ? max_rows : 1), GS_BLOCK);
    if (cb > 4096) cb = 4096;
    hipLaunchKernelGGL(k_apply_check, dim3(cb), dim3(GS_BLOCK), 0, st, a, static_cast<const uint32_t*>(msg),
                       (uint64_t)msg_capacity, n_rows, max_rows, status);
    const dim3 grid(row_blocks(max_rows, a.rows_per_wave * kRowsInFlight));
    if (a.rows_per_wave == 1)
        hipLaunchKernelGGL(k_apply<true>, grid, dim3(GS_BLOCK), 0, st, a, static_cast<const uint32_t*>(msg), mode,
                           prim_version, status);
    else
        hipLaunchKernelGGL(k_apply<false>, grid, dim3(GS_BLOCK), 0, st, a, static_cast<const uint32_t*>(msg), mode,
                           prim_version, status);
    return hipGetLastError();
}

}  // namespace gsmi
