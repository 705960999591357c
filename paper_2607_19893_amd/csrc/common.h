// Internal helpers shared by the gfx950 kernels of libgsmi (wave64 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/gsmi.h"

#define GS_WAVE 64
#define GS_BLOCK 256              // 4 waves
#define GS_ITEMS 8                // items per thread in scans / sorts
#define GS_TILE_ITEMS (GS_BLOCK * GS_ITEMS)

namespace gsmi {

__device__ __forceinline__ int lane_id() { return __lane_id(); }

__device__ __forceinline__ uint64_t lanemask_lt() {
    const int l = lane_id();
    return (l == 0) ? 0ull : (~0ull >> (64 - l));
}

__device__ __forceinline__ int popc64(uint64_t m) { return __popcll(m); }

// Pins a loaded value in place: the loads issued before it complete here, and
// the compiler cannot sink them past it (a kernel that issues the loads of
// several rows first and then stores them would otherwise get a load moved
// into each row's store and wait for it there, one row at a time).
template <typename T>
__device__ __forceinline__ void loaded(T& v) {
    asm volatile("" : "+v"(v));
}

// Inclusive prefix sum over the 64 lanes of a wave.
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t v) {
    const int l = lane_id();
#pragma unroll
    for (int d = 1; d < GS_WAVE; d <<= 1) {
        uint32_t o = __shfl_up(v, d, GS_WAVE);
        if (l >= d) v += o;
    }
    return v;
}

// Sum over each 16-lane row; every lane of the row gets its row's sum.
// quad_perm [1,0,3,2], quad_perm [2,3,0,1], row_half_mirror, row_mirror.  The
// permuted operand is taken with old = 0 and bound_ctrl set (a lane outside
// EXEC contributes 0), which lets the compiler fold each step into a single
// v_add_f32 with a DPP source and interleave independent reductions.
__device__ __forceinline__ float dpp_row_sum(float v) {
    v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xF, 0xF, true));
    v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x4E, 0xF, 0xF, true));
    v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x141, 0xF, 0xF, true));
    v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x140, 0xF, 0xF, true));
    return v;
}

// Sum over a wave; every lane gets the result.  DPP row reductions followed
// by a combination of the four 16-lane rows through readlane.
__device__ __forceinline__ float wave_sum(float v) {
    v = dpp_row_sum(v);
    float r0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
    float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16));
    float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32));
    float r3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
    return (r0 + r1) + (r2 + r3);
}

__device__ __forceinline__ uint32_t wave_sum_u32(uint32_t v) {
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) v += __shfl_xor(v, d, GS_WAVE);
    return v;
}

// Exclusive scan over a 256-thread block.  `scratch` holds >= 4 uint32.
// Returns the exclusive prefix of v; *total receives the block sum.
__device__ __forceinline__ uint32_t block_excl_scan(uint32_t v, uint32_t* scratch, uint32_t* total) {
    const int w = threadIdx.x / GS_WAVE;
    const int l = lane_id();
    uint32_t inc = wave_incl_scan(v);
    if (l == GS_WAVE - 1) scratch[w] = inc;
    __syncthreads();
    uint32_t s0 = scratch[0], s1 = scratch[1], s2 = scratch[2], s3 = scratch[3];
    uint32_t before = (w > 0 ? s0 : 0) + (w > 1 ? s1 : 0) + (w > 2 ? s2 : 0);
    *total = s0 + s1 + s2 + s3;
    __syncthreads();
    return before + inc - v;
}

__device__ __forceinline__ uint32_t block_sum_u32(uint32_t v, uint32_t* scratch) {
    uint32_t t;
    block_excl_scan(v, scratch, &t);
    return t;
}

// Sum of c[0..m) by the whole workgroup, for a block's offset among the
// per-block counts of a compaction (in place of a separate scan pass).  c is
// 16-byte aligned; every thread keeps up to four 16-byte loads in flight.
__device__ __forceinline__ uint32_t block_sum_prefix(const uint32_t* __restrict__ c, uint32_t m, uint32_t* scratch) {
    const uint4* c4 = reinterpret_cast<const uint4*>(c);
    const uint32_t m4 = m / 4;
    uint32_t s = 0;
    for (uint32_t i = threadIdx.x; i < m4; i += 4 * GS_BLOCK) {
        uint4 v[4];
#pragma unroll
        for (uint32_t j = 0; j < 4; ++j) v[j] = i + j * GS_BLOCK < m4 ? c4[i + j * GS_BLOCK] : make_uint4(0u, 0u, 0u, 0u);
#pragma unroll
        for (int j = 0; j < 4; ++j) s += (v[j].x + v[j].y) + (v[j].z + v[j].w);
    }
    if (threadIdx.x < m - 4 * m4) s += c[4 * m4 + threadIdx.x];
    return block_sum_u32(s, scratch);
}

// The same over c[0..m_all), also returning in *before the sum of c[0..m_before)
// (m_before <= m_all): a block's offset and the grand total in one pass.
__device__ __forceinline__ uint32_t block_sum_prefix2(const uint32_t* __restrict__ c, uint32_t m_before,
                                                      uint32_t m_all, uint32_t* scratch, uint32_t* before) {
    const uint4* c4 = reinterpret_cast<const uint4*>(c);
    const uint32_t m4 = m_all / 4;
    uint32_t sa = 0, sb = 0;
    for (uint32_t i = threadIdx.x; i < m4; i += 4 * GS_BLOCK) {
        uint4 v[4];
#pragma unroll
        for (uint32_t j = 0; j < 4; ++j) v[j] = i + j * GS_BLOCK < m4 ? c4[i + j * GS_BLOCK] : make_uint4(0u, 0u, 0u, 0u);
#pragma unroll
        for (uint32_t j = 0; j < 4; ++j) {
            const uint32_t e = 4 * (i + j * GS_BLOCK);
            sa += (v[j].x + v[j].y) + (v[j].z + v[j].w);
            sb += (e < m_before ? v[j].x : 0u) + (e + 1 < m_before ? v[j].y : 0u) +
                  (e + 2 < m_before ? v[j].z : 0u) + (e + 3 < m_before ? v[j].w : 0u);
        }
    }
    if (threadIdx.x < m_all - 4 * m4) {
        const uint32_t e = 4 * m4 + threadIdx.x;
        sa += c[e];
        sb += e < m_before ? c[e] : 0u;
    }
    *before = block_sum_u32(sb, scratch);
    return block_sum_u32(sa, scratch);
}

}  // namespace gsmi

// ---------------------------------------------------------------------------
// Host-side helpers shared by the launch wrappers.
// ---------------------------------------------------------------------------

namespace gsmi {

// Publication message layout (see gs_delta_pack): 8 header words, the group
// widths padded to a multiple of 4 words, K ids, zero padding to 16 bytes,
// then K rows of row_len floats.
__host__ __device__ inline uint64_t msg_words_before_rows(uint64_t count, int32_t n_groups) {
    const uint64_t gw = (uint64_t)((n_groups + 3) / 4) * 4;
    return ((8 + gw + count) + 3) / 4 * 4;
}

__host__ __device__ inline uint64_t msg_bytes(uint64_t count, int32_t row_len, int32_t n_groups) {
    return 4 * (msg_words_before_rows(count, n_groups) + count * (uint64_t)row_len);
}

inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }
inline uint32_t div_up(uint64_t a, uint64_t b) { return (uint32_t)((a + b - 1) / b); }

}  // namespace gsmi
