// Scope extraction: ordered (ascending) stream compaction of a per-primitive
// predicate (a uint32 or uint8 array, or a scope bitmap), plus the small device-wide scan used by several passes.
//
// Two launches: per-block counts (blocked arrangement, 2048 items per block),
// then the scatter, in which each block adds up the counts of the blocks
// before it for its offset (a few 16-byte loads per thread: no separate scan
// pass) and recomputes each item's rank within its block; the last block
// writes the total.
#include <mutex>

#include "common.h"
#include "internal.h"

namespace gsmi {

// Fixed workspace of the visible-set compaction for callers that cannot
// allocate (gs_visible_set_noalloc).  Each GPU the library runs on holds its
// own copy until the process ends.  In host code this name is only a
// stand-in for the device symbol: host code uses the address that
// hipGetSymbolAddress returns for the current device, never the name.
static __device__ __align__(256) uint32_t scratch[GS_NOALLOC_SCRATCH_BYTES / sizeof(uint32_t)];

namespace {

template <int KIND>
__device__ __forceinline__ void load_pred(const void* src, int32_t n, int32_t base, uint32_t (&on)[GS_ITEMS]) {
    if (KIND == GS_PRED_U32_NONZERO) {
        const uint32_t* s = static_cast<const uint32_t*>(src);
        if (base + GS_ITEMS <= n) {
            const uint4 a = *reinterpret_cast<const uint4*>(s + base);
            const uint4 b = *reinterpret_cast<const uint4*>(s + base + 4);
            on[0] = a.x != 0; on[1] = a.y != 0; on[2] = a.z != 0; on[3] = a.w != 0;
            on[4] = b.x != 0; on[5] = b.y != 0; on[6] = b.z != 0; on[7] = b.w != 0;
        } else {
#pragma unroll
            for (int k = 0; k < GS_ITEMS; ++k) on[k] = (base + k < n) ? (s[base + k] != 0) : 0;
        }
    } else if (KIND == GS_PRED_BITMAP) {
        // bit i & 31 of word i >> 5; base is a multiple of 8, so the 8 items share a word
        const uint32_t word = base < n ? static_cast<const uint32_t*>(src)[base >> 5] >> (base & 31) : 0u;
#pragma unroll
        for (int k = 0; k < GS_ITEMS; ++k) on[k] = (base + k < n) ? ((word >> k) & 1u) : 0u;
    } else {
        const uint8_t* s = static_cast<const uint8_t*>(src);
        if (base + GS_ITEMS <= n) {
            const uint2 a = *reinterpret_cast<const uint2*>(s + base);
#pragma unroll
            for (int k = 0; k < 4; ++k) on[k] = ((a.x >> (8 * k)) & 0xFF) != 0;
#pragma unroll
            for (int k = 0; k < 4; ++k) on[4 + k] = ((a.y >> (8 * k)) & 0xFF) != 0;
        } else {
#pragma unroll
            for (int k = 0; k < GS_ITEMS; ++k) on[k] = (base + k < n) ? (s[base + k] != 0) : 0;
        }
    }
}

template <int KIND>
__global__ void __launch_bounds__(GS_BLOCK) k_vis_count(const void* __restrict__ src, int32_t n,
                                                        uint32_t* __restrict__ counts) {
    __shared__ uint32_t scratch[4];
    const int32_t base = blockIdx.x * GS_TILE_ITEMS + threadIdx.x * GS_ITEMS;
    uint32_t on[GS_ITEMS];
    load_pred<KIND>(src, n, base, on);
    uint32_t c = 0;
#pragma unroll
    for (int k = 0; k < GS_ITEMS; ++k) c += on[k];
    const uint32_t tot = block_sum_u32(c, scratch);
    if (threadIdx.x == 0) counts[blockIdx.x] = tot;
}

template <int KIND>
__global__ void __launch_bounds__(GS_BLOCK) k_vis_scatter(const void* __restrict__ src, int32_t n,
                                                          const uint32_t* __restrict__ counts,
                                                          uint32_t* __restrict__ out_idx,
                                                          uint32_t* __restrict__ out_count) {
    __shared__ uint32_t scratch[4];
    const uint32_t before = block_sum_prefix(counts, blockIdx.x, scratch);
    const int32_t base = blockIdx.x * GS_TILE_ITEMS + threadIdx.x * GS_ITEMS;
    uint32_t on[GS_ITEMS];
    load_pred<KIND>(src, n, base, on);
    uint32_t c = 0;
#pragma unroll
    for (int k = 0; k < GS_ITEMS; ++k) c += on[k];
    if (KIND == GS_PRED_U8_NONZERO_CLEAR && c) {
        // the flags this thread found set go back to 0 (it alone reads and writes
        // them here; the count pass read them in an earlier launch)
        uint8_t* s = static_cast<uint8_t*>(const_cast<void*>(src));
        if (base + GS_ITEMS <= n) {
            *reinterpret_cast<uint2*>(s + base) = make_uint2(0u, 0u);
        } else {
#pragma unroll
            for (int k = 0; k < GS_ITEMS; ++k)
                if (on[k]) s[base + k] = 0;
        }
    }
    uint32_t tot;
    uint32_t pos = block_excl_scan(c, scratch, &tot) + before;
#pragma unroll
    for (int k = 0; k < GS_ITEMS; ++k)
        if (on[k]) out_idx[pos++] = (uint32_t)(base + k);
    if (blockIdx.x == gridDim.x - 1 && threadIdx.x == 0) *out_count = before + tot;
}

__global__ void k_fill_u32(uint32_t* __restrict__ p, uint32_t value, size_t n) {
    const size_t i = (size_t)blockIdx.x * GS_BLOCK + threadIdx.x;
    const size_t stride = (size_t)gridDim.x * GS_BLOCK;
    for (size_t j = i; j < n; j += stride) p[j] = value;
}

}  // namespace

hipError_t launch_fill_u32(uint32_t* p, uint32_t value, size_t n, hipStream_t st) {
    if (n == 0) return hipSuccess;
    uint32_t blocks = div_up(n, GS_BLOCK);
    if (blocks > 4096) blocks = 4096;
    hipLaunchKernelGGL(k_fill_u32, dim3(blocks), dim3(GS_BLOCK), 0, st, p, value, n);
    return hipGetLastError();
}

void* noalloc_scratch(hipError_t* err) {
    // One lookup per device, made with that device current; later calls read
    // the cached address.
    constexpr int kMaxDevices = 64;
    static std::mutex mu;
    static void* ptr[kMaxDevices] = {};
    int dev = -1;
    *err = hipGetDevice(&dev);
    if (*err != hipSuccess) return nullptr;
    if (dev < 0 || dev >= kMaxDevices) {
        *err = hipErrorInvalidDevice;
        return nullptr;
    }
    std::lock_guard<std::mutex> lock(mu);
    if (ptr[dev] == nullptr) {
        void* p = nullptr;
        *err = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (*err != hipSuccess) return nullptr;
        ptr[dev] = p;
    }
    *err = hipSuccess;
    return ptr[dev];
}

size_t visible_ws_bytes(int32_t n) {
    return align256(sizeof(uint32_t) * (size_t)(div_up((uint64_t)(n > 0 ? n : 0), GS_TILE_ITEMS) + 1));
}

hipError_t launch_visible(int kind, const void* src, int32_t n, uint32_t* out_idx, uint32_t* out_count, void* ws,
                          hipStream_t st) {
    uint32_t* counts = static_cast<uint32_t*>(ws);
    const uint32_t nb = div_up((uint64_t)n, GS_TILE_ITEMS);
    if (nb == 0) return launch_fill_u32(out_count, 0u, 1, st);
    if (kind == GS_PRED_U32_NONZERO)
        hipLaunchKernelGGL(k_vis_count<GS_PRED_U32_NONZERO>, dim3(nb), dim3(GS_BLOCK), 0, st, src, n, counts);
    else if (kind == GS_PRED_BITMAP)
        hipLaunchKernelGGL(k_vis_count<GS_PRED_BITMAP>, dim3(nb), dim3(GS_BLOCK), 0, st, src, n, counts);
    else if (kind == GS_PRED_U8_NONZERO_CLEAR)
        hipLaunchKernelGGL(k_vis_count<GS_PRED_U8_NONZERO_CLEAR>, dim3(nb), dim3(GS_BLOCK), 0, st, src, n, counts);
    else
        hipLaunchKernelGGL(k_vis_count<GS_PRED_U8_NONZERO>, dim3(nb), dim3(GS_BLOCK), 0, st, src, n, counts);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (kind == GS_PRED_U32_NONZERO)
        hipLaunchKernelGGL(k_vis_scatter<GS_PRED_U32_NONZERO>, dim3(nb), dim3(GS_BLOCK), 0, st, src, n, counts,
                           out_idx, out_count);
    else if (kind == GS_PRED_BITMAP)
        hipLaunchKernelGGL(k_vis_scatter<GS_PRED_BITMAP>, dim3(nb), dim3(GS_BLOCK), 0, st, src, n, counts,
                           out_idx, out_count);
    else if (kind == GS_PRED_U8_NONZERO_CLEAR)
        hipLaunchKernelGGL(k_vis_scatter<GS_PRED_U8_NONZERO_CLEAR>, dim3(nb), dim3(GS_BLOCK), 0, st, src, n, counts,
                           out_idx, out_count);
    else
        hipLaunchKernelGGL(k_vis_scatter<GS_PRED_U8_NONZERO>, dim3(nb), dim3(GS_BLOCK), 0, st, src, n, counts,
                           out_idx, out_count);
    return hipGetLastError();
}

}  // namespace gsmi
