// Rendering phase, part 1: duplicate visible primitives per touched tile and
// order the pairs by (tile, depth, primitive id).
//
// Instead of one wide radix sort over 64-bit (tile, depth) keys:
//   1. every visible primitive's tile pairs are emitted in visible-set order
//      (ascending ids), each primitive's rectangle row-major, so a primitive's
//      pairs are contiguous ("emission order"); each emission block also
//      counts its pairs per tile in LDS and adds the non-zero counts to the
//      per-tile totals (one device atomic per distinct tile of the block);
//   2. one workgroup turns the totals into the tile ranges and the dispatch
//      order (tiles by a code of their pair count, the longest first: a
//      stable counting sort over 256 codes);
//   3. the pairs are placed in their tile's range: each block ranks its pairs
//      per tile in LDS and claims one run of slots per distinct tile from the
//      tile's cursor (a device atomic), so the order of a tile's pairs inside
//      its range depends on scheduling;
//   4. each tile's segment is sorted by (depth bits, emission position), tiles
//      taken in the dispatch order by a persistent grid: a wave sorts a tile of
//      fewer than 512 pairs in registers, a workgroup one of up to 2048 (each
//      wave 512 in registers, merges across waves through LDS), two exact runs
//      in LDS merged by rank up to 4096, and a network in global memory beyond.
//      The key is unique per pair, so the result does not depend on the order
//      step 3 left; emission positions grow with the primitive id inside a
//      tile, so this is exactly the (tile, depth bits, id) order.
// The per-tile kernels that follow (this sort, the forward and backward
// raster) end when their longest tile ends; taking the longest first lets
// the short ones fill in beside it instead of after it.
#include <algorithm>

#include "common.h"
#include "internal.h"

namespace gsmi {

namespace {

// Tile counters per LDS histogram pass of the emission and placement blocks
// (32 KB); images with more tiles take several passes over the block's keys.
constexpr uint32_t kTileChunk = 8192;

// Lanes of a wave whose digit equals this lane's digit (a 64-lane match built
// from one ballot per digit bit), restricted to the valid lanes.
__device__ __forceinline__ uint64_t match_digit(uint32_t d, bool valid, int nbits) {
    uint64_t peers = __ballot(valid);
    for (int b = 0; b < nbits; ++b) {
        const bool bit = (d >> b) & 1u;
        const uint64_t bb = __ballot(bit);
        peers &= bit ? bb : ~bb;
    }
    return peers;
}

// per-block sums of tiles[] in visible-set order
// The grid also zeroes the per-tile pair totals (T words) that the emission
// blocks add to.
__global__ void __launch_bounds__(GS_BLOCK) k_tile_sums(const uint32_t* __restrict__ order,
                                                        const uint32_t* __restrict__ vis_count,
                                                        const uint32_t* __restrict__ tiles,
                                                        uint32_t* __restrict__ bsum, uint32_t* __restrict__ tcount,
                                                        uint32_t T) {
    __shared__ uint32_t scratch[4];
    for (uint32_t i = blockIdx.x * GS_BLOCK + threadIdx.x; i < T; i += gridDim.x * GS_BLOCK) tcount[i] = 0u;
    const uint32_t V = *vis_count;
    const uint32_t base = blockIdx.x * GS_TILE_ITEMS + threadIdx.x * GS_ITEMS;
    uint32_t s = 0;
    if (blockIdx.x * GS_TILE_ITEMS < V) {
#pragma unroll
        for (int k = 0; k < GS_ITEMS; ++k)
            if (base + k < V) s += tiles[order[base + k]];
    }
    const uint32_t t = block_sum_u32(s, scratch);
    if (threadIdx.x == 0) bsum[blockIdx.x] = t;
}

// Exclusive offsets in visible-set order: pair_offset[id] and offs_r[rank],
// with offs_r[V] = M as a sentinel.  Each block adds up the per-block sums of
// k_tile_sums itself, those before it for its offset and all of them for M
// (no separate scan pass).  Also publishes the pair count and the
// overflow flag, and for every 2048-pair emission block m the rank that holds
// its first pair (bstart[m], m < nbs): the rank whose pairs [off, off + t)
// contain m * 2048 writes it, so each entry has one writer.  On overflow
// (M > capacity) no pair is emitted and pair_offset[id] = 0xFFFFFFFF, so the
// per-primitive backward finds none of its slots in the buffer.
__global__ void __launch_bounds__(GS_BLOCK) k_offsets(
    const uint32_t* __restrict__ order, const uint32_t* __restrict__ vis_count, const uint32_t* __restrict__ tiles,
    const uint32_t* __restrict__ bsum, uint32_t capacity,
    uint32_t* __restrict__ pair_offset, uint32_t* __restrict__ offs_r, uint32_t* __restrict__ sort_count,
    uint32_t* __restrict__ num_pairs, gs_device_status* __restrict__ status, uint32_t* __restrict__ bstart,
    uint32_t nbs) {
    __shared__ uint32_t scratch[4];
    const uint32_t V = *vis_count;
    const uint32_t nbv = (V + GS_TILE_ITEMS - 1) / GS_TILE_ITEMS;     // blocks that hold visible ranks
    if (blockIdx.x > 0 && blockIdx.x >= nbv) return;
    uint32_t before;
    const uint32_t M = block_sum_prefix2(bsum, min(blockIdx.x, nbv), nbv, scratch, &before);
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        *num_pairs = M;
        *sort_count = M <= capacity ? M : 0u;
        offs_r[V] = M;
        if (M > capacity && status) {
            atomicOr(&status->flags, GS_DEV_PAIR_OVERFLOW);
            atomicMax(&status->required, M);
        }
    }
    if (blockIdx.x * GS_TILE_ITEMS >= V) return;
    const uint32_t base = blockIdx.x * GS_TILE_ITEMS + threadIdx.x * GS_ITEMS;
    uint32_t t[GS_ITEMS], g[GS_ITEMS];
    uint32_t s = 0;
#pragma unroll
    for (int k = 0; k < GS_ITEMS; ++k) {
        g[k] = (base + k < V) ? order[base + k] : 0u;
        t[k] = (base + k < V) ? tiles[g[k]] : 0u;
        s += t[k];
    }
    uint32_t tot;
    uint32_t off = block_excl_scan(s, scratch, &tot) + before;
#pragma unroll
    for (int k = 0; k < GS_ITEMS; ++k) {
        if (base + k >= V) break;
        pair_offset[g[k]] = M <= capacity ? off : 0xFFFFFFFFu;
        offs_r[base + k] = off;
        const uint64_t end = (uint64_t)off + t[k];
        for (uint64_t m = ((uint64_t)off + GS_TILE_ITEMS - 1) / GS_TILE_ITEMS; m < nbs && m * GS_TILE_ITEMS < end; ++m)
            bstart[m] = base + k;
        off += t[k];
    }
}

// The pairs [base, hi) of one emission block: pair i belongs to the last of
// the block's nr ranks whose offset is <= i (a zero-tile rank shares its
// successor's offset and is passed over; the offset after the range is taken
// as +inf).  STAGED: offsets, ids and rectangles are read from the block's LDS
// copy, else from global memory (g_off, g_order: the range's first rank).
// Per pair: tile (pkeys), primitive (pvals) and the primitive's depth bits
// (pdepth); the tile of each of the thread's pairs is also left in key[]
// (0xFFFFFFFF past hi).
template <bool STAGED>
__device__ __forceinline__ void emit_block_pairs(uint32_t base, uint32_t hi, uint32_t nr, const uint32_t* s_off,
                                                 const uint32_t* s_gid, const ushort4* s_rect,
                                                 const uint32_t* __restrict__ g_off,
                                                 const uint32_t* __restrict__ g_order,
                                                 const ushort4* __restrict__ rect, int32_t tiles_x,
                                                 const float* __restrict__ depth, uint32_t* __restrict__ pkeys,
                                                 uint32_t* __restrict__ pvals, uint32_t* __restrict__ pdepth,
                                                 uint32_t (&key)[GS_ITEMS]) {
#pragma unroll
    for (int k = 0; k < GS_ITEMS; ++k) {
        const uint32_t i = base + k * GS_BLOCK + threadIdx.x;
        key[k] = 0xFFFFFFFFu;
        if (i >= hi) continue;
        uint32_t lo = 0, up = nr;
        while (up - lo > 1) {
            const uint32_t mid = (lo + up) >> 1;
            if ((STAGED ? s_off[mid] : g_off[mid]) <= i) lo = mid; else up = mid;
        }
        const uint32_t gid = STAGED ? s_gid[lo] : g_order[lo];
        const ushort4 rc = STAGED ? s_rect[lo] : rect[gid];
        const uint32_t local = i - (STAGED ? s_off[lo] : g_off[lo]);
        const uint32_t w = (uint32_t)(rc.z - rc.x);
        const uint32_t ty = rc.y + local / w;
        const uint32_t tx = rc.x + local % w;
        key[k] = ty * (uint32_t)tiles_x + tx;
        pkeys[i] = key[k];
        pvals[i] = gid;
        pdepth[i] = __float_as_uint(depth[gid]);
    }
}

// One thread per pair: pair i belongs to the rank r with offs_r[r] <= i <
// offs_r[r+1] and covers tile number i - offs_r[r] of that primitive's
// rectangle (row-major).  Each block locates its rank range once, stages the
// offsets, ids and rectangles of those ranks in LDS and binary-searches
// there; key (tile id) and value (primitive id) stores are contiguous.  Then
// the block counts its pairs per tile in LDS (the staging memory reused) and
// adds every non-zero count to the tile's total.
__global__ void __launch_bounds__(GS_BLOCK) k_emit_pairs(
    const uint32_t* __restrict__ order, const uint32_t* __restrict__ vis_count, const uint32_t* __restrict__ offs_r,
    const uint32_t* __restrict__ bstart, const ushort4* __restrict__ rect, const float* __restrict__ depth,
    const uint32_t* __restrict__ sort_count, int32_t tiles_x, uint32_t T, uint32_t* __restrict__ pkeys,
    uint32_t* __restrict__ pvals, uint32_t* __restrict__ pdepth, uint32_t* __restrict__ tcount) {
    constexpr uint32_t kStage = GS_TILE_ITEMS + 1;
    static_assert(kStage * 16 >= kTileChunk * 4, "the tile histogram fits in the staging memory");
    __shared__ __align__(16) unsigned char s_mem[kStage * 16];
    ushort4* s_rect = reinterpret_cast<ushort4*>(s_mem);
    uint32_t* s_off = reinterpret_cast<uint32_t*>(s_mem + kStage * 8);
    uint32_t* s_gid = reinterpret_cast<uint32_t*>(s_mem + kStage * 12);
    __shared__ uint32_t s_range[2];
    const uint32_t M = *sort_count;
    const uint32_t base = blockIdx.x * GS_TILE_ITEMS;
    if (base >= M) return;
    const uint32_t hi = min(base + (uint32_t)GS_TILE_ITEMS, M);
    if (threadIdx.x == 0) {
        // the ranks of the block's first and last pairs: the first from the table
        // k_offsets wrote; the last is the next block's first rank, or the one
        // before it when that rank starts exactly at hi (the last rank for the
        // last block), stepping back over ranks that start later
        const uint32_t r0 = bstart[blockIdx.x];
        uint32_t r1 = hi == M ? *vis_count - 1u : bstart[blockIdx.x + 1];
        while (r1 > r0 && offs_r[r1] > hi - 1u) --r1;
        s_range[0] = r0;
        s_range[1] = r1;
    }
    __syncthreads();
    const uint32_t r0 = s_range[0];
    // Ranks holding pairs of this block: at most GS_TILE_ITEMS + 1 when every
    // rank holds >= 1 pair (the visible set of gs_project's tile counts); a
    // caller list with zero-tile ids can span more, and then the block
    // searches the offsets in global memory instead of staging them.
    const uint32_t nr = s_range[1] - r0 + 1;
    const bool staged = nr <= kStage;
    if (staged) {
        for (uint32_t j = threadIdx.x; j < nr; j += GS_BLOCK) {
            const uint32_t g = order[r0 + j];
            s_off[j] = offs_r[r0 + j];
            s_gid[j] = g;
            s_rect[j] = rect[g];
        }
    }
    __syncthreads();
    uint32_t key[GS_ITEMS];
    if (staged)
        emit_block_pairs<true>(base, hi, nr, s_off, s_gid, s_rect, offs_r + r0, order + r0, rect, tiles_x, depth,
                               pkeys, pvals, pdepth, key);
    else
        emit_block_pairs<false>(base, hi, nr, s_off, s_gid, s_rect, offs_r + r0, order + r0, rect, tiles_x, depth,
                                pkeys, pvals, pdepth, key);
    uint32_t* h = reinterpret_cast<uint32_t*>(s_mem);
    for (uint32_t c0 = 0; c0 < T; c0 += kTileChunk) {
        const uint32_t nc = min(kTileChunk, T - c0);
        __syncthreads();    // the staging (first chunk) or the last chunk's flush is done
        for (uint32_t d = threadIdx.x; d < nc; d += GS_BLOCK) h[d] = 0u;
        __syncthreads();
#pragma unroll
        for (int k = 0; k < GS_ITEMS; ++k)
            if (key[k] - c0 < nc) atomicAdd(&h[key[k] - c0], 1u);
        __syncthreads();
        for (uint32_t d = threadIdx.x; d < nc; d += GS_BLOCK) {
            const uint32_t c = h[d];
            if (c) atomicAdd(&tcount[c0 + d], c);
        }
    }
}

// Dispatch key of a tile from its pair count: an 8-bit code that never
// decreases with the count (exact below 16, then 16 steps per octave; counts
// of 2^19 and more share the top code), inverted so that ascending keys put
// the longest tiles first.
__device__ __forceinline__ uint32_t tile_order_key(uint32_t n) {
    uint32_t code = n;
    if (n >= 16u) {
        const uint32_t e = 31u - (uint32_t)__clz(n);      // >= 4
        code = e > 18u ? 255u : 16u * (e - 3u) + ((n >> (e - 4u)) & 15u);
    }
    return 255u - code;
}

// Tiles with fewer pairs than this are depth-sorted by one wave in registers;
// the order key is monotone in the count, so these are exactly the tiles with
// keys above kLongKey, and the dispatch order puts all others first.
constexpr uint32_t kWaveSortMax = 512;
constexpr uint32_t kLongKey = 255u - 96u;   // tile_order_key(512): code 16 * (9 - 3) + 0
static_assert(kWaveSortMax == 512u, "kLongKey is the key of 512 pairs");

// Exclusive scan over the 4 waves of a workgroup of GS_BLOCK threads is
// block_excl_scan.

// Tiles per workgroup of the finishing grid (2 per thread), and the totals
// each thread loads per pass over all tiles (one pass up to 8192 tiles).
constexpr uint32_t kFinishPer = 2;
constexpr uint32_t kFinishSeg = kFinishPer * GS_BLOCK;
constexpr int kFinishLoads = 32;

// From the per-tile totals: the tile ranges (exclusive scan in tile order;
// [0, 0) for a tile without pairs), the placement cursors (each range's
// start), the dispatch order (tiles by ascending tile_order_key, equal keys
// by ascending id) with one record per dispatch position (tile, range start,
// pair count), and the number of tiles with kWaveSortMax pairs or more, which
// the order puts first.  Workgroup b owns the tiles [b*kFinishSeg, ..) of one
// segment.  It reads every total (all loads of a pass in flight together):
// their sum before the segment starts its ranges, and the key counts over all
// tiles and over the tiles before the segment give each key's first position
// for the segment; the segment's own totals and range starts stay in LDS.
// Inside the segment, wave w owns a contiguous quarter: it counts its keys,
// the counts give every (wave, key) its first position, and the wave then
// places its tiles 64 at a time, each lane ranked among the earlier lanes
// with its key.
__global__ void __launch_bounds__(GS_BLOCK) k_tile_finish(const uint32_t* __restrict__ tcount, uint32_t T,
                                                          uint32_t* __restrict__ ranges,
                                                          uint32_t* __restrict__ cursor,
                                                          uint32_t* __restrict__ order, uint4* __restrict__ rec,
                                                          uint32_t* __restrict__ n_long) {
    constexpr int kWaves = GS_BLOCK / GS_WAVE;
    __shared__ uint32_t s_all[256], s_before[256];
    __shared__ uint32_t s_wc[kWaves][256];
    __shared__ uint32_t s_cnt[kFinishSeg], s_sta[kFinishSeg];
    __shared__ uint32_t scratch[4];
    const uint32_t tid = threadIdx.x;
    const uint32_t w = tid / GS_WAVE;
    const uint32_t lane = lane_id();
    const uint32_t lo = blockIdx.x * kFinishSeg, hi = min(lo + kFinishSeg, T);
    s_all[tid] = 0u;
    s_before[tid] = 0u;
    s_wc[0][tid] = 0u; s_wc[1][tid] = 0u; s_wc[2][tid] = 0u; s_wc[3][tid] = 0u;
    __syncthreads();
    // every total: key counts over all tiles and before the segment, the pairs
    // before it; the segment's totals to LDS
    uint32_t before = 0;
    for (uint32_t r0 = 0; r0 < T; r0 += GS_BLOCK * kFinishLoads) {
        uint32_t c[kFinishLoads];
#pragma unroll
        for (int k = 0; k < kFinishLoads; ++k) c[k] = tcount[min(r0 + k * GS_BLOCK + tid, T - 1u)];
#pragma unroll
        for (int k = 0; k < kFinishLoads; ++k) loaded(c[k]);
#pragma unroll
        for (int k = 0; k < kFinishLoads; ++k) {
            const uint32_t t = r0 + k * GS_BLOCK + tid;
            if (t < T) {
                const uint32_t key = tile_order_key(c[k]);
                atomicAdd(&s_all[key], 1u);
                if (t < lo) {
                    atomicAdd(&s_before[key], 1u);
                    before += c[k];
                } else if (t < hi) {
                    s_cnt[t - lo] = c[k];
                }
            }
        }
    }
    __syncthreads();
    // the segment: kFinishPer consecutive tiles per thread
    const uint32_t l0 = tid * kFinishPer;
    uint32_t c[kFinishPer], csum = 0;
#pragma unroll
    for (uint32_t k = 0; k < kFinishPer; ++k) {
        c[k] = lo + l0 + k < hi ? s_cnt[l0 + k] : 0u;
        csum += c[k];
    }
    uint32_t tot;
    const uint32_t pre = block_sum_u32(before, scratch);       // (the block's sum of `before`)
    uint32_t run = block_excl_scan(csum, scratch, &tot) + pre;
#pragma unroll
    for (uint32_t k = 0; k < kFinishPer; ++k) {
        const uint32_t t = lo + l0 + k;
        if (t < hi) {
            ranges[2 * t] = c[k] ? run : 0u;
            ranges[2 * t + 1] = c[k] ? run + c[k] : 0u;
            cursor[t] = run;
            s_sta[l0 + k] = c[k] ? run : 0u;
        }
        run += c[k];
    }
    // key d (thread d): its first position for the segment
    {
        uint32_t ktot;
        const uint32_t kstart = block_excl_scan(s_all[tid], scratch, &ktot);
        if (blockIdx.x == 0 && tid == kLongKey + 1u) *n_long = kstart;   // tiles with key <= kLongKey come first
        s_all[tid] = kstart + s_before[tid];
    }
    // per wave: key counts of its quarter of the segment (its lanes' tiles, in order)
    const uint32_t qlo = w * (kFinishSeg / kWaves);                         // segment-relative
    const uint32_t qhi = min(qlo + kFinishSeg / kWaves, hi - lo);
    uint32_t* wc = s_wc[w];
    __syncthreads();
    for (uint32_t l = qlo + lane; l < qhi; l += GS_WAVE) atomicAdd(&wc[tile_order_key(s_cnt[l])], 1u);
    __syncthreads();
    {
        uint32_t b = s_all[tid];
        const uint32_t c0 = s_wc[0][tid], c1 = s_wc[1][tid], c2 = s_wc[2][tid];
        s_wc[0][tid] = b;
        s_wc[1][tid] = b + c0;
        s_wc[2][tid] = b + c0 + c1;
        s_wc[3][tid] = b + c0 + c1 + c2;
    }
    __syncthreads();
    // placement: the quarter's tiles 64 at a time
    const uint64_t lt = lanemask_lt();
    for (uint32_t b0 = qlo; b0 < qhi; b0 += GS_WAVE) {
        const uint32_t l = b0 + lane;
        const bool valid = l < qhi;
        const uint32_t cnt = valid ? s_cnt[l] : 0u;
        const uint32_t sta = valid ? s_sta[l] : 0u;
        const uint32_t key = tile_order_key(cnt);
        const uint64_t peers = match_digit(key, valid, 8);
        const uint32_t bw = valid ? wc[key] : 0u;
        if (valid) {
            const uint32_t pos = bw + (uint32_t)popc64(peers & lt);
            order[pos] = lo + l;
            rec[pos] = make_uint4(lo + l, sta, cnt, 0u);
        }
        // all reads of this round precede the leaders' updates
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        if (valid && (peers & lt) == 0ull) wc[key] = bw + (uint32_t)popc64(peers);
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
}

// Placement of the emitted pairs in their tiles' ranges: the block ranks its
// pairs per tile in LDS, claims one run of slots per distinct tile from the
// tile's cursor, and writes each pair's depth-sort key at its slot (the depth
// bits above the emission position) and the pair's primitive beside it.
__global__ void __launch_bounds__(GS_BLOCK) k_tile_scatter(const uint32_t* __restrict__ pkeys,
                                                           const uint32_t* __restrict__ pvals,
                                                           const uint32_t* __restrict__ pdepth,
                                                           const uint32_t* __restrict__ sort_count, uint32_t T,
                                                           uint32_t* __restrict__ cursor,
                                                           unsigned long long* __restrict__ skey,
                                                           uint32_t* __restrict__ sval) {
    __shared__ uint32_t h[kTileChunk];
    const uint32_t M = *sort_count;
    const uint32_t base = blockIdx.x * GS_TILE_ITEMS + threadIdx.x;
    if (blockIdx.x * GS_TILE_ITEMS >= M) return;
    uint32_t key[GS_ITEMS], dep[GS_ITEMS], gid[GS_ITEMS], rk[GS_ITEMS];
#pragma unroll
    for (int k = 0; k < GS_ITEMS; ++k) {
        const uint32_t i = base + k * GS_BLOCK;
        key[k] = i < M ? pkeys[i] : 0xFFFFFFFFu;
        dep[k] = i < M ? pdepth[i] : 0u;
        gid[k] = i < M ? pvals[i] : 0u;
        rk[k] = 0u;
    }
    for (uint32_t c0 = 0; c0 < T; c0 += kTileChunk) {
        const uint32_t nc = min(kTileChunk, T - c0);
        for (uint32_t d = threadIdx.x; d < nc; d += GS_BLOCK) h[d] = 0u;
        __syncthreads();
#pragma unroll
        for (int k = 0; k < GS_ITEMS; ++k)
            if (key[k] - c0 < nc) rk[k] = atomicAdd(&h[key[k] - c0], 1u);
        __syncthreads();
        for (uint32_t d = threadIdx.x; d < nc; d += GS_BLOCK) {
            const uint32_t c = h[d];
            if (c) h[d] = atomicAdd(&cursor[c0 + d], c);
        }
        __syncthreads();
#pragma unroll
        for (int k = 0; k < GS_ITEMS; ++k)
            if (key[k] - c0 < nc) {
                const uint32_t at = h[key[k] - c0] + rk[k];
                skey[at] = ((unsigned long long)dep[k] << 32) | (base + k * GS_BLOCK);
                sval[at] = gid[k];
            }
        __syncthreads();    // before the next chunk clears the counters
    }
}

// Per-tile ordering.  A tile's pairs arrive in its range in any order, each
// as a 64-bit key (depth bits above the emission position) and the pair's
// primitive.  The fast paths sort the 32-bit depth bits alone, each with the
// index of its slot as payload; pairs with equal depth bits (a run of
// neighbours in that order) are then placed by their emission positions,
// which gives the order by (depth bits, emission position).  A tile with a
// run longer than kRunMax (or a depth key equal to the padding value) is
// sorted again, exactly, on the 64-bit keys.
constexpr unsigned long long kKeyMax = ~0ull;
constexpr uint32_t kDepthPad = 0xFFFFFFFFu;
constexpr uint32_t kRunMax = 64;

// Bitonic network, in the variant whose compare-exchanges all put the smaller
// key at the lower index: each merge of width k (a power of two) first
// compares i with its mirror i ^ (k - 1), then i with i ^ j for j = k/4 .. 1.

// The exact network on a segment of global memory of any length n, by a
// whole workgroup: entries at n and beyond are taken as kKeyMax, so a
// compare-exchange that reaches past the data leaves the lower (real) entry
// in place.  Payloads move with their keys.
__device__ void bitonic_global(unsigned long long* s, uint32_t* pay, uint32_t n) {
    uint32_t np = 1;
    while (np < n) np <<= 1;
    for (uint32_t k = 2; k <= np; k <<= 1) {
        for (uint32_t j = k >> 1; j > 0; j >>= 1) {
            const uint32_t mask = (j == (k >> 1)) ? (k - 1) : j;
            for (uint32_t c = threadIdx.x; c < (np >> 1); c += GS_BLOCK) {
                const uint32_t i = ((c & ~(j - 1)) << 1) | (c & (j - 1));
                const uint32_t q = i ^ mask;
                if (q >= n) continue;
                const unsigned long long a = s[i], b = s[q];
                if (b < a) {
                    const uint32_t pa = pay[i], pb = pay[q];
                    s[i] = b;
                    s[q] = a;
                    pay[i] = pb;
                    pay[q] = pa;
                }
            }
            __threadfence_block();
            __syncthreads();
        }
    }
}

// LDS accesses of one wave, ordered (no other wave touches the memory).
__device__ __forceinline__ void wave_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Writes sorted pair `at` of tile t: its emission position, primitive id and
// optional 64-bit key.
__device__ __forceinline__ void put_sorted(uint32_t t, uint32_t at, unsigned long long k, uint32_t gid,
                                           uint32_t* __restrict__ pair_emit, uint32_t* __restrict__ vals,
                                           uint64_t* __restrict__ keys64) {
    vals[at] = gid;
    pair_emit[at] = (uint32_t)k;
    if (keys64) keys64[at] = ((uint64_t)t << 32) | (k >> 32);
}

// The exact network over the n (<= 512) 64-bit keys of a tile by one wave,
// in the wave's own LDS (sk, sv: 512 entries).
__device__ void wave_sort_tile64(uint32_t t, uint32_t start, uint32_t n, const unsigned long long* __restrict__ skey,
                                 const uint32_t* __restrict__ sval, unsigned long long* sk, uint32_t* sv,
                                 uint32_t* __restrict__ pair_emit, uint32_t* __restrict__ vals,
                                 uint64_t* __restrict__ keys64) {
    const uint32_t lane = lane_id();
    uint32_t np = 2;
    while (np < n) np <<= 1;
    for (uint32_t i = lane; i < np; i += GS_WAVE) {
        sk[i] = i < n ? skey[start + i] : kKeyMax;
        sv[i] = i < n ? sval[start + i] : 0u;
    }
    wave_sync();
    for (uint32_t k = 2; k <= np; k <<= 1) {
        for (uint32_t j = k >> 1; j > 0; j >>= 1) {
            const uint32_t mask = (j == (k >> 1)) ? (k - 1) : j;
            for (uint32_t c = lane; c < (np >> 1); c += GS_WAVE) {
                const uint32_t i = ((c & ~(j - 1)) << 1) | (c & (j - 1));
                const uint32_t q = i ^ mask;
                const unsigned long long a = sk[i], b = sk[q];
                if (b < a) {
                    const uint32_t pa = sv[i], pb = sv[q];
                    sk[i] = b;
                    sk[q] = a;
                    sv[i] = pb;
                    sv[q] = pa;
                }
            }
            wave_sync();
        }
    }
    for (uint32_t i = lane; i < n; i += GS_WAVE) put_sorted(t, start + i, sk[i], sv[i], pair_emit, vals, keys64);
    wave_sync();
}

// Lane l's value of lane l ^ M: DPP inside rows for the masks 1, 2, 3, 7 and
// 15, a swizzle inside 32-lane halves for the other masks below 32, a
// permute for 32 and 63.  Every lane of the wave must be active.
template <int M>
__device__ __forceinline__ uint32_t lane_xor(uint32_t v) {
    if constexpr (M == 1)
        return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xF, 0xF, false);    // quad_perm 1,0,3,2
    else if constexpr (M == 2)
        return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xF, 0xF, false);    // quad_perm 2,3,0,1
    else if constexpr (M == 3)
        return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x1B, 0xF, 0xF, false);    // quad_perm 3,2,1,0
    else if constexpr (M == 7)
        return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x141, 0xF, 0xF, false);   // row_half_mirror
    else if constexpr (M == 15)
        return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x140, 0xF, 0xF, false);   // row_mirror
    else if constexpr (M < 32)
        return (uint32_t)__builtin_amdgcn_ds_swizzle((int)v, (M << 10) | 0x1F);            // and 31, xor M
    else
        return __shfl_xor(v, M, GS_WAVE);
}

// Compare-exchange inside a lane: the smaller key (and its payload) to a.
__device__ __forceinline__ void cmpx32(uint32_t& a, uint32_t& pa, uint32_t& b, uint32_t& pb) {
    const bool sw = b < a;
    const uint32_t lo = sw ? b : a, hi = sw ? a : b, plo = sw ? pb : pa, phi = sw ? pa : pb;
    a = lo;
    b = hi;
    pa = plo;
    pb = phi;
}

// One side of a step across lanes or waves: the lower side keeps the
// smaller key, the upper side the larger.
__device__ __forceinline__ void keep32(uint32_t& v, uint32_t& p, uint32_t o, uint32_t op, bool lower) {
    const bool take = lower ? (o < v) : (v < o);
    v = take ? o : v;
    p = take ? op : p;
}

// The network on the 64 K keys of one wave in registers: element i = lane * K
// + r sits in register r of its lane, so a step at distance below K stays
// inside a lane and one at a larger distance pairs lane l with lane l ^
// (distance / K), same register.

// Steps i against i ^ j for j = J, J/2, .. 1.
template <int K, int J>
__device__ __forceinline__ void tail32(uint32_t (&v)[K], uint32_t (&p)[K], uint32_t lane) {
    if constexpr (J > 0) {
        if constexpr (J < K) {
#pragma unroll
            for (int r = 0; r < K; ++r)
                if ((r & J) == 0) cmpx32(v[r], p[r], v[r | J], p[r | J]);
        } else {
            const bool lower = (lane & (uint32_t)(J / K)) == 0;
#pragma unroll
            for (int r = 0; r < K; ++r) keep32(v[r], p[r], lane_xor<J / K>(v[r]), lane_xor<J / K>(p[r]), lower);
        }
        tail32<K, J / 2>(v, p, lane);
    }
}

// Mirror step of a merge of width KK: i against i ^ (KK - 1).
template <int K, int KK>
__device__ __forceinline__ void mirror32(uint32_t (&v)[K], uint32_t (&p)[K], uint32_t lane) {
    if constexpr (KK <= K) {
#pragma unroll
        for (int r = 0; r < K; ++r)
            if ((r & (KK / 2)) == 0) cmpx32(v[r], p[r], v[r ^ (KK - 1)], p[r ^ (KK - 1)]);
    } else {
        const bool lower = (lane & (uint32_t)(KK / K / 2)) == 0;
        uint32_t o[K], op[K];
#pragma unroll
        for (int r = 0; r < K; ++r) {
            o[r] = lane_xor<KK / K - 1>(v[r ^ (K - 1)]);
            op[r] = lane_xor<KK / K - 1>(p[r ^ (K - 1)]);
        }
#pragma unroll
        for (int r = 0; r < K; ++r) keep32(v[r], p[r], o[r], op[r], lower);
    }
}

// Merges of width 2 .. KK: every block of KK elements ascending.
template <int K, int KK>
__device__ __forceinline__ void net32(uint32_t (&v)[K], uint32_t (&p)[K], uint32_t lane) {
    if constexpr (KK >= 2) {
        net32<K, KK / 2>(v, p, lane);
        mirror32<K, KK>(v, p, lane);
        tail32<K, KK / 4>(v, p, lane);
    }
}

// Depth bits and emission position of key i (its high and low words).
__device__ __forceinline__ uint32_t key_depth(const unsigned long long* __restrict__ skey, uint32_t i) {
    return reinterpret_cast<const uint32_t*>(skey)[2 * (size_t)i + 1];
}
__device__ __forceinline__ uint32_t key_emit(const unsigned long long* __restrict__ skey, uint32_t i) {
    return reinterpret_cast<const uint32_t*>(skey)[2 * (size_t)i];
}

// Writes the pairs of a tile sorted by depth bits: sorted pair i is slot p.
__device__ __forceinline__ void put_by_slot(uint32_t t, uint32_t start, uint32_t i, uint32_t depth, uint32_t p,
                                            const unsigned long long* __restrict__ skey,
                                            const uint32_t* __restrict__ sval, uint32_t* __restrict__ pair_emit,
                                            uint32_t* __restrict__ vals, uint64_t* __restrict__ keys64) {
    put_sorted(t, start + i, ((unsigned long long)depth << 32) | key_emit(skey, start + p), sval[start + p], pair_emit,
               vals, keys64);
}

// Runs of equal depth bits.  sk[0..n) holds a tile's keys in the order of
// their depth bits (ties in any order), sv their primitives.  long_run: some
// run is longer than kRunMax (then entry i and entry i - kRunMax share their
// depth bits).  place_runs writes sorted pair i for i = first, first + step,
// ..: an entry outside a run stays at i; one inside a run [a, b) goes to a +
// the number of the run's entries with a smaller key (emission position).
__device__ __forceinline__ uint32_t hi32(unsigned long long k) { return (uint32_t)(k >> 32); }

__device__ __forceinline__ bool long_run(const unsigned long long* sk, uint32_t n, uint32_t first, uint32_t step) {
    bool bad = false;
    for (uint32_t i = first + kRunMax; i < n; i += step) bad |= hi32(sk[i]) == hi32(sk[i - kRunMax]);
    return bad;
}

__device__ __forceinline__ void place_runs(uint32_t t, uint32_t start, uint32_t n, const unsigned long long* sk,
                                           const uint32_t* sv, uint32_t first, uint32_t step,
                                           uint32_t* __restrict__ pair_emit, uint32_t* __restrict__ vals,
                                           uint64_t* __restrict__ keys64) {
    for (uint32_t i = first; i < n; i += step) {
        const unsigned long long k = sk[i];
        const uint32_t d = hi32(k);
        uint32_t a = i, b = i + 1;
        while (a > 0 && hi32(sk[a - 1]) == d) --a;
        while (b < n && hi32(sk[b]) == d) ++b;
        uint32_t at = a;
        for (uint32_t j = a; j < b; ++j) at += sk[j] < k ? 1u : 0u;
        put_sorted(t, start + at, k, sv[i], pair_emit, vals, keys64);
    }
}

// One wave sorts the n (<= 64 K) pairs of one tile: the fast path in
// registers, else wave_sort_tile64 in the wave's LDS.
template <int K>
__device__ __forceinline__ void wave_sort_tile(uint32_t t, uint32_t start, uint32_t n,
                                               const unsigned long long* __restrict__ skey,
                                               const uint32_t* __restrict__ sval, unsigned long long* sk, uint32_t* sv,
                                               uint32_t* __restrict__ pair_emit, uint32_t* __restrict__ vals,
                                               uint64_t* __restrict__ keys64) {
    const uint32_t lane = lane_id();
    uint32_t v[K], p[K];
    bool odd = false;
#pragma unroll
    for (int r = 0; r < K; ++r) {
        const uint32_t i = lane * K + r;
        v[r] = i < n ? key_depth(skey, start + i) : kDepthPad;
        p[r] = i;
        odd |= i < n && v[r] == kDepthPad;
    }
    bool tie = false;
    if (__ballot(odd) == 0ull) {
        net32<K, GS_WAVE * K>(v, p, lane);
        // equal neighbours in the sorted order: i and i + 1 < n
#pragma unroll
        for (int r = 0; r + 1 < K; ++r) tie |= lane * K + r + 1 < n && v[r] == v[r + 1];
        const uint32_t next = __shfl_down(v[0], 1, GS_WAVE);
        tie |= lane + 1 < GS_WAVE && (lane + 1) * K < n && v[K - 1] == next;
    }
    if (__ballot(odd) != 0ull) {
        wave_sort_tile64(t, start, n, skey, sval, sk, sv, pair_emit, vals, keys64);
        return;
    }
    if (__ballot(tie) == 0ull) {
#pragma unroll
        for (int r = 0; r < K; ++r)
            if (lane * K + r < n) put_by_slot(t, start, lane * K + r, v[r], p[r], skey, sval, pair_emit, vals, keys64);
        return;
    }
    // equal depth bits: the sorted keys to LDS, then each run placed by emission position
#pragma unroll
    for (int r = 0; r < K; ++r) {
        const uint32_t i = lane * K + r;
        if (i < n) {
            sk[i] = ((unsigned long long)v[r] << 32) | key_emit(skey, start + p[r]);
            sv[i] = sval[start + p[r]];
        }
    }
    wave_sync();
    if (__ballot(long_run(sk, n, lane, GS_WAVE)) != 0ull) {
        wave_sync();
        wave_sort_tile64(t, start, n, skey, sval, sk, sv, pair_emit, vals, keys64);
        return;
    }
    place_runs(t, start, n, sk, sv, lane, GS_WAVE, pair_emit, vals, keys64);
    wave_sync();
}

// Long tiles: kWaveSortMax .. kLongCap pairs are sorted by the workgroup's
// waves in registers, kWaveSortMax keys each; merges wider than one wave take
// their cross-wave steps through LDS.  Longer tiles take the exact network in
// global memory.
constexpr int kSortWaves = GS_BLOCK / GS_WAVE;
constexpr uint32_t kLongCap = kSortWaves * kWaveSortMax;
constexpr int kLongK = (int)kWaveSortMax / GS_WAVE;     // keys per lane
// Workgroups per compute unit of the persistent depth-sort grid.
constexpr uint32_t kDepthSortBlocksPerCU = 8;

// The exact network over the n (<= kLongCap) 64-bit keys skey[start ..
// start + n) by the whole workgroup in LDS: sorted keys in sk[0..n), their
// primitives in sv.
__device__ void block_sort_lds64(uint32_t start, uint32_t n, const unsigned long long* __restrict__ skey,
                                 const uint32_t* __restrict__ sval, unsigned long long* sk, uint32_t* sv) {
    uint32_t np = 2;
    while (np < n) np <<= 1;
    for (uint32_t i = threadIdx.x; i < np; i += GS_BLOCK) {
        sk[i] = i < n ? skey[start + i] : kKeyMax;
        sv[i] = i < n ? sval[start + i] : 0u;
    }
    __syncthreads();
    for (uint32_t k = 2; k <= np; k <<= 1) {
        for (uint32_t j = k >> 1; j > 0; j >>= 1) {
            const uint32_t mask = (j == (k >> 1)) ? (k - 1) : j;
            for (uint32_t c = threadIdx.x; c < (np >> 1); c += GS_BLOCK) {
                const uint32_t i = ((c & ~(j - 1)) << 1) | (c & (j - 1));
                const uint32_t q = i ^ mask;
                const unsigned long long a = sk[i], b = sk[q];
                if (b < a) {
                    const uint32_t pa = sv[i], pb = sv[q];
                    sk[i] = b;
                    sk[q] = a;
                    sv[i] = pb;
                    sv[q] = pa;
                }
            }
            __syncthreads();
        }
    }
}

// The exact network over the n (<= kLongCap) 64-bit keys of a tile by the
// whole workgroup in LDS, written out in order.
__device__ void block_sort_tile64(uint32_t t, uint32_t start, uint32_t n, const unsigned long long* __restrict__ skey,
                                  const uint32_t* __restrict__ sval, unsigned long long* sk, uint32_t* sv,
                                  uint32_t* __restrict__ pair_emit, uint32_t* __restrict__ vals,
                                  uint64_t* __restrict__ keys64) {
    block_sort_lds64(start, n, skey, sval, sk, sv);
    for (uint32_t i = threadIdx.x; i < n; i += GS_BLOCK) put_sorted(t, start + i, sk[i], sv[i], pair_emit, vals, keys64);
    __syncthreads();
}

// Number of keys below each of the thread's R keys in the ascending keys
// sk[0..m) (keys are unique): a branch-free binary search, the R searches
// stepping together.
template <int R>
__device__ __forceinline__ void rank_in(const unsigned long long* sk, uint32_t m, const unsigned long long (&key)[R],
                                        uint32_t (&pos)[R]) {
    uint32_t step = 1;
    while (step <= m) step <<= 1;
#pragma unroll
    for (int k = 0; k < R; ++k) pos[k] = 0;
    for (step >>= 1; step > 0; step >>= 1) {
#pragma unroll
        for (int k = 0; k < R; ++k)
            if (pos[k] + step <= m && sk[pos[k] + step - 1] < key[k]) pos[k] += step;
    }
}

// A tile of kLongCap < n <= 2 kLongCap pairs: its first kLongCap keys and the
// rest are each sorted exactly in LDS, and every key goes to its index in
// its own run plus its rank in the other run (the merged order; keys are
// unique).  Each sorted run is kept in its own place in global memory (this
// workgroup's segment) while the other one sits in LDS; the ranks are
// searched kRankGroup keys at a time per thread.
constexpr int kRankGroup = 4;

// The keys of run [r0, r0 + m) of the segment, ranked in the ascending keys
// sk[0..mo) in LDS; key i of the run goes to r_out + i + its rank.
__device__ __forceinline__ void place_ranked(uint32_t t, uint32_t start, uint32_t r0, uint32_t m, uint32_t r_out,
                                             const unsigned long long* __restrict__ skey,
                                             const uint32_t* __restrict__ sval, const unsigned long long* sk,
                                             uint32_t mo, uint32_t* __restrict__ pair_emit,
                                             uint32_t* __restrict__ vals, uint64_t* __restrict__ keys64) {
    constexpr uint32_t kGroupSpan = kRankGroup * GS_BLOCK;
#pragma unroll 1
    for (uint32_t g = 0; g < m; g += kGroupSpan) {
        unsigned long long kk[kRankGroup];
        uint32_t pk[kRankGroup], rk[kRankGroup];
#pragma unroll
        for (int k = 0; k < kRankGroup; ++k) {
            const uint32_t i = min(g + threadIdx.x + k * GS_BLOCK, m - 1u);
            kk[k] = skey[start + r0 + i];
            pk[k] = sval[start + r0 + i];
        }
        rank_in<kRankGroup>(sk, mo, kk, rk);
#pragma unroll
        for (int k = 0; k < kRankGroup; ++k) {
            const uint32_t i = g + threadIdx.x + k * GS_BLOCK;
            if (i < m) put_sorted(t, start + r_out + i + rk[k], kk[k], pk[k], pair_emit, vals, keys64);
        }
    }
}

__device__ void sort_two_runs(uint32_t t, uint32_t start, uint32_t n, unsigned long long* __restrict__ skey,
                              uint32_t* __restrict__ sval, unsigned long long* sk, uint32_t* sv,
                              uint32_t* __restrict__ pair_emit, uint32_t* __restrict__ vals,
                              uint64_t* __restrict__ keys64) {
    const uint32_t tid = threadIdx.x;
    const uint32_t na = kLongCap, nb = n - kLongCap;
    // the first run sorted, to its place
    block_sort_lds64(start, na, skey, sval, sk, sv);
    for (uint32_t i = tid; i < na; i += GS_BLOCK) {
        skey[start + i] = sk[i];
        sval[start + i] = sv[i];
    }
    __threadfence_block();
    __syncthreads();
    // the second run sorted (in LDS); the first run's keys placed by their ranks in it
    block_sort_lds64(start + na, nb, skey, sval, sk, sv);
    place_ranked(t, start, 0u, na, 0u, skey, sval, sk, nb, pair_emit, vals, keys64);
    // the second run to its place, the first back to LDS; the second run's keys placed
    for (uint32_t i = tid; i < nb; i += GS_BLOCK) {
        skey[start + na + i] = sk[i];
        sval[start + na + i] = sv[i];
    }
    __threadfence_block();
    __syncthreads();
    for (uint32_t i = tid; i < na; i += GS_BLOCK) sk[i] = skey[start + i];
    __syncthreads();
    place_ranked(t, start, na, nb, 0u, skey, sval, sk, na, pair_emit, vals, keys64);
    __syncthreads();
}

// A tile by the whole workgroup, exactly: up to 2 kLongCap pairs as two runs
// in LDS, longer ones in place in global memory.
__device__ void sort_huge_tile(uint32_t t, uint32_t start, uint32_t n, unsigned long long* __restrict__ skey,
                               uint32_t* __restrict__ sval, unsigned long long* sk, uint32_t* sv,
                               uint32_t* __restrict__ pair_emit, uint32_t* __restrict__ vals,
                               uint64_t* __restrict__ keys64) {
    if (n <= 2 * kLongCap) {
        sort_two_runs(t, start, n, skey, sval, sk, sv, pair_emit, vals, keys64);
        return;
    }
    unsigned long long* key = skey + start;
    uint32_t* val = sval + start;
    bitonic_global(key, val, n);
    for (uint32_t i = threadIdx.x; i < n; i += GS_BLOCK) put_sorted(t, start + i, key[i], val[i], pair_emit, vals, keys64);
}

// One cross-wave step of a long tile: element i (register r of lane l of
// wave w, i = w * 512 + l * 8 + r) against element i ^ mask.  Key and slot
// go through LDS as one word pair, r-major (address r * 256 + i / 8), so the
// lanes of one access touch consecutive words.
__device__ __forceinline__ void long_exchange(uint32_t (&v)[kLongK], uint32_t (&p)[kLongK], bool act, uint32_t ibase,
                                              uint32_t mask, unsigned long long* s_kv) {
    constexpr uint32_t kStride = kLongCap / kLongK;
    const uint32_t hb = 1u << (31 - __clz(mask));          // the highest bit of mask decides the side
    if (act) {
#pragma unroll
        for (int r = 0; r < kLongK; ++r) s_kv[r * kStride + (ibase >> 3)] = ((unsigned long long)p[r] << 32) | v[r];
    }
    __syncthreads();
    if (act) {
        const bool lower = (ibase & hb) == 0;              // hb >= 512 > r: one side for all r
#pragma unroll
        for (int r = 0; r < kLongK; ++r) {
            const uint32_t q = (ibase + r) ^ mask;
            const unsigned long long kv = s_kv[(q & 7u) * kStride + (q >> 3)];
            keep32(v[r], p[r], (uint32_t)kv, (uint32_t)(kv >> 32), lower);
        }
    }
    __syncthreads();
}

// A long tile (n in [kWaveSortMax, kLongCap]) by the whole workgroup.
__device__ void sort_long_tile(uint32_t t, uint32_t start, uint32_t n, unsigned long long* __restrict__ skey,
                               uint32_t* __restrict__ sval, unsigned long long* s_kv, uint32_t* s_v,
                               uint32_t* s_first, uint32_t* __restrict__ pair_emit, uint32_t* __restrict__ vals,
                               uint64_t* __restrict__ keys64) {
    const uint32_t w = threadIdx.x / GS_WAVE, lane = lane_id();
    uint32_t np = kWaveSortMax;
    while (np < n) np <<= 1;
    const bool act = w < np / kWaveSortMax;
    const uint32_t ibase = w * kWaveSortMax + lane * kLongK;
    uint32_t v[kLongK], p[kLongK];
    bool odd = false;
#pragma unroll
    for (int r = 0; r < kLongK; ++r) {
        const uint32_t i = ibase + r;
        v[r] = act && i < n ? key_depth(skey, start + i) : kDepthPad;
        p[r] = i;
        odd |= act && i < n && v[r] == kDepthPad;
    }
    if (__syncthreads_or(odd)) {
        block_sort_tile64(t, start, n, skey, sval, s_kv, s_v, pair_emit, vals, keys64);
        return;
    }
    if (act) net32<kLongK, (int)kWaveSortMax>(v, p, lane);
    for (uint32_t kk = 2 * kWaveSortMax; kk <= np; kk <<= 1) {
        long_exchange(v, p, act, ibase, kk - 1, s_kv);
        for (uint32_t j = kk >> 2; j >= kWaveSortMax; j >>= 1) long_exchange(v, p, act, ibase, j, s_kv);
        if (act) tail32<kLongK, (int)kWaveSortMax / 2>(v, p, lane);
    }
    // equal neighbours: inside a lane, to the next lane, to the next wave
    if (act && lane == 0) s_first[w] = v[0];
    __syncthreads();
    bool tie = false;
    if (act) {
#pragma unroll
        for (int r = 0; r + 1 < kLongK; ++r) tie |= ibase + r + 1 < n && v[r] == v[r + 1];
        const uint32_t next = __shfl_down(v[0], 1, GS_WAVE);
        if (lane + 1 < GS_WAVE)
            tie |= ibase + kLongK < n && v[kLongK - 1] == next;
        else if (w + 1 < np / kWaveSortMax)
            tie |= ibase + kLongK < n && v[kLongK - 1] == s_first[w + 1];
    }
    if (!__syncthreads_or(tie)) {
        if (act) {
#pragma unroll
            for (int r = 0; r < kLongK; ++r)
                if (ibase + r < n) put_by_slot(t, start, ibase + r, v[r], p[r], skey, sval, pair_emit, vals, keys64);
        }
        return;
    }
    // equal depth bits: the sorted keys to LDS, then each run placed by emission position
    if (act) {
#pragma unroll
        for (int r = 0; r < kLongK; ++r) {
            const uint32_t i = ibase + r;
            if (i < n) {
                s_kv[i] = ((unsigned long long)v[r] << 32) | key_emit(skey, start + p[r]);
                s_v[i] = sval[start + p[r]];
            }
        }
    }
    __syncthreads();
    if (__syncthreads_or(long_run(s_kv, n, threadIdx.x, GS_BLOCK))) {
        block_sort_tile64(t, start, n, skey, sval, s_kv, s_v, pair_emit, vals, keys64);
        return;
    }
    place_runs(t, start, n, s_kv, s_v, threadIdx.x, GS_BLOCK, pair_emit, vals, keys64);
    __syncthreads();
}

// Per-tile depth sort, a persistent grid over the dispatch records.  The
// first n_long records (kWaveSortMax pairs or more) go to whole workgroups,
// records b, b + G, .. to workgroup b; then every wave takes the remaining
// records from the shortest up, records T-1-s for s = 4b + w, 4b + w + 4G, ..
// Output: the tiles' pairs ordered by (depth bits, emission position), with
// the primitive ids, the sorted -> emission map and the optional 64-bit keys.
__global__ void __launch_bounds__(GS_BLOCK) k_tile_depth_sort(const uint4* __restrict__ rec,
                                                              const uint32_t* __restrict__ n_long_ptr, uint32_t T,
                                                              unsigned long long* __restrict__ skey,
                                                              uint32_t* __restrict__ sval,
                                                              uint32_t* __restrict__ pair_emit,
                                                              uint32_t* __restrict__ vals,
                                                              uint64_t* __restrict__ keys64) {
    __shared__ unsigned long long s_kv[kLongCap];      // long tiles; a 512-entry quarter per wave otherwise
    __shared__ uint32_t s_v[kLongCap];
    __shared__ uint32_t s_first[kSortWaves];
    const uint32_t G = gridDim.x;                             // <= T
    const uint32_t w = threadIdx.x / GS_WAVE;
    const uint32_t s0 = blockIdx.x * kSortWaves + w;
    // the first records of the block and of the wave load beside the count
    uint4 rl = rec[blockIdx.x];
    uint4 rs = rec[T - 1u - min(s0, T - 1u)];
    const uint32_t n_long = *n_long_ptr;
    for (uint32_t pos = blockIdx.x; pos < n_long; pos += G) {
        if (pos != blockIdx.x) rl = rec[pos];
        if (rl.z <= kLongCap)
            sort_long_tile(rl.x, rl.y, rl.z, skey, sval, s_kv, s_v, s_first, pair_emit, vals, keys64);
        else
            sort_huge_tile(rl.x, rl.y, rl.z, skey, sval, s_kv, s_v, pair_emit, vals, keys64);
    }
    unsigned long long* sk = s_kv + w * kWaveSortMax;
    uint32_t* sv = s_v + w * kWaveSortMax;
    for (uint32_t s = s0; s < T - n_long; s += kSortWaves * G) {
        if (s != s0) rs = rec[T - 1u - s];
        const uint32_t t = rs.x, start = rs.y, n = rs.z;
        if (n == 0u || n >= kWaveSortMax) continue;     // (the order puts every longer tile first)
        if (n <= 64u)
            wave_sort_tile<1>(t, start, n, skey, sval, sk, sv, pair_emit, vals, keys64);
        else if (n <= 128u)
            wave_sort_tile<2>(t, start, n, skey, sval, sk, sv, pair_emit, vals, keys64);
        else if (n <= 256u)
            wave_sort_tile<4>(t, start, n, skey, sval, sk, sv, pair_emit, vals, keys64);
        else
            wave_sort_tile<8>(t, start, n, skey, sval, sk, sv, pair_emit, vals, keys64);
    }
}

struct BinsortLayout {
    size_t pkeys, emit_id;    // per emission position: tile and primitive of the pair
    size_t pdepth;            // per emission position: the primitive's depth bits
    size_t skey, sval;        // per sorted position: the 64-bit depth-sort key and its primitive
    size_t order;             // the dispatch order when the caller keeps none
    size_t rec;               // per dispatch position: tile, range start, pair count
    size_t tcount, cursor;    // per tile: pair total, placement cursor
    size_t bsum, offs, bstart, counters;
    size_t bytes;
};

uint32_t tile_count(int32_t width, int32_t height) {
    const int64_t TX = (width + GS_TILE - 1) / GS_TILE, TY = (height + GS_TILE - 1) / GS_TILE;
    return (uint32_t)(TX * TY);
}

BinsortLayout binsort_layout(int32_t n, uint32_t capacity, int32_t width, int32_t height) {
    BinsortLayout L;
    size_t o = 0;
    const size_t nn = (size_t)(n > 0 ? n : 1), cc = (size_t)(capacity > 0 ? capacity : 1);
    const size_t tt = (size_t)(width > 0 && height > 0 ? tile_count(width, height) : 1u);
    L.pkeys = o; o += align256(4 * cc);
    L.emit_id = o; o += align256(4 * cc);
    L.pdepth = o; o += align256(4 * cc);
    L.skey = o; o += align256(8 * cc);
    L.sval = o; o += align256(4 * cc);
    L.order = o; o += align256(4 * tt);
    L.rec = o; o += align256(16 * tt);
    L.tcount = o; o += align256(4 * tt);
    L.cursor = o; o += align256(4 * tt);
    L.bsum = o; o += align256(4 * ((size_t)div_up(nn, GS_TILE_ITEMS) + 1));
    L.offs = o; o += align256(4 * (nn + 1));
    L.bstart = o; o += align256(4 * ((size_t)div_up(cc, GS_TILE_ITEMS) + 1));
    L.counters = o; o += 256;
    L.bytes = o;
    return L;
}

template <typename T>
T* at(void* ws, size_t off) { return reinterpret_cast<T*>(static_cast<char*>(ws) + off); }

}  // namespace

size_t binsort_ws_bytes(int32_t n, uint32_t capacity, int32_t width, int32_t height) {
    return binsort_layout(n, capacity, width, height).bytes;
}

hipError_t launch_binsort(const gs_proj& proj, int32_t n, const uint32_t* vis_idx, const uint32_t* vis_count,
                          int32_t width, int32_t height, uint32_t capacity, uint32_t* vals, uint32_t* ranges,
                          uint32_t* tile_order, uint32_t* pair_offset, uint32_t* pair_emit, uint64_t* keys,
                          uint32_t* num_pairs, gs_device_status* status, void* ws, hipStream_t st) {
    const BinsortLayout L = binsort_layout(n, capacity, width, height);
    const int32_t TX = (width + GS_TILE - 1) / GS_TILE;
    const uint32_t T = tile_count(width, height);
    uint32_t* bsum = at<uint32_t>(ws, L.bsum);
    uint32_t* ctr = at<uint32_t>(ws, L.counters);   // [1] sort count, [2] long tiles
    uint32_t* tcount = at<uint32_t>(ws, L.tcount);
    uint32_t* cursor = at<uint32_t>(ws, L.cursor);
    uint32_t* order = tile_order ? tile_order : at<uint32_t>(ws, L.order);
    // ranges, cursors and the dispatch order from the per-tile totals
    auto finish = [&]() {
        hipLaunchKernelGGL(k_tile_finish, dim3(div_up(T, kFinishSeg)), dim3(GS_BLOCK), 0, st, tcount, T, ranges,
                           cursor, order, at<uint4>(ws, L.rec), ctr + 2);
        return hipGetLastError();
    };
    // no pairs: empty ranges, and the order (then the tile ids)
    auto no_pairs = [&]() {
        if (T == 0) return hipGetLastError();
        hipError_t e = launch_fill_u32(tcount, 0u, T, st);
        if (e != hipSuccess) return e;
        return finish();
    };
    if (n == 0) {
        hipError_t e = launch_fill_u32(num_pairs, 0u, 1, st);
        if (e != hipSuccess) return e;
        return no_pairs();
    }
    // 1. emission offsets in visible-set order
    const uint32_t* vorder = vis_idx;
    const uint32_t nb = div_up(n, GS_TILE_ITEMS);
    hipLaunchKernelGGL(k_tile_sums, dim3(nb), dim3(GS_BLOCK), 0, st, vorder, vis_count, proj.tiles, bsum, tcount, T);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    uint32_t* offs_r = at<uint32_t>(ws, L.offs);
    const uint32_t nbs = div_up(capacity, GS_TILE_ITEMS) + 1u;
    hipLaunchKernelGGL(k_offsets, dim3(nb), dim3(GS_BLOCK), 0, st, vorder, vis_count, proj.tiles, bsum, capacity, pair_offset, offs_r, ctr + 1, num_pairs, status, at<uint32_t>(ws, L.bstart), nbs);
    if (capacity == 0 || T == 0) return no_pairs();
    // 2. emission: one (tile, primitive) pair per touched tile, and the per-tile totals
    const uint32_t nbp = div_up(capacity, GS_TILE_ITEMS);
    hipLaunchKernelGGL(k_emit_pairs, dim3(nbp), dim3(GS_BLOCK), 0, st, vorder, vis_count, offs_r,
                       at<uint32_t>(ws, L.bstart), reinterpret_cast<const ushort4*>(proj.rect), proj.depth, ctr + 1,
                       TX, T, at<uint32_t>(ws, L.pkeys), at<uint32_t>(ws, L.emit_id), at<uint32_t>(ws, L.pdepth),
                       tcount);
    // 3. tile ranges and the dispatch order
    e = finish();
    if (e != hipSuccess) return e;
    // 4. every pair's depth-sort key placed in its tile's range
    unsigned long long* skey = at<unsigned long long>(ws, L.skey);
    uint32_t* sval = at<uint32_t>(ws, L.sval);
    hipLaunchKernelGGL(k_tile_scatter, dim3(nbp), dim3(GS_BLOCK), 0, st, at<uint32_t>(ws, L.pkeys),
                       at<uint32_t>(ws, L.emit_id), at<uint32_t>(ws, L.pdepth), ctr + 1, T, cursor, skey, sval);
    // 5. per tile, longest first: depth order, primitive ids (+ optional 64-bit keys)
    const uint32_t cus = compute_units();
    const uint32_t grid = std::min<uint32_t>(T, (cus ? cus : 256u) * kDepthSortBlocksPerCU);
    hipLaunchKernelGGL(k_tile_depth_sort, dim3(grid), dim3(GS_BLOCK), 0, st, at<uint4>(ws, L.rec), ctr + 2, T, skey,
                       sval, pair_emit, vals, keys);
    return hipGetLastError();
}

}  // namespace gsmi
