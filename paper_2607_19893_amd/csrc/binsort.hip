// Rendering phase, part 1: duplicate visible primitives per touched tile and
// order the pairs by (tile, depth, primitive id).
//
// Instead of one wide radix sort over 64-bit (tile, depth) keys:
//   1. every visible primitive's tile pairs are emitted in visible-set order
//      (ascending ids), each primitive's rectangle row-major, so a primitive's
//      pairs are contiguous ("emission order");
//   2. the M pairs are sorted by tile id only (ceil(log2 T) bits: 1-2 LSD
//      passes), carrying each pair's emission position;
//   3. the tile ranges come from the segment bounds of the sorted keys, and
//      one stable 8-bit radix pass over a code of each tile's pair count gives
//      the dispatch order: the longest tiles first;
//   4. each tile's segment is sorted by (depth bits, emission position) in LDS
//      by one workgroup (a bitonic network; segments longer than the LDS
//      capacity are sorted in global memory by the same workgroup), tiles
//      taken in the dispatch order.  Emission positions grow with the
//      primitive id inside a tile, so this is exactly the (tile, depth bits,
//      id) order.
// Step 4 replaces a 4-pass radix sort of the visible set by depth (12
// latency-bound launches) with one launch whose work is local to a tile.
// The per-tile kernels that follow (this sort, the forward and backward
// raster) end when their longest tile ends; taking the longest first lets
// the short ones fill in beside it instead of after it.
//
// Each LSD pass is three launches: per-block digit histograms (digit-major
// matrix), a per-digit scan across blocks, and a scatter whose in-block rank
// comes from a 64-lane match built from ballots; every wave of a block owns a
// contiguous quarter of the block's keys, so the order is stable.
#include "common.h"
#include "internal.h"

namespace gsmi {

namespace {

// Digit widths (8 bits: wider digits cost more per pass in these small,
// latency-bound launches than the pass they save).  Every kernel takes the
// digit width as a template parameter; a block holds 2^BITS counters in LDS.
constexpr int kTileBits = 8;
// Up to this many 2048-item blocks (32768 tiles: a 4K image has 32400)
// the tile-order scatter sums its digit offsets itself instead of a scan launch.
constexpr uint32_t kSelfScanBlocks = 16;

template <int BITS>
__global__ void __launch_bounds__(GS_BLOCK) k_radix_hist(const uint32_t* __restrict__ keys,
                                                         const uint32_t* __restrict__ count_ptr, int shift,
                                                         uint32_t mask, uint32_t* __restrict__ hist,
                                                         uint32_t nblocks) {
    constexpr int R = 1 << BITS;
    __shared__ uint32_t h[R];
    for (int d = threadIdx.x; d < R; d += GS_BLOCK) h[d] = 0;
    __syncthreads();
    const uint32_t cnt = *count_ptr;
    const uint32_t base = blockIdx.x * GS_TILE_ITEMS;
    if (base < cnt) {
#pragma unroll
        for (int k = 0; k < GS_ITEMS; ++k) {
            const uint32_t i = base + k * GS_BLOCK + threadIdx.x;
            if (i < cnt) atomicAdd(&h[(keys[i] >> shift) & mask], 1u);
        }
    }
    __syncthreads();
    for (int d = threadIdx.x; d < R; d += GS_BLOCK) hist[(size_t)d * nblocks + blockIdx.x] = h[d];
}

// One workgroup per digit row: exclusive scan across blocks, row total -> totals[d].
__global__ void __launch_bounds__(GS_BLOCK) k_radix_scan(uint32_t* __restrict__ hist, uint32_t nblocks,
                                                         uint32_t* __restrict__ totals) {
    __shared__ uint32_t scratch[4];
    uint32_t* row = hist + (size_t)blockIdx.x * nblocks;
    uint32_t carry = 0;
    for (uint32_t chunk = 0; chunk < nblocks; chunk += GS_TILE_ITEMS) {
        const uint32_t base = chunk + threadIdx.x * GS_ITEMS;
        uint32_t v[GS_ITEMS];
        uint32_t s = 0;
#pragma unroll
        for (int k = 0; k < GS_ITEMS; ++k) {
            v[k] = (base + k < nblocks) ? row[base + k] : 0u;
            s += v[k];
        }
        uint32_t tot;
        uint32_t run = block_excl_scan(s, scratch, &tot) + carry;
#pragma unroll
        for (int k = 0; k < GS_ITEMS; ++k) {
            if (base + k < nblocks) row[base + k] = run;
            run += v[k];
        }
        carry += tot;
    }
    if (threadIdx.x == 0) totals[blockIdx.x] = carry;
}

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

// Stable scatter of block b's 2048 keys.  With SELF_SCAN the histogram
// matrix is the unscanned per-block counts and each block sums its digit
// offsets from it (for a few blocks: saves the scan launch).  Wave w ranks its own 512 keys
// (contiguous, 64 per round) against a wave-private running count per digit,
// so the rounds need no block barrier; one barrier then turns the four
// waves' digit counts into per-wave offsets.  Position of a key = start of
// its digit over all blocks + its block's offset (from the scanned matrix) +
// the keys of earlier waves with that digit + its rank inside its wave.
template <int BITS, bool SELF_SCAN = false>
__global__ void __launch_bounds__(GS_BLOCK) k_radix_scatter(
    const uint32_t* __restrict__ keys_in, const uint32_t* __restrict__ vals_in, uint32_t* __restrict__ keys_out,
    uint32_t* __restrict__ vals_out, const uint32_t* __restrict__ count_ptr, int shift, uint32_t mask,
    int nbits, const uint32_t* __restrict__ hist, const uint32_t* __restrict__ totals, uint32_t nblocks) {
    constexpr int R = 1 << BITS;
    constexpr int PER = (R + GS_BLOCK - 1) / GS_BLOCK;    // digits per thread in the per-digit steps
    __shared__ uint32_t s_base[R];
    __shared__ uint32_t s_wc[4][R];
    __shared__ uint32_t scratch[4];
    const uint32_t cnt = *count_ptr;
    if (blockIdx.x * GS_TILE_ITEMS >= cnt) return;
    const int tid = threadIdx.x;
    const int w = tid / GS_WAVE;
    const int lane = lane_id();
    // digit starts: exclusive scan of the digit totals, thread t owning digits [t*PER, t*PER+PER)
    {
        uint32_t tv[PER], bq[PER];
        uint32_t sum = 0;
#pragma unroll
        for (int q = 0; q < PER; ++q) {
            const int d = tid * PER + q;
            if (SELF_SCAN) {
                uint32_t before = 0, all = 0;
                if (d < R)
                    for (uint32_t j = 0; j < nblocks; ++j) {
                        const uint32_t c = hist[(size_t)d * nblocks + j];
                        before += j < blockIdx.x ? c : 0u;
                        all += c;
                    }
                tv[q] = all;
                bq[q] = before;
            } else {
                tv[q] = d < R ? totals[d] : 0u;
            }
            sum += tv[q];
        }
        uint32_t tot;
        uint32_t run = block_excl_scan(sum, scratch, &tot);
#pragma unroll
        for (int q = 0; q < PER; ++q) {
            const int d = tid * PER + q;
            if (d < R) {
                s_base[d] = run + (SELF_SCAN ? bq[q] : hist[(size_t)d * nblocks + blockIdx.x]);
                s_wc[0][d] = 0; s_wc[1][d] = 0; s_wc[2][d] = 0; s_wc[3][d] = 0;
            }
            run += tv[q];
        }
    }
    const uint32_t base = blockIdx.x * GS_TILE_ITEMS + w * (GS_WAVE * GS_ITEMS);
    uint32_t key[GS_ITEMS], val[GS_ITEMS], rk[GS_ITEMS];
#pragma unroll
    for (int k = 0; k < GS_ITEMS; ++k) {
        const uint32_t i = base + k * GS_WAVE + lane;
        key[k] = (i < cnt) ? keys_in[i] : 0u;
        val[k] = (i < cnt) ? (vals_in ? vals_in[i] : i) : 0u;    // no input values: the input position
    }
    __syncthreads();
    const uint64_t lt = lanemask_lt();
    uint32_t* wc = s_wc[w];
#pragma unroll
    for (int k = 0; k < GS_ITEMS; ++k) {
        const uint32_t i = base + k * GS_WAVE + lane;
        const bool valid = i < cnt;
        const uint32_t d = (key[k] >> shift) & mask;
        const uint64_t peers = match_digit(d, valid, nbits);
        const uint32_t before = valid ? wc[d] : 0u;
        rk[k] = before + (uint32_t)popc64(peers & lt);
        // all reads of this round precede the leaders' updates
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        if (valid && (peers & lt) == 0ull) wc[d] = before + (uint32_t)popc64(peers);
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
    __syncthreads();
    // per digit: offsets of waves 1..3 folded into s_wc (wave 0 takes 0)
#pragma unroll
    for (int q = 0; q < PER; ++q) {
        const int d = tid * PER + q;
        if (d < R) {
            const uint32_t c0 = s_wc[0][d], c1 = s_wc[1][d], c2 = s_wc[2][d];
            s_wc[0][d] = 0;
            s_wc[1][d] = c0;
            s_wc[2][d] = c0 + c1;
            s_wc[3][d] = c0 + c1 + c2;
        }
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < GS_ITEMS; ++k) {
        const uint32_t i = base + k * GS_WAVE + lane;
        if (i < cnt) {
            const uint32_t d = (key[k] >> shift) & mask;
            const uint32_t pos = s_base[d] + wc[d] + rk[k];
            keys_out[pos] = key[k];
            vals_out[pos] = val[k];
        }
    }
}

// per-block sums of tiles[] in visible-set order
// The grid also zeroes the tile ranges (n_ranges words) for the segment
// bounds written later.
__global__ void __launch_bounds__(GS_BLOCK) k_tile_sums(const uint32_t* __restrict__ order,
                                                        const uint32_t* __restrict__ vis_count,
                                                        const uint32_t* __restrict__ tiles,
                                                        uint32_t* __restrict__ bsum, uint32_t* __restrict__ ranges,
                                                        uint32_t n_ranges) {
    __shared__ uint32_t scratch[4];
    for (uint32_t i = blockIdx.x * GS_BLOCK + threadIdx.x; i < n_ranges; i += gridDim.x * GS_BLOCK) ranges[i] = 0u;
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
// with offs_r[V] = M as a sentinel.  Also publishes the pair count and the
// overflow flag, and for every 2048-pair emission block m the rank that holds
// its first pair (bstart[m], m < nbs): the rank whose pairs [off, off + t)
// contain m * 2048 writes it, so each entry has one writer.  On overflow
// (M > capacity) no pair is emitted and pair_offset[id] = 0xFFFFFFFF, so the
// per-primitive backward finds none of its slots in the buffer.
__global__ void __launch_bounds__(GS_BLOCK) k_offsets(
    const uint32_t* __restrict__ order, const uint32_t* __restrict__ vis_count, const uint32_t* __restrict__ tiles,
    const uint32_t* __restrict__ bsum, const uint32_t* __restrict__ total, uint32_t capacity,
    uint32_t* __restrict__ pair_offset, uint32_t* __restrict__ offs_r, uint32_t* __restrict__ sort_count,
    uint32_t* __restrict__ num_pairs, gs_device_status* __restrict__ status, uint32_t* __restrict__ bstart,
    uint32_t nbs) {
    __shared__ uint32_t scratch[4];
    const uint32_t V = *vis_count;
    const uint32_t M = *total;
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
    uint32_t off = block_excl_scan(s, scratch, &tot) + bsum[blockIdx.x];
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
template <bool STAGED>
__device__ __forceinline__ void emit_block_pairs(uint32_t base, uint32_t hi, uint32_t nr, const uint32_t* s_off,
                                                 const uint32_t* s_gid, const ushort4* s_rect,
                                                 const uint32_t* __restrict__ g_off,
                                                 const uint32_t* __restrict__ g_order,
                                                 const ushort4* __restrict__ rect, int32_t tiles_x,
                                                 uint32_t* __restrict__ pkeys, uint32_t* __restrict__ pvals,
                                                 uint32_t mask0, uint32_t* h) {
#pragma unroll
    for (int k = 0; k < GS_ITEMS; ++k) {
        const uint32_t i = base + k * GS_BLOCK + threadIdx.x;
        if (i >= hi) break;
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
        const uint32_t key = ty * (uint32_t)tiles_x + tx;
        pkeys[i] = key;
        pvals[i] = gid;
        atomicAdd(&h[key & mask0], 1u);
    }
}

// One thread per pair: pair i belongs to the rank r with offs_r[r] <= i <
// offs_r[r+1] and covers tile number i - offs_r[r] of that primitive's
// rectangle (row-major).  Each block locates its rank range once, stages the
// offsets, ids and rectangles of those ranks in LDS and binary-searches
// there; key (tile id) and value (primitive id) stores are contiguous.  Each
// block also writes its histogram of the tile sort's first digit (key & mask0)
// as column b of the digit-major matrix (zeros past the last pair).
__global__ void __launch_bounds__(GS_BLOCK) k_emit_pairs(
    const uint32_t* __restrict__ order, const uint32_t* __restrict__ vis_count, const uint32_t* __restrict__ offs_r,
    const uint32_t* __restrict__ bstart, const ushort4* __restrict__ rect, const uint32_t* __restrict__ sort_count,
    int32_t tiles_x, uint32_t* __restrict__ pkeys, uint32_t* __restrict__ pvals, uint32_t mask0,
    uint32_t* __restrict__ hist, uint32_t nblocks) {
    __shared__ uint32_t s_off[GS_TILE_ITEMS + 1];
    __shared__ uint32_t s_gid[GS_TILE_ITEMS + 1];
    __shared__ ushort4 s_rect[GS_TILE_ITEMS + 1];
    __shared__ uint32_t s_range[2];
    __shared__ uint32_t h[1 << kTileBits];
    for (int d = threadIdx.x; d < (1 << kTileBits); d += GS_BLOCK) h[d] = 0;
    const uint32_t M = *sort_count;
    const uint32_t base = blockIdx.x * GS_TILE_ITEMS;
    if (base >= M) {
        for (int d = threadIdx.x; d < (1 << kTileBits); d += GS_BLOCK) hist[(size_t)d * nblocks + blockIdx.x] = 0u;
        return;
    }
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
    const bool staged = nr <= GS_TILE_ITEMS + 1;
    if (staged) {
        for (uint32_t j = threadIdx.x; j < nr; j += GS_BLOCK) {
            const uint32_t g = order[r0 + j];
            s_off[j] = offs_r[r0 + j];
            s_gid[j] = g;
            s_rect[j] = rect[g];
        }
    }
    __syncthreads();
    if (staged)
        emit_block_pairs<true>(base, hi, nr, s_off, s_gid, s_rect, offs_r + r0, order + r0, rect, tiles_x, pkeys,
                               pvals, mask0, h);
    else
        emit_block_pairs<false>(base, hi, nr, s_off, s_gid, s_rect, offs_r + r0, order + r0, rect, tiles_x, pkeys,
                                pvals, mask0, h);
    __syncthreads();
    for (int d = threadIdx.x; d < (1 << kTileBits); d += GS_BLOCK) hist[(size_t)d * nblocks + blockIdx.x] = h[d];
}

// Per-tile ordering: LDS capacity in pairs (8 per thread) and the largest key.
constexpr int kSortCap = GS_TILE_ITEMS;
constexpr unsigned long long kKeyMax = ~0ull;

// Dispatch key of a tile from its pair count: an 8-bit code that never
// decreases with the count (exact below 16, then 16 steps per octave; counts
// of 2^19 and more share the top code), inverted so that an ascending radix
// pass puts the longest tiles first.
__device__ __forceinline__ uint32_t tile_order_key(uint32_t n) {
    uint32_t code = n;
    if (n >= 16u) {
        const uint32_t e = 31u - (uint32_t)__clz(n);      // >= 4
        code = e > 18u ? 255u : 16u * (e - 3u) + ((n >> (e - 4u)) & 15u);
    }
    return 255u - code;
}

// Segment bounds of the M tile-sorted pair keys: the pair that opens tile
// t's segment writes ranges[2t], the pair that closes it ranges[2t+1]; tiles
// without pairs keep the zeros written before.  Thread i of block b looks at
// pairs b*2048 + k*256 + i and their neighbours.
__global__ void __launch_bounds__(GS_BLOCK) k_tile_bounds(const uint32_t* __restrict__ skeys,
                                                          const uint32_t* __restrict__ sort_count,
                                                          uint32_t* __restrict__ ranges) {
    const uint32_t M = *sort_count;
    const uint32_t base = blockIdx.x * GS_TILE_ITEMS + threadIdx.x;
    if (blockIdx.x * GS_TILE_ITEMS >= M) return;
#pragma unroll
    for (int k = 0; k < GS_ITEMS; ++k) {
        const uint32_t i = base + k * GS_BLOCK;
        if (i < M) {
            const uint32_t t = skeys[i];
            if (i == 0 || skeys[i - 1] != t) ranges[2 * t] = i;
            if (i + 1 == M || skeys[i + 1] != t) ranges[2 * t + 1] = i + 1;
        }
    }
}

// Every tile's dispatch key from its range; block b covers tiles
// [b*2048, b*2048+2048) and leaves its per-digit key counts in column b of the
// digit-major histogram matrix that the radix scan reads.
__global__ void __launch_bounds__(GS_BLOCK) k_tile_keys(const uint32_t* __restrict__ ranges, uint32_t T,
                                                        uint32_t* __restrict__ tkeys, uint32_t* __restrict__ hist,
                                                        uint32_t nblocks, uint32_t* __restrict__ tile_count) {
    static_assert(GS_BLOCK == 256, "one digit counter per thread");
    __shared__ uint32_t h[256];
    const uint32_t tid = threadIdx.x;
    h[tid] = 0;
    if (blockIdx.x == 0 && tid == 0) *tile_count = T;
    __syncthreads();
#pragma unroll
    for (int k = 0; k < GS_ITEMS; ++k) {
        const uint32_t t = blockIdx.x * GS_TILE_ITEMS + k * GS_BLOCK + tid;
        if (t < T) {
            const uint32_t key = tile_order_key(ranges[2 * t + 1] - ranges[2 * t]);
            tkeys[t] = key;
            atomicAdd(&h[key], 1u);
        }
    }
    __syncthreads();
    hist[(size_t)tid * nblocks + blockIdx.x] = h[tid];
}

// Bitonic network over s[0..np) (np a power of two, entries past the data
// hold kKeyMax), in the variant whose compare-exchanges all put the smaller
// key at the lower index: each merge of width k first compares i with its
// mirror i ^ (k - 1), then i with i ^ j for j = k/4 .. 1.
__device__ __forceinline__ void bitonic_lds(unsigned long long* s, uint32_t np) {
    for (uint32_t k = 2; k <= np; k <<= 1) {
        for (uint32_t j = k >> 1; j > 0; j >>= 1) {
            const uint32_t mask = (j == (k >> 1)) ? (k - 1) : j;
            for (uint32_t c = threadIdx.x; c < (np >> 1); c += GS_BLOCK) {
                // c-th compare-exchange: lower index i has bit log2(j) clear
                const uint32_t i = ((c & ~(j - 1)) << 1) | (c & (j - 1));
                const uint32_t q = i ^ mask;
                const unsigned long long a = s[i], b = s[q];
                if (b < a) {
                    s[i] = b;
                    s[q] = a;
                }
            }
            __syncthreads();
        }
    }
}

// The same network on a segment of global memory of any length n: entries
// at n and beyond are taken as kKeyMax, so a compare-exchange that reaches
// past the data leaves the lower (real) entry in place.
__device__ void bitonic_global(unsigned long long* s, uint32_t n) {
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
                    s[i] = b;
                    s[q] = a;
                }
            }
            __threadfence_block();
            __syncthreads();
        }
    }
}

// One workgroup per tile, tiles taken in dispatch order (longest first):
// order the tile's segment of the tile-sorted pairs by (depth bits, emission
// position) and write the primitive ids, the sorted -> emission map and the
// optional 64-bit keys.  pair_emit holds the segment's emission positions on
// entry (any order).
__global__ void __launch_bounds__(GS_BLOCK) k_tile_depth_sort(const uint32_t* __restrict__ tile_order,
                                                              const uint32_t* __restrict__ ranges,
                                                              const uint32_t* __restrict__ emit_id,
                                                              const float* __restrict__ depth,
                                                              uint32_t* __restrict__ pair_emit,
                                                              uint32_t* __restrict__ vals,
                                                              uint64_t* __restrict__ keys64,
                                                              unsigned long long* __restrict__ scratch) {
    __shared__ unsigned long long s_key[kSortCap];
    const uint32_t t = tile_order[blockIdx.x];
    const uint32_t start = ranges[2 * t], end = ranges[2 * t + 1];
    const uint32_t n = end - start;
    if (n == 0) return;
    unsigned long long* key = s_key;
    if (n <= (uint32_t)kSortCap) {
        uint32_t np = 2;
        while (np < n) np <<= 1;
        for (uint32_t i = threadIdx.x; i < np; i += GS_BLOCK) {
            unsigned long long k = kKeyMax;
            if (i < n) {
                const uint32_t e = pair_emit[start + i];
                k = ((unsigned long long)__float_as_uint(depth[emit_id[e]]) << 32) | e;
            }
            s_key[i] = k;
        }
        __syncthreads();
        bitonic_lds(s_key, np);
    } else {
        key = scratch + start;
        for (uint32_t i = threadIdx.x; i < n; i += GS_BLOCK) {
            const uint32_t e = pair_emit[start + i];
            key[i] = ((unsigned long long)__float_as_uint(depth[emit_id[e]]) << 32) | e;
        }
        __threadfence_block();
        __syncthreads();
        bitonic_global(key, n);
    }
    for (uint32_t i = threadIdx.x; i < n; i += GS_BLOCK) {
        const unsigned long long k = key[i];
        const uint32_t e = (uint32_t)k;
        vals[start + i] = emit_id[e];
        pair_emit[start + i] = e;
        if (keys64) keys64[start + i] = ((uint64_t)t << 32) | (k >> 32);
    }
}

struct BinsortLayout {
    size_t pk[3], pv[3];      // pair sort keys: in, tmp, out; pv[0] = primitive of each emitted pair,
                              // pv[1..2] = value ping-pong (values out = caller's pair_emit)
    size_t scratch;           // 64-bit keys of tiles longer than the LDS sort
    size_t tkey[2], order;    // tile dispatch keys (in, sorted) and the order when the caller keeps none
    size_t hist, totals, bsum, offs, bstart, counters;
    size_t bytes;
    uint32_t nblocks_hist;
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
    for (int i = 0; i < 3; ++i) { L.pk[i] = o; o += align256(4 * cc); }
    for (int i = 0; i < 3; ++i) { L.pv[i] = o; o += align256(4 * cc); }
    L.scratch = o; o += align256(8 * cc);
    for (int i = 0; i < 2; ++i) { L.tkey[i] = o; o += align256(4 * tt); }
    L.order = o; o += align256(4 * tt);
    size_t most = nn > cc ? nn : cc;
    most = most > tt ? most : tt;
    L.nblocks_hist = div_up(most, GS_TILE_ITEMS);
    L.hist = o; o += align256(4 * ((size_t)1 << kTileBits) * L.nblocks_hist);
    L.totals = o; o += align256(4 * ((size_t)1 << kTileBits));
    L.bsum = o; o += align256(4 * ((size_t)div_up(nn, GS_TILE_ITEMS) + 1));
    L.offs = o; o += align256(4 * (nn + 1));
    L.bstart = o; o += align256(4 * ((size_t)div_up(cc, GS_TILE_ITEMS) + 1));
    L.counters = o; o += 256;
    L.bytes = o;
    return L;
}

template <typename T>
T* at(void* ws, size_t off) { return reinterpret_cast<T*>(static_cast<char*>(ws) + off); }

// LSD passes over bits [0, total_bits) of `count` keys, BITS per pass.
// Buffers: in, tmp, out.
// vin may be null: the values are then the input positions.  Value buffers
// ping-pong between vtmp0 and vtmp1.
// The first pass's histogram matrix is already in hist (written by the
// kernel that produced the keys).
template <int BITS>
hipError_t radix_sort(uint32_t* kin, const uint32_t* vin, uint32_t* ktmp, uint32_t* vtmp0, uint32_t* vtmp1,
                      uint32_t* kout, uint32_t* vout, const uint32_t* count, uint32_t max_count, int total_bits,
                      uint32_t* hist, uint32_t* totals, hipStream_t st) {
    const uint32_t nblocks = div_up(max_count > 0 ? max_count : 1, GS_TILE_ITEMS);
    const int passes = (total_bits + BITS - 1) / BITS;
    uint32_t* kb[2] = {ktmp, kin};
    uint32_t* vb[2] = {vtmp0, vtmp1};
    for (int p = 0; p < passes; ++p) {
        const int shift = p * BITS;
        const int nbits = (total_bits - shift) < BITS ? (total_bits - shift) : BITS;
        const uint32_t mask = (1u << nbits) - 1u;
        const uint32_t* ks = (p == 0) ? kin : kb[(p - 1) & 1];
        const uint32_t* vs = (p == 0) ? vin : vb[(p - 1) & 1];
        uint32_t* kd = (p == passes - 1) ? kout : kb[p & 1];
        uint32_t* vd = (p == passes - 1) ? vout : vb[p & 1];
        if (p > 0)
            hipLaunchKernelGGL(k_radix_hist<BITS>, dim3(nblocks), dim3(GS_BLOCK), 0, st, ks, count, shift, mask, hist,
                               nblocks);
        hipLaunchKernelGGL(k_radix_scan, dim3(1u << nbits), dim3(GS_BLOCK), 0, st, hist, nblocks, totals);
        hipLaunchKernelGGL(k_radix_scatter<BITS>, dim3(nblocks), dim3(GS_BLOCK), 0, st, ks, vs, kd, vd, count, shift,
                           mask, nbits, hist, totals, nblocks);
    }
    return hipGetLastError();
}

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
    uint32_t* hist = at<uint32_t>(ws, L.hist);
    uint32_t* totals = at<uint32_t>(ws, L.totals);
    uint32_t* bsum = at<uint32_t>(ws, L.bsum);
    uint32_t* ctr = at<uint32_t>(ws, L.counters);   // [0] M, [1] sort count, [2] T
    uint32_t* order = tile_order ? tile_order : at<uint32_t>(ws, L.order);
    // ranges, dispatch keys and the dispatch order (tiles by pair count
    // descending, ties by tile id: one stable radix pass over 8-bit keys)
    // (ranges must hold zeros on entry)
    auto tile_pass = [&](const uint32_t* skeys, const uint32_t* sort_count) {
        const uint32_t nbT = div_up(T, GS_TILE_ITEMS);
        if (skeys)
            hipLaunchKernelGGL(k_tile_bounds, dim3(div_up(capacity, GS_TILE_ITEMS)), dim3(GS_BLOCK), 0, st, skeys,
                               sort_count, ranges);
        hipLaunchKernelGGL(k_tile_keys, dim3(nbT), dim3(GS_BLOCK), 0, st, ranges, T, at<uint32_t>(ws, L.tkey[0]),
                           hist, nbT, ctr + 2);
        if (nbT <= kSelfScanBlocks) {
            hipLaunchKernelGGL((k_radix_scatter<8, true>), dim3(nbT), dim3(GS_BLOCK), 0, st,
                               at<uint32_t>(ws, L.tkey[0]), nullptr, at<uint32_t>(ws, L.tkey[1]), order, ctr + 2, 0,
                               255u, 8, hist, totals, nbT);
        } else {
            hipLaunchKernelGGL(k_radix_scan, dim3(256), dim3(GS_BLOCK), 0, st, hist, nbT, totals);
            hipLaunchKernelGGL(k_radix_scatter<8>, dim3(nbT), dim3(GS_BLOCK), 0, st, at<uint32_t>(ws, L.tkey[0]),
                               nullptr, at<uint32_t>(ws, L.tkey[1]), order, ctr + 2, 0, 255u, 8, hist, totals, nbT);
        }
        return hipGetLastError();
    };
    // no pairs: empty ranges, and the order (then the tile ids) when the caller keeps it
    auto no_pairs = [&]() {
        if (T == 0) return hipGetLastError();
        hipError_t e = launch_fill_u32(ranges, 0u, 2 * (size_t)T, st);
        if (e != hipSuccess || !tile_order) return e;
        return tile_pass(nullptr, nullptr);
    };
    if (n == 0) {
        hipError_t e = launch_fill_u32(num_pairs, 0u, 1, st);
        if (e != hipSuccess) return e;
        return no_pairs();
    }
    // 1. emission offsets in visible-set order
    const uint32_t* vorder = vis_idx;
    const uint32_t nb = div_up(n, GS_TILE_ITEMS);
    hipLaunchKernelGGL(k_tile_sums, dim3(nb), dim3(GS_BLOCK), 0, st, vorder, vis_count, proj.tiles, bsum, ranges,
                       2 * T);
    hipError_t e = launch_scan_blocks(bsum, nb, ctr + 0, nullptr, st);
    if (e != hipSuccess) return e;
    uint32_t* offs_r = at<uint32_t>(ws, L.offs);
    const uint32_t nbs = div_up(capacity, GS_TILE_ITEMS) + 1u;
    hipLaunchKernelGGL(k_offsets, dim3(nb), dim3(GS_BLOCK), 0, st, vorder, vis_count, proj.tiles, bsum, ctr + 0,
                       capacity, pair_offset, offs_r, ctr + 1, num_pairs, status, at<uint32_t>(ws, L.bstart), nbs);
    int tbits = 1;
    while (tbits < 32 && (1u << tbits) < T) ++tbits;
    const uint32_t mask0 = (1u << (tbits < kTileBits ? tbits : kTileBits)) - 1u;
    if (capacity == 0 || T == 0) return no_pairs();
    // 2. emission: one (tile, primitive) pair per touched tile
    hipLaunchKernelGGL(k_emit_pairs, dim3(div_up(capacity, GS_TILE_ITEMS)), dim3(GS_BLOCK), 0, st, vorder,
                       vis_count, offs_r, at<uint32_t>(ws, L.bstart), reinterpret_cast<const ushort4*>(proj.rect),
                       ctr + 1, TX,
                       at<uint32_t>(ws, L.pk[0]), at<uint32_t>(ws, L.pv[0]), mask0, hist,
                       div_up(capacity, GS_TILE_ITEMS));
    // 3. sort of the pairs by tile id, carrying every pair's emission position
    e = radix_sort<kTileBits>(at<uint32_t>(ws, L.pk[0]), nullptr, at<uint32_t>(ws, L.pk[1]), at<uint32_t>(ws, L.pv[1]),
                              at<uint32_t>(ws, L.pv[2]), at<uint32_t>(ws, L.pk[2]), pair_emit, ctr + 1, capacity,
                              tbits, hist, totals, st);
    if (e != hipSuccess) return e;
    // 4. tile ranges and the dispatch order
    e = tile_pass(at<uint32_t>(ws, L.pk[2]), ctr + 1);
    if (e != hipSuccess) return e;
    // 5. per tile, longest first: depth order, primitive ids (+ optional 64-bit keys)
    hipLaunchKernelGGL(k_tile_depth_sort, dim3(T), dim3(GS_BLOCK), 0, st, order, ranges, at<uint32_t>(ws, L.pv[0]),
                       proj.depth, pair_emit, vals, keys, at<unsigned long long>(ws, L.scratch));
    return hipGetLastError();
}

}  // namespace gsmi
