// Rendering phase part 2 (forward alpha blending), the L1 image loss, and the
// backward phase (pixel replay + per-primitive chain rule).
//
// Forward: one 256-thread workgroup per 16x16 tile, one pixel per thread.
// The tile's sorted pairs are staged through LDS in batches of 256
// (mean2d, conic+opacity, rgb, footprint half-extents); a workgroup-wide
// count of finished pixels ends the batch loop early.
//
// Backward: same tile/pixel mapping, walking each tile's pairs back to front.
// Each pixel recovers the transmittance in front of a pair by dividing by
// (1 - alpha) and keeps the projection of the suffix colour sum on its
// upstream gradient; per pair, six moment and colour sums are taken over each
// 16-lane pixel row with DPP, stored in the row's LDS record of the pair,
// combined over the rows of a wave and over the 4 waves in a fixed order, and
// written to the pair's slot at its emission position (a primitive's pairs
// side by side).  Per visible primitive, k_slot_sum adds its slots in order
// -- deterministic, no floating-point atomics in global memory -- and
// k_project_bwd applies the projection and colour chain rule (geometry in
// fp64) and writes one compact gradient row.
#include "common.h"
#include "internal.h"

namespace gsmi {

namespace {

constexpr float kAlphaMin = 1.0f / 255.0f;
constexpr float kAlphaMax = 0.99f;
constexpr float kTMin = 1e-4f;
constexpr float kCutMargin = 1e-3f;   // extra sigma beyond the 1/255 cut-off when bounding a footprint

// One pair's primitive as staged in LDS: 72 bytes in five arrays, every lane
// of a wave reading the same record (a broadcast):
//   P (u, v) and Q (A/2, B) in fp64, R = (C/2 in fp64, opacity, hx),
//   S = (r, g, b, hy), T = (cut, slope) for the row lists (computed once per
//   staged entry rather than by every wave that tests it).
// The pixel-space mean and conic are fp32 values held exactly in fp64, so
// that the quadratic form is evaluated in fp64 without per-pair conversions.
// hx, hy bound the pixel offsets at which o*exp(-sigma) can reach 1/255: for
// sigma = d^T Q d / 2 <= s the offsets obey |dx| <= sqrt(2 s C / det Q) and
// |dy| <= sqrt(2 s A / det Q); s = cut = ln(255 o) + kCutMargin keeps every
// skipped pair at least 0.1% below the threshold, far outside fp32 rounding.
// slope = -B/A (fp32) is the vertex of sigma along a pixel row per unit dy.
struct __align__(16) SplatR {
    double c2;
    float o;
    float hx;
};

template <int NB>
struct SplatLds {
    double2 P[NB];
    double2 Q[NB];
    SplatR R[NB];
    float4 S[NB];
    float2 T[NB];
};

template <int NB>
__device__ __forceinline__ void stage_splat(SplatLds<NB>& L, int k, float2 m, float4 co,
                                            const float* __restrict__ rgb3) {
    const float cut = logf(255.0f * co.w) + kCutMargin;
    const float det = co.x * co.z - co.y * co.y;
    float hx, hy;
    if (!(cut > 0.0f)) {
        hx = hy = -1e30f;                 // opacity below 1/255: no pixel can take it
    } else if (!(det > 0.0f)) {
        hx = hy = 1e30f;                  // degenerate conic in fp32: never skip
    } else {
        hx = sqrtf(2.0f * cut * co.z / det);
        hy = sqrtf(2.0f * cut * co.x / det);
    }
    L.P[k] = make_double2((double)m.x, (double)m.y);
    L.Q[k] = make_double2(0.5 * (double)co.x, (double)co.y);
    SplatR r;
    r.c2 = 0.5 * (double)co.z;
    r.o = co.w;
    r.hx = hx;
    L.R[k] = r;
    L.S[k] = make_float4(rgb3[0], rgb3[1], rgb3[2], hy);
    L.T[k] = make_float2(cut, co.x > 0.0f ? -co.y * __builtin_amdgcn_rcpf(co.x) : 0.0f);
}

// Can any pixel centre of the wave's strip [x0,x1] x [y0,y1] reach the cut-off?
template <int NB>
__device__ __forceinline__ bool splat_touches(const SplatLds<NB>& L, int k, float x0, float x1, float y0, float y1) {
    const double2 p = L.P[k];
    const float u = (float)p.x, v = (float)p.y;        // exact: staged from fp32
    const float hx = L.R[k].hx, hy = L.S[k].w;
    return (u + hx >= x0) && (u - hx <= x1) && (v + hy >= y0) && (v - hy <= y1);
}

// sigma of one (pixel, primitive) pair, in fp64: for elongated footprints far
// from their centre the three terms of the quadratic form are large and
// cancel, and fp32 loses up to ~1e-3 of sigma there (the error grows with the
// conic's condition number).  The offsets are exact in fp64.  Forward and
// backward both call this on the same staged record, so they take identical
// decisions.  bdy = B dy and cdy = (C/2) dy are returned for the backward's
// d sigma / d(u, v).  px, py are the pixel centre.
#pragma clang fp contract(off)
__device__ __forceinline__ float splat_sigma(double2 P, double2 Q, double c2, double px, double py, double& ddx,
                                             double& ddy, double& inner, double& cdy) {
    ddx = P.x - px;
    ddy = P.y - py;
    inner = fma(Q.x, ddx, Q.y * ddy);            // A/2 dx + B dy
    cdy = c2 * ddy;                              // C/2 dy
    return (float)fma(ddx, inner, cdy * ddy);
}
#pragma clang fp contract(on)

// exp(-sigma) = 2^-t with t = sigma log2(e) carried as hi + lo (log2(e)
// split into an fp32 head and tail; hi = sigma * head rounded, lo its exact
// rounding error plus sigma * tail, |lo| < 2e-5 for the sigmas that matter).
// 2^-t = 2^-hi * 2^-lo with 2^-lo = 1 - lo ln2 up to (lo ln2)^2 / 2 < 1e-10;
// the hardware base-2 exponential (1 ulp) takes -hi directly.  About two ulps
// in all, far inside the alpha decision band; forward and backward call the
// same code, so they take identical decisions.  Very large sigmas give 0,
// negative ones are rejected by the caller.
__device__ __forceinline__ float exp_neg(float sigma) {
    constexpr float kLog2eHi = 1.44269502162933349609375f;    // log2(e) rounded to fp32
    constexpr float kLog2eLo = 1.925963033500011e-08f;        // log2(e) - kLog2eHi
    constexpr float kLn2 = 0.693147180559945309417f;
    const float hi = sigma * kLog2eHi;
    float lo = fmaf(sigma, kLog2eHi, -hi);
    lo = fmaf(sigma, kLog2eLo, lo);
    return __builtin_amdgcn_exp2f(-hi) * fmaf(-lo, kLn2, 1.0f);
}


// Row-wise lists: each 16-lane row of a wave (one pixel row of the tile)
// keeps its own ascending list of the batch entries whose footprint reaches
// that row's pixel centres (and lie below the row's limit).  The four rows of
// a wave then walk their lists in lockstep, so an entry costs a quarter of a
// wave step for every pixel row it reaches instead of a whole step for every
// 16x4 strip.  cnt[r] receives the length of row r's list.  With REV (one
// ballot round, NB = 64) each list is stored back to front, so that a walk
// from the last entry to the first reads positions 0, 1, 2, ...
//
// An entry reaches row y if sigma <= s somewhere on the row's segment of
// pixel centres [x0, x1] (s = cut = ln(255 o) + kCutMargin as for hx, hy):
// the footprint box is tested first, then sigma at the quadratic's vertex dx =
// slope dy (slope = -B/A in fp32) clamped to the segment's offsets [u - x1,
// u - x0], in fp64 (the staged values are exact).  Off the exact vertex by the
// slope's rounding (a few 1e-7 relative), sigma there exceeds the segment's
// minimum by at most about 4e-13 (B^2 / det), i.e. 4e-13 times the squared
// axis ratio of the footprint: inside the 1e-3 margin up to ratios near 5e4,
// where the fp32 conic itself has lost its accuracy.  Any pixel of a skipped
// row stays below the 1/255 threshold.
template <int NB, bool REV = false>
__device__ __forceinline__ void compact_rows(const SplatLds<NB>& L, int nb, float x0, float x1, float y0,
                                             const uint32_t* lim, uint8_t (*list)[NB], uint32_t* cnt) {
    static_assert(!REV || NB == GS_WAVE, "a list is reversed within its one ballot round");
    const int lane = lane_id();
    const uint64_t lt = lanemask_lt();
#pragma unroll
    for (int q = 0; q < 4; ++q) cnt[q] = 0;
#pragma unroll
    for (int r = 0; r < NB / GS_WAVE; ++r) {
        const int k = r * GS_WAVE + lane;
        const bool valid = k < nb;
        const int kk = valid ? k : 0;
        const double2 p = L.P[kk];
        const double2 qd = L.Q[kk];
        const SplatR R = L.R[kk];
        const float u = (float)p.x, v = (float)p.y;
        const float hx = R.hx, hy = L.S[kk].w;
        const bool bx = valid && (u + hx >= x0) && (u - hx <= x1);
        const float2 cs = L.T[kk];
        const double cut = (double)cs.x;
        const bool convex = qd.x > 0.0;                      // A > 0 for every projected conic; else no row test
        const double slope = (double)cs.y;                   // vertex offset per unit dy: -B / A (0 unless A > 0)
        const double dlo = p.x - (double)x1, dhi = p.x - (double)x0;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const float y = y0 + (float)q;
            const double dy = p.y - (double)y;
            const double dx = fmin(fmax(slope * dy, dlo), dhi);
            const double smin = dx * fma(qd.x, dx, qd.y * dy) + R.c2 * dy * dy;
            const bool t = bx && (uint32_t)k < lim[q] && (v + hy >= y) && (v - hy <= y) && (smin <= cut || !convex);
            const uint64_t m = __ballot(t);
            if (t) list[q][REV ? popc64(m) - 1u - popc64(m & lt) : cnt[q] + popc64(m & lt)] = (uint8_t)k;
            cnt[q] += popc64(m);
        }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// The value of a wave-uniform per-row quantity for this lane's row.
__device__ __forceinline__ uint32_t for_row(const uint32_t* v, int row) {
    return row == 0 ? v[0] : (row == 1 ? v[1] : (row == 2 ? v[2] : v[3]));
}

// |a - t| and the sign of a - t scaled by inv (0 for a tie): one L1 term and its derivative.
__device__ __forceinline__ float l1_elem(float a, float t, float inv, float& dl) {
    const float d = a - t;
    dl = d > 0.0f ? inv : (d < 0.0f ? -inv : 0.0f);
    return fabsf(d);
}

// The tile a workgroup renders: the grid covers the tiles once, in the
// caller's dispatch order (longest first from gs_bin_sort), else row-major.
// Pixels, losses and pair records are per tile, so the order changes no
// result, only how the longest tiles overlap the rest.
__device__ __forceinline__ uint32_t dispatch_tile(const uint32_t* __restrict__ tile_order) {
    return tile_order ? tile_order[blockIdx.x] : blockIdx.x;
}

// LOSS: the L1 loss of the view is taken in the same pass (the image loss of
// the view, Section 2.1): each pixel compares its three fp32 channels with
// the target exactly as k_loss_l1 does, writes dL/dimg, and each tile leaves
// its sum of |img - target| in loss_partial[tile] for k_loss_final.
template <bool STATS, bool LOSS>
__global__ void __launch_bounds__(GS_BLOCK, STATS ? 5 : 7) k_raster_fwd(
    const uint32_t* __restrict__ tile_order, const uint32_t* __restrict__ ranges, const uint32_t* __restrict__ vals,
    const float2* __restrict__ mean2d, const float4* __restrict__ conic_op, const float* __restrict__ rgb, int32_t W,
    int32_t H, int32_t TX, float bg0, float bg1, float bg2, float* __restrict__ img, float* __restrict__ final_T,
    uint32_t* __restrict__ n_contrib,
    uint8_t* __restrict__ active, unsigned long long* __restrict__ pair_stats, const float* __restrict__ target,
    float inv_total, float* __restrict__ dL, float* __restrict__ loss_partial) {
    __shared__ SplatLds<GS_BLOCK> L;
    // entries some pixel included (active flags): every including lane stores 1 to
    // the entry's byte, plain stores of one value (LDS atomics on one word from a
    // whole row serialize)
    __shared__ uint8_t s_hit[GS_BLOCK];
    __shared__ uint8_t s_list[4][4][GS_BLOCK];
    __shared__ uint32_t s_stat[4][4];
    const uint32_t tile = dispatch_tile(tile_order);
    if (tile >= gridDim.x) return;
    const int tid = threadIdx.x;
    const int w = tid / GS_WAVE;
    const int lane = lane_id();
    const int row = lane >> 4;
    const int tx = (int)tile % TX, ty = (int)tile / TX;
    const int px = tx * GS_TILE + (tid % GS_TILE);
    const int py = ty * GS_TILE + (tid / GS_TILE);
    const bool inside = px < W && py < H;
    const double fx = px + 0.5, fy = py + 0.5;
    // pixel-centre bounds of this wave's 16x4 strip
    const float wx0 = tx * GS_TILE + 0.5f, wx1 = wx0 + 15.0f;
    const float wy0 = ty * GS_TILE + 4 * w + 0.5f;
    const uint32_t start = ranges[2 * tile], end = ranges[2 * tile + 1];
    float T = 1.0f, c0 = 0.0f, c1 = 0.0f, c2 = 0.0f;
    uint32_t last = 0, n_inc = 0, term_at = 0, w_iter = 0, w_hit = 0;
    bool done = !inside, terminated = false;
    // the ids of the next batch load while this one is walked
    uint32_t g = start + tid < end ? vals[start + tid] : 0u;
    for (uint32_t bs = start; bs < end; bs += GS_BLOCK) {
        if (__syncthreads_count(done) == GS_BLOCK) break;
        const uint32_t j = bs + tid;
        const uint32_t gj = g;
        if (j < end) stage_splat(L, tid, mean2d[gj], conic_op[gj], rgb + 3 * (size_t)gj);
        if (j + GS_BLOCK < end) g = vals[j + GS_BLOCK];
        s_hit[tid] = 0;
        __syncthreads();
        const int nb = (int)min((uint32_t)GS_BLOCK, end - bs);
        // rows whose 16 pixels are all finished take no entries
        const uint64_t live = __ballot(!done);
        uint32_t lim[4], nl[4] = {0u, 0u, 0u, 0u};
#pragma unroll
        for (int q = 0; q < 4; ++q) lim[q] = ((live >> (16 * q)) & 0xFFFFull) ? (uint32_t)GS_BLOCK : 0u;
        if (live) compact_rows(L, nb, wx0, wx1, wy0, lim, s_list[w], nl);
        const uint32_t my_n = for_row(nl, row);
        // the counts come from ballots, so every lane holds the same values
        const uint32_t steps = __builtin_amdgcn_readfirstlane(max(max(nl[0], nl[1]), max(nl[2], nl[3])));
        uint64_t live_w = live;     // lanes not yet done, kept as a scalar mask
        for (uint32_t jj = 0; jj < steps; ++jj) {
            if (live_w == 0ull) break;
            const bool act = jj < my_n;
            // the list read needs no branch (every byte indexes the 256-entry batch), but
            // past the row's count the byte is stale and may name a slot this batch never
            // staged, whose colour could be Inf or NaN (0 * Inf poisons the sums): such
            // lanes take entry 0, which every batch stages
            const int k_list = s_list[w][row][jj];
            const int k = act ? k_list : 0;
            const SplatR R = L.R[k];
            double ddx, ddy, inner, cdy;
            const float sigma = splat_sigma(L.P[k], L.Q[k], R.c2, fx, fy, ddx, ddy, inner, cdy);
            const float alpha = fminf(kAlphaMax, R.o * exp_neg(sigma));
            bool ok = act && !done && !(sigma < 0.0f) && !(alpha < kAlphaMin);
            const float Tn = T * (1.0f - alpha);
            const bool term = ok && (Tn < kTMin);
            const uint32_t pos = bs - start + (uint32_t)k;
            if (STATS && term) term_at = pos;
            terminated = terminated || term;
            done = done || term;
            // the terminating lanes, as ballots of the comparisons themselves (a ballot of
            // a compare is its lane mask; a ballot of a combined flag costs two VALU ops)
            live_w &= ~(__builtin_amdgcn_ballot_w64(act) & live_w & __builtin_amdgcn_ballot_w64(!(sigma < 0.0f)) &
                        __builtin_amdgcn_ballot_w64(!(alpha < kAlphaMin)) & __builtin_amdgcn_ballot_w64(Tn < kTMin));
            ok = ok && !term;
            const float4 col = L.S[k];
            const float wgt = ok ? alpha * T : 0.0f;
            c0 = fmaf(wgt, col.x, c0);
            c1 = fmaf(wgt, col.y, c1);
            c2 = fmaf(wgt, col.z, c2);
            T = ok ? Tn : T;
            last = ok ? pos + 1u : last;
            if (STATS) {
                n_inc += ok ? 1u : 0u;
                const uint64_t am = __ballot(act), om = __ballot(ok);
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    w_iter += ((am >> (16 * q)) & 0xFFFFull) ? 1u : 0u;
                    w_hit += ((om >> (16 * q)) & 0xFFFFull) ? 1u : 0u;
                }
            }
            if (active != nullptr && ok) s_hit[k] = 1;
        }
        __syncthreads();
        if (active && j < end && s_hit[tid]) active[gj] = 1;
    }
    if (STATS) {
        // entries the per-pixel definition examines: up to and including the
        // terminating one, else the whole list
        const uint32_t n_eval = !inside ? 0u : (terminated ? term_at + 1u : end - start);
        const uint32_t e = wave_sum_u32(n_eval), i = wave_sum_u32(n_inc);
        if (lane_id() == 0) {
            s_stat[0][w] = e;
            s_stat[1][w] = i;
            s_stat[2][w] = w_iter;      // wave-uniform counts
            s_stat[3][w] = w_hit;
        }
        __syncthreads();
        if (tid < 4)
            atomicAdd(&pair_stats[tid], (unsigned long long)s_stat[tid][0] + s_stat[tid][1] + s_stat[tid][2] +
                                            s_stat[tid][3]);
    }
    float lsum = 0.0f;
    if (inside) {
        const size_t HW = (size_t)W * H, p = (size_t)py * W + px;
        const float o0 = fmaf(T, bg0, c0), o1 = fmaf(T, bg1, c1), o2 = fmaf(T, bg2, c2);
        img[p] = o0;
        img[HW + p] = o1;
        img[2 * HW + p] = o2;
        final_T[p] = T;
        n_contrib[p] = last;
        if (LOSS) {
            float g0, g1, g2;
            lsum += l1_elem(o0, target[p], inv_total, g0);
            lsum += l1_elem(o1, target[HW + p], inv_total, g1);
            lsum += l1_elem(o2, target[2 * HW + p], inv_total, g2);
            dL[p] = g0;
            dL[HW + p] = g1;
            dL[2 * HW + p] = g2;
        }
    }
    if (LOSS) {
        __shared__ float s_loss[4];
        lsum = wave_sum(lsum);
        if (lane_id() == 0) s_loss[w] = lsum;
        __syncthreads();
        if (tid == 0) loss_partial[tile] = (s_loss[0] + s_loss[1]) + (s_loss[2] + s_loss[3]);
    }
}

// ---------------------------------------------------------------------------
// L1 loss
// ---------------------------------------------------------------------------


// Block b covers elements [b*2048, b*2048+2048): with VEC, as 512 float4
// (all three arrays 16-byte aligned; elements past the last whole float4
// are done one by one by the last block), else element by element.
template <bool VEC>
__global__ void __launch_bounds__(GS_BLOCK) k_loss_l1(const float* __restrict__ img, const float* __restrict__ tgt,
                                                      uint32_t total, float inv, float* __restrict__ dL,
                                                      float* __restrict__ partial) {
    __shared__ float s_red[4];
    float acc = 0.0f;
    if (VEC) {
        const uint32_t n4 = total / 4;
        const float4* a4 = reinterpret_cast<const float4*>(img);
        const float4* t4 = reinterpret_cast<const float4*>(tgt);
        float4* d4 = reinterpret_cast<float4*>(dL);
        const uint32_t base = blockIdx.x * (GS_TILE_ITEMS / 4) + threadIdx.x;
#pragma unroll
        for (int k = 0; k < GS_ITEMS / 4; ++k) {
            const uint32_t i = base + k * GS_BLOCK;
            if (i < n4) {
                const float4 a = a4[i], t = t4[i];
                float4 g;
                acc += l1_elem(a.x, t.x, inv, g.x);
                acc += l1_elem(a.y, t.y, inv, g.y);
                acc += l1_elem(a.z, t.z, inv, g.z);
                acc += l1_elem(a.w, t.w, inv, g.w);
                d4[i] = g;
            }
        }
        if (blockIdx.x == gridDim.x - 1 && threadIdx.x < total - 4 * n4) {
            const uint32_t i = 4 * n4 + threadIdx.x;
            float g;
            acc += l1_elem(img[i], tgt[i], inv, g);
            dL[i] = g;
        }
    } else {
        const uint32_t base = blockIdx.x * GS_TILE_ITEMS + threadIdx.x;
#pragma unroll
        for (int k = 0; k < GS_ITEMS; ++k) {
            const uint32_t i = base + k * GS_BLOCK;
            if (i < total) {
                float g;
                acc += l1_elem(img[i], tgt[i], inv, g);
                dL[i] = g;
            }
        }
    }
    acc = wave_sum(acc);
    if (lane_id() == 0) s_red[threadIdx.x / GS_WAVE] = acc;
    __syncthreads();
    if (threadIdx.x == 0) partial[blockIdx.x] = (s_red[0] + s_red[1]) + (s_red[2] + s_red[3]);
}

__global__ void __launch_bounds__(GS_BLOCK) k_loss_final(const float* __restrict__ partial, uint32_t nb,
                                                         double inv_total, float* __restrict__ loss) {
    __shared__ double s[GS_BLOCK / GS_WAVE];
    constexpr int U = 8;
    double acc = 0.0;
    // all of a thread's loads are issued before its sums (float4 when aligned)
    uint32_t done = 0;
    if ((reinterpret_cast<uintptr_t>(partial) & 15u) == 0u) {
        const uint32_t n4 = nb / 4u;
        const float4* p4 = reinterpret_cast<const float4*>(partial);
        for (uint32_t i0 = threadIdx.x; i0 < n4; i0 += U * GS_BLOCK) {
            float4 v[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const uint32_t i = i0 + (uint32_t)u * GS_BLOCK;
                v[u] = i < n4 ? p4[i] : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
            }
#pragma unroll
            for (int u = 0; u < U; ++u)
                acc += ((double)v[u].x + (double)v[u].y) + ((double)v[u].z + (double)v[u].w);
        }
        done = 4u * n4;
    }
    for (uint32_t i = done + threadIdx.x; i < nb; i += GS_BLOCK) acc += (double)partial[i];
#pragma unroll
    for (int d = GS_WAVE / 2; d >= 1; d >>= 1) acc += __shfl_xor(acc, d, GS_WAVE);
    if (lane_id() == 0) s[threadIdx.x / GS_WAVE] = acc;
    __syncthreads();
    if (threadIdx.x == 0) *loss = (float)(((s[0] + s[1]) + (s[2] + s[3])) * inv_total);
}

// ---------------------------------------------------------------------------
// backward, part 1: per pixel, back to front
// ---------------------------------------------------------------------------

constexpr int kG = 9;   // du dv dA dB dC dopacity dr dg db
constexpr int kSlot = 12;          // floats per pair slot (9 used, padded for 16-byte stores)
constexpr int kRowSums = 6;        // per-row sums: sum ds, sum ds dx, sum ds dx^2, three colour sums
// Pairs staged per batch: one per lane, so that after the walk each wave adds
// its four rows' sums of entry k in lane k.  The per-row sums (16 rows x 6
// floats per staged pair, 24 KB) dominate the workgroup's LDS.
constexpr int kBwdBatch = GS_WAVE;

// Per pixel, walking back to front: T is recovered in front of each included
// pair as T / (1 - alpha), and instead of the three suffix colour sums S_c
// (the colour still to come behind the pair, background included) the pixel
// keeps their projection gS = sum_c dL/dC_c S_c on its upstream gradient,
// which is all that d alpha needs:
//   dL/dalpha = T_k (g . rgb) - gS / (1 - alpha),  gS += alpha T_k (g . rgb).
// Each 16-lane pixel row walks its own list of the batch (compact_rows),
// back to front, only up to the last pair any of its pixels included.
//
// The 2D gradient of a pair is linear in moments of ds = dL/dsigma over its
// pixels: with sigma = (A dx^2 + 2B dx dy + C dy^2) / 2 and (dx, dy) the offset
// of the splat centre from the pixel centre,
//   dL/du = A m_x + B m_y,  dL/dv = B m_x + C m_y,
//   dL/dA = m_xx / 2,  dL/dB = m_xy,  dL/dC = m_yy / 2,  dL/dopacity = -m / o,
// with m = sum ds, m_x = sum ds dx, m_xy = sum ds dx dy and so on (the opacity
// line because ds = -dL/dalpha * o e^-sigma below the 0.99 cap, and both are 0
// at it).  A pixel row shares dy, so a row needs only m, m_x and m_xx (plus
// the three colour sums) over its lanes.  A row visits an entry at most once
// per batch, so two lanes of the row (one holding the moment sums, one the
// colour sums) store the six sums with plain LDS writes into the row's own
// record of that entry (no atomics); after the walk lane k of each
// wave scales its four rows' records of entry k by their dy and adds them,
// and the four waves' results are added in a fixed order.  A pair slot holds
// (m_x, m_y, m_xx, m_xy, m_yy, m, colour); k_project_bwd expands it with the
// conic once per primitive.
__global__ void __launch_bounds__(GS_BLOCK) k_raster_bwd(
    const uint32_t* __restrict__ tile_order, const uint32_t* __restrict__ ranges, const uint32_t* __restrict__ vals,
    const float2* __restrict__ mean2d, const float4* __restrict__ conic_op, const float* __restrict__ rgb, int32_t W,
    int32_t H, int32_t TX, float bg0,
    float bg1, float bg2, const float* __restrict__ final_T, const uint32_t* __restrict__ n_contrib,
    const float* __restrict__ dL_dimg, const uint32_t* __restrict__ pair_emit, float* __restrict__ slots) {
    __shared__ SplatLds<kBwdBatch> L;
    // [wave][row][sum][entry]; after the walk a wave's part holds its 9 combined
    // sums per entry, [q][entry]
    __shared__ float s_row[4][4][kRowSums][kBwdBatch];
    __shared__ uint8_t s_list[4][4][kBwdBatch];
    __shared__ uint32_t s_max;
    static_assert(kG * kBwdBatch <= 4 * kRowSums * kBwdBatch, "combined sums fit a wave's row records");
    const uint32_t tile = dispatch_tile(tile_order);
    if (tile >= gridDim.x) return;
    const int tid = threadIdx.x;
    const int w = tid / GS_WAVE;
    const int lane = lane_id();
    const int row = lane >> 4;
    const int tx = (int)tile % TX, ty = (int)tile / TX;
    const int px = tx * GS_TILE + (tid % GS_TILE);
    const int py = ty * GS_TILE + (tid / GS_TILE);
    const bool inside = px < W && py < H;
    const double fx = px + 0.5, fy = py + 0.5;
    const float wx0 = tx * GS_TILE + 0.5f, wx1 = wx0 + 15.0f;
    const float wy0 = ty * GS_TILE + 4 * w + 0.5f;
    const uint32_t start = ranges[2 * tile], end = ranges[2 * tile + 1];
    const size_t HW = (size_t)W * H, pix = (size_t)py * W + px;
    float T = inside ? final_T[pix] : 1.0f;
    const uint32_t last = inside ? n_contrib[pix] : 0u;
    const float gC0 = inside ? dL_dimg[pix] : 0.0f;
    const float gC1 = inside ? dL_dimg[HW + pix] : 0.0f;
    const float gC2 = inside ? dL_dimg[2 * HW + pix] : 0.0f;
    float gS = T * (gC0 * bg0 + gC1 * bg1 + gC2 * bg2);
    if (tid == 0) s_max = 0;
    {
        // a walk reads list bytes past its row's count too (without a branch): every
        // byte must name an entry of the batch arrays, and every entry must hold
        // finite values, also before a batch has written them
        static_assert(sizeof(s_list) == 4 * GS_BLOCK, "one word of the lists per thread");
        reinterpret_cast<uint32_t*>(&s_list[0][0][0])[tid] = 0u;
        float4* zs = reinterpret_cast<float4*>(&L);
        for (int i = tid; i < (int)(sizeof(L) / 16); i += GS_BLOCK) zs[i] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    }
    __syncthreads();
    if (last > 0) atomicMax(&s_max, last);
    __syncthreads();
    const uint32_t maxlast = s_max;
    const bool hi_half = (lane & 8) != 0;       // high half of the lane's 16-lane row
    const int q_half = hi_half ? 3 : 0;         // the half's three sums in a row record
    // the colour sums of entry k sit at index k ^ 16: the row's two storing lanes
    // (same entry, records 3 x 64 floats apart) then hit different banks
    const int k_half = hi_half ? 16 : 0;
    // largest n_contrib of each pixel row of this wave (wave-uniform values)
    uint32_t rl = last;
#pragma unroll
    for (int d = 8; d >= 1; d >>= 1) rl = max(rl, (uint32_t)__shfl_xor((int)rl, d, GS_WAVE));
    uint32_t row_last[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) row_last[q] = (uint32_t)__builtin_amdgcn_readlane((int)rl, 16 * q);
    const uint32_t n = end - start;
    for (int64_t be = n; be > 0; be -= kBwdBatch) {
        const uint32_t bs = (uint32_t)(be > kBwdBatch ? be - kBwdBatch : 0);
        const uint32_t cnt = (uint32_t)be - bs;
        const bool work = bs < maxlast;
        const uint32_t last_b = last > bs ? last - bs : 0u;    // the pixel's entries in this batch: k < last_b
        if ((uint32_t)tid < cnt && work) {
            const uint32_t g = vals[start + bs + tid];
            stage_splat(L, tid, mean2d[g], conic_op[g], rgb + 3 * (size_t)g);
        }
        if (work) {
            // rows that never take an entry leave its record at zero
            float4* z = reinterpret_cast<float4*>(&s_row[w][0][0][0]);
#pragma unroll
            for (int i = 0; i < 4 * kRowSums * kBwdBatch / 4 / GS_WAVE; ++i)
                z[i * GS_WAVE + lane] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
        }
        __syncthreads();
        uint32_t lim[4], nl[4] = {0u, 0u, 0u, 0u};
        bool any = false;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            lim[q] = row_last[q] > bs ? row_last[q] - bs : 0u;
            any = any || lim[q] > 0u;
        }
        if (work && any) compact_rows<kBwdBatch, true>(L, (int)cnt, wx0, wx1, wy0, lim, s_list[w], nl);
        const uint32_t my_n = for_row(nl, row);
        // the counts come from ballots, so every lane holds the same values
        uint32_t nls[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) nls[q] = __builtin_amdgcn_readfirstlane(nl[q]);
        const uint32_t steps = __builtin_amdgcn_readfirstlane(max(max(nls[0], nls[1]), max(nls[2], nls[3])));
        for (uint32_t jj = 0; jj < steps; ++jj) {
            const bool act = jj < my_n;
            // act's lanes from the rows' list lengths, in scalar registers
            uint64_t act_mask = 0ull;
#pragma unroll
            for (int q = 0; q < 4; ++q) act_mask |= jj < nls[q] ? 0xFFFFull << (16 * q) : 0ull;
            // the lists are stored back to front; past the row's count the byte is stale
            // (or cleared) but names an entry whose values are finite, and the lane is
            // not ok
            const int k = s_list[w][row][jj];
            const SplatR R = L.R[k];
            double ddx, ddy, inner, cdy;
            const float sigma = splat_sigma(L.P[k], L.Q[k], R.c2, fx, fy, ddx, ddy, inner, cdy);
            const float e = exp_neg(sigma);
            const float gv = R.o * e;
            const float alpha = fminf(kAlphaMax, gv);
            const bool ok = act & ((uint32_t)k < last_b) & !(sigma < 0.0f) & !(alpha < kAlphaMin);
            // the lanes of ok, as ballots of the comparisons themselves (a ballot of a
            // compare is its lane mask; a ballot of a combined flag costs two VALU ops)
            const uint64_t mask = act_mask & __builtin_amdgcn_ballot_w64((uint32_t)k < last_b) &
                                  __builtin_amdgcn_ballot_w64(!(sigma < 0.0f)) &
                                  __builtin_amdgcn_ballot_w64(!(alpha < kAlphaMin));
            if (mask == 0ull) continue;
            const float4 col = L.S[k];
            // a lane that is not ok takes alpha = 0: 1 / (1 - 0) = 1 leaves its T as it
            // is, and its weight and d sigma are 0
            const float a_ok = ok ? alpha : 0.0f;
            const float inv_om = __builtin_amdgcn_rcpf(1.0f - a_ok);
            const float Tk = T * inv_om;
            const float gcol = gC0 * col.x + gC1 * col.y + gC2 * col.z;
            const float dalpha = Tk * gcol - gS * inv_om;
            const float wgt = a_ok * Tk;
            gS = fmaf(wgt, gcol, gS);
            T = Tk;
            const float a_geo = gv < kAlphaMax ? a_ok : 0.0f;   // the 0.99 cap stops d/d(opacity, sigma)
            const float ds = -dalpha * a_geo;
            const float dsx = ds * (float)ddx;
            // the six sums over each 16-lane row (all its lanes hold the same entry)
            // in 18 DPP adds instead of 24: the first stage pairs lane i with lane
            // 15 - i, the low half of the row keeping the three moment terms and the
            // high half the three colour terms (each adds its partner's copy of the
            // term it keeps); three butterfly stages within each half of eight lanes
            // then leave the moment sums in every low lane and the colour sums in
            // every high lane
            const float mo[3] = {ds, dsx, dsx * (float)ddx};
            const float co[3] = {gC0 * wgt, gC1 * wgt, gC2 * wgt};
            float gr[3];
#pragma unroll
            for (int q = 0; q < 3; ++q) {
                const float keep = hi_half ? co[q] : mo[q];
                const float send = hi_half ? mo[q] : co[q];
                gr[q] = keep + __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(send), 0x140, 0xF, 0xF,
                                                                          true));
            }
#pragma unroll
            for (int q = 0; q < 3; ++q) {
                gr[q] += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(gr[q]), 0xB1, 0xF, 0xF, true));
                gr[q] += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(gr[q]), 0x4E, 0xF, 0xF, true));
                gr[q] += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(gr[q]), 0x141, 0xF, 0xF, true));
                // keep the last add in front of the branch (all lanes active), where
                // it folds into the DPP instruction
                asm volatile("" : "+v"(gr[q]));
            }
            // lanes 0 and 8 of every row that walks an entry store (moments and colour
            // sums): a row without a contributing pixel stores zero sums into its
            // record, which holds zeros (records are cleared per batch and a row
            // visits an entry once)
            if ((lane & 7) == 0 && act) {
#pragma unroll
                for (int q = 0; q < 3; ++q) s_row[w][row][q_half + q][k ^ k_half] = gr[q];
            }
        }
        // lane k adds this wave's four row records of entry k: only this wave
        // wrote them, so a wave-level barrier orders the writes before the reads
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        if (work) {
            float acc[kG] = {0, 0, 0, 0, 0, 0, 0, 0, 0};
            const double vk = L.P[lane].y;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const float dy = (float)(vk - (double)(wy0 + (float)q));   // the row's common offset
                const float m = s_row[w][q][0][lane], mx = s_row[w][q][1][lane];
                const float my = dy * m;
                acc[0] += mx;
                acc[1] += my;
                acc[2] += s_row[w][q][2][lane];
                acc[3] += dy * mx;
                acc[4] += dy * my;
                acc[5] += m;
                acc[6] += s_row[w][q][3][lane ^ 16];
                acc[7] += s_row[w][q][4][lane ^ 16];
                acc[8] += s_row[w][q][5][lane ^ 16];
            }
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
            float* comb = &s_row[w][0][0][0];
#pragma unroll
            for (int q = 0; q < kG; ++q) comb[q * kBwdBatch + lane] = acc[q];
        }
        __syncthreads();
        if ((uint32_t)tid < cnt) {
            // the pair's slot is its emission position: a primitive's pairs end up
            // side by side, for k_project_bwd to read contiguously
            float v[kSlot] = {0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0};
            if (work) {
                const float* c0 = &s_row[0][0][0][0];
                const float* c1 = &s_row[1][0][0][0];
                const float* c2 = &s_row[2][0][0][0];
                const float* c3 = &s_row[3][0][0][0];
#pragma unroll
                for (int q = 0; q < kG; ++q) {
                    const int i = q * kBwdBatch + tid;
                    v[q] = (c0[i] + c1[i]) + (c2[i] + c3[i]);
                }
            }
            float4* dst = reinterpret_cast<float4*>(slots + (size_t)pair_emit[start + bs + tid] * kSlot);
            dst[0] = make_float4(v[0], v[1], v[2], v[3]);
            dst[1] = make_float4(v[4], v[5], v[6], v[7]);
            dst[2] = make_float4(v[8], v[9], v[10], v[11]);
        }
        __syncthreads();
    }
}

// ---------------------------------------------------------------------------
// backward, part 2: per visible primitive
// ---------------------------------------------------------------------------

constexpr float kY1 = 0.48860251190291992f;
constexpr float kY2a = 1.0925484305920792f;
constexpr float kY2b = 0.31539156525252005f;
constexpr float kY2c = 0.54627421529603959f;
constexpr float kY3a = 0.59004358992664352f;
constexpr float kY3b = 2.8906114426405538f;
constexpr float kY3c = 0.45704579946446572f;
constexpr float kY3d = 0.37317633259011546f;
constexpr float kY3e = 1.4453057213202769f;

// SH basis values and gradients of their polynomial form at d.
template <int DEG>
__device__ __forceinline__ void sh_basis_grad(float x, float y, float z, float* Y, float (*G)[3]) {
    Y[0] = 0.28209479177387814f;
    G[0][0] = G[0][1] = G[0][2] = 0.0f;
    if (DEG < 1) return;
    Y[1] = -kY1 * y; G[1][0] = 0.0f; G[1][1] = -kY1; G[1][2] = 0.0f;
    Y[2] = kY1 * z;  G[2][0] = 0.0f; G[2][1] = 0.0f; G[2][2] = kY1;
    Y[3] = -kY1 * x; G[3][0] = -kY1; G[3][1] = 0.0f; G[3][2] = 0.0f;
    if (DEG < 2) return;
    const float xx = x * x, yy = y * y, zz = z * z;
    Y[4] = kY2a * x * y;  G[4][0] = kY2a * y; G[4][1] = kY2a * x; G[4][2] = 0.0f;
    Y[5] = -kY2a * y * z; G[5][0] = 0.0f; G[5][1] = -kY2a * z; G[5][2] = -kY2a * y;
    Y[6] = kY2b * (2.0f * zz - xx - yy);
    G[6][0] = -2.0f * kY2b * x; G[6][1] = -2.0f * kY2b * y; G[6][2] = 4.0f * kY2b * z;
    Y[7] = -kY2a * x * z; G[7][0] = -kY2a * z; G[7][1] = 0.0f; G[7][2] = -kY2a * x;
    Y[8] = kY2c * (xx - yy); G[8][0] = 2.0f * kY2c * x; G[8][1] = -2.0f * kY2c * y; G[8][2] = 0.0f;
    if (DEG < 3) return;
    Y[9] = -kY3a * y * (3.0f * xx - yy);
    G[9][0] = -6.0f * kY3a * x * y; G[9][1] = -3.0f * kY3a * (xx - yy); G[9][2] = 0.0f;
    Y[10] = kY3b * x * y * z;
    G[10][0] = kY3b * y * z; G[10][1] = kY3b * x * z; G[10][2] = kY3b * x * y;
    Y[11] = -kY3c * y * (4.0f * zz - xx - yy);
    G[11][0] = 2.0f * kY3c * x * y; G[11][1] = -kY3c * (4.0f * zz - xx - 3.0f * yy); G[11][2] = -8.0f * kY3c * y * z;
    Y[12] = kY3d * z * (2.0f * zz - 3.0f * xx - 3.0f * yy);
    G[12][0] = -6.0f * kY3d * x * z; G[12][1] = -6.0f * kY3d * y * z; G[12][2] = kY3d * (6.0f * zz - 3.0f * xx - 3.0f * yy);
    Y[13] = -kY3c * x * (4.0f * zz - xx - yy);
    G[13][0] = -kY3c * (4.0f * zz - 3.0f * xx - yy); G[13][1] = 2.0f * kY3c * x * y; G[13][2] = -8.0f * kY3c * x * z;
    Y[14] = kY3e * z * (xx - yy);
    G[14][0] = 2.0f * kY3e * x * z; G[14][1] = -2.0f * kY3e * y * z; G[14][2] = kY3e * (xx - yy);
    Y[15] = -kY3a * x * (xx - 3.0f * yy);
    G[15][0] = -3.0f * kY3a * (xx - yy); G[15][1] = 6.0f * kY3a * x * y; G[15][2] = 0.0f;
}

__device__ __forceinline__ float dot3(const float* a, const float* b) { return a[0] * b[0] + a[1] * b[1] + a[2] * b[2]; }

// Per-primitive work: k_project_bwd, one thread per visible row, adds the
// primitive's pair slots and applies the chain rule.

template <int DEG>
struct RowLayout {
    static constexpr int K = (DEG + 1) * (DEG + 1);
    static constexpr int SH = 3 * K;
    static constexpr int ROW = 11 + SH;                        // mean 3, log_scale 3, quat 4, opacity 1, sh
    static constexpr int ROW4 = (ROW + 3) / 4 * 4;
};

// Chain rule from one primitive's 2D gradient (du, dv, dA, dB, dC in g2) back
// to mean, log-scale and quaternion, evaluated in scalar type Rl.  gpw
// receives the projection path's camera-space mean gradient (the world-space
// one is R^T gpw, formed by the caller together with the colour path's part);
// out receives log_scale (3..5) and quat (6..9) gradients.
template <typename Rl>
__device__ __forceinline__ void geometry_bwd(const float* mu_f, const float* ls_f, const float* qr_f,
                                             const float* g2, const CamArgs& c, Rl* gpw, float* out) {
    Rl R[9];
#pragma unroll
    for (int k = 0; k < 9; ++k) R[k] = (Rl)c.R[k];
    const Rl mu[3] = {(Rl)mu_f[0], (Rl)mu_f[1], (Rl)mu_f[2]};
    const Rl fx = (Rl)c.fx, fy = (Rl)c.fy;
    Rl p[3];
#pragma unroll
    for (int k = 0; k < 3; ++k) p[k] = R[3 * k] * mu[0] + R[3 * k + 1] * mu[1] + R[3 * k + 2] * mu[2] + (Rl)c.t[k];
    const Rl s[3] = {exp((Rl)ls_f[0]), exp((Rl)ls_f[1]), exp((Rl)ls_f[2])};
    const Rl q0 = (Rl)qr_f[0], q1 = (Rl)qr_f[1], q2 = (Rl)qr_f[2], q3 = (Rl)qr_f[3];
    const Rl iq = (Rl)1 / sqrt(q0 * q0 + q1 * q1 + q2 * q2 + q3 * q3);
    const Rl w = q0 * iq, x = q1 * iq, y = q2 * iq, z = q3 * iq;
    const Rl Rq[3][3] = {{1 - 2 * (y * y + z * z), 2 * (x * y - w * z), 2 * (x * z + w * y)},
                         {2 * (x * y + w * z), 1 - 2 * (x * x + z * z), 2 * (y * z - w * x)},
                         {2 * (x * z - w * y), 2 * (y * z + w * x), 1 - 2 * (x * x + y * y)}};
    Rl M[3][3], Sg[3][3];
#pragma unroll
    for (int a = 0; a < 3; ++a)
#pragma unroll
        for (int b = 0; b < 3; ++b) M[a][b] = Rq[a][b] * s[b];
#pragma unroll
    for (int a = 0; a < 3; ++a)
#pragma unroll
        for (int b = 0; b < 3; ++b) Sg[a][b] = M[a][0] * M[b][0] + M[a][1] * M[b][1] + M[a][2] * M[b][2];
    const Rl tz = p[2], itz = (Rl)1 / tz;
    const Rl lx = (Rl)(1.3f * c.tan_fovx), ly = (Rl)(1.3f * c.tan_fovy);
    const Rl rx = p[0] * itz, ry = p[1] * itz;
    const bool clx = rx < -lx || rx > lx, cly = ry < -ly || ry > ly;
    const Rl xr = rx < -lx ? -lx : (rx > lx ? lx : rx);
    const Rl yr = ry < -ly ? -ly : (ry > ly ? ly : ry);
    const Rl j00 = fx * itz, j11 = fy * itz;
    const Rl j02 = -fx * xr * itz, j12 = -fy * yr * itz;
    Rl T0[3], T1[3];
#pragma unroll
    for (int k = 0; k < 3; ++k) {
        T0[k] = j00 * R[k] + j02 * R[6 + k];
        T1[k] = j11 * R[3 + k] + j12 * R[6 + k];
    }
    Rl ST0[3], ST1[3];   // Sigma T0, Sigma T1
#pragma unroll
    for (int a = 0; a < 3; ++a) {
        ST0[a] = Sg[a][0] * T0[0] + Sg[a][1] * T0[1] + Sg[a][2] * T0[2];
        ST1[a] = Sg[a][0] * T1[0] + Sg[a][1] * T1[1] + Sg[a][2] * T1[2];
    }
    const Rl ca = T0[0] * ST0[0] + T0[1] * ST0[1] + T0[2] * ST0[2] + (Rl)0.3f;
    const Rl cb = T0[0] * ST1[0] + T0[1] * ST1[1] + T0[2] * ST1[2];
    const Rl cc = T1[0] * ST1[0] + T1[1] * ST1[1] + T1[2] * ST1[2] + (Rl)0.3f;
    const Rl det = ca * cc - cb * cb;
    const Rl id2 = (Rl)1 / (det * det);
    // conic (A,B,C) = (c, -b, a)/det  ->  gradient w.r.t. (a, b, c)
    const Rl gA = g2[2], gB = g2[3], gC = g2[4];
    const Rl ga = (-gA * cc * cc + gB * cb * cc - gC * cb * cb) * id2;
    const Rl gb = (2 * gA * cb * cc - gB * (ca * cc + cb * cb) + 2 * gC * ca * cb) * id2;
    const Rl gcv = (-gA * cb * cb + gB * ca * cb - gC * ca * ca) * id2;
    // a = T0.S.T0, b = T0.S.T1, c = T1.S.T1
    Rl gT0[3], gT1[3];
#pragma unroll
    for (int a = 0; a < 3; ++a) {
        gT0[a] = 2 * ga * ST0[a] + gb * ST1[a];
        gT1[a] = gb * ST0[a] + 2 * gcv * ST1[a];
    }
    const Rl gj00 = gT0[0] * R[0] + gT0[1] * R[1] + gT0[2] * R[2];
    const Rl gj02 = gT0[0] * R[6] + gT0[1] * R[7] + gT0[2] * R[8];
    const Rl gj11 = gT1[0] * R[3] + gT1[1] * R[4] + gT1[2] * R[5];
    const Rl gj12 = gT1[0] * R[6] + gT1[1] * R[7] + gT1[2] * R[8];
    const Rl itz2 = itz * itz;
    Rl gp[3] = {0, 0, 0};
    gp[2] -= (gj00 * fx + gj11 * fy) * itz2;
    if (clx) {
        gp[2] += gj02 * fx * xr * itz2;
    } else {
        gp[0] -= gj02 * fx * itz2;
        gp[2] += 2 * gj02 * fx * p[0] * itz2 * itz;
    }
    if (cly) {
        gp[2] += gj12 * fy * yr * itz2;
    } else {
        gp[1] -= gj12 * fy * itz2;
        gp[2] += 2 * gj12 * fy * p[1] * itz2 * itz;
    }
    const Rl gu = g2[0], gv = g2[1];
    gp[0] += gu * fx * itz;
    gp[1] += gv * fy * itz;
    gp[2] -= (gu * fx * p[0] + gv * fy * p[1]) * itz2;
    gpw[0] = gp[0];
    gpw[1] = gp[1];
    gpw[2] = gp[2];
    // Sigma = M M^T with symmetric gradient Gs = ga T0T0^T + gb (T0T1^T + T1T0^T)/2 + gc T1T1^T
    Rl Gs[3][3];
#pragma unroll
    for (int a = 0; a < 3; ++a)
#pragma unroll
        for (int b = 0; b < 3; ++b)
            Gs[a][b] = ga * T0[a] * T0[b] + (Rl)0.5 * gb * (T0[a] * T1[b] + T1[a] * T0[b]) + gcv * T1[a] * T1[b];
    Rl gR[3][3];
#pragma unroll
    for (int b = 0; b < 3; ++b) {
        Rl gsb = 0;
#pragma unroll
        for (int a = 0; a < 3; ++a) {
            const Rl gM = 2 * (Gs[a][0] * M[0][b] + Gs[a][1] * M[1][b] + Gs[a][2] * M[2][b]);
            gR[a][b] = gM * s[b];
            gsb += gM * Rq[a][b];
        }
        out[3 + b] = (float)(gsb * s[b]);
    }
    const Rl gw = 2 * (x * (gR[2][1] - gR[1][2]) + y * (gR[0][2] - gR[2][0]) + z * (gR[1][0] - gR[0][1]));
    const Rl gx = 2 * (w * (gR[2][1] - gR[1][2]) - 2 * x * (gR[1][1] + gR[2][2]) + y * (gR[0][1] + gR[1][0]) +
                       z * (gR[0][2] + gR[2][0]));
    const Rl gy = 2 * (w * (gR[0][2] - gR[2][0]) + x * (gR[0][1] + gR[1][0]) - 2 * y * (gR[0][0] + gR[2][2]) +
                       z * (gR[1][2] + gR[2][1]));
    const Rl gz = 2 * (w * (gR[1][0] - gR[0][1]) + x * (gR[0][2] + gR[2][0]) + y * (gR[1][2] + gR[2][1]) -
                       2 * z * (gR[0][0] + gR[1][1]));
    const Rl along = w * gw + x * gx + y * gy + z * gz;
    out[6] = (float)((gw - w * along) * iq);
    out[7] = (float)((gx - x * along) * iq);
    out[8] = (float)((gy - y * along) * iq);
    out[9] = (float)((gz - z * along) * iq);
}

// Lists of up to kSerialSlots slots are summed by their own thread; longer
// ones (a primitive spanning many tiles) by the whole wave, 256 slots a
// round.  Either way the order is fixed, so the result is deterministic.
constexpr uint32_t kSerialSlots = 8;

template <int N>
__device__ __forceinline__ void load_row(const float* __restrict__ src, float* dst) {
    if constexpr (N % 4 == 0) {
        const float4* s4 = reinterpret_cast<const float4*>(src);
#pragma unroll
        for (int k = 0; k < N / 4; ++k) {
            const float4 v = s4[k];
            dst[4 * k] = v.x; dst[4 * k + 1] = v.y; dst[4 * k + 2] = v.z; dst[4 * k + 3] = v.w;
        }
    } else {
#pragma unroll
        for (int k = 0; k < N; ++k) dst[k] = src[k];
    }
}

// Position of id in the ascending list u[0..m), or m if absent.
__device__ __forceinline__ uint32_t find_row(const uint32_t* __restrict__ u, uint32_t m, uint32_t id) {
    uint32_t lo = 0, hi = m;
    while (lo < hi) {
        const uint32_t mid = (lo + hi) >> 1;
        if (u[mid] < id) lo = mid + 1; else hi = mid;
    }
    return (lo < m && u[lo] == id) ? lo : m;
}

// Per visible row r: the sum of the primitive's pair slots (emission
// positions pair_offset[id] .. + tiles[id], side by side; none if the pair
// list overflowed its capacity), as one kSlot-float row at sums + kSlot r.
// A kernel of its own: the chain rule's registers would leave the slot
// stream too few waves to keep its loads in flight.
__global__ void __launch_bounds__(GS_BLOCK) k_slot_sum(const uint32_t* __restrict__ vis_idx,
                                                       const uint32_t* __restrict__ vis_count,
                                                       const uint32_t* __restrict__ tiles,
                                                       const uint32_t* __restrict__ pair_offset,
                                                       const float* __restrict__ slots, uint32_t capacity,
                                                       float* __restrict__ sums) {
    const uint32_t V = *vis_count;
    // Rows in chunks of 16 consecutive ones (neighbouring rows' slots share
    // cache lines); workgroup b takes chunks b, b + NB, b + 2 NB, ... (NB the
    // workgroups needed), so a wave's four chunks lie across the whole list.
    // In a spatially ordered pool the long slot lists of neighbours near the
    // camera come in runs; taken whole by one wave they would be summed one
    // after the other while the rest of the chip idles.
    const uint32_t nb = (V + GS_BLOCK - 1) / GS_BLOCK;
    if (blockIdx.x >= nb) return;
    const uint32_t r = ((threadIdx.x >> 4) * nb + blockIdx.x) * 16u + (threadIdx.x & 15u);
    const bool valid = r < V;
    const uint32_t id = valid ? vis_idx[r] : 0u;
    float g2[kG] = {0, 0, 0, 0, 0, 0, 0, 0, 0};
    const uint32_t first = valid ? pair_offset[id] : 0u;
    const uint32_t nt = valid ? tiles[id] : 0u;
    const bool fits = (uint64_t)first + nt <= capacity;
    if (fits && nt <= kSerialSlots) {
        // up to four slots per round, all loads in flight
        for (uint32_t k = 0; k < nt; k += 4) {
            float4 v[4][3];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const uint32_t q = first + min(k + j, nt - 1u);     // past the list: the last slot again, unused
                const float4* sl = reinterpret_cast<const float4*>(slots + (size_t)q * kSlot);
                v[j][0] = sl[0]; v[j][1] = sl[1]; v[j][2] = sl[2];
            }
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                if (k + j < nt) {
                    g2[0] += v[j][0].x; g2[1] += v[j][0].y; g2[2] += v[j][0].z; g2[3] += v[j][0].w;
                    g2[4] += v[j][1].x; g2[5] += v[j][1].y; g2[6] += v[j][1].z; g2[7] += v[j][1].w;
                    g2[8] += v[j][2].x;
                }
            }
        }
    }
    // longer lists: the whole wave, 4 x 64 slots per round with coalesced loads,
    // the lanes' partial sums added in a fixed order
    uint64_t big = __ballot(fits && nt > kSerialSlots);
    while (big) {
        const int owner = __ffsll((unsigned long long)big) - 1;
        big &= big - 1;
        const uint32_t f = (uint32_t)__builtin_amdgcn_readlane((int)first, owner);
        const uint32_t nb2 = (uint32_t)__builtin_amdgcn_readlane((int)nt, owner);
        float acc[kG] = {0, 0, 0, 0, 0, 0, 0, 0, 0};
        for (uint32_t k0 = 0; k0 < nb2; k0 += 4 * GS_WAVE) {
            float4 v[4][3];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const uint32_t k = min(k0 + j * GS_WAVE + lane_id(), nb2 - 1u);
                const float4* sl = reinterpret_cast<const float4*>(slots + (size_t)(f + k) * kSlot);
                v[j][0] = sl[0]; v[j][1] = sl[1]; v[j][2] = sl[2];
            }
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                if (k0 + j * GS_WAVE + lane_id() < nb2) {
                    acc[0] += v[j][0].x; acc[1] += v[j][0].y; acc[2] += v[j][0].z; acc[3] += v[j][0].w;
                    acc[4] += v[j][1].x; acc[5] += v[j][1].y; acc[6] += v[j][1].z; acc[7] += v[j][1].w;
                    acc[8] += v[j][2].x;
                }
            }
        }
#pragma unroll
        for (int q = 0; q < kG; ++q) {
            const float sv = wave_sum(acc[q]);
            if (lane_id() == owner) g2[q] = sv;
        }
    }
    if (!valid) return;
    float4* dst = reinterpret_cast<float4*>(sums + (size_t)r * kSlot);
    dst[0] = make_float4(g2[0], g2[1], g2[2], g2[3]);
    dst[1] = make_float4(g2[4], g2[5], g2[6], g2[7]);
    dst[2] = make_float4(g2[8], 0.0f, 0.0f, 0.0f);
}

// Per visible row r: the primitive's 2D gradient (from its slot sums, row r
// of k_slot_sum), then the chain rule to the parameters; writes the row's
// gradient record at grad_rows + r * ld.  ACCUM (a task unit
// of several views): the record is added to row u instead, u the position of
// id in the unit's ascending union list, and |dL/d(u,v)| is added to
// grad_norm[id].
template <int DEG, bool ACCUM>
__global__ void __launch_bounds__(GS_BLOCK) k_project_bwd(
    const uint32_t* __restrict__ vis_idx, const uint32_t* __restrict__ vis_count, const float* __restrict__ sums,
    const float4* __restrict__ conic_op, const uint8_t* __restrict__ clampm, const float* __restrict__ mean, const float* __restrict__ log_scale,
    const float* __restrict__ quat, const float* __restrict__ opacity, const float* __restrict__ sh, SceneLd pld,
    CamArgs c, float* __restrict__ grad_rows, int32_t ld, float* __restrict__ grad2d, float* __restrict__ grad_norm,
    const uint32_t* __restrict__ union_idx, const uint32_t* __restrict__ union_count) {
    using L = RowLayout<DEG>;
    constexpr int K = L::K;
    const uint32_t V = *vis_count;
    const uint32_t r = blockIdx.x * GS_BLOCK + threadIdx.x;
    if (r >= V) return;
    const uint32_t id = vis_idx[r];
    float g2[kG];
    {
        const float4* src = reinterpret_cast<const float4*>(sums + (size_t)r * kSlot);
        const float4 a0 = src[0], a1 = src[1], a2 = src[2];
        g2[0] = a0.x; g2[1] = a0.y; g2[2] = a0.z; g2[3] = a0.w;
        g2[4] = a1.x; g2[5] = a1.y; g2[6] = a1.z; g2[7] = a1.w; g2[8] = a2.x;
    }
    {
        // moments -> 2D gradient, with the conic the pixels used; fp64 because
        // A m_x and B m_y can nearly cancel for elongated footprints
        const float4 co = conic_op[id];
        const double mx = g2[0], my = g2[1];
        g2[0] = (float)((double)co.x * mx + (double)co.y * my);
        g2[1] = (float)((double)co.y * mx + (double)co.z * my);
        g2[2] = 0.5f * g2[2];
        g2[4] = 0.5f * g2[4];
        g2[5] = co.w > 0.0f ? -g2[5] / co.w : 0.0f;
    }
    uint32_t row = r;
    if (ACCUM) {
        const uint32_t m = *union_count;
        row = find_row(union_idx, m, id);
        if (row == m) return;                 // not in the unit's union: nothing to add to
    }
    if (grad2d) {
#pragma unroll
        for (int q = 0; q < kG; ++q) grad2d[(size_t)id * kG + q] = g2[q];
    }
    if (grad_norm) {
        const float gn = sqrtf(g2[0] * g2[0] + g2[1] * g2[1]);
        grad_norm[id] = ACCUM ? grad_norm[id] + gn : gn;
    }
    float mu[3], ls[3], qr[4];
    load_row<3>(mean + (size_t)id * pld.mean, mu);
    load_row<4>(quat + (size_t)id * pld.quat, qr);
    float logit;
    if (pld.head) {
        float h[4];
        load_row<4>(quat + (size_t)id * pld.quat + 4, h);
        ls[0] = h[0]; ls[1] = h[1]; ls[2] = h[2]; logit = h[3];
    } else {
        load_row<3>(log_scale + (size_t)id * pld.log_scale, ls);
        logit = opacity[(size_t)id * pld.opacity];
    }
    const uint8_t cm = clampm[id];
    float out[L::ROW4];

    // 1. geometry, in fp64: for wide footprints the conic gradient is large
    //    while the scale / rotation gradients it produces are tiny, and the
    //    chain cancels too much for fp32
    double gp[3];
    geometry_bwd<double>(mu, ls, qr, g2, c, gp, out);

    // 2. opacity
    const float o = 1.0f / (1.0f + expf(-logit));
    out[10] = g2[5] * o * (1.0f - o);

    // 3. colour: dL/dsh and the view-direction path to the mean
    float gmu[3];
    {
        float v[3] = {mu[0] - c.campos[0], mu[1] - c.campos[1], mu[2] - c.campos[2]};
        const float len = sqrtf(dot3(v, v));
        const float il = 1.0f / len;
        const float d[3] = {v[0] * il, v[1] * il, v[2] * il};
        float Y[16], G[16][3];
        sh_basis_grad<DEG>(d[0], d[1], d[2], Y, G);
        const float gc[3] = {(cm & 1) ? 0.0f : g2[6], (cm & 2) ? 0.0f : g2[7], (cm & 4) ? 0.0f : g2[8]};
        float co[3 * K];
        load_row<3 * K>(sh + (size_t)id * pld.sh, co);
        float gd[3] = {0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int k = 0; k < K; ++k) {
            const float a = gc[0] * co[3 * k] + gc[1] * co[3 * k + 1] + gc[2] * co[3 * k + 2];
            gd[0] += a * G[k][0];
            gd[1] += a * G[k][1];
            gd[2] += a * G[k][2];
            out[11 + 3 * k + 0] = gc[0] * Y[k];
            out[11 + 3 * k + 1] = gc[1] * Y[k];
            out[11 + 3 * k + 2] = gc[2] * Y[k];
        }
        const float rad = dot3(gd, d);
        gmu[0] = (gd[0] - d[0] * rad) * il;
        gmu[1] = (gd[1] - d[1] * rad) * il;
        gmu[2] = (gd[2] - d[2] * rad) * il;
    }
#pragma unroll
    for (int k = 0; k < 3; ++k)
        out[k] = (float)((double)gmu[k] + (double)c.R[k] * gp[0] + (double)c.R[3 + k] * gp[1] +
                         (double)c.R[6 + k] * gp[2]);
#pragma unroll
    for (int k = L::ROW; k < L::ROW4; ++k) out[k] = 0.0f;

    float4* dst = reinterpret_cast<float4*>(grad_rows + (size_t)row * ld);
    if (ACCUM) {
#pragma unroll
        for (int k = 0; k < L::ROW4 / 4; ++k) {
            const float4 a = dst[k];
            dst[k] = make_float4(a.x + out[4 * k], a.y + out[4 * k + 1], a.z + out[4 * k + 2], a.w + out[4 * k + 3]);
        }
        return;
    }
#pragma unroll
    for (int k = 0; k < L::ROW4 / 4; ++k) dst[k] = make_float4(out[4 * k], out[4 * k + 1], out[4 * k + 2], out[4 * k + 3]);
    for (int k = L::ROW4 / 4; k < ld / 4; ++k) dst[k] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
}

// First view of a task unit: the union's gradient rows (all ld columns) and
// the grad_norm entries of its ids start at zero.
__global__ void __launch_bounds__(GS_BLOCK) k_clear_union_rows(const uint32_t* __restrict__ union_idx,
                                                               const uint32_t* __restrict__ union_count,
                                                               float* __restrict__ grad_rows, int32_t ld,
                                                               float* __restrict__ grad_norm) {
    const uint32_t m = *union_count;
    const uint32_t q4 = (uint32_t)ld / 4;
    const uint64_t total = (uint64_t)m * q4;
    float4* rows = reinterpret_cast<float4*>(grad_rows);
    for (uint64_t i = (uint64_t)blockIdx.x * GS_BLOCK + threadIdx.x; i < total; i += (uint64_t)gridDim.x * GS_BLOCK) {
        rows[i] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
        if (grad_norm && i % q4 == 0) grad_norm[union_idx[i / q4]] = 0.0f;
    }
}

}  // namespace

hipError_t launch_raster_fwd(const gs_proj& proj, const uint32_t* vals, const uint32_t* ranges,
                             const uint32_t* tile_order, int32_t width, int32_t height, const float bg[3],
                             float* img, float* final_T, uint32_t* n_contrib, uint8_t* active, uint64_t* pair_stats,
                             hipStream_t st) {
    const int32_t TX = (width + GS_TILE - 1) / GS_TILE, TY = (height + GS_TILE - 1) / GS_TILE;
    if (TX * TY == 0) return hipSuccess;
    if (pair_stats)
        hipLaunchKernelGGL((k_raster_fwd<true, false>), dim3(TX * TY), dim3(GS_BLOCK), 0, st, tile_order, ranges, vals,
                           reinterpret_cast<const float2*>(proj.mean2d),
                           reinterpret_cast<const float4*>(proj.conic_opacity), proj.rgb, width, height, TX, bg[0],
                           bg[1], bg[2], img, final_T, n_contrib, active,
                           reinterpret_cast<unsigned long long*>(pair_stats), nullptr, 0.0f, nullptr, nullptr);
    else
        hipLaunchKernelGGL((k_raster_fwd<false, false>), dim3(TX * TY), dim3(GS_BLOCK), 0, st, tile_order, ranges, vals,
                           reinterpret_cast<const float2*>(proj.mean2d),
                           reinterpret_cast<const float4*>(proj.conic_opacity), proj.rgb, width, height, TX, bg[0],
                           bg[1], bg[2], img, final_T, n_contrib, active, nullptr, nullptr, 0.0f, nullptr, nullptr);
    return hipGetLastError();
}

size_t raster_fwd_l1_ws_bytes(int32_t width, int32_t height) {
    const uint64_t T = (uint64_t)div_up((uint64_t)(width > 0 ? width : 0), GS_TILE) *
                       div_up((uint64_t)(height > 0 ? height : 0), GS_TILE);
    return align256(sizeof(float) * (T + 1));
}

hipError_t launch_raster_fwd_l1(const gs_proj& proj, const uint32_t* vals, const uint32_t* ranges,
                                const uint32_t* tile_order, int32_t width, int32_t height, const float bg[3],
                                const float* target, float* img, float* final_T, uint32_t* n_contrib, uint8_t* active,
                                float* loss, float* dL, void* ws, hipStream_t st) {
    const int32_t TX = (width + GS_TILE - 1) / GS_TILE, TY = (height + GS_TILE - 1) / GS_TILE;
    const uint64_t total = 3ull * (uint64_t)width * (uint64_t)height;
    float* partial = static_cast<float*>(ws);
    if (TX * TY > 0)
        hipLaunchKernelGGL((k_raster_fwd<false, true>), dim3(TX * TY), dim3(GS_BLOCK), 0, st, tile_order, ranges, vals,
                           reinterpret_cast<const float2*>(proj.mean2d),
                           reinterpret_cast<const float4*>(proj.conic_opacity), proj.rgb, width, height, TX, bg[0],
                           bg[1], bg[2], img, final_T, n_contrib, active, nullptr, target,
                           (float)(1.0 / (double)(total ? total : 1)), dL, partial);
    hipLaunchKernelGGL(k_loss_final, dim3(1), dim3(GS_BLOCK), 0, st, partial, (uint32_t)(TX * TY),
                       total ? 1.0 / (double)total : 0.0, loss);
    return hipGetLastError();
}

size_t loss_ws_bytes(int32_t width, int32_t height) {
    return align256(sizeof(float) * (div_up(3ull * (uint64_t)width * (uint64_t)height, GS_TILE_ITEMS) + 1));
}

hipError_t launch_loss_l1(const float* img, const float* target, int32_t width, int32_t height, float* loss,
                          float* dL, void* ws, hipStream_t st) {
    const uint64_t total = 3ull * (uint64_t)width * (uint64_t)height;
    const uint32_t nb = div_up(total, GS_TILE_ITEMS);
    float* partial = static_cast<float*>(ws);
    const float inv = (float)(1.0 / (double)total);
    if (nb > 0)
    {
        const bool vec = ((reinterpret_cast<uintptr_t>(img) | reinterpret_cast<uintptr_t>(target) |
                           reinterpret_cast<uintptr_t>(dL)) & 15u) == 0;
        if (vec)
            hipLaunchKernelGGL(k_loss_l1<true>, dim3(nb), dim3(GS_BLOCK), 0, st, img, target, (uint32_t)total, inv,
                               dL, partial);
        else
            hipLaunchKernelGGL(k_loss_l1<false>, dim3(nb), dim3(GS_BLOCK), 0, st, img, target, (uint32_t)total, inv,
                               dL, partial);
    }
    hipLaunchKernelGGL(k_loss_final, dim3(1), dim3(GS_BLOCK), 0, st, partial, nb,
                       total ? 1.0 / (double)total : 0.0, loss);
    return hipGetLastError();
}

// Workspace: the pair slots (capacity x kSlot floats), then the slot sums of
// the visible rows (n x kSlot floats; the pixel half alone needs only the
// slots, n = 0).
size_t raster_bwd_ws_bytes(int32_t n, uint32_t capacity) {
    return align256(sizeof(float) * kSlot * (size_t)(capacity > 0 ? capacity : 1)) +
           (n > 0 ? align256(sizeof(float) * kSlot * (size_t)n) : 0);
}

hipError_t launch_raster_bwd(const gs_scene& scene, const CamArgs& cam, const gs_proj& proj, const uint32_t* vals,
                             const uint32_t* ranges, const uint32_t* tile_order, const uint32_t* pair_offset,
                             const uint32_t* pair_emit, const uint32_t* vis_idx, const uint32_t* vis_count,
                             uint32_t capacity, const float* final_T, const uint32_t* n_contrib, const float* dL_dimg,
                             const float bg[3], float* grad_rows, int32_t grad_ld, float* grad2d, float* grad_norm,
                             void* ws, int stages, hipStream_t st, const uint32_t* union_idx, const uint32_t* union_count, int first) {
    float* slots = static_cast<float*>(ws);
    const int32_t T = cam.tiles_x * cam.tiles_y;
    if ((stages & 1) && T > 0)
        hipLaunchKernelGGL(k_raster_bwd, dim3(T), dim3(GS_BLOCK), 0, st, tile_order, ranges, vals,
                           reinterpret_cast<const float2*>(proj.mean2d),
                           reinterpret_cast<const float4*>(proj.conic_opacity), proj.rgb, cam.width, cam.height,
                           cam.tiles_x, bg[0], bg[1], bg[2], final_T, n_contrib, dL_dimg, pair_emit, slots);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || scene.n == 0 || !(stages & 2)) return e;
    const dim3 grid(div_up(scene.n, GS_BLOCK));
    float* sums = slots + align256(sizeof(float) * kSlot * (size_t)(capacity > 0 ? capacity : 1)) / sizeof(float);
    hipLaunchKernelGGL(k_slot_sum, grid, dim3(GS_BLOCK), 0, st, vis_idx, vis_count, proj.tiles, pair_offset, slots,
                       capacity, sums);
    if (union_idx) {
        if (first) {
            uint32_t cb = div_up((uint64_t)scene.n * (uint64_t)(grad_ld / 4), GS_BLOCK);
            if (cb > 8192) cb = 8192;
            hipLaunchKernelGGL(k_clear_union_rows, dim3(cb), dim3(GS_BLOCK), 0, st, union_idx, union_count, grad_rows,
                               grad_ld, grad_norm);
        }
    }
#define GS_LAUNCH_PBWD(D, A)                                                                                     \
    hipLaunchKernelGGL((k_project_bwd<D, A>), grid, dim3(GS_BLOCK), 0, st, vis_idx, vis_count, sums,             \
                       reinterpret_cast<const float4*>(proj.conic_opacity),                                       \
                       proj.clamp, scene.mean, scene.log_scale, scene.quat, scene.opacity, scene.sh,              \
                       scene_ld(scene), cam,                                                                      \
                       grad_rows, grad_ld, grad2d, grad_norm, union_idx, union_count)
    if (union_idx) {
        switch (scene.sh_degree) {
            case 0: GS_LAUNCH_PBWD(0, true); break;
            case 1: GS_LAUNCH_PBWD(1, true); break;
            case 2: GS_LAUNCH_PBWD(2, true); break;
            default: GS_LAUNCH_PBWD(3, true); break;
        }
    } else {
        switch (scene.sh_degree) {
            case 0: GS_LAUNCH_PBWD(0, false); break;
            case 1: GS_LAUNCH_PBWD(1, false); break;
            case 2: GS_LAUNCH_PBWD(2, false); break;
            default: GS_LAUNCH_PBWD(3, false); break;
        }
    }
#undef GS_LAUNCH_PBWD
    return hipGetLastError();
}

}  // namespace gsmi
