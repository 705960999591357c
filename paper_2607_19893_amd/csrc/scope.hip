// Primitive scopes as bitmaps over primitive ids (bit i & 31 of word i >> 5),
// the quality-first hazard sets between an earlier task unit A and a later
// unit B, and the throughput-first admission of B's delayed reads.
//
// Hazards, per bitmap word (one thread per word):
//   WAW = W(B) & W(A),  RAW = R(B) & ~W(B) & W(A),  WAR = W(B) & R(A) & ~W(A)
// Three launches: per-block popcounts, one workgroup that turns them into
// per-block offsets and totals, and the scatter of ascending ids (skipped
// when no id list is asked for).
//
// Admission, for the delayed set D = RAW: per-block partial counts
// (|R(B)|, |D|, |C_A|, delayed ids without evidence, delayed ids whose
// publication metadata names another producer), the fp64 sum of ||g_A|| over
// C_A and the largest ||g_A|| over D; one workgroup reduces the partials in a
// fixed order and takes the decision in fp64; a last launch stamps the
// producer version into the metadata of the delayed ids when admitted.  The
// ||g_A|| gathers are done one id per lane (coalesced), with each lane taking
// its bit from the word of a neighbouring lane.
#include "common.h"
#include "internal.h"

namespace gsmi {

namespace {

constexpr int kWordsPerBlock = GS_BLOCK;   // one word (32 ids) per thread

__device__ __forceinline__ uint32_t tail_mask(uint32_t w, uint32_t nwords, int32_t n) {
    if (w + 1 < nwords) return 0xFFFFFFFFu;
    const uint32_t r = (uint32_t)n & 31u;
    return r ? ((1u << r) - 1u) : 0xFFFFFFFFu;
}

__device__ __forceinline__ uint32_t load_word(const uint32_t* __restrict__ s, uint32_t w, uint32_t nwords,
                                              uint32_t mask) {
    return (w < nwords) ? (s[w] & mask) : 0u;
}

// ---------------------------------------------------------------------------
// building scopes
// ---------------------------------------------------------------------------

__global__ void __launch_bounds__(GS_BLOCK) k_scope_from_ids(const uint32_t* __restrict__ idx,
                                                             const uint32_t* __restrict__ count, int32_t max_rows,
                                                             int32_t n, uint32_t* __restrict__ scope) {
    const uint32_t k = min(*count, (uint32_t)max_rows);
    for (uint32_t i = blockIdx.x * GS_BLOCK + threadIdx.x; i < k; i += gridDim.x * GS_BLOCK) {
        const uint32_t id = idx[i];
        if (id < (uint32_t)n) atomicOr(&scope[id >> 5], 1u << (id & 31u));
    }
}

// One id per lane: a wave's ballot is two words of the bitmap.
template <int KIND>
__global__ void __launch_bounds__(GS_BLOCK) k_scope_from_pred(const void* __restrict__ src, int32_t n,
                                                              int32_t accumulate, uint32_t* __restrict__ scope) {
    const uint32_t i = blockIdx.x * GS_BLOCK + threadIdx.x;
    bool on = false;
    if (i < (uint32_t)n) {
        if (KIND == GS_PRED_U32_NONZERO)
            on = static_cast<const uint32_t*>(src)[i] != 0u;
        else
            on = static_cast<const uint8_t*>(src)[i] != 0u;
    }
    const uint64_t m = __ballot(on);
    const uint32_t w0 = i >> 5;                 // even word of this wave's pair (lane 0's word)
    const uint32_t nwords = ((uint32_t)n + 31u) >> 5;
    const int lane = lane_id();
    if (lane < 2 && w0 + lane < nwords) {
        const uint32_t v = lane == 0 ? (uint32_t)m : (uint32_t)(m >> 32);
        scope[w0 + lane] = accumulate ? (scope[w0 + lane] | v) : v;
    }
}

// ---------------------------------------------------------------------------
// hazard sets
// ---------------------------------------------------------------------------

struct ScopeIn {
    const uint32_t* RA;
    const uint32_t* WA;
    const uint32_t* RB;
    const uint32_t* WB;
};

struct Hazards {
    uint32_t waw, raw, war, rb;
};

__device__ __forceinline__ Hazards hazard_words(const ScopeIn& s, uint32_t w, uint32_t nwords, int32_t n) {
    const uint32_t mask = tail_mask(w, nwords, n);
    const uint32_t ra = load_word(s.RA, w, nwords, mask), wa = load_word(s.WA, w, nwords, mask);
    const uint32_t rb = load_word(s.RB, w, nwords, mask), wb = load_word(s.WB, w, nwords, mask);
    Hazards h;
    h.waw = wb & wa;
    h.raw = rb & ~wb & wa;
    h.war = wb & ra & ~wa;
    h.rb = rb;
    return h;
}

__global__ void __launch_bounds__(GS_BLOCK) k_hazard_count(ScopeIn s, int32_t n, uint32_t nwords,
                                                           uint32_t* __restrict__ waw_out,
                                                           uint32_t* __restrict__ raw_out,
                                                           uint32_t* __restrict__ war_out,
                                                           uint32_t* __restrict__ partial) {
    __shared__ uint32_t scratch[4];
    const uint32_t w = blockIdx.x * kWordsPerBlock + threadIdx.x;
    const Hazards h = hazard_words(s, w, nwords, n);
    if (w < nwords) {
        if (waw_out) waw_out[w] = h.waw;
        if (raw_out) raw_out[w] = h.raw;
        if (war_out) war_out[w] = h.war;
    }
    const uint32_t c0 = block_sum_u32(__popc(h.waw), scratch);
    const uint32_t c1 = block_sum_u32(__popc(h.raw), scratch);
    const uint32_t c2 = block_sum_u32(__popc(h.war), scratch);
    const uint32_t c3 = block_sum_u32(__popc(h.rb), scratch);
    if (threadIdx.x == 0) {
        partial[4 * blockIdx.x + 0] = c0;
        partial[4 * blockIdx.x + 1] = c1;
        partial[4 * blockIdx.x + 2] = c2;
        partial[4 * blockIdx.x + 3] = c3;
    }
}

// One workgroup: exclusive offsets of the three id lists per block (in
// place, fields 0..2 of each record) and the totals.
__global__ void __launch_bounds__(GS_BLOCK) k_hazard_offsets(uint32_t* __restrict__ partial, uint32_t nb,
                                                             uint32_t* __restrict__ counts) {
    __shared__ uint32_t scratch[4];
    uint32_t carry[4] = {0u, 0u, 0u, 0u};
    for (uint32_t c0 = 0; c0 < nb; c0 += GS_BLOCK) {
        const uint32_t b = c0 + threadIdx.x;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const uint32_t v = b < nb ? partial[4 * b + k] : 0u;
            uint32_t tot;
            const uint32_t ex = block_excl_scan(v, scratch, &tot);
            if (b < nb && k < 3) partial[4 * b + k] = carry[k] + ex;
            carry[k] += tot;
        }
    }
    if (threadIdx.x == 0) {
        counts[0] = carry[0];
        counts[1] = carry[1];
        counts[2] = carry[2];
        counts[3] = carry[3];
    }
}

__device__ __forceinline__ void scatter_bits(uint32_t word, uint32_t base_id, uint32_t pos, uint32_t* out) {
    while (word) {
        const int b = __ffs(word) - 1;
        out[pos++] = base_id + (uint32_t)b;
        word &= word - 1u;
    }
}

__global__ void __launch_bounds__(GS_BLOCK) k_hazard_scatter(ScopeIn s, int32_t n, uint32_t nwords,
                                                             const uint32_t* __restrict__ offsets,
                                                             uint32_t* __restrict__ waw_idx,
                                                             uint32_t* __restrict__ raw_idx,
                                                             uint32_t* __restrict__ war_idx) {
    __shared__ uint32_t scratch[4];
    const uint32_t w = blockIdx.x * kWordsPerBlock + threadIdx.x;
    const Hazards h = hazard_words(s, w, nwords, n);
    uint32_t tot;
    const uint32_t p0 = block_excl_scan(__popc(h.waw), scratch, &tot) + offsets[4 * blockIdx.x + 0];
    const uint32_t p1 = block_excl_scan(__popc(h.raw), scratch, &tot) + offsets[4 * blockIdx.x + 1];
    const uint32_t p2 = block_excl_scan(__popc(h.war), scratch, &tot) + offsets[4 * blockIdx.x + 2];
    const uint32_t base = w << 5;
    if (waw_idx) scatter_bits(h.waw, base, p0, waw_idx);
    if (raw_idx) scatter_bits(h.raw, base, p1, raw_idx);
    if (war_idx) scatter_bits(h.war, base, p2, war_idx);
}

// ---------------------------------------------------------------------------
// throughput-first admission
// ---------------------------------------------------------------------------

struct GateIn {
    const uint32_t* RB;
    const uint32_t* D;
    const uint32_t* CA;
    const uint32_t* E;          // evidence; == CA when the caller passes none
    const float* g;
    const uint32_t* skip;       // may be null
    uint32_t version;
};

struct __align__(16) GatePartial {
    uint32_t n_read, n_delayed, n_active, n_missing;
    uint32_t n_second, max_bits, pad0, pad1;
    double sum_g;
    double pad2;
};

__device__ __forceinline__ double wave_sum_f64(double v) {
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) v += __shfl_xor(v, d, GS_WAVE);
    return v;
}

__device__ __forceinline__ float wave_max_f32(float v) {
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) v = fmaxf(v, __shfl_xor(v, d, GS_WAVE));
    return v;
}

__global__ void __launch_bounds__(GS_BLOCK) k_gate_partial(GateIn in, int32_t n, uint32_t nwords,
                                                           GatePartial* __restrict__ partial) {
    __shared__ uint32_t scratch[4];
    __shared__ double s_sum[4];
    __shared__ float s_max[4];
    const uint32_t w = blockIdx.x * kWordsPerBlock + threadIdx.x;
    const uint32_t mask = tail_mask(w, nwords, n);
    const uint32_t rb = load_word(in.RB, w, nwords, mask);
    const uint32_t d = load_word(in.D, w, nwords, mask);
    const uint32_t ca = load_word(in.CA, w, nwords, mask);
    const uint32_t ev = load_word(in.E, w, nwords, mask);
    uint32_t second = 0;
    if (in.skip != nullptr) {
        uint32_t x = d;
        while (x) {
            const int b = __ffs(x) - 1;
            const uint32_t s = in.skip[(w << 5) + (uint32_t)b];
            second += (s != 0u && s != in.version) ? 1u : 0u;
            x &= x - 1u;
        }
    }
    // ||g_A|| gathers: the wave's 64 words are 2048 consecutive ids; pass j
    // covers ids [64 j, 64 j + 64) of them, lane l taking id 64 j + l, whose
    // bit sits in the word of lane 2 j + (l >> 5).
    const int lane = lane_id();
    const uint32_t wave_w0 = w - (uint32_t)lane;
    double sum = 0.0;
    float mx = 0.0f;
#pragma unroll 4
    for (int j = 0; j < 32; ++j) {
        const int src = 2 * j + (lane >> 5);
        const uint32_t cw = (uint32_t)__shfl((int)ca, src, GS_WAVE);
        const uint32_t dw = (uint32_t)__shfl((int)d, src, GS_WAVE);
        const uint32_t bit = 1u << (lane & 31);
        if ((cw | dw) & bit) {
            const float gv = in.g[((wave_w0 + (uint32_t)src) << 5) + (uint32_t)(lane & 31)];
            if (cw & bit) sum += (double)gv;
            if (dw & bit) mx = fmaxf(mx, gv);
        }
    }
    sum = wave_sum_f64(sum);
    mx = wave_max_f32(mx);
    const int wv = threadIdx.x / GS_WAVE;
    if (lane == 0) {
        s_sum[wv] = sum;
        s_max[wv] = mx;
    }
    const uint32_t nR = block_sum_u32(__popc(rb), scratch);
    const uint32_t nD = block_sum_u32(__popc(d), scratch);
    const uint32_t nC = block_sum_u32(__popc(ca), scratch);
    const uint32_t nM = block_sum_u32(__popc(d & ~ev), scratch);
    const uint32_t nS = block_sum_u32(second, scratch);
    if (threadIdx.x == 0) {
        GatePartial p;
        p.n_read = nR;
        p.n_delayed = nD;
        p.n_active = nC;
        p.n_missing = nM;
        p.n_second = nS;
        p.max_bits = __float_as_uint(fmaxf(fmaxf(s_max[0], s_max[1]), fmaxf(s_max[2], s_max[3])));
        p.pad0 = p.pad1 = 0;
        p.sum_g = (s_sum[0] + s_sum[1]) + (s_sum[2] + s_sum[3]);
        p.pad2 = 0.0;
        partial[blockIdx.x] = p;
    }
}

// One workgroup: fixed-order reduction of the partials, then the decision.
__global__ void __launch_bounds__(GS_BLOCK) k_gate_decide(const GatePartial* __restrict__ partial, uint32_t nb,
                                                          double tau, gs_gate_result* __restrict__ out) {
    __shared__ double s_sum[GS_BLOCK];
    __shared__ uint32_t s_cnt[5][GS_BLOCK];
    __shared__ float s_max[GS_BLOCK];
    uint32_t c[5] = {0u, 0u, 0u, 0u, 0u};
    double sum = 0.0;
    float mx = 0.0f;
    for (uint32_t b = threadIdx.x; b < nb; b += GS_BLOCK) {
        const GatePartial p = partial[b];
        c[0] += p.n_read;
        c[1] += p.n_delayed;
        c[2] += p.n_active;
        c[3] += p.n_missing;
        c[4] += p.n_second;
        sum += p.sum_g;
        mx = fmaxf(mx, __uint_as_float(p.max_bits));
    }
    s_sum[threadIdx.x] = sum;
    s_max[threadIdx.x] = mx;
#pragma unroll
    for (int k = 0; k < 5; ++k) s_cnt[k][threadIdx.x] = c[k];
    __syncthreads();
    for (int h = GS_BLOCK / 2; h > 0; h >>= 1) {
        if ((int)threadIdx.x < h) {
            s_sum[threadIdx.x] += s_sum[threadIdx.x + h];
            s_max[threadIdx.x] = fmaxf(s_max[threadIdx.x], s_max[threadIdx.x + h]);
#pragma unroll
            for (int k = 0; k < 5; ++k) s_cnt[k][threadIdx.x] += s_cnt[k][threadIdx.x + h];
        }
        __syncthreads();
    }
    if (threadIdx.x != 0) return;
    const uint32_t nR = s_cnt[0][0], nD = s_cnt[1][0], nC = s_cnt[2][0], nM = s_cnt[3][0], nS = s_cnt[4][0];
    const double rho = nR > 0 ? (double)nD / (double)nR : 0.0;
    const double mean = nC > 0 ? s_sum[0] / (double)nC : 0.0;
    const double thr = tau * mean;
    const double max_g = (double)s_max[0];
    uint32_t reason;
    if (nD == 0)
        reason = GS_GATE_NO_DELAY;
    else if (rho > tau)
        reason = GS_GATE_WAIT_RHO;
    else if (nC == 0)
        reason = GS_GATE_WAIT_NO_ACTIVE;
    else if (nM != 0)
        reason = GS_GATE_WAIT_MISSING;
    else if (nS != 0)
        reason = GS_GATE_WAIT_SECOND;
    else if (max_g > thr)
        reason = GS_GATE_WAIT_GRADIENT;
    else
        reason = GS_GATE_ADMIT;
    gs_gate_result r;
    r.admit = (reason == GS_GATE_NO_DELAY || reason == GS_GATE_ADMIT) ? 1u : 0u;
    r.reason = reason;
    r.n_read = nR;
    r.n_delayed = nD;
    r.n_active = nC;
    r.n_missing = nM;
    r.n_second = nS;
    r.reserved = 0u;
    r.rho = rho;
    r.mean_g = mean;
    r.max_g = max_g;
    r.threshold = thr;
    *out = r;
}

// After an admission, every delayed id records the producer version whose
// pending update its readers skip.
__global__ void __launch_bounds__(GS_BLOCK) k_gate_mark(const uint32_t* __restrict__ D, int32_t n, uint32_t nwords,
                                                        const gs_gate_result* __restrict__ res, uint32_t version,
                                                        uint32_t* __restrict__ skip) {
    if (res->reason != GS_GATE_ADMIT) return;
    const uint32_t w = blockIdx.x * kWordsPerBlock + threadIdx.x;
    uint32_t x = load_word(D, w, nwords, tail_mask(w, nwords, n));
    while (x) {
        const int b = __ffs(x) - 1;
        skip[(w << 5) + (uint32_t)b] = version;
        x &= x - 1u;
    }
}

}  // namespace

size_t scope_ws_bytes(int32_t n) {
    const uint32_t nb = div_up(div_up((uint64_t)(n > 0 ? n : 0), 32), kWordsPerBlock);
    return align256(sizeof(GatePartial) * (size_t)(nb + 1));
}

hipError_t launch_scope_from_ids(const uint32_t* idx, const uint32_t* count, int32_t max_rows, int32_t n,
                                 int32_t accumulate, uint32_t* scope, hipStream_t st) {
    const uint32_t nwords = div_up((uint64_t)n, 32);
    if (nwords == 0) return hipSuccess;
    if (!accumulate) {
        hipError_t e = launch_fill_u32(scope, 0u, nwords, st);
        if (e != hipSuccess) return e;
    }
    if (max_rows <= 0) return hipSuccess;
    uint32_t blocks = div_up((uint64_t)max_rows, GS_BLOCK);
    if (blocks > 8192) blocks = 8192;
    hipLaunchKernelGGL(k_scope_from_ids, dim3(blocks), dim3(GS_BLOCK), 0, st, idx, count, max_rows, n, scope);
    return hipGetLastError();
}

hipError_t launch_scope_from_pred(int kind, const void* src, int32_t n, int32_t accumulate, uint32_t* scope,
                                  hipStream_t st) {
    if (n <= 0) return hipSuccess;
    const dim3 grid(div_up((uint64_t)n, GS_BLOCK));
    if (kind == GS_PRED_U32_NONZERO)
        hipLaunchKernelGGL(k_scope_from_pred<GS_PRED_U32_NONZERO>, grid, dim3(GS_BLOCK), 0, st, src, n, accumulate,
                           scope);
    else
        hipLaunchKernelGGL(k_scope_from_pred<GS_PRED_U8_NONZERO>, grid, dim3(GS_BLOCK), 0, st, src, n, accumulate,
                           scope);
    return hipGetLastError();
}

hipError_t launch_scope_conflicts(const uint32_t* RA, const uint32_t* WA, const uint32_t* RB, const uint32_t* WB,
                                  int32_t n, uint32_t* waw, uint32_t* raw, uint32_t* war, uint32_t* waw_idx,
                                  uint32_t* raw_idx, uint32_t* war_idx, uint32_t* counts, void* ws, hipStream_t st) {
    const uint32_t nwords = div_up((uint64_t)n, 32);
    if (nwords == 0) return launch_fill_u32(counts, 0u, 4, st);
    const uint32_t nb = div_up(nwords, kWordsPerBlock);
    uint32_t* partial = static_cast<uint32_t*>(ws);
    const ScopeIn s{RA, WA, RB, WB};
    hipLaunchKernelGGL(k_hazard_count, dim3(nb), dim3(GS_BLOCK), 0, st, s, n, nwords, waw, raw, war, partial);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_hazard_offsets, dim3(1), dim3(GS_BLOCK), 0, st, partial, nb, counts);
    e = hipGetLastError();
    if (e != hipSuccess || !(waw_idx || raw_idx || war_idx)) return e;
    hipLaunchKernelGGL(k_hazard_scatter, dim3(nb), dim3(GS_BLOCK), 0, st, s, n, nwords, partial, waw_idx, raw_idx,
                       war_idx);
    return hipGetLastError();
}

hipError_t launch_admission_gate(const uint32_t* RB, const uint32_t* D, const gs_gate_args& a, int32_t n,
                                 gs_gate_result* result, void* ws, hipStream_t st) {
    const uint32_t nwords = div_up((uint64_t)(n > 0 ? n : 0), 32);
    const uint32_t nb = div_up(nwords, kWordsPerBlock);
    GatePartial* partial = static_cast<GatePartial*>(ws);
    const GateIn in{RB, D, a.active, a.evidence ? a.evidence : a.active, a.g, a.skip, a.producer_version};
    if (nb > 0) {
        hipLaunchKernelGGL(k_gate_partial, dim3(nb), dim3(GS_BLOCK), 0, st, in, n, nwords, partial);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(k_gate_decide, dim3(1), dim3(GS_BLOCK), 0, st, partial, nb, a.tau, result);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || a.skip == nullptr || nb == 0) return e;
    hipLaunchKernelGGL(k_gate_mark, dim3(nb), dim3(GS_BLOCK), 0, st, D, n, nwords, result, a.producer_version,
                       a.skip);
    return hipGetLastError();
}

}  // namespace gsmi
