// Ahead-of-time planner on the host: the relative locality graph (Section
// 4.1.1, Eq. 1), logical partitioning (Section 4.2, LP: balanced k-means over
// the camera centres, refined on the graph so that strong coupling stays
// within groups) and static data scheduling (Section 4.2, SDS, Eq. 2).
//
// Every floating-point value is produced by one fixed sequence of IEEE double
// operations (this file is built without FMA contraction), so the results do
// not depend on the thread count: the graph's rows are built in parallel, one
// row per view, and each row's arithmetic is the row's own.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <thread>
#include <vector>

#include "planner.h"

namespace gsmi {

namespace {

int plan_fail(char* err, size_t len, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    if (err && len) vsnprintf(err, len, fmt, ap);
    va_end(ap);
    return GS_ERR_INVALID_ARG;
}

int worker_count(int64_t work) {
    unsigned hw = std::thread::hardware_concurrency();
    int t = (int)std::min<unsigned>(hw ? hw : 1, 16);
    if (work < (int64_t)1 << 16) t = 1;
    return std::max(t, 1);
}

template <class F>
void parallel_rows(int32_t n, int threads, F&& f) {
    if (threads <= 1 || n < 2) {
        f(0, n, 0);
        return;
    }
    std::vector<std::thread> pool;
    const int32_t chunk = (n + threads - 1) / threads;
    for (int t = 0; t < threads; ++t) {
        const int32_t a = t * chunk, b = std::min(n, a + chunk);
        if (a >= b) break;
        pool.emplace_back([&, a, b, t] { f(a, b, t); });
    }
    for (auto& th : pool) th.join();
}

struct Cand {
    double w;
    int32_t j;
};

inline double sqdist(const double* p, const double* c) {
    const double dx = p[0] - c[0], dy = p[1] - c[1], dz = p[2] - c[2];
    return dx * dx + dy * dy + dz * dz;
}

}  // namespace

int rlg_build(int32_t n, int32_t n_tracks, const int64_t* item_ptr, const int32_t* item_tracks, int32_t track_cap,
              int32_t top_k, int64_t* edge_ptr, int32_t* edge_dst, double* edge_w, int64_t edge_capacity,
              int64_t* n_edges, char* err, size_t errlen) {
    // input checks: monotone offsets, track ids in range, strictly ascending per view
    if (item_ptr[0] != 0) return plan_fail(err, errlen, "item_ptr[0] must be 0");
    for (int32_t i = 0; i < n; ++i) {
        if (item_ptr[i + 1] < item_ptr[i]) return plan_fail(err, errlen, "item_ptr decreases at view %d", i);
        for (int64_t e = item_ptr[i]; e < item_ptr[i + 1]; ++e) {
            const int32_t t = item_tracks[e];
            if (t < 0 || t >= n_tracks) return plan_fail(err, errlen, "view %d: track id %d outside [0, %d)", i, t,
                                                         n_tracks);
            if (e > item_ptr[i] && item_tracks[e - 1] >= t)
                return plan_fail(err, errlen, "view %d: track ids not strictly ascending", i);
        }
    }
    // track lengths, the outlier cap, each view's kept-set size
    std::vector<int32_t> len((size_t)n_tracks, 0);
    const int64_t nnz = item_ptr[n];
    for (int64_t e = 0; e < nnz; ++e) ++len[item_tracks[e]];
    std::vector<uint8_t> kept((size_t)n_tracks);
    for (int32_t t = 0; t < n_tracks; ++t) kept[t] = track_cap <= 0 || len[t] <= track_cap;
    std::vector<int32_t> psize((size_t)n, 0);
    for (int32_t i = 0; i < n; ++i)
        for (int64_t e = item_ptr[i]; e < item_ptr[i + 1]; ++e) psize[i] += kept[item_tracks[e]];
    // inverse track -> view mapping over kept tracks (views ascending)
    std::vector<int64_t> tptr((size_t)n_tracks + 1, 0);
    for (int32_t t = 0; t < n_tracks; ++t) tptr[t + 1] = tptr[t] + (kept[t] ? len[t] : 0);
    std::vector<int32_t> tviews((size_t)tptr[n_tracks]);
    {
        std::vector<int64_t> fill(tptr.begin(), tptr.end() - 1);
        for (int32_t i = 0; i < n; ++i)
            for (int64_t e = item_ptr[i]; e < item_ptr[i + 1]; ++e)
                if (kept[item_tracks[e]]) tviews[fill[item_tracks[e]]++] = i;
    }
    // each view's retained neighbours: Jaccard of the shared-track count, top_k by (w desc, id asc)
    std::vector<std::vector<Cand>> sel((size_t)n);
    int64_t pair_work = 0;
    for (int32_t t = 0; t < n_tracks; ++t) pair_work += kept[t] ? (int64_t)len[t] * len[t] : 0;
    const int threads = worker_count(pair_work);
    parallel_rows(n, threads, [&](int32_t a, int32_t b, int) {
        std::vector<int32_t> cnt((size_t)n, 0);
        std::vector<int32_t> touched;
        std::vector<Cand> cand;
        for (int32_t i = a; i < b; ++i) {
            touched.clear();
            for (int64_t e = item_ptr[i]; e < item_ptr[i + 1]; ++e) {
                const int32_t t = item_tracks[e];
                if (!kept[t]) continue;
                for (int64_t q = tptr[t]; q < tptr[t + 1]; ++q) {
                    const int32_t j = tviews[q];
                    if (j == i) continue;
                    if (cnt[j]++ == 0) touched.push_back(j);
                }
            }
            cand.clear();
            for (int32_t j : touched) {
                const int32_t inter = cnt[j];
                const int32_t uni = psize[i] + psize[j] - inter;
                cand.push_back({(double)inter / (double)uni, j});
                cnt[j] = 0;
            }
            auto better = [](const Cand& x, const Cand& y) { return x.w > y.w || (x.w == y.w && x.j < y.j); };
            if (top_k > 0 && (int64_t)cand.size() > top_k) {
                std::partial_sort(cand.begin(), cand.begin() + top_k, cand.end(), better);
                cand.resize((size_t)top_k);
            }
            sel[i] = cand;
        }
    });
    // symmetric retention: an edge stays when either end keeps it
    std::vector<int64_t> deg((size_t)n + 1, 0);
    for (int32_t i = 0; i < n; ++i)
        for (const Cand& c : sel[i]) {
            ++deg[i];
            ++deg[c.j];
        }
    std::vector<int64_t> rp((size_t)n + 1, 0);
    for (int32_t i = 0; i < n; ++i) rp[i + 1] = rp[i] + deg[i];
    std::vector<Cand> rows((size_t)rp[n]);
    {
        std::vector<int64_t> fill(rp.begin(), rp.end() - 1);
        for (int32_t i = 0; i < n; ++i)
            for (const Cand& c : sel[i]) {
                rows[fill[i]++] = {c.w, c.j};
                rows[fill[c.j]++] = {c.w, i};
            }
    }
    int64_t total = 0;
    std::vector<int64_t> out_deg((size_t)n, 0);
    for (int32_t i = 0; i < n; ++i) {
        auto b = rows.begin() + rp[i], e = rows.begin() + rp[i + 1];
        std::sort(b, e, [](const Cand& x, const Cand& y) { return x.j < y.j; });
        auto last = std::unique(b, e, [](const Cand& x, const Cand& y) { return x.j == y.j; });
        out_deg[i] = last - b;
        total += out_deg[i];
    }
    *n_edges = total;
    if (total > edge_capacity) return GS_ERR_WORKSPACE;
    edge_ptr[0] = 0;
    for (int32_t i = 0; i < n; ++i) {
        const int64_t o = edge_ptr[i];
        for (int64_t k = 0; k < out_deg[i]; ++k) {
            edge_dst[o + k] = rows[rp[i] + k].j;
            edge_w[o + k] = rows[rp[i] + k].w;
        }
        edge_ptr[i + 1] = o + out_deg[i];
    }
    return GS_OK;
}

int check_graph(int32_t n, const int64_t* edge_ptr, const int32_t* edge_dst, const double* edge_w, char* err,
                size_t errlen) {
    if (edge_ptr[0] != 0) return plan_fail(err, errlen, "edge_ptr[0] must be 0");
    for (int32_t i = 0; i < n; ++i) {
        if (edge_ptr[i + 1] < edge_ptr[i]) return plan_fail(err, errlen, "edge_ptr decreases at view %d", i);
        for (int64_t e = edge_ptr[i]; e < edge_ptr[i + 1]; ++e) {
            const int32_t j = edge_dst[e];
            if (j < 0 || j >= n || j == i) return plan_fail(err, errlen, "view %d: neighbour %d invalid", i, j);
            if (e > edge_ptr[i] && edge_dst[e - 1] >= j)
                return plan_fail(err, errlen, "view %d: neighbours not strictly ascending", i);
            if (!(edge_w[e] > 0.0 && edge_w[e] <= 1.0))
                return plan_fail(err, errlen, "view %d: edge weight outside (0, 1]", i);
        }
    }
    return GS_OK;
}

// Passes of the LP refinement at most.
constexpr int kRefinePasses = 16;

int lp_partition(int32_t n, const double* pos, const int64_t* edge_ptr, const int32_t* edge_dst,
                 const double* edge_w, int32_t K, int32_t max_iters, int32_t* group, double* coupling,
                 int32_t* iters_run, char* err, size_t errlen) {
    for (int64_t q = 0; q < 3 * (int64_t)n; ++q)
        if (!std::isfinite(pos[q])) return plan_fail(err, errlen, "camera centre %lld not finite", (long long)(q / 3));
    int s = check_graph(n, edge_ptr, edge_dst, edge_w, err, errlen);
    if (s != GS_OK) return s;
    for (int64_t q = 0; q < (int64_t)K * K; ++q) coupling[q] = 0.0;
    *iters_run = 0;
    if (n == 0) return GS_OK;
    const int32_t cap = (n + K - 1) / K;
    // farthest-point seeds from view 0 (ties: lowest view id)
    std::vector<double> cen((size_t)3 * K);
    std::vector<double> near((size_t)n);
    for (int c = 0; c < 3; ++c) cen[c] = pos[c];
    for (int32_t i = 0; i < n; ++i) near[i] = sqdist(pos + 3 * (size_t)i, pos);
    for (int32_t g = 1; g < K; ++g) {
        int32_t far = 0;
        for (int32_t i = 1; i < n; ++i)
            if (near[i] > near[far]) far = i;
        for (int c = 0; c < 3; ++c) cen[3 * g + c] = pos[3 * (size_t)far + c];
        for (int32_t i = 0; i < n; ++i) near[i] = std::min(near[i], sqdist(pos + 3 * (size_t)i, pos + 3 * (size_t)far));
    }
    struct Tri {
        double d;
        int32_t i, g;
    };
    std::vector<Tri> tri((size_t)n * K);
    std::vector<int32_t> cur((size_t)n, -1), nxt((size_t)n), count((size_t)K);
    bool first = true;
    for (int32_t it = 0; it < max_iters; ++it) {
        ++*iters_run;
        // balanced assignment: (distance, view, group) ascending, each group up to ceil(n / K)
        for (int32_t i = 0; i < n; ++i)
            for (int32_t g = 0; g < K; ++g)
                tri[(size_t)i * K + g] = {sqdist(pos + 3 * (size_t)i, &cen[3 * g]), i, g};
        std::sort(tri.begin(), tri.end(), [](const Tri& x, const Tri& y) {
            if (x.d != y.d) return x.d < y.d;
            if (x.i != y.i) return x.i < y.i;
            return x.g < y.g;
        });
        std::fill(nxt.begin(), nxt.end(), -1);
        std::fill(count.begin(), count.end(), 0);
        for (const Tri& t : tri)
            if (nxt[t.i] < 0 && count[t.g] < cap) {
                nxt[t.i] = t.g;
                ++count[t.g];
            }
        if (!first && nxt == cur) break;
        first = false;
        cur.swap(nxt);
        // centres: member means, summed in ascending view order
        std::vector<double> sum((size_t)3 * K, 0.0);
        std::vector<int32_t> c((size_t)K, 0);
        for (int32_t i = 0; i < n; ++i) {
            const int32_t g = cur[i];
            sum[3 * g + 0] += pos[3 * (size_t)i + 0];
            sum[3 * g + 1] += pos[3 * (size_t)i + 1];
            sum[3 * g + 2] += pos[3 * (size_t)i + 2];
            ++c[g];
        }
        for (int32_t g = 0; g < K; ++g)
            if (c[g])
                for (int k = 0; k < 3; ++k) cen[3 * g + k] = sum[3 * g + k] / (double)c[g];
    }
    // Refinement on the graph, so that strong coupling stays within groups: in
    // passes over the views in ascending order, a view moves to the group its
    // retained edges weigh most towards (neighbours summed in ascending order;
    // the lowest group on ties) when that beats the weight towards its own
    // group, within the size band floor(n/K) - s .. ceil(n/K) + s, s =
    // max(1, ceil(n/K) / 16); until a pass moves nothing.
    if (K >= 2) {
        const int32_t top = (n + K - 1) / K;
        const int32_t slack = std::max(1, top / 16);
        const int32_t lo = n / K - slack, hi = top + slack;
        std::vector<int32_t> size((size_t)K, 0);
        for (int32_t i = 0; i < n; ++i) ++size[cur[i]];
        std::vector<double> W((size_t)K);
        for (int pass = 0; pass < kRefinePasses; ++pass) {
            bool moved = false;
            for (int32_t u = 0; u < n; ++u) {
                const int32_t a = cur[u];
                std::fill(W.begin(), W.end(), 0.0);
                for (int64_t e = edge_ptr[u]; e < edge_ptr[u + 1]; ++e) W[cur[edge_dst[e]]] += edge_w[e];
                int32_t best = -1;
                double gain = 0.0;
                for (int32_t b = 0; b < K; ++b) {
                    if (b == a || size[b] >= hi) continue;
                    const double d = W[b] - W[a];
                    if (d > gain) {
                        best = b;
                        gain = d;
                    }
                }
                if (best >= 0 && size[a] > lo) {
                    cur[u] = best;
                    --size[a];
                    ++size[best];
                    moved = true;
                }
            }
            if (!moved) break;
        }
    }
    for (int32_t i = 0; i < n; ++i) group[i] = cur[i];
    // region-level coupling: retained edge weights summed per group pair, views ascending
    for (int32_t i = 0; i < n; ++i)
        for (int64_t e = edge_ptr[i]; e < edge_ptr[i + 1]; ++e) {
            const int32_t j = edge_dst[e];
            if (j <= i) continue;
            const int32_t a = cur[i], b = cur[j];
            coupling[(size_t)a * K + b] += edge_w[e];
            if (a != b) coupling[(size_t)b * K + a] += edge_w[e];
        }
    return GS_OK;
}

int sds_order(int32_t n, const int32_t* group, int32_t K, const double* coupling, const int64_t* edge_ptr,
              const int32_t* edge_dst, const double* edge_w, int32_t unit_size, int32_t* cycle, int32_t* n_cycle,
              int32_t* order, int32_t* unit_group, double* transition, int32_t* n_units, char* err,
              size_t errlen) {
    for (int32_t i = 0; i < n; ++i)
        if (group[i] < 0 || group[i] >= K) return plan_fail(err, errlen, "view %d: group %d outside [0, %d)", i,
                                                            group[i], K);
    int s = check_graph(n, edge_ptr, edge_dst, edge_w, err, errlen);
    if (s != GS_OK) return s;
    // members of each group, ascending
    std::vector<std::vector<int32_t>> mem((size_t)K);
    for (int32_t i = 0; i < n; ++i) mem[group[i]].push_back(i);
    // the traversal: from the first non-empty group, always to the least coupled unvisited one
    std::vector<int32_t> cyc;
    std::vector<uint8_t> used((size_t)K, 0);
    for (int32_t g = 0; g < K; ++g)
        if (!mem[g].empty()) {
            cyc.push_back(g);
            used[g] = 1;
            break;
        }
    for (;;) {
        const int32_t last = cyc.empty() ? -1 : cyc.back();
        int32_t best = -1;
        for (int32_t g = 0; g < K && last >= 0; ++g)
            if (!used[g] && !mem[g].empty() &&
                (best < 0 || coupling[(size_t)last * K + g] < coupling[(size_t)last * K + best]))
                best = g;
        if (best < 0) break;
        cyc.push_back(best);
        used[best] = 1;
    }
    const int32_t L = (int32_t)cyc.size();
    *n_cycle = L;
    for (int32_t g = 0; g < K; ++g) cycle[g] = g < L ? cyc[g] : -1;
    // units take turns over the cycle; each is filled by Eq. 2 against the previous unit
    std::vector<size_t> cursor((size_t)K, 0);
    std::vector<int32_t> left_in((size_t)K);
    for (int32_t g = 0; g < K; ++g) left_in[g] = (int32_t)mem[g].size();
    std::vector<uint8_t> removed((size_t)n, 0);
    std::vector<double> score((size_t)n, 0.0);
    std::vector<int64_t> stamp((size_t)n, -1), in_unit((size_t)n, -1);
    std::vector<int32_t> prev, unit, touched;
    int64_t fill_id = 0;
    int32_t left = n, pos = 0, units = 0, written = 0;
    while (left > 0) {
        while (left_in[cyc[pos % L]] == 0) ++pos;
        const int32_t start = pos % L;
        ++pos;
        unit.clear();
        int32_t k = start;
        std::vector<int32_t> prev_sorted(prev);
        std::sort(prev_sorted.begin(), prev_sorted.end());
        while ((int32_t)unit.size() < unit_size && left > 0) {
            while (left_in[cyc[k % L]] == 0) ++k;
            const int32_t g = cyc[k % L];
            int32_t need = unit_size - (int32_t)unit.size();
            // scores of this group's remaining views that neighbour the previous unit
            ++fill_id;
            touched.clear();
            for (int32_t u : prev_sorted)
                for (int64_t e = edge_ptr[u]; e < edge_ptr[u + 1]; ++e) {
                    const int32_t v = edge_dst[e];
                    if (group[v] != g || removed[v]) continue;
                    if (stamp[v] != fill_id) {
                        stamp[v] = fill_id;
                        score[v] = 0.0;
                        touched.push_back(v);
                    }
                    score[v] += edge_w[e];
                }
            // score-0 views first (ascending id), then the neighbours by (score, id)
            std::vector<int32_t>& m = mem[g];
            while (cursor[g] < m.size() && removed[m[cursor[g]]]) ++cursor[g];
            for (size_t q = cursor[g]; q < m.size() && need > 0; ++q) {
                const int32_t v = m[q];
                if (removed[v] || stamp[v] == fill_id) continue;
                removed[v] = 1;
                unit.push_back(v);
                --need;
                --left_in[g];
                --left;
            }
            if (need > 0) {
                std::sort(touched.begin(), touched.end(), [&](int32_t x, int32_t y) {
                    return score[x] < score[y] || (score[x] == score[y] && x < y);
                });
                for (size_t q = 0; q < touched.size() && need > 0; ++q) {
                    const int32_t v = touched[q];
                    removed[v] = 1;
                    unit.push_back(v);
                    --need;
                    --left_in[g];
                    --left;
                }
            }
        }
        // transition summary: the largest retained weight between the two units
        double t = 0.0;
        for (int32_t v : unit) in_unit[v] = units;
        for (int32_t u : prev)
            for (int64_t e = edge_ptr[u]; e < edge_ptr[u + 1]; ++e)
                if (in_unit[edge_dst[e]] == units) t = std::max(t, edge_w[e]);
        for (int32_t v : unit) order[written++] = v;
        unit_group[units] = cyc[start];
        transition[units] = t;
        ++units;
        prev.swap(unit);
    }
    *n_units = units;
    return GS_OK;
}

}  // namespace gsmi
