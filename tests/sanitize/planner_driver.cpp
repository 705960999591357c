// Drives the host planner (graph, partition, schedule) over a seeded synthetic
// capture and over malformed inputs, and prints a digest of every result: the
// sanitizer test runs it built with and without AddressSanitizer/UBSan and
// compares the two digests.
#include <algorithm>
#include <cstdint>
#include <cstdio>
#include <vector>

#include "planner.h"

namespace {

uint64_t lcg(uint64_t& s) {
    s = s * 6364136223846793005ull + 1442695040888963407ull;
    return s >> 33;
}

uint64_t fnv(uint64_t h, const void* p, size_t n) {
    const unsigned char* b = static_cast<const unsigned char*>(p);
    for (size_t i = 0; i < n; ++i) h = (h ^ b[i]) * 1099511628211ull;
    return h;
}

}  // namespace

int main() {
    char err[256];
    uint64_t digest = 1469598103934665603ull;
    for (int run = 0; run < 4; ++run) {
        uint64_t s = 12345 + run;
        // the last run is large enough for the graph to be built by several threads
        const int32_t n = run < 3 ? 200 + 150 * run : 4000, n_tracks = run < 3 ? 3000 : 20000;
        std::vector<int64_t> item_ptr(n + 1, 0);
        std::vector<int32_t> item_tracks;
        std::vector<double> pos(3 * (size_t)n);
        for (int32_t i = 0; i < n; ++i) {
            // views along a path: each sees a window of tracks around its position
            const int32_t c = (int32_t)((int64_t)i * n_tracks / n);
            std::vector<int32_t> t;
            for (int32_t k = 0; k < 40; ++k) {
                const int32_t tr = (c + (int32_t)(lcg(s) % 200) - 100 + n_tracks) % n_tracks;
                t.push_back(tr);
            }
            std::sort(t.begin(), t.end());
            t.erase(std::unique(t.begin(), t.end()), t.end());
            item_tracks.insert(item_tracks.end(), t.begin(), t.end());
            item_ptr[i + 1] = (int64_t)item_tracks.size();
            for (int k = 0; k < 3; ++k) pos[3 * (size_t)i + k] = (double)(lcg(s) % 1000) / 100.0 + (k == 0 ? i : 0);
        }
        int64_t cap = 2 * (int64_t)n * 8, ne = 0;
        std::vector<int64_t> eptr(n + 1);
        std::vector<int32_t> edst;
        std::vector<double> ew;
        int st;
        for (int attempt = 0; attempt < 2; ++attempt) {
            edst.assign((size_t)cap, 0);
            ew.assign((size_t)cap, 0.0);
            st = gsmi::rlg_build(n, n_tracks, item_ptr.data(), item_tracks.data(), 64, 8, eptr.data(), edst.data(),
                                 ew.data(), cap, &ne, err, sizeof err);
            if (st != GS_ERR_WORKSPACE) break;
            cap = ne;
        }
        if (st != GS_OK) {
            std::printf("rlg_build failed: %s\n", err);
            return 1;
        }
        digest = fnv(digest, eptr.data(), eptr.size() * sizeof(int64_t));
        digest = fnv(digest, edst.data(), (size_t)ne * sizeof(int32_t));
        digest = fnv(digest, ew.data(), (size_t)ne * sizeof(double));
        const int32_t K = 4;
        std::vector<int32_t> group(n);
        std::vector<double> coupling(K * K);
        int32_t iters = 0;
        st = gsmi::lp_partition(n, pos.data(), eptr.data(), edst.data(), ew.data(), K, 20, group.data(),
                                coupling.data(), &iters, err, sizeof err);
        if (st != GS_OK) {
            std::printf("lp_partition failed: %s\n", err);
            return 1;
        }
        digest = fnv(digest, group.data(), group.size() * sizeof(int32_t));
        digest = fnv(digest, coupling.data(), coupling.size() * sizeof(double));
        const int32_t unit = 2 + run;
        std::vector<int32_t> cycle(K), order(n), unit_group(n);
        std::vector<double> transition(n);
        int32_t n_cycle = 0, n_units = 0;
        st = gsmi::sds_order(n, group.data(), K, coupling.data(), eptr.data(), edst.data(), ew.data(), unit,
                             cycle.data(), &n_cycle, order.data(), unit_group.data(), transition.data(), &n_units,
                             err, sizeof err);
        if (st != GS_OK) {
            std::printf("sds_order failed: %s\n", err);
            return 1;
        }
        digest = fnv(digest, order.data(), order.size() * sizeof(int32_t));
        digest = fnv(digest, transition.data(), (size_t)n_units * sizeof(double));
        // malformed inputs: each must be refused with a message, touching nothing out of bounds
        std::vector<int64_t> bad_ptr(item_ptr);
        bad_ptr[0] = 1;
        int refused = 0;
        refused += gsmi::rlg_build(n, n_tracks, bad_ptr.data(), item_tracks.data(), 64, 8, eptr.data(), edst.data(),
                                   ew.data(), cap, &ne, err, sizeof err) == GS_ERR_INVALID_ARG;
        std::vector<int32_t> bad_tracks(item_tracks);
        bad_tracks[0] = n_tracks + 5;
        refused += gsmi::rlg_build(n, n_tracks, item_ptr.data(), bad_tracks.data(), 64, 8, eptr.data(), edst.data(),
                                   ew.data(), cap, &ne, err, sizeof err) == GS_ERR_INVALID_ARG;
        std::vector<int32_t> bad_group(group);
        bad_group[n - 1] = K;
        refused += gsmi::sds_order(n, bad_group.data(), K, coupling.data(), eptr.data(), edst.data(), ew.data(), unit,
                                   cycle.data(), &n_cycle, order.data(), unit_group.data(), transition.data(),
                                   &n_units, err, sizeof err) == GS_ERR_INVALID_ARG;
        if (refused != 3) {
            std::printf("malformed input accepted (%d of 3 refused)\n", refused);
            return 1;
        }
    }
    std::printf("digest %016llx\n", (unsigned long long)digest);
    return 0;
}
