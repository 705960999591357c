// Host planner (planner.cpp): declarations without any GPU type, so that the
// planner also builds as plain C++ (the sanitizer test builds it with g++).
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "../../include/gsmi.h"

namespace gsmi {

// planner.cpp (host): return GS_OK, GS_ERR_INVALID_ARG (message in err) or GS_ERR_WORKSPACE
int rlg_build(int32_t n, int32_t n_tracks, const int64_t* item_ptr, const int32_t* item_tracks, int32_t track_cap,
              int32_t top_k, int64_t* edge_ptr, int32_t* edge_dst, double* edge_w, int64_t edge_capacity,
              int64_t* n_edges, char* err, size_t errlen);
int lp_partition(int32_t n, const double* pos, const int64_t* edge_ptr, const int32_t* edge_dst,
                 const double* edge_w, int32_t K, int32_t max_iters, int32_t* group, double* coupling,
                 int32_t* iters_run, char* err, size_t errlen);
int sds_order(int32_t n, const int32_t* group, int32_t K, const double* coupling, const int64_t* edge_ptr,
              const int32_t* edge_dst, const double* edge_w, int32_t unit_size, int32_t* cycle, int32_t* n_cycle,
              int32_t* order, int32_t* unit_group, double* transition, int32_t* n_units, char* err,
              size_t errlen);

}  // namespace gsmi
