// Host-side entry points of the single-buffer pipelined resolve kernel
// (refill.hip), for the API layer.
#pragma once

#include "internal.h"

namespace bkmoo {

constexpr int kRefillMaxK = 10;
constexpr int kRefMaxGroups = 32;  // bucket groups (and solvers) at most

// Single-buffer pipelined resolve (K <= kRefillMaxK): cooperative grid
// (0 if it cannot run), elements of a segment it can keep on chip, launch.
// Its data workgroups hold equal segments; refill_stream_min() vectors per
// row and thread of each segment are always streamed.
int refill_grid(int K, int dt, int out_dt);
int64_t refill_held_elems(int K, int dt, int out_dt);
int refill_stream_min();
// Streamed vectors per row and thread a data workgroup reads with the
// temporal cache policy, for `groups` groups over a grid of `grid`.
int refill_temporal_slots(int K, int dt, int grid, int groups);
// Solver workgroups for `groups` groups of data workgroups: group g takes
// buckets g, g + groups, ..., each spread over (grid - solvers) / groups
// data workgroups.
int refill_solvers(int groups);
hipError_t launch_refill(int K, int dt, int out_dt, const void *const *rows, const int64_t *offs, int B,
                         int shift, int method, int iters, double c, const int8_t *order, double *gram,
                         float *weights, double *aux, void *out, double *partials, uint32_t *arrive,
                         uint32_t *recs, uint32_t *err, uint32_t spin_limit, int grid, int groups,
                         int tslots, hipStream_t s);

}  // namespace bkmoo
