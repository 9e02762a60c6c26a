// Kernel selection rules compiled into libgeot_hip (Section III-C: the rules
// are a decision tree over cheap input features, emitted as if/else).
//
// This is the hand-written starting rule set; the offline tuner replaces this
// file with a tree fitted to MI355X timings (same function signature).
//
// Inputs: nnz, num_segments, F, op (0 sum, 1 mean, 2 max), gather (0/1),
// has_stats (0/1) and, when has_stats, cv = stddev / mean of the segment
// lengths and max_rel = longest segment / mean.
// Output: out[0] family (1 EP, 2 SP), out[1] vec (0 auto), out[2] lanes
// (0 auto), out[3] rows (0 auto), out[4] groups (0 auto).
#pragma once

#include <cstdint>

namespace geot {

static inline void tree_select(double nnz, double num_segments, double F, int op, int gather,
                               int has_stats, double cv, double max_rel, int32_t out[5]) {
    (void)nnz; (void)F; (void)op; (void)gather;
    const double mean = num_segments > 0 ? nnz / num_segments : 0.0;
    out[0] = 1; out[1] = 0; out[2] = 0; out[3] = 0; out[4] = 0;
    if (has_stats && cv <= 0.5 && max_rel <= 4.0 && mean <= 64.0) {
        out[0] = 2;
    }
}

}  // namespace geot
