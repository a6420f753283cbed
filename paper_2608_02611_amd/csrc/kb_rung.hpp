// kb_rung.hpp -- declarations of the rung kernels (kb_rung.hip): statistics
// and the promotion decision,
// shared with the host side of the C interface.
#pragma once

#include <hip/hip_runtime.h>

#include "../../include/kb.h"

namespace kb {

constexpr int kRungMaxIter = KB_RUNG_MAX_ITER;

struct RungParams {
    int n_cands, n_shapes, n_iter, base, rung;
    double budget, alpha, beta;
};

hipError_t launch_rung_stats(const RungParams& p, const double* samples, kb_sample_stats* rows,
                             kb_rung_score* scores, hipStream_t stream);

hipError_t launch_rung_promote(const kb_rung_score* scores, int n, int base, int num, int den,
                               int32_t* rank, int32_t* order, int32_t* promoted, hipStream_t stream);

}  // namespace kb
