// rows.h -- per-query outputs of a query that draws no candidates.
//
// A query draws no candidates when it is skipped (no positive, or an anchor
// or relation id the shape uses is out of range) or when it asks for no
// negatives (n_neg = 0).  What such a query writes depends on the call:
//   shared_mode 0  per-query sampling: its negatives row is all -1, its draw
//                  count is 0 (n_neg = 0) or -1 (skipped);
//   shared_mode 1  a shared-candidate minibatch: no per-query row and no draw
//                  count exist (their pointers may be NULL);
//   shared_mode 2  verification of given candidates: likewise.
// n_valid is 0, or -1 for a skipped query, in every mode.
//
// The function is __host__ __device__ so that a host build (with the
// address sanitizer) can check that modes 1 and 2 never touch the
// per-query arrays.
#pragma once

#include "smore_internal.h"

namespace smore {

__host__ __device__ inline void write_undrawn_row(const SampleParams& p, const smore_sample_out& out,
                                                  int32_t b, bool ok)
{
    if (p.shared_mode == 0) {
        if (p.n_neg > 0) {
            int32_t* row = out.negatives + (int64_t)b * p.n_neg;
            for (int32_t k = 0; k < p.n_neg; ++k) row[k] = -1;
        }
        out.neg_draws[b] = ok ? 0 : -1;
    }
    out.n_valid[b] = ok ? 0 : -1;
}

}  // namespace smore
