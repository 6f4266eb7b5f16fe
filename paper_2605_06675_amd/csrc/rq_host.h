// Host-only helpers of the library (no device code).
#pragma once

#include <stdint.h>

#include "../../include/rq.h"

namespace rq {

rq_status fit_distortion(const double* mse, int n_comp, const int32_t* bits,
                         int n_bits, double* alpha, double* beta, double* r2);
int64_t budget(int n, double avg_bits);
void waterfill(int n, const double* w, const double* alpha, const double* beta,
               int64_t B, int bmin, int bmax, double* out);
void greedy(int n, const double* w, const double* alpha, const double* beta,
            int64_t B, int bmin, int bmax, int32_t* out);
// TurboQuant codebook table, host float [8][2][256] (computed once)
const float* turbo_table();

}  // namespace rq
