// Internal declarations shared by the calibration translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace masq {

// C (i, j) at c[i * crs + j * ccs] := alpha * sum_k A(i, k) B(k, j) (+ beta C),
// fp64, A (i, k) at a[i * ars + k * acs], B (k, j) at b[k * brs + j * bcs];
// each sum in increasing k by fused multiply-adds.  lower: only tiles that
// hold an element with j <= i are computed (the others are left as they
// are).  C must not share an element with A or B.  Enqueues on s.
hipError_t launch_dgemm(int64_t m, int64_t n, int64_t k, const double* a, int64_t ars,
                        int64_t acs, const double* b, int64_t brs, int64_t bcs, double alpha,
                        double beta, double* c, int64_t crs, int64_t ccs, bool lower,
                        hipStream_t s);

}  // namespace masq
