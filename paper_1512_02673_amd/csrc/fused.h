// The bf16 single pass (encode and all worker products in one pass over A)
// started from X itself: X^T for the products and the zeroed Y are prepared
// in one launch ahead of the pass instead of two.
#pragma once
#include "internal.h"

namespace coded {

// a.xt receives X^T (s x r, s = 64); X is r x s bf16 with row stride ldx.
hipError_t launch_fused_bf16_from_x(FusedArgs a, const uint16_t* X, int64_t s, int64_t ldx, int compute_units,
                                    hipStream_t st);

}  // namespace coded
