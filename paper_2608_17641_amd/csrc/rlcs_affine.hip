// The bare recurrence with supplied coefficients (Section 4.1).
#include "rlcs_dispatch.h"

using namespace rlcs;
using namespace rlcs::host;

extern "C" {

rlcs_status rlcs_affine_scan(const void* alpha, const void* beta, const void* carry, float* out,
                             int64_t N, int64_t T, rlcs_direction direction, rlcs_dtype dtype,
                             void* ws, size_t ws_bytes, rlcs_stream_t stream) {
    rlcs_status st = check_common(N, T, dtype, {alpha, beta, carry}, {out});
    if (st != RLCS_OK) return st;
    if (direction != RLCS_BACKWARD && direction != RLCS_FORWARD) return RLCS_ERR_INVALID_ARG;
    if (N == 0 || T == 0) return RLCS_OK;
    if (!alpha || !beta || !out) return RLCS_ERR_INVALID_ARG;
    Args a = make_args(N, T, 1.f, 1.f, 1.f, 1.f);
    a.in[0] = alpha; a.in[1] = beta;
    a.row_value = carry;
    a.out0 = out;
    if (direction == RLCS_FORWARD)
        return dispatch<AffineOp<false>>(a, dtype, false, ws, ws_bytes, stream);
    return dispatch<AffineOp<true>>(a, dtype, false, ws, ws_bytes, stream);
}

}  // extern "C"
