// GAE entry point (Table 1; Section 3.3.1).
#include "rlcs_dispatch.h"

using namespace rlcs;
using namespace rlcs::host;

extern "C" {

rlcs_status rlcs_gae(const void* r, const void* v, const uint8_t* term, const uint8_t* trunc,
                     const void* bv, const void* boot, float* adv, float* ret, int64_t N,
                     int64_t T, float gamma, float lambda, rlcs_dtype dtype, void* ws,
                     size_t ws_bytes, rlcs_stream_t stream) {
    rlcs_status st = check_common(N, T, dtype, {r, v, bv, boot}, {adv, ret});
    if (st != RLCS_OK) return st;
    if (!unit_interval(gamma) || !unit_interval(lambda)) return RLCS_ERR_INVALID_ARG;
    if (N == 0 || T == 0) return RLCS_OK;
    if (!r || !v || !adv || (trunc && !bv)) return RLCS_ERR_INVALID_ARG;
    Args a = make_args(N, T, gamma, lambda, 1.f, 1.f);
    a.in[0] = r; a.in[1] = v; a.in[2] = bv;
    a.term = term; a.trunc = trunc; a.row_value = boot;
    a.out0 = adv; a.out1 = ret;
    return dispatch<GaeOp>(a, dtype, trunc != nullptr, ws, ws_bytes, stream);
}

}  // extern "C"
