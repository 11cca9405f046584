// Forward-scan entry points: eligibility traces and episodic prefix sums (Table 1; Sections 3.3.5-3.3.6).
#include "rlcs_dispatch.h"

using namespace rlcs;
using namespace rlcs::host;

extern "C" {

rlcs_status rlcs_elig_trace(const void* x, const uint8_t* term, const uint8_t* trunc, float* z,
                            int64_t N, int64_t T, float gamma, float lambda, rlcs_dtype dtype,
                            void* ws, size_t ws_bytes, rlcs_stream_t stream) {
    rlcs_status st = check_common(N, T, dtype, {x}, {z});
    if (st != RLCS_OK) return st;
    if (!unit_interval(gamma) || !unit_interval(lambda)) return RLCS_ERR_INVALID_ARG;
    if (N == 0 || T == 0) return RLCS_OK;
    if (!x || !z) return RLCS_ERR_INVALID_ARG;
    Args a = make_args(N, T, gamma, lambda, 1.f, 1.f);
    a.in[0] = x;
    a.term = term; a.trunc = trunc;
    a.out0 = z;
    return dispatch<ForwardOp<true, false>>(a, dtype, trunc != nullptr, ws, ws_bytes, stream);
}

rlcs_status rlcs_episodic_prefix(const void* x, const uint8_t* term, const uint8_t* trunc,
                                 float* c, int64_t N, int64_t T, rlcs_boundary boundary,
                                 rlcs_dtype dtype, void* ws, size_t ws_bytes,
                                 rlcs_stream_t stream) {
    rlcs_status st = check_common(N, T, dtype, {x}, {c});
    if (st != RLCS_OK) return st;
    if (boundary != RLCS_ENDS_AT && boundary != RLCS_STARTS_AT) return RLCS_ERR_INVALID_ARG;
    if (N == 0 || T == 0) return RLCS_OK;
    if (!x || !c) return RLCS_ERR_INVALID_ARG;
    Args a = make_args(N, T, 1.f, 1.f, 1.f, 1.f);
    a.in[0] = x;
    a.term = term; a.trunc = trunc;
    a.out0 = c;
    if (boundary == RLCS_STARTS_AT)
        return dispatch<ForwardOp<false, true>>(a, dtype, trunc != nullptr, ws, ws_bytes, stream);
    return dispatch<ForwardOp<false, false>>(a, dtype, trunc != nullptr, ws, ws_bytes, stream);
}

}  // extern "C"
