// Retrace(lambda) entry points, per-step and full form (Table 1; Sections 3.3.3 and 7.3).
#include "rlcs_dispatch.h"

using namespace rlcs;
using namespace rlcs::host;

extern "C" {

rlcs_status rlcs_retrace(const void* r, const void* q, const void* eq, const void* log_rho,
                         const uint8_t* term, const uint8_t* trunc, const void* bv,
                         const void* boot, float* delta, float* q_ret, int64_t N, int64_t T,
                         float gamma, float lambda, float c_bar, rlcs_dtype dtype, void* ws,
                         size_t ws_bytes, rlcs_stream_t stream) {
    rlcs_status st = check_common(N, T, dtype, {r, q, eq, log_rho, bv, boot}, {delta, q_ret});
    if (st != RLCS_OK) return st;
    if (!unit_interval(gamma) || !unit_interval(lambda) || !positive(c_bar)) return RLCS_ERR_INVALID_ARG;
    if (N == 0 || T == 0) return RLCS_OK;
    if (!r || !q || !eq || !log_rho || !delta || (trunc && !bv)) return RLCS_ERR_INVALID_ARG;
    Args a = make_args(N, T, gamma, lambda, 1.f, c_bar);
    a.in[0] = r; a.in[1] = q; a.in[2] = eq; a.in[3] = log_rho; a.in[4] = bv;
    a.term = term; a.trunc = trunc; a.row_value = boot;
    a.out0 = delta; a.out1 = q_ret;
    return dispatch<RetraceOp>(a, dtype, trunc != nullptr, ws, ws_bytes, stream);
}

rlcs_status rlcs_retrace_full(const void* r, const void* q, const void* pi,
                              const int32_t* actions, const void* mu, const uint8_t* term,
                              const uint8_t* trunc, const void* bv, const void* boot,
                              float* delta, float* q_ret, int64_t N, int64_t T, int64_t A,
                              float gamma, float lambda, float c_bar, rlcs_dtype dtype,
                              void* ws, size_t ws_bytes, rlcs_stream_t stream) {
    rlcs_status st = check_common(N, T, dtype, {r, q, pi, mu, bv, boot}, {delta, q_ret});
    if (st != RLCS_OK) return st;
    if (!unit_interval(gamma) || !unit_interval(lambda) || !positive(c_bar)) return RLCS_ERR_INVALID_ARG;
    if (A < 1 || A > INT32_MAX) return RLCS_ERR_INVALID_ARG;
    if (N == 0 || T == 0) return RLCS_OK;
    if (N * T > INT64_MAX / A) return RLCS_ERR_INVALID_ARG;
    if (!r || !q || !pi || !actions || !mu || !delta || (trunc && !bv)) return RLCS_ERR_INVALID_ARG;
    if (!aligned(actions, 4)) return RLCS_ERR_INVALID_ARG;
    Args a = make_args(N, T, gamma, lambda, 1.f, c_bar);
    a.in[0] = r; a.in[1] = q; a.in[2] = pi; a.in[3] = mu; a.in[4] = bv;
    a.actions = actions; a.A = A;
    a.stage_vec = (aligned(q, 16) && aligned(pi, 16)) ? 1 : 0;
    a.term = term; a.trunc = trunc; a.row_value = boot;
    a.out0 = delta; a.out1 = q_ret;
    // a workspace, if given, receives the out-of-range-action report in its error word
    a.ws = (ws && ws_bytes >= sizeof(WsHeader) && aligned(ws, 64)) ? ws : nullptr;
    if (A > kMaxActions)
        return dispatch<RetraceFullSlicedOp>(a, dtype, trunc != nullptr, nullptr, 0, stream);
    return dispatch<RetraceFullOp>(a, dtype, trunc != nullptr, nullptr, 0, stream);
}

}  // extern "C"
