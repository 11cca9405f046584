// Strided [N, T] entry points of the backward estimators (Table 1; Sections 3.3.1-3.3.4): the
// same recurrences as the row-major entry points, for any layout with element (n, t) at
// n * stride_n + t * stride_t (time-major buffers, strided rows). The plain row-major layout
// goes to the row-major entry point; every other to the column scans.
#include "rlcs_columns_dispatch.h"

using namespace rlcs;
using namespace rlcs::host;

extern "C" {

rlcs_status rlcs_gae_strided(const void* r, const void* v, const uint8_t* term,
                             const uint8_t* trunc, const void* bv, const void* boot, float* adv,
                             float* ret, int64_t N, int64_t T, int64_t stride_n, int64_t stride_t,
                             float gamma, float lambda, rlcs_dtype dtype, void* ws,
                             size_t ws_bytes, rlcs_stream_t stream) {
    ColGeom g;
    bool dense;
    rlcs_status st = check_strided(N, T, stride_n, stride_t, dtype, {r, v, bv, boot}, {adv, ret}, g, dense);
    if (st != RLCS_OK) return st;
    if (!unit_interval(gamma) || !unit_interval(lambda)) return RLCS_ERR_INVALID_ARG;
    if (N == 0 || T == 0) return RLCS_OK;
    if (!r || !v || !adv || (trunc && !bv)) return RLCS_ERR_INVALID_ARG;
    if (dense) return rlcs_gae(r, v, term, trunc, bv, boot, adv, ret, N, T, gamma, lambda, dtype, ws, ws_bytes, stream);
    Args a = make_args(N, T, gamma, lambda, 1.f, 1.f);
    a.in[0] = r; a.in[1] = v; a.in[2] = bv;
    a.term = term; a.trunc = trunc; a.row_value = boot;
    a.out0 = adv; a.out1 = ret;
    if (stride_t == 1) return dispatch_strided_rows<GaeOp>(a, stride_n, dtype, trunc != nullptr, stream);
    return col_dispatch<GaeOp>(a, g, dtype, trunc != nullptr, ws, ws_bytes, stream);
}

rlcs_status rlcs_vtrace_strided(const void* r, const void* v, const void* log_rho,
                                const uint8_t* term, const uint8_t* trunc, const void* bv,
                                const void* boot, float* vs, float* pg, int64_t N, int64_t T,
                                int64_t stride_n, int64_t stride_t, float gamma, float rho_bar,
                                float c_bar, rlcs_dtype dtype, void* ws, size_t ws_bytes,
                                rlcs_stream_t stream) {
    ColGeom g;
    bool dense;
    rlcs_status st = check_strided(N, T, stride_n, stride_t, dtype, {r, v, log_rho, bv, boot}, {vs, pg}, g, dense);
    if (st != RLCS_OK) return st;
    if (!unit_interval(gamma) || !positive(rho_bar) || !positive(c_bar)) return RLCS_ERR_INVALID_ARG;
    if (N == 0 || T == 0) return RLCS_OK;
    if (!r || !v || !log_rho || !vs || (trunc && !bv)) return RLCS_ERR_INVALID_ARG;
    if (dense) return rlcs_vtrace(r, v, log_rho, term, trunc, bv, boot, vs, pg, N, T, gamma, rho_bar, c_bar, dtype, ws, ws_bytes, stream);
    Args a = make_args(N, T, gamma, 1.f, rho_bar, c_bar);
    a.in[0] = r; a.in[1] = v; a.in[2] = log_rho; a.in[3] = bv;
    a.term = term; a.trunc = trunc; a.row_value = boot;
    a.out0 = vs; a.out1 = pg;
    if (stride_t == 1) return dispatch_strided_rows<VtraceOp>(a, stride_n, dtype, trunc != nullptr, stream);
    return col_dispatch<VtraceOp>(a, g, dtype, trunc != nullptr, ws, ws_bytes, stream);
}

rlcs_status rlcs_retrace_strided(const void* r, const void* q, const void* eq, const void* log_rho,
                                 const uint8_t* term, const uint8_t* trunc, const void* bv,
                                 const void* boot, float* delta, float* q_ret, int64_t N,
                                 int64_t T, int64_t stride_n, int64_t stride_t, float gamma,
                                 float lambda, float c_bar, rlcs_dtype dtype, void* ws,
                                 size_t ws_bytes, rlcs_stream_t stream) {
    ColGeom g;
    bool dense;
    rlcs_status st = check_strided(N, T, stride_n, stride_t, dtype, {r, q, eq, log_rho, bv, boot},
                                   {delta, q_ret}, g, dense);
    if (st != RLCS_OK) return st;
    if (!unit_interval(gamma) || !unit_interval(lambda) || !positive(c_bar)) return RLCS_ERR_INVALID_ARG;
    if (N == 0 || T == 0) return RLCS_OK;
    if (!r || !q || !eq || !log_rho || !delta || (trunc && !bv)) return RLCS_ERR_INVALID_ARG;
    if (dense) return rlcs_retrace(r, q, eq, log_rho, term, trunc, bv, boot, delta, q_ret, N, T, gamma, lambda, c_bar, dtype, ws, ws_bytes, stream);
    Args a = make_args(N, T, gamma, lambda, 1.f, c_bar);
    a.in[0] = r; a.in[1] = q; a.in[2] = eq; a.in[3] = log_rho; a.in[4] = bv;
    a.term = term; a.trunc = trunc; a.row_value = boot;
    a.out0 = delta; a.out1 = q_ret;
    if (stride_t == 1) return dispatch_strided_rows<RetraceOp>(a, stride_n, dtype, trunc != nullptr, stream);
    return col_dispatch<RetraceOp>(a, g, dtype, trunc != nullptr, ws, ws_bytes, stream);
}

rlcs_status rlcs_td_lambda_strided(const void* r, const void* v, const uint8_t* term,
                                   const uint8_t* trunc, const void* bv, const void* boot,
                                   float* ret, int64_t N, int64_t T, int64_t stride_n,
                                   int64_t stride_t, float gamma, float lambda, rlcs_dtype dtype,
                                   void* ws, size_t ws_bytes, rlcs_stream_t stream) {
    ColGeom g;
    bool dense;
    rlcs_status st = check_strided(N, T, stride_n, stride_t, dtype, {r, v, bv, boot}, {ret}, g, dense);
    if (st != RLCS_OK) return st;
    if (!unit_interval(gamma) || !unit_interval(lambda)) return RLCS_ERR_INVALID_ARG;
    if (N == 0 || T == 0) return RLCS_OK;
    if (!r || !v || !ret || (trunc && !bv)) return RLCS_ERR_INVALID_ARG;
    if (dense) return rlcs_td_lambda(r, v, term, trunc, bv, boot, ret, N, T, gamma, lambda, dtype, ws, ws_bytes, stream);
    Args a = make_args(N, T, gamma, lambda, 1.f, 1.f);
    a.in[0] = r; a.in[1] = v; a.in[2] = bv;
    a.term = term; a.trunc = trunc; a.row_value = boot;
    a.out0 = ret;
    if (stride_t == 1) return dispatch_strided_rows<TdLambdaOp>(a, stride_n, dtype, trunc != nullptr, stream);
    return col_dispatch<TdLambdaOp>(a, g, dtype, trunc != nullptr, ws, ws_bytes, stream);
}

rlcs_status rlcs_discounted_strided(const void* r, const uint8_t* term, const uint8_t* trunc,
                                    const void* bv, const void* boot, float* ret, int64_t N,
                                    int64_t T, int64_t stride_n, int64_t stride_t, float gamma,
                                    rlcs_dtype dtype, void* ws, size_t ws_bytes,
                                    rlcs_stream_t stream) {
    ColGeom g;
    bool dense;
    rlcs_status st = check_strided(N, T, stride_n, stride_t, dtype, {r, bv, boot}, {ret}, g, dense);
    if (st != RLCS_OK) return st;
    if (!unit_interval(gamma)) return RLCS_ERR_INVALID_ARG;
    if (N == 0 || T == 0) return RLCS_OK;
    if (!r || !ret || (trunc && !bv)) return RLCS_ERR_INVALID_ARG;
    if (dense) return rlcs_discounted(r, term, trunc, bv, boot, ret, N, T, gamma, dtype, ws, ws_bytes, stream);
    Args a = make_args(N, T, gamma, 1.f, 1.f, 1.f);
    a.in[0] = r; a.in[1] = bv;
    a.term = term; a.trunc = trunc; a.row_value = boot;
    a.out0 = ret;
    if (stride_t == 1) return dispatch_strided_rows<DiscountedOp>(a, stride_n, dtype, trunc != nullptr, stream);
    return col_dispatch<DiscountedOp>(a, g, dtype, trunc != nullptr, ws, ws_bytes, stream);
}

}  // extern "C"
