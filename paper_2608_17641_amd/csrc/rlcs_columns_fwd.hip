// Column-scan entry points of the forward recurrences (Table 1; Sections 3.3.5-3.3.6):
// strided eligibility traces and prefix sums, eligibility traces of F-vectors, and the
// workspace size of the column scans.
#include "rlcs_columns_dispatch.h"
#include "rlcs_vec.h"

using namespace rlcs;
using namespace rlcs::host;

extern "C" {

rlcs_status rlcs_elig_trace_strided(const void* x, const uint8_t* term, const uint8_t* trunc,
                                    float* z, int64_t N, int64_t T, int64_t stride_n,
                                    int64_t stride_t, float gamma, float lambda, rlcs_dtype dtype,
                                    void* ws, size_t ws_bytes, rlcs_stream_t stream) {
    ColGeom g;
    bool dense;
    rlcs_status st = check_strided(N, T, stride_n, stride_t, dtype, {x}, {z}, g, dense);
    if (st != RLCS_OK) return st;
    if (!unit_interval(gamma) || !unit_interval(lambda)) return RLCS_ERR_INVALID_ARG;
    if (N == 0 || T == 0) return RLCS_OK;
    if (!x || !z) return RLCS_ERR_INVALID_ARG;
    if (dense) return rlcs_elig_trace(x, term, trunc, z, N, T, gamma, lambda, dtype, ws, ws_bytes, stream);
    Args a = make_args(N, T, gamma, lambda, 1.f, 1.f);
    a.in[0] = x;
    a.term = term; a.trunc = trunc;
    a.out0 = z;
    if (stride_t == 1) return dispatch_strided_rows<ForwardOp<true, false>>(a, stride_n, dtype, trunc != nullptr, stream);
    return col_dispatch<ForwardOp<true, false>>(a, g, dtype, trunc != nullptr, ws, ws_bytes, stream);
}

rlcs_status rlcs_episodic_prefix_strided(const void* x, const uint8_t* term, const uint8_t* trunc,
                                         float* c, int64_t N, int64_t T, int64_t stride_n,
                                         int64_t stride_t, rlcs_boundary boundary,
                                         rlcs_dtype dtype, void* ws, size_t ws_bytes,
                                         rlcs_stream_t stream) {
    ColGeom g;
    bool dense;
    rlcs_status st = check_strided(N, T, stride_n, stride_t, dtype, {x}, {c}, g, dense);
    if (st != RLCS_OK) return st;
    if (boundary != RLCS_ENDS_AT && boundary != RLCS_STARTS_AT) return RLCS_ERR_INVALID_ARG;
    if (N == 0 || T == 0) return RLCS_OK;
    if (!x || !c) return RLCS_ERR_INVALID_ARG;
    if (dense) return rlcs_episodic_prefix(x, term, trunc, c, N, T, boundary, dtype, ws, ws_bytes, stream);
    Args a = make_args(N, T, 1.f, 1.f, 1.f, 1.f);
    a.in[0] = x;
    a.term = term; a.trunc = trunc;
    a.out0 = c;
    if (boundary == RLCS_STARTS_AT) {
        if (stride_t == 1) return dispatch_strided_rows<ForwardOp<false, true>>(a, stride_n, dtype, trunc != nullptr, stream);
        return col_dispatch<ForwardOp<false, true>>(a, g, dtype, trunc != nullptr, ws, ws_bytes, stream);
    }
    if (stride_t == 1) return dispatch_strided_rows<ForwardOp<false, false>>(a, stride_n, dtype, trunc != nullptr, stream);
    return col_dispatch<ForwardOp<false, false>>(a, g, dtype, trunc != nullptr, ws, ws_bytes, stream);
}

rlcs_status rlcs_elig_trace_vec(const void* x, const uint8_t* term, const uint8_t* trunc,
                                float* z, int64_t N, int64_t T, int64_t F, float gamma,
                                float lambda, rlcs_dtype dtype, void* ws, size_t ws_bytes,
                                rlcs_stream_t stream) {
    if (N < 0 || T < 0 || F < 0) return RLCS_ERR_INVALID_ARG;
    if (dtype != RLCS_F32 && dtype != RLCS_BF16) return RLCS_ERR_DTYPE;
    if (T > kMaxT || (T > 0 && F > 0 && N > INT64_MAX / T / F)) return RLCS_ERR_INVALID_ARG;
    if (x && !aligned(x, dtype_size(dtype))) return RLCS_ERR_INVALID_ARG;
    if (z && !aligned(z, 4)) return RLCS_ERR_INVALID_ARG;
    if (!unit_interval(gamma) || !unit_interval(lambda)) return RLCS_ERR_INVALID_ARG;
    if (N == 0 || T == 0 || F == 0) return RLCS_OK;
    if (!x || !z) return RLCS_ERR_INVALID_ARG;
    Args a = make_args(N, T, gamma, lambda, 1.f, 1.f);
    a.in[0] = x;
    a.term = term; a.trunc = trunc;
    a.out0 = z;
    // Rows of vectors when they fit the row kernel (not under a forced column variant).
    if (g_variant == 0 && aligned(x, 16) && aligned(z, 16)) {
        const int wf = T % 4 == 0 && (!term || aligned(term, 4)) && (!trunc || aligned(trunc, 4));
        hipStream_t s = reinterpret_cast<hipStream_t>(stream);
        bool done;
        if (dtype == RLCS_BF16)
            done = trunc ? vec_rows_launch<bf16_t, true>(a, F, wf, s) : vec_rows_launch<bf16_t, false>(a, F, wf, s);
        else
            done = trunc ? vec_rows_launch<float, true>(a, F, wf, s) : vec_rows_launch<float, false>(a, F, wf, s);
        if (done) return hipGetLastError() == hipSuccess ? RLCS_OK : RLCS_ERR_LAUNCH;
    }
    // column n*F + f: feature f of row n; flags one per step of a row; non-temporal stores
    // when a step's F outputs fill whole 128-byte lines
    const ColGeom g{N * F, F, F, T * F, 1, T, 0, F % 32 == 0 ? 1 : 0};
    return col_dispatch<ForwardOp<true, false>>(a, g, dtype, trunc != nullptr, ws, ws_bytes, stream);
}

size_t rlcs_workspace_size_columns(int64_t columns, int64_t T) {
    if (columns < 0 || T < 0) return 0;
    return col_ws_need(columns, T);
}

}  // extern "C"
