// V-Trace entry point (Table 1; Section 3.3.2).
#include "rlcs_dispatch.h"

using namespace rlcs;
using namespace rlcs::host;

extern "C" {

rlcs_status rlcs_vtrace(const void* r, const void* v, const void* log_rho, const uint8_t* term,
                        const uint8_t* trunc, const void* bv, const void* boot, float* vs,
                        float* pg, int64_t N, int64_t T, float gamma, float rho_bar, float c_bar,
                        rlcs_dtype dtype, void* ws, size_t ws_bytes, rlcs_stream_t stream) {
    rlcs_status st = check_common(N, T, dtype, {r, v, log_rho, bv, boot}, {vs, pg});
    if (st != RLCS_OK) return st;
    if (!unit_interval(gamma) || !positive(rho_bar) || !positive(c_bar)) return RLCS_ERR_INVALID_ARG;
    if (N == 0 || T == 0) return RLCS_OK;
    if (!r || !v || !log_rho || !vs || (trunc && !bv)) return RLCS_ERR_INVALID_ARG;
    Args a = make_args(N, T, gamma, 1.f, rho_bar, c_bar);
    a.in[0] = r; a.in[1] = v; a.in[2] = log_rho; a.in[3] = bv;
    a.term = term; a.trunc = trunc; a.row_value = boot;
    a.out0 = vs; a.out1 = pg;
    return dispatch<VtraceOp>(a, dtype, trunc != nullptr, ws, ws_bytes, stream);
}

}  // extern "C"
