// Host side of the rlcs C ABI: argument checks (all before any HIP call), choice of kernel
// variant, and launches. The kernels themselves are in rlcs_kernels.h.
#include <hip/hip_runtime.h>

#include <atomic>
#include <climits>
#include <cstdint>

#include "rlcs.h"
#include "rlcs_kernels.h"

using namespace rlcs;

namespace {

// Waves per workgroup: 4 for rows of up to 4*64*K steps (several rows per workgroup), 16 for
// longer rows (one row, or a 16*64*K-step tile of one, per workgroup).
constexpr int kSmallWaves = 4;
constexpr int kLargeWaves = 16;
// Staged policies (full-form Retrace) use 4 waves, or 1 when the action axis is too long for
// a 4-wave chunk's slices to fit the LDS budget.
constexpr int kStagedWaves = 1;
constexpr int64_t kStagedLdsBudget = 64 * 1024;

// Steps per lane: one 16-byte vector of each input.
template <typename DT> struct Width;
template <> struct Width<float> { static constexpr int K = 4; };
template <> struct Width<bf16_t> { static constexpr int K = 8; };

// Smallest tile of the split-row variant (float32), which sizes the workspace.
constexpr int64_t kMinTile = int64_t(kLargeWaves) * kWave * Width<float>::K;

// Rows longer than one large workgroup's chunk are split across workgroups (when a workspace
// is given) only if there are too few rows for whole-row workgroups to fill the GPU.
constexpr int64_t kSplitBelowRows = 1024;

// Largest action axis of full-form Retrace (its [steps, A] slices are staged in LDS).
constexpr int64_t kMaxActions = 28;

// Longest supported row (the kernels keep offsets within a row range in 32 bits).
constexpr int64_t kMaxT = int64_t(1) << 30;

std::atomic<int> g_variant{0};

bool aligned(const void* p, size_t a) { return reinterpret_cast<uintptr_t>(p) % a == 0; }
bool unit_interval(float x) { return x >= 0.f && x <= 1.f; }  // false for NaN
bool positive(float x) { return x > 0.f; }                     // false for NaN, true for +inf

size_t dtype_size(rlcs_dtype d) { return d == RLCS_BF16 ? 2 : 4; }

// Common checks of sizes, dtype and the element alignment of every given pointer.
rlcs_status check_common(int64_t N, int64_t T, rlcs_dtype dtype,
                         std::initializer_list<const void*> data, std::initializer_list<const void*> outs) {
    if (N < 0 || T < 0) return RLCS_ERR_INVALID_ARG;
    if (dtype != RLCS_F32 && dtype != RLCS_BF16) return RLCS_ERR_DTYPE;
    if (T > kMaxT || (T > 0 && N > INT64_MAX / T)) return RLCS_ERR_INVALID_ARG;
    const size_t es = dtype_size(dtype);
    for (const void* p : data)
        if (p && !aligned(p, es)) return RLCS_ERR_INVALID_ARG;
    for (const void* p : outs)
        if (p && !aligned(p, 4)) return RLCS_ERR_INVALID_ARG;
    return RLCS_OK;
}

// How one call is run.
struct Plan {
    bool split;           // tiles kernel (rows split across workgroups) vs rows kernel
    int waves;            // waves per workgroup
    int64_t num_tiles;    // tiles kernel: grid size
    int64_t rows_per_wg;  // rows kernel: rows per workgroup
    int wave_local;       // rows kernel: no carry crosses waves
    size_t lds_bytes;     // dynamic LDS (staged policies)
};

template <class Op, typename DT, bool VEC, bool TR, int W>
void launch_w(const Args& a, const Plan& p, hipStream_t stream) {
    constexpr int K = Width<DT>::K;
    const dim3 block(W * kWave);
    if constexpr (Op::kStaged == 0) {
        if (p.split) {
            hipLaunchKernelGGL((tiles_kernel<Op, DT, K, W, VEC, TR>), dim3(unsigned(p.num_tiles)),
                               block, 0, stream, a, p.num_tiles);
            return;
        }
    }
    const int64_t groups = (a.N + p.rows_per_wg - 1) / p.rows_per_wg;
    hipLaunchKernelGGL((rows_kernel<Op, DT, K, W, VEC, TR>), dim3(unsigned(groups)), block,
                       p.lds_bytes, stream, a, p.rows_per_wg, p.wave_local);
}

template <class Op, typename DT, bool VEC, bool TR>
rlcs_status launch(const Args& a, const Plan& p, hipStream_t stream) {
    if constexpr (Op::kStaged > 0) {
        if (p.waves == kStagedWaves) launch_w<Op, DT, VEC, TR, kStagedWaves>(a, p, stream);
        else launch_w<Op, DT, VEC, TR, kSmallWaves>(a, p, stream);
    } else {
        if (p.split) launch_w<Op, DT, VEC, TR, kLargeWaves>(a, p, stream);
        else if (p.waves == kSmallWaves) launch_w<Op, DT, VEC, TR, kSmallWaves>(a, p, stream);
        else launch_w<Op, DT, VEC, TR, kLargeWaves>(a, p, stream);
    }
    return hipGetLastError() == hipSuccess ? RLCS_OK : RLCS_ERR_LAUNCH;
}

// LDS bytes of a staged policy's chunk with W waves: the staged slots plus the two
// [steps, A] slices.
template <class Op, typename DT>
constexpr int64_t staged_lds_bytes(int W, int64_t A) {
    const int64_t E = int64_t(W) * kWave * Width<DT>::K;
    return int64_t(sizeof(float)) * Op::kStaged * (E + 4) + 2 * (E + 1) * A * int64_t(sizeof(DT));
}

template <class Op, typename DT>
rlcs_status dispatch_dt(Args& a, bool has_trunc, void* ws, size_t ws_bytes, hipStream_t stream) {
    constexpr int K = Width<DT>::K;
    constexpr int64_t E_small = int64_t(kSmallWaves) * kWave * K;
    constexpr int64_t E_large = int64_t(kLargeWaves) * kWave * K;
    const int64_t N = a.N, T = a.T, total = N * T;

    // Vector path: 16-byte data and output vectors, K-byte flag vectors.
    bool vec = true;
    for (int s = 0; s < Op::kSlots; ++s)
        if (Op::slot_used(s, has_trunc) && !aligned(a.in[s], 16)) vec = false;
    if (!aligned(a.out0, 16) || (a.out1 && !aligned(a.out1, 16))) vec = false;
    if (Op::kFlags && ((a.term && !aligned(a.term, K)) || (has_trunc && !aligned(a.trunc, K)))) vec = false;

    Plan p{};
    p.num_tiles = (total + E_large - 1) / E_large;
    const size_t ws_need = sizeof(WsHeader) + size_t(p.num_tiles) * kWsRecordBytes;
    const bool ws_ok = ws && ws_bytes >= ws_need && aligned(ws, 64) && p.num_tiles < int64_t(UINT32_MAX);
    const int forced = g_variant.load(std::memory_order_relaxed);
    if constexpr (Op::kStaged > 0) {
        // Staged policies keep whole rows in one workgroup (chunk loop for long rows).
        p.split = false;
        if (staged_lds_bytes<Op, DT>(kSmallWaves, a.A) <= kStagedLdsBudget) p.waves = kSmallWaves;
        else if (staged_lds_bytes<Op, DT>(kStagedWaves, a.A) <= kStagedLdsBudget) p.waves = kStagedWaves;
        else return RLCS_ERR_INVALID_ARG;
        p.lds_bytes = size_t(staged_lds_bytes<Op, DT>(p.waves, a.A));
    } else {
        if (forced == 2) {
            if (!ws_ok) return RLCS_ERR_WORKSPACE;
            p.split = true;
        } else if (forced == 1) {
            p.split = false;
        } else {
            p.split = T > E_large && ws_ok && N < kSplitBelowRows;
        }
        p.waves = p.split ? kLargeWaves : ((T <= E_small) ? kSmallWaves : kLargeWaves);
        p.lds_bytes = 0;
    }
    if (p.split) {
        if (p.num_tiles > INT32_MAX) return RLCS_ERR_INVALID_ARG;
        a.ws = ws;
    } else {
        const int64_t E = int64_t(p.waves) * kWave * K;
        // Whole rows per workgroup: as many as fit in one chunk (at least one). When T is not
        // a multiple of K a row range may start mid-vector, costing up to K-1 extra slots.
        const int64_t slack = (T % K == 0) ? 0 : K - 1;
        p.rows_per_wg = (T <= E - slack) ? (E - slack) / T : 1;
        if ((N + p.rows_per_wg - 1) / p.rows_per_wg > INT32_MAX) return RLCS_ERR_INVALID_ARG;
        // Rows never straddle waves when T divides a wave's span (and is a multiple of K).
        p.wave_local = (T % K == 0 && (int64_t(kWave) * K) % T == 0) ? 1 : 0;
    }

    if constexpr (Op::kFlags) {
        if (has_trunc) {
            return vec ? launch<Op, DT, true, true>(a, p, stream)
                       : launch<Op, DT, false, true>(a, p, stream);
        }
    }
    return vec ? launch<Op, DT, true, false>(a, p, stream)
               : launch<Op, DT, false, false>(a, p, stream);
}

template <class Op>
rlcs_status dispatch(Args& a, rlcs_dtype dtype, bool has_trunc, void* ws, size_t ws_bytes,
                     rlcs_stream_t stream) {
    if (a.N == 0 || a.T == 0) return RLCS_OK;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    if (dtype == RLCS_BF16) return dispatch_dt<Op, bf16_t>(a, has_trunc, ws, ws_bytes, s);
    return dispatch_dt<Op, float>(a, has_trunc, ws, ws_bytes, s);
}

Args make_args(int64_t N, int64_t T, float gamma, float lambda, float rho_bar, float c_bar) {
    Args a{};
    a.N = N;
    a.T = T;
    a.inv_T = T > 0 ? 1.f / float(T) : 0.f;
    a.p = Params{gamma, lambda, rho_bar, c_bar};
    return a;
}

}  // namespace

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
    if (A < 1 || A > kMaxActions) return RLCS_ERR_INVALID_ARG;
    if (N == 0 || T == 0) return RLCS_OK;
    if (N * T > INT64_MAX / A) return RLCS_ERR_INVALID_ARG;
    if (!r || !q || !pi || !actions || !mu || !delta || (trunc && !bv)) return RLCS_ERR_INVALID_ARG;
    if (!aligned(actions, 4)) return RLCS_ERR_INVALID_ARG;
    Args a = make_args(N, T, gamma, lambda, 1.f, c_bar);
    a.in[0] = r; a.in[1] = q; a.in[2] = pi; a.in[3] = mu; a.in[4] = bv;
    a.actions = actions; a.A = A;
    a.term = term; a.trunc = trunc; a.row_value = boot;
    a.out0 = delta; a.out1 = q_ret;
    return dispatch<RetraceFullOp>(a, dtype, trunc != nullptr, ws, ws_bytes, stream);
}

rlcs_status rlcs_td_lambda(const void* r, const void* v, const uint8_t* term,
                           const uint8_t* trunc, const void* bv, const void* boot, float* ret,
                           int64_t N, int64_t T, float gamma, float lambda, rlcs_dtype dtype,
                           void* ws, size_t ws_bytes, rlcs_stream_t stream) {
    rlcs_status st = check_common(N, T, dtype, {r, v, bv, boot}, {ret});
    if (st != RLCS_OK) return st;
    if (!unit_interval(gamma) || !unit_interval(lambda)) return RLCS_ERR_INVALID_ARG;
    if (N == 0 || T == 0) return RLCS_OK;
    if (!r || !v || !ret || (trunc && !bv)) return RLCS_ERR_INVALID_ARG;
    Args a = make_args(N, T, gamma, lambda, 1.f, 1.f);
    a.in[0] = r; a.in[1] = v; a.in[2] = bv;
    a.term = term; a.trunc = trunc; a.row_value = boot;
    a.out0 = ret;
    return dispatch<TdLambdaOp>(a, dtype, trunc != nullptr, ws, ws_bytes, stream);
}

rlcs_status rlcs_discounted(const void* r, const uint8_t* term, const uint8_t* trunc,
                            const void* bv, const void* boot, float* ret, int64_t N, int64_t T,
                            float gamma, rlcs_dtype dtype, void* ws, size_t ws_bytes,
                            rlcs_stream_t stream) {
    rlcs_status st = check_common(N, T, dtype, {r, bv, boot}, {ret});
    if (st != RLCS_OK) return st;
    if (!unit_interval(gamma)) return RLCS_ERR_INVALID_ARG;
    if (N == 0 || T == 0) return RLCS_OK;
    if (!r || !ret || (trunc && !bv)) return RLCS_ERR_INVALID_ARG;
    Args a = make_args(N, T, gamma, 1.f, 1.f, 1.f);
    a.in[0] = r; a.in[1] = bv;
    a.term = term; a.trunc = trunc; a.row_value = boot;
    a.out0 = ret;
    return dispatch<DiscountedOp>(a, dtype, trunc != nullptr, ws, ws_bytes, stream);
}

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

size_t rlcs_workspace_size(int64_t N, int64_t T) {
    if (N <= 0 || T <= 0) return sizeof(WsHeader);
    if (N > INT64_MAX / T) return 0;
    const int64_t tiles = (N * T + kMinTile - 1) / kMinTile;
    return sizeof(WsHeader) + size_t(tiles) * kWsRecordBytes;
}

const char* rlcs_status_string(rlcs_status status) {
    switch (status) {
        case RLCS_OK: return "RLCS_OK";
        case RLCS_ERR_INVALID_ARG: return "RLCS_ERR_INVALID_ARG: invalid size, pointer, parameter or enum";
        case RLCS_ERR_DTYPE: return "RLCS_ERR_DTYPE: unsupported dtype";
        case RLCS_ERR_WORKSPACE: return "RLCS_ERR_WORKSPACE: workspace missing or too small";
        case RLCS_ERR_LAUNCH: return "RLCS_ERR_LAUNCH: kernel launch failed";
    }
    return "unknown rlcs_status";
}

int rlcs_version(void) { return 100; }

rlcs_status rlcs_set_variant_override(int variant) {
    if (variant < 0 || variant > 2) return RLCS_ERR_INVALID_ARG;
    g_variant.store(variant, std::memory_order_relaxed);
    return RLCS_OK;
}

}  // extern "C"
