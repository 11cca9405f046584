// GAE with observation-skip masking and optional advantage whitening (Section 9.3; Table 1 and
// Section 3.3.1 for the unmasked steps).
#include <mutex>

#include "rlcs_dispatch.h"
#include "rlcs_masked.h"

using namespace rlcs;
using namespace rlcs::host;

namespace {

// Bytes of the whitening workspace of an [N, T] call (at most one workgroup per row): the
// 64-byte header (statistics, arrival word, statistics record), the one-pass form's moments
// records (kFusedMaxGroups of 48 bytes), then the two-pass form's partials: one 32-byte
// partial per workgroup (room for N), then one per block of kDirectPartials partials.
constexpr size_t masked_rows(int64_t N) { return size_t(N > 0 ? N : 1); }
constexpr size_t masked_ws_need(int64_t N) {
    return kMaskedTwoPassOff +
           sizeof(Moments) * (masked_rows(N) + (masked_rows(N) + kDirectPartials - 1) / kDirectPartials);
}

template <typename DT, bool VEC, bool TR, bool HM, bool STATS>
void launch_masked(const MaskedArgs& ma, int waves, int64_t groups, int64_t rows_per_wg,
                   int wave_local, hipStream_t s) {
    constexpr int K = Width<DT>::K;
    if (waves == 1)
        hipLaunchKernelGGL((masked_gae_kernel<DT, K, 1, VEC, TR, HM, STATS>),
                           dim3(unsigned(groups)), dim3(kWave), 0, s, ma,
                           rows_per_wg, wave_local);
    else if (waves == kSmallWaves)
        hipLaunchKernelGGL((masked_gae_kernel<DT, K, kSmallWaves, VEC, TR, HM, STATS>),
                           dim3(unsigned(groups)), dim3(kSmallWaves * kWave), 0, s, ma,
                           rows_per_wg, wave_local);
    else
        hipLaunchKernelGGL((masked_gae_kernel<DT, K, kLargeWaves, VEC, TR, HM, STATS>),
                           dim3(unsigned(groups)), dim3(kLargeWaves * kWave), 0, s, ma,
                           rows_per_wg, wave_local);
}

// The one-pass whitened call (16-wave workgroups) when its grid is resident at once; false
// when it is not (the caller then runs the two-pass form).
template <typename DT, bool VEC, bool TR, bool HM>
bool launch_fused(const MaskedArgs& ma, int64_t groups, int64_t rows_per_wg, int wave_local,
                  float eps, void* ws, hipStream_t s) {
    constexpr int K = Width<DT>::K;
    constexpr int W = kLargeWaves;
    const auto kernel = masked_gae_fused_kernel<DT, K, W, VEC, TR, HM>;
    if (groups > int64_t(W) * kWave || groups > resident_groups(kernel, W * kWave)) return false;
    hipLaunchKernelGGL(kernel, dim3(unsigned(groups)), dim3(W * kWave), 0, s, ma, rows_per_wg,
                       wave_local, eps, static_cast<char*>(ws));
    return true;
}

template <typename DT>
rlcs_status run_masked(MaskedArgs& ma, bool normalize, float eps, void* ws, hipStream_t s) {
    constexpr int K = Width<DT>::K;
    const Args& a = ma.a;
    const int64_t N = a.N, T = a.T;
    constexpr int64_t E_small = int64_t(kSmallWaves) * kWave * K;
    // Rows of 32*K to 64*K steps without whitening: one-wave workgroups, as for GAE (4096 x 256
    // multi-turn 5.79 -> 5.54 us). With whitening they would quadruple the partials that every
    // normalize workgroup adds up (12.4 -> 13.6 us), so those calls keep four waves.
    const bool one_wave = !normalize && T % K == 0 && (int64_t(kWave) * K) % T == 0 && T >= 32 * K;
    const int waves = (T <= E_small) ? (one_wave ? 1 : kSmallWaves) : kLargeWaves;
    const int64_t E = int64_t(waves) * kWave * K;
    const int64_t slack = (T % K == 0) ? 0 : K - 1;
    const int64_t rows_per_wg = (T <= E - slack) ? (E - slack) / T : 1;
    const int64_t groups = (N + rows_per_wg - 1) / rows_per_wg;
    if (groups > INT32_MAX) return RLCS_ERR_INVALID_ARG;
    const int wave_local = (T % K == 0 && (int64_t(kWave) * K) % T == 0) ? 1 : 0;
    bool vec = aligned(a.in[0], 16) && aligned(a.in[1], 16) && (!a.trunc || aligned(a.in[2], 16)) &&
               aligned(a.out0, 16) && (!a.out1 || aligned(a.out1, 16)) &&
               (!a.term || aligned(a.term, K)) && (!a.trunc || aligned(a.trunc, K)) &&
               (!ma.mask || aligned(ma.mask, K));
    const bool tr = a.trunc != nullptr, hm = ma.mask != nullptr;
    constexpr int64_t E_large = int64_t(kLargeWaves) * kWave * K;
    if (normalize && T <= E_large - slack && g_variant != 1) {
        // every row in one 16-wave chunk: the one-pass form when the grid is resident at once
        const int64_t rows16 = (E_large - slack) / T;
        const int64_t groups16 = (N + rows16 - 1) / rows16;
        bool fused = false;
#define RLCS_FUSED(V, TRV, HMV) fused = launch_fused<DT, V, TRV, HMV>(ma, groups16, rows16, wave_local, eps, ws, s)
#define RLCS_FUSED_HM(V, TRV) \
    if (hm) { RLCS_FUSED(V, TRV, true); } else { RLCS_FUSED(V, TRV, false); }
#define RLCS_FUSED_TR(V) \
    if (tr) { RLCS_FUSED_HM(V, true); } else { RLCS_FUSED_HM(V, false); }
        if (groups16 <= kFusedMaxGroups) {
            if (vec) { RLCS_FUSED_TR(true); } else { RLCS_FUSED_TR(false); }
        }
#undef RLCS_FUSED_TR
#undef RLCS_FUSED_HM
#undef RLCS_FUSED
        if (fused) return hipGetLastError() == hipSuccess ? RLCS_OK : RLCS_ERR_LAUNCH;
    }
    double* stats = reinterpret_cast<double*>(ws);
    Moments* level2 = nullptr;
    if (normalize) {
        ma.partials = reinterpret_cast<Moments*>(reinterpret_cast<char*>(ws) + kMaskedTwoPassOff);
        level2 = ma.partials + masked_rows(N);
    }
#define RLCS_MASKED(V, TRV, HMV, ST) launch_masked<DT, V, TRV, HMV, ST>(ma, waves, groups, rows_per_wg, wave_local, s)
#define RLCS_MASKED_ST(V, TRV, HMV) \
    if (normalize) RLCS_MASKED(V, TRV, HMV, true); else RLCS_MASKED(V, TRV, HMV, false)
#define RLCS_MASKED_HM(V, TRV) \
    if (hm) { RLCS_MASKED_ST(V, TRV, true); } else { RLCS_MASKED_ST(V, TRV, false); }
#define RLCS_MASKED_TR(V) \
    if (tr) { RLCS_MASKED_HM(V, true); } else { RLCS_MASKED_HM(V, false); }
    if (vec) { RLCS_MASKED_TR(true); } else { RLCS_MASKED_TR(false); }
#undef RLCS_MASKED_TR
#undef RLCS_MASKED_HM
#undef RLCS_MASKED_ST
#undef RLCS_MASKED
    if (normalize) {
        const int64_t total = N * T;
        const int64_t per_wg = int64_t(kNormThreads) * kNormVec * 4;  // elements
        const int64_t grid = (total + per_wg - 1) / per_wg;
        if (grid > INT32_MAX) return RLCS_ERR_INVALID_ARG;
        const Moments* part = ma.partials;
        int64_t G = groups;
        if (G > kDirectPartials) {
            const int64_t blocks = (G + kDirectPartials - 1) / kDirectPartials;
            hipLaunchKernelGGL(masked_sum_partials_kernel, dim3(unsigned(blocks)), dim3(kNormThreads),
                               0, s, ma.partials, G, level2);
            part = level2;
            G = blocks;
        }
        hipLaunchKernelGGL(masked_normalize_kernel, dim3(unsigned(grid)), dim3(kNormThreads), 0, s,
                           a.out0, total, part, G, eps, stats, aligned(a.out0, 16) ? 1 : 0);
    }
    return hipGetLastError() == hipSuccess ? RLCS_OK : RLCS_ERR_LAUNCH;
}

// The whitening workspace of rlcs_gae_masked_noalloc: a static device array sized for calls of
// up to kNoAllocMaxRows rows (2.2 MiB), zero-filled when the library's code is loaded on a
// device (static storage), one copy per GPU, held until the process ends. Host code
// never uses the array's name as an address: the device address comes from
// hipGetSymbolAddress, once per device, and every call on a device shares that device's copy.
constexpr int64_t kNoAllocMaxRows = 65536;
constexpr size_t kNoAllocScratchBytes = masked_ws_need(kNoAllocMaxRows);
static_assert(kNoAllocScratchBytes % 64 == 0, "the scratch holds whole 64-byte units");

constexpr int kMaxDevices = 64;

}  // namespace

static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace {

// Device address of `scratch` on the current device (nullptr if it cannot be had), looked up
// with that device current on its first use and kept per device.
void* scratch_address() {
    static std::mutex mu;
    static void* addr[kMaxDevices] = {};
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> lock(mu);
    if (!addr[dev]) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess) return nullptr;
        addr[dev] = p;
    }
    return addr[dev];
}

// Argument checks of the masked entry points (host only, before any HIP call).
rlcs_status check_masked(const void* r, const void* v, const uint8_t* trunc, const void* bv,
                         const void* boot, const float* adv, const float* ret, int64_t N, int64_t T,
                         float gamma, float lambda, int normalize, float eps, rlcs_dtype dtype) {
    const rlcs_status st = check_common(N, T, dtype, {r, v, bv, boot}, {adv, ret});
    if (st != RLCS_OK) return st;
    if (!unit_interval(gamma) || !unit_interval(lambda)) return RLCS_ERR_INVALID_ARG;
    if (normalize != 0 && normalize != 1) return RLCS_ERR_INVALID_ARG;
    if (normalize && !(eps >= 0.f && eps < INFINITY)) return RLCS_ERR_INVALID_ARG;
    if (N == 0 || T == 0) return RLCS_OK;
    if (!r || !v || !adv || (trunc && !bv)) return RLCS_ERR_INVALID_ARG;
    return RLCS_OK;
}

// A checked, non-empty call (ws: the whitening workspace when normalize).
rlcs_status masked_call(const void* r, const void* v, const uint8_t* mask, const uint8_t* term,
                        const uint8_t* trunc, const void* bv, const void* boot, float* adv,
                        float* ret, int64_t N, int64_t T, float gamma, float lambda, bool normalize,
                        float eps, rlcs_dtype dtype, void* ws, hipStream_t s) {
    MaskedArgs ma{};
    ma.a = make_args(N, T, gamma, lambda, 1.f, 1.f);
    ma.a.in[0] = r; ma.a.in[1] = v; ma.a.in[2] = bv;
    ma.a.term = term; ma.a.trunc = trunc; ma.a.row_value = boot;
    ma.a.out0 = adv; ma.a.out1 = ret;
    ma.mask = mask;
    if (dtype == RLCS_BF16) return run_masked<bf16_t>(ma, normalize, eps, ws, s);
    return run_masked<float>(ma, normalize, eps, ws, s);
}

}  // namespace

extern "C" {

rlcs_status rlcs_gae_masked_noalloc(const void* r, const void* v, const uint8_t* mask,
                                    const uint8_t* term, const uint8_t* trunc, const void* bv,
                                    const void* boot, float* adv, float* ret, int64_t N, int64_t T,
                                    float gamma, float lambda, int normalize, float eps,
                                    rlcs_dtype dtype, rlcs_stream_t stream) {
    if (N > kNoAllocMaxRows) return RLCS_ERR_WORKSPACE;
    const rlcs_status st = check_masked(r, v, trunc, bv, boot, adv, ret, N, T, gamma, lambda,
                                        normalize, eps, dtype);
    if (st != RLCS_OK || N == 0 || T == 0) return st;
    void* ws = nullptr;
    if (normalize) {
        ws = scratch_address();
        if (!ws) return RLCS_ERR_LAUNCH;
    }
    return masked_call(r, v, mask, term, trunc, bv, boot, adv, ret, N, T, gamma, lambda,
                       normalize != 0, eps, dtype, ws, reinterpret_cast<hipStream_t>(stream));
}

rlcs_status rlcs_gae_masked(const void* r, const void* v, const uint8_t* mask,
                            const uint8_t* term, const uint8_t* trunc, const void* bv,
                            const void* boot, float* adv, float* ret, int64_t N, int64_t T,
                            float gamma, float lambda, int normalize, float eps,
                            rlcs_dtype dtype, void* ws, size_t ws_bytes, rlcs_stream_t stream) {
    const rlcs_status st = check_masked(r, v, trunc, bv, boot, adv, ret, N, T, gamma, lambda,
                                        normalize, eps, dtype);
    if (st != RLCS_OK || N == 0 || T == 0) return st;
    if (normalize && (!ws || ws_bytes < masked_ws_need(N) || !aligned(ws, 64)))
        return RLCS_ERR_WORKSPACE;
    return masked_call(r, v, mask, term, trunc, bv, boot, adv, ret, N, T, gamma, lambda,
                       normalize != 0, eps, dtype, ws, reinterpret_cast<hipStream_t>(stream));
}

size_t rlcs_workspace_size_masked(int64_t N, int64_t T) {
    if (N < 0 || T < 0) return 0;
    return masked_ws_need(N);
}

}  // extern "C"
